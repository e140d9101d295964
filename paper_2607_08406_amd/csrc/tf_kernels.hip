// HIP kernels (gfx950) of the decoder Transformer path of MCA (Sec. 2.5):
// the candidate stream over all parameter tensors,
// each candidate's forward pass from the first stage its parameter changes,
// the per-position cross-entropy and its change against the committed
// per-position losses, and the commit.
//
// Every candidate has a slot: its own copy of the mutated tensor (patched
// with the new value), a table of tensor pointers, and its activations.  A
// launch covers all K candidates (grid z or y); a candidate whose parameter
// lies in a later stage skips the stage and the next stage reads the
// committed residual stream.  The kernels are deterministic and treat every
// position alike, so a position the mutation cannot reach (before a changed
// position-embedding row, say) reproduces its committed loss bit for bit and
// adds exactly zero to the loss change.  The commit copies the winner's slot
// into the committed state.
//
// The model (pre-LN blocks, learned positions, erf GELU, final LayerNorm,
// untied output layer with bias; linear layers y = x W^T + b) is the reading
// of the paper fixed for the oracle.  The dense products run on the matrix
// cores (v_mfma_f32_16x16x4f32); LayerNorm, attention, GELU and the loss in
// fp32 on the vector units.
#include <algorithm>

#include "tf_kernels.hpp"

namespace mca {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGemmThreads = 256;  // 4 waves, a 128 x 128 output tile, 64 x 64 per wave
constexpr int kGemmRows = 128;     // rows (positions) per block
constexpr int kGemmCols = 128;     // output columns per block
constexpr int kChunkK = 16;        // reduction chunk staged in LDS
constexpr int kLnThreads = 256;    // a wave per row, kLnRows rows per wave
constexpr int kLnRows = 16;
constexpr int kLossThreads = 256;
constexpr int kCopyThreads = 256;
constexpr int kCopyChunk = 4096;   // floats of a private tensor copy per block
constexpr int kEmbedPer = 4;       // embedding elements per thread

__device__ __forceinline__ float* slot_x(const TfDev* tf, int k, int b) {
  return tf->sx + ((int64_t)k * (tf->NB + 1) + b) * tf->N * tf->D;
}
__device__ __forceinline__ float* slot_h(const TfDev* tf, int k, int b) {
  return tf->sh + ((int64_t)k * tf->NB + b) * tf->N * tf->D;
}
__device__ __forceinline__ float* slot_ln2(const TfDev* tf, int k, int b) {
  return tf->sln2 + ((int64_t)k * tf->NB + b) * tf->N * tf->D;
}
__device__ __forceinline__ float* slot_u(const TfDev* tf, int k, int b) {
  return tf->su + ((int64_t)k * tf->NB + b) * tf->N * tf->M;
}
__device__ __forceinline__ float* slot_fc(const TfDev* tf, int k) { return tf->sfc + (int64_t)k * tf->N * tf->M; }
__device__ __forceinline__ float* slot_log(const TfDev* tf, int k) { return tf->slog + (int64_t)k * tf->N * tf->V; }
__device__ __forceinline__ float* slot_nhat(const TfDev* tf, int k) { return tf->snhat + (int64_t)k * tf->N * tf->D; }
// x_{stage-1}, the residual stream entering stage `stage` (1..NB+1): the
// candidate's own once it has changed, the committed one before
__device__ __forceinline__ const float* stage_input(const TfDev* tf, int k, int stage) {
  return (tf->xin[k] > stage - 1) ? tf->x[stage - 1] : slot_x(tf, k, stage - 1);
}
// erf by Abramowitz and Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf x = 1 - (a1 t + ... + a5 t^5) e^{-x^2}, t = 1 / (1 + p x), x >= 0,
// absolute error at most 1.5e-7 (odd extension for x < 0).
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  float p = 1.061405429f;
  p = fmaf(p, t, -1.453152027f);
  p = fmaf(p, t, 1.421413741f);
  p = fmaf(p, t, -0.284496736f);
  p = fmaf(p, t, 0.254829592f);
  p *= t;
  const float e = __builtin_amdgcn_exp2f(-(ax * ax) * 1.4426950408889634f);
  const float r = 1.0f - p * e;
  return copysignf(r, x);
}
// GELU with the exact (erf) form; the erf error above is about one fp32 ulp
// of the result.
__device__ __forceinline__ float gelu(float y) {
  return 0.5f * y * (1.0f + erf_as(y * 0.70710678118654752f));
}

// The change of logit v at position n under an output-layer candidate
// (kTfOutCol: only logit c.j moves, by de times the final LayerNorm output
// of column c.i, or de for the bias) or a final-LayerNorm candidate
// (kTfLnfCol: column c.j of that output moves by de times its normalized
// value, or de for the bias, and reaches every logit through W_out[:, c.j]).
// The evaluation and the commit use this one expression.
__device__ __forceinline__ float out_delta(const TfDev* tf, int kind, const mca_cand& c, float de,
                                           int64_t n, int v) {
  const int D = tf->D, nt = tf->n_tensors;
  if (kind == kTfOutCol) {
    if (v != c.j) return 0.f;
    if (c.layer == nt - 1) return de;
    const float lnf = tf->cnhat[n * D + c.i] * tf->param[nt - 4][c.i] + tf->param[nt - 3][c.i];
    return de * lnf;
  }
  const float dl = (c.layer == nt - 4) ? de * tf->cnhat[n * D + c.j] : de;
  return dl * tf->param[nt - 2][(int64_t)v * D + c.j];
}

// The new pre-activation of hidden unit c.j of block b at position n under an
// up-projection candidate (weight: de times the LN2 output of column c.i;
// bias: de), and the change of its GELU.
__device__ __forceinline__ float fc_new_u(const TfDev* tf, const mca_cand& c, float de, int b,
                                          int role, int64_t n) {
  const float u = tf->cu[b][n * tf->M + c.j];
  const float du = (role == kBfc) ? de : de * tf->cln2[b][n * tf->D + c.i];
  return u + du;
}
__device__ __forceinline__ float fc_change(const TfDev* tf, const mca_cand& c, float de, int b,
                                           int role, int64_t n) {
  return gelu(fc_new_u(tf, c, de, b, role, n)) - gelu(tf->cu[b][n * tf->M + c.j]);
}

}  // namespace

// ---------------------------------------------------------------------------
// candidate stream (Eq. 1) over the canonical parameter order
// ---------------------------------------------------------------------------

__global__ void k_tf_propose(const TfDev* tf, uint64_t t_host, int use_dev_t,
                             const DevState* st, int K, mca_cand* cands, Aux* aux) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const uint64_t t = use_dev_t ? st->t : t_host;
  const Words w = philox4x64_10(t, (uint64_t)k, 0, 0, tf->seed, tf->tag);
  const int64_t flat = (int64_t)__umul64hi(w.w0, (uint64_t)tf->P);
  int layer = 0;
  for (int l = 1; l < tf->n_tensors; ++l)
    if (flat >= tf->offs[l]) layer = l;
  const int64_t off = flat - tf->offs[layer];
  const int64_t cols = tf->cols[layer];
  mca_cand c;
  c.flat = flat;
  c.layer = layer;
  c.j = (int32_t)(off / cols);
  c.i = (int32_t)(off - (int64_t)c.j * cols);
  const float m = (float)(uint32_t)(w.w2 >> 40);
  const float r = m * 0x1p-23f - 1.0f;
  c.d = tf->delta * r;
  c.code = 0;
  c.flags = 0;
  cands[k] = c;
  Aux a;
  a.w_old = tf->param[layer][off];
  a.w_new = a.w_old + c.d;
  a.de = a.w_new - a.w_old;
  a.valid = !(tf->bound > 0.f && fabsf(a.w_new) >= tf->bound);
  a.theta = accept_theta(tf->rule, tf->beta, tf->seed, tf->tag, t, (uint64_t)k);
  aux[k] = a;
}

__global__ void k_tf_prepare(const TfDev* tf, const mca_cand* cands, int K, Aux* aux) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const mca_cand c = cands[k];
  Aux a;
  a.w_old = tf->param[c.layer][(int64_t)c.j * tf->cols[c.layer] + c.i];
  a.w_new = a.w_old + c.d;
  a.de = a.w_new - a.w_old;
  a.valid = !(tf->bound > 0.f && fabsf(a.w_new) >= tf->bound);
  a.theta = 0.0;
  aux[k] = a;
}

// Blocks (x, k): candidate k's patched private copy of its tensor, a chunk of
// kCopyChunk floats per block; block (0, k) also writes the tensor table and
// the candidate's first stage.  identity: slot 0 with the committed tensors.
// mode kPrepEval: every candidate of the batch; kPrepIdentity: slot 0 with
// the committed tensors (cache fill); kPrepRedo (before a commit, a grid of
// one slot): the chosen candidate (k_host, or st->chosen when negative) is
// recomputed as a dense candidate if it was evaluated incrementally, and
// the pass does nothing otherwise.  The kind array is left as the
// evaluation wrote it, so that every block takes the same decision.
enum { kPrepEval = 0, kPrepIdentity = 1, kPrepRedo = 2 };
__global__ __launch_bounds__(kCopyThreads) void k_tf_prep(const TfDev* tf, const mca_cand* cands,
                                                          const Aux* aux, int mode, int k_host,
                                                          const DevState* st) {
  int k = blockIdx.y;
  if (mode == kPrepRedo) {
    const int kc = (k_host >= 0) ? k_host : st->chosen;
    const bool redo = kc >= 0 && tf->kind[kc] != kTfDense;
    k = kc >= 0 ? kc : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      *tf->pass = k;
      if (!redo) tf->run[k] = tf->NB + 2;
    }
    if (!redo) return;
  } else if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
    *tf->pass = -1;
  }
  const int nt = tf->n_tensors;
  float** tab = tf->table + (int64_t)k * nt;
  if (mode == kPrepIdentity) {
    if (blockIdx.x == 0) {
      for (int t = threadIdx.x; t < nt; t += blockDim.x) tab[t] = tf->param[t];
      if (threadIdx.x == 0) {
        tf->start[k] = tf->run[k] = 0;
        tf->xin[k] = 0;
        tf->kind[k] = kTfDense;
      }
    }
    return;
  }
  const mca_cand c = cands[k];
  const Aux a = aux[k];
  const int l = c.layer, NB = tf->NB;
  int kind = kTfDense;
  if (l >= nt - 2) kind = kTfOutCol;
  else if (l >= nt - 4) kind = kTfLnfCol;
  else if (l >= 2) {
    const int role = (l - 2) % kBlockTensors;
    if (role == kWproj || role == kBproj) kind = kTfProjCol;
    if (role == kWfc || role == kBfc) kind = kTfFcCol;
  }
  if (mode == kPrepRedo) kind = kTfDense;
  const bool dense = kind == kTfDense;
  float* cp = tf->scopy + (int64_t)k * tf->copy_stride;
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < nt; t += blockDim.x)
      tab[t] = (t == l && a.valid && dense) ? cp : tf->param[t];
    if (threadIdx.x == 0) {
      const int blk = (l - 2) / kBlockTensors;
      int start = NB + 2, xin = NB + 2;  // nothing recomputed: rejected, or the last stage's own
      if (a.valid && dense) start = xin = tf_stage(l, NB);
      if (a.valid && (kind == kTfProjCol || kind == kTfFcCol)) {
        start = blk + 2;  // the stages after the block, from its patched output stream
        xin = blk + 1;
      }
      tf->start[k] = tf->run[k] = start;
      tf->xin[k] = xin;
      if (mode != kPrepRedo) tf->kind[k] = a.valid ? kind : kTfDense;
    }
  }
  if (!a.valid || !dense) return;
  const int64_t n = (int64_t)tf->rows[l] * tf->cols[l];
  const int64_t at = (int64_t)c.j * tf->cols[l] + c.i;
  const float* src = tf->param[l];
  const int64_t e0 = (int64_t)blockIdx.x * kCopyChunk;
  for (int64_t e = e0 + threadIdx.x; e < n && e < e0 + kCopyChunk; e += blockDim.x)
    cp[e] = (e == at) ? a.w_new : src[e];
}

// x_{b+1} of an MLP candidate of block b (kTfProjCol, kTfFcCol): the
// committed stream plus the candidate's change, from the committed
// pre-activations and LN2 output of the block.
__global__ __launch_bounds__(kCopyThreads) void k_tf_patch(const TfDev* tf, const mca_cand* cands,
                                                           const Aux* aux) {
  const int k = tf_slot(tf, blockIdx.y);
  const int kind = tf->kind[k];
  if (kind != kTfProjCol && kind != kTfFcCol) return;
  const mca_cand c = cands[k];
  const float de = aux[k].de;
  const int D = tf->D, M = tf->M;
  const int b = (c.layer - 2) / kBlockTensors, role = (c.layer - 2) % kBlockTensors;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= tf->N * D) return;
  const int64_t n = e / D;
  const int col = (int)(e - n * D);
  float dx = 0.f;
  if (kind == kTfProjCol) {
    if (col == c.j) dx = (role == kBproj) ? de : de * gelu(tf->cu[b][n * M + c.i]);
  } else {
    dx = fc_change(tf, c, de, b, role, n) *
         tf->param[2 + kBlockTensors * b + kWproj][(int64_t)col * M + c.j];
  }
  slot_x(tf, k, b + 1)[e] = tf->x[b + 1][e] + dx;
}

// x_0 = tok_emb[token] + pos_emb[position] for the candidates of stage 0
__global__ __launch_bounds__(kCopyThreads) void k_tf_embed(const TfDev* tf) {
  const int k = tf_slot(tf, blockIdx.y);
  if (tf->run[k] != 0) return;
  const int D = tf->D;
  const int64_t ND = tf->N * D;
  float* const* tab = tf->table + (int64_t)k * tf->n_tensors;
  const float* te = tab[0];
  const float* pe = tab[1];
  float* x0 = slot_x(tf, k, 0);
  const int64_t e0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * kEmbedPer;
#pragma unroll
  for (int u = 0; u < kEmbedPer; ++u) {
    const int64_t e = e0 + u;
    if (e < ND) {
      const int64_t n = e / D;
      const int c = (int)(e - n * D);
      const int pos = (int)(n % tf->T);
      x0[e] = te[(int64_t)tf->tok[n] * D + c] + pe[(int64_t)pos * D + c];
    }
  }
}

// LayerNorm (biased variance, eps inside the root, affine), a wave per row.
// which: 0 LN1 of the stage's block (input x_{stage-1}), 1 LN2 (input: after
// attention), 2 the final LayerNorm (stage NB+1).
__global__ __launch_bounds__(kLnThreads) void k_tf_ln(const TfDev* tf, int stage, int which) {
  const int k = tf_slot(tf, blockIdx.y);
  if (tf->run[k] > stage) return;
  const int D = tf->D;
  const int64_t N = tf->N, ND = N * D;
  const int lane = threadIdx.x & 63;
  float* const* tab = tf->table + (int64_t)k * tf->n_tensors;
  const int tb = 2 + kBlockTensors * (stage - 1);
  const float* in;
  const float *g, *bb;
  if (which == 0) {
    in = stage_input(tf, k, stage);
    g = tab[tb + kLn1G];
    bb = tab[tb + kLn1B];
  } else if (which == 1) {
    in = slot_h(tf, k, stage - 1);
    g = tab[tb + kLn2G];
    bb = tab[tb + kLn2B];
  } else {
    in = stage_input(tf, k, stage);
    g = tab[tf->n_tensors - 4];
    bb = tab[tf->n_tensors - 3];
  }
  const float eps = tf->eps;
  float* const outk = (which == 1) ? slot_ln2(tf, k, stage - 1) : tf->sln + k * ND;
  float* const nhk = (which == 2) ? slot_nhat(tf, k) : nullptr;  // the final one, before its affine part
  constexpr int kMaxPer = 4;  // D <= 256
  float gv[kMaxPer], bv[kMaxPer];
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    gv[u] = (c < D) ? g[c] : 0.f;
    bv[u] = (c < D) ? bb[c] : 0.f;
  }
  const int64_t r0 = ((int64_t)blockIdx.x * (kLnThreads / 64) + (threadIdx.x >> 6)) * kLnRows;
  for (int64_t n = r0; n < r0 + kLnRows && n < N; ++n) {
    const float* inr = in + n * D;
    float v[kMaxPer];
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      const int c = lane + 64 * u;
      v[u] = (c < D) ? inr[c] : 0.f;
      s += v[u];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    const float mean = s / (float)D;
    float q = 0.f;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      const int c = lane + 64 * u;
      const float dv = (c < D) ? v[u] - mean : 0.f;
      q += dv * dv;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
    const float rstd = 1.0f / sqrtf(q / (float)D + eps);
    float* out = outk + n * D;
#pragma unroll
    for (int u = 0; u < kMaxPer; ++u) {
      const int c = lane + 64 * u;
      const float nh = (v[u] - mean) * rstd;
      if (c < D) out[c] = nh * gv[u] + bv[u];
      if (nhk != nullptr && c < D) nhk[n * D + c] = nh;
    }
  }
}

// Y = X W^T + b with an epilogue, for the candidates active in `stage`.
// A 128 x 128 output tile per block; wave (wr, wc) takes the 64 x 64
// quarter (wr, wc) as four by four 16 x 16 MFMA tiles, so each operand
// fragment read from LDS feeds four MFMAs.  The reduction dimension runs in
// chunks of 16 staged in LDS (double-buffered: the next chunk's global loads
// are in flight while the current one is multiplied).  Inside a chunk, k runs in blocks of 16; lane group q holds
// k = 16 kb + 4 q + t (t = 0..3), used by four MFMAs in turn, so each lane
// reads its operands as float4.  Rows and columns beyond the matrix are
// clamped on load and dropped on store.  Requires Kd % 16 == 0.  The Q, K and
// V projections are one product with 3 D output columns: column n takes its
// weight row and bias from tensor n / D of the three.
// EPI: 0 bias only (Q, K, V; output layer), 1 GELU (MLP up), 2 residual
// (attention output, MLP down): each epilogue gets its own register budget;
// without a residual to hold, three blocks share a CU (40 KB of LDS each).
template <int EPI>
__global__ __launch_bounds__(kGemmThreads, EPI == 2 ? 2 : 3) void k_tf_gemm(const TfDev* tf, int stage, int role) {
  const int k = tf_slot(tf, blockIdx.z);
  if (tf->run[k] > stage) return;
  const int D = tf->D, M = tf->M, V = tf->V;
  const int64_t N = tf->N, ND = N * D;
  float* const* tab = tf->table + (int64_t)k * tf->n_tensors;
  const int b = stage - 1;
  const int tb = 2 + kBlockTensors * b;
  const float* X = tf->sln + k * ND;
  int ldX = D, Kd = D, ldY = D, Nout = D;
  bool qkv = false;
  const float *W = nullptr, *bias = nullptr, *R = nullptr;
  float* Y = nullptr;
  float* Y2 = nullptr;  // the MLP's pre-activations (before the GELU epilogue)
  switch (role) {
    case kGemmQKV:
      Y = tf->sqkv + 3 * k * ND; ldY = 3 * D; Nout = 3 * D; qkv = true;
      break;
    case kGemmO:
      X = tf->satt + k * ND; W = tab[tb + kWo]; bias = tab[tb + kBo]; Y = slot_h(tf, k, b);
      R = stage_input(tf, k, stage);
      break;
    case kGemmFc:
      X = slot_ln2(tf, k, b); W = tab[tb + kWfc]; bias = tab[tb + kBfc]; Y = slot_fc(tf, k);
      Y2 = slot_u(tf, k, b); ldY = M; Nout = M;
      break;
    case kGemmProj:
      X = slot_fc(tf, k); ldX = M; Kd = M; W = tab[tb + kWproj]; bias = tab[tb + kBproj];
      Y = slot_x(tf, k, b + 1); R = slot_h(tf, k, b);
      break;
    default:  // kGemmOut: logits of the final stage
      W = tab[tf->n_tensors - 2]; bias = tab[tf->n_tensors - 1]; Y = slot_log(tf, k); ldY = V;
      Nout = V;
      break;
  }
  const int n0 = blockIdx.y * kGemmCols;
  if (n0 >= Nout) return;
  // weight row and bias of output column n
  auto wrow = [&](int n) -> const float* {
    if (!qkv) return W + (int64_t)n * Kd;
    const int w = n / D;
    return tab[tb + kWq + 2 * w] + (int64_t)(n - w * D) * Kd;
  };
  auto bias_of = [&](int n) -> float {
    if (!qkv) return bias[n];
    const int w = n / D;
    return tab[tb + kBq + 2 * w][n - w * D];
  };
  __shared__ __attribute__((aligned(16))) float As[2][kGemmRows][kChunkK + 4];
  __shared__ __attribute__((aligned(16))) float Bs[2][kGemmCols][kChunkK + 4];
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, q = lane >> 4, li = lane & 15;
  const int wr = wave >> 1, wc = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.x * kGemmRows;
  // staging: thread tid loads float4 number tid + 256 u of the A chunk
  // (128 rows x 8 float4) and of the B chunk (128 rows x 8 float4)
  constexpr int kA4 = kGemmRows * kChunkK / 4 / kGemmThreads;  // 4
  constexpr int kB4 = kGemmCols * kChunkK / 4 / kGemmThreads;  // 4
  const float* ga[kA4];
  const float* gb[kB4];
#pragma unroll
  for (int u = 0; u < kA4; ++u) {
    const int e = tid + kGemmThreads * u;
    const int64_t r = m0 + e / (kChunkK / 4);
    ga[u] = X + (r < N ? r : N - 1) * ldX + 4 * (e % (kChunkK / 4));
  }
#pragma unroll
  for (int u = 0; u < kB4; ++u) {
    const int e = tid + kGemmThreads * u;
    const int n = n0 + e / (kChunkK / 4);
    gb[u] = wrow(n < Nout ? n : Nout - 1) + 4 * (e % (kChunkK / 4));
  }
  floatx4 ra0[kA4], rb0[kB4];
  auto fetch = [&](int c, floatx4 (&ra)[kA4], floatx4 (&rb)[kB4]) {
#pragma unroll
    for (int u = 0; u < kA4; ++u) ra[u] = gload(reinterpret_cast<const floatx4*>(ga[u] + kChunkK * c));
#pragma unroll
    for (int u = 0; u < kB4; ++u) rb[u] = gload(reinterpret_cast<const floatx4*>(gb[u] + kChunkK * c));
  };
  auto store = [&](int buf, const floatx4 (&ra)[kA4], const floatx4 (&rb)[kB4]) {
#pragma unroll
    for (int u = 0; u < kA4; ++u) {
      const int e = tid + kGemmThreads * u;
      *reinterpret_cast<floatx4*>(&As[buf][e / (kChunkK / 4)][4 * (e % (kChunkK / 4))]) = ra[u];
    }
#pragma unroll
    for (int u = 0; u < kB4; ++u) {
      const int e = tid + kGemmThreads * u;
      *reinterpret_cast<floatx4*>(&Bs[buf][e / (kChunkK / 4)][4 * (e % (kChunkK / 4))]) = rb[u];
    }
  };
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  floatx4 acc[4][4];
#pragma unroll
  for (int sb = 0; sb < 4; ++sb)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[sb][cb] = zero;
  auto compute = [&](int buf) {
#pragma unroll
    for (int kb = 0; kb < kChunkK / 16; ++kb) {
      floatx4 a[4], bv[4];
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
        a[sb] = *reinterpret_cast<const floatx4*>(&As[buf][64 * wr + 16 * sb + li][16 * kb + 4 * q]);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        bv[cb] = *reinterpret_cast<const floatx4*>(&Bs[buf][64 * wc + 16 * cb + li][16 * kb + 4 * q]);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
          for (int cb = 0; cb < 4; ++cb)
            acc[sb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[sb][t], bv[cb][t], acc[sb][cb], 0, 0, 0);
    }
  };
  // D layout: lane (q, li), element v -> row 16 sb + 4 q + v, column 16 cb + li.
  // The residual a lane adds is loaded before the last chunk's products, so
  // its latency hides behind them.
  float res[4][4][4];
  (void)res;
  auto load_residual = [&]() {
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int64_t m = m0 + 64 * wr + 16 * sb + 4 * q + v;
          const int n = n0 + 64 * wc + 16 * cb + li;
          res[sb][cb][v] = (m < N && n < Nout) ? R[m * D + n] : 0.f;
        }
  };
  const int nc = Kd / kChunkK;
  fetch(0, ra0, rb0);
  store(0, ra0, rb0);
  __syncthreads();
  for (int c = 0; c < nc; ++c) {
    const int buf = c & 1;
    if (c + 1 < nc) fetch(c + 1, ra0, rb0);
    if constexpr (EPI == 2)
      if (c + 1 == nc) load_residual();
    compute(buf);
    if (c + 1 < nc) store(buf ^ 1, ra0, rb0);
    __syncthreads();
  }
  float bvv[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    const int n = n0 + 64 * wc + 16 * cb + li;
    bvv[cb] = (n < Nout) ? bias_of(n) : 0.f;
  }
#pragma unroll
  for (int sb = 0; sb < 4; ++sb)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t m = m0 + 64 * wr + 16 * sb + 4 * q + v;
        const int n = n0 + 64 * wc + 16 * cb + li;
        if (m < N && n < Nout) {
          float y = acc[sb][cb][v] + bvv[cb];
          if constexpr (EPI == 1) {
            Y2[m * ldY + n] = y;
            y = gelu(y);
          }
          if constexpr (EPI == 2) y = res[sb][cb][v] + y;
          Y[m * ldY + n] = y;
        }
      }
}

// Causal softmax attention, scale 1/sqrt(32), on the matrix cores: a block
// of 4 waves per (sequence, head) of one candidate.  Q, K and V of the
// sequence and head sit in LDS (rows padded).  Row block rb (16 queries)
// takes key blocks 0..rb: the scores S = Q K^T tile by tile (16 x 16, two
// k-blocks of 16 over the head dimension, operands read as float4), the row
// maximum and the sum of exponentials by a fixed butterfly over the 16 lanes
// that hold a row, then O = P V with P re-laid out through LDS into the
// A-operand layout.  Wave w takes row blocks w and 7-w (T = 128: every wave
// walks 9 tiles); keys after the query are masked.
__global__ __launch_bounds__(256) void k_tf_attn(const TfDev* tf, int stage) {
  const int k = tf_slot(tf, blockIdx.y);
  if (tf->run[k] > stage) return;
  constexpr int kS = kTfHeadDim + 4;  // padded row
  __shared__ __attribute__((aligned(16))) float Qs[kTfMaxCtx][kS];
  __shared__ __attribute__((aligned(16))) float Ks[kTfMaxCtx][kS];
  __shared__ __attribute__((aligned(16))) float Vs[kTfMaxCtx][kS];
  __shared__ float Ps[4][16][17];
  const int T = tf->T, D = tf->D, H = tf->H;
  const int s = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
  const int64_t ND = tf->N * D;
  const float* base = tf->sqkv + 3 * k * ND + (int64_t)s * T * 3 * D + h * kTfHeadDim;
  {
    // 128 rows x 8 float4 per tensor: four float4 of each per thread, every
    // load issued before the LDS stores
    constexpr int kPer = kTfMaxCtx * kTfHeadDim / 4 / 256;
    floatx4 rq[kPer], rk[kPer], rv[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int t = e / (kTfHeadDim / 4), c4 = e - t * (kTfHeadDim / 4);
      const bool ok = t < T;
      const float* row = base + (int64_t)(ok ? t : 0) * 3 * D + 4 * c4;
      const floatx4 z = {0.f, 0.f, 0.f, 0.f};
      rq[u] = ok ? gload(reinterpret_cast<const floatx4*>(row)) : z;
      rk[u] = ok ? gload(reinterpret_cast<const floatx4*>(row + D)) : z;
      rv[u] = ok ? gload(reinterpret_cast<const floatx4*>(row + 2 * D)) : z;
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int t = e / (kTfHeadDim / 4), c4 = e - t * (kTfHeadDim / 4);
      *reinterpret_cast<floatx4*>(&Qs[t][4 * c4]) = rq[u];
      *reinterpret_cast<floatx4*>(&Ks[t][4 * c4]) = rk[u];
      *reinterpret_cast<floatx4*>(&Vs[t][4 * c4]) = rv[u];
    }
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, q = lane >> 4, li = lane & 15;
  const int nrb = (T + 15) / 16;
  const float scale = 0.17677669529663687f;  // 1/sqrt(32)
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  float* outb = tf->satt + k * ND + (int64_t)s * T * D + h * kTfHeadDim;
  for (int pass = 0; pass < 2; ++pass) {
    const int rb = (pass == 0) ? wave : 7 - wave;
    if (rb >= nrb || (pass == 1 && rb == wave)) continue;
    // scores of row block rb against key blocks 0..rb
    floatx4 sc[kTfMaxCtx / 16];
    floatx4 qa[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      qa[kb] = *reinterpret_cast<const floatx4*>(&Qs[16 * rb + li][16 * kb + 4 * q]);
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb) {
      sc[cb] = zero;
      if (cb <= rb) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const floatx4 kk = *reinterpret_cast<const floatx4*>(&Ks[16 * cb + li][16 * kb + 4 * q]);
#pragma unroll
          for (int t = 0; t < 4; ++t)
            sc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(qa[kb][t], kk[t], sc[cb], 0, 0, 0);
        }
      }
    }
    // lane (q, li) holds scores of rows 16 rb + 4 q + v, keys 16 cb + li
    float mx[4], sm[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 16 * rb + 4 * q + v;
      float m = -__builtin_huge_valf();
#pragma unroll
      for (int cb = 0; cb < kTfMaxCtx / 16; ++cb)
        if (cb <= rb && 16 * cb + li <= row) m = fmaxf(m, sc[cb][v] * scale);
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      mx[v] = m;
      float sum = 0.f;
#pragma unroll
      for (int cb = 0; cb < kTfMaxCtx / 16; ++cb) {
        const float p = (cb <= rb && 16 * cb + li <= row) ? fast_exp(sc[cb][v] * scale - m) : 0.f;
        sc[cb][v] = p;
        sum += p;
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) sum += __shfl_xor(sum, o, 64);
      sm[v] = sum;
    }
    // O = P V: per key block, P through LDS into the A layout (row li, key 4 t + q)
    floatx4 oc[2] = {zero, zero};
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb) {
      if (cb > rb) break;  // uniform over the wave
#pragma unroll
      for (int v = 0; v < 4; ++v) Ps[wave][4 * q + v][li] = sc[cb][v];
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float pa = Ps[wave][li][4 * t + q];
        const int key = 16 * cb + 4 * t + q;
#pragma unroll
        for (int db = 0; db < 2; ++db)
          oc[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(pa, Vs[key][16 * db + li], oc[db], 0, 0, 0);
      }
      __builtin_amdgcn_wave_barrier();  // every lane read Ps before the next tile rewrites it
    }
    // lane (q, li) holds O rows 16 rb + 4 q + v, columns 16 db + li
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = 16 * rb + 4 * q + v;
      if (row < T) {
#pragma unroll
        for (int db = 0; db < 2; ++db) outb[(int64_t)row * D + 16 * db + li] = oc[db][v] / sm[v];
      }
    }
  }
}

// Per-position cross-entropy of the candidate's logits, its change against
// the committed loss, and the block's sum of changes over its 256 positions
// (in order).  The block's logits are contiguous; they are staged in LDS with
// coalesced loads and each thread then takes one position (row stride V).
__global__ __launch_bounds__(kLossThreads) void k_tf_ce(const TfDev* tf, const mca_cand* cands,
                                                        const Aux* aux, float* partial, int nblk,
                                                        int redo) {
  __shared__ float zl[kLossThreads * kTfMaxVocab];
  __shared__ float dl[kLossThreads];
  const int k = tf_slot(tf, blockIdx.y);
  const int kind = tf->kind[k];
  // from the committed logits (evaluation only: a redo reads the slot's own)
  const bool col = !redo && (kind == kTfOutCol || kind == kTfLnfCol);
  const bool active = tf->run[k] <= tf->NB + 1 || col;
  const int V = tf->V;
  const int64_t n0 = (int64_t)blockIdx.x * kLossThreads;
  const int64_t nrows = (tf->N - n0 < kLossThreads) ? tf->N - n0 : kLossThreads;
  if (active) {
    const float* zk = (col ? tf->cz : slot_log(tf, k)) + n0 * V;
    for (int64_t e = threadIdx.x; e < nrows * V; e += kLossThreads) zl[e] = zk[e];
  }
  __syncthreads();
  if (col) {  // the committed logits plus the candidate's change (out_delta)
    const mca_cand c = cands[k];
    const float de = aux[k].de;
    for (int64_t e = threadIdx.x; e < nrows * V; e += kLossThreads) {
      const int64_t r = e / V;
      const int v = (int)(e - r * V);
      zl[e] = zl[e] + out_delta(tf, kind, c, de, n0 + r, v);
    }
    __syncthreads();
  }
  const int r = threadIdx.x;
  float d = 0.f;
  if (active && r < nrows) {
    const float* z = zl + r * V;
    float m = z[0];
    for (int v = 1; v < V; ++v) m = fmaxf(m, z[v]);
    float sum = 0.f;
    for (int v = 0; v < V; ++v) sum += fast_exp(z[v] - m);
    const int64_t n = n0 + r;
    const float ln = (fast_log(sum) + m) - z[tf->tgt[n]];
    tf->sell[k * tf->N + n] = ln;
    d = ln - tf->ell[n];
  }
  dl[r] = d;
  __syncthreads();
  for (int o = kLossThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) dl[threadIdx.x] += dl[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[(int64_t)k * nblk + blockIdx.x] = dl[0];
}

// The winner's (or slot 0's, fill) state becomes the committed one: its
// residual streams from the first one it changed, the intermediate fields of
// every block it recomputed, the final normalized stream, the logits and the
// per-position losses (the winner was recomputed densely first when it had
// been evaluated incrementally); block 0 applies the parameter and the
// state.  One thread per element of the largest array (N x max(M, D, V)).
__global__ __launch_bounds__(kCopyThreads) void k_tf_commit(const TfDev* tf, const mca_cand* cands,
                                                            const Aux* aux, const double* dL,
                                                            DevState* st, int k_host, int fill) {
  const int k = fill ? 0 : ((k_host >= 0) ? k_host : st->chosen);
  if (k < 0) return;
  const int D = tf->D, M = tf->M, V = tf->V, NB = tf->NB;
  const int64_t N = tf->N, ND = N * D, NM = N * M, NV = N * V;
  const int s0 = fill ? 0 : tf->start[k];
  const int x0 = fill ? 0 : tf->xin[k];
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s0 <= NB + 1) {
    if (e < ND)
      for (int b = x0; b <= NB; ++b) tf->x[b][e] = slot_x(tf, k, b)[e];
    for (int b = 0; b < NB; ++b) {
      if (b + 1 < s0) continue;  // block b (stage b + 1) was not recomputed
      if (e < ND) {
        tf->ch[b][e] = slot_h(tf, k, b)[e];
        tf->cln2[b][e] = slot_ln2(tf, k, b)[e];
      }
      if (e < NM) tf->cu[b][e] = slot_u(tf, k, b)[e];
    }
    if (e < ND) tf->cnhat[e] = slot_nhat(tf, k)[e];
    if (e < NV) tf->cz[e] = slot_log(tf, k)[e];
    if (e < N) tf->ell[e] = tf->sell[(int64_t)k * N + e];
  }
  if (!fill && blockIdx.x == 0 && threadIdx.x == 0) {
    const mca_cand c = cands[k];
    tf->param[c.layer][(int64_t)c.j * tf->cols[c.layer] + c.i] = aux[k].w_new;
    st->L += dL[k];
    st->accepted += 1;
  }
}

__global__ __launch_bounds__(kLossThreads) void k_tf_loss_blocks(const TfDev* tf, double* bsum) {
  __shared__ double red[kLossThreads];
  const int64_t n = (int64_t)blockIdx.x * kLossThreads + threadIdx.x;
  red[threadIdx.x] = (n < tf->N) ? (double)tf->ell[n] : 0.0;
  __syncthreads();
  for (int o = kLossThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = red[0];
}

__global__ void k_tf_loss_total(const TfDev* tf, const double* bsum, int nb, DevState* st) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int b = 0; b < nb; ++b) s += bsum[b];
  st->L = s / (double)tf->N;
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

int tf_loss_blocks(int64_t N) { return (int)((N + kLossThreads - 1) / kLossThreads); }

hipError_t tf_launch_propose(const TfDev* tf, const TfDev& h, uint64_t t, bool use_dev_t,
                             const DevState* st, int K, mca_cand* cands, Aux* aux,
                             hipStream_t s) {
  (void)h;
  hipLaunchKernelGGL(k_tf_propose, dim3((K + 63) / 64), dim3(64), 0, s, tf, t, use_dev_t ? 1 : 0,
                     st, K, cands, aux);
  return hipGetLastError();
}

hipError_t tf_launch_prepare(const TfDev* tf, const mca_cand* cands, int K, Aux* aux,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_tf_prepare, dim3((K + 63) / 64), dim3(64), 0, s, tf, cands, K, aux);
  return hipGetLastError();
}

namespace {
// One pass of the stage kernels over the K slots: the patch of the MLP
// candidates (evaluation only), the embedding, each block, the final stage
// and the per-position losses.
hipError_t run_pass(const TfDev* tf, const TfDev& h, const mca_cand* cands, const Aux* aux,
                    unsigned KK, int mode, int k_host, const DevState* st, float* partial,
                    int nblk, hipStream_t s) {
  const int64_t N = h.N;
  const unsigned mt = (unsigned)((N + kGemmRows - 1) / kGemmRows);
  hipLaunchKernelGGL(k_tf_prep,
                     dim3((unsigned)((h.copy_stride + kCopyChunk - 1) / kCopyChunk), KK),
                     dim3(kCopyThreads), 0, s, tf, cands, aux, mode, k_host, st);
  if (mode == kPrepEval)
    hipLaunchKernelGGL(k_tf_patch,
                       dim3((unsigned)((N * h.D + kCopyThreads - 1) / kCopyThreads), KK),
                       dim3(kCopyThreads), 0, s, tf, cands, aux);
  hipLaunchKernelGGL(k_tf_embed,
                     dim3((unsigned)((N * h.D + kCopyThreads * kEmbedPer - 1) / (kCopyThreads * kEmbedPer)), KK),
                     dim3(kCopyThreads), 0, s, tf);
  const int64_t ln_rows = (int64_t)(kLnThreads / 64) * kLnRows;
  const dim3 lng((unsigned)((N + ln_rows - 1) / ln_rows), KK);
  for (int b = 0; b < h.NB; ++b) {
    const int stage = b + 1;
    hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, stage, 0);
    hipLaunchKernelGGL(k_tf_gemm<0>, dim3(mt, (unsigned)((3 * h.D + kGemmCols - 1) / kGemmCols), KK),
                       dim3(kGemmThreads), 0, s, tf, stage, (int)kGemmQKV);
    hipLaunchKernelGGL(k_tf_attn, dim3((unsigned)(h.S * h.H), KK), dim3(256), 0, s, tf, stage);
    hipLaunchKernelGGL(k_tf_gemm<2>, dim3(mt, (unsigned)((h.D + kGemmCols - 1) / kGemmCols), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmO);
    hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, stage, 1);
    hipLaunchKernelGGL(k_tf_gemm<1>, dim3(mt, (unsigned)((h.M + kGemmCols - 1) / kGemmCols), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmFc);
    hipLaunchKernelGGL(k_tf_gemm<2>, dim3(mt, (unsigned)((h.D + kGemmCols - 1) / kGemmCols), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmProj);
  }
  const int fin = h.NB + 1;
  hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, fin, 2);
  hipLaunchKernelGGL(k_tf_gemm<0>, dim3(mt, (unsigned)((h.V + kGemmCols - 1) / kGemmCols), KK), dim3(kGemmThreads), 0,
                     s, tf, fin, (int)kGemmOut);
  hipLaunchKernelGGL(k_tf_ce, dim3((unsigned)nblk, KK), dim3(kLossThreads), 0, s, tf, cands, aux,
                     partial, nblk, mode == kPrepRedo ? 1 : 0);
  return hipGetLastError();
}
}  // namespace

hipError_t tf_launch_eval(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                          const Aux* aux, int K, bool identity, float* partial, int nblk,
                          hipStream_t s) {
  return run_pass(tf, h, cands, aux, identity ? 1u : (unsigned)K,
                  identity ? kPrepIdentity : kPrepEval, -1, nullptr, partial, nblk, s);
}

hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, float* partial, int nblk, hipStream_t s) {
  if (!fill) {
    // the winner, if it was evaluated incrementally, recomputed densely
    const hipError_t e = run_pass(tf, h, cands, aux, 1u, kPrepRedo, k, st, partial, nblk, s);
    if (e != hipSuccess) return e;
  }
  const int64_t w = std::max(std::max(h.M, h.D), h.V);
  const int64_t n = h.N * w;
  hipLaunchKernelGGL(k_tf_commit, dim3((unsigned)((n + kCopyThreads - 1) / kCopyThreads)),
                     dim3(kCopyThreads), 0, s, tf, cands, aux, dL, st, k, fill ? 1 : 0);
  if (fill) {
    const int nb = tf_loss_blocks(h.N);
    hipLaunchKernelGGL(k_tf_loss_blocks, dim3(nb), dim3(kLossThreads), 0, s, tf, bsum);
    hipLaunchKernelGGL(k_tf_loss_total, dim3(1), dim3(64), 0, s, tf, bsum, nb, st);
  }
  return hipGetLastError();
}

}  // namespace mca
