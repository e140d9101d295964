// HIP kernels (gfx950) of the decoder Transformer path of MCA ("MCA Training
// of Transformer Networks"): the candidate stream over all parameter tensors,
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
#include "tf_kernels.hpp"

namespace mca {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGemmThreads = 256;  // 4 waves, a 64 x 64 output tile
constexpr int kLnThreads = 256;    // a wave per row
constexpr int kLossThreads = 256;
constexpr int kCopyThreads = 256;

__device__ __forceinline__ int64_t fc_width(const TfDev* tf) {
  return tf->M > tf->V ? tf->M : tf->V;
}
__device__ __forceinline__ float* slot_x(const TfDev* tf, int k, int b) {
  return tf->sx + ((int64_t)k * (tf->NB + 1) + b) * tf->N * tf->D;
}
// x_{stage-1}, the residual stream entering stage `stage` (1..NB+1)
__device__ __forceinline__ const float* stage_input(const TfDev* tf, int k, int stage) {
  return (tf->start[k] == stage) ? tf->x[stage - 1] : slot_x(tf, k, stage - 1);
}
__device__ __forceinline__ float gelu(float y) {
  return 0.5f * y * (1.0f + erff(y * 0.70710678118654752f));
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
  c.reserved = 0;
  cands[k] = c;
  Aux a;
  a.w_old = tf->param[layer][off];
  a.w_new = a.w_old + c.d;
  a.de = a.w_new - a.w_old;
  a.valid = !(tf->bound > 0.f && fabsf(a.w_new) >= tf->bound);
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
  aux[k] = a;
}

// Block k: the candidate's tensor table, its first stage, and the patched
// private copy of its tensor.  identity: slot 0 with the committed tensors.
__global__ __launch_bounds__(kCopyThreads) void k_tf_prep(const TfDev* tf, const mca_cand* cands,
                                                          const Aux* aux, int identity) {
  const int k = blockIdx.x;
  const int nt = tf->n_tensors;
  float** tab = tf->table + (int64_t)k * nt;
  for (int t = threadIdx.x; t < nt; t += blockDim.x) tab[t] = tf->param[t];
  if (identity) {
    if (threadIdx.x == 0) tf->start[k] = 0;
    return;
  }
  const mca_cand c = cands[k];
  const Aux a = aux[k];
  if (!a.valid) {
    if (threadIdx.x == 0) tf->start[k] = tf->NB + 2;
    return;
  }
  const int l = c.layer;
  const int64_t n = (int64_t)tf->rows[l] * tf->cols[l];
  float* cp = tf->scopy + (int64_t)k * tf->copy_stride;
  const float* src = tf->param[l];
  for (int64_t e = threadIdx.x; e < n; e += blockDim.x) cp[e] = src[e];
  __syncthreads();
  if (threadIdx.x == 0) {
    cp[(int64_t)c.j * tf->cols[l] + c.i] = a.w_new;
    tab[l] = cp;
    tf->start[k] = tf_stage(l, tf->NB);
  }
}

// x_0 = tok_emb[token] + pos_emb[position] for the candidates of stage 0
__global__ __launch_bounds__(kCopyThreads) void k_tf_embed(const TfDev* tf) {
  const int k = blockIdx.y;
  if (tf->start[k] != 0) return;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int D = tf->D;
  if (e >= tf->N * D) return;
  const int64_t n = e / D;
  const int c = (int)(e - n * D);
  float* const* tab = tf->table + (int64_t)k * tf->n_tensors;
  const int pos = (int)(n % tf->T);
  slot_x(tf, k, 0)[e] = tab[0][(int64_t)tf->tok[n] * D + c] + tab[1][(int64_t)pos * D + c];
}

// LayerNorm (biased variance, eps inside the root, affine), a wave per row.
// which: 0 LN1 of the stage's block (input x_{stage-1}), 1 LN2 (input: after
// attention), 2 the final LayerNorm (stage NB+1).
__global__ __launch_bounds__(kLnThreads) void k_tf_ln(const TfDev* tf, int stage, int which) {
  const int k = blockIdx.y;
  if (tf->start[k] > stage) return;
  const int D = tf->D;
  const int64_t N = tf->N, ND = N * D;
  const int64_t n = (int64_t)blockIdx.x * (kLnThreads / 64) + (threadIdx.x >> 6);
  if (n >= N) return;
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
    in = tf->sh + k * ND;
    g = tab[tb + kLn2G];
    bb = tab[tb + kLn2B];
  } else {
    in = stage_input(tf, k, stage);
    g = tab[tf->n_tensors - 4];
    bb = tab[tf->n_tensors - 3];
  }
  in += n * D;
  constexpr int kMaxPer = 4;  // D <= 256
  float v[kMaxPer];
  float s = 0.f;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    v[u] = (c < D) ? in[c] : 0.f;
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
  const float rstd = 1.0f / sqrtf(q / (float)D + tf->eps);
  float* out = tf->sln + k * ND + n * D;
#pragma unroll
  for (int u = 0; u < kMaxPer; ++u) {
    const int c = lane + 64 * u;
    if (c < D) out[c] = (v[u] - mean) * rstd * g[c] + bb[c];
  }
}

// Y = X W^T + b with an epilogue, for the candidates active in `stage`.
// A 64 x 64 output tile per block: wave w takes rows 16w.., as four 16 x 16
// MFMA tiles.  The reduction dimension runs in blocks of 16; lane group q
// holds k = 16 kb + 4 q + t (t = 0..3), used by four MFMAs in turn, so each
// lane loads its operands as float4.  Requires Kd % 16 == 0.
__global__ __launch_bounds__(kGemmThreads) void k_tf_gemm(const TfDev* tf, int stage, int role) {
  const int k = blockIdx.z;
  if (tf->start[k] > stage) return;
  const int D = tf->D, M = tf->M, V = tf->V;
  const int64_t N = tf->N, ND = N * D, FC = N * fc_width(tf);
  float* const* tab = tf->table + (int64_t)k * tf->n_tensors;
  const int b = stage - 1;
  const int tb = 2 + kBlockTensors * b;
  const float* X = tf->sln + k * ND;
  int ldX = D, Kd = D, ldY = D, Nout = D, epi = 0;
  const float *W = nullptr, *bias = nullptr, *R = nullptr;
  float* Y = nullptr;
  switch (role) {
    case kGemmQ:
      W = tab[tb + kWq]; bias = tab[tb + kBq]; Y = tf->sqkv + 3 * k * ND; ldY = 3 * D;
      break;
    case kGemmK:
      W = tab[tb + kWk]; bias = tab[tb + kBk]; Y = tf->sqkv + 3 * k * ND + D; ldY = 3 * D;
      break;
    case kGemmV:
      W = tab[tb + kWv]; bias = tab[tb + kBv]; Y = tf->sqkv + 3 * k * ND + 2 * D; ldY = 3 * D;
      break;
    case kGemmO:
      X = tf->satt + k * ND; W = tab[tb + kWo]; bias = tab[tb + kBo]; Y = tf->sh + k * ND;
      R = stage_input(tf, k, stage); epi = 2;
      break;
    case kGemmFc:
      W = tab[tb + kWfc]; bias = tab[tb + kBfc]; Y = tf->sfc + k * FC; ldY = M; Nout = M; epi = 1;
      break;
    case kGemmProj:
      X = tf->sfc + k * FC; ldX = M; Kd = M; W = tab[tb + kWproj]; bias = tab[tb + kBproj];
      Y = slot_x(tf, k, b + 1); R = tf->sh + k * ND; epi = 2;
      break;
    default:  // kGemmOut: logits of the final stage
      W = tab[tf->n_tensors - 2]; bias = tab[tf->n_tensors - 1]; Y = tf->sfc + k * FC; ldY = V;
      Nout = V;
      break;
  }
  const int n0 = blockIdx.y * 64;
  if (n0 >= Nout) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, q = lane >> 4, li = lane & 15;
  const int64_t m0 = (int64_t)blockIdx.x * 64;
  const int64_t arow = m0 + 16 * wave + li;
  const bool aok = arow < N;
  const float* Xr = X + arow * ldX + 4 * q;
  const float* Wr[4];
  bool bok[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    const int n = n0 + 16 * cb + li;
    bok[cb] = n < Nout;
    Wr[cb] = W + (int64_t)(bok[cb] ? n : 0) * Kd + 4 * q;
  }
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  floatx4 acc[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) acc[cb] = zero;
  floatx4 a = aok ? *reinterpret_cast<const floatx4*>(Xr) : zero;
  floatx4 bv[4];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) bv[cb] = bok[cb] ? *reinterpret_cast<const floatx4*>(Wr[cb]) : zero;
  const int nkb = Kd / 16;
  for (int kb = 0; kb < nkb; ++kb) {
    floatx4 an = zero, bn[4] = {zero, zero, zero, zero};
    if (kb + 1 < nkb) {
      an = aok ? *reinterpret_cast<const floatx4*>(Xr + 16 * (kb + 1)) : zero;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        bn[cb] = bok[cb] ? *reinterpret_cast<const floatx4*>(Wr[cb] + 16 * (kb + 1)) : zero;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t], bv[cb][t], acc[cb], 0, 0, 0);
    a = an;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) bv[cb] = bn[cb];
  }
  // D layout: lane (q, li), element v -> row 16 w + 4 q + v, column 16 cb + li
#pragma unroll
  for (int cb = 0; cb < 4; ++cb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t m = m0 + 16 * wave + 4 * q + v;
      const int n = n0 + 16 * cb + li;
      if (m < N && n < Nout) {
        float y = acc[cb][v] + bias[n];
        if (epi == 1) y = gelu(y);
        if (epi == 2) y = R[m * D + n] + y;
        Y[m * ldY + n] = y;
      }
    }
}

// Causal softmax attention, scale 1/sqrt(32): block (sequence, head) of one
// candidate, a thread per query position.
__global__ __launch_bounds__(kTfMaxCtx) void k_tf_attn(const TfDev* tf, int stage) {
  const int k = blockIdx.y;
  if (tf->start[k] > stage) return;
  __shared__ float Ks[kTfMaxCtx][kTfHeadDim + 1];
  __shared__ float Vs[kTfMaxCtx][kTfHeadDim + 1];
  const int T = tf->T, D = tf->D, H = tf->H;
  const int s = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
  const int t = threadIdx.x;
  const int64_t ND = tf->N * D;
  const float* base = tf->sqkv + 3 * k * ND + (int64_t)s * T * 3 * D + h * kTfHeadDim;
  float qv[kTfHeadDim];
  if (t < T) {
    const float* row = base + (int64_t)t * 3 * D;
#pragma unroll
    for (int c = 0; c < kTfHeadDim; ++c) {
      qv[c] = row[c];
      Ks[t][c] = row[D + c];
      Vs[t][c] = row[2 * D + c];
    }
  }
  __syncthreads();
  if (t >= T) return;
  const float scale = 0.17677669529663687f;  // 1/sqrt(32)
  float mx = -__builtin_huge_valf();
  for (int j = 0; j <= t; ++j) {
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < kTfHeadDim; ++c) dot = fmaf(qv[c], Ks[j][c], dot);
    mx = fmaxf(mx, dot * scale);
  }
  float sum = 0.f, o[kTfHeadDim];
#pragma unroll
  for (int c = 0; c < kTfHeadDim; ++c) o[c] = 0.f;
  for (int j = 0; j <= t; ++j) {
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < kTfHeadDim; ++c) dot = fmaf(qv[c], Ks[j][c], dot);
    const float p = fast_exp(dot * scale - mx);
    sum += p;
#pragma unroll
    for (int c = 0; c < kTfHeadDim; ++c) o[c] = fmaf(p, Vs[j][c], o[c]);
  }
  float* out = tf->satt + k * ND + ((int64_t)s * T + t) * D + h * kTfHeadDim;
#pragma unroll
  for (int c = 0; c < kTfHeadDim; ++c) out[c] = o[c] / sum;
}

// Per-position cross-entropy of the candidate's logits, its change against
// the committed loss, and the block's sum of changes (fixed order).
__global__ __launch_bounds__(kLossThreads) void k_tf_ce(const TfDev* tf, float* partial, int nblk) {
  __shared__ float red[kLossThreads];
  const int k = blockIdx.y;
  const bool active = tf->start[k] <= tf->NB + 1;
  const int64_t n = (int64_t)blockIdx.x * kLossThreads + threadIdx.x;
  const int V = tf->V;
  float d = 0.f;
  if (active && n < tf->N) {
    const float* z = tf->sfc + k * tf->N * fc_width(tf) + n * V;
    float m = z[0];
    for (int v = 1; v < V; ++v) m = fmaxf(m, z[v]);
    float s = 0.f;
    for (int v = 0; v < V; ++v) s += fast_exp(z[v] - m);
    const float ln = (fast_log(s) + m) - z[tf->tgt[n]];
    tf->sell[k * tf->N + n] = ln;
    d = ln - tf->ell[n];
  }
  red[threadIdx.x] = d;
  __syncthreads();
  for (int o = kLossThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[(int64_t)k * nblk + blockIdx.x] = red[0];
}

// The winner's (or slot 0's, fill) residual streams from its first stage on
// and its per-position losses become the committed ones; block 0 applies the
// parameter and the state.
__global__ __launch_bounds__(kCopyThreads) void k_tf_commit(const TfDev* tf, const mca_cand* cands,
                                                            const Aux* aux, const double* dL,
                                                            DevState* st, int k_host, int fill) {
  const int k = fill ? 0 : ((k_host >= 0) ? k_host : st->chosen);
  if (k < 0) return;
  const int64_t ND = tf->N * tf->D;
  const int s0 = fill ? 0 : tf->start[k];
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < ND)
    for (int b = s0; b <= tf->NB; ++b) tf->x[b][e] = slot_x(tf, k, b)[e];
  if (e < tf->N) tf->ell[e] = tf->sell[(int64_t)k * tf->N + e];
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

hipError_t tf_launch_eval(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                          const Aux* aux, int K, bool identity, float* partial, int nblk,
                          hipStream_t s) {
  const unsigned KK = identity ? 1u : (unsigned)K;
  const int64_t N = h.N;
  const unsigned mt = (unsigned)((N + 63) / 64);
  hipLaunchKernelGGL(k_tf_prep, dim3(KK), dim3(kCopyThreads), 0, s, tf, cands, aux,
                     identity ? 1 : 0);
  hipLaunchKernelGGL(k_tf_embed, dim3((unsigned)((N * h.D + kCopyThreads - 1) / kCopyThreads), KK),
                     dim3(kCopyThreads), 0, s, tf);
  const dim3 lng((unsigned)((N + kLnThreads / 64 - 1) / (kLnThreads / 64)), KK);
  for (int b = 0; b < h.NB; ++b) {
    const int stage = b + 1;
    hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, stage, 0);
    for (int role : {kGemmQ, kGemmK, kGemmV})
      hipLaunchKernelGGL(k_tf_gemm, dim3(mt, (unsigned)((h.D + 63) / 64), KK), dim3(kGemmThreads),
                         0, s, tf, stage, role);
    hipLaunchKernelGGL(k_tf_attn, dim3((unsigned)(h.S * h.H), KK), dim3(kTfMaxCtx), 0, s, tf,
                       stage);
    hipLaunchKernelGGL(k_tf_gemm, dim3(mt, (unsigned)((h.D + 63) / 64), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmO);
    hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, stage, 1);
    hipLaunchKernelGGL(k_tf_gemm, dim3(mt, (unsigned)((h.M + 63) / 64), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmFc);
    hipLaunchKernelGGL(k_tf_gemm, dim3(mt, (unsigned)((h.D + 63) / 64), KK), dim3(kGemmThreads), 0,
                       s, tf, stage, (int)kGemmProj);
  }
  const int fin = h.NB + 1;
  hipLaunchKernelGGL(k_tf_ln, lng, dim3(kLnThreads), 0, s, tf, fin, 2);
  hipLaunchKernelGGL(k_tf_gemm, dim3(mt, (unsigned)((h.V + 63) / 64), KK), dim3(kGemmThreads), 0,
                     s, tf, fin, (int)kGemmOut);
  hipLaunchKernelGGL(k_tf_ce, dim3((unsigned)nblk, KK), dim3(kLossThreads), 0, s, tf, partial,
                     nblk);
  return hipGetLastError();
}

hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, hipStream_t s) {
  const int64_t ND = h.N * h.D;
  hipLaunchKernelGGL(k_tf_commit, dim3((unsigned)((ND + kCopyThreads - 1) / kCopyThreads)),
                     dim3(kCopyThreads), 0, s, tf, cands, aux, dL, st, k, fill ? 1 : 0);
  if (fill) {
    const int nb = tf_loss_blocks(h.N);
    hipLaunchKernelGGL(k_tf_loss_blocks, dim3(nb), dim3(kLossThreads), 0, s, tf, bsum);
    hipLaunchKernelGGL(k_tf_loss_total, dim3(1), dim3(64), 0, s, tf, bsum, nb, st);
  }
  return hipGetLastError();
}

}  // namespace mca
