// HIP kernels (gfx950) of the decoder Transformer path of MCA (Sec. 2.5):
// the candidate stream over all parameter tensors, each candidate's loss
// change, and the commit.
//
// Every candidate has a slot.  A candidate whose parameter sits in the
// embeddings, a LayerNorm before attention or the MLP, or the attention
// projections is evaluated densely: its own copy of the mutated tensor and a
// forward pass from the first stage that tensor enters.  The others follow
// the structure of the network: an MLP parameter of block b moves block b's
// output stream by a rank-1 term (then the later stages run densely), an
// output-layer or final-LayerNorm parameter moves the logits by a rank-1
// term (then only the cross-entropy runs).  A launch covers all slots (grid
// y or z); a slot whose first stage is later skips the stage and the next
// stage reads the committed state.  The kernels are deterministic and treat
// every position alike, so a position a dense candidate cannot reach (before
// a changed position-embedding row, say) reproduces its committed loss bit
// for bit and adds exactly zero to the loss change.
//
// The committed fields are always those of a dense pass: a winner scored
// incrementally is recomputed densely in slot kr of the next evaluation pass
// (see TfRedo), and the next commit folds that slot in before the new
// winner's own.
//
// The model (pre-LN blocks, learned positions, erf GELU, final LayerNorm,
// untied output layer with bias; linear layers y = x W^T + b) is the reading
// of the paper fixed for the oracle.  The dense products run on the matrix
// cores (v_mfma_f32_16x16x4f32) with each LayerNorm folded into the product
// that reads it; attention, GELU and the loss run in fp32 on the vector units.
#include <algorithm>

#include "tf_kernels.hpp"

namespace mca {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

constexpr int kGemmThreads = 256;  // 4 waves per output tile of 128 rows x 16 CB WC columns
constexpr int kGemmRows = 128;     // rows (positions) per block
constexpr int kChunkK = 16;        // reduction chunk staged in LDS
constexpr int kStatSteps = 4;      // groups of four rows whose LayerNorm statistics a wave takes at once
constexpr int kRowThreads = 256;   // row kernels: a wave per row
constexpr int kDlSteps = 4;        // groups of four rows a wave of the loss-change kernel loads at once
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
__device__ __forceinline__ float* slot_fc(const TfDev* tf, int k) { return tf->sfc + (int64_t)k * tf->N * tf->M; }
__device__ __forceinline__ float* slot_log(const TfDev* tf, int k) { return tf->slog + (int64_t)k * tf->N * tf->V; }
__device__ __forceinline__ float* slot_ell(const TfDev* tf, int k) { return tf->sell + (int64_t)k * tf->N; }

// Grid row idx of a launch over ncand candidates: candidate idx, or the
// pending recomputation's slot for the extra last row.
__device__ __forceinline__ int slot_of(const TfDev* tf, unsigned idx, int ncand) {
  return (int)idx < ncand ? (int)idx : tf->kr;
}
// Whether the pending recomputation runs in this pass, and the committed
// fields as the rest of the pass sees them (TfRedo).
__device__ __forceinline__ bool redo_on(const TfDev* tf) { return tf->run[tf->kr] <= tf->NB + 1; }
__device__ __forceinline__ bool runs_attention(const TfDev* tf, int k, int b) {
  return tf->run[k] <= b + 1 && tf->half[k] != b + 1;
}
__device__ __forceinline__ const float* view_x(const TfDev* tf, int j) {
  const int kr = tf->kr;
  return (redo_on(tf) && j >= tf->xin[kr]) ? slot_x(tf, kr, j) : tf->x[j];
}
__device__ __forceinline__ const float* view_h(const TfDev* tf, int b) {
  return runs_attention(tf, tf->kr, b) ? slot_h(tf, tf->kr, b) : tf->ch[b];
}
__device__ __forceinline__ const float* view_z(const TfDev* tf) {
  return redo_on(tf) ? slot_log(tf, tf->kr) : tf->cz;
}
__device__ __forceinline__ const float* view_ell(const TfDev* tf) {
  return redo_on(tf) ? slot_ell(tf, tf->kr) : tf->ell;
}
// x_{stage-1}, the residual stream entering stage `stage` (1..NB+1): the
// slot's own once it has changed, the committed one before
__device__ __forceinline__ const float* stage_input(const TfDev* tf, int k, int stage) {
  return (tf->xin[k] > stage - 1) ? view_x(tf, stage - 1) : slot_x(tf, k, stage - 1);
}
// the attention output block b's MLP half reads: the slot's own, or the
// committed one (as this pass sees it) for a slot that starts at that MLP
// half
__device__ __forceinline__ const float* mlp_input(const TfDev* tf, int k, int b) {
  return (tf->half[k] == b + 1) ? view_h(tf, b) : slot_h(tf, k, b);
}

// Rows held by 16 lanes (a quarter wave): lane l of the group holds the
// column pairs (32 i + 2 l, 32 i + 2 l + 1), i < np = D / 32, so that a
// float2 load of the group is 128 contiguous bytes; sums over the group by
// a fixed butterfly.
template <int P>
__device__ __forceinline__ void load_pairs(const float* row, int np, int l, floatx2 (&v)[P]) {
  const floatx2 z2 = {0.f, 0.f};
#pragma unroll
  for (int i = 0; i < P; ++i)
    v[i] = (i < np) ? gload(reinterpret_cast<const floatx2*>(row + 32 * i + 2 * l)) : z2;
}
__device__ __forceinline__ float sum16(float s) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) s += __shfl_xor(s, o, 16);
  return s;
}
__device__ __forceinline__ float max16(float s) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) s = fmaxf(s, __shfl_xor(s, o, 16));
  return s;
}
// mean and 1/sqrt(biased variance + eps) of a row (zeros beyond np pairs)
template <int P>
__device__ __forceinline__ void stats16(const floatx2 (&v)[P], int np, int D, float eps,
                                        float& mean, float& rstd) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < P; ++i) s += v[i].x + v[i].y;
  mean = sum16(s) / (float)D;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < P; ++i) {
    if (i < np) {
      const float a = v[i].x - mean, b = v[i].y - mean;
      q += a * a + b * b;
    }
  }
  rstd = 1.0f / sqrtf(sum16(q) / (float)D + eps);
}
// column c of a row held by the group whose first lane is gbase (every lane
// of the group gets it)
template <int P>
__device__ __forceinline__ float col16(const floatx2 (&v)[P], int c, int gbase) {
  const int i = c >> 5;
  float sel = 0.f;
#pragma unroll
  for (int ii = 0; ii < P; ++ii)
    if (ii == i) sel = (c & 1) ? v[ii].y : v[ii].x;
  return __shfl(sel, gbase + ((c & 31) >> 1), 64);
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

// Cross-entropy of one position from its V logits (max-shifted).
__device__ __forceinline__ float cross_entropy(const float* z, int V, int y) {
  float m = z[0];
  for (int v = 1; v < V; ++v) m = fmaxf(m, z[v]);
  float sum = 0.f;
  for (int v = 0; v < V; ++v) sum += fast_exp(z[v] - m);
  return (fast_log(sum) + m) - z[y];
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

// Blocks (x, row): the slot's tensor table, first stage and kind (block 0),
// and a candidate's patched private copy of its tensor, kCopyChunk floats per
// block.  kPrepEval: candidates 0..ncand-1 and, in the extra last row, the
// pending recomputation (every committed tensor, its stages from TfRedo);
// kPrepIdentity: slot 0 with the committed tensors (cache fill), and no
// recomputation.
enum { kPrepEval = 0, kPrepIdentity = 1 };
__global__ __launch_bounds__(kCopyThreads) void k_tf_prep(const TfDev* tf, const mca_cand* cands,
                                                          const Aux* aux, int mode, int ncand) {
  const int k = slot_of(tf, blockIdx.y, ncand);
  const int nt = tf->n_tensors, NB = tf->NB;
  float** tab = tf->table + (int64_t)k * nt;
  if (mode == kPrepIdentity || k == tf->kr) {
    if (blockIdx.x == 0) {
      for (int t = threadIdx.x; t < nt; t += blockDim.x) tab[t] = tf->param[t];
      if (threadIdx.x == 0) {
        tf->kind[k] = kTfDense;
        if (mode == kPrepIdentity) {
          tf->start[k] = tf->run[k] = 0;
          tf->xin[k] = 0;
          tf->half[k] = 0;
          tf->run[tf->kr] = NB + 2;  // nothing else runs in a cache fill
        } else {
          tf->start[k] = tf->run[k] = tf->redo[kRedoStart];
          tf->half[k] = tf->redo[kRedoHalf];
          tf->xin[k] = tf->redo[kRedoXin];
        }
      }
    }
    return;
  }
  const mca_cand c = cands[k];
  const Aux a = aux[k];
  const int l = c.layer;
  int kind = kTfDense;
  if (l >= nt - 2) kind = kTfOutCol;
  else if (l >= nt - 4) kind = kTfLnfCol;
  else if (l >= 2) {
    const int role = (l - 2) % kBlockTensors;
    if (role == kWproj || role == kBproj) kind = kTfProjCol;
    if (role == kWfc || role == kBfc) kind = kTfFcCol;
  }
  const bool dense = kind == kTfDense;
  float* cp = tf->scopy + (int64_t)k * tf->copy_stride;
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < nt; t += blockDim.x)
      tab[t] = (t == l && a.valid && dense) ? cp : tf->param[t];
    if (threadIdx.x == 0) {
      const int blk = (l - 2) / kBlockTensors;
      int start = NB + 2, xin = NB + 2;  // nothing recomputed: rejected, or the last stage's own
      int half = 0;
      if (a.valid && dense) start = xin = tf_stage(l, NB);
      if (a.valid && dense && l >= 2 && l < nt - 4) {
        // an LN2 gain or bias leaves its block's attention half as committed
        const int role = (l - 2) % kBlockTensors;
        if (role == kLn2G || role == kLn2B) half = blk + 1;
      }
      if (a.valid && (kind == kTfProjCol || kind == kTfFcCol)) {
        start = blk + 2;  // the stages after the block, from its patched output stream
        xin = blk + 1;
      }
      tf->start[k] = tf->run[k] = start;
      tf->xin[k] = xin;
      tf->half[k] = half;
      tf->kind[k] = a.valid ? kind : kTfDense;
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

// x_0 = tok_emb[token] + pos_emb[position] for the slots of stage 0
__global__ __launch_bounds__(kCopyThreads) void k_tf_embed(const TfDev* tf, int ncand) {
  const int k = slot_of(tf, blockIdx.y, ncand);
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

// Mean and 1/sqrt(biased variance + eps) of every row of a LayerNorm's
// input, for the slots that run it: which 0 LN1 (the input of stage
// `stage`), 1 LN2 (the attention output block stage-1's MLP reads), 2 the
// final LayerNorm (the input of stage NB+1).  Rows in the 16-lane layout; a
// wave takes four rows at a time and kStatSteps such groups with every load
// in flight.  Every product that folds a LayerNorm in takes its statistics
// from here.  P = D / 32 rounded up to 4 or 8.
//
// An MLP candidate of block b (kTfProjCol, kTfFcCol) enters stage b + 2 here
// with its patched x_{b+1}: the committed stream plus its change, written
// to its slot before the statistics are taken.  The one pre-activation it
// needs (unit c.j of an up-projection candidate, unit c.i of a
// down-projection weight) is recomputed from the committed attention
// output: LN2 of the row, its dot product with the unit's weight row, plus
// the unit's bias.  An up-projection candidate moves that pre-activation by
// de times LN2 column c.i (de for the bias), and the change of its GELU
// enters every column through the down-projection's column c.j; a
// down-projection candidate moves column c.j by de times the GELU of unit
// c.i (de for the bias).
template <int P>
__global__ __launch_bounds__(kRowThreads) void k_tf_stats(const TfDev* tf, const mca_cand* cands,
                                                          const Aux* aux, int stage, int which,
                                                          int ncand) {
  const int k = slot_of(tf, blockIdx.y, ncand);
  if (which == 0 ? !runs_attention(tf, k, stage - 1) : tf->run[k] > stage) return;
  const int D = tf->D, np = D / 32, lane = threadIdx.x & 63, g = lane >> 4, l = lane & 15;
  const int64_t N = tf->N;
  float2* out = tf->sst + (int64_t)k * N;
  constexpr int kRowsPerWave = 4 * kStatSteps;
  const int64_t r0 = ((int64_t)blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6)) * kRowsPerWave;
  const int kind = tf->kind[k];
  const bool patch = which != 1 && (kind == kTfProjCol || kind == kTfFcCol) && tf->run[k] == stage;
  if (!patch) {
    const float* X = (which == 1) ? mlp_input(tf, k, stage - 1) : stage_input(tf, k, stage);
    floatx2 v[kStatSteps][P];
#pragma unroll
    for (int st = 0; st < kStatSteps; ++st) {
      const int64_t m = r0 + 4 * st + g;
      load_pairs(X + (m < N ? m : N - 1) * D, np, l, v[st]);
    }
#pragma unroll
    for (int st = 0; st < kStatSteps; ++st) {
      float mean, rstd;
      stats16(v[st], np, D, tf->eps, mean, rstd);
      const int64_t m = r0 + 4 * st + g;
      if (l == 0 && m < N) out[m] = make_float2(mean, rstd);
    }
    return;
  }
  const mca_cand c = cands[k];
  const int b = stage - 2, M = tf->M;
  const int role = (c.layer - 2) % kBlockTensors, tb = 2 + kBlockTensors * b;
  const float de = aux[k].de;
  const bool fc = kind == kTfFcCol, need_u = fc || role == kWproj;
  const int unit = fc ? c.j : c.i;
  const float* g2 = tf->param[tb + kLn2G];
  const float* b2 = tf->param[tb + kLn2B];
  const float* wfc = tf->param[tb + kWfc] + (int64_t)unit * D;
  const float* wproj = tf->param[tb + kWproj];
  const floatx2 z2 = {0.f, 0.f};
  floatx2 gv[P], bv[P], wu[P], wp[P];
#pragma unroll
  for (int i = 0; i < P; ++i) {
    const int cc = 32 * i + 2 * l;
    const bool ok = i < np;
    gv[i] = ok ? gload(reinterpret_cast<const floatx2*>(g2 + cc)) : z2;
    bv[i] = ok ? gload(reinterpret_cast<const floatx2*>(b2 + cc)) : z2;
    wu[i] = (ok && need_u) ? gload(reinterpret_cast<const floatx2*>(wfc + cc)) : z2;
    wp[i] = z2;
    if (ok && fc) {
      wp[i].x = wproj[(int64_t)cc * M + c.j];
      wp[i].y = wproj[(int64_t)(cc + 1) * M + c.j];
    }
  }
  const float bu = need_u ? tf->param[tb + kBfc][unit] : 0.f;
  const float* hc = view_h(tf, b);
  const float* xc = view_x(tf, b + 1);
  float* xo = slot_x(tf, k, b + 1);
  floatx2 hv[kStatSteps][P], xv[kStatSteps][P];
#pragma unroll
  for (int st = 0; st < kStatSteps; ++st) {
    const int64_t m0 = r0 + 4 * st + g, m = m0 < N ? m0 : N - 1;
    if (need_u) load_pairs(hc + m * D, np, l, hv[st]);
    load_pairs(xc + m * D, np, l, xv[st]);
  }
#pragma unroll
  for (int st = 0; st < kStatSteps; ++st) {
    float dg = de;  // a down-projection bias
    if (need_u) {
      float mean, rstd;
      stats16(hv[st], np, D, tf->eps, mean, rstd);
      floatx2 lnv[P];
      float dot = 0.f;
#pragma unroll
      for (int i = 0; i < P; ++i) {
        lnv[i] = z2;
        if (i < np) {
          lnv[i].x = (hv[st][i].x - mean) * rstd * gv[i].x + bv[i].x;
          lnv[i].y = (hv[st][i].y - mean) * rstd * gv[i].y + bv[i].y;
          dot += lnv[i].x * wu[i].x + lnv[i].y * wu[i].y;
        }
      }
      const float uu = sum16(dot) + bu;
      if (fc) {
        const float du = (role == kWfc) ? de * col16(lnv, c.i, lane & ~15) : de;
        dg = gelu(uu + du) - gelu(uu);
      } else {
        dg = de * gelu(uu);
      }
    }
#pragma unroll
    for (int i = 0; i < P; ++i) {
      const int cc = 32 * i + 2 * l;
      if (fc) {
        xv[st][i].x += dg * wp[i].x;
        xv[st][i].y += dg * wp[i].y;
      } else {
        if (cc == c.j) xv[st][i].x += dg;
        if (cc + 1 == c.j) xv[st][i].y += dg;
      }
    }
    const int64_t m = r0 + 4 * st + g;
    if (m < N) {
#pragma unroll
      for (int i = 0; i < P; ++i)
        if (i < np) *reinterpret_cast<floatx2*>(xo + m * D + 32 * i + 2 * l) = xv[st][i];
    }
    float mean, rstd;
    stats16(xv[st], np, D, tf->eps, mean, rstd);
    if (l == 0 && m < N) out[m] = make_float2(mean, rstd);
  }
}

// Y = LN(X) W^T + b (LN: the LayerNorm of the input rows, for the products
// that read one) with an epilogue, for the slots active in `stage`.
// A 128 x 16 CB WC output tile per block: the 4 waves form a (4 / WC) x WC
// grid and wave (wr, wc) takes its 16 SB x 16 CB part (SB = 2 WC) as SB by
// CB 16 x 16 MFMA tiles, so each operand fragment read from LDS feeds
// several MFMAs.  The reduction dimension runs in
// chunks of 16 staged in LDS (two buffers; the loads run two chunks ahead of
// the products).  Inside a chunk, k
// runs in blocks of 16; lane group q holds k = 16 kb + 4 q + t (t = 0..3),
// used by four MFMAs in turn, so each lane reads its operands as float4.
// Rows and columns beyond the matrix are clamped on load and dropped on
// store.  Requires Kd % 32 == 0.  The Q, K and V projections are one
// product with 3 D output columns: column n takes its weight row and bias
// from tensor n / D of the three.
// LayerNorm (Q, K, V: LN1 of the stage input; MLP up: LN2 of the attention
// output; output layer: the final LayerNorm): with the mean and
// 1/sqrt(variance + eps) of each input row from k_tf_stats and the gain and
// bias staged in LDS, each staged operand element becomes
// (x - mean) rstd g + b on its way into LDS.
// EPI: 0 bias only (Q, K, V), 1 GELU (MLP up), 2 residual (attention
// output, MLP down), 3 logits and each position's cross-entropy (output layer; one column
// tile, with the logit tile in LDS).
template <int EPI, int CB, int WC>
__global__ __launch_bounds__(kGemmThreads, (EPI == 2 && CB == 4) || (EPI == 3 && CB == 8) ? 2 : 3) void k_tf_gemm(
    const TfDev* tf, int stage, int role, int ncand) {
  const int k = slot_of(tf, blockIdx.z, ncand);
  const bool attn_half = role == kGemmQKV || role == kGemmO;
  if (tf->run[k] > stage || (attn_half && tf->half[k] == stage)) return;
  const int D = tf->D, M = tf->M, V = tf->V, nt = tf->n_tensors;
  const int64_t N = tf->N, ND = N * D;
  float* const* tab = tf->table + (int64_t)k * nt;
  const int b = stage - 1;
  const int tb = 2 + kBlockTensors * b;
  const float* X = nullptr;
  int ldX = D, Kd = D, ldY = D, Nout = D;
  bool qkv = false;
  const float *W = nullptr, *bias = nullptr, *R = nullptr;
  const float *lg = nullptr, *lb = nullptr;  // LayerNorm gain and bias of the input rows
  float* Y = nullptr;
  switch (role) {
    case kGemmQKV:
      X = stage_input(tf, k, stage); lg = tab[tb + kLn1G]; lb = tab[tb + kLn1B];
      Y = tf->sqkv + 3 * k * ND; ldY = 3 * D; Nout = 3 * D; qkv = true;
      break;
    case kGemmO:
      X = tf->satt + k * ND; W = tab[tb + kWo]; bias = tab[tb + kBo]; Y = slot_h(tf, k, b);
      R = stage_input(tf, k, stage);
      break;
    case kGemmFc:
      X = mlp_input(tf, k, b); lg = tab[tb + kLn2G]; lb = tab[tb + kLn2B];
      W = tab[tb + kWfc]; bias = tab[tb + kBfc]; Y = slot_fc(tf, k); ldY = M; Nout = M;
      break;
    case kGemmProj:
      X = slot_fc(tf, k); ldX = M; Kd = M; W = tab[tb + kWproj]; bias = tab[tb + kBproj];
      Y = slot_x(tf, k, b + 1); R = mlp_input(tf, k, b);
      break;
    default:  // kGemmOut: logits of the final stage
      X = stage_input(tf, k, stage); lg = tab[nt - 4]; lb = tab[nt - 3];
      W = tab[nt - 2]; bias = tab[nt - 1]; Y = slot_log(tf, k); ldY = V; Nout = V;
      break;
  }
  constexpr int kWR = 4 / WC;          // waves along the rows
  constexpr int SB = 8 / kWR;          // 16-row MFMA tiles per wave
  constexpr int kTileN = 16 * CB * WC; // output columns of the block, 16 CB per wave
  const int n0 = blockIdx.y * kTileN;
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
  constexpr int kStage = 2 * kGemmRows * (kChunkK + 4);  // floats of the A operand's double buffer
  constexpr int kStageB = 2 * kTileN * (kChunkK + 4);
  constexpr int kZ = kGemmRows * (kTileN + 1);           // the output layer's logit tile
  constexpr int kSmem = (EPI == 3 && kZ > kStage + kStageB) ? kZ : kStage + kStageB;
  __shared__ __attribute__((aligned(16))) float smem[kSmem];
  auto As = reinterpret_cast<float (*)[kGemmRows][kChunkK + 4]>(smem);
  auto Bs = reinterpret_cast<float (*)[kTileN][kChunkK + 4]>(smem + kStage);
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, q = lane >> 4, li = lane & 15;
  const int wr = wave / WC, wc = wave % WC;
  const int64_t m0 = (int64_t)blockIdx.x * kGemmRows;
  constexpr bool ln = EPI != 2;  // the products that read a LayerNorm
  const float2* stats = tf->sst + (int64_t)k * N;  // the input rows' LayerNorm statistics
  __shared__ __attribute__((aligned(16))) float s_g[ln ? 256 : 4], s_b[ln ? 256 : 4];
  if constexpr (ln) {
    for (int c = threadIdx.x; c < Kd; c += kGemmThreads) {
      s_g[c] = lg[c];
      s_b[c] = lb[c];
    }
  }
  // staging: thread tid loads float4 number tid + 256 u of the A chunk
  // (128 rows x 4 float4) and of the B chunk (128 rows x 4 float4); its A
  // elements sit in one float4 column group of every chunk
  constexpr int kA4 = kGemmRows * kChunkK / 4 / kGemmThreads;  // 2
  // (the B chunk has kTileN x 4 float4: threads beyond it load a clamped row
  // and store nothing)
  constexpr int kB4 = (kTileN * kChunkK / 4 + kGemmThreads - 1) / kGemmThreads;
  const int acol = 4 * (tid % (kChunkK / 4));
  const float* ga[kA4];
  const float* gb[kB4];
  float amu[kA4], ars[kA4];
#pragma unroll
  for (int u = 0; u < kA4; ++u) {
    const int e = tid + kGemmThreads * u;
    const int r = e / (kChunkK / 4);
    const int64_t m = m0 + r;
    ga[u] = X + (m < N ? m : N - 1) * ldX + acol;
    const float2 st2 = ln ? stats[m < N ? m : N - 1] : make_float2(0.f, 1.f);
    amu[u] = st2.x;
    ars[u] = st2.y;
  }
#pragma unroll
  for (int u = 0; u < kB4; ++u) {
    const int e = tid + kGemmThreads * u;
    const int n = n0 + e / (kChunkK / 4);
    gb[u] = wrow(n < Nout ? n : Nout - 1) + 4 * (e % (kChunkK / 4));
  }
  const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
  // a chunk's operands on their way from memory into LDS
  struct Staged {
    floatx4 a[kA4];
    floatx4 b[kB4];
  };
  auto fetch = [&](int c, Staged& S) {
#pragma unroll
    for (int u = 0; u < kA4; ++u) S.a[u] = gload(reinterpret_cast<const floatx4*>(ga[u] + kChunkK * c));
#pragma unroll
    for (int u = 0; u < kB4; ++u) S.b[u] = gload(reinterpret_cast<const floatx4*>(gb[u] + kChunkK * c));
  };
  auto store = [&](int c, const Staged& S) {
    const int buf = c & 1;
#pragma unroll
    for (int u = 0; u < kA4; ++u) {
      const int e = tid + kGemmThreads * u;
      floatx4 a = S.a[u];
      if constexpr (ln) {
        const floatx4 g4 = *reinterpret_cast<const floatx4*>(&s_g[kChunkK * c + acol]);
        const floatx4 b4 = *reinterpret_cast<const floatx4*>(&s_b[kChunkK * c + acol]);
#pragma unroll
        for (int t = 0; t < 4; ++t) a[t] = fmaf((a[t] - amu[u]) * ars[u], g4[t], b4[t]);
      }
      *reinterpret_cast<floatx4*>(&As[buf][e / (kChunkK / 4)][acol]) = a;
    }
#pragma unroll
    for (int u = 0; u < kB4; ++u) {
      const int e = tid + kGemmThreads * u;
      if ((kTileN * kChunkK / 4) % kGemmThreads == 0 || e < kTileN * kChunkK / 4)
        *reinterpret_cast<floatx4*>(&Bs[buf][e / (kChunkK / 4)][4 * (e % (kChunkK / 4))]) = S.b[u];
    }
  };
  floatx4 acc[SB][CB];
#pragma unroll
  for (int sb = 0; sb < SB; ++sb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) acc[sb][cb] = zero;
  auto compute = [&](int buf) {
#pragma unroll
    for (int kb = 0; kb < kChunkK / 16; ++kb) {
      floatx4 a[SB], bv[CB];
#pragma unroll
      for (int sb = 0; sb < SB; ++sb)
        a[sb] = *reinterpret_cast<const floatx4*>(&As[buf][16 * SB * wr + 16 * sb + li][16 * kb + 4 * q]);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        bv[cb] = *reinterpret_cast<const floatx4*>(&Bs[buf][16 * CB * wc + 16 * cb + li][16 * kb + 4 * q]);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int sb = 0; sb < SB; ++sb)
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            acc[sb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[sb][t], bv[cb][t], acc[sb][cb], 0, 0, 0);
    }
  };
  // D layout: lane (q, li), element v -> row 16 sb + 4 q + v, column 16 cb + li.
  // The residual a lane adds is loaded before the last chunk's products, so
  // its latency hides behind them.
  float res[SB][CB][4];
  (void)res;
  auto load_residual = [&]() {
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int64_t m = m0 + 16 * SB * wr + 16 * sb + 4 * q + v;
          const int n = n0 + 16 * CB * wc + 16 * cb + li;
          res[sb][cb][v] = (m < N && n < Nout) ? R[m * D + n] : 0.f;
        }
  };
  // Chunk c + 2's loads are issued while chunk c is multiplied and chunk
  // c + 1 (loaded one chunk earlier) goes into the other LDS buffer: two
  // register sets, the loop unrolled by two so that each is fixed.  The
  // number of chunks is even (Kd % 32 == 0), so every load in the loop is
  // unconditional and each store waits only for its own chunk's loads.
  const int nc = Kd / kChunkK;
  Staged S0, S1;
  fetch(0, S0);
  fetch(1, S1);
  if constexpr (ln) __syncthreads();  // the LayerNorm gain and bias are in LDS
  store(0, S0);
  __syncthreads();
  for (int c = 0; c + 2 < nc; c += 2) {
    fetch(c + 2, S0);
    compute(0);
    store(c + 1, S1);
    __syncthreads();
    fetch(c + 3, S1);
    compute(1);
    store(c + 2, S0);
    __syncthreads();
  }
  compute(0);
  store(nc - 1, S1);
  __syncthreads();
  if constexpr (EPI == 2) load_residual();
  compute(1);
  __syncthreads();
  float bvv[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    const int n = n0 + 16 * CB * wc + 16 * cb + li;
    bvv[cb] = (n < Nout) ? bias_of(n) : 0.f;
  }
  if constexpr (EPI == 3) {
    // the logits into LDS (the operand buffers are free) and to the slot,
    // then a thread per position
    const int ldz = V + 1;
    float* Z = smem;
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = 16 * SB * wr + 16 * sb + 4 * q + v;
          const int n = 16 * CB * wc + 16 * cb + li;
          if (n < Nout) {
            const float y = acc[sb][cb][v] + bvv[cb];
            Z[r * ldz + n] = y;
            if (m0 + r < N) Y[(m0 + r) * ldY + n] = y;
          }
        }
    __syncthreads();
    if (tid < kGemmRows && m0 + tid < N)
      slot_ell(tf, k)[m0 + tid] = cross_entropy(Z + tid * ldz, V, tf->tgt[m0 + tid]);
    return;
  }
#pragma unroll
  for (int sb = 0; sb < SB; ++sb)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t m = m0 + 16 * SB * wr + 16 * sb + 4 * q + v;
        const int n = n0 + 16 * CB * wc + 16 * cb + li;
        if (m < N && n < Nout) {
          float y = acc[sb][cb][v] + bvv[cb];
          if constexpr (EPI == 1) y = gelu(y);
          if constexpr (EPI == 2) y = res[sb][cb][v] + y;
          Y[m * ldY + n] = y;
        }
      }
}

// Causal softmax attention, scale 1/sqrt(32), on the matrix cores: a block
// of 4 waves per (sequence, head) of one slot.  K and V of the sequence and
// head sit in LDS (rows padded); each wave reads its own queries from
// memory.  Query block rb (16 queries) takes key
// blocks 0..rb and works on transposed tiles: the scores S^T = K Q^T (keys
// as rows, queries as columns; two k-blocks of 16 over the head dimension,
// operands read as float4), so that lane (q, li) holds keys 4 q + v of each
// key block for query li.  The softmax of a query is then a reduction over
// the lane's registers and the four lanes li, li + 16, li + 32, li + 48 (a
// fixed butterfly), and the probabilities are already in the B-operand
// layout of O^T = V^T P^T: the product's k index runs over keys
// 16 cb + 4 q + t, the same order for both operands, with V read from LDS.
// Wave w takes query blocks w and 7-w (T = 128: every wave walks 9 tiles);
// keys after the query are masked.
__global__ __launch_bounds__(256) void k_tf_attn(const TfDev* tf, int stage, int ncand) {
  const int k = slot_of(tf, blockIdx.y, ncand);
  if (!runs_attention(tf, k, stage - 1)) return;
  constexpr int kS = kTfHeadDim + 4;  // padded row
  __shared__ __attribute__((aligned(16))) float Ks[kTfMaxCtx][kS];
  __shared__ __attribute__((aligned(16))) float Vs[kTfMaxCtx][kS];
  const int T = tf->T, D = tf->D, H = tf->H;
  const int s = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
  const int64_t ND = tf->N * D;
  const float* base = tf->sqkv + 3 * k * ND + (int64_t)s * T * 3 * D + h * kTfHeadDim;
  {
    // 128 rows x 8 float4 per tensor: four float4 of each per thread, every
    // load issued before the LDS stores
    constexpr int kPer = kTfMaxCtx * kTfHeadDim / 4 / 256;
    floatx4 rk[kPer], rv[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int t = e / (kTfHeadDim / 4), c4 = e - t * (kTfHeadDim / 4);
      const bool ok = t < T;
      const float* row = base + (int64_t)(ok ? t : 0) * 3 * D + 4 * c4;
      const floatx4 z = {0.f, 0.f, 0.f, 0.f};
      rk[u] = ok ? gload(reinterpret_cast<const floatx4*>(row + D)) : z;
      rv[u] = ok ? gload(reinterpret_cast<const floatx4*>(row + 2 * D)) : z;
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int e = threadIdx.x + 256 * u;
      const int t = e / (kTfHeadDim / 4), c4 = e - t * (kTfHeadDim / 4);
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
    const int query = 16 * rb + li;
    // scores S^T of key blocks 0..rb against query block rb
    floatx4 sc[kTfMaxCtx / 16];
    floatx4 qb[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      qb[kb] = (query < T) ? gload(reinterpret_cast<const floatx4*>(base + (int64_t)query * 3 * D + 16 * kb + 4 * q))
                           : zero;
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb) {
      sc[cb] = zero;
      if (cb <= rb) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const floatx4 kk = *reinterpret_cast<const floatx4*>(&Ks[16 * cb + li][16 * kb + 4 * q]);
#pragma unroll
          for (int t = 0; t < 4; ++t)
            sc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(kk[t], qb[kb][t], sc[cb], 0, 0, 0);
        }
      }
    }
    // lane (q, li): keys 16 cb + 4 q + v of query li
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (cb <= rb && 16 * cb + 4 * q + v <= query) m = fmaxf(m, sc[cb][v] * scale);
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float p = (cb <= rb && 16 * cb + 4 * q + v <= query) ? fast_exp(sc[cb][v] * scale - m) : 0.f;
        sc[cb][v] = p;
        sum += p;
      }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    // O^T = V^T P^T, dims 16 db + row, queries as columns
    floatx4 oc[2] = {zero, zero};
#pragma unroll
    for (int cb = 0; cb < kTfMaxCtx / 16; ++cb) {
      if (cb > rb) break;  // uniform over the wave
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int key = 16 * cb + 4 * q + t;
#pragma unroll
        for (int db = 0; db < 2; ++db)
          oc[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(Vs[key][16 * db + li], sc[cb][t], oc[db], 0, 0, 0);
      }
    }
    // lane (q, li) holds O[query li][dims 16 db + 4 q + v]
    if (query < T) {
      const float inv = 1.0f / sum;
#pragma unroll
      for (int db = 0; db < 2; ++db) {
        floatx4 o;
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = oc[db][v] * inv;
        *reinterpret_cast<floatx4*>(outb + (int64_t)query * D + 16 * db + 4 * q) = o;
      }
    }
  }
}

// Per-position loss changes of candidate k against the committed losses,
// and the block's sum over its 256 positions (in order).  A dense or MLP
// candidate's losses come from its own final stage.  An output-layer or
// final-LayerNorm candidate's come from the committed logits plus its change:
// an output weight (j, i) moves logit j by de times column i of the final
// LayerNorm's output (de for the bias); a final-LayerNorm gain or bias of
// column j moves that column by de times its normalized value (or de), which
// reaches every logit through column j of the output weights.  The
// normalized value is recomputed from the committed x_NB.  Rows of such a
// candidate in the 16-lane layout (logit v on lane v mod 16), kDlSteps
// groups of four rows per wave with every load in flight.
template <int P>
__global__ __launch_bounds__(kLossThreads) void k_tf_dl(const TfDev* tf, const mca_cand* cands,
                                                        const Aux* aux, float* partial, int nblk) {
  __shared__ float dl[kLossThreads];
  const int k = blockIdx.y;
  const int kind = tf->kind[k];
  const bool col = kind == kTfOutCol || kind == kTfLnfCol;
  const bool active = tf->run[k] <= tf->NB + 1;
  const int V = tf->V, D = tf->D, nt = tf->n_tensors;
  const int64_t N = tf->N;
  const int64_t n0 = (int64_t)blockIdx.x * kLossThreads;
  const int nrows = (int)((N - n0 < kLossThreads) ? N - n0 : kLossThreads);
  const float* ell = view_ell(tf);
  const int r = threadIdx.x;
  dl[r] = (!col && active && r < nrows) ? slot_ell(tf, k)[n0 + r] - ell[n0 + r] : 0.f;
  if (col) {
    __syncthreads();
    const mca_cand c = cands[k];
    const float de = aux[k].de;
    const bool out_w = c.layer == nt - 2, lnf_g = c.layer == nt - 4, need_nh = out_w || lnf_g;
    const int cc = out_w ? c.i : c.j;
    const float* zc = view_z(tf);
    const float* xs = view_x(tf, tf->NB);
    const float* wo = tf->param[nt - 2];
    const int lane = threadIdx.x & 63, g = lane >> 4, l = lane & 15, wave = threadIdx.x >> 6;
    const int np = D / 32;
    constexpr int kVPer = kTfMaxVocab / 16;
    float wov[kVPer];
#pragma unroll
    for (int j = 0; j < kVPer; ++j) {
      const int v = l + 16 * j;
      wov[j] = (kind == kTfLnfCol && v < V) ? wo[(int64_t)v * D + c.j] : 0.f;
    }
    const float gi = out_w ? tf->param[nt - 4][c.i] : 0.f;
    const float bi = out_w ? tf->param[nt - 3][c.i] : 0.f;
    constexpr int kBatch = 4 * (kLossThreads / 64) * kDlSteps;  // rows per batch of the block
    for (int base = 0; base < nrows; base += kBatch) {
      floatx2 xv[kDlSteps][P];
      float z[kDlSteps][kVPer];
#pragma unroll
      for (int st = 0; st < kDlSteps; ++st) {
        const int rr = base + (wave * kDlSteps + st) * 4 + g;
        const int64_t n = n0 + (rr < nrows ? rr : 0);
        if (need_nh) load_pairs(xs + n * D, np, l, xv[st]);
#pragma unroll
        for (int j = 0; j < kVPer; ++j) {
          const int v = l + 16 * j;
          z[st][j] = (v < V) ? zc[n * V + v] : 0.f;
        }
      }
#pragma unroll
      for (int st = 0; st < kDlSteps; ++st) {
        const int rr = base + (wave * kDlSteps + st) * 4 + g;
        const int64_t n = n0 + (rr < nrows ? rr : 0);
        float nhv = 0.f;
        if (need_nh) {
          float mean, rstd;
          stats16(xv[st], np, D, tf->eps, mean, rstd);
          nhv = (col16(xv[st], cc, lane & ~15) - mean) * rstd;
        }
        const float dz = out_w ? de * fmaf(nhv, gi, bi) : de;
        const float dcol = lnf_g ? de * nhv : de;
        float mx = -__builtin_huge_valf();
#pragma unroll
        for (int j = 0; j < kVPer; ++j) {
          const int v = l + 16 * j;
          if (kind == kTfOutCol) {
            if (v == c.j) z[st][j] += dz;
          } else {
            z[st][j] += dcol * wov[j];
          }
          if (v < V) mx = fmaxf(mx, z[st][j]);
        }
        mx = max16(mx);
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < kVPer; ++j)
          if (l + 16 * j < V) sum += fast_exp(z[st][j] - mx);
        sum = sum16(sum);
        const int yt = tf->tgt[n];
        float sel = 0.f;
#pragma unroll
        for (int j = 0; j < kVPer; ++j)
          if (j == (yt >> 4)) sel = z[st][j];
        const float zt = __shfl(sel, (lane & ~15) + (yt & 15), 64);
        if (l == 0 && rr < nrows) dl[rr] = ((fast_log(sum) + mx) - zt) - ell[n];
      }
    }
  }
  __syncthreads();
  for (int o = kLossThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) dl[threadIdx.x] += dl[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[(int64_t)k * nblk + blockIdx.x] = dl[0];
}

// The commit: first the pending recomputation's fields (slot kr, where it
// ran this pass), then the winner's own if it was evaluated densely (or
// slot 0 of a fill): its residual streams from the first one it changed,
// the attention outputs of the blocks whose attention it ran, the logits
// and the per-position losses.  One thread per element of the largest array
// (N x max(D, V)); block 0 applies the parameter and the state and records
// the winner as the next pending recomputation if it was scored
// incrementally.
__global__ __launch_bounds__(kCopyThreads) void k_tf_commit(const TfDev* tf, const mca_cand* cands,
                                                            const Aux* aux, const double* dL,
                                                            DevState* st, int k_host, int fill) {
  const int NB = tf->NB, kr = tf->kr;
  // k_host -2: no winner (only the pending recomputation is folded in)
  const int w = fill ? 0 : (k_host >= 0 ? k_host : (k_host == -2 ? -1 : st->chosen));
  const bool wd = w >= 0 && tf->kind[w] == kTfDense && tf->start[w] <= NB + 1;
  const bool rd = !fill && redo_on(tf);
  const int64_t N = tf->N, ND = N * tf->D, NV = N * tf->V;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < ND) {
    for (int j = 0; j <= NB; ++j) {
      const float* src = (wd && j >= tf->xin[w]) ? slot_x(tf, w, j)
                         : (rd && j >= tf->xin[kr]) ? slot_x(tf, kr, j) : nullptr;
      if (src != nullptr) tf->x[j][e] = src[e];
    }
    for (int b = 0; b < NB; ++b) {
      const float* src = (wd && runs_attention(tf, w, b)) ? slot_h(tf, w, b)
                         : (rd && runs_attention(tf, kr, b)) ? slot_h(tf, kr, b) : nullptr;
      if (src != nullptr) tf->ch[b][e] = src[e];
    }
  }
  const float* zs = wd ? slot_log(tf, w) : (rd ? slot_log(tf, kr) : nullptr);
  if (zs != nullptr && e < NV) tf->cz[e] = zs[e];
  const float* ls = wd ? slot_ell(tf, w) : (rd ? slot_ell(tf, kr) : nullptr);
  if (ls != nullptr && e < N) tf->ell[e] = ls[e];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    int rs = NB + 2, rh = 0, rx = NB + 2;  // no recomputation pending
    if (!fill && w >= 0) {
      const mca_cand c = cands[w];
      tf->param[c.layer][(int64_t)c.j * tf->cols[c.layer] + c.i] = aux[w].w_new;
      st->L += dL[w];
      st->accepted += 1;
      const int kind = tf->kind[w];
      if (kind == kTfProjCol || kind == kTfFcCol) {
        rs = rh = rx = (c.layer - 2) / kBlockTensors + 1;  // from the block's MLP half
      } else if (kind != kTfDense) {
        rs = rx = NB + 1;  // the final stage
      }
    }
    tf->redo[kRedoStart] = rs;
    tf->redo[kRedoHalf] = rh;
    tf->redo[kRedoXin] = rx;
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
  const int ncand = identity ? 1 : K;
  const unsigned rows = identity ? 1u : (unsigned)(K + 1);  // + the pending recomputation
  const int64_t N = h.N;
  const unsigned mt = (unsigned)((N + kGemmRows - 1) / kGemmRows);
  auto tiles = [](int64_t n, int w) { return (unsigned)((n + w - 1) / w); };
  hipLaunchKernelGGL(k_tf_prep,
                     dim3((unsigned)((h.copy_stride + kCopyChunk - 1) / kCopyChunk), rows),
                     dim3(kCopyThreads), 0, s, tf, cands, aux, identity ? kPrepIdentity : kPrepEval,
                     ncand);
  hipLaunchKernelGGL(k_tf_embed,
                     dim3((unsigned)((N * h.D + kCopyThreads * kEmbedPer - 1) / (kCopyThreads * kEmbedPer)), rows),
                     dim3(kCopyThreads), 0, s, tf, ncand);
  const dim3 srow((unsigned)((N + (kRowThreads / 64) * 4 * kStatSteps - 1) / ((kRowThreads / 64) * 4 * kStatSteps)), rows);
  const bool wide = h.D > 128;  // row pairs per lane of the 16-lane layout: 4 or 8
  auto stats = [&](int stage, int which) {
    if (wide)
      hipLaunchKernelGGL(k_tf_stats<8>, srow, dim3(kRowThreads), 0, s, tf, cands, aux, stage, which, ncand);
    else
      hipLaunchKernelGGL(k_tf_stats<4>, srow, dim3(kRowThreads), 0, s, tf, cands, aux, stage, which, ncand);
  };
  for (int b = 0; b < h.NB; ++b) {
    const int stage = b + 1;
    stats(stage, 0);
    hipLaunchKernelGGL((k_tf_gemm<0, 2, 2>), dim3(mt, tiles(3 * h.D, 64), rows), dim3(kGemmThreads), 0, s, tf,
                       stage, (int)kGemmQKV, ncand);
    hipLaunchKernelGGL(k_tf_attn, dim3((unsigned)(h.S * h.H), rows), dim3(256), 0, s, tf, stage, ncand);
    hipLaunchKernelGGL((k_tf_gemm<2, 2, 2>), dim3(mt, tiles(h.D, 64), rows), dim3(kGemmThreads), 0, s, tf, stage,
                       (int)kGemmO, ncand);
    stats(stage, 1);
    hipLaunchKernelGGL((k_tf_gemm<1, 2, 2>), dim3(mt, tiles(h.M, 64), rows), dim3(kGemmThreads), 0, s, tf, stage,
                       (int)kGemmFc, ncand);
    hipLaunchKernelGGL((k_tf_gemm<2, 2, 2>), dim3(mt, tiles(h.D, 64), rows), dim3(kGemmThreads), 0, s, tf, stage,
                       (int)kGemmProj, ncand);
  }
  stats(h.NB + 1, 2);
  // the output layer: one column tile over the vocabulary (80 or 128 wide)
  if (h.V <= 80)
    hipLaunchKernelGGL((k_tf_gemm<3, 5, 1>), dim3(mt, 1, rows), dim3(kGemmThreads), 0, s, tf, h.NB + 1,
                       (int)kGemmOut, ncand);
  else
    hipLaunchKernelGGL((k_tf_gemm<3, 8, 1>), dim3(mt, 1, rows), dim3(kGemmThreads), 0, s, tf, h.NB + 1,
                       (int)kGemmOut, ncand);
  if (!identity && K > 0) {
    if (wide)
      hipLaunchKernelGGL(k_tf_dl<8>, dim3((unsigned)nblk, (unsigned)K), dim3(kLossThreads), 0, s, tf,
                         cands, aux, partial, nblk);
    else
      hipLaunchKernelGGL(k_tf_dl<4>, dim3((unsigned)nblk, (unsigned)K), dim3(kLossThreads), 0, s, tf,
                         cands, aux, partial, nblk);
  }
  return hipGetLastError();
}

hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, hipStream_t s) {
  const int64_t n = h.N * std::max(h.D, h.V);
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
