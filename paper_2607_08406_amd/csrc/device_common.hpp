// Device-side building blocks shared by every MCA kernel: the network
// description passed by value to each launch, the per-candidate prepared
// values, the device state word block, the transfer functions, the loss
// change of one sample in difference form, and the Philox4x64-10 candidate
// stream.
//
// All floating point here is IEEE fp32 with contraction disabled at build
// time; the only fused multiply-adds are the explicit fmaf() calls, so the
// same expression evaluates to the same bits in every kernel that uses it.
//
// Loss changes are formed from the *changes* of the local fields, never as
// the difference of two losses: a sample's loss is ~2.3 (ulp 2.4e-7) while a
// mutation moves it by as little as 1e-11 in a deep net.  With exact
// identities (tanh and Gaussian differences, the log-sum-exp difference) and
// an expm1/log1p that keep relative precision near zero, every change keeps
// a few ulp of relative precision whatever its size.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mca.h"

namespace mca {

constexpr int kTile = 256;          // samples per block in the column kernels
constexpr int kMaxK = 1024;         // candidates per step (one select thread each)
constexpr int kCMax = MCA_MAX_CLASSES;

// Everything a kernel needs to know about the net and where it lives in HBM.
// Unit-major caches: Z[l] is [n_{l+1}][Ns] (the samples of one unit are
// contiguous), XT is [n_0][Ns]; weights stay [n_{l+1}][n_l] row-major.
struct NetDev {
  int32_t L;        // weight matrices
  int32_t C;        // logits per sample (= widths[L])
  int32_t act;      // MCA_ACT_*
  float gamma;
  int32_t ternary;  // weights are code * scale
  int32_t pick;     // MCA_PICK_*
  float delta;
  float bound;      // > 0: reject |w'| >= bound
  int32_t ties;     // accept dL <= 0
  int32_t rule;     // MCA_RULE_*
  uint64_t seed, tag;
  double beta;      // Metropolis selection intensity
  int32_t n_prune;  // candidates 0 .. n_prune-1 of a step set their weight to zero
  int32_t pad0;
  int64_t sub_size, sub_period;  // minibatch window (0: every sample)
  int64_t N, Ns;    // samples, row stride of the unit-major caches
  int64_t P;        // parameters
  int32_t widths[MCA_MAX_LAYERS + 1];
  int64_t offs[MCA_MAX_LAYERS + 1];   // flat offset of each layer, offs[L] = P
  float scales[MCA_MAX_LAYERS];
  float* W[MCA_MAX_LAYERS];
  int8_t* codes[MCA_MAX_LAYERS];
  float* Z[MCA_MAX_LAYERS];           // Z[l] = output local fields of layer l
  const float* XT;
  float* ell;                         // per-sample loss cache
  float* prob;                        // softmax of the logits, [C][Ns] (unit-major like Z)
  const int32_t* y;
  float* WT;                          // L >= 3: W_{L-2} transposed ([n_{L-2}][n_{L-1}]), else null
  int32_t mutation;                   // MCA_MUTATE_*
  int32_t pad1;
  float chan_amp[MCA_MAX_LAYERS];     // fl32(sqrt(8 / n_l)): amplitude of a re-drawn channel weight
  // deep nets of Sec. 2.1: biases (candidate column i = n_l of layer l),
  // normalized hidden fields, the layer-sticky schedule
  int32_t bias;                       // 1: every layer has a bias vector B[l]
  int32_t ln;                         // 1: hidden fields are normalized over their layer
  float ln_eps;
  int32_t sticky;                     // steps per block of the MCA_PICK_STICKY schedule
  float* B[MCA_MAX_LAYERS];           // biases [n_{l+1}], or null
};

// Kernels index the pointer and size arrays of NetDev with runtime values (the
// candidate's layer).  Indexing the by-value kernel argument that way makes
// the compiler fetch each pointer from the kernel-argument segment with a
// dependent vector load; the block therefore copies the descriptor to LDS
// once (one word per thread) and every lane indexes the LDS copy.  Every
// thread of the block must call this (it synchronises the block).
// Blocks have at least 64 threads; every load is issued before the stores.
__device__ __forceinline__ void stage_net(NetDev& dst, const NetDev& src) {
  static_assert(sizeof(NetDev) % 4 == 0, "descriptor copied in words");
  constexpr int kWords = (int)(sizeof(NetDev) / 4);
  constexpr int kPer = (kWords + 63) / 64;
  const uint32_t* s = reinterpret_cast<const uint32_t*>(&src);
  uint32_t* d = reinterpret_cast<uint32_t*>(&dst);
  uint32_t v[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int w = (int)threadIdx.x + u * (int)blockDim.x;
    v[u] = (w < kWords) ? s[w] : 0u;
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int w = (int)threadIdx.x + u * (int)blockDim.x;
    if (w < kWords) d[w] = v[u];
  }
  __syncthreads();
}

// Accesses through NetDev's pointers.  A pointer read from the LDS copy of the
// descriptor has no known address space, so a plain dereference becomes a
// flat access; a flat access counts on the LDS counter too, so every later LDS
// wait would also wait for it.  These helpers state that the pointee is in
// global memory.
template <class T>
__device__ __forceinline__ T gload(const T* p) {
  return *(const __attribute__((address_space(1))) T*)p;
}
template <class T>
__device__ __forceinline__ void gstore(T* p, T v) {
  *(__attribute__((address_space(1))) T*)p = v;
}

// A candidate's new value, prepared once per step against the committed state.
struct Aux {
  float w_old;
  float w_new;
  float de;       // fl32(w_new - w_old): the increment the caches apply
  int32_t valid;  // 0: |w_new| >= bound, rejected without evaluation
  double theta;   // acceptance threshold: 0 greedy (Eq. 6), -ln(U) / beta Metropolis (Eq. 7)
};

// Committed scalars and counters, one 256-byte block in the workspace.
struct DevState {
  double L;              // committed loss
  uint64_t t;            // next step index
  int32_t chosen;        // decision of the last selected step (-1: none)
  int32_t K;
  uint64_t steps, evaluated, accepted, wasted, tie;
  uint64_t trace_base;   // step index stored at trace slot 0
  uint32_t sel_done;     // blocks of the selection kernel done (zero between launches)
  uint32_t pad32;
  uint64_t pad[5];
};
static_assert(sizeof(DevState) <= 256, "state block");

// ---------------------------------------------------------------------------
// transfer function and loss
// ---------------------------------------------------------------------------

// The transcendentals of the hot path use the hardware exp2/log2/rcp units:
// e^x = 2^(x log2 e), ln x = log2(x) ln 2.  Their error is a few ulp; every
// kernel (forward, evaluation, commit) calls these same functions, so an
// unchanged sample evaluates to the same bits everywhere.
__device__ __forceinline__ float fast_exp(float x) {
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}
__device__ __forceinline__ float fast_log(float x) {
  return __builtin_amdgcn_logf(x) * 0.6931471805599453f;
}

// e^x - 1 for |x| < kEm1Small: the degree-5 Taylor polynomial (truncation
// below x^5 / 720 < 2^-24 relative there).
constexpr float kEm1Small = 0.125f;
__device__ __forceinline__ float em1_small(float x) {
  float p = fmaf(x, 1.0f / 120.0f, 1.0f / 24.0f);
  p = fmaf(x, p, 1.0f / 6.0f);
  p = fmaf(x, p, 0.5f);
  p = fmaf(x, p, 1.0f);
  return x * p;
}

// tanh z with a few ulp of relative error for every z: near zero
// e / (e + 2) with e = expm1(2z) from the polynomial, elsewhere
// sign(z) (1 - t) / (1 + t) with t = e^{-2|z|} (1 - 2 / (e^{2z} + 1) would
// cancel near zero: deep nets with small weights carry activations of 1e-6,
// which it gets wrong by percents).
__device__ __forceinline__ float fast_tanh(float z) {
  const float e = em1_small(z + z);
  const float near = e * __builtin_amdgcn_rcpf(e + 2.0f);
  const float t = fast_exp(-2.0f * fabsf(z));
  const float far = copysignf((1.0f - t) * __builtin_amdgcn_rcpf(1.0f + t), z);
  return (fabsf(z + z) < kEm1Small) ? near : far;
}

__device__ __forceinline__ float act_fn(float z, int act, float gamma) {
  if (act == MCA_ACT_TANH) return fast_tanh(z);
  if (act == MCA_ACT_RELU) return fmaxf(z, 0.0f);
  float t = gamma * z;
  t = t * z;
  return fast_exp(-t);
}

// e^x - 1 away from zero (|x| >= kEm1Small), a few ulp: Kahan's
// (u - 1) x / ln u with u = e^x, which cancels the rounding of u.
__device__ __forceinline__ float em1_large(float x) {
  const float u = fast_exp(x);
  const float k = (u - 1.0f) * (x * __builtin_amdgcn_rcpf(fast_log(u)));
  const float r = (x < -17.0f) ? -1.0f : k;  // fl32(e^x - 1) = -1 below -17
  return (u == __builtin_huge_valf()) ? u : r;
}

// e^x - 1 for every x, a few ulp: the polynomial near zero, Kahan's form
// elsewhere.
__device__ __forceinline__ float em1(float x) {
  return (fabsf(x) < kEm1Small) ? em1_small(x) : em1_large(x);
}

// ln(1 + s) for s > -1, a few ulp: Kahan's ln(u) s / (u - 1) with u = 1 + s.
__device__ __forceinline__ float lg1p(float s) {
  const float u = 1.0f + s;
  const float r = fast_log(u) * (s * __builtin_amdgcn_rcpf(u - 1.0f));
  return (u == 1.0f) ? s : r;
}

// tanh(z + dz) - tanh(z) without cancellation: tanh(dz) (1 - tanh z tanh(z + dz)),
// where, with u = e^{-2|z|} and v = e^{-2|z + dz|}, 1 - tanh a tanh b is
// 2 (u + v) / ((1 + u)(1 + v)) when a and b share a sign and
// 2 (1 + u v) / ((1 + u)(1 + v)) otherwise (no difference of near-equal
// values either way), and tanh(dz) = e / (e + 2) with e = expm1(2 dz).
// Exactly zero where dz is zero.
__device__ __forceinline__ float dtanh(float z, float dz) {
  const float zn = z + dz;
  const float u = fast_exp(-2.0f * fabsf(z)), v = fast_exp(-2.0f * fabsf(zn));
  const bool same = (z < 0.0f) == (zn < 0.0f);
  const float w = same ? u + v : fmaf(u, v, 1.0f);
  const float f = (2.0f * w) * __builtin_amdgcn_rcpf((1.0f + u) * (1.0f + v));
  const float e = em1(fminf(fmaxf(2.0f * dz, -40.0f), 40.0f));
  return (e * __builtin_amdgcn_rcpf(e + 2.0f)) * f;
}

// exp(-g (z + dz)^2) - exp(-g z^2) = exp(-g z^2) expm1(-g dz (2 z + dz));
// a move out of a far tail (the expm1 argument above 30) has nothing to
// cancel and takes the plain difference.  The far tail lies in the branch of
// arguments away from zero, so the common case of a small move costs one
// exponential.  Exactly zero where dz is zero.
__device__ __forceinline__ float dgauss(float z, float dz, float g) {
  const float x = (-g * dz) * fmaf(2.0f, z, dz);
  const float pz = act_fn(z, MCA_ACT_GAUSS, g);
  if (fabsf(x) < kEm1Small) return pz * em1_small(x);
  return (x > 30.0f) ? act_fn(z + dz, MCA_ACT_GAUSS, g) - pz : pz * em1_large(x);
}

// max(0, z + dz) - max(0, z): dz itself where both fields are positive (no
// rounding), zero where neither is, the one non-zero activation where they
// straddle zero.  Exactly zero where dz is zero.
__device__ __forceinline__ float drelu(float z, float dz) {
  const float zn = z + dz;
  return (z > 0.0f && zn > 0.0f) ? dz : fmaxf(zn, 0.0f) - fmaxf(z, 0.0f);
}

// phi(z + dz) - phi(z) for the net's transfer function.
__device__ __forceinline__ float dphi(float z, float dz, int act, float gamma) {
  if (act == MCA_ACT_RELU) return drelu(z, dz);
  return (act == MCA_ACT_TANH) ? dtanh(z, dz) : dgauss(z, dz, gamma);
}

// Softmax p of C <= CM logits and the cross-entropy logsumexp(z) - z[y]
// (maximum subtracted first; summation order c = 0..C-1, so every CM >= C
// gives the same bits).  p is zero beyond C.
template <int CM>
__device__ __forceinline__ float softmax_ce(const float (&z)[CM], int C, int y, float (&p)[CM]) {
  float m = z[0];
#pragma unroll
  for (int c = 1; c < CM; ++c)
    if (c < C) m = fmaxf(m, z[c]);
  float s = 0.f, zy = 0.f;
#pragma unroll
  for (int c = 0; c < CM; ++c) {
    p[c] = (c < C) ? fast_exp(z[c] - m) : 0.f;
    s += p[c];
    zy = (c == y) ? z[c] : zy;
  }
  const float r = __builtin_amdgcn_rcpf(s);
#pragma unroll
  for (int c = 0; c < CM; ++c) p[c] *= r;
  return (fast_log(s) + m) - zy;
}

// Change of one sample's cross-entropy when its logits move by dz[c] (Eq. 2):
// ln(sum_c p_c e^{dz_c}) - dz_y = log1p(sum_c p_c expm1(dz_c)) - dz_y, with p
// the softmax of the committed logits.  Zero exactly where every dz is zero.
template <int CM>
__device__ __forceinline__ float ce_change(const float (&p)[CM], const float (&dz)[CM], int C,
                                           float dzy) {
  float amax = 0.f;
#pragma unroll
  for (int c = 0; c < CM; ++c)
    if (c < C) amax = fmaxf(amax, fabsf(dz[c]));
  float s = 0.f;
  if (amax < kEm1Small) {
#pragma unroll
    for (int c = 0; c < CM; ++c)
      if (c < C) s = fmaf(p[c], em1_small(dz[c]), s);
  } else {
    // large changes (rare): one class at a time, so the general expm1's
    // temporaries of different classes are never live together
#pragma unroll
    for (int c = 0; c < CM; ++c) {
      if (c < C) s = fmaf(p[c], em1(dz[c]), s);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  return lg1p(s) - dzy;
}

// ---------------------------------------------------------------------------
// one (candidate, sample) pair of a mutation in the last two layers
// ---------------------------------------------------------------------------

// One (candidate, sample) pair: the mutated weight's input ain moves its unit
// by dz = de * ain.  A logit-layer weight moves logit j by dz; a hidden unit's
// activation moves by da = phi(zh + dz) - phi(zh) (zh its cached local field)
// and the logits by da * wcol[c] (the unit's logit-layer column).  wcol is
// one-hot at j for a logit-layer weight, so one expression serves both:
// da = dz there and dz_c = dz * [c == j].  w holds wcol's C values (the
// caller loads them: scalars when the pairs share a candidate).  wmax bounds |wcol[c]|: when
// |da| wmax is small every expm1 takes the polynomial (no per-class test).
// pL: the sample's softmax in LDS (class stride ZS).  Returns the sample's
// loss change; da comes back for a commit.  Written without branches on the
// candidate's layer (pairs of different candidates share a wave); the step
// loop and the batched evaluation both score pairs with it.
template <int CM, int ZS = 64>
__device__ __forceinline__ float pair_change(int C, int act, float gamma, bool logit, float zh,
                                             float de, const float (&w)[CM], const float* wcol,
                                             float wmax, float ain, const float* pL, int y,
                                             float& da) {
  const float dz = de * ain;
  da = logit ? dz : dphi(zh, dz, act, gamma);
  // every softmax operand is loaded unconditionally (the LDS rows hold CM
  // entries, zero beyond C) so the loads issue together
  float p[CM];
#pragma unroll
  for (int cc = 0; cc < CM; ++cc) p[cc] = pL[cc * ZS];
  const float wy = wcol[y];
  float s = 0.f;
  if (fabsf(da) * wmax < kEm1Small) {
#pragma unroll
    for (int cc = 0; cc < CM; ++cc)
      if (cc < C) s = fmaf(p[cc], em1_small(da * w[cc]), s);
  } else {
    // large changes (rare on wide nets): one class at a time from LDS, so the
    // general expm1's temporaries of different classes are never live together
#pragma unroll 1
    for (int cc = 0; cc < C; ++cc) s = fmaf(pL[cc * ZS], em1(da * wcol[cc]), s);
  }
  return lg1p(s) - da * wy;
}

// Maximum of v over lanes 0..15 (one DPP row), returned wave-uniform.  All
// 64 lanes must be active.
template <int kCtrl>
__device__ __forceinline__ float dpp_max_f32(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xF, 0xF, true));
}
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, dpp_max_f32<0xB1>(v));   // lane ^ 1
  v = fmaxf(v, dpp_max_f32<0x4E>(v));   // lane ^ 2
  v = fmaxf(v, dpp_max_f32<0x141>(v));  // mirror within eight
  v = fmaxf(v, dpp_max_f32<0x140>(v));  // mirror within sixteen
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
}

// The committed logits after a pair's change: z[c] + da * wcol[c] (for a
// logit-layer weight, wcol one-hot: only logit j moves, by dz).
template <int CM>
__device__ __forceinline__ void moved_logits(int C, float da, const float (&wc)[CM],
                                             const float (&zc)[CM], float (&z)[CM]) {
#pragma unroll
  for (int cc = 0; cc < CM; ++cc) z[cc] = (cc < C) ? fmaf(da, wc[cc], zc[cc]) : 0.f;
}

// ---------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11)
// ---------------------------------------------------------------------------

struct Words { uint64_t w0, w1, w2, w3; };

__device__ __forceinline__ Words philox4x64_10(uint64_t x0, uint64_t x1, uint64_t x2,
                                               uint64_t x3, uint64_t k0, uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) { k0 += W0; k1 += W1; }
    const uint64_t lo0 = M0 * x0, hi0 = __umul64hi(M0, x0);
    const uint64_t lo1 = M1 * x2, hi1 = __umul64hi(M1, x2);
    const uint64_t n0 = hi1 ^ x1 ^ k0, n2 = hi0 ^ x3 ^ k1;
    x0 = n0; x1 = lo1; x2 = n2; x3 = lo0;
  }
  return Words{x0, x1, x2, x3};
}

// Decode draw (t, k) into a candidate (Eq. 1; Eq. 12 for ternary codes) in
// two parts.  decode_index() needs no state: parameter, row, column and, for
// continuous weights, the increment; for ternary weights it leaves the
// selecting bit (w3 >> 63) in c.code.  finish_ternary() then picks the new
// code from the committed one.
__device__ __forceinline__ mca_cand decode_index(const NetDev& net, uint64_t t, uint64_t k) {
  const Words w = philox4x64_10(t, k, 0, 0, net.seed, net.tag);
  int layer;
  int64_t off;
  if (net.pick == MCA_PICK_LAYER || net.pick == MCA_PICK_STICKY) {
    if (net.pick == MCA_PICK_LAYER) {
      layer = (int)__umul64hi(w.w1, (uint64_t)net.L);
    } else {  // the layer of the step's block: word 0 of counter (t / sticky, 0, 0, 1)
      const Words b = philox4x64_10(t / (uint64_t)net.sticky, 0, 0, 1, net.seed, net.tag);
      layer = (int)__umul64hi(b.w0, (uint64_t)net.L);
    }
    const int64_t size = net.offs[layer + 1] - net.offs[layer];
    off = (int64_t)__umul64hi(w.w0, (uint64_t)size);
  } else {
    const int64_t flat = (int64_t)__umul64hi(w.w0, (uint64_t)net.P);
    layer = 0;
    for (int l = 1; l < net.L; ++l)
      if (flat >= net.offs[l]) layer = l;
    off = flat - net.offs[layer];
  }
  // every layer has fewer than 2^31 entries: 32-bit division suffices; a
  // row of a biased layer ends with its bias (column n_l)
  const uint32_t nin = (uint32_t)(net.widths[layer] + net.bias);
  mca_cand c;
  c.flat = net.offs[layer] + off;
  c.layer = layer;
  c.j = (int32_t)((uint32_t)off / nin);
  c.i = (int32_t)((uint32_t)off - (uint32_t)c.j * nin);
  c.flags = ((int64_t)k < (int64_t)net.n_prune) ? MCA_CAND_PRUNE : 0;
  if (net.ternary) {
    c.d = 0.f;
    c.code = (int)(w.w3 >> 63);
  } else {
    const float m = (float)(uint32_t)(w.w2 >> 40);
    const float r = m * 0x1p-23f - 1.0f;
    c.d = net.delta * r;
    c.code = 0;
  }
  return c;
}

// c.code holds the selecting bit on entry and the new code on return.
__device__ __forceinline__ void finish_ternary(const NetDev& net, mca_cand& c, int cur) {
  const int b = c.code;
  // the b-th of the two other codes, ascending
  const int nc = (cur == -1) ? (b ? 1 : 0) : (cur == 0 ? (b ? 1 : -1) : (b ? 0 : -1));
  const float s = net.scales[c.layer];
  const float a = (float)nc * s;
  const float o = (float)cur * s;
  c.d = a - o;
  c.code = nc;
}

// The committed value of a candidate's parameter: a weight, or a bias (column n_l).
__device__ __forceinline__ float param_value(const NetDev& net, int l, int j, int i) {
  if (i == net.widths[l]) return net.B[l][j];
  return net.W[l][(int64_t)j * net.widths[l] + i];
}

__device__ __forceinline__ mca_cand decode_candidate(const NetDev& net, uint64_t t, uint64_t k) {
  mca_cand c = decode_index(net, t, k);
  const int64_t idx = (int64_t)c.j * net.widths[c.layer] + c.i;
  if (net.ternary) finish_ternary(net, c, net.codes[c.layer][idx]);
  if (c.flags & MCA_CAND_PRUNE) {  // w' = 0: the increment is -w
    c.code = 0;
    c.d = 0.0f - param_value(net, c.layer, c.j, c.i);
  }
  return c;
}

// New value of a candidate against the committed weights (a pruning
// candidate's is zero).
__device__ __forceinline__ Aux prepare_candidate(const NetDev& net, const mca_cand& c) {
  Aux a;
  a.w_old = param_value(net, c.layer, c.j, c.i);
  a.w_new = (c.flags & MCA_CAND_PRUNE) ? 0.0f
            : (net.ternary ? (float)c.code * net.scales[c.layer] : a.w_old + c.d);
  a.de = a.w_new - a.w_old;
  a.valid = !(net.bound > 0.f && fabsf(a.w_new) >= net.bound);
  a.theta = 0.0;
  return a;
}

// The selection test: Eq. 6 (dL < 0, or dL <= 0 with ties) when theta is 0;
// the Metropolis rule of Eq. 7 as dL < theta otherwise (theta > 0).  NaN
// compares false either way, +inf never passes.
// Minibatch (Sec. 2.2): step t averages its loss changes over the window of
// sub_size samples starting at ((t / sub_period) mod N) * sub_size mod N,
// wrapping around the sample order; without one, over every sample.
__device__ __forceinline__ int64_t subset_start(const NetDev& net, uint64_t t) {
  if (net.sub_size == 0) return 0;
  const uint64_t e = t / (uint64_t)net.sub_period;
  return (int64_t)(((e % (uint64_t)net.N) * (uint64_t)net.sub_size) % (uint64_t)net.N);
}
__device__ __forceinline__ bool in_subset(const NetDev& net, int64_t start, int64_t n) {
  if (net.sub_size == 0) return true;
  int64_t d = n - start;
  d += (d < 0) ? net.N : 0;
  return d < net.sub_size;
}
__device__ __forceinline__ double subset_count(const NetDev& net) {
  return (double)(net.sub_size ? net.sub_size : net.N);
}

__device__ __forceinline__ bool accepts(double dL, int ties, double theta = 0.0) {
  if (theta > 0.0) return dL < theta;
  return ties ? (dL <= 0.0) : (dL < 0.0);
}

// A first-layer weight multiplies the raw input: the evaluation tiles where
// its feature is zero throughout cannot change (fmask null: no such list).
__device__ __forceinline__ uint64_t candidate_tiles(const mca_cand& c, const uint64_t* fmask) {
  return (c.layer == 0 && fmask != nullptr) ? fmask[c.i] : ~0ull;
}

// Metropolis threshold of candidate k of step t (Eq. 7): U from word 0 of the
// Philox block at counter (t, k, 1, 0), U = (w0 >> 11) 2^-53, and
// U < exp(-beta dL) exactly when dL < -ln(U) / beta.  0 under the greedy rule.
__device__ __forceinline__ double accept_theta(int rule, double beta, uint64_t seed,
                                               uint64_t tag, uint64_t t, uint64_t k) {
  if (rule != MCA_RULE_METROPOLIS) return 0.0;
  const Words w = philox4x64_10(t, k, 1, 0, seed, tag);
  const double u = (double)(w.w0 >> 11) * 0x1p-53;
  return (u == 0.0) ? __builtin_huge_val() : -log(u) / beta;
}

// Sum of v over the 64 lanes of a wave in one fixed order (a butterfly within
// rows of 16 by DPP, then across rows), returned in every lane.  All 64
// lanes must be active.
template <int kCtrl>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xF, 0xF, true));
}
__device__ __forceinline__ float wave_sum_f32(float v) {
  v += dpp_f32<0xB1>(v);   // lane ^ 1
  v += dpp_f32<0x4E>(v);   // lane ^ 2
  v += dpp_f32<0x141>(v);  // mirror within eight
  v += dpp_f32<0x140>(v);  // mirror within sixteen
  v += __shfl_xor(v, 16, 64);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0)) +
         __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
}

// Sum of v over a block of kTile threads (4 waves of 64), fixed order.
// The result is valid in thread 0.
__device__ __forceinline__ float block_sum_256(float v, float* smem4) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) smem4[wave] = v;
  __syncthreads();
  float r = 0.f;
  if (threadIdx.x == 0) r = ((smem4[0] + smem4[1]) + smem4[2]) + smem4[3];
  return r;
}

// Commit of candidate (l, j, i, de) on sample n, for a weight in the last
// two layers: the mutated unit's local field moves by dz = de * ain; the
// logits move by dz (a logit-layer weight) or by da * W_{L-1}[:, j] with
// da = phi(z + dz) - phi(z) (the expressions of the evaluation); the
// sample's softmax and loss are recomputed from its new logits.
__device__ __forceinline__ void column_commit(const NetDev& net, int l, int j, int i, float de,
                                              int64_t n) {
  const int L = net.L, C = net.C;
  const int64_t Ns = net.Ns;
  const float ain = (l == 0) ? gload(&net.XT[(int64_t)i * Ns + n])
                             : act_fn(gload(&net.Z[l - 1][(int64_t)i * Ns + n]), net.act, net.gamma);
  if (ain == 0.f) return;  // nothing changes for this sample
  float* zrow = net.Z[l] + (int64_t)j * Ns;
  const float zl = gload(&zrow[n]);
  const float dz = de * ain;
  float* ZL = net.Z[L - 1];
  float zc[kCMax], wc[kCMax];
#pragma unroll
  for (int c = 0; c < kCMax; ++c) zc[c] = (c < C) ? gload(&ZL[(int64_t)c * Ns + n]) : 0.f;
  float da;
  if (l == L - 1) {
    da = dz;  // the mutated weight feeds logit j directly
#pragma unroll
    for (int c = 0; c < kCMax; ++c) wc[c] = (c == j) ? 1.f : 0.f;
  } else {
    // last hidden layer: rank-1 update of the logits through W_L[:, j]
    da = dphi(zl, dz, net.act, net.gamma);
    const float* WL = net.W[L - 1];
    const int nh = net.widths[L - 1];
#pragma unroll
    for (int c = 0; c < kCMax; ++c) wc[c] = (c < C) ? gload(&WL[(int64_t)c * nh + j]) : 0.f;
  }
  gstore(&zrow[n], zl + dz);
  if (da == 0.f) return;
  float z[kCMax], p[kCMax];
  moved_logits(C, da, wc, zc, z);
  const float ln = softmax_ce(z, C, gload(&net.y[n]), p);
#pragma unroll
  for (int c = 0; c < kCMax; ++c)
    if (c < C) {
      gstore(&ZL[(int64_t)c * Ns + n], z[c]);
      gstore(&net.prob[(int64_t)c * Ns + n], p[c]);
    }
  gstore(&net.ell[n], ln);
}

}  // namespace mca
