// Device-side building blocks shared by every MCA kernel: the network
// description passed by value to each launch, the per-candidate prepared
// values, the device state word block, the transfer functions, the per-sample
// cross-entropy, and the Philox4x64-10 candidate stream.
//
// All floating point here is IEEE fp32 with contraction disabled at build
// time; the only fused multiply-adds are the explicit fmaf() calls, so the
// same expression evaluates to the same bits in every kernel that uses it
// (evaluation, commit and the full forward pass agree bit for bit on an
// unchanged sample).
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
  int32_t pad0;
  uint64_t seed, tag;
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
  const int32_t* y;
  float* WT;                          // L >= 3: W_{L-2} transposed ([n_{L-2}][n_{L-1}]), else null
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
};

// Committed scalars and counters, one 256-byte block in the workspace.
struct DevState {
  double L;              // committed loss
  uint64_t t;            // next step index
  int32_t chosen;        // decision of the last selected step (-1: none)
  int32_t K;
  uint64_t steps, evaluated, accepted, wasted, tie;
  uint64_t trace_base;   // step index stored at trace slot 0
  uint64_t pad[6];
};
static_assert(sizeof(DevState) <= 256, "state block");

// ---------------------------------------------------------------------------
// transfer function and loss
// ---------------------------------------------------------------------------

// The transcendentals of the hot path use the hardware exp2/log2/rcp units:
// e^x = 2^(x log2 e), ln x = log2(x) ln 2, tanh z = 1 - 2 / (e^{2z} + 1).
// Their error (a few ulp, absolute error of tanh near 1e-7) is far below the
// fp32 rounding of the caches; every kernel (forward, evaluation, commit)
// calls these same functions, so an unchanged sample evaluates to the same
// bits everywhere.
__device__ __forceinline__ float fast_exp(float x) {
  return __builtin_amdgcn_exp2f(x * 1.4426950408889634f);
}
__device__ __forceinline__ float fast_log(float x) {
  return __builtin_amdgcn_logf(x) * 0.6931471805599453f;
}
__device__ __forceinline__ float fast_tanh(float z) {
  const float e = fast_exp(z + z);
  return 1.0f - 2.0f * __builtin_amdgcn_rcpf(e + 1.0f);
}

__device__ __forceinline__ float act_fn(float z, int act, float gamma) {
  if (act == MCA_ACT_TANH) return fast_tanh(z);
  float t = gamma * z;
  t = t * z;
  return fast_exp(-t);
}

// Cross-entropy of one sample from its C <= CM logits: logsumexp(z) - z[y],
// with the maximum subtracted first.  Summation order c = 0..C-1, so every
// CM >= C gives the same bits.
template <int CM>
__device__ __forceinline__ float ce_loss(const float (&z)[CM], int C, int y) {
  float m = z[0];
#pragma unroll
  for (int c = 1; c < CM; ++c)
    if (c < C) m = fmaxf(m, z[c]);
  float s = 0.f, zy = 0.f;
#pragma unroll
  for (int c = 0; c < CM; ++c) {
    if (c < C) s += fast_exp(z[c] - m);
    zy = (c == y) ? z[c] : zy;
  }
  return (fast_log(s) + m) - zy;
}

// ---------------------------------------------------------------------------
// one (candidate, sample) pair of a mutation in the last two layers
// ---------------------------------------------------------------------------

// One (candidate, sample) pair.  ain: the input of the mutated weight (x, or
// the activation feeding it); zh: the cached local field of the mutated unit
// when it is a hidden unit; zL: the sample's logits in LDS (class stride ZS).  The
// new local field, logits and loss come back for a commit.  Written without
// branches on the candidate's layer (pairs of different candidates share a
// wave); the step loop and the batched evaluation both score pairs with
// these expressions, and the column commit applies the same arithmetic.
// pair_logits_of takes the sample's logits zc and the column wc as values.
template <int CM>
__device__ __forceinline__ bool pair_logits_of(int C, int act, float gamma, bool logit, float zb,
                                               float de, const float (&wc)[CM], float ain,
                                               const float (&zc)[CM], float& zn, float& da,
                                               float (&z)[CM]) {
  const float dz = de * ain;
  zn = zb + dz;
  // A logit-layer candidate's staged column is one-hot at its logit j, which
  // moves by dz itself: fma(dz, 1, z_j) = z_j + dz = zn and fma(dz, 0, z) = z
  // exactly, so one expression serves both kinds of candidate.
  da = logit ? dz : act_fn(zn, act, gamma) - act_fn(zb, act, gamma);
#pragma unroll
  for (int cc = 0; cc < CM; ++cc) z[cc] = (cc < C) ? fmaf(da, wc[cc], zc[cc]) : 0.f;
  return logit ? dz != 0.f : da != 0.f;  // the logits changed
}

template <int CM, int ZS = 64>
__device__ __forceinline__ bool pair_logits(int L, int C, int act, float gamma, int layer, int j,
                                            float de, const float* wcol, float ain, float zh,
                                            const float* zL, float& zn, float& da,
                                            float (&z)[CM]) {
  const bool logit = layer == L - 1;
  // every operand is loaded unconditionally (the LDS rows hold CM entries,
  // zero beyond C) so the loads issue together
  float zc[CM], wc[CM];
#pragma unroll
  for (int cc = 0; cc < CM; ++cc) {
    zc[cc] = zL[cc * ZS];
    wc[cc] = wcol[cc];
  }
  const float zb = logit ? zL[j * ZS] : zh;
  return pair_logits_of<CM>(C, act, gamma, logit, zb, de, wc, ain, zc, zn, da, z);
}

// The pair's new loss ln; returns its loss change.
template <int CM, int ZS = 64>
__device__ __forceinline__ float pair_eval(int L, int C, int act, float gamma, int layer, int j,
                                           float de, const float* wcol, float ain, float zh,
                                           const float* zL, float ell, int y, float& ln) {
  float zn, da, z[CM];
  const bool changed = pair_logits<CM, ZS>(L, C, act, gamma, layer, j, de, wcol, ain, zh, zL, zn, da, z);
  // ce_loss() with the label's logit computed by the same fma instead of
  // selected from z: the same bits, without a compare per class
  const float zy = fmaf(da, wcol[y], zL[y * ZS]);
  float m = z[0];
#pragma unroll
  for (int c = 1; c < CM; ++c)
    if (c < C) m = fmaxf(m, z[c]);
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < CM; ++c)
    if (c < C) s += fast_exp(z[c] - m);
  ln = (fast_log(s) + m) - zy;
  return changed ? ln - ell : 0.f;
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
  if (net.pick == MCA_PICK_LAYER) {
    layer = (int)__umul64hi(w.w1, (uint64_t)net.L);
    const int64_t size = net.offs[layer + 1] - net.offs[layer];
    off = (int64_t)__umul64hi(w.w0, (uint64_t)size);
  } else {
    const int64_t flat = (int64_t)__umul64hi(w.w0, (uint64_t)net.P);
    layer = 0;
    for (int l = 1; l < net.L; ++l)
      if (flat >= net.offs[l]) layer = l;
    off = flat - net.offs[layer];
  }
  // every layer has fewer than 2^31 entries: 32-bit division suffices
  const uint32_t nin = (uint32_t)net.widths[layer];
  mca_cand c;
  c.flat = net.offs[layer] + off;
  c.layer = layer;
  c.j = (int32_t)((uint32_t)off / nin);
  c.i = (int32_t)((uint32_t)off - (uint32_t)c.j * nin);
  c.reserved = 0;
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

__device__ __forceinline__ mca_cand decode_candidate(const NetDev& net, uint64_t t, uint64_t k) {
  mca_cand c = decode_index(net, t, k);
  if (net.ternary)
    finish_ternary(net, c, net.codes[c.layer][(int64_t)c.j * net.widths[c.layer] + c.i]);
  return c;
}

// New value of a candidate against the committed weights.
__device__ __forceinline__ Aux prepare_candidate(const NetDev& net, const mca_cand& c) {
  Aux a;
  const int64_t idx = (int64_t)c.j * net.widths[c.layer] + c.i;
  a.w_old = net.W[c.layer][idx];
  a.w_new = net.ternary ? (float)c.code * net.scales[c.layer] : a.w_old + c.d;
  a.de = a.w_new - a.w_old;
  a.valid = !(net.bound > 0.f && fabsf(a.w_new) >= net.bound);
  return a;
}

__device__ __forceinline__ bool accepts(double dL, int ties) {
  // NaN compares false either way, +inf never passes
  return ties ? (dL <= 0.0) : (dL < 0.0);
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

}  // namespace mca
