// Single mutations in the deep nets of Sec. 2.1: every layer may carry a bias
// per unit, and every hidden field may be normalized over its layer, sample
// by sample, before the transfer function.  Normalization couples the units
// of a layer: changing one field moves that sample's mean and variance, so
// every unit of the layer (and of each later layer) changes.  A candidate in
// layer l therefore moves column j of z_l by de times its input (1 for a
// bias), and from there the kernel carries dense changes layer to layer:
//   normalization, for each sample with mean mu, S = var + eps, c = z - mu:
//     dmu = mean(dz), e = dz - dmu, dS = mean(e (2c + e))   (exact identity),
//     dh = e / sqrt(S + dS) - c dS / (sqrt S sqrt(S + dS) (sqrt S + sqrt(S + dS))),
//   so that h + dh = (z' - mu') / sqrt(S') with no difference of near-equal
//   values; then da = phi(h + dh) - phi(h) (dphi), and the next field's change
//   W_m da on the matrix cores (v_mfma_f32_16x16x4f32); the logits' change
//   gives each sample's loss change with the cached softmax (ce_change).
// A block takes T = 16384 / W consecutive samples of one candidate and keeps
// their changes in an LDS tile [T][W + 4]; the normalization pass gives each
// sample TPR = 256 / T threads (64 units each) and adds across them with a
// fixed butterfly.  The commit runs the same arithmetic, stores the moved
// fields and recomputes each moved sample's statistics from them; a second
// kernel then writes the parameter.
#include "device_common.hpp"
#include "norm_kernels.hpp"

namespace mca {

namespace {

constexpr int kNThreads = 256;
typedef float floatx4 __attribute__((ext_vector_type(4)));

// Sum over the TPR consecutive lanes of a row group (a butterfly: the same
// bits in every lane of the group).
template <int TPR>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = 1; o < TPR; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float inv_sqrt(float s) { return 1.0f / sqrtf(s); }

// Activation of hidden unit i of layer l for sample n from the caches.
__device__ __forceinline__ float hidden_act(const NetDev& net, const NormDev& nd, int l, int i,
                                            int64_t n) {
  const float z = gload(&net.Z[l][(int64_t)i * net.Ns + n]);
  if (!net.ln) return act_fn(z, net.act, net.gamma);
  const float h = (z - gload(&nd.MU[l][n])) * inv_sqrt(gload(&nd.S[l][n]));
  return act_fn(h, net.act, net.gamma);
}

// The activation change of hidden layer m from its field change dz (in the
// tile, replaced in place): thread (r, p) takes units p + TPR x of row r.
// A commit also stores the moved fields and, for a normalized layer, the
// moved samples' new statistics.
template <int W>
__device__ void norm_pass(const NetDev& net, const NormDev& nd, int m, float* ta, int64_t n0,
                          bool commit) {
  constexpr int T = 16384 / W, RS = W + 4, TPR = kNThreads / T, UPT = W / TPR;
  const int tid = threadIdx.x, r = tid / TPR, p = tid % TPR;
  const int64_t n = n0 + r, Ns = net.Ns;
  const bool live = n < net.N;  // rows past N read the padding and stay zero
  float* Zm = net.Z[m];
  float* row = ta + r * RS + p;  // this thread's units: row[TPR x], field z at zrow[TPR x Ns]
  const float* zrow = Zm + (int64_t)p * Ns + n;
  const int64_t zstep = (int64_t)TPR * Ns;
  const int act = net.act;
  const float gamma = net.gamma;
  float new_mu = 0.f, new_S = 0.f;
  // the moved rows (every pass below reads the fields again: they stay in cache)
  float sa = 0.f;
#pragma unroll 8
  for (int x = 0; x < UPT; ++x) sa += fabsf(row[TPR * x]);
  const bool moved = live && group_sum<TPR>(sa) != 0.f;  // the same in every lane of the row
  if (net.ln && commit && moved) {
    // a commit: the moved sample's statistics from its new fields z + dz
    // (taken before the fields are overwritten)
    float s = 0.f;
#pragma unroll 8
    for (int x = 0; x < UPT; ++x) s += gload(&zrow[zstep * x]) + row[TPR * x];
    const float mu1 = group_sum<TPR>(s) * (1.0f / W);
    float v = 0.f;
#pragma unroll 8
    for (int x = 0; x < UPT; ++x) {
      const float c = (gload(&zrow[zstep * x]) + row[TPR * x]) - mu1;
      v += c * c;
    }
    const float S1 = group_sum<TPR>(v) * (1.0f / W) + net.ln_eps;
    if (p == 0) {
      // stored after this sample's evaluation below has read the old ones
      new_mu = mu1;
      new_S = S1;
    }
  }
  if (net.ln) {
    float s1 = 0.f;
#pragma unroll 8
    for (int x = 0; x < UPT; ++x) s1 += row[TPR * x];
    const float dmu = group_sum<TPR>(s1) * (1.0f / W);
    const float mu = gload(&nd.MU[m][n]), S = gload(&nd.S[m][n]);
    float s2 = 0.f;
#pragma unroll 8
    for (int x = 0; x < UPT; ++x) {
      const float c = gload(&zrow[zstep * x]) - mu, e = row[TPR * x] - dmu;
      s2 += e * (c + c + e);
    }
    const float dS = group_sum<TPR>(s2) * (1.0f / W);
    const float q0 = sqrtf(S), q1 = sqrtf(S + dS);
    const float rs = 1.0f / q0, rs1 = 1.0f / q1;
    const float f = ((dS * rs) * rs1) / (q0 + q1);
#pragma unroll 4
    for (int x = 0; x < UPT; ++x) {
      const float z = gload(&zrow[zstep * x]), d = row[TPR * x];
      const float c = z - mu, e = d - dmu;
      const float dh = e * rs1 - c * f;
      row[TPR * x] = moved ? dphi(c * rs, dh, act, gamma) : 0.f;
      if (commit && moved) gstore(&Zm[(int64_t)(p + TPR * x) * Ns + n], z + d);
    }
    if (commit && moved && p == 0) {
      gstore(&nd.MU[m][n], new_mu);
      gstore(&nd.S[m][n], new_S);
    }
  } else {
#pragma unroll 4
    for (int x = 0; x < UPT; ++x) {
      const float z = gload(&zrow[zstep * x]), d = row[TPR * x];
      row[TPR * x] = moved ? dphi(z, d, act, gamma) : 0.f;
      if (commit && moved) gstore(&Zm[(int64_t)(p + TPR * x) * Ns + n], z + d);
    }
  }
}

}  // namespace

// grid (ntiles, K) for an evaluation, (ntiles, 1) for a commit.
template <int CM, int W>
__global__ __launch_bounds__(kNThreads, (W >= 1024) ? 1 : 2) void k_norm(
    NetDev net_arg, NormDev nd, const mca_cand* cands, const Aux* aux, float* partial,
    int ntiles, int k_mode, DevState* st) {
  constexpr int T = 16384 / W, SB = T / 16, UW = W / 4, CB = UW / 16, RS = W + 4;
  constexpr int TPR = kNThreads / T;
  static_assert(SB * CB == 16, "sixteen accumulator tiles per wave");
  __shared__ NetDev net;
  stage_net(net, net_arg);
  __shared__ __attribute__((aligned(16))) float ta[T * RS];
  __shared__ float incol[T];
  __shared__ float logit[T][CM];
  __shared__ float dls[T];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool commit = k_mode != -2;
  const int k = commit ? ((k_mode >= 0) ? k_mode : st->chosen) : (int)blockIdx.y;
  if (k < 0) return;
  const int tile = blockIdx.x;
  if (!commit && !aux[k].valid) {  // rejected unevaluated: selection gives +inf
    if (tid == 0) partial[(int64_t)k * ntiles + tile] = 0.f;
    return;
  }
  const mca_cand c = cands[k];
  const float de = aux[k].de;
  const int L = net.L, l = c.layer;
  const int C = (CM < kCMax) ? CM : net.C;
  const int64_t N = net.N, Ns = net.Ns;
  const int64_t n0 = (int64_t)tile * T;
  const bool is_bias = c.i == net.widths[l];

  // 1. the changed parameter's input on each sample (1 for a bias)
  if (tid < T) {
    const int64_t n = n0 + tid;
    float x = 0.f;
    if (n < N)
      x = is_bias ? 1.0f
                  : (l == 0 ? gload(&net.XT[(int64_t)c.i * Ns + n]) : hidden_act(net, nd, l - 1, c.i, n));
    incol[tid] = x;
  }
  __syncthreads();
  const int r4 = tid / TPR, cq = tid % TPR;  // logits: thread (row, class group)
  if (l == L - 1) {
    // a logit-layer parameter: only logit j moves
#pragma unroll
    for (int c0 = 0; c0 < CM; c0 += TPR) {
      const int cl = c0 + cq;
      if (cl < C) logit[r4][cl] = (cl == c.j) ? de * incol[r4] : 0.f;
    }
  } else {
    // 2. field change of layer l: column j
    for (int e = tid; e < T * W; e += kNThreads) {
      const int r = e / W, u = e - r * W;
      ta[r * RS + u] = (u == c.j) ? de * incol[r] : 0.f;
    }
    __syncthreads();
    norm_pass<W>(net, nd, l, ta, n0, commit);
    __syncthreads();
    // 3. dense layers m = l+1 .. L-2
    const int q = lane >> 4, li = lane & 15;
    for (int m = l + 1; m <= L - 2; ++m) {
      const float* Wm = net.W[m];
      floatx4 acc[SB][CB];
#pragma unroll
      for (int sb = 0; sb < SB; ++sb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) acc[sb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
      floatx4 bcur[CB], bnext[CB];
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        bcur[cb] = gload(reinterpret_cast<const floatx4*>(&Wm[(int64_t)(UW * wave + 16 * cb + li) * W + 4 * q]));
      for (int kb = 0; kb < W / 16; ++kb) {
        if (kb + 1 < W / 16) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            bnext[cb] = gload(reinterpret_cast<const floatx4*>(
                &Wm[(int64_t)(UW * wave + 16 * cb + li) * W + 16 * (kb + 1) + 4 * q]));
        }
        floatx4 a4[SB];
#pragma unroll
        for (int sb = 0; sb < SB; ++sb)
          a4[sb] = *reinterpret_cast<const floatx4*>(&ta[(16 * sb + li) * RS + 16 * kb + 4 * q]);
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
          for (int sb = 0; sb < SB; ++sb)
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
              acc[sb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[sb][t], bcur[cb][t], acc[sb][cb], 0, 0, 0);
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) bcur[cb] = bnext[cb];
      }
      __syncthreads();  // every wave has read the tile
#pragma unroll
      for (int sb = 0; sb < SB; ++sb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            ta[(16 * sb + 4 * q + v) * RS + UW * wave + 16 * cb + li] = acc[sb][cb][v];
      __syncthreads();
      norm_pass<W>(net, nd, m, ta, n0, commit);
      __syncthreads();
    }
    // 4. logit changes: the last hidden layer's change through W_{L-1}
    const float* WL = net.W[L - 1];
#pragma unroll
    for (int c0 = 0; c0 < CM; c0 += TPR) {
      const int cl = c0 + cq;
      if (cl < C) {
        float a = 0.f;
        for (int u = 0; u < W; ++u) a = fmaf(ta[r4 * RS + u], gload(&WL[(int64_t)cl * W + u]), a);
        logit[r4][cl] = a;
      }
    }
  }
  __syncthreads();
  // 5. per-sample loss change from the logit change and the cached softmax
  // (an evaluation counts the step's minibatch only); the tile's sum in row order
  if (tid < T) {
    const int64_t n = n0 + tid;
    float d = 0.f;
    if (n < N) {
      const int y = gload(&net.y[n]);
      float dz[CM], pr[CM], dzy = 0.f;
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) {
        dz[cc] = (cc < C) ? logit[tid][cc] : 0.f;
        pr[cc] = (cc < C) ? gload(&net.prob[(int64_t)cc * Ns + n]) : 0.f;
        dzy = (cc == y) ? dz[cc] : dzy;
      }
      d = ce_change<CM>(pr, dz, C, dzy);
      if (!commit && !in_subset(net, subset_start(net, st->t), n)) d = 0.f;
      if (commit) {
        float* ZL = net.Z[L - 1];
        float z[CM], pn[CM];
#pragma unroll
        for (int cc = 0; cc < CM; ++cc) z[cc] = (cc < C) ? gload(&ZL[(int64_t)cc * Ns + n]) + dz[cc] : 0.f;
        const float ln = softmax_ce<CM>(z, C, y, pn);
#pragma unroll
        for (int cc = 0; cc < CM; ++cc)
          if (cc < C) {
            gstore(&ZL[(int64_t)cc * Ns + n], z[cc]);
            gstore(&net.prob[(int64_t)cc * Ns + n], pn[cc]);
          }
        gstore(&net.ell[n], ln);
      }
    }
    dls[tid] = d;
  }
  __syncthreads();
  if (!commit && tid == 0) {
    float v = 0.f;
    for (int r = 0; r < T; ++r) v += dls[r];
    partial[(int64_t)k * ntiles + tile] = v;
  }
}

// After the field commit: the new parameter (weight or bias), the committed
// loss (a minibatch's change is not the loss's) and the count.
__global__ void k_norm_param(NetDev net, const mca_cand* cands, const Aux* aux, int k_mode,
                             DevState* st, const double* dL) {
  const int k = (k_mode >= 0) ? k_mode : st->chosen;
  if (k < 0 || threadIdx.x != 0) return;
  const mca_cand c = cands[k];
  const float w = aux[k].w_new;
  if (c.i == net.widths[c.layer]) net.B[c.layer][c.j] = w;
  else net.W[c.layer][(int64_t)c.j * net.widths[c.layer] + c.i] = w;
  if (net.sub_size == 0) st->L += dL[k];
  st->accepted += 1;
}

// Statistics of hidden layer l, one thread per sample, units in order.
__global__ void k_norm_stats(NetDev net, NormDev nd, int l) {
  const int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= net.N) return;
  const int W = net.widths[l + 1];
  const float* Z = net.Z[l];
  const float inv = 1.0f / (float)W;  // W is a power of two
  float s = 0.f;
  for (int u = 0; u < W; ++u) s += gload(&Z[(int64_t)u * net.Ns + n]);
  const float mu = s * inv;
  float v = 0.f;
  for (int u = 0; u < W; ++u) {
    const float c = gload(&Z[(int64_t)u * net.Ns + n]) - mu;
    v += c * c;
  }
  gstore(&nd.MU[l][n], mu);
  gstore(&nd.S[l][n], v * inv + net.ln_eps);
}

hipError_t launch_norm_stats(const NetDev& net, const NormDev& nd, int l, hipStream_t s) {
  hipLaunchKernelGGL(k_norm_stats, dim3((unsigned)((net.N + 255) / 256)), dim3(256), 0, s, net, nd, l);
  return hipGetLastError();
}

namespace {
template <int CM>
hipError_t launch_norm_width(const NetDev& net, const NormDev& nd, dim3 grid,
                             const mca_cand* cands, const Aux* aux, float* partial, int ntiles,
                             int k_mode, DevState* st, hipStream_t s) {
  switch (net.widths[1]) {
    case 256:
      hipLaunchKernelGGL((k_norm<CM, 256>), grid, dim3(kNThreads), 0, s, net, nd, cands, aux,
                         partial, ntiles, k_mode, st);
      break;
    case 512:
      hipLaunchKernelGGL((k_norm<CM, 512>), grid, dim3(kNThreads), 0, s, net, nd, cands, aux,
                         partial, ntiles, k_mode, st);
      break;
    case 1024:
      hipLaunchKernelGGL((k_norm<CM, 1024>), grid, dim3(kNThreads), 0, s, net, nd, cands, aux,
                         partial, ntiles, k_mode, st);
      break;
    default:
      return hipErrorInvalidValue;  // the context's validation admits no other width
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_norm(const NetDev& net, const NormDev& nd, const mca_cand* cands,
                       const Aux* aux, int K, float* partial, int ntiles, int k_mode,
                       DevState* st, const double* dL, hipStream_t s) {
  const bool commit = k_mode != -2;
  const dim3 grid((unsigned)ntiles, commit ? 1u : (unsigned)K);
  hipError_t e = (net.C <= 10)
                     ? launch_norm_width<10>(net, nd, grid, cands, aux, partial, ntiles, k_mode, st, s)
                     : launch_norm_width<kCMax>(net, nd, grid, cands, aux, partial, ntiles, k_mode, st, s);
  if (e != hipSuccess || !commit) return e;
  hipLaunchKernelGGL(k_norm_param, dim3(1), dim3(64), 0, s, net, cands, aux, k_mode, st, dL);
  return hipGetLastError();
}

}  // namespace mca
