// Channel mutation (Sec. 2.3): one weight per layer on a path from input unit
// u_0 to class u_L changes at once (re-drawn with the He amplitude of its
// fan-in, or set to zero).  From the cached local fields the change is:
//  - first layer: column u_1 of the field moves by de_0 * x[:, u_0];
//  - every later layer m: its field moves by W_m times the change of its
//    input (rank-1 through column W_m[:, u_1] for m = 1, a dense product
//    after that) plus the path weight's own change, de_m times the new
//    activation of the input unit u_m, at unit u_{m+1}
//    (W'_m a' - W_m a = W_m (a' - a) + (w'_m - w_m) a'[u_m]);
//  - the logits' change gives each sample's loss change with the cached
//    softmax (ce_change).
// Every sample can change (the later path weights reach every sample whose
// activation at the path unit is non-zero), so a block takes T consecutive
// samples of one channel, keeps their activation changes in an LDS tile
// [T][W + 4] (T = 16384 / W: 64, 32 or 16 rows, 66 KB), runs the dense layers
// on the matrix cores (v_mfma_f32_16x16x4f32, four waves of W / 4 output
// units each), and sums its T loss changes in row order.  The commit runs the
// same arithmetic for the chosen channel and moves every cached field by its
// change; a second kernel then writes the path's weights.
#include "device_common.hpp"
#include "channel_kernels.hpp"

namespace mca {

namespace {

constexpr int kChThreads = 256;
typedef float floatx4 __attribute__((ext_vector_type(4)));

// The channel of draw (t, k): 2L + 1 words of the Philox blocks at counters
// (t, k, 2 + b, 0), four words per block, in order.
__device__ mca_channel draw_channel(const NetDev& net, uint64_t t, uint64_t k) {
  mca_channel ch;
  const int L = net.L, nw = 2 * L + 1;
  for (int q = 0; q <= MCA_MAX_LAYERS; ++q) ch.units[q] = 0;
  for (int m = 0; m < MCA_MAX_LAYERS; ++m) ch.w_new[m] = 0.0f;
  for (int q0 = 0; q0 < nw; q0 += 4) {
    const Words w = philox4x64_10(t, k, 2 + (uint64_t)(q0 / 4), 0, net.seed, net.tag);
    const uint64_t ws[4] = {w.w0, w.w1, w.w2, w.w3};
    for (int e = 0; e < 4 && q0 + e < nw; ++e) {
      const int q = q0 + e;
      if (q <= L) {
        ch.units[q] = (int32_t)__umul64hi(ws[e], (uint64_t)net.widths[q]);
      } else if (net.mutation == MCA_MUTATE_CHANNEL_REDRAW) {
        const int m = q - L - 1;
        const float r = (float)(uint32_t)(ws[e] >> 40) * 0x1p-23f - 1.0f;
        ch.w_new[m] = net.chan_amp[m] * r;
      }
    }
  }
  return ch;
}

// Acceptance data of a channel: the weight bound (every re-drawn weight must
// stay inside it, Eq. 1) and the selection threshold.
__device__ Aux channel_aux(const NetDev& net, const mca_channel& ch) {
  Aux a;
  a.w_old = a.w_new = a.de = 0.0f;
  int ok = 1;
  for (int m = 0; m < net.L; ++m) ok &= !(net.bound > 0.f && fabsf(ch.w_new[m]) >= net.bound);
  a.valid = ok;
  a.theta = 0.0;
  return a;
}

__device__ __forceinline__ mca_cand placeholder() {
  mca_cand c;
  c.flat = 0;
  c.layer = 0;
  c.j = c.i = 0;
  c.d = 0.0f;
  c.code = 0;
  c.flags = 0;
  return c;
}

}  // namespace

__global__ void k_channel_propose(NetDev net_arg, uint64_t t_host, int use_dev_t,
                                  const DevState* st, int K, mca_channel* chans, mca_cand* cands,
                                  Aux* aux) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const uint64_t t = use_dev_t ? st->t : t_host;
  const mca_channel ch = draw_channel(net, t, (uint64_t)k);
  chans[k] = ch;
  Aux a = channel_aux(net, ch);
  a.theta = accept_theta(net.rule, net.beta, net.seed, net.tag, t, (uint64_t)k);
  aux[k] = a;
  cands[k] = placeholder();
}

__global__ void k_channel_prepare(NetDev net_arg, const mca_channel* chans, int K,
                                  mca_cand* cands, Aux* aux) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  aux[k] = channel_aux(net, chans[k]);
  cands[k] = placeholder();
}

// grid (ntiles, K) for an evaluation, (ntiles, 1) for a commit.
template <int CM, int W>
__global__ __launch_bounds__(kChThreads, (W >= 1024) ? 1 : 2) void k_channel(
    NetDev net_arg, const mca_channel* chans, const Aux* aux, float* partial, int ntiles,
    int k_mode, DevState* st) {
  constexpr int T = 16384 / W;        // samples of the block
  constexpr int SB = T / 16;          // 16-row blocks of the tile
  constexpr int UW = W / 4;           // output units per wave
  constexpr int CB = UW / 16;         // 16-unit blocks per wave
  constexpr int RS = W + 4;           // floats per padded LDS row
  constexpr int TPR = kChThreads / T; // threads per row for the logits
  static_assert(SB * CB == 16, "sixteen accumulator tiles per wave");
  __shared__ NetDev net;
  stage_net(net, net_arg);
  // activation changes [sample][unit], rewritten in place layer by layer
  __shared__ __attribute__((aligned(16))) float ta[T * RS];
  __shared__ float wcol[W];
  __shared__ float apath[2][T];  // new activation of the path unit feeding the next layer
  __shared__ float da0[T];       // activation change of the first layer's path unit
  __shared__ float logit[T][CM];
  __shared__ float dls[T];
  __shared__ int units[MCA_MAX_LAYERS + 1];
  __shared__ float de[MCA_MAX_LAYERS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool commit = k_mode != -2;
  const int k = commit ? ((k_mode >= 0) ? k_mode : st->chosen) : (int)blockIdx.y;
  if (k < 0) return;
  const int tile = blockIdx.x;
  if (!commit && !aux[k].valid) {  // rejected unevaluated: selection gives +inf
    if (tid == 0) partial[(int64_t)k * ntiles + tile] = 0.f;
    return;
  }
  const int L = net.L;
  const int C = (CM < kCMax) ? CM : net.C;
  const int act = net.act;
  const float gamma = net.gamma;
  const int64_t N = net.N, Ns = net.Ns;
  const int64_t n0 = (int64_t)tile * T;

  // 0. the path and the increments fl32(w' - w) of its weights (committed
  // weights: a commit writes the new ones only after this kernel)
  if (tid <= L) units[tid] = chans[k].units[tid];
  if (tid < T) apath[0][tid] = apath[1][tid] = 0.f;
  __syncthreads();
  if (tid < L) {
    const float wo = net.W[tid][(int64_t)units[tid + 1] * net.widths[tid] + units[tid]];
    de[tid] = chans[k].w_new[tid] - wo;
  }
  __syncthreads();

  // 1. the first field's path column
  if (tid < T) {
    const int64_t n = n0 + tid;
    float d = 0.f, ap = 0.f;
    if (n < N) {
      const float x = gload(&net.XT[(int64_t)units[0] * Ns + n]);
      float* zp = &net.Z[0][(int64_t)units[1] * Ns + n];
      const float z = gload(zp);
      const float dz = de[0] * x;
      if (L > 1) {
        d = dphi(z, dz, act, gamma);
        ap = act_fn(z + dz, act, gamma);
        if (commit) gstore(zp, z + dz);
      } else {
        d = dz;  // a one-layer net: the field is a logit (moved at step 5)
      }
    }
    da0[tid] = d;
    apath[0][tid] = ap;
  }
  // 2. the second layer: rank-1 through W_1[:, u_1] plus the path weight's change
  int cur = 0;  // apath buffer of the layer feeding the next product
  if (L >= 2) {
    const int n_out = net.widths[2];
    for (int u = tid; u < n_out; u += kChThreads)
      wcol[u] = gload(&net.W[1][(int64_t)u * net.widths[1] + units[1]]);
    __syncthreads();
    if (L >= 3) {
      const int j2 = units[2];
      float* Z1 = net.Z[1];
      for (int e = tid; e < T * W; e += kChThreads) {
        const int r = e % T, u = e / T;
        const int64_t n = n0 + r;
        float v = 0.f;
        if (n < N) {
          float dz = da0[r] * wcol[u];
          if (u == j2) dz = fmaf(de[1], apath[0][r], dz);
          const float z = gload(&Z1[(int64_t)u * Ns + n]);
          v = dphi(z, dz, act, gamma);
          if (u == j2) apath[1][r] = act_fn(z + dz, act, gamma);
          if (commit) gstore(&Z1[(int64_t)u * Ns + n], z + dz);
        }
        ta[r * RS + u] = v;
      }
      cur = 1;
    }
    __syncthreads();
  }
  // 3. dense layers m = 2 .. L-2: dz = tile W_m^T plus the path change at
  // u_{m+1}; the tile becomes phi(z_m + dz) - phi(z_m) once every wave has
  // read it
  const int q = lane >> 4, li = lane & 15;
  for (int m = 2; m <= L - 2; ++m) {
    const float* Wm = net.W[m];
    const int jn = units[m + 1];
    floatx4 acc[SB][CB];
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) acc[sb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    // k in blocks of 16: lane group q holds k = 16 kb + 4 q + t, t = 0..3,
    // for the four MFMAs of the block in turn
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
    // D layout: lane (q, li), element v -> row 16 sb + 4 q + v, unit
    // UW w + 16 cb + li.  A lane's four rows are four consecutive samples:
    // one 16-byte load of the cached fields each (the tile starts at a
    // multiple of 16 samples; rows past N read the padding and are unused).
    float* Zm = net.Z[m];
    floatx4 zc[SB][CB];
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        zc[sb][cb] = gload(reinterpret_cast<const floatx4*>(
            &Zm[(int64_t)(UW * wave + 16 * cb + li) * Ns + n0 + 16 * sb + 4 * q]));
    __syncthreads();
#pragma unroll
    for (int sb = 0; sb < SB; ++sb)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = 16 * sb + 4 * q + v, u = UW * wave + 16 * cb + li;
          const int64_t n = n0 + r;
          float out = 0.f;
          if (n < N) {
            float dz = acc[sb][cb][v];
            if (u == jn) dz = fmaf(de[m], apath[cur][r], dz);
            const float z = zc[sb][cb][v];
            out = dphi(z, dz, act, gamma);
            if (u == jn) apath[cur ^ 1][r] = act_fn(z + dz, act, gamma);
            if (commit) gstore(&Zm[(int64_t)u * Ns + n], z + dz);
          }
          ta[r * RS + u] = out;
        }
    __syncthreads();
    cur ^= 1;
  }
  // 4. logit changes: a dense product of the last hidden layer's change plus
  // the path change at class u_L (L >= 3); the rank-1 term plus the path
  // change (L = 2); the one moved logit (L = 1)
  {
    const int r = tid / TPR, cq = tid % TPR;
    const int cls = units[L];
#pragma unroll
    for (int c0 = 0; c0 < CM; c0 += TPR) {
      const int c = c0 + cq;
      if (c < C) {
        float a = 0.f;
        if (L >= 3) {
          const float* WL = net.W[L - 1];
          for (int u = 0; u < W; ++u) a = fmaf(ta[r * RS + u], gload(&WL[(int64_t)c * W + u]), a);
          if (c == cls) a = fmaf(de[L - 1], apath[cur][r], a);
        } else if (L == 2) {
          a = da0[r] * wcol[c];
          if (c == cls) a = fmaf(de[1], apath[0][r], a);
        } else {
          a = (c == cls) ? da0[r] : 0.f;
        }
        logit[r][c] = a;
      }
    }
  }
  __syncthreads();
  // 5. per-sample loss change from the logit change and the cached softmax;
  // the tile's sum in row order
  if (tid < T) {
    const int64_t n = n0 + tid;
    float d = 0.f;
    if (n < N) {
      const int y = gload(&net.y[n]);
      float dz[CM], p[CM], dzy = 0.f;
#pragma unroll
      for (int c = 0; c < CM; ++c) {
        dz[c] = (c < C) ? logit[tid][c] : 0.f;
        p[c] = (c < C) ? gload(&net.prob[(int64_t)c * Ns + n]) : 0.f;
        dzy = (c == y) ? dz[c] : dzy;
      }
      d = ce_change<CM>(p, dz, C, dzy);
      if (commit) {
        float* ZL = net.Z[L - 1];
        float z[CM], pn[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) z[c] = (c < C) ? gload(&ZL[(int64_t)c * Ns + n]) + dz[c] : 0.f;
        const float ln = softmax_ce<CM>(z, C, y, pn);
#pragma unroll
        for (int c = 0; c < CM; ++c)
          if (c < C) {
            gstore(&ZL[(int64_t)c * Ns + n], z[c]);
            gstore(&net.prob[(int64_t)c * Ns + n], pn[c]);
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

// After the field commit: the path's new weights (and the transposed copy of
// W_{L-2} where one is kept), the committed loss and the count.
__global__ void k_channel_weights(NetDev net, const mca_channel* chans, int k_mode, DevState* st,
                                  const double* dL) {
  const int k = (k_mode >= 0) ? k_mode : st->chosen;
  if (k < 0) return;
  const int m = threadIdx.x;
  if (m < net.L) {
    const int j = chans[k].units[m + 1], i = chans[k].units[m];
    const float w = chans[k].w_new[m];
    net.W[m][(int64_t)j * net.widths[m] + i] = w;
    if (net.WT != nullptr && m == net.L - 2) net.WT[(int64_t)i * net.widths[m + 1] + j] = w;
  }
  if (m == 0) {
    st->L += dL[k];
    st->accepted += 1;
  }
}

hipError_t launch_channel_propose(const NetDev& net, uint64_t t, bool use_dev_t,
                                  const DevState* st, int K, mca_channel* ch, mca_cand* cands,
                                  Aux* aux, hipStream_t s) {
  hipLaunchKernelGGL(k_channel_propose, dim3((K + 63) / 64), dim3(64), 0, s, net, t,
                     use_dev_t ? 1 : 0, st, K, ch, cands, aux);
  return hipGetLastError();
}

hipError_t launch_channel_prepare(const NetDev& net, const mca_channel* ch, int K,
                                  mca_cand* cands, Aux* aux, hipStream_t s) {
  hipLaunchKernelGGL(k_channel_prepare, dim3((K + 63) / 64), dim3(64), 0, s, net, ch, K, cands,
                     aux);
  return hipGetLastError();
}

namespace {
template <int CM>
hipError_t launch_width(const NetDev& net, dim3 grid, const mca_channel* ch, const Aux* aux,
                        float* partial, int ntiles, int k_mode, DevState* st, hipStream_t s) {
  switch (net.widths[1]) {
    case 256:
      hipLaunchKernelGGL((k_channel<CM, 256>), grid, dim3(kChThreads), 0, s, net, ch, aux,
                         partial, ntiles, k_mode, st);
      break;
    case 512:
      hipLaunchKernelGGL((k_channel<CM, 512>), grid, dim3(kChThreads), 0, s, net, ch, aux,
                         partial, ntiles, k_mode, st);
      break;
    case 1024:
      hipLaunchKernelGGL((k_channel<CM, 1024>), grid, dim3(kChThreads), 0, s, net, ch, aux,
                         partial, ntiles, k_mode, st);
      break;
    default:
      return hipErrorInvalidValue;  // the context's validation admits no other width
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_channel(const NetDev& net, const mca_channel* ch, const Aux* aux, int K,
                          float* partial, int ntiles, int k_mode, DevState* st,
                          const double* dL, hipStream_t s) {
  const bool commit = k_mode != -2;
  const dim3 grid((unsigned)ntiles, commit ? 1u : (unsigned)K);
  hipError_t e = (net.C <= 10)
                     ? launch_width<10>(net, grid, ch, aux, partial, ntiles, k_mode, st, s)
                     : launch_width<kCMax>(net, grid, ch, aux, partial, ntiles, k_mode, st, s);
  if (e != hipSuccess || !commit) return e;
  hipLaunchKernelGGL(k_channel_weights, dim3(1), dim3(64), 0, s, net, ch, k_mode, st, dL);
  return hipGetLastError();
}

}  // namespace mca
