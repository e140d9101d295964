// Evaluation and commit of mutations in the deep layers of an MLP (layers
// 0..L-4, Sec. 2.1): changing W_l[j, i] moves unit j of layer l for every
// sample whose input a_{l-1}[n, i] is nonzero; its activation change da[n]
// moves every unit of layer l+1 by da[n] * W_{l+1}[:, j] (rank-1), and from
// there on every later layer changes densely.  The kernels carry the
// *changes*: dz_m = W_m dA_{m-1} for m = l+2 .. L-2, with
// dA_m = phi(z_m + dz_m) - phi(z_m) formed by dphi() from the cached field
// z_m, then the logit change dz_{L-1} = W_{L-1} dA_{L-2} and each sample's
// loss change from it and the cached softmax (ce_change).  A deep net with
// small weights changes its loss by 1e-11 per mutation; a recomputed loss
// minus the cached one would keep none of it in fp32.  The dense products are
// the dominant work and run on the matrix cores (v_mfma_f32_16x16x4f32).
//
// k_rows lists, per candidate and in increasing sample order, the samples
// whose activation changes, with their da.  A block of k_chain takes one
// candidate and 64 listed samples: it builds dA_{l+1} in an LDS tile
// ([64][256], rows padded), runs the dense layers tile to tile (4 waves, each
// 64 samples x 64 output units as 4 x 4 MFMA tiles), computes the logit
// changes and the loss change of each sample, and adds the 64 changes in
// list order.  The commit runs the same arithmetic for the chosen candidate
// and moves every cached field by its change.
//
// The hidden layers touched here must be exactly kChainUnits wide.
#include "device_common.hpp"
#include "chain_kernels.hpp"

namespace mca {

namespace {

constexpr int kRowsThreads = 1024;
constexpr int kChainThreads = 256;
constexpr int kRowStride = kChainUnits + 4;  // floats per padded LDS row
static_assert(kChainThreads == kChainUnits, "one thread per unit loads W_s[:, j]");

typedef float floatx4 __attribute__((ext_vector_type(4)));

}  // namespace

// Block k (eval) or the committed candidate: samples n with a nonzero input
// a_{l-1}[n, i] and a changed activation, in increasing n: rows[k * N + e] =
// n, rda[k * N + e] = da; cnt[k] = their number (0 unless the candidate is in
// layers 0..L-4 and valid).  A commit also stores the new z_l[n, j] of every
// sample with a nonzero input, the new weight (and code) and the state.
__global__ __launch_bounds__(kRowsThreads) void k_rows(NetDev net_arg, const mca_cand* cands,
                                                       const Aux* aux, int k_mode,
                                                       DevState* st, const double* dL, int* rows,
                                                       float* rda, int* cnt) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  __shared__ int wave_n[kRowsThreads / 64];
  const bool commit = k_mode != -2;
  const int k = commit ? ((k_mode >= 0) ? k_mode : st->chosen) : (int)blockIdx.x;
  if (k < 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const mca_cand c = cands[k];
  const int L = net.L, l = c.layer;
  if (l > L - 4 || (!commit && !aux[k].valid)) {
    if (tid == 0) cnt[k] = 0;
    return;
  }
  const int act = net.act;
  const float gamma = net.gamma;
  const float de = aux[k].de;
  const int64_t N = net.N, Ns = net.Ns;
  const float* in = (l == 0) ? net.XT : net.Z[l - 1];
  float* zrow = net.Z[l] + (int64_t)c.j * Ns;
  // an evaluation lists the step's minibatch only; a commit moves every sample
  const int64_t sub0 = subset_start(net, commit ? 0 : st->t);
  int base = 0;
  for (int64_t n0 = 0; n0 < N; n0 += kRowsThreads) {
    const int64_t n = n0 + tid;
    float da = 0.f;
    if (n < N) {
      const float xr = gload(&in[(int64_t)c.i * Ns + n]);
      const float x = (l == 0) ? xr : act_fn(xr, act, gamma);
      if (x != 0.f) {
        const float zl = gload(&zrow[n]);
        const float dz = de * x;
        da = dphi(zl, dz, act, gamma);
        if (commit) gstore(&zrow[n], zl + dz);
      }
    }
    const bool take = da != 0.f && (commit || in_subset(net, sub0, n));
    const uint64_t b = __ballot(take);
    if (lane == 0) wave_n[wave] = (int)__popcll(b);
    __syncthreads();
    int off = base, tot = 0;
    for (int v = 0; v < kRowsThreads / 64; ++v) {
      if (v < wave) off += wave_n[v];
      tot += wave_n[v];
    }
    if (take) {
      const int e = off + (int)__popcll(b & ((1ull << lane) - 1ull));
      gstore(&rows[(int64_t)k * N + e], (int)n);
      gstore(&rda[(int64_t)k * N + e], da);
    }
    base += tot;
    __syncthreads();
  }
  if (tid == 0) {
    cnt[k] = base;
    if (commit) {
      const Aux a = aux[k];
      const int64_t idx = (int64_t)c.j * net.widths[l] + c.i;
      gstore(&net.W[l][idx], a.w_new);
      if (net.ternary) gstore(&net.codes[l][idx], (int8_t)c.code);
      if (net.sub_size == 0) st->L += dL[k];
      st->accepted += 1;
    }
  }
}

// grid (ceil(N / 64), K) for an evaluation, (ceil(N / 64), 1) for a commit.
template <int CM>
__global__ __launch_bounds__(kChainThreads, 2) void k_chain(NetDev net_arg, const mca_cand* cands,
                                                         const Aux* aux, const int* rows,
                                                         const float* rda, const int* cnt,
                                                         float* partial, int nchain, int k_mode,
                                                         const DevState* st) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  // activation changes, [sample][unit], rewritten in place layer by layer
  // (one tile keeps two blocks resident per CU)
  __shared__ float ta[kChainT * kRowStride];
  __shared__ float wcol[kChainUnits];
  __shared__ int rown[kChainT];
  __shared__ float rowda[kChainT];
  __shared__ float logit[kChainT][CM];
  __shared__ float dls[kChainT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool commit = k_mode != -2;
  const int k = commit ? ((k_mode >= 0) ? k_mode : st->chosen) : (int)blockIdx.y;
  if (k < 0) return;
  const mca_cand c = cands[k];
  const int L = net.L, l = c.layer;
  if (l > L - 4) return;  // scored by another kernel
  const int tile = blockIdx.x;
  const int nrows = cnt[k];
  const int e0 = tile * kChainT;
  if (e0 >= nrows) {
    if (!commit && tid == 0) partial[(int64_t)k * nchain + tile] = 0.f;
    return;
  }
  const int C = (CM < kCMax) ? CM : net.C;
  const int act = net.act;
  const float gamma = net.gamma;
  const int64_t N = net.N, Ns = net.Ns;
  const int s = l + 1;  // the layer the rank-1 update reaches

  // 1. the tile's samples and the column W_s[:, j]
  if (tid < kChainT) {
    const int e = e0 + tid;
    rown[tid] = (e < nrows) ? gload(&rows[(int64_t)k * N + e]) : -1;
    rowda[tid] = (e < nrows) ? gload(&rda[(int64_t)k * N + e]) : 0.f;
  }
  {
    const float* Ws = net.W[s];
    wcol[tid] = gload(&Ws[(int64_t)tid * kChainUnits + c.j]);  // kChainThreads == kChainUnits
  }
  __syncthreads();
  // 2. dA_s = phi(z_s + da W_s[:, j]) - phi(z_s) into the tile (unit-major
  // source: consecutive threads take consecutive rows of one unit)
  {
    float* Zs = net.Z[s];
    for (int e = tid; e < kChainT * kChainUnits; e += kChainThreads) {
      const int r = e & (kChainT - 1), u = e / kChainT;
      const int n = rown[r];
      float v = 0.f;
      if (n >= 0) {
        const float z = gload(&Zs[(int64_t)u * Ns + n]);
        const float dz = rowda[r] * wcol[u];
        v = dphi(z, dz, act, gamma);
        if (commit) gstore(&Zs[(int64_t)u * Ns + n], z + dz);
      }
      ta[r * kRowStride + u] = v;
    }
  }
  __syncthreads();
  // 3. dense layers m = s+1 .. L-2: dz = tile W_m^T, then the tile becomes
  // phi(z_m + dz) - phi(z_m); every wave has read the whole tile before any
  // writes its new values
  float* const tin = ta;
  const int q = lane >> 4, li = lane & 15;
  // the samples of this lane's output rows 16 sb + 4 q + v (row 0 for padding
  // rows: their changes are zero)
  int nrow[4][4];
#pragma unroll
  for (int sb = 0; sb < 4; ++sb)
#pragma unroll
    for (int v = 0; v < 4; ++v) nrow[sb][v] = rown[16 * sb + 4 * q + v];
  // every row of the tile holds the next sample after the one before
  const bool rows_dense = rown[kChainT - 1] == rown[0] + kChainT - 1 && (rown[0] & 3) == 0;
  for (int m = s + 1; m <= L - 2; ++m) {
    const float* Wm = net.W[m];
    floatx4 acc[4][4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) acc[sb][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
    // k is split in blocks of 16: lane group q holds k = 16 kb + 4 q + t for
    // t = 0..3, used by the four MFMAs of the block in turn
    floatx4 bcur[4], bnext[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb)
      bcur[cb] = gload(reinterpret_cast<const floatx4*>(
          &Wm[(int64_t)(64 * wave + 16 * cb + li) * kChainUnits + 4 * q]));
    for (int kb = 0; kb < kChainUnits / 16; ++kb) {
      if (kb + 1 < kChainUnits / 16) {
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
          bnext[cb] = gload(reinterpret_cast<const floatx4*>(
              &Wm[(int64_t)(64 * wave + 16 * cb + li) * kChainUnits + 16 * (kb + 1) + 4 * q]));
      }
      floatx4 a4[4];
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
        a4[sb] = *reinterpret_cast<const floatx4*>(&tin[(16 * sb + li) * kRowStride + 16 * kb + 4 * q]);
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
          for (int cb = 0; cb < 4; ++cb)
            acc[sb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[sb][t], bcur[cb][t],
                                                               acc[sb][cb], 0, 0, 0);
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) bcur[cb] = bnext[cb];
    }
    // D layout: lane (q, li), element v -> row 16 sb + 4 q + v, unit 64 w + 16 cb + li;
    // the cached fields of those elements, all requested before any is used.
    // A lane's four rows v = 0..3 are four consecutive samples whenever the
    // tile lists every sample (a candidate past the first layer): one 16-byte
    // load each then (16-byte aligned: the tile starts at a multiple of 64).
    float* Zm = net.Z[m];
    float zc[4][4][4];
    if (rows_dense) {
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) {
          const int u = 64 * wave + 16 * cb + li;
          const floatx4 z4 = gload(reinterpret_cast<const floatx4*>(&Zm[(int64_t)u * Ns + nrow[sb][0]]));
#pragma unroll
          for (int v = 0; v < 4; ++v) zc[sb][cb][v] = z4[v];
        }
    } else {
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int u = 64 * wave + 16 * cb + li, nr = nrow[sb][v];
            zc[sb][cb][v] = gload(&Zm[(int64_t)u * Ns + (nr >= 0 ? nr : 0)]);
          }
    }
    __syncthreads();
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
#pragma unroll
      for (int cb = 0; cb < 4; ++cb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = 16 * sb + 4 * q + v, u = 64 * wave + 16 * cb + li;
          const float dz = acc[sb][cb][v];
          const float z = zc[sb][cb][v];
          if (commit && nrow[sb][v] >= 0) gstore(&Zm[(int64_t)u * Ns + nrow[sb][v]], z + dz);
          tin[r * kRowStride + u] = dphi(z, dz, act, gamma);
        }
    __syncthreads();
  }
  // 4. logit changes dz_{L-1} = W_{L-1} dA_{L-2}: thread (r, cq) takes classes cq, cq+4, ...
  {
    const float* WL = net.W[L - 1];
    const int r = tid >> 2, cq = tid & 3;
#pragma unroll
    for (int cc = 0; cc < (CM + 3) / 4; ++cc) {
      const int cl = cq + 4 * cc;
      if (cl < C) {
        float a = 0.f;
        for (int u = 0; u < kChainUnits; ++u)
          a = fmaf(tin[r * kRowStride + u], gload(&WL[(int64_t)cl * kChainUnits + u]), a);
        logit[r][cl] = a;
      }
    }
  }
  __syncthreads();
  // 5. per-sample loss change from the logit change and the cached softmax;
  // the tile's sum in list order
  if (tid < kChainT) {
    const int n = rown[tid];
    float d = 0.f;
    if (n >= 0) {
      const int y = gload(&net.y[n]);
      float dz[CM], p[CM], dzy = 0.f;
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) {
        dz[cc] = (cc < C) ? logit[tid][cc] : 0.f;
        p[cc] = (cc < C) ? gload(&net.prob[(int64_t)cc * Ns + n]) : 0.f;
        dzy = (cc == y) ? dz[cc] : dzy;
      }
      d = ce_change<CM>(p, dz, C, dzy);
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
    for (int r = 0; r < kChainT; ++r) v += dls[r];
    partial[(int64_t)k * nchain + tile] = v;
  }
}

hipError_t launch_chain(const NetDev& net, const mca_cand* cands, const Aux* aux, int K,
                        int* rows, float* rda, int* cnt, float* partial, int nchain, int k_mode,
                        DevState* st, const double* dL, hipStream_t s) {
  const bool commit = k_mode != -2;
  hipLaunchKernelGGL(k_rows, dim3(commit ? 1 : K), dim3(kRowsThreads), 0, s, net, cands, aux,
                     k_mode, st, dL, rows, rda, cnt);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid((unsigned)nchain, commit ? 1u : (unsigned)K);
  if (net.C <= 10)
    hipLaunchKernelGGL(k_chain<10>, grid, dim3(kChainThreads), 0, s, net, cands, aux, rows, rda,
                       cnt, partial, nchain, k_mode, st);
  else
    hipLaunchKernelGGL(k_chain<kCMax>, grid, dim3(kChainThreads), 0, s, net, cands, aux, rows,
                       rda, cnt, partial, nchain, k_mode, st);
  return hipGetLastError();
}

}  // namespace mca
