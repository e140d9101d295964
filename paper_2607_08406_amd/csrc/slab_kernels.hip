// Evaluation and commit of mutations of a first-layer weight in a
// three-layer MLP (Sec. 2.4, the two-hidden-layer case): changing W_0[j, i] moves z_1[n, j] by de * x[n, i] for every
// sample whose input x[n, i] is nonzero; its activation change da[n] moves
// every unit m of the second hidden layer by da[n] * W_1[m, j] (the O(n_2)
// multiplications per sample the paper describes), and the logits then change
// by W_2 (phi(z_2') - phi(z_2)) for that sample.  Every activation change is
// formed by dphi() and the loss change from the logit change and the cached
// softmax (ce_change), never as a difference of two losses.
//
// Per step, k_columns lists the nonzero entries (m, W_1[m, j]) of each such
// candidate's column in increasing m (a unit with W_1[m, j] = 0 does not move;
// about half of a ternary column).  A block of k_slab owns T consecutive
// samples.  It stages their second-hidden-layer local fields ([n_2][T],
// unit-major as in HBM, rows padded to T+1 floats), the logit-layer weights
// transposed ([n_2][C]) and the tile's logits, softmax and labels in LDS, lists
// every affected (candidate, sample) pair, and scores each pair with 32 lanes:
// lane g adds the list entries g, g+32, ... in order (the next entries are
// requested while the current ones are used), then the 32 lane sums meet in a
// fixed butterfly.  The commit runs the same expressions in the same order for
// the chosen candidate, so the caches hold exactly the values that were
// scored.
#include "device_common.hpp"
#include "slab_kernels.hpp"

namespace mca {

namespace {

constexpr int kSlabThreads = 1024;
constexpr int kGroupK = 64;  // candidate slots listed at a time
constexpr int kLanesPerPair = 32;    // a half-wave scores one candidate's pairs
constexpr int kHalves = kSlabThreads / kLanesPerPair;
constexpr int kPairChunk = 2;        // pairs of one candidate scored together
constexpr int kChunk = 2;    // list entries a lane loads at once (two batches in flight)
constexpr int kStageU = 8;   // tile elements a thread loads at once

template <int CM>
struct SlabTile;
template <>
struct SlabTile<10> { static constexpr int T = 16; };
template <>
struct SlabTile<kCMax> { static constexpr int T = 12; };
constexpr int kSlabTileMax = 16;

template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xF, 0xF, true));
}
// Sum over the 32 lanes of a half-wave in one fixed order, valid in its lane
// 0: DPP within rows of 16 (lane ^ 1, ^ 2, then the mirrored partners), then
// the other row.
__device__ __forceinline__ float half_sum(float v) {
  v += dpp_mov<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);  // row_half_mirror
  v += dpp_mov<0x140>(v);  // row_mirror
  return v + __shfl_xor(v, 16, 64);
}

// Logit changes of up to kPairChunk pairs of one candidate (samples tp[p],
// activation changes dp[p] of its first-hidden-layer unit, p < np); the 32
// lanes of a half-wave share them: lane g takes the list entries g, g+32, ...
// in order, reads each entry's logit-layer weights once for all the pairs,
// and the lane sums meet in half_sum().  zt: the block's tile (row stride
// TS); w2: [n2][CM]; col: the candidate's nnz column entries (m in the low
// word, the bits of W_1[m, j] in the high word).  With STORE each lane writes
// its units' new local fields into the tile.  All 64 lanes of the wave must
// call this.
template <int CM, int ACT, int TS, bool STORE>
__device__ __forceinline__ void chunk_logit_delta(float* zt, const float* w2, const uint64_t* col,
                                                  int nnz, const int (&tp)[kPairChunk],
                                                  const float (&dp)[kPairChunk], int np,
                                                  float gamma, bool active,
                                                  float (&acc)[kPairChunk][CM]) {
  const int g = threadIdx.x & (kLanesPerPair - 1);
#pragma unroll
  for (int p = 0; p < kPairChunk; ++p)
#pragma unroll
    for (int c = 0; c < CM; ++c) acc[p][c] = 0.f;
  // The entries of the next batch are requested before the current batch is
  // used (two register sets, alternating by position in the loop, so no copy
  // waits for loads in flight); a load is issued from a clamped index and its
  // entry is skipped where it is used.
  auto fetch = [&](int e0, uint64_t (&ent)[kChunk]) {
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int e = e0 + kLanesPerPair * u;
      ent[u] = gload(&col[e < nnz ? e : 0]);
    }
  };
  auto use = [&](int e0, const uint64_t (&ent)[kChunk]) {
#pragma unroll
    for (int u = 0; u < kChunk; ++u) {
      const int e = e0 + kLanesPerPair * u;
      if (e < nnz) {
        const int m = (int)(uint32_t)ent[u];
        const float w = __uint_as_float((uint32_t)(ent[u] >> 32));
        float wr[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) wr[c] = w2[m * CM + c];
#pragma unroll
        for (int p = 0; p < kPairChunk; ++p) {
          if (p < np) {
            const float zo = zt[m * TS + tp[p]];
            const float dz = dp[p] * w;
            const float d = dphi(zo, dz, ACT, gamma);
            if (STORE) zt[m * TS + tp[p]] = zo + dz;
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[p][c] = fmaf(d, wr[c], acc[p][c]);
          }
        }
      }
    }
  };
  if (active && nnz > 0) {
    constexpr int kStride = kLanesPerPair * kChunk;
    uint64_t ea[kChunk], eb[kChunk];
    fetch(g, ea);
#pragma unroll 1
    for (int e0 = g; e0 < nnz; e0 += 2 * kStride) {
      fetch(e0 + kStride, eb);
      use(e0, ea);
      fetch(e0 + 2 * kStride, ea);
      use(e0 + kStride, eb);
    }
  }
#pragma unroll
  for (int p = 0; p < kPairChunk; ++p)
#pragma unroll
    for (int c = 0; c < CM; ++c) acc[p][c] = half_sum(acc[p][c]);
}

}  // namespace

// The nonzero entries of column j of W_1 (the candidate's unit) in increasing
// unit order, by the whole block: cols[k * n2 + e] = m | bits(W_1[m, j]) << 32,
// nnz[k] = their count.
__device__ void list_column(const NetDev& net, int j, int k, uint64_t* cols, int* nnz) {
  __shared__ int wave_n[kSlabThreads / 64];
  const int L = net.L;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n2 = net.widths[L - 1];
  const float* row = net.WT + (int64_t)j * n2;
  int base = 0;
  for (int m0 = 0; m0 < n2; m0 += kSlabThreads) {
    const int m = m0 + tid;
    const float w = (m < n2) ? gload(&row[m]) : 0.f;
    const bool nz = w != 0.f;
    const uint64_t b = __ballot(nz);
    if (lane == 0) wave_n[wave] = (int)__popcll(b);
    __syncthreads();
    int off = base;
    for (int v = 0; v < wave; ++v) off += wave_n[v];
    int tot = 0;
    for (int v = 0; v < kSlabThreads / 64; ++v) tot += wave_n[v];
    if (nz) {
      const int e = off + (int)__popcll(b & ((1ull << lane) - 1ull));
      gstore(&cols[(int64_t)k * n2 + e], (uint64_t)m | ((uint64_t)__float_as_uint(w) << 32));
    }
    base += tot;
    __syncthreads();
  }
  if (tid == 0) nnz[k] = base;
}

// Block k lists the column of candidate k when it is in layer L-3 (and valid);
// otherwise nnz[k] = 0.
__global__ __launch_bounds__(kSlabThreads) void k_columns(NetDev net_arg, const mca_cand* cands,
                                                          const Aux* aux, int k_mode,
                                                          const DevState* st, uint64_t* cols,
                                                          int* nnz) {
  const int k = (k_mode >= 0) ? k_mode : (k_mode == -1 ? st->chosen : (int)blockIdx.x);
  if (k < 0) return;
  const mca_cand c = cands[k];
  const bool take = c.layer == net_arg.L - 3 && (k_mode != -2 || aux[k].valid);
  if (!take) {
    if (threadIdx.x == 0) nnz[k] = 0;
    return;
  }
  list_column(net_arg, c.j, k, cols, nnz);
}

// The candidates of the step st->t (decoded as the proposal kernel does:
// record, new value, acceptance threshold, tile mask) and, for a valid weight
// in layer L-3, its column list: block k, candidate k.  Every thread decodes
// the candidate (the stream needs no state); thread 0 stores it.
__global__ __launch_bounds__(kSlabThreads) void k_propose_columns(
    NetDev net_arg, const DevState* st, int K, mca_cand* cands, Aux* aux, const uint64_t* fmask,
    uint64_t* cmask, uint64_t* cols, int* nnz) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = blockIdx.x;
  const uint64_t t = st->t;
  const mca_cand c = decode_candidate(net, t, (uint64_t)k);
  Aux a = prepare_candidate(net, c);
  if (threadIdx.x == 0) {
    cands[k] = c;
    a.theta = accept_theta(net.rule, net.beta, net.seed, net.tag, t, (uint64_t)k);
    aux[k] = a;
    cmask[k] = candidate_tiles(c, fmask);
  }
  if (c.layer == net.L - 3 && a.valid)
    list_column(net, c.j, k, cols, nnz);
  else if (threadIdx.x == 0)
    nnz[k] = 0;
}

// k_mode: -2 evaluate every listed candidate of layer L-3; -1 commit the
// device decision st->chosen; >= 0 commit that candidate.  A commit applies a
// candidate of layer L-3, and with `columns` also one of the last two layers
// (the column commit, as k_commit_column); others are no-ops here.  ACT is
// the net's transfer function (MCA_ACT_*), fixed at compile time.
template <int CM, int ACT>
__global__ __launch_bounds__(kSlabThreads) void k_slab(NetDev net_arg, const mca_cand* cands,
                                                       const Aux* aux, int K, const uint64_t* cols,
                                                       const int* nnz, float* partial, int nblk,
                                                       int k_mode, DevState* st,
                                                       const double* dL, int columns) {
  constexpr int T = SlabTile<CM>::T, TS = T + 1;
  __shared__ NetDev net;
  stage_net(net, net_arg);
  __shared__ float zt[kSlabMaxUnits * TS];
  __shared__ float w2[kSlabMaxUnits * CM];
  __shared__ float pdt[kGroupK * T];       // activation change of slot s at sample t
  __shared__ uint32_t pmask[kGroupK];      // slot s's samples with a change
  __shared__ uint16_t items[kGroupK * ((kSlabTileMax + kPairChunk - 1) / kPairChunk)];
  __shared__ float dlp[kGroupK * T];
  __shared__ int gk[kGroupK], gj[kGroupK], gi[kGroupK], gnnz[kGroupK];
  __shared__ float zlt[CM * kSlabTileMax];  // the tile's logits [class][sample]
  __shared__ float plt[CM * kSlabTileMax];  // their softmax
  __shared__ int yt[kSlabTileMax];
  __shared__ float gde[kGroupK];
  __shared__ int ngroup, nitems;
  __shared__ uint32_t touched;  // commit: samples of the tile whose fields changed

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = net.L, C = (CM < kCMax) ? CM : net.C;
  const int l = L - 3;  // the layer whose weights this kernel mutates
  constexpr int act = ACT;
  const float gamma = net.gamma;
  const int n2 = net.widths[L - 1];
  const int64_t Ns = net.Ns, N = net.N;
  const int64_t n0 = (int64_t)blockIdx.x * T;
  const bool commit = k_mode != -2;
  int kc = -1;
  if (commit) {
    kc = (k_mode >= 0) ? k_mode : st->chosen;
    if (kc < 0) return;  // uniform over the block
    const mca_cand cw = cands[kc];
    if (cw.layer >= L - 2) {
      // a winner in the last two layers: the column commit on the block's
      // samples (the grid covers every sample), the weight by block 0
      if (!columns) return;
      const Aux aw = aux[kc];
      if (tid < T && n0 + tid < N) column_commit(net, cw.layer, cw.j, cw.i, aw.de, n0 + tid);
      if (blockIdx.x == 0 && tid == 0) {
        const int64_t idx = (int64_t)cw.j * net.widths[cw.layer] + cw.i;
        gstore(&net.W[cw.layer][idx], aw.w_new);
        if (net.ternary) gstore(&net.codes[cw.layer][idx], (int8_t)cw.code);
        // the transposed copy of W_{L-2}, which the column lists read
        if (cw.layer == L - 2)
          gstore(&net.WT[(int64_t)cw.i * net.widths[cw.layer + 1] + cw.j], aw.w_new);
        if (net.sub_size == 0) st->L += dL[kc];
        st->accepted += 1;
      }
      return;
    }
    if (cw.layer != l) return;
  }
  float* const Z1 = net.Z[l];       // fields of the mutated unit's layer
  float* const Z2 = net.Z[l + 1];   // the next hidden layer (the tile)
  float* const ZL = net.Z[L - 1];   // logits
  const float* in = (l == 0) ? net.XT : net.Z[l - 1];
  if (tid == 0) touched = 0u;
  // The tile and the logit-layer weights go to LDS: in an evaluation first
  // (their loads are independent of the candidates, so their latency overlaps
  // the listing); in a commit only when the block has a pair to score.
  // Every load is issued from an index clamped into its array and its value
  // selected when it is stored (a load under a branch would make the merge
  // wait for every load in flight).
  auto stage = [&]() {
    for (int e0 = tid; e0 < n2 * T; e0 += kStageU * kSlabThreads) {
      float v[kStageU];
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int m = e / T, t = e - m * T;
        const bool ok = e < n2 * T && n0 + t < N;
        v[u] = gload(&Z2[ok ? (int64_t)m * Ns + n0 + t : 0]);
      }
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int m = e / T, t = e - m * T;
        if (e < n2 * T) zt[m * TS + t] = (n0 + t < N) ? v[u] : 0.f;
      }
    }
    const float* WL = net.W[L - 1];
    for (int e0 = tid; e0 < CM * n2; e0 += kStageU * kSlabThreads) {
      float v[kStageU];
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int c = e / n2, m = e - c * n2;
        const bool ok = e < CM * n2 && c < C;
        v[u] = gload(&WL[ok ? (int64_t)c * n2 + m : 0]);
      }
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int c = e / n2, m = e - c * n2;
        if (e < CM * n2) w2[m * CM + c] = (c < C) ? v[u] : 0.f;
      }
    }
  };
  // The commit reads and writes only the units of the winner's column list:
  // their rows of the tile and of the logit-layer weights.
  auto stage_listed = [&](const uint64_t* col, int cnt) {
    for (int e0 = tid; e0 < cnt * T; e0 += kStageU * kSlabThreads) {
      float v[kStageU];
      int mu[kStageU];
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int q = e / T, t = e - q * T;
        const bool ok = e < cnt * T && n0 + t < N;
        mu[u] = (int)(uint32_t)gload(&col[e < cnt * T ? q : 0]);
        v[u] = gload(&Z2[ok ? (int64_t)mu[u] * Ns + n0 + t : 0]);
      }
#pragma unroll
      for (int u = 0; u < kStageU; ++u) {
        const int e = e0 + u * kSlabThreads;
        const int q = e / T, t = e - q * T;
        if (e < cnt * T) zt[mu[u] * TS + t] = (n0 + t < N) ? v[u] : 0.f;
      }
    }
    const float* WL = net.W[L - 1];
    for (int e = tid; e < cnt * CM; e += kSlabThreads) {
      const int q = e / CM, c = e - q * CM;
      const int m = (int)(uint32_t)gload(&col[q]);
      w2[m * CM + c] = (c < C) ? gload(&WL[(int64_t)c * n2 + m]) : 0.f;
    }
  };
  // The tile's logits, softmax and labels (the loss change of a pair reads
  // the softmax and labels, a commit the logits), one value per thread.
  static_assert((2 * kCMax + 1) * kSlabTileMax <= kSlabThreads, "one value per thread");
  if (tid < (2 * CM + 1) * T) {
    const int r = tid / T, t = tid - r * T;
    const int rc = (r < CM) ? r : r - CM;  // class of a logit or softmax row
    const bool ok = n0 + t < N && (r >= 2 * CM || rc < C);
    const int64_t n = ok ? n0 + t : 0;
    const int64_t ro = (int64_t)(rc < C ? rc : 0) * Ns + n;
    const float v = (r < CM) ? gload(&ZL[ro])
                             : (r < 2 * CM ? gload(&net.prob[ro]) : __int_as_float(gload(&net.y[n])));
    if (r < CM) zlt[r * T + t] = ok ? v : 0.f;
    else if (r < 2 * CM) plt[rc * T + t] = ok ? v : 0.f;
    else yt[t] = ok ? __float_as_int(v) : 0;
  }
  // The first group's candidate fields (wave 0, lane = slot) are requested
  // before the tile, so their latency overlaps the staging.
  int f_layer = -1, f_j = 0, f_i = 0, f_valid = 0, f_nnz = 0;
  float f_de = 0.f;
  if (wave == 0) {
    // a commit names its candidate (kc < the evaluated batch; K is 0 then)
    const int kk = commit ? kc : (lane < K ? lane : K - 1);
    f_layer = cands[kk].layer;
    f_j = cands[kk].j;
    f_i = cands[kk].i;
    f_valid = aux[kk].valid;
    f_de = aux[kk].de;
    f_nnz = nnz[kk];
  }
  if (!commit) stage();

  for (int g0 = 0; g0 < (commit ? 1 : K); g0 += kGroupK) {
    // 1. the group's candidates in layer l (wave 0 lists them in order)
    if (wave == 0) {
      const int k = commit ? kc : g0 + lane;
      if (g0 > 0) {  // later groups of an evaluation (K > 64)
        const int kk = k < K ? k : K - 1;
        f_layer = cands[kk].layer;
        f_j = cands[kk].j;
        f_i = cands[kk].i;
        f_valid = aux[kk].valid;
        f_de = aux[kk].de;
        f_nnz = nnz[kk];
      }
      const bool in_l = commit ? lane == 0 : (k < K && f_layer == l && f_valid);
      const uint64_t m = __ballot(in_l);
      if (in_l) {
        const int s = (int)__popcll(m & ((1ull << lane) - 1ull));
        gk[s] = k;
        gj[s] = f_j;
        gi[s] = f_i;
        gde[s] = f_de;
        gnnz[s] = f_nnz;
      }
      if (lane == 0) ngroup = (int)__popcll(m);
    }
    __syncthreads();
    const int ng = ngroup;
    if (ng == 0) continue;
    // 2. the affected pairs: a nonzero input and a changed activation (an
    // evaluation scores the step's minibatch only; a commit moves every sample)
    const int64_t sub0 = subset_start(net, commit ? 0 : st->t);
    for (int e = tid; e < ng * T; e += kSlabThreads) {
      const int s = e / T, t = e - s * T;
      const int64_t n = n0 + t;
      dlp[s * T + t] = 0.f;
      float da = 0.f;
      if (n < N && (commit || in_subset(net, sub0, n))) {
        const float xr = gload(&in[(int64_t)gi[s] * Ns + n]);
        const float x = (l == 0) ? xr : act_fn(xr, act, gamma);
        if (x != 0.f) {
          const float zl = gload(&Z1[(int64_t)gj[s] * Ns + n]);
          const float dz = gde[s] * x;
          da = dphi(zl, dz, act, gamma);
          if (commit) gstore(&Z1[(int64_t)gj[s] * Ns + n], zl + dz);
        }
      }
      pdt[s * T + t] = da;
    }
    __syncthreads();
    // 3. the work items: each slot's changed samples in chunks of kPairChunk
    // (wave 0: lane s counts its slot's, the offsets by a prefix sum)
    if (wave == 0) {
      uint32_t pm = 0u;
      int nch = 0;
      if (lane < ng) {
        for (int t = 0; t < T; ++t)
          if (pdt[lane * T + t] != 0.f) pm |= 1u << t;
        nch = ((int)__popc(pm) + kPairChunk - 1) / kPairChunk;
        pmask[lane] = pm;
      }
      int incl = nch;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int v = __shfl_up(incl, o, 64);
        if (lane >= o) incl += v;
      }
      for (int c = 0; c < nch; ++c) items[incl - nch + c] = (uint16_t)((lane << 4) | c);
      if (lane == 63) nitems = incl;
    }
    __syncthreads();
    const int ni = nitems;
    if (commit && ni > 0) {  // uniform over the block
      stage_listed(cols + (int64_t)kc * n2, nnz[kc]);
      __syncthreads();
    }
    // 4. score: half-wave h takes items h, h + kHalves, ...; every half-wave
    // runs the same rounds (the wave shares its shuffles)
    for (int i0 = 0; i0 < ni; i0 += kHalves) {
      const int it = i0 + (tid >> 5);
      const bool active = it < ni;
      const int code = active ? items[it] : 0;
      const int s = code >> 4, ch = code & 15;
      uint32_t pm = active ? pmask[s] : 0u;
      for (int r = 0; r < kPairChunk * ch; ++r) pm &= pm - 1u;  // the earlier chunks' samples
      int tp[kPairChunk];
      float dp[kPairChunk];
      int np = 0;
#pragma unroll
      for (int p = 0; p < kPairChunk; ++p) {
        tp[p] = 0;
        dp[p] = 0.f;
        if (pm) {
          const int t = __ffs(pm) - 1;
          pm &= pm - 1u;
          tp[p] = t;
          dp[p] = pdt[s * T + t];
          np = p + 1;
        }
      }
      const int k = gk[s];
      const uint64_t* col = cols + (int64_t)k * n2;
      const int cnt = active ? gnnz[s] : 0;
      float acc[kPairChunk][CM];
      if (commit)  // the commit also writes the new fields into the tile
        chunk_logit_delta<CM, ACT, TS, true>(zt, w2, col, cnt, tp, dp, np, gamma, active, acc);
      else
        chunk_logit_delta<CM, ACT, TS, false>(zt, w2, col, cnt, tp, dp, np, gamma, active, acc);
      if (active && (tid & (kLanesPerPair - 1)) == 0) {
#pragma unroll
        for (int p = 0; p < kPairChunk; ++p) {
          if (p < np) {
            const int t = tp[p];
            const int64_t n = n0 + t;
            float pr[CM], dz[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c) {
              pr[c] = plt[c * T + t];
              dz[c] = (c < C) ? acc[p][c] : 0.f;
            }
            const int y = yt[t];
            float dzy = 0.f;
#pragma unroll
            for (int c = 0; c < CM; ++c) dzy = (c == y) ? dz[c] : dzy;
            dlp[s * T + t] = ce_change<CM>(pr, dz, C, dzy);
            if (commit) {
              float z[CM], pn[CM];
#pragma unroll
              for (int c = 0; c < CM; ++c) z[c] = (c < C) ? zlt[c * T + t] + dz[c] : 0.f;
              const float ln = softmax_ce<CM>(z, C, y, pn);
#pragma unroll
              for (int c = 0; c < CM; ++c)
                if (c < C) {
                  gstore(&ZL[(int64_t)c * Ns + n], z[c]);
                  gstore(&net.prob[(int64_t)c * Ns + n], pn[c]);
                }
              gstore(&net.ell[n], ln);
              atomicOr(&touched, 1u << t);
            }
          }
        }
      }
    }
    __syncthreads();
    // 5. each candidate's partial sum over the tile, in sample order
    if (!commit && tid < ng) {
      float v = 0.f;
      for (int t = 0; t < T; ++t) v += dlp[tid * T + t];
      partial[(int64_t)gk[tid] * nblk + blockIdx.x] = v;
    }
    __syncthreads();
  }
  if (!commit) return;
  // the tile's second-layer fields go back to HBM when any sample changed:
  // the whole rows of T samples of the listed units (the unchanged samples
  // are rewritten with the values they hold), so each unit is one contiguous
  // store instead of scattered ones; a unit off the list did not move
  if (touched != 0u) {
    const uint64_t* col = cols + (int64_t)kc * n2;
    const int cnt = nnz[kc];
    for (int e = tid; e < cnt * T; e += kSlabThreads) {
      const int q = e / T, t = e - q * T;
      const int m = (int)(uint32_t)gload(&col[q]);
      if (n0 + t < N) gstore(&Z2[(int64_t)m * Ns + n0 + t], zt[m * TS + t]);
    }
  }
  if (blockIdx.x == 0 && tid == 0) {
    const mca_cand c = cands[kc];
    const Aux a = aux[kc];
    const int64_t idx = (int64_t)c.j * net.widths[l] + c.i;
    gstore(&net.W[l][idx], a.w_new);
    if (net.ternary) gstore(&net.codes[l][idx], (int8_t)c.code);
    if (net.sub_size == 0) st->L += dL[kc];
    st->accepted += 1;
  }
}

// dst[c][r] = src[r][c]
__global__ void k_transpose(const float* src, int rows, int cols, float* dst) {
  __shared__ float tile[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8)
    if (r0 + r < rows && c0 + tx < cols) tile[r][tx] = src[(int64_t)(r0 + r) * cols + c0 + tx];
  __syncthreads();
  for (int c = ty; c < 32; c += 8)
    if (c0 + c < cols && r0 + tx < rows) dst[(int64_t)(c0 + c) * rows + r0 + tx] = tile[tx][c];
}

int slab_tile(int C) { return C <= 10 ? SlabTile<10>::T : SlabTile<kCMax>::T; }

hipError_t launch_propose_columns(const NetDev& net, const DevState* st, int K, mca_cand* cands,
                                 Aux* aux, const uint64_t* fmask, uint64_t* cmask,
                                 uint64_t* cols, int* nnz, hipStream_t s) {
  hipLaunchKernelGGL(k_propose_columns, dim3(K), dim3(kSlabThreads), 0, s, net, st, K, cands, aux,
                     fmask, cmask, cols, nnz);
  return hipGetLastError();
}

hipError_t launch_slab(const NetDev& net, const mca_cand* cands, const Aux* aux, int K,
                       uint64_t* cols, int* nnz, float* partial, int nblk, int k_mode, DevState* st,
                       const double* dL, hipStream_t s, bool listed, bool columns) {
  // the column lists of every candidate, built by an evaluation (or with the
  // proposal, `listed`); a commit follows the evaluation of its batch
  // (nothing changes W_1 in between) and reads its candidate's list from there
  if (k_mode == -2 && !listed) {
    hipLaunchKernelGGL(k_columns, dim3(K), dim3(kSlabThreads), 0, s, net, cands, aux, k_mode, st,
                       cols, nnz);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3(nblk), dim3(kSlabThreads), 0, s, net, cands, aux, K, cols,
                       nnz, partial, nblk, k_mode, st, dL, columns ? 1 : 0);
  };
  const bool small = net.C <= 10;
  if (net.act == MCA_ACT_TANH)
    small ? go(k_slab<10, MCA_ACT_TANH>) : go(k_slab<kCMax, MCA_ACT_TANH>);
  else if (net.act == MCA_ACT_RELU)
    small ? go(k_slab<10, MCA_ACT_RELU>) : go(k_slab<kCMax, MCA_ACT_RELU>);
  else
    small ? go(k_slab<10, MCA_ACT_GAUSS>) : go(k_slab<kCMax, MCA_ACT_GAUSS>);
  return hipGetLastError();
}

hipError_t launch_transpose(const float* src, int rows, int cols, float* dst, hipStream_t s) {
  hipLaunchKernelGGL(k_transpose, dim3((cols + 31) / 32, (rows + 31) / 32), dim3(256), 0, s, src,
                     rows, cols, dst);
  return hipGetLastError();
}

}  // namespace mca
