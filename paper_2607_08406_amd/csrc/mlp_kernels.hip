// HIP kernels (gfx950) for the MLP hot path of MCA: candidate stream,
// incremental evaluation, selection, commit, and the full forward pass that
// fills the caches.
//
// Incremental evaluation (Sec. 2.4): a change of W_l[j, i] moves only row j of
// the unit-major cache Z_l, by de * a_{l-1}[i, n] for every sample n; if layer
// l is the output layer that is a logit row, otherwise the changed activation
// da[n] = phi(z'[n]) - phi(z[n]) moves the next layer's local fields by the
// rank-1 term da[n] * W_{l+1}[:, j].  Samples whose input a_{l-1}[i, n] is zero
// (about 81 % of an image column) are skipped: nothing changes for them.  The
// loss change is dL = (1/N) sum_n dl_n over the changed samples only, each
// dl_n formed from the sample's logit change and the cached softmax of its
// logits (difference form: no difference of two losses near 2.3).
#include <type_traits>

#include "device_common.hpp"
#include "mlp_kernels.hpp"
#include "norm_kernels.hpp"

namespace mca {

// ---------------------------------------------------------------------------
// candidate stream
// ---------------------------------------------------------------------------

__global__ void k_propose(NetDev net_arg, uint64_t t_host, int use_dev_t, const DevState* st,
                          int K, mca_cand* cands, Aux* aux, const uint64_t* fmask,
                          uint64_t* cmask) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const uint64_t t = use_dev_t ? st->t : t_host;
  const mca_cand c = decode_candidate(net, t, (uint64_t)k);
  cands[k] = c;
  Aux a = prepare_candidate(net, c);
  a.theta = accept_theta(net.rule, net.beta, net.seed, net.tag, t, (uint64_t)k);
  aux[k] = a;
  cmask[k] = candidate_tiles(c, fmask);
}

__global__ void k_prepare(NetDev net_arg, const mca_cand* cands, int K, Aux* aux,
                          const uint64_t* fmask, uint64_t* cmask) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k >= K) return;
  const mca_cand c = cands[k];
  aux[k] = prepare_candidate(net, c);
  cmask[k] = candidate_tiles(c, fmask);
}

// ---------------------------------------------------------------------------
// per-sample incremental update for a mutation in one of the last two layers
// ---------------------------------------------------------------------------

// Batched scoring of the candidates whose weight is in the last two layers
// (a mutated hidden unit of layer L-2 moves the logits by a rank-1 update; a
// logit-layer weight moves one logit), against the committed state.
// The samples are cut into tiles of kEvT = 256.  Each tile is shared out to
// bpt blocks (as many as the GPU holds at once, over the tiles): a block
// loads its tile's logits, per-sample losses and labels into LDS once, and
// each of its waves then walks its own candidates of the tile (wave v of the
// tile's waves takes candidates v, v + waves, ...) with no further block
// barrier.  Per candidate, one wave:
//  - lands the input of the mutated weight and, for a hidden unit, its local
//    field over the tile (lane l holds samples 4l .. 4l+3, one 16-byte load
//    per row), requested three candidates earlier;
//  (the block's tile holds each sample's softmax and label: the loss change
//    of a pair is formed from its logit change, pair_change)
//  - lists the samples whose input is non-zero (the others cannot change:
//    about 81 % of an image column is zero) in sample order, in the wave's
//    own LDS list, with their operands;
//  - scores the list 64 pairs at a time with the pair expressions of the step
//    loop, lane l adding pairs l, l+64, l+128, l+192 in that order, then one
//    butterfly; the sum is the tile's partial sum partial[k * ntiles + tile],
//    which the selection kernel adds over the tiles in fp64.
// The sums depend on the candidate and the tile only, not on the grid.  Every
// row load is issued unconditionally from an address inside its array (a
// candidate that is not scored here reads row 0; a sample group past the
// padded rows reads the tile's first group) and the three row sets change
// roles by position in an unrolled loop: a load under a branch, or a copy of
// registers still being loaded, would make the wave wait for every load in
// flight.
constexpr int kEvT = 256;                // samples per tile (four per lane)
constexpr int kEvWaves = 4;              // waves per block
constexpr int kEvThreads = 64 * kEvWaves;
static_assert(kEvT == 256, "lane l holds samples 4l .. 4l+3 of a tile");

// The caches the batched evaluation reads, resolved on the host.
struct EvArgs {
  const float* in_hid;   // input rows of layer L-2: XT (L = 2) or Z[L-3]
  const float* in_log;   // input rows of layer L-1: XT (L = 1) or Z[L-2]
  const float* z_hid;    // local fields of layer L-2 (L = 1: the logits, never used)
  const float* p_log;    // softmax of the logits, [C][Ns]
  const float* w_log;    // W[L-1], [C][n_{L-1}]
  const int32_t* y;      // [Ns]
  const mca_cand* cands;
  const Aux* aux;
  const uint64_t* cmask;  // per candidate: bit b set when tile b can change
  float* partial;
  const DevState* st;     // the step whose minibatch is scored (st->t)
  int64_t sub_size, sub_period;
  int64_t N, Ns;
  int L, C, act, nh, K, ntiles, bpt;  // bpt: blocks per tile
  float gamma;
};

// One candidate's rows over the tile as loaded: lane l holds samples
// 4l .. 4l+3 of the input and of the local field, and lane c < C the
// logit-layer weight W[L-1][c][j].
struct EvRows {
  float4 a4, z4;
  float wc;
};

template <int CM>
__global__ __launch_bounds__(kEvThreads) __attribute__((amdgpu_waves_per_eu(CM <= 10 ? 5 : 1))) void k_eval_tiles(EvArgs a) {
  constexpr int kRows = CM + 1;                            // softmax rows, labels
  __shared__ float pl_lds[CM * kEvT];                      // softmax, [class][sample]
  __shared__ int y_lds[kEvT];
  __shared__ float wcol_lds[kEvWaves][CM];                 // logit-layer column (one-hot for a logit weight)
  __shared__ uint16_t code_lds[kEvWaves][kEvT];            // pair e: its sample in the tile
  __shared__ float ain_lds[kEvWaves][kEvT];                // pair e: input of the mutated weight
  __shared__ float zh_lds[kEvWaves][kEvT];                 // pair e: local field of a mutated hidden unit
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int C = (CM < kCMax) ? CM : a.C, L = a.L;
  const int act = a.act;
  const float gamma = a.gamma;
  const int64_t Ns = a.Ns, N = a.N;
  const int ntiles = a.ntiles, K = a.K, bpt = a.bpt;
  const int wpt = bpt * kEvWaves;  // waves per tile
  const int nslots = ntiles * bpt;
  // the minibatch window of the step being scored (every sample without one)
  NetDev sub{};
  sub.N = N;
  sub.sub_size = a.sub_size;
  sub.sub_period = a.sub_period;
  const int64_t sub0 = subset_start(sub, a.sub_size ? a.st->t : 0);
  uint16_t* const code = code_lds[wave];
  float* const ainl = ain_lds[wave];
  float* const zhl = zh_lds[wave];
  float* const wcol = wcol_lds[wave];

  for (int slot = (int)blockIdx.x; slot < nslots; slot += (int)gridDim.x) {
    const int b = slot / bpt;
    const int64_t t0 = (int64_t)b * kEvT;
    const int64_t sl = t0 + 4 * lane;              // the lane's first sample
    const int64_t s0 = sl < Ns ? sl : t0;          // ... clamped into the rows
    // this wave's candidates of the tile: k = kw + m * wpt
    const int kw = (slot % bpt) * kEvWaves + wave;
    const int nu = kw < K ? (K - 1 - kw) / wpt + 1 : 0;
    const float* const ih = a.in_hid + s0;
    const float* const il = a.in_log + s0;
    const float* const zh = a.z_hid + s0;
    const float* const wl = a.w_log + (int64_t)(lane < C ? lane : 0) * a.nh;
    __syncthreads();  // the last slot's pairs are done with the tile

    // One pass over up to 64 of the wave's candidates: lane q holds candidate
    // pass + q.  The first pass (every wave makes it) also brings in the
    // tile: its rows are requested after the candidates' fields, so both
    // arrive within one memory latency, and land in LDS before the first
    // candidates' rows are requested; the block barrier comes after those.
    auto run_pass = [&](int pass, auto first_pass) {
      constexpr bool kFirst = decltype(first_pass)::value;
      const int n = nu - pass < 64 ? nu - pass : 64;
      const int qk = lane < n ? lane : (n > 0 ? n - 1 : 0);
      int k = kw + (pass + qk) * wpt;
      k = k < K ? k : K - 1;  // read from a clamped index: no load under a branch
      const int layer0 = a.cands[k].layer, j0 = a.cands[k].j, i0 = a.cands[k].i;
      const int valid = a.aux[k].valid;
      const float de0 = a.aux[k].de;
      const uint64_t tmask = a.cmask[k];
      constexpr int kRowsPer = (kRows + kEvWaves - 1) / kEvWaves;
      float4 r4[kRowsPer];
      if (kFirst) {
#pragma unroll
        for (int u = 0; u < kRowsPer; ++u) {
          const int r = wave + kEvWaves * u;  // row r: softmax r < C, then labels
          const float* row = (r < C) ? a.p_log + (int64_t)r * Ns : (const float*)a.y;
          r4[u] = *(const float4*)&row[s0];
        }
      }
      // scored here: the weight is in the last two layers and within the
      // bound (its partial sum is written); live: the tile can change too
      // (a first-layer weight whose feature is zero over the tile cannot)
      const bool scored = lane < n && layer0 >= L - 2 && valid != 0;
      const bool live = scored && ((tmask >> b) & 1ull);
      const uint64_t livem = __ballot(live);
      const int nl = (int)__popcll(livem);
      // the live candidates move to lanes 0 .. nl-1, in order (the others
      // push to lane 63, which is live only when all are)
      const int dst = live ? (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(livem >> 32),
                                                             __builtin_amdgcn_mbcnt_lo((uint32_t)livem, 0u))
                           : 63;
      auto perm = [&](int v) { return __builtin_amdgcn_ds_permute(dst * 4, v); };
      const int layer = perm(layer0), j = perm(j0), i = perm(i0), qo = perm(lane);
      const float de = __int_as_float(perm(__float_as_int(de0)));
      // bit q: lane q holds a live candidate; a hidden-unit weight; one
      // taking the raw input
      const uint64_t okm = __ballot(lane < nl);
      const uint64_t hm = __ballot(layer == L - 2) & okm;
      const uint64_t rawm = __ballot(layer == 0);
      const int64_t io = (int64_t)i * Ns, jo = (int64_t)j * Ns;
      if (kFirst) {
#pragma unroll
        for (int u = 0; u < kRowsPer; ++u) {
          const int r = wave + kEvWaves * u;
          if (r < kRows) {
            float* dst = (r < CM) ? &pl_lds[r * kEvT] : (float*)y_lds;
            const bool keep = r >= CM || r < C;  // softmax rows past C stay zero
            const float4 v = r4[u];
            float4 w;
            w.x = (keep && sl + 0 < N) ? v.x : 0.f;
            w.y = (keep && sl + 1 < N) ? v.y : 0.f;
            w.z = (keep && sl + 2 < N) ? v.z : 0.f;
            w.w = (keep && sl + 3 < N) ? v.w : 0.f;
            *(float4*)&dst[4 * lane] = w;
          }
        }
      }
      // row offsets of candidate q, zero for one not scored here (and past
      // the pass); hidden-unit rows come from the hidden layer's arrays
      const int64_t io_s = ((okm >> lane) & 1ull) ? io : 0;
      const int64_t jo_s = ((hm >> lane) & 1ull) ? jo : 0;
      const int j_s = ((hm >> lane) & 1ull) ? j : 0;
      auto issue = [&](int q, EvRows& R) {
        const int qq = q & 63;
        const bool in_pass = q < 64;
        const bool hid = in_pass && ((hm >> qq) & 1ull);
        int64_t oi = (int64_t)(uint32_t)__builtin_amdgcn_readlane((int)io_s, qq) |
                     ((int64_t)__builtin_amdgcn_readlane((int)(io_s >> 32), qq) << 32);
        int64_t oj = (int64_t)(uint32_t)__builtin_amdgcn_readlane((int)jo_s, qq) |
                     ((int64_t)__builtin_amdgcn_readlane((int)(jo_s >> 32), qq) << 32);
        int jj = __builtin_amdgcn_readlane(j_s, qq);
        oi = in_pass ? oi : 0;
        oj = in_pass ? oj : 0;
        jj = in_pass ? jj : 0;
        R.a4 = *(const float4*)&(hid ? ih : il)[oi];
        // a logit-layer weight reads the input's row 0 (unused); the select
        // keeps the row addresses in registers (an unselected load of zh
        // made the compiler demote them to scratch)
        R.z4 = *(const float4*)&(hid ? zh : ih)[oj];
        R.wc = wl[jj];
      };
      int q = 0;
      float pv = 0.f;  // lane q: candidate q's partial sum
      // candidate q: list its pairs, request candidate q + 3 into R, score.
      // The request is made on every path (a candidate not scored here lists
      // no pairs): a load under a branch would make the merge wait for every
      // load in flight.
      auto unit = [&](EvRows& R) {
        const bool use = (okm >> q) & 1ull;
        const bool hid = (hm >> q) & 1ull, raw = (rawm >> q) & 1ull;
        const int jq = __builtin_amdgcn_readlane(j, q);
        const float deq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(de), q));
        float in[4] = {R.a4.x, R.a4.y, R.a4.z, R.a4.w};
        if (!raw) {
#pragma unroll
          for (int t = 0; t < 4; ++t) in[t] = act_fn(in[t], act, gamma);
        }
        const float wv = (hid && lane < C) ? R.wc : ((lane == jq) ? 1.f : 0.f);
        if (lane < CM) wcol[lane] = wv;
        const float wmax = row16_max(lane < C ? fabsf(wv) : 0.f);
        float wr[CM];  // the column, wave-uniform (scalar registers)
#pragma unroll
        for (int cc = 0; cc < CM; ++cc)
          wr[cc] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wv), cc));
        const float zv[4] = {R.z4.x, R.z4.y, R.z4.z, R.z4.w};
        bool pr[4];  // sample 4l + t is a pair
        uint64_t bt[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          pr[t] = use && sl + t < N && in[t] != 0.f && in_subset(sub, sub0, sl + t);
          bt[t] = __ballot(pr[t]);
        }
        const int npairs = (int)(__popcll(bt[0]) + __popcll(bt[1]) + __popcll(bt[2]) + __popcll(bt[3]));
        // pairs of lower lanes come first (mbcnt: set bits below the lane),
        // then the lane's own in sample order
        uint32_t e = 0;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          e = __builtin_amdgcn_mbcnt_hi((uint32_t)(bt[t] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bt[t], e));
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (pr[t]) {
            code[e] = (uint16_t)(4 * lane + t);
            ainl[e] = in[t];
            zhl[e] = zv[t];
          }
          e += pr[t] ? 1u : 0u;
        }
        issue(q + 3, R);
        __builtin_amdgcn_wave_barrier();
        float v = 0.f;
        for (int e0 = 0; e0 < npairs; e0 += 64) {
          const int ee = e0 + lane;
          const int ec = ee < npairs ? ee : 0;
          const int s = code[ec];
          float da;
          const float dl = pair_change<CM, kEvT>(C, act, gamma, !hid, zhl[ec], deq, wr, wcol,
                                                 wmax, ainl[ec], &pl_lds[s], y_lds[s], da);
          v += (ee < npairs) ? dl : 0.f;
        }
        __builtin_amdgcn_wave_barrier();
        const float tot = npairs ? wave_sum_f32(v) : 0.f;
        pv = (lane == q) ? tot : pv;
        ++q;
      };
      // the requests go out in candidate order, as in the loop below, so the
      // waits there hold on every path into it
      EvRows R0, R1, R2;
      issue(0, R0);
      __builtin_amdgcn_sched_barrier(0);
      issue(1, R1);
      __builtin_amdgcn_sched_barrier(0);
      issue(2, R2);
      __builtin_amdgcn_sched_barrier(0);
      if (kFirst) __syncthreads();
      // whole rounds of three (up to two units past nl list no pairs): no
      // exit between the positions, whose merged paths would blur the waits
      for (int q3 = 0; q3 < nl; q3 += 3) {
        unit(R0);
        unit(R1);
        unit(R2);
      }
      // lane q writes candidate q's partial sum: no store among the row
      // requests, whose waits count every memory operation in flight
      if (lane < nl) a.partial[(int64_t)(kw + (pass + qo) * wpt) * ntiles + b] = pv;
      if (scored && !live) a.partial[(int64_t)(kw + (pass + lane) * wpt) * ntiles + b] = 0.f;
    };
    run_pass(0, std::true_type{});
    for (int pass = 64; pass < nu; pass += 64) run_pass(pass, std::false_type{});
  }
}

// ---------------------------------------------------------------------------
// selection (Eq. 6): one block, thread k owns candidate k
// ---------------------------------------------------------------------------

// Where candidate k's tile sums are.
struct PartialSrc {
  const float* partial;  // last two layers: partial[k * ntiles + b]
  int ntiles;
  const float* pslab;    // layer slab_layer (L-3 for nets of three or more layers)
  int nslab, slab_layer;
  const float* pchain;   // layers 0..chain_top (L-4 for deeper nets)
  int nchain, chain_top;
};

// The loss change of candidate k (+inf when rejected by the bound) from its
// tile sums, by sixteen lanes: lane r adds tiles r, r+16, ... in order, then
// a fixed butterfly joins the sixteen (fp64).  Valid in lane r = 0; every
// lane of the sixteen must call it.
__device__ __forceinline__ double candidate_dl(const NetDev& net, const PartialSrc& src,
                                               const mca_cand* cands, const Aux* aux, int K,
                                               int k, int r) {
  double s = 0.0;
  if (k < K) {
    const int layer = cands[k].layer;
    const float* p = src.partial + (int64_t)k * src.ntiles;
    int nt = src.ntiles;
    if (layer <= src.chain_top) {
      p = src.pchain + (int64_t)k * src.nchain;
      nt = src.nchain;
    } else if (layer == src.slab_layer) {
      p = src.pslab + (int64_t)k * src.nslab;
      nt = src.nslab;
    }
    // 32 loads in flight (up to 512 partials in one round trip), added in
    // order: lane r adds partials r, r+16, r+32, ...
    constexpr int kLoads = 32;
    for (int t0 = r; t0 < nt; t0 += 16 * kLoads) {
      float v[kLoads];
#pragma unroll
      for (int u = 0; u < kLoads; ++u) v[u] = (t0 + 16 * u < nt) ? gload(&p[t0 + 16 * u]) : 0.f;
#pragma unroll
      for (int u = 0; u < kLoads; ++u)
        if (t0 + 16 * u < nt) s += (double)v[u];
    }
  }
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  return (k < K && aux[k].valid) ? s / subset_count(net) : __builtin_huge_val();
}

// Loss changes and the selection in one launch.  Block b adds the tile sums
// of candidates 4b .. 4b+3 (16 lanes each, in the order of candidate_dl) into
// dL, so the partial sums of a batch are read by many CUs at once.  With
// do_select, the block that finishes last (counted in st->sel_done, which is
// zero between launches) reads every dL and takes the decision: the first
// candidate that passes the test (Eq. 6 or Eq. 7), the trace and the
// counters.
constexpr int kSelThreads = 64;
constexpr int kSelPerBlock = kSelThreads / 16;
__global__ __launch_bounds__(kSelThreads) void k_reduce_select(
    const NetDev net, PartialSrc src, const mca_cand* cands, const Aux* aux, int K, double* dL,
    DevState* st, int do_select, int32_t* tr_chosen, double* tr_dl, int64_t tr_cap) {
  const int tid = threadIdx.x;
  {
    const int k = blockIdx.x * kSelPerBlock + (tid >> 4), r = tid & 15;
    const double v = candidate_dl(net, src, cands, aux, K, k, r);
    if (k < K && r == 0) dL[k] = v;
  }
  if (!do_select) return;
  __shared__ int last;
  __threadfence();  // this block's loss changes before its count
  __syncthreads();
  if (tid == 0) last = atomicAdd(&st->sel_done, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();  // every block's loss changes after the count
  // one pass over chunks of 64 candidates (lane = candidate): the first that
  // passes the test, the tie-band count up to it, the trace of every change
  const uint64_t t = st->t, tb = st->trace_base;
  const int64_t slot = (int64_t)(t - tb);
  const bool traced = tr_chosen != nullptr && slot >= 0 && slot < tr_cap;
  int kc = K;
  uint64_t nt = 0;
  for (int k0 = 0; k0 < K; k0 += kSelThreads) {
    const int k = k0 + tid;
    double v = 0.0, th = 0.0;
    if (k < K) {
      v = __hip_atomic_load(&dL[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      th = aux[k].theta;
    }
    if (traced && tr_dl != nullptr && k < K) tr_dl[slot * K + k] = v;
    if (kc < K) continue;  // decided in an earlier chunk
    const uint64_t acc = __ballot(k < K && accepts(v, net.ties, th));
    const uint64_t tie = __ballot(k < K && fabs(v) < 1e-6);
    if (acc != 0ull) {
      const int f = (int)__ffsll((unsigned long long)acc) - 1;
      kc = k0 + f;
      nt += (uint64_t)__popcll(tie & ((f == 63) ? ~0ull : ((2ull << f) - 1ull)));
    } else {
      nt += (uint64_t)__popcll(tie);
    }
  }
  if (tid == 0) {
    if (traced) tr_chosen[slot] = (kc < K) ? kc : -1;
    st->chosen = (kc < K) ? kc : -1;
    st->t = t + 1;
    st->steps += 1;
    st->evaluated += (uint64_t)K;
    st->tie += nt;
    st->sel_done = 0u;
  }
}

// ---------------------------------------------------------------------------
// commit (Eq. 6 accept branch): k_host >= 0 commits that candidate, otherwise
// the device decision st->chosen (no-op when -1)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kTile) void k_commit_column(NetDev net_arg, const mca_cand* cands,
                                                         const Aux* aux, const double* dL,
                                                         DevState* st, int k_host) {
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int k = (k_host >= 0) ? k_host : st->chosen;
  if (k < 0) return;
  const mca_cand c = cands[k];
  if (c.layer < net.L - 2) return;  // committed by the kernel that scored it
  const Aux a = aux[k];
  const int64_t n = (int64_t)blockIdx.x * kTile + threadIdx.x;
  if (n < net.N) column_commit(net, c.layer, c.j, c.i, a.de, n);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    net.W[c.layer][(int64_t)c.j * net.widths[c.layer] + c.i] = a.w_new;
    if (net.ternary) net.codes[c.layer][(int64_t)c.j * net.widths[c.layer] + c.i] = (int8_t)c.code;
    // the transposed copy of W_{L-2}: W_T[i][j] = W[j][i]
    if (net.WT != nullptr && c.layer == net.L - 2)
      net.WT[(int64_t)c.i * net.widths[c.layer + 1] + c.j] = a.w_new;
    if (net.sub_size == 0) st->L += dL[k];  // a minibatch's change is not the loss's
    st->accepted += 1;
  }
}

// ---------------------------------------------------------------------------
// full forward pass (cache fill): Z_l = W_l phi(Z_{l-1}) with phi applied while
// the B tile is staged in LDS, then the per-sample losses and their mean
// ---------------------------------------------------------------------------

// C[M][ldc] = A[M][Kd] * f(B[Kd][ldb]), 64x64 tile per block, 4x4 per thread.
// C = A op(B) (+ bias): op applies the transfer function to each input, after
// normalizing it with its column's statistics when bmu is given
// ((b - mu) / sqrt(S)); bias (may be null) adds one value per output row.
template <int ACT>  // -1: identity, else MCA_ACT_*
__global__ __launch_bounds__(256) void k_gemm_fwd(const float* __restrict__ A, int M, int Kd,
                                                  const float* __restrict__ B, int64_t ldb,
                                                  int64_t ncols, float* __restrict__ Cm,
                                                  int64_t ldc, float gamma,
                                                  const float* __restrict__ bmu,
                                                  const float* __restrict__ bS,
                                                  const float* __restrict__ bias) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int64_t m0 = (int64_t)blockIdx.y * 64, n0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.f;
  for (int k0 = 0; k0 < Kd; k0 += 16) {
    for (int e = threadIdx.x; e < 1024; e += 256) {
      const int r = e >> 4, kk = e & 15;
      const int64_t gm = m0 + r;
      const int gk = k0 + kk;
      As[kk][r] = (gm < M && gk < Kd) ? A[gm * Kd + gk] : 0.f;
    }
    for (int e = threadIdx.x; e < 1024; e += 256) {
      const int kk = e >> 6, cc = e & 63;
      const int gk = k0 + kk;
      const int64_t gn = n0 + cc;
      float v = 0.f;
      if (gk < Kd && gn < ncols) {
        v = B[(int64_t)gk * ldb + gn];
        if (bmu != nullptr) v = (v - bmu[gn]) * (1.0f / sqrtf(bS[gn]));
        if (ACT >= 0) v = act_fn(v, ACT, gamma);
      }
      Bs[kk][cc] = v;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) av[r] = As[kk][ty * 4 + r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = Bs[kk][tx * 4 + c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(av[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t gm = m0 + ty * 4 + r;
    if (gm >= M) continue;
    const float b = (bias != nullptr) ? bias[gm] : 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t gn = n0 + tx * 4 + c;
      if (gn < ncols) Cm[gm * ldc + gn] = (bias != nullptr) ? acc[r][c] + b : acc[r][c];
    }
  }
}

// The same product on the matrix cores (v_mfma_f32_16x16x4f32), for Kd a
// multiple of 16: a 128 x 128 tile of C per block, wave (wr, wc) its 64 x 64
// quarter as four by four 16 x 16 MFMA tiles.  The reduction runs in chunks
// of 16: A's rows (row-major, 16 k) staged as float4 and read back as float4
// (lane group q holds k = 4 q + t of the chunk, t = 0..3, one per MFMA); B's
// chunk ([16 k][128 columns], columns contiguous) transformed by op on its
// way into LDS and read one value per MFMA (conflict-free: the 16 lanes of a
// group read consecutive columns, the four groups rows 4 apart on a padded
// row).  The next chunk's loads are in flight while the current one is
// multiplied (double-buffered LDS).  Rows and columns beyond the matrix are
// clamped on load and dropped on store.
constexpr int kFwdT = 128;       // rows and columns of the block's tile
constexpr int kFwdK = 16;        // reduction chunk
constexpr int kFwdThreads = 256;
typedef float fwdx4 __attribute__((ext_vector_type(4)));

template <int ACT>  // -1: identity, else MCA_ACT_*
__global__ __launch_bounds__(kFwdThreads, 3) void k_gemm_fwd_mfma(
    const float* __restrict__ A, int M, int Kd, const float* __restrict__ B, int64_t ldb,
    int64_t ncols, float* __restrict__ Cm, int64_t ldc, float gamma,
    const float* __restrict__ bmu, const float* __restrict__ bS,
    const float* __restrict__ bias) {
  __shared__ __attribute__((aligned(16))) float As[2][kFwdT][kFwdK + 4];
  __shared__ __attribute__((aligned(16))) float Bs[2][kFwdK][kFwdT + 4];
  const int64_t m0 = (int64_t)blockIdx.y * kFwdT, n0 = (int64_t)blockIdx.x * kFwdT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, q = lane >> 4, li = lane & 15;
  const int wr = wave >> 1, wc = wave & 1;
  // staging: thread tid loads float4 number tid + 256 u of A's chunk
  // (128 rows x 4 float4) and of B's chunk (16 rows x 32 float4)
  constexpr int kA4 = kFwdT * kFwdK / 4 / kFwdThreads;  // 2
  constexpr int kB4 = kFwdK * kFwdT / 4 / kFwdThreads;  // 2
  const float* ga[kA4];
  const float* gb[kB4];
  float nmu[kB4][4], nrs[kB4][4];  // B's column statistics (normalized inputs)
#pragma unroll
  for (int u = 0; u < kA4; ++u) {
    const int e = tid + kFwdThreads * u;
    const int64_t m = m0 + e / (kFwdK / 4);
    ga[u] = A + (m < M ? m : M - 1) * (int64_t)Kd + 4 * (e % (kFwdK / 4));
  }
#pragma unroll
  for (int u = 0; u < kB4; ++u) {
    const int e = tid + kFwdThreads * u;
    const int kk = e / (kFwdT / 4);
    const int64_t nb = n0 + 4 * (e % (kFwdT / 4));
    gb[u] = B + (int64_t)kk * ldb + (nb < ncols ? nb : 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t nn = nb + t < ncols ? nb + t : 0;
      nmu[u][t] = bmu != nullptr ? bmu[nn] : 0.f;
      nrs[u][t] = bmu != nullptr ? 1.0f / sqrtf(bS[nn]) : 1.f;
    }
  }
  fwdx4 ra[kA4], rb[kB4];
  auto fetch = [&](int c) {
#pragma unroll
    for (int u = 0; u < kA4; ++u) ra[u] = *reinterpret_cast<const fwdx4*>(ga[u] + kFwdK * c);
#pragma unroll
    for (int u = 0; u < kB4; ++u) rb[u] = *reinterpret_cast<const fwdx4*>(gb[u] + (int64_t)kFwdK * c * ldb);
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < kA4; ++u) {
      const int e = tid + kFwdThreads * u;
      *reinterpret_cast<fwdx4*>(&As[buf][e / (kFwdK / 4)][4 * (e % (kFwdK / 4))]) = ra[u];
    }
#pragma unroll
    for (int u = 0; u < kB4; ++u) {
      const int e = tid + kFwdThreads * u;
      const int kk = e / (kFwdT / 4), c4 = e % (kFwdT / 4);
      const int64_t nb = n0 + 4 * c4;
      fwdx4 v = rb[u];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float x = v[t];
        if (bmu != nullptr) x = (x - nmu[u][t]) * nrs[u][t];
        if (ACT >= 0) x = act_fn(x, ACT, gamma);
        v[t] = (nb + t < ncols) ? x : 0.f;
      }
      *reinterpret_cast<fwdx4*>(&Bs[buf][kk][4 * c4]) = v;
    }
  };
  const fwdx4 zero = {0.f, 0.f, 0.f, 0.f};
  fwdx4 acc[4][4];
#pragma unroll
  for (int sb = 0; sb < 4; ++sb)
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[sb][cb] = zero;
  auto compute = [&](int buf) {
    fwdx4 a[4];
#pragma unroll
    for (int sb = 0; sb < 4; ++sb)
      a[sb] = *reinterpret_cast<const fwdx4*>(&As[buf][64 * wr + 16 * sb + li][4 * q]);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float bv[4];
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) bv[cb] = Bs[buf][4 * q + t][64 * wc + 16 * cb + li];
#pragma unroll
      for (int sb = 0; sb < 4; ++sb)
#pragma unroll
        for (int cb = 0; cb < 4; ++cb)
          acc[sb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[sb][t], bv[cb], acc[sb][cb], 0, 0, 0);
    }
  };
  const int nc = Kd / kFwdK;
  fetch(0);
  store(0);
  __syncthreads();
  for (int c = 0; c < nc; ++c) {
    if (c + 1 < nc) fetch(c + 1);
    compute(c & 1);
    if (c + 1 < nc) store((c + 1) & 1);
    __syncthreads();
  }
  // D layout: lane (q, li), element v -> row 16 sb + 4 q + v, column 16 cb + li
#pragma unroll
  for (int sb = 0; sb < 4; ++sb)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t m = m0 + 64 * wr + 16 * sb + 4 * q + v;
      if (m >= M) continue;
      const float b = (bias != nullptr) ? bias[m] : 0.f;
#pragma unroll
      for (int cb = 0; cb < 4; ++cb) {
        const int64_t n = n0 + 64 * wc + 16 * cb + li;
        if (n < ncols) Cm[m * ldc + n] = (bias != nullptr) ? acc[sb][cb][v] + b : acc[sb][cb][v];
      }
    }
}

// The product for at most 16 output rows (a logit layer): a block takes 64
// columns and eight waves, each wave an eighth of the reduction (Kd a
// multiple of 128) as four 16 x 16 MFMA tiles.  Lane (q, li) holds columns
// n0 + 4 li + j of tile j, so that op(B) arrives as one float4 per row, and
// k = 4 q + t of each block of 16 (A's row li as one float4); the next
// block's values are requested before the current one's products.  The
// eight partial tiles meet in LDS and are added in wave order.
constexpr int kSkinnyCols = 64;
constexpr int kSkinnyWaves = 8;
template <int ACT>
__global__ __launch_bounds__(64 * kSkinnyWaves) void k_gemm_fwd_skinny(
    const float* __restrict__ A, int M, int Kd, const float* __restrict__ B, int64_t ldb,
    int64_t ncols, float* __restrict__ Cm, int64_t ldc, float gamma,
    const float* __restrict__ bmu, const float* __restrict__ bS,
    const float* __restrict__ bias) {
  __shared__ float part[kSkinnyWaves][16][kSkinnyCols + 1];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, q = lane >> 4, li = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * kSkinnyCols, nb = n0 + 4 * li;
  float nmu[4], nrs[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t nn = nb + j < ncols ? nb + j : 0;
    nmu[j] = bmu != nullptr ? bmu[nn] : 0.f;
    nrs[j] = bmu != nullptr ? 1.0f / sqrtf(bS[nn]) : 1.f;
  }
  const int kq = Kd / kSkinnyWaves, nkb = kq / 16;
  const int64_t k0 = (int64_t)wave * kq + 4 * q;
  const bool mrow = li < M;
  const float* arow = A + (int64_t)(mrow ? li : 0) * Kd + k0;
  const float* bp = B + k0 * ldb + (nb < ncols ? nb : 0);
  const fwdx4 zero = {0.f, 0.f, 0.f, 0.f};
  fwdx4 acc[4] = {zero, zero, zero, zero};
  fwdx4 a_nx, b_nx[4];
  auto fetch = [&](int kb) {
    a_nx = *reinterpret_cast<const fwdx4*>(arow + 16 * kb);
#pragma unroll
    for (int t = 0; t < 4; ++t) b_nx[t] = *reinterpret_cast<const fwdx4*>(bp + (int64_t)(16 * kb + t) * ldb);
  };
  fetch(0);
  for (int kb = 0; kb < nkb; ++kb) {
    const fwdx4 a4 = mrow ? a_nx : zero;
    fwdx4 bv[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) bv[t] = b_nx[t];
    if (kb + 1 < nkb) fetch(kb + 1);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float x = bv[t][j];
        if (bmu != nullptr) x = (x - nmu[j]) * nrs[j];
        if (ACT >= 0) x = act_fn(x, ACT, gamma);
        x = (nb + j < ncols) ? x : 0.f;
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4[t], x, acc[j], 0, 0, 0);
      }
  }
  // D layout: lane (q, li), element v of tile j -> row 4 q + v, column 4 li + j
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int v = 0; v < 4; ++v) part[wave][4 * q + v][4 * li + j] = acc[j][v];
  __syncthreads();
  for (int e = tid; e < 16 * kSkinnyCols; e += 64 * kSkinnyWaves) {
    const int m = e / kSkinnyCols, c = e - m * kSkinnyCols;
    const int64_t n = n0 + c;
    if (m < M && n < ncols) {
      float v = part[0][m][c];
#pragma unroll
      for (int w = 1; w < kSkinnyWaves; ++w) v += part[w][m][c];
      Cm[(int64_t)m * ldc + n] = (bias != nullptr) ? v + bias[m] : v;
    }
  }
}

// One layer of the forward pass: the skinny matrix-core product for a logit
// layer (at most 16 rows, reduction a multiple of 128), the tiled one when the
// reduction width is a multiple of 16, the vector one otherwise.
template <int ACT>
hipError_t forward_layer(const float* A, int M, int Kd, const float* B, int64_t ldb, int64_t N,
                         float* Cm, int64_t ldc, float gamma, const float* mu, const float* S,
                         const float* bias, hipStream_t s) {
  if (M <= 16 && Kd % (16 * kSkinnyWaves) == 0 && ldb % 4 == 0) {
    hipLaunchKernelGGL(k_gemm_fwd_skinny<ACT>, dim3((unsigned)((N + kSkinnyCols - 1) / kSkinnyCols)),
                       dim3(64 * kSkinnyWaves), 0, s, A, M, Kd, B, ldb, N, Cm, ldc, gamma, mu, S, bias);
  } else if (Kd % kFwdK == 0) {
    dim3 grid((unsigned)((N + kFwdT - 1) / kFwdT), (unsigned)((M + kFwdT - 1) / kFwdT));
    hipLaunchKernelGGL(k_gemm_fwd_mfma<ACT>, grid, dim3(kFwdThreads), 0, s, A, M, Kd, B, ldb, N,
                       Cm, ldc, gamma, mu, S, bias);
  } else {
    dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
    hipLaunchKernelGGL(k_gemm_fwd<ACT>, grid, dim3(256), 0, s, A, M, Kd, B, ldb, N, Cm, ldc,
                       gamma, mu, S, bias);
  }
  return hipGetLastError();
}
hipError_t forward_layer_act(int act, bool first, const float* A, int M, int Kd, const float* B,
                             int64_t ldb, int64_t N, float* Cm, int64_t ldc, float gamma,
                             const float* mu, const float* S, const float* bias, hipStream_t s) {
  if (first) return forward_layer<-1>(A, M, Kd, B, ldb, N, Cm, ldc, gamma, mu, S, bias, s);
  if (act == MCA_ACT_TANH)
    return forward_layer<MCA_ACT_TANH>(A, M, Kd, B, ldb, N, Cm, ldc, gamma, mu, S, bias, s);
  if (act == MCA_ACT_RELU)
    return forward_layer<MCA_ACT_RELU>(A, M, Kd, B, ldb, N, Cm, ldc, gamma, mu, S, bias, s);
  return forward_layer<MCA_ACT_GAUSS>(A, M, Kd, B, ldb, N, Cm, ldc, gamma, mu, S, bias, s);
}

// l_n and the softmax of every sample from the cached logits; fp64 block sums
// of l_n.
__global__ __launch_bounds__(kTile) void k_ce_forward(NetDev net_arg, double* bsum) {
  __shared__ double red[kTile];
  __shared__ NetDev net;
  stage_net(net, net_arg);
  const int64_t n = (int64_t)blockIdx.x * kTile + threadIdx.x;
  double v = 0.0;
  if (n < net.N) {
    float z[kCMax];
#pragma unroll
    for (int c = 0; c < kCMax; ++c) z[c] = (c < net.C) ? gload(&net.Z[net.L - 1][(int64_t)c * net.Ns + n]) : 0.f;
    float p[kCMax];
    const float l = softmax_ce(z, net.C, gload(&net.y[n]), p);
    gstore(&net.ell[n], l);
#pragma unroll
    for (int c = 0; c < kCMax; ++c)
      if (c < net.C) gstore(&net.prob[(int64_t)c * net.Ns + n], p[c]);
    v = (double)l;
  }
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = kTile / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = red[0];
}

__global__ void k_loss_total(NetDev net, const double* bsum, int nb, DevState* st) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int b = 0; b < nb; ++b) s += bsum[b];
  st->L = s / (double)net.N;
}

// ---------------------------------------------------------------------------
// host-side launchers
// ---------------------------------------------------------------------------

hipError_t launch_propose(const NetDev& net, uint64_t t, bool use_dev_t, const DevState* st,
                          int K, mca_cand* cands, Aux* aux, const uint64_t* fmask,
                          uint64_t* cmask, hipStream_t s) {
  hipLaunchKernelGGL(k_propose, dim3((K + 63) / 64), dim3(64), 0, s, net, t, use_dev_t ? 1 : 0,
                     st, K, cands, aux, fmask, cmask);
  return hipGetLastError();
}

hipError_t launch_prepare(const NetDev& net, const mca_cand* cands, int K, Aux* aux,
                          const uint64_t* fmask, uint64_t* cmask, hipStream_t s) {
  hipLaunchKernelGGL(k_prepare, dim3((K + 63) / 64), dim3(64), 0, s, net, cands, K, aux, fmask,
                     cmask);
  return hipGetLastError();
}

int eval_tiles(int64_t n_samples) { return (int)((n_samples + kEvT - 1) / kEvT); }
int eval_tile_size() { return kEvT; }

namespace {
// Blocks of k_eval_tiles that fit the device at once (queried once per
// device and class-count variant).
int eval_grid(const void* kernel, int variant) {
  static int cached[16][2];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return 0;
  if (cached[dev][variant] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kEvThreads, 0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return 0;
    cached[dev][variant] = (per_cu > 0 ? per_cu : 1) * cus;
  }
  return cached[dev][variant];
}
}  // namespace

hipError_t launch_eval(const NetDev& net, const mca_cand* cands, const Aux* aux,
                       const uint64_t* cmask, int K, float* partial, int ntiles,
                       const DevState* st, hipStream_t s) {
  const int L = net.L;
  EvArgs a{};
  a.in_hid = (L >= 3) ? net.Z[L - 3] : net.XT;
  a.in_log = (L >= 2) ? net.Z[L - 2] : net.XT;
  a.z_hid = (L >= 2) ? net.Z[L - 2] : net.Z[L - 1];
  a.p_log = net.prob;
  a.w_log = net.W[L - 1];
  a.y = net.y;
  a.cands = cands;
  a.aux = aux;
  a.cmask = cmask;
  a.partial = partial;
  a.st = st;
  a.sub_size = net.sub_size;
  a.sub_period = net.sub_period;
  a.N = net.N;
  a.Ns = net.Ns;
  a.L = L;
  a.C = net.C;
  a.act = net.act;
  a.nh = net.widths[L - 1];
  a.K = K;
  a.ntiles = ntiles;
  a.gamma = net.gamma;
  const bool c10 = net.C == 10;
  const void* kernel = c10 ? (const void*)k_eval_tiles<10> : (const void*)k_eval_tiles<kCMax>;
  const int fit = eval_grid(kernel, c10 ? 0 : 1);
  if (fit <= 0) return hipErrorInvalidDevice;
  // blocks per tile: share the resident blocks out over the tiles, no more
  // than the candidates need
  const int per_tile = fit / ntiles > 1 ? fit / ntiles : 1;
  const int need = (K + kEvWaves - 1) / kEvWaves;
  a.bpt = per_tile < need ? per_tile : need;
  if (a.bpt < 1) a.bpt = 1;  // no candidates: one block per tile finds no work
  if (K <= 0) return hipSuccess;  // nothing to score (the kernel reads candidate K - 1)
  const int64_t slots = (int64_t)ntiles * a.bpt;
  const dim3 grid((unsigned)(slots < fit ? slots : fit));
  if (c10)
    hipLaunchKernelGGL(k_eval_tiles<10>, grid, dim3(kEvThreads), 0, s, a);
  else
    hipLaunchKernelGGL(k_eval_tiles<kCMax>, grid, dim3(kEvThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_select(const NetDev& net, const float* partial, int ntiles,
                         const mca_cand* cands, const float* pslab, int nslab,
                         const float* pchain, int nchain, const Aux* aux, int K, double* dL,
                         DevState* st, bool do_select, int32_t* tr_chosen, double* tr_dl,
                         int64_t tr_cap, hipStream_t s) {
  PartialSrc src;
  src.partial = partial;
  src.ntiles = ntiles;
  src.pslab = pslab;
  src.nslab = nslab;
  src.slab_layer = (net.L >= 3) ? net.L - 3 : -1;
  src.pchain = pchain;
  src.nchain = nchain;
  src.chain_top = (net.L >= 4) ? net.L - 4 : -1;
  const int nblk = K > 0 ? (K + kSelPerBlock - 1) / kSelPerBlock : 1;
  hipLaunchKernelGGL(k_reduce_select, dim3(nblk), dim3(kSelThreads), 0, s, net, src, cands, aux,
                     K, dL, st, do_select ? 1 : 0, tr_chosen, tr_dl, tr_cap);
  return hipGetLastError();
}

hipError_t launch_commit(const NetDev& net, const mca_cand* cands, const Aux* aux,
                         const double* dL, DevState* st, int k_host, int ntiles, hipStream_t s) {
  hipLaunchKernelGGL(k_commit_column, dim3(ntiles), dim3(kTile), 0, s, net, cands, aux, dL, st,
                     k_host);
  return hipGetLastError();
}

hipError_t launch_loss_refresh(const NetDev& net, double* bsum, DevState* st, hipStream_t s) {
  const int nb = (int)((net.N + kTile - 1) / kTile);
  hipLaunchKernelGGL(k_ce_forward, dim3(nb), dim3(kTile), 0, s, net, bsum);
  hipLaunchKernelGGL(k_loss_total, dim3(1), dim3(64), 0, s, net, bsum, nb, st);
  return hipGetLastError();
}

// Forward pass of a net with biases and / or normalized hidden fields: each
// layer's GEMM normalizes and transforms its input with the statistics of the
// layer before, adds the biases, then the layer's own statistics.
hipError_t launch_forward_norm(const NetDev& net, const NormDev& nd, double* bsum, DevState* st,
                               hipStream_t s) {
  const int64_t N = net.N;
  for (int l = 0; l < net.L; ++l) {
    const int M = net.widths[l + 1], Kd = net.widths[l];
    const float* B = (l == 0) ? net.XT : net.Z[l - 1];
    const float* mu = (l > 0 && net.ln) ? nd.MU[l - 1] : nullptr;
    const float* S = (l > 0 && net.ln) ? nd.S[l - 1] : nullptr;
    hipError_t e = forward_layer_act(net.act, l == 0, net.W[l], M, Kd, B, net.Ns, N, net.Z[l],
                                     net.Ns, net.gamma, mu, S, net.B[l], s);
    if (e != hipSuccess) return e;
    if (net.ln && l < net.L - 1) {
      e = launch_norm_stats(net, nd, l, s);
      if (e != hipSuccess) return e;
    }
  }
  const int nb = (int)((N + kTile - 1) / kTile);
  hipLaunchKernelGGL(k_ce_forward, dim3(nb), dim3(kTile), 0, s, net, bsum);
  hipLaunchKernelGGL(k_loss_total, dim3(1), dim3(64), 0, s, net, bsum, nb, st);
  return hipGetLastError();
}

hipError_t launch_forward(const NetDev& net, double* bsum, DevState* st, hipStream_t s) {
  const int64_t N = net.N;
  for (int l = 0; l < net.L; ++l) {
    const int M = net.widths[l + 1], Kd = net.widths[l];
    const float* B = (l == 0) ? net.XT : net.Z[l - 1];
    hipError_t e = forward_layer_act(net.act, l == 0, net.W[l], M, Kd, B, net.Ns, N, net.Z[l],
                                     net.Ns, net.gamma, nullptr, nullptr, nullptr, s);
    if (e != hipSuccess) return e;
  }
  const int nb = (int)((N + kTile - 1) / kTile);
  hipLaunchKernelGGL(k_ce_forward, dim3(nb), dim3(kTile), 0, s, net, bsum);
  hipLaunchKernelGGL(k_loss_total, dim3(1), dim3(64), 0, s, net, bsum, nb, st);
  return hipGetLastError();
}

}  // namespace mca
