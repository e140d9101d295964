// One-workgroup step loop for MLPs whose mutations touch only the last two
// layers and whose samples and weights fit one workgroup (N <= 1024 samples,
// at most kOneMaxParams weights, at most 10 classes): the logits, softmax,
// labels and weights live in LDS for the whole launch, so a step's loss
// changes (Eq. 2, R = 0) are summed, the first candidate that passes the test
// is chosen (Eq. 6 or 7) and committed inside the workgroup, with no exchange
// between workgroups.  This suits a small net with one or two candidates per
// step, where the multi-workgroup loop would spend most of each step waiting
// for the decision to cross the chip.
//
// The loop runs in passes of two slots.  With K = 2 a pass is one step.  With
// K = 1 a pass scores steps t and t + 1 against the same committed state:
// while step t rejects, nothing changes before step t + 1, so its candidate
// and its loss change are exactly those of the one-step order, and the pass
// resolves both steps; when step t accepts, step t + 1's score is discarded
// (counted as wasted) and step t + 1 opens the next pass.
//
// The part of the candidate stream that needs no state (the counter-based
// records and acceptance thresholds) is decoded ahead into an LDS ring, one
// (step, candidate) per thread.  Thread n owns sample n.  Per pass:
//  1. every thread patches its rows (requested before the last commit) with
//     that commit, stages its input and field for each slot in LDS,
//     and appends the slots with a non-zero input to that slot's work list;
//  2. the workgroup scores the listed pairs (pair_change, from the cached
//     softmax) into per-pair slots, so only about a fifth of the samples of
//     an image-like input cost any work, and keeps each pair's activation
//     change for the commit;
//  3. each thread adds its sample's slots: a fixed-order sum over the 64
//     lanes of each wave (fp32), then over the 16 waves (fp64, one DPP order
//     within a row of 16 lanes), which every wave takes, so every wave knows
//     the decision at once;
//  4. the listed pairs of the chosen slot are committed with the expressions
//     the scoring used.
// Candidates are completed (new value, threshold, logit-layer column) one
// pass ahead: while a pass is scored, the last wave completes those of the
// pass that would start at t + S (S: steps per pass) from the LDS weights
// into a ring indexed by step; a commit then patches the completed
// candidates of the steps after it that it touches (the same weight,
// completed again from the committed value and code, or a logit weight of a
// hidden candidate's column).
// Rows need no state to be located (parameter, row and column come from the
// ring), so each pass requests, at its start, the rows of the pass that
// follows should none of its steps but the last accept; with K = 1 a pass
// that resolves one step carries its second step's rows over.
// The trace is kept in LDS and written out every 64 steps.
#include "device_common.hpp"
#include "one_loop.hpp"

namespace mca {

namespace {

constexpr int kOneThreads = kOneMaxSamples;
constexpr int kOneWaves = kOneThreads / 64;
constexpr int kSlots = 2;     // candidates scored per pass
constexpr int kRing = 64;     // steps of decoded records kept in LDS (a power of two)
constexpr int kRefill = 32;   // steps decoded per refill of the ring
constexpr int kTrace = 64;    // steps of trace kept in LDS
constexpr int kAhead = 8;     // steps of completed candidates kept in LDS (a power of two)
constexpr int kOneCM = 10;    // class bound of the LDS logit tile
constexpr int kDrawWave = kOneWaves - 1;
constexpr int kStoreWave = kOneWaves - 2;  // stores the committed weight to HBM
static_assert(kSlots * 16 <= 64, "the draw takes one (slot, class) per lane");
static_assert(kOneMaxK <= kSlots, "a step fits one pass");
static_assert(kOneThreads < 65536 && kSlots <= 2, "two 16-bit list counts share one word");

template <int kCtrl>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), kCtrl, 0xF, 0xF, true));
}
// Sum over the 64 lanes of a wave in one fixed order, the same in every
// lane: DPP within rows of 16 (lane ^ 1, ^ 2, then the mirrored partners),
// then the four rows in order.
__device__ __forceinline__ float wave_sum_f32(float v) {
  v += dpp_f32<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f32<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);  // row_half_mirror
  v += dpp_f32<0x140>(v);  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}

template <int kCtrl>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, kCtrl, 0xF, 0xF, true);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), kCtrl, 0xF, 0xF, true);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Sum over each row of 16 lanes in one fixed order (fp64): every step adds
// a lane's value to its partner's, so both hold the same bits, and after
// four steps every lane of the row holds the row's sum.
__device__ __forceinline__ double wave_row_sum_f64(double v) {
  v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f64<0x141>(v);  // row_half_mirror
  v += dpp_f64<0x140>(v);  // row_mirror
  return v;
}

__global__ __launch_bounds__(kOneThreads) void k_one_loop(OneArgs a) {
  constexpr int CM = kOneCM;
  __shared__ NetDev net;
  stage_net(net, a.net);
  __shared__ float zl_lds[CM * kOneThreads];  // logits, [class][sample]
  __shared__ float pl_lds[CM * kOneThreads];  // their softmax
  __shared__ int y_lds[kOneThreads];
  __shared__ float w_lds[kOneMaxParams];      // every layer's weights, layer by layer
  __shared__ int8_t c_lds[kOneMaxParams];     // their ternary codes
  __shared__ mca_cand ring_lds[kRing][kOneMaxK];  // decode_index of step t at t mod kRing
  __shared__ double theta_ring[kRing][kOneMaxK];
  // the record's row offsets (elements): its input row, and its field row for
  // a hidden unit (-1 for a logit weight, whose field row is not read)
  __shared__ int2 roff_ring[kRing][kOneMaxK];
  // completed candidates of step t at t mod kAhead
  __shared__ mca_cand cand_lds[kAhead][kOneMaxK];
  __shared__ Aux aux_lds[kAhead][kOneMaxK];
  __shared__ int64_t sub_lds[kAhead];                // the step's minibatch start
  __shared__ float wcol_lds[kAhead][kOneMaxK][CM];   // logit-layer column (one-hot for a logit weight)
  __shared__ float wmax_lds[kAhead][kOneMaxK];
  __shared__ float ain_lds[kSlots][kOneThreads];  // the pass's input of each pair
  __shared__ float zh_lds[kSlots][kOneThreads];   // and the mutated unit's field
  __shared__ float dlp_lds[kSlots][kOneThreads];  // per-pair loss changes (0 unless listed)
  __shared__ float da_lds[kSlots][kOneThreads];   // and activation changes
  __shared__ uint16_t list_lds[kSlots][kOneThreads];  // listed samples, by slot
  __shared__ float zrow_lds[kOneThreads];  // a committed hidden unit's new field, per sample
  __shared__ float red_lds[kOneWaves][kSlots];
  __shared__ int32_t trc_lds[kTrace];  // trace of the current 64 steps
  __shared__ double trd_lds[kTrace][kOneMaxK];
  __shared__ uint32_t list_n;  // listed pairs: slot 0 in the low half, slot 1 in the high

  const int K = a.K;
  const int kshift = K - 1;  // slot q is candidate q & (K - 1) of step t + (q >> kshift)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = net.L, C = net.C;
  const int act = net.act;
  const float gamma = net.gamma;
  const int64_t N = net.N, Ns = net.Ns;
  const int n = tid;
  const bool live = n < N;
  const int64_t n_ld = live ? n : 0;
  const int n32 = (int)n_ld, ns32 = (int)Ns;
  const bool two = L == 2;
  const float* const in_hid = net.XT;                   // input of the hidden layer (L = 2)
  const float* const in_log = two ? net.Z[0] : net.XT;  // input of the logit layer
  float* const z_hid = net.Z[0];                        // hidden local fields (L = 2)
  const int nh = net.widths[L - 1];
  const int woff1 = two ? net.widths[1] * net.widths[0] : 0;  // the logit layer in w_lds
  const int n_par = woff1 + net.widths[L] * net.widths[L - 1];
  const uint64_t t0 = a.st->t;
  const uint64_t t_end = t0 + a.n_steps;
  auto woff = [&](int layer) { return layer == 0 ? 0 : woff1; };
  // slots of the pass that starts at step tp, and slot q's entry of the
  // candidate ring
  auto slots = [&](uint64_t tp) { return (K == 2 || tp + 1 < t_end) ? kSlots : 1; };
  auto ent = [&](uint64_t tp, int q) { return (int)((tp + (uint64_t)(q >> kshift)) & (kAhead - 1)); };

  // the sample's logits, softmax and label, and the weights, move to LDS
  for (int c = 0; c < CM; ++c) {
    zl_lds[c * kOneThreads + n] = (live && c < C) ? gload(&net.Z[L - 1][(int64_t)c * Ns + n_ld]) : 0.f;
    pl_lds[c * kOneThreads + n] = (live && c < C) ? gload(&net.prob[(int64_t)c * Ns + n_ld]) : 0.f;
  }
  y_lds[n] = live ? gload(&net.y[n_ld]) : 0;
  for (int e = tid; e < n_par; e += kOneThreads) {
    const int l = (two && e >= woff1) ? 1 : 0;
    const int64_t idx = e - woff(l);
    w_lds[e] = gload(&net.W[l][idx]);
    c_lds[e] = net.ternary ? gload(&net.codes[l][idx]) : (int8_t)0;
  }
#pragma unroll
  for (int q = 0; q < kSlots; ++q) dlp_lds[q][n] = 0.f;

  // every thread: the stream's records and thresholds of steps t_from ..
  // t_from + m_steps - 1 (those before t_end), one (step, candidate) each
  auto fill = [&](uint64_t t_from, int m_steps) {
    for (int e = tid; e < m_steps * K; e += kOneThreads) {
      const int m = e >> kshift, k = e & (K - 1);
      const uint64_t t = t_from + (uint64_t)m;
      if (t < t_end) {
        const mca_cand r = decode_index(net, t, (uint64_t)k);
        ring_lds[t & (kRing - 1)][k] = r;
        theta_ring[t & (kRing - 1)][k] = accept_theta(net.rule, net.beta, net.seed, net.tag, t,
                                                      (uint64_t)k);
        roff_ring[t & (kRing - 1)][k] = make_int2(r.i * ns32, r.layer == L - 2 ? r.j * ns32 : -1);
      }
    }
  };
  // the draw wave, lane l: slot q = l / 16 of the pass at step tp and its
  // class entry cc = l mod 16, completed into the candidate ring as
  // decode_candidate and prepare_candidate do, from the LDS weights and codes
  auto draw = [&](uint64_t tp) {
    const int q = lane >> 4, cc = lane & 15;
    const bool on = tp < t_end && q < slots(tp);
    const int bb = ent(tp, q), k = q & (K - 1);
    float wv = 0.f;
    if (on) {
      const uint64_t step = tp + (uint64_t)(q >> kshift);
      const mca_cand r = ring_lds[step & (kRing - 1)][k];
      const bool hid = r.layer == L - 2;
      wv = hid ? ((cc < C) ? w_lds[woff1 + cc * nh + r.j] : 0.f) : ((cc == r.j) ? 1.f : 0.f);
      if (cc < CM) wcol_lds[bb][k][cc] = wv;
      if (cc == 0) {
        const int e = woff(r.layer) + r.j * net.widths[r.layer] + r.i;
        const float w = w_lds[e];
        mca_cand c = r;
        if (net.ternary) finish_ternary(net, c, (int)c_lds[e]);
        if (c.flags & MCA_CAND_PRUNE) {
          c.code = 0;
          c.d = 0.0f - w;
        }
        Aux x;
        x.w_old = w;
        x.w_new = (c.flags & MCA_CAND_PRUNE) ? 0.0f
                  : (net.ternary ? (float)c.code * net.scales[c.layer] : w + c.d);
        x.de = x.w_new - x.w_old;
        x.valid = !(net.bound > 0.f && fabsf(x.w_new) >= net.bound);
        x.theta = theta_ring[step & (kRing - 1)][k];
        cand_lds[bb][k] = c;
        aux_lds[bb][k] = x;
        sub_lds[bb] = subset_start(net, step);
      }
    }
    // the column's largest magnitude: a maximum over each row of 16 lanes
    float wm = fabsf(wv);
    wm = fmaxf(wm, dpp_f32<0xB1>(wm));   // lane ^ 1
    wm = fmaxf(wm, dpp_f32<0x4E>(wm));   // lane ^ 2
    wm = fmaxf(wm, dpp_f32<0x141>(wm));  // mirror within eight
    wm = fmaxf(wm, dpp_f32<0x140>(wm));  // mirror within sixteen
    if (on && cc == 0) wmax_lds[bb][k] = wm;
  };
  // every thread: the sample's rows for the slots of the pass at step tp
  // (those before t_end), from the ring's records: the mutated weight's
  // input and, for a hidden unit, its local field (a logit weight's field
  // row is not read)
  auto load_rows = [&](uint64_t tp, float (&av)[kSlots], float (&zv)[kSlots]) {
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
      av[q] = 0.f;
      zv[q] = 0.f;
      const uint64_t step = tp + (uint64_t)(q >> kshift);
      if (step < t_end) {
        // rows are short (N <= 1024): 32-bit offsets
        const int2 o = roff_ring[step & (kRing - 1)][q & (K - 1)];
        const bool hid = o.y >= 0;
        av[q] = gload(&(hid ? in_hid : in_log)[o.x + n32]);
        zv[q] = gload(&z_hid[(hid ? o.y : 0) + n32]);
      }
    }
  };
  // rows of this pass (a_cur, z_cur) and of the pass that follows when no
  // step before its last accepts (a_pre, z_pre, requested at its start)
  float a_cur[kSlots], z_cur[kSlots], a_pre[kSlots], z_pre[kSlots];
  const int S = kSlots >> kshift;  // steps per pass

  if (tid == 0) list_n = 0;
  fill(t0, kRing);
  uint64_t filled = t0 + kRing;  // the ring holds every step before this one
  __syncthreads();
  if (wave == kDrawWave) draw(t0);
  load_rows(t0, a_cur, z_cur);
  __syncthreads();

  // committed scalars, carried in registers by thread 0
  double L_acc = 0.0;
  uint64_t n_acc = 0, n_tie = 0, n_waste = 0;
  int last_k = -1;
  if (tid == 0) {
    L_acc = a.st->L;
    n_acc = a.st->accepted;
    n_tie = a.st->tie;
    n_waste = a.st->wasted;
  }
  // the last commit (uniform) and whether it moved this thread's sample
  int lc_layer = -1, lc_j = 0;
  bool lc_moved = false;
  const double count = subset_count(net);

  for (uint64_t t = t0; t < t_end;) {
    const uint64_t s = t - t0;
    const int nq = slots(t);
    // the ring must hold the records of this pass and of the next one
    if (filled < t_end && filled < t + 2 * kSlots) {
      fill(filled, kRefill);
      filled += kRefill;
      __syncthreads();
    }
    // the rows of the pass after this one, should it start at t + S: they
    // go out first, so that they have landed before any spill reload of the
    // pass (a reload waits for every memory operation in flight)
    load_rows(t + (uint64_t)S, a_pre, z_pre);
    // 1. this pass's rows with the last commit applied (a hidden unit's
    // field row, or a logit weight's input fed by that unit), staged in LDS;
    // the pairs with a non-zero input go on their slot's list (every sample
    // moves on a commit; only the step's minibatch is scored).  Every row
    // requested before the last commit took the commits before it.
    {
      const float zr = lc_moved ? zrow_lds[n] : 0.f;
      uint64_t m[kSlots];
#pragma unroll
      for (int q = 0; q < kSlots; ++q) {
        m[q] = 0;
        if (q < nq) {
          const mca_cand c = cand_lds[ent(t, q)][q & (K - 1)];
          float av = a_cur[q], zv = z_cur[q];
          if (lc_moved && lc_layer == L - 2) {
            if (c.layer == L - 2 && c.j == lc_j) zv = zr;
            if (c.layer == L - 1 && two && c.i == lc_j) av = zr;
          }
          a_cur[q] = av;  // a row carried into the next pass
          z_cur[q] = zv;
          // the logit layer's input is an activation when a hidden layer feeds it
          const float ain = (c.layer == L - 1 && two) ? act_fn(av, act, gamma) : av;
          ain_lds[q][n] = live ? ain : 0.f;
          zh_lds[q][n] = zv;
          m[q] = __ballot(live && ain != 0.f);
        }
      }
      const uint32_t tot = (uint32_t)__popcll(m[0]) | ((uint32_t)__popcll(m[1]) << 16);
      uint32_t base = 0;
      if (lane == 0 && tot) base = atomicAdd(&list_n, tot);
      base = (uint32_t)__shfl((int)base, 0, 64);
      const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
      for (int q = 0; q < kSlots; ++q) {
        const uint32_t bq = (base >> (16 * q)) & 0xFFFFu;
        if ((m[q] >> lane) & 1ull) list_lds[q][bq + (uint32_t)__popcll(m[q] & below)] = (uint16_t)n;
      }
    }
    __syncthreads();  // A: the lists
    const uint32_t ln = list_n;
    const int nl0 = (int)(ln & 0xFFFFu), nl1 = (int)(ln >> 16);
    // the draw wave completes the candidates of the pass at t + S (against
    // this state; the commit below patches what it touches)
    if (wave == kDrawWave) draw(t + (uint64_t)S);
    // 2. score the listed pairs (those of the slot's minibatch) and keep each
    // pair's activation change for the commit
    for (int e = tid; e < nl0 + nl1; e += kOneThreads) {
      const int q = e < nl0 ? 0 : 1;
      const int sn = list_lds[q][e < nl0 ? e : e - nl0];
      const int eq = ent(t, q), k = q & (K - 1);
      const bool logit = cand_lds[eq][k].layer == L - 1;
      float w[CM];
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) w[cc] = wcol_lds[eq][k][cc];
      float da;
      const float dl = pair_change<CM, kOneThreads>(C, act, gamma, logit, zh_lds[q][sn],
                                                    aux_lds[eq][k].de, w, wcol_lds[eq][k],
                                                    wmax_lds[eq][k], ain_lds[q][sn], &pl_lds[sn],
                                                    y_lds[sn], da);
      if (in_subset(net, sub_lds[eq], sn)) dlp_lds[q][sn] = dl;
      da_lds[q][sn] = da;
    }
    __syncthreads();  // B
    // 3. the sample's slots summed over each wave in one order (and cleared)
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
      if (q < nq) {
        const float v = wave_sum_f32(dlp_lds[q][n]);
        dlp_lds[q][n] = 0.f;
        if (lane == 0) red_lds[wave][q] = v;
      }
    }
    if (tid == 0) list_n = 0;  // every thread has read the counts
    __syncthreads();  // C
    // every wave adds the 16 wave sums of each slot (fp64, lanes 16q ..
    // 16q + 15, one DPP order that leaves the same bits in every lane of the
    // row) and takes the same decision
    const double row = wave_row_sum_f64((lane >> 4) < nq ? (double)red_lds[lane & 15][(lane >> 4) & 1] : 0.0);
    double v = 0.0;
    bool pass = false;
    {
      const uint64_t u = (uint64_t)__double_as_longlong(row);
      const uint32_t lo0 = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 0);
      const uint32_t hi0 = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 0);
      const uint32_t lo1 = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 16);
      const uint32_t hi1 = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 16);
      const uint64_t w0 = ((uint64_t)hi0 << 32) | lo0, w1 = ((uint64_t)hi1 << 32) | lo1;
      v = __longlong_as_double((long long)(lane == 0 ? w0 : w1));
    }
    if (lane < nq) {
      const Aux& xq = aux_lds[ent(t, lane)][lane & (K - 1)];
      const bool valid = xq.valid != 0;
      v = valid ? v / count : __builtin_huge_val();
      pass = accepts(v, net.ties, xq.theta);
    }
    const uint64_t acc = __ballot(pass);
    const int qc = acc ? (int)__ffsll((unsigned long long)acc) - 1 : -1;
    // steps the pass resolves: up to the chosen slot's step, else all of them
    const int adv = (qc >= 0) ? (qc >> kshift) + 1 : (nq >> kshift);
    const uint64_t tn = t + (uint64_t)adv;
    // 4a. the next pass's rows: those requested for t + S, after this pass's
    // second step when only the first one resolved (K = 1)
    if (adv == S) {
#pragma unroll
      for (int q = 0; q < kSlots; ++q) {
        a_cur[q] = a_pre[q];
        z_cur[q] = z_pre[q];
      }
    } else {
      a_cur[0] = a_cur[1];
      z_cur[0] = z_cur[1];
      a_cur[1] = a_pre[0];
      z_cur[1] = z_pre[0];
    }
    // taken here, before the commit's stores: a copy placed after them would
    // wait for the stores too
#pragma unroll
    for (int q = 0; q < kSlots; ++q) asm volatile("" : "+v"(a_cur[q]), "+v"(z_cur[q]));
    if (wave == 0) {
      const uint64_t upto = (qc >= 0) ? ((2ull << qc) - 1ull) : ((1ull << nq) - 1ull);
      const uint64_t tie = __ballot(lane < nq && fabs(v) < 1e-6) & upto;
      if (lane == 0) {
        n_tie += (uint64_t)__popcll(tie);
        if (qc >= 0) {
          const uint64_t u = (uint64_t)__double_as_longlong(v);
          const uint64_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), qc);
          const uint64_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, qc);
          if (net.sub_size == 0)  // a minibatch's change is not the loss's
            L_acc += __longlong_as_double((long long)((hi << 32) | lo));
          ++n_acc;
          n_waste += (uint64_t)(nq - ((qc >> kshift) + 1) * K);  // scored past the chosen step
        }
        last_k = (qc >= 0) ? (qc & (K - 1)) : -1;
      }
      if (a.tr_chosen != nullptr) {
        // the resolved steps in order; the ring of 64 steps goes out when
        // full and at the launch's end
        for (int i = 0; i < adv; ++i) {
          const uint64_t si = s + (uint64_t)i;
          const int r = (int)(si & (kTrace - 1));
          if (lane == 0) trc_lds[r] = (qc >= 0 && (qc >> kshift) == i) ? (qc & (K - 1)) : -1;
          if ((lane >> kshift) == i && lane < nq) trd_lds[r][lane & (K - 1)] = v;
          if (r == kTrace - 1 || si + 1 == a.n_steps) {
            const uint64_t base = si - (uint64_t)r;
            for (int e = lane; e <= r; e += 64)
              if ((int64_t)(base + e) < a.tr_cap) a.tr_chosen[base + e] = trc_lds[e];
            if (a.tr_dl != nullptr)
              for (int e = lane; e < (r + 1) * K; e += 64) {
                const int mm = e >> kshift, k = e & (K - 1);
                if ((int64_t)(base + mm) < a.tr_cap)
                  a.tr_dl[(int64_t)(base + mm) * K + k] = trd_lds[mm][k];
              }
          }
        }
      }
    }
    // 4b. the commit: the chosen slot's listed pairs with the scoring's
    // expressions; the draw wave writes the weight and patches the completed
    // candidates of the later steps that the commit touches
    lc_layer = -1;
    lc_moved = false;
    if (qc >= 0) {
      const int ec = ent(t, qc), kc = qc & (K - 1);
      const mca_cand c = cand_lds[ec][kc];
      const Aux x = aux_lds[ec][kc];
      const bool chid = c.layer == L - 2;
      if (wave == kDrawWave) {
        const int64_t idx = (int64_t)c.j * net.widths[c.layer] + c.i;
        if (lane == 0) {
          w_lds[woff(c.layer) + idx] = x.w_new;
          c_lds[woff(c.layer) + idx] = (int8_t)c.code;
        }
        // lane l: candidate l & (K - 1) of step t + (l >> kshift), for the
        // steps after the chosen one that are already completed
        const int d = lane >> kshift, k = lane & (K - 1);
        const uint64_t step = t + (uint64_t)d;
        if (lane < 2 * kSlots && d > (qc >> kshift) && step < t_end) {
          const int e = (int)(step & (kAhead - 1));
          const mca_cand dc = cand_lds[e][k];
          if (dc.layer == c.layer && dc.j == c.j && dc.i == c.i) {
            // the same parameter: completed again from the committed value
            mca_cand cn = ring_lds[step & (kRing - 1)][k];
            if (net.ternary) finish_ternary(net, cn, c.code);
            if (cn.flags & MCA_CAND_PRUNE) {
              cn.code = 0;
              cn.d = 0.0f - x.w_new;
            }
            Aux xn = aux_lds[e][k];
            xn.w_old = x.w_new;
            xn.w_new = (cn.flags & MCA_CAND_PRUNE) ? 0.0f
                       : (net.ternary ? (float)cn.code * net.scales[cn.layer] : x.w_new + cn.d);
            xn.de = xn.w_new - xn.w_old;
            xn.valid = !(net.bound > 0.f && fabsf(xn.w_new) >= net.bound);
            cand_lds[e][k] = cn;
            aux_lds[e][k] = xn;
          }
          if (c.layer == L - 1 && dc.layer == L - 2 && dc.j == c.i) {
            // a logit weight of the hidden unit's column
            wcol_lds[e][k][c.j] = x.w_new;
            float wm = 0.f;
#pragma unroll
            for (int cc = 0; cc < CM; ++cc) wm = fmaxf(wm, fabsf(wcol_lds[e][k][cc]));
            wmax_lds[e][k] = wm;
          }
        }
      }
      const int nlc = qc == 0 ? nl0 : nl1;
      for (int e = tid; e < nlc; e += kOneThreads) {
        const int sn = list_lds[qc][e];
        const float ain = ain_lds[qc][sn];
        const float z_raw = zh_lds[qc][sn];
        const float da = da_lds[qc][sn];  // the scoring's dphi(z, de ain), or de ain
        const float zn = z_raw + x.de * ain;
        if (chid) {
          gstore(&z_hid[(int64_t)c.j * Ns + sn], zn);
          zrow_lds[sn] = zn;
        }
        float wc[CM], zc[CM], z[CM], p[CM];
#pragma unroll
        for (int cc = 0; cc < CM; ++cc) {
          wc[cc] = wcol_lds[ec][kc][cc];
          zc[cc] = zl_lds[cc * kOneThreads + sn];
        }
        moved_logits<CM>(C, da, wc, zc, z);
        (void)softmax_ce<CM>(z, C, y_lds[sn], p);
#pragma unroll
        for (int cc = 0; cc < CM; ++cc) {
          zl_lds[cc * kOneThreads + sn] = z[cc];
          pl_lds[cc * kOneThreads + sn] = p[cc];
        }
      }
      lc_layer = c.layer;
      lc_j = c.j;
      lc_moved = chid && live && ain_lds[qc][n] != 0.f;  // this sample's field moved
      // the weight's HBM copy last: nothing in this pass waits for the store;
      // a wave other than the draw wave (whose patch ends the commit) makes it
      if (wave == kStoreWave && lane == 0) {
        const int64_t idx = (int64_t)c.j * net.widths[c.layer] + c.i;
        gstore(&net.W[c.layer][idx], x.w_new);
        if (net.ternary) gstore(&net.codes[c.layer][idx], (int8_t)c.code);
      }
    }
    __syncthreads();  // D
    t = tn;
  }

  // the logits and softmax go back to HBM with the losses of the final
  // logits; thread 0 writes the state
  if (live) {
    float z[CM], p[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) z[c] = zl_lds[c * kOneThreads + n];
    const float ln = softmax_ce<CM>(z, C, y_lds[n], p);
    for (int c = 0; c < C; ++c) {
      gstore(&net.Z[L - 1][(int64_t)c * Ns + n], z[c]);
      gstore(&net.prob[(int64_t)c * Ns + n], pl_lds[c * kOneThreads + n]);
    }
    gstore(&net.ell[n], ln);
  }
  if (tid == 0) {
    DevState* st = a.st;
    st->L = L_acc;
    st->t = t_end;
    st->steps += a.n_steps;
    st->evaluated += a.n_steps * (uint64_t)K;
    st->accepted = n_acc;
    st->wasted = n_waste;
    st->tie = n_tie;
    st->chosen = last_k;
  }
}

}  // namespace

bool one_loop_fits(const NetDev& net, int K) {
  if (net.L < 1 || net.L > 2) return false;
  const int64_t params = (net.L == 2 ? (int64_t)net.widths[1] * net.widths[0] : 0) +
                         (int64_t)net.widths[net.L] * net.widths[net.L - 1];
  return net.N <= kOneMaxSamples && K >= 1 && K <= kOneMaxK && net.C <= kOneCM &&
         params <= kOneMaxParams;
}

hipError_t launch_one_loop(const OneArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_one_loop, dim3(1), dim3(kOneThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace mca
