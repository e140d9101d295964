// Persistent step loop for MLPs whose mutations touch only the last two
// layers (one hidden layer, or a logit-layer weight): one cooperative launch
// runs many steps of propose -> evaluate -> select -> commit.
//
// Work split: tile workgroup g < G owns T <= 64 consecutive samples for the
// whole launch.  Its share of the logits, their softmax and the labels stays
// in LDS (a pair's loss change is formed from its logit change and the
// softmax, pair_change; the per-sample losses are recomputed from the final
// logits when the launch ends); the hidden local fields Z_l stay in HBM but each tile of a row
// is only ever read and written by its owner.  Every tile workgroup decodes
// the step's K candidates itself (the stream is counter-based), scores all of
// them on its tile and publishes one partial loss change per candidate
// (+inf for a candidate rejected by the weight bound).  The reduction is
// sharded by candidate: wave w < 4 of reducer workgroup r owns candidate 4r + w,
// adds its G partial sums in a fixed order (fp64) and publishes the loss
// change dL_k.  Wave 0 of every tile workgroup reads the loss changes of the
// candidates up to the first that passes the test (Eq. 6) and takes the same
// decision itself: that candidate.  It then applies the commit to its own
// tile with the same expressions the evaluation used.  Tile 0 also keeps the
// committed loss and the counters.  While wave 0 waits for the loss changes,
// the other waves work ahead (the draw needs no state): wave 1 draws the
// candidates of step s+3, the staging waves write the operands and weights of
// step s+1 to a second LDS buffer, list its pairs and start the loads of step
// s+2.  The commit made after those loads were issued (one hidden row of the
// tile, one weight, code or logit-layer column entry) is applied at landing;
// the commit of the step just before, by wave 0 right after it commits, in
// the rare case that it touches a candidate.  A step thus takes two
// workgroup barriers: after the scoring, and at its end.
//
// Sparse inputs: a sample whose input to the mutated weight is zero does not
// change (about 81 % of an image column), so the (candidate, sample) pairs
// with a non-zero input are compacted into an LDS work list, which the whole
// workgroup then shares out over its lanes.  Each pair writes its loss change to
// its own (candidate, sample) slot and the slots are summed in sample order,
// so the order in which the list was built does not change any result.
//
// Weights are read with ordinary cached loads.  Every tile workgroup writes
// every committed weight itself, so each CU's L1 and each XCD's L2 that may
// hold the old value is updated by a local store; wave 0 waits for its
// commit stores during the next step, before any wave issues loads again, and
// until then the value comes from LDS.
//
// Cross-workgroup words carry their own step tag, so no separate flag, fence
// or L2 writeback is needed: a partial sum is one 64-bit word (fp32 value |
// 32-bit step tag), stored candidate-major so a reducer polls one candidate's
// G contiguous words, in one of two sets by step parity; a loss change is one
// fp64 word whose 16 low
// mantissa bits are replaced by the step tag (2^-36 relative truncation, the
// same bits for every reader).  They are written and read with relaxed
// agent-scope atomics, which the compiler emits as coherent (sc1) accesses.
// A reader polls until the tag is the one it expects.  Tags are cleared
// before each launch.
//
// Every wait is bounded: a spin that exceeds its limit raises an abort flag
// that all other waits observe, so the grid always drains.
#include "device_common.hpp"
#include "loop_kernel.hpp"

namespace mca {

namespace {

constexpr int kWaves = 16;  // 1024 threads: four waves per SIMD hide the list's latencies
constexpr int kLoopThreads = 64 * kWaves;
constexpr int kReducerWaves = 4;      // candidates per reducer workgroup
constexpr int kMaxTilesPerLane = kLoopMaxTiles / 64;
constexpr int kPollWindow = 16;  // candidates a tile polls first
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <class T>
__device__ __forceinline__ T ld_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <class T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// wait until every memory operation this wave issued has completed
__device__ __forceinline__ void wait_own_memory() { __builtin_amdgcn_s_waitcnt(0); }

__device__ __forceinline__ uint64_t pack(float v, uint32_t tag) {
  return ((uint64_t)__float_as_uint(v) << 32) | tag;
}
// 16-bit step tag of a loss-change word: 1..65535, never the cleared value 0,
// and different for consecutive steps.
__device__ __forceinline__ uint32_t tag16(uint64_t s) { return (uint32_t)(s % 65535u) + 1u; }
__device__ __forceinline__ uint64_t pack_dl(double v, uint32_t tag) {
  return ((uint64_t)__double_as_longlong(v) & ~0xFFFFull) | tag;
}
__device__ __forceinline__ double unpack_dl(uint64_t w) {
  return __longlong_as_double((long long)(w & ~0xFFFFull));
}

// Sum over the 64 lanes in one fixed order, the same bits in every lane: a
// butterfly within rows of 16 (DPP on both halves of the double; both lanes of
// a pair add the same two values, and after the quad steps the mirrored
// partners hold equal sums), then across the two rows of each half, then the
// two halves read into scalars and added once.
template <int kCtrl>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const int lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, kCtrl, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), kCtrl, 0xF, 0xF, true);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}
__device__ __forceinline__ double wave_sum_f64(double v) {
  v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]: lane ^ 1
  v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]: lane ^ 2
  v += dpp_f64<0x141>(v);  // row_half_mirror: lane 7 - i within eight
  v += dpp_f64<0x140>(v);  // row_mirror: lane 15 - i within sixteen
  v += __shfl_xor(v, 16, 64);
  const uint64_t u = (uint64_t)__double_as_longlong(v);
  const uint64_t a0 = ((uint64_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 0) << 32) |
                      (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 0);
  const uint64_t a1 = ((uint64_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 32) << 32) |
                      (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 32);
  return __longlong_as_double((long long)a0) + __longlong_as_double((long long)a1);
}

// Bounded spin helper: returns true when the grid must abort.
__device__ __forceinline__ bool spin_step(uint32_t& spins, const LoopArgs& a) {
  ++spins;
  if ((spins & 255u) == 0u && ld_agent(&a.sync->abort) != 0u) return true;
  if (spins > a.spin_limit) {
    st_agent(&a.sync->abort, 1u);
    return true;
  }
  __builtin_amdgcn_s_sleep(1);
  return false;
}

// A committed mutation, kept in LDS for two steps.
struct LastCommit {
  int layer, j, i, code;
  float w_new;
  int valid;
};

// A candidate's new value against the committed weights, with its new code.
struct Prep {
  float w_old, w_new;
  float de;    // fl32(w_new - w_old): the increment the caches apply
  int valid;   // 0: |w_new| >= bound, rejected without evaluation
  int code;    // new ternary code
  int pad[3];
};

// c.code holds the selecting bit of a ternary draw (decode_index); w and cur
// are the committed weight and code.
__device__ __forceinline__ Prep make_prep(const NetDev& net, const mca_cand& c, float w, int cur) {
  Prep x;
  x.w_old = w;
  if (c.flags & MCA_CAND_PRUNE) {  // w' = 0 (Sec. 2.2)
    x.code = 0;
    x.w_new = 0.0f;
  } else if (net.ternary) {
    mca_cand t = c;
    finish_ternary(net, t, cur);
    x.code = t.code;
    x.w_new = (float)t.code * net.scales[c.layer];
  } else {
    x.code = 0;
    x.w_new = w + c.d;
  }
  x.de = x.w_new - x.w_old;
  x.valid = !(net.bound > 0.f && fabsf(x.w_new) >= net.bound);
  return x;
}

__device__ __forceinline__ float input_of(const NetDev& net, int layer, float a_raw) {
  return (layer == 0) ? a_raw : act_fn(a_raw, net.act, net.gamma);
}

}  // namespace

// CM = bound on the class count (a compile-time count for C = 10).
template <int CM>
__global__ __launch_bounds__(kLoopThreads) void k_step_loop(LoopArgs a) {
  __shared__ NetDev net;
  stage_net(net, a.net);
  // an earlier launch of this call gave up: nothing runs
  if (ld_agent(&a.sync->abort) != 0u) return;
  // the first step's index, from the committed state (every workgroup reads
  // it before tile 0 can write the next one: no step completes without all)
  const uint64_t t0 = a.st->t;
  __shared__ float zl_lds[CM * 64];  // logits, [class][sample]
  __shared__ float pl_lds[CM * 64];  // their softmax
  __shared__ int y_lds[64];
  __shared__ mca_cand cand_lds[4][kLoopMaxK];  // draws of steps s .. s+3, by step mod 4
  __shared__ double theta_lds[4][kLoopMaxK];   // their acceptance thresholds (Eq. 7; 0 greedy)
  // each draw's row offsets in the unit-major arrays (elements): its input
  // row and, for a hidden unit, its field row (row 0 otherwise)
  __shared__ uint2 soff_lds[4][kLoopMaxK];
  __shared__ Prep prep_lds[2][kLoopMaxK];       // staged per step parity
  __shared__ float wcol_lds[2][kLoopMaxK][CM];  // logit-layer column (one-hot for a logit weight)
  __shared__ float wmax_lds[2][kLoopMaxK];      // max |column entry|
  __shared__ float ain_lds[2][kLoopMaxK][64];  // staged per step parity
  __shared__ float zh_lds[2][kLoopMaxK][64];
  // per-pair loss changes, [candidate][sample]; rows of 68 floats keep every
  // row 16-byte aligned and a 16-byte read of the same column by 16 lanes
  // (rows k .. k+15) conflict-free
  __shared__ __attribute__((aligned(16))) float dlp_lds[kLoopMaxK][68];
  __shared__ uint16_t list_lds[2][kLoopMaxK * 64];  // work lists, by step parity
  __shared__ int list_n[2];
  __shared__ uint32_t stage_cnt;  // waves 1-15 that have landed a step (15 per step)
  __shared__ LastCommit last[2];     // commits of the last two steps, by step parity
  __shared__ float zrow_lds[2][64];  // their committed hidden rows of this tile
  __shared__ int aborted;

  const int K = a.K, T = a.T, G = a.G;
  const int g = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // the CM < kCMax variants run only for C == CM: a compile-time class count
  const int C = (CM < kCMax) ? CM : net.C, L = net.L;
  const int act = net.act;
  const float gamma = net.gamma;
  if (tid == 0) aborted = 0;

  if (g >= G) {
    // ---------------------------------------------------- candidate reducers
    // Waves 0-3 of each reducer workgroup own one candidate each (one wave
    // per SIMD: a single polling wave per SIMD is not starved by the issue
    // priority of older waves); the other waves have nothing to do.
    if (wave >= kReducerWaves) return;  // no block barrier follows in the reducers
    const int k = (g - G) * kReducerWaves + wave;
    if (k >= K) return;
    for (uint64_t s = 0; s < a.n_steps; ++s) {
      // candidate-major: G words of step s's set
      const uint64_t* mine = a.partials + ((s & 1) * (size_t)K + (size_t)k) * a.gpad;
      const uint32_t tag = (uint32_t)(s + 1);
      // lane l adds tiles l, l+64, ... in that order
      uint64_t w[kMaxTilesPerLane];
#pragma unroll
      for (int b = 0; b < kMaxTilesPerLane; ++b) w[b] = 0;
      uint32_t spins = 0;
      bool fresh = false, ab = false;
      while (!fresh && !ab) {
        fresh = true;
#pragma unroll
        for (int b = 0; b < kMaxTilesPerLane; ++b) {
          const int gg = lane + 64 * b;
          if (gg < G && (uint32_t)w[b] != tag) w[b] = ld_agent(&mine[gg]);
        }
#pragma unroll
        for (int b = 0; b < kMaxTilesPerLane; ++b) {
          const int gg = lane + 64 * b;
          fresh = fresh && (gg >= G || (uint32_t)w[b] == tag);
        }
        fresh = __all(fresh);
        if (!fresh) ab = __any(spin_step(spins, a));
      }
      if (ab) return;
      double acc = 0.0;
#pragma unroll
      for (int b = 0; b < kMaxTilesPerLane; ++b)
        if (lane + 64 * b < G) acc += (double)__uint_as_float((uint32_t)(w[b] >> 32));
      const double tot = wave_sum_f64(acc);
      const uint64_t word = pack_dl(tot / subset_count(net), tag16(s));  // +inf: rejected
      if (lane < kLoopReplicas) st_agent(&a.dls[lane * kLoopMaxK + k], word);
    }
    return;
  }

  // ------------------------------------------------------------ tile workgroup
  const int64_t n = (int64_t)g * T + lane;
  const bool live = lane < T && n < net.N;
  const int nh = net.widths[L - 1];
  const int64_t Ns = net.Ns;
  // the tile's logits, softmax and labels move to LDS for the whole launch
  if (wave == 0) {
    for (int c = 0; c < CM; ++c) {
      zl_lds[c * 64 + lane] = (live && c < C) ? gload(&net.Z[L - 1][(int64_t)c * Ns + n]) : 0.f;
      pl_lds[c * 64 + lane] = (live && c < C) ? gload(&net.prob[(int64_t)c * Ns + n]) : 0.f;
    }
    y_lds[lane] = live ? gload(&net.y[n]) : 0;
  }
  if (tid < 2) last[tid].valid = 0;
  // committed scalars, carried in registers by tile 0, lane 0
  double L_acc = 0.0;
  uint64_t n_acc = 0, n_tie = 0;
  int last_k = -1;
  if (g == 0 && tid == 0) {
    L_acc = a.st->L;
    n_acc = a.st->accepted;
    n_tie = a.st->tie;
  }
  bool committed = false;  // this wave committed last step: its stores are in flight
  // The stream is drawn three steps ahead: wave 1, lane k decodes candidate
  // k of step t into cand_lds[t mod 4] (one Philox block per lane, so the
  // 64-bit multiplies of a draw cost one wave's issue time).  The operands of
  // a step are staged in two parts: the loads of step s+2 are issued during
  // step s into registers and land in LDS buffer (s+2) mod 2 during step s+1,
  // so their latency hides behind a whole step.  Landing applies the commit
  // made after the loads were issued; the commit of the step just before is
  // applied at the start of the step itself.
  //  - per candidate (wave 1, lane k): the weight, its code and, for a hidden
  //    unit, its logit-layer column; landing computes the new value (Prep);
  //  - per sample (waves 2-15, candidates k = w-2, w+12, ... of wave w, the
  //    candidate's fields in scalar registers): the input of the mutated weight
  //    and the cached local field of a mutated hidden unit.
  // The persistent loop runs L <= 2, so the layer pointers are taken from the
  // kernel argument with constant indices (scalar registers).
  const int Lk = a.net.L;
  const bool two = Lk == 2;
  const float* const in_hid = a.net.XT;                       // input of layer 0 (L = 2)
  const float* const in_log = two ? a.net.Z[0] : a.net.XT;    // input of the logit layer
  float* const z_hid = a.net.Z[0];                      // hidden local fields (L = 2)
  float* const w_log = two ? a.net.W[1] : a.net.W[0];
  int8_t* const c_log = two ? a.net.codes[1] : a.net.codes[0];
  const int nin_log = two ? a.net.widths[1] : a.net.widths[0];
  const int nin_hid = a.net.widths[0];
  const bool ternary = a.net.ternary != 0;
  constexpr int kStagers = kWaves - 2;
  constexpr int kPer = (kLoopMaxK + kStagers - 1) / kStagers;  // candidates per staging wave
  float a_raw[kPer], z_raw[kPer];  // per-sample loads in flight
  float w_reg = 0.f, col_reg[CM];  // per-candidate loads in flight (wave 1)
  int code_reg = 0;

#pragma unroll
  for (int cc = 0; cc < CM; ++cc) col_reg[cc] = 0.f;
  auto draw = [&](uint64_t t, int cb) {
    if (lane < K) {
      const mca_cand c = decode_index(net, t, (uint64_t)lane);
      cand_lds[cb][lane] = c;
      theta_lds[cb][lane] = accept_theta(net.rule, net.beta, net.seed, net.tag, t, (uint64_t)lane);
      const bool hid = c.layer == Lk - 2;
      soff_lds[cb][lane] = make_uint2((uint32_t)c.i * (uint32_t)Ns, hid ? (uint32_t)c.j * (uint32_t)Ns : 0u);
    }
  };
  auto issue_cand = [&](int cb) {
    if (lane < K) {
      const mca_cand c = cand_lds[cb][lane];
      const bool hid = c.layer == Lk - 2;
      const int64_t idx = (int64_t)c.j * (hid ? nin_hid : nin_log) + c.i;
      w_reg = gload(hid ? &a.net.W[0][idx] : &w_log[idx]);
      code_reg = ternary ? (int)gload(hid ? &a.net.codes[0][idx] : &c_log[idx]) : 0;
      // Every lane loads a column (a logit-layer candidate the first, unused:
      // landing makes its column one-hot at its logit).  A load under a
      // per-lane branch would make the other branch's write of the same
      // register wait for every load in flight.
      const int64_t jc = hid ? c.j : 0;
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) col_reg[cc] = (cc < C) ? gload(&w_log[(int64_t)cc * nh + jc]) : 0.f;
    }
  };
  // slot: the commit applied while landing
  auto land_cand = [&](int cb, int b, int slot) {
    if (lane < K) {
      const mca_cand c = cand_lds[cb][lane];
      const LastCommit lc = last[slot];
      float w = w_reg;
      int cur = code_reg;
      if (lc.valid && lc.layer == c.layer && lc.j == c.j && lc.i == c.i) {
        w = lc.w_new;
        cur = lc.code;
      }
      const bool hid = c.layer == Lk - 2;
      const bool colhit = lc.valid && lc.layer == Lk - 1 && hid && lc.i == c.j;
      float wm = 0.f;
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) {
        const float wv = !hid ? ((cc == c.j) ? 1.f : 0.f)
                              : ((colhit && cc == lc.j) ? lc.w_new : col_reg[cc]);
        wcol_lds[b][lane][cc] = wv;
        wm = fmaxf(wm, fabsf(wv));
      }
      wmax_lds[b][lane] = wm;
      prep_lds[b][lane] = make_prep(net, c, w, cur);
    }
  };
  // Lane q < kPer of a staging wave reads the layer, input and unit of the
  // wave's q-th candidate of draw buffer cb (one LDS round trip for all of
  // them); the wave then takes them into scalars lane by lane.
  auto stage_fields = [&](int cb, int& lv, int& iv, int& jv, uint32_t& io, uint32_t& zo) {
    const int kq = __builtin_amdgcn_readfirstlane(wave) - 2 + kStagers * lane;
    lv = -1;
    iv = jv = 0;
    io = zo = 0u;
    if (lane < kPer && kq < K) {
      const mca_cand c = cand_lds[cb][kq];
      const uint2 o = soff_lds[cb][kq];
      lv = c.layer;
      iv = c.i;
      jv = c.j;
      io = o.x;
      zo = o.y;
    }
  };
  // The lane's sample in each row array, as per-lane addresses (vector
  // registers): issuing a load then needs no scalar base pointer, which the
  // compiler would otherwise reload from the kernel arguments per candidate.
  // A dead lane (n >= N) points at sample 0 and its value is not used.
  const int64_t n_ld = live ? n : 0;
  const float* const in_hid_n = in_hid + n_ld;
  const float* const in_log_n = in_log + n_ld;
  const float* const z_hid_n = z_hid + n_ld;
  // Both rows of a candidate are loaded at the offsets its draw computed (a
  // logit-layer candidate's field row is row 0, unused), so issuing takes no
  // per-candidate address arithmetic on the scalar unit.
  auto issue_samples = [&](int cb) {
    const int w = __builtin_amdgcn_readfirstlane(wave) - 2;
    int lv, iv, jv;
    uint32_t io, zo;
    stage_fields(cb, lv, iv, jv, io, zo);
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int k = w + kStagers * q;
      a_raw[q] = 0.f;
      z_raw[q] = 0.f;
      if (k < K) {
        const bool hid = __builtin_amdgcn_readlane(lv, q) == Lk - 2;
        a_raw[q] = gload(&(hid ? in_hid_n : in_log_n)[(uint32_t)__builtin_amdgcn_readlane((int)io, q)]);
        z_raw[q] = gload(&z_hid_n[(uint32_t)__builtin_amdgcn_readlane((int)zo, q)]);
      }
    }
  };
  // Landing also lists the (candidate, sample) pairs of the wave's
  // candidates that can change: a non-zero input; for a logit-layer weight
  // fed by a hidden layer every live sample, since the commit of the step
  // before may still change that input (a pair whose input is zero adds
  // exactly 0).  Results do not depend on the order of the list.
  auto land_samples = [&](int cb, int b, int slot, uint64_t t_land) {
    const int w = __builtin_amdgcn_readfirstlane(wave) - 2;
    // the landed step's minibatch: only its samples are listed and scored
    const bool mem = in_subset(net, subset_start(net, t_land), n);
    // every LDS read of the landing is issued here, before any is used
    const LastCommit lc = last[slot];
    const float zrow_v = zrow_lds[slot][lane];
    int lv, iv, jv;
    uint32_t io, zo;
    stage_fields(cb, lv, iv, jv, io, zo);
    const bool row = lc.valid && lc.layer == Lk - 2;  // a hidden row of this tile changed
    // per candidate (lane q): a hidden-unit weight; its field row, or its
    // input row, is the committed row
    const uint64_t hmask = __ballot(lv == Lk - 2);
    const uint64_t pz = __ballot(row && lv == Lk - 2 && jv == lc.j);
    const uint64_t pa = __ballot(row && lv == Lk - 1 && iv == lc.j);
    uint64_t m[kPer];
    int tot = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int k = w + kStagers * q;
      m[q] = 0;
      if (k < K) {
        const bool hid = (hmask >> q) & 1ull;
        const float zz = ((pz >> q) & 1ull) ? zrow_v : z_raw[q];
        const float ar = ((pa >> q) & 1ull) ? zrow_v : a_raw[q];
        // the logit layer's input is an activation when a hidden layer feeds it
        const float in = (!hid && two) ? act_fn(ar, act, gamma) : ar;
        ain_lds[b][k][lane] = live ? in : 0.f;
        zh_lds[b][k][lane] = zz;
        m[q] = __ballot(live && mem && (in != 0.f || (two && !hid)));
        tot += (int)__popcll(m[q]);
      }
    }
    int base = 0;
    if (lane == 0 && tot) base = atomicAdd(&list_n[b], tot);
    base = __shfl(base, 0, 64);
    const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      if ((m[q] >> lane) & 1ull)
        list_lds[b][base + (int)__popcll(m[q] & below)] = (uint16_t)(((w + kStagers * q) << 6) | lane);
      base += (int)__popcll(m[q]);
    }
  };
  // Waves 1-15 count the steps they have landed, so that wave 0 can patch a
  // landed step (rarely) once they are done with it.
  auto landed = [&]() {
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (lane == 0) atomicAdd(&stage_cnt, 1u);
  };

  if (tid < 2) list_n[tid] = 0;
  if (tid == 0) stage_cnt = 0;
  // pair slots start clear; after each step wave 0 clears those it summed
  for (int i = tid; i < kLoopMaxK * 68; i += kLoopThreads) (&dlp_lds[0][0])[i] = 0.f;
  // the first step's draw, its loads, and the next two draws while those
  // loads are in flight
  if (wave == 1) draw(t0, 0);
  __syncthreads();
  if (wave == 1) {
    issue_cand(0);
    for (uint64_t d = 1; d < 3 && d < a.n_steps; ++d) draw(t0 + d, (int)d);
    land_cand(0, 0, 1);
  } else if (wave >= 2) {
    issue_samples(0);
    land_samples(0, 0, 1, t0);
  }
  __syncthreads();
  if (a.n_steps > 1) {
    if (wave == 1) issue_cand(1);
    else if (wave >= 2) issue_samples(1);
  }

  // A step takes two workgroup barriers: after the scoring, and at its end,
  // when wave 0 has decided and committed and waves 1-15 have staged and
  // listed the next step.
  for (uint64_t s = 0; s < a.n_steps; ++s) {
    const uint32_t tag = (uint32_t)(s + 1);
    const int buf = (int)(s & 1);
    const int cb = (int)(s & 3);
    mca_cand* cands = cand_lds[cb];
    // 1. every lane of the workgroup scores list entries (the list of step s
    // was built during step s-1); the list of step s+1 starts empty
    const int n_list = list_n[buf];
    for (int e = tid; e < n_list; e += kLoopThreads) {
      const int code = list_lds[buf][e];
      const int k = code >> 6, sl = code & 63;
      const mca_cand& c = cands[k];
      float da, w[CM];
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) w[cc] = wcol_lds[buf][k][cc];
      dlp_lds[k][sl] = pair_change<CM>(C, act, gamma, c.layer == L - 1, zh_lds[buf][k][sl],
                                       prep_lds[buf][k].de, w, wcol_lds[buf][k], wmax_lds[buf][k],
                                       ain_lds[buf][k][sl], &pl_lds[sl], y_lds[sl], da);
    }
    if (tid == 0) list_n[buf ^ 1] = 0;
    // last step's commit stores land before this step's staging reads HBM
    if (committed) wait_own_memory();
    committed = false;
    __syncthreads();
    // 2. wave 0, lane k: sum candidate k's 64 slots (four runs of 16
    // consecutive samples in order, then the runs pairwise), publish the tile's
    // partial sum and clear the slots for the next step.  Only wave 0 stores
    // to global memory here: a store still in flight would make the staging
    // waves' waits for their own loads wait for it too.
    uint64_t* part = a.partials + (size_t)buf * K * a.gpad + g;  // candidate k: part[k * gpad]
    if (wave == 0 && lane < K) {
      // the row in two halves of eight 16-byte reads, each issued before its
      // first add
      const floatx4* row = reinterpret_cast<const floatx4*>(&dlp_lds[lane][0]);
      float r[4];
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        floatx4 q4[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) q4[i] = row[8 * half + i];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          float acc = 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc += q4[4 * h + i][t];
          r[2 * half + h] = acc;
        }
      }
      const float v = (r[0] + r[1]) + (r[2] + r[3]);
      st_agent(&part[(size_t)lane * a.gpad], pack(prep_lds[buf][lane].valid ? v : __builtin_huge_valf(), tag));
      const floatx4 zero4 = {0.f, 0.f, 0.f, 0.f};
      floatx4* wrow = reinterpret_cast<floatx4*>(&dlp_lds[lane][0]);
#pragma unroll
      for (int i = 0; i < 16; ++i) wrow[i] = zero4;
    }
    // 3. wave 1 draws step s+3, waves 2-15 land and list step s+1 and issue
    // step s+2
    if (wave == 1) {
      if (s + 1 < a.n_steps) land_cand((int)((s + 1) & 3), buf ^ 1, buf ^ 1);
      landed();
      if (s + 2 < a.n_steps) issue_cand((int)((s + 2) & 3));
      if (s + 3 < a.n_steps) draw(t0 + s + 3, (int)((s + 3) & 3));
    } else if (wave >= 2) {
      if (s + 1 < a.n_steps) land_samples((int)((s + 1) & 3), buf ^ 1, buf ^ 1, t0 + s + 1);
      landed();
      if (s + 2 < a.n_steps) issue_samples((int)((s + 2) & 3));
    }
    if (wave == 0) {
      // what the commit and the patch check need whichever candidate wins:
      // the lane's logits, this step's candidates with their new values and
      // the candidates of step s+1 (lane = candidate)
      float zc[CM];
#pragma unroll
      for (int cc = 0; cc < CM; ++cc) zc[cc] = zl_lds[cc * 64 + lane];
      mca_cand c0{}, c1{};
      Prep p0{};
      if (lane < K) {
        c0 = cands[lane];
        p0 = prep_lds[buf][lane];
        c1 = cand_lds[(s + 1) & 3][lane];
      }
      const uint32_t t16 = tag16(s);
      const double th = lane < K ? theta_lds[cb][lane] : 0.0;
      const uint64_t* dls = a.dls + (g % kLoopReplicas) * kLoopMaxK;
      uint64_t d = 0;
      uint32_t spins = 0;
      bool ab = false;
      // The decision needs the loss changes of candidates 0 .. kc only (kc
      // the first that passes, or all K when none does, or when every dL is
      // traced).  Before the set of step s-1 can be overwritten (next step),
      // every reducer must be done with it: its word carries the tag of step
      // s-1 or s.
      const uint32_t t16p = tag16(s + 65534u);  // tag of step s-1
      const bool need_all = g == 0 && a.tr_dl != nullptr;
      uint64_t fm = 0, am = 0;
      // Polls read the first kPollWindow candidates (one line of words) and
      // widen to all K only when those hold no improver; every lane reads
      // until its reducer is past step s-1.  Fewer coherent loads in flight
      // make each of them return sooner.
      int lim = need_all ? 64 : kPollWindow;
      while (true) {
        {
          const uint32_t tg0 = (uint32_t)(d & 0xFFFFu);
          if (lane < K && tg0 != t16 && (lane < lim || !(s == 0 || tg0 == t16p))) d = ld_agent(&dls[lane]);
        }
        const uint32_t tg = (uint32_t)(d & 0xFFFFu);
        const bool fresh = lane >= K || tg == t16;
        const bool done_prev = fresh || s == 0 || tg == t16p;
        fm = __ballot(fresh);
        am = __ballot(lane < K && tg == t16 && accepts(unpack_dl(d), net.ties, th));
        const int pre = (~fm) ? (int)__ffsll((unsigned long long)~fm) - 1 : 64;  // first stale
        const int fa = am ? (int)__ffsll((unsigned long long)am) - 1 : 64;
        if (__all(done_prev) && (pre >= 64 || (!need_all && fa < pre))) break;
        if (fa >= pre && pre >= lim) lim = 64;
        if ((ab = __any(spin_step(spins, a)))) break;
      }
      const double v = unpack_dl(d);
      const int kc = (!ab && am) ? (int)__ffsll((unsigned long long)am) - 1 : -1;
      // 4. commit on this tile (lane = sample; the winner's operands are
      // staged in LDS, its fields come from lane kc); every workgroup writes
      // the new weight.  The loop's layers are the last two, so the
      // destinations are the scalar pointers of the staging code.
      const int kq = kc >= 0 ? kc : 0;
      mca_cand c{};
      c.layer = __builtin_amdgcn_readlane(c0.layer, kq);
      c.j = __builtin_amdgcn_readlane(c0.j, kq);
      c.i = __builtin_amdgcn_readlane(c0.i, kq);
      Prep au{};
      au.de = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p0.de), kq));
      au.w_new = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(p0.w_new), kq));
      au.code = __builtin_amdgcn_readlane(p0.code, kq);
      const bool chid = c.layer == Lk - 2;  // the winner is a hidden-unit weight
      float zr = 0.f;  // the committed unit's row of this tile, lane = sample
      if (kc >= 0) {
        // the logits move by the activation change, by the scoring's
        // expressions (the same bits for a scored sample; a sample outside
        // the step's minibatch was not scored but moves all the same)
        const float ain = ain_lds[buf][kc][lane];
        const float z_raw = zh_lds[buf][kc][lane];
        const float dz0 = au.de * ain;
        const float da = chid ? dphi(z_raw, dz0, act, gamma) : dz0;
        float wc[CM];
#pragma unroll
        for (int cc = 0; cc < CM; ++cc) wc[cc] = wcol_lds[buf][kc][cc];
        const float zn = z_raw + au.de * ain;
        const bool ch = live && ain != 0.f;
        if (ch) {
          if (chid) gstore(&z_hid[(int64_t)c.j * Ns + n], zn);
          float z[CM], p[CM];
          moved_logits<CM>(C, da, wc, zc, z);
          (void)softmax_ce<CM>(z, C, y_lds[lane], p);
#pragma unroll
          for (int cc = 0; cc < CM; ++cc) {
            zl_lds[cc * 64 + lane] = z[cc];
            pl_lds[cc * 64 + lane] = p[cc];
          }
        }
        zr = ch ? zn : z_raw;
        zrow_lds[buf][lane] = zr;
        if (lane == 0) {
          const int64_t idx = (int64_t)c.j * (chid ? nin_hid : nin_log) + c.i;
          gstore(&(chid ? a.net.W[0] : w_log)[idx], au.w_new);
          if (ternary) gstore(&(chid ? a.net.codes[0] : c_log)[idx], (int8_t)au.code);
          LastCommit& lc = last[buf];
          lc.layer = c.layer;
          lc.j = c.j;
          lc.i = c.i;
          lc.code = au.code;
          lc.w_new = au.w_new;
          lc.valid = 1;
        }
        committed = true;
      } else if (lane == 0) {
        last[buf].valid = 0;
      }
      // 5. the commit may touch a candidate of step s+1 (its weight, its
      // unit's row of this tile, or its logit-layer column), which is rare:
      // once waves 1-15 have landed step s+1, patch it (lane = candidate for
      // its value and column, lane = sample for rows)
      if (kc >= 0 && s + 1 < a.n_steps) {
        bool row = false, same = false, col = false;
        if (lane < K) {
          const bool hid = c1.layer == L - 2;
          same = c.layer == c1.layer && c.j == c1.j && c.i == c1.i;
          col = c.layer == L - 1 && hid && c.i == c1.j;
          row = c.layer == L - 2 && ((hid && c1.j == c.j) || (c1.layer == L - 1 && c1.i == c.j));
        }
        if (__any(row || same || col)) {
          const uint32_t want = (uint32_t)(kWaves - 1) * (uint32_t)(s + 1);
          while (__hip_atomic_load(&stage_cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != want)
            __builtin_amdgcn_s_sleep(1);
          __asm__ volatile("" ::: "memory");
          if (same) prep_lds[buf ^ 1][lane] = make_prep(net, c1, au.w_new, au.code);
          if (col) {
            wcol_lds[buf ^ 1][lane][c.j] = au.w_new;
            float wm = 0.f;
#pragma unroll
            for (int cc = 0; cc < CM; ++cc) wm = fmaxf(wm, fabsf(wcol_lds[buf ^ 1][lane][cc]));
            wmax_lds[buf ^ 1][lane] = wm;
          }
          uint64_t rows = __ballot(row);
          while (rows) {
            const int k = (int)__ffsll((unsigned long long)rows) - 1;
            rows &= rows - 1;
            const int l = __shfl(c1.layer, k, 64);
            if (l == L - 2) zh_lds[buf ^ 1][k][lane] = zr;
            else ain_lds[buf ^ 1][k][lane] = live ? input_of(net, l, zr) : 0.f;
          }
        }
      }
      if (lane == 0) aborted = ab ? 1 : 0;
      // tile 0 keeps the committed loss, the counters and the trace
      if (g == 0 && !ab) {
        const uint64_t tie_mask = __ballot(lane < K && fabs(v) < 1e-6);
        const double vk = __shfl(v, kc < 0 ? 0 : kc, 64);
        if (lane == 0) {
          const uint64_t upto = (kc >= 0) ? ((kc == 63) ? ~0ull : ((2ull << kc) - 1ull)) : ~0ull;
          n_tie += (uint64_t)__popcll(tie_mask & upto);
          if (kc >= 0) {
            if (net.sub_size == 0) L_acc += vk;  // a minibatch's change is not the loss's
            ++n_acc;
          }
          last_k = kc;
        }
        if (a.tr_chosen != nullptr) {
          const int64_t slot = (int64_t)s;  // the trace chunk starts at this launch's first step
          if (slot < a.tr_cap) {
            if (lane == 0) a.tr_chosen[slot] = kc;
            if (a.tr_dl != nullptr && lane < K) a.tr_dl[slot * K + lane] = v;
          }
        }
      }
    }
    __syncthreads();
    if (aborted) break;
  }
  // the tile's logits and softmax go back to HBM with the losses of the
  // final logits; tile 0 writes the state
  if (wave == 0 && live) {
    float z[CM], p[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) z[c] = zl_lds[c * 64 + lane];
    const float ln = softmax_ce<CM>(z, C, y_lds[lane], p);
    for (int c = 0; c < C; ++c) {
      gstore(&net.Z[L - 1][(int64_t)c * Ns + n], z[c]);
      gstore(&net.prob[(int64_t)c * Ns + n], pl_lds[c * 64 + lane]);
    }
    gstore(&net.ell[n], ln);
  }
  if (g == 0 && tid == 0 && !aborted) {
    DevState* st = a.st;
    st->L = L_acc;
    st->t = t0 + a.n_steps;
    st->steps += a.n_steps;
    st->evaluated += a.n_steps * (uint64_t)K;
    st->accepted = n_acc;
    st->tie = n_tie;
    st->chosen = last_k;
  }
}

// Clears the tags before a launch (a fill kernel, so the sequence can be
// captured in a graph).  With snap given (the first launch of a call) it also
// records the counters the call's statistics are taken against and clears the
// abort word; later launches of the call keep it, so a launch after one that
// gave up sees it.
__global__ void k_reset_loop(uint64_t* partials, int64_t n_words, uint64_t* dls,
                             const DevState* st, DevState* snap, LoopSync* sync) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_words) partials[i] = 0;
  if (i < (int64_t)kLoopReplicas * kLoopMaxK) dls[i] = 0;
  if (snap != nullptr && i == 0) {
    *snap = *st;
    sync->abort = 0;
  }
}

namespace {
const void* pick_loop(int K, int C) {
  (void)K;
  return C == 10 ? (const void*)k_step_loop<10> : (const void*)k_step_loop<kCMax>;
}
}  // namespace

int step_loop_reducers(int K) { return (K + kReducerWaves - 1) / kReducerWaves; }

hipError_t launch_loop_reset(const LoopArgs& a, DevState* snap, hipStream_t s) {
  const int64_t words = 2 * (int64_t)a.K * a.gpad;
  const int64_t n = words > (int64_t)kLoopReplicas * kLoopMaxK ? words : (int64_t)kLoopReplicas * kLoopMaxK;
  hipLaunchKernelGGL(k_reset_loop, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                     a.partials, words, a.dls, a.st, snap, a.sync);
  return hipGetLastError();
}

hipError_t launch_step_loop(const LoopArgs& a, bool cooperative, hipStream_t s) {
  // G tile workgroups and the candidate reducers; every workgroup must be
  // resident at once (the caller checked the occupancy).  The cooperative
  // launch has the runtime guarantee it; the ordinary one relies on the
  // check and on the bounded waits (a workgroup that never starts makes the
  // others give up and abort, never hang).
  const dim3 grid(a.G + step_loop_reducers(a.K));
  if (!cooperative) {
    if (a.net.C == 10)
      hipLaunchKernelGGL(k_step_loop<10>, grid, dim3(kLoopThreads), 0, s, a);
    else
      hipLaunchKernelGGL(k_step_loop<kCMax>, grid, dim3(kLoopThreads), 0, s, a);
    return hipGetLastError();
  }
  void* args[] = {(void*)&a};
  return hipLaunchCooperativeKernel(pick_loop(a.K, a.net.C), grid, dim3(kLoopThreads), args, 0, s);
}

hipError_t step_loop_max_blocks(int K, int C, int* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  int per_cu = 0, cus = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, pick_loop(K, C), kLoopThreads, 0);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  *out = per_cu * cus;
  return hipSuccess;
}

}  // namespace mca
