// Persistent cooperative step loop (loop_kernel.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

constexpr int kLoopMaxK = 64;  // candidates per step in the persistent loop
#ifndef MCA_LOOP_REPLICAS
#define MCA_LOOP_REPLICAS 32
#endif
constexpr int kLoopReplicas = MCA_LOOP_REPLICAS;  // copies of each published loss change (<= 64)

// Abort word of the step loop, on its own 256-byte line.
struct LoopSync {
  uint32_t abort;      // set when a bounded wait ran out
  uint32_t pad[63];
};

struct LoopArgs {
  NetDev net;
  int K;                // candidates per step (<= kLoopMaxK)
  int T;                // samples per workgroup tile (<= 64)
  int G;                // tile workgroups (<= kLoopMaxTiles)
  int gpad;             // words per candidate row of partials: G rounded up to 16
  uint64_t n_steps;     // steps in this launch (< 2^32); the first is st->t
  uint64_t* partials;   // [2][K][gpad] tagged per-tile loss-change sums, by step parity
  uint64_t* dls;        // [kLoopReplicas][kLoopMaxK] tagged loss changes
  LoopSync* sync;
  DevState* st;
  int32_t* tr_chosen;   // trace (nullable): slot s = this launch's step s
  double* tr_dl;        // trace of every dL (nullable)
  int64_t tr_cap;
  uint32_t spin_limit;  // polls before a wait gives up and aborts the grid
};

constexpr int kLoopMaxTiles = 64 * 4;  // one workgroup per CU: at most the CU count

// Workgroups of the candidate reducers for K candidates (four candidates each).
int step_loop_reducers(int K);
// Clears the exchange words before each launch; snap non-null (a call's first
// launch): also snapshots the counters into snap and clears the abort word.
hipError_t launch_loop_reset(const LoopArgs& a, DevState* snap, hipStream_t s);
// The loop kernel alone (its words cleared by launch_loop_reset first).
hipError_t launch_step_loop(const LoopArgs& a, bool cooperative, hipStream_t s);
hipError_t step_loop_max_blocks(int K, int C, int* out);

}  // namespace mca
