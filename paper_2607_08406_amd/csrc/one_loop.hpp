// One-workgroup step loop for small MLPs (implemented in one_loop.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

constexpr int kOneMaxSamples = 1024;  // one sample per thread of the workgroup
constexpr int kOneMaxK = 2;           // candidates per step
constexpr int kOneMaxParams = 3072;   // weights kept in LDS

struct OneArgs {
  NetDev net;
  int K;                // candidates per step (<= kOneMaxK)
  uint64_t n_steps;     // steps in this launch; the first is st->t
  DevState* st;
  int32_t* tr_chosen;   // trace (nullable): slot s = this launch's step s
  double* tr_dl;        // trace of every dL (nullable)
  int64_t tr_cap;
};

// Whether the one-workgroup loop takes this net and batch: one or two
// layers, N <= kOneMaxSamples, K <= kOneMaxK, at most 10 classes and
// kOneMaxParams weights.
bool one_loop_fits(const NetDev& net, int K);
hipError_t launch_one_loop(const OneArgs& a, hipStream_t s);

}  // namespace mca
