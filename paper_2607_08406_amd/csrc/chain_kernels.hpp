// Host-side launcher of the deep-layer kernels (implemented in
// chain_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

constexpr int kChainT = 64;       // listed samples per block
constexpr int kChainUnits = 256;  // width every hidden layer of a deep net must have

// k_mode -2: write partial[k * nchain + tile] for every candidate k in layers
// 0..L-4 (others untouched); -1: commit st->chosen if it is in those layers;
// >= 0: commit that candidate if it is.  rows, rda (k_max * N) and cnt (k_max)
// are scratch for the lists of affected samples; nchain = ceil(N / kChainT).
hipError_t launch_chain(const NetDev& net, const mca_cand* cands, const Aux* aux, int K,
                        int* rows, float* rda, int* cnt, float* partial, int nchain, int k_mode,
                        DevState* st, const double* dL, hipStream_t s);

}  // namespace mca
