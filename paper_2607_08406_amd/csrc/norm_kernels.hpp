// Deep nets with biases and normalized hidden fields (norm_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

// Per-sample statistics of each normalized hidden layer: the mean MU[l][n]
// and S[l][n] = var + eps of sample n's fields z_l[:, n] (null where a layer
// is not normalized).
struct NormDev {
  float* MU[MCA_MAX_LAYERS];
  float* S[MCA_MAX_LAYERS];
};

inline bool norm_width_ok(int w) { return w == 256 || w == 512 || w == 1024; }
// Samples per block: one LDS tile of changes is [T][W + 4] floats.
inline int norm_tile(int w) { return 16384 / w; }
inline int norm_tiles(int64_t n_samples, int w) {
  const int T = norm_tile(w);
  return (int)((n_samples + T - 1) / T);
}

// MU[l], S[l] of hidden layer l from the cached fields Z[l].
hipError_t launch_norm_stats(const NetDev& net, const NormDev& nd, int l, hipStream_t s);
// k_mode -2: partial[k * ntiles + tile] for every candidate k < K; -1: commit
// st->chosen (nothing when -1); >= 0: commit that candidate.  A commit moves
// every cached field and statistic and writes the parameter, the loss and
// the count.
hipError_t launch_norm(const NetDev& net, const NormDev& nd, const mca_cand* cands,
                       const Aux* aux, int K, float* partial, int ntiles, int k_mode,
                       DevState* st, const double* dL, hipStream_t s);

}  // namespace mca
