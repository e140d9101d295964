// Host-side launchers of the channel-mutation kernels (channel_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

// Hidden widths the channel kernels take (every hidden layer the same).
inline bool channel_width_ok(int w) { return w == 256 || w == 512 || w == 1024; }
// Samples per block: one LDS tile of changes is [T][W + 4] floats (66 KB).
inline int channel_tile(int w) { return 16384 / w; }
inline int channel_tiles(int64_t n_samples, int w) {
  const int T = channel_tile(w);
  return (int)((n_samples + T - 1) / T);
}

// Draws channels k = 0..K-1 of step t (use_dev_t: st->t) into ch, with
// their acceptance data in aux and a placeholder record per candidate in
// cands (the shared selection reads one).
hipError_t launch_channel_propose(const NetDev& net, uint64_t t, bool use_dev_t,
                                  const DevState* st, int K, mca_channel* ch, mca_cand* cands,
                                  Aux* aux, hipStream_t s);
// The same acceptance data for K channels given by the caller (threshold 0).
hipError_t launch_channel_prepare(const NetDev& net, const mca_channel* ch, int K,
                                  mca_cand* cands, Aux* aux, hipStream_t s);
// k_mode -2: partial[k * ntiles + tile] for every channel k < K; -1: commit
// st->chosen (nothing when -1); >= 0: commit that channel.  A commit moves
// every cached field and writes the path's weights, the loss and the count.
hipError_t launch_channel(const NetDev& net, const mca_channel* ch, const Aux* aux, int K,
                          float* partial, int ntiles, int k_mode, DevState* st,
                          const double* dL, hipStream_t s);

}  // namespace mca
