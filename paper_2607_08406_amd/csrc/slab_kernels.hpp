// Host-side launchers of the first-layer kernels of three-layer MLPs
// (implemented in slab_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"

namespace mca {

constexpr int kSlabMaxUnits = 1024;  // second-hidden-layer width the LDS tile holds

// Samples per block for a net with C classes.
int slab_tile(int C);

// k_mode -2: write partial[k * nblk + block] for every candidate k in layer
// L-3 (others untouched); -1: commit st->chosen if it is in layer L-3;
// >= 0: commit that candidate if it is in layer L-3.  cols (k_max * n_2
// entries) and nnz (k_max) are scratch for the candidates' column lists.
// `listed`: the column lists are already built (launch_propose_columns).
// `columns`: a commit also applies a winner of the last two layers (then
// k_commit_column is not launched); nblk blocks must cover every sample.
hipError_t launch_slab(const NetDev& net, const mca_cand* cands, const Aux* aux, int K,
                       uint64_t* cols, int* nnz, float* partial, int nblk, int k_mode, DevState* st,
                       const double* dL, hipStream_t s, bool listed = false,
                       bool columns = false);

// The proposal of step st->t (as launch_propose with the device's step) fused
// with the column lists of its layer L-3 candidates, for nets with L >= 3.
hipError_t launch_propose_columns(const NetDev& net, const DevState* st, int K, mca_cand* cands,
                                 Aux* aux, const uint64_t* fmask, uint64_t* cmask,
                                 uint64_t* cols, int* nnz, hipStream_t s);

// dst[c][r] = src[r][c] for a rows x cols matrix.
hipError_t launch_transpose(const float* src, int rows, int cols, float* dst, hipStream_t s);

}  // namespace mca
