// Host-side launchers of the MLP kernels (implemented in mlp_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "device_common.hpp"
#include "norm_kernels.hpp"

namespace mca {

hipError_t launch_propose(const NetDev& net, uint64_t t, bool use_dev_t, const DevState* st,
                          int K, mca_cand* cands, Aux* aux, const uint64_t* fmask,
                          uint64_t* cmask, hipStream_t s);
// fmask (may be null): per input feature, bit b set when tile b of the
// batched evaluation holds a non-zero input sample; cmask[k] receives
// candidate k's tiles that can change (all ones but for first-layer weights).
hipError_t launch_prepare(const NetDev& net, const mca_cand* cands, int K, Aux* aux,
                          const uint64_t* fmask, uint64_t* cmask, hipStream_t s);
// Tiles of the batched evaluation for n samples; launch_eval writes
// partial[k * ntiles + tile] for the candidates in the last two layers.
int eval_tiles(int64_t n_samples);
int eval_tile_size();
hipError_t launch_eval(const NetDev& net, const mca_cand* cands, const Aux* aux,
                       const uint64_t* cmask, int K, float* partial, int ntiles,
                       const DevState* st, hipStream_t s);
hipError_t launch_select(const NetDev& net, const float* partial, int ntiles,
                         const mca_cand* cands, const float* pslab, int nslab,
                         const float* pchain, int nchain, const Aux* aux, int K, double* dL,
                         DevState* st, bool do_select, int32_t* tr_chosen, double* tr_dl,
                         int64_t tr_cap, hipStream_t s);
hipError_t launch_commit(const NetDev& net, const mca_cand* cands, const Aux* aux,
                         const double* dL, DevState* st, int k_host, int ntiles, hipStream_t s);
// The committed loss from the cached logits (the losses and softmax cached
// from them again): with a minibatch the loss is not the sum of the changes.
hipError_t launch_loss_refresh(const NetDev& net, double* bsum, DevState* st, hipStream_t s);
hipError_t launch_forward(const NetDev& net, double* bsum, DevState* st, hipStream_t s);
// The forward pass of a net with biases and / or normalized hidden fields.
hipError_t launch_forward_norm(const NetDev& net, const NormDev& nd, double* bsum, DevState* st,
                               hipStream_t s);

}  // namespace mca
