// The decoder Transformer of Sec. 2.5 on the device: its description, and the host-side launchers of its kernels
// (implemented in tf_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "device_common.hpp"
#include "mca.h"

namespace mca {

constexpr int kTfMaxTensors = 64;
constexpr int kTfHeadDim = 32;    // d_model / n_head
constexpr int kTfMaxCtx = 128;    // positions per sequence (one attention block)
constexpr int kTfMaxVocab = 128;
constexpr int kTfMaxBlocks = 8;

// The tensors of one block, in canonical order after tok_emb and pos_emb.
enum TfRole {
  kLn1G, kLn1B, kWq, kBq, kWk, kBk, kWv, kBv, kWo, kBo,
  kLn2G, kLn2B, kWfc, kBfc, kWproj, kBproj, kBlockTensors
};

// Everything the kernels need, in device memory (passed by pointer).
// Stages: 0 the embedding (writes x_0), b+1 block b (x_b -> x_{b+1}),
// NB+1 the final LayerNorm, output layer and loss.  Activations are
// position-major [N][width], N = S * T positions.
struct TfDev {
  int32_t V, T, D, NB, H, M, S;   // vocab, ctx, d_model, blocks, heads, d_mlp, sequences
  int32_t n_tensors;
  int64_t N, P;                   // positions, parameters
  float eps, delta, bound;
  int32_t ties;
  uint64_t seed, tag;
  double beta;                    // Metropolis selection intensity
  int32_t rule;                   // MCA_RULE_*
  int32_t pad0;
  int64_t offs[kTfMaxTensors + 1];   // flat offset of each tensor, offs[n_tensors] = P
  int32_t rows[kTfMaxTensors], cols[kTfMaxTensors];  // 1-D tensors: cols = 1
  float* param[kTfMaxTensors];       // committed tensors
  const int32_t* tok;                // [N] input symbols
  const int32_t* tgt;                // [N] next-symbol targets
  float* x[kTfMaxBlocks + 1];        // committed residual streams x_0 .. x_NB
  float* ell;                        // committed per-position losses
  // per-candidate slots
  float* sx;      // [K][NB+1][N][D] the candidate's residual streams
  float* sh;      // [K][N][D] after attention
  float* sln;     // [K][N][D] LayerNorm output
  float* sqkv;    // [K][N][3D]
  float* satt;    // [K][N][D]
  float* sfc;     // [K][N][max(M, V)] MLP hidden / logits
  float* sell;    // [K][N] the candidate's per-position losses
  float* scopy;   // [K][copy_stride] private copy of the mutated tensor
  int64_t copy_stride;
  float** table;  // [K][n_tensors] tensor pointers per candidate
  int32_t* start; // [K] first stage the candidate changes (NB+2: not evaluated)
};

// Stage of tensor t.
__host__ __device__ inline int tf_stage(int t, int NB) {
  if (t < 2) return 0;
  if (t < 2 + kBlockTensors * NB) return 1 + (t - 2) / kBlockTensors;
  return NB + 1;
}

// GEMM roles inside a stage.
enum TfGemmRole { kGemmQKV, kGemmO, kGemmFc, kGemmProj, kGemmOut };

// Candidates k < K of step t (t from st->t when use_dev_t): records and new values.
hipError_t tf_launch_propose(const TfDev* tf, const TfDev& h, uint64_t t, bool use_dev_t,
                             const DevState* st, int K, mca_cand* cands, Aux* aux,
                             hipStream_t s);
// New values of given candidate records (explicit evaluation).
hipError_t tf_launch_prepare(const TfDev* tf, const mca_cand* cands, int K, Aux* aux,
                             hipStream_t s);
// Every stage of every candidate's forward pass from its first changed stage,
// and the tile sums of its per-position loss changes: partial[k * nblk + b].
// K = 0 with `identity` runs one unmutated pass in slot 0 (cache fill).
hipError_t tf_launch_eval(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                          const Aux* aux, int K, bool identity, float* partial, int nblk,
                          hipStream_t s);
// Commit candidate k (k < 0: st->chosen) from its slot into the committed
// state; `fill` copies slot 0 of an identity pass instead and sets the loss.
hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, hipStream_t s);
int tf_loss_blocks(int64_t N);

}  // namespace mca
