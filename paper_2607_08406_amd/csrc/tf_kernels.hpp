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
  // committed intermediate fields, kept for the incremental evaluation of
  // the MLP, final-LayerNorm and output-layer parameters
  float* ch[kTfMaxBlocks];           // [N][D] residual stream after attention
  float* cln2[kTfMaxBlocks];         // [N][D] LN2 output (the MLP input)
  float* cu[kTfMaxBlocks];           // [N][M] MLP pre-activations
  float* cnhat;                      // [N][D] final LayerNorm before its gain and bias
  float* cz;                         // [N][V] logits
  // per-candidate slots
  float* sx;      // [K][NB+1][N][D] the candidate's residual streams
  float* sh;      // [K][NB][N][D] after attention, per block
  float* sln;     // [K][N][D] LN1 / final LayerNorm output (the next product's input)
  float* sln2;    // [K][NB][N][D] LN2 output, per block
  float* su;      // [K][NB][N][M] MLP pre-activations, per block
  float* sqkv;    // [K][N][3D]
  float* satt;    // [K][N][D]
  float* sfc;     // [K][N][M] MLP hidden (GELU of the pre-activations)
  float* snhat;   // [K][N][D] final LayerNorm before its gain and bias
  float* slog;    // [K][N][V] logits
  float* sell;    // [K][N] the candidate's per-position losses
  float* scopy;   // [K][copy_stride] private copy of the mutated tensor
  int64_t copy_stride;
  float** table;  // [K][n_tensors] tensor pointers per candidate
  int32_t* start; // [K] first stage the candidate recomputes (NB+2: none)
  int32_t* run;   // [K] first stage it runs in the current pass (NB+2: none)
  int32_t* xin;   // [K] first residual stream the candidate changes (its slot holds x_xin .. x_NB)
  int32_t* kind;  // [K] TfKind of the candidate
  int32_t* pass;  // [1] the slot every block of a one-slot pass works on (-1: its blockIdx)
};

// The slot a block works on: its grid index, or the one slot of a pass that
// recomputes a single candidate.
__device__ inline int tf_slot(const TfDev* tf, unsigned grid_index) {
  const int p = *tf->pass;
  return p >= 0 ? p : (int)grid_index;
}

// How a candidate is evaluated (by its tensor):
//  kTfDense   the stages from its tensor's on, densely (embeddings, LayerNorm
//             1 and 2, attention projections);
//  kTfOutCol  an output-layer weight or bias: one logit column moves by
//             de times the final LayerNorm column (1 for the bias), then the
//             cross-entropy;
//  kTfLnfCol  a final-LayerNorm gain or bias: one column of its output moves
//             by de times the normalized column (1 for the bias), a rank-1
//             term into the logits, then the cross-entropy;
//  kTfProjCol an MLP down-projection weight or bias of block b: one column
//             of x_{b+1} moves by de times a GELU column (1 for the bias),
//             then the stages after block b densely;
//  kTfFcCol   an MLP up-projection weight or bias of block b: one
//             pre-activation column moves by de times an LN2 column (1 for
//             the bias); its GELU change enters x_{b+1} as a rank-1 term
//             through the down-projection's column, then the stages after
//             block b densely.
enum TfKind { kTfDense = 0, kTfOutCol = 1, kTfLnfCol = 2, kTfProjCol = 3, kTfFcCol = 4 };

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
// Commit candidate k (k < 0: st->chosen) into the committed state; `fill`
// copies slot 0 of an identity pass instead and sets the loss.  A candidate
// that was evaluated incrementally (an MLP, final-LayerNorm or output-layer
// parameter) is first recomputed densely from its stage, so that the
// committed fields are always those a dense pass gives (a later dense
// evaluation then reproduces every position it does not reach, bit for bit).
hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, float* partial, int nblk, hipStream_t s);
int tf_loss_blocks(int64_t N);

}  // namespace mca
