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
  float* ch[kTfMaxBlocks];           // committed residual stream after attention, per block
  float* cz;                         // committed logits [N][V]
  float* ell;                        // committed per-position losses
  // per-slot activations: slots 0 .. K-1 hold the candidates of a batch,
  // slot kr the dense recomputation of the last winner that was scored
  // incrementally (see TfRedo)
  float* sx;      // [K+1][NB+1][N][D] the slot's residual streams
  float* sh;      // [K+1][NB][N][D] after attention, per block
  float* sqkv;    // [K+1][N][3D]
  float* satt;    // [K+1][N][D]
  float* sfc;     // [K+1][N][M] MLP hidden (GELU of the pre-activations)
  float* slog;    // [K+1][N][V] logits
  float* sell;    // [K+1][N] the slot's per-position losses
  float2* sst;    // [K+1][N] mean and 1/sqrt(var + eps) of the rows entering the next LayerNorm
  float* scopy;   // [K+1][copy_stride] private copy of the mutated tensor
  int64_t copy_stride;
  float** table;  // [K+1][n_tensors] tensor pointers per slot
  int32_t* start; // [K+1] first stage the slot recomputes (NB+2: none)
  int32_t* run;   // [K+1] first stage it runs in the current pass (NB+2: none)
  int32_t* xin;   // [K+1] first residual stream it changes (its slot holds x_xin .. x_NB)
  int32_t* half;  // [K+1] stage whose attention half it takes from the committed state (0: none)
  int32_t* kind;  // [K+1] TfKind of the candidate
  int32_t* redo;  // [3] TfRedo: the pending dense recomputation (start, half, xin)
  int32_t kr;     // the slot of that recomputation (= the largest batch)
  int32_t pad1;
};

// How a candidate is evaluated (by its tensor):
//  kTfDense   the stages from its tensor's on, densely (embeddings, LayerNorm
//             1 and 2, attention projections); an LN2 gain or bias from its
//             block's MLP half, reading the committed attention output;
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

// A winner scored incrementally changes the committed parameters at once,
// but its fields are recomputed densely (with the committed parameters) in
// the slot kr of the next evaluation pass, so that the committed fields stay
// exactly those of a dense pass.  Until the commit after that pass folds
// them in, the committed state is read through views: x_j from slot kr for
// j >= xin, the attention output of block b from slot kr where it recomputed
// that block's attention, the logits and losses from slot kr.  An MLP
// winner of block b starts at block b's MLP half (half = start = b + 1),
// an output-layer or final-LayerNorm winner at the final stage.
enum TfRedo { kRedoStart = 0, kRedoHalf = 1, kRedoXin = 2 };

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
// Every stage of every candidate's forward pass from its first changed stage
// (and the pending dense recomputation in slot kr), and the tile sums of
// each candidate's per-position loss changes: partial[k * nblk + b].
// K = 0 with `identity` runs one unmutated pass in slot 0 (cache fill);
// K = 0 without it runs only the pending recomputation.
hipError_t tf_launch_eval(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                          const Aux* aux, int K, bool identity, float* partial, int nblk,
                          hipStream_t s);
// Commit candidate k (-1: st->chosen, none if that is negative; -2: none)
// into the committed state after the pending recomputation of the previous
// pass; a
// winner scored incrementally becomes the next pending recomputation.
// `fill` copies slot 0 of an identity pass instead, clears the pending
// recomputation and sets the loss.  Because every committed field is one a
// dense pass gives, a later dense evaluation reproduces every position it
// does not reach, bit for bit.
hipError_t tf_launch_commit(const TfDev* tf, const TfDev& h, const mca_cand* cands,
                            const Aux* aux, const double* dL, DevState* st, int k, bool fill,
                            double* bsum, hipStream_t s);
int tf_loss_blocks(int64_t N);

}  // namespace mca
