// C ABI of the MCA library: validation, workspace layout, uploads, and the
// host side of the step loop.  The device work lives in the kernel files; this
// file only enqueues it on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mca.h"
#include "device_common.hpp"
#include "one_loop.hpp"
#include "loop_kernel.hpp"
#include "mlp_kernels.hpp"
#include "slab_kernels.hpp"
#include "chain_kernels.hpp"
#include "channel_kernels.hpp"
#include "norm_kernels.hpp"
#include "tf_kernels.hpp"

using mca::Aux;
using mca::DevState;
using mca::NetDev;

// Per-call buffers of mca_eval_losses_noalloc: one array per GPU, for the
// process's lifetime.  Host code never uses this name as an address: it is a
// host-side stand-in; the device address comes from hipGetSymbolAddress.
constexpr size_t kScratchBytes = (size_t)8 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int64_t kTraceCap = 4096;  // steps per trace chunk kept on the device
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of this GPU's scratch array, looked up once per device
// with that device current (mca_init calls it).  nullptr on failure.
hipError_t scratch_for_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
constexpr size_t kAlign = 256;
constexpr int kMinLoopTile = 16;
// The committed state (DevState), the snapshot of its counters taken when a
// run_steps call starts, and the step loop's abort word, on three 256-byte
// lines of one block: a call reads all three back with one copy.
constexpr size_t kStateBlock = 3 * 256;
static_assert(sizeof(DevState) <= 256 && sizeof(mca::LoopSync) <= 256, "state block lines");

thread_local std::string g_thread_error;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Byte offsets of every buffer inside the caller's workspace.
struct Layout {
  int64_t Ns = 0;
  int ntiles = 0;     // blocks of the column commit (kTile samples each)
  int ntiles_ev = 0;  // tiles of the batched evaluation (partial sums per candidate)
  size_t xt = 0, ell = 0, pr = 0, y = 0, cands = 0, aux = 0, partial = 0, dl = 0, bsum = 0, state = 0;
  size_t fmask = 0, cmask = 0;  // batched evaluation: tiles where a feature / candidate can change
  size_t tr_chosen = 0, tr_dl = 0, loop_partials = 0, loop_sync = 0, loop_dls = 0;
  size_t wt = 0, pslab = 0;  // three-layer nets: W_1 transposed, first-layer tile sums
  size_t cols = 0, nnz = 0;  // nonzero entries of layer L-3 candidates' W_{L-2} columns
  size_t rows = 0, rda = 0, rcnt = 0, pchain = 0;  // deep nets: affected samples, tile sums
  size_t chans = 0, pchan = 0;                      // channel mutations: records, tile sums
  size_t pnorm = 0;                                 // nets with biases / normalization: tile sums
  size_t b[MCA_MAX_LAYERS] = {}, mu[MCA_MAX_LAYERS] = {}, S[MCA_MAX_LAYERS] = {};
  int nchain = 0, nchan = 0, nnorm = 0;
  int nslab = 0;
  int loop_T = 0, loop_G = 0;
  size_t w[MCA_MAX_LAYERS] = {}, codes[MCA_MAX_LAYERS] = {}, z[MCA_MAX_LAYERS] = {};
  size_t total = 0;
};

// Selection rule, pruning and minibatch fields (shared by both net kinds).
std::string check_selection(const mca_net_desc* net, int64_t n_samples, int* code) {
  *code = MCA_EINVAL;
  if (net->accept_rule != MCA_RULE_GREEDY && net->accept_rule != MCA_RULE_METROPOLIS)
    return "unknown accept rule";
  if (net->accept_rule == MCA_RULE_METROPOLIS && !(std::isfinite(net->beta) && net->beta > 0.0))
    return "Metropolis beta must be finite and positive";
  if (net->n_prune < 0) return "n_prune must be >= 0";
  if (net->subset_size < 0 || net->subset_size > n_samples) return "subset_size out of range [0, n_samples]";
  if (net->subset_size > 0 && net->subset_period < 1) return "subset_period must be >= 1";
  *code = MCA_EUNSUPPORTED;
  if (net->kind == MCA_NET_TRANSFORMER && net->n_prune != 0)
    return "pruning candidates are built for MLPs only";
  if (net->kind == MCA_NET_TRANSFORMER && net->subset_size != 0)
    return "minibatches are built for MLPs only";
  *code = MCA_OK;
  return "";
}
// Nets scored layer by layer with dense products (k_norm): those with
// biases or normalized hidden fields, and plain deep nets (four or more
// layers) whose hidden layers are all 512 or all 1024 wide (the column and
// chain kernels of plain deep nets take 256).
bool dense_path(const mca_net_desc* net) {
  if (net->biases || net->layer_norm) return true;
  const int L = net->n_layers;
  if (L < 4 || net->mutation != MCA_MUTATE_SINGLE) return false;
  for (int l = 1; l < L; ++l)
    if (net->widths[l] != net->widths[1]) return false;
  return net->widths[1] != mca::kChainUnits && mca::norm_width_ok(net->widths[1]);
}


std::string check_desc(const mca_net_desc* net, int64_t n_samples, int32_t k_max, int* code) {
  *code = MCA_EINVAL;
  if (net == nullptr) return "net description is NULL";
  if (net->kind != MCA_NET_MLP) return "unknown net kind";
  const int L = net->n_layers;
  if (L < 1 || L > MCA_MAX_LAYERS) return "n_layers out of range [1, 32]";
  for (int l = 0; l <= L; ++l)
    if (net->widths[l] < 1) return "widths must be positive";
  if (net->widths[L] > MCA_MAX_CLASSES) return "output width exceeds MCA_MAX_CLASSES (16)";
  for (int l = 0; l < L; ++l)
    if ((int64_t)net->widths[l] * net->widths[l + 1] >= (int64_t)1 << 31)
      return "a weight matrix has 2^31 or more entries";
  if (net->act != MCA_ACT_TANH && net->act != MCA_ACT_GAUSS && net->act != MCA_ACT_RELU)
    return "unknown transfer function";
  if (net->mutation != MCA_MUTATE_SINGLE && net->mutation != MCA_MUTATE_CHANNEL_REDRAW &&
      net->mutation != MCA_MUTATE_CHANNEL_ZERO)
    return "unknown mutation kind";
  if (net->act == MCA_ACT_GAUSS && !(std::isfinite(net->gamma) && net->gamma > 0.f))
    return "gamma must be finite and positive";
  if (net->weight_mode != MCA_WEIGHTS_FP32 && net->weight_mode != MCA_WEIGHTS_TERNARY)
    return "unknown weight mode";
  if (net->weight_mode == MCA_WEIGHTS_TERNARY)
    for (int l = 0; l < L; ++l)
      if (!(std::isfinite(net->scales[l]) && net->scales[l] > 0.f))
        return "ternary scales must be finite and positive";
  if (net->pick != MCA_PICK_WEIGHT && net->pick != MCA_PICK_LAYER && net->pick != MCA_PICK_STICKY)
    return "unknown pick mode";
  if (net->pick == MCA_PICK_STICKY && net->sticky_steps < 1) return "sticky_steps must be >= 1";
  if ((net->biases != 0 && net->biases != 1) || (net->layer_norm != 0 && net->layer_norm != 1))
    return "biases and layer_norm take 0 or 1";
  if (net->layer_norm && !(std::isfinite(net->ln_eps) && net->ln_eps > 0.f))
    return "ln_eps must be finite and positive";
  if (!std::isfinite(net->delta) || net->delta < 0.f) return "delta must be finite and >= 0";
  if (!std::isfinite(net->bound)) return "bound must be finite (<= 0 disables it)";
  if (n_samples < 1 || n_samples > ((int64_t)1 << 31)) return "n_samples out of range";
  if (k_max < 1 || k_max > mca::kMaxK) return "k_max out of range [1, 1024]";
  {
    std::string m = check_selection(net, n_samples, code);
    if (!m.empty()) return m;
  }
  if (dense_path(net)) {
    *code = MCA_EUNSUPPORTED;
    if (L < 2) return "biases and normalization need at least one hidden layer";
    if (net->weight_mode != MCA_WEIGHTS_FP32)
      return "biases, normalization and deep hidden layers 512 or 1024 wide take continuous weights";
    if (net->mutation != MCA_MUTATE_SINGLE) return "channel mutations take no biases or normalization";
    for (int l = 1; l < L; ++l)
      if (net->widths[l] != net->widths[1] || !mca::norm_width_ok(net->widths[l]))
        return "nets with biases or normalization need every hidden layer 256, 512 or 1024 units wide";
    *code = MCA_OK;
    return "";
  }
  if (net->mutation != MCA_MUTATE_SINGLE) {
    *code = MCA_EUNSUPPORTED;
    if (L < 2) return "channel mutations need at least one hidden layer";
    if (net->weight_mode != MCA_WEIGHTS_FP32) return "channel mutations take continuous weights";
    for (int l = 1; l < L; ++l)
      if (net->widths[l] != net->widths[1] || !mca::channel_width_ok(net->widths[l]))
        return "channel mutations need every hidden layer 256, 512 or 1024 units wide";
    if (net->n_prune != 0) return "channel mutations take no pruning candidates";
    if (net->subset_size != 0) return "channel mutations score every sample";
    *code = MCA_OK;
    return "";
  }
  if (L >= 3 && net->widths[L - 1] > mca::kSlabMaxUnits) {
    *code = MCA_EUNSUPPORTED;
    return "MLPs with three or more layers need a last hidden layer of at most 1024 units";
  }
  if (L >= 4)
    for (int l = 1; l < L; ++l)
      if (net->widths[l] != mca::kChainUnits) {
        *code = MCA_EUNSUPPORTED;
        return "MLPs with four or more layers need every hidden layer 256 units wide (all 512 or all 1024 with continuous weights)";
      }
  *code = MCA_OK;
  return "";
}

// ---------------------------------------------------------------------------
// Transformer nets: shapes, validation and workspace layout
// ---------------------------------------------------------------------------

struct TfShape {
  int64_t rows, cols;  // 1-D tensors: cols = 1
};

// Canonical parameter order: tok_emb, pos_emb, per block ln1.g, ln1.b, wq, bq,
// wk, bk, wv, bv, wo, bo, ln2.g, ln2.b, wfc, bfc, wproj, bproj, then lnf.g,
// lnf.b, wout, bout; linear weights [out][in].
std::vector<TfShape> tf_shapes(const mca_net_desc* d) {
  const int64_t V = d->vocab, T = d->ctx, D = d->d_model, M = d->d_mlp;
  std::vector<TfShape> s = {{V, D}, {T, D}};
  for (int b = 0; b < d->n_block; ++b) {
    const TfShape blk[mca::kBlockTensors] = {{D, 1}, {D, 1}, {D, D}, {D, 1}, {D, D}, {D, 1},
                                             {D, D}, {D, 1}, {D, D}, {D, 1}, {D, 1}, {D, 1},
                                             {M, D}, {M, 1}, {D, M}, {D, 1}};
    s.insert(s.end(), blk, blk + mca::kBlockTensors);
  }
  s.push_back({D, 1});
  s.push_back({D, 1});
  s.push_back({V, D});
  s.push_back({V, 1});
  return s;
}

std::string tf_check_desc(const mca_net_desc* d, int64_t n_samples, int32_t k_max, int* code) {
  *code = MCA_EINVAL;
  if (d->vocab < 2 || d->ctx < 1 || d->d_model < 1 || d->n_block < 1 || d->n_head < 1 ||
      d->d_mlp < 1)
    return "transformer sizes must be positive (vocab >= 2)";
  if (!(std::isfinite(d->ln_eps) && d->ln_eps > 0.f)) return "ln_eps must be finite and positive";
  if (!std::isfinite(d->delta) || d->delta < 0.f) return "delta must be finite and >= 0";
  if (!std::isfinite(d->bound)) return "bound must be finite (<= 0 disables it)";
  if (k_max < 1 || k_max > mca::kMaxK) return "k_max out of range [1, 1024]";
  if (n_samples < 1 || n_samples > ((int64_t)1 << 31) || n_samples % d->ctx != 0)
    return "n_samples must be a positive multiple of ctx";
  {
    std::string m = check_selection(d, n_samples, code);
    if (!m.empty()) return m;
  }
  *code = MCA_EUNSUPPORTED;
  if (d->weight_mode != MCA_WEIGHTS_FP32) return "Transformer nets take continuous weights only";
  if (d->pick != MCA_PICK_WEIGHT) return "Transformer nets draw uniformly over all parameters only";
  if (d->d_model != mca::kTfHeadDim * d->n_head) return "d_model must be 32 * n_head";
  if (d->d_model > 256) return "d_model must be at most 256";
  if (d->d_mlp % 32 != 0) return "d_mlp must be a multiple of 32";
  if (d->vocab > mca::kTfMaxVocab) return "vocab must be at most 128";
  if (d->ctx > mca::kTfMaxCtx) return "ctx must be at most 128";
  if (d->n_block > mca::kTfMaxBlocks) return "at most 8 blocks";
  *code = MCA_OK;
  return "";
}

struct TfLayout {
  size_t param[mca::kTfMaxTensors] = {};
  size_t tok = 0, tgt = 0, x = 0, ell = 0, cands = 0, aux = 0, partial = 0, dl = 0, bsum = 0;
  size_t state = 0, tr_chosen = 0, tr_dl = 0;
  size_t sx = 0, sh = 0, sqkv = 0, satt = 0, sfc = 0, slog = 0, sell = 0, sst = 0, scopy = 0;
  size_t ch = 0, cz = 0;  // committed attention outputs and logits
  size_t table = 0, start = 0, xin = 0, kind = 0, run = 0, half = 0, redo = 0, dev = 0;
  int64_t copy_stride = 0;
  int nblk = 0, n_tensors = 0;
  size_t total = 0;
};

TfLayout tf_make_layout(const mca_net_desc* d, int64_t N, int32_t k_max) {
  TfLayout lo;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const std::vector<TfShape> shapes = tf_shapes(d);
  lo.n_tensors = (int)shapes.size();
  int64_t maxsz = 0;
  for (size_t t = 0; t < shapes.size(); ++t) {
    const int64_t n = shapes[t].rows * shapes[t].cols;
    lo.param[t] = take((size_t)n * sizeof(float));
    maxsz = std::max(maxsz, n);
  }
  const size_t K = (size_t)k_max, n = (size_t)N, D = (size_t)d->d_model;
  const size_t NB = (size_t)d->n_block, M = (size_t)d->d_mlp, V = (size_t)d->vocab;
  lo.nblk = mca::tf_loss_blocks(N);
  lo.tok = take(n * sizeof(int32_t));
  lo.tgt = take(n * sizeof(int32_t));
  lo.x = take((NB + 1) * n * D * sizeof(float));
  lo.ell = take(n * sizeof(float));
  lo.cands = take(K * sizeof(mca_cand));
  lo.aux = take(K * sizeof(Aux));
  lo.partial = take(K * lo.nblk * sizeof(float));
  lo.dl = take(K * sizeof(double));
  lo.bsum = take((size_t)lo.nblk * sizeof(double));
  lo.state = take(kStateBlock);
  lo.tr_chosen = take((size_t)kTraceCap * sizeof(int32_t));
  lo.tr_dl = take((size_t)kTraceCap * K * sizeof(double));
  lo.ch = take(NB * n * D * sizeof(float));
  lo.cz = take(n * V * sizeof(float));
  // K candidate slots and one for the pending dense recomputation of a winner
  const size_t KS = K + 1;
  lo.sx = take(KS * (NB + 1) * n * D * sizeof(float));
  lo.sh = take(KS * NB * n * D * sizeof(float));
  lo.satt = take(KS * n * D * sizeof(float));
  lo.sqkv = take(KS * n * 3 * D * sizeof(float));
  lo.sfc = take(KS * n * M * sizeof(float));
  lo.slog = take(KS * n * V * sizeof(float));
  lo.sell = take(KS * n * sizeof(float));
  lo.sst = take(KS * n * 2 * sizeof(float));
  lo.copy_stride = (maxsz + 63) / 64 * 64;
  lo.scopy = take(KS * (size_t)lo.copy_stride * sizeof(float));
  lo.table = take(KS * (size_t)lo.n_tensors * sizeof(float*));
  lo.start = take(KS * sizeof(int32_t));
  lo.xin = take(KS * sizeof(int32_t));
  lo.kind = take(KS * sizeof(int32_t));
  lo.run = take(KS * sizeof(int32_t));
  lo.half = take(KS * sizeof(int32_t));
  lo.redo = take(4 * sizeof(int32_t));
  lo.dev = take(sizeof(mca::TfDev));
  lo.total = off;
  return lo;
}

Layout make_layout(const mca_net_desc* net, int64_t N, int32_t k_max) {
  Layout lo;
  lo.Ns = (N + 63) / 64 * 64;
  lo.ntiles = (int)((N + mca::kTile - 1) / mca::kTile);
  lo.ntiles_ev = mca::eval_tiles(N);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const int L = net->n_layers;
  const bool norm = dense_path(net);
  lo.xt = take((size_t)net->widths[0] * lo.Ns * sizeof(float));
  for (int l = 0; l < L; ++l) lo.w[l] = take((size_t)net->widths[l + 1] * net->widths[l] * sizeof(float));
  if (net->biases)
    for (int l = 0; l < L; ++l) lo.b[l] = take((size_t)net->widths[l + 1] * sizeof(float));
  if (net->layer_norm)
    for (int l = 0; l + 1 < L; ++l) {
      lo.mu[l] = take(lo.Ns * sizeof(float));
      lo.S[l] = take(lo.Ns * sizeof(float));
    }
  if (net->weight_mode == MCA_WEIGHTS_TERNARY)
    for (int l = 0; l < L; ++l) lo.codes[l] = take((size_t)net->widths[l + 1] * net->widths[l]);
  for (int l = 0; l < L; ++l) lo.z[l] = take((size_t)net->widths[l + 1] * lo.Ns * sizeof(float));
  lo.ell = take(lo.Ns * sizeof(float));
  lo.pr = take((size_t)net->widths[L] * lo.Ns * sizeof(float));
  lo.y = take(lo.Ns * sizeof(int32_t));
  lo.cands = take((size_t)k_max * sizeof(mca_cand));
  lo.aux = take((size_t)k_max * sizeof(Aux));
  lo.fmask = take((size_t)net->widths[0] * sizeof(uint64_t));
  lo.cmask = take((size_t)k_max * sizeof(uint64_t));
  lo.partial = take((size_t)k_max * lo.ntiles_ev * sizeof(float));
  lo.dl = take((size_t)k_max * sizeof(double));
  lo.bsum = take((size_t)lo.ntiles * sizeof(double));
  lo.state = take(kStateBlock);
  lo.tr_chosen = take((size_t)kTraceCap * sizeof(int32_t));
  lo.tr_dl = take((size_t)kTraceCap * k_max * sizeof(double));
  const bool chan = net->mutation != MCA_MUTATE_SINGLE;
  if (L >= 3 && !norm) {
    lo.wt = take((size_t)net->widths[L - 2] * net->widths[L - 1] * sizeof(float));
    const int T = mca::slab_tile(net->widths[L]);
    lo.nslab = (int)((N + T - 1) / T);
    lo.pslab = take((size_t)k_max * lo.nslab * sizeof(float));
    lo.cols = take((size_t)k_max * net->widths[L - 1] * sizeof(uint64_t));
    lo.nnz = take((size_t)k_max * sizeof(int32_t));
  }
  if (L >= 4 && !chan && !norm) {
    lo.nchain = (int)((N + mca::kChainT - 1) / mca::kChainT);
    lo.rows = take((size_t)k_max * N * sizeof(int32_t));
    lo.rda = take((size_t)k_max * N * sizeof(float));
    lo.rcnt = take((size_t)k_max * sizeof(int32_t));
    lo.pchain = take((size_t)k_max * lo.nchain * sizeof(float));
  }
  if (norm) {
    lo.nnorm = mca::norm_tiles(N, net->widths[1]);
    lo.pnorm = take((size_t)k_max * lo.nnorm * sizeof(float));
  }
  if (net->mutation != MCA_MUTATE_SINGLE) {
    lo.nchan = mca::channel_tiles(N, net->widths[1]);
    lo.chans = take((size_t)k_max * sizeof(mca_channel));
    lo.pchan = take((size_t)k_max * lo.nchan * sizeof(float));
  }
  // persistent loop: tiles of T samples (16..64), one workgroup each; the
  // partial sums are sized for the smallest tile
  lo.loop_T = 64;
  lo.loop_G = (int)((N + lo.loop_T - 1) / lo.loop_T);
  const int64_t g_max = (N + kMinLoopTile - 1) / kMinLoopTile;
  const int64_t gpad = (g_max + 15) / 16 * 16;
  lo.loop_partials = take((size_t)2 * std::min<int32_t>(k_max, mca::kLoopMaxK) * gpad * sizeof(uint64_t));
  lo.loop_dls = take((size_t)mca::kLoopReplicas * mca::kLoopMaxK * sizeof(uint64_t));
  lo.total = off;
  return lo;
}

__global__ void k_set_trace_base(DevState* st) { st->trace_base = st->t; }
__global__ void k_set_next_step(DevState* st, uint64_t v) { st->t = v; }
// Start of a run_steps call: the counters as they stand, and a clear abort word.
__global__ void k_call_start(const DevState* st, DevState* snap, mca::LoopSync* sync) {
  *snap = *st;
  sync->abort = 0;
}

}  // namespace

struct mca_ctx {
  mca_net_desc desc{};
  NetDev net{};
  Layout lo;
  hipStream_t stream = nullptr;
  int32_t k_max = 0;
  char* ws = nullptr;
  mca_cand* cands = nullptr;
  Aux* aux = nullptr;
  uint64_t* fmask = nullptr;  // null: more evaluation tiles than bits
  uint64_t* cmask = nullptr;
  float* partial = nullptr;
  float* pslab = nullptr;
  uint64_t* cols = nullptr;
  int* nnz = nullptr;
  int* rows = nullptr;
  float* rda = nullptr;
  int* rcnt = nullptr;
  float* pchain = nullptr;
  bool chan = false;             // candidates are channel mutations (Sec. 2.3)
  mca_channel* chans = nullptr;  // their records
  float* pchan = nullptr;        // their tile sums
  bool norm = false;             // biases and / or normalized hidden fields (Sec. 2.1)
  mca::NormDev nd{};             // normalization statistics
  float* pnorm = nullptr;        // tile sums of the dense evaluation
  double* dl = nullptr;
  double* bsum = nullptr;
  DevState* st = nullptr;
  int32_t* tr_chosen = nullptr;
  double* tr_dl = nullptr;
  uint64_t* loop_partials = nullptr;
  uint64_t* loop_dls = nullptr;
  mca::LoopSync* loop_sync = nullptr;
  DevState* snap = nullptr;  // counters at the start of the current run_steps call
  unsigned char* host_blk = nullptr;  // pinned host copy of the state block (null: none)
  bool use_loop = true;
  bool loop_coop = false;    // cooperative launch of the step loop (default: ordinary)
  void* scratch_dev = nullptr;  // this device's static scratch array (no-allocation entry point)
  int loop_fit_K = -1, loop_fit = 0;  // resident workgroups of the loop, cached per K
  // Transformer nets
  bool tf = false;
  mca::TfDev tfh{};           // host copy of the device description
  mca::TfDev* tfd = nullptr;  // device copy, in the workspace
  int tf_nblk = 0;            // loss tiles of 256 positions
  bool pending = false;
  int32_t pending_K = 0;
  std::vector<double> pending_dl;  // loss changes of the pending batch (+inf: rejected unevaluated)
  bool poisoned = false;
  std::string err;
  // phase timing
  int32_t timing = 0;  // bit mask of timed phases
  struct Rec { int phase; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  mca_timing acc{};
};

namespace {

int fail(mca_ctx* ctx, int code, const std::string& msg) {
  if (ctx) ctx->err = msg; else g_thread_error = msg;
  return code;
}

int device_fail(mca_ctx* ctx, hipError_t e, const char* what) {
  std::string msg = std::string(what) + ": " + hipGetErrorString(e);
  if (ctx) { ctx->poisoned = true; ctx->err = msg; } else g_thread_error = msg;
  return MCA_EDEVICE;
}

#define MCA_HIP(ctx, expr)                                   \
  do {                                                       \
    hipError_t e_ = (expr);                                  \
    if (e_ != hipSuccess) return device_fail(ctx, e_, #expr); \
  } while (0)

#define MCA_LIVE(ctx)                                                  \
  do {                                                                 \
    if ((ctx) == nullptr) return fail(nullptr, MCA_EINVAL, "ctx is NULL"); \
    if ((ctx)->poisoned) return fail(ctx, MCA_EPOISONED, "context poisoned by an earlier device error: " + (ctx)->err); \
  } while (0)

// Waits for the stream by polling it for up to a millisecond, then blocks: a
// blocking wait may put the thread to sleep, and waking it costs tens of
// microseconds, a large share of a call of a few dozen steps.
hipError_t wait_stream(hipStream_t s) {
  const auto t0 = std::chrono::steady_clock::now();
  while (true) {
    const hipError_t e = hipStreamQuery(s);
    if (e != hipErrorNotReady) return e;
    if (std::chrono::steady_clock::now() - t0 > std::chrono::microseconds(1000)) break;
  }
  return hipStreamSynchronize(s);
}

// Events made ahead when timing is switched on (a step-loop call records one
// pair per launch; the per-phase loop four pairs per step).
constexpr size_t kEventsAhead = 32;

hipEvent_t get_event(mca_ctx* ctx) {
  if (!ctx->pool.empty()) {
    hipEvent_t e = ctx->pool.back();
    ctx->pool.pop_back();
    return e;
  }
  // Phase timers only order work on this stream: without the system-scope
  // fence on completion a record adds no idle gap between the kernels.
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Wraps one launch in a pair of events when timing is on.
template <class F>
hipError_t timed(mca_ctx* ctx, int phase, F&& launch) {
  if (!(ctx->timing & (1 << phase))) return launch();
  hipEvent_t a = get_event(ctx), b = get_event(ctx);
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, ctx->stream);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, ctx->stream);
  if (e != hipSuccess) return e;
  ctx->recs.push_back({phase, a, b});
  return hipSuccess;
}

int flush_timing(mca_ctx* ctx) {
  if (ctx->recs.empty()) return MCA_OK;
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  for (auto& r : ctx->recs) {
    float ms = 0.f;
    MCA_HIP(ctx, hipEventElapsedTime(&ms, r.a, r.b));
    ctx->acc.ms[r.phase] += ms;
    ctx->acc.launches[r.phase] += 1;
    ctx->pool.push_back(r.a);
    ctx->pool.push_back(r.b);
  }
  ctx->recs.clear();
  return MCA_OK;
}

int run_forward(mca_ctx* ctx) {
  if (ctx->tf) {
    // one unmutated pass in slot 0, copied into the committed state
    MCA_HIP(ctx, timed(ctx, 5, [&] {
      hipError_t e = mca::tf_launch_eval(ctx->tfd, ctx->tfh, ctx->cands, ctx->aux, 0, true,
                                         ctx->partial, ctx->tf_nblk, ctx->stream);
      if (e == hipSuccess)
        e = mca::tf_launch_commit(ctx->tfd, ctx->tfh, ctx->cands, ctx->aux, ctx->dl, ctx->st, 0,
                                  true, ctx->bsum, ctx->stream);
      return e;
    }));
    return MCA_OK;
  }
  if (ctx->norm)
    MCA_HIP(ctx, timed(ctx, 5, [&] {
      return mca::launch_forward_norm(ctx->net, ctx->nd, ctx->bsum, ctx->st, ctx->stream);
    }));
  else
    MCA_HIP(ctx, timed(ctx, 5, [&] { return mca::launch_forward(ctx->net, ctx->bsum, ctx->st, ctx->stream); }));
  return MCA_OK;
}

int tf_upload_params(mca_ctx* ctx, const float* const* params) {
  if (params == nullptr) return fail(ctx, MCA_EINVAL, "params is NULL");
  const std::vector<TfShape> shapes = tf_shapes(&ctx->desc);
  for (size_t t = 0; t < shapes.size(); ++t) {
    if (params[t] == nullptr) return fail(ctx, MCA_EINVAL, "a parameter pointer is NULL");
    const int64_t n = shapes[t].rows * shapes[t].cols;
    for (int64_t e = 0; e < n; ++e)
      if (!std::isfinite(params[t][e])) return fail(ctx, MCA_EINVAL, "non-finite parameter");
  }
  for (size_t t = 0; t < shapes.size(); ++t) {
    const size_t n = (size_t)(shapes[t].rows * shapes[t].cols);
    MCA_HIP(ctx, hipMemcpyAsync(ctx->tfh.param[t], params[t], n * sizeof(float), hipMemcpyHostToDevice, ctx->stream));
  }
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int upload_params(mca_ctx* ctx, const float* const* params, const int8_t* const* codes) {
  if (ctx->tf) return tf_upload_params(ctx, params);
  const mca_net_desc& d = ctx->desc;
  const int L = d.n_layers;
  if (params == nullptr) return fail(ctx, MCA_EINVAL, "params is NULL");
  const bool tern = d.weight_mode == MCA_WEIGHTS_TERNARY;
  if (tern && codes == nullptr) return fail(ctx, MCA_EINVAL, "ternary weights need codes");
  for (int l = 0; l < L; ++l) {
    if (params[l] == nullptr) return fail(ctx, MCA_EINVAL, "a parameter pointer is NULL");
    const size_t n = (size_t)d.widths[l + 1] * (d.widths[l] + d.biases);
    if (tern) {
      if (codes[l] == nullptr) return fail(ctx, MCA_EINVAL, "a code pointer is NULL");
      for (size_t e = 0; e < n; ++e) {
        const int c = codes[l][e];
        if (c < -1 || c > 1) return fail(ctx, MCA_EINVAL, "ternary code outside {-1, 0, 1}");
        const float v = (float)c * d.scales[l];
        if (std::memcmp(&v, &params[l][e], sizeof(float)) != 0 && !(v == 0.f && params[l][e] == 0.f))
          return fail(ctx, MCA_EINVAL, "ternary parameter differs from code * scale");
      }
    } else {
      for (size_t e = 0; e < n; ++e)
        if (!std::isfinite(params[l][e])) return fail(ctx, MCA_EINVAL, "non-finite parameter");
    }
  }
  for (int l = 0; l < L; ++l) {
    const size_t n = (size_t)d.widths[l + 1] * d.widths[l];
    if (d.biases) {  // the augmented matrix [n_{l+1}][n_l + 1]: weights, then the bias column
      const size_t w = (size_t)d.widths[l], rows = (size_t)d.widths[l + 1];
      MCA_HIP(ctx, hipMemcpy2DAsync(ctx->net.W[l], w * sizeof(float), params[l], (w + 1) * sizeof(float),
                                    w * sizeof(float), rows, hipMemcpyHostToDevice, ctx->stream));
      MCA_HIP(ctx, hipMemcpy2DAsync(ctx->net.B[l], sizeof(float), params[l] + w, (w + 1) * sizeof(float),
                                    sizeof(float), rows, hipMemcpyHostToDevice, ctx->stream));
      continue;
    }
    MCA_HIP(ctx, hipMemcpyAsync(ctx->net.W[l], params[l], n * sizeof(float), hipMemcpyHostToDevice, ctx->stream));
    if (tern) MCA_HIP(ctx, hipMemcpyAsync(ctx->net.codes[l], codes[l], n, hipMemcpyHostToDevice, ctx->stream));
  }
  if (ctx->net.WT != nullptr)  // W_{L-2} [n_{L-1}][n_{L-2}] -> W_T [n_{L-2}][n_{L-1}]
    MCA_HIP(ctx, mca::launch_transpose(ctx->net.W[L - 2], d.widths[L - 1], d.widths[L - 2],
                                       ctx->net.WT, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int write_state(mca_ctx* ctx, uint64_t t, bool keep_counters) {
  DevState s{};
  if (keep_counters) {
    MCA_HIP(ctx, hipMemcpyAsync(&s, ctx->st, sizeof s, hipMemcpyDeviceToHost, ctx->stream));
    MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  }
  s.t = t;
  s.chosen = -1;
  MCA_HIP(ctx, hipMemcpyAsync(ctx->st, &s, sizeof s, hipMemcpyHostToDevice, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int read_state(mca_ctx* ctx, DevState* s) {
  MCA_HIP(ctx, hipMemcpyAsync(s, ctx->st, sizeof *s, hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int check_cands(mca_ctx* ctx, const mca_cand* c, int K) {
  const mca_net_desc& d = ctx->desc;
  if (ctx->tf) {
    for (int k = 0; k < K; ++k) {
      const int l = c[k].layer;
      if (l < 0 || l >= ctx->tfh.n_tensors) return fail(ctx, MCA_EINVAL, "candidate tensor out of range");
      if (c[k].j < 0 || c[k].j >= ctx->tfh.rows[l] || c[k].i < 0 || c[k].i >= ctx->tfh.cols[l])
        return fail(ctx, MCA_EINVAL, "candidate index out of range");
      if (!std::isfinite(c[k].d)) return fail(ctx, MCA_EINVAL, "candidate increment is not finite");
      if (c[k].flags != 0) return fail(ctx, MCA_EINVAL, "Transformer candidates take no flags");
    }
    return MCA_OK;
  }
  for (int k = 0; k < K; ++k) {
    const int l = c[k].layer;
    if (l < 0 || l >= d.n_layers) return fail(ctx, MCA_EINVAL, "candidate layer out of range");
    if (c[k].j < 0 || c[k].j >= d.widths[l + 1] || c[k].i < 0 || c[k].i >= d.widths[l] + d.biases)
      return fail(ctx, MCA_EINVAL, "candidate index out of range");
    if (c[k].flags & ~MCA_CAND_PRUNE) return fail(ctx, MCA_EINVAL, "unknown candidate flags");
    if (d.weight_mode == MCA_WEIGHTS_TERNARY) {
      if (c[k].code < -1 || c[k].code > 1) return fail(ctx, MCA_EINVAL, "candidate code outside {-1, 0, 1}");
    } else if (!std::isfinite(c[k].d)) {
      return fail(ctx, MCA_EINVAL, "candidate increment is not finite");
    }
  }
  return MCA_OK;
}

// Where one evaluation's per-call buffers live: the context's workspace, or
// the static scratch array of the no-allocation entry point.
struct Bufs {
  mca_cand* cands;
  Aux* aux;
  uint64_t* cmask;
  float* partial;
  double* dl;
  float* pslab;
  uint64_t* cols;
  int* nnz;
  int* rows;
  float* rda;
  int* rcnt;
  float* pchain;
};

Bufs ctx_bufs(const mca_ctx* ctx) {
  return Bufs{ctx->cands, ctx->aux, ctx->cmask, ctx->partial, ctx->dl, ctx->pslab,
              ctx->cols, ctx->nnz, ctx->rows, ctx->rda, ctx->rcnt, ctx->pchain};
}

hipError_t propose_dev(mca_ctx* ctx, uint64_t step, bool use_dev_t, int K) {
  if (ctx->chan)
    return mca::launch_channel_propose(ctx->net, step, use_dev_t, ctx->st, K, ctx->chans,
                                       ctx->cands, ctx->aux, ctx->stream);
  if (ctx->tf)
    return mca::tf_launch_propose(ctx->tfd, ctx->tfh, step, use_dev_t, ctx->st, K, ctx->cands,
                                  ctx->aux, ctx->stream);
  // (a bias of a first-layer unit has no input feature: no tile list for it)
  return mca::launch_propose(ctx->net, step, use_dev_t, ctx->st, K, ctx->cands, ctx->aux,
                             ctx->norm ? nullptr : ctx->fmask, ctx->cmask, ctx->stream);
}

hipError_t prepare_into(mca_ctx* ctx, const Bufs& b, int K) {
  if (ctx->chan)
    return mca::launch_channel_prepare(ctx->net, ctx->chans, K, b.cands, b.aux, ctx->stream);
  if (ctx->tf) return mca::tf_launch_prepare(ctx->tfd, b.cands, K, b.aux, ctx->stream);
  return mca::launch_prepare(ctx->net, b.cands, K, b.aux, ctx->norm ? nullptr : ctx->fmask,
                             b.cmask, ctx->stream);
}
hipError_t prepare_dev(mca_ctx* ctx, int K) { return prepare_into(ctx, ctx_bufs(ctx), K); }

// Scores the K staged candidates: the column kernel for the last two layers,
// the tile kernel for layer L-3, the dense chain for layers 0..L-4.
// `listed`: the layer L-3 column lists came with the proposal.
hipError_t eval_into(mca_ctx* ctx, const NetDev& net, const Bufs& b, int K, bool listed = false) {
  if (ctx->norm)
    return mca::launch_norm(net, ctx->nd, b.cands, b.aux, K, ctx->pnorm, ctx->lo.nnorm, -2,
                            ctx->st, b.dl, ctx->stream);
  if (ctx->chan)
    return mca::launch_channel(net, ctx->chans, b.aux, K, ctx->pchan, ctx->lo.nchan, -2,
                               ctx->st, b.dl, ctx->stream);
  if (ctx->tf)
    return mca::tf_launch_eval(ctx->tfd, ctx->tfh, b.cands, b.aux, K, false, b.partial,
                               ctx->tf_nblk, ctx->stream);
  hipError_t e = mca::launch_eval(net, b.cands, b.aux, b.cmask, K, b.partial,
                                  ctx->lo.ntiles_ev, ctx->st, ctx->stream);
  if (e == hipSuccess && net.L >= 3)
    e = mca::launch_slab(net, b.cands, b.aux, K, b.cols, b.nnz, b.pslab, ctx->lo.nslab, -2,
                         ctx->st, b.dl, ctx->stream, listed);
  if (e == hipSuccess && net.L >= 4)
    e = mca::launch_chain(net, b.cands, b.aux, K, b.rows, b.rda, b.rcnt, b.pchain,
                          ctx->lo.nchain, -2, ctx->st, b.dl, ctx->stream);
  return e;
}
hipError_t eval_all(mca_ctx* ctx, const NetDev& net, int K, bool listed = false) {
  return eval_into(ctx, net, ctx_bufs(ctx), K, listed);
}

// The device step's proposal; for a plain MLP with a layer L-3 it also lists
// the columns that layer's candidates score (one launch instead of two).
// Returns whether it did.
bool fused_proposal(const mca_ctx* ctx, const NetDev& net) {
  return !ctx->chan && !ctx->tf && !ctx->norm && net.L >= 3;
}
hipError_t propose_step(mca_ctx* ctx, const NetDev& net, int K) {
  if (fused_proposal(ctx, net))
    return mca::launch_propose_columns(net, ctx->st, K, ctx->cands, ctx->aux, ctx->fmask,
                                       ctx->cmask, ctx->cols, ctx->nnz, ctx->stream);
  return propose_dev(ctx, 0, true, K);
}

hipError_t select_into(mca_ctx* ctx, const NetDev& net, const Bufs& b, int K, bool do_select,
                       int32_t* trc, double* trd) {
  if (ctx->norm) {
    NetDev one = net;  // one source of tile sums for every candidate
    one.L = 0;
    return mca::launch_select(one, ctx->pnorm, ctx->lo.nnorm, b.cands, nullptr, 0, nullptr, 0,
                              b.aux, K, b.dl, ctx->st, do_select, trc, trd, kTraceCap,
                              ctx->stream);
  }
  if (ctx->chan) {
    // every channel has one source of tile sums (an L = 0 view of the net
    // selects it)
    NetDev one = net;
    one.L = 0;
    return mca::launch_select(one, ctx->pchan, ctx->lo.nchan, b.cands, nullptr, 0, nullptr, 0,
                              b.aux, K, b.dl, ctx->st, do_select, trc, trd, kTraceCap,
                              ctx->stream);
  }
  if (ctx->tf)
    return mca::launch_select(net, b.partial, ctx->tf_nblk, b.cands, nullptr, 0, nullptr, 0,
                              b.aux, K, b.dl, ctx->st, do_select, trc, trd, kTraceCap,
                              ctx->stream);
  return mca::launch_select(net, b.partial, ctx->lo.ntiles_ev, b.cands, b.pslab,
                            ctx->lo.nslab, b.pchain, ctx->lo.nchain, b.aux, K, b.dl,
                            ctx->st, do_select, trc, trd, kTraceCap, ctx->stream);
}
hipError_t select_all(mca_ctx* ctx, const NetDev& net, int K, bool do_select, int32_t* trc,
                      double* trd) {
  return select_into(ctx, net, ctx_bufs(ctx), K, do_select, trc, trd);
}

// Commits candidate k (k < 0: the device decision) of a batch of K; each
// kernel applies only the candidates of the layers it scores.
hipError_t commit_all(mca_ctx* ctx, const NetDev& net, int k, int K) {
  if (ctx->norm)
    return mca::launch_norm(net, ctx->nd, ctx->cands, ctx->aux, 0, ctx->pnorm, ctx->lo.nnorm, k,
                            ctx->st, ctx->dl, ctx->stream);
  if (ctx->chan)
    return mca::launch_channel(net, ctx->chans, ctx->aux, 0, ctx->pchan, ctx->lo.nchan, k,
                               ctx->st, ctx->dl, ctx->stream);
  if (ctx->tf)
    return mca::tf_launch_commit(ctx->tfd, ctx->tfh, ctx->cands, ctx->aux, ctx->dl, ctx->st, k,
                                 false, ctx->bsum, ctx->stream);
  // with a layer L-3, its tile kernel also applies a winner of the last two
  // layers (one launch instead of two)
  hipError_t e = hipSuccess;
  if (net.L >= 3)
    e = mca::launch_slab(net, ctx->cands, ctx->aux, 0, ctx->cols, ctx->nnz, ctx->pslab,
                         ctx->lo.nslab, k, ctx->st, ctx->dl, ctx->stream, false, true);
  else
    e = mca::launch_commit(net, ctx->cands, ctx->aux, ctx->dl, ctx->st, k, ctx->lo.ntiles, ctx->stream);
  if (e == hipSuccess && net.L >= 4)
    e = mca::launch_chain(net, ctx->cands, ctx->aux, 0, ctx->rows, ctx->rda, ctx->rcnt,
                          ctx->pchain, ctx->lo.nchain, k, ctx->st, ctx->dl, ctx->stream);
  return e;
}

// Transformer context: validate, lay out, upload, fill the caches.
int tf_init(mca_ctx** out, const mca_net_desc* net, const float* const* params, int32_t n_params,
            const mca_data* data, int32_t k_max, void* workspace, size_t workspace_bytes,
            void* hip_stream) {
  int code;
  std::string msg = tf_check_desc(net, data->n_samples, k_max, &code);
  if (code != MCA_OK) return fail(nullptr, code, msg);
  const TfLayout lo = tf_make_layout(net, data->n_samples, k_max);
  if (n_params != lo.n_tensors) return fail(nullptr, MCA_EINVAL, "n_params must equal the number of Transformer tensors");
  if (data->tokens == nullptr || data->y == nullptr) return fail(nullptr, MCA_EINVAL, "data.tokens or data.y is NULL");
  if (data->n_seq < 1 || (int64_t)data->n_seq * net->ctx != data->n_samples)
    return fail(nullptr, MCA_EINVAL, "n_samples must equal n_seq * ctx");
  if (workspace == nullptr) return fail(nullptr, MCA_EINVAL, "workspace is NULL");
  if (((uintptr_t)workspace) % kAlign != 0) return fail(nullptr, MCA_EINVAL, "workspace is not 256-byte aligned");
  if (workspace_bytes < lo.total) return fail(nullptr, MCA_ENOSPACE, "workspace smaller than mca_plan()");
  const int64_t N = data->n_samples;
  for (int64_t n = 0; n < N; ++n) {
    if (data->tokens[n] < 0 || data->tokens[n] >= net->vocab) return fail(nullptr, MCA_EINVAL, "token out of range");
    if (data->y[n] < 0 || data->y[n] >= net->vocab) return fail(nullptr, MCA_EINVAL, "target out of range");
  }
  mca_ctx* ctx = new (std::nothrow) mca_ctx();
  if (ctx == nullptr) return fail(nullptr, MCA_EINVAL, "out of host memory");
  ctx->tf = true;
  ctx->use_loop = false;
  ctx->desc = *net;
  ctx->k_max = k_max;
  ctx->stream = (hipStream_t)hip_stream;
  ctx->ws = (char*)workspace;
  char* ws = ctx->ws;
  mca::TfDev& h = ctx->tfh;
  h.V = net->vocab;
  h.T = net->ctx;
  h.D = net->d_model;
  h.NB = net->n_block;
  h.H = net->n_head;
  h.M = net->d_mlp;
  h.S = data->n_seq;
  h.n_tensors = lo.n_tensors;
  h.N = N;
  h.eps = net->ln_eps;
  h.delta = net->delta;
  h.bound = net->bound;
  h.ties = net->accept_ties ? 1 : 0;
  h.rule = net->accept_rule;
  h.beta = net->beta;
  h.seed = net->seed;
  h.tag = net->stream_tag;
  const std::vector<TfShape> shapes = tf_shapes(net);
  int64_t off = 0;
  for (int t = 0; t < lo.n_tensors; ++t) {
    h.offs[t] = off;
    h.rows[t] = (int32_t)shapes[t].rows;
    h.cols[t] = (int32_t)shapes[t].cols;
    off += shapes[t].rows * shapes[t].cols;
    h.param[t] = (float*)(ws + lo.param[t]);
  }
  h.offs[lo.n_tensors] = off;
  h.P = off;
  h.tok = (const int32_t*)(ws + lo.tok);
  h.tgt = (const int32_t*)(ws + lo.tgt);
  const int64_t ND = N * h.D;
  for (int b = 0; b <= h.NB; ++b) h.x[b] = (float*)(ws + lo.x) + (int64_t)b * ND;
  h.ell = (float*)(ws + lo.ell);
  for (int b = 0; b < h.NB; ++b) {
    h.ch[b] = (float*)(ws + lo.ch) + (int64_t)b * ND;
  }
  h.cz = (float*)(ws + lo.cz);
  h.sx = (float*)(ws + lo.sx);
  h.sh = (float*)(ws + lo.sh);
  h.slog = (float*)(ws + lo.slog);
  h.sqkv = (float*)(ws + lo.sqkv);
  h.satt = (float*)(ws + lo.satt);
  h.sfc = (float*)(ws + lo.sfc);
  h.sell = (float*)(ws + lo.sell);
  h.sst = (float2*)(ws + lo.sst);
  h.scopy = (float*)(ws + lo.scopy);
  h.copy_stride = lo.copy_stride;
  h.table = (float**)(ws + lo.table);
  h.start = (int32_t*)(ws + lo.start);
  h.xin = (int32_t*)(ws + lo.xin);
  h.kind = (int32_t*)(ws + lo.kind);
  h.run = (int32_t*)(ws + lo.run);
  h.half = (int32_t*)(ws + lo.half);
  h.redo = (int32_t*)(ws + lo.redo);
  h.kr = k_max;
  ctx->tfd = (mca::TfDev*)(ws + lo.dev);
  ctx->tf_nblk = lo.nblk;
  ctx->cands = (mca_cand*)(ws + lo.cands);
  ctx->aux = (Aux*)(ws + lo.aux);
  ctx->partial = (float*)(ws + lo.partial);
  ctx->dl = (double*)(ws + lo.dl);
  ctx->bsum = (double*)(ws + lo.bsum);
  ctx->st = (DevState*)(ws + lo.state);
  ctx->snap = (DevState*)(ws + lo.state + 256);
  ctx->loop_sync = (mca::LoopSync*)(ws + lo.state + 512);
  ctx->tr_chosen = (int32_t*)(ws + lo.tr_chosen);
  ctx->tr_dl = (double*)(ws + lo.tr_dl);
  // what the shared selection and state calls read
  NetDev& nd = ctx->net;
  nd.L = 0;
  nd.C = h.V;
  nd.ties = h.ties;
  nd.rule = h.rule;
  nd.beta = h.beta;
  nd.N = N;
  nd.Ns = N;
  nd.P = h.P;
  nd.ell = h.ell;
  {
    hipError_t e = hipMemcpyAsync((void*)h.tok, data->tokens, (size_t)N * sizeof(int32_t), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync((void*)h.tgt, data->y, (size_t)N * sizeof(int32_t), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync(ctx->tfd, &h, sizeof h, hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) {
      device_fail(nullptr, e, "upload of the data set");
      delete ctx;
      return MCA_EDEVICE;
    }
  }
  int rc = upload_params(ctx, params, nullptr);
  if (rc == MCA_OK) rc = write_state(ctx, 0, false);
  if (rc == MCA_OK) rc = run_forward(ctx);
  if (rc == MCA_OK) {
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) rc = device_fail(ctx, e, "forward pass");
  }
  if (rc != MCA_OK) {
    g_thread_error = ctx->err;
    delete ctx;
    return rc;
  }
  // pinned host memory for the state read-back of every run_steps call (a
  // plain host buffer is used if it cannot be had)
  if (hipHostMalloc((void**)&ctx->host_blk, kStateBlock, hipHostMallocDefault) != hipSuccess) {
    ctx->host_blk = nullptr;
    (void)hipGetLastError();
  }
  *out = ctx;
  return MCA_OK;
}

}  // namespace

extern "C" {

int mca_abi_version(void) { return MCA_ABI_VERSION; }

size_t mca_struct_size(int32_t which) {
  switch (which) {
    case 0: return sizeof(mca_net_desc);
    case 1: return sizeof(mca_cand);
    case 2: return sizeof(mca_data);
    case 3: return sizeof(mca_stats);
    case 4: return sizeof(mca_trace);
    case 5: return sizeof(mca_timing);
    case 6: return sizeof(mca_channel);
    default: return 0;
  }
}

int mca_plan(const mca_net_desc* net, int64_t n_samples, int32_t k_max, size_t* workspace_bytes) {
  int code;
  if (net != nullptr && net->kind == MCA_NET_TRANSFORMER) {
    std::string msg = tf_check_desc(net, n_samples, k_max, &code);
    if (code != MCA_OK) return fail(nullptr, code, msg);
    if (workspace_bytes == nullptr) return fail(nullptr, MCA_EINVAL, "workspace_bytes is NULL");
    *workspace_bytes = tf_make_layout(net, n_samples, k_max).total;
    return MCA_OK;
  }
  std::string msg = check_desc(net, n_samples, k_max, &code);
  if (code != MCA_OK) return fail(nullptr, code, msg);
  if (workspace_bytes == nullptr) return fail(nullptr, MCA_EINVAL, "workspace_bytes is NULL");
  *workspace_bytes = make_layout(net, n_samples, k_max).total;
  return MCA_OK;
}

int mca_init(mca_ctx** out, const mca_net_desc* net, const float* const* params, int32_t n_params,
             const int8_t* const* codes, const mca_data* data, int32_t k_max, void* workspace,
             size_t workspace_bytes, void* hip_stream) {
  if (out == nullptr) return fail(nullptr, MCA_EINVAL, "out is NULL");
  *out = nullptr;
  if (data == nullptr) return fail(nullptr, MCA_EINVAL, "data is NULL");
  if (net != nullptr && net->kind == MCA_NET_TRANSFORMER)
    return tf_init(out, net, params, n_params, data, k_max, workspace, workspace_bytes, hip_stream);
  int code;
  std::string msg = check_desc(net, data->n_samples, k_max, &code);
  if (code != MCA_OK) return fail(nullptr, code, msg);
  if (n_params != net->n_layers) return fail(nullptr, MCA_EINVAL, "n_params must equal n_layers");
  if (data->x == nullptr || data->y == nullptr) return fail(nullptr, MCA_EINVAL, "data.x or data.y is NULL");
  if (workspace == nullptr) return fail(nullptr, MCA_EINVAL, "workspace is NULL");
  if (((uintptr_t)workspace) % kAlign != 0) return fail(nullptr, MCA_EINVAL, "workspace is not 256-byte aligned");
  const int64_t N = data->n_samples;
  const Layout lo = make_layout(net, N, k_max);
  if (workspace_bytes < lo.total) return fail(nullptr, MCA_ENOSPACE, "workspace smaller than mca_plan()");
  const int L = net->n_layers, C = net->widths[L], n0 = net->widths[0];
  for (int64_t n = 0; n < N; ++n)
    if (data->y[n] < 0 || data->y[n] >= C) return fail(nullptr, MCA_EINVAL, "label out of range");
  for (int64_t e = 0; e < N * n0; ++e)
    if (!std::isfinite(data->x[e])) return fail(nullptr, MCA_EINVAL, "non-finite input");

  mca_ctx* ctx = new (std::nothrow) mca_ctx();
  if (ctx == nullptr) return fail(nullptr, MCA_EINVAL, "out of host memory");
  ctx->desc = *net;
  ctx->lo = lo;
  ctx->k_max = k_max;
  ctx->stream = (hipStream_t)hip_stream;
  ctx->ws = (char*)workspace;
  char* ws = ctx->ws;
  NetDev& nd = ctx->net;
  nd.L = L;
  nd.C = C;
  nd.act = net->act;
  nd.gamma = net->gamma;
  nd.ternary = net->weight_mode == MCA_WEIGHTS_TERNARY;
  nd.pick = net->pick;
  nd.delta = net->delta;
  nd.bound = net->bound;
  nd.ties = net->accept_ties ? 1 : 0;
  nd.rule = net->accept_rule;
  nd.beta = net->beta;
  nd.n_prune = net->n_prune;
  nd.sub_size = net->subset_size;
  nd.sub_period = net->subset_size ? net->subset_period : 1;
  nd.seed = net->seed;
  nd.tag = net->stream_tag;
  nd.N = N;
  nd.Ns = lo.Ns;
  nd.mutation = net->mutation;
  for (int l = 0; l < L; ++l) nd.chan_amp[l] = (float)std::sqrt(8.0 / (double)net->widths[l]);
  nd.bias = net->biases;
  nd.ln = net->layer_norm;
  nd.ln_eps = net->ln_eps;
  nd.sticky = net->pick == MCA_PICK_STICKY ? net->sticky_steps : 1;
  int64_t off = 0;
  for (int l = 0; l <= L; ++l) nd.widths[l] = net->widths[l];
  for (int l = 0; l < L; ++l) {
    nd.offs[l] = off;
    off += (int64_t)net->widths[l + 1] * (net->widths[l] + net->biases);
    nd.B[l] = net->biases ? (float*)(ws + lo.b[l]) : nullptr;
    nd.scales[l] = net->scales[l];
    nd.W[l] = (float*)(ws + lo.w[l]);
    nd.codes[l] = nd.ternary ? (int8_t*)(ws + lo.codes[l]) : nullptr;
    nd.Z[l] = (float*)(ws + lo.z[l]);
  }
  nd.offs[L] = off;
  nd.P = off;
  nd.XT = (const float*)(ws + lo.xt);
  nd.ell = (float*)(ws + lo.ell);
  nd.prob = (float*)(ws + lo.pr);
  nd.y = (const int32_t*)(ws + lo.y);
  ctx->norm = dense_path(net);
  const bool slab = L >= 3 && !ctx->norm;
  nd.WT = slab ? (float*)(ws + lo.wt) : nullptr;
  ctx->pslab = slab ? (float*)(ws + lo.pslab) : nullptr;
  ctx->cols = slab ? (uint64_t*)(ws + lo.cols) : nullptr;
  ctx->nnz = slab ? (int*)(ws + lo.nnz) : nullptr;
  if (ctx->norm) {
    for (int l = 0; l + 1 < L && net->layer_norm; ++l) {
      ctx->nd.MU[l] = (float*)(ws + lo.mu[l]);
      ctx->nd.S[l] = (float*)(ws + lo.S[l]);
    }
    ctx->pnorm = (float*)(ws + lo.pnorm);
    ctx->use_loop = false;
  }
  ctx->chan = net->mutation != MCA_MUTATE_SINGLE;
  const bool deep = L >= 4 && !ctx->chan && !ctx->norm;
  ctx->rows = deep ? (int*)(ws + lo.rows) : nullptr;
  ctx->rda = deep ? (float*)(ws + lo.rda) : nullptr;
  ctx->rcnt = deep ? (int*)(ws + lo.rcnt) : nullptr;
  ctx->pchain = deep ? (float*)(ws + lo.pchain) : nullptr;
  ctx->chans = ctx->chan ? (mca_channel*)(ws + lo.chans) : nullptr;
  ctx->pchan = ctx->chan ? (float*)(ws + lo.pchan) : nullptr;
  if (ctx->chan) ctx->use_loop = false;
  ctx->cands = (mca_cand*)(ws + lo.cands);
  ctx->aux = (Aux*)(ws + lo.aux);
  ctx->fmask = lo.ntiles_ev <= 64 ? (uint64_t*)(ws + lo.fmask) : nullptr;
  ctx->cmask = (uint64_t*)(ws + lo.cmask);
  ctx->partial = (float*)(ws + lo.partial);
  ctx->dl = (double*)(ws + lo.dl);
  ctx->bsum = (double*)(ws + lo.bsum);
  ctx->st = (DevState*)(ws + lo.state);
  ctx->snap = (DevState*)(ws + lo.state + 256);
  ctx->loop_sync = (mca::LoopSync*)(ws + lo.state + 512);
  ctx->tr_chosen = (int32_t*)(ws + lo.tr_chosen);
  ctx->tr_dl = (double*)(ws + lo.tr_dl);
  ctx->loop_partials = (uint64_t*)(ws + lo.loop_partials);
  ctx->loop_dls = (uint64_t*)(ws + lo.loop_dls);

  // inputs, transposed to the unit-major layout (zero padding to Ns)
  {
    std::vector<float> xt((size_t)n0 * lo.Ns, 0.f);
    for (int64_t n = 0; n < N; ++n)
      for (int i = 0; i < n0; ++i) xt[(size_t)i * lo.Ns + n] = data->x[(size_t)n * n0 + i];
    std::vector<int32_t> y((size_t)lo.Ns, 0);
    std::memcpy(y.data(), data->y, (size_t)N * sizeof(int32_t));
    // per feature, the evaluation tiles holding a non-zero sample
    std::vector<uint64_t> fm((size_t)n0, 0);
    if (ctx->fmask)
      for (int i = 0; i < n0; ++i)
        for (int64_t n = 0; n < N; ++n)
          if (xt[(size_t)i * lo.Ns + n] != 0.f) fm[i] |= 1ull << (n / mca::eval_tile_size());
    hipError_t e = hipMemcpyAsync((void*)nd.XT, xt.data(), xt.size() * sizeof(float), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess && ctx->fmask)
      e = hipMemcpyAsync(ctx->fmask, fm.data(), fm.size() * sizeof(uint64_t), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipMemcpyAsync((void*)nd.y, y.data(), y.size() * sizeof(int32_t), hipMemcpyHostToDevice, ctx->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) {
      device_fail(nullptr, e, "upload of the data set");
      delete ctx;
      return MCA_EDEVICE;
    }
  }
  int rc = upload_params(ctx, params, codes);
  if (rc == MCA_OK) rc = write_state(ctx, 0, false);
  if (rc == MCA_OK) rc = run_forward(ctx);
  if (rc == MCA_OK) {
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) rc = device_fail(ctx, e, "forward pass");
  }
  if (rc == MCA_OK) {
    hipError_t e = scratch_for_current_device(&ctx->scratch_dev);
    if (e != hipSuccess) rc = device_fail(ctx, e, "hipGetSymbolAddress(scratch)");
  }
  if (rc != MCA_OK) {
    g_thread_error = ctx->err;
    delete ctx;
    return rc;
  }
  // pinned host memory for the state read-back of every run_steps call (a
  // plain host buffer is used if it cannot be had)
  if (hipHostMalloc((void**)&ctx->host_blk, kStateBlock, hipHostMallocDefault) != hipSuccess) {
    ctx->host_blk = nullptr;
    (void)hipGetLastError();
  }
  *out = ctx;
  return MCA_OK;
}

int mca_propose(mca_ctx* ctx, uint64_t step, int32_t K, mca_cand* out_host) {
  MCA_LIVE(ctx);
  if (ctx->chan) return fail(ctx, MCA_EINVAL, "a channel context proposes mca_channel records (mca_propose_channels)");
  if (K < 1 || K > ctx->k_max) return fail(ctx, MCA_EINVAL, "K out of range [1, k_max]");
  if (out_host == nullptr) return fail(ctx, MCA_EINVAL, "out_host is NULL");
  // the proposal reuses the candidate buffers of a pending batch
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  MCA_HIP(ctx, timed(ctx, 0, [&] { return propose_dev(ctx, step, false, K); }));
  MCA_HIP(ctx, hipMemcpyAsync(out_host, ctx->cands, (size_t)K * sizeof(mca_cand), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int mca_eval_losses(mca_ctx* ctx, const mca_cand* cands_host, int32_t K, double* loss_out,
                    double* dloss_out) {
  MCA_LIVE(ctx);
  if (ctx->chan) return fail(ctx, MCA_EINVAL, "a channel context scores mca_channel records (mca_eval_channels)");
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is already pending");
  if (K < 1 || K > ctx->k_max) return fail(ctx, MCA_EINVAL, "K out of range [1, k_max]");
  if (cands_host == nullptr) return fail(ctx, MCA_EINVAL, "cands_host is NULL");
  int rc = check_cands(ctx, cands_host, K);
  if (rc != MCA_OK) return rc;
  MCA_HIP(ctx, hipMemcpyAsync(ctx->cands, cands_host, (size_t)K * sizeof(mca_cand), hipMemcpyHostToDevice, ctx->stream));
  MCA_HIP(ctx, timed(ctx, 0, [&] { return prepare_dev(ctx, K); }));
  MCA_HIP(ctx, timed(ctx, 1, [&] { return eval_all(ctx, ctx->net, K); }));
  MCA_HIP(ctx, timed(ctx, 2, [&] { return select_all(ctx, ctx->net, K, false, nullptr, nullptr); }));
  std::vector<double> dl(K);
  DevState s{};
  MCA_HIP(ctx, hipMemcpyAsync(dl.data(), ctx->dl, (size_t)K * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipMemcpyAsync(&s, ctx->st, sizeof s, hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  for (int k = 0; k < K; ++k) {
    if (loss_out) loss_out[k] = s.L + dl[k];
    if (dloss_out) dloss_out[k] = dl[k];
  }
  ctx->pending = true;
  ctx->pending_K = K;
  ctx->pending_dl = dl;
  return MCA_OK;
}

int mca_commit(mca_ctx* ctx, int32_t k) {
  MCA_LIVE(ctx);
  if (!ctx->pending) return fail(ctx, MCA_ESTATE, "no pending batch");
  if (k < 0 || k >= ctx->pending_K) return fail(ctx, MCA_EINVAL, "k outside the pending batch");
  if (k < (int)ctx->pending_dl.size() && !std::isfinite(ctx->pending_dl[k]))
    return fail(ctx, MCA_EINVAL, "candidate k was rejected unevaluated (weight bound): it cannot be committed");
  MCA_HIP(ctx, timed(ctx, 3, [&] { return commit_all(ctx, ctx->net, k, ctx->pending_K); }));
  if (!ctx->tf && ctx->net.sub_size > 0)  // the loss over every sample, from the logits
    MCA_HIP(ctx, mca::launch_loss_refresh(ctx->net, ctx->bsum, ctx->st, ctx->stream));
  ctx->pending = false;
  ctx->pending_K = 0;
  return MCA_OK;
}

int mca_rollback(mca_ctx* ctx) {
  MCA_LIVE(ctx);
  if (!ctx->pending) return fail(ctx, MCA_ESTATE, "no pending batch");
  ctx->pending = false;
  ctx->pending_K = 0;
  return MCA_OK;
}

int mca_propose_channels(mca_ctx* ctx, uint64_t step, int32_t K, mca_channel* out_host) {
  MCA_LIVE(ctx);
  if (!ctx->chan) return fail(ctx, MCA_EINVAL, "not a channel context");
  if (K < 1 || K > ctx->k_max) return fail(ctx, MCA_EINVAL, "K out of range [1, k_max]");
  if (out_host == nullptr) return fail(ctx, MCA_EINVAL, "out_host is NULL");
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  MCA_HIP(ctx, timed(ctx, 0, [&] { return propose_dev(ctx, step, false, K); }));
  MCA_HIP(ctx, hipMemcpyAsync(out_host, ctx->chans, (size_t)K * sizeof(mca_channel), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int mca_eval_channels(mca_ctx* ctx, const mca_channel* chans_host, int32_t K, double* loss_out,
                      double* dloss_out) {
  MCA_LIVE(ctx);
  if (!ctx->chan) return fail(ctx, MCA_EINVAL, "not a channel context");
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is already pending");
  if (K < 1 || K > ctx->k_max) return fail(ctx, MCA_EINVAL, "K out of range [1, k_max]");
  if (chans_host == nullptr) return fail(ctx, MCA_EINVAL, "chans_host is NULL");
  const mca_net_desc& d = ctx->desc;
  for (int k = 0; k < K; ++k) {
    for (int m = 0; m <= d.n_layers; ++m)
      if (chans_host[k].units[m] < 0 || chans_host[k].units[m] >= d.widths[m])
        return fail(ctx, MCA_EINVAL, "channel unit out of range");
    for (int m = 0; m < d.n_layers; ++m)
      if (!std::isfinite(chans_host[k].w_new[m])) return fail(ctx, MCA_EINVAL, "channel weight is not finite");
  }
  MCA_HIP(ctx, hipMemcpyAsync(ctx->chans, chans_host, (size_t)K * sizeof(mca_channel), hipMemcpyHostToDevice, ctx->stream));
  MCA_HIP(ctx, timed(ctx, 0, [&] { return prepare_dev(ctx, K); }));
  MCA_HIP(ctx, timed(ctx, 1, [&] { return eval_all(ctx, ctx->net, K); }));
  MCA_HIP(ctx, timed(ctx, 2, [&] { return select_all(ctx, ctx->net, K, false, nullptr, nullptr); }));
  std::vector<double> dl(K);
  DevState s{};
  MCA_HIP(ctx, hipMemcpyAsync(dl.data(), ctx->dl, (size_t)K * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipMemcpyAsync(&s, ctx->st, sizeof s, hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  for (int k = 0; k < K; ++k) {
    if (loss_out) loss_out[k] = s.L + dl[k];
    if (dloss_out) dloss_out[k] = dl[k];
  }
  ctx->pending = true;
  ctx->pending_K = K;
  ctx->pending_dl = dl;
  return MCA_OK;
}

int mca_eval_losses_noalloc(mca_ctx* ctx, const mca_cand* cands_host, int32_t K,
                            double* loss_out, double* dloss_out) {
  MCA_LIVE(ctx);
  if (ctx->tf) return fail(ctx, MCA_EUNSUPPORTED, "the no-allocation evaluation takes MLP contexts");
  if (ctx->chan || ctx->norm)
    return fail(ctx, MCA_EUNSUPPORTED, "the no-allocation evaluation takes nets without biases or normalization and single mutations");
  if (K < 1 || K > mca::kMaxK) return fail(ctx, MCA_EINVAL, "K out of range [1, 1024]");
  if (cands_host == nullptr) return fail(ctx, MCA_EINVAL, "cands_host is NULL");
  if (ctx->scratch_dev == nullptr) return fail(ctx, MCA_EDEVICE, "no scratch array on this device");
  int rc = check_cands(ctx, cands_host, K);
  if (rc != MCA_OK) return rc;
  // the per-call buffers, carved from the scratch array in the workspace's
  // order and alignment
  const Layout& lo = ctx->lo;
  const NetDev& net = ctx->net;
  const int L = net.L;
  const size_t kk = (size_t)K;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t o_cands = take(kk * sizeof(mca_cand)), o_aux = take(kk * sizeof(Aux));
  const size_t o_cmask = take(kk * sizeof(uint64_t));
  const size_t o_partial = take(kk * lo.ntiles_ev * sizeof(float)), o_dl = take(kk * sizeof(double));
  size_t o_pslab = 0, o_cols = 0, o_nnz = 0, o_rows = 0, o_rda = 0, o_rcnt = 0, o_pchain = 0;
  if (L >= 3) {
    o_pslab = take(kk * lo.nslab * sizeof(float));
    o_cols = take(kk * net.widths[L - 1] * sizeof(uint64_t));
    o_nnz = take(kk * sizeof(int32_t));
  }
  if (L >= 4) {
    o_rows = take(kk * net.N * sizeof(int32_t));
    o_rda = take(kk * net.N * sizeof(float));
    o_rcnt = take(kk * sizeof(int32_t));
    o_pchain = take(kk * lo.nchain * sizeof(float));
  }
  if (off > kScratchBytes)
    return fail(ctx, MCA_EINVAL, "K candidates on this net need " + std::to_string(off) +
                                     " bytes of scratch, more than the static array's " +
                                     std::to_string(kScratchBytes));
  char* base = (char*)ctx->scratch_dev;
  const Bufs b{(mca_cand*)(base + o_cands), (Aux*)(base + o_aux), (uint64_t*)(base + o_cmask),
               (float*)(base + o_partial), (double*)(base + o_dl),
               L >= 3 ? (float*)(base + o_pslab) : nullptr,
               L >= 3 ? (uint64_t*)(base + o_cols) : nullptr,
               L >= 3 ? (int*)(base + o_nnz) : nullptr,
               L >= 4 ? (int*)(base + o_rows) : nullptr,
               L >= 4 ? (float*)(base + o_rda) : nullptr,
               L >= 4 ? (int*)(base + o_rcnt) : nullptr,
               L >= 4 ? (float*)(base + o_pchain) : nullptr};
  // every scratch word a kernel reads is written earlier in this call (the
  // prepared values, masks, lists, counts, tile sums and loss changes), so
  // nothing is cleared; overlapping calls on one GPU would race on them
  MCA_HIP(ctx, hipMemcpyAsync(b.cands, cands_host, kk * sizeof(mca_cand), hipMemcpyHostToDevice, ctx->stream));
  MCA_HIP(ctx, prepare_into(ctx, b, K));
  MCA_HIP(ctx, eval_into(ctx, net, b, K));
  MCA_HIP(ctx, select_into(ctx, net, b, K, false, nullptr, nullptr));
  std::vector<double> dl(K);
  double L_c = 0.0;
  MCA_HIP(ctx, hipMemcpyAsync(dl.data(), b.dl, kk * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipMemcpyAsync(&L_c, &ctx->st->L, sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  for (int k = 0; k < K; ++k) {
    if (loss_out) loss_out[k] = L_c + dl[k];
    if (dloss_out) dloss_out[k] = dl[k];
  }
  return MCA_OK;
}

int mca_set_option(mca_ctx* ctx, int32_t option, int64_t value) {
  MCA_LIVE(ctx);
  if (option == MCA_OPT_PERSISTENT_LOOP) {
    if (value != 0 && value != 1) return fail(ctx, MCA_EINVAL, "MCA_OPT_PERSISTENT_LOOP takes 0 or 1");
    // nets with biases or normalization and channel mutations have no device
    // loop kernel: they keep the per-phase loop either way
    ctx->use_loop = value != 0 && !ctx->norm && !ctx->chan;
    return MCA_OK;
  }
  if (option == MCA_OPT_LOOP_LAUNCH) {
    if (value != 0 && value != 1) return fail(ctx, MCA_EINVAL, "MCA_OPT_LOOP_LAUNCH takes 0 or 1");
    ctx->loop_coop = value == 0;
    return MCA_OK;
  }
  if (option == MCA_OPT_LOOP_TILE) {
    if (ctx->tf) return fail(ctx, MCA_EINVAL, "MCA_OPT_LOOP_TILE applies to MLP contexts");
    if (value < kMinLoopTile || value > 64) return fail(ctx, MCA_EINVAL, "MCA_OPT_LOOP_TILE takes 16..64");
    ctx->lo.loop_T = (int)value;
    ctx->lo.loop_G = (int)((ctx->net.N + value - 1) / value);
    return MCA_OK;
  }
  return fail(ctx, MCA_EINVAL, "unknown option");
}

int mca_set_step(mca_ctx* ctx, uint64_t next_step) {
  MCA_LIVE(ctx);
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  hipLaunchKernelGGL(k_set_next_step, dim3(1), dim3(1), 0, ctx->stream, ctx->st, next_step);
  MCA_HIP(ctx, hipGetLastError());
  return MCA_OK;
}

int mca_run_steps(mca_ctx* ctx, uint64_t n_steps, int32_t K, mca_trace* trace, mca_stats* stats) {
  MCA_LIVE(ctx);
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  if (K < 1 || K > ctx->k_max) return fail(ctx, MCA_EINVAL, "K out of range [1, k_max]");
  if (trace != nullptr && trace->chosen == nullptr) return fail(ctx, MCA_EINVAL, "trace.chosen is NULL");
  // Nothing is read back until the end: the device state supplies each
  // launch's first step, a snapshot kernel records the counters the call's
  // statistics are taken against, and one copy returns state, snapshot and
  // abort word together.
  const NetDev& net = ctx->net;
  uint64_t done = 0;
  const bool mlp2 = !ctx->tf && net.L <= 2;
  if (ctx->use_loop && mlp2 && K <= mca::kLoopMaxK && ctx->loop_fit_K != K) {
    int fit = 0;
    MCA_HIP(ctx, mca::step_loop_max_blocks(K, net.C, &fit));
    ctx->loop_fit = fit;
    ctx->loop_fit_K = K;
  }
  // row offsets of the loop's arrays are 32-bit element counts
  bool offsets_fit = true;
  for (int l = 0; l < net.L; ++l)
    if ((uint64_t)net.widths[l] * (uint64_t)net.Ns >= ((uint64_t)1 << 32)) offsets_fit = false;
  // a net whose samples fit one workgroup, with a few candidates per step:
  // the one-workgroup loop (no exchange between workgroups)
  const bool one_ok = ctx->use_loop && mlp2 && mca::one_loop_fits(net, K);
  // G tile workgroups plus the candidate reducers must all be resident at once
  const bool loop_ok = !one_ok && ctx->use_loop && mlp2 && offsets_fit && K <= mca::kLoopMaxK &&
                       ctx->lo.loop_G <= mca::kLoopMaxTiles &&
                       ctx->lo.loop_G + mca::step_loop_reducers(K) <= ctx->loop_fit;
  // the call's start (counter snapshot, abort word cleared): in the loop's
  // first reset launch, or a launch of its own
  bool started = false;
  if (!loop_ok || n_steps == 0) {
    hipLaunchKernelGGL(k_call_start, dim3(1), dim3(1), 0, ctx->stream, ctx->st, ctx->snap,
                       ctx->loop_sync);
    MCA_HIP(ctx, hipGetLastError());
    started = true;
  }
  while (one_ok && done < n_steps) {
    const uint64_t cap = trace ? (uint64_t)kTraceCap : ((uint64_t)1 << 22);
    const uint64_t chunk = std::min<uint64_t>(n_steps - done, cap);
    mca::OneArgs a{};
    a.net = net;
    a.K = K;
    a.n_steps = chunk;
    a.st = ctx->st;
    a.tr_chosen = trace ? ctx->tr_chosen : nullptr;
    a.tr_dl = (trace && trace->dloss) ? ctx->tr_dl : nullptr;
    a.tr_cap = kTraceCap;
    MCA_HIP(ctx, timed(ctx, 6, [&] { return mca::launch_one_loop(a, ctx->stream); }));
    if (trace != nullptr) {  // the next chunk reuses the device trace buffers
      MCA_HIP(ctx, hipMemcpyAsync(trace->chosen + done, ctx->tr_chosen, chunk * sizeof(int32_t), hipMemcpyDeviceToHost, ctx->stream));
      if (trace->dloss)
        MCA_HIP(ctx, hipMemcpyAsync(trace->dloss + done * K, ctx->tr_dl, chunk * K * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
      MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
    }
    done += chunk;
  }
  while (loop_ok && done < n_steps) {
    const uint64_t cap = trace ? (uint64_t)kTraceCap : ((uint64_t)1 << 22);
    const uint64_t chunk = std::min<uint64_t>(n_steps - done, cap);
    mca::LoopArgs a{};
    a.net = net;
    a.K = K;
    a.T = ctx->lo.loop_T;
    a.n_steps = chunk;
    a.G = ctx->lo.loop_G;
    a.gpad = (ctx->lo.loop_G + 15) / 16 * 16;
    a.partials = ctx->loop_partials;
    a.dls = ctx->loop_dls;
    a.sync = ctx->loop_sync;
    a.st = ctx->st;
    a.tr_chosen = trace ? ctx->tr_chosen : nullptr;
    a.tr_dl = (trace && trace->dloss) ? ctx->tr_dl : nullptr;
    a.tr_cap = kTraceCap;
    a.spin_limit = 1u << 22;
    MCA_HIP(ctx, mca::launch_loop_reset(a, started ? nullptr : ctx->snap, ctx->stream));
    started = true;
    MCA_HIP(ctx, timed(ctx, 4, [&] { return mca::launch_step_loop(a, ctx->loop_coop, ctx->stream); }));
    if (trace != nullptr) {  // the next chunk reuses the device trace buffers
      MCA_HIP(ctx, hipMemcpyAsync(trace->chosen + done, ctx->tr_chosen, chunk * sizeof(int32_t), hipMemcpyDeviceToHost, ctx->stream));
      if (trace->dloss)
        MCA_HIP(ctx, hipMemcpyAsync(trace->dloss + done * K, ctx->tr_dl, chunk * K * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
      MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
    }
    done += chunk;
  }
  while (done < n_steps) {
    const uint64_t chunk = std::min<uint64_t>(n_steps - done, (uint64_t)kTraceCap);
    int32_t* trc = nullptr;
    double* trd = nullptr;
    if (trace != nullptr) {
      hipLaunchKernelGGL(k_set_trace_base, dim3(1), dim3(1), 0, ctx->stream, ctx->st);
      MCA_HIP(ctx, hipGetLastError());
      trc = ctx->tr_chosen;
      trd = trace->dloss ? ctx->tr_dl : nullptr;
    }
    for (uint64_t s = 0; s < chunk; ++s) {
      MCA_HIP(ctx, timed(ctx, 0, [&] { return propose_step(ctx, net, K); }));
      MCA_HIP(ctx, timed(ctx, 1, [&] { return eval_all(ctx, net, K, fused_proposal(ctx, net)); }));
      MCA_HIP(ctx, timed(ctx, 2, [&] { return select_all(ctx, net, K, true, trc, trd); }));
      MCA_HIP(ctx, timed(ctx, 3, [&] { return commit_all(ctx, net, -1, K); }));
    }
    if (trace != nullptr) {
      MCA_HIP(ctx, hipMemcpyAsync(trace->chosen + done, ctx->tr_chosen, chunk * sizeof(int32_t), hipMemcpyDeviceToHost, ctx->stream));
      if (trace->dloss)
        MCA_HIP(ctx, hipMemcpyAsync(trace->dloss + done * K, ctx->tr_dl, chunk * K * sizeof(double), hipMemcpyDeviceToHost, ctx->stream));
      MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
    }
    done += chunk;
  }
  if (!ctx->tf && net.sub_size > 0)  // the loss over every sample, from the logits
    MCA_HIP(ctx, mca::launch_loss_refresh(net, ctx->bsum, ctx->st, ctx->stream));
  // state, snapshot and abort word: one copy (into pinned memory when the
  // context has it)
  alignas(8) unsigned char local[kStateBlock];
  unsigned char* blk = ctx->host_blk ? ctx->host_blk : local;
  MCA_HIP(ctx, hipMemcpyAsync(blk, ctx->st, kStateBlock, hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, wait_stream(ctx->stream));
  DevState after, before;
  mca::LoopSync sync;
  std::memcpy(&after, blk, sizeof after);
  std::memcpy(&before, blk + 256, sizeof before);
  std::memcpy(&sync, blk + 512, sizeof sync);
  if (sync.abort != 0) {
    ctx->poisoned = true;
    return fail(ctx, MCA_EDEVICE, "step loop aborted: a bounded wait between workgroups ran out");
  }
  if (stats != nullptr) {
    stats->steps = after.steps - before.steps;
    stats->evaluated = after.evaluated - before.evaluated;
    stats->accepted = after.accepted - before.accepted;
    stats->wasted = after.wasted - before.wasted;
    stats->tie_band = after.tie - before.tie;
    stats->loss = after.L;
    stats->next_step = after.t;
  }
  return MCA_OK;
}

int mca_get_params(mca_ctx* ctx, float* const* params_out, int8_t* const* codes_out) {
  MCA_LIVE(ctx);
  if (params_out == nullptr) return fail(ctx, MCA_EINVAL, "params_out is NULL");
  const mca_net_desc& d = ctx->desc;
  if (ctx->tf) {
    for (int t = 0; t < ctx->tfh.n_tensors; ++t) {
      if (params_out[t] == nullptr) return fail(ctx, MCA_EINVAL, "a params_out pointer is NULL");
      const size_t n = (size_t)ctx->tfh.rows[t] * ctx->tfh.cols[t];
      MCA_HIP(ctx, hipMemcpyAsync(params_out[t], ctx->tfh.param[t], n * sizeof(float), hipMemcpyDeviceToHost, ctx->stream));
    }
    MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
    return MCA_OK;
  }
  for (int l = 0; l < d.n_layers; ++l) {
    const size_t n = (size_t)d.widths[l + 1] * d.widths[l];
    if (params_out[l] == nullptr) return fail(ctx, MCA_EINVAL, "a params_out pointer is NULL");
    if (d.biases) {
      const size_t w = (size_t)d.widths[l], rows = (size_t)d.widths[l + 1];
      MCA_HIP(ctx, hipMemcpy2DAsync(params_out[l], (w + 1) * sizeof(float), ctx->net.W[l], w * sizeof(float),
                                    w * sizeof(float), rows, hipMemcpyDeviceToHost, ctx->stream));
      MCA_HIP(ctx, hipMemcpy2DAsync(params_out[l] + w, (w + 1) * sizeof(float), ctx->net.B[l], sizeof(float),
                                    sizeof(float), rows, hipMemcpyDeviceToHost, ctx->stream));
      continue;
    }
    MCA_HIP(ctx, hipMemcpyAsync(params_out[l], ctx->net.W[l], n * sizeof(float), hipMemcpyDeviceToHost, ctx->stream));
    if (codes_out != nullptr && ctx->net.ternary && codes_out[l] != nullptr)
      MCA_HIP(ctx, hipMemcpyAsync(codes_out[l], ctx->net.codes[l], n, hipMemcpyDeviceToHost, ctx->stream));
  }
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int mca_get_loss(mca_ctx* ctx, double* loss, uint64_t* next_step) {
  MCA_LIVE(ctx);
  DevState s{};
  int rc = read_state(ctx, &s);
  if (rc != MCA_OK) return rc;
  if (loss) *loss = s.L;
  if (next_step) *next_step = s.t;
  return MCA_OK;
}

int mca_set_state(mca_ctx* ctx, const float* const* params, const int8_t* const* codes,
                  uint64_t next_step) {
  MCA_LIVE(ctx);
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  int rc = upload_params(ctx, params, codes);
  if (rc == MCA_OK) rc = write_state(ctx, next_step, true);
  if (rc == MCA_OK) rc = run_forward(ctx);
  if (rc == MCA_OK) MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return rc;
}

int mca_refresh(mca_ctx* ctx) {
  MCA_LIVE(ctx);
  if (ctx->pending) return fail(ctx, MCA_ESTATE, "a batch is pending: commit or roll back first");
  int rc = run_forward(ctx);
  if (rc == MCA_OK) MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return rc;
}

int mca_get_sample_losses(mca_ctx* ctx, float* out_host) {
  MCA_LIVE(ctx);
  if (out_host == nullptr) return fail(ctx, MCA_EINVAL, "out_host is NULL");
  if (ctx->tf) {
    // a winner scored incrementally has its per-position losses recomputed
    // in the next evaluation pass: run that recomputation alone and fold it
    // in (no winner), so the copy holds the committed losses
    MCA_HIP(ctx, mca::tf_launch_eval(ctx->tfd, ctx->tfh, ctx->cands, ctx->aux, 0, false,
                                     ctx->partial, ctx->tf_nblk, ctx->stream));
    MCA_HIP(ctx, mca::tf_launch_commit(ctx->tfd, ctx->tfh, ctx->cands, ctx->aux, ctx->dl,
                                       ctx->st, -2, false, ctx->bsum, ctx->stream));
  }
  MCA_HIP(ctx, hipMemcpyAsync(out_host, ctx->net.ell, (size_t)ctx->net.N * sizeof(float), hipMemcpyDeviceToHost, ctx->stream));
  MCA_HIP(ctx, hipStreamSynchronize(ctx->stream));
  return MCA_OK;
}

int mca_set_timing(mca_ctx* ctx, int32_t phase_mask) {
  MCA_LIVE(ctx);
  ctx->timing = phase_mask;
  // events for the first timed launches are made here, not inside them: an
  // event's creation costs tens of microseconds of host time
  while (phase_mask != 0 && ctx->pool.size() < kEventsAhead) {
    hipEvent_t e = nullptr;
    MCA_HIP(ctx, hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    ctx->pool.push_back(e);
  }
  return MCA_OK;
}

int mca_get_timing(mca_ctx* ctx, mca_timing* out, int32_t reset) {
  MCA_LIVE(ctx);
  int rc = flush_timing(ctx);
  if (rc != MCA_OK) return rc;
  if (out) *out = ctx->acc;
  if (reset) ctx->acc = mca_timing{};
  return MCA_OK;
}

void mca_destroy(mca_ctx* ctx) {
  if (ctx == nullptr) return;
  if (!ctx->poisoned) (void)hipStreamSynchronize(ctx->stream);
  for (auto& r : ctx->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : ctx->pool) (void)hipEventDestroy(e);
  if (ctx->host_blk) (void)hipHostFree(ctx->host_blk);
  delete ctx;
}

const char* mca_last_error(const mca_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_thread_error.c_str();
}

}  // extern "C"
