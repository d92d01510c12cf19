// C ABI of the hot path: argument validation, the flat parameter layout, the
// workspace layout, and the launch plans of the forward and gradient functions.
//
// The gradient function follows DLVM's adjoint code generation (section
// 3.1.3): it takes the original inputs, recomputes the forward keeping every
// layer output, then walks the layers backwards emitting the adjoint of each
// dot (two products, transposes never materialised) fused with the adjoint of
// the element-wise operators around it. The input gradient of the first layer
// is dead unless x is differentiated, and is not computed (aggressive dead
// code elimination, section 3.1.4).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "dlvm.h"
#include "common.hpp"
#include "kernels.hpp"

using dlvm::GemmDesc;
using dlvm::Layout;
using dlvm::PacketEvents;
using dlvm::packet_events;

dlvm::PacketEvents& dlvm::packet_events() {
  thread_local PacketEvents e;
  return e;
}

// Events of the timing probe (see dlvm_probe_arm).
struct ProbeState {
  bool armed = false;
  int32_t index = -1;
  int32_t capacity = 0;
  int32_t used = 0;
  std::vector<hipEvent_t> start, stop;
  std::vector<int32_t> pos;
};

struct dlvm_model {
  int L = 0;
  std::vector<int32_t> widths;
  std::vector<int32_t> acts;
  int32_t dtype = DLVM_F32;
  int32_t loss = DLVM_LOSS_SOFTMAX_CE;
  int32_t wrt_x = 0;
  int64_t batch_max = 0;
  int32_t ckpt = 1;              // keep every ckpt-th hidden activation (1: all)
  int32_t chain_epi = 0;         // CHAIN8: run the chain in the product's epilogue
  // Recurrent networks (kind 1): T steps of the cell
  // hs[t+1] = act(xs[t] . W + hs[t] . U + b); L = 1 and widths = {Kx + H, H},
  // the one "layer" being the stacked [W; U] and b.
  int32_t kind = 0;              // 0: dense network, 1: recurrent network, 2: matrix chain
  int64_t rnn_T = 0, rnn_Kx = 0, rnn_H = 0;
  std::vector<int64_t> chain_dims;   // matrix chains (kind 2): shapes and order
  std::vector<int32_t> chain_cuts;
  int32_t wrt_h0 = 0;
  mutable int32_t n_fwd_launches = 0;  // launches of a recurrent forward call
  std::vector<int64_t> offsets;  // element offsets: W_l, b_l interleaved
  std::vector<int64_t> ldw;      // row stride of W_l (N_l, or N_L rounded up to 8)
  int64_t param_count = 0;
  dlvm::ZeroGaps gaps{};         // padding ranges of the flat buffer
  // Launches of the most recent gradient call (the SGD launch that follows it
  // is the next position of the step for the timing probe).
  mutable int32_t n_grad_launches = 0;
  mutable ProbeState probe;
};

struct dlvm_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

namespace {

thread_local std::string g_last_error;

dlvm_status fail(dlvm_status code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

dlvm_status hip_fail(hipError_t e, const char* where) {
  return fail(DLVM_ERR_HIP, std::string(where) + ": " + hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
size_t elem_size(int dtype) { return dtype == DLVM_BF16 ? 2 : 4; }
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool valid_dtype(int32_t d) { return d == DLVM_F32 || d == DLVM_BF16; }
bool valid_act(int32_t a) { return a >= DLVM_ACT_NONE && a <= DLVM_ACT_RELU; }

// Workspace layout for a given batch. Offsets in bytes from the base.
struct WsLayout {
  size_t flags = 0;         // int32[4]: [0] label out of range, [1] non-finite loss
  size_t partials = 0;      // float32 loss partials
  size_t bad = 0;           // int32 bad-label counts, one per loss partial
  std::vector<size_t> H;    // H[l], l = 1 .. L-1: where layer output H_l lives (storage dtype):
                            // its own buffer if l is a multiple of ckpt (a checkpoint), else
                            // segment slot l % ckpt - 1, shared by the segments in turn
  size_t logits = 0;        // float32 [B, widths[L]] (logits, or z for the chain)
  std::vector<size_t> dz;   // dz[l], l = 0 .. L-1: adjoint of layer l's pre-activation output,
                            // [B, ldw[l]] (storage dtype; float32 for the chain)
  size_t splitk = 0;        // float32 partials of a split adjoint product wrt the weights
  int64_t splitk_elems = 0;
  std::vector<size_t> mask; // mask[l], l = 1 .. L-1: rectifier mask of H_l (0: none; see
                            // relu_mask_planned), after every other region
  size_t total = 0;
};

GemmDesc gemm_tn(int dtype, int64_t M, int64_t N, int64_t K, const void* X, const void* dY,
                 int64_t ldy, float* dW, int64_t ldw, float* db, int64_t nvec);
GemmDesc gemm_nn(int dtype, int out_dtype, int act, int64_t M, int64_t N, int64_t K, float alpha,
                 const void* X, const void* W, int64_t ldw, const void* bias, void* H,
                 int64_t ldh);

// k-slices of the output layer's product in a gradient call (1: none). A
// softmax head with few classes has few output tiles per batch; its
// contraction is split so that more workgroups share it, and the slices are
// summed (with the bias) by the softmax cross-entropy kernel that follows.
int head_splits(const dlvm_model* m, int64_t B) {
  if (m->loss != DLVM_LOSS_SOFTMAX_CE) return 1;
  const int64_t C = m->widths[m->L], K = m->widths[m->L - 1];
  if (C > 256 || K < 128) return 1;
  const int64_t tiles = (B + 31) / 32 * ((C + 31) / 32);
  int s = 1;
  while (s < 8 && K / (2 * s) >= 64 && tiles * 2 * s <= 256) s *= 2;
  return s;
}

bool relu_mask_planned(const dlvm_model* m, const void* params, const void* x, int64_t batch,
                       void* ws, const WsLayout& w, int l);

WsLayout ws_layout(const dlvm_model* m, int64_t B) {
  WsLayout w;
  size_t off = 0;
  w.flags = off;
  off = align_up(off + 16);
  int64_t np = std::max<int64_t>(dlvm::softmax_xent_partials(B),
                                 dlvm::chain8_partials(B, m->widths[m->L]));
  // the chain epilogue writes one partial per wavefront; every register-staged
  // configuration gives each wavefront at least a 32 x 32 block
  if (m->chain_epi) np = std::max<int64_t>(np, (B + 31) / 32 * ((m->widths[m->L] + 31) / 32));
  w.partials = off;
  off = align_up(off + static_cast<size_t>(np) * 4);
  w.bad = off;
  off = align_up(off + static_cast<size_t>(np) * 4);
  const size_t es = elem_size(m->dtype);
  w.H.assign(m->L + 1, 0);
  const int k = m->ckpt;
  int64_t maxw = 0;
  for (int l = 1; l < m->L; ++l) {
    if (l % k == 0) {
      w.H[l] = off;
      off = align_up(off + static_cast<size_t>(B) * m->widths[l] * es);
    } else {
      maxw = std::max<int64_t>(maxw, m->widths[l]);
    }
  }
  if (maxw > 0) {
    for (int j = 0; j < k - 1; ++j) {
      const size_t slot = off;
      off = align_up(off + static_cast<size_t>(B) * maxw * es);
      for (int l = 1; l < m->L; ++l)
        if (l % k == j + 1) w.H[l] = slot;
    }
  }
  w.logits = off;
  off = align_up(off + static_cast<size_t>(B) * m->widths[m->L] * 4);
  const size_t dz_es = m->loss == DLVM_LOSS_CHAIN8 ? 4 : es;
  w.dz.assign(m->L, 0);
  for (int l = 0; l < m->L; ++l) {
    w.dz[l] = off;
    off = align_up(off + static_cast<size_t>(B) * m->ldw[l] * dz_es);
  }
  // Scratch for the partials of the largest split among the adjoint products
  // wrt the weights (the planner splits their batch reduction when their
  // output has too few tiles to occupy the device).
  for (int l = 0; l < m->L; ++l) {
    const int64_t K = m->widths[l], N = m->widths[l + 1], Np = m->ldw[l];
    const GemmDesc d = gemm_tn(m->dtype, B, Np, K, nullptr, nullptr, Np, nullptr, Np, nullptr, N);
    w.splitk_elems = std::max<int64_t>(w.splitk_elems, dlvm::split_ws_elems(d));
  }
  for (int l = 0; l + 1 < m->L; ++l) {  // the hidden layers' forward products (shapes only)
    GemmDesc d = gemm_nn(m->dtype, m->dtype, m->acts[l], B, m->widths[l + 1], m->widths[l], 1.0f,
                         nullptr, nullptr, m->ldw[l], nullptr, nullptr, m->widths[l + 1]);
    d.split_epilogue = true;
    w.splitk_elems = std::max<int64_t>(w.splitk_elems, dlvm::split_ws_elems(d));
  }
  const int hs = head_splits(m, B);
  if (hs > 1) {
    const int64_t C = m->widths[m->L];
    w.splitk_elems = std::max<int64_t>(w.splitk_elems, int64_t(hs) * (B * C + C));
  }
  w.splitk = off;
  off = align_up(off + static_cast<size_t>(w.splitk_elems) * 4);
  // Rectifier masks, where the products' shapes allow them (the pointers of
  // a call decide again, with the same rule, whether they are used).
  w.mask.assign(m->L, 0);
  for (int l = 1; l < m->L; ++l) {
    if (!relu_mask_planned(m, nullptr, nullptr, B, nullptr, w, l)) continue;
    w.mask[l] = off;
    off = align_up(off + static_cast<size_t>(dlvm::mask_bytes(B, m->widths[l])));
  }
  w.total = off;
  return w;
}

// Address arithmetic on integers: a dry run (plan description) uses null bases.
template <typename T> T* at(const void* base, size_t off) {
  return reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(base) + off);
}

const void* param_ptr(const dlvm_model* m, const void* params, int64_t elem_off) {
  return at<const void>(params, static_cast<size_t>(elem_off) * elem_size(m->dtype));
}

dlvm_status check_batch(const dlvm_model* m, int64_t batch) {
  if (batch < 1 || batch > m->batch_max)
    return fail(DLVM_ERR_INVALID_ARG, "batch must be in [1, batch_max]");
  return DLVM_OK;
}

size_t ws_total(const dlvm_model* m, int64_t batch);

dlvm_status check_ws(const dlvm_model* m, int64_t batch, const void* ws, size_t ws_bytes) {
  if (ws == nullptr) return fail(DLVM_ERR_WORKSPACE, "workspace is null");
  if (!aligned16(ws)) return fail(DLVM_ERR_MISALIGNED, "workspace is not 16-byte aligned");
  if (ws_bytes < ws_total(m, batch))
    return fail(DLVM_ERR_WORKSPACE, "workspace is smaller than dlvm_workspace_bytes");
  return DLVM_OK;
}

dlvm_status run_gemm(const GemmDesc& d, hipStream_t s) {
  const hipError_t e = dlvm::launch_gemm(d, dlvm::plan_gemm(d), s);
  if (e != hipSuccess) return hip_fail(e, "gemm launch");
  return DLVM_OK;
}

// H[M,N] (row stride ldh) = act(alpha * X[M,K] . W[K,N] (row stride ldw) + bias[N])
GemmDesc gemm_nn(int dtype, int out_dtype, int act, int64_t M, int64_t N, int64_t K, float alpha,
                 const void* X, const void* W, int64_t ldw, const void* bias, void* H,
                 int64_t ldh) {
  GemmDesc d{};
  d.layout = Layout::NN; d.dtype = dtype; d.out_dtype = out_dtype; d.act = act;
  d.M = M; d.N = N; d.K = K;
  d.A = X; d.lda = K; d.B = W; d.ldb = ldw; d.C = H; d.ldc = ldh;
  d.bias = bias; d.alpha = alpha; d.nvec = N;
  return d;
}

// dX[M,K] = (dY[M,N] (stride ldy) . W[K,N]^T (stride ldw)) * act'(Hprev) + R
GemmDesc gemm_nt(int dtype, int out_dtype, int act_prev, int64_t M, int64_t N, int64_t K,
                 const void* dY, int64_t ldy, const void* W, int64_t ldw, const void* Hprev,
                 const void* R, void* dX) {
  GemmDesc d{};
  d.layout = Layout::NT; d.dtype = dtype; d.out_dtype = out_dtype; d.act = act_prev;
  d.M = M; d.N = K; d.K = N;
  d.A = dY; d.lda = ldy; d.B = W; d.ldb = ldw; d.C = dX; d.ldc = K;
  d.aux = Hprev; d.residual = R; d.alpha = 1.0f; d.nvec = K;
  return d;
}

// dW[K,N] (stride ldw) = X[M,K]^T . dY[M,N] (stride ldy); db = column sums of
// the first nvec columns of dY
GemmDesc gemm_tn(int dtype, int64_t M, int64_t N, int64_t K, const void* X, const void* dY,
                 int64_t ldy, float* dW, int64_t ldw, float* db, int64_t nvec) {
  GemmDesc d{};
  d.layout = Layout::TN; d.dtype = dtype; d.out_dtype = DLVM_F32; d.act = DLVM_ACT_NONE;
  d.M = K; d.N = N; d.K = M;
  d.A = X; d.lda = K; d.B = dY; d.ldb = ldy; d.C = dW; d.ldc = ldw;
  d.colsum = db; d.alpha = 1.0f; d.nvec = nvec;
  return d;
}

// Description of one launch (name, sizes, algorithmic work).
struct LaunchInfo {
  std::string name;
  int64_t M = 0, N = 0, K = 0;
  double flops = 0.0, bytes = 0.0;
};

LaunchInfo gemm_info(const GemmDesc& d) {
  static const char* lay[] = {"nn", "nt", "tn"};
  LaunchInfo i;
  i.name = std::string("gemm_") + lay[static_cast<int>(d.layout)] + (d.dtype == DLVM_F32 ? "_f32" : "_bf16");
  // Work of the unpadded problem: padding columns and padded contraction
  // entries are zeros that the algorithm does not need.
  const double M = double(d.M);
  const double N = double(d.nvec > 0 && d.nvec < d.N ? d.nvec : d.N);
  const double K = double(d.kvalid > 0 ? d.kvalid : d.K);
  i.M = d.M; i.N = static_cast<int64_t>(N); i.K = static_cast<int64_t>(K);
  i.flops = 2.0 * M * N * K;
  const double es = double(elem_size(d.dtype)), eo = double(elem_size(d.out_dtype));
  double b = (M * K + K * N) * es + M * N * eo;
  if (d.bias) b += N * es;
  if (d.layout == Layout::NT && d.act != DLVM_ACT_NONE) b += d.mask ? M * N / 8.0 : M * N * es;
  if (d.layout == Layout::NN && d.mask) b += M * N / 8.0;  // the rectifier mask written
  if (d.residual) b += M * N * eo;
  if (d.colsum) b += N * 4.0;
  i.bytes = b;
  return i;
}

LaunchInfo elementwise_info(const char* name, int64_t rows, int64_t cols, double bytes) {
  LaunchInfo i;
  i.name = name;
  i.M = rows; i.N = cols; i.K = 0;
  i.bytes = bytes;
  return i;
}

// Every launch of the model-level calls goes through one Launcher. With a
// plan vector it only records what it would launch (no pointer is touched);
// otherwise it enqueues the launch on the caller's stream, bracketed by the
// probe's events when the probe is armed for this position.
class Launcher {
 public:
  Launcher(const dlvm_model* m, hipStream_t s, std::vector<LaunchInfo>* plan, int32_t first)
      : m_(m), main_(s), plan_(plan), index_(first) {
    dlvm::tuning_scope_begin();
  }
  ~Launcher() { dlvm::tuning_scope_end(); }
  Launcher(const Launcher&) = delete;
  Launcher& operator=(const Launcher&) = delete;

  template <class F>
  dlvm_status run(LaunchInfo info, F&& launch, const char* what) {
    const int32_t idx = index_++;
    if (plan_ != nullptr) {
      plan_->push_back(std::move(info));
      return DLVM_OK;
    }
    if (m_ == nullptr) {  // a call without a model handle: nothing to record
      const hipError_t e = launch(main_);
      return e != hipSuccess ? hip_fail(e, what) : DLVM_OK;
    }
    ProbeState& p = m_->probe;
    const bool rec = p.armed && (p.index < 0 || p.index == idx) && p.used < p.capacity;
    if (rec) packet_events() = PacketEvents{p.start[p.used], p.stop[p.used]};
    const hipError_t e = launch(main_);
    if (rec) {
      packet_events() = PacketEvents{};
      p.pos[p.used] = idx;
      ++p.used;
    }
    if (e != hipSuccess) return hip_fail(e, what);
    return DLVM_OK;
  }

  dlvm_status gemm(const GemmDesc& d) {
    const dlvm::GemmPlan pl = dlvm::plan_gemm(d);
    LaunchInfo info = gemm_info(d);
    info.name += "_" + std::to_string(pl.bm) + "x" + std::to_string(pl.bn) + "c" + std::to_string(pl.cfg);
    if (pl.splits > 1) info.name += "s" + std::to_string(pl.splits);
    dlvm_status st = run(std::move(info), [&](hipStream_t s) { return dlvm::launch_gemm(d, pl, s); },
                         "gemm launch");
    if (st != DLVM_OK) return st;
    return reduce_split(d, pl);
  }

  // The k-slices' partial products (and column sums) of a split product,
  // summed in slice order (nothing if the product is not split).
  dlvm_status reduce_split(const GemmDesc& d, const dlvm::GemmPlan& pl) {
    if (pl.splits <= 1) return DLVM_OK;
    const int64_t nv = d.nvec > 0 ? d.nvec : d.N;
    const int64_t c_split = d.M * d.ldc;
    if (d.layout != Layout::TN) {
      // a forward (NN) or input-adjoint (NT) product: its epilogue follows the sum
      const double mn = double(d.M) * double(d.N);
      const double eo = elem_size(d.out_dtype), ei = elem_size(d.dtype);
      const double bytes = double(pl.splits) * mn * 4.0 + mn * eo +
                           (d.aux && d.act != DLVM_ACT_NONE ? mn * ei : 0.0) +
                           (d.residual ? mn * eo : 0.0) + (d.bias ? double(nv) * ei : 0.0);
      return run(elementwise_info("split_epilogue", d.M, d.N, bytes),
                 [&](hipStream_t s) {
                   return dlvm::launch_split_epilogue(
                       d.dtype, d.out_dtype, d.layout == Layout::NN ? 0 : 1, pl.splits, d.M, d.N,
                       d.ldc, d.split_ws, c_split, d.act, d.alpha, d.bias, nv, d.aux, d.residual,
                       d.res_pre, d.C, s);
                 },
                 "split epilogue launch");
    }
    const float* cs = d.split_ws + pl.splits * c_split;
    const double bytes = (double(pl.splits) + 1.0) * double(d.M) * double(d.N) * 4.0 +
                         (d.colsum ? (double(pl.splits) + 1.0) * double(nv) * 4.0 : 0.0);
    return run(elementwise_info("splitk_reduce", d.M, d.N, bytes),
               [&](hipStream_t s) {
                 return dlvm::launch_splitk_reduce(pl.splits, d.M, d.N, d.ldc, d.split_ws, c_split,
                                                   static_cast<float*>(d.C), cs, nv, d.colsum, nv, s);
               },
               "split reduction launch");
  }

  // One product without the reduction of its k-slices (the caller sums them).
  dlvm_status gemm_raw(const GemmDesc& d, dlvm::GemmPlan& pl) {
    pl = dlvm::plan_gemm(d);
    LaunchInfo info = gemm_info(d);
    info.name += "_" + std::to_string(pl.bm) + "x" + std::to_string(pl.bn) + "c" + std::to_string(pl.cfg);
    if (pl.splits > 1) info.name += "s" + std::to_string(pl.splits);
    return run(std::move(info), [&](hipStream_t s) { return dlvm::launch_gemm(d, pl, s); },
               "gemm launch");
  }

  // A layer's two adjoint products (tn: wrt the weights, nt: wrt the input):
  // one launch when both are planned on a configuration that has a paired
  // kernel, else two; then the split reduction of the product wrt the weights.
  dlvm_status gemm_pair(const GemmDesc& tn, const GemmDesc& nt) {
    const dlvm::GemmPlan p1 = dlvm::plan_gemm(tn), p2 = dlvm::plan_gemm(nt);
    if (!dlvm::pairable(tn, p1, nt, p2)) {
      dlvm_status st = gemm(tn);
      return st != DLVM_OK ? st : gemm(nt);
    }
    LaunchInfo a = gemm_info(tn), b = gemm_info(nt);
    LaunchInfo info;
    info.name = std::string("gemm_pair_") + (tn.dtype == DLVM_F32 ? "f32_" : "bf16_") +
                std::to_string(p1.bm) + "x" + std::to_string(p1.bn) + "c" + std::to_string(p1.cfg) +
                (p1.splits > 1 ? "s" + std::to_string(p1.splits) : std::string());
    info.M = a.M; info.N = a.N; info.K = a.K;  // the product wrt the weights
    info.flops = a.flops + b.flops;
    info.bytes = a.bytes + b.bytes;
    dlvm_status st = run(std::move(info),
                         [&](hipStream_t s) { return dlvm::launch_gemm_pair(tn, p1, nt, p2, s); },
                         "paired gemm launch");
    if (st != DLVM_OK) return st;
    return reduce_split(tn, p1);
  }

  hipStream_t stream() const { return main_; }
  bool dry() const { return plan_ != nullptr; }
  int32_t launches() const { return index_; }

 private:
  const dlvm_model* m_;
  hipStream_t main_;
  std::vector<LaunchInfo>* plan_;
  int32_t index_;
};

// The adjoint of the dense layers, last first, from the adjoint of the output
// layer's output in dz[L-1]: for each layer the products wrt its parameters
// and wrt its input (the latter dead for the first layer unless x is
// differentiated, section 3.1.4).
// Forward product of layer l (0-based): H_{l+1} = act_l(H_l . W_l + b_l), from
// where H_l lives (x for l = 0) to where H_{l+1} lives.
// The forward product of hidden layer l; the planner may split it over k
// (the bias and activation then follow the in-order sum of the slices).
GemmDesc hidden_desc(const dlvm_model* m, const void* params, const void* in, int64_t batch,
                     void* out, float* split_ws, int64_t split_elems, int l) {
  const int dt = m->dtype;
  GemmDesc d = gemm_nn(dt, dt, m->acts[l], batch, m->widths[l + 1], m->widths[l], 1.0f, in,
                       param_ptr(m, params, m->offsets[2 * l]), m->ldw[l],
                       param_ptr(m, params, m->offsets[2 * l + 1]), out, m->widths[l + 1]);
  d.split_epilogue = true;
  d.split_ws = split_ws;
  d.split_ws_elems = split_elems;
  return d;
}

// The product wrt the input of layer l >= 1 (dX = dZ_l . W_l^T times the
// derivative of layer l - 1's activation, from H_l), into dz[l - 1].
GemmDesc input_adjoint_desc(const dlvm_model* m, const void* params, int64_t batch, void* ws,
                            const WsLayout& w, int l) {
  const int64_t K = m->widths[l], N = m->widths[l + 1], Np = m->ldw[l];
  GemmDesc d = gemm_nt(m->dtype, m->dtype, m->acts[l - 1], batch, Np, K, at<void>(ws, w.dz[l]), Np,
                       param_ptr(m, params, m->offsets[2 * l]), Np, at<void>(ws, w.H[l]), nullptr,
                       at<void>(ws, w.dz[l - 1]));
  d.kvalid = N;
  return d;
}

// Rectifier masks (section 3.1.3: the adjoint of the rectifier needs only the
// sign of its saved output). Layer output H_l (1 <= l < L) of a bf16 network
// whose layer l - 1 is rectified: when the forward product that writes H_l and
// the product wrt the input of layer l, whose epilogue applies the
// derivative, both pass dlvm::mask_ok as they will be launched, the forward
// also writes the derivative's bits in accumulator order and the adjoint reads
// them instead of H_l (one bit per element instead of two bytes). Both sides
// ask this function with the same arguments, so they agree.
// DLVM_RELU_MASK=0 turns the masks off (tests compare the two paths).
bool relu_mask_planned(const dlvm_model* m, const void* params, const void* x, int64_t batch,
                       void* ws, const WsLayout& w, int l) {
  const char* env = std::getenv("DLVM_RELU_MASK");
  if (env != nullptr && std::strcmp(env, "0") == 0) return false;
  if (m->kind != 0 || m->loss == DLVM_LOSS_CHAIN8 || m->dtype != DLVM_BF16) return false;
  if (l < 1 || l >= m->L || m->acts[l - 1] != DLVM_ACT_RELU) return false;
  const void* in = l == 1 ? x : at<void>(ws, w.H[l - 1]);
  const GemmDesc f = hidden_desc(m, params, in, batch, at<void>(ws, w.H[l]),
                                 at<float>(ws, w.splitk), w.splitk_elems, l - 1);
  const GemmDesc a = input_adjoint_desc(m, params, batch, ws, w, l);
  const dlvm::GemmPlan pf = dlvm::plan_gemm(f), pa = dlvm::plan_gemm(a);
  // (the mask is in the accumulator order of one tile configuration)
  return pf.cfg == pa.cfg && dlvm::mask_ok(f, pf) && dlvm::mask_ok(a, pa);
}

// The rectifier mask of H_l a call uses, or null.
uint32_t* relu_mask(const dlvm_model* m, const void* params, const void* x, int64_t batch,
                    void* ws, const WsLayout& w, int l) {
  if (l < 1 || l >= static_cast<int>(w.mask.size()) || w.mask[l] == 0) return nullptr;
  if (!relu_mask_planned(m, params, x, batch, ws, w, l)) return nullptr;
  return at<uint32_t>(ws, w.mask[l]);
}

dlvm_status plan_hidden_layer(const dlvm_model* m, const void* params, const void* x,
                              int64_t batch, void* ws, const WsLayout& w, int l, Launcher& run) {
  const void* in = l == 0 ? x : at<void>(ws, w.H[l]);
  GemmDesc d = hidden_desc(m, params, in, batch, at<void>(ws, w.H[l + 1]),
                           at<float>(ws, w.splitk), w.splitk_elems, l);
  d.mask = relu_mask(m, params, x, batch, ws, w, l + 1);
  return run.gemm(d);
}

// The hidden layers' forward (H_1 .. H_{L-1}, each written where it lives).
dlvm_status plan_hidden_forward(const dlvm_model* m, const void* params, const void* x,
                                int64_t batch, void* ws, const WsLayout& w, Launcher& run) {
  for (int l = 0; l < m->L - 1; ++l) {
    const dlvm_status st = plan_hidden_layer(m, params, x, batch, ws, w, l, run);
    if (st != DLVM_OK) return st;
  }
  return DLVM_OK;
}

// First layer of the segment whose outputs the segment slots hold after the
// hidden layers' forward (-1: no slots).
int resident_segment(const dlvm_model* m) {
  for (int l = m->L - 1; l >= 1; --l)
    if (l % m->ckpt != 0) return l - l % m->ckpt;
  return -1;
}

dlvm_status plan_adjoint_layers(const dlvm_model* m, const void* params, const void* x,
                                int64_t batch, float* dparams, float* dx, void* ws,
                                const WsLayout& w, Launcher& run) {
  const int L = m->L;
  const int dt = m->dtype;
  auto P = [&](int idx) { return param_ptr(m, params, m->offsets[idx]); };
  auto G = [&](int idx) { return at<float>(dparams, static_cast<size_t>(m->offsets[idx]) * 4); };
  dlvm_status st = DLVM_OK;
  // Checkpointing (section 3.1.3): layer l's adjoint needs H_l. A layer output
  // that is not a checkpoint is recomputed, with the rest of its segment, from
  // the segment's checkpoint the first time the sweep needs it.
  int resident = resident_segment(m);
  // Last layer first. On the padded class columns dZ_L and W_L
  // are zero, so the products run over the padded width and the padding
  // columns of dW_L come out zero.
  for (int l = L - 1; l >= 0; --l) {
    if (l > 0 && l % m->ckpt != 0 && l - l % m->ckpt != resident) {
      const int c = l - l % m->ckpt;
      for (int j = c; j < l; ++j)  // H_{c+1} .. H_l from H_c
        if ((st = plan_hidden_layer(m, params, x, batch, ws, w, j, run)) != DLVM_OK) return st;
      resident = c;
    }
    const void* hin = l == 0 ? x : at<void>(ws, w.H[l]);
    const int64_t K = m->widths[l], N = m->widths[l + 1];
    const int64_t Np = m->ldw[l];  // padded width (== N except the last layer)
    void* dzl = at<void>(ws, w.dz[l]);
    GemmDesc dw = gemm_tn(dt, batch, Np, K, hin, dzl, Np, G(2 * l), Np, G(2 * l + 1), N);
    dw.split_ws = at<float>(ws, w.splitk);
    dw.split_ws_elems = w.splitk_elems;
    // The product wrt the input (dead for the first layer unless x is
    // differentiated) reads the same adjoint: the two share one launch.
    if (l > 0) {
      GemmDesc d = input_adjoint_desc(m, params, batch, ws, w, l);
      d.mask = relu_mask(m, params, x, batch, ws, w, l);
      if ((st = run.gemm_pair(dw, d)) != DLVM_OK) return st;
    } else if (m->wrt_x) {
      GemmDesc d = gemm_nt(dt, DLVM_F32, DLVM_ACT_NONE, batch, Np, K, dzl, Np, P(0), Np, nullptr,
                           nullptr, dx);
      d.kvalid = N;
      if ((st = run.gemm_pair(dw, d)) != DLVM_OK) return st;
    } else if ((st = run.gemm(dw)) != DLVM_OK) {
      return st;
    }
  }
  return DLVM_OK;
}

// The launches of one gradient call (section 3.1.3): forward keeping every
// layer output, the loss adjoint, then the adjoint of each layer, last first.
// The one-workgroup gradient of small networks is used unless DLVM_SMALL_STEP=0
// (for tests that compare it with the general plan).
bool small_step_allowed() {
  const char* v = std::getenv("DLVM_SMALL_STEP");
  return v == nullptr || std::strcmp(v, "0") != 0;
}

dlvm_status plan_gradient(const dlvm_model* m, const void* params, const void* x,
                          const int32_t* labels, int64_t batch, float* loss, float* dparams,
                          float* dx, void* ws, Launcher& run) {
  const WsLayout w = ws_layout(m, batch);
  const int L = m->L;
  const int dt = m->dtype;
  const double es = double(elem_size(dt));
  float* partials = at<float>(ws, w.partials);
  int32_t* bad = at<int32_t>(ws, w.bad);
  int32_t* flags = at<int32_t>(ws, w.flags);
  auto P = [&](int idx) { return param_ptr(m, params, m->offsets[idx]); };
  auto G = [&](int idx) { return at<float>(dparams, static_cast<size_t>(m->offsets[idx]) * 4); };
  dlvm_status st = DLVM_OK;
  int np = 0;
  float scale = 1.0f;
  const bool chain = m->loss == DLVM_LOSS_CHAIN8;
  const int32_t* badp = chain ? nullptr : bad;
  auto finalize = [&]() {
    return run.run(elementwise_info("finalize", np, 1, 8.0 * np + 4.0),
                   [&](hipStream_t s) {
                     return dlvm::launch_finalize(partials, badp, np, scale, loss, flags, dparams,
                                                  m->gaps, s);
                   },
                   "loss finalisation launch");
  };

  if (chain) {
    const int64_t N = m->widths[1], K = m->widths[0];
    float* z = at<float>(ws, w.logits);
    float* zbar = at<float>(ws, w.dz[0]);
    scale = static_cast<float>(1.0 / (static_cast<double>(batch) * static_cast<double>(N)));
    if (m->chain_epi) {
      // The chain in the product's epilogue (z is never stored): zbar to the
      // workspace, xbar into dx, one loss partial per wavefront.
      GemmDesc d = gemm_nn(dt, DLVM_F32, DLVM_ACT_NONE, batch, N, K, 1.0f, x, P(0), N, P(1), zbar, N);
      d.aux = x;
      d.chain_epilogue = true;
      d.C2 = dx;
      d.partials = partials;
      d.inv_n = scale;
      const dlvm::GemmPlan pl = dlvm::plan_gemm(d);
      np = static_cast<int>(dlvm::chain_partials(pl));
      LaunchInfo info = gemm_info(d);
      info.name = "gemm_nn_chain8_f32_" + std::to_string(pl.bm) + "x" + std::to_string(pl.bn) + "c" +
                  std::to_string(pl.cfg);
      info.bytes += 12.0 * double(batch) * double(N);  // x_skip read, zbar and xbar written
      st = run.run(std::move(info), [&](hipStream_t s) { return dlvm::launch_gemm(d, pl, s); },
                   "chain product launch");
    } else {
      if ((st = run.gemm(gemm_nn(dt, DLVM_F32, DLVM_ACT_NONE, batch, N, K, 1.0f, x, P(0), N,
                                 nullptr, z, N))) != DLVM_OK)
        return st;
      np = dlvm::chain8_partials(batch, N);
      st = run.run(elementwise_info("chain8", batch, N, 16.0 * double(batch) * N + 4.0 * N),
                   [&](hipStream_t s) {
                     int n = 0;
                     return dlvm::launch_chain8(batch, N, z, static_cast<const float*>(P(1)),
                                                static_cast<const float*>(x), zbar, dx, partials,
                                                false, &n, s);
                   },
                   "chain launch");
    }
    if (st != DLVM_OK) return st;
    GemmDesc dw = gemm_tn(dt, batch, N, K, x, zbar, N, G(0), N, G(1), N);
    dw.split_ws = at<float>(ws, w.splitk);
    dw.split_ws_elems = w.splitk_elems;
    // dx = zbar . W^T + xbar (xbar already in dx: in-place accumulate)
    const GemmDesc dxd = gemm_nt(dt, DLVM_F32, DLVM_ACT_NONE, batch, N, K, zbar, N, P(0), N,
                                 nullptr, dx, dx);
    if ((st = run.gemm_pair(dw, dxd)) != DLVM_OK) return st;
    return finalize();
  }

  // A small float32 network: the whole gradient in one workgroup (one launch).
  dlvm::SmallNet sn{};
  if (small_step_allowed() && m->dtype == DLVM_F32 &&
      dlvm::small_net(L, m->widths.data(), m->acts.data(), m->offsets.data(), m->ldw.data(),
                      batch, m->wrt_x != 0, sn)) {
    double flops = 0.0, bytes = 0.0;
    for (int l = 0; l < L; ++l) {
      const double k = m->widths[l], n = m->widths[l + 1];
      flops += 2.0 * batch * k * n * ((l > 0 || m->wrt_x) ? 3.0 : 2.0);
      bytes += 8.0 * (k * n + n);  // parameters read, their gradient written
    }
    bytes += 4.0 * batch * (m->widths[0] + (m->wrt_x ? m->widths[0] : 0) + 1);
    LaunchInfo info;
    info.name = "small_step_f32";
    info.M = batch; info.N = m->widths[L]; info.K = m->widths[0];
    info.flops = flops;
    info.bytes = bytes;
    return run.run(std::move(info),
                   [&](hipStream_t s) {
                     return dlvm::launch_small_step(sn, static_cast<const float*>(params),
                                                    static_cast<const float*>(x), labels, loss,
                                                    dparams, dx, flags, m->gaps, s);
                   },
                   "small-network gradient launch");
  }

  // Forward, keeping the layer outputs (every one, or the checkpoints and the
  // last segment).
  if ((st = plan_hidden_forward(m, params, x, batch, ws, w, run)) != DLVM_OK) return st;
  const void* h = L > 1 ? at<void>(ws, w.H[L - 1]) : x;
  const int64_t C = m->widths[L];
  const int64_t ldc = m->ldw[L - 1];  // dZ_L rows are padded like W_L's
  scale = static_cast<float>(1.0 / static_cast<double>(batch));
  np = dlvm::softmax_xent_partials(batch);
  // Output layer: logits, then softmax cross-entropy and its adjoint. A split
  // product leaves its k-slices in the scratch; the loss kernel sums them.
  GemmDesc head = gemm_nn(dt, DLVM_F32, DLVM_ACT_NONE, batch, C, m->widths[L - 1], 1.0f, h,
                          P(2 * (L - 1)), m->ldw[L - 1], P(2 * L - 1), at<void>(ws, w.logits), C);
  head.split_ws = at<float>(ws, w.splitk);
  head.split_ws_elems = w.splitk_elems;
  head.splits_hint = head_splits(m, batch);
  dlvm::GemmPlan hp{};
  if ((st = run.gemm_raw(head, hp)) != DLVM_OK) return st;
  if (hp.splits > 1) {
    st = run.run(elementwise_info("split_softmax_xent", batch, C,
                                  double(batch) * C * (4.0 * hp.splits + es) + 4.0 * batch),
                 [&](hipStream_t s) {
                   return dlvm::launch_split_softmax_xent(
                       dt, hp.splits, batch, C, head.split_ws, batch * C, C, P(2 * L - 1), labels,
                       scale, at<void>(ws, w.dz[L - 1]), ldc, partials, bad, &np, s);
                 },
                 "softmax cross-entropy launch");
  } else {
    // (the kernel chosen decides how many loss partials it writes)
    st = run.run(elementwise_info("softmax_xent", batch, C, double(batch) * C * (4.0 + es) + 4.0 * batch),
                 [&](hipStream_t s) {
                   return dlvm::launch_softmax_xent(dt, batch, C, at<float>(ws, w.logits), labels,
                                                    scale, at<void>(ws, w.dz[L - 1]), ldc, partials,
                                                    bad, &np, s);
                 },
                 "softmax cross-entropy launch");
  }
  if (st != DLVM_OK) return st;
  // The loss and its flags right away, while the loss kernel's partials are
  // still in the caches (nothing in the adjoint sweep reads or writes them).
  if ((st = finalize()) != DLVM_OK) return st;
  return plan_adjoint_layers(m, params, x, batch, dparams, dx, ws, w, run);
}

// The launches of one seedable gradient call (Fig. 3's seedable
// declaration, wrt the parameters [and x]): the hidden layers' forward keeping
// their outputs, the seed stored as the output layer's adjoint, the adjoint
// sweep, the padding of dparams zeroed. The output layer's own product is
// dead (its value is not kept) and is not computed.
dlvm_status plan_vjp(const dlvm_model* m, const void* params, const void* x, const float* seed,
                     int64_t batch, float* dparams, float* dx, void* ws, Launcher& run) {
  const WsLayout w = ws_layout(m, batch);
  const int L = m->L;
  const int dt = m->dtype;
  dlvm_status st = DLVM_OK;
  if ((st = plan_hidden_forward(m, params, x, batch, ws, w, run)) != DLVM_OK) return st;
  const int64_t C = m->widths[L], ldc = m->ldw[L - 1];
  st = run.run(elementwise_info("seed", batch, C, double(batch) * (4.0 * C + elem_size(dt) * ldc)),
               [&](hipStream_t s) {
                 return dlvm::launch_seed(dt, batch, C, ldc, seed, at<void>(ws, w.dz[L - 1]), s);
               },
               "seed launch");
  if (st != DLVM_OK) return st;
  if ((st = plan_adjoint_layers(m, params, x, batch, dparams, dx, ws, w, run)) != DLVM_OK) return st;
  return run.run(elementwise_info("zero_padding", 0, 1, 4.0 * m->param_count),
                 [&](hipStream_t s) {
                   return dlvm::launch_finalize(nullptr, nullptr, 0, 1.0f, nullptr, nullptr, dparams,
                                                m->gaps, s);
                 },
                 "padding launch");
}

// The launches of one forward call: nothing is kept; layer l's output goes to
// the adjoint buffer of layer l (unused by a forward call).
dlvm_status plan_forward(const dlvm_model* m, const void* params, const void* x, int64_t batch,
                         float* out, void* ws, Launcher& run) {
  const WsLayout w = ws_layout(m, batch);
  dlvm_status st = DLVM_OK;
  const int L = m->L;
  const int dt = m->dtype;
  if (m->loss == DLVM_LOSS_CHAIN8) {
    const int64_t N = m->widths[1];
    float* z = at<float>(ws, w.logits);
    if ((st = run.gemm(gemm_nn(dt, DLVM_F32, DLVM_ACT_NONE, batch, N, m->widths[0], 1.0f, x,
                               param_ptr(m, params, m->offsets[0]), N, nullptr, z, N))) != DLVM_OK)
      return st;
    const float* bias = static_cast<const float*>(param_ptr(m, params, m->offsets[1]));
    return run.run(elementwise_info("chain8_forward", batch, N, 12.0 * double(batch) * N + 4.0 * N),
                   [&](hipStream_t s) {
                     int n = 0;
                     return dlvm::launch_chain8(batch, N, z, bias, static_cast<const float*>(x),
                                                out, nullptr, at<float>(ws, w.partials), true, &n, s);
                   },
                   "chain launch");
  }
  const void* h = x;
  for (int l = 0; l < L; ++l) {
    const bool last = l == L - 1;
    void* dst = last ? static_cast<void*>(out) : at<void>(ws, w.dz[l]);
    if ((st = run.gemm(gemm_nn(dt, last ? DLVM_F32 : dt, m->acts[l], batch, m->widths[l + 1],
                               m->widths[l], 1.0f, h, param_ptr(m, params, m->offsets[2 * l]),
                               m->ldw[l], param_ptr(m, params, m->offsets[2 * l + 1]), dst,
                               m->widths[l + 1]))) != DLVM_OK)
      return st;
    h = dst;
  }
  return DLVM_OK;
}

// ---------------------------------------------------------------------------
// Recurrent network: the cell h_t = f(W x_{t-1} + U h_{t-1} + b) of section
// 3.1.2, unrolled over T steps (row-major batch form:
// hs[t+1] = act(xs[t] . W + hs[t] . U + b)), with its linear-algebra fusion:
// the polynomial of two products and two additions is one product over the
// concatenated contraction [xs[t] hs[t]] . [W; U] + b. The parameters are
// stored concatenated in the first place (the interprocedural form of the
// fusion): [W; U] is one [Kx + H, H] matrix of the flat buffer. The operand
// [xs[t] hs[t]] is never materialised: the product reads its first Kx
// columns from xs[t] and the rest from hs[t] (a two-phase contraction).
// ---------------------------------------------------------------------------
struct RnnWs {
  size_t dz = 0;          // [T, B, H] storage dtype: adjoints of the pre-activations
  size_t splitk = 0;      // float32 partials of the split products wrt the weights
  int64_t splitk_elems = 0;
  size_t total = 0;
};

// The two products wrt the weights: d[W] = xs^T dz (+ db) and d[U] = hs^T dz
// over all T * B rows at once.
GemmDesc rnn_dw(const dlvm_model* m, int64_t B, const void* xs, const void* dz, float* dWU,
                float* db) {
  return gemm_tn(m->dtype, m->rnn_T * B, m->rnn_H, m->rnn_Kx, xs, dz, m->rnn_H, dWU, m->rnn_H,
                 db, m->rnn_H);
}
GemmDesc rnn_du(const dlvm_model* m, int64_t B, const void* hs, const void* dz, float* dU) {
  return gemm_tn(m->dtype, m->rnn_T * B, m->rnn_H, m->rnn_H, hs, dz, m->rnn_H, dU, m->rnn_H,
                 nullptr, m->rnn_H);
}

// k-slices for one of the recurrent step's products (a cell product or a
// recurrent adjoint). One step's product has few output tiles (B x H over
// the 64 x 128 tiles of the k-group kernel: 128 for a 1024 x 1024 output) and
// the steps run one after the other, so the contraction is split until there
// are as many tile-slices as compute units, at most 4 ways, each slice at
// least 256 deep and, for a two-phase product, within one phase. (Measured on
// 1024 x 1024 products, K = 2048 / 1024, batch 1024 and T = 32: two slices on
// that tile 673 steps/s against 607 for four on the 128 x 128 tile, one slice
// 597.)
int rnn_split_hint(int64_t M, int64_t N, int64_t K, int64_t K1) {
  const int64_t tiles = (M + 63) / 64 * ((N + 127) / 128);
  int s = 1;
  while (s < 4 && tiles * s < 256) {
    const int64_t kc = ((K + 2 * s - 1) / (2 * s) + 63) / 64 * 64;  // k per slice at 2s slices
    if (kc < 256 || (K + kc - 1) / kc < 2 * s || (K1 > 0 && K1 % kc != 0)) break;
    s *= 2;
  }
  return s;
}

// Cell t's fused product: hs[t+1] = act([xs[t] hs[t]] . [W; U] + b), its
// contraction in two phases (Kx columns of xs[t], then H of hs[t]).
GemmDesc rnn_cell(const dlvm_model* m, int64_t B, const void* x, const void* h, const void* WU,
                  const void* bias, void* out) {
  const int64_t Kx = m->rnn_Kx, H = m->rnn_H;
  GemmDesc d = gemm_nn(m->dtype, m->dtype, m->acts[0], B, H, Kx + H, 1.0f, x, WU, H, bias, out, H);
  d.lda = Kx;
  d.A2 = h;
  d.lda2 = H;
  d.K1 = Kx;
  d.split_epilogue = true;
  d.splits_hint = rnn_split_hint(B, H, Kx + H, Kx);
  return d;
}

// The recurrent adjoint dz[t-1] = (dz[t] . U^T + dhs[t-1]) * act'(hs[t]).
GemmDesc rnn_recur(const dlvm_model* m, int64_t B, const void* dz, const void* U, const void* h,
                   const void* seed, void* out) {
  const int64_t H = m->rnn_H;
  GemmDesc d = gemm_nt(m->dtype, m->dtype, m->acts[0], B, H, H, dz, H, U, H, h, seed, out);
  d.res_pre = true;
  d.split_epilogue = true;
  d.splits_hint = rnn_split_hint(B, H, H, 0);
  return d;
}

RnnWs rnn_ws_layout(const dlvm_model* m, int64_t B) {
  RnnWs w;
  size_t off = 0;
  w.dz = off;
  off = align_up(off + static_cast<size_t>(m->rnn_T * B * m->rnn_H) * elem_size(m->dtype));
  w.splitk = off;
  w.splitk_elems = std::max(
      std::max(dlvm::split_ws_elems(rnn_dw(m, B, nullptr, nullptr, nullptr, nullptr)),
               dlvm::split_ws_elems(rnn_du(m, B, nullptr, nullptr, nullptr))),
      std::max(dlvm::split_ws_elems(rnn_cell(m, B, nullptr, nullptr, nullptr, nullptr, nullptr)),
               dlvm::split_ws_elems(rnn_recur(m, B, nullptr, nullptr, nullptr, nullptr, nullptr))));
  off = align_up(off + static_cast<size_t>(w.splitk_elems) * 4);
  w.total = off;
  return w;
}

size_t chain_model_ws(const dlvm_model* m);
dlvm_status chain_model_run(const dlvm_model* m, const void* const* mats, float* out, void* ws,
                            Launcher& run);

size_t ws_total(const dlvm_model* m, int64_t batch) {
  if (m->kind == 2) return chain_model_ws(m);
  return m->kind == 1 ? rnn_ws_layout(m, batch).total : ws_layout(m, batch).total;
}

// Row block t of a [*, B, width] sequence tensor.
template <typename T>
T* seq_at(T* base, int64_t t, int64_t B, int64_t width, size_t es) {
  return at<T>(base, static_cast<size_t>(t * B * width) * es);
}

// The T fused cell products of a forward call.
// The T fused cell products of a forward call (each split over its
// contraction, with its epilogue after the sum, when the planner prefers;
// the k-slices go to `split` when given).
dlvm_status plan_rnn_forward(const dlvm_model* m, const void* params, const void* xs, int64_t B,
                             void* hs, float* split, int64_t split_elems, Launcher& run) {
  const size_t es = elem_size(m->dtype);
  const int64_t Kx = m->rnn_Kx, H = m->rnn_H;
  const void* WU = param_ptr(m, params, m->offsets[0]);
  const void* bias = param_ptr(m, params, m->offsets[1]);
  for (int64_t t = 0; t < m->rnn_T; ++t) {
    GemmDesc d = rnn_cell(m, B, seq_at(xs, t, B, Kx, es), seq_at(hs, t, B, H, es), WU, bias,
                          seq_at(hs, t + 1, B, H, es));
    d.split_ws = split;
    d.split_ws_elems = split != nullptr ? split_elems : 0;
    const dlvm_status st = run.gemm(d);
    if (st != DLVM_OK) return st;
  }
  return DLVM_OK;
}

// The launches of a backward call (backpropagation through time, the
// adjoint of the unrolled cell, section 3.1.3), with dz[t] the adjoint of
// cell t's pre-activation and dhs[t] the seed (direct adjoint) of hs[t+1]:
//   dz[T-1] = dhs[T-1] * act'(hs[T])
//   dz[t-1] = (dz[t] . U^T + dhs[t-1]) * act'(hs[t])      t = T-1 .. 1
//   dh0 = dz[0] . U^T                                      (iff wrt_h0)
//   [dW; dU] = [xs hs[0..T-1]]^T . dz, db = colsum(dz)    (all steps in one contraction)
//   dxs = dz . W^T                                         (iff wrt_x)
// The adjoint of the concatenation is the split of the product's output into
// its W and U rows; d[W] and dxs share dz and run as one launch when they can.
dlvm_status plan_rnn_backward(const dlvm_model* m, const void* params, const void* xs,
                              const void* hs, const void* dhs, int64_t B, float* dparams,
                              float* dxs, float* dh0, void* ws, Launcher& run) {
  const RnnWs w = rnn_ws_layout(m, B);
  const int dt = m->dtype;
  const size_t es = elem_size(dt);
  const int64_t T = m->rnn_T, Kx = m->rnn_Kx, H = m->rnn_H;
  const void* WU = param_ptr(m, params, m->offsets[0]);
  const void* U = at<const void>(WU, static_cast<size_t>(Kx * H) * es);
  float* dWU = at<float>(dparams, static_cast<size_t>(m->offsets[0]) * 4);
  float* db = at<float>(dparams, static_cast<size_t>(m->offsets[1]) * 4);
  void* dz = at<void>(ws, w.dz);
  dlvm_status st = run.run(
      elementwise_info("act_adjoint", B, H, 3.0 * double(B) * H * es), [&](hipStream_t s) {
        return dlvm::launch_act_adjoint(dt, m->acts[0], B * H, seq_at(dhs, T - 1, B, H, es),
                                        seq_at(hs, T, B, H, es), seq_at(dz, T - 1, B, H, es), s);
      },
      "activation adjoint launch");
  if (st != DLVM_OK) return st;
  for (int64_t t = T - 1; t >= 1; --t) {
    GemmDesc d = rnn_recur(m, B, seq_at(dz, t, B, H, es), U, seq_at(hs, t, B, H, es),
                           seq_at(dhs, t - 1, B, H, es), seq_at(dz, t - 1, B, H, es));
    d.split_ws = at<float>(ws, w.splitk);
    d.split_ws_elems = w.splitk_elems;
    if ((st = run.gemm(d)) != DLVM_OK) return st;
  }
  if (m->wrt_h0 &&
      (st = run.gemm(gemm_nt(dt, DLVM_F32, DLVM_ACT_NONE, B, H, H, dz, H, U, H, nullptr, nullptr,
                             dh0))) != DLVM_OK)
    return st;
  GemmDesc dw = rnn_dw(m, B, xs, dz, dWU, db);
  GemmDesc du = rnn_du(m, B, hs, dz, dWU + Kx * H);
  for (GemmDesc* d : {&dw, &du}) {
    d->split_ws = at<float>(ws, w.splitk);
    d->split_ws_elems = w.splitk_elems;
  }
  if (m->wrt_x) {
    st = run.gemm_pair(dw, gemm_nt(dt, DLVM_F32, DLVM_ACT_NONE, T * B, H, Kx, dz, H, WU, H,
                                   nullptr, nullptr, dxs));
  } else {
    st = run.gemm(dw);
  }
  if (st != DLVM_OK) return st;
  if ((st = run.gemm(du)) != DLVM_OK) return st;
  return run.run(elementwise_info("zero_padding", 0, 1, 4.0 * m->param_count),
                 [&](hipStream_t s) {
                   return dlvm::launch_finalize(nullptr, nullptr, 0, 1.0f, nullptr, nullptr, dparams,
                                                m->gaps, s);
                 },
                 "padding launch");
}

// The launches of one training step up to the update, without running them:
// a gradient call (dense networks), or a forward and a backward call
// (recurrent networks).
void plan_step(const dlvm_model* m, int64_t batch, std::vector<LaunchInfo>* plan) {
  Launcher dry(m, nullptr, plan, 0);
  if (m->kind == 2) {
    std::vector<const void*> mats(m->chain_dims.size() - 1, nullptr);
    chain_model_run(m, mats.data(), nullptr, nullptr, dry);
  } else if (m->kind == 1) {
    const RnnWs w = rnn_ws_layout(m, batch);
    plan_rnn_forward(m, nullptr, nullptr, batch, nullptr, at<float>(nullptr, w.splitk),
                     w.splitk_elems, dry);
    plan_rnn_backward(m, nullptr, nullptr, nullptr, nullptr, batch, nullptr, nullptr, nullptr,
                      nullptr, dry);
  } else {
    plan_gradient(m, nullptr, nullptr, nullptr, batch, nullptr, nullptr, nullptr, nullptr, dry);
  }
}

// The flat parameter layout of m->widths / m->ldw (every tensor on a 256-byte
// boundary in every view; the gaps between tensors are recorded).
void build_layout(dlvm_model* m) {
  // storage dtype and float32 share element offsets: 128 elements is 256
  // bytes of bf16 and 512 bytes of float32
  const int64_t step = 128;
  int64_t off = 0;
  m->gaps.n = 0;
  m->offsets.clear();
  for (int l = 0; l < m->L; ++l) {
    for (int t = 0; t < 2; ++t) {
      const int64_t n = t == 0 ? int64_t(m->widths[l]) * m->ldw[l] : m->widths[l + 1];
      m->offsets.push_back(off);
      const int64_t end = off + n;
      const int64_t next = (end + step - 1) / step * step;
      if (next > end) {
        m->gaps.off[m->gaps.n] = end;
        m->gaps.len[m->gaps.n] = static_cast<int32_t>(next - end);
        ++m->gaps.n;
      }
      off = next;
    }
  }
  m->param_count = off;
}

LaunchInfo sgd_info(const dlvm_model* m) {
  const double per = m->dtype == DLVM_BF16 ? 14.0 : 12.0;  // master/params, grads, (shadow)
  return elementwise_info(m->dtype == DLVM_BF16 ? "sgd_bf16" : "sgd_f32", m->param_count, 1,
                          per * double(m->param_count));
}

void probe_release(ProbeState& p) {
  for (hipEvent_t e : p.start)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : p.stop)
    if (e) (void)hipEventDestroy(e);
  p = ProbeState();
}

}  // namespace

extern "C" {

const char* dlvm_last_error(void) { return g_last_error.c_str(); }

dlvm_status dlvm_create(const dlvm_mlp_desc* desc, dlvm_model** out) {
  if (out == nullptr || desc == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  const int L = desc->n_layers;
  if (L < 1 || L > 30) return fail(DLVM_ERR_INVALID_ARG, "n_layers must be in [1, 30]");
  if (desc->widths == nullptr || desc->acts == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "widths and acts must be given");
  if (!valid_dtype(desc->dtype)) return fail(DLVM_ERR_INVALID_ARG, "unknown dtype");
  if (desc->loss != DLVM_LOSS_SOFTMAX_CE && desc->loss != DLVM_LOSS_CHAIN8)
    return fail(DLVM_ERR_INVALID_ARG, "unknown loss");
  if (desc->batch_max < 1 || desc->batch_max > (int64_t(1) << 24))
    return fail(DLVM_ERR_INVALID_ARG, "batch_max must be in [1, 2^24]");
  for (int l = 0; l <= L; ++l)
    if (desc->widths[l] < 1 || desc->widths[l] > (1 << 20))
      return fail(DLVM_ERR_INVALID_ARG, "every width must be in [1, 2^20]");
  for (int l = 0; l < L; ++l)
    if (!valid_act(desc->acts[l])) return fail(DLVM_ERR_INVALID_ARG, "unknown activation");
  if (desc->acts[L - 1] != DLVM_ACT_NONE)
    return fail(DLVM_ERR_INVALID_ARG, "the last layer must have no activation");
  if (desc->checkpoint_every < 0 || desc->checkpoint_every > L)
    return fail(DLVM_ERR_INVALID_ARG, "checkpoint_every must be in [0, n_layers]");
  if (desc->loss == DLVM_LOSS_CHAIN8) {
    if (L != 1 || desc->widths[0] != desc->widths[1])
      return fail(DLVM_ERR_UNSUPPORTED, "the chain loss needs one layer with in == out");
    if (desc->dtype != DLVM_F32) return fail(DLVM_ERR_UNSUPPORTED, "the chain loss is float32");
    if (!desc->wrt_x) return fail(DLVM_ERR_UNSUPPORTED, "the chain loss differentiates x too");
  }
  for (int l = 0; l < L; ++l) {
    const int64_t es = static_cast<int64_t>(elem_size(desc->dtype));
    const int64_t bytes = static_cast<int64_t>(desc->widths[l]) * desc->widths[l + 1] * es;
    if (bytes > (int64_t(1) << 34)) return fail(DLVM_ERR_INVALID_ARG, "a weight matrix is too large");
  }
  dlvm_model* m = new (std::nothrow) dlvm_model();
  if (m == nullptr) return fail(DLVM_ERR_INVALID_ARG, "out of host memory");
  m->L = L;
  m->widths.assign(desc->widths, desc->widths + L + 1);
  m->acts.assign(desc->acts, desc->acts + L);
  m->dtype = desc->dtype;
  m->loss = desc->loss;
  m->wrt_x = desc->wrt_x ? 1 : 0;
  m->batch_max = desc->batch_max;
  m->ckpt = desc->checkpoint_every > 1 ? desc->checkpoint_every : 1;
  m->chain_epi = desc->loss == DLVM_LOSS_CHAIN8 && desc->chain_in_epilogue ? 1 : 0;
  // The class dimension of a softmax network's last weight matrix is padded
  // to a multiple of 8 (zero columns), so every row is 16-byte aligned.
  for (int l = 0; l < L; ++l) {
    const int64_t n = m->widths[l + 1];
    m->ldw.push_back(m->loss == DLVM_LOSS_SOFTMAX_CE && l == L - 1 ? (n + 7) / 8 * 8 : n);
  }
  build_layout(m);
  std::vector<LaunchInfo> plan;
  plan_step(m, 1, &plan);
  m->n_grad_launches = static_cast<int32_t>(plan.size());
  *out = m;
  return DLVM_OK;
}

dlvm_status dlvm_rnn_create(const dlvm_rnn_desc* desc, dlvm_model** out) {
  if (out == nullptr || desc == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  if (!valid_dtype(desc->dtype)) return fail(DLVM_ERR_INVALID_ARG, "unknown dtype");
  if (!valid_act(desc->act)) return fail(DLVM_ERR_INVALID_ARG, "unknown activation");
  if (desc->steps < 1 || desc->steps > 4096) return fail(DLVM_ERR_INVALID_ARG, "steps must be in [1, 4096]");
  if (desc->in_width < 1 || desc->in_width > (1 << 20) || desc->hidden < 1 || desc->hidden > (1 << 20))
    return fail(DLVM_ERR_INVALID_ARG, "in_width and hidden must be in [1, 2^20]");
  if (desc->batch_max < 1 || desc->batch_max > (int64_t(1) << 24))
    return fail(DLVM_ERR_INVALID_ARG, "batch_max must be in [1, 2^24]");
  const int64_t es = static_cast<int64_t>(elem_size(desc->dtype));
  if ((desc->in_width + desc->hidden) * desc->hidden * es > (int64_t(1) << 34) ||
      desc->steps * desc->batch_max * std::max(desc->in_width, desc->hidden) * 4 > (int64_t(1) << 40))
    return fail(DLVM_ERR_INVALID_ARG, "the network is too large");
  dlvm_model* m = new (std::nothrow) dlvm_model();
  if (m == nullptr) return fail(DLVM_ERR_INVALID_ARG, "out of host memory");
  m->kind = 1;
  m->L = 1;
  m->rnn_T = desc->steps;
  m->rnn_Kx = desc->in_width;
  m->rnn_H = desc->hidden;
  m->widths = {static_cast<int32_t>(desc->in_width + desc->hidden), static_cast<int32_t>(desc->hidden)};
  m->acts = {desc->act};
  m->dtype = desc->dtype;
  m->loss = -1;
  m->wrt_x = desc->wrt_x ? 1 : 0;
  m->wrt_h0 = desc->wrt_h0 ? 1 : 0;
  m->batch_max = desc->batch_max;
  m->ldw = {desc->hidden};
  build_layout(m);
  std::vector<LaunchInfo> plan;
  Launcher dry(m, nullptr, &plan, 0);
  const RnnWs w1 = rnn_ws_layout(m, 1);
  plan_rnn_forward(m, nullptr, nullptr, 1, nullptr, at<float>(nullptr, w1.splitk), w1.splitk_elems,
                   dry);
  m->n_fwd_launches = static_cast<int32_t>(plan.size());
  plan.clear();
  plan_step(m, 1, &plan);
  m->n_grad_launches = static_cast<int32_t>(plan.size());
  *out = m;
  return DLVM_OK;
}

void dlvm_destroy(dlvm_model* m) {
  if (m == nullptr) return;
  probe_release(m->probe);
  delete m;
}

int64_t dlvm_param_count(const dlvm_model* m) { return m ? m->param_count : 0; }

dlvm_status dlvm_param_layout(const dlvm_model* m, int64_t* offsets, int64_t* lds) {
  if (m == nullptr || offsets == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  std::memcpy(offsets, m->offsets.data(), m->offsets.size() * sizeof(int64_t));
  if (lds != nullptr) std::memcpy(lds, m->ldw.data(), m->ldw.size() * sizeof(int64_t));
  return DLVM_OK;
}

size_t dlvm_workspace_bytes(const dlvm_model* m, int64_t batch) {
  if (m == nullptr || batch < 1 || batch > m->batch_max) return 0;
  return ws_total(m, batch);
}

dlvm_status dlvm_workspace_tensor(const dlvm_model* m, int64_t batch, int32_t kind, int32_t layer,
                                  size_t* offset, int64_t* ld, int32_t* dtype) {
  if (m == nullptr || offset == nullptr || ld == nullptr || dtype == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 0) return fail(DLVM_ERR_UNSUPPORTED, "only dense networks keep these tensors");
  const dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  const int L = m->L;
  const bool chain = m->loss == DLVM_LOSS_CHAIN8;
  dlvm::SmallNet sn{};
  if (!chain && small_step_allowed() && m->dtype == DLVM_F32 &&
      dlvm::small_net(L, m->widths.data(), m->acts.data(), m->offsets.data(), m->ldw.data(),
                      batch, m->wrt_x != 0, sn))
    return fail(DLVM_ERR_UNSUPPORTED,
                "the one-workgroup gradient of this network keeps its tensors in LDS only");
  const WsLayout w = ws_layout(m, batch);
  switch (kind) {
    case DLVM_WS_HIDDEN:
      if (layer < 1 || layer >= L) return fail(DLVM_ERR_INVALID_ARG, "hidden layer outside [1, L-1]");
      *offset = w.H[layer];
      *ld = m->widths[layer];
      *dtype = m->dtype;
      return DLVM_OK;
    case DLVM_WS_LOGITS:
      if (chain ? m->chain_epi != 0 : head_splits(m, batch) > 1)
        return fail(DLVM_ERR_UNSUPPORTED,
                    "this plan never stores the output layer's product (its loss kernel sums "
                    "the product's k-slices, or the chain runs in the product's epilogue)");
      *offset = w.logits;
      *ld = m->widths[L];
      *dtype = DLVM_F32;
      return DLVM_OK;
    case DLVM_WS_ADJOINT:
      if (layer < 1 || layer > L) return fail(DLVM_ERR_INVALID_ARG, "layer outside [1, L]");
      *offset = w.dz[layer - 1];
      *ld = m->ldw[layer - 1];
      *dtype = chain ? DLVM_F32 : m->dtype;
      return DLVM_OK;
    default:
      return fail(DLVM_ERR_INVALID_ARG, "unknown workspace tensor kind");
  }
}

dlvm_status dlvm_forward(const dlvm_model* m, const void* params, const void* x, int64_t batch,
                         float* out, void* ws, size_t ws_bytes, void* stream) {
  if (m == nullptr || params == nullptr || x == nullptr || out == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 0) return fail(DLVM_ERR_UNSUPPORTED, "a recurrent model runs dlvm_rnn_forward");
  if (!aligned16(params) || !aligned16(x) || !aligned16(out))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  if ((st = check_ws(m, batch, ws, ws_bytes)) != DLVM_OK) return st;
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, 0);
  return plan_forward(m, params, x, batch, out, ws, run);
}

}  // extern "C"

namespace {
dlvm_status check_gradient_args(const dlvm_model* m, const void* params, const void* x,
                                const int32_t* labels, int64_t batch, float* loss,
                                float* dparams, float* dx, void* ws, size_t ws_bytes) {
  if (m == nullptr || params == nullptr || x == nullptr || loss == nullptr || dparams == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 0) return fail(DLVM_ERR_UNSUPPORTED, "a recurrent model runs dlvm_rnn_backward");
  if (m->loss == DLVM_LOSS_SOFTMAX_CE && labels == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "labels are required for the softmax cross-entropy loss");
  if (m->wrt_x && dx == nullptr) return fail(DLVM_ERR_INVALID_ARG, "dx is required when wrt_x");
  if (!aligned16(params) || !aligned16(x) || !aligned16(dparams) ||
      (labels && !aligned16(labels)) || (dx && !aligned16(dx)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  return check_ws(m, batch, ws, ws_bytes);
}

dlvm_status check_sgd_args(const dlvm_model* m, void* params, float* master, const float* dparams) {
  if (m == nullptr || params == nullptr || dparams == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind == 2) return fail(DLVM_ERR_UNSUPPORTED, "a matrix chain has no parameters to update");
  if (m->dtype == DLVM_BF16 && master == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "bf16 models need float32 master weights");
  if (!aligned16(params) || !aligned16(dparams) || (master && !aligned16(master)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  return DLVM_OK;
}

dlvm_status enqueue_sgd(const dlvm_model* m, void* params, float* master, const float* dparams,
                        float lr, hipStream_t s) {
  Launcher run(m, s, nullptr, m->n_grad_launches);
  float* mst = m->dtype == DLVM_BF16 ? master : nullptr;
  return run.run(sgd_info(m),
                 [&](hipStream_t st) {
                   return dlvm::launch_sgd(m->dtype, m->param_count, params, mst, dparams, lr, st);
                 },
                 "sgd launch");
}
}  // namespace

extern "C" {

dlvm_status dlvm_gradient(const dlvm_model* m, const void* params, const void* x,
                          const int32_t* labels, int64_t batch, float* loss, float* dparams,
                          float* dx, void* ws, size_t ws_bytes, void* stream) {
  dlvm_status st = check_gradient_args(m, params, x, labels, batch, loss, dparams, dx, ws, ws_bytes);
  if (st != DLVM_OK) return st;
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, 0);
  st = plan_gradient(m, params, x, labels, batch, loss, dparams, dx, ws, run);
  m->n_grad_launches = run.launches();
  return st;
}

dlvm_status dlvm_vjp(const dlvm_model* m, const void* params, const void* x, const float* seed,
                     int64_t batch, float* dparams, float* dx, void* ws, size_t ws_bytes,
                     void* stream) {
  if (m == nullptr || params == nullptr || x == nullptr || seed == nullptr || dparams == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 0 || m->loss != DLVM_LOSS_SOFTMAX_CE)
    return fail(DLVM_ERR_UNSUPPORTED, "the seedable gradient is defined for softmax networks' logits");
  if (m->wrt_x && dx == nullptr) return fail(DLVM_ERR_INVALID_ARG, "dx is required when wrt_x");
  if (!aligned16(params) || !aligned16(x) || !aligned16(dparams) || !aligned16(seed) ||
      (dx && !aligned16(dx)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  if ((st = check_ws(m, batch, ws, ws_bytes)) != DLVM_OK) return st;
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, 0);
  return plan_vjp(m, params, x, seed, batch, dparams, dx, ws, run);
}

dlvm_status dlvm_sgd_step(const dlvm_model* m, void* params, float* master, const float* dparams,
                          float lr, void* stream) {
  const dlvm_status st = check_sgd_args(m, params, master, dparams);
  if (st != DLVM_OK) return st;
  return enqueue_sgd(m, params, master, dparams, lr, static_cast<hipStream_t>(stream));
}

dlvm_status dlvm_step_graph_create(const dlvm_model* m, void* params, float* master,
                                   const void* x, const int32_t* labels, int64_t batch,
                                   float* loss, float* dparams, float* dx, void* ws,
                                   size_t ws_bytes, int32_t update, float lr, dlvm_graph** out) {
  if (out == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  dlvm_status st = check_gradient_args(m, params, x, labels, batch, loss, dparams, dx, ws, ws_bytes);
  if (st != DLVM_OK) return st;
  if (update && (st = check_sgd_args(m, params, master, dparams)) != DLVM_OK) return st;
  if (m->probe.armed)
    return fail(DLVM_ERR_UNSUPPORTED, "disarm the timing probe before capturing a step");
  hipStream_t cs = nullptr;
  hipError_t e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  if (e != hipSuccess) return hip_fail(e, "creating the capture stream");
  dlvm_graph* g = new (std::nothrow) dlvm_graph();
  if (g == nullptr) {
    (void)hipStreamDestroy(cs);
    return fail(DLVM_ERR_INVALID_ARG, "out of host memory");
  }
  e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    delete g;
    (void)hipStreamDestroy(cs);
    return hip_fail(e, "beginning the capture");
  }
  {
    Launcher run(m, cs, nullptr, 0);
    st = plan_gradient(m, params, x, labels, batch, loss, dparams, dx, ws, run);
    m->n_grad_launches = run.launches();
  }
  if (st == DLVM_OK && update) st = enqueue_sgd(m, params, master, dparams, lr, cs);
  const std::string err = st == DLVM_OK ? std::string() : g_last_error;
  e = hipStreamEndCapture(cs, &g->graph);
  if (st == DLVM_OK && e != hipSuccess) st = hip_fail(e, "ending the capture");
  if (st == DLVM_OK) {
    e = hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0);
    if (e != hipSuccess) st = hip_fail(e, "instantiating the step graph");
  } else if (!err.empty()) {
    g_last_error = err;
  }
  (void)hipStreamDestroy(cs);
  if (st != DLVM_OK) {
    dlvm_graph_destroy(g);
    return st;
  }
  *out = g;
  return DLVM_OK;
}

dlvm_status dlvm_graph_launch(dlvm_graph* g, void* stream) {
  if (g == nullptr || g->exec == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null graph");
  const hipError_t e = hipGraphLaunch(g->exec, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "launching the step graph");
  return DLVM_OK;
}

void dlvm_graph_destroy(dlvm_graph* g) {
  if (g == nullptr) return;
  if (g->exec) (void)hipGraphExecDestroy(g->exec);
  if (g->graph) (void)hipGraphDestroy(g->graph);
  delete g;
}

int32_t dlvm_plan_size(const dlvm_model* m, int64_t batch) {
  if (m == nullptr || batch < 1 || batch > m->batch_max) return 0;
  std::vector<LaunchInfo> plan;
  plan_step(m, batch, &plan);
  return static_cast<int32_t>(plan.size()) + 1;
}

dlvm_status dlvm_plan_entry(const dlvm_model* m, int64_t batch, int32_t index,
                            dlvm_launch_info* info) {
  if (m == nullptr || info == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  std::vector<LaunchInfo> plan;
  plan_step(m, batch, &plan);
  plan.push_back(sgd_info(m));
  if (index < 0 || index >= static_cast<int32_t>(plan.size()))
    return fail(DLVM_ERR_INVALID_ARG, "launch index out of range");
  const LaunchInfo& li = plan[index];
  std::memset(info, 0, sizeof(*info));
  std::strncpy(info->name, li.name.c_str(), sizeof(info->name) - 1);
  info->M = li.M; info->N = li.N; info->K = li.K;
  info->flops = li.flops;
  info->bytes = li.bytes;
  return DLVM_OK;
}

dlvm_status dlvm_probe_arm(dlvm_model* m, int32_t index, int32_t capacity) {
  if (m == nullptr || capacity < 1 || capacity > (1 << 20) || index < -1)
    return fail(DLVM_ERR_INVALID_ARG, "bad probe arguments");
  probe_release(m->probe);
  ProbeState& p = m->probe;
  p.start.assign(capacity, nullptr);
  p.stop.assign(capacity, nullptr);
  p.pos.assign(capacity, -1);
  for (int32_t i = 0; i < capacity; ++i) {
    hipError_t e = hipEventCreate(&p.start[i]);
    if (e == hipSuccess) e = hipEventCreate(&p.stop[i]);
    if (e != hipSuccess) {
      probe_release(p);
      return hip_fail(e, "creating probe events");
    }
  }
  p.index = index;
  p.capacity = capacity;
  p.used = 0;
  p.armed = true;
  return DLVM_OK;
}

dlvm_status dlvm_probe_read(dlvm_model* m, int32_t index, int64_t* count, double* total_ms) {
  if (m == nullptr || count == nullptr || total_ms == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  ProbeState& p = m->probe;
  *count = 0;
  *total_ms = 0.0;
  for (int32_t i = 0; i < p.used; ++i) {
    if (index >= 0 && p.pos[i] != index) continue;
    hipError_t e = hipEventSynchronize(p.stop[i]);
    float ms = 0.0f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.start[i], p.stop[i]);
    if (e != hipSuccess) return hip_fail(e, "reading probe events");
    *count += 1;
    *total_ms += ms;
  }
  return DLVM_OK;
}

dlvm_status dlvm_probe_disarm(dlvm_model* m) {
  if (m == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  probe_release(m->probe);
  return DLVM_OK;
}

dlvm_status dlvm_check(const dlvm_model* m, void* ws, void* stream) {
  if (m == nullptr || ws == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 0) return fail(DLVM_ERR_UNSUPPORTED, "only dense-network calls write device flags");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t flags[4] = {0, 0, 0, 0};
  hipError_t e = hipMemcpyAsync(flags, ws, 2 * sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "reading the workspace flags");
  if (flags[0]) return fail(DLVM_ERR_LABEL_RANGE, "a label was outside [0, classes)");
  if (flags[1]) return fail(DLVM_ERR_NONFINITE, "the loss was not finite");
  return DLVM_OK;
}

dlvm_status dlvm_rnn_forward(const dlvm_model* m, const void* params, const void* xs,
                             int64_t batch, void* hs, void* ws, size_t ws_bytes, void* stream) {
  if (m == nullptr || params == nullptr || xs == nullptr || hs == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 1) return fail(DLVM_ERR_UNSUPPORTED, "not a recurrent model");
  if (!aligned16(params) || !aligned16(xs) || !aligned16(hs))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  if (ws != nullptr && (st = check_ws(m, batch, ws, ws_bytes)) != DLVM_OK) return st;
  const RnnWs w = rnn_ws_layout(m, batch);
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, 0);
  return plan_rnn_forward(m, params, xs, batch, hs,
                          ws != nullptr ? at<float>(ws, w.splitk) : nullptr, w.splitk_elems, run);
}

dlvm_status dlvm_rnn_backward(const dlvm_model* m, const void* params, const void* xs,
                              const void* hs, const void* dhs, int64_t batch, float* dparams,
                              float* dxs, float* dh0, void* ws, size_t ws_bytes, void* stream) {
  if (m == nullptr || params == nullptr || xs == nullptr || hs == nullptr || dhs == nullptr ||
      dparams == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 1) return fail(DLVM_ERR_UNSUPPORTED, "not a recurrent model");
  if (m->wrt_x && dxs == nullptr) return fail(DLVM_ERR_INVALID_ARG, "dxs is required when wrt_x");
  if (m->wrt_h0 && dh0 == nullptr) return fail(DLVM_ERR_INVALID_ARG, "dh0 is required when wrt_h0");
  if (!aligned16(params) || !aligned16(xs) || !aligned16(hs) || !aligned16(dhs) ||
      !aligned16(dparams) || (dxs && !aligned16(dxs)) || (dh0 && !aligned16(dh0)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  dlvm_status st = check_batch(m, batch);
  if (st != DLVM_OK) return st;
  if ((st = check_ws(m, batch, ws, ws_bytes)) != DLVM_OK) return st;
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, m->n_fwd_launches);
  st = plan_rnn_backward(m, params, xs, hs, dhs, batch, dparams, dxs, dh0, ws, run);
  m->n_grad_launches = run.launches();
  return st;
}

// ---------------------------------------------------------------------------
// Matrix multiplication reordering (section 3.1.2)
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

constexpr int kChainMax = 32;

// Multiply-adds of the best order of every sub-chain A_i..A_j (A_i is
// d[i] x d[i+1]; a p x q by q x r product costs p q r), sub-chains taken by
// increasing length, the outermost cut of each recorded in split[i * n + j]
// (the smallest cut among equal costs). Returns the whole chain's cost.
unsigned __int128 chain_optimal(int n, const int64_t* d, int32_t* split) {
  std::vector<unsigned __int128> cost(static_cast<size_t>(n) * n, 0);
  for (int len = 2; len <= n; ++len) {
    for (int i = 0; i + len - 1 < n; ++i) {
      const int j = i + len - 1;
      bool have = false;
      for (int k = i; k < j; ++k) {
        const unsigned __int128 c = cost[i * n + k] + cost[(k + 1) * n + j] +
                                    static_cast<unsigned __int128>(d[i]) * d[k + 1] * d[j + 1];
        if (!have || c < cost[i * n + j]) {
          cost[i * n + j] = c;
          split[i * n + j] = k;
          have = true;
        }
      }
    }
  }
  return cost[n - 1];
}

// Every cut reachable from the whole chain lies inside its sub-chain.
bool chain_split_valid(int n, const int32_t* split, int i, int j) {
  if (i == j) return true;
  const int k = split[i * n + j];
  return k >= i && k < j && chain_split_valid(n, split, i, k) &&
         chain_split_valid(n, split, k + 1, j);
}

// The product that computes A_i..A_j from its two sides (a and b), into dst:
// the planner may split its contraction (the k-slices' sum then applies the
// epilogue) when the scratch holds the slices.
GemmDesc chain_product(int dtype, int n, const int64_t* d, const int32_t* split, int i, int j,
                       const void* a, const void* b, void* dst) {
  const int k = split[i * n + j];
  const bool root = i == 0 && j == n - 1;
  GemmDesc g = gemm_nn(dtype, root ? DLVM_F32 : dtype, DLVM_ACT_NONE, d[i], d[j + 1], d[k + 1],
                       1.0f, a, b, d[j + 1], nullptr, dst, d[j + 1]);
  g.split_epilogue = true;
  return g;
}

// Workspace offsets of the intermediate products (every inner node of the
// order but the whole chain), in evaluation order; returns the end offset.
// `split_elems` receives the largest float32 k-slice scratch any product of
// the order may use.
size_t chain_layout(int dtype, int n, const int64_t* d, const int32_t* split, int i, int j,
                    std::vector<size_t>& off, size_t base, int64_t& split_elems) {
  if (i == j) return base;
  const int k = split[i * n + j];
  base = chain_layout(dtype, n, d, split, i, k, off, base, split_elems);
  base = chain_layout(dtype, n, d, split, k + 1, j, off, base, split_elems);
  split_elems = std::max(split_elems, dlvm::split_ws_elems(chain_product(
                                          dtype, n, d, split, i, j, nullptr, nullptr, nullptr)));
  if (!(i == 0 && j == n - 1)) {
    off[i * n + j] = base;
    base = align_up(base + static_cast<size_t>(d[i] * d[j + 1]) * elem_size(dtype));
  }
  return base;
}

// Total workspace of an order: the intermediates, then the k-slice scratch.
size_t chain_ws(int dtype, int n, const int64_t* d, const int32_t* split,
                std::vector<size_t>& off, size_t& split_off, int64_t& split_elems) {
  split_elems = 0;
  split_off = chain_layout(dtype, n, d, split, 0, n - 1, off, 0, split_elems);
  return align_up(split_off + static_cast<size_t>(split_elems) * 4);
}

dlvm_status chain_args(int32_t dtype, int32_t n, const int64_t* dims, const int32_t* split) {
  if (!valid_dtype(dtype)) return fail(DLVM_ERR_INVALID_ARG, "unknown dtype");
  if (n < 2 || n > kChainMax || dims == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "a chain has 2 to 32 matrices and their dims");
  for (int i = 0; i <= n; ++i)
    if (dims[i] < 1 || dims[i] > (int64_t(1) << 20))
      return fail(DLVM_ERR_INVALID_ARG, "every dimension must be in [1, 2^20]");
  if (split != nullptr && !chain_split_valid(n, split, 0, n - 1))
    return fail(DLVM_ERR_INVALID_ARG, "the split table is not an order of the chain");
  return DLVM_OK;
}

// The order to run: the caller's, or the optimal one.
std::vector<int32_t> chain_split(int n, const int64_t* dims, const int32_t* split) {
  std::vector<int32_t> s(static_cast<size_t>(n) * n, -1);
  if (split != nullptr)
    std::memcpy(s.data(), split, s.size() * sizeof(int32_t));
  else
    chain_optimal(n, dims, s.data());
  return s;
}

// Evaluate A_i..A_j into dst (the whole chain: float32 `out`; an inner node:
// its workspace buffer in the storage dtype); returns the operand pointer.
struct ChainRun {
  int dtype, n;
  const int64_t* d;
  const void* const* mats;
  const int32_t* split;
  const std::vector<size_t>* off;
  float* out;
  void* ws;
  float* split_ws;
  int64_t split_elems;
};

dlvm_status chain_eval(const ChainRun& c, int i, int j, const void** result, Launcher& run) {
  if (i == j) {
    *result = c.mats[i];
    return DLVM_OK;
  }
  const int k = c.split[i * c.n + j];
  const void* a = nullptr;
  const void* b = nullptr;
  dlvm_status st = chain_eval(c, i, k, &a, run);
  if (st == DLVM_OK) st = chain_eval(c, k + 1, j, &b, run);
  if (st != DLVM_OK) return st;
  const bool root = i == 0 && j == c.n - 1;
  void* dst = root ? static_cast<void*>(c.out) : at<void>(c.ws, (*c.off)[i * c.n + j]);
  GemmDesc g = chain_product(c.dtype, c.n, c.d, c.split, i, j, a, b, dst);
  g.split_ws = c.split_ws;
  g.split_ws_elems = c.split_elems;
  *result = dst;
  return run.gemm(g);
}

size_t chain_model_ws(const dlvm_model* m) {
  const int n = static_cast<int>(m->chain_dims.size()) - 1;
  std::vector<size_t> off(static_cast<size_t>(n) * n, 0);
  size_t split_off = 0;
  int64_t split_elems = 0;
  return std::max<size_t>(
      chain_ws(m->dtype, n, m->chain_dims.data(), m->chain_cuts.data(), off, split_off, split_elems),
      16);
}

dlvm_status chain_model_run(const dlvm_model* m, const void* const* mats, float* out, void* ws,
                            Launcher& run) {
  const int n = static_cast<int>(m->chain_dims.size()) - 1;
  std::vector<size_t> off(static_cast<size_t>(n) * n, 0);
  size_t split_off = 0;
  int64_t split_elems = 0;
  chain_ws(m->dtype, n, m->chain_dims.data(), m->chain_cuts.data(), off, split_off, split_elems);
  const ChainRun c{m->dtype, n, m->chain_dims.data(), mats, m->chain_cuts.data(), &off, out, ws,
                   split_elems > 0 ? at<float>(ws, split_off) : nullptr, split_elems};
  const void* res = nullptr;
  return chain_eval(c, 0, n - 1, &res, run);
}

}  // namespace

extern "C" {

dlvm_status dlvm_chain_create(int32_t dtype, int32_t n, const int64_t* dims, const int32_t* split,
                              dlvm_model** out) {
  if (out == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  *out = nullptr;
  const dlvm_status st = chain_args(dtype, n, dims, split);
  if (st != DLVM_OK) return st;
  dlvm_model* m = new (std::nothrow) dlvm_model();
  if (m == nullptr) return fail(DLVM_ERR_INVALID_ARG, "out of host memory");
  m->kind = 2;
  m->dtype = dtype;
  m->loss = -1;
  m->batch_max = 1;
  m->chain_dims.assign(dims, dims + n + 1);
  m->chain_cuts = chain_split(n, dims, split);
  std::vector<LaunchInfo> plan;
  plan_step(m, 1, &plan);
  m->n_grad_launches = static_cast<int32_t>(plan.size());
  *out = m;
  return DLVM_OK;
}

dlvm_status dlvm_chain_run(const dlvm_model* m, const void* const* mats, float* out, void* ws,
                           size_t ws_bytes, void* stream) {
  if (m == nullptr || mats == nullptr || out == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (m->kind != 2) return fail(DLVM_ERR_UNSUPPORTED, "not a matrix-chain handle");
  const int n = static_cast<int>(m->chain_dims.size()) - 1;
  for (int i = 0; i < n; ++i) {
    if (mats[i] == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null matrix");
    if (!aligned16(mats[i])) return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  }
  if (!aligned16(out)) return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  const dlvm_status st = check_ws(m, 1, ws, ws_bytes);
  if (st != DLVM_OK) return st;
  Launcher run(m, static_cast<hipStream_t>(stream), nullptr, 0);
  return chain_model_run(m, mats, out, ws, run);
}

int64_t dlvm_chain_order(int32_t n, const int64_t* dims, int32_t* split) {
  if (n < 1 || n > kChainMax || dims == nullptr) return -1;
  for (int i = 0; i <= n; ++i)
    if (dims[i] < 1 || dims[i] > (int64_t(1) << 20)) return -1;
  std::vector<int32_t> s(static_cast<size_t>(n) * n, -1);
  const unsigned __int128 c = chain_optimal(n, dims, s.data());
  if (split != nullptr) std::memcpy(split, s.data(), s.size() * sizeof(int32_t));
  const unsigned __int128 lim = static_cast<unsigned __int128>(INT64_MAX);
  return static_cast<int64_t>(c > lim ? lim : c);
}

size_t dlvm_matrix_chain_ws_bytes(int32_t dtype, int32_t n, const int64_t* dims,
                                  const int32_t* split) {
  if (chain_args(dtype, n, dims, split) != DLVM_OK) return 0;
  const std::vector<int32_t> sp = chain_split(n, dims, split);
  std::vector<size_t> off(static_cast<size_t>(n) * n, 0);
  size_t split_off = 0;
  int64_t split_elems = 0;
  return std::max<size_t>(chain_ws(dtype, n, dims, sp.data(), off, split_off, split_elems), 16);
}

dlvm_status dlvm_matrix_chain(int32_t dtype, int32_t n, const int64_t* dims,
                              const void* const* mats, const int32_t* split, float* out, void* ws,
                              size_t ws_bytes, void* stream) {
  dlvm_status st = chain_args(dtype, n, dims, split);
  if (st != DLVM_OK) return st;
  if (mats == nullptr || out == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  for (int i = 0; i < n; ++i) {
    if (mats[i] == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null matrix");
    if (!aligned16(mats[i])) return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  }
  if (!aligned16(out)) return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  const std::vector<int32_t> sp = chain_split(n, dims, split);
  std::vector<size_t> off(static_cast<size_t>(n) * n, 0);
  size_t split_off = 0;
  int64_t split_elems = 0;
  const size_t need = chain_ws(dtype, n, dims, sp.data(), off, split_off, split_elems);
  if (need > 0 && (ws == nullptr || ws_bytes < need))
    return fail(DLVM_ERR_WORKSPACE, "workspace is smaller than dlvm_matrix_chain_ws_bytes");
  if (ws != nullptr && !aligned16(ws)) return fail(DLVM_ERR_MISALIGNED, "workspace is not 16-byte aligned");
  const ChainRun c{dtype, n, dims, mats, sp.data(), &off, out, ws,
                   split_elems > 0 ? at<float>(ws, split_off) : nullptr, split_elems};
  Launcher run(nullptr, static_cast<hipStream_t>(stream), nullptr, 0);
  const void* res = nullptr;
  return chain_eval(c, 0, n - 1, &res, run);
}

// ---------------------------------------------------------------------------
// Step-level entry points
// ---------------------------------------------------------------------------
dlvm_status dlvm_dense_forward(int32_t dtype, int32_t out_dtype, int32_t act, int64_t M, int64_t N,
                               int64_t K, float alpha, const void* X, const void* W,
                               const void* bias, void* H, void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(out_dtype) || !valid_act(act))
    return fail(DLVM_ERR_INVALID_ARG, "bad dtype or activation");
  if (dtype == DLVM_F32 && out_dtype != DLVM_F32)
    return fail(DLVM_ERR_UNSUPPORTED, "float32 operands give float32 outputs");
  if (M < 1 || N < 1 || K < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (X == nullptr || W == nullptr || H == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (!aligned16(X) || !aligned16(W) || !aligned16(H) || (bias && !aligned16(bias)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  return run_gemm(gemm_nn(dtype, out_dtype, act, M, N, K, alpha, X, W, N, bias, H, N),
                  static_cast<hipStream_t>(stream));
}

dlvm_status dlvm_rnn_cell_forward(int32_t dtype, int32_t act, int64_t M, int64_t Kx, int64_t Kh,
                                  int64_t N, const void* X, const void* H, const void* WU,
                                  const void* bias, void* Hout, void* stream) {
  if (!valid_dtype(dtype) || !valid_act(act)) return fail(DLVM_ERR_INVALID_ARG, "bad dtype or activation");
  if (M < 1 || Kx < 1 || Kh < 1 || N < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (X == nullptr || H == nullptr || WU == nullptr || Hout == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (!aligned16(X) || !aligned16(H) || !aligned16(WU) || !aligned16(Hout) ||
      (bias && !aligned16(bias)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  GemmDesc d = gemm_nn(dtype, dtype, act, M, N, Kx + Kh, 1.0f, X, WU, N, bias, Hout, N);
  d.lda = Kx;
  d.A2 = H;
  d.lda2 = Kh;
  d.K1 = Kx;
  return run_gemm(d, static_cast<hipStream_t>(stream));
}

dlvm_status dlvm_dense_backward_data(int32_t dtype, int32_t out_dtype, int32_t act_prev, int64_t M,
                                     int64_t N, int64_t K, const void* dY, const void* W,
                                     const void* Hprev, const void* R, void* dX, void* stream) {
  if (!valid_dtype(dtype) || !valid_dtype(out_dtype) || !valid_act(act_prev))
    return fail(DLVM_ERR_INVALID_ARG, "bad dtype or activation");
  if (dtype == DLVM_F32 && out_dtype != DLVM_F32)
    return fail(DLVM_ERR_UNSUPPORTED, "float32 operands give float32 outputs");
  if (M < 1 || N < 1 || K < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (dY == nullptr || W == nullptr || dX == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (act_prev != DLVM_ACT_NONE && Hprev == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "Hprev is required for an activation derivative");
  if (!aligned16(dY) || !aligned16(W) || !aligned16(dX) || (Hprev && !aligned16(Hprev)) ||
      (R && !aligned16(R)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  return run_gemm(gemm_nt(dtype, out_dtype, act_prev, M, N, K, dY, N, W, N, Hprev, R, dX),
                  static_cast<hipStream_t>(stream));
}

dlvm_status dlvm_dense_backward_params(int32_t dtype, int64_t M, int64_t N, int64_t K,
                                       const void* X, const void* dY, float* dW, float* db,
                                       void* stream) {
  if (!valid_dtype(dtype)) return fail(DLVM_ERR_INVALID_ARG, "bad dtype");
  if (M < 1 || N < 1 || K < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (X == nullptr || dY == nullptr || dW == nullptr) return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (!aligned16(X) || !aligned16(dY) || !aligned16(dW) || (db && !aligned16(db)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  return run_gemm(gemm_tn(dtype, M, N, K, X, dY, N, dW, N, db, N), static_cast<hipStream_t>(stream));
}

size_t dlvm_softmax_xent_ws_bytes(int64_t rows) {
  if (rows < 1) return 0;
  return align_up(16) + 2 * align_up(static_cast<size_t>(dlvm::softmax_xent_partials(rows)) * 4);
}

dlvm_status dlvm_softmax_xent(int32_t dtype, int64_t rows, int64_t classes, const float* logits,
                              const int32_t* labels, float scale, void* dlogits, float* loss,
                              void* ws, size_t ws_bytes, void* stream) {
  if (!valid_dtype(dtype)) return fail(DLVM_ERR_INVALID_ARG, "bad dtype");
  if (rows < 1 || classes < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (logits == nullptr || labels == nullptr || dlogits == nullptr || loss == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (ws == nullptr || ws_bytes < dlvm_softmax_xent_ws_bytes(rows))
    return fail(DLVM_ERR_WORKSPACE, "workspace missing or too small");
  if (!aligned16(logits) || !aligned16(labels) || !aligned16(dlogits) || !aligned16(loss) ||
      !aligned16(ws))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* flags = at<int32_t>(ws, 0);
  float* partials = at<float>(ws, align_up(16));
  int32_t* bad = at<int32_t>(ws, align_up(16) +
                                     align_up(static_cast<size_t>(dlvm::softmax_xent_partials(rows)) * 4));
  int np = 0;
  hipError_t e = dlvm::launch_softmax_xent(dtype, rows, classes, logits, labels, scale, dlogits,
                                           classes, partials, bad, &np, s);
  if (e != hipSuccess) return hip_fail(e, "softmax cross-entropy launch");
  dlvm::ZeroGaps none{};
  e = dlvm::launch_finalize(partials, bad, np, scale, loss, flags, nullptr, none, s);
  if (e != hipSuccess) return hip_fail(e, "loss finalisation launch");
  return DLVM_OK;
}

}  // extern "C"

// Scratch of the allocation-free softmax cross-entropy: the per-block loss
// partials and bad-label counts of at most kNoAllocMaxRows rows (2 MiB), in a
// device array each GPU holds for the life of the process. In host code the
// array's name is only a stand-in: its device address on the current device
// comes from hipGetSymbolAddress, looked up once per device and kept.
constexpr int64_t kNoAllocMaxRows = int64_t(1) << 20;
constexpr int64_t kNoAllocPartials = (kNoAllocMaxRows + 3) / 4;  // >= softmax_xent_partials(max)
static __device__ __align__(256) float scratch[2 * kNoAllocPartials];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch[kMaxDevices] = {};

dlvm_status scratch_on_current_device(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(DLVM_ERR_UNSUPPORTED, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || ptr == nullptr) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    g_scratch[dev] = static_cast<float*>(ptr);
  }
  *out = g_scratch[dev];
  return DLVM_OK;
}
}  // namespace

extern "C" {

dlvm_status dlvm_softmax_xent_noalloc(int32_t dtype, int64_t rows, int64_t classes,
                                      const float* logits, const int32_t* labels, float scale,
                                      void* dlogits, float* loss, int32_t* flags, void* stream) {
  if (!valid_dtype(dtype)) return fail(DLVM_ERR_INVALID_ARG, "bad dtype");
  if (rows < 1 || classes < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (rows > kNoAllocMaxRows)
    return fail(DLVM_ERR_INVALID_ARG,
                "rows exceed the 1048576 that the static scratch of dlvm_softmax_xent_noalloc holds");
  if (logits == nullptr || labels == nullptr || dlogits == nullptr || loss == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (!aligned16(logits) || !aligned16(labels) || !aligned16(dlogits) || !aligned16(loss) ||
      (flags != nullptr && !aligned16(flags)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  float* base = nullptr;
  dlvm_status st = scratch_on_current_device(&base);
  if (st != DLVM_OK) return st;
  // every partial and count the finalisation reads is written by the loss
  // launch just before it: nothing needs clearing between calls
  float* partials = base;
  int32_t* bad = reinterpret_cast<int32_t*>(base + kNoAllocPartials);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int np = 0;
  hipError_t e = dlvm::launch_softmax_xent(dtype, rows, classes, logits, labels, scale, dlogits,
                                           classes, partials, bad, &np, s);
  if (e != hipSuccess) return hip_fail(e, "softmax cross-entropy launch");
  dlvm::ZeroGaps none{};
  e = dlvm::launch_finalize(partials, bad, np, scale, loss, flags, nullptr, none, s);
  if (e != hipSuccess) return hip_fail(e, "loss finalisation launch");
  return DLVM_OK;
}

size_t dlvm_chain8_ws_bytes(int64_t rows, int64_t cols) {
  if (rows < 1 || cols < 1) return 0;
  return align_up(16) + align_up(static_cast<size_t>(dlvm::chain8_partials(rows, cols)) * 4);
}

dlvm_status dlvm_chain8(int64_t rows, int64_t cols, const float* z, const float* bias,
                        const float* x_skip, float* zbar, float* xbar, float* loss, void* ws,
                        size_t ws_bytes, void* stream) {
  if (rows < 1 || cols < 1) return fail(DLVM_ERR_INVALID_ARG, "sizes must be positive");
  if (z == nullptr || bias == nullptr || x_skip == nullptr || zbar == nullptr || xbar == nullptr ||
      loss == nullptr)
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (ws == nullptr || ws_bytes < dlvm_chain8_ws_bytes(rows, cols))
    return fail(DLVM_ERR_WORKSPACE, "workspace missing or too small");
  if (!aligned16(z) || !aligned16(bias) || !aligned16(x_skip) || !aligned16(zbar) ||
      !aligned16(xbar) || !aligned16(loss) || !aligned16(ws))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* flags = at<int32_t>(ws, 0);
  float* partials = at<float>(ws, align_up(16));
  int np = 0;
  hipError_t e = dlvm::launch_chain8(rows, cols, z, bias, x_skip, zbar, xbar, partials, false, &np, s);
  if (e != hipSuccess) return hip_fail(e, "chain launch");
  dlvm::ZeroGaps none{};
  const float scale = static_cast<float>(1.0 / (static_cast<double>(rows) * static_cast<double>(cols)));
  e = dlvm::launch_finalize(partials, nullptr, np, scale, loss, flags, nullptr, none, s);
  if (e != hipSuccess) return hip_fail(e, "loss finalisation launch");
  return DLVM_OK;
}

dlvm_status dlvm_sgd(int32_t dtype, int64_t n, void* params, float* master, const float* grads,
                     float lr, void* stream) {
  if (!valid_dtype(dtype)) return fail(DLVM_ERR_INVALID_ARG, "bad dtype");
  if (n < 1) return fail(DLVM_ERR_INVALID_ARG, "n must be positive");
  if (params == nullptr || grads == nullptr || (dtype == DLVM_BF16 && master == nullptr))
    return fail(DLVM_ERR_INVALID_ARG, "null argument");
  if (!aligned16(params) || !aligned16(grads) || (master && !aligned16(master)))
    return fail(DLVM_ERR_MISALIGNED, "device pointers must be 16-byte aligned");
  const hipError_t e = dlvm::launch_sgd(dtype, n, params, master, grads, lr,
                                        static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "sgd launch");
  return DLVM_OK;
}

}  // extern "C"
