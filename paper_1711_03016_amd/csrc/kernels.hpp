// Host-side launch interface of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dlvm {

// Timing events for the next kernel launches of the calling host thread. When
// `start` is set, launch_kernel records both events from the kernel's own
// dispatch packet (its begin and end on the GPU), so their difference is the
// kernel's duration without the gap an event recorded beside the launch adds.
struct PacketEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
PacketEvents& packet_events();

template <typename K, typename... Args>
inline void launch_kernel(K kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  const PacketEvents& e = packet_events();
  if (e.start != nullptr)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, e.start, e.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

enum class Layout : int {
  NN = 0,  // C = A.B        A [M,K] K-contiguous, B [K,N] N-contiguous (forward)
  NT = 1,  // C = A.B^T      A [M,K] K-contiguous, B [N,K] K-contiguous (adjoint wrt input)
  TN = 2,  // C = A^T.B      A [K,M] M-contiguous, B [K,N] N-contiguous (adjoint wrt weights)
};

struct GemmDesc {
  Layout layout;
  int dtype;       // operand storage: F32 or BF16
  int out_dtype;   // C storage: F32 or BF16
  int act;         // NN: activation applied; NT: activation whose derivative is applied
  int64_t M, N, K;
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  void* C; int64_t ldc;
  const void* bias;      // NN: [N] in operand dtype, or null
  const void* aux;       // NT: saved activation [M, ldc] in operand dtype, or null
  const void* residual;  // NT: [M, ldc] in out dtype added after act' (before, with res_pre), or null
  float* colsum;         // TN: [nvec] float32 sum over k of B(k, n), or null
  float alpha;           // NN: scale of the product
  int64_t nvec;          // entries of bias / colsum (0 means N). Columns n >= nvec
                         // have none; with a padded operand they are zero.
  int64_t kvalid;        // unpadded contraction extent, for work accounting (0 means K)
  // Float32 scratch for a split reduction over K (null: no split). The
  // planner splits products wrt the weights (TN) by its estimate; another
  // layout is split only when splits_hint asks for it (its caller sums the
  // slices: an NN product's slices are the raw products, without bias or
  // activation).
  float* split_ws;
  int64_t split_ws_elems;
  int splits_hint;  // > 0: use exactly this many k-slices if the scratch holds them
  // Second source of A (null: none). The contraction then has two phases:
  // k < K1 from A (stride lda) and k in [K1, K) from A2 (stride lda2, column
  // or row k - K1), accumulated into the same outputs; B spans all K. Such a
  // product is never split over K.
  const void* A2;
  int64_t lda2, K1;
  bool res_pre;  // NT: the residual is added before act' is applied
  // NN / NT: the planner may split K (scratch permitting): the k-slices write
  // raw float32 partials to split_ws and launch_split_epilogue sums them and
  // applies the product's epilogue. A two-phase product is split only at
  // slice boundaries that fall on K1.
  bool split_epilogue;
  // NN float32 only: the eight-operator chain in the epilogue (z = the
  // product; bias, x_skip = aux): C receives zbar, C2 xbar, and partials one
  // loss term (sum of e^2) per wavefront of each tile (chain_partials of them);
  // inv_n is the seed 1 / (M N) of the mean. Never split.
  bool chain_epilogue;
  void* C2;
  float* partials;
  float inv_n;
  // bf16 rectified layers on the 256 x 256 or 64 x 128 direct-to-LDS tile,
  // unsplit (mask_ok): an NN product writes the rectifier bits of its output
  // here, an NT product reads them in place of aux. Null: none.
  uint32_t* mask;
};

// How one product is launched: tile configuration and grid.
struct GemmPlan {
  int cfg;               // tile configuration index
  int bm, bn;            // tile shape
  int tiles_m, tiles_n;
  int splits;            // k-slices (1: none); partials in GemmDesc::split_ws
  int64_t k_chunk;       // k per slice
};

// Float32 scratch elements a split reduction of this product may use: enough
// for the largest split the planner can choose (0 for products it never splits).
int64_t split_ws_elems(const GemmDesc& d);

// Choose the launch of a product.
GemmPlan plan_gemm(const GemmDesc& d);

// Whether a product so planned can write (NN) or read (NT) rectifier masks
// (GemmDesc::mask): bf16 operands and output, the rectifier, the 256 x 256 or
// 64 x 128 direct-to-LDS tile (configurations 10 and 16: the mask is in the
// tile's accumulator order), one k-slice, one phase, no residual. Both
// products of a layer output must pass, on the same configuration, for the
// mask to be used.
bool mask_ok(const GemmDesc& d, const GemmPlan& plan);
// Bytes of the mask of an M x N output (one bit per element of whole tiles of
// either configuration: 8 KiB per 256 x 256 tile, 1 KiB per 64 x 128).
int64_t mask_bytes(int64_t M, int64_t N);

// Between begin and end (nestable; one library call), the tuning variables
// DLVM_GEMM_CONFIG / DLVM_GEMM_SPLITS are read once instead of per product.
void tuning_scope_begin();
void tuning_scope_end();

// Loss partials a chain-epilogue product writes (one per wavefront of a tile).
int64_t chain_partials(const GemmPlan& plan);

// Enqueue one GEMM with its fused epilogue as planned. Returns hipSuccess or
// the launch error. The caller has validated shapes and pointers.
hipError_t launch_gemm(const GemmDesc& d, const GemmPlan& plan, hipStream_t s);

// The two adjoint products of one layer (tn: wrt the weights, nt: wrt the
// input) can run as one launch when planned on the same configuration.
bool pairable(const GemmDesc& tn, const GemmPlan& ptn, const GemmDesc& nt, const GemmPlan& pnt);
hipError_t launch_gemm_pair(const GemmDesc& tn, const GemmPlan& ptn, const GemmDesc& nt,
                            const GemmPlan& pnt, hipStream_t s);

// Softmax cross-entropy rows: one partial loss per row block into `partials`.
// Returns the number of partials written through *n_partials.
// `bad` receives, per row block, the number of labels outside [0, classes).
// dlogits rows have stride ld_dlogits >= classes; columns [classes, ld) are written as 0.
// Softmax cross-entropy whose logits arrive as the k-slices of a split
// product: z[r, c] = sum_s part[s * c_split + r * ld_part + c] (slice order)
// + bias[c] (bias in the storage dtype `dtype`), then as launch_softmax_xent.
hipError_t launch_split_softmax_xent(int dtype, int splits, int64_t rows, int64_t classes,
                                     const float* part, int64_t c_split, int64_t ld_part,
                                     const void* bias, const int32_t* labels, float scale,
                                     void* dlogits, int64_t ld_dlogits, float* partials,
                                     int32_t* bad, int* n_partials, hipStream_t s);

hipError_t launch_softmax_xent(int dtype, int64_t rows, int64_t classes, const float* logits,
                               const int32_t* labels, float scale, void* dlogits,
                               int64_t ld_dlogits, float* partials, int32_t* bad, int* n_partials,
                               hipStream_t s);
int softmax_xent_partials(int64_t rows);

// Fused chain; `fwd_only` writes e into zbar and skips the adjoint.
hipError_t launch_chain8(int64_t rows, int64_t cols, const float* z, const float* bias,
                         const float* x_skip, float* zbar, float* xbar, float* partials,
                         bool fwd_only, int* n_partials, hipStream_t s);
int chain8_partials(int64_t rows, int64_t cols);

// Sum `n` partials in a fixed order, multiply by `scale`, write *out. Writes
// flags[0] = (any bad label counted in `bad`, which may be null) and
// flags[1] = (loss not finite) on every call. With out == null only zeroes.
// Zeroes the `gaps` ranges of `zero_base` (may be null).
struct ZeroGaps {
  static constexpr int kMax = 64;
  int n;
  int64_t off[kMax];
  int32_t len[kMax];
};
hipError_t launch_finalize(const float* partials, const int32_t* bad, int n, float scale,
                           float* out, int32_t* flags, float* zero_base, const ZeroGaps& gaps,
                           hipStream_t s);

hipError_t launch_sgd(int dtype, int64_t n, void* params, float* master, const float* grads,
                      float lr, hipStream_t s);

// dz[r, c] (row stride ld, storage dtype) = seed[r, c] for c < classes, 0 for
// classes <= c < ld.
hipError_t launch_seed(int dtype, int64_t rows, int64_t classes, int64_t ld, const float* seed,
                       void* dz, hipStream_t s);

// Sum of the k-slices of a split NN (mode 0) or NT (mode 1) product in slice
// order, then its epilogue: mode 0 out = act(alpha * sum + bias[c]) (bias for
// c < nvec, operand dtype); mode 1 out = sum * act'(aux) + res, or
// (sum + res) * act'(aux) with res_pre (aux operand dtype; res, out output
// dtype). part[s * c_split + r * ld + c], out[r * ld + c], c < cols.
hipError_t launch_split_epilogue(int dtype, int out_dtype, int mode, int splits, int64_t rows,
                                 int64_t cols, int64_t ld, const float* part, int64_t c_split,
                                 int act, float alpha, const void* bias, int64_t nvec,
                                 const void* aux, const void* res, bool res_pre, void* out,
                                 hipStream_t s);

// A small float32 softmax network whose whole gradient runs in one workgroup
// (its input, weights and activations in LDS): see small_step.hip.
constexpr int kSmallMaxLayers = 8;
constexpr int kSmallThreads = 1024;
constexpr int kSmallMaxLds = 64 * 1024;                   // bytes of LDS for everything
constexpr int64_t kSmallMaxMacs = int64_t(1) << 21;       // forward + both adjoints
struct SmallNet {
  int L, B, maxw, wrt_x;
  int w[kSmallMaxLayers + 1];
  int act[kSmallMaxLayers];
  // LDS word offsets: the parameter block (params[pbase, pbase + pwords) as
  // it lies in memory, so W_l at woff[l] with row stride ldw[l] and b_l at
  // boff[l]), the layer outputs H_0 (= x) .. H_L, the adjoint ping-pong, the
  // per-row loss and label marks, the labels
  int woff[kSmallMaxLayers], boff[kSmallMaxLayers];
  int hoff[kSmallMaxLayers + 1];
  int g0, g1, rowloss, rowbad, labels;
  int64_t pbase;
  int pwords;
  int64_t offW[kSmallMaxLayers], offB[kSmallMaxLayers];  // in dparams
  int ldw[kSmallMaxLayers];
  float scale;  // 1 / B
};
// Fill t for a network; false if it does not fit one workgroup (layers,
// batch, LDS) or has too much work for one compute unit.
bool small_net(int L, const int32_t* widths, const int32_t* acts, const int64_t* offsets,
               const int64_t* ldw, int64_t B, bool wrt_x, SmallNet& t);
// The whole gradient (loss, dparams with zero padding, dx if t.wrt_x, flags).
hipError_t launch_small_step(const SmallNet& t, const float* params, const float* x,
                             const int32_t* labels, float* loss, float* dparams, float* dx,
                             int32_t* flags, const ZeroGaps& gaps, hipStream_t s);

// out[i] = g[i] * act'(h[i]) for i < n, act' from the saved output h = act(z)
// (storage dtype `dtype` for all three).
hipError_t launch_act_adjoint(int dtype, int act, int64_t n, const void* g, const void* h,
                              void* out, hipStream_t s);

// Sum of the k-slices of a split product in slice order: out[r, c] (row
// stride ld) = sum_s part[s * c_split + r * ld + c] for c < cols, and
// colsum[n] = sum_s cs_part[s * cs_split + n] for n < nvec (if colsum).
hipError_t launch_splitk_reduce(int splits, int64_t rows, int64_t cols, int64_t ld,
                                const float* part, int64_t c_split, float* out,
                                const float* cs_part, int64_t cs_split, float* colsum,
                                int64_t nvec, hipStream_t s);

}  // namespace dlvm
