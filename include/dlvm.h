/*
 * dlvm.h - C ABI of the MI355X (gfx950) hot path of a DLVM-compiled network:
 * a differentiable linear-algebra function (dense layers plus element-wise
 * chains) and its generated adjoint.
 *
 * Paper: R. Wei, L. Schwartz, V. Adve, "DLVM: A modern compiler infrastructure
 * for deep learning systems", arXiv 1711.03016.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Tensors are row-major and dense. A layer maps K inputs to N outputs on a
 *   batch of B rows: X is [B, K], W is [K, N], b is [N], H = act(X.W + b) is
 *   [B, N] (the orientation of Fig. 3: x <1 x 784>, w <784 x 10>).
 * - Every tensor argument is a DEVICE pointer owned by the caller; the
 *   library never allocates, frees or keeps tensor memory. Device pointers must
 *   be 16-byte aligned (else DLVM_ERR_MISALIGNED).
 * - "dtype" is the storage type: DLVM_F32 (float32 storage and arithmetic) or
 *   DLVM_BF16 (bfloat16 storage, float32 accumulation and epilogue arithmetic,
 *   round-to-nearest-even on every float32 -> bf16 store). Losses, logits,
 *   gradients of parameters and of x, and SGD master weights are float32.
 * - Every call is asynchronous on the given stream (a hipStream_t passed as
 *   void*; NULL is the default stream). Errors found on the host return at once
 *   and enqueue nothing. A launch failure returns DLVM_ERR_HIP. Device-side
 *   conditions (a label out of range, a non-finite loss) are latched in the
 *   workspace and reported by dlvm_check.
 * - No call allocates device memory or issues a memset, so the calls can be
 *   captured into a HIP graph (dlvm_step_graph_create does so for a whole
 *   training step).
 * - Results are deterministic: the same inputs give bitwise-identical outputs
 *   (fixed reduction orders, no floating-point atomics).
 * - No C++ exception crosses this interface. dlvm_last_error() returns a
 *   thread-local message describing the last failure on the calling thread.
 */
#ifndef DLVM_H
#define DLVM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dlvm_status;
enum {
  DLVM_OK = 0,
  DLVM_ERR_INVALID_ARG = -1,  /* null pointer, bad shape/dtype, batch > batch_max */
  DLVM_ERR_MISALIGNED = -2,   /* a device pointer is not 16-byte aligned */
  DLVM_ERR_WORKSPACE = -3,    /* workspace missing or smaller than required */
  DLVM_ERR_UNSUPPORTED = -4,  /* a combination this library does not implement */
  DLVM_ERR_HIP = -5,          /* a HIP launch or runtime call failed */
  DLVM_ERR_LABEL_RANGE = -6,  /* dlvm_check: a label was outside [0, classes) */
  DLVM_ERR_NONFINITE = -7     /* dlvm_check: the loss was NaN or infinite */
};

enum { DLVM_F32 = 0, DLVM_BF16 = 1 };
enum { DLVM_ACT_NONE = 0, DLVM_ACT_SIGMOID = 1, DLVM_ACT_TANH = 2, DLVM_ACT_RELU = 3 };
enum { DLVM_LOSS_SOFTMAX_CE = 0, DLVM_LOSS_CHAIN8 = 1 };

/* Static description of a network: the shape-specialised function of the
 * NNKit JIT (section 3.4) fixed once per handle. */
typedef struct dlvm_mlp_desc {
  int32_t n_layers;        /* L >= 1 */
  const int32_t* widths;   /* L + 1 host ints: widths[0] = K0 (input), widths[L] = classes */
  const int32_t* acts;     /* L host ints (DLVM_ACT_*); acts[L-1] must be DLVM_ACT_NONE */
  int32_t dtype;           /* DLVM_F32 or DLVM_BF16 */
  int32_t loss;            /* DLVM_LOSS_SOFTMAX_CE, or DLVM_LOSS_CHAIN8 (L == 1, widths[0] == widths[1]) */
  int32_t wrt_x;           /* 1: dlvm_gradient also returns dL/dx (required for CHAIN8) */
  int64_t batch_max;       /* largest batch any call will use */
  int32_t checkpoint_every; /* 0 or 1: keep every hidden layer output for the adjoint sweep;
                             * k in [2, n_layers]: keep only H_l with l % k == 0 and
                             * recompute the others, one segment at a time, during the
                             * sweep (checkpointing, section 3.1.3). Results are bitwise
                             * the same for every k; the workspace shrinks. */
  int32_t chain_in_epilogue; /* CHAIN8 only: 1 runs the eight-operator chain and its
                              * adjoint in the epilogue of the dense layer's product (z is
                              * never stored; zbar, xbar are bitwise those of the
                              * standalone chain kernel); 0 runs the standalone kernel. */
} dlvm_mlp_desc;

typedef struct dlvm_model dlvm_model;

/* ---------------------------------------------------------------------------
 * Model-level entry points
 * ------------------------------------------------------------------------- */

/* Create a handle for a network (host only; touches no device). The handle
 * owns the copied description and the launch plan, never tensor memory.
 * Softmax cross-entropy networks (section 3.1.1: softmax composed from
 * primitives): H_l = act_l(H_{l-1}.W_l + b_l), logits = H_L, loss = mean over
 * rows of logsumexp(logits_i) - logits_i[y_i]. CHAIN8 networks: one dense
 * layer z = x.W, then the element-wise chain e = sigmoid(0.5 tanh(z + b) + 1)
 * * x, loss = mean(e * e) (x_skip = x). */
dlvm_status dlvm_create(const dlvm_mlp_desc* desc, dlvm_model** out);
void dlvm_destroy(dlvm_model* m);

/* Number of elements of the flat parameter buffer (including padding). The
 * flat buffer holds W_1, b_1, ..., W_L, b_L, each starting on a 256-byte
 * boundary (linear-algebra fusion passes pre-concatenated parameters,
 * section 3.1.2). The same element layout is used for params (storage dtype),
 * master weights (float32) and dparams (float32). */
int64_t dlvm_param_count(const dlvm_model* m);

/* Element offsets of W_l and b_l: offsets[2l] = W_{l+1}, offsets[2l+1] = b_{l+1}
 * for l in [0, L), and the row stride of each W: element (k, n) of W_{l+1} is
 * at offsets[2l] + k * lds[l] + n. lds[l] is the layer width, except that the
 * class dimension of a softmax network's last layer is rounded up to a
 * multiple of 8 (16-byte rows, the padded tensors of section 3.1.2); its
 * padding columns must be zero in params (they stay zero under dlvm_sgd_step)
 * and are written as zero in dparams. `offsets` is a host array of 2L int64,
 * `lds` (may be NULL) of L int64. */
dlvm_status dlvm_param_layout(const dlvm_model* m, int64_t* offsets, int64_t* lds);

/* Bytes of workspace a forward or gradient call at `batch` rows needs
 * (0 if the batch is invalid). Holds saved activations, adjoints, loss
 * partials, the float32 partial products of a split batch reduction (an
 * adjoint product wrt the weights whose output has too few tiles to occupy
 * the device is computed in k-slices and summed in slice order), the device
 * error flags and, for a bf16 network whose rectified hidden outputs are
 * produced and consumed by products on the same 256 x 256 or 64 x 128 tile
 * configuration, one bit per
 * element of each such output: the rectifier's derivative (output > 0), which
 * the forward product writes and the adjoint product of the next layer reads
 * instead of the saved output (section 3.1.3; the results are the same;
 * the environment variable DLVM_RELU_MASK=0 turns the masks off). One
 * workspace must not be used by two calls that may run concurrently. */
size_t dlvm_workspace_bytes(const dlvm_model* m, int64_t batch);

/* Where a gradient call keeps the intermediate values of the adjoint code
 * (section 3.1.3: the gradient function recomputes the forward keeping the
 * layer outputs, then writes one adjoint per layer) inside a workspace for
 * `batch` rows, so that a caller can read them after the call has completed
 * (e.g. to check one layer at a time). Host only. On success *offset is the
 * byte offset from the workspace base, *ld the row stride in elements and
 * *dtype the element type (DLVM_F32 / DLVM_BF16) of a row-major
 * [batch, ...] tensor:
 *   DLVM_WS_HIDDEN,  layer l in [1, L-1]: H_l, the output of hidden layer l
 *     (widths[l] columns, ld = widths[l], storage dtype), the input of layer
 *     l + 1's products. With checkpoint_every k > 1, an H_l with l % k != 0
 *     shares a slot with other layers and holds whatever was computed there last.
 *   DLVM_WS_LOGITS (layer ignored): the output layer's product, float32
 *     [batch, widths[L]] (the logits; z = x.W for CHAIN8). DLVM_ERR_UNSUPPORTED
 *     when the plan never stores it: a softmax head whose product the loss
 *     kernel receives as k-slices, or a chain run in the product's epilogue.
 *   DLVM_WS_ADJOINT, layer l in [1, L]: dZ_l, the adjoint of layer l's output
 *     before its activation (l = L: the adjoint of the logits, (softmax(z) -
 *     onehot(y)) / batch for SOFTMAX_CE), ld = the row stride of W_l
 *     (dlvm_param_layout; the padding columns hold zero), storage dtype
 *     (float32 for CHAIN8).
 * DLVM_ERR_INVALID_ARG for an unknown kind, a layer out of range or an
 * invalid batch; DLVM_ERR_UNSUPPORTED for recurrent and matrix-chain handles
 * and for a network whose gradient runs as one workgroup (see dlvm_gradient:
 * that launch keeps every intermediate value in LDS). */
enum { DLVM_WS_HIDDEN = 0, DLVM_WS_LOGITS = 1, DLVM_WS_ADJOINT = 2 };
dlvm_status dlvm_workspace_tensor(const dlvm_model* m, int64_t batch, int32_t kind, int32_t layer,
                                  size_t* offset, int64_t* ld, int32_t* dtype);

/* The original function (Fig. 3's @foo): writes `out`, float32 [batch, widths[L]]:
 * the logits for SOFTMAX_CE, the chain value e for CHAIN8. Saves nothing (the
 * forward of a function that is not differentiated keeps no activations). */
dlvm_status dlvm_forward(const dlvm_model* m, const void* params, const void* x,
                         int64_t batch, float* out, void* ws, size_t ws_bytes,
                         void* stream);

/* The gradient function (section 3.1.3; gradient declaration "wrt params
 * [, x] keeping loss"): recomputes the forward from the original inputs,
 * then runs the adjoint. Writes loss (one float32 on the device), dparams
 * (float32, flat layout, padding set to zero) and, iff wrt_x, dx (float32
 * [batch, widths[0]]). `labels` are int32 [batch] in [0, classes) for
 * SOFTMAX_CE and NULL for CHAIN8. The input gradient of the first layer is
 * not computed unless wrt_x (dead code elimination, section 3.1.3).
 * A float32 SOFTMAX_CE network of at most 8 layers and 1024 rows whose
 * input, weights and layer outputs fit in 64 KB (and at most 2^21
 * multiply-adds a call) runs as one launch of one workgroup, which writes
 * only the error flags of the workspace; setting the environment variable DLVM_SMALL_STEP=0
 * selects the multi-launch plan for it as well. */
dlvm_status dlvm_gradient(const dlvm_model* m, const void* params, const void* x,
                          const int32_t* labels, int64_t batch, float* loss,
                          float* dparams, float* dx, void* ws, size_t ws_bytes,
                          void* stream);

/* The seedable gradient function (Fig. 3's "seedable" declaration,
 * [gradient @mlp wrt params (, x) seedable]) of a softmax network's logits,
 * without the loss: given `seed`, float32 [batch, classes] (the adjoint of the
 * logits, caller's device memory), writes dparams = seed-weighted gradient of
 * the logits wrt the parameters (float32, flat layout, padding set to zero)
 * and, iff wrt_x, dx (float32 [batch, widths[0]]). The hidden layers' forward
 * is recomputed; the output layer's own product is dead (its value is not
 * kept) and not computed. No loss, no device flags. DLVM_ERR_UNSUPPORTED for
 * CHAIN8 models. Workspace as for dlvm_gradient. */
dlvm_status dlvm_vjp(const dlvm_model* m, const void* params, const void* x, const float* seed,
                     int64_t batch, float* dparams, float* dx, void* ws, size_t ws_bytes,
                     void* stream);

/* Plain SGD over the whole flat buffer in one launch: params -= lr * dparams.
 * F32 models update params in place and take master == NULL. BF16 models
 * update the float32 `master` copy and write params = bf16(master). Dense and
 * recurrent handles; DLVM_ERR_UNSUPPORTED for a matrix chain. */
dlvm_status dlvm_sgd_step(const dlvm_model* m, void* params, float* master,
                          const float* dparams, float lr, void* stream);

/* ---------------------------------------------------------------------------
 * Recurrent network (section 3.1.2's RNN cell, linear-algebra fusion of a
 * polynomial of products)
 * ------------------------------------------------------------------------- */

/* The cell h_t = f(W x_{t-1} + U h_{t-1} + b) unrolled over `steps`, in
 * row-major batch form: hs[t+1] = act(xs[t].W + hs[t].U + b), t = 0..T-1.
 * Each step is ONE matrix product over the concatenated contraction
 * [xs[t] hs[t]].[W; U] with the bias add and activation fused (section
 * 3.1.2); the parameters are stored concatenated in the first place (the
 * interprocedural form of the fusion): the flat buffer (dlvm_param_count,
 * dlvm_param_layout with offsets[0] = [W; U], offsets[1] = b, lds[0] = hidden)
 * holds [W; U] as one [in_width + hidden, hidden] row-major matrix (W's rows
 * first) and b [hidden]. The operand [xs[t] hs[t]] is not materialised. */
typedef struct dlvm_rnn_desc {
  int32_t dtype;       /* DLVM_F32 or DLVM_BF16 (storage of xs, hs, params, dhs) */
  int32_t act;         /* DLVM_ACT_* of the cell */
  int64_t steps;       /* T in [1, 4096] */
  int64_t in_width;    /* Kx >= 1 */
  int64_t hidden;      /* H >= 1 */
  int64_t batch_max;   /* largest batch any call will use */
  int32_t wrt_x;       /* 1: dlvm_rnn_backward also returns dL/dxs */
  int32_t wrt_h0;      /* 1: dlvm_rnn_backward also returns dL/dh0 */
} dlvm_rnn_desc;

/* Create a recurrent model handle (host only). dlvm_destroy, dlvm_param_count,
 * dlvm_param_layout, dlvm_workspace_bytes, dlvm_sgd_step, dlvm_plan_size /
 * dlvm_plan_entry (a step is a forward call, a backward call and the update)
 * and the timing probe take it; dlvm_forward, dlvm_gradient, dlvm_vjp and
 * dlvm_step_graph_create return DLVM_ERR_UNSUPPORTED for it. */
dlvm_status dlvm_rnn_create(const dlvm_rnn_desc* desc, dlvm_model** out);

/* Forward over the T steps: xs [T, batch, Kx] and hs [T + 1, batch, H] in the
 * storage dtype, caller's device memory; the caller writes the initial state
 * into hs[0], the call writes hs[1..T] (one fused product per step). hs is
 * what dlvm_rnn_backward needs (the adjoint uses the saved outputs). `ws`
 * (dlvm_workspace_bytes, or NULL) holds the float32 k-slices of products the
 * planner splits over their contraction (summed in slice order, then bias
 * and activation applied); with NULL no product is split. The launch plan
 * (dlvm_plan_entry) describes calls given a workspace. */
dlvm_status dlvm_rnn_forward(const dlvm_model* m, const void* params, const void* xs,
                             int64_t batch, void* hs, void* ws, size_t ws_bytes, void* stream);

/* Seedable gradient of the T outputs (backpropagation through time, the
 * adjoint of the unrolled cell, section 3.1.3): dhs [T, batch, H] (storage
 * dtype) holds the adjoints of hs[1..T] (dhs[t] for hs[t+1]; zeros where a
 * step's output does not reach the loss); xs and hs as written by
 * dlvm_rnn_forward with the same params. Writes dparams (float32, flat
 * layout: d[W; U], db; padding zero), and iff wrt_x dxs (float32 [T, batch,
 * Kx]), iff wrt_h0 dh0 (float32 [batch, H]); neither is computed otherwise
 * (dead code elimination, section 3.1.4). The weight gradient over all steps
 * is one contraction over T * batch rows. `ws` needs dlvm_workspace_bytes. */
dlvm_status dlvm_rnn_backward(const dlvm_model* m, const void* params, const void* xs,
                              const void* hs, const void* dhs, int64_t batch, float* dparams,
                              float* dxs, float* dh0, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Matrix multiplication reordering (section 3.1.2)
 * ------------------------------------------------------------------------- */

/* The chain A_0 A_1 ... A_{n-1}, A_i of shape dims[i] x dims[i+1], can be
 * evaluated in any order (associativity); a p x q by q x r product costs
 * p q r multiply-adds. Computes the order of least total cost (over every
 * sub-chain, the best outermost cut given the best orders of both sides; the
 * smallest cut among equal costs) and returns that cost (saturated at
 * INT64_MAX), or -1 for invalid arguments (n outside [1, 32], a dimension
 * outside [1, 2^20]). If `split` is not NULL it receives the n x n row-major
 * table of cuts: split[i * n + j] = k means A_i..A_j is computed as
 * (A_i..A_k)(A_{k+1}..A_j); entries with i >= j are -1. Host only. */
int64_t dlvm_chain_order(int32_t n, const int64_t* dims, int32_t* split);

/* Workspace bytes dlvm_matrix_chain needs for this chain and order (split
 * NULL: the optimal order), 0 for invalid arguments. */
size_t dlvm_matrix_chain_ws_bytes(int32_t dtype, int32_t n, const int64_t* dims,
                                  const int32_t* split);

/* out (float32 [dims[0], dims[n]]) = A_0 ... A_{n-1}, evaluated in the order
 * of `split` (an n x n table as above, caller's host memory), or in the
 * optimal order when split is NULL. n in [2, 32]. `mats` is a host array of n
 * device pointers to row-major matrices of `dtype` (F32, or BF16 with float32
 * accumulate); intermediate products are kept in `ws` in `dtype` (bf16
 * intermediates are rounded to nearest even). One matrix-core product per
 * cut, in evaluation order on `stream`; a product with too few output tiles
 * for the device may be computed in k-slices (float32, in `ws`) summed in
 * slice order by one more launch. DLVM_ERR_INVALID_ARG for a split table
 * that is not an order of the chain. */
dlvm_status dlvm_matrix_chain(int32_t dtype, int32_t n, const int64_t* dims,
                              const void* const* mats, const int32_t* split, float* out,
                              void* ws, size_t ws_bytes, void* stream);

/* A chain of fixed shapes and order as a handle (order: split, or the
 * optimal one when NULL): dlvm_chain_run computes the same product as
 * dlvm_matrix_chain; dlvm_workspace_bytes (batch 1), dlvm_plan_size /
 * dlvm_plan_entry (batch 1: the chain's products and slice sums, then an
 * empty update entry), the timing probe and dlvm_destroy take the handle;
 * the network calls refuse it. */
dlvm_status dlvm_chain_create(int32_t dtype, int32_t n, const int64_t* dims, const int32_t* split,
                              dlvm_model** out);
dlvm_status dlvm_chain_run(const dlvm_model* m, const void* const* mats, float* out, void* ws,
                           size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * Captured training step (HIP graph)
 * ------------------------------------------------------------------------- */

/* A training step recorded once and replayed: the launches of one
 * dlvm_gradient call followed (if `update`) by those of one dlvm_sgd_step call
 * with learning rate `lr`, captured into a HIP graph with the given device
 * pointers baked in. Replaying it (dlvm_graph_launch) does exactly the work of
 * those two calls on the same buffers, with a smaller per-launch cost; the
 * caller refills x and labels in place between replays. Arguments and errors
 * as for dlvm_gradient and dlvm_sgd_step; the timing probe must be disarmed.
 * Capturing runs nothing on the device. The graph is owned by the caller
 * (dlvm_graph_destroy) and must not outlive the model or the buffers. */
typedef struct dlvm_graph dlvm_graph;
dlvm_status dlvm_step_graph_create(const dlvm_model* m, void* params, float* master,
                                   const void* x, const int32_t* labels, int64_t batch,
                                   float* loss, float* dparams, float* dx, void* ws,
                                   size_t ws_bytes, int32_t update, float lr, dlvm_graph** out);
/* Enqueue one replay of the captured step on `stream`. */
dlvm_status dlvm_graph_launch(dlvm_graph* g, void* stream);
void dlvm_graph_destroy(dlvm_graph* g);

/* Synchronise `stream` and read the device flags that the last gradient call
 * using `ws` wrote (every gradient call rewrites them): returns
 * DLVM_ERR_LABEL_RANGE if a label was outside [0, classes) (that row's loss
 * term is NaN), else DLVM_ERR_NONFINITE if the loss was NaN or infinite, else
 * DLVM_OK. The step-level loss calls write the same flags at the start of
 * their `ws`, so dlvm_check also reads those. DLVM_ERR_UNSUPPORTED for a
 * recurrent or matrix-chain handle (their calls write no flags). */
dlvm_status dlvm_check(const dlvm_model* m, void* ws, void* stream);

/* Message describing the last failure on this thread ("" if none). */
const char* dlvm_last_error(void);

/* ---------------------------------------------------------------------------
 * Launch plan and timing probe (instrumentation)
 * ------------------------------------------------------------------------- */

/* One kernel launch of a training step: a dlvm_gradient call followed by a
 * dlvm_sgd_step call. `flops` counts 2*M*N*K for a matrix product (else 0);
 * `bytes` is the algorithmic minimum of device-memory traffic: every operand
 * read once and every result written once. */
typedef struct dlvm_launch_info {
  char name[48];
  int64_t M, N, K;
  double flops;
  double bytes;
} dlvm_launch_info;

/* Number of launches in one step at `batch` rows (gradient launches, then
 * the one SGD launch), or 0 if the batch is invalid. */
int32_t dlvm_plan_size(const dlvm_model* m, int64_t batch);
/* Description of launch `index` (0-based, in enqueue order) of a step. */
dlvm_status dlvm_plan_entry(const dlvm_model* m, int64_t batch, int32_t index,
                            dlvm_launch_info* info);

/* Arm the probe: subsequent launches at position `index` of a step (-1: every
 * position) made by this handle's dlvm_gradient / dlvm_sgd_step calls are
 * bracketed by HIP events recorded on the call's stream, for the first
 * `capacity` such launches. Arming creates the events (a runtime call, done
 * before any timed region); recording them allocates nothing. Re-arming
 * discards earlier records. */
dlvm_status dlvm_probe_arm(dlvm_model* m, int32_t index, int32_t capacity);
/* Synchronise on the recorded events and return how many launches at position
 * `index` were recorded and their summed duration in milliseconds. */
dlvm_status dlvm_probe_read(dlvm_model* m, int32_t index, int64_t* count, double* total_ms);
/* Stop recording and release the events. */
dlvm_status dlvm_probe_disarm(dlvm_model* m);

/* ---------------------------------------------------------------------------
 * Step-level entry points: the individual steps the model-level calls are
 * made of, exported so each can be driven and checked on its own.
 * ------------------------------------------------------------------------- */

/* Dense layer forward with the bias add and activation fused into the matrix
 * product (linear-algebra fusion, section 3.1.2; element-wise operator
 * fusion, section 1): H[M,N] = act(alpha * X[M,K].W[K,N] + bias[N]).
 * X, W, bias (may be NULL) are `dtype`; H is `out_dtype` (F32, or BF16 when
 * dtype is BF16). */
dlvm_status dlvm_dense_forward(int32_t dtype, int32_t out_dtype, int32_t act,
                               int64_t M, int64_t N, int64_t K, float alpha,
                               const void* X, const void* W, const void* bias,
                               void* H, void* stream);

/* One recurrent cell as one fused product (section 3.1.2): Hout[M,N] =
 * act(X[M,Kx].WU[0:Kx,:] + H[M,Kh].WU[Kx:Kx+Kh,:] + bias[N]), i.e. the product
 * of the concatenation [X H] (read in place from the two buffers, never
 * copied) with WU [Kx + Kh, N]. All tensors contiguous row-major, `dtype`
 * (F32 or BF16) for inputs and output; bias may be NULL. */
dlvm_status dlvm_rnn_cell_forward(int32_t dtype, int32_t act, int64_t M, int64_t Kx,
                                  int64_t Kh, int64_t N, const void* X, const void* H,
                                  const void* WU, const void* bias, void* Hout, void* stream);

/* Adjoint of the dense layer with respect to its input (adjoint of dot:
 * dX = dY.W^T, transpose never materialised), fused with the adjoint of the
 * previous layer's activation taken from its saved output Hprev, plus an
 * optional second adjoint contribution R to the same value (a value used in
 * two places receives the sum of both adjoints):
 * dX[M,K] = (dY[M,N].W[K,N]^T) * act'(Hprev[M,K]) + R[M,K].
 * act' is s(1-s) for sigmoid, 1-t^2 for tanh, [h > 0] for relu, 1 for none
 * (Hprev may then be NULL). R (may be NULL) has dX's type. dY, W, Hprev are
 * `dtype`; dX is `out_dtype`. dX may alias R (in-place accumulate). */
dlvm_status dlvm_dense_backward_data(int32_t dtype, int32_t out_dtype,
                                     int32_t act_prev, int64_t M, int64_t N,
                                     int64_t K, const void* dY, const void* W,
                                     const void* Hprev, const void* R, void* dX,
                                     void* stream);

/* Adjoint of the dense layer with respect to its parameters: dW[K,N] =
 * X[M,K]^T.dY[M,N] and db[N] = sum over rows of dY (the padded product
 * [X 1]^T.dY = [dW; db] of section 3.1.2). X, dY are `dtype`; dW, db are
 * float32 (db may be NULL). */
dlvm_status dlvm_dense_backward_params(int32_t dtype, int64_t M, int64_t N,
                                       int64_t K, const void* X, const void* dY,
                                       float* dW, float* db, void* stream);

/* Softmax cross-entropy and its adjoint on float32 logits [rows, classes]
 * (softmax composed of exp, reduce-add, log; section 3.1.1):
 * loss = scale * sum_i (logsumexp(z_i) - z_i[y_i]),
 * dlogits = scale * (softmax(z) - onehot(y)), stored as `dtype`.
 * `ws` needs dlvm_softmax_xent_ws_bytes(rows) bytes; flags latch in it. */
size_t dlvm_softmax_xent_ws_bytes(int64_t rows);
dlvm_status dlvm_softmax_xent(int32_t dtype, int64_t rows, int64_t classes,
                              const float* logits, const int32_t* labels,
                              float scale, void* dlogits, float* loss, void* ws,
                              size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation as dlvm_softmax_xent, with the loss partials and bad-label
 * counts in a static device array of the library (2 MiB per GPU, held until
 * the process ends) instead of a caller workspace. The first call on a device
 * looks the array's address up (hipGetSymbolAddress); no call allocates or
 * frees memory. rows in [1, 1048576] (DLVM_ERR_INVALID_ARG beyond, before
 * anything is enqueued). `flags` (may be NULL) is an int32[2] device output:
 * flags[0] = 1 if a label was outside [0, classes) (the loss is then NaN),
 * flags[1] = 1 if the loss is not finite. loss and dlogits are bitwise those
 * of dlvm_softmax_xent. Every call on a GPU uses that GPU's one array: calls
 * that may run concurrently on one GPU (different streams or threads) race
 * and must not overlap. */
dlvm_status dlvm_softmax_xent_noalloc(int32_t dtype, int64_t rows, int64_t classes,
                                      const float* logits, const int32_t* labels, float scale,
                                      void* dlogits, float* loss, int32_t* flags, void* stream);

/* The eight-operator element-wise chain, forward and adjoint fused in one
 * pass over float32 [rows, cols] tensors: a = tanh(z + b), s = sigmoid(0.5a + 1),
 * e = s * x_skip, loss = mean(e^2) (x^2 simplified to x*x, section 3.1.2);
 * zbar = dL/dz, xbar = dL/dx_skip. `ws` needs dlvm_chain8_ws_bytes(rows, cols). */
size_t dlvm_chain8_ws_bytes(int64_t rows, int64_t cols);
dlvm_status dlvm_chain8(int64_t rows, int64_t cols, const float* z,
                        const float* bias, const float* x_skip, float* zbar,
                        float* xbar, float* loss, void* ws, size_t ws_bytes,
                        void* stream);

/* Fused SGD over n elements: F32: params -= lr * grads (master NULL).
 * BF16: master -= lr * grads, params = bf16(master). */
dlvm_status dlvm_sgd(int32_t dtype, int64_t n, void* params, float* master,
                     const float* grads, float lr, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DLVM_H */
