// Fused element-wise kernels of the hot path (element-wise operator fusion,
// DLVM section 1): softmax cross-entropy with its adjoint, the eight-operator
// chain with its adjoint, the deterministic loss reduction, and SGD.
//
// Reductions are deterministic: every block writes one partial in a fixed
// order (butterfly within a wavefront, then wavefronts in index order), and a
// single-block kernel sums the partials in a fixed order. No floating-point
// atomics are used anywhere.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace dlvm {
namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Block sum in a fixed order; result valid in thread 0.
__device__ __forceinline__ float block_sum(float v, float* scratch) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float t = 0.0f;
  if (threadIdx.x == 0) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += scratch[w];
  }
  return t;
}

// ---------------------------------------------------------------------------
// Softmax cross-entropy, one wavefront per row. Softmax is composed of a
// max-shift, exp, reduce-add and log (section 3.1.1); the row maximum and
// the sum of exponentials are found in one pass with the usual rescaling of
// the running sum when the maximum grows. The gradient is scale*(p - onehot).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  const float a = (m == -INFINITY) ? 0.0f : s * __expf(m - M);
  const float b = (m2 == -INFINITY) ? 0.0f : s2 * __expf(m2 - M);
  m = M;
  s = a + b;
}

template <typename TD>
__global__ __launch_bounds__(kBlock) void dlvm_softmax_xent_kernel(
    int64_t rows, int64_t C, const float* __restrict__ Z, const int32_t* __restrict__ labels,
    float scale, TD* __restrict__ dZ, int64_t ld_dz, float* __restrict__ partials,
    int32_t* __restrict__ bad) {
  __shared__ float red[kWaves];
  __shared__ int32_t nbad[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kWaves + wave;
  float li = 0.0f;
  int32_t badrow = 0;
  if (row < rows) {
    const float* z = Z + row * C;
    float m = -INFINITY, s = 0.0f;
    for (int64_t j = lane; j < C; j += 64) lse_combine(m, s, z[j], 1.0f);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float m2 = __shfl_xor(m, o, 64);
      const float s2 = __shfl_xor(s, o, 64);
      lse_combine(m, s, m2, s2);
    }
    const float lse = m + __logf(s);
    const int32_t y = labels[row];
    const bool ok = y >= 0 && y < C;
    badrow = ok ? 0 : 1;
    li = ok ? lse - z[y] : NAN;
    TD* d = dZ + row * ld_dz;
    for (int64_t j = lane; j < C; j += 64) {
      const float pj = __expf(z[j] - lse);
      d[j] = store_cast<TD>(scale * (pj - (j == y ? 1.0f : 0.0f)));
    }
    for (int64_t j = C + lane; j < ld_dz; j += 64) d[j] = store_cast<TD>(0.0f);
  }
  if (lane == 0) {
    red[wave] = li;
    nbad[wave] = badrow;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    int32_t b = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      t += red[w];
      b += nbad[w];
    }
    partials[blockIdx.x] = t;
    bad[blockIdx.x] = b;
  }
}

// ---------------------------------------------------------------------------
// Eight-operator chain, forward and adjoint in one pass. With L the mean of
// e^2 over rows*cols elements the seed of e is known before the reduction,
// so the adjoint needs nothing from the forward reduction:
//   zb = z + b, a = tanh zb, c = a/2, d = c + 1, s = sigmoid d, e = s x, f = e e
//   ebar = 2 e / (rows cols), xbar = ebar s, zbar = ebar x s (1 - s) (1/2) (1 - a^2)
// ---------------------------------------------------------------------------
constexpr int kChainBlocks = 2048;

__device__ __forceinline__ float chain_elem(float z, float b, float x, float inv_n, bool fwd_only,
                                            float& zbar, float& xbar, float& e_out) {
  const float a = tanhf(z + b);
  const float d = 0.5f * a + 1.0f;
  const float s = sigmoidf_(d);
  const float e = s * x;
  e_out = e;
  if (!fwd_only) {
    const float eb = 2.0f * e * inv_n;
    xbar = eb * s;
    zbar = eb * x * (s * (1.0f - s)) * 0.5f * (1.0f - a * a);
  }
  return e * e;
}

template <bool VEC, bool FWD_ONLY>
__global__ __launch_bounds__(kBlock) void dlvm_chain8_kernel(
    int64_t rows, int64_t cols, const float* __restrict__ z, const float* __restrict__ bias,
    const float* __restrict__ xs, float* __restrict__ zbar, float* __restrict__ xbar,
    float* __restrict__ partials, float inv_n) {
  __shared__ float red[kWaves];
  float acc = 0.0f;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  if constexpr (VEC) {
    const int64_t n4 = rows * cols / 4;
    const int64_t c4 = cols / 4;
    const float4* z4 = reinterpret_cast<const float4*>(z);
    const float4* x4 = reinterpret_cast<const float4*>(xs);
    const float4* b4 = reinterpret_cast<const float4*>(bias);
    float4* zb4 = reinterpret_cast<float4*>(zbar);
    float4* xb4 = reinterpret_cast<float4*>(xbar);
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n4; i += stride) {
      const float4 zv = z4[i], xv = x4[i], bv = b4[i % c4];
      float4 zo, xo, eo;
      acc += chain_elem(zv.x, bv.x, xv.x, inv_n, FWD_ONLY, zo.x, xo.x, eo.x);
      acc += chain_elem(zv.y, bv.y, xv.y, inv_n, FWD_ONLY, zo.y, xo.y, eo.y);
      acc += chain_elem(zv.z, bv.z, xv.z, inv_n, FWD_ONLY, zo.z, xo.z, eo.z);
      acc += chain_elem(zv.w, bv.w, xv.w, inv_n, FWD_ONLY, zo.w, xo.w, eo.w);
      if constexpr (FWD_ONLY) {
        zb4[i] = eo;
      } else {
        zb4[i] = zo;
        xb4[i] = xo;
      }
    }
  } else {
    const int64_t n = rows * cols;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride) {
      float zo = 0.0f, xo = 0.0f, eo = 0.0f;
      acc += chain_elem(z[i], bias[i % cols], xs[i], inv_n, FWD_ONLY, zo, xo, eo);
      if constexpr (FWD_ONLY) {
        zbar[i] = eo;
      } else {
        zbar[i] = zo;
        xbar[i] = xo;
      }
    }
  }
  const float t = block_sum(acc, red);
  if (threadIdx.x == 0) partials[blockIdx.x] = t;
}

// ---------------------------------------------------------------------------
// Loss finalisation: fixed-order sum of the partials, times the seed scale.
// Also zeroes the padding gaps of the flat gradient buffer.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void dlvm_finalize_kernel(const float* __restrict__ partials,
                                                               const int32_t* __restrict__ bad,
                                                               int n, float scale,
                                                               float* __restrict__ out,
                                                               int32_t* __restrict__ flags,
                                                               float* __restrict__ zero_base,
                                                               ZeroGaps gaps) {
  __shared__ float red[kWaves];
  __shared__ float redb[kWaves];
  float v = 0.0f, nb = 0.0f;
  for (int i = threadIdx.x; i < n; i += kBlock) {
    v += partials[i];
    if (bad != nullptr) nb += static_cast<float>(bad[i]);
  }
  const float t = block_sum(v, red);
  const float tb = block_sum(nb, redb);
  if (threadIdx.x == 0) {
    const float loss = t * scale;
    out[0] = loss;
    if (flags != nullptr) {
      flags[0] = tb > 0.0f ? 1 : 0;
      flags[1] = isfinite(loss) ? 0 : 1;
    }
  }
  if (zero_base != nullptr) {
    for (int g = 0; g < gaps.n; ++g)
      for (int i = threadIdx.x; i < gaps.len[g]; i += kBlock) zero_base[gaps.off[g] + i] = 0.0f;
  }
}

// ---------------------------------------------------------------------------
// SGD over a flat buffer: w <- w - lr * g (fused multiply-add, one rounding).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void dlvm_sgd_f32_kernel(int64_t n, float* __restrict__ w,
                                                              const float* __restrict__ g,
                                                              float lr) {
  const int64_t n4 = n / 4;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  float4* w4 = reinterpret_cast<float4*>(w);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n4; i += stride) {
    float4 a = w4[i];
    const float4 b = g4[i];
    a.x = fmaf(-lr, b.x, a.x);
    a.y = fmaf(-lr, b.y, a.y);
    a.z = fmaf(-lr, b.z, a.z);
    a.w = fmaf(-lr, b.w, a.w);
    w4[i] = a;
  }
  for (int64_t i = n4 * 4 + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += stride)
    w[i] = fmaf(-lr, g[i], w[i]);
}

__global__ __launch_bounds__(kBlock) void dlvm_sgd_bf16_kernel(int64_t n, bf16_t* __restrict__ w,
                                                               float* __restrict__ master,
                                                               const float* __restrict__ g,
                                                               float lr) {
  const int64_t n4 = n / 4;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  float4* m4 = reinterpret_cast<float4*>(master);
  const float4* g4 = reinterpret_cast<const float4*>(g);
  uint2* w4 = reinterpret_cast<uint2*>(w);
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n4; i += stride) {
    float4 a = m4[i];
    const float4 b = g4[i];
    a.x = fmaf(-lr, b.x, a.x);
    a.y = fmaf(-lr, b.y, a.y);
    a.z = fmaf(-lr, b.z, a.z);
    a.w = fmaf(-lr, b.w, a.w);
    m4[i] = a;
    uint2 o;
    o.x = static_cast<uint32_t>(f32_to_bf16(a.x)) | (static_cast<uint32_t>(f32_to_bf16(a.y)) << 16);
    o.y = static_cast<uint32_t>(f32_to_bf16(a.z)) | (static_cast<uint32_t>(f32_to_bf16(a.w)) << 16);
    w4[i] = o;
  }
  for (int64_t i = n4 * 4 + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += stride) {
    const float a = fmaf(-lr, g[i], master[i]);
    master[i] = a;
    w[i] = f32_to_bf16(a);
  }
}

unsigned grid_for(int64_t work_items, int64_t cap) {
  int64_t b = (work_items + kBlock - 1) / kBlock;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<unsigned>(b);
}

}  // namespace

int softmax_xent_partials(int64_t rows) { return static_cast<int>((rows + kWaves - 1) / kWaves); }

hipError_t launch_softmax_xent(int dtype, int64_t rows, int64_t classes, const float* logits,
                               const int32_t* labels, float scale, void* dlogits,
                               int64_t ld_dlogits, float* partials, int32_t* bad, int* n_partials,
                               hipStream_t s) {
  const int nb = softmax_xent_partials(rows);
  *n_partials = nb;
  if (dtype == F32)
    launch_kernel(dlvm_softmax_xent_kernel<float>, dim3(nb), dim3(kBlock), s, rows,
                       classes, logits, labels, scale, static_cast<float*>(dlogits), ld_dlogits,
                       partials, bad);
  else
    launch_kernel(dlvm_softmax_xent_kernel<bf16_t>, dim3(nb), dim3(kBlock), s, rows,
                       classes, logits, labels, scale, static_cast<bf16_t*>(dlogits), ld_dlogits,
                       partials, bad);
  return hipGetLastError();
}

int chain8_partials(int64_t rows, int64_t cols) {
  const bool vec = cols % 4 == 0;
  const int64_t items = vec ? rows * cols / 4 : rows * cols;
  return static_cast<int>(grid_for(items, kChainBlocks));
}

hipError_t launch_chain8(int64_t rows, int64_t cols, const float* z, const float* bias,
                         const float* x_skip, float* zbar, float* xbar, float* partials,
                         bool fwd_only, int* n_partials, hipStream_t s) {
  const bool vec = cols % 4 == 0 && ((reinterpret_cast<uintptr_t>(z) | reinterpret_cast<uintptr_t>(bias) |
                                      reinterpret_cast<uintptr_t>(x_skip) |
                                      reinterpret_cast<uintptr_t>(zbar) |
                                      reinterpret_cast<uintptr_t>(xbar)) & 15u) == 0;
  const int nb = chain8_partials(rows, cols);
  *n_partials = nb;
  const float inv_n = static_cast<float>(1.0 / (static_cast<double>(rows) * static_cast<double>(cols)));
  if (vec) {
    if (fwd_only)
      launch_kernel((dlvm_chain8_kernel<true, true>), dim3(nb), dim3(kBlock), s, rows, cols,
                         z, bias, x_skip, zbar, xbar, partials, inv_n);
    else
      launch_kernel((dlvm_chain8_kernel<true, false>), dim3(nb), dim3(kBlock), s, rows,
                         cols, z, bias, x_skip, zbar, xbar, partials, inv_n);
  } else {
    if (fwd_only)
      launch_kernel((dlvm_chain8_kernel<false, true>), dim3(nb), dim3(kBlock), s, rows,
                         cols, z, bias, x_skip, zbar, xbar, partials, inv_n);
    else
      launch_kernel((dlvm_chain8_kernel<false, false>), dim3(nb), dim3(kBlock), s, rows,
                         cols, z, bias, x_skip, zbar, xbar, partials, inv_n);
  }
  return hipGetLastError();
}

hipError_t launch_finalize(const float* partials, const int32_t* bad, int n, float scale,
                           float* out, int32_t* flags, float* zero_base, const ZeroGaps& gaps,
                           hipStream_t s) {
  launch_kernel(dlvm_finalize_kernel, dim3(1), dim3(kBlock), s, partials, bad, n, scale,
                     out, flags, zero_base, gaps);
  return hipGetLastError();
}

hipError_t launch_sgd(int dtype, int64_t n, void* params, float* master, const float* grads,
                      float lr, hipStream_t s) {
  const unsigned nb = grid_for((n + 3) / 4, 4096);
  if (dtype == F32)
    launch_kernel(dlvm_sgd_f32_kernel, dim3(nb), dim3(kBlock), s, n,
                       static_cast<float*>(params), grads, lr);
  else
    launch_kernel(dlvm_sgd_bf16_kernel, dim3(nb), dim3(kBlock), s, n,
                       static_cast<bf16_t*>(params), master, grads, lr);
  return hipGetLastError();
}

}  // namespace dlvm
