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

// Softmax cross-entropy of logits that arrive as the k-slices of a split
// product (summed in slice order, plus the bias): one wavefront per row, each
// lane holding up to SPL logits of its row in registers.
template <typename TB>
__device__ __forceinline__ float bias_at(const TB* b, int64_t j);
template <>
__device__ __forceinline__ float bias_at<float>(const float* b, int64_t j) { return b[j]; }
template <>
__device__ __forceinline__ float bias_at<bf16_t>(const bf16_t* b, int64_t j) {
  return bf16_to_f32(b[j]);
}

template <typename TD, typename TB, int SPL>
__global__ __launch_bounds__(kBlock) void dlvm_split_softmax_xent_kernel(
    int S, int64_t rows, int64_t C, const float* __restrict__ part, int64_t c_split, int64_t ldp,
    const TB* __restrict__ bias, const int32_t* __restrict__ labels, float scale,
    TD* __restrict__ dZ, int64_t ld_dz, float* __restrict__ partials, int32_t* __restrict__ bad) {
  __shared__ float red[kWaves];
  __shared__ int32_t nbad[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = static_cast<int64_t>(blockIdx.x) * kWaves + wave;
  float li = 0.0f;
  int32_t badrow = 0;
  if (row < rows) {
    const int32_t y = labels[row];
    float z[SPL];
    float m = -INFINITY, zy = 0.0f;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
      const int64_t j = lane + 64 * c;
      z[c] = -INFINITY;
      if (j < C) {
        float v = part[row * ldp + j];
        for (int q = 1; q < S; ++q) v += part[q * c_split + row * ldp + j];
        v += bias != nullptr ? bias_at<TB>(bias, j) : 0.0f;
        z[c] = v;
        zy = j == y ? v : zy;
      }
      m = fmaxf(m, z[c]);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      m = fmaxf(m, __shfl_xor(m, o, 64));
      zy += __shfl_xor(zy, o, 64);  // one nonzero term: exact
    }
    float sum = 0.0f;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
      z[c] = lane + 64 * c < C ? __expf(z[c] - m) : 0.0f;
      sum += z[c];
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    const bool ok = y >= 0 && y < C;
    badrow = ok ? 0 : 1;
    li = ok ? (m + __logf(sum)) - zy : NAN;
    const float ps = scale / sum;
    TD* d = dZ + row * ld_dz;
#pragma unroll
    for (int c = 0; c < SPL; ++c) {
      const int64_t j = lane + 64 * c;
      if (j < C) d[j] = store_cast<TD>(ps * z[c] - (j == y ? scale : 0.0f));
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

// Rows whose logits and dlogits move as 16-byte float32 chunks (classes and
// the dlogits row stride multiples of 4, aligned bases) and fit in registers:
// lane l of the row's wavefront holds chunks l, l + 64, ... (NCH of them), so
// each logit is read from memory once and exponentiated once. The maximum and
// the sum of exponentials are wavefront butterflies (fixed order).
template <typename TD>
__device__ __forceinline__ void store4(TD* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
template <>
__device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float a, float b, float c, float d) {
  uint2 o;
  o.x = static_cast<uint32_t>(f32_to_bf16(a)) | (static_cast<uint32_t>(f32_to_bf16(b)) << 16);
  o.y = static_cast<uint32_t>(f32_to_bf16(c)) | (static_cast<uint32_t>(f32_to_bf16(d)) << 16);
  store_nt(reinterpret_cast<uint2*>(p), o);
}

template <typename TD, int NCH, int NR>
__global__ __launch_bounds__(kBlock) void dlvm_softmax_xent_rows_kernel(
    int64_t rows, int64_t C, const float* __restrict__ Z, const int32_t* __restrict__ labels,
    float scale, TD* __restrict__ dZ, int64_t ld_dz, float* __restrict__ partials,
    int32_t* __restrict__ bad) {
  // Each wavefront takes NR rows, all of whose loads are issued before the
  // first reduction (more bytes in flight per wavefront, fewer wavefronts).
  __shared__ float red[kWaves];
  __shared__ int32_t nbad[kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * kWaves + wave) * NR;
  const int64_t C4 = C / 4;
  float li = 0.0f;
  int32_t badrow = 0;
  float4 v[NR][NCH];
  int32_t y[NR];
#pragma unroll
  for (int q = 0; q < NR; ++q) {
    const int64_t row = row0 + q;
    y[q] = row < rows ? labels[row] : 0;
    const float4* __restrict__ z4 = reinterpret_cast<const float4*>(Z + row * C);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int64_t j = lane + 64 * c;
      v[q][c] = (row < rows && j < C4)
                    ? z4[j]
                    : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
  }
#pragma unroll
  for (int q = 0; q < NR; ++q) {
    const int64_t row = row0 + q;
    if (row >= rows) continue;  // uniform across the wavefront
    float m = -INFINITY;
    float zy = 0.0f;  // the label's logit, held by exactly one lane
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const float4 t = v[q][c];
      m = fmaxf(m, fmaxf(fmaxf(t.x, t.y), fmaxf(t.z, t.w)));
      const int64_t k = 4 * (lane + 64 * c);
      zy = k == y[q] ? t.x : k + 1 == y[q] ? t.y : k + 2 == y[q] ? t.z : k + 3 == y[q] ? t.w : zy;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      m = fmaxf(m, __shfl_xor(m, o, 64));
      zy += __shfl_xor(zy, o, 64);  // one nonzero term: exact
    }
    float sum = 0.0f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      v[q][c].x = __expf(v[q][c].x - m);
      v[q][c].y = __expf(v[q][c].y - m);
      v[q][c].z = __expf(v[q][c].z - m);
      v[q][c].w = __expf(v[q][c].w - m);
      sum += (v[q][c].x + v[q][c].y) + (v[q][c].z + v[q][c].w);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o, 64);
    const bool ok = y[q] >= 0 && y[q] < C;
    badrow += ok ? 0 : 1;
    li += ok ? (m + __logf(sum)) - zy : NAN;
    const float ps = scale / sum;
    TD* d = dZ + row * ld_dz;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int64_t j = lane + 64 * c;
      if (j < C4) {
        const int64_t k = 4 * j;
        store4<TD>(d + k, ps * v[q][c].x - (k == y[q] ? scale : 0.0f),
                   ps * v[q][c].y - (k + 1 == y[q] ? scale : 0.0f),
                   ps * v[q][c].z - (k + 2 == y[q] ? scale : 0.0f),
                   ps * v[q][c].w - (k + 3 == y[q] ? scale : 0.0f));
      }
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
constexpr int kChainUnroll = 4;

template <bool VEC, bool FWD_ONLY>
__global__ __launch_bounds__(kBlock) void dlvm_chain8_kernel(
    int64_t rows, int64_t cols, const float* __restrict__ z, const float* __restrict__ bias,
    const float* __restrict__ xs, float* __restrict__ zbar, float* __restrict__ xbar,
    float* __restrict__ partials, float inv_n) {
  __shared__ float red[kWaves];
  float acc = 0.0f;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  if constexpr (VEC) {
    // kChainUnroll 16-byte chunks of each operand per thread and iteration,
    // loads first; z and x_skip are read once (nontemporal).
    const int64_t n4 = rows * cols / 4;
    const int64_t c4 = cols / 4;
    const float4* z4 = reinterpret_cast<const float4*>(z);
    const float4* x4 = reinterpret_cast<const float4*>(xs);
    const float4* b4 = reinterpret_cast<const float4*>(bias);
    float4* zb4 = reinterpret_cast<float4*>(zbar);
    float4* xb4 = reinterpret_cast<float4*>(xbar);
    constexpr int64_t kStep = int64_t(kBlock) * kChainUnroll;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * kStep + threadIdx.x; base < n4;
         base += static_cast<int64_t>(gridDim.x) * kStep) {
      float4 zv[kChainUnroll], xv[kChainUnroll];
#pragma unroll
      for (int u = 0; u < kChainUnroll; ++u) {
        const int64_t i = base + u * kBlock;
        if (i < n4) {
          zv[u] = load_nt(z4 + i);
          xv[u] = load_nt(x4 + i);
        }
      }
#pragma unroll
      for (int u = 0; u < kChainUnroll; ++u) {
        const int64_t i = base + u * kBlock;
        if (i < n4) {
          const float4 bv = b4[i % c4];
          float4 zo, xo, eo;
          acc += chain_elem(zv[u].x, bv.x, xv[u].x, inv_n, FWD_ONLY, zo.x, xo.x, eo.x);
          acc += chain_elem(zv[u].y, bv.y, xv[u].y, inv_n, FWD_ONLY, zo.y, xo.y, eo.y);
          acc += chain_elem(zv[u].z, bv.z, xv[u].z, inv_n, FWD_ONLY, zo.z, xo.z, eo.z);
          acc += chain_elem(zv[u].w, bv.w, xv[u].w, inv_n, FWD_ONLY, zo.w, xo.w, eo.w);
          if constexpr (FWD_ONLY) {
            zb4[i] = eo;
          } else {
            zb4[i] = zo;
            xb4[i] = xo;
          }
        }
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
// Loss finalisation: fixed-order sum of the partials, times the seed scale
// (skipped when out is null). Also zeroes the padding gaps of the flat
// gradient buffer.
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
  if (threadIdx.x == 0 && out != nullptr) {
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
// The seed of a seedable gradient (the adjoint of the output layer's output),
// float32 [rows, C], stored as the layer's adjoint: storage dtype, row stride
// ld >= C, columns [C, ld) zero.
// ---------------------------------------------------------------------------
template <typename TD>
__global__ __launch_bounds__(kBlock) void dlvm_seed_kernel(int64_t rows, int64_t C, int64_t ld,
                                                           const float* __restrict__ seed,
                                                           TD* __restrict__ dz) {
  const int64_t n = rows * ld;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const int64_t r = i / ld, c = i - r * ld;
    dz[i] = store_cast<TD>(c < C ? seed[r * C + c] : 0.0f);
  }
}

// ---------------------------------------------------------------------------
// The k-slices of a split forward or input-adjoint product summed in slice
// order (fixed order: the same result on every run), then the epilogue the
// unsplit product applies in its last k-tile:
//   mode 0 (forward):        out = act(alpha * sum + bias[c])      (bias for c < nvec)
//   mode 1 (input adjoint):  out = sum * act'(aux) + R, or (sum + R) * act'(aux) with res_pre
// aux and bias in the operand dtype TA, R and out in the output dtype TO.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void load4f(const T* p, float (&v)[4]);
template <>
__device__ __forceinline__ void load4f<float>(const float* p, float (&v)[4]) {
  const float4 x = *reinterpret_cast<const float4*>(p);
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}
template <>
__device__ __forceinline__ void load4f<bf16_t>(const bf16_t* p, float (&v)[4]) {
  const uint2 x = *reinterpret_cast<const uint2*>(p);
  v[0] = __uint_as_float(x.x << 16); v[1] = __uint_as_float(x.x & 0xffff0000u);
  v[2] = __uint_as_float(x.y << 16); v[3] = __uint_as_float(x.y & 0xffff0000u);
}

__device__ __forceinline__ float split_epi(int mode, int act, float alpha, float v, float b,
                                           float g, float r, int res_pre) {
  if (mode == 0) return apply_act(act, alpha * v + b);
  if (res_pre) v += r;
  if (act != ACT_NONE) v *= act_grad_from_output(act, g);
  if (!res_pre) v += r;
  return v;
}

template <typename TA, typename TO, bool VEC>
__global__ __launch_bounds__(kBlock) void dlvm_split_epilogue_kernel(
    int S, int64_t rows, int64_t cols, int64_t ld, const float* __restrict__ part,
    int64_t c_split, int mode, int act, float alpha, const TA* __restrict__ bias, int64_t nvec,
    const TA* __restrict__ aux, const TO* __restrict__ res, int res_pre, TO* __restrict__ out) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const bool use_aux = mode == 1 && act != ACT_NONE && aux != nullptr;
  const bool use_res = mode == 1 && res != nullptr;
  if constexpr (VEC) {
    const int64_t c4 = cols / 4;
    for (int64_t i = t0; i < rows * c4; i += stride) {
      const int64_t r = i / c4, c = (i - r * c4) * 4;
      const int64_t o = r * ld + c;
      float4 acc = load_nt(reinterpret_cast<const float4*>(part + o));
      int q = 1;
      for (; q + 3 < S; q += 4) {  // four slices in flight, added in slice order
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          v[u] = load_nt(reinterpret_cast<const float4*>(part + (q + u) * c_split + o));
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w;
        }
      }
      for (; q < S; ++q) {
        const float4 v = load_nt(reinterpret_cast<const float4*>(part + q * c_split + o));
        acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
      }
      float b[4] = {0.0f, 0.0f, 0.0f, 0.0f}, g[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      float rv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if (mode == 0 && bias != nullptr) {
        if (c + 4 <= nvec) {
          load4f<TA>(bias + c, b);
        } else {
          for (int e = 0; e < 4; ++e) b[e] = c + e < nvec ? load_as_f32<TA>(bias + c + e) : 0.0f;
        }
      }
      if (use_aux) load4f<TA>(aux + o, g);
      if (use_res) load4f<TO>(res + o, rv);
      const float a[4] = {acc.x, acc.y, acc.z, acc.w};
      float y[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = split_epi(mode, act, alpha, a[e], b[e], g[e], rv[e], res_pre);
      store4<TO>(out + o, y[0], y[1], y[2], y[3]);
    }
  } else {
    for (int64_t i = t0; i < rows * cols; i += stride) {
      const int64_t r = i / cols, c = i - r * cols;
      const int64_t o = r * ld + c;
      float acc = part[o];
      for (int q = 1; q < S; ++q) acc += part[q * c_split + o];
      const float b = (mode == 0 && bias != nullptr && c < nvec) ? load_as_f32<TA>(bias + c) : 0.0f;
      const float g = use_aux ? load_as_f32<TA>(aux + o) : 0.0f;
      const float rv = use_res ? load_as_f32<TO>(res + o) : 0.0f;
      out[o] = store_cast<TO>(split_epi(mode, act, alpha, acc, b, g, rv, res_pre));
    }
  }
}

// ---------------------------------------------------------------------------
// Adjoint of an element-wise activation through its saved output:
// out = g * act'(h), act' taken from h = act(z) (storage dtype throughout).
// ---------------------------------------------------------------------------
template <typename TD>
__global__ __launch_bounds__(kBlock) void dlvm_act_adjoint_kernel(int64_t n, int act,
                                                                  const TD* __restrict__ g,
                                                                  const TD* __restrict__ h,
                                                                  TD* __restrict__ out) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    float v = load_as_f32<TD>(g + i);
    if (act != ACT_NONE) v *= act_grad_from_output(act, load_as_f32<TD>(h + i));
    out[i] = store_cast<TD>(v);
  }
}

// ---------------------------------------------------------------------------
// SGD over a flat buffer: w <- w - lr * g (fused multiply-add, one rounding).
// Each thread moves kSgdUnroll 16-byte chunks of every operand per iteration,
// all loads issued before the first store, so that enough bytes are in flight
// to keep HBM busy; the chunks of one wave instruction are contiguous. Every
// byte is touched once, so the accesses are nontemporal.
// ---------------------------------------------------------------------------
constexpr int kSgdUnroll = 4;
constexpr int64_t kSgdChunk = int64_t(kBlock) * kSgdUnroll;  // float4 per block iteration

__device__ __forceinline__ float4 sgd4(float4 w, float4 g, float lr) {
  w.x = fmaf(-lr, g.x, w.x);
  w.y = fmaf(-lr, g.y, w.y);
  w.z = fmaf(-lr, g.z, w.z);
  w.w = fmaf(-lr, g.w, w.w);
  return w;
}

__global__ __launch_bounds__(kBlock) void dlvm_sgd_f32_kernel(int64_t n, float* __restrict__ w,
                                                              const float* __restrict__ g,
                                                              float lr) {
  const int64_t n4 = n / 4;
  float4* __restrict__ w4 = reinterpret_cast<float4*>(w);
  const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
  for (int64_t base = static_cast<int64_t>(blockIdx.x) * kSgdChunk + threadIdx.x; base < n4;
       base += static_cast<int64_t>(gridDim.x) * kSgdChunk) {
    float4 a[kSgdUnroll], b[kSgdUnroll];
#pragma unroll
    for (int u = 0; u < kSgdUnroll; ++u) {
      const int64_t i = base + u * kBlock;
      if (i < n4) {
        a[u] = load_nt(w4 + i);
        b[u] = load_nt(g4 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kSgdUnroll; ++u) {
      const int64_t i = base + u * kBlock;
      if (i < n4) store_nt(w4 + i, sgd4(a[u], b[u], lr));
    }
  }
  for (int64_t i = n4 * 4 + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock)
    w[i] = fmaf(-lr, g[i], w[i]);
}

__global__ __launch_bounds__(kBlock) void dlvm_sgd_bf16_kernel(int64_t n, bf16_t* __restrict__ w,
                                                               float* __restrict__ master,
                                                               const float* __restrict__ g,
                                                               float lr) {
  const int64_t n4 = n / 4;
  float4* __restrict__ m4 = reinterpret_cast<float4*>(master);
  const float4* __restrict__ g4 = reinterpret_cast<const float4*>(g);
  bf16_t* __restrict__ wb = w;
  for (int64_t base = static_cast<int64_t>(blockIdx.x) * kSgdChunk + threadIdx.x; base < n4;
       base += static_cast<int64_t>(gridDim.x) * kSgdChunk) {
    float4 a[kSgdUnroll], b[kSgdUnroll];
#pragma unroll
    for (int u = 0; u < kSgdUnroll; ++u) {
      const int64_t i = base + u * kBlock;
      if (i < n4) {
        a[u] = load_nt(m4 + i);
        b[u] = load_nt(g4 + i);
      }
    }
#pragma unroll
    for (int u = 0; u < kSgdUnroll; ++u) {
      const int64_t i = base + u * kBlock;
      if (i < n4) {
        const float4 r = sgd4(a[u], b[u], lr);
        store_nt(m4 + i, r);
        uint2 o;
        o.x = static_cast<uint32_t>(f32_to_bf16(r.x)) | (static_cast<uint32_t>(f32_to_bf16(r.y)) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16(r.z)) | (static_cast<uint32_t>(f32_to_bf16(r.w)) << 16);
        store_nt(reinterpret_cast<uint2*>(wb + 4 * i), o);
      }
    }
  }
  for (int64_t i = n4 * 4 + static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kBlock) {
    const float a = fmaf(-lr, g[i], master[i]);
    master[i] = a;
    w[i] = f32_to_bf16(a);
  }
}

// ---------------------------------------------------------------------------
// Split reduction: the k-slices of a product summed in slice order (fixed
// order, so the result is the same on every run). The partials are read once.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void dlvm_splitk_reduce_kernel(
    int S, int64_t rows, int64_t cols, int64_t ld, const float* __restrict__ part,
    int64_t c_split, float* __restrict__ out, const float* __restrict__ cs_part,
    int64_t cs_split, float* __restrict__ colsum, int64_t nvec, bool vec) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (vec) {
    const int64_t c4 = cols / 4;
    const int64_t n4 = rows * c4;
    for (int64_t i = t0; i < n4; i += stride) {
      const int64_t r = i / c4, c = (i - r * c4) * 4;
      const int64_t o = r * ld + c;
      float4 acc = load_nt(reinterpret_cast<const float4*>(part + o));
      int q = 1;
      for (; q + 3 < S; q += 4) {  // four slices in flight, added in slice order
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          v[u] = load_nt(reinterpret_cast<const float4*>(part + (q + u) * c_split + o));
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          acc.x += v[u].x; acc.y += v[u].y; acc.z += v[u].z; acc.w += v[u].w;
        }
      }
      for (; q < S; ++q) {
        const float4 v = load_nt(reinterpret_cast<const float4*>(part + q * c_split + o));
        acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
      }
      *reinterpret_cast<float4*>(out + o) = acc;
    }
  } else {
    const int64_t n = rows * cols;
    for (int64_t i = t0; i < n; i += stride) {
      const int64_t r = i / cols, c = i - r * cols;
      const int64_t o = r * ld + c;
      float acc = part[o];
      int q = 1;
      for (; q + 3 < S; q += 4) {
        float v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = part[(q + u) * c_split + o];
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += v[u];
      }
      for (; q < S; ++q) acc += part[q * c_split + o];
      out[o] = acc;
    }
  }
  if (colsum != nullptr) {
    for (int64_t i = t0; i < nvec; i += stride) {
      float acc = cs_part[i];
      int q = 1;
      for (; q + 3 < S; q += 4) {
        float v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = cs_part[(q + u) * cs_split + i];
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += v[u];
      }
      for (; q < S; ++q) acc += cs_part[q * cs_split + i];
      colsum[i] = acc;
    }
  }
}

unsigned grid_for(int64_t work_items, int64_t cap) {
  int64_t b = (work_items + kBlock - 1) / kBlock;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<unsigned>(b);
}

// Rows per wavefront of the register-resident kernel (its grid has
// ceil(rows / (kWaves * NR)) blocks, each writing one loss partial). Measured
// on 16384 x 1000 float32 logits with bf16 adjoints: one row per wavefront
// 19.3 us from HBM (logits rotated over 786 MB) and 16.6 us resident in the
// Infinity Cache, against 21.7 and 18.9 with two rows and 22.4 and 19.2 with
// four; a copy of the same bytes in the same access pattern takes 19.1 and
// 15.5 us.
int softmax_rows_per_wave(int64_t chunks) { return chunks <= 2 ? 2 : 1; }

template <typename TD>
hipError_t launch_softmax_rows(int64_t chunks, int nb, int64_t rows, int64_t classes,
                               const float* logits, const int32_t* labels, float scale, TD* dlogits,
                               int64_t ld, float* partials, int32_t* bad, hipStream_t s) {
  const dim3 g(nb), b(kBlock);
  if (chunks <= 1)
    launch_kernel(dlvm_softmax_xent_rows_kernel<TD, 1, 2>, g, b, s, rows, classes, logits, labels,
                  scale, dlogits, ld, partials, bad);
  else if (chunks <= 2)
    launch_kernel(dlvm_softmax_xent_rows_kernel<TD, 2, 2>, g, b, s, rows, classes, logits, labels,
                  scale, dlogits, ld, partials, bad);
  else if (chunks <= 4)
    launch_kernel(dlvm_softmax_xent_rows_kernel<TD, 4, 1>, g, b, s, rows, classes, logits, labels,
                  scale, dlogits, ld, partials, bad);
  else if (chunks <= 8)
    launch_kernel(dlvm_softmax_xent_rows_kernel<TD, 8, 1>, g, b, s, rows, classes, logits, labels,
                  scale, dlogits, ld, partials, bad);
  else
    launch_kernel(dlvm_softmax_xent_rows_kernel<TD, 16, 1>, g, b, s, rows, classes, logits, labels,
                  scale, dlogits, ld, partials, bad);
  return hipGetLastError();
}

}  // namespace

int softmax_xent_partials(int64_t rows) { return static_cast<int>((rows + kWaves - 1) / kWaves); }

hipError_t launch_softmax_xent(int dtype, int64_t rows, int64_t classes, const float* logits,
                               const int32_t* labels, float scale, void* dlogits,
                               int64_t ld_dlogits, float* partials, int32_t* bad, int* n_partials,
                               hipStream_t s) {
  int nb = softmax_xent_partials(rows);
  const bool vec = classes % 4 == 0 && ld_dlogits % 4 == 0 &&
                   ((reinterpret_cast<uintptr_t>(logits) | reinterpret_cast<uintptr_t>(dlogits)) &
                    15u) == 0;
  const int64_t chunks = (classes / 4 + 63) / 64;  // 16-byte chunks per lane
  if (vec && chunks <= 16) {
    const int nr = softmax_rows_per_wave(chunks);
    nb = static_cast<int>((rows + kWaves * nr - 1) / (kWaves * nr));  // <= softmax_xent_partials
    *n_partials = nb;
    if (dtype == F32)
      return launch_softmax_rows<float>(chunks, nb, rows, classes, logits, labels, scale,
                                        static_cast<float*>(dlogits), ld_dlogits, partials, bad, s);
    return launch_softmax_rows<bf16_t>(chunks, nb, rows, classes, logits, labels, scale,
                                       static_cast<bf16_t*>(dlogits), ld_dlogits, partials, bad, s);
  }
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
  const int64_t items = vec ? (rows * cols / 4 + kChainUnroll - 1) / kChainUnroll : rows * cols;
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
  // one block per kSgdChunk float4 chunks, up to 32 blocks per compute unit
  // (measured on 138M bf16 parameters: 8192 blocks 326 us, 4096 blocks 334)
  int64_t nb64 = ((n / 4) + kSgdChunk - 1) / kSgdChunk;
  nb64 = nb64 < 1 ? 1 : (nb64 > 8192 ? 8192 : nb64);
  const unsigned nb = static_cast<unsigned>(nb64);
  if (dtype == F32)
    launch_kernel(dlvm_sgd_f32_kernel, dim3(nb), dim3(kBlock), s, n,
                       static_cast<float*>(params), grads, lr);
  else
    launch_kernel(dlvm_sgd_bf16_kernel, dim3(nb), dim3(kBlock), s, n,
                       static_cast<bf16_t*>(params), master, grads, lr);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(int splits, int64_t rows, int64_t cols, int64_t ld,
                                const float* part, int64_t c_split, float* out,
                                const float* cs_part, int64_t cs_split, float* colsum,
                                int64_t nvec, hipStream_t s) {
  const bool vec = cols % 4 == 0 && ld % 4 == 0 && c_split % 4 == 0 &&
                   ((reinterpret_cast<uintptr_t>(part) | reinterpret_cast<uintptr_t>(out)) & 15u) == 0;
  const unsigned nb = grid_for(vec ? rows * cols / 4 : rows * cols, 8192);
  launch_kernel(dlvm_splitk_reduce_kernel, dim3(nb), dim3(kBlock), s, splits, rows, cols, ld, part,
                c_split, out, cs_part, cs_split, colsum, nvec, vec);
  return hipGetLastError();
}

namespace {
template <typename TD, typename TB>
hipError_t launch_split_softmax_typed(int splits, int64_t rows, int64_t classes, const float* part,
                                      int64_t c_split, int64_t ldp, const TB* bias,
                                      const int32_t* labels, float scale, TD* dlogits, int64_t ld,
                                      float* partials, int32_t* bad, int nb, hipStream_t s) {
  const dim3 g(nb), b(kBlock);
  if (classes <= 64)
    launch_kernel(dlvm_split_softmax_xent_kernel<TD, TB, 1>, g, b, s, splits, rows, classes, part,
                  c_split, ldp, bias, labels, scale, dlogits, ld, partials, bad);
  else
    launch_kernel(dlvm_split_softmax_xent_kernel<TD, TB, 4>, g, b, s, splits, rows, classes, part,
                  c_split, ldp, bias, labels, scale, dlogits, ld, partials, bad);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_split_softmax_xent(int dtype, int splits, int64_t rows, int64_t classes,
                                     const float* part, int64_t c_split, int64_t ld_part,
                                     const void* bias, const int32_t* labels, float scale,
                                     void* dlogits, int64_t ld_dlogits, float* partials,
                                     int32_t* bad, int* n_partials, hipStream_t s) {
  if (classes > 256) return hipErrorInvalidValue;  // the callers split only narrow heads
  const int nb = softmax_xent_partials(rows);
  *n_partials = nb;
  if (dtype == F32)
    return launch_split_softmax_typed<float, float>(
        splits, rows, classes, part, c_split, ld_part, static_cast<const float*>(bias), labels,
        scale, static_cast<float*>(dlogits), ld_dlogits, partials, bad, nb, s);
  return launch_split_softmax_typed<bf16_t, bf16_t>(
      splits, rows, classes, part, c_split, ld_part, static_cast<const bf16_t*>(bias), labels,
      scale, static_cast<bf16_t*>(dlogits), ld_dlogits, partials, bad, nb, s);
}

namespace {
template <typename TA, typename TO>
hipError_t launch_split_epilogue_typed(int splits, int64_t rows, int64_t cols, int64_t ld,
                                       const float* part, int64_t c_split, int mode, int act,
                                       float alpha, const void* bias, int64_t nvec,
                                       const void* aux, const void* res, bool res_pre, void* out,
                                       hipStream_t s) {
  const bool vec = cols % 4 == 0 && ld % 4 == 0 && c_split % 4 == 0 &&
                   ((reinterpret_cast<uintptr_t>(part) | reinterpret_cast<uintptr_t>(out) |
                     reinterpret_cast<uintptr_t>(aux) | reinterpret_cast<uintptr_t>(res) |
                     reinterpret_cast<uintptr_t>(bias)) & 15u) == 0;
  const unsigned nb = grid_for(vec ? rows * cols / 4 : rows * cols, 8192);
  const TA* b = static_cast<const TA*>(bias);
  const TA* a = static_cast<const TA*>(aux);
  const TO* r = static_cast<const TO*>(res);
  TO* o = static_cast<TO*>(out);
  if (vec)
    launch_kernel(dlvm_split_epilogue_kernel<TA, TO, true>, dim3(nb), dim3(kBlock), s, splits, rows,
                  cols, ld, part, c_split, mode, act, alpha, b, nvec, a, r, res_pre ? 1 : 0, o);
  else
    launch_kernel(dlvm_split_epilogue_kernel<TA, TO, false>, dim3(nb), dim3(kBlock), s, splits,
                  rows, cols, ld, part, c_split, mode, act, alpha, b, nvec, a, r, res_pre ? 1 : 0, o);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_split_epilogue(int dtype, int out_dtype, int mode, int splits, int64_t rows,
                                 int64_t cols, int64_t ld, const float* part, int64_t c_split,
                                 int act, float alpha, const void* bias, int64_t nvec,
                                 const void* aux, const void* res, bool res_pre, void* out,
                                 hipStream_t s) {
  if (dtype == F32)
    return launch_split_epilogue_typed<float, float>(splits, rows, cols, ld, part, c_split, mode,
                                                     act, alpha, bias, nvec, aux, res, res_pre,
                                                     out, s);
  if (out_dtype == F32)
    return launch_split_epilogue_typed<bf16_t, float>(splits, rows, cols, ld, part, c_split, mode,
                                                      act, alpha, bias, nvec, aux, res, res_pre,
                                                      out, s);
  return launch_split_epilogue_typed<bf16_t, bf16_t>(splits, rows, cols, ld, part, c_split, mode,
                                                     act, alpha, bias, nvec, aux, res, res_pre,
                                                     out, s);
}

hipError_t launch_act_adjoint(int dtype, int act, int64_t n, const void* g, const void* h,
                              void* out, hipStream_t s) {
  const unsigned nb = grid_for(n, 4096);
  if (dtype == F32)
    launch_kernel(dlvm_act_adjoint_kernel<float>, dim3(nb), dim3(kBlock), s, n, act,
                  static_cast<const float*>(g), static_cast<const float*>(h),
                  static_cast<float*>(out));
  else
    launch_kernel(dlvm_act_adjoint_kernel<bf16_t>, dim3(nb), dim3(kBlock), s, n, act,
                  static_cast<const bf16_t*>(g), static_cast<const bf16_t*>(h),
                  static_cast<bf16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_seed(int dtype, int64_t rows, int64_t classes, int64_t ld, const float* seed,
                       void* dz, hipStream_t s) {
  const unsigned nb = grid_for(rows * ld, 4096);
  if (dtype == F32)
    launch_kernel(dlvm_seed_kernel<float>, dim3(nb), dim3(kBlock), s, rows, classes, ld, seed,
                  static_cast<float*>(dz));
  else
    launch_kernel(dlvm_seed_kernel<bf16_t>, dim3(nb), dim3(kBlock), s, rows, classes, ld, seed,
                  static_cast<bf16_t*>(dz));
  return hipGetLastError();
}

}  // namespace dlvm
