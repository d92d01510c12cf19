// Device helpers shared by the gfx950 kernels: storage types, bf16 rounding,
// activations and their derivatives from saved outputs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dlvm {

typedef uint16_t bf16_t;  // raw bfloat16 bits in memory
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

enum Dtype { F32 = 0, BF16 = 1 };
enum Act { ACT_NONE = 0, ACT_SIGMOID = 1, ACT_TANH = 2, ACT_RELU = 3 };

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float32 -> bfloat16, round to nearest, ties to even, by gfx950's conversion
// instruction (v_cvt_pk_bf16_f32; two values per instruction where the
// compiler pairs them). Compared on the device over all 2^32 float32 bit
// patterns with the integer rounding u + 0x7fff + ((u >> 16) & 1) >> 16: equal
// for every non-NaN input (denormals, infinities and signed zeros included);
// a NaN stays a NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

// Streaming 16-byte and 8-byte accesses that bypass cache retention
// (nontemporal): for data touched exactly once per pass.
typedef float f32v4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32v2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float4 load_nt(const float4* p) {
  const f32v4 v = __builtin_nontemporal_load(reinterpret_cast<const f32v4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void store_nt(float4* p, const float4& v) {
  f32v4 w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<f32v4*>(p));
}
__device__ __forceinline__ void store_nt(uint2* p, const uint2& v) {
  u32v2 w = {v.x, v.y};
  __builtin_nontemporal_store(w, reinterpret_cast<u32v2*>(p));
}

template <typename T> __device__ __forceinline__ float load_as_f32(const T* p);
template <> __device__ __forceinline__ float load_as_f32<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_as_f32<bf16_t>(const bf16_t* p) {
  return bf16_to_f32(*p);
}

template <typename T> __device__ __forceinline__ T store_cast(float v);
template <> __device__ __forceinline__ float store_cast<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t store_cast<bf16_t>(float v) { return f32_to_bf16(v); }

// sigmoid(v) = 1 / (1 + exp(-v)); exp overflow gives exactly 0 for v -> -inf.
__device__ __forceinline__ float sigmoidf_(float v) { return 1.0f / (1.0f + __expf(-v)); }

__device__ __forceinline__ float apply_act(int act, float v) {
  switch (act) {
    case ACT_SIGMOID: return sigmoidf_(v);
    case ACT_TANH: return tanhf(v);
    case ACT_RELU: return v > 0.0f ? v : 0.0f;
    default: return v;
  }
}

// Derivative of the activation expressed through its saved output h
// (common subexpression reuse: no exp/tanh is recomputed in the adjoint).
__device__ __forceinline__ float act_grad_from_output(int act, float h) {
  switch (act) {
    case ACT_SIGMOID: return h * (1.0f - h);
    case ACT_TANH: return 1.0f - h * h;
    case ACT_RELU: return h > 0.0f ? 1.0f : 0.0f;
    default: return 1.0f;
  }
}

// One element of the eight-operator chain and its adjoint: a = tanh(z + b),
// s = sigmoid(0.5 a + 1), e = s x; returns e^2 (the loss term before the
// mean); with the seed 1 / n of the mean, zbar = dL/dz and xbar = dL/dx (the
// x_skip path), unless fwd_only.
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

}  // namespace dlvm
