// Shared device/host helpers of the JAGG HIP library (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include <string>

namespace jg {

enum DType { F32 = 0, BF16 = 1 };

// ---------------------------------------------------------------- bf16 bits
// bf16 is carried as raw uint16_t; conversions are round-to-nearest-even with
// NaN kept quiet.
__device__ __host__ inline float bf2f(uint16_t v) {
  union { uint32_t u; float f; } c;
  c.u = (uint32_t)v << 16;
  return c.f;
}
// fp32 -> bf16, round to nearest even: the hardware conversion
// (v_cvt_pk_bf16_f32), branch-free; pairs of calls fuse into one instruction
__device__ inline uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __host__ inline float ld(const float* p, size_t i) { return p[i]; }
  static __device__ __host__ inline void st(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
  static __device__ __host__ inline float ld(const uint16_t* p, size_t i) { return bf2f(p[i]); }
  static __device__ __host__ inline void st(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }
};
template <typename T> __device__ inline float ldf(const T* p, size_t i) { return Elem<T>::ld(p, i); }
template <typename T> __device__ inline void stf(T* p, size_t i, float v) { Elem<T>::st(p, i, v); }

// dtype-erased load/store (used where a kernel's operand dtype is a runtime flag)
__device__ inline float ld_any(const void* p, int dt, size_t i) {
  return dt == BF16 ? bf2f(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}
__device__ inline void st_any(void* p, int dt, size_t i, float v) {
  if (dt == BF16) ((uint16_t*)p)[i] = f2bf(v); else ((float*)p)[i] = v;
}

inline size_t dsize(int dt) { return dt == BF16 ? 2 : 4; }

// ------------------------------------------------------------- wave helpers
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); `sh` holds >= 16 floats.
__device__ inline float block_sum(float v, float* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < nw; ++i) r += sh[i];
  return r;
}

// GELU, tanh form: u = c (x + a x^3), tanh(u) = 1 - 2r with
// r = 1 / (exp(2u) + 1) (one exp2 and one hardware reciprocal, v_rcp_f32, 1
// ulp; exact limits at +-inf: rcp(inf) = 0, rcp(1) = 1).  Then 1 + tanh = 2(1 - r)
// and 1 - tanh^2 = 4 r (1 - r), so
//   gelu(x)  = x (1 - r)
//   gelu'(x) = (1 - r) (1 + 2 x r u'(x)),  u'(x) = c (1 + 3 a x^2).
constexpr float GELU_C = 0.7978845608028654f, GELU_A = 0.044715f;
__device__ __forceinline__ float gelu_r(float x, float x2) {
  // 2u log2(e) = x (2c log2(e) + 2ca log2(e) x^2)
  const float kc = 2.f * GELU_C * 1.4426950408889634f, ka = kc * GELU_A;
  return __builtin_amdgcn_rcpf(__builtin_amdgcn_exp2f(x * fmaf(ka, x2, kc)) + 1.f);
}
__device__ __forceinline__ float gelu_tanh(float x) { return x * (1.f - gelu_r(x, x * x)); }
__device__ __forceinline__ float gelu_tanh_grad(float x) {
  const float x2 = x * x, r = gelu_r(x, x2);
  return (1.f - r) * fmaf(x * r, fmaf(6.f * GELU_A * GELU_C, x2, 2.f * GELU_C), 1.f);
}
__device__ inline float silu(float x) { return x / (1.f + expf(-x)); }
__device__ inline float silu_grad(float x) {
  float s = 1.f / (1.f + expf(-x));
  return s * (1.f + x * (1.f - s));
}

// ------------------------------------------------------------ host errors
void set_error(const std::string& msg);
const char* get_error();

struct Status {
  int code;  // 0 ok, 1 invalid argument, 2 no memory, 3 device error, 4 unsupported
};

}  // namespace jg

#define JG_CHECK_LAUNCH(name)                                                   \
  do {                                                                          \
    hipError_t e_ = hipGetLastError();                                          \
    if (e_ != hipSuccess) {                                                     \
      ::jg::set_error(std::string(name) + ": " + hipGetErrorString(e_));        \
      return 3;                                                                 \
    }                                                                           \
  } while (0)
