// Device-side helpers shared by the TADM kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define TADM_WAVE 64

__device__ __forceinline__ float f32_of(float x) { return x; }
__device__ __forceinline__ float f32_of(bf16 x) { return (float)x; }

template <class T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// Store 4 consecutive values (8 B for bf16, 16 B for float).
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *reinterpret_cast<bf16x4*>(p) = v;
}

// Store 2 consecutive values (4 B for bf16, 8 B for float).
__device__ __forceinline__ void store2(float* p, float a, float b) { *reinterpret_cast<float2*>(p) = make_float2(a, b); }
__device__ __forceinline__ void store2(bf16* p, float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v = {(bf16)a, (bf16)b};
  *reinterpret_cast<bf16x2*>(p) = v;
}

// The value held by lane l ^ 16 (xor16) or l ^ 32 (xor32) of the wave, exchanged with
// v_permlane16_swap / v_permlane32_swap (a VALU operation; __shfl_xor goes through the
// LDS crossbar).  A swap of v with itself leaves, in every lane, the value of the lower
// and of the upper row (16 lanes) or half (32 lanes) of its pair; the lane takes the
// other one.  Block sizes are multiples of 64, so bit 4 / 5 of threadIdx.x is the lane's.
__device__ __forceinline__ uint32_t xor16(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return (threadIdx.x & 16) ? r[0] : r[1];
}
__device__ __forceinline__ uint32_t xor32(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return (threadIdx.x & 32) ? r[0] : r[1];
}
__device__ __forceinline__ float xor16(float v) { return __uint_as_float(xor16(__float_as_uint(v))); }
__device__ __forceinline__ float xor32(float v) { return __uint_as_float(xor32(__float_as_uint(v))); }
__device__ __forceinline__ int xor16(int v) { return (int)xor16((uint32_t)v); }
__device__ __forceinline__ int xor32(int v) { return (int)xor32((uint32_t)v); }
__device__ __forceinline__ double xor16(double v) {
  const uint64_t b = __double_as_longlong(v);
  return __longlong_as_double((long long)(((uint64_t)xor16((uint32_t)(b >> 32)) << 32) | xor16((uint32_t)b)));
}
__device__ __forceinline__ double xor32(double v) {
  const uint64_t b = __double_as_longlong(v);
  return __longlong_as_double((long long)(((uint64_t)xor32((uint32_t)(b >> 32)) << 32) | xor32((uint32_t)b)));
}

// Workgroups of a launch are dispatched round-robin over the 8 XCDs (id % 8), each with
// its own L2.  Renumber ids so that XCD x runs one contiguous range of logical ids:
// neighbouring work items that read the same data then share an L2.
__device__ __forceinline__ int xcd_contiguous(int id, int n) {
  const int x = id % 8, local = id / 8, q = n / 8, r = n % 8;
  return x < r ? x * (q + 1) + local : r * (q + 1) + (x - r) * q + local;
}

// Whole-wave sum / max, every lane receiving the result: within each 16-lane row by DPP
// (quad swaps of 1 and 2 lanes, then the half-row and row mirrors, each pairing the
// groups built so far), across rows by the permlane swaps.  Each step combines two
// values with a commutative operation, so every lane ends with the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_f<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_f<0x141>(v);  // row_half_mirror
  v += dpp_f<0x140>(v);  // row_mirror
  v += xor16(v);
  v += xor32(v);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x141>(v));
  v = fmaxf(v, dpp_f<0x140>(v));
  v = fmaxf(v, xor16(v));
  v = fmaxf(v, xor32(v));
  return v;
}

// Block-wide sum of one float per thread (blockDim.x a multiple of 64, <= 1024).
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / TADM_WAVE, lane = threadIdx.x % TADM_WAVE;
  const int nw = blockDim.x / TADM_WAVE;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ __forceinline__ float sigmoidf_(float x) { return 1.f / (1.f + __expf(-x)); }
__device__ __forceinline__ float siluf_(float x) { return x * sigmoidf_(x); }

// Activations of products whose results are stored in bf16 (relative resolution 2^-8):
// GELU as x Phi(x) with erfc(z), z = |x| / sqrt(2), from Abramowitz & Stegun 7.1.26
// (Hastings' rational approximation, absolute error <= 1.5e-7), Phi(x) = erfc(z) / 2 for
// x < 0 and 1 - erfc(z) / 2 otherwise; the sigmoid with the hardware reciprocal (1 ulp).
// About a third of the instructions of the library erf and the IEEE division.
__device__ __forceinline__ float gelu_bf16out(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(0.3275911f, z, 1.0f));
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float erfc = poly * __builtin_amdgcn_exp2f(-1.4426950408889634f * z * z);
  return x * (x < 0.f ? 0.5f * erfc : 1.0f - 0.5f * erfc);
}
__device__ __forceinline__ float sigmoid_bf16out(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }
__device__ __forceinline__ float silu_bf16out(float x) { return x * sigmoid_bf16out(x); }
// T = the product's operand type: float32 models keep the library erf and IEEE division
template <class T>
__device__ __forceinline__ float gelu_act(float x) {
  if constexpr (sizeof(T) == 2) return gelu_bf16out(x);
  else return gelu_erf(x);
}
template <class T>
__device__ __forceinline__ float sigmoid_act(float x) {
  if constexpr (sizeof(T) == 2) return sigmoid_bf16out(x);
  else return sigmoidf_(x);
}
template <class T>
__device__ __forceinline__ float silu_act(float x) {
  return x * sigmoid_act<T>(x);
}
