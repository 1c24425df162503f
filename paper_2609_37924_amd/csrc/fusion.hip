// Row kernels of the paired-attention fusion: token-wise RMS scales, row scaling,
// the feature concatenation F = [U; Z0; Z - Z0; M] and the scalar gate.
// One wave64 per row, float4 accesses, wave-shuffle reductions.
#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

__global__ __launch_bounds__(256) void row_rms_kernel(const float* x, int n_rows, int d, float eps,
                                                      float* s) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= n_rows) return;
  const float* xr = x + (size_t)r * d;
  float ss = 0.f;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  if (lane == 0) s[r] = sqrtf(ss / d + eps);
}

template <class T>
__global__ __launch_bounds__(256) void scale_rows_kernel(const float* x, const float* s, int n_rows,
                                                         int d, T* y) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= n_rows) return;
  const float inv = 1.f / s[r];
  const float* xr = x + (size_t)r * d;
  T* yr = y + (size_t)r * d;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    store4(yr + c, v.x * inv, v.y * inv, v.z * inv, v.w * inv);
  }
}

template <class T>
__global__ void to_type_kernel(const float* x, size_t n4, T* y) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  const float4 v = reinterpret_cast<const float4*>(x)[i];
  store4(y + 4 * i, v.x, v.y, v.z, v.w);
}

template <class T>
__global__ void features_kernel(const float* U, const float* Z0, const float* Z, const T* M, int n_rows,
                                int r, T* F) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;  // one thread per 4 features of a part
  const int q = r / 4;
  if (i >= (long)n_rows * 4 * q) return;
  const int row = (int)(i / (4 * q)), rem = (int)(i % (4 * q)), part = rem / q, c = 4 * (rem % q);
  const size_t o = (size_t)row * r + c;
  T* dst = F + (size_t)row * 4 * r + part * r + c;
  if (part == 3) {
    *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(M + o);  // 4 bf16 (or half of 4 float)
    if (sizeof(T) == 4) *reinterpret_cast<uint2*>(dst + 2) = *reinterpret_cast<const uint2*>(M + o + 2);
    return;
  }
  float4 v;
  if (part == 0) v = *reinterpret_cast<const float4*>(U + o);
  else if (part == 1) v = *reinterpret_cast<const float4*>(Z0 + o);
  else {
    const float4 a = *reinterpret_cast<const float4*>(Z + o), b = *reinterpret_cast<const float4*>(Z0 + o);
    v = make_float4(a.x - b.x, a.y - b.y, a.z - b.z, a.w - b.w);
  }
  store4(dst, v.x, v.y, v.z, v.w);
}

template <class T>
__global__ __launch_bounds__(256) void gate_kernel(const T* G1, const float* w, const float* b, int n_rows,
                                                   int r, float* g) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n_rows) return;
  float acc = 0.f;
  for (int c = lane; c < r; c += 64) acc += f32_of(G1[(size_t)row * r + c]) * w[c];
  acc = wave_sum(acc);
  if (lane == 0) g[row] = sigmoidf_(acc + b[0]);
}

inline unsigned nblk(long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t row_rms(const float* x, int n_rows, int d, float eps, float* s, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(row_rms_kernel, dim3(nblk(n_rows, 4)), dim3(256), 0, st, x, n_rows, d, eps, s);
  return hipGetLastError();
}

hipError_t scale_rows(DType dt, const float* x, const float* s, int n_rows, int d, void* y, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(scale_rows_kernel<bf16>, dim3(nblk(n_rows, 4)), dim3(256), 0, st, x, s, n_rows, d,
                       static_cast<bf16*>(y));
  else
    hipLaunchKernelGGL(scale_rows_kernel<float>, dim3(nblk(n_rows, 4)), dim3(256), 0, st, x, s, n_rows, d,
                       static_cast<float*>(y));
  return hipGetLastError();
}

hipError_t to_type(DType dt, const float* x, size_t n, void* y, hipStream_t st) {
  const size_t n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(to_type_kernel<bf16>, dim3(nblk((long)n4, 256)), dim3(256), 0, st, x, n4,
                       static_cast<bf16*>(y));
  else
    hipLaunchKernelGGL(to_type_kernel<float>, dim3(nblk((long)n4, 256)), dim3(256), 0, st, x, n4,
                       static_cast<float*>(y));
  return hipGetLastError();
}

hipError_t paired_features(DType dt, const float* U, const float* Z0, const float* Z, const void* M, int n_rows,
                           int r, void* F, hipStream_t st) {
  const long n = (long)n_rows * r;  // threads: 4 parts x r/4 per row
  if (n == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(features_kernel<bf16>, dim3(nblk(n, 256)), dim3(256), 0, st, U, Z0, Z,
                       static_cast<const bf16*>(M), n_rows, r, static_cast<bf16*>(F));
  else
    hipLaunchKernelGGL(features_kernel<float>, dim3(nblk(n, 256)), dim3(256), 0, st, U, Z0, Z,
                       static_cast<const float*>(M), n_rows, r, static_cast<float*>(F));
  return hipGetLastError();
}

hipError_t row_gate(DType dt, const void* G1, const float* w, const float* b, int n_rows, int r, float* g,
                    hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(gate_kernel<bf16>, dim3(nblk(n_rows, 4)), dim3(256), 0, st, static_cast<const bf16*>(G1),
                       w, b, n_rows, r, g);
  else
    hipLaunchKernelGGL(gate_kernel<float>, dim3(nblk(n_rows, 4)), dim3(256), 0, st, static_cast<const float*>(G1),
                       w, b, n_rows, r, g);
  return hipGetLastError();
}

}  // namespace tadm
