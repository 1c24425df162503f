// Bandwidth-bound row kernels: embedding gather, RMSNorm, LayerNorm and small
// conversions.  One wave64 per row, float4 accesses, wave-shuffle reductions.
#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

template <class T>
__device__ __forceinline__ float4 load4(const T* p);
template <>
__device__ __forceinline__ float4 load4<float>(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
template <>
__device__ __forceinline__ float4 load4<bf16>(const bf16* p) {
  const bf16x4 v = *reinterpret_cast<const bf16x4*>(p);
  return make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
}

template <class T>
__global__ void embed_kernel(const int32_t* tok, int n_tok, const T* E, int d, int max_row,
                             float* out) {
  const int q = d / 4;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)n_tok * q) return;
  const int t = (int)(idx / q), c = (int)(idx % q);
  int row = tok[t];
  row = row < 0 ? 0 : (row > max_row ? max_row : row);  // memory safety for bad ids
  *reinterpret_cast<float4*>(out + (size_t)t * d + 4 * c) = load4(E + (size_t)row * d + 4 * c);
}

// y[r] = x[map(r)] * rsqrt(mean(x^2) + eps) * g.  NV > 0: d <= 256 NV and the row stays in
// registers between the two passes (one read of x); NV = 0: any d, x read twice.
template <class T, int NV>
__global__ __launch_bounds__(256) void rms_kernel(const float* x, const float* g, float eps,
                                                  int n_rows, int d, int rows_per_b,
                                                  int in_stride_b, int in_off, T* y) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= n_rows) return;
  const long src = (long)(r / rows_per_b) * in_stride_b + in_off + (r % rows_per_b);
  const float* xr = x + src * d;
  T* yr = y + (size_t)r * d;
  float ss = 0.f;
  if constexpr (NV > 0) {
    // the gains are loaded with the row, so that their latency overlaps the row's
    float4 v[NV], w[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane * 4 + 256 * i;
      v[i] = c < d ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      w[i] = c < d ? *reinterpret_cast<const float4*>(g + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    ss = wave_sum(ss);
    const float rs = rsqrtf(ss / d + eps);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane * 4 + 256 * i;
      if (c < d) store4(yr + c, v[i].x * rs * w[i].x, v[i].y * rs * w[i].y, v[i].z * rs * w[i].z, v[i].w * rs * w[i].w);
    }
  } else {
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    ss = wave_sum(ss);
    const float rs = rsqrtf(ss / d + eps);
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      const float4 w = *reinterpret_cast<const float4*>(g + c);
      store4(yr + c, v.x * rs * w.x, v.y * rs * w.y, v.z * rs * w.z, v.w * rs * w.w);
    }
  }
}

template <class T>
__global__ __launch_bounds__(256) void rms_gather_kernel(const float* x, const float* g, float eps,
                                                         const int32_t* cidx, const int* count,
                                                         int Lc, int L, int off, int d, T* y) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= *count) return;
  const int c = cidx[r];
  const float* xr = x + ((size_t)(c / Lc) * L + off + c % Lc) * d;
  float ss = 0.f;
  for (int k = lane * 4; k < d; k += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  const float rs = rsqrtf(ss / d + eps);
  T* yr = y + (size_t)r * d;
  for (int k = lane * 4; k < d; k += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    const float4 w = *reinterpret_cast<const float4*>(g + k);
    store4(yr + k, v.x * rs * w.x, v.y * rs * w.y, v.z * rs * w.z, v.w * rs * w.w);
  }
}

template <class T>
__global__ __launch_bounds__(256) void ln_kernel(const float* x, const float* w, const float* b,
                                                 float eps, int n_rows, int d, T* y_t, float* y_f) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= n_rows) return;
  const float* xr = x + (size_t)r * d;
  float s = 0.f;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    s += v.x + v.y + v.z + v.w;
  }
  const float mu = wave_sum(s) / d;
  float ss = 0.f;
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    const float a = v.x - mu, bb = v.y - mu, cc = v.z - mu, dd = v.w - mu;
    ss += a * a + bb * bb + cc * cc + dd * dd;
  }
  const float rs = rsqrtf(wave_sum(ss) / d + eps);
  for (int c = lane * 4; c < d; c += 256) {
    const float4 v = *reinterpret_cast<const float4*>(xr + c);
    const float4 ww = *reinterpret_cast<const float4*>(w + c);
    const float4 bb = *reinterpret_cast<const float4*>(b + c);
    const float o0 = (v.x - mu) * rs * ww.x + bb.x, o1 = (v.y - mu) * rs * ww.y + bb.y;
    const float o2 = (v.z - mu) * rs * ww.z + bb.z, o3 = (v.w - mu) * rs * ww.w + bb.w;
    if (y_t) store4(y_t + (size_t)r * d + c, o0, o1, o2, o3);
    if (y_f) store4(y_f + (size_t)r * d + c, o0, o1, o2, o3);
  }
}

// LayerNorm of x in place (float32), then the RMSNorm of its result into y (the next
// layer's normalised input): the two kernels' arithmetic in one pass over the row.
// NV > 0: d <= 256 NV and the row stays in registers; NV = 0: any d, rows re-read.
template <class T, int NV>
__global__ __launch_bounds__(256) void ln_rms_kernel(float* x, const float* w, const float* b, float ln_eps,
                                                     const float* g, float rms_eps, int n_rows, int d, T* y) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= n_rows) return;
  float* xr = x + (size_t)r * d;
  T* yr = y + (size_t)r * d;
  if constexpr (NV > 0) {
    float4 v[NV];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane * 4 + 256 * i;
      v[i] = c < d ? *reinterpret_cast<const float4*>(xr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      s += v[i].x + v[i].y + v[i].z + v[i].w;
    }
    const float mu = wave_sum(s) / d;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (lane * 4 + 256 * i < d) {
        const float a = v[i].x - mu, bb = v[i].y - mu, cc = v[i].z - mu, dd = v[i].w - mu;
        ss += a * a + bb * bb + cc * cc + dd * dd;
      }
    const float rs = rsqrtf(wave_sum(ss) / d + ln_eps);
    float sq = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane * 4 + 256 * i;
      if (c < d) {
        const float4 ww = *reinterpret_cast<const float4*>(w + c);
        const float4 bv = *reinterpret_cast<const float4*>(b + c);
        v[i] = make_float4((v[i].x - mu) * rs * ww.x + bv.x, (v[i].y - mu) * rs * ww.y + bv.y,
                           (v[i].z - mu) * rs * ww.z + bv.z, (v[i].w - mu) * rs * ww.w + bv.w);
        *reinterpret_cast<float4*>(xr + c) = v[i];
      } else {
        v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
      sq += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
    const float rr = rsqrtf(wave_sum(sq) / d + rms_eps);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = lane * 4 + 256 * i;
      if (c < d) {
        const float4 gg = *reinterpret_cast<const float4*>(g + c);
        store4(yr + c, v[i].x * rr * gg.x, v[i].y * rr * gg.y, v[i].z * rr * gg.z, v[i].w * rr * gg.w);
      }
    }
  } else {
    float s = 0.f;
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      s += v.x + v.y + v.z + v.w;
    }
    const float mu = wave_sum(s) / d;
    float ss = 0.f;
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      const float a = v.x - mu, bb = v.y - mu, cc = v.z - mu, dd = v.w - mu;
      ss += a * a + bb * bb + cc * cc + dd * dd;
    }
    const float rs = rsqrtf(wave_sum(ss) / d + ln_eps);
    float sq = 0.f;
    for (int c = lane * 4; c < d; c += 256) {
      const float4 v = *reinterpret_cast<const float4*>(xr + c);
      const float4 ww = *reinterpret_cast<const float4*>(w + c);
      const float4 bv = *reinterpret_cast<const float4*>(b + c);
      const float4 o = make_float4((v.x - mu) * rs * ww.x + bv.x, (v.y - mu) * rs * ww.y + bv.y,
                                   (v.z - mu) * rs * ww.z + bv.z, (v.w - mu) * rs * ww.w + bv.w);
      *reinterpret_cast<float4*>(xr + c) = o;
      sq += o.x * o.x + o.y * o.y + o.z * o.z + o.w * o.w;
    }
    const float rr = rsqrtf(wave_sum(sq) / d + rms_eps);
    for (int c = lane * 4; c < d; c += 256) {  // this lane's own writes above
      const float4 o = *reinterpret_cast<const float4*>(xr + c);
      const float4 gg = *reinterpret_cast<const float4*>(g + c);
      store4(yr + c, o.x * rr * gg.x, o.y * rr * gg.y, o.z * rr * gg.z, o.w * rr * gg.w);
    }
  }
}

__global__ void copy_kernel(const float4* src, float4* dst, size_t n4) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n4) dst[i] = src[i];
}

template <class T>
__global__ void to_f32_kernel(const T* src, float* dst, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = f32_of(src[i]);
}

__global__ void glu_kernel(const float* pre, int n_rows, int F, int silu, float* out) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)n_rows * F) return;
  const int r = (int)(i / F), f = (int)(i % F);
  const int gr = 32 * (f / 16) + (f % 16);
  const float g = pre[(size_t)r * 2 * F + gr], u = pre[(size_t)r * 2 * F + gr + 16];
  out[i] = (silu ? siluf_(g) : gelu_erf(g)) * u;
}

inline unsigned blocks(long n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

hipError_t embed_gather(DType dt, const int32_t* tok, int n_tok, const void* embed, int table_rows,
                        int d, float* out, hipStream_t s) {
  const long n = (long)n_tok * (d / 4);
  if (n == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(embed_kernel<bf16>, dim3(blocks(n, 256)), dim3(256), 0, s, tok, n_tok,
                       static_cast<const bf16*>(embed), d, table_rows - 1, out);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(blocks(n, 256)), dim3(256), 0, s, tok, n_tok,
                       static_cast<const float*>(embed), d, table_rows - 1, out);
  return hipGetLastError();
}

hipError_t rms_norm(DType dt, const float* x, const float* g, float eps, int n_rows, int d,
                    int rows_per_b, int in_stride_b, int in_off, void* y, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  const dim3 grid(blocks(n_rows, 4));
  if (dt == BF16) {
    bf16* yb = static_cast<bf16*>(y);
    if (d <= 1024)
      hipLaunchKernelGGL((rms_kernel<bf16, 4>), grid, dim3(256), 0, s, x, g, eps, n_rows, d, rows_per_b,
                         in_stride_b, in_off, yb);
    else if (d <= 2048)
      hipLaunchKernelGGL((rms_kernel<bf16, 8>), grid, dim3(256), 0, s, x, g, eps, n_rows, d, rows_per_b,
                         in_stride_b, in_off, yb);
    else if (d <= 4608)
      hipLaunchKernelGGL((rms_kernel<bf16, 18>), grid, dim3(256), 0, s, x, g, eps, n_rows, d, rows_per_b,
                         in_stride_b, in_off, yb);
    else
      hipLaunchKernelGGL((rms_kernel<bf16, 0>), grid, dim3(256), 0, s, x, g, eps, n_rows, d, rows_per_b,
                         in_stride_b, in_off, yb);
  } else {
    hipLaunchKernelGGL((rms_kernel<float, 0>), grid, dim3(256), 0, s, x, g, eps, n_rows, d, rows_per_b,
                       in_stride_b, in_off, static_cast<float*>(y));
  }
  return hipGetLastError();
}

hipError_t rms_norm_gather(DType dt, const float* x, const float* g, float eps, const int32_t* cidx,
                           const int* count, int max_rows, int Lc, int L, int off, int d, void* y,
                           hipStream_t s) {
  if (max_rows == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(rms_gather_kernel<bf16>, dim3(blocks(max_rows, 4)), dim3(256), 0, s, x, g, eps, cidx,
                       count, Lc, L, off, d, static_cast<bf16*>(y));
  else
    hipLaunchKernelGGL(rms_gather_kernel<float>, dim3(blocks(max_rows, 4)), dim3(256), 0, s, x, g, eps, cidx,
                       count, Lc, L, off, d, static_cast<float*>(y));
  return hipGetLastError();
}

hipError_t layer_norm(DType dt, const float* x, const float* w, const float* b, float eps, int n_rows,
                      int d, void* y_t, float* y_f, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(ln_kernel<bf16>, dim3(blocks(n_rows, 4)), dim3(256), 0, s, x, w, b, eps, n_rows,
                       d, static_cast<bf16*>(y_t), y_f);
  else
    hipLaunchKernelGGL(ln_kernel<float>, dim3(blocks(n_rows, 4)), dim3(256), 0, s, x, w, b, eps, n_rows,
                       d, static_cast<float*>(y_t), y_f);
  return hipGetLastError();
}

hipError_t layer_rms_norm(DType dt, float* x, const float* w, const float* b, float ln_eps, const float* g,
                          float rms_eps, int n_rows, int d, void* y, hipStream_t s) {
  if (n_rows == 0) return hipSuccess;
  const dim3 grid(blocks(n_rows, 4));
  if (dt == BF16) {
    if (d <= 1024)
      hipLaunchKernelGGL((ln_rms_kernel<bf16, 4>), grid, dim3(256), 0, s, x, w, b, ln_eps, g, rms_eps, n_rows, d,
                         static_cast<bf16*>(y));
    else
      hipLaunchKernelGGL((ln_rms_kernel<bf16, 0>), grid, dim3(256), 0, s, x, w, b, ln_eps, g, rms_eps, n_rows, d,
                         static_cast<bf16*>(y));
  } else {
    hipLaunchKernelGGL((ln_rms_kernel<float, 0>), grid, dim3(256), 0, s, x, w, b, ln_eps, g, rms_eps, n_rows, d,
                       static_cast<float*>(y));
  }
  return hipGetLastError();
}

hipError_t copy_f32(const float* src, float* dst, size_t n, hipStream_t s) {
  const size_t n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  hipLaunchKernelGGL(copy_kernel, dim3(blocks((long)n4, 256)), dim3(256), 0, s,
                     reinterpret_cast<const float4*>(src), reinterpret_cast<float4*>(dst), n4);
  return hipGetLastError();
}

hipError_t to_f32(DType dt, const void* src, float* dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (dt == BF16)
    hipLaunchKernelGGL(to_f32_kernel<bf16>, dim3(blocks((long)n, 256)), dim3(256), 0, s,
                       static_cast<const bf16*>(src), dst, n);
  else
    hipLaunchKernelGGL(to_f32_kernel<float>, dim3(blocks((long)n, 256)), dim3(256), 0, s,
                       static_cast<const float*>(src), dst, n);
  return hipGetLastError();
}

hipError_t glu_f32(const float* pre, int n_rows, int F, int silu, float* out, hipStream_t s) {
  const long n = (long)n_rows * F;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(glu_kernel, dim3(blocks(n, 256)), dim3(256), 0, s, pre, n_rows, F, silu, out);
  return hipGetLastError();
}

}  // namespace tadm

namespace tadm {
namespace {
template <class T, class D>
__global__ void scatter_kernel(const T* src, long rows, int cols, D* dst, long row_off, int glu_half,
                               int rope_dh) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const long r = i / cols;
  const int c = (int)(i % cols);
  long dr = glu_half < 0 ? row_off + r : row_off + 32 * (r / 16) + 16 * glu_half + r % 16;
  if (rope_dh > 0) {
    const int h = rope_dh / 2, w = (int)(r % rope_dh);
    dr = row_off + (r / rope_dh) * rope_dh + (w < h ? 2 * w : 2 * (w - h) + 1);
  }
  dst[dr * cols + c] = from_f32<D>(f32_of(src[i]));
}
__global__ void init_canvas_kernel(const int32_t* prompt, int B, int P, int gen, int mask_id,
                                   int32_t* dst) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int L = P + gen;
  if (i >= (long)B * L) return;
  const int b = (int)(i / L), l = (int)(i % L);
  dst[i] = l < P ? prompt[(size_t)b * P + l] : mask_id;
}
__global__ void fill_kernel(int32_t* dst, size_t n, int32_t v) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = v;
}
}  // namespace

hipError_t scatter_rows(DType dt, const void* src, long rows, int cols, void* dst, int dst_f32,
                        long row_off, int glu_half, int rope_dh, hipStream_t s) {
  const long n = rows * cols;
  if (n == 0) return hipSuccess;
  const unsigned g = (unsigned)((n + 255) / 256);
  if (dt == BF16) {
    if (dst_f32)
      hipLaunchKernelGGL((scatter_kernel<bf16, float>), dim3(g), dim3(256), 0, s,
                         static_cast<const bf16*>(src), rows, cols, static_cast<float*>(dst), row_off,
                         glu_half, rope_dh);
    else
      hipLaunchKernelGGL((scatter_kernel<bf16, bf16>), dim3(g), dim3(256), 0, s,
                         static_cast<const bf16*>(src), rows, cols, static_cast<bf16*>(dst), row_off,
                         glu_half, rope_dh);
  } else {
    hipLaunchKernelGGL((scatter_kernel<float, float>), dim3(g), dim3(256), 0, s,
                       static_cast<const float*>(src), rows, cols, static_cast<float*>(dst), row_off,
                       glu_half, rope_dh);
  }
  return hipGetLastError();
}

hipError_t init_canvas(const int32_t* prompt, int B, int P, int gen, int mask_id, int32_t* dst,
                       hipStream_t s) {
  const long n = (long)B * (P + gen);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(init_canvas_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, prompt, B,
                     P, gen, mask_id, dst);
  return hipGetLastError();
}

hipError_t fill_i32(int32_t* dst, size_t n, int32_t v, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, dst, n, v);
  return hipGetLastError();
}
}  // namespace tadm
