// Uniform-state reverse step: the entropy-bound sampler of Algorithm 2.
//
// Determinism contract (shared with the masked sampler's: Philox4x32-10 keyed by the
// seed, own float32 log / exp, this file compiled without contraction):
//  * x_hat = argmax_v l_v (ties to the smaller v); l' = l * inv_temp, m = max l';
//  * x_tilde = argmax_v (l'_v + G_v), G from the vocabulary counters (v/4, pos, row, step);
//  * y = l' - m, e = exp(y), A = sum rint(e 2^40), B = sum rint((-y e) 2^40) (zero where
//    e = 0), H = log(float(A) 2^-40) + float(B) / float(A), Hq = rint(H 2^40): integer
//    sums, so any reduction order gives the same H;
//  * a position is accepted iff the sum of the Hq ranked before it, in (Hq, position)
//    order, is at most rint(eta 2^40); the others take (w * V) >> 32 with w word 0 of
//    Philox at counter (2^31 + 1, pos, row, step); the last step writes x_hat;
//  * a block's first canvas: (w * V) >> 32, w word 0 at counter (2^31 + 2, pos, row, block).
// The self-conditioning signal s = softmax(l') E is the product (1/Z) e E, taken by the
// bf16 (or fp32) GEMM with the row factor 2^40 / float(A) in its epilogue.
#include "common.h"
#include "kernels.h"
#include "sampler_math.h"

#pragma clang fp contract(off)

namespace tadm {
namespace {

constexpr float TWO40 = 1099511627776.0f;
constexpr uint32_t RENOISE_WORD0 = 0x80000001u, INIT_WORD0 = 0x80000002u;

__device__ __forceinline__ int32_t uniform_token(uint32_t word0, uint32_t pos, uint32_t row, uint32_t c3, uint32_t k0,
                                                 uint32_t k1, int V) {
  uint32_t c[4] = {word0, pos, row, c3};
  philox4x32_10(c, k0, k1);
  return (int32_t)(((unsigned long long)c[0] * (uint32_t)V) >> 32);
}

__device__ __forceinline__ void store_weight(float* p, float e) { *p = e; }
__device__ __forceinline__ void store_weight(bf16* p, float e) { *p = (bf16)e; }

// Exact contract score l' + G of entry v.
__device__ __forceinline__ float gumbel_score(const float* lg, int v, uint32_t pos, uint32_t row, uint32_t step_id,
                                              uint32_t k0, uint32_t k1, float inv_temp) {
  uint32_t c[4] = {(uint32_t)(v >> 2), pos, row, step_id};
  philox4x32_10(c, k0, k1);
  return exact_score_of(lg[v] * inv_temp, uniform01(c[v & 3]));
}

// grid B * Lc (row = b * Lc + j), 256 threads.  Two passes over the row: the argmax and
// maximum, then exponentials, the two fixed-point sums, the optional weights e_v for the
// self-conditioning product (P[row, v], zero on the padding v in [V, ldp)) and the
// screened Gumbel-max draw (the masked sampler's certified window, exact fallback).
template <class PT>
__global__ __launch_bounds__(256) void entropy_kernel(const float* logits, int V, int Lc, int pos_base,
                                                      uint32_t step_id, uint32_t k0, uint32_t k1, float inv_temp,
                                                      int32_t* xhat, int32_t* xtilde, float* H, long long* Hq,
                                                      float* rscale, PT* P, int ldp) {
  __shared__ float s_f[4], s_g[4];
  __shared__ int s_i[4], s_flag[4];
  __shared__ long long s_a[4], s_b[4];
  const int row = blockIdx.x, b = row / Lc, j = row % Lc;
  const uint32_t pos = (uint32_t)(pos_base + j);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* lg = logits + (size_t)row * V;

  // argmax of the raw logits, smallest index among equal maxima (each thread's entries in
  // increasing order, so a strict > keeps its smallest; float4 granules when V % 4 == 0,
  // four of them in flight)
  const bool vec = (V & 3) == 0;  // whole float4 granules (then ldp % 4 == 0 too)
  Best am{-INFINITY, 0x7FFFFFFF};
  if (vec) {
    const int nq = V >> 2;
    for (int q0 = tid; q0 < nq; q0 += 4 * 256) {
      float4 x[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int q = q0 + 256 * u;
        x[u] = q < nq ? *reinterpret_cast<const float4*>(lg + 4 * q)
                      : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = 4 * (q0 + 256 * u);
        if (x[u].x > am.score) am = Best{x[u].x, v};
        if (x[u].y > am.score) am = Best{x[u].y, v + 1};
        if (x[u].z > am.score) am = Best{x[u].z, v + 2};
        if (x[u].w > am.score) am = Best{x[u].w, v + 3};
      }
    }
  } else {
    for (int v = tid; v < V; v += 256) {
      const float x = lg[v];
      if (x > am.score) am = Best{x, v};
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) am = better(am, Best{__shfl_xor(am.score, o, 64), __shfl_xor(am.v, o, 64)});
  if (lane == 0) {
    s_f[wave] = am.score;
    s_i[wave] = am.v;
  }
  __syncthreads();
  am = Best{s_f[0], s_i[0]};
  for (int w = 1; w < 4; ++w) am = better(am, Best{s_f[w], s_i[w]});
  if (am.v >= V) am.v = 0;  // only with non-finite logits
  const float m = lg[am.v] * inv_temp;  // max l' (rounding is monotone)

  // A and B as float64 sums of their integer terms (each < 2^41, V / 256 of them per
  // thread: 1024 at V = 262144, so every partial sum stays below 2^51 < 2^53): exact,
  // then converted once
  double Ad = 0.0, Bd = 0.0;
  Top2 top;
  for (int q = tid; 4 * q < V; q += 256) {
    float l[4];
    if (vec) {
      const float4 x = *reinterpret_cast<const float4*>(lg + 4 * q);
      l[0] = x.x; l[1] = x.y; l[2] = x.z; l[3] = x.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) l[e] = 4 * q + e < V ? lg[4 * q + e] : 0.f;
    }
    uint32_t c[4] = {(uint32_t)q, pos, (uint32_t)b, step_id};
    philox4x32_10(c, k0, k1);
    float w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * q + e;
      w[e] = 0.f;
      if (v >= V) continue;
      const float lp = l[e] * inv_temp;
      const float y = lp - m;
      const float ex = own_exp(y);
      w[e] = ex;
      Ad += (double)rintf(ex * TWO40);
      Bd += ex > 0.f ? (double)rintf(((-y) * ex) * TWO40) : 0.0;
      // the running top two, by selects
      const float sc = screen_score(lp, uniform01(c[e]));
      const bool t1 = sc > top.a1;
      top.a2 = t1 ? top.a1 : fmaxf(top.a2, sc);
      top.v1 = t1 ? v : top.v1;
      top.a1 = t1 ? sc : top.a1;
    }
    if (P) {
      PT* dst = P + (size_t)row * ldp + 4 * q;
      if (vec)
        store4(dst, w[0], w[1], w[2], w[3]);
      else
        for (int e = 0; e < 4 && 4 * q + e < V; ++e) store_weight(dst + e, w[e]);
    }
  }
  if (P)
    for (int v = V + tid; v < ldp; v += 256) store_weight(P + (size_t)row * ldp + v, 0.f);
  long long A = (long long)Ad, Bs = (long long)Bd;
  float amax = top.a1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    A += __shfl_xor(A, o, 64);
    Bs += __shfl_xor(Bs, o, 64);
    amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  }
  __syncthreads();  // s_f / s_i of the argmax are read
  if (lane == 0) {
    s_a[wave] = A;
    s_b[wave] = Bs;
    s_g[wave] = amax;
  }
  __syncthreads();
  amax = fmaxf(fmaxf(s_g[0], s_g[1]), fmaxf(s_g[2], s_g[3]));
  const float delta = 1e-3f + 2.4e-6f * (fabsf(m) + 32.f);  // screening error bound, x 100
  const float lo = amax - 2.5f * delta;
  const int multi = __any(top.a2 >= lo) ? 1 : 0;
  if (lane == 0) s_flag[wave] = multi;
  __syncthreads();
  const bool slow = s_flag[0] | s_flag[1] | s_flag[2] | s_flag[3];
  Best best{-INFINITY, 0x7FFFFFFF};
  if (!slow) {
    if (top.a1 >= lo && top.v1 < V)
      best = Best{gumbel_score(lg, top.v1, pos, (uint32_t)b, step_id, k0, k1, inv_temp), top.v1};
  } else {
    for (int q = tid; 4 * q < V; q += 256) {
      uint32_t c[4] = {(uint32_t)q, pos, (uint32_t)b, step_id};
      philox4x32_10(c, k0, k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 4 * q + e;
        if (v >= V) break;
        const float sc = exact_score_of(lg[v] * inv_temp, uniform01(c[e]));
        if (sc > best.score) best = Best{sc, v};
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) best = better(best, Best{__shfl_xor(best.score, o, 64), __shfl_xor(best.v, o, 64)});
  __syncthreads();
  if (lane == 0) {
    s_f[wave] = best.score;
    s_i[wave] = best.v;
  }
  __syncthreads();
  if (tid == 0) {
    best = Best{s_f[0], s_i[0]};
    for (int w = 1; w < 4; ++w) best = better(best, Best{s_f[w], s_i[w]});
    if (best.v >= V) best.v = 0;  // only with non-finite logits
    const long long At = s_a[0] + s_a[1] + s_a[2] + s_a[3], Bt = s_b[0] + s_b[1] + s_b[2] + s_b[3];
    const float fA = (float)At, fB = (float)Bt;
    const float h = own_log(fA * 9.094947017729282379150390625e-13f) + fB / fA;  // 2^-40 exact
    xhat[row] = am.v;
    xtilde[row] = best.v;
    H[row] = h;
    Hq[row] = (long long)rintf(h * TWO40);
    rscale[row] = TWO40 / fA;
  }
}

// grid B, 1024 threads, dynamic LDS Lc x 8 B.  Position j is accepted iff the exact sum of
// the Hq ranked before it ((Hq, position) order) is <= etaq.  next may alias canvas.
__global__ __launch_bounds__(1024) void accept_kernel(const long long* Hq, const int32_t* xhat, const int32_t* xtilde,
                                                      const int32_t* canvas, int32_t* next, int L, int off, int Lc,
                                                      int pos_base, uint32_t step_id, uint32_t k0, uint32_t k1, int V,
                                                      long long etaq, int last) {
  extern __shared__ long long s_h[];
  const int b = blockIdx.x, tid = threadIdx.x;
  for (int j = tid; j < Lc; j += 1024) s_h[j] = Hq[(size_t)b * Lc + j];
  if (next != canvas)
    for (int t = tid; t < off; t += 1024) next[(size_t)b * L + t] = canvas[(size_t)b * L + t];
  __syncthreads();
  for (int j = tid; j < Lc; j += 1024) {
    const size_t row = (size_t)b * Lc + j;
    int32_t tok;
    if (last) {
      tok = xhat[row];
    } else {
      const long long hj = s_h[j];
      long long before = 0;
      for (int k = 0; k < Lc; ++k) {
        const long long hk = s_h[k];
        if (hk < hj || (hk == hj && k < j)) before += hk;
      }
      tok = before <= etaq ? xtilde[row]
                           : uniform_token(RENOISE_WORD0, (uint32_t)(pos_base + j), (uint32_t)b, step_id, k0, k1, V);
    }
    next[(size_t)b * L + off + j] = tok;
  }
}

// tok[b * ld + col0 + t] = uniform token of position pos_base + t, t < n
__global__ void init_uniform_kernel(int32_t* tok, int ld, int col0, int B, int n, int pos_base, uint32_t block,
                                    uint32_t k0, uint32_t k1, int V) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)B * n) return;
  const int b = (int)(i / n), t = (int)(i % n);
  tok[(size_t)b * ld + col0 + t] = uniform_token(INIT_WORD0, (uint32_t)(pos_base + t), (uint32_t)b, block, k0, k1, V);
}

// c[b, off + j, :] += sc[b * Lc + j, :] (float4 granules; d % 4 == 0)
__global__ void add_selfcond_kernel(float* c, const float* sc, int B, int L, int off, int Lc, int d) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x, d4 = d / 4;
  if (i >= (long)B * Lc * d4) return;
  const long r = i / d4, k = i % d4;
  const int b = (int)(r / Lc), j = (int)(r % Lc);
  float4* dst = reinterpret_cast<float4*>(c + ((size_t)b * L + off + j) * d) + k;
  const float4 s = reinterpret_cast<const float4*>(sc + (size_t)r * d)[k];
  float4 x = *dst;
  x.x += s.x;
  x.y += s.y;
  x.z += s.z;
  x.w += s.w;
  *dst = x;
}

// ET[n, v] = E[v, n] for v < V, 0 for V <= v < ldt; 64 x 64 tiles through LDS
template <class T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* E, int V, int d, T* ET, int ldt) {
  __shared__ T tile[64][65];
  const int v0 = blockIdx.x * 64, n0 = blockIdx.y * 64, tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int r = ty; r < 64; r += 4) {
    const int v = v0 + r, n = n0 + tx;
    tile[r][tx] = (v < V && n < d) ? E[(size_t)v * d + n] : from_f32<T>(0.f);
  }
  __syncthreads();
  for (int r = ty; r < 64; r += 4) {
    const int n = n0 + r, v = v0 + tx;
    if (n < d && v < ldt) ET[(size_t)n * ldt + v] = tile[tx][r];
  }
}

}  // namespace

hipError_t entropy_stats(const float* logits, int B, int Lc, int V, int pos_base, uint32_t step_id, uint64_t seed,
                         float inv_temp, int32_t* xhat, int32_t* xtilde, float* H, long long* Hq, float* rscale,
                         DType pt, void* P, int ldp, hipStream_t s) {
  if (B * Lc == 0) return hipSuccess;
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  if (pt == BF16)
    launch_timed(entropy_kernel<bf16>, dim3(B * Lc), dim3(256), 0, s, logits, V, Lc, pos_base, step_id, k0, k1,
                 inv_temp, xhat, xtilde, H, Hq, rscale, static_cast<bf16*>(P), ldp);
  else
    launch_timed(entropy_kernel<float>, dim3(B * Lc), dim3(256), 0, s, logits, V, Lc, pos_base, step_id, k0, k1,
                 inv_temp, xhat, xtilde, H, Hq, rscale, static_cast<float*>(P), ldp);
  return hipGetLastError();
}

hipError_t entropy_accept(const long long* Hq, const int32_t* xhat, const int32_t* xtilde, const int32_t* canvas,
                          int32_t* next, int B, int L, int off, int pos_base, uint32_t step_id, uint64_t seed, int V,
                          long long etaq, int last, hipStream_t s) {
  const int Lc = L - off;
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(accept_kernel, dim3(B), dim3(1024), (size_t)Lc * 8, s, Hq, xhat, xtilde, canvas, next, L, off,
                     Lc, pos_base, step_id, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), V, etaq, last);
  return hipGetLastError();
}

hipError_t init_uniform_tokens(int32_t* tok, int ld, int col0, int B, int n, int pos_base, uint32_t block,
                               uint64_t seed, int V, hipStream_t s) {
  const long total = (long)B * n;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(init_uniform_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, tok, ld, col0, B, n,
                     pos_base, block, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), V);
  return hipGetLastError();
}

hipError_t add_selfcond(float* c, const float* sc, int B, int L, int off, int d, hipStream_t s) {
  const int Lc = L - off;
  const long total = (long)B * Lc * (d / 4);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(add_selfcond_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, c, sc, B, L, off,
                     Lc, d);
  return hipGetLastError();
}

hipError_t transpose_rows(DType dt, const void* E, int V, int d, void* ET, int ldt, hipStream_t s) {
  const dim3 grid((ldt + 63) / 64, (d + 63) / 64);
  if (dt == BF16)
    hipLaunchKernelGGL(transpose_kernel<bf16>, grid, dim3(256), 0, s, static_cast<const bf16*>(E), V, d,
                       static_cast<bf16*>(ET), ldt);
  else
    hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(E), V, d,
                       static_cast<float*>(ET), ldt);
  return hipGetLastError();
}

}  // namespace tadm
