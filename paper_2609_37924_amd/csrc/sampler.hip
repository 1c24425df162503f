// Masked-diffusion reverse step: Gumbel-max sampling with fixed-point confidence and
// confidence-ranked unmasking (MDLM zero-masking and carry-over, sigma_t = 0).
//
// Determinism contract (token choices and unmask order are reproducible bit for bit
// by any IEEE float32 implementation of the same operations):
//  * Philox4x32-10 (Salmon et al., SC'11): counter (v/4, position, row, step id),
//    key (seed low word, seed high word); word v%4 -> u = (2*(x>>9)+1) * 2^-24.
//  * Own float32 log / exp built only from individually rounded +,-,*,/:
//    log: x = 2^e m, m in [sqrt(1/2), sqrt(2)], log m = 2 atanh(s), s = (m-1)/(m+1),
//         series in z = s^2 up to z^5, ln 2 split in a 15-bit head and a tail;
//    exp: Cody-Waite reduction k = rint(y/ln2), degree-7 Taylor polynomial, 2^k from
//         the exponent bits; 0 below -30.
//    This file is compiled with -ffp-contract=off so that no multiply-add is fused,
//    and with correctly rounded float32 division.
//  * token = argmax_v (l_v * inv_temp + G_v), G = -log(-log u), ties to smaller v;
//    confidence = (l'_x - m) - log(float(S) * 2^-40), S = sum_v rint(exp(l'_v - m) 2^40)
//    accumulated in int64, so any reduction order gives the same bits.
//  * ranking: confidence descending, then position ascending.
#include "common.h"
#include "kernels.h"

#pragma clang fp contract(off)

namespace tadm {
namespace {

__device__ __forceinline__ float bits_f(uint32_t b) { return __uint_as_float(b); }

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c[0], hi0 = __umulhi(0xD2511F53u, c[0]);
    const uint32_t lo1 = 0xCD9E8D57u * c[2], hi1 = __umulhi(0xCD9E8D57u, c[2]);
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

__device__ __forceinline__ float uniform01(uint32_t x) {
  return (float)((x >> 9) * 2u + 1u) * 5.9604644775390625e-8f;  // * 2^-24, exact
}

__device__ __forceinline__ float own_log(float x) {
  const float LN2_HI = bits_f(0x3F317200u), LN2_LO = bits_f(0x35BFBE8Eu);
  const uint32_t bits = __float_as_uint(x);
  int e = (int)(bits >> 23) - 127;
  uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
  if (mb > 0x3FB504F3u) {  // m above sqrt(2): halve it
    mb -= 0x00800000u;
    e += 1;
  }
  const float m = __uint_as_float(mb);
  const float f = m - 1.0f;
  const float s = f / (2.0f + f);
  const float z = s * s;
  float p = bits_f(0x3E3A2E8Cu);       // 2/11
  p = p * z + bits_f(0x3E638E39u);     // 2/9
  p = p * z + bits_f(0x3E924925u);     // 2/7
  p = p * z + bits_f(0x3ECCCCCDu);     // 2/5
  p = p * z + bits_f(0x3F2AAAABu);     // 2/3
  p = p * z + 2.0f;
  const float t = s * p;
  const float ef = (float)e;
  return ef * LN2_HI + (ef * LN2_LO + t);
}

__device__ __forceinline__ float own_exp(float y) {
  if (y < -30.0f) return 0.0f;
  const float LN2_HI = bits_f(0x3F317200u), LN2_LO = bits_f(0x35BFBE8Eu);
  const float k = rintf(y * bits_f(0x3FB8AA3Bu));
  const float r = (y - k * LN2_HI) - k * LN2_LO;
  float p = bits_f(0x39500D01u);       // 1/5040
  p = p * r + bits_f(0x3AB60B61u);     // 1/720
  p = p * r + bits_f(0x3C088889u);     // 1/120
  p = p * r + bits_f(0x3D2AAAABu);     // 1/24
  p = p * r + bits_f(0x3E2AAAABu);     // 1/6
  p = p * r + 0.5f;
  p = p * r + 1.0f;
  p = p * r + 1.0f;
  const float scale = __uint_as_float((uint32_t)((int)k + 127) << 23);
  return p * scale;
}

struct Best {
  float score;
  int v;
};
__device__ __forceinline__ Best better(Best a, Best b) {
  return (b.score > a.score || (b.score == a.score && b.v < a.v)) ? b : a;
}

// Screening logarithm: the same exponent/mantissa split and atanh series as own_log,
// with an approximate reciprocal and a shorter series.  Relative error below 1e-6 on
// the sampler's arguments; it only ranks entries and never decides a token.
__device__ __forceinline__ float screen_log(float x) {
  const float LN2 = bits_f(0x3F317218u);
  const uint32_t bits = __float_as_uint(x);
  int e = (int)(bits >> 23) - 127;
  uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
  if (mb > 0x3FB504F3u) {
    mb -= 0x00800000u;
    e += 1;
  }
  const float f = __uint_as_float(mb) - 1.0f;
  const float s = f * __builtin_amdgcn_rcpf(2.0f + f);
  const float z = s * s;
  const float p = fmaf(z, fmaf(z, fmaf(z, 0.2857142857f, 0.4f), 0.6666666667f), 2.0f);
  return fmaf((float)e, LN2, s * p);
}

// Exact contract score of entry v: l'_v + G_v with G = -log(-log u), u from Philox.
__device__ __forceinline__ float exact_score(const float* lg, int v, uint32_t pos, uint32_t b,
                                             uint32_t step_id, uint32_t k0, uint32_t k1, float inv_temp) {
  uint32_t c[4] = {(uint32_t)(v >> 2), pos, b, step_id};
  philox4x32_10(c, k0, k1);
  const float E = -own_log(uniform01(c[v & 3]));
  const float G = -own_log(E);
  return lg[v] * inv_temp + G;
}

template <bool VEC4>
__device__ __forceinline__ void load4(const float* lg, int g, int V, float l4[4]) {
  if (VEC4) {
    const float4 v4 = *reinterpret_cast<const float4*>(lg + 4 * g);
    l4[0] = v4.x; l4[1] = v4.y; l4[2] = v4.z; l4[3] = v4.w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) l4[e] = 4 * g + e < V ? lg[4 * g + e] : 0.f;
  }
}

// grid (Lc, B); one workgroup per canvas position; only masked positions work.
//
// Pass 1: m = max_v l'_v.  Pass 2: the fixed-point normaliser S (exact, every entry)
// and a screening value r_v = exp(l'_v - m) / E_v with E_v = -log u_v from the
// screening log, so log r_v approximates the contract score minus m to within
// ~2e-5 (|logits| < 1e3).  Only entries with r_v >= w * max r (a window of 1e-3 plus
// the rounding of large scores, in log space) can hold the contract argmax; when each
// thread has at most one such entry they are evaluated exactly and compared as
// (score, smaller v); otherwise the row falls back to the exact scan of every entry.
template <bool VEC4>
__global__ __launch_bounds__(256) void sample_kernel(const float* logits, const int32_t* row_map,
                                                     const int32_t* canvas,
                                                     int L, int off, int Lc, int V, int mask_id,
                                                     int pos0, uint32_t step_id, uint32_t k0,
                                                     uint32_t k1, float inv_temp, int32_t* choice,
                                                     float* conf) {
  __shared__ float s_f[4];
  __shared__ float s_score[4];
  __shared__ int s_v[4];
  __shared__ int s_flag[4];
  __shared__ long long s_sum[4];
  const int j = blockIdx.x, b = blockIdx.y;
  const int row = b * Lc + j;
  if (canvas[(size_t)b * L + off + j] != mask_id) {
    if (threadIdx.x == 0) {
      choice[row] = -1;
      conf[row] = -INFINITY;
    }
    return;
  }
  const float* lg = logits + (size_t)(row_map ? row_map[row] : row) * V;
  const uint32_t pos = (uint32_t)(pos0 + off + j);
  const int ngroups = (V + 3) / 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  // ---- pass 1: max scaled logit
  float mx = -INFINITY;
  for (int g = threadIdx.x; g < ngroups; g += 256) {
    float l4[4];
    load4<VEC4>(lg, g, V, l4);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (VEC4 || 4 * g + e < V) mx = fmaxf(mx, l4[e] * inv_temp);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) s_f[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(s_f[0], s_f[1]), fmaxf(s_f[2], s_f[3]));
  __syncthreads();

  // ---- pass 2: exact normaliser, screening values (top two per thread)
  long long S = 0;
  float r1 = 0.f, r2 = 0.f;
  int v1 = 0x7FFFFFFF;
  for (int g = threadIdx.x; g < ngroups; g += 256) {
    float l4[4];
    load4<VEC4>(lg, g, V, l4);
    uint32_t c[4] = {(uint32_t)g, pos, (uint32_t)b, step_id};
    philox4x32_10(c, k0, k1);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int v = 4 * g + e;
      if (!VEC4 && v >= V) break;
      const float ev = own_exp(l4[e] * inv_temp - mx);
      S += (long long)rintf(ev * 1099511627776.0f);  // * 2^40, exact
      const float r = ev * __builtin_amdgcn_rcpf(-screen_log(uniform01(c[e])));
      if (r > r1) {
        r2 = r1;
        r1 = r;
        v1 = v;
      } else if (r > r2) {
        r2 = r;
      }
    }
  }
  float rmax = r1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    S += __shfl_xor(S, o, 64);
    rmax = fmaxf(rmax, __shfl_xor(rmax, o, 64));
  }
  if (lane == 0) {
    s_sum[wave] = S;
    s_f[wave] = rmax;
  }
  __syncthreads();
  rmax = fmaxf(fmaxf(s_f[0], s_f[1]), fmaxf(s_f[2], s_f[3]));
  const float delta = 1e-3f + 2.4e-6f * (fabsf(mx) + 32.f);   // bound on |log r - (score - m)|, x 100
  const float w = 1.f - 2.5f * delta;                           // below exp(-2 delta)
  const bool cand = r1 >= w * rmax;
  // ---- exact decision among candidates (or all entries if a thread has two)
  const int multi = __any(r2 >= w * rmax) ? 1 : 0;
  if (lane == 0) s_flag[wave] = multi;
  __syncthreads();
  const bool slow = s_flag[0] | s_flag[1] | s_flag[2] | s_flag[3];
  Best best{-INFINITY, 0x7FFFFFFF};
  if (!slow) {
    if (cand) best = Best{exact_score(lg, v1, pos, (uint32_t)b, step_id, k0, k1, inv_temp), v1};
  } else {
    for (int g = threadIdx.x; g < ngroups; g += 256) {
      float l4[4];
      load4<VEC4>(lg, g, V, l4);
      uint32_t c[4] = {(uint32_t)g, pos, (uint32_t)b, step_id};
      philox4x32_10(c, k0, k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 4 * g + e;
        if (!VEC4 && v >= V) break;
        const float E = -own_log(uniform01(c[e]));
        const float sc = l4[e] * inv_temp + (-own_log(E));
        if (sc > best.score) best = Best{sc, v};
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const Best other{__shfl_xor(best.score, o, 64), __shfl_xor(best.v, o, 64)};
    best = better(best, other);
  }
  if (lane == 0) {
    s_score[wave] = best.score;
    s_v[wave] = best.v;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    best = Best{s_score[0], s_v[0]};
    for (int k = 1; k < 4; ++k) best = better(best, Best{s_score[k], s_v[k]});
    S = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    if (best.v >= V) best.v = 0;  // only reachable with non-finite logits
    const float lpx = lg[best.v] * inv_temp;
    const float norm = (float)S * 9.094947017729282379150390625e-13f;  // * 2^-40, exact
    choice[row] = best.v;
    conf[row] = (lpx - mx) - own_log(norm);
  }
}

// One workgroup of 1024 threads scans every canvas entry in row-major order.
__global__ __launch_bounds__(1024) void compact_kernel(const int32_t* canvas, int B, int L, int off,
                                                       int mask_id, int32_t* idx, int32_t* row_map,
                                                       int* count) {
  __shared__ int wsum[16];
  __shared__ int base;
  const int Lc = L - off, n = B * Lc;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (threadIdx.x == 0) base = 0;
  __syncthreads();
  for (int c0 = 0; c0 < n; c0 += 1024) {
    const int c = c0 + threadIdx.x;
    const int m = c < n && canvas[(size_t)(c / Lc) * L + off + c % Lc] == mask_id;
    // wave prefix via ballot
    const unsigned long long bal = __ballot(m);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wave] = __popcll(bal);
    __syncthreads();
    int woff = 0;
    for (int w = 0; w < wave; ++w) woff += wsum[w];
    const int r = base + woff + before;
    if (c < n) {
      row_map[c] = m ? r : -1;
      if (m) idx[r] = c;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int t = 0;
      for (int w = 0; w < 16; ++w) t += wsum[w];
      base += t;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *count = base;
}

// one workgroup per row; rank by (conf desc, position asc) among masked positions.
__global__ __launch_bounds__(256) void select_kernel(const int32_t* canvas, const int32_t* choice,
                                                     const float* conf, int L, int off, int Lc,
                                                     int mask_id, int n_unmask, int32_t* next) {
  extern __shared__ float smem[];
  float* sc = smem;
  int* cand = reinterpret_cast<int*>(smem + Lc);
  __shared__ float red[4];
  const int b = blockIdx.x;
  float cnt = 0.f;
  for (int p = threadIdx.x; p < Lc; p += blockDim.x) {
    const int m = canvas[(size_t)b * L + off + p] == mask_id;
    cand[p] = m;
    sc[p] = conf[(size_t)b * Lc + p];
    cnt += (float)m;
  }
  const int n_masked = (int)block_sum(cnt, red);  // exact: counts < 2^24
  const int n = min(n_unmask, n_masked);
  __syncthreads();
  for (int l = threadIdx.x; l < L; l += blockDim.x) {
    int t = canvas[(size_t)b * L + l];
    const int p = l - off;
    if (p >= 0 && p < Lc && cand[p] && n > 0) {
      const float cp = sc[p];
      int rank = 0;
      for (int q = 0; q < Lc; ++q)
        rank += (cand[q] && (sc[q] > cp || (sc[q] == cp && q < p))) ? 1 : 0;
      if (rank < n) t = choice[(size_t)b * Lc + p];
    }
    next[(size_t)b * L + l] = t;
  }
}

}  // namespace

hipError_t compact_masked(const int32_t* canvas, int B, int L, int canvas_off, int mask_id,
                          int32_t* idx, int32_t* row_map, int* count, hipStream_t s) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, s, canvas, B, L, canvas_off, mask_id, idx,
                     row_map, count);
  return hipGetLastError();
}

hipError_t sample_tokens(const float* logits, const int32_t* row_map, const int32_t* canvas, int B,
                         int L, int canvas_off, int V, int mask_id, int pos0, uint32_t step_id,
                         uint64_t seed, float inv_temp, int32_t* choice, float* conf, hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B * Lc == 0) return hipSuccess;
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  const dim3 grid(Lc, B);
  if (V % 4 == 0)
    launch_timed(sample_kernel<true>, grid, dim3(256), 0, s, logits, row_map, canvas, L, canvas_off, Lc, V, mask_id,
                 pos0, step_id, k0, k1, inv_temp, choice, conf);
  else
    launch_timed(sample_kernel<false>, grid, dim3(256), 0, s, logits, row_map, canvas, L, canvas_off, Lc, V,
                 mask_id, pos0, step_id, k0, k1, inv_temp, choice, conf);
  return hipGetLastError();
}

hipError_t select_unmask(const int32_t* canvas, const int32_t* choice, const float* conf, int B, int L,
                         int canvas_off, int mask_id, int n_unmask, int32_t* next, hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(256), (size_t)Lc * 8, s, canvas, choice, conf, L,
                     canvas_off, Lc, mask_id, n_unmask, next);
  return hipGetLastError();
}

}  // namespace tadm
