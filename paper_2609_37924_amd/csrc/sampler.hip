// Masked-diffusion reverse step: Gumbel-max sampling with fixed-point confidence and
// confidence-ranked unmasking (MDLM zero-masking and carry-over, sigma_t = 0).
//
// Determinism contract (token choices and unmask order are reproducible bit for bit
// by any IEEE float32 implementation of the same operations):
//  * Philox4x32-10 (Salmon et al., SC'11): counter (v/4, position, row, step id),
//    key (seed low word, seed high word); word v%4 -> u = (2*(x>>9)+1) * 2^-24.
//  * Own float32 log / exp (sampler_math.h) built only from individually rounded
//    +,-,*,/; this file is compiled with -ffp-contract=off and correctly rounded
//    float32 division.
//  * token = argmax_v (l_v * inv_temp + G_v), G = -log(-log u), ties to smaller v;
//  * confidence = (l'_x - m) - log(float(S) * 2^-40) with the normaliser in 2^-40 fixed
//    point over groups of 64 entries: m_g = max of group g, S_g = sum_{v in g}
//    rint(exp(l'_v - m_g) 2^40), S = sum_g rint(float(S_g) exp(m_g - m)); every sum is
//    over integers, so any reduction order (and any tiling) gives the same bits.
//  * ranking: confidence descending, then position ascending.
#include <cfloat>

#include "common.h"
#include "kernels.h"
#include "sampler_math.h"

#pragma clang fp contract(off)

namespace tadm {
namespace {

// Exact contract score of entry v of a logits row.
__device__ __forceinline__ float exact_score(const float* lg, int v, uint32_t pos, uint32_t b,
                                             uint32_t step_id, uint32_t k0, uint32_t k1, float inv_temp) {
  uint32_t c[4] = {(uint32_t)(v >> 2), pos, b, step_id};
  philox4x32_10(c, k0, k1);
  return exact_score_of(lg[v] * inv_temp, uniform01(c[v & 3]));
}

constexpr int GROUP = SAMPLE_GROUP;  // one normaliser group: 16 lanes x 4 entries
constexpr int CHUNK = 1024;     // entries per block pass: 256 threads x 4
constexpr int UNROLL = 4;       // chunks whose loads are in flight together

// grid (Lc, B), 256 threads; one workgroup per canvas position, only masked positions
// work.  One pass over the row's logits: lanes 16k..16k+15 of a wave hold the 64
// entries of one group, reduce its maximum m_g and its fixed-point sum S_g (int64,
// exact) with lane shuffles and park them in LDS; each thread also keeps its two best
// screening scores.  Afterwards m = max m_g, S = sum_g rint(float(S_g) exp(m_g - m))
// (exact integer sum).  The contract argmax is within 2.5 delta of the best screening
// score (delta bounds the screening error, with a wide margin); when no thread has
// a second entry in that window the threads' best entries are the only candidates and
// are scored exactly, otherwise every entry is scored exactly in a second pass.
// Dynamic LDS: ceil(V / 64) x (float + int64).
__global__ __launch_bounds__(256) void sample_kernel(const float* logits, const int32_t* row_map,
                                                     const NucleusThr* thr, const int32_t* canvas, int L, int off,
                                                     int Lc, int V, int mask_id, int pos0, uint32_t step_id, uint32_t k0,
                                                     uint32_t k1, float inv_temp, int32_t* choice,
                                                     float* conf) {
  extern __shared__ long long s_dyn[];
  __shared__ float s_f[4];
  __shared__ float s_score[4];
  __shared__ int s_v[4];
  __shared__ int s_flag[4];
  __shared__ long long s_sum[4];
  const int j = blockIdx.x, b = blockIdx.y;
  const int row = b * Lc + j;
  // not masked, or masked without a logits row (beyond the rows computed): not sampled
  if (canvas[(size_t)b * L + off + j] != mask_id || (row_map && row_map[row] < 0)) {
    if (threadIdx.x == 0) {
      choice[row] = -1;
      conf[row] = -INFINITY;
    }
    return;
  }
  const int ng = (V + GROUP - 1) / GROUP;
  long long* s_S = s_dyn;
  float* s_m = reinterpret_cast<float*>(s_dyn + ng);
  const float* lg = logits + (size_t)(row_map ? row_map[row] : row) * V;
  const uint32_t pos = (uint32_t)(pos0 + off + j);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool vec = (V & 3) == 0;
  const int nchunk = (V + CHUNK - 1) / CHUNK;
  // nucleus: entry v takes part iff rint(exp(l'_v - nm) 2^40) >= ntau
  const bool nuc = thr != nullptr;
  const float nm = nuc ? thr[row].m : 0.f;
  const float y_in = nuc ? thr[row].y_in : -INFINITY, y_out = nuc ? thr[row].y_out : -INFINITY;
  const long long ntau = nuc ? thr[row].tau : 0;
  auto in_nucleus = [&](float lp) {
    const float y = lp - nm;
    if (y >= y_in) return true;
    if (y < y_out) return false;
    return (long long)rintf(own_exp(y) * 1099511627776.0f) >= ntau;
  };

  Top2 top;
  for (int c0 = 0; c0 < nchunk; c0 += UNROLL) {
    float l[UNROLL][4];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {  // issue every load first
      const int v0 = (c0 + u) * CHUNK + 4 * tid;
      if (vec && v0 + 3 < V) {
        const float4 x = *reinterpret_cast<const float4*>(lg + v0);
        l[u][0] = x.x; l[u][1] = x.y; l[u][2] = x.z; l[u][3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) l[u][e] = v0 + e < V ? lg[v0 + e] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      const int c = c0 + u;
      if (c >= nchunk) break;  // uniform over the block
      const int q = c * (CHUNK / 4) + tid;  // float4 index = Philox counter word 0
      const int g = q / (GROUP / 4);
      float lp[4];
      float mx = -INFINITY;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lp[e] = 4 * q + e < V ? l[u][e] * inv_temp : -INFINITY;
        mx = fmaxf(mx, lp[e]);
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      long long sg = 0;
      if (g < ng) {  // four integer terms below 2^41: exact in float64, converted once
        double sd = 0.0;
#pragma unroll
        for (int e = 0; e < 4; ++e) sd += (double)rintf(own_exp(lp[e] - mx) * 1099511627776.0f);  // * 2^40
        sg = (long long)sd;
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) sg += __shfl_xor(sg, o, 64);
      if ((lane & 15) == 0 && g < ng) {
        s_S[g] = sg;
        s_m[g] = mx;
      }
      uint32_t ctr[4] = {(uint32_t)q, pos, (uint32_t)b, step_id};
      philox4x32_10(ctr, k0, k1);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (4 * q + e < V && in_nucleus(lp[e])) top.add(screen_score(lp[e], uniform01(ctr[e])), 4 * q + e);
    }
  }
  __syncthreads();

  // m = max_g m_g; S = sum_g rint(float(S_g) * exp(m_g - m))
  float mx = -INFINITY;
  for (int g = tid; g < ng; g += 256) mx = fmaxf(mx, s_m[g]);
  float amax = top.a1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    amax = fmaxf(amax, __shfl_xor(amax, o, 64));
  }
  if (lane == 0) {
    s_f[wave] = mx;
    s_score[wave] = amax;
  }
  __syncthreads();
  mx = fmaxf(fmaxf(s_f[0], s_f[1]), fmaxf(s_f[2], s_f[3]));
  amax = fmaxf(fmaxf(s_score[0], s_score[1]), fmaxf(s_score[2], s_score[3]));
  long long S = 0;
  for (int g = tid; g < ng; g += 256)
    S += (long long)rintf((float)s_S[g] * own_exp(s_m[g] - mx));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o, 64);
  const float delta = 1e-3f + 2.4e-6f * (fabsf(mx) + 32.f);  // screening error bound, x 100
  const float lo = amax - 2.5f * delta;
  const int multi = __any(top.a2 >= lo) ? 1 : 0;
  __syncthreads();  // every wave has read s_f / s_score
  if (lane == 0) {
    s_sum[wave] = S;
    s_flag[wave] = multi;
  }
  __syncthreads();
  const bool slow = s_flag[0] | s_flag[1] | s_flag[2] | s_flag[3];
  Best best{-INFINITY, 0x7FFFFFFF};
  if (!slow) {
    if (top.a1 >= lo && top.v1 < V) best = Best{exact_score(lg, top.v1, pos, (uint32_t)b, step_id, k0, k1, inv_temp), top.v1};
  } else {
    for (int q = tid; 4 * q < V; q += 256) {
      uint32_t ctr[4] = {(uint32_t)q, pos, (uint32_t)b, step_id};
      philox4x32_10(ctr, k0, k1);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int v = 4 * q + e;
        if (v >= V) break;
        const float lpv = lg[v] * inv_temp;
        if (!in_nucleus(lpv)) continue;
        const float sc = exact_score_of(lpv, uniform01(ctr[e]));
        if (sc > best.score) best = Best{sc, v};
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const Best other{__shfl_xor(best.score, o, 64), __shfl_xor(best.v, o, 64)};
    best = better(best, other);
  }
  __syncthreads();
  if (lane == 0) {
    s_score[wave] = best.score;
    s_v[wave] = best.v;
  }
  __syncthreads();
  if (tid == 0) {
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

// grid (Lc, B), NUC_THREADS threads: the nucleus threshold of each masked position.
// Weights q_v = rint(exp(l'_v - m) 2^40) (int64), Q = sum q_v, target = ceil(top_p Q) (exact,
// in 128-bit integers); tau is found by four radix passes over the 41-bit weights (digits of
// 11, 11, 11 and 8 bits, high to low): each pass sums, per digit, the weights of the entries
// that share the digits chosen so far, and keeps the highest digit at which the weights
// above plus that digit's reach the target.  All sums are integers: any order, same tau.
// The first pass also accumulates Q.  Digit 0 collects every small weight of a pass (most
// of the vocabulary), so it is not accumulated by atomics: its sum is the pass's total (Q,
// then the previous pass's chosen digit's sum) minus the other digits'.
// A weight is held as the float w = rint(exp(l'_v - m) 2^40), an integer below 2^41 with
// 24 significant bits, so its digits and prefixes are exact float operations:
// floor(w 2^-s) is q >> s, and floor(w 2^-s) - floor(w 2^-(s+b)) 2^b is its b-bit digit.
// PER > 0: V <= NUC_THREADS * PER and V % 4 == 0; each thread keeps the weights of its PER
// entries in registers, read once as float4.  PER = 0: every pass recomputes them.
constexpr int NUC_THREADS = 1024;
template <int PER>
__global__ __launch_bounds__(NUC_THREADS) void nucleus_kernel(const float* logits, const int32_t* row_map,
                                                              const int32_t* canvas, int L, int off, int Lc, int V,
                                                              int mask_id, float inv_temp, float top_p,
                                                              NucleusThr* thr) {
  constexpr int NW = NUC_THREADS / 64;
  constexpr bool CACHED = PER > 0;
  constexpr int NE = CACHED ? PER : 1;
  constexpr float TWO40 = 1099511627776.0f;
  __shared__ unsigned long long hist[2048];
  __shared__ float s_f[NW];
  __shared__ unsigned long long s_u[NW];
  __shared__ unsigned long long s_sel[3];
  const int j = blockIdx.x, b = blockIdx.y, row = b * Lc + j;
  if (canvas[(size_t)b * L + off + j] != mask_id || (row_map && row_map[row] < 0)) return;
  const float* lg = logits + (size_t)(row_map ? row_map[row] : row) * V;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // cached entry i of this thread: v = 4 (tid + NUC_THREADS (i / 4)) + i % 4
  auto vof = [&](int i) { return 4 * (tid + NUC_THREADS * (i >> 2)) + (i & 3); };

  float ev[NE];  // l'_v, then the weight w_v
  float mx = -INFINITY;
  if constexpr (CACHED) {
#pragma unroll
    for (int i = 0; i < NE; i += 4) {
      const float4 x = vof(i) < V ? *reinterpret_cast<const float4*>(lg + vof(i))
                                  : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
      ev[i] = x.x * inv_temp;
      ev[i + 1] = x.y * inv_temp;
      ev[i + 2] = x.z * inv_temp;
      ev[i + 3] = x.w * inv_temp;
      mx = fmaxf(mx, fmaxf(fmaxf(ev[i], ev[i + 1]), fmaxf(ev[i + 2], ev[i + 3])));
    }
  } else {
    for (int v = tid; v < V; v += NUC_THREADS) mx = fmaxf(mx, lg[v] * inv_temp);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) s_f[wave] = mx;
  __syncthreads();
  mx = s_f[0];
  for (int w = 1; w < NW; ++w) mx = fmaxf(mx, s_f[w]);
  if constexpr (CACHED) {
#pragma unroll
    for (int i = 0; i < NE; i += 4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) ev[i + e] = rintf(own_exp_sel(ev[i + e] - mx) * TWO40);  // padding: 0
      asm volatile("" : "+v"(ev[i]), "+v"(ev[i + 1]), "+v"(ev[i + 2]), "+v"(ev[i + 3])::"memory");
    }
  }
  // calls f(w) for every entry of the row (the cached padding entries have w = 0)
  auto for_each_weight = [&](auto f) {
    if constexpr (CACHED) {
#pragma unroll
      for (int i = 0; i < NE; i += 4) {
        // four entries at a time, in order: fresh copies per pass (the int64 conversions are
        // not kept live across passes) and a barrier per group (bounded temporaries)
        float w0 = ev[i], w1 = ev[i + 1], w2 = ev[i + 2], w3 = ev[i + 3];
        asm volatile("" : "+v"(w0), "+v"(w1), "+v"(w2), "+v"(w3)::"memory");
        f(w0);
        f(w1);
        f(w2);
        f(w3);
      }
    } else {
      for (int v = tid; v < V; v += NUC_THREADS) f(rintf(own_exp(lg[v] * inv_temp - mx) * TWO40));
    }
  };

  // first pass: Q and the top 11-bit digit (q >> 30) of every weight
  for (int i = tid; i < 2048; i += NUC_THREADS) hist[i] = 0;
  __syncthreads();
  unsigned long long Q = 0;
  for_each_weight([&](float w) {
    const unsigned long long q = (unsigned long long)w;
    Q += q;
    const int d = (int)(w * 0x1p-30f);  // truncation = floor (w >= 0)
    if (d != 0) atomicAdd(&hist[d], q);
  });
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) Q += __shfl_xor(Q, o, 64);
  if (lane == 0) s_u[wave] = Q;
  __syncthreads();
  Q = 0;
  for (int w = 0; w < NW; ++w) Q += s_u[w];
  // target = ceil(top_p Q): top_p = mant 2^-sh with a 24-bit integer mant (normal, < 1)
  const uint32_t pb = __float_as_uint(top_p);
  const unsigned long long mant = (pb & 0x7FFFFFu) | 0x800000u;
  const int sh = 150 - (int)((pb >> 23) & 0xFF);
  const unsigned __int128 prod = (unsigned __int128)mant * Q;  // < 2^82
  const unsigned long long target =
      sh >= 100 ? 1ull : (unsigned long long)((prod + (((unsigned __int128)1 << sh) - 1)) >> sh);

  unsigned long long prefix = 0, above = 0, total = Q;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int shk = k == 0 ? 30 : k == 1 ? 19 : k == 2 ? 8 : 0, bk = k == 3 ? 8 : 11;
    const int nb = 1 << bk;
    if (k > 0) {  // histogram of digit k over the weights whose higher digits equal prefix
      const float top_scale = __uint_as_float((uint32_t)(127 - shk - bk) << 23);  // 2^-(shk + bk)
      const float dig_scale = __uint_as_float((uint32_t)(127 - shk) << 23);       // 2^-shk
      const float pre_f = (float)prefix;  // exact: the prefix of an existing weight
      const float base = (float)(1 << bk);
      for_each_weight([&](float w) {
        const float hi = floorf(w * top_scale);
        if (hi == pre_f) {
          const int d = (int)(floorf(w * dig_scale) - hi * base);
          if (d != 0) atomicAdd(&hist[d], (unsigned long long)w);
        }
      });
      __syncthreads();
    }
    if (wave == 0) {  // lane l owns digits [l c, (l + 1) c); suffix sums over lanes, high to low
      const int c = nb / 64;
      unsigned long long own = 0;
      for (int i = 0; i < c; ++i) own += hist[lane * c + i];
      unsigned long long rest = own;  // digits 1.. of the pass
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) rest += __shfl_xor(rest, o, 64);
      if (lane == 0) {  // digit 0 is the remainder of the pass's total
        hist[0] = total - rest;
        own += total - rest;
      }
      unsigned long long suf = own;  // sum over this lane's digits and every higher lane's
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned long long t = __shfl_down(suf, o, 64);
        if (lane + o < 64) suf += t;
      }
      const unsigned long long higher = above + (suf - own);  // weight in digits above this lane's
      if (higher < target && higher + own >= target) {
        unsigned long long acc = higher;
        for (int d = lane * c + c - 1; d >= lane * c; --d) {
          if (acc + hist[d] >= target) {
            s_sel[0] = (unsigned long long)d;
            s_sel[1] = acc;
            s_sel[2] = hist[d];
            break;
          }
          acc += hist[d];
        }
      }
    }
    __syncthreads();
    prefix = (prefix << bk) | s_sel[0];
    above = s_sel[1];
    total = s_sel[2];
    if (k < 3) {
      const int nb_next = k == 2 ? 256 : 2048;
      for (int i = tid; i < nb_next; i += NUC_THREADS) hist[i] = 0;
    }
    __syncthreads();
  }
  if (tid == 0) {
    // exp(y) >= (tau + 1/2) 2^-40 e^(1e-4) makes the float32 weight round to >= tau; below
    // (tau - 1/2) 2^-40 e^(-1e-4) it rounds below tau (the float32 exponential and the
    // rounding of y = l' - m are within 1e-5 relative of exp(y))
    const double t = (double)prefix;
    const float y_in = (float)(log((t + 0.5) * 0x1p-40) + 1e-4);
    const float y_out = t > 0.5 ? (float)(log((t - 0.5) * 0x1p-40) - 1e-4) : -INFINITY;
    thr[row] = NucleusThr{mx, y_in, y_out, 0, (long long)prefix};
  }
}

// One workgroup of 1024 threads scans every canvas entry in row-major order.
// Masked canvas positions in order get rows 0, 1, ... (idx: row -> position, row_map:
// position -> row or -1); rows from `bound` on are not assigned (row_map -1): a caller
// that sized its work for `bound` rows never reads a row it did not compute.
__global__ __launch_bounds__(1024) void compact_kernel(const int32_t* canvas, int B, int L, int off,
                                                       int mask_id, int bound, int32_t* idx, int32_t* row_map,
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
      const bool kept = m && r < bound;
      row_map[c] = kept ? r : -1;
      if (kept) idx[r] = c;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int t = 0;
      for (int w = 0; w < 16; ++w) t += wsum[w];
      base += t;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *count = min(base, bound);
}

// One workgroup of 1024 threads per row; rank by (conf desc, position asc) among the
// masked positions.  The row's confidences go to LDS with -inf for entries that are not
// masked (a finite confidence never ranks below them); four threads share a position,
// each counting the better entries in a quarter of the row with float4 reads, and
// lanes 4k..4k+3 add their counts.  One workgroup per row keeps the update in place:
// every canvas read of the row happens before the barrier, and each position is written
// only by its own threads.
constexpr int SELECT_THREADS = 1024;
__global__ __launch_bounds__(SELECT_THREADS) void select_kernel(const int32_t* canvas, const int32_t* choice,
                                                                const float* conf, int L, int off, int Lc,
                                                                int mask_id, int n_unmask,
                                                                const int32_t* n_rows, int32_t* next) {
  extern __shared__ float sc[];  // Lc rounded up to a multiple of 16, padded with -inf
  __shared__ float red[SELECT_THREADS / 64];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int Lc16 = (Lc + 15) & ~15, quarter = Lc16 / 4;  // each quarter: whole float4s
  float cnt = 0.f;
  // the candidates are the masked positions that were sampled (choice >= 0); a
  // candidate's confidence is at least -FLT_MAX, so it ranks ahead of every other slot
  for (int p = tid; p < Lc16; p += SELECT_THREADS) {
    const bool m = p < Lc && canvas[(size_t)b * L + off + p] == mask_id && choice[(size_t)b * Lc + p] >= 0;
    sc[p] = m ? fmaxf(conf[(size_t)b * Lc + p], -FLT_MAX) : -INFINITY;
    cnt += m ? 1.f : 0.f;
  }
  const int n_masked = (int)block_sum(cnt, red);  // exact: counts < 2^24; ends with a barrier
  const int n = min(n_rows ? max(n_rows[b], 0) : n_unmask, n_masked);
  const int sub = tid & 3;
  for (int l0 = 0; l0 < L; l0 += SELECT_THREADS / 4) {
    const int l = l0 + (tid >> 2), p = l - off;
    const bool mine = l < L;
    const int t = mine ? canvas[(size_t)b * L + l] : 0;
    const bool cand = mine && p >= 0 && p < Lc && t == mask_id && n > 0 && sc[p] != -INFINITY;
    int rank = 0;
    if (__any(cand)) {
      const float cp = cand ? sc[p] : 0.f;
      for (int q = sub * quarter; q < (sub + 1) * quarter; q += 4) {
        const float4 v = *reinterpret_cast<const float4*>(sc + q);
        rank += (v.x > cp || (v.x == cp && q < p)) + (v.y > cp || (v.y == cp && q + 1 < p)) +
                (v.z > cp || (v.z == cp && q + 2 < p)) + (v.w > cp || (v.w == cp && q + 3 < p));
      }
      rank += __shfl_xor(rank, 1, 64);
      rank += __shfl_xor(rank, 2, 64);
    }
    if (mine && sub == 0) next[(size_t)b * L + l] = (cand && rank < n) ? choice[(size_t)b * Lc + p] : t;
  }
}

// grid (ceil(L / 256), B): one thread per canvas entry; in place (each entry is read and
// written by its own thread).
__global__ __launch_bounds__(256) void remask_kernel(const int32_t* canvas, const int32_t* choice, int L, int off,
                                                     int mask_id, int pos0, uint32_t step_id, uint32_t k0,
                                                     uint32_t k1, float p_unmask, float sigma, int32_t* next) {
  const int l = blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;
  if (l >= L) return;
  const int t = canvas[(size_t)b * L + l];
  int nt = t;
  if (l >= off) {
    const int j = l - off, Lc = L - off;
    uint32_t c[4] = {0x80000000u, (uint32_t)(pos0 + l), (uint32_t)b, step_id};
    philox4x32_10(c, k0, k1);
    const float u = uniform01(c[0]);
    if (t == mask_id)
      nt = u < p_unmask ? choice[(size_t)b * Lc + j] : mask_id;
    else if (u < sigma)
      nt = mask_id;
  }
  next[(size_t)b * L + l] = nt;
}

}  // namespace

hipError_t remask_update(const int32_t* canvas, const int32_t* choice, int B, int L, int canvas_off, int mask_id,
                         int pos0, uint32_t step_id, uint64_t seed, float p_unmask, float sigma, int32_t* next,
                         hipStream_t s) {
  if (B * L == 0) return hipSuccess;
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  hipLaunchKernelGGL(remask_kernel, dim3((L + 255) / 256, B), dim3(256), 0, s, canvas, choice, L, canvas_off, mask_id,
                     pos0, step_id, k0, k1, p_unmask, sigma, next);
  return hipGetLastError();
}

hipError_t compact_masked(const int32_t* canvas, int B, int L, int canvas_off, int mask_id, int bound,
                          int32_t* idx, int32_t* row_map, int* count, hipStream_t s) {
  hipLaunchKernelGGL(compact_kernel, dim3(1), dim3(1024), 0, s, canvas, B, L, canvas_off, mask_id, bound, idx,
                     row_map, count);
  return hipGetLastError();
}

hipError_t nucleus_thresholds(const float* logits, const int32_t* row_map, const int32_t* canvas, int B, int L,
                              int canvas_off, int V, int mask_id, float inv_temp, float top_p, NucleusThr* thr,
                              hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B * Lc == 0) return hipSuccess;
  auto kernel = nucleus_kernel<0>;
  if (V % 4 == 0 && V <= NUC_THREADS * 32) kernel = V <= NUC_THREADS * 16 ? nucleus_kernel<16> : nucleus_kernel<32>;
  hipLaunchKernelGGL(kernel, dim3(Lc, B), dim3(NUC_THREADS), 0, s, logits, row_map, canvas, L, canvas_off, Lc, V,
                     mask_id, inv_temp, top_p, thr);
  return hipGetLastError();
}

hipError_t sample_tokens(const float* logits, const int32_t* row_map, const NucleusThr* thr, const int32_t* canvas,
                         int B, int L, int canvas_off, int V, int mask_id, int pos0, uint32_t step_id,
                         uint64_t seed, float inv_temp, int32_t* choice, float* conf, hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B * Lc == 0) return hipSuccess;
  if (V > SAMPLE_MAX_VOCAB) return hipErrorInvalidValue;
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  const uint32_t lds = (uint32_t)(((V + GROUP - 1) / GROUP) * (sizeof(long long) + sizeof(float)));
  launch_timed(sample_kernel, dim3(Lc, B), dim3(256), lds, s, logits, row_map, thr, canvas, L, canvas_off, Lc, V,
               mask_id, pos0, step_id, k0, k1, inv_temp, choice, conf);
  return hipGetLastError();
}

hipError_t select_unmask(const int32_t* canvas, const int32_t* choice, const float* conf, int B, int L,
                         int canvas_off, int mask_id, int n_unmask, const int32_t* n_rows, int32_t* next,
                         hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B == 0) return hipSuccess;
  hipLaunchKernelGGL(select_kernel, dim3(B), dim3(SELECT_THREADS), (size_t)((Lc + 15) & ~15) * 4, s, canvas, choice,
                     conf, L, canvas_off, Lc, mask_id, n_unmask, n_rows, next);
  return hipGetLastError();
}

}  // namespace tadm
