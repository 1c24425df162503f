// Vocabulary projection with the reverse step's sampling in its epilogue: the logits
// of the masked rows stay in registers.  A wave's 64 output columns of a row are one
// normaliser group of the sampling contract (64 consecutive vocabulary entries), held
// by the four lanes (lane & 15) + 16 q, q = 0..3.  Per (row, group) the epilogue
// emits the group maximum m_g, the fixed-point sum S_g and the group's exact best
// Gumbel score; sample_finalize merges the groups of a row exactly as the standalone
// sampler merges its own groups, so both paths give the same bits.
//
// This file is compiled with -ffp-contract=off and correctly rounded float32 division
// (the contract arithmetic of sampler_math.h); the MFMA main loop is unaffected.
#include "gemm_kernel.h"
#include "sampler_math.h"

namespace tadm {
namespace {

struct Cand {  // exact score, entry and its scaled logit
  float score;
  int v;
  float lp;
};
__device__ __forceinline__ Cand better_cand(Cand a, Cand b) {
  return (b.score > a.score || (b.score == a.score && b.v < a.v)) ? b : a;
}
__device__ __forceinline__ Cand shfl_cand(Cand c, int o) {
  return Cand{__shfl_xor(c.score, o, 64), __shfl_xor(c.v, o, 64), __shfl_xor(c.lp, o, 64)};
}
__device__ __forceinline__ Cand cand_xor16(Cand c) { return Cand{xor16(c.score), xor16(c.v), xor16(c.lp)}; }
__device__ __forceinline__ Cand cand_xor32(Cand c) { return Cand{xor32(c.score), xor32(c.v), xor32(c.lp)}; }

template <class T>
struct Epi<EPI_SAMPLE, T> {
  static constexpr bool kTile = true;

  // acc[a][b][jj] = C[n = nb + 16 a + 4 (lane >> 4) + jj][m = mb + 16 b + (lane & 15)]
  template <int TN, int TM>
  __device__ __forceinline__ static void tile(const EpiParams& e, const GemmProblem& p, const f32x4 (&acc)[TN][TM],
                                              int mb,
                              int nb, int lane) {
    static_assert(TN * 16 == SAMPLE_GROUP, "one wave column strip must be one normaliser group");
    const int fr = lane & 15, fq = lane >> 4;
    const int g = nb / SAMPLE_GROUP;
#pragma unroll 1
    for (int b = 0; b < TM; ++b) {
      // this row subtile's accumulators, picked with static indices (a runtime index
      // into acc would move the whole tile to scratch)
      f32x4 cb[TN];
#pragma unroll
      for (int a = 0; a < TN; ++a) {
        cb[a] = acc[a][0];
#pragma unroll
        for (int k = 1; k < TM; ++k)
          if (b == k) cb[a] = acc[a][k];
      }
      const int m = mb + 16 * b + fr;
      const bool row_ok = m < p.M;
      const int ci = e.rows_idx[row_ok ? m : 0];
      const uint32_t brow = (uint32_t)(ci / e.Lc), pos = (uint32_t)(e.pos_base + ci % e.Lc);
      float lp[TN][4];
      float mx = -INFINITY;
      const bool whole = nb + TN * 16 <= p.N;  // the strip lies inside the vocabulary
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int n = nb + 16 * a + 4 * fq + jj;
          lp[a][jj] = (whole || n < p.N) ? cb[a][jj] * e.inv_temp : -INFINITY;
          mx = fmaxf(mx, lp[a][jj]);
        }
      mx = fmaxf(mx, xor16(mx));
      mx = fmaxf(mx, xor32(mx));
      // S_g: each rint(exp(l' - m_g) 2^40) <= 2^40 is an integer, so float64 sums of up to
      // 2^13 of them are exact
      double S = 0.0;
      // screening: this lane's two best scores, with the best entry's l' and u
      float a1 = -INFINITY, a2 = -INFINITY, lp1 = 0.f, u1 = 0.5f;
      int v1 = 0x7FFFFFFF;
      // one vocabulary entry; the first loop is for strips wholly inside the vocabulary
      auto entry = [&](float l, float u, int v) {
        S += (double)rintf(own_exp_sel_2p40(l - mx));
        const float sc = screen_score(l, u);
        const bool top = sc > a1;  // selects, not branches: the update runs on every lane
        a2 = top ? a1 : fmaxf(a2, sc);
        a1 = top ? sc : a1;
        v1 = top ? v : v1;
        lp1 = top ? l : lp1;
        u1 = top ? u : u1;
      };
      if (whole) {
#pragma unroll
        for (int a = 0; a < TN; ++a) {
          const int n0 = nb + 16 * a + 4 * fq;
          uint32_t c[4] = {(uint32_t)n0 >> 2, pos, brow, e.step_id};
          philox4x32_10(c, e.k0, e.k1);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) entry(lp[a][jj], uniform01(c[jj]), n0 + jj);
        }
      } else {
#pragma unroll
        for (int a = 0; a < TN; ++a) {
          const int n0 = nb + 16 * a + 4 * fq;
          uint32_t c[4] = {(uint32_t)n0 >> 2, pos, brow, e.step_id};
          philox4x32_10(c, e.k0, e.k1);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            if (n0 + jj < p.N) entry(lp[a][jj], uniform01(c[jj]), n0 + jj);
        }
      }
      S += xor16(S);
      S += xor32(S);
      float amax = fmaxf(a1, xor16(a1));
      amax = fmaxf(amax, xor32(amax));
      const float delta = 1e-3f + 2.4e-6f * (fabsf(mx) + 32.f);  // screening error bound, x 100
      const float wlo = amax - 2.5f * delta;
      int multi = a2 >= wlo ? 1 : 0;
      multi |= xor16(multi);
      multi |= xor32(multi);
      Cand best{-INFINITY, 0x7FFFFFFF, 0.f};
      if (multi) {  // a second entry of some lane is in the window: score the group exactly
#pragma unroll
        for (int a = 0; a < TN; ++a) {
          const int n0 = nb + 16 * a + 4 * fq;
          uint32_t c[4] = {(uint32_t)n0 >> 2, pos, brow, e.step_id};
          philox4x32_10(c, e.k0, e.k1);
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            if (n0 + jj < p.N)
              best = better_cand(best, Cand{exact_score_of(lp[a][jj], uniform01(c[jj])), n0 + jj, lp[a][jj]});
        }
      } else if (a1 >= wlo && v1 < p.N) {
        best = Cand{exact_score_of(lp1, u1), v1, lp1};
      }
      best = better_cand(best, cand_xor16(best));
      best = better_cand(best, cand_xor32(best));
      if (fq == 0 && row_ok && nb < p.N) {
        SamplePart r;
        r.m = mx;
        r.score = best.score;
        r.lp = best.lp;
        r.v = best.v;
        r.S = (long long)S;
        static_cast<SamplePart*>(e.part)[(size_t)m * e.n_groups + g] = r;
      }
    }
  }
};

// groups a finalize thread merges at most (n_groups <= SAMPLE_MAX_VOCAB / 64, 256 threads)
constexpr int FIN_GROUPS = SAMPLE_MAX_VOCAB / 64 / 256;

// grid (Lc, B), 256 threads: one workgroup per canvas position.  A thread reads each of
// its groups' partials once and keeps m_g and S_g in registers for the normaliser pass
// (reading them again missed the L2 for wide rows: 2x the partial bytes fetched).
__global__ __launch_bounds__(256) void finalize_kernel(const SamplePart* part, int n_groups, int V,
                                                       const int32_t* row_map, const int32_t* canvas, int L,
                                                       int off, int Lc, int mask_id, int32_t* choice,
                                                       float* conf) {
  __shared__ float s_m[4];
  __shared__ Cand s_c[4];
  __shared__ long long s_S[4];
  const int j = blockIdx.x, b = blockIdx.y, row = b * Lc + j;
  // not masked, or masked beyond the rows the head computed (row_map -1): not sampled,
  // so the selection leaves it masked; no partial of another step is ever read
  if (canvas[(size_t)b * L + off + j] != mask_id || row_map[row] < 0) {
    if (threadIdx.x == 0) {
      choice[row] = -1;
      conf[row] = -INFINITY;
    }
    return;
  }
  const SamplePart* P = part + (size_t)row_map[row] * n_groups;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float mx = -INFINITY, gm[FIN_GROUPS];
  long long gS[FIN_GROUPS];
  Cand best{-INFINITY, 0x7FFFFFFF, 0.f};
#pragma unroll
  for (int i = 0; i < FIN_GROUPS; ++i) {
    const int g = tid + 256 * i;
    if (g < n_groups) {
      const SamplePart q = P[g];
      gm[i] = q.m;
      gS[i] = q.S;
      mx = fmaxf(mx, q.m);
      best = better_cand(best, Cand{q.score, q.v, q.lp});
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    best = better_cand(best, shfl_cand(best, o));
  }
  if (lane == 0) {
    s_m[wave] = mx;
    s_c[wave] = best;
  }
  __syncthreads();
  mx = fmaxf(fmaxf(s_m[0], s_m[1]), fmaxf(s_m[2], s_m[3]));
  long long S = 0;
#pragma unroll
  for (int i = 0; i < FIN_GROUPS; ++i)
    if (tid + 256 * i < n_groups) S += (long long)rintf((float)gS[i] * own_exp(gm[i] - mx));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) S += __shfl_xor(S, o, 64);
  if (lane == 0) s_S[wave] = S;
  __syncthreads();
  if (tid == 0) {
    best = s_c[0];
    for (int k = 1; k < 4; ++k) best = better_cand(best, s_c[k]);
    S = s_S[0] + s_S[1] + s_S[2] + s_S[3];
    if (best.v >= V) best = Cand{0.f, 0, 0.f};  // only reachable with non-finite logits
    const float norm = (float)S * 9.094947017729282379150390625e-13f;  // * 2^-40, exact
    choice[row] = best.v;
    conf[row] = (best.lp - mx) - own_log(norm);
  }
}

}  // namespace

hipError_t head_sample(const GemmProblem& p, const EpiParams& e, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  // Large vocabularies: 128 x 128 tiles on 2 x 2 waves (64 x 64 per wave, a third less
  // LDS traffic per product), two blocks per CU; 26B-class head (V = 262144): 507 -> 407
  // ms per generation against the tiles below.  Smaller ones: 128 x 64 tiles on 4 x 1
  // waves, three blocks per CU (48 KB of LDS each), so that a block's VALU-heavy
  // epilogue overlaps the others' MFMA main loops (1 % ahead on V = 32768).
  if (p.N >= 40000) return launch_bf16<128, 128, 2, 2, 2, 2, EPI_SAMPLE>(p, e, s);
  return launch_bf16<128, 64, 2, 4, 1, 3, EPI_SAMPLE>(p, e, s);
}

hipError_t sample_finalize(const SamplePart* part, int n_groups, int V, const int32_t* row_map,
                           const int32_t* canvas, int B, int L, int canvas_off, int mask_id, int32_t* choice,
                           float* conf, hipStream_t s) {
  const int Lc = L - canvas_off;
  if (B * Lc == 0) return hipSuccess;
  if (n_groups > FIN_GROUPS * 256) return hipErrorInvalidValue;
  launch_timed(finalize_kernel, dim3(Lc, B), dim3(256), 0, s, part, n_groups, V, row_map, canvas, L, canvas_off, Lc,
               mask_id, choice, conf);
  return hipGetLastError();
}

}  // namespace tadm
