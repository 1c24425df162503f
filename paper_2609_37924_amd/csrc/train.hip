// Training objective of TADM:Pretraining (Theorem T-ANELBO with gamma = 0, sigma = 0):
// the stale pair (z_t, z_t') of eq. fwd / eq. fwd_t_t' and the 1/t-weighted masked
// cross-entropy of the denoiser's prediction.
//
// Corruption: one uniform u per (row b, position l) -- Philox4x32-10 word 0 at counter
// (2^31 + 3, l, b, step), u = (2 (w >> 9) + 1) 2^-24 -- masks x^l in z_t iff
// u < float((1 - eps) t_b) and in z_t' iff u < float((1 - eps) t'_b) (thresholds in
// double, rounded once), so z_t' is z_t further corrupted with probability
// 1 - alpha_t'/alpha_t per kept position.
#include "common.h"
#include "kernels.h"
#include "sampler_math.h"

namespace tadm {
namespace {

constexpr uint32_t CORRUPT_WORD0 = 0x80000003u;

__global__ void corrupt_kernel(const int32_t* x, int B, int L, const float* t, const float* ts, double keep_scale,
                               uint32_t step, uint32_t k0, uint32_t k1, int mask_id, int32_t* zt, int32_t* zs) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long)B * L) return;
  const int b = (int)(i / L), l = (int)(i % L);
  uint32_t c[4] = {CORRUPT_WORD0, (uint32_t)l, (uint32_t)b, step};
  philox4x32_10(c, k0, k1);
  const float u = uniform01(c[0]);
  const float pt = (float)(keep_scale * (double)t[b]), ps = (float)(keep_scale * (double)ts[b]);
  const int32_t tok = x[i];
  zt[i] = u < pt ? mask_id : tok;
  zs[i] = u < ps ? mask_id : tok;
}

// grid max_rows, 256 threads: row r < *count of the compacted logits is canvas entry
// idx[r]; ce[r] = log sum_v exp(l_v) - l_target, with a fixed reduction order.
__global__ __launch_bounds__(256) void ce_kernel(const float* logits, int V, const int* count, const int32_t* idx,
                                                 const int32_t* x, float* ce) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  if (r >= *count) return;
  const float* lg = logits + (size_t)r * V;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float mx = -INFINITY;
  for (int v = tid; v < V; v += 256) mx = fmaxf(mx, lg[v]);
  mx = wave_max(mx);
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float z = 0.f;
  for (int v = tid; v < V; v += 256) z += expf(lg[v] - mx);
  z = wave_sum(z);
  if (lane == 0) red[wave] = z;
  __syncthreads();
  if (tid == 0) {
    const float zt = (red[0] + red[1]) + (red[2] + red[3]);
    ce[r] = (mx + logf(zt)) - lg[x[idx[r]]];
  }
}

// grid B, 256 threads: loss[b] = (1 / t_b) * sum over masked positions of ce (fixed order)
// and the masked count.
__global__ __launch_bounds__(256) void loss_kernel(const float* ce, const int32_t* row_map, int L, const float* t,
                                                   float* loss, int32_t* n_masked) {
  __shared__ float red[4];
  __shared__ int cnt[4];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float s = 0.f;
  int n = 0;
  for (int l = tid; l < L; l += 256) {
    const int r = row_map[(size_t)b * L + l];
    if (r >= 0) {
      s += ce[r];
      ++n;
    }
  }
  s = wave_sum(s);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) n += __shfl_xor(n, o, 64);
  if (lane == 0) {
    red[wave] = s;
    cnt[wave] = n;
  }
  __syncthreads();
  if (tid == 0) {
    const float tot = (red[0] + red[1]) + (red[2] + red[3]);
    loss[b] = tot * (float)(1.0 / (double)t[b]);
    if (n_masked) n_masked[b] = cnt[0] + cnt[1] + cnt[2] + cnt[3];
  }
}

}  // namespace

hipError_t corrupt_pair(const int32_t* x, int B, int L, const float* t, const float* ts, float eps, uint64_t seed,
                        uint32_t step, int mask_id, int32_t* zt, int32_t* zs, hipStream_t s) {
  const long n = (long)B * L;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(corrupt_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, x, B, L, t, ts,
                     1.0 - (double)eps, step, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), mask_id, zt, zs);
  return hipGetLastError();
}

hipError_t masked_ce(const float* logits, int V, int max_rows, const int* count, const int32_t* idx, const int32_t* x,
                     float* ce, hipStream_t s) {
  if (max_rows == 0) return hipSuccess;
  launch_timed(ce_kernel, dim3(max_rows), dim3(256), 0, s, logits, V, count, idx, x, ce);
  return hipGetLastError();
}

hipError_t weighted_loss(const float* ce, const int32_t* row_map, int B, int L, const float* t, float* loss,
                         int32_t* n_masked, hipStream_t s) {
  hipLaunchKernelGGL(loss_kernel, dim3(B), dim3(256), 0, s, ce, row_map, L, t, loss, n_masked);
  return hipGetLastError();
}

}  // namespace tadm
