// Dense contractions of the TADM step: C = A W^T with fused epilogues.
//
// bf16 operands run on the MFMA kernel template of gemm_kernel.h with the epilogues
// below; the tile shape is picked per call from the number of blocks it yields.
// float32 operands (small fp32 models) run on a register-blocked VALU kernel with
// the same epilogues.
#include "gemm_kernel.h"

namespace tadm {
namespace {

// ------------------------------------------------------------------ epilogues

template <class T>
struct Epi<EPI_STORE, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, v[0], v[1], v[2], v[3]);
  }
};
template <class T>
struct Epi<EPI_STORE_F32, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    store4(static_cast<float*>(e.out) + (size_t)m * e.ldo + n, v[0], v[1], v[2], v[3]);
  }
};
template <class T>
struct Epi<EPI_SCALE_F32, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float r = e.row1[m];
    store4(static_cast<float*>(e.out) + (size_t)m * e.ldo + n, r * v[0], r * v[1], r * v[2], r * v[3]);
  }
};
template <class T>
struct Epi<EPI_RESID, T> {
  static constexpr bool kGlu = false;
  static constexpr int kPre = 1;
  __device__ static void pre(const EpiParams& e, int m, int n, float4* o) {
    o[0] = *reinterpret_cast<const float4*>(e.resid + (size_t)m * e.ldr + n);
  }
  __device__ static void apply_pre(const EpiParams& e, int m, int n, f32x4 v, const float4* o) {
    float4 x = o[0];
    x.x += v[0]; x.y += v[1]; x.z += v[2]; x.w += v[3];
    *reinterpret_cast<float4*>(e.resid + (size_t)m * e.ldr + n) = x;
  }
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    float4 o;
    pre(e, m, n, &o);
    apply_pre(e, m, n, v, &o);
  }
};
template <class T>
struct Epi<EPI_GELU, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, gelu_act<T>(v[0]), gelu_act<T>(v[1]),
           gelu_act<T>(v[2]), gelu_act<T>(v[3]));
  }
};
template <class T>
struct Epi<EPI_FUSION1, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
    if (n < e.split) {
      store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, gelu_act<T>(v[0] + b.x),
             gelu_act<T>(v[1] + b.y), gelu_act<T>(v[2] + b.z), gelu_act<T>(v[3] + b.w));
    } else {
      store4(e.out2 + (size_t)m * e.ldo2 + (n - e.split), sigmoid_act<T>(v[0] + b.x),
             sigmoid_act<T>(v[1] + b.y), sigmoid_act<T>(v[2] + b.z), sigmoid_act<T>(v[3] + b.w));
    }
  }
};
template <class T>
struct Epi<EPI_FUSION2, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
    const float4 h = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
    const float4 g = *reinterpret_cast<const float4*>(e.gate + (size_t)m * e.ldg + n);
    store4(e.resid + (size_t)m * e.ldr + n, h.x + g.x * (v[0] + b.x), h.y + g.y * (v[1] + b.y),
           h.z + g.z * (v[2] + b.z), h.w + g.w * (v[3] + b.w));
  }
};
template <class T>
struct Epi<EPI_SILU, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, silu_act<T>(v[0]), silu_act<T>(v[1]),
           silu_act<T>(v[2]), silu_act<T>(v[3]));
  }
};
template <class T>
struct Epi<EPI_ADD_F32, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 a = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
    store4(static_cast<float*>(e.out) + (size_t)m * e.ldo + n, a.x + v[0], a.y + v[1], a.z + v[2],
           a.w + v[3]);
  }
};
template <class T>
struct Epi<EPI_ADD_BOTH, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 a = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
    const float r0 = a.x + v[0], r1 = a.y + v[1], r2 = a.z + v[2], r3 = a.w + v[3];
    store4(static_cast<float*>(e.out) + (size_t)m * e.ldo + n, r0, r1, r2, r3);
    store4(static_cast<T*>(e.out_t) + (size_t)m * e.ld_out_t + n, r0, r1, r2, r3);
  }
};
template <class T>
struct Epi<EPI_ADD_SUB, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 a = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
    const float4 b = *reinterpret_cast<const float4*>(e.aux2 + (size_t)m * e.ld_aux2 + n);
    store4(static_cast<T*>(e.out_t) + (size_t)m * e.ld_out_t + n, (a.x + v[0]) - b.x, (a.y + v[1]) - b.y,
           (a.z + v[2]) - b.z, (a.w + v[3]) - b.w);
  }
};
template <class T>
struct Epi<EPI_PAIRED, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 h = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
    const float f = e.row1[m] * e.row2[m];
    store4(static_cast<float*>(e.out) + (size_t)m * e.ldo + n, h.x + f * v[0], h.y + f * v[1],
           h.z + f * v[2], h.w + f * v[3]);
  }
};
template <class T>
struct Epi<EPI_QKV_ROPE, T> {
  static constexpr bool kGlu = false;
  static constexpr bool kTileLds = true;  // bf16 kernel: staged through LDS (tile_lds)
  __device__ static int fdiv(int n, uint32_t mul, int shift) {
    return (int)((__umulhi((uint32_t)n, mul) + (uint32_t)n) >> shift);
  }
  // one 4-feature fragment, stored directly (float32 kernel, and head widths whose
  // slots a wave strip does not tile)
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const int b = fdiv(m, e.l_mul, e.l_shift), l = m - b * e.L;
    const int slot = fdiv(n, e.dh_mul, e.dh_shift), c = n - slot * e.dh;  // c is a multiple of 4
    if (slot < e.H + e.Hkv) {
      // (v0, v1) = pair j, (v2, v3) = pair j + 1 with j = c / 2
      const int j = c >> 1, half = e.dh >> 1;
      // (cos j, sin j, cos j+1, sin j+1): j is even, so the load is 16-byte aligned
      const float4 r = *reinterpret_cast<const float4*>(e.rope + ((size_t)(e.pos0 + l) * half + j) * 2);
      const float a0 = v[0] * r.x - v[1] * r.y, b0 = v[1] * r.x + v[0] * r.y;
      const float a1 = v[2] * r.z - v[3] * r.w, b1 = v[3] * r.z + v[2] * r.w;
      T* row = slot < e.H
                   ? static_cast<T*>(e.q) + (((size_t)b * e.H + slot) * e.L + l) * e.dh
                   : static_cast<T*>(e.k) + (((size_t)b * e.Hkv + (slot - e.H)) * e.kv_cap + e.kv_off + l) * e.dh;
      store2(row + j, a0, a1);  // j is even: 4-byte (bf16) or 8-byte (float) aligned pairs
      store2(row + j + half, b0, b1);
    } else {
      T* col = static_cast<T*>(e.vt) + (((size_t)b * e.Hkv + (slot - e.H - e.Hkv)) * e.dh + c) * e.kv_cap +
               e.kv_off + l;
#pragma unroll
      for (int t = 0; t < 4; ++t) col[(size_t)t * e.kv_cap] = from_f32<T>(v[t]);
    }
  }

  // Byte offset of element (r, col) of a [rows][C] bf16 staging tile: the 16-byte chunks
  // of row r rotated by r + r / 8, so that the fragment writes (16 rows of one chunk)
  // and the chunk reads (whole rows) meet distinct LDS banks.
  template <int C>
  __device__ static int staged(int r, int col) {
    constexpr int NCH = C / 8;
    return r * (C * 2) + (((col >> 3) + r + (r >> 3)) % NCH) * 16 + (col & 7) * 2;
  }

  // The wave's WTM tokens x WTN features lie in one head slot (dh % WTN == 0).  Q and K
  // strips are rotated in registers and staged token-major, with the pair halves j and
  // j + dh/2 already apart, so that each token's run of the head row leaves as 16-byte
  // stores; V strips are staged feature-major and leave as 16-byte runs of 8 tokens of a
  // V^T row.  Two phases with a block barrier between them (every wave of the block runs
  // this function; the barrier orders each wave's LDS writes before its reads).
  template <int TN, int TM>
  __device__ static void tile_lds(const EpiParams& e, const GemmProblem& p, const f32x4 (&acc)[TN][TM], int mb,
                                  int nb, int lane, char* lds) {
    constexpr int WTN = TN * 16, WTM = TM * 16;
    const int fr = lane & 15, fq = lane >> 4;
    if (e.dh % WTN != 0) {  // the same for every wave of the grid
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int b = 0; b < TM; ++b) {
          const int m = mb + 16 * b + fr, n = nb + 16 * a + 4 * fq;
          if (m < p.M && n < p.N) apply(e, m, n, acc[a][b]);
        }
      return;
    }
    const bool live = nb < p.N;
    const int slot = fdiv(nb, e.dh_mul, e.dh_shift), c0 = nb - slot * e.dh;  // strip offset in the head
    const int half = e.dh >> 1, jbase = c0 >> 1;
    const bool is_v = slot >= e.H + e.Hkv;
    // phase 1: stage
    if (live && !is_v) {
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int r = 16 * b + fr;
        const int m = min(mb + r, p.M - 1);  // rows past M are staged but never stored
        const int bb = fdiv(m, e.l_mul, e.l_shift), l = m - bb * e.L;
        const float* rp = e.rope + ((size_t)(e.pos0 + l) * half + jbase) * 2;
#pragma unroll
        for (int a = 0; a < TN; ++a) {
          const int pl = 8 * a + 2 * fq;  // local pair index of (v0, v1); (v2, v3) is pl + 1
          const f32x4 v = acc[a][b];
          const float4 rr = *reinterpret_cast<const float4*>(rp + 2 * pl);  // cos, sin of pl and pl + 1
          const float a0 = v[0] * rr.x - v[1] * rr.y, b0 = v[1] * rr.x + v[0] * rr.y;
          const float a1 = v[2] * rr.z - v[3] * rr.w, b1 = v[3] * rr.z + v[2] * rr.w;
          store2(reinterpret_cast<bf16*>(lds + staged<WTN>(r, pl)), a0, a1);
          store2(reinterpret_cast<bf16*>(lds + staged<WTN>(r, WTN / 2 + pl)), b0, b1);
        }
      }
    } else if (live) {
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int b = 0; b < TM; ++b)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
            *reinterpret_cast<bf16*>(lds + staged<WTM>(16 * a + 4 * fq + jj, 16 * b + fr)) = (bf16)acc[a][b][jj];
    }
    __syncthreads();
    // phase 2: 16-byte chunks to the attention layouts
    if (live && !is_v) {
      constexpr int NC = WTN / 8;
      T* base = slot < e.H ? static_cast<T*>(e.q) : static_cast<T*>(e.k);
#pragma unroll
      for (int idx = lane; idx < WTM * NC; idx += 64) {
        const int r = idx / NC, c = idx % NC, m = mb + r;
        if (m >= p.M) continue;
        const int bb = fdiv(m, e.l_mul, e.l_shift), l = m - bb * e.L;
        const size_t row = slot < e.H ? ((size_t)bb * e.H + slot) * e.L + l
                                      : ((size_t)bb * e.Hkv + (slot - e.H)) * e.kv_cap + e.kv_off + l;
        const int col = c < NC / 2 ? jbase + 8 * c : jbase + half + 8 * (c - NC / 2);
        *reinterpret_cast<bf16x8*>(base + row * e.dh + col) = *reinterpret_cast<const bf16x8*>(lds + staged<WTN>(r, 8 * c));
      }
    } else if (live) {
      constexpr int NC = WTM / 8;
      const int hv = slot - e.H - e.Hkv;
#pragma unroll
      for (int idx = lane; idx < WTN * NC; idx += 64) {
        const int f = idx / NC, c = idx % NC, m0 = mb + 8 * c;
        if (m0 >= p.M) continue;
        const bf16x8 v = *reinterpret_cast<const bf16x8*>(lds + staged<WTM>(f, 8 * c));
        T* vrow = static_cast<T*>(e.vt) + (((size_t)0 * e.Hkv + hv) * e.dh + c0 + f) * e.kv_cap + e.kv_off;
        const int b0 = fdiv(m0, e.l_mul, e.l_shift), l0 = m0 - b0 * e.L;
        const size_t bstride = (size_t)e.Hkv * e.dh * e.kv_cap;  // one batch row of V^T
        if (m0 + 8 <= p.M && l0 + 8 <= e.L && ((e.kv_off + l0) & 7) == 0) {
          *reinterpret_cast<bf16x8*>(vrow + b0 * bstride + l0) = v;
        } else {
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            const int m = m0 + u;
            if (m >= p.M) break;
            const int bb = fdiv(m, e.l_mul, e.l_shift), l = m - bb * e.L;
            vrow[bb * bstride + l] = v[u];
          }
        }
      }
    }
  }
};
template <class T>
struct Epi<EPI_GLU_SILU, T> {
  static constexpr bool kGlu = true;
  __device__ static void glu(const EpiParams& e, int m, int f, f32x4 g, f32x4 u) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + f, silu_act<T>(g[0]) * u[0],
           silu_act<T>(g[1]) * u[1], silu_act<T>(g[2]) * u[2], silu_act<T>(g[3]) * u[3]);
  }
};
template <class T>
struct Epi<EPI_GLU_GELU, T> {
  static constexpr bool kGlu = true;
  __device__ static void glu(const EpiParams& e, int m, int f, f32x4 g, f32x4 u) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + f, gelu_act<T>(g[0]) * u[0],
           gelu_act<T>(g[1]) * u[1], gelu_act<T>(g[2]) * u[2], gelu_act<T>(g[3]) * u[3]);
  }
};

// ------------------------------------------------------------ fp32 VALU kernel
// Tile 64 (rows) x 64 (features), K step 16; each thread computes 4 x 4 outputs.
template <EpiKind KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmProblem p, EpiParams ep) {
  using E = Epi<KIND, float>;
  __shared__ float sA[16][64 + 4];
  __shared__ float sW[16][64 + 4];
  __shared__ float xch[64][64 + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int tiles_m = (p.M + 63) / 64;
  const int m0 = (blockIdx.x % tiles_m) * 64, n0 = (blockIdx.x / tiles_m) * 64;
  const float* A1 = static_cast<const float*>(p.A1);
  const float* A2 = static_cast<const float*>(p.A2);
  const float* W = static_cast<const float*>(p.W);
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i, r = c >> 4, kk = c & 15, k = k0 + kk;
      float av = 0.f, wv = 0.f;
      if (k < p.K) {
        const int gr = min(m0 + r, p.M - 1), gn = min(n0 + r, p.N - 1);
        av = k < p.K1 ? A1[(size_t)gr * p.lda1 + k] : A2[(size_t)gr * p.lda2 + (k - p.K1)];
        wv = W[(size_t)gn * p.ldw + k];
      }
      sA[kk][r] = av;
      sW[kk][r] = wv;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { a[i] = sA[kk][ty * 4 + i]; w[i] = sW[kk][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * w[j];
    }
    __syncthreads();
  }
  const int n = n0 + tx * 4;
  if constexpr (E::kGlu) {
    // features of the up half (offset 16 inside each 32-row block) come from thread tx + 4
    const bool up = ((tx * 4) & 31) >= 16;
    if (up)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) xch[ty * 4 + i][tx * 4 + j] = acc[i][j];
    __syncthreads();
    if (!up && n < p.N)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + ty * 4 + i;
        if (m >= p.M) continue;
        const float* u = &xch[ty * 4 + i][tx * 4 + 16];
        const int f = ((n >> 5) << 4) + (n & 15);
        E::glu(ep, m, f, f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]}, f32x4{u[0], u[1], u[2], u[3]});
      }
  } else {
    if (n >= p.N) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + ty * 4 + i;
      if (m < p.M) E::apply(ep, m, n, f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]});
    }
  }
}

template <EpiKind K>
hipError_t dispatch(DType dt, const GemmProblem& p, const EpiParams& e, hipStream_t s) {
  if (dt == F32) {
    const int tiles = ((p.M + 63) / 64) * ((p.N + 63) / 64);
    launch_timed(gemm_f32_kernel<K>, dim3(tiles), dim3(256), 0, s, p, e);
    return hipGetLastError();
  }
  // tile choice by how many blocks each shape yields (256 CUs): GEMMs with many rows
  // take 256 x 256 tiles on 8 waves, mid-size ones 128 x 128 at two blocks per CU, and
  // the narrow (N = d_model) projections 64 x 64 at three blocks per CU
  const long t256 = (long)((p.M + 255) / 256) * ((p.N + 255) / 256);
  const long t128 = (long)((p.M + 127) / 128) * ((p.N + 127) / 128);
  if ((p.M >= 4096 || p.N >= 16384) && t256 >= 128) {
    if constexpr (K == EPI_GLU_SILU || K == EPI_GLU_GELU) {
      // one block per CU runs in rounds of 256: 256 x 192 tiles (waves 64 x 96) win when
      // they fill the last round better (26B-class gate/up, 1024 x 73728: 1152 tiles of
      // 256 x 256 = 4.5 rounds -> 1536 of 256 x 192 = 6 rounds: 747 -> 669 us)
      const long t192 = (long)((p.M + 255) / 256) * ((p.N + 191) / 192);
      if ((t192 + 255) / 256 * 192 < (t256 + 255) / 256 * 256) return launch_bf16<256, 192, 2, 4, 2, 1, K>(p, e, s);
    }
    return launch_bf16<256, 256, 2, 2, 4, 1, K>(p, e, s);
  }
  if (t128 >= 256) {
    // two blocks per CU run in rounds of 512; 192 x 128 tiles win when they need fewer
    // rounds for the same rows (e.g. 768 tiles of 128 x 128 = 1.5 rounds -> 512 of 192 x 128)
    const long t192 = (long)((p.M + 191) / 192) * ((p.N + 127) / 128);
    const long cost128 = (t128 + 511) / 512 * 128 * 128, cost192 = (t192 + 511) / 512 * 192 * 128;
    if (cost192 < cost128) return launch_bf16<192, 128, 2, 2, 2, 2, K>(p, e, s);
    return launch_bf16<128, 128, 2, 2, 2, 2, K>(p, e, s);
  }
  return launch_bf16<64, 64, 2, 2, 2, 3, K>(p, e, s);
}

// out[m, n] = row1[m] * sum_s part[s, m, n], s ascending (float4 granules, N % 4 == 0)
__global__ void splitk_reduce_kernel(const float* part, int S, int M, int N, const float* row1, float* out, int ldo) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x, n4 = N / 4;
  if (i >= (long)M * n4) return;
  const int m = (int)(i / n4), n = (int)(i % n4) * 4;
  const size_t MN = (size_t)M * N;
  float4 acc = *reinterpret_cast<const float4*>(part + (size_t)m * N + n);
  for (int k = 1; k < S; ++k) {
    const float4 v = *reinterpret_cast<const float4*>(part + k * MN + (size_t)m * N + n);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  const float r = row1[m];
  store4(out + (size_t)m * ldo + n, r * acc.x, r * acc.y, r * acc.z, r * acc.w);
}

// Row-scaled product with a long K and few output tiles (the self-conditioning product:
// K = vocabulary, N = d_model): 128 x 128 tiles split over K so that the grid fills the
// chip, the slices' fp32 products go to part [S, M, N], then an ordered reduction.
// Returns false when the split does not apply.
// K slices: double while the grid has fewer than 512 blocks, each slice keeps >= 8 K
// tiles and the tiles divide evenly (at most 16)
int split_slices(int M, int N, int K) {
  const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128);
  const int nk = K / 64;
  int S = 1;
  while (S < 16 && tiles * S < 512 && nk % (2 * S) == 0 && nk / (2 * S) >= 8) S *= 2;
  return S;
}

bool splitk_scale(const GemmProblem& p, const EpiParams& e, hipStream_t s, hipError_t* err) {
  if (!e.part || p.M_dev || p.N % 4 || p.K1 != p.K) return false;
  const int S = split_slices(p.M, p.N, p.K);
  if (S == 1) return false;
  GemmProblem q = p;
  q.ksplit = S;
  EpiParams f;
  f.out = e.part;
  f.ldo = p.N;
  f.split_stride = (size_t)p.M * p.N;
  *err = launch_bf16<128, 128, 2, 2, 2, 2, EPI_STORE_F32>(q, f, s);
  if (*err != hipSuccess) return true;
  const long total = (long)p.M * (p.N / 4);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     static_cast<const float*>(e.part), S, p.M, p.N, e.row1, static_cast<float*>(e.out), e.ldo);
  *err = hipGetLastError();
  return true;
}

// resid[m, n] += sum_s part[s, m, n], s ascending (float4 granules, N % 4 == 0)
__global__ void resid_reduce_kernel(const float* part, int S, int M, int N, float* resid, int ldr) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x, n4 = N / 4;
  if (i >= (long)M * n4) return;
  const int m = (int)(i / n4), n = (int)(i % n4) * 4;
  const size_t MN = (size_t)M * N;
  float4 acc = *reinterpret_cast<const float4*>(part + (size_t)m * N + n);
  for (int k = 1; k < S; ++k) {
    const float4 v = *reinterpret_cast<const float4*>(part + k * MN + (size_t)m * N + n);
    acc.x += v.x;
    acc.y += v.y;
    acc.z += v.z;
    acc.w += v.w;
  }
  float4* r = reinterpret_cast<float4*>(resid + (size_t)m * ldr + n);
  float4 x = *r;
  x.x += acc.x;
  x.y += acc.y;
  x.z += acc.z;
  x.w += acc.w;
  *r = x;
}

// resid[m, :] += sum_s part[s, m, :] as above, then y[m, :] = bf16(resid[m, :] * rsqrt(
// mean(resid[m, :]^2) + eps) * g): the RMSNorm that follows a residual product, in the
// same pass over the row.  One block of 256 threads per row, NV float4 per thread
// (N <= 1024 NV): every slice load of the row is independent, so the row costs one
// round trip; the row's sum of squares is a block reduction.
template <int NV>
__global__ __launch_bounds__(256) void resid_reduce_rms_kernel(const float* part, int S, int M, int N, float* resid,
                                                               int ldr, const float* g, float eps, bf16* y) {
  __shared__ float red[4];
  const int m = blockIdx.x, t = threadIdx.x;
  const size_t MN = (size_t)M * N;
  float4 x[NV];
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (t + 256 * i) * 4;
    if (c < N) {
      float4 acc = *reinterpret_cast<const float4*>(part + (size_t)m * N + c);
      for (int k = 1; k < S; ++k) {
        const float4 v = *reinterpret_cast<const float4*>(part + k * MN + (size_t)m * N + c);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
      }
      float4* r = reinterpret_cast<float4*>(resid + (size_t)m * ldr + c);
      float4 v = *r;
      v.x += acc.x;
      v.y += acc.y;
      v.z += acc.z;
      v.w += acc.w;
      *r = v;
      x[i] = v;
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
  }
  ss = block_sum(ss, red);
  const float rs = rsqrtf(ss / N + eps);
  bf16* yr = y + (size_t)m * N;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = (t + 256 * i) * 4;
    if (c < N) {
      const float4 w = *reinterpret_cast<const float4*>(g + c);
      store4(yr + c, x[i].x * rs * w.x, x[i].y * rs * w.y, x[i].z * rs * w.z, x[i].w * rs * w.w);
    }
  }
}

// K slices of a residual product on 256 x 256 tiles, one block per CU: the S in
// [2, 16] (each slice >= 8 K tiles, slices as even as the tile count allows) that
// minimises the modelled time, in K-step units: rounds of 256 blocks x (K tiles per
// slice + 2 for a block's prologue and epilogue), plus 1.5 per slice for the ordered
// reduction's read of the slice's [M, N] partial; 1 when no split beats the unsplit
// grid.  Products with fewer than 128 K tiles are split only from 64 output tiles on:
// smaller ones run sooner on the 64 x 64 or 128 x 128 tiles at two or three blocks per CU
// (block workload's attention output, 1024 x 2048 x 2048, and the small workload's FFN
// down, 3072 x 768 x 2048: 2.5 % and 6.6 % slower per generation when split).  26B-class
// FFN down (1024 x 4608 x 36864): S = 7, 504 blocks in two rounds (468 -> 354 us against
// 128 x 128 tiles in 8 slices); its attention output (1024 x 4608 x 4096): S = 3.
int resid_slices256(int M, int N, int K) {
  const long tiles = (long)((M + 255) / 256) * ((N + 255) / 256);
  const int nk = K / 64;
  if (N % 4 || nk < 32 || (nk < 128 && tiles < 64)) return 1;
  int best = 1;
  double best_t = (double)((tiles + 255) / 256) * (nk + 2);
  for (int S = 2; S <= 16 && nk / S >= 8; ++S) {
    const double t = (double)((tiles * S + 255) / 256) * ((double)nk / S + 2) + 1.5 * S;
    if (t < best_t - 1e-9) {
      best = S;
      best_t = t;
    }
  }
  return best;
}

// K slices of a residual product with a long K and fewer than two 128 x 128 tiles per
// CU (512 resident blocks): the S in {2, 4, 8} (each slice >= 16 K tiles) whose grid
// best fills whole rounds of 512 blocks, the smaller S on ties
int resid_slices(int M, int N, int K) {
  const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128);
  const int nk = K / 64;
  if (tiles >= 512 || nk < 64 || N % 4) return 1;
  int best = 1;
  double best_fill = 0.0;
  for (int S = 2; S <= 8; S *= 2) {
    if (nk % S || nk / S < 16) break;
    const long blocks = tiles * S, rounds = (blocks + 511) / 512;
    const double fill = (double)blocks / (512.0 * rounds);
    if (fill > best_fill + 1e-9) {
      best = S;
      best_fill = fill;
    }
  }
  return best;
}

}  // namespace

int gemm_split_slices(int M, int N, int K) { return split_slices(M, N, K); }
int gemm_resid_slices(int M, int N, int K) {
  const int S256 = resid_slices256(M, N, K);
  return S256 > 1 ? S256 : resid_slices(M, N, K);
}
bool gemm_resid_norms(int M, int N, int K) { return gemm_resid_slices(M, N, K) > 1 && N % 4 == 0 && N <= 8192; }

hipError_t gemm(DType dt, const GemmProblem& p, EpiKind kind, const EpiParams& e, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (kind == EPI_SCALE_F32 && dt == BF16) {
    hipError_t err = hipSuccess;
    if (splitk_scale(p, e, s, &err)) return err;
  }
  if (kind == EPI_RESID && dt == BF16 && e.part && !p.M_dev && p.K1 == p.K) {
    const int S256 = resid_slices256(p.M, p.N, p.K);
    const int S = S256 > 1 ? S256 : resid_slices(p.M, p.N, p.K);
    if (S > 1) {  // the slices' products to part [S, M, N], then an ordered sum into resid
      GemmProblem q = p;
      q.ksplit = S;
      EpiParams f;
      f.out = e.part;
      f.ldo = p.N;
      f.split_stride = (size_t)p.M * p.N;
      hipError_t err = S256 > 1 ? launch_bf16<256, 256, 2, 2, 4, 1, EPI_STORE_F32>(q, f, s)
                                : launch_bf16<128, 128, 2, 2, 2, 2, EPI_STORE_F32>(q, f, s);
      if (err != hipSuccess) return err;
      if (e.norm_out) {  // the ordered sum and the RMSNorm of the updated rows in one pass
        if (!gemm_resid_norms(p.M, p.N, p.K) || !e.norm_g) return hipErrorInvalidValue;
        const float* part = static_cast<const float*>(e.part);
        bf16* y = static_cast<bf16*>(e.norm_out);
        const int nv = (p.N + 1023) / 1024;
        if (nv <= 1)
          hipLaunchKernelGGL(resid_reduce_rms_kernel<1>, dim3(p.M), dim3(256), 0, s, part, S, p.M, p.N, e.resid, e.ldr,
                             e.norm_g, e.norm_eps, y);
        else if (nv <= 2)
          hipLaunchKernelGGL(resid_reduce_rms_kernel<2>, dim3(p.M), dim3(256), 0, s, part, S, p.M, p.N, e.resid, e.ldr,
                             e.norm_g, e.norm_eps, y);
        else if (nv <= 5)
          hipLaunchKernelGGL(resid_reduce_rms_kernel<5>, dim3(p.M), dim3(256), 0, s, part, S, p.M, p.N, e.resid, e.ldr,
                             e.norm_g, e.norm_eps, y);
        else
          hipLaunchKernelGGL(resid_reduce_rms_kernel<8>, dim3(p.M), dim3(256), 0, s, part, S, p.M, p.N, e.resid, e.ldr,
                             e.norm_g, e.norm_eps, y);
        return hipGetLastError();
      }
      const long total = (long)p.M * (p.N / 4);
      hipLaunchKernelGGL(resid_reduce_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                         static_cast<const float*>(e.part), S, p.M, p.N, e.resid, e.ldr);
      return hipGetLastError();
    }
  }
  switch (kind) {
    case EPI_STORE: return dispatch<EPI_STORE>(dt, p, e, s);
    case EPI_STORE_F32: return dispatch<EPI_STORE_F32>(dt, p, e, s);
    case EPI_SCALE_F32: return dispatch<EPI_SCALE_F32>(dt, p, e, s);
    case EPI_RESID: return dispatch<EPI_RESID>(dt, p, e, s);
    case EPI_GELU: return dispatch<EPI_GELU>(dt, p, e, s);
    case EPI_GLU_SILU: return dispatch<EPI_GLU_SILU>(dt, p, e, s);
    case EPI_GLU_GELU: return dispatch<EPI_GLU_GELU>(dt, p, e, s);
    case EPI_FUSION1: return dispatch<EPI_FUSION1>(dt, p, e, s);
    case EPI_FUSION2: return dispatch<EPI_FUSION2>(dt, p, e, s);
    case EPI_SILU: return dispatch<EPI_SILU>(dt, p, e, s);
    case EPI_ADD_F32: return dispatch<EPI_ADD_F32>(dt, p, e, s);
    case EPI_ADD_BOTH: return dispatch<EPI_ADD_BOTH>(dt, p, e, s);
    case EPI_ADD_SUB: return dispatch<EPI_ADD_SUB>(dt, p, e, s);
    case EPI_PAIRED: return dispatch<EPI_PAIRED>(dt, p, e, s);
    case EPI_QKV_ROPE: {
      EpiParams f = e;
      fast_divider((uint32_t)e.L, f.l_mul, f.l_shift);
      fast_divider((uint32_t)e.dh, f.dh_mul, f.dh_shift);
      return dispatch<EPI_QKV_ROPE>(dt, p, f, s);
    }
    case EPI_SAMPLE: break;  // head_sample
  }
  return hipErrorInvalidValue;
}

}  // namespace tadm
