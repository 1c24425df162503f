// Dense contractions of the TADM step: C = A W^T with fused epilogues.
//
// bf16 path (gfx950): WGM x WGN wave64s per block, block tile BM x BN, K tiles of
// 64.  Tiles move global -> LDS with global_load_lds_dwordx4 (no register staging) through a STAGES-deep ring of LDS buffers, so that STAGES-1 tiles are in
// flight while one is multiplied.  LDS rows are 128 B (64 bf16); the 16-byte chunk c
// of row r is stored in slot c ^ (r & 7), which makes the MFMA fragment reads
// (16 rows x one chunk) hit distinct banks; the permutation is applied through the
// global addresses because each lane's 16 bytes land at a fixed LDS slot.
// Products use v_mfma_f32_16x16x32_bf16 with the weight tile as the "A" operand and
// the activation tile as "B", so every lane ends with 4 consecutive output features
// of one row and stores them as one vector.  Blocks are renumbered so that the
// tiles sharing a weight panel run on the same XCD (each XCD has its own L2).
// float32 path (small fp32 models): a register-blocked VALU kernel, same epilogues.
#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

// ------------------------------------------------------------------ epilogues
template <EpiKind K, class T>
struct Epi;

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
struct Epi<EPI_RESID, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    float4* r = reinterpret_cast<float4*>(e.resid + (size_t)m * e.ldr + n);
    float4 x = *r;
    x.x += v[0]; x.y += v[1]; x.z += v[2]; x.w += v[3];
    *r = x;
  }
};
template <class T>
struct Epi<EPI_GELU, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, gelu_erf(v[0]), gelu_erf(v[1]),
           gelu_erf(v[2]), gelu_erf(v[3]));
  }
};
template <class T>
struct Epi<EPI_FUSION1, T> {
  static constexpr bool kGlu = false;
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
    if (n < e.split) {
      store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, gelu_erf(v[0] + b.x),
             gelu_erf(v[1] + b.y), gelu_erf(v[2] + b.z), gelu_erf(v[3] + b.w));
    } else {
      store4(e.out2 + (size_t)m * e.ldo2 + (n - e.split), sigmoidf_(v[0] + b.x),
             sigmoidf_(v[1] + b.y), sigmoidf_(v[2] + b.z), sigmoidf_(v[3] + b.w));
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
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + n, siluf_(v[0]), siluf_(v[1]), siluf_(v[2]),
           siluf_(v[3]));
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
  __device__ static void apply(const EpiParams& e, int m, int n, f32x4 v) {
    const int b = m / e.L, l = m % e.L;
    const int slot = n / e.dh, c = n % e.dh;  // c is a multiple of 4
    if (slot < e.H + e.Hkv) {
      // (v0, v1) = pair j, (v2, v3) = pair j + 1 with j = c / 2
      const int j = c >> 1, half = e.dh >> 1;
      const float* cs = e.cos_t + (size_t)(e.pos0 + l) * half + j;
      const float* sn = e.sin_t + (size_t)(e.pos0 + l) * half + j;
      const float a0 = v[0] * cs[0] - v[1] * sn[0], b0 = v[1] * cs[0] + v[0] * sn[0];
      const float a1 = v[2] * cs[1] - v[3] * sn[1], b1 = v[3] * cs[1] + v[2] * sn[1];
      T* row = slot < e.H
                   ? static_cast<T*>(e.q) + (((size_t)b * e.H + slot) * e.L + l) * e.dh
                   : static_cast<T*>(e.k) + (((size_t)b * e.Hkv + (slot - e.H)) * e.kv_cap + e.kv_off + l) * e.dh;
      row[j] = from_f32<T>(a0);
      row[j + 1] = from_f32<T>(a1);
      row[j + half] = from_f32<T>(b0);
      row[j + half + 1] = from_f32<T>(b1);
    } else {
      T* col = static_cast<T*>(e.vt) + (((size_t)b * e.Hkv + (slot - e.H - e.Hkv)) * e.dh + c) * e.kv_cap +
               e.kv_off + l;
#pragma unroll
      for (int t = 0; t < 4; ++t) col[(size_t)t * e.kv_cap] = from_f32<T>(v[t]);
    }
  }
};
template <class T>
struct Epi<EPI_GLU_SILU, T> {
  static constexpr bool kGlu = true;
  __device__ static void glu(const EpiParams& e, int m, int f, f32x4 g, f32x4 u) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + f, siluf_(g[0]) * u[0], siluf_(g[1]) * u[1],
           siluf_(g[2]) * u[2], siluf_(g[3]) * u[3]);
  }
};
template <class T>
struct Epi<EPI_GLU_GELU, T> {
  static constexpr bool kGlu = true;
  __device__ static void glu(const EpiParams& e, int m, int f, f32x4 g, f32x4 u) {
    store4(static_cast<T*>(e.out) + (size_t)m * e.ldo + f, gelu_erf(g[0]) * u[0],
           gelu_erf(g[1]) * u[1], gelu_erf(g[2]) * u[2], gelu_erf(g[3]) * u[3]);
  }
};

// waitcnt immediate for "at most n vector-memory operations outstanding" (gfx9 encoding)
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

typedef __attribute__((address_space(3))) void* lds_ptr;
typedef const __attribute__((address_space(1))) void* gbl_ptr;

// Block index -> (m tile, n tile).  Workgroups are dealt to the 8 XCDs round-robin,
// so block b runs on XCD b % 8 as its (b / 8)-th block.  When the tile grid splits
// into 8 regions of rm x rn tiles, XCD x works through region x (m fastest), so the
// A rows and W rows it reads (rm*BM + rn*BN rows) stay in its own L2.
__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int rm, int rn, int& tm, int& tn) {
  const int b = blockIdx.x;
  if (rm > 0) {
    const int x = b % 8, i = b / 8, regions_m = tiles_m / rm;
    tm = (x % regions_m) * rm + i % rm;
    tn = (x / regions_m) * rn + i / rm;
    return;
  }
  tm = b % tiles_m;
  tn = b / tiles_m;
}

// ------------------------------------------------------------ bf16 MFMA kernel
template <int BM, int BN, int STAGES, int WGM, int WGN, int MINB, EpiKind KIND>
__global__ __launch_bounds__(64 * WGM * WGN, MINB) void gemm_bf16_kernel(GemmProblem p, EpiParams ep) {
  using E = Epi<KIND, bf16>;
  constexpr int NW = WGM * WGN;                 // waves per block
  constexpr int ROW = 128;                      // bytes per LDS row (64 bf16)
  constexpr int STAGE_BYTES = (BM + BN) * ROW;
  constexpr int LA = BM / 8 / NW, LW = BN / 8 / NW;  // load instructions per wave per stage
  static_assert(LA * 8 * NW == BM && LW * 8 * NW == BN, "tile rows must split evenly over waves");
  constexpr int LPS = LA + LW;
  constexpr int WTM = BM / WGM, WTN = BN / WGN; // wave tile
  constexpr int TM = WTM / 16, TN = WTN / 16;   // 16x16 subtiles per wave
  static_assert(WTN % 32 == 0, "GLU pairs need 32-row weight blocks per wave");
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WGM, wn = wave / WGM;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tmi, tni;
  tile_of(tiles_m, tiles_n, p.rm, p.rn, tmi, tni);
  const int m0 = tmi * BM, n0 = tni * BN;
  if (p.M_dev) {  // rows present this call; the grid was sized for p.M
    p.M = min(*p.M_dev, p.M);
    if (m0 >= p.M) return;
  }

  const bf16* A1 = static_cast<const bf16*>(p.A1);
  const bf16* A2 = static_cast<const bf16*>(p.A2);
  const bf16* W = static_cast<const bf16*>(p.W);

  // this lane's source row inside an 8-row group and its swizzled chunk
  const int lrow = lane >> 3, lchunk = (lane & 7) ^ (lane >> 3);

  auto issue = [&](int kt, int buf) {
    const int k0 = kt * 64;
    const bf16* Ab = A1;
    int lda = p.lda1, kk = k0;
    if (k0 >= p.K1) { Ab = A2; lda = p.lda2; kk = k0 - p.K1; }
    char* sb = smem + buf * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < LA; ++j) {
      const int g = wave + NW * j;              // 8-row group
      const int r = min(m0 + g * 8 + lrow, p.M - 1);
      const bf16* src = Ab + (size_t)r * lda + kk + lchunk * 8;
      __builtin_amdgcn_global_load_lds((gbl_ptr)src, (lds_ptr)(sb + g * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < LW; ++j) {
      const int g = wave + NW * j;
      const int r = min(n0 + g * 8 + lrow, p.N - 1);
      const bf16* src = W + (size_t)r * p.ldw + k0 + lchunk * 8;
      __builtin_amdgcn_global_load_lds((gbl_ptr)src, (lds_ptr)(sb + BM * ROW + g * 1024), 16, 0, 0);
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / 64;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s, s);

  const int fr = lane & 15, fq = lane >> 4, sw = lane & 7;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + STAGES - 2 < nk)
      __builtin_amdgcn_s_waitcnt(vmcnt_imm((STAGES - 2) * LPS));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    const char* sa = smem + (kt % STAGES) * STAGE_BYTES;
    const char* swt = sa + BM * ROW;
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int slot = ((kk * 4 + fq) ^ sw) * 16;
      bf16x8 fa[TM], fw[TN];
#pragma unroll
      for (int t = 0; t < TM; ++t)
        fa[t] = *reinterpret_cast<const bf16x8*>(sa + (wm * WTM + t * 16 + fr) * ROW + slot);
#pragma unroll
      for (int t = 0; t < TN; ++t)
        fw[t] = *reinterpret_cast<const bf16x8*>(swt + (wn * WTN + t * 16 + fr) * ROW + slot);
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int b = 0; b < TM; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[a], fa[b], acc[a][b], 0, 0, 0);
    }
  }

  // lane holds C[n = nb + 4*(lane>>4) + j][m = mb + (lane & 15)]
  const int mw = m0 + wm * WTM + fr;
  if constexpr (E::kGlu) {
#pragma unroll
    for (int a = 0; a < TN; a += 2)
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int m = mw + b * 16;
        const int ng = n0 + wn * WTN + a * 16;  // multiple of 32: gate rows of a 32-row block
        if (m < p.M && ng < p.N) E::glu(ep, m, ng / 2 + 4 * fq, acc[a][b], acc[a + 1][b]);
      }
  } else {
    const int nw = n0 + wn * WTN + 4 * fq;
#pragma unroll
    for (int a = 0; a < TN; ++a)
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int m = mw + b * 16, n = nw + a * 16;
        if (m < p.M && n < p.N) E::apply(ep, m, n, acc[a][b]);
      }
  }
}

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

// Per-XCD region rm x rn with (tiles_m / rm) * (tiles_n / rn) = 8 that minimises the
// rows each XCD reads (rm * BM + rn * BN); 0 when the grid does not split evenly.
inline void xcd_regions(int tiles_m, int tiles_n, int BM, int BN, int& rm, int& rn) {
  rm = rn = 0;
  long best = -1;
  for (int gm = 1; gm <= 8; gm *= 2) {
    const int gn = 8 / gm;
    if (tiles_m % gm || tiles_n % gn) continue;
    const long cost = (long)(tiles_m / gm) * BM + (long)(tiles_n / gn) * BN;
    if (best < 0 || cost < best) {
      best = cost;
      rm = tiles_m / gm;
      rn = tiles_n / gn;
    }
  }
}

template <int BM, int BN, int ST, int WGM, int WGN, int MINB, EpiKind K>
hipError_t launch_bf16(const GemmProblem& p0, const EpiParams& e, hipStream_t s) {
  GemmProblem p = p0;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  xcd_regions(tiles_m, tiles_n, BM, BN, p.rm, p.rn);
  launch_timed(gemm_bf16_kernel<BM, BN, ST, WGM, WGN, MINB, K>, dim3(tiles_m * tiles_n), dim3(64 * WGM * WGN),
               0, s, p, e);
  return hipGetLastError();
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
  if ((p.M >= 4096 || p.N >= 16384) && t256 >= 128) return launch_bf16<256, 256, 2, 2, 4, 1, K>(p, e, s);
  if (t128 >= 256) return launch_bf16<128, 128, 2, 2, 2, 2, K>(p, e, s);
  return launch_bf16<64, 64, 2, 2, 2, 3, K>(p, e, s);
}

}  // namespace

hipError_t gemm(DType dt, const GemmProblem& p, EpiKind kind, const EpiParams& e, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  switch (kind) {
    case EPI_STORE: return dispatch<EPI_STORE>(dt, p, e, s);
    case EPI_STORE_F32: return dispatch<EPI_STORE_F32>(dt, p, e, s);
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
    case EPI_QKV_ROPE: return dispatch<EPI_QKV_ROPE>(dt, p, e, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace tadm
