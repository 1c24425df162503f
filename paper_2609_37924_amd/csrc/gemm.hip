// Dense contractions of the TADM step: C = A W^T with fused epilogues.
//
// bf16 path: v_mfma_f32_16x16x32_bf16 on LDS-staged, double-buffered 64-deep K
// tiles.  The weight tile is the MFMA "A" operand and the activation tile the "B"
// operand, so each lane ends with 4 consecutive output features of one row and
// stores them as one 8/16-byte vector.  256 threads = 4 wave64s in a 2x2 grid.
// float32 path (small fp32 models): a register-blocked VALU kernel with the same
// epilogues.
#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

template <class T>
struct Epi {
  EpiKind kind;
  EpiParams e;

  __device__ __forceinline__ void operator()(int m, int n, f32x4 v) const {
    switch (kind) {
      case EPI_STORE: {
        T* o = static_cast<T*>(e.out) + (size_t)m * e.ldo + n;
        store4(o, v[0], v[1], v[2], v[3]);
        break;
      }
      case EPI_STORE_F32: {
        float* o = static_cast<float*>(e.out) + (size_t)m * e.ldo + n;
        store4(o, v[0], v[1], v[2], v[3]);
        break;
      }
      case EPI_RESID: {
        float4* r = reinterpret_cast<float4*>(e.resid + (size_t)m * e.ldr + n);
        float4 x = *r;
        x.x += v[0]; x.y += v[1]; x.z += v[2]; x.w += v[3];
        *r = x;
        break;
      }
      case EPI_GELU: {
        T* o = static_cast<T*>(e.out) + (size_t)m * e.ldo + n;
        store4(o, gelu_erf(v[0]), gelu_erf(v[1]), gelu_erf(v[2]), gelu_erf(v[3]));
        break;
      }
      case EPI_FUSION1: {
        const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
        if (n < e.split) {
          T* o = static_cast<T*>(e.out) + (size_t)m * e.ldo + n;
          store4(o, gelu_erf(v[0] + b.x), gelu_erf(v[1] + b.y), gelu_erf(v[2] + b.z),
                 gelu_erf(v[3] + b.w));
        } else {
          float* o = e.out2 + (size_t)m * e.ldo2 + (n - e.split);
          store4(o, sigmoidf_(v[0] + b.x), sigmoidf_(v[1] + b.y), sigmoidf_(v[2] + b.z),
                 sigmoidf_(v[3] + b.w));
        }
        break;
      }
      case EPI_FUSION2: {
        const float4 b = *reinterpret_cast<const float4*>(e.bias + n);
        const float4 h = *reinterpret_cast<const float4*>(e.aux + (size_t)m * e.ld_aux + n);
        const float4 g = *reinterpret_cast<const float4*>(e.gate + (size_t)m * e.ldg + n);
        float* o = e.resid + (size_t)m * e.ldr + n;
        store4(o, h.x + g.x * (v[0] + b.x), h.y + g.y * (v[1] + b.y), h.z + g.z * (v[2] + b.z),
               h.w + g.w * (v[3] + b.w));
        break;
      }
      default:
        break;
    }
  }

  // Gate/up pair of a GLU feed-forward: features f .. f+3.
  __device__ __forceinline__ void glu(int m, int f, f32x4 g, f32x4 u) const {
    T* o = static_cast<T*>(e.out) + (size_t)m * e.ldo + f;
    if (kind == EPI_GLU_SILU)
      store4(o, siluf_(g[0]) * u[0], siluf_(g[1]) * u[1], siluf_(g[2]) * u[2], siluf_(g[3]) * u[3]);
    else
      store4(o, gelu_erf(g[0]) * u[0], gelu_erf(g[1]) * u[1], gelu_erf(g[2]) * u[2],
             gelu_erf(g[3]) * u[3]);
  }

  __device__ __forceinline__ bool is_glu() const { return kind == EPI_GLU_SILU || kind == EPI_GLU_GELU; }
};

// ------------------------------------------------------------ bf16 MFMA kernel
constexpr int BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // elements; 144-byte rows keep 16-byte alignment

template <int BM, int BN>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmProblem p, Epi<bf16> epi) {
  constexpr int CA = BM / 32, CW = BN / 32;      // 16-byte chunks per thread per stage
  constexpr int TM = BM / 32, TN = BN / 32;      // 16x16 subtiles per wave
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) bf16 sW[2][BN * LDS_STRIDE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int tiles_m = (p.M + BM - 1) / BM;
  const int m0 = (blockIdx.x % tiles_m) * BM;
  const int n0 = (blockIdx.x / tiles_m) * BN;

  const bf16* A1 = static_cast<const bf16*>(p.A1);
  const bf16* A2 = static_cast<const bf16*>(p.A2);
  const bf16* W = static_cast<const bf16*>(p.W);

  uint4 ra[CA], rw[CW];
  auto gload = [&](int kt) {
    const int k0 = kt * BK;
    const bf16* Ab = A1;
    int lda = p.lda1, kk = k0;
    if (k0 >= p.K1) { Ab = A2; lda = p.lda2; kk = k0 - p.K1; }
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + 256 * i, r = c >> 3, ch = c & 7;
      const int gr = min(m0 + r, p.M - 1);
      ra[i] = *reinterpret_cast<const uint4*>(Ab + (size_t)gr * lda + kk + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < CW; ++i) {
      const int c = tid + 256 * i, r = c >> 3, ch = c & 7;
      const int gn = min(n0 + r, p.N - 1);
      rw[i] = *reinterpret_cast<const uint4*>(W + (size_t)gn * p.ldw + k0 + ch * 8);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + 256 * i, r = c >> 3, ch = c & 7;
      *reinterpret_cast<uint4*>(&sA[buf][r * LDS_STRIDE + ch * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CW; ++i) {
      const int c = tid + 256 * i, r = c >> 3, ch = c & 7;
      *reinterpret_cast<uint4*>(&sW[buf][r * LDS_STRIDE + ch * 8]) = rw[i];
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = p.K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 32) {
      bf16x8 fa[TM], fw[TN];
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        const int row = wm * (BM / 2) + t * 16 + (lane & 15);
        fa[t] = *reinterpret_cast<const bf16x8*>(&sA[buf][row * LDS_STRIDE + kk + (lane >> 4) * 8]);
      }
#pragma unroll
      for (int t = 0; t < TN; ++t) {
        const int row = wn * (BN / 2) + t * 16 + (lane & 15);
        fw[t] = *reinterpret_cast<const bf16x8*>(&sW[buf][row * LDS_STRIDE + kk + (lane >> 4) * 8]);
      }
#pragma unroll
      for (int a = 0; a < TN; ++a)
#pragma unroll
        for (int b = 0; b < TM; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[a], fa[b], acc[a][b], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // lane holds C[n = nb + 4*(lane>>4) + j][m = mb + (lane & 15)]
  const int mw = m0 + wm * (BM / 2) + (lane & 15);
  const int nw = n0 + wn * (BN / 2) + 4 * (lane >> 4);
  if (epi.is_glu()) {
#pragma unroll
    for (int a = 0; a < TN; a += 2)
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int m = mw + b * 16;
        const int ng = n0 + wn * (BN / 2) + a * 16;  // multiple of 32: gate block
        if (m < p.M && ng < p.N) epi.glu(m, ng / 2 + 4 * (lane >> 4), acc[a][b], acc[a + 1][b]);
      }
  } else {
#pragma unroll
    for (int a = 0; a < TN; ++a)
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int m = mw + b * 16, n = nw + a * 16;
        if (m < p.M && n < p.N) epi(m, n, acc[a][b]);
      }
  }
}

// ------------------------------------------------------------ fp32 VALU kernel
// Tile 64 (rows) x 64 (features), K step 16; each thread computes 4 x 4 outputs.
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmProblem p, Epi<float> epi) {
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
  if (epi.is_glu()) {
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
        epi.glu(m, f, f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]}, f32x4{u[0], u[1], u[2], u[3]});
      }
    return;
  }
  if (n >= p.N) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m < p.M) epi(m, n, f32x4{acc[i][0], acc[i][1], acc[i][2], acc[i][3]});
  }
}

template <int BM, int BN>
hipError_t launch_bf16(const GemmProblem& p, const Epi<bf16>& epi, hipStream_t s) {
  const int tiles = ((p.M + BM - 1) / BM) * ((p.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN>), dim3(tiles), dim3(256), 0, s, p, epi);
  return hipGetLastError();
}

}  // namespace

hipError_t gemm(DType dt, const GemmProblem& p, EpiKind kind, const EpiParams& e, hipStream_t s) {
  if (p.M <= 0 || p.N <= 0) return hipSuccess;
  if (dt == F32) {
    Epi<float> epi{kind, e};
    const int tiles = ((p.M + 63) / 64) * ((p.N + 63) / 64);
    hipLaunchKernelGGL(gemm_f32_kernel, dim3(tiles), dim3(256), 0, s, p, epi);
    return hipGetLastError();
  }
  Epi<bf16> epi{kind, e};
  const long t128 = (long)((p.M + 127) / 128) * ((p.N + 127) / 128);
  const long t64 = (long)((p.M + 63) / 64) * ((p.N + 127) / 128);
  if (t128 >= 512) return launch_bf16<128, 128>(p, epi, s);
  if (t64 >= 512) return launch_bf16<64, 128>(p, epi, s);
  return launch_bf16<64, 64>(p, epi, s);
}

}  // namespace tadm
