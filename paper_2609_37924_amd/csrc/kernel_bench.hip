// kernel_bench: the layer kernels of one denoiser pass of a workload, each launched on
// its own at the workload's shapes, through the library's kernel launchers (the code
// that tadm_generate runs), with a plain copy kernel of known size beside them.  It is
// the program that per-kernel hardware counters (HBM bytes, MFMA use) are taken on.
//
//   kernel_bench key=value ...   (the arguments of tadm_run; reps=N launches per stage)
//
// Shapes: M = batch x pass length (block_len in block mode, prompt_len + gen_len
// otherwise); q/k/v [M, d] x [(H + 2 Hkv) dh, d] with the rotary epilogue; attention over
// the pass's queries and its keys (the prompt as context plus the block in block mode);
// attention output [M, H dh] x [d, H dh] and FFN down [M, d_ffn] x [d, d_ffn] with the
// residual epilogue (K-sliced as the library slices them, the slice sum also writing the
// following RMSNorm where the library's does); FFN up [M, d] x [2 d_ffn or
// d_ffn, d] with its GLU / GELU epilogue; the vocabulary projection [Mh, d] x [V, d]
// with the sampling epilogue, Mh the masked rows a reverse step sees on average under
// the linear schedule, and the merge of its partials into tokens; with the gated-MLP
// fusion, its two products ([M, 2d] x [5d, 2d] with the GELU / sigmoid split and
// [M, 4d] x [d, 4d] with the gated residual).  Operands are seeded uniform bf16 values.
// Prints each stage's mean time per launch from HIP events.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "kernels.h"

namespace tadm {
namespace {

#define HIP_OK(x)                                                                               \
  do {                                                                                          \
    hipError_t e_ = (x);                                                                        \
    if (e_ != hipSuccess) {                                                                     \
      fprintf(stderr, "kernel_bench: %s at line %d: %s\n", #x, __LINE__, hipGetErrorString(e_)); \
      exit(2);                                                                                  \
    }                                                                                           \
  } while (0)

__device__ __forceinline__ uint32_t mix32(uint64_t x) {
  x ^= x >> 33;
  x *= 0xff51afd7ed558ccdull;
  x ^= x >> 33;
  x *= 0xc4ceb9fe1a85ec53ull;
  x ^= x >> 33;
  return (uint32_t)x;
}

// bf16 values scale * u, u uniform in [-1, 1) (upper half of the float32 pattern)
__global__ void fill_bf16(uint16_t* out, size_t n, float scale, uint64_t seed) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const float v = scale * ((float)(mix32(seed * 0x9e3779b97f4a7c15ull + i) >> 8) * (1.0f / 8388608.0f) - 1.0f);
    uint32_t b;
    memcpy(&b, &v, 4);
    out[i] = (uint16_t)(b >> 16);
  }
}

__global__ void fill_iota(int32_t* out, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) out[i] = i;
}

// row_map of the finalize merge: the first `rows` canvas entries have partial rows
__global__ void fill_row_map(int32_t* out, int n, int rows) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) out[i] = i < rows ? i : -1;
}

__global__ void fill_i32(int32_t* out, int n, int32_t v) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) out[i] = v;
}

__global__ void fill_f32(float* out, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) out[i] = v;
}

// the calibration kernel: one thread per 16 bytes, grid = bytes / 16 exactly
__global__ void copy_kernel(const float4* a, float4* b, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) b[i] = a[i];
}

double num(const std::map<std::string, std::string>& kv, const char* k, double dflt, bool required = false) {
  auto it = kv.find(k);
  if (it == kv.end()) {
    if (required) {
      fprintf(stderr, "kernel_bench: missing %s=...\n", k);
      exit(1);
    }
    return dflt;
  }
  char* end = nullptr;
  const double v = strtod(it->second.c_str(), &end);
  if (!end || *end) {
    fprintf(stderr, "kernel_bench: bad value %s=%s\n", k, it->second.c_str());
    exit(1);
  }
  return v;
}

template <class T>
T* alloc(size_t n) {
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, n * sizeof(T) + 256));
  return static_cast<T*>(p);
}

uint16_t* random_bf16(size_t n, float scale, uint64_t seed) {
  uint16_t* p = alloc<uint16_t>(n);
  hipLaunchKernelGGL(fill_bf16, dim3(4096), dim3(256), 0, 0, p, n, scale, seed);
  HIP_OK(hipGetLastError());
  return p;
}

}  // namespace
}  // namespace tadm

using namespace tadm;

int main(int argc, char** argv) {
  std::map<std::string, std::string> kv;
  for (int a = 1; a < argc; ++a) {
    const char* eq = strchr(argv[a], '=');
    if (!eq) {
      fprintf(stderr, "usage: kernel_bench key=value ...  (bad argument '%s')\n", argv[a]);
      return 1;
    }
    kv[std::string(argv[a], eq - argv[a])] = eq + 1;
  }
  const int B = (int)num(kv, "batch", 0, true), P = (int)num(kv, "prompt_len", 0, true);
  const int G = (int)num(kv, "gen_len", 0, true), BL = (int)num(kv, "block_len", G);
  const int d = (int)num(kv, "d_model", 0, true), H = (int)num(kv, "n_heads", 0, true);
  const int Hkv = (int)num(kv, "n_kv_heads", H), dh = (int)num(kv, "head_dim", 0, true);
  const int F = (int)num(kv, "d_ffn", 0, true), ffn_kind = (int)num(kv, "ffn_kind", 1);
  const int V = (int)num(kv, "vocab", 0, true), T = (int)num(kv, "T", 0, true);
  const int reps = (int)num(kv, "reps", 5), fusion_kind = (int)num(kv, "fusion_kind", 0);
  const double theta = num(kv, "rope_theta", 10000.0);
  if ((int)num(kv, "dtype", 1) != 1) {
    fprintf(stderr, "kernel_bench: bf16 workloads only\n");
    return 1;
  }
  if (B <= 0 || G <= 0 || BL <= 0 || P < 0 || d <= 0 || H <= 0 || Hkv <= 0 || H % Hkv || dh <= 0 || F <= 0 ||
      reps <= 0 || d % 64 || F % 64 || (H * dh) % 64 || (dh != 64 && dh != 128) || V <= 0 || T <= 0) {
    fprintf(stderr, "kernel_bench: unsupported shape\n");
    return 1;
  }
  const bool block_mode = BL < G;
  const int L = block_mode ? BL : P + G;        // positions of one denoiser pass
  const int ctx = block_mode ? P : 0;           // context keys ahead of them
  const int Lk = ctx + L, cap = Lk + 64;       // keys; K/V capacity (whole key tiles)
  const int M = B * L, Nqkv = (H + 2 * Hkv) * dh, Nup = ffn_kind == 0 ? F : 2 * F;
  // head rows: the positions still masked before a reverse step, floor(BL i / T) of each
  // row's BL at step i, averaged over the T steps of a block
  long long head_sum = 0;
  for (int i = 1; i <= T; ++i) head_sum += (long long)B * (((long long)BL * i) / T);
  const int Mh = std::max(1, (int)((head_sum + T / 2) / T)), ng = (V + 63) / 64;
  HIP_OK(hipSetDevice(0));
  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));

  // operands
  uint16_t* xn = random_bf16((size_t)M * d, 1.0f, 1);
  uint16_t* wqkv = random_bf16((size_t)Nqkv * d, 1.0f / sqrtf((float)d), 2);
  uint16_t* wo = random_bf16((size_t)d * H * dh, 1.0f / sqrtf((float)(H * dh)), 3);
  uint16_t* wup = random_bf16((size_t)Nup * d, 1.0f / sqrtf((float)d), 4);
  uint16_t* wdown = random_bf16((size_t)d * F, 1.0f / sqrtf((float)F), 5);
  uint16_t* ao = random_bf16((size_t)M * H * dh, 1.0f, 6);
  uint16_t* ffn = random_bf16((size_t)M * F, 1.0f, 7);
  uint16_t* q = alloc<uint16_t>((size_t)B * H * L * dh);
  uint16_t* kc = random_bf16((size_t)B * Hkv * cap * dh, 1.0f, 8);
  uint16_t* vt = random_bf16((size_t)B * Hkv * dh * cap, 1.0f, 9);
  float* x = alloc<float>((size_t)M * d);
  hipLaunchKernelGGL(fill_f32, dim3(1024), dim3(256), 0, 0, x, (size_t)M * d, 0.0f);
  std::vector<float> rope_h((size_t)(P + G) * (dh / 2) * 2);
  for (int p = 0; p < P + G; ++p)
    for (int j = 0; j < dh / 2; ++j) {
      const double ang = p * std::pow(theta, -2.0 * j / dh);
      rope_h[((size_t)p * (dh / 2) + j) * 2] = (float)std::cos(ang);
      rope_h[((size_t)p * (dh / 2) + j) * 2 + 1] = (float)std::sin(ang);
    }
  float* rope = alloc<float>(rope_h.size());
  HIP_OK(hipMemcpy(rope, rope_h.data(), rope_h.size() * 4, hipMemcpyHostToDevice));
  const int S_o = gemm_resid_slices(M, d, H * dh), S_d = gemm_resid_slices(M, d, F);
  float* part = alloc<float>((size_t)(S_o > S_d ? S_o : S_d) * M * d);
  // the RMSNorm that the residual products' slice sums write when they can (unit gains)
  float* gain = alloc<float>((size_t)d);
  hipLaunchKernelGGL(fill_f32, dim3(16), dim3(256), 0, 0, gain, (size_t)d, 1.0f);
  uint16_t* xn2 = alloc<uint16_t>((size_t)M * d);
  uint16_t* wout = random_bf16((size_t)V * d, 1.0f / sqrtf((float)d), 10);
  int32_t* hidx = alloc<int32_t>((size_t)Mh);
  hipLaunchKernelGGL(fill_iota, dim3(64), dim3(256), 0, 0, hidx, Mh);
  SamplePart* hpart = alloc<SamplePart>((size_t)Mh * ng);
  int32_t* row_map = alloc<int32_t>((size_t)M);
  int32_t* canvas = alloc<int32_t>((size_t)M);
  int32_t* choice = alloc<int32_t>((size_t)M);
  float* conf = alloc<float>((size_t)M);
  hipLaunchKernelGGL(fill_row_map, dim3(64), dim3(256), 0, 0, row_map, M, Mh);
  hipLaunchKernelGGL(fill_i32, dim3(64), dim3(256), 0, 0, canvas, M, V);  // every position masked
  // gated-MLP fusion: [LN(c); anchor] [M, 2d] x [5d, 2d] -> GELU hidden [M, 4d] and gate [M, d];
  // hidden x [d, 4d] -> x = h + gate * (. + b2)
  const bool gated = fusion_kind == 0;
  uint16_t* fa = gated ? random_bf16((size_t)M * d, 1.0f, 11) : nullptr;
  uint16_t* w1g = gated ? random_bf16((size_t)5 * d * 2 * d, 1.0f / sqrtf(2.0f * d), 12) : nullptr;
  uint16_t* w2 = gated ? random_bf16((size_t)d * 4 * d, 1.0f / sqrtf(4.0f * d), 13) : nullptr;
  uint16_t* fus_h = gated ? alloc<uint16_t>((size_t)M * 4 * d) : nullptr;
  float* fus_g = gated ? alloc<float>((size_t)M * d) : nullptr;
  float* fbias = gated ? alloc<float>((size_t)5 * d) : nullptr;
  float* fh = gated ? alloc<float>((size_t)M * d) : nullptr;
  if (gated) {
    hipLaunchKernelGGL(fill_f32, dim3(64), dim3(256), 0, 0, fbias, (size_t)5 * d, 0.01f);
    hipLaunchKernelGGL(fill_f32, dim3(1024), dim3(256), 0, 0, fh, (size_t)M * d, 0.5f);
  }
  const size_t copy_n = (size_t)M * d / 4;  // float4 granules of one [M, d] float32 row block
  float* copy_dst = alloc<float>((size_t)M * d);
  HIP_OK(hipDeviceSynchronize());

  printf("kernel_bench: M = %d x %d = %d rows, d %d, heads %d/%d x %d, ffn %d (%s), keys %d; K slices %d / %d; "
         "head %d rows x V %d\n", B, L, M, d, H, Hkv, dh, F, ffn_kind == 0 ? "gelu" : ffn_kind == 1 ? "swiglu" : "geglu",
         Lk, S_o, S_d, Mh, V);
  fflush(stdout);
  hipEvent_t e0, e1;
  HIP_OK(hipEventCreate(&e0));
  HIP_OK(hipEventCreate(&e1));
  auto stage = [&](const char* name, double flops, auto&& launch) {
    HIP_OK(launch());
    HIP_OK(hipStreamSynchronize(st));
    HIP_OK(hipEventRecord(e0, st));
    for (int r = 0; r < reps; ++r) HIP_OK(launch());
    HIP_OK(hipEventRecord(e1, st));
    HIP_OK(hipEventSynchronize(e1));
    float ms = 0;
    HIP_OK(hipEventElapsedTime(&ms, e0, e1));
    const double us = 1e3 * ms / reps;
    printf("kernel_bench: %-8s %10.2f us per launch", name, us);
    if (flops > 0) printf("  %8.1f TFLOP/s", flops / (us * 1e-6) / 1e12);
    printf("\n");
    fflush(stdout);
  };
  stage("copy", 0.0, [&]() {
    hipLaunchKernelGGL(copy_kernel, dim3((unsigned)((copy_n + 255) / 256)), dim3(256), 0, st,
                       reinterpret_cast<const float4*>(x), reinterpret_cast<float4*>(copy_dst), copy_n);
    return hipGetLastError();
  });
  stage("qkv", 2.0 * M * d * Nqkv, [&]() {
    GemmProblem p{M, Nqkv, d, xn, d, d, nullptr, 0, wqkv, d};
    EpiParams e;
    e.L = L;
    e.pos0 = ctx;
    e.H = H;
    e.Hkv = Hkv;
    e.dh = dh;
    e.kv_cap = cap;
    e.kv_off = ctx;
    e.rope = rope;
    e.q = q;
    e.k = kc;
    e.vt = vt;
    return gemm(BF16, p, EPI_QKV_ROPE, e, st);
  });
  stage("attn", 4.0 * B * H * (double)L * Lk * dh,
        [&]() { return attention(BF16, q, kc, vt, ao, B, H, Hkv, L, Lk, cap, dh, st); });
  stage("oproj", 2.0 * M * H * dh * d, [&]() {
    GemmProblem p{M, d, H * dh, ao, H * dh, H * dh, nullptr, 0, wo, H * dh};
    EpiParams e;
    e.resid = x;
    e.ldr = d;
    if (S_o > 1) e.part = part;
    if (gemm_resid_norms(M, d, H * dh)) {
      e.norm_g = gain;
      e.norm_eps = 1e-6f;
      e.norm_out = xn2;
    }
    return gemm(BF16, p, EPI_RESID, e, st);
  });
  stage("ffn_up", 2.0 * M * d * Nup, [&]() {
    GemmProblem p{M, Nup, d, xn, d, d, nullptr, 0, wup, d};
    EpiParams e;
    e.out = ffn;
    e.ldo = F;
    return gemm(BF16, p, ffn_kind == 0 ? EPI_GELU : ffn_kind == 1 ? EPI_GLU_SILU : EPI_GLU_GELU, e, st);
  });
  stage("ffn_down", 2.0 * M * F * d, [&]() {
    GemmProblem p{M, d, F, ffn, F, F, nullptr, 0, wdown, F};
    EpiParams e;
    e.resid = x;
    e.ldr = d;
    if (S_d > 1) e.part = part;
    if (gemm_resid_norms(M, d, F)) {
      e.norm_g = gain;
      e.norm_eps = 1e-6f;
      e.norm_out = xn2;
    }
    return gemm(BF16, p, EPI_RESID, e, st);
  });
  stage("head", 2.0 * Mh * d * V, [&]() {
    GemmProblem p{Mh, V, d, xn, d, d, nullptr, 0, wout, d};
    EpiParams e;
    e.rows_idx = hidx;
    e.Lc = L;
    e.pos_base = ctx;
    e.n_groups = ng;
    e.step_id = 1;
    e.k0 = 0x2545F491u;
    e.k1 = 0x4F6CDD1Du;
    e.part = hpart;
    return head_sample(p, e, st);
  });
  stage("sample", 0.0, [&]() { return sample_finalize(hpart, ng, V, row_map, canvas, B, L, 0, V, choice, conf, st); });
  if (gated) {
    stage("fusion1", 2.0 * M * 5.0 * d * 2 * d, [&]() {
      GemmProblem p{M, 5 * d, 2 * d, xn, d, d, fa, d, w1g, 2 * d};
      EpiParams e;
      e.out = fus_h;
      e.ldo = 4 * d;
      e.bias = fbias;
      e.out2 = fus_g;
      e.ldo2 = d;
      e.split = 4 * d;
      return gemm(BF16, p, EPI_FUSION1, e, st);
    });
    stage("fusion2", 2.0 * M * d * 4.0 * d, [&]() {
      GemmProblem p{M, d, 4 * d, fus_h, 4 * d, 4 * d, nullptr, 0, w2, 4 * d};
      EpiParams e;
      e.resid = x;
      e.ldr = d;
      e.bias = fbias;
      e.aux = fh;
      e.ld_aux = d;
      e.gate = fus_g;
      e.ldg = d;
      return gemm(BF16, p, EPI_FUSION2, e, st);
    });
  }
  HIP_OK(hipStreamSynchronize(st));
  for (void* p : {(void*)row_map, (void*)canvas, (void*)choice, (void*)conf, (void*)fa, (void*)w1g, (void*)w2,
                  (void*)fus_h, (void*)fus_g, (void*)fbias, (void*)fh})
    if (p) HIP_OK(hipFree(p));
  for (void* p : {(void*)xn, (void*)wqkv, (void*)wo, (void*)wup, (void*)wdown, (void*)ao, (void*)ffn, (void*)q,
                  (void*)kc, (void*)vt, (void*)x, (void*)rope, (void*)part, (void*)copy_dst, (void*)gain,
                  (void*)xn2, (void*)wout, (void*)hidx, (void*)hpart})
    HIP_OK(hipFree(p));
  HIP_OK(hipStreamDestroy(st));
  return 0;
}
