// tadm_run: one or more whole generations of a workload through the C ABI of
// libtadm.so, from C++ without Python or PyTorch.  It serves as a native example of
// the boundary and as the program that per-kernel hardware counters are taken on.
//
//   tadm_run key=value ...
//
// Model keys are the tadm_config fields (vocab, d_model, n_heads, n_kv_heads,
// head_dim, d_ffn, ffn_kind, n_shared, n_anchor, n_denoise, fusion_kind, fusion_rank,
// paired_heads, dtype, rms_eps, ln_eps, rope_theta); workload keys are batch,
// prompt_len, gen_len, block_len, T, K, seed, temperature and gens (generations to
// run, default 1).  max_batch / max_seq follow from the workload.  Weights are seeded
// uniform values scaled by 1/sqrt(fan-in) (vectors: 1), prompts seeded uniform token
// ids: the work of each kernel depends on the shapes and the unmask schedule only.
// Prints one line per generation (its time from HIP events) and a checksum of the
// tokens; exits non-zero on any error, or (4) when the output lost a prompt token or
// holds an id outside [0, vocab).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "tadm.h"

namespace {

#define HIP_OK(x)                                                                      \
  do {                                                                                 \
    hipError_t e_ = (x);                                                               \
    if (e_ != hipSuccess) {                                                            \
      fprintf(stderr, "tadm_run: %s at line %d: %s\n", #x, __LINE__, hipGetErrorString(e_)); \
      exit(2);                                                                         \
    }                                                                                  \
  } while (0)
#define TADM_OK_(x)                                                                    \
  do {                                                                                 \
    tadm_status s_ = (x);                                                              \
    if (s_ != TADM_OK) {                                                               \
      fprintf(stderr, "tadm_run: %s: status %d: %s\n", #x, (int)s_, tadm_last_error()); \
      exit(3);                                                                         \
    }                                                                                  \
  } while (0)

__device__ __forceinline__ uint32_t mix32(uint64_t x) {
  x ^= x >> 33;
  x *= 0xff51afd7ed558ccdull;
  x ^= x >> 33;
  x *= 0xc4ceb9fe1a85ec53ull;
  x ^= x >> 33;
  return (uint32_t)x;
}

// out[i] = scale * u, u uniform in [-1, 1) from a hash of (seed, i); bf16 keeps the
// upper half of the float32 pattern
__global__ void fill_kernel(void* out, size_t n, int bf16, float scale, uint64_t seed) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const float u = (float)(mix32(seed * 0x9e3779b97f4a7c15ull + i) >> 8) * (1.0f / 8388608.0f) - 1.0f;
    const float v = scale * u;
    if (bf16) {
      uint32_t b;
      memcpy(&b, &v, 4);
      static_cast<uint16_t*>(out)[i] = (uint16_t)(b >> 16);
    } else {
      static_cast<float*>(out)[i] = v;
    }
  }
}

__global__ void fill_const_kernel(void* out, size_t n, int bf16, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    if (bf16) {
      uint32_t b;
      memcpy(&b, &v, 4);
      static_cast<uint16_t*>(out)[i] = (uint16_t)(b >> 16);
    } else {
      static_cast<float*>(out)[i] = v;
    }
  }
}

__global__ void tokens_kernel(int32_t* out, size_t n, int32_t vocab, uint64_t seed) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    out[i] = (int32_t)((uint64_t)mix32(seed * 0x9e3779b97f4a7c15ull + i) * (uint64_t)vocab >> 32);
}

double num(const std::map<std::string, std::string>& kv, const char* k, double dflt, bool required = false) {
  auto it = kv.find(k);
  if (it == kv.end()) {
    if (required) {
      fprintf(stderr, "tadm_run: missing %s=...\n", k);
      exit(1);
    }
    return dflt;
  }
  char* end = nullptr;
  const double v = strtod(it->second.c_str(), &end);
  if (!end || *end) {
    fprintf(stderr, "tadm_run: bad value %s=%s\n", k, it->second.c_str());
    exit(1);
  }
  return v;
}

}  // namespace

int main(int argc, char** argv) {
  std::map<std::string, std::string> kv;
  for (int a = 1; a < argc; ++a) {
    const char* eq = strchr(argv[a], '=');
    if (!eq) {
      fprintf(stderr, "usage: tadm_run key=value ...  (bad argument '%s')\n", argv[a]);
      return 1;
    }
    kv[std::string(argv[a], eq - argv[a])] = eq + 1;
  }
  const int B = (int)num(kv, "batch", 0, true), P = (int)num(kv, "prompt_len", 0, true);
  const int G = (int)num(kv, "gen_len", 0, true), T = (int)num(kv, "T", 0, true);
  const int K = (int)num(kv, "K", 4), BL = (int)num(kv, "block_len", G), gens = (int)num(kv, "gens", 1);
  const uint64_t seed = (uint64_t)num(kv, "seed", 2);
  const float temperature = (float)num(kv, "temperature", 1.0);

  tadm_config c{};
  c.vocab = (int)num(kv, "vocab", 0, true);
  c.d_model = (int)num(kv, "d_model", 0, true);
  c.n_heads = (int)num(kv, "n_heads", 0, true);
  c.n_kv_heads = (int)num(kv, "n_kv_heads", c.n_heads);
  c.head_dim = (int)num(kv, "head_dim", 0, true);
  c.d_ffn = (int)num(kv, "d_ffn", 0, true);
  c.ffn_kind = (int)num(kv, "ffn_kind", TADM_FFN_SWIGLU);
  c.n_shared = (int)num(kv, "n_shared", 0);
  c.n_anchor = (int)num(kv, "n_anchor", 0, true);
  c.n_denoise = (int)num(kv, "n_denoise", 0, true);
  c.fusion_kind = (int)num(kv, "fusion_kind", TADM_FUSION_GATED_MLP);
  c.fusion_rank = (int)num(kv, "fusion_rank", 0);
  c.paired_heads = (int)num(kv, "paired_heads", 4);
  c.dtype = (int)num(kv, "dtype", TADM_DTYPE_BF16);
  c.max_batch = B;
  c.max_seq = P + G;
  c.rms_eps = (float)num(kv, "rms_eps", 1e-6);
  c.ln_eps = (float)num(kv, "ln_eps", 1e-5);
  c.rope_theta = (float)num(kv, "rope_theta", 10000.0);
  if (B <= 0 || G <= 0 || T <= 0 || K <= 0 || BL <= 0 || gens <= 0 || P < 0) {
    fprintf(stderr, "tadm_run: batch, gen_len, T, K, block_len and gens must be positive, prompt_len >= 0\n");
    return 1;
  }

  HIP_OK(hipSetDevice(0));
  tadm_model* m = nullptr;
  TADM_OK_(tadm_model_create(&c, &m));
  const int bf16 = c.dtype == TADM_DTYPE_BF16, esz = bf16 ? 2 : 4;
  const int nw = tadm_weight_count(&c);
  size_t most = 0;
  std::vector<std::pair<int64_t, int64_t>> shapes(nw);
  for (int i = 0; i < nw; ++i) {
    TADM_OK_(tadm_weight_info(&c, i, &shapes[i].first, &shapes[i].second));
    const size_t n = (size_t)shapes[i].first * (size_t)(shapes[i].second > 0 ? shapes[i].second : 1);
    most = n > most ? n : most;
  }
  void* staging = nullptr;
  HIP_OK(hipMalloc(&staging, most * esz));
  for (int i = 0; i < nw; ++i) {
    const int64_t rows = shapes[i].first, cols = shapes[i].second;
    const size_t n = (size_t)rows * (size_t)(cols > 0 ? cols : 1);
    if (cols > 0)
      hipLaunchKernelGGL(fill_kernel, dim3(4096), dim3(256), 0, 0, staging, n, bf16, 1.0f / sqrtf((float)cols),
                         (uint64_t)1000 + i);
    else
      hipLaunchKernelGGL(fill_const_kernel, dim3(1024), dim3(256), 0, 0, staging, n, bf16, 1.0f);
    HIP_OK(hipGetLastError());
    HIP_OK(hipDeviceSynchronize());
    TADM_OK_(tadm_model_load_weight(m, i, staging, n * esz, 1));
  }
  HIP_OK(hipFree(staging));

  int32_t *prompt = nullptr, *tokens = nullptr;
  if (P > 0) {
    HIP_OK(hipMalloc(&prompt, (size_t)B * P * sizeof(int32_t)));
    hipLaunchKernelGGL(tokens_kernel, dim3(256), dim3(256), 0, 0, prompt, (size_t)B * P, c.vocab, (uint64_t)1);
    HIP_OK(hipGetLastError());
  }
  HIP_OK(hipMalloc(&tokens, (size_t)B * (P + G) * sizeof(int32_t)));
  hipStream_t st;
  HIP_OK(hipStreamCreate(&st));
  TADM_OK_(tadm_set_stream(m, st));
  HIP_OK(hipDeviceSynchronize());
  hipEvent_t e0, e1;
  HIP_OK(hipEventCreate(&e0));
  HIP_OK(hipEventCreate(&e1));
  printf("tadm_run: d%d %dx%d heads (%d kv) ffn %d V%d, %d + %d layers; B=%d, prompt %d + %d generated (block %d), "
         "T=%d, K=%d\n",
         c.d_model, c.n_heads, c.head_dim, c.n_kv_heads, c.d_ffn, c.vocab, c.n_anchor, c.n_denoise, B, P, G, BL, T, K);
  fflush(stdout);
  for (int g = 0; g < gens; ++g) {
    HIP_OK(hipEventRecord(e0, st));
    TADM_OK_(tadm_generate(m, prompt, B, P, G, T, K, BL, seed, temperature, tokens));
    HIP_OK(hipEventRecord(e1, st));
    HIP_OK(hipEventSynchronize(e1));
    float ms = 0;
    HIP_OK(hipEventElapsedTime(&ms, e0, e1));
    printf("tadm_run: generation %d: %.3f ms, %.1f tokens/s\n", g, ms, (double)B * G / (ms * 1e-3));
    fflush(stdout);
  }
  HIP_OK(hipStreamSynchronize(st));
  // the output keeps the prompt and holds real token ids only (no mask id left)
  std::vector<int32_t> host((size_t)B * (P + G)), hprompt((size_t)B * P);
  HIP_OK(hipMemcpy(host.data(), tokens, host.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  if (P > 0) HIP_OK(hipMemcpy(hprompt.data(), prompt, hprompt.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  size_t bad = 0;
  uint64_t sum = 0;
  for (int b = 0; b < B; ++b)
    for (int j = 0; j < P + G; ++j) {
      const int32_t t = host[(size_t)b * (P + G) + j];
      if (j < P ? t != hprompt[(size_t)b * P + j] : (t < 0 || t >= c.vocab)) ++bad;
      sum = sum * 1000003u + (uint32_t)t;
    }
  printf("tadm_run: tokens checksum %016llx, %zu invalid\n", (unsigned long long)sum, bad);
  TADM_OK_(tadm_model_destroy(m));
  HIP_OK(hipStreamDestroy(st));
  if (prompt) HIP_OK(hipFree(prompt));
  HIP_OK(hipFree(tokens));
  return bad ? 4 : 0;
}
