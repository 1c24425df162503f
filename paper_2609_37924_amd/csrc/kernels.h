// Host-side launchers of the TADM kernels.  All enqueue on the given stream and
// return the launch status; shapes are validated by the caller (runtime.cpp).
#pragma once
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stdint.h>

namespace tadm {

// Start/stop events for the next timed launch made on this host thread (null: untimed).
// The events take the dispatch's own begin and end timestamps (hipExtLaunchKernel), so
// timing a kernel adds no packets to the stream.  The launch consumes them.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchEvents next_launch_events;

template <typename F, typename... Args>
inline void launch_timed(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  const LaunchEvents ev = next_launch_events;
  next_launch_events = LaunchEvents{};
  if (ev.start)
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev.start, ev.stop, 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}

enum DType { F32 = 0, BF16 = 1 };

// C[m, n] = sum_k A[m, k] * W[n, k].  A is [M, K] row-major, split along K:
// columns [0, K1) come from A1 (row stride lda1), [K1, K) from A2 (lda2).
// W is [N, K] row-major (row n = weights of output feature n).
struct GemmProblem {
  int M, N, K;
  const void* A1; int lda1; int K1;
  const void* A2; int lda2;
  const void* W;  int ldw;
  const int* M_dev = nullptr;  // if set: rows actually present (<= M; M sizes the grid)
  int rm = 0, rn = 0;          // per-XCD tile region (set by the launcher)
  int gm = 0, gn = 0;          // blocks an XCD runs at once, as gm x gn tiles of its region (0: m first)
  int band = 0;                // no even region split: band height of the banded walk (set by the launcher)
  int ksplit = 1;              // K slices (grid.y); slice s writes out + s * split_stride
  int w_first = 0;             // more weight rows than activation rows (N > M; set by the launcher)
};

enum EpiKind {
  EPI_STORE = 0,      // out(T)[m, n] = acc
  EPI_STORE_F32,      // out(float)[m, n] = acc
  EPI_RESID,          // resid(float)[m, n] += acc (bf16 with part set and a long K: split
                      // over K into part [S, M, N], then an ordered sum into resid)
  EPI_GELU,           // out(T)[m, n] = gelu(acc)
  EPI_GLU_SILU,       // out(T)[m, f] = silu(gate) * up   (16-row interleaved weights)
  EPI_GLU_GELU,       // out(T)[m, f] = gelu(gate) * up
  EPI_FUSION1,        // n < split: out(T)[m, n] = gelu(acc + bias[n]);  else out2(float)[m, n-split] = sigmoid(acc + bias[n])
  EPI_FUSION2,        // resid(float)[m, n] = aux[m, n] + gate[m, n] * (acc + bias[n])
  EPI_SILU,           // out(T)[m, n] = silu(acc)
  EPI_ADD_F32,        // out(float)[m, n] = aux[m, n] + acc
  EPI_ADD_BOTH,       // out(float)[m, n] = aux[m, n] + acc and out_t(T)[m, n] = the same value
  EPI_ADD_SUB,        // out_t(T)[m, n] = (aux[m, n] + acc) - aux2[m, n]
  EPI_PAIRED,         // out(float)[m, n] = aux[m, n] + row1[m] * row2[m] * acc
  EPI_QKV_ROPE,       // q/k/v projection: rotary embedding on q, k (pair-interleaved
                      // weight rows) and scatter into the attention layouts (see EpiParams)
  EPI_SAMPLE,         // vocabulary projection: sampling partials per (row, 64-column
                      // group) instead of logits (head_sample only; see EpiParams)
  EPI_SCALE_F32,      // out(float)[m, n] = row1[m] * acc; with part set and long K the
                      // product is split over K into part [S, M, N] and reduced in order
};

struct EpiParams {
  void* out = nullptr;  int ldo = 0;
  float* resid = nullptr; int ldr = 0;
  const float* bias = nullptr;
  const float* aux = nullptr; int ld_aux = 0;
  const float* gate = nullptr; int ldg = 0;
  float* out2 = nullptr; int ldo2 = 0;
  int split = 0;
  const float* aux2 = nullptr; int ld_aux2 = 0;
  const float* row1 = nullptr;   // per-row factors
  const float* row2 = nullptr;
  void* out_t = nullptr; int ld_out_t = 0;
  // EPI_QKV_ROPE: token m is (row m / L, position pos0 + m % L).  Output feature n is in
  // head slot n / dh (q heads, then k heads, then v heads); within a q/k head the weight
  // rows are ordered (0, dh/2, 1, dh/2 + 1, ...), so features 2j, 2j + 1 are the rotary
  // pair (j, j + dh/2).  Q [B, H, L, dh], K rows kv_off + l of [B, Hkv, kv_cap, dh],
  // V^T columns kv_off + l of [B, Hkv, dh, kv_cap].
  int L = 0, pos0 = 0, H = 0, Hkv = 0, dh = 0, kv_cap = 0, kv_off = 0;
  // n / L and n / dh as (umulhi(n, mul) + n) >> shift (n < 2^31), set by gemm()
  uint32_t l_mul = 0, dh_mul = 0;
  int l_shift = 0, dh_shift = 0;
  const float* rope = nullptr;  // (cos, sin) of position p and rotary pair j at rope[2 (p dh/2 + j)]
  void* q = nullptr;
  void* k = nullptr;
  void* vt = nullptr;
  // EPI_SAMPLE: row m is canvas entry rows_idx[m] = b * Lc + j at absolute position
  // pos_base + j; the sampling contract's Philox key (k0, k1), step id and 1/temp;
  // part receives n_groups SamplePart records per row.
  const int32_t* rows_idx = nullptr;
  int Lc = 0, pos_base = 0, n_groups = 0;
  uint32_t step_id = 0, k0 = 0, k1 = 0;
  float inv_temp = 1.f;
  void* part = nullptr;
  size_t split_stride = 0;  // elements between the K slices' outputs (EPI_STORE_F32, ksplit > 1)
  // EPI_RESID split over K with gemm_resid_norms(M, N, K): the ordered sum of the slices
  // also writes the RMSNorm of each updated row, norm_out[m, :] (bf16) =
  // resid[m, :] * rsqrt(mean(resid[m, :]^2) + norm_eps) * norm_g
  const float* norm_g = nullptr;
  float norm_eps = 0.f;
  void* norm_out = nullptr;
};

// Sampling partial of one (row, 64-entry vocabulary group): the group maximum m_g of
// the scaled logits, its fixed-point sum S_g, and its exact best Gumbel score with the
// entry's id and scaled logit.
struct SamplePart {
  float m, score, lp;
  int v;
  long long S;
};

hipError_t gemm(DType dt, const GemmProblem& p, EpiKind epi, const EpiParams& e, hipStream_t s);
// Division by a fixed d >= 1 as q = (umulhi(n, mul) + n) >> shift, exact for 0 <= n < 2^31
// (Granlund-Montgomery; mul = floor(2^32 (2^shift - d) / d) + 1, shift = ceil(log2 d)).
inline void fast_divider(uint32_t d, uint32_t& mul, int& shift) {
  shift = 0;
  while ((1ull << shift) < d) ++shift;
  mul = (uint32_t)(((1ull << 32) * ((1ull << shift) - d)) / d + 1);
}
// K slices the bf16 EPI_SCALE_F32 product uses (1: no split); its part buffer needs
// slices * M * N floats.
int gemm_split_slices(int M, int N, int K);
// K slices of a bf16 EPI_RESID product given a part buffer (1: no split; else
// part holds slices * M * N floats): long K with few 128 x 128 tiles.
int gemm_resid_slices(int M, int N, int K);
// Whether a bf16 EPI_RESID product of this shape (split over K) can also write the RMSNorm
// of its updated rows (EpiParams::norm_out); otherwise the caller normalises them.
bool gemm_resid_norms(int M, int N, int K);

// ---- norms / embedding / elementwise (norm.hip)
// out[t, :] = embed[tok[t], :] as float32; `embed` has table_rows rows of length d
// (ids outside [0, table_rows) are clamped so that the gather stays in bounds).
hipError_t embed_gather(DType dt, const int32_t* tok, int n_tok, const void* embed, int table_rows,
                        int d, float* out, hipStream_t s);
// y(T) = x / sqrt(mean(x^2) + eps) * g over rows of length d.  Row r of the
// output is taken from input row map(r) = (r / rows_per_b) * in_stride_b + in_off + r % rows_per_b
// (a gather of the canvas columns); pass rows_per_b = n_rows, in_stride_b = 0, in_off = 0 for identity.
hipError_t rms_norm(DType dt, const float* x, const float* g, float eps, int n_rows, int d,
                    int rows_per_b, int in_stride_b, int in_off, void* y, hipStream_t s);
// Gathered RMSNorm: output row r < *count is input token row
// (c / Lc) * L + off + c % Lc with c = canvas_idx[r]; rows >= *count are skipped.
hipError_t rms_norm_gather(DType dt, const float* x, const float* g, float eps, const int32_t* canvas_idx,
                           const int* count, int max_rows, int Lc, int L, int off, int d, void* y,
                           hipStream_t s);
// LayerNorm with affine; output as T (y_t) or float (y_f), whichever is non-null.
hipError_t layer_norm(DType dt, const float* x, const float* w, const float* b, float eps,
                      int n_rows, int d, void* y_t, float* y_f, hipStream_t s);
// x = LayerNorm(x) (affine w, b; in place), then y(T) = RMSNorm(x) * g: a layer_norm followed
// by rms_norm of its result, with the same arithmetic, in one kernel.
hipError_t layer_rms_norm(DType dt, float* x, const float* w, const float* b, float ln_eps, const float* g,
                          float rms_eps, int n_rows, int d, void* y, hipStream_t s);
hipError_t copy_f32(const float* src, float* dst, size_t n, hipStream_t s);
hipError_t to_f32(DType dt, const void* src, float* dst, size_t n, hipStream_t s);
// out[r, f] = act(pre[r, gate_row(f)]) * pre[r, up_row(f)] for the fp32 GLU path.
hipError_t glu_f32(const float* pre, int n_rows, int F, int silu, float* out, hipStream_t s);

// ---- paired-attention fusion helpers (fusion.hip)
// s[r] = sqrt(mean_j x[r, j]^2 + eps)
hipError_t row_rms(const float* x, int n_rows, int d, float eps, float* s, hipStream_t st);
// y(T)[r, :] = x[r, :] / s[r]
hipError_t scale_rows(DType dt, const float* x, const float* s, int n_rows, int d, void* y, hipStream_t st);
// y(T) = x (float -> model type), n elements
hipError_t to_type(DType dt, const float* x, size_t n, void* y, hipStream_t st);
// F(T) [N, 4r] = [U; Z0; Z - Z0; M] (feature concatenation); U, Z0, Z float, M in T
hipError_t paired_features(DType dt, const float* U, const float* Z0, const float* Z, const void* M, int n_rows,
                           int r, void* F, hipStream_t st);
// g[r] = sigmoid(sum_j G1(T)[r, j] * w[j] + b)
hipError_t row_gate(DType dt, const void* G1, const float* w, const float* b, int n_rows, int r, float* g,
                    hipStream_t st);

// ---- rotary + head split (attention.hip)
// qkv(T) [B*L, (H + 2*Hkv)*dh] -> Q(T) [B, H, L, dh] (rotated), K(T) rows
// [b, hk, off + l, :] of a [B, Hkv, kv_cap, dh] buffer (rotated), Vt(T) [b, hk, :, off + l]
// of a [B, Hkv, dh, kv_cap] buffer.  Positions pos0 + l; cos/sin tables [max_pos, dh/2];
// with null tables the heads are split without rotation.
hipError_t rope_split(DType dt, const void* qkv, int B, int L, int H, int Hkv, int dh, int pos0,
                      const float* cos_t, const float* sin_t, void* Q, void* K, void* Vt,
                      int kv_cap, int kv_off, hipStream_t s);
// O(T) [B*Lq, H*dh] = softmax(Q K^T / sqrt(dh)) V over keys [0, Lk) of the K/Vt buffers.
hipError_t attention(DType dt, const void* Q, const void* K, const void* Vt, void* O, int B, int H,
                     int Hkv, int Lq, int Lk, int kv_cap, int dh, hipStream_t s);

// ---- sampler (sampler.hip)
// List of masked canvas positions: idx[r] = b * Lc + j for the r-th masked entry
// (row-major order), row_map[b * Lc + j] = r or -1, *count = number of entries; only
// the first `bound` masked entries get a row (the rest row_map -1, count <= bound).
hipError_t compact_masked(const int32_t* canvas, int B, int L, int canvas_off, int mask_id, int bound,
                          int32_t* idx, int32_t* row_map, int* count, hipStream_t s);
// Vocabulary projection of the masked rows with the sampler in the epilogue (bf16):
// p is the head GEMM (M = compacted masked rows, M_dev their device count, N = V);
// e carries the EPI_SAMPLE fields.  Writes p.M x ceil(V / 64) partials to e.part.
hipError_t head_sample(const GemmProblem& p, const EpiParams& e, hipStream_t s);
// Merges the partials of every masked canvas position into its token and confidence
// (row_map: canvas entry -> partial row); other positions get -1 / -inf.
hipError_t sample_finalize(const SamplePart* part, int n_groups, int V, const int32_t* row_map,
                           const int32_t* canvas, int B, int L, int canvas_off, int mask_id, int32_t* choice,
                           float* conf, hipStream_t s);
// Remasking posterior: per entry of canvas rows [b, off + j), one uniform u = Philox
// word 0 at counter (2^31, pos0 + off + j, b, step_id); masked -> choice iff
// u < p_unmask, decoded -> mask iff u < sigma; columns before off are copied.
hipError_t remask_update(const int32_t* canvas, const int32_t* choice, int B, int L, int canvas_off, int mask_id,
                         int pos0, uint32_t step_id, uint64_t seed, float p_unmask, float sigma, int32_t* next,
                         hipStream_t s);
// Entropy-bound sampler of Algorithm 2 (usdm.hip), rows b * Lc + j at absolute
// positions pos_base + j.  Per row: xhat = argmax of the logits, xtilde = Gumbel-max
// draw of softmax(l * inv_temp), H / Hq = entropy in float and 2^-40 fixed point,
// rscale = 2^40 / A (the softmax normaliser's reciprocal, for the self-conditioning
// product); P (nullable, element type pt, leading dimension ldp >= V) receives the
// unnormalised weights exp(l' - m), zero on columns [V, ldp).
hipError_t entropy_stats(const float* logits, int B, int Lc, int V, int pos_base, uint32_t step_id, uint64_t seed,
                         float inv_temp, int32_t* xhat, int32_t* xtilde, float* H, long long* Hq, float* rscale,
                         DType pt, void* P, int ldp, hipStream_t s);
// Acceptance and next canvas [B, L] (columns before off copied; next may alias canvas):
// accepted positions take xtilde, the others a uniform token; last != 0 writes xhat.
// Needs (L - off) * 8 bytes of LDS (L - off <= 8192).
hipError_t entropy_accept(const long long* Hq, const int32_t* xhat, const int32_t* xtilde, const int32_t* canvas,
                          int32_t* next, int B, int L, int off, int pos_base, uint32_t step_id, uint64_t seed, int V,
                          long long etaq, int last, hipStream_t s);
// A block's first canvas: uniform tokens of positions pos_base + t into tok[b * ld + col0 + t].
hipError_t init_uniform_tokens(int32_t* tok, int ld, int col0, int B, int n, int pos_base, uint32_t block,
                               uint64_t seed, int V, hipStream_t s);
// c[b, off + j, :] += sc[b * (L - off) + j, :] (d % 4 == 0).
hipError_t add_selfcond(float* c, const float* sc, int B, int L, int off, int d, hipStream_t s);
// ET[n, v] = E[v, n] (v < V), zero for V <= v < ldt: E [V, d] row-major, ET [d, ldt].
hipError_t transpose_rows(DType dt, const void* E, int V, int d, void* ET, int ldt, hipStream_t s);
constexpr int ENTROPY_MAX_CANVAS = 8192;
// Training objective (train.hip).  zt / zs [B, L] = the stale pair of clean tokens x:
// masked iff u < float((1 - eps) t_b) (resp. t'_b), u from Philox word 0 at counter
// (2^31 + 3, l, b, step).
hipError_t corrupt_pair(const int32_t* x, int B, int L, const float* t, const float* ts, float eps, uint64_t seed,
                        uint32_t step, int mask_id, int32_t* zt, int32_t* zs, hipStream_t s);
// ce[r] = logsumexp(logits[r]) - logits[r][x[idx[r]]] for the rows r < *count (grid max_rows).
hipError_t masked_ce(const float* logits, int V, int max_rows, const int* count, const int32_t* idx, const int32_t* x,
                     float* ce, hipStream_t s);
// loss[b] = (1 / t_b) sum_{l masked} ce[row_map[b L + l]] (row_map -1: not masked); n_masked nullable.
hipError_t weighted_loss(const float* ce, const int32_t* row_map, int B, int L, const float* t, float* loss,
                         int32_t* n_masked, hipStream_t s);
// Largest vocabulary the sampler handles: its per-group partials (64 entries per
// group, 12 bytes each) live in 48 KB of LDS.
constexpr int SAMPLE_MAX_VOCAB = 4096 * 64;
// For every masked canvas position: Gumbel-max token and fixed-point confidence.
// Logits row of position (b, j) is row_map[b * Lc + j] if row_map is set, else b * Lc + j.
// Nucleus threshold of one masked position: the global maximum m of the scaled logits
// and the weight threshold tau of the top-p nucleus {v : rint(exp(l'_v - m) 2^40) >= tau}.
// y_in / y_out screen membership without the exponential: y = l'_v - m >= y_in implies
// v is in the nucleus, y < y_out that it is not (margins cover the error of the float32
// exponential and the rounding to integer weights); only y in between is tested exactly.
struct NucleusThr {
  float m;
  float y_in, y_out;
  int pad;
  long long tau;
};
// For every masked canvas position, its nucleus threshold at top_p (0 < top_p < 1);
// thr is indexed like choice / conf (b * Lc + j).
hipError_t nucleus_thresholds(const float* logits, const int32_t* row_map, const int32_t* canvas, int B, int L,
                              int canvas_off, int V, int mask_id, float inv_temp, float top_p, NucleusThr* thr,
                              hipStream_t s);
// thr (nullable): draw each token from its position's nucleus.
hipError_t sample_tokens(const float* logits, const int32_t* row_map, const NucleusThr* thr, const int32_t* canvas,
                         int B, int L, int canvas_off, int V, int mask_id, int pos0, uint32_t step_id,
                         uint64_t seed, float inv_temp, int32_t* choice, float* conf, hipStream_t s);
// Per row: reveal the n most confident masked positions (n = n_rows[b] if n_rows is
// set, else n_unmask; clamped to the row's masked count); copy the rest.
hipError_t select_unmask(const int32_t* canvas, const int32_t* choice, const float* conf, int B,
                         int L, int canvas_off, int mask_id, int n_unmask, const int32_t* n_rows, int32_t* next,
                         hipStream_t s);

}  // namespace tadm

namespace tadm {
// ---- weight placement and small copies (norm.hip)
// dst row map(r) <- src row r (cols elements) for r < rows.  map(r) = row_off + r,
// or, for glu_half >= 0, row_off + 32*(r/16) + 16*glu_half + r%16 (gate/up interleave
// in 16-row blocks).  Elements keep the model type (dst_f32 = 0) or become float32.
// rope_dh > 0: rows are heads of rope_dh rows reordered as (0, h, 1, h + 1, ...), h = rope_dh / 2.
hipError_t scatter_rows(DType dt, const void* src, long rows, int cols, void* dst, int dst_f32,
                        long row_off, int glu_half, int rope_dh, hipStream_t s);
// canvas rows: dst[b, :] = concat(prompt[b, :P], mask_id * gen)
hipError_t init_canvas(const int32_t* prompt, int B, int P, int gen, int mask_id, int32_t* dst,
                       hipStream_t s);
hipError_t fill_i32(int32_t* dst, size_t n, int32_t v, hipStream_t s);
}  // namespace tadm
