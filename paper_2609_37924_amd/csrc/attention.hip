// Rotary embedding + head split, and bidirectional softmax attention.
//
// bf16 attention: one workgroup = 64 queries of one batch row for the G query heads
// that share one K/V head (grouped-query attention: G = H / Hkv), 4 G wave64s with 16
// queries of one head each, so that every K/V tile brought into LDS serves all G heads.
// K (64 keys x dh) and V^T (dh x 64 keys) tiles move global -> LDS
// with global_load_lds_dwordx4 into a 2-stage ring (16-byte chunks swizzled by row).  Scores are computed transposed, S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16, so that each lane owns one query: the online-softmax
// statistics live in the lane and the probabilities feed the O^T = V^T P^T MFMA
// directly from registers (the k index of that product walks keys in the order the
// score accumulators hold them, and V^T is read in the same order).
#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

// grid: x = B * ceil(L/64) token tiles, y = H + 2*Hkv head slots.
template <class T>
__global__ __launch_bounds__(256) void rope_split_kernel(const T* qkv, int B, int L, int H, int Hkv,
                                                         int dh, int pos0, const float* cos_t,
                                                         const float* sin_t, T* Q, T* K, T* Vt,
                                                         int kv_cap, int kv_off) {
  __shared__ float tile[64][129];
  const int ntile = (L + 63) / 64;
  const int b = blockIdx.x / ntile, l0 = (blockIdx.x % ntile) * 64;
  const int slot = blockIdx.y;
  const int width = (H + 2 * Hkv) * dh;
  const int half = dh / 2;
  if (slot < H + Hkv) {
    const bool isq = slot < H;
    const int hh = isq ? slot : slot - H;
    for (int idx = threadIdx.x; idx < 64 * half; idx += 256) {
      const int l = l0 + idx / half, j = idx % half;
      if (l >= L) continue;
      const T* src = qkv + ((size_t)b * L + l) * width + slot * dh;
      const float x1 = f32_of(src[j]), x2 = f32_of(src[j + half]);
      const int pos = pos0 + l;
      const float c = cos_t ? cos_t[(size_t)pos * half + j] : 1.f;
      const float s = sin_t ? sin_t[(size_t)pos * half + j] : 0.f;
      T* dst = isq ? Q + (((size_t)b * H + hh) * L + l) * dh
                   : K + (((size_t)b * Hkv + hh) * kv_cap + kv_off + l) * dh;
      dst[j] = from_f32<T>(x1 * c - x2 * s);
      dst[j + half] = from_f32<T>(x2 * c + x1 * s);
    }
  } else {
    const int hh = slot - H - Hkv;
    for (int idx = threadIdx.x; idx < 64 * dh; idx += 256) {
      const int l = idx / dh, d = idx % dh;
      if (l0 + l < L) tile[l][d] = f32_of(qkv[((size_t)b * L + l0 + l) * width + slot * dh + d]);
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 64 * dh; idx += 256) {
      const int d = idx / 64, l = idx % 64;
      if (l0 + l < L)
        Vt[(((size_t)b * Hkv + hh) * dh + d) * kv_cap + kv_off + l0 + l] = from_f32<T>(tile[l][d]);
    }
  }
}

typedef __attribute__((address_space(3))) void* lds_ptr;
typedef const __attribute__((address_space(1))) void* gbl_ptr;
// waitcnt immediate for "at most n vector-memory operations outstanding" (gfx9 encoding)
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// K tile: 64 keys x DH, stored as DH/64 planes of [64 keys][128 B]; V^T tile: DH rows x
// 64 keys of 128 B.  Chunk c (8 bf16) of K row r sits in slot c ^ (r & 7), of V^T row r
// in slot c ^ (r & 7) ^ ((r >> 3) & 1): the V^T fragments are read 8 bytes per lane, 32
// lanes per LDS pass over rows r and r + 8, which the extra bit sends to other banks.
// G = 0: one query head per block for any head ratio (its K/V head floor(h Hkv / H)).
// QS: query strips of 16 per wave; the block's query tile is 64 QS queries (strip s of
// wave w: queries 64 s + 16 w + [0, 16)), and every K and V^T fragment read from LDS
// feeds QS products, so a wave reads the K/V tile once for 16 QS queries.
// KS = 2: the keys of each K/V tile are split between two groups of 4 waves (keys 0-31 and
// 32-63), each with its own running maximum, sum and output, merged in LDS at the end:
// twice the waves per block for the same LDS, when the grid alone leaves the SIMDs short
// of waves.
template <int DH, int NS, int G, int QS, int KS>
__global__ __launch_bounds__(256 * (G > 0 ? G : 1) * KS, G == 4 ? 1 : 2) void attn_bf16_kernel(
    const bf16* Q, const bf16* K, const bf16* Vt, bf16* O, int H, int Hkv, int Lq, int Lk, int kv_cap,
    float scale_log2) {
  static_assert(KS == 1 || (KS == 2 && G <= 1), "key split: one query head per wave");
  constexpr int KT = 64, NW = 4 * (G > 0 ? G : 1) * KS;  // waves per block: 4 query strips x G heads x KS
  constexpr int KB = 4 / KS;                              // 16-key blocks of a tile per wave
  constexpr int KBYTES = KT * DH * 2, VBYTES = DH * KT * 2, STAGE = KBYTES + VBYTES;
  constexpr int LK = KBYTES / 1024 / NW, LV = VBYTES / 1024 / NW;  // load instructions per wave
  static_assert(LK * 1024 * NW == KBYTES && LV * 1024 * NW == VBYTES, "tile rows must split over the waves");
  constexpr int LPT = LK + LV;                                      // per wave per tile
  __shared__ __attribute__((aligned(1024))) char smem[NS * STAGE];

  // wave index as a scalar: the K/V tile destinations in LDS are formed in scalar registers
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), grp = lane >> 4,
            fr = lane & 15;
  const int kh = KS > 1 ? wave / 4 : 0;  // this wave's key group: keys 64 kh / KS + [0, 64 / KS) of a tile
  // one block per (64-query tile, K/V head, batch row), query tiles fastest: the tiles of
  // a K/V head run on one XCD and read K/V from its L2
  const int nqt = (Lq + 64 * QS - 1) / (64 * QS);
  const int id = xcd_contiguous(blockIdx.x, gridDim.x);
  int qt, h, hk, b;
  if constexpr (G > 0) {
    qt = id % nqt;
    hk = (id / nqt) % Hkv;
    b = id / (nqt * Hkv);
    h = hk * G + (KS > 1 ? 0 : wave / 4);  // query heads hk G .. hk G + G - 1 read K/V head hk
  } else {
    qt = id % nqt;
    h = (id / nqt) % H;
    b = id / (nqt * H);
    hk = (h * Hkv) / H;
  }
  const bf16* Kb = K + ((size_t)b * Hkv + hk) * kv_cap * DH;
  const bf16* Vb = Vt + ((size_t)b * Hkv + hk) * DH * kv_cap;
  int q[QS];
  bf16x8 qf[QS][DH / 32];
#pragma unroll
  for (int u = 0; u < QS; ++u) {
    q[u] = qt * 64 * QS + u * 64 + (wave % 4) * 16 + fr;
    const bf16* Qr = Q + (((size_t)b * H + h) * Lq + min(q[u], Lq - 1)) * DH;
#pragma unroll
    for (int kc = 0; kc < DH / 32; ++kc) qf[u][kc] = *reinterpret_cast<const bf16x8*>(Qr + 32 * kc + 8 * grp);
  }

  const int lrow = lane >> 3, lchunk = (lane & 7) ^ (lane >> 3);
  const int lchunk_v = lchunk ^ (wave & 1);  // V^T rows 8 g + lrow with g = wave + NW j (NW even)
  const int nt = (Lk + KT - 1) / KT;
  auto issue = [&](int t, int buf) {
    const int k0 = t * KT;
    char* sb = smem + buf * STAGE;
#pragma unroll
    for (int j = 0; j < LK; ++j) {  // 8-row groups of the K planes
      const int g = wave + NW * j, plane = g / 8, r = (g % 8) * 8 + lrow;
      const bf16* src = Kb + (size_t)min(k0 + r, Lk - 1) * DH + plane * 64 + lchunk * 8;
      __builtin_amdgcn_global_load_lds((gbl_ptr)src, (lds_ptr)(sb + g * 1024), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < LV; ++j) {  // 8-row groups of V^T
      const int g = wave + NW * j, r = g * 8 + lrow;
      const bf16* src = Vb + (size_t)r * kv_cap + k0 + lchunk_v * 8;  // k0 + 64 <= kv_cap
      __builtin_amdgcn_global_load_lds((gbl_ptr)src, (lds_ptr)(sb + KBYTES + g * 1024), 16, 0, 0);
    }
  };

  f32x4 o[QS][DH / 16];
  float m_run[QS], l_run[QS];
#pragma unroll
  for (int u = 0; u < QS; ++u) {
#pragma unroll
    for (int d = 0; d < DH / 16; ++d) o[u][d] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run[u] = -INFINITY;
    l_run[u] = 0.f;
  }

  // this lane's LDS byte offsets inside a stage, the same for every K tile: K row fr of
  // each 16-key block, chunk 4 (kc & 1) + grp; V^T row fr of each 16-row block, the
  // half chunks of keys 32 kc2 + 4 grp + [0, 4) (chunk 4 kc2 + grp / 2) and 16 keys on
  const int vsw = (fr & 7) ^ (fr >> 3);
  int kofs[2], vofs[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    kofs[i] = fr * 128 + (((4 * i + grp) ^ (fr & 7)) * 16);
    const int c0 = 4 * i + (grp >> 1);
    vofs[i][0] = KBYTES + fr * 128 + ((c0 ^ vsw) * 16) + (grp & 1) * 8;
    vofs[i][1] = KBYTES + fr * 128 + (((c0 + 2) ^ vsw) * 16) + (grp & 1) * 8;
  }

#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nt) issue(s, s);
  for (int t = 0; t < nt; ++t) {
    const int buf = t % NS;
    if (t + NS - 2 < nt)  // tile t is in once at most NS - 2 younger tiles are in flight
      __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 2) * LPT));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    const char* sk = smem + buf * STAGE;
    if ((t + 1) * KT > Lk) {
      // last, partial tile: keys past the end get V = 0 so that p = 0 meets finite values
      char* svw = const_cast<char*>(sk + KBYTES);
      for (int idx = tid; idx < DH * KT; idx += 64 * NW) {
        const int r = idx / KT, key = idx % KT;
        if (t * KT + key >= Lk) {
          const int slot = (key >> 3) ^ (r & 7) ^ ((r >> 3) & 1);
          *reinterpret_cast<bf16*>(svw + r * 128 + slot * 16 + (key & 7) * 2) = (bf16)0.f;
        }
      }
      __syncthreads();
    }
    // the buffer of tile t - 1, which every wave finished before the barrier above
    if (t + NS - 1 < nt) issue(t + NS - 1, (t + NS - 1) % NS);
    // a key group whose keys of this tile all lie past the end skips it (its scores
    // would all be -inf)
    if (KS > 1 && t * KT + kh * (KT / KS) >= Lk) continue;
    f32x4 s[QS][KB];
#pragma unroll
    for (int ks = 0; ks < KB; ++ks) {
#pragma unroll
      for (int u = 0; u < QS; ++u) s[u][ks] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < DH / 32; ++kc) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(sk + (kc >> 1) * 8192 + (kh * KB + ks) * 2048 + kofs[kc & 1]);
#pragma unroll
        for (int u = 0; u < QS; ++u) s[u][ks] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[u][kc], s[u][ks], 0, 0, 0);
      }
    }
    bf16x8 pf[QS][KB / 2];
#pragma unroll
    for (int u = 0; u < QS; ++u) {
      // s[u][ks][j] = score(query q[u], key t*64 + (kh*KB + ks)*16 + 4*grp + j), unscaled: the
      // softmax runs in base 2 on s * scale_log2, the scale folded into one FMA per score
      float mt = -INFINITY;
      if ((t + 1) * KT <= Lk) {  // a whole tile: no key is masked
#pragma unroll
        for (int ks = 0; ks < KB; ++ks)
#pragma unroll
          for (int j = 0; j < 4; ++j) mt = fmaxf(mt, s[u][ks][j]);
      } else {
#pragma unroll
        for (int ks = 0; ks < KB; ++ks)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int key = t * KT + (kh * KB + ks) * 16 + 4 * grp + j;
            if (key >= Lk) s[u][ks][j] = -INFINITY;
            mt = fmaxf(mt, s[u][ks][j]);
          }
      }
      mt = fmaxf(mt, xor16(mt));
      mt = fmaxf(mt, xor32(mt));
      // The probabilities are taken relative to a reference m_run that only moves when the
      // tile's maximum exceeds it by more than 2^8 (in base 2): until then they stay below
      // 256 (exact in bf16's exponent range) and the accumulators need no rescaling; the
      // row sum l_run uses the same reference, so o / l is unchanged.
      const float mt2 = mt * scale_log2;  // scale_log2 > 0: the max commutes
      const bool move = mt2 > m_run[u] + 8.f;  // also true on the first tile (m_run = -inf)
      const float m_new = move ? mt2 : m_run[u];
      // raw v_exp_f32: results below 2^-126 flush to 0 (a probability that small adds nothing)
      const float alpha = m_run[u] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[u] - m_new);
      float ps = 0.f;
#pragma unroll
      for (int ks = 0; ks < KB; ++ks)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[u][ks][j], scale_log2, -m_new));
          s[u][ks][j] = p;
          ps += p;
        }
      l_run[u] = l_run[u] * alpha + ps;
      m_run[u] = m_new;
      if (__builtin_amdgcn_ballot_w64(move))  // some lane of the wave moved its reference
#pragma unroll
        for (int d = 0; d < DH / 16; ++d) o[u][d] *= alpha;
#pragma unroll
      for (int c = 0; c < KB / 2; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          pf[u][c][j] = (bf16)s[u][2 * c][j];
          pf[u][c][4 + j] = (bf16)s[u][2 * c + 1][j];
        }
    }
#pragma unroll
    for (int c = 0; c < KB / 2; ++c) {
      const int kc2 = kh * (KB / 2) + c;  // 32-key half of the tile
#pragma unroll
      for (int d = 0; d < DH / 16; ++d) {
        const bf16x4 v0 = *reinterpret_cast<const bf16x4*>(sk + d * 2048 + vofs[kc2][0]);
        const bf16x4 v1 = *reinterpret_cast<const bf16x4*>(sk + d * 2048 + vofs[kc2][1]);
        const bf16x8 vf = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
        for (int u = 0; u < QS; ++u) o[u][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[u][c], o[u][d], 0, 0, 0);
      }
    }
  }
  if constexpr (KS > 1) {
    // merge the second key group into the first, one query strip at a time: each group's
    // output and sum are relative to its own reference m; both are rescaled to the larger
    // one.  Per lane: m, l and the DH / 4 output values, in [wave - 4][value][lane] floats.
    constexpr int NV = 2 + DH / 4;
    static_assert(4 * NV * 64 * 4 <= NS * STAGE, "merge area larger than the K/V ring");
    float* xs = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int u = 0; u < QS; ++u) {
      __syncthreads();  // every wave is done with the K/V ring (or the previous strip's merge)
      if (kh == 1) {
        float* w = xs + (size_t)(wave - 4) * NV * 64 + lane;
        w[0] = m_run[u];
        w[64] = l_run[u];
#pragma unroll
        for (int d = 0; d < DH / 16; ++d)
#pragma unroll
          for (int j = 0; j < 4; ++j) w[(2 + 4 * d + j) * 64] = o[u][d][j];
      }
      __syncthreads();
      if (kh == 0) {
        const float* r = xs + (size_t)wave * NV * 64 + lane;
        const float m1 = r[0], m0 = m_run[u], mm = fmaxf(m0, m1);
        const float a0 = m0 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m0 - mm);
        const float a1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - mm);
        l_run[u] = l_run[u] * a0 + r[64] * a1;
#pragma unroll
        for (int d = 0; d < DH / 16; ++d)
#pragma unroll
          for (int j = 0; j < 4; ++j) o[u][d][j] = o[u][d][j] * a0 + r[(2 + 4 * d + j) * 64] * a1;
      }
    }
    if (kh == 1) return;
  }
#pragma unroll
  for (int u = 0; u < QS; ++u) {
    float l_tot = l_run[u] + xor16(l_run[u]);
    l_tot += xor32(l_tot);
    const float inv = 1.f / l_tot;
    if (q[u] < Lq) {
      bf16* orow = O + ((size_t)b * Lq + q[u]) * H * DH + h * DH;
#pragma unroll
      for (int d = 0; d < DH / 16; ++d)
        store4(orow + d * 16 + 4 * grp, o[u][d][0] * inv, o[u][d][1] * inv, o[u][d][2] * inv, o[u][d][3] * inv);
    }
  }
}

// float32 attention for small fp32 models: one wave per query, scores in LDS.
__global__ __launch_bounds__(256) void attn_f32_kernel(const float* Q, const float* K, const float* Vt,
                                                       float* O, int H, int Hkv, int Lq, int Lk,
                                                       int kv_cap, int dh, float scale) {
  extern __shared__ float sp[];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q = blockIdx.x * 4 + wave, h = blockIdx.y, b = blockIdx.z;
  const int hk = (h * Hkv) / H;
  const int qc = min(q, Lq - 1);
  float* p = sp + wave * Lk;
  const float* qr = Q + (((size_t)b * H + h) * Lq + qc) * dh;
  const float* Kb = K + ((size_t)b * Hkv + hk) * kv_cap * dh;
  const float* Vb = Vt + ((size_t)b * Hkv + hk) * dh * kv_cap;
  float mx = -INFINITY;
  for (int k = lane; k < Lk; k += 64) {
    float acc = 0.f;
    for (int d = 0; d < dh; ++d) acc += qr[d] * Kb[(size_t)k * dh + d];
    p[k] = acc * scale;
    mx = fmaxf(mx, acc * scale);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int k = lane; k < Lk; k += 64) {
    const float e = __expf(p[k] - mx);
    p[k] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  __syncthreads();
  if (q < Lq)
    for (int d = lane; d < dh; d += 64) {
      float acc = 0.f;
      for (int k = 0; k < Lk; ++k) acc += p[k] * Vb[(size_t)d * kv_cap + k];
      O[((size_t)b * Lq + q) * H * dh + h * dh + d] = acc / sum;
    }
}

}  // namespace

hipError_t rope_split(DType dt, const void* qkv, int B, int L, int H, int Hkv, int dh, int pos0,
                      const float* cos_t, const float* sin_t, void* Q, void* K, void* Vt, int kv_cap,
                      int kv_off, hipStream_t s) {
  if (B * L == 0) return hipSuccess;
  const dim3 grid(B * ((L + 63) / 64), H + 2 * Hkv);
  if (dt == BF16)
    hipLaunchKernelGGL(rope_split_kernel<bf16>, grid, dim3(256), 0, s, static_cast<const bf16*>(qkv), B,
                       L, H, Hkv, dh, pos0, cos_t, sin_t, static_cast<bf16*>(Q), static_cast<bf16*>(K),
                       static_cast<bf16*>(Vt), kv_cap, kv_off);
  else
    hipLaunchKernelGGL(rope_split_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(qkv),
                       B, L, H, Hkv, dh, pos0, cos_t, sin_t, static_cast<float*>(Q),
                       static_cast<float*>(K), static_cast<float*>(Vt), kv_cap, kv_off);
  return hipGetLastError();
}

hipError_t attention(DType dt, const void* Q, const void* K, const void* Vt, void* O, int B, int H,
                     int Hkv, int Lq, int Lk, int kv_cap, int dh, hipStream_t s) {
  if (B * Lq == 0) return hipSuccess;
  if (dt == BF16) {
    const float sl2 = 1.4426950408889634f / sqrtf((float)dh);
    const int nqt = (Lq + 63) / 64, G = H % Hkv == 0 ? H / Hkv : 0;
    auto go = [&](auto kernel, int g, int qs, int ks) {
      const int tiles = (Lq + 64 * qs - 1) / (64 * qs);
      const dim3 grid(tiles * (g > 0 ? Hkv : H) * B), block(256 * (g > 0 ? g : 1) * ks);
      launch_timed(kernel, grid, block, 0, s, static_cast<const bf16*>(Q), static_cast<const bf16*>(K),
                   static_cast<const bf16*>(Vt), static_cast<bf16*>(O), H, Hkv, Lq, Lk, kv_cap, sl2);
      return hipGetLastError();
    };
    // The query heads sharing a K/V head go to one block (G = 2 or 4 of them, the K/V
    // tile split over the 4 G waves) only when the packed grid still gives every CU two
    // blocks: packing divides the block count by G, and at the benchmark's shapes that
    // leaves CUs idle (block workload, G = 4: 64 blocks of 16 waves, attention 47.8 ->
    // 94.7 ms per generation; 26B-class, G = 2: 256 blocks of 8 waves, no faster).
    const bool pack = (long)nqt * Hkv * B >= 512;
    // Two query strips per wave (128 queries per block) halve the LDS reads per product
    // (each K / V^T fragment feeds two MFMAs), when the grid keeps two blocks per CU.
    const long n128 = (long)((Lq + 127) / 128) * H * B;
    const bool two = n128 >= 512;
    // Otherwise the keys of each tile are split between two wave groups (KS = 2), which
    // doubles the waves per block: with two strips per wave when the query tiles of 128
    // still give every CU a block, else with one.
    const bool two_split = !two && Lq >= 128 && n128 >= 256;
    if (dh == 64) {  // the key split measured slower at this width (small workload 3.66 -> 4.01 ms)
      if (G == 1) return two ? go(attn_bf16_kernel<64, 2, 1, 2, 1>, 1, 2, 1) : go(attn_bf16_kernel<64, 2, 1, 1, 1>, 1, 1, 1);
      return two ? go(attn_bf16_kernel<64, 2, 0, 2, 1>, 0, 2, 1) : go(attn_bf16_kernel<64, 2, 0, 1, 1>, 0, 1, 1);
    }
    if (dh == 128) {
      if (G == 1) {
        if (two) return go(attn_bf16_kernel<128, 2, 1, 2, 1>, 1, 2, 1);
        return two_split ? go(attn_bf16_kernel<128, 2, 1, 2, 2>, 1, 2, 2) : go(attn_bf16_kernel<128, 2, 1, 1, 2>, 1, 1, 2);
      }
      if (pack && G == 2) return go(attn_bf16_kernel<128, 2, 2, 1, 1>, 2, 1, 1);
      if (pack && G == 4) return go(attn_bf16_kernel<128, 2, 4, 1, 1>, 4, 1, 1);
      if (two) return go(attn_bf16_kernel<128, 2, 0, 2, 1>, 0, 2, 1);
      return two_split ? go(attn_bf16_kernel<128, 2, 0, 2, 2>, 0, 2, 2) : go(attn_bf16_kernel<128, 2, 0, 1, 2>, 0, 1, 2);
    }
    return hipErrorInvalidValue;
  }
  const dim3 grid((Lq + 3) / 4, H, B);
  launch_timed(attn_f32_kernel, grid, dim3(256), (uint32_t)(4 * Lk * sizeof(float)), s,
               static_cast<const float*>(Q), static_cast<const float*>(K), static_cast<const float*>(Vt),
               static_cast<float*>(O), H, Hkv, Lq, Lk, kv_cap, dh, 1.f / sqrtf((float)dh));
  return hipGetLastError();
}

}  // namespace tadm
