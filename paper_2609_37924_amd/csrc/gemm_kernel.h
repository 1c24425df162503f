// bf16 GEMM kernel template C = A W^T for gfx950, shared by the translation units
// that instantiate it with their own epilogues.
//
// WGM x WGN wave64s per block, block tile BM x BN, K tiles of 64.  Tiles move
// global -> LDS with global_load_lds_dwordx4 (no register staging) through a
// two-stage ring of LDS buffers: the next K tile lands while one is multiplied.  Each
// wave holds one set of MFMA fragments and reads the next 32-deep half's fragments in
// their place as the products that use them issue (a rolling prefetch), so that its
// LDS reads overlap its own MFMAs instead of all waves reading at once after each
// barrier.  LDS rows are 128 B (64 bf16); the 16-byte chunk c of row r is stored
// in slot c ^ (r & 7), which makes the MFMA fragment reads (16 rows x one chunk) hit
// distinct banks; the permutation is applied through the global addresses because
// each lane's 16 bytes land at a fixed LDS slot.  Products use
// v_mfma_f32_16x16x32_bf16 with the weight tile as the "A" operand and the activation
// tile as "B", so every lane ends with 4 consecutive output features of one row.
// Blocks are renumbered so that the tiles sharing a weight panel run on the same XCD
// (each XCD has its own L2).
#pragma once
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace tadm {
namespace {

// Epi<K, T> supplies the epilogue of kind K for operand type T: either apply() per
// 4-feature fragment (with kGlu for gate/up pairs), or, when it defines kTile, a
// tile<TN, TM>() that receives the wave's whole accumulator tile, or, when it defines
// kTileLds, a tile_lds<TN, TM>() that also receives WTM x WTN x 2 bytes of LDS of its
// own (the K tiles' ring, free once every wave has left the main loop).
template <EpiKind K, class T>
struct Epi;

template <class E, class = void>
struct TileEpi : std::false_type {};
template <class E>
struct TileEpi<E, std::void_t<decltype(E::kTile)>> : std::true_type {};
template <class E, class = void>
struct TileLdsEpi : std::false_type {};
template <class E>
struct TileLdsEpi<E, std::void_t<decltype(E::kTileLds)>> : std::true_type {};

// An epilogue that reads other tensors may define kPre (float4 loads per fragment),
// pre() and apply_pre(): the kernel then issues those loads before the main loop,
// where their latency hides behind the K tiles, when the tile keeps them in at most
// 16 float4 registers per lane.
template <class E, class = void>
struct PreCount { static constexpr int value = 0; };
template <class E>
struct PreCount<E, std::void_t<decltype(E::kPre)>> { static constexpr int value = E::kPre; };

// waitcnt immediate for "at most n vector-memory operations outstanding" (gfx9 encoding)
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

typedef __attribute__((address_space(3))) void* lds_ptr;
typedef const __attribute__((address_space(1))) void* gbl_ptr;

// Block index -> (m tile, n tile).  Workgroups are dealt to the 8 XCDs round-robin,
// so block b runs on XCD b % 8 as its (b / 8)-th block.  When the tile grid splits
// into 8 regions of rm x rn tiles, XCD x works through region x, so the A rows and W
// rows it reads (rm*BM + rn*BN rows) stay in its own L2.  Inside the region the blocks
// an XCD holds at once (gm * gn of them) cover a gm x gn patch of tiles, which keeps the
// A and W rows that the XCD streams in at each K step (gm*BM + gn*BN) low; without a
// patch (gm = 0) the region is walked m first.
// A grid with no even split into 8 regions is walked in bands of `band` tile rows, each
// band column by column, and XCD x takes the x-th eighth of that walk: the blocks it
// holds at once cover about band x (R / band) tiles.  The grid is then padded to a
// multiple of 8 blocks; a padded block gets tm = tiles_m and does nothing.
__device__ __forceinline__ void tile_of(const GemmProblem& p, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int b = blockIdx.x;
  if (p.band > 0) {
    const int tiles = tiles_m * tiles_n, chunk = (tiles + 7) / 8, o = (b % 8) * chunk + b / 8;
    if (o >= tiles) {
      tm = tiles_m;
      tn = 0;
      return;
    }
    const int per = p.band * tiles_n, g = o / per, first = g * p.band, j = o - g * per;
    const int h = min(p.band, tiles_m - first);
    tm = first + j % h;
    tn = j / h;
    return;
  }
  if (p.rm > 0) {
    const int x = b % 8, i = b / 8, regions_m = tiles_m / p.rm;
    int lm, ln;
    if (p.gm > 0) {
      const int R = p.gm * p.gn, g = i / R, j = i % R, per_m = p.rm / p.gm;
      lm = (g % per_m) * p.gm + j % p.gm;
      ln = (g / per_m) * p.gn + j / p.gm;
    } else {
      lm = i % p.rm;
      ln = i / p.rm;
    }
    tm = (x % regions_m) * p.rm + lm;
    tn = (x / regions_m) * p.rn + ln;
    return;
  }
  tm = b % tiles_m;
  tn = b / tiles_m;
}

// MFMA on an accumulator held in four AGPRs, written in place (dst == srcC).  Keeping
// the accumulator tied to one register quadruple over the whole K loop stops the
// register allocator from rotating accumulators through VGPRs between iterations.
// The chain of products on one accumulator needs no wait states (full-register srcC
// overlap); the operands come from LDS reads, whose waits the compiler inserts.
__device__ __forceinline__ void mfma_acc(f32x4& acc, const bf16x8& w, const bf16x8& a) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(w), "v"(a));
}
// The first product of an accumulator: srcC is the constant 0, so no VALU write
// initialises the accumulator (a VALU write read by an MFMA would need wait states).
__device__ __forceinline__ void mfma_first(f32x4& acc, const bf16x8& w, const bf16x8& a) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(acc) : "v"(w), "v"(a));
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
  static_assert(STAGES == 2, "the K loop is written for a two-stage ring");
  constexpr int WTM = BM / WGM, WTN = BN / WGN; // wave tile
  constexpr int TM = WTM / 16, TN = WTN / 16;   // 16x16 subtiles per wave
  static_assert(WTN % 32 == 0, "GLU pairs need 32-row weight blocks per wave");
  __shared__ __attribute__((aligned(1024))) char smem[STAGES * STAGE_BYTES];

  // the wave index as a wave-uniform (scalar) value: LDS destinations of the tile loads are
  // then formed in scalar registers
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WGM, wn = wave / WGM;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  int tmi, tni;
  tile_of(p, tiles_m, tiles_n, tmi, tni);
  if (tmi >= tiles_m) return;  // padding of a banded grid
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

  // this block's K slice: K tiles [kt_base, kt_base + nk), slices as even as the tile
  // count allows (they differ by at most one tile)
  const int NKT = p.K / 64, kt_base = (int)((long)blockIdx.y * NKT / p.ksplit);
  const int nk = (int)((long)(blockIdx.y + 1) * NKT / p.ksplit) - kt_base;
  // this lane's source rows, fixed over the K loop: a K tile only adds its offset.  A
  // second operand A2 (K columns from K1 on) gets its own row pointers, shifted by -K1.
  const bf16* arow1[LA];
  const bf16* arow2[LA];
  const bf16* wrow[LW];
#pragma unroll
  for (int j = 0; j < LA; ++j) {
    const int r = min(m0 + (wave + NW * j) * 8 + lrow, p.M - 1);
    arow1[j] = A1 + (size_t)r * p.lda1 + lchunk * 8;
    arow2[j] = A2 ? A2 + (size_t)r * p.lda2 + lchunk * 8 - p.K1 : arow1[j];
  }
#pragma unroll
  for (int j = 0; j < LW; ++j) {
    const int r = min(n0 + (wave + NW * j) * 8 + lrow, p.N - 1);
    wrow[j] = W + (size_t)r * p.ldw + lchunk * 8;
  }
  // the activation rows (issue_a) and the weight rows (issue_w) of K tile kt into buffer buf
  auto issue_a = [&](int kt, int buf) {
    const int k0 = (kt_base + kt) * 64;
    const bool second = k0 >= p.K1;
    char* sb = smem + buf * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < LA; ++j) {
      const int g = wave + NW * j;  // 8-row group
      const bf16* src = (second ? arow2[j] : arow1[j]) + k0;
      __builtin_amdgcn_global_load_lds((gbl_ptr)src, (lds_ptr)(sb + g * 1024), 16, 0, 0);
    }
  };
  auto issue_w = [&](int kt, int buf) {
    const int k0 = (kt_base + kt) * 64;
    char* sb = smem + buf * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < LW; ++j) {
      const int g = wave + NW * j;
      __builtin_amdgcn_global_load_lds((gbl_ptr)(wrow[j] + k0), (lds_ptr)(sb + BM * ROW + g * 1024), 16, 0, 0);
    }
  };
  auto issue = [&](int kt, int buf) {
    issue_a(kt, buf);
    issue_w(kt, buf);
  };

  f32x4 acc[TN][TM];

  // epilogue operands, loaded before the K tiles so that they are the oldest
  // vector-memory operations (the vmcnt waits below only ever wait for older ones)
  constexpr int NPRE = PreCount<E>::value;
  constexpr bool PRE = NPRE > 0 && TN * TM * NPRE <= 16;
  float4 pre[PRE ? TN : 1][PRE ? TM : 1][PRE ? NPRE : 1];
  if constexpr (PRE) {
    const int mw0 = m0 + wm * WTM + (lane & 15), nw0 = n0 + wn * WTN + 4 * (lane >> 4);
#pragma unroll
    for (int a = 0; a < TN; ++a)
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        const int m = mw0 + b * 16, n = nw0 + a * 16;
        if (m < p.M && n < p.N) E::pre(ep, m, n, pre[a][b]);
      }
  }

  const int fr = lane & 15, fq = lane >> 4, sw = lane & 7;
  const int aoff = (wm * WTM + fr) * ROW, woff = BM * ROW + (wn * WTN + fr) * ROW;
  // fragment t of the 32-deep half kk of the K tile in LDS buffer buf
  auto fa_at = [&](int buf, int kk, int t) {
    return *reinterpret_cast<const bf16x8*>(smem + buf * STAGE_BYTES + aoff + t * 16 * ROW + ((kk * 4 + fq) ^ sw) * 16);
  };
  auto fw_at = [&](int buf, int kk, int t) {
    return *reinterpret_cast<const bf16x8*>(smem + buf * STAGE_BYTES + woff + t * 16 * ROW + ((kk * 4 + fq) ^ sw) * 16);
  };
  bf16x8 fa[TM], fw[TN];
  // the products of one 32-deep half; each fragment is replaced by the same fragment of
  // the half (nbuf, nkk) as soon as its last product has issued
  auto half = [&](auto first, auto prefetch, int nbuf, int nkk) {
#pragma unroll
    for (int a = 0; a < TN; ++a) {
#pragma unroll
      for (int b = 0; b < TM; ++b) {
        if constexpr (decltype(first)::value)
          mfma_first(acc[a][b], fw[a], fa[b]);
        else
          mfma_acc(acc[a][b], fw[a], fa[b]);
        if constexpr (decltype(prefetch)::value)
          if (a == TN - 1) fa[b] = fa_at(nbuf, nkk, b);
      }
      if constexpr (decltype(prefetch)::value) fw[a] = fw_at(nbuf, nkk, a);
    }
  };
  using Yes = std::true_type;
  using No = std::false_type;
  // Up projections (GLU / GELU epilogues) with more weight rows than activation rows
  // issue each K tile's loads in two parts (26B-class gate/up, 1 024 x 73 728 x 4 608:
  // 2 634 -> 2 542 ms per generation); the other products, and up projections with more
  // activation rows, measured faster issuing the whole tile at once.
  constexpr bool kSplitIssue = KIND == EPI_GLU_SILU || KIND == EPI_GLU_GELU || KIND == EPI_GELU;

  // K tile 0 landed and published, K tile 1 in flight, the first half's fragments read
  issue(0, 0);
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  __syncthreads();
  if (nk > 1) issue(1, 1);
#pragma unroll
  for (int t = 0; t < TM; ++t) fa[t] = fa_at(0, 0, t);
#pragma unroll
  for (int t = 0; t < TN; ++t) fw[t] = fw_at(0, 0, t);
  half(Yes{}, Yes{}, 0, 1);
  // iteration kt: the second half of K tile kt, then the first half of K tile kt + 1
  for (int kt = 0; kt + 1 < nk; ++kt) {
    const int buf = kt & 1;
    // every wave has read K tile kt's buffer (its last fragments are the ones in
    // registers) and K tile kt + 1 has landed: the buffer can take K tile kt + 2
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    __syncthreads();
    // K tile kt + 2 into the buffer just freed: all of it at once, or, for the up
    // projections whose weight is the larger operand, its weight rows now and its
    // activation rows after the first half of the products
    const bool more = kt + 2 < nk, split = kSplitIssue && p.w_first;
    if (more) {
      if (split) issue_w(kt + 2, buf);
      else issue(kt + 2, buf);
    }
    half(No{}, Yes{}, buf ^ 1, 0);
    if (more && split) issue_a(kt + 2, buf);
    half(No{}, Yes{}, buf ^ 1, 1);
  }
  half(No{}, No{}, 0, 0);
  // the last products must be written before any accumulator is read back: wait
  // states after the final MFMA, then every accumulator passes through an empty asm
  // that is ordered after the wait, so no read can be scheduled before it
  asm volatile("s_nop 15\n s_nop 15\n s_nop 15" ::: "memory");
#pragma unroll
  for (int a = 0; a < TN; ++a)
#pragma unroll
    for (int b = 0; b < TM; ++b) asm volatile("" : "+a"(acc[a][b]));

  // lane holds C[n = nb + 4*(lane>>4) + j][m = mb + (lane & 15)]
  const int mw = m0 + wm * WTM + fr;
  if constexpr (KIND == EPI_STORE_F32)
    if (p.ksplit > 1) ep.out = static_cast<float*>(ep.out) + (size_t)blockIdx.y * ep.split_stride;
  if constexpr (TileLdsEpi<E>::value) {  // the wave's whole tile, staged through LDS
    static_assert(BM * BN * 2 <= STAGES * STAGE_BYTES, "staging area larger than the ring");
    __syncthreads();  // every wave has finished reading the K tiles
    E::template tile_lds<TN, TM>(ep, p, acc, m0 + wm * WTM, n0 + wn * WTN, lane, smem + wave * (WTM * WTN * 2));
  } else if constexpr (TileEpi<E>::value) {  // the epilogue takes the wave's whole tile
    E::template tile<TN, TM>(ep, p, acc, m0 + wm * WTM, n0 + wn * WTN, lane);
  } else if constexpr (E::kGlu) {
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
        if (m < p.M && n < p.N) {
          if constexpr (PRE)
            E::apply_pre(ep, m, n, acc[a][b], pre[a][b]);
          else
            E::apply(ep, m, n, acc[a][b]);
        }
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

// Patch gm x gn (gm * gn = R, the blocks an XCD holds at once: 32 CUs x resident blocks
// per CU) that tiles the rm x rn region and streams the fewest rows per K step
// (gm * BM + gn * BN), when that is fewer than the m-first walk's; else gm = gn = 0.
// 1B-class FFN up, 32 768 x 8 192 x 2 048 on 256 x 256 tiles: region 32 x 16, the m-first
// walk holds 32 x 1 tiles (33 panels of rows), a 8 x 4 patch 12: 1 364 -> 1 101 us.
inline void xcd_patch(int rm, int rn, int BM, int BN, int R, int& gm, int& gn) {
  gm = gn = 0;
  if (rm <= 0 || rn <= 0 || rm * rn < R) return;
  const int wm = rm < R ? rm : R, wn = (R + wm - 1) / wm;  // the m-first walk's extent
  long best = (long)wm * BM + (long)(wn < rn ? wn : rn) * BN;
  for (int m = R; m >= 1; m /= 2) {
    const int n = R / m;
    if (rm % m || rn % n) continue;
    const long cost = (long)m * BM + (long)n * BN;
    // on a tie, a patch as wide as the region: each A panel is then streamed once per
    // region (the 1B-class FFN down, 32 768 x 2 048 x 8 192, region 16 x 8: 4 x 8 rather
    // than 8 x 4, whose two patches per row band read each 4 MB A panel twice)
    if (cost < best || (cost == best && gm > 0 && n == rn)) {
      best = cost;
      gm = m;
      gn = n;
    }
  }
}

// Band height h <= tiles_m of the banded walk that streams the fewest rows per K step
// for R blocks held at once (h * BM + ceil(R / h) * BN).  1B-class head, 16 512 x 50 304 x
// 2 048 on 128 x 128 tiles (129 x 393, no even split): h = 8.
inline int xcd_band(int tiles_m, int BM, int BN, int R) {
  int best_h = 1;
  long best = -1;
  for (int h = 1; h <= tiles_m && h <= R; ++h) {
    const long cost = (long)h * BM + (long)((R + h - 1) / h) * BN;
    if (best < 0 || cost < best) {
      best = cost;
      best_h = h;
    }
  }
  return best_h;
}

template <int BM, int BN, int ST, int WGM, int WGN, int MINB, EpiKind K>
hipError_t launch_bf16(const GemmProblem& p0, const EpiParams& e, hipStream_t s) {
  GemmProblem p = p0;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = (p.N + BN - 1) / BN;
  xcd_regions(tiles_m, tiles_n, BM, BN, p.rm, p.rn);
  // one block per CU for the 8-wave tiles, MINB per CU otherwise (LDS bounds both)
  if (MINB <= 2) xcd_patch(p.rm, p.rn, BM, BN, 32 * MINB, p.gm, p.gn);
  p.band = p.rm > 0 ? 0 : xcd_band(tiles_m, BM, BN, 32 * MINB);
  const int blocks = p.band > 0 ? (tiles_m * tiles_n + 7) / 8 * 8 : tiles_m * tiles_n;
  p.w_first = p.N > p.M;
  launch_timed(gemm_bf16_kernel<BM, BN, ST, WGM, WGN, MINB, K>, dim3(blocks, p.ksplit), dim3(64 * WGM * WGN), 0, s, p,
               e);
  return hipGetLastError();
}

}  // namespace
}  // namespace tadm
