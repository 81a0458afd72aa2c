// Decoder GEMMs on gfx950: Y = X W^T, X [R, K] (row-major), W [N, K].
//
// bf16 weights are stored in the tiled layout (pack_weight below): in every
// complete group of 16 rows and block of 128 columns the 16 x 16 matrix of
// 16-byte chunks is transposed, so chunk j (columns 8j..8j+7) of row r of the
// group sits in row j of the group at chunk position r.  A trailing group of
// fewer than 16 rows stays row-major.  With this layout every load the
// kernels issue for a 16-feature tile covers whole 256-byte runs of memory
// rows; row-major MFMA operand loads only give 64-byte runs of 16 rows.
//
// bf16 paths use v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  Operand
// fragments: lane l supplies A[l % 16][kgroup(l / 16)] and B[kgroup(l / 16)][l % 16],
// and receives D[4 (l / 16) + r][l % 16], r = 0..3.  The reduction only needs
// A and B to agree on which k each (lane group, element) carries: lane group
// g of step s carries k = 32 s + 8 g .. +7 of a 128-wide block, which in the
// tiled layout is row 4 s + g of the tile.
//
//  * gemv (R <= 2): vector-FMA weight streaming, one tile per workgroup.
//  * skinny (R <= 64, except where use_mfma picks the MFMA kernel): weight
//    streaming, HBM-bound.  A workgroup owns one 16-feature tile (for SwiGLU
//    the gate tile and its up tile); its waves split K and reduce through LDS
//    in a fixed order (deterministic, no atomics).  M is padded to 16 per
//    tile; MFMA throughput is ~10x what the weight stream needs.
//  * mfma2 (R > 64, and the LM head / large projections above 8 / 40 rows):
//    (32 MTW) x 256 workgroup tiles, one workgroup per CU, accumulators in
//    AGPRs, X and W brought into LDS by direct-to-LDS loads four k-steps
//    ahead, XCD-aware tile order, split-K with a fixed-order reduction when
//    the grid is small.
//  * fp32 (the fp32 configuration): a plain LDS-tiled FMA kernel on row-major
//    weights; no reduced-precision arithmetic.

#include <algorithm>
#include <cstdio>
#include <mutex>

#include "common.h"
#include "gemm.h"
#include "kv_layout.h"

namespace spec {
namespace {

// x * sigmoid(x) with a hardware reciprocal (1 ulp) instead of an IEEE
// division, which costs ten instructions per element in the epilogues.
__device__ __forceinline__ float silu(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

// ---------------------------------------------------------------------------
// tiled weight layout

// Element offset of 16-byte chunk `ch` (columns 8 ch .. 8 ch + 7) of row n of
// a tiled [N, K] weight, as base + (ch % 16) * s1 + (ch / 16) * 128.
struct ChunkAddr {
  size_t base;
  int s1;
};
__device__ __forceinline__ ChunkAddr chunk_addr(int n, int N, int K) {
  if (n < (N & ~15)) return {static_cast<size_t>(n & ~15) * K + (n & 15) * 8, K};
  return {static_cast<size_t>(n) * K, 8};
}

// Position, inside its head, of rotary row `dim` in the QKV weight's tiled
// row order: the q and k heads are laid out as hd / 16 tiles of 8 rotary
// pairs (i, i + hd / 2), rows 8t..8t+7 then hd/2+8t..hd/2+8t+7 in tile t, so
// that the two halves of a pair meet in one 16-feature tile (lanes l and
// l ^ 8 of a 16-lane group).
__host__ __device__ __forceinline__ int rot_tile_pos(int dim, int hd) {
  const int half = hd / 2, i = dim % half;
  return 16 * (i / 8) + (dim >= half ? 8 : 0) + (i % 8);
}
__host__ __device__ __forceinline__ int rot_tile_dim(int p, int hd) {
  const int t = p / 16, i = p % 16;
  return (i < 8 ? 0 : hd / 2) + 8 * t + (i & 7);
}

// In place: row-major [rows, K] -> tiled.  Rows [0, rot_rows) form rotary
// heads of hd rows, first reordered by rot_tile_dim.  One workgroup per (row
// group, 128-column block) reads the block (hd or 16 rows x 256 bytes) into
// LDS and writes it back transformed; blocks are disjoint, so in place is safe.
__global__ __launch_bounds__(256) void pack_weight_kernel(bf16_t* __restrict__ W, int rows, int K,
                                                          int rot_rows, int hd) {
  extern __shared__ u32x4 blk[];  // [G rows][16 chunks]
  const int nb = K / 128;
  const int kb = blockIdx.x % nb, grp = blockIdx.x / nb;
  const int n_rot = rot_rows > 0 ? rot_rows / hd : 0;
  const bool rot = grp < n_rot;
  const int G = rot ? hd : 16;
  const int r0 = rot ? grp * hd : rot_rows + (grp - n_rot) * 16;
  if (r0 + G > rows) return;  // a trailing partial group stays row-major
  bf16_t* base = W + static_cast<size_t>(r0) * K + kb * 128;
  for (int e = threadIdx.x; e < G * 16; e += blockDim.x)
    blk[e] = *reinterpret_cast<const u32x4*>(base + static_cast<size_t>(e / 16) * K + (e % 16) * 8);
  __syncthreads();
  for (int e = threadIdx.x; e < G * 16; e += blockDim.x) {
    const int p = e / 16, c = e % 16;  // destination row of the group, chunk position
    const int pos = (p & ~15) + c;     // feature (in tile order) whose chunk p % 16 lands here
    const int src = rot ? rot_tile_dim(pos, G) : pos;
    *reinterpret_cast<u32x4*>(base + static_cast<size_t>(p) * K + c * 8) = blk[src * 16 + (p & 15)];
  }
}

// ---------------------------------------------------------------------------
// skinny bf16

constexpr int kSkinnyMaxWaves = 8;

// Output (head, dim) of column l16 of tile `tile` of the QKV projection,
// whose q and k heads are in rotary tile order; the v heads follow in plain
// order.  Returns the natural row head * hd + dim.
__device__ __forceinline__ int qkv_tile_row(const GemmFuse& f, int tile, int l16, int* head, int* dim) {
  const int per_head = f.hd / 16;
  *head = tile / per_head;
  *dim = rot_tile_dim(16 * (tile % per_head) + l16, f.hd);
  return *head * f.hd + *dim;
}

// 1 / rms of each X row (R <= 16) from the producer's sums of squares per 8
// columns, into s_rs.  Wave w takes rows w, w + waves, ...; lane l sums
// entries l, l + 64, ... of the row, eight loads issued together per round,
// then a fixed-order shuffle tree.  Run by the whole workgroup.
__device__ __forceinline__ void row_rscale(const GemmFuse& fu, int R, int K, float* s_rs) {
  const int np = K / 8;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave, nw = blockDim.x / kWave;
  for (int rr = wave; rr < R; rr += nw) {
    const float* sp = fu.ss + static_cast<size_t>(fu.xrow ? fu.xrow[rr] : rr) * np;
    float a = 0.f;
    for (int p0 = 0; p0 < np; p0 += 8 * kWave) {
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int p = p0 + j * kWave + lane;
        v[j] = p < np ? sp[p] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) a += v[j];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o, kWave);
    if (lane == 0) s_rs[rr] = 1.f / sqrtf(a / static_cast<float>(K) + fu.eps);
  }
}

// Operands of the fused epilogue that do not depend on the GEMM result, read
// before the main loop so that their latency hides under the weight stream:
// the residual and norm weight (kEpiAddF32), the slot and position
// (kEpiQKVRope).
struct EpiPre {
  float h = 0.f, wn = 0.f;
  int slot = 0, pos = 0;
};

template <int EPI>
__device__ __forceinline__ EpiPre epi_prefetch(const GemmFuse& fu, int m, int l16, int tile, int R, int N,
                                               const void* __restrict__ Y) {
  EpiPre p;
  const int n = tile * 16 + l16;
  if (m >= R) return p;
  if (EPI == kEpiAddF32 && n < N) {
    p.h = static_cast<const float*>(Y)[static_cast<size_t>(m) * N + n];
    if (fu.hb) p.wn = bf16_to_f32(static_cast<const bf16_t*>(fu.wn)[n]);
  } else if (EPI == kEpiQKVRope) {
    p.slot = fu.slot[m];
    p.pos = fu.pos[m];
  }
  return p;
}

// Epilogue of the fused GEMMs for output row m (< 16) and tile column l16 of
// 16-feature tile `tile`, given the (row-scaled) dot products v (and vu,
// the up rows of SwiGLU) and the prefetched operands.  Run by whole waves:
// threads 0..255 with m = 4 (lane / 16) + r, so the 16 lanes of a group hold
// the 16 columns of a row and exchange values with shuffles.
template <int EPI>
__device__ __forceinline__ void fused_epilogue(const GemmFuse& fu, const EpiPre& p, int m, int l16, int tile,
                                               int R, int N, float v, float vu, void* __restrict__ Y,
                                               const int32_t* __restrict__ row_map, int qk_tiles,
                                               int half = -1) {
  const int n0 = tile * 16;
  constexpr bool QKV = (EPI == kEpiQKVRope);
  const int n = n0 + l16;
  // half >= 0 (kEpiAddF32 only): the workgroup owns columns 8 half .. 8 half + 7 of the tile
  const bool ok = m < R && n < N && (half < 0 || (l16 >> 3) == half);
  if (EPI == kEpiAddF32) {
    float hn = 0.f;
    if (ok) {
      hn = p.h + v;
      static_cast<float*>(Y)[static_cast<size_t>(m) * N + n] = hn;
      if (fu.hb) static_cast<bf16_t*>(fu.hb)[static_cast<size_t>(m) * N + n] = f32_to_bf16(hn * p.wn);
    }
    if (fu.ss_out) {
      float sq = hn * hn;
#pragma unroll
      for (int o = 1; o < 8; o <<= 1) sq += __shfl_xor(sq, o, kWave);
      if ((l16 & 7) == 0 && ok) fu.ss_out[static_cast<size_t>(m) * (N / 8) + n / 8] = sq;
    }
  } else if (QKV) {
    const float partner = __shfl_xor(v, 8, kWave);
    if (m < R) {
      const int page = p.slot >> 4, off = p.slot & 15;
      if (tile < qk_tiles) {
        int head, dim;
        qkv_tile_row(fu, tile, l16, &head, &dim);
        const int i = dim % (fu.hd / 2);
        double sn, cs;
        sincos(static_cast<double>(p.pos) * exp(-(2.0 * i / fu.hd) * log(static_cast<double>(fu.theta))), &sn,
               &cs);
        const float c = static_cast<float>(cs), sv = static_cast<float>(sn);
        // first half: a cos - b sin; second half: b cos + a sin (a, b = pair)
        const float o = (l16 < 8) ? v * c - partner * sv : v * c + partner * sv;
        if (head < fu.Hq)
          static_cast<bf16_t*>(fu.qout)[(static_cast<size_t>(m) * fu.Hq + head) * fu.hd + dim] = f32_to_bf16(o);
        else
          static_cast<bf16_t*>(fu.kpool)[(static_cast<size_t>(page) * fu.Hkv + (head - fu.Hq)) * 16 * fu.hd +
                                         kv_k_off(off, dim)] = f32_to_bf16(o);
      } else if (n < N) {
        const int vi = n - (fu.Hq + fu.Hkv) * fu.hd;
        const int kh = vi / fu.hd, dd = vi % fu.hd;
        static_cast<bf16_t*>(fu.vpool)[(static_cast<size_t>(page) * fu.Hkv + kh) * fu.hd * 16 + kv_v_off(off, dd)] =
            f32_to_bf16(v);
      }
    }
  } else if (ok) {
    const size_t o = static_cast<size_t>(row_map ? row_map[m] : m) * N + n;
    if (EPI == kEpiStoreF32) static_cast<float*>(Y)[o] = v;
    if (EPI == kEpiSwiGLU) static_cast<bf16_t*>(Y)[o] = f32_to_bf16(silu(v) * vu);
  }
}

template <int MT, int EPI, bool FUSE>
__global__ __launch_bounds__(kSkinnyMaxWaves * kWave) void gemm_skinny_bf16(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, void* __restrict__ Y, int R, int N,
    int K, int kb_per_wave, const int32_t* __restrict__ row_map, const GemmFuse fu) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr bool QKV = (EPI == kEpiQKVRope);
  constexpr int NS = SW ? 2 : 1;  // weight streams: gate and up tiles for SwiGLU
  constexpr int NACC = MT * NS;
  static_assert(!FUSE || MT == 1, "the fused path covers up to 16 rows");
  static_assert(FUSE || !QKV, "the QKV epilogue is fused only");
  extern __shared__ float red[];  // [waves][NACC][4][64]
  __shared__ float s_rs[16];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int row = lane & 15, g = lane >> 4;
  const int tile = blockIdx.x;
  const int qk_tiles = QKV ? (fu.Hq + fu.Hkv) * fu.hd / 16 : 0;
  // Step s of lane group g reads row 4 s + g of the tile at chunk position
  // `row` (tiled layout): 16 bytes of W[tile * 16 + row][32 s + 8 g ..].  A
  // trailing partial tile is row-major, read at clamped rows.
  const bf16_t* wp[NS];
  int ws;  // element stride between steps
  {
    const bool full = (tile + 1) * 16 <= N;
    ws = full ? 4 * K : 32;
#pragma unroll
    for (int h = 0; h < NS; ++h)
      wp[h] = W + static_cast<size_t>(h) * N * K +
              (full ? static_cast<size_t>(tile * 16 + g) * K + row * 8
                    : static_cast<size_t>(min(tile * 16 + row, N - 1)) * K + g * 8);
  }
  const bf16_t* xr[MT];
  bool xv[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + row;
    xv[mt] = m < R;
    const int src = !xv[mt] ? 0 : ((FUSE && fu.xrow) ? fu.xrow[m] : m);
    xr[mt] = X + static_cast<size_t>(src) * K + g * 8;
  }
  // (measured: before the main loop here, after it in the GEMV)
  if (FUSE && fu.ss) row_rscale(fu, R, K, s_rs);
  // the fused epilogue (MT = 1) is run by threads 0..255, one element each
  EpiPre pre;
  const int e_r = (threadIdx.x / kWave) & 3;
  const int e_m = 4 * (lane >> 4) + e_r, e_l16 = lane & 15;
  if (FUSE && threadIdx.x < 256) pre = epi_prefetch<EPI>(fu, e_m, e_l16, tile, R, N, Y);
  f32x4 acc[MT][NS];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int h = 0; h < NS; ++h) acc[mt][h] = f32x4{0.f, 0.f, 0.f, 0.f};
  // KB 128-wide blocks per iteration (8 weight loads per lane in flight),
  // every load of the iteration issued before its first MFMA
  constexpr int KB = (NS * MT >= 2) ? 1 : 2;
  const int nb = K / 128;
  const int kb0 = wave * kb_per_wave;
  const int kb1 = min(nb, kb0 + kb_per_wave);
  for (int kb = kb0; kb < kb1; kb += KB) {
    uint4 w[KB][NS][4], x[KB][MT][4];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int ko = (kb + b < kb1 ? kb + b : kb) * 128;
#pragma unroll
      for (int h = 0; h < NS; ++h)
#pragma unroll
        for (int s = 0; s < 4; ++s) w[b][h][s] = ld_stream(reinterpret_cast<const uint4*>(wp[h] + ko + s * ws));
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int s = 0; s < 4; ++s)
          x[b][mt][s] = xv[mt] ? reinterpret_cast<const uint4*>(xr[mt] + ko)[4 * s] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      if (kb + b >= kb1) break;
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int h = 0; h < NS; ++h) acc[mt][h] = mfma16x16x32(x[b][mt][s], w[b][h][s], acc[mt][h]);
    }
  }
  // red[wave][(mt, h)][r][lane]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int h = 0; h < NS; ++h)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[((wave * NACC + mt * NS + h) * 4 + r) * kWave + lane] = acc[mt][h][r];
  __syncthreads();
  // element e: row block mt = e / 256, output row m = 16 mt + 4 (lane / 16) + r,
  // column l16.  Whole waves take the same mt, as the fused epilogue's 16-lane
  // exchanges need.
  for (int e = threadIdx.x; e < MT * 256; e += blockDim.x) {
    const int mt = e / 256, r = (e / kWave) & 3, ln = e & (kWave - 1);
    const int m = mt * 16 + 4 * (ln >> 4) + r, l16 = ln & 15;
    float v = 0.f, vu = 0.f;
    for (int wv = 0; wv < nw; ++wv) {
      v += red[((wv * NACC + mt * NS) * 4 + r) * kWave + ln];
      if (SW) vu += red[((wv * NACC + mt * NS + 1) * 4 + r) * kWave + ln];
    }
    if (FUSE) {
      if (fu.ss) {
        const float rs = s_rs[m];
        v *= rs;
        vu *= rs;
      }
      fused_epilogue<EPI>(fu, pre, m, l16, tile, R, N, v, vu, Y, row_map, qk_tiles);
      continue;
    }
    const int n = tile * 16 + l16;
    if (m < R && n < N) {
      const size_t o = static_cast<size_t>(row_map ? row_map[m] : m) * N + n;
      if (EPI == kEpiStoreF32) static_cast<float*>(Y)[o] = v;
      if (EPI == kEpiAddF32) static_cast<float*>(Y)[o] += v;
      if (EPI == kEpiSwiGLU) static_cast<bf16_t*>(Y)[o] = f32_to_bf16(silu(v) * vu);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMV for 1-2 rows (a single sequence's draft step): vector FMAs, no
// MFMA.  A workgroup owns one 16-feature tile (for SwiGLU its gate tile and
// its up tile).  Per 128-wide block a wave reads the tile's 16 rows in four
// loads of 4 rows x 256 bytes: lane (r = lane / 16, c = lane % 16) gets
// 16 bytes of feature c, chunk 4 q + r.  Waves split K (SwiGLU: waves 0-3 gate,
// 4-7 up); lanes of a feature reduce with shuffles, waves through LDS, then
// the fused epilogue.  HALF (residual-add projections with fewer tiles than
// compute units): two workgroups per tile, each owning 8 of its features and
// reading 8 rows x 128 bytes per load (lane r = lane / 8, c = lane % 8:
// feature 8 half + c, chunk 8 q + r), so that every compute unit streams
// weights: one workgroup moves only about 28 GB/s, whatever its loads in
// flight.

constexpr int kGemvRows = 2;  // measured: the MFMA skinny kernel wins from 3 rows on

// Shapes the fused one- and two-row path sends to the skinny MFMA kernel
// instead of the GEMV, measured on the batch-1 steps: the LM head of a model
// with d_model <= 2048 (the drafter's 128256 x 2048: 87.4 -> 77.8 us per
// draft step, 6.0 -> 6.8 TB/s; with d_model 4096 the GEMV stays ahead), and
// residual-add projections with K <= 2048 (the drafter's O projection:
// batch-1 step 7.07 -> 7.03 ms).  Sending the larger-K residual-add
// projections too was slower (7.11 ms).
__host__ inline bool gemv_lm_skinny(int R, int N, int K, int epi) {
  if (R > kGemvRows || K > 2048) return false;
  return (epi == kEpiStoreF32 && N >= 65536) || epi == kEpiAddF32;
}

// Half tiles for residual-add projections with fewer 16-feature tiles than
// compute units.
bool gemv_half(int epi, int N) { return epi == kEpiAddF32 && (N + 15) / 16 < 256; }

__device__ __forceinline__ float dot8(const u32x4& w, const u32x4& x) {
  float a = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    a = fmaf(__uint_as_float(w[j] << 16), __uint_as_float(x[j] << 16), a);
    a = fmaf(__uint_as_float(w[j] & 0xFFFF0000u), __uint_as_float(x[j] & 0xFFFF0000u), a);
  }
  return a;
}

template <int EPI, int RM, bool HALF>
__global__ __launch_bounds__(512) void gemv_bf16(const bf16_t* __restrict__ X, const bf16_t* __restrict__ W,
                                                 void* __restrict__ Y, int R, int N, int K,
                                                 const int32_t* __restrict__ row_map, const GemmFuse fu) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr bool QKV = (EPI == kEpiQKVRope);
  static_assert(!HALF || EPI == kEpiAddF32, "half tiles: residual-add projections");
  constexpr int NQ = HALF ? 2 : 4;   // weight loads per 128-wide block
  constexpr int KB = HALF ? 4 : 2;   // blocks per iteration: 8 weight loads in flight per lane
  constexpr int XS = HALF ? 64 : 32;  // element step of X between the loads of a block
  __shared__ float part[8][RM][16];  // [wave][row][feature]
  __shared__ float s_rs[16];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int tile = HALF ? static_cast<int>(blockIdx.x) >> 1 : blockIdx.x;
  const int half = HALF ? static_cast<int>(blockIdx.x & 1) : -1;
  const int c = HALF ? 8 * half + (lane & 7) : (lane & 15);  // feature within the tile
  const int r = HALF ? lane >> 3 : lane >> 4;
  const int qk_tiles = QKV ? (fu.Hq + fu.Hkv) * fu.hd / 16 : 0;
  const int grp = SW ? (wave >> 2) : 0;  // SwiGLU: gate (0) or up (1) tile
  const int gw = SW ? (wave & 3) : wave, ngw = SW ? 4 : 8;
  const bf16_t* wh = W + (grp ? static_cast<size_t>(N) * K : 0);
  // load q of block kb: wp + q * qs + kb * 128 (tiled: memory row
  // (16 / NQ) q + r at position c; a trailing partial tile is row-major at
  // clamped rows)
  const bool full = (tile + 1) * 16 <= N;
  const bf16_t* wp = wh + (full ? static_cast<size_t>(tile * 16 + r) * K + c * 8
                                : static_cast<size_t>(min(tile * 16 + c, N - 1)) * K + r * 8);
  const int qs = full ? (16 / NQ) * K : XS;
  const bf16_t* xp[RM];
#pragma unroll
  for (int m = 0; m < RM; ++m)
    xp[m] = X + static_cast<size_t>(m < R ? (fu.xrow ? fu.xrow[m] : m) : 0) * K + r * 8;
  // threads 0..255 run the epilogue: output row m = 4 (lane / 16) + (wave % 4)
  const int em = 4 * (lane >> 4) + (wave & 3);
  EpiPre pre;
  if (threadIdx.x < 256) pre = epi_prefetch<EPI>(fu, em, lane & 15, tile, R, N, Y);
  const int nb = K / 128;
  const int per = (nb + ngw - 1) / ngw;
  const int kb0 = gw * per, kb1 = min(nb, kb0 + per);
  float a[RM];
#pragma unroll
  for (int m = 0; m < RM; ++m) a[m] = 0.f;
  for (int kb = kb0; kb < kb1; kb += KB) {
    u32x4 w[KB][NQ], x[KB][RM][NQ];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int o = min(kb + b, kb1 - 1) * 128;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        w[b][q] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wp + o + q * qs));
#pragma unroll
        for (int m = 0; m < RM; ++m)
          if (m < R) x[b][m][q] = *reinterpret_cast<const u32x4*>(xp[m] + o + XS * q);
      }
    }
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      if (kb + b >= kb1) break;
#pragma unroll
      for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int m = 0; m < RM; ++m)
          if (m < R) a[m] += dot8(w[b][q], x[b][m][q]);
    }
  }
  if (fu.ss) row_rscale(fu, R, K, s_rs);
#pragma unroll
  for (int m = 0; m < RM; ++m) {
    if (HALF) a[m] += __shfl_xor(a[m], 8, kWave);
    a[m] += __shfl_xor(a[m], 16, kWave);
    a[m] += __shfl_xor(a[m], 32, kWave);
    if (lane < (HALF ? 8 : 16)) part[wave][m][c] = a[m];
  }
  __syncthreads();
  if (threadIdx.x >= 256) return;
  const int e = threadIdx.x, rr = (e / kWave) & 3, ln = e & (kWave - 1);
  const int m = 4 * (ln >> 4) + rr, l16 = ln & 15;
  float v = 0.f, vu = 0.f;
  if (m < R) {
    if (SW) {
      for (int wv = 0; wv < 4; ++wv) {
        v += part[wv][m][l16];
        vu += part[4 + wv][m][l16];
      }
    } else {
      for (int wv = 0; wv < 8; ++wv) v += part[wv][m][l16];
    }
    if (fu.ss) {
      v *= s_rs[m];
      vu *= s_rs[m];
    }
  }
  // (HALF: the other half's entries of part are not written; its lanes
  // store nothing)
  fused_epilogue<EPI>(fu, pre, m, l16, tile, R, N, v, vu, Y, row_map, qk_tiles, half);
}

template <int EPI>
hipError_t gemv(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                const int32_t* row_map, const GemmFuse& fu) {
  const int tiles = (N + 15) / 16;
  const bf16_t* x = static_cast<const bf16_t*>(X);
  const bf16_t* w = static_cast<const bf16_t*>(W);
  if (R > kGemvRows) return hipErrorInvalidValue;
  if constexpr (EPI == kEpiAddF32) {
    if (gemv_half(EPI, N)) {
      launch_kernel(gemv_bf16<EPI, kGemvRows, true>, dim3(2 * tiles), dim3(512), 0, st, x, w, Y, R, N, K, row_map, fu);
      return hipGetLastError();
    }
  }
  launch_kernel(gemv_bf16<EPI, kGemvRows, false>, dim3(tiles), dim3(512), 0, st, x, w, Y, R, N, K, row_map, fu);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// MFMA bf16, large tiles fed by direct-to-LDS loads: workgroup tile (32 MTW)
// rows x 256 W rows (128 gate + 128 up rows for SwiGLU), 4 waves as 2 (M) x
// 2 (N) of (16 MTW) x 128, one workgroup per CU (the accumulators, MTW x 8
// MFMA blocks, sit in the AGPR half of the register file).  Every k-step
// (BK = 32) of X and W is brought into LDS by global_load_lds_dwordx4, which
// writes each lane's 16 bytes in lane order with no register staging; four
// LDS stages, k-steps k + 1 .. k + 4 in flight while step k is multiplied.
// X: one load covers 16 rows x 64 bytes (chunks XOR-swizzled across banks).
// W (tiled layout): one load is one 16 x 32 MFMA fragment of a tile (4 memory
// rows x 256 bytes), so LDS holds the fragments in lane order and each lane
// reads back its own 16 bytes.  The fragments of step k + 1 are read from LDS
// while the MFMAs of step k run from registers; one barrier per k-step
// publishes the next stage.  Stages are separate LDS arrays.  The 1-D grid
// is decoded XCD-aware: workgroups are dispatched round-robin over the 8
// XCDs, so consecutive tile ids go to one XCD and the row tiles of a W tile
// share that XCD's L2.  Split-K writes raw fp32 partials by W row, which
// splitk_reduce sums in a fixed order; k-splits are multiples of 128
// (K % 128 == 0), so the step count is a multiple of 4 and the k-loop
// unrolls by 4 without remainders.

// MFMA accumulating in place, as inline asm: each accumulator stays in one
// AGPR tuple across the k-loop.  Compiler-generated MFMAs in this loop rotate
// the loop-carried accumulators through spare AGPRs, with four copies and a
// wait state per MFMA (measured in a register-only loop of 6 x 8 blocks:
// 1.5 PFLOP/s compiler-generated, 2.15 PFLOP/s in place).  The s_nop covers a
// VALU write of an operand or accumulator right before the MFMA; after the
// loop the kernel passes every accumulator through one compiler-generated
// MFMA, so that the reads of the epilogue follow an MFMA the compiler's
// hazard checks know about.
__device__ __forceinline__ void mfma_acc(f32x4& acc, const u32x4& a, const u32x4& b) {
  asm volatile("s_nop 1\n\tv_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

template <int EPI, int MTW, int NTW>
__global__ __launch_bounds__(256, 1) void gemm_mfma2_bf16(const bf16_t* __restrict__ X,
                                                          const bf16_t* __restrict__ W,
                                                          void* __restrict__ Y, float* __restrict__ part,
                                                          int R, int N, int K, int k_len, int MT, int NT,
                                                          const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr int TM = 32 * MTW;
  constexpr int NTG = 2 * NTW;      // 16-feature W tiles per workgroup
  constexpr int LA = TM / 64;       // X loads per wave per k-step (16 rows each)
  constexpr int LB = NTG / 4;       // W fragment loads per wave per k-step
  constexpr int NL = LA + LB;       // loads per wave per stage
  constexpr int SAU = TM * 4;       // 16-byte units of X per stage
  constexpr int STU = SAU + NTG * 64;
  static_assert(MTW % 2 == 0 && NTW % 2 == 0 && NTW >= 2, "MTW, NTW even");
  __shared__ u32x4 st0[STU], st1[STU], st2[STU], st3[STU];
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1), wave = t / kWave;
  const int wm = wave & 1, wn = wave >> 1;
  const int g = lane >> 4, l16 = lane & 15;
  const int total = gridDim.x, nid = blockIdx.x;
  const int xcd = nid & 7, slot = nid >> 3, per = total >> 3, rem = total & 7;
  const int tix = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
  const int mt = tix % MT, rest = tix / MT, sp = rest / NT, nt = rest % NT;
  const int m0 = mt * TM;
  const int f0 = nt * (SW ? 8 * NTG : 16 * NTG);
  const int kbeg = sp * k_len;
  const int nk = (min(K, kbeg + k_len) - kbeg) / 32;  // multiple of 4

  // X load q of this wave: row group wave * LA + q.  LDS unit u of a group
  // holds row u / 4, chunk (u % 4) ^ (u / 16): the XOR spreads the 16 rows a
  // fragment read touches over all 64 banks.  Lane l of a load writes unit l,
  // so it fetches that chunk.  Rows past R clamped (read, never written back).
  uint32_t xo[LA];
#pragma unroll
  for (int q = 0; q < LA; ++q)
    xo[q] = static_cast<uint32_t>(min(m0 + (wave * LA + q) * 16 + (lane >> 2), R - 1)) * K +
            ((lane & 3) ^ (lane >> 4)) * 8;
  // W load q of this wave: tile slot ts = wave * LB + q (SwiGLU: the first
  // NTG / 2 slots gate tiles f0 / 16 + ts, the rest the same up tiles); lane (l16, g) of k-step e
  // reads, in a full tile, memory row tile * 16 + 4 ((e / 32) % 4) + g at
  // chunk position l16 of block e / 128; a trailing partial tile is row-major
  // (row clamped to N - 1); tiles past N clamp to the last one.  Element
  // offsets fit 32 bits (checked by the launcher).
  const int ntiles = (N + 15) / 16;
  uint32_t wo[LB];
  uint32_t wfull = 0;
#pragma unroll
  for (int q = 0; q < LB; ++q) {
    const int ts = wave * LB + q;
    const int tile = min(SW ? (f0 / 16 + ts % (NTG / 2)) : (f0 / 16 + ts), ntiles - 1);
    const uint32_t half = (SW && ts >= NTG / 2) ? static_cast<uint32_t>(N) * K : 0u;
    const bool full = (tile + 1) * 16 <= N;
    wfull |= full ? (1u << q) : 0u;
    wo[q] = half + (full ? static_cast<uint32_t>(tile * 16 + g) * K + l16 * 8
                         : static_cast<uint32_t>(min(tile * 16 + l16, N - 1)) * K + g * 8);
  }
  auto issue = [&](u32x4* stage, int kt) {
    const uint32_t e = kbeg + 32 * kt;
    const uint32_t sb = lds_addr(stage);
#pragma unroll
    for (int q = 0; q < LA; ++q) load_lds16(X, (xo[q] + e) * 2, sb + (wave * LA + q) * 1024);
    const uint32_t of = ((e >> 5) & 3) * 4 * K + (e >> 7) * 128;
#pragma unroll
    for (int q = 0; q < LB; ++q)
      load_lds16(W, (wo[q] + (((wfull >> q) & 1) ? of : e)) * 2, sb + (SAU + (wave * LB + q) * 64) * 16);
  };

  f32x4 acc[MTW][NTW];
#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int j = 0; j < NTW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fragment reads: A row block i of the wave is row group MTW wm + i, lane
  // (l16, g) at unit l16 * 4 + (g ^ l16 / 4); B fragment j is tile slot
  // NTW wn + j (SwiGLU: gate slots (NTW / 2) wn + j for j < NTW / 2, and the
  // matching up slots NTG / 2 + (NTW / 2) wn + j - NTW / 2), each lane at its
  // own unit
  auto read_frags = [&](const u32x4* stage, u32x4 (&fa)[MTW], u32x4 (&fb)[NTW]) {
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int ts = SW ? ((j < NTW / 2 ? 0 : NTG / 2) + (NTW / 2) * wn + j % (NTW / 2)) : (NTW * wn + j);
      fb[j] = stage[SAU + ts * 64 + lane];
    }
#pragma unroll
    for (int i = 0; i < MTW; ++i) fa[i] = stage[(MTW * wm + i) * 64 + l16 * 4 + (g ^ (l16 >> 2))];
  };
  auto mma = [&](const u32x4 (&fa)[MTW], const u32x4 (&fb)[NTW]) {
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int j = 0; j < NTW; ++j) mfma_acc(acc[i][j], fa[i], fb[j]);
  };
  // Step k (fragments of k-step k already in registers): wait for this
  // wave's loads of stage k + 1 (later stages stay in flight) and its LDS
  // reads of stage k; a bare s_barrier publishes stage k + 1 to every wave and
  // ends all reads of stage k, whose buffer is refilled with k-step k + 4;
  // then the MFMAs of step k run while the fragments of step k + 1 are read.
  // (A __syncthreads would wait for every outstanding load: its workgroup
  // fence has to cover the LDS writes of the loads in flight.)  The signal
  // fences keep the compiler from moving LDS accesses across the barrier.
#define SPEC_M2_STEP(K_, SR, SN, FA, FB, GA, GB)                                                   \
  {                                                                                                \
    const int k_ = (K_);                                                                           \
    if (k_ + 3 < nk) {                                                                             \
      SPEC_WAIT_VM_LDS(2 * NL);                                                                    \
    } else if (k_ + 2 < nk) {                                                                      \
      SPEC_WAIT_VM_LDS(NL);                                                                        \
    } else {                                                                                       \
      SPEC_WAIT_VM_LDS(0);                                                                         \
    }                                                                                              \
    __atomic_signal_fence(__ATOMIC_SEQ_CST);                                                       \
    __builtin_amdgcn_s_barrier();                                                                  \
    __atomic_signal_fence(__ATOMIC_SEQ_CST);                                                       \
    if (k_ + 4 < nk) issue(SR, k_ + 4);                                                            \
    if (k_ + 1 < nk) read_frags(SN, GA, GB);                                                       \
    mma(FA, FB);                                                                                   \
  }
  u32x4 fa0[MTW], fb0[NTW], fa1[MTW], fb1[NTW];
  if (nk > 0) {
    issue(st0, 0);
    issue(st1, 1);
    issue(st2, 2);
    issue(st3, 3);
    SPEC_WAIT_VM_LDS(3 * NL);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    read_frags(st0, fa0, fb0);
  }
  for (int kt = 0; kt < nk; kt += 4) {
    SPEC_M2_STEP(kt, st0, st1, fa0, fb0, fa1, fb1);
    SPEC_M2_STEP(kt + 1, st1, st2, fa1, fb1, fa0, fb0);
    SPEC_M2_STEP(kt + 2, st2, st3, fa0, fb0, fa1, fb1);
    SPEC_M2_STEP(kt + 3, st3, st0, fa1, fb1, fa0, fb0);
  }
#undef SPEC_M2_STEP
  {  // acc + 0 * 0 (exact), by MFMAs the compiler sees
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int j = 0; j < NTW; ++j) acc[i][j] = mfma16x16x32v(z, z, acc[i][j]);
  }

#pragma unroll
  for (int i = 0; i < MTW; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 16 * MTW * wm + 16 * i + 4 * g + r;
      if (m >= R) continue;
      if (part) {
        float* pr = part + (static_cast<size_t>(sp) * R + m) * (SW ? 2 * N : N);
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          int n, wrow;
          if (SW) {
            n = f0 + 8 * NTW * wn + 16 * (j % (NTW / 2)) + l16;
            wrow = (j < NTW / 2 ? 0 : N) + n;
          } else {
            n = f0 + 16 * NTW * wn + 16 * j + l16;
            wrow = n;
          }
          if (n < N) pr[wrow] = acc[i][j][r];
        }
        continue;
      }
      const size_t mo = static_cast<size_t>(row_map ? row_map[m] : m);
      if (SW) {
#pragma unroll
        for (int j = 0; j < NTW / 2; ++j) {
          const int n = f0 + 8 * NTW * wn + 16 * j + l16;
          if (n < N)
            static_cast<bf16_t*>(Y)[mo * N + n] = f32_to_bf16(silu(acc[i][j][r]) * acc[i][j + NTW / 2][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
          const int n = f0 + 16 * NTW * wn + 16 * j + l16;
          if (n >= N) continue;
          float* y = static_cast<float*>(Y) + mo * N + n;
          if (EPI == kEpiStoreF32) *y = acc[i][j][r];
          if (EPI == kEpiAddF32) *y += acc[i][j][r];
        }
      }
    }
}

// ---------------------------------------------------------------------------
// MFMA bf16 with the weights streamed straight into registers, for the large
// single-pass shapes (SwiGLU gate/up and the LM head at 160+ rows): workgroup
// tile 16 MB rows x 4 NB 16-feature W tiles, 4 waves side by side along W
// (wave w owns W tiles w NB .. w NB + NB - 1; SwiGLU: gate tiles w NB / 2 ..
// and the same up tiles) against all 16 MB rows.  A W fragment is used by one
// wave only, so it goes global -> B-operand registers with no LDS round trip
// (tiled layout: one load is one fragment), D - 1 k-steps ahead.  The X tile
// of a k-step (16 MB rows x 64 bytes) goes to LDS by direct-to-LDS loads, D
// k-steps ahead, and every wave reads its A fragments from there one k-step
// ahead (two register buffers).  The loads and fragment reads of a step are
// spread between its MFMAs (one global load every MB NB / (NB + MB / 4)
// MFMAs): issued together at the start of the step they held the wave at the
// memory pipeline while its MFMAs waited (364-row gate/up: 130 -> 100 us).
// All global loads are inline asm with explicit waits; loads complete in
// issue order, so one s_waitcnt per k-step covers the X stage and the W
// fragments it needs.  The epilogue transposes each 4 x 4 quad of outputs so
// that a lane stores four consecutive columns of one row at once.
__device__ __forceinline__ void load_reg16(u32x4& d, const void* base, uint32_t off_bytes) {
  asm volatile("global_load_dwordx4 %0, %1, %2" : "=v"(d) : "v"(off_bytes), "s"(base));
}

// 4 x 4 transpose across each quad of lanes: lane q of a quad holds
// v[r] = M[r][q]; afterwards it holds v[c] = M[q][c].  Two rounds of
// neighbour exchanges (quad_perm 1,0,3,2 then 2,3,0,1), each lane keeping the
// elements whose index agrees with its own position in the bit exchanged.
__device__ __forceinline__ void quad_transpose(float (&v)[4]) {
  const int q = threadIdx.x & 3;
  float u[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float nb = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[r ^ 1]), 0xB1, 0xF, 0xF, false));
    u[r] = ((q ^ r) & 1) ? nb : v[r];
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const float nb = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(u[r ^ 2]), 0x4E, 0xF, 0xF, false));
    v[r] = ((q ^ r) & 2) ? nb : u[r];
  }
}

// Four consecutive outputs of a row, `left` of them inside the matrix: one
// wide store when all four are in and the address is aligned, else element
// by element (add: Y += v).
__device__ __forceinline__ void store_f32x4(float* y, const float (&v)[4], int left, bool add) {
  if (left >= 4 && (reinterpret_cast<uintptr_t>(y) & 15) == 0) {
    float4 o = make_float4(v[0], v[1], v[2], v[3]);
    if (add) {
      const float4 h = *reinterpret_cast<const float4*>(y);
      o.x += h.x;
      o.y += h.y;
      o.z += h.z;
      o.w += h.w;
    }
    *reinterpret_cast<float4*>(y) = o;
    return;
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (c < left) y[c] = add ? y[c] + v[c] : v[c];
}
__device__ __forceinline__ void store_bf16x4(bf16_t* y, const float (&v)[4], int left) {
  if (left >= 4 && (reinterpret_cast<uintptr_t>(y) & 7) == 0) {
    *reinterpret_cast<uint2*>(y) = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
    return;
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
    if (c < left) y[c] = f32_to_bf16(v[c]);
}

template <int EPI, int MB, int NB, int D>
__global__ __launch_bounds__(256, 1) void gemm_mfma3_bf16(const bf16_t* __restrict__ X,
                                                          const bf16_t* __restrict__ W, void* __restrict__ Y,
                                                          float* __restrict__ part, int R, int N, int K,
                                                          int k_len, int MT, int NT,
                                                          const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr int TM = 16 * MB;
  constexpr int NTG = 4 * NB;   // 16-feature W tiles per workgroup
  constexpr int LX = MB / 4;    // X loads per wave per k-step
  constexpr int XU = TM * 4;    // 16-byte units of X per stage
  constexpr int PER = NB + LX;  // loads per wave per k-step
  constexpr int NM = MB * NB;   // MFMAs per wave per k-step
  constexpr int GAP = NM / PER;
  static_assert(MB % 4 == 0 && (!SW || NB % 2 == 0) && D % 2 == 0 && (D - 2) * PER <= 63 && GAP >= 1, "shape");
  __shared__ u32x4 sx[D][XU];
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1), wave = t / kWave;
  const int g = lane >> 4, l16 = lane & 15;
  const int total = gridDim.x, nid = blockIdx.x;
  const int xcd = nid & 7, slot = nid >> 3, per = total >> 3, rem = total & 7;
  const int tix = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
  const int mt = tix % MT, rest = tix / MT, sp = rest / NT, nt = rest % NT;
  const int m0 = mt * TM;
  const int f0 = nt * (SW ? 8 * NTG : 16 * NTG);
  const int kbeg = sp * k_len;
  const int nk = (min(K, kbeg + k_len) - kbeg) / 32;  // a multiple of D (checked by the launcher)

  // X load q of this wave: row group wave * LX + q (16 rows x 64 bytes); LDS
  // unit u of a group holds row u / 4, chunk (u % 4) ^ (u / 16), so that an
  // A-fragment read (16 rows, one chunk each) touches all 64 banks; rows past
  // R clamped (read, never written back).
  uint32_t xo[LX];
#pragma unroll
  for (int q = 0; q < LX; ++q)
    xo[q] = static_cast<uint32_t>(min(m0 + (wave * LX + q) * 16 + (lane >> 2), R - 1)) * K + kbeg +
            ((lane & 3) ^ (lane >> 4)) * 8;
  // W fragment j: lane (l16, g) of k-step e reads memory row tile * 16 +
  // 4 ((e / 32) % 4) + g at chunk position l16 of block e / 128 (full tile);
  // a trailing partial tile is row-major (row clamped to N - 1); tiles past N
  // clamp to the last one.
  const int ntiles = (N + 15) / 16;
  uint32_t wo[NB];
  uint32_t wfull = 0;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int tl = SW ? (f0 / 16 + wave * (NB / 2) + j % (NB / 2)) : (f0 / 16 + wave * NB + j);
    const int tile = min(tl, ntiles - 1);
    const uint32_t half = (SW && j >= NB / 2) ? static_cast<uint32_t>(N) * K : 0u;
    const bool full = (tile + 1) * 16 <= N;
    wfull |= full ? (1u << j) : 0u;
    wo[j] = half + (full ? static_cast<uint32_t>(tile * 16 + g) * K + l16 * 8
                         : static_cast<uint32_t>(min(tile * 16 + l16, N - 1)) * K + g * 8);
  }
  // k-steps past the end are clamped to the last one (redundant cache hits),
  // so that every k-step issues the same loads and the wait counts hold
  auto w_off = [&](int j, int k) {
    const uint32_t e = kbeg + 32 * min(k, nk - 1);
    return (wo[j] + (((wfull >> j) & 1) ? ((e >> 5) & 3) * 4 * K + (e >> 7) * 128 : e)) * 2;
  };
  auto x_load = [&](int q, int s, int k) {
    load_lds16(X, (xo[q] + 32 * min(k, nk - 1)) * 2, lds_addr(&sx[s][0]) + (wave * LX + q) * 1024);
  };

  f32x4 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 wr[D][NB];
  u32x4 fa[2][MB];
  // prologue: X(0), then W(p), X(p + 1) for p < D - 1; A fragments of X(0)
#pragma unroll
  for (int q = 0; q < LX; ++q) x_load(q, 0, 0);
#pragma unroll
  for (int p = 0; p < D - 1; ++p) {
#pragma unroll
    for (int j = 0; j < NB; ++j) load_reg16(wr[p][j], W, w_off(j, p));
#pragma unroll
    for (int q = 0; q < LX; ++q) x_load(q, p + 1, p + 1);
  }
  SPEC_WAIT_VM_LDS((D - 1) * PER);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
#pragma unroll
  for (int i = 0; i < MB; ++i) fa[0][i] = sx[0][i * 64 + l16 * 4 + (g ^ (l16 >> 2))];

  // k-step k (slot s = k % D): wait until X(k + 1) has landed (and with it
  // W(k), issued just before it) and this wave's LDS reads are done; the
  // barrier publishes stage (k + 1) % D and ends every read of stage s.  Then
  // the MFMAs of k, with W(k + D - 1) going into the slot W(k - 1) used,
  // X(k + D) into stage s and the A fragments of k + 1 read in between.
  for (int kt = 0; kt < nk; kt += D) {
#pragma unroll
    for (int s = 0; s < D; ++s) {
      const int k = kt + s;
      SPEC_WAIT_VM_LDS((D - 2) * PER);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_barrier();
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      const int sn = (s + 1) % D;
#pragma unroll
      for (int u = 0; u < NM; ++u) {
        const int i = u / NB, j = u % NB;
        if (u % GAP == 0 && u / GAP < PER) {
          const int q = u / GAP;
          if (q < NB) load_reg16(wr[(s + D - 1) % D][q], W, w_off(q, k + D - 1));
          else x_load(q - NB, s, k + D);
        }
        // past the end: stale data, never used
        if (j == 0) fa[(s + 1) & 1][i] = sx[sn][i * 64 + l16 * 4 + (g ^ (l16 >> 2))];
        mfma_acc(acc[i][j], fa[s & 1][i], wr[s][j]);
      }
    }
  }
  // The clamped loads past the end land before their registers are reused:
  // the compiler does not see the inline-asm loads in flight, so every W
  // register stays live (an empty asm reads it) until after the wait.
  SPEC_WAIT_VM_LDS(0);
#pragma unroll
  for (int s = 0; s < D; ++s)
#pragma unroll
    for (int j = 0; j < NB; ++j) asm volatile("" ::"v"(wr[s][j]));
  {  // acc + 0 * 0 (exact), by MFMAs the compiler sees
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[i][j] = mfma16x16x32v(z, z, acc[i][j]);
  }

  // Split K: raw fp32 partials by W row, which splitk_reduce* sums in a fixed
  // order, stored lane by lane (16 lanes of a row write 64 contiguous bytes;
  // measured faster here than the transposed form below).
  if (part) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 16 * i + 4 * g + r;
        if (m >= R) continue;
        float* pr = part + (static_cast<size_t>(sp) * R + m) * (SW ? 2 * N : N);
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = f0 + 16 * (SW ? wave * (NB / 2) + j % (NB / 2) : wave * NB + j) + l16;
          if (n < N) pr[(SW && j >= NB / 2 ? N : 0) + n] = acc[i][j][r];
        }
      }
    return;
  }
  // Lane (l16, g) holds rows 4 g + r of column l16 of each 16 x 16 block;
  // after the quad transpose it holds row 4 g + l16 % 4, columns
  // 4 (l16 / 4) .. + 3.
  const int q4 = l16 & 3, c4 = (l16 >> 2) * 4;
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const int m = m0 + 16 * i + 4 * g + q4;
    const size_t mo = (m < R && row_map) ? static_cast<size_t>(row_map[m]) : static_cast<size_t>(m);
#pragma unroll
    for (int j = 0; j < (SW ? NB / 2 : NB); ++j) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = SW ? silu(acc[i][j][r]) * acc[i][j + NB / 2][r] : acc[i][j][r];
      quad_transpose(v);
      const int n = f0 + 16 * (SW ? wave * (NB / 2) + j : wave * NB + j) + c4;
      if (m >= R || n >= N) continue;
      if (SW)
        store_bf16x4(static_cast<bf16_t*>(Y) + mo * N + n, v, N - n);
      else
        store_f32x4(static_cast<float*>(Y) + mo * N + n, v, N - n, EPI == kEpiAddF32);
    }
  }
}

// Sum split-K partials [S][R][Nw] in split order and apply the epilogue.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce(const float* __restrict__ part, int S, int R, int N,
                                                     void* __restrict__ Y, const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  const int Nw = SW ? 2 * N : N;
  const size_t total = static_cast<size_t>(R) * N;
  for (size_t e = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
       e += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int m = static_cast<int>(e / N), n = static_cast<int>(e % N);
    float v = 0.f, u = 0.f;
    for (int s = 0; s < S; ++s) {
      const float* pr = part + (static_cast<size_t>(s) * R + m) * Nw;
      v += pr[n];
      if (SW) u += pr[N + n];
    }
    const size_t o = static_cast<size_t>(row_map ? row_map[m] : m) * N + n;
    if (EPI == kEpiStoreF32) static_cast<float*>(Y)[o] = v;
    if (EPI == kEpiAddF32) static_cast<float*>(Y)[o] += v;
    if (EPI == kEpiSwiGLU) static_cast<bf16_t*>(Y)[o] = f32_to_bf16(silu(v) * u);
  }
}

// The same sum for N % 4 == 0, 4 columns per thread: every split's loads
// (gate and up for SwiGLU) go out in batches of 8 before the first add, and
// the output row index with them, so that a reduction over S splits costs
// one or two round trips rather than S.  Sums in split order, as above.
template <int EPI>
__global__ __launch_bounds__(256) void splitk_reduce4(const float* __restrict__ part, int S, int R, int N,
                                                      void* __restrict__ Y, const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr int B = 8;
  const int n4 = N / 4, nw4 = SW ? 2 * n4 : n4;
  const size_t ps = static_cast<size_t>(R) * nw4;  // float4 stride between splits
  const size_t total = static_cast<size_t>(R) * n4;
  for (size_t e = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < total;
       e += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int m = static_cast<int>(e / n4), c = static_cast<int>(e % n4);
    const int row = row_map ? row_map[m] : m;
    const float4* pr = reinterpret_cast<const float4*>(part) + static_cast<size_t>(m) * nw4 + c;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f), u = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < S; s0 += B) {
      float4 p[B], q[SW ? B : 1];
#pragma unroll
      for (int b = 0; b < B; ++b) {
        const size_t o = static_cast<size_t>(min(s0 + b, S - 1)) * ps;
        p[b] = pr[o];
        if (SW) q[b] = pr[o + n4];
      }
#pragma unroll
      for (int b = 0; b < B; ++b) {
        if (s0 + b >= S) break;
        v.x += p[b].x;
        v.y += p[b].y;
        v.z += p[b].z;
        v.w += p[b].w;
        if (SW) {
          u.x += q[b].x;
          u.y += q[b].y;
          u.z += q[b].z;
          u.w += q[b].w;
        }
      }
    }
    const size_t o = static_cast<size_t>(row) * n4 + c;
    if (EPI == kEpiStoreF32) reinterpret_cast<float4*>(Y)[o] = v;
    if (EPI == kEpiAddF32) {
      float4 h = reinterpret_cast<float4*>(Y)[o];
      h.x += v.x;
      h.y += v.y;
      h.z += v.z;
      h.w += v.w;
      reinterpret_cast<float4*>(Y)[o] = h;
    }
    if (EPI == kEpiSwiGLU)
      reinterpret_cast<uint2*>(Y)[o] = make_uint2(pack_bf16x2(silu(v.x) * u.x, silu(v.y) * u.y),
                                                  pack_bf16x2(silu(v.z) * u.z, silu(v.w) * u.w));
  }
}

// Split-K sum of a residual-add GEMM fused with the RMSNorm after it, one
// workgroup of T threads per row m (N % 4 == 0, N <= 4 * 1024 * kNormRegChunks):
// thread t holds the NCH 4-column chunks t, t + T, ... of the row in
// registers, adds the partials in split order to h (as splitk_reduce does),
// writes h, then y[m] = bf16(h[m] / rms(h[m]) (.) w) with the sum of squares
// taken per thread in chunk order, then over the wave and the waves in a
// fixed order.  Every load of a thread goes out before the first is used (h,
// w, then the partials in batches of 8 / NCH splits, indexes clamped so that
// the loads are unconditional): with up to 1024 threads a row of 4096 columns
// split 8 ways is one round trip (256 threads took four).
constexpr int kNormRegChunks = 4;

template <int NCH, int T>
__global__ __launch_bounds__(T) void splitk_reduce_norm(const float* __restrict__ part, int S, int R, int N,
                                                        float* __restrict__ Y, const bf16_t* __restrict__ w,
                                                        float eps, bf16_t* __restrict__ y) {
  constexpr int B = NCH >= 8 ? 1 : 8 / NCH;  // splits per batch of loads
  constexpr int NW = T / kWave;
  const int m = blockIdx.x;
  const int nch = N / 4;
  const float4* pp = reinterpret_cast<const float4*>(part) + static_cast<size_t>(m) * nch;
  const size_t ps = static_cast<size_t>(R) * nch;  // float4 stride between splits
  float4* hp = reinterpret_cast<float4*>(Y + static_cast<size_t>(m) * N);
  int ch[NCH];
  float4 h[NCH], v[NCH];
  uint2 wv[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    ch[c] = min(static_cast<int>(threadIdx.x) + c * T, nch - 1);
    h[c] = hp[ch[c]];
    wv[c] = reinterpret_cast<const uint2*>(w)[ch[c]];
    v[c] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  for (int s0 = 0; s0 < S; s0 += B) {
    float4 p[B][NCH];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
      for (int c = 0; c < NCH; ++c) p[b][c] = pp[min(s0 + b, S - 1) * ps + ch[c]];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      if (s0 + b >= S) break;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        v[c].x += p[b][c].x;
        v[c].y += p[b][c].y;
        v[c].z += p[b][c].z;
        v[c].w += p[b][c].w;
      }
    }
  }
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (static_cast<int>(threadIdx.x) + c * T >= nch) continue;
    h[c].x += v[c].x;
    h[c].y += v[c].y;
    h[c].z += v[c].z;
    h[c].w += v[c].w;
    hp[ch[c]] = h[c];
    ss = fmaf(h[c].x, h[c].x, ss);
    ss = fmaf(h[c].y, h[c].y, ss);
    ss = fmaf(h[c].z, h[c].z, ss);
    ss = fmaf(h[c].w, h[c].w, ss);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, kWave);
  __shared__ float s_part[NW];
  if ((threadIdx.x & (kWave - 1)) == 0) s_part[threadIdx.x / kWave] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) tot += s_part[i];
  const float inv = 1.f / sqrtf(tot / static_cast<float>(N) + eps);
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    if (static_cast<int>(threadIdx.x) + c * T >= nch) continue;
    const float v0 = h[c].x * inv * __uint_as_float(wv[c].x << 16);
    const float v1 = h[c].y * inv * __uint_as_float(wv[c].x & 0xFFFF0000u);
    const float v2 = h[c].z * inv * __uint_as_float(wv[c].y << 16);
    const float v3 = h[c].w * inv * __uint_as_float(wv[c].y & 0xFFFF0000u);
    reinterpret_cast<uint2*>(y + static_cast<size_t>(m) * N)[ch[c]] =
        make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
  }
}

// ---------------------------------------------------------------------------
// fp32: 64x64 tiles (64x32 features + their up rows for SwiGLU), BK = 16

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32(const float* __restrict__ X,
                                                const float* __restrict__ W, void* __restrict__ Y,
                                                int R, int N, int K,
                                                const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const int t = threadIdx.x, tx = t & 15, ty = t >> 4;
  const int m0 = blockIdx.y * 64;
  const int ncols = SW ? 32 : 64;
  const int f0 = blockIdx.x * ncols;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = t; e < 64 * 16; e += 256) {
      const int r = e >> 4, kk = e & 15;
      const int m = m0 + r, k = k0 + kk;
      As[kk][r] = (m < R && k < K) ? X[static_cast<size_t>(m) * K + k] : 0.f;
      int wrow;
      bool ok;
      if (SW) {
        const int f = f0 + (r & 31);
        ok = f < N;
        wrow = (r < 32 ? 0 : N) + f;
      } else {
        wrow = f0 + r;
        ok = wrow < N;
      }
      Bs[kk][r] = (ok && k < K) ? W[static_cast<size_t>(wrow) * K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int col = SW ? (c < 2 ? tx * 2 + c : 32 + tx * 2 + (c - 2)) : tx * 4 + c;
        b[c] = Bs[kk][col];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[i][c] = fmaf(a[i], b[c], acc[i][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= R) continue;
    const size_t mo = static_cast<size_t>(row_map ? row_map[m] : m);
    if (SW) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int n = f0 + tx * 2 + c;
        if (n < N) {
          const float gv = acc[i][c];
          static_cast<float*>(Y)[mo * N + n] = gv / (1.f + expf(-gv)) * acc[i][c + 2];
        }
      }
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int n = f0 + tx * 4 + c;
        if (n >= N) continue;
        float* y = static_cast<float*>(Y) + mo * N + n;
        if (EPI == kEpiStoreF32) *y = acc[i][c];
        if (EPI == kEpiAddF32) *y += acc[i][c];
      }
    }
  }
}

// Waves per workgroup of the skinny kernel: 8 split K when there are few
// tiles, else 4 (measured on the 8B/1B-shaped projections at 6 rows).
int skinny_waves(int tiles, int K) { return (tiles <= 512 && K >= 2048) ? 8 : 4; }

template <int MT, int EPI, bool FUSE = false>
hipError_t skinny(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                  const int32_t* row_map, const GemmFuse& fu = GemmFuse{}) {
  constexpr int NACC = MT * (EPI == kEpiSwiGLU ? 2 : 1);
  const int tiles = (N + 15) / 16;
  const int nb = K / 128;
  int nw = std::max(FUSE ? 4 : 1, std::min(skinny_waves(tiles, K), nb));
  if (FUSE && nw < 4) return hipErrorInvalidValue;  // the fused epilogue needs 256 threads
  const int kbpw = (nb + nw - 1) / nw;
  const size_t lds = static_cast<size_t>(nw) * NACC * 256 * sizeof(float);
  launch_kernel(gemm_skinny_bf16<MT, EPI, FUSE>, dim3(tiles), dim3(nw * kWave), lds, st, static_cast<const bf16_t*>(X),
                static_cast<const bf16_t*>(W), Y, R, N, K, kbpw, row_map, fu);
  return hipGetLastError();
}

// Split-K of gemm_mfma2_bf16: grids under 192 tiles are split so that
// tiles x splits fills the 256 CUs about once (k-splits multiples of 128,
// partials within the workspace).  Returns S and the k-split length.
int mfma2_splits(int MT, int NT, int R, int Nw, int K, size_t ws_bytes, int* k_len) {
  int S = 1;
  if (ws_bytes && MT * NT < 192) {
    S = std::max(1, std::min(8, 256 / (MT * NT)));
    while (S > 1 && static_cast<size_t>(S) * R * Nw * sizeof(float) > ws_bytes) --S;
  }
  *k_len = ((K + S - 1) / S + 127) / 128 * 128;
  return (K + *k_len - 1) / *k_len;
}

// Tile shape of gemm_mfma2_bf16: rows per workgroup 32 MTW (64 .. 256) and W
// rows per workgroup 32 NTW (64 .. 256), the pair with the least estimated
// time in a cost model fitted (least squares, median error 10%) to measured
// launches of every shape at 64, 128 and 364 rows of the 8B/1B-shaped
// projections: per-step terms for the MFMAs and the LDS loads of a
// workgroup, times the k-steps and the rounds of workgroups over the 256
// CUs, plus the split-K partial traffic.  Wide tiles waste rows or feed too
// few CUs on small problems; narrow ones reload X and W more often.  A split
// SwiGLU pays its second pass as a launch of its own (≈ 6 us; the residual-add
// and QKV reductions ride on launches that follow anyway: the RMSNorm and the
// rotary embedding): with it the 41-128-row gate/up projections take narrow
// unsplit tiles (41-row 1B-shaped gate/up 19.6 -> 16.9 us, 8B-shaped
// 40.8 -> 36.2 us).
struct Mfma2Shape {
  int mtw, ntw;
};

Mfma2Shape mfma2_shape(int R, int N, int Nw, int K, size_t ws_bytes, bool swiglu) {
  Mfma2Shape best{2, 2};
  double best_t = 1e300;
  for (int mtw : {2, 4, 6, 8}) {
    if (32 * mtw > 2 * R + 64) continue;  // tiles far taller than R
    for (int ntw : {2, 4, 8}) {
      const int MT = (R + 32 * mtw - 1) / (32 * mtw), NT = (Nw + 32 * ntw - 1) / (32 * ntw);
      int k_len = K;
      const int S = mfma2_splits(MT, NT, R, Nw, K, ws_bytes, &k_len);
      const double rounds = (MT * NT * S + 255) / 256;  // whole rounds of workgroups over the CUs
      const double steps = rounds * (k_len / 32);
      const double red_mb = S > 1 ? (S + 1.0) * R * N * 4.0 / 1e6 : 0.0;
      const double t = 0.0119 * steps * mtw * ntw + 0.0056 * steps * (32.0 * (mtw + ntw)) * 64.0 / 1024.0 +
                       0.0574 * steps + 0.3048 * red_mb + (S > 1 ? (swiglu ? 6.0 : -6.41) : 0.0);
      if (t < best_t) {
        best_t = t;
        best = {mtw, ntw};
      }
    }
  }
  return best;
}

template <int EPI>
hipError_t splitk_finish(const float* ws, int S, int R, int N, void* Y, hipStream_t st, const int32_t* rm,
                         GemmNorm* norm);

template <int EPI, int MTW, int NTW>
hipError_t mfma2_t(int R, int N, int K, const bf16_t* x, const bf16_t* w, void* Y, hipStream_t st,
                   const int32_t* rm, float* ws, size_t ws_bytes, GemmNorm* norm = nullptr) {
  const int Nw = (EPI == kEpiSwiGLU) ? 2 * N : N;
  if (static_cast<double>(Nw) * K >= 2147483648.0 || static_cast<double>(R) * K >= 2147483648.0 || K % 128)
    return hipErrorInvalidValue;  // 32-bit byte offsets; whole 128-wide blocks
  const int MT = (R + 32 * MTW - 1) / (32 * MTW), NT = (Nw + 32 * NTW - 1) / (32 * NTW);
  int k_len = K;
  const int S = mfma2_splits(MT, NT, R, Nw, K, ws ? ws_bytes : 0, &k_len);
  const int grid = MT * NT * S;
  if (S <= 1) {
    launch_kernel(gemm_mfma2_bf16<EPI, MTW, NTW>, dim3(grid), dim3(256), 0, st, x, w, Y, static_cast<float*>(nullptr), R,
                  N, K, K, MT, NT, rm);
    return hipGetLastError();
  }
  launch_kernel(gemm_mfma2_bf16<EPI, MTW, NTW>, dim3(grid), dim3(256), 0, st, x, w, static_cast<void*>(nullptr), ws, R,
                N, K, k_len, MT, NT, rm);
  return splitk_finish<EPI>(ws, S, R, N, Y, st, rm, norm);
}

// The second pass of a split-K GEMM: the partials [S][R][Nw] summed in split
// order with the epilogue applied (for a residual add followed by RMSNorm,
// the norm too).
template <int EPI>
hipError_t splitk_finish(const float* ws, int S, int R, int N, void* Y, hipStream_t st, const int32_t* rm,
                         GemmNorm* norm) {
  if (EPI == kEpiStoreF32 && norm && norm->defer && !rm) {  // the consumer sums the partials
    norm->split = S;
    norm->part = ws;
    return hipSuccess;
  }
  if (EPI == kEpiAddF32 && norm && !rm && N % 4 == 0 && N <= 4 * 1024 * kNormRegChunks) {
    const int n4 = N / 4;
    auto* k = n4 <= 256 ? splitk_reduce_norm<1, 256> : n4 <= 512 ? splitk_reduce_norm<1, 512>
            : n4 <= 1024 ? splitk_reduce_norm<1, 1024> : n4 <= 2048 ? splitk_reduce_norm<2, 1024>
            : splitk_reduce_norm<4, 1024>;
    const int T = n4 <= 256 ? 256 : n4 <= 512 ? 512 : 1024;
    k<<<R, T, 0, st>>>(ws, S, R, N, static_cast<float*>(Y), static_cast<const bf16_t*>(norm->w), norm->eps,
                       static_cast<bf16_t*>(norm->y));
    norm->done = true;
    return hipGetLastError();
  }
  if (N % 4 == 0) {
    const size_t total = static_cast<size_t>(R) * (N / 4);
    const int blocks = static_cast<int>(std::min<size_t>(2048, (total + 255) / 256));
    splitk_reduce4<EPI><<<blocks, 256, 0, st>>>(ws, S, R, N, Y, rm);
    return hipGetLastError();
  }
  const size_t total = static_cast<size_t>(R) * N;
  const int blocks = static_cast<int>(std::min<size_t>(2048, (total + 255) / 256));
  splitk_reduce<EPI><<<blocks, 256, 0, st>>>(ws, S, R, N, Y, rm);
  return hipGetLastError();
}

template <int EPI, int MTW>
hipError_t mfma2_m(int ntw, int R, int N, int K, const bf16_t* x, const bf16_t* w, void* Y, hipStream_t st,
                   const int32_t* rm, float* ws, size_t ws_bytes, GemmNorm* norm = nullptr) {
  switch (ntw) {
    case 2: return mfma2_t<EPI, MTW, 2>(R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
    case 4: return mfma2_t<EPI, MTW, 4>(R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
    default: return mfma2_t<EPI, MTW, 8>(R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
  }
}

// gemm_mfma3_bf16 (weights straight to registers), 192 x 256 tiles for the
// shapes it was measured to win: SwiGLU gate/up from 160 rows in one pass
// (364-row serving verify 114 -> 97 us, 2048-row prefill 508 -> 433 us, 8192
// rows 1966 -> 1641 us), store-only projections of 65536+ rows in one pass
// (the LM head: 425 -> 404 us at 364 rows), each when the tiles fill the 256
// CUs at least 3 / 4 of the way; and residual-add projections with K >= 8192
// whose grid splits K (the 364-row down projection: 76 -> 64 us).  Elsewhere
// (the QKV and O projections, the unsplit 2048-row down projection)
// gemm_mfma2_bf16 was as fast or faster.
constexpr int kM3MB = 12, kM3NB = 4, kM3D = 4;
// Small form: 64-row tiles (MB 4) of 64 NB W rows, K split to fill the CUs,
// for the drafter's and the target's 41-128-row projections, where every
// workgroup streams all of X: a 64-row tile streams 4 KB of X per k-step
// through LDS against the 16 KB of the 192-row form.
constexpr int kM3sMB = 4;

struct Mfma3Plan {
  int MT, NT, S, k_len;
  int nb;  // 0: the 192 x 256 form; else the small form with NB = nb
};

// NB of the small form for a projection of R rows, or 0 where
// gemm_mfma2_bf16 is used (more than 128 rows; the 65536+-row LM heads).  From
// a sweep of NB in {1, 2, 4} against gemm_mfma2_bf16 over 13-150 rows of the
// 8B- and 1B-shaped projections: a residual add or plain store wants about 64
// tiles (K split 4 ways), so the narrowest W tile with at most 64 tiles; a
// SwiGLU, whose split costs a launch of its own, the widest tile that still
// fills 192 CUs unsplit, else NB = 2.  Measured against gemm_mfma2_bf16:
// 8B-shaped O projection at 41 rows 13.6 -> 11.3 us, gate/up at 96 rows 47.0 ->
// 37.9 us, down at 96 rows 31.4 -> 27.6 us; 1B-shaped down at 41 rows 13.5 ->
// 12.3 us, gate/up at 78 rows 20.1 -> 17.6 us; elsewhere within a few percent.
int mfma3_small_nb(int R, int Nw, int K, int epi) {
  (void)K;
  if (R > 128 || Nw >= 65536) return 0;
  const int MT = (R + 16 * kM3sMB - 1) / (16 * kM3sMB);
  auto tiles = [&](int nb) { return MT * ((Nw + 64 * nb - 1) / (64 * nb)); };
  if (epi == kEpiSwiGLU) return tiles(4) >= 192 ? 4 : 2;
  for (int nb : {1, 2}) if (tiles(nb) <= 64) return nb;
  return 4;
}

bool use_mfma3(int R, int Nw, int K, int epi, size_t ws_bytes, Mfma3Plan* plan = nullptr) {
  if (K % (32 * kM3D)) return false;
  if (static_cast<double>(Nw) * K >= 2147483648.0 || static_cast<double>(R) * K >= 2147483648.0) return false;
  if (R < 160) {
    const int nb = ws_bytes ? mfma3_small_nb(R, Nw, K, epi) : 0;
    if (nb == 0 || (epi == kEpiSwiGLU && nb % 2)) return false;
    const int MT = (R + 16 * kM3sMB - 1) / (16 * kM3sMB), NT = (Nw + 64 * nb - 1) / (64 * nb);
    int k_len = K;
    const int S = mfma2_splits(MT, NT, R, Nw, K, ws_bytes, &k_len);  // k_len: a multiple of 128 = 32 D
    if (plan) *plan = {MT, NT, S, k_len, nb};
    return true;
  }
  const int MT = (R + 16 * kM3MB - 1) / (16 * kM3MB), NT = (Nw + 64 * kM3NB - 1) / (64 * kM3NB);
  int k_len = K, S = 1;
  bool ok;
  if (epi == kEpiAddF32) {
    S = mfma2_splits(MT, NT, R, Nw, K, ws_bytes, &k_len);  // k_len: a multiple of 128 = 32 D
    ok = K >= 8192 && S >= 2;
  } else {
    ok = (epi == kEpiSwiGLU || (epi == kEpiStoreF32 && Nw >= 65536)) && MT * NT >= 192;
  }
  if (!ok && epi == kEpiAddF32 && K < 8192 && Nw >= 4096 && Nw < 65536 && R <= 384) {
    // the residual-add projections of the 8B-shaped target at 160-384 rows
    // (the serving verify's O projection): the 64-row form with 256-row W
    // tiles, K split (364 rows 29.2 -> 25.4 us against gemm_mfma2_bf16)
    const int MTs = (R + 16 * kM3sMB - 1) / (16 * kM3sMB), NTs = (Nw + 255) / 256;
    int kl = K;
    const int Ss = mfma2_splits(MTs, NTs, R, Nw, K, ws_bytes, &kl);
    if (ws_bytes && plan) *plan = {MTs, NTs, Ss, kl, 4};
    return ws_bytes != 0;
  }
  if (ok && plan) *plan = {MT, NT, S, k_len, 0};
  return ok;
}

template <int EPI>
auto mfma3_kernel(int nb) {
  if constexpr (EPI == kEpiSwiGLU) {
    return nb == 0 ? gemm_mfma3_bf16<EPI, kM3MB, kM3NB, kM3D>
                   : nb == 2 ? gemm_mfma3_bf16<EPI, kM3sMB, 2, kM3D> : gemm_mfma3_bf16<EPI, kM3sMB, 4, kM3D>;
  } else {
    return nb == 0 ? gemm_mfma3_bf16<EPI, kM3MB, kM3NB, kM3D>
                   : nb == 1 ? gemm_mfma3_bf16<EPI, kM3sMB, 1, kM3D>
                             : nb == 2 ? gemm_mfma3_bf16<EPI, kM3sMB, 2, kM3D> : gemm_mfma3_bf16<EPI, kM3sMB, 4, kM3D>;
  }
}

template <int EPI>
hipError_t mfma3(int R, int N, int K, const bf16_t* x, const bf16_t* w, void* Y, hipStream_t st, const int32_t* rm,
                 float* ws, const Mfma3Plan& p, GemmNorm* norm) {
  auto* kern = mfma3_kernel<EPI>(p.nb);
  if (p.S <= 1) {
    launch_kernel(kern, dim3(p.MT * p.NT), dim3(256), 0, st, x, w, Y, static_cast<float*>(nullptr), R, N, K, K, p.MT,
                  p.NT, rm);
    return hipGetLastError();
  }
  launch_kernel(kern, dim3(p.MT * p.NT * p.S), dim3(256), 0, st, x, w, static_cast<void*>(nullptr), ws, R, N, K,
                p.k_len, p.MT, p.NT, rm);
  return splitk_finish<EPI>(ws, p.S, R, N, Y, st, rm, norm);
}

template <int EPI>
hipError_t mfma2(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                 const int32_t* rm, float* ws, size_t ws_bytes, GemmNorm* norm = nullptr) {
  const bf16_t* x = static_cast<const bf16_t*>(X);
  const bf16_t* w = static_cast<const bf16_t*>(W);
  Mfma3Plan p3;
  if (use_mfma3(R, EPI == kEpiSwiGLU ? 2 * N : N, K, EPI, ws ? ws_bytes : 0, &p3))
    return mfma3<EPI>(R, N, K, x, w, Y, st, rm, ws, p3, norm);
  const Mfma2Shape sh = mfma2_shape(R, N, EPI == kEpiSwiGLU ? 2 * N : N, K, ws ? ws_bytes : 0, EPI == kEpiSwiGLU);
  switch (sh.mtw) {
    case 2: return mfma2_m<EPI, 2>(sh.ntw, R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
    case 4: return mfma2_m<EPI, 4>(sh.ntw, R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
    case 6: return mfma2_m<EPI, 6>(sh.ntw, R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
    default: return mfma2_m<EPI, 8>(sh.ntw, R, N, K, x, w, Y, st, rm, ws, ws_bytes, norm);
  }
}

// Skinny (weight streaming, X re-read per 16-feature tile) or MFMA tiles (X
// staged once per workgroup tile): measured at 9..64 rows on the 8B- and
// 1B-shaped projections, the MFMA kernel wins above 40 rows, above 12 rows
// for long reductions (K >= 8192) and the 128256-row LM heads, and above 24
// rows for projections of >= 16M weights.
bool use_mfma(int R, int Nw, int K) {
  if (R > 40) return true;
  if (R > 12 && (K >= 8192 || Nw >= 65536)) return true;
  return R > 24 && static_cast<double>(Nw) * K >= 16.0 * (1 << 20);
}

template <int EPI>
hipError_t dispatch(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                    hipStream_t st, const int32_t* rm, float* ws, size_t ws_bytes, GemmNorm* norm = nullptr) {
  if (dtype == 0) {
    const int ncols = (EPI == kEpiSwiGLU) ? 32 : 64;
    dim3 grid((N + ncols - 1) / ncols, (R + 63) / 64);
    gemm_f32<EPI><<<grid, 256, 0, st>>>(static_cast<const float*>(X), static_cast<const float*>(W),
                                        Y, R, N, K, rm);
    return hipGetLastError();
  }
  if (K % 128 != 0) return hipErrorInvalidValue;
  if (R <= kGemvRows) return gemv<EPI>(R, N, K, X, W, Y, st, rm, GemmFuse{});
  if (use_mfma(R, EPI == kEpiSwiGLU ? 2 * N : N, K)) return mfma2<EPI>(R, N, K, X, W, Y, st, rm, ws, ws_bytes, norm);
  if (R <= 16) return skinny<1, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 32) return skinny<2, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 48) return skinny<3, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 64) return skinny<4, EPI>(R, N, K, X, W, Y, st, rm);
  return mfma2<EPI>(R, N, K, X, W, Y, st, rm, ws, ws_bytes, norm);
}

}  // namespace

hipError_t launch_pack_weight(void* W, int rows, int K, int rot_rows, int hd, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  if (K <= 0 || K % 128 != 0 || rot_rows < 0 || rot_rows > rows) return hipErrorInvalidValue;
  if (rot_rows > 0 && (hd <= 0 || hd % 16 != 0 || hd > 256 || rot_rows % hd != 0)) return hipErrorInvalidValue;
  const int n_rot = rot_rows > 0 ? rot_rows / hd : 0;
  const int groups = n_rot + (rows - rot_rows + 15) / 16;
  const int G = std::max(16, rot_rows > 0 ? hd : 16);
  const size_t lds = static_cast<size_t>(G) * 16 * sizeof(u32x4);
  pack_weight_kernel<<<groups * (K / 128), 256, lds, st>>>(static_cast<bf16_t*>(W), rows, K, rot_rows, hd);
  return hipGetLastError();
}

size_t gemm_splitk_bytes(int R_max, int Nw_max) {
  // only grids of fewer than 192 tiles split, into S <= min(8, 256 / tiles)
  // parts; tiles >= R Nw / (256 * 256), so the partials S R Nw stay below
  // 256 * 256 * 256 floats (and below 8 R Nw)
  const double cap = std::min(8.0 * R_max * Nw_max, 256.0 * 256.0 * 256.0);
  return static_cast<size_t>(cap) * sizeof(float);
}

hipError_t launch_gemm_fused(int R, int N, int K, const void* X, const void* W, void* Y, int epi,
                             const GemmFuse& f, hipStream_t st, const int32_t* row_map) {
  if (R <= 0 || N <= 0) return hipSuccess;
  if (R > 16 || K % 128 != 0 || N % 16 != 0) return hipErrorInvalidValue;
  if (epi == kEpiQKVRope && (f.hd % 16 != 0 || N != (f.Hq + 2 * f.Hkv) * f.hd)) return hipErrorInvalidValue;
  if (R <= kGemvRows && !gemv_lm_skinny(R, N, K, epi)) {
    switch (epi) {
      case kEpiStoreF32: return gemv<kEpiStoreF32>(R, N, K, X, W, Y, st, row_map, f);
      case kEpiAddF32: return gemv<kEpiAddF32>(R, N, K, X, W, Y, st, nullptr, f);
      case kEpiSwiGLU: return gemv<kEpiSwiGLU>(R, N, K, X, W, Y, st, row_map, f);
      case kEpiQKVRope: return gemv<kEpiQKVRope>(R, N, K, X, W, Y, st, nullptr, f);
      default: return hipErrorInvalidValue;
    }
  }
  switch (epi) {
    case kEpiStoreF32: return skinny<1, kEpiStoreF32, true>(R, N, K, X, W, Y, st, row_map, f);
    case kEpiAddF32: return skinny<1, kEpiAddF32, true>(R, N, K, X, W, Y, st, nullptr, f);
    case kEpiSwiGLU: return skinny<1, kEpiSwiGLU, true>(R, N, K, X, W, Y, st, row_map, f);
    case kEpiQKVRope: return skinny<1, kEpiQKVRope, true>(R, N, K, X, W, Y, st, nullptr, f);
    default: return hipErrorInvalidValue;
  }
}

const char* gemm_kernel_name(int dtype, int R, int N, int K, int epi, bool fused, size_t splitk_bytes) {
  static const char* gv[4] = {"gemv_bf16<0, 2, false>", "gemv_bf16<1, 2, false>", "gemv_bf16<2, 2, false>",
                              "gemv_bf16<3, 2, false>"};
  if (dtype == 1 && R <= kGemvRows && !(fused && gemv_lm_skinny(R, N, K, epi)))
    return gemv_half(epi, N) ? "gemv_bf16<1, 2, true>" : ((epi >= 0 && epi <= 3) ? gv[epi] : "");
  // skinny names [MT - 1][epi][fused]
  static char names[4][4][2][40];
  static std::once_flag once;
  std::call_once(once, [] {
    for (int mt = 0; mt < 4; ++mt)
      for (int e = 0; e < 4; ++e)
        for (int f = 0; f < 2; ++f)
          snprintf(names[mt][e][f], sizeof(names[mt][e][f]), "gemm_skinny_bf16<%d, %d, %s>", mt + 1, e,
                   f ? "true" : "false");
  });
  if (epi < 0 || epi > 3) return "";
  if (fused) return names[0][epi][1];
  if (epi > 2) return "";
  static const char* f32[3] = {"gemm_f32<0>", "gemm_f32<1>", "gemm_f32<2>"};
  static char tiled[3][4][3][40];
  static std::once_flag once_t;
  std::call_once(once_t, [] {
    for (int e = 0; e < 3; ++e)
      for (int m = 0; m < 4; ++m)
        for (int n = 0; n < 3; ++n)
          snprintf(tiled[e][m][n], sizeof(tiled[e][m][n]), "gemm_mfma2_bf16<%d, %d, %d>", e, 2 * m + 2, 2 << n);
  });
  if (dtype == 0) return f32[epi];
  const int Nw = epi == kEpiSwiGLU ? 2 * N : N;
  if (use_mfma(R, Nw, K)) {
    static char m3[3][5][40];  // [epi][nb: 0 the 192-row form, 1, 2, 4]
    static std::once_flag once3;
    std::call_once(once3, [] {
      for (int e = 0; e < 3; ++e) {
        snprintf(m3[e][0], sizeof(m3[e][0]), "gemm_mfma3_bf16<%d, %d, %d, %d>", e, kM3MB, kM3NB, kM3D);
        for (int nb : {1, 2, 4})
          snprintf(m3[e][nb], sizeof(m3[e][nb]), "gemm_mfma3_bf16<%d, %d, %d, %d>", e, kM3sMB, nb, kM3D);
      }
    });
    Mfma3Plan p3;
    if (use_mfma3(R, Nw, K, epi, splitk_bytes, &p3)) return m3[epi][p3.nb];
    const Mfma2Shape sh = mfma2_shape(R, N, Nw, K, splitk_bytes, epi == kEpiSwiGLU);
    return tiled[epi][sh.mtw / 2 - 1][sh.ntw == 2 ? 0 : (sh.ntw == 4 ? 1 : 2)];
  }
  return names[(std::max(R, 1) - 1) / 16][epi][0];
}

hipError_t launch_gemm(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                       int epi, hipStream_t st, const int32_t* row_map, float* splitk_ws,
                       size_t splitk_bytes, GemmNorm* norm) {
  if (norm) {
    norm->done = false;
    norm->split = 0;
    norm->part = nullptr;
  }
  if (R <= 0 || N <= 0) return hipSuccess;
  switch (epi) {
    case kEpiStoreF32:
      return dispatch<kEpiStoreF32>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes,
                                    dtype == 1 ? norm : nullptr);
    case kEpiAddF32:
      return dispatch<kEpiAddF32>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes,
                                  dtype == 1 ? norm : nullptr);
    case kEpiSwiGLU:
      return dispatch<kEpiSwiGLU>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes);
  }
  return hipErrorInvalidValue;
}

}  // namespace spec
