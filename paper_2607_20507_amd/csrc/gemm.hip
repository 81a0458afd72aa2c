// Decoder GEMMs on gfx950: Y = X W^T, X [R, K], W [N, K] (both K-contiguous).
//
// bf16 paths use v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  Operand
// fragments: lane l supplies A[l % 16][kgroup(l / 16)] and B[kgroup(l / 16)][l % 16],
// and receives D[4 (l / 16) + r][l % 16], r = 0..3.  Because the reduction only
// needs A and B to agree on which k each (lane group, element) carries, each
// lane reads one contiguous 64-byte run of its X row and W row and feeds it to
// four consecutive MFMAs, so a W row's 256-byte block is read by four lanes
// with 16-byte loads straight from HBM.
//
//  * gemv (R <= 2): vector-FMA weight streaming with 256-byte row runs.
//  * skinny (R <= 64, except where use_mfma picks the MFMA kernel): weight
//    streaming, HBM-bound.  A workgroup owns 16 output
//    features (gate+up pairs for SwiGLU); its waves split K and reduce through
//    LDS in a fixed order (deterministic, no atomics).  M is padded to 16 per
//    tile; MFMA throughput is ~10x what the weight stream needs.
//  * mfma (R > 64): 128x256 workgroup tiles, BK = 32, two workgroups per CU,
//    loads two k-steps ahead, LDS double buffering with an XOR swizzle of
//    16-byte chunks, 4 waves of 64x128, XCD-aware tile order, split-K with a
//    fixed-order reduction when the grid is small.
//  * fp32 (the fp32 configuration): a plain LDS-tiled FMA kernel; no
//    reduced-precision arithmetic.

#include <algorithm>
#include <cstdio>
#include <mutex>

#include "common.h"
#include "gemm.h"

namespace spec {
namespace {

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }

// ---------------------------------------------------------------------------
// skinny bf16

constexpr int kSkinnyMaxWaves = 8;

// Tiles of the fused QKV epilogue: the q and k heads come first, each as
// hd / 16 tiles of 8 rotary pairs (i, i + hd / 2), so that a pair meets in one
// workgroup (lanes l and l ^ 8 of a 16-lane group); the v heads follow in
// plain order.
__device__ __forceinline__ int qkv_tile_row(const GemmFuse& f, int tile, int l16, int* head, int* dim) {
  const int per_head = f.hd / 16;
  *head = tile / per_head;
  const int i = 8 * (tile % per_head) + (l16 & 7);
  *dim = i + (l16 >> 3) * (f.hd / 2);
  return *head * f.hd + *dim;
}

// 1 / rms of each X row (R <= 16) from the producer's sums of squares per 16
// columns, into s_rs: 32 lanes per row, fixed order (strided sums, then a
// tree).  Run by the whole workgroup.
__device__ __forceinline__ void row_rscale(const GemmFuse& fu, int R, int K, float* s_rs) {
  const int np = K / 16;
  for (int base = 0; base < 16; base += blockDim.x / 32) {
    const int rr = base + static_cast<int>(threadIdx.x) / 32, sub = threadIdx.x & 31;
    float a = 0.f;
    if (rr < R) {
      const float* sp = fu.ss + static_cast<size_t>(fu.xrow ? fu.xrow[rr] : rr) * np;
      for (int p = sub; p < np; p += 32) a += sp[p];
    }
#pragma unroll
    for (int o = 16; o > 0; o >>= 1) a += __shfl_xor(a, o, kWave);
    if (sub == 0 && rr < 16) s_rs[rr] = 1.f / sqrtf(a / static_cast<float>(K) + fu.eps);
  }
}

// Epilogue of the fused GEMMs for output row m (< 16) and tile column l16 of
// 16-feature tile `tile`, given the (row-scaled) dot products v (and vu,
// the up rows of SwiGLU).  Run by whole waves: threads 0..255 with
// m = 4 (lane / 16) + r, so the 16 lanes of a group hold the 16 columns of a
// row and exchange values with shuffles.
template <int EPI>
__device__ __forceinline__ void fused_epilogue(const GemmFuse& fu, int m, int l16, int tile, int R, int N,
                                               float v, float vu, void* __restrict__ Y,
                                               const int32_t* __restrict__ row_map, int qk_tiles) {
  const int n0 = tile * 16;
  constexpr bool QKV = (EPI == kEpiQKVRope);
  const int n = n0 + l16;
  const bool ok = m < R && n < N;
  if (EPI == kEpiAddF32) {
    float hn = 0.f;
    if (ok) {
      float* y = static_cast<float*>(Y) + static_cast<size_t>(m) * N + n;
      hn = *y + v;
      *y = hn;
      if (fu.hb)
        static_cast<bf16_t*>(fu.hb)[static_cast<size_t>(m) * N + n] =
            f32_to_bf16(hn * bf16_to_f32(static_cast<const bf16_t*>(fu.wn)[n]));
    }
    if (fu.ss_out) {
      float sq = hn * hn;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) sq += __shfl_xor(sq, o, kWave);
      if (l16 == 0 && m < R && n0 < N) fu.ss_out[static_cast<size_t>(m) * (N / 16) + n0 / 16] = sq;
    }
  } else if (QKV) {
    const float partner = __shfl_xor(v, 8, kWave);
    if (m < R) {
      const int sl = fu.slot[m];
      const int page = sl >> 4, off = sl & 15;
      if (tile < qk_tiles) {
        int head, dim;
        qkv_tile_row(fu, tile, l16, &head, &dim);
        const int i = dim % (fu.hd / 2);
        double sn, cs;
        sincos(static_cast<double>(fu.pos[m]) * exp(-(2.0 * i / fu.hd) * log(static_cast<double>(fu.theta))),
               &sn, &cs);
        const float c = static_cast<float>(cs), sv = static_cast<float>(sn);
        // first half: a cos - b sin; second half: b cos + a sin (a, b = pair)
        const float o = (l16 < 8) ? v * c - partner * sv : v * c + partner * sv;
        if (head < fu.Hq)
          static_cast<bf16_t*>(fu.qout)[(static_cast<size_t>(m) * fu.Hq + head) * fu.hd + dim] = f32_to_bf16(o);
        else
          static_cast<bf16_t*>(fu.kpool)[((static_cast<size_t>(page) * fu.Hkv + (head - fu.Hq)) * 16 + off) * fu.hd + dim] =
              f32_to_bf16(o);
      } else if (n < N) {
        const int vi = n - (fu.Hq + fu.Hkv) * fu.hd;
        const int kh = vi / fu.hd, dd = vi % fu.hd;
        static_cast<bf16_t*>(fu.vpool)[((static_cast<size_t>(page) * fu.Hkv + kh) * fu.hd + dd) * 16 + off] =
            f32_to_bf16(v);
      }
    }
  } else if (ok) {
    const size_t o = static_cast<size_t>(row_map ? row_map[m] : m) * N + n;
    if (EPI == kEpiStoreF32) static_cast<float*>(Y)[o] = v;
    if (EPI == kEpiSwiGLU) static_cast<bf16_t*>(Y)[o] = f32_to_bf16(silu(v) * vu);
  }
}

template <int MT, int NT, int EPI, bool FUSE>
__global__ __launch_bounds__(kSkinnyMaxWaves * kWave) void gemm_skinny_bf16(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, void* __restrict__ Y, int R, int N,
    int K, int kb_per_wave, const int32_t* __restrict__ row_map, const GemmFuse fu) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr bool QKV = (EPI == kEpiQKVRope);
  constexpr int NS = SW ? 2 : 1;  // weight streams: gate and up rows for SwiGLU
  constexpr int NACC = MT * NT * NS;
  static_assert(!FUSE || MT == 1, "the fused path covers up to 16 rows");
  static_assert(FUSE || !QKV, "the QKV epilogue is fused only");
  extern __shared__ float red[];  // [waves][NACC][4][64]
  __shared__ float s_rs[16];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int row = lane & 15, g = lane >> 4;
  const int tile0 = blockIdx.x * NT;
  const int qk_tiles = QKV ? (fu.Hq + fu.Hkv) * fu.hd / 16 : 0;
  // lane group g, step s carries k = 32 s + 8 g .. +7 of each 128-wide block:
  // the four lanes of a row read one contiguous 64-byte run per load
  const bf16_t* wp[NT][NS];
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    int feat = (tile0 + j) * 16 + row;
    if (QKV && tile0 + j < qk_tiles) {
      int hh, dd;
      feat = qkv_tile_row(fu, tile0 + j, row, &hh, &dd);
    }
    const int nrow = min(feat, N - 1);
    wp[j][0] = W + static_cast<size_t>(nrow) * K + g * 8;
    if (SW) wp[j][NS - 1] = W + static_cast<size_t>(N + nrow) * K + g * 8;
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
  if (FUSE && fu.ss) row_rscale(fu, R, K, s_rs);
  f32x4 acc[MT][NT][NS];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int h = 0; h < NS; ++h) acc[mt][j][h] = f32x4{0.f, 0.f, 0.f, 0.f};
  // KB 128-wide blocks per iteration, every load of the iteration issued
  // before its first MFMA; each X fragment feeds NT x NS weight tiles
  constexpr int KB = (NT * NS * MT >= 4) ? 1 : ((NT * NS * MT >= 2) ? 2 : 4);
  const int nb = K / 128;
  const int kb0 = wave * kb_per_wave;
  const int kb1 = min(nb, kb0 + kb_per_wave);
  for (int kb = kb0; kb < kb1; kb += KB) {
    uint4 w[KB][NT][NS][4], x[KB][MT][4];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int ko = (kb + b < kb1 ? kb + b : kb) * 128;
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int h = 0; h < NS; ++h)
#pragma unroll
          for (int s = 0; s < 4; ++s) w[b][j][h][s] = ld_stream(reinterpret_cast<const uint4*>(wp[j][h] + ko) + 4 * s);
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
          for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int h = 0; h < NS; ++h) acc[mt][j][h] = mfma16x16x32(x[b][mt][s], w[b][j][h][s], acc[mt][j][h]);
    }
  }
  // red[wave][(mt, j, h)][r][lane]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int h = 0; h < NS; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          red[((wave * NACC + (mt * NT + j) * NS + h) * 4 + r) * kWave + lane] = acc[mt][j][h][r];
  __syncthreads();
  // element e: accumulator set e / 256 = (mt, j), output row m = 16 mt +
  // 4 (lane / 16) + r, column l16 of tile tile0 + j.  Whole waves take the
  // same (mt, j), as the fused epilogue's 16-lane exchanges need.
  for (int e = threadIdx.x; e < MT * NT * 256; e += blockDim.x) {
    const int set = e / 256, r = (e / kWave) & 3, ln = e & (kWave - 1);
    const int mt = set / NT, j = set % NT;
    const int m = mt * 16 + 4 * (ln >> 4) + r, l16 = ln & 15;
    float v = 0.f, vu = 0.f;
    for (int wv = 0; wv < nw; ++wv) {
      v += red[((wv * NACC + set * NS) * 4 + r) * kWave + ln];
      if (SW) vu += red[((wv * NACC + set * NS + 1) * 4 + r) * kWave + ln];
    }
    if (FUSE) {
      if (fu.ss) {
        const float rs = s_rs[m];
        v *= rs;
        vu *= rs;
      }
      fused_epilogue<EPI>(fu, m, l16, tile0 + j, R, N, v, vu, Y, row_map, qk_tiles);
      continue;
    }
    const int n = (tile0 + j) * 16 + l16;
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
// MFMA.  A workgroup owns 16 features (for SwiGLU their 16 gate and 16 up
// rows); each wave reads 4 weight rows, 16 lanes per row with 16-byte loads,
// so every load instruction covers 256 contiguous bytes of each of its rows
// (the MFMA operand layout can only give 64).  Waves split K in two halves
// (SwiGLU: gate and up instead); lanes of a row reduce with shuffles, halves
// through LDS, then the fused epilogue.

constexpr int kGemvRows = 2;  // measured: the MFMA skinny kernel wins from 3 rows on

__device__ __forceinline__ float dot8(const u32x4& w, const u32x4& x) {
  float a = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    a = fmaf(__uint_as_float(w[j] << 16), __uint_as_float(x[j] << 16), a);
    a = fmaf(__uint_as_float(w[j] & 0xFFFF0000u), __uint_as_float(x[j] & 0xFFFF0000u), a);
  }
  return a;
}

template <int EPI, int RM>
__global__ __launch_bounds__(512) void gemv_bf16(const bf16_t* __restrict__ X, const bf16_t* __restrict__ W,
                                                 void* __restrict__ Y, int R, int N, int K,
                                                 const int32_t* __restrict__ row_map, const GemmFuse fu) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr bool QKV = (EPI == kEpiQKVRope);
  constexpr int KB = 8;  // 128-wide chunks per batch: 8 weight loads in flight per lane
  __shared__ float part[2][RM][16];  // [K half or gate/up][row][tile column]
  __shared__ float s_rs[16];
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int c = lane & 15, trow = 4 * (wave & 3) + (lane >> 4);
  const int half = wave >> 2;  // K half, or (SwiGLU) 0 gate / 1 up
  const int n0 = blockIdx.x * 16;
  const int qk_tiles = QKV ? (fu.Hq + fu.Hkv) * fu.hd / 16 : 0;
  int feat = n0 + trow;
  if (QKV && static_cast<int>(blockIdx.x) < qk_tiles) {
    int hh, dd;
    feat = qkv_tile_row(fu, blockIdx.x, trow, &hh, &dd);
  }
  const int wrow = (SW && half ? N : 0) + min(feat, N - 1);
  const bf16_t* wp = W + static_cast<size_t>(wrow) * K + c * 8;
  const bf16_t* xp[RM];
#pragma unroll
  for (int m = 0; m < RM; ++m)
    xp[m] = X + static_cast<size_t>(m < R ? (fu.xrow ? fu.xrow[m] : m) : 0) * K + c * 8;
  const int chunks = K / 128;
  const int per = SW ? chunks : (chunks + 1) / 2;
  const int c0 = SW ? 0 : half * per, c1 = min(chunks, c0 + per);
  float a[RM];
#pragma unroll
  for (int m = 0; m < RM; ++m) a[m] = 0.f;
  for (int ch = c0; ch < c1; ch += KB) {
    u32x4 w[KB], x[KB][RM];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int o = min(ch + b, c1 - 1) * 128;
      w[b] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wp + o));
#pragma unroll
      for (int m = 0; m < RM; ++m)
        if (m < R) x[b][m] = *reinterpret_cast<const u32x4*>(xp[m] + o);
    }
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      if (ch + b >= c1) break;
#pragma unroll
      for (int m = 0; m < RM; ++m)
        if (m < R) a[m] += dot8(w[b], x[b][m]);
    }
  }
#pragma unroll
  for (int m = 0; m < RM; ++m) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) a[m] += __shfl_xor(a[m], o, kWave);
    if (c == 0) part[half][m][trow] = a[m];
  }
  if (fu.ss) row_rscale(fu, R, K, s_rs);
  __syncthreads();
  if (threadIdx.x >= 256) return;
  const int e = threadIdx.x, r = (e / kWave) & 3, ln = e & (kWave - 1);
  const int m = 4 * (ln >> 4) + r, l16 = ln & 15;
  float v = 0.f, vu = 0.f;
  if (m < R) {
    v = SW ? part[0][m][l16] : part[0][m][l16] + part[1][m][l16];
    if (SW) vu = part[1][m][l16];
    if (fu.ss) {
      v *= s_rs[m];
      vu *= s_rs[m];
    }
  }
  fused_epilogue<EPI>(fu, m, l16, blockIdx.x, R, N, v, vu, Y, row_map, qk_tiles);
}

template <int EPI>
hipError_t gemv(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                const int32_t* row_map, const GemmFuse& fu) {
  const dim3 grid((N + 15) / 16);
  const bf16_t* x = static_cast<const bf16_t*>(X);
  const bf16_t* w = static_cast<const bf16_t*>(W);
  if (R > kGemvRows) return hipErrorInvalidValue;
  gemv_bf16<EPI, kGemvRows><<<grid, 512, 0, st>>>(x, w, Y, R, N, K, row_map, fu);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// MFMA bf16 for R > 64: 128 x 256 workgroup tile (256 W rows; 128 gate + 128
// up rows for SwiGLU), BK = 32, 4 waves of 64 x 128.  Two workgroups share a
// CU (48 KB of LDS and at most 256 registers per lane each), so one
// workgroup's MFMAs cover the other's barrier and load waits.  Global loads
// run two k-steps ahead through two register staging sets: tile kt+2 is in
// flight while tile kt is multiplied and tile kt+1 waits to be stored into the
// LDS double buffer (XOR-swizzled 16-byte chunks, one barrier per k-step).
// The 1-D grid is decoded XCD-aware: workgroups are dispatched round-robin
// over the 8 XCDs, so consecutive tile ids are mapped to one XCD, and the row
// tiles of a column tile are consecutive, sharing that XCD's L2 for the W tile.
// Split-K writes raw fp32 partials by W row; a reduction pass applies the
// epilogue in a fixed order.

constexpr int kMM = 128, kMN = 256, kMK = 32;
constexpr int kMCh = kMK / 8;           // 16-byte chunks per tile row per k-step
constexpr int kMRows = 256 / kMCh;      // tile rows one staging pass covers
constexpr int kMPA = kMM / kMRows, kMPB = kMN / kMRows;

template <int EPI>
__global__ __launch_bounds__(256, 2) void gemm_mfma_bf16(const bf16_t* __restrict__ X,
                                                         const bf16_t* __restrict__ W,
                                                         void* __restrict__ Y, float* __restrict__ part,
                                                         int R, int N, int K, int k_len, int MT, int NT,
                                                         const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  __shared__ u32x4 As[2][kMM * kMCh];
  __shared__ u32x4 Bs[2][kMN * kMCh];
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1), wave = t / kWave;
  const int wm = wave & 1, wn = wave >> 1;
  const int g = lane >> 4, l16 = lane & 15;
  const int total = gridDim.x, nid = blockIdx.x;
  const int xcd = nid & 7, slot = nid >> 3, per = total >> 3, rem = total & 7;
  const int tix = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
  const int mt = tix % MT, rest = tix / MT, sp = rest / NT, nt = rest % NT;
  const int m0 = mt * kMM;
  const int f0 = nt * (SW ? kMN / 2 : kMN);
  const int kbeg = sp * k_len;
  const int nk = (min(K, kbeg + k_len) - kbeg) / kMK;  // even: k_len and K - kbeg are multiples of 64

  // staging: thread t moves chunk t % kMCh of tile rows t / kMCh + kMRows i.
  // Rows past R or N are clamped to the last valid row: read, never written back.
  const int sr = t / kMCh, sc = t % kMCh;
  const int lds_st = sr * kMCh + (sc ^ (sr & (kMCh - 1)));
  const bf16_t* xs = X + kbeg + sc * 8;
  const bf16_t* ws = W + kbeg + sc * 8;
  uint32_t aoff[kMPA], boff[kMPB];
#pragma unroll
  for (int i = 0; i < kMPA; ++i) aoff[i] = static_cast<uint32_t>(min(m0 + sr + kMRows * i, R - 1));
#pragma unroll
  for (int i = 0; i < kMPB; ++i) {
    const int br = sr + kMRows * i;
    if (SW)
      boff[i] = static_cast<uint32_t>((br < 128 ? 0 : N) + min(f0 + (br & 127), N - 1));
    else
      boff[i] = static_cast<uint32_t>(min(f0 + br, N - 1));
  }
  // native vector types keep the staging values in registers
  u32x4 sa[kMPA], sb[kMPB], ta[kMPA], tb[kMPB];
#define SPEC_MFMA_LOAD(SA, SB, KT)                                                                 \
  do {                                                                                             \
    const int ko_ = (KT) * kMK;                                                                    \
    _Pragma("unroll") for (int i = 0; i < kMPA; ++i)                                               \
        SA[i] = *reinterpret_cast<const u32x4*>(xs + static_cast<size_t>(aoff[i]) * K + ko_);      \
    _Pragma("unroll") for (int i = 0; i < kMPB; ++i)                                               \
        SB[i] = *reinterpret_cast<const u32x4*>(ws + static_cast<size_t>(boff[i]) * K + ko_);      \
  } while (0)
#define SPEC_MFMA_STORE(SA, SB, AL, BL)                                                            \
  do {                                                                                             \
    _Pragma("unroll") for (int i = 0; i < kMPA; ++i) AL[lds_st + 256 * i] = SA[i];                 \
    _Pragma("unroll") for (int i = 0; i < kMPB; ++i) BL[lds_st + 256 * i] = SB[i];                 \
  } while (0)

  f32x4 acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int c = g ^ (l16 & (kMCh - 1));  // chunk of k-group g in a fragment row
#define SPEC_MFMA_COMPUTE(AL, BL)                                                                  \
  {                                                                                                \
    u32x4 a[4], b[8];                                                                              \
    _Pragma("unroll") for (int i = 0; i < 4; ++i) a[i] = AL[(64 * wm + 16 * i + l16) * kMCh + c];  \
    _Pragma("unroll") for (int j = 0; j < 8; ++j) {                                                \
      const int r = SW ? ((j < 4) ? (64 * wn + 16 * j) : (128 + 64 * wn + 16 * (j - 4)))           \
                       : (128 * wn + 16 * j);                                                      \
      b[j] = BL[(r + l16) * kMCh + c];                                                             \
    }                                                                                              \
    _Pragma("unroll") for (int i = 0; i < 4; ++i)                                                  \
        _Pragma("unroll") for (int j = 0; j < 8; ++j) acc[i][j] = mfma16x16x32v(a[i], b[j], acc[i][j]); \
  }

  // prefetches past the end are clamped, in-bounds reloads; the scheduling
  // barriers keep each k-step's loads ahead of its MFMAs
  if (nk > 0) {
    SPEC_MFMA_LOAD(sa, sb, 0);
    SPEC_MFMA_STORE(sa, sb, As[0], Bs[0]);
    SPEC_MFMA_LOAD(ta, tb, min(1, nk - 1));
  }
  __syncthreads();
  for (int kt = 0; kt < nk; kt += 2) {
    SPEC_MFMA_LOAD(sa, sb, min(kt + 2, nk - 1));
    __builtin_amdgcn_sched_barrier(0);
    SPEC_MFMA_COMPUTE(As[0], Bs[0]);
    SPEC_MFMA_STORE(ta, tb, As[1], Bs[1]);
    __syncthreads();
    SPEC_MFMA_LOAD(ta, tb, min(kt + 3, nk - 1));
    __builtin_amdgcn_sched_barrier(0);
    SPEC_MFMA_COMPUTE(As[1], Bs[1]);
    SPEC_MFMA_STORE(sa, sb, As[0], Bs[0]);
    __syncthreads();
  }
#undef SPEC_MFMA_COMPUTE
#undef SPEC_MFMA_STORE
#undef SPEC_MFMA_LOAD

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 64 * wm + 16 * i + 4 * g + r;
      if (m >= R) continue;
      if (part) {
        float* pr = part + (static_cast<size_t>(sp) * R + m) * (SW ? 2 * N : N);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          int n, wrow;
          if (SW) {
            n = f0 + 64 * wn + 16 * (j & 3) + l16;
            wrow = (j < 4 ? 0 : N) + n;
          } else {
            n = f0 + 128 * wn + 16 * j + l16;
            wrow = n;
          }
          if (n < N) pr[wrow] = acc[i][j][r];
        }
        continue;
      }
      const size_t mo = static_cast<size_t>(row_map ? row_map[m] : m);
      if (SW) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = f0 + 64 * wn + 16 * j + l16;
          if (n < N)
            static_cast<bf16_t*>(Y)[mo * N + n] = f32_to_bf16(silu(acc[i][j][r]) * acc[i][j + 4][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int n = f0 + 128 * wn + 16 * j + l16;
          if (n >= N) continue;
          float* y = static_cast<float*>(Y) + mo * N + n;
          if (EPI == kEpiStoreF32) *y = acc[i][j][r];
          if (EPI == kEpiAddF32) *y += acc[i][j][r];
        }
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

template <int MT, int NT, int EPI, bool FUSE>
hipError_t skinny_nt(int nw, int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                     const int32_t* row_map, const GemmFuse& fu) {
  constexpr int NACC = MT * NT * (EPI == kEpiSwiGLU ? 2 : 1);
  const int groups = ((N + 15) / 16 + NT - 1) / NT;
  const int nb = K / 128;
  nw = std::max(FUSE ? 4 : 1, std::min(nw, nb));
  if (FUSE && nw < 4) return hipErrorInvalidValue;  // the fused epilogue needs 256 threads
  const int kbpw = (nb + nw - 1) / nw;
  const size_t lds = static_cast<size_t>(nw) * NACC * 256 * sizeof(float);
  gemm_skinny_bf16<MT, NT, EPI, FUSE><<<groups, nw * kWave, lds, st>>>(
      static_cast<const bf16_t*>(X), static_cast<const bf16_t*>(W), Y, R, N, K, kbpw, row_map, fu);
  return hipGetLastError();
}

// Feature tiles per workgroup and waves per workgroup of the skinny kernel,
// measured at 6..64 rows on the projections of the 8B/1B-shaped pair: several
// tiles per workgroup share each X fragment load (the L2 traffic of X limits
// the wide LM head and gate/up), but cost parallelism on narrow projections;
// 8 waves split K when there are few workgroups and K is mid-sized.
int skinny_tiles_per_wg(int MT, int N, bool sw) {
  const int tiles = (N + 15) / 16;
  int nt = sw ? (tiles >= 768 ? 4 : 1) : (tiles >= 2048 ? 4 : (tiles >= 384 ? 2 : 1));
  while (nt > 1 && MT * nt * (sw ? 2 : 1) > 8) nt /= 2;  // bounds registers
  return nt;
}

int skinny_waves(int groups, int K) { return (groups <= 256 && K >= 4096 && K < 12288) ? 8 : 4; }

template <int MT, int EPI, bool FUSE = false>
hipError_t skinny(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                  const int32_t* row_map, const GemmFuse& fu = GemmFuse{}) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  const int nt = skinny_tiles_per_wg(MT, N, SW);
  const int nw = skinny_waves(((N + 15) / 16 + nt - 1) / nt, K);
  if (nt == 4 && MT * 4 * (SW ? 2 : 1) <= 8)
    return skinny_nt<MT, (MT * 4 * (SW ? 2 : 1) <= 8 ? 4 : 1), EPI, FUSE>(nw, R, N, K, X, W, Y, st, row_map, fu);
  if (nt == 2 && MT * 2 * (SW ? 2 : 1) <= 8)
    return skinny_nt<MT, (MT * 2 * (SW ? 2 : 1) <= 8 ? 2 : 1), EPI, FUSE>(nw, R, N, K, X, W, Y, st, row_map, fu);
  return skinny_nt<MT, 1, EPI, FUSE>(nw, R, N, K, X, W, Y, st, row_map, fu);
}

// Split-K factor for the MFMA kernel: grids under 256 tiles are split so that
// tiles x splits stays within one wave of the 256 CUs (measured at the
// 364-row verify shapes: more splits lose to the partials' traffic and to
// short k-loops), k-splits multiples of 64, partials within the workspace.
template <int EPI>
int mfma_splits(int R, int N, int K, size_t ws_bytes, int* k_len) {
  const int Nw = (EPI == kEpiSwiGLU) ? 2 * N : N;
  const int tiles = ((Nw + kMN - 1) / kMN) * ((R + kMM - 1) / kMM);
  int S = 1;
  if (ws_bytes && tiles < 256) {
    S = std::max(1, std::min(8, 256 / tiles));
    while (S > 1 && static_cast<size_t>(S) * R * Nw * sizeof(float) > ws_bytes) --S;
  }
  *k_len = ((K + S - 1) / S + 2 * kMK - 1) / (2 * kMK) * (2 * kMK);
  return (K + *k_len - 1) / *k_len;
}

template <int EPI>
hipError_t mfma(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                const int32_t* rm, float* ws, size_t ws_bytes) {
  int k_len = K;
  const int S = mfma_splits<EPI>(R, N, K, ws ? ws_bytes : 0, &k_len);
  const int Nw = (EPI == kEpiSwiGLU) ? 2 * N : N;
  const int MT = (R + kMM - 1) / kMM, NT = (Nw + kMN - 1) / kMN;
  const int grid = MT * NT * S;
  const bf16_t* x = static_cast<const bf16_t*>(X);
  const bf16_t* w = static_cast<const bf16_t*>(W);
  if (S <= 1) {
    gemm_mfma_bf16<EPI><<<grid, 256, 0, st>>>(x, w, Y, nullptr, R, N, K, K, MT, NT, rm);
    return hipGetLastError();
  }
  gemm_mfma_bf16<EPI><<<grid, 256, 0, st>>>(x, w, nullptr, ws, R, N, K, k_len, MT, NT, rm);
  const size_t total = static_cast<size_t>(R) * N;
  const int blocks = static_cast<int>(std::min<size_t>(2048, (total + 255) / 256));
  splitk_reduce<EPI><<<blocks, 256, 0, st>>>(ws, S, R, N, Y, rm);
  return hipGetLastError();
}

// Skinny (weight streaming, X re-read per workgroup) or MFMA tiles (X staged
// once per 128 rows): measured at 8..64 rows on the 1B-shaped projections, the
// MFMA kernel wins for the 128256-row LM head above 8 rows and for the large
// projections (>= 16M weights) above 40 rows.
bool use_mfma(int R, int Nw, int K) {
  if (R > 64) return true;
  if (R > 8 && Nw >= 65536) return true;
  return R > 40 && static_cast<double>(Nw) * K >= 16.0 * (1 << 20);
}

template <int EPI>
hipError_t dispatch(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                    hipStream_t st, const int32_t* rm, float* ws, size_t ws_bytes) {
  if (dtype == 0) {
    const int ncols = (EPI == kEpiSwiGLU) ? 32 : 64;
    dim3 grid((N + ncols - 1) / ncols, (R + 63) / 64);
    gemm_f32<EPI><<<grid, 256, 0, st>>>(static_cast<const float*>(X), static_cast<const float*>(W),
                                        Y, R, N, K, rm);
    return hipGetLastError();
  }
  if (K % 128 != 0) return hipErrorInvalidValue;
  if (R <= kGemvRows) return gemv<EPI>(R, N, K, X, W, Y, st, rm, GemmFuse{});
  if (use_mfma(R, EPI == kEpiSwiGLU ? 2 * N : N, K)) return mfma<EPI>(R, N, K, X, W, Y, st, rm, ws, ws_bytes);
  if (R <= 16) return skinny<1, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 32) return skinny<2, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 48) return skinny<3, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 64) return skinny<4, EPI>(R, N, K, X, W, Y, st, rm);
  return mfma<EPI>(R, N, K, X, W, Y, st, rm, ws, ws_bytes);
}

}  // namespace

size_t gemm_splitk_bytes(int R_max, int Nw_max) {
  // only grids of fewer than 256 tiles split, into S <= 256 / tiles parts, so
  // the partials S * R * Nw stay below 256 * kMM * kMN floats; smaller
  // problems need less
  const size_t tiles = static_cast<size_t>((Nw_max + kMN - 1) / kMN) * ((R_max + kMM - 1) / kMM);
  return std::min<size_t>(256, 8 * tiles) * kMM * kMN * sizeof(float);
}

hipError_t launch_gemm_fused(int R, int N, int K, const void* X, const void* W, void* Y, int epi,
                             const GemmFuse& f, hipStream_t st, const int32_t* row_map) {
  if (R <= 0 || N <= 0) return hipSuccess;
  if (R > 16 || K % 128 != 0 || N % 16 != 0) return hipErrorInvalidValue;
  if (epi == kEpiQKVRope && (f.hd % 16 != 0 || N != (f.Hq + 2 * f.Hkv) * f.hd)) return hipErrorInvalidValue;
  if (R <= kGemvRows) {
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

const char* gemm_kernel_name(int dtype, int R, int N, int K, int epi, bool fused) {
  static const char* gv[4] = {"gemv_bf16<0, 2>", "gemv_bf16<1, 2>", "gemv_bf16<2, 2>", "gemv_bf16<3, 2>"};
  if (dtype == 1 && R <= kGemvRows) return (epi >= 0 && epi <= 3) ? gv[epi] : "";
  // skinny names [MT - 1][log2 NT][epi][fused]
  static char names[4][3][4][2][48];
  static std::once_flag once;
  std::call_once(once, [] {
    for (int mt = 0; mt < 4; ++mt)
      for (int t = 0; t < 3; ++t)
        for (int e = 0; e < 4; ++e)
          for (int f = 0; f < 2; ++f)
            snprintf(names[mt][t][e][f], sizeof(names[mt][t][e][f]), "gemm_skinny_bf16<%d, %d, %d, %s>", mt + 1,
                     1 << t, e, f ? "true" : "false");
  });
  auto skinny_name = [&](int MT, bool f) {
    const int nt = skinny_tiles_per_wg(MT, N, epi == kEpiSwiGLU);
    return names[MT - 1][nt == 4 ? 2 : (nt == 2 ? 1 : 0)][epi][f ? 1 : 0];
  };
  if (epi < 0 || epi > 3) return "";
  if (fused) return skinny_name(1, true);
  if (epi > 2) return "";
  static const char* f32[3] = {"gemm_f32<0>", "gemm_f32<1>", "gemm_f32<2>"};
  static const char* tiled[3] = {"gemm_mfma_bf16<0>", "gemm_mfma_bf16<1>", "gemm_mfma_bf16<2>"};
  if (dtype == 0) return f32[epi];
  if (use_mfma(R, epi == kEpiSwiGLU ? 2 * N : N, K)) return tiled[epi];
  return skinny_name((std::max(R, 1) - 1) / 16 + 1, false);
}

hipError_t launch_gemm(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                       int epi, hipStream_t st, const int32_t* row_map, float* splitk_ws,
                       size_t splitk_bytes) {
  if (R <= 0 || N <= 0) return hipSuccess;
  switch (epi) {
    case kEpiStoreF32:
      return dispatch<kEpiStoreF32>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes);
    case kEpiAddF32:
      return dispatch<kEpiAddF32>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes);
    case kEpiSwiGLU:
      return dispatch<kEpiSwiGLU>(dtype, R, N, K, X, W, Y, st, row_map, splitk_ws, splitk_bytes);
  }
  return hipErrorInvalidValue;
}

}  // namespace spec
