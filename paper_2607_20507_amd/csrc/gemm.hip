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
//  * skinny (R <= 64): weight streaming, HBM-bound.  A workgroup owns 16 output
//    features (gate+up pairs for SwiGLU); its waves split K and reduce through
//    LDS in a fixed order (deterministic, no atomics).  M is padded to 16 per
//    tile; MFMA throughput is ~10x what the weight stream needs.
//  * tiled (R > 64): 128x128 workgroup tiles, BK = 64, LDS double buffering
//    with an XOR swizzle of 16-byte chunks, 2x2 waves of 64x64.
//  * fp32 (the fp32 configuration): a plain LDS-tiled FMA kernel; no
//    reduced-precision arithmetic.

#include <algorithm>

#include "common.h"
#include "gemm.h"

namespace spec {
namespace {

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }

// ---------------------------------------------------------------------------
// skinny bf16

constexpr int kSkinnyMaxWaves = 8;

template <int MT, int EPI>
__global__ __launch_bounds__(kSkinnyMaxWaves * kWave) void gemm_skinny_bf16(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, void* __restrict__ Y, int R, int N,
    int K, int kb_per_wave, const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  constexpr int NACC = MT * (SW ? 2 : 1);
  __shared__ float red[kSkinnyMaxWaves * NACC * 256];

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  const int row = lane & 15, g = lane >> 4;
  const int n0 = blockIdx.x * 16;
  const int nrow = min(n0 + row, N - 1);
  // lane group g, step s carries k = 32 s + 8 g .. +7 of each 128-wide block:
  // the four lanes of a row read one contiguous 64-byte run per load
  const bf16_t* wg = W + static_cast<size_t>(nrow) * K + g * 8;
  const bf16_t* wu = SW ? W + static_cast<size_t>(N + nrow) * K + g * 8 : nullptr;
  const bf16_t* xr[MT];
  bool xv[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = mt * 16 + row;
    xv[mt] = m < R;
    xr[mt] = X + static_cast<size_t>(xv[mt] ? m : 0) * K + g * 8;
  }
  f32x4 acc[MT], accu[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    accu[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // KB 128-wide blocks per iteration, every load of the iteration issued
  // before its first MFMA (fewer blocks for larger M to bound registers)
  constexpr int KB = MT == 1 ? 4 : (MT == 2 ? 2 : 1);
  const int nb = K / 128;
  const int kb0 = wave * kb_per_wave;
  const int kb1 = min(nb, kb0 + kb_per_wave);
  for (int kb = kb0; kb < kb1; kb += KB) {
    uint4 w[KB][4], u[KB][4], x[KB][MT][4];
#pragma unroll
    for (int b = 0; b < KB; ++b) {
      const int ko = (kb + b < kb1 ? kb + b : kb) * 128;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        w[b][s] = ld_stream(reinterpret_cast<const uint4*>(wg + ko) + 4 * s);
        if (SW) u[b][s] = ld_stream(reinterpret_cast<const uint4*>(wu + ko) + 4 * s);
      }
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
        for (int mt = 0; mt < MT; ++mt) {
          acc[mt] = mfma16x16x32(x[b][mt][s], w[b][s], acc[mt]);
          if (SW) accu[mt] = mfma16x16x32(x[b][mt][s], u[b][s], accu[mt]);
        }
    }
  }
  // red[wave][a][r][lane]
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      red[((wave * NACC + mt) * 4 + r) * kWave + lane] = acc[mt][r];
      if (SW) red[((wave * NACC + MT + mt) * 4 + r) * kWave + lane] = accu[mt][r];
    }
  __syncthreads();
  for (int e = threadIdx.x; e < MT * 256; e += blockDim.x) {
    const int mt = e / 256, r = (e / kWave) & 3, ln = e & (kWave - 1);
    const int m = mt * 16 + 4 * (ln >> 4) + r;
    const int n = n0 + (ln & 15);
    float v = 0.f, vu = 0.f;
    for (int wv = 0; wv < nw; ++wv) {
      v += red[((wv * NACC + mt) * 4 + r) * kWave + ln];
      if (SW) vu += red[((wv * NACC + MT + mt) * 4 + r) * kWave + ln];
    }
    if (m < R && n < N) {
      const size_t o = static_cast<size_t>(row_map ? row_map[m] : m) * N + n;
      if (EPI == kEpiStoreF32) static_cast<float*>(Y)[o] = v;
      if (EPI == kEpiAddF32) static_cast<float*>(Y)[o] += v;
      if (EPI == kEpiSwiGLU) static_cast<bf16_t*>(Y)[o] = f32_to_bf16(silu(v) * vu);
    }
  }
}

// ---------------------------------------------------------------------------
// tiled bf16: BM = BN = 128, BK = 64, 256 threads (2x2 waves of 64x64)

constexpr int kTM = 128, kTN = 128, kTK = 64;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_tiled_bf16(const bf16_t* __restrict__ X,
                                                       const bf16_t* __restrict__ W,
                                                       void* __restrict__ Y, int R, int N, int K,
                                                       const int32_t* __restrict__ row_map) {
  constexpr bool SW = (EPI == kEpiSwiGLU);
  __shared__ uint4 As[2][kTM * 8];
  __shared__ uint4 Bs[2][kTN * 8];
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1), wave = t / kWave;
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 4, l16 = lane & 15;
  const int m0 = blockIdx.y * kTM;
  const int ncols = SW ? kTN / 2 : kTN;  // output features per tile
  const int f0 = blockIdx.x * ncols;

  // global source rows for the 4 chunks each thread stages per operand
  const uint4* asrc[4];
  const uint4* bsrc[4];
  bool av[4], bv[4];
  int lds_off[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int idx = t + 256 * i;
    const int r = idx >> 3, c = idx & 7;
    lds_off[i] = r * 8 + (c ^ (r & 7));
    const int m = m0 + r;
    av[i] = m < R;
    asrc[i] = reinterpret_cast<const uint4*>(X + static_cast<size_t>(av[i] ? m : 0) * K) + c;
    int wrow;
    if (SW) {
      const int f = f0 + (r & 63);
      bv[i] = f < N;
      wrow = (r < 64 ? 0 : N) + (bv[i] ? f : 0);
    } else {
      const int f = f0 + r;
      bv[i] = f < N;
      wrow = bv[i] ? f : 0;
    }
    bsrc[i] = reinterpret_cast<const uint4*>(W + static_cast<size_t>(wrow) * K) + c;
  }
  const uint4 zero = make_uint4(0, 0, 0, 0);
  uint4 ra[4], rb[4];
  auto gload = [&](int kt) {
    const int co = kt * (kTK / 8);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = av[i] ? asrc[i][co] : zero;
      rb[i] = bv[i] ? bsrc[i][co] : zero;
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      As[buf][lds_off[i]] = ra[i];
      Bs[buf][lds_off[i]] = rb[i];
    }
  };
  // B-tile row of the wave's n-subtile j
  auto brow = [&](int j) -> int {
    if (SW) return (j < 2) ? (32 * wn + 16 * j) : (64 + 32 * wn + 16 * (j - 2));
    return 64 * wn + 16 * j;
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = K / kTK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = 4 * ks + g;
      uint4 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 64 * wm + 16 * i + l16;
        a[i] = As[buf][r * 8 + (c ^ (r & 7))];
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = brow(j) + l16;
        b[j] = Bs[buf][r * 8 + (c ^ (r & 7))];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma16x16x32(a[i], b[j], acc[i][j]);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }
  // epilogue
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 64 * wm + 16 * i + 4 * g + r;
      if (m >= R) continue;
      const size_t mo = static_cast<size_t>(row_map ? row_map[m] : m);
      if (SW) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const int n = f0 + 32 * wn + 16 * j + l16;
          if (n < N)
            static_cast<bf16_t*>(Y)[mo * N + n] = f32_to_bf16(silu(acc[i][j][r]) * acc[i][j + 2][r]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = f0 + 64 * wn + 16 * j + l16;
          if (n >= N) continue;
          float* y = static_cast<float*>(Y) + mo * N + n;
          if (EPI == kEpiStoreF32) *y = acc[i][j][r];
          if (EPI == kEpiAddF32) *y += acc[i][j][r];
        }
      }
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

template <int MT, int EPI>
hipError_t skinny(int R, int N, int K, const void* X, const void* W, void* Y, hipStream_t st,
                  const int32_t* row_map) {
  const int tiles = (N + 15) / 16;
  const int nb = K / 128;
  // waves per workgroup split K: 8 when there are few feature tiles (and K is
  // not long enough to keep 4 waves busy), else 4 (measured at the verify and
  // draft shapes of the 8B/1B-shaped pair)
  int nw = (tiles <= 256 && K < 12288) ? 8 : 4;
  nw = std::max(1, std::min(nw, nb));
  const int kbpw = (nb + nw - 1) / nw;
  gemm_skinny_bf16<MT, EPI><<<tiles, nw * kWave, 0, st>>>(
      static_cast<const bf16_t*>(X), static_cast<const bf16_t*>(W), Y, R, N, K, kbpw, row_map);
  return hipGetLastError();
}

template <int EPI>
hipError_t dispatch(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                    hipStream_t st, const int32_t* rm) {
  if (dtype == 0) {
    const int ncols = (EPI == kEpiSwiGLU) ? 32 : 64;
    dim3 grid((N + ncols - 1) / ncols, (R + 63) / 64);
    gemm_f32<EPI><<<grid, 256, 0, st>>>(static_cast<const float*>(X), static_cast<const float*>(W),
                                        Y, R, N, K, rm);
    return hipGetLastError();
  }
  if (K % 128 != 0) return hipErrorInvalidValue;
  if (R <= 16) return skinny<1, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 32) return skinny<2, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 48) return skinny<3, EPI>(R, N, K, X, W, Y, st, rm);
  if (R <= 64) return skinny<4, EPI>(R, N, K, X, W, Y, st, rm);
  const int ncols = (EPI == kEpiSwiGLU) ? kTN / 2 : kTN;
  dim3 grid((N + ncols - 1) / ncols, (R + kTM - 1) / kTM);
  gemm_tiled_bf16<EPI><<<grid, 256, 0, st>>>(static_cast<const bf16_t*>(X),
                                             static_cast<const bf16_t*>(W), Y, R, N, K, rm);
  return hipGetLastError();
}

}  // namespace

const char* gemm_kernel_name(int dtype, int R, int epi) {
  static const char* f32[3] = {"gemm_f32<0>", "gemm_f32<1>", "gemm_f32<2>"};
  static const char* tiled[3] = {"gemm_tiled_bf16<0>", "gemm_tiled_bf16<1>", "gemm_tiled_bf16<2>"};
  static const char* skinny[4][3] = {
      {"gemm_skinny_bf16<1, 0>", "gemm_skinny_bf16<1, 1>", "gemm_skinny_bf16<1, 2>"},
      {"gemm_skinny_bf16<2, 0>", "gemm_skinny_bf16<2, 1>", "gemm_skinny_bf16<2, 2>"},
      {"gemm_skinny_bf16<3, 0>", "gemm_skinny_bf16<3, 1>", "gemm_skinny_bf16<3, 2>"},
      {"gemm_skinny_bf16<4, 0>", "gemm_skinny_bf16<4, 1>", "gemm_skinny_bf16<4, 2>"}};
  if (epi < 0 || epi > 2) return "";
  if (dtype == 0) return f32[epi];
  if (R <= 64) return skinny[(std::max(R, 1) - 1) / 16][epi];
  return tiled[epi];
}

hipError_t launch_gemm(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                       int epi, hipStream_t st, const int32_t* row_map) {
  if (R <= 0 || N <= 0) return hipSuccess;
  switch (epi) {
    case kEpiStoreF32: return dispatch<kEpiStoreF32>(dtype, R, N, K, X, W, Y, st, row_map);
    case kEpiAddF32: return dispatch<kEpiAddF32>(dtype, R, N, K, X, W, Y, st, row_map);
    case kEpiSwiGLU: return dispatch<kEpiSwiGLU>(dtype, R, N, K, X, W, Y, st, row_map);
  }
  return hipErrorInvalidValue;
}

}  // namespace spec
