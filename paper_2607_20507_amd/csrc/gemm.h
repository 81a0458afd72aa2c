// Decoder GEMMs: Y = X W^T with W [N, K] (reduction dim innermost): row-major
// for fp32, in the tiled layout of launch_pack_weight for bf16.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

enum GemmEpi {
  kEpiStoreF32 = 0,  // Y fp32 [R, N] = X W^T
  kEpiAddF32 = 1,    // Y fp32 [R, N] += X W^T (residual stream)
  kEpiSwiGLU = 2,    // W has 2N rows (gate then up); Y (element type) [R, N] = silu(g) * u
  kEpiQKVRope = 3    // fused path only: RoPE on q and k, q out, k and v into the paged cache
};

// Extras of the fused skinny GEMM (bf16, R <= 16), which folds the RMSNorm
// and the RoPE / KV append of the decoder into the GEMMs around them.
struct GemmFuse {
  // Consumer side of RMSNorm: X holds rows bf16(h (.) w) written by the
  // producer, and output row m is scaled by 1/sqrt(mean(h[m]^2) + eps), the
  // mean taken from `ss`, the producer's sums of squares per 8 columns
  // ([rows][K / 8]).  xrow (optional): X and ss row of output row m.
  const float* ss = nullptr;
  const int32_t* xrow = nullptr;
  float eps = 0.f;
  // Producer side (kEpiAddF32): with the new residual h also write
  // hb = bf16(h (.) wn) [R][N] and its sums of squares ss_out [R][N / 8].
  void* hb = nullptr;
  const void* wn = nullptr;
  float* ss_out = nullptr;
  // kEpiQKVRope: W is the [(Hq + 2 Hkv) hd, K] QKV projection; rotate-half
  // RoPE (angle pos[m] * theta^(-2i/hd), evaluated in fp64) on the q and k
  // heads; q to qout [R][Hq][hd], k and v to K [page][Hkv][16][hd] and
  // V^T [page][Hkv][hd][16] at slot[m] = page * 16 + offset.
  int Hq = 0, Hkv = 0, hd = 0;
  float theta = 0.f;
  const int32_t* pos = nullptr;
  const int32_t* slot = nullptr;
  void* qout = nullptr;
  void* kpool = nullptr;
  void* vpool = nullptr;
};

// Fused skinny GEMM (bf16, R <= 16, K % 128 == 0); epi as above.
hipError_t launch_gemm_fused(int R, int N, int K, const void* X, const void* W, void* Y, int epi,
                             const GemmFuse& f, hipStream_t st, const int32_t* row_map = nullptr);

// RMSNorm of the residual-add GEMM's updated rows (kEpiAddF32, bf16 model):
// y[m] = bf16(Y[m] / sqrt(mean(Y[m]^2) + eps) (.) w).  launch_gemm folds it
// into the split-K reduction when the launch splits K and sets `done`; the
// caller runs the separate RMSNorm otherwise.
struct GemmNorm {
  const void* w = nullptr;  // bf16 [N]
  float eps = 0.f;
  void* y = nullptr;        // bf16 [R][N]
  bool done = false;
  // kEpiStoreF32 (bf16, no row map): with defer set, a launch that splits K
  // leaves its partials [split][R][N] in the split-K workspace at `part`
  // for the consumer to sum (launch_rope_kv) and skips the reduction;
  // split = 0 when it did not split (Y then holds the output).
  bool defer = false;
  int split = 0;
  const float* part = nullptr;
};

// dtype: 0 = fp32 (X, W, SwiGLU output fp32), 1 = bf16 (X, W, SwiGLU output bf16).
// bf16 requires K % 128 == 0 (returns hipErrorInvalidValue otherwise).
// row_map (device, optional): output row m goes to Y row row_map[m].
// splitk_ws (device, optional): fp32 partials for split-K on small grids
// (R > 64); without it the kernel does not split K.
// norm (optional, kEpiAddF32 only): see GemmNorm.
hipError_t launch_gemm(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                       int epi, hipStream_t st, const int32_t* row_map = nullptr,
                       float* splitk_ws = nullptr, size_t splitk_bytes = 0, GemmNorm* norm = nullptr);

// In place: bf16 row-major [rows, K] -> the tiled layout every bf16 GEMM
// reads (K % 128 == 0).  In each complete group of 16 rows and 128-column
// block the 16 x 16 matrix of 16-byte chunks is transposed; a trailing group
// of fewer than 16 rows stays row-major.  rot_rows > 0 (the QKV weight's q
// and k heads, head dim hd, hd % 16 == 0): those rows are first reordered in
// each head to the rotary tile order, rows 8t..8t+7 then hd/2+8t..hd/2+8t+7
// forming tile t, so that GEMM output column 16 t + j is that row.
hipError_t launch_pack_weight(void* W, int rows, int K, int rot_rows, int hd, hipStream_t st);

// Bytes of split-K workspace that cover every launch shape.
size_t gemm_splitk_bytes(int R_max, int Nw_max);

// Profiler name of the kernel launch_gemm uses for (dtype, R, N, K, epi) with
// a split-K workspace of splitk_bytes, or launch_gemm_fused when fused.
const char* gemm_kernel_name(int dtype, int R, int N, int K, int epi, bool fused = false,
                             size_t splitk_bytes = 0);

}  // namespace spec
