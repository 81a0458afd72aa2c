// Decoder GEMMs: Y = X W^T with W stored [N, K] (reduction dim innermost).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

enum GemmEpi {
  kEpiStoreF32 = 0,  // Y fp32 [R, N] = X W^T
  kEpiAddF32 = 1,    // Y fp32 [R, N] += X W^T (residual stream)
  kEpiSwiGLU = 2     // W has 2N rows (gate then up); Y (element type) [R, N] = silu(g) * u
};

// dtype: 0 = fp32 (X, W, SwiGLU output fp32), 1 = bf16 (X, W, SwiGLU output bf16).
// bf16 requires K % 128 == 0 (returns hipErrorInvalidValue otherwise).
// row_map (device, optional): output row m goes to Y row row_map[m].
// splitk_ws (device, optional): fp32 partials for split-K on small grids
// (R > 64); without it the kernel does not split K.
hipError_t launch_gemm(int dtype, int R, int N, int K, const void* X, const void* W, void* Y,
                       int epi, hipStream_t st, const int32_t* row_map = nullptr,
                       float* splitk_ws = nullptr, size_t splitk_bytes = 0);

// Bytes of split-K workspace that cover every launch shape.
size_t gemm_splitk_bytes(int R_max, int Nw_max);

// Profiler name of the kernel launch_gemm uses for (dtype, R, N, K, epi).
const char* gemm_kernel_name(int dtype, int R, int N, int K, int epi);

}  // namespace spec
