// Element order of one (page, kv head) block of the bf16 KV cache: 16 tokens
// x hd dims for K, and the same for V.  The order follows the MFMA operands
// of the attention kernel so that each operand load instruction reads whole
// 512-byte runs (two pages per instruction at most):
//  * K, token k of the page, dim d: 16-byte unit ((s * 2 + h) * 4 + g) * 8 + j
//    holds dims 8 c .. 8 c + 7 (c = d / 8, s = c / 4, g = c % 4) of token
//    k = 4 h + (j % 4) + 8 (j / 4), i.e. h = (k / 4) % 2, j = k % 4 + 4 (k / 8):
//    the key tile h of a 32-key chunk, step s, lane group g, row j (or j + 8
//    for the chunk's second page).
//  * V, token k, dim d: unit ((d / 16) * 2 + k / 8) * 16 + d % 16 holds tokens
//    8 (k / 8) .. + 7 of dim d (the V^T operand: 16 dims x 8 tokens per lane
//    group).
// The fp32 cache keeps the plain order: K [16][hd], V^T [hd][16].
#pragma once

namespace spec {

__host__ __device__ __forceinline__ int kv_k_off(int k, int d) {
  const int c = d >> 3, s = c >> 2, g = c & 3;
  const int h = (k >> 2) & 1, j = (k & 3) + 4 * (k >> 3);
  return ((((s * 2 + h) * 4 + g) * 8 + j) << 3) + (d & 7);
}

__host__ __device__ __forceinline__ int kv_v_off(int k, int d) {
  return (((((d >> 4) * 2 + (k >> 3)) * 16) + (d & 15)) << 3) + (k & 7);
}

}  // namespace spec
