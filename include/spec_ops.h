/*
 * spec_ops.h - single-kernel entry points of the verify step, for checking
 * each kernel on its own at full workload sizes.  Same conventions as spec.h:
 * "device" pointers are HIP device addresses, "host" pointers CPU memory,
 * stream is a hipStream_t as void*, errors are spec_status codes and the
 * caller owns every buffer.
 */
#ifndef SPEC_OPS_H_
#define SPEC_OPS_H_

#include "spec.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { SPEC_EPI_STORE_F32 = 0, SPEC_EPI_ADD_F32 = 1, SPEC_EPI_SWIGLU = 2 };

/* One bf16 weight [rows, K] (device) from row-major to the tiled layout, in
 * place (the per-matrix step of spec_pack_model; K % 128 == 0, else
 * SPEC_E_UNSUPPORTED).  rot_rows > 0 marks the first rot_rows rows as rotary
 * heads of head_dim rows (head_dim % 16 == 0, rot_rows % head_dim == 0),
 * reordered as wqkv's q and k heads are.  Asynchronous. */
SPEC_API spec_status spec_pack_weight(void* w, int32_t rows, int32_t K, int32_t rot_rows,
                                      int32_t head_dim, void* stream);

/* Decoder projection Y = X W^T (the QKV, O, gate/up, down and LM-head
 * products of the Llama layer).  X device [R, K] row-major, W device [N, K]
 * (SwiGLU: [2N, K], gate rows then up rows), element type dtype; fp32
 * accumulation.  fp32 W is row-major; bf16 W is in the tiled layout
 * (spec_pack_weight; for SwiGLU the gate and up halves packed separately).
 *   SPEC_EPI_STORE_F32: Y fp32 [R, N] = X W^T
 *   SPEC_EPI_ADD_F32:   Y fp32 [R, N] += X W^T   (residual add)
 *   SPEC_EPI_SWIGLU:    Y dtype [R, N] = silu(X Wg^T) * (X Wu^T)
 * bf16 needs K % 128 == 0 (else SPEC_E_UNSUPPORTED).  workspace (device,
 * optional, NULL allowed): fp32 split-K partials for R > 64 when the output
 * grid is small; size it with spec_op_gemm_workspace_bytes(R, N_w). */
SPEC_API size_t spec_op_gemm_workspace_bytes(int32_t R, int32_t Nw);
SPEC_API spec_status spec_op_gemm(int32_t dtype, int32_t R, int32_t N, int32_t K, const void* X,
                                  const void* W, void* Y, int32_t epilogue, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* RMSNorm: y[r] (dtype) = h[r] / sqrt(mean(h[r]^2) + eps) * w, h fp32 [R, d]. */
SPEC_API spec_status spec_op_rmsnorm(int32_t dtype, int32_t R, int32_t d, const float* h,
                                     const void* w, float eps, void* y, void* stream);

/* Rotary embedding + paged KV append for one layer.  qkv device fp32
 * [R, (Hq + 2 Hkv) hd]; pos and slot device int32 [R] (slot = page * 16 + offset);
 * q_out device [R, Hq, hd]; k_pages [pages][Hkv][16][hd]; v_pages [pages][Hkv][hd][16].
 * head_dim even and at most 256 (SPEC_E_INVALID otherwise). */
SPEC_API spec_status spec_op_rope_kv(int32_t dtype, int32_t R, int32_t n_heads, int32_t n_kv_heads,
                                     int32_t head_dim, float theta, const float* qkv,
                                     const int32_t* pos, const int32_t* slot, void* q_out,
                                     void* k_pages, void* v_pages, void* stream);

/* Paged causal attention of n_seqs row groups: group i has rows[i] query rows
 * (packed in order in q, device [sum rows, Hq, hd]) at positions pos0[i]..,
 * attending keys 0..position through page table row i of page_table (host
 * int32 [n_seqs, max_pages]).  out device [sum rows, Hq * hd], dtype.
 * workspace: device, >= spec_op_attention_workspace_bytes(...). */
SPEC_API size_t spec_op_attention_workspace_bytes(int32_t n_seqs, int32_t total_rows,
                                                  int32_t max_pages, int32_t n_kv_heads,
                                                  int32_t head_dim);
SPEC_API spec_status spec_op_attention(int32_t dtype, int32_t n_seqs, const int32_t* rows,
                                       const int32_t* pos0, const int32_t* page_table,
                                       int32_t max_pages, int32_t n_heads, int32_t n_kv_heads,
                                       int32_t head_dim, const void* q, const void* k_pages,
                                       const void* v_pages, void* out, void* workspace,
                                       size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SPEC_OPS_H_ */
