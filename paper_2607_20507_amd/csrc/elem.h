// Embedding gather, RMSNorm, RoPE + paged KV append, KV slot clearing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

// h[r] = E[tok(r)] (fp32), tok(r) = tok_src[r] if >= 0 else tok_pool[-1 - tok_src[r]];
// the resolved ids are written to row_tok[r].  Optional (for the fused GEMMs'
// RMSNorm): hb[r] = h[r] (.) wn in the model dtype, and ss[r][j] = the sum of
// squares of h[r][8 j .. 8 j + 7] (d % 16 == 0).
hipError_t launch_embed(int dtype, int R, int d, const int32_t* tok_src, const int32_t* tok_pool,
                        const void* E, float* h, int32_t* row_tok, hipStream_t st, void* hb = nullptr,
                        const void* wn = nullptr, float* ss = nullptr);

// y[i] = h[src(i)] / sqrt(mean(h^2) + eps) * w, src(i) = row_idx ? row_idx[i] : i.
hipError_t launch_rmsnorm(int dtype, int R, int d, const float* h, const int32_t* row_idx,
                          const void* w, float eps, void* y, hipStream_t st);

// From qkv fp32 [R, (Hq + 2 Hkv) hd]: q <- RoPE(q) [R, Hq, hd]; K page slot
// slot[r] <- RoPE(k); V^T page slot <- v.  Rotate-half pairs (i, i + hd/2)
// at angle pos[r] * theta^(-2i/hd), angles and sin/cos evaluated in fp64.
// rot_tiled: the q and k head columns of qkv are in the rotary tile order of
// the tiled QKV weight (what the bf16 GEMMs produce from it): position
// 16 (i / 8) + i % 8 holds dim i, and the position 8 further holds dim
// i + hd / 2 (i < hd / 2); v columns are in plain order.  splits > 0: qkv
// holds that many split-K partials [splits][R][width] of the QKV GEMM (the
// deferred reduction of GemmNorm::defer), summed here in split order; the
// columns of one KV head group ((Hq / Hkv + 2) hd floats, hd % 4 == 0) are
// staged in LDS.  One workgroup per (row, KV head).
constexpr int kRopeSplitMaxWidth = 12288;
hipError_t launch_rope_kv(int dtype, int R, int Hq, int Hkv, int hd, float theta, const float* qkv,
                          const int32_t* pos, const int32_t* slot, void* q, void* kpool,
                          void* vpool, hipStream_t st, bool rot_tiled = false, int splits = 0);

// Zero the K and V entries of `n` flat slots (device list) in every layer of
// a pool whose layer l holds K at kv + l * layer_stride and V at + v_off
// (elements).
constexpr int kKvClearInline = 16;

struct KvClearJob {
  const int32_t* slots = nullptr;  // device list, or null: the first n of `inl`
  int32_t inl[kKvClearInline] = {};
  int n = 0;
  void* kv = nullptr;
  int n_layers = 0;
  size_t layer_stride = 0, v_off = 0;
  int Hkv = 0, hd = 0;
};

// Both jobs (the target's and the drafter's pool, same dtype) in one launch.
hipError_t launch_kv_clear(int dtype, const KvClearJob& a, const KvClearJob& b, hipStream_t st);

// Moves of K/V cache entries (tree verification: the accepted path's entries
// go to consecutive positions).  Group g holds the (src slot, dst slot) pairs
// pairs[2 off[g]] .. pairs[2 off[g + 1] - 1], applied in order: one sequence's
// moves may read a slot an earlier move of the group wrote, never one a later
// move writes.  Groups touch disjoint pages.
struct KvMoveJob {
  const int32_t* pairs = nullptr;  // device
  const int32_t* off = nullptr;    // device [n_groups + 1]
  int n_groups = 0;
  void* kv = nullptr;
  int n_layers = 0;
  size_t layer_stride = 0, v_off = 0;
  int Hkv = 0, hd = 0;
};
hipError_t launch_kv_move(int dtype, const KvMoveJob& j, hipStream_t st);

}  // namespace spec
