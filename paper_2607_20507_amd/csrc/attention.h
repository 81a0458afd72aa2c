// Paged causal attention for verify / draft / prefill rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

// One unit of work: rows [row0, row0 + nrows) of one sequence (positions
// pos0.. consecutive) against keys [t0, t1) of that sequence, for all kv heads
// (grid.y).  part >= 0: write an unnormalised partial for a later combine;
// part < 0: write the normalised output.
struct AttnItem {
  int32_t row0, nrows, pos0, seq, t0, t1, part, pad;
};

// Split items of one (rows) group, combined into the output.
struct AttnGroup {
  int32_t row0, nrows, part0, nparts;
};

struct AttnArgs {
  int dtype;             // 0 fp32, 1 bf16 (q, pools, out)
  int Hq, Hkv, hd;
  const void* q;         // [R, Hq, hd]
  const void* kpool;     // layer K pages [P][Hkv][16][hd]
  const void* vpool;     // layer V pages, transposed [P][Hkv][hd][16]
  const int32_t* page_table;  // [seq slots][max_pages]
  int max_pages;
  void* out;             // [R, Hq * hd]
  float* part_o;         // [parts][Hkv][64][hd]
  float* part_ml;        // [parts][Hkv][64][2]
  // Tree verification (optional, per row): row r sees cache indices
  // 0..tree_base[r] and tree_base[r] + 1 + j for every bit j of
  // tree_mask[r] (its ancestors and itself in the draft tree) instead of
  // 0..its position.  Null: causal by position.
  const int32_t* tree_base = nullptr;
  const uint32_t* tree_mask = nullptr;
};

// bf16: items/groups as above, nt = 16-wide query-vector tiles per item
// (query vectors per item = nrows * Hq / Hkv <= 16 * nt, nt in {1, 2, 4}),
// w = waves per workgroup sharing an item's key range (1, 2, 4; at most 2
// for nt = 4).
hipError_t launch_attention_bf16(const AttnArgs& a, const AttnItem* d_items, int n_items,
                                 const AttnGroup* d_groups, int n_groups, int nt, int w, hipStream_t st);

// bf16 causal prefill: items from plan_attention's prefill form (blocks of
// 256 / G consecutive rows of one sequence against keys 0 .. t1 - 1, t0 = 0,
// part < 0), heaviest first; grid n_items x Hkv (kv head = block % Hkv).
hipError_t launch_attention_prefill_bf16(const AttnArgs& a, const AttnItem* d_items, int n_items, hipStream_t st);
const char* attn_prefill_kernel_name(int hd);

// fp32: one wave per (row, head); row r of sequence slot row_seq[r] at
// position row_pos[r] attends keys 0..row_pos[r] (or its tree keys).
hipError_t launch_attention_f32(const AttnArgs& a, int R, const int32_t* d_row_seq,
                                const int32_t* d_row_pos, hipStream_t st);

// Profiler name of the bf16 attention kernel for (hd, nt, w), the tree-masked
// variant with `tree`.
const char* attn_kernel_name(int hd, int nt, int w, bool tree = false);

}  // namespace spec
