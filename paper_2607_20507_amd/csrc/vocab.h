// Vocabulary-wide decision pass: row statistics, the acceptance scan, the
// residual / bonus draw and the draft sampler (host-side launch interface).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "host_util.h"

namespace spec {

// One logits row of the decision pass: fp32 pointer and 1/T (0 for greedy).
struct VRow {
  const float* ptr;
  float inv_t;
  int32_t greedy;
};

// One sequence of the decision pass.  Rows are indices into the VRow table:
// target rows p_row .. p_row + k, draft rows q_row .. q_row + k - 1; draft
// tokens draft_tok[tok_row .. tok_row + k - 1].
struct VSeq {
  int32_t k;
  int32_t p_row;
  int32_t q_row;
  int32_t tok_row;
  int32_t base_pos;
  float t;
  uint32_t seq_lo, seq_hi;
};

// One row of the draft sampler: its logits, temperature, the absolute position
// of the token being drawn, the sequence id, where the token is written and
// an optional guide token (-1: none; see launch_draft_guide).
struct DRow {
  const float* ptr;
  float t;
  int32_t pos;
  uint32_t seq_lo, seq_hi;
  int32_t out;
  int32_t guide;
};

struct VocabPlan {
  int B = 0, n_rows = 0, V = 0;
  int chunk1 = 0, n_chunks1 = 0;  // statistics pass (n_chunks1 <= 64)
  int chunk2 = 0, n_chunks2 = 0;  // residual draw (n_chunks2 <= 64)
};

// Chunking follows chunk_rows (default n_rows): the two context-free entry
// points both chunk for B * (2 k_max + 1) rows, so that they compute the same
// partial sums whatever rows a call actually has.
VocabPlan vocab_plan(int B, int n_rows, int V, int chunk_rows = -1);
size_t vocab_ws_bytes(const VocabPlan& p);

// Full decision pass: statistics, one decision per sequence, the residual or
// bonus draw of sampled sequences, the merge of its chunk winners.  Outputs
// n_acc[B], out_tok[B * (kmax + 1)] (device).  d_seed (optional, device): read
// the Philox seed there instead of `seed`, so that a captured graph of the pass
// takes a new seed with each replay.  A sequence's rows must be 16-byte aligned
// when V % 4 == 0 (the vector path); `aligned` = false forces the scalar path.
// d_n_rows (optional, device): the rows that exist, when the tables were
// built on the device (launch_vocab_setup); grid rows beyond it exit at once.
// A sequence whose k is -1 is not decided: n_acc = -1 and tokens -1.
hipError_t launch_vocab_pass(const VocabPlan& p, const VRow* d_rows, const VSeq* d_seqs,
                             const int32_t* d_draft_tok, uint64_t seed, int kmax,
                             int32_t* d_n_acc, int32_t* d_out_tok, void* d_ws, hipStream_t st,
                             KernelTimer* timer = nullptr, const uint64_t* d_seed = nullptr,
                             bool aligned = true, const int32_t* d_n_rows = nullptr);

// Row and sequence tables of the decision pass built on the device from
// device arrays (B <= 256, one workgroup): sequence b's target rows are p
// rows sum_{c<b}(k_c + 1) .., its draft rows q rows sum_{c<b} k_c ...  If any
// k[b] is outside 0..kmax or any temperature is negative or NaN, no row is
// built and every sequence is marked undecided (k = -1).
constexpr int kSetupMaxSeqs = 256;
hipError_t launch_vocab_setup(int B, int kmax, const int32_t* d_k, const float* d_temp, const int64_t* d_ids,
                              const int32_t* d_base, const float* d_p, const float* d_q, int V, VRow* d_rows,
                              VSeq* d_seqs, int32_t* d_n_rows, hipStream_t st);

// Tree verification (multi-step speculative sampling over a tree of sampled
// candidates).  Node i of sequence b is nodes[node0 + i]; its parent is -1
// (the root: the pending token) or a node with a smaller index, and siblings
// are tried in index order.  p_row: the node's target row (its token is
// row_tok[p_row], the token that row was fed); q_row: the row its children
// were drawn from (-1: no children).  The root's rows are in the sequence
// record.  A chain of k drafts is the tree parents[i] = i - 1.
struct VTreeNode {
  int32_t parent, p_row, q_row, pad;
};
struct VTreeSeq {
  int32_t m, node0, p_row, q_row;
  int32_t base_pos;
  float t;
  uint32_t seq_lo, seq_hi;
};

// Statistics of every row (p and q), then the walk: at a node, children are
// accepted while v_j q(x) < r(x) fails, r becoming norm(max(0, r - q)) after
// each rejection; the walk ends with a draw from r (RESAMPLE noise) at a node
// whose children were all rejected, or from p (BONUS noise) at a leaf.  The
// residual masses of every node and level (max_kids levels: the most
// children of any node) and every node's draw are chip-wide passes before
// the walk.  Outputs n_acc[B] (accepted depth), out_tok[B * (kmax + 1)] (the
// path's tokens, then the drawn one, -1 after), out_path[B * kmax] (the
// accepted node indices, -1 after).  Workspace: tree_ws_bytes(p).
size_t tree_ws_bytes(const VocabPlan& p);
// Workspace that covers every plan of at most B sequences and n_rows rows
// (decision pass, tree pass) or n draft rows: for a workspace sized once for
// calls of varying size.
size_t vocab_ws_bound(int B, int n_rows);
size_t tree_ws_bound(int B, int n_rows);
size_t draft_ws_bound(int n);
hipError_t launch_tree_pass(const VocabPlan& p, const VRow* d_rows, const VTreeSeq* d_seqs,
                            const VTreeNode* d_nodes, const int32_t* d_row_tok, uint64_t seed,
                            const uint64_t* d_seed, int kmax, int max_kids,
                            int32_t* d_n_acc, int32_t* d_out_tok, int32_t* d_out_path, void* d_ws,
                            hipStream_t st, KernelTimer* timer = nullptr);

struct DraftPlan {
  int n = 0, V = 0, chunk = 0, n_chunks = 0;
};
DraftPlan draft_plan(int n, int V);
size_t draft_ws_bytes(const DraftPlan& p);
// Draft guidance (workload shaping, before launch_draft_sample): in each row
// with guide >= 0 the guide token's logit becomes the row maximum + boost, in
// place, so the stored row is the proposal the token is drawn from.
hipError_t launch_draft_guide(int n, int V, const DRow* d_rows, float boost, hipStream_t st);

hipError_t launch_draft_sample(const DraftPlan& p, const DRow* d_rows, uint64_t seed,
                               int32_t* d_tokens, void* d_ws, hipStream_t st,
                               const uint64_t* d_seed = nullptr);

hipError_t launch_philox_uniform(uint64_t seed, uint64_t seq_id, int32_t pos, int32_t purpose,
                                 int32_t n, float* out, hipStream_t st);

}  // namespace spec
