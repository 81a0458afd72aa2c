/*
 * spec.h - C ABI of the speculative-decoding verify step on MI355X (gfx950).
 *
 * The operation is the draft-and-verify generation of CacheSpec (Section 3.4,
 * "Cache-Miss Branch"; Section 2, speculative-decoding paragraph): a small
 * draft model proposes k tokens, the target model scores all of them in one
 * batched forward pass, and speculative sampling accepts each draft x~_j with
 * probability min(1, p_j(x~_j) / q_j(x~_j)); at the first rejection one token
 * is drawn from norm(max(0, p_j - q_j)) instead, and if all k are accepted a
 * bonus token is drawn from p_{k+1}.  Temperature 0 is greedy: drafts are
 * accepted while they equal the target's argmax.
 *
 * Conventions
 *  - Every pointer documented "device" is a HIP device address; "host" is CPU
 *    memory.  Sizes are element counts unless stated.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *    calls enqueue work on it and return without waiting, except where a call
 *    says it blocks.
 *  - Ownership: the caller owns every device buffer it passes (weights, KV
 *    pools, workspace, inputs, outputs) and keeps them alive for as long as a
 *    context that refers to them exists.  The library never frees them.  The
 *    library owns the context, its host metadata, pinned staging memory and
 *    events.
 *  - Errors are returned as spec_status; no exception crosses the ABI.  On any
 *    error other than SPEC_E_HIP the context's state is unchanged (page
 *    exhaustion is detected before anything is enqueued).  SPEC_E_HIP is
 *    sticky: destroy the context.  spec_last_error() explains the last failure.
 *  - A context is not thread-safe.
 *
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11) keyed by the 64-bit
 * `seed`; the counter is (block, position, seq_id bits 0..31, seq_id bits
 * 32..55 << 8 | purpose) with purpose DRAFT=0, ACCEPT=1, RESAMPLE=2, BONUS=3.
 * A uniform is ((word >> 9) + 0.5) * 2^-23; vocabulary noise for token i is
 * word i & 3 of block i >> 2.  Because noise is keyed by the caller's stable
 * seq_id and the absolute position of the token being decided, results do not
 * depend on batch composition or on the order of sequences in a call.
 */
#ifndef SPEC_H_
#define SPEC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEC_API __attribute__((visibility("default")))

typedef int32_t spec_status;
enum {
  SPEC_OK = 0,
  SPEC_E_INVALID = 1,     /* bad argument (null pointer, size out of range, unknown seq) */
  SPEC_E_NOPAGES = 2,     /* a KV page pool is exhausted; nothing was changed */
  SPEC_E_HIP = 3,         /* a HIP runtime call failed; the context is unusable */
  SPEC_E_STATE = 4,       /* call out of order (verify twice, commit without verify, ...) */
  SPEC_E_UNSUPPORTED = 5  /* valid but unsupported shape (e.g. head_dim not 64/128) */
};

enum { SPEC_F32 = 0, SPEC_BF16 = 1 };
enum { SPEC_LAYOUT_ROWMAJOR = 0, SPEC_LAYOUT_TILED = 1 };
enum { SPEC_DRAFT = 0, SPEC_ACCEPT = 1, SPEC_RESAMPLE = 2, SPEC_BONUS = 3 };

/* One decoder layer's weights (device pointers, element type = model dtype,
 * reduction dimension innermost; the projections wqkv, wo, w_gate_up and
 * w_down are row-major for fp32 models and in the tiled layout of
 * spec_pack_model for bf16 models, the norms are plain vectors):
 *   attn_norm, mlp_norm  [d]
 *   wqkv       [(Hq + 2*Hkv) * hd, d]   rows: q heads, then k heads, then v heads
 *   wo         [d, Hq * hd]
 *   w_gate_up  [2 * ffn, d]             rows 0..ffn-1 gate, ffn..2ffn-1 up
 *   w_down     [d, ffn]                                                       */
typedef struct spec_layer_weights {
  const void* attn_norm;
  const void* wqkv;
  const void* wo;
  const void* mlp_norm;
  const void* w_gate_up;
  const void* w_down;
} spec_layer_weights;

/* A Llama-style decoder: RMSNorm -> QKV -> rotate-half RoPE -> causal GQA
 * attention -> O (+ residual) -> RMSNorm -> SwiGLU MLP (+ residual); final
 * RMSNorm and an untied LM head producing fp32 logits.  Residual stream fp32. */
typedef struct spec_model_desc {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  int32_t dtype;          /* SPEC_F32 or SPEC_BF16: weights, KV cache, GEMM inputs */
  float rope_theta, rms_eps;
  const void* embed;      /* device [vocab, d] */
  const void* final_norm; /* device [d] */
  const void* lm_head;    /* device [vocab, d] (a projection: tiled for bf16) */
  const spec_layer_weights* layers; /* host array [n_layers]; copied by spec_ctx_create */
  int32_t weight_layout;  /* SPEC_LAYOUT_ROWMAJOR (fp32 models) or SPEC_LAYOUT_TILED
                             (bf16 models, set by spec_pack_model); checked by spec_ctx_create */
} spec_model_desc;

/* Convert the projection weights of a bf16 model in place from row-major to
 * the tiled layout that the bf16 kernels stream, and set m->weight_layout to
 * SPEC_LAYOUT_TILED.  Requires m->weight_layout == SPEC_LAYOUT_ROWMAJOR
 * (SPEC_E_STATE otherwise: converting twice would scramble the weights) and
 * d_model, ffn_dim and n_heads * head_dim multiples of 128, head_dim % 16 == 0
 * (SPEC_E_UNSUPPORTED).  Weights shared by two descriptors are converted
 * once.  The layout, per matrix W [N, K]: in every complete group of 16 rows
 * and block of 128 columns, the 16 x 16 matrix of 16-byte chunks is
 * transposed (chunk j of row r moves to row j, chunk position r); a trailing
 * group of fewer than 16 rows stays row-major; wqkv's q and k heads are first
 * reordered inside each head so that rows 8t..8t+7 and hd/2+8t..hd/2+8t+7
 * (rotary pairs) form tile t; w_gate_up is converted as two [ffn, d]
 * matrices.  Asynchronous on `stream`; fp32 models are left unchanged
 * (SPEC_OK, layout stays row-major). */
SPEC_API spec_status spec_pack_model(spec_model_desc* m, void* stream);

/* Paged KV cache.  Each pool holds, per layer, K pages [page][Hkv][16 x hd] and
 * V pages [page][Hkv][16 x hd], element type = model dtype; size it with
 * spec_kv_pool_bytes().  Inside a (page, kv head) block, fp32 stores K as
 * [16 tokens][hd] and V transposed as [hd][16 tokens]; bf16 orders the block
 * for the attention kernel's operand loads: token k, dim d of K at
 * 8 * (((s * 2 + h) * 4 + g) * 8 + j) + d % 8 with c = d / 8, s = c / 4,
 * g = c % 4, h = (k / 4) % 2, j = k % 4 + 4 * (k / 8); of V at
 * 8 * (((d / 16) * 2 + k / 8) * 16 + d % 16) + k % 8.  The library alone
 * writes the pools. */
typedef struct spec_cache_desc {
  int32_t page_size;          /* must be 16 */
  int32_t num_pages_target;
  int32_t num_pages_draft;
  int32_t max_seqs;           /* live sequences at once */
  int32_t max_pages_per_seq;
  int32_t k_max;              /* most drafts per sequence per step (1..15) */
  int32_t max_rows;           /* most rows per forward launch; prefill is chunked to it */
  void* kv_target;            /* device */
  void* kv_draft;             /* device */
} spec_cache_desc;

typedef struct spec_ctx spec_ctx;

/* Bytes one KV pool of `num_pages` pages needs for model `m`. */
SPEC_API size_t spec_kv_pool_bytes(const spec_model_desc* m, int32_t num_pages);

/* Create a context for a target/draft pair (same vocabulary and dtype): the
 * two models of speculative decoding, the small one proposing tokens that the
 * large one verifies (paper, Section 3.4 Cache-Miss Branch and the
 * speculative-decoding paragraph of Section 2).  draft == NULL makes a
 * decode-only context over `target` alone, for plain batched decoding with
 * spec_decode (the small model's other role, generating on its own:
 * Section 3.3 Cache-Hit Branch); its cache descriptor's draft pool and page
 * count are ignored and k_max may be 0, and the draft calls return
 * SPEC_E_STATE.  Models may share weights with another context's models
 * (the descriptors hold the caller's device pointers). */
SPEC_API spec_status spec_ctx_create(const spec_model_desc* target, const spec_model_desc* draft,
                                     const spec_cache_desc* cache, spec_ctx** out);
SPEC_API void spec_ctx_destroy(spec_ctx* ctx);
/* Message of the last failure; owned by ctx (or static for ctx == NULL), valid
 * until the next call on it. */
SPEC_API const char* spec_last_error(const spec_ctx* ctx);

/* Device workspace the context needs (activations, logits, draft rows,
 * attention partials, metadata).  Call spec_set_workspace once before any
 * compute call; the buffer must be 256-byte aligned and stay alive. */
SPEC_API size_t spec_workspace_bytes(const spec_ctx* ctx);
SPEC_API spec_status spec_set_workspace(spec_ctx* ctx, void* dev_ptr, size_t bytes);

/* Prefill: register `n` new sequences (caller-chosen, distinct, stable ids)
 * with prompts `tokens` (host, packed, prompt_lens[i] >= 1 tokens each) and run
 * positions 0..P-2 through both models (no LM head): the request enters the
 * target LLM and its drafter before draft-and-verify generation starts
 * (Section 3.4 Cache-Miss Branch; the request lengths of Section 4.7 Length
 * Robustness set the prompt sizes).  The last prompt token
 * becomes the pending token.  Pages: lowest-numbered free page first, in list
 * order.  Blocks until the work is done. */
SPEC_API spec_status spec_prefill(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                  const int32_t* prompt_lens, const int32_t* tokens, void* stream);

/* One draft step for each listed sequence (Section 3.4 Cache-Miss Branch:
 * the small model proposes candidate tokens; Section 2, speculative-decoding
 * paragraph): the draft model consumes its
 * pending tokens (the committed tail not yet in the draft cache on the first
 * step after a commit, else the previous draft) and draws the next draft token
 * x~_j at position n+j from softmax(z/T) by Gumbel-max with DRAFT noise
 * (argmax for T == 0).  The draft logits row is kept for the verify.  A
 * sequence is drafted at most k_max times between verifies.
 * temperature: host [n], >= 0.  Asynchronous. */
SPEC_API spec_status spec_draft_step(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                     const float* temperature, uint64_t seed, void* stream);

/* Several draft steps in one call (Section 2, speculative-decoding
 * paragraph: the small model proposes k tokens autoregressively): sequence i
 * takes part in steps[i] consecutive draft steps (0 <= steps[i], its draft
 * count + steps[i] <= k_max), each exactly spec_draft_step with this seed,
 * so the result (draft tokens, kept draft logits rows, caches) is the one
 * steps[i] spec_draft_step calls give.  Each step's token is drawn on the
 * device and feeds the next step there, so no step waits on the host: the
 * draft pages of every step are taken at the start (list order), step 0 runs
 * as one graph (the GPU starts while the host lays out the rest) and steps
 * 1 .. max(steps) - 1 as a second one, their metadata uploaded once.
 * temperature, steps: host [n].
 * Errors as spec_draft_step; on an error no step has run.  Asynchronous. */
SPEC_API spec_status spec_draft_loop(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                     const float* temperature, uint64_t seed, const int32_t* steps,
                                     void* stream);

/* WORKLOAD / TEST HOOK, not a step of the method.
 * spec_draft_step with draft guidance, a workload-shaping hook: for each
 * sequence i with guide[i] >= 0 (host int32 [n]; -1 = none), the guide
 * token's draft logit is raised to the row maximum + boost (>= 0) before the
 * draw, and the raised row is kept as that draft's proposal q (so the rule
 * stays exact).  Used to give random-init drafters a target-like acceptance
 * rate: the caller passes the target's top-1 token at that position for a
 * seeded fraction of the drafts. */
SPEC_API spec_status spec_draft_step_guided(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                            const float* temperature, uint64_t seed,
                                            const int32_t* guide, float boost, void* stream);

/* WORKLOAD / TEST HOOK, not a step of the method (the verify below runs the
 * same forward and decides).
 * The verify's target forward alone: rows x_n, x~_1..x~_k at positions n..n+k
 * of each listed sequence (their K/V are written, as the verify that follows
 * writes them), fp32 logits where spec_last_logits points, no decision pass.
 * Committed state is unchanged; the drafts stay pending.  Asynchronous. */
SPEC_API spec_status spec_target_forward(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, void* stream);

/* WORKLOAD / TEST HOOK, not a step of the method: it stands in for the draft
 * model when a test or bench supplies seeded drafts.
 * Replace a sequence's drafts by externally supplied ones: k tokens (host) and
 * their draft logits rows (device fp32 [k, vocab], which must stay alive until
 * the verify has run). */
SPEC_API spec_status spec_set_drafts(spec_ctx* ctx, int64_t seq_id, int32_t k,
                                     const int32_t* tokens, const float* q_logits, void* stream);

/* Replace a sequence's drafts by a draft tree (tree / multi-candidate
 * verification, which the paper's Section 2 lists among the variants of
 * speculative decoding): m nodes (1 <= m <= k_max), node i with token
 * tokens[i] and parent parents[i] (-1: the pending token x_n; otherwise a
 * node with a smaller index), so that node i stands at position n + its depth;
 * siblings are tried in index order.  q_logits: device fp32 [m + 1, vocab],
 * row 0 the draft logits the root's children were drawn from and row i + 1
 * those of node i's children (rows of leaves are not read); it must stay
 * alive until the verify has run.  The next spec_verify feeds x_n and every
 * node (node i's K/V at cache index n + 1 + i, each row attending to the
 * committed cache and its own ancestors), then applies multi-step speculative
 * sampling: at each node, children are accepted with probability
 * min(1, r(x) / q(x)) (uniform of candidate j: ACCEPT noise block j at
 * position n + depth + 1), r becoming norm(max(0, r - q)) after each
 * rejection; when every child of a node is rejected a token is drawn from r
 * (RESAMPLE noise), at a leaf from p (BONUS noise); greedy follows the child
 * whose token is the argmax.  n_accepted is the accepted depth, out_tokens
 * the accepted path's tokens and the drawn one; spec_kv_commit moves the
 * accepted nodes' K/V to positions n + 1 .. n + a.  A chain (parents[i] =
 * i - 1) gives exactly the results of spec_set_drafts.  Also allowed in a
 * decode-only context (the drafts need no draft model). */
SPEC_API spec_status spec_set_draft_tree(spec_ctx* ctx, int64_t seq_id, int32_t m, const int32_t* parents,
                                         const int32_t* tokens, const float* q_logits, void* stream);

/* Verify (Section 3.4 Cache-Miss Branch: the target LLM verifies the
 * candidates in one parallel pass and corrects or continues the generation;
 * Section 2, speculative-decoding paragraph, with the speculative sampling
 * rule of the works it cites, Leviathan et al. 2023 and Chen et al. 2023):
 * feed [x_n, x~_1..x~_k] at positions n..n+k through the target (their
 * K/V are written to the cache first, then each row attends causally), produce
 * fp32 logits, and apply the speculative sampling rule per sequence with its
 * own temperature.  Outputs (host): n_accepted[i] = a_i in 0..k_i and
 * out_tokens[i * (k_max + 1) + j] for j <= a_i (x~_1..x~_a, then the resampled
 * or bonus token); other entries are -1.  Committed lengths do not change.
 * Blocks until the outputs are on the host. */
SPEC_API spec_status spec_verify(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                 const float* temperature, uint64_t seed,
                                 int32_t* n_accepted, int32_t* out_tokens, void* stream);

/* Commit (Section 3.4 Cache-Miss Branch: the verified prefix and the
 * corrected token become the generation, the rejected candidates are
 * discarded) the last verify of each listed sequence with a accepted drafts
 * (normally the a returned by spec_verify): the target cache keeps positions
 * <= n+a, the draft cache keeps min(its length, n+a+1) positions, the emitted
 * tokens join the history, rejected K/V slots are cleared in place and pages
 * holding no kept position return to the free pool.  Asynchronous. */
SPEC_API spec_status spec_kv_commit(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                    const int32_t* n_accepted, void* stream);

/* The tail of one speculative round and the start of the next in one call,
 * so that the host round trip between them stays inside the library:
 * spec_verify (verify_seed; outputs as there, on the host when the call
 * returns), then spec_kv_commit of every listed sequence with the a the
 * verify returned, then spec_draft_loop of the next round (draft_seed,
 * steps[i] drafts for sequence i, host [n]).  The result equals the three
 * calls made in that order.  On an error the calls before it have taken
 * effect (a verify that failed commits nothing; a failed commit drafts
 * nothing).  The drafts are asynchronous, as in spec_draft_loop. */
SPEC_API spec_status spec_verify_commit_draft(spec_ctx* ctx, int32_t n, const int64_t* seq_ids,
                                              const float* temperature, uint64_t verify_seed,
                                              int32_t* n_accepted, int32_t* out_tokens,
                                              uint64_t draft_seed, const int32_t* steps, void* stream);

/* Plain autoregressive decoding of the context's target model, `steps` tokens
 * for each listed sequence (Section 3.3 Cache-Hit Branch: the small model
 * generates by itself; in a decode-only context the target is that model).
 * Each step feeds every sequence's pending token x_n at position n (its K/V
 * are written), draws the next token from softmax(z/T) by Gumbel-max with
 * BONUS noise keyed (seed, seq, n + 1) (argmax for T == 0, ties to the
 * lowest id) and commits it: exactly a spec_verify with no drafts followed by
 * spec_kv_commit.  The sequences must hold no drafts and no uncommitted
 * verify (SPEC_E_STATE); every page the call needs is checked before any
 * step runs (SPEC_E_NOPAGES).  temperature: host [n], >= 0.  out_tokens: host
 * int32 [n][steps], row i the tokens of sequence i in order.  Blocks until
 * the last step's tokens are on the host. */
SPEC_API spec_status spec_decode(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                                 uint64_t seed, int32_t steps, int32_t* out_tokens, void* stream);

/* Rollback (the discard half of the commit above, Section 3.4 Cache-Miss
 * Branch, for a caller that drops generated tokens itself).
 * Truncate both caches of a sequence to `new_len` positions (0 <= new_len <=
 * target length); history[new_len] becomes the pending token and outstanding
 * drafts are dropped.  Cleared in place like a commit.  Asynchronous. */
SPEC_API spec_status spec_kv_rollback(spec_ctx* ctx, int64_t seq_id, int32_t new_len, void* stream);

/* Forget a sequence and free its pages (the request's generation has ended,
 * Section 3.4 Cache-Miss Branch). */
SPEC_API spec_status spec_seq_release(spec_ctx* ctx, int64_t seq_id);

/* Introspection (host outputs): committed target/draft lengths, pending token
 * position n, and the page tables (*n_pages_* entries are written, at most
 * max_pages each).  Useful for checking KV indices. */
SPEC_API spec_status spec_seq_info(const spec_ctx* ctx, int64_t seq_id, int32_t* target_len,
                                   int32_t* draft_len, int32_t* pending_pos,
                                   int32_t* pages_target, int32_t* n_pages_target,
                                   int32_t* pages_draft, int32_t* n_pages_draft, int32_t max_pages);

/* Device address of the last verify's target logits, fp32 [rows, vocab] in
 * call order (sequence i's k_i + 1 rows are contiguous), and the row count. */
SPEC_API spec_status spec_last_logits(const spec_ctx* ctx, const float** logits, int32_t* rows);

/* Device address of the draft logits row (fp32 [vocab]) from which draft j
 * (0-based) of the sequence's current drafts was drawn (for spec_set_drafts
 * drafts: the caller's row).  Valid until the sequence's next commit,
 * rollback or release. */
SPEC_API spec_status spec_draft_logits(const spec_ctx* ctx, int64_t seq_id, int32_t j, const float** row);

/* The sequence's current drafts, copied to the host: tokens[0 .. *k - 1]
 * (room for k_max entries), *k = their count.  Waits for `stream`. */
SPEC_API spec_status spec_draft_tokens(spec_ctx* ctx, int64_t seq_id, int32_t* tokens, int32_t* k,
                                       void* stream);

/* Graph replay of the draft step and the verify (on by default).  Their
 * kernel sequence depends only on the batch shape (rows, sequences, attention
 * work items), so the second call of a shape captures it into a HIP graph and
 * later calls of that shape upload their metadata and replay the graph: one
 * launch instead of ~10 per layer.  Up to 16 shapes are kept (least recently
 * used replaced); a new workspace drops them.  Calls whose forwards have more
 * than 16 rows always launch eagerly (their kernels are long enough that a
 * replay saves nothing, and their shapes rarely recur).  Results are
 * identical with and without graphs.  While kernel timing is on, calls run
 * eagerly so that each launch can be timed.  enable = 0 turns replay off. */
SPEC_API spec_status spec_set_graphs(spec_ctx* ctx, int32_t enable);

/* Kernel timing for roofline measurement.  While a kernel name is set, the
 * context times every launch of that kernel with HIP events that record the
 * kernel's own start and end (the GEMM, attention and vocab-statistics
 * kernels; other kernels: events on the call's stream around the launch).
 * Names as the profiler reports them without namespaces and argument lists,
 * e.g. "gemm_skinny_bf16<1, 2, true>", "gemm_mfma2_bf16<2, 6, 8>",
 * "attn_bf16_kernel<128, 2, 4>", "stats_kernel<true>"; "tree_decision" times
 * the tree verify's decision after its statistics pass (several kernels) as
 * one span.  It accumulates the
 * elapsed time, the launch count and each launch's algorithmic HBM bytes and
 * flops (weights, activations and KV actually required, each read once).
 * name NULL or "" disables timing.  spec_timing_read waits for the recorded
 * events and returns the totals since the last spec_timing_enable. */
SPEC_API spec_status spec_timing_enable(spec_ctx* ctx, const char* kernel_name);
SPEC_API spec_status spec_timing_read(spec_ctx* ctx, double* total_ms, int64_t* launches,
                                      double* bytes, double* flops);

/* ---------------------------------------------------------------------------
 * The decision pass alone, on caller-provided device logits: the acceptance
 * scan, the residual resample and the bonus draw of speculative sampling
 * (Section 3.4 Cache-Miss Branch and Section 2, speculative-decoding
 * paragraph; the rule of the cited Leviathan et al. 2023 / Chen et al. 2023).
 *
 * B sequences; sequence b has k[b] drafts (0..15), temperature[b] >= 0,
 * stable id seq_ids[b] and pending-token position base_pos[b] (all host arrays).
 * p_logits: device fp32 [sum(k+1), V], sequence b's rows contiguous in order.
 * q_logits: device fp32 [sum(k), V], likewise.  draft_tokens: device int32
 * [sum(k)].  Outputs (device): n_accepted[B], out_tokens[B * (k_max + 1)]
 * where k_max = max k[b].  workspace: device, >= spec_sample_workspace_bytes.
 * Asynchronous; host arrays are consumed before return. */
SPEC_API size_t spec_sample_workspace_bytes(int32_t B, int32_t total_rows, int32_t V);
SPEC_API spec_status spec_sample_verify(int32_t B, const int32_t* k, const float* temperature,
                                        const int64_t* seq_ids, const int32_t* base_pos,
                                        const float* p_logits, const float* q_logits,
                                        const int32_t* draft_tokens, int32_t V, uint64_t seed,
                                        int32_t* n_accepted, int32_t* out_tokens,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* The decision pass of spec_sample_verify for callers that cannot allocate
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): it calls no allocating routine and copies nothing from
 * the host.  The per-sequence inputs are device arrays: k[B] (int32, each in
 * 0..k_max), temperature[B] (fp32, >= 0), seq_ids[B] (int64), base_pos[B]
 * (int32); the logits, drafts and outputs are as in spec_sample_verify, with
 * out_tokens [B * (k_max + 1)].  Given k_max = max k[b], the outputs are bit
 * for bit those of spec_sample_verify.  Tables and partial results live in a
 * 512 KiB device array that the library holds on each GPU it runs on until
 * the process ends: B <= 256 and k_max <= 15 (SPEC_E_INVALID otherwise); a
 * shape whose tables exceed the array returns SPEC_E_UNSUPPORTED before
 * anything is enqueued.  If any k[b] is outside 0..k_max or any temperature
 * is negative or NaN, nothing is decided and every n_accepted[b] and token is
 * -1 (the inputs are on the device, so this is reported there).  Every call
 * on one GPU uses the same array: calls that overlap on one GPU (different
 * streams, or threads) race, and must be serialised by the caller.
 * Asynchronous on `stream`; spec_last_error(NULL) explains a failure. */
SPEC_API spec_status spec_sample_verify_noalloc(int32_t B, int32_t k_max, const int32_t* k,
                                                const float* temperature, const int64_t* seq_ids,
                                                const int32_t* base_pos, const float* p_logits,
                                                const float* q_logits, const int32_t* draft_tokens,
                                                int32_t V, uint64_t seed, int32_t* n_accepted,
                                                int32_t* out_tokens, void* stream);

/* The drafter's draw (Section 3.4: the small model proposes candidate
 * tokens), for callers holding their own draft logits.
 * Draw one draft token per row: row i of `logits` (device fp32 [n, V]) is the
 * draft distribution for position pos[i] of sequence seq_ids[i] (host arrays);
 * tokens (device int32 [n]) <- Gumbel-max with DRAFT noise, argmax if T == 0. */
SPEC_API spec_status spec_sample_draft(int32_t n, const float* logits, int32_t V,
                                       const float* temperature, const int64_t* seq_ids,
                                       const int32_t* pos, uint64_t seed, int32_t* tokens,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* The generator itself: out (device fp32 [n]) <- uniforms of stream
 * (seed, seq_id, pos, purpose), words 0..n-1. */
SPEC_API spec_status spec_philox_uniform(uint64_t seed, int64_t seq_id, int32_t pos, int32_t purpose,
                                         int32_t n, float* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SPEC_H_ */
