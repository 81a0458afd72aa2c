// Host orchestration of the draft-and-verify step: the C ABI of include/spec.h.
//
// Sequence model (pending token): a sequence's committed tokens are
// x_0..x_n; x_n (position n) is pending, i.e. not in the target cache, whose
// length is n.  The draft cache has length len_d <= n.  Draft step j feeds the
// draft model the pending tail (j = 1) or x~_{j-1} and draws x~_j at position
// n + j.  Verify feeds x_n, x~_1..x~_k at positions n..n+k to the target,
// writes their K/V, and applies the speculative sampling rule.  Commit keeps
// target positions <= n + a and draft positions < min(len_d, n + a + 1).
//
// One metadata block (rows, positions, KV slots, page tables, attention work
// items, decision tables, the Philox seed) is uploaded per call through a
// pinned ring; the decision outputs come back in one small copy per verify.
// The kernel sequence of a draft step or a verify depends only on the batch
// shape (rows, sequences, attention work items), so it is captured once per
// shape into a HIP graph whose kernels read that call's metadata from a fixed
// device area, and replayed: one launch instead of ~10 per layer.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <functional>
#include <queue>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "../../include/spec.h"
#include "attention.h"
#include "elem.h"
#include "gemm.h"
#include "host_util.h"
#include "pages.h"
#include "vocab.h"

using namespace spec;

namespace {

constexpr int kMaxParts = 1024;
constexpr int kMetaRing = 4;
constexpr int kGraphSlots = 16;

struct Model {
  spec_model_desc d{};
  std::vector<spec_layer_weights> layers;
  int esz = 2;
  char* kv = nullptr;
  int num_pages = 0;
  size_t layer_stride = 0, v_off = 0;  // elements
  PagePool pool;
  int dt() const { return d.dtype == SPEC_F32 ? 0 : 1; }
  int G() const { return d.n_heads / d.n_kv_heads; }
  int qkvw() const { return (d.n_heads + 2 * d.n_kv_heads) * d.head_dim; }
  int qdim() const { return d.n_heads * d.head_dim; }
  void* kl(int l) const { return kv + static_cast<size_t>(l) * layer_stride * esz; }
  void* vl(int l) const { return kv + (static_cast<size_t>(l) * layer_stride + v_off) * esz; }
};

struct Seq {
  int64_t id = 0;
  int slot = 0;
  std::vector<int32_t> hist;
  int len_t = 0, len_d = 0;
  int written_t = 0;
  std::vector<int32_t> pages_t, pages_d;
  int k = 0;
  std::vector<const float*> qrow;
  std::vector<int32_t> dsrc;  // >= 0 token id, < 0: -(1 + index into the device draft-token pool)
  bool external = false;
  bool verified = false;
  int a_ver = 0;
  std::vector<int32_t> emitted;
  // draft tree (spec_set_draft_tree): parent of node i (-1: the pending
  // token), empty for a chain; the accepted nodes after a verify
  std::vector<int32_t> tparent, tpath;
  int n() const { return static_cast<int>(hist.size()) - 1; }
};

struct Ws {
  size_t h = 0, y = 0, qkv = 0, q = 0, o = 0, u = 0, logits = 0, dq = 0, dtok = 0, rowtok = 0;
  size_t part_o = 0, part_ml = 0, vocab = 0, draft = 0, meta = 0, gmeta = 0;
  size_t splitk = 0, splitk_bytes = 0, ss = 0;
  size_t meta_cap = 0, total = 0;
};

// Host description of one forward launch.
struct Fwd {
  std::vector<int32_t> tok_src, pos, slot, seqi;
  std::vector<int32_t> tbase;   // tree verification: per row, the last cache index all of it sees
  std::vector<uint32_t> tmask;  // and the tree slots beyond it (bit j: index tbase + 1 + j)
  std::vector<AttnSegment> segs;
  std::vector<int32_t> ptab;
  int ptab_stride = 1;
  std::vector<int32_t> lm_rows, lm_map;
};

struct FwdOff {
  size_t tok, pos, slot, seqi, pt, items, groups, lmr, lmm, tb = 0, tm = 0;
  bool tree = false, prefill = false;
  int n_items = 0, n_groups = 0, nt = 1, w = 1, R = 0, n_lm = 0, ptab_stride = 1;
  bool lm_map = false;
  double attn_keys = 0, attn_qk = 0;  // sum of context lengths; sum over rows of (pos + 1)
};

size_t pool_layer_elems(const spec_model_desc& m, int num_pages) {
  return static_cast<size_t>(num_pages) * m.n_kv_heads * 16 * m.head_dim * 2;
}

bool valid_model(const spec_model_desc* m, std::string& why) {
  if (!m) { why = "null model"; return false; }
  if (m->n_layers <= 0 || m->d_model <= 0 || m->n_heads <= 0 || m->n_kv_heads <= 0 ||
      m->head_dim <= 0 || m->ffn_dim <= 0 || m->vocab <= 0) { why = "non-positive model size"; return false; }
  if (m->n_heads % m->n_kv_heads != 0) { why = "n_heads must be a multiple of n_kv_heads"; return false; }
  if (m->dtype != SPEC_F32 && m->dtype != SPEC_BF16) { why = "dtype must be SPEC_F32 or SPEC_BF16"; return false; }
  if (m->weight_layout != (m->dtype == SPEC_BF16 ? SPEC_LAYOUT_TILED : SPEC_LAYOUT_ROWMAJOR)) {
    why = m->dtype == SPEC_BF16 ? "bf16 weights must be in the tiled layout (spec_pack_model)"
                                : "fp32 weights must be row-major";
    return false;
  }
  if (!m->embed || !m->final_norm || !m->lm_head || !m->layers) { why = "null weight pointer"; return false; }
  for (int l = 0; l < m->n_layers; ++l) {
    const auto& L = m->layers[l];
    if (!L.attn_norm || !L.wqkv || !L.wo || !L.mlp_norm || !L.w_gate_up || !L.w_down) {
      why = "null layer weight pointer"; return false;
    }
  }
  return true;
}

int unsupported_model(const spec_model_desc* m, std::string& why) {
  if (m->head_dim != 64 && m->head_dim != 128) { why = "head_dim must be 64 or 128"; return 1; }
  if (m->dtype == SPEC_BF16) {
    if (m->d_model % 128 || m->ffn_dim % 128 || (m->n_heads * m->head_dim) % 128) {
      why = "bf16 models need d_model, ffn_dim and n_heads*head_dim multiples of 128"; return 1;
    }
    if (m->n_heads / m->n_kv_heads > 16) { why = "at most 16 query heads per kv head"; return 1; }
  }
  return 0;
}

}  // namespace

struct spec_ctx {
  Model m[2];  // 0 target, 1 draft
  int n_models = 2;  // 1: a decode-only context (no draft model)
  spec_cache_desc cache{};
  int R_max = 0, V = 0, k_max = 0, max_seqs = 0, max_pages = 0;
  int d_max = 0, qkv_max = 0, q_max = 0, ffn_max = 0, hkv_max = 0, hd_max = 0, esz_max = 2;
  Ws ws;
  char* wsp = nullptr;
  size_t ws_bytes = 0;
  std::unordered_map<int64_t, Seq> seqs;
  std::priority_queue<int, std::vector<int>, std::greater<int>> free_slots;
  Stager stager;
  int meta_next = 0;
  // pinned, written by the decision pass's last kernel itself: n_acc [max_seqs],
  // tokens [max_seqs * (k_max + 1)], then the accepted tree nodes
  // [max_seqs * k_max]; h_out_dev is its device address
  int32_t* h_out = nullptr;
  int32_t* h_out_dev = nullptr;
  hipEvent_t out_ev = nullptr;
  std::string err;
  bool broken = false;
  int last_rows = 0;
  EventTimer timer;
  // captured kernel sequences, one per batch shape (least recently used out)
  struct Graph {
    std::vector<int64_t> key;
    hipGraphExec_t exec = nullptr;
    uint64_t used = 0;
  };
  Graph graphs[kGraphSlots];
  uint64_t graph_clock = 0;
  // shapes seen recently but not captured: a shape is captured when it comes
  // back, so batches whose shape changes every call (growing contexts across
  // many sequences) run eagerly instead of paying a capture per call
  std::vector<std::vector<int64_t>> seen;
  bool use_graphs = true;
  hipStream_t cap_stream = nullptr;  // capture only: nothing runs on it
  void drop_graphs() {
    for (auto& g : graphs) {
      if (g.exec) (void)hipGraphExecDestroy(g.exec);
      g = Graph{};
    }
  }
};

static thread_local std::string g_err;

namespace spec {
void set_global_error(const char* msg) { g_err = msg ? msg : ""; }
}  // namespace spec

#define FAIL(code, msg)          \
  do {                           \
    ctx->err = (msg);            \
    return (code);               \
  } while (0)

#define HIPC(expr)                                                              \
  do {                                                                          \
    hipError_t e_ = (expr);                                                     \
    if (e_ != hipSuccess) {                                                     \
      ctx->broken = true;                                                       \
      ctx->err = std::string("HIP error in ") + #expr + ": " + hipGetErrorString(e_); \
      return SPEC_E_HIP;                                                        \
    }                                                                           \
  } while (0)

namespace {

void compute_ws(spec_ctx* c) {
  Ws& w = c->ws;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const size_t R = c->R_max;
  const size_t nq = static_cast<size_t>(c->max_seqs) * c->k_max;
  w.h = take(R * c->d_max * 4);
  w.y = take(R * std::max(c->d_max, c->q_max) * c->esz_max);
  w.qkv = take(R * c->qkv_max * 4);
  w.q = take(R * c->q_max * c->esz_max);
  w.o = take(R * c->q_max * c->esz_max);
  w.u = take(R * c->ffn_max * c->esz_max);
  const size_t vr = static_cast<size_t>(c->max_seqs) * (c->k_max + 1);
  w.logits = take(vr * c->V * 4);
  w.dq = take(nq * c->V * 4);
  w.dtok = take(nq * 4);
  w.rowtok = take(R * 4);
  w.ss = take(R * (c->d_max / 8 + 1) * 4);
  w.part_o = take(static_cast<size_t>(kMaxParts) * c->hkv_max * 64 * c->hd_max * 4);
  w.part_ml = take(static_cast<size_t>(kMaxParts) * c->hkv_max * 64 * 2 * 4);
  const int vrows = c->max_seqs * (2 * c->k_max + 1);
  // bounds over every call size (a smaller call can take more chunks per row)
  w.vocab = take(std::max(vocab_ws_bound(c->max_seqs, vrows), tree_ws_bound(c->max_seqs, vrows)));
  w.draft = take(draft_ws_bound(c->max_seqs));
  w.splitk_bytes = gemm_splitk_bytes(c->R_max, std::max(c->qkv_max, 2 * c->ffn_max));
  w.splitk = take(w.splitk_bytes);
  // metadata bound for one call
  size_t mc = 0;
  mc += 8 * align_up(R * 4);  // tokens, positions, slots, rows, LM rows and map; tree bases and masks
  mc += align_up(R * sizeof(VTreeNode));
  mc += align_up(static_cast<size_t>(c->max_seqs) * c->max_pages * 4);
  mc += align_up((R + kMaxParts) * sizeof(AttnItem)) + align_up(R * sizeof(AttnGroup));
  mc += align_up(static_cast<size_t>(vrows) * sizeof(VRow)) + align_up(c->max_seqs * sizeof(VSeq));
  mc += align_up(c->max_seqs * sizeof(DRow));
  const size_t clears = std::max<size_t>(static_cast<size_t>(c->max_seqs) * (c->k_max + 2),
                                         static_cast<size_t>(c->max_pages) * 16);
  mc += 2 * align_up(clears * 4);
  mc += 16 * 256;
  w.meta_cap = align_up(mc);
  w.meta = take(w.meta_cap * kMetaRing);
  w.gmeta = take(w.meta_cap * kGraphSlots);
  w.total = off;
}

template <typename T>
T* wsptr(spec_ctx* c, size_t off) {
  return reinterpret_cast<T*>(c->wsp + off);
}

// Upload a metadata block; returns the device base.
spec_status upload_meta(spec_ctx* ctx, const MetaBlock& mb, hipStream_t st, char** dev) {
  if (mb.size() > ctx->ws.meta_cap) FAIL(SPEC_E_UNSUPPORTED, "call metadata exceeds its bound");
  char* base = ctx->wsp + ctx->ws.meta + static_cast<size_t>(ctx->meta_next) * ctx->ws.meta_cap;
  ctx->meta_next = (ctx->meta_next + 1) % kMetaRing;
  HIPC(ctx->stager.upload(base, mb.data(), mb.size(), st));
  *dev = base;
  return SPEC_OK;
}

FwdOff add_forward(spec_ctx* ctx, const Model& M, const Fwd& f, MetaBlock& mb) {
  FwdOff o;
  o.R = static_cast<int>(f.tok_src.size());
  o.tok = mb.add(f.tok_src);
  o.pos = mb.add(f.pos);
  o.slot = mb.add(f.slot);
  o.seqi = mb.add(f.seqi);
  o.pt = mb.add(f.ptab);
  o.ptab_stride = f.ptab_stride;
  if (M.dt() == 1) {
    AttnPlan p = plan_attention(f.segs, M.G(), M.d.n_kv_heads, kMaxParts, kAttnTargetWgs, f.tbase.empty());
    o.prefill = p.prefill;
    o.items = mb.add(p.items);
    o.groups = mb.add(p.groups);
    o.n_items = static_cast<int>(p.items.size());
    o.n_groups = static_cast<int>(p.groups.size());
    o.nt = p.nt;
    o.w = p.w;
  }
  for (const auto& s : f.segs) {
    o.attn_keys += s.pos0 + s.nrows;
    for (int r = 0; r < s.nrows; ++r) o.attn_qk += s.pos0 + r + 1;
  }
  if (!f.tbase.empty()) {
    o.tree = true;
    o.tb = mb.add(f.tbase);
    o.tm = mb.add(f.tmask);
  }
  o.n_lm = static_cast<int>(f.lm_rows.size());
  o.lmr = mb.add(f.lm_rows);
  o.lm_map = !f.lm_map.empty();
  o.lmm = mb.add(f.lm_map);
  (void)ctx;
  return o;
}

spec_status launch_forward(spec_ctx* ctx, const Model& M, const FwdOff& o, const char* dev,
                           float* logits, hipStream_t st) {
  const int dt = M.dt();
  const int R = o.R;
  const auto& d = M.d;
  auto I = [&](size_t off) { return reinterpret_cast<const int32_t*>(dev + off); };
  float* h = wsptr<float>(ctx, ctx->ws.h);
  void* y = ctx->wsp + ctx->ws.y;
  float* qkv = wsptr<float>(ctx, ctx->ws.qkv);
  void* q = ctx->wsp + ctx->ws.q;
  void* ob = ctx->wsp + ctx->ws.o;
  void* u = ctx->wsp + ctx->ws.u;
  // Up to 8 rows (batch-1 verify and draft steps) RMSNorm and RoPE / KV
  // append run inside the GEMMs (launch_gemm_fused): each residual-add GEMM
  // (and the embedding) also writes bf16(h (.) w_next) into y and per-8-column
  // sums of squares into ss; the next GEMM reads y and scales its output rows
  // by 1/rms; the QKV GEMM applies RoPE and writes q and the KV cache itself.
  const bool fused = dt == 1 && R <= 8 && d.head_dim % 16 == 0 && d.d_model % 16 == 0;
  float* ss = wsptr<float>(ctx, ctx->ws.ss);
  HIPC(launch_embed(dt, R, d.d_model, I(o.tok), wsptr<int32_t>(ctx, ctx->ws.dtok), d.embed, h,
                    wsptr<int32_t>(ctx, ctx->ws.rowtok), st, fused ? y : nullptr,
                    fused ? M.layers[0].attn_norm : nullptr, fused ? ss : nullptr));
  AttnArgs a;
  a.dtype = dt;
  a.Hq = d.n_heads;
  a.Hkv = d.n_kv_heads;
  a.hd = d.head_dim;
  a.q = q;
  a.page_table = I(o.pt);
  a.max_pages = o.ptab_stride;
  a.out = ob;
  a.part_o = wsptr<float>(ctx, ctx->ws.part_o);
  a.part_ml = wsptr<float>(ctx, ctx->ws.part_ml);
  if (o.tree) {
    a.tree_base = I(o.tb);
    a.tree_mask = reinterpret_cast<const uint32_t*>(dev + o.tm);
  }
  EventTimer& tm = ctx->timer;
  const double esz = M.esz;
  // GEMM launch, timed when selected: algorithmic bytes = weights + inputs +
  // outputs (read-modify-write for the residual add), flops = 2 R N_w K.
  auto gemm = [&](int rows, int N, int K, const void* X, const void* W, void* Y, int epi,
                  const int32_t* rm, const GemmFuse* f = nullptr, GemmNorm* nrm = nullptr) -> hipError_t {
    const bool timed = tm.wants(gemm_kernel_name(dt, rows, N, K, epi, f != nullptr, ctx->ws.splitk_bytes));
    if (timed) tm.begin(st);
    const hipError_t e =
        f ? launch_gemm_fused(rows, N, K, X, W, Y, epi, *f, st, rm)
          : launch_gemm(dt, rows, N, K, X, W, Y, epi, st, rm, wsptr<float>(ctx, ctx->ws.splitk),
                        ctx->ws.splitk_bytes, nrm);
    if (timed) {
      const double nw = epi == kEpiSwiGLU ? 2.0 * N : N;
      const double ob = epi == kEpiStoreF32 ? 4.0 : (epi == kEpiAddF32 ? 8.0 : esz);
      tm.end(st, (nw * K + double(rows) * K) * esz + double(rows) * N * ob, 2.0 * rows * nw * K);
    }
    return e;
  };
  // Above 8 rows each RMSNorm is its own kernel, unless the residual-add GEMM
  // before it splits K: then the split-K reduction applies it (GemmNorm).
  bool normed = false;  // y already holds the next RMSNorm's rows
  for (int l = 0; l < d.n_layers; ++l) {
    const auto& L = M.layers[l];
    if (fused) {
      GemmFuse fq;
      fq.ss = ss;
      fq.eps = d.rms_eps;
      fq.Hq = d.n_heads;
      fq.Hkv = d.n_kv_heads;
      fq.hd = d.head_dim;
      fq.theta = d.rope_theta;
      fq.pos = I(o.pos);
      fq.slot = I(o.slot);
      fq.qout = q;
      fq.kpool = M.kl(l);
      fq.vpool = M.vl(l);
      HIPC(gemm(R, M.qkvw(), d.d_model, y, L.wqkv, nullptr, kEpiQKVRope, nullptr, &fq));
    } else {
      if (!normed) HIPC(launch_rmsnorm(dt, R, d.d_model, h, nullptr, L.attn_norm, d.rms_eps, y, st));
      // a split-K QKV projection leaves its partials for rope_kv to sum
      GemmNorm defer;
      defer.defer = d.head_dim % 4 == 0 && (d.n_heads / d.n_kv_heads + 2) * d.head_dim <= kRopeSplitMaxWidth;
      HIPC(gemm(R, M.qkvw(), d.d_model, y, L.wqkv, qkv, kEpiStoreF32, nullptr, nullptr, &defer));
      HIPC(launch_rope_kv(dt, R, d.n_heads, d.n_kv_heads, d.head_dim, d.rope_theta,
                          defer.split > 0 ? defer.part : qkv, I(o.pos), I(o.slot), q, M.kl(l), M.vl(l), st,
                          dt == 1, defer.split));
    }
    a.kpool = M.kl(l);
    a.vpool = M.vl(l);
    if (dt == 1) {
      // bytes: every cached key and value once, queries in, output out
      const bool timed = tm.wants(o.prefill ? attn_prefill_kernel_name(d.head_dim)
                                            : attn_kernel_name(d.head_dim, o.nt, o.w, o.tree));
      if (timed) tm.begin(st);
      if (o.prefill)
        HIPC(launch_attention_prefill_bf16(a, reinterpret_cast<const AttnItem*>(dev + o.items), o.n_items, st));
      else
        HIPC(launch_attention_bf16(a, reinterpret_cast<const AttnItem*>(dev + o.items), o.n_items,
                                   reinterpret_cast<const AttnGroup*>(dev + o.groups), o.n_groups,
                                   o.nt, o.w, st));
      if (timed)
        tm.end(st, (o.attn_keys * d.n_kv_heads * 2.0 + 2.0 * R * d.n_heads) * d.head_dim * esz,
               4.0 * o.attn_qk * d.n_heads * d.head_dim);
    } else {
      HIPC(launch_attention_f32(a, R, I(o.seqi), I(o.pos), st));
    }
    if (fused) {
      GemmFuse fo;
      fo.hb = y;
      fo.wn = L.mlp_norm;
      fo.ss_out = ss;
      HIPC(gemm(R, d.d_model, M.qdim(), ob, L.wo, h, kEpiAddF32, nullptr, &fo));
      GemmFuse fg;
      fg.ss = ss;
      fg.eps = d.rms_eps;
      HIPC(gemm(R, d.ffn_dim, d.d_model, y, L.w_gate_up, u, kEpiSwiGLU, nullptr, &fg));
      GemmFuse fd;
      fd.hb = y;
      fd.wn = l + 1 < d.n_layers ? M.layers[l + 1].attn_norm : d.final_norm;
      fd.ss_out = ss;
      HIPC(gemm(R, d.d_model, d.ffn_dim, u, L.w_down, h, kEpiAddF32, nullptr, &fd));
    } else {
      GemmNorm no;
      no.w = L.mlp_norm;
      no.eps = d.rms_eps;
      no.y = y;
      HIPC(gemm(R, d.d_model, M.qdim(), ob, L.wo, h, kEpiAddF32, nullptr, nullptr, &no));
      if (!no.done) HIPC(launch_rmsnorm(dt, R, d.d_model, h, nullptr, L.mlp_norm, d.rms_eps, y, st));
      HIPC(gemm(R, d.ffn_dim, d.d_model, y, L.w_gate_up, u, kEpiSwiGLU, nullptr));
      GemmNorm nd;  // the next layer's attention norm (the last layer's final norm is per LM row)
      nd.w = l + 1 < d.n_layers ? M.layers[l + 1].attn_norm : nullptr;
      nd.eps = d.rms_eps;
      nd.y = y;
      HIPC(gemm(R, d.d_model, d.ffn_dim, u, L.w_down, h, kEpiAddF32, nullptr, nullptr, nd.w ? &nd : nullptr));
      normed = nd.done;
    }
  }
  if (o.n_lm > 0) {
    // the fused GEMM takes whole 16-row tiles of W: a vocabulary that is not a
    // multiple of 16 goes through the row-gathering RMSNorm and the plain GEMM
    // (h holds the residual stream either way)
    if (fused && d.vocab % 16 == 0) {
      GemmFuse fl;
      fl.ss = ss;
      fl.xrow = I(o.lmr);
      fl.eps = d.rms_eps;
      HIPC(gemm(o.n_lm, d.vocab, d.d_model, y, d.lm_head, logits, kEpiStoreF32, o.lm_map ? I(o.lmm) : nullptr,
                &fl));
    } else {
      HIPC(launch_rmsnorm(dt, o.n_lm, d.d_model, h, I(o.lmr), d.final_norm, d.rms_eps, y, st));
      HIPC(gemm(o.n_lm, d.vocab, d.d_model, y, d.lm_head, logits, kEpiStoreF32, o.lm_map ? I(o.lmm) : nullptr));
    }
  }
  return SPEC_OK;
}

// Page table of the listed sequences (row i = sequence i), `stride` entries per
// row (the per-sequence maximum, so that the layout depends on the batch shape
// only).
void build_ptab(const std::vector<const std::vector<int32_t>*>& tabs, Fwd& f, int stride) {
  size_t w = static_cast<size_t>(std::max(1, stride));
  for (auto* t : tabs) w = std::max(w, t->size());
  f.ptab_stride = static_cast<int>(w);
  f.ptab.assign(tabs.size() * w, 0);
  for (size_t i = 0; i < tabs.size(); ++i)
    std::copy(tabs[i]->begin(), tabs[i]->end(), f.ptab.begin() + i * w);
}

int32_t dev_tok_ref(int slot, int k_max, int j) { return -(1 + slot * k_max + j); }

bool check_ids(spec_ctx* ctx, int32_t n, const int64_t* ids, bool must_exist) {
  std::unordered_set<int64_t> seen;
  for (int i = 0; i < n; ++i) {
    if (!seen.insert(ids[i]).second) {
      ctx->err = "duplicate seq_id in call";
      return false;
    }
    if (must_exist && !ctx->seqs.count(ids[i])) {
      ctx->err = "unknown seq_id " + std::to_string(ids[i]);
      return false;
    }
  }
  return true;
}

// Run a call's kernels: eagerly through the metadata ring while kernel timing
// is on, graphs are off or a forward of the call has more than
// kGraphMaxRows rows, else by replaying the graph captured for `key`
// (captured the second time the shape occurs; the metadata goes to that
// graph's fixed area).  Graphs pay where launches are short (batch-1 draft
// and verify steps: 7.20 -> 7.11 ms per step); on the 64-sequence serving
// batch the shapes drift with the contexts, each capture cost 0.3-1 ms of
// host time and replays ran no faster than eager launches.
constexpr int kGraphMaxRows = 16;

spec_status run_kernels(spec_ctx* ctx, const std::vector<int64_t>& key, int rows, const MetaBlock& mb,
                        hipStream_t st,
                        const std::function<spec_status(const char*, hipStream_t)>& launches) {
  if (!ctx->use_graphs || !ctx->timer.name.empty() || rows > kGraphMaxRows) {
    char* dev = nullptr;
    spec_status s = upload_meta(ctx, mb, st, &dev);
    if (s != SPEC_OK) return s;
    return launches(dev, st);
  }
  if (mb.size() > ctx->ws.meta_cap) FAIL(SPEC_E_UNSUPPORTED, "call metadata exceeds its bound");
  int slot = -1;
  for (int i = 0; i < kGraphSlots && slot < 0; ++i)
    if (ctx->graphs[i].exec && ctx->graphs[i].key == key) slot = i;
  if (slot < 0) {
    auto it = std::find(ctx->seen.begin(), ctx->seen.end(), key);
    if (it == ctx->seen.end()) {
      if (ctx->seen.size() >= 4 * kGraphSlots) ctx->seen.erase(ctx->seen.begin());
      ctx->seen.push_back(key);
      char* dev = nullptr;
      spec_status s = upload_meta(ctx, mb, st, &dev);
      if (s != SPEC_OK) return s;
      return launches(dev, st);
    }
    ctx->seen.erase(it);
    slot = 0;
    for (int i = 1; i < kGraphSlots; ++i)
      if (ctx->graphs[i].used < ctx->graphs[slot].used) slot = i;
  }
  auto& g = ctx->graphs[slot];
  char* dev = ctx->wsp + ctx->ws.gmeta + static_cast<size_t>(slot) * ctx->ws.meta_cap;
  HIPC(ctx->stager.upload(dev, mb.data(), mb.size(), st));
  if (!g.exec || g.key != key) {
    if (g.exec) {
      // the slot's previous graph may still be queued on `st`: destroy it
      // after everything enqueued so far has run
      HIPC(hipStreamSynchronize(st));
      HIPC(hipGraphExecDestroy(g.exec));
      g = spec_ctx::Graph{};
    }
    if (!ctx->cap_stream) HIPC(hipStreamCreateWithFlags(&ctx->cap_stream, hipStreamNonBlocking));
    HIPC(hipStreamBeginCapture(ctx->cap_stream, hipStreamCaptureModeThreadLocal));
    spec_status s = launches(dev, ctx->cap_stream);
    hipGraph_t graph = nullptr;
    const hipError_t e = hipStreamEndCapture(ctx->cap_stream, &graph);
    if (s != SPEC_OK) {
      if (graph) (void)hipGraphDestroy(graph);
      return s;
    }
    HIPC(e);
    const hipError_t ei = hipGraphInstantiate(&g.exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    HIPC(ei);
    g.key = key;
  }
  g.used = ++ctx->graph_clock;
  HIPC(hipGraphLaunch(g.exec, st));
  return SPEC_OK;
}

// Shape key of a forward: everything its grids and metadata layout depend on.
void key_forward(std::vector<int64_t>& k, const FwdOff& o) {
  const int64_t v[] = {o.R, o.n_items, o.n_groups, o.nt, o.w, o.prefill, o.n_lm, o.lm_map, o.ptab_stride,
                       static_cast<int64_t>(o.tok), static_cast<int64_t>(o.pos),
                       static_cast<int64_t>(o.slot), static_cast<int64_t>(o.seqi),
                       static_cast<int64_t>(o.pt), static_cast<int64_t>(o.items),
                       static_cast<int64_t>(o.groups), static_cast<int64_t>(o.lmr),
                       static_cast<int64_t>(o.lmm), o.tree, static_cast<int64_t>(o.tb),
                       static_cast<int64_t>(o.tm)};
  k.insert(k.end(), std::begin(v), std::end(v));
}

spec_status launch_clears(spec_ctx* ctx, const std::vector<int32_t>& ct, const std::vector<int32_t>& cd,
                          hipStream_t st) {
  if (ct.empty() && cd.empty()) return SPEC_OK;
  const Model& T = ctx->m[0];
  const Model& D = ctx->m[1];
  auto job = [&](const Model& M, const std::vector<int32_t>& c) {
    KvClearJob j;
    j.n = static_cast<int>(c.size());
    j.kv = M.kv;
    j.n_layers = M.d.n_layers;
    j.layer_stride = M.layer_stride;
    j.v_off = M.v_off;
    j.Hkv = M.d.n_kv_heads;
    j.hd = M.d.head_dim;
    return j;
  };
  KvClearJob a = job(T, ct), b = job(D, cd);
  if (ct.size() <= static_cast<size_t>(kKvClearInline) && cd.size() <= static_cast<size_t>(kKvClearInline)) {
    // few slots (a single sequence's commit): they travel in the kernel
    // arguments, with no metadata upload before the launch
    std::copy(ct.begin(), ct.end(), a.inl);
    std::copy(cd.begin(), cd.end(), b.inl);
  } else {
    MetaBlock mb;
    const size_t ot = mb.add(ct), od = mb.add(cd);
    char* dev = nullptr;
    spec_status s = upload_meta(ctx, mb, st, &dev);
    if (s != SPEC_OK) return s;
    a.slots = reinterpret_cast<const int32_t*>(dev + ot);
    b.slots = reinterpret_cast<const int32_t*>(dev + od);
  }
  HIPC(launch_kv_clear(T.dt(), a, b, st));  // one launch for both pools
  return SPEC_OK;
}

// The accepted path of tree verifications to consecutive cache positions:
// mv holds (src, dst) slot pairs, off the group (sequence) boundaries.
spec_status launch_moves(spec_ctx* ctx, const std::vector<int32_t>& mv, const std::vector<int32_t>& off,
                         hipStream_t st) {
  if (mv.empty()) return SPEC_OK;
  MetaBlock mb;
  const size_t op = mb.add(mv), oo = mb.add(off);
  char* dev = nullptr;
  spec_status s = upload_meta(ctx, mb, st, &dev);
  if (s != SPEC_OK) return s;
  const Model& T = ctx->m[0];
  KvMoveJob j;
  j.pairs = reinterpret_cast<const int32_t*>(dev + op);
  j.off = reinterpret_cast<const int32_t*>(dev + oo);
  j.n_groups = static_cast<int>(off.size()) - 1;
  j.kv = T.kv;
  j.n_layers = T.d.n_layers;
  j.layer_stride = T.layer_stride;
  j.v_off = T.v_off;
  j.Hkv = T.d.n_kv_heads;
  j.hd = T.d.head_dim;
  HIPC(launch_kv_move(T.dt(), j, st));
  return SPEC_OK;
}

}  // namespace

extern "C" {

size_t spec_kv_pool_bytes(const spec_model_desc* m, int32_t num_pages) {
  if (!m || num_pages < 0) return 0;
  const size_t esz = m->dtype == SPEC_F32 ? 4 : 2;
  return static_cast<size_t>(m->n_layers) * pool_layer_elems(*m, num_pages) * esz;
}

spec_status spec_ctx_create(const spec_model_desc* target, const spec_model_desc* draft,
                            const spec_cache_desc* cache, spec_ctx** out) {
  std::string why;
  if (!out) { g_err = "null out"; return SPEC_E_INVALID; }
  *out = nullptr;
  const bool pair = draft != nullptr;
  if (!valid_model(target, why) || (pair && !valid_model(draft, why))) { g_err = why; return SPEC_E_INVALID; }
  if (!cache || cache->page_size != 16 || cache->num_pages_target <= 0 || cache->max_seqs <= 0 ||
      cache->max_pages_per_seq <= 0 || cache->k_max < (pair ? 1 : 0) || cache->k_max > 15 ||
      cache->max_rows <= 0 || !cache->kv_target ||
      (pair && (cache->num_pages_draft <= 0 || !cache->kv_draft))) {
    g_err = "invalid cache descriptor (page_size must be 16, k_max in 1..15 (0..15 without a draft model), "
            "pools non-null)";
    return SPEC_E_INVALID;
  }
  if (pair && (target->vocab != draft->vocab || target->dtype != draft->dtype)) {
    g_err = "target and draft must share vocab and dtype";
    return SPEC_E_INVALID;
  }
  if (unsupported_model(target, why) || (pair && unsupported_model(draft, why))) {
    g_err = why;
    return SPEC_E_UNSUPPORTED;
  }
  spec_ctx* c = new spec_ctx();
  c->n_models = pair ? 2 : 1;
  const spec_model_desc* ms[2] = {target, draft};
  void* pools[2] = {cache->kv_target, cache->kv_draft};
  const int np[2] = {cache->num_pages_target, pair ? cache->num_pages_draft : 0};
  for (int i = 0; i < c->n_models; ++i) {
    Model& M = c->m[i];
    M.d = *ms[i];
    M.layers.assign(ms[i]->layers, ms[i]->layers + ms[i]->n_layers);
    M.d.layers = nullptr;
    M.esz = M.d.dtype == SPEC_F32 ? 4 : 2;
    M.kv = static_cast<char*>(pools[i]);
    M.num_pages = np[i];
    M.layer_stride = pool_layer_elems(M.d, np[i]);
    M.v_off = M.layer_stride / 2;
    M.pool.reset(np[i], 16);
    c->d_max = std::max(c->d_max, M.d.d_model);
    c->qkv_max = std::max(c->qkv_max, M.qkvw());
    c->q_max = std::max(c->q_max, M.qdim());
    c->ffn_max = std::max(c->ffn_max, M.d.ffn_dim);
    c->hkv_max = std::max(c->hkv_max, M.d.n_kv_heads);
    c->hd_max = std::max(c->hd_max, M.d.head_dim);
    c->esz_max = std::max(c->esz_max, M.esz);
  }
  c->cache = *cache;
  c->V = target->vocab;
  c->k_max = cache->k_max;
  c->max_seqs = cache->max_seqs;
  c->max_pages = cache->max_pages_per_seq;
  c->R_max = std::max(cache->max_rows, cache->max_seqs * (cache->k_max + 1));
  for (int s = 0; s < c->max_seqs; ++s) c->free_slots.push(s);
  compute_ws(c);
  // coherent: the kernel's stores go straight to host memory
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&c->h_out),
                               sizeof(int32_t) * c->max_seqs * (2 * c->k_max + 2), hipHostMallocCoherent);
  if (e == hipSuccess) e = hipHostGetDevicePointer(reinterpret_cast<void**>(&c->h_out_dev), c->h_out, 0);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->out_ev, hipEventDisableTiming);
  if (e != hipSuccess) {
    g_err = std::string("hipHostMalloc/hipEventCreate: ") + hipGetErrorString(e);
    if (c->h_out) (void)hipHostFree(c->h_out);
    delete c;
    return SPEC_E_HIP;
  }
  *out = c;
  return SPEC_OK;
}

void spec_ctx_destroy(spec_ctx* ctx) {
  if (!ctx) return;
  (void)hipDeviceSynchronize();  // queued copies and graph launches still use ctx resources
  ctx->drop_graphs();
  if (ctx->cap_stream) (void)hipStreamDestroy(ctx->cap_stream);
  ctx->stager.release();
  if (ctx->h_out) (void)hipHostFree(ctx->h_out);
  if (ctx->out_ev) (void)hipEventDestroy(ctx->out_ev);
  delete ctx;
}

const char* spec_last_error(const spec_ctx* ctx) { return ctx ? ctx->err.c_str() : g_err.c_str(); }

size_t spec_workspace_bytes(const spec_ctx* ctx) { return ctx ? ctx->ws.total : 0; }

spec_status spec_set_workspace(spec_ctx* ctx, void* dev_ptr, size_t bytes) {
  if (!ctx) return SPEC_E_INVALID;
  if (!dev_ptr || bytes < ctx->ws.total || (reinterpret_cast<uintptr_t>(dev_ptr) & 255))
    FAIL(SPEC_E_INVALID, "workspace null, too small or not 256-byte aligned");
  if (ctx->wsp != dev_ptr) {
    // captured graphs hold workspace addresses
    if (ctx->wsp) (void)hipDeviceSynchronize();
    ctx->drop_graphs();
  }
  ctx->wsp = static_cast<char*>(dev_ptr);
  ctx->ws_bytes = bytes;
  return SPEC_OK;
}

#define CHECK_READY()                                                    \
  do {                                                                   \
    if (!ctx) return SPEC_E_INVALID;                                     \
    if (ctx->broken) FAIL(SPEC_E_HIP, "context unusable after a HIP error"); \
    if (!ctx->wsp) FAIL(SPEC_E_STATE, "spec_set_workspace not called");  \
  } while (0)

spec_status spec_prefill(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const int32_t* prompt_lens,
                         const int32_t* tokens, void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n < 0 || (n > 0 && (!seq_ids || !prompt_lens || !tokens))) FAIL(SPEC_E_INVALID, "bad arguments");
  if (!check_ids(ctx, n, seq_ids, false)) return SPEC_E_INVALID;
  int need_t = 0, need_d = 0;
  for (int i = 0; i < n; ++i) {
    if (ctx->seqs.count(seq_ids[i])) FAIL(SPEC_E_INVALID, "seq_id already live");
    const int P = prompt_lens[i];
    if (P < 1) FAIL(SPEC_E_INVALID, "prompt_lens must be >= 1");
    if (ctx->m[0].pool.pages_for(P + ctx->k_max + 1) > ctx->max_pages)
      FAIL(SPEC_E_INVALID, "prompt too long for max_pages_per_seq");
    need_t += ctx->m[0].pool.pages_for(P - 1);
    if (ctx->n_models == 2) need_d += ctx->m[1].pool.pages_for(P - 1);
  }
  if (static_cast<int>(ctx->free_slots.size()) < n) FAIL(SPEC_E_INVALID, "more live sequences than max_seqs");
  if (need_t > ctx->m[0].pool.free_pages() || need_d > ctx->m[1].pool.free_pages())
    FAIL(SPEC_E_NOPAGES, "KV page pool exhausted");
  {
    size_t off = 0;
    for (int i = 0; i < n; ++i) {
      for (int j = 0; j < prompt_lens[i]; ++j)
        if (tokens[off + j] < 0 || tokens[off + j] >= ctx->V) FAIL(SPEC_E_INVALID, "token id out of range");
      off += prompt_lens[i];
    }
  }
  // commit host state
  std::vector<Seq*> ss;
  size_t off = 0;
  for (int i = 0; i < n; ++i) {
    Seq s;
    s.id = seq_ids[i];
    s.slot = ctx->free_slots.top();
    ctx->free_slots.pop();
    s.hist.assign(tokens + off, tokens + off + prompt_lens[i]);
    off += prompt_lens[i];
    const int P = prompt_lens[i];
    ctx->m[0].pool.ensure(s.pages_t, P - 1);
    if (ctx->n_models == 2) ctx->m[1].pool.ensure(s.pages_d, P - 1);
    s.len_t = s.written_t = P - 1;
    s.len_d = ctx->n_models == 2 ? P - 1 : 0;
    ss.push_back(&(ctx->seqs[s.id] = std::move(s)));
  }
  // chunked forward of positions 0..P-2 through both models
  struct Piece { Seq* s; int pos0, nrows; };
  std::vector<Piece> pieces;
  for (Seq* s : ss)
    for (int p = 0; p < s->len_t; p += ctx->R_max)
      pieces.push_back(Piece{s, p, std::min(ctx->R_max, s->len_t - p)});
  size_t pi = 0;
  while (pi < pieces.size()) {
    std::vector<Piece> chunk;
    int rows = 0;
    while (pi < pieces.size() && rows + pieces[pi].nrows <= ctx->R_max) {
      chunk.push_back(pieces[pi]);
      rows += pieces[pi].nrows;
      ++pi;
    }
    for (int mi = 0; mi < ctx->n_models; ++mi) {
      const Model& M = ctx->m[mi];
      Fwd f;
      std::vector<const std::vector<int32_t>*> tabs;
      for (size_t c = 0; c < chunk.size(); ++c) {
        const Piece& p = chunk[c];
        const auto& tab = mi == 0 ? p.s->pages_t : p.s->pages_d;
        tabs.push_back(&tab);
        f.segs.push_back(AttnSegment{static_cast<int32_t>(c), static_cast<int32_t>(f.tok_src.size()),
                                     p.nrows, p.pos0});
        for (int r = 0; r < p.nrows; ++r) {
          const int pos = p.pos0 + r;
          f.tok_src.push_back(p.s->hist[pos]);
          f.pos.push_back(pos);
          f.slot.push_back(M.pool.slot(tab, pos));
          f.seqi.push_back(static_cast<int32_t>(c));
        }
      }
      build_ptab(tabs, f, 1);
      MetaBlock mb;
      FwdOff o = add_forward(ctx, M, f, mb);
      char* dev = nullptr;
      spec_status s = upload_meta(ctx, mb, st, &dev);
      if (s != SPEC_OK) return s;
      s = launch_forward(ctx, M, o, dev, nullptr, st);
      if (s != SPEC_OK) return s;
    }
  }
  HIPC(hipStreamSynchronize(st));
  ctx->timer.flush();
  return SPEC_OK;
}

namespace {

spec_status draft_step_impl(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                            uint64_t seed, const int32_t* guide, float boost, void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n < 0 || (n > 0 && (!seq_ids || !temperature))) FAIL(SPEC_E_INVALID, "bad arguments");
  if (n == 0) return SPEC_OK;
  if (ctx->n_models < 2) FAIL(SPEC_E_STATE, "context has no draft model");
  if (!check_ids(ctx, n, seq_ids, true)) return SPEC_E_INVALID;
  Model& D = ctx->m[1];
  int rows = 0, need = 0;
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    if (!(temperature[i] >= 0.f)) FAIL(SPEC_E_INVALID, "temperature must be >= 0");
    if (s.verified) FAIL(SPEC_E_STATE, "draft step after verify without commit");
    if (s.external) FAIL(SPEC_E_STATE, "sequence holds external drafts");
    if (s.k >= ctx->k_max) FAIL(SPEC_E_STATE, "sequence already has k_max drafts");
    const int c = s.k == 0 ? s.n() + 1 - s.len_d : 1;
    rows += c;
    if (D.pool.pages_for(s.len_d + c) > ctx->max_pages) FAIL(SPEC_E_INVALID, "sequence exceeds max_pages_per_seq");
    need += D.pool.need(s.pages_d, s.len_d + c);
  }
  if (rows > ctx->R_max) FAIL(SPEC_E_UNSUPPORTED, "draft rows exceed max_rows");
  if (need > D.pool.free_pages()) FAIL(SPEC_E_NOPAGES, "draft KV page pool exhausted");
  Fwd f;
  std::vector<const std::vector<int32_t>*> tabs;
  std::vector<DRow> dr;
  float* dq = wsptr<float>(ctx, ctx->ws.dq);
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    const int c = s.k == 0 ? s.n() + 1 - s.len_d : 1;
    D.pool.ensure(s.pages_d, s.len_d + c);
    tabs.push_back(&s.pages_d);
    f.segs.push_back(AttnSegment{i, static_cast<int32_t>(f.tok_src.size()), c, s.len_d});
    for (int r = 0; r < c; ++r) {
      const int pos = s.len_d + r;
      f.tok_src.push_back(s.k == 0 ? s.hist[pos] : s.dsrc[s.k - 1]);
      f.pos.push_back(pos);
      f.slot.push_back(D.pool.slot(s.pages_d, pos));
      f.seqi.push_back(i);
    }
    const int qidx = s.slot * ctx->k_max + s.k;
    f.lm_rows.push_back(static_cast<int32_t>(f.tok_src.size()) - 1);
    f.lm_map.push_back(qidx);
    DRow d{};
    d.ptr = dq + static_cast<size_t>(qidx) * ctx->V;
    d.t = temperature[i];
    d.pos = s.n() + s.k + 1;
    d.seq_lo = static_cast<uint32_t>(static_cast<uint64_t>(s.id));
    d.seq_hi = static_cast<uint32_t>(static_cast<uint64_t>(s.id) >> 32);
    d.out = qidx;
    d.guide = guide ? guide[i] : -1;
    dr.push_back(d);
  }
  build_ptab(tabs, f, ctx->max_pages);
  MetaBlock mb;
  FwdOff o = add_forward(ctx, D, f, mb);
  const size_t odr = mb.add(dr);
  const size_t osd = mb.add(&seed, 1);
  uint32_t boost_bits = 0;
  std::memcpy(&boost_bits, &boost, sizeof(boost_bits));
  std::vector<int64_t> key = {1, n, static_cast<int64_t>(odr), static_cast<int64_t>(osd), guide ? 1 : 0,
                              static_cast<int64_t>(boost_bits)};
  key_forward(key, o);
  spec_status s = run_kernels(ctx, key, o.R, mb, st, [&](const char* dev, hipStream_t ls) -> spec_status {
    spec_status r = launch_forward(ctx, D, o, dev, dq, ls);
    if (r != SPEC_OK) return r;
    if (guide) HIPC(launch_draft_guide(n, ctx->V, reinterpret_cast<const DRow*>(dev + odr), boost, ls));
    HIPC(launch_draft_sample(draft_plan(n, ctx->V), reinterpret_cast<const DRow*>(dev + odr), seed,
                             wsptr<int32_t>(ctx, ctx->ws.dtok), ctx->wsp + ctx->ws.draft, ls,
                             reinterpret_cast<const uint64_t*>(dev + osd)));
    return SPEC_OK;
  });
  if (s != SPEC_OK) return s;
  for (int i = 0; i < n; ++i) {
    Seq& q = ctx->seqs[seq_ids[i]];
    const int c = q.k == 0 ? q.n() + 1 - q.len_d : 1;
    const int qidx = q.slot * ctx->k_max + q.k;
    q.len_d += c;
    q.qrow.push_back(dq + static_cast<size_t>(qidx) * ctx->V);
    q.dsrc.push_back(dev_tok_ref(q.slot, ctx->k_max, q.k));
    q.k += 1;
  }
  return SPEC_OK;
}

// Draft steps 0 .. max(steps) - 1 of the listed sequences (sequence i in the
// first steps[i]) as one graph, from the sequences' current state.  Callers
// have validated the call and taken the pages of every step.  Each step is
// the draft step above; since each step's token sources are the previous
// step's device draws, the host lays all steps out at once: the page table is
// shared by the steps and the metadata goes up in one block.  Metadata over
// the call bound runs one draft_step_impl call per step instead.
spec_status draft_steps_graph(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                              uint64_t seed, const int32_t* steps, hipStream_t st) {
  Model& D = ctx->m[1];
  int n_steps = 0;
  std::vector<int> first(n);  // rows of the sequence's first step (catch-up rows after a commit)
  for (int i = 0; i < n; ++i) {
    const Seq& s = ctx->seqs[seq_ids[i]];
    first[i] = s.k == 0 ? s.n() + 1 - s.len_d : 1;
    n_steps = std::max(n_steps, steps[i]);
  }
  if (n_steps == 0) return SPEC_OK;
  std::vector<const std::vector<int32_t>*> tabs;
  for (int i = 0; i < n; ++i) tabs.push_back(&ctx->seqs[seq_ids[i]].pages_d);
  float* dq = wsptr<float>(ctx, ctx->ws.dq);
  MetaBlock mb;
  std::vector<FwdOff> fo(n_steps);
  std::vector<size_t> odr(n_steps);
  std::vector<int> nrow(n_steps);
  for (int j = 0; j < n_steps; ++j) {
    Fwd f;
    std::vector<DRow> dr;
    for (int i = 0; i < n; ++i) {
      if (steps[i] <= j) continue;
      const Seq& s = ctx->seqs[seq_ids[i]];
      const int k = s.k + j;                                           // drafts before this step
      const int len = j == 0 ? s.len_d : s.len_d + first[i] + j - 1;  // draft cache length
      const int c = j == 0 ? first[i] : 1;
      f.segs.push_back(AttnSegment{i, static_cast<int32_t>(f.tok_src.size()), c, len});
      for (int r = 0; r < c; ++r) {
        const int pos = len + r;
        f.tok_src.push_back(k == 0 ? s.hist[pos] : (k - 1 < s.k ? s.dsrc[k - 1] : dev_tok_ref(s.slot, ctx->k_max, k - 1)));
        f.pos.push_back(pos);
        f.slot.push_back(D.pool.slot(s.pages_d, pos));
        f.seqi.push_back(i);
      }
      const int qidx = s.slot * ctx->k_max + k;
      f.lm_rows.push_back(static_cast<int32_t>(f.tok_src.size()) - 1);
      f.lm_map.push_back(qidx);
      DRow d{};
      d.ptr = dq + static_cast<size_t>(qidx) * ctx->V;
      d.t = temperature[i];
      d.pos = s.n() + k + 1;
      d.seq_lo = static_cast<uint32_t>(static_cast<uint64_t>(s.id));
      d.seq_hi = static_cast<uint32_t>(static_cast<uint64_t>(s.id) >> 32);
      d.out = qidx;
      d.guide = -1;
      dr.push_back(d);
    }
    if (j == 0) build_ptab(tabs, f, ctx->max_pages);
    fo[j] = add_forward(ctx, D, f, mb);
    if (j > 0) {  // the page table of step 0 (row i = sequence i) serves every step
      fo[j].pt = fo[0].pt;
      fo[j].ptab_stride = fo[0].ptab_stride;
    }
    odr[j] = mb.add(dr);
    nrow[j] = static_cast<int>(dr.size());
  }
  const size_t osd = mb.add(&seed, 1);
  if (mb.size() > ctx->ws.meta_cap) {
    for (int j = 0; j < n_steps; ++j) {
      std::vector<int64_t> ids;
      std::vector<float> ts;
      for (int i = 0; i < n; ++i)
        if (steps[i] > j) {
          ids.push_back(seq_ids[i]);
          ts.push_back(temperature[i]);
        }
      spec_status r = draft_step_impl(ctx, static_cast<int32_t>(ids.size()), ids.data(), ts.data(), seed,
                                      nullptr, 0.f, st);
      if (r != SPEC_OK) return r;
    }
    return SPEC_OK;
  }
  std::vector<int64_t> key = {3, n, n_steps, static_cast<int64_t>(osd)};
  int max_rows = 0;
  for (int j = 0; j < n_steps; ++j) {
    key.push_back(static_cast<int64_t>(odr[j]));
    key.push_back(nrow[j]);
    key_forward(key, fo[j]);
    max_rows = std::max(max_rows, fo[j].R);
  }
  spec_status s = run_kernels(ctx, key, max_rows, mb, st, [&](const char* dev, hipStream_t ls) -> spec_status {
    for (int j = 0; j < n_steps; ++j) {
      spec_status r = launch_forward(ctx, D, fo[j], dev, dq, ls);
      if (r != SPEC_OK) return r;
      HIPC(launch_draft_sample(draft_plan(nrow[j], ctx->V), reinterpret_cast<const DRow*>(dev + odr[j]), seed,
                               wsptr<int32_t>(ctx, ctx->ws.dtok), ctx->wsp + ctx->ws.draft, ls,
                               reinterpret_cast<const uint64_t*>(dev + osd)));
    }
    return SPEC_OK;
  });
  if (s != SPEC_OK) return s;
  for (int i = 0; i < n; ++i) {
    Seq& q = ctx->seqs[seq_ids[i]];
    for (int j = 0; j < steps[i]; ++j) {
      const int qidx = q.slot * ctx->k_max + q.k;
      q.len_d += j == 0 ? first[i] : 1;
      q.qrow.push_back(dq + static_cast<size_t>(qidx) * ctx->V);
      q.dsrc.push_back(dev_tok_ref(q.slot, ctx->k_max, q.k));
      q.k += 1;
    }
  }
  return SPEC_OK;
}

// Several draft steps in one call: validated as a whole (an error runs no
// step), the pages of every step taken in list order, then step 0 on its own
// graph, so that the GPU starts while the host lays out the later steps, and
// steps 1 .. on one graph.
spec_status draft_loop_impl(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                            uint64_t seed, const int32_t* steps, void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n < 0 || (n > 0 && (!seq_ids || !temperature || !steps))) FAIL(SPEC_E_INVALID, "bad arguments");
  if (n == 0) return SPEC_OK;
  if (!check_ids(ctx, n, seq_ids, true)) return SPEC_E_INVALID;
  Model& D = ctx->m[1];
  int n_steps = 0, need = 0;
  std::vector<int> first(n), total(n);  // rows of the first step, rows over all steps
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    if (!(temperature[i] >= 0.f)) FAIL(SPEC_E_INVALID, "temperature must be >= 0");
    if (steps[i] < 0) FAIL(SPEC_E_INVALID, "steps must be >= 0");
    if (steps[i] == 0) continue;
    if (s.verified) FAIL(SPEC_E_STATE, "draft step after verify without commit");
    if (s.external) FAIL(SPEC_E_STATE, "sequence holds external drafts");
    if (s.k + steps[i] > ctx->k_max) FAIL(SPEC_E_STATE, "steps would exceed k_max drafts");
    first[i] = s.k == 0 ? s.n() + 1 - s.len_d : 1;
    total[i] = first[i] + steps[i] - 1;
    if (D.pool.pages_for(s.len_d + total[i]) > ctx->max_pages)
      FAIL(SPEC_E_INVALID, "sequence exceeds max_pages_per_seq");
    need += D.pool.need(s.pages_d, s.len_d + total[i]);
    n_steps = std::max(n_steps, steps[i]);
  }
  if (n_steps == 0) return SPEC_OK;
  if (ctx->n_models < 2) FAIL(SPEC_E_STATE, "context has no draft model");
  for (int j = 0; j < n_steps; ++j) {
    int rows = 0;
    for (int i = 0; i < n; ++i)
      if (steps[i] > j) rows += j == 0 ? first[i] : 1;
    if (rows > ctx->R_max) FAIL(SPEC_E_UNSUPPORTED, "draft rows exceed max_rows");
  }
  if (need > D.pool.free_pages()) FAIL(SPEC_E_NOPAGES, "draft KV page pool exhausted");
  for (int i = 0; i < n; ++i)
    if (steps[i] > 0) D.pool.ensure(ctx->seqs[seq_ids[i]].pages_d, ctx->seqs[seq_ids[i]].len_d + total[i]);
  std::vector<int32_t> one(n), rest(n);
  for (int i = 0; i < n; ++i) {
    one[i] = std::min(steps[i], 1);
    rest[i] = steps[i] - one[i];
  }
  spec_status s = draft_steps_graph(ctx, n, seq_ids, temperature, seed, one.data(), st);
  if (s != SPEC_OK) return s;
  return draft_steps_graph(ctx, n, seq_ids, temperature, seed, rest.data(), st);
}

}  // namespace

spec_status spec_draft_step(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                            uint64_t seed, void* stream) {
  return draft_step_impl(ctx, n, seq_ids, temperature, seed, nullptr, 0.f, stream);
}

spec_status spec_draft_loop(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                            uint64_t seed, const int32_t* steps, void* stream) {
  return draft_loop_impl(ctx, n, seq_ids, temperature, seed, steps, stream);
}

spec_status spec_draft_step_guided(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                                   uint64_t seed, const int32_t* guide, float boost, void* stream) {
  if (ctx && n > 0 && !guide) FAIL(SPEC_E_INVALID, "guide tokens missing");
  if (ctx && !(boost >= 0.f)) FAIL(SPEC_E_INVALID, "boost must be >= 0");
  return draft_step_impl(ctx, n, seq_ids, temperature, seed, guide, boost, stream);
}

spec_status spec_set_drafts(spec_ctx* ctx, int64_t seq_id, int32_t k, const int32_t* tokens,
                            const float* q_logits, void* stream) {
  CHECK_READY();
  (void)stream;
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) FAIL(SPEC_E_INVALID, "unknown seq_id");
  Seq& s = it->second;
  if (k < 0 || k > ctx->k_max || (k > 0 && (!tokens || !q_logits))) FAIL(SPEC_E_INVALID, "bad drafts");
  if (s.verified) FAIL(SPEC_E_STATE, "set_drafts after verify without commit");
  if (s.k > 0 && !s.external) FAIL(SPEC_E_STATE, "sequence already has drafts from spec_draft_step");
  for (int j = 0; j < k; ++j)
    if (tokens[j] < 0 || tokens[j] >= ctx->V) FAIL(SPEC_E_INVALID, "draft token out of range");
  if (k > 0 && ctx->V % 4 == 0 && (reinterpret_cast<uintptr_t>(q_logits) & 15))
    FAIL(SPEC_E_INVALID, "draft logits must be 16-byte aligned");
  s.k = k;
  s.external = k > 0;
  s.qrow.clear();
  s.dsrc.clear();
  s.tparent.clear();
  for (int j = 0; j < k; ++j) {
    s.qrow.push_back(q_logits + static_cast<size_t>(j) * ctx->V);
    s.dsrc.push_back(tokens[j]);
  }
  return SPEC_OK;
}

spec_status spec_set_draft_tree(spec_ctx* ctx, int64_t seq_id, int32_t m, const int32_t* parents,
                                const int32_t* tokens, const float* q_logits, void* stream) {
  CHECK_READY();
  (void)stream;
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) FAIL(SPEC_E_INVALID, "unknown seq_id");
  Seq& s = it->second;
  if (m < 1 || m > ctx->k_max || !parents || !tokens || !q_logits) FAIL(SPEC_E_INVALID, "bad draft tree");
  if (s.verified) FAIL(SPEC_E_STATE, "set_draft_tree after verify without commit");
  if (s.k > 0 && !s.external) FAIL(SPEC_E_STATE, "sequence already has drafts from spec_draft_step");
  for (int i = 0; i < m; ++i) {
    if (parents[i] < -1 || parents[i] >= i) FAIL(SPEC_E_INVALID, "parents[i] must be in -1 .. i - 1");
    if (tokens[i] < 0 || tokens[i] >= ctx->V) FAIL(SPEC_E_INVALID, "draft token out of range");
  }
  if (ctx->V % 4 == 0 && (reinterpret_cast<uintptr_t>(q_logits) & 15))
    FAIL(SPEC_E_INVALID, "draft logits must be 16-byte aligned");
  s.k = m;
  s.external = true;
  s.qrow.clear();
  s.dsrc.clear();
  for (int i = 0; i <= m; ++i) s.qrow.push_back(q_logits + static_cast<size_t>(i) * ctx->V);
  s.dsrc.assign(tokens, tokens + m);
  s.tparent.assign(parents, parents + m);
  return SPEC_OK;
}

namespace {

// The verify's target forward; with `decide` also the decision pass and the
// outputs' copy to the host (the verify), else logits only.
spec_status verify_impl(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                        uint64_t seed, int32_t* n_accepted, int32_t* out_tokens, bool decide, void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n < 0 || (n > 0 && (!seq_ids || (decide && (!temperature || !n_accepted || !out_tokens)))))
    FAIL(SPEC_E_INVALID, "bad arguments");
  if (n == 0) return SPEC_OK;
  if (!check_ids(ctx, n, seq_ids, true)) return SPEC_E_INVALID;
  Model& T = ctx->m[0];
  int need = 0;
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    if (decide && !(temperature[i] >= 0.f)) FAIL(SPEC_E_INVALID, "temperature must be >= 0");
    if (s.verified) FAIL(SPEC_E_STATE, "verify twice without commit");
    if (T.pool.pages_for(s.n() + s.k + 1) > ctx->max_pages) FAIL(SPEC_E_INVALID, "sequence exceeds max_pages_per_seq");
    need += T.pool.need(s.pages_t, s.n() + s.k + 1);
  }
  if (need > T.pool.free_pages()) FAIL(SPEC_E_NOPAGES, "target KV page pool exhausted");
  // a batch with a draft tree runs the tree-masked attention and the tree
  // decision for all of its sequences (a chain is the tree parents[i] = i - 1)
  bool tree_mode = false;
  int R_all = 0;  // rows of the call: the tree decision's q rows follow them
  for (int i = 0; i < n; ++i) {
    tree_mode = tree_mode || !ctx->seqs[seq_ids[i]].tparent.empty();
    R_all += ctx->seqs[seq_ids[i]].k + 1;
  }
  Fwd f;
  std::vector<const std::vector<int32_t>*> tabs;
  std::vector<VRow> prow, qrow, tq;
  std::vector<VSeq> vs;
  std::vector<VTreeSeq> ts;
  std::vector<VTreeNode> tn;
  int max_kids = 0;  // the most children of any tree node: residual-mass levels of the tree pass
  float* logits = wsptr<float>(ctx, ctx->ws.logits);
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    const int nn = s.n();
    T.pool.ensure(s.pages_t, nn + s.k + 1);
    // parent and depth of each draft node (chain: the previous draft)
    std::vector<int32_t> par(s.k), dep(s.k);
    std::vector<uint32_t> anc(s.k);
    for (int j = 0; j < s.k; ++j) {
      par[j] = s.tparent.empty() ? j - 1 : s.tparent[j];
      dep[j] = par[j] < 0 ? 1 : dep[par[j]] + 1;
      anc[j] = (par[j] < 0 ? 0u : anc[par[j]]) | (1u << j);
    }
    tabs.push_back(&s.pages_t);
    const int row0 = static_cast<int>(f.tok_src.size());
    f.segs.push_back(AttnSegment{i, row0, s.k + 1, nn});
    const float t = decide ? temperature[i] : 1.f;
    const float it = t > 0.f ? 1.f / t : 0.f;
    VSeq q{};
    q.k = s.k;
    q.p_row = row0;
    q.q_row = static_cast<int32_t>(qrow.size());
    q.tok_row = row0 + 1;
    q.base_pos = nn;
    q.t = t;
    q.seq_lo = static_cast<uint32_t>(static_cast<uint64_t>(s.id));
    q.seq_hi = static_cast<uint32_t>(static_cast<uint64_t>(s.id) >> 32);
    vs.push_back(q);
    // row r: the pending token (r = 0) or draft node r - 1, at position n +
    // its depth; its K/V go to cache index n + r
    for (int r = 0; r <= s.k; ++r) {
      f.tok_src.push_back(r == 0 ? s.hist[nn] : s.dsrc[r - 1]);
      f.pos.push_back(nn + (r == 0 ? 0 : dep[r - 1]));
      f.slot.push_back(T.pool.slot(s.pages_t, nn + r));
      f.seqi.push_back(i);
      f.lm_rows.push_back(row0 + r);
      if (tree_mode) {
        f.tbase.push_back(nn);
        f.tmask.push_back(r == 0 ? 0u : anc[r - 1]);
      }
      prow.push_back(VRow{logits + static_cast<size_t>(row0 + r) * ctx->V, it, t > 0.f ? 0 : 1});
    }
    if (tree_mode) {
      // q row of a node with children: the row its children were drawn from
      // (chain drafts: draft j + 1's row for node j - 1; trees: row u + 1)
      std::vector<int> kids(s.k + 1, 0);
      for (int j = 0; j < s.k; ++j) ++kids[par[j] + 1];
      for (int c : kids) max_kids = std::max(max_kids, c);
      auto qidx = [&](int u) -> int32_t {  // u = -1: the root
        if (!kids[u + 1]) return -1;
        tq.push_back(VRow{s.qrow[u + 1], it, t > 0.f ? 0 : 1});
        return R_all + static_cast<int32_t>(tq.size()) - 1;
      };
      VTreeSeq tsq{};
      tsq.m = s.k;
      tsq.node0 = static_cast<int32_t>(tn.size());
      tsq.p_row = row0;
      tsq.q_row = qidx(-1);
      tsq.base_pos = nn;
      tsq.t = t;
      tsq.seq_lo = q.seq_lo;
      tsq.seq_hi = q.seq_hi;
      ts.push_back(tsq);
      for (int j = 0; j < s.k; ++j) tn.push_back(VTreeNode{par[j], row0 + 1 + j, qidx(j), 0});
    } else {
      for (int j = 0; j < s.k; ++j) qrow.push_back(VRow{s.qrow[j], it, t > 0.f ? 0 : 1});
    }
    s.written_t = std::max(s.written_t, nn + s.k + 1);
  }
  const int R = static_cast<int>(f.tok_src.size());
  for (auto& q : vs) q.q_row += R;
  std::vector<VRow> rows = prow;
  rows.insert(rows.end(), qrow.begin(), qrow.end());
  rows.insert(rows.end(), tq.begin(), tq.end());
  build_ptab(tabs, f, ctx->max_pages);
  MetaBlock mb;
  FwdOff o = add_forward(ctx, T, f, mb);
  const size_t orow = mb.add(rows), oseq = tree_mode ? mb.add(ts) : mb.add(vs);
  const size_t onode = mb.add(tn);
  const size_t osd = mb.add(&seed, 1);
  // the decision pass writes its outputs into pinned host memory (no copies)
  int32_t* d_nacc = ctx->h_out_dev;
  int32_t* d_otok = ctx->h_out_dev + ctx->max_seqs;
  int32_t* d_opath = ctx->h_out_dev + ctx->max_seqs * (ctx->k_max + 2);
  const VocabPlan vp = vocab_plan(n, static_cast<int>(rows.size()), ctx->V);
  std::vector<int64_t> key = {decide ? 0 : 2, n, static_cast<int64_t>(rows.size()), static_cast<int64_t>(orow),
                              static_cast<int64_t>(oseq), static_cast<int64_t>(osd), tree_mode, max_kids,
                              static_cast<int64_t>(onode)};
  key_forward(key, o);
  spec_status s = run_kernels(ctx, key, o.R, mb, st, [&](const char* dev, hipStream_t ls) -> spec_status {
    spec_status r = launch_forward(ctx, T, o, dev, logits, ls);
    if (r != SPEC_OK || !decide) return r;
    if (tree_mode) {
      HIPC(launch_tree_pass(vp, reinterpret_cast<const VRow*>(dev + orow),
                            reinterpret_cast<const VTreeSeq*>(dev + oseq),
                            reinterpret_cast<const VTreeNode*>(dev + onode), wsptr<int32_t>(ctx, ctx->ws.rowtok),
                            seed, reinterpret_cast<const uint64_t*>(dev + osd), ctx->k_max, max_kids, d_nacc, d_otok,
                            d_opath, ctx->wsp + ctx->ws.vocab, ls, &ctx->timer));
      return SPEC_OK;
    }
    HIPC(launch_vocab_pass(vp, reinterpret_cast<const VRow*>(dev + orow),
                           reinterpret_cast<const VSeq*>(dev + oseq), wsptr<int32_t>(ctx, ctx->ws.rowtok),
                           seed, ctx->k_max, d_nacc, d_otok, ctx->wsp + ctx->ws.vocab, ls, &ctx->timer,
                           reinterpret_cast<const uint64_t*>(dev + osd)));
    return SPEC_OK;
  });
  if (s != SPEC_OK) return s;
  ctx->last_rows = R;
  if (!decide) return SPEC_OK;
  const int W = ctx->k_max + 1;
  HIPC(hipEventRecord(ctx->out_ev, st));
  // poll instead of sleeping in hipEventSynchronize: the next draft step waits
  // on this host round trip, and a blocking wait adds its wake-up to it
  for (;;) {
    const hipError_t q = hipEventQuery(ctx->out_ev);
    if (q == hipSuccess) break;
    if (q != hipErrorNotReady) HIPC(q);
  }
  std::memcpy(n_accepted, ctx->h_out, sizeof(int32_t) * n);
  std::memcpy(out_tokens, ctx->h_out + ctx->max_seqs, sizeof(int32_t) * n * W);
  const int32_t* h_path = ctx->h_out + ctx->max_seqs * (ctx->k_max + 2);
  for (int i = 0; i < n; ++i) {
    Seq& q = ctx->seqs[seq_ids[i]];
    q.verified = true;
    q.a_ver = n_accepted[i];
    q.emitted.assign(out_tokens + i * W, out_tokens + i * W + q.a_ver + 1);
    if (tree_mode)
      q.tpath.assign(h_path + static_cast<size_t>(i) * ctx->k_max, h_path + static_cast<size_t>(i) * ctx->k_max + q.a_ver);
    else
      q.tpath.clear();
  }
  ctx->timer.flush();
  return SPEC_OK;
}

}  // namespace

spec_status spec_verify(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                        uint64_t seed, int32_t* n_accepted, int32_t* out_tokens, void* stream) {
  return verify_impl(ctx, n, seq_ids, temperature, seed, n_accepted, out_tokens, true, stream);
}

spec_status spec_target_forward(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, void* stream) {
  return verify_impl(ctx, n, seq_ids, nullptr, 0, nullptr, nullptr, false, stream);
}

spec_status spec_draft_logits(const spec_ctx* ctx, int64_t seq_id, int32_t j, const float** row) {
  if (!ctx || !row) return SPEC_E_INVALID;
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end() || j < 0 || j >= it->second.k) return SPEC_E_INVALID;
  *row = it->second.qrow[j];
  return SPEC_OK;
}

spec_status spec_draft_tokens(spec_ctx* ctx, int64_t seq_id, int32_t* tokens, int32_t* k, void* stream) {
  CHECK_READY();
  if (!tokens || !k) FAIL(SPEC_E_INVALID, "bad arguments");
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) FAIL(SPEC_E_INVALID, "unknown seq_id");
  const Seq& s = it->second;
  HIPC(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  const int32_t* pool = wsptr<int32_t>(ctx, ctx->ws.dtok);
  for (int j = 0; j < s.k; ++j) {
    if (s.dsrc[j] >= 0) {
      tokens[j] = s.dsrc[j];
    } else {
      HIPC(hipMemcpy(tokens + j, pool + (-1 - s.dsrc[j]), sizeof(int32_t), hipMemcpyDeviceToHost));
    }
  }
  *k = s.k;
  return SPEC_OK;
}

spec_status spec_set_graphs(spec_ctx* ctx, int32_t enable) {
  if (!ctx) return SPEC_E_INVALID;
  ctx->use_graphs = enable != 0;
  return SPEC_OK;
}

spec_status spec_timing_enable(spec_ctx* ctx, const char* kernel_name) {
  EventTimer& t = ctx ? ctx->timer : global_timer();
  t.reset(kernel_name);
  return SPEC_OK;
}

spec_status spec_timing_read(spec_ctx* ctx, double* total_ms, int64_t* launches, double* bytes,
                             double* flops) {
  EventTimer& t = ctx ? ctx->timer : global_timer();
  t.flush();
  if (total_ms) *total_ms = t.ms;
  if (launches) *launches = t.launches;
  if (bytes) *bytes = t.bytes;
  if (flops) *flops = t.flops;
  return SPEC_OK;
}

spec_status spec_kv_commit(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const int32_t* n_accepted,
                           void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n < 0 || (n > 0 && (!seq_ids || !n_accepted))) FAIL(SPEC_E_INVALID, "bad arguments");
  if (!check_ids(ctx, n, seq_ids, true)) return SPEC_E_INVALID;
  for (int i = 0; i < n; ++i) {
    const Seq& s = ctx->seqs[seq_ids[i]];
    if (!s.verified) FAIL(SPEC_E_STATE, "commit without verify");
    if (n_accepted[i] < 0 || n_accepted[i] > s.a_ver) FAIL(SPEC_E_INVALID, "n_accepted outside 0..verified count");
  }
  std::vector<int32_t> ct, cd, mv, moff{0};
  for (int i = 0; i < n; ++i) {
    Seq& s = ctx->seqs[seq_ids[i]];
    const int a = n_accepted[i];
    const int nn = s.n();
    // a tree's accepted nodes sit at cache indices n + 1 + node: they move to
    // n + 1 .. n + a, in order (an earlier move never overwrites a later source)
    for (int j = 0; j < a && j < static_cast<int>(s.tpath.size()); ++j)
      if (s.tpath[j] != j) {
        mv.push_back(ctx->m[0].pool.slot(s.pages_t, nn + 1 + s.tpath[j]));
        mv.push_back(ctx->m[0].pool.slot(s.pages_t, nn + 1 + j));
      }
    if (static_cast<int>(mv.size()) / 2 > moff.back()) moff.push_back(static_cast<int32_t>(mv.size() / 2));
    s.hist.insert(s.hist.end(), s.emitted.begin(), s.emitted.begin() + a + 1);
    const int new_t = nn + a + 1;
    const int new_d = std::min(s.len_d, new_t);
    for (int p = new_t; p < s.written_t; ++p) ct.push_back(ctx->m[0].pool.slot(s.pages_t, p));
    for (int p = new_d; p < s.len_d; ++p) cd.push_back(ctx->m[1].pool.slot(s.pages_d, p));
    ctx->m[0].pool.truncate(s.pages_t, new_t);
    ctx->m[1].pool.truncate(s.pages_d, new_d);
    s.len_t = s.written_t = new_t;
    s.len_d = new_d;
    s.k = 0;
    s.qrow.clear();
    s.dsrc.clear();
    s.external = false;
    s.verified = false;
    s.emitted.clear();
    s.tparent.clear();
    s.tpath.clear();
  }
  spec_status r = launch_moves(ctx, mv, moff, st);
  if (r != SPEC_OK) return r;
  return launch_clears(ctx, ct, cd, st);
}

spec_status spec_verify_commit_draft(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                                     uint64_t verify_seed, int32_t* n_accepted, int32_t* out_tokens,
                                     uint64_t draft_seed, const int32_t* steps, void* stream) {
  if (!ctx || (n > 0 && !steps)) return SPEC_E_INVALID;
  spec_status s = spec_verify(ctx, n, seq_ids, temperature, verify_seed, n_accepted, out_tokens, stream);
  if (s != SPEC_OK) return s;
  s = spec_kv_commit(ctx, n, seq_ids, n_accepted, stream);
  if (s != SPEC_OK) return s;
  return spec_draft_loop(ctx, n, seq_ids, temperature, draft_seed, steps, stream);
}

spec_status spec_decode(spec_ctx* ctx, int32_t n, const int64_t* seq_ids, const float* temperature,
                        uint64_t seed, int32_t steps, int32_t* out_tokens, void* stream) {
  CHECK_READY();
  if (n < 0 || steps < 0 || (n > 0 && steps > 0 && (!seq_ids || !temperature || !out_tokens)))
    FAIL(SPEC_E_INVALID, "bad arguments");
  if (n == 0 || steps == 0) return SPEC_OK;
  if (!check_ids(ctx, n, seq_ids, true)) return SPEC_E_INVALID;
  Model& T = ctx->m[0];
  int need = 0;
  for (int i = 0; i < n; ++i) {
    const Seq& s = ctx->seqs[seq_ids[i]];
    if (!(temperature[i] >= 0.f)) FAIL(SPEC_E_INVALID, "temperature must be >= 0");
    if (s.k > 0 || s.verified) FAIL(SPEC_E_STATE, "decode of a sequence with drafts or an uncommitted verify");
    if (T.pool.pages_for(s.n() + steps) > ctx->max_pages) FAIL(SPEC_E_INVALID, "sequence exceeds max_pages_per_seq");
    need += T.pool.need(s.pages_t, s.n() + steps);
  }
  if (need > T.pool.free_pages()) FAIL(SPEC_E_NOPAGES, "target KV page pool exhausted");
  // each step is a verify of no drafts (the one row's bonus draw is the next
  // token) and its commit
  const int W = ctx->k_max + 1;
  std::vector<int32_t> acc(n), tok(static_cast<size_t>(n) * W), none(n, 0);
  for (int j = 0; j < steps; ++j) {
    spec_status s = verify_impl(ctx, n, seq_ids, temperature, seed, acc.data(), tok.data(), true, stream);
    if (s != SPEC_OK) return s;
    for (int i = 0; i < n; ++i) out_tokens[static_cast<size_t>(i) * steps + j] = tok[static_cast<size_t>(i) * W];
    s = spec_kv_commit(ctx, n, seq_ids, none.data(), stream);
    if (s != SPEC_OK) return s;
  }
  return SPEC_OK;
}

spec_status spec_kv_rollback(spec_ctx* ctx, int64_t seq_id, int32_t new_len, void* stream) {
  CHECK_READY();
  hipStream_t st = static_cast<hipStream_t>(stream);
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) FAIL(SPEC_E_INVALID, "unknown seq_id");
  Seq& s = it->second;
  if (new_len < 0 || new_len > s.len_t) FAIL(SPEC_E_INVALID, "new_len outside 0..target length");
  std::vector<int32_t> ct, cd;
  const int new_d = std::min(s.len_d, new_len);
  for (int p = new_len; p < s.written_t; ++p) ct.push_back(ctx->m[0].pool.slot(s.pages_t, p));
  for (int p = new_d; p < s.len_d; ++p) cd.push_back(ctx->m[1].pool.slot(s.pages_d, p));
  ctx->m[0].pool.truncate(s.pages_t, new_len);
  ctx->m[1].pool.truncate(s.pages_d, new_d);
  s.hist.resize(new_len + 1);
  s.len_t = s.written_t = new_len;
  s.len_d = new_d;
  s.k = 0;
  s.qrow.clear();
  s.dsrc.clear();
  s.external = false;
  s.verified = false;
  s.emitted.clear();
  s.tparent.clear();
  s.tpath.clear();
  return launch_clears(ctx, ct, cd, st);
}

spec_status spec_seq_release(spec_ctx* ctx, int64_t seq_id) {
  if (!ctx) return SPEC_E_INVALID;
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) FAIL(SPEC_E_INVALID, "unknown seq_id");
  ctx->m[0].pool.truncate(it->second.pages_t, 0);
  ctx->m[1].pool.truncate(it->second.pages_d, 0);
  ctx->free_slots.push(it->second.slot);
  ctx->seqs.erase(it);
  return SPEC_OK;
}

spec_status spec_seq_info(const spec_ctx* ctx, int64_t seq_id, int32_t* target_len, int32_t* draft_len,
                          int32_t* pending_pos, int32_t* pages_target, int32_t* n_pages_target,
                          int32_t* pages_draft, int32_t* n_pages_draft, int32_t max_pages) {
  if (!ctx) return SPEC_E_INVALID;
  auto it = ctx->seqs.find(seq_id);
  if (it == ctx->seqs.end()) return SPEC_E_INVALID;
  const Seq& s = it->second;
  if (target_len) *target_len = s.len_t;
  if (draft_len) *draft_len = s.len_d;
  if (pending_pos) *pending_pos = s.n();
  auto put = [&](const std::vector<int32_t>& t, int32_t* out, int32_t* cnt) {
    if (cnt) *cnt = static_cast<int32_t>(t.size());
    if (out)
      for (int i = 0; i < static_cast<int>(t.size()) && i < max_pages; ++i) out[i] = t[i];
  };
  put(s.pages_t, pages_target, n_pages_target);
  put(s.pages_d, pages_draft, n_pages_draft);
  return SPEC_OK;
}

spec_status spec_last_logits(const spec_ctx* ctx, const float** logits, int32_t* rows) {
  if (!ctx || !logits || !rows || !ctx->wsp) return SPEC_E_INVALID;
  *logits = reinterpret_cast<const float*>(ctx->wsp + ctx->ws.logits);
  *rows = ctx->last_rows;
  return SPEC_OK;
}

}  // extern "C"
