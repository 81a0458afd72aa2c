// Context-free entry points: the decision pass on caller logits, the draft
// sampler, the generator, and single-kernel entry points (include/spec_ops.h).

#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/spec.h"
#include "../../include/spec_ops.h"
#include "attention.h"
#include "elem.h"
#include "gemm.h"
#include "host_util.h"
#include "vocab.h"

using namespace spec;

namespace {

constexpr int kOpMaxParts = 4096;

std::mutex g_mu;
Stager& stager() {
  static Stager s;
  return s;
}

spec_status hip_status(hipError_t e) {
  if (e == hipSuccess) return SPEC_OK;
  if (e == hipErrorInvalidValue) return SPEC_E_UNSUPPORTED;
  return SPEC_E_HIP;
}

}  // namespace

namespace spec {
EventTimer& global_timer() {
  static EventTimer t;
  return t;
}
}  // namespace spec

extern "C" {

size_t spec_sample_workspace_bytes(int32_t B, int32_t total_rows, int32_t V) {
  if (B <= 0 || total_rows <= 0 || V <= 0) return 0;
  return align_up(sizeof(VRow) * total_rows) + align_up(sizeof(VSeq) * B) +
         vocab_ws_bytes(vocab_plan(B, total_rows, V));
}

spec_status spec_sample_verify(int32_t B, const int32_t* k, const float* temperature,
                               const int64_t* seq_ids, const int32_t* base_pos,
                               const float* p_logits, const float* q_logits,
                               const int32_t* draft_tokens, int32_t V, uint64_t seed,
                               int32_t* n_accepted, int32_t* out_tokens, void* workspace,
                               size_t workspace_bytes, void* stream) {
  if (B < 0 || V <= 0) return SPEC_E_INVALID;
  if (B == 0) return SPEC_OK;
  if (!k || !temperature || !seq_ids || !base_pos || !p_logits || !n_accepted || !out_tokens || !workspace)
    return SPEC_E_INVALID;
  int kmax = 0, np = 0, nq = 0;
  for (int b = 0; b < B; ++b) {
    if (k[b] < 0 || k[b] > 15 || !(temperature[b] >= 0.f)) return SPEC_E_INVALID;
    kmax = std::max(kmax, k[b]);
    np += k[b] + 1;
    nq += k[b];
  }
  if (nq > 0 && (!q_logits || !draft_tokens)) return SPEC_E_INVALID;
  const int rows_n = np + nq;
  if (workspace_bytes < spec_sample_workspace_bytes(B, rows_n, V)) return SPEC_E_INVALID;
  std::vector<VRow> rows(rows_n);
  std::vector<VSeq> seqs(B);
  int pr = 0, qr = 0;
  for (int b = 0; b < B; ++b) {
    const float t = temperature[b];
    const float it = t > 0.f ? 1.f / t : 0.f;
    VSeq s{};
    s.k = k[b];
    s.p_row = pr;
    s.q_row = np + qr;
    s.tok_row = qr;
    s.base_pos = base_pos[b];
    s.t = t;
    s.seq_lo = static_cast<uint32_t>(static_cast<uint64_t>(seq_ids[b]));
    s.seq_hi = static_cast<uint32_t>(static_cast<uint64_t>(seq_ids[b]) >> 32);
    seqs[b] = s;
    for (int j = 0; j <= k[b]; ++j)
      rows[pr + j] = VRow{p_logits + static_cast<size_t>(pr + j) * V, it, t > 0.f ? 0 : 1};
    for (int j = 0; j < k[b]; ++j)
      rows[np + qr + j] = VRow{q_logits + static_cast<size_t>(qr + j) * V, it, t > 0.f ? 0 : 1};
    pr += k[b] + 1;
    qr += k[b];
  }
  char* ws = static_cast<char*>(workspace);
  const size_t orow = 0, oseq = align_up(sizeof(VRow) * rows_n);
  const size_t ovoc = oseq + align_up(sizeof(VSeq) * B);
  MetaBlock mb;
  mb.add(rows);
  mb.add(seqs);
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::lock_guard<std::mutex> lk(g_mu);
  // the metadata block lays rows then seqs out exactly at orow / oseq
  hipError_t e = stager().upload(ws, mb.data(), oseq + sizeof(VSeq) * B, st);
  if (e != hipSuccess) return SPEC_E_HIP;
  // the vector path reads 16-byte units from each row
  const bool aligned = (reinterpret_cast<uintptr_t>(p_logits) & 15) == 0 &&
                       (nq == 0 || (reinterpret_cast<uintptr_t>(q_logits) & 15) == 0);
  e = launch_vocab_pass(vocab_plan(B, rows_n, V, B * (2 * kmax + 1)), reinterpret_cast<const VRow*>(ws + orow),
                        reinterpret_cast<const VSeq*>(ws + oseq), draft_tokens, seed, kmax, n_accepted,
                        out_tokens, ws + ovoc, st, &global_timer(), nullptr, aligned);
  return hip_status(e);
}

spec_status spec_sample_draft(int32_t n, const float* logits, int32_t V, const float* temperature,
                              const int64_t* seq_ids, const int32_t* pos, uint64_t seed,
                              int32_t* tokens, void* workspace, size_t workspace_bytes, void* stream) {
  if (n < 0 || V <= 0) return SPEC_E_INVALID;
  if (n == 0) return SPEC_OK;
  if (!logits || !temperature || !seq_ids || !pos || !tokens || !workspace) return SPEC_E_INVALID;
  const DraftPlan p = draft_plan(n, V);
  const size_t odr = 0, ows = align_up(sizeof(DRow) * n);
  if (workspace_bytes < ows + draft_ws_bytes(p)) return SPEC_E_INVALID;
  std::vector<DRow> rows(n);
  for (int i = 0; i < n; ++i) {
    if (!(temperature[i] >= 0.f)) return SPEC_E_INVALID;
    DRow d{};
    d.ptr = logits + static_cast<size_t>(i) * V;
    d.t = temperature[i];
    d.pos = pos[i];
    d.seq_lo = static_cast<uint32_t>(static_cast<uint64_t>(seq_ids[i]));
    d.seq_hi = static_cast<uint32_t>(static_cast<uint64_t>(seq_ids[i]) >> 32);
    d.out = i;
    d.guide = -1;
    rows[i] = d;
  }
  char* ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::lock_guard<std::mutex> lk(g_mu);
  hipError_t e = stager().upload(ws + odr, rows.data(), sizeof(DRow) * n, st);
  if (e != hipSuccess) return SPEC_E_HIP;
  return hip_status(launch_draft_sample(p, reinterpret_cast<const DRow*>(ws + odr), seed, tokens, ws + ows, st));
}

spec_status spec_philox_uniform(uint64_t seed, int64_t seq_id, int32_t pos, int32_t purpose, int32_t n,
                                float* out, void* stream) {
  if (n < 0 || (n > 0 && !out)) return SPEC_E_INVALID;
  return hip_status(launch_philox_uniform(seed, static_cast<uint64_t>(seq_id), pos, purpose, n, out,
                                          static_cast<hipStream_t>(stream)));
}

size_t spec_op_gemm_workspace_bytes(int32_t R, int32_t Nw) {
  return (R <= 0 || Nw <= 0) ? 0 : gemm_splitk_bytes(R, Nw);
}

spec_status spec_pack_weight(void* w, int32_t rows, int32_t K, int32_t rot_rows, int32_t head_dim,
                             void* stream) {
  if (!w || rows < 0 || K <= 0 || rot_rows < 0 || rot_rows > rows) return SPEC_E_INVALID;
  if (K % 128 != 0) return SPEC_E_UNSUPPORTED;
  if (rot_rows > 0 && (head_dim <= 0 || head_dim % 16 != 0 || head_dim > 256 || rot_rows % head_dim != 0))
    return SPEC_E_UNSUPPORTED;
  return hip_status(launch_pack_weight(w, rows, K, rot_rows, head_dim, static_cast<hipStream_t>(stream)));
}

spec_status spec_pack_model(spec_model_desc* m, void* stream) {
  if (!m || !m->layers || !m->lm_head) return SPEC_E_INVALID;
  if (m->weight_layout != SPEC_LAYOUT_ROWMAJOR) return SPEC_E_STATE;
  if (m->dtype == SPEC_F32) return SPEC_OK;
  if (m->dtype != SPEC_BF16 || m->n_layers <= 0 || m->d_model <= 0 || m->ffn_dim <= 0 || m->n_heads <= 0 ||
      m->n_kv_heads <= 0 || m->head_dim <= 0 || m->vocab <= 0)
    return SPEC_E_INVALID;
  const int d = m->d_model, f = m->ffn_dim, hd = m->head_dim, qd = m->n_heads * hd;
  if (d % 128 || f % 128 || qd % 128 || hd % 16) return SPEC_E_UNSUPPORTED;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int qkv_rows = (m->n_heads + 2 * m->n_kv_heads) * hd, rot = (m->n_heads + m->n_kv_heads) * hd;
  const size_t esz = 2;
  std::vector<const void*> done;  // matrices shared between layers are converted once
  auto once = [&](const void* p) {
    if (std::find(done.begin(), done.end(), p) != done.end()) return false;
    done.push_back(p);
    return true;
  };
  auto pack = [&](const void* p, int rows, int K, int rr) -> hipError_t {
    if (!p || !once(p)) return hipSuccess;
    return launch_pack_weight(const_cast<void*>(p), rows, K, rr, hd, st);
  };
  for (int l = 0; l < m->n_layers; ++l) {
    const spec_layer_weights& L = m->layers[l];
    hipError_t e = pack(L.wqkv, qkv_rows, d, rot);
    if (e == hipSuccess) e = pack(L.wo, d, qd, 0);
    if (e == hipSuccess && L.w_gate_up && once(L.w_gate_up)) {
      e = launch_pack_weight(const_cast<void*>(L.w_gate_up), f, d, 0, hd, st);
      if (e == hipSuccess)
        e = launch_pack_weight(static_cast<char*>(const_cast<void*>(L.w_gate_up)) + static_cast<size_t>(f) * d * esz,
                               f, d, 0, hd, st);
    }
    if (e == hipSuccess) e = pack(L.w_down, d, f, 0);
    if (e != hipSuccess) return hip_status(e);
  }
  const hipError_t e = pack(m->lm_head, m->vocab, d, 0);
  if (e != hipSuccess) return hip_status(e);
  m->weight_layout = SPEC_LAYOUT_TILED;
  return SPEC_OK;
}

spec_status spec_op_gemm(int32_t dtype, int32_t R, int32_t N, int32_t K, const void* X, const void* W,
                         void* Y, int32_t epilogue, void* workspace, size_t workspace_bytes, void* stream) {
  if ((dtype != SPEC_F32 && dtype != SPEC_BF16) || R < 0 || N < 0 || K <= 0 || !X || !W || !Y)
    return SPEC_E_INVALID;
  if (epilogue < SPEC_EPI_STORE_F32 || epilogue > SPEC_EPI_SWIGLU) return SPEC_E_INVALID;
  if (dtype == SPEC_BF16 && K % 128 != 0) return SPEC_E_UNSUPPORTED;
  return hip_status(launch_gemm(dtype == SPEC_F32 ? 0 : 1, R, N, K, X, W, Y, epilogue,
                                static_cast<hipStream_t>(stream), nullptr, static_cast<float*>(workspace),
                                workspace ? workspace_bytes : 0));
}

spec_status spec_op_rmsnorm(int32_t dtype, int32_t R, int32_t d, const float* h, const void* w, float eps,
                            void* y, void* stream) {
  if ((dtype != SPEC_F32 && dtype != SPEC_BF16) || R < 0 || d <= 0 || !h || !w || !y) return SPEC_E_INVALID;
  return hip_status(launch_rmsnorm(dtype == SPEC_F32 ? 0 : 1, R, d, h, nullptr, w, eps, y,
                                   static_cast<hipStream_t>(stream)));
}

spec_status spec_op_rope_kv(int32_t dtype, int32_t R, int32_t n_heads, int32_t n_kv_heads, int32_t head_dim,
                            float theta, const float* qkv, const int32_t* pos, const int32_t* slot,
                            void* q_out, void* k_pages, void* v_pages, void* stream) {
  if ((dtype != SPEC_F32 && dtype != SPEC_BF16) || R < 0 || n_heads <= 0 || n_kv_heads <= 0 ||
      head_dim <= 0 || head_dim % 2 || head_dim > 256)
    return SPEC_E_INVALID;
  if (R == 0) return SPEC_OK;
  if (!qkv || !pos || !slot || !q_out || !k_pages || !v_pages) return SPEC_E_INVALID;
  return hip_status(launch_rope_kv(dtype == SPEC_F32 ? 0 : 1, R, n_heads, n_kv_heads, head_dim, theta, qkv,
                                   pos, slot, q_out, k_pages, v_pages, static_cast<hipStream_t>(stream)));
}

size_t spec_op_attention_workspace_bytes(int32_t n_seqs, int32_t total_rows, int32_t max_pages,
                                         int32_t n_kv_heads, int32_t head_dim) {
  if (n_seqs <= 0 || total_rows <= 0) return 0;
  const size_t meta = align_up(sizeof(int32_t) * (static_cast<size_t>(n_seqs) * max_pages + 2 * total_rows)) +
                      align_up(sizeof(AttnItem) * (static_cast<size_t>(total_rows) + kOpMaxParts)) +
                      align_up(sizeof(AttnGroup) * total_rows);
  return meta + align_up(sizeof(float) * static_cast<size_t>(kOpMaxParts) * n_kv_heads * 64 * head_dim) +
         align_up(sizeof(float) * static_cast<size_t>(kOpMaxParts) * n_kv_heads * 64 * 2);
}

spec_status spec_op_attention(int32_t dtype, int32_t n_seqs, const int32_t* rows, const int32_t* pos0,
                              const int32_t* page_table, int32_t max_pages, int32_t n_heads,
                              int32_t n_kv_heads, int32_t head_dim, const void* q, const void* k_pages,
                              const void* v_pages, void* out, void* workspace, size_t workspace_bytes,
                              void* stream) {
  if ((dtype != SPEC_F32 && dtype != SPEC_BF16) || n_seqs < 0 || max_pages <= 0 || n_heads <= 0 ||
      n_kv_heads <= 0 || n_heads % n_kv_heads)
    return SPEC_E_INVALID;
  if (head_dim != 64 && head_dim != 128) return SPEC_E_UNSUPPORTED;
  if (n_seqs == 0) return SPEC_OK;
  if (!rows || !pos0 || !page_table || !q || !k_pages || !v_pages || !out || !workspace) return SPEC_E_INVALID;
  int R = 0;
  std::vector<AttnSegment> segs;
  std::vector<int32_t> rseq, rpos;
  for (int i = 0; i < n_seqs; ++i) {
    if (rows[i] <= 0 || pos0[i] < 0 || ((pos0[i] + rows[i] + 15) / 16) > max_pages) return SPEC_E_INVALID;
    segs.push_back(AttnSegment{i, R, rows[i], pos0[i]});
    for (int r = 0; r < rows[i]; ++r) {
      rseq.push_back(i);
      rpos.push_back(pos0[i] + r);
    }
    R += rows[i];
  }
  if (workspace_bytes < spec_op_attention_workspace_bytes(n_seqs, R, max_pages, n_kv_heads, head_dim))
    return SPEC_E_INVALID;
  AttnPlan plan = plan_attention(segs, n_heads / n_kv_heads, n_kv_heads, kOpMaxParts);
  MetaBlock mb;
  const size_t opt = mb.add(page_table, static_cast<size_t>(n_seqs) * max_pages);
  const size_t ors = mb.add(rseq), orp = mb.add(rpos);
  const size_t oit = mb.add(plan.items), ogr = mb.add(plan.groups);
  char* ws = static_cast<char*>(workspace);
  const size_t meta_bytes = align_up(sizeof(int32_t) * (static_cast<size_t>(n_seqs) * max_pages + 2 * R)) +
                            align_up(sizeof(AttnItem) * (static_cast<size_t>(R) + kOpMaxParts)) +
                            align_up(sizeof(AttnGroup) * R);
  if (mb.size() > meta_bytes + 4 * 256) return SPEC_E_UNSUPPORTED;
  char* part = ws + align_up(meta_bytes + 4 * 256);
  hipStream_t st = static_cast<hipStream_t>(stream);
  {
    std::lock_guard<std::mutex> lk(g_mu);
    if (stager().upload(ws, mb.data(), mb.size(), st) != hipSuccess) return SPEC_E_HIP;
  }
  AttnArgs a;
  a.dtype = dtype == SPEC_F32 ? 0 : 1;
  a.Hq = n_heads;
  a.Hkv = n_kv_heads;
  a.hd = head_dim;
  a.q = q;
  a.kpool = k_pages;
  a.vpool = v_pages;
  a.page_table = reinterpret_cast<const int32_t*>(ws + opt);
  a.max_pages = max_pages;
  a.out = out;
  a.part_o = reinterpret_cast<float*>(part);
  a.part_ml = reinterpret_cast<float*>(part + align_up(sizeof(float) * static_cast<size_t>(kOpMaxParts) *
                                                       n_kv_heads * 64 * head_dim));
  if (a.dtype == 1 && plan.prefill)
    return hip_status(launch_attention_prefill_bf16(a, reinterpret_cast<const AttnItem*>(ws + oit),
                                                    static_cast<int>(plan.items.size()), st));
  if (a.dtype == 1)
    return hip_status(launch_attention_bf16(a, reinterpret_cast<const AttnItem*>(ws + oit),
                                            static_cast<int>(plan.items.size()),
                                            reinterpret_cast<const AttnGroup*>(ws + ogr),
                                            static_cast<int>(plan.groups.size()), plan.nt, plan.w, st));
  return hip_status(launch_attention_f32(a, R, reinterpret_cast<const int32_t*>(ws + ors),
                                         reinterpret_cast<const int32_t*>(ws + orp), st));
}

}  // extern "C"
