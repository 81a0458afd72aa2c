// Vocabulary-wide decision pass of the verify step, for gfx950.
//
// Speculative sampling (the draft-and-verify rule CacheSpec's drafter follows,
// Section 3.4): draft x~_j is accepted iff u_j * q_j(x~_j) < p_j(x~_j); at the
// first rejection a token is drawn from norm(max(0, p_j - q_j)); if every draft
// is accepted a bonus token is drawn from p_{k+1}.  Categorical draws use the
// Gumbel-max trick with per-token Philox noise: argmax_i (log w_i + G_i), or,
// where the weights are known only up to a factor, the equivalent exponential
// race argmax_i w_i / E_i with E_i = -log u_i.
//
// Four launches:
//   1. stats    grid (chunks, rows), HBM-streaming with 16-byte loads: per
//               row chunk, max, first argmax and sum exp((z - max) / T) in one
//               online pass.
//   2. decide   one workgroup per sequence: every chunk record of the
//               sequence's 2k + 1 rows and the gathered p(x~), q(x~) in one
//               round of loads, then the acceptance scan (one lane per draft,
//               one Philox draw each).  Greedy outcomes are final here; a
//               sampled sequence leaves the row to draw from and its
//               normalisers.
//   3. draw     grid (chunks, sequences): only sampled sequences stream the
//               row they draw from: a rejected (p, q) pair for the residual
//               max(0, p - q), or the bonus row p_{k+1}.  Both by exponential
//               race, which needs no logarithm of the weights.
//   4. final    one wave per sampled sequence: merge the chunk winners.
// Carrying the bonus winner along in the statistics pass (one Gumbel score
// per token of the bonus row) measured 40 us slower at 256 x 8 x 128256: its
// workgroups run several times longer than the others.
// Every kernel keeps its loads of a thread in flight together and merges in a
// fixed order, so results do not depend on timing.

#include <algorithm>
#include <climits>
#include <cmath>

#include "common.h"
#include "philox.h"
#include "vocab.h"

namespace spec {
namespace {

constexpr int kThreads = 256;
constexpr int kTargetBlocks = 2048;  // enough workgroups to cover 256 CUs several times
constexpr int kMaxChunks = 64;
constexpr float kLog2e = 1.4426950408889634f;

// Chunk record of the statistics pass: (max, sum of exp((z - max) / T),
// first argmax).
struct VStat {
  float m, s;
  int32_t idx, pad;
};
struct VPick {
  float score;
  int32_t idx;
  float fb_score;
  int32_t fb_idx;
};
enum { kGreedy = 0, kResample = 1, kBonus = 2 };
// Decision of one sequence: accepted count, mode and, for a sampled draw,
// the normalisers of the rows it reads (p only for the bonus).
struct VDec {
  int32_t a, mode;
  float Mp, Sp, Mq, Sq;
  int32_t pad[2];
};

__device__ __forceinline__ float scaled(float s, float m, float M, float it) {
  return (m == -INFINITY) ? 0.f : s * __expf((m - M) * it);
}

// Merge (m, s, idx) triples; ties of the max go to the lower index.
__device__ __forceinline__ void stat_merge(float& m, float& s, int& idx, float m2, float s2, int i2,
                                           float it, bool greedy) {
  const float M = fmaxf(m, m2);
  if (!greedy) s = scaled(s, m, M, it) + scaled(s2, m2, M, it);
  if (m2 > m || (m2 == m && i2 < idx)) idx = i2;
  m = M;
}

__device__ __forceinline__ void stat_update1(float v, int i, float it, bool greedy, float& m, float& s,
                                             int& idx) {
  if (v > m) {
    if (!greedy) s = scaled(s, m, v, it);
    m = v;
    idx = i;
  }
  if (!greedy) s += __expf((v - m) * it);
}

__device__ __forceinline__ void stat_update4(float4 v, int base, float it, bool greedy, float& m, float& s,
                                             int& idx) {
  const float vm = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
  if (vm > m) {
    const int j = (v.x == vm) ? 0 : (v.y == vm) ? 1 : (v.z == vm) ? 2 : 3;
    if (!greedy) s = scaled(s, m, vm, it);
    m = vm;
    idx = base + j;
  }
  if (!greedy)
    s += __expf((v.x - m) * it) + __expf((v.y - m) * it) + __expf((v.z - m) * it) + __expf((v.w - m) * it);
}

__device__ __forceinline__ void pick_update(float sc, int i, float& best, int& bi) {
  if (sc > best || (sc == best && i < bi)) {
    best = sc;
    bi = i;
  }
}

__device__ __forceinline__ uint32_t word_of(uint4 w, int e) {
  return e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
}

__device__ __forceinline__ void wave_pick(float& best, int& bi) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float b2 = __shfl_xor(best, o, kWave);
    const int i2 = __shfl_xor(bi, o, kWave);
    pick_update(b2, i2, best, bi);
  }
}

// Statistics of one row chunk.
template <bool VEC>
__device__ __forceinline__ void stats_chunk(const float* __restrict__ z, int beg, int end, float it, bool greedy,
                                            float& m, float& s, int& idx) {
  if (VEC) {
    const float4* p4 = reinterpret_cast<const float4*>(z);
    const int b4 = beg >> 2, e4 = end >> 2;
    int i = b4 + threadIdx.x;
    for (; i + 3 * kThreads < e4; i += 4 * kThreads) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = ld_stream(p4 + i + u * kThreads);
#pragma unroll
      for (int u = 0; u < 4; ++u) stat_update4(v[u], 4 * (i + u * kThreads), it, greedy, m, s, idx);
    }
    for (; i < e4; i += kThreads) stat_update4(p4[i], 4 * i, it, greedy, m, s, idx);
  } else {
    for (int i = beg + threadIdx.x; i < end; i += kThreads) stat_update1(z[i], i, it, greedy, m, s, idx);
  }
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void stats_kernel(const VRow* __restrict__ rows, int V, int chunk,
                                                         VStat* __restrict__ stats, int n_chunks,
                                                         const int32_t* __restrict__ n_rows) {
  const int r = blockIdx.y, c = blockIdx.x;
  if (n_rows && r >= *n_rows) return;
  const VRow row = rows[r];
  const float it = row.inv_t;
  const bool greedy = row.greedy != 0;
  const int beg = c * chunk;
  const int end = min(V, beg + chunk);
  float m = -INFINITY, s = 0.f;
  int idx = INT_MAX;
  stats_chunk<VEC>(row.ptr, beg, end, it, greedy, m, s, idx);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, kWave);
    const float s2 = __shfl_xor(s, o, kWave);
    const int i2 = __shfl_xor(idx, o, kWave);
    stat_merge(m, s, idx, m2, s2, i2, it, greedy);
  }
  __shared__ float sm[kThreads / kWave], ss[kThreads / kWave];
  __shared__ int si[kThreads / kWave];
  const int w = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    sm[w] = m;
    ss[w] = s;
    si[w] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / kWave; ++k) stat_merge(m, s, idx, sm[k], ss[k], si[k], it, greedy);
    stats[static_cast<size_t>(r) * n_chunks + c] = VStat{m, s, idx, 0};
  }
}

// One workgroup per sequence.  Thread t takes row t % 32 of the sequence
// (target rows 0..k, then draft rows 0..k-1) and the chunks c = t / 32 + 8 i,
// all its records loaded before the first is used; threads 224 + j gather
// p and q at draft j's token meanwhile.  Partials merge through LDS in group
// order, then one lane per draft runs the acceptance test.
constexpr int kDecGroups = kThreads / 32;

__global__ __launch_bounds__(kThreads) void decide_kernel(
    const VRow* __restrict__ rows, const VSeq* __restrict__ seqs, const int32_t* __restrict__ draft_tok,
    const VStat* __restrict__ stats, int n_chunks, int V, uint64_t seed, const uint64_t* __restrict__ seed_ptr,
    VDec* __restrict__ decs, int kmax, int32_t* __restrict__ n_acc, int32_t* __restrict__ out_tok) {
  const int b = blockIdx.x;
  const VSeq sq = seqs[b];
  const int t = threadIdx.x;
  if (sq.k < 0) {  // not decided (invalid input): -1 everywhere
    if (t == 0) {
      n_acc[b] = -1;
      decs[b] = VDec{-1, kGreedy, 0.f, 0.f, 0.f, 0.f, {0, 0}};
    }
    if (t <= kmax) out_tok[static_cast<size_t>(b) * (kmax + 1) + t] = -1;
    return;
  }
  const bool greedy = !(sq.t > 0.f);
  const float it = rows[sq.p_row].inv_t;
  const int nr = 2 * sq.k + 1;
  __shared__ float pm[kDecGroups][32], ps[kDecGroups][32];
  __shared__ int pi[kDecGroups][32];
  __shared__ float rM[32], rS[32], gzp[16], gzq[16];
  __shared__ int rI[32], gx[16];
  {
    const int r = t & 31, g = t >> 5;
    float m = -INFINITY, s = 0.f;
    int idx = INT_MAX;
    if (r < nr) {
      const int row = r <= sq.k ? sq.p_row + r : sq.q_row + (r - sq.k - 1);
      const VStat* st = stats + static_cast<size_t>(row) * n_chunks;
      VStat v[kMaxChunks / kDecGroups];
#pragma unroll
      for (int i = 0; i < kMaxChunks / kDecGroups; ++i) {
        const int c = g + kDecGroups * i;
        if (c < n_chunks) v[i] = st[c];
      }
#pragma unroll
      for (int i = 0; i < kMaxChunks / kDecGroups; ++i) {
        const int c = g + kDecGroups * i;
        if (c < n_chunks) stat_merge(m, s, idx, v[i].m, v[i].s, v[i].idx, it, greedy);
      }
    }
    pm[g][r] = m;
    ps[g][r] = s;
    pi[g][r] = idx;
    // draft tokens and the gathered logits at them
    const int j = t - (kThreads - 32);
    if (j >= 0 && j < sq.k) {
      const int x = draft_tok[sq.tok_row + j];
      gx[j] = x;
      if (!greedy && static_cast<unsigned>(x) < static_cast<unsigned>(V)) {
        gzp[j] = rows[sq.p_row + j].ptr[x];
        gzq[j] = rows[sq.q_row + j].ptr[x];
      }
    }
  }
  __syncthreads();
  if (t < 32) {
    float m = pm[0][t], s = ps[0][t];
    int idx = pi[0][t];
    for (int g = 1; g < kDecGroups; ++g) stat_merge(m, s, idx, pm[g][t], ps[g][t], pi[g][t], it, greedy);
    rM[t] = m;
    rS[t] = s;
    rI[t] = idx;
  }
  __syncthreads();
  if (t >= kWave) return;
  const int j = t;  // 0-based draft index
  bool acc = true;
  if (j < sq.k) {
    const int x = gx[j];
    if (static_cast<unsigned>(x) >= static_cast<unsigned>(V)) {
      acc = false;  // a draft id outside the vocabulary is never accepted
    } else if (greedy) {
      acc = (x == rI[j]);
    } else {
      const float px = __expf((gzp[j] - rM[j]) * it) / rS[j];
      const float qx = __expf((gzq[j] - rM[sq.k + 1 + j]) * it) / rS[sq.k + 1 + j];
      const uint64_t seq_id = (static_cast<uint64_t>(sq.seq_hi) << 32) | sq.seq_lo;
      const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);
      const uint4 w = philox_block(key, stream_id(seq_id, sq.base_pos + j + 1, 1 /*ACCEPT*/), 0);
      acc = (u01(w.x) * qx < px);
    }
  }
  const uint64_t rej = ~__ballot(acc);
  const int a = (rej == 0) ? sq.k : min(sq.k, static_cast<int>(__ffsll(static_cast<long long>(rej))) - 1);
  const int mode = greedy ? kGreedy : (a < sq.k ? kResample : kBonus);
  if (j == 0) {
    VDec d{};
    d.a = a;
    d.mode = mode;
    if (mode != kGreedy) {
      d.Mp = rM[a];
      d.Sp = rS[a];
      if (mode == kResample) {
        d.Mq = rM[sq.k + 1 + a];
        d.Sq = rS[sq.k + 1 + a];
      }
    }
    decs[b] = d;
  }
  if (mode != kGreedy) return;  // the outputs come from the draw
  if (j == 0) n_acc[b] = a;
  if (j <= kmax) out_tok[static_cast<size_t>(b) * (kmax + 1) + j] = j < a ? gx[j] : (j == a ? rI[a] : -1);
}

// The draw of a sampled sequence over one chunk of the row(s) it reads, by
// exponential race with E_i = -log2 u_i: for a rejection r_i = p_i - q_i,
// score r_i / E_i where r_i > 0, and the fallback p_i / E_i (a draw from p,
// used only if no r_i is positive); for the bonus p_i / E_i on row k.
template <bool VEC, bool RESID>
__device__ __forceinline__ void draw_chunk(const float* __restrict__ zp, const float* __restrict__ zq, int beg,
                                           int end, float cs, float dp, float dq, float rsp, float rsq,
                                           PhiloxKey key, StreamId sid, float& best, int& bi, float& fb, int& fi) {
  auto score = [&](float zpi, float zqi, uint32_t word, int i) {
    const float p = __builtin_amdgcn_exp2f(fmaf(zpi, cs, -dp)) * rsp;
    const float ie = __builtin_amdgcn_rcpf(exp2_variate(word));
    if (RESID) {
      const float r = p - __builtin_amdgcn_exp2f(fmaf(zqi, cs, -dq)) * rsq;
      pick_update(r > 0.f ? r * ie : -1.f, i, best, bi);
    }
    pick_update(p * ie, i, fb, fi);
  };
  if (VEC) {
    // batches of 4 float4 of each row per thread (clamped loads, all in
    // flight before the first is used), then the per-element order
    const int e4 = end >> 2;
    for (int i0 = (beg >> 2) + threadIdx.x; i0 < e4; i0 += 4 * kThreads) {
      float4 pv[4], qv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int jj = min(i0 + u * kThreads, e4 - 1);
        pv[u] = reinterpret_cast<const float4*>(zp)[jj];
        if (RESID) qv[u] = reinterpret_cast<const float4*>(zq)[jj];
        else qv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i4 = i0 + u * kThreads;
        if (i4 >= e4) break;
        const uint4 w = philox_block(key, sid, static_cast<uint32_t>(i4));
        score(pv[u].x, qv[u].x, w.x, 4 * i4);
        score(pv[u].y, qv[u].y, w.y, 4 * i4 + 1);
        score(pv[u].z, qv[u].z, w.z, 4 * i4 + 2);
        score(pv[u].w, qv[u].w, w.w, 4 * i4 + 3);
      }
    }
  } else {
    for (int i = beg + threadIdx.x; i < end; i += kThreads) {
      const uint4 w = philox_block(key, sid, static_cast<uint32_t>(i >> 2));
      score(zp[i], RESID ? zq[i] : 0.f, word_of(w, i & 3), i);
    }
  }
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void draw_kernel(const VRow* __restrict__ rows, const VSeq* __restrict__ seqs,
                                                        const VDec* __restrict__ decs, int V, int chunk,
                                                        int n_chunks, uint64_t seed,
                                                        const uint64_t* __restrict__ seed_ptr,
                                                        VPick* __restrict__ picks) {
  const int b = blockIdx.y, c = blockIdx.x;
  const VDec d = decs[b];
  if (d.mode == kGreedy) return;
  const VSeq sq = seqs[b];
  const bool resid = d.mode == kResample;
  const VRow rp = rows[sq.p_row + d.a];
  const float cs = rp.inv_t * kLog2e;  // p_i S_p = 2^(z_i cs - M cs)
  const uint64_t seq_id = (static_cast<uint64_t>(sq.seq_hi) << 32) | sq.seq_lo;
  const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);
  // RESAMPLE noise at the rejected position n + a + 1, BONUS at n + k + 1
  const StreamId sid = stream_id(seq_id, sq.base_pos + d.a + 1, resid ? 2 : 3);
  float best = -1.f, fb = -1.f;
  int bi = INT_MAX, fi = INT_MAX;
  const int beg = c * chunk;
  const int end = min(V, beg + chunk);
  if (resid)
    draw_chunk<VEC, true>(rp.ptr, rows[sq.q_row + d.a].ptr, beg, end, cs, d.Mp * cs, d.Mq * cs, 1.f / d.Sp,
                          1.f / d.Sq, key, sid, best, bi, fb, fi);
  else
    draw_chunk<VEC, false>(rp.ptr, nullptr, beg, end, cs, d.Mp * cs, 0.f, 1.f / d.Sp, 0.f, key, sid, best, bi,
                           fb, fi);
  wave_pick(best, bi);
  wave_pick(fb, fi);
  __shared__ VPick sp[kThreads / kWave];
  const int wv = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sp[wv] = VPick{best, bi, fb, fi};
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / kWave; ++k) {
      pick_update(sp[k].score, sp[k].idx, best, bi);
      pick_update(sp[k].fb_score, sp[k].fb_idx, fb, fi);
    }
    picks[static_cast<size_t>(b) * n_chunks + c] = VPick{best, bi, fb, fi};
  }
}

// One wave per sampled sequence: lane c holds chunk c's winners (at most 64
// chunks), merged by shuffles.
__global__ __launch_bounds__(kWave) void final_kernel(const VSeq* __restrict__ seqs,
                                                      const int32_t* __restrict__ draft_tok,
                                                      const VDec* __restrict__ decs,
                                                      const VPick* __restrict__ picks, int n_chunks, int kmax,
                                                      int32_t* __restrict__ n_acc, int32_t* __restrict__ out_tok) {
  const int b = blockIdx.x;
  const VDec d = decs[b];
  if (d.mode == kGreedy) return;
  const int l = threadIdx.x;
  const VSeq sq = seqs[b];
  float best = -1.f, fb = -1.f;
  int bi = INT_MAX, fi = INT_MAX;
  if (l < n_chunks) {
    const VPick p = picks[static_cast<size_t>(b) * n_chunks + l];
    best = p.score;
    bi = p.idx;
    fb = p.fb_score;
    fi = p.fb_idx;
  }
  const int x = l < d.a ? draft_tok[sq.tok_row + l] : -1;
  wave_pick(best, bi);
  wave_pick(fb, fi);
  // residual scores are positive; with none (only possible when p and q agree
  // in fp32) the draw falls back to p; the bonus draws from p
  const int t = (d.mode == kResample && best > 0.f) ? bi : fi;
  if (l == 0) n_acc[b] = d.a;
  if (l <= kmax) out_tok[static_cast<size_t>(b) * (kmax + 1) + l] = l < d.a ? x : (l == d.a ? t : -1);
}

// ---------------------------------------------------------------------------
// Tree verification.  At node u the target distribution is r_0 = p_u; each
// rejected child replaces r_l by r_{l+1} = max(0, r_l - q_u) / Z_{l+1}, where
// Z_{l+1} is the residual's mass (a residual with no mass keeps r_l), so
// r_l(y) is evaluated from p_u(y), q_u(y) and Z_1..Z_l alone.  Every child of
// u is drawn from the same q_u, so Z_l depends on how many children were
// rejected, not on which: the masses of every node and level, and each node's
// final draw (from r_{c(u)} once its c(u) children are all rejected, from p
// at a leaf), are computed for all nodes at once by chip-wide passes
// (tree_z_kernel per level, tree_draw_kernel); one wave per sequence then
// walks the tree with the acceptance tests alone (tree_walk_kernel).  Each
// vocabulary pass is a grid of (chunk, node slot) workgroups; the masses are
// chunk partials summed in chunk order wherever they are used.

constexpr int kTreeMaxNodes = 16;  // slots per sequence: the root and at most 15 nodes
constexpr int kTreeWaves = kThreads / kWave;

// Slot s of a sequence: s = 0 the root, s = i + 1 node i.
struct TreeSlot {
  int prow, qrow, kids, depth;
};
__device__ __forceinline__ TreeSlot tree_slot(const VTreeSeq& sq, const VTreeNode* __restrict__ nodes, int s) {
  const int u = s - 1;
  TreeSlot r;
  r.prow = u < 0 ? sq.p_row : nodes[sq.node0 + u].p_row;
  r.qrow = u < 0 ? sq.q_row : nodes[sq.node0 + u].q_row;
  r.kids = 0;
  for (int i = 0; i < sq.m; ++i) r.kids += nodes[sq.node0 + i].parent == u ? 1 : 0;
  r.depth = 0;
  // parents have smaller indices; at most m steps
  for (int v = u, n = 0; v >= 0 && n < sq.m; v = nodes[sq.node0 + v].parent, ++n) ++r.depth;
  return r;
}

// Partial masses of the residuals: zpart[((b * kTreeMaxNodes + s) * kTreeMaxNodes + l - 1) * kMaxChunks + c]
// is chunk c's share of Z_l at slot s of sequence b.
__device__ __forceinline__ size_t tree_z_index(int b, int s, int l, int c) {
  return ((static_cast<size_t>(b) * kTreeMaxNodes + s) * kTreeMaxNodes + (l - 1)) * kMaxChunks + c;
}

// Z_l summed over the chunks in chunk order (the same value wherever used).
__device__ __forceinline__ float tree_z_total(const float* __restrict__ zpart, int b, int s, int l, int n_chunks) {
  float z = 0.f;
  for (int c = 0; c < n_chunks; ++c) z += zpart[tree_z_index(b, s, l, c)];
  return z;
}

// Merged (max, sum, first argmax) of one row's chunk records, by one wave.
__device__ void tree_row_stats(const VStat* __restrict__ st, int n_chunks, float it, bool greedy, float& m,
                               float& s, int& idx) {
  const int l = threadIdx.x & (kWave - 1);
  m = -INFINITY;
  s = 0.f;
  idx = INT_MAX;
  if (l < n_chunks) {
    const VStat v = st[l];
    m = v.m;
    s = v.s;
    idx = v.idx;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o, kWave), s2 = __shfl_xor(s, o, kWave);
    const int i2 = __shfl_xor(idx, o, kWave);
    stat_merge(m, s, idx, m2, s2, i2, it, greedy);
  }
}

// The state a node's residuals are evaluated from: the p and q row statistics
// (scaled into exp2 form) and the masses Z_1..Z_lv.
struct TreeRes {
  const float* zp;
  const float* zq;
  float cs, mpc, isp, mqc, isq;
  float invz[kTreeMaxNodes];
  int keep[kTreeMaxNodes];
};

// r_lv(y) from p(y), q(y) and the residual normalisers so far (levels
// unrolled so that the tables stay in registers)
__device__ __forceinline__ float tree_r_at(const TreeRes& R, int y, int lv) {
  float r = exp2f(R.zp[y] * R.cs - R.mpc) * R.isp;
  if (lv > 0) {
    const float q = exp2f(R.zq[y] * R.cs - R.mqc) * R.isq;
#pragma unroll
    for (int l = 1; l < kTreeMaxNodes; ++l)
      if (l <= lv && !R.keep[l]) r = fmaxf(r - q, 0.f) * R.invz[l];
  }
  return r;
}

// The residual state of slot s through level lv (a sampled sequence), for a
// whole workgroup: waves 0 and 1 merge the p and q statistics, threads
// 1 .. lv sum the masses.
__device__ void tree_res(const VRow* __restrict__ rows, const VTreeSeq& sq, const TreeSlot& ts,
                         const VStat* __restrict__ stats, const float* __restrict__ zpart, int b, int s, int lv,
                         int n_chunks, TreeRes& R) {
  __shared__ float s_st[4];
  __shared__ float s_z[kTreeMaxNodes];
  const float it = rows[sq.p_row].inv_t;
  const int t = threadIdx.x;
  if (t < kWave) {
    float m, sm;
    int idx;
    tree_row_stats(stats + static_cast<size_t>(ts.prow) * n_chunks, n_chunks, it, false, m, sm, idx);
    if (t == 0) {
      s_st[0] = m;
      s_st[1] = sm;
    }
  } else if (t < 2 * kWave && ts.qrow >= 0) {
    float m, sm;
    int idx;
    tree_row_stats(stats + static_cast<size_t>(ts.qrow) * n_chunks, n_chunks, it, false, m, sm, idx);
    if (t == kWave) {
      s_st[2] = m;
      s_st[3] = sm;
    }
  }
  if (t > 0 && t <= lv) s_z[t] = tree_z_total(zpart, b, s, t, n_chunks);
  __syncthreads();
  R.cs = it * kLog2e;
  R.zp = rows[ts.prow].ptr;
  R.zq = ts.qrow >= 0 ? rows[ts.qrow].ptr : nullptr;
  R.mpc = s_st[0] * R.cs;
  R.isp = 1.f / s_st[1];
  R.mqc = ts.qrow >= 0 ? s_st[2] * R.cs : 0.f;
  R.isq = ts.qrow >= 0 ? 1.f / s_st[3] : 0.f;
#pragma unroll
  for (int l = 1; l < kTreeMaxNodes; ++l) {
    const float z = l <= lv ? s_z[l] : 1.f;
    R.keep[l] = !(z > 0.f);
    R.invz[l] = z > 0.f ? 1.f / z : 1.f;
  }
}

// Chunk c's share of Z_L at every slot with at least L children.
__global__ __launch_bounds__(kThreads) void tree_z_kernel(const VRow* __restrict__ rows,
                                                          const VTreeSeq* __restrict__ seqs,
                                                          const VTreeNode* __restrict__ nodes,
                                                          const VStat* __restrict__ stats, int n_chunks, int chunk,
                                                          int V, int L, float* __restrict__ zpart) {
  const int c = blockIdx.x, b = blockIdx.y / kTreeMaxNodes, s = blockIdx.y % kTreeMaxNodes;
  const VTreeSeq sq = seqs[b];
  if (s > sq.m || !(sq.t > 0.f)) return;
  const TreeSlot ts = tree_slot(sq, nodes, s);
  if (ts.qrow < 0 || ts.kids < L) return;
  TreeRes R;
  tree_res(rows, sq, ts, stats, zpart, b, s, L - 1, n_chunks, R);
  const int beg = c * chunk, end = min(V, beg + chunk);
  float part = 0.f;
  for (int y = beg + static_cast<int>(threadIdx.x); y < end; y += kThreads) {
    const float q = exp2f(R.zq[y] * R.cs - R.mqc) * R.isq;
    part += fmaxf(tree_r_at(R, y, L - 1) - q, 0.f);
  }
  // fixed-order workgroup sum
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, kWave);
  __shared__ float red[kTreeWaves];
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    float z = 0.f;
    for (int w = 0; w < kTreeWaves; ++w) z += red[w];
    zpart[tree_z_index(b, s, L, c)] = z;
  }
}

// Chunk c's winner of each slot's final draw: from r_{c(u)} (RESAMPLE noise)
// at a node with children, from p (BONUS noise) at a leaf, by exponential
// race over 4 tokens per Philox block at stream position base + depth + 1.
__global__ __launch_bounds__(kThreads) void tree_draw_kernel(const VRow* __restrict__ rows,
                                                             const VTreeSeq* __restrict__ seqs,
                                                             const VTreeNode* __restrict__ nodes,
                                                             const VStat* __restrict__ stats, int n_chunks,
                                                             int chunk, int V, uint64_t seed,
                                                             const uint64_t* __restrict__ seed_ptr,
                                                             const float* __restrict__ zpart,
                                                             VPick* __restrict__ picks) {
  const int c = blockIdx.x, b = blockIdx.y / kTreeMaxNodes, s = blockIdx.y % kTreeMaxNodes;
  const VTreeSeq sq = seqs[b];
  if (s > sq.m || !(sq.t > 0.f)) return;
  const TreeSlot ts = tree_slot(sq, nodes, s);
  const int lv = ts.qrow >= 0 ? ts.kids : 0;
  TreeRes R;
  tree_res(rows, sq, ts, stats, zpart, b, s, lv, n_chunks, R);
  const uint64_t seq_id = (static_cast<uint64_t>(sq.seq_hi) << 32) | sq.seq_lo;
  const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);
  const StreamId sid = stream_id(seq_id, sq.base_pos + ts.depth + 1, ts.qrow >= 0 ? 2 : 3);
  const int beg = c * chunk, end = min(V, beg + chunk);  // chunk starts are multiples of 1024
  float best = -1.f;
  int bi = INT_MAX;
  for (int y4 = beg / 4 + static_cast<int>(threadIdx.x); 4 * y4 < end; y4 += kThreads) {
    const uint4 w = philox_block(key, sid, static_cast<uint32_t>(y4));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int y = 4 * y4 + e;
      if (y < end) pick_update(tree_r_at(R, y, lv) / exp2_variate(word_of(w, e)), y, best, bi);
    }
  }
  wave_pick(best, bi);
  __shared__ float rf[kTreeWaves];
  __shared__ int ri[kTreeWaves];
  if ((threadIdx.x & (kWave - 1)) == 0) {
    rf[threadIdx.x / kWave] = best;
    ri[threadIdx.x / kWave] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kTreeWaves; ++w) pick_update(rf[w], ri[w], rf[0], ri[0]);
    picks[(static_cast<size_t>(b) * kTreeMaxNodes + s) * kMaxChunks + c] = VPick{rf[0], ri[0], 0.f, 0};
  }
}

// One wave per sequence walks its tree: at a node, children are accepted in
// index order while v_j q(x) < r_lv(x) fails (lv = children rejected so
// far); a greedy sequence follows the argmax of p.  The walk ends at a node
// with no accepted child, whose token is the merged winner of its draw.  All
// lanes take the same steps; lane 0 keeps the walk's state in LDS.
__global__ __launch_bounds__(kWave) void tree_walk_kernel(
    const VRow* __restrict__ rows, const VTreeSeq* __restrict__ seqs, const VTreeNode* __restrict__ nodes,
    const int32_t* __restrict__ row_tok, const VStat* __restrict__ stats, int n_chunks, int V, uint64_t seed,
    const uint64_t* __restrict__ seed_ptr, const float* __restrict__ zpart, const VPick* __restrict__ picks,
    int kmax, int32_t* __restrict__ n_acc, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_path) {
  const int b = blockIdx.x, t = threadIdx.x;
  const VTreeSeq sq = seqs[b];
  const bool greedy = !(sq.t > 0.f);
  const float it = rows[sq.p_row].inv_t;
  const float cs = it * kLog2e;
  const uint64_t seq_id = (static_cast<uint64_t>(sq.seq_hi) << 32) | sq.seq_lo;
  const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);
  __shared__ int s_tok[kTreeMaxNodes + 1], s_path[kTreeMaxNodes];
  __shared__ float s_invz[kTreeMaxNodes];
  __shared__ int s_keep[kTreeMaxNodes];
  int u = -1, d = 0;
  for (;;) {
    const int s = u + 1;
    const int prow = u < 0 ? sq.p_row : nodes[sq.node0 + u].p_row;
    const int qrow = u < 0 ? sq.q_row : nodes[sq.node0 + u].q_row;
    float mp, sp, mq = 0.f, sqs = 1.f;
    int ip, iq = 0;
    tree_row_stats(stats + static_cast<size_t>(prow) * n_chunks, n_chunks, it, greedy, mp, sp, ip);
    if (greedy) {
      int nxt = -1;
      for (int i = 0; i < sq.m; ++i) {
        const VTreeNode nd = nodes[sq.node0 + i];
        if (nd.parent == u && row_tok[nd.p_row] == ip) {
          nxt = i;
          break;
        }
      }
      if (t == 0) {
        s_tok[d] = ip;
        if (nxt >= 0) s_path[d] = nxt;
      }
      if (nxt < 0) break;
      u = nxt;
      ++d;
      continue;
    }
    if (qrow >= 0) tree_row_stats(stats + static_cast<size_t>(qrow) * n_chunks, n_chunks, it, greedy, mq, sqs, iq);
    const float* zp = rows[prow].ptr;
    const float* zq = qrow >= 0 ? rows[qrow].ptr : nullptr;
    const float mpc = mp * cs, isp = 1.f / sp, mqc = mq * cs, isq = 1.f / sqs;
    const StreamId sid_acc = stream_id(seq_id, sq.base_pos + d + 1, 1);
    int lv = 0, acc = -1, j = 0;
    if (qrow >= 0) {
      for (int i = 0; i < sq.m; ++i) {
        const VTreeNode nd = nodes[sq.node0 + i];
        if (nd.parent != u) continue;
        const int x = row_tok[nd.p_row];
        bool ok = false;
        if (static_cast<unsigned>(x) < static_cast<unsigned>(V)) {  // an id outside the vocabulary is rejected
          float r = exp2f(zp[x] * cs - mpc) * isp;
          const float qx = exp2f(zq[x] * cs - mqc) * isq;
          for (int l = 1; l <= lv; ++l)
            if (!s_keep[l]) r = fmaxf(r - qx, 0.f) * s_invz[l];
          const float v = u01(philox_block(key, sid_acc, static_cast<uint32_t>(j)).x);
          ok = v * qx < r;
        }
        if (ok) {
          acc = i;
          break;
        }
        ++lv;
        const float z = tree_z_total(zpart, b, s, lv, n_chunks);
        __syncthreads();
        if (t == 0) {
          s_keep[lv] = !(z > 0.f);
          s_invz[lv] = z > 0.f ? 1.f / z : 1.f;
        }
        __syncthreads();
        ++j;
      }
    }
    if (acc >= 0) {
      if (t == 0) {
        s_tok[d] = row_tok[nodes[sq.node0 + acc].p_row];
        s_path[d] = acc;
      }
      u = acc;
      ++d;
      continue;
    }
    // the node's draw: the chunk winners merged across the wave
    float best = -1.f;
    int bi = INT_MAX;
    if (t < n_chunks) {
      const VPick pk = picks[(static_cast<size_t>(b) * kTreeMaxNodes + s) * kMaxChunks + t];
      best = pk.score;
      bi = pk.idx;
    }
    wave_pick(best, bi);
    if (t == 0) s_tok[d] = bi;
    break;
  }
  __syncthreads();
  if (t == 0) n_acc[b] = d;
  if (t <= kmax) out_tok[static_cast<size_t>(b) * (kmax + 1) + t] = t <= d ? s_tok[t] : -1;
  if (t < kmax) out_path[static_cast<size_t>(b) * kmax + t] = t < d ? s_path[t] : -1;
}

// Tables of the decision pass from device arrays: thread b takes sequence b;
// row offsets are exclusive prefix sums of k + 1 (target rows) and k (draft
// rows), scanned in LDS.
__global__ __launch_bounds__(kSetupMaxSeqs) void setup_kernel(int B, int kmax, const int32_t* __restrict__ k,
                                                             const float* __restrict__ temp,
                                                             const int64_t* __restrict__ ids,
                                                             const int32_t* __restrict__ base,
                                                             const float* __restrict__ p,
                                                             const float* __restrict__ q, int V,
                                                             VRow* __restrict__ rows, VSeq* __restrict__ seqs,
                                                             int32_t* __restrict__ n_rows) {
  __shared__ int sp[kSetupMaxSeqs], sq[kSetupMaxSeqs];
  __shared__ int any_bad;
  const int b = threadIdx.x;
  if (b == 0) any_bad = 0;
  int kb = 0;
  float tb = 0.f;
  if (b < B) {
    kb = k[b];
    tb = temp[b];
  }
  __syncthreads();
  if (b < B && (kb < 0 || kb > kmax || !(tb >= 0.f))) atomicOr(&any_bad, 1);
  sp[b] = b < B ? kb + 1 : 0;
  sq[b] = b < B ? kb : 0;
  __syncthreads();
  const bool bad = any_bad != 0;
  // inclusive Hillis-Steele scans
  for (int o = 1; o < kSetupMaxSeqs; o <<= 1) {
    const int ap = b >= o ? sp[b - o] : 0, aq = b >= o ? sq[b - o] : 0;
    __syncthreads();
    sp[b] += ap;
    sq[b] += aq;
    __syncthreads();
  }
  const int NP = sp[kSetupMaxSeqs - 1];
  const int p_off = sp[b] - (b < B ? kb + 1 : 0), q_off = sq[b] - (b < B ? kb : 0);
  if (b == 0) *n_rows = bad ? 0 : NP + sq[kSetupMaxSeqs - 1];
  if (b >= B) return;
  VSeq s{};
  s.k = bad ? -1 : kb;
  s.p_row = p_off;
  s.q_row = NP + q_off;
  s.tok_row = q_off;
  s.base_pos = base[b];
  s.t = tb;
  const uint64_t id = static_cast<uint64_t>(ids[b]);
  s.seq_lo = static_cast<uint32_t>(id);
  s.seq_hi = static_cast<uint32_t>(id >> 32);
  seqs[b] = s;
  if (bad) return;
  const float it = tb > 0.f ? 1.f / tb : 0.f;
  const int32_t greedy = tb > 0.f ? 0 : 1;
  for (int j = 0; j <= kb; ++j) rows[p_off + j] = VRow{p + static_cast<size_t>(p_off + j) * V, it, greedy};
  for (int j = 0; j < kb; ++j) rows[NP + q_off + j] = VRow{q + static_cast<size_t>(q_off + j) * V, it, greedy};
}

// ---------------------------------------------------------------------------
// Draft sampler: Gumbel-max over z / T with DRAFT noise (argmax for T = 0).

template <bool VEC>
__global__ __launch_bounds__(kThreads) void draft_kernel(int V, const DRow* __restrict__ rows, int chunk,
                                                         int n_chunks, uint64_t seed,
                                                         const uint64_t* __restrict__ seed_ptr,
                                                         VPick* __restrict__ picks) {
  const int r = blockIdx.y, c = blockIdx.x;
  const DRow row = rows[r];
  const float* z = row.ptr;
  const bool greedy = !(row.t > 0.f);
  const float it = greedy ? 0.f : 1.f / row.t;
  const uint64_t seq_id = (static_cast<uint64_t>(row.seq_hi) << 32) | row.seq_lo;
  const StreamId sid = stream_id(seq_id, row.pos, 0 /*DRAFT*/);
  const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);
  const int beg = c * chunk, end = min(V, beg + chunk);
  float best = -INFINITY;
  int bi = INT_MAX;
  if (VEC) {
    // batches of 4 float4 per thread, as in draw_chunk
    const int e4 = end >> 2;
    for (int i0 = (beg >> 2) + threadIdx.x; i0 < e4; i0 += 4 * kThreads) {
      float4 vv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) vv[u] = reinterpret_cast<const float4*>(z)[min(i0 + u * kThreads, e4 - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i4 = i0 + u * kThreads;
        if (i4 >= e4) break;
        const float4 v = vv[u];
        if (greedy) {
          pick_update(v.x, 4 * i4, best, bi);
          pick_update(v.y, 4 * i4 + 1, best, bi);
          pick_update(v.z, 4 * i4 + 2, best, bi);
          pick_update(v.w, 4 * i4 + 3, best, bi);
        } else {
          const uint4 w = philox_block(key, sid, static_cast<uint32_t>(i4));
          pick_update(fmaf(v.x, it, gumbel_shift(w.x)), 4 * i4, best, bi);
          pick_update(fmaf(v.y, it, gumbel_shift(w.y)), 4 * i4 + 1, best, bi);
          pick_update(fmaf(v.z, it, gumbel_shift(w.z)), 4 * i4 + 2, best, bi);
          pick_update(fmaf(v.w, it, gumbel_shift(w.w)), 4 * i4 + 3, best, bi);
        }
      }
    }
  } else {
    for (int i = beg + threadIdx.x; i < end; i += kThreads) {
      if (greedy) {
        pick_update(z[i], i, best, bi);
      } else {
        const uint4 w = philox_block(key, sid, static_cast<uint32_t>(i >> 2));
        pick_update(fmaf(z[i], it, gumbel_shift(word_of(w, i & 3))), i, best, bi);
      }
    }
  }
  wave_pick(best, bi);
  __shared__ float sb[kThreads / kWave];
  __shared__ int sbi[kThreads / kWave];
  const int wv = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    sb[wv] = best;
    sbi[wv] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / kWave; ++k) pick_update(sb[k], sbi[k], best, bi);
    picks[static_cast<size_t>(r) * n_chunks + c] = VPick{best, bi, 0.f, 0};
  }
}

// One workgroup of 1024 threads per guided row: the row maximum with 16-byte
// streaming loads, four in flight per thread, then z[guide] = max + boost
// (all reads of the row finish before the write).
constexpr int kGuideThreads = 1024;

__global__ __launch_bounds__(kGuideThreads) void draft_guide_kernel(int V, const DRow* __restrict__ rows,
                                                                     float boost) {
  const DRow row = rows[blockIdx.x];
  if (row.guide < 0 || row.guide >= V) return;
  const float* z = row.ptr;
  float mx = -INFINITY;
  int tail = 0;
  if ((reinterpret_cast<uintptr_t>(z) & 15) == 0) {
    const float4* p4 = reinterpret_cast<const float4*>(z);
    const int n4 = V >> 2;
    int i = threadIdx.x;
    for (; i + 3 * kGuideThreads < n4; i += 4 * kGuideThreads) {
      const float4 v0 = ld_stream(p4 + i), v1 = ld_stream(p4 + i + kGuideThreads);
      const float4 v2 = ld_stream(p4 + i + 2 * kGuideThreads), v3 = ld_stream(p4 + i + 3 * kGuideThreads);
      mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(v0.x, v0.y), fmaxf(v0.z, v0.w)), fmaxf(fmaxf(v1.x, v1.y), fmaxf(v1.z, v1.w))));
      mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(v2.x, v2.y), fmaxf(v2.z, v2.w)), fmaxf(fmaxf(v3.x, v3.y), fmaxf(v3.z, v3.w))));
    }
    for (; i < n4; i += kGuideThreads) {
      const float4 v = ld_stream(p4 + i);
      mx = fmaxf(mx, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
    }
    tail = n4 * 4;
  }
  for (int i = tail + threadIdx.x; i < V; i += kGuideThreads) mx = fmaxf(mx, z[i]);
  mx = wave_max(mx);
  __shared__ float part[kGuideThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    float m = part[0];
    for (int w = 1; w < kGuideThreads / kWave; ++w) m = fmaxf(m, part[w]);
    const_cast<float*>(z)[row.guide] = m + boost;
  }
}

// One wave per row: lane c holds chunk c's winner, merged by shuffles.
__global__ __launch_bounds__(kWave) void draft_final_kernel(const DRow* __restrict__ rows,
                                                            const VPick* __restrict__ picks, int n_chunks,
                                                            int32_t* __restrict__ tokens) {
  const int r = blockIdx.x, l = threadIdx.x;
  float best = -INFINITY;
  int bi = INT_MAX;
  if (l < n_chunks) {
    const VPick p = picks[static_cast<size_t>(r) * n_chunks + l];
    best = p.score;
    bi = p.idx;
  }
  wave_pick(best, bi);
  if (l == 0) tokens[rows[r].out] = bi;
}

__global__ void philox_uniform_kernel(uint64_t seed, StreamId sid, int n, float* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint4 w = philox_block(philox_key(seed), sid, static_cast<uint32_t>(i >> 2));
  out[i] = u01(word_of(w, i & 3));
}

inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

void chunking(int units, int V, int& chunk, int& n_chunks) {
  int want = std::max(1, (kTargetBlocks + units - 1) / std::max(1, units));
  want = std::min(want, std::max(1, V / 4096));
  // at most kMaxChunks chunks (the decision and merge kernels hold one per
  // lane), each a multiple of 1024 elements (the vector paths need chunk
  // starts on 16-byte boundaries)
  chunk = std::max((V + want - 1) / want, (V + kMaxChunks - 1) / kMaxChunks);
  chunk = (chunk + 1023) / 1024 * 1024;
  n_chunks = (V + chunk - 1) / chunk;
}

}  // namespace

VocabPlan vocab_plan(int B, int n_rows, int V, int chunk_rows) {
  VocabPlan p;
  p.B = B;
  p.n_rows = n_rows;
  p.V = V;
  chunking(chunk_rows >= 0 ? chunk_rows : n_rows, V, p.chunk1, p.n_chunks1);
  chunking(B, V, p.chunk2, p.n_chunks2);
  return p;
}

// Entries rows x chunks of any plan over at most `units` rows (or
// sequences): a plan's chunk count grows as its units shrink, so the product
// is not monotonic in the units, but a chunk count never exceeds
// ceil(kTargetBlocks / units) nor kMaxChunks.
static size_t chunk_entries_bound(int units) {
  const size_t u = static_cast<size_t>(std::max(units, 0));
  return std::min(u * kMaxChunks, static_cast<size_t>(kTargetBlocks) + u);
}

size_t vocab_ws_bound(int B, int n_rows) {
  return align256(sizeof(VStat) * chunk_entries_bound(n_rows)) + align256(sizeof(VPick) * chunk_entries_bound(B)) +
         align256(sizeof(VDec) * static_cast<size_t>(std::max(B, 0)));
}

size_t tree_ws_bound(int B, int n_rows) {
  const size_t b = static_cast<size_t>(std::max(B, 0));
  return align256(sizeof(VStat) * chunk_entries_bound(n_rows)) +
         align256(sizeof(float) * b * kTreeMaxNodes * kTreeMaxNodes * kMaxChunks) +
         align256(sizeof(VPick) * b * kTreeMaxNodes * kMaxChunks);
}

size_t draft_ws_bound(int n) { return align256(sizeof(VPick) * chunk_entries_bound(n)); }

size_t vocab_ws_bytes(const VocabPlan& p) {
  return align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1) +
         align256(sizeof(VPick) * static_cast<size_t>(p.B) * p.n_chunks2) +
         align256(sizeof(VDec) * static_cast<size_t>(p.B));
}

hipError_t launch_vocab_pass(const VocabPlan& p, const VRow* d_rows, const VSeq* d_seqs,
                             const int32_t* d_draft_tok, uint64_t seed, int kmax, int32_t* d_n_acc,
                             int32_t* d_out_tok, void* d_ws, hipStream_t st, KernelTimer* timer,
                             const uint64_t* d_seed, bool aligned, const int32_t* d_n_rows) {
  if (p.B == 0) return hipSuccess;
  if (p.n_chunks1 > kMaxChunks || p.n_chunks2 > kMaxChunks) return hipErrorInvalidValue;
  char* ws = static_cast<char*>(d_ws);
  VStat* stats = reinterpret_cast<VStat*>(ws);
  ws += align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1);
  VPick* picks = reinterpret_cast<VPick*>(ws);
  ws += align256(sizeof(VPick) * static_cast<size_t>(p.B) * p.n_chunks2);
  VDec* decs = reinterpret_cast<VDec*>(ws);
  const bool vec = aligned && (p.V % 4) == 0;
  // the timer names one kernel; bytes are each launch's algorithmic HBM bytes
  auto timed = [&](const char* name) { return timer && timer->wants(name); };
  const char* n1 = vec ? "stats_kernel<true>" : "stats_kernel<false>";
  dim3 g1(p.n_chunks1, p.n_rows);
  if (timed(n1)) timer->begin(st);
  if (vec)
    launch_kernel(stats_kernel<true>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1,
                  d_n_rows);
  else
    launch_kernel(stats_kernel<false>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1,
                  d_n_rows);
  if (timed(n1)) timer->end(st, 4.0 * p.n_rows * p.V, 0.0);
  if (timed("decide_kernel")) timer->begin(st);
  launch_kernel(decide_kernel, dim3(p.B), dim3(kThreads), 0, st, d_rows, d_seqs, d_draft_tok, stats, p.n_chunks1,
                p.V, seed, d_seed, decs, kmax, d_n_acc, d_out_tok);
  if (timed("decide_kernel")) timer->end(st, 0.0, 0.0);
  // the draw reads one (p, q) row pair per rejected sequence, one p row per bonus
  const char* n3 = vec ? "draw_kernel<true>" : "draw_kernel<false>";
  dim3 g3(p.n_chunks2, p.B);
  if (timed(n3)) timer->begin(st);
  if (vec)
    launch_kernel(draw_kernel<true>, g3, dim3(kThreads), 0, st, d_rows, d_seqs, decs, p.V, p.chunk2,
                  p.n_chunks2, seed, d_seed, picks);
  else
    launch_kernel(draw_kernel<false>, g3, dim3(kThreads), 0, st, d_rows, d_seqs, decs, p.V, p.chunk2,
                  p.n_chunks2, seed, d_seed, picks);
  if (timed(n3)) timer->end(st, 0.0, 0.0);
  launch_kernel(final_kernel, dim3(p.B), dim3(kWave), 0, st, d_seqs, d_draft_tok, decs, picks, p.n_chunks2, kmax,
                d_n_acc, d_out_tok);
  return hipGetLastError();
}

hipError_t launch_vocab_setup(int B, int kmax, const int32_t* d_k, const float* d_temp, const int64_t* d_ids,
                              const int32_t* d_base, const float* d_p, const float* d_q, int V, VRow* d_rows,
                              VSeq* d_seqs, int32_t* d_n_rows, hipStream_t st) {
  if (B <= 0 || B > kSetupMaxSeqs) return hipErrorInvalidValue;
  setup_kernel<<<1, kSetupMaxSeqs, 0, st>>>(B, kmax, d_k, d_temp, d_ids, d_base, d_p, d_q, V, d_rows, d_seqs,
                                            d_n_rows);
  return hipGetLastError();
}

size_t tree_ws_bytes(const VocabPlan& p) {
  return align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1) +
         align256(sizeof(float) * static_cast<size_t>(p.B) * kTreeMaxNodes * kTreeMaxNodes * kMaxChunks) +
         align256(sizeof(VPick) * static_cast<size_t>(p.B) * kTreeMaxNodes * kMaxChunks);
}

hipError_t launch_tree_pass(const VocabPlan& p, const VRow* d_rows, const VTreeSeq* d_seqs,
                            const VTreeNode* d_nodes, const int32_t* d_row_tok, uint64_t seed,
                            const uint64_t* d_seed, int kmax, int max_kids,
                            int32_t* d_n_acc, int32_t* d_out_tok, int32_t* d_out_path, void* d_ws,
                            hipStream_t st, KernelTimer* timer) {
  if (p.B == 0) return hipSuccess;
  if (p.n_chunks1 > kMaxChunks || kmax >= kTreeMaxNodes || max_kids < 0 || max_kids > kmax)
    return hipErrorInvalidValue;
  char* ws = static_cast<char*>(d_ws);
  VStat* stats = reinterpret_cast<VStat*>(ws);
  ws += align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1);
  float* zpart = reinterpret_cast<float*>(ws);
  ws += align256(sizeof(float) * static_cast<size_t>(p.B) * kTreeMaxNodes * kTreeMaxNodes * kMaxChunks);
  VPick* picks = reinterpret_cast<VPick*>(ws);
  auto timed = [&](const char* name) { return timer && timer->wants(name); };
  // the vector path needs every row 16-byte aligned: rows are whole fp32
  // vocabulary rows of 16-byte aligned buffers when V % 4 == 0
  const bool vec = (p.V % 4) == 0;
  dim3 g1(p.n_chunks1, p.n_rows);
  const char* n1 = vec ? "stats_kernel<true>" : "stats_kernel<false>";
  if (timed(n1)) timer->begin(st);
  if (vec)
    launch_kernel(stats_kernel<true>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1,
                  nullptr);
  else
    launch_kernel(stats_kernel<false>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1,
                  nullptr);
  if (timed(n1)) timer->end(st, 4.0 * p.n_rows * p.V, 0.0);
  // the decision after the statistics: a residual-mass pass per level, the
  // draws of every node, the walk (timed together as "tree_decision")
  if (timed("tree_decision")) timer->begin(st);
  const dim3 g2(p.n_chunks1, p.B * kTreeMaxNodes);
  for (int L = 1; L <= max_kids; ++L)
    launch_kernel(tree_z_kernel, g2, dim3(kThreads), 0, st, d_rows, d_seqs, d_nodes, stats, p.n_chunks1,
                  p.chunk1, p.V, L, zpart);
  launch_kernel(tree_draw_kernel, g2, dim3(kThreads), 0, st, d_rows, d_seqs, d_nodes, stats, p.n_chunks1,
                p.chunk1, p.V, seed, d_seed, zpart, picks);
  launch_kernel(tree_walk_kernel, dim3(p.B), dim3(kWave), 0, st, d_rows, d_seqs, d_nodes, d_row_tok, stats,
                p.n_chunks1, p.V, seed, d_seed, zpart, picks, kmax, d_n_acc, d_out_tok, d_out_path);
  if (timed("tree_decision")) timer->end(st, 0.0, 0.0);
  return hipGetLastError();
}

DraftPlan draft_plan(int n, int V) {
  DraftPlan p;
  p.n = n;
  p.V = V;
  chunking(n, V, p.chunk, p.n_chunks);
  return p;
}

size_t draft_ws_bytes(const DraftPlan& p) {
  return align256(sizeof(VPick) * static_cast<size_t>(p.n) * p.n_chunks);
}

hipError_t launch_draft_sample(const DraftPlan& p, const DRow* d_rows, uint64_t seed,
                               int32_t* d_tokens, void* d_ws, hipStream_t st, const uint64_t* d_seed) {
  if (p.n == 0) return hipSuccess;
  if (p.n_chunks > kMaxChunks) return hipErrorInvalidValue;
  VPick* picks = static_cast<VPick*>(d_ws);
  dim3 g(p.n_chunks, p.n);
  if (p.V % 4 == 0)
    draft_kernel<true><<<g, kThreads, 0, st>>>(p.V, d_rows, p.chunk, p.n_chunks, seed, d_seed, picks);
  else
    draft_kernel<false><<<g, kThreads, 0, st>>>(p.V, d_rows, p.chunk, p.n_chunks, seed, d_seed, picks);
  draft_final_kernel<<<p.n, kWave, 0, st>>>(d_rows, picks, p.n_chunks, d_tokens);
  return hipGetLastError();
}

hipError_t launch_draft_guide(int n, int V, const DRow* d_rows, float boost, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  draft_guide_kernel<<<n, kGuideThreads, 0, st>>>(V, d_rows, boost);
  return hipGetLastError();
}

hipError_t launch_philox_uniform(uint64_t seed, uint64_t seq_id, int32_t pos, int32_t purpose,
                                 int32_t n, float* out, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  philox_uniform_kernel<<<(n + 255) / 256, 256, 0, st>>>(seed, stream_id(seq_id, pos, purpose), n, out);
  return hipGetLastError();
}

}  // namespace spec
