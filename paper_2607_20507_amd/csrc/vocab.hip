// Vocabulary-wide decision pass of the verify step, for gfx950.
//
// Speculative sampling (the draft-and-verify rule CacheSpec's drafter follows,
// Section 3.4): draft x~_j is accepted iff u_j * q_j(x~_j) < p_j(x~_j); at the
// first rejection a token is drawn from norm(max(0, p_j - q_j)); if every draft
// is accepted a bonus token is drawn from p_{k+1}.  Categorical draws use the
// Gumbel-max trick, argmax_i (log w_i + G_i), with per-token Philox noise.
//
// Three launches, all HBM-streaming with 16-byte coalesced loads:
//   1. stats   grid (chunks, rows): per row chunk, max, first argmax and
//              sum exp((z - max) / T) in one online pass.
//   2. decide  grid (chunks, seqs): every workgroup of a sequence repeats the
//              cheap acceptance scan (one lane per draft, merged chunk stats,
//              two gathered logits, one Philox draw), then streams its chunk
//              of the one row that is sampled (residual or bonus).
//   3. final   one thread per sequence: merge chunk winners, write outputs.
// A greedy sequence (T = 0) needs no second pass: the first mismatch between
// a draft and the target's argmax decides, and that argmax is the token.

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
struct VDec {
  int32_t a, mode, token, pad;
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

__device__ __forceinline__ void stat_update4(float4 v, int base, float it, bool greedy, float& m,
                                             float& s, int& idx) {
  const float vm = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
  if (vm > m) {
    const int j = (v.x == vm) ? 0 : (v.y == vm) ? 1 : (v.z == vm) ? 2 : 3;
    if (!greedy) s = scaled(s, m, vm, it);
    m = vm;
    idx = base + j;
  }
  if (!greedy)
    s += __expf((v.x - m) * it) + __expf((v.y - m) * it) + __expf((v.z - m) * it) +
         __expf((v.w - m) * it);
}

__device__ __forceinline__ void stat_update1(float v, int i, float it, bool greedy, float& m,
                                             float& s, int& idx) {
  if (v > m) {
    if (!greedy) s = scaled(s, m, v, it);
    m = v;
    idx = i;
  }
  if (!greedy) s += __expf((v - m) * it);
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void stats_kernel(const VRow* __restrict__ rows, int V,
                                                         int chunk, VStat* __restrict__ stats,
                                                         int n_chunks) {
  const int r = blockIdx.y, c = blockIdx.x;
  const VRow row = rows[r];
  const float it = row.inv_t;
  const bool greedy = row.greedy != 0;
  const int beg = c * chunk;
  const int end = min(V, beg + chunk);
  float m = -INFINITY, s = 0.f;
  int idx = INT_MAX;
  if (VEC) {
    const float4* p4 = reinterpret_cast<const float4*>(row.ptr + beg);
    const int n4 = (end - beg) >> 2;
    int i = threadIdx.x;
    for (; i + 3 * kThreads < n4; i += 4 * kThreads) {
      float4 v0 = ld_stream(p4 + i);
      float4 v1 = ld_stream(p4 + i + kThreads);
      float4 v2 = ld_stream(p4 + i + 2 * kThreads);
      float4 v3 = ld_stream(p4 + i + 3 * kThreads);
      stat_update4(v0, beg + 4 * i, it, greedy, m, s, idx);
      stat_update4(v1, beg + 4 * (i + kThreads), it, greedy, m, s, idx);
      stat_update4(v2, beg + 4 * (i + 2 * kThreads), it, greedy, m, s, idx);
      stat_update4(v3, beg + 4 * (i + 3 * kThreads), it, greedy, m, s, idx);
    }
    for (; i < n4; i += kThreads) stat_update4(p4[i], beg + 4 * i, it, greedy, m, s, idx);
  } else {
    for (int i = beg + threadIdx.x; i < end; i += kThreads)
      stat_update1(row.ptr[i], i, it, greedy, m, s, idx);
  }
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

__device__ __forceinline__ void pick_update(float sc, int i, float& best, int& bi) {
  if (sc > best || (sc == best && i < bi)) {
    best = sc;
    bi = i;
  }
}

// Merge all chunk statistics of one row.  Chunk records are read in batches
// of kStatBatch (indexes clamped, so that every load of a batch is in flight
// before the first is used) and still taken in chunk order.
constexpr int kStatBatch = 8;

__device__ __forceinline__ void row_stats(const VStat* st, int n_chunks, float it, bool greedy,
                                          float& M, float& S, int& idx) {
  M = -INFINITY;
  idx = INT_MAX;
  for (int c0 = 0; c0 < n_chunks; c0 += kStatBatch) {
    VStat v[kStatBatch];
#pragma unroll
    for (int b = 0; b < kStatBatch; ++b) v[b] = st[min(c0 + b, n_chunks - 1)];
#pragma unroll
    for (int b = 0; b < kStatBatch; ++b)
      if (c0 + b < n_chunks && v[b].m > M) {  // chunks in index order: the first chunk holding the max wins ties
        M = v[b].m;
        idx = v[b].idx;
      }
  }
  S = 0.f;
  if (!greedy)
    for (int c0 = 0; c0 < n_chunks; c0 += kStatBatch) {
      VStat v[kStatBatch];
#pragma unroll
      for (int b = 0; b < kStatBatch; ++b) v[b] = st[min(c0 + b, n_chunks - 1)];
#pragma unroll
      for (int b = 0; b < kStatBatch; ++b)
        if (c0 + b < n_chunks) S += scaled(v[b].s, v[b].m, M, it);
    }
}

// Best pick (and fallback pick) over a row's chunk records, in chunk order.
__device__ __forceinline__ void merge_picks(const VPick* pk, int n_chunks, float& best, int& bi, float& fb,
                                            int& fi) {
  for (int c0 = 0; c0 < n_chunks; c0 += kStatBatch) {
    VPick v[kStatBatch];
#pragma unroll
    for (int b = 0; b < kStatBatch; ++b) v[b] = pk[min(c0 + b, n_chunks - 1)];
#pragma unroll
    for (int b = 0; b < kStatBatch; ++b)
      if (c0 + b < n_chunks) {
        pick_update(v[b].score, v[b].idx, best, bi);
        pick_update(v[b].fb_score, v[b].fb_idx, fb, fi);
      }
  }
}

__device__ __forceinline__ uint32_t word_of(uint4 w, int e) {
  return e == 0 ? w.x : e == 1 ? w.y : e == 2 ? w.z : w.w;
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void decide_kernel(
    const VRow* __restrict__ rows, const VSeq* __restrict__ seqs,
    const int32_t* __restrict__ draft_tok, const VStat* __restrict__ stats, int n_chunks1, int V,
    int chunk2, int n_chunks2, uint64_t seed, const uint64_t* __restrict__ seed_ptr,
    VPick* __restrict__ picks, VDec* __restrict__ decs) {
  const int b = blockIdx.y, c = blockIdx.x;
  const VSeq sq = seqs[b];
  const bool greedy = !(sq.t > 0.f);
  const float it = greedy ? 0.f : 1.f / sq.t;
  const uint64_t seq_id = (static_cast<uint64_t>(sq.seq_hi) << 32) | sq.seq_lo;
  const PhiloxKey key = philox_key(seed_ptr ? *seed_ptr : seed);

  __shared__ int s_a, s_tok;
  __shared__ float s_mp, s_sp, s_mq, s_sq;
  if (threadIdx.x < kWave) {
    const int j = threadIdx.x;  // 0-based draft index; lane k handles the bonus row
    bool acc = true;
    float Mp = 0.f, Sp = 1.f, Mq = 0.f, Sq = 1.f;
    int ap = 0, aq = 0;
    if (j <= sq.k) {
      row_stats(stats + static_cast<size_t>(sq.p_row + j) * n_chunks1, n_chunks1, it, greedy, Mp,
                Sp, ap);
    }
    if (j < sq.k) {
      const int x = draft_tok[sq.tok_row + j];
      if (static_cast<unsigned>(x) >= static_cast<unsigned>(V)) {
        acc = false;  // a draft id outside the vocabulary is never accepted
      } else if (greedy) {
        acc = (x == ap);
      } else {
        row_stats(stats + static_cast<size_t>(sq.q_row + j) * n_chunks1, n_chunks1, it, false, Mq,
                  Sq, aq);
        const float zp = rows[sq.p_row + j].ptr[x];
        const float zq = rows[sq.q_row + j].ptr[x];
        const float px = __expf((zp - Mp) * it) / Sp;
        const float qx = __expf((zq - Mq) * it) / Sq;
        const uint4 w = philox_block(key, stream_id(seq_id, sq.base_pos + j + 1, 1 /*ACCEPT*/), 0);
        acc = (u01(w.x) * qx < px);
      }
    }
    const uint64_t rej = ~__ballot(acc);
    const int a = (rej == 0) ? sq.k : min(sq.k, static_cast<int>(__ffsll(static_cast<long long>(rej))) - 1);
    if (j == a) {
      s_a = a;
      s_tok = ap;
      s_mp = Mp;
      s_sp = Sp;
      s_mq = Mq;
      s_sq = Sq;
    }
  }
  __syncthreads();
  const int a = s_a;
  const int mode = greedy ? kGreedy : (a < sq.k ? kResample : kBonus);
  if (c == 0 && threadIdx.x == 0) decs[b] = VDec{a, mode, s_tok, 0};
  if (mode == kGreedy) return;

  const float Mp = s_mp, Sp = s_sp, Mq = s_mq, Sq = s_sq;
  const float* zp = rows[sq.p_row + a].ptr;
  const float* zq = (mode == kResample) ? rows[sq.q_row + a].ptr : nullptr;
  const StreamId sid = stream_id(seq_id, sq.base_pos + a + 1, mode == kResample ? 2 : 3);
  const float rp = 1.f / Sp, rq = 1.f / Sq;

  float best = -INFINITY, fb = -INFINITY;
  int bi = INT_MAX, fi = INT_MAX;
  const int beg = c * chunk2;
  const int end = min(V, beg + chunk2);
  auto score = [&](float p_logit, float q_logit, uint32_t word, int i) {
    const float g = gumbel_of(word);
    const float lp = (p_logit - Mp) * it;  // log p_i + log S_p
    if (mode == kResample) {
      const float r = __expf(lp) * rp - __expf((q_logit - Mq) * it) * rq;
      const float sc = (r > 0.f) ? logf(r) + g : -INFINITY;
      pick_update(sc, i, best, bi);
      pick_update(lp + g, i, fb, fi);
    } else {
      pick_update(lp + g, i, best, bi);
    }
  };
  if (VEC) {
    // batches of 4 float4 per thread (clamped loads, all in flight before the
    // first is used), then the same per-element order as one at a time
    const int e4 = end >> 2;
    for (int i0 = (beg >> 2) + threadIdx.x; i0 < e4; i0 += 4 * kThreads) {
      float4 pv[4], qv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = min(i0 + u * kThreads, e4 - 1);
        pv[u] = reinterpret_cast<const float4*>(zp)[j];
        qv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (mode == kResample) qv[u] = reinterpret_cast<const float4*>(zq)[j];  // zq is null otherwise
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
      score(zp[i], zq ? zq[i] : 0.f, word_of(w, i & 3), i);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float b2 = __shfl_xor(best, o, kWave);
    const int i2 = __shfl_xor(bi, o, kWave);
    pick_update(b2, i2, best, bi);
    const float f2 = __shfl_xor(fb, o, kWave);
    const int j2 = __shfl_xor(fi, o, kWave);
    pick_update(f2, j2, fb, fi);
  }
  __shared__ VPick sp[kThreads / kWave];
  const int wv = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) sp[wv] = VPick{best, bi, fb, fi};
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kThreads / kWave; ++k) {
      pick_update(sp[k].score, sp[k].idx, best, bi);
      pick_update(sp[k].fb_score, sp[k].fb_idx, fb, fi);
    }
    picks[static_cast<size_t>(b) * n_chunks2 + c] = VPick{best, bi, fb, fi};
  }
}

__global__ void final_kernel(const VSeq* __restrict__ seqs, const int32_t* __restrict__ draft_tok,
                             const VDec* __restrict__ decs, const VPick* __restrict__ picks,
                             int n_chunks2, int B, int kmax, int32_t* __restrict__ n_acc,
                             int32_t* __restrict__ out_tok) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const VSeq sq = seqs[b];
  const VDec d = decs[b];
  int t = d.token;
  if (d.mode != kGreedy) {
    float best = -INFINITY, fb = -INFINITY;
    int bi = INT_MAX, fi = INT_MAX;
    merge_picks(picks + static_cast<size_t>(b) * n_chunks2, n_chunks2, best, bi, fb, fi);
    // an empty residual (only possible when p == q) falls back to drawing from p
    t = (best == -INFINITY) ? fi : bi;
  }
  n_acc[b] = d.a;
  int32_t* o = out_tok + static_cast<size_t>(b) * (kmax + 1);
  for (int j = 0; j <= kmax; ++j) o[j] = (j < d.a) ? draft_tok[sq.tok_row + j] : (j == d.a ? t : -1);
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
    // batches of 4 float4 per thread, as in decide_kernel
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
          pick_update(v.x * it + gumbel_of(w.x), 4 * i4, best, bi);
          pick_update(v.y * it + gumbel_of(w.y), 4 * i4 + 1, best, bi);
          pick_update(v.z * it + gumbel_of(w.z), 4 * i4 + 2, best, bi);
          pick_update(v.w * it + gumbel_of(w.w), 4 * i4 + 3, best, bi);
        }
      }
    }
  } else {
    for (int i = beg + threadIdx.x; i < end; i += kThreads) {
      if (greedy) {
        pick_update(z[i], i, best, bi);
      } else {
        const uint4 w = philox_block(key, sid, static_cast<uint32_t>(i >> 2));
        pick_update(z[i] * it + gumbel_of(word_of(w, i & 3)), i, best, bi);
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float b2 = __shfl_xor(best, o, kWave);
    const int i2 = __shfl_xor(bi, o, kWave);
    pick_update(b2, i2, best, bi);
  }
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

// One workgroup per row: row maximum, then the guide token's logit becomes
// maximum + boost (all reads of the row finish before the write).
// One workgroup of 1024 threads per guided row: the row maximum with 16-byte
// streaming loads, four in flight per thread, then z[guide] = max + boost.
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

__global__ void draft_final_kernel(const DRow* __restrict__ rows, const VPick* __restrict__ picks,
                                   int n_chunks, int n, int32_t* __restrict__ tokens) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  float best = -INFINITY, fb = -INFINITY;
  int bi = INT_MAX, fi = INT_MAX;
  merge_picks(picks + static_cast<size_t>(r) * n_chunks, n_chunks, best, bi, fb, fi);
  tokens[rows[r].out] = bi;
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
  chunk = (V + want - 1) / want;
  chunk = (chunk + 1023) / 1024 * 1024;
  n_chunks = (V + chunk - 1) / chunk;
}

}  // namespace

VocabPlan vocab_plan(int B, int n_rows, int V) {
  VocabPlan p;
  p.B = B;
  p.n_rows = n_rows;
  p.V = V;
  chunking(n_rows, V, p.chunk1, p.n_chunks1);
  chunking(B, V, p.chunk2, p.n_chunks2);
  return p;
}

size_t vocab_ws_bytes(const VocabPlan& p) {
  return align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1) +
         align256(sizeof(VPick) * static_cast<size_t>(p.B) * p.n_chunks2) +
         align256(sizeof(VDec) * static_cast<size_t>(p.B));
}

hipError_t launch_vocab_pass(const VocabPlan& p, const VRow* d_rows, const VSeq* d_seqs,
                             const int32_t* d_draft_tok, uint64_t seed, int kmax, int32_t* d_n_acc,
                             int32_t* d_out_tok, void* d_ws, hipStream_t st, KernelTimer* timer,
                             const uint64_t* d_seed) {
  if (p.B == 0) return hipSuccess;
  char* ws = static_cast<char*>(d_ws);
  VStat* stats = reinterpret_cast<VStat*>(ws);
  ws += align256(sizeof(VStat) * static_cast<size_t>(p.n_rows) * p.n_chunks1);
  VPick* picks = reinterpret_cast<VPick*>(ws);
  ws += align256(sizeof(VPick) * static_cast<size_t>(p.B) * p.n_chunks2);
  VDec* decs = reinterpret_cast<VDec*>(ws);
  const bool vec = (p.V % 4) == 0;
  dim3 g1(p.n_chunks1, p.n_rows);
  const bool timed = timer && timer->wants(vec ? "stats_kernel<true>" : "stats_kernel<false>");
  if (timed) timer->begin(st);
  if (vec)
    launch_kernel(stats_kernel<true>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1);
  else
    launch_kernel(stats_kernel<false>, g1, dim3(kThreads), 0, st, d_rows, p.V, p.chunk1, stats, p.n_chunks1);
  if (timed) timer->end(st, 4.0 * p.n_rows * p.V, 0.0);
  dim3 g2(p.n_chunks2, p.B);
  if (vec)
    decide_kernel<true><<<g2, kThreads, 0, st>>>(d_rows, d_seqs, d_draft_tok, stats, p.n_chunks1,
                                                 p.V, p.chunk2, p.n_chunks2, seed, d_seed, picks, decs);
  else
    decide_kernel<false><<<g2, kThreads, 0, st>>>(d_rows, d_seqs, d_draft_tok, stats, p.n_chunks1,
                                                  p.V, p.chunk2, p.n_chunks2, seed, d_seed, picks, decs);
  final_kernel<<<(p.B + 63) / 64, 64, 0, st>>>(d_seqs, d_draft_tok, decs, picks, p.n_chunks2, p.B,
                                               kmax, d_n_acc, d_out_tok);
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
  VPick* picks = static_cast<VPick*>(d_ws);
  dim3 g(p.n_chunks, p.n);
  if (p.V % 4 == 0)
    draft_kernel<true><<<g, kThreads, 0, st>>>(p.V, d_rows, p.chunk, p.n_chunks, seed, d_seed, picks);
  else
    draft_kernel<false><<<g, kThreads, 0, st>>>(p.V, d_rows, p.chunk, p.n_chunks, seed, d_seed, picks);
  draft_final_kernel<<<(p.n + 63) / 64, 64, 0, st>>>(d_rows, picks, p.n_chunks, p.n, d_tokens);
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
