// Paged causal grouped-query attention on gfx950.
//
// Row r of sequence s sits at absolute position pos_r and attends keys
// 0..pos_r of its own cache (the verify window's K/V are written before this
// kernel runs, so drafts see each other causally).  Query head h reads kv head
// h / (Hq / Hkv).  Scale 1/sqrt(hd).
//
// KV pages hold 16 tokens per (page, kv head) block, in the operand order of
// kv_layout.h for bf16 (K as [16][hd] and V transposed as [hd][16] for fp32).
// The bf16 kernel gives each workgroup of W waves one (rows of one sequence,
// kv head, key range) work item and runs both products on MFMA:
//   S^T = K Q^T : A = 16 keys x 32 dims of K, B = 32 dims x 16 query vectors.
//   O^T = V^T P^T: A = 16 dims x 32 keys of V^T, B = P^T.
// Keys inside each 32-key chunk are permuted (A row i of key tile h reads key
// 8 (i / 4) + 4 h + i % 4) so that the S^T accumulators a lane ends up with are
// exactly the 8 consecutive keys it must supply as the P^T operand, and the
// softmax statistics of query vector (l % 16) stay lane-local: no shuffles of
// P, no LDS in the loop.  With the page layout of kv_layout.h every K and V^T
// operand load of a wave reads two contiguous 512-byte runs.  Long contexts
// are split into key ranges (multiples of 32) whose unnormalised partials a
// combine kernel merges.

#include <algorithm>
#include <cmath>
#include <cstdio>

#include "attention.h"
#include "common.h"

namespace spec {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kAttnStagedPages = 256;  // page ids of one work item kept in LDS (4096 keys)

__device__ __forceinline__ uint32_t mask_pair(uint32_t w, int valid) {
  // keep the first `valid` (0, 1, 2) bf16 halves of a 32-bit word
  return valid >= 2 ? w : (valid == 1 ? (w & 0xFFFFu) : 0u);
}

// W waves per workgroup share one work item: wave w takes the 32-key chunks
// w, w + W, ... of the item's key range, and the waves' softmax states are
// merged through LDS at the end (exact rescaling by exp2(m_w - m)).
template <int HD, int NT, int W, bool TREE>
__device__ __forceinline__ void attn_bf16_body(const AttnArgs& a, const AttnItem* __restrict__ items) {
  constexpr int DS = HD / 32;   // MFMA k-steps over the head dim
  constexpr int DT = HD / 16;   // 16-dim output tiles
  const AttnItem it = items[blockIdx.x];
  const int gkv = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int g = lane >> 4, l16 = lane & 15;
  const int G = a.Hq / a.Hkv;
  const int M = it.nrows * G;
  const bf16_t* q = static_cast<const bf16_t*>(a.q);
  const bf16_t* kp = static_cast<const bf16_t*>(a.kpool);
  const bf16_t* vp = static_cast<const bf16_t*>(a.vpool);
  const int32_t* pt = a.page_table + static_cast<size_t>(it.seq) * a.max_pages;
  // the item's page ids, staged once in LDS so that no chunk waits on a
  // page-table load before its K / V loads can go out (items spanning more
  // pages than the stage holds read the table directly)
  __shared__ int32_t s_pt[kAttnStagedPages];
  const int p0 = it.t0 >> 4;
  const int np = it.t1 > it.t0 ? ((it.t1 - 1) >> 4) - p0 + 1 : 0;
  const bool staged = np <= kAttnStagedPages;
  if (staged)
    for (int i = threadIdx.x; i < np; i += kWave * W) s_pt[i] = pt[p0 + i];
  __syncthreads();
  auto page = [&](int t) { return staged ? s_pt[(t >> 4) - p0] : pt[t >> 4]; };

  uint4 qf[NT][DS];
  int vpos[NT];
  uint32_t tmask[NT];
  bool vval[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int m = 16 * nt + l16;
    vval[nt] = m < M;
    const int mm = vval[nt] ? m : 0;
    if constexpr (TREE) {
      // vpos: the last index every row sees; beyond it the tree's bits
      vpos[nt] = a.tree_base[it.row0 + mm / G];
      tmask[nt] = a.tree_mask[it.row0 + mm / G];
    } else {
      vpos[nt] = it.pos0 + mm / G;
      tmask[nt] = 0u;
    }
    const bf16_t* base =
        q + (static_cast<size_t>(it.row0 + mm / G) * a.Hq + gkv * G + mm % G) * HD + g * 8;
#pragma unroll
    for (int s = 0; s < DS; ++s)
      qf[nt][s] = vval[nt] ? reinterpret_cast<const uint4*>(base)[4 * s] : make_uint4(0, 0, 0, 0);
  }
  const float scale = kLog2e / sqrtf(static_cast<float>(HD));
  float mrun[NT], lrun[NT];
  f32x4 acc[DT][NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    mrun[nt] = -INFINITY;
    lrun[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // K and V^T operands of one 32-key chunk (keys past t1 are clamped to a
  // valid address; their scores are masked and their V entries zeroed)
  auto load_k = [&](int c0, uint4 (&kf)[2][DS]) {
    // lanes 0-7 / 8-15 of a group read the chunk's first / second page:
    // unit ((s * 2 + hh) * 4 + g) * 8 + l16 % 8 of the page's K block holds
    // dims 32 s + 8 g .. of key 8 (l16 / 4) + 4 hh + l16 % 4 (kv_layout.h)
    const int tk = min(c0 + 16 * (l16 >> 3), it.t1 - 1);
    const uint4* kb = reinterpret_cast<const uint4*>(kp + static_cast<size_t>(page(tk) * a.Hkv + gkv) * 16 * HD);
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int s = 0; s < DS; ++s) kf[hh][s] = ld_stream(kb + ((s * 2 + hh) * 4 + g) * 8 + (l16 & 7));
  };
  auto load_v = [&](int c0, uint4 (&vf)[DT]) {
    // V^T: unit (dt * 2 + g % 2) * 16 + l16 holds keys 8 (g % 2) .. + 7 of
    // dim 16 dt + l16 of page (c0 + 8 g) / 16
    const int tvc = min(c0 + 8 * g, it.t1 - 1);
    const uint4* vb = reinterpret_cast<const uint4*>(vp + static_cast<size_t>(page(tvc) * a.Hkv + gkv) * HD * 16);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vf[dt] = ld_stream(vb + (dt * 2 + (g & 1)) * 16 + l16);
  };
  // One K and one V^T buffer: the next chunk's K is loaded once this chunk's
  // scores are computed, its V^T once this chunk's output update is done
  // (loads are unconditional, clamped past the end, so that the compiler's
  // waits stay exact).
  uint4 kf[2][DS], vf[DT];
  const int cfirst = it.t0 + 32 * wave;
  if (cfirst < it.t1) {
    load_k(cfirst, kf);
    load_v(cfirst, vf);
  }
  for (int c0 = cfirst; c0 < it.t1; c0 += 32 * W) {
    const int cn = min(c0 + 32 * W, it.t1 - 1);
    const int tv = c0 + 8 * g;
    const int nvalid = min(max(it.t1 - tv, 0), 8);

    f32x4 sc[NT][2];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        s0 = mfma16x16x32(kf[0][s], qf[nt][s], s0);
        s1 = mfma16x16x32(kf[1][s], qf[nt][s], s1);
      }
      sc[nt][0] = s0;
      sc[nt][1] = s1;
    }
    load_k(cn, kf);
    uint4 pf[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float sv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int t = c0 + 8 * g + j;
        const float raw = (j < 4) ? sc[nt][0][j] : sc[nt][1][j - 4];
        bool ok = vval[nt] && t < it.t1;
        if constexpr (TREE) {
          const int rel = t - vpos[nt];
          ok = ok && (rel <= 0 || (rel <= 32 && ((tmask[nt] >> (rel - 1)) & 1u)));
        } else {
          ok = ok && t <= vpos[nt];
        }
        sv[j] = ok ? raw * scale : -INFINITY;
      }
      float mx = sv[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, sv[j]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float mnew = fmaxf(mrun[nt], mx);
      float p[8];
      float alpha = 1.f;
      if (mnew == -INFINITY) {
#pragma unroll
        for (int j = 0; j < 8; ++j) p[j] = 0.f;
      } else {
        alpha = (mrun[nt] == -INFINITY) ? 0.f : exp2f(mrun[nt] - mnew);
#pragma unroll
        for (int j = 0; j < 8; ++j) p[j] = exp2f(sv[j] - mnew);
      }
      float ps = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) ps += p[j];
      lrun[nt] = lrun[nt] * alpha + ps;
      mrun[nt] = mnew;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[dt][nt] *= alpha;
      pf[nt] = make_uint4(pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]),
                          pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7]));
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      uint4 v = vf[dt];
      if (nvalid < 8) {
        v.x = mask_pair(v.x, nvalid);
        v.y = mask_pair(v.y, nvalid - 2);
        v.z = mask_pair(v.z, nvalid - 4);
        v.w = mask_pair(v.w, nvalid - 6);
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[dt][nt] = mfma16x16x32(v, pf[nt], acc[dt][nt]);
    }
    load_v(cn, vf);
  }

  float ltot[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float lt = lrun[nt];
    lt += __shfl_xor(lt, 16, kWave);
    lt += __shfl_xor(lt, 32, kWave);
    ltot[nt] = lt;
  }
  if (W > 1) {
    // waves 1..W-1 hand their state to wave 0 (same lane layout in every wave)
    __shared__ float s_acc[W > 1 ? W - 1 : 1][NT][DT][4][kWave];
    __shared__ float s_ml[W > 1 ? W - 1 : 1][NT][2][kWave];
    if (wave > 0) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        s_ml[wave - 1][nt][0][lane] = mrun[nt];
        s_ml[wave - 1][nt][1][lane] = ltot[nt];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) s_acc[wave - 1][nt][dt][r][lane] = acc[dt][nt][r];
      }
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float mm = mrun[nt];
      for (int w = 0; w < W - 1; ++w) mm = fmaxf(mm, s_ml[w][nt][0][lane]);
      if (mm == -INFINITY) continue;  // no key of the item for this query vector
      const float e0 = (mrun[nt] == -INFINITY) ? 0.f : exp2f(mrun[nt] - mm);
      float lt = ltot[nt] * e0;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[dt][nt] *= e0;
      for (int w = 0; w < W - 1; ++w) {
        const float mw = s_ml[w][nt][0][lane];
        const float ew = (mw == -INFINITY) ? 0.f : exp2f(mw - mm);
        lt += ew * s_ml[w][nt][1][lane];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[dt][nt][r] += ew * s_acc[w][nt][dt][r][lane];
      }
      mrun[nt] = mm;
      ltot[nt] = lt;
    }
  }
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const float lt = ltot[nt];
    const int m = 16 * nt + l16;
    if (m >= M) continue;
    if (it.part < 0) {
      const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
      bf16_t* o = static_cast<bf16_t*>(a.out) +
                  (static_cast<size_t>(it.row0 + m / G) * a.Hq + gkv * G + m % G) * HD;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const f32x4 v = acc[dt][nt];
        *reinterpret_cast<uint2*>(o + 16 * dt + 4 * g) =
            make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
      }
    } else {
      const size_t pm = static_cast<size_t>(it.part * a.Hkv + gkv) * 64 + m;
      float* po = a.part_o + pm * HD;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        *reinterpret_cast<float4*>(po + 16 * dt + 4 * g) =
            make_float4(acc[dt][nt][0], acc[dt][nt][1], acc[dt][nt][2], acc[dt][nt][3]);
      if (g == 0) {
        a.part_ml[pm * 2] = mrun[nt];
        a.part_ml[pm * 2 + 1] = lt;
      }
    }
  }
}

// One workgroup per (group, kv head, 4 query vectors), one thread per (query
// vector, DPT consecutive head dims: DPT = 4 (float4 loads of the partial
// outputs) for head dim 128, 1 for head dim 64, as measured).  Up
// to kCombineOnePass parts: every part's (max, sum) and output vector is
// loaded before the first is used (one round trip), then the maximum and the
// weighted sums.  More parts: two passes (maximum, then weighted sums), each
// issuing batches of 8 independent loads.  Both sum the parts in index order,
// per element as a one-element-per-thread combine would.
constexpr int kCombineQv = 4;
constexpr int kCombineOnePass = 32;

template <int DPT>
struct CombVec;
template <>
struct CombVec<1> {
  float v[1];
  __device__ __forceinline__ void load(const float* p) { v[0] = *p; }
};
template <>
struct CombVec<4> {
  float v[4];
  __device__ __forceinline__ void load(const float* p) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  }
};

template <int HD, int NT, int W>
__global__ __launch_bounds__(64 * W, NT <= 2 ? 2 : 1) void attn_bf16_kernel(AttnArgs a, const AttnItem* __restrict__ items) {
  attn_bf16_body<HD, NT, W, false>(a, items);
}

// The same with the rows' tree masks (tree verification).
template <int HD, int NT, int W>
__global__ __launch_bounds__(64 * W, NT <= 2 ? 2 : 1) void attn_tree_bf16_kernel(AttnArgs a,
                                                                                  const AttnItem* __restrict__ items) {
  attn_bf16_body<HD, NT, W, true>(a, items);
}

// ---------------------------------------------------------------------------
// Causal prefill: long runs of consecutive rows of one sequence.  One
// workgroup of 8 waves (two per SIMD, so that one wave's softmax arithmetic
// overlaps the other's MFMAs) per (block of 256 / G rows, kv head): its 256
// query vectors (rows x the G query heads of the kv head) share every K / V
// load.  The keys 0 .. last row's position are brought into LDS 64 at a time
// (four pages of K and of V, three stage buffers, two stages in flight) by
// direct-to-LDS loads of whole page blocks, and each wave runs both products
// for its own 32 query vectors (2 tiles) from there, with the key permutation
// and lane-local softmax of attn_bf16_body.  Each wave sees every key of its
// rows, so it normalises its own output: no key splits, no combine.
// The running maximum of a query vector is raised only when a score exceeds
// it by more than 2^8 (scores are base-2 logits): each lane compares its own
// 8 scores against it, and only when some lane of the wave finds a larger
// one does the wave take the cross-lane maximum and rescale its output
// accumulators.  Probabilities stay below 2^8 in between; the shared maximum
// is the same in every lane of a query vector, so the products stay exact.
// Chunks entirely at or below every row of a wave skip the causal mask.
// Two fp32 -> bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
constexpr int kPrefillStagedPages = 1024;  // page ids kept in LDS (16384 keys)
constexpr float kPrefillRescaleLog2 = 8.f;

template <int HD>
__global__ __launch_bounds__(512, 1) void attn_prefill_bf16_kernel(AttnArgs a, const AttnItem* __restrict__ items) {
  constexpr int DS = HD / 32;    // MFMA k-steps over the head dim
  constexpr int DT = HD / 16;    // 16-dim output tiles
  constexpr int NT = 2;          // 16-vector query tiles per wave
  constexpr int NW = 8;          // waves
  constexpr int BU = 2 * HD;     // 16-byte units of one (page, kv head) block
  constexpr int SU = 4 * BU;     // units of K (and of V) per 64-key stage
  constexpr int NB = 3;          // stage buffers
  constexpr int LPW = 2 * SU / (64 * NW);  // direct-to-LDS loads per wave per stage
  __shared__ uint4 sk[NB][SU], sv[NB][SU];
  __shared__ int32_t s_pt[kPrefillStagedPages];
  const int gkv = blockIdx.x % a.Hkv;
  const AttnItem it = items[blockIdx.x / a.Hkv];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform: load bases in SGPRs
  const int g = lane >> 4, l16 = lane & 15;
  const int G = a.Hq / a.Hkv;
  const bf16_t* q = static_cast<const bf16_t*>(a.q);
  const bf16_t* kp = static_cast<const bf16_t*>(a.kpool);
  const bf16_t* vp = static_cast<const bf16_t*>(a.vpool);
  const int32_t* pt = a.page_table + static_cast<size_t>(it.seq) * a.max_pages;
  const int t1 = it.t1;                 // keys 0 .. t1 - 1 (t0 = 0)
  const int np = (t1 + 15) >> 4;
  const int ns = (t1 + 63) >> 6;        // stages
  // (the planner keeps t1 <= 16 kPrefillStagedPages)
  for (int i = threadIdx.x; i < np; i += 64 * NW) s_pt[i] = pt[i];
  __syncthreads();

  // stage j (keys 64 j ..) into buffer b: wave w moves one page block, K of
  // page w of the stage for w < 4, V of page w - 4 after (its LPW loads of
  // 64 units each); pages past the sequence's last clamped to it (those keys
  // are masked)
  static_assert(LPW * 64 == BU && NW == 8, "one page block per wave and stage");
  const bool wv = wave >= 4;
  const int wpg = wave & 3;
  auto issue = [&](int j, int b) {
    const int page = __builtin_amdgcn_readfirstlane(s_pt[min(4 * j + wpg, np - 1)]);
    const bf16_t* blk = (wv ? vp : kp) + static_cast<size_t>(page * a.Hkv + gkv) * 16 * HD;
    const uint32_t dst = lds_addr(wv ? &sv[b][wpg * BU] : &sk[b][wpg * BU]);
#pragma unroll
    for (int i = 0; i < LPW; ++i) load_lds16(blk, (i * 64 + lane) * 16, dst + i * 1024);
  };

  uint4 qf[NT][DS];
  bool vval[NT];
  int vpos[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int m = 32 * wave + 16 * nt + l16;
    vval[nt] = m / G < it.nrows;
    const int mm = vval[nt] ? m : 0;
    vpos[nt] = it.pos0 + mm / G;
    const bf16_t* base = q + (static_cast<size_t>(it.row0 + mm / G) * a.Hq + gkv * G + mm % G) * HD + g * 8;
#pragma unroll
    for (int s = 0; s < DS; ++s)
      qf[nt][s] = vval[nt] ? reinterpret_cast<const uint4*>(base)[4 * s] : make_uint4(0, 0, 0, 0);
  }
  // the last key each query vector sees (-1: none, a padding vector)
  int klim[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) klim[nt] = vval[nt] ? min(vpos[nt], t1 - 1) : -1;
  // the wave's rows: positions pos_lo .. pos_hi
  const int pos_lo = it.pos0 + (32 * wave) / G;
  const int pos_hi = it.pos0 + min((32 * wave + 31) / G, it.nrows - 1);
  const float scale = kLog2e / sqrtf(static_cast<float>(HD));
  float mrun[NT], lrun[NT];
  f32x4 acc[DT][NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    mrun[nt] = -INFINITY;
    lrun[nt] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[dt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // one 32-key chunk (keys c0 .., pages 2 h, 2 h + 1 of buffer b)
  // K and V^T operands of chunk h of buffer b, read from LDS
  auto read_k = [&](int b, int h, uint4 (&kf)[2][DS]) {
    const uint4* kb = &sk[b][(2 * h + (l16 >> 3)) * BU];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int s = 0; s < DS; ++s) kf[hh][s] = kb[((s * 2 + hh) * 4 + g) * 8 + (l16 & 7)];
  };
  auto read_v = [&](int b, int h, uint4 (&vf)[DT]) {
    const uint4* vb = &sv[b][(2 * h + (g >> 1)) * BU];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) vf[dt] = vb[(dt * 2 + (g & 1)) * 16 + l16];
  };
  auto chunk = [&](int c0, const uint4 (&kf)[2][DS], const uint4 (&vf)[DT]) {
    // every key at or below every row of the wave and inside the sequence
    const bool full = c0 + 31 <= pos_lo && c0 + 31 < t1;
    uint4 pf[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        s0 = mfma16x16x32(kf[0][s], qf[nt][s], s0);
        s1 = mfma16x16x32(kf[1][s], qf[nt][s], s1);
      }
      float raw[8];  // raw scores, -inf where masked
#pragma unroll
      for (int j = 0; j < 8; ++j) raw[j] = (j < 4) ? s0[j] : s1[j - 4];
      if (!full) {
        asm volatile("");  // keeps the mask a branch around diagonal chunks (not selects everywhere)
#pragma unroll
        for (int j = 0; j < 8; ++j) raw[j] = (c0 + 8 * g + j <= klim[nt]) ? raw[j] : -INFINITY;
      }
      float mx = raw[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, raw[j]);
      mx *= scale;  // base-2 logit (scale > 0)
      if (__any(mx > mrun[nt] + kPrefillRescaleLog2)) {
        // the query vector's maximum over the chunk, from all lanes holding it
        mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        const bool grow = mx > mrun[nt] + kPrefillRescaleLog2;
        const float alpha = grow ? ((mrun[nt] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mrun[nt] - mx)) : 1.f;
        if (grow) mrun[nt] = mx;
        lrun[nt] *= alpha;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[dt][nt] *= alpha;
      }
      // p = 2^(raw scale - m): one FMA per score; with no maximum yet (no key
      // of the query vector so far) every p is 0
      const float mneg = (mrun[nt] == -INFINITY) ? -INFINITY : -mrun[nt];
      float p[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) p[j] = __builtin_amdgcn_exp2f(fmaf(raw[j], scale, mneg));
      float ps = 0.f;
#pragma unroll
      for (int j = 0; j < 8; ++j) ps += p[j];
      lrun[nt] += ps;
      pf[nt] = make_uint4(cvt_pk_bf16(p[0], p[1]), cvt_pk_bf16(p[2], p[3]), cvt_pk_bf16(p[4], p[5]),
                          cvt_pk_bf16(p[6], p[7]));
    }
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[dt][nt] = mfma16x16x32(vf[dt], pf[nt], acc[dt][nt]);
  };

  issue(0, 0);
  if (ns > 1) issue(1, 1);
  for (int j = 0; j < ns; ++j) {
    // stage j has landed (stage j + 1 may still be in flight), every wave is
    // done with stage j - 1, whose buffer stage j + 2 now fills
    if (j + 1 < ns) {
      SPEC_WAIT_VM_LDS(LPW);
    } else {
      SPEC_WAIT_VM_LDS(0);
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (j + 2 < ns) issue(j + 2, (j + 2) % NB);
    const int b = j % NB;
    if (j == ns - 1 && t1 < 64 * ns) {
      // keys past the sequence in the last stage hold stale or uninitialised
      // V (their probabilities are 0, but 0 x NaN is not): zero them in LDS.
      // Unit ((d / 16) 2 + k / 8) 16 + d % 16 of a page block holds keys
      // 8 (k / 8) .. + 7 of dim d.
      for (int u = threadIdx.x; u < SU; u += 64 * NW) {
        const int k0 = 64 * j + (u / BU) * 16 + ((u % BU) / 16 % 2) * 8;
        const int keep = min(max(t1 - k0, 0), 8);
        if (keep < 8) {
          uint4 v = sv[b][u];
          v.x = mask_pair(v.x, keep);
          v.y = mask_pair(v.y, keep - 2);
          v.z = mask_pair(v.z, keep - 4);
          v.w = mask_pair(v.w, keep - 6);
          sv[b][u] = v;
        }
      }
      __syncthreads();
    }
    // the first chunk's operands and the second's K read up front, so that
    // their LDS latency hides under the first chunk's arithmetic (the
    // second's V^T after it: registers)
    uint4 kf0[2][DS], vf0[DT], kf1[2][DS], vf1[DT];
    read_k(b, 0, kf0);
    read_v(b, 0, vf0);
    read_k(b, 1, kf1);
    if (64 * j <= pos_hi) chunk(64 * j, kf0, vf0);  // else above every row of this wave
    read_v(b, 1, vf1);
    if (64 * j + 32 <= pos_hi) chunk(64 * j + 32, kf1, vf1);
  }

#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float lt = lrun[nt];
    lt += __shfl_xor(lt, 16, kWave);
    lt += __shfl_xor(lt, 32, kWave);
    const int m = 32 * wave + 16 * nt + l16;
    if (!vval[nt]) continue;
    const float inv = (lt > 0.f) ? 1.f / lt : 0.f;
    bf16_t* o = static_cast<bf16_t*>(a.out) + (static_cast<size_t>(it.row0 + m / G) * a.Hq + gkv * G + m % G) * HD;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const f32x4 v = acc[dt][nt];
      *reinterpret_cast<uint2*>(o + 16 * dt + 4 * g) =
          make_uint2(pack_bf16x2(v[0] * inv, v[1] * inv), pack_bf16x2(v[2] * inv, v[3] * inv));
    }
  }
}

template <int HD, int DPT>
__global__ __launch_bounds__(HD / DPT * kCombineQv) void attn_combine_kernel(AttnArgs a,
                                                                              const AttnGroup* __restrict__ groups) {
  constexpr int TQ = HD / DPT;  // threads per query vector
  const AttnGroup gr = groups[blockIdx.x];
  const int gkv = blockIdx.y;
  const int m = blockIdx.z * kCombineQv + static_cast<int>(threadIdx.x) / TQ;
  const int G = a.Hq / a.Hkv;
  if (m >= gr.nrows * G) return;
  const int d0 = DPT * (threadIdx.x % TQ);  // dims d0 .. d0 + DPT - 1
  const int n = gr.nparts;
  const size_t base = static_cast<size_t>(gr.part0 * a.Hkv + gkv) * 64 + m;
  const size_t stride = static_cast<size_t>(a.Hkv) * 64;
  const float2* ml = reinterpret_cast<const float2*>(a.part_ml);
  float num[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) num[i] = 0.f;
  float den = 0.f;
  auto acc = [&](float w, const CombVec<DPT>& o, float l) {
#pragma unroll
    for (int i = 0; i < DPT; ++i) num[i] += w * o.v[i];
    den += w * l;
  };
  if (n <= kCombineOnePass) {
    float2 mlc[kCombineOnePass];
    CombVec<DPT> oc[kCombineOnePass];
#pragma unroll
    for (int j = 0; j < kCombineOnePass; ++j)
      if (j < n) {
        const size_t pm = base + j * stride;
        mlc[j] = ml[pm];
        oc[j].load(a.part_o + pm * HD + d0);
      }
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < kCombineOnePass; ++j)
      if (j < n) mx = fmaxf(mx, mlc[j].x);
    if (mx != -INFINITY) {
#pragma unroll
      for (int j = 0; j < kCombineOnePass; ++j)
        if (j < n) acc(mlc[j].x != -INFINITY ? exp2f(mlc[j].x - mx) : 0.f, oc[j], mlc[j].y);
    }
  } else {
    constexpr int B = 8;
    float mx = -INFINITY;
    for (int c0 = 0; c0 < n; c0 += B) {
      float mc[B];
#pragma unroll
      for (int j = 0; j < B; ++j) mc[j] = ml[base + min(c0 + j, n - 1) * stride].x;
#pragma unroll
      for (int j = 0; j < B; ++j) mx = fmaxf(mx, mc[j]);
    }
    if (mx != -INFINITY) {
      for (int c0 = 0; c0 < n; c0 += B) {
        float2 mc[B];
        CombVec<DPT> oc[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
          const size_t pm = base + min(c0 + j, n - 1) * stride;
          mc[j] = ml[pm];
          oc[j].load(a.part_o + pm * HD + d0);
        }
#pragma unroll
        for (int j = 0; j < B; ++j)
          if (c0 + j < n) acc(mc[j].x != -INFINITY ? exp2f(mc[j].x - mx) : 0.f, oc[j], mc[j].y);
      }
    }
  }
  const size_t o = (static_cast<size_t>(gr.row0 + m / G) * a.Hq + gkv * G + m % G) * HD + d0;
  const bool ok = den > 0.f;
  bf16_t* out = static_cast<bf16_t*>(a.out) + o;
  if constexpr (DPT == 4) {
    *reinterpret_cast<uint2*>(out) = make_uint2(pack_bf16x2(ok ? num[0] / den : 0.f, ok ? num[1] / den : 0.f),
                                                pack_bf16x2(ok ? num[2] / den : 0.f, ok ? num[3] / den : 0.f));
  } else {
    out[0] = f32_to_bf16(ok ? num[0] / den : 0.f);
  }
}

// fp32: one wave per (row, head); each lane runs an online softmax over keys
// lane, lane + 64, ...; lanes are merged through LDS.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a, const int32_t* __restrict__ row_seq,
                                                      const int32_t* __restrict__ row_pos) {
  const int r = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int G = a.Hq / a.Hkv, gkv = h / G;
  // causal by position, or the row's tree keys: 0..base and base + 1 + j for
  // the bits j of its mask
  const bool tree = a.tree_base != nullptr;
  const int base = tree ? a.tree_base[r] : row_pos[r];
  const uint32_t tm = tree ? a.tree_mask[r] : 0u;
  const int tlim = base + 1 + (tm ? 32 - __clz(static_cast<int>(tm)) : 0);
  const int32_t* pt = a.page_table + static_cast<size_t>(row_seq[r]) * a.max_pages;
  const float* kp = static_cast<const float*>(a.kpool);
  const float* vp = static_cast<const float*>(a.vpool);
  __shared__ float qs[HD];
  __shared__ float red[kWave][HD + 1];
  __shared__ float ms[kWave], ls[kWave];
  const float* qv = static_cast<const float*>(a.q) + (static_cast<size_t>(r) * a.Hq + h) * HD;
  for (int d = lane; d < HD; d += kWave) qs[d] = qv[d];
  __syncthreads();
  const float scale = 1.f / sqrtf(static_cast<float>(HD));
  float m = -INFINITY, l = 0.f, acc[HD];
#pragma unroll
  for (int d = 0; d < HD; ++d) acc[d] = 0.f;
  for (int t = lane; t < tlim; t += kWave) {
    if (t > base && !((tm >> (t - base - 1)) & 1u)) continue;
    const size_t pb = static_cast<size_t>(pt[t >> 4] * a.Hkv + gkv);
    const float* kr = kp + (pb * 16 + (t & 15)) * HD;
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < HD; ++d) s = fmaf(qs[d], kr[d], s);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float al = (m == -INFINITY) ? 0.f : expf(m - mn);
    const float p = expf(s - mn);
    l = l * al + p;
    const float* vr = vp + pb * HD * 16 + (t & 15);
#pragma unroll
    for (int d = 0; d < HD; ++d) acc[d] = acc[d] * al + p * vr[d * 16];
    m = mn;
  }
  ms[lane] = m;
  __syncthreads();
  float mx = -INFINITY;
  for (int i = 0; i < kWave; ++i) mx = fmaxf(mx, ms[i]);
  const float w = (m == -INFINITY) ? 0.f : expf(m - mx);
  ls[lane] = l * w;
#pragma unroll
  for (int d = 0; d < HD; ++d) red[lane][d] = acc[d] * w;
  __syncthreads();
  float den = 0.f;
  for (int i = 0; i < kWave; ++i) den += ls[i];
  float* o = static_cast<float*>(a.out) + (static_cast<size_t>(r) * a.Hq + h) * HD;
  for (int d = lane; d < HD; d += kWave) {
    float num = 0.f;
    for (int i = 0; i < kWave; ++i) num += red[i][d];
    o[d] = num / den;
  }
}

template <int HD, int NT>
void launch_item_kernel(const AttnArgs& a, const AttnItem* items, dim3 grid, int w, hipStream_t st) {
  if (a.tree_base) {
    if (w >= 4) launch_kernel(attn_tree_bf16_kernel<HD, NT, 4>, grid, dim3(4 * kWave), 0, st, a, items);
    else if (w == 2) launch_kernel(attn_tree_bf16_kernel<HD, NT, 2>, grid, dim3(2 * kWave), 0, st, a, items);
    else launch_kernel(attn_tree_bf16_kernel<HD, NT, 1>, grid, dim3(kWave), 0, st, a, items);
    return;
  }
  if (w >= 4) launch_kernel(attn_bf16_kernel<HD, NT, 4>, grid, dim3(4 * kWave), 0, st, a, items);
  else if (w == 2) launch_kernel(attn_bf16_kernel<HD, NT, 2>, grid, dim3(2 * kWave), 0, st, a, items);
  else launch_kernel(attn_bf16_kernel<HD, NT, 1>, grid, dim3(kWave), 0, st, a, items);
}

template <int HD>
hipError_t launch_bf16_hd(const AttnArgs& a, const AttnItem* items, int n_items,
                          const AttnGroup* groups, int n_groups, int nt, int w, hipStream_t st) {
  dim3 grid(n_items, a.Hkv);
  if (n_items > 0) {
    if (nt <= 1) launch_item_kernel<HD, 1>(a, items, grid, w, st);
    else if (nt == 2) launch_item_kernel<HD, 2>(a, items, grid, w, st);
    else launch_item_kernel<HD, 4>(a, items, grid, std::min(w, 2), st);
  }
  if (n_groups > 0) {
    constexpr int DPT = HD == 128 ? 4 : 1;
    attn_combine_kernel<HD, DPT><<<dim3(n_groups, a.Hkv, 16 * nt / kCombineQv), HD / DPT * kCombineQv, 0, st>>>(
        a, groups);
  }
  return hipGetLastError();
}

}  // namespace

const char* attn_kernel_name(int hd, int nt, int w, bool tree) {
  if (tree) {
    static char tnames[2][3][3][48];
    static bool init = false;
    if (!init) {
      for (int h = 0; h < 2; ++h)
        for (int i = 0; i < 3; ++i)
          for (int j = 0; j < 3; ++j)
            snprintf(tnames[h][i][j], sizeof(tnames[h][i][j]), "attn_tree_bf16_kernel<%d, %d, %d>", h ? 128 : 64,
                     1 << i, i == 2 ? std::min(2, 1 << j) : 1 << j);
      init = true;
    }
    return tnames[hd == 128 ? 1 : 0][nt <= 1 ? 0 : (nt == 2 ? 1 : 2)][w <= 1 ? 0 : (w == 2 ? 1 : 2)];
  }
  // [hd 64 / 128][nt 1 / 2 / 4][w 1 / 2 / 4]
  static const char* names[2][3][3] = {
      {{"attn_bf16_kernel<64, 1, 1>", "attn_bf16_kernel<64, 1, 2>", "attn_bf16_kernel<64, 1, 4>"},
       {"attn_bf16_kernel<64, 2, 1>", "attn_bf16_kernel<64, 2, 2>", "attn_bf16_kernel<64, 2, 4>"},
       {"attn_bf16_kernel<64, 4, 1>", "attn_bf16_kernel<64, 4, 2>", "attn_bf16_kernel<64, 4, 2>"}},
      {{"attn_bf16_kernel<128, 1, 1>", "attn_bf16_kernel<128, 1, 2>", "attn_bf16_kernel<128, 1, 4>"},
       {"attn_bf16_kernel<128, 2, 1>", "attn_bf16_kernel<128, 2, 2>", "attn_bf16_kernel<128, 2, 4>"},
       {"attn_bf16_kernel<128, 4, 1>", "attn_bf16_kernel<128, 4, 2>", "attn_bf16_kernel<128, 4, 2>"}}};
  const int i = nt <= 1 ? 0 : (nt == 2 ? 1 : 2);
  const int j = w <= 1 ? 0 : (w == 2 ? 1 : 2);
  return names[hd == 128 ? 1 : 0][i][j];
}

hipError_t launch_attention_bf16(const AttnArgs& a, const AttnItem* d_items, int n_items,
                                 const AttnGroup* d_groups, int n_groups, int nt, int w, hipStream_t st) {
  if (nt > 4 || w > 4) return hipErrorInvalidValue;
  if (a.hd == 128) return launch_bf16_hd<128>(a, d_items, n_items, d_groups, n_groups, nt, w, st);
  if (a.hd == 64) return launch_bf16_hd<64>(a, d_items, n_items, d_groups, n_groups, nt, w, st);
  return hipErrorInvalidValue;
}

hipError_t launch_attention_prefill_bf16(const AttnArgs& a, const AttnItem* d_items, int n_items, hipStream_t st) {
  if (n_items <= 0) return hipSuccess;
  if (256 % (a.Hq / a.Hkv)) return hipErrorInvalidValue;
  dim3 grid(n_items * a.Hkv);
  if (a.hd == 128) launch_kernel(attn_prefill_bf16_kernel<128>, grid, dim3(512), 0, st, a, d_items);
  else if (a.hd == 64) launch_kernel(attn_prefill_bf16_kernel<64>, grid, dim3(512), 0, st, a, d_items);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

const char* attn_prefill_kernel_name(int hd) {
  return hd == 128 ? "attn_prefill_bf16_kernel<128>" : "attn_prefill_bf16_kernel<64>";
}

hipError_t launch_attention_f32(const AttnArgs& a, int R, const int32_t* d_row_seq,
                                const int32_t* d_row_pos, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  dim3 grid(R, a.Hq);
  if (a.hd == 64) attn_f32_kernel<64><<<grid, 64, 0, st>>>(a, d_row_seq, d_row_pos);
  else if (a.hd == 128) attn_f32_kernel<128><<<grid, 64, 0, st>>>(a, d_row_seq, d_row_pos);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace spec
