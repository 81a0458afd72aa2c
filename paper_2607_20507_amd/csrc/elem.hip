// Row-wise decoder kernels: embedding gather, RMSNorm (Llama definition,
// x / sqrt(mean(x^2) + eps) * w), rotate-half RoPE fused with the paged KV
// append, and in-place clearing of rolled-back KV slots.

#include <algorithm>
#include <cmath>

#include "common.h"
#include "elem.h"
#include "kv_layout.h"

namespace spec {
namespace {

// Index of (token k of the page, dim d) in a (page, kv head) block: the bf16
// cache uses the operand order of the attention kernel (kv_layout.h), the
// fp32 cache K [16][hd] and V^T [hd][16].
template <typename T>
__device__ __forceinline__ int k_index(int k, int d, int hd) {
  return sizeof(T) == 2 ? kv_k_off(k, d) : k * hd + d;
}
template <typename T>
__device__ __forceinline__ int v_index(int k, int d) {
  return sizeof(T) == 2 ? kv_v_off(k, d) : d * 16 + k;
}

template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(int d, const int32_t* __restrict__ tok_src,
                                                    const int32_t* __restrict__ tok_pool,
                                                    const T* __restrict__ E, float* __restrict__ h,
                                                    int32_t* __restrict__ row_tok, T* __restrict__ hb,
                                                    const T* __restrict__ wn, float* __restrict__ ss) {
  const int r = blockIdx.x;
  const int s = tok_src[r];
  const int tok = s >= 0 ? s : tok_pool[-1 - s];
  if (threadIdx.x == 0) row_tok[r] = tok;
  const T* e = E + static_cast<size_t>(tok) * d;
  float* o = h + static_cast<size_t>(r) * d;
  // whole waves run every iteration: 8 consecutive lanes hold the 8
  // columns whose sum of squares is one entry of ss
  for (int i0 = 0; i0 < d; i0 += blockDim.x) {
    const int i = i0 + threadIdx.x;
    const float x = i < d ? Elem<T>::to_f32(e[i]) : 0.f;
    if (i < d) {
      o[i] = x;
      if (hb) hb[static_cast<size_t>(r) * d + i] = Elem<T>::from_f32(x * Elem<T>::to_f32(wn[i]));
    }
    if (ss) {
      float sq = x * x;
#pragma unroll
      for (int k = 1; k < 8; k <<= 1) sq += __shfl_xor(sq, k, kWave);
      if ((threadIdx.x & 7) == 0 && i < d) ss[static_cast<size_t>(r) * (d / 8) + i / 8] = sq;
    }
  }
}

// 8 consecutive elements widened to fp32 (16 bytes of bf16, 32 of fp32), and
// back in the element type.
__device__ __forceinline__ void load8(const bf16_t* p, float (&v)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __uint_as_float(w[k] << 16);
    v[2 * k + 1] = __uint_as_float(w[k] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void load8(const float* p, float (&v)[8]) {
  const float4 a = reinterpret_cast<const float4*>(p)[0], b = reinterpret_cast<const float4*>(p)[1];
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(bf16_t* p, const float (&v)[8]) {
  *reinterpret_cast<uint4*>(p) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                            pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
}
__device__ __forceinline__ void store8(float* p, const float (&v)[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(v[0], v[1], v[2], v[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(v[4], v[5], v[6], v[7]);
}

// The same gather for rows of 8-column chunks (d % 8 == 0, d <= 2048 * NCH):
// thread t holds chunks t, t + 256, ... so that every load of the row (and of
// the norm weight) is issued before the first store, one round trip instead
// of one per 256 columns.  ss adds the eight squares pairwise, in the order
// of the shuffle tree above, so both kernels give the same bits.
template <typename T, int NCH>
__global__ __launch_bounds__(256) void embed_vec_kernel(int d, const int32_t* __restrict__ tok_src,
                                                        const int32_t* __restrict__ tok_pool,
                                                        const T* __restrict__ E, float* __restrict__ h,
                                                        int32_t* __restrict__ row_tok, T* __restrict__ hb,
                                                        const T* __restrict__ wn, float* __restrict__ ss) {
  const int r = blockIdx.x;
  const int s = tok_src[r];
  const int tok = s >= 0 ? s : tok_pool[-1 - s];
  if (threadIdx.x == 0) row_tok[r] = tok;
  const T* e = E + static_cast<size_t>(tok) * d;
  const int nc = d / 8;
  float x[NCH][8], w[NCH][8];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int j = min(static_cast<int>(threadIdx.x) + 256 * c, nc - 1);  // clamped: loads unconditional
    load8(e + 8 * j, x[c]);
    if (hb) load8(wn + 8 * j, w[c]);
  }
  float* o = h + static_cast<size_t>(r) * d;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int j = static_cast<int>(threadIdx.x) + 256 * c;
    if (j >= nc) continue;
    store8(o + 8 * j, x[c]);
    if (hb) {
      float y[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) y[k] = x[c][k] * w[c][k];
      store8(hb + static_cast<size_t>(r) * d + 8 * j, y);
    }
    if (ss) {
      float q[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) q[k] = x[c][k] * x[c][k];
      ss[static_cast<size_t>(r) * nc + j] = ((q[0] + q[1]) + (q[2] + q[3])) + ((q[4] + q[5]) + (q[6] + q[7]));
    }
  }
}

// One workgroup per row.  Rows of up to 8192 columns (d % 4 == 0): thread t
// holds 4-column chunks t, t + 256, ... of the row in registers (one round of
// 16-byte loads, the norm weight's with them), so the row is read once and
// written with 8- / 16-byte stores; wider rows take a strided two-pass loop.
// The sum of squares is taken per thread in chunk order, then over the wave
// and the waves in a fixed order.
constexpr int kNormChunks = 8;  // 4-column chunks per thread held in registers

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(int d, const float* __restrict__ h,
                                                      const int32_t* __restrict__ row_idx,
                                                      const T* __restrict__ w, float eps,
                                                      T* __restrict__ y) {
  const int r = blockIdx.x;
  const int src = row_idx ? row_idx[r] : r;
  const float* x = h + static_cast<size_t>(src) * d;
  T* o = y + static_cast<size_t>(r) * d;
  __shared__ float part[256 / kWave];
  auto total = [&](float ss) {
    ss = wave_sum(ss);
    if ((threadIdx.x & (kWave - 1)) == 0) part[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = 0.f;
    for (int k = 0; k < static_cast<int>(blockDim.x) / kWave; ++k) tot += part[k];
    return 1.f / sqrtf(tot / static_cast<float>(d) + eps);
  };
  const int nch = d / 4;
  if (d % 4 == 0 && nch <= kNormChunks * static_cast<int>(blockDim.x)) {
    float4 xv[kNormChunks];
    float wv[kNormChunks][4];
#pragma unroll
    for (int c = 0; c < kNormChunks; ++c) {
      const int ch = threadIdx.x + c * blockDim.x;
      if (ch < nch) {
        xv[c] = reinterpret_cast<const float4*>(x)[ch];
#pragma unroll
        for (int e = 0; e < 4; ++e) wv[c][e] = Elem<T>::to_f32(w[4 * ch + e]);
      }
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < kNormChunks; ++c)
      if (threadIdx.x + c * blockDim.x < nch) {
        ss = fmaf(xv[c].x, xv[c].x, ss);
        ss = fmaf(xv[c].y, xv[c].y, ss);
        ss = fmaf(xv[c].z, xv[c].z, ss);
        ss = fmaf(xv[c].w, xv[c].w, ss);
      }
    const float inv = total(ss);
#pragma unroll
    for (int c = 0; c < kNormChunks; ++c) {
      const int ch = threadIdx.x + c * blockDim.x;
      if (ch < nch) {
        const float v0 = xv[c].x * inv * wv[c][0], v1 = xv[c].y * inv * wv[c][1];
        const float v2 = xv[c].z * inv * wv[c][2], v3 = xv[c].w * inv * wv[c][3];
        if constexpr (sizeof(T) == 2)
          reinterpret_cast<uint2*>(o)[ch] = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
        else
          reinterpret_cast<float4*>(o)[ch] = make_float4(v0, v1, v2, v3);
      }
    }
    return;
  }
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) ss = fmaf(x[i], x[i], ss);
  const float inv = total(ss);
  for (int i = threadIdx.x; i < d; i += blockDim.x) o[i] = Elem<T>::from_f32(x[i] * inv * Elem<T>::to_f32(w[i]));
}

// One workgroup per (row, KV head group): workgroup (r, g) of a grid (R, ng)
// handles the KV heads [g Hkv / ng, (g + 1) Hkv / ng) and the query heads
// that share them; thread (head, i) rotates the pair (i, i + hd/2).
constexpr int kRopeMaxHalf = 128;  // head_dim <= 256

// SPLIT: qkv holds S split-K partials [S][R][width] (split stride sstride
// floats) of the QKV GEMM instead of its output; the workgroup's columns,
// summed over the splits in split order as splitk_reduce4 takes them, go to
// LDS first (all of a thread's loads of 8 splits in flight together), which
// saves the reduction's launch and its round trip through memory.
template <typename T, bool SPLIT>
__global__ __launch_bounds__(256) void rope_kv_kernel(int Hq, int Hkv, int hd, float theta,
                                                      const float* __restrict__ qkv,
                                                      const int32_t* __restrict__ pos,
                                                      const int32_t* __restrict__ slot,
                                                      T* __restrict__ q, T* __restrict__ kpool,
                                                      T* __restrict__ vpool, bool rot_tiled, int S,
                                                      size_t sstride) {
  const int r = blockIdx.x;
  const int half = hd / 2;
  const int width = (Hq + 2 * Hkv) * hd;
  const int kh0 = blockIdx.y * Hkv / gridDim.y, kh1 = (blockIdx.y + 1) * Hkv / gridDim.y;
  const int qh0 = kh0 * (Hq / Hkv), qh1 = kh1 * (Hq / Hkv);
  const int nq = qh1 - qh0, nk = kh1 - kh0;
  const float* x = qkv + static_cast<size_t>(r) * width;
  // xq / xk / xv: the first column of query head qh0, key head kh0, value head kh0
  const float* xq = x + qh0 * hd;
  const float* xk = x + (Hq + kh0) * hd;
  const float* xv = x + (Hq + Hkv + kh0) * hd;
  if constexpr (SPLIT) {
    extern __shared__ float4 s_cols[];  // (nq + 2 nk) hd floats, sized by the launch
    // local column lc of [q heads | k heads | v heads] comes from row column gc
    const int nqc = nq * hd, nkc = nk * hd;
    const size_t st4 = sstride / 4;
    constexpr int B = 8;
    for (int c = threadIdx.x; c < (nqc + 2 * nkc) / 4; c += blockDim.x) {
      const int lc = 4 * c;
      const int gc = lc < nqc ? qh0 * hd + lc
                              : (lc < nqc + nkc ? (Hq + kh0) * hd + lc - nqc : (Hq + Hkv + kh0) * hd + lc - nqc - nkc);
      const float4* src = reinterpret_cast<const float4*>(x + gc);
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s0 = 0; s0 < S; s0 += B) {
        float4 p[B];
#pragma unroll
        for (int b = 0; b < B; ++b) p[b] = src[static_cast<size_t>(min(s0 + b, S - 1)) * st4];
#pragma unroll
        for (int b = 0; b < B; ++b) {
          if (s0 + b >= S) break;
          v.x += p[b].x;
          v.y += p[b].y;
          v.z += p[b].z;
          v.w += p[b].w;
        }
      }
      s_cols[c] = v;
    }
    xq = reinterpret_cast<const float*>(s_cols);
    xk = xq + nqc;
    xv = xk + nkc;
  }
  const double p = static_cast<double>(pos[r]);
  const int sl = slot[r];
  const int page = sl >> 4, off = sl & 15;
  const double lt = log(static_cast<double>(theta));
  // the row's rotation angles (they depend on the pair index only, not on
  // the head), once per workgroup in fp64, by the last hd / 2 threads (with
  // the split, while the first ones wait for the partials)
  __shared__ float s_cos[kRopeMaxHalf], s_sin[kRopeMaxHalf];
  const int ai = static_cast<int>(threadIdx.x) - (static_cast<int>(blockDim.x) - half);
  if (ai >= 0) {
    double sn, cs;
    sincos(p * exp(-(2.0 * ai / hd) * lt), &sn, &cs);
    s_cos[ai] = static_cast<float>(cs);
    s_sin[ai] = static_cast<float>(sn);
  }
  __syncthreads();
  // Groups of 8 consecutive pairs (half % 8 == 0): in both column orders
  // their a and b values are 8 consecutive floats, and their outputs 8
  // consecutive elements of q and of the K page (one 16-byte unit of the
  // bf16 page layout), so one thread moves them with vector loads / stores.
  auto put8 = [](T* dst, const float (&v)[8]) {
    if constexpr (sizeof(T) == 2) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                  pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
    } else {
      reinterpret_cast<float4*>(dst)[0] = make_float4(v[0], v[1], v[2], v[3]);
      reinterpret_cast<float4*>(dst)[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
  };
  // local head h < nq: query head qh0 + h; else key head kh0 + h - nq
  if (half % 8 == 0) {
    const int groups = half / 8;
    for (int e = threadIdx.x; e < (nq + nk) * groups; e += blockDim.x) {
      const int h = e / groups, t = e % groups, i0 = 8 * t;
      // rot_tiled: the q and k columns of each head are in the rotary tile
      // order of the tiled QKV weight (rows 8t..8t+7, then hd/2+8t.. of tile t)
      const float* src = h < nq ? xq + h * hd : xk + (h - nq) * hd;
      const int ia = rot_tiled ? 16 * t : i0;
      const int ib = rot_tiled ? ia + 8 : i0 + half;
      const float4 a0 = reinterpret_cast<const float4*>(src + ia)[0], a1 = reinterpret_cast<const float4*>(src + ia)[1];
      const float4 b0 = reinterpret_cast<const float4*>(src + ib)[0], b1 = reinterpret_cast<const float4*>(src + ib)[1];
      const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
      float ra[8], rb[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float c = s_cos[i0 + j], sn = s_sin[i0 + j];
        ra[j] = av[j] * c - bv[j] * sn;
        rb[j] = bv[j] * c + av[j] * sn;
      }
      if (h < nq) {
        T* o = q + (static_cast<size_t>(r) * Hq + qh0 + h) * hd;
        put8(o + i0, ra);
        put8(o + i0 + half, rb);
      } else {
        T* o = kpool + (static_cast<size_t>(page) * Hkv + kh0 + h - nq) * 16 * hd;
        put8(o + k_index<T>(off, i0, hd), ra);
        put8(o + k_index<T>(off, i0 + half, hd), rb);
      }
    }
  } else {
    for (int e = threadIdx.x; e < (nq + nk) * half; e += blockDim.x) {
      const int h = e / half, i = e % half;
      const float c = s_cos[i], s = s_sin[i];
      const float* src = h < nq ? xq + h * hd : xk + (h - nq) * hd;
      const int ia = rot_tiled ? 16 * (i / 8) + (i % 8) : i;
      const int ib = rot_tiled ? ia + 8 : i + half;
      const float a = src[ia], b = src[ib];
      const float ra = a * c - b * s, rb = b * c + a * s;
      if (h < nq) {
        T* o = q + (static_cast<size_t>(r) * Hq + qh0 + h) * hd;
        o[i] = Elem<T>::from_f32(ra);
        o[i + half] = Elem<T>::from_f32(rb);
      } else {
        T* o = kpool + (static_cast<size_t>(page) * Hkv + kh0 + h - nq) * 16 * hd;
        o[k_index<T>(off, i, hd)] = Elem<T>::from_f32(ra);
        o[k_index<T>(off, i + half, hd)] = Elem<T>::from_f32(rb);
      }
    }
  }
  for (int e = threadIdx.x; e < nk * hd; e += blockDim.x) {
    const int kh = kh0 + e / hd, dd = e % hd;
    vpool[(static_cast<size_t>(page) * Hkv + kh) * hd * 16 + v_index<T>(off, dd)] = Elem<T>::from_f32(xv[e]);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void kv_clear_kernel(KvClearJob j0, KvClearJob j1) {
  const KvClearJob& j = blockIdx.z ? j1 : j0;
  const int i = blockIdx.x, l = blockIdx.y;
  if (i >= j.n || l >= j.n_layers) return;
  const int sl = j.slots ? j.slots[i] : j.inl[i];
  const int page = sl >> 4, off = sl & 15;
  T* K = static_cast<T*>(j.kv) + l * j.layer_stride;
  T* V = K + j.v_off;
  for (int e = threadIdx.x; e < j.Hkv * j.hd; e += blockDim.x) {
    const int h = e / j.hd, dd = e % j.hd;
    const size_t blk = (static_cast<size_t>(page) * j.Hkv + h) * 16 * j.hd;
    K[blk + k_index<T>(off, dd, j.hd)] = T(0);
    V[blk + v_index<T>(off, dd)] = T(0);
  }
}

// One workgroup per (group, layer); thread e owns element e of every token,
// so the group's moves, applied in order by each thread, see each other's
// writes without barriers.
template <typename T>
__global__ __launch_bounds__(256) void kv_move_kernel(KvMoveJob j) {
  const int g = blockIdx.x, l = blockIdx.y;
  if (g >= j.n_groups || l >= j.n_layers) return;
  T* K = static_cast<T*>(j.kv) + l * j.layer_stride;
  T* V = K + j.v_off;
  const int i0 = j.off[g], i1 = j.off[g + 1];
  for (int e = threadIdx.x; e < j.Hkv * j.hd; e += blockDim.x) {
    const int h = e / j.hd, dd = e % j.hd;
    for (int i = i0; i < i1; ++i) {
      const int src = j.pairs[2 * i], dst = j.pairs[2 * i + 1];
      const size_t bs = (static_cast<size_t>(src >> 4) * j.Hkv + h) * 16 * j.hd;
      const size_t bd = (static_cast<size_t>(dst >> 4) * j.Hkv + h) * 16 * j.hd;
      K[bd + k_index<T>(dst & 15, dd, j.hd)] = K[bs + k_index<T>(src & 15, dd, j.hd)];
      V[bd + v_index<T>(dst & 15, dd)] = V[bs + v_index<T>(src & 15, dd)];
    }
  }
}

}  // namespace

hipError_t launch_kv_move(int dtype, const KvMoveJob& j, hipStream_t st) {
  if (j.n_groups <= 0 || j.n_layers <= 0) return hipSuccess;
  dim3 grid(j.n_groups, j.n_layers);
  if (dtype == 0)
    kv_move_kernel<float><<<grid, 256, 0, st>>>(j);
  else
    kv_move_kernel<bf16_t><<<grid, 256, 0, st>>>(j);
  return hipGetLastError();
}

hipError_t launch_embed(int dtype, int R, int d, const int32_t* tok_src, const int32_t* tok_pool,
                        const void* E, float* h, int32_t* row_tok, hipStream_t st, void* hb, const void* wn,
                        float* ss) {
  if (R <= 0) return hipSuccess;
  if (ss && d % 16 != 0) return hipErrorInvalidValue;
  const auto aligned = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  const int nch = (d / 8 + 255) / 256;
  if (d % 8 == 0 && nch <= 4 && aligned(E) && aligned(h) && aligned(hb) && aligned(wn)) {
    if (dtype == 0) {
      auto* k = nch == 1 ? embed_vec_kernel<float, 1> : nch == 2 ? embed_vec_kernel<float, 2>
              : nch == 3 ? embed_vec_kernel<float, 3> : embed_vec_kernel<float, 4>;
      k<<<R, 256, 0, st>>>(d, tok_src, tok_pool, static_cast<const float*>(E), h, row_tok,
                           static_cast<float*>(hb), static_cast<const float*>(wn), ss);
    } else {
      auto* k = nch == 1 ? embed_vec_kernel<bf16_t, 1> : nch == 2 ? embed_vec_kernel<bf16_t, 2>
              : nch == 3 ? embed_vec_kernel<bf16_t, 3> : embed_vec_kernel<bf16_t, 4>;
      k<<<R, 256, 0, st>>>(d, tok_src, tok_pool, static_cast<const bf16_t*>(E), h, row_tok,
                           static_cast<bf16_t*>(hb), static_cast<const bf16_t*>(wn), ss);
    }
    return hipGetLastError();
  }
  if (dtype == 0)
    embed_kernel<float><<<R, 256, 0, st>>>(d, tok_src, tok_pool, static_cast<const float*>(E), h, row_tok,
                                           static_cast<float*>(hb), static_cast<const float*>(wn), ss);
  else
    embed_kernel<bf16_t><<<R, 256, 0, st>>>(d, tok_src, tok_pool, static_cast<const bf16_t*>(E), h, row_tok,
                                            static_cast<bf16_t*>(hb), static_cast<const bf16_t*>(wn), ss);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, int R, int d, const float* h, const int32_t* row_idx,
                          const void* w, float eps, void* y, hipStream_t st) {
  if (R <= 0) return hipSuccess;
  if (dtype == 0)
    rmsnorm_kernel<float><<<R, 256, 0, st>>>(d, h, row_idx, static_cast<const float*>(w), eps,
                                             static_cast<float*>(y));
  else
    rmsnorm_kernel<bf16_t><<<R, 256, 0, st>>>(d, h, row_idx, static_cast<const bf16_t*>(w), eps,
                                              static_cast<bf16_t*>(y));
  return hipGetLastError();
}

hipError_t launch_rope_kv(int dtype, int R, int Hq, int Hkv, int hd, float theta, const float* qkv,
                          const int32_t* pos, const int32_t* slot, void* q, void* kpool,
                          void* vpool, hipStream_t st, bool rot_tiled, int splits) {
  if (R <= 0) return hipSuccess;
  if (hd % 2 != 0 || hd > 2 * kRopeMaxHalf || (rot_tiled && hd % 16 != 0)) return hipErrorInvalidValue;
  if (Hkv <= 0 || Hq % Hkv != 0) return hipErrorInvalidValue;
  const int width = (Hq + 2 * Hkv) * hd;
  // one workgroup per (row, KV head): its query heads, key head and value head
  const dim3 grid(R, Hkv);
  if (splits > 0 && (hd % 4 || (Hq / Hkv + 2) * hd > kRopeSplitMaxWidth)) return hipErrorInvalidValue;
  const size_t sstride = static_cast<size_t>(R) * width;
  const size_t lds = static_cast<size_t>(Hq / Hkv + 2) * hd * sizeof(float);  // split partial sums
  if (dtype == 0 && splits > 0)
    rope_kv_kernel<float, true><<<grid, 256, lds, st>>>(Hq, Hkv, hd, theta, qkv, pos, slot, static_cast<float*>(q),
                                                   static_cast<float*>(kpool), static_cast<float*>(vpool),
                                                   rot_tiled, splits, sstride);
  else if (dtype == 0)
    rope_kv_kernel<float, false><<<grid, 256, 0, st>>>(Hq, Hkv, hd, theta, qkv, pos, slot, static_cast<float*>(q),
                                                    static_cast<float*>(kpool), static_cast<float*>(vpool),
                                                    rot_tiled, 0, 0);
  else if (splits > 0)
    rope_kv_kernel<bf16_t, true><<<grid, 256, lds, st>>>(Hq, Hkv, hd, theta, qkv, pos, slot, static_cast<bf16_t*>(q),
                                                    static_cast<bf16_t*>(kpool), static_cast<bf16_t*>(vpool),
                                                    rot_tiled, splits, sstride);
  else
    rope_kv_kernel<bf16_t, false><<<grid, 256, 0, st>>>(Hq, Hkv, hd, theta, qkv, pos, slot, static_cast<bf16_t*>(q),
                                                     static_cast<bf16_t*>(kpool), static_cast<bf16_t*>(vpool),
                                                     rot_tiled, 0, 0);
  return hipGetLastError();
}

hipError_t launch_kv_clear(int dtype, const KvClearJob& a, const KvClearJob& b, hipStream_t st) {
  const int n = std::max(a.n, b.n);
  if (n <= 0) return hipSuccess;
  dim3 grid(n, std::max(a.n > 0 ? a.n_layers : 0, b.n > 0 ? b.n_layers : 0), 2);
  if (dtype == 0)
    kv_clear_kernel<float><<<grid, 256, 0, st>>>(a, b);
  else
    kv_clear_kernel<bf16_t><<<grid, 256, 0, st>>>(a, b);
  return hipGetLastError();
}

}  // namespace spec
