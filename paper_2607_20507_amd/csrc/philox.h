// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11, Section 3): ten rounds of
// two 32x32->64 multiplies with round keys bumped by the Weyl constants.
// Keying of the verify step's random streams: key = seed (lo, hi); counter =
// (block, position, seq_id lo32, seq_id bits 32..55 << 8 | purpose).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

struct PhiloxKey {
  uint32_t k0, k1;
};

__host__ __device__ __forceinline__ PhiloxKey philox_key(uint64_t seed) {
  return PhiloxKey{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)};
}

// The 32 x 32 -> 64 products are written as 64-bit multiplies so that each
// is one v_mad_u64_u32 (both halves at once): measured 712 against 547 G
// blocks/s for the __umulhi / low-product form, bit-identical results.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, PhiloxKey key) {
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = static_cast<uint64_t>(c.x) * 0xD2511F53u;
    const uint64_t p1 = static_cast<uint64_t>(c.z) * 0xCD9E8D57u;
    c = make_uint4(static_cast<uint32_t>(p1 >> 32) ^ c.y ^ k0, static_cast<uint32_t>(p1),
                   static_cast<uint32_t>(p0 >> 32) ^ c.w ^ k1, static_cast<uint32_t>(p0));
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Counter words 1..3 of stream (seq_id, pos, purpose).
struct StreamId {
  uint32_t pos, seq_lo, tag;
};

__host__ __device__ __forceinline__ StreamId stream_id(uint64_t seq_id, int32_t pos, int32_t purpose) {
  return StreamId{static_cast<uint32_t>(pos), static_cast<uint32_t>(seq_id),
                  (static_cast<uint32_t>((seq_id >> 32) & 0xFFFFFFu) << 8) |
                      (static_cast<uint32_t>(purpose) & 0xFFu)};
}

__device__ __forceinline__ uint4 philox_block(PhiloxKey key, StreamId s, uint32_t block) {
  return philox4x32_10(make_uint4(block, s.pos, s.seq_lo, s.tag), key);
}

// ((x >> 9) + 0.5) * 2^-23: exact in fp32, strictly inside (0, 1).
__device__ __forceinline__ float u01(uint32_t x) {
  return (static_cast<float>(x >> 9) + 0.5f) * 1.1920928955078125e-07f;
}

// -log2(u) of word x, an Exp(1) variate scaled by 1/ln 2.  v_log_f32 is
// log2 to about 1 ulp relative over (0, 1), including next to 1 (checked
// against float64 over all 2^23 values of u: 1.2e-7 relative).
__device__ __forceinline__ float exp2_variate(uint32_t x) { return -__builtin_amdgcn_logf(u01(x)); }

// Gumbel-max scores: argmax_i (log w_i + G_i) with G_i = -log(-log u_i).
// With E2_i = -log2 u_i, G_i = -log(E2_i) - log(ln 2): the constant does not
// move the argmax, so a score of z_i / T - ln 2 * log2(E2_i) ranks tokens as
// z_i / T + G_i does.  For weights known only up to a common factor (the
// residual max(0, p - q)) the equivalent exponential race w_i / E2_i needs no
// logarithm of w.
__device__ __forceinline__ float gumbel_shift(uint32_t x) {
  return -0.69314718055994531f * __builtin_amdgcn_logf(exp2_variate(x));
}

}  // namespace spec
