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

__device__ __forceinline__ uint4 philox4x32_10(uint4 c, PhiloxKey key) {
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint32_t lo0 = 0xD2511F53u * c.x;
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x);
    const uint32_t lo1 = 0xCD9E8D57u * c.z;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
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

// Gumbel(0,1) from a uniform: -log(-log u).
__device__ __forceinline__ float gumbel_of(uint32_t x) {
  return -logf(-logf(u01(x)));
}

}  // namespace spec
