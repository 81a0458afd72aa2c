// Host-side helpers: pinned metadata staging, packed metadata blocks and the
// attention work planner.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "attention.h"

namespace spec {

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// A packed block of host arrays, each 256-byte aligned, uploaded in one copy.
class MetaBlock {
 public:
  template <typename T>
  size_t add(const T* p, size_t n) {
    const size_t off = align_up(buf_.size());
    buf_.resize(off + n * sizeof(T));
    if (n) std::memcpy(buf_.data() + off, p, n * sizeof(T));
    return off;
  }
  template <typename T>
  size_t add(const std::vector<T>& v) { return add(v.data(), v.size()); }
  size_t size() const { return align_up(buf_.size()); }
  const char* data() const { return buf_.data(); }
  void clear() { buf_.clear(); }

 private:
  std::vector<char> buf_;
};

// Ring of pinned host buffers.  A slot is reused only after the copy that last
// read it has completed (event), so callers can run ahead of the GPU.
class Stager {
 public:
  static constexpr int kSlots = 4;
  ~Stager() { release(); }
  void release() {
    for (auto& s : slots_) {
      if (s.host) (void)hipHostFree(s.host);
      if (s.ev) (void)hipEventDestroy(s.ev);
      s = Slot{};
    }
  }
  // Copy `n` bytes of `src` to device `dst` on stream `st` through a pinned slot.
  hipError_t upload(void* dst, const void* src, size_t n, hipStream_t st, int* slot_used = nullptr) {
    if (n == 0) return hipSuccess;
    Slot& s = slots_[next_];
    if (slot_used) *slot_used = next_;
    next_ = (next_ + 1) % kSlots;
    hipError_t e;
    if (s.ev && s.pending) {
      if ((e = hipEventSynchronize(s.ev)) != hipSuccess) return e;
      s.pending = false;
    }
    if (s.cap < n) {
      if (s.host) (void)hipHostFree(s.host);
      s.host = nullptr;
      s.cap = 0;
      if ((e = hipHostMalloc(&s.host, n, hipHostMallocDefault)) != hipSuccess) return e;
      s.cap = n;
    }
    if (!s.ev && (e = hipEventCreateWithFlags(&s.ev, hipEventDisableTiming)) != hipSuccess) return e;
    std::memcpy(s.host, src, n);
    if ((e = hipMemcpyAsync(dst, s.host, n, hipMemcpyHostToDevice, st)) != hipSuccess) return e;
    if ((e = hipEventRecord(s.ev, st)) != hipSuccess) return e;
    s.pending = true;
    return hipSuccess;
  }

 private:
  struct Slot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
  };
  Slot slots_[kSlots];
  int next_ = 0;
};

// Attention work for rows of one sequence: rows [row0, row0 + nrows) at
// positions pos0.., page table row `seq` of the launch's compact table.
struct AttnSegment {
  int32_t seq, row0, nrows, pos0;
};

struct AttnPlan {
  int nt = 1;
  std::vector<AttnItem> items;
  std::vector<AttnGroup> groups;
  int n_parts = 0;
};

// Tile rows into query tiles of (16 nt / G) rows and split key ranges so that
// the launch has about `target_waves` waves; at most `max_parts` partials.
AttnPlan plan_attention(const std::vector<AttnSegment>& segs, int G, int Hkv, int max_parts,
                        int target_waves = 2048);

}  // namespace spec
