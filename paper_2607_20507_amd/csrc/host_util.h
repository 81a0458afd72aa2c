// Host-side helpers: pinned metadata staging, packed metadata blocks and the
// attention work planner.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "attention.h"
#include "common.h"

namespace spec {

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Optional timing of one kernel's launches: the launcher asks whether the
// kernel (by its profiler name) is wanted and brackets each launch.
struct KernelTimer {
  virtual ~KernelTimer() {}
  virtual bool wants(const char* kernel) const = 0;
  virtual void begin(hipStream_t st) = 0;
  virtual void end(hipStream_t st, double bytes, double flops) = 0;
};

// Events around the launches of one kernel; elapsed times are collected at
// the next synchronisation point.
class EventTimer : public KernelTimer {
 public:
  std::string name;
  double ms = 0, bytes = 0, flops = 0;
  int64_t launches = 0;

  ~EventTimer() override {
    flush();
    for (hipEvent_t e : free_) (void)hipEventDestroy(e);
  }
  bool wants(const char* k) const override { return !name.empty() && name == k; }
  // begin arms a kernel-level event pair for the next launch_kernel (the
  // timed kernel's own start and end) and also records an event on the
  // stream; end uses the kernel-level pair if a launch consumed it, else
  // the stream events around the launch call.
  void begin(hipStream_t st) override {
    cur_ = take();
    if (cur_) (void)hipEventRecord(cur_, st);
    ka_ = take();
    kb_ = take();
    if (ka_ && kb_) launch_events() = LaunchEvents{ka_, kb_};
  }
  void end(hipStream_t st, double b, double f) override {
    LaunchEvents& le = launch_events();
    const bool kernel_level = ka_ && kb_ && le.start == nullptr;
    le = LaunchEvents{};
    if (kernel_level) {
      recs_.push_back(Rec{ka_, kb_, b, f});
      if (cur_) free_.push_back(cur_);
    } else {
      if (ka_) free_.push_back(ka_);
      if (kb_) free_.push_back(kb_);
      hipEvent_t e = take();
      if (cur_ && e) {
        (void)hipEventRecord(e, st);
        recs_.push_back(Rec{cur_, e, b, f});
      }
    }
    cur_ = ka_ = kb_ = nullptr;
  }
  void flush() {
    for (auto& r : recs_) {
      float t = 0.f;
      if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&t, r.a, r.b) == hipSuccess) {
        ms += t;
        bytes += r.bytes;
        flops += r.flops;
        ++launches;
      }
      free_.push_back(r.a);
      free_.push_back(r.b);
    }
    recs_.clear();
  }
  void reset(const char* k) {
    flush();
    name = k ? k : "";
    ms = bytes = flops = 0;
    launches = 0;
  }

 private:
  struct Rec {
    hipEvent_t a, b;
    double bytes, flops;
  };
  hipEvent_t take() {
    if (!free_.empty()) {
      hipEvent_t e = free_.back();
      free_.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    return hipEventCreate(&e) == hipSuccess ? e : nullptr;
  }
  std::vector<hipEvent_t> free_;
  std::vector<Rec> recs_;
  hipEvent_t cur_ = nullptr, ka_ = nullptr, kb_ = nullptr;
};

// Timer of the context-free entry points (spec_timing_enable with no context).
EventTimer& global_timer();

// Message that spec_last_error(NULL) returns (the calling thread's last
// context-free failure).
void set_global_error(const char* msg);

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
  size_t size() const { return buf_.size(); }
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
// Workgroups an attention launch aims for (measured on the 8B/1B-shaped
// verify and draft steps and the 64-sequence serving batch).
constexpr int kAttnTargetWgs = 512;

struct AttnSegment {
  int32_t seq, row0, nrows, pos0;
};

struct AttnPlan {
  bool prefill = false;  // items for attn_prefill_bf16_kernel (nt, w, groups unused)
  int nt = 1;
  int w = 1;  // waves per workgroup
  std::vector<AttnItem> items;
  std::vector<AttnGroup> groups;
  int n_parts = 0;
};

// Tile rows into query tiles of (16 nt / G) rows and split key ranges so that
// the launch has about `target_wgs` workgroups; at most `max_parts` partials.
// Runs of at least kPrefillMinRows rows in every segment (prefill chunks) with
// 256 % G == 0 and at most kPrefillMaxKeys keys take the prefill form instead: blocks of 256 / G rows against
// all their keys, heaviest first (allow_prefill = false keeps the tiled form).
constexpr int kPrefillMinRows = 64;
constexpr int kPrefillMaxKeys = 16384;  // the prefill kernel stages at most 1024 page ids
AttnPlan plan_attention(const std::vector<AttnSegment>& segs, int G, int Hkv, int max_parts,
                        int target_wgs = kAttnTargetWgs, bool allow_prefill = true);

}  // namespace spec
