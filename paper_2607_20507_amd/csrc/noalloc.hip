// The decision pass for callers that cannot allocate (code under HIP graph
// capture, tight serving loops): spec_sample_verify_noalloc.  Its tables and
// partial results live in one file-scope device array per GPU, so a call
// allocates nothing and copies nothing from the host: the per-sequence inputs
// are device arrays and a setup kernel lays the tables out on the device.

#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/spec.h"
#include "host_util.h"
#include "vocab.h"

using namespace spec;

namespace {

// Bound of the tables and partial results of one call: at B = 256
// sequences of 15 drafts (7936 rows) over any vocabulary they need about
// 0.3 MiB (rows and sequence tables, chunk statistics, chunk winners).
constexpr size_t kScratchBytes = size_t(512) << 10;
static __device__ __align__(256) char scratch[kScratchBytes];

// The array's device address, per device, taken once with that device
// current (each GPU holds its own copy of the array).
constexpr int kMaxDevices = 64;
std::mutex g_mu;
char* g_scratch[kMaxDevices] = {};

spec_status scratch_of_current_device(char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_global_error("spec_sample_verify_noalloc: no current HIP device");
    return SPEC_E_HIP;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_global_error("spec_sample_verify_noalloc: hipGetSymbolAddress failed");
      return SPEC_E_HIP;
    }
    g_scratch[dev] = static_cast<char*>(p);
  }
  *out = g_scratch[dev];
  return SPEC_OK;
}

}  // namespace

extern "C" {

spec_status spec_sample_verify_noalloc(int32_t B, int32_t k_max, const int32_t* k, const float* temperature,
                                       const int64_t* seq_ids, const int32_t* base_pos, const float* p_logits,
                                       const float* q_logits, const int32_t* draft_tokens, int32_t V,
                                       uint64_t seed, int32_t* n_accepted, int32_t* out_tokens, void* stream) {
  if (B == 0) return SPEC_OK;
  if (B < 0 || B > kSetupMaxSeqs || k_max < 0 || k_max > 15 || V <= 0) {
    set_global_error("spec_sample_verify_noalloc: need 0 <= B <= 256, 0 <= k_max <= 15, V > 0");
    return SPEC_E_INVALID;
  }
  if (!k || !temperature || !seq_ids || !base_pos || !p_logits || !n_accepted || !out_tokens ||
      (k_max > 0 && (!q_logits || !draft_tokens))) {
    set_global_error("spec_sample_verify_noalloc: null pointer");
    return SPEC_E_INVALID;
  }
  const int rows_max = B * (2 * k_max + 1);
  const VocabPlan plan = vocab_plan(B, rows_max, V, rows_max);
  const size_t o_seqs = align_up(sizeof(VRow) * rows_max);
  const size_t o_nrows = o_seqs + align_up(sizeof(VSeq) * B);
  const size_t o_ws = o_nrows + 256;
  if (o_ws + vocab_ws_bytes(plan) > kScratchBytes) {
    set_global_error("spec_sample_verify_noalloc: the call needs more than the 512 KiB scratch");
    return SPEC_E_UNSUPPORTED;
  }
  char* sc = nullptr;
  const spec_status s = scratch_of_current_device(&sc);
  if (s != SPEC_OK) return s;
  VRow* rows = reinterpret_cast<VRow*>(sc);
  VSeq* seqs = reinterpret_cast<VSeq*>(sc + o_seqs);
  int32_t* n_rows = reinterpret_cast<int32_t*>(sc + o_nrows);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = launch_vocab_setup(B, k_max, k, temperature, seq_ids, base_pos, p_logits, q_logits, V, rows,
                                    seqs, n_rows, st);
  if (e != hipSuccess) return SPEC_E_HIP;
  // the vector path reads 16-byte units from each row
  const bool aligned = (reinterpret_cast<uintptr_t>(p_logits) & 15) == 0 &&
                       (k_max == 0 || (reinterpret_cast<uintptr_t>(q_logits) & 15) == 0);
  e = launch_vocab_pass(plan, rows, seqs, draft_tokens, seed, k_max, n_accepted, out_tokens, sc + o_ws, st,
                        nullptr, nullptr, aligned, n_rows);
  return e == hipSuccess ? SPEC_OK : SPEC_E_HIP;
}

}  // extern "C"
