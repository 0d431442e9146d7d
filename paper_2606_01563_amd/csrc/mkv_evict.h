// Launch interface of the decode step with eviction (see evict.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

// Decode step with eviction (Algorithm 1 Phase 1): scoring and selection ahead of the
// corrected attention, which then runs through launch_decode on the updated state.
struct EvictArgs {
  const void* q;            // [B, Hq, D]
  void* k_cache;            // [B, Hkv, cap, D]
  void* v_cache;
  int32_t* lens;            // [B, Hkv]
  const void* k_new;        // [B, Hkv, D]
  const void* v_new;
  int32_t* n_e;             // [B, Hkv]      raw summary, updated in place
  float* s_k;               // [B, Hkv, D]
  float* s_v;
  float* S;                 // [B, Hkv, D, D]
  int32_t* evicted;         // [B, Hkv] or null: slot evicted by this call, -1 if none
  float* rec;               // [B*Hkv, G + 2, rec_len]  per row: G base-2 logits, log2 ||r||,
                            // then a row that takes the logits of padded query slots
  int32_t* flag;            // sticky flag: 1 no room for the new row, 2 lens past max_len,
                            // 4 no finite score, 8 lens above budget before the append
  int n_heads, G, cap, max_len, budget;
  int nslice, slice_len;    // scoring workgroups per KV head, rows per workgroup (x 32)
  int rec_len;              // max_len rounded up to 32: whole blocks of records fit
  float scale, tau;
};

hipError_t launch_evict(const EvictArgs& e, bool bf16, int d, hipStream_t st);

}  // namespace mkv
