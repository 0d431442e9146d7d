// Launch interface of the decode step with eviction (see evict.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

// Decode step with eviction (Algorithm 1: Phase 1, then Phase 2 on the new state).  Fused
// (one read of the cache): a scoring and attention launch over nwg workgroups that share
// the heads' 32-row blocks evenly, then a finishing launch with one workgroup per head.
// Otherwise one launch with one workgroup per head: scoring, selection, the update, then
// the attention over the new cache.
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
  void* out;                // [B, Hq, D]
  float* lse_out;           // [B, Hq] or null: log Z_R
  float* w_r_out;           // [B, Hq] or null: mixing weight of the retained part
  int32_t* evicted;         // [B, Hkv] or null: slot evicted by this call, -1 if none
  float* rec;               // [B*Hkv, G + 2, rec_len]  per row: G base-2 logits, log2 ||r||,
                            // then a row that takes the logits of padded query slots
  float* blkm;              // [B*Hkv, G + 1, rec_len / 32]  per 32-row block and query: the
                            // running max (base 2) the block's terms were scaled by; row G
                            // takes padded query slots
  float* part_o;            // [B*Hkv, maxslots, G, D]  unnormalised partial states
  float* part_ml;           // [B*Hkv, maxslots, G, 2]  (max in log2 units, sum)
  int32_t* flag;            // sticky flag: 1 no room for the new row, 2 lens past max_len,
                            // 4 no finite score, 8 lens above budget before the append
  int n_heads, G, cap, max_len, budget;
  int hblocks;              // 32-row blocks per head: ceil(max_len / 32); the last one also
                            // takes rows past max_len
  int nwg;                  // scoring workgroups (each takes a contiguous share of blocks)
  int maxslots;             // the most partial states one head can have
  int rec_len;              // 32 * hblocks: whole blocks of records fit
  int order;                // correction order: -1 none, 0 v_bar only, 1 first order
  int fused;                // 1: the attention in the same pass (see above)
  float scale, tau;
};

hipError_t launch_evict(const EvictArgs& e, bool bf16, int d, hipStream_t st);
// Waves of a scoring workgroup (one workgroup per CU) for the element type and group size,
// and the most partial states per head the finishing launch merges.
int evict_waves(bool bf16, int G);
int evict_max_slices();

}  // namespace mkv
