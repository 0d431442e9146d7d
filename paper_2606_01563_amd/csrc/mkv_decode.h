// Host <-> device interface of the decode kernels (decode.hip): the argument block passed
// by value and the launchers the C ABI layer calls.  Pointers are device pointers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mkv {

struct DecodeArgs {
  const void* q;            // [B, Hq, D]
  void* k_cache;            // [B, Hkv, cap, D]
  void* v_cache;
  int32_t* lens;            // [B, Hkv]
  const void* k_new;        // [B, Hkv, D] or null
  const void* v_new;
  const int32_t* n_e;       // [B, Hkv]
  const float* s_k;         // [B, Hkv, D]
  const float* s_v;
  const float* S;           // [B, Hkv, D, D] raw fp32 sum (summary 0), the prepared form
                            // (1, 2), or the raw sum stored in bf16 (3)
  void* out;                // [B, Hq, D]
  float* lse_out;           // [B, Hq] or null
  float* w_r_out;           // [B, Hq] or null
  float* part_o;            // [B*Hkv, nsplit, G, D]  unnormalised slice outputs
  float* part_ml;           // [B*Hkv, nsplit, G, 2]  (max in log2 units, sum)
  float* sq;                // [B*Hkv, G, D]  S_tilde q (unscaled)
  int32_t* flag;            // sticky append-overflow flag
  int32_t* cnt;             // [n_heads] arrival counters of the split launch, zero between calls
  int n_heads;              // B * Hkv
  int n_pairs;              // B * Hq
  int Hkv, G, cap;
  int fused;                // 1: one workgroup per KV head, single launch
  int nsplit, split_len;    // split launch: token slices per KV head, rows per slice (x 32)
  int nsq;                  // S_tilde q waves per KV head (D / 32 rows each; 0 at order 0)
  int summary;              // 0: raw fp32 S; 1, 2: prepared forms; 3: raw bf16 S
  int order;
  float scale, tau;
};

hipError_t launch_decode(const DecodeArgs& a, bool bf16, int d, hipStream_t st);
// Prepared summary from a.n_e, a.s_k, a.s_v, a.S (raw) into `prepared`.
hipError_t launch_prepare_summary(const DecodeArgs& a, void* prepared, bool bf16, int d,
                                  hipStream_t st);

}  // namespace mkv
