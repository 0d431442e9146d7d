// Host-side helpers shared by the C ABI translation units (argument checks, workspace
// carving); not part of the public interface.
#pragma once

#include <cstddef>
#include <cstdint>

#include "../../include/momentkv.h"
#include "mkv_decode.h"

namespace mkv {
namespace abi {

constexpr size_t kAlign = 256;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// Bump allocator over a caller's workspace (base = null: only sizes are computed).
struct Carver {
  size_t off = 0;
  char* base = nullptr;
  template <class P> P* take(size_t bytes) {
    P* p = base ? reinterpret_cast<P*>(base + off) : nullptr;
    off += align_up(bytes);
    return p;
  }
};

inline bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

inline size_t elem_size(int32_t dtype) { return dtype == MKV_BF16 ? 2 : 4; }

// Decode parameters and workspace layout (defined with the decode entry points).
mkv_status check_decode_params(const mkv_decode_params* p);
// The arrival counters take max(cnt_slots, heads) slots after the flag (a fixed region when
// one buffer serves calls of every shape).
DecodeArgs decode_layout(const mkv_decode_params* p, void* ws, size_t* total, size_t cnt_slots);
// Required pointers present and the caches, query and output disjoint.
mkv_status check_decode_buffers(const mkv_decode_params* p, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* lens, const void* k_new,
                                const void* v_new, const int32_t* n_e, const float* s_k,
                                const float* s_v, const void* S, const void* out);
// Whether [buf, buf + bytes) overlaps the caches or the output.
bool decode_overlaps(const mkv_decode_params* p, const void* buf, size_t bytes,
                     const void* k_cache, const void* v_cache, const void* out);
// The caller's buffers into the argument block.
void set_decode_buffers(DecodeArgs& a, const void* q, void* k_cache, void* v_cache, int32_t* lens,
                        const void* k_new, const void* v_new, const int32_t* n_e, const float* s_k,
                        const float* s_v, const void* S, void* out, float* lse_out,
                        float* w_r_out);

}  // namespace abi
}  // namespace mkv
