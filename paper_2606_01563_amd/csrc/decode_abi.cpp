// C ABI of the corrected decode: argument checks, launch shape, workspace layout and the
// launches.  Nothing here allocates, frees or synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "../../include/momentkv.h"
#include "mkv_abi.h"
#include "mkv_decode.h"

using namespace mkv::abi;

namespace {

constexpr int64_t kDecodeWaves = 768;      // target slice count of an automatic decode split
constexpr int64_t kMaxDecodeWaves = 1 << 24;  // decode grid limit (single-wave workgroups)
constexpr int kFusedMaxLen = 384;          // automatic decode: single launch up to this length

// ----------------------------------------------------------------------- decode
// Token slices per KV head.  Automatic (n_split = 0): about kDecodeWaves single-wave
// slices in the whole grid (three per CU), at least 32 rows each.  Measured on a 288-head
// stack, longer slices (fewer partials to merge) beat finer splits once every CU holds a
// few slices.  Rows per slice are a multiple of the 32-row block.
void decode_split(const mkv_decode_params* p, int* split_len, int* nsplit) {
  const int64_t heads = (int64_t)p->batch * p->n_kv_heads;
  const int want = p->n_split > 0 ? p->n_split
                                  : (int)std::min<int64_t>(std::max<int64_t>((kDecodeWaves + heads - 1) / heads, 1), 1 << 20);
  int sl = ceil_div(p->max_len, want);
  sl = std::max(32, ceil_div(sl, 32) * 32);
  *split_len = sl;
  *nsplit = ceil_div(p->max_len, sl);
}

// One workgroup per KV head (single launch) for n_split = 1, or automatically for short
// caches, where a call is bound by latency rather than by how the heads spread over CUs.
bool decode_fused(const mkv_decode_params* p) {
  return p->n_split == 1 || (p->n_split == 0 && p->max_len <= kFusedMaxLen);
}

}  // namespace

namespace mkv {
namespace abi {

mkv_status check_decode_params(const mkv_decode_params* p) {
  if (!p) return MKV_ERR_NULL;
  if (p->dtype != MKV_F32 && p->dtype != MKV_BF16) return MKV_ERR_DTYPE;
  if (p->batch < 1 || p->n_q_heads < 1 || p->n_kv_heads < 1 || p->head_dim < 1 || p->cap < 1)
    return MKV_ERR_SHAPE;
  if (p->n_q_heads % p->n_kv_heads) return MKV_ERR_SHAPE;
  if (p->order < -1 || p->order > 1) return MKV_ERR_SHAPE;
  if (!(p->scale >= 0.f) || !std::isfinite(p->scale) || !(p->tau >= 0.f) || !std::isfinite(p->tau))
    return MKV_ERR_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return MKV_ERR_UNSUPPORTED;
  if (p->n_q_heads / p->n_kv_heads > 16) return MKV_ERR_UNSUPPORTED;
  if (p->n_split < 0) return MKV_ERR_SHAPE;
  if (p->summary < 0 || p->summary > 3) return MKV_ERR_SHAPE;
  if (p->summary == 2 && p->dtype != MKV_BF16) return MKV_ERR_SHAPE;  // half precision: bf16 only
  if (p->max_len < 1 || p->max_len > p->cap) return MKV_ERR_CAPACITY;
  // grid of single-wave workgroups: B * Hkv * (slices + covariance waves)
  int split_len = 0, nsplit = 0;
  decode_split(p, &split_len, &nsplit);
  const int64_t waves = (int64_t)p->batch * p->n_kv_heads * (nsplit + p->head_dim / 32);
  if (waves > kMaxDecodeWaves) return MKV_ERR_UNSUPPORTED;
  return MKV_OK;
}

mkv::DecodeArgs decode_layout(const mkv_decode_params* p, void* ws, size_t* total,
                              size_t cnt_slots) {
  mkv::DecodeArgs a;
  std::memset(&a, 0, sizeof a);
  a.n_heads = p->batch * p->n_kv_heads;
  a.G = p->n_q_heads / p->n_kv_heads;
  a.n_pairs = p->batch * p->n_q_heads;
  a.Hkv = p->n_kv_heads;
  a.cap = p->cap;
  a.order = p->order;
  a.scale = p->scale > 0.f ? p->scale : 1.0f / std::sqrt((float)p->head_dim);
  a.tau = p->tau;
  decode_split(p, &a.split_len, &a.nsplit);
  a.fused = decode_fused(p) ? 1 : 0;
  a.nsq = p->order >= 1 ? p->head_dim / 32 : 0;
  a.summary = p->summary;
  const size_t H = a.n_heads, D = p->head_dim, G = a.G;
  Carver c;
  c.base = static_cast<char*>(ws);
  // The leading bytes (the flag, then one arrival counter per head) are zero-filled by
  // the caller before first use; every call leaves the counters at zero.
  a.flag = c.take<int32_t>(sizeof(int32_t));
  a.cnt = c.take<int32_t>(std::max<size_t>(cnt_slots, H) * sizeof(int32_t));
  a.part_o = c.take<float>(H * a.nsplit * G * D * sizeof(float));
  a.part_ml = c.take<float>(H * a.nsplit * G * 2 * sizeof(float));
  a.sq = c.take<float>(H * G * D * sizeof(float));
  *total = c.off;
  return a;
}

mkv_status check_decode_buffers(const mkv_decode_params* p, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* lens, const void* k_new,
                                const void* v_new, const int32_t* n_e, const float* s_k,
                                const float* s_v, const void* S, const void* out) {
  if (!q || !k_cache || !v_cache || !lens || !n_e || !s_k || !s_v || !S || !out) return MKV_ERR_NULL;
  if ((k_new == nullptr) != (v_new == nullptr)) return MKV_ERR_NULL;
  const size_t es = elem_size(p->dtype);
  const size_t cache_bytes = (size_t)p->batch * p->n_kv_heads * p->cap * p->head_dim * es;
  const size_t out_bytes = (size_t)p->batch * p->n_q_heads * p->head_dim * es;
  if (ranges_overlap(out, out_bytes, k_cache, cache_bytes) ||
      ranges_overlap(out, out_bytes, v_cache, cache_bytes) ||
      ranges_overlap(out, out_bytes, q, out_bytes) ||
      ranges_overlap(k_cache, cache_bytes, v_cache, cache_bytes))
    return MKV_ERR_ALIAS;
  return MKV_OK;
}

bool decode_overlaps(const mkv_decode_params* p, const void* buf, size_t bytes,
                     const void* k_cache, const void* v_cache, const void* out) {
  const size_t es = elem_size(p->dtype);
  const size_t cache_bytes = (size_t)p->batch * p->n_kv_heads * p->cap * p->head_dim * es;
  const size_t out_bytes = (size_t)p->batch * p->n_q_heads * p->head_dim * es;
  return ranges_overlap(buf, bytes, k_cache, cache_bytes) ||
         ranges_overlap(buf, bytes, v_cache, cache_bytes) || ranges_overlap(buf, bytes, out, out_bytes);
}

void set_decode_buffers(DecodeArgs& a, const void* q, void* k_cache, void* v_cache, int32_t* lens,
                        const void* k_new, const void* v_new, const int32_t* n_e, const float* s_k,
                        const float* s_v, const void* S, void* out, float* lse_out,
                        float* w_r_out) {
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.lens = lens;
  a.k_new = k_new;
  a.v_new = v_new;
  a.n_e = n_e;
  a.s_k = s_k;
  a.s_v = s_v;
  a.S = static_cast<const float*>(S);
  a.out = out;
  a.lse_out = lse_out;
  a.w_r_out = w_r_out;
}

}  // namespace abi
}  // namespace mkv

extern "C" {

size_t momentkv_decode_workspace_size(const mkv_decode_params* p) {
  if (check_decode_params(p) != MKV_OK) return 0;
  size_t total = 0;
  decode_layout(p, nullptr, &total, 0);
  return total;
}

size_t momentkv_decode_workspace_bytes(const mkv_decode_params* p) {
  return momentkv_decode_workspace_size(p);
}

size_t momentkv_decode_workspace_zero_bytes(const mkv_decode_params* p) {
  if (check_decode_params(p) != MKV_OK) return 0;
  const size_t heads = (size_t)p->batch * p->n_kv_heads;
  return align_up(sizeof(int32_t)) + align_up(heads * sizeof(int32_t));
}

size_t momentkv_prepared_summary_size(const mkv_decode_params* p) {
  if (check_decode_params(p) != MKV_OK || p->summary == 3) return 0;
  return (size_t)p->batch * p->n_kv_heads * p->head_dim * p->head_dim * (p->summary == 2 ? 2 : 4);
}

mkv_status momentkv_prepare_summary(const mkv_decode_params* p, const int32_t* n_e,
                                    const float* s_k, const float* s_v, const float* S,
                                    void* prepared, void* stream) {
  mkv_status st = check_decode_params(p);
  if (st != MKV_OK) return st;
  if (p->summary == 3) return MKV_ERR_SHAPE;  // the raw bf16 form has no prepared form
  if (!n_e || !s_k || !s_v || !S || !prepared) return MKV_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(prepared) % 16) return MKV_ERR_SHAPE;
  const size_t heads = (size_t)p->batch * p->n_kv_heads, d = p->head_dim;
  const size_t out_bytes = heads * d * d * (p->summary == 2 ? 2 : 4);
  if (ranges_overlap(prepared, out_bytes, S, heads * d * d * 4) ||
      ranges_overlap(prepared, out_bytes, s_k, heads * d * 4) ||
      ranges_overlap(prepared, out_bytes, s_v, heads * d * 4) ||
      ranges_overlap(prepared, out_bytes, n_e, heads * 4))
    return MKV_ERR_ALIAS;
  size_t total = 0;
  mkv::DecodeArgs a = decode_layout(p, nullptr, &total, 0);
  a.n_e = n_e;
  a.s_k = s_k;
  a.s_v = s_v;
  a.S = S;
  hipError_t e = mkv::launch_prepare_summary(a, prepared, p->dtype == MKV_BF16, p->head_dim,
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

mkv_status momentkv_decode_attn(const mkv_decode_params* p, const void* q, void* k_cache,
                                void* v_cache, int32_t* lens, const void* k_new,
                                const void* v_new, const int32_t* n_e, const float* s_k,
                                const float* s_v, const void* S, void* out, float* lse_out,
                                float* w_r_out, void* workspace, size_t workspace_bytes,
                                void* stream) {
  mkv_status st = check_decode_params(p);
  if (st != MKV_OK) return st;
  st = check_decode_buffers(p, q, k_cache, v_cache, lens, k_new, v_new, n_e, s_k, s_v, S, out);
  if (st != MKV_OK) return st;
  size_t need = 0;
  decode_layout(p, nullptr, &need, 0);
  if (!workspace || workspace_bytes < need) return MKV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign) return MKV_ERR_WORKSPACE;
  if (decode_overlaps(p, workspace, need, k_cache, v_cache, out)) return MKV_ERR_ALIAS;
  size_t total = 0;
  mkv::DecodeArgs a = decode_layout(p, workspace, &total, 0);
  set_decode_buffers(a, q, k_cache, v_cache, lens, k_new, v_new, n_e, s_k, s_v, S, out, lse_out,
                     w_r_out);
  hipError_t e = mkv::launch_decode(a, p->dtype == MKV_BF16, p->head_dim,
                                    static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

}  // extern "C"
