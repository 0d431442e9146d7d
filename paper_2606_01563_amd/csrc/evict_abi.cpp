// C ABI of the decode step with eviction: argument checks, workspace layout (the decode
// layout followed by the per-row score records) and the launch sequence.  Nothing here
// allocates, frees or synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdint>
#include <cstring>

#include "../../include/momentkv.h"
#include "mkv_abi.h"
#include "mkv_evict.h"
#include "mkv_decode.h"

using namespace mkv::abi;

namespace {

// ------------------------------------------------------------------ decode + eviction
// Workspace: the decode layout (its flag first), then the per-row score records.  Scoring
// workgroups: slices of a multiple of 32 rows (at least 128), as many per head as keep
// the busiest CU's work lowest (a CU's scoring throughput is shared by the workgroups it
// holds), counting each workgroup's forming of S_tilde as 96 rows and, with more than
// one slice per head, the separate selection launch as 384.
mkv::EvictArgs evict_layout(const mkv_decode_params* p, int32_t budget, void* ws,
                            size_t* total, mkv::DecodeArgs* da) {
  size_t dec = 0;
  *da = decode_layout(p, ws, &dec);
  mkv::EvictArgs e;
  std::memset(&e, 0, sizeof e);
  e.n_heads = da->n_heads;
  e.G = da->G;
  e.cap = p->cap;
  e.max_len = p->max_len;
  e.budget = budget;
  e.scale = da->scale;
  e.tau = da->tau;
  e.flag = da->flag;
  constexpr int64_t kCUs = 256, kBuildRows = 96, kSelectRows = 384;
  int best = 1;
  int64_t best_cost = INT64_MAX;
  for (int ns = 1; ns <= std::max(1, p->max_len / 128); ++ns) {
    const int64_t rows = (int64_t)ceil_div(ceil_div(p->max_len, ns), 32) * 32;
    const int64_t cost = ((int64_t)e.n_heads * ns + kCUs - 1) / kCUs * (rows + kBuildRows) +
                         (ns > 1 ? kSelectRows : 0);
    if (cost < best_cost) {
      best_cost = cost;
      best = ns;
    }
  }
  e.slice_len = ceil_div(ceil_div(p->max_len, best), 32) * 32;
  e.nslice = ceil_div(p->max_len, e.slice_len);
  Carver c;
  c.base = static_cast<char*>(ws);
  c.off = dec;
  e.rec_len = ceil_div(p->max_len, 32) * 32;
  e.rec = c.take<float>((size_t)e.n_heads * (e.G + 2) * e.rec_len * sizeof(float));
  *total = c.off;
  return e;
}

mkv_status check_evict_params(const mkv_decode_params* p, int32_t budget) {
  mkv_status st = check_decode_params(p);
  if (st != MKV_OK) return st;
  if (p->summary != 0) return MKV_ERR_SHAPE;
  if (budget < 1) return MKV_ERR_BUDGET;
  return MKV_OK;
}

}  // namespace

extern "C" {

size_t momentkv_decode_evict_workspace_size(const mkv_decode_params* p) {
  if (check_evict_params(p, 1) != MKV_OK) return 0;
  size_t total = 0;
  mkv::DecodeArgs da;
  evict_layout(p, 1, nullptr, &total, &da);
  return total;
}

mkv_status momentkv_decode_evict(const mkv_decode_params* p, int32_t budget, const void* q,
                                 void* k_cache, void* v_cache, int32_t* lens,
                                 const void* k_new, const void* v_new, int32_t* n_e,
                                 float* s_k, float* s_v, float* S, void* out, float* lse_out,
                                 float* w_r_out, int32_t* evicted_out, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  mkv_status st = check_evict_params(p, budget);
  if (st != MKV_OK) return st;
  if (!q || !k_cache || !v_cache || !lens || !k_new || !v_new || !n_e || !s_k || !s_v || !S || !out)
    return MKV_ERR_NULL;
  size_t need = 0;
  mkv::DecodeArgs da;
  evict_layout(p, budget, nullptr, &need, &da);
  if (!workspace || workspace_bytes < need) return MKV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign) return MKV_ERR_WORKSPACE;
  const size_t es = elem_size(p->dtype);
  const size_t heads = (size_t)p->batch * p->n_kv_heads, d = p->head_dim;
  const size_t cache_bytes = heads * p->cap * d * es;
  const size_t out_bytes = (size_t)p->batch * p->n_q_heads * d * es;
  const size_t s_bytes = heads * d * d * 4, vec_bytes = heads * d * 4;
  const void* outs[] = {k_cache, v_cache, out, S, s_k, s_v, workspace};
  const size_t outn[] = {cache_bytes, cache_bytes, out_bytes, s_bytes, vec_bytes, vec_bytes, need};
  for (int i = 0; i < 7; ++i)
    for (int j = i + 1; j < 7; ++j)
      if (ranges_overlap(outs[i], outn[i], outs[j], outn[j])) return MKV_ERR_ALIAS;
  if (ranges_overlap(out, out_bytes, q, out_bytes)) return MKV_ERR_ALIAS;
  size_t total = 0;
  mkv::EvictArgs e = evict_layout(p, budget, workspace, &total, &da);
  e.q = q;
  e.k_cache = k_cache;
  e.v_cache = v_cache;
  e.lens = lens;
  e.k_new = k_new;
  e.v_new = v_new;
  e.n_e = n_e;
  e.s_k = s_k;
  e.s_v = s_v;
  e.S = S;
  e.evicted = evicted_out;
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  hipError_t err = mkv::launch_evict(e, p->dtype == MKV_BF16, p->head_dim, hs);
  if (err != hipSuccess) return MKV_ERR_HIP;
  da.q = q;
  da.k_cache = k_cache;
  da.v_cache = v_cache;
  da.lens = lens;
  da.k_new = nullptr;  // appended by the eviction step
  da.v_new = nullptr;
  da.n_e = n_e;
  da.s_k = s_k;
  da.s_v = s_v;
  da.S = S;
  da.out = out;
  da.lse_out = lse_out;
  da.w_r_out = w_r_out;
  err = mkv::launch_decode(da, p->dtype == MKV_BF16, p->head_dim, hs);
  return err == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

}  // extern "C"
