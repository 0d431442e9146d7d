// C ABI of the decode step with eviction: argument checks, workspace layout and the
// launches.  Nothing here allocates, frees or synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "../../include/momentkv.h"
#include "mkv_abi.h"
#include "mkv_evict.h"

using namespace mkv::abi;

namespace {

// ------------------------------------------------------------------ decode + eviction
// Two launch shapes.  Fused (one read of the cache; from kFusedMinLen rows, or whenever
// n_split > 0): the scoring launch has one workgroup per CU of the target (kCUs; n_split
// per head when n_split > 0), each taking an equal contiguous share of the flattened
// (head, 32-row block) range, so that a head has at most maxslots partial states (at most
// evict_max_slices(); fewer workgroups otherwise); a finishing launch follows.  Short
// caches: one launch with one workgroup per head (two per CU) that scores, selects,
// updates and then attends to the new cache itself (a second read of a short cache,
// mostly from L2); a fused workgroup holds one head's summary and V tiles alone on its
// CU, which there costs more than that second read.
// Workspace: the flag first, then the score records and the per-block running maxima;
// fused: then the heads' partial states.
constexpr int kCUs = 256;
// max_len from which the one-read shape runs (on a 288-head stack it was the faster one
// from 384 rows up and the slower one at 256)
constexpr int kFusedMinLen = 320;

mkv::EvictArgs evict_layout(const mkv_decode_params* p, int32_t budget, void* ws, size_t* total) {
  mkv::EvictArgs e;
  std::memset(&e, 0, sizeof e);
  e.n_heads = p->batch * p->n_kv_heads;
  e.G = p->n_q_heads / p->n_kv_heads;
  e.cap = p->cap;
  e.max_len = p->max_len;
  e.budget = budget;
  e.order = p->order;
  e.scale = p->scale > 0.f ? p->scale : 1.0f / std::sqrt((float)p->head_dim);
  e.tau = p->tau;
  e.hblocks = ceil_div(p->max_len, 32);
  e.rec_len = 32 * e.hblocks;
  e.fused = (p->n_split > 0 || p->max_len >= kFusedMinLen) ? 1 : 0;
  const size_t H = e.n_heads, G = e.G, D = p->head_dim;
  Carver c;
  c.base = static_cast<char*>(ws);
  if (e.fused) {
    const int64_t T = (int64_t)e.n_heads * e.hblocks;
    int64_t nwg = p->n_split > 0 ? (int64_t)p->n_split * e.n_heads : kCUs;
    nwg = std::max<int64_t>(1, std::min(nwg, T));
    auto slots = [&](int64_t n) {
      const int64_t per = std::max<int64_t>(1, T / n);  // the fewest blocks a workgroup takes
      return std::min<int64_t>(n, (e.hblocks + per - 1) / per + 1);
    };
    while (nwg > 1 && slots(nwg) > mkv::evict_max_slices()) --nwg;
    e.nwg = (int)nwg;
    e.maxslots = (int)slots(nwg);
  }
  e.flag = c.take<int32_t>(sizeof(int32_t));  // zero-filled once by the caller
  e.rec = c.take<float>(H * (G + 2) * e.rec_len * sizeof(float));
  e.blkm = c.take<float>(H * (G + 1) * e.hblocks * sizeof(float));
  if (e.fused) {
    e.part_o = c.take<float>(H * e.maxslots * G * D * sizeof(float));
    e.part_ml = c.take<float>(H * e.maxslots * G * 2 * sizeof(float));
  }
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
  evict_layout(p, 1, nullptr, &total);
  return total;
}

size_t momentkv_decode_evict_workspace_bytes(const mkv_decode_params* p) {
  return momentkv_decode_evict_workspace_size(p);
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
  evict_layout(p, budget, nullptr, &need);
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
  mkv::EvictArgs e = evict_layout(p, budget, workspace, &total);
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
  e.out = out;
  e.lse_out = lse_out;
  e.w_r_out = w_r_out;
  const hipStream_t hs = static_cast<hipStream_t>(stream);
  return mkv::launch_evict(e, p->dtype == MKV_BF16, p->head_dim, hs) == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

}  // extern "C"
