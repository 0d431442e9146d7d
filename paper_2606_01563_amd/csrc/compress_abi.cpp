// C ABI of the prefill compression: argument checks, workspace layout and the launch.
// Nothing here allocates, frees or synchronises; every launch goes to the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "../../include/momentkv.h"
#include "mkv_abi.h"
#include "mkv_compress.h"

using namespace mkv::abi;

namespace {

constexpr int kMaxCandidates = 1 << 20;  // top-k: at most 512 slices of 2048 candidates
constexpr int kMaxRounds = 8;          // moment rounds after the provisional one

// ----------------------------------------------------------------------- compress
mkv_status check_compress_params(const mkv_compress_params* p) {
  if (!p) return MKV_ERR_NULL;
  if (p->dtype != MKV_F32 && p->dtype != MKV_BF16) return MKV_ERR_DTYPE;
  if (p->batch < 1 || p->n_q_heads < 1 || p->n_kv_heads < 1 || p->head_dim < 1 || p->ctx_len < 2)
    return MKV_ERR_SHAPE;
  if (p->n_q_heads % p->n_kv_heads) return MKV_ERR_SHAPE;
  if (p->window < 1 || p->window >= p->ctx_len) return MKV_ERR_SHAPE;
  if (p->n_sink < 0 || p->n_sink > p->ctx_len - p->window) return MKV_ERR_SHAPE;
  if (p->chunk < 1 || p->budget < 1) return MKV_ERR_SHAPE;
  if (!(p->scale >= 0.f) || !std::isfinite(p->scale) || !(p->tau >= 0.f) || !std::isfinite(p->tau))
    return MKV_ERR_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return MKV_ERR_UNSUPPORTED;
  if (p->n_q_heads / p->n_kv_heads > 16) return MKV_ERR_UNSUPPORTED;
  if ((p->n_q_heads / p->n_kv_heads) * p->window > 512) return MKV_ERR_UNSUPPORTED;
  if (64 % p->chunk) return MKV_ERR_UNSUPPORTED;
  if (p->mi_rounds < -1 || p->mi_rounds > kMaxRounds) return MKV_ERR_UNSUPPORTED;
  if (p->ctx_len - p->window - p->n_sink > kMaxCandidates) return MKV_ERR_UNSUPPORTED;
  if (p->budget < p->ctx_len && p->budget < p->n_sink + p->window) return MKV_ERR_BUDGET;
  if (p->adaptive != 0 && p->adaptive != 1) return MKV_ERR_SHAPE;
  if (p->moment_dtype != MKV_F32 && p->moment_dtype != MKV_BF16) return MKV_ERR_DTYPE;
  int n_out = p->budget < p->ctx_len ? p->budget : p->ctx_len;
  if (p->adaptive && p->budget < p->ctx_len) {
    const int64_t n_c = p->ctx_len - p->window - p->n_sink;
    const int64_t k_keep = p->budget - p->n_sink - p->window;
    if ((int64_t)p->n_kv_heads * n_c > kMaxCandidates) return MKV_ERR_UNSUPPORTED;
    n_out = (int)(p->n_sink + p->window + std::min<int64_t>(n_c, (int64_t)p->n_kv_heads * k_keep));
  }
  if (p->cap < n_out) return MKV_ERR_CAPACITY;
  const double elems = (double)p->batch * p->n_kv_heads * p->ctx_len * p->head_dim;
  if (elems > 4.0e12) return MKV_ERR_UNSUPPORTED;
  return MKV_OK;
}

mkv::CompressArgs compress_layout(const mkv_compress_params* p, void* ws, size_t* total) {
  mkv::CompressArgs a;
  std::memset(&a, 0, sizeof a);
  a.B = p->batch;
  a.Hq = p->n_q_heads;
  a.Hkv = p->n_kv_heads;
  a.G = p->n_q_heads / p->n_kv_heads;
  a.D = p->head_dim;
  a.N = p->ctx_len;
  a.L = p->budget;
  a.w = p->window;
  a.n_s = p->n_sink;
  a.chunk = p->chunk;
  a.mi_rounds = p->mi_rounds;
  a.cap = p->cap;
  a.H = a.B * a.Hkv;
  a.R = a.G * a.w;
  a.n_c = a.N - a.w - a.n_s;
  a.k_keep = a.L < a.N ? a.L - a.n_s - a.w : 0;
  a.adaptive = (p->adaptive && a.L < a.N) ? 1 : 0;
  // rows of the kept-candidate buffers: k_keep, or the most any head can take
  const int kcap = a.adaptive ? std::min(a.n_c, a.Hkv * a.k_keep) : a.k_keep;
  a.kmax = kcap > 1 ? kcap : 1;
  a.idx_stride = a.adaptive ? p->cap : std::min(a.L, a.N);
  a.scale = p->scale > 0.f ? p->scale : 1.0f / std::sqrt((float)a.D);
  a.tau = p->tau;
  a.ntile = ceil_div(a.N, 64);
  // window-row / covariance pass: about one workgroup per CU (it runs one per CU),
  // whole 64-token tiles each, at most kRowsMaxTiles
  a.nsl1 = clampi(ceil_div(256, a.H), 1, a.ntile);
  a.tps1 = std::min(ceil_div(a.ntile, a.nsl1), mkv::kRowsMaxTiles);
  a.nsl1 = ceil_div(a.ntile, a.tps1);
  // window-mass pass: about 1024 workgroups of 256 threads
  a.nsl2 = clampi(ceil_div(1024, a.H), 1, a.ntile);
  a.tps2 = std::min(ceil_div(a.ntile, a.nsl2), mkv::kMassMaxTiles);
  a.nsl2 = ceil_div(a.ntile, a.tps2);
  // top-k slices of 2048 candidates (at most 512 for kMaxCandidates); each slice's
  // workgroup also writes one covariance slot of its kept (or evicted) rows
  a.ntk = ceil_div(a.n_c > 0 ? a.n_c : 1, 2048);
  a.nslot = a.nsl1 + (a.k_keep > 0 ? a.ntk : 0);
  // residual pass: 64-candidate tiles, about 512 workgroups
  {
    const int nu = ceil_div(a.n_c > 0 ? a.n_c : 1, 64);
    a.nsl3 = clampi(ceil_div(512, a.H), 1, nu);
    a.tps3 = std::min(ceil_div(nu, a.nsl3), mkv::kResMaxTiles);
    a.nsl3 = ceil_div(nu, a.tps3);
  }
  a.ntk_g = a.adaptive ? ceil_div(a.Hkv * a.n_c, 2048) : 1;
  const size_t H = a.H, D = a.D;
  const size_t nc = a.n_c > 0 ? a.n_c : 1;
  Carver c;
  c.base = static_cast<char*>(ws);
  a.rowpart = c.take<float>(H * a.nsl1 * a.R * 2 * sizeof(float));
  a.rowstat = c.take<float>(H * a.R * 2 * sizeof(float));
  a.vnorm = c.take<float>(H * nc * sizeof(float));
  a.abar = c.take<float>(H * nc * sizeof(float));
  a.score0 = c.take<float>(H * nc * sizeof(float));
  a.score = c.take<float>(H * nc * sizeof(float));
  a.kept0 = c.take<int32_t>(H * a.kmax * sizeof(int32_t));
  a.kept = c.take<int32_t>(H * a.kmax * sizeof(int32_t));
  a.tk_hh = c.take<uint32_t>(2 * H * 2048 * sizeof(uint32_t));
  a.tk_state = c.take<int32_t>(H * 2 * sizeof(int32_t));
  a.tk_cnt = c.take<int32_t>(H * a.ntk * 2 * sizeof(int32_t));
  a.tk_cand = c.take<uint32_t>(H * a.ntk * 2048 * sizeof(uint32_t));
  a.spart = c.take<float>(H * a.nslot * D * D * sizeof(float));
  a.svkpart = c.take<float>(H * a.nslot * 2 * D * sizeof(float));
  a.s0 = c.take<float>(H * D * D * sizeof(float));
  a.sv0 = c.take<float>(H * D * sizeof(float));
  a.sk0 = c.take<float>(H * D * sizeof(float));
  if (a.adaptive) {
    const size_t Bs = a.B;
    a.kh = c.take<int32_t>(H * sizeof(int32_t));
    a.kept_all = c.take<int32_t>(Bs * a.Hkv * std::max(a.k_keep, 1) * sizeof(int32_t));
    a.tk_hs = c.take<uint32_t>(Bs * 2048 * sizeof(uint32_t));
    a.tk_state_g = c.take<int32_t>(Bs * 2 * sizeof(int32_t));
    a.tk_cnt_g = c.take<int32_t>(Bs * a.ntk_g * 2 * sizeof(int32_t));
    a.tk_cand_g = c.take<uint32_t>(Bs * a.ntk_g * 2048 * sizeof(uint32_t));
  }
  *total = c.off;
  return a;
}

}  // namespace

extern "C" {

size_t momentkv_compress_workspace_size(const mkv_compress_params* p) {
  if (check_compress_params(p) != MKV_OK) return 0;
  size_t total = 0;
  compress_layout(p, nullptr, &total);
  return total;
}

size_t momentkv_compress_workspace_bytes(const mkv_compress_params* p) {
  return momentkv_compress_workspace_size(p);
}

mkv_status momentkv_compress(const mkv_compress_params* p, const void* q_win, const void* k,
                             const void* v, void* k_out, void* v_out, int32_t* idx_out,
                             int32_t* lens_out, int32_t* n_e, float* s_k, float* s_v, void* S,
                             const mkv_compress_debug* dbg, void* workspace,
                             size_t workspace_bytes, void* stream) {
  mkv_status st = check_compress_params(p);
  if (st != MKV_OK) return st;
  if (!q_win || !k || !v || !k_out || !v_out || !idx_out || !lens_out || !n_e || !s_k || !s_v || !S)
    return MKV_ERR_NULL;
  size_t need = 0;
  compress_layout(p, nullptr, &need);
  if (!workspace || workspace_bytes < need) return MKV_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign) return MKV_ERR_WORKSPACE;
  const size_t es = elem_size(p->dtype);
  const size_t in_bytes = (size_t)p->batch * p->n_kv_heads * p->ctx_len * p->head_dim * es;
  const size_t out_bytes = (size_t)p->batch * p->n_kv_heads * p->cap * p->head_dim * es;
  if (ranges_overlap(k_out, out_bytes, k, in_bytes) || ranges_overlap(k_out, out_bytes, v, in_bytes) ||
      ranges_overlap(v_out, out_bytes, k, in_bytes) || ranges_overlap(v_out, out_bytes, v, in_bytes) ||
      ranges_overlap(k_out, out_bytes, v_out, out_bytes) ||
      ranges_overlap(workspace, need, k, in_bytes) || ranges_overlap(workspace, need, v, in_bytes) ||
      ranges_overlap(workspace, need, k_out, out_bytes) || ranges_overlap(workspace, need, v_out, out_bytes))
    return MKV_ERR_ALIAS;
  size_t total = 0;
  mkv::CompressArgs a = compress_layout(p, workspace, &total);
  a.q_win = q_win;
  a.k = k;
  a.v = v;
  a.k_out = k_out;
  a.v_out = v_out;
  a.idx_out = idx_out;
  a.lens_out = lens_out;
  a.n_e = n_e;
  a.s_k = s_k;
  a.s_v = s_v;
  a.S = S;
  a.S_bf16 = p->moment_dtype == MKV_BF16 ? 1 : 0;
  hipError_t e = mkv::launch_compress(a, p->dtype == MKV_BF16, static_cast<hipStream_t>(stream),
                                      dbg ? dbg->abar : nullptr, dbg ? dbg->score0 : nullptr,
                                      dbg ? dbg->score : nullptr, dbg ? dbg->kept0 : nullptr);
  return e == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

}  // extern "C"
