// The corrected decode without a workspace argument, for callers that cannot allocate
// device memory: its partial results live in a file-scope device array of this library,
// one copy per GPU, whose device address is looked up once per device.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "../../include/momentkv.h"
#include "mkv_abi.h"
#include "mkv_decode.h"

using namespace mkv::abi;

namespace {

constexpr size_t kScratchBytes = MOMENTKV_NOALLOC_SCRATCH_BYTES;
// Arrival counters of the split launch: a fixed region at the start of the array, so that
// calls of every shape find them where the previous call left them (at zero).  A call
// needs at least 512 bytes of partials per KV head, so no call that fits the array has
// more heads than this.
constexpr size_t kCounterSlots = kScratchBytes / 512;

// The decode workspace of momentkv_decode_attn_noalloc.  In host code this name is only a
// stand-in for the symbol: its device address comes from hipGetSymbolAddress, per device.
// Zero when the code object is loaded; every call leaves its counter region at zero.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each GPU (null: not looked up)

// Device address of the current GPU's copy of `scratch`, looked up on the first call with
// that device current (hipGetSymbolAddress allocates nothing: the array is part of the
// loaded code object).
hipError_t scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

mkv_status momentkv_decode_attn_noalloc(const mkv_decode_params* p, const void* q, void* k_cache,
                                        void* v_cache, int32_t* lens, const void* k_new,
                                        const void* v_new, const int32_t* n_e, const float* s_k,
                                        const float* s_v, const void* S, void* out,
                                        float* lse_out, float* w_r_out, int32_t* flag,
                                        void* stream) {
  mkv_status st = check_decode_params(p);
  if (st != MKV_OK) return st;
  size_t need = 0;
  decode_layout(p, nullptr, &need, kCounterSlots);
  if (need > kScratchBytes || (size_t)p->batch * p->n_kv_heads > kCounterSlots)
    return MKV_ERR_WORKSPACE;
  st = check_decode_buffers(p, q, k_cache, v_cache, lens, k_new, v_new, n_e, s_k, s_v, S, out);
  if (st != MKV_OK) return st;
  if (flag && decode_overlaps(p, flag, sizeof(int32_t), k_cache, v_cache, out)) return MKV_ERR_ALIAS;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return MKV_ERR_HIP;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev) != hipSuccess) return MKV_ERR_HIP;
    if (sdev != dev) return MKV_ERR_UNSUPPORTED;
  }
  void* ws = nullptr;
  if (scratch_address(dev, &ws) != hipSuccess) return MKV_ERR_HIP;
  size_t total = 0;
  mkv::DecodeArgs a = decode_layout(p, ws, &total, kCounterSlots);
  if (flag) a.flag = flag;  // otherwise the flag slot of the scratch, which nobody reads
  set_decode_buffers(a, q, k_cache, v_cache, lens, k_new, v_new, n_e, s_k, s_v, S, out, lse_out,
                     w_r_out);
  const hipError_t e = mkv::launch_decode(a, p->dtype == MKV_BF16, p->head_dim,
                                          static_cast<hipStream_t>(stream));
  return e == hipSuccess ? MKV_OK : MKV_ERR_HIP;
}

}  // extern "C"
