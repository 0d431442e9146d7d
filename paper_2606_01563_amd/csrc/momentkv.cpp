// C ABI of libmomentkv.so: status strings and the ABI version.  The entry points of each
// path live beside it: compress_abi.cpp, decode_abi.cpp, evict_abi.cpp.
#include <cstdint>

#include "../../include/momentkv.h"

extern "C" {

const char* momentkv_status_string(int32_t s) {
  switch (s) {
    case MKV_OK: return "ok";
    case MKV_ERR_NULL: return "a required pointer is NULL";
    case MKV_ERR_SHAPE: return "invalid shape or parameter";
    case MKV_ERR_BUDGET: return "budget too small (below sink + window, or below 1 row)";
    case MKV_ERR_DTYPE: return "unsupported dtype";
    case MKV_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case MKV_ERR_CAPACITY: return "cache capacity too small";
    case MKV_ERR_ALIAS: return "output buffer overlaps an input";
    case MKV_ERR_HIP: return "HIP launch failed";
    case MKV_ERR_UNSUPPORTED: return "request outside this build's limits";
    default: return "unknown status";
  }
}

int32_t momentkv_abi_version(void) { return MOMENTKV_ABI_VERSION; }

}  // extern "C"
