// Library-wide entry points of liblipcache: status strings and ABI version.
#include "lc_common.hpp"

extern "C" const char* lipcache_status_string(lipcache_status status) {
  switch (status) {
    case LIPCACHE_OK: return "ok";
    case LIPCACHE_EINVAL: return "invalid argument";
    case LIPCACHE_EDEGENERATE: return "degenerate head: sigma_max(W) <= 0";
    case LIPCACHE_ENOCONV: return "power iteration did not converge within max_iters";
    case LIPCACHE_ECAPACITY: return "insert exceeds the cache capacity; nothing appended";
    case LIPCACHE_EUNSUPPORTED: return "unsupported by this build";
    case LIPCACHE_EWORKSPACE: return "workspace missing, too small or not 256-byte aligned";
    case LIPCACHE_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

extern "C" int32_t lipcache_abi_version(void) { return LIPCACHE_ABI_VERSION; }
