// Library-wide C entry points that launch nothing.
#include "common.hpp"

extern "C" const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_EINVAL: return "MOE_EINVAL: invalid argument";
    case MOE_EUNSUPPORTED: return "MOE_EUNSUPPORTED: unsupported request";
    case MOE_EHIP: return "MOE_EHIP: HIP launch failed";
    case MOE_EWORKSPACE: return "MOE_EWORKSPACE: workspace missing or too small";
    default: return "unknown moe_status";
  }
}

extern "C" int moe_abi_version(void) { return 1; }
