// Status strings and version of the libdpgrad C ABI.
#include "common.hpp"

extern "C" const char *dp_status_string(dp_status s)
{
    switch (s) {
    case DP_OK: return "DP_OK: success";
    case DP_EINVAL: return "DP_EINVAL: invalid argument (null pointer, size, or workspace too small)";
    case DP_EDTYPE: return "DP_EDTYPE: unknown dtype";
    case DP_EUNSUPPORTED: return "DP_EUNSUPPORTED: valid request not implemented by this library";
    case DP_ECAP: return "DP_ECAP: capacity too small";
    case DP_EHIP: return "DP_EHIP: HIP kernel launch failed";
    }
    return "unknown dp_status";
}

extern "C" int dp_abi_version(void) { return 1; }
