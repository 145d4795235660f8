// abi.hip -- status strings and the version of libstagefrontier.

#include "sf_host.h"

SF_API const char* sf_strerror(int status)
{
    switch (status) {
    case SF_OK: return "success";
    case SF_EINVAL: return "invalid argument";
    case SF_ERANGE: return "value out of range";
    case SF_EHIP: return "HIP kernel launch failed";
    default: return "unknown status";
    }
}

SF_API const char* sf_version(void) { return "libstagefrontier 0.1.0 (gfx950)"; }
