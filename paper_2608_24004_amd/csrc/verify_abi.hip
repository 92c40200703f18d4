// verify_abi.hip -- status strings and the ABI version of the verify library
// (host code only; kept apart from the kernels so that a version bump leaves
// the kernel sources unchanged).
#include "common.h"

extern "C" const char* verify_status_string(int status) {
    switch (status) {
        case VERIFY_OK: return "ok";
        case VERIFY_EINVAL: return "invalid argument";
        case VERIFY_EUNSUPPORTED: return "unsupported shape or dtype";
        case VERIFY_EWORKSPACE: return "workspace too small";
        case VERIFY_EHIP: return "HIP launch failure";
        default: return "unknown status";
    }
}

extern "C" int verify_abi_version(void) { return 10800; }
