// Status names and version string of libleap.
#include "leap_common.h"

LEAP_API const char* leap_status_string(leap_status s) {
    switch (s) {
        case LEAP_OK: return "LEAP_OK";
        case LEAP_ERR_INVALID_ARG: return "LEAP_ERR_INVALID_ARG";
        case LEAP_ERR_MISALIGNED: return "LEAP_ERR_MISALIGNED";
        case LEAP_ERR_WORKSPACE: return "LEAP_ERR_WORKSPACE";
        case LEAP_ERR_UNSUPPORTED: return "LEAP_ERR_UNSUPPORTED";
        case LEAP_ERR_HIP: return "LEAP_ERR_HIP";
    }
    return "LEAP_ERR_UNKNOWN";
}

LEAP_API const char* leap_version(void) { return "0.1.0"; }
