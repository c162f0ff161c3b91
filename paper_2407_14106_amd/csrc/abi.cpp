// Status codes, error text and ABI version of libgt.
#include <string>

#include "common.h"

namespace gt {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

gt_status fail(gt_status code, const std::string& msg) {
    g_last_error = msg;
    return code;
}

gt_status hip_fail(hipError_t e, const char* what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return GT_ERR_HIP;
}

}  // namespace gt

extern "C" {

int32_t gt_abi_version(void) { return 2; }

const char* gt_status_string(gt_status status) {
    switch (status) {
        case GT_OK: return "ok";
        case GT_ERR_INVALID_ARG: return "invalid argument";
        case GT_ERR_UNSUPPORTED: return "unsupported configuration";
        case GT_ERR_UNSORTED: return "CSR row not strictly increasing";
        case GT_ERR_DUPLICATE: return "duplicate CSR entry";
        case GT_ERR_OUT_OF_RANGE: return "index out of range";
        case GT_ERR_WORKSPACE: return "workspace too small";
        case GT_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char* gt_last_error(void) { return gt::g_last_error.c_str(); }

}  // extern "C"
