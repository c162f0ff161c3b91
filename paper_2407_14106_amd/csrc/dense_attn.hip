// Full softmax attention (§2.1 Eq. (1)) on the matrix cores (placeholder).
#include "attn_common.h"

using namespace gt;

static gt_status dense_check(const char* who, int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q,
                             const void* K, const void* V) {
    if (n < 0 || n >= (int64_t(1) << 31)) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": n out of range");
    if (n > 0 && (!Q || !K || !V)) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null pointer");
    if (dt != GT_BF16 || (d != 32 && d != 64) || H < 1 || H > 64)
        return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": bf16, d in {32, 64}, 1 <= H <= 64 only");
    return GT_OK;
}

extern "C" gt_status gt_dense_attn_fwd(int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q, const void* K,
                                       const void* V, float, void* O, float* LSE, hipStream_t) {
    gt_status st = dense_check("gt_dense_attn_fwd", n, H, d, dt, Q, K, V);
    if (st != GT_OK) return st;
    if (n > 0 && (!O || !LSE)) return fail(GT_ERR_INVALID_ARG, "gt_dense_attn_fwd: null pointer");
    return fail(GT_ERR_UNSUPPORTED, "gt_dense_attn_fwd: not built yet");
}
extern "C" size_t gt_dense_attn_bwd_workspace_size(int64_t, int32_t, int32_t, gt_dtype) { return 256; }
extern "C" gt_status gt_dense_attn_bwd(int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q, const void* K,
                                       const void* V, const void*, const void*, const float*, float, void*, void*,
                                       void*, void*, size_t, hipStream_t) {
    gt_status st = dense_check("gt_dense_attn_bwd", n, H, d, dt, Q, K, V);
    if (st != GT_OK) return st;
    return fail(GT_ERR_UNSUPPORTED, "gt_dense_attn_bwd: not built yet");
}
