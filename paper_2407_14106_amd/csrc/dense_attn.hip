// Full softmax attention (§2.1 Eq. (1)): the interleaved fully-connected layer
// of §3.2.  bf16 features run the streaming kernels of dense_mfma.hip; fp32
// features run the matrix-core tile kernels with every pair attended.
#include "tile_attn.h"

using namespace gt;

namespace {

gt_status dense_check(const char* who, int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q, const void* K,
                      const void* V) {
    if (n < 0 || n >= (int64_t(1) << 31)) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": n out of range");
    if (n > 0 && (!Q || !K || !V)) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null pointer");
    if ((dt != GT_BF16 && dt != GT_F32) || (d != 32 && d != 64) ||
        !(H == 1 || H == 2 || H == 4 || H == 8 || H == 16))
        return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": unsupported (dtype, d, H)");
    return GT_OK;
}

template <typename T, int D, int H>
gt_status run_dense_fwd(int64_t n, const void* Q, const void* K, const void* V, float scale, void* O, float* LSE,
                        hipStream_t s) {
    if (n == 0) return GT_OK;
    if constexpr (sizeof(T) == 2)
        return full_fwd_bf16<D>(n, H, static_cast<const T*>(Q), static_cast<const T*>(K), static_cast<const T*>(V),
                                scale * kLog2e, static_cast<T*>(O), LSE, s);
    return full_fwd<T, D, H>(n, static_cast<const T*>(Q), static_cast<const T*>(K), static_cast<const T*>(V),
                             scale * kLog2e, static_cast<T*>(O), LSE, s);
}

template <typename T, int D, int H>
gt_status run_dense_bwd(int64_t n, const void* Q, const void* K, const void* V, const void* O, const void* dO,
                        const float* LSE, float scale, void* dQ, void* dK, void* dV, void* ws, hipStream_t s) {
    if (n == 0) return GT_OK;
    Ws w(ws);
    float* Dv = w.take<float>(size_t(n) * H);
    if constexpr (sizeof(T) == 2)
        return full_bwd_bf16<D>(n, H, static_cast<const T*>(Q), static_cast<const T*>(K), static_cast<const T*>(V),
                                static_cast<const T*>(O), static_cast<const T*>(dO), LSE, scale * kLog2e, scale,
                                static_cast<T*>(dQ), static_cast<T*>(dK), static_cast<T*>(dV), Dv, s);
    return full_bwd<T, D, H>(n, static_cast<const T*>(Q), static_cast<const T*>(K), static_cast<const T*>(V),
                             static_cast<const T*>(O), static_cast<const T*>(dO), LSE, scale * kLog2e, scale,
                             static_cast<T*>(dQ), static_cast<T*>(dK), static_cast<T*>(dV), Dv, s);
}

}  // namespace

extern "C" gt_status gt_dense_attn_fwd(int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q, const void* K,
                                       const void* V, float scale, void* O, float* LSE, hipStream_t stream) {
    gt_status st = dense_check("gt_dense_attn_fwd", n, H, d, dt, Q, K, V);
    if (st != GT_OK) return st;
    if (n > 0 && (!O || !LSE)) return fail(GT_ERR_INVALID_ARG, "gt_dense_attn_fwd: null pointer");
    return GT_DISPATCH_ATTN(dt, d, H, run_dense_fwd, n, Q, K, V, scale, O, LSE, stream);
}

extern "C" size_t gt_dense_attn_bwd_workspace_size(int64_t n, int32_t H, int32_t, gt_dtype) {
    Ws w(nullptr);
    w.take<float>(size_t(n > 0 ? n : 1) * size_t(H > 0 ? H : 1));
    return w.size();
}

extern "C" gt_status gt_dense_attn_bwd(int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q, const void* K,
                                       const void* V, const void* O, const void* dO, const float* LSE, float scale,
                                       void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream) {
    gt_status st = dense_check("gt_dense_attn_bwd", n, H, d, dt, Q, K, V);
    if (st != GT_OK) return st;
    if (n > 0 && (!O || !dO || !LSE || !dQ || !dK || !dV || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_dense_attn_bwd: null pointer");
    if (ws_bytes < gt_dense_attn_bwd_workspace_size(n, H, d, dt))
        return fail(GT_ERR_WORKSPACE, "gt_dense_attn_bwd: workspace too small");
    return GT_DISPATCH_ATTN(dt, d, H, run_dense_bwd, n, Q, K, V, O, dO, LSE, scale, dQ, dK, dV, ws, stream);
}
