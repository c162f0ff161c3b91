// Full softmax attention (§2.1 Eq. (1)): the interleaved fully-connected layer
// of §3.2.  bf16 features run the streaming kernels of dense_mfma.hip; fp32
// features run the matrix-core tile kernels with every pair attended.
#include <atomic>

#include "tile_attn.h"

using namespace gt;

namespace {

// Scratch of gt_dense_attn_bwd_noalloc, for callers that cannot allocate: the
// backward's row statistic D (fp32 [n, H]) in a device array of the library's
// own, one copy per GPU, held until the process ends.  On the host the name
// `scratch` is only a stand-in for the device array: host code takes the
// array's device address once per device with hipGetSymbolAddress and passes
// that address, never the name, to the kernels.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];

// Device address of `scratch` on the current device, looked up on the first
// call there.  The stream must belong to the current device.
gt_status scratch_address(const char* who, hipStream_t stream, void** out) {
    int dev = -1;
    GT_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": device index above 63");
    if (stream) {
        hipDevice_t sdev = -1;
        GT_HIP(hipStreamGetDevice(stream, &sdev));
        if (sdev != dev)
            return fail(GT_ERR_INVALID_ARG, std::string(who) + ": the stream belongs to another device than the "
                                                               "current one");
    }
    void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
    if (!p) {
        GT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(GT_ERR_HIP, std::string(who) + ": no device address for the scratch array");
        g_scratch_addr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return GT_OK;
}

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

extern "C" size_t gt_dense_attn_bwd_noalloc_max_bytes(void) { return kNoAllocScratchBytes; }

extern "C" gt_status gt_dense_attn_bwd_noalloc(int64_t n, int32_t H, int32_t d, gt_dtype dt, const void* Q,
                                               const void* K, const void* V, const void* O, const void* dO,
                                               const float* LSE, float scale, void* dQ, void* dK, void* dV,
                                               hipStream_t stream) {
    const char* who = "gt_dense_attn_bwd_noalloc";
    gt_status st = dense_check(who, n, H, d, dt, Q, K, V);
    if (st != GT_OK) return st;
    if (n > 0 && (!O || !dO || !LSE || !dQ || !dK || !dV))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null pointer");
    if (gt_dense_attn_bwd_workspace_size(n, H, d, dt) > kNoAllocScratchBytes)
        return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": n * H * 4 bytes of scratch exceed its 64 MiB "
                                                           "(n * H above 16,777,216); use gt_dense_attn_bwd");
    if (n == 0) return GT_OK;
    void* ws = nullptr;
    if ((st = scratch_address(who, stream, &ws)) != GT_OK) return st;
    return GT_DISPATCH_ATTN(dt, d, H, run_dense_bwd, n, Q, K, V, O, dO, LSE, scale, dQ, dK, dV, ws, stream);
}
