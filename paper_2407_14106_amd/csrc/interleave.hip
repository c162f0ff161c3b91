// The interleave decision of Dual-interleaved Attention (§3.2): the quick
// checks of the three conditions under which the topology-induced pattern is
// used alone, otherwise a fully connected layer is interleaved.
//   C1 (every node attends to itself): rows without their self-loop, exact.
//   C2 (a Hamiltonian path): Dirac's condition on the minimum degree without
//      self-loops, 2 min_deg >= n for n >= 3 (n <= 1 holds, n = 2 needs the
//      edge); anything else is not confirmed.
//   C3 (everything reachable within L layers): breadth-first search from node
//      0 cut at depth L + 1; 2 ecc <= L confirms, depth L + 1 or an unreached
//      node refutes, otherwise a second search from the smallest-id node at
//      the last depth (double sweep) refutes or leaves it undetermined.
// The searches are level-synchronous: one launch per depth, a wavefront per
// node whose lanes stride over the frontier node's edges, claims by CAS (the
// depths are unique, so the result does not depend on the order of claims).
#include "prim.h"

namespace gt {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

// stats[0] += rows without a self-loop; stats[1] = min over rows of the degree without the self-loop
__global__ __launch_bounds__(kThreads) void k_self_degree(int64_t n, const int64_t* __restrict__ rowptr,
                                                          const int32_t* __restrict__ col,
                                                          unsigned long long* stats) {
    __shared__ unsigned long long s_miss[kWavesPerBlock];
    __shared__ unsigned long long s_min[kWavesPerBlock];
    unsigned long long miss = 0, mn = ~0ull;
    for (int64_t i = blockIdx.x * int64_t(kThreads) + threadIdx.x; i < n; i += int64_t(gridDim.x) * kThreads) {
        int64_t lo = rowptr[i], hi = rowptr[i + 1];
        const int64_t deg = hi - lo;
        while (lo < hi) {  // first position with col >= i
            const int64_t mid = (lo + hi) >> 1;
            if (col[mid] < i) lo = mid + 1;
            else hi = mid;
        }
        const bool has = lo < rowptr[i + 1] && col[lo] == i;
        miss += has ? 0 : 1;
        const unsigned long long d = static_cast<unsigned long long>(deg - (has ? 1 : 0));
        mn = d < mn ? d : mn;
    }
    miss = wave_sum(miss);
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long w = __shfl_xor(mn, o, kWave);
        mn = w < mn ? w : mn;
    }
    const int wv = threadIdx.x / kWave;
    if (lane_id() == 0) {
        s_miss[wv] = miss;
        s_min[wv] = mn;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long a = 0, b = ~0ull;
        for (int x = 0; x < kWavesPerBlock; ++x) {
            a += s_miss[x];
            b = s_min[x] < b ? s_min[x] : b;
        }
        if (a) atomicAdd(&stats[0], a);
        atomicMin(&stats[1], b);
    }
}

// One depth of the search: every node at depth d claims its unvisited out-neighbours for depth d + 1.
__global__ __launch_bounds__(kThreads) void k_bfs_step(int64_t n, const int64_t* __restrict__ rowptr,
                                                       const int32_t* __restrict__ col, int32_t* levels, int32_t d,
                                                       unsigned int* claimed) {
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * kWavesPerBlock;
    unsigned int mine = 0;
    for (int64_t v = int64_t(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave; v < n; v += waves) {
        if (levels[v] != d) continue;
        const int64_t a = rowptr[v], b = rowptr[v + 1];
        for (int64_t e = a + lane; e < b; e += kWave) {
            const int32_t u = col[e];
            if (levels[u] == -1 && atomicCAS(&levels[u], -1, d + 1) == -1) ++mine;
        }
    }
    mine = wave_sum(mine);
    if (lane == 0 && mine) atomicAdd(claimed, mine);
}

__global__ void k_first_at(int64_t n, const int32_t* __restrict__ levels, int32_t d, unsigned int* out) {
    for (int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; v < n; v += int64_t(gridDim.x) * blockDim.x)
        if (levels[v] == d) atomicMin(out, static_cast<unsigned int>(v));
}

__global__ void k_set_one(int32_t* p, int64_t at, int32_t value) { p[at] = value; }

struct IlWs {
    uint32_t* flags;
    unsigned long long* stats;
    unsigned int* claimed;
    unsigned int* far;
    int32_t* lev1;
    int32_t* lev2;
};

IlWs carve(Ws& ws, int64_t n) {
    const int64_t n1 = n > 0 ? n : 1;
    IlWs w;
    w.flags = ws.take<uint32_t>(1);
    w.stats = ws.take<unsigned long long>(2);
    w.claimed = ws.take<unsigned int>(1);
    w.far = ws.take<unsigned int>(1);
    w.lev1 = ws.take<int32_t>(n1);
    w.lev2 = ws.take<int32_t>(n1);
    return w;
}

// Depth-capped search from root into lev: returns the deepest depth reached and the nodes reached.
gt_status bfs(int64_t n, const int64_t* rowptr, const int32_t* col, int64_t root, int32_t cap, int32_t* lev,
              unsigned int* claimed, int32_t* depth, int64_t* reached, hipStream_t s) {
    gt_status st;
    if ((st = fill_u32(reinterpret_cast<uint32_t*>(lev), n, 0xFFFFFFFFu, s)) != GT_OK) return st;
    k_set_one<<<1, 1, 0, s>>>(lev, root, 0);
    GT_LAUNCH_CHECK("bfs_root");
    *depth = 0;
    *reached = 1;
    const unsigned g = grid_for(n, kWavesPerBlock, 1 << 16);
    for (int32_t d = 0; d < cap; ++d) {
        if ((st = fill_u32(claimed, 1, 0u, s)) != GT_OK) return st;
        k_bfs_step<<<g, kThreads, 0, s>>>(n, rowptr, col, lev, d, claimed);
        GT_LAUNCH_CHECK("bfs_step");
        unsigned int got = 0;
        GT_HIP(hipMemcpyAsync(&got, claimed, 4, hipMemcpyDeviceToHost, s));
        GT_HIP(hipStreamSynchronize(s));
        if (got == 0) break;
        *depth = d + 1;
        *reached += got;
    }
    return GT_OK;
}

}  // namespace
}  // namespace gt

using namespace gt;

extern "C" size_t gt_interleave_workspace_size(int64_t n) {
    if (n < 0) return 0;
    Ws ws(nullptr);
    carve(ws, n);
    return ws.size();
}

extern "C" gt_status gt_interleave_check(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                                         int32_t L, gt_interleave_report* report, int32_t* levels, void* ws_ptr,
                                         size_t ws_bytes, hipStream_t stream) {
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << 32))
        return fail(GT_ERR_INVALID_ARG, "gt_interleave_check: n or nnz out of range");
    if (L < 0 || L >= (1 << 30)) return fail(GT_ERR_INVALID_ARG, "gt_interleave_check: L out of range");
    if (!rowptr || !report || (nnz > 0 && !col) || !ws_ptr)
        return fail(GT_ERR_INVALID_ARG, "gt_interleave_check: null pointer");
    if (ws_bytes < gt_interleave_workspace_size(n))
        return fail(GT_ERR_WORKSPACE, "gt_interleave_check: workspace too small");
    Ws ws(ws_ptr);
    IlWs w = carve(ws, n);
    gt_interleave_report r{};
    r.n = n;
    r.ecc_far = -1;
    gt_status st;
    if (n == 0) {
        r.c1 = r.c2 = r.c3 = r.use_sparse = 1;
        *report = r;
        return GT_OK;
    }
    if ((st = launch_validate_csr(n, nnz, rowptr, col, w.flags, stream)) != GT_OK) return st;
    if ((st = read_validation(w.flags, stream)) != GT_OK) return st;
    // C1 and the minimum degree
    if ((st = fill_u32(reinterpret_cast<uint32_t*>(w.stats), 2, 0u, stream)) != GT_OK) return st;
    if ((st = fill_u32(reinterpret_cast<uint32_t*>(w.stats) + 2, 2, 0xFFFFFFFFu, stream)) != GT_OK) return st;
    k_self_degree<<<grid_for(n, kThreads, 2048), kThreads, 0, stream>>>(n, rowptr, col, w.stats);
    GT_LAUNCH_CHECK("interleave_self_degree");
    unsigned long long h[2];
    GT_HIP(hipMemcpyAsync(h, w.stats, sizeof(h), hipMemcpyDeviceToHost, stream));
    GT_HIP(hipStreamSynchronize(stream));
    r.missing_self_loops = int64_t(h[0]);
    r.min_degree = int64_t(h[1]);
    r.c1 = r.missing_self_loops == 0 ? 1 : 0;
    if (n <= 1) r.c2 = 1;
    else if (n == 2) r.c2 = r.min_degree >= 1 ? 1 : 0;
    else r.c2 = 2 * r.min_degree >= n ? 1 : 0;
    // C3: depth-capped search from node 0, then the double sweep
    int32_t* lev = levels ? levels : w.lev1;
    int32_t ecc = 0;
    int64_t reached = 0;
    if ((st = bfs(n, rowptr, col, 0, L + 1, lev, w.claimed, &ecc, &reached, stream)) != GT_OK) return st;
    r.ecc_root = ecc;
    r.reached = reached;
    if (ecc > L || reached < n) {
        r.c3 = 0;
    } else if (2 * int64_t(ecc) <= L) {
        r.c3 = 1;
    } else {
        if ((st = fill_u32(w.far, 1, 0xFFFFFFFFu, stream)) != GT_OK) return st;
        k_first_at<<<grid_for(n, 256, 4096), 256, 0, stream>>>(n, lev, ecc, w.far);
        GT_LAUNCH_CHECK("interleave_far");
        unsigned int far = 0;
        GT_HIP(hipMemcpyAsync(&far, w.far, 4, hipMemcpyDeviceToHost, stream));
        GT_HIP(hipStreamSynchronize(stream));
        int32_t ecc2 = 0;
        int64_t reached2 = 0;
        if ((st = bfs(n, rowptr, col, int64_t(far), L + 1, w.lev2, w.claimed, &ecc2, &reached2, stream)) != GT_OK)
            return st;
        r.ecc_far = ecc2;
        r.c3 = (ecc2 > L || reached2 < n) ? 0 : -1;
    }
    r.use_sparse = (r.c1 == 1 && r.c2 == 1 && r.c3 == 1) ? 1 : 0;
    *report = r;
    return GT_OK;
}
