// The paper's lossy Elastic Computation Reformation (§3.4, cluster sparsity and
// transfer strategy), as an opt-in rewrite of the graph.  The clustered layout
// is cut into k x k clusters of edge c = ceil(n / k); a cluster whose density
// cnt / area is below the threshold num / den has its edges (self-loops
// excepted) replaced by m = ceil(moved / d_b^2) full d_b x d_b sub-blocks, put
// at the blocks of the cluster (cut from its corner) that held the most of its
// moved edges, ties to the smaller (block row, block column).  The result E'
// is a CSR; the exact attention path then runs on it.
//
// Stages, all on the device (five counts are read back to size the next one):
//  1. per-cluster edge and self-loop counts (LDS histograms, k <= 64);
//  2. transfer flags and sub-block counts m per cluster, the density test as
//     an exact 128-bit comparison cnt * den < num * area;
//  3. the moved edges' block keys (cluster, block row, block column),
//     compacted in CSR order (per-row counts, scan, ballot ranks), radix-sorted;
//  4. run lengths of equal keys = edges per block; the blocks re-sorted by
//     (cluster, d_b^2 - count, block) and the first m of each cluster chosen;
//  5. candidate edges, every cell of a chosen block plus every kept edge, as
//     packed (row, column) keys, radix-sorted and made unique into the CSR.
#include "prim.h"

namespace gt {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;
constexpr int kMaxK = 64;

struct Geom {
    int64_t n;
    int64_t c;   // cluster edge
    int64_t nb;  // blocks per cluster edge, ceil(c / d_b)
    int32_t k;
    int32_t db;
    int kb;      // bits of a block index inside a cluster (nb^2 values)
    int cb;      // bits of d_b^2 - count (0 .. d_b^2)
    int nbits;   // bits of a node id
};

__device__ __forceinline__ int64_t rows_of(const Geom& g, int64_t I) {
    const int64_t r = g.n - I * g.c;
    return r < 0 ? 0 : (r < g.c ? r : g.c);
}

// ---- 1. counts
__global__ __launch_bounds__(kThreads) void k_cluster_counts(Geom g, const int64_t* __restrict__ rowptr,
                                                             const int32_t* __restrict__ col, uint32_t* cnt,
                                                             uint32_t* loops) {
    __shared__ uint32_t h[kMaxK * kMaxK];
    __shared__ uint32_t hl[kMaxK];
    const int kk = g.k * g.k;
    for (int x = threadIdx.x; x < kk; x += kThreads) h[x] = 0;
    for (int x = threadIdx.x; x < g.k; x += kThreads) hl[x] = 0;
    __syncthreads();
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * kWavesPerBlock;
    for (int64_t i = int64_t(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave; i < g.n; i += waves) {
        const int64_t a = rowptr[i], b = rowptr[i + 1];
        const int I = int(i / g.c);
        for (int64_t e = a + lane; e < b; e += kWave) {
            const int64_t j = col[e];
            atomicAdd(&h[I * g.k + int(j / g.c)], 1u);
            if (j == i) atomicAdd(&hl[I], 1u);
        }
    }
    __syncthreads();
    for (int x = threadIdx.x; x < kk; x += kThreads)
        if (h[x]) atomicAdd(&cnt[x], h[x]);
    for (int x = threadIdx.x; x < g.k; x += kThreads)
        if (hl[x]) atomicAdd(&loops[x], hl[x]);
}

// ---- 2. transfer decision: cnt >= 1 and cnt * den < num * area (exact)
__global__ void k_transfer(Geom g, const uint32_t* __restrict__ cnt, const uint32_t* __restrict__ loops,
                           uint64_t num, uint64_t den, uint32_t* flag, uint32_t* m) {
    const int x = blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= g.k * g.k) return;
    const int I = x / g.k, J = x % g.k;
    const uint64_t area = uint64_t(rows_of(g, I)) * uint64_t(rows_of(g, J));
    const uint64_t c = cnt[x];
    const bool t = c >= 1 && (unsigned __int128)c * den < (unsigned __int128)num * area;
    const uint64_t moved = c - (I == J ? loops[I] : 0u);
    const uint64_t cells = uint64_t(g.db) * uint64_t(g.db);
    flag[x] = t ? 1u : 0u;
    m[x] = t ? uint32_t((moved + cells - 1) / cells) : 0u;
}

__device__ __forceinline__ bool is_moved(const Geom& g, const uint32_t* flag, int64_t i, int64_t j) {
    return i != j && flag[(i / g.c) * g.k + j / g.c];
}

// ---- 3. moved edges: per-row counts, then keys in CSR order
__global__ __launch_bounds__(kThreads) void k_moved_per_row(Geom g, const int64_t* __restrict__ rowptr,
                                                            const int32_t* __restrict__ col,
                                                            const uint32_t* __restrict__ flag, int32_t* rowcnt) {
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * kWavesPerBlock;
    for (int64_t i = int64_t(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave; i < g.n; i += waves) {
        const int64_t a = rowptr[i], b = rowptr[i + 1];
        int c = 0;
        for (int64_t e = a + lane; e < b; e += kWave) c += is_moved(g, flag, i, col[e]) ? 1 : 0;
        c = wave_sum(c);
        if (lane == 0) rowcnt[i] = c;
    }
}

// Writes, for each row, the moved edges (kMoved) or the kept ones (!kMoved) in CSR order starting at
// base + off(i), off(i) = moved_off[i] for moved edges and rowptr[i] - moved_off[i] for kept ones.
template <bool kMoved>
__global__ __launch_bounds__(kThreads) void k_emit_edges(Geom g, const int64_t* __restrict__ rowptr,
                                                         const int32_t* __restrict__ col,
                                                         const uint32_t* __restrict__ flag,
                                                         const int64_t* __restrict__ moved_off, int64_t base,
                                                         uint64_t* __restrict__ out) {
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * kWavesPerBlock;
    for (int64_t i = int64_t(blockIdx.x) * kWavesPerBlock + threadIdx.x / kWave; i < g.n; i += waves) {
        const int64_t a = rowptr[i], b = rowptr[i + 1];
        int64_t pos = base + (kMoved ? moved_off[i] : a - moved_off[i]);
        const int64_t I = i / g.c;
        for (int64_t e0 = a; e0 < b; e0 += kWave) {
            const int64_t e = e0 + lane;
            const bool live = e < b;
            const int64_t j = live ? col[e] : 0;
            const bool pick = live && (is_moved(g, flag, i, j) == kMoved);
            const uint64_t bal = ballot(pick);
            if (pick) {
                const int64_t at = pos + __popcll(bal & lanemask_lt());
                if (kMoved) {
                    const int64_t J = j / g.c;
                    const uint64_t blk = uint64_t((i - I * g.c) / g.db) * uint64_t(g.nb) + uint64_t((j - J * g.c) / g.db);
                    out[at] = (uint64_t(I * g.k + J) << g.kb) | blk;
                } else {
                    out[at] = (uint64_t(i) << g.nbits) | uint64_t(j);
                }
            }
            pos += __popcll(bal);
        }
    }
}

// ---- run heads of a sorted key array
__global__ void k_heads(const uint64_t* __restrict__ keys, int64_t len, uint32_t* head) {
    for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < len; p += int64_t(gridDim.x) * blockDim.x)
        head[p] = (p == 0 || keys[p] != keys[p - 1]) ? 1u : 0u;
}

// ---- 4. blocks: (cluster, d_b^2 - count, block) selection keys
__global__ void k_block_keys(Geom g, const uint64_t* __restrict__ keys, int64_t len,
                             const uint32_t* __restrict__ head, const int64_t* __restrict__ hoff, int64_t U,
                             int64_t* __restrict__ ustart) {
    for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < len; p += int64_t(gridDim.x) * blockDim.x)
        if (head[p]) ustart[hoff[p]] = p;
    if (blockIdx.x == 0 && threadIdx.x == 0) ustart[U] = len;
}

__global__ void k_select_keys(Geom g, const uint64_t* __restrict__ keys, const int64_t* __restrict__ ustart, int64_t U,
                              uint64_t* __restrict__ key2) {
    const uint64_t cells = uint64_t(g.db) * uint64_t(g.db);
    const uint64_t blk_mask = (uint64_t(1) << g.kb) - 1;
    for (int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; q < U; q += int64_t(gridDim.x) * blockDim.x) {
        const uint64_t key = keys[ustart[q]];
        const uint64_t count = uint64_t(ustart[q + 1] - ustart[q]);
        const uint64_t cid = key >> g.kb;
        key2[q] = (cid << (g.cb + g.kb)) | ((cells - count) << g.kb) | (key & blk_mask);
    }
}

__global__ void k_cluster_first(Geom g, const uint64_t* __restrict__ key2, int64_t U, int64_t* __restrict__ first) {
    const int sh = g.cb + g.kb;
    for (int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; q < U; q += int64_t(gridDim.x) * blockDim.x) {
        const uint64_t cid = key2[q] >> sh;
        if (q == 0 || (key2[q - 1] >> sh) != cid) first[cid] = q;
    }
}

// selected blocks: sel[q] = 1 for the first m of their cluster; cells[q] = clipped cell count (0 if not)
__global__ void k_select(Geom g, const uint64_t* __restrict__ key2, int64_t U, const int64_t* __restrict__ first,
                         const uint32_t* __restrict__ m, int64_t* __restrict__ cells) {
    const int sh = g.cb + g.kb;
    const uint64_t blk_mask = (uint64_t(1) << g.kb) - 1;
    for (int64_t q = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; q < U; q += int64_t(gridDim.x) * blockDim.x) {
        const uint64_t cid = key2[q] >> sh;
        int64_t nc = 0;
        if (q - first[cid] < int64_t(m[cid])) {
            const int64_t I = int64_t(cid) / g.k, J = int64_t(cid) % g.k;
            const uint64_t blk = key2[q] & blk_mask;
            const int64_t a = int64_t(blk / uint64_t(g.nb)), b = int64_t(blk % uint64_t(g.nb));
            const int64_t hr = rows_of(g, I) - a * g.db, hc = rows_of(g, J) - b * g.db;
            nc = (hr < g.db ? hr : g.db) * (hc < g.db ? hc : g.db);
        }
        cells[q] = nc;
    }
}

// ---- 5. every cell of the chosen blocks: one workgroup per block (grid-stride)
__global__ __launch_bounds__(kThreads) void k_emit_cells(Geom g, const uint64_t* __restrict__ key2, int64_t U,
                                                         const int64_t* __restrict__ cells,
                                                         const int64_t* __restrict__ coff,
                                                         uint64_t* __restrict__ out) {
    const int sh = g.cb + g.kb;
    const uint64_t blk_mask = (uint64_t(1) << g.kb) - 1;
    for (int64_t q = blockIdx.x; q < U; q += gridDim.x) {
        const int64_t nc = cells[q];
        if (nc == 0) continue;
        const uint64_t cid = key2[q] >> sh;
        const int64_t I = int64_t(cid) / g.k, J = int64_t(cid) % g.k;
        const uint64_t blk = key2[q] & blk_mask;
        const int64_t r0 = I * g.c + int64_t(blk / uint64_t(g.nb)) * g.db;
        const int64_t c0 = J * g.c + int64_t(blk % uint64_t(g.nb)) * g.db;
        const int64_t hc = rows_of(g, J) - (c0 - J * g.c);
        const int64_t w = hc < g.db ? hc : g.db;
        const int64_t base = coff[q];
        for (int64_t t = threadIdx.x; t < nc; t += kThreads) {
            const int64_t r = r0 + t / w, cc = c0 + t % w;
            out[base + t] = (uint64_t(r) << g.nbits) | uint64_t(cc);
        }
    }
}

// ---- output CSR from the sorted candidates
__global__ void k_emit_cols(const uint64_t* __restrict__ keys, int64_t len, const uint32_t* __restrict__ head,
                            const int64_t* __restrict__ hoff, uint64_t mask, int32_t* __restrict__ col_out) {
    for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < len; p += int64_t(gridDim.x) * blockDim.x)
        if (head[p]) col_out[hoff[p]] = int32_t(keys[p] & mask);
}

// rowptr_out[r] = the first unique position whose row is >= r (rows between two heads' rows are empty).
__global__ void k_row_bounds(const uint64_t* __restrict__ keys, int64_t len, const uint32_t* __restrict__ head,
                             const int64_t* __restrict__ hoff, int nbits, int64_t n, int64_t* __restrict__ rowptr_out) {
    for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p <= len; p += int64_t(gridDim.x) * blockDim.x) {
        if (p < len && !head[p]) continue;
        const int64_t prev = p == 0 ? -1 : int64_t(keys[p - 1] >> nbits);
        const int64_t r = p == len ? n : int64_t(keys[p] >> nbits);
        for (int64_t rr = prev + 1; rr <= r; ++rr) rowptr_out[rr] = hoff[p];
    }
}

struct EcrWs {
    uint32_t* flags;  // validation
    uint32_t* cnt;
    uint32_t* loops;
    uint32_t* transfer;
    uint32_t* m;
    int64_t* first;
    int32_t* rowcnt;
    int64_t* moff;
    uint64_t* keys;    // moved keys, then candidates
    uint64_t* key2;
    int64_t* ustart;
    int64_t* cells;
    int64_t* coff;
    uint32_t* head;
    int64_t* hoff;
    ScanTmp scan;
    SortTmp sort;
};

int64_t max_candidates(int64_t nnz, int32_t k, int32_t db) {
    return nnz + int64_t(k) * k * (int64_t(db) * db - 1);
}

EcrWs carve(Ws& ws, int64_t n, int64_t nnz, int32_t k, int32_t db) {
    EcrWs w;
    const int64_t n1 = n > 0 ? n : 1, e1 = nnz > 0 ? nnz : 1;
    const int64_t cap = max_candidates(e1, k, db);
    const int64_t kk = int64_t(k) * k;
    w.flags = ws.take<uint32_t>(1);
    w.cnt = ws.take<uint32_t>(kk);
    w.loops = ws.take<uint32_t>(k);
    w.transfer = ws.take<uint32_t>(kk);
    w.m = ws.take<uint32_t>(kk);
    w.first = ws.take<int64_t>(kk);
    w.rowcnt = ws.take<int32_t>(n1);
    w.moff = ws.take<int64_t>(n1 + 1);
    w.keys = ws.take<uint64_t>(cap);
    w.key2 = ws.take<uint64_t>(e1);
    w.ustart = ws.take<int64_t>(e1 + 1);
    w.cells = ws.take<int64_t>(e1);
    w.coff = ws.take<int64_t>(e1 + 1);
    w.head = ws.take<uint32_t>(cap);
    w.hoff = ws.take<int64_t>(cap + 1);
    w.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(cap + 1)));
    w.sort = sort_tmp(ws, cap, 8, false);
    return w;
}

gt_status read_i64(const int64_t* src, int64_t* dst, hipStream_t s) {
    GT_HIP(hipMemcpyAsync(dst, src, 8, hipMemcpyDeviceToHost, s));
    GT_HIP(hipStreamSynchronize(s));
    return GT_OK;
}

bool geometry(int64_t n, int32_t k, int32_t db, Geom& g) {
    g.n = n;
    g.k = k;
    g.db = db;
    g.c = n > 0 ? cdiv(n, k) : 1;
    g.nb = cdiv(g.c, db);
    g.kb = bits_for(g.nb * g.nb);
    g.cb = bits_for(int64_t(db) * db + 1);
    g.nbits = bits_for(n > 1 ? n : 2);
    const int cid_bits = bits_for(int64_t(k) * k > 1 ? int64_t(k) * k : 2);
    return cid_bits + g.cb + g.kb <= 64 && cid_bits + g.kb <= 64 && 2 * g.nbits <= 64;
}

}  // namespace
}  // namespace gt

using namespace gt;

extern "C" int64_t gt_ecr_max_nnz(int64_t nnz, int32_t k, int32_t d_b) {
    if (nnz < 0 || k < 1 || k > kMaxK || d_b < 1 || d_b > 256) return -1;
    return max_candidates(nnz, k, d_b);
}

extern "C" size_t gt_ecr_workspace_size(int64_t n, int64_t nnz, int32_t k, int32_t d_b) {
    if (n < 0 || nnz < 0 || k < 1 || k > kMaxK || d_b < 1 || d_b > 256) return 0;
    Ws ws(nullptr);
    carve(ws, n, nnz, k, d_b);
    return ws.size();
}

extern "C" gt_status gt_ecr_compact(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t k,
                                    int32_t d_b, uint64_t num, uint64_t den, int64_t* rowptr_out, int32_t* col_out,
                                    int64_t cap, int64_t* nnz_out, int32_t* n_transferred, void* ws_ptr,
                                    size_t ws_bytes, hipStream_t stream) {
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << 31))
        return fail(GT_ERR_INVALID_ARG, "gt_ecr_compact: n or nnz out of range");
    if (k < 1 || k > kMaxK || d_b < 1 || d_b > 256)
        return fail(GT_ERR_UNSUPPORTED, "gt_ecr_compact: k must be in [1, 64] and d_b in [1, 256]");
    if (den == 0) return fail(GT_ERR_INVALID_ARG, "gt_ecr_compact: den must be positive");
    if (!rowptr || !rowptr_out || !nnz_out || (nnz > 0 && !col) || !ws_ptr)
        return fail(GT_ERR_INVALID_ARG, "gt_ecr_compact: null pointer");
    const int64_t need = max_candidates(nnz, k, d_b);
    if (cap < need || (need > 0 && !col_out))
        return fail(GT_ERR_INVALID_ARG, "gt_ecr_compact: col_out capacity below gt_ecr_max_nnz");
    if (need >= (int64_t(1) << 32)) return fail(GT_ERR_UNSUPPORTED, "gt_ecr_compact: k^2 d_b^2 + nnz must be < 2^32");
    if (ws_bytes < gt_ecr_workspace_size(n, nnz, k, d_b))
        return fail(GT_ERR_WORKSPACE, "gt_ecr_compact: workspace too small");
    Geom g;
    if (!geometry(n, k, d_b, g)) return fail(GT_ERR_UNSUPPORTED, "gt_ecr_compact: keys do not fit 64 bits");
    Ws ws(ws_ptr);
    EcrWs w = carve(ws, n, nnz, k, d_b);
    gt_status st;
    *nnz_out = 0;
    if (n_transferred) *n_transferred = 0;
    if (n == 0) return fill_i64(rowptr_out, 1, 0, stream);
    if ((st = launch_validate_csr(n, nnz, rowptr, col, w.flags, stream)) != GT_OK) return st;
    if ((st = read_validation(w.flags, stream)) != GT_OK) return st;
    const int kk = k * k;
    // 1-2: cluster counts, decisions
    if ((st = fill_u32(w.cnt, kk, 0u, stream)) != GT_OK) return st;
    if ((st = fill_u32(w.loops, k, 0u, stream)) != GT_OK) return st;
    const unsigned gw = grid_for(n, kWavesPerBlock, 4096);
    k_cluster_counts<<<gw, kThreads, 0, stream>>>(g, rowptr, col, w.cnt, w.loops);
    GT_LAUNCH_CHECK("ecr_cluster_counts");
    k_transfer<<<grid_for(kk, 256), 256, 0, stream>>>(g, w.cnt, w.loops, num, den, w.transfer, w.m);
    GT_LAUNCH_CHECK("ecr_transfer");
    if (n_transferred) {
        uint32_t h[kMaxK * kMaxK];
        GT_HIP(hipMemcpyAsync(h, w.transfer, size_t(kk) * 4, hipMemcpyDeviceToHost, stream));
        GT_HIP(hipStreamSynchronize(stream));
        int32_t t = 0;
        for (int x = 0; x < kk; ++x) t += h[x] ? 1 : 0;
        *n_transferred = t;
    }
    // 3: moved edges
    const unsigned gr = grid_for(n, kWavesPerBlock, 65536);
    k_moved_per_row<<<gr, kThreads, 0, stream>>>(g, rowptr, col, w.transfer, w.rowcnt);
    GT_LAUNCH_CHECK("ecr_moved_per_row");
    if ((st = exclusive_scan_i32(w.rowcnt, n, w.moff, w.scan, stream)) != GT_OK) return st;
    int64_t M = 0;
    if ((st = read_i64(w.moff + n, &M, stream)) != GT_OK) return st;
    int64_t X = 0, U = 0;
    if (M > 0) {
        k_emit_edges<true><<<gr, kThreads, 0, stream>>>(g, rowptr, col, w.transfer, w.moff, 0, w.keys);
        GT_LAUNCH_CHECK("ecr_moved_keys");
        const int cid_bits = bits_for(int64_t(kk) > 1 ? int64_t(kk) : 2);
        if ((st = radix_sort_u64(w.keys, nullptr, M, cid_bits + g.kb, w.sort, stream)) != GT_OK) return st;
        // 4: blocks and their counts, selection
        const unsigned ge = grid_for(M, 256, 65536);
        k_heads<<<ge, 256, 0, stream>>>(w.keys, M, w.head);
        GT_LAUNCH_CHECK("ecr_block_heads");
        if ((st = exclusive_scan_u32(w.head, M, w.hoff, w.scan, stream)) != GT_OK) return st;
        if ((st = read_i64(w.hoff + M, &U, stream)) != GT_OK) return st;
        k_block_keys<<<ge, 256, 0, stream>>>(g, w.keys, M, w.head, w.hoff, U, w.ustart);
        GT_LAUNCH_CHECK("ecr_block_starts");
        const unsigned gu = grid_for(U, 256, 65536);
        k_select_keys<<<gu, 256, 0, stream>>>(g, w.keys, w.ustart, U, w.key2);
        GT_LAUNCH_CHECK("ecr_select_keys");
        if ((st = radix_sort_u64(w.key2, nullptr, U, cid_bits + g.cb + g.kb, w.sort, stream)) != GT_OK) return st;
        k_cluster_first<<<gu, 256, 0, stream>>>(g, w.key2, U, w.first);
        GT_LAUNCH_CHECK("ecr_cluster_first");
        k_select<<<gu, 256, 0, stream>>>(g, w.key2, U, w.first, w.m, w.cells);
        GT_LAUNCH_CHECK("ecr_select");
        if ((st = exclusive_scan_i64(w.cells, U, w.coff, w.scan, stream)) != GT_OK) return st;
        if ((st = read_i64(w.coff + U, &X, stream)) != GT_OK) return st;
    }
    // 5: candidates = chosen cells + kept edges
    const int64_t total = X + (nnz - M);
    if (total > need) return fail(GT_ERR_HIP, "gt_ecr_compact: internal count exceeds its bound");
    if (X > 0) {
        k_emit_cells<<<grid_for(U, 1, 65536), kThreads, 0, stream>>>(g, w.key2, U, w.cells, w.coff, w.keys);
        GT_LAUNCH_CHECK("ecr_emit_cells");
    }
    if (nnz - M > 0) {
        k_emit_edges<false><<<gr, kThreads, 0, stream>>>(g, rowptr, col, w.transfer, w.moff, X, w.keys);
        GT_LAUNCH_CHECK("ecr_kept_keys");
    }
    int64_t out = 0;
    if (total > 0) {
        if ((st = radix_sort_u64(w.keys, nullptr, total, 2 * g.nbits, w.sort, stream)) != GT_OK) return st;
        const unsigned gt_ = grid_for(total, 256, 65536);
        k_heads<<<gt_, 256, 0, stream>>>(w.keys, total, w.head);
        GT_LAUNCH_CHECK("ecr_edge_heads");
        if ((st = exclusive_scan_u32(w.head, total, w.hoff, w.scan, stream)) != GT_OK) return st;
        k_emit_cols<<<gt_, 256, 0, stream>>>(w.keys, total, w.head, w.hoff, (uint64_t(1) << g.nbits) - 1, col_out);
        GT_LAUNCH_CHECK("ecr_emit_cols");
        if ((st = read_i64(w.hoff + total, &out, stream)) != GT_OK) return st;
    } else {
        if ((st = fill_i64(w.hoff, 1, 0, stream)) != GT_OK) return st;
    }
    k_row_bounds<<<grid_for(total + 1, 256, 65536), 256, 0, stream>>>(w.keys, total, w.head, w.hoff, g.nbits, n,
                                                                        rowptr_out);
    GT_LAUNCH_CHECK("ecr_row_bounds");
    *nnz_out = out;
    return GT_OK;
}
