// Device-wide building blocks: fills, scans, key counts, stable radix sort,
// CSR validation.  See prim.h.
#include "prim.h"

namespace gt {

// ============================================================== fills/copies

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        p[i] = v;
}
__global__ void k_fill_i64(int64_t* p, int64_t n, int64_t v) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        p[i] = v;
}
__global__ void k_iota_u32(uint32_t* p, int64_t n) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        p[i] = uint32_t(i);
}

gt_status fill_u32(uint32_t* p, int64_t n, uint32_t value, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_fill_u32<<<grid_for(n, 256, 8192), 256, 0, s>>>(p, n, value);
    GT_LAUNCH_CHECK("fill_u32");
    return GT_OK;
}
gt_status fill_i64(int64_t* p, int64_t n, int64_t value, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_fill_i64<<<grid_for(n, 256, 8192), 256, 0, s>>>(p, n, value);
    GT_LAUNCH_CHECK("fill_i64");
    return GT_OK;
}
gt_status iota_u32(uint32_t* p, int64_t n, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_iota_u32<<<grid_for(n, 256, 8192), 256, 0, s>>>(p, n);
    GT_LAUNCH_CHECK("iota_u32");
    return GT_OK;
}
// ============================================================= side streams

gt_status spread_open(const char* who, hipStream_t main, const hipStream_t* side, const hipEvent_t* events,
                      int n_side, Spread* sp) {
    sp->main = main;
    sp->n_side = 0;
    if (n_side < 0 || n_side > kMaxSide || (n_side > 0 && (!side || !events)))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": n_side must be in [0, 2], with stream and event arrays");
    if (n_side == 0) return GT_OK;
    for (int k = 0; k < n_side; ++k) {
        if (!side[k] || side[k] == main)
            return fail(GT_ERR_INVALID_ARG, std::string(who) + ": a side stream is null or the call's own stream");
        for (int j = 0; j < k; ++j)
            if (side[j] == side[k]) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": a side stream repeats");
    }
    for (int k = 0; k <= n_side; ++k) {
        if (!events[k]) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": a null event");
        for (int j = 0; j < k; ++j)
            if (events[j] == events[k]) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": an event repeats");
    }
    hipDevice_t dev = -1;
    if (main) {
        GT_HIP(hipStreamGetDevice(main, &dev));
    } else {
        int d = -1;
        GT_HIP(hipGetDevice(&d));
        dev = d;
    }
    for (int k = 0; k < n_side; ++k) {
        hipDevice_t sdev = -1;
        GT_HIP(hipStreamGetDevice(side[k], &sdev));
        if (sdev != dev) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": a side stream is on another device");
    }
    sp->fork_ev = events[0];
    for (int k = 0; k < n_side; ++k) {
        sp->side[k] = side[k];
        sp->join_ev[k] = events[k + 1];
    }
    sp->n_side = n_side;
    return GT_OK;
}

gt_status Spread::fork() {
    if (n_side == 0) return GT_OK;
    GT_HIP(hipEventRecord(fork_ev, main));
    for (int k = 0; k < n_side; ++k) GT_HIP(hipStreamWaitEvent(side[k], fork_ev, 0));
    forked = true;
    return GT_OK;
}

gt_status Spread::join() {
    if (n_side == 0 || !forked) return GT_OK;
    for (int k = 0; k < n_side; ++k) {
        GT_HIP(hipEventRecord(join_ev[k], side[k]));
        GT_HIP(hipStreamWaitEvent(main, join_ev[k], 0));
    }
    forked = false;
    return GT_OK;
}

gt_status copy_bytes(void* dst, const void* src, int64_t bytes, hipStream_t s) {
    if (bytes <= 0) return GT_OK;
    GT_HIP(hipMemcpyAsync(dst, src, size_t(bytes), hipMemcpyDeviceToDevice, s));
    return GT_OK;
}

// ===================================================================== scan

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

int64_t scan_tmp_elems(int64_t n) { return cdiv(n, kScanTile) + 1; }

template <typename In>
__device__ __forceinline__ int64_t load_as_i64(const In* p, int64_t i, int64_t n) {
    return i < n ? static_cast<int64_t>(p[i]) : 0;
}

// Block-wide exclusive scan of one value per thread; returns the block total.
__device__ __forceinline__ int64_t block_exscan(int64_t v, int64_t* excl) {
    __shared__ int64_t s_w[kScanThreads / kWave];
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_w[w] = x;
    __syncthreads();
    int64_t before = 0, total = 0;
#pragma unroll
    for (int i = 0; i < kScanThreads / kWave; ++i) {
        int64_t t = s_w[i];
        if (i < w) before += t;
        total += t;
    }
    __syncthreads();
    *excl = before + x - v;
    return total;
}

template <typename In>
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const In* in, int64_t n, int64_t* sums) {
    const int64_t base = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
    int64_t acc = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) acc += load_as_i64(in, base + k, n);
    int64_t ex;
    int64_t tot = block_exscan(acc, &ex);
    if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// Single block: exclusive scan of nb sums in place; sums[nb] = total.
__global__ __launch_bounds__(kScanThreads) void k_scan_sums(int64_t* sums, int64_t nb) {
    const int64_t per = cdiv(nb, kScanThreads);
    const int64_t lo = int64_t(threadIdx.x) * per;
    const int64_t hi = lo + per < nb ? lo + per : nb;
    int64_t acc = 0;
    for (int64_t i = lo; i < hi; ++i) acc += sums[i];
    int64_t ex;
    int64_t tot = block_exscan(acc, &ex);
    for (int64_t i = lo; i < hi; ++i) {
        int64_t t = sums[i];
        sums[i] = ex;
        ex += t;
    }
    if (threadIdx.x == 0) sums[nb] = tot;
}

template <typename In>
__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const In* in, int64_t n, const int64_t* sums,
                                                              int64_t nb, int64_t* out) {
    const int64_t base = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
    int64_t v[kScanItems];
    int64_t acc = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = load_as_i64(in, base + k, n);
        acc += v[k];
    }
    int64_t ex;
    block_exscan(acc, &ex);
    ex += sums[blockIdx.x];
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) out[base + k] = ex;
        ex += v[k];
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = sums[nb];
}

// Up to kScanFewBlocks blocks: each block adds the sums of the blocks before
// it itself, so the scan of the block sums needs no launch of its own; the
// last block writes the total.
constexpr int64_t kScanFewBlocks = 1024;
template <typename In>
__global__ __launch_bounds__(kScanThreads) void k_scan_apply_few(const In* in, int64_t n, const int64_t* sums,
                                                                  int64_t* out) {
    __shared__ int64_t s_pre;
    int64_t before = 0;
    for (int64_t b = threadIdx.x; b < int64_t(blockIdx.x); b += kScanThreads) before += sums[b];
    int64_t ex0;
    before = block_exscan(before, &ex0);  // the sum over the threads
    if (threadIdx.x == 0) s_pre = before;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
    int64_t v[kScanItems];
    int64_t acc = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = load_as_i64(in, base + k, n);
        acc += v[k];
    }
    int64_t ex;
    const int64_t tot = block_exscan(acc, &ex);
    ex += s_pre;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) out[base + k] = ex;
        ex += v[k];
    }
    if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = s_pre + tot;
}

template <typename In>
static gt_status exscan(const In* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s) {
    if (n <= 0) return fill_i64(out, 1, 0, s);
    const int64_t nb = cdiv(n, kScanTile);
    if (nb == 1) {  // one block: no block sums at all
        k_scan_apply_few<In><<<1, kScanThreads, 0, s>>>(in, n, nullptr, out);
        GT_LAUNCH_CHECK("scan_one_block");
        return GT_OK;
    }
    k_scan_reduce<In><<<unsigned(nb), kScanThreads, 0, s>>>(in, n, tmp.block_sums);
    if (nb <= kScanFewBlocks) {
        GT_LAUNCH_CHECK("scan_reduce");
        k_scan_apply_few<In><<<unsigned(nb), kScanThreads, 0, s>>>(in, n, tmp.block_sums, out);
        GT_LAUNCH_CHECK("scan_apply");
        return GT_OK;
    }
    GT_LAUNCH_CHECK("scan_reduce");
    k_scan_sums<<<1, kScanThreads, 0, s>>>(tmp.block_sums, nb);
    GT_LAUNCH_CHECK("scan_sums");
    k_scan_apply<In><<<unsigned(nb), kScanThreads, 0, s>>>(in, n, tmp.block_sums, nb, out);
    GT_LAUNCH_CHECK("scan_apply");
    return GT_OK;
}

gt_status exclusive_scan_i32(const int32_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s) {
    return exscan(in, n, out, tmp, s);
}
gt_status exclusive_scan_u32(const uint32_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s) {
    return exscan(in, n, out, tmp, s);
}
gt_status exclusive_scan_i64(const int64_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s) {
    return exscan(in, n, out, tmp, s);
}

// =============================================================== key counts

__global__ void k_count_keys(const int32_t* keys, int64_t n, uint32_t* counts) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        atomicAdd(&counts[keys[i]], 1u);
}

gt_status count_keys(const int32_t* keys, int64_t n, uint32_t* counts, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_count_keys<<<grid_for(n, 256, 16384), 256, 0, s>>>(keys, n, counts);
    GT_LAUNCH_CHECK("count_keys");
    return GT_OK;
}

// =============================================================== radix sort
// 8-bit digits, least significant first.  A tile of 2048 keys per workgroup of
// four wavefronts; wavefront w owns keys [512 w, 512 w + 512) of its tile, in
// rounds of 64.  Each key's rank among the tile's keys of its digit follows
// (wavefront, round, lane) order, which is the input order, so every pass is
// stable and so is the whole sort.  The tile is put in digit order in LDS
// first, so the keys of one digit leave in one contiguous run.

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kSortRounds = 8;  // rounds of 64 keys per wavefront
constexpr int kSortTile = kSortWaves * kSortRounds * kWave;

int64_t sort_tiles(int64_t n) { return cdiv(n, kSortTile); }

SortTmp sort_tmp(Ws& ws, int64_t n, int key_bytes, bool with_values) {
    SortTmp t;
    const int64_t tiles = sort_tiles(n > 0 ? n : 1);
    t.keys_alt = ws.take<char>(size_t(n > 0 ? n : 1) * key_bytes);
    t.vals_alt = with_values ? ws.take<uint32_t>(size_t(n > 0 ? n : 1)) : nullptr;
    t.hist = ws.take<uint32_t>(size_t(256 * tiles));
    t.offsets = ws.take<int64_t>(size_t(256 * tiles + 1));
    t.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(256 * tiles)));
    return t;
}

// Digit counts of one tile.  The lanes of a wavefront holding the same digit
// are found with eight ballots (one per digit bit) and counted with one LDS
// add by the first of them, so a tile whose keys share few digits does not
// serialise on a few LDS addresses.
template <typename K>
__global__ __launch_bounds__(kSortThreads) void k_sort_hist(const K* keys, int64_t n, int shift, int64_t tiles,
                                                             uint32_t* hist) {
    __shared__ uint32_t s_h[256];
    s_h[threadIdx.x] = 0;
    __syncthreads();
    constexpr int R = kSortTile / kSortThreads;
    const int64_t base = int64_t(blockIdx.x) * kSortTile;
    K key[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t i = base + r * kSortThreads + threadIdx.x;
        key[r] = i < n ? keys[i] : K(0);
    }
    const uint64_t lt = lanemask_lt();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool valid = base + r * kSortThreads + threadIdx.x < n;
        const uint32_t d = uint32_t(key[r] >> shift) & 255u;
        uint64_t peers = ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bm = ballot(bit);
            peers &= bit ? bm : ~bm;
        }
        if (valid && (peers & lt) == 0) atomicAdd(&s_h[d], uint32_t(__popcll(peers)));
    }
    __syncthreads();
    hist[int64_t(threadIdx.x) * tiles + blockIdx.x] = s_h[threadIdx.x];
}

template <typename K>
__global__ __launch_bounds__(kSortThreads) void k_sort_scatter(const K* keys, const uint32_t* vals, int64_t n,
                                                                int shift, int64_t tiles, const int64_t* offsets,
                                                                K* keys_out, uint32_t* vals_out) {
    __shared__ int s_wc[kSortWaves][256];  // per-wavefront digit counts, then their starts in the tile
    __shared__ int s_ds[256];              // tile-local start of each digit
    __shared__ int s_part[kSortWaves];
    __shared__ int64_t s_go[256];          // output start of the tile's keys of each digit
    __shared__ K s_k[kSortTile];
    __shared__ uint32_t s_v[kSortTile];
    const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) s_wc[k][tid] = 0;
    s_go[tid] = offsets[int64_t(tid) * tiles + blockIdx.x];
    const int64_t tile0 = int64_t(blockIdx.x) * kSortTile;
    const int64_t base = tile0 + w * (kSortRounds * kWave);
    K key[kSortRounds];
    uint32_t val[kSortRounds];
    int rk[kSortRounds];
#pragma unroll
    for (int r = 0; r < kSortRounds; ++r) {
        const int64_t i = base + r * kWave + lane;
        key[r] = i < n ? keys[i] : K(0);
        val[r] = (i < n && vals) ? vals[i] : 0u;
    }
    __syncthreads();
    const uint64_t lt = lanemask_lt();
#pragma unroll
    for (int r = 0; r < kSortRounds; ++r) {
        const bool valid = base + r * kWave + lane < n;
        const uint32_t d = uint32_t(key[r] >> shift) & 255u;
        uint64_t peers = ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bm = ballot(bit);
            peers &= bit ? bm : ~bm;
        }
        const int rank = __popcll(peers & lt);
        // the wavefront's count of digit d so far: read by every lane of the
        // digit, then advanced by its first lane (a wavefront's LDS accesses
        // complete in order)
        const int before = valid ? s_wc[w][d] : 0;
        if (valid && rank == 0) s_wc[w][d] = before + __popcll(peers);
        rk[r] = before + rank;
    }
    __syncthreads();
    // thread tid takes digit tid: the tile's count of it and each wavefront's share
    int tot = 0, wp[kSortWaves];
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
        wp[k] = tot;
        tot += s_wc[k][tid];
    }
    int x = tot;  // inclusive scan over the 256 digits
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_part[w] = x;
    __syncthreads();
    int ds = x - tot;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k)
        if (k < w) ds += s_part[k];
    s_ds[tid] = ds;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) s_wc[k][tid] = ds + wp[k];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kSortRounds; ++r) {
        if (base + r * kWave + lane < n) {
            const uint32_t d = uint32_t(key[r] >> shift) & 255u;
            const int p = s_wc[w][d] + rk[r];
            s_k[p] = key[r];
            s_v[p] = val[r];
        }
    }
    __syncthreads();
    const int64_t left = n - tile0;
    const int cnt = left < kSortTile ? int(left) : kSortTile;
    for (int p = tid; p < cnt; p += kSortThreads) {
        const K k = s_k[p];
        const uint32_t d = uint32_t(k >> shift) & 255u;
        const int64_t pos = s_go[d] + (p - s_ds[d]);
        keys_out[pos] = k;
        if (vals) vals_out[pos] = s_v[p];
    }
}

template <typename K>
static gt_status radix_sort(K* keys, uint32_t* values, int64_t n, int key_bits, SortTmp tmp, hipStream_t s) {
    if (n <= 1) return GT_OK;
    const int64_t tiles = sort_tiles(n);
    K* src_k = keys;
    K* dst_k = static_cast<K*>(tmp.keys_alt);
    uint32_t* src_v = values;
    uint32_t* dst_v = values ? tmp.vals_alt : nullptr;
    int passes = 0;
    for (int shift = 0; shift < key_bits; shift += 8, ++passes) {
        k_sort_hist<K><<<unsigned(tiles), kSortThreads, 0, s>>>(src_k, n, shift, tiles, tmp.hist);
        GT_LAUNCH_CHECK("sort_hist");
        gt_status st = exclusive_scan_u32(tmp.hist, 256 * tiles, tmp.offsets, tmp.scan, s);
        if (st != GT_OK) return st;
        k_sort_scatter<K><<<unsigned(tiles), kSortThreads, 0, s>>>(src_k, src_v, n, shift, tiles, tmp.offsets,
                                                                   dst_k, dst_v);
        GT_LAUNCH_CHECK("sort_scatter");
        K* tk = src_k;
        src_k = dst_k;
        dst_k = tk;
        uint32_t* tv = src_v;
        src_v = dst_v;
        dst_v = tv;
    }
    if (passes & 1) {
        gt_status st = copy_bytes(keys, src_k, n * int64_t(sizeof(K)), s);
        if (st != GT_OK) return st;
        if (values) {
            st = copy_bytes(values, src_v, n * 4, s);
            if (st != GT_OK) return st;
        }
    }
    return GT_OK;
}

gt_status radix_sort_u32(uint32_t* keys, uint32_t* values, int64_t n, int key_bits, SortTmp tmp, hipStream_t s) {
    return radix_sort<uint32_t>(keys, values, n, key_bits, tmp, s);
}
gt_status radix_sort_u64(uint64_t* keys, uint32_t* values, int64_t n, int key_bits, SortTmp tmp, hipStream_t s) {
    return radix_sort<uint64_t>(keys, values, n, key_bits, tmp, s);
}

// ========================================================== row partition

constexpr int kPartBlock = 256;

// Per-wavefront counts of each class in s[w][c]; returns the lane's rank
// among its wavefront's lanes of the same class.
__device__ __forceinline__ int part_ballots(int c, int ncls, int (*s)[kMaxClasses]) {
    const int w = threadIdx.x / kWave;
    int rank = 0;
    for (int k = 0; k < ncls; ++k) {
        const uint64_t m = __ballot(c == k);
        if (lane_id() == 0) s[w][k] = __popcll(m);
        if (c == k) rank = __popcll(m & lanemask_lt());
    }
    return rank;
}

__global__ __launch_bounds__(kPartBlock) void k_part_count(const int8_t* cls, int64_t n, int ncls, int64_t nblk,
                                                           int32_t* blk_cnt) {
    __shared__ int s[kPartBlock / kWave][kMaxClasses];
    const int64_t v = int64_t(blockIdx.x) * kPartBlock + threadIdx.x;
    part_ballots(v < n ? int(cls[v]) : -1, ncls, s);
    __syncthreads();
    if (int(threadIdx.x) < ncls) {
        int t = 0;
        for (int w = 0; w < kPartBlock / kWave; ++w) t += s[w][threadIdx.x];
        blk_cnt[threadIdx.x * nblk + blockIdx.x] = t;
    }
}

__global__ __launch_bounds__(kPartBlock) void k_part_scatter(const int8_t* cls, int64_t n, int ncls, int64_t nblk,
                                                             const int64_t* blk_off, int32_t* list) {
    __shared__ int s[kPartBlock / kWave][kMaxClasses];
    const int64_t v = int64_t(blockIdx.x) * kPartBlock + threadIdx.x;
    const int c = v < n ? int(cls[v]) : -1;
    const int rank = part_ballots(c, ncls, s);
    __syncthreads();
    if (c >= 0 && c < ncls) {
        int64_t pos = blk_off[c * nblk + blockIdx.x] + rank;
        for (int w = 0; w < int(threadIdx.x / kWave); ++w) pos += s[w][c];
        list[pos] = int32_t(v);
    }
}

__global__ void k_part_info(int ncls, int64_t nblk, const int64_t* blk_off, int64_t* info) {
    const int c = threadIdx.x;
    if (blockIdx.x != 0 || c >= ncls) return;
    info[c] = blk_off[c * nblk];
    info[ncls + c] = blk_off[(c + 1) * nblk] - blk_off[c * nblk];
}

PartitionTmp partition_tmp(Ws& ws, int64_t n) {
    PartitionTmp t;
    const int64_t nblk = cdiv(n > 0 ? n : 1, kPartBlock);
    t.blk_cnt = ws.take<int32_t>(size_t(kMaxClasses * nblk));
    t.blk_off = ws.take<int64_t>(size_t(kMaxClasses * nblk + 1));
    t.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(kMaxClasses * nblk + 1)));
    return t;
}

gt_status partition_rows(const int8_t* cls, int64_t n, int ncls, int32_t* list, int64_t* info, PartitionTmp t,
                         hipStream_t s) {
    if (n <= 0 || ncls < 1 || ncls > kMaxClasses) return fail(GT_ERR_INVALID_ARG, "partition_rows: bad sizes");
    const int64_t nblk = cdiv(n, kPartBlock);
    k_part_count<<<unsigned(nblk), kPartBlock, 0, s>>>(cls, n, ncls, nblk, t.blk_cnt);
    GT_LAUNCH_CHECK("partition_count");
    gt_status st = exclusive_scan_i32(t.blk_cnt, ncls * nblk, t.blk_off, t.scan, s);
    if (st != GT_OK) return st;
    k_part_scatter<<<unsigned(nblk), kPartBlock, 0, s>>>(cls, n, ncls, nblk, t.blk_off, list);
    GT_LAUNCH_CHECK("partition_scatter");
    k_part_info<<<1, 64, 0, s>>>(ncls, nblk, t.blk_off, info);
    GT_LAUNCH_CHECK("partition_info");
    return GT_OK;
}

// =========================================================== CSR validation

// Validation in two coalesced passes.  k_validate_rows checks every row's
// bounds (one thread per row).  k_validate_entries cuts col into chunks of
// kValidateChunk entries, one workgroup per chunk: it finds the chunk's first
// row by a binary search on rowptr, marks in LDS the chunk's entries that start
// a non-empty row, then every thread checks its entries (0 <= col < n, and
// col[e - 1] < col[e] unless e starts a row).  Every workgroup does the same
// work whatever the row lengths, and every read stays inside rowptr[0..n] and
// col[0..nnz) even when rowptr is wrong (then the rows pass reports it).
constexpr int kValidateChunk = 2048;
constexpr int kValidateThreads = 256;

__global__ void k_validate_rows(int64_t n, int64_t nnz, const int64_t* __restrict__ rowptr, uint32_t* flags) {
    uint32_t f = 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        if (rowptr[0] != 0 || rowptr[n] != nnz) f |= kOutOfRange;
    }
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t a = rowptr[i], b = rowptr[i + 1];
        if (a > b) f |= kUnsorted;
        else if (a < 0 || b > nnz) f |= kOutOfRange;
        else if (b - a > kLongRow) f |= kLongRowSeen;
    }
    if (f) atomicOr(flags, f);
}

__global__ __launch_bounds__(kValidateThreads) void k_validate_entries(int64_t n, int64_t nnz,
                                                                       const int64_t* __restrict__ rowptr,
                                                                       const int32_t* __restrict__ col,
                                                                       uint32_t* flags) {
    __shared__ uint32_t s_start[kValidateChunk / 32];
    __shared__ int64_t s_row;
    uint32_t f = 0;
    const int64_t chunks = cdiv(nnz, kValidateChunk);
    for (int64_t c = blockIdx.x; c < chunks; c += gridDim.x) {
        const int64_t c0 = c * kValidateChunk, c1 = c0 + kValidateChunk < nnz ? c0 + kValidateChunk : nnz;
        for (int w = threadIdx.x; w < kValidateChunk / 32; w += kValidateThreads) s_start[w] = 0;
        if (threadIdx.x == 0) {  // the last row r with rowptr[r] <= c0
            int64_t lo = 0, hi = n;
            while (hi - lo > 1) {
                const int64_t mid = (lo + hi) >> 1;
                if (rowptr[mid] <= c0) lo = mid;
                else hi = mid;
            }
            s_row = lo;
        }
        __syncthreads();
        // rows r0, r0 + 1, ... while they start before c1; a non-empty row starting
        // inside the chunk marks its first entry
        for (int64_t r = s_row + threadIdx.x;; r += kValidateThreads) {
            const bool in = r < n;
            const int64_t a = in ? rowptr[r] : c1;
            const bool more = __syncthreads_or(in && a < c1);
            if (in && a >= c0 && a < c1 && a < rowptr[r + 1]) {
                const int64_t k = a - c0;
                atomicOr(&s_start[k >> 5], 1u << (k & 31));
            }
            if (!more) break;
        }
        __syncthreads();
        for (int64_t e = c0 + threadIdx.x; e < c1; e += kValidateThreads) {
            const int64_t x = col[e];
            if (x < 0 || x >= n) f |= kOutOfRange;
            const int64_t k = e - c0;
            if (e > 0 && !((s_start[k >> 5] >> (k & 31)) & 1u)) {
                const int64_t prev = col[e - 1];
                if (x == prev) f |= kDuplicate;
                else if (x < prev) f |= kUnsorted;
            }
        }
        __syncthreads();
    }
    if (f) atomicOr(flags, f);
}

gt_status launch_validate_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, uint32_t* flags,
                              hipStream_t s) {
    gt_status st = fill_u32(flags, 1, 0, s);
    if (st != GT_OK) return st;
    k_validate_rows<<<grid_for(n > 0 ? n : 1, 256, 4096), 256, 0, s>>>(n, nnz, rowptr, flags);
    GT_LAUNCH_CHECK("validate_rows");
    if (n > 0 && nnz > 0) {
        k_validate_entries<<<grid_for(nnz, kValidateChunk, 8192), kValidateThreads, 0, s>>>(n, nnz, rowptr, col,
                                                                                            flags);
        GT_LAUNCH_CHECK("validate_entries");
    }
    return GT_OK;
}

gt_status read_validation(const uint32_t* flags, hipStream_t s) {
    uint32_t f = 0;
    GT_HIP(hipMemcpyAsync(&f, flags, sizeof(f), hipMemcpyDeviceToHost, s));
    GT_HIP(hipStreamSynchronize(s));
    return validation_result(f);
}

gt_status validation_result(uint32_t f) {
    if (f & kOutOfRange) return fail(GT_ERR_OUT_OF_RANGE, "CSR: rowptr or column index out of range");
    if (f & kDuplicate) return fail(GT_ERR_DUPLICATE, "CSR: repeated column inside a row");
    if (f & kUnsorted) return fail(GT_ERR_UNSORTED, "CSR: row not strictly increasing or rowptr decreasing");
    return GT_OK;
}

}  // namespace gt

using namespace gt;

extern "C" size_t gt_validate_csr_workspace_size(void) { return 256; }

extern "C" gt_status gt_validate_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, void* ws,
                                     size_t ws_bytes, hipStream_t stream) {
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << 32))
        return fail(GT_ERR_INVALID_ARG, "gt_validate_csr: n or nnz out of range");
    if (!rowptr || (nnz > 0 && !col) || !ws) return fail(GT_ERR_INVALID_ARG, "gt_validate_csr: null pointer");
    if (ws_bytes < gt_validate_csr_workspace_size()) return fail(GT_ERR_WORKSPACE, "gt_validate_csr: workspace too small");
    uint32_t* flags = static_cast<uint32_t*>(ws);
    gt_status st = launch_validate_csr(n, nnz, rowptr, col, flags, stream);
    if (st != GT_OK) return st;
    return read_validation(flags, stream);
}
