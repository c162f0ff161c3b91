// Dense/sparse tile plan (§3.4, cluster sparsity and the transfer threshold),
// read as an exact execution plan over T x T tiles of the reordered adjacency.
//
// One workgroup per tile row I keeps a direct-indexed count per tile column J
// in LDS (R <= 16384 columns: 64 KiB), so counting touches only the edges of
// the tile row.  The same kernel, run a second time with the output offsets
// known, writes the (I, J)-sorted dense tile list, the tile bit masks and the
// remainder CSR.  Rows of more than kLongRow edges (hubs, a global token) are
// left out of the tile row's workgroup: the count pass publishes each tile
// row's dense/sparse split as a bit set, and their edges are counted and
// written chunk by chunk over the whole grid.
//
// The remainder's transpose comes from the count pass: it tags every edge with
// its column if the edge stays in the remainder (else with n), in CSR order,
// and a stable radix sort of (tag, row) leaves the remainder's rows grouped by
// column, rows ascending; the column pointers are binary searches in the
// sorted tags.  No step adds into a shared counter, so every output is
// deterministic.

#include "prim.h"

namespace gt {
namespace {

constexpr int kThreads = 256;      // the long-row kernels
constexpr int kTileThreads = 1024;  // one workgroup per tile row: 16 wavefronts share its LDS count table
constexpr int kMaxR = 16384;
constexpr int kMaxT = 128;
constexpr int kRowsPerWave = kMaxT / (kTileThreads / kWave);  // rows of a tile row per wavefront
constexpr int kCountBatch = 8;                                 // column loads in flight per thread when counting
constexpr int kShortRow = kWave;  // rows of at most one slice of 64 edges stay in the tile row's workgroup
constexpr int kMedBatch = 4;      // 64-edge slices of a medium row loaded at once
// Tile rows of more than kHeavyEdges edges (hubs gathered by the reordering)
// are counted before the tile-row pass by many workgroups, kHeavyChunk edges
// each, into a count row of their own (at most kMaxHeavy of them; the rest
// count in their own workgroup).
constexpr int64_t kHeavyEdges = 32768;
constexpr int kMaxHeavy = 64;
constexpr int64_t kHeavyChunk = 65536;
constexpr uint32_t kDense = 0x80000000u;

// Exclusive prefix of a 0/1 flag over the workgroup, in thread order; *total = the sum.
__device__ __forceinline__ int64_t block_flag_scan(bool flag, int64_t* s, int64_t* total) {
    const uint64_t b = __ballot(flag);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) s[w] = __popcll(b);
    __syncthreads();
    int64_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kThreads / kWave; ++i) {
        const int64_t t = s[i];
        if (i < w) before += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return before + __popcll(b & lanemask_lt());
}

__device__ __forceinline__ int64_t block_exscan_i64(int64_t v, int64_t* s, int64_t* total) {
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s[w] = x;
    __syncthreads();
    int64_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kTileThreads / kWave; ++i) {
        const int64_t t = s[i];
        if (i < w) before += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return before + x - v;
}

// kFill = false: dense tiles per tile row, remainder degree per row, and the
// remainder tags: tag[e] = col[e] if edge e stays in the remainder, else n;
// row_of_e[e] = its row.
// kFill = true: the plan arrays (offsets from the count pass).
// The count pass also publishes the split of tile row I for the long rows:
// bit J of dense_bits[I * W + J / 32] marks a dense tile, dense_pre[I * W + w]
// counts the dense tiles in words before w (W = ceil(R / 32)).
template <bool kFill>
__global__ __launch_bounds__(kTileThreads) void k_tiles(int64_t n, const int64_t* rowptr, const int32_t* col, int T,
                                                    int R, uint32_t tau_ppm, int32_t* dense_per_tilerow,
                                                    int32_t* sp_deg, const int64_t* tile_rowptr, int32_t* tile_col,
                                                    int32_t* tile_nnz, uint32_t* tile_mask,
                                                    const int64_t* sp_rowptr, int32_t* sp_col, uint32_t* tag,
                                                    uint32_t* row_of_e, int W, uint32_t* dense_bits,
                                                    uint32_t* dense_pre, int32_t* sp_pos, int32_t* tile_pos,
                                                    const int32_t* heavy_slot, const uint32_t* heavy_cnt) {
    __shared__ uint32_t s_cnt[kMaxR];
    __shared__ int64_t s_red[kTileThreads / kWave];
    __shared__ int64_t s_rp[kMaxT + 1];
    __shared__ int64_t s_sp[kFill ? kMaxT : 1];  // fill: each row's first remainder position
    __shared__ uint64_t s_gbits[kMaxR / kWave];
    __shared__ uint32_t s_gpre[kMaxR / kWave];
    const int I = blockIdx.x;
    const int64_t r0 = int64_t(I) * T;
    const int64_t r1 = r0 + T < n ? r0 + T : n;
    const int64_t rows = r1 - r0;
    for (int J = threadIdx.x; J < R; J += kTileThreads) s_cnt[J] = 0;
    for (int j = threadIdx.x; j <= rows; j += kTileThreads) s_rp[j] = rowptr[r0 + j];
    if (kFill)
        for (int j = threadIdx.x; j < rows; j += kTileThreads) s_sp[j] = sp_rowptr[r0 + j];
    __syncthreads();
    const int64_t e0 = s_rp[0], e1 = s_rp[rows];
    const int tshift = __builtin_ctz(unsigned(T));
    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    // the columns of this wavefront's short rows (rows w, w + 16, ...), for the
    // per-row pass at the end: loaded now, so they arrive while the tile row is counted
    int first[kRowsPerWave];
#pragma unroll
    for (int k = 0; k < kRowsPerWave; ++k) {
        const int64_t rl = w + int64_t(k) * (kTileThreads / kWave);
        first[k] = 0;
        if (rl < rows) {
            const int64_t a = s_rp[rl], b = s_rp[rl + 1];
            if (b - a <= kShortRow && a + lane < b) first[k] = col[a + lane];
        }
    }
    // every edge of the tile row, long rows included (taken from the heavy
    // count row if the tile row has one); kCountBatch loads in flight per
    // thread, so a tile row holding hubs is not a chain of round trips
    const int hslot = heavy_slot[I];
    if (hslot >= 0)
        for (int J = threadIdx.x; J < R; J += kTileThreads) s_cnt[J] = heavy_cnt[int64_t(hslot) * R + J];
    for (int64_t base = e0 + threadIdx.x; hslot < 0 && base < e1; base += kCountBatch * kTileThreads) {
        int c[kCountBatch];
#pragma unroll
        for (int u = 0; u < kCountBatch; ++u) {
            const int64_t e = base + int64_t(u) * kTileThreads;
            c[u] = e < e1 ? col[e] : -1;
        }
#pragma unroll
        for (int u = 0; u < kCountBatch; ++u)
            if (c[u] >= 0) atomicAdd(&s_cnt[c[u] >> tshift], 1u);
    }
    __syncthreads();
    // classify 64 tile columns per wavefront step (lane j takes column 64 m + j,
    // so LDS reads do not collide in banks); keep the count in the low bits and
    // each group's dense bits in s_gbits[m]
    const int ngroups = (R + kWave - 1) / kWave;
    const uint64_t lt = lanemask_lt();
    for (int m = w; m < ngroups; m += kTileThreads / kWave) {
        const int J = m * kWave + lane;
        const uint32_t c = J < R ? s_cnt[J] : 0u;
        const int64_t wcols = n - int64_t(J) * T < T ? n - int64_t(J) * T : T;
        const uint64_t area = uint64_t(rows) * uint64_t(wcols > 0 ? wcols : 0);
        const bool dense = c >= 1 && uint64_t(c) * 1000000ull >= uint64_t(tau_ppm) * area;
        if (dense) s_cnt[J] = c | kDense;
        const uint64_t bits = ballot(dense);
        if (lane == 0) s_gbits[m] = bits;
    }
    __syncthreads();
    // dense tiles before each group
    int64_t total;
    const int64_t gpre = block_exscan_i64(int(threadIdx.x) < ngroups ? __popcll(s_gbits[threadIdx.x]) : 0, s_red,
                                          &total);
    if (int(threadIdx.x) < ngroups) s_gpre[threadIdx.x] = uint32_t(gpre);
    __syncthreads();
    if (!kFill) {
        if (threadIdx.x == 0) dense_per_tilerow[I] = int32_t(total);
        for (int m = threadIdx.x; m < ngroups; m += kTileThreads) {
            const uint64_t bits = s_gbits[m];
            for (int q = 0; q < 2; ++q) {
                const int wd = 2 * m + q;
                if (wd >= W) break;
                dense_bits[int64_t(I) * W + wd] = uint32_t(bits >> (32 * q));
                dense_pre[int64_t(I) * W + wd] = s_gpre[m] + (q ? uint32_t(__popc(uint32_t(bits))) : 0u);
            }
        }
    } else {
        const int64_t base = tile_rowptr[I];
        for (int m = w; m < ngroups; m += kTileThreads / kWave) {
            const int J = m * kWave + lane;
            const uint64_t bits = s_gbits[m];
            if ((bits >> lane) & 1u) {
                const uint32_t k = s_gpre[m] + uint32_t(__popcll(bits & lt));
                tile_col[base + k] = J;
                tile_nnz[base + k] = int32_t(s_cnt[J] & ~kDense);
                s_cnt[J] = kDense | k;
            }
        }
    }
    __syncthreads();
    // per row of at most kShortRow edges: remainder degree and tags (count) or
    // remainder edges and mask bits (fill), from the columns loaded at the
    // start.  Longer rows are k_tiles_med's (up to kLongRow) or the long-row
    // kernels'.
    const int wpr = T / 32;  // mask words per tile row
#pragma unroll
    for (int k = 0; k < kRowsPerWave; ++k) {
        const int64_t rl = w + int64_t(k) * (kTileThreads / kWave);
        if (rl >= rows) break;
        const int64_t i = r0 + rl;
        const int64_t a = s_rp[rl], b = s_rp[rl + 1];
        if (b - a > kShortRow) {
            if (!kFill && lane == 0 && b - a > kLongRow) sp_deg[i] = 0;  // the long-row kernels add theirs
            continue;
        }
        const int64_t e = a + lane;
        const bool valid = e < b;
        const int c = first[k];
        const int J = c >> tshift;
        const uint32_t f = valid ? s_cnt[J] : 0u;
        const bool dense = valid && (f & kDense);
        const bool sparse = valid && !dense;
        const uint64_t sb = ballot(sparse);
        if (kFill) {
            if (dense) {
                const int64_t kk = tile_rowptr[I] + int64_t(f & ~kDense);
                const int cl = c - J * T;
                const int64_t word = kk * int64_t(T) * wpr + rl * wpr + cl / 32;
                atomicOr(&tile_mask[word], 1u << (cl & 31));
                // the row's first edge in this tile (its columns are sorted)
                if (tile_pos && (e == a || (col[e - 1] >> tshift) != J)) tile_pos[kk * T + rl] = int32_t(e);
            }
            if (sparse) {
                const int64_t pos = s_sp[rl] + __popcll(sb & lt);
                sp_col[pos] = c;
                if (sp_pos) sp_pos[pos] = int32_t(e);
            }
        } else {
            if (valid) {
                tag[e] = sparse ? uint32_t(c) : uint32_t(n);
                row_of_e[e] = uint32_t(i);
            }
            if (lane == 0) sp_deg[i] = int32_t(__popcll(sb));
        }
    }
}

// One workgroup: the heavy tile rows (more than kHeavyEdges edges), the first
// kMaxHeavy of them in order: heavy_slot[I] = their number (else -1),
// heavy_list[h] = the tile row of number h, *heavy_n = how many.
// Thread t takes tile rows [kSlotsPer t, kSlotsPer t + kSlotsPer), all loaded at once.
constexpr int kSlotsPer = kMaxR / kTileThreads;
__global__ __launch_bounds__(kTileThreads) void k_heavy_slots(int64_t n, const int64_t* rowptr, int T, int R,
                                                              int32_t* heavy_slot, int32_t* heavy_list,
                                                              int32_t* heavy_n) {
    __shared__ int64_t s_red[kTileThreads / kWave];
    const int I0 = threadIdx.x * kSlotsPer;
    int64_t at[kSlotsPer + 1];
#pragma unroll
    for (int k = 0; k <= kSlotsPer; ++k) {
        const int64_t r = int64_t(I0 + k) * T;
        at[k] = I0 + k <= R ? rowptr[r < n ? r : n] : 0;
    }
    uint32_t heavy = 0;
    int cnt = 0;
#pragma unroll
    for (int k = 0; k < kSlotsPer; ++k)
        if (I0 + k < R && at[k + 1] - at[k] > kHeavyEdges) {
            heavy |= 1u << k;
            ++cnt;
        }
    int64_t tot;
    int64_t pre = block_exscan_i64(cnt, s_red, &tot);
#pragma unroll
    for (int k = 0; k < kSlotsPer; ++k) {
        const int I = I0 + k;
        if (I >= R) break;
        const bool kept = ((heavy >> k) & 1u) && pre < kMaxHeavy;
        heavy_slot[I] = kept ? int32_t(pre) : -1;
        if (kept) heavy_list[pre] = I;
        if ((heavy >> k) & 1u) ++pre;
    }
    if (threadIdx.x == 0) *heavy_n = int32_t(tot < kMaxHeavy ? tot : kMaxHeavy);
}

// The heavy tile rows' edges in chunks of kHeavyChunk, dealt over the grid:
// each chunk counted per tile column in LDS, then added to its tile row's
// count row (which starts at zero).
__global__ __launch_bounds__(kTileThreads) void k_heavy_count(int64_t n, const int64_t* rowptr, const int32_t* col,
                                                              int T, int R, const int32_t* heavy_list,
                                                              const int32_t* heavy_n, uint32_t* heavy_cnt) {
    __shared__ uint32_t s_cnt[kMaxR];
    const int nh = *heavy_n;
    const int tshift = __builtin_ctz(unsigned(T));
    int64_t q0 = 0;  // chunks of the heavy rows before h
    for (int h = 0; h < nh; ++h) {
        const int64_t I = heavy_list[h];
        const int64_t r0 = I * T, r1 = r0 + T < n ? r0 + T : n;
        const int64_t E0 = rowptr[r0], E1 = rowptr[r1];
        const int64_t nch = cdiv(E1 - E0, kHeavyChunk);
        // this workgroup's chunks of row h: global numbers q0 + j with (q0 + j) % grid == block
        int64_t j = (int64_t(blockIdx.x) - q0 % gridDim.x + gridDim.x) % gridDim.x;
        for (; j < nch; j += gridDim.x) {
            for (int J = threadIdx.x; J < R; J += kTileThreads) s_cnt[J] = 0;
            __syncthreads();
            const int64_t c0 = E0 + j * kHeavyChunk, c1 = c0 + kHeavyChunk < E1 ? c0 + kHeavyChunk : E1;
            for (int64_t base = c0 + threadIdx.x; base < c1; base += kCountBatch * kTileThreads) {
                int c[kCountBatch];
#pragma unroll
                for (int u = 0; u < kCountBatch; ++u) {
                    const int64_t e = base + int64_t(u) * kTileThreads;
                    c[u] = e < c1 ? col[e] : -1;
                }
#pragma unroll
                for (int u = 0; u < kCountBatch; ++u)
                    if (c[u] >= 0) atomicAdd(&s_cnt[c[u] >> tshift], 1u);
            }
            __syncthreads();
            for (int J = threadIdx.x; J < R; J += kTileThreads)
                if (s_cnt[J]) atomicAdd(&heavy_cnt[int64_t(h) * R + J], s_cnt[J]);
            __syncthreads();
        }
        q0 += nch;
    }
}

__device__ __forceinline__ bool tile_is_dense(const uint32_t* __restrict__ bits, int J) {
    return (bits[J >> 5] >> (J & 31)) & 1u;
}

// Rows of kShortRow + 1 to kLongRow edges: class 0 of the medium-row list.
__global__ void k_med_class(int64_t n, const int64_t* rowptr, int8_t* cls) {
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x) {
        const int64_t d = rowptr[i + 1] - rowptr[i];
        cls[i] = (d > kShortRow && d <= kLongRow) ? int8_t(0) : int8_t(-1);
    }
}

// One wavefront per listed medium row, its slices of 64 edges kMedBatch at a
// time: the dense test and the tile's number come from the count pass's bit
// sets (dense_bits, dense_pre).  kFill = false: remainder degree and tags;
// true: remainder edges, mask bits and edge positions.
template <bool kFill>
__global__ __launch_bounds__(256) void k_tiles_med(int64_t n, const int32_t* list, const int64_t* list_len,
                                                   const int64_t* rowptr, const int32_t* col, int T, int W,
                                                   const uint32_t* dense_bits, const uint32_t* dense_pre,
                                                   int32_t* sp_deg, uint32_t* tag, uint32_t* row_of_e,
                                                   const int64_t* tile_rowptr, uint32_t* tile_mask,
                                                   const int64_t* sp_rowptr, int32_t* sp_col, int32_t* sp_pos,
                                                   int32_t* tile_pos) {
    const int lane = lane_id();
    const uint64_t lt = lanemask_lt();
    const int tshift = __builtin_ctz(unsigned(T));
    const int wpr = T / 32;
    const int64_t len = *list_len;
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t idx = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave; idx < len; idx += waves) {
        const int64_t i = list[idx];
        const int64_t I = i / T, rl = i - I * T;
        const uint32_t* bits = dense_bits + I * W;
        const uint32_t* pre = dense_pre + I * W;
        const int64_t a = rowptr[i], b = rowptr[i + 1];
        int64_t sp = kFill ? sp_rowptr[i] : 0;
        const int64_t tbase = kFill ? tile_rowptr[I] : 0;
        for (int64_t eb0 = a; eb0 < b; eb0 += kMedBatch * kWave) {
            int cb[kMedBatch];
#pragma unroll
            for (int u = 0; u < kMedBatch; ++u) {
                const int64_t e = eb0 + u * kWave + lane;
                cb[u] = e < b ? col[e] : 0;
            }
#pragma unroll
            for (int u = 0; u < kMedBatch; ++u) {
                const int64_t eb = eb0 + u * kWave;
                if (eb >= b) break;
                const int64_t e = eb + lane;
                const bool valid = e < b;
                const int c = cb[u];
                const int J = c >> tshift;
                const uint32_t wd = valid ? bits[J >> 5] : 0u;
                const bool dense = valid && ((wd >> (J & 31)) & 1u);
                const bool sparse = valid && !dense;
                const uint64_t sb = ballot(sparse);
                if (kFill) {
                    if (dense) {
                        const int64_t kk = tbase + pre[J >> 5] + __popc(wd & ((1u << (J & 31)) - 1u));
                        const int cl = c - J * T;
                        atomicOr(&tile_mask[kk * int64_t(T) * wpr + rl * wpr + cl / 32], 1u << (cl & 31));
                        if (tile_pos && (e == a || (col[e - 1] >> tshift) != J))
                            tile_pos[kk * T + rl] = int32_t(e);
                    }
                    if (sparse) {
                        const int64_t pos = sp + __popcll(sb & lt);
                        sp_col[pos] = c;
                        if (sp_pos) sp_pos[pos] = int32_t(e);
                    }
                } else if (valid) {
                    tag[e] = sparse ? uint32_t(c) : uint32_t(n);
                    row_of_e[e] = uint32_t(i);
                }
                sp += __popcll(sb);
            }
        }
        if (!kFill && lane == 0) sp_deg[i] = int32_t(sp);
    }
}

// Count pass of the long rows: remainder degree (added to the zero the tile
// row's workgroup left) and the remainder tags of their edges.
__global__ __launch_bounds__(kThreads) void k_tiles_long_count(int64_t n, int64_t nnz, const int64_t* rowptr,
                                                               const int32_t* col, int T, int W,
                                                               const uint32_t* dense_bits, int32_t* sp_deg,
                                                               uint32_t* tag, uint32_t* row_of_e) {
    __shared__ int64_t s_red[kThreads / kWave];
    const int64_t chunks = long_chunks_of(nnz);
    for (int64_t ch = blockIdx.x; ch < chunks; ch += gridDim.x) {
        LongSeg seg[2];
        const int k = long_segments(rowptr, n, nnz, ch, seg);
        for (int j = 0; j < k; ++j) {
            const int64_t r = seg[j].row;
            const uint32_t* bits = dense_bits + (r / T) * W;
            int64_t total = 0;
            for (int64_t e0 = seg[j].a; e0 < seg[j].b; e0 += kThreads) {
                const int64_t e = e0 + threadIdx.x;
                bool sparse = false;
                if (e < seg[j].b) {
                    const int c = col[e];
                    sparse = !tile_is_dense(bits, c / T);
                    tag[e] = sparse ? uint32_t(c) : uint32_t(n);
                    row_of_e[e] = uint32_t(r);
                }
                int64_t t;
                block_flag_scan(sparse, s_red, &t);
                total += t;
            }
            if (threadIdx.x == 0 && total) atomicAdd(&sp_deg[r], int32_t(total));
        }
    }
}

// Fill pass of the long rows, first step: remainder edges per (chunk, segment).
__global__ __launch_bounds__(kThreads) void k_tiles_long_segs(int64_t n, int64_t nnz, const int64_t* rowptr,
                                                              const int32_t* col, int T, int W,
                                                              const uint32_t* dense_bits, int32_t* segcnt) {
    __shared__ int64_t s_red[kThreads / kWave];
    const int64_t chunks = long_chunks_of(nnz);
    for (int64_t ch = blockIdx.x; ch < chunks; ch += gridDim.x) {
        LongSeg seg[2];
        const int k = long_segments(rowptr, n, nnz, ch, seg);
        for (int j = 0; j < k; ++j) {
            const uint32_t* bits = dense_bits + (seg[j].row / T) * W;
            int64_t total = 0;
            for (int64_t e0 = seg[j].a; e0 < seg[j].b; e0 += kThreads) {
                const int64_t e = e0 + threadIdx.x;
                const bool sparse = e < seg[j].b && !tile_is_dense(bits, col[e] / T);
                int64_t t;
                block_flag_scan(sparse, s_red, &t);
                total += t;
            }
            if (threadIdx.x == 0) segcnt[2 * ch + seg[j].s] = int32_t(total);
        }
    }
}

// Fill pass of the long rows, second step: mask bits and remainder entries.
// segoff is the exclusive scan of segcnt; a row's entries before a segment are
// segoff[segment] - segoff[the row's first segment].
__global__ __launch_bounds__(kThreads) void k_tiles_long_fill(int64_t n, int64_t nnz, const int64_t* rowptr,
                                                              const int32_t* col, int T, int W,
                                                              const uint32_t* dense_bits,
                                                              const uint32_t* dense_pre, const int64_t* segoff,
                                                              const int64_t* tile_rowptr, uint32_t* tile_mask,
                                                              const int64_t* sp_rowptr, int32_t* sp_col,
                                                              int32_t* sp_pos, int32_t* tile_pos) {
    __shared__ int64_t s_red[kThreads / kWave];
    const int64_t chunks = long_chunks_of(nnz);
    const int wpr = T / 32;
    for (int64_t ch = blockIdx.x; ch < chunks; ch += gridDim.x) {
        LongSeg seg[2];
        const int k = long_segments(rowptr, n, nnz, ch, seg);
        for (int j = 0; j < k; ++j) {
            const int64_t r = seg[j].row;
            const int64_t I = r / T;
            const uint32_t* bits = dense_bits + I * W;
            const uint32_t* pre = dense_pre + I * W;
            const int64_t first = rowptr[r];
            const int64_t c0 = first / kLongRow;
            const int s0 = first == c0 * kLongRow ? 0 : 1;
            int64_t base = sp_rowptr[r] + segoff[2 * ch + seg[j].s] - segoff[2 * c0 + s0];
            for (int64_t e0 = seg[j].a; e0 < seg[j].b; e0 += kThreads) {
                const int64_t e = e0 + threadIdx.x;
                const bool valid = e < seg[j].b;
                const int c = valid ? col[e] : 0;
                const int J = c / T;
                const bool dense = valid && tile_is_dense(bits, J);
                const bool sparse = valid && !dense;
                int64_t t;
                const int64_t before = block_flag_scan(sparse, s_red, &t);
                if (dense) {
                    const uint32_t wd = bits[J >> 5];
                    const int64_t kk = tile_rowptr[I] + pre[J >> 5] + __popc(wd & ((1u << (J & 31)) - 1u));
                    const int cl = c - J * T;
                    atomicOr(&tile_mask[kk * int64_t(T) * wpr + (r - I * T) * wpr + cl / 32], 1u << (cl & 31));
                    if (tile_pos && (e == first || col[e - 1] / T != J)) tile_pos[kk * T + (r - I * T)] = int32_t(e);
                }
                if (sparse) {
                    const int64_t pos = base + before;
                    sp_col[pos] = c;
                    if (sp_pos) sp_pos[pos] = int32_t(e);
                }
                base += t;
            }
        }
    }
}

// flags[i] = value[i] > threshold
template <typename V>
__global__ void k_over(int64_t m, const V* value, int64_t threshold, int32_t* flags) {
    for (int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; e < m; e += int64_t(gridDim.x) * blockDim.x)
        flags[e] = int64_t(value[e]) > threshold ? 1 : 0;
}

// colptr[c] = the first position of a tag >= c in the sorted tags (c in [0, n]):
// the remainder transpose's column pointers, colptr[n] = the remainder size.
__global__ void k_col_ptr(int64_t n, int64_t nnz, const uint32_t* __restrict__ tag, int64_t* __restrict__ colptr) {
    for (int64_t c = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; c <= n; c += int64_t(gridDim.x) * blockDim.x) {
        int64_t lo = 0, hi = nnz;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (int64_t(tag[mid]) < c) lo = mid + 1;
            else hi = mid;
        }
        colptr[c] = lo;
    }
}

// flags[c] = the remainder column c holds more than threshold entries
__global__ void k_long_cols(int64_t n, const int64_t* colptr, int64_t threshold, int32_t* flags) {
    for (int64_t c = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; c < n; c += int64_t(gridDim.x) * blockDim.x)
        flags[c] = colptr[c + 1] - colptr[c] > threshold ? 1 : 0;
}

__global__ void k_compact_list(int64_t m, const int32_t* flags, const int64_t* pos, int32_t* list) {
    for (int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; e < m; e += int64_t(gridDim.x) * blockDim.x)
        if (flags[e]) list[pos[e]] = int32_t(e);
}

__global__ void k_u32_to_i32(int64_t m, const uint32_t* src, int32_t* dst) {
    for (int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; e < m; e += int64_t(gridDim.x) * blockDim.x)
        dst[e] = int32_t(src[e]);
}

constexpr int kRecordWords = 8;

struct TilesWs {
    uint32_t* flags;
    unsigned long long* csum;  // checksum of the count results (kept below); right after the record
    uint64_t* record;          // [kRecordWords]: what gt_tiles_count left here (CountRecord)
    int64_t* sizes;            // [4]: dense tiles, remainder edges, long rows, long columns
    uint32_t* tag;             // [nnz]: remainder tags (column, or n), sorted by the count pass
    uint32_t* counts;          // per tile column
    // The count results, one contiguous range of the workspace (kept_words
    // 8-byte words from kept_begin: dense_per_tilerow .. rows), so that
    // gt_build_tiles can take them from gt_tiles_count's workspace.  The
    // medium-row list is among them.
    int32_t* dense_per_tilerow;
    int32_t* sp_deg;
    int64_t* tmp_tile_rowptr;
    int64_t* tmp_sp_rowptr;
    int64_t* colptr;    // [n + 1]: the remainder transpose's column pointers
    int32_t* long_row_flag;
    int32_t* long_col_flag;
    int64_t* long_row_pos;
    int64_t* long_col_pos;
    uint32_t* dense_bits;  // [R, W]: the dense/sparse split of each tile row
    uint32_t* dense_pre;   // [R, W]: dense tiles before each word
    int32_t* heavy_slot;   // [R]: the heavy count row of each tile row, or -1
    int32_t* heavy_list;   // [kMaxHeavy]: the tile row of each heavy count row
    int32_t* heavy_n;      // how many heavy count rows
    uint32_t* heavy_cnt;   // [kMaxHeavy, R]: edges of each heavy tile row per tile column
    int32_t* med_list;     // [n]: the medium rows
    int64_t* med_info;     // [2]: their list start and number
    uint32_t* rows;        // [nnz]: the row of each edge, then (sorted with the tags) the remainder transpose's rows
    const uint64_t* kept_begin;
    int64_t kept_words;    // 8-byte words of the count results' range
    int8_t* med_cls;       // [n]: medium-row class of each row
    PartitionTmp part;
    int32_t* segcnt;       // [2 * long chunks]: remainder edges of each long-row segment
    int64_t* segoff;       // [2 * long chunks + 1]
    int W;
    ScanTmp scan;
    SortTmp sort;
};

TilesWs carve(Ws& ws, int64_t n, int64_t nnz, int32_t T) {
    TilesWs t;
    const int64_t n1 = n > 0 ? n : 1, e1 = nnz > 0 ? nnz : 1;
    const int64_t R = cdiv(n1, T > 0 ? T : 1);
    t.flags = ws.take<uint32_t>(1);
    // the record, then the checksum, then the plan sizes: read back with one copy each
    t.record = ws.take<uint64_t>(kRecordWords + 1 + 4);
    t.csum = reinterpret_cast<unsigned long long*>(t.record + kRecordWords);
    t.sizes = reinterpret_cast<int64_t*>(t.record + kRecordWords + 1);
    t.W = int(cdiv(R, 32));
    t.tag = ws.take<uint32_t>(e1);
    t.counts = ws.take<uint32_t>(n1 + 1);
    t.dense_per_tilerow = ws.take<int32_t>(R);
    t.sp_deg = ws.take<int32_t>(n1);
    t.tmp_tile_rowptr = ws.take<int64_t>(R + 1);
    t.tmp_sp_rowptr = ws.take<int64_t>(n1 + 1);
    t.colptr = ws.take<int64_t>(n1 + 1);
    t.long_row_flag = ws.take<int32_t>(n1);
    t.long_col_flag = ws.take<int32_t>(n1);
    t.long_row_pos = ws.take<int64_t>(n1 + 1);
    t.long_col_pos = ws.take<int64_t>(n1 + 1);
    t.dense_bits = ws.take<uint32_t>(size_t(R * t.W));
    t.dense_pre = ws.take<uint32_t>(size_t(R * t.W));
    t.heavy_slot = ws.take<int32_t>(size_t(R));
    t.heavy_list = ws.take<int32_t>(size_t(kMaxHeavy));
    t.heavy_n = ws.take<int32_t>(2);
    t.heavy_cnt = ws.take<uint32_t>(size_t(kMaxHeavy) * R);
    t.med_list = ws.take<int32_t>(size_t(n1 + (n1 & 1)));
    t.med_info = ws.take<int64_t>(2);
    t.rows = ws.take<uint32_t>(size_t(e1 + (e1 & 1)));  // an even count: the range ends on an 8-byte word
    {
        const char* b = reinterpret_cast<const char*>(t.dense_per_tilerow);
        const char* e = reinterpret_cast<const char*>(t.rows + e1 + (e1 & 1));
        t.kept_begin = reinterpret_cast<const uint64_t*>(t.dense_per_tilerow);
        t.kept_words = int64_t((e - b) / 8);
    }
    t.med_cls = ws.take<int8_t>(n1);
    t.part = partition_tmp(ws, n1);
    const int64_t segs = 2 * long_chunks_of(e1);
    t.segcnt = ws.take<int32_t>(size_t(segs));
    t.segoff = ws.take<int64_t>(size_t(segs + 1));
    t.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(n1 + 1 > segs + 1 ? n1 + 1 : segs + 1)));
    t.sort = sort_tmp(ws, e1, 4, true);
    return t;
}

// Checksum of the count results: the sum over the range's 8-byte words w_i of
// mix64(w_i + i * 0x9E3779B97F4A7C15) (mod 2^64, so the order of the sums does
// not matter); a changed or moved word changes it.
// The wavefront sums meet in LDS, so each workgroup adds one value to the
// total (a few hundred atomics on one address instead of one per wavefront).
constexpr int kCsumBlocks = 512;
constexpr int kCsumBatch = 8;
__global__ __launch_bounds__(256) void k_ws_checksum(const uint64_t* __restrict__ p, int64_t words,
                                                     unsigned long long* __restrict__ out) {
    __shared__ uint64_t s_part[256 / kWave];
    uint64_t acc = 0;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    // kCsumBatch words in flight per thread
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i + (kCsumBatch - 1) * stride < words; i += kCsumBatch * stride) {
        uint64_t x[kCsumBatch];
#pragma unroll
        for (int k = 0; k < kCsumBatch; ++k) x[k] = p[i + k * stride];
#pragma unroll
        for (int k = 0; k < kCsumBatch; ++k) acc += mix64(x[k] + uint64_t(i + k * stride) * 0x9E3779B97F4A7C15ull);
    }
    for (; i < words; i += stride) acc += mix64(p[i] + uint64_t(i) * 0x9E3779B97F4A7C15ull);
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const uint32_t lo = __shfl_xor(uint32_t(acc), o, kWave), hi = __shfl_xor(uint32_t(acc >> 32), o, kWave);
        acc += (uint64_t(hi) << 32) | lo;
    }
    if (lane_id() == 0) s_part[threadIdx.x / kWave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t t = 0;
#pragma unroll
        for (int w = 0; w < 256 / kWave; ++w) t += s_part[w];
        if (t) atomicAdd(out, (unsigned long long)t);
    }
}

gt_status ws_checksum(const TilesWs& t, hipStream_t s) {
    gt_status st = fill_u32(reinterpret_cast<uint32_t*>(t.csum), 2, 0u, s);
    if (st != GT_OK) return st;
    k_ws_checksum<<<grid_for(t.kept_words, 256, kCsumBlocks), 256, 0, s>>>(t.kept_begin, t.kept_words, t.csum);
    GT_LAUNCH_CHECK("tiles_checksum");
    return GT_OK;
}

// The dense tiles grouped by tile column for plans of at most
// kSmallTranspose tiles, in one workgroup: column counts in LDS, their scan
// (tileT_ptr), then the tiles placed in index order, 64 at a time by one
// wavefront.  A tile row holds at most one tile per column, and tile indices
// run in (I, J) order, so placing them in index order keeps each column's
// tiles in ascending I: within a 64-tile slice, a tile's rank among the
// slice's tiles of its column comes from comparing the slice's columns by
// readlane.
constexpr int kSmallTranspose = 8192;
constexpr int kTransposeThreads = 1024;
__global__ __launch_bounds__(kTransposeThreads) void k_tile_transpose(int64_t d, int R, const int32_t* tile_col,
                                                                      int64_t* tileT_ptr, int32_t* tileT_idx) {
    __shared__ int s_next[kMaxR];
    __shared__ int s_part[kTransposeThreads / kWave];
    for (int J = threadIdx.x; J < R; J += kTransposeThreads) s_next[J] = 0;
    __syncthreads();
    for (int64_t i = threadIdx.x; i < d; i += kTransposeThreads) atomicAdd(&s_next[tile_col[i]], 1);
    __syncthreads();
    // exclusive scan: each thread a run of `per` consecutive columns
    const int per = (R + kTransposeThreads - 1) / kTransposeThreads;
    const int j0 = threadIdx.x * per, j1 = j0 + per < R ? j0 + per : R;
    int sum = 0;
    for (int J = j0; J < j1; ++J) sum += s_next[J];
    const int lane = lane_id(), w = threadIdx.x / kWave;
    int x = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s_part[w] = x;
    __syncthreads();
    int before = x - sum;
    for (int k = 0; k < w; ++k) before += s_part[k];
    for (int J = j0; J < j1; ++J) {
        const int c = s_next[J];
        tileT_ptr[J] = before;
        s_next[J] = before;
        before += c;
    }
    if (threadIdx.x == 0) tileT_ptr[R] = d;
    __syncthreads();
    if (threadIdx.x >= kWave) return;
    for (int64_t base = 0; base < d; base += kWave) {
        const int64_t i = base + lane;
        const int J = i < d ? tile_col[i] : -1;
        int rank = 0, same = 0;
        for (int k = 0; k < kWave; ++k) {
            const int Jk = __builtin_amdgcn_readlane(J, k);
            if (Jk == J) {
                rank += k < lane ? 1 : 0;
                ++same;
            }
        }
        const int pos = J >= 0 ? s_next[J] + rank : 0;
        __builtin_amdgcn_wave_barrier();  // every lane has read its column's next slot
        if (J >= 0) {
            tileT_idx[pos] = int32_t(i);
            if (rank == same - 1) s_next[J] = pos + 1;  // the slice's last tile of the column
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// What gt_tiles_count leaves in its workspace, next to the count results: its
// arguments and the checksum of those results, written by the device after the
// checksum kernel.  gt_build_tiles with the same workspace and arguments takes
// the counts from there when the checksum still matches, and clears the
// record's tag (a record is used once).  The record lives in the caller's
// memory, so the library keeps nothing between the two calls.
constexpr uint64_t kRecordTag = 0x67745F74696C6573ull;
constexpr uint64_t kLongRowTag = 0x6C6F6E675F726F77ull;
struct CountRecord {
    uint64_t w[kRecordWords];  // tag, n, nnz, rowptr, col, T << 32 | tau_ppm, checksum, rows over kLongRow
};

// The plan's four sizes, next to each other for one copy to the host.
__global__ void k_plan_sizes(const int64_t* tile_rowptr_end, const int64_t* sp_rowptr_end,
                             const int64_t* long_row_end, const int64_t* long_col_end, int64_t* sizes) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    sizes[0] = *tile_rowptr_end;
    sizes[1] = *sp_rowptr_end;
    sizes[2] = *long_row_end;
    sizes[3] = *long_col_end;
}

__global__ void k_put_record(uint64_t* __restrict__ rec, int64_t n, int64_t nnz, const int64_t* rowptr,
                             const int32_t* col, int32_t T, uint32_t tau_ppm, const unsigned long long* __restrict__ sum,
                             bool has_long) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    rec[0] = kRecordTag;
    rec[1] = uint64_t(n);
    rec[2] = uint64_t(nnz);
    rec[3] = uint64_t(reinterpret_cast<uintptr_t>(rowptr));
    rec[4] = uint64_t(reinterpret_cast<uintptr_t>(col));
    rec[5] = (uint64_t(uint32_t(T)) << 32) | tau_ppm;
    // the long-row flag goes into the stored checksum too, so a changed flag fails the check
    rec[6] = uint64_t(*sum) ^ (has_long ? kLongRowTag : 0ull);
    rec[7] = has_long ? 1 : 0;
}

bool record_matches(const CountRecord& r, int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                    int32_t T, uint32_t tau_ppm) {
    return r.w[0] == kRecordTag && r.w[1] == uint64_t(n) && r.w[2] == uint64_t(nnz) &&
           r.w[3] == uint64_t(reinterpret_cast<uintptr_t>(rowptr)) &&
           r.w[4] == uint64_t(reinterpret_cast<uintptr_t>(col)) &&
           r.w[5] == ((uint64_t(uint32_t(T)) << 32) | tau_ppm);
}

gt_status check_common(const char* who, int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T,
                       void* ws_ptr, size_t ws_bytes) {
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << 32))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": n or nnz out of range");
    if (T != 64 && T != 128) return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": T must be 64 or 128");
    if (cdiv(n, T) > kMaxR)
        return fail(GT_ERR_UNSUPPORTED, std::string(who) + ": more than 16384 tile rows (n > 16384 * T)");
    if (!rowptr || (nnz > 0 && !col) || !ws_ptr) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null pointer");
    if (ws_bytes < gt_tiles_workspace_size(n, nnz, T))
        return fail(GT_ERR_WORKSPACE, std::string(who) + ": workspace too small");
    return GT_OK;
}

// Count pass shared by gt_tiles_count and gt_build_tiles: dense tiles per tile
// row (scanned into tile_rowptr), remainder degrees (scanned into sp_rowptr)
// and the long-row / long-column flags and positions.
inline unsigned long_grid(int64_t nnz) {
    const int64_t c = long_chunks_of(nnz);
    return unsigned(c < 8192 ? c : 8192);
}

// The list of rows of kShortRow + 1 to kLongRow edges (its length on the device, in med_info[1]).
gt_status medium_rows(int64_t n, const int64_t* rowptr, TilesWs& t, hipStream_t stream) {
    k_med_class<<<grid_for(n, 256, 8192), 256, 0, stream>>>(n, rowptr, t.med_cls);
    GT_LAUNCH_CHECK("tiles_medium_class");
    return partition_rows(t.med_cls, n, 1, t.med_list, t.med_info, t.part, stream);
}

// The heavy tile rows and their zeroed count rows: reads rowptr only, at
// positions clamped to [0, n], so it may run before the CSR check is read back.
gt_status heavy_prelude(int64_t n, const int64_t* rowptr, int32_t T, TilesWs& t, hipStream_t stream) {
    const int R = int(cdiv(n, T));
    k_heavy_slots<<<1, kTileThreads, 0, stream>>>(n, rowptr, T, R, t.heavy_slot, t.heavy_list, t.heavy_n);
    GT_LAUNCH_CHECK("tiles_heavy_slots");
    return fill_u32(t.heavy_cnt, int64_t(kMaxHeavy) * R, 0u, stream);
}

// The rest of the count pass, after heavy_prelude.
// has_long: some row has more than kLongRow entries (else the long-row kernel is skipped).
gt_status count_pass(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T, uint32_t tau_ppm,
                     TilesWs& t, int64_t* tile_rowptr, int64_t* sp_rowptr, bool has_long, hipStream_t stream) {
    gt_status st;
    const int R = int(cdiv(n, T));
    k_heavy_count<<<1024, kTileThreads, 0, stream>>>(n, rowptr, col, T, R, t.heavy_list, t.heavy_n, t.heavy_cnt);
    GT_LAUNCH_CHECK("tiles_heavy_count");
    k_tiles<false><<<R, kTileThreads, 0, stream>>>(n, rowptr, col, T, R, tau_ppm, t.dense_per_tilerow, t.sp_deg,
                                                   nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, t.tag,
                                                   t.rows, t.W, t.dense_bits, t.dense_pre, nullptr, nullptr,
                                                   t.heavy_slot, t.heavy_cnt);
    GT_LAUNCH_CHECK("tiles_count");
    if ((st = medium_rows(n, rowptr, t, stream)) != GT_OK) return st;
    k_tiles_med<false><<<grid_for(n, 4, 16384), 256, 0, stream>>>(
        n, t.med_list, t.med_info + 1, rowptr, col, T, t.W, t.dense_bits, t.dense_pre, t.sp_deg, t.tag, t.rows,
        nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    GT_LAUNCH_CHECK("tiles_count_medium");
    if (has_long) {
        k_tiles_long_count<<<long_grid(nnz), kThreads, 0, stream>>>(n, nnz, rowptr, col, T, t.W, t.dense_bits,
                                                                   t.sp_deg, t.tag, t.rows);
        GT_LAUNCH_CHECK("tiles_long_count");
    }
    if ((st = exclusive_scan_i32(t.dense_per_tilerow, R, tile_rowptr, t.scan, stream)) != GT_OK) return st;
    if ((st = exclusive_scan_i32(t.sp_deg, n, sp_rowptr, t.scan, stream)) != GT_OK) return st;
    // the remainder transpose: (tag, row) pairs in CSR order, stably sorted by tag
    if (nnz > 0 && (st = radix_sort_u32(t.tag, t.rows, nnz, bits_for(n + 1), t.sort, stream)) != GT_OK) return st;
    const unsigned g = grid_for(n, 256, 8192);
    k_col_ptr<<<grid_for(n + 1, 256, 8192), 256, 0, stream>>>(n, nnz, t.tag, t.colptr);
    GT_LAUNCH_CHECK("tiles_colptr");
    k_over<int32_t><<<g, 256, 0, stream>>>(n, t.sp_deg, GT_LONG_ROW, t.long_row_flag);
    GT_LAUNCH_CHECK("tiles_long_rows");
    k_long_cols<<<g, 256, 0, stream>>>(n, t.colptr, GT_LONG_ROW, t.long_col_flag);
    GT_LAUNCH_CHECK("tiles_long_cols");
    if ((st = exclusive_scan_i32(t.long_row_flag, n, t.long_row_pos, t.scan, stream)) != GT_OK) return st;
    if ((st = exclusive_scan_i32(t.long_col_flag, n, t.long_col_pos, t.scan, stream)) != GT_OK) return st;
    return GT_OK;
}

}  // namespace
}  // namespace gt

using namespace gt;

extern "C" size_t gt_tiles_workspace_size(int64_t n, int64_t nnz, int32_t T) {
    Ws ws(nullptr);
    carve(ws, n, nnz, T);
    return ws.size();
}

extern "C" gt_status gt_tiles_count(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T,
                                    uint32_t tau_ppm, gt_tiles* plan, void* ws_ptr, size_t ws_bytes,
                                    hipStream_t stream) {
    gt_status st = check_common("gt_tiles_count", n, nnz, rowptr, col, T, ws_ptr, ws_bytes);
    if (st != GT_OK) return st;
    if (!plan) return fail(GT_ERR_INVALID_ARG, "gt_tiles_count: null plan");
    plan->n = n;
    plan->T = T;
    plan->n_row_tiles = n > 0 ? cdiv(n, T) : 0;
    plan->n_dense = plan->nnz_sparse = plan->n_long_rows = plan->n_long_cols = 0;
    if (n == 0) return GT_OK;
    Ws ws(ws_ptr);
    TilesWs t = carve(ws, n, nnz, T);
    if ((st = launch_validate_csr(n, nnz, rowptr, col, t.flags, stream)) != GT_OK) return st;
    if ((st = heavy_prelude(n, rowptr, T, t, stream)) != GT_OK) return st;
    uint32_t vf = 0;
    GT_HIP(hipMemcpyAsync(&vf, t.flags, sizeof(vf), hipMemcpyDeviceToHost, stream));
    GT_HIP(hipStreamSynchronize(stream));
    if ((st = validation_result(vf)) != GT_OK) return st;
    const bool has_long = (vf & kLongRowSeen) != 0;
    if ((st = count_pass(n, nnz, rowptr, col, T, tau_ppm, t, t.tmp_tile_rowptr, t.tmp_sp_rowptr, has_long,
                         stream)) != GT_OK)
        return st;
    if ((st = ws_checksum(t, stream)) != GT_OK) return st;
    k_put_record<<<1, 64, 0, stream>>>(t.record, n, nnz, rowptr, col, T, tau_ppm, t.csum, has_long);
    GT_LAUNCH_CHECK("tiles_count_record");
    const int64_t R = plan->n_row_tiles;
    k_plan_sizes<<<1, 64, 0, stream>>>(t.tmp_tile_rowptr + R, t.tmp_sp_rowptr + n, t.long_row_pos + n,
                                       t.long_col_pos + n, t.sizes);
    GT_LAUNCH_CHECK("tiles_sizes");
    int64_t h[4] = {0, 0, 0, 0};
    GT_HIP(hipMemcpyAsync(h, t.sizes, sizeof(h), hipMemcpyDeviceToHost, stream));
    GT_HIP(hipStreamSynchronize(stream));
    plan->n_dense = h[0];
    plan->nnz_sparse = h[1];
    plan->n_long_rows = h[2];
    plan->n_long_cols = h[3];
    return GT_OK;
}

extern "C" gt_status gt_build_tiles(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T,
                                    uint32_t tau_ppm, gt_tiles* plan, void* ws_ptr, size_t ws_bytes,
                                    hipStream_t stream) {
    gt_status st = check_common("gt_build_tiles", n, nnz, rowptr, col, T, ws_ptr, ws_bytes);
    if (st != GT_OK) return st;
    if (!plan) return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: null plan");
    if (plan->n != n || plan->T != T) return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: plan->n / plan->T mismatch");
    if (plan->n_dense < 0 || plan->nnz_sparse < 0 || plan->n_dense > nnz || plan->nnz_sparse > nnz ||
        plan->n_long_rows < 0 || plan->n_long_cols < 0 || plan->n_long_rows > n || plan->n_long_cols > n)
        return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: plan sizes out of range");
    if ((plan->n_long_rows > 0 && !plan->long_rows) || (plan->n_long_cols > 0 && !plan->long_cols))
        return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: null long-row list");
    if (!plan->tile_rowptr || !plan->sp_rowptr || !plan->sp_colptr || !plan->tileT_ptr ||
        (plan->n_dense > 0 && (!plan->tile_col || !plan->tile_nnz || !plan->tile_mask || !plan->tileT_idx)) ||
        (plan->nnz_sparse > 0 && (!plan->sp_col || !plan->sp_row)))
        return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: null plan array");
    if ((plan->sp_pos || plan->tile_pos) && nnz >= (int64_t(1) << 31))
        return fail(GT_ERR_INVALID_ARG, "gt_build_tiles: edge positions need nnz < 2^31");
    const int R = n > 0 ? int(cdiv(n, T)) : 0;
    plan->n_row_tiles = R;
    if (n == 0) {
        if ((st = fill_i64(plan->tile_rowptr, 1, 0, stream)) != GT_OK) return st;
        if ((st = fill_i64(plan->tileT_ptr, 1, 0, stream)) != GT_OK) return st;
        if ((st = fill_i64(plan->sp_rowptr, 1, 0, stream)) != GT_OK) return st;
        return fill_i64(plan->sp_colptr, 1, 0, stream);
    }
    Ws ws(ws_ptr);
    TilesWs t = carve(ws, n, nnz, T);
    // the counts of the gt_tiles_count call that used this workspace with these
    // arguments, if they are still there unchanged; else count again
    bool reuse = false;
    bool has_long = nnz > kLongRow;  // without the count call's record: whether the CSR has a row that long
    {
        if ((st = ws_checksum(t, stream)) != GT_OK) return st;
        uint64_t words[kRecordWords + 1];  // the record and the checksum just taken
        GT_HIP(hipMemcpyAsync(words, t.record, sizeof(words), hipMemcpyDeviceToHost, stream));
        GT_HIP(hipStreamSynchronize(stream));
        CountRecord rec;
        for (int i = 0; i < kRecordWords; ++i) rec.w[i] = words[i];
        const uint64_t have = words[kRecordWords];
        reuse = record_matches(rec, n, nnz, rowptr, col, T, tau_ppm) && rec.w[7] <= 1 &&
                rec.w[6] == (have ^ (rec.w[7] ? kLongRowTag : 0ull));
        if (reuse) has_long = rec.w[7] != 0;
        if (!reuse && rec.w[0] == kRecordTag &&
            (st = fill_u32(reinterpret_cast<uint32_t*>(t.record), 2, 0u, stream)) != GT_OK)
            return st;
    }
    if (!reuse) {
        if ((st = heavy_prelude(n, rowptr, T, t, stream)) != GT_OK) return st;
        if ((st = count_pass(n, nnz, rowptr, col, T, tau_ppm, t, plan->tile_rowptr, plan->sp_rowptr, has_long,
                             stream)) !=
            GT_OK)
            return st;
    }
    // the fill reads the offsets where the count pass left them; the plan's copies and the other small
    // launches follow the fill's first kernel, so that kernel starts right after the check above
    const int64_t* trp = reuse ? t.tmp_tile_rowptr : plan->tile_rowptr;
    const int64_t* srp = reuse ? t.tmp_sp_rowptr : plan->sp_rowptr;
    const int64_t words = plan->n_dense * int64_t(T) * (T / 32);
    if ((st = fill_u32(plan->tile_mask, words, 0u, stream)) != GT_OK) return st;
    if (plan->tile_pos && plan->n_dense > 0 &&
        (st = fill_u32(reinterpret_cast<uint32_t*>(plan->tile_pos), plan->n_dense * T, 0u, stream)) != GT_OK)
        return st;
    k_tiles<true><<<R, kTileThreads, 0, stream>>>(n, rowptr, col, T, R, tau_ppm, nullptr, nullptr, trp,
                                              plan->tile_col, plan->tile_nnz, plan->tile_mask, srp, plan->sp_col,
                                              nullptr, nullptr, t.W, nullptr, nullptr, plan->sp_pos, plan->tile_pos,
                                              t.heavy_slot, t.heavy_cnt);
    GT_LAUNCH_CHECK("tiles_fill");
    if (reuse) {
        if ((st = fill_u32(reinterpret_cast<uint32_t*>(t.record), 2, 0u, stream)) != GT_OK) return st;  // used once
        if ((st = copy_bytes(plan->tile_rowptr, t.tmp_tile_rowptr, size_t(R + 1) * 8, stream)) != GT_OK) return st;
        if ((st = copy_bytes(plan->sp_rowptr, t.tmp_sp_rowptr, size_t(n + 1) * 8, stream)) != GT_OK) return st;
    }
    {
        const unsigned g = grid_for(n, 256, 8192);
        if (plan->n_long_rows > 0) {
            k_compact_list<<<g, 256, 0, stream>>>(n, t.long_row_flag, t.long_row_pos, plan->long_rows);
            GT_LAUNCH_CHECK("tiles_long_row_list");
        }
        if (plan->n_long_cols > 0) {
            k_compact_list<<<g, 256, 0, stream>>>(n, t.long_col_flag, t.long_col_pos, plan->long_cols);
            GT_LAUNCH_CHECK("tiles_long_col_list");
        }
    }
    // the medium-row list: the count pass made it (here, or in gt_tiles_count's workspace, checked above)
    k_tiles_med<true><<<grid_for(n, 4, 16384), 256, 0, stream>>>(
        n, t.med_list, t.med_info + 1, rowptr, col, T, t.W, t.dense_bits, t.dense_pre, nullptr, nullptr, nullptr,
        trp, plan->tile_mask, srp, plan->sp_col, plan->sp_pos, plan->tile_pos);
    GT_LAUNCH_CHECK("tiles_fill_medium");
    if (has_long) {
        const int64_t segs = 2 * long_chunks_of(nnz);
        if ((st = fill_u32(reinterpret_cast<uint32_t*>(t.segcnt), segs, 0u, stream)) != GT_OK) return st;
        k_tiles_long_segs<<<long_grid(nnz), kThreads, 0, stream>>>(n, nnz, rowptr, col, T, t.W, t.dense_bits,
                                                                  t.segcnt);
        GT_LAUNCH_CHECK("tiles_long_segs");
        if ((st = exclusive_scan_i32(t.segcnt, segs, t.segoff, t.scan, stream)) != GT_OK) return st;
        k_tiles_long_fill<<<long_grid(nnz), kThreads, 0, stream>>>(
            n, nnz, rowptr, col, T, t.W, t.dense_bits, t.dense_pre, t.segoff, trp, plan->tile_mask, srp,
            plan->sp_col, plan->sp_pos, plan->tile_pos);
        GT_LAUNCH_CHECK("tiles_long_fill");
    }
    // remainder transpose: the count pass sorted it; its first nnz_sparse rows are the remainder's
    const int64_t m = plan->nnz_sparse;
    if (m > 0) {
        k_u32_to_i32<<<grid_for(m, 256, 16384), 256, 0, stream>>>(m, t.rows, plan->sp_row);
        GT_LAUNCH_CHECK("tiles_sp_row");
    }
    if ((st = copy_bytes(plan->sp_colptr, t.colptr, size_t(n + 1) * 8, stream)) != GT_OK) return st;
    // tiles grouped by column: stable sort of (J, tile index) by J
    const int64_t d = plan->n_dense;
    if (d <= kSmallTranspose) {
        k_tile_transpose<<<1, kTransposeThreads, 0, stream>>>(d, R, plan->tile_col, plan->tileT_ptr,
                                                              plan->tileT_idx);
        GT_LAUNCH_CHECK("tiles_tileT_small");
        return GT_OK;
    }
    if ((st = fill_u32(t.counts, R, 0u, stream)) != GT_OK) return st;
    if (d > 0) {
        if ((st = count_keys(plan->tile_col, d, t.counts, stream)) != GT_OK) return st;
        // t.tag and t.rows are free once sp_row is out
        if ((st = copy_bytes(t.tag, plan->tile_col, d * 4, stream)) != GT_OK) return st;
        if ((st = iota_u32(t.rows, d, stream)) != GT_OK) return st;
        if ((st = radix_sort_u32(t.tag, t.rows, d, bits_for(R), t.sort, stream)) != GT_OK) return st;
        k_u32_to_i32<<<grid_for(d, 256, 16384), 256, 0, stream>>>(d, t.rows, plan->tileT_idx);
        GT_LAUNCH_CHECK("tiles_tileT");
    }
    if ((st = exclusive_scan_u32(t.counts, R, plan->tileT_ptr, t.scan, stream)) != GT_OK) return st;
    return GT_OK;
}

// CSC -> CSR position map of the remainder: the same stable sort by column
// that orders the transpose, carrying each edge's remainder position, then
// mapped to the input CSR through sp_pos when the plan has it.
__global__ void k_map_positions(int64_t m, const uint32_t* rem, const int32_t* sp_pos, int32_t* out) {
    for (int64_t e = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; e < m; e += int64_t(gridDim.x) * blockDim.x)
        out[e] = sp_pos ? sp_pos[rem[e]] : int32_t(rem[e]);
}

static size_t edge_map_ws(int64_t m) {
    Ws ws(nullptr);
    const int64_t e1 = m > 0 ? m : 1;
    ws.take<uint32_t>(e1);
    ws.take<uint32_t>(e1);
    sort_tmp(ws, e1, 4, true);
    return ws.size();
}

extern "C" size_t gt_edge_map_workspace_size(const gt_tiles* plan) {
    if (!plan) return 0;
    return edge_map_ws(plan->nnz_sparse);
}

extern "C" gt_status gt_edge_map(const gt_tiles* plan, int32_t* csc_pos, void* ws_ptr, size_t ws_bytes,
                                 hipStream_t stream) {
    if (!plan) return fail(GT_ERR_INVALID_ARG, "gt_edge_map: null plan");
    const int64_t n = plan->n, m = plan->nnz_sparse;
    if (n < 0 || n >= (int64_t(1) << 31) || m < 0 || m >= (int64_t(1) << 31))
        return fail(GT_ERR_INVALID_ARG, "gt_edge_map: n or nnz_sparse out of range");
    if (m == 0) return GT_OK;
    if (!plan->sp_col || !csc_pos || !ws_ptr) return fail(GT_ERR_INVALID_ARG, "gt_edge_map: null pointer");
    if (ws_bytes < edge_map_ws(m)) return fail(GT_ERR_WORKSPACE, "gt_edge_map: workspace too small");
    Ws ws(ws_ptr);
    uint32_t* keys = ws.take<uint32_t>(m);
    uint32_t* vals = ws.take<uint32_t>(m);
    SortTmp sort = sort_tmp(ws, m, 4, true);
    gt_status st;
    if ((st = copy_bytes(keys, plan->sp_col, m * 4, stream)) != GT_OK) return st;
    if ((st = iota_u32(vals, m, stream)) != GT_OK) return st;
    if ((st = radix_sort_u32(keys, vals, m, bits_for(n), sort, stream)) != GT_OK) return st;
    k_map_positions<<<grid_for(m, 256, 16384), 256, 0, stream>>>(m, vals, plan->sp_pos, csc_pos);
    GT_LAUNCH_CHECK("edge_map");
    return GT_OK;
}
