// Relabelling of the CSR by a node permutation (§3.3: the layout is
// reorganised by cluster once the full sequence is on the device), and row
// gathers/scatters of feature tensors.
//
// Rows move whole to their new place, so only each row's relabelled columns
// need sorting.  A row of at most kShortRow entries is sorted by a group of
// 4, 8, 16, 32 or 64 lanes of a wavefront (a bitonic network across the
// group's lanes; the row classes come from one stable partition of the new
// rows), a row of up to kWaveRow entries by one wavefront (2, 4 or 8 entries
// per lane), and written straight to its place.  The longer rows' edges are
// packed as keys (rank of the new row among them << B) | new column and put
// in order by one stable radix sort: sorted, they are grouped by new row and
// ascending inside each row, each at its rank inside the row.
#include "lanes.h"
#include "prim.h"

namespace gt {
namespace {

constexpr int kShortRow = 64;  // rows sorted by a group of lanes
constexpr int kWaveRow = 512;  // rows sorted by one wavefront, kWaveRow / 64 entries per lane

// Row classes of the relabelling: rows of 1-4, 5-8, 9-16, 17-32 and 33-64
// entries (sorted by lane groups), 65 to kWaveRow (one wavefront each),
// kWaveRow + 1 to kLongRow entries (keys written by one wavefront per row);
// empty rows and rows over kLongRow are in no list.
enum { kRl4, kRl8, kRl16, kRl32, kRl64, kRlWave, kRlMed, kRlClasses };

__device__ __forceinline__ int8_t relabel_class(int64_t d) {
    return d <= 0 ? int8_t(-1)
           : d <= 4 ? int8_t(kRl4)
           : d <= 8 ? int8_t(kRl8)
           : d <= 16 ? int8_t(kRl16)
           : d <= 32 ? int8_t(kRl32)
           : d <= kShortRow ? int8_t(kRl64)
           : d <= kWaveRow ? int8_t(kRlWave)
           : d <= kLongRow ? int8_t(kRlMed)
                           : int8_t(-1);
}

// Entry count of every new row r (old row perm[r]), its class, the entries it
// sends to the radix sort (its count when longer than kWaveRow, else 0) and
// whether it sends any.
__global__ void k_new_degrees(int64_t n, const int64_t* rowptr, const int32_t* perm, int64_t* deg_new, int8_t* cls,
                              int64_t* sdeg, int32_t* sflag) {
    for (int64_t r = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; r < n; r += int64_t(gridDim.x) * blockDim.x) {
        const int64_t u = perm[r];
        const int64_t d = rowptr[u + 1] - rowptr[u];
        deg_new[r] = d;
        cls[r] = relabel_class(d);
        sdeg[r] = d > kWaveRow ? d : 0;
        sflag[r] = d > kWaveRow ? 1 : 0;
    }
}

// srow[srank[r]] = r for the rows that send entries to the radix sort.
__global__ void k_sorted_rows(int64_t n, const int32_t* sflag, const int64_t* srank, int32_t* srow) {
    for (int64_t r = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; r < n; r += int64_t(gridDim.x) * blockDim.x)
        if (sflag[r]) srow[srank[r]] = int32_t(r);
}

// Rows of kShortRow + 1 to kWaveRow entries, one wavefront each: element
// i = 64 k + lane of the row sits in register k of the lane, R registers
// (N = 64 R >= the row's entries; padding sorts last).  A bitonic network over
// the N elements: exchanges across lanes by lane permutes, across registers
// inside the lane.
template <int R, bool kMap>
__device__ __forceinline__ void relabel_wave_row(int64_t r, int64_t a, int d, const int32_t* __restrict__ col,
                                                 const int32_t* __restrict__ iperm,
                                                 const int64_t* __restrict__ rowptr_out,
                                                 int32_t* __restrict__ col_out, int32_t* __restrict__ src_pos) {
    constexpr int N = kWave * R;
    const int lane = lane_id();
    uint32_t key[R], pos[R];
    int c[R];
#pragma unroll
    for (int k = 0; k < R; ++k) c[k] = kWave * k + lane < d ? col[a + kWave * k + lane] : 0;
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const bool in = kWave * k + lane < d;
        key[k] = in ? uint32_t(iperm[c[k]]) : 0xFFFFFFFFu;
        pos[k] = uint32_t(a + kWave * k + lane);
    }
#pragma unroll
    for (int sz = 2; sz <= N; sz <<= 1) {
#pragma unroll
        for (int j = sz >> 1; j > 0; j >>= 1) {
            if (j >= kWave) {  // partner: register k ^ (j / 64) of the same lane
#pragma unroll
                for (int k = 0; k < R; ++k) {
                    const int kk = k ^ (j / kWave);
                    if (kk < k) continue;
                    const bool up = ((kWave * k + lane) & sz) == 0;  // ascending block
                    const bool swap = up ? key[kk] < key[k] : key[kk] > key[k];
                    if (swap) {
                        const uint32_t tk = key[k], tp = pos[k];
                        key[k] = key[kk];
                        pos[k] = pos[kk];
                        key[kk] = tk;
                        pos[kk] = tp;
                    }
                }
            } else {  // partner: lane ^ j, same register
#pragma unroll
                for (int k = 0; k < R; ++k) {
                    const int i = kWave * k + lane;
                    const uint32_t ok = uint32_t(xor_lane_pow2(int(key[k]), j));
                    const uint32_t op = kMap ? uint32_t(xor_lane_pow2(int(pos[k]), j)) : 0u;
                    const bool take_min = ((i & j) == 0) == ((i & sz) == 0);
                    if (take_min ? ok < key[k] : ok > key[k]) {
                        key[k] = ok;
                        pos[k] = op;
                    }
                }
            }
        }
    }
    const int64_t o = rowptr_out[r];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int i = kWave * k + lane;
        if (i < d) {
            col_out[o + i] = int32_t(key[k]);
            if (kMap) src_pos[o + i] = int32_t(pos[k]);
        }
    }
}

template <bool kMap>
__global__ __launch_bounds__(256) void k_relabel_wave(const int32_t* __restrict__ list, int64_t len,
                                                      const int64_t* __restrict__ rowptr,
                                                      const int32_t* __restrict__ col,
                                                      const int32_t* __restrict__ perm,
                                                      const int32_t* __restrict__ iperm,
                                                      const int64_t* __restrict__ rowptr_out,
                                                      int32_t* __restrict__ col_out, int32_t* __restrict__ src_pos) {
    const int64_t waves = int64_t(gridDim.x) * (256 / kWave);
    for (int64_t idx = int64_t(blockIdx.x) * (256 / kWave) + threadIdx.x / kWave; idx < len; idx += waves) {
        const int64_t r = list[idx];
        const int64_t u = perm[r];
        const int64_t a = rowptr[u];
        const int d = int(rowptr[u + 1] - a);  // kShortRow < d <= kWaveRow, uniform over the wavefront
        if (d <= 2 * kWave)
            relabel_wave_row<2, kMap>(r, a, d, col, iperm, rowptr_out, col_out, src_pos);
        else if (d <= 4 * kWave)
            relabel_wave_row<4, kMap>(r, a, d, col, iperm, rowptr_out, col_out, src_pos);
        else
            relabel_wave_row<8, kMap>(r, a, d, col, iperm, rowptr_out, col_out, src_pos);
    }
}

// The rows of one class list of at most S entries, 64 / S per wavefront: the
// lanes of a row's group hold iperm of its columns (padding sorts last) and,
// for the edge map, their old CSR positions; a bitonic network over the S
// lanes sorts them ascending (the columns of a row are distinct), exchanging
// by quad permutes and lane swizzles with every lane active.
template <int S, bool kMap>
__device__ __forceinline__ void relabel_rows(const int32_t* __restrict__ list, int64_t len, unsigned blk,
                                             unsigned nblk, const int64_t* __restrict__ rowptr,
                                             const int32_t* __restrict__ col, const int32_t* __restrict__ perm,
                                             const int32_t* __restrict__ iperm,
                                             const int64_t* __restrict__ rowptr_out, int32_t* __restrict__ col_out,
                                             int32_t* __restrict__ src_pos) {
    constexpr int G = kWave / S;
    const int lane = lane_id(), sub = lane / S, sl = lane % S;
    const int64_t waves = int64_t(nblk) * (256 / kWave);
    for (int64_t base = (int64_t(blk) * (256 / kWave) + threadIdx.x / kWave) * G; base < len; base += waves * G) {
        const int64_t idx = base + sub;
        int64_t r = -1, a = 0;
        int d = 0;
        if (idx < len) {
            r = list[idx];
            const int64_t u = perm[r];
            a = rowptr[u];
            d = int(rowptr[u + 1] - a);
        }
        uint32_t key = 0xFFFFFFFFu, pos = 0u;
        if (sl < d) {
            key = uint32_t(iperm[col[a + sl]]);
            pos = uint32_t(a + sl);
        }
#pragma unroll
        for (int k = 2; k <= S; k <<= 1) {
#pragma unroll
            for (int j = k >> 1; j > 0; j >>= 1) {
                const uint32_t ok = uint32_t(xor_lane_pow2(int(key), j));
                const uint32_t op = kMap ? uint32_t(xor_lane_pow2(int(pos), j)) : 0u;
                const bool take_min = ((sl & j) == 0) == ((sl & k) == 0);
                if (take_min ? ok < key : ok > key) {
                    key = ok;
                    pos = op;
                }
            }
        }
        if (sl < d) {
            const int64_t o = rowptr_out[r] + sl;
            col_out[o] = int32_t(key);
            if (kMap) src_pos[o] = int32_t(pos);
        }
    }
}

// The five short-row lists in one launch: the grid's blocks are cut into five
// consecutive ranges, one per list (first[5] is the grid).
struct ShortLists {
    const int32_t* list[5];
    int64_t len[5];
    unsigned first[6];
};

template <bool kMap>
__global__ __launch_bounds__(256) void k_relabel_short(ShortLists sl, const int64_t* __restrict__ rowptr,
                                                       const int32_t* __restrict__ col,
                                                       const int32_t* __restrict__ perm,
                                                       const int32_t* __restrict__ iperm,
                                                       const int64_t* __restrict__ rowptr_out,
                                                       int32_t* __restrict__ col_out, int32_t* __restrict__ src_pos) {
    const unsigned b = blockIdx.x;
    int k = 0;
    while (k + 1 < 5 && b >= sl.first[k + 1]) ++k;
    const unsigned blk = b - sl.first[k], nblk = sl.first[k + 1] - sl.first[k];
    switch (k) {
        case 0:
            relabel_rows<64, kMap>(sl.list[0], sl.len[0], blk, nblk, rowptr, col, perm, iperm, rowptr_out, col_out,
                                   src_pos);
            break;
        case 1:
            relabel_rows<32, kMap>(sl.list[1], sl.len[1], blk, nblk, rowptr, col, perm, iperm, rowptr_out, col_out,
                                   src_pos);
            break;
        case 2:
            relabel_rows<16, kMap>(sl.list[2], sl.len[2], blk, nblk, rowptr, col, perm, iperm, rowptr_out, col_out,
                                   src_pos);
            break;
        case 3:
            relabel_rows<8, kMap>(sl.list[3], sl.len[3], blk, nblk, rowptr, col, perm, iperm, rowptr_out, col_out,
                                  src_pos);
            break;
        default:
            relabel_rows<4, kMap>(sl.list[4], sl.len[4], blk, nblk, rowptr, col, perm, iperm, rowptr_out, col_out,
                                  src_pos);
            break;
    }
}

// The sorted rows' entry count, the CSR check's flags and the number of
// sorted rows, after the class starts and sizes, so that one copy brings all
// of them to the host.
__global__ void k_host_words(const int64_t* sorted, const uint32_t* flags, const int64_t* sorted_rows,
                             int64_t* out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    out[0] = *sorted;
    out[1] = int64_t(*flags);
    out[2] = *sorted_rows;
}

// Keys of the listed rows (kWaveRow + 1 to kLongRow entries), one wavefront
// per new row, at the row's offset soff[r] among the sorted rows' entries,
// with the row's rank srank[r] among the sorted rows; for the edge map, the
// old CSR position as the value.
template <bool kMap>
__global__ __launch_bounds__(256) void k_edge_keys(const int32_t* list, int64_t len, const int64_t* rowptr,
                                                   const int32_t* col, const int32_t* perm, const int32_t* iperm,
                                                   int bits, const int64_t* soff, const int64_t* srank,
                                                   uint64_t* keys, uint32_t* vals) {
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t idx = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave; idx < len; idx += waves) {
        const int64_t r = list[idx];
        const int64_t u = perm[r];
        const int64_t a = rowptr[u], d = rowptr[u + 1] - a;
        const uint64_t hi = uint64_t(srank[r]) << bits;
        const int64_t base = soff[r];
        for (int64_t e = lane; e < d; e += kWave) {
            keys[base + e] = hi | uint64_t(uint32_t(iperm[col[a + e]]));
            if (kMap) vals[base + e] = uint32_t(a + e);
        }
    }
}

// The keys of the rows of more than kLongRow entries, chunk by chunk over the grid.
template <bool kMap>
__global__ __launch_bounds__(256) void k_edge_keys_long(int64_t n, int64_t nnz, const int64_t* rowptr,
                                                        const int32_t* col, const int32_t* iperm, int bits,
                                                        const int64_t* soff, const int64_t* srank, uint64_t* keys,
                                                        uint32_t* vals) {
    const int64_t chunks = long_chunks_of(nnz);
    for (int64_t c = blockIdx.x; c < chunks; c += gridDim.x) {
        LongSeg seg[2];
        const int k = long_segments(rowptr, n, nnz, c, seg);
        for (int j = 0; j < k; ++j) {
            const int64_t r = iperm[seg[j].row];
            const uint64_t hi = uint64_t(srank[r]) << bits;
            const int64_t shift = soff[r] - rowptr[seg[j].row];  // key position = soff[r] + (e - row start)
            for (int64_t e = seg[j].a + threadIdx.x; e < seg[j].b; e += blockDim.x) {
                keys[shift + e] = hi | uint64_t(uint32_t(iperm[col[e]]));
                if (kMap) vals[shift + e] = uint32_t(e);
            }
        }
    }
}

// Sorted key i of new row r (rank key >> bits among the sorted rows) goes to
// rank i - soff[r] inside the row.
__global__ void k_place_sorted(int64_t m, const uint64_t* keys, const uint32_t* vals, int bits, const int64_t* soff,
                               const int32_t* srow, const int64_t* rowptr_out, int32_t* col_out, int32_t* src_pos) {
    const uint64_t mask = (uint64_t(1) << bits) - 1;
    for (int64_t i = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; i < m; i += int64_t(gridDim.x) * blockDim.x) {
        const uint64_t key = keys[i];
        const int64_t r = srow[key >> bits];
        const int64_t o = rowptr_out[r] + (i - soff[r]);
        col_out[o] = int32_t(key & mask);
        if (src_pos) src_pos[o] = int32_t(vals[i]);
    }
}

// Rows of fewer than 32 dwords (per-edge values): one lane per dword.
template <bool kGather>
__global__ __launch_bounds__(256) void k_move_small_rows(int64_t n, int32_t words, const uint32_t* src,
                                                         const int32_t* perm, uint32_t* dst) {
    const int64_t total = n * words;
    for (int64_t x = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; x < total; x += int64_t(gridDim.x) * blockDim.x) {
        const int64_t r = x / words, w = x - r * words;
        const int64_t p = perm[r];
        if (kGather)
            dst[x] = src[p * words + w];
        else
            dst[p * words + w] = src[x];
    }
}

// Rows of a multiple of 16 bytes: one 16-byte vector per lane, consecutive lanes
// on consecutive vectors of a row (rows of 512 bytes: two per wavefront).
template <bool kGather, typename I>
__global__ __launch_bounds__(256) void k_move_rows16(I n, I vpr, const uint4* __restrict__ src,
                                                     const int32_t* __restrict__ perm, uint4* __restrict__ dst) {
    const I total = n * vpr;
    const I stride = I(gridDim.x) * I(blockDim.x);
    for (I x = I(blockIdx.x) * I(blockDim.x) + I(threadIdx.x); x < total; x += stride) {
        const I r = x / vpr, w = x - r * vpr;
        const I p = I(perm[r]);
        if (kGather)
            dst[x] = src[p * vpr + w];
        else
            dst[p * vpr + w] = src[x];
    }
}

// One wavefront per row; dwords per lane.
template <bool kGather>
__global__ __launch_bounds__(256) void k_move_rows(int64_t n, int64_t words, const uint32_t* src,
                                                   const int32_t* perm, uint32_t* dst) {
    const int lane = lane_id();
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t r = int64_t(blockIdx.x) * 4 + threadIdx.x / kWave; r < n; r += waves) {
        const int64_t p = perm[r];
        const uint32_t* s = src + (kGather ? p : r) * words;
        uint32_t* d = dst + (kGather ? r : p) * words;
        for (int64_t w = lane; w < words; w += kWave) d[w] = s[w];
    }
}

struct PermuteWs {
    uint32_t* flags;
    int64_t* deg_new;
    int8_t* cls;      // [n]: the relabelling class of each new row
    int32_t* list;    // [n]: the new rows by class
    int64_t* info;    // [2 * kRlClasses + 3]: class starts and sizes; the sorted entries; the CSR check; the
                      // sorted rows
    PartitionTmp part;
    int64_t* sdeg;  // entries of each new row that go to the radix sort
    int64_t* soff;  // [n + 1]: their exclusive scan
    int32_t* sflag;  // [n]: 1 for the rows that go to the radix sort
    int64_t* srank;  // [n + 1]: its exclusive scan (a row's rank among them)
    int32_t* srow;   // [n]: the row of each rank
    uint64_t* keys;
    uint32_t* vals;  // source positions (edge map only)
    ScanTmp scan;
    SortTmp sort;
};

PermuteWs carve(Ws& ws, int64_t n, int64_t nnz, bool with_map) {
    PermuteWs p;
    const int64_t n1 = n > 0 ? n : 1, e1 = nnz > 0 ? nnz : 1;
    p.flags = ws.take<uint32_t>(1);
    p.deg_new = ws.take<int64_t>(n1);
    p.cls = ws.take<int8_t>(n1);
    p.list = ws.take<int32_t>(n1);
    p.info = ws.take<int64_t>(2 * kRlClasses + 3);
    p.part = partition_tmp(ws, n1);
    p.sdeg = ws.take<int64_t>(n1);
    p.soff = ws.take<int64_t>(n1 + 1);
    p.sflag = ws.take<int32_t>(n1);
    p.srank = ws.take<int64_t>(n1 + 1);
    p.srow = ws.take<int32_t>(n1);
    p.keys = ws.take<uint64_t>(e1);
    p.vals = with_map ? ws.take<uint32_t>(e1) : nullptr;
    p.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(n1)));
    p.sort = sort_tmp(ws, e1, 8, with_map);
    return p;
}

// Relabelled CSR; with src_pos, also the old CSR position of every new edge
// (the sort carries it as the value), so per-edge values follow the edges.
gt_status permute(const char* who, int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                  const int32_t* perm, const int32_t* iperm, int64_t* rowptr_out, int32_t* col_out, int32_t* src_pos,
                  void* ws_ptr, size_t ws_bytes, hipStream_t stream) {
    const bool with_map = src_pos != nullptr;
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << (with_map ? 31 : 32)))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": n or nnz out of range");
    if (!rowptr || !rowptr_out || (nnz > 0 && (!col || !col_out)) || (n > 0 && (!perm || !iperm)) || !ws_ptr)
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null pointer");
    Ws need(nullptr);
    carve(need, n, nnz, with_map);
    if (ws_bytes < need.size()) return fail(GT_ERR_WORKSPACE, std::string(who) + ": workspace too small");
    Ws ws(ws_ptr);
    PermuteWs p = carve(ws, n, nnz, with_map);
    gt_status st;
    if (n == 0) return fill_i64(rowptr_out, 1, 0, stream);
    // the CSR check is read back with the class sizes below: nothing before that reads col
    if ((st = launch_validate_csr(n, nnz, rowptr, col, p.flags, stream)) != GT_OK) return st;
    const unsigned g = grid_for(n, 256, 8192);
    k_new_degrees<<<g, 256, 0, stream>>>(n, rowptr, perm, p.deg_new, p.cls, p.sdeg, p.sflag);
    GT_LAUNCH_CHECK("permute_degrees");
    if ((st = exclusive_scan_i64(p.deg_new, n, rowptr_out, p.scan, stream)) != GT_OK) return st;
    if (nnz == 0) return read_validation(p.flags, stream);
    // the rows of more than kWaveRow entries go to the radix sort: their offsets there and their ranks
    if ((st = exclusive_scan_i64(p.sdeg, n, p.soff, p.scan, stream)) != GT_OK) return st;
    if ((st = exclusive_scan_i32(p.sflag, n, p.srank, p.scan, stream)) != GT_OK) return st;
    k_sorted_rows<<<g, 256, 0, stream>>>(n, p.sflag, p.srank, p.srow);
    GT_LAUNCH_CHECK("permute_sorted_rows");
    if ((st = partition_rows(p.cls, n, kRlClasses, p.list, p.info, p.part, stream)) != GT_OK) return st;
    k_host_words<<<1, 64, 0, stream>>>(p.soff + n, p.flags, p.srank + n, p.info + 2 * kRlClasses);
    GT_LAUNCH_CHECK("permute_host_words");
    int64_t info[2 * kRlClasses + 3] = {};
    GT_HIP(hipMemcpyAsync(info, p.info, sizeof(info), hipMemcpyDeviceToHost, stream));
    GT_HIP(hipStreamSynchronize(stream));
    if ((st = validation_result(uint32_t(info[2 * kRlClasses + 1]))) != GT_OK) return st;
    const int64_t m = info[2 * kRlClasses];
    const int64_t m_rows = info[2 * kRlClasses + 2];
    {
        // the short-row lists in one launch, largest rows first, blocks in proportion to their rows
        ShortLists sl;
        const int order[5] = {kRl64, kRl32, kRl16, kRl8, kRl4};
        const int per_block[5] = {256 / 64, 256 / 32, 256 / 16, 256 / 8, 256 / 4};
        unsigned at = 0;
        for (int k = 0; k < 5; ++k) {
            const int c = order[k];
            sl.list[k] = p.list + info[c];
            sl.len[k] = info[kRlClasses + c];
            sl.first[k] = at;
            if (sl.len[k] > 0) {
                const int64_t gk = cdiv(sl.len[k], per_block[k]);
                at += unsigned(gk < 16384 ? gk : 16384);
            }
        }
        sl.first[5] = at;
        if (at > 0) {
            if (with_map)
                k_relabel_short<true><<<at, 256, 0, stream>>>(sl, rowptr, col, perm, iperm, rowptr_out, col_out,
                                                              src_pos);
            else
                k_relabel_short<false><<<at, 256, 0, stream>>>(sl, rowptr, col, perm, iperm, rowptr_out, col_out,
                                                               nullptr);
            GT_LAUNCH_CHECK("permute_short_rows");
        }
    }
    const int64_t n_wave = info[kRlClasses + kRlWave];
    if (n_wave > 0) {
        const int32_t* rows = p.list + info[kRlWave];
        const unsigned gw = grid_for(n_wave, 256 / kWave, 65536);
        if (with_map)
            k_relabel_wave<true><<<gw, 256, 0, stream>>>(rows, n_wave, rowptr, col, perm, iperm, rowptr_out, col_out,
                                                         src_pos);
        else
            k_relabel_wave<false><<<gw, 256, 0, stream>>>(rows, n_wave, rowptr, col, perm, iperm, rowptr_out,
                                                          col_out, nullptr);
        GT_LAUNCH_CHECK("permute_wave_rows");
    }
    if (m == 0) return GT_OK;
    const int bits = bits_for(n);
    const int64_t n_med = info[kRlClasses + kRlMed];
    if (n_med > 0) {
        const int32_t* med = p.list + info[kRlMed];
        const unsigned gm = grid_for(n_med, 4, 65536);
        if (with_map)
            k_edge_keys<true><<<gm, 256, 0, stream>>>(med, n_med, rowptr, col, perm, iperm, bits, p.soff, p.srank,
                                                      p.keys, p.vals);
        else
            k_edge_keys<false><<<gm, 256, 0, stream>>>(med, n_med, rowptr, col, perm, iperm, bits, p.soff, p.srank,
                                                       p.keys, nullptr);
        GT_LAUNCH_CHECK("permute_keys");
    }
    if (uint32_t(info[2 * kRlClasses + 1]) & kLongRowSeen) {  // some row has more than kLongRow entries
        const int64_t ch = long_chunks_of(nnz);
        const unsigned gl = unsigned(ch < 8192 ? ch : 8192);
        if (with_map)
            k_edge_keys_long<true><<<gl, 256, 0, stream>>>(n, nnz, rowptr, col, iperm, bits, p.soff, p.srank,
                                                           p.keys, p.vals);
        else
            k_edge_keys_long<false><<<gl, 256, 0, stream>>>(n, nnz, rowptr, col, iperm, bits, p.soff, p.srank,
                                                            p.keys, nullptr);
        GT_LAUNCH_CHECK("permute_keys_long");
    }
    // keys: (the row's rank among the m_rows sorted rows) << bits | new column
    if ((st = radix_sort_u64(p.keys, p.vals, m, bits + bits_for(m_rows), p.sort, stream)) != GT_OK) return st;
    k_place_sorted<<<grid_for(m, 256, 16384), 256, 0, stream>>>(m, p.keys, p.vals, bits, p.soff, p.srow, rowptr_out,
                                                                col_out, with_map ? src_pos : nullptr);
    GT_LAUNCH_CHECK("permute_place");
    return GT_OK;
}

}  // namespace
}  // namespace gt

using namespace gt;

extern "C" size_t gt_permute_workspace_size(int64_t n, int64_t nnz) {
    Ws ws(nullptr);
    carve(ws, n, nnz, false);
    return ws.size();
}

extern "C" gt_status gt_permute_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                                    const int32_t* perm, const int32_t* iperm, int64_t* rowptr_out,
                                    int32_t* col_out, void* ws_ptr, size_t ws_bytes, hipStream_t stream) {
    return permute("gt_permute_csr", n, nnz, rowptr, col, perm, iperm, rowptr_out, col_out, nullptr, ws_ptr,
                   ws_bytes, stream);
}

extern "C" size_t gt_permute_edges_workspace_size(int64_t n, int64_t nnz) {
    Ws ws(nullptr);
    carve(ws, n, nnz, true);
    return ws.size();
}

extern "C" gt_status gt_permute_csr_edges(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                                          const int32_t* perm, const int32_t* iperm, int64_t* rowptr_out,
                                          int32_t* col_out, int32_t* src_pos, void* ws_ptr, size_t ws_bytes,
                                          hipStream_t stream) {
    if (nnz > 0 && !src_pos) return fail(GT_ERR_INVALID_ARG, "gt_permute_csr_edges: null src_pos");
    return permute("gt_permute_csr_edges", n, nnz, rowptr, col, perm, iperm, rowptr_out, col_out, src_pos, ws_ptr,
                   ws_bytes, stream);
}

static gt_status move_rows(bool gather, int64_t n, int64_t row_bytes, const void* src, const int32_t* perm,
                           void* dst, hipStream_t stream) {
    if (n < 0 || row_bytes < 0 || row_bytes % 4 != 0)
        return fail(GT_ERR_INVALID_ARG, "gt_gather_rows/gt_scatter_rows: bad n or row_bytes (must be a multiple of 4)");
    if (n == 0 || row_bytes == 0) return GT_OK;
    if (!src || !dst || !perm) return fail(GT_ERR_INVALID_ARG, "gt_gather_rows/gt_scatter_rows: null pointer");
    if (row_bytes < 128) {
        const int32_t words = int32_t(row_bytes / 4);
        const unsigned gs = grid_for(n * words, 256, 65536);
        if (gather)
            k_move_small_rows<true><<<gs, 256, 0, stream>>>(n, words, static_cast<const uint32_t*>(src), perm,
                                                              static_cast<uint32_t*>(dst));
        else
            k_move_small_rows<false><<<gs, 256, 0, stream>>>(n, words, static_cast<const uint32_t*>(src), perm,
                                                               static_cast<uint32_t*>(dst));
        GT_LAUNCH_CHECK("move_small_rows");
        return GT_OK;
    }
    const bool aligned = (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) % 16 == 0;
    if (row_bytes % 16 == 0 && aligned) {
        const int64_t vpr = row_bytes / 16, total = n * vpr;
        const unsigned gv = grid_for(total, 256, 16384);
        const uint4* s4 = static_cast<const uint4*>(src);
        uint4* d4 = static_cast<uint4*>(dst);
        if (total < (int64_t(1) << 32)) {
            const uint32_t n32 = uint32_t(n), v32 = uint32_t(vpr);
            if (gather) k_move_rows16<true, uint32_t><<<gv, 256, 0, stream>>>(n32, v32, s4, perm, d4);
            else k_move_rows16<false, uint32_t><<<gv, 256, 0, stream>>>(n32, v32, s4, perm, d4);
        } else {
            if (gather) k_move_rows16<true, int64_t><<<gv, 256, 0, stream>>>(n, vpr, s4, perm, d4);
            else k_move_rows16<false, int64_t><<<gv, 256, 0, stream>>>(n, vpr, s4, perm, d4);
        }
        GT_LAUNCH_CHECK("move_rows16");
        return GT_OK;
    }
    const unsigned g = grid_for(n, 4, 65536);
    if (gather)
        k_move_rows<true><<<g, 256, 0, stream>>>(n, row_bytes / 4, static_cast<const uint32_t*>(src), perm,
                                                  static_cast<uint32_t*>(dst));
    else
        k_move_rows<false><<<g, 256, 0, stream>>>(n, row_bytes / 4, static_cast<const uint32_t*>(src), perm,
                                                   static_cast<uint32_t*>(dst));
    GT_LAUNCH_CHECK("move_rows");
    return GT_OK;
}

extern "C" gt_status gt_gather_rows(int64_t n, int64_t row_bytes, const void* src, const int32_t* perm, void* dst,
                                    hipStream_t stream) {
    return move_rows(true, n, row_bytes, src, perm, dst, stream);
}

extern "C" gt_status gt_scatter_rows(int64_t n, int64_t row_bytes, const void* src, const int32_t* perm, void* dst,
                                     hipStream_t stream) {
    return move_rows(false, n, row_bytes, src, perm, dst, stream);
}
