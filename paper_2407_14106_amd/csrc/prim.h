// Device-wide building blocks used by the integer stages (validation, reorder,
// relabelling, tile plan): fills, exclusive scans, key counting and a stable
// LSD radix sort.  Every routine is stream-ordered and draws its scratch from
// the caller's workspace through gt::Ws.
#pragma once

#include "common.h"

namespace gt {

// ---- work spread over the caller's stream and side streams the caller gives
// A call may spread independent work over up to kMaxSide further streams of
// the caller's (on the same device), ordered by events the caller also gives
// (one to fork, one per side stream to join), so the library creates nothing.
// fork(): the side streams wait for the work enqueued on the caller's stream
// so far; join(): the caller's stream waits for the work enqueued on the side
// streams.  A Spread still forked when destroyed joins first, so the caller's
// stream never finishes before the side streams' work.  With no side streams
// everything runs on the caller's stream.
constexpr int kMaxSide = 2;
struct Spread {
    hipStream_t main = nullptr;
    hipStream_t side[kMaxSide] = {};
    hipEvent_t fork_ev = nullptr;
    hipEvent_t join_ev[kMaxSide] = {};
    int n_side = 0;
    bool forked = false;
    // stream k: 0 the caller's, 1 .. kMaxSide the side streams (dealt round the ones given)
    hipStream_t at(int k) const { return (k == 0 || n_side == 0) ? main : side[(k - 1) % n_side]; }
    gt_status fork();
    gt_status join();
    Spread() = default;
    Spread(const Spread&) = delete;
    Spread& operator=(const Spread&) = delete;
    ~Spread() { (void)join(); }
};
// events: n_side + 1 of them.  Checks that the side streams and events are
// non-null and distinct and the side streams are not main, then that the side
// streams are on main's device.
gt_status spread_open(const char* who, hipStream_t main, const hipStream_t* side, const hipEvent_t* events,
                      int n_side, Spread* sp);

// ---- fills
gt_status fill_u32(uint32_t* p, int64_t n, uint32_t value, hipStream_t s);
gt_status fill_i64(int64_t* p, int64_t n, int64_t value, hipStream_t s);
gt_status iota_u32(uint32_t* p, int64_t n, hipStream_t s);
gt_status copy_bytes(void* dst, const void* src, int64_t bytes, hipStream_t s);  // bytes % 4 == 0

// ---- exclusive scan: out[i] = sum(in[0..i)), out[n] = total; out has n+1 entries.
struct ScanTmp {
    int64_t* block_sums = nullptr;  // scan_tmp_elems(n) entries
};
int64_t scan_tmp_elems(int64_t n);
gt_status exclusive_scan_i32(const int32_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s);
gt_status exclusive_scan_u32(const uint32_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s);
gt_status exclusive_scan_i64(const int64_t* in, int64_t n, int64_t* out, ScanTmp tmp, hipStream_t s);

// ---- counts[k] += number of i with keys[i] == k (counts must be zeroed by the caller).
gt_status count_keys(const int32_t* keys, int64_t n, uint32_t* counts, hipStream_t s);

// ---- stable LSD radix sort of (key, value) pairs on bits [0, key_bits), 8 bits per pass.
// `values` may be null (keys only).  The result ends in keys/values.
struct SortTmp {
    void* keys_alt = nullptr;       // n keys
    uint32_t* vals_alt = nullptr;   // n values (if values are sorted)
    uint32_t* hist = nullptr;       // 256 * tiles
    int64_t* offsets = nullptr;     // 256 * tiles + 1
    ScanTmp scan;
};
int64_t sort_tiles(int64_t n);
// Measure/carve a SortTmp for n pairs with keys of key_bytes (4 or 8).
SortTmp sort_tmp(Ws& ws, int64_t n, int key_bytes, bool with_values);
gt_status radix_sort_u32(uint32_t* keys, uint32_t* values, int64_t n, int key_bits, SortTmp tmp, hipStream_t s);
gt_status radix_sort_u64(uint64_t* keys, uint32_t* values, int64_t n, int key_bits, SortTmp tmp, hipStream_t s);

// Number of bits needed to hold values in [0, n).
inline int bits_for(int64_t n) {
    int b = 1;
    while ((int64_t(1) << b) < n) ++b;
    return b;
}

// ---- long rows, spread over the grid.
// Rows of more than kLongRow entries are handled by a pass of their own that cuts
// the CSR's entry range into chunks of kLongRow entries.  A long row is longer
// than a chunk, so at most two long rows overlap a chunk: the row of its first
// entry and the row of its last entry.
constexpr int64_t kLongRow = 2048;

__host__ __device__ inline int64_t long_chunks_of(int64_t nnz) { return (nnz + kLongRow - 1) / kLongRow; }

// The row r with rowptr[r] <= e < rowptr[r + 1], for 0 <= e < rowptr[n]
// (empty rows are skipped); stays in [0, n - 1] for any rowptr.
__device__ __forceinline__ int64_t row_of(const int64_t* __restrict__ rowptr, int64_t n, int64_t e) {
    int64_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (rowptr[mid] <= e) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

struct LongSeg {
    int64_t row;   // the row
    int64_t a, b;  // its entries inside the chunk, [a, b)
    int s;         // 0: the row of the chunk's first entry, 1: of its last
};

// The segments of long rows inside chunk c of a CSR with nnz entries; returns
// their number (0, 1 or 2).  Entry bounds are clamped to the chunk, so an
// invalid rowptr still only yields entries in [0, nnz).
__device__ __forceinline__ int long_segments(const int64_t* __restrict__ rowptr, int64_t n, int64_t nnz, int64_t c,
                                             LongSeg seg[2]) {
    const int64_t e0 = c * kLongRow, e1 = e0 + kLongRow < nnz ? e0 + kLongRow : nnz;
    int k = 0;
    if (e0 >= e1 || n <= 0) return 0;
    const int64_t ra = row_of(rowptr, n, e0), rb = row_of(rowptr, n, e1 - 1);
    const int64_t rows[2] = {ra, rb};
    for (int s = 0; s < 2; ++s) {
        const int64_t r = rows[s];
        if (s == 1 && rb == ra) break;
        const int64_t p = rowptr[r], q = rowptr[r + 1];
        if (q - p <= kLongRow) continue;
        LongSeg g;
        g.row = r;
        g.a = p > e0 ? p : e0;
        g.b = q < e1 ? q : e1;
        g.s = s;
        if (g.a < g.b) seg[k++] = g;
    }
    return k;
}

// ---- Stable partition of rows [0, n) by a class per row (cls[v] in [0, ncls),
// or -1 for no list; ncls <= kMaxClasses): list holds the rows of class 0 in
// ascending order, then those of class 1, ...; info[c] = the first list
// position of class c and info[ncls + c] = its rows.  One counting pass over
// 256-row blocks, one scan of the class-major [class][block] counts, one
// writing pass.
constexpr int kMaxClasses = 8;
struct PartitionTmp {
    int32_t* blk_cnt = nullptr;  // [kMaxClasses * blocks]
    int64_t* blk_off = nullptr;  // [kMaxClasses * blocks + 1]
    ScanTmp scan;
};
PartitionTmp partition_tmp(Ws& ws, int64_t n);
gt_status partition_rows(const int8_t* cls, int64_t n, int ncls, int32_t* list, int64_t* info, PartitionTmp t,
                         hipStream_t s);

// ---- CSR validation: accumulates error bits into *flags (one uint32, zeroed by the caller).
enum : uint32_t { kBadRowptr = 1u, kOutOfRange = 2u, kUnsorted = 4u, kDuplicate = 8u };
// Not an error: the rows pass saw a row of more than kLongRow entries (the
// stages whose long-row kernels scan every entry chunk skip them without one).
constexpr uint32_t kLongRowSeen = 16u;
gt_status launch_validate_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, uint32_t* flags,
                              hipStream_t s);
// Reads the flags back (SYNC) and maps them to a status.
gt_status read_validation(const uint32_t* flags, hipStream_t s);
// The status of a validation flag word already on the host.
gt_status validation_result(uint32_t flags);

}  // namespace gt
