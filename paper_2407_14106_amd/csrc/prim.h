// Device-wide building blocks used by the integer stages (validation, reorder,
// relabelling, tile plan): fills, exclusive scans, key counting and a stable
// LSD radix sort.  Every routine is stream-ordered and draws its scratch from
// the caller's workspace through gt::Ws.
#pragma once

#include "common.h"

namespace gt {

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

// ---- CSR validation: accumulates error bits into *flags (one uint32, zeroed by the caller).
enum : uint32_t { kBadRowptr = 1u, kOutOfRange = 2u, kUnsorted = 4u, kDuplicate = 8u };
gt_status launch_validate_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, uint32_t* flags,
                              hipStream_t s);
// Reads the flags back (SYNC) and maps them to a status.
gt_status read_validation(const uint32_t* flags, hipStream_t s);

}  // namespace gt
