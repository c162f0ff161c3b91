// Cluster reordering (§3.3): label propagation with hashed tie-breaks and
// hashed partial activation, then a stable sort by (label, -degree, id).
//
// Rows are handled by size:
//   deg <= 4 / 8 / 16 / 32
//                      16 / 8 / 4 / 2 rows per wavefront, 4 / 8 / 16 / 32
//                      lanes each;
//   32 < deg <= 64     one wavefront per row; one neighbour label per lane.
//                      Multiplicities by peeling the distinct labels (ballots)
//                      or, past a few, an all-pairs compare (readlane); rows
//                      of up to 8 compare by fixed lane patterns.  These five
//                      classes run in one launch, their entries in padded
//                      slots found from the row's list position.
//   64 < deg <= 512    one wavefront per row, open-addressing count table in
//                      the wavefront's share of LDS (no workgroup barriers).
//   512 < deg <= 4096  one workgroup per row, open-addressing count table in LDS.
//   deg > 4096         the whole grid (hubs, a global token attending to every
//                      node): each row's count table in the workspace, filled
//                      chunk by chunk by every workgroup, then, for tables of up
//                      to 64K slots, reduced, decided and cleared by one
//                      workgroup per row; larger tables are reduced by every
//                      workgroup in three passes (best count, smallest hash,
//                      smallest label).
// All compute the same function of the neighbour-label multiset.  The first
// sweep, whose labels are the node ids, reduces to a minimum over each row's
// columns and uses none of the tables.
//
// The sweeps after the first run on the graph renumbered by list position
// (each row's place in the class-major row list): the rows' entries are laid
// out in list order (roff, ncol for the rows of more than 64 entries, padded
// slots for the others; written once, during the first sweep) and a node's
// label is kept at its list position.  A class's rows then read their row
// offsets and entries in runs, and the classes gather the long rows, whose
// labels most rows read, into a few cache lines.  The label values stay node
// ids, so the result does not depend on this numbering.  With side streams
// from the caller, a sweep's classes run side by side where the rows of more
// than 64 entries hold at least a quarter of the entries.
#include <limits.h>

#include "lanes.h"
#include "prim.h"

namespace gt {

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kActivitySalt = 0xD6E8FEB86659FD93ull;
constexpr int kWaveRowMax = 64;
constexpr int kSub4 = 4, kSub8 = 8, kSub16 = 16, kSub32 = 32;  // rows of up to 4 ... 32 edges share a wavefront
constexpr int kWaveTabRowMax = 512;
constexpr int kWaveTab = 2 * kWaveTabRowMax;  // per-wavefront table entries
constexpr int kLdsTable = 8192;      // entries (int32 key + uint32 count): 64 KiB
constexpr int kLdsRowMax = kLdsTable / 2;
constexpr int kBlock = 256;
constexpr int kMedBlock = 1024;  // threads per row of kWaveTabRowMax + 1 to kLdsRowMax edges
constexpr int kMaxSweeps = 1000;
constexpr int kBigGrid = 2048;  // workgroups sharing the very long rows
constexpr int kBigEdgeChunk = 1024;  // edges of a very long row counted in one workgroup's LDS table
constexpr int kBigChunkTab = 2 * kBigEdgeChunk;

__device__ __forceinline__ bool is_active(int64_t v, uint64_t key) {
    return (mix64(uint64_t(v) ^ key ^ kActivitySalt) >> 61) != 0;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    uint32_t lo = __shfl_xor(uint32_t(v), o, kWave);
    uint32_t hi = __shfl_xor(uint32_t(v >> 32), o, kWave);
    return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        uint64_t w = shfl_xor_u64(v, o);
        v = w < v ? w : v;
    }
    return v;
}
__device__ __forceinline__ int wave_min_i32(int v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        int w = __shfl_xor(v, o, kWave);
        v = w < v ? w : v;
    }
    return v;
}

// -------------------------------------------------------------- per-row classes
// Every row falls in one class by its entry count; the rows of all classes go
// to one list, class after class, each class in ascending row order.  One
// pass counts each 256-row block's rows per class, one scan over the
// class-major [class][block] counts gives every (class, block) its place in
// the list, and a second pass writes the rows there.

enum { kClsS4, kClsS8, kClsS16, kClsS32, kClsWav, kClsWmed, kClsMed, kClsHuge, kClasses };
constexpr int kClsBlock = 256;

__device__ __forceinline__ int row_class(int64_t deg) {
    return deg <= kSub4           ? kClsS4
           : deg <= kSub8         ? kClsS8
           : deg <= kSub16        ? kClsS16
           : deg <= kSub32        ? kClsS32
           : deg <= kWaveRowMax   ? kClsWav
           : deg <= kWaveTabRowMax ? kClsWmed
           : deg <= kLdsRowMax    ? kClsMed
                                  : kClsHuge;
}

// Per-wavefront counts of each class in s[w][c]; returns the lane's rank among
// the wavefront's lanes of its own class (cls < 0: no row).
__device__ __forceinline__ int class_ballots(int cls, int (*s)[kClasses]) {
    const int w = threadIdx.x / kWave;
    int rank = 0;
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
        const uint64_t m = __ballot(cls == c);
        if (lane_id() == 0) s[w][c] = __popcll(m);
        if (cls == c) rank = __popcll(m & lanemask_lt());
    }
    return rank;
}

// Off-diagonal entry count of every row (for the final order; the block's
// largest in blk_max[block]), the block's rows per class, in
// blk_cnt[c * nblk + block], and the entries of its rows of more than
// kWaveRowMax entries, in blk_long[block].  It runs before the CSR check is
// read back, so every read stays in col[0, nnz) whatever rowptr holds.
__global__ __launch_bounds__(kClsBlock) void k_classify(int64_t n, int64_t nnz, const int64_t* rowptr,
                                                        const int32_t* col, uint32_t* deg_off, int32_t* blk_cnt,
                                                        int64_t nblk, uint32_t* blk_max, uint32_t* blk_long) {
    __shared__ int s_cnt[kClsBlock / kWave][kClasses];
    __shared__ uint32_t s_max[kClsBlock / kWave];
    __shared__ uint32_t s_long[kClsBlock / kWave];
    uint32_t dv = 0, lv = 0;
    const int64_t v = int64_t(blockIdx.x) * kClsBlock + threadIdx.x;
    int cls = -1;
    if (v < n) {
        int64_t a = rowptr[v], b = rowptr[v + 1];
        a = a < 0 ? 0 : (a > nnz ? nnz : a);
        b = b < a ? a : (b > nnz ? nnz : b);
        // self-loop present?  rows are sorted: binary search for v.
        int64_t lo = a, hi = b;
        while (lo < hi) {
            int64_t m = (lo + hi) >> 1;
            if (col[m] < v) lo = m + 1;
            else hi = m;
        }
        const bool self = lo < b && col[lo] == v;
        dv = uint32_t(b - a - (self ? 1 : 0));
        deg_off[v] = dv;
        cls = row_class(b - a);
        lv = b - a > kWaveRowMax ? uint32_t(b - a) : 0u;
    }
    class_ballots(cls, s_cnt);
    dv = wave_max(dv);
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) lv += __shfl_xor(lv, o, kWave);  // < 2^32: entries of the block's rows
    if (lane_id() == 0) {
        s_max[threadIdx.x / kWave] = dv;
        s_long[threadIdx.x / kWave] = lv;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t m = 0, l = 0;
#pragma unroll
        for (int w = 0; w < kClsBlock / kWave; ++w) {
            m = s_max[w] > m ? s_max[w] : m;
            l += s_long[w];
        }
        blk_max[blockIdx.x] = m;
        blk_long[blockIdx.x] = l;
    }
    if (threadIdx.x < kClasses) {
        int t = 0;
#pragma unroll
        for (int w = 0; w < kClsBlock / kWave; ++w) t += s_cnt[w][threadIdx.x];
        blk_cnt[threadIdx.x * nblk + blockIdx.x] = t;
    }
}

// list[pos] = v, lpos[v] = pos (the row's list position) and ldeg[pos] = its
// entry count.
__global__ __launch_bounds__(kClsBlock) void k_class_scatter(int64_t n, const int64_t* rowptr,
                                                             const int64_t* blk_off, int64_t nblk, int32_t* list,
                                                             int32_t* lpos, uint32_t* ldeg) {
    __shared__ int s_cnt[kClsBlock / kWave][kClasses];
    const int64_t v = int64_t(blockIdx.x) * kClsBlock + threadIdx.x;
    const int64_t deg = v < n ? rowptr[v + 1] - rowptr[v] : 0;
    const int cls = v < n ? row_class(deg) : -1;
    const int rank = class_ballots(cls, s_cnt);
    __syncthreads();
    if (cls >= 0) {
        int64_t pos = blk_off[cls * nblk + blockIdx.x] + rank;
        for (int w = 0; w < int(threadIdx.x / kWave); ++w) pos += s_cnt[w][cls];
        list[pos] = int32_t(v);
        lpos[v] = int32_t(pos);
        ldeg[pos] = uint32_t(deg);
    }
}

// info[c] = the first list position of class c, info[kClasses + c] = its rows.
__global__ void k_class_totals(int64_t nblk, const int64_t* blk_off, int64_t* info) {
    const int c = threadIdx.x;
    if (blockIdx.x != 0 || c >= kClasses) return;
    info[c] = blk_off[c * nblk];
    info[kClasses + c] = blk_off[(c + 1) * nblk] - blk_off[c * nblk];
}

// The largest of the blocks' maxima, in *out_max, and the sum of their long
// rows' entries, in *out_long (both start at zero): each workgroup reduces
// kMaxSpan blocks and adds one atomic to each.
constexpr int kMaxSpan = 4096;
__global__ __launch_bounds__(256) void k_blocks_max(int64_t nblk, const uint32_t* blk_max, const uint32_t* blk_long,
                                                    unsigned long long* out_max, unsigned long long* out_long) {
    __shared__ uint32_t s_max[256 / kWave];
    __shared__ uint64_t s_sum[256 / kWave];
    uint32_t m = 0;
    uint64_t l = 0;
    const int64_t b0 = int64_t(blockIdx.x) * kMaxSpan;
    for (int64_t b = b0 + threadIdx.x; b < nblk && b < b0 + kMaxSpan; b += 256) {
        m = blk_max[b] > m ? blk_max[b] : m;
        l += blk_long[b];
    }
    m = wave_max(m);
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) l += shfl_xor_u64(l, o);
    if (lane_id() == 0) {
        s_max[threadIdx.x / kWave] = m;
        s_sum[threadIdx.x / kWave] = l;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < 256 / kWave; ++w) {
            m = s_max[w] > m ? s_max[w] : m;
            l += s_sum[w];
        }
        if (m) atomicMax(out_max, (unsigned long long)m);
        if (l) atomicAdd(out_long, (unsigned long long)l);
    }
}

// ------------------------------------------------------------------ short rows
// Rows of up to kWaveRowMax edges, in five lists by size, all in one launch:
// the grid's blocks are cut into one range per list, each range running its
// list with a grid-stride loop over tasks (one wavefront's rows).  Their
// entries (as list positions) sit in slots padded to the list's largest row
// (S = 64, 32, 16, 8 or 4 slots a row, -1 past the row's entries), so a row's
// slots are found from its list position alone: the entries' load does not
// wait for a row offset.  Every class holds rows of more than S / 2 entries
// except the 0-4 one, so the slots number at most 2 nnz + 4 n.

// Reductions over the S lanes of a row group (S = 4, 8, 16 or 32), O = S / 2 down to 1.
template <int S, int O = S / 2>
__device__ __forceinline__ int group_max_i32(int v) {
    if constexpr (O == 0) {
        return v;
    } else {
        const int w = xor_lane<O>(v);
        return group_max_i32<S, O / 2>(w > v ? w : v);
    }
}
template <int S, int O = S / 2>
__device__ __forceinline__ int group_min_i32(int v) {
    if constexpr (O == 0) {
        return v;
    } else {
        const int w = xor_lane<O>(v);
        return group_min_i32<S, O / 2>(w < v ? w : v);
    }
}
template <int S, int O = S / 2>
__device__ __forceinline__ uint64_t group_min_u64(uint64_t v) {
    if constexpr (O == 0) {
        return v;
    } else {
        const uint64_t w = xor_lane_u64<O>(v);
        return group_min_u64<S, O / 2>(w < v ? w : v);
    }
}

// Lanes of this lane's S-lane group (S <= 16) other than itself holding L.
template <int S, int K = 1>
__device__ __forceinline__ int xor_matches(int L) {
    if constexpr (K >= S) {
        return 0;
    } else {
        return (xor_lane<K>(L) == L ? 1 : 0) + xor_matches<S, K + 1>(L);
    }
}

// How many valid lanes of this lane's S-lane group hold its label L (0 for
// an invalid lane), for G = 64 / S <= 4 groups a wavefront.  Once clusters
// form a row's neighbours carry few distinct labels, so they are peeled off
// one per group and step (the group's first uncounted lane, read with
// readlane, and one ballot); rows with more than kPeel distinct labels count
// their remaining lanes by comparing every lane's label in turn (dmax: the
// wavefront's largest row).
constexpr int kPeel = 6;
template <int S>
__device__ __forceinline__ int group_counts(int L, bool valid, int dmax) {
    constexpr int G = kWave / S;
    static_assert(G <= 4, "peeling reads one lane per group");
    const int lane = lane_id(), sub = lane / S;
    const uint64_t gmask = (S == kWave ? ~0ull : ((1ull << S) - 1)) << (sub * S);
    int cnt = 0;
    uint64_t todo = __ballot(valid);
    for (int it = 0; it < kPeel && todo; ++it) {
        int Ld = -2;  // never a label
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const uint64_t t = todo & ((S == kWave ? ~0ull : ((1ull << S) - 1)) << (g * S));
            const int x = t ? __builtin_amdgcn_readlane(L, __builtin_ctzll(t)) : -2;
            Ld = sub == g ? x : Ld;
        }
        const bool eq = valid && L == Ld;
        const uint64_t same = __ballot(eq);
        if (eq) cnt = __popcll(same & gmask);
        todo &= ~same;
    }
    if (todo) {
        int c2 = 0;
        for (int k = 0; k < dmax; ++k) {
            int Lk = __builtin_amdgcn_readlane(L, k);
#pragma unroll
            for (int g = 1; g < G; ++g) {
                const int x = __builtin_amdgcn_readlane(L, g * S + k);
                Lk = sub == g ? x : Lk;
            }
            c2 += (Lk == L) ? 1 : 0;
        }
        if ((todo >> lane) & 1ull) cnt = c2;
    }
    return valid ? cnt : 0;
}

// Row at list position p (kSub32 + 1 to kWaveRowMax edges), one wavefront:
// every lane counts how many of the row's labels equal its own, reading the
// others with readlane (the lane index is uniform over the wavefront).  slots:
// the row's 64 entry slots (list positions, -1 past its entries); labels are
// indexed by list position.
__device__ __forceinline__ void lp_wave_row(int64_t p, const int32_t* list, const int32_t* slots,
                                            const int32_t* lab_in, int32_t* lab_out, uint64_t key, bool converged,
                                            uint32_t* flag_next) {
    const int lane = lane_id();
    const int own = lab_in[p];
    if (converged) {
        if (lane == 0) lab_out[p] = own;
        return;
    }
    const int64_t v = list[p];
    const int c = slots[lane];
    const int deg = __popcll(ballot(c >= 0));  // the entries fill the first deg slots
    const bool valid = c >= 0 && c != p;
    const int L = valid ? lab_in[c] : -1;
    const int cnt = group_counts<kWave>(L, valid, deg);
    const int best = wave_max(cnt);
    int cand = own;
    if (best > 0) {
        const int own_cnt = __popcll(ballot(valid && L == own));
        if (own_cnt != best) {
            const bool top = valid && cnt == best;
            const uint64_t h = top ? mix64(uint64_t(uint32_t(L)) ^ key) : ~0ull;
            const uint64_t hmin = wave_min_u64(h);
            cand = wave_min_i32((top && h == hmin) ? L : INT_MAX);
        }
    }
    if (lane == 0) {
        lab_out[p] = is_active(v, key) ? cand : own;
        if (cand != own) *flag_next = 1u;
    }
}

// Rows g0 .. g0 + 64 / S - 1 of a list of rows of at most S edges (S = 4, 8,
// 16 or 32) at list positions base + [0, len), row idx's S slots at
// slots + S idx: the same function as lp_wave_row with every reduction
// confined to the row's S lanes.
template <int S>
__device__ __forceinline__ void lp_sub_group(int64_t g0, int64_t base, int64_t len, const int32_t* list,
                                             const int32_t* slots, const int32_t* lab_in, int32_t* lab_out,
                                             uint64_t key, bool converged, uint32_t* flag_next) {
    constexpr int G = kWave / S;
    const int lane = lane_id(), sub = lane / S, sl = lane % S;
    const uint64_t gmask = (S == kWave ? ~0ull : ((1ull << S) - 1)) << (sub * S);
    const int64_t idx = g0 + sub;
    const bool live = idx < len;
    const int64_t p = base + idx;
    const int own = live ? lab_in[p] : -1;
    if (converged) {
        if (live && sl == 0) lab_out[p] = own;
        return;
    }
    const int64_t v = live ? list[p] : 0;
    const int c = live ? slots[idx * S + sl] : -1;
    const int deg = __popcll(__ballot(c >= 0) & gmask);  // the entries fill the row's first deg slots
    const bool valid = c >= 0 && c != p;
    const int L = valid ? lab_in[c] : -1;
    const int dmax = wave_max(deg);
    int cnt = 0;
    if constexpr (G <= 4) {
        cnt = group_counts<S>(L, valid, dmax);
    } else {
        // eight or sixteen rows a wavefront: every other lane of the group by a fixed lane pattern
        // (an invalid lane's -1 matches no label), exchanged with every lane active
        const int m = xor_matches<S>(L);
        cnt = valid ? 1 + m : 0;
    }
    const int best = group_max_i32<S>(cnt);
    const int own_cnt = __popcll(__ballot(valid && L == own) & gmask);
    const bool moves = best > 0 && own_cnt != best;
    int cand = own;
    if (__ballot(moves)) {  // the tie-break, unless every row of the wavefront keeps its label
        const bool top = valid && cnt == best && moves;
        const uint64_t h = top ? mix64(uint64_t(uint32_t(L)) ^ key) : ~0ull;
        const uint64_t hmin = group_min_u64<S>(h);
        const int lmin = group_min_i32<S>((top && h == hmin) ? L : INT_MAX);
        if (moves) cand = lmin;
    }
    if (live && sl == 0) {
        lab_out[p] = is_active(v, key) ? cand : own;
        if (cand != own) *flag_next = 1u;
    }
}

// The five short-row lists (rows of 33-64, 17-32, 9-16, 5-8 and 0-4 edges, in
// that order): their first list positions and lengths, the first entry slot
// of each, and the first block of each one's range; first[5] is the grid.
enum { kSmWave, kSm32, kSm16, kSm8, kSm4, kSmLists };
struct SmallRows {
    const int32_t* list;
    int64_t base[kSmLists];
    int64_t len[kSmLists];
    int64_t slot[kSmLists];
    unsigned first[kSmLists + 1];
};

// The list of this block's range, the block's index in it and the range's size.
__device__ __forceinline__ int small_list(const SmallRows& sr, unsigned* blk, unsigned* nblk) {
    const unsigned b = blockIdx.x;
    int k = 0;
    while (k + 1 < kSmLists && b >= sr.first[k + 1]) ++k;
    *blk = b - sr.first[k];
    *nblk = sr.first[k + 1] - sr.first[k];
    return k;
}

template <int S>
__device__ __forceinline__ void lp_sub_rows(const SmallRows& sr, int k, unsigned blk, unsigned nblk,
                                            const int32_t* slots, const int32_t* lab_in, int32_t* lab_out,
                                            uint64_t key, bool converged, uint32_t* flag_next) {
    constexpr int G = kWave / S;
    const int64_t waves = int64_t(nblk) * (kBlock / kWave);
    for (int64_t g0 = (int64_t(blk) * (kBlock / kWave) + threadIdx.x / kWave) * G; g0 < sr.len[k]; g0 += waves * G)
        lp_sub_group<S>(g0, sr.base[k], sr.len[k], sr.list, slots + sr.slot[k], lab_in, lab_out, key, converged,
                        flag_next);
}

// The sweeps after the first over the five lists; slots: the rows' padded entries.
__global__ __launch_bounds__(kBlock) void k_lp_small(SmallRows sr, const int32_t* slots, const int32_t* lab_in,
                                                     int32_t* lab_out, uint64_t key, const uint32_t* flag_prev,
                                                     uint32_t* flag_next) {
    const bool converged = *flag_prev == 0;
    unsigned blk, nblk;
    const int k = small_list(sr, &blk, &nblk);
    switch (k) {
        case kSmWave: {
            const int64_t waves = int64_t(nblk) * (kBlock / kWave);
            for (int64_t g = int64_t(blk) * (kBlock / kWave) + threadIdx.x / kWave; g < sr.len[k]; g += waves)
                lp_wave_row(sr.base[k] + g, sr.list, slots + sr.slot[k] + g * kWave, lab_in, lab_out, key,
                            converged, flag_next);
            break;
        }
        case kSm32:
            lp_sub_rows<kSub32>(sr, k, blk, nblk, slots, lab_in, lab_out, key, converged, flag_next);
            break;
        case kSm16:
            lp_sub_rows<kSub16>(sr, k, blk, nblk, slots, lab_in, lab_out, key, converged, flag_next);
            break;
        case kSm8:
            lp_sub_rows<kSub8>(sr, k, blk, nblk, slots, lab_in, lab_out, key, converged, flag_next);
            break;
        default:
            lp_sub_rows<kSub4>(sr, k, blk, nblk, slots, lab_in, lab_out, key, converged, flag_next);
            break;
    }
}

// ----------------------------------------------------------- the first sweep
// The first sweep starts from every node's own id as its label, so the labels
// of a row's neighbours all differ and each counts once: the best count is 1
// (0 without a neighbour other than the node itself), the node's own label is
// not among them, and the tie-break takes the neighbour whose id hashes
// smallest.  The hash is a bijection of the 64-bit word, so that neighbour is
// unique.  The first sweep therefore reads no labels and builds no tables: it
// takes a minimum over each row's columns.

// Rows of at most S edges, 64 / S per wavefront.  Every entry is read here
// once: its column's list position goes to the row's slots (row idx's S slots
// at slots + S idx, -1 past its entries) for the later sweeps.
template <int S>
__device__ __forceinline__ void first_rows(const int32_t* list, int64_t base, int64_t len, unsigned blk,
                                           unsigned nblk, const int64_t* rowptr, const int32_t* col,
                                           const int32_t* lpos, int32_t* slots, int32_t* lab_out, uint64_t key,
                                           uint32_t* flag_next) {
    constexpr int G = kWave / S;
    const int lane = lane_id(), sub = lane / S, sl = lane % S;
    const uint64_t gmask = (S == kWave ? ~0ull : ((1ull << S) - 1)) << (sub * S);
    const int64_t waves = int64_t(nblk) * (kBlock / kWave);
    for (int64_t g0 = (int64_t(blk) * (kBlock / kWave) + threadIdx.x / kWave) * G; g0 < len; g0 += waves * G) {
        const int64_t idx = g0 + sub;
        const bool live = idx < len;
        const int64_t p = base + idx;
        const int64_t v = live ? list[p] : 0;
        int64_t a = 0;
        int deg = 0;
        if (live) {
            a = rowptr[v];
            deg = int(rowptr[v + 1] - a);
        }
        const int c = sl < deg ? col[a + sl] : -1;
        if (live) slots[idx * S + sl] = sl < deg ? lpos[c] : -1;
        const bool valid = sl < deg && c != v;
        const uint64_t h = valid ? mix64(uint64_t(uint32_t(c)) ^ key) : ~0ull;
        const uint64_t hmin = group_min_u64<S>(h);
        const int lmin = group_min_i32<S>((valid && h == hmin) ? c : INT_MAX);
        const bool any = (__ballot(valid) & gmask) != 0;
        if (live && sl == 0) {
            const int own = int(v), cand = any ? lmin : own;
            lab_out[p] = is_active(v, key) ? cand : own;
            if (cand != own) *flag_next = 1u;
        }
    }
}

// The first sweep over the five short-row lists; slots: their padded entries.
__global__ __launch_bounds__(kBlock) void k_first_small(SmallRows fr, const int64_t* rowptr, const int32_t* col,
                                                        const int32_t* lpos, int32_t* slots, int32_t* lab_out,
                                                        uint64_t key, uint32_t* flag_next) {
    unsigned blk, nblk;
    const int k = small_list(fr, &blk, &nblk);
    const int64_t len = fr.len[k];
    int32_t* sk = slots + fr.slot[k];
    switch (k) {
        case kSmWave:
            first_rows<kWave>(fr.list, fr.base[k], len, blk, nblk, rowptr, col, lpos, sk, lab_out, key, flag_next);
            break;
        case kSm32:
            first_rows<kSub32>(fr.list, fr.base[k], len, blk, nblk, rowptr, col, lpos, sk, lab_out, key, flag_next);
            break;
        case kSm16:
            first_rows<kSub16>(fr.list, fr.base[k], len, blk, nblk, rowptr, col, lpos, sk, lab_out, key, flag_next);
            break;
        case kSm8:
            first_rows<kSub8>(fr.list, fr.base[k], len, blk, nblk, rowptr, col, lpos, sk, lab_out, key, flag_next);
            break;
        default:
            first_rows<kSub4>(fr.list, fr.base[k], len, blk, nblk, rowptr, col, lpos, sk, lab_out, key, flag_next);
            break;
    }
}

// ------------------------------------------------------------- workgroup rows

template <int BS = kBlock>
__device__ __forceinline__ int block_max_i32(int v, int* s) {
    v = wave_max(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) s[w] = v;
    __syncthreads();
    int r = s[0];
    for (int i = 1; i < BS / kWave; ++i) r = s[i] > r ? s[i] : r;
    __syncthreads();
    return r;
}
template <int BS = kBlock>
__device__ __forceinline__ uint64_t block_min_u64(uint64_t v, uint64_t* s) {
    v = wave_min_u64(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) s[w] = v;
    __syncthreads();
    uint64_t r = s[0];
    for (int i = 1; i < BS / kWave; ++i) r = s[i] < r ? s[i] : r;
    __syncthreads();
    return r;
}


// A count-table slot holds its label in the high and its count in the low 32
// bits (in LDS and in the workspace alike), so claiming a free slot and counting
// the first occurrences take one atomic.
constexpr unsigned long long kSlotEmpty = 0xFFFFFFFF00000000ull;  // label -1, count 0
__device__ __forceinline__ int slot_label(unsigned long long e) { return int(uint32_t(e >> 32)); }
__device__ __forceinline__ int slot_count(unsigned long long e) { return int(uint32_t(e)); }

// Adds k to the count of label L in an open-addressing table of cap slots.
__device__ __forceinline__ void tab_add(unsigned long long* t, int64_t cap, int L, int k) {
    const unsigned long long mine = (uint64_t(uint32_t(L)) << 32) | uint32_t(k);
    int64_t slot = int64_t(mix64(uint64_t(uint32_t(L))) & uint64_t(cap - 1));
    while (true) {
        const unsigned long long prev = atomicCAS(&t[slot], kSlotEmpty, mine);
        if (prev == kSlotEmpty) return;  // claimed with the count
        if (slot_label(prev) == L) {
            atomicAdd(&t[slot], (unsigned long long)uint32_t(k));
            return;
        }
        slot = (slot + 1) & (cap - 1);
    }
}

// Inserts the labels of one wavefront's 64 edges (L valid where `valid`): the
// most frequent labels of the slice (once clusters form, most neighbours share
// one) are peeled off by ballot and added once each, the rest lane by lane.
// Must be reached by the whole wavefront.
__device__ __forceinline__ void tab_add_wave(unsigned long long* t, int64_t cap, bool valid, int L) {
    bool pending = valid;
    for (int it = 0; it < 3; ++it) {
        const uint64_t m = __ballot(pending);
        if (!m) return;
        const int leader = __builtin_ctzll(m);
        const int Ld = __shfl(L, leader, kWave);
        const uint64_t same = __ballot(pending && L == Ld);
        if (lane_id() == leader) tab_add(t, cap, Ld, __popcll(same));
        if (pending && L == Ld) pending = false;
    }
    if (pending) tab_add(t, cap, L, 1);
}

// Inserts the labels of the edges [first + 64 k stride ... ) of one row, k <
// R, each wavefront's 64-edge slices: every column and label load is issued
// before the first insertion, so a row costs one round trip to memory, not one
// per slice.  first and stride are uniform over the wavefront.
template <int R>
__device__ __forceinline__ void tab_add_row(unsigned long long* t, int64_t cap, int64_t first, int64_t stride,
                                            int64_t b, int64_t p, const int32_t* ncol, const int32_t* lab_in) {
    int c[R], L[R];
#pragma unroll
    for (int k = 0; k < R; ++k) {
        const int64_t e = first + k * stride + lane_id();
        c[k] = e < b ? ncol[e] : int(p);
    }
#pragma unroll
    for (int k = 0; k < R; ++k) L[k] = c[k] != p ? lab_in[c[k]] : -1;
#pragma unroll
    for (int k = 0; k < R; ++k)
        if (first + k * stride < b) tab_add_wave(t, cap, c[k] != p, L[k]);
}

// One workgroup per listed row (rows up to kLdsRowMax).  Table: keys (label or
// -1) and counts in LDS.  The rows are list[base + [0, len)]; roff, ncol and
// the labels are by list position.
template <int BS>
__global__ __launch_bounds__(BS) void k_lp_block(const int32_t* list, int64_t base, const int64_t* list_len,
                                                 const int64_t* roff, const int32_t* ncol, const int32_t* lab_in,
                                                 int32_t* lab_out, uint64_t key, const uint32_t* flag_prev,
                                                 uint32_t* flag_next) {
    __shared__ unsigned long long s_tab[kLdsTable];
    __shared__ int s_red[BS / kWave];
    __shared__ uint64_t s_red64[BS / kWave];
    const bool converged = *flag_prev == 0;
    const int64_t len = *list_len;
    for (int64_t idx = blockIdx.x; idx < len; idx += gridDim.x) {
        const int64_t p = base + idx;
        const int own = lab_in[p];
        if (converged) {
            if (threadIdx.x == 0) lab_out[p] = own;
            continue;
        }
        const int64_t v = list[p];
        const int64_t a = roff[p], b = roff[p + 1];
        const int64_t deg = b - a;
        int64_t cap = 1;
        while (cap < 2 * deg) cap <<= 1;
        unsigned long long* t = s_tab;
        for (int64_t s = threadIdx.x; s < cap; s += BS) t[s] = kSlotEmpty;
        __syncthreads();
        // wave-uniform rounds: each wavefront takes 64 consecutive edges per round
        tab_add_row<(kLdsRowMax + BS - 1) / BS>(t, cap, a + (threadIdx.x & ~(kWave - 1)), BS, b, p, ncol, lab_in);
        __syncthreads();
        int best = 0, own_cnt = 0;
        for (int64_t s = threadIdx.x; s < cap; s += BS) {
            const unsigned long long en = t[s];
            const int k = slot_label(en);
            if (k < 0) continue;
            const int c = slot_count(en);
            best = c > best ? c : best;
            if (k == own) own_cnt = c;
        }
        best = block_max_i32<BS>(best, s_red);
        own_cnt = block_max_i32<BS>(own_cnt, s_red);
        int cand = own;
        if (best > 0 && own_cnt != best) {
            uint64_t hbest = ~0ull;
            for (int64_t s = threadIdx.x; s < cap; s += BS) {
                const unsigned long long en = t[s];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(k)) ^ key);
                hbest = h < hbest ? h : hbest;
            }
            hbest = block_min_u64<BS>(hbest, s_red64);
            uint64_t lbest = ~0ull;
            for (int64_t s = threadIdx.x; s < cap; s += BS) {
                const unsigned long long en = t[s];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                if (mix64(uint64_t(uint32_t(k)) ^ key) != hbest) continue;
                lbest = uint64_t(uint32_t(k)) < lbest ? uint64_t(uint32_t(k)) : lbest;
            }
            cand = int(block_min_u64<BS>(lbest, s_red64));
        }
        if (threadIdx.x == 0) {
            lab_out[p] = is_active(v, key) ? cand : own;
            if (cand != own) *flag_next = 1u;
        }
        __syncthreads();
    }
}

// One wavefront per listed row (64 < deg <= kWaveTabRowMax), the same
// function as k_lp_block with the count table in the wavefront's own slice of
// LDS: the lanes of one wavefront meet only at wavefront-scope fences.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__global__ __launch_bounds__(kBlock) void k_lp_wavetab(const int32_t* list, int64_t base, const int64_t* list_len,
                                                       const int64_t* roff, const int32_t* ncol,
                                                       const int32_t* lab_in, int32_t* lab_out, uint64_t key,
                                                       const uint32_t* flag_prev, uint32_t* flag_next) {
    __shared__ unsigned long long s_tab[kBlock / kWave][kWaveTab];
    const int w = threadIdx.x / kWave, lane = lane_id();
    unsigned long long* t = s_tab[w];
    const bool converged = *flag_prev == 0;
    const int64_t len = *list_len;
    const int64_t waves = int64_t(gridDim.x) * (kBlock / kWave);
    for (int64_t idx = int64_t(blockIdx.x) * (kBlock / kWave) + w; idx < len; idx += waves) {
        const int64_t p = base + idx;
        const int own = lab_in[p];
        if (converged) {
            if (lane == 0) lab_out[p] = own;
            continue;
        }
        const int64_t v = list[p];
        const int64_t a = roff[p], b = roff[p + 1];
        int cap = 1;
        while (cap < 2 * (b - a)) cap <<= 1;  // <= kWaveTab
        for (int s2 = lane; s2 < cap; s2 += kWave) t[s2] = kSlotEmpty;
        wave_lds_sync();
        tab_add_row<kWaveTabRowMax / kWave>(t, cap, a, kWave, b, p, ncol, lab_in);
        wave_lds_sync();
        int best = 0, own_cnt = 0;
        for (int s2 = lane; s2 < cap; s2 += kWave) {
            const unsigned long long en = t[s2];
            const int k = slot_label(en);
            if (k < 0) continue;
            const int c = slot_count(en);
            best = c > best ? c : best;
            if (k == own) own_cnt = c;
        }
        best = wave_max(best);
        own_cnt = wave_max(own_cnt);
        int cand = own;
        if (best > 0 && own_cnt != best) {
            uint64_t hbest = ~0ull;
            for (int s2 = lane; s2 < cap; s2 += kWave) {
                const unsigned long long en = t[s2];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(k)) ^ key);
                hbest = h < hbest ? h : hbest;
            }
            hbest = wave_min_u64(hbest);
            int lbest = INT_MAX;
            for (int s2 = lane; s2 < cap; s2 += kWave) {
                const unsigned long long en = t[s2];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                if (mix64(uint64_t(uint32_t(k)) ^ key) != hbest) continue;
                lbest = k < lbest ? k : lbest;
            }
            cand = wave_min_i32(lbest);
        }
        if (lane == 0) {
            lab_out[p] = is_active(v, key) ? cand : own;
            if (cand != own) *flag_next = 1u;
        }
        wave_lds_sync();  // every lane is done with the table before the next row clears it
    }
}

// First sweep, rows of more than 64 edges: BS threads per row (one wavefront,
// or the workgroup), each lane keeping the smallest hash of its edges and
// writing their list positions to ncol.
template <int BS>
__global__ __launch_bounds__(BS > kBlock ? BS : kBlock) void k_first_wide(const int32_t* list, int64_t base,
                                                                          const int64_t* list_len,
                                                                          const int64_t* rowptr, const int32_t* col,
                                                                          const int64_t* roff, const int32_t* lpos,
                                                                          int32_t* ncol, int32_t* lab_out,
                                                                          uint64_t key, uint32_t* flag_next) {
    constexpr int kThreads = BS > kBlock ? BS : kBlock;
    constexpr int kRowsPer = kThreads / BS;  // rows a workgroup takes at once
    __shared__ uint64_t s_red64[kThreads / kWave];
    __shared__ int s_any[kThreads / kWave];
    const int64_t len = *list_len;
    const int t = threadIdx.x % BS;
    for (int64_t idx0 = int64_t(blockIdx.x) * kRowsPer; idx0 < len; idx0 += int64_t(gridDim.x) * kRowsPer) {
        const int64_t idx = idx0 + threadIdx.x / BS;
        const bool live = idx < len;  // uniform over a row's BS threads
        const int64_t p = base + idx;
        const int64_t v = live ? list[p] : 0;
        uint64_t hb = ~0ull;
        int cb = INT_MAX;
        bool any = false;
        if (live) {
            const int64_t a = rowptr[v], b = rowptr[v + 1];
            const int64_t shift = roff[p] - a;  // entry e of the row goes to ncol[e + shift]
            for (int64_t e = a + t; e < b; e += BS) {
                const int c = col[e];
                ncol[e + shift] = lpos[c];
                if (c == v) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(c)) ^ key);
                if (h < hb || (h == hb && c < cb)) {
                    hb = h;
                    cb = c;
                }
                any = true;
            }
        }
        uint64_t hmin;
        int lmin;
        bool anyr;
        if constexpr (BS == kWave) {
            hmin = wave_min_u64(hb);
            lmin = wave_min_i32(hb == hmin ? cb : INT_MAX);
            anyr = __ballot(any) != 0;
        } else {
            hmin = block_min_u64<BS>(hb, s_red64);
            lmin = int(block_min_u64<BS>(hb == hmin ? uint64_t(uint32_t(cb)) : ~0ull, s_red64));
            anyr = block_max_i32<BS>(any ? 1 : 0, s_any) != 0;
        }
        if (live && t == 0) {
            const int own = int(v), cand = anyr ? lmin : own;
            lab_out[p] = is_active(v, key) ? cand : own;
            if (cand != own) *flag_next = 1u;
        }
    }
}

// -------------------------------------------------------------- very long rows
// The edges and the table slots of each listed row are cut into chunks,
// numbered one after the other over all listed rows and dealt over the grid,
// so a row of a million edges is spread over the chip and many long rows share
// it.  Per-row
// results: best count, own label's count, smallest hash among the best, and the
// smallest label with that hash, combined with atomics (max / min: the result
// does not depend on the order).

struct BigRows {
    const int32_t* list;  // the listed rows, at list positions base + [0, len)
    int64_t base;
    const int64_t* len;
    const int64_t* off;   // table offset of each listed row
    const int64_t* echunk;  // [listed rows + 1]: first edge chunk of each row (kBigEdgeChunk edges per chunk)
    const int64_t* schunk;  // [listed rows + 1]: first table-slot chunk of each row (kSlotChunk slots per chunk)
    unsigned long long* tab;  // count tables: slot = label << 32 | count, kSlotEmpty when free
    int* best;            // [listed rows]
    int* own_cnt;
    unsigned long long* hbest;
    unsigned long long* lbest;
};

__device__ __forceinline__ int64_t table_cap(int64_t deg) {
    int64_t cap = 1;
    while (cap < 2 * deg) cap <<= 1;
    return cap;
}

// Table slots of every listed row in chunks of kSlotChunk; the chunks of all
// rows are numbered one after the other (the offsets are computed once per
// call) and dealt over the grid, so every row gets as many workgroups as its
// table needs and a workgroup finds its row by a binary search.
constexpr int64_t kSlotChunk = 2048;

// The listed row holding global chunk c (the last idx with off[idx] <= c).
__device__ __forceinline__ int64_t chunk_row(const int64_t* __restrict__ off, int64_t len, int64_t c) {
    int64_t lo = 0, hi = len;
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (off[mid] <= c) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Exclusive prefix of v over the workgroup in thread order; *total = the sum.
constexpr int kPrepThreads = 1024;
__device__ __forceinline__ int64_t prep_exscan(int64_t v, int64_t* s, int64_t* total) {
    const int lane = lane_id(), w = threadIdx.x / kWave;
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) s[w] = x;
    __syncthreads();
    int64_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < kPrepThreads / kWave; ++i) {
        const int64_t t = s[i];
        if (i < w) before += t;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return before + x - v;
}

// One workgroup: the first edge chunk (echunk), first slot chunk (schunk) and
// table offset (off) of every listed row, each an exclusive scan with the
// total at [len].
__global__ __launch_bounds__(kPrepThreads) void k_big_prep(const int32_t* __restrict__ list,
                                                           const int64_t* __restrict__ len_p,
                                                           const int64_t* __restrict__ rowptr,
                                                           int64_t* __restrict__ echunk, int64_t* __restrict__ schunk,
                                                           int64_t* __restrict__ off) {
    __shared__ int64_t s[kPrepThreads / kWave];
    const int64_t len = *len_p;
    int64_t run_e = 0, run_s = 0, run_o = 0;
    for (int64_t base = 0; base < len; base += kPrepThreads) {
        const int64_t idx = base + threadIdx.x;
        int64_t ne = 0, ns = 0, cap = 0;
        if (idx < len) {
            const int64_t v = list[idx];
            const int64_t deg = rowptr[v + 1] - rowptr[v];
            cap = table_cap(deg);
            ne = cdiv(deg, kBigEdgeChunk);
            ns = cdiv(cap, kSlotChunk);
        }
        int64_t te, ts, to;
        const int64_t pe = prep_exscan(ne, s, &te);
        const int64_t ps = prep_exscan(ns, s, &ts);
        const int64_t po = prep_exscan(cap, s, &to);
        if (idx < len) {
            echunk[idx] = run_e + pe;
            schunk[idx] = run_s + ps;
            off[idx] = run_o + po;
        }
        run_e += te;
        run_s += ts;
        run_o += to;
    }
    if (threadIdx.x == 0) {
        echunk[len] = run_e;
        schunk[len] = run_s;
        off[len] = run_o;
    }
}

// Tables of up to kFusedCap slots are reduced, decided and cleared by one
// workgroup each (k_big_fused); the chunked passes below handle the larger ones.
constexpr int64_t kFusedCap = 65536;
constexpr int kFusedThreads = 1024;

// all: every table (its first use); else only those over kFusedCap slots.
__global__ __launch_bounds__(kBlock) void k_big_clear(BigRows br, const int64_t* rowptr, const uint32_t* flag_prev,
                                                      bool all) {
    if (*flag_prev == 0) return;
    const int64_t len = *br.len;
    const int64_t total = br.schunk[len];
    for (int64_t c = blockIdx.x; c < total; c += gridDim.x) {
        const int64_t idx = chunk_row(br.schunk, len, c);
        const int64_t v = br.list[idx];
        const int64_t cap = table_cap(rowptr[v + 1] - rowptr[v]);
        if (!all && cap <= kFusedCap) continue;
        const int64_t j = c - br.schunk[idx];
        unsigned long long* tab = br.tab + br.off[idx];
        const int64_t s1 = (j + 1) * kSlotChunk < cap ? (j + 1) * kSlotChunk : cap;
        for (int64_t s = j * kSlotChunk + threadIdx.x; s < s1; s += kBlock) tab[s] = kSlotEmpty;
    }
    const int64_t stride = int64_t(gridDim.x) * kBlock, start = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    for (int64_t idx = start; idx < len; idx += stride) {
        br.best[idx] = 0;
        br.own_cnt[idx] = 0;
        br.hbest[idx] = ~0ull;
        br.lbest[idx] = ~0ull;
    }
}

// Chunks of kBigEdgeChunk edges of every listed row, dealt over the grid: each
// chunk is counted in an LDS table first, then its distinct labels are added
// to the row's table in the workspace (far fewer global atomics where
// neighbour labels repeat, as they do once clusters form).
__global__ __launch_bounds__(kBlock) void k_big_insert(BigRows br, const int64_t* roff, const int32_t* ncol,
                                                       const int32_t* lab_in, const uint32_t* flag_prev) {
    __shared__ unsigned long long s_tab[kBigChunkTab];
    if (*flag_prev == 0) return;
    const int64_t len = *br.len;
    const int64_t total = br.echunk[len];
    for (int64_t c = blockIdx.x; c < total; c += gridDim.x) {
        const int64_t idx = chunk_row(br.echunk, len, c);
        const int64_t p = br.base + idx;
        const int64_t a = roff[p], b = roff[p + 1];
        const int64_t cap = table_cap(b - a);
        const int64_t j = c - br.echunk[idx];
        unsigned long long* tab = br.tab + br.off[idx];
        for (int x = threadIdx.x; x < kBigChunkTab; x += kBlock) s_tab[x] = kSlotEmpty;
        __syncthreads();
        const int64_t e0 = a + j * kBigEdgeChunk;
        const int64_t e1 = e0 + kBigEdgeChunk < b ? e0 + kBigEdgeChunk : b;
        // every slice's column and label loads are issued before the first insertion
        constexpr int R = kBigEdgeChunk / kBlock;
        const int64_t w0 = e0 + (threadIdx.x & ~(kWave - 1));
        int cc[R], L[R];
#pragma unroll
        for (int k = 0; k < R; ++k) {
            const int64_t e = w0 + k * kBlock + lane_id();
            cc[k] = e < e1 ? ncol[e] : int(p);
        }
#pragma unroll
        for (int k = 0; k < R; ++k) L[k] = cc[k] != p ? lab_in[cc[k]] : -1;
#pragma unroll
        for (int k = 0; k < R; ++k)
            if (w0 + k * kBlock < e1) tab_add_wave(s_tab, kBigChunkTab, cc[k] != p, L[k]);
        __syncthreads();
        // the chunk's distinct labels into the row's table: the first probe of every slot the thread holds is
        // issued before any result is used, so a chunk of many distinct labels costs about one round trip
        constexpr int Q = kBigChunkTab / kBlock;
        unsigned long long en[Q], prev[Q];
        int64_t slot[Q];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            en[q] = s_tab[threadIdx.x + q * kBlock];  // the chunk's count of its label
            slot[q] = int64_t(mix64(uint64_t(uint32_t(slot_label(en[q])))) & uint64_t(cap - 1));
        }
#pragma unroll
        for (int q = 0; q < Q; ++q) prev[q] = slot_label(en[q]) >= 0 ? atomicCAS(&tab[slot[q]], kSlotEmpty, en[q])
                                                                     : kSlotEmpty;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int Lq = slot_label(en[q]);
            unsigned long long pv = prev[q];
            int64_t sl = slot[q];
            while (pv != kSlotEmpty) {  // kSlotEmpty: claimed with the count (or no label)
                if (slot_label(pv) == Lq) {
                    atomicAdd(&tab[sl], (unsigned long long)uint32_t(slot_count(en[q])));
                    break;
                }
                sl = (sl + 1) & (cap - 1);
                pv = atomicCAS(&tab[sl], kSlotEmpty, en[q]);
            }
        }
        __syncthreads();
    }
}

// pass 0: best count and the own label's count; 1: smallest hash among the
// best labels; 2: smallest label with that hash (passes 1-2 only where the own
// label is not among the best).  Each slot chunk reduces in its workgroup and
// adds its result with one atomic.
template <int kPass>
__global__ __launch_bounds__(kBlock) void k_big_reduce(BigRows br, const int64_t* rowptr, const int32_t* lab_in,
                                                       uint64_t key, const uint32_t* flag_prev) {
    __shared__ int s_red[kBlock / kWave];
    __shared__ uint64_t s_red64[kBlock / kWave];
    if (*flag_prev == 0) return;
    const int64_t len = *br.len;
    const int64_t total = br.schunk[len];
    for (int64_t c = blockIdx.x; c < total; c += gridDim.x) {
        const int64_t idx = chunk_row(br.schunk, len, c);
        const int64_t v = br.list[idx];
        const int64_t cap = table_cap(rowptr[v + 1] - rowptr[v]);
        if (cap <= kFusedCap) continue;  // k_big_fused's (uniform across the workgroup)
        const int64_t j = c - br.schunk[idx];
        const int64_t s0 = j * kSlotChunk, s1 = (j + 1) * kSlotChunk < cap ? (j + 1) * kSlotChunk : cap;
        const int own = lab_in[br.base + idx];
        const unsigned long long* tab = br.tab + br.off[idx];
        if (kPass == 0) {
            int best = 0, oc = 0;
            for (int64_t s = s0 + threadIdx.x; s < s1; s += kBlock) {
                const unsigned long long en = tab[s];
                const int k = slot_label(en);
                if (k < 0) continue;
                const int cnt = slot_count(en);
                best = cnt > best ? cnt : best;
                if (k == own) oc = cnt;
            }
            best = block_max_i32(best, s_red);
            oc = block_max_i32(oc, s_red);
            if (threadIdx.x == 0) {
                if (best) atomicMax(&br.best[idx], best);
                if (oc) atomicMax(&br.own_cnt[idx], oc);
            }
        } else {
            const int best = br.best[idx];
            if (best == 0 || br.own_cnt[idx] == best) continue;  // uniform across the workgroup
            const uint64_t hb = kPass == 2 ? br.hbest[idx] : 0;
            uint64_t r = ~0ull;
            for (int64_t s = s0 + threadIdx.x; s < s1; s += kBlock) {
                const unsigned long long en = tab[s];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(k)) ^ key);
                if (kPass == 1) r = h < r ? h : r;
                else if (h == hb) r = uint64_t(uint32_t(k)) < r ? uint64_t(uint32_t(k)) : r;
            }
            r = block_min_u64(r, s_red64);
            if (threadIdx.x == 0 && r != ~0ull) atomicMin(kPass == 1 ? &br.hbest[idx] : &br.lbest[idx], r);
        }
    }
}

// One workgroup per row whose table has at most kFusedCap slots: the best
// count and the own label's count, the tie-break when the own label is not
// among the best, the new label, then the table cleared for the next sweep.
__global__ __launch_bounds__(kFusedThreads) void k_big_fused(BigRows br, const int64_t* rowptr,
                                                             const int32_t* lab_in, int32_t* lab_out, uint64_t key,
                                                             const uint32_t* flag_prev, uint32_t* flag_next) {
    __shared__ int s_red[kFusedThreads / kWave];
    __shared__ uint64_t s_red64[kFusedThreads / kWave];
    const bool converged = *flag_prev == 0;
    const int64_t len = *br.len;
    for (int64_t idx = blockIdx.x; idx < len; idx += gridDim.x) {
        const int64_t v = br.list[idx];
        const int64_t cap = table_cap(rowptr[v + 1] - rowptr[v]);
        if (cap > kFusedCap) continue;  // uniform across the workgroup
        const int64_t p = br.base + idx;
        const int own = lab_in[p];
        if (converged) {  // the insert did not run: the table is still clear
            if (threadIdx.x == 0) lab_out[p] = own;
            continue;
        }
        unsigned long long* tab = br.tab + br.off[idx];
        int best = 0, own_cnt = 0;
        for (int64_t q = threadIdx.x; q < cap; q += kFusedThreads) {
            const unsigned long long en = tab[q];
            const int k = slot_label(en);
            if (k < 0) continue;
            const int c = slot_count(en);
            best = c > best ? c : best;
            if (k == own) own_cnt = c;
        }
        best = block_max_i32<kFusedThreads>(best, s_red);
        own_cnt = block_max_i32<kFusedThreads>(own_cnt, s_red);
        int cand = own;
        if (best > 0 && own_cnt != best) {
            uint64_t hbest = ~0ull;
            for (int64_t q = threadIdx.x; q < cap; q += kFusedThreads) {
                const unsigned long long en = tab[q];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(k)) ^ key);
                hbest = h < hbest ? h : hbest;
            }
            hbest = block_min_u64<kFusedThreads>(hbest, s_red64);
            uint64_t lbest = ~0ull;
            for (int64_t q = threadIdx.x; q < cap; q += kFusedThreads) {
                const unsigned long long en = tab[q];
                const int k = slot_label(en);
                if (k < 0 || slot_count(en) != best) continue;
                if (mix64(uint64_t(uint32_t(k)) ^ key) != hbest) continue;
                lbest = uint64_t(uint32_t(k)) < lbest ? uint64_t(uint32_t(k)) : lbest;
            }
            cand = int(block_min_u64<kFusedThreads>(lbest, s_red64));
        }
        if (threadIdx.x == 0) {
            lab_out[p] = is_active(v, key) ? cand : own;
            if (cand != own) *flag_next = 1u;
        }
        __syncthreads();  // every read of the table is done
        for (int64_t q = threadIdx.x; q < cap; q += kFusedThreads) tab[q] = kSlotEmpty;
    }
}

// skip_fused: rows of tables up to kFusedCap slots are k_big_fused's.
__global__ void k_big_decide(BigRows br, const int64_t* rowptr, const int32_t* lab_in, int32_t* lab_out,
                             uint64_t key, const uint32_t* flag_prev, uint32_t* flag_next, bool skip_fused) {
    const bool converged = *flag_prev == 0;
    const int64_t len = *br.len;
    for (int64_t idx = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; idx < len;
         idx += int64_t(gridDim.x) * blockDim.x) {
        const int64_t v = br.list[idx];
        if (skip_fused && table_cap(rowptr[v + 1] - rowptr[v]) <= kFusedCap) continue;
        const int64_t p = br.base + idx;
        const int own = lab_in[p];
        if (converged) {
            lab_out[p] = own;
            continue;
        }
        const int best = br.best[idx];
        const int cand = (best > 0 && br.own_cnt[idx] != best) ? int(br.lbest[idx]) : own;
        lab_out[p] = is_active(v, key) ? cand : own;
        if (cand != own) *flag_next = 1u;
    }
}

// First sweep of the very long rows: per-row results reset (the tables are
// not used), the smallest hash over every chunk of edges (combined with a 64-bit
// atomic minimum; the columns' list positions go to ncol), then the neighbour
// with that hash; k_big_decide finishes.
__global__ void k_big_first_reset(BigRows br) {
    const int64_t len = *br.len;
    for (int64_t idx = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; idx < len;
         idx += int64_t(gridDim.x) * blockDim.x) {
        br.best[idx] = 0;
        br.own_cnt[idx] = 0;
        br.hbest[idx] = ~0ull;
        br.lbest[idx] = ~0ull;
    }
}

template <int kPass>
__global__ __launch_bounds__(kBlock) void k_big_first(BigRows br, const int64_t* rowptr, const int32_t* col,
                                                      const int64_t* roff, const int32_t* lpos, int32_t* ncol,
                                                      uint64_t key) {
    __shared__ uint64_t s_red64[kBlock / kWave];
    __shared__ int s_any[kBlock / kWave];
    const int64_t len = *br.len;
    const int64_t total = br.echunk[len];
    for (int64_t ch = blockIdx.x; ch < total; ch += gridDim.x) {
        const int64_t idx = chunk_row(br.echunk, len, ch);
        const int64_t v = br.list[idx];
        const int64_t a = rowptr[v], b = rowptr[v + 1];
        const int64_t j = ch - br.echunk[idx];
        const int64_t e0 = a + j * kBigEdgeChunk;
        const int64_t e1 = e0 + kBigEdgeChunk < b ? e0 + kBigEdgeChunk : b;
        if (kPass == 0) {
            uint64_t hb = ~0ull;
            bool any = false;
            const int64_t shift = roff[br.base + idx] - a;  // entry e of the row goes to ncol[e + shift]
            for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
                const int c = col[e];
                ncol[e + shift] = lpos[c];
                if (c == v) continue;
                const uint64_t h = mix64(uint64_t(uint32_t(c)) ^ key);
                hb = h < hb ? h : hb;
                any = true;
            }
            hb = block_min_u64(hb, s_red64);
            const bool anyr = block_max_i32(any ? 1 : 0, s_any) != 0;
            if (threadIdx.x == 0 && anyr) {
                atomicMin(&br.hbest[idx], (unsigned long long)hb);
                atomicMax(&br.best[idx], 1);
            }
        } else {
            const uint64_t hb = br.hbest[idx];
            for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
                const int c = col[e];
                if (c != v && mix64(uint64_t(uint32_t(c)) ^ key) == hb) br.lbest[idx] = uint64_t(uint32_t(c));
            }
        }
    }
}

// --------------------------------------------------------------------- order

// lab[list[p]] = lab_pos[p]: the labels from list positions to node ids.
__global__ void k_labels_by_node(int64_t n, const int32_t* list, const int32_t* lab_pos, int32_t* lab) {
    for (int64_t p = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; p < n; p += int64_t(gridDim.x) * blockDim.x)
        lab[list[p]] = lab_pos[p];
}

// Sort key of row v: (label, dmax - off-diagonal entries) in bits_for(n) +
// dbits bits, dmax the largest off-diagonal entry count (< 2^dbits).
__global__ void k_order_keys(int64_t n, const int32_t* lab, const uint32_t* deg_off, uint32_t dmax, int dbits,
                             uint64_t* keys) {
    for (int64_t v = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; v < n; v += int64_t(gridDim.x) * blockDim.x)
        keys[v] = (uint64_t(uint32_t(lab[v])) << dbits) | uint64_t(dmax - deg_off[v]);
}

__global__ void k_finish_order(int64_t n, const uint32_t* sorted_ids, const int32_t* lab, int32_t* perm,
                               int32_t* iperm, int32_t* labels) {
    for (int64_t r = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; r < n; r += int64_t(gridDim.x) * blockDim.x) {
        const uint32_t old = sorted_ids[r];
        perm[r] = int32_t(old);
        iperm[old] = int32_t(r);
        if (labels) labels[r] = lab[r];
    }
}

struct ReorderWs {
    uint32_t* flags;
    int32_t* lab[2];
    uint32_t* deg_off;
    int32_t* blk_cnt;     // [kClasses * blocks]: rows of each class in each 256-row block
    int64_t* blk_off;     // [kClasses * blocks + 1]: their exclusive scan
    int32_t* list;        // [n]: the rows, class after class
    int32_t* lpos;        // [n]: each row's position in list
    uint32_t* ldeg;       // [n]: entry counts by list position
    int64_t* roff;        // [n + 1]: their exclusive scan
    int32_t* ncol;        // [nnz]: the rows' entries in list order, as list positions (longer rows)
    int32_t* slots;       // [2 nnz + 4 n]: the short rows' entries, padded per list
    int64_t* class_info;  // [2 * kClasses + 3]: first list position and rows of each class; largest
                          // off-diagonal entry count; the CSR check's flags (low 32 bits); entries of the
                          // rows of more than kWaveRowMax entries
    uint32_t* blk_max;    // [blocks]: largest off-diagonal entry count of each 256-row block
    uint32_t* blk_long;   // [blocks]: entries of each block's rows of more than kWaveRowMax entries
    int64_t* huge_off;
    int64_t* huge_echunk;
    int64_t* huge_schunk;
    unsigned long long* tab;
    int* big_best;
    int* big_own;
    unsigned long long* big_hbest;
    unsigned long long* big_lbest;
    uint64_t* sort_keys;
    uint32_t* sort_vals;
    ScanTmp scan;
    SortTmp sort;
};

inline unsigned grid_cap(int64_t rows, int64_t per_block, unsigned cap) {
    const int64_t g = cdiv(rows, per_block);
    return unsigned(g < 1 ? 1 : (g > cap ? cap : g));
}

ReorderWs carve(Ws& ws, int64_t n, int64_t nnz, int32_t iters) {
    ReorderWs r;
    const int64_t n1 = n > 0 ? n : 1;
    (void)iters;
    r.flags = ws.take<uint32_t>(size_t(kMaxSweeps + 2));
    r.lab[0] = ws.take<int32_t>(n1);
    r.lab[1] = ws.take<int32_t>(n1);
    r.deg_off = ws.take<uint32_t>(n1);
    const int64_t nblk = cdiv(n1, kClsBlock);
    r.blk_cnt = ws.take<int32_t>(size_t(kClasses * nblk));
    r.blk_off = ws.take<int64_t>(size_t(kClasses * nblk + 1));
    r.list = ws.take<int32_t>(n1);
    r.lpos = ws.take<int32_t>(n1);
    r.ldeg = ws.take<uint32_t>(n1);
    r.roff = ws.take<int64_t>(n1 + 1);
    r.ncol = ws.take<int32_t>(size_t(nnz > 0 ? nnz : 1));
    r.slots = ws.take<int32_t>(size_t(2 * (nnz > 0 ? nnz : 1) + 4 * n1));
    r.class_info = ws.take<int64_t>(2 * kClasses + 3);
    r.blk_max = ws.take<uint32_t>(size_t(nblk));
    r.blk_long = ws.take<uint32_t>(size_t(nblk));
    r.huge_off = ws.take<int64_t>(n1 + 1);
    r.huge_echunk = ws.take<int64_t>(n1 + 1);
    r.huge_schunk = ws.take<int64_t>(n1 + 1);
    const int64_t tab = 4 * (nnz > 0 ? nnz : 1);  // sum over big rows of cap <= 4 * deg
    r.tab = ws.take<unsigned long long>(size_t(tab));
    r.big_best = ws.take<int>(n1);
    r.big_own = ws.take<int>(n1);
    r.big_hbest = ws.take<unsigned long long>(n1);
    r.big_lbest = ws.take<unsigned long long>(n1);
    r.sort_keys = ws.take<uint64_t>(n1);
    r.sort_vals = ws.take<uint32_t>(n1);
    const int64_t scan_n = n1 + 1 > kClasses * nblk + 1 ? n1 + 1 : kClasses * nblk + 1;
    r.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(scan_n)));
    r.sort = sort_tmp(ws, n1, 8, true);
    return r;
}

}  // namespace

}  // namespace gt

using namespace gt;

extern "C" size_t gt_reorder_workspace_size(int64_t n, int64_t nnz) {
    Ws ws(nullptr);
    carve(ws, n, nnz, kMaxSweeps);
    return ws.size();
}

extern "C" gt_status gt_reorder_streams(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                                        int32_t iters, uint64_t seed, int32_t* perm, int32_t* iperm, int32_t* labels,
                                        int32_t* sweeps_done, void* ws_ptr, size_t ws_bytes, hipStream_t stream,
                                        const hipStream_t* side_streams, const hipEvent_t* events,
                                        int32_t n_side) {
    if (n < 0 || nnz < 0 || n >= (int64_t(1) << 31) || nnz >= (int64_t(1) << 32))
        return fail(GT_ERR_INVALID_ARG, "gt_reorder: n or nnz out of range");
    if (iters < 0 || iters > kMaxSweeps) return fail(GT_ERR_INVALID_ARG, "gt_reorder: iters must be in [0, 1000]");
    if (!rowptr || (nnz > 0 && !col) || (n > 0 && (!perm || !iperm)) || !ws_ptr)
        return fail(GT_ERR_INVALID_ARG, "gt_reorder: null pointer");
    if (ws_bytes < gt_reorder_workspace_size(n, nnz))
        return fail(GT_ERR_WORKSPACE, "gt_reorder: workspace too small");
    // The classes of a sweep read the sweep's input labels and write disjoint rows of its output: with side
    // streams they run side by side, the short rows and then the rows of 513 to 4096 entries on the caller's
    // stream, the long rows on the first side stream, the rows of 65 to 512 entries on the second (or the
    // first); each sweep starts when the previous one has finished on all of them.
    Spread sp;
    gt_status st = spread_open("gt_reorder", stream, side_streams, events, n_side, &sp);
    if (st != GT_OK) return st;
    if (n == 0) {
        if (sweeps_done) *sweeps_done = 0;
        return GT_OK;
    }
    Ws ws(ws_ptr);
    ReorderWs r = carve(ws, n, nnz, iters);
    // the CSR check and the row classes in one go: both come back to the host with one synchronisation,
    // and nothing past the classification runs unless the check passed
    uint32_t* vflag = reinterpret_cast<uint32_t*>(r.class_info + 2 * kClasses + 1);
    if ((st = fill_u32(vflag, 2, 0u, stream)) != GT_OK) return st;  // the high half of the slot too
    if ((st = launch_validate_csr(n, nnz, rowptr, col, vflag, stream)) != GT_OK) return st;
    const unsigned g = grid_for(n, 256, 8192);
    const int64_t nblk = cdiv(n, kClsBlock);
    unsigned long long* deg_max = reinterpret_cast<unsigned long long*>(r.class_info + 2 * kClasses);
    unsigned long long* long_sum = reinterpret_cast<unsigned long long*>(r.class_info + 2 * kClasses + 2);
    if ((st = fill_u32(reinterpret_cast<uint32_t*>(deg_max), 2, 0u, stream)) != GT_OK) return st;
    if ((st = fill_u32(reinterpret_cast<uint32_t*>(long_sum), 2, 0u, stream)) != GT_OK) return st;
    k_classify<<<unsigned(nblk), kClsBlock, 0, stream>>>(n, nnz, rowptr, col, r.deg_off, r.blk_cnt, nblk, r.blk_max,
                                                         r.blk_long);
    GT_LAUNCH_CHECK("reorder_classify");
    k_blocks_max<<<unsigned(cdiv(nblk, kMaxSpan)), 256, 0, stream>>>(nblk, r.blk_max, r.blk_long, deg_max, long_sum);
    GT_LAUNCH_CHECK("reorder_degree_max");
    if ((st = exclusive_scan_i32(r.blk_cnt, kClasses * nblk, r.blk_off, r.scan, stream)) != GT_OK) return st;
    k_class_scatter<<<unsigned(nblk), kClsBlock, 0, stream>>>(n, rowptr, r.blk_off, nblk, r.list, r.lpos,
                                                              r.ldeg);
    GT_LAUNCH_CHECK("reorder_class_scatter");
    if ((st = exclusive_scan_u32(r.ldeg, n, r.roff, r.scan, stream)) != GT_OK) return st;
    k_class_totals<<<1, 64, 0, stream>>>(nblk, r.blk_off, r.class_info);
    GT_LAUNCH_CHECK("reorder_class_totals");

    // the labels are kept by list position and start as the node ids
    GT_HIP(hipMemcpyAsync(r.lab[0], r.list, size_t(n) * sizeof(int32_t), hipMemcpyDeviceToDevice, stream));
    if ((st = fill_u32(r.flags, iters + 1, 0, stream)) != GT_OK) return st;
    if ((st = fill_u32(r.flags, 1, 1, stream)) != GT_OK) return st;

    // the class sizes on the host: empty classes are not launched and grids fit the lists
    int64_t info[2 * kClasses + 3] = {};
    GT_HIP(hipMemcpyAsync(info, r.class_info, sizeof(info), hipMemcpyDeviceToHost, stream));
    GT_HIP(hipStreamSynchronize(stream));
    if ((st = validation_result(uint32_t(uint64_t(info[2 * kClasses + 1])))) != GT_OK) return st;
    const int64_t* cnt = info + kClasses;
    const int32_t* list_of[kClasses];
    const int64_t* len_of[kClasses];
    for (int c = 0; c < kClasses; ++c) {
        list_of[c] = r.list + info[c];
        len_of[c] = r.class_info + kClasses + c;
    }
    const int64_t n_huge = cnt[kClsHuge];
    BigRows br{list_of[kClsHuge], info[kClsHuge], len_of[kClsHuge], r.huge_off, r.huge_echunk, r.huge_schunk,
               r.tab, r.big_best, r.big_own, r.big_hbest, r.big_lbest};
    if (n_huge > 0) {  // the chunk numbering of the long rows' edges and table slots, and their table offsets
        k_big_prep<<<1, kPrepThreads, 0, stream>>>(list_of[kClsHuge], len_of[kClsHuge], rowptr, r.huge_echunk,
                                                    r.huge_schunk, r.huge_off);
        GT_LAUNCH_CHECK("reorder_big_prep");
    }
    // the short-row lists in one launch, blocks in proportion to their rows
    SmallRows sr;
    {
        const int cls[kSmLists] = {kClsWav, kClsS32, kClsS16, kClsS8, kClsS4};
        const int per_wave[kSmLists] = {1, kWave / kSub32, kWave / kSub16, kWave / kSub8, kWave / kSub4};
        sr.list = r.list;
        unsigned at = 0;
        int64_t slot = 0;
        for (int k = 0; k < kSmLists; ++k) {
            const int64_t rows = cnt[cls[k]];
            sr.base[k] = info[cls[k]];
            sr.len[k] = rows;
            sr.slot[k] = slot;
            slot += rows * (kWave / per_wave[k]);  // the list's rows, padded to its largest
            sr.first[k] = at;
            if (rows > 0) at += grid_cap(rows, int64_t(per_wave[k]) * (kBlock / kWave), 16384);
        }
        sr.first[kSmLists] = at;
        // within the workspace's 2 nnz + 4 n slots: every list but the 0-4 one holds rows of more than half its width
        if (slot > 2 * nnz + 4 * n)
            return fail(GT_ERR_WORKSPACE, "gt_reorder: short-row slots exceed the workspace");
    }
    // rows whose count table is over kFusedCap slots (more than kFusedCap / 2 entries) take the chunked passes
    const bool giant = info[2 * kClasses] + 1 > kFusedCap / 2;
    const unsigned gwt = grid_cap(cnt[kClsWmed], kBlock / kWave, 1024);
    const unsigned gmed = grid_cap(cnt[kClsMed], 1, 1024);
    // side streams pay where the rows of more than kWaveRowMax entries hold at least a quarter of the
    // entries; with fewer, their launches would mostly wait behind the short rows, so all stays on `stream`
    const bool side = sp.n_side > 0 && 4 * info[2 * kClasses + 2] >= nnz;
    const hipStream_t s_short = stream, s_big = side ? sp.at(1) : stream, s_wide = side ? sp.at(2) : stream;
    for (int t = 0; t < iters; ++t) {
        const uint64_t key = seed + uint64_t(t + 1) * kGolden;
        const int32_t* in = r.lab[t & 1];
        int32_t* out = r.lab[(t + 1) & 1];
        if (side && (st = sp.fork()) != GT_OK) return st;
        if (t == 0) {  // labels are the node ids: a minimum over each row's columns
            if (n_huge > 0) {
                k_big_first_reset<<<grid_for(n_huge, 256, 1024), 256, 0, s_big>>>(br);
                k_big_first<0><<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, col, r.roff, r.lpos, r.ncol, key);
                k_big_first<1><<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, col, r.roff, r.lpos, r.ncol, key);
                GT_LAUNCH_CHECK("reorder_big_first");
                k_big_decide<<<grid_for(n_huge, 256, 1024), 256, 0, s_big>>>(br, rowptr, in, out, key, r.flags,
                                                                             r.flags + 1, false);
                GT_LAUNCH_CHECK("reorder_big_decide");
            }
            if (sr.first[kSmLists] > 0) {
                k_first_small<<<sr.first[kSmLists], kBlock, 0, s_short>>>(sr, rowptr, col, r.lpos, r.slots, out,
                                                                         key, r.flags + 1);
                GT_LAUNCH_CHECK("reorder_first_small");
            }
            if (cnt[kClsWmed] > 0) {
                k_first_wide<kWave><<<gwt, kBlock, 0, s_wide>>>(r.list, info[kClsWmed], len_of[kClsWmed], rowptr,
                                                               col, r.roff, r.lpos, r.ncol, out, key, r.flags + 1);
                GT_LAUNCH_CHECK("reorder_first_wave");
            }
            if (cnt[kClsMed] > 0) {
                k_first_wide<kMedBlock><<<gmed, kMedBlock, 0, s_wide>>>(r.list, info[kClsMed], len_of[kClsMed],
                                                                        rowptr, col, r.roff, r.lpos, r.ncol, out,
                                                                        key, r.flags + 1);
                GT_LAUNCH_CHECK("reorder_first_block");
            }
            if ((st = sp.join()) != GT_OK) return st;
            continue;
        }
        if (n_huge > 0) {
            const uint32_t* fp = r.flags + t;
            // the tables' first use clears them all; later, k_big_fused clears its own
            if (t == 1 || giant) {
                k_big_clear<<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, fp, t == 1);
                GT_LAUNCH_CHECK("reorder_big_clear");
            }
            k_big_insert<<<kBigGrid, kBlock, 0, s_big>>>(br, r.roff, r.ncol, in, fp);
            GT_LAUNCH_CHECK("reorder_big_insert");
            k_big_fused<<<unsigned(n_huge < 2048 ? n_huge : 2048), kFusedThreads, 0, s_big>>>(br, rowptr, in, out,
                                                                                            key, fp,
                                                                                            r.flags + t + 1);
            GT_LAUNCH_CHECK("reorder_big_fused");
            if (giant) {
                k_big_reduce<0><<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, in, key, fp);
                k_big_reduce<1><<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, in, key, fp);
                k_big_reduce<2><<<kBigGrid, kBlock, 0, s_big>>>(br, rowptr, in, key, fp);
                GT_LAUNCH_CHECK("reorder_big_reduce");
                k_big_decide<<<grid_for(n_huge, 256, 1024), 256, 0, s_big>>>(br, rowptr, in, out, key, fp,
                                                                             r.flags + t + 1, true);
                GT_LAUNCH_CHECK("reorder_big_decide");
            }
        }
        if (sr.first[kSmLists] > 0) {
            k_lp_small<<<sr.first[kSmLists], kBlock, 0, s_short>>>(sr, r.slots, in, out, key, r.flags + t,
                                                                   r.flags + t + 1);
            GT_LAUNCH_CHECK("reorder_lp_small");
        }
        if (cnt[kClsWmed] > 0) {
            k_lp_wavetab<<<gwt, kBlock, 0, s_wide>>>(r.list, info[kClsWmed], len_of[kClsWmed], r.roff, r.ncol, in,
                                                     out, key, r.flags + t, r.flags + t + 1);
            GT_LAUNCH_CHECK("reorder_lp_wavetab");
        }
        if (cnt[kClsMed] > 0) {
            k_lp_block<kMedBlock><<<gmed, kMedBlock, 0, s_short>>>(r.list, info[kClsMed], len_of[kClsMed], r.roff,
                                                                  r.ncol, in, out, key, r.flags + t,
                                                                  r.flags + t + 1);
            GT_LAUNCH_CHECK("reorder_lp_lds");
        }
        if ((st = sp.join()) != GT_OK) return st;
    }
    int32_t* final_lab = r.lab[(iters + 1) & 1];
    k_labels_by_node<<<g, 256, 0, stream>>>(n, r.list, r.lab[iters & 1], final_lab);
    GT_LAUNCH_CHECK("reorder_labels_by_node");
    const uint32_t dmax = uint32_t(info[2 * kClasses]);
    const int dbits = bits_for(int64_t(dmax) + 1);
    k_order_keys<<<g, 256, 0, stream>>>(n, final_lab, r.deg_off, dmax, dbits, r.sort_keys);
    GT_LAUNCH_CHECK("reorder_keys");
    if ((st = iota_u32(r.sort_vals, n, stream)) != GT_OK) return st;
    if ((st = radix_sort_u64(r.sort_keys, r.sort_vals, n, bits_for(n) + dbits, r.sort, stream)) != GT_OK) return st;
    k_finish_order<<<g, 256, 0, stream>>>(n, r.sort_vals, final_lab, perm, iperm, labels);
    GT_LAUNCH_CHECK("reorder_finish");
    if (sweeps_done) {
        uint32_t* host = new uint32_t[size_t(iters) + 1];
        hipError_t e = hipMemcpyAsync(host, r.flags + 1, size_t(iters) * 4 + 4, hipMemcpyDeviceToHost, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        int done = 0;
        for (int t = 0; t < iters; ++t)
            if (host[t]) done = t + 1;
        delete[] host;
        if (e != hipSuccess) return hip_fail(e, "gt_reorder: read sweep flags");
        *sweeps_done = done;
    }
    return GT_OK;
}

extern "C" gt_status gt_reorder(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t iters,
                                uint64_t seed, int32_t* perm, int32_t* iperm, int32_t* labels,
                                int32_t* sweeps_done, void* ws_ptr, size_t ws_bytes, hipStream_t stream) {
    return gt_reorder_streams(n, nnz, rowptr, col, iters, seed, perm, iperm, labels, sweeps_done, ws_ptr, ws_bytes,
                              stream, nullptr, nullptr, 0);
}
