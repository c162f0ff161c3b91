// Dense-tile attention (§3.4: tiles of the reordered adjacency dense enough to
// be computed whole on the matrix cores) and the partial results it hands to
// the edge kernels, which finish every row and column.
#pragma once

#include "attn_common.h"

namespace gt {

// The dense tiles of a tile row (tile column) are dealt out in chunks of CH
// tiles, one workgroup each, so a row of many dense tiles (the hubs of a
// power-law graph) is spread over the chip.  The first chunk of a row writes
// the row's partial state; the others write extra slots, which a merge then
// folds in (in slot order, so the result is deterministic).
struct TileChunks {
    int64_t* chunk_off = nullptr;  // [R + 1]: first chunk of each tile row (column)
    int64_t* extra_off = nullptr;  // [R + 1]: first extra slot of each tile row (column)
    int32_t* merge_rows = nullptr;  // tile rows (columns) with extra slots, the first *merge_cnt entries
    uint32_t* merge_cnt = nullptr;
    int CH = 1;
    int64_t max_chunks = 0;
    int64_t max_merge = 0;  // bound on the rows with extra slots
    float* m = nullptr;     // extra slots: [slots, T, H] (forward max, or the dQ pass's D sum)
    float* l = nullptr;     // [slots, T, H] forward only
    float* acc = nullptr;   // [slots, T, H, d]
    float* acc2 = nullptr;  // [slots, T, H, d] dQ pass only
};

constexpr int kTileChunkMin = 4;        // tiles per chunk, at least
constexpr int64_t kTileChunks = 512;    // the chunk size grows so that extra slots stay below this

// Per-(node, head) partial state left by the dense tiles of a tile row (or
// tile column).  `ptr` is tile_rowptr (or tileT_ptr): a node has a partial iff
// its tile row (column) holds at least one dense tile.
struct TilePartials {
    const int64_t* ptr = nullptr;
    int tshift = 0;
    float* m = nullptr;     // [n, H] forward: running max (log2 domain); dQ: partial D sum
    float* l = nullptr;     // [n, H] forward: running sum
    float* acc = nullptr;   // [n, H, d] unnormalised output / gradient sums (dQ: A)
    float* acc2 = nullptr;  // [n, H, d] dQ only: B
    TileChunks ck;
    __device__ __forceinline__ bool has(int64_t node) const {
        if (!ptr) return false;
        const int64_t I = node >> tshift;
        return ptr[I + 1] > ptr[I];
    }
    __device__ __forceinline__ bool has_row(int64_t node) const { return has(node); }
    __device__ __forceinline__ bool has_col(int64_t node) const { return has(node); }
};

struct TileBwdPartials {
    TilePartials dq, dk, dv;
};

// A per-edge bias on the dense tiles (the graph encoding of §2.1 Eq. (3)),
// laid out per tile in the workspace: b[((k H + h) T + r) T + c] for local row
// r and column c of dense tile k, -inf off the tile's edges (adding it masks
// the cell).  The column pass writes dS into db at the same places (every
// cell).  Null b: no bias.
struct TileBias {
    const float* b = nullptr;
    float* db = nullptr;
    __device__ __forceinline__ static int64_t at(int64_t k, int H, int h, int T, int r, int c) {
        return ((k * H + h) * int64_t(T) + r) * T + c;
    }
};

inline int tile_shift(int T) { return T == 128 ? 7 : 6; }

// Carve the chunk plan and its extra slots (floats per slot row: per_row) out of the workspace.
inline TileChunks tile_chunks(Ws& ws, const gt_tiles* p, int64_t per_row_m, int64_t per_row_acc, bool with_l,
                              bool with_acc2) {
    TileChunks c;
    const int64_t R = p->n_row_tiles > 0 ? p->n_row_tiles : 1;
    const int64_t nd = p->n_dense;
    c.CH = int(cdiv(nd, kTileChunks) > kTileChunkMin ? cdiv(nd, kTileChunks) : kTileChunkMin);
    const int64_t slots = nd / c.CH + 1;
    c.max_chunks = (R < nd ? R : nd) + nd / c.CH + 1;
    c.chunk_off = ws.take<int64_t>(R + 1);
    c.extra_off = ws.take<int64_t>(R + 1);
    c.max_merge = R < slots ? R : slots;
    c.merge_rows = ws.take<int32_t>(size_t(c.max_merge));
    c.merge_cnt = ws.take<uint32_t>(1);
    const int64_t rows = slots * p->T;
    c.m = ws.take<float>(size_t(rows * per_row_m));
    if (with_l) c.l = ws.take<float>(size_t(rows * per_row_m));
    c.acc = ws.take<float>(size_t(rows * per_row_acc));
    if (with_acc2) c.acc2 = ws.take<float>(size_t(rows * per_row_acc));
    return c;
}

// Carve the partial buffers out of the workspace (nothing when no tile is dense).
inline TilePartials tile_partials_fwd(Ws& ws, const gt_tiles* p, int H, int D) {
    TilePartials t;
    if (p->n_dense <= 0 || p->n <= 0) return t;
    t.ptr = p->tile_rowptr;
    t.tshift = tile_shift(p->T);
    t.m = ws.take<float>(size_t(p->n) * H);
    t.l = ws.take<float>(size_t(p->n) * H);
    t.acc = ws.take<float>(size_t(p->n) * H * D);
    t.ck = tile_chunks(ws, p, H, int64_t(H) * D, true, false);
    return t;
}

inline TileBwdPartials tile_partials_bwd(Ws& ws, const gt_tiles* p, int H, int D, bool rows, bool cols) {
    TileBwdPartials b;
    if (p->n_dense <= 0 || p->n <= 0) return b;
    if (rows) {
        b.dq.ptr = p->tile_rowptr;
        b.dq.tshift = tile_shift(p->T);
        b.dq.acc = ws.take<float>(size_t(p->n) * H * D);
        b.dq.acc2 = ws.take<float>(size_t(p->n) * H * D);
        b.dq.m = ws.take<float>(size_t(p->n) * H);
        b.dq.ck = tile_chunks(ws, p, H, int64_t(H) * D, false, true);
    }
    if (cols) {
        b.dk.ptr = b.dv.ptr = p->tileT_ptr;
        b.dk.tshift = b.dv.tshift = tile_shift(p->T);
        b.dk.acc = ws.take<float>(size_t(p->n) * H * D);
        b.dv.acc = ws.take<float>(size_t(p->n) * H * D);
        b.dk.ck = tile_chunks(ws, p, 0, int64_t(H) * D, false, true);  // acc: dk slots, acc2: dv slots
    }
    return b;
}

// Forward over the dense tiles: for every node of a tile row with dense
// tiles, writes (m, l, acc) of the online softmax over its dense-tile edges.
template <typename T, int D, int H>
gt_status tile_fwd(const gt_tiles* p, const T* Q, const T* K, const T* V, float sl2, TilePartials tp,
                   TileBias tb, hipStream_t s);

// Backward over the dense tiles, row-owned: for every node of a tile row with
// dense tiles, the sums over its dense-tile edges of P dP K (acc), P K (acc2)
// and P dP (m); the edge kernels add the remainder and form
// dQ = scale (A - D B) with D the total P dP sum.
template <typename T, int D, int H>
gt_status tile_bwd_dq(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                      float sl2, TilePartials dq, TileBias tb, hipStream_t s);

// Backward over the dense tiles, column-owned: dk (unscaled) and dv sums over
// the dense-tile edges of every node of a tile column with dense tiles; with a
// bias, dS of every tile edge into tb.db.
template <typename T, int D, int H>
gt_status tile_bwd_dkdv(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                        const float* Dv, float sl2, TilePartials dk, TilePartials dv, TileBias tb, hipStream_t s);

// The full softmax layer (every node attends to all n nodes) on the same
// kernels: O and LSE; then D = <dO, O> (into Dv) and dQ; then dK and dV.
template <typename T, int D, int H>
gt_status full_fwd(int64_t n, const T* Q, const T* K, const T* V, float sl2, T* O, float* LSE, hipStream_t s);
template <typename T, int D, int H>
gt_status full_bwd(int64_t n, const T* Q, const T* K, const T* V, const T* O, const T* dO, const float* LSE,
                   float sl2, float scale, T* dQ, T* dK, T* dV, float* Dv, hipStream_t s);

// The full layer for bf16 features (dense_mfma.hip): the streaming kernels
// with two 32-row blocks per wavefront; same results contract as full_fwd /
// full_bwd.  H is a runtime value.
template <int D>
gt_status full_fwd_bf16(int64_t n, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V, float sl2,
                        uint16_t* O, float* LSE, hipStream_t s);
template <int D>
gt_status full_bwd_bf16(int64_t n, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* O, const uint16_t* dO, const float* LSE, float sl2, float scale,
                        uint16_t* dQ, uint16_t* dK, uint16_t* dV, float* Dv, hipStream_t s);

// The dense tiles of a plan for bf16 features (dense_mfma.hip): same partial
// sums as tile_fwd / tile_bwd_dq / tile_bwd_dkdv, which call them for bf16.
template <int D>
gt_status tiles_fwd_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         float sl2, TilePartials tp, TileBias tb, hipStream_t s);
template <int D>
gt_status tiles_dq_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* dO, const float* LSE, float sl2, TilePartials dq, TileBias tb,
                        hipStream_t s);
template <int D>
gt_status tiles_dkdv_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                          const uint16_t* dO, const float* LSE, const float* Dv, float sl2, TilePartials dk,
                          TilePartials dv, TileBias tb, hipStream_t s);

}  // namespace gt
