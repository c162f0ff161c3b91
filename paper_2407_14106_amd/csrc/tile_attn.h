// Dense-tile attention (§3.4: tiles of the reordered adjacency dense enough to
// be computed whole on the matrix cores) and the partial results it hands to
// the edge kernels, which finish every row and column.
#pragma once

#include "attn_common.h"

namespace gt {

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

inline int tile_shift(int T) { return T == 128 ? 7 : 6; }

// Carve the partial buffers out of the workspace (nothing when no tile is dense).
inline TilePartials tile_partials_fwd(Ws& ws, const gt_tiles* p, int H, int D) {
    TilePartials t;
    if (p->n_dense <= 0 || p->n <= 0) return t;
    t.ptr = p->tile_rowptr;
    t.tshift = tile_shift(p->T);
    t.m = ws.take<float>(size_t(p->n) * H);
    t.l = ws.take<float>(size_t(p->n) * H);
    t.acc = ws.take<float>(size_t(p->n) * H * D);
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
    }
    if (cols) {
        b.dk.ptr = b.dv.ptr = p->tileT_ptr;
        b.dk.tshift = b.dv.tshift = tile_shift(p->T);
        b.dk.acc = ws.take<float>(size_t(p->n) * H * D);
        b.dv.acc = ws.take<float>(size_t(p->n) * H * D);
    }
    return b;
}

// Forward over the dense tiles: for every node of a tile row with dense
// tiles, writes (m, l, acc) of the online softmax over its dense-tile edges.
template <typename T, int D, int H>
gt_status tile_fwd(const gt_tiles* p, const T* Q, const T* K, const T* V, float sl2, TilePartials tp,
                   hipStream_t s);

// Backward over the dense tiles, row-owned: for every node of a tile row with
// dense tiles, the sums over its dense-tile edges of P dP K (acc), P K (acc2)
// and P dP (m); the edge kernels add the remainder and form
// dQ = scale (A - D B) with D the total P dP sum.
template <typename T, int D, int H>
gt_status tile_bwd_dq(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                      float sl2, TilePartials dq, hipStream_t s);

// Backward over the dense tiles, column-owned: dk (unscaled) and dv sums over
// the dense-tile edges of every node of a tile column with dense tiles.
template <typename T, int D, int H>
gt_status tile_bwd_dkdv(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                        const float* Dv, float sl2, TilePartials dk, TilePartials dv, hipStream_t s);

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
                         float sl2, TilePartials tp, hipStream_t s);
template <int D>
gt_status tiles_dq_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* dO, const float* LSE, float sl2, TilePartials dq, hipStream_t s);
template <int D>
gt_status tiles_dkdv_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                          const uint16_t* dO, const float* LSE, const float* Dv, float sl2, TilePartials dk,
                          TilePartials dv, hipStream_t s);

}  // namespace gt
