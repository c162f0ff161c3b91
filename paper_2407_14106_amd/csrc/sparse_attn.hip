// Neighbourhood softmax attention (§3.2, local topology-induced pattern) on the
// remainder edges of a tile plan, forward and backward, plus the two entry
// points that also run the dense-tile kernels (tile_attn.hip).
//
// Edge kernels ("rows" and "cols"): a wavefront serves 64 / (H * d/F) nodes at
// once, each (node, head) owned by d/F lanes that hold F consecutive features
// (64 bytes) of it.  The node's own vectors stay in registers while the lanes
// walk its edge list two edges at a time, gathering the neighbours' 64-byte
// slices; every gathered row is read as whole 64-byte pieces by neighbouring
// lanes.  Scores use the paper's scaled dot product in the exp2 domain; the
// forward keeps an online max / sum per (node, head), so nothing per edge is
// ever written to memory.
//
// Nodes with more than GT_LONG_ROW remainder edges are left to the "long"
// kernels: one workgroup per node, its edges dealt round-robin over the
// workgroup's lane groups and the partial results merged in LDS.
//
// The backward never uses atomics: dQ is gathered per row over the CSR, dK and
// dV per column over the remainder's transpose.
#include "attn_common.h"
#include "prim.h"
#include "tile_attn.h"

namespace gt {
namespace {

constexpr int kThreads = 256;
constexpr float kNegInf = -__builtin_huge_valf();

template <typename T, int D, int H>
struct Lanes {
    using C = EdgeCfg<T, D, H>;
    int slot, h, part;
    __device__ __forceinline__ explicit Lanes(int t) {
        slot = t / C::G;
        h = (t / C::L) % H;
        part = t % C::L;
    }
    __device__ __forceinline__ int64_t off(int64_t node) const { return (node * H + h) * D + part * C::F; }
};

// Per-edge additive bias (the graph encoding added to the scaled product,
// §2.1 Eq. (3); it shares the attention's sparse layout, §3.3): fp32
// [nnz, H] indexed by the edge's position in the input CSR of the plan.  A
// remainder edge's input position is sp_pos[remainder position] (the same
// position when the plan has no dense tile and no sp_pos).  The column pass
// finds an in-edge's input position through csc_pos and writes dB = dS there.
// The dense tiles take the bias laid out per tile (tile).
struct EdgeBias {
    const float* b = nullptr;  // null: no bias on the remainder edges
    const int32_t* sp_pos = nullptr;
    const int32_t* csc_pos = nullptr;
    float* db = nullptr;
    TileBias tile;
    // bias of remainder position pos, head h, in the exp2 domain
    __device__ __forceinline__ float at(int64_t pos, int H, int h) const {
        return b[(sp_pos ? int64_t(sp_pos[pos]) : pos) * H + h] * kLog2e;
    }
    // bias of input-CSR position e, head h, in the exp2 domain
    __device__ __forceinline__ float at_input(int64_t e, int H, int h) const { return b[e * H + h] * kLog2e; }
};

// F fp32 accumulators of one (node, head) slice.
template <int F>
struct Acc {
    float v[F];
    __device__ __forceinline__ Acc() {
#pragma unroll
        for (int i = 0; i < F; ++i) v[i] = 0.f;
    }
};

// Online-softmax state of one (node, head) slice.
template <int F>
struct Online {
    float m = kNegInf;  // running max, log2 domain
    float l = 0.f;      // running sum of exp2(s - m)
    float acc[F];       // running sum of exp2(s - m) * v
    __device__ __forceinline__ Online() {
#pragma unroll
        for (int i = 0; i < F; ++i) acc[i] = 0.f;
    }
};

template <typename T, int D, int H>
__device__ __forceinline__ void load_fwd_partial(Online<EdgeCfg<T, D, H>::F>& st, const TilePartials& tp, int64_t node,
                                                 int h, int64_t off) {
    constexpr int F = EdgeCfg<T, D, H>::F;
    st.m = tp.m[node * H + h];
    st.l = tp.l[node * H + h];
    const float4* a = reinterpret_cast<const float4*>(tp.acc + off);
#pragma unroll
    for (int i = 0; i < F / 4; ++i) {
        float4 v = a[i];
        st.acc[4 * i] = v.x;
        st.acc[4 * i + 1] = v.y;
        st.acc[4 * i + 2] = v.z;
        st.acc[4 * i + 3] = v.w;
    }
}

// The running max is a lazy reference: it moves only when a score exceeds it
// by more than 2^8 (in the exp2 domain), so the accumulator is rescaled
// rarely; weights stay below 2^8 and the result is unchanged.
constexpr float kRescale = 8.f;

// Weight p as the bf16 pairs (p, 0) and (0, p) for Slice::axpy_w.
__device__ __forceinline__ void weight_pairs(float p, uint32_t& lo, uint32_t& hi) {
    lo = uint32_t(f32_to_bf16(p));
    hi = lo << 16;
}

// One block of two edges for the forward state.  j0/j1 are always valid
// node ids (callers substitute a valid id for missing edges); ok0/ok1 say
// which of the two are edges.
template <typename T, int D, int H, bool kBias = false>
__device__ __forceinline__ void fwd_step(Online<EdgeCfg<T, D, H>::F>& st, const Slice<T, EdgeCfg<T, D, H>::F>& q,
                                         const T* __restrict__ K, const T* __restrict__ V, int64_t j0, int64_t j1,
                                         bool ok0, bool ok1, const Lanes<T, D, H>& ln, float sl2, float b0 = 0.f,
                                         float b1 = 0.f) {
    using C = EdgeCfg<T, D, H>;
    Slice<T, C::F> k0, k1, v0, v1;
    k0.load(K + ln.off(j0));
    k1.load(K + ln.off(j1));
    v0.load(V + ln.off(j0));
    v1.load(V + ln.off(j1));
    float s0 = ok0 ? group_sum<C::L>(q.dot(k0)) * sl2 : kNegInf;
    float s1 = ok1 ? group_sum<C::L>(q.dot(k1)) * sl2 : kNegInf;
    if constexpr (kBias) {
        s0 += b0;
        s1 += b1;
    }
    const float mb = fmaxf(s0, s1);
    if (mb > st.m + kRescale) {
        const float alpha = st.m == kNegInf ? 0.f : exp2f(st.m - mb);
        st.l *= alpha;
#pragma unroll
        for (int i = 0; i < C::F; ++i) st.acc[i] *= alpha;
        st.m = mb;
    }
    const float p0 = ok0 ? exp2f(s0 - st.m) : 0.f;
    const float p1 = ok1 ? exp2f(s1 - st.m) : 0.f;
    st.l += p0 + p1;
    if constexpr (sizeof(T) == 2) {
        uint32_t a0, b0, a1, b1;
        weight_pairs(p0, a0, b0);
        weight_pairs(p1, a1, b1);
        v0.axpy_w(st.acc, a0, b0);
        v1.axpy_w(st.acc, a1, b1);
    } else {
#pragma unroll
        for (int i = 0; i < C::F; ++i) st.acc[i] = fmaf(p1, v1.f(i), fmaf(p0, v0.f(i), st.acc[i]));
    }
}

// Neighbour ids of edges t .. t+3 of a row whose list is cl[a, a + deg) in an
// array of `len` entries: one 16-byte load where the array allows it (ids past
// the row are read but replaced).  Missing edges get a valid id: the row's
// edge t if it exists, else `self`.
__device__ __forceinline__ int4 edge_quad(const int32_t* __restrict__ cl, int64_t len, int64_t a, int deg, int t,
                                          int32_t self) {
    if (deg <= t) return make_int4(self, self, self, self);
    int4 v;
    if (a + t + 4 <= len) {
        v = *reinterpret_cast<const int4*>(cl + a + t);
    } else {
        const int last = deg - 1;
        v.x = cl[a + t];
        v.y = cl[a + (t + 1 < last ? t + 1 : last)];
        v.z = cl[a + (t + 2 < last ? t + 2 : last)];
        v.w = cl[a + (t + 3 < last ? t + 3 : last)];
    }
    if (t + 1 >= deg) v.y = v.x;
    if (t + 2 >= deg) v.z = v.x;
    if (t + 3 >= deg) v.w = v.x;
    return v;
}

// Walk a row's edges four at a time up to the wavefront maximum dmax, the ids
// of the next four fetched before the current four are used; step(j0, j1, t,
// ok0, ok1) takes two edges, the row's edges t and t + 1.
template <class Step>
__device__ __forceinline__ void walk_edges(const int32_t* __restrict__ cl, int64_t len, int64_t a, int deg, int dmax,
                                           int32_t self, Step step) {
    int4 cur = edge_quad(cl, len, a, deg, 0, self), nxt = cur;
    for (int t = 0; t < dmax; t += 4) {
        if (t + 4 < dmax) nxt = edge_quad(cl, len, a, deg, t + 4, self);
        step(cur.x, cur.y, t, t < deg, t + 1 < deg);
        if (t + 2 < dmax) step(cur.z, cur.w, t + 2, t + 2 < deg, t + 3 < deg);
        cur = nxt;
    }
}

// The value of lane 0 of each L-lane group, in every lane of the group.
template <int L>
__device__ __forceinline__ float group_bcast0(float x) {
    if constexpr (L == 2) return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xA0, 0xF, 0xF, false));
    if constexpr (L == 4) return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x00, 0xF, 0xF, false));
    return x;
}

// The value of the first lane of each G-lane group (one node's lanes), in
// every lane of the group.
template <int G>
__device__ __forceinline__ int group_first(int x) {
    if constexpr (G == 1) return x;
    else if constexpr (G == 2) return __builtin_amdgcn_mov_dpp(x, 0xA0, 0xF, 0xF, false);  // quad_perm 0,0,2,2
    else if constexpr (G == 4) return __builtin_amdgcn_mov_dpp(x, 0x00, 0xF, 0xF, false);  // quad_perm 0,0,0,0
    else if constexpr (G == 16) return __builtin_amdgcn_mov_dpp(x, 0x150, 0xF, 0xF, false);  // row_newbcast:0
    else if constexpr (G == 64) return __builtin_amdgcn_readfirstlane(x);
    else return __shfl(x, lane_id() & ~(G - 1), kWave);
}

// Bias (exp2 domain) of a row's edges t and t + 1 at CSR offset a; 0 where
// the edge is missing.  One lane of each (node, head) group reads it.
template <typename LN>
__device__ __forceinline__ void bias_pair(const EdgeBias& eb, int64_t a, int t, bool ok0, bool ok1, int H,
                                          const LN& ln, float& b0, float& b1) {
    float x0 = 0.f, x1 = 0.f;
    if (ln.part == 0) {
        x0 = ok0 ? eb.at(a + t, H, ln.h) : 0.f;
        x1 = ok1 ? eb.at(a + t + 1, H, ln.h) : 0.f;
    }
    b0 = group_bcast0<LN::C::L>(x0);
    b1 = group_bcast0<LN::C::L>(x1);
}

// The bias of four edges of each of a wavefront's nodes moves through LDS, so
// that a lane reads one vector (the floats 4H/G g .. of the quad's block, all
// within one edge) instead of one float per edge: kPer floats per lane, each
// group's block of 4H floats at `s`.  The wavefront alone uses its block, and
// its LDS operations take effect in program order, so no barrier is needed.
template <typename T, int D, int H>
struct BiasStage {
    using C = EdgeCfg<T, D, H>;
    static constexpr int kPer = 4 * H / C::G;
    static constexpr bool kOn = kPer >= 1 && kPer <= H;
    static constexpr int kWaveFloats = C::NPW * 4 * H;
};

// Input-CSR positions of a row's (column's) edges t .. t + 3: base + off[u].
struct Quad {
    int64_t base;
    int4 off;
    __device__ __forceinline__ int64_t at(int u) const {
        return base + (u == 0 ? off.x : u == 1 ? off.y : u == 2 ? off.z : off.w);
    }
};

template <int P>
__device__ __forceinline__ void ld_floats(float (&v)[P], const float* __restrict__ src) {
    if constexpr (P == 4) {
        const float4 x = *reinterpret_cast<const float4*>(src);
        v[0] = x.x, v[1] = x.y, v[2] = x.z, v[3] = x.w;
    } else if constexpr (P == 2) {
        const float2 x = *reinterpret_cast<const float2*>(src);
        v[0] = x.x, v[1] = x.y;
    } else {
        v[0] = *src;
    }
}
template <int P>
__device__ __forceinline__ void st_floats(float* __restrict__ dst, const float (&v)[P]) {
    if constexpr (P == 4) *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
    else if constexpr (P == 2) *reinterpret_cast<float2*>(dst) = make_float2(v[0], v[1]);
    else *dst = v[0];
}

__device__ __forceinline__ void lds_order() {
    __builtin_amdgcn_wave_barrier();
    asm volatile("" ::: "memory");
}

// This lane's share of the quad's bias block (kPer floats of one edge); 0 past deg.
template <typename T, int D, int H, int P>
__device__ __forceinline__ void bias_share(float (&v)[P], const float* __restrict__ b, const Quad& q, int t, int deg,
                                           const Lanes<T, D, H>& ln) {
    const int e0 = (ln.h * EdgeCfg<T, D, H>::L + ln.part) * P, u = e0 / H;
#pragma unroll
    for (int k = 0; k < P; ++k) v[k] = 0.f;
    if (t + u < deg) ld_floats<P>(v, b + q.at(u) * H + e0 % H);
}

// The shares of a group through LDS: the bias (exp2 domain) of the quad's four
// edges for this lane's head.
template <typename T, int D, int H, int P>
__device__ __forceinline__ float4 bias_swap(const float (&v)[P], const Lanes<T, D, H>& ln, float* s) {
    const int e0 = (ln.h * EdgeCfg<T, D, H>::L + ln.part) * P;
    lds_order();
#pragma unroll
    for (int k = 0; k < P; ++k) s[e0 + k] = v[k];
    lds_order();
    float4 x = make_float4(s[ln.h], s[H + ln.h], s[2 * H + ln.h], s[3 * H + ln.h]);
    lds_order();
    x.x *= kLog2e, x.y *= kLog2e, x.z *= kLog2e, x.w *= kLog2e;
    return x;
}

// Write ds (this lane's head, edges t .. t + 3) to db at the quad's positions.
template <typename T, int D, int H>
__device__ __forceinline__ void db_quad(float* __restrict__ db, const Quad& q, int t, int deg, float4 ds,
                                        const Lanes<T, D, H>& ln, float* s) {
    constexpr int P = BiasStage<T, D, H>::kPer;
    lds_order();
    if (ln.part == 0) {
        s[ln.h] = ds.x;
        s[H + ln.h] = ds.y;
        s[2 * H + ln.h] = ds.z;
        s[3 * H + ln.h] = ds.w;
    }
    lds_order();
    const int e0 = (ln.h * EdgeCfg<T, D, H>::L + ln.part) * P, u = e0 / H;
    float v[P];
#pragma unroll
    for (int k = 0; k < P; ++k) v[k] = s[e0 + k];
    lds_order();
    if (t + u < deg) st_floats<P>(db + q.at(u) * H + e0 % H, v);
}

// Positions of a row's remainder edges t .. t + 3 (through sp_pos when the
// plan has one) or of a column's in-edges (through csc_pos); past deg they
// repeat a valid position.
__device__ __forceinline__ Quad row_quad(const EdgeBias& eb, int64_t len, int64_t a, int deg, int t) {
    Quad q;
    if (eb.sp_pos) {
        q.base = 0;
        q.off = edge_quad(eb.sp_pos, len, a, deg, t, 0);
    } else {
        q.base = a;
        q.off = make_int4(t, t + 1 < deg ? t + 1 : t, t + 2 < deg ? t + 2 : t, t + 3 < deg ? t + 3 : t);
    }
    return q;
}
__device__ __forceinline__ Quad col_quad(const EdgeBias& eb, int64_t len, int64_t a, int deg, int t) {
    Quad q;
    q.base = 0;
    q.off = edge_quad(eb.csc_pos, len, a, deg, t, 0);
    return q;
}

// walk_edges for a bias kernel, the bias exchanged in LDS when a quad starts;
// step(j0, j1, t, ok0, ok1, b0, b1) takes two edges, after(t, q) runs once the
// quad's steps are done (the column pass writes dB there).  kAhead: positions
// two quads ahead and bias shares one quad ahead, their loads in flight across
// a quad's steps (the forward and the column pass; the row pass, with more
// live registers, reads each quad's when it starts).
template <typename T, int D, int H, bool kAhead, class QuadOf, class Step, class After>
__device__ __forceinline__ void walk_edges_bias(const int32_t* __restrict__ cl, int64_t len, int64_t a, int deg,
                                                int dmax, int32_t self, const float* __restrict__ b,
                                                const Lanes<T, D, H>& ln, float* s, QuadOf quad_of, Step step,
                                                After after) {
    constexpr int P = BiasStage<T, D, H>::kPer;
    int4 cur = edge_quad(cl, len, a, deg, 0, self), nxt = cur;
    if constexpr (kAhead) {
        Quad q0 = quad_of(0);
        Quad q1 = 4 < dmax ? quad_of(4) : q0;
        float v[P];
        bias_share<T, D, H, P>(v, b, q0, 0, deg, ln);
        for (int t = 0; t < dmax; t += 4) {
            float vn[P];
#pragma unroll
            for (int k = 0; k < P; ++k) vn[k] = 0.f;
            Quad q2 = q1;
            if (t + 4 < dmax) {
                nxt = edge_quad(cl, len, a, deg, t + 4, self);
                bias_share<T, D, H, P>(vn, b, q1, t + 4, deg, ln);
            }
            if (t + 8 < dmax) q2 = quad_of(t + 8);
            const float4 x = bias_swap<T, D, H, P>(v, ln, s);
            step(cur.x, cur.y, t, t < deg, t + 1 < deg, x.x, x.y);
            if (t + 2 < dmax) step(cur.z, cur.w, t + 2, t + 2 < deg, t + 3 < deg, x.z, x.w);
            after(t, q0);
            cur = nxt;
            q0 = q1;
            q1 = q2;
#pragma unroll
            for (int k = 0; k < P; ++k) v[k] = vn[k];
        }
    } else {
        for (int t = 0; t < dmax; t += 4) {
            if (t + 4 < dmax) nxt = edge_quad(cl, len, a, deg, t + 4, self);
            const Quad q = quad_of(t);
            float v[P];
            bias_share<T, D, H, P>(v, b, q, t, deg, ln);
            const float4 x = bias_swap<T, D, H, P>(v, ln, s);
            step(cur.x, cur.y, t, t < deg, t + 1 < deg, x.x, x.y);
            if (t + 2 < dmax) step(cur.z, cur.w, t + 2, t + 2 < deg, t + 3 < deg, x.z, x.w);
            after(t, q);
            cur = nxt;
        }
    }
}

// ------------------------------------------------------------------ forward

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_fwd_rows(int64_t n, const int64_t* __restrict__ rp,
                                                       const int32_t* __restrict__ cl, int64_t len,
                                                       const T* __restrict__ Q,
                                                       const T* __restrict__ K, const T* __restrict__ V, float sl2,
                                                       T* __restrict__ O, float* __restrict__ LSE, TilePartials tp,
                                                       EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    const Lanes<T, D, H> ln(lane_id());
    const int64_t wave = xcd_block(blockIdx.x, gridDim.x) * (kThreads / kWave) + threadIdx.x / kWave;
    const int64_t i = wave * C::NPW + ln.slot;
    const bool live = i < n;
    const int64_t self = live ? i : 0;
    int64_t a = 0;
    int deg = 0;
    if (live) {
        a = rp[i];
        const int64_t dg = rp[i + 1] - a;
        deg = dg > GT_LONG_ROW ? -1 : int(dg);
    }
    const int dmax = wave_max(deg);
    const int64_t off = ln.off(self);
    Slice<T, C::F> q;
    q.load(Q + off);
    Online<C::F> st;
    if (live && deg >= 0 && tp.has_row(i)) load_fwd_partial<T, D, H>(st, tp, i, ln.h, off);
    using BS = BiasStage<T, D, H>;
    if constexpr (kBias && BS::kOn) {
        __shared__ float s_bias[kThreads / kWave][BS::kWaveFloats];
        float* sb = s_bias[threadIdx.x / kWave] + ln.slot * 4 * H;
        walk_edges_bias<T, D, H, true>(
            cl, len, a, deg, dmax, int32_t(self), eb.b, ln, sb,
            [&](int t) { return row_quad(eb, len, a, deg, t); },
            [&](int64_t j0, int64_t j1, int, bool ok0, bool ok1, float b0, float b1) {
                fwd_step<T, D, H, true>(st, q, K, V, j0, j1, ok0, ok1, ln, sl2, b0, b1);
            },
            [](int, const Quad&) {});
    } else {
        walk_edges(cl, len, a, deg, dmax, int32_t(self), [&](int64_t j0, int64_t j1, int t, bool ok0, bool ok1) {
            float b0 = 0.f, b1 = 0.f;
            if constexpr (kBias) bias_pair(eb, a, t, ok0, ok1, H, ln, b0, b1);
            fwd_step<T, D, H, kBias>(st, q, K, V, j0, j1, ok0, ok1, ln, sl2, b0, b1);
        });
    }
    if (live && deg >= 0) {
        const float inv = st.l > 0.f ? 1.f / st.l : 0.f;
        store_slice<T, C::F>(O + off, st.acc, inv);
        if (ln.part == 0) LSE[i * H + ln.h] = st.l > 0.f ? (st.m + __log2f(st.l)) * kLn2 : kNegInf;
    }
}

// ----------------------------------------------------------------- backward

// Row pass.  With D_i = sum_j P_ij dP_ij (which equals <dO_i, O_i> for the
// exact output O; the stored O is rounded to the feature dtype, so D is formed
// from the edges instead),
//   dQ_i = scale * sum_j P_ij (dP_ij - D_i) K_j = scale * (A_i - D_i B_i),
//   A_i = sum_j P_ij dP_ij K_j,  B_i = sum_j P_ij K_j,
// so one pass over the row yields A, B and D together.
template <int F>
struct RowSums {
    Acc<F> a, b;
    float d = 0.f;
};

template <typename T, int D, int H, bool kBias = false>
__device__ __forceinline__ void dq_step(RowSums<EdgeCfg<T, D, H>::F>& rs, const Slice<T, EdgeCfg<T, D, H>::F>& q,
                                        const Slice<T, EdgeCfg<T, D, H>::F>& g, float lse2, const T* __restrict__ K,
                                        const T* __restrict__ V, int64_t j0, int64_t j1, bool ok0, bool ok1,
                                        const Lanes<T, D, H>& ln, float sl2, float b0 = 0.f, float b1 = 0.f) {
    using C = EdgeCfg<T, D, H>;
    Slice<T, C::F> k0, k1, v0, v1;
    k0.load(K + ln.off(j0));
    k1.load(K + ln.off(j1));
    v0.load(V + ln.off(j0));
    v1.load(V + ln.off(j1));
    float s0 = group_sum<C::L>(q.dot(k0)) * sl2;
    float s1 = group_sum<C::L>(q.dot(k1)) * sl2;
    if constexpr (kBias) {
        s0 += b0;
        s1 += b1;
    }
    const float dp0 = group_sum<C::L>(g.dot(v0));
    const float dp1 = group_sum<C::L>(g.dot(v1));
    const float p0 = ok0 ? exp2f(s0 - lse2) : 0.f;
    const float p1 = ok1 ? exp2f(s1 - lse2) : 0.f;
    const float w0 = p0 * dp0;
    const float w1 = p1 * dp1;
    rs.d += w0 + w1;
#pragma unroll
    for (int f = 0; f < C::F; ++f) {
        const float x0 = k0.f(f), x1 = k1.f(f);
        rs.a.v[f] = fmaf(w1, x1, fmaf(w0, x0, rs.a.v[f]));
        rs.b.v[f] = fmaf(p1, x1, fmaf(p0, x0, rs.b.v[f]));
    }
}

template <int F>
__device__ __forceinline__ void load_f32_slice(float (&dst)[F], const float* src) {
    const float4* a = reinterpret_cast<const float4*>(src);
#pragma unroll
    for (int i = 0; i < F / 4; ++i) {
        float4 v = a[i];
        dst[4 * i] = v.x;
        dst[4 * i + 1] = v.y;
        dst[4 * i + 2] = v.z;
        dst[4 * i + 3] = v.w;
    }
}

template <typename T, int D, int H>
__device__ __forceinline__ void load_row_partial(RowSums<EdgeCfg<T, D, H>::F>& rs, const TilePartials& tp,
                                                 int64_t node, int h, int64_t off) {
    constexpr int F = EdgeCfg<T, D, H>::F;
    load_f32_slice<F>(rs.a.v, tp.acc + off);
    load_f32_slice<F>(rs.b.v, tp.acc2 + off);
    rs.d = tp.m[node * H + h];
}

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_bwd_rows(int64_t n, const int64_t* __restrict__ rp,
                                                       const int32_t* __restrict__ cl, int64_t len,
                                                       const T* __restrict__ Q,
                                                       const T* __restrict__ K, const T* __restrict__ V,
                                                       const T* __restrict__ dO, const float* __restrict__ LSE,
                                                       float* __restrict__ Dv, float sl2, float scale,
                                                       T* __restrict__ dQ, TilePartials tp, EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    const Lanes<T, D, H> ln(lane_id());
    const int64_t wave = xcd_block(blockIdx.x, gridDim.x) * (kThreads / kWave) + threadIdx.x / kWave;
    const int64_t i = wave * C::NPW + ln.slot;
    const bool live = i < n;
    const int64_t self = live ? i : 0;
    int64_t a = 0;
    int deg = 0;
    if (live) {
        a = rp[i];
        const int64_t dg = rp[i + 1] - a;
        deg = dg > GT_LONG_ROW ? -1 : int(dg);
    }
    const int dmax = wave_max(deg);
    const int64_t off = ln.off(self);
    Slice<T, C::F> q, g;
    q.load(Q + off);
    g.load(dO + off);
    const float lse2 = LSE[self * H + ln.h] * kLog2e;
    RowSums<C::F> rs;
    if (live && deg >= 0 && tp.has_row(i)) load_row_partial<T, D, H>(rs, tp, i, ln.h, off);
    using BS = BiasStage<T, D, H>;
    if constexpr (kBias && BS::kOn) {
        __shared__ float s_bias[kThreads / kWave][BS::kWaveFloats];
        float* sb = s_bias[threadIdx.x / kWave] + ln.slot * 4 * H;
        walk_edges_bias<T, D, H, false>(
            cl, len, a, deg, dmax, int32_t(self), eb.b, ln, sb,
            [&](int t) { return row_quad(eb, len, a, deg, t); },
            [&](int64_t j0, int64_t j1, int, bool ok0, bool ok1, float b0, float b1) {
                dq_step<T, D, H, true>(rs, q, g, lse2, K, V, j0, j1, ok0, ok1, ln, sl2, b0, b1);
            },
            [](int, const Quad&) {});
    } else {
        walk_edges(cl, len, a, deg, dmax, int32_t(self), [&](int64_t j0, int64_t j1, int t, bool ok0, bool ok1) {
            float b0 = 0.f, b1 = 0.f;
            if constexpr (kBias) bias_pair(eb, a, t, ok0, ok1, H, ln, b0, b1);
            dq_step<T, D, H, kBias>(rs, q, g, lse2, K, V, j0, j1, ok0, ok1, ln, sl2, b0, b1);
        });
    }
    if (live && deg >= 0) {
#pragma unroll
        for (int f = 0; f < C::F; ++f) rs.a.v[f] = fmaf(-rs.d, rs.b.v[f], rs.a.v[f]);
        store_slice<T, C::F>(dQ + off, rs.a.v, scale);
        if (ln.part == 0) Dv[i * H + ln.h] = rs.d;
    }
}

// Column pass: dK_j = scale * sum_i dS_ij Q_i, dV_j = sum_i P_ij dO_i over the in-edges of j.
// With a bias, c0/c1 are the two in-edges' CSC positions; the bias is read and
// dB = dS written at their CSR positions.
template <typename T, int D, int H, bool kBias = false>
__device__ __forceinline__ void dkv_step(Acc<EdgeCfg<T, D, H>::F>& dk, Acc<EdgeCfg<T, D, H>::F>& dv,
                                         const Slice<T, EdgeCfg<T, D, H>::F>& k,
                                         const Slice<T, EdgeCfg<T, D, H>::F>& v, const T* __restrict__ Q,
                                         const T* __restrict__ dO, const float2* __restrict__ stat, int64_t i0,
                                         int64_t i1, bool ok0, bool ok1, const Lanes<T, D, H>& ln, float sl2,
                                         const EdgeBias& eb = EdgeBias{}, int64_t c0 = 0, int64_t c1 = 0,
                                         float* staged = nullptr) {
    using C = EdgeCfg<T, D, H>;
    Slice<T, C::F> q0, q1, g0, g1;
    q0.load(Q + ln.off(i0));
    q1.load(Q + ln.off(i1));
    g0.load(dO + ln.off(i0));
    g1.load(dO + ln.off(i1));
    // one lane of each (node, head) group reads the pair; the others take it by DPP
    float2 st0 = make_float2(0.f, 0.f), st1 = make_float2(0.f, 0.f);
    if (ln.part == 0) {
        st0 = stat[i0 * H + ln.h];
        st1 = stat[i1 * H + ln.h];
    }
    const float l0 = group_bcast0<C::L>(st0.x), D0 = group_bcast0<C::L>(st0.y);
    const float l1 = group_bcast0<C::L>(st1.x), D1 = group_bcast0<C::L>(st1.y);
    float s0 = group_sum<C::L>(q0.dot(k)) * sl2;
    float s1 = group_sum<C::L>(q1.dot(k)) * sl2;
    int64_t e0 = 0, e1 = 0;
    if (kBias && staged) {
        // staged: the bias came through LDS (staged[0..1]), dS goes back in staged[2..3]
        s0 += staged[0];
        s1 += staged[1];
    } else if constexpr (kBias) {
        // the node's first lane reads the CSR positions, one lane per head the bias
        int p0 = 0, p1 = 0;
        if ((lane_id() & (C::G - 1)) == 0) {
            p0 = ok0 ? eb.csc_pos[c0] : 0;
            p1 = ok1 ? eb.csc_pos[c1] : 0;
        }
        e0 = group_first<C::G>(p0);
        e1 = group_first<C::G>(p1);
        float x0 = 0.f, x1 = 0.f;
        if (ln.part == 0) {
            x0 = ok0 ? eb.at_input(e0, H, ln.h) : 0.f;
            x1 = ok1 ? eb.at_input(e1, H, ln.h) : 0.f;
        }
        s0 += group_bcast0<C::L>(x0);
        s1 += group_bcast0<C::L>(x1);
    }
    const float dp0 = group_sum<C::L>(g0.dot(v));
    const float dp1 = group_sum<C::L>(g1.dot(v));
    const float p0 = ok0 ? exp2f(s0 - l0) : 0.f;
    const float p1 = ok1 ? exp2f(s1 - l1) : 0.f;
    const float ds0 = p0 * (dp0 - D0);
    const float ds1 = p1 * (dp1 - D1);
    if (kBias && staged) {
        staged[2] = ok0 ? ds0 : 0.f;
        staged[3] = ok1 ? ds1 : 0.f;
    } else if constexpr (kBias) {
        if (ln.part == 0) {
            if (ok0) eb.db[e0 * H + ln.h] = ds0;
            if (ok1) eb.db[e1 * H + ln.h] = ds1;
        }
    }
#pragma unroll
    for (int f = 0; f < C::F; ++f) {
        dk.v[f] = fmaf(ds1, q1.f(f), fmaf(ds0, q0.f(f), dk.v[f]));
        dv.v[f] = fmaf(p1, g1.f(f), fmaf(p0, g0.f(f), dv.v[f]));
    }
}

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_bwd_cols(int64_t n, const int64_t* __restrict__ cp,
                                                       const int32_t* __restrict__ rw, int64_t len,
                                                       const T* __restrict__ Q,
                                                       const T* __restrict__ K, const T* __restrict__ V,
                                                       const T* __restrict__ dO, const float2* __restrict__ stat,
                                                       float sl2, float scale, T* __restrict__ dK,
                                                       T* __restrict__ dV, TilePartials tpk, TilePartials tpv,
                                                       EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    const Lanes<T, D, H> ln(lane_id());
    const int64_t wave = xcd_block(blockIdx.x, gridDim.x) * (kThreads / kWave) + threadIdx.x / kWave;
    const int64_t j = wave * C::NPW + ln.slot;
    const bool live = j < n;
    const int64_t self = live ? j : 0;
    int64_t a = 0;
    int deg = 0;
    if (live) {
        a = cp[j];
        const int64_t dg = cp[j + 1] - a;
        deg = dg > GT_LONG_ROW ? -1 : int(dg);
    }
    const int dmax = wave_max(deg);
    const int64_t off = ln.off(self);
    Slice<T, C::F> k, v;
    k.load(K + off);
    v.load(V + off);
    Acc<C::F> dk, dv;
    if (live && deg >= 0 && tpk.has_col(j)) {
        load_f32_slice<C::F>(dk.v, tpk.acc + off);
        load_f32_slice<C::F>(dv.v, tpv.acc + off);
    }
    using BS = BiasStage<T, D, H>;
    if constexpr (kBias && BS::kOn) {
        __shared__ float s_bias[kThreads / kWave][BS::kWaveFloats];
        float* sb = s_bias[threadIdx.x / kWave] + ln.slot * 4 * H;
        float4 ds = make_float4(0.f, 0.f, 0.f, 0.f);
        walk_edges_bias<T, D, H, true>(
            rw, len, a, deg, dmax, int32_t(self), eb.b, ln, sb,
            [&](int t) { return col_quad(eb, len, a, deg, t); },
            [&](int64_t i0, int64_t i1, int t, bool ok0, bool ok1, float b0, float b1) {
                float x[4] = {b0, b1, 0.f, 0.f};
                dkv_step<T, D, H, true>(dk, dv, k, v, Q, dO, stat, i0, i1, ok0, ok1, ln, sl2, eb, 0, 0, x);
                if (t & 2) ds.z = x[2], ds.w = x[3];
                else ds.x = x[2], ds.y = x[3], ds.z = 0.f, ds.w = 0.f;
            },
            [&](int t, const Quad& q) { db_quad<T, D, H>(eb.db, q, t, deg, ds, ln, sb); });
    } else {
        walk_edges(rw, len, a, deg, dmax, int32_t(self), [&](int64_t i0, int64_t i1, int t, bool ok0, bool ok1) {
            dkv_step<T, D, H, kBias>(dk, dv, k, v, Q, dO, stat, i0, i1, ok0, ok1, ln, sl2, eb, a + t, a + t + 1);
        });
    }
    if (live && deg >= 0) {
        store_slice<T, C::F>(dK + off, dk.v, scale);
        store_slice<T, C::F>(dV + off, dv.v, 1.f);
    }
}

// ------------------------------------------------------------- long rows
// Remainder rows (columns) with more than GT_LONG_ROW edges, up to a row that
// attends to every node: each is cut into chunks of kChunk edges, one
// workgroup per chunk leaves a partial state (its lane groups take the edges
// round-robin and merge in LDS), and one workgroup per long row merges its
// chunks with the row's dense-tile partial and writes the result.  The chunk
// table is built on the device; the chunk grid is launched at its upper bound
// (one chunk per long row plus one per kChunk remainder edges) and surplus
// workgroups return at once.
constexpr int kChunk = 2048;

template <int H, int D>
constexpr int64_t FwdLongF = int64_t(H) * D + 2 * H;  // floats per chunk: m[H], l[H], acc[H D]
template <int H, int D>
constexpr int64_t RowLongF = 2 * int64_t(H) * D + H;  // a[H D], b[H D], d[H]
template <int H, int D>
constexpr int64_t ColLongF = 2 * int64_t(H) * D;      // dk[H D], dv[H D]

struct LongPlan {
    int32_t* counts = nullptr;     // [n_long]: chunks of each long row
    int64_t* chunk_off = nullptr;  // [n_long + 1]: exclusive scan of counts
    float* part = nullptr;         // [max_chunks, floats per chunk]
    int64_t max_chunks = 0;
    ScanTmp scan;
};

inline LongPlan long_plan_take(Ws& ws, int64_t n_long, int64_t nnz, int64_t per_chunk) {
    LongPlan lp;
    if (n_long <= 0) return lp;
    lp.max_chunks = n_long + nnz / kChunk + 1;
    lp.counts = ws.take<int32_t>(size_t(n_long));
    lp.chunk_off = ws.take<int64_t>(size_t(n_long + 1));
    lp.scan.block_sums = ws.take<int64_t>(size_t(scan_tmp_elems(n_long)));
    lp.part = ws.take<float>(size_t(lp.max_chunks * per_chunk));
    return lp;
}

__global__ void k_long_counts(const int32_t* __restrict__ list, int64_t n_long, const int64_t* __restrict__ ptr,
                              int32_t* __restrict__ counts) {
    const int64_t r = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (r >= n_long) return;
    const int64_t i = list[r];
    counts[r] = int32_t(cdiv(ptr[i + 1] - ptr[i], kChunk));
}

gt_status long_chunks(const int32_t* list, int64_t n_long, const int64_t* ptr, const LongPlan& lp, hipStream_t s) {
    k_long_counts<<<grid_for(n_long, 256), 256, 0, s>>>(list, n_long, ptr, lp.counts);
    GT_LAUNCH_CHECK("long_counts");
    return exclusive_scan_i32(lp.counts, n_long, lp.chunk_off, lp.scan, s);
}

// Chunk b -> (long row r, chunk c of that row, its edge range [e0, e1) inside
// the row); false for the surplus of the grid.
__device__ __forceinline__ bool chunk_of(const int64_t* __restrict__ off, int64_t n_long, int64_t b, int64_t& r,
                                         int& e0) {
    if (b >= off[n_long]) return false;
    int64_t lo = 0, hi = n_long;  // the last r with off[r] <= b
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (off[mid] <= b) lo = mid;
        else hi = mid;
    }
    r = lo;
    e0 = int(b - off[lo]) * kChunk;
    return true;
}

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_fwd_long(const int32_t* __restrict__ list, int64_t n_long,
                                                       const int64_t* __restrict__ chunk_off,
                                                       const int64_t* __restrict__ rp,
                                                       const int32_t* __restrict__ cl, const T* __restrict__ Q,
                                                       const T* __restrict__ K, const T* __restrict__ V, float sl2,
                                                       float* __restrict__ part, EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    constexpr int S = kThreads / C::G;  // lane groups per workgroup
    __shared__ float s_m[S][H];
    __shared__ float s_l[S][H];
    __shared__ float s_acc[S][H * D];
    int64_t r;
    int e0;
    if (!chunk_of(chunk_off, n_long, blockIdx.x, r, e0)) return;
    const Lanes<T, D, H> ln(threadIdx.x);
    const int64_t i = list[r];
    const int64_t a = rp[i];
    const int deg = int(rp[i + 1] - a);
    const int e1 = e0 + kChunk < deg ? e0 + kChunk : deg;
    const int64_t off = ln.off(i);
    Slice<T, C::F> q;
    q.load(Q + off);
    Online<C::F> st;
    for (int t = e0 + ln.slot; t < e1; t += 2 * S) {
        const bool ok1 = t + S < e1;
        const int64_t j0 = cl[a + t];
        const int64_t j1 = ok1 ? cl[a + t + S] : j0;
        float b0 = 0.f, b1 = 0.f;
        if constexpr (kBias) {
            b0 = eb.at(a + t, H, ln.h);
            b1 = ok1 ? eb.at(a + t + S, H, ln.h) : 0.f;
        }
        fwd_step<T, D, H, kBias>(st, q, K, V, j0, j1, true, ok1, ln, sl2, b0, b1);
    }
    if (ln.part == 0) {
        s_m[ln.slot][ln.h] = st.m;
        s_l[ln.slot][ln.h] = st.l;
    }
#pragma unroll
    for (int f = 0; f < C::F; ++f) s_acc[ln.slot][ln.h * D + ln.part * C::F + f] = st.acc[f];
    __syncthreads();
    float* out = part + blockIdx.x * FwdLongF<H, D>;
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        const int h = idx / D;
        float M = kNegInf;
        for (int g = 0; g < S; ++g) M = fmaxf(M, s_m[g][h]);
        float lsum = 0.f, o = 0.f;
        if (M != kNegInf) {
            for (int g = 0; g < S; ++g) {
                const float w = exp2f(s_m[g][h] - M);
                lsum += s_l[g][h] * w;
                o += s_acc[g][idx] * w;
            }
        }
        out[2 * H + idx] = o;
        if (idx % D == 0) {
            out[h] = M;
            out[H + h] = lsum;
        }
    }
}

template <typename T, int D, int H>
__global__ __launch_bounds__(kThreads) void k_fwd_long_merge(const int32_t* __restrict__ list,
                                                             const int64_t* __restrict__ chunk_off,
                                                             const float* __restrict__ part, TilePartials tp,
                                                             T* __restrict__ O, float* __restrict__ LSE) {
    const int64_t i = list[blockIdx.x];
    const int64_t c0 = chunk_off[blockIdx.x], c1 = chunk_off[blockIdx.x + 1];
    const bool tile = tp.has_row(i);
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        const int h = idx / D;
        float M = tile ? tp.m[i * H + h] : kNegInf;
        for (int64_t c = c0; c < c1; ++c) M = fmaxf(M, part[c * FwdLongF<H, D> + h]);
        float lsum = 0.f, o = 0.f;
        if (M != kNegInf) {
            if (tile) {
                const float w = exp2f(tp.m[i * H + h] - M);
                lsum = tp.l[i * H + h] * w;
                o = tp.acc[i * H * D + idx] * w;
            }
            for (int64_t c = c0; c < c1; ++c) {
                const float* pc = part + c * FwdLongF<H, D>;
                const float w = exp2f(pc[h] - M);
                lsum += pc[H + h] * w;
                o += pc[2 * H + idx] * w;
            }
        }
        const float val = lsum > 0.f ? o / lsum : 0.f;
        if (sizeof(T) == 2)
            reinterpret_cast<uint16_t*>(O)[i * H * D + idx] = f32_to_bf16(val);
        else
            reinterpret_cast<float*>(O)[i * H * D + idx] = val;
        if (idx % D == 0) LSE[i * H + h] = lsum > 0.f ? (M + __log2f(lsum)) * kLn2 : kNegInf;
    }
}

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_bwd_rows_long(const int32_t* __restrict__ list, int64_t n_long,
                                                            const int64_t* __restrict__ chunk_off,
                                                            const int64_t* __restrict__ rp,
                                                            const int32_t* __restrict__ cl, const T* __restrict__ Q,
                                                            const T* __restrict__ K, const T* __restrict__ V,
                                                            const T* __restrict__ dO, const float* __restrict__ LSE,
                                                            float sl2, float* __restrict__ part, EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    constexpr int S = kThreads / C::G;
    __shared__ float s_a[S][H * D];
    __shared__ float s_b[S][H * D];
    __shared__ float s_d[S][H];
    int64_t r;
    int e0;
    if (!chunk_of(chunk_off, n_long, blockIdx.x, r, e0)) return;
    const Lanes<T, D, H> ln(threadIdx.x);
    const int64_t i = list[r];
    const int64_t a = rp[i];
    const int deg = int(rp[i + 1] - a);
    const int e1 = e0 + kChunk < deg ? e0 + kChunk : deg;
    const int64_t off = ln.off(i);
    Slice<T, C::F> q, g;
    q.load(Q + off);
    g.load(dO + off);
    const float lse2 = LSE[i * H + ln.h] * kLog2e;
    RowSums<C::F> rs;
    for (int t = e0 + ln.slot; t < e1; t += 2 * S) {
        const bool ok1 = t + S < e1;
        const int64_t j0 = cl[a + t];
        const int64_t j1 = ok1 ? cl[a + t + S] : j0;
        float b0 = 0.f, b1 = 0.f;
        if constexpr (kBias) {
            b0 = eb.at(a + t, H, ln.h);
            b1 = ok1 ? eb.at(a + t + S, H, ln.h) : 0.f;
        }
        dq_step<T, D, H, kBias>(rs, q, g, lse2, K, V, j0, j1, true, ok1, ln, sl2, b0, b1);
    }
#pragma unroll
    for (int f = 0; f < C::F; ++f) {
        s_a[ln.slot][ln.h * D + ln.part * C::F + f] = rs.a.v[f];
        s_b[ln.slot][ln.h * D + ln.part * C::F + f] = rs.b.v[f];
    }
    if (ln.part == 0) s_d[ln.slot][ln.h] = rs.d;
    __syncthreads();
    float* out = part + blockIdx.x * RowLongF<H, D>;
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        const int h = idx / D;
        float sa = 0.f, sb = 0.f, sd = 0.f;
        for (int gi = 0; gi < S; ++gi) {
            sa += s_a[gi][idx];
            sb += s_b[gi][idx];
            sd += s_d[gi][h];
        }
        out[idx] = sa;
        out[H * D + idx] = sb;
        if (idx % D == 0) out[2 * H * D + h] = sd;
    }
}

template <typename T, int D, int H>
__global__ __launch_bounds__(kThreads) void k_bwd_rows_long_merge(const int32_t* __restrict__ list,
                                                                  const int64_t* __restrict__ chunk_off,
                                                                  const float* __restrict__ part, TilePartials tp,
                                                                  float scale, T* __restrict__ dQ,
                                                                  float* __restrict__ Dv) {
    const int64_t i = list[blockIdx.x];
    const int64_t c0 = chunk_off[blockIdx.x], c1 = chunk_off[blockIdx.x + 1];
    const bool tile = tp.has_row(i);
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        const int h = idx / D;
        float sa = tile ? tp.acc[i * H * D + idx] : 0.f;
        float sb = tile ? tp.acc2[i * H * D + idx] : 0.f;
        float sd = tile ? tp.m[i * H + h] : 0.f;
        for (int64_t c = c0; c < c1; ++c) {
            const float* pc = part + c * RowLongF<H, D>;
            sa += pc[idx];
            sb += pc[H * D + idx];
            sd += pc[2 * H * D + h];
        }
        const float v = fmaf(-sd, sb, sa) * scale;
        if (sizeof(T) == 2)
            reinterpret_cast<uint16_t*>(dQ)[i * H * D + idx] = f32_to_bf16(v);
        else
            reinterpret_cast<float*>(dQ)[i * H * D + idx] = v;
        if (idx % D == 0) Dv[i * H + h] = sd;
    }
}

template <typename T, int D, int H, bool kBias>
__global__ __launch_bounds__(kThreads) void k_bwd_cols_long(const int32_t* __restrict__ list, int64_t n_long,
                                                            const int64_t* __restrict__ chunk_off,
                                                            const int64_t* __restrict__ cp,
                                                            const int32_t* __restrict__ rw, const T* __restrict__ Q,
                                                            const T* __restrict__ K, const T* __restrict__ V,
                                                            const T* __restrict__ dO,
                                                            const float2* __restrict__ stat, float sl2,
                                                            float* __restrict__ part, EdgeBias eb) {
    using C = EdgeCfg<T, D, H>;
    constexpr int S = kThreads / C::G;
    __shared__ float s_k[S][H * D];
    __shared__ float s_v[S][H * D];
    int64_t r;
    int e0;
    if (!chunk_of(chunk_off, n_long, blockIdx.x, r, e0)) return;
    const Lanes<T, D, H> ln(threadIdx.x);
    const int64_t j = list[r];
    const int64_t a = cp[j];
    const int deg = int(cp[j + 1] - a);
    const int e1 = e0 + kChunk < deg ? e0 + kChunk : deg;
    const int64_t off = ln.off(j);
    Slice<T, C::F> k, v;
    k.load(K + off);
    v.load(V + off);
    Acc<C::F> dk, dv;
    for (int t = e0 + ln.slot; t < e1; t += 2 * S) {
        const bool ok1 = t + S < e1;
        const int64_t i0 = rw[a + t];
        const int64_t i1 = ok1 ? rw[a + t + S] : i0;
        dkv_step<T, D, H, kBias>(dk, dv, k, v, Q, dO, stat, i0, i1, true, ok1, ln, sl2, eb, a + t, a + t + S);
    }
#pragma unroll
    for (int f = 0; f < C::F; ++f) {
        s_k[ln.slot][ln.h * D + ln.part * C::F + f] = dk.v[f];
        s_v[ln.slot][ln.h * D + ln.part * C::F + f] = dv.v[f];
    }
    __syncthreads();
    float* out = part + blockIdx.x * ColLongF<H, D>;
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        float ak = 0.f, av = 0.f;
        for (int g = 0; g < S; ++g) {
            ak += s_k[g][idx];
            av += s_v[g][idx];
        }
        out[idx] = ak;
        out[H * D + idx] = av;
    }
}

template <typename T, int D, int H>
__global__ __launch_bounds__(kThreads) void k_bwd_cols_long_merge(const int32_t* __restrict__ list,
                                                                  const int64_t* __restrict__ chunk_off,
                                                                  const float* __restrict__ part, TilePartials tpk,
                                                                  TilePartials tpv, float scale,
                                                                  T* __restrict__ dK, T* __restrict__ dV) {
    const int64_t j = list[blockIdx.x];
    const int64_t c0 = chunk_off[blockIdx.x], c1 = chunk_off[blockIdx.x + 1];
    const bool tile = tpk.has_col(j);
    for (int idx = threadIdx.x; idx < H * D; idx += kThreads) {
        float ak = tile ? tpk.acc[j * H * D + idx] : 0.f;
        float av = tile ? tpv.acc[j * H * D + idx] : 0.f;
        for (int64_t c = c0; c < c1; ++c) {
            const float* pc = part + c * ColLongF<H, D>;
            ak += pc[idx];
            av += pc[H * D + idx];
        }
        ak *= scale;
        if (sizeof(T) == 2) {
            reinterpret_cast<uint16_t*>(dK)[j * H * D + idx] = f32_to_bf16(ak);
            reinterpret_cast<uint16_t*>(dV)[j * H * D + idx] = f32_to_bf16(av);
        } else {
            reinterpret_cast<float*>(dK)[j * H * D + idx] = ak;
            reinterpret_cast<float*>(dV)[j * H * D + idx] = av;
        }
    }
}

// The column pass reads each in-edge's row statistics as one (LSE log2 e, D)
// pair: one 8-byte gather per edge instead of two 4-byte ones.
__global__ void k_pack_stats(int64_t m, const float* __restrict__ LSE, const float* __restrict__ Dv,
                             float2* __restrict__ out) {
    for (int64_t x = blockIdx.x * int64_t(blockDim.x) + threadIdx.x; x < m; x += int64_t(gridDim.x) * blockDim.x)
        out[x] = make_float2(LSE[x] * kLog2e, Dv[x]);
}

// ------------------------------------------------------------ gather probe
// Measurement only: the forward edge kernel's data movement (every remainder
// edge of a row of at most GT_LONG_ROW edges reads its partner's two feature
// rows, same lanes, same edge walk) with no arithmetic but an XOR, so the rate
// the gather path allows for a plan can be timed beside the real kernels.
template <int F>
__device__ __forceinline__ uint32_t xor_words(const Slice<uint16_t, F>& x) {
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < F / 2; ++i) r ^= x.w[i];
    return r;
}
template <int F>
__device__ __forceinline__ uint32_t xor_words(const Slice<float, F>& x) {
    uint32_t r = 0;
#pragma unroll
    for (int i = 0; i < F; ++i) r ^= __float_as_uint(x.w[i]);
    return r;
}

constexpr uint32_t kProbeSinkKey = 0x9E3779B9u;

template <typename T, int D, int H>
__global__ __launch_bounds__(kThreads) void k_gather_probe(int64_t n, const int64_t* __restrict__ rp,
                                                           const int32_t* __restrict__ cl, int64_t len,
                                                           const T* __restrict__ A, const T* __restrict__ B,
                                                           uint32_t* __restrict__ sink) {
    using C = EdgeCfg<T, D, H>;
    const Lanes<T, D, H> ln(lane_id());
    const int64_t wave = xcd_block(blockIdx.x, gridDim.x) * (kThreads / kWave) + threadIdx.x / kWave;
    const int64_t i = wave * C::NPW + ln.slot;
    const bool live = i < n;
    const int64_t self = live ? i : 0;
    int64_t a = 0;
    int deg = 0;
    if (live) {
        a = rp[i];
        const int64_t dg = rp[i + 1] - a;
        deg = dg > GT_LONG_ROW ? -1 : int(dg);
    }
    const int dmax = wave_max(deg);
    uint32_t acc = 0;
    walk_edges(cl, len, a, deg, dmax, int32_t(self), [&](int64_t j0, int64_t j1, int, bool, bool) {
        Slice<T, C::F> a0, a1, b0, b1;
        a0.load(A + ln.off(j0));
        a1.load(A + ln.off(j1));
        b0.load(B + ln.off(j0));
        b1.load(B + ln.off(j1));
        acc ^= xor_words(a0) ^ xor_words(a1) ^ xor_words(b0) ^ xor_words(b1);
    });
    if (acc == kProbeSinkKey) sink[0] = acc;  // keeps the loads; practically never taken
}

template <typename T, int D, int H>
gt_status run_probe(const gt_tiles* p, const void* A, const void* B, uint32_t* sink, hipStream_t s) {
    using C = EdgeCfg<T, D, H>;
    if (p->n == 0) return GT_OK;
    const unsigned grid = xcd_grid(cdiv(cdiv(p->n, C::NPW), kThreads / kWave));
    k_gather_probe<T, D, H><<<grid, kThreads, 0, s>>>(p->n, p->sp_rowptr, p->sp_col, p->nnz_sparse,
                                                      static_cast<const T*>(A), static_cast<const T*>(B), sink);
    GT_LAUNCH_CHECK("gather_probe");
    return GT_OK;
}

// ---------------------------------------------------------------- launchers

struct FwdWs {
    TilePartials tp;
};

template <typename T, int D, int H, bool kBias>
gt_status run_fwd_t(const gt_tiles* p, const void* Q, const void* K, const void* V, float scale, void* O, float* LSE,
                    void* ws_ptr, EdgeBias eb, hipStream_t s) {
    using C = EdgeCfg<T, D, H>;
    const int64_t n = p->n;
    if (n == 0) return GT_OK;
    Ws ws(ws_ptr);
    ws.take<char>(256);
    TilePartials tp = tile_partials_fwd(ws, p, H, D);
    LongPlan lp = long_plan_take(ws, p->n_long_rows, p->nnz_sparse, FwdLongF<H, D>);
    const float sl2 = scale * kLog2e;
    gt_status st;
    if (p->n_dense > 0) {
        if ((st = tile_fwd<T, D, H>(p, static_cast<const T*>(Q), static_cast<const T*>(K),
                                    static_cast<const T*>(V), sl2, tp, eb.tile, s)) != GT_OK)
            return st;
    } else {
        tp = TilePartials{};
    }
    const int64_t waves = cdiv(n, C::NPW);
    k_fwd_rows<T, D, H, kBias><<<xcd_grid(cdiv(waves, kThreads / kWave)), kThreads, 0, s>>>(
        n, p->sp_rowptr, p->sp_col, p->nnz_sparse, static_cast<const T*>(Q), static_cast<const T*>(K),
        static_cast<const T*>(V), sl2, static_cast<T*>(O), LSE, tp, eb);
    GT_LAUNCH_CHECK("sparse_fwd_rows");
    if (p->n_long_rows > 0) {
        if ((st = long_chunks(p->long_rows, p->n_long_rows, p->sp_rowptr, lp, s)) != GT_OK) return st;
        k_fwd_long<T, D, H, kBias><<<unsigned(lp.max_chunks), kThreads, 0, s>>>(
            p->long_rows, p->n_long_rows, lp.chunk_off, p->sp_rowptr, p->sp_col, static_cast<const T*>(Q),
            static_cast<const T*>(K), static_cast<const T*>(V), sl2, lp.part, eb);
        GT_LAUNCH_CHECK("sparse_fwd_long");
        k_fwd_long_merge<T, D, H><<<unsigned(p->n_long_rows), kThreads, 0, s>>>(
            p->long_rows, lp.chunk_off, lp.part, tp, static_cast<T*>(O), LSE);
        GT_LAUNCH_CHECK("sparse_fwd_long_merge");
    }
    return GT_OK;
}

template <typename T, int D, int H>
gt_status run_fwd(const gt_tiles* p, const void* Q, const void* K, const void* V, float scale, void* O, float* LSE,
                  void* ws_ptr, EdgeBias eb, hipStream_t s) {
    return eb.b ? run_fwd_t<T, D, H, true>(p, Q, K, V, scale, O, LSE, ws_ptr, eb, s)
                : run_fwd_t<T, D, H, false>(p, Q, K, V, scale, O, LSE, ws_ptr, eb, s);
}

template <typename T, int D, int H, bool kBias>
gt_status run_bwd_rows_t(const gt_tiles* p, const void* Q, const void* K, const void* V, const void* dO,
                         const float* LSE, float scale, void* dQ, float* Dv, void* ws_ptr, EdgeBias eb,
                         hipStream_t s) {
    using C = EdgeCfg<T, D, H>;
    const int64_t n = p->n;
    if (n == 0) return GT_OK;
    Ws ws(ws_ptr);
    ws.take<char>(256);
    TileBwdPartials tb = tile_partials_bwd(ws, p, H, D, true, false);
    LongPlan lp = long_plan_take(ws, p->n_long_rows, p->nnz_sparse, RowLongF<H, D>);
    const float sl2 = scale * kLog2e;
    const T *q = static_cast<const T*>(Q), *k = static_cast<const T*>(K), *v = static_cast<const T*>(V);
    const T* g = static_cast<const T*>(dO);
    gt_status st;
    if (p->n_dense > 0) {
        if ((st = tile_bwd_dq<T, D, H>(p, q, k, v, g, LSE, sl2, tb.dq, eb.tile, s)) != GT_OK) return st;
    }
    const unsigned grid = xcd_grid(cdiv(cdiv(n, C::NPW), kThreads / kWave));
    k_bwd_rows<T, D, H, kBias><<<grid, kThreads, 0, s>>>(n, p->sp_rowptr, p->sp_col, p->nnz_sparse, q, k, v, g,
                                                         LSE, Dv, sl2, scale, static_cast<T*>(dQ), tb.dq, eb);
    GT_LAUNCH_CHECK("sparse_bwd_rows");
    if (p->n_long_rows > 0) {
        if ((st = long_chunks(p->long_rows, p->n_long_rows, p->sp_rowptr, lp, s)) != GT_OK) return st;
        k_bwd_rows_long<T, D, H, kBias><<<unsigned(lp.max_chunks), kThreads, 0, s>>>(
            p->long_rows, p->n_long_rows, lp.chunk_off, p->sp_rowptr, p->sp_col, q, k, v, g, LSE, sl2, lp.part, eb);
        GT_LAUNCH_CHECK("sparse_bwd_rows_long");
        k_bwd_rows_long_merge<T, D, H><<<unsigned(p->n_long_rows), kThreads, 0, s>>>(
            p->long_rows, lp.chunk_off, lp.part, tb.dq, scale, static_cast<T*>(dQ), Dv);
        GT_LAUNCH_CHECK("sparse_bwd_rows_long_merge");
    }
    return GT_OK;
}

template <typename T, int D, int H>
gt_status run_bwd_rows(const gt_tiles* p, const void* Q, const void* K, const void* V, const void* dO,
                       const float* LSE, float scale, void* dQ, float* Dv, void* ws_ptr, EdgeBias eb, hipStream_t s) {
    return eb.b ? run_bwd_rows_t<T, D, H, true>(p, Q, K, V, dO, LSE, scale, dQ, Dv, ws_ptr, eb, s)
                : run_bwd_rows_t<T, D, H, false>(p, Q, K, V, dO, LSE, scale, dQ, Dv, ws_ptr, eb, s);
}

template <typename T, int D, int H, bool kBias>
gt_status run_bwd_cols_t(const gt_tiles* p, const void* Q, const void* K, const void* V, const void* dO,
                         const float* LSE, const float* Dv, float scale, void* dK, void* dV, void* ws_ptr,
                         EdgeBias eb, hipStream_t s) {
    using C = EdgeCfg<T, D, H>;
    const int64_t n = p->n;
    if (n == 0) return GT_OK;
    Ws ws(ws_ptr);
    ws.take<char>(256);
    TileBwdPartials tb = tile_partials_bwd(ws, p, H, D, false, true);
    LongPlan lp = long_plan_take(ws, p->n_long_cols, p->nnz_sparse, ColLongF<H, D>);
    float2* stat = ws.take<float2>(size_t(n) * H);
    const float sl2 = scale * kLog2e;
    const T *q = static_cast<const T*>(Q), *k = static_cast<const T*>(K), *v = static_cast<const T*>(V);
    const T* g = static_cast<const T*>(dO);
    gt_status st;
    if (p->n_dense > 0) {
        if ((st = tile_bwd_dkdv<T, D, H>(p, q, k, v, g, LSE, Dv, sl2, tb.dk, tb.dv, eb.tile, s)) != GT_OK)
            return st;
    }
    k_pack_stats<<<grid_for(n * H, 256, 8192), 256, 0, s>>>(n * H, LSE, Dv, stat);
    GT_LAUNCH_CHECK("sparse_bwd_pack_stats");
    const unsigned grid = xcd_grid(cdiv(cdiv(n, C::NPW), kThreads / kWave));
    k_bwd_cols<T, D, H, kBias><<<grid, kThreads, 0, s>>>(n, p->sp_colptr, p->sp_row, p->nnz_sparse, q, k, v, g,
                                                         stat, sl2, scale, static_cast<T*>(dK),
                                                         static_cast<T*>(dV), tb.dk, tb.dv, eb);
    GT_LAUNCH_CHECK("sparse_bwd_cols");
    if (p->n_long_cols > 0) {
        if ((st = long_chunks(p->long_cols, p->n_long_cols, p->sp_colptr, lp, s)) != GT_OK) return st;
        k_bwd_cols_long<T, D, H, kBias><<<unsigned(lp.max_chunks), kThreads, 0, s>>>(
            p->long_cols, p->n_long_cols, lp.chunk_off, p->sp_colptr, p->sp_row, q, k, v, g, stat, sl2, lp.part,
            eb);
        GT_LAUNCH_CHECK("sparse_bwd_cols_long");
        k_bwd_cols_long_merge<T, D, H><<<unsigned(p->n_long_cols), kThreads, 0, s>>>(
            p->long_cols, lp.chunk_off, lp.part, tb.dk, tb.dv, scale, static_cast<T*>(dK), static_cast<T*>(dV));
        GT_LAUNCH_CHECK("sparse_bwd_cols_long_merge");
    }
    return GT_OK;
}

template <typename T, int D, int H>
gt_status run_bwd_cols(const gt_tiles* p, const void* Q, const void* K, const void* V, const void* dO,
                       const float* LSE, const float* Dv, float scale, void* dK, void* dV, void* ws_ptr, EdgeBias eb,
                       hipStream_t s) {
    return eb.b ? run_bwd_cols_t<T, D, H, true>(p, Q, K, V, dO, LSE, Dv, scale, dK, dV, ws_ptr, eb, s)
                : run_bwd_cols_t<T, D, H, false>(p, Q, K, V, dO, LSE, Dv, scale, dK, dV, ws_ptr, eb, s);
}

template <typename T, int D, int H>
gt_status run_bwd(const gt_tiles* p, const void* Q, const void* K, const void* V, const void* dO, const float* LSE,
                  float scale, void* dQ, void* dK, void* dV, void* ws_ptr, EdgeBias eb, hipStream_t s) {
    if (p->n == 0) return GT_OK;
    Ws ws(ws_ptr);
    float* Dv = ws.take<float>(size_t(p->n) * H);
    char* rest = ws.take<char>(1);
    gt_status st = run_bwd_rows<T, D, H>(p, Q, K, V, dO, LSE, scale, dQ, Dv, rest, eb, s);
    if (st != GT_OK) return st;
    return run_bwd_cols<T, D, H>(p, Q, K, V, dO, LSE, Dv, scale, dK, dV, rest, eb, s);
}

bool supported(int32_t H, int32_t d, gt_dtype dt) {
    return (d == 32 || d == 64) && (H == 1 || H == 2 || H == 4 || H == 8 || H == 16) && (dt == GT_F32 || dt == GT_BF16);
}

gt_status check_plan(const char* who, const gt_tiles* p) {
    if (!p) return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null plan");
    if (p->n < 0 || p->n >= (int64_t(1) << 31) || (p->T != 64 && p->T != 128))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": plan not built (n or T invalid)");
    if (p->n > 0 && (!p->sp_rowptr || !p->sp_colptr || !p->tile_rowptr || !p->tileT_ptr))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": plan arrays missing");
    if ((p->nnz_sparse > 0 && (!p->sp_col || !p->sp_row)) || (p->n_long_rows > 0 && !p->long_rows) ||
        (p->n_long_cols > 0 && !p->long_cols) ||
        (p->n_dense > 0 && (!p->tile_col || !p->tile_mask || !p->tileT_idx)))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": plan arrays missing");
    return GT_OK;
}

size_t fwd_ws(const gt_tiles* p, int32_t H, int32_t d) {
    Ws ws(nullptr);
    ws.take<char>(256);
    tile_partials_fwd(ws, p, H, d);
    long_plan_take(ws, p->n_long_rows, p->nnz_sparse, int64_t(H) * d + 2 * H);
    return ws.size();
}
size_t bwd_part_ws(const gt_tiles* p, int32_t H, int32_t d, bool rows, bool cols) {
    Ws ws(nullptr);
    ws.take<char>(256);
    tile_partials_bwd(ws, p, H, d, rows, cols);
    if (rows) long_plan_take(ws, p->n_long_rows, p->nnz_sparse, 2 * int64_t(H) * d + H);
    if (cols) {
        long_plan_take(ws, p->n_long_cols, p->nnz_sparse, 2 * int64_t(H) * d);
        ws.take<float2>(size_t(p->n > 0 ? p->n : 1) * H);
    }
    return ws.size();
}
size_t bwd_ws(const gt_tiles* p, int32_t H, int32_t d) {
    Ws ws(nullptr);
    ws.take<float>(size_t(p->n > 0 ? p->n : 1) * H);
    const size_t a = bwd_part_ws(p, H, d, true, false), b = bwd_part_ws(p, H, d, false, true);
    ws.take<char>(a > b ? a : b);
    return ws.size();
}

}  // namespace
}  // namespace gt

using namespace gt;

extern "C" size_t gt_sparse_attn_fwd_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return fwd_ws(plan, H, d);
}

extern "C" gt_status gt_sparse_attn_fwd(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                                        const void* K, const void* V, float scale, void* O, float* LSE, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_fwd", plan);
    if (st != GT_OK) return st;
    if (!supported(H, d, dtype)) return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_fwd: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !O || !LSE || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_fwd: null pointer");
    if (ws_bytes < fwd_ws(plan, H, d)) return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_fwd: workspace too small");
    return GT_DISPATCH_ATTN(dtype, d, H, run_fwd, plan, Q, K, V, scale, O, LSE, ws, EdgeBias{}, stream);
}

extern "C" size_t gt_sparse_attn_bwd_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return bwd_ws(plan, H, d);
}

extern "C" size_t gt_sparse_attn_bwd_rows_workspace_size(const gt_tiles* plan, int32_t H, int32_t d,
                                                         gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return bwd_part_ws(plan, H, d, true, false);
}

extern "C" gt_status gt_sparse_attn_bwd_rows(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype,
                                             const void* Q, const void* K, const void* V, const void* dO,
                                             const float* LSE, float scale, void* dQ, float* Dstat, void* ws,
                                             size_t ws_bytes, hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_bwd_rows", plan);
    if (st != GT_OK) return st;
    if (!supported(H, d, dtype)) return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_bwd_rows: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !dO || !LSE || !dQ || !Dstat || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_bwd_rows: null pointer");
    if (ws_bytes < bwd_part_ws(plan, H, d, true, false))
        return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_bwd_rows: workspace too small");
    return GT_DISPATCH_ATTN(dtype, d, H, run_bwd_rows, plan, Q, K, V, dO, LSE, scale, dQ, Dstat, ws, EdgeBias{},
                            stream);
}

extern "C" size_t gt_sparse_attn_bwd_cols_workspace_size(const gt_tiles* plan, int32_t H, int32_t d,
                                                         gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return bwd_part_ws(plan, H, d, false, true);
}

extern "C" gt_status gt_sparse_attn_bwd_cols(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype,
                                             const void* Q, const void* K, const void* V, const void* dO,
                                             const float* LSE, const float* Dstat, float scale, void* dK, void* dV,
                                             void* ws, size_t ws_bytes, hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_bwd_cols", plan);
    if (st != GT_OK) return st;
    if (!supported(H, d, dtype)) return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_bwd_cols: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !dO || !LSE || !Dstat || !dK || !dV || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_bwd_cols: null pointer");
    if (ws_bytes < bwd_part_ws(plan, H, d, false, true))
        return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_bwd_cols: workspace too small");
    return GT_DISPATCH_ATTN(dtype, d, H, run_bwd_cols, plan, Q, K, V, dO, LSE, Dstat, scale, dK, dV, ws,
                            EdgeBias{}, stream);
}

extern "C" gt_status gt_sparse_attn_bwd(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                                        const void* K, const void* V, const void* dO, const float* LSE, float scale,
                                        void* dQ, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_bwd", plan);
    if (st != GT_OK) return st;
    if (!supported(H, d, dtype)) return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_bwd: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !dO || !LSE || !dQ || !dK || !dV || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_bwd: null pointer");
    if (ws_bytes < bwd_ws(plan, H, d)) return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_bwd: workspace too small");
    return GT_DISPATCH_ATTN(dtype, d, H, run_bwd, plan, Q, K, V, dO, LSE, scale, dQ, dK, dV, ws, EdgeBias{}, stream);
}

// ------------------------------------------------------------ with a bias
// The bias is indexed by input-CSR position.  Remainder edges read it through
// sp_pos (forward, row pass) or csc_pos (column pass).  On a plan with dense
// tiles it is first laid out per tile in the workspace (TileBias: the tile
// kernels read it with the same cell indexing as their masks), and the column
// pass's tile dS are written back to dbias at the tile edges' positions.

namespace gt {
namespace {

int64_t tile_bias_elems(const gt_tiles* p, int32_t H) {
    return p->n_dense > 0 ? p->n_dense * int64_t(H) * p->T * p->T : 0;
}

// The cells of local row r, word w (32 columns) of dense tile k: each thread
// takes one (r, w), whose first edge position is tile_pos[k T + r] plus the
// edges of the row's earlier words.  kToTiles: bias -> per-tile layout (-inf
// off the edges, so the tile kernels need no mask test where they add it);
// else per-tile dS -> dbias at the edges' positions.
template <bool kToTiles>
__global__ __launch_bounds__(256) void k_tile_bias_move(int H, int T, const uint32_t* __restrict__ mask,
                                                        const int32_t* __restrict__ tile_pos,
                                                        const float* __restrict__ src, float* __restrict__ dst) {
    const int64_t k = blockIdx.x;
    const int h = blockIdx.y;
    const int W = T / 32;
    for (int x = threadIdx.x; x < T * W; x += blockDim.x) {
        const int r = x / W, w = x % W;
        const uint32_t* row = mask + (k * T + r) * W;
        int pre = 0;
        for (int u = 0; u < w; ++u) pre += __popc(row[u]);
        const uint32_t word = row[w];
        const int64_t p0 = int64_t(tile_pos[k * T + r]) + pre;
        const int64_t cell = TileBias::at(k, H, h, T, r, 32 * w);
        for (int bit = 0; bit < 32; ++bit) {
            const bool on = (word >> bit) & 1u;
            const int64_t e = p0 + __popc(word & ((1u << bit) - 1u));
            if (kToTiles) dst[cell + bit] = on ? src[e * H + h] : -__builtin_huge_valf();
            else if (on) dst[e * H + h] = src[cell + bit];
        }
    }
}

gt_status tile_bias_move(bool to_tiles, const gt_tiles* p, int32_t H, const float* src, float* dst, hipStream_t s) {
    if (p->n_dense <= 0) return GT_OK;
    const dim3 grid(unsigned(p->n_dense), unsigned(H));
    if (to_tiles) k_tile_bias_move<true><<<grid, 256, 0, s>>>(H, p->T, p->tile_mask, p->tile_pos, src, dst);
    else k_tile_bias_move<false><<<grid, 256, 0, s>>>(H, p->T, p->tile_mask, p->tile_pos, src, dst);
    GT_LAUNCH_CHECK("tile_bias_move");
    return GT_OK;
}

gt_status check_bias(const char* who, const gt_tiles* plan, const float* bias) {
    if (plan->nnz_sparse >= (int64_t(1) << 31))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": more than 2^31 - 1 edges");
    if (plan->n_dense > 0 && ((plan->nnz_sparse > 0 && !plan->sp_pos) || !plan->tile_pos))
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": a plan with dense tiles needs sp_pos and tile_pos "
                                                            "(pass them to gt_build_tiles)");
    if ((plan->nnz_sparse > 0 || plan->n_dense > 0) && !bias)
        return fail(GT_ERR_INVALID_ARG, std::string(who) + ": null bias");
    return GT_OK;
}

size_t fwd_bias_ws(const gt_tiles* p, int32_t H, int32_t d) {
    Ws ws(nullptr);
    ws.take<char>(fwd_ws(p, H, d));
    ws.take<float>(size_t(tile_bias_elems(p, H)));
    return ws.size();
}
size_t bwd_bias_ws(const gt_tiles* p, int32_t H, int32_t d) {
    Ws ws(nullptr);
    ws.take<char>(bwd_ws(p, H, d));
    ws.take<float>(size_t(tile_bias_elems(p, H)));
    ws.take<float>(size_t(tile_bias_elems(p, H)));
    return ws.size();
}

}  // namespace
}  // namespace gt

extern "C" size_t gt_sparse_attn_fwd_bias_workspace_size(const gt_tiles* plan, int32_t H, int32_t d,
                                                         gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return fwd_bias_ws(plan, H, d);
}

extern "C" size_t gt_sparse_attn_bwd_bias_workspace_size(const gt_tiles* plan, int32_t H, int32_t d,
                                                         gt_dtype dtype) {
    if (!plan || !supported(H, d, dtype)) return 0;
    return bwd_bias_ws(plan, H, d);
}

extern "C" gt_status gt_sparse_attn_fwd_bias(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype,
                                             const void* Q, const void* K, const void* V, const float* bias,
                                             float scale, void* O, float* LSE, void* ws, size_t ws_bytes,
                                             hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_fwd_bias", plan);
    if (st != GT_OK) return st;
    if ((st = check_bias("gt_sparse_attn_fwd_bias", plan, bias)) != GT_OK) return st;
    if (!supported(H, d, dtype))
        return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_fwd_bias: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !O || !LSE || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_fwd_bias: null pointer");
    if (ws_bytes < fwd_bias_ws(plan, H, d))
        return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_fwd_bias: workspace too small");
    if (plan->n == 0) return GT_OK;
    Ws w(ws);
    void* main = w.take<char>(fwd_ws(plan, H, d));
    EdgeBias eb;
    if (plan->nnz_sparse > 0) {
        eb.b = bias;
        eb.sp_pos = plan->sp_pos;
    }
    if (plan->n_dense > 0) {
        float* bt = w.take<float>(size_t(tile_bias_elems(plan, H)));
        if ((st = tile_bias_move(true, plan, H, bias, bt, stream)) != GT_OK) return st;
        eb.tile.b = bt;
    }
    return GT_DISPATCH_ATTN(dtype, d, H, run_fwd, plan, Q, K, V, scale, O, LSE, main, eb, stream);
}

extern "C" gt_status gt_sparse_attn_bwd_bias(const gt_tiles* plan, const int32_t* csc_pos, int32_t H, int32_t d,
                                             gt_dtype dtype, const void* Q, const void* K, const void* V,
                                             const float* bias, const void* dO, const float* LSE, float scale,
                                             void* dQ, void* dK, void* dV, float* dbias, void* ws, size_t ws_bytes,
                                             hipStream_t stream) {
    gt_status st = check_plan("gt_sparse_attn_bwd_bias", plan);
    if (st != GT_OK) return st;
    if ((st = check_bias("gt_sparse_attn_bwd_bias", plan, bias)) != GT_OK) return st;
    if (!supported(H, d, dtype))
        return fail(GT_ERR_UNSUPPORTED, "gt_sparse_attn_bwd_bias: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!Q || !K || !V || !dO || !LSE || !dQ || !dK || !dV || !ws))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_bwd_bias: null pointer");
    if ((plan->nnz_sparse > 0 && !csc_pos) || ((plan->nnz_sparse > 0 || plan->n_dense > 0) && !dbias))
        return fail(GT_ERR_INVALID_ARG, "gt_sparse_attn_bwd_bias: null csc_pos or dbias");
    if (ws_bytes < bwd_bias_ws(plan, H, d))
        return fail(GT_ERR_WORKSPACE, "gt_sparse_attn_bwd_bias: workspace too small");
    if (plan->n == 0) return GT_OK;
    Ws w(ws);
    void* main = w.take<char>(bwd_ws(plan, H, d));
    EdgeBias eb;
    if (plan->nnz_sparse > 0) {
        eb.b = bias;
        eb.sp_pos = plan->sp_pos;
        eb.csc_pos = csc_pos;
        eb.db = dbias;
    }
    float* dbt = nullptr;
    if (plan->n_dense > 0) {
        float* bt = w.take<float>(size_t(tile_bias_elems(plan, H)));
        dbt = w.take<float>(size_t(tile_bias_elems(plan, H)));
        if ((st = tile_bias_move(true, plan, H, bias, bt, stream)) != GT_OK) return st;
        eb.tile.b = bt;
        eb.tile.db = dbt;
    }
    st = GT_DISPATCH_ATTN(dtype, d, H, run_bwd, plan, Q, K, V, dO, LSE, scale, dQ, dK, dV, main, eb, stream);
    if (st != GT_OK) return st;
    return dbt ? tile_bias_move(false, plan, H, dbt, dbias, stream) : GT_OK;
}

extern "C" gt_status gt_gather_probe(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* A,
                                     const void* B, uint32_t* sink, hipStream_t stream) {
    gt_status st = check_plan("gt_gather_probe", plan);
    if (st != GT_OK) return st;
    if (!supported(H, d, dtype)) return fail(GT_ERR_UNSUPPORTED, "gt_gather_probe: unsupported (H, d, dtype)");
    if (plan->n > 0 && (!A || !B || !sink)) return fail(GT_ERR_INVALID_ARG, "gt_gather_probe: null pointer");
    return GT_DISPATCH_ATTN(dtype, d, H, run_probe, plan, A, B, sink, stream);
}
