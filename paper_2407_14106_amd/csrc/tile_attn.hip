// Dense-tile attention on the matrix cores (§3.4: tiles of the reordered
// adjacency at or above the density threshold are computed whole, masked by
// the tile's bit mask, instead of edge by edge).
//
// Layout choices (CDNA4, wave64):
//   - 32x32 MFMA blocks; a workgroup owns one tile row (forward, dQ) or one
//     tile column (dK, dV) of T nodes, one wavefront per 32 of them.
//   - Scores are formed transposed (keys x queries for the row-owned kernels,
//     queries x keys for the column-owned one) so that every lane holds one
//     owned node and 16 of its partners: the softmax row statistics then need
//     one cross-lane exchange (between the two half-waves) per block.
//   - The probabilities stay in registers and feed the next product as its B
//     operand; the key order inside each 16-wide K step is permuted to match
//     the accumulator layout, and the A operand (V^T, K^T, Q^T, dO^T) is read
//     from an LDS copy transposed once per tile with the same permutation.
//   - bf16 inputs use v_mfma_f32_32x32x16_bf16 (probabilities rounded to bf16
//     for the second product); fp32 inputs use v_mfma_f32_32x32x2_f32.
// Each kernel leaves fp32 partial sums per (node, head); the edge kernels add
// the remainder edges and write the final results.
#include "tile_attn.h"

namespace gt {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kNegInf = -__builtin_huge_valf();

// Row (M index) of accumulator element i held by lane l: 8*(i/4) + 4*(l/32) + i%4.
__device__ __forceinline__ int crow(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16_t zero16() {
    f32x16_t z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// ---------------------------------------------------------------- operands

template <typename T>
struct Mma;

// bf16: K = 16 per instruction.  A[m][k] / B[k][n] operands hold 8 values:
// lane l covers m (or n) = l%32 and k = 8*(l/32) .. +7.
template <>
struct Mma<uint16_t> {
    static constexpr bool kBf16 = true;
    static constexpr int kStep = 16;
    using Op = bf16x8_t;
    // 8 consecutive elements of a row starting at 16*c + 8*(lane/32).
    __device__ static __forceinline__ Op row8(const uint16_t* row, int c, int lane) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + 16 * c + 8 * (lane >> 5));
        return __builtin_bit_cast(Op, v);
    }
    // Elements base+4*(l/32)+{0..3} and base+8+4*(l/32)+{0..3}: the K order of an
    // accumulator-layout B operand (see from_acc).
    __device__ static __forceinline__ Op perm8(const uint16_t* row, int base, int lane) {
        const int o = base + 4 * (lane >> 5);
        const uint2 a = *reinterpret_cast<const uint2*>(row + o);
        const uint2 b = *reinterpret_cast<const uint2*>(row + o + 8);
        return __builtin_bit_cast(Op, make_uint4(a.x, a.y, b.x, b.y));
    }
    // Accumulator elements 8*half .. 8*half+7 as a B operand (K = 16 rows of the block).
    __device__ static __forceinline__ Op from_acc(const f32x16_t& c, int half) {
        Op o;
#pragma unroll
        for (int t = 0; t < 8; ++t) o[t] = (__bf16)c[8 * half + t];
        return o;
    }
    __device__ static __forceinline__ f32x16_t mma(Op a, Op b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};

// fp32: K = 2 per instruction; lane l covers m (or n) = l%32 and k = l/32.
template <>
struct Mma<float> {
    static constexpr bool kBf16 = false;
    static constexpr int kStep = 2;
    __device__ static __forceinline__ f32x16_t mma(float a, float b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
};

// Register fragment of one owned node's row (d features) as the B operand of a
// product whose K dimension is d (e.g. S^T = K Q^T with Q owned).
template <typename T, int D>
struct RowFrag;

template <int D>
struct RowFrag<uint16_t, D> {
    bf16x8_t v[D / 16];
    __device__ __forceinline__ void load(const uint16_t* row, bool ok, int lane) {
#pragma unroll
        for (int c = 0; c < D / 16; ++c) {
            uint4 x = make_uint4(0, 0, 0, 0);
            if (ok) x = *reinterpret_cast<const uint4*>(row + 16 * c + 8 * (lane >> 5));
            v[c] = __builtin_bit_cast(bf16x8_t, x);
        }
    }
    // partial <this, other> over the lane's features
    __device__ __forceinline__ float dot(const RowFrag& o) const {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < D / 16; ++c)
#pragma unroll
            for (int t = 0; t < 8; ++t) s = fmaf(float(v[c][t]), float(o.v[c][t]), s);
        return s;
    }
};

template <int D>
struct RowFrag<float, D> {
    float v[D / 2];
    __device__ __forceinline__ void load(const float* row, bool ok, int lane) {
#pragma unroll
        for (int c = 0; c < D / 2; ++c) v[c] = ok ? row[2 * c + (lane >> 5)] : 0.f;
    }
    __device__ __forceinline__ float dot(const RowFrag& o) const {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < D / 2; ++c) s = fmaf(v[c], o.v[c], s);
        return s;
    }
};

// acc (32 partners x 32 owned) += A_rows (32 partner rows of a row-major LDS
// tile, d features) . frag^T : the "S^T = K Q^T" product, K dimension = d.
template <typename T, int D>
__device__ __forceinline__ f32x16_t prod_rows(const T* rows, int stride, const RowFrag<T, D>& f, int lane) {
    f32x16_t acc = zero16();
    const T* r = rows + (lane & 31) * stride;
    if constexpr (Mma<T>::kBf16) {
#pragma unroll
        for (int c = 0; c < D / 16; ++c) acc = Mma<T>::mma(Mma<T>::row8(r, c, lane), f.v[c], acc);
    } else {
#pragma unroll
        for (int c = 0; c < D / 2; ++c) acc = Mma<T>::mma(r[2 * c + (lane >> 5)], f.v[c], acc);
    }
    return acc;
}

// acc (32 features x 32 owned) += At_rows (transposed LDS tile: row = feature,
// columns = the block's 32 partners starting at col0) . P (accumulator layout,
// partners x owned): the "O^T = V^T P^T" product, K dimension = partners.
template <typename T>
__device__ __forceinline__ f32x16_t prod_acc(f32x16_t acc, const T* trow, int col0, const f32x16_t& p, int lane) {
    if constexpr (Mma<T>::kBf16) {
#pragma unroll
        for (int half = 0; half < 2; ++half)
            acc = Mma<T>::mma(Mma<T>::perm8(trow, col0 + 16 * half, lane), Mma<T>::from_acc(p, half), acc);
    } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) acc = Mma<T>::mma(trow[col0 + crow(i, lane)], p[i], acc);
    }
    return acc;
}

// As prod_acc, but the bf16 B operand is split into hi + lo parts (two
// products), so the weights keep about 16 mantissa bits: used where sums of
// many large weights meet (a hub attended by many low-degree rows) and where
// two such sums are subtracted (dQ = A - D B).
template <typename T>
__device__ __forceinline__ f32x16_t prod_acc_split(f32x16_t acc, const T* trow, int col0, const f32x16_t& p, int lane) {
    if constexpr (Mma<T>::kBf16) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const bf16x8_t a = Mma<T>::perm8(trow, col0 + 16 * half, lane);
            bf16x8_t hi, lo;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                hi[t] = (__bf16)p[8 * half + t];
                lo[t] = (__bf16)(p[8 * half + t] - float(hi[t]));
            }
            acc = Mma<T>::mma(a, hi, acc);
            acc = Mma<T>::mma(a, lo, acc);
        }
    } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) acc = Mma<T>::mma(trow[col0 + crow(i, lane)], p[i], acc);
    }
    return acc;
}

// ------------------------------------------------------------ LDS staging

template <typename T, int D>
struct Pad {
    static constexpr int kRow = D + 16 / int(sizeof(T));  // row-major tile row stride (elements)
};
template <typename T, int TT>
struct PadT {
    static constexpr int kRow = TT + 4 / int(sizeof(T)) * 2;  // transposed tile row stride (elements)
};

// Copy rows [base, base+TT) of X[:, h, :] into a row-major LDS tile (and, if
// `tr` is set, into a transposed tile tr[d][row]).  Rows >= n read as zero.
template <typename T, int D, int H, int TT, int NT>
__device__ __forceinline__ void stage(T* rm, T* tr, const T* __restrict__ X, int64_t base, int64_t n, int h) {
    constexpr int kPer = 16 / int(sizeof(T));  // elements per 16-byte chunk
    constexpr int kChunks = D / kPer;          // chunks per row
    for (int c = threadIdx.x; c < TT * kChunks; c += NT) {
        int r, part;
        if (tr) {  // consecutive threads take consecutive rows: conflict-free transposed writes
            r = c % TT;
            part = c / TT;
        } else {
            r = c / kChunks;
            part = c % kChunks;
        }
        const int64_t node = base + r;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (node < n) v = *reinterpret_cast<const uint4*>(X + (node * H + h) * D + part * kPer);
        if (rm) *reinterpret_cast<uint4*>(rm + r * Pad<T, D>::kRow + part * kPer) = v;
        if (tr) {
            const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
            for (int t = 0; t < kPer; ++t) tr[(part * kPer + t) * PadT<T, TT>::kRow + r] = e[t];
        }
    }
}

// Validity bits of the 32 partners of block (J, kb) when every pair is an
// edge (the full layer): all partners below n.
__device__ __forceinline__ uint32_t full_word(int64_t first, int64_t n) {
    const int64_t left = n - first;
    return left >= 32 ? 0xFFFFFFFFu : (left <= 0 ? 0u : ((1u << left) - 1u));
}

// ------------------------------------------------------------------ forward
// Grid (tile rows, heads).  kFull: every node attends to all n nodes (the
// interleaved full layer) and the kernel writes O and LSE; otherwise it walks
// the tile row's dense tiles and leaves (m, l, acc) partials.

template <typename T, int D, int H, int TT, bool kFull, bool kBias = false>
__global__ __launch_bounds__(2 * TT) void k_tile_fwd(int64_t n, const int64_t* __restrict__ tile_rowptr,
                                                      const int32_t* __restrict__ tile_col,
                                                      const uint32_t* __restrict__ tile_mask,
                                                      const T* __restrict__ Q, const T* __restrict__ K,
                                                      const T* __restrict__ V, float sl2, float* __restrict__ pm,
                                                      float* __restrict__ pl, float* __restrict__ pacc,
                                                      T* __restrict__ O, float* __restrict__ LSE, TileBias tb) {
    constexpr int NT = 2 * TT;  // threads: one wavefront per 32 rows
    constexpr int KB = TT / 32;
    constexpr int W = TT / 32;  // mask words per tile row
    __shared__ __attribute__((aligned(16))) T sK[TT * Pad<T, D>::kRow];
    __shared__ __attribute__((aligned(16))) T sVt[D * PadT<T, TT>::kRow];
    const int I = blockIdx.x;
    const int h = blockIdx.y;
    int64_t t0, t1;
    if (kFull) {
        t0 = 0;
        t1 = gridDim.x;
    } else {
        t0 = tile_rowptr[I];
        t1 = tile_rowptr[I + 1];
        if (t0 == t1) return;
    }
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int qlocal = 32 * wv + (lane & 31);
    const int64_t q = int64_t(I) * TT + qlocal;
    const bool qok = q < n;
    RowFrag<T, D> qf;
    qf.load(Q + (q * H + h) * D, qok, lane);
    float m = kNegInf, l = 0.f;
    f32x16_t acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) acc[db] = zero16();
    for (int64_t k = t0; k < t1; ++k) {
        const int64_t kbase = (kFull ? k : int64_t(tile_col[k])) * TT;
        __syncthreads();
        stage<T, D, H, TT, NT>(sK, nullptr, K, kbase, n, h);
        stage<T, D, H, TT, NT>(nullptr, sVt, V, kbase, n, h);
        __syncthreads();
        f32x16_t s[KB];
        float mloc = kNegInf;
        const uint32_t* mrow = tile_mask + (k * TT + qlocal) * W;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            s[kb] = prod_rows<T, D>(sK + 32 * kb * Pad<T, D>::kRow, Pad<T, D>::kRow, qf, lane);
            const uint32_t mw = kFull ? full_word(kbase + 32 * kb, n) : mrow[kb];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float v;
                if constexpr (kBias) {
                    // the per-tile bias is -inf off the edges, so it masks the cell itself: no test and
                    // no branch, which keeps the wait states of the accumulator reads that follow
                    v = fmaf(s[kb][i], sl2, tb.b[TileBias::at(k, H, h, TT, qlocal, 32 * kb + crow(i, lane))] * kLog2e);
                } else {
                    v = ((mw >> crow(i, lane)) & 1u) ? s[kb][i] * sl2 : kNegInf;
                }
                s[kb][i] = v;
                mloc = fmaxf(mloc, v);
            }
        }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, kWave));
        const float mnew = fmaxf(m, mloc);
        const float alpha = mnew == kNegInf ? 1.f : ex2(m - mnew);
        float lsum = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = s[kb][i] == kNegInf ? 0.f : ex2(s[kb][i] - mnew);
                s[kb][i] = p;
                lsum += p;
            }
        lsum += __shfl_xor(lsum, 32, kWave);
        l = l * alpha + lsum;
        m = mnew;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[db][i] *= alpha;
            const T* trow = sVt + (32 * db + (lane & 31)) * PadT<T, TT>::kRow;
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) acc[db] = prod_acc<T>(acc[db], trow, 32 * kb, s[kb], lane);
        }
    }
    if (!qok) return;
    if (kFull) {
        const float inv = l > 0.f ? 1.f / l : 0.f;
        if (lane < 32) LSE[q * H + h] = l > 0.f ? (m + __log2f(l)) * kLn2 : kNegInf;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float v = acc[db][i] * inv;
                const int64_t o = (q * H + h) * D + 32 * db + crow(i, lane);
                if constexpr (Mma<T>::kBf16)
                    O[o] = f32_to_bf16(v);
                else
                    O[o] = v;
            }
    } else {
        if (lane < 32) {
            pm[q * H + h] = m;
            pl[q * H + h] = l;
        }
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) pacc[(q * H + h) * D + 32 * db + crow(i, lane)] = acc[db][i];
    }
}

// ---------------------------------------------------------------- dQ (rows)
// Sparse tiles: dQ = scale (A - D B) with A = sum P dP K, B = sum P K and
// D = sum P dP over the row's partners (D equals <dO, O> of the exact output);
// the kernel leaves A, B and the D sum as partials, with the weights of both
// products split into bf16 hi + lo parts so that A - D B keeps its precision.
// Full layer (kFull): every weight is about 1/n, so D = <dO, O> from the given
// O is used directly and dQ = scale K^T (P (dP - D)) is finished here.

template <typename T, int D, int H, int TT, bool kFull, bool kBias = false>
__global__ __launch_bounds__(2 * TT) void k_tile_dq(int64_t n, const int64_t* __restrict__ tile_rowptr,
                                                     const int32_t* __restrict__ tile_col,
                                                     const uint32_t* __restrict__ tile_mask,
                                                     const T* __restrict__ Q, const T* __restrict__ K,
                                                     const T* __restrict__ V, const T* __restrict__ O,
                                                     const T* __restrict__ dO, const float* __restrict__ LSE,
                                                     float sl2, float* __restrict__ pa, float* __restrict__ pb,
                                                     float* __restrict__ pd, T* __restrict__ dQ,
                                                     float* __restrict__ Dv, float scale, TileBias tb) {
    constexpr int NT = 2 * TT;
    constexpr int KB = TT / 32;
    constexpr int W = TT / 32;
    __shared__ __attribute__((aligned(16))) T sK[TT * Pad<T, D>::kRow];
    __shared__ __attribute__((aligned(16))) T sV[TT * Pad<T, D>::kRow];
    __shared__ __attribute__((aligned(16))) T sKt[D * PadT<T, TT>::kRow];
    const int I = blockIdx.x;
    const int h = blockIdx.y;
    int64_t t0, t1;
    if (kFull) {
        t0 = 0;
        t1 = gridDim.x;
    } else {
        t0 = tile_rowptr[I];
        t1 = tile_rowptr[I + 1];
        if (t0 == t1) return;
    }
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int qlocal = 32 * wv + (lane & 31);
    const int64_t q = int64_t(I) * TT + qlocal;
    const bool qok = q < n;
    RowFrag<T, D> qf, gf;
    qf.load(Q + (q * H + h) * D, qok, lane);
    gf.load(dO + (q * H + h) * D, qok, lane);
    const float lse2 = qok ? LSE[q * H + h] * kLog2e : 0.f;
    float Dq = 0.f;
    if (kFull) {
        RowFrag<T, D> of;
        of.load(O + (q * H + h) * D, qok, lane);
        Dq = gf.dot(of);
        Dq += __shfl_xor(Dq, 32, kWave);
        if (qok && lane < 32) Dv[q * H + h] = Dq;
    }
    f32x16_t accA[D / 32], accB[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) accA[db] = accB[db] = zero16();
    float dsum = 0.f;
    for (int64_t k = t0; k < t1; ++k) {
        const int64_t kbase = (kFull ? k : int64_t(tile_col[k])) * TT;
        __syncthreads();
        stage<T, D, H, TT, NT>(sK, sKt, K, kbase, n, h);
        stage<T, D, H, TT, NT>(sV, nullptr, V, kbase, n, h);
        __syncthreads();
        const uint32_t* mrow = tile_mask + (k * TT + qlocal) * W;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            f32x16_t p = prod_rows<T, D>(sK + 32 * kb * Pad<T, D>::kRow, Pad<T, D>::kRow, qf, lane);
            f32x16_t w = prod_rows<T, D>(sV + 32 * kb * Pad<T, D>::kRow, Pad<T, D>::kRow, gf, lane);
            const uint32_t mw = kFull ? (qok ? full_word(kbase + 32 * kb, n) : 0u) : mrow[kb];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                float pv;
                if constexpr (kBias) {
                    const float bb = tb.b[TileBias::at(k, H, h, TT, qlocal, 32 * kb + crow(i, lane))];
                    pv = ex2(fmaf(p[i], sl2, bb * kLog2e) - lse2);  // 0 off the edges (bias -inf)
                } else {
                    pv = ((mw >> crow(i, lane)) & 1u) ? ex2(p[i] * sl2 - lse2) : 0.f;
                }
                p[i] = pv;
                if (kFull) {
                    w[i] = pv * (w[i] - Dq);
                } else {
                    w[i] *= pv;
                    dsum += w[i];
                }
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db) {
                const T* trow = sKt + (32 * db + (lane & 31)) * PadT<T, TT>::kRow;
                if (kFull) {
                    accA[db] = prod_acc<T>(accA[db], trow, 32 * kb, w, lane);
                } else {
                    accA[db] = prod_acc_split<T>(accA[db], trow, 32 * kb, w, lane);
                    accB[db] = prod_acc_split<T>(accB[db], trow, 32 * kb, p, lane);
                }
            }
        }
    }
    dsum += __shfl_xor(dsum, 32, kWave);
    if (!qok) return;
    if (!kFull && lane < 32) pd[q * H + h] = dsum;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int64_t o = (q * H + h) * D + 32 * db + crow(i, lane);
            if (kFull) {
                const float v = accA[db][i] * scale;
                if constexpr (Mma<T>::kBf16)
                    dQ[o] = f32_to_bf16(v);
                else
                    dQ[o] = v;
            } else {
                pa[o] = accA[db][i];
                pb[o] = accB[db][i];
            }
        }
}

// ----------------------------------------------------------- dK, dV (cols)

template <typename T, int D, int H, int TT, bool kFull, bool kSplit, bool kBias = false>
__global__ __launch_bounds__(2 * TT) void k_tile_dkdv(int64_t n, const int64_t* __restrict__ tileT_ptr,
                                                       const int32_t* __restrict__ tileT_idx,
                                                       const int64_t* __restrict__ tile_rowptr,
                                                       const uint32_t* __restrict__ tile_mask,
                                                       const T* __restrict__ Q, const T* __restrict__ K,
                                                       const T* __restrict__ V, const T* __restrict__ dO,
                                                       const float* __restrict__ LSE, const float* __restrict__ Dv,
                                                       float sl2, float* __restrict__ pdk, float* __restrict__ pdv,
                                                       T* __restrict__ dK, T* __restrict__ dV, float scale,
                                                       TileBias tb) {
    constexpr int NT = 2 * TT;
    constexpr int QB = TT / 32;
    constexpr int W = TT / 32;
    __shared__ __attribute__((aligned(16))) T sQ[TT * Pad<T, D>::kRow];
    __shared__ __attribute__((aligned(16))) T sG[TT * Pad<T, D>::kRow];
    __shared__ __attribute__((aligned(16))) T sQt[D * PadT<T, TT>::kRow];
    __shared__ __attribute__((aligned(16))) T sGt[D * PadT<T, TT>::kRow];
    __shared__ float sL[TT];
    __shared__ float sD[TT];
    __shared__ uint32_t sM[kFull ? 1 : TT * W];
    const int J = blockIdx.x;
    const int h = blockIdx.y;
    int64_t u0, u1;
    if (kFull) {
        u0 = 0;
        u1 = gridDim.x;
    } else {
        u0 = tileT_ptr[J];
        u1 = tileT_ptr[J + 1];
        if (u0 == u1) return;
    }
    const int lane = lane_id();
    const int wv = threadIdx.x / kWave;
    const int klocal = 32 * wv + (lane & 31);
    const int64_t key = int64_t(J) * TT + klocal;
    const bool kok = key < n;
    RowFrag<T, D> kf, vf;
    kf.load(K + (key * H + h) * D, kok, lane);
    vf.load(V + (key * H + h) * D, kok, lane);
    f32x16_t dk[D / 32], dv[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db) dk[db] = dv[db] = zero16();
    for (int64_t u = u0; u < u1; ++u) {
        int64_t I, k = 0;
        if (kFull) {
            I = u;
        } else {
            k = tileT_idx[u];
            // tile row of tile k: the last I with tile_rowptr[I] <= k
            int64_t lo = 0, hi = int64_t(gridDim.x);
            while (hi - lo > 1) {
                const int64_t mid = (lo + hi) >> 1;
                if (tile_rowptr[mid] <= k) lo = mid;
                else hi = mid;
            }
            I = lo;
        }
        const int64_t qbase = I * TT;
        __syncthreads();
        stage<T, D, H, TT, NT>(sQ, sQt, Q, qbase, n, h);
        stage<T, D, H, TT, NT>(sG, sGt, dO, qbase, n, h);
        for (int r = threadIdx.x; r < TT; r += NT) {
            const int64_t qn = qbase + r;
            sL[r] = qn < n ? LSE[qn * H + h] * kLog2e : 0.f;
            sD[r] = qn < n ? Dv[qn * H + h] : 0.f;
        }
        if (!kFull)
            for (int w = threadIdx.x; w < TT * W; w += NT) sM[w] = tile_mask[k * TT * W + w];
        __syncthreads();
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            f32x16_t s = prod_rows<T, D>(sQ + 32 * qb * Pad<T, D>::kRow, Pad<T, D>::kRow, kf, lane);
            const f32x16_t dp = prod_rows<T, D>(sG + 32 * qb * Pad<T, D>::kRow, Pad<T, D>::kRow, vf, lane);
            f32x16_t p;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = 32 * qb + crow(i, lane);
                const bool on = kFull ? (qbase + r < n) : ((sM[r * W + wv] >> (lane & 31)) & 1u);
                float pv;
                if constexpr (kBias) {
                    const int64_t x = TileBias::at(k, H, h, TT, r, klocal);
                    pv = ex2(fmaf(s[i], sl2, tb.b[x] * kLog2e) - sL[r]);  // 0 off the edges (bias -inf)
                    s[i] = pv * (dp[i] - sD[r]);
                    tb.db[x] = s[i];  // every cell (0 off the edges), so no branch is needed
                } else {
                    pv = on ? ex2(s[i] * sl2 - sL[r]) : 0.f;
                    s[i] = pv * (dp[i] - sD[r]);
                }
                p[i] = pv;
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db) {
                const T* grow = sGt + (32 * db + (lane & 31)) * PadT<T, TT>::kRow;
                const T* qrow = sQt + (32 * db + (lane & 31)) * PadT<T, TT>::kRow;
                if (kSplit) {
                    dv[db] = prod_acc_split<T>(dv[db], grow, 32 * qb, p, lane);
                    dk[db] = prod_acc_split<T>(dk[db], qrow, 32 * qb, s, lane);
                } else {
                    dv[db] = prod_acc<T>(dv[db], grow, 32 * qb, p, lane);
                    dk[db] = prod_acc<T>(dk[db], qrow, 32 * qb, s, lane);
                }
            }
        }
    }
    if (!kok) return;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int64_t o = (key * H + h) * D + 32 * db + crow(i, lane);
            if (kFull) {
                if constexpr (Mma<T>::kBf16) {
                    dK[o] = f32_to_bf16(dk[db][i] * scale);
                    dV[o] = f32_to_bf16(dv[db][i]);
                } else {
                    dK[o] = dk[db][i] * scale;
                    dV[o] = dv[db][i];
                }
            } else {
                pdk[o] = dk[db][i];
                pdv[o] = dv[db][i];
            }
        }
}

}  // namespace

// ---------------------------------------------------------------- launchers

#define GT_TILE_SWITCH(T_, CALL)                                                 \
    do {                                                                         \
        if ((T_) == 128) {                                                       \
            constexpr int TT = 128;                                              \
            CALL;                                                                \
        } else if ((T_) == 64) {                                                 \
            constexpr int TT = 64;                                               \
            CALL;                                                                \
        } else {                                                                 \
            return fail(GT_ERR_UNSUPPORTED, "dense tiles: T must be 64 or 128"); \
        }                                                                        \
    } while (0)

template <typename T, int D, int H>
gt_status tile_fwd(const gt_tiles* p, const T* Q, const T* K, const T* V, float sl2, TilePartials tp, TileBias tb,
                   hipStream_t s) {
    if constexpr (Mma<T>::kBf16) return tiles_fwd_bf16<D>(p, H, Q, K, V, sl2, tp, tb, s);
    const dim3 grid(unsigned(p->n_row_tiles), H);
    if (tb.b)
        GT_TILE_SWITCH(p->T, (k_tile_fwd<T, D, H, TT, false, true><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, sl2, tp.m, tp.l, tp.acc,
                                 nullptr, nullptr, tb)));
    else
        GT_TILE_SWITCH(p->T, (k_tile_fwd<T, D, H, TT, false><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, sl2, tp.m, tp.l, tp.acc,
                                 nullptr, nullptr, tb)));
    GT_LAUNCH_CHECK("tile_fwd");
    return GT_OK;
}

template <typename T, int D, int H>
gt_status tile_bwd_dq(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                      float sl2, TilePartials dq, TileBias tb, hipStream_t s) {
    if constexpr (Mma<T>::kBf16) return tiles_dq_bf16<D>(p, H, Q, K, V, dO, LSE, sl2, dq, tb, s);
    const dim3 grid(unsigned(p->n_row_tiles), H);
    if (tb.b)
        GT_TILE_SWITCH(p->T, (k_tile_dq<T, D, H, TT, false, true><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, nullptr, dO, LSE, sl2,
                                 dq.acc, dq.acc2, dq.m, nullptr, nullptr, 1.f, tb)));
    else
        GT_TILE_SWITCH(p->T, (k_tile_dq<T, D, H, TT, false><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, nullptr, dO, LSE, sl2,
                                 dq.acc, dq.acc2, dq.m, nullptr, nullptr, 1.f, tb)));
    GT_LAUNCH_CHECK("tile_bwd_dq");
    return GT_OK;
}

template <typename T, int D, int H>
gt_status tile_bwd_dkdv(const gt_tiles* p, const T* Q, const T* K, const T* V, const T* dO, const float* LSE,
                        const float* Dv, float sl2, TilePartials dk, TilePartials dv, TileBias tb, hipStream_t s) {
    if constexpr (Mma<T>::kBf16) return tiles_dkdv_bf16<D>(p, H, Q, K, V, dO, LSE, Dv, sl2, dk, dv, tb, s);
    const dim3 grid(unsigned(p->n_row_tiles), H);
    if (tb.b)
        GT_TILE_SWITCH(p->T, (k_tile_dkdv<T, D, H, TT, false, true, true><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tileT_ptr, p->tileT_idx, p->tile_rowptr, p->tile_mask, Q, K, V, dO, LSE,
                                 Dv, sl2, dk.acc, dv.acc, nullptr, nullptr, 1.f, tb)));
    else
        GT_TILE_SWITCH(p->T, (k_tile_dkdv<T, D, H, TT, false, true><<<grid, 2 * TT, 0, s>>>(
                                 p->n, p->tileT_ptr, p->tileT_idx, p->tile_rowptr, p->tile_mask, Q, K, V, dO, LSE,
                                 Dv, sl2, dk.acc, dv.acc, nullptr, nullptr, 1.f, tb)));
    GT_LAUNCH_CHECK("tile_bwd_dkdv");
    return GT_OK;
}

// The full layer: 128-node blocks, every pair attended.
template <typename T, int D, int H>
gt_status full_fwd(int64_t n, const T* Q, const T* K, const T* V, float sl2, T* O, float* LSE, hipStream_t s) {
    constexpr int TT = 128;
    const dim3 grid(unsigned(cdiv(n, TT)), H);
    k_tile_fwd<T, D, H, TT, true><<<grid, 2 * TT, 0, s>>>(n, nullptr, nullptr, nullptr, Q, K, V, sl2, nullptr,
                                                          nullptr, nullptr, O, LSE, TileBias{});
    GT_LAUNCH_CHECK("full_fwd");
    return GT_OK;
}

template <typename T, int D, int H>
gt_status full_bwd(int64_t n, const T* Q, const T* K, const T* V, const T* O, const T* dO, const float* LSE,
                   float sl2, float scale, T* dQ, T* dK, T* dV, float* Dv, hipStream_t s) {
    constexpr int TT = 128;
    const dim3 grid(unsigned(cdiv(n, TT)), H);
    k_tile_dq<T, D, H, TT, true><<<grid, 2 * TT, 0, s>>>(n, nullptr, nullptr, nullptr, Q, K, V, O, dO, LSE, sl2,
                                                         nullptr, nullptr, nullptr, dQ, Dv, scale, TileBias{});
    GT_LAUNCH_CHECK("full_bwd_dq");
    k_tile_dkdv<T, D, H, TT, true, false><<<grid, 2 * TT, 0, s>>>(n, nullptr, nullptr, nullptr, nullptr, Q, K, V,
                                                                  dO, LSE, Dv, sl2, nullptr, nullptr, dK, dV, scale,
                                                                  TileBias{});
    GT_LAUNCH_CHECK("full_bwd_dkdv");
    return GT_OK;
}

#define GT_INST(T, D, H)                                                                                          \
    template gt_status tile_fwd<T, D, H>(const gt_tiles*, const T*, const T*, const T*, float, TilePartials,      \
                                         TileBias, hipStream_t);                                                  \
    template gt_status tile_bwd_dq<T, D, H>(const gt_tiles*, const T*, const T*, const T*, const T*,              \
                                            const float*, float, TilePartials, TileBias, hipStream_t);            \
    template gt_status tile_bwd_dkdv<T, D, H>(const gt_tiles*, const T*, const T*, const T*, const T*,            \
                                              const float*, const float*, float, TilePartials, TilePartials,      \
                                              TileBias, hipStream_t);                                             \
    template gt_status full_fwd<T, D, H>(int64_t, const T*, const T*, const T*, float, T*, float*, hipStream_t); \
    template gt_status full_bwd<T, D, H>(int64_t, const T*, const T*, const T*, const T*, const T*, const float*, \
                                         float, float, T*, T*, T*, float*, hipStream_t);
#define GT_INST_H(T, D) GT_INST(T, D, 1) GT_INST(T, D, 2) GT_INST(T, D, 4) GT_INST(T, D, 8) GT_INST(T, D, 16)
GT_INST_H(uint16_t, 32)
GT_INST_H(uint16_t, 64)
GT_INST_H(float, 32)
GT_INST_H(float, 64)

}  // namespace gt
