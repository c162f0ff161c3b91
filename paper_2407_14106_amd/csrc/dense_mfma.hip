// Full softmax attention for bf16 features on the matrix cores: the
// interleaved fully-connected layer of §3.2 (every node attends to every node,
// Eq. (1) of §2.1), forward and backward, streaming over the keys with no
// n x n buffer.
//
// Design (CDNA4, wave64, v_mfma_f32_32x32x16_bf16):
//   - A workgroup owns 256 rows of one head.  In the forward each wavefront
//     owns 64 of them (two 32-row MFMA blocks), so every operand fragment read
//     from LDS feeds two products; the backward passes give each wavefront one
//     block (8 wavefronts), which halves their registers and leaves 2-3
//     wavefronts per SIMD.  The partner rows stream through LDS in 64-row stages,
//     double buffered: the next stage is loaded into registers while the
//     current one is multiplied, then written to the other buffer, with one
//     barrier per stage.
//   - Scores are formed transposed (partners x owned rows), so each lane holds
//     one owned row and 16 of its partners; per-row statistics need one
//     v_permlane32_swap between the half-waves.  The probabilities (or dS)
//     become the next product's B operand straight from the accumulators; the
//     A operand of that product (V^T, K^T, dO^T, Q^T) is read from a
//     transposed LDS copy written as 4-partner x 4-feature blocks.
//   - The forward's running maximum is lazy: the accumulators are rescaled
//     only when some row's block maximum exceeds it by 2^8 (exp2 domain), so
//     weights stay below 256 and the result is unchanged.
//   - D_i = <dO_i, O_i> from the given O: every full-layer weight is O(1/n),
//     so no cancellation-prone sum over partners is needed.
//   - Workgroups are remapped so that each XCD works on one range of
//     (head, row block) pairs and shares that head's K and V in its L2.
#include "tile_attn.h"

namespace gt {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kRowsWg = 256;             // owned rows per workgroup of the full layer
constexpr int kStage = 64;               // partner rows per LDS stage
constexpr int kTS = kStage + 4;          // transposed LDS row stride (elements)
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLazy = 8.f;             // lazy-max slack, exp2 domain

template <int D>
struct RS {
    static constexpr int v = D + 8;  // row-major LDS row stride (elements)
};

__device__ __forceinline__ int crow(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// A compile-time flag passed as a value (generic lambdas take it as auto).
template <bool B>
struct Flag {
    static constexpr bool value = B;
};
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x16_t zero16() {
    f32x16_t z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

__device__ __forceinline__ f32x16_t mma(bf16x8_t a, bf16x8_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The value of x held by the partner lane (lane ^ 32) combined with x.
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// A operand from a row-major LDS tile: row r, features 16c + 8(lane/32) .. +7.
template <int D>
__device__ __forceinline__ bf16x8_t lds_row8(const uint16_t* s, int r, int c, int lane) {
    return __builtin_bit_cast(bf16x8_t,
                              *reinterpret_cast<const uint4*>(s + r * RS<D>::v + 16 * c + 8 * (lane >> 5)));
}
// A operand from a transposed LDS tile (row = feature f): partners
// base + 4(lane/32) + {0..3} and base + 8 + 4(lane/32) + {0..3}, the partner
// order of an accumulator-layout B operand (acc_b16).
__device__ __forceinline__ bf16x8_t lds_perm8(const uint16_t* s, int f, int base, int lane) {
    const uint16_t* p = s + f * kTS + base + 4 * (lane >> 5);
    const uint2 a = *reinterpret_cast<const uint2*>(p);
    const uint2 b = *reinterpret_cast<const uint2*>(p + 8);
    return __builtin_bit_cast(bf16x8_t, make_uint4(a.x, a.y, b.x, b.y));
}
// Accumulator elements 8*half .. +7 as a bf16 B operand.
__device__ __forceinline__ bf16x8_t acc_b16(const f32x16_t& c, int half) {
    bf16x8_t o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = (__bf16)c[8 * half + t];
    return o;
}

// B operand fragments of one owned row (global memory): features
// 16c + 8(lane/32) .. +7 for c < D/16; zero for rows >= n.
template <int D>
struct Frag {
    bf16x8_t v[D / 16];
    __device__ __forceinline__ void load(const uint16_t* X, int64_t row, int64_t n, int H, int h, int lane) {
        const int64_t src = row < n ? row : n - 1;
#pragma unroll
        for (int c = 0; c < D / 16; ++c) {
            uint4 x = *reinterpret_cast<const uint4*>(X + (src * H + h) * D + 16 * c + 8 * (lane >> 5));
            if (row >= n) x = make_uint4(0, 0, 0, 0);
            v[c] = __builtin_bit_cast(bf16x8_t, x);
        }
    }
    // this lane's share of <this, o>
    __device__ __forceinline__ float dot(const Frag& o) const {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < D / 16; ++c)
#pragma unroll
            for (int t = 0; t < 8; ++t) s = fmaf(float(v[c][t]), float(o.v[c][t]), s);
        return s;
    }
};

// One thread's share of a 64-row stage of X[:, h, :] for a workgroup of NT
// threads: blocks of 4 rows x 4 features (8 bytes per row), kept in registers
// between the global load and the LDS stores.  Loads are unconditional (rows
// past n read row n-1) so the compiler can keep them in flight across the
// stage's products; rows >= n are zeroed when stored.
template <int D, int NT>
struct Stager {
    static constexpr int FG = D / 4;                        // feature groups per row
    static constexpr int kItems = 16 * FG;                  // (row group, feature group) blocks
    static constexpr int PER = kItems >= NT ? kItems / NT : 1;
    static_assert(kItems >= NT ? kItems % NT == 0 : NT % kItems == 0, "stage does not fit the workgroup");
    uint2 r[PER][4];
    uint32_t valid;  // bit 4k + j: row j of block k is below n
    // Threads beyond kItems (whole wavefronts) only mirror the loads.
    __device__ __forceinline__ static bool on() { return kItems >= NT || threadIdx.x < kItems; }
    __device__ __forceinline__ static int item(int k) {
        return kItems >= NT ? int(threadIdx.x) + k * NT : int(threadIdx.x) % kItems;
    }
    __device__ __forceinline__ void load(const uint16_t* __restrict__ X, int64_t base, int64_t n, int H, int h) {
        valid = 0;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it = item(k), rg = it / FG, fg = it % FG;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t node = base + 4 * rg + j;
                const int64_t src = node < n ? node : n - 1;
                valid |= uint32_t(node < n) << (4 * k + j);
                r[k][j] = *reinterpret_cast<const uint2*>(X + (src * H + h) * D + 4 * fg);
            }
        }
    }
    // A stage whose 64 rows are all below n: one uniform base address, per-lane
    // 32-bit offsets that do not change from stage to stage, no clamping.
    __device__ __forceinline__ void load_in(const uint16_t* __restrict__ X, int64_t base, int H, int h) {
        const uint16_t* xb = X + (base * H + h) * D;
        const int rs = H * D;
        valid = ~0u;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it = item(k), rg = it / FG, fg = it % FG;
            const uint16_t* p = xb + 4 * rg * rs + 4 * fg;
#pragma unroll
            for (int j = 0; j < 4; ++j) r[k][j] = *reinterpret_cast<const uint2*>(p + j * rs);
        }
    }
    // Either form, by where the stage ends.
    __device__ __forceinline__ void load_any(const uint16_t* __restrict__ X, int64_t base, int64_t n, int H, int h) {
        if (base + kStage <= n) load_in(X, base, H, h);
        else load(X, base, n, H, h);
    }
    __device__ __forceinline__ uint2 row(int k, int j) const {
        return (valid >> (4 * k + j)) & 1u ? r[k][j] : make_uint2(0, 0);
    }
    __device__ __forceinline__ void store_rm(uint16_t* s) const {
        if (!on()) return;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it = item(k), rg = it / FG, fg = it % FG;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                *reinterpret_cast<uint2*>(s + (4 * rg + j) * RS<D>::v + 4 * fg) = row(k, j);
        }
    }
    // s[f * kTS + row]: the 4 rows of each of the 4 features as one 8-byte store.
    __device__ __forceinline__ void store_tr(uint16_t* s) const {
        if (!on()) return;
        const uint32_t lo = 0xFFFFu, hi = 0xFFFF0000u;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int it = item(k), rg = it / FG, fg = it % FG;
            const uint2 a = row(k, 0), b = row(k, 1), c = row(k, 2), d = row(k, 3);
            uint16_t* p = s + (4 * fg) * kTS + 4 * rg;
            *reinterpret_cast<uint2*>(p) = make_uint2((a.x & lo) | (b.x << 16), (c.x & lo) | (d.x << 16));
            *reinterpret_cast<uint2*>(p + kTS) = make_uint2((a.x >> 16) | (b.x & hi), (c.x >> 16) | (d.x & hi));
            *reinterpret_cast<uint2*>(p + 2 * kTS) = make_uint2((a.y & lo) | (b.y << 16), (c.y & lo) | (d.y << 16));
            *reinterpret_cast<uint2*>(p + 3 * kTS) = make_uint2((a.y >> 16) | (b.y & hi), (c.y >> 16) | (d.y & hi));
        }
    }
};

// All outstanding memory operations of this wavefront are complete (so the
// compiler's wait counting starts the streaming loop from a clean state).
__device__ __forceinline__ void drain() { __builtin_amdgcn_s_waitcnt(0); }

// Workgroup -> (head, first owned row); false for the padding of the grid.
__device__ __forceinline__ bool wg_coords(int64_t n, int H, int& h, int64_t& row0) {
    const int64_t blocks = cdiv(n, kRowsWg);
    const int64_t b = xcd_block(blockIdx.x, gridDim.x);
    if (b >= blocks * H) return false;
    h = int(b / blocks);
    row0 = (b % blocks) * kRowsWg;
    return true;
}

inline unsigned full_grid(int64_t n, int H) { return xcd_grid(cdiv(n, kRowsWg) * H); }

// 32-row MFMA blocks per wavefront in the full layer (the kernels are
// templated on it) and the threads per workgroup that hold kRowsWg rows.  The
// forward keeps two blocks (every K and V fragment read from LDS feeds two
// products; measured faster: 10.9 against 13.7 ms at 65,536 x 8 x 64); the
// backward passes take one, which leaves them 2-3 wavefronts per SIMD instead
// of one (44.1 -> 35.3 ms).
constexpr int kFullFwdNB = 2, kFullBwdNB = 1;
constexpr int kFullFwdThr = kRowsWg / (32 * kFullFwdNB) * kWave;
constexpr int kFullBwdThr = kRowsWg / (32 * kFullBwdNB) * kWave;

// ------------------------------------------------------------------ forward

template <int D, int NB>
__global__ __launch_bounds__(kRowsWg / (32 * NB) * kWave) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 3 : 2))) void k_full_fwd(int64_t n, int H, const uint16_t* __restrict__ Q,
                                                      const uint16_t* __restrict__ K,
                                                      const uint16_t* __restrict__ V, float sl2,
                                                      uint16_t* __restrict__ O, float* __restrict__ LSE) {
    __shared__ __attribute__((aligned(16))) uint16_t sK[2][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sVt[2][D * kTS];
    int h;
    int64_t row0;
    if (!wg_coords(n, H, h, row0)) return;
    const int lane = lane_id();
    const int64_t q0 = row0 + (threadIdx.x / kWave) * 32 * NB;
    Frag<D> qf[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) qf[b].load(Q, q0 + 32 * b + (lane & 31), n, H, h, lane);
    if (sl2 < 0.f) {  // keep the exp2-domain scale positive: negate Q instead (exact in bf16)
        sl2 = -sl2;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int c = 0; c < D / 16; ++c)
                qf[b].v[c] = __builtin_bit_cast(bf16x8_t, __builtin_bit_cast(uint4, qf[b].v[c]) ^
                                                              make_uint4(0x80008000u, 0x80008000u, 0x80008000u,
                                                                         0x80008000u));
    }
    f32x16_t acc[NB][D / 32];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) acc[b][db] = zero16();
    float m[NB], l[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        m[b] = kNegInf;
        l[b] = 0.f;
    }

    Stager<D, kRowsWg / (32 * NB) * kWave> gk, gv;
    gk.load(K, 0, n, H, h);
    gv.load(V, 0, n, H, h);
    gk.store_rm(sK[0]);
    gv.store_tr(sVt[0]);
    drain();
    __syncthreads();
    const int64_t stages = cdiv(n, kStage);
    for (int64_t t = 0; t < stages; ++t) {
        const int buf = int(t & 1);
        const int64_t kbase = t * kStage;
        if (t + 1 < stages) {
            gk.load_any(K, kbase + kStage, n, H, h);
            gv.load_any(V, kbase + kStage, n, H, h);
        }
        const uint16_t* k_s = sK[buf];
        const uint16_t* v_s = sVt[buf];
#pragma unroll
        for (int kb = 0; kb < kStage / 32; ++kb) {
            f32x16_t s[NB];
            #pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(k_s, 32 * kb + (lane & 31), c, lane);
                #pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, qf[b].v[c], s[b]);
            }
            const int64_t key0 = kbase + 32 * kb;
            if (__builtin_expect(key0 + 32 > n, 0)) {  // ragged last block: partners >= n take no weight
                // kept as a branch (the empty asm stops the compiler from turning
                // it into selects on every block)
                asm volatile("" ::: "memory");
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (key0 + crow(i, lane) >= n)
#pragma unroll
                        for (int b = 0; b < NB; ++b) s[b][i] = kNegInf;
            }
            bool grow = false;
            float mt[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                float mx = s[b][0];
#pragma unroll
                for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s[b][i]);
                mt[b] = pair_max(mx) * sl2;
                grow |= mt[b] > m[b] + kLazy;
            }
            if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const float mn = fmaxf(m[b], mt[b]);
                    const float alpha = ex2(m[b] - mn);
                    l[b] *= alpha;
#pragma unroll
                    for (int db = 0; db < D / 32; ++db)
#pragma unroll
                        for (int i = 0; i < 16; ++i) acc[b][db][i] *= alpha;
                    m[b] = mn;
                }
            }
            bf16x8_t pb[NB][2];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                float ls = 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = ex2(fmaf(s[b][i], sl2, -m[b]));
                    s[b][i] = p;
                    ls += p;
                }
                l[b] += ls;
                pb[b][0] = acc_b16(s[b], 0);
                pb[b][1] = acc_b16(s[b], 1);
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t a = lds_perm8(v_s, 32 * db + (lane & 31), 32 * kb + 16 * half, lane);
                    #pragma unroll
                    for (int b = 0; b < NB; ++b) acc[b][db] = mma(a, pb[b][half], acc[b][db]);
                }
        }
        if (t + 1 < stages) {
            gk.store_rm(sK[buf ^ 1]);
            gv.store_tr(sVt[buf ^ 1]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        const float lt = pair_sum(l[b]);
        if (q >= n) continue;
        const float inv = lt > 0.f ? 1.f / lt : 0.f;
        if (lane < 32) LSE[q * H + h] = lt > 0.f ? (m[b] + __log2f(lt)) * kLn2 : kNegInf;
        uint16_t* o = O + (q * H + h) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x16_t& a = acc[b][db];
                *reinterpret_cast<uint2*>(o + 32 * db + 8 * j + 4 * (lane >> 5)) =
                    make_uint2(pack_bf16x2(a[4 * j] * inv, a[4 * j + 1] * inv),
                               pack_bf16x2(a[4 * j + 2] * inv, a[4 * j + 3] * inv));
            }
    }
}

// ---------------------------------------------------------------- dQ (rows)
// dQ_i = scale sum_j P_ij (dP_ij - D_i) K_j with dP_ij = <dO_i, V_j>; also
// writes D_i for the column pass.

template <int D, int NB>
__global__ __launch_bounds__(kRowsWg / (32 * NB) * kWave) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 2 : 1))) void k_full_dq(int64_t n, int H, const uint16_t* __restrict__ Q,
                                                     const uint16_t* __restrict__ K,
                                                     const uint16_t* __restrict__ V,
                                                     const uint16_t* __restrict__ O,
                                                     const uint16_t* __restrict__ dO,
                                                     const float* __restrict__ LSE, float sl2, float scale,
                                                     uint16_t* __restrict__ dQ, float* __restrict__ Dv) {
    __shared__ __attribute__((aligned(16))) uint16_t sK[2][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sV[2][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sKt[2][D * kTS];
    int h;
    int64_t row0;
    if (!wg_coords(n, H, h, row0)) return;
    const int lane = lane_id();
    const int64_t q0 = row0 + (threadIdx.x / kWave) * 32 * NB;
    Frag<D> qf[NB], gf[NB];
    float lse2[NB], Dq[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        qf[b].load(Q, q, n, H, h, lane);
        gf[b].load(dO, q, n, H, h, lane);
        Frag<D> of;
        of.load(O, q, n, H, h, lane);
        Dq[b] = pair_sum(gf[b].dot(of));
        lse2[b] = q < n ? LSE[q * H + h] * kLog2e : 0.f;
        if (q < n && lane < 32) Dv[q * H + h] = Dq[b];
    }
    f32x16_t acc[NB][D / 32];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) acc[b][db] = zero16();

    Stager<D, kRowsWg / (32 * NB) * kWave> gk, gv;
    gk.load(K, 0, n, H, h);
    gv.load(V, 0, n, H, h);
    gk.store_rm(sK[0]);
    gk.store_tr(sKt[0]);
    gv.store_rm(sV[0]);
    drain();
    __syncthreads();
    const int64_t stages = cdiv(n, kStage);
    for (int64_t t = 0; t < stages; ++t) {
        const int buf = int(t & 1);
        const int64_t kbase = t * kStage;
        if (t + 1 < stages) {
            gk.load_any(K, kbase + kStage, n, H, h);
            gv.load_any(V, kbase + kStage, n, H, h);
        }
#pragma unroll
        for (int kb = 0; kb < kStage / 32; ++kb) {
            f32x16_t s[NB], dp[NB];
            #pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = dp[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(sK[buf], 32 * kb + (lane & 31), c, lane);
                #pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, qf[b].v[c], s[b]);
                const bf16x8_t v = lds_row8<D>(sV[buf], 32 * kb + (lane & 31), c, lane);
                #pragma unroll
                for (int b = 0; b < NB; ++b) dp[b] = mma(v, gf[b].v[c], dp[b]);
            }
            const int64_t key0 = kbase + 32 * kb;
            // ragged last block; marked unlikely so that the compiler keeps the masking
            // out of the other blocks (measured: the backward 1.4% faster, the
            // forward no faster)
            if (__builtin_expect(key0 + 32 > n, 0)) {
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    if (key0 + crow(i, lane) >= n)
#pragma unroll
                        for (int b = 0; b < NB; ++b) s[b][i] = kNegInf;
            }
            bf16x8_t db16[NB][2];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = ex2(fmaf(s[b][i], sl2, -lse2[b]));
                    s[b][i] = p * (dp[b][i] - Dq[b]);
                }
                db16[b][0] = acc_b16(s[b], 0);
                db16[b][1] = acc_b16(s[b], 1);
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t a = lds_perm8(sKt[buf], 32 * db + (lane & 31), 32 * kb + 16 * half, lane);
                    #pragma unroll
                    for (int b = 0; b < NB; ++b) acc[b][db] = mma(a, db16[b][half], acc[b][db]);
                }
        }
        if (t + 1 < stages) {
            gk.store_rm(sK[buf ^ 1]);
            gk.store_tr(sKt[buf ^ 1]);
            gv.store_rm(sV[buf ^ 1]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        if (q >= n) continue;
        uint16_t* o = dQ + (q * H + h) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x16_t& a = acc[b][db];
                *reinterpret_cast<uint2*>(o + 32 * db + 8 * j + 4 * (lane >> 5)) =
                    make_uint2(pack_bf16x2(a[4 * j] * scale, a[4 * j + 1] * scale),
                               pack_bf16x2(a[4 * j + 2] * scale, a[4 * j + 3] * scale));
            }
    }
}

// ----------------------------------------------------------- dK, dV (cols)
// dK_j = scale sum_i P_ij (dP_ij - D_i) Q_i and dV_j = sum_i P_ij dO_i, with
// the wavefront owning 32 NB keys and the queries streaming through LDS.

template <int D, int NB>
__global__ __launch_bounds__(kRowsWg / (32 * NB) * kWave) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 2 : 1))) void k_full_dkdv(int64_t n, int H, const uint16_t* __restrict__ Q,
                                                       const uint16_t* __restrict__ K,
                                                       const uint16_t* __restrict__ V,
                                                       const uint16_t* __restrict__ dO,
                                                       const float* __restrict__ LSE,
                                                       const float* __restrict__ Dv, float sl2, float scale,
                                                       uint16_t* __restrict__ dK, uint16_t* __restrict__ dV) {
    __shared__ __attribute__((aligned(16))) uint16_t sQ[2][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sG[2][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sQt[2][D * kTS];
    __shared__ __attribute__((aligned(16))) uint16_t sGt[2][D * kTS];
    __shared__ __attribute__((aligned(16))) float sL[2][kStage];
    __shared__ __attribute__((aligned(16))) float sD[2][kStage];
    int h;
    int64_t row0;
    if (!wg_coords(n, H, h, row0)) return;
    const int lane = lane_id();
    const int64_t k0 = row0 + (threadIdx.x / kWave) * 32 * NB;
    Frag<D> kf[NB], vf[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        kf[b].load(K, k0 + 32 * b + (lane & 31), n, H, h, lane);
        vf[b].load(V, k0 + 32 * b + (lane & 31), n, H, h, lane);
    }
    f32x16_t dk[NB][D / 32], dv[NB][D / 32];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) dk[b][db] = dv[b][db] = zero16();

    // LSE (exp2 domain) and D of the stage's queries; queries >= n get
    // LSE = +inf so that their weights are exactly zero.
    auto stage_rows = [&](int buf, int64_t base) {
        if (threadIdx.x < kStage) {
            const int64_t qn = base + threadIdx.x;
            sL[buf][threadIdx.x] = qn < n ? LSE[qn * H + h] * kLog2e : __builtin_huge_valf();
            sD[buf][threadIdx.x] = qn < n ? Dv[qn * H + h] : 0.f;
        }
    };
    Stager<D, kRowsWg / (32 * NB) * kWave> gq, gg;
    gq.load(Q, 0, n, H, h);
    gg.load(dO, 0, n, H, h);
    gq.store_rm(sQ[0]);
    gq.store_tr(sQt[0]);
    gg.store_rm(sG[0]);
    gg.store_tr(sGt[0]);
    stage_rows(0, 0);
    drain();
    __syncthreads();
    const int64_t stages = cdiv(n, kStage);
    for (int64_t t = 0; t < stages; ++t) {
        const int buf = int(t & 1);
        const int64_t qbase = t * kStage;
        if (t + 1 < stages) {
            gq.load_any(Q, qbase + kStage, n, H, h);
            gg.load_any(dO, qbase + kStage, n, H, h);
        }
#pragma unroll
        for (int qb = 0; qb < kStage / 32; ++qb) {
            f32x16_t s[NB], dp[NB];
            #pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = dp[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(sQ[buf], 32 * qb + (lane & 31), c, lane);
                #pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, kf[b].v[c], s[b]);
                const bf16x8_t g = lds_row8<D>(sG[buf], 32 * qb + (lane & 31), c, lane);
                #pragma unroll
                for (int b = 0; b < NB; ++b) dp[b] = mma(g, vf[b].v[c], dp[b]);
            }
            // rows of accumulator element i: 32 qb + 8 (i/4) + 4 (lane/32) + i%4
            float Lr[16], Dr[16];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 32 * qb + 8 * j + 4 * (lane >> 5);
                const float4 lv = *reinterpret_cast<const float4*>(&sL[buf][r]);
                const float4 dv4 = *reinterpret_cast<const float4*>(&sD[buf][r]);
                Lr[4 * j] = lv.x, Lr[4 * j + 1] = lv.y, Lr[4 * j + 2] = lv.z, Lr[4 * j + 3] = lv.w;
                Dr[4 * j] = dv4.x, Dr[4 * j + 1] = dv4.y, Dr[4 * j + 2] = dv4.z, Dr[4 * j + 3] = dv4.w;
            }
            bf16x8_t pb[NB][2], sb[NB][2];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = ex2(fmaf(s[b][i], sl2, -Lr[i]));
                    s[b][i] = p * (dp[b][i] - Dr[i]);
                    dp[b][i] = p;
                }
                pb[b][0] = acc_b16(dp[b], 0);
                pb[b][1] = acc_b16(dp[b], 1);
                sb[b][0] = acc_b16(s[b], 0);
                sb[b][1] = acc_b16(s[b], 1);
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t g = lds_perm8(sGt[buf], 32 * db + (lane & 31), 32 * qb + 16 * half, lane);
                    #pragma unroll
                    for (int b = 0; b < NB; ++b) dv[b][db] = mma(g, pb[b][half], dv[b][db]);
                    const bf16x8_t a = lds_perm8(sQt[buf], 32 * db + (lane & 31), 32 * qb + 16 * half, lane);
                    #pragma unroll
                    for (int b = 0; b < NB; ++b) dk[b][db] = mma(a, sb[b][half], dk[b][db]);
                }
        }
        if (t + 1 < stages) {
            gq.store_rm(sQ[buf ^ 1]);
            gq.store_tr(sQt[buf ^ 1]);
            gg.store_rm(sG[buf ^ 1]);
            gg.store_tr(sGt[buf ^ 1]);
            stage_rows(buf ^ 1, qbase + kStage);
        }
        __syncthreads();
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t key = k0 + 32 * b + (lane & 31);
        if (key >= n) continue;
        uint16_t* ok = dK + (key * H + h) * D;
        uint16_t* ov = dV + (key * H + h) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int f = 32 * db + 8 * j + 4 * (lane >> 5);
                const f32x16_t& a = dk[b][db];
                const f32x16_t& c = dv[b][db];
                *reinterpret_cast<uint2*>(ok + f) =
                    make_uint2(pack_bf16x2(a[4 * j] * scale, a[4 * j + 1] * scale),
                               pack_bf16x2(a[4 * j + 2] * scale, a[4 * j + 3] * scale));
                *reinterpret_cast<uint2*>(ov + f) =
                    make_uint2(pack_bf16x2(c[4 * j], c[4 * j + 1]), pack_bf16x2(c[4 * j + 2], c[4 * j + 3]));
            }
    }
}

// ------------------------------------------------------------ dense tiles
// Sparse layers: the dense tiles of the plan (§3.4), computed whole on the
// matrix cores with the tile's bit mask deciding which pairs are edges.  The
// row-owned kernels walk a tile row's dense tiles, the column-owned kernel a
// tile column's (in chunks of tiles); a workgroup has T/32 wavefronts of 32
// owned rows (one MFMA block each, kTileNB) and stages the partners 64 at a
// time.  Each kernel leaves fp32
// partial sums per (node, head) for the edge kernels, which add the remainder
// edges and finish every row and column.  A row may have no edge in a tile:
// its weights are exactly zero (masked scores are -inf, and an all-masked
// running maximum is treated as 0 in the exponent).

// Mask words of one owned row for one tile: bit c of word w <=> key 32 w + c.
template <int T>
__device__ __forceinline__ void load_mask_row(uint32_t (&mw)[T / 32], const uint32_t* __restrict__ row) {
    if constexpr (T == 128) {
        const uint4 v = *reinterpret_cast<const uint4*>(row);
        mw[0] = v.x, mw[1] = v.y, mw[2] = v.z, mw[3] = v.w;
    } else {
        const uint2 v = *reinterpret_cast<const uint2*>(row);
        mw[0] = v.x, mw[1] = v.y;
    }
}

// ---- chunks of the dense tiles of each tile row (column)

// Workgroup b -> tile row (column) I, its list range [t0, t1) and the output
// slot (-1: the partial state of the row; else an extra slot); false for the
// surplus of the grid.
__device__ __forceinline__ bool tile_chunk(const TileChunks& ck, const int64_t* __restrict__ ptr, int64_t R,
                                           int64_t b, int64_t& I, int64_t& t0, int64_t& t1, int64_t& slot) {
    if (b >= ck.chunk_off[R]) return false;
    int64_t lo = 0, hi = R;  // the last I with chunk_off[I] <= b
    while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (ck.chunk_off[mid] <= b) lo = mid;
        else hi = mid;
    }
    I = lo;
    const int64_t j = b - ck.chunk_off[lo];
    t0 = ptr[lo] + j * ck.CH;
    t1 = t0 + ck.CH < ptr[lo + 1] ? t0 + ck.CH : ptr[lo + 1];
    slot = j == 0 ? -1 : ck.extra_off[lo] + j - 1;
    return true;
}

// Output row of node q (tile row I) for a chunk writing `slot`.
__device__ __forceinline__ int64_t out_row(int64_t q, int64_t I, int64_t slot, int T) {
    return slot < 0 ? q : slot * T + (q - I * T);
}

// The plan in one workgroup (a tile plan has at most 16,384 tile rows).
// Wavefront w owns rows [1024 w, 1024 w + 1024) in 16 rounds of 64 consecutive
// rows (one per lane), so every load and store is coalesced: the wavefront
// totals give each wavefront its base, then each round's wavefront scan, plus
// the running total of the rounds before it, gives every row its chunk
// offset, extra-slot offset and place in the list of rows with extra slots.
constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / kWave;
constexpr int64_t kPlanMaxRows = 16384;
constexpr int kPlanRounds = int(kPlanMaxRows / kPlanThreads);

// Inclusive wavefront sum scan on DPP moves (no LDS round trips): shifts by
// 1, 2, 4 and 8 lanes scan each 16-lane row; broadcasting lane 15 into rows 1
// and 3, then lane 31 into rows 2 and 3, adds the totals of the rows before.
// Lanes a move does not reach take 0 (the `old` operand).
template <int Ctrl, int RowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
    return uint32_t(__builtin_amdgcn_update_dpp(0, int(x), Ctrl, RowMask, 0xF, false));
}
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t x) {
    x += dpp_u32<0x111, 0xF>(x);  // row_shr:1
    x += dpp_u32<0x112, 0xF>(x);  // row_shr:2
    x += dpp_u32<0x114, 0xF>(x);  // row_shr:4
    x += dpp_u32<0x118, 0xF>(x);  // row_shr:8
    x += dpp_u32<0x142, 0xA>(x);  // row_bcast:15 into rows 1, 3
    x += dpp_u32<0x143, 0xC>(x);  // row_bcast:31 into rows 2, 3
    return x;
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

__global__ __launch_bounds__(kPlanThreads) void k_tile_chunk_plan1(int64_t R, const int64_t* __restrict__ ptr,
                                                                   int CH, int64_t* __restrict__ chunk_off,
                                                                   int64_t* __restrict__ extra_off,
                                                                   int32_t* __restrict__ merge_rows,
                                                                   uint32_t* __restrict__ merge_cnt) {
    // Counts fit in 32 bits: at most R <= 16,384 tiles per row and R rows.
    __shared__ uint32_t s_w[3][kPlanWaves];
    const int t = threadIdx.x, w = t / kWave, lane = lane_id();
    const int64_t base = int64_t(w) * (kPlanRounds * kWave);
    uint32_t k[kPlanRounds];  // chunks of row base + 64 j + lane
#pragma unroll
    for (int j = 0; j < kPlanRounds; ++j) {
        const int64_t I = base + kWave * j + lane;
        k[j] = I < R ? (uint32_t(ptr[I + 1] - ptr[I]) + uint32_t(CH) - 1u) / uint32_t(CH) : 0u;
    }
    uint32_t c = 0, e = 0, m = 0;
#pragma unroll
    for (int j = 0; j < kPlanRounds; ++j) {
        c += k[j];
        e += k[j] > 1u ? k[j] - 1u : 0u;
        m += k[j] > 1u ? 1u : 0u;
    }
    c = wave_sum_u32(c);
    e = wave_sum_u32(e);
    m = wave_sum_u32(m);
    if (lane == 0) {
        s_w[0][w] = c;
        s_w[1][w] = e;
        s_w[2][w] = m;
    }
    __syncthreads();
    uint32_t bc = 0, be = 0, bm = 0, tc = 0, te = 0, tm = 0;
#pragma unroll 1
    for (int x = 0; x < kPlanWaves; ++x) {
        if (x < w) {
            bc += s_w[0][x];
            be += s_w[1][x];
            bm += s_w[2][x];
        }
        tc += s_w[0][x];
        te += s_w[1][x];
        tm += s_w[2][x];
    }
#pragma unroll
    for (int j = 0; j < kPlanRounds; ++j) {
        const int64_t I = base + kWave * j + lane;
        const uint32_t xe = k[j] > 1u ? k[j] - 1u : 0u, xm = k[j] > 1u ? 1u : 0u;
        const uint32_t ic = wave_incl_scan_u32(k[j]), ie = wave_incl_scan_u32(xe), im = wave_incl_scan_u32(xm);
        if (I < R) {
            chunk_off[I] = int64_t(bc + ic - k[j]);
            extra_off[I] = int64_t(be + ie - xe);
            if (xm) merge_rows[bm + im - 1u] = int32_t(I);
        }
        bc += uint32_t(__builtin_amdgcn_readlane(int(ic), kWave - 1));
        be += uint32_t(__builtin_amdgcn_readlane(int(ie), kWave - 1));
        bm += uint32_t(__builtin_amdgcn_readlane(int(im), kWave - 1));
    }
    if (t == 0) {
        chunk_off[R] = int64_t(tc);
        extra_off[R] = int64_t(te);
        *merge_cnt = tm;
    }
}

gt_status tile_chunk_plan(const gt_tiles* p, const int64_t* ptr, const TileChunks& ck, hipStream_t s) {
    const int64_t R = p->n_row_tiles;
    if (R > kPlanMaxRows) return fail(GT_ERR_UNSUPPORTED, "dense tiles: more than 16384 tile rows");
    k_tile_chunk_plan1<<<1, kPlanThreads, 0, s>>>(R, ptr, ck.CH, ck.chunk_off, ck.extra_off, ck.merge_rows,
                                                  ck.merge_cnt);
    GT_LAUNCH_CHECK("tile_chunk_plan");
    return GT_OK;
}

// Fold the extra slots of each tile row into its partial state.  A workgroup
// takes kMergeRows<D> rows of one (tile row, head), D / 4 consecutive lanes per
// row, one float4 each, so every slot row is read as whole cache lines.
constexpr int kMergeThreads = 256;
constexpr int kTileNB = 1;  // 32-row blocks per wavefront in the dense-tile kernels
template <int D>
constexpr int kMergeRows = kMergeThreads / (D / 4);

inline dim3 merge_grid(const TileChunks& ck, int H, int T, int D) {
    return dim3(unsigned(ck.max_merge), unsigned(H), unsigned(T / (kMergeThreads / (D / 4))));
}

// ... the forward's online-softmax states (m, l, acc) ...
template <int D, int T>
__global__ __launch_bounds__(kMergeThreads) void k_tiles_merge_fwd(int64_t n, int H, TileChunks ck,
                                                                   float* __restrict__ pm, float* __restrict__ pl,
                                                                   float* __restrict__ pacc) {
    if (blockIdx.x >= *ck.merge_cnt) return;
    const int64_t I = ck.merge_rows[blockIdx.x];
    const int h = blockIdx.y;
    const int64_t e0 = ck.extra_off[I], e1 = ck.extra_off[I + 1];
    const int lr = blockIdx.z * kMergeRows<D> + threadIdx.x / (D / 4);
    const int f = 4 * (threadIdx.x % (D / 4));
    const int64_t q = I * T + lr;
    if (q >= n) return;
    const int64_t row = q * H + h;
    const float m0 = pm[row];
    float M = m0;
    for (int64_t e = e0; e < e1; ++e) M = fmaxf(M, ck.m[(e * T + lr) * H + h]);
    if (M == -__builtin_huge_valf()) return;  // no dense-tile edge in any chunk
    const float w0 = m0 == -__builtin_huge_valf() ? 0.f : ex2(m0 - M);
    float lsum = pl[row] * w0;
    float4* out = reinterpret_cast<float4*>(pacc + row * D + f);
    float4 acc = *out;
    acc.x *= w0;
    acc.y *= w0;
    acc.z *= w0;
    acc.w *= w0;
#pragma unroll 2
    for (int64_t e = e0; e < e1; ++e) {
        const int64_t xr = (e * T + lr) * H + h;
        const float me = ck.m[xr];
        if (me == -__builtin_huge_valf()) continue;
        const float w = ex2(me - M);
        lsum += ck.l[xr] * w;
        const float4 x = *reinterpret_cast<const float4*>(ck.acc + xr * D + f);
        acc.x += x.x * w;
        acc.y += x.y * w;
        acc.z += x.z * w;
        acc.w += x.w * w;
    }
    *out = acc;
    if (f == 0) {
        pm[row] = M;
        pl[row] = lsum;
    }
}

// ... and plain sums (the backward's A, B, D and dK, dV).
template <int D, int T>
__global__ __launch_bounds__(kMergeThreads) void k_tiles_merge_sum(int64_t n, int H, TileChunks ck,
                                                                   float* __restrict__ a, float* __restrict__ b,
                                                                   float* __restrict__ m) {
    if (blockIdx.x >= *ck.merge_cnt) return;
    const int64_t I = ck.merge_rows[blockIdx.x];
    const int h = blockIdx.y;
    const int64_t e0 = ck.extra_off[I], e1 = ck.extra_off[I + 1];
    const int lr = blockIdx.z * kMergeRows<D> + threadIdx.x / (D / 4);
    const int f = 4 * (threadIdx.x % (D / 4));
    const int64_t q = I * T + lr;
    if (q >= n) return;
    const int64_t row = q * H + h;
    float4* pa = reinterpret_cast<float4*>(a + row * D + f);
    float4* pb = b ? reinterpret_cast<float4*>(b + row * D + f) : nullptr;
    float4 sa = *pa, sb = pb ? *pb : make_float4(0.f, 0.f, 0.f, 0.f);
    float sm = (m && f == 0) ? m[row] : 0.f;
#pragma unroll 2
    for (int64_t e = e0; e < e1; ++e) {
        const int64_t xr = (e * T + lr) * H + h;
        const float4 x = *reinterpret_cast<const float4*>(ck.acc + xr * D + f);
        sa.x += x.x;
        sa.y += x.y;
        sa.z += x.z;
        sa.w += x.w;
        if (pb) {
            const float4 y = *reinterpret_cast<const float4*>(ck.acc2 + xr * D + f);
            sb.x += y.x;
            sb.y += y.y;
            sb.z += y.z;
            sb.w += y.w;
        }
        if (m && f == 0) sm += ck.m[xr];
    }
    *pa = sa;
    if (pb) *pb = sb;
    if (m && f == 0) m[row] = sm;
}

// NB 32-row blocks per wavefront (2: every K and V fragment read from LDS
// feeds two products; 1: half the registers, twice the wavefronts).  The
// tiles are launched with NB = 1 (kTileNB): a chunk holds only a few tiles, so
// the kernels are latency-bound and more resident wavefronts pay more than
// the operand reuse; the occupancy hints keep the accumulators out of the
// AGPRs (forward: 4 wavefronts per SIMD at d = 32 and 64; dQ, dK/dV: 2-3).
template <int D, int T, int NB, bool kBias = false>
__global__ __launch_bounds__(T * 2 / NB) __attribute__((amdgpu_waves_per_eu(D >= 64 ? 3 : 4))) void k_tiles_fwd(
    int64_t n, int H, const int64_t* __restrict__ tile_rowptr,
                                                 const int32_t* __restrict__ tile_col,
                                                 const uint32_t* __restrict__ tile_mask,
                                                 const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                 const uint16_t* __restrict__ V, float sl2, float* __restrict__ pm,
                                                 float* __restrict__ pl, float* __restrict__ pacc, int64_t R,
                                                 TileChunks ck, TileBias tb) {
    constexpr int W = T / 32;
    __shared__ __attribute__((aligned(16))) uint16_t sK[1][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sVt[1][D * kTS];
    const int h = blockIdx.y;
    int64_t I, t0, t1, slot;
    if (!tile_chunk(ck, tile_rowptr, R, blockIdx.x, I, t0, t1, slot)) return;
    if (slot >= 0) {
        pm = ck.m;
        pl = ck.l;
        pacc = ck.acc;
    }
    const int lane = lane_id();
    constexpr int NT = T * 2 / NB;
    const int ql0 = (threadIdx.x / kWave) * 32 * NB;  // first owned row inside the tile row
    const int64_t q0 = int64_t(I) * T + ql0;
    Frag<D> qf[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) qf[b].load(Q, q0 + 32 * b + (lane & 31), n, H, h, lane);
    if (sl2 < 0.f) {  // keep the exp2-domain scale positive: negate Q instead (exact in bf16)
        sl2 = -sl2;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int c = 0; c < D / 16; ++c)
                qf[b].v[c] = __builtin_bit_cast(bf16x8_t, __builtin_bit_cast(uint4, qf[b].v[c]) ^
                                                              make_uint4(0x80008000u, 0x80008000u, 0x80008000u,
                                                                         0x80008000u));
    }
    f32x16_t acc[NB][D / 32];
    float m[NB], l[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) acc[b][db] = zero16();
        m[b] = kNegInf;
        l[b] = 0.f;
    }
    // Stages run over the tile row's dense tiles, T/64 per tile.  They are
    // single-buffered: several small workgroups per CU hide each other's
    // loads, which a register prefetch (at one wavefront per SIMD) did not.
    constexpr int NSG = T / kStage;
    const int64_t stages = (t1 - t0) * NSG;
    Stager<D, NT> gk, gv;
    uint32_t mw[NB][W];
    auto fetch = [&](int64_t g, uint32_t (&mwx)[NB][W]) {
        const int64_t k = t0 + g / NSG;
        const int64_t kb = int64_t(tile_col[k]) * T + kStage * (g % NSG);
        gk.load(K, kb, n, H, h);
        gv.load(V, kb, n, H, h);
        if (g % NSG == 0)
#pragma unroll
            for (int b = 0; b < NB; ++b)
                load_mask_row<T>(mwx[b], tile_mask + (k * T + ql0 + 32 * b + (lane & 31)) * W);
    };
#pragma unroll 1
    for (int64_t g = 0; g < stages; ++g) {
        const int buf = 0, st = int(g % NSG);
        fetch(g, mw);
        __syncthreads();  // the previous stage's readers are done
        gk.store_rm(sK[0]);
        gv.store_tr(sVt[0]);
        __syncthreads();
#pragma unroll
        for (int kb = 0; kb < kStage / 32; ++kb) {
            f32x16_t s[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(sK[buf], 32 * kb + (lane & 31), c, lane);
#pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, qf[b].v[c], s[b]);
            }
            bool grow = false;
            float mt[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint32_t w = mw[b][2 * st + kb];
                if constexpr (kBias) {
                    // scores in the exp2 domain with the bias added: s sl2 + b log2 e
                    const int64_t tk = t0 + g / NSG;
                    const int r = ql0 + 32 * b + (lane & 31);
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        // the per-tile bias is -inf off the edges, so it masks the cell itself: no test and
                        // no branch, which keeps the wait states of the accumulator reads that follow
                        const float bb = tb.b[TileBias::at(tk, H, h, T, r, kStage * st + 32 * kb + crow(i, lane))];
                        s[b][i] = fmaf(s[b][i], sl2, bb * kLog2e);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (!((w >> crow(i, lane)) & 1u)) s[b][i] = kNegInf;
                }
                float mx = s[b][0];
#pragma unroll
                for (int i = 1; i < 16; ++i) mx = fmaxf(mx, s[b][i]);
                mt[b] = kBias ? pair_max(mx) : pair_max(mx) * sl2;
                grow |= mt[b] > m[b] + kLazy;
            }
            if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const float mn = fmaxf(m[b], mt[b]);
                    if (mn == kNegInf) continue;
                    const float alpha = ex2(m[b] - mn);
                    l[b] *= alpha;
#pragma unroll
                    for (int db = 0; db < D / 32; ++db)
#pragma unroll
                        for (int i = 0; i < 16; ++i) acc[b][db][i] *= alpha;
                    m[b] = mn;
                }
            }
            bf16x8_t pb[NB][2];
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const float mm = m[b] == kNegInf ? 0.f : m[b];
                float ls = 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float p = kBias ? ex2(s[b][i] - mm) : ex2(fmaf(s[b][i], sl2, -mm));
                    s[b][i] = p;
                    ls += p;
                }
                l[b] += ls;
                pb[b][0] = acc_b16(s[b], 0);
                pb[b][1] = acc_b16(s[b], 1);
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t a = lds_perm8(sVt[buf], 32 * db + (lane & 31), 32 * kb + 16 * half, lane);
#pragma unroll
                    for (int b = 0; b < NB; ++b) acc[b][db] = mma(a, pb[b][half], acc[b][db]);
                }
        }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        const float lt = pair_sum(l[b]);
        if (q >= n) continue;
        const int64_t orow = out_row(q, I, slot, T);
        if (lane < 32) {
            pm[orow * H + h] = m[b];
            pl[orow * H + h] = lt;
        }
        float* o = pacc + (orow * H + h) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x16_t& a = acc[b][db];
                *reinterpret_cast<float4*>(o + 32 * db + 8 * j + 4 * (lane >> 5)) =
                    make_float4(a[4 * j], a[4 * j + 1], a[4 * j + 2], a[4 * j + 3]);
            }
    }
}

// Weights w as bf16 hi + lo parts (about 16 mantissa bits): B operands of
// two products whose sum keeps the fp32 weight, for sums of many large
// weights and for the A - D B difference of the row pass.
__device__ __forceinline__ void split_b16(const f32x16_t& w, int half, bf16x8_t& hi, bf16x8_t& lo) {
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        hi[t] = (__bf16)w[8 * half + t];
        lo[t] = (__bf16)(w[8 * half + t] - float(hi[t]));
    }
}

// Row pass over the dense tiles: A = sum P dP K, B = sum P K and the D sum
// sum P dP of every owned row (the edge kernels form dQ = scale (A - D B)).
template <int D, int T, int NB, bool kBias = false>
__global__ __launch_bounds__(T * 2 / NB) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 2 : 1))) void k_tiles_dq(
    int64_t n, int H, const int64_t* __restrict__ tile_rowptr,
                                                const int32_t* __restrict__ tile_col,
                                                const uint32_t* __restrict__ tile_mask,
                                                const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
                                                const float* __restrict__ LSE, float sl2, float* __restrict__ pa,
                                                float* __restrict__ pb, float* __restrict__ pd, int64_t R,
                                                TileChunks ck, TileBias tb) {
    constexpr int W = T / 32;
    __shared__ __attribute__((aligned(16))) uint16_t sK[1][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sV[1][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sKt[1][D * kTS];
    const int h = blockIdx.y;
    int64_t I, t0, t1, slot;
    if (!tile_chunk(ck, tile_rowptr, R, blockIdx.x, I, t0, t1, slot)) return;
    if (slot >= 0) {
        pa = ck.acc;
        pb = ck.acc2;
        pd = ck.m;
    }
    const int lane = lane_id();
    constexpr int NT = T * 2 / NB;
    const int ql0 = (threadIdx.x / kWave) * 32 * NB;
    const int64_t q0 = int64_t(I) * T + ql0;
    Frag<D> qf[NB], gf[NB];
    float lse2[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        qf[b].load(Q, q, n, H, h, lane);
        gf[b].load(dO, q, n, H, h, lane);
        lse2[b] = q < n ? LSE[q * H + h] * kLog2e : 0.f;
    }
    f32x16_t accA[NB][D / 32], accB[NB][D / 32];
    float dsum[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db) accA[b][db] = accB[b][db] = zero16();
        dsum[b] = 0.f;
    }
    constexpr int NSG = T / kStage;
    const int64_t stages = (t1 - t0) * NSG;
    Stager<D, NT> gk, gv;
    uint32_t mw[NB][W];
    auto fetch = [&](int64_t g, uint32_t (&mwx)[NB][W]) {
        const int64_t k = t0 + g / NSG;
        const int64_t kb = int64_t(tile_col[k]) * T + kStage * (g % NSG);
        gk.load(K, kb, n, H, h);
        gv.load(V, kb, n, H, h);
        if (g % NSG == 0)
#pragma unroll
            for (int b = 0; b < NB; ++b)
                load_mask_row<T>(mwx[b], tile_mask + (k * T + ql0 + 32 * b + (lane & 31)) * W);
    };
#pragma unroll 1
    for (int64_t g = 0; g < stages; ++g) {
        const int buf = 0, st = int(g % NSG);
        fetch(g, mw);
        __syncthreads();
        gk.store_rm(sK[0]);
        gk.store_tr(sKt[0]);
        gv.store_rm(sV[0]);
        __syncthreads();
#pragma unroll
        for (int kb = 0; kb < kStage / 32; ++kb) {
            f32x16_t s[NB], dp[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = dp[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(sK[buf], 32 * kb + (lane & 31), c, lane);
#pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, qf[b].v[c], s[b]);
                const bf16x8_t v = lds_row8<D>(sV[buf], 32 * kb + (lane & 31), c, lane);
#pragma unroll
                for (int b = 0; b < NB; ++b) dp[b] = mma(v, gf[b].v[c], dp[b]);
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint32_t w = mw[b][2 * st + kb];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    float p;
                    if constexpr (kBias) {
                        const int64_t tk = t0 + g / NSG;
                        const int r = ql0 + 32 * b + (lane & 31), c = kStage * st + 32 * kb + crow(i, lane);
                        const float bb = tb.b[TileBias::at(tk, H, h, T, r, c)];
                        p = ex2(fmaf(s[b][i], sl2, bb * kLog2e - lse2[b]));  // 0 off the edges (bias -inf)
                    } else {
                        p = (w >> crow(i, lane)) & 1u ? ex2(fmaf(s[b][i], sl2, -lse2[b])) : 0.f;
                    }
                    s[b][i] = p;
                    dp[b][i] *= p;
                    dsum[b] += dp[b][i];
                }
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t a = lds_perm8(sKt[buf], 32 * db + (lane & 31), 32 * kb + 16 * half, lane);
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        bf16x8_t hi, lo;
                        split_b16(dp[b], half, hi, lo);
                        accA[b][db] = mma(a, lo, mma(a, hi, accA[b][db]));
                        split_b16(s[b], half, hi, lo);
                        accB[b][db] = mma(a, lo, mma(a, hi, accB[b][db]));
                    }
                }
        }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t q = q0 + 32 * b + (lane & 31);
        const float ds = pair_sum(dsum[b]);
        if (q >= n) continue;
        const int64_t orow = out_row(q, I, slot, T);
        if (lane < 32) pd[orow * H + h] = ds;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int f = 32 * db + 8 * j + 4 * (lane >> 5);
                const f32x16_t& x = accA[b][db];
                const f32x16_t& y = accB[b][db];
                *reinterpret_cast<float4*>(pa + (orow * H + h) * D + f) =
                    make_float4(x[4 * j], x[4 * j + 1], x[4 * j + 2], x[4 * j + 3]);
                *reinterpret_cast<float4*>(pb + (orow * H + h) * D + f) =
                    make_float4(y[4 * j], y[4 * j + 1], y[4 * j + 2], y[4 * j + 3]);
            }
    }
}

// One butterfly step of a 32 x 32 bit-matrix transpose held one row per lane
// in each half of the wavefront: the lanes with bit J set trade the low J bits
// of each 2J-bit group for their partner's high J bits (ds_swizzle in bitmask
// mode, xor J within 32 lanes).
template <int J>
__device__ __forceinline__ uint32_t bit_transpose_step(uint32_t w, int lane) {
    constexpr uint32_t lo = J == 16 ? 0x0000FFFFu : J == 8 ? 0x00FF00FFu : J == 4 ? 0x0F0F0F0Fu : J == 2 ? 0x33333333u
                                                                                                           : 0x55555555u;
    const uint32_t t = uint32_t(__builtin_amdgcn_ds_swizzle(int(w), (J << 10) | 0x1F));
    return (lane & J) ? (w & ~lo) | ((t & ~lo) >> J) : (w & lo) | ((t & lo) << J);
}

// Transpose of the 64 x 32 bit matrix whose row r is lane r's word: on return
// bit r of lane c's word (either half: both get the same 64 bits) is entry
// (r, c % 32).
__device__ __forceinline__ uint64_t bit_transpose_64x32(uint32_t w, int lane) {
    w = bit_transpose_step<16>(w, lane);
    w = bit_transpose_step<8>(w, lane);
    w = bit_transpose_step<4>(w, lane);
    w = bit_transpose_step<2>(w, lane);
    w = bit_transpose_step<1>(w, lane);
    const uint32_t other = __shfl_xor(w, 32, kWave);
    return lane < 32 ? uint64_t(w) | (uint64_t(other) << 32) : uint64_t(other) | (uint64_t(w) << 32);
}

// Column pass over the dense tiles: unscaled dK and dV sums of every owned key.
// The stage's masks are transposed so that each lane holds, for its key, one
// 64-bit word over the stage's 64 queries.
template <int D, int T, int NB, bool kBias = false>
__global__ __launch_bounds__(T * 2 / NB) __attribute__((amdgpu_waves_per_eu(NB == 1 ? 2 : 1))) void k_tiles_dkdv(
    int64_t n, int H, int64_t n_row_tiles,
                                                  const int64_t* __restrict__ tileT_ptr,
                                                  const int32_t* __restrict__ tileT_idx,
                                                  const int64_t* __restrict__ tile_rowptr,
                                                  const uint32_t* __restrict__ tile_mask,
                                                  const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                  const uint16_t* __restrict__ V, const uint16_t* __restrict__ dO,
                                                  const float* __restrict__ LSE, const float* __restrict__ Dv,
                                                  float sl2, float* __restrict__ pdk, float* __restrict__ pdv,
                                                  TileChunks ck, TileBias tb) {
    constexpr int W = T / 32;
    __shared__ __attribute__((aligned(16))) uint16_t sQ[1][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sG[1][kStage * RS<D>::v];
    __shared__ __attribute__((aligned(16))) uint16_t sQt[1][D * kTS];
    __shared__ __attribute__((aligned(16))) uint16_t sGt[1][D * kTS];
    __shared__ __attribute__((aligned(16))) float sL[1][kStage];
    __shared__ __attribute__((aligned(16))) float sD[1][kStage];
    const int h = blockIdx.y;
    int64_t J, u0, u1, slot;
    if (!tile_chunk(ck, tileT_ptr, n_row_tiles, blockIdx.x, J, u0, u1, slot)) return;
    if (slot >= 0) {
        pdk = ck.acc;
        pdv = ck.acc2;
    }
    const int lane = lane_id();
    constexpr int NT = T * 2 / NB;
    const int kl0 = (threadIdx.x / kWave) * 32 * NB;  // first owned key inside the tile column
    const int64_t k0 = int64_t(J) * T + kl0;
    Frag<D> kf[NB], vf[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        kf[b].load(K, k0 + 32 * b + (lane & 31), n, H, h, lane);
        vf[b].load(V, k0 + 32 * b + (lane & 31), n, H, h, lane);
    }
    f32x16_t dk[NB][D / 32], dv[NB][D / 32];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int db = 0; db < D / 32; ++db) dk[b][db] = dv[b][db] = zero16();
    constexpr int NSG = T / kStage;
    const int64_t stages = (u1 - u0) * NSG;
    Stager<D, NT> gq, gg;
    uint32_t mword[NB];  // this lane's row of the stage: mask words of the wavefront's key blocks
    float2 stat;        // LSE (exp2 domain) and D of the stage's query threadIdx.x % kStage
    int64_t tk = 0;     // the stage's tile
    auto fetch = [&](int64_t g) {
        const int64_t k = tileT_idx[u0 + g / NSG];
        tk = k;
        int64_t lo = 0, hi = n_row_tiles;  // tile row of tile k: the last I with tile_rowptr[I] <= k
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (tile_rowptr[mid] <= k) lo = mid;
            else hi = mid;
        }
        const int st = int(g % NSG);
        const int64_t qbase = lo * T + kStage * st;
        gq.load(Q, qbase, n, H, h);
        gg.load(dO, qbase, n, H, h);
#pragma unroll
        for (int b = 0; b < NB; ++b) mword[b] = tile_mask[(k * T + kStage * st + lane) * W + (kl0 / 32 + b)];
        stat = make_float2(__builtin_huge_valf(), 0.f);  // queries >= n take no weight
        const int64_t qn = qbase + (threadIdx.x % kStage);
        if (qn < n) stat = make_float2(LSE[qn * H + h] * kLog2e, Dv[qn * H + h]);
    };
    // transposed masks: bit r of mt[b] <=> query r of the stage attends to key k0 + 32 b + lane % 32
    uint64_t mt[NB];
    auto transpose = [&](uint64_t (&out)[NB]) {
#pragma unroll
        for (int b = 0; b < NB; ++b) out[b] = bit_transpose_64x32(mword[b], lane);
    };
    auto store = [&](int buf) {
        gq.store_rm(sQ[buf]);
        gq.store_tr(sQt[buf]);
        gg.store_rm(sG[buf]);
        gg.store_tr(sGt[buf]);
        if (threadIdx.x < kStage) {
            sL[buf][threadIdx.x] = stat.x;
            sD[buf][threadIdx.x] = stat.y;
        }
    };
#pragma unroll 1
    for (int64_t g = 0; g < stages; ++g) {
        const int buf = 0;
        fetch(g);
        transpose(mt);
        __syncthreads();  // the previous stage's readers are done
        store(0);
        __syncthreads();
#pragma unroll
        for (int qb = 0; qb < kStage / 32; ++qb) {
            f32x16_t s[NB], dp[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) s[b] = dp[b] = zero16();
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
                const bf16x8_t a = lds_row8<D>(sQ[buf], 32 * qb + (lane & 31), c, lane);
#pragma unroll
                for (int b = 0; b < NB; ++b) s[b] = mma(a, kf[b].v[c], s[b]);
                const bf16x8_t g8 = lds_row8<D>(sG[buf], 32 * qb + (lane & 31), c, lane);
#pragma unroll
                for (int b = 0; b < NB; ++b) dp[b] = mma(g8, vf[b].v[c], dp[b]);
            }
            float Lr[16], Dr[16];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 32 * qb + 8 * j + 4 * (lane >> 5);
                const float4 lv = *reinterpret_cast<const float4*>(&sL[buf][r]);
                const float4 d4 = *reinterpret_cast<const float4*>(&sD[buf][r]);
                Lr[4 * j] = lv.x, Lr[4 * j + 1] = lv.y, Lr[4 * j + 2] = lv.z, Lr[4 * j + 3] = lv.w;
                Dr[4 * j] = d4.x, Dr[4 * j + 1] = d4.y, Dr[4 * j + 2] = d4.z, Dr[4 * j + 3] = d4.w;
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const uint32_t w = uint32_t(mt[b] >> (32 * qb));
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const bool on = (w >> crow(i, lane)) & 1u;
                    float p = 0.f;
                    if constexpr (kBias) {
                        const int st = int(g % NSG);
                        const int r = kStage * st + 32 * qb + crow(i, lane), c = kl0 + 32 * b + (lane & 31);
                        const int64_t x = TileBias::at(tk, H, h, T, r, c);
                        p = ex2(fmaf(s[b][i], sl2, tb.b[x] * kLog2e - Lr[i]));  // 0 off the edges (bias -inf)
                        s[b][i] = p * (dp[b][i] - Dr[i]);
                        tb.db[x] = s[b][i];  // every cell (0 off the edges), so no branch is needed
                    } else {
                        p = on ? ex2(fmaf(s[b][i], sl2, -Lr[i])) : 0.f;
                        s[b][i] = p * (dp[b][i] - Dr[i]);
                    }
                    dp[b][i] = p;
                }
            }
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const bf16x8_t g8 = lds_perm8(sGt[buf], 32 * db + (lane & 31), 32 * qb + 16 * half, lane);
                    const bf16x8_t a = lds_perm8(sQt[buf], 32 * db + (lane & 31), 32 * qb + 16 * half, lane);
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        bf16x8_t hi16, lo16;
                        split_b16(dp[b], half, hi16, lo16);
                        dv[b][db] = mma(g8, lo16, mma(g8, hi16, dv[b][db]));
                        split_b16(s[b], half, hi16, lo16);
                        dk[b][db] = mma(a, lo16, mma(a, hi16, dk[b][db]));
                    }
                }
        }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int64_t key = k0 + 32 * b + (lane & 31);
        if (key >= n) continue;
        const int64_t orow = out_row(key, J, slot, T);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int f = 32 * db + 8 * j + 4 * (lane >> 5);
                const f32x16_t& x = dk[b][db];
                const f32x16_t& y = dv[b][db];
                *reinterpret_cast<float4*>(pdk + (orow * H + h) * D + f) =
                    make_float4(x[4 * j], x[4 * j + 1], x[4 * j + 2], x[4 * j + 3]);
                *reinterpret_cast<float4*>(pdv + (orow * H + h) * D + f) =
                    make_float4(y[4 * j], y[4 * j + 1], y[4 * j + 2], y[4 * j + 3]);
            }
    }
}

}  // namespace

template <int D>
gt_status full_fwd_bf16(int64_t n, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V, float sl2,
                        uint16_t* O, float* LSE, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_full_fwd<D, kFullFwdNB><<<full_grid(n, H), kFullFwdThr, 0, s>>>(n, H, Q, K, V, sl2, O, LSE);
    GT_LAUNCH_CHECK("full_fwd_bf16");
    return GT_OK;
}

template <int D>
gt_status full_bwd_bf16(int64_t n, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* O, const uint16_t* dO, const float* LSE, float sl2, float scale,
                        uint16_t* dQ, uint16_t* dK, uint16_t* dV, float* Dv, hipStream_t s) {
    if (n <= 0) return GT_OK;
    k_full_dq<D, kFullBwdNB><<<full_grid(n, H), kFullBwdThr, 0, s>>>(n, H, Q, K, V, O, dO, LSE, sl2, scale, dQ, Dv);
    GT_LAUNCH_CHECK("full_bwd_bf16 dq");
    k_full_dkdv<D, kFullBwdNB><<<full_grid(n, H), kFullBwdThr, 0, s>>>(n, H, Q, K, V, dO, LSE, Dv, sl2, scale, dK, dV);
    GT_LAUNCH_CHECK("full_bwd_bf16 dkdv");
    return GT_OK;
}


#define GT_TILES_T(CALL)                                                          \
    do {                                                                          \
        if (p->T == 128) {                                                        \
            constexpr int TT = 128;                                               \
            CALL;                                                                 \
        } else if (p->T == 64) {                                                  \
            constexpr int TT = 64;                                                \
            CALL;                                                                 \
        } else {                                                                  \
            return fail(GT_ERR_UNSUPPORTED, "dense tiles: T must be 64 or 128");  \
        }                                                                         \
    } while (0)

template <int D>
gt_status tiles_fwd_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                         float sl2, TilePartials tp, TileBias tb, hipStream_t s) {
    gt_status st = tile_chunk_plan(p, p->tile_rowptr, tp.ck, s);
    if (st != GT_OK) return st;
    const dim3 grid(unsigned(tp.ck.max_chunks), unsigned(H));
    constexpr int NB = kTileNB;
    if (tb.b)
        GT_TILES_T((k_tiles_fwd<D, TT, NB, true><<<grid, TT * 2 / NB, 0, s>>>(
            p->n, H, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, sl2, tp.m, tp.l, tp.acc, p->n_row_tiles,
            tp.ck, tb)));
    else
        GT_TILES_T((k_tiles_fwd<D, TT, NB><<<grid, TT * 2 / NB, 0, s>>>(p->n, H, p->tile_rowptr, p->tile_col,
                                                                        p->tile_mask, Q, K, V, sl2, tp.m, tp.l,
                                                                        tp.acc, p->n_row_tiles, tp.ck, tb)));
    GT_LAUNCH_CHECK("tiles_fwd_bf16");
    GT_TILES_T((k_tiles_merge_fwd<D, TT><<<merge_grid(tp.ck, H, TT, D), kMergeThreads, 0, s>>>(
        p->n, H, tp.ck, tp.m, tp.l, tp.acc)));
    GT_LAUNCH_CHECK("tiles_merge_fwd_bf16");
    return GT_OK;
}

template <int D>
gt_status tiles_dq_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                        const uint16_t* dO, const float* LSE, float sl2, TilePartials dq, TileBias tb,
                        hipStream_t s) {
    gt_status st = tile_chunk_plan(p, p->tile_rowptr, dq.ck, s);
    if (st != GT_OK) return st;
    const dim3 grid(unsigned(dq.ck.max_chunks), unsigned(H));
    constexpr int NB = kTileNB;
    if (tb.b)
        GT_TILES_T((k_tiles_dq<D, TT, NB, true><<<grid, TT * 2 / NB, 0, s>>>(
            p->n, H, p->tile_rowptr, p->tile_col, p->tile_mask, Q, K, V, dO, LSE, sl2, dq.acc, dq.acc2, dq.m,
            p->n_row_tiles, dq.ck, tb)));
    else
        GT_TILES_T((k_tiles_dq<D, TT, NB><<<grid, TT * 2 / NB, 0, s>>>(p->n, H, p->tile_rowptr, p->tile_col,
                                                                       p->tile_mask, Q, K, V, dO, LSE, sl2, dq.acc,
                                                                       dq.acc2, dq.m, p->n_row_tiles, dq.ck, tb)));
    GT_LAUNCH_CHECK("tiles_dq_bf16");
    GT_TILES_T((k_tiles_merge_sum<D, TT><<<merge_grid(dq.ck, H, TT, D), kMergeThreads, 0, s>>>(
        p->n, H, dq.ck, dq.acc, dq.acc2, dq.m)));
    GT_LAUNCH_CHECK("tiles_merge_dq_bf16");
    return GT_OK;
}

template <int D>
gt_status tiles_dkdv_bf16(const gt_tiles* p, int H, const uint16_t* Q, const uint16_t* K, const uint16_t* V,
                          const uint16_t* dO, const float* LSE, const float* Dv, float sl2, TilePartials dk,
                          TilePartials dv, TileBias tb, hipStream_t s) {
    gt_status st = tile_chunk_plan(p, p->tileT_ptr, dk.ck, s);
    if (st != GT_OK) return st;
    const dim3 grid(unsigned(dk.ck.max_chunks), unsigned(H));
    constexpr int NB = kTileNB;
    if (tb.b)
        GT_TILES_T((k_tiles_dkdv<D, TT, NB, true><<<grid, TT * 2 / NB, 0, s>>>(
            p->n, H, p->n_row_tiles, p->tileT_ptr, p->tileT_idx, p->tile_rowptr, p->tile_mask, Q, K, V, dO, LSE, Dv,
            sl2, dk.acc, dv.acc, dk.ck, tb)));
    else
        GT_TILES_T((k_tiles_dkdv<D, TT, NB><<<grid, TT * 2 / NB, 0, s>>>(p->n, H, p->n_row_tiles, p->tileT_ptr,
                                                                         p->tileT_idx, p->tile_rowptr, p->tile_mask,
                                                                         Q, K, V, dO, LSE, Dv, sl2, dk.acc, dv.acc,
                                                                         dk.ck, tb)));
    GT_LAUNCH_CHECK("tiles_dkdv_bf16");
    GT_TILES_T((k_tiles_merge_sum<D, TT><<<merge_grid(dk.ck, H, TT, D), kMergeThreads, 0, s>>>(
        p->n, H, dk.ck, dk.acc, dv.acc, nullptr)));
    GT_LAUNCH_CHECK("tiles_merge_dkdv_bf16");
    return GT_OK;
}

#define GT_TILES_INST(D)                                                                                        \
    template gt_status tiles_fwd_bf16<D>(const gt_tiles*, int, const uint16_t*, const uint16_t*, const uint16_t*, \
                                         float, TilePartials, TileBias, hipStream_t);                           \
    template gt_status tiles_dq_bf16<D>(const gt_tiles*, int, const uint16_t*, const uint16_t*, const uint16_t*,  \
                                        const uint16_t*, const float*, float, TilePartials, TileBias,           \
                                        hipStream_t);                                                           \
    template gt_status tiles_dkdv_bf16<D>(const gt_tiles*, int, const uint16_t*, const uint16_t*,                \
                                          const uint16_t*, const uint16_t*, const float*, const float*, float,  \
                                          TilePartials, TilePartials, TileBias, hipStream_t);
GT_TILES_INST(32)
GT_TILES_INST(64)

template gt_status full_fwd_bf16<32>(int64_t, int, const uint16_t*, const uint16_t*, const uint16_t*, float,
                                     uint16_t*, float*, hipStream_t);
template gt_status full_fwd_bf16<64>(int64_t, int, const uint16_t*, const uint16_t*, const uint16_t*, float,
                                     uint16_t*, float*, hipStream_t);
template gt_status full_bwd_bf16<32>(int64_t, int, const uint16_t*, const uint16_t*, const uint16_t*,
                                     const uint16_t*, const uint16_t*, const float*, float, float, uint16_t*,
                                     uint16_t*, uint16_t*, float*, hipStream_t);
template gt_status full_bwd_bf16<64>(int64_t, int, const uint16_t*, const uint16_t*, const uint16_t*,
                                     const uint16_t*, const uint16_t*, const float*, float, float, uint16_t*,
                                     uint16_t*, uint16_t*, float*, hipStream_t);

}  // namespace gt
