/*
 * gt.h - C ABI of libgt, graph-topology sparse attention for AMD MI355X (gfx950).
 *
 * Operations follow TorchGT (arXiv 2407.14106):
 *   - neighbourhood softmax attention, §3.2 (local topology-induced pattern):
 *     node i attends only to the nodes j of its CSR row N(i);
 *   - full softmax attention, §2.1 Eq. (1), for the interleaved dense layer
 *     of §3.2 (interleave fully-connected pattern);
 *   - cluster reordering of the nodes, §3.3 (utilisation of graph cluster),
 *     here a deterministic label-propagation order instead of METIS;
 *   - the dense/sparse tile plan of §3.4 (cluster sparsity and the transfer
 *     threshold), read as an exact execution plan: a T x T tile of the
 *     reordered adjacency whose share of non-zeros reaches the threshold is
 *     computed with matrix cores over the whole tile (masked), every other
 *     edge is computed edge by edge.  The split never changes the result.
 *
 * Conventions shared by every entry point:
 *   - Every pointer is device memory unless its comment says "host".  All
 *     memory is owned by the caller; the library allocates nothing, creates no
 *     stream or event, and keeps no state between calls except the
 *     thread-local error text (what one call leaves for another, such as the
 *     tile counts, stays in the caller's workspace) and, for the one entry
 *     point that takes no workspace (gt_dense_attn_bwd_noalloc), its device
 *     scratch array and that array's address on each device.
 *   - Scratch memory comes from a caller workspace `ws` of at least the size
 *     returned by the matching *_workspace_size() function (256-byte aligned
 *     base).  A smaller workspace gives GT_ERR_WORKSPACE.
 *   - Every call is enqueued on `stream` and returns without waiting, except
 *     the calls marked SYNC, which wait for `stream` to read back a count or a
 *     validation result.
 *   - Arguments are checked on the host before anything is enqueued; on an
 *     error nothing touches the device and a negative gt_status is returned
 *     (gt_last_error() gives the reason).
 *   - Feature tensors Q, K, V, O, dO, dQ, dK, dV are [n, H, d] row-major
 *     (node, head, feature) in the element type `dtype`; LSE is [n, H] fp32.
 *     Supported: d in {32, 64}; H in {1, 2, 4, 8, 16}; dtype GT_F32 or GT_BF16.
 *     bf16: bf16 storage, scores, softmax statistics and every sum accumulated
 *     in fp32, bf16 results rounded to nearest even; where a softmax weight
 *     multiplies a bf16 row (the value sums, and the dense tiles' products of
 *     weights or score gradients with K, Q or dO) the weight is rounded to
 *     bf16 first, kept as a bf16 hi + lo pair where many large weights are
 *     summed or two such sums are subtracted (a relative error of about 2^-9
 *     per single-part weight); the softmax denominator sums the fp32 weights.
 *     GT_F32 keeps every weight in fp32.
 *   - CSR: rowptr int64[n+1] with rowptr[0] = 0 and rowptr[n] = nnz; col
 *     int32[nnz], 0 <= col < n, strictly increasing inside each row.  Row i
 *     attends to the columns of row i (its out-neighbours).  The library adds
 *     no self-loops: condition C1 of §3.2 (each node attends to itself) is the
 *     caller's to add.  n < 2^31, nnz < 2^32.
 */
#ifndef GT_H
#define GT_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gt_status;
#define GT_OK 0
#define GT_ERR_INVALID_ARG (-1)  /* null pointer, negative size, inconsistent sizes */
#define GT_ERR_UNSUPPORTED (-2)  /* d, H, T or dtype outside the supported set */
#define GT_ERR_UNSORTED (-3)     /* CSR row not strictly increasing (or rowptr decreasing) */
#define GT_ERR_DUPLICATE (-4)    /* repeated column inside a CSR row */
#define GT_ERR_OUT_OF_RANGE (-5) /* column outside [0, n), or rowptr[0] != 0 / rowptr[n] != nnz */
#define GT_ERR_WORKSPACE (-6)    /* workspace smaller than the size query returned */
#define GT_ERR_HIP (-7)          /* a HIP runtime call failed; gt_last_error() has its text */

typedef int32_t gt_dtype;
#define GT_F32 0
#define GT_BF16 1

/* Version of this ABI (incremented on any incompatible change). */
int32_t gt_abi_version(void);
/* Static text for a status code. */
const char* gt_status_string(gt_status status);
/* Text of the last error raised on the calling thread ("" if none). */
const char* gt_last_error(void);

/* ------------------------------------------------------------------------ */
/* CSR validation (the input convention above).                              */
/* ------------------------------------------------------------------------ */

size_t gt_validate_csr_workspace_size(void);
/* SYNC.  GT_OK, or the first of GT_ERR_OUT_OF_RANGE, GT_ERR_UNSORTED,
 * GT_ERR_DUPLICATE found on the device.  Never reads outside rowptr[0..n] and,
 * for rows whose rowptr bounds are inside [0, nnz], col[rowptr[i]..rowptr[i+1]). */
gt_status gt_validate_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, void* ws,
                          size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Cluster reordering, §3.3.                                                 */
/* ------------------------------------------------------------------------ */
/* Label propagation on the CSR (self-loops ignored), then a stable order by
 * (label, -degree, id).  With k_t = seed + (t+1)*0x9E3779B97F4A7C15 (mod 2^64)
 * and mix64 the SplitMix64 output function, sweep t moves every active node
 * (the top three bits of mix64(v ^ k_t ^ 0xD6E8FEB86659FD93) not all zero) to
 * the most frequent label among its neighbours, keeping its own label when
 * that is among the most frequent and otherwise taking the smallest
 * (mix64(label ^ k_t), label).  Propagation stops early when no node would
 * move.  The result is a pure function of (CSR, iters, seed).
 *   perm  int32[n]  out: perm[new] = old
 *   iperm int32[n]  out: iperm[old] = new
 *   labels int32[n] out (may be NULL): final label of each (old) node
 *   sweeps_done (host, may be NULL): SYNC if given; sweeps that changed a label.
 * The CSR must satisfy the input convention (see gt_validate_csr); it is
 * validated here first (SYNC) and an invalid CSR returns its error code.
 * Every kernel runs on `stream`. */
size_t gt_reorder_workspace_size(int64_t n, int64_t nnz);
gt_status gt_reorder(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t iters,
                     uint64_t seed, int32_t* perm, int32_t* iperm, int32_t* labels, int32_t* sweeps_done,
                     void* ws, size_t ws_bytes, hipStream_t stream);
/* gt_reorder with the rows of each sweep spread over `stream` and n_side
 * further streams of the caller's, so that the sweep's row classes (short
 * rows, long rows, rows of 65 to 4096 entries) run side by side.
 *   side_streams (host) hipStream_t[n_side], n_side in [0, 2]: non-null,
 *     distinct, not `stream`, on stream's device;
 *   events (host) hipEvent_t[n_side + 1]: distinct events of the caller's on
 *     stream's device, which the call records and waits on to order the
 *     streams (timing not needed); no other work may record them until the
 *     call has returned.
 * The side streams are used only when the rows of more than 64 entries hold
 * at least a quarter of the entries (else the short rows' kernel dominates a
 * sweep and the others gain nothing beside it).
 * Same results, workspace and errors as gt_reorder (which is this call with
 * n_side = 0); a bad side-stream or event argument is GT_ERR_INVALID_ARG
 * before anything is enqueued.  When the call returns, every later call on
 * `stream` runs after all of its work; work enqueued on the side streams
 * before the call runs before the call's work there. */
gt_status gt_reorder_streams(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t iters,
                             uint64_t seed, int32_t* perm, int32_t* iperm, int32_t* labels, int32_t* sweeps_done,
                             void* ws, size_t ws_bytes, hipStream_t stream, const hipStream_t* side_streams,
                             const hipEvent_t* events, int32_t n_side);

/* ------------------------------------------------------------------------ */
/* Relabelling, §3.3 (the layout is reorganised by cluster).                 */
/* ------------------------------------------------------------------------ */
/* Row r of the output holds {iperm[c] : c in row perm[r]}, ascending.
 * rowptr_out int64[n+1], col_out int32[nnz].  perm/iperm must be inverse
 * permutations of [0, n) (not checked).  SYNC: the CSR is validated first and
 * an invalid CSR returns its error code. */
size_t gt_permute_workspace_size(int64_t n, int64_t nnz);
gt_status gt_permute_csr(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, const int32_t* perm,
                         const int32_t* iperm, int64_t* rowptr_out, int32_t* col_out, void* ws, size_t ws_bytes,
                         hipStream_t stream);
/* gt_permute_csr that also returns, for every edge e of the output,
 * src_pos[e] = its position in the input CSR (int32[nnz], device), so that
 * per-edge values (a bias, §2.1 Eq. (3)) follow their edges:
 * gt_gather_rows(nnz, bytes per edge, values, src_pos, values_out).
 * nnz < 2^31.  Same validation and errors as gt_permute_csr. */
size_t gt_permute_edges_workspace_size(int64_t n, int64_t nnz);
gt_status gt_permute_csr_edges(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col,
                               const int32_t* perm, const int32_t* iperm, int64_t* rowptr_out, int32_t* col_out,
                               int32_t* src_pos, void* ws, size_t ws_bytes, hipStream_t stream);
/* dst row r = src row perm[r] (rows of row_bytes bytes, a multiple of 4). */
gt_status gt_gather_rows(int64_t n, int64_t row_bytes, const void* src, const int32_t* perm, void* dst,
                         hipStream_t stream);
/* dst row perm[r] = src row r (the inverse of gt_gather_rows). */
gt_status gt_scatter_rows(int64_t n, int64_t row_bytes, const void* src, const int32_t* perm, void* dst,
                          hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Tile plan, §3.4 (cluster sparsity; transfer threshold).                   */
/* ------------------------------------------------------------------------ */
/* R = ceil(n/T) tile rows/columns.  Tile (I, J) holds the edges (i, j) with
 * i/T = I, j/T = J; cnt is their number, area = min(T, n-I*T)*min(T, n-J*T).
 * The tile is dense iff cnt >= 1 and cnt*10^6 >= tau_ppm*area (exact integer
 * comparison).  T in {64, 128}; R <= 16384. */
/* Remainder rows (columns) with more than GT_LONG_ROW edges are processed by
 * a whole workgroup each instead of a slice of a wavefront; the plan lists them. */
#define GT_LONG_ROW 256

typedef struct gt_tiles {
    int64_t n;             /* nodes */
    int32_t T;             /* tile edge */
    int32_t reserved;
    int64_t n_row_tiles;   /* R */
    int64_t n_dense;       /* dense tiles */
    int64_t nnz_sparse;    /* edges outside the dense tiles */
    int64_t n_long_rows;   /* remainder rows with more than GT_LONG_ROW edges */
    int64_t n_long_cols;   /* remainder columns with more than GT_LONG_ROW edges */
    int64_t* tile_rowptr;  /* int64[R+1]: dense tiles of tile row I are [tile_rowptr[I], tile_rowptr[I+1]) */
    int32_t* tile_col;     /* int32[n_dense]: J of each dense tile, sorted by (I, J) */
    int32_t* tile_nnz;     /* int32[n_dense]: edges in the tile */
    uint32_t* tile_mask;   /* uint32[n_dense*T*T/32]: row-major bit mask; bit b of word w of local row r
                              marks column J*T + 32*w + b */
    int64_t* sp_rowptr;    /* int64[n+1]: remainder CSR (edges outside dense tiles, CSR order) */
    int32_t* sp_col;       /* int32[nnz_sparse] */
    int64_t* sp_colptr;    /* int64[n+1]: remainder transpose (rows ascending in each column) */
    int32_t* sp_row;       /* int32[nnz_sparse] */
    int64_t* tileT_ptr;    /* int64[R+1]: dense tiles of tile column J, sorted by (J, I) */
    int32_t* tileT_idx;    /* int32[n_dense]: index into the (I, J)-sorted list */
    int32_t* long_rows;    /* int32[n_long_rows]: ascending */
    int32_t* long_cols;    /* int32[n_long_cols]: ascending */
    /* Edge positions (optional, for a per-edge bias on a plan with dense
     * tiles): when non-NULL at gt_build_tiles they are filled, and the input
     * CSR must have nnz < 2^31.  Positions are those of the input CSR. */
    int32_t* sp_pos;       /* int32[nnz_sparse]: position of each remainder edge */
    int32_t* tile_pos;     /* int32[n_dense*T]: [k*T + r] = position of the first edge of local row r of dense
                              tile k; the row's edges in the tile are the next popcount(mask row r) positions
                              (0 where the row has none) */
} gt_tiles;

size_t gt_tiles_workspace_size(int64_t n, int64_t nnz, int32_t T);
/* SYNC.  Validates the CSR, then sets plan->n, T, n_row_tiles, n_dense,
 * nnz_sparse, n_long_rows and n_long_cols (host struct; array pointers are
 * left untouched). */
gt_status gt_tiles_count(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T,
                         uint32_t tau_ppm, gt_tiles* plan, void* ws, size_t ws_bytes, hipStream_t stream);
/* Fills every array of *plan.  The size fields must be those set by
 * gt_tiles_count for the same arguments and every array pointer a caller
 * allocation of the size given above.  The CSR is the one gt_tiles_count
 * validated.  gt_tiles_count leaves in its workspace a record of its
 * arguments and a checksum of its count results.  SYNC: this call reads that
 * record back and recomputes the checksum; when ws holds the record of a
 * gt_tiles_count with the same arguments and the checksum still matches, the
 * counts are taken from there, otherwise (another workspace, or one written to
 * in between) they are counted again.  The record is cleared once read.
 * Either way the plan is the same. */
gt_status gt_build_tiles(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t T,
                         uint32_t tau_ppm, gt_tiles* plan, void* ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* The paper's lossy reformation, §3.4 (cluster sparsity, transfer strategy). */
/* ------------------------------------------------------------------------ */
/* An opt-in rewrite of the (clustered) graph into E'; the attention calls then
 * run exactly on E'.  With c = ceil(n/k), cluster (I, J) holds the edges (i, j)
 * with i/c = I, j/c = J; cnt counts them, area = rows(I)*rows(J) with
 * rows(I) = min(c, n - I*c).  The cluster is transferred iff cnt >= 1 and
 * cnt*den < num*area (density below num/den, exact).  In a transferred cluster
 * the self-loops stay and its other `moved` edges are replaced by
 * m = ceil(moved / d_b^2) full d_b x d_b sub-blocks: the cluster is cut into
 * d_b x d_b blocks from its corner (clipped at its edge) and the m blocks that
 * held the most moved edges are chosen, ties to the smaller (block row, block
 * column).  Edges of other clusters are kept.  rowptr_out int64[n+1] and
 * col_out int32[cap] receive E' (sorted, no duplicates); *nnz_out (host) its
 * size.  cap must be at least gt_ecr_max_nnz(nnz, k, d_b); 1 <= k <= 64,
 * 1 <= d_b <= 256.  *n_transferred (host, may be NULL) counts the transferred
 * clusters.  SYNC: validates the CSR first and reads back counts. */
int64_t gt_ecr_max_nnz(int64_t nnz, int32_t k, int32_t d_b);
size_t gt_ecr_workspace_size(int64_t n, int64_t nnz, int32_t k, int32_t d_b);
gt_status gt_ecr_compact(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t k, int32_t d_b,
                         uint64_t num, uint64_t den, int64_t* rowptr_out, int32_t* col_out, int64_t cap,
                         int64_t* nnz_out, int32_t* n_transferred, void* ws, size_t ws_bytes, hipStream_t stream);

/* Auto Tuner of the transfer threshold, §3.4 (hyperparameter modeling).  Host
 * only (no device memory, no stream).  The caller owns the state.  Running
 * loss F_t = 0.9 F_{t-1} + 0.1 L_t (F_0 = L_0); loss descent rate
 * LDR_t = (F_t - F_{t-1}) / et_t (et_t the epoch's time); the threshold walks the
 * ladder {0, bG, 1.5 bG, 5 bG, 7 bG, 10 bG, 1}, bG = nnz/n^2, each capped at 1,
 * starting at bG.  At epoch t, once LDR_{t-delta} exists and delta epochs have
 * passed since the last change, LDR_t >= LDR_{t-delta} moves one rung up and
 * LDR_t < LDR_{t-delta} one rung down (clamped).  Each rung is the exact
 * fraction num/den to pass to gt_ecr_compact. */
#define GT_AUTOTUNER_RUNGS 7
#define GT_AUTOTUNER_HISTORY 64
typedef struct gt_autotuner {
    double F;                             /* running loss */
    double ldr[GT_AUTOTUNER_HISTORY];     /* LDR_t at t mod GT_AUTOTUNER_HISTORY */
    int64_t t;                            /* index of the last epoch fed (-1 before the first) */
    int64_t last_change;                  /* epoch of the last rung change (0 at the start) */
    int32_t level;                        /* current rung, 0 .. GT_AUTOTUNER_RUNGS-1 */
    int32_t delta;                        /* comparison distance, 1 .. GT_AUTOTUNER_HISTORY-1 */
    uint64_t num[GT_AUTOTUNER_RUNGS];     /* ladder numerators */
    uint64_t den[GT_AUTOTUNER_RUNGS];     /* ladder denominators */
} gt_autotuner;
/* n >= 1, 0 <= nnz < 2^32 (the graph bG refers to). */
gt_status gt_autotuner_init(gt_autotuner* state, int64_t n, int64_t nnz, int32_t delta);
/* Feed epoch t's loss (finite) and time (> 0); returns the rung for the next
 * epoch in *level and its threshold *num / *den (each output may be NULL). */
gt_status gt_autotuner_step(gt_autotuner* state, double loss, double epoch_seconds, int32_t* level, uint64_t* num,
                            uint64_t* den);

/* ------------------------------------------------------------------------ */
/* Interleave decision, §3.2 (conditions C1-C3 for the sparse pattern alone). */
/* ------------------------------------------------------------------------ */
/* The CSR is read as an undirected graph (symmetric); reach follows out-edges.
 *   C1: every row holds its self-loop (exact): missing_self_loops == 0.
 *   C2: a Hamiltonian path, confirmed by Dirac's condition on min_degree (the
 *       minimum degree without self-loops): 2*min_degree >= n for n >= 3; n <= 1
 *       holds; n = 2 holds iff min_degree >= 1; otherwise 0 (not confirmed).
 *   C3: every node within L hops of every node.  Breadth-first search from
 *       node 0 cut at depth L+1 gives ecc_root and reached (nodes within the
 *       cut).  ecc_root > L or reached < n: 0.  2*ecc_root <= L: 1.  Otherwise a
 *       second search from the smallest-id node at depth ecc_root gives ecc_far:
 *       ecc_far > L or a node beyond the cut: 0, else -1 (undetermined).
 * c1, c2, c3 are 1 (holds), 0 (does not) or -1 (undetermined); use_sparse is 1
 * iff all three are 1, else a fully connected layer should be interleaved.
 * ecc_far is -1 when the second search is not run.  levels (int32[n], may be
 * NULL) receives the first search's depths (-1 beyond the cut).  0 <= L < 2^30.
 * SYNC: validates the CSR first and reads back a count per depth. */
typedef struct gt_interleave_report {
    int64_t n;
    int64_t missing_self_loops;
    int64_t min_degree;
    int64_t reached;
    int32_t ecc_root;
    int32_t ecc_far;
    int32_t c1;
    int32_t c2;
    int32_t c3;
    int32_t use_sparse;
} gt_interleave_report;
size_t gt_interleave_workspace_size(int64_t n);
gt_status gt_interleave_check(int64_t n, int64_t nnz, const int64_t* rowptr, const int32_t* col, int32_t L,
                              gt_interleave_report* report, int32_t* levels, void* ws, size_t ws_bytes,
                              hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Neighbourhood softmax attention, §3.2, over a plan (reordered index space).*/
/* ------------------------------------------------------------------------ */
/* For each node i and head h, over j in N(i) (the dense tiles plus the remainder):
 *   s_ij = scale*<Q[i,h],K[j,h]>, LSE[i,h] = log sum_j exp(s_ij),
 *   O[i,h] = sum_j exp(s_ij - LSE[i,h]) V[j,h].
 * An empty row gives O = 0 and LSE = -inf.  `plan` is a host struct built by
 * gt_build_tiles (its arrays stay valid until the call has run). */
size_t gt_sparse_attn_fwd_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
gt_status gt_sparse_attn_fwd(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                             const void* K, const void* V, float scale, void* O, float* LSE, void* ws,
                             size_t ws_bytes, hipStream_t stream);

/* Backward for an upstream gradient dO, given LSE of the forward:
 *   P_ij = exp(s_ij - LSE_i), dP_ij = <dO_i, V_j>, D_i = sum_j P_ij dP_ij,
 *   dS_ij = P_ij (dP_ij - D_i),
 *   dQ_i = scale sum_j dS_ij K_j, dK_j = scale sum_i dS_ij Q_i, dV_j = sum_i P_ij dO_i.
 * D_i equals <dO_i, O_i> for the exact output O; it is formed from the edges
 * because the stored O is rounded to the feature dtype, so O is not an input.
 * dK and dV are gathered per column (no atomics): results are bitwise
 * reproducible for a fixed plan. */
size_t gt_sparse_attn_bwd_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
gt_status gt_sparse_attn_bwd(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                             const void* K, const void* V, const void* dO, const float* LSE, float scale, void* dQ,
                             void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream);

/* The backward in its two halves, for callers that schedule them apart (the
 * combined call above is rows then cols).
 * _rows: dQ (row-owned) and the row statistic Dstat[i, h] = D_i
 *        (fp32 [n, H], written here, read by _cols).
 * _cols: dK and dV (column-owned), from Dstat of the _rows call. */
size_t gt_sparse_attn_bwd_rows_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
gt_status gt_sparse_attn_bwd_rows(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                                  const void* K, const void* V, const void* dO, const float* LSE, float scale,
                                  void* dQ, float* Dstat, void* ws, size_t ws_bytes, hipStream_t stream);
size_t gt_sparse_attn_bwd_cols_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
gt_status gt_sparse_attn_bwd_cols(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                                  const void* K, const void* V, const void* dO, const float* LSE, const float* Dstat,
                                  float scale, void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream);

/* With a per-edge additive bias, §2.1 Eq. (3) (the graph's structural
 * encoding, stored in the attention's sparse layout per §3.3):
 *   s_ij = scale*<Q[i,h],K[j,h]> + bias[e,h],
 * e the position of edge (i, j) in the input CSR the plan was built from, on
 * remainder edges and dense-tile edges alike; bias and dbias are fp32 [nnz, H]
 * device arrays (nnz = nnz_sparse + the dense tiles' edges, < 2^31).  The
 * backward also writes dbias[e,h] = dS_ij (every entry written).  A plan with
 * dense tiles must carry sp_pos and tile_pos (gt_build_tiles fills them when
 * given); for a plan without dense tiles the remainder is the input CSR and
 * they may be NULL.  On dense tiles the bias is laid out per tile in the
 * workspace before the tile kernels run, and their dS written back to dbias
 * at the edges' positions.
 * csc_pos (int32[nnz_sparse], device) comes from gt_edge_map for this plan:
 * csc_pos[c] is the input-CSR position of the c-th entry of sp_row (the
 * remainder position where the plan has no sp_pos). */
size_t gt_edge_map_workspace_size(const gt_tiles* plan);
gt_status gt_edge_map(const gt_tiles* plan, int32_t* csc_pos, void* ws, size_t ws_bytes, hipStream_t stream);
size_t gt_sparse_attn_fwd_bias_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
size_t gt_sparse_attn_bwd_bias_workspace_size(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype);
gt_status gt_sparse_attn_fwd_bias(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* Q,
                                  const void* K, const void* V, const float* bias, float scale, void* O, float* LSE,
                                  void* ws, size_t ws_bytes, hipStream_t stream);
gt_status gt_sparse_attn_bwd_bias(const gt_tiles* plan, const int32_t* csc_pos, int32_t H, int32_t d, gt_dtype dtype,
                                  const void* Q, const void* K, const void* V, const float* bias, const void* dO,
                                  const float* LSE, float scale, void* dQ, void* dK, void* dV, float* dbias,
                                  void* ws, size_t ws_bytes, hipStream_t stream);

/* Measurement only (not part of the method): the remainder forward's data
 * movement with no arithmetic.  Every remainder edge (i, j) of a row with at
 * most GT_LONG_ROW edges reads row j of A and of B ([n, H, d], dtype) with the
 * lanes and edge walk of gt_sparse_attn_fwd; the values are only XORed.  Used
 * to time the rate the gather path allows for a plan.  sink: device uint32[1],
 * written only if the XOR of a lane's words hits a fixed constant (ignore it). */
gt_status gt_gather_probe(const gt_tiles* plan, int32_t H, int32_t d, gt_dtype dtype, const void* A, const void* B,
                          uint32_t* sink, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Full softmax attention, §2.1 Eq. (1) (the interleaved dense layer of §3.2).*/
/* ------------------------------------------------------------------------ */
/* Same formulas with N(i) = all n nodes; same dtype / d / H support as the
 * sparse calls.  No n x n buffer is formed. */
gt_status gt_dense_attn_fwd(int64_t n, int32_t H, int32_t d, gt_dtype dtype, const void* Q, const void* K,
                            const void* V, float scale, void* O, float* LSE, hipStream_t stream);
size_t gt_dense_attn_bwd_workspace_size(int64_t n, int32_t H, int32_t d, gt_dtype dtype);
/* Backward of the full layer given O and LSE of its forward.  Here every
 * weight is about 1/n, so D_i = <dO_i, O_i> is taken from the given O. */
gt_status gt_dense_attn_bwd(int64_t n, int32_t H, int32_t d, gt_dtype dtype, const void* Q, const void* K,
                            const void* V, const void* O, const void* dO, const float* LSE, float scale, void* dQ,
                            void* dK, void* dV, void* ws, size_t ws_bytes, hipStream_t stream);
/* For callers that cannot allocate (code under stream capture, tight serving
 * loops, harnesses that forbid allocation): gt_dense_attn_bwd with its scratch
 * (the row statistic D, fp32 [n, H]) in a device array of the library's own
 * instead of a caller workspace.  It allocates and frees nothing.  The array
 * holds gt_dense_attn_bwd_noalloc_max_bytes() = 64 MiB; n * H above 16,777,216
 * returns GT_ERR_UNSUPPORTED (use gt_dense_attn_bwd).  Each GPU the library
 * runs this on holds its own copy until the process ends; its device address
 * is looked up on the first call on that device.  The stream must belong to
 * the current device.  Every call on one GPU shares that GPU's array, so calls
 * that overlap on one GPU (other streams, other host threads) race: order them.
 * Nothing in the array needs clearing between calls (D is written before it is
 * read).  Results equal gt_dense_attn_bwd's bit for bit. */
size_t gt_dense_attn_bwd_noalloc_max_bytes(void);
gt_status gt_dense_attn_bwd_noalloc(int64_t n, int32_t H, int32_t d, gt_dtype dtype, const void* Q, const void* K,
                                    const void* V, const void* O, const void* dO, const float* LSE, float scale,
                                    void* dQ, void* dK, void* dV, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* GT_H */
