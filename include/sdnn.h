/*
 * sdnn.h -- C ABI of the MI355X (gfx950) sparse-weight x dense-activation product.
 *
 * The operator is the core of SparseDNN (Wang, arXiv 2101.07948): a sparse matrix
 * (pruned weights) times a dense matrix (activations), Sec. 2.2 and Sec. 3.2.2, with
 * a fused bias + element-wise activation epilogue (layer fusion, Sec. 3.1):
 *
 *     C[i][n] = act( sum_p W[i][c_p] * B[c_p][n] + bias[i] )
 *
 * It follows the paper's two-stage engine (Sec. 2.1, Sec. 3): a one-time preparation
 * stage (sdnn_plan_create: CSR validation, the greedy weight-row permutation of
 * Sec. 3.1.2 / Algorithm 1, and repacking of W into a per-matrix traversal-ordered
 * stream, Sec. 3.2.2) and a per-request execution stage (sdnn_spmm).
 *
 * Conventions shared by every entry point:
 *   - Every call returns an sdnn_status; no C++ exception crosses this boundary.
 *   - Host pointers are read during the call only and never retained.
 *   - Device pointers are raw HIP device addresses; "stream" is a hipStream_t passed
 *     as void* (NULL = the default stream).
 *   - Dense matrices are row-major with no padding: B is K x N (ld = N), C is M x N
 *     (ld = N).  Lanes of the GPU kernel run along N, so a PyTorch activation of
 *     shape (tokens, hidden) is B transposed.
 *   - CSR input: row_ptr[M+1] with row_ptr[0] = 0, non-decreasing, row_ptr[M] = nnz;
 *     col_idx[nnz] in [0, K), strictly increasing within each row (no duplicates);
 *     values[nnz] fp32.  Explicitly stored zeros count as nonzeros.
 *   - Inputs must be finite; results for NaN/Inf inputs are unspecified.
 */
#ifndef SDNN_H_
#define SDNN_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque plan; immutable after creation except for the launch shapes that
 * sdnn_plan_tune records. */
typedef struct sdnn_plan_s* sdnn_plan;

typedef enum {
  SDNN_OK = 0,
  SDNN_ERR_NULL = 1,   /* a required pointer is NULL */
  SDNN_ERR_DIM = 2,    /* negative or too-large size, or overlapping B/C/bias ranges */
  SDNN_ERR_CSR = 3,    /* malformed CSR: row_ptr, column range, unsorted/duplicate cols */
  SDNN_ERR_ALLOC = 4,  /* host or device allocation failed */
  SDNN_ERR_HIP = 5,    /* a HIP runtime call or kernel launch failed */
  SDNN_ERR_DEVICE = 6, /* plan used on a device other than the one it was created on */
  SDNN_ERR_INTERNAL = 7 /* the packed stream failed its own consistency check */
} sdnn_status;

/* Fused epilogue applied after the bias add (Sec. 3.1 layer fusion; GELU is the exact
 * erf form x * Phi(x), named in Sec. 5). */
typedef enum {
  SDNN_EPI_NONE = 0,
  SDNN_EPI_RELU = 1, /* max(x, 0) */
  SDNN_EPI_GELU = 2  /* 0.5 * x * (1 + erf(x / sqrt(2))) */
} sdnn_epilogue;

/* Options for sdnn_plan_create; pass NULL for the defaults {0, 1, 0, 0, NULL, 0, 0}.
 *   panel_rows:   rows per register panel.  0 (default) packs W four times, with
 *                 panels of 4, 12, 8 and 16 rows, and a fifth time with 32-row panels
 *                 for 128-column tiles unless tile_cols = 256.  sdnn_spmm picks one per
 *                 call: the 32-row panels (with 12 consumer waves per workgroup) when W
 *                 holds under 20 entries per 16 rows and 32 columns and their grid fills
 *                 the compute units; otherwise the fewest rounds of workgroups over the
 *                 compute units, then the most units busy, then the shortest panels
 *                 averaging at least 8 entries per 32 columns of W (4-row panels are not
 *                 used below 8); sdnn_plan_tune can replace that choice by a timed one,
 *                 and sdnn_plan_launch_shape reports it.  4, 8, 12 or 16 packs that
 *                 height only; 32 too, with tile_cols = 128 (else SDNN_ERR_DIM).
 *   permute:      1 = apply Algorithm 1 (default), 0 = identity order (ablation),
 *                 2 = panel-balancing order: rows, by nonzero count descending, each
 *                 go to the 4-row panel with the fewest nonzeros so far that has room,
 *                 so that every panel (and every 12-row panel) carries about the same
 *                 work.  3 = panel-union greedy: 4-row panels filled in turn, each
 *                 headed by the remaining row with the most nonzeros and continued
 *                 by the remaining row with the largest overlap with the union of
 *                 the panel's column sets so far (ties: more nonzeros, lower index).
 *                 4 = MinHash clustering (locality-sensitive hashing): rows sorted by
 *                 a 4-word MinHash signature of their column sets, then nonzeros
 *                 descending, then index.  5 = bin-then-greedy: rows binned by
 *                 floor(log2(nnz + 1)), densest bin first, Algorithm 1 within each bin.
 *   out_permuted: 0 (default) = C row i is output row i; 1 = C is written in the
 *                 plan's permuted row order, C row i = output row perm[i] (Sec. 3.1.2:
 *                 the rows stay permuted and the next layer's columns compensate).
 *                 The bias is always given in the original row order.
 *   split_chunks: 0 (default) = no K-segments.  S > 0 cuts K into segments of S chunks
 *                 (S * k_chunk rows of B; nseg = ceil(ceil(K / k_chunk) / S) segments)
 *                 so that sdnn_spmm_split / sdnn_conv3x3_split can give each run of
 *                 consecutive segments of a tile its own workgroup (the split-K tiling
 *                 of Sec. 3.2.2 extended across workgroups); small S leaves the call
 *                 more choice, at the cost of more stored groups.  Such plans also serve sdnn_spmm and
 *                 sdnn_conv3x3, unsplit.  Negative: SDNN_ERR_DIM.
 *   in_perm:      NULL (default) = B row c is input feature c; otherwise K int32 (host,
 *                 read during the call only), a permutation of 0..K-1 giving the order
 *                 of B's rows: B row i holds input feature in_perm[i].  Pass the
 *                 previous layer's perm when that layer used out_permuted = 1.
 *                 Not a permutation: SDNN_ERR_DIM.
 *   grouping:     which rows share a panel.  The plan's permutation (permute) is what
 *                 sdnn_plan_get_perm reports and what out_permuted stores by in every
 *                 case; the panels are either consecutive rows of it (1) or balanced
 *                 panels (2: the panel-balancing rule of permute = 2 applied to W's
 *                 rows), each row still summing its entries in ascending column order,
 *                 so C is bit-identical either way.  0 (default) = the library's
 *                 choice, at present balanced panels: the panels of a workgroup advance
 *                 together through the staged chunks of B, so the heaviest panel, and
 *                 the one whose nonzeros bunch into the fewest chunks, set the pace.
 *                 Outside 0..2: SDNN_ERR_DIM.
 *   tile_cols:    columns of C per workgroup tile (the microkernel's output tile width,
 *                 Sec. 3.2.2).  0 (default) = the plan holds its stream for tiles of 256
 *                 columns (4 per lane, one workgroup per compute unit) and for tiles of 128
 *                 (2 per lane, half the LDS ring, two workgroups per compute unit), and
 *                 sdnn_spmm picks one per call (sdnn_plan_launch_tile reports which);
 *                 256 = 256-column tiles only (half the device memory for the streams);
 *                 128 = 128-column tiles wherever the call allows them.  128-column tiles
 *                 serve sdnn_spmm and sdnn_spmm_split with N % 4 == 0 and 16-byte aligned
 *                 B and C; convolutions and other calls use 256.  Other values:
 *                 SDNN_ERR_DIM. */
typedef struct {
  int32_t panel_rows;
  int32_t permute;
  int32_t out_permuted;
  int32_t split_chunks;
  const int32_t* in_perm;
  int32_t grouping;
  int32_t tile_cols;
} sdnn_plan_opts;

/* Plan statistics (of the first packing; the tall_* fields describe the second one, the
 * mid_* fields the third, the tallest_* fields the fourth and the deep_* fields the fifth,
 * or are 0 when the plan holds fewer packings).
 *   panels:       number of row panels (ceil(M / panel_rows)).
 *   packed_bytes: device bytes of every packed weight stream and its indexes.
 *   rho:          nnz / sum over panels of |union of the panel rows' column sets|,
 *                 the reuse an ideal panel kernel gets per staged B row (>= 1).
 *   fill:         nnz / stored stream entries (1.0 = no padding).
 *   k_chunk:      rows of B per LDS staging slot.
 *   splits:       K-segments of a plan created with split_chunks > 0 (else 0); the
 *                 workspace of a K-split call holds splits * M * N floats. */
typedef struct {
  int32_t M, K;
  int64_t nnz, panels, packed_bytes;
  double rho, fill;
  int32_t panel_rows, k_chunk;
  int32_t tall_panel_rows, splits;
  double tall_rho, tall_fill;
  int32_t out_permuted, in_permuted;  /* the plan's options (in_permuted: in_perm given) */
  int32_t mid_panel_rows, packings;   /* third packing's height (0: none); packings held */
  double mid_rho, mid_fill;
  int32_t grouping, tile_cols;        /* panel grouping used: 1 consecutive rows of perm,
                                         2 balanced panels (see sdnn_plan_opts.grouping);
                                         the tile_cols option the plan was created with */
  int32_t tallest_panel_rows, reserved2;  /* fourth packing's height (0: none) */
  double tallest_rho, tallest_fill;
  int32_t deep_panel_rows, reserved3;     /* fifth packing's height (0: none) */
  double deep_rho, deep_fill;
} sdnn_plan_info_t;

/* Greedy weight-row permutation (Sec. 3.1.2, Algorithm 1), host only, no GPU needed.
 * perm_out[i] is the original row placed at position i (gather convention:
 * W_perm[i] = W[perm_out[i]]).  First pick: most nonzeros (ties: lower index); each
 * next pick: the remaining row with the largest |cols(prev) ∩ cols(x)| (ties: more
 * nonzeros, then lower index).  perm_out has M entries, caller-owned.
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM, SDNN_ERR_CSR, SDNN_ERR_ALLOC. */
sdnn_status sdnn_reorder_rows(const int32_t* row_ptr, const int32_t* col_idx, int32_t M,
                              int32_t K, int32_t* perm_out);

/* The row order a plan with option `permute` uses (see sdnn_plan_opts), host only, no
 * GPU needed: 0 identity, 1 Algorithm 1 (as sdnn_reorder_rows), 2 panel-balancing,
 * 3 panel-union greedy, 4 MinHash clustering, 5 bin-then-greedy (see sdnn_plan_opts).
 * Sec. 3.1.2 notes that other reorderings (hashing, clustering) performed comparably
 * to Algorithm 1; orders 2-5 are such alternatives.  perm_out[i] is the original row
 * placed at position i; M entries, caller-owned.
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM (negative sizes, permute outside 0..5),
 * SDNN_ERR_CSR, SDNN_ERR_ALLOC. */
sdnn_status sdnn_row_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                           int32_t permute, int32_t* perm_out);

/* Preparation stage (Sec. 2.1, Sec. 3.1.2, Sec. 3.2.2).  Validates the host CSR,
 * computes the row permutation, packs W into the kernel's traversal-ordered stream
 * and uploads it to the current HIP device.  The caller keeps ownership of the CSR
 * arrays (they are copied).  The plan owns its device memory and is bound to the
 * device current at creation.  values may be NULL only when nnz = 0.  Limits: K at most
 * 2^19 = 524288 (16384 staging chunks of 32 rows: the stream's chunk fields), and at
 * most 2^31 - 1 stored stream entries; beyond either, SDNN_ERR_DIM.
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM, SDNN_ERR_CSR, SDNN_ERR_ALLOC, SDNN_ERR_HIP. */
sdnn_status sdnn_plan_create(const int32_t* row_ptr, const int32_t* col_idx,
                             const float* values, int32_t M, int32_t K,
                             const sdnn_plan_opts* opts, sdnn_plan* out);

/* Host-only self-check of the preparation stage (no GPU needed): validates the CSR,
 * computes the permutation and packs the stream exactly as sdnn_plan_create does,
 * then re-walks the stream and checks that every stored entry appears exactly once,
 * in its row's panel and K-chunk, in ascending column order, with unchanged weight
 * bits and a column offset inside its chunk.  On success fills *info if non-NULL.
 * Errors: as sdnn_plan_create, plus SDNN_ERR_INTERNAL if the stream is inconsistent. */
sdnn_status sdnn_plan_check_host(const int32_t* row_ptr, const int32_t* col_idx,
                                 const float* values, int32_t M, int32_t K,
                                 const sdnn_plan_opts* opts, sdnn_plan_info_t* info);

/* Copies the plan's permutation (M int32, host memory) to perm_out. */
sdnn_status sdnn_plan_get_perm(sdnn_plan p, int32_t* perm_out);

/* Fills *out with the plan's statistics. */
sdnn_status sdnn_plan_info(sdnn_plan p, sdnn_plan_info_t* out);

/* Execution stage (Sec. 3.2.2): C = act(W * B + bias), enqueued on `stream`.
 *   B:    device, K x N row-major fp32, read only.
 *   C:    device, M x N row-major fp32, written once, in the ORIGINAL row order.
 *   N:    columns of B and C, 0 <= N < 2^29 (N = 0 or M = 0 is a no-op); larger N gives
 *         SDNN_ERR_DIM, since the kernels address a row of B or C with 32-bit byte
 *         offsets.
 *   bias: device, M fp32 in original row order, or NULL (treated as zeros).
 *   With out_permuted plans, C row i is output row perm[i] (see sdnn_plan_opts); with
 *   in_perm plans, B's rows are in that order.
 * Asynchronous: no allocation, no synchronisation, no pointer retained, so a call may
 * be captured in a HIP graph and replayed.  A plan may be used from several streams at
 * once.  B must not overlap C or bias; the bias may
 * not overlap C (SDNN_ERR_DIM).  Device faults surface at the caller's next sync.
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM, SDNN_ERR_DEVICE, SDNN_ERR_HIP. */
sdnn_status sdnn_spmm(sdnn_plan p, const float* B, float* C, int32_t N, const float* bias,
                      sdnn_epilogue epi, void* stream);

/* K-split execution (Sec. 3.2.2 splits K into tiles that a block walks in turn; here runs
 * of a tile's K-segments also go to different workgroups, which fills the device when
 * M * ceil(N / 256) alone gives too few workgroups).  Same result contract, layouts and
 * stream semantics as sdnn_spmm; the plan must have been created with split_chunks > 0.
 *   splits:           workgroups along K.  0 = the library's choice for this N (the count
 *                     sdnn_plan_tune measured fastest at this N, else a cost model of
 *                     staging rounds against the reduction's traffic); k > 0 = runs of
 *                     ceil(nseg / k) consecutive segments each (at most nseg runs, nseg =
 *                     sdnn_plan_info's `splits`); sdnn_plan_split_runs reports the count.
 *                     Negative: SDNN_ERR_DIM.
 * With R runs (R > 1), each workgroup writes its run's partial product (no bias, no
 * epilogue) to workspace[r][row][n]; a second kernel on the same stream sums the runs in
 * order r = 0, 1, ..., adds the bias and applies epi into C.  Results can differ from
 * sdnn_spmm in rounding only (another summation order); they depend on nothing but
 * W, B, bias, epi and the run boundaries (R and split_chunks).
 *   workspace:        device, at least nseg * M * N fp32, 16-byte aligned, clear of B, C
 *                     and bias; scratch of this call only (its contents afterwards are
 *                     unspecified).  Not touched, and may be NULL, when R = 1: the call
 *                     is then sdnn_spmm.
 *   workspace_floats: its size in floats.
 * Errors: as sdnn_spmm, plus SDNN_ERR_DIM (plan without split_chunks, splits < 0,
 * workspace too small, misaligned or overlapping) and SDNN_ERR_NULL (workspace NULL
 * when the plan has more than one segment). */
sdnn_status sdnn_spmm_split(sdnn_plan p, const float* B, float* C, int32_t N, const float* bias,
                            sdnn_epilogue epi, int32_t splits, float* workspace,
                            int64_t workspace_floats, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): sdnn_spmm_split with the partial
 * products kept in a fixed scratch array that the library holds on every device it runs
 * on (16 Mi floats = 64 MiB per device, reserved when the library is loaded and held
 * until the process ends), so the call itself allocates nothing.  Same arguments,
 * result contract, run counts and kernels as sdnn_spmm_split without the workspace.
 *   Limit: R runs need R * M * N floats of scratch; beyond 16 Mi floats the call returns
 *   SDNN_ERR_DIM (use sdnn_spmm_split with a caller workspace instead).  With R = 1 it
 *   is sdnn_spmm and touches no scratch.
 * Every call on one device shares that device's scratch array: two such calls that
 * overlap in time on one device (different streams, or different host threads without
 * ordering) race and give unspecified results; calls ordered on one stream are safe.
 * The first call on a device looks the array's address up (no allocation); a caller
 * about to capture a graph should make one call on that device before capturing.
 * Errors: as sdnn_spmm_split, with SDNN_ERR_DIM for a scratch need above the limit. */
sdnn_status sdnn_spmm_split_noalloc(sdnn_plan p, const float* B, float* C, int32_t N,
                                    const float* bias, sdnn_epilogue epi, int32_t splits,
                                    void* stream);

/* The launch shape sdnn_spmm uses for this plan at N columns (the tuned one if
 * sdnn_plan_tune recorded one for N, else the rule described under panel_rows):
 * *panel_rows = the packing's panel height, *waves = consumer waves per workgroup
 * (either pointer may be NULL).  Host only; touches no device memory.
 * Errors: SDNN_ERR_NULL (p), SDNN_ERR_DIM (N <= 0 or M = 0). */
sdnn_status sdnn_plan_launch_shape(sdnn_plan p, int32_t N, int32_t* panel_rows, int32_t* waves);

/* The workgroups along K that sdnn_spmm_split runs for this plan at N columns when asked
 * for `splits` (0: the library's choice, see sdnn_spmm_split); 1 for a plan without
 * K-segments.  Host only.  Errors: SDNN_ERR_NULL (p or runs), SDNN_ERR_DIM (N <= 0, M = 0,
 * splits < 0). */
sdnn_status sdnn_plan_split_runs(sdnn_plan p, int32_t N, int32_t splits, int32_t* runs);

/* The tile width (columns of C per workgroup) sdnn_spmm uses for this plan at N columns
 * when B and C are 16-byte aligned and N % 4 == 0 (otherwise it is 256): the tuned one if
 * sdnn_plan_tune recorded one for N, else the plan's tile_cols option, else the library's
 * rule.  Host only.  Errors: SDNN_ERR_NULL (p or tile_cols), SDNN_ERR_DIM (N <= 0, M = 0). */
sdnn_status sdnn_plan_launch_tile(sdnn_plan p, int32_t N, int32_t* tile_cols);

/* Per-plan variant selection by timing (the paper's preparation stage chooses the best
 * kernel implementation per operator, Sec. 3.1, and autotunes the microkernel and the
 * split-K tiling factor per sparse matrix, Sec. 3.2.2): times sdnn_spmm at this N for every
 * packing the plan holds (panel height) with several consumer-wave counts per workgroup, on
 * each tile width the call allows (256 and 128 columns, see tile_cols), on the caller's B
 * (K x N) and C (M x N, overwritten with unspecified values), and records the fastest in
 * the plan; later sdnn_spmm calls with the same N use it (up to 8 N values are kept).  For
 * a plan with K-segments it then times sdnn_spmm_split at every workgroup count along K
 * (up to 32) in a workspace it allocates for the search and frees (skipped if that
 * allocation fails), and records the fastest, one meaning the unsplit call, for
 * sdnn_spmm_split calls with splits = 0 at this N.  Blocking (synchronises `stream`).
 * Must not run concurrently with any other call on the same plan.  Results of sdnn_spmm
 * do not depend on the shape.  On success *panel_rows and *waves (either may be NULL)
 * hold the chosen shape (sdnn_plan_launch_tile and sdnn_plan_split_runs report the rest).
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM (N <= 0, N >= 2^29, M = 0, B overlapping C, or a
 * plan of 32-row panels alone with N % 4 != 0 or B or C not 16-byte aligned),
 * SDNN_ERR_DEVICE, SDNN_ERR_HIP. */
sdnn_status sdnn_plan_tune(sdnn_plan p, const float* B, float* C, int32_t N, void* stream,
                           int32_t* panel_rows, int32_t* waves);

/* Sparse 3x3 convolution, stride 1, zero padding 1 (Sec. 3.2.3: direct convolution as
 * an SpMM whose dense operand is a virtual matrix built on the fly from the input; the
 * paper's convolution benchmark, Sec. 4.1, uses this filter size and padding):
 *     C[o][y][x][b] = act( sum_{i,ky,kx} F[o][i][ky][kx] * X[i][y+ky-1][x+kx-1][b]
 *                          + bias[o] )       (X is zero outside the image)
 *   p:    a plan created from the filters as an OC x (IC * 9) CSR whose column is
 *         i * 9 + ky * 3 + kx (M = OC, K = IC * 9), without in_perm.
 *   X:    device, IC x H x W x NB fp32 (channel, image row, image column, image),
 *         16-byte aligned, read only.
 *   C:    device, OC x H x W x NB fp32, same layout (a following layer takes it as its
 *         X), 16-byte aligned; with an out_permuted plan its channels are in perm order.
 *   NB:   images per call, a multiple of 4 (a lane's four columns are four images of
 *         one pixel).  H = 0, W = 0 or NB = 0 is a no-op.
 *   bias: device, OC fp32, or NULL.
 * Same stream, allocation and concurrency semantics as sdnn_spmm.
 * Errors: SDNN_ERR_NULL; SDNN_ERR_DIM (K not a multiple of 9, in_perm plan, NB % 4 != 0,
 * misaligned or overlapping buffers, H * W * NB * 4 >= 2^31); SDNN_ERR_DEVICE;
 * SDNN_ERR_HIP. */
sdnn_status sdnn_conv3x3(sdnn_plan p, const float* X, float* C, int32_t H, int32_t W,
                         int32_t NB, const float* bias, sdnn_epilogue epi, void* stream);

/* K-split variant of sdnn_conv3x3 (N = H * W * NB columns), with the workspace
 * contract of sdnn_spmm_split.  Errors: as sdnn_conv3x3 and sdnn_spmm_split. */
sdnn_status sdnn_conv3x3_split(sdnn_plan p, const float* X, float* C, int32_t H, int32_t W,
                               int32_t NB, const float* bias, sdnn_epilogue epi, int32_t splits,
                               float* workspace, int64_t workspace_floats, void* stream);

/* Frees the plan and its device memory.  NULL is a no-op. */
void sdnn_plan_destroy(sdnn_plan p);

/* Static, human-readable name of a status code. */
const char* sdnn_status_str(sdnn_status s);

/* Dense comparison kernel (the dense GEMM the paper measures its sparse kernels
 * against, Sec. 3.2.1 / Sec. 4.1): C = act(W * B + bias) with W dense M x K row-major
 * fp32 on the device, same layouts, epilogue and stream semantics as sdnn_spmm.
 * It is a measurement aid, not part of the sparse method.
 * Errors: SDNN_ERR_NULL, SDNN_ERR_DIM, SDNN_ERR_HIP. */
sdnn_status sdnn_dense_gemm(const float* W, const float* B, float* C, int32_t M, int32_t K,
                            int32_t N, const float* bias, sdnn_epilogue epi, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SDNN_H_ */
