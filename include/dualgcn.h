/*
 * dualgcn.h -- C ABI of the MI355X (gfx950) DualGCN aggregation library.
 *
 * The library computes the aggregation phase of a GCN layer, the sparse-dense
 * product Y = A X of the DualGCN paper (Sec. 1 and Sec. 2.1), scheduled by the
 * paper's dual-metric partition (Sec. 3.2) and run by two kernels, one for the
 * sparse region and one for the dense region of the partition (Sec. 3.3), and
 * the update phase X W of a layer (Sec. 1), also fused with the aggregation of the
 * layer before it; for training, the loss gradient and
 * the backward products of a layer; the values of other aggregators on the same
 * structure; and plans saved and loaded across runs.
 *
 * Conventions for every entry point
 *   - Pointers named *_h are host memory; every other array pointer is device
 *     memory on the current HIP device.  No entry point copies user arrays.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *     Work is enqueued on that stream.  Only dualgcn_partition,
 *     dualgcn_plan_load, dualgcn_plan_export, dualgcn_plan_save,
 *     dualgcn_aggregator_values and dualgcn_arw_patterns wait for the device
 *     (dualgcn_partition and dualgcn_plan_load for all but their last kernel).
 *   - Every function returns a dualgcn_status (0 = success).  Arguments are
 *     checked before the device is touched.  Outputs are undefined after an
 *     error.  No C++ exception crosses this interface.
 *   - Entry points may be called from several host threads at once (the
 *     library's shared state is locked; the last HIP error is per thread).
 *   - A plan may be used by one stream at a time.  Results do not depend on
 *     the launch order of the kernels: every output element is written by
 *     exactly one workgroup, in a fixed summation order (bit-reproducible).
 */
#ifndef DUALGCN_H
#define DUALGCN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------ status */

typedef enum dualgcn_status {
    DUALGCN_OK = 0,
    DUALGCN_ERR_INVALID_ARG = -1,  /* NULL pointer, size out of range, bad rational */
    DUALGCN_ERR_BAD_CSR = -2,      /* row pointers not monotone, rowptr[0] != 0,
                                      rowptr[n] != nnz, or a column outside [0, n) */
    DUALGCN_ERR_UNSUPPORTED = -3,  /* sizes the library does not handle (see each call) */
    DUALGCN_ERR_OOM = -4,          /* a device allocation failed (for tests, the environment
                                      variable DUALGCN_TEST_FAIL_ALLOC=N makes the N-th
                                      allocation after it is set fail) */
    DUALGCN_ERR_HIP = -5,          /* a HIP runtime call failed; see dualgcn_last_hip_error */
    DUALGCN_ERR_NO_DEVICE = -6     /* no usable HIP device */
} dualgcn_status;

/* Static text for a status code (never NULL). */
const char *dualgcn_status_str(int status);

/* hipError_t of the last failing HIP call made by the library in this thread (0 if none). */
int dualgcn_last_hip_error(void);

/* ------------------------------------------------------------------ inputs */

/*
 * A sparse matrix in CSR form (the adjacency A of Sec. 1; the degree metric of
 * Sec. 3.2 is read from its row pointers).  The arrays are BORROWED: they must
 * stay alive and unmodified for the lifetime of any plan built on them.
 *   n       rows = columns, 1 <= n < 2^31
 *   nnz     stored entries, 0 <= nnz <= 2^31 - 2^16 (int32 row pointers; larger
 *           matrices return DUALGCN_ERR_UNSUPPORTED)
 *   rowptr  int32[n+1], rowptr[0] = 0, non-decreasing, rowptr[n] = nnz
 *   col     int32[nnz], each in [0, n); order inside a row is free and
 *           duplicates are allowed (they add in the product and weight walks)
 *   val     float[nnz] entry values (any finite floats)
 */
typedef struct dualgcn_csr {
    int32_t n;
    int64_t nnz;
    const int32_t *rowptr;
    const int32_t *col;
    const float *val;
} dualgcn_csr;

enum { DUALGCN_FORCE_AUTO = 0, DUALGCN_FORCE_SPARSE = 1, DUALGCN_FORCE_DENSE = 2 };

/* alpha_num values that select an adaptive weight (see dualgcn_thresholds). */
#define DUALGCN_ALPHA_ADAPTIVE 0xFFFFFFFFu
#define DUALGCN_ALPHA_BALANCED 0xFFFFFFFEu

/*
 * Partition parameters, as exact rationals.
 *   alpha = alpha_num / alpha_den, the weight of density against degree in the
 *           hybrid metric H_v = alpha N_v + (1 - alpha) D_v (Sec. 3.2); the
 *           paper's default is 1/2.  Requires alpha_num <= alpha_den, den > 0.
 *           alpha_num = DUALGCN_ALPHA_ADAPTIVE asks for the adaptive weight of
 *           Sec. 3.2 ("Time Complexity and Overhead Analysis"), for which the
 *           paper gives no formula.  This library takes each metric's share of
 *           the total spread, alpha = Var(N) / (Var(N) + Var(D)) (population
 *           variances over all nodes), rounded down to a multiple of
 *           1 / alpha_den, and 1/2 (alpha_num = floor(alpha_den / 2)) when
 *           neither metric varies.  alpha_num = DUALGCN_ALPHA_BALANCED reads the
 *           variance analysis as balancing the two terms instead: alpha such that
 *           alpha sigma_N = (1 - alpha) sigma_D, i.e. alpha = sigma_D / (sigma_N +
 *           sigma_D) (population standard deviations), rounded down to a multiple
 *           of 1 / alpha_den; then both terms of H spread alike and equal spreads
 *           give the paper's default 1/2.  A metric that does not vary gets no
 *           weight (alpha = 0 when N is constant, 1 when D is), and 1/2 when
 *           neither varies.  The weight chosen is reported by dualgcn_plan_query.
 *   beta  = beta_num / beta_den, the threshold tau = mu_H + beta sigma_H of
 *           Eq. (1) (Sec. 3.3); the paper uses 1/2.  Requires den > 0.
 *   force_mode  DUALGCN_FORCE_AUTO applies Eq. (1); FORCE_SPARSE / FORCE_DENSE
 *           send every row to one kernel (the plan's order and K* are unchanged).
 * Numerators and denominators must be below 2^16.  A NULL pointer means
 * {1, 2, 1, 2, DUALGCN_FORCE_AUTO}.
 */
typedef struct dualgcn_thresholds {
    uint32_t alpha_num, alpha_den;
    uint32_t beta_num, beta_den;
    int32_t force_mode;
} dualgcn_thresholds;

/* ------------------------------------------------------------------ plan */

typedef struct dualgcn_plan dualgcn_plan;

/*
 * dualgcn_partition -- the dual-metric partition of Sec. 3.2 and Eq. (1).
 *
 * For every node v, `walks_per_node` (k) anonymous random walks of `walk_len`
 * (d) steps give S_v = sum over the walks of the number of distinct nodes seen
 * (start included), so the neighbour density of Theorem 1 is N_v = S_v / k.
 * A step moves to entry floor(r * deg / 2^32) of the current CSR row, r being
 * the 32-bit half (low for even s, high for odd s) of 64-bit word floor(s/2) mod 4
 * of Philox-4x64-10 (Salmon et al., SC'11) with counter (v, w, floor(s / 8), 0)
 * and key (seed, 0); an empty row keeps the walk in place.
 * D_v is the row length.  With alpha = p/q the hybrid metric is kept as the
 * exact integer K_v = q k H_v = p S_v + (q - p) k D_v.  The threshold key K* is
 * the least integer with K* >= mu_K + beta sigma_K (population statistics over
 * all n nodes, evaluated exactly in 128-bit integers), so row v is dense iff
 * K_v >= K* (Eq. (1), ties dense).  `perm` lists the nodes sorted by (K_v, v)
 * ascending; its first n_sparse entries form the sparse region.
 *
 * Requirements: 1 <= k, 1 <= d <= 255, k (d + 1) < 2^32 (S_v is 32-bit),
 * q k max(d + 1, nnz) < 2^63 and the moment sums must fit 128 bits (else
 * DUALGCN_ERR_UNSUPPORTED).  The CSR is
 * validated on the device first (DUALGCN_ERR_BAD_CSR).
 *
 * The plan owns one block of device memory of about 9 nnz + 28 n bytes (S, K,
 * perm, the processing order, a copy of the matrix with its rows in that order,
 * the sparse tasks, the dense-region schedule and the partial sums of split
 * rows), released by dualgcn_plan_destroy; a scratch block is allocated and
 * released inside the call.  The processing order keeps perm's split into the
 * sparse and the dense region; inside a region rows go by row-length octave,
 * then node id (balanced work, and the locality of the node numbering).  The
 * call waits for `stream` twice (to read the moment sums and the schedule sizes),
 * and once more with the adaptive weight (to read the moments of S and D).  It
 * returns while the last kernel, which writes the sorted copy of the matrix from
 * the CSR arrays, may still run on `stream`: every call that uses the plan orders
 * its work after it, on any stream, and dualgcn_plan_destroy waits for it.  The
 * CSR arrays must stay unchanged until then (they are borrowed for the plan's
 * lifetime in any case).  *out is set to NULL on error.
 */
int dualgcn_partition(const dualgcn_csr *csr, uint64_t seed, uint32_t walks_per_node,
                      uint32_t walk_len, const dualgcn_thresholds *th, void *stream,
                      dualgcn_plan **out);

/* Releases a plan and its device memory, after waiting for the plan's own build and for
 * the work queued by every call that used the plan (on any stream).  NULL is a no-op. */
void dualgcn_plan_destroy(dualgcn_plan *plan);

/*
 * dualgcn_plan_save / dualgcn_plan_load -- keep a partition across runs (Sec. 3.2: the
 * preprocessing is amortised over the training epochs).  The saved form is a host byte
 * buffer: a header (parameters, the weight an adaptive alpha chose, the sizes and a
 * 64-bit checksum of the row pointers and columns) and the density sums S (4 n bytes).
 * Loading rebuilds the plan from S on the given CSR without walking: keys, threshold,
 * sort and schedule are recomputed, so the plan equals the saved one exactly.
 *
 * save: with buf NULL, *bytes receives the size needed; otherwise *bytes must be at
 * least that (else DUALGCN_ERR_INVALID_ARG, *bytes set to it) and receives the size
 * written.  Waits for the device.
 * load: csr must hold the same structure as the saved plan's matrix (same n, nnz and
 * checksum, else DUALGCN_ERR_INVALID_ARG; the values may differ, e.g. another
 * aggregator); a buffer that is not a saved plan (magic, version, size) is
 * DUALGCN_ERR_INVALID_ARG.  Waits for `stream` like dualgcn_partition.  *out is NULL
 * on error.
 */
int dualgcn_plan_save(const dualgcn_plan *plan, void *buf, size_t *bytes);
int dualgcn_plan_load(const dualgcn_csr *csr, const void *buf, size_t bytes, void *stream,
                      dualgcn_plan **out);

/*
 * dualgcn_spmm -- Y = A X, the aggregation SpMM (Sec. 1, Sec. 2.1).
 *
 * X and Y are float32 row-major n x F, contiguous (leading dimension F), and
 * must not overlap.  Rows of the sparse region are computed by the sparse
 * path (runs of up to 8 short rows per lane group of a wavefront); rows of the
 * dense region by the dense path (a lane group per row under 512 entries -- 256,
 * 128, 64 for F <= 64, 32, 16 --, a wavefront per longer row; rows longer than the
 * dense chunk are split over
 * several wavefronts and combined in a fixed order).
 * Every row of Y is written, rows without entries with zeros.  Products are
 * float32; sums are formed in float32 over at most 16 terms and then in
 * float64, and each output is rounded once to float32, so results do not
 * depend on timing (bit-reproducible for a given plan and F).  On plans that mark
 * cold columns (dualgcn_plan_info.cold_marked) and X larger than 256 MiB and
 * smaller than 4 GiB, rows of X outside the hottest 65,536 are read with
 * non-temporal loads, which keeps the hottest rows in the L2; the results are the
 * same.  1 <= F < 2^20.  Asynchronous.
 */
int dualgcn_spmm(const dualgcn_plan *plan, const float *X, float *Y, int32_t F, void *stream);

/* ------------------------------------------------------------------ GCN layer */

/* Flags of the GCN-layer entry points. */
#define DUALGCN_RELU 1u       /* act = ReLU (else the identity) */
#define DUALGCN_OUT_BF16 2u   /* the output is stored as bfloat16: the nearest-even rounding of
                                 the float32 result (2 bytes per element, same row-major layout) */
#define DUALGCN_IN_BF16 4u    /* the input X of the update holds bfloat16 values */

/*
 * dualgcn_spmm_act -- Y = act(A X): dualgcn_spmm with the activation of a GCN
 * layer applied to every output before it is stored (Sec. 1: a layer ends with
 * a non-linearity).  act is ReLU if `flags & DUALGCN_RELU`, else the identity.
 * With DUALGCN_OUT_BF16, Y receives the bfloat16 rounding of each float32 output
 * (after the activation): exactly what the next layer's update rounds its input
 * to, so a layer chain through a bfloat16 intermediate gives bit-identical
 * results with half the intermediate's bytes.  Other flag bits are
 * DUALGCN_ERR_INVALID_ARG.  Same summation and errors as dualgcn_spmm.
 * Asynchronous.
 */
int dualgcn_spmm_act(const dualgcn_plan *plan, const float *X, void *Y, int32_t F,
                     uint32_t flags, void *stream);

/*
 * dualgcn_update -- the update phase of a GCN layer alone, T = X W (Sec. 1: the
 * aggregated features are multiplied by a small dense weight matrix).
 *
 * X is float32 n x F_in row-major (16-byte aligned) -- or bfloat16 when `flags`
 * holds DUALGCN_IN_BF16 --, W float32 F_in x F_out row-major, T float32
 * n x F_out row-major, n >= 1.  Computed on the matrix cores with X and W rounded
 * to bfloat16 (nearest-even; bfloat16 X is used as stored) and float32
 * accumulation.  F_in and F_out must be multiples of 32 with F_in <= 1024 and
 * F_out <= 256 (else DUALGCN_ERR_UNSUPPORTED).  X and T must not overlap; other
 * flag bits are DUALGCN_ERR_INVALID_ARG.  No plan and no workspace: the update
 * does not depend on the partition, so it may run on another stream while
 * dualgcn_partition works.  Asynchronous.
 */
int dualgcn_update(const void *X, const float *W, float *T, int32_t n, int32_t F_in,
                   int32_t F_out, uint32_t flags, void *stream);

/*
 * dualgcn_spmm_update -- the aggregation of one GCN layer fused with the update of the
 * next: T = bf16(act(A X)) bf16(W), float32 accumulation (Sec. 1: a layer's aggregated
 * output, after its non-linearity, is what the next layer multiplies by its weights).
 *
 * The same result as dualgcn_spmm_act with DUALGCN_OUT_BF16 into a buffer H followed
 * by dualgcn_update of H with DUALGCN_IN_BF16 -- bit for bit: every row of act(A X) is
 * summed as in dualgcn_spmm, rounded to bfloat16 (nearest-even), and multiplied on the
 * matrix cores in the update's order --, without reading H back: with H = NULL the
 * n x F_in intermediate never goes through device memory at all.
 *
 * Route (Sec. 3.3: the execution path follows the data).  The fused kernel pays where
 * the aggregation is bound by the memory fabric; where the operand fits the memory-side
 * cache, or the kernel's LDS leaves fewer than three workgroups per CU, the two calls are
 * faster.  dualgcn_spmm_update_route tells which; when H is given (16-byte aligned) this
 * call takes the faster route itself, with H as the intermediate.  With H = NULL it
 * always runs the fused kernel.  Either route writes the same T (and H).
 *
 * X is float32 n x F_in row-major (16-byte aligned), W float32 F_in x F_out row-major
 * (rounded to bfloat16 as in dualgcn_update), T float32 n x F_out row-major (16-byte
 * aligned), overlapping neither X nor W.  H is NULL, or bfloat16 n x F_in row-major
 * (8-byte aligned, overlapping none of X, W and T) that also receives bf16(act(A X)),
 * the output dualgcn_spmm_act would write with DUALGCN_OUT_BF16 (training keeps it for
 * the backward pass).  flags: DUALGCN_RELU (others are DUALGCN_ERR_INVALID_ARG).  F_in and F_out must be multiples of 32, at most 256, and
 * W^T in bfloat16 plus the row tiles must fit a workgroup's LDS (F_in = F_out = 256
 * does not; everything with F_in <= 128 does), else DUALGCN_ERR_UNSUPPORTED.
 * Asynchronous.
 */
int dualgcn_spmm_update(const dualgcn_plan *plan, const float *X, const float *W, float *T,
                        void *H, int32_t F_in, int32_t F_out, uint32_t flags, void *stream);

/* Host-only: *fused = 1 when the fused kernel of dualgcn_spmm_update is the faster route
 * for this plan and shape (the operand n x F_in float32 exceeds the 256 MiB memory-side
 * cache and at least three workgroups fit a CU), 0 when the two calls are.  Shape limits
 * and status as for dualgcn_spmm_update; *fused is left unchanged on error. */
int dualgcn_spmm_update_route(const dualgcn_plan *plan, int32_t F_in, int32_t F_out,
                              int32_t *fused);

/* Bytes of device workspace dualgcn_gcn_layer needs (host-only, no device use):
 * room for the float32 n x F_out product T. */
int dualgcn_gcn_layer_workspace(const dualgcn_plan *plan, int32_t F_in, int32_t F_out,
                                size_t *bytes);

/*
 * dualgcn_gcn_layer -- one GCN layer Y = act(A (X W)): dualgcn_update into the
 * workspace followed by dualgcn_spmm_act (Sec. 1: update, aggregation, no bias).
 *
 * X is n x F_in row-major (float32, or bfloat16 with DUALGCN_IN_BF16), W float32
 * F_in x F_out row-major, Y n x F_out row-major (float32, or bfloat16 with
 * DUALGCN_OUT_BF16); X and Y may be the same buffer.  flags: DUALGCN_RELU,
 * DUALGCN_IN_BF16, DUALGCN_OUT_BF16 (others are DUALGCN_ERR_INVALID_ARG).
 * `workspace` is caller-owned device memory of at least
 * dualgcn_gcn_layer_workspace() bytes, 256-byte aligned, overlapping neither X
 * nor Y (else DUALGCN_ERR_INVALID_ARG).  Shape limits as for dualgcn_update.
 * Asynchronous.
 */
int dualgcn_gcn_layer(const dualgcn_plan *plan, const void *X, const float *W, void *Y,
                      int32_t F_in, int32_t F_out, uint32_t flags, void *workspace,
                      size_t workspace_bytes, void *stream);

/* ------------------------------------------------------------------ aggregators */

enum { DUALGCN_AGG_GCN = 0, DUALGCN_AGG_MEAN = 1, DUALGCN_AGG_SUM = 2 };

/*
 * dualgcn_aggregator_values -- fills val (device, float32[nnz]) with the values of an
 * aggregation matrix on the structure of csr (its rowptr and col; csr->val is not read
 * and may be the same buffer as val).  Sec. 2.1: the aggregation phase multiplies by a
 * matrix derived from the adjacency; the SpMM kernels take any values, so other
 * aggregators run on the same plan.  With d_v the row length of v in the matrix as
 * given (self-loops included when present):
 *   DUALGCN_AGG_GCN   1 / sqrt(d_r d_c)                      (symmetric normalisation)
 *   DUALGCN_AGG_MEAN  1 / d_r                                (GraphSAGE mean)
 *   DUALGCN_AGG_SUM   1, and 1 + eps on self-loop entries    (GIN: A + (1 + eps) I
 *                     when every row holds its self-loop once)
 * computed in float64 and rounded once to float32.  The CSR is validated on the device
 * first and the call waits for `stream` to report DUALGCN_ERR_BAD_CSR (val is then
 * undefined).  A plan built before keeps its own copy of the values: build it again, or
 * build it after filling val.
 */
int dualgcn_aggregator_values(const dualgcn_csr *csr, int32_t kind, float eps, float *val,
                              void *stream);

/* ------------------------------------------------------------------ training */

/*
 * The backward pass of a GCN layer H = act(P), P = A T, T = X W (Sec. 1: the paper
 * accelerates GCN training, whose gradients repeat the aggregation).  With
 * G = dL/dH the chain rule gives, in order:
 *   G_P = G * act'(P)          ReLU' = [P > 0]; folded into the product that makes G
 *   G_T = A^T G_P              dualgcn_spmm_act on a plan of A^T.  The symmetric
 *                              normalised adjacency is its own transpose, so there
 *                              the forward plan serves; for another matrix, partition
 *                              its transpose.
 *   dW  = X^T G_T              dualgcn_weight_grad
 *   dX  = (G_T W^T) * [M > 0]  dualgcn_backward_data, M the previous layer's output
 * and the loss gradient of the last layer comes from dualgcn_softmax_xent.
 */

/* Flag of the training entry points: the gradient operand G holds bfloat16 values. */
#define DUALGCN_GRAD_BF16 8u

/* float64 slots of the loss buffer of dualgcn_softmax_xent. */
#define DUALGCN_LOSS_SLOTS 1025

/*
 * dualgcn_softmax_xent -- mean softmax cross-entropy over labeled rows.
 *
 * Y (device, float32 n x C row-major) holds the logits, labels (device, int32[n])
 * the class of every row; rows whose label is outside [0, C) are unlabeled.
 * Writes G (device, float32 n x C) = scale * (softmax(Y_v) - e_label_v) on labeled
 * rows and 0 on the others, and loss[0] = scale * sum over labeled rows of
 * -log softmax(Y_v)[label_v]; pass scale = 1 / (number of labeled rows) for the
 * mean.  loss is a device float64 buffer of DUALGCN_LOSS_SLOTS entries: the others
 * receive per-workgroup partial sums, added in a fixed order, so the loss does not
 * depend on timing.  float32 arithmetic (expf, logf), the loss summed in float64.
 * G must not overlap Y.  1 <= C < 2^20.  Asynchronous.
 */
int dualgcn_softmax_xent(const float *Y, const int32_t *labels, int32_t n, int32_t C,
                         float scale, float *G, double *loss, void *stream);

/* Bytes of the workspace dualgcn_weight_grad needs for n rows (host only). */
int dualgcn_weight_grad_workspace(int32_t n, int32_t F_in, int32_t F_out, size_t *bytes);

/*
 * dualgcn_weight_grad -- dW = X^T G, the weight gradient of the update phase.
 *
 * X (device, n x F_in) is float32, or bfloat16 with DUALGCN_IN_BF16; G (device,
 * n x F_out) is float32, or bfloat16 with DUALGCN_GRAD_BF16; dW (device, float32
 * F_in x F_out row-major).  Both operands are rounded to bfloat16 (nearest-even)
 * and multiplied on the matrix cores with float32 accumulation over chunks of
 * rows; the per-workgroup partial matrices (in `workspace`, device, 256-byte
 * aligned, at least dualgcn_weight_grad_workspace bytes) are summed in a fixed
 * order in float64, so results do not depend on timing, nor on which operands come
 * in bfloat16 (an operand passed as its bfloat16 rounding gives the same bits as the
 * float32 original; with both in bfloat16 half the bytes are read).  If W (device, float32
 * F_in x F_out) is not NULL, the same call applies the SGD step W -= lr dW.
 * Shapes: F_in and F_out multiples of 32, F_in <= 1024, F_out <= 256 (else
 * DUALGCN_ERR_UNSUPPORTED); X and G 16-byte aligned.  Asynchronous.
 */
int dualgcn_weight_grad(const void *X, const void *G, float *dW, int32_t n, int32_t F_in,
                        int32_t F_out, uint32_t flags, float lr, float *W, void *workspace,
                        size_t workspace_bytes, void *stream);

/* Size of the library's static device array that dualgcn_weight_grad_noalloc keeps its
 * partial dW matrices in (64 MiB, held on every device the library runs on). */
#define DUALGCN_WGRAD_NOALLOC_BYTES (64u << 20)

/*
 * dualgcn_weight_grad_noalloc -- dualgcn_weight_grad without a workspace and without any
 * device allocation, for callers that cannot allocate (code under HIP graph capture, tight
 * serving or training loops, harnesses that forbid hipMalloc).  The per-workgroup partial
 * dW matrices go to a static device array of DUALGCN_WGRAD_NOALLOC_BYTES bytes that the
 * library holds on each device; the kernels, their workgroup count and the fixed
 * summation order are those of dualgcn_weight_grad, so dW (and W after the SGD step) are
 * bit-identical to what dualgcn_weight_grad writes on the same device.
 *
 * Arguments, flags and shape limits as for dualgcn_weight_grad.  The partials need
 * (workgroups) x F_in x F_out x 4 bytes, the workgroups being as many as the device holds
 * at once (one per compute unit on MI355X), at most one per 64 rows: shapes whose partials
 * exceed the array return DUALGCN_ERR_UNSUPPORTED before any work is queued (F_in x F_out
 * up to 256 x 128 fits on MI355X for any n).  Every call on a device shares that device's
 * array: two calls that overlap in time on one device (other streams, other host threads)
 * race and give undefined results; calls on one stream are ordered.  Asynchronous.
 */
int dualgcn_weight_grad_noalloc(const void *X, const void *G, float *dW, int32_t n,
                                int32_t F_in, int32_t F_out, uint32_t flags, float lr, float *W,
                                void *stream);

/*
 * dualgcn_backward_data -- dX = (G W^T) * [M > 0], the gradient that flows from a
 * layer's update phase to its input, masked by the ReLU that produced that input.
 *
 * G (device, n x F_out) is float32, or bfloat16 with DUALGCN_GRAD_BF16; W (device,
 * float32 F_in x F_out, the layer's weights as used forward); M (device, n x F_in)
 * is the previous layer's output H (float32, or bfloat16 with DUALGCN_IN_BF16), or
 * NULL for no mask; dX (device, float32 n x F_in).  G and W are rounded to
 * bfloat16 and multiplied on the matrix cores with float32 accumulation (the
 * kernel of dualgcn_update).  dX must not overlap G or M.  Shape limits as for
 * dualgcn_update (F_in and F_out multiples of 32, F_in <= 1024, F_out <= 256); G
 * 16-byte aligned, and with a mask M and dX too.  Asynchronous.
 */
int dualgcn_backward_data(const void *G, const float *W, const void *M, float *dX, int32_t n,
                          int32_t F_in, int32_t F_out, uint32_t flags, void *stream);

/* ------------------------------------------------------------------ measurement */

enum { DUALGCN_PROBE_COPY = 0, DUALGCN_PROBE_READ = 1 };

/*
 * dualgcn_bandwidth_probe -- a plain streaming kernel that shows the memory bandwidth the
 * device delivers, the yardstick next to which the SpMM's rates are read (the paper reports
 * kernel times only, Sec. 4.1; this library reports each kernel's bytes against the
 * memory system).
 *   DUALGCN_PROBE_COPY  dst = src over `bytes` (read once, written once with
 *                       non-temporal stores); src and dst must not overlap.
 *   DUALGCN_PROBE_READ  every byte of src read once and summed; dst receives one float per
 *                       workgroup, at most dualgcn_bandwidth_probe_out_floats() of them.
 * src and dst are device memory, 16-byte aligned; `bytes` a positive multiple of 16
 * (else DUALGCN_ERR_INVALID_ARG).  Time it with events on `stream`.  Asynchronous.
 */
int dualgcn_bandwidth_probe(int32_t kind, const void *src, void *dst, size_t bytes, void *stream);

/* Floats the read probe writes at most (host-only). */
int32_t dualgcn_bandwidth_probe_out_floats(void);

/* ------------------------------------------------------------------ introspection */

typedef struct dualgcn_plan_info {
    int32_t n;
    int64_t nnz;
    int32_t n_sparse;        /* rows in the sparse region: perm[0 .. n_sparse) */
    int32_t n_dense;         /* n - n_sparse */
    uint64_t kstar;          /* threshold key K* */
    uint64_t s1_hi, s1_lo;   /* sum of K_v, 128-bit */
    uint64_t s2_hi, s2_lo;   /* sum of K_v^2, 128-bit */
    uint64_t kmax;           /* largest K_v */
    uint32_t alpha_num, alpha_den, beta_num, beta_den;
    int32_t force_mode;
    uint64_t seed;
    uint32_t walks_per_node, walk_len;
    int32_t max_degree;
    int32_t dense_chunk;     /* entries per dense-region wavefront: 4096 below 2^20
                                entries, else the largest power of two from 512 to 4096
                                not above nnz / 2048 */
    int32_t n_split_rows;    /* dense rows longer than dense_chunk */
    int32_t n_split_parts;   /* wavefronts those rows are split over */
    int32_t n_tasks;         /* sparse-region tasks (runs of at most 8 short rows) */
    int32_t n_long_rows;     /* dense rows of >= 512 entries (a wavefront each; the
                                shorter dense rows get a lane group each; for F <= 64
                                the bound is 256, for F <= 32 128, for F <= 16 64) */
    int32_t cold_marked;     /* 1 when the plan marks the columns outside the hottest
                                65,536 (plans of more than 2^18 nodes): an SpMM whose
                                operand is larger than 256 MiB and smaller than 4 GiB then
                                gathers their rows with non-temporal loads (same results) */
} dualgcn_plan_info;

/* Fills *out from host-side copies kept in the plan (no device use). */
int dualgcn_plan_query(const dualgcn_plan *plan, dualgcn_plan_info *out);

/*
 * Copies the plan's perm (int32[n]), S (uint32[n]) and K (uint64[n]) to host
 * buffers; any of them may be NULL.  Waits for the device.
 */
int dualgcn_plan_export(const dualgcn_plan *plan, int32_t *perm_h, uint32_t *S_h,
                        uint64_t *K_h);

/*
 * dualgcn_arw_patterns -- the anonymous walks themselves (Sec. 3.2), for tests:
 * out (device, uint8[n][k][d+1]) receives, for walk w of node v, the label of
 * each visited position (1 + order of first occurrence), with the random
 * stream of dualgcn_partition.  Requires n k (d + 1) < 2^40, k (d + 1) < 2^32
 * and d <= 255 (else DUALGCN_ERR_UNSUPPORTED).  Waits for `stream`.
 */
int dualgcn_arw_patterns(const dualgcn_csr *csr, uint64_t seed, uint32_t walks_per_node,
                         uint32_t walk_len, uint8_t *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DUALGCN_H */
