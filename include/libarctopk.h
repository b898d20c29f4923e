/*
 * libarctopk -- the ARC-Top-K + EF21M compressor step on one AMD Instinct
 * MI355X (gfx950), behind a plain C ABI.
 *
 * Method: C. Chen, C. Ma, Z. Li, Y. He, Y. Dong, K. Yuan, "An All-Reduce
 * Compatible Top-K Compressor for Communication-Efficient Distributed
 * Learning", arXiv:2510.26709.  Equation numbers are the paper's: (3) the
 * reshape g -> G (m x n), (4) row importance Sigma = diag(P P^T) and
 * I = arg top_K(Sigma), (5) the row aggregation, (11a)/(11b) the EF21M
 * momentum and error-feedback lines.  "Alg. 1" is the ARC-Top-K algorithm box
 * of Sec. IV.
 *
 * The N data-parallel nodes of the paper are simulated as the leading axis of
 * an [N][d] batch on one GPU.  One call of arc_step performs, for step t:
 *
 *   h^(i)   <- (1 - eta) h^(i) + eta grad^(i)                       (11a)
 *   Delta^(i) = h^(i) - g^(i)      (the compressor's argument in (11b))
 *   V_t     = n x r Gaussian matrix from (seed, t)           (Sec. IV, Alg. 1)
 *   P       = sum_i Delta^(i)_{m x n} V_t                        (Alg. 1)
 *   Sigma_p = ||P_p||^2,  I = arg top_K(Sigma)                        (4)
 *   agg     = sum_i rows I of Delta^(i)  (packed, index-free payload; (5))
 *   g^(i)   <- g^(i) + (rows I of Delta^(i))                        (11b)
 *
 * Numerics (the contract shared with the reference CPU implementation):
 * binary32 everywhere; every sum in ascending index order; the dot products
 * over a row and the squares in Sigma use fused multiply-add chains starting
 * at +0; the worker sums are plain additions in ascending worker order; V_t
 * is rounded once from a binary64 Box-Muller value.  Ties in Sigma go to the
 * lower row.  With these rules the selected rows are exactly reproducible.
 * The 1/sqrt(r) and 1/N factors of the text are not applied: they cannot
 * change I, and agg is the SUM over workers (divide by N for the mean of (5)).
 *
 * Layout: worker i's vector is elements [i*d, (i+1)*d) of each [N][d] array.
 * Row p of its m x n view (row-major, Eq. (3)) is elements [p*n, p*n + n)
 * clipped at d; m = ceil(d / n).  Elements past d in a ragged last row do
 * not exist: they are never read or written and give +0 in agg.
 *
 * Streams: all device work of a context is enqueued on the HIP stream given
 * to arc_create.  arc_step returns after enqueueing; its outputs are valid
 * once that stream has completed the work.  A context is not thread-safe; use
 * one per stream.  Preconditions: finite inputs (non-finite values give
 * unspecified selections).
 *
 * Errors: every entry point returns an arc_status.  Invalid arguments are
 * detected before any device work is enqueued and leave all buffers
 * untouched.  After ARC_ERR_DEVICE the context must be destroyed.
 * arc_last_error() gives a human-readable reason for the last failure on the
 * calling thread.
 */
#ifndef LIBARCTOPK_H
#define LIBARCTOPK_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct arc_ctx arc_ctx;

typedef enum {
  ARC_OK = 0,
  ARC_ERR_INVALID = 1,     /* bad argument or configuration                  */
  ARC_ERR_NOMEM = 2,       /* device or pinned host allocation failed        */
  ARC_ERR_DEVICE = 3,      /* HIP runtime or launch failure                  */
  ARC_ERR_UNSUPPORTED = 4  /* valid request this build does not implement    */
} arc_status;

typedef enum { ARC_DTYPE_F32 = 0, ARC_DTYPE_BF16 = 1 } arc_dtype;

/*
 * Compressor inside the EF21M step (Table I).  All keep K rows per bucket
 * (or tensor) of Delta^(i) = h_t^(i) - g_{t-1}^(i) and move g^(i) by the kept
 * rows (Eq. (11b)).
 *   ARC_COMP_ARC    ARC-Top-K (Alg. 1): rows by the sketched importance,
 *                   shared by every node; payload summed over nodes.
 *   ARC_COMP_RANDK  Rand-K: rows drawn uniformly with the shared seed, the
 *                   same on every node, unscaled; payload summed over nodes.
 *                   Row p's key is (float)(x >> 40) for x the SplitMix64
 *                   output number t*m + p of the stream seeded with `seed`;
 *                   the K largest keys are kept, ties to the lower row.
 *   ARC_COMP_TOPK   Top-K: every node its own K rows of largest ||Delta_p||^2
 *                   (fmaf chain of squares over the row in ascending column
 *                   order from +0, ties to the lower row); each node's rows
 *                   and values are returned as they are (the All-Gather
 *                   payload), nothing summed.
 */
typedef enum { ARC_COMP_ARC = 0, ARC_COMP_RANDK = 1, ARC_COMP_TOPK = 2 } arc_compressor;

/* Largest projection dimension r accepted. */
#define ARC_MAX_R 32

/*
 * One tensor of the per-tensor mode: `rows` x `cols` consecutive coordinates
 * viewed row-major, compressed with its own K (Sec. VI: each 2-D tensor in
 * its own view, convolution kernels as out x (in*kh*kw), 1-D tensors kept
 * whole, e.g. as one row with K = 1).
 */
typedef struct {
  int64_t rows; /* >= 1 */
  int64_t cols; /* >= 1 */
  int64_t K;    /* rows kept, >= 0; K >= rows keeps the tensor whole */
} arc_tensor;

/*
 * Problem description (Alg. 1 inputs, EF21M step size, shared seed).
 *   d            coordinates per worker (> 0)
 *   n            row width of the m x n view (> 0); m = ceil(d/n) <= 2^31-1
 *   K            selected ROWS when num_buckets == 0 (>= 0; K >= m keeps
 *                every row, i.e. the identity compressor).  The paper's
 *                K = ceil(mu * m) for a compression ratio mu.
 *   seed         shared seed s; V_t is a function of (seed, t) only
 *   bucket_row_begin, bucket_K
 *                optional independent selections (num_buckets > 0): bucket b
 *                is rows [bucket_row_begin[b], bucket_row_begin[b+1]) with its
 *                own K (bucket_K[b] >= 0, clamped to the bucket's rows).
 *                bucket_row_begin has num_buckets+1 strictly increasing
 *                entries from 0 to m.  Host arrays, copied by arc_create.
 *   N            workers (> 0)
 *   r            projection dimension, 1..ARC_MAX_R (the paper uses 4)
 *   grad_dtype   arc_dtype of the gradients; h and g are always binary32
 *   num_buckets  0 for one global selection over all m rows
 *   eta          EF21M momentum weight, 0 <= eta <= 1
 *   tensors, num_tensors
 *                per-tensor mode (num_tensors > 0): the d coordinates are
 *                tensors[0], tensors[1], ... in order (sum of rows*cols ==
 *                d); each tensor is its own m_b x n_b view with its own K_b,
 *                the global rows are tensor 0's rows, then tensor 1's, ...;
 *                n, K and num_buckets must then be 0.  A tensor of width w
 *                uses the projection V_t of width w (tensors of equal width
 *                share it).  Host array, copied by arc_create.
 *   compressor   arc_compressor (0 = ARC-Top-K); r and V are unused by
 *                Rand-K and Top-K
 */
typedef struct {
  int64_t d;
  int64_t n;
  int64_t K;
  uint64_t seed;
  const int64_t *bucket_row_begin;
  const int64_t *bucket_K;
  int32_t N;
  int32_t r;
  int32_t grad_dtype;
  int32_t num_buckets;
  float eta;
  int32_t reserved; /* must be 0 */
  const arc_tensor *tensors;
  int32_t num_tensors;
  int32_t compressor; /* arc_compressor */
} arc_config;

/*
 * Validate cfg, allocate the device workspace (projection, per-worker sketch,
 * importance, selection scratch) on the current HIP device and bind the
 * context to `hip_stream` (a hipStream_t; NULL = the default stream).
 * On failure *out is set to NULL.  Workspace bytes are about
 * 4*(n*r + N*m*r + 3*m) plus a few kilobytes per bucket, and for
 * ARC_COMP_TOPK another 8*N*m (the rows each node kept, for the merge of the
 * model step) plus 4*N*K; pinned host memory 16*n*r.
 */
arc_status arc_create(const arc_config *cfg, void *hip_stream, arc_ctx **out);

/*
 * One compressor step t (t >= 0 selects V_t).  Device pointers:
 *   grad     [N*d] gradients (grad_dtype), read only; must not overlap h or g
 *   h        [N*d] binary32 momentum, read and written (Eq. (11a))
 *   g        [N*d] binary32 error-feedback state; rows in I are updated
 *            (Eq. (11b)), all other elements are left bit-for-bit unchanged
 *   out_idx  [arc_selected_rows(ctx)] int32: the selected rows, ascending
 *            within each bucket, buckets in order
 *   out_agg  [arc_payload_elems(ctx)] binary32: the selected rows in
 *            out_idx order, each as sum_i Delta^(i) of that row (ascending
 *            worker order).  Single view: rows of n values, +0 past d.
 *            Per-tensor mode: packed, each row with its tensor's width.
 *   ARC_COMP_TOPK: out_idx is [N][K] (node i's rows at [i*K, (i+1)*K)) and
 *            out_agg [N][L] (node i's rows of Delta^(i), laid out as above),
 *            with K and L one node's row count and payload length.
 * out_idx / out_agg may be NULL only when no row is kept; otherwise they must
 * not overlap each other or grad, h, g (ARC_ERR_INVALID).  With grad, h and
 * g 16-byte aligned, d % 4 == 0 and r in {1, 2, 4, 8}, rows whose width is a
 * multiple of 4 (per tensor: tensors that also start at a multiple of 4
 * coordinates) take the vectorised path; anything else takes a slower path
 * with identical results.
 * The call returns once the work is queued on the context's stream.  On the
 * host it generates V_t (ARC_COMP_ARC; V_{t+1} is then prepared in the
 * background for the next call) into one of four pinned staging buffers
 * used in turn, waiting only until the device has read the projection
 * staged three calls earlier (the first work of that step): the host can
 * queue up to three steps ahead of the device.  The host work makes the
 * call unsuitable for capture into a HIP graph.
 * On rows longer than the streaming kernel's column chunk (32 to 256
 * values, by how many rows it streams together), its workgroups each hold
 * just over half of a compute unit's LDS, so that one runs per compute
 * unit: while it runs, another kernel's workgroups that need more than the
 * remaining LDS wait for a compute unit to free up.  When every bucket has
 * at most 32,768 rows, the selection runs one 1024-thread workgroup per
 * bucket holding the bucket's importances in up to 143 KB of LDS.
 */
arc_status arc_step(arc_ctx *ctx, int64_t t, const void *grad, float *h,
                    float *g, int32_t *out_idx, float *out_agg);

/*
 * The model step around the compressor (Eq. (11c), the optimisers of the
 * experiments in Sec. VI, and the dense iterations before compression
 * starts).  The nodes keep G = sum_i g^(i): each step's summed payload is
 * added to G at the coordinates it covers, and Eq. (11c) becomes
 * x <- x - (lr / N) * G for SGD.
 *
 * For every coordinate, with dir = fmaf(weight_decay, x, G / N):
 *   ARC_OPT_SGD:  x = fmaf(-lr, dir, x)
 *   ARC_OPT_MSGD: m = fmaf(momentum, m, dir);  x = fmaf(-lr, m, x)
 *   ARC_OPT_ADAM: m = fmaf(beta1, m, fl((1-beta1) * dir));
 *                 v = fmaf(beta2, v, fl((1-beta2) * fl(dir * dir)));
 *                 x = fmaf(-lr, fl(fl(m / c1) / fl(sqrt(fl(v / c2)) + eps)), x)
 *   with T = t + 1, c1 = fl(1 - beta1^T), c2 = fl(1 - beta2^T) (beta^T as T
 *   binary64 products, 1 - beta^T in binary64, rounded once) and (1 - beta)
 *   rounded to binary32.  All operations binary32, correctly rounded.
 */
typedef enum { ARC_OPT_SGD = 0, ARC_OPT_MSGD = 1, ARC_OPT_ADAM = 2 } arc_optimizer;

typedef struct {
  int32_t optimizer;   /* arc_optimizer                                      */
  int32_t dense_steps; /* iterations t < dense_steps are dense (see below)   */
  float lr;            /* step size gamma, finite                            */
  float momentum;      /* MSGD, in [0, 1)                                    */
  float beta1, beta2;  /* Adam, in [0, 1)                                    */
  float eps;           /* Adam, >= 0                                         */
  float weight_decay;  /* L2 coefficient, finite                             */
} arc_model_config;

/*
 * One EF21M iteration (11a)-(11c) on the context's stream, for every
 * compressor.
 *   t < dense_steps: the identity compressor (no compression yet): for every
 *     coordinate, Eq. (11a), Delta_i = h_i - g_i, g_i = g_i + Delta_i, and
 *     G = G + (Delta_0 + Delta_1 + ...); out_idx and out_agg are not written.
 *     The same bits as arc_step with every row kept followed by G += agg.
 *   otherwise: arc_step (same outputs), and G = G + agg at the selected
 *     coordinates.  ARC_COMP_TOPK (Sec. III: the All-Gather is followed by a
 *     merge): every coordinate of a row that some node kept gets the values
 *     of the nodes that kept it, summed in ascending node order (the first as
 *     it is, then plain additions), added to G; with every node keeping the
 *     same rows, the same bits as the shared-row compressors.
 * Then the optimiser updates x (and opt_m, opt_v) over all d coordinates.
 *   G, x          device [d] binary32, in/out; G starts at sum_i g^(i) (0 for
 *                 h = g = 0)
 *   opt_m, opt_v  device [d] binary32 optimiser state: opt_m for MSGD and
 *                 Adam, opt_v for Adam (start at 0); may be NULL otherwise
 * G, x, opt_m and opt_v must not overlap one another, grad, h, g or (on a
 * compressed iteration) out_idx and out_agg.
 * 16-byte aligned pointers with d % 4 == 0 take the vectorised kernels.
 * Invalid model settings give ARC_ERR_INVALID before any work is enqueued.
 */
arc_status arc_model_step(arc_ctx *ctx, const arc_model_config *mc, int64_t t,
                          const void *grad, float *h, float *g, float *G, float *x,
                          float *opt_m, float *opt_v, int32_t *out_idx, float *out_agg);

/*
 * Allocation-free step, for callers that cannot allocate device memory
 * (tight serving loops, harnesses that forbid hipMalloc): the same step as
 * arc_create + arc_step (same kernels, same
 * bits for every output) from a configuration, with no context.  Every
 * device buffer the step needs beyond the caller's grad, h, g, out_idx and
 * out_agg (the kernels' tables, V_t, the per-worker sketch, the importance,
 * the selection's scratch) lives in one static device array of
 * ARC_STATIC_SCRATCH_BYTES per device, which the library holds from the
 * first call on a device until the process ends.  The call allocates no
 * device or pinned host memory; it plans the step on the host (ordinary heap
 * memory), generates V_t on the host and copies the tables and V_t into the
 * static array on hip_stream, then enqueues the step there.
 *   cfg, t, grad, h, g, out_idx, out_agg  as for arc_create and arc_step
 *                 (out_idx [K_total], out_agg [payload]: arc_selected_rows /
 *                 arc_payload_elems of a context of the same cfg)
 *   hip_stream    the hipStream_t to run on (NULL = the default stream)
 * A configuration whose buffers exceed ARC_STATIC_SCRATCH_BYTES (about
 * 16*N*m*r + 4*m bytes plus the tables) gives ARC_ERR_INVALID, as do the
 * invalid arguments arc_create and arc_step reject, before any device work.
 * Every call on one device shares that device's array and leaves its
 * contents behind: calls on one device that overlap in time (two streams,
 * or two host threads) race and give undefined results; calls in stream
 * order, or on one stream, are safe.  Before refilling its host copy of the
 * tables the call waits until the device has read the previous call's.  As
 * it copies from host memory and may wait on the device, the call is not
 * meant for capture into a HIP graph.
 */
#define ARC_STATIC_SCRATCH_BYTES (64u * 1024u * 1024u)
arc_status arc_step_static(const arc_config *cfg, void *hip_stream, int64_t t,
                           const void *grad, float *h, float *g, int32_t *out_idx,
                           float *out_agg);

/* Release the context and its workspace.  NULL is accepted.  Waits for the
 * context's stream to finish its work first. */
arc_status arc_destroy(arc_ctx *ctx);

/* Rows of the m x n view (m = ceil(d/n)); -1 for NULL. */
int64_t arc_num_rows(const arc_ctx *ctx);

/* Entries of out_idx per step: the rows kept after clamping each K to its
 * bucket (N times that for ARC_COMP_TOPK, one list per node); -1 for NULL. */
int64_t arc_selected_rows(const arc_ctx *ctx);

/* Elements of out_agg per step; -1 for NULL. */
int64_t arc_payload_elems(const arc_ctx *ctx);

/* V_t of width n (n x r binary32, row-major) for a shared seed, written to
 * host memory V: the projection every step of that seed uses for rows of
 * width n.  Host only; needs no device. */
arc_status arc_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                          float *V);

/* Static string naming a status code. */
const char *arc_status_str(arc_status s);

/* Reason for the most recent failure on the calling thread ("" if none). */
const char *arc_last_error(void);

/* ---- Inspection hooks (tests and benchmarks; not needed by the method) ---- */

/* Write a one-line, NUL-terminated description of how the context runs a
 * step for pointers that take the vectorised path (kernel variants, LDS per
 * block and the device limit, the selection's path: one workgroup per
 * bucket or its number of blocks) into buf (at most len bytes, truncated).
 * Host only. */
arc_status arc_describe(const arc_ctx *ctx, char *buf, int64_t len);

/* Enqueue a copy of the last step's importance Sigma ([m] binary32) into the
 * device buffer out_sigma. */
arc_status arc_debug_sigma(arc_ctx *ctx, float *out_sigma);

/* Enqueue a copy of the last step's per-worker sketch S ([N][m][r] binary32,
 * S[i][p][k] = sum_j Delta^(i)[p*n+j] V[j][k]) into the device buffer out_S. */
arc_status arc_debug_sketch(arc_ctx *ctx, float *out_S);

/* Write V_t ([n][r] binary32, row-major) for step t into host memory out_V,
 * exactly as arc_step would use it (honours arc_set_projection).  Single-view
 * mode only; in per-tensor mode use arc_projection with the tensor's width. */
arc_status arc_debug_projection(arc_ctx *ctx, int64_t t, float *out_V);

/* Use the host matrix V ([n][r] binary32, copied) for every later step
 * instead of V_t; NULL restores the seeded projection.  Single-view mode
 * only (ARC_ERR_UNSUPPORTED in per-tensor mode). */
arc_status arc_set_projection(arc_ctx *ctx, const float *V);

/* Stage timing: when enabled, arc_step records HIP events on the context's
 * stream around its stages.  arc_timing_read waits for those events and
 * writes, for each of the ARC_NUM_STAGES stages, the summed milliseconds
 * (ms[stage]) over the steps recorded since the last read (*steps); then it
 * clears the record.  Stages: 0 streaming sketch (momentum + residual +
 * per-worker sketch), 1 worker sum + importance, 2 top-K selection, 3 gather +
 * worker sum + error-feedback update, 4 the whole step. */
#define ARC_NUM_STAGES 5
arc_status arc_timing_enable(arc_ctx *ctx, int32_t on);
arc_status arc_timing_read(arc_ctx *ctx, double *ms, int64_t *steps);

#ifdef __cplusplus
}
#endif
#endif
