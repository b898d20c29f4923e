/*
 * arc_oracle.h -- plain CPU oracle of the ARC-Top-K + EF21M compressor step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path
 * (libarctopk) never links, loads or calls it, and the two share no code.
 *
 * Paper: C. Chen, C. Ma, Z. Li, Y. He, Y. Dong, K. Yuan, "An All-Reduce
 * Compatible Top-K Compressor for Communication-Efficient Distributed
 * Learning", arXiv:2510.26709.  Equation numbers follow the paper's own
 * numbering: (3) reshape g -> G, (4) row importance and arg-top-K,
 * (5) row aggregation, (6) unbiasedness of the importance, (11a)-(11c) the
 * EF21M recursion; "Alg. 1" is the ARC-Top-K algorithm box of Sec. IV.
 *
 * Precision: the paper fixes none.  The arg-top-K turns floating point into
 * an integer decision, so this oracle takes that decision in the same
 * precision as the GPU path: IEEE binary32, every operation correctly
 * rounded, in the fixed sequential order documented on each function, with
 * no contraction other than the explicit fmaf calls.
 *
 * Layout: worker i's d-vector occupies elements [i*d, (i+1)*d) of an [N][d]
 * array; its m x n view (Eq. (3)) is row-major, row p = elements
 * [p*n, p*n + n) clipped at d, with m = ceil(d / n).  Elements past d in the
 * last row are absent (they take part in no sum and are never written).
 *
 * All functions return 0 on success and 1 on an invalid argument.
 */
#ifndef ARC_ORACLE_H
#define ARC_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Gaussian projection V (n x r, row-major V[j*r + k]) for seed s, step t. */
int oracle_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                      float *V);

/* SplitMix64: output number x (0-based) of the stream seeded with `seed`. */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t x);

/* EF21M momentum, Eq. (11a), in place on h[N*d].  grad is fp32
 * (grad_is_bf16 == 0) or bf16 bit patterns (grad_is_bf16 == 1). */
int oracle_momentum(int32_t N, int64_t d, float eta, const void *grad,
                    int32_t grad_is_bf16, float *h);

/* Per-worker sketch S[i][p][k] of the residual h - g (Alg. 1, local
 * projection), S is [N][m][r]. */
int oracle_sketch(int32_t N, int64_t d, int64_t n, int32_t r, const float *h,
                  const float *g, const float *V, float *S);

/* Worker sum P[p][k] over i (Alg. 1, first All-Reduce), P is [m][r]. */
int oracle_worker_sum(int32_t N, int64_t m, int32_t r, const float *S,
                      float *P);

/* Row importance sigma[p] = sum_k P[p][k]^2 (Eq. (4), diag(P P^T)). */
int oracle_importance(int64_t m, int32_t r, const float *P, float *sigma);

/* Per-bucket arg-top-K of sigma (Eq. (4)); ties to the lower row, output
 * ascending within a bucket, buckets concatenated in order.  num_buckets == 0
 * means one bucket [0, m) with K = K_global.  Returns the number of indices
 * written through *K_total. */
int oracle_select(int64_t m, const float *sigma, int64_t K_global,
                  int32_t num_buckets, const int64_t *bucket_row_begin,
                  const int64_t *bucket_K, int32_t *idx, int64_t *K_total);

/* Gather + worker sum + error-feedback update at the shared rows (Eq. (5),
 * Alg. 1 second All-Reduce, Eq. (11b)).  agg is [K_total][n]. */
int oracle_gather_update(int32_t N, int64_t d, int64_t n, int64_t K_total,
                         const int32_t *idx, const float *h, float *g,
                         float *agg);

/* One full compressor step: momentum, sketch, worker sum, importance,
 * selection, gather/update.  V_override (n*r floats) replaces the generated
 * projection when non-NULL.  sigma_out ([m]) and S_out ([N][m][r]) are
 * optional copies of the intermediates. */
int oracle_step(int32_t N, int64_t d, int64_t n, int32_t r, float eta,
                uint64_t seed, int64_t t, int64_t K_global,
                int32_t num_buckets, const int64_t *bucket_row_begin,
                const int64_t *bucket_K, const void *grad,
                int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                float *agg, int64_t *K_total, const float *V_override,
                float *sigma_out, float *S_out);

/* Per-tensor mode (Sec. VI: each tensor of the model is compressed in its own
 * 2-D view with its own K; 1-D tensors are kept whole).  Tensor b covers the
 * rows[b]*cols[b] consecutive coordinates after tensor b-1 (sum = d), viewed
 * row-major; its rows are global rows [row_b, row_b + rows[b]) of Sigma, S and
 * idx.  V for a tensor of width w is oracle_projection(seed, t, w, r).  agg is
 * packed: tensor b's K_b selected rows of cols[b] values follow tensor b-1's.
 * *K_total and *agg_len receive the output sizes. */
int oracle_step_tensors(int32_t N, int32_t r, float eta, uint64_t seed,
                        int64_t t, int32_t num_tensors, const int64_t *rows,
                        const int64_t *cols, const int64_t *K,
                        const void *grad, int32_t grad_is_bf16, float *h,
                        float *g, int32_t *idx, float *agg, int64_t *K_total,
                        int64_t *agg_len, float *sigma_out, float *S_out);

/* Model step around the compressor (Eq. (11c), Sec. VI optimisers and dense
 * warm-up).  G is the node-summed tracker sum_i g^(i), kept by adding each
 * step's payload.  Dense step: Eq. (11a) and (11b) with the identity
 * compressor, the payload added straight into G. */
int oracle_dense_step(int32_t N, int64_t d, float eta, const void *grad,
                      int32_t grad_is_bf16, float *h, float *g, float *G);

/* G += agg at the selected rows (single m x n view, or per-tensor packed). */
int oracle_accumulate_rows(int64_t d, int64_t n, int64_t K_total,
                           const int32_t *idx, const float *agg, float *G);
int oracle_accumulate_tensors(int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K,
                              const int32_t *idx, const float *agg, float *G);

/* x update from G: optimizer 0 SGD (Eq. (11c)), 1 MSGD, 2 Adam; T is Adam's
 * step count (>= 1); m, v are the optimiser state ([d] each, as needed). */
int oracle_optimizer(int32_t optimizer, int32_t N, int64_t d, int64_t T,
                     float lr, float momentum, float beta1, float beta2,
                     float eps, float weight_decay, const float *G, float *x,
                     float *m, float *v);

/* Comparison compressors of Table I inside the same EF21M step.
 * Rand-K: K rows per bucket drawn uniformly (shared seed, unscaled); row p's
 * key is (float)(SplitMix64 output t*m + p of the seed's stream >> 40), the K
 * largest keys kept (ties to the lower row); payload summed over nodes as for
 * ARC-Top-K.  keys_out ([m]) is optional. */
int oracle_randk_keys(uint64_t seed, int64_t t, int64_t m, float *keys);
int oracle_step_randk(int32_t N, int64_t d, int64_t n, float eta, uint64_t seed,
                      int64_t t, int64_t K_global, int32_t num_buckets,
                      const int64_t *bucket_row_begin, const int64_t *bucket_K,
                      const void *grad, int32_t grad_is_bf16, float *h, float *g,
                      int32_t *idx, float *agg, int64_t *K_total, float *keys_out);
int oracle_step_randk_tensors(int32_t N, float eta, uint64_t seed, int64_t t,
                              int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K, const void *grad,
                              int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                              float *agg, int64_t *K_total, int64_t *agg_len,
                              float *keys_out);

/* Top-K (All-Gather): node i keeps its own K rows of largest ||Delta^(i)_p||^2
 * (fmaf chain of squares, ascending columns, from +0; ties to the lower
 * row).  idx is [N][K_total] (K_total per node), agg [N][L]: node i's rows of
 * Delta^(i) (single view: K_total x n, +0 past d; tensors: packed), nothing
 * summed; g^(i) += Delta^(i) on node i's rows.  norms_out ([N][m]) optional. */
int oracle_step_topk(int32_t N, int64_t d, int64_t n, float eta, int64_t K_global,
                     int32_t num_buckets, const int64_t *bucket_row_begin,
                     const int64_t *bucket_K, const void *grad, int32_t grad_is_bf16,
                     float *h, float *g, int32_t *idx, float *agg, int64_t *K_total,
                     float *norms_out);
int oracle_step_topk_tensors(int32_t N, float eta, int32_t num_tensors, const int64_t *rows,
                             const int64_t *cols, const int64_t *K, const void *grad,
                             int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                             float *agg, int64_t *K_total, int64_t *agg_len,
                             float *norms_out);

/* Top-K's merge into G = sum_i g^(i) (Sec. III, Prop. 1): for every
 * coordinate of a row some node kept, the kept values of the nodes that kept
 * it are summed in ascending node order (first value as it is, then plain
 * additions) and the sum is added to G.  idx and agg as oracle_step_topk (and
 * _tensors) return them: [N][K_node] rows of the view, [N][L] payload. */
int oracle_merge_topk_rows(int32_t N, int64_t d, int64_t n, int64_t K_node,
                           const int32_t *idx, const float *agg, float *G);
int oracle_merge_topk_tensors(int32_t N, int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K, const int32_t *idx,
                              const float *agg, float *G);

/* Number of threads the oracle's parallel loops use. */
int oracle_num_threads(void);
void oracle_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
