/*
 * arc_oracle.c -- plain CPU oracle of the ARC-Top-K + EF21M compressor step.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg.  It shares no code with libarctopk.
 *
 * Each function follows one step of the paper (arXiv:2510.26709) in the
 * paper's order and notation; the comment above it names the passage.
 * Arithmetic is IEEE binary32 with the explicit fmaf calls shown and nothing
 * else contracted (build with -ffp-contract=off, no fast-math).  Sums run in
 * the plain ascending order of their index.  The parallel loops only split
 * independent outputs between threads; no output depends on the thread count.
 */
#include "arc_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of later parallel loops (n >= 1); results do not depend on it. */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* ---------------------------------------------------------------------------
 * Shared random seed -> Gaussian projection V.
 *
 * Sec. IV ("Compressor Design") and Alg. 1: at iteration t all nodes agree on
 * a seed s that deterministically generates V in R^{n x r} with
 * vec(V) ~ N(0, I_{nr}).  The paper names no generator.  This oracle uses the
 * SplitMix64 generator of Steele, Lea and Flood ("Fast splittable
 * pseudorandom number generators", OOPSLA 2014): state starts at the seed and
 * advances by the golden-gamma constant; each output is the state passed
 * through the variant-13 mixing function.  Output x of the stream (0-based)
 * is therefore mix(seed + (x + 1) * gamma).
 *
 * Entry V[j][k] uses the counter c = (t*n + j)*r + k: outputs 2c and 2c+1
 * give u1 in (0,1] and u2 in [0,1) with 53 random bits each, and the
 * Box-Muller transform (Box and Muller, 1958; cosine branch) gives
 * z = sqrt(-2 ln u1) * cos(2 pi u2) in binary64, rounded once to binary32.
 * ------------------------------------------------------------------------- */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t x) {
  uint64_t z = seed + (x + 1u) * UINT64_C(0x9E3779B97F4A7C15);
  z = (z ^ (z >> 30)) * UINT64_C(0xBF58476D1CE4E5B9);
  z = (z ^ (z >> 27)) * UINT64_C(0x94D049BB133111EB);
  return z ^ (z >> 31);
}

int oracle_projection(uint64_t seed, int64_t t, int64_t n, int32_t r,
                      float *V) {
  if (n < 1 || r < 1 || V == NULL) return 1;
  const double two_pi = 6.283185307179586476925286766559;
  for (int64_t j = 0; j < n; ++j) {
    for (int32_t k = 0; k < r; ++k) {
      uint64_t c = ((uint64_t)t * (uint64_t)n + (uint64_t)j) * (uint64_t)r +
                   (uint64_t)k;
      uint64_t b1 = oracle_splitmix64(seed, 2u * c);
      uint64_t b2 = oracle_splitmix64(seed, 2u * c + 1u);
      double u1 = (double)((b1 >> 11) + 1u) * 0x1.0p-53; /* (0, 1] */
      double u2 = (double)(b2 >> 11) * 0x1.0p-53;        /* [0, 1) */
      double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
      V[j * r + k] = (float)z;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * EF21M momentum, Eq. (11a):  h_t = (1 - eta) h_{t-1} + eta * grad.
 * Binary32: a = fl(1 - eta); h = fmaf(eta, grad, fl(a * h)).
 * bf16 gradients widen to binary32 exactly (the 16 bits become the high half).
 * ------------------------------------------------------------------------- */
static float grad_at(const void *grad, int32_t is_bf16, int64_t idx) {
  if (is_bf16) {
    uint32_t bits = (uint32_t)((const uint16_t *)grad)[idx] << 16;
    float x;
    memcpy(&x, &bits, sizeof x);
    return x;
  }
  return ((const float *)grad)[idx];
}

int oracle_momentum(int32_t N, int64_t d, float eta, const void *grad,
                    int32_t grad_is_bf16, float *h) {
  if (N < 1 || d < 1 || grad == NULL || h == NULL) return 1;
  if (!(eta >= 0.0f && eta <= 1.0f)) return 1;
  const float a = 1.0f - eta;
  const int64_t total = (int64_t)N * d;
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < total; ++e) {
    float x = grad_at(grad, grad_is_bf16, e);
    float ah = a * h[e];
    h[e] = fmaf(eta, x, ah);
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Local sketch (Sec. IV and Alg. 1): P_t^{(i)} = G_t^{(i)} V, where G^{(i)} is
 * the row-major m x n view (Eq. (3)) of the compressor's argument.  In EF21M
 * (Eq. (11b)) that argument is the residual Delta^{(i)} = h_t^{(i)} -
 * g_{t-1}^{(i)}, so element e of row p is fl(h[i][e] - g[i][e]).
 * The 1/sqrt(r) factor of the text is left out, as in Alg. 1: a positive
 * scale cannot change the arg-top-K.
 * Dot product order: s = +0; s = fmaf(Delta[p*n + j], V[j][k], s) for
 * j = 0, 1, ..., n-1, stopping at the end of the vector in a ragged last row.
 * ------------------------------------------------------------------------- */
int oracle_sketch(int32_t N, int64_t d, int64_t n, int32_t r, const float *h,
                  const float *g, const float *V, float *S) {
  if (N < 1 || d < 1 || n < 1 || r < 1) return 1;
  if (h == NULL || g == NULL || V == NULL || S == NULL) return 1;
  const int64_t m = ceil_div(d, n);
  const int64_t rows = (int64_t)N * m;
#pragma omp parallel for schedule(static)
  for (int64_t ip = 0; ip < rows; ++ip) {
    const int64_t i = ip / m, p = ip % m;
    const float *hi = h + i * d, *gi = g + i * d;
    for (int32_t k = 0; k < r; ++k) {
      float s = 0.0f;
      for (int64_t j = 0; j < n; ++j) {
        const int64_t e = p * n + j;
        if (e >= d) break;
        const float delta = hi[e] - gi[e];
        s = fmaf(delta, V[j * r + k], s);
      }
      S[ip * r + k] = s;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Sketch All-Reduce (Alg. 1): P = sum over workers of P^{(i)}.
 * The paper writes a mean; the 1/N is left out because it cannot change the
 * arg-top-K.  Order: P = S[0]; P = fl(P + S[i]) for i = 1, ..., N-1.
 * ------------------------------------------------------------------------- */
int oracle_worker_sum(int32_t N, int64_t m, int32_t r, const float *S,
                      float *P) {
  if (N < 1 || m < 1 || r < 1 || S == NULL || P == NULL) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < m; ++p) {
    for (int32_t k = 0; k < r; ++k) {
      float acc = S[p * r + k];
      for (int32_t i = 1; i < N; ++i) acc = acc + S[((int64_t)i * m + p) * r + k];
      P[p * r + k] = acc;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Row importance, Eq. (4): Sigma = diag(P P^T), i.e. the squared Euclidean
 * norm of each row of P.  Order: s = +0; s = fmaf(P[p][k], P[p][k], s) for
 * k = 0, ..., r-1.
 * ------------------------------------------------------------------------- */
int oracle_importance(int64_t m, int32_t r, const float *P, float *sigma) {
  if (m < 1 || r < 1 || P == NULL || sigma == NULL) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < m; ++p) {
    float s = 0.0f;
    for (int32_t k = 0; k < r; ++k) s = fmaf(P[p * r + k], P[p * r + k], s);
    sigma[p] = s;
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Eq. (4): I = arg top_K(Sigma), the K rows of largest importance.
 * The paper does not say how ties are broken; here the lower row index wins,
 * and the selected rows are returned in ascending order.  Sigma >= +0, so
 * comparing the binary32 bit patterns as unsigned integers orders the values.
 * K larger than the number of rows selects every row (alpha = K/m = 1, the
 * identity compressor).  With buckets, each bucket [lo, hi) is an independent
 * m x n block with its own K, and the per-bucket results are concatenated.
 * Method: sort all rows of the bucket by (key descending, row ascending),
 * keep the first K, sort those ascending.
 * ------------------------------------------------------------------------- */
typedef struct {
  uint32_t key;
  int32_t row;
} keyed_row;

static int by_key_desc_row_asc(const void *pa, const void *pb) {
  const keyed_row *a = (const keyed_row *)pa, *b = (const keyed_row *)pb;
  if (a->key != b->key) return a->key > b->key ? -1 : 1;
  return (a->row > b->row) - (a->row < b->row);
}

static int by_int_asc(const void *pa, const void *pb) {
  const int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
  return (a > b) - (a < b);
}

int oracle_select(int64_t m, const float *sigma, int64_t K_global,
                  int32_t num_buckets, const int64_t *bucket_row_begin,
                  const int64_t *bucket_K, int32_t *idx, int64_t *K_total) {
  if (m < 1 || m > INT32_MAX || sigma == NULL || idx == NULL ||
      K_total == NULL)
    return 1;
  int64_t one_begin[2] = {0, m};
  int64_t one_K[1] = {K_global};
  const int64_t *begin = one_begin, *Kb = one_K;
  int32_t nb = 1;
  if (num_buckets < 0) return 1;
  if (num_buckets > 0) {
    if (bucket_row_begin == NULL || bucket_K == NULL) return 1;
    begin = bucket_row_begin;
    Kb = bucket_K;
    nb = num_buckets;
    if (begin[0] != 0 || begin[nb] != m) return 1;
    for (int32_t b = 0; b < nb; ++b)
      if (begin[b + 1] <= begin[b]) return 1;
  }
  for (int32_t b = 0; b < nb; ++b)
    if (Kb[b] < 0) return 1;

  keyed_row *rows = (keyed_row *)malloc((size_t)m * sizeof(keyed_row));
  if (rows == NULL) return 1;
  int64_t out = 0;
  for (int32_t b = 0; b < nb; ++b) {
    const int64_t lo = begin[b], hi = begin[b + 1], cnt = hi - lo;
    int64_t k = Kb[b] < cnt ? Kb[b] : cnt;
    for (int64_t p = lo; p < hi; ++p) {
      uint32_t bits;
      memcpy(&bits, &sigma[p], sizeof bits);
      rows[p - lo].key = bits;
      rows[p - lo].row = (int32_t)p;
    }
    qsort(rows, (size_t)cnt, sizeof(keyed_row), by_key_desc_row_asc);
    for (int64_t q = 0; q < k; ++q) idx[out + q] = rows[q].row;
    qsort(idx + out, (size_t)k, sizeof(int32_t), by_int_asc);
    out += k;
  }
  free(rows);
  *K_total = out;
  return 0;
}

/* ---------------------------------------------------------------------------
 * Row gather and payload All-Reduce (Eq. (5), Alg. 1 last steps) with the
 * error-feedback update of Eq. (11b).
 * C_local(Delta^{(i)}) keeps rows I of Delta^{(i)} = h_t^{(i)} - g_{t-1}^{(i)}
 * and zeroes the others; every node uses the same I, so the sum over nodes
 * needs no indices.  For each selected row p = I[q] and column j < n with
 * e = p*n + j < d:
 *   Delta_i = fl(h[i][e] - g[i][e])                      (same bits as before)
 *   agg[q][j] = Delta_0 + Delta_1 + ... + Delta_{N-1}     (ascending i)
 *   g[i][e]   = fl(g[i][e] + Delta_i)                     (Eq. (11b))
 * agg is the sum over nodes (Alg. 1's output line); the mean of Eq. (5) is
 * agg / N.  Columns past d in a ragged last row give agg = +0.
 * ------------------------------------------------------------------------- */
int oracle_gather_update(int32_t N, int64_t d, int64_t n, int64_t K_total,
                         const int32_t *idx, const float *h, float *g,
                         float *agg) {
  if (N < 1 || d < 1 || n < 1 || K_total < 0) return 1;
  if (K_total > 0 && (idx == NULL || h == NULL || g == NULL || agg == NULL))
    return 1;
  const int64_t m = ceil_div(d, n);
  for (int64_t q = 0; q < K_total; ++q)
    if (idx[q] < 0 || idx[q] >= m) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t q = 0; q < K_total; ++q) {
    const int64_t p = idx[q];
    for (int64_t j = 0; j < n; ++j) {
      const int64_t e = p * n + j;
      if (e >= d) {
        agg[q * n + j] = 0.0f;
        continue;
      }
      float acc = 0.0f;
      for (int32_t i = 0; i < N; ++i) {
        const int64_t at = (int64_t)i * d + e;
        const float delta = h[at] - g[at];
        acc = (i == 0) ? delta : acc + delta;
        g[at] = g[at] + delta;
      }
      agg[q * n + j] = acc;
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * One compressor step: Eq. (11a), then Alg. 1 applied to Delta = h_t -
 * g_{t-1}, then Eq. (11b).  The model update Eq. (11c) lies outside the
 * compressor and is not part of this step.
 * ------------------------------------------------------------------------- */
int oracle_step(int32_t N, int64_t d, int64_t n, int32_t r, float eta,
                uint64_t seed, int64_t t, int64_t K_global,
                int32_t num_buckets, const int64_t *bucket_row_begin,
                const int64_t *bucket_K, const void *grad,
                int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                float *agg, int64_t *K_total, const float *V_override,
                float *sigma_out, float *S_out) {
  if (N < 1 || d < 1 || n < 1 || r < 1 || K_total == NULL) return 1;
  const int64_t m = ceil_div(d, n);
  if (m > INT32_MAX) return 1;
  int rc = 1;
  float *V = (float *)malloc((size_t)(n * r) * sizeof(float));
  float *S = S_out ? S_out : (float *)malloc((size_t)((int64_t)N * m * r) * sizeof(float));
  float *P = (float *)malloc((size_t)(m * r) * sizeof(float));
  float *sigma = sigma_out ? sigma_out : (float *)malloc((size_t)m * sizeof(float));
  if (V == NULL || S == NULL || P == NULL || sigma == NULL) goto done;

  if (V_override)
    memcpy(V, V_override, (size_t)(n * r) * sizeof(float));
  else if (oracle_projection(seed, t, n, r, V))
    goto done;
  /* Reject a bad selection configuration before any state is touched. */
  if (num_buckets < 0 || (num_buckets == 0 && K_global < 0)) goto done;
  if (num_buckets > 0) {
    if (bucket_row_begin == NULL || bucket_K == NULL) goto done;
    if (bucket_row_begin[0] != 0 || bucket_row_begin[num_buckets] != m)
      goto done;
    for (int32_t b = 0; b < num_buckets; ++b)
      if (bucket_row_begin[b + 1] <= bucket_row_begin[b] || bucket_K[b] < 0)
        goto done;
  }
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) goto done;
  if (oracle_sketch(N, d, n, r, h, g, V, S)) goto done;
  if (oracle_worker_sum(N, m, r, S, P)) goto done;
  if (oracle_importance(m, r, P, sigma)) goto done;
  if (oracle_select(m, sigma, K_global, num_buckets, bucket_row_begin,
                    bucket_K, idx, K_total))
    goto done;
  if (oracle_gather_update(N, d, n, *K_total, idx, h, g, agg)) goto done;
  rc = 0;
done:
  free(V);
  if (!S_out) free(S);
  free(P);
  if (!sigma_out) free(sigma);
  return rc;
}

/* Gather + worker sum + EF update of the per-tensor layout (Eq. (5), (11b)),
 * tensor by tensor; tensor b's K_b selected rows (global row numbers) carry
 * cols[b] values each in the packed payload.  Returns the payload length. */
static int64_t gather_update_tensors(int32_t N, int64_t d, int32_t num_tensors,
                                     const int64_t *rows, const int64_t *cols,
                                     const int64_t *K, const int32_t *idx,
                                     const float *h, float *g, float *agg) {
  int64_t off = 0, row0 = 0, q0 = 0, a0 = 0;
  for (int32_t b = 0; b < num_tensors; ++b) {
    const int64_t mb = rows[b], nb = cols[b];
    const int64_t kb = K[b] < mb ? K[b] : mb;
#pragma omp parallel for schedule(static)
    for (int64_t q = 0; q < kb; ++q) {
      const int64_t p = idx[q0 + q] - row0;
      for (int64_t j = 0; j < nb; ++j) {
        const int64_t e = off + p * nb + j;
        float acc = 0.0f;
        for (int32_t i = 0; i < N; ++i) {
          const int64_t at = (int64_t)i * d + e;
          const float delta = h[at] - g[at];
          acc = (i == 0) ? delta : acc + delta;
          g[at] = g[at] + delta;
        }
        agg[a0 + q * nb + j] = acc;
      }
    }
    off += mb * nb;
    row0 += mb;
    q0 += kb;
    a0 += kb * nb;
  }
  return a0;
}

/* ---------------------------------------------------------------------------
 * Per-tensor mode (Sec. VI): the model's tensors are compressed one by one,
 * each in its own m_b x n_b view (2-D weights as they are, convolution
 * kernels as out x (in*kh*kw), 1-D tensors as one row kept whole), with its
 * own K_b.  Per tensor, the step is Alg. 1 applied to Delta = h_t - g_{t-1}
 * inside EF21M (11a), (11b), exactly as in oracle_step: the sketch with the
 * projection of the tensor's width, the worker sum, the importance, the
 * arg-top-K of the tensor's rows, and the gather/update of its selected
 * rows.  Tensors of the same width share V_t (V depends on (seed, t, width)).
 * Global row numbering: tensor b's rows follow tensor b-1's.
 * ------------------------------------------------------------------------- */
int oracle_step_tensors(int32_t N, int32_t r, float eta, uint64_t seed,
                        int64_t t, int32_t num_tensors, const int64_t *rows,
                        const int64_t *cols, const int64_t *K,
                        const void *grad, int32_t grad_is_bf16, float *h,
                        float *g, int32_t *idx, float *agg, int64_t *K_total,
                        int64_t *agg_len, float *sigma_out, float *S_out) {
  if (N < 1 || r < 1 || num_tensors < 1 || rows == NULL || cols == NULL ||
      K == NULL || grad == NULL || h == NULL || g == NULL || idx == NULL ||
      agg == NULL || K_total == NULL || agg_len == NULL)
    return 1;
  int64_t d = 0, m = 0;
  for (int32_t b = 0; b < num_tensors; ++b) {
    if (rows[b] < 1 || cols[b] < 1 || K[b] < 0) return 1;
    d += rows[b] * cols[b];
    m += rows[b];
  }
  if (m > INT32_MAX) return 1;
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) return 1;

  float *S = S_out ? S_out : (float *)malloc((size_t)((int64_t)N * m * r) * sizeof(float));
  float *P = (float *)malloc((size_t)(m * r) * sizeof(float));
  float *sigma = sigma_out ? sigma_out : (float *)malloc((size_t)m * sizeof(float));
  int rc = 1;
  if (S == NULL || P == NULL || sigma == NULL) goto done;

  /* Sketch, tensor by tensor, each with the projection of its width. */
  {
    int64_t off = 0, row0 = 0;
    for (int32_t b = 0; b < num_tensors; ++b) {
      const int64_t mb = rows[b], nb = cols[b];
      float *V = (float *)malloc((size_t)(nb * r) * sizeof(float));
      if (V == NULL || oracle_projection(seed, t, nb, r, V)) {
        free(V);
        goto done;
      }
#pragma omp parallel for schedule(static)
      for (int64_t ip = 0; ip < (int64_t)N * mb; ++ip) {
        const int64_t i = ip / mb, p = ip % mb;
        const float *hi = h + i * d + off + p * nb, *gi = g + i * d + off + p * nb;
        for (int32_t k = 0; k < r; ++k) {
          float acc = 0.0f;
          for (int64_t j = 0; j < nb; ++j) acc = fmaf(hi[j] - gi[j], V[j * r + k], acc);
          S[((int64_t)i * m + row0 + p) * r + k] = acc;
        }
      }
      free(V);
      off += mb * nb;
      row0 += mb;
    }
  }
  if (oracle_worker_sum(N, m, r, S, P)) goto done;
  if (oracle_importance(m, r, P, sigma)) goto done;

  /* Arg-top-K per tensor: the tensors are the buckets of the selection. */
  {
    int64_t *begin = (int64_t *)malloc((size_t)(num_tensors + 1) * sizeof(int64_t));
    if (begin == NULL) goto done;
    begin[0] = 0;
    for (int32_t b = 0; b < num_tensors; ++b) begin[b + 1] = begin[b] + rows[b];
    const int bad = oracle_select(m, sigma, 0, num_tensors, begin, K, idx, K_total);
    free(begin);
    if (bad) goto done;
  }

  *agg_len = gather_update_tensors(N, d, num_tensors, rows, cols, K, idx, h, g, agg);
  rc = 0;
done:
  if (!S_out) free(S);
  free(P);
  if (!sigma_out) free(sigma);
  return rc;
}

/* ---------------------------------------------------------------------------
 * The model step around the compressor: Eq. (11c), the optimisers of the
 * experiments (Sec. VI) and the dense warm-up before compression starts.
 *
 * The nodes never see each other's g^(i); what the second All-Reduce of
 * Alg. 1 delivers each step is the summed payload.  So every node keeps
 * G_t = sum_i g_t^(i) by adding that payload, G_t = G_{t-1} + agg_t on the
 * selected coordinates, and Eq. (11c) reads x_{t+1} = x_t - (gamma/N) G_t.
 * In exact arithmetic this equals the sum over the nodes' trackers.
 * ------------------------------------------------------------------------- */

/* Dense (identity-compressor) step: Eq. (11a), then Eq. (11b) with C = I,
 * the payload added straight into G.  Per coordinate e:
 *   Delta_i = h_i - g_i, acc = Delta_0 + Delta_1 + ... (ascending i),
 *   g_i = fl(g_i + Delta_i), G[e] = fl(G[e] + acc).                       */
int oracle_dense_step(int32_t N, int64_t d, float eta, const void *grad,
                      int32_t grad_is_bf16, float *h, float *g, float *G) {
  if (N < 1 || d < 1 || grad == NULL || h == NULL || g == NULL || G == NULL) return 1;
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < d; ++e) {
    float acc = 0.0f;
    for (int32_t i = 0; i < N; ++i) {
      const int64_t at = (int64_t)i * d + e;
      const float delta = h[at] - g[at];
      acc = (i == 0) ? delta : acc + delta;
      g[at] = g[at] + delta;
    }
    G[e] = G[e] + acc;
  }
  return 0;
}

/* G += agg at the selected rows of one m x n view: agg row q goes to the
 * coordinates [idx[q]*n, idx[q]*n + n) clipped at d. */
int oracle_accumulate_rows(int64_t d, int64_t n, int64_t K_total,
                           const int32_t *idx, const float *agg, float *G) {
  if (d < 1 || n < 1 || K_total < 0 || G == NULL) return 1;
  if (K_total > 0 && (idx == NULL || agg == NULL)) return 1;
  const int64_t m = ceil_div(d, n);
  for (int64_t q = 0; q < K_total; ++q)
    if (idx[q] < 0 || idx[q] >= m) return 1;
  for (int64_t q = 0; q < K_total; ++q)
    for (int64_t j = 0; j < n; ++j) {
      const int64_t e = (int64_t)idx[q] * n + j;
      if (e < d) G[e] = G[e] + agg[q * n + j];
    }
  return 0;
}

/* The same for the per-tensor layout: tensor b's selected rows (global row
 * numbers, tensors' rows in order) carry cols[b] values each in the packed
 * payload. */
int oracle_accumulate_tensors(int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K,
                              const int32_t *idx, const float *agg, float *G) {
  if (num_tensors < 1 || rows == NULL || cols == NULL || K == NULL || G == NULL) return 1;
  int64_t off = 0, row0 = 0, q0 = 0, a0 = 0;
  for (int32_t b = 0; b < num_tensors; ++b) {
    const int64_t kb = K[b] < rows[b] ? (K[b] < 0 ? 0 : K[b]) : rows[b];
    for (int64_t q = 0; q < kb; ++q) {
      const int64_t p = (int64_t)idx[q0 + q] - row0;
      if (p < 0 || p >= rows[b]) return 1;
      for (int64_t j = 0; j < cols[b]; ++j) {
        const int64_t e = off + p * cols[b] + j;
        G[e] = G[e] + agg[a0 + q * cols[b] + j];
      }
    }
    off += rows[b] * cols[b];
    row0 += rows[b];
    q0 += kb;
    a0 += kb * cols[b];
  }
  return 0;
}

/* Top-K's merge step (Sec. III, "System-Level Limitations of Top-K", and
 * Prop. 1): after the All-Gather every node holds the N sparse payloads
 * C_local(Delta^(i)) and sums them, C(g) = (1/N) sum_i C_local(g^(i)); the
 * nodes keep the sum G = sum_i g^(i).  Written out per coordinate e of row p:
 * the nodes i that kept row p, in ascending i, contribute their value of e;
 * the contributions are summed (the first as it is, then plain additions)
 * and the sum is added to G[e].  Rows no node kept leave G unchanged.  Node
 * i's list is idx[i*K_node .. +K_node) (rows of the view, as oracle_step_topk
 * returns them) with payload agg[i*L + q*w ..] for its q-th row of width w.
 * When every node keeps the same rows this is G += agg of the shared-row
 * compressors, whose payload is the same ascending sum. */
static int tensor_buckets(int32_t num_tensors, const int64_t *rows, const int64_t *cols,
                          const int64_t *K, int64_t *d_out, int64_t *m_out,
                          int64_t **begin_out);

static int merge_topk(int32_t N, int64_t m, const int64_t *row_off, const int64_t *row_len,
                      const int64_t *slot_of_pos, int64_t K_node, const int32_t *idx,
                      const float *agg, int64_t L, float *G) {
  int64_t *pos = (int64_t *)malloc((size_t)(N * m) * sizeof(int64_t));
  if (pos == NULL) return 1;
  for (int64_t k = 0; k < (int64_t)N * m; ++k) pos[k] = -1;
  for (int32_t i = 0; i < N; ++i)
    for (int64_t q = 0; q < K_node; ++q) {
      const int64_t p = idx[(int64_t)i * K_node + q];
      if (p < 0 || p >= m || pos[(int64_t)i * m + p] >= 0) {
        free(pos);
        return 1;
      }
      pos[(int64_t)i * m + p] = q;
    }
  for (int64_t p = 0; p < m; ++p)
    for (int64_t j = 0; j < row_len[p]; ++j) {
      float acc = 0.0f;
      int have = 0;
      for (int32_t i = 0; i < N; ++i) {
        const int64_t q = pos[(int64_t)i * m + p];
        if (q < 0) continue;
        const float c = agg[(int64_t)i * L + slot_of_pos[q] + j];
        acc = have ? acc + c : c;
        have = 1;
      }
      if (have) G[row_off[p] + j] = G[row_off[p] + j] + acc;
    }
  free(pos);
  return 0;
}

int oracle_merge_topk_rows(int32_t N, int64_t d, int64_t n, int64_t K_node,
                           const int32_t *idx, const float *agg, float *G) {
  if (N < 1 || d < 1 || n < 1 || K_node < 0 || G == NULL) return 1;
  if (K_node > 0 && (idx == NULL || agg == NULL)) return 1;
  const int64_t m = ceil_div(d, n);
  if (K_node > m) return 1;
  int64_t *row_off = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *row_len = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *slot = (int64_t *)malloc((size_t)(K_node > 0 ? K_node : 1) * sizeof(int64_t));
  int rc = 1;
  if (row_off && row_len && slot) {
    for (int64_t p = 0; p < m; ++p) {
      row_off[p] = p * n;
      row_len[p] = p * n + n <= d ? n : d - p * n;
    }
    for (int64_t q = 0; q < K_node; ++q) slot[q] = q * n;
    rc = merge_topk(N, m, row_off, row_len, slot, K_node, idx, agg, K_node * n, G);
  }
  free(row_off);
  free(row_len);
  free(slot);
  return rc;
}

int oracle_merge_topk_tensors(int32_t N, int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K, const int32_t *idx,
                              const float *agg, float *G) {
  int64_t d, m, *begin = NULL;
  if (N < 1 || G == NULL) return 1;
  if (tensor_buckets(num_tensors, rows, cols, K, &d, &m, &begin)) return 1;
  int64_t K_node = 0, L = 0;
  for (int32_t b = 0; b < num_tensors; ++b) {
    const int64_t kb = K[b] < rows[b] ? K[b] : rows[b];
    K_node += kb;
    L += kb * cols[b];
  }
  int64_t *row_off = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *row_len = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *slot = (int64_t *)malloc((size_t)(K_node > 0 ? K_node : 1) * sizeof(int64_t));
  int rc = 1;
  if (row_off && row_len && slot && (K_node == 0 || (idx != NULL && agg != NULL))) {
    int64_t off = 0, p = 0, q = 0, a0 = 0;
    for (int32_t b = 0; b < num_tensors; ++b) {
      for (int64_t r = 0; r < rows[b]; ++r, ++p) {
        row_off[p] = off + r * cols[b];
        row_len[p] = cols[b];
      }
      off += rows[b] * cols[b];
      const int64_t kb = K[b] < rows[b] ? K[b] : rows[b];
      for (int64_t r = 0; r < kb; ++r, ++q, a0 += cols[b]) slot[q] = a0;
    }
    /* A node's q-th kept row must lie in the tensor whose list holds q. */
    int ok = 1;
    {
      int64_t q0 = 0, row0 = 0;
      for (int32_t b = 0; b < num_tensors && ok; ++b) {
        const int64_t kb = K[b] < rows[b] ? K[b] : rows[b];
        for (int32_t i = 0; i < N && ok; ++i)
          for (int64_t r = 0; r < kb; ++r) {
            const int64_t pr = (int64_t)idx[(int64_t)i * K_node + q0 + r];
            if (pr < row0 || pr >= row0 + rows[b]) {
              ok = 0;
              break;
            }
          }
        q0 += kb;
        row0 += rows[b];
      }
    }
    if (ok) rc = merge_topk(N, m, row_off, row_len, slot, K_node, idx, agg, L, G);
  }
  free(row_off);
  free(row_len);
  free(slot);
  free(begin);
  return rc;
}

/* Model update x_{t+1} from G_t, coordinate by coordinate.  The direction is
 * the node average plus the L2 term: dir = fmaf(wd, x, G / N).
 *   SGD  (Eq. (11c)):  x = fmaf(-lr, dir, x)
 *   MSGD (heavy ball): u = fmaf(beta, u, dir);  x = fmaf(-lr, u, x)
 *   Adam (Kingma & Ba, Alg. 1 of "Adam", step count T >= 1):
 *     m = fmaf(beta1, m, fl((1 - beta1) * dir))
 *     v = fmaf(beta2, v, fl((1 - beta2) * fl(dir * dir)))
 *     x = fmaf(-lr, fl(fl(m / c1) / fl(sqrt(fl(v / c2)) + eps)), x)
 *   with c1 = fl(1 - beta1^T), c2 = fl(1 - beta2^T): beta^T as T binary64
 *   multiplications of 1.0 by beta, 1 - beta^T in binary64, rounded once to
 *   binary32; (1 - beta) is rounded to binary32.
 * optimizer: 0 SGD, 1 MSGD (state m = u), 2 Adam (state m, v). */
int oracle_optimizer(int32_t optimizer, int32_t N, int64_t d, int64_t T,
                     float lr, float momentum, float beta1, float beta2,
                     float eps, float weight_decay, const float *G, float *x,
                     float *m, float *v) {
  if (N < 1 || d < 1 || G == NULL || x == NULL) return 1;
  if (optimizer < 0 || optimizer > 2) return 1;
  if (optimizer >= 1 && m == NULL) return 1;
  if (optimizer == 2 && (v == NULL || T < 1)) return 1;
  const float fN = (float)N;
  const float b1c = 1.0f - beta1, b2c = 1.0f - beta2;
  double p1 = 1.0, p2 = 1.0;
  if (optimizer == 2)
    for (int64_t s = 0; s < T; ++s) {
      p1 *= (double)beta1;
      p2 *= (double)beta2;
    }
  const float c1 = (float)(1.0 - p1), c2 = (float)(1.0 - p2);
#pragma omp parallel for schedule(static)
  for (int64_t e = 0; e < d; ++e) {
    const float dir = fmaf(weight_decay, x[e], G[e] / fN);
    if (optimizer == 0) {
      x[e] = fmaf(-lr, dir, x[e]);
    } else if (optimizer == 1) {
      m[e] = fmaf(momentum, m[e], dir);
      x[e] = fmaf(-lr, m[e], x[e]);
    } else {
      m[e] = fmaf(beta1, m[e], b1c * dir);
      v[e] = fmaf(beta2, v[e], b2c * (dir * dir));
      const float mh = m[e] / c1, vh = v[e] / c2;
      const float step = mh / (sqrtf(vh) + eps);
      x[e] = fmaf(-lr, step, x[e]);
    }
  }
  return 0;
}

/* ---------------------------------------------------------------------------
 * Comparison compressors of Table I, inside the same EF21M recursion
 * (11a)-(11b) and on the same m x n row views; each keeps K rows (per bucket
 * or tensor) of Delta^(i) = h_t^(i) - g_{t-1}^(i).
 *
 * Rand-K (Sec. I-A; All-Reduce compatible): K rows drawn uniformly at random,
 * the same rows on every node (shared seed), unscaled so that the compressor
 * stays contractive with alpha = K/m.  The draw: row p gets the key
 * u_p = floor(x / 2^40), x = SplitMix64 output number t*m + p of the stream
 * seeded with the shared seed (the generator of oracle_splitmix64), as a
 * binary32 integer in [0, 2^24); the K rows with the largest keys are kept,
 * ties to the lower row, exactly the arg-top-K of Eq. (4) with u in place of
 * Sigma.  The payload is summed over nodes as for ARC-Top-K.
 *
 * Top-K (Sec. III, Prop. 1; All-Gather): each node keeps its own K rows of
 * largest squared norm ||Delta^(i)_p||^2 (an fmaf chain of squares over the
 * row's columns in ascending order from +0), ties to the lower row, and sends
 * them with their indices; nothing is summed on the wire.  idx holds node i's
 * rows at [i*K_total, (i+1)*K_total), agg its rows at [i*L, (i+1)*L) with L
 * the payload length of one node.
 * ------------------------------------------------------------------------- */
int oracle_randk_keys(uint64_t seed, int64_t t, int64_t m, float *keys) {
  if (m < 1 || t < 0 || keys == NULL) return 1;
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < m; ++p)
    keys[p] = (float)(oracle_splitmix64(seed, (uint64_t)(t * m + p)) >> 40);
  return 0;
}

int oracle_step_randk(int32_t N, int64_t d, int64_t n, float eta, uint64_t seed,
                      int64_t t, int64_t K_global, int32_t num_buckets,
                      const int64_t *bucket_row_begin, const int64_t *bucket_K,
                      const void *grad, int32_t grad_is_bf16, float *h, float *g,
                      int32_t *idx, float *agg, int64_t *K_total, float *keys_out) {
  if (N < 1 || d < 1 || n < 1 || K_total == NULL) return 1;
  const int64_t m = ceil_div(d, n);
  if (m > INT32_MAX) return 1;
  float *keys = keys_out ? keys_out : (float *)malloc((size_t)m * sizeof(float));
  int rc = 1;
  if (keys == NULL) return 1;
  if (oracle_randk_keys(seed, t, m, keys)) goto done;
  /* Validate the selection on the keys before touching the state. */
  if (oracle_select(m, keys, K_global, num_buckets, bucket_row_begin, bucket_K, idx, K_total))
    goto done;
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) goto done;
  if (oracle_gather_update(N, d, n, *K_total, idx, h, g, agg)) goto done;
  rc = 0;
done:
  if (!keys_out) free(keys);
  return rc;
}

static int tensor_buckets(int32_t num_tensors, const int64_t *rows, const int64_t *cols,
                          const int64_t *K, int64_t *d_out, int64_t *m_out,
                          int64_t **begin_out) {
  if (num_tensors < 1 || rows == NULL || cols == NULL || K == NULL) return 1;
  int64_t d = 0, m = 0;
  for (int32_t b = 0; b < num_tensors; ++b) {
    if (rows[b] < 1 || cols[b] < 1 || K[b] < 0) return 1;
    d += rows[b] * cols[b];
    m += rows[b];
  }
  if (m > INT32_MAX) return 1;
  int64_t *begin = (int64_t *)malloc((size_t)(num_tensors + 1) * sizeof(int64_t));
  if (begin == NULL) return 1;
  begin[0] = 0;
  for (int32_t b = 0; b < num_tensors; ++b) begin[b + 1] = begin[b] + rows[b];
  *d_out = d;
  *m_out = m;
  *begin_out = begin;
  return 0;
}

int oracle_step_randk_tensors(int32_t N, float eta, uint64_t seed, int64_t t,
                              int32_t num_tensors, const int64_t *rows,
                              const int64_t *cols, const int64_t *K, const void *grad,
                              int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                              float *agg, int64_t *K_total, int64_t *agg_len,
                              float *keys_out) {
  int64_t d, m, *begin = NULL;
  if (N < 1 || idx == NULL || agg == NULL || K_total == NULL || agg_len == NULL) return 1;
  if (tensor_buckets(num_tensors, rows, cols, K, &d, &m, &begin)) return 1;
  float *keys = keys_out ? keys_out : (float *)malloc((size_t)m * sizeof(float));
  int rc = 1;
  if (keys == NULL) goto done;
  if (oracle_randk_keys(seed, t, m, keys)) goto done;
  if (oracle_select(m, keys, 0, num_tensors, begin, K, idx, K_total)) goto done;
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) goto done;
  *agg_len = gather_update_tensors(N, d, num_tensors, rows, cols, K, idx, h, g, agg);
  rc = 0;
done:
  if (!keys_out) free(keys);
  free(begin);
  return rc;
}

/* Squared norm of row p of node i's Delta: columns [off, off + len) of the
 * node's vector, fmaf chain in ascending column order from +0. */
static float row_norm2(const float *h, const float *g, int64_t off, int64_t len) {
  float acc = 0.0f;
  for (int64_t j = 0; j < len; ++j) {
    const float delta = h[off + j] - g[off + j];
    acc = fmaf(delta, delta, acc);
  }
  return acc;
}

/* Node i's own rows: payload values are Delta^(i) itself (nothing summed),
 * and g^(i) = fl(g^(i) + Delta^(i)) on those rows (Eq. (11b)). */
static void gather_own_row(const float *hi, float *gi, int64_t off, int64_t len, int64_t width,
                           float *out) {
  for (int64_t j = 0; j < width; ++j) {
    if (j >= len) {
      out[j] = 0.0f;
      continue;
    }
    const float delta = hi[off + j] - gi[off + j];
    out[j] = delta;
    gi[off + j] = gi[off + j] + delta;
  }
}

int oracle_step_topk(int32_t N, int64_t d, int64_t n, float eta, int64_t K_global,
                     int32_t num_buckets, const int64_t *bucket_row_begin,
                     const int64_t *bucket_K, const void *grad, int32_t grad_is_bf16,
                     float *h, float *g, int32_t *idx, float *agg, int64_t *K_total,
                     float *norms_out) {
  if (N < 1 || d < 1 || n < 1 || idx == NULL || K_total == NULL) return 1;
  const int64_t m = ceil_div(d, n);
  if (m > INT32_MAX) return 1;
  float *norms = norms_out ? norms_out : (float *)malloc((size_t)(N * m) * sizeof(float));
  int rc = 1;
  if (norms == NULL) return 1;
  /* Validate the selection configuration (on zero keys) before the state. */
  for (int64_t p = 0; p < m; ++p) norms[p] = 0.0f;
  if (oracle_select(m, norms, K_global, num_buckets, bucket_row_begin, bucket_K, idx, K_total))
    goto done;
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) goto done;
#pragma omp parallel for schedule(static)
  for (int64_t ip = 0; ip < (int64_t)N * m; ++ip) {
    const int64_t i = ip / m, p = ip % m;
    const int64_t len = p * n + n <= d ? n : d - p * n;
    norms[ip] = row_norm2(h + i * d, g + i * d, p * n, len);
  }
  {
    int64_t kt = 0;
    for (int32_t i = 0; i < N; ++i) {
      if (oracle_select(m, norms + (int64_t)i * m, K_global, num_buckets, bucket_row_begin,
                        bucket_K, idx + (int64_t)i * *K_total, &kt))
        goto done;
    }
  }
  if (*K_total > 0 && agg == NULL) goto done;
#pragma omp parallel for schedule(static)
  for (int64_t iq = 0; iq < (int64_t)N * *K_total; ++iq) {
    const int64_t i = iq / *K_total, p = idx[iq];
    const int64_t len = p * n + n <= d ? n : d - p * n;
    gather_own_row(h + i * d, g + i * d, p * n, len, n, agg + iq * n);
  }
  rc = 0;
done:
  if (!norms_out) free(norms);
  return rc;
}

int oracle_step_topk_tensors(int32_t N, float eta, int32_t num_tensors, const int64_t *rows,
                             const int64_t *cols, const int64_t *K, const void *grad,
                             int32_t grad_is_bf16, float *h, float *g, int32_t *idx,
                             float *agg, int64_t *K_total, int64_t *agg_len,
                             float *norms_out) {
  int64_t d, m, *begin = NULL;
  if (N < 1 || idx == NULL || K_total == NULL || agg_len == NULL) return 1;
  if (tensor_buckets(num_tensors, rows, cols, K, &d, &m, &begin)) return 1;
  float *norms = norms_out ? norms_out : (float *)malloc((size_t)(N * m) * sizeof(float));
  int64_t *row_off = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *row_len = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int64_t *slot = (int64_t *)malloc((size_t)m * sizeof(int64_t));
  int rc = 1;
  if (norms == NULL || row_off == NULL || row_len == NULL || slot == NULL) goto done;
  /* Row p of tensor b starts at the tensor's offset + (p - row0_b) * cols_b. */
  {
    int64_t off = 0, p = 0;
    for (int32_t b = 0; b < num_tensors; ++b) {
      for (int64_t r = 0; r < rows[b]; ++r, ++p) {
        row_off[p] = off + r * cols[b];
        row_len[p] = cols[b];
      }
      off += rows[b] * cols[b];
    }
  }
  /* Validate the selection configuration (on zero keys) before the state. */
  for (int64_t p = 0; p < m; ++p) norms[p] = 0.0f;
  if (oracle_select(m, norms, 0, num_tensors, begin, K, idx, K_total)) goto done;
  if (*K_total > 0 && agg == NULL) goto done;
  /* Payload slot of output position q: tensors in order, K_b rows of cols_b. */
  {
    int64_t q = 0, a0 = 0;
    for (int32_t b = 0; b < num_tensors; ++b) {
      const int64_t kb = K[b] < rows[b] ? K[b] : rows[b];
      for (int64_t r = 0; r < kb; ++r, ++q, a0 += cols[b]) slot[q] = a0;
    }
    *agg_len = a0;
  }
  if (oracle_momentum(N, d, eta, grad, grad_is_bf16, h)) goto done;
#pragma omp parallel for schedule(static)
  for (int64_t ip = 0; ip < (int64_t)N * m; ++ip) {
    const int64_t i = ip / m, p = ip % m;
    norms[ip] = row_norm2(h + i * d, g + i * d, row_off[p], row_len[p]);
  }
  {
    int64_t kt = 0;
    for (int32_t i = 0; i < N; ++i)
      if (oracle_select(m, norms + (int64_t)i * m, 0, num_tensors, begin, K,
                        idx + (int64_t)i * *K_total, &kt))
        goto done;
  }
#pragma omp parallel for schedule(static)
  for (int64_t iq = 0; iq < (int64_t)N * *K_total; ++iq) {
    const int64_t i = iq / *K_total, q = iq % *K_total, p = idx[iq];
    gather_own_row(h + i * d, g + i * d, row_off[p], row_len[p], row_len[p],
                   agg + i * *agg_len + slot[q]);
  }
  rc = 0;
done:
  if (!norms_out) free(norms);
  free(row_off);
  free(row_len);
  free(slot);
  free(begin);
  return rc;
}
