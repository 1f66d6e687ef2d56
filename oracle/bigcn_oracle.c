/*
 * Plain CPU oracle for binarized-GCN (Bi-GCN) inference.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the GPU path is
 * compared against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it; the product path never does.  It shares no
 * code, header or table with the HIP library.
 *
 * It follows the paper ("Bi-GCN: Binary Graph Convolutional Network",
 * Wang et al., CVPR 2021) step by step, slowly and in double precision:
 *
 *   Sec. 3.1   Â = A + I, D̂_ii = sum_j Â_ij (the CSR given holds Â).
 *   Eq. (1)    Ã = D̂^-1/2 Â D̂^-1/2 (symmetric normalisation); the
 *              mean-aggregation variant Ã = D̂^-1 Â is also offered.
 *   Eq. (3)    B_j = sign(W_:,j)          one bucket per column of W
 *   Eq. (4)    α_j = ||W_:,j||_1 / d_in   (see reading R1 below)
 *   Eq. (7)    β_i = ||H_i,:||_1 / d_in   (see reading R2 below)
 *   Eq. (8)    F_i = sign(H_i,:)          one bucket per row of H
 *   Eq. (11)   ζ_ij = β_i α_j (F_i,: · B_:,j)   a ±1 inner product
 *   Eq. (13)   H_b = Ã ζ
 *
 * Readings of points the paper leaves open (each is listed in the design
 * notes of the repository):
 *   R1  Eq. (4) prints the divisor d_out; the oracle divides by d_in, the
 *       length of the bucket, which is the optimal scale of vector
 *       binarisation the text invokes and the only divisor consistent with
 *       the 1/d_in term of the weight gradient, Eq. (15).
 *   R2  Eq. (7) prints the divisor N; the oracle divides by d_in for the
 *       same reason (β_i is the mean magnitude of the bucket H_i,:).
 *   R3  sign(y) = +1 if y >= 0 else -1 (IEEE compare; +0 and -0 give +1),
 *       since F and B are stated to lie in {-1, 1}.  Inputs must be finite.
 *   R4  Bit layout: element k of a row goes to 64-bit word k / 64, bit
 *       k % 64; a set bit means +1.  Bits at k >= d_in and any further pad
 *       words are zero.
 *   R5  Layer-0 input standardisation (the input batch normalisation of the
 *       evaluation set-up, Sec. 6.2): y = fl32(fl32(x - mu) * rstd), two
 *       separately rounded fp32 operations.
 *   R6  No activation by default (the binarisation of the next layer's
 *       input acts as the non-linearity, Sec. 4.1); ReLU is optional.  A
 *       per-channel bias is optional.
 *   R10 The two-weight GraphSAGE layer (oracle_sage_layer) transforms
 *       before it aggregates, as Eq. (13) does; see that function.
 *   R12 Back propagation (oracle_layer_backward): Eq. (14) as printed,
 *       the indicator on the magnitude of dL/dH~ itself; no term for the
 *       dependence of β on H (Eq. (14) has none); the straight-through
 *       estimator 1[|W| < 1] for dB/dW in Eq. (15).
 *
 * Every reduction runs sequentially in a fixed order in double precision;
 * OpenMP only splits independent rows, so results do not depend on the
 * thread count.  Built with -ffp-contract=off.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_NORM_SYM 0
#define ORACLE_NORM_MEAN 1
#define ORACLE_ACT_NONE 0
#define ORACLE_ACT_RELU 1

/* ---------------------------------------------------------------------
 * Binarisation of one bucket (Eqs. (3)-(4) for a column of W, read from a
 * row of W^T; Eqs. (7)-(8) for a row of H).
 *   bits  : ldw words, R4 layout
 *   scale : mean |y| over the bucket (R1/R2)
 * If mu and rstd are given, the bucket is first standardised (R5).
 * Returns 0, or -1 if an element is not finite.
 * ------------------------------------------------------------------- */
static int binarize_bucket(const float* x, int32_t len, const float* mu,
                           const float* rstd, uint64_t* bits, int64_t ldw,
                           double* scale) {
  double l1 = 0.0;
  for (int64_t w = 0; w < ldw; ++w) bits[w] = 0;
  for (int32_t k = 0; k < len; ++k) {
    float y = x[k];
    if (mu != NULL) {
      float t = x[k] - mu[k]; /* first fp32 rounding */
      y = t * rstd[k];        /* second fp32 rounding */
    }
    if (!isfinite(y)) return -1;
    if (y >= 0.0f) bits[k / 64] |= (uint64_t)1 << (k % 64);
    l1 += fabs((double)y);
  }
  *scale = l1 / (double)len;
  return 0;
}

/* Sign of element k of a packed bucket: +1 for a set bit, -1 otherwise. */
static int sign_at(const uint64_t* bits, int32_t k) {
  return ((bits[k / 64] >> (k % 64)) & 1u) ? 1 : -1;
}

/* ---------------------------------------------------------------------
 * oracle_binarize: binarise rows of a row-major fp32 matrix.
 *   x      [rows][ldx], the first `cols` elements of each row are used
 *   mu, rstd  nullable pair of fp32[cols] (R5)
 *   ids    nullable list of n_ids row indices; NULL = all rows in order
 *   bits   [n_out][ldw] with n_out = n_ids or rows
 *   scale  [n_out] doubles (β for node rows, α for rows of W^T)
 * Returns 0, or -1 on a non-finite input.
 * ------------------------------------------------------------------- */
int oracle_binarize(const float* x, int64_t rows, int32_t cols, int64_t ldx,
                    const float* mu, const float* rstd, const int64_t* ids,
                    int64_t n_ids, uint64_t* bits, int64_t ldw,
                    double* scale) {
  int64_t n_out = ids ? n_ids : rows;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t r = 0; r < n_out; ++r) {
    int64_t src = ids ? ids[r] : r;
    if (binarize_bucket(x + src * ldx, cols, mu, rstd, bits + r * ldw, ldw,
                        scale + r) != 0)
      bad = 1;
  }
  return bad ? -1 : 0;
}

/* ---------------------------------------------------------------------
 * oracle_sign_dot: the ±1 inner products of Eq. (11),
 *   dot[i][j] = sum_{k<K} s(F_i, k) * s(B_j, k),
 * decoding each sign from its bit and multiplying, term by term.
 *   F [m][ldf], B [nout][ldb], dot [m][ldd] (int64)
 * ------------------------------------------------------------------- */
void oracle_sign_dot(const uint64_t* F, int64_t m, int64_t ldf,
                     const uint64_t* B, int32_t nout, int64_t ldb, int32_t K,
                     int64_t* dot, int64_t ldd) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < m; ++i) {
    for (int32_t j = 0; j < nout; ++j) {
      int64_t acc = 0;
      for (int32_t k = 0; k < K; ++k)
        acc += (int64_t)sign_at(F + i * ldf, k) * sign_at(B + j * ldb, k);
      dot[i * ldd + j] = acc;
    }
  }
}

/* Normalised adjacency entry Ã_ij for an edge (i, j) of Â, Eq. (1). */
static double atilde(int norm, int64_t deg_i, int64_t deg_j) {
  if (norm == ORACLE_NORM_MEAN) return 1.0 / (double)deg_i;
  return 1.0 / sqrt((double)deg_i * (double)deg_j);
}

/* Eq. (13) for listed output rows.  Source node j's β and dot row sit at
 * position slot[j] of beta / dot (slot == NULL: position j).  Row i of
 * the result is the sum over the neighbours j of row i of Â, taken in CSR
 * order, of Ã_ij times the row ζ_j: each element z_ik is a sequential sum
 * 0 + t_1k + t_2k + ... (+ b_k), the neighbours visited in CSR order. */
static void aggregate_rows(const int64_t* rowptr, const int32_t* colidx,
                           int norm, const int64_t* slot, const double* beta,
                           const double* alpha, const int64_t* dot,
                           int64_t ldd, int32_t d, const float* bias, int act,
                           const int64_t* ids, int64_t n_out, double* z,
                           double* mass, float* out) {
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t r = 0; r < n_out; ++r) {
    int64_t i = ids ? ids[r] : r;
    int64_t deg_i = rowptr[i + 1] - rowptr[i];
    double* zr = z + r * d;
    double* mr = mass + r * d;
    for (int32_t k = 0; k < d; ++k) {
      zr[k] = 0.0;
      mr[k] = 0.0;
    }
    for (int64_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      int64_t j = colidx[e];
      int64_t c = slot ? slot[j] : j;
      int64_t deg_j = rowptr[j + 1] - rowptr[j];
      for (int32_t k = 0; k < d; ++k) {
        double zeta = beta[c] * alpha[k] * (double)dot[c * ldd + k]; /* (11) */
        double t = atilde(norm, deg_i, deg_j) * zeta;                /* (13) */
        zr[k] += t;
        mr[k] += fabs(t);
      }
    }
    for (int32_t k = 0; k < d; ++k) {
      if (bias != NULL) {
        zr[k] += (double)bias[k];
        mr[k] += fabs((double)bias[k]);
      }
      double v = (act == ORACLE_ACT_RELU && zr[k] < 0.0) ? 0.0 : zr[k];
      out[r * d + k] = (float)v;
    }
  }
}

/* ---------------------------------------------------------------------
 * oracle_aggregate: Eq. (13) with ζ from Eq. (11), for listed output rows:
 *   z[i][k]    = sum_{j in row i of Â} Ã_ij * (β_j * α_k * dot[j][k]) + b_k
 *   mass[i][k] = sum_j |Ã_ij * β_j * α_k * dot[j][k]| + |b_k|
 *   out[i][k]  = fl32(act(z[i][k]))
 * Neighbours are visited in CSR order and summed sequentially.
 *   beta  [n] doubles, alpha [d] doubles, dot [n][ldd] int64
 *   bias  nullable fp32[d]
 *   ids   nullable list of n_ids output rows (NULL = all n rows)
 *   z, mass [n_out][d] doubles; out [n_out][d] fp32
 * ------------------------------------------------------------------- */
void oracle_aggregate(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                      int norm, const double* beta, const double* alpha,
                      const int64_t* dot, int64_t ldd, int32_t d,
                      const float* bias, int act, const int64_t* ids,
                      int64_t n_ids, double* z, double* mass, float* out) {
  aggregate_rows(rowptr, colidx, norm, NULL, beta, alpha, dot, ldd, d, bias,
                 act, ids, ids ? n_ids : n, z, mass, out);
}

/* ---------------------------------------------------------------------
 * oracle_layer: one binarised graph-convolution layer, Eqs. (3)-(13), for
 * the listed output rows (all rows if ids == NULL).
 *   h     [n][ldh] fp32 layer input H^(l); mu/rstd nullable (layer 0, R5)
 *   wt    [d_out][d_in] fp32 = W^T (row j of W^T is column j of W)
 *   bias  nullable fp32[d_out]; act = ORACLE_ACT_NONE or _RELU
 * Only the source nodes some listed row reaches are binarised and
 * multiplied.  Outputs as in oracle_aggregate; alpha_out (nullable,
 * [d_out]) receives α.  Returns 0, -1 on a non-finite input, -2 on
 * allocation failure.
 * ------------------------------------------------------------------- */
int oracle_layer(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                 int norm, const float* h, int64_t ldh, int32_t d_in,
                 const float* mu, const float* rstd, const float* wt,
                 int32_t d_out, const float* bias, int act, const int64_t* ids,
                 int64_t n_ids, double* z, double* mass, float* out,
                 double* alpha_out) {
  const int64_t ldw = (d_in + 63) / 64;
  int64_t n_out = ids ? n_ids : n;
  int rc = 0;

  /* Weights: B and α, one bucket per output channel. */
  uint64_t* wbits = calloc((size_t)d_out * ldw, sizeof(uint64_t));
  double* alpha = calloc((size_t)d_out, sizeof(double));
  /* Source nodes reached by the listed rows, in node order. */
  int64_t* slot = malloc((size_t)n * sizeof(int64_t));
  if (!wbits || !alpha || !slot) {
    rc = -2;
    goto done_w;
  }
  if (oracle_binarize(wt, d_out, d_in, d_in, NULL, NULL, NULL, 0, wbits, ldw,
                      alpha) != 0) {
    rc = -1;
    goto done_w;
  }
  if (alpha_out) memcpy(alpha_out, alpha, (size_t)d_out * sizeof(double));

  for (int64_t j = 0; j < n; ++j) slot[j] = -1;
  for (int64_t r = 0; r < n_out; ++r) {
    int64_t i = ids ? ids[r] : r;
    for (int64_t e = rowptr[i]; e < rowptr[i + 1]; ++e) slot[colidx[e]] = 0;
  }
  int64_t n_src = 0;
  for (int64_t j = 0; j < n; ++j)
    if (slot[j] == 0) slot[j] = n_src++;
    else slot[j] = -1;

  {
    int64_t* src_ids = malloc((size_t)(n_src ? n_src : 1) * sizeof(int64_t));
    uint64_t* fbits = calloc((size_t)(n_src ? n_src : 1) * ldw, sizeof(uint64_t));
    double* beta_c = calloc((size_t)(n_src ? n_src : 1), sizeof(double));
    int64_t* dot_c = calloc((size_t)(n_src ? n_src : 1) * d_out, sizeof(int64_t));
    if (!src_ids || !fbits || !beta_c || !dot_c) {
      rc = -2;
      goto done_s;
    }
    for (int64_t j = 0; j < n; ++j)
      if (slot[j] >= 0) src_ids[slot[j]] = j;
    /* Node features: F and β, one bucket per row (Eqs. (7)-(8)). */
    if (oracle_binarize(h, n, d_in, ldh, mu, rstd, src_ids, n_src, fbits, ldw,
                        beta_c) != 0) {
      rc = -1;
      goto done_s;
    }
    /* ±1 inner products (Eq. (11)). */
    oracle_sign_dot(fbits, n_src, ldw, wbits, d_out, ldw, d_in, dot_c, d_out);

    /* Aggregation (Eq. (13)), row by row, neighbours in CSR order. */
    aggregate_rows(rowptr, colidx, norm, slot, beta_c, alpha, dot_c, d_out,
                   d_out, bias, act, ids, n_out, z, mass, out);
  done_s:
    free(src_ids);
    free(fbits);
    free(beta_c);
    free(dot_c);
  }
done_w:
  free(wbits);
  free(alpha);
  free(slot);
  return rc;
}

/* ---------------------------------------------------------------------
 * oracle_sage_layer: a binarised two-weight GraphSAGE layer with the mean
 * aggregator.  The paper binarises every feature-extraction step of the
 * models it generalises (Sec. 6, Table 3); GraphSAGE has a self and a
 * neighbour weight matrix (the model sizes of Table 3 are twice those of
 * the one-matrix GCN), and its cycle-operation count charges the
 * aggregation at the output width, i.e. the transform comes first as in
 * Eq. (13) (reading R10):
 *   ζs_ik = β_i α^s_k (F_i · B^s_k),   ζn_jk = β_j α^n_k (F_j · B^n_k)
 *   z_ik  = ζs_ik + sum_{j in N(i)} ζn_jk / |N(i)| + b_k
 * with N(i) the CSR row of i (the graph A without self-loops; an empty row
 * contributes nothing), F, β, B, α from Eqs. (3)-(8).
 *   mass_ik = |ζs_ik| + sum_j |ζn_jk| / |N(i)| + |b_k|;  out = fl32(act(z))
 *   wt_self, wt_neigh  [d_out][d_in] fp32 = W^T of the two matrices
 *   alpha_self / alpha_neigh  nullable [d_out] outputs
 * Only the listed rows and their neighbours are binarised.  Returns 0, -1
 * on a non-finite input, -2 on allocation failure.
 * ------------------------------------------------------------------- */
int oracle_sage_layer(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                      const float* h, int64_t ldh, int32_t d_in, const float* mu,
                      const float* rstd, const float* wt_self,
                      const float* wt_neigh, int32_t d_out, const float* bias,
                      int act, const int64_t* ids, int64_t n_ids, double* z,
                      double* mass, float* out, double* alpha_self_out,
                      double* alpha_neigh_out) {
  const int64_t ldw = (d_in + 63) / 64;
  int64_t n_out = ids ? n_ids : n;
  int rc = 0;
  uint64_t* bs = calloc((size_t)d_out * ldw, sizeof(uint64_t));
  uint64_t* bn = calloc((size_t)d_out * ldw, sizeof(uint64_t));
  double* as = calloc((size_t)d_out, sizeof(double));
  double* an = calloc((size_t)d_out, sizeof(double));
  int64_t* slot = malloc((size_t)(n ? n : 1) * sizeof(int64_t));
  int64_t* src_ids = NULL;
  uint64_t* fbits = NULL;
  double* beta = NULL;
  int64_t *dots = NULL, *dotn = NULL;
  if (!bs || !bn || !as || !an || !slot) {
    rc = -2;
    goto done;
  }
  /* Both weight matrices: B and α, one bucket per output channel. */
  if (oracle_binarize(wt_self, d_out, d_in, d_in, NULL, NULL, NULL, 0, bs, ldw,
                      as) != 0 ||
      oracle_binarize(wt_neigh, d_out, d_in, d_in, NULL, NULL, NULL, 0, bn, ldw,
                      an) != 0) {
    rc = -1;
    goto done;
  }
  if (alpha_self_out) memcpy(alpha_self_out, as, (size_t)d_out * sizeof(double));
  if (alpha_neigh_out) memcpy(alpha_neigh_out, an, (size_t)d_out * sizeof(double));

  /* Nodes needed: the listed rows (self term) and their neighbours. */
  for (int64_t j = 0; j < n; ++j) slot[j] = -1;
  for (int64_t r = 0; r < n_out; ++r) {
    int64_t i = ids ? ids[r] : r;
    slot[i] = 0;
    for (int64_t e = rowptr[i]; e < rowptr[i + 1]; ++e) slot[colidx[e]] = 0;
  }
  int64_t n_src = 0;
  for (int64_t j = 0; j < n; ++j) slot[j] = slot[j] == 0 ? n_src++ : -1;
  src_ids = malloc((size_t)(n_src ? n_src : 1) * sizeof(int64_t));
  fbits = calloc((size_t)(n_src ? n_src : 1) * ldw, sizeof(uint64_t));
  beta = calloc((size_t)(n_src ? n_src : 1), sizeof(double));
  dots = calloc((size_t)(n_src ? n_src : 1) * d_out, sizeof(int64_t));
  dotn = calloc((size_t)(n_src ? n_src : 1) * d_out, sizeof(int64_t));
  if (!src_ids || !fbits || !beta || !dots || !dotn) {
    rc = -2;
    goto done;
  }
  for (int64_t j = 0; j < n; ++j)
    if (slot[j] >= 0) src_ids[slot[j]] = j;
  /* Node features: F and β (Eqs. (7)-(8)); both ±1 products (Eq. (11)). */
  if (oracle_binarize(h, n, d_in, ldh, mu, rstd, src_ids, n_src, fbits, ldw,
                      beta) != 0) {
    rc = -1;
    goto done;
  }
  oracle_sign_dot(fbits, n_src, ldw, bs, d_out, ldw, d_in, dots, d_out);
  oracle_sign_dot(fbits, n_src, ldw, bn, d_out, ldw, d_in, dotn, d_out);

  /* Row i: the self term, then the neighbours in CSR order, then the
   * bias, each element a sequential sum in that order. */
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t r = 0; r < n_out; ++r) {
    int64_t i = ids ? ids[r] : r;
    int64_t deg = rowptr[i + 1] - rowptr[i];
    int64_t ci = slot[i];
    double* zr = z + r * d_out;
    double* mr = mass + r * d_out;
    for (int32_t k = 0; k < d_out; ++k) {
      double self = beta[ci] * as[k] * (double)dots[ci * d_out + k];
      zr[k] = self;
      mr[k] = fabs(self);
    }
    for (int64_t e = rowptr[i]; e < rowptr[i + 1]; ++e) {
      int64_t c = slot[colidx[e]];
      for (int32_t k = 0; k < d_out; ++k) {
        double t = beta[c] * an[k] * (double)dotn[c * d_out + k] / (double)deg;
        zr[k] += t;
        mr[k] += fabs(t);
      }
    }
    for (int32_t k = 0; k < d_out; ++k) {
      if (bias != NULL) {
        zr[k] += (double)bias[k];
        mr[k] += fabs((double)bias[k]);
      }
      double v = (act == ORACLE_ACT_RELU && zr[k] < 0.0) ? 0.0 : zr[k];
      out[r * d_out + k] = (float)v;
    }
  }
done:
  free(bs);
  free(bn);
  free(as);
  free(an);
  free(slot);
  free(src_ids);
  free(fbits);
  free(beta);
  free(dots);
  free(dotn);
  return rc;
}

/* ---------------------------------------------------------------------
 * oracle_layer_backward: the back propagation of one binarised layer,
 * Alg. 1 with Eqs. (14)-(15), in the order the algorithm states it:
 *   G      = dL/dH^(l+1), masked by 1[out > 0] when the layer has ReLU
 *   db_k   = sum_i G_ik                         (the optional bias)
 *   dζ     = Ã^T G                              (first step of Alg. 1)
 *   dW~    = H~^T dζ,   H~ = diag(β) F          (Eqs. (7)-(8))
 *   dH~    = dζ W~^T,   W~ = B diag(α)          (Eqs. (3)-(4))
 *   dH     = dH~ * 1[|dH~| < 1]                 (Eq. (14), reading R12)
 *   dW_ij  = (1/d_in) B_ij sum_k dW~_kj B_kj + α_j dW~_ij 1[|W_ij| < 1]
 *                                               (Eq. (15), straight-through
 *                                                estimator for sign)
 * Ã^T is taken on the CSR of Â, which must be structurally symmetric (an
 * undirected graph with self-loops): (Ã^T G)_j = sum_{i in N(j)} Ã_ij G_i.
 * Every sum runs sequentially in a fixed order in double precision.
 *   h     [n][ldh] fp32 layer input H (before binarisation)
 *   wt    [d_out][d_in] fp32 W^T;  gout [n][d_out] fp32 dL/dH^(l+1)
 *   out   [n][d_out] fp32 forward output (read only for ReLU; nullable else)
 * Outputs (doubles):  dzeta, mass_dzeta [n][d_out]; dwt_tilde, mass_dwt
 *   [d_out][d_in] (W^T layout); dh_tilde, mass_dh [n][d_in]; dh [n][d_in];
 *   dwt [d_out][d_in]; db [d_out].  mass_* hold the sum of the absolute
 *   values of the terms of each entry.
 * Returns 0, -1 on a non-finite input, -2 on allocation failure.
 * ------------------------------------------------------------------- */
int oracle_layer_backward(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                          int norm, const float* h, int64_t ldh, int32_t d_in,
                          const float* wt, int32_t d_out, const float* gout,
                          const float* out, int act, double* dzeta,
                          double* mass_dzeta, double* dwt_tilde, double* mass_dwt,
                          double* dh_tilde, double* mass_dh, double* dh, double* dwt,
                          double* db) {
  const int64_t ldw = (d_in + 63) / 64;
  int rc = 0;
  uint64_t* fbits = calloc((size_t)(n ? n : 1) * ldw, sizeof(uint64_t));
  double* beta = calloc((size_t)(n ? n : 1), sizeof(double));
  uint64_t* wbits = calloc((size_t)d_out * ldw, sizeof(uint64_t));
  double* alpha = calloc((size_t)d_out, sizeof(double));
  double* G = calloc((size_t)(n ? n : 1) * d_out, sizeof(double));
  if (!fbits || !beta || !wbits || !alpha || !G) {
    rc = -2;
    goto done;
  }
  if (oracle_binarize(h, n, d_in, ldh, NULL, NULL, NULL, 0, fbits, ldw, beta) != 0 ||
      oracle_binarize(wt, d_out, d_in, d_in, NULL, NULL, NULL, 0, wbits, ldw, alpha) != 0) {
    rc = -1;
    goto done;
  }
  /* The incoming gradient, through the activation. */
  for (int64_t i = 0; i < n; ++i)
    for (int32_t k = 0; k < d_out; ++k) {
      double gv = (double)gout[i * d_out + k];
      if (act == ORACLE_ACT_RELU && !(out[i * d_out + k] > 0.0f)) gv = 0.0;
      G[i * d_out + k] = gv;
    }
  /* Bias: dL/db_k = sum_i G_ik. */
  for (int32_t k = 0; k < d_out; ++k) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += G[i * d_out + k];
    db[k] = s;
  }
  /* dζ = Ã^T G, row j gathering the rows i of its (symmetric) neighbourhood. */
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t j = 0; j < n; ++j) {
    int64_t deg_j = rowptr[j + 1] - rowptr[j];
    for (int32_t k = 0; k < d_out; ++k) {
      double s = 0.0, m = 0.0;
      for (int64_t e = rowptr[j]; e < rowptr[j + 1]; ++e) {
        int64_t i = colidx[e];
        int64_t deg_i = rowptr[i + 1] - rowptr[i];
        double t = atilde(norm, deg_i, deg_j) * G[i * d_out + k];  /* Ã_ij G_ik */
        s += t;
        m += fabs(t);
      }
      dzeta[j * d_out + k] = s;
      mass_dzeta[j * d_out + k] = m;
    }
  }
  /* dW~ = H~^T dζ: entry (k in d_in, j in d_out), stored at [j][k]. */
#pragma omp parallel for schedule(dynamic, 4)
  for (int32_t j = 0; j < d_out; ++j)
    for (int32_t k = 0; k < d_in; ++k) {
      double s = 0.0, m = 0.0;
      for (int64_t i = 0; i < n; ++i) {
        double ht = beta[i] * (double)sign_at(fbits + i * ldw, k);  /* H~_ik */
        double t = ht * dzeta[i * d_out + j];
        s += t;
        m += fabs(t);
      }
      dwt_tilde[(int64_t)j * d_in + k] = s;
      mass_dwt[(int64_t)j * d_in + k] = m;
    }
  /* dH~ = dζ W~^T and Eq. (14). */
#pragma omp parallel for schedule(dynamic, 16)
  for (int64_t i = 0; i < n; ++i)
    for (int32_t k = 0; k < d_in; ++k) {
      double s = 0.0, m = 0.0;
      for (int32_t j = 0; j < d_out; ++j) {
        double wtl = (double)sign_at(wbits + (int64_t)j * ldw, k) * alpha[j];  /* W~_kj */
        double t = dzeta[i * d_out + j] * wtl;
        s += t;
        m += fabs(t);
      }
      dh_tilde[i * d_in + k] = s;
      mass_dh[i * d_in + k] = m;
      dh[i * d_in + k] = fabs(s) < 1.0 ? s : 0.0;
    }
  /* Eq. (15) per weight, W_ij = wt[j][i]. */
  for (int32_t j = 0; j < d_out; ++j) {
    double colsum = 0.0;  /* sum_k dW~_kj B_kj */
    for (int32_t k = 0; k < d_in; ++k)
      colsum += dwt_tilde[(int64_t)j * d_in + k] * (double)sign_at(wbits + (int64_t)j * ldw, k);
    for (int32_t i = 0; i < d_in; ++i) {
      double bij = (double)sign_at(wbits + (int64_t)j * ldw, i);
      double ste = fabs((double)wt[(int64_t)j * d_in + i]) < 1.0 ? 1.0 : 0.0;
      dwt[(int64_t)j * d_in + i] = bij * colsum / (double)d_in +
                                   alpha[j] * dwt_tilde[(int64_t)j * d_in + i] * ste;
    }
  }
done:
  free(fbits);
  free(beta);
  free(wbits);
  free(alpha);
  free(G);
  return rc;
}

/* ---------------------------------------------------------------------
 * oracle_layer_backward_at: the same back propagation (Alg. 1, Eqs. (14)-
 * (15)) for a subset of its outputs, for graphs too large for the whole
 * layer: the rows listed in `rows` of dζ and dH~ / dH, the columns j listed
 * in `cols` of dW~ and dW (every k of each), and all of db.  Every entry is
 * the sum oracle_layer_backward forms, over the same terms in the same
 * order, so the two agree bit for bit; only the entries asked for are
 * formed (column j of dW~ needs dζ_:j for every node, row i of dH~ needs
 * dζ_i,: for every column), and the masked gradient is read in place.
 *   rows [n_rows] node ids;  cols [n_cols] output columns (< d_out)
 * Outputs (doubles):  dzeta, mass_dzeta [n_rows][d_out]; dh_tilde, mass_dh,
 *   dh [n_rows][d_in]; dwt_tilde, mass_dwt, dwt [n_cols][d_in]; db [d_out].
 * Returns 0, -1 on a non-finite input, -2 on allocation failure, -3 on an
 * id out of range.
 * ------------------------------------------------------------------- */
static double g_masked(const float* gout, const float* out, int act, int32_t d_out,
                       int64_t i, int32_t k) {
  if (act == ORACLE_ACT_RELU && !(out[i * d_out + k] > 0.0f)) return 0.0;
  return (double)gout[i * d_out + k];
}

/* dζ_jk = sum_{i in N(j)} Ã_ij G_ik and the mass of its terms. */
static double dzeta_at(const int64_t* rowptr, const int32_t* colidx, int norm,
                       const float* gout, const float* out, int act, int32_t d_out,
                       int64_t j, int32_t k, double* mass) {
  int64_t deg_j = rowptr[j + 1] - rowptr[j];
  double s = 0.0, m = 0.0;
  for (int64_t e = rowptr[j]; e < rowptr[j + 1]; ++e) {
    int64_t i = colidx[e];
    int64_t deg_i = rowptr[i + 1] - rowptr[i];
    double t = atilde(norm, deg_i, deg_j) * g_masked(gout, out, act, d_out, i, k);
    s += t;
    m += fabs(t);
  }
  *mass = m;
  return s;
}

int oracle_layer_backward_at(int64_t n, const int64_t* rowptr, const int32_t* colidx,
                             int norm, const float* h, int64_t ldh, int32_t d_in,
                             const float* wt, int32_t d_out, const float* gout,
                             const float* out, int act, int64_t n_rows,
                             const int64_t* rows, int32_t n_cols, const int32_t* cols,
                             double* dzeta, double* mass_dzeta, double* dh_tilde,
                             double* mass_dh, double* dh, double* dwt_tilde,
                             double* mass_dwt, double* dwt, double* db) {
  const int64_t ldw = (d_in + 63) / 64;
  int rc = 0;
  for (int64_t r = 0; r < n_rows; ++r)
    if (rows[r] < 0 || rows[r] >= n) return -3;
  for (int32_t c = 0; c < n_cols; ++c)
    if (cols[c] < 0 || cols[c] >= d_out) return -3;
  uint64_t* fbits = calloc((size_t)(n ? n : 1) * ldw, sizeof(uint64_t));
  double* beta = calloc((size_t)(n ? n : 1), sizeof(double));
  uint64_t* wbits = calloc((size_t)d_out * ldw, sizeof(uint64_t));
  double* alpha = calloc((size_t)d_out, sizeof(double));
  double* zcol = calloc((size_t)(n ? n : 1), sizeof(double));
  if (!fbits || !beta || !wbits || !alpha || !zcol) {
    rc = -2;
    goto done;
  }
  if (oracle_binarize(h, n, d_in, ldh, NULL, NULL, NULL, 0, fbits, ldw, beta) != 0 ||
      oracle_binarize(wt, d_out, d_in, d_in, NULL, NULL, NULL, 0, wbits, ldw, alpha) != 0) {
    rc = -1;
    goto done;
  }
  /* Bias: dL/db_k = sum_i G_ik. */
  for (int32_t k = 0; k < d_out; ++k) {
    double s = 0.0;
    for (int64_t i = 0; i < n; ++i) s += g_masked(gout, out, act, d_out, i, k);
    db[k] = s;
  }
  /* Listed columns j: dζ_:j, then dW~_kj = sum_i H~_ik dζ_ij and Eq. (15). */
  for (int32_t c = 0; c < n_cols; ++c) {
    const int32_t j = cols[c];
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t i = 0; i < n; ++i) {
      double m;
      zcol[i] = dzeta_at(rowptr, colidx, norm, gout, out, act, d_out, i, j, &m);
    }
#pragma omp parallel for schedule(dynamic, 4)
    for (int32_t k = 0; k < d_in; ++k) {
      double s = 0.0, m = 0.0;
      for (int64_t i = 0; i < n; ++i) {
        double ht = beta[i] * (double)sign_at(fbits + i * ldw, k);  /* H~_ik */
        double t = ht * zcol[i];
        s += t;
        m += fabs(t);
      }
      dwt_tilde[(int64_t)c * d_in + k] = s;
      mass_dwt[(int64_t)c * d_in + k] = m;
    }
    double colsum = 0.0;  /* sum_k dW~_kj B_kj */
    for (int32_t k = 0; k < d_in; ++k)
      colsum += dwt_tilde[(int64_t)c * d_in + k] * (double)sign_at(wbits + (int64_t)j * ldw, k);
    for (int32_t i = 0; i < d_in; ++i) {
      double bij = (double)sign_at(wbits + (int64_t)j * ldw, i);
      double ste = fabs((double)wt[(int64_t)j * d_in + i]) < 1.0 ? 1.0 : 0.0;
      dwt[(int64_t)c * d_in + i] = bij * colsum / (double)d_in +
                                   alpha[j] * dwt_tilde[(int64_t)c * d_in + i] * ste;
    }
  }
  /* Listed rows i: dζ_i,:, then dH~_ik = sum_j dζ_ij W~_kj and Eq. (14). */
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t r = 0; r < n_rows; ++r) {
    const int64_t i = rows[r];
    for (int32_t j = 0; j < d_out; ++j)
      dzeta[r * d_out + j] = dzeta_at(rowptr, colidx, norm, gout, out, act, d_out, i, j,
                                      &mass_dzeta[r * d_out + j]);
    for (int32_t k = 0; k < d_in; ++k) {
      double s = 0.0, m = 0.0;
      for (int32_t j = 0; j < d_out; ++j) {
        double wtl = (double)sign_at(wbits + (int64_t)j * ldw, k) * alpha[j];  /* W~_kj */
        double t = dzeta[r * d_out + j] * wtl;
        s += t;
        m += fabs(t);
      }
      dh_tilde[r * d_in + k] = s;
      mass_dh[r * d_in + k] = m;
      dh[r * d_in + k] = fabs(s) < 1.0 ? s : 0.0;
    }
  }
done:
  free(fbits);
  free(beta);
  free(wbits);
  free(alpha);
  free(zcol);
  return rc;
}

/* Number of threads the oracle's parallel loops use. */
int oracle_threads(void) { return omp_get_max_threads(); }

/* Sets that number (n >= 1) for the calls that follow on this thread. */
void oracle_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
