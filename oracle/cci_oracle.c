/*
 * CCI-sparsity oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct CPU implementation of what the CCI-sparse
 * forward path computes (Yu et al., "Cross-Channel Intragroup Sparsity Neural
 * Network", arXiv:1910.11971).  Only the test-suite, the smoke check and the
 * benchmark's cpu_baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library; it includes nothing from it.
 *
 * Arithmetic: every product and sum is taken in double precision; results are
 * returned unrounded (double) except where a function's job is rounding.
 * Loops follow the paper's definitions directly; the only addition is an
 * OpenMP work split over independent output blocks, which does not change
 * the order of any sum.
 *
 * Notation (paper Sec. 3.1): a layer H = W X with W of M x N; here W is
 * [O][C] (O output channels, C inputs), X is [N][C] (N rows = samples or
 * output pixels) and Y = X W^T is [N][O].  A CCI group is G contiguous
 * output channels at one input column; it keeps exactly K (the paper's s)
 * nonzeros, stored packed as K values plus K intra-group row indices.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)

/* |w| as an orderable unsigned key: the fp32 bit pattern with the sign bit
 * cleared.  For non-negative IEEE floats the bit pattern orders exactly like
 * the value; NaN patterns order above +Inf.  (Selection is made on the fp32
 * master weight, never on a rounded copy.) */
static uint32_t abs_key(float w) {
  uint32_t u;
  memcpy(&u, &w, sizeof u);
  return u & 0x7fffffffu;
}

static int check_group_args(int64_t O, int64_t C, int32_t G, int32_t K) {
  if (G < 1 || G > 256 || K < 1 || K > G) return ORACLE_EINVAL;
  if (O < 1 || C < 1 || O % G != 0) return ORACLE_EINVAL;
  return ORACLE_OK;
}

/*
 * Magnitude projection onto CCI sparsity (paper Sec. 5.1: weights of low
 * absolute magnitude are pruned; Sec. 3.1 and Fig. 1: a group is G
 * contiguous output channels at one input position and keeps exactly s = K
 * nonzeros).
 *
 * For every group g in [0, O/G) and column c in [0, C) with w_r = W[gG+r][c]:
 *   rank_r = #{ r' : key_r' > key_r  or  (key_r' == key_r and r' < r) }
 *   r is kept iff rank_r < K            (ties between equal |w|: lower r wins)
 * The kept r are emitted in ascending r:  idx[g][k][c] = r,
 * vals[g][k][c] = w_r (an exact copy of the fp32 weight).
 * Layout: vals, idx are [O/G][K][C].
 */
int oracle_pack(const float *W, int64_t O, int64_t C, int32_t G, int32_t K,
                float *vals, uint8_t *idx) {
  if (check_group_args(O, C, G, K) != ORACLE_OK) return ORACLE_EINVAL;
  const int64_t ngroups = O / G;
#pragma omp parallel for schedule(static)
  for (int64_t g = 0; g < ngroups; ++g) {
    for (int64_t c = 0; c < C; ++c) {
      int32_t slot = 0;
      for (int32_t r = 0; r < G; ++r) {
        const uint32_t kr = abs_key(W[(g * G + r) * C + c]);
        int32_t rank = 0;
        for (int32_t q = 0; q < G; ++q) {
          const uint32_t kq = abs_key(W[(g * G + q) * C + c]);
          if (kq > kr || (kq == kr && q < r)) ++rank;
        }
        if (rank < K) {
          vals[(g * K + slot) * C + c] = W[(g * G + r) * C + c];
          idx[(g * K + slot) * C + c] = (uint8_t)r;
          ++slot;
        }
      }
    }
  }
  return ORACLE_OK;
}

/*
 * Inverse of the packing: the dense masked matrix W_hat [O][C] that the
 * packed groups describe (paper Sec. 3.1: every G rows of W_hat are
 * compressed into exactly s rows with the same column count; the index
 * names the row inside the group).  Entries not named by any slot are 0.
 */
int oracle_unpack(const float *vals, const uint8_t *idx, int64_t O, int64_t C,
                  int32_t G, int32_t K, float *Wd) {
  if (check_group_args(O, C, G, K) != ORACLE_OK) return ORACLE_EINVAL;
  for (int64_t i = 0; i < O * C; ++i) Wd[i] = 0.0f;
  const int64_t ngroups = O / G;
  for (int64_t g = 0; g < ngroups; ++g)
    for (int32_t k = 0; k < K; ++k)
      for (int64_t c = 0; c < C; ++c) {
        const int32_t r = idx[(g * K + k) * C + c];
        if (r >= G) return ORACLE_EINVAL;
        Wd[(g * G + r) * C + c] = vals[(g * K + k) * C + c];
      }
  return ORACLE_OK;
}

/* Fused epilogue applied to one exact accumulator value, in double:
 *   y = acc * scale[o] + bias[o] + residual[n][o], then max(y, 0) if relu.
 * Missing (NULL) terms are skipped (scale defaults to 1, others to 0). */
static double epilogue(double acc, int64_t o, const float *scale,
                       const float *bias, const float *res_row, int32_t relu) {
  double y = acc;
  if (scale) y = y * (double)scale[o];
  if (bias) y = y + (double)bias[o];
  if (res_row) y = y + (double)res_row[o];
  if (relu && !(y > 0.0)) y = (y != y) ? y : 0.0;
  return y;
}

/*
 * CCI-sparse matrix product (paper Sec. 3.2, Alg. 1, generalised from s = 1
 * to s = K slots per group: packed row gK+k is slot k of group g).
 *
 * For every group g, sample row n, input column c and slot k:
 *   Y[n][gG + idx[g][k][c]] += vals[g][k][c] * X[n][c]
 * starting from Y = 0, all in double; then the epilogue.  Because the inner
 * loops run c ascending with k inside c, each output receives its terms in
 * ascending c -- the same order as the dense triple loop (Alg. 0) applied to
 * the unpacked masked matrix.
 *
 * `rows` (length nrows) selects which sample rows to compute (NULL: all N,
 * nrows must equal N); output row i of Y / Yabs corresponds to rows[i].
 * Yabs (optional) receives sum |vals * X| per output, the scale of the
 * rounding error any finite-precision evaluation can make.
 * residual, if given, is [N][O] fp32 (indexed by the true row n).
 */
int oracle_spmm_rows(const float *X, int64_t N, int64_t C, const float *vals,
                     const uint8_t *idx, int64_t O, int32_t G, int32_t K,
                     const float *scale, const float *bias,
                     const float *residual, int32_t relu, const int64_t *rows,
                     int64_t nrows, double *Y, double *Yabs) {
  if (check_group_args(O, C, G, K) != ORACLE_OK || N < 0) return ORACLE_EINVAL;
  if (!rows && nrows != N) return ORACLE_EINVAL;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    if (n < 0 || n >= N) return ORACLE_EINVAL;
  }
  for (int64_t i = 0; i < nrows * O; ++i) {
    Y[i] = 0.0;
    if (Yabs) Yabs[i] = 0.0;
  }
  const int64_t ngroups = O / G;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t g = 0; g < ngroups; ++g) {
    for (int64_t i = 0; i < nrows; ++i) {
      const int64_t n = rows ? rows[i] : i;
      for (int64_t c = 0; c < C; ++c) {
        const double x = (double)X[n * C + c];
        for (int32_t k = 0; k < K; ++k) {
          const int32_t r = idx[(g * K + k) * C + c];
          if (r >= G) { bad = 1; continue; }
          const double v = (double)vals[(g * K + k) * C + c];
          Y[i * O + g * G + r] += v * x;
          if (Yabs) Yabs[i * O + g * G + r] += fabs(v * x);
        }
      }
    }
  }
  if (bad) return ORACLE_EINVAL;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    const float *res_row = residual ? residual + n * O : NULL;
    for (int64_t o = 0; o < O; ++o)
      Y[i * O + o] = epilogue(Y[i * O + o], o, scale, bias, res_row, relu);
  }
  return ORACLE_OK;
}

/*
 * Dense matrix product (paper Sec. 3.2, Alg. 0) on an unpacked matrix
 * Wd [O][C]:  Y[n][o] = sum_c Wd[o][c] * X[n][c], c ascending, in double;
 * then the epilogue.  Used as the textbook comparator for Alg. 1.
 */
int oracle_dense_rows(const float *X, int64_t N, int64_t C, const float *Wd,
                      int64_t O, const float *scale, const float *bias,
                      const float *residual, int32_t relu, const int64_t *rows,
                      int64_t nrows, double *Y) {
  if (O < 1 || C < 1 || N < 0) return ORACLE_EINVAL;
  if (!rows && nrows != N) return ORACLE_EINVAL;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    if (n < 0 || n >= N) return ORACLE_EINVAL;
  }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    const float *res_row = residual ? residual + n * O : NULL;
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int64_t c = 0; c < C; ++c)
        acc += (double)Wd[o * C + c] * (double)X[n * C + c];
      Y[i * O + o] = epilogue(acc, o, scale, bias, res_row, relu);
    }
  }
  return ORACLE_OK;
}

/*
 * Direct 2-D convolution, NHWC activations, weights Wd [O][KH][KW][Cin]
 * (dense; pass the unpacked masked matrix for a CCI layer):
 *   Y[b][oh][ow][o] = sum_{kh,kw,ci} X[b][oh*sh-ph+kh][ow*sw-pw+kw][ci]
 *                                     * Wd[o][kh][kw][ci]
 * with X taken as 0 outside the image; double accumulation in (kh, kw, ci)
 * order; then the epilogue.  Output pixel p = (b*Ho + oh)*Wo + ow;
 * `pixels` selects which to compute (NULL: all).  residual is NHWC [.. O].
 */
int oracle_conv2d_nhwc_rows(const float *X, int64_t B, int64_t H, int64_t W,
                            int64_t Cin, const float *Wd, int64_t O, int32_t KH,
                            int32_t KW, int32_t sh, int32_t sw, int32_t ph,
                            int32_t pw, const float *scale, const float *bias,
                            const float *residual, int32_t relu,
                            const int64_t *pixels, int64_t npix, double *Y,
                            double *Yabs) {
  if (B < 0 || H < 1 || W < 1 || Cin < 1 || O < 1 || KH < 1 || KW < 1 ||
      sh < 1 || sw < 1 || ph < 0 || pw < 0)
    return ORACLE_EINVAL;
  const int64_t Ho = (H + 2 * ph - KH) / sh + 1;
  const int64_t Wo = (W + 2 * pw - KW) / sw + 1;
  if (H + 2 * ph < KH || W + 2 * pw < KW) return ORACLE_EINVAL;
  const int64_t P = B * Ho * Wo;
  if (!pixels && npix != P) return ORACLE_EINVAL;
  for (int64_t i = 0; i < npix; ++i) {
    const int64_t p = pixels ? pixels[i] : i;
    if (p < 0 || p >= P) return ORACLE_EINVAL;
  }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < npix; ++i) {
    const int64_t p = pixels ? pixels[i] : i;
    const int64_t b = p / (Ho * Wo);
    const int64_t oh = (p / Wo) % Ho;
    const int64_t ow = p % Wo;
    const float *res_row = residual ? residual + p * O : NULL;
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0, aabs = 0.0;
      for (int32_t kh = 0; kh < KH; ++kh) {
        const int64_t ih = oh * sh - ph + kh;
        if (ih < 0 || ih >= H) continue;
        for (int32_t kw = 0; kw < KW; ++kw) {
          const int64_t iw = ow * sw - pw + kw;
          if (iw < 0 || iw >= W) continue;
          for (int64_t ci = 0; ci < Cin; ++ci) {
            const double t =
                (double)X[((b * H + ih) * W + iw) * Cin + ci] *
                (double)Wd[((o * KH + kh) * KW + kw) * Cin + ci];
            acc += t;
            aabs += fabs(t);
          }
        }
      }
      Y[i * O + o] = epilogue(acc, o, scale, bias, res_row, relu);
      if (Yabs) Yabs[i * O + o] = aabs;
    }
  }
  return ORACLE_OK;
}

/*
 * Explicit im2col of an NHWC tensor (paper Sec. 3.2: convolution is computed
 * as a GEMM).  Row p = (b*Ho + oh)*Wo + ow; column (kh*KW + kw)*Cin + ci;
 * value X[b][oh*sh-ph+kh][ow*sw-pw+kw][ci], or 0 outside the image.
 * A is [B*Ho*Wo][KH*KW*Cin].
 */
int oracle_im2col_nhwc(const float *X, int64_t B, int64_t H, int64_t W,
                       int64_t Cin, int32_t KH, int32_t KW, int32_t sh,
                       int32_t sw, int32_t ph, int32_t pw, float *A) {
  if (B < 0 || H < 1 || W < 1 || Cin < 1 || KH < 1 || KW < 1 || sh < 1 ||
      sw < 1 || ph < 0 || pw < 0 || H + 2 * ph < KH || W + 2 * pw < KW)
    return ORACLE_EINVAL;
  const int64_t Ho = (H + 2 * ph - KH) / sh + 1;
  const int64_t Wo = (W + 2 * pw - KW) / sw + 1;
  const int64_t Cc = (int64_t)KH * KW * Cin;
  for (int64_t b = 0; b < B; ++b)
    for (int64_t oh = 0; oh < Ho; ++oh)
      for (int64_t ow = 0; ow < Wo; ++ow) {
        const int64_t p = (b * Ho + oh) * Wo + ow;
        for (int32_t kh = 0; kh < KH; ++kh)
          for (int32_t kw = 0; kw < KW; ++kw)
            for (int64_t ci = 0; ci < Cin; ++ci) {
              const int64_t ih = oh * sh - ph + kh, iw = ow * sw - pw + kw;
              const int64_t col = ((int64_t)kh * KW + kw) * Cin + ci;
              A[p * Cc + col] = (ih < 0 || ih >= H || iw < 0 || iw >= W)
                                    ? 0.0f
                                    : X[((b * H + ih) * W + iw) * Cin + ci];
            }
      }
  return ORACLE_OK;
}

/*
 * Balanced sparsity (paper Sec. 2.4 and Sec. 3.3, Fig. 2b): the comparison
 * structure of the paper.  Its groups are G contiguous weights of one output
 * row -- weights of different inputs, instead of CCI's weights of different
 * output channels at one input -- and each group keeps its K (the paper's s)
 * largest-magnitude weights; the index of a kept weight names the input
 * inside its group that the weight multiplies.
 *
 * For every row o in [0, O) and group j in [0, C/G) with w_r = W[o][jG+r]:
 *   rank_r = #{ r' : key_r' > key_r  or  (key_r' == key_r and r' < r) }
 *   r is kept iff rank_r < K            (same magnitude order and tie rule
 *                                        as the CCI projection above)
 * kept r in ascending order: idx[o][j][k] = r, vals[o][j][k] = w_r.
 * Layout: vals, idx are [O][C/G][K] (a row's groups, then its slots).
 */
static int check_bbs_args(int64_t O, int64_t C, int32_t G, int32_t K) {
  if (G < 1 || G > 256 || K < 1 || K > G) return ORACLE_EINVAL;
  if (O < 1 || C < 1 || C % G != 0) return ORACLE_EINVAL;
  return ORACLE_OK;
}

int oracle_bbs_pack(const float *W, int64_t O, int64_t C, int32_t G, int32_t K,
                    float *vals, uint8_t *idx) {
  if (check_bbs_args(O, C, G, K) != ORACLE_OK) return ORACLE_EINVAL;
  const int64_t ngroups = C / G;
#pragma omp parallel for schedule(static)
  for (int64_t o = 0; o < O; ++o) {
    for (int64_t j = 0; j < ngroups; ++j) {
      const float *w = W + o * C + j * G;
      int32_t slot = 0;
      for (int32_t r = 0; r < G; ++r) {
        const uint32_t kr = abs_key(w[r]);
        int32_t rank = 0;
        for (int32_t q = 0; q < G; ++q) {
          const uint32_t kq = abs_key(w[q]);
          if (kq > kr || (kq == kr && q < r)) ++rank;
        }
        if (rank < K) {
          vals[(o * ngroups + j) * K + slot] = w[r];
          idx[(o * ngroups + j) * K + slot] = (uint8_t)r;
          ++slot;
        }
      }
    }
  }
  return ORACLE_OK;
}

/* The dense masked matrix W_hat [O][C] a balanced-sparse packing describes:
 * W_hat[o][jG + idx[o][j][k]] = vals[o][j][k], every other entry 0. */
int oracle_bbs_unpack(const float *vals, const uint8_t *idx, int64_t O,
                      int64_t C, int32_t G, int32_t K, float *Wd) {
  if (check_bbs_args(O, C, G, K) != ORACLE_OK) return ORACLE_EINVAL;
  for (int64_t i = 0; i < O * C; ++i) Wd[i] = 0.0f;
  const int64_t ngroups = C / G;
  for (int64_t o = 0; o < O; ++o)
    for (int64_t j = 0; j < ngroups; ++j)
      for (int32_t k = 0; k < K; ++k) {
        const int32_t r = idx[(o * ngroups + j) * K + k];
        if (r >= G) return ORACLE_EINVAL;
        Wd[o * C + j * G + r] = vals[(o * ngroups + j) * K + k];
      }
  return ORACLE_OK;
}

/*
 * Balanced-sparse product (Sec. 3.3, Fig. 2b): the index of each kept weight
 * selects the input element inside its group that it multiplies,
 *   Y[n][o] = sum_j sum_k vals[o][j][k] * X[n][jG + idx[o][j][k]],
 * in double, j ascending and k ascending inside j (so the terms of an output
 * arrive in ascending input order, as in Alg. 0 on the unpacked matrix);
 * then the epilogue.  rows / Yabs / residual as for oracle_spmm_rows.
 */
int oracle_bbs_spmm_rows(const float *X, int64_t N, int64_t C,
                         const float *vals, const uint8_t *idx, int64_t O,
                         int32_t G, int32_t K, const float *scale,
                         const float *bias, const float *residual,
                         int32_t relu, const int64_t *rows, int64_t nrows,
                         double *Y, double *Yabs) {
  if (check_bbs_args(O, C, G, K) != ORACLE_OK || N < 0) return ORACLE_EINVAL;
  if (!rows && nrows != N) return ORACLE_EINVAL;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    if (n < 0 || n >= N) return ORACLE_EINVAL;
  }
  const int64_t ngroups = C / G;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t n = rows ? rows[i] : i;
    const float *res_row = residual ? residual + n * O : NULL;
    for (int64_t o = 0; o < O; ++o) {
      double acc = 0.0, aabs = 0.0;
      for (int64_t j = 0; j < ngroups; ++j)
        for (int32_t k = 0; k < K; ++k) {
          const int32_t r = idx[(o * ngroups + j) * K + k];
          if (r >= G) { bad = 1; continue; }
          const double t = (double)vals[(o * ngroups + j) * K + k] * (double)X[n * C + j * G + r];
          acc += t;
          aabs += fabs(t);
        }
      Y[i * O + o] = epilogue(acc, o, scale, bias, res_row, relu);
      if (Yabs) Yabs[i * O + o] = aabs;
    }
  }
  return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/*
 * Improved targeted dropout (paper Sec. 5.1, schedule of Sec. 6).
 *
 * Schedule.  Over a run of T steps, with f = step / T: during the first half
 * the targeted rate (the share of each group's weights that are pruning
 * candidates) ramps from 0 to its target 1 - K/G while candidates are
 * dropped with probability 1/2; during the second half the targeted rate
 * stays at its target and the dropout rate ramps from 1/2 to 1 (reading:
 * both ramps linear in f).  Per group of G that is
 *   n_target = floor((G - K) * min(1, 2 f) + 1/2)   candidates,
 *   drop_rate = max(1/2, f).
 * At f = 1 every candidate is dropped: the weights seen by the forward are
 * exactly the CCI projection (Sec. 5.1's magnitude policy with the group
 * constraint of Sec. 3.1).
 */
int oracle_td_schedule(int64_t step, int64_t total, int32_t G, int32_t K,
                       int32_t *n_target, double *drop_rate) {
  if (total < 1 || step < 0 || step > total || G < 1 || K < 1 || K > G) return ORACLE_EINVAL;
  const double f = (double)step / (double)total;
  const double ramp = 2.0 * f < 1.0 ? 2.0 * f : 1.0;
  *n_target = (int32_t)floor((double)(G - K) * ramp + 0.5);
  *drop_rate = f > 0.5 ? f : 0.5;
  return ORACLE_OK;
}

/*
 * Candidate dropout of one step.  For every CCI group (G contiguous output
 * channels at column c) the n_target weights of lowest magnitude are the
 * candidates: with rank_r counted as in oracle_pack (larger |w| first, ties
 * to the lower row), r is a candidate iff rank_r >= G - n_target.  A
 * candidate is dropped iff its random word bits[o][c] (uniform 32-bit, drawn
 * by the caller) is below floor(drop_rate * 2^32).  Outputs: W_eff [O][C],
 * the weight or 0 where dropped; keep [O][C], 0 where dropped else 1.
 */
int oracle_td_mask(const float *W, int64_t O, int64_t C, int32_t G,
                   int32_t n_target, const uint32_t *bits, double drop_rate,
                   float *W_eff, uint8_t *keep) {
  if (O < 1 || C < 1 || G < 1 || G > 256 || O % G != 0 || n_target < 0 ||
      n_target > G || !(drop_rate >= 0.0 && drop_rate <= 1.0))
    return ORACLE_EINVAL;
  const uint64_t thr = (uint64_t)floor(drop_rate * 4294967296.0);
  const int64_t ngroups = O / G;
#pragma omp parallel for schedule(static)
  for (int64_t g = 0; g < ngroups; ++g)
    for (int64_t c = 0; c < C; ++c)
      for (int32_t r = 0; r < G; ++r) {
        const int64_t o = g * G + r;
        const uint32_t kr = abs_key(W[o * C + c]);
        int32_t rank = 0;
        for (int32_t q = 0; q < G; ++q) {
          const uint32_t kq = abs_key(W[(g * G + q) * C + c]);
          if (kq > kr || (kq == kr && q < r)) ++rank;
        }
        const int candidate = rank >= G - n_target;
        const int dropped = candidate && (uint64_t)bits[o * C + c] < thr;
        W_eff[o * C + c] = dropped ? 0.0f : W[o * C + c];
        keep[o * C + c] = (uint8_t)(dropped ? 0 : 1);
      }
  return ORACLE_OK;
}

/*
 * Gradient of the packed values of a CCI layer Y = X W_hat^T (Alg. 1's
 * product), given dY = dL/dY:  dL/dvals[g][k][c] = sum_n dY[n][gG + idx[g][k][c]]
 * * X[n][c], in double, n ascending.  (Each kept value multiplies X[.][c]
 * into output row gG + idx, so its derivative gathers that row of dY.)
 */
int oracle_grad_packed(const float *dY, const float *X, int64_t N, int64_t C,
                       const uint8_t *idx, int64_t O, int32_t G, int32_t K,
                       double *dvals) {
  if (check_group_args(O, C, G, K) != ORACLE_OK || N < 0) return ORACLE_EINVAL;
  const int64_t ngroups = O / G;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t g = 0; g < ngroups; ++g)
    for (int32_t k = 0; k < K; ++k)
      for (int64_t c = 0; c < C; ++c) {
        const int32_t r = idx[(g * K + k) * C + c];
        if (r >= G) { bad = 1; continue; }
        double acc = 0.0;
        for (int64_t n = 0; n < N; ++n)
          acc += (double)dY[n * O + g * G + r] * (double)X[n * C + c];
        dvals[(g * K + k) * C + c] = acc;
      }
  return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/*
 * Plain log2(G)-bit indices (paper Sec. 3.1: each kept weight carries the
 * plain index of its row inside the group, log2 G bits).  With
 * b = ceil(log2 G) (at least 1), entry e of an index array occupies bits
 * e*b .. e*b + b - 1 of a little-endian bit stream: stream bit t is bit
 * t % 32 of 32-bit word t / 32.  The stream has ceil(n * b / 32) words;
 * bits past the last entry are 0.  (With b = 8 the stream is the byte array
 * itself.)
 */
int32_t oracle_index_width(int32_t G) {
  if (G < 1 || G > 256) return -1;
  int32_t b = 1;
  while ((1 << b) < G) ++b;
  return b;
}

int oracle_index_bits(const uint8_t *idx, int64_t n, int32_t b, uint32_t *words) {
  if (n < 0 || b < 1 || b > 8) return ORACLE_EINVAL;
  const int64_t nw = (n * b + 31) / 32;
  for (int64_t w = 0; w < nw; ++w) words[w] = 0u;
  for (int64_t e = 0; e < n; ++e) {
    if (idx[e] >> b) return ORACLE_EINVAL; /* the value does not fit */
    for (int32_t j = 0; j < b; ++j) {
      const int64_t t = e * b + j;
      if ((idx[e] >> j) & 1u) words[t / 32] |= 1u << (t % 32);
    }
  }
  return ORACLE_OK;
}

int oracle_index_unbits(const uint32_t *words, int64_t n, int32_t b, uint8_t *idx) {
  if (n < 0 || b < 1 || b > 8) return ORACLE_EINVAL;
  for (int64_t e = 0; e < n; ++e) {
    uint32_t v = 0;
    for (int32_t j = 0; j < b; ++j) {
      const int64_t t = e * b + j;
      v |= ((words[t / 32] >> (t % 32)) & 1u) << j;
    }
    idx[e] = (uint8_t)v;
  }
  return ORACLE_OK;
}

/*
 * Round-to-nearest-even conversion of an fp32 value to bfloat16 (the upper
 * 16 bits of an IEEE binary32), written from the definition: the result is
 * the representable bf16 nearest to x; on an exact tie the one whose last
 * mantissa bit is 0.  NaN maps to a quiet NaN with the same sign; +-Inf and
 * +-0 are preserved; values above the largest bf16 round to +-Inf.
 */
uint16_t oracle_bf16_rne(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  if ((u & 0x7fffffffu) > 0x7f800000u) /* NaN */
    return (uint16_t)((u >> 16) | 0x0040u);
  const uint32_t upper = u >> 16;       /* truncated candidate */
  const uint32_t lower = u & 0xffffu;   /* discarded bits      */
  uint32_t r = upper;
  if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) r = upper + 1u;
  return (uint16_t)r;
}

void oracle_bf16_rne_array(const float *x, uint16_t *out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_rne(x[i]);
}

/*
 * Max pooling, NHWC, window k x k, stride s, zero-size padding p treated as
 * -infinity (so padding never wins).  Exact (no arithmetic).
 */
int oracle_maxpool2d_nhwc(const float *X, int64_t B, int64_t H, int64_t W,
                          int64_t C, int32_t k, int32_t s, int32_t p,
                          float *Y) {
  if (B < 0 || H < 1 || W < 1 || C < 1 || k < 1 || s < 1 || p < 0 ||
      H + 2 * p < k || W + 2 * p < k || 2 * p > k)
    return ORACLE_EINVAL;
  const int64_t Ho = (H + 2 * p - k) / s + 1, Wo = (W + 2 * p - k) / s + 1;
  for (int64_t b = 0; b < B; ++b)
    for (int64_t oh = 0; oh < Ho; ++oh)
      for (int64_t ow = 0; ow < Wo; ++ow)
        for (int64_t c = 0; c < C; ++c) {
          float m = -INFINITY;
          for (int32_t i = 0; i < k; ++i)
            for (int32_t j = 0; j < k; ++j) {
              const int64_t ih = oh * s - p + i, iw = ow * s - p + j;
              if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
              const float v = X[((b * H + ih) * W + iw) * C + c];
              if (v > m) m = v;
            }
          Y[((b * Ho + oh) * Wo + ow) * C + c] = m;
        }
  return ORACLE_OK;
}

/* Global average pooling, NHWC -> [B][C], sum in double then divide. */
int oracle_global_avgpool_nhwc(const float *X, int64_t B, int64_t H, int64_t W,
                               int64_t C, double *Y) {
  if (B < 0 || H < 1 || W < 1 || C < 1) return ORACLE_EINVAL;
  for (int64_t b = 0; b < B; ++b)
    for (int64_t c = 0; c < C; ++c) {
      double acc = 0.0;
      for (int64_t i = 0; i < H * W; ++i) acc += (double)X[(b * H * W + i) * C + c];
      Y[b * C + c] = acc / (double)(H * W);
    }
  return ORACLE_OK;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Thread count of later parallel loops started from the calling thread (a
 * timing knob: no result depends on it). */
void oracle_set_num_threads(int n) {
#ifdef _OPENMP
  extern void omp_set_num_threads(int);
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
