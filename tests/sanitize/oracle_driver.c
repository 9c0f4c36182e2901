/* Runs every oracle function on small inputs (edge sizes included) in a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer: any out-of-
 * bounds access or undefined operation aborts with a report.  Prints
 * "oracle driver ok" on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_pack(const float *, int64_t, int64_t, int32_t, int32_t, float *, uint8_t *);
int oracle_unpack(const float *, const uint8_t *, int64_t, int64_t, int32_t, int32_t, float *);
int oracle_spmm_rows(const float *, int64_t, int64_t, const float *, const uint8_t *, int64_t, int32_t, int32_t,
                     const float *, const float *, const float *, int32_t, const int64_t *, int64_t, double *, double *);
int oracle_dense_rows(const float *, int64_t, int64_t, const float *, int64_t, const float *, const float *,
                      const float *, int32_t, const int64_t *, int64_t, double *);
int oracle_conv2d_nhwc_rows(const float *, int64_t, int64_t, int64_t, int64_t, const float *, int64_t, int32_t, int32_t,
                            int32_t, int32_t, int32_t, int32_t, const float *, const float *, const float *, int32_t,
                            const int64_t *, int64_t, double *, double *);
int oracle_im2col_nhwc(const float *, int64_t, int64_t, int64_t, int64_t, int32_t, int32_t, int32_t, int32_t, int32_t,
                       int32_t, float *);
void oracle_bf16_rne_array(const float *, uint16_t *, int64_t);
int oracle_maxpool2d_nhwc(const float *, int64_t, int64_t, int64_t, int64_t, int32_t, int32_t, int32_t, float *);
int oracle_global_avgpool_nhwc(const float *, int64_t, int64_t, int64_t, int64_t, double *);
int oracle_bbs_pack(const float *, int64_t, int64_t, int32_t, int32_t, float *, uint8_t *);
int oracle_bbs_unpack(const float *, const uint8_t *, int64_t, int64_t, int32_t, int32_t, float *);
int oracle_bbs_spmm_rows(const float *, int64_t, int64_t, const float *, const uint8_t *, int64_t, int32_t, int32_t,
                         const float *, const float *, const float *, int32_t, const int64_t *, int64_t, double *,
                         double *);
int oracle_td_schedule(int64_t, int64_t, int32_t, int32_t, int32_t *, double *);
int oracle_td_mask(const float *, int64_t, int64_t, int32_t, int32_t, const uint32_t *, double, float *, uint8_t *);
int oracle_grad_packed(const float *, const float *, int64_t, int64_t, const uint8_t *, int64_t, int32_t, int32_t,
                       double *);
int32_t oracle_index_width(int32_t);
int oracle_index_bits(const uint8_t *, int64_t, int32_t, uint32_t *);
int oracle_index_unbits(const uint32_t *, int64_t, int32_t, uint8_t *);

static float frand(unsigned *s) {
  *s = *s * 1664525u + 1013904223u;
  return (float)((int)(*s >> 8) - (1 << 23)) / (float)(1 << 23);
}

#define CHECK(c)                                                \
  do {                                                          \
    if (!(c)) {                                                 \
      fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #c);    \
      return 1;                                                 \
    }                                                           \
  } while (0)

int main(void) {
  unsigned s = 1;
  const int shapes[][4] = {{8, 5, 4, 2}, {16, 1, 8, 8}, {6, 7, 3, 1}, {256, 3, 256, 5}, {2, 9, 2, 1}};
  for (unsigned t = 0; t < sizeof shapes / sizeof shapes[0]; ++t) {
    const int O = shapes[t][0], C = shapes[t][1], G = shapes[t][2], K = shapes[t][3], N = 3;
    float *W = malloc(sizeof(float) * O * C), *X = malloc(sizeof(float) * N * C), *Wd = malloc(sizeof(float) * O * C);
    float *v = malloc(sizeof(float) * O / G * K * C);
    uint8_t *ix = malloc((size_t)O / G * K * C);
    double *Y = malloc(sizeof(double) * N * O), *Ya = malloc(sizeof(double) * N * O);
    for (int i = 0; i < O * C; ++i) W[i] = frand(&s);
    for (int i = 0; i < N * C; ++i) X[i] = frand(&s);
    CHECK(oracle_pack(W, O, C, G, K, v, ix) == 0);
    CHECK(oracle_unpack(v, ix, O, C, G, K, Wd) == 0);
    CHECK(oracle_spmm_rows(X, N, C, v, ix, O, G, K, NULL, NULL, NULL, 1, NULL, N, Y, Ya) == 0);
    CHECK(oracle_dense_rows(X, N, C, Wd, O, NULL, NULL, NULL, 0, NULL, N, Y) == 0);
    double *dv = malloc(sizeof(double) * O / G * K * C);
    float *dY = malloc(sizeof(float) * N * O);
    for (int i = 0; i < N * O; ++i) dY[i] = frand(&s);
    CHECK(oracle_grad_packed(dY, X, N, C, ix, O, G, K, dv) == 0);
    uint32_t *bits = malloc(sizeof(uint32_t) * O * C);
    for (int i = 0; i < O * C; ++i) bits[i] = (uint32_t)(frand(&s) * 4e9f);
    uint8_t *keep = malloc((size_t)O * C);
    CHECK(oracle_td_mask(W, O, C, G, G - K, bits, 0.5, Wd, keep) == 0);
    const int b = oracle_index_width(G);
    const int64_t n = (int64_t)O / G * K * C;
    uint32_t *st = malloc(sizeof(uint32_t) * (size_t)((n * b + 31) / 32 + 1));
    uint8_t *back = malloc((size_t)n);
    CHECK(oracle_index_bits(ix, n, b, st) == 0 && oracle_index_unbits(st, n, b, back) == 0);
    for (int64_t i = 0; i < n; ++i) CHECK(back[i] == ix[i]);
    if (C % G == 0) {
      float *bv = malloc(sizeof(float) * O * (C / G) * K);
      uint8_t *bi = malloc((size_t)O * (C / G) * K);
      CHECK(oracle_bbs_pack(W, O, C, G, K, bv, bi) == 0);
      CHECK(oracle_bbs_unpack(bv, bi, O, C, G, K, Wd) == 0);
      CHECK(oracle_bbs_spmm_rows(X, N, C, bv, bi, O, G, K, NULL, NULL, NULL, 0, NULL, N, Y, Ya) == 0);
      free(bv);
      free(bi);
    }
    free(W), free(X), free(Wd), free(v), free(ix), free(Y), free(Ya), free(dv), free(dY), free(bits), free(keep);
    free(st), free(back);
  }
  /* convolution, im2col, pooling, rounding on a tiny image with padding */
  {
    const int B = 2, H = 5, Wi = 4, Cin = 3, O = 4, k = 3;
    float X[2 * 5 * 4 * 3], Wt[4 * 3 * 3 * 3], A[2 * 5 * 4 * 27], P[2 * 3 * 2 * 3];
    double Y[2 * 5 * 4 * 4], Ya[2 * 5 * 4 * 4], av[2 * 3];
    uint16_t r[2 * 5 * 4 * 3];
    for (unsigned i = 0; i < sizeof X / sizeof X[0]; ++i) X[i] = frand(&s);
    for (unsigned i = 0; i < sizeof Wt / sizeof Wt[0]; ++i) Wt[i] = frand(&s);
    CHECK(oracle_conv2d_nhwc_rows(X, B, H, Wi, Cin, Wt, O, k, k, 1, 1, 1, 1, NULL, NULL, NULL, 1, NULL, B * H * Wi, Y, Ya) == 0);
    CHECK(oracle_im2col_nhwc(X, B, H, Wi, Cin, k, k, 1, 1, 1, 1, A) == 0);
    CHECK(oracle_maxpool2d_nhwc(X, B, H, Wi, Cin, 3, 2, 1, P) == 0);
    CHECK(oracle_global_avgpool_nhwc(X, B, H, Wi, Cin, av) == 0);
    oracle_bf16_rne_array(X, r, B * H * Wi * Cin);
    const int64_t pix[2] = {0, B * H * Wi - 1};
    CHECK(oracle_conv2d_nhwc_rows(X, B, H, Wi, Cin, Wt, O, k, k, 2, 2, 0, 0, NULL, NULL, NULL, 0, pix, 1, Y, NULL) == 0);
  }
  int32_t nt;
  double p;
  CHECK(oracle_td_schedule(7, 10, 16, 4, &nt, &p) == 0 && nt == 12 && p == 0.7);
  /* rejected arguments return an error without touching memory */
  CHECK(oracle_pack(NULL, 12, 5, 8, 2, NULL, NULL) != 0);
  CHECK(oracle_index_bits(NULL, 4, 9, NULL) != 0);
  printf("oracle driver ok\n");
  return 0;
}
