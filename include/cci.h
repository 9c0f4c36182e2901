/*
 * cci.h -- C ABI of the MI355X (gfx950) CCI-sparse forward path.
 *
 * Cross-channel intragroup (CCI) sparsity (Yu et al., arXiv:1910.11971):
 * the weights W [O][C] of a layer are split into groups of G contiguous output
 * channels at one input column; each group keeps exactly K nonzeros (the
 * paper's s), stored packed as K values plus K intra-group row indices
 * (Sec. 3.1, Fig. 1).  The forward product Y = X W^T is computed from the
 * packed form (Sec. 3.2, Alg. 1); convolution is lowered to that product
 * (Sec. 3.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Memory.  Every tensor argument is a device pointer to caller-owned,
 *    contiguous, row-major memory on the current HIP device.  The library
 *    never allocates, frees or synchronises.
 *  - State.  Between calls the library keeps only (a) a thread-local error
 *    string and (b) per-device launch set-up computed on the first launch of
 *    a kernel with that device current: the kernel's dynamic-LDS limit
 *    (hipFuncSetAttribute) and, for the narrow kernels, the number of
 *    resident waves (an occupancy query).  (b) is written once per device
 *    (a racing first call recomputes the same value) and read-only after;
 *    no call's result depends on an earlier call's data.
 *  - Streams.  `stream` is a hipStream_t passed as void* (NULL = the default
 *    stream).  Calls only enqueue work; results are ready once the stream is.
 *  - Errors.  Arguments are validated before anything is enqueued; on a
 *    validation failure the call returns a non-OK status and outputs are left
 *    untouched.  A launch failure reported by the HIP runtime returns
 *    CCI_EHIP.  cci_last_error() gives a message for the last failure on the
 *    calling thread.  No C++ exception crosses this interface.
 *  - Alignment.  Device pointers must be 16-byte aligned (CCI_EALIGN).
 *  - Aliasing.  Outputs must not overlap any input.
 *  - Limits.  1 <= K <= G <= 256; O % G == 0; C >= 1; N >= 0 (N == 0 is a
 *    no-op).  The index is stored as one byte per kept weight.
 *  - Arithmetic.  Products and sums are taken in fp32 (bf16 inputs widen
 *    exactly); a bf16 output is rounded once, to nearest even, after the
 *    fused epilogue.
 */
#ifndef CCI_H
#define CCI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CCI_OK = 0,
  CCI_EINVAL = 1,       /* bad sizes, null pointer, K/G/O out of range      */
  CCI_EUNSUPPORTED = 2, /* valid request this build does not implement      */
  CCI_EALIGN = 3,       /* a device pointer is not 16-byte aligned          */
  CCI_EHIP = 4          /* the HIP runtime reported an error                */
} cci_status;

typedef enum { CCI_F32 = 0, CCI_BF16 = 1 } cci_dtype;

/* Which kernel family computes a product.
 *  CCI_ALGO_AUTO            the library's choice (cost model on the shape).
 *  CCI_ALGO_SPARSE_MAC      Alg. 1 dataflow on the vector ALUs: only the K
 *                           kept weights of each group are multiplied; the G
 *                           outputs of a group stay in registers.  Any dtype
 *                           combination and any C; G in {2,4,8,16,32}.
 *  CCI_ALGO_DENSE_TILE_MFMA packed groups are expanded to dense bf16 tiles in
 *                           LDS and multiplied on the matrix cores.  Needs
 *                           bf16 X and vals, C % 32 == 0 (conv: Cin % 32 ==
 *                           0) and 64 % G == 0.
 *  CCI_ALGO_WIDE_TILE_MFMA  the same expansion with 256-pixel x 256-output
 *                           workgroup tiles (four waves of 128 x 128
 *                           accumulators), for large FC products and 1x1
 *                           convolutions with stride 1 and no padding.  Needs
 *                           bf16 X and vals, C % 64 == 0, O % 256 == 0,
 *                           64 % G == 0, X, vals and Y 16-byte aligned and
 *                           idx 8-byte aligned.
 *  CCI_ALGO_NARROW_MFMA     the same expansion for short reductions: a wave
 *                           keeps the expanded weights of up to 80 outputs
 *                           in registers and streams pixels through them
 *                           (the 1x1 layers of narrow networks, a CNN's
 *                           first conv).  FC products, 1x1 convolutions
 *                           with stride 1 and no padding, and convolutions
 *                           of any geometry with Cin % 8 == 0, or Cin == 4
 *                           and an even KW; bf16 X and vals, C <= 256 (conv:
 *                           KH*KW*Cin), C % 8 == 0, O % 4 == 0, G <= 256;
 *                           X and vals 16-byte aligned, idx 8-byte aligned,
 *                           Y (and residual) 8-byte aligned for bf16 and
 *                           16-byte aligned for fp32 output.
 *  CCI_ALGO_RESIDENT_MFMA   the same expansion for small k x k
 *                           convolutions: the whole expanded tile is kept in
 *                           registers for the launch and each workgroup
 *                           stages the input rows under its band of output
 *                           rows in LDS once.  3x3 convolutions with unit
 *                           stride and padding 0..2, Cin 32 or 64, O 32 or
 *                           64, bf16 X and vals, O/G*K*C/8 <= 5120; X, vals
 *                           and Y 16-byte aligned, idx 8-byte aligned.
 *  CCI_ALGO_FEW_ROWS_MFMA   the few-row product of cci_spmm_bits reading
 *                           cci_pack's byte indices: FC products and 1x1
 *                           convolutions with stride 1 and no padding,
 *                           N <= 64, C % 32 == 0, O % 4 == 0, bf16 X and
 *                           vals (the packed bytes set the time; each is
 *                           read once).
 *  CCI_ALGO_TAP_TILE_MFMA   the same expansion with 128-pixel x 128-output
 *                           workgroup tiles, two workgroups per CU, and a
 *                           reduction in chunks of 64 input channels under
 *                           one filter tap: convolutions of any stride and
 *                           padding through implicit im2col, and FC
 *                           products, with long reductions and few output
 *                           tiles (64 outputs for grids of fewer than 128
 *                           such tiles, or O % 128 != 0).  Needs bf16 X and
 *                           vals, Cin % 64 == 0 (FC: C % 64 == 0), O % 128
 *                           == 0 and 32 % G == 0, or O % 64 == 0 and 16 % G
 *                           == 0; 2 K <= G or K == G; KH*KW <= 32; X, vals
 *                           and Y 16-byte aligned, idx 8-byte aligned.
 *  CCI_ALGO_STREAM_TILE_MFMA the same expansion, done once per workgroup for
 *                           all of a 128- (O % 128 == 0) or 64-output tile's
 *                           reduction and kept in LDS while 128-row tiles of
 *                           X stream past it, their chunks prefetched two
 *                           steps ahead and their epilogues overlapping the
 *                           next tile's loads: short reductions over many
 *                           rows (the 1x1 layers of a CNN's early stages).
 *                           FC products and 1x1 convolutions with stride 1
 *                           and no padding; bf16 X and vals, C % 64 == 0,
 *                           C <= 256, O % 64 == 0, 32 % G == 0; X 16-byte
 *                           aligned, Y (and residual) 8-byte aligned for
 *                           bf16 and 16-byte aligned for fp32 output.
 *  CCI_ALGO_SPLIT_K_MFMA    few row tiles over a long reduction (the
 *                           projecting 1x1 layers of a CNN's late stages):
 *                           eight waves of a workgroup split the reduction
 *                           of one 64 x 32, 32 x 64, 32 x 32 or 32 x 16 (rows
 *                           x outputs) tile, each issuing the loads of its
 *                           k-steps together and building its weight
 *                           fragments in registers from the kept entries
 *                           (Alg. 1's routing: a value lands in the output
 *                           row its index names); the partial tiles are
 *                           added in LDS.  FC products and 1x1 convolutions
 *                           with stride 1 and no padding; bf16 X and vals,
 *                           C % 32 == 0, O % 16 == 0, K <= 4, G <= 256; X,
 *                           vals, idx, Y, scale, bias and residual 16-byte
 *                           aligned. */
typedef enum {
  CCI_ALGO_AUTO = 0,
  CCI_ALGO_SPARSE_MAC = 1,
  CCI_ALGO_DENSE_TILE_MFMA = 2,
  CCI_ALGO_WIDE_TILE_MFMA = 3,
  CCI_ALGO_NARROW_MFMA = 4,
  CCI_ALGO_RESIDENT_MFMA = 5,
  CCI_ALGO_FEW_ROWS_MFMA = 6,
  CCI_ALGO_TAP_TILE_MFMA = 7,
  CCI_ALGO_STREAM_TILE_MFMA = 8,
  CCI_ALGO_SPLIT_K_MFMA = 9
} cci_algo;

/* Optional fused epilogue, applied per output element before rounding:
 *   y = acc * scale[o] + bias[o] + residual[n][o];  y = max(y, 0) if relu.
 * Any pointer may be NULL (scale = 1, bias = 0, residual = 0).  scale and
 * bias are fp32 [O]; residual has Y's shape and dtype.  (Not from the paper:
 * this is the folded batch-norm / residual / ReLU of a CNN layer.) */
typedef struct {
  const float *scale;
  const float *bias;
  const void *residual;
  int32_t relu;
} cci_epilogue;

/* Byte sizes of the packed arrays for an [O][C] weight matrix with groups of
 * G and K kept per group (Sec. 3.1: G rows compress to K rows of C entries).
 * vals: [O/G][K][C] of val_t; idx: [O/G][K][C] uint8.  Pure host arithmetic. */
cci_status cci_packed_sizes(int64_t O, int64_t C, int32_t G, int32_t K,
                            cci_dtype val_t, size_t *val_bytes,
                            size_t *idx_bytes);

/* Magnitude projection onto CCI sparsity (Sec. 5.1: low-|w| weights are
 * pruned; Sec. 3.1: exactly K per group).  For every group g and column c,
 * among w_r = W[gG+r][c] keep the K largest |w| (equal |w|: lower r first;
 * compared as fp32 bit patterns with the sign cleared, so NaN ranks above
 * Inf) and write them in ascending r:
 *   idx[g][k][c] = r,  vals[g][k][c] = w_r  (fp32 copy, or bf16 rounded to
 *   nearest even when val_t == CCI_BF16).
 * W: device fp32 [O][C] (conv: [O][KH][KW][Cin], C = KH*KW*Cin).
 * vals, idx: device outputs of cci_packed_sizes() bytes.  Any G <= 256. */
cci_status cci_pack(const float *W, int64_t O, int64_t C, int32_t G,
                    int32_t K, void *vals, cci_dtype val_t, uint8_t *idx,
                    void *stream);

/* CCI-sparse product (Sec. 3.2, Alg. 1, generalised to K slots):
 *   Y[n][o] = epilogue( sum_c sum_k [gG + idx[g][k][c] == o]
 *                                     vals[g][k][c] * X[n][c] ),  g = o / G.
 * X: device [N][C] of x_t.  vals/idx as produced by cci_pack.  Y: device
 * [N][O] of y_t.  Supported (x_t, val_t, y_t): (F32, F32, F32) and
 * (BF16, BF16, BF16 or F32); anything else is CCI_EUNSUPPORTED.  The kernel
 * family is the library's choice (CCI_ALGO_AUTO). */
cci_status cci_spmm(const void *X, cci_dtype x_t, int64_t N, int64_t C,
                    const void *vals, cci_dtype val_t, const uint8_t *idx,
                    int64_t O, int32_t G, int32_t K, const cci_epilogue *ep,
                    void *Y, cci_dtype y_t, void *stream);

/* Convolution lowered to the CCI product (Sec. 3.2) without materialising
 * the im2col matrix.  X: device NHWC [B][H][W][Cin].  The packed weights
 * describe W [O][KH][KW][Cin] as an [O][C] matrix with C = KH*KW*Cin in
 * (kh, kw, cin) order.  Output pixel p = (b*Ho + oh)*Wo + ow with
 * Ho = (H + 2*pad_h - KH)/stride_h + 1 (Wo likewise); Y: device NHWC
 * [B][Ho][Wo][O], i.e. [N][O] with N = B*Ho*Wo.  Input taps outside the
 * image read as 0.  Dtypes and epilogue as for cci_spmm; the kernel family
 * is the library's choice. */
cci_status cci_conv_im2col(const void *X, cci_dtype x_t, int64_t B, int64_t H,
                           int64_t W, int64_t Cin, int32_t KH, int32_t KW,
                           int32_t stride_h, int32_t stride_w, int32_t pad_h,
                           int32_t pad_w, const void *vals, cci_dtype val_t,
                           const uint8_t *idx, int64_t O, int32_t G, int32_t K,
                           const cci_epilogue *ep, void *Y, cci_dtype y_t,
                           void *stream);

/* cci_spmm / cci_conv_im2col with the kernel family pinned (see cci_algo;
 * CCI_ALGO_AUTO gives the plain calls).  Same arguments, result and
 * errors; an explicit family whose requirements the shape does not meet
 * returns CCI_EUNSUPPORTED.  For benchmarking and testing each family. */
cci_status cci_spmm_algo(const void *X, cci_dtype x_t, int64_t N, int64_t C,
                         const void *vals, cci_dtype val_t, const uint8_t *idx,
                         int64_t O, int32_t G, int32_t K,
                         const cci_epilogue *ep, void *Y, cci_dtype y_t,
                         cci_algo algo, void *stream);
cci_status cci_conv_im2col_algo(const void *X, cci_dtype x_t, int64_t B,
                                int64_t H, int64_t W, int64_t Cin, int32_t KH,
                                int32_t KW, int32_t stride_h, int32_t stride_w,
                                int32_t pad_h, int32_t pad_w, const void *vals,
                                cci_dtype val_t, const uint8_t *idx, int64_t O,
                                int32_t G, int32_t K, const cci_epilogue *ep,
                                void *Y, cci_dtype y_t, cci_algo algo,
                                void *stream);

/* Which family CCI_ALGO_AUTO picks for a product of N x C x O (conv: pass
 * N = B*Ho*Wo, C = KH*KW*Cin and cin = Cin; FC: cin = C).  Host-only.  A
 * 1x1 convolution reported as CCI_ALGO_WIDE_TILE_MFMA runs on the tap-chunk
 * kernels (else the dense-tile ones) when its stride or padding rules the
 * wide-tile ones out; one reported as CCI_ALGO_NARROW_MFMA then runs on the
 * dense-tile kernels if they take its shape, else on the sparse-MAC ones;
 * one reported as CCI_ALGO_RESIDENT_MFMA or CCI_ALGO_TAP_TILE_MFMA runs on
 * the dense-tile kernels when a stride, alignment or size limit of that
 * family rules it out; one reported as CCI_ALGO_STREAM_TILE_MFMA runs on the
 * tap-chunk kernels (else the dense-tile ones) when its stride, padding or
 * alignment rules the streaming ones out; one reported as
 * CCI_ALGO_SPLIT_K_MFMA runs on the dense-tile kernels when its stride,
 * padding or alignment rules the split-reduction ones out. */
cci_algo cci_auto_algo(cci_dtype x_t, cci_dtype val_t, int64_t N, int64_t C,
                       int64_t cin, int64_t O, int32_t G, int32_t K);

/* ------------------------------------------------------------------------
 * Balanced sparsity (Sec. 2.4, Sec. 3.3, Fig. 2b): the paper's comparison
 * structure.  Its groups are G contiguous weights of one output row (weights
 * of different inputs); each keeps exactly K, and the index of a kept weight
 * names the input of its group it multiplies.
 * ------------------------------------------------------------------------ */

/* Byte sizes of the balanced packing of an O x C matrix: vals [O][C/G][K]
 * of val_t, idx [O][C/G][K] uint8.  CCI_EINVAL unless C % G == 0 and
 * 1 <= K <= G <= 256. */
cci_status cci_bbs_packed_sizes(int64_t O, int64_t C, int32_t G, int32_t K,
                                cci_dtype val_t, size_t *val_bytes,
                                size_t *idx_bytes);

/* Balanced projection of a dense fp32 W [O][C]: for each row o and group j
 * (inputs jG .. jG+G-1) keep the K largest |w| (magnitude order and ties as
 * for cci_pack: lower position wins), in ascending position:
 *   vals[o][j][k] = W[o][jG + idx[o][j][k]]  (exact, or rounded once to bf16).
 * Errors as for cci_pack. */
cci_status cci_bbs_pack(const float *W, int64_t O, int64_t C, int32_t G,
                        int32_t K, void *vals, cci_dtype val_t, uint8_t *idx,
                        void *stream);

/* The 2:4 operand of gfx950's sparse matrix cores.  A matrix A [M][R] in
 * which every aligned run of 4 reduction positions holds at most 2 nonzeros
 * is stored as 2 bf16 values and 2-bit positions per run, in fragment order:
 *   a_vals bf16 [R/64][M/16][64][8], a_idx uint16 [R/64][M/16][64]
 * (lane l of fragment (s, mb): row 16 mb + l % 16, reduction columns
 * 64 s + 16 (l / 16) .. +15; value e sits at column 4 (e / 2) + bits
 * 2e..2e+1 of the index word of those).  M % 16 == 0 and R % 64 == 0
 * (CCI_EUNSUPPORTED otherwise); sizes in bytes M*R and M*R/8. */
cci_status cci_2of4_sizes(int64_t M, int64_t R, size_t *val_bytes,
                          size_t *idx_bytes);

/* The 2:4 operand of a balanced packing (bf16 vals, as from cci_bbs_pack) of
 * an O x C matrix: rows M = O, reduction R = C.  Each run of 4 inputs holds
 * at most 2 kept weights when G % 4 == 0 and K <= 2; other (G, K) return
 * CCI_EUNSUPPORTED.  Unused slots hold 0. */
cci_status cci_bbs_to_2of4(const void *vals, cci_dtype val_t,
                           const uint8_t *idx, int64_t O, int64_t C, int32_t G,
                           int32_t K, void *a_vals, uint16_t *a_idx,
                           void *stream);

/* The 2:4 operand of W_hat^T for a CCI packing of W_hat [O][C] (bf16 vals,
 * as from cci_pack): rows M = C, reduction R = O.  Along the output channels
 * a CCI group keeps K of G (Sec. 3.1), so the backward product
 * dX = dY . W_hat reduces over 2:4-sparse runs when G % 4 == 0 and K <= 2
 * (else CCI_EUNSUPPORTED). */
cci_status cci_to_2of4_transposed(const void *vals, cci_dtype val_t,
                                  const uint8_t *idx, int64_t O, int64_t C,
                                  int32_t G, int32_t K, void *a_vals,
                                  uint16_t *a_idx, void *stream);

/* Y[n][m] = epilogue( sum_r A[m][r] * X[n][r] ) on the sparse matrix cores
 * (v_smfmac_f32_16x16x64_bf16; fp32 accumulation, one rounding of a bf16
 * Y).  X: device bf16 [N][R]; A: a prepared 2:4 operand [M][R]; Y: device
 * [N][M] of y_t (BF16 or F32); epilogue as for cci_spmm (vectors of M).
 * With A from cci_bbs_to_2of4 this is the balanced-sparse forward product;
 * with A from cci_to_2of4_transposed and X = dY it is dX = dY . W_hat.
 * X is read as exact products of the stored values: unused slots multiply
 * their (finite) inputs by 0. */
cci_status cci_spmm_2of4(const void *X, cci_dtype x_t, int64_t N, int64_t R,
                         const void *a_vals, const uint16_t *a_idx, int64_t M,
                         const cci_epilogue *ep, void *Y, cci_dtype y_t,
                         void *stream);

/* ------------------------------------------------------------------------
 * Improved targeted dropout (Sec. 5.1; schedule of Sec. 6): training a CCI
 * layer from a dense W.  Each step drops some of the "candidates" -- the
 * n_target lowest-|w| weights of every CCI group -- with probability
 * drop_rate; the forward and backward use the result W_eff.  Over the run the
 * candidate count ramps up, then the dropout rate ramps to 1, where W_eff is
 * exactly the CCI projection (cci_pack).  Once the mask is fixed the layer's
 * backward products are dX = dY . W_hat (cci_to_2of4_transposed +
 * cci_spmm_2of4) and the gradient of the packed values (cci_grad_packed).
 * ------------------------------------------------------------------------ */

/* The schedule at `step` of `total` (0 <= step <= total), f = step/total:
 *   *n_target  = floor((G - K) * min(1, 2 f) + 1/2)   candidates per group,
 *   *drop_rate = max(1/2, f).
 * (The first half ramps the candidates at dropout 1/2, the second ramps the
 * dropout from 1/2 to 1; both ramps linear.)  Host-only. */
cci_status cci_td_schedule(int64_t step, int64_t total, int32_t G, int32_t K,
                           int32_t *n_target, double *drop_rate);

/* Candidate dropout of one step.  W: device fp32 [O][C] (O % G == 0).  In
 * each CCI group (rows gG .. gG+G-1 at column c) the weights of rank
 * >= G - n_target by |w| (larger first, ties to the lower row, as in
 * cci_pack) are candidates; a candidate is dropped iff its random word
 * bits[o][c] (device uint32 [O][C], uniform, drawn by the caller) is below
 * floor(drop_rate * 2^32).  Writes W_eff [O][C] of w_t (the weight, rounded
 * once for bf16, or 0 if dropped) and keep [O][C] uint8 (0 if dropped, else
 * 1).  0 <= n_target <= G, 0 <= drop_rate <= 1. */
cci_status cci_td_mask(const float *W, int64_t O, int64_t C, int32_t G,
                       int32_t n_target, const uint32_t *bits,
                       double drop_rate, void *W_eff, cci_dtype w_t,
                       uint8_t *keep, void *stream);

/* Gradient of the packed values of Y = X . W_hat^T (Alg. 1's product):
 *   dvals[g][k][c] = sum_n dY[n][gG + idx[g][k][c]] * X[n][c],
 * fp32 accumulation.  dY: device [N][O], X: device [N][C], both of dtype t
 * (F32 or BF16); idx as from cci_pack; dvals: device fp32 [O/G][K][C].
 * bf16 operands with N >= 32, O % 8 == 0, C % 8 == 0 and 128 % G == 0 run
 * on the matrix cores (the dense tiles of dY^T X, summed over samples in
 * steps of 32, kept entries written); other calls multiply only kept
 * weights on the vector ALUs, summing in n order. */
cci_status cci_grad_packed(const void *dY, const void *X, cci_dtype t,
                           int64_t N, int64_t C, const uint8_t *idx, int64_t O,
                           int32_t G, int32_t K, float *dvals, void *stream);

/* ------------------------------------------------------------------------
 * Plain log2(G)-bit indices (Sec. 3.1: each kept weight's index into its
 * group is stored in log2 G bits).  Stream format: with b bits per entry,
 * entry e of an index array occupies bits e*b .. e*b+b-1 of a little-endian
 * stream of 32-bit words (stream bit t is bit t % 32 of word t / 32); bits
 * past the last entry are 0.  b = 8 is exactly the byte array of cci_pack.
 * ------------------------------------------------------------------------ */

/* ceil(log2 G), at least 1: the plain index width of groups of G.  -1 if G
 * is outside [1, 256].  Host-only. */
int32_t cci_index_width(int32_t G);

/* Bytes of the stream of n entries of `bits` bits: ceil(n*bits/32)*4. */
cci_status cci_index_stream_bytes(int64_t n, int32_t bits, size_t *bytes);

/* The byte index array idx (n entries, as from cci_pack) as a stream of
 * `bits`-bit entries (1 <= bits <= 8).  Entries must be < 2^bits (a packing
 * with G <= 2^bits; higher bits are dropped).  words: device uint32 of
 * cci_index_stream_bytes bytes. */
cci_status cci_index_bits(const uint8_t *idx, int64_t n, int32_t bits,
                          uint32_t *words, void *stream);

/* The CCI product of cci_spmm with the indices read as `idx_bits`-bit
 * entries: idx is the stream of cci_index_bits for
 * cci_index_width(G) <= idx_bits < 8, or the byte array of cci_pack for
 * idx_bits = 8.  This is the few-row product (N <= 64: a decode-sized batch)
 * where the packed weight bytes set the time; bf16 X and values, C % 32 == 0,
 * O % 4 == 0 (CCI_EUNSUPPORTED otherwise).  Epilogue and output as for
 * cci_spmm. */
cci_status cci_spmm_bits(const void *X, cci_dtype x_t, int64_t N, int64_t C,
                         const void *vals, cci_dtype val_t, const void *idx,
                         int32_t idx_bits, int64_t O, int32_t G, int32_t K,
                         const cci_epilogue *ep, void *Y, cci_dtype y_t,
                         void *stream);

/* CNN glue for the ResNet-shaped forward (not from the paper).
 * Max pooling, NHWC, window k, stride s, padding p (padding never wins).
 * X, Y: device [B][H][W][C] -> [B][Ho][Wo][C] of dtype t (F32 or BF16). */
cci_status cci_maxpool2d_nhwc(const void *X, cci_dtype t, int64_t B, int64_t H,
                              int64_t W, int64_t C, int32_t k, int32_t s,
                              int32_t p, void *Y, void *stream);

/* Global average pooling, NHWC [B][H][W][C] of x_t -> [B][C] of y_t, summed
 * in fp32 then divided by H*W. */
cci_status cci_global_avgpool_nhwc(const void *X, cci_dtype x_t, int64_t B,
                                   int64_t H, int64_t W, int64_t C, void *Y,
                                   cci_dtype y_t, void *stream);

/* Static description of a status code. */
const char *cci_status_str(cci_status s);

/* Message for the last non-OK status returned on the calling thread
 * ("" if none).  Valid until the next library call on that thread. */
const char *cci_last_error(void);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int32_t cci_version(void);

#ifdef __cplusplus
}
#endif

#endif /* CCI_H */
