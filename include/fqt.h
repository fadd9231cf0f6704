/*
 * fqt.h -- C ABI of libfqt.so: the fully-quantized-training (FQT) backward of
 * one linear or conv layer on an MI355X (gfx950).
 *
 * Method: Chen, Gai, Yao, Mahoney, Gonzalez, "A Statistical Framework for
 * Low-bitwidth Training of Deep Neural Networks" (NeurIPS 2020).
 *   Sec. 2.2, Eq. (linear-sq-backprop):  grad_W = Q_b(G)^T Q_f(X),
 *                                         grad_X = Q_b(G)   Q_theta(W)
 *   Sec. 3.3  per-tensor quantizer (PTQ) with stochastic rounding SR
 *   Sec. 4.1  per-sample quantizer (PSQ)
 *   Sec. 4.2, App. C.4, App. D  block Householder quantizer (BHQ)
 *   App. E    gradient bifurcation: Q_b1 (8-bit stochastic PTQ) feeds
 *             grad_W, Q_b2 (PTQ / PSQ / BHQ, 4-8 bits) feeds grad_X;
 *             Q_f and Q_theta are deterministic 8-bit PTQ.
 *
 * Conventions for every entry point
 *   - Row-major; a row is a sample (or token).  PyTorch orientation:
 *     X [N, d_in], W [d_out, d_in], G = dL/dY [N, d_out].
 *   - All array pointers are DEVICE pointers owned by the caller; only the
 *     small configuration structs (`cfg`, `shape`) are host memory.
 *   - `ws` is a caller-owned device workspace of at least the size the
 *     matching *_workspace() query returns; the library never allocates.
 *   - Work is enqueued asynchronously on `stream` (0 = the null stream).
 *     The library keeps no state between calls; calls on different
 *     workspaces may run concurrently.
 *   - Argument errors are reported synchronously, before anything is
 *     enqueued.  Data errors (a NaN or Inf in an input, or a range that
 *     overflows float32) are recorded in the workspace and returned by
 *     fqt_workspace_status(); outputs are then unspecified.
 *   - Stochastic rounding draw for logical element e (row-major index in the
 *     quantized matrix) = Philox4x32-7 (Salmon et al., SC'11, seven rounds)
 *     with key = seed, counter = (e >> 2, stream, 0), word e & 3; its low
 *     24 bits are the uniform.
 *     Results are a deterministic function of (inputs, seed, stream).
 *   - Codes are stored as int8 offset codes q = code - 2^(bits-1), where code
 *     in [0, 2^bits - 1] is the quantization bin of Sec. 3.3.
 */
#ifndef FQT_H_
#define FQT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* fqt_stream_t; /* same object as hipStream_t */

typedef enum {
  FQT_OK = 0,
  FQT_EINVAL = 1,        /* bad argument (NULL, size <= 0, bits outside 1..8, ...) */
  FQT_EUNSUPPORTED = 2,  /* valid per the paper but not implemented here */
  FQT_ENONFINITE = 3,    /* NaN / Inf input or float32 range overflow */
  FQT_EWORKSPACE = 4,    /* ws NULL or ws_bytes below the query */
  FQT_EDEVICE = 5        /* a HIP runtime call failed */
} fqt_status;

/* FQT_SHIFT: per-tensor range with per-sample power-of-two steps (Sec. 4.3,
 * the variant for integer hardware): a grad_W quantizer (qb_w) whose
 * per-sample scales survive the int8 contraction over samples.           */
typedef enum { FQT_PTQ = 0, FQT_PSQ = 1, FQT_BHQ = 2, FQT_SHIFT = 3 } fqt_kind;

/* One quantized matrix (Sec. 3.3 / Eq. matrix-quantizer).  Every pointer is
 * caller-owned device memory; a NULL optional pointer is skipped.
 *   q         codes, offset form.  Natural layout [rows, cols]; for BHQ the
 *             rows are in slot order (grouped, see perm).  Transposed layout
 *             [cols, rows] where the entry point says so.
 *   scale     PTQ: [1] s.  PSQ: [rows] s_i.  BHQ: [rows] per slot d_p
 *             (s1 for a group's first slot, s2 for the others; a one-row
 *             group holds its PSQ scale).
 *   zero      PTQ: [1] z.  PSQ: [rows] z_i = row min.  BHQ: [rows] per slot:
 *             the group's transformed-domain offset c_g (one-row group: its
 *             row min, as PSQ).
 *   perm      BHQ only: [rows] slot -> original row.
 *   group_off BHQ only, optional: [rows + 1]; the first G + 1 entries are
 *             the group boundaries in slot order.
 *   code_sum  optional int32 sums of q along the contiguous axis of the
 *             stored layout: [rows] for natural, [cols] for transposed.
 *   num_groups BHQ only, optional: one int32, the number of groups G.
 * Dequantized value: PTQ/PSQ code / s + z.  BHQ group of k_g > 1 slots:
 * diag(d)^-1 H (code + c_g), H the k_g x k_g Householder reflection with
 * normal 1/sqrt(k_g) - e_1 (Sec. 4.2).                                      */
typedef struct {
  int8_t* q;
  float* scale;
  float* zero;
  int32_t* perm;
  int32_t* group_off;
  int32_t* code_sum;
  int8_t* shift;  /* FQT_SHIFT only: [rows] left shift of each row's offset codes */
  int32_t* num_groups;
} fqt_qtensor;

/* Per-tensor quantizer, Sec. 3.3: z = min x, s = B / (max x - min x),
 * code = SR(s (x - z)) (stochastic != 0) or round-half-even (stochastic == 0),
 * clamped to [0, B], B = 2^bits - 1.  transpose != 0 stores q as [cols, rows].
 * Needs out->q, out->scale, out->zero.  bits in 1..8.                        */
fqt_status fqt_quantize_ptq(const float* x, int64_t rows, int64_t cols, int bits, int stochastic,
                            uint64_t seed, uint32_t stream, int transpose, const fqt_qtensor* out,
                            void* ws, size_t ws_bytes, fqt_stream_t s);

/* Per-sample quantizer, Sec. 4.1: per row z_i = min, s_i = B / R_i, SR.
 * Natural layout.  Needs out->q, out->scale [rows], out->zero [rows].       */
fqt_status fqt_quantize_psq(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed,
                            uint32_t stream, const fqt_qtensor* out, void* ws, size_t ws_bytes,
                            fqt_stream_t s);

/* fqt_quantize_psq without a workspace argument, for callers that cannot
 * allocate device memory (code under stream capture, tight serving loops,
 * harnesses that forbid allocation).  The same kernels and results as
 * fqt_quantize_psq; the scratch memory they need comes from a fixed 4 MiB
 * array that the library holds on each GPU until the process ends.  The
 * call itself allocates nothing.  Sizes whose fqt_quantize_workspace(FQT_PSQ,
 * rows, cols, 0) exceeds 4 MiB return FQT_EUNSUPPORTED (for cols <= 8192
 * that allows about 250 000 rows).  status (optional, device, 4 uint32
 * words) receives the data status: bit 0 set in any word means a non-finite
 * input.  Every call on one GPU shares that GPU's array, which keeps the
 * last call's contents: calls that overlap on one GPU (several streams or
 * host threads) race and must be serialized by the caller.                 */
fqt_status fqt_quantize_psq_noalloc(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed,
                                    uint32_t stream, const fqt_qtensor* out, uint32_t* status, fqt_stream_t s);

/* Block Householder quantizer, Sec. 4.2 / App. C.4 / App. D.  Rows are
 * sorted by infinity norm M (descending, ties by row index); each group
 * holds one of the G largest rows and a run of the sorted tail.
 *   block_size = k >= 1: G = ceil(rows / k) groups, group g takes the g-th
 *     largest row and the next k - 1 rows of the tail (the last groups may
 *     be shorter, see group_off).
 *   block_size = 0: App. D's adaptive groups (fqt_bhq_adaptive_groups), all
 *     on the device, nothing waits; rows <= 65536 (FQT_EUNSUPPORTED beyond).
 * The transform Q diag(d) G_g of each group sums its column over the group's
 * slots one at a time in slot order (float32).  Codes are in slot order,
 * natural layout.  Needs out->q, scale, zero, perm.                         */
fqt_status fqt_quantize_bhq(const float* x, int64_t rows, int64_t cols, int bits, int block_size,
                            uint64_t seed, uint32_t stream, const fqt_qtensor* out, void* ws,
                            size_t ws_bytes, fqt_stream_t s);

/* Per-tensor range with per-sample power-of-two steps, Sec. 4.3: R = max_i
 * R_i (the largest row range), s = B / R; row i has z_i = row min and the
 * largest e_i in [0, E], E = min(4, 8 - bits), with R_i 2^e_i <= R, so
 * s_i = s 2^e_i (saturating at FLT_MAX); code = SR(s_i (x - z_i)) as PSQ.
 * q holds each row's offset code shifted left by shift[i] = E - e_i, which
 * stays in int8: every row then counts in the common step 1 / (s 2^E), so an
 * int8 contraction over rows is exact.  code_sum sums the shifted codes.
 * Natural ([rows, cols]) or transposed (transpose != 0) layout.  Needs
 * out->q, out->scale [rows] (s_i), out->zero [rows] (z_i), out->shift.     */
fqt_status fqt_quantize_shift(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed,
                              uint32_t stream, int transpose, const fqt_qtensor* out, void* ws,
                              size_t ws_bytes, fqt_stream_t s);

size_t fqt_quantize_workspace(fqt_kind kind, int64_t rows, int64_t cols, int block_size);

/* Seed batch of one stochastic quantizer (Sec. 3.3 SR; the unbiasedness of
 * Sec. 2.2 and the variance of App. C measured over seeds): the quantizer
 * kind (FQT_PTQ, FQT_PSQ or FQT_BHQ with block_size as for
 * fqt_quantize_bhq) plans once and rounds the same transformed values under
 * the keys seed, seed + 1, .., seed + nseeds - 1 (1 <= nseeds <= 32768),
 * each exactly as the single-seed quantizer with that seed would.  Instead
 * of codes it writes, per element of the natural layout (BHQ: slot order),
 * sum_code = sum over seeds of the code in [0, B] and sum_code2 = the sum of
 * its squares (int32, [rows, cols], 16-byte aligned).  plan receives scale,
 * zero (and perm, group_off, num_groups for BHQ) as for the single
 * quantizers; plan->q is not used.  cols % 4 == 0 and x 16-byte aligned
 * (FQT_EUNSUPPORTED otherwise).  Workspace: fqt_quantize_workspace(kind, ..). */
fqt_status fqt_quantize_seeds(const float* x, int64_t rows, int64_t cols, fqt_kind kind, int bits, int block_size,
                              uint64_t seed, int32_t nseeds, uint32_t stream, const fqt_qtensor* plan,
                              int32_t* sum_code, int32_t* sum_code2, void* ws, size_t ws_bytes, fqt_stream_t s);

/* Adaptive grouping of the block Householder quantizer, App. D step 2: for
 * every number of groups G = 1..rows, the G largest rows lead the groups
 * and the rows - G others are shared out in sorted order in proportion to
 * the leaders' norms: the first i groups take floor((rows - G) P_i / P_G +
 * 1/2) of them, P_i = M_(1) + .. + M_(i) summed in float64 one at a time.
 * Each G is scored by the exact |S^-1|_F^2 of its plan (the factor of the
 * variance bound (D/4)|S^-1|_F^2, Eq. matrix-quantizer-variance), groups
 * added in order in float64; the least wins, ties to the smaller G.  (App.
 * D's own estimate, sum_i M_i^2 / ((N - G) M_i / sum_j M_j), grows with G
 * and would always keep one group.)  Asynchronous on `stream`: writes the
 * chosen G to num_groups (one device int32) and, if objective is not NULL,
 * the score of every G to objective[G - 1] (device, [rows] float64).
 * O(rows^2) work; rows <= 65536 (FQT_EUNSUPPORTED beyond).  A non-finite x
 * is reported by fqt_workspace_status (the plan then treats its norms as 0). */
fqt_status fqt_bhq_adaptive_groups(const float* x, int64_t rows, int64_t cols, int bits, int32_t* num_groups,
                                   double* objective, void* ws, size_t ws_bytes, fqt_stream_t s);
size_t fqt_bhq_adaptive_workspace(int64_t rows, int64_t cols);

/* Quantizer choice for one gradient quantizer. */
typedef struct {
  fqt_kind kind;   /* FQT_PTQ, FQT_PSQ or FQT_BHQ */
  int bits;        /* 1..8 */
  int block_size;  /* BHQ only: block size k >= 1, or 0 for App. D's adaptive groups
                   * (fqt_bhq_adaptive_groups; needs N <= 65536) */
} fqt_qspec;

/* Optional per-phase timing: when fqt_bwd_cfg.trace is non-NULL, the layer
 * backward records start[i] / stop[i] (caller-created hipEvent_t handles)
 * around phase i on `stream`, for i < count.  Phases of the layer backward:
 *   0 workspace init   1 stats X, W, G   2 scales / BHQ plan
 *   3 quantize X       4 quantize W      5 quantize G (Q_b1 and Q_b2)
 *   6 grad_W contraction (with any split-K reduction)
 *   7 grad_X contraction                                                    */
#define FQT_TRACE_PHASES 8
typedef struct {
  void* start[FQT_TRACE_PHASES];
  void* stop[FQT_TRACE_PHASES];
  int count;
} fqt_trace;

/* Layer backward configuration (App. E).  qb_w feeds grad_W and must be PTQ
 * or, for the linear layer, FQT_SHIFT (per-row scales lie on grad_W's
 * contraction axis; power-of-two ones survive it as shifted codes; PSQ / BHQ
 * return FQT_EUNSUPPORTED).  qb_x feeds grad_X (PTQ, PSQ or BHQ).  f_bits / theta_bits are the
 * deterministic PTQ widths of X and W.  Q_b1 draws from stream 0 and Q_b2
 * from stream 1 of `seed`.
 * relu_input (linear layer only; the conv returns FQT_EUNSUPPORTED): X is the
 * output of a ReLU, and grad_X is multiplied by that ReLU's derivative,
 * 1[X > 0], so it is the gradient of the previous layer's pre-activation.
 * The ReLU takes no gradient quantizer: its Jacobian is applied exactly to
 * the float result, as to any elementwise layer of a multi-layer chain
 * (Sec. 2.2, Eq. (quantized-back-prop) with the identity as its quantizer). */
typedef struct {
  fqt_qspec qb_w;
  fqt_qspec qb_x;
  int f_bits;
  int theta_bits;
  uint64_t seed;
  const fqt_trace* trace; /* optional, NULL for none */
  int relu_input;         /* 0: plain grad_X; 1: grad_X * 1[X > 0] */
  /* Optional caller buffers (device; linear layer only, the conv ignores
   * them) that receive the gradient codes the contractions read, in place of
   * the workspace copies:
   *   qb2_codes [N, d_out]  Q_b2(G) offset codes, rows in slot order; with
   *                         packed_codes they are [N, d_out / 2] bytes,
   *                         code + 2^(b-1) in a nibble (column 2i in the low
   *                         half of byte i)
   *   qb1_codes [d_out, N]  Q_b1(G) offset codes, transposed, slot order
   *   perm      [N]         BHQ: slot -> row (not written for PTQ / PSQ,
   *                         whose slot order is the row order)             */
  int8_t* qb2_codes;
  int8_t* qb1_codes;
  int32_t* perm;
  /* packed_codes (linear layer): 1 stores Q_b2 codes of at most 4 bits two
   * per byte (qb_x.bits <= 4, d_out % 16 == 0; ignored otherwise), halving
   * their bytes; the grad_X contraction unpacks them as it loads them (its
   * register-staged loop, slower than the int8 path's direct-to-LDS loop).
   * 0 keeps one byte per code.                                             */
  int packed_codes;
} fqt_bwd_cfg;

/* Linear layer FQT backward, Eq. (linear-sq-backprop) with bifurcation:
 *   grad_W [d_out, d_in] = Q_b1(G)^T Q_f(X)
 *   grad_X [N, d_in]     = Q_b2(G)   Q_theta(W)
 * both contracted on int8 matrix cores with exact int32 accumulators
 * (int64 across K-splits) and dequantized in float64, rounded to float32.
 * With cfg->packed_codes, Q_b2 codes of at most 4 bits are stored two per
 * byte and unpacked as the grad_X contraction loads them.
 * Outputs are overwritten.  N, d_in, d_out >= 1.                            */
fqt_status fqt_linear_backward(const float* X, const float* W, const float* G, int64_t N, int64_t d_in,
                               int64_t d_out, const fqt_bwd_cfg* cfg, float* grad_W, float* grad_X,
                               void* ws, size_t ws_bytes, fqt_stream_t s);

size_t fqt_linear_backward_workspace(int64_t N, int64_t d_in, int64_t d_out, const fqt_bwd_cfg* cfg);

/* Linear layer forward of quantization-aware training (Sec. 2.1, Eq.
 * (quantized-forward-propagation)):
 *   Y [N, d_out] = Q_f(X) Q_theta(W)^T,   optionally Y = max(Y, 0) (relu != 0)
 * with Q_f, Q_theta the deterministic per-tensor PTQ of X [N, d_in] and
 * W [d_out, d_in] at f_bits / theta_bits (round half to even, Sec. 3.3
 * ranges), contracted on int8 matrix cores with exact int32 accumulators
 * (int64 across K-splits of d_in > 65536) and dequantized in float64, rounded
 * to float32.  The same quantizers as the backward, so a layer's forward and
 * backward see identical Q_f(X) and Q_theta(W).  Y is overwritten; a
 * non-finite X or W is reported through the workspace status word.
 * N, d_in, d_out >= 1; bits in 1..8.                                        */
fqt_status fqt_linear_forward(const float* X, const float* W, int64_t N, int64_t d_in, int64_t d_out, int f_bits,
                              int theta_bits, int relu, float* Y, void* ws, size_t ws_bytes, fqt_stream_t s);

size_t fqt_linear_forward_workspace(int64_t N, int64_t d_in, int64_t d_out);

/* Conv geometry: X NHWC [n, h, w, c], W [o, kh, kw, c], G NHWC [n, ho, wo, o],
 * ho = (h + 2 pad - kh) / stride + 1 (likewise wo); zero padding.           */
typedef struct {
  int n, c, h, w, o, kh, kw, stride, pad, ho, wo;
} fqt_conv_shape;

/* Conv layer FQT backward (Sec. 2.2 applied to the conv as the linear layer
 * Y = im2col(X) W^T): grad_W = Q_b1(G)^T im2col(Q_f(X)) and
 * grad_X = col2im(Q_b2(G) Q_theta(W)).  Quantizer rows are samples
 * (Sec. 4.1): X and W per tensor, G [n, ho*wo*o] per sample / group.
 * Padding taps contribute exactly zero.
 *   cfg->qb_x: Q_b2, PTQ / PSQ / BHQ (any block size, 0 = App. D groups).
 *   cfg->qb_w: Q_b1, PTQ, or PSQ (Sec. 4.1's per-sample scales on grad_W:
 *              each sample's output pixels are one int32-exact K block of
 *              the contraction, scaled by the sample's 1 / s in float64;
 *              ho * wo <= 65536 and n <= 65535, else FQT_EUNSUPPORTED).
 *              The shift form is linear-only (FQT_EUNSUPPORTED here).
 *   cfg->relu_input must be 0 (FQT_EUNSUPPORTED).
 * Outputs grad_W [o, kh, kw, c] and grad_X [n, h, w, c] are overwritten.
 * grad_X may be NULL: the input gradient is then not formed (no Q_b2, no
 * Q_theta(W), no grad_X contraction), as for a first layer whose input
 * takes no gradient; grad_W is the same as with it.  o % 16 == 0.          */
fqt_status fqt_conv_backward_im2col(const float* X, const float* W, const float* G,
                                    const fqt_conv_shape* shape, const fqt_bwd_cfg* cfg, float* grad_W,
                                    float* grad_X, void* ws, size_t ws_bytes, fqt_stream_t s);

size_t fqt_conv_backward_workspace(const fqt_conv_shape* shape, const fqt_bwd_cfg* cfg);

/* Exact int8 contraction C[m, n] = sum_k A[m, k] B[n, k] (both K-contiguous,
 * row strides lda, ldb in bytes >= K), int64 output [M, N].  int32
 * accumulation over K-chunks of at most 65536, summed in int64.  The same
 * kernels as the layer backward; exported to test accumulators bit-exactly. */
fqt_status fqt_gemm_s8s8_s64(const int8_t* A, const int8_t* B, int64_t M, int64_t N, int64_t K, int64_t lda,
                             int64_t ldb, int64_t* C, void* ws, size_t ws_bytes, fqt_stream_t s);

size_t fqt_gemm_workspace(int64_t M, int64_t N, int64_t K);

/* The same exact contraction for 4-bit offset codes (A, B int8 in [-8, 7]) on
 * the 6-bit float matrix cores: both operands are repacked as e3m2 (every
 * integer in [-8, 8] is one) into the workspace and contracted with float32
 * accumulation, which stays exact for K chunks of at most 131072 (|sum| <
 * 2^24); chunks are summed in int64 into C [M, N].  A code outside [-8, 7]
 * is a data error: the workspace status reports FQT_ENONFINITE.  Sub-8-bit
 * matrix formats for small codes (the storage and contraction of b <= 4-bit
 * codes; Sec. 3.3 codes are integers in [0, 2^b - 1]).                     */
fqt_status fqt_gemm_s4s4_bf6(const int8_t* A, const int8_t* B, int64_t M, int64_t N, int64_t K, int64_t lda,
                             int64_t ldb, int64_t* C, void* ws, size_t ws_bytes, fqt_stream_t s);
size_t fqt_gemm_s4s4_bf6_workspace(int64_t M, int64_t N, int64_t K);

/* Waits for `s`, then reports the data status recorded in `ws` by the last
 * call that used it: FQT_OK or FQT_ENONFINITE (FQT_EDEVICE if the wait or
 * copy fails).                                                              */
fqt_status fqt_workspace_status(const void* ws, fqt_stream_t s);

/* Machine probes for measured peaks (the roofline's second reference).
 * fqt_probe_mfma_i8: iters back-to-back v_mfma_i32_32x32x32_i8 on four
 * independent register accumulators in every wave of 2048 blocks x 4 waves;
 * *ops (host) receives the int8 operation count, to be divided by the time
 * the caller measures on `s`.  sink: one device int32 (written only by an
 * improbable checksum).  fqt_probe_copy: a streaming 16-byte copy of `bytes`
 * (a multiple of 16, 16-byte aligned device buffers); moved bytes = 2 bytes. */
fqt_status fqt_probe_mfma_i8(int64_t iters, int32_t* sink, double* ops, fqt_stream_t s);
fqt_status fqt_probe_copy(const void* src, void* dst, size_t bytes, fqt_stream_t s);

const char* fqt_status_str(fqt_status st);

/* Library version string. */
const char* fqt_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FQT_H_ */
