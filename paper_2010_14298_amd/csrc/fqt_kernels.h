// Internal launch interface between the FQT host layer (api.hip) and the
// kernels (quant.hip, gemm.hip, conv.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fqt {

// ---- quantizer front end -------------------------------------------------

// Statistics: each block reduces one chunk of a flat tensor (rows = 1) or
// of one row, into part[row * chunks + chunk] = (min, max); min is NaN when
// the chunk holds a non-finite value.
// A per-row segment whose rows fit one block (chunks == 1) also gets the
// row ranges written directly: rmin[row] (+inf for a non-finite row, as the
// finalize combination of one NaN-flagged partial gives) and rmax[row].
struct StatsSeg {
  const float* x;
  int64_t rows, cols;
  int64_t chunk;   // columns per block
  int64_t chunks;  // blocks per row
  float2* part;
  float* rmin;     // direct per-row ranges (chunks == 1), else nullptr
  float* rmax;
};
StatsSeg stats_flat_seg(const float* x, int64_t n);
StatsSeg stats_rows_seg(const float* x, int64_t rows, int64_t cols);
// Route the row ranges of a per-row segment straight to rmin / rmax when a
// block covers a whole row.
inline void stats_direct_rows(StatsSeg& g, float* rmin, float* rmax) {
  if (g.chunks == 1) {
    g.rmin = rmin;
    g.rmax = rmax;
  }
}
__host__ __device__ inline int64_t stats_partials(const StatsSeg& g) { return g.rows * g.chunks; }
struct StatsPlan {
  StatsSeg seg[3];
  int nseg;
  int64_t block_start[4];
};
hipError_t launch_stats(StatsPlan sp, hipStream_t s);

// One finalize block: per-tensor PTQ scale / zero (Sec. 3.3), per-row PSQ
// scale / zero (Sec. 4.1), per-row min / max of the row segment, cleared
// int32 arrays and the status word.
// per_row: 0 per tensor (PTQ), 1 per row (PSQ), 2 per-tensor range with
// per-row power-of-two steps (Sec. 4.3): s_i = s 2^e_i, shift[row] = E - e_i,
// E = min(4, 8 - bits), and s itself in tensor_scale[0].
struct ScaleOut {
  int seg;
  int bits;
  int per_row;
  float* scale;
  float* zero;
  int8_t* shift;
  float* tensor_scale;
  double* zeta;  // per_row == 2, optional: [rows] half / s_i + z_i (float64), the rows' zero-point terms
};
struct FinalizePlan {
  StatsSeg seg[3];
  int nseg;
  int row_seg;       // index of the per-row segment, -1 if none
  float* rmin;       // [rows] of the row segment
  float* rmax;
  ScaleOut out[4];
  int nout;
  int32_t* zero_i32[6];
  int64_t zero_n[6];
  int nzero;
  uint32_t* status;
};
hipError_t launch_finalize(const FinalizePlan& fp, hipStream_t s);

// Fixed-block BHQ layout, all data independent (see bhq_layout()).
struct BhqLayout {
  int64_t rows;
  int k;        // block size
  int64_t G;    // number of groups
  int64_t full; // groups of exactly k rows (first in slot order)
  int part;     // size of the one partial group after them (0: none)
  double sk_k, sk_p;        // sqrt(k), sqrt(part)
  double inv_sk_k, inv_sk_p;  // 1/sqrt(k), 1/sqrt(part) in float64 (dequantization)
  float a_k, oma_k, a_p, oma_p;  // float32(1/sqrt(size)) and float32(1 - that)
};
BhqLayout bhq_layout(int64_t rows, int k);

// Slot kind under a fixed-block layout: 0 = one-row group, 1 = full group,
// 2 = the partial group.  Groups are stored full ones first, then the
// partial one, then the one-row groups, each full / partial group starting
// at a multiple of k.
__device__ __forceinline__ int bhq_slot_kind(const BhqLayout& L, int64_t slot) {
  if (slot < L.full * L.k) return 1;
  if (L.part > 0 && slot < L.full * L.k + L.part) return 2;
  return 0;
}

// Workspace for the BHQ plan: sorted chunk keys, rank (must be zero before
// the plan runs), sigma = rows in sorted order.
size_t bhq_plan_workspace(int64_t rows);
struct BhqPlanWs {
  uint64_t* sorted;
  int32_t* rank;
  int32_t* sigma;
};
BhqPlanWs bhq_plan_carve(void* plan_ws, int64_t rows);
// fin: run this finalize step inside the first plan launch (only when the
// row ranges rmin / rmax were stored by the statistics kernel); nullptr when
// the finalize kernel already ran.
hipError_t launch_bhq_plan(const float* rmin, const float* rmax, const BhqLayout& L, int bits, void* plan_ws,
                           int32_t* perm, float* scale, float* zero, int32_t* group_off, int32_t* num_groups, const FinalizePlan* fin,
                           hipStream_t s);


// Rows in sorted order (M descending, ties by row index), for the general
// plans below; fin as for launch_bhq_plan.
hipError_t launch_bhq_sort(const float* rmin, const float* rmax, int64_t rows, void* plan_ws, int32_t* sigma,
                           const FinalizePlan* fin, hipStream_t s);

// ---- general BHQ plans: groups of any size, in slot order ----------------
// Slot record: the slot's group starts at slot `base` and has `size` slots;
// alpha = float32(1 / sqrt(size)), oma = float32(1 - alpha) (multi-row groups).
struct SlotInfo {
  int32_t base, size;
  float alpha, oma;
};
// Per sorted position r (row sigma[r]): its infinity norm M and range R
// (non-finite values read as 0, so that a plan over bad data stays a valid
// permutation), cbrt_rn(R), cbrt_rn(2 M); prefix sums P of M (float64,
// P[0] = 0, added one at a time in sorted order); the App. D objective of
// every number of groups G = 1..rows and the chosen G.
struct AppdWs {
  int32_t* sigma;
  float *Ms, *Rs, *ca, *cc;
  double* P;
  double* obj;
  int32_t* G;
};
size_t appd_workspace(int64_t rows);
AppdWs appd_carve(void* ws, int64_t rows);
// Everything of the plan after the sort: the sorted-position scalars, and
// for block_size = 0 the App. D search over G (objective into obj_out when
// given, else the workspace's), then the groups (block_size > 0: the fixed
// layout of bhq_layout).  Writes perm, scale, zero, group_off [G + 1], slot
// and num_groups (device scalar).
hipError_t launch_general_plan(const float* rmin, const float* rmax, int64_t rows, int bits, int block_size,
                               const AppdWs& w, double* obj_out, int32_t* perm, float* scale, float* zero,
                               int32_t* group_off, SlotInfo* slot, int32_t* num_groups, hipStream_t s);
// The App. D search alone (objective and chosen G), after the sort.
hipError_t launch_appd_search(const float* rmin, const float* rmax, int64_t rows, int bits, const AppdWs& w,
                              double* obj_out, int32_t* num_groups, hipStream_t s);
// Per multi-row group and column: tau = (alpha S - v_0) / (1 - alpha), S the
// group's column sum of v_p = d_p x[perm[p]] in slot order (float32),
// stored at tau[(base / 2) * cols + col] (group bases are at least 2 apart).
hipError_t launch_bhq_tau(const float* x, int64_t rows, int64_t cols, const int32_t* perm, const float* scale,
                          const SlotInfo* slot, float* tau, hipStream_t s);
// Inverse transform of the general plans' grad_X rows.  Rows of T are (block
// b, slot p) at T[(b * tstride + p) * ldt + col] (float64: the dequantized
// code row times the weights, see EPI_BHQT); per multi-row group S = sum of
// its T rows (float64, slot order), tau = (alpha S - T_0) / (1 - alpha),
// alpha = 1 / sqrt(k); out row = perm[p] * ostride + b * obstride, value
// (T_0 + (1 - alpha) tau or T_p - alpha tau) / d_p; zero where mask <= 0.
struct InverseParams {
  const double* T;
  int64_t ldt, tstride, nblk, rows, cols;
  const SlotInfo* slot;
  const int32_t* perm;
  const float* scale;
  float* out;
  int64_t ldo, ostride, obstride;
  const float* mask;
};
hipError_t launch_bhq_inverse(const InverseParams& p, hipStream_t s);

struct QuantParams {
  const float* x;
  int64_t rows, cols;
  const int32_t* perm;  // slot -> source row; nullptr = identity
  int bits;
  int stoch;
  uint64_t seed;
  uint32_t stream;
  const float* scale;  // per tensor: [1]; per row / BHQ: [rows] per slot
  const float* zero;
  int8_t* q_nat;       // [rows, cols] slot order, or nullptr (packed: [rows, cols / 2] bytes)
  int packed;          // natural codes of bits <= 4 stored two per byte (float4 rows only)
  int64_t pm_o;        // > 0: natural codes pixel-major, column j of row (slot) i at
                       // ((j / pm_o) rows + i) pm_o + j % pm_o (cols % pm_o == 0, pm_o % 4 == 0)
  int32_t* sum_nat;    // [rows] row sums, or nullptr
  int8_t* q_t;         // [cols, rows] slot order, or nullptr
  int32_t* sum_t;      // [cols] column sums, or nullptr
  // second, per-tensor stochastic quantizer of the same rows (Q_b1); transposed only
  int bits2;
  uint32_t stream2;
  const float* scale2;
  const float* zero2;
  int8_t* q2_t;
  int32_t* sum2_t;
  const int8_t* shift;   // QM_ROW: per-row left shift of the offset codes, or nullptr
  const int8_t* shift2;  // Q_b1 with per-row scale2 / zero2 / shift2 (source-row order), or nullptr
  BhqLayout L;           // BHQ: L.k = 0 selects the general plan (slot, tau)
  const SlotInfo* slot;
  const float* tau;
  // seed batch (launch_quant_seeds): nseeds roundings under keys seed + b,
  // per element [rows, cols] (slot order) the sum of the codes and of their squares
  int nseeds;
  int32_t* sum_c;
  int32_t* sum_c2;
};
enum QuantMode { QM_TENSOR = 0, QM_ROW = 1, QM_BHQ = 2 };
hipError_t launch_quant(const QuantParams& p, int mode, hipStream_t s);
// The seed batch of one quantizer (natural layout, cols % 4 == 0).
hipError_t launch_quant_seeds(const QuantParams& p, int mode, hipStream_t s);
// Two per-tensor quantizations with transposed outputs only, one launch.
hipError_t launch_quant_pair(const QuantParams& p0, const QuantParams& p1, hipStream_t s);
// The gradient quantizer pg (with its transposed second quantizer) and the
// per-tensor transposed quantizers px, pw in one launch when the shapes
// allow it, else as separate launches.
hipError_t launch_quant_fused(const QuantParams& pg, int mode, const QuantParams& px, const QuantParams& pw,
                              hipStream_t s);

// Narrow transposing per-tensor quantizer (conv activations and Q_b1 of a
// conv gradient): logical [rows, cols], row r of the output taken from source
// row perm[r / blk] * blk + r % blk; codes [cols][ldt], rows >= rows get 0.
struct NarrowQParams {
  const float* x;
  int64_t rows, cols;
  const int32_t* perm;
  int64_t blk;
  int bits;
  int stoch;
  uint64_t seed;
  uint32_t stream;
  const float* scale;
  const float* zero;
  int8_t* q_t;
  int64_t ldt;
  int64_t vblk;  // rows of each block of blk that exist in x (the rest are zero codes); 0: blk
  int rowscale;  // scale / zero per block (indexed by the block's source block), else per tensor
  // 2-D blocks (gw > 0, replaces vblk): row br of a block is (y, x) = (br / gw,
  // br % gw) of a grid with rows of gw; it exists iff y < gho and x < gwo and
  // reads source row y gwo + x of its block
  int64_t gw, gwo, gho;
};
hipError_t launch_quant_narrow_t(const NarrowQParams& p, hipStream_t s);

// ---- int8 contractions ---------------------------------------------------

enum Epilogue {
  EPI_RAW_I32 = 0,   // int32 partials [splits][M][N] (caller reduces)
  EPI_TENSOR = 1,    // per-tensor A, per-tensor B: grad_W
  EPI_ROW = 2,       // per-row A (PTQ broadcasts), per-tensor B: grad_X
  EPI_BHQ = 3,       // per-group Householder on A rows, per-tensor B: grad_X
  EPI_BHQT = 4       // general BHQ plan: one-row groups finished, other rows' T into tbuf
};

struct GemmParams {
  const int8_t* A;  // [M, K] row stride lda (bytes)
  int packedA;      // A holds codes of at most 4 bits two per byte (as the quantizer packs them), K % 16 == 0
  const int8_t* B;  // [N, K] row stride ldb
  int64_t M, N, K, lda, ldb;
  // conv B row map (bmap_c > 0, fast K loop only): row j = (tap, c) with
  // tap = (r, s) of a bmap_kw-wide kernel starts at B + (s bmap_c + c) ldb +
  // r bmap_wp (shifted activation-code grids, see ConvGeom)
  int64_t bmap_c, bmap_kw, bmap_wp;
  int64_t kchunk;   // K per split (multiple of 128 when split, <= 65536)
  int splits;
  int32_t* part;    // EPI_RAW_I32 output [splits][M][N]
  // epilogue data (float64 arithmetic, float32 result)
  float* out;       // [M, N] (row index remapped through perm when given)
  int64_t ldo;
  const int32_t* perm;   // A row (slot) -> output row; nullptr = identity
  const int32_t* sumA;   // [M] sum over K of A's codes
  const int32_t* sumB;   // [N] sum over K of B's codes
  const float* scaleA;   // [1] or [M]
  const float* zeroA;
  int rowwiseA;          // scaleA / zeroA indexed per row
  int halfA;             // 2^(bitsA - 1)
  const float* scaleB;   // [1]
  const float* zeroB;
  int halfB;
  BhqLayout L;           // EPI_BHQ group structure
  int relu;              // EPI_TENSOR: store max(v, 0)
  int expA;              // EPI_TENSOR: A's step is 1 / (scaleA[0] 2^expA)
  const double* colvec;  // EPI_TENSOR: nullptr, or [N] replacing A's zero-point terms (per-row zeros of A)
  const float* mask;     // EPI_ROW / EPI_BHQ: nullptr, or [M, ldo] in output-row order; out = 0 where mask <= 0
  const SlotInfo* slot;  // EPI_BHQT: the general plan
  double* tbuf;          // EPI_BHQT: [M, ldt] T of the rows of multi-row groups
  int64_t ldt;
};
hipError_t launch_gemm(const GemmParams& p, int epi, hipStream_t s);

// Sum int32 split partials in int64; either store int64 (out64) or apply the
// per-tensor epilogue (EPI_TENSOR) into p.out.
hipError_t launch_splitk_reduce(const GemmParams& p, int64_t* out64, int epi, hipStream_t s);

// Zero-point term of a contraction over samples whose A rows (samples) carry
// their own zero points: v[c] = sum_n zeta_n Xt[n, c] (zeta_n = half / s_n +
// z_n from the finalize), Xt[n, c] = dx q[c, n] + zx (q: [cols, rows]
// transposed codes in slot order, perm slot -> row or nullptr), float64.
struct ColvecParams {
  const int8_t* q_t;
  int64_t rows, cols;
  const int32_t* perm;
  const double* zeta;   // zeta_n [rows], source-row order
  const float* scaleX;  // [1]
  const float* zeroX;   // [1]
  int halfX;
  double* part;         // scratch [colvec_splits(rows)][cols + 1]
  double* out;          // [cols]
};
int64_t colvec_splits(int64_t rows);
hipError_t launch_colvec(const ColvecParams& p, hipStream_t s);

// ---- machine probes -------------------------------------------------------
hipError_t launch_mfma_probe(int64_t blocks, int64_t iters, int32_t* sink, hipStream_t s);
hipError_t launch_copy_probe(int64_t blocks, const void* src, void* dst, int64_t n16, hipStream_t s);

// ---- 4-bit codes on 6-bit float matrix cores ---------------------------
// Packed e3m2 operands (rows of bf6_row_bytes(K) bytes, K padded to 128),
// exact int32 partials [splits][M][N] (reduce with launch_splitk_reduce).
struct Bf6Params {
  const int8_t* A;  // [M] packed rows, stride lda bytes
  const int8_t* B;  // [N] packed rows, stride ldb bytes
  int64_t M, N, Kpad, lda, ldb;
  int64_t kchunk;   // codes per split, multiple of 128, <= 131072
  int splits;
  int32_t* part;
};
int64_t bf6_row_bytes(int64_t K);
hipError_t launch_pack_e3m2(const int8_t* src, int64_t rows, int64_t K, int64_t ld, int8_t* dst, uint32_t* status,
                            hipStream_t s);
hipError_t launch_status_clear(uint32_t* status, hipStream_t s);
hipError_t launch_gemm_bf6(const Bf6Params& p, hipStream_t s);

constexpr int NUM_XCD = 8;  // accelerator dies of the GPU, each with its own L2; blocks go to them round robin

// ---- conv ----------------------------------------------------------------
struct ConvGeom {
  int n, c, h, w, o, kh, kw, stride, pad, ho, wo;
  int64_t npad;  // slots per input pixel in the grad_X rows (multiple of 64)
  int64_t psp;   // K pitch of a slot's output pixels in the grad_W operands (ho wo, or
                 // ho wo rounded up to 128 with zero codes after them when Q_b1 is per sample;
                 // the grid's ghp gwp rounded up to 128 for the implicit form)
  // implicit grad_W (gwp > 0, stride 1): output pixel (y, x) of slot n is K
  // index n psp + y gwp + x of Q_b1 (zero codes elsewhere); the activation
  // codes sit on a zero-halo grid of ghp = h + 2 pad rows of gwp bytes (input
  // pixel (iy, ix) at (iy + pad, ix + pad)), stored kw times [s][c][ldx], copy
  // s shifted left by s bytes, so that tap (r, s) reads copy s at K offset
  // r gwp: no im2col matrix
  int64_t gwp, ghp, ldx;
};
hipError_t launch_conv_wq(const float* W, const ConvGeom& g, int bits, const float* scale, const float* zero,
                          int8_t* wq_t, int32_t* swq, hipStream_t s);
hipError_t launch_conv_im2col_w(const ConvGeom& g, const int8_t* xq_t, int8_t* bw, int64_t ldb, int32_t* xs,
                                int32_t* sumB, hipStream_t s);
hipError_t launch_conv_tapsums(const ConvGeom& g, const int8_t* q1_t, int64_t ldq, int32_t* qs, int32_t* sumA_tap,
                               int32_t* count_tap, hipStream_t s);
hipError_t launch_conv_gradw_reduce(const GemmParams& p, const ConvGeom& g, const int32_t* sumA_tap,
                                    const int32_t* count_tap, hipStream_t s);
// per-sample Q_b1 (K-blocked grad_W): slot weights dA = 1 / s, zA = z + half / s
// and their sum; float64 weighted code sums over slots and their tap
// rectangles; the weighted reduction of the per-slot int32 contractions
struct ConvPsqSums {
  double *dA, *zA, *zsum;  // [n], [n], [1]
  double *qw, *xw;         // [o][ho wo], [c][h w]
  double *WA, *WB;         // [o][taps], [(tap, c)]
};
hipError_t launch_conv_psq_sums(const ConvGeom& g, const float* scale, const float* zero, const int32_t* perm,
                                int half, const int8_t* q1_t, int64_t ldq, const int8_t* xq_t, const ConvPsqSums& ps,
                                int32_t* count_tap, hipStream_t s);
hipError_t launch_conv_gradw_psq_reduce(const GemmParams& p, const ConvGeom& g, const ConvPsqSums& ps,
                                        const int32_t* count_tap, hipStream_t s);
hipError_t launch_conv_gradx_prep(const ConvGeom& g, const int8_t* q2, const int32_t* swq, int32_t* sg, int32_t* rs,
                                  int32_t* ct,
                                  int32_t* cnt, hipStream_t s);
hipError_t launch_conv_gradx(const GemmParams& p, int epi, const ConvGeom& g, const int8_t* q2, const int32_t* rs,
                             const int32_t* ct, const int32_t* cnt, hipStream_t s);

}  // namespace fqt
