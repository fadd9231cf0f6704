// int8 x int8 -> int32 contractions of the FQT backward on gfx950 matrix
// cores (v_mfma_i32_32x32x32_i8), with the dequantization fused in the
// epilogue (float64 arithmetic, float32 result):
//
//   grad_W = Q_b1(G)^T Q_f(X):  per-tensor x per-tensor affine codes
//   grad_X = Q_b2(G) Q_theta(W): per-row (PTQ / PSQ) or block Householder
//            rows (BHQ: diag(d)^-1 H applied to each group of rows inside
//            the tile, then rows scattered back to sample order)
//
// Both operands are K-contiguous (A [M, K], B [N, K]).  Three tile shapes
// of 8 waves (gemm_core.h): 256 x 128 per block with 64 x 64 per wave and
// three stage buffers (problems with at least 256 such tiles), 128 x 128
// with 32 x 64 per wave and four buffers, and 64 x 128 for at most 64 rows.
// The K loop moves 128-byte stages straight from HBM into LDS
// (global_load_lds); a register-staged loop serves unaligned operands and
// packed 4-bit A codes.  Blocks are numbered so that each of the 8 XCDs
// works on a contiguous run of output tiles (sharing A panels in its L2);
// split-K launches keep every tile of a split on one XCD.  Exact int32
// accumulation over K-chunks of at most 65536 (|q| <= 128, so 65536 * 2^14 <
// 2^31); longer K is split and the int32 partials are summed in int64.
#include "gemm_core.h"

namespace fqt {

// Per-row epilogue data of the grad_X contraction, staged in LDS.
struct RowStage {
  double rterm;  // zW * rowsum
  double hz;     // BHQ group row: half + c_g;  affine row: zeta = z + half / s
  double dq;     // 1 / s  (Delta for an affine row, 1 / d_p for a group row)
  int64_t obase; // output row * ldo (EPI_BHQT group row: slot * ldt into tbuf), -1 past M
  int trow;      // EPI_BHQT: the row belongs to a multi-row group (its T goes to tbuf)
};
// Per 64-row run and group of the BHQ epilogue: rows of the group that take
// part in the Householder sum (full group: KG, partial group: its size, one-row
// groups: 0) and the float64 sum of their rterm.
struct GroupStage {
  double rsum;
  int m;
  int kind;
};

// grad_X store; with a mask (the layer input X, for the ReLU that produced
// it) entries where the mask is not positive are zero.
__device__ __forceinline__ void store_masked(const GemmParams& p, int64_t idx, double v) {
  const float f = (float)v;
  p.out[idx] = (p.mask && !(p.mask[idx] > 0.0f)) ? 0.0f : f;
}

template <class C, int EPI>
struct GemmLdsSize {
  static constexpr int EP_BYTES = C::BM * C::BN * 4 + C::BM * (int)sizeof(RowStage) + C::BM * (int)sizeof(GroupStage);
  static constexpr bool STAGED = (EPI == EPI_ROW || EPI == EPI_BHQ || EPI == EPI_BHQT);
  static constexpr int BYTES = (STAGED && EP_BYTES > C::OP_BYTES) ? EP_BYTES : C::OP_BYTES;
};

template <class C, int EPI, int KG, bool FAST, bool PK = false>
__global__ __launch_bounds__(C::THREADS) void gemm_i8_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) int8_t lds[GemmLdsSize<C, EPI>::BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
  const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
  int64_t tile;
  int split;
  if (p.splits > 1 && p.splits % NUM_XCD == 0) {
    // split-K: blocks go to the XCDs round robin in launch order; give one
    // XCD every tile of its splits, so that the tiles sharing a split's A
    // panel (and, for the conv taps, overlapping B rows) meet in its L2
    const int64_t T = tiles_m * tiles_n;
    const int64_t L = (int64_t)blockIdx.x + (int64_t)gridDim.x * blockIdx.y;
    const int64_t j = L / NUM_XCD;
    tile = j % T;
    split = (int)(L % NUM_XCD + NUM_XCD * (j / T));
  } else {
    tile = xcd_tile(blockIdx.x, tiles_m * tiles_n);
    split = blockIdx.y;
  }
  const int64_t m0 = (tile / tiles_n) * C::BM;
  const int64_t n0 = (tile % tiles_n) * C::BN;
  const int64_t kbeg = (int64_t)split * p.kchunk;
  const int64_t kend = (kbeg + p.kchunk < p.K) ? kbeg + p.kchunk : p.K;
  const int lrow = lane & 31;

  v16i acc[C::IT][C::JT];
#pragma unroll
  for (int i = 0; i < C::IT; ++i)
#pragma unroll
    for (int j = 0; j < C::JT; ++j) acc[i][j] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  if constexpr (PK) {
    // packed A: the register-staged loop, unpacking in the loader
    const bool alB = ((p.ldb & 15) == 0) && (((uintptr_t)p.B & 15) == 0);
    generic_mainloop<C>(p, PackedALoader{p.A, p.lda, p.M, kend}, PlainBLoader{p.B, p.ldb, p.N, kend, alB}, lds, m0,
                        n0, kbeg, kend, acc);
  } else {
    const PlainALoader aload{p.A, p.lda, p.M, kend, ((p.lda & 15) == 0) && (((uintptr_t)p.A & 15) == 0)};
    gemm_mainloop<C, FAST>(p, aload, lds, m0, n0, kbeg, kend, acc);
  }

  // ---- epilogue.  Accumulator (i, j, r) of lane l holds
  //   row = wm*WM + i*32 + 8*(r/4) + 4*(l/32) + r%4,  col = wn*WN + j*32 + l%32
  const int h = lane >> 5;
  if constexpr (EPI == EPI_RAW_I32) {
    int32_t* out = p.part + (int64_t)split * p.M * p.N;
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int j = 0; j < C::JT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
          if (row < p.M && col < p.N) out[row * p.N + col] = acc[i][j][r];
        }
  } else if constexpr (EPI == EPI_TENSOR) {
    // with a column vector, A's rows carry their own zero points: their
    // terms sum_k zeta_k B~[k, col] arrive precomputed per column
    const double dA = ldexp(1.0 / (double)p.scaleA[0], -p.expA);
    const double zA = p.colvec ? 0.0 : (double)p.zeroA[0] + (double)p.halfA * dA;
    const double dB = 1.0 / (double)p.scaleB[0];
    const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
    const double kzz = (double)p.K * zA * zB;
    const double dAB = dA * dB;
    // all code sums are loaded before the first store (for the compiler the
    // stores could alias them, which would serialize one load per row)
    int32_t sa[C::IT][16], sb[C::JT];
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        sa[i][r] = row < p.M ? p.sumA[row] : 0;
      }
#pragma unroll
    for (int j = 0; j < C::JT; ++j) {
      const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
      sb[j] = col < p.N ? p.sumB[col] : 0;
    }
    double cterm[C::JT];
#pragma unroll
    for (int j = 0; j < C::JT; ++j) {
      const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
      cterm[j] = p.colvec ? (col < p.N ? p.colvec[col] : 0.0) : zA * dB * (double)sb[j];
    }
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (row >= p.M) continue;
        const double rterm = dA * zB * (double)sa[i][r] + kzz;
#pragma unroll
        for (int j = 0; j < C::JT; ++j) {
          const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
          if (col < p.N) {
            const float v = (float)(dAB * (double)acc[i][j][r] + rterm + cterm[j]);
            p.out[row * p.ldo + col] = (p.relu && !(v > 0.0f)) ? 0.0f : v;
          }
        }
      }
  } else {
    // grad_X: per-tensor B (weights), per-row or per-group A (gradient).
    // Stage the accumulators and per-row data in LDS (the operand tiles are
    // dead after the loop), then thread t owns column t % BN and a run of
    // consecutive rows: group sums are sequential in one thread.
    int32_t* sacc = reinterpret_cast<int32_t*>(lds);                                   // [BM][BN]
    RowStage* srow = reinterpret_cast<RowStage*>(lds + C::BM * C::BN * 4);            // [BM]
    GroupStage* sgrp = reinterpret_cast<GroupStage*>(srow + C::BM);                   // [BM / KG]
    const double dW = 1.0 / (double)p.scaleB[0];
    const double zW = (double)p.zeroB[0] + (double)p.halfB * dW;
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int j = 0; j < C::JT; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sacc[(wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3)) * C::BN + wn * C::WN + j * 32 + lrow] =
              acc[i][j][r];
    for (int rr = tid; rr < C::BM; rr += C::THREADS) {
      const int64_t row = m0 + rr;
      RowStage q{};
      if (row < p.M) {
        const float s = p.rowwiseA ? p.scaleA[row] : p.scaleA[0];
        const float z = p.rowwiseA ? p.zeroA[row] : p.zeroA[0];
        const int kind = (EPI == EPI_BHQ) ? bhq_slot_kind(p.L, row) : (EPI == EPI_BHQT ? (p.slot[row].size > 1) : 0);
        q.rterm = zW * (double)p.sumA[row];
        q.dq = 1.0 / (double)s;
        q.hz = kind != 0 ? (double)p.halfA + (double)z : (double)z + (double)p.halfA * q.dq;
        q.obase = (int64_t)(p.perm ? p.perm[row] : (int)row) * p.ldo;
        if (EPI == EPI_BHQT && kind != 0) {
          q.trow = 1;
          q.obase = row * p.ldt;
        }
      } else {
        q.obase = -1;
      }
      srow[rr] = q;
    }
    static_assert(C::BM % 64 == 0 && KG <= 64, "64-row epilogue runs");
    if constexpr (EPI == EPI_BHQ && KG > 1) {
      __syncthreads();
      // per group: Householder rows (they come first in the group) and their rterm sum
      for (int gi = tid; gi < C::BM / KG; gi += C::THREADS) {
        const int64_t g0 = m0 + (int64_t)gi * KG;
        GroupStage gs{0.0, 0, 0};
        if (g0 < p.M) {
          gs.kind = bhq_slot_kind(p.L, g0);
          if (gs.kind != 0) {
            gs.m = gs.kind == 1 ? KG : p.L.part;
            for (int t = 0; t < gs.m; ++t) gs.rsum += srow[gi * KG + t].rterm;
          }
        }
        sgrp[gi] = gs;
      }
    }
    __syncthreads();
    // Wave w takes the (64-row run, 64-column half) units w, w + WAVES, ...;
    // lane l holds the four columns 4 (l % 16) .. +3 of the half and rows
    // 4 i + l / 16 of the run, so one step covers four rows with 16-byte
    // loads and stores.  A BHQ group of KG rows (KG <= 64, aligned) lies
    // inside its run; its accumulator column sums meet across the row lanes
    // (the lanes that share the columns) by xor shuffles.
    constexpr int NRUN = C::BM / 64, NHALF = C::BN / 64;
    const int cq = lane & 15, rsub = lane >> 4;
    const bool al = (p.ldo & 3) == 0 && (((uintptr_t)p.out | (uintptr_t)p.mask) & 15) == 0;
    for (int u = wave; u < NRUN * NHALF; u += C::WAVES) {
      const int rbase = (u / NHALF) * 64;
      const int cb = (u % NHALF) * 64 + 4 * cq;  // tile column of this lane's first column
      const int64_t col = n0 + cb;
      if (col >= p.N) continue;  // the shuffle partners share the columns
      const bool vec = al && col + 3 < p.N;
      // sum over K of the dequantized weight column: dW * sum q_W + K zW
      double colterm[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) colterm[e] = col + e < p.N ? dW * (double)p.sumB[col + e] + (double)p.K * zW : 0.0;
      auto row_acc = [&](int row, double (&a)[4]) {
        const int4 v = *reinterpret_cast<const int4*>(&sacc[row * C::BN + cb]);
        a[0] = (double)v.x;
        a[1] = (double)v.y;
        a[2] = (double)v.z;
        a[3] = (double)v.w;
      };
      auto put = [&](int64_t obase, const double (&v)[4]) {
        const int64_t idx = obase + col;
        if (vec) {
          float4 f = make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
          if (p.mask) {
            const float4 m = *reinterpret_cast<const float4*>(p.mask + idx);
            f.x = m.x > 0.0f ? f.x : 0.0f;
            f.y = m.y > 0.0f ? f.y : 0.0f;
            f.z = m.z > 0.0f ? f.z : 0.0f;
            f.w = m.w > 0.0f ? f.w : 0.0f;
          }
          *reinterpret_cast<float4*>(p.out + idx) = f;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < p.N) store_masked(p, idx + e, v[e]);
        }
      };
      if constexpr (EPI == EPI_BHQ && KG > 1) {
        constexpr int RB = KG > 4 ? KG : 4;  // rows per block of steps: one group, or 4 / KG groups
        for (int blk = rbase; blk < rbase + 64; blk += RB) {
          const int g0 = (blk + rsub) & ~(KG - 1);  // first row of this lane's group
          const GroupStage gs = sgrp[g0 / KG];
          // Row t of a group: T_t = (code_t + c_g) . W~ = dW a_t + rterm_t + hz colterm;
          // the Householder sum S = sum of T_t over its m rows, with the
          // accumulators summed exactly (integers below 2^53 in float64)
          double asum[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
          for (int i = 0; i < RB / 4; ++i) {
            const int row = blk + 4 * i + rsub;
            if (row - g0 < gs.m) {
              double a[4];
              row_acc(row, a);
#pragma unroll
              for (int e = 0; e < 4; ++e) asum[e] += a[e];
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            asum[e] += __shfl_xor(asum[e], 16);
            if constexpr (KG >= 4) asum[e] += __shfl_xor(asum[e], 32);
          }
          const double hz = srow[g0].hz;
          double up0[4] = {0.0, 0.0, 0.0, 0.0}, dn[4] = {0.0, 0.0, 0.0, 0.0};
          if (gs.m > 0) {
            double a0[4];
            row_acc(g0, a0);
            const double alpha = gs.kind == 2 ? p.L.inv_sk_p : p.L.inv_sk_k;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const double S = dW * asum[e] + (gs.rsum + (double)gs.m * (hz * colterm[e]));
              const double T0 = dW * a0[e] + (srow[g0].rterm + hz * colterm[e]);
              const double tau = (alpha * S - T0) / (1.0 - alpha);
              up0[e] = (1.0 - alpha) * tau;
              dn[e] = alpha * tau;
            }
          }
#pragma unroll
          for (int i = 0; i < RB / 4; ++i) {
            const int row = blk + 4 * i + rsub;
            const RowStage q = srow[row];
            if (q.obase < 0) continue;
            const int t = row - g0;
            double a[4], v[4];
            row_acc(row, a);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              if (t < gs.m) {
                const double T = dW * a[e] + (q.rterm + q.hz * colterm[e]);
                v[e] = (t == 0 ? T + up0[e] : T - dn[e]) * q.dq;
              } else {
                v[e] = q.dq * (dW * a[e] + q.rterm) + q.hz * colterm[e];
              }
            }
            put(q.obase, v);
          }
        }
      } else {
#pragma unroll 4
        for (int i = 0; i < 16; ++i) {
          const int row = rbase + 4 * i + rsub;
          const RowStage q = srow[row];
          if (q.obase < 0) continue;
          double a[4], v[4];
          row_acc(row, a);
          if (EPI == EPI_BHQT && q.trow) {
            double* dst = p.tbuf + q.obase + col;
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (col + e < p.N) dst[e] = dW * a[e] + (q.rterm + q.hz * colterm[e]);
            continue;
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = q.dq * (dW * a[e] + q.rterm) + q.hz * colterm[e];
          put(q.obase, v);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// split-K reduction: int32 partials -> int64 sum -> raw or per-tensor epilogue
// ---------------------------------------------------------------------------
__global__ void splitk_reduce_kernel(GemmParams p, int64_t* out64, int epi) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t MN = p.M * p.N;
  if (idx >= MN) return;
  int64_t sum = 0;
  for (int s = 0; s < p.splits; ++s) sum += (int64_t)p.part[(int64_t)s * MN + idx];
  if (epi == EPI_RAW_I32) {
    out64[idx] = sum;
    return;
  }
  const int64_t row = idx / p.N, col = idx % p.N;
  const double dA = ldexp(1.0 / (double)p.scaleA[0], -p.expA);
  const double zA = p.colvec ? 0.0 : (double)p.zeroA[0] + (double)p.halfA * dA;
  const double dB = 1.0 / (double)p.scaleB[0];
  const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
  const double cterm = p.colvec ? p.colvec[col] : zA * dB * (double)p.sumB[col];
  const double v = dA * dB * (double)sum + dA * zB * (double)p.sumA[row] + cterm + (double)p.K * zA * zB;
  const float f = (float)v;
  p.out[row * p.ldo + col] = (p.relu && !(f > 0.0f)) ? 0.0f : f;
}

// ---------------------------------------------------------------------------
// zero-point column vector, float64: v[c] = sum_n zeta_row(n) (dx q[c, n] + zx),
// in two deterministic launches.  Partials: block (x, y) takes COLVEC_C
// columns (COLVEC_C / 4 per wave) and samples [y COLVEC_N, (y + 1) COLVEC_N),
// 16 consecutive per lane (one 16-byte load per column row); the wave sums
// its lanes and stores part[y][c] (and the zeta sum in part[y][cols], from
// x = 0).  The reduce adds the partials of each column in order of y.
// ---------------------------------------------------------------------------
constexpr int COLVEC_C = 64;
constexpr int COLVEC_N = 1024;

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void colvec_partial_kernel(ColvecParams p) {
  constexpr int CW = COLVEC_C / 4;  // columns per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t cw = (int64_t)blockIdx.x * COLVEC_C + wave * CW;
  const int64_t n0 = (int64_t)blockIdx.y * COLVEC_N + 16 * lane;
  const bool full = n0 + 16 <= p.rows && (p.rows & 15) == 0;
  double z[16], zs = 0.0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int64_t n = n0 + k;
    z[k] = n < p.rows ? p.zeta[p.perm ? p.perm[n] : (int32_t)n] : 0.0;
    zs += z[k];
  }
  double* part = p.part + (int64_t)blockIdx.y * (p.cols + 1);
  // every column's 16 codes first (independent loads in flight together)
  uint4 v[CW];
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    const int64_t col = cw + c;
    const int8_t* q = p.q_t + col * p.rows + n0;
    if (col >= p.cols) {
      v[c] = make_uint4(0u, 0u, 0u, 0u);
    } else if (full) {
      v[c] = *reinterpret_cast<const uint4*>(q);
    } else {
      uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int k = 0; k < 16; ++k)
        if (n0 + k < p.rows) w[k >> 2] |= (uint32_t)(uint8_t)q[k] << (8 * (k & 3));
      v[c] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
#pragma unroll
  for (int c = 0; c < CW; ++c) {
    const uint32_t w[4] = {v[c].x, v[c].y, v[c].z, v[c].w};
    double acc = 0.0;
#pragma unroll
    for (int k = 0; k < 16; ++k) acc += z[k] * (double)(int8_t)((w[k >> 2] >> (8 * (k & 3))) & 255u);
    acc = wave_sum_f64(acc);
    if (lane == 0 && cw + c < p.cols) part[cw + c] = acc;
  }
  if (blockIdx.x == 0 && wave == 0) {
    zs = wave_sum_f64(zs);
    if (lane == 0) part[p.cols] = zs;
  }
}

__global__ __launch_bounds__(256) void colvec_reduce_kernel(ColvecParams p, int64_t nsplit) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= p.cols) return;
  double a = 0.0, zs = 0.0;
  for (int64_t y = 0; y < nsplit; ++y) {
    a += p.part[y * (p.cols + 1) + c];
    zs += p.part[y * (p.cols + 1) + p.cols];
  }
  const double dx = 1.0 / (double)p.scaleX[0];
  const double zx = (double)p.zeroX[0] + (double)p.halfX * dx;
  p.out[c] = dx * a + zx * zs;
}

int64_t colvec_splits(int64_t rows) { return (rows + COLVEC_N - 1) / COLVEC_N; }

hipError_t launch_colvec(const ColvecParams& p, hipStream_t s) {
  const int64_t cb = (p.cols + COLVEC_C - 1) / COLVEC_C, ns = colvec_splits(p.rows);
  if (p.cols < 1 || p.rows < 1 || cb > 0x7FFFFFFF || ns > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(colvec_partial_kernel, dim3((unsigned)cb, (unsigned)ns), dim3(256), 0, s, p);
  hipLaunchKernelGGL(colvec_reduce_kernel, dim3((unsigned)((p.cols + 255) / 256)), dim3(256), 0, s, p, ns);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce(const GemmParams& p, int64_t* out64, int epi, hipStream_t s) {
  const int64_t MN = p.M * p.N;
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, p, out64, epi);
  return hipGetLastError();
}

template <class C>
int64_t gemm_tiles(int64_t M, int64_t N) {
  return ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
}

// Large tiles when they still give every CU a block; small ones otherwise.
static bool gemm_use_large(int64_t M, int64_t N) { return gemm_tiles<CfgLarge>(M, N) >= 256; }

template <class C, int EPI, int KG>
static hipError_t launch_gemm_t(GemmParams p, hipStream_t s) {
  const int64_t tiles = gemm_tiles<C>(p.M, p.N);
  if (tiles > 0x7FFFFFFF || p.splits > 65535) return hipErrorInvalidValue;
  // fast K loop: aligned rows, whole stages per split
  const bool whole = (p.kchunk % C::BK == 0) && (p.K % C::BK == 0);
  const bool fast = ((p.lda & 15) == 0) && ((p.ldb & 15) == 0) && (((uintptr_t)p.A & 15) == 0) &&
                    (((uintptr_t)p.B & 15) == 0) && whole;
  const dim3 grid((unsigned)tiles, (unsigned)p.splits);
  if constexpr (EPI == EPI_ROW || EPI == EPI_BHQ || EPI == EPI_BHQT) {
    if (p.packedA) {
      if (p.K % 16 != 0 || (p.lda & 7) != 0 || ((uintptr_t)p.A & 7) != 0) return hipErrorInvalidValue;
      hipLaunchKernelGGL((gemm_i8_kernel<C, EPI, KG, false, true>), grid, dim3(C::THREADS), 0, s, p);
      return hipGetLastError();
    }
  }
  if (p.packedA) return hipErrorInvalidValue;
  if (p.bmap_c > 0 && (!fast || (p.bmap_wp & 15) != 0)) return hipErrorInvalidValue;  // mapped rows: fast loop only
  if (fast)
    hipLaunchKernelGGL((gemm_i8_kernel<C, EPI, KG, true>), grid, dim3(C::THREADS), 0, s, p);
  else
    hipLaunchKernelGGL((gemm_i8_kernel<C, EPI, KG, false>), grid, dim3(C::THREADS), 0, s, p);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_gemm_c(const GemmParams& p, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_RAW_I32: return launch_gemm_t<C, EPI_RAW_I32, 0>(p, s);
    case EPI_TENSOR: return launch_gemm_t<C, EPI_TENSOR, 0>(p, s);
    case EPI_ROW: return launch_gemm_t<C, EPI_ROW, 0>(p, s);
    case EPI_BHQT: return p.slot && p.tbuf ? launch_gemm_t<C, EPI_BHQT, 0>(p, s) : hipErrorInvalidValue;
    case EPI_BHQ:
      switch (p.L.k) {
        case 1: return launch_gemm_t<C, EPI_BHQ, 1>(p, s);
        case 2: return launch_gemm_t<C, EPI_BHQ, 2>(p, s);
        case 4: return launch_gemm_t<C, EPI_BHQ, 4>(p, s);
        case 8: return launch_gemm_t<C, EPI_BHQ, 8>(p, s);
        case 16: return launch_gemm_t<C, EPI_BHQ, 16>(p, s);
        case 32: return launch_gemm_t<C, EPI_BHQ, 32>(p, s);
        case 64: return launch_gemm_t<C, EPI_BHQ, 64>(p, s);
        default: return hipErrorInvalidValue;
      }
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(const GemmParams& p, int epi, hipStream_t s) {
  if (p.M <= 64 && epi == EPI_RAW_I32) return launch_gemm_t<CfgNarrow, EPI_RAW_I32, 0>(p, s);
  return gemm_use_large(p.M, p.N) ? launch_gemm_c<CfgLarge>(p, epi, s) : launch_gemm_c<CfgSmall>(p, epi, s);
}

}  // namespace fqt

namespace fqt {

// ---------------------------------------------------------------------------
// machine probes for the measured peaks: a register-only int8 matrix-core
// loop (four independent accumulators per wave, so the instructions issue
// back to back) and a streaming 16-byte copy
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void mfma_probe_kernel(int64_t iters, int32_t* sink) {
  const int lane = threadIdx.x & 63;
  v4i a = {lane, lane + 1, lane + 2, lane + 3};
  v4i b = {lane ^ 5, lane ^ 6, lane ^ 7, lane ^ 9};
  v16i acc[4];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[u][r] = 0;
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[u] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[u], 0, 0, 0);
  }
  int32_t x = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) x ^= acc[u][r];
  if (x == 0x7FFFFFFF) sink[0] = x;  // keeps the loop; practically never stores
}

__global__ __launch_bounds__(256) void copy_probe_kernel(const uint4* src, uint4* dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

hipError_t launch_mfma_probe(int64_t blocks, int64_t iters, int32_t* sink, hipStream_t s) {
  hipLaunchKernelGGL(mfma_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, s, iters, sink);
  return hipGetLastError();
}

hipError_t launch_copy_probe(int64_t blocks, const void* src, void* dst, int64_t n16, hipStream_t s) {
  hipLaunchKernelGGL(copy_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<const uint4*>(src),
                     static_cast<uint4*>(dst), n16);
  return hipGetLastError();
}

}  // namespace fqt
