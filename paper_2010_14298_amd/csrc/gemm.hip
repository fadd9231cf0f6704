// int8 x int8 -> int32 contractions of the FQT backward on gfx950 matrix
// cores (v_mfma_i32_32x32x32_i8), with the dequantization fused in the
// epilogue (float64 arithmetic, float32 result):
//
//   grad_W = Q_b1(G)^T Q_f(X):  per-tensor x per-tensor affine codes
//   grad_X = Q_b2(G) Q_theta(W): per-row (PTQ / PSQ) or block Householder
//            rows (BHQ: diag(d)^-1 H applied to each group of rows inside
//            the tile, then rows scattered back to sample order)
//
// Both operands are K-contiguous (A [M, K], B [N, K]).  Two tile shapes:
// 256 x 128 per block with 128 x 64 per wave (large problems), and
// 128 x 128 with 64 x 64 per wave; 4 waves per block, K in steps of 64
// bytes through double-buffered LDS.  Blocks are numbered so that each of
// the 8 XCDs works on a contiguous run of output tiles (sharing A panels in
// its L2).  Exact int32 accumulation over K-chunks of at most 65536 (|q| <=
// 128, so 65536 * 2^14 < 2^31); longer K is split and the int32 partials
// are summed in int64.
#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BK = 128;          // K bytes per pipeline stage
constexpr int KCH = BK / 16;     // 16-byte chunks per row per stage
constexpr int LDS_STRIDE = 144;  // bytes per tile row in LDS: 128 + 16 (conflict-free 8- and 16-lane phases)
constexpr int NUM_XCD = 8;

template <int BM_, int BN_, int WM_, int WN_>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int WAVES_N = BN / WN;
  static constexpr int THREADS = (BM / WM) * (BN / WN) * 64;
  static constexpr int IT = WM / 32, JT = WN / 32;
  static constexpr int A_CHUNKS = BM * KCH / THREADS;  // 16-byte chunks per thread per K stage
  static constexpr int B_CHUNKS = BN * KCH / THREADS;
  static constexpr int OP_BYTES = 2 * (BM + BN) * LDS_STRIDE;
};
using CfgLarge = TileCfg<256, 128, 128, 64>;
using CfgSmall = TileCfg<128, 128, 64, 64>;

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
struct alignas(16) Chunk16 {
  uint32_t w[4];
};

// One 16-byte chunk of row r, K offset k (zero outside the matrix / K range).
__device__ __forceinline__ Chunk16 load_chunk(const int8_t* base, int64_t ld, int64_t r, int64_t nrows, int64_t k,
                                              int64_t kend, bool aligned) {
  Chunk16 c{{0u, 0u, 0u, 0u}};
  if (r >= nrows) return c;
  const int8_t* p = base + r * ld + k;
  if (aligned && k + 16 <= kend) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    c.w[0] = v.x;
    c.w[1] = v.y;
    c.w[2] = v.z;
    c.w[3] = v.w;
  } else {
#pragma unroll
    for (int b = 0; b < 16; ++b) {
      const uint32_t byte = (k + b < kend) ? (uint32_t)(uint8_t)p[b] : 0u;
      c.w[b >> 2] |= byte << (8 * (b & 3));
    }
  }
  return c;
}

// Per-row epilogue data of the grad_X contraction, staged in LDS.
struct RowStage {
  double rterm;  // zW * rowsum
  double hz;     // BHQ group row: half + c_g;  affine row: zeta = z + half / s
  double dq;     // 1 / s  (Delta for an affine row, 1 / d_p for a group row)
  int kind;      // 0 affine / one-row group, 1 full group, 2 partial group
  int orow;      // output row, -1 past M
};

template <class C, int EPI>
struct GemmLdsSize {
  static constexpr int EP_BYTES = C::BM * C::BN * 4 + C::BM * (int)sizeof(RowStage);
  static constexpr bool STAGED = (EPI == EPI_ROW || EPI == EPI_BHQ);
  static constexpr int BYTES = (STAGED && EP_BYTES > C::OP_BYTES) ? EP_BYTES : C::OP_BYTES;
};

// Bijective block -> tile map: the first 8 * floor(T / 8) blocks give each
// XCD (block id mod 8) a contiguous run of tiles; the rest map to themselves.
__device__ __forceinline__ int64_t xcd_tile(int64_t id, int64_t ntiles) {
  const int64_t q = ntiles / NUM_XCD;
  if (id < q * NUM_XCD) return (id % NUM_XCD) * q + id / NUM_XCD;
  return id;
}

// The K loop.  FAST requires 16-byte aligned rows, a K range that is a
// whole number of stages and 32-bit byte offsets; then each thread keeps
// constant offsets into a wave-uniform base pointer that advances by one
// stage per iteration (global loads in base + offset form), rows past the
// matrix edge are clamped to the last row (their outputs are never stored),
// and LDS addresses are constants: the loop carries almost no vector ALU
// work besides the matrix-core instructions.
template <class C, bool FAST>
__device__ __forceinline__ void gemm_mainloop(const GemmParams& p, int8_t* lds, int64_t m0, int64_t n0, int64_t kbeg,
                                              int64_t kend, v16i (&acc)[C::IT][C::JT]) {
  int8_t* sA = lds;                          // [2][BM * LDS_STRIDE]
  int8_t* sB = lds + 2 * C::BM * LDS_STRIDE;  // [2][BN * LDS_STRIDE]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const bool alA = ((p.lda & 15) == 0) && (((uintptr_t)p.A & 15) == 0);
  const bool alB = ((p.ldb & 15) == 0) && (((uintptr_t)p.B & 15) == 0);
  const int64_t nk = (kend - kbeg + BK - 1) / BK;

  uint32_t offA[C::A_CHUNKS], offB[C::B_CHUNKS];
  if constexpr (FAST) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      const int64_t r = (m0 + c / KCH < p.M) ? m0 + c / KCH : p.M - 1;
      offA[i] = (uint32_t)(r * p.lda) + 16u * (uint32_t)(c % KCH);
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      const int64_t r = (n0 + c / KCH < p.N) ? n0 + c / KCH : p.N - 1;
      offB[i] = (uint32_t)(r * p.ldb) + 16u * (uint32_t)(c % KCH);
    }
  }
  const int8_t* Ak = p.A + kbeg;
  const int8_t* Bk = p.B + kbeg;

  // Two register staging sets: the loads of stage t + 1 are issued one
  // iteration before the stage is stored to LDS, so each global load has two
  // iterations of matrix-core work to land.
  struct Stage {
    u32x4v a[C::A_CHUNKS];
    u32x4v b[C::B_CHUNKS];
  };
  Stage st0, st1;
  auto gload = [&](Stage& st, int64_t t) __attribute__((always_inline)) {
    if constexpr (FAST) {
      const int8_t* a = Ak + t * BK;
      const int8_t* b = Bk + t * BK;
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i) st.a[i] = *reinterpret_cast<const u32x4v*>(a + offA[i]);
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i) st.b[i] = *reinterpret_cast<const u32x4v*>(b + offB[i]);
    } else {
      const int64_t k0 = kbeg + t * BK;
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i) {
        const int c = tid + C::THREADS * i;
        const Chunk16 v = load_chunk(p.A, p.lda, m0 + c / KCH, p.M, k0 + 16 * (c % KCH), kend, alA);
        st.a[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
      }
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i) {
        const int c = tid + C::THREADS * i;
        const Chunk16 v = load_chunk(p.B, p.ldb, n0 + c / KCH, p.N, k0 + 16 * (c % KCH), kend, alB);
        st.b[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
      }
    }
  };
  auto sstore = [&](const Stage& st, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      *reinterpret_cast<u32x4v*>(&sA[buf * C::BM * LDS_STRIDE + (c / KCH) * LDS_STRIDE + 16 * (c % KCH)]) = st.a[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      *reinterpret_cast<u32x4v*>(&sB[buf * C::BN * LDS_STRIDE + (c / KCH) * LDS_STRIDE + 16 * (c % KCH)]) = st.b[i];
    }
  };
  const int lrow = lane & 31;
  const int lk = 16 * (lane >> 5);
  const int8_t* a_lane = sA + (wm * C::WM + lrow) * LDS_STRIDE + lk;
  const int8_t* b_lane = sB + (wn * C::WN + lrow) * LDS_STRIDE + lk;
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const int8_t* a_base = a_lane + buf * C::BM * LDS_STRIDE;
    const int8_t* b_base = b_lane + buf * C::BN * LDS_STRIDE;
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      v4i a[C::IT], b[C::JT];
#pragma unroll
      for (int i = 0; i < C::IT; ++i) a[i] = *reinterpret_cast<const v4i*>(a_base + i * 32 * LDS_STRIDE + kk * 32);
#pragma unroll
      for (int j = 0; j < C::JT; ++j) b[j] = *reinterpret_cast<const v4i*>(b_base + j * 32 * LDS_STRIDE + kk * 32);
#pragma unroll
      for (int i = 0; i < C::IT; ++i)
#pragma unroll
        for (int j = 0; j < C::JT; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };
  // iteration t: LDS buffer t % 2 holds stage t; the register set (t + 1) % 2
  // holds the in-flight loads of stage t + 1; stage t + 2 is loaded into the
  // set that stage t came from.
  auto iter = [&](int64_t t, int buf, Stage& next, Stage& far) __attribute__((always_inline)) {
    if (t + 2 < nk) gload(far, t + 2);
    compute(buf);
    if (t + 1 < nk) sstore(next, buf ^ 1);
    __syncthreads();
  };
  if (nk > 0) {
    gload(st0, 0);
    sstore(st0, 0);
  }
  if (nk > 1) gload(st1, 1);
  __syncthreads();
  int64_t t = 0;
  for (; t + 1 < nk; t += 2) {
    iter(t, 0, st1, st0);
    iter(t + 1, 1, st0, st1);
  }
  if (t < nk) iter(t, 0, st1, st0);
}

template <class C, int EPI, int KG, bool FAST>
__global__ __launch_bounds__(C::THREADS) void gemm_i8_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) int8_t lds[GemmLdsSize<C, EPI>::BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
  const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
  const int64_t tile = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  const int64_t m0 = (tile / tiles_n) * C::BM;
  const int64_t n0 = (tile % tiles_n) * C::BN;
  const int split = blockIdx.y;
  const int64_t kbeg = (int64_t)split * p.kchunk;
  const int64_t kend = (kbeg + p.kchunk < p.K) ? kbeg + p.kchunk : p.K;
  const int lrow = lane & 31;

  v16i acc[C::IT][C::JT];
#pragma unroll
  for (int i = 0; i < C::IT; ++i)
#pragma unroll
    for (int j = 0; j < C::JT; ++j) acc[i][j] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  gemm_mainloop<C, FAST>(p, lds, m0, n0, kbeg, kend, acc);

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
    const double dA = 1.0 / (double)p.scaleA[0];
    const double zA = (double)p.zeroA[0] + (double)p.halfA * dA;
    const double dB = 1.0 / (double)p.scaleB[0];
    const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
    const double kzz = (double)p.K * zA * zB;
    const double dAB = dA * dB;
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (row >= p.M) continue;
        const double rterm = dA * zB * (double)p.sumA[row] + kzz;
#pragma unroll
        for (int j = 0; j < C::JT; ++j) {
          const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
          if (col < p.N)
            p.out[row * p.ldo + col] =
                (float)(dAB * (double)acc[i][j][r] + rterm + zA * dB * (double)p.sumB[col]);
        }
      }
  } else {
    // grad_X: per-tensor B (weights), per-row or per-group A (gradient).
    // Stage the accumulators and per-row data in LDS (the operand tiles are
    // dead after the loop), then thread t owns column t % BN and a run of
    // consecutive rows: group sums are sequential in one thread.
    int32_t* sacc = reinterpret_cast<int32_t*>(lds);                               // [BM][BN]
    RowStage* srow = reinterpret_cast<RowStage*>(lds + C::BM * C::BN * 4);        // [BM]
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
        q.kind = (EPI == EPI_BHQ) ? bhq_slot_kind(p.L, row) : 0;
        q.rterm = zW * (double)p.sumA[row];
        q.dq = 1.0 / (double)s;
        q.hz = q.kind != 0 ? (double)p.halfA + (double)z : (double)z + (double)p.halfA * q.dq;
        q.orow = p.perm ? p.perm[row] : (int)row;
      } else {
        q.orow = -1;
      }
      srow[rr] = q;
    }
    __syncthreads();
    constexpr int RUNS = C::THREADS / C::BN;      // row runs per column
    constexpr int RUN = C::BM / RUNS;             // rows per run (multiple of 64)
    const int c = tid % C::BN;
    const int rbase = (tid / C::BN) * RUN;
    const int64_t col = n0 + c;
    if (col >= p.N) return;
    // sum over K of the dequantized weight column: dW * sum q_W + K zW
    const double colterm = dW * (double)p.sumB[col] + (double)p.K * zW;
    if constexpr (EPI == EPI_BHQ && KG > 1) {
      for (int g0 = rbase; g0 < rbase + RUN; g0 += KG) {
        // T_p = (code_p + c_g) . W~ ; S = sum over the group's multi-row slots
        double S = 0.0, T0 = 0.0;
        for (int t = 0; t < KG; ++t) {
          const RowStage& q = srow[g0 + t];
          const double T = dW * (double)sacc[(g0 + t) * C::BN + c] + (q.rterm + q.hz * colterm);
          if (q.kind != 0) S += T;
          if (t == 0) T0 = T;
        }
        const int gkind = srow[g0].kind;
        const double alpha = gkind == 2 ? p.L.inv_sk_p : p.L.inv_sk_k;
        const double tau = (alpha * S - T0) / (1.0 - alpha);
        for (int t = 0; t < KG; ++t) {
          const RowStage& q = srow[g0 + t];
          if (q.orow < 0) continue;
          const double a = (double)sacc[(g0 + t) * C::BN + c];
          double v;
          if (q.kind != 0) {
            const double T = dW * a + (q.rterm + q.hz * colterm);
            const double Z = (t == 0) ? T + (1.0 - alpha) * tau : T - alpha * tau;
            v = Z * q.dq;
          } else {
            v = q.dq * (dW * a + q.rterm) + q.hz * colterm;
          }
          p.out[(int64_t)q.orow * p.ldo + col] = (float)v;
        }
      }
    } else {
      for (int t = rbase; t < rbase + RUN; ++t) {
        const RowStage& q = srow[t];
        if (q.orow < 0) continue;
        const double a = (double)sacc[t * C::BN + c];
        p.out[(int64_t)q.orow * p.ldo + col] = (float)(q.dq * (dW * a + q.rterm) + q.hz * colterm);
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
  const double dA = 1.0 / (double)p.scaleA[0];
  const double zA = (double)p.zeroA[0] + (double)p.halfA * dA;
  const double dB = 1.0 / (double)p.scaleB[0];
  const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
  const double v = dA * dB * (double)sum + dA * zB * (double)p.sumA[row] + zA * dB * (double)p.sumB[col] +
                   (double)p.K * zA * zB;
  p.out[row * p.ldo + col] = (float)v;
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
  // fast K loop: aligned rows, whole stages per split, 32-bit offsets
  const bool whole = (p.kchunk % BK == 0) && (p.K % BK == 0);
  const bool fast = ((p.lda & 15) == 0) && ((p.ldb & 15) == 0) && (((uintptr_t)p.A & 15) == 0) &&
                    (((uintptr_t)p.B & 15) == 0) && whole && (p.M * p.lda < ((int64_t)1 << 32)) &&
                    (p.N * p.ldb < ((int64_t)1 << 32));
  const dim3 grid((unsigned)tiles, (unsigned)p.splits);
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
  return gemm_use_large(p.M, p.N) ? launch_gemm_c<CfgLarge>(p, epi, s) : launch_gemm_c<CfgSmall>(p, epi, s);
}

}  // namespace fqt
