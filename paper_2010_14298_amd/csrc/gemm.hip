// int8 x int8 -> int32 contractions of the FQT backward on gfx950 matrix
// cores (v_mfma_i32_32x32x32_i8), with the dequantization fused in the
// epilogue (float64 arithmetic, float32 result):
//
//   grad_W = Q_b1(G)^T Q_f(X):  per-tensor x per-tensor affine codes
//   grad_X = Q_b2(G) Q_theta(W): per-row (PTQ / PSQ) or block Householder
//            rows (BHQ: diag(d)^-1 H applied to each group of rows inside
//            the tile, then rows scattered back to sample order)
//
// Both operands are K-contiguous ("A [M, K], B [N, K]").  A 128 x 128 tile
// per 256-thread block (2 x 2 waves of 64 x 64), K in steps of 64 bytes,
// double-buffered LDS.  Exact int32 accumulation over K-chunks of at most
// 65536 (|q| <= 128, so 65536 * 2^14 < 2^31); longer K is split and the
// int32 partials are summed in int64.
#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = 80;  // bytes per tile row in LDS: 64 + 16 (no bank conflicts on 16-lane phases)

struct alignas(16) Chunk16 {
  uint32_t w[4];
};

// Load one 16-byte chunk of row `r` (global row index), K offset `k`.
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

// LDS: the double-buffered operand tiles during the K loop; afterwards the
// int32 accumulator tile and per-row epilogue data of the grad_X epilogue.
struct RowStage {
  double rterm;  // zW * rowsum (+ nothing else): row part of (code + c) . W~ / (Delta q + zeta) . W~
  double hz;     // BHQ group row: half + c_g;  affine row: zeta = z + half / s
  double dq;     // affine row: Delta = 1 / s
  double inv_d;  // BHQ group row: 1 / d_p
  int kind;      // 0 affine / one-row group, 1 full group, 2 partial group
  int orow;      // output row, -1 past M
};
struct OperandTiles {
  int8_t a[2][BM * LDS_STRIDE];
  int8_t b[2][BN * LDS_STRIDE];
};
struct EpilogueTiles {
  int32_t acc[BM][BN];
  RowStage rows[BM];
};
union __attribute__((aligned(16))) GemmLds {
  OperandTiles op;
  EpilogueTiles ep;
};

template <int EPI, int KG>
__global__ __launch_bounds__(256) void gemm_i8_kernel(GemmParams p) {
  __shared__ GemmLds lds;
  int8_t(*sA)[BM * LDS_STRIDE] = lds.op.a;
  int8_t(*sB)[BN * LDS_STRIDE] = lds.op.b;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  const int64_t n0 = (int64_t)blockIdx.x * BN;
  const int split = blockIdx.z;
  const int64_t kbeg = (int64_t)split * p.kchunk;
  const int64_t kend = (kbeg + p.kchunk < p.K) ? kbeg + p.kchunk : p.K;
  const bool alA = ((p.lda & 15) == 0) && (((uintptr_t)p.A & 15) == 0);
  const bool alB = ((p.ldb & 15) == 0) && (((uintptr_t)p.B & 15) == 0);

  // global -> register staging: 2 chunks of A and 2 of B per thread
  Chunk16 ra[2], rb[2];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + 256 * i;
      const int row = c >> 2, kc = c & 3;
      ra[i] = load_chunk(p.A, p.lda, m0 + row, p.M, k0 + 16 * kc, kend, alA);
      rb[i] = load_chunk(p.B, p.ldb, n0 + row, p.N, k0 + 16 * kc, kend, alB);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + 256 * i;
      const int row = c >> 2, kc = c & 3;
      *reinterpret_cast<Chunk16*>(&sA[buf][row * LDS_STRIDE + 16 * kc]) = ra[i];
      *reinterpret_cast<Chunk16*>(&sB[buf][row * LDS_STRIDE + 16 * kc]) = rb[i];
    }
  };

  v16i acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};

  const int64_t nk = (kend - kbeg + BK - 1) / BK;
  if (nk > 0) {
    gload(kbeg);
    sstore(0);
  }
  __syncthreads();
  const int lrow = lane & 31;
  const int lk = 16 * (lane >> 5);
  for (int64_t t = 0; t < nk; ++t) {
    const int buf = (int)(t & 1);
    if (t + 1 < nk) gload(kbeg + (t + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      v4i a[2], b[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        a[i] = *reinterpret_cast<const v4i*>(&sA[buf][(wm * 64 + i * 32 + lrow) * LDS_STRIDE + kk * 32 + lk]);
        b[i] = *reinterpret_cast<const v4i*>(&sB[buf][(wn * 64 + i * 32 + lrow) * LDS_STRIDE + kk * 32 + lk]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (t + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue.  Accumulator (i, j, r) of lane l holds
  //   row = wm*64 + i*32 + 8*(r/4) + 4*(l/32) + r%4,  col = wn*64 + j*32 + l%32
  const int h = lane >> 5;
  if constexpr (EPI == EPI_RAW_I32) {
    int32_t* out = p.part + (int64_t)split * p.M * p.N;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          const int64_t col = n0 + wn * 64 + j * 32 + lrow;
          if (row < p.M && col < p.N) out[row * p.N + col] = acc[i][j][r];
        }
    return;
  } else if constexpr (EPI == EPI_TENSOR) {
    const double dA = 1.0 / (double)p.scaleA[0];
    const double zA = (double)p.zeroA[0] + (double)p.halfA * dA;
    const double dB = 1.0 / (double)p.scaleB[0];
    const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
    const double kzz = (double)p.K * zA * zB;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t col = n0 + wn * 64 + j * 32 + lrow;
      const double cterm = col < p.N ? zA * dB * (double)p.sumB[col] : 0.0;
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          if (row < p.M && col < p.N) {
            const double v = dA * dB * (double)acc[i][j][r] + dA * zB * (double)p.sumA[row] + cterm + kzz;
            p.out[row * p.ldo + col] = (float)v;
          }
        }
    }
    return;
  } else {
    // grad_X: per-tensor B (weights), per-row or per-group A (gradient).
    // Stage the accumulators and per-row data in LDS (the operand buffers
    // are dead after the loop), then thread t owns column t % 128 and the
    // 64 rows of half t / 128: group sums are sequential in one thread.
    const double dW = 1.0 / (double)p.scaleB[0];
    const double zW = (double)p.zeroB[0] + (double)p.halfB * dW;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          lds.ep.acc[wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3)][wn * 64 + j * 32 + lrow] = acc[i][j][r];
    if (tid < BM) {
      const int64_t row = m0 + tid;
      RowStage q{};
      if (row < p.M) {
        const float s = p.rowwiseA ? p.scaleA[row] : p.scaleA[0];
        const float z = p.rowwiseA ? p.zeroA[row] : p.zeroA[0];
        q.kind = (EPI == EPI_BHQ) ? bhq_slot_kind(p.L, row) : 0;
        q.rterm = zW * (double)p.sumA[row];
        q.dq = 1.0 / (double)s;
        if (q.kind != 0) {
          q.hz = (double)p.halfA + (double)z;
          q.inv_d = q.dq;
        } else {
          q.hz = (double)z + (double)p.halfA * q.dq;
        }
        q.orow = p.perm ? p.perm[row] : (int)row;
      } else {
        q.orow = -1;
      }
      lds.ep.rows[tid] = q;
    }
    __syncthreads();
    const int c = tid & (BN - 1);
    const int rbase = (tid >> 7) * 64;
    const int64_t col = n0 + c;
    if (col >= p.N) return;
    // sum over K of the dequantized weight column: dW * sum q_W + K zW
    const double colterm = dW * (double)p.sumB[col] + (double)p.K * zW;
    if constexpr (EPI == EPI_BHQ && KG > 1) {
      for (int g0 = rbase; g0 < rbase + 64; g0 += KG) {
        // T_p = (code_p + c_g) . W~ ; S = sum over the group's multi-row slots
        double S = 0.0, T0 = 0.0;
        for (int t = 0; t < KG; ++t) {
          const RowStage& q = lds.ep.rows[g0 + t];
          const double T = dW * (double)lds.ep.acc[g0 + t][c] + (q.rterm + q.hz * colterm);
          if (q.kind != 0) S += T;
          if (t == 0) T0 = T;
        }
        const int gkind = lds.ep.rows[g0].kind;
        const double alpha = gkind == 2 ? p.L.inv_sk_p : p.L.inv_sk_k;
        const double tau = (alpha * S - T0) / (1.0 - alpha);
        for (int t = 0; t < KG; ++t) {
          const RowStage& q = lds.ep.rows[g0 + t];
          if (q.orow < 0) continue;
          const double a = (double)lds.ep.acc[g0 + t][c];
          double v;
          if (q.kind != 0) {
            const double T = dW * a + (q.rterm + q.hz * colterm);
            const double Z = (t == 0) ? T + (1.0 - alpha) * tau : T - alpha * tau;
            v = Z * q.inv_d;
          } else {
            v = q.dq * (dW * a + q.rterm) + q.hz * colterm;
          }
          p.out[(int64_t)q.orow * p.ldo + col] = (float)v;
        }
      }
    } else {
      for (int t = rbase; t < rbase + 64; ++t) {
        const RowStage& q = lds.ep.rows[t];
        if (q.orow < 0) continue;
        const double a = (double)lds.ep.acc[t][c];
        const double v = q.dq * (dW * a + q.rterm) + q.hz * colterm;
        p.out[(int64_t)q.orow * p.ldo + col] = (float)v;
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

template <int EPI, int KG>
static hipError_t launch_gemm_t(const GemmParams& p, hipStream_t s) {
  const int64_t gx = (p.N + BN - 1) / BN, gy = (p.M + BM - 1) / BM;
  if (gx > 0x7FFFFFFF || gy > 65535 || p.splits > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemm_i8_kernel<EPI, KG>), dim3((unsigned)gx, (unsigned)gy, (unsigned)p.splits), dim3(256), 0,
                     s, p);
  return hipGetLastError();
}

hipError_t launch_gemm(const GemmParams& p, int epi, hipStream_t s) {
  switch (epi) {
    case EPI_RAW_I32: return launch_gemm_t<EPI_RAW_I32, 0>(p, s);
    case EPI_TENSOR: return launch_gemm_t<EPI_TENSOR, 0>(p, s);
    case EPI_ROW: return launch_gemm_t<EPI_ROW, 0>(p, s);
    case EPI_BHQ:
      switch (p.L.k) {
        case 1: return launch_gemm_t<EPI_BHQ, 1>(p, s);
        case 2: return launch_gemm_t<EPI_BHQ, 2>(p, s);
        case 4: return launch_gemm_t<EPI_BHQ, 4>(p, s);
        case 8: return launch_gemm_t<EPI_BHQ, 8>(p, s);
        case 16: return launch_gemm_t<EPI_BHQ, 16>(p, s);
        case 32: return launch_gemm_t<EPI_BHQ, 32>(p, s);
        case 64: return launch_gemm_t<EPI_BHQ, 64>(p, s);
        default: return hipErrorInvalidValue;
      }
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fqt
