// Shared int8 matrix-core contraction core (gfx950): tile shapes, 16-byte
// operand chunks, and the double-buffered K loop on v_mfma_i32_32x32x32_i8.
// Used by the linear-layer contractions (gemm.hip) and the conv ones
// (conv.hip).
#pragma once

#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int NUM_XCD = 8;

// Block tile BM x BN, wave tile WM x WN, BK_ K bytes per pipeline stage.
// LDS rows are padded by 16 bytes (conflict-free 8- and 16-lane phases).
template <int BM_, int BN_, int WM_, int WN_, int BK_ = 128>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, BK = BK_;
  static constexpr int KCH = BK / 16;          // 16-byte chunks per row per stage
  static constexpr int LDS_STRIDE = BK + 16;
  static constexpr int WAVES_N = BN / WN;
  static constexpr int THREADS = (BM / WM) * (BN / WN) * 64;
  static constexpr int IT = WM / 32, JT = WN / 32;
  static constexpr int A_CHUNKS = BM * KCH / THREADS;  // 16-byte chunks per thread per K stage
  static constexpr int B_CHUNKS = BN * KCH / THREADS;
  static constexpr int OP_BYTES = 2 * (BM + BN) * LDS_STRIDE;
};
// Configurations measured best on MI355X for the layer shapes (8 waves each).
using CfgLarge = TileCfg<256, 128, 64, 64, 128>;
using CfgSmall = TileCfg<128, 128, 32, 64, 128>;

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
// The generic path takes the A operand through `aload(row, k)` (a 16-byte
// chunk, zero outside the operand), which is how the conv input-gradient
// contraction gathers its implicit im2col rows.
struct PlainALoader {
  const int8_t* A;
  int64_t lda, M, kend;
  bool aligned;
  __device__ __forceinline__ Chunk16 operator()(int64_t r, int64_t k) const {
    return load_chunk(A, lda, r, M, k, kend, aligned);
  }
};

template <class C, bool FAST, class ALoader>
__device__ __forceinline__ void gemm_mainloop(const GemmParams& p, const ALoader& aload, int8_t* lds, int64_t m0,
                                              int64_t n0, int64_t kbeg, int64_t kend, v16i (&acc)[C::IT][C::JT]) {
  int8_t* sA = lds;                          // [2][BM * C::LDS_STRIDE]
  int8_t* sB = lds + 2 * C::BM * C::LDS_STRIDE;  // [2][BN * C::LDS_STRIDE]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const bool alB = ((p.ldb & 15) == 0) && (((uintptr_t)p.B & 15) == 0);
  const int64_t nk = (kend - kbeg + C::BK - 1) / C::BK;

  uint32_t offA[C::A_CHUNKS], offB[C::B_CHUNKS];
  if constexpr (FAST) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      const int64_t r = (m0 + c / C::KCH < p.M) ? m0 + c / C::KCH : p.M - 1;
      offA[i] = (uint32_t)(r * p.lda) + 16u * (uint32_t)(c % C::KCH);
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      const int64_t r = (n0 + c / C::KCH < p.N) ? n0 + c / C::KCH : p.N - 1;
      offB[i] = (uint32_t)(r * p.ldb) + 16u * (uint32_t)(c % C::KCH);
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
      const int8_t* a = Ak + t * C::BK;
      const int8_t* b = Bk + t * C::BK;
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i) st.a[i] = *reinterpret_cast<const u32x4v*>(a + offA[i]);
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i) st.b[i] = *reinterpret_cast<const u32x4v*>(b + offB[i]);
    } else {
      const int64_t k0 = kbeg + t * C::BK;
#pragma unroll
      for (int i = 0; i < C::A_CHUNKS; ++i) {
        const int c = tid + C::THREADS * i;
        const Chunk16 v = aload(m0 + c / C::KCH, k0 + 16 * (c % C::KCH));
        st.a[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
      }
#pragma unroll
      for (int i = 0; i < C::B_CHUNKS; ++i) {
        const int c = tid + C::THREADS * i;
        const Chunk16 v = load_chunk(p.B, p.ldb, n0 + c / C::KCH, p.N, k0 + 16 * (c % C::KCH), kend, alB);
        st.b[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
      }
    }
  };
  auto sstore = [&](const Stage& st, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      *reinterpret_cast<u32x4v*>(&sA[buf * C::BM * C::LDS_STRIDE + (c / C::KCH) * C::LDS_STRIDE + 16 * (c % C::KCH)]) = st.a[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      *reinterpret_cast<u32x4v*>(&sB[buf * C::BN * C::LDS_STRIDE + (c / C::KCH) * C::LDS_STRIDE + 16 * (c % C::KCH)]) = st.b[i];
    }
  };
  const int lrow = lane & 31;
  const int lk = 16 * (lane >> 5);
  const int8_t* a_lane = sA + (wm * C::WM + lrow) * C::LDS_STRIDE + lk;
  const int8_t* b_lane = sB + (wn * C::WN + lrow) * C::LDS_STRIDE + lk;
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const int8_t* a_base = a_lane + buf * C::BM * C::LDS_STRIDE;
    const int8_t* b_base = b_lane + buf * C::BN * C::LDS_STRIDE;
#pragma unroll
    for (int kk = 0; kk < C::BK / 32; ++kk) {
      v4i a[C::IT], b[C::JT];
#pragma unroll
      for (int i = 0; i < C::IT; ++i) a[i] = *reinterpret_cast<const v4i*>(a_base + i * 32 * C::LDS_STRIDE + kk * 32);
#pragma unroll
      for (int j = 0; j < C::JT; ++j) b[j] = *reinterpret_cast<const v4i*>(b_base + j * 32 * C::LDS_STRIDE + kk * 32);
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

}  // namespace fqt
