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


// Block tile BM x BN, wave tile WM x WN, BK_ K bytes per pipeline stage.
// Generic K loop: LDS rows padded by 16 bytes (conflict-free 8- and 16-lane
// phases), two stages.  Fast K loop: NS_ stages of swizzled 128-byte rows.
template <int BM_, int BN_, int WM_, int WN_, int BK_ = 128, int NS_ = 2>
struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, BK = BK_, NS = NS_;
  static constexpr int KCH = BK / 16;          // 16-byte chunks per row per stage
  static constexpr int LDS_STRIDE = BK + 16;
  static constexpr int WAVES_N = BN / WN;
  static constexpr int WAVES = (BM / WM) * (BN / WN);
  static constexpr int THREADS = WAVES * 64;
  static constexpr int IT = WM / 32, JT = WN / 32;
  static constexpr int A_CHUNKS = BM * KCH / THREADS;  // 16-byte chunks per thread per K stage
  static constexpr int B_CHUNKS = BN * KCH / THREADS;
  // fast loop: one stage holds A then B; each wave fills whole 1 KB blocks
  static constexpr int STAGE = (BM + BN) * BK;
  static constexpr int A_INS = BM * BK / 1024 / WAVES, B_INS = BN * BK / 1024 / WAVES;
  static constexpr int GEN_BYTES = 2 * (BM + BN) * LDS_STRIDE;
  static constexpr int OP_BYTES = GEN_BYTES > NS * STAGE ? GEN_BYTES : NS * STAGE;
};
// Configurations measured best on MI355X for the layer shapes (8 waves each).
using CfgLarge = TileCfg<256, 128, 64, 64, 128, 3>;
using CfgSmall = TileCfg<128, 128, 32, 64, 128, 4>;
// at most 64 rows (the conv grad_W contraction over output channels): no
// half-empty 128-row tiles
using CfgNarrow = TileCfg<64, 128, 32, 64, 128, 3>;

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

template <class C>
inline int64_t gemm_tiles_of(int64_t M, int64_t N) {
  return ((M + C::BM - 1) / C::BM) * ((N + C::BN - 1) / C::BN);
}

// Bijective block -> tile map: the first 8 * floor(T / 8) blocks give each
// XCD (block id mod 8) a contiguous run of tiles; the rest map to themselves.
__device__ __forceinline__ int64_t xcd_tile(int64_t id, int64_t ntiles) {
  const int64_t q = ntiles / NUM_XCD;
  if (id < q * NUM_XCD) return (id % NUM_XCD) * q + id / NUM_XCD;
  return id;
}

// The K loops.  The fast one (dma_mainloop below) requires 16-byte aligned
// rows and a K range that is a whole number of 128-byte stages.  The generic
// one (register-staged, two LDS buffers) takes both operands through loaders
// (16-byte chunks, zero outside the operand and past the end of K, where the
// loop also loads), which is how the conv input-gradient contraction gathers
// its implicit im2col rows, and handles ragged K and unaligned rows.  An A
// loader maps a row once to a per-row state (`row`), then loads 16-byte
// chunks of it (`load`) stage by stage, so per-row index arithmetic stays out
// of the K loop; a thread's chunks of one stage share their K offset, decoded
// once (`kstate`).
struct PlainALoader {
  const int8_t* A;
  int64_t lda, M, kend;
  bool aligned;
  struct Row {
    int64_t r;
  };
  typedef int64_t KState;
  __device__ __forceinline__ Row row(int64_t r) const { return Row{r}; }
  __device__ __forceinline__ KState kstate(int64_t k) const { return k; }
  __device__ __forceinline__ Chunk16 load(const Row& rw, const KState& k) const {
    return load_chunk(A, lda, rw.r, M, k, kend, aligned);
  }
};

// A operand of codes of at most 4 bits stored two per byte (code + 8 in a
// nibble, column 2i in the low half of byte i): 16 codes from 8 bytes,
// unpacked to int8 offset codes.  K is a multiple of 16 (checked at launch),
// so a chunk is whole or past the end (zero).
struct PackedALoader {
  const int8_t* A;
  int64_t lda, M, kend;  // lda in bytes
  struct Row {
    int64_t r;
  };
  typedef int64_t KState;
  __device__ __forceinline__ Row row(int64_t r) const { return Row{r}; }
  __device__ __forceinline__ KState kstate(int64_t k) const { return k; }
  // 8 nibbles of w -> 8 offset codes in two words
  __device__ __forceinline__ static void unpack8(uint32_t w, uint32_t& o0, uint32_t& o1) {
    const uint32_t lo = w & 0x0F0F0F0Fu, hi = (w >> 4) & 0x0F0F0F0Fu;
    // bytes (lo0, hi0, lo1, hi1) and (lo2, hi2, lo3, hi3); u -> u - 8 as int8 is (u + 0x78) ^ 0x80
    o0 = (__builtin_amdgcn_perm(hi, lo, 0x05010400u) + 0x78787878u) ^ 0x80808080u;
    o1 = (__builtin_amdgcn_perm(hi, lo, 0x07030602u) + 0x78787878u) ^ 0x80808080u;
  }
  __device__ __forceinline__ Chunk16 load(const Row& rw, const KState& k) const {
    Chunk16 c{{0u, 0u, 0u, 0u}};
    if (rw.r >= M || k >= kend) return c;
    const uint2 v = *reinterpret_cast<const uint2*>(A + rw.r * lda + (k >> 1));
    unpack8(v.x, c.w[0], c.w[1]);
    unpack8(v.y, c.w[2], c.w[3]);
    return c;
  }
};

// The B operand of the generic loop: 16-byte chunks of K-contiguous rows,
// zero outside the matrix / K range (`load_chunk`).
struct PlainBLoader {
  const int8_t* B;
  int64_t ldb, N, kend;
  bool aligned;
  __device__ __forceinline__ Chunk16 load(int64_t r, int64_t k) const {
    return load_chunk(B, ldb, r, N, k, kend, aligned);
  }
};

typedef __attribute__((address_space(1))) void gmem_void;
typedef __attribute__((address_space(3))) void lmem_void;

// 16-byte slot of (row r, chunk c) in one operand of a fast-loop stage:
// 8-row blocks of 1 KB, row-major, chunk index XOR-swizzled by (r / 2) mod 8.
// One load instruction of a wave fills one block with eight whole 128-byte
// rows (consecutive lanes read consecutive chunks of one row), and the 16
// rows one matrix-core operand read touches at a fixed chunk fall on 16
// distinct 16-byte bank groups.
__device__ __forceinline__ int kslot(int r, int c) { return 8 * r + (c ^ ((r >> 1) & 7)); }

// One stage of the fast loop: wait for this wave's loads of stage t, then the
// barrier (everyone's have landed, and everyone is done reading the buffer
// that the loads of stage t + NS - 1 now fill), then the matrix-core work on
// `cur`, each MFMA followed by one LDS read of the next K step, with this
// wave's loads of stage t + NS - 1 spread over the MFMAs (one after every
// second MFMA where there are enough): issued back to back they queue up in
// the address unit and hold up the MFMA issue behind them.  `cur` and `nxt` are never the same
// buffer; the caller passes them as distinct restrict pointers so that the
// pending loads into `nxt` do not hold up the reads of `cur`.
template <class C>
__device__ __forceinline__ void dma_stage(const int8_t* __restrict__ cur, int8_t* __restrict__ nxt,
                                          const int8_t* const (&srcA)[C::A_INS], const int8_t* const (&srcB)[C::B_INS],
                                          int64_t t, int64_t nk, v16i (&acc)[C::IT][C::JT]) {
  constexpr int PER = C::A_INS + C::B_INS;
  constexpr int NMF = C::IT * C::JT * (C::BK / 32);  // MFMAs per stage
  constexpr int SPREAD = 2 * PER <= NMF ? 2 : 1;  // MFMAs per load slot
  static_assert(PER <= (NMF + SPREAD - 1) / SPREAD, "every load of a stage gets an MFMA slot");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  if (t + C::NS - 2 < nk)
    __builtin_amdgcn_s_waitcnt(0x3F70 | ((C::NS - 2) * PER));  // vmcnt: later stages may stay in flight
  else
    __builtin_amdgcn_s_waitcnt(0x3F70);                          // vmcnt(0)
  __builtin_amdgcn_s_barrier();
  const bool more = t + C::NS - 1 < nk;
  const int64_t ko = (t + C::NS - 1) * C::BK;
  // load q of the next stage (q < A_INS: A, else B), in its MFMA slot
  auto load = [&](int q) __attribute__((always_inline)) {
    if (q < C::A_INS)
      __builtin_amdgcn_global_load_lds((gmem_void*)(srcA[q] + ko), (lmem_void*)(nxt + (wave * C::A_INS + q) * 1024), 16,
                                       0, 0);
    else
      __builtin_amdgcn_global_load_lds((gmem_void*)(srcB[q - C::A_INS] + ko),
                                       (lmem_void*)(nxt + C::BM * C::BK + (wave * C::B_INS + q - C::A_INS) * 1024), 16,
                                       0, 0);
  };
  const int lrow = lane & 31, lh = lane >> 5;
  const int8_t* sa = cur;
  const int8_t* sb = cur + C::BM * C::BK;
  v4i a[2][C::IT], b[2][C::JT];
  auto rd = [&](int set, int kk) __attribute__((always_inline)) {
    const int c = 2 * kk + lh;
#pragma unroll
    for (int i = 0; i < C::IT; ++i) a[set][i] = *reinterpret_cast<const v4i*>(sa + 16 * kslot(wm * C::WM + i * 32 + lrow, c));
#pragma unroll
    for (int j = 0; j < C::JT; ++j) b[set][j] = *reinterpret_cast<const v4i*>(sb + 16 * kslot(wn * C::WN + j * 32 + lrow, c));
  };
  rd(0, 0);
#pragma unroll
  for (int kk = 0; kk < C::BK / 32; ++kk) {
    const int cs = kk & 1;
    if (kk + 1 < C::BK / 32) rd(cs ^ 1, kk + 1);
#pragma unroll
    for (int i = 0; i < C::IT; ++i)
#pragma unroll
      for (int j = 0; j < C::JT; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[cs][i], b[cs][j], acc[i][j], 0, 0, 0);
        const int m = (kk * C::IT + i) * C::JT + j;
        if (m % SPREAD == 0 && m / SPREAD < PER && more) load(m / SPREAD);
      }
  }
}

// The fast K loop: operands loaded straight into LDS (global_load_lds_dwordx4,
// NS - 1 stages in flight), 128-byte K stages, rows past the matrix edge
// clamped to its last row (their outputs are never stored).  Ends with a
// barrier, so the caller may reuse the LDS.
template <class C>
__device__ __forceinline__ void dma_mainloop(const GemmParams& p, int8_t* __restrict__ b0, int8_t* __restrict__ b1,
                                             int8_t* __restrict__ b2, int8_t* __restrict__ b3, int64_t m0, int64_t n0,
                                             int64_t kbeg, int64_t kend, v16i (&acc)[C::IT][C::JT]) {
  static_assert(C::BK == 128 && C::NS >= 2 && C::NS <= 4, "fast loop: 128-byte stages, 2..4 buffers");
  static_assert(C::A_INS * 1024 * C::WAVES == C::BM * C::BK && C::B_INS * 1024 * C::WAVES == C::BN * C::BK,
                "whole 1 KB blocks per wave");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int8_t* srcA[C::A_INS];
  const int8_t* srcB[C::B_INS];
#pragma unroll
  for (int i = 0; i < C::A_INS; ++i) {
    const int r = 8 * (wave * C::A_INS + i) + (lane >> 3);
    const int64_t row = (m0 + r < p.M) ? m0 + r : p.M - 1;
    srcA[i] = p.A + row * p.lda + kbeg + 16 * ((lane & 7) ^ ((r >> 1) & 7));
  }
#pragma unroll
  for (int i = 0; i < C::B_INS; ++i) {
    const int r = 8 * (wave * C::B_INS + i) + (lane >> 3);
    const int64_t row = (n0 + r < p.N) ? n0 + r : p.N - 1;
    int64_t off = row * p.ldb;
    if (p.bmap_c > 0) {  // conv tap (kr, ks), channel ch: copy ks, K offset kr gwp
      const int64_t tap = row / p.bmap_c, ch = row - tap * p.bmap_c;
      const int64_t kr = tap / p.bmap_kw, ks = tap - kr * p.bmap_kw;
      off = (ks * p.bmap_c + ch) * p.ldb + kr * p.bmap_wp;
    }
    srcB[i] = p.B + off + kbeg + 16 * ((lane & 7) ^ ((r >> 1) & 7));
  }
  const int64_t nk = (kend - kbeg) / C::BK;
  int8_t* bufs[4] = {b0, b1, b2, b3};
#pragma unroll
  for (int s = 0; s < C::NS - 1; ++s) {
    if (s < nk) {
#pragma unroll
      for (int i = 0; i < C::A_INS; ++i)
        __builtin_amdgcn_global_load_lds((gmem_void*)(srcA[i] + s * C::BK),
                                         (lmem_void*)(bufs[s] + (wave * C::A_INS + i) * 1024), 16, 0, 0);
#pragma unroll
      for (int i = 0; i < C::B_INS; ++i)
        __builtin_amdgcn_global_load_lds((gmem_void*)(srcB[i] + s * C::BK),
                                         (lmem_void*)(bufs[s] + C::BM * C::BK + (wave * C::B_INS + i) * 1024), 16,
                                         0, 0);
    }
  }
  // stage t reads buffer t % NS and fills buffer (t + NS - 1) % NS
  for (int64_t t = 0; t < nk; t += C::NS) {
    dma_stage<C>(b0, C::NS == 2 ? b1 : (C::NS == 3 ? b2 : b3), srcA, srcB, t, nk, acc);
    if (t + 1 < nk) dma_stage<C>(b1, b0, srcA, srcB, t + 1, nk, acc);
    if (C::NS > 2 && t + 2 < nk) dma_stage<C>(b2, b1, srcA, srcB, t + 2, nk, acc);
    if (C::NS > 3 && t + 3 < nk) dma_stage<C>(b3, b2, srcA, srcB, t + 3, nk, acc);
  }
  __syncthreads();
}

// K offsets of the stages a K loop runs: stage t starts at kbeg + t bk, n
// stages (offsets past the end load zero chunks)
struct KRange {
  int64_t kbeg, bk, n;
  __device__ __forceinline__ int64_t k(int64_t t) const { return kbeg + t * bk; }
};

// The register-staged K loop over the stages of a stage map KM (km.n stages,
// stage t at K offset km.k(t); for t >= km.n, km.k(t) must lie past the
// loaders' K range so that they load zeros).
template <class C, class ALoader, class BLoader, class KM>
__device__ __forceinline__ void generic_mainloop_km(const GemmParams& p, const ALoader& aload, const BLoader& bload,
                                                    int8_t* lds, int64_t m0, int64_t n0, const KM& km,
                                                    v16i (&acc)[C::IT][C::JT]) {
  int8_t* sA = lds;                          // [2][BM * C::LDS_STRIDE]
  int8_t* sB = lds + 2 * C::BM * C::LDS_STRIDE;  // [2][BN * C::LDS_STRIDE]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const int64_t nk = km.n;

  // Two register staging sets: the loads of stage t + 1 are issued one
  // iteration before the stage is stored to LDS, so each global load has two
  // iterations of matrix-core work to land.
  struct Stage {
    u32x4v a[C::A_CHUNKS];
    u32x4v b[C::B_CHUNKS];
  };
  Stage st0, st1;
  typename ALoader::Row arow[C::A_CHUNKS];
#pragma unroll
  for (int i = 0; i < C::A_CHUNKS; ++i) arow[i] = aload.row(m0 + (tid + C::THREADS * i) / C::KCH);
  static_assert(C::THREADS % C::KCH == 0, "a thread keeps one chunk column");
  const int kch = 16 * (tid % C::KCH);  // the K offset of every A chunk this thread loads
  auto gload = [&](Stage& st, int64_t t) __attribute__((always_inline)) {
    const int64_t k0 = km.k(t);
    const typename ALoader::KState ks = aload.kstate(k0 + kch);  // once per stage: shared by the thread's rows
#pragma unroll
    for (int i = 0; i < C::A_CHUNKS; ++i) {
      const Chunk16 v = aload.load(arow[i], ks);
      st.a[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
    }
#pragma unroll
    for (int i = 0; i < C::B_CHUNKS; ++i) {
      const int c = tid + C::THREADS * i;
      const Chunk16 v = bload.load(n0 + c / C::KCH, k0 + 16 * (c % C::KCH));
      st.b[i] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
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
  // set that stage t came from.  Loads and stores are unconditional (stages
  // past the end of K load zero chunks into a buffer nobody reads), so the
  // loop body has no branches and the compiler's count of loads in flight
  // stays exact across iterations: the stores of stage t + 1 wait for its
  // own loads only, while those of stage t + 2 stay in flight.
  // The loads of stage t + 2 go out between the MFMAs of stage t (one after
  // each MFMA, or after every second when there are twice as many MFMAs):
  // issued as one burst they queue in the address unit and hold up the
  // MFMAs behind them.
  constexpr int NLD = C::A_CHUNKS + C::B_CHUNKS;
  constexpr int NMF = C::IT * C::JT * (C::BK / 32);
  constexpr int SPREAD = 2 * NLD <= NMF ? 2 : 1;
  auto iter = [&](int64_t t, int buf, Stage& next, Stage& far) __attribute__((always_inline)) {
    if constexpr (NLD <= (NMF + SPREAD - 1) / SPREAD) {
      const int64_t k0 = km.k(t + 2);
      const typename ALoader::KState ks = aload.kstate(k0 + kch);
      auto load = [&](int q) __attribute__((always_inline)) {
        if (q < C::A_CHUNKS) {
          const Chunk16 v = aload.load(arow[q], ks);
          far.a[q] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
        } else {
          const int c = tid + C::THREADS * (q - C::A_CHUNKS);
          const Chunk16 v = bload.load(n0 + c / C::KCH, k0 + 16 * (c % C::KCH));
          far.b[q - C::A_CHUNKS] = u32x4v{v.w[0], v.w[1], v.w[2], v.w[3]};
        }
      };
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
          for (int j = 0; j < C::JT; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[i], b[j], acc[i][j], 0, 0, 0);
            const int m = (kk * C::IT + i) * C::JT + j;
            if (m % SPREAD == 0 && m / SPREAD < NLD) load(m / SPREAD);
          }
      }
    } else {
      gload(far, t + 2);
      compute(buf);
    }
    sstore(next, buf ^ 1);
    __syncthreads();
  };
  if (nk <= 0) return;
  gload(st0, 0);
  sstore(st0, 0);
  gload(st1, 1);
  __syncthreads();
  int64_t t = 0;
  for (; t + 1 < nk; t += 2) {
    iter(t, 0, st1, st0);
    iter(t + 1, 1, st0, st1);
  }
  if (t < nk) iter(t, 0, st1, st0);
}

template <class C, class ALoader, class BLoader>
__device__ __forceinline__ void generic_mainloop(const GemmParams& p, const ALoader& aload, const BLoader& bload,
                                                 int8_t* lds, int64_t m0, int64_t n0, int64_t kbeg, int64_t kend,
                                                 v16i (&acc)[C::IT][C::JT]) {
  generic_mainloop_km<C>(p, aload, bload, lds, m0, n0, KRange{kbeg, C::BK, (kend - kbeg + C::BK - 1) / C::BK}, acc);
}

template <class C, bool FAST, class ALoader>
__device__ __forceinline__ void gemm_mainloop(const GemmParams& p, const ALoader& aload, int8_t* lds, int64_t m0,
                                              int64_t n0, int64_t kbeg, int64_t kend, v16i (&acc)[C::IT][C::JT]) {
  if constexpr (FAST) {
    // distinct stage buffers of one LDS array
    dma_mainloop<C>(p, lds, lds + C::STAGE, lds + (C::NS > 2 ? 2 : 1) * C::STAGE, lds + (C::NS > 3 ? 3 : 1) * C::STAGE,
                    m0, n0, kbeg, kend, acc);
  } else {
    const bool alB = ((p.ldb & 15) == 0) && (((uintptr_t)p.B & 15) == 0);
    generic_mainloop<C>(p, aload, PlainBLoader{p.B, p.ldb, p.N, kend, alB}, lds, m0, n0, kbeg, kend, acc);
  }
}

}  // namespace fqt
