// Exact contraction of 4-bit offset codes on the gfx950 scaled matrix-core
// instruction with 6-bit float operands (v_mfma_scale_f32_32x32x64_f8f6f4,
// both operands e3m2, unit scales): every integer in [-8, 8] is an e3m2
// value, products are at most 64 in magnitude and float32 sums of integers
// stay exact below 2^24, so K chunks of at most 131072 give exact integer
// accumulators (int32 partials, summed in int64 across chunks).
//
// Packed operand layout: rows of ceil(K / 128) * 96 bytes; each 24-byte
// group holds 32 consecutive codes, code j at bits 6j .. 6j + 5 of the
// group's six little-endian dwords (the instruction's per-lane operand:
// lane l takes row l % 32 and codes 32 (l / 32) .. + 31 of a 64-code step).
#include "gemm_core.h"

namespace fqt {

// e3m2 bits of an integer q with |q| <= 8: sign, exponent e + 3, two
// mantissa bits, |q| = (1 + m / 4) 2^e.
__device__ __forceinline__ uint32_t e3m2_of_int(int q) {
  const uint32_t a = (uint32_t)(q < 0 ? -q : q);
  if (a == 0) return 0u;
  const uint32_t e = 31u - __builtin_clz(a);
  const uint32_t m = ((a << 2) >> e) - 4u;
  return (q < 0 ? 0x20u : 0u) | ((e + 3u) << 2) | m;
}

__global__ void pack_status_clear_kernel(uint32_t* status) {
  if (threadIdx.x < STATUS_WORDS) status[threadIdx.x] = 0u;
}

// One thread per 32-code group: codes past K are zero; a code outside
// [-8, 7] sets the status flag (it has no exact place in the contraction).
__global__ __launch_bounds__(256) void pack_e3m2_kernel(const int8_t* src, int64_t rows, int64_t K, int64_t ld,
                                                         uint32_t* dst, int64_t groups, uint32_t* status) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * groups) return;
  const int64_t row = idx / groups, g = idx % groups;
  const int8_t* s = src + row * ld + 32 * g;
  // the group's 32 codes: two 16-byte loads when whole and aligned
  int8_t v[32];
  if (32 * g + 32 <= K && ((uintptr_t)s & 15) == 0) {
    *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(s);
    *reinterpret_cast<uint4*>(v + 16) = *reinterpret_cast<const uint4*>(s + 16);
  } else {
#pragma unroll
    for (int j = 0; j < 32; ++j) v[j] = (32 * g + j < K) ? s[j] : (int8_t)0;
  }
  uint32_t w[6] = {0u, 0u, 0u, 0u, 0u, 0u};
  int bad = 0;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int q = (int)v[j];
    bad |= (q < -8) | (q > 7);
    const uint32_t e = e3m2_of_int(q < -8 ? -8 : (q > 7 ? 7 : q));
    const int bit = 6 * j, wi = bit >> 5, o = bit & 31;
    w[wi] |= e << o;
    if (o > 26) w[wi + 1] |= e >> (32 - o);
  }
  uint2* d = reinterpret_cast<uint2*>(dst + idx * 6);
  d[0] = make_uint2(w[0], w[1]);
  d[1] = make_uint2(w[2], w[3]);
  d[2] = make_uint2(w[4], w[5]);
  if (bad) atomicOr(status, STATUS_NONFINITE);
}

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

constexpr int F6_BK = 128;        // codes per stage
constexpr int F6_ROWB = 96;       // bytes per row per stage
constexpr int F6_LS = 104;        // LDS row stride: 26 dwords, so 32 rows of 8-byte reads hit distinct banks
constexpr int F6_CH = F6_ROWB / 8;  // 8-byte chunks per row per stage

template <class C>
__global__ __launch_bounds__(C::THREADS) void gemm_bf6_kernel(Bf6Params p) {
  __shared__ __attribute__((aligned(16))) int8_t lds[2 * (C::BM + C::BN) * F6_LS];
  constexpr int ACH = C::BM * F6_CH / C::THREADS, BCH = C::BN * F6_CH / C::THREADS;
  static_assert(ACH * C::THREADS == C::BM * F6_CH && BCH * C::THREADS == C::BN * F6_CH, "whole chunks");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const int64_t tiles_n = (p.N + C::BN - 1) / C::BN, tiles_m = (p.M + C::BM - 1) / C::BM;
  const int64_t tile = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  const int64_t m0 = (tile / tiles_n) * C::BM, n0 = (tile % tiles_n) * C::BN;
  const int split = blockIdx.y;
  const int64_t kbeg = (int64_t)split * p.kchunk;
  const int64_t kend = (kbeg + p.kchunk < p.Kpad) ? kbeg + p.kchunk : p.Kpad;
  const int64_t nk = (kend - kbeg) / F6_BK;
  int8_t* sA = lds;
  int8_t* sB = lds + 2 * C::BM * F6_LS;
  // per-thread source pointers (rows past the edge read the last row; never stored)
  const int8_t* srcA[ACH];
  const int8_t* srcB[BCH];
  int offA[ACH], offB[BCH];
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    const int c = tid + C::THREADS * i, r = c / F6_CH, ch = c % F6_CH;
    const int64_t row = (m0 + r < p.M) ? m0 + r : p.M - 1;
    srcA[i] = p.A + row * p.lda + (kbeg / F6_BK) * F6_ROWB + 8 * ch;
    offA[i] = r * F6_LS + 8 * ch;
  }
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    const int c = tid + C::THREADS * i, r = c / F6_CH, ch = c % F6_CH;
    const int64_t row = (n0 + r < p.N) ? n0 + r : p.N - 1;
    srcB[i] = p.B + row * p.ldb + (kbeg / F6_BK) * F6_ROWB + 8 * ch;
    offB[i] = r * F6_LS + 8 * ch;
  }
  struct Stage {
    uint2 a[ACH];
    uint2 b[BCH];
  };
  Stage st0, st1;
  auto gload = [&](Stage& st, int64_t t) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) st.a[i] = *reinterpret_cast<const uint2*>(srcA[i] + t * F6_ROWB);
#pragma unroll
    for (int i = 0; i < BCH; ++i) st.b[i] = *reinterpret_cast<const uint2*>(srcB[i] + t * F6_ROWB);
  };
  auto sstore = [&](const Stage& st, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) *reinterpret_cast<uint2*>(sA + buf * C::BM * F6_LS + offA[i]) = st.a[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i) *reinterpret_cast<uint2*>(sB + buf * C::BN * F6_LS + offB[i]) = st.b[i];
  };
  v16f acc[C::IT][C::JT];
#pragma unroll
  for (int i = 0; i < C::IT; ++i)
#pragma unroll
    for (int j = 0; j < C::JT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  const int lrow = lane & 31, h = lane >> 5;
  auto rd = [&](const int8_t* base) __attribute__((always_inline)) {
    const uint2 x0 = *reinterpret_cast<const uint2*>(base);
    const uint2 x1 = *reinterpret_cast<const uint2*>(base + 8);
    const uint2 x2 = *reinterpret_cast<const uint2*>(base + 16);
    return v8i{(int)x0.x, (int)x0.y, (int)x1.x, (int)x1.y, (int)x2.x, (int)x2.y, 0, 0};
  };
  auto compute = [&](int buf) __attribute__((always_inline)) {
    const int8_t* a_base = sA + buf * C::BM * F6_LS + (wm * C::WM + lrow) * F6_LS + 24 * h;
    const int8_t* b_base = sB + buf * C::BN * F6_LS + (wn * C::WN + lrow) * F6_LS + 24 * h;
#pragma unroll
    for (int ks = 0; ks < F6_BK / 64; ++ks) {
      v8i a[C::IT], b[C::JT];
#pragma unroll
      for (int i = 0; i < C::IT; ++i) a[i] = rd(a_base + i * 32 * F6_LS + 48 * ks);
#pragma unroll
      for (int j = 0; j < C::JT; ++j) b[j] = rd(b_base + j * 32 * F6_LS + 48 * ks);
#pragma unroll
      for (int i = 0; i < C::IT; ++i)
#pragma unroll
        for (int j = 0; j < C::JT; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[i], b[j], acc[i][j], 3, 3, 0, 127, 0, 127);
    }
  };
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
  // exact integers in float32 -> int32 partials of this split
  int32_t* out = p.part + (int64_t)split * p.M * p.N;
#pragma unroll
  for (int i = 0; i < C::IT; ++i)
#pragma unroll
    for (int j = 0; j < C::JT; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * C::WM + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        const int64_t col = n0 + wn * C::WN + j * 32 + lrow;
        if (row < p.M && col < p.N) out[row * p.N + col] = (int32_t)acc[i][j][r];
      }
}

int64_t bf6_row_bytes(int64_t K) { return (K + F6_BK - 1) / F6_BK * F6_ROWB; }

hipError_t launch_pack_e3m2(const int8_t* src, int64_t rows, int64_t K, int64_t ld, int8_t* dst, uint32_t* status,
                            hipStream_t s) {
  const int64_t groups = bf6_row_bytes(K) / 24;
  const int64_t n = rows * groups;
  if (n < 1 || (n + 255) / 256 > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(pack_e3m2_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, rows, K, ld,
                     reinterpret_cast<uint32_t*>(dst), groups, status);
  return hipGetLastError();
}

hipError_t launch_status_clear(uint32_t* status, hipStream_t s) {
  hipLaunchKernelGGL(pack_status_clear_kernel, dim3(1), dim3(64), 0, s, status);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_bf6_c(const Bf6Params& p, hipStream_t s) {
  const int64_t tiles = gemm_tiles_of<C>(p.M, p.N);
  if (tiles > 0x7FFFFFFF || p.splits > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL((gemm_bf6_kernel<C>), dim3((unsigned)tiles, (unsigned)p.splits), dim3(C::THREADS), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_gemm_bf6(const Bf6Params& p, hipStream_t s) {
  if (p.kchunk % F6_BK != 0 || p.Kpad % F6_BK != 0) return hipErrorInvalidValue;
  return gemm_tiles_of<CfgLarge>(p.M, p.N) >= 256 ? launch_bf6_c<CfgLarge>(p, s) : launch_bf6_c<CfgSmall>(p, s);
}

}  // namespace fqt
