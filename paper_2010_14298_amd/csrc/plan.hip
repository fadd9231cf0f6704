// General block Householder plans on gfx950: groups of any size in slot
// order (App. D's adaptive grouping, and fixed block sizes that are not a
// power of two up to 64), the forward transform's per-group column term, and
// the inverse transform of the input gradient.
//
//   sort        rows by infinity norm (launch_bhq_sort, quant.hip)
//   prep        per sorted position: M, R, their cube roots; prefix sums of M
//   objective   App. D, step 2: for every number of groups G the groups take
//               the G largest rows and small-row shares proportional to M_i
//               (cumulative rounding); scored by the exact |S^-1|_F^2
//   argmin      least objective, ties to fewer groups
//   build       perm, per-slot scale / zero, group offsets, slot records
//   tau         per multi-row group and column: the rank-1 term of the
//               reflection, from the column sum in slot order
//   inverse     diag(d)^-1 H of each multi-row group on the input gradient
#include <math.h>

#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {

// ---------------------------------------------------------------------------
// workspace
// ---------------------------------------------------------------------------
static size_t up256(size_t b) { return (b + 255) / 256 * 256; }

size_t appd_workspace(int64_t rows) {
  const size_t n = (size_t)rows;
  return up256(n * 4) + 4 * up256(n * 4) + up256((n + 1) * 8) + up256(n * 8) + 256;
}

AppdWs appd_carve(void* ws, int64_t rows) {
  const size_t n = (size_t)rows;
  char* p = static_cast<char*>(ws);
  AppdWs w{};
  w.sigma = reinterpret_cast<int32_t*>(p);
  p += up256(n * 4);
  w.Ms = reinterpret_cast<float*>(p);
  p += up256(n * 4);
  w.Rs = reinterpret_cast<float*>(p);
  p += up256(n * 4);
  w.ca = reinterpret_cast<float*>(p);
  p += up256(n * 4);
  w.cc = reinterpret_cast<float*>(p);
  p += up256(n * 4);
  w.P = reinterpret_cast<double*>(p);
  p += up256((n + 1) * 8);
  w.obj = reinterpret_cast<double*>(p);
  p += up256(n * 8);
  w.G = reinterpret_cast<int32_t*>(p);
  return w;
}

// ---------------------------------------------------------------------------
// prep: sorted-position scalars (one thread per position)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void appd_prep_kernel(const float* rmin, const float* rmax, int64_t rows, AppdWs w) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= rows) return;
  const int32_t row = w.sigma[r];
  const float lo = rmin[row], hi = rmax[row];
  float M = fmaxf(fabsf(lo), fabsf(hi));
  float R = hi - lo;
  if (!isfinite(M)) M = 0.0f;
  if (!isfinite(R)) R = 0.0f;
  w.Ms[r] = M;
  w.Rs[r] = R;
  w.ca[r] = cbrt_rn(R);
  w.cc[r] = cbrt_rn(2.0f * M);
}

// P[i] = P[i - 1] + M_(i), one addition at a time in sorted order (one
// thread; the loads of a batch are issued before its additions).
__global__ __launch_bounds__(64) void appd_prefix_kernel(int64_t rows, AppdWs w) {
  if (threadIdx.x != 0) return;
  double P = 0.0;
  w.P[0] = 0.0;
  int64_t i = 0;
  constexpr int U = 16;
  for (; i + U <= rows; i += U) {
    float m[U];
#pragma unroll
    for (int u = 0; u < U; ++u) m[u] = w.Ms[i + u];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      P = P + (double)m[u];
      w.P[i + u + 1] = P;
    }
  }
  for (; i < rows; ++i) {
    P = P + (double)w.Ms[i];
    w.P[i + 1] = P;
  }
}

// First j groups' share of the small rows for G groups (App. D, step 2):
// floor((N - G) P_j / P_G + 1/2) in float64 (product, quotient, sum), with
// c_0 = 0 and c_G = N - G; P_j replaced by j when P_G = 0.
__device__ __forceinline__ int64_t appd_cum(const double* P, int64_t N, int64_t G, int64_t j) {
  const int64_t small = N - G;
  if (j <= 0) return 0;
  if (j >= G) return small;
  const double S = P[G];
  const double q = S > 0.0 ? ((double)small * P[j]) / S : (double)(small * j) / (double)G;
  const int64_t c = (int64_t)floor(q + 0.5);
  return c < small ? c : small;
}

// The term of group i (0-based) of the G-group plan: a one-row group's PSQ
// scale, or the Householder pair of App. C.4.
__device__ __forceinline__ double appd_term(const AppdWs& w, int64_t G, int64_t i, int64_t c0, int64_t c1, int B) {
  const int64_t n = c1 - c0;
  if (n == 0) {
    const float s = scale_from_range(w.Rs[i], B);
    return group_term(s, s, 1);
  }
  const int64_t f = G + c0;  // sorted position of the group's first small row
  float s1, s2;
  group_scales(w.Rs[i], 2.0f * w.Ms[f], w.ca[i], w.cc[f], n + 1, sqrt((double)(n + 1)), B, s1, s2);
  return group_term(s1, s2, n + 1);
}

// One wave per G (four per block, the largest G first): 64 groups' terms
// at a time in parallel, then added to the total one at a time in group
// order (float64).
__global__ __launch_bounds__(256) void appd_objective_kernel(int64_t rows, int B, AppdWs w, double* obj) {
  const int lane = threadIdx.x & 63;
  const int64_t id = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (id >= rows) return;
  const int64_t G = rows - id;
  double total = 0.0;
  for (int64_t i0 = 0; i0 < G; i0 += 64) {
    const int64_t i = i0 + lane;
    double t = 0.0;
    if (i < G) t = appd_term(w, G, i, appd_cum(w.P, rows, G, i), appd_cum(w.P, rows, G, i + 1), B);
    const int nl = (int)(G - i0 < 64 ? G - i0 : 64);
    for (int l = 0; l < nl; ++l) {
      total = total + __shfl(t, l, 64);
    }
  }
  if (lane == 0) obj[G - 1] = total;
}

// Least objective over G = 1..rows, ties to the smaller G (one block).
__global__ __launch_bounds__(1024) void appd_argmin_kernel(int64_t rows, const double* obj, int32_t* G_out) {
  __shared__ double sv[1024];
  __shared__ int64_t sg[1024];
  const int t = threadIdx.x;
  double best = 0.0;
  int64_t bg = -1;
  for (int64_t g = t; g < rows; g += 1024) {
    const double v = obj[g];
    if (bg < 0 || v < best) {
      best = v;
      bg = g;
    }
  }
  sv[t] = best;
  sg[t] = bg;
  __syncthreads();
  for (int h = 512; h > 0; h >>= 1) {
    if (t < h) {
      const double v = sv[t + h];
      const int64_t g = sg[t + h];
      if (g >= 0 && (sg[t] < 0 || v < sv[t] || (v == sv[t] && g < sg[t]))) {
        sv[t] = v;
        sg[t] = g;
      }
    }
    __syncthreads();
  }
  if (t == 0) *G_out = (int32_t)(sg[0] + 1);
}

// One wave per group g of the chosen plan (App. D: G from the device; fixed
// block size k: G = ceil(rows / k) and c_g = min(N - G, g (k - 1))).
__global__ __launch_bounds__(256) void plan_build_kernel(const float* rmin, int64_t rows, int B, int k, AppdWs w,
                                                         const int32_t* Gdev, int32_t* perm, float* scale,
                                                         float* zero, int32_t* group_off, SlotInfo* slot,
                                                         int32_t* num_groups) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  int64_t G = k > 0 ? (rows + k - 1) / k : (int64_t)*Gdev;
  G = G < 1 ? 1 : (G > rows ? rows : G);  // the search writes 1..rows; kept in range regardless
  if (g >= G) return;
  const int64_t small = rows - G;
  int64_t c0, c1;
  if (k > 0) {
    c0 = min(small, g * (int64_t)(k - 1));
    c1 = min(small, (g + 1) * (int64_t)(k - 1));
  } else {
    c0 = appd_cum(w.P, rows, G, g);
    c1 = appd_cum(w.P, rows, G, g + 1);
  }
  const int64_t n = c1 - c0, base = g + c0, size = n + 1;
  if (lane == 0) {
    group_off[g] = (int32_t)base;
    if (g == G - 1) {
      group_off[G] = (int32_t)rows;
      if (num_groups) *num_groups = (int32_t)G;
    }
  }
  const int32_t big = w.sigma[g];
  const float mn0 = rmin[big];
  if (n == 0) {
    if (lane == 0) {
      perm[base] = big;
      scale[base] = scale_from_range(w.Rs[g], B);
      zero[base] = mn0;
      slot[base] = SlotInfo{(int32_t)base, 1, 0.0f, 0.0f};
    }
    return;
  }
  const int64_t f = G + c0;
  const float lam2 = 2.0f * w.Ms[f];
  const double sk = sqrt((double)size);
  float s1, s2;
  group_scales(w.Rs[g], lam2, w.ca[g], w.cc[f], size, sk, B, s1, s2);
  const float alpha = (float)(1.0 / sk);
  const float oma = 1.0f - alpha;
  const double t1 = ((double)alpha * (double)s1) * (double)mn0;
  const double t2 = ((0.5 * (double)lam2) * (double)s2) * sk;
  const float cg = (float)(t1 - t2);
  const SlotInfo si{(int32_t)base, (int32_t)size, alpha, oma};
  for (int64_t j = lane; j < size; j += 64) {
    perm[base + j] = j == 0 ? big : w.sigma[f + j - 1];
    scale[base + j] = j == 0 ? s1 : s2;
    zero[base + j] = cg;
    slot[base + j] = si;
  }
}

static hipError_t launch_prep(const float* rmin, const float* rmax, int64_t rows, const AppdWs& w, hipStream_t s) {
  hipLaunchKernelGGL(appd_prep_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, rmin, rmax, rows, w);
  return hipGetLastError();
}

hipError_t launch_appd_search(const float* rmin, const float* rmax, int64_t rows, int bits, const AppdWs& w,
                              double* obj_out, int32_t* num_groups, hipStream_t s) {
  if (rows < 1 || rows > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipError_t e = launch_prep(rmin, rmax, rows, w, s);
  if (e != hipSuccess) return e;
  const int B = (1 << bits) - 1;
  double* obj = obj_out ? obj_out : w.obj;
  hipLaunchKernelGGL(appd_prefix_kernel, dim3(1), dim3(64), 0, s, rows, w);
  hipLaunchKernelGGL(appd_objective_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rows, B, w, obj);
  hipLaunchKernelGGL(appd_argmin_kernel, dim3(1), dim3(1024), 0, s, rows, obj, num_groups ? num_groups : w.G);
  return hipGetLastError();
}

hipError_t launch_general_plan(const float* rmin, const float* rmax, int64_t rows, int bits, int block_size,
                               const AppdWs& w, double* obj_out, int32_t* perm, float* scale, float* zero,
                               int32_t* group_off, SlotInfo* slot, int32_t* num_groups, hipStream_t s) {
  if (rows < 1 || rows > 0x7FFFFFFF || block_size < 0) return hipErrorInvalidValue;
  hipError_t e;
  if (block_size == 0) {
    e = launch_appd_search(rmin, rmax, rows, bits, w, obj_out, w.G, s);
  } else {
    e = launch_prep(rmin, rmax, rows, w, s);
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(plan_build_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rmin, rows,
                     (1 << bits) - 1, block_size, w, w.G, perm, scale, zero, group_off, slot, num_groups);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// tau: block (column tile of 256, chunk of 64 slots); the groups whose first
// slot lies in the chunk, one column per thread, their rows one at a time
// in slot order (each batch's loads issued before its additions).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bhq_tau_kernel(const float* x, int64_t rows, int64_t cols, const int32_t* perm,
                                                      const float* scale, const SlotInfo* slot, float* tau) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t s0 = (int64_t)blockIdx.y * 64;
  const int64_t s1 = s0 + 64 < rows ? s0 + 64 : rows;
  const int64_t cc = col < cols ? col : cols - 1;  // clamped: loads stay inside x, the store is skipped
  for (int64_t sb = s0; sb < s1; ++sb) {
    const SlotInfo si = slot[sb];
    if (si.base != sb || si.size < 2) continue;
    float S = 0.0f, v0 = 0.0f;
    int64_t p = 0;
    constexpr int U = 8;
    for (; p + U <= si.size; p += U) {
      float v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = scale[sb + p + u] * x[(int64_t)perm[sb + p + u] * cols + cc];
      if (p == 0) v0 = v[0];
#pragma unroll
      for (int u = 0; u < U; ++u) S = S + v[u];
    }
    for (; p < si.size; ++p) {
      const float v = scale[sb + p] * x[(int64_t)perm[sb + p] * cols + cc];
      if (p == 0) v0 = v;
      S = S + v;
    }
    const float m = si.alpha * S - v0;
    if (col < cols) tau[(sb >> 1) * cols + col] = __fdiv_rn(m, si.oma);
  }
}

hipError_t launch_bhq_tau(const float* x, int64_t rows, int64_t cols, const int32_t* perm, const float* scale,
                          const SlotInfo* slot, float* tau, hipStream_t s) {
  const int64_t cb = (cols + 255) / 256, rb = (rows + 63) / 64;
  if (cb > 0x7FFFFFFF || rb > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bhq_tau_kernel, dim3((unsigned)cb, (unsigned)rb), dim3(256), 0, s, x, rows, cols, perm, scale,
                     slot, tau);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// inverse: block (column tile of 256, chunk of 64 slots, row block b); the
// multi-row groups whose first slot lies in the chunk
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void bhq_inverse_kernel(InverseParams p) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t s0 = (int64_t)blockIdx.y * 64;
  const int64_t s1 = s0 + 64 < p.rows ? s0 + 64 : p.rows;
  const int64_t b = blockIdx.z;
  if (col >= p.cols) return;
  const double* T = p.T + (b * p.tstride) * p.ldt + col;
  for (int64_t sb = s0; sb < s1; ++sb) {
    const SlotInfo si = p.slot[sb];
    if (si.base != sb || si.size < 2) continue;
    double S = 0.0;
    for (int64_t q = 0; q < si.size; ++q) S = S + T[(sb + q) * p.ldt];
    const double T0 = T[sb * p.ldt];
    const double alpha = 1.0 / sqrt((double)si.size);
    const double tau = (alpha * S - T0) / (1.0 - alpha);
    const double up0 = (1.0 - alpha) * tau, dn = alpha * tau;
    for (int64_t q = 0; q < si.size; ++q) {
      const double t = T[(sb + q) * p.ldt];
      const double v = (q == 0 ? t + up0 : t - dn) / (double)p.scale[sb + q];
      const int64_t o = ((int64_t)p.perm[sb + q] * p.ostride + b * p.obstride) * p.ldo + col;
      const float f = (float)v;
      p.out[o] = (p.mask && !(p.mask[o] > 0.0f)) ? 0.0f : f;
    }
  }
}

hipError_t launch_bhq_inverse(const InverseParams& p, hipStream_t s) {
  const int64_t cb = (p.cols + 255) / 256, rb = (p.rows + 63) / 64;
  if (cb > 0x7FFFFFFF || rb > 65535 || p.nblk > 65535 || p.nblk < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bhq_inverse_kernel, dim3((unsigned)cb, (unsigned)rb, (unsigned)p.nblk), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace fqt
