// Gradient / activation / weight quantizers of the FQT backward on gfx950.
//
//   stats      per-row and per-tensor min / max by wavefront shuffles; each
//              block stores its partial, no atomics (min / max are exact in
//              any order)
//   finalize   PTQ scale s = B / R, zero z = min (Sec. 3.3); PSQ per row
//              (Sec. 4.1)
//   bhq plan   sort by row infinity norm, grouping and per-group scalars of
//              the block Householder quantizer (Sec. 4.2, App. C.4); the
//              search over every number of groups of App. D is in plan.hip
//   quant      one pass over the matrix: affine map or block Householder
//              transform, stochastic rounding from a Philox stream, int8
//              offset codes in natural and / or transposed layout with code
//              sums; optionally a second per-tensor quantizer (the
//              bifurcated Q_b1 of App. E) from the same read.
#include <math.h>

#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {

// ---------------------------------------------------------------------------
// reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Sums over the 64 lanes of each of 4 per-lane values v[0..3], all in
// vector registers: lanes 32 apart add up with one half-wave swap per pair
// (v[i] keeps the low half, v[i + 2] the high one), rows of 16 lanes with
// one row swap, then each row adds up by shifted adds within the row.  Lane
// l with l % 16 == 15 returns the sum of v[l / 16].
__device__ __forceinline__ int32_t wave_sum4(int32_t (&v)[4]) {
  int32_t h[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const auto sw = __builtin_amdgcn_permlane32_swap(v[i], v[i + 2], false, false);
    h[i] = (int32_t)sw[0] + (int32_t)sw[1];
  }
  const auto sw = __builtin_amdgcn_permlane16_swap(h[0], h[1], false, false);
  int32_t s = (int32_t)sw[0] + (int32_t)sw[1];
  // row_shr:n (source lane l - n of the same row; 0 where that leaves the row)
  s += __builtin_amdgcn_update_dpp(0, s, 0x111, 0xf, 0xf, false);
  s += __builtin_amdgcn_update_dpp(0, s, 0x112, 0xf, 0xf, false);
  s += __builtin_amdgcn_update_dpp(0, s, 0x114, 0xf, 0xf, false);
  s += __builtin_amdgcn_update_dpp(0, s, 0x118, 0xf, 0xf, false);
  return s;
}

// Block-wide (min, max, any-bad); every thread gets the result.
struct MinMax {
  float mn, mx;
  int bad;
};
template <int NW>
__device__ __forceinline__ MinMax block_minmax(float mn, float mx, int bad) {
  __shared__ float smn[NW], smx[NW];
  __shared__ int sbad[NW];
  mn = wave_min(mn);
  mx = wave_max(mx);
  bad = __any(bad) ? 1 : 0;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) {
    smn[w] = mn;
    smx[w] = mx;
    sbad[w] = bad;
  }
  __syncthreads();
  MinMax r{smn[0], smx[0], sbad[0]};
  for (int i = 1; i < NW; ++i) {
    r.mn = fminf(r.mn, smn[i]);
    r.mx = fmaxf(r.mx, smx[i]);
    r.bad |= sbad[i];
  }
  return r;
}

// ---------------------------------------------------------------------------
// stats: one launch over up to three tensors.  Every block reduces its chunk
// (a piece of a flat tensor, or a piece of one row) and stores the partial
// (min, max); a non-finite element turns the partial's min into NaN.  No
// atomics: the finalize block combines the partials.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void stats_kernel(StatsPlan sp) {
  int si = 0;
  while (si + 1 < sp.nseg && (int64_t)blockIdx.x >= sp.block_start[si + 1]) ++si;
  const StatsSeg g = sp.seg[si];
  const int64_t b = (int64_t)blockIdx.x - sp.block_start[si];
  const int64_t row = b / g.chunks;
  const int64_t c_begin = (b % g.chunks) * g.chunk;
  const int64_t c_end = (c_begin + g.chunk < g.cols) ? c_begin + g.chunk : g.cols;
  const float* xr = g.x + row * g.cols;
  float mn = INFINITY, mx = -INFINITY;
  int bad = 0;
  if ((g.cols & 3) == 0 && ((uintptr_t)g.x & 15) == 0) {
    const float4* x4 = reinterpret_cast<const float4*>(xr);
    // unrolled: a thread's loads are all in flight before the reductions
#pragma unroll 4
    for (int64_t i = (c_begin >> 2) + threadIdx.x; i < (c_end >> 2); i += blockDim.x) {
      const float4 v = x4[i];
      mn = fminf(fminf(mn, v.x), fminf(v.y, fminf(v.z, v.w)));
      mx = fmaxf(fmaxf(mx, v.x), fmaxf(v.y, fmaxf(v.z, v.w)));
      bad |= !(isfinite(v.x) && isfinite(v.y) && isfinite(v.z) && isfinite(v.w));
    }
  } else {
    for (int64_t i = c_begin + threadIdx.x; i < c_end; i += blockDim.x) {
      const float v = xr[i];
      mn = fminf(mn, v);
      mx = fmaxf(mx, v);
      bad |= !isfinite(v);
    }
  }
  const MinMax r = block_minmax<4>(mn, mx, bad);
  if (threadIdx.x == 0) {
    g.part[b] = make_float2(r.bad ? NAN : r.mn, r.mx);
    if (g.rmin) {
      g.rmin[row] = r.bad ? INFINITY : r.mn;
      g.rmax[row] = r.mx;
    }
  }
}

StatsSeg stats_flat_seg(const float* x, int64_t n) {
  StatsSeg g{};
  g.x = x;
  g.rows = 1;
  g.cols = n;
  g.chunk = 16384;
  g.chunks = (n + g.chunk - 1) / g.chunk;
  return g;
}

StatsSeg stats_rows_seg(const float* x, int64_t rows, int64_t cols) {
  StatsSeg g{};
  g.x = x;
  g.rows = rows;
  g.cols = cols;
  g.chunk = 8192;
  g.chunks = (cols + g.chunk - 1) / g.chunk;
  return g;
}


hipError_t launch_stats(StatsPlan sp, hipStream_t s) {
  int64_t total = 0;
  for (int i = 0; i < sp.nseg; ++i) {
    sp.block_start[i] = total;
    total += stats_partials(sp.seg[i]);
  }
  sp.block_start[sp.nseg] = total;
  if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(stats_kernel, dim3((unsigned)total), dim3(256), 0, s, sp);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// finalize: one block per statistics segment.  Block si combines segment
// si's partials into its per-tensor range (and, for the per-row segment, the
// per-row ranges), writes the PTQ scale / zero (Sec. 3.3) and PSQ per-row
// scales / zeros (Sec. 4.1) that derive from it, clears its share of the
// code-sum / rank arrays, and records a non-finite input or a range beyond
// float32 in status word si.
// ---------------------------------------------------------------------------
template <int NW>
__device__ void finalize_block(const FinalizePlan& fp, int si) {
  const int t = threadIdx.x;
  const int nparts = fp.nseg;
  for (int z = 0; z < fp.nzero; ++z) {
    const int64_t n = fp.zero_n[z];
    const int64_t lo = n * si / nparts, hi = n * (si + 1) / nparts;
    for (int64_t i = lo + t; i < hi; i += blockDim.x) fp.zero_i32[z][i] = 0;
  }
  if (si == 0)
    for (int w = fp.nseg + t; w < STATUS_WORDS; w += blockDim.x) fp.status[w] = 0u;
  const StatsSeg& g = fp.seg[si];
  float mn = INFINITY, mx = -INFINITY;
  int bad = 0;
  if (si == fp.row_seg && g.rmin) {
    // row ranges already stored by the stats blocks: a load-only reduction
    // (no stores in the loop, so the loads of several rows are in flight)
#pragma unroll 8
    for (int64_t r = t; r < g.rows; r += blockDim.x) {
      const float2 p = g.part[r];
      const float rmn = fminf(INFINITY, p.x);
      bad |= isnan(p.x) || !isfinite(p.y - rmn);
      mn = fminf(mn, rmn);
      mx = fmaxf(mx, p.y);
    }
  } else if (si == fp.row_seg) {
    for (int64_t r = t; r < g.rows; r += blockDim.x) {
      float rmn = INFINITY, rmx = -INFINITY;
      const float2* pr = g.part + r * g.chunks;
      // the row's partials eight at a time, all eight loads in flight
      int64_t c = 0;
      for (; c + 8 <= g.chunks; c += 8) {
        float2 q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) q[u] = pr[c + u];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (isnan(q[u].x)) bad = 1;
          rmn = fminf(rmn, q[u].x);
          rmx = fmaxf(rmx, q[u].y);
        }
      }
      for (; c < g.chunks; ++c) {
        const float2 p = pr[c];
        if (isnan(p.x)) bad = 1;
        rmn = fminf(rmn, p.x);
        rmx = fmaxf(rmx, p.y);
      }
      fp.rmin[r] = rmn;
      fp.rmax[r] = rmx;
      if (!isfinite(rmx - rmn)) bad = 1;
      mn = fminf(mn, rmn);
      mx = fmaxf(mx, rmx);
    }
  } else {
#pragma unroll 8
    for (int64_t i = t; i < stats_partials(g); i += blockDim.x) {
      const float2 p = g.part[i];
      if (isnan(p.x)) bad = 1;
      mn = fminf(mn, p.x);
      mx = fmaxf(mx, p.y);
    }
  }
  const MinMax r = block_minmax<NW>(mn, mx, bad);
  if (si == fp.row_seg) __syncthreads();  // per-row ranges of this block visible to all its threads
  for (int o = 0; o < fp.nout; ++o) {
    const ScaleOut& so = fp.out[o];
    if (so.seg != si) continue;
    const int B = (1 << so.bits) - 1;
    if (so.per_row == 2) {
      // per-tensor range R = max_i R_i, step s = B / R; row i takes the
      // largest e <= E with R_i 2^e <= R (power-of-two scalings are exact)
      const float* __restrict__ rmn = fp.rmin;
      const float* __restrict__ rmx = fp.rmax;
      float lmax = 0.0f;
#pragma unroll 8
      for (int64_t row = t; row < g.rows; row += blockDim.x) lmax = fmaxf(lmax, rmx[row] - rmn[row]);
      const float Rt = block_minmax<NW>(INFINITY, lmax, 0).mx;
      const float st = scale_from_range(Rt, B);
      const int E = min(4, 8 - so.bits);
      const double half = (double)(1 << (so.bits - 1));
      if (t == 0) so.tensor_scale[0] = st;
      // rows in batches of 4 per thread: loads first, then the stores
      for (int64_t r0 = t; r0 < g.rows; r0 += 4 * (int64_t)blockDim.x) {
        float lo[4], Ri[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int64_t row = r0 + k * (int64_t)blockDim.x;
          lo[k] = row < g.rows ? rmn[row] : 0.0f;
          Ri[k] = row < g.rows ? rmx[row] - lo[k] : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int64_t row = r0 + k * (int64_t)blockDim.x;
          if (row >= g.rows) break;
          int e = 0;
          while (e < E && Ri[k] * (float)(2 << e) <= Rt) ++e;
          float si = st * (float)(1 << e);
          si = si > FLT_MAX_F ? FLT_MAX_F : si;
          so.scale[row] = si;
          so.zero[row] = lo[k];
          so.shift[row] = (int8_t)(E - e);
          if (so.zeta) so.zeta[row] = half / (double)si + (double)lo[k];
        }
      }
    } else if (so.per_row) {
      for (int64_t row = t; row < g.rows; row += blockDim.x) {
        so.scale[row] = scale_from_range(fp.rmax[row] - fp.rmin[row], B);
        so.zero[row] = fp.rmin[row];
      }
    } else if (t == 0) {
      so.scale[0] = scale_from_range(r.mx - r.mn, B);
      so.zero[0] = r.mn;
    }
  }
  if (t == 0) fp.status[si] = (r.bad || !isfinite(r.mx - r.mn)) ? STATUS_NONFINITE : 0u;
}

__global__ __launch_bounds__(1024) void finalize_kernel(FinalizePlan fp) { finalize_block<16>(fp, blockIdx.x); }

hipError_t launch_finalize(const FinalizePlan& fp, hipStream_t s) {
  hipLaunchKernelGGL(finalize_kernel, dim3((unsigned)fp.nseg), dim3(1024), 0, s, fp);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// BHQ plan
// ---------------------------------------------------------------------------
BhqLayout bhq_layout(int64_t rows, int k) {
  BhqLayout L{};
  L.rows = rows;
  L.k = k;
  L.G = (rows + k - 1) / k;
  const int64_t small = rows - L.G;
  if (k > 1) {
    L.full = small / (k - 1);
    const int64_t rem = small % (k - 1);
    L.part = rem > 0 ? (int)(1 + rem) : 0;
  } else {
    L.full = 0;
    L.part = 0;
  }
  // Per-size scalars, IEEE double on the host: sqrt(size), float32(1/sqrt)
  // and the float32 difference 1 - alpha.
  L.sk_k = sqrt((double)k);
  L.a_k = (float)(1.0 / L.sk_k);
  L.oma_k = 1.0f - L.a_k;
  const int ps = L.part > 0 ? L.part : 1;
  L.sk_p = sqrt((double)ps);
  L.a_p = (float)(1.0 / L.sk_p);
  L.oma_p = 1.0f - L.a_p;
  L.inv_sk_k = 1.0 / L.sk_k;
  L.inv_sk_p = 1.0 / L.sk_p;
  return L;
}

constexpr int SORT_CH = 1024;  // keys per sorted chunk

static int64_t sort_pad(int64_t rows) { return (rows + SORT_CH - 1) / SORT_CH * SORT_CH; }

size_t bhq_plan_workspace(int64_t rows) {
  const int64_t np = sort_pad(rows);
  // sorted chunk keys (uint64), rank and sigma (int32 each)
  return (size_t)np * 8 + (size_t)rows * 4 * 2 + 256;
}

// key = (~bits(M_i) << 32) | i: ascending order = M descending, index ascending.
__device__ __forceinline__ uint64_t bhq_key(const float* rmin, const float* rmax, int64_t rows, int64_t i) {
  if (i >= rows) return ~0ull;
  const float M = fmaxf(fabsf(rmin[i]), fabsf(rmax[i]));
  return ((uint64_t)(~__float_as_uint(M)) << 32) | (uint64_t)(uint32_t)i;
}

// Keys of one 1024-row chunk, bitonic-sorted in LDS.
__device__ void bhq_sort_chunk(const float* rmin, const float* rmax, int64_t rows, uint64_t* sorted, int64_t chunk) {
  __shared__ uint64_t sk[SORT_CH];
  const int t = threadIdx.x;
  const int64_t base = chunk * SORT_CH;
  sk[t] = bhq_key(rmin, rmax, rows, base + t);
  sk[t + 512] = bhq_key(rmin, rmax, rows, base + t + 512);
  for (int size = 2; size <= SORT_CH; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      __syncthreads();
      const int i = (t / stride) * 2 * stride + (t % stride);
      const int j = i + stride;
      const bool asc = (i & size) == 0;
      const uint64_t a = sk[i], b = sk[j];
      if ((a > b) == asc) {
        sk[i] = b;
        sk[j] = a;
      }
    }
  }
  __syncthreads();
  sorted[base + t] = sk[t];
  sorted[base + t + 512] = sk[t + 512];
}

// The chunk sorts (blocks [0, nch)) and, when the row ranges come straight
// from the statistics kernel, the finalize step (block nch) in one launch.
__global__ __launch_bounds__(512) void bhq_sort_chunks_kernel(const float* rmin, const float* rmax, int64_t rows,
                                                              uint64_t* sorted, int64_t nch, FinalizePlan fp) {
  if ((int64_t)blockIdx.x < nch)
    bhq_sort_chunk(rmin, rmax, rows, sorted, blockIdx.x);
  else
    finalize_block<8>(fp, (int)(blockIdx.x - nch));
}

// rank(key) = number of keys below it, summed over every sorted chunk.
__global__ __launch_bounds__(256) void bhq_rank_kernel(const uint64_t* sorted, int32_t* rank) {
  __shared__ uint64_t sk[SORT_CH];
  const int t = threadIdx.x;
  const int64_t cbase = (int64_t)blockIdx.x * SORT_CH;
  const int64_t sbase = (int64_t)blockIdx.y * SORT_CH;
#pragma unroll
  for (int e = 0; e < 4; ++e) sk[t + 256 * e] = sorted[sbase + t + 256 * e];
  __syncthreads();
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint64_t key = sorted[cbase + t + 256 * e];
    if (key == ~0ull) continue;
    int lo = 0, hi = SORT_CH;  // first index with sk[idx] >= key
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (sk[mid] < key)
        lo = mid + 1;
      else
        hi = mid;
    }
    if (lo > 0) atomicAdd(&rank[(uint32_t)key], lo);
  }
}

__global__ void bhq_scatter_kernel(const int32_t* rank, int64_t rows, int32_t* sigma) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < rows) sigma[rank[i]] = (int32_t)i;
}

// First slot of group g under the fixed-block layout: full groups, then the
// partial one, then the one-row groups.
__device__ __forceinline__ int64_t bhq_group_base(const BhqLayout& L, int64_t g) {
  if (g < L.full) return g * L.k;
  if (g == L.full && L.part > 0) return L.full * L.k;
  return L.full * L.k + L.part + (g - L.full - (L.part > 0 ? 1 : 0));
}

// Slot of the row whose sorted position is r: the G largest rows lead the
// groups (position g -> group g, slot 0); the rest fill the groups' other
// slots k - 1 at a time, in sorted order.
__device__ __forceinline__ int64_t bhq_slot_of_rank(const BhqLayout& L, int64_t r) {
  if (r < L.G || L.k <= 1) return bhq_group_base(L, r);
  const int64_t q = r - L.G;
  const int64_t g = q / (L.k - 1);
  return bhq_group_base(L, g) + 1 + q % (L.k - 1);
}

// Sorted position of every row by counting, for up to RANK_MAX_ROWS rows:
// rank_i = #{j : M_j > M_i, or M_j = M_i and j < i}, the number of keys that
// sort before row i (M = row infinity norm compared as float32 bits, which
// orders the non-negative values exactly as bhq_key does).  The bits of all
// M are staged in LDS once, zero padded to a multiple of 256 (a padding key
// never counts: it exceeds no M, and equals M_i only at j > i).  Each wave
// owns 4 consecutive rows r0 .. r0 + 3, which share the 4-key group r0 / 4;
// its 64 lanes split the key groups, so one LDS read feeds 16 comparisons:
// keys before that group count when >= M_i, keys after it when > M_i, and
// the shared group takes the exact test.  The row is then stored at its slot
// of perm.  Blocks nrank .. nrank + nseg - 1 run the finalize step.
constexpr int RK_THREADS = 512;
constexpr int RK_ROWS = RK_THREADS / 64 * 4;
constexpr int64_t RANK_MAX_ROWS = 16384;  // keys staged in at most 64 KB of LDS

__host__ __device__ inline int64_t rank_pad(int64_t rows) { return (rows + 255) / 256 * 256; }

__global__ __launch_bounds__(RK_THREADS) void bhq_rank_perm_kernel(const float* rmin, const float* rmax, BhqLayout L,
                                                                   int32_t* perm, int64_t nrank, FinalizePlan fp) {
  if ((int64_t)blockIdx.x >= nrank) {
    finalize_block<RK_THREADS / 64>(fp, (int)(blockIdx.x - nrank));
    return;
  }
  extern __shared__ uint4 rk_lds[];
  uint32_t* mk = reinterpret_cast<uint32_t*>(rk_lds);
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int rows = (int)L.rows;
  const int npad = (int)rank_pad(rows);
  // all loads of a round in flight before the LDS stores: the loads are
  // unconditional (indices past the end are clamped to the last row and
  // their keys replaced below), since a load under a branch makes the
  // compiler wait for each one before issuing the next
  constexpr int U = 16;
  for (int base = 0; base < npad; base += RK_THREADS * U) {
    float lo[U], hi[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = base + t + u * RK_THREADS;
      const int ec = e < rows ? e : rows - 1;
      lo[u] = rmin[ec];
      hi[u] = rmax[ec];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int e = base + t + u * RK_THREADS;
      if (e < npad) mk[e] = e < rows ? __float_as_uint(fmaxf(fabsf(lo[u]), fabsf(hi[u]))) : 0u;
    }
  }
  __syncthreads();
  const int r0 = (int)blockIdx.x * RK_ROWS + wave * 4;
  const int gs = r0 / 4;
  uint32_t mu[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) mu[q] = r0 + q < rows ? mk[r0 + q] : 0xFFFFFFFFu;
  int cnt[4] = {0, 0, 0, 0};
  const int ng = npad / 4;
  int gi = lane;
#pragma unroll 2
  for (; gi < gs; gi += 64) {
    const uint4 v = rk_lds[gi];
#pragma unroll
    for (int q = 0; q < 4; ++q) cnt[q] += (v.x >= mu[q]) + (v.y >= mu[q]) + (v.z >= mu[q]) + (v.w >= mu[q]);
  }
  if (gi == gs && gs < ng) {
    // key 4 gs + e sorts before row r0 + q when its M is larger, or equal with e < q
    const uint4 v = rk_lds[gi];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      cnt[q] += (v.x > mu[q] || (v.x == mu[q] && 0 < q)) + (v.y > mu[q] || (v.y == mu[q] && 1 < q)) +
                (v.z > mu[q] || (v.z == mu[q] && 2 < q)) + (v.w > mu[q] || (v.w == mu[q] && 3 < q));
    gi += 64;
  }
#pragma unroll 2
  for (; gi < ng; gi += 64) {
    const uint4 v = rk_lds[gi];
#pragma unroll
    for (int q = 0; q < 4; ++q) cnt[q] += (v.x > mu[q]) + (v.y > mu[q]) + (v.z > mu[q]) + (v.w > mu[q]);
  }
  // lane 16 q + 15 gets the count of row r0 + q
  const int c = wave_sum4(cnt);
  const int q = lane >> 4;
  if ((lane & 15) == 15 && r0 + q < rows) perm[bhq_slot_of_rank(L, c)] = r0 + q;
}

// One group of a fixed-block plan, one wave (lane j handles the group's slot
// j + 1): the per-slot scale d_p and zero (c_g, or the row min for a one-row
// group).  FROM_PERM: perm already holds the rows in slot order
// (bhq_rank_perm_kernel); otherwise the rows come from sigma (sorted order)
// and are stored into perm here.
template <bool FROM_PERM>
__device__ void bhq_group(const float* rmin, const float* rmax, const int32_t* sigma, const BhqLayout& L, int B,
                          int64_t g, int32_t* perm, float* scale, float* zero, int32_t* group_off) {
  const int lane = threadIdx.x;
  const int k = L.k;
  int kg;
  int64_t base;
  if (g < L.full) {
    kg = k;
    base = g * k;
  } else if (g == L.full && L.part > 0) {
    kg = L.part;
    base = L.full * k;
  } else {
    kg = 1;
    base = L.full * k + L.part + (g - L.full - (L.part > 0 ? 1 : 0));
  }
  if (group_off && lane == 0) {
    group_off[g] = (int32_t)base;
    if (g == L.G - 1) group_off[L.G] = (int32_t)L.rows;
  }
  const int32_t big = FROM_PERM ? perm[base] : sigma[g];
  const float mn0 = rmin[big];
  const float mx0 = rmax[big];
  if (kg == 1) {
    const float s0 = scale_from_range(mx0 - mn0, B);
    if (lane == 0) {
      if (!FROM_PERM) perm[base] = big;
      scale[base] = s0;
      zero[base] = mn0;
    }
    return;
  }
  const int64_t tail = L.G + g * (int64_t)(k - 1);
  int32_t r = -1;
  float M = 0.0f;
  if (lane < kg - 1) {
    r = FROM_PERM ? perm[base + 1 + lane] : sigma[tail + lane];
    M = fmaxf(fabsf(rmin[r]), fabsf(rmax[r]));
  }
  const float m2 = wave_max(M);
  const float lam2 = 2.0f * m2;
  const float lam1 = mx0 - mn0;
  const double sk = (kg == k) ? L.sk_k : L.sk_p;
  const float alpha = (kg == k) ? L.a_k : L.a_p;
  float s1, s2;
  group_scales(lam1, lam2, cbrt_rn(lam1), cbrt_rn(lam2), kg, sk, B, s1, s2);
  const double t1 = ((double)alpha * (double)s1) * (double)mn0;
  const double t2 = ((0.5 * (double)lam2) * (double)s2) * sk;
  const float cg = (float)(t1 - t2);
  if (lane == 0) {
    if (!FROM_PERM) perm[base] = big;
    scale[base] = s1;
    zero[base] = cg;
  }
  if (lane < kg - 1) {
    if (!FROM_PERM) perm[base + 1 + lane] = r;
    scale[base + 1 + lane] = s2;
    zero[base + 1 + lane] = cg;
  }
}

template <bool FROM_PERM>
__global__ __launch_bounds__(64) void bhq_groups_kernel(const float* rmin, const float* rmax, const int32_t* sigma,
                                                        BhqLayout L, int B, int32_t* perm, float* scale, float* zero,
                                                        int32_t* group_off, int32_t* num_groups) {
  bhq_group<FROM_PERM>(rmin, rmax, sigma, L, B, blockIdx.x, perm, scale, zero, group_off);
  if (num_groups && blockIdx.x == 0 && threadIdx.x == 0) *num_groups = (int32_t)L.G;
}

BhqPlanWs bhq_plan_carve(void* plan_ws, int64_t rows) {
  const int64_t np = sort_pad(rows);
  char* w = static_cast<char*>(plan_ws);
  BhqPlanWs p{};
  p.sorted = reinterpret_cast<uint64_t*>(w);
  p.rank = reinterpret_cast<int32_t*>(p.sorted + np);
  p.sigma = p.rank + rows;
  return p;
}

hipError_t launch_bhq_plan(const float* rmin, const float* rmax, const BhqLayout& L, int bits, void* plan_ws,
                           int32_t* perm, float* scale, float* zero, int32_t* group_off, int32_t* num_groups,
                           const FinalizePlan* fin, hipStream_t s) {
  const int64_t rows = L.rows;
  const int64_t np = sort_pad(rows);
  const int64_t nch = np / SORT_CH;
  if (nch > 65535 || L.G > 0x7FFFFFFF) return hipErrorInvalidValue;
  const BhqPlanWs w = bhq_plan_carve(plan_ws, rows);
  const FinalizePlan none{};
  if (rows <= RANK_MAX_ROWS) {
    // two launches: positions by counting (plus the finalize block), then the groups
    const int64_t nrank = (rows + RK_ROWS - 1) / RK_ROWS;
    const size_t lds = (size_t)rank_pad(rows) * 4;
    hipLaunchKernelGGL(bhq_rank_perm_kernel, dim3((unsigned)(nrank + (fin ? fin->nseg : 0))), dim3(RK_THREADS), lds,
                       s, rmin, rmax, L, perm, nrank, fin ? *fin : none);
    hipLaunchKernelGGL(bhq_groups_kernel<true>, dim3((unsigned)L.G), dim3(64), 0, s, rmin, rmax, w.sigma, L,
                       (1 << bits) - 1, perm, scale, zero, group_off, num_groups);
    return hipGetLastError();
  }
  // w.rank must be zero before the rank kernel: the finalize step clears it,
  // either before this call or (fin) in the sort launch
  hipLaunchKernelGGL(bhq_sort_chunks_kernel, dim3((unsigned)(nch + (fin ? fin->nseg : 0))), dim3(512), 0, s, rmin, rmax, rows,
                     w.sorted, nch, fin ? *fin : none);
  hipLaunchKernelGGL(bhq_rank_kernel, dim3((unsigned)nch, (unsigned)nch), dim3(256), 0, s, w.sorted, w.rank);
  hipLaunchKernelGGL(bhq_scatter_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, w.rank, rows,
                     w.sigma);
  hipLaunchKernelGGL(bhq_groups_kernel<false>, dim3((unsigned)L.G), dim3(64), 0, s, rmin, rmax, w.sigma, L,
                     (1 << bits) - 1, perm, scale, zero, group_off, num_groups);
  return hipGetLastError();
}

// Rows in sorted order (M descending, ties by row index) into sigma: the
// counting rank for up to RANK_MAX_ROWS rows (its k = 1 layout stores each
// row at its sorted position), else chunk sorts, rank merge and scatter.
hipError_t launch_bhq_sort(const float* rmin, const float* rmax, int64_t rows, void* plan_ws, int32_t* sigma,
                           const FinalizePlan* fin, hipStream_t s) {
  const int64_t nch = sort_pad(rows) / SORT_CH;
  if (nch > 65535) return hipErrorInvalidValue;
  const FinalizePlan none{};
  if (rows <= RANK_MAX_ROWS) {
    const BhqLayout L1 = bhq_layout(rows, 1);
    const int64_t nrank = (rows + RK_ROWS - 1) / RK_ROWS;
    hipLaunchKernelGGL(bhq_rank_perm_kernel, dim3((unsigned)(nrank + (fin ? fin->nseg : 0))), dim3(RK_THREADS),
                       (size_t)rank_pad(rows) * 4, s, rmin, rmax, L1, sigma, nrank, fin ? *fin : none);
    return hipGetLastError();
  }
  // the rank array must be zero here: the finalize step clears it (before
  // this call, or in the sort launch with fin)
  const BhqPlanWs w = bhq_plan_carve(plan_ws, rows);
  hipLaunchKernelGGL(bhq_sort_chunks_kernel, dim3((unsigned)(nch + (fin ? fin->nseg : 0))), dim3(512), 0, s, rmin,
                     rmax, rows, w.sorted, nch, fin ? *fin : none);
  hipLaunchKernelGGL(bhq_rank_kernel, dim3((unsigned)nch, (unsigned)nch), dim3(256), 0, s, w.sorted, w.rank);
  hipLaunchKernelGGL(bhq_scatter_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, w.rank, rows, sigma);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// quant: tile = 64 slots x 256 columns, 4 waves of 16 slots, 4 columns / lane
// ---------------------------------------------------------------------------
constexpr int QT_SLOTS = 64;
constexpr int QT_COLS = 256;
constexpr int QT_ROWS_PER_WAVE = 16;

// Offset codes of four consecutive columns of one row from transformed values
// y, in the top-byte form of sr_top / rne_top: stochastic rounding with the
// Philox blocks of elements e0 .. e0 + 3 (VEC: the argument is the block
// index e0 / 4 of the one block that holds all four) or round-half-even.
template <bool VEC>
__device__ __forceinline__ void sr4(const float (&y)[4], uint64_t e0, uint64_t seed, uint32_t stream, float Bf,
                                    uint32_t hoff, int32_t (&t)[4]) {
  if constexpr (VEC) {
    const u32x4 o = philox_of_block(e0, seed, stream);
    t[0] = sr_top(y[0], o.x, Bf, hoff);
    t[1] = sr_top(y[1], o.y, Bf, hoff);
    t[2] = sr_top(y[2], o.z, Bf, hoff);
    t[3] = sr_top(y[3], o.w, Bf, hoff);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t e = e0 + j;
      const u32x4 o = philox_block(e, seed, stream);
      t[j] = sr_top(y[j], philox_word(o, (int)(e & 3)), Bf, hoff);
    }
  }
}
__device__ __forceinline__ void rne4(const float (&y)[4], float Bf, uint32_t hoff, int32_t (&t)[4]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) t[j] = rne_top(y[j], Bf, hoff);
}

// Tile = 64 slots x 256 columns; 4 waves of 16 slots; 4 columns per lane.
// The loaded tile stays in registers; each row is then finished in one step
// (transform, both quantizers, packing, code sums) so its data dies early.
// VEC: cols % 4 == 0 (float4 loads, one Philox block per lane and row).
// TRANS: the primary codes go out transposed ([cols, rows], column sums)
// instead of in natural order ([rows, cols], row sums).
// One 64 x 256 tile: column tile bx, slot tile by.
// H2: the second (transposed, stochastic) quantizer of the same rows, Q_b1:
// 0 none, 1 per tensor, 2 per row with power-of-two shifted codes.
template <int MODE, int K, int H2, bool VEC, bool TRANS, bool SD = false>
__device__ __forceinline__ void quant_tile(const QuantParams& p, int64_t bx, int64_t by) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: slot bookkeeping stays scalar
  const int64_t tile0 = by * QT_SLOTS;
  const int64_t slot0 = tile0 + wave * QT_ROWS_PER_WAVE;
  const int64_t c0 = bx * QT_COLS + lane * 4;
  const int64_t rows = p.rows, cols = p.cols;
  const int B = (1 << p.bits) - 1;
  const int half = 1 << (p.bits - 1);
  const bool lane_ok = c0 < cols;
  // per-row tests as 32-bit counts from slot0, worked out once per wave: row
  // r of the wave lies inside the matrix iff r < nok, in a full block
  // Householder group iff r < nk1, in the partial group iff nk1 <= r < nk2
  // (64-bit comparisons per row would go through vector compares and lane
  // masks)
  auto clamp16 = [](int64_t v) { return (int)(v < 0 ? 0 : (v > QT_ROWS_PER_WAVE ? QT_ROWS_PER_WAVE : v)); };
  const int nok = clamp16(rows - slot0);
  int nk1 = 0, nk2 = 0;
  if constexpr (MODE == QM_BHQ && K != 0) {
    const int64_t end1 = p.L.full * (int64_t)p.L.k;
    nk1 = clamp16(end1 - slot0);
    nk2 = clamp16(end1 + (p.L.part > 0 ? p.L.part : 0) - slot0);
  }
  // bhq_slot_kind of row r of the wave
  auto kind_of = [&](int r) { return r < nk1 ? 1 : (r < nk2 ? 2 : 0); };

  __shared__ float s_part[4][QT_COLS];   // per-wave partial group sums (BHQ, K >= 16)
  __shared__ float s_v0[4][QT_COLS];     // v of a group's first slot (BHQ, K >= 16)
  __shared__ int s_csum[2][4][QT_COLS];  // per-wave column code sums (transposed outputs)

  // source row of each of the wave's 16 slots, lane l holding slot l: one
  // load, so that the 16 row loads below issue back to back
  int32_t lrow = 0;
  {
    const int64_t sl = slot0 + (lane & 15);
    if (sl < rows) lrow = p.perm ? p.perm[sl] : (int32_t)sl;
  }
  auto src_row = [&](int r) { return __builtin_amdgcn_readlane(lrow, r); };

  // ---- load 16 rows x 4 columns
  float g[QT_ROWS_PER_WAVE][4];
#pragma unroll
  for (int r = 0; r < QT_ROWS_PER_WAVE; ++r) {
    const bool ok = r < nok;
    const int32_t row = src_row(r);
    const float* xr = p.x + (int64_t)row * cols;
    if constexpr (VEC) {
      if (ok && lane_ok) {
        const float4 v = *reinterpret_cast<const float4*>(xr + c0);
        g[r][0] = v.x;
        g[r][1] = v.y;
        g[r][2] = v.z;
        g[r][3] = v.w;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) g[r][j] = 0.0f;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) g[r][j] = (ok && c0 + j < cols) ? xr[c0 + j] : 0.0f;
    }
  }

  // per-slot scale and zero of the wave's 16 rows, lane l holding row l:
  // loaded with the tile, so that the row loop reads them from registers
  // instead of loads that would queue behind its code stores
  float lscale = 1.0f, lzero = 0.0f;
  if constexpr (MODE == QM_ROW || (MODE == QM_BHQ && K != 0)) {
    const int64_t sl = slot0 + (lane & 15);
    if (sl < rows) {
      lscale = p.scale[sl];
      lzero = p.zero[sl];
    }
  }
  auto row_scale = [&](int r) { return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lscale), r)); };
  auto row_zero = [&](int r) { return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, lzero), r)); };
  // ---- block Householder (K >= 16): a group spans K / 16 waves.  Its column
  // sum adds the slots one at a time in slot order, so the running sum is
  // handed from wave to wave through LDS: in step i the i-th wave of every
  // group continues the sum its predecessor left (K / 16 barrier steps).
  float ta[4] = {0.0f, 0.0f, 0.0f, 0.0f}, tb[4] = {0.0f, 0.0f, 0.0f, 0.0f};  // alpha tau, (1 - alpha) tau
  if constexpr (MODE == QM_BHQ && K >= 16) {
    const BhqLayout& L = p.L;
    constexpr int nw = K / 16;            // waves per group
    const int w0 = (wave / nw) * nw;      // first wave of this wave's group
    for (int step = 0; step < nw; ++step) {
      if (wave - w0 == step) {
        float P[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        if (step > 0) {
#pragma unroll
          for (int j = 0; j < 4; ++j) P[j] = s_part[wave - 1][lane * 4 + j];
        }
#pragma unroll
        for (int r = 0; r < QT_ROWS_PER_WAVE; ++r) {
          const bool multi = kind_of(r) != 0;
          const float d = row_scale(r);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float v = d * g[r][j];
            P[j] = P[j] + (multi ? v : 0.0f);
            if (r == 0 && step == 0) s_v0[wave][lane * 4 + j] = v;
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) s_part[wave][lane * 4 + j] = P[j];
      }
      __syncthreads();
    }
    const int64_t gfirst = tile0 + w0 * 16;
    const int gkind = gfirst < rows ? bhq_slot_kind(L, gfirst) : 0;
    const float alpha = gkind == 2 ? L.a_p : L.a_k;
    const float oma = gkind == 2 ? L.oma_p : L.oma_k;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float S = s_part[w0 + nw - 1][lane * 4 + j];
      const float m = alpha * S - s_v0[w0][lane * 4 + j];
      const float tau = __fdiv_rn(m, oma);
      ta[j] = alpha * tau;
      tb[j] = oma * tau;
    }
  }

  // ---- finish row by row.  Offset codes are carried in the top-byte form
  // (sr_top / rne_top), packed four to a word with byte permutes (natural:
  // four columns of one row; transposed: four rows of one column) and summed
  // with int8 dot products of the packed words.
  const float Bf = (float)B;
  const uint32_t hoff = (uint32_t)half << 24;
  // bytes of the packed natural word that belong to columns inside the matrix
  uint32_t colmask = 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    if (c0 + j < cols) colmask |= 0xFFu << (8 * j);
  // pixel-major natural codes: this lane's four columns lie in one pixel of pm_o channels
  // natural codes of row r go to nat0 + r * nat_step (bytes; with packed
  // codes to nat0 / 2 + r * nat_step / 2, cols % 4 == 0)
  const int64_t nat0 = p.pm_o > 0 ? (c0 / p.pm_o) * rows * p.pm_o + c0 % p.pm_o + slot0 * p.pm_o : slot0 * cols + c0;
  const int64_t nat_step = p.pm_o > 0 ? p.pm_o : cols;
  int32_t rs4[4];                // per-lane partial row sums of the natural codes, 4 rows at a time
  uint32_t tq[4][4], tq2[4][4];  // transposed codes: [column][4 words of 16 slots]; rows past the end stay 0
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      tq[j][w] = 0u;
      tq2[j][w] = 0u;
    }
  const float s_t = (MODE == QM_TENSOR) ? p.scale[0] : 0.0f;
  const float z_t = (MODE == QM_TENSOR) ? p.zero[0] : 0.0f;
  float Bf2 = 0.0f, s2 = 0.0f, z2 = 0.0f;
  uint32_t hoff2 = 0u;
  if constexpr (H2 != 0) {
    Bf2 = (float)((1 << p.bits2) - 1);
    hoff2 = (uint32_t)(1 << (p.bits2 - 1)) << 24;
  }
  if constexpr (H2 == 1) {
    s2 = p.scale2[0];
    z2 = p.zero2[0];
  }
#pragma unroll
  for (int r = 0; r < QT_ROWS_PER_WAVE; ++r) {
    const int64_t slot = slot0 + r;
    const bool ok = r < nok;
    float y[4];
    if constexpr (MODE == QM_TENSOR) {
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = s_t * (g[r][j] - z_t);
    } else if constexpr (MODE == QM_ROW) {
      const float s = row_scale(r);
      const float z = row_zero(r);
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = s * (g[r][j] - z);
    } else if constexpr (K == 0) {
      // general plan: the group's rank-1 term comes precomputed per column
      const SlotInfo si = ok ? p.slot[slot] : SlotInfo{0, 1, 0.0f, 0.0f};
      const float d = ok ? p.scale[slot] : 1.0f;
      const float c = ok ? p.zero[slot] : 0.0f;
      if (si.size > 1) {
        float t[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        const float* tp = p.tau + (int64_t)(si.base >> 1) * cols + c0;
        if constexpr (VEC) {
          if (lane_ok) {
            const float4 v = *reinterpret_cast<const float4*>(tp);
            t[0] = v.x;
            t[1] = v.y;
            t[2] = v.z;
            t[3] = v.w;
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (c0 + j < cols) t[j] = tp[j];
        }
        const bool first = slot == si.base;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float v = d * g[r][j];
          const float Y = first ? v + si.oma * t[j] : v - si.alpha * t[j];
          y[j] = Y - c;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = d * (g[r][j] - c);
      }
    } else {
      const BhqLayout& L = p.L;
      const int kind = kind_of(r);
      const float d = row_scale(r);
      const float c = row_zero(r);
      if constexpr (K > 1 && K < 16) {
        // groups of K rows inside this wave: their sums from the registers
        if (r % K == 0) {
          const int gkind = kind_of(r);
          const float alpha = gkind == 2 ? L.a_p : L.a_k;
          const float oma = gkind == 2 ? L.oma_p : L.oma_k;
          float S[4] = {0.0f, 0.0f, 0.0f, 0.0f}, v0[4];
#pragma unroll
          for (int rr = 0; rr < K; ++rr) {
            const bool multi = kind_of(r + rr) != 0;
            const float dr = row_scale(r + rr);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float v = dr * g[r + rr][j];
              S[j] = S[j] + (multi ? v : 0.0f);
              if (rr == 0) v0[j] = v;
            }
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float m = alpha * S[j] - v0[j];
            const float tau = __fdiv_rn(m, oma);
            ta[j] = alpha * tau;
            tb[j] = oma * tau;
          }
        }
      }
      // one branch per row (the test is the same for the four columns)
      if (K > 1 && kind != 0) {
        // slot0 is a multiple of 16, so a group of K >= 16 starts at row 0
        // of a wave
        const bool first = K >= 16 ? (r == 0 && (wave * QT_ROWS_PER_WAVE) % (K > 1 ? K : 1) == 0)
                                   : (r % (K > 1 ? K : 1) == 0);
        if (first) {
#pragma unroll
          for (int j = 0; j < 4; ++j) y[j] = (d * g[r][j] + tb[j]) - c;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) y[j] = (d * g[r][j] - ta[j]) - c;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = d * (g[r][j] - c);
      }
    }
    // logical element index of the row's first column (VEC: its Philox
    // block index, row * cols / 4 + c0 / 4 with cols % 4 == c0 % 4 == 0)
    uint64_t e0;
    if constexpr (VEC) {
      // the row's product stays on the scalar unit; one 64-bit vector add
      const uint64_t rb = (uint64_t)(uint32_t)src_row(r) * (uint64_t)(cols >> 2);
      const uint32_t rlo = __builtin_amdgcn_readfirstlane((uint32_t)rb);
      const uint32_t rhi = __builtin_amdgcn_readfirstlane((uint32_t)(rb >> 32));
      e0 = (((uint64_t)rhi << 32) | rlo) + (uint64_t)(c0 >> 2);
    } else {
      e0 = (uint64_t)(uint32_t)src_row(r) * (uint64_t)cols + (uint64_t)c0;
    }
    if constexpr (SD) {
      // seed batch: the same transformed values rounded under keys seed + b,
      // b < nseeds; per element the sum of the codes and of their squares
      if (ok && lane_ok) {
        int32_t c1[4] = {0, 0, 0, 0}, c2[4] = {0, 0, 0, 0};
        for (int b = 0; b < p.nseeds; ++b) {
          int32_t tb[4];
          sr4<VEC>(y, e0, p.seed + (uint64_t)b, p.stream, Bf, hoff, tb);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int32_t c = (tb[j] >> 24) + half;
            c1[j] += c;
            c2[j] += c * c;
          }
        }
        const int64_t o = slot * cols + c0;
        *reinterpret_cast<int4*>(p.sum_c + o) = make_int4(c1[0], c1[1], c1[2], c1[3]);
        *reinterpret_cast<int4*>(p.sum_c2 + o) = make_int4(c2[0], c2[1], c2[2], c2[3]);
      }
      continue;
    }
    int32_t t[4];
    // with a second quantizer the first is stochastic too (launch_quant checks)
    if (H2 != 0 || p.stoch)
      sr4<VEC>(y, e0, p.seed, p.stream, Bf, hoff, t);
    else
      rne4(y, Bf, hoff, t);
    if constexpr (MODE == QM_ROW) {
      if (p.shift && ok) {
        const int sh = p.shift[slot];
#pragma unroll
        for (int j = 0; j < 4; ++j) t[j] = shift_top(t[j], sh);
      }
    }
    if constexpr (H2 != 0) {
      // Q_b1 of the same row: always stochastic, its own Philox stream (the
      // counter and key are shared, so the compiler shares the first two
      // rounds' products with the call above)
      float s2r = s2, z2r = z2;
      int sh2 = 0;
      if constexpr (H2 == 2) {
        if (ok) {
          const int32_t sr = src_row(r);
          s2r = p.scale2[sr];
          z2r = p.zero2[sr];
          sh2 = p.shift2[sr];
        }
      }
      float y2[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) y2[j] = s2r * (g[r][j] - z2r);
      int32_t t2[4];
      sr4<VEC>(y2, e0, p.seed, p.stream2, Bf2, hoff2, t2);
      if constexpr (H2 == 2) {
#pragma unroll
        for (int j = 0; j < 4; ++j) t2[j] = shift_top(t2[j], sh2);
      }
      if (ok) {
#pragma unroll
        for (int j = 0; j < 4; ++j) tq2[j][r >> 2] = insert_top(tq2[j][r >> 2], t2[j], r & 3);
      }
    }
    if constexpr (!TRANS) {
      const uint32_t w = pack_top4(t[0], t[1], t[2], t[3]);
      if (p.q_nat && ok && lane_ok) {
        int8_t* dst = p.q_nat + nat0 + r * nat_step;
        if (VEC && p.packed) {
          // codes of at most 4 bits, two per byte: the nibble of column 2i is
          // the low half of byte i, the code stored as q + 8 in [0, 15]
          const uint32_t nb = (w ^ 0x08080808u) & 0x0F0F0F0Fu;
          const uint32_t x2 = nb | (nb >> 4);
          const uint32_t pk = __builtin_amdgcn_perm(0u, x2, 0x0c0c0200u);  // bytes 0 and 2 of x2
          *reinterpret_cast<uint16_t*>(p.q_nat + nat0 / 2 + r * (nat_step / 2)) = (uint16_t)pk;
        } else if constexpr (VEC) {
          *reinterpret_cast<uint32_t*>(dst) = w;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (c0 + j < cols) dst[j] = (int8_t)(t[j] >> 24);
        }
      }
      rs4[r & 3] = sum4_i8(w & colmask, 0);
      // row sums of the natural codes: one exchange tree per 4 rows
      if ((r & 3) == 3 && p.sum_nat) {
        const int32_t t = wave_sum4(rs4);
        const int rl = (r - 3) + (lane >> 4);
        if ((lane & 15) == 15 && rl < nok) atomicAdd(p.sum_nat + slot0 + rl, t);
      }
    } else if (ok) {
#pragma unroll
      for (int j = 0; j < 4; ++j) tq[j][r >> 2] = insert_top(tq[j][r >> 2], t[j], r & 3);
    }
  }

  // ---- transposed stores: 16 consecutive slots per column
  const bool tvec = ((rows & 15) == 0) && nok == QT_ROWS_PER_WAVE;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t col = c0 + j;
    if (col >= cols) continue;
    if constexpr (TRANS) {
      int8_t* dst = p.q_t + col * rows + slot0;
      if (tvec) {
        *reinterpret_cast<uint4*>(dst) = make_uint4(tq[j][0], tq[j][1], tq[j][2], tq[j][3]);
      } else {
#pragma unroll
        for (int r = 0; r < QT_ROWS_PER_WAVE; ++r)
          if (r < nok) dst[r] = (int8_t)((tq[j][r >> 2] >> (8 * (r & 3))) & 255);
      }
    }
    if constexpr (H2 != 0) {
      int8_t* dst = p.q2_t + col * rows + slot0;
      if (tvec) {
        *reinterpret_cast<uint4*>(dst) = make_uint4(tq2[j][0], tq2[j][1], tq2[j][2], tq2[j][3]);
      } else {
#pragma unroll
        for (int r = 0; r < QT_ROWS_PER_WAVE; ++r)
          if (r < nok) dst[r] = (int8_t)((tq2[j][r >> 2] >> (8 * (r & 3))) & 255);
      }
    }
  }

  // ---- column sums of the transposed outputs: reduce the 4 waves in LDS
  if ((TRANS && p.sum_t) || (H2 != 0 && p.sum2_t)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int32_t cs = 0, cs2 = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if constexpr (TRANS) cs = sum4_i8(tq[j][w], cs);
        if constexpr (H2 != 0) cs2 = sum4_i8(tq2[j][w], cs2);
      }
      s_csum[0][wave][lane * 4 + j] = cs;
      s_csum[1][wave][lane * 4 + j] = cs2;
    }
    __syncthreads();
    const int c = threadIdx.x;  // 256 threads = 256 columns of the tile
    const int64_t col = bx * QT_COLS + c;
    if (col < cols) {
      if (TRANS && p.sum_t) {
        const int t = s_csum[0][0][c] + s_csum[0][1][c] + s_csum[0][2][c] + s_csum[0][3][c];
        atomicAdd(p.sum_t + col, t);
      }
      if (H2 != 0 && p.sum2_t) {
        const int t = s_csum[1][0][c] + s_csum[1][1][c] + s_csum[1][2][c] + s_csum[1][3][c];
        atomicAdd(p.sum2_t + col, t);
      }
    }
  }
}


template <int MODE, int K, int H2, bool VEC, bool TRANS>
__global__ __launch_bounds__(256) void quant_tile_kernel(QuantParams p) {
  quant_tile<MODE, K, H2, VEC, TRANS>(p, blockIdx.x, blockIdx.y);
}

// Two independent per-tensor transposed quantizations in one launch (Q_f(X)
// and Q_theta(W)): blocks [0, nb0) tile the first, the rest the second, each
// over a row-major grid of ct column tiles.
template <bool VEC>
__global__ __launch_bounds__(256) void quant_tile2_kernel(QuantParams p0, QuantParams p1, int64_t nb0, int64_t ct0,
                                                          int64_t ct1) {
  const int64_t b = blockIdx.x;
  if (b < nb0)
    quant_tile<QM_TENSOR, 0, 0, VEC, true>(p0, b % ct0, b / ct0);
  else
    quant_tile<QM_TENSOR, 0, 0, VEC, true>(p1, (b - nb0) % ct1, (b - nb0) / ct1);
}

// The gradient pass (natural codes plus the transposed Q_b1) and the two
// per-tensor transposed passes (Q_f(X), Q_theta(W)) in one grid.  Every
// period-th block (while they last) is an X / W tile, so that those
// memory-light tiles interleave with the arithmetic-heavy gradient tiles;
// the other blocks take the gradient tiles in order.
template <int MODE, int K, int H2>
__global__ __launch_bounds__(256) void quant_fused_kernel(QuantParams pg, QuantParams px, QuantParams pw, int64_t nbx,
                                                          int64_t nbw, int64_t period, int64_t ctg, int64_t ctx,
                                                          int64_t ctw) {
  const int64_t b = blockIdx.x;
  const int64_t nxw = nbx + nbw;
  if (b % period == period - 1 && b / period < nxw) {
    const int64_t t = b / period;
    if (t < nbx)
      quant_tile<QM_TENSOR, 0, 0, true, true>(px, t % ctx, t / ctx);
    else
      quant_tile<QM_TENSOR, 0, 0, true, true>(pw, (t - nbx) % ctw, (t - nbx) / ctw);
  } else {
    const int64_t before = (b + 1) / period < nxw ? (b + 1) / period : nxw;
    const int64_t t = b - before;
    quant_tile<MODE, K, H2, true, false>(pg, t % ctg, t / ctg);
  }
}

template <int MODE, int K>
static hipError_t launch_quant_fused_k(const QuantParams& pg, const QuantParams& px, const QuantParams& pw,
                                       hipStream_t s) {
  const int64_t ctg = (pg.cols + QT_COLS - 1) / QT_COLS, rtg = (pg.rows + QT_SLOTS - 1) / QT_SLOTS;
  const int64_t ctx = (px.cols + QT_COLS - 1) / QT_COLS, rtx = (px.rows + QT_SLOTS - 1) / QT_SLOTS;
  const int64_t ctw = (pw.cols + QT_COLS - 1) / QT_COLS, rtw = (pw.rows + QT_SLOTS - 1) / QT_SLOTS;
  const int64_t nbg = ctg * rtg, nbx = ctx * rtx, nbw = ctw * rtw;
  const int64_t nb = nbg + nbx + nbw;
  if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
  const int64_t period = nb / (nbx + nbw);
  if (pg.shift2)
    hipLaunchKernelGGL((quant_fused_kernel<MODE, K, 2>), dim3((unsigned)nb), dim3(256), 0, s, pg, px, pw, nbx, nbw,
                       period, ctg, ctx, ctw);
  else
    hipLaunchKernelGGL((quant_fused_kernel<MODE, K, 1>), dim3((unsigned)nb), dim3(256), 0, s, pg, px, pw, nbx, nbw,
                       period, ctg, ctx, ctw);
  return hipGetLastError();
}

template <int MODE, int K>
static hipError_t launch_quant_k(const QuantParams& p, hipStream_t s) {
  const int64_t ct = (p.cols + QT_COLS - 1) / QT_COLS;
  const int64_t rt = (p.rows + QT_SLOTS - 1) / QT_SLOTS;
  if (ct > 0x7FFFFFFF || rt > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)ct, (unsigned)rt);
  const bool vec = (p.cols % 4 == 0) && (((uintptr_t)p.x & 15) == 0);
  if (p.packed && (!vec || p.bits > 4 || p.q_t)) return hipErrorInvalidValue;
  // one primary layout: natural (with an optional transposed Q_b1) or transposed
  if ((p.q_nat || p.sum_nat) && (p.q_t || p.sum_t)) return hipErrorInvalidValue;
  if (p.pm_o < 0 || (p.pm_o > 0 && ((p.pm_o & 3) != 0 || p.cols % p.pm_o != 0 || p.packed || (p.cols & 3) != 0)))
    return hipErrorInvalidValue;
  const bool trans = p.q_t || p.sum_t;
  if (p.shift && MODE != QM_ROW) return hipErrorInvalidValue;
  if (p.q2_t) {
    if (trans || !p.stoch) return hipErrorInvalidValue;
    if (p.shift2) {
      if (vec)
        hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 2, true, false>), grid, dim3(256), 0, s, p);
      else
        hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 2, false, false>), grid, dim3(256), 0, s, p);
    } else if (vec) {
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 1, true, false>), grid, dim3(256), 0, s, p);
    } else {
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 1, false, false>), grid, dim3(256), 0, s, p);
    }
  } else if (trans) {
    if (vec)
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 0, true, true>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 0, false, true>), grid, dim3(256), 0, s, p);
  } else {
    if (vec)
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 0, true, false>), grid, dim3(256), 0, s, p);
    else
      hipLaunchKernelGGL((quant_tile_kernel<MODE, K, 0, false, false>), grid, dim3(256), 0, s, p);
  }
  return hipGetLastError();
}

hipError_t launch_quant_pair(const QuantParams& p0, const QuantParams& p1, hipStream_t s) {
  for (const QuantParams* p : {&p0, &p1})
    if (p->q_nat || p->sum_nat || p->q2_t || !p->q_t) return hipErrorInvalidValue;
  const int64_t ct0 = (p0.cols + QT_COLS - 1) / QT_COLS, rt0 = (p0.rows + QT_SLOTS - 1) / QT_SLOTS;
  const int64_t ct1 = (p1.cols + QT_COLS - 1) / QT_COLS, rt1 = (p1.rows + QT_SLOTS - 1) / QT_SLOTS;
  const int64_t nb0 = ct0 * rt0, nb = nb0 + ct1 * rt1;
  if (nb > 0x7FFFFFFF) return hipErrorInvalidValue;
  const bool vec = (p0.cols % 4 == 0) && (((uintptr_t)p0.x & 15) == 0) && (p1.cols % 4 == 0) &&
                   (((uintptr_t)p1.x & 15) == 0);
  if (vec)
    hipLaunchKernelGGL(quant_tile2_kernel<true>, dim3((unsigned)nb), dim3(256), 0, s, p0, p1, nb0, ct0, ct1);
  else
    hipLaunchKernelGGL(quant_tile2_kernel<false>, dim3((unsigned)nb), dim3(256), 0, s, p0, p1, nb0, ct0, ct1);
  return hipGetLastError();
}

hipError_t launch_quant_fused(const QuantParams& pg, int mode, const QuantParams& px, const QuantParams& pw,
                              hipStream_t s) {
  // float4 rows everywhere, natural + transposed Q_b1 for the gradient,
  // transposed only for X and W; anything else goes out as three launches
  auto vec = [](const QuantParams& p) { return (p.cols % 4 == 0) && (((uintptr_t)p.x & 15) == 0); };
  if (pg.packed && (!vec(pg) || pg.bits > 4)) return hipErrorInvalidValue;
  const bool shape = vec(pg) && vec(px) && vec(pw) && pg.q2_t && pg.stoch && !pg.q_t && !pg.sum_t && !px.q_nat &&
                     !px.sum_nat && !px.q2_t && px.q_t && !pw.q_nat && !pw.sum_nat && !pw.q2_t && pw.q_t;
  if (!shape) {
    hipError_t e = launch_quant_pair(px, pw, s);
    if (e != hipSuccess) return e;
    return launch_quant(pg, mode, s);
  }
  if (mode == QM_TENSOR) return launch_quant_fused_k<QM_TENSOR, 0>(pg, px, pw, s);
  if (mode == QM_ROW) return launch_quant_fused_k<QM_ROW, 0>(pg, px, pw, s);
  switch (pg.L.k) {
    case 0: return pg.slot && pg.tau ? launch_quant_fused_k<QM_BHQ, 0>(pg, px, pw, s) : hipErrorInvalidValue;
    case 1: return launch_quant_fused_k<QM_BHQ, 1>(pg, px, pw, s);
    case 2: return launch_quant_fused_k<QM_BHQ, 2>(pg, px, pw, s);
    case 4: return launch_quant_fused_k<QM_BHQ, 4>(pg, px, pw, s);
    case 8: return launch_quant_fused_k<QM_BHQ, 8>(pg, px, pw, s);
    case 16: return launch_quant_fused_k<QM_BHQ, 16>(pg, px, pw, s);
    case 32: return launch_quant_fused_k<QM_BHQ, 32>(pg, px, pw, s);
    case 64: return launch_quant_fused_k<QM_BHQ, 64>(pg, px, pw, s);
    default: return hipErrorInvalidValue;
  }
}

// Seed batch (natural layout, float4 rows): one block per 64 x 256 tile.
template <int MODE, int K>
__global__ __launch_bounds__(256) void quant_seeds_kernel(QuantParams p) {
  quant_tile<MODE, K, 0, true, false, true>(p, blockIdx.x, blockIdx.y);
}

template <int MODE, int K>
static hipError_t launch_seeds_k(const QuantParams& p, hipStream_t s) {
  const int64_t ct = (p.cols + QT_COLS - 1) / QT_COLS;
  const int64_t rt = (p.rows + QT_SLOTS - 1) / QT_SLOTS;
  if (ct > 0x7FFFFFFF || rt > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL((quant_seeds_kernel<MODE, K>), dim3((unsigned)ct, (unsigned)rt), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_quant_seeds(const QuantParams& p, int mode, hipStream_t s) {
  if (p.nseeds < 1 || !p.sum_c || !p.sum_c2 || p.cols % 4 != 0 || ((uintptr_t)p.x & 15) ||
      ((uintptr_t)p.sum_c & 15) || ((uintptr_t)p.sum_c2 & 15))
    return hipErrorInvalidValue;
  if (mode == QM_TENSOR) return launch_seeds_k<QM_TENSOR, 0>(p, s);
  if (mode == QM_ROW) return launch_seeds_k<QM_ROW, 0>(p, s);
  switch (p.L.k) {
    case 0: return p.slot && p.tau ? launch_seeds_k<QM_BHQ, 0>(p, s) : hipErrorInvalidValue;
    case 1: return launch_seeds_k<QM_BHQ, 1>(p, s);
    case 2: return launch_seeds_k<QM_BHQ, 2>(p, s);
    case 4: return launch_seeds_k<QM_BHQ, 4>(p, s);
    case 8: return launch_seeds_k<QM_BHQ, 8>(p, s);
    case 16: return launch_seeds_k<QM_BHQ, 16>(p, s);
    case 32: return launch_seeds_k<QM_BHQ, 32>(p, s);
    case 64: return launch_seeds_k<QM_BHQ, 64>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_quant(const QuantParams& p, int mode, hipStream_t s) {
  if (mode == QM_TENSOR) return launch_quant_k<QM_TENSOR, 0>(p, s);
  if (mode == QM_ROW) return launch_quant_k<QM_ROW, 0>(p, s);
  switch (p.L.k) {
    case 0: return p.slot && p.tau ? launch_quant_k<QM_BHQ, 0>(p, s) : hipErrorInvalidValue;
    case 1: return launch_quant_k<QM_BHQ, 1>(p, s);
    case 2: return launch_quant_k<QM_BHQ, 2>(p, s);
    case 4: return launch_quant_k<QM_BHQ, 4>(p, s);
    case 8: return launch_quant_k<QM_BHQ, 8>(p, s);
    case 16: return launch_quant_k<QM_BHQ, 16>(p, s);
    case 32: return launch_quant_k<QM_BHQ, 32>(p, s);
    case 64: return launch_quant_k<QM_BHQ, 64>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fqt
