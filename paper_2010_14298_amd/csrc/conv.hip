// Conv layer FQT backward on gfx950 (NHWC tensors, rows = samples).
//
// The conv is the linear layer Y = im2col(X) W^T (Sec. 2.1 for linear layers),
// so its backward is grad_W = Q_b1(G)^T im2col(Q_f(X)) and
// grad_X = col2im(Q_b2(G) Q_theta(W)) (Sec. 2.2).  Layouts:
//
//   X codes    [c][pixels]           per-tensor PTQ, samples in slot order
//   Q_b1(G)    [o][pixels (padded)]  stochastic PTQ or PSQ, slot order; on
//                                    the zero-halo grid for the implicit form
//   im2col     [(r, s, c)][pixels]   X codes per tap, zero codes on padding
//   X grids    [s][c][grid]          implicit form (stride 1): kw shifted
//                                    copies of the zero-halo activation grid
//   W codes    [c][(r, s, o)]        per-tensor PTQ
//   Q_b2(G)    [(y, x)][slot][o]     PTQ / PSQ / BHQ, pixel-major
//
// grad_W is a split-K int8 contraction over output pixels (over im2col rows,
// or over tap rows of the shifted grids) with per-tap masked zero-point sums
// in its reduction; a per-sample Q_b1 takes one K block per sample.  grad_X
// is an implicit-im2col
// contraction: its A rows (input pixel, slot) are gathered 16 output
// channels at a time from Q_b2(G); padded taps load zero codes and the
// epilogue subtracts nothing for them (their zero-point sums are built from
// the valid taps only).  A tile row block holds the slots of one input pixel,
// so the block Householder inverse of a group runs inside the tile.
#include "gemm_core.h"

namespace fqt {

template <typename T>
__device__ __forceinline__ T wave_sum_t(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_sum4_i(int v) { return wave_sum_t<int>(v); }


// ---------------------------------------------------------------------------
// narrow transposing quantizer: logical [rows, cols] -> codes [cols][ldt].
// Rows come in blocks of blk (a sample's pixels); block b takes source block
// perm[b] (slot order) of vblk rows, and its rows past vblk, like rows in
// [rows, ldt), get code 0.  Scale and zero are per tensor, or per source
// block (a per-sample quantizer).  A block covers 4 * LPR columns (grid.y
// walks wider rows in chunks of 256).
// ---------------------------------------------------------------------------
template <int LPR, bool TWO, bool VEC>
__global__ __launch_bounds__(256) void quant_narrow_t_kernel(NarrowQParams p) {
  constexpr int RG = 64 / LPR;  // row groups of 16 per wave
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int q = lane / LPR, cl = lane % LPR;
  // row indices in 32 bits: the launch checks that ldt, rows + blk (which
  // bounds every source row) and cols stay below 2^31
  const int blk = (int)p.blk;
  const int r0 = (int)blockIdx.x * (4 * RG * 16) + wave * (RG * 16) + q * 16;
  const int64_t c0 = (int64_t)blockIdx.y * (LPR * 4) + (int64_t)cl * 4;  // column chunks of 4 * LPR
  const int B = (1 << p.bits) - 1;
  const int half = 1 << (p.bits - 1);
  const float s0 = p.scale[0], z0 = p.zero[0];
  const int vblk = p.vblk > 0 ? (int)p.vblk : blk;
  // VEC: cols % 4 == 0, so a lane's four columns are all inside or all past the end
  const bool full = VEC && c0 < p.cols;
  // Rows r0 .. r0 + 15: row (bq, br) reads row br of source block perm[bq]
  // (or bq) of vblk rows.  TWO (blk >= 16): the 16 rows lie in blocks bq0
  // and bq0 + 1, whose source blocks and scales are read once up front.
  const int bq0 = r0 / blk, br0 = r0 - bq0 * blk;
  int sbA = 0, sbB = 0;
  float sA = s0, zA = z0, sB = s0, zB = z0;
  if constexpr (TWO) {
    const int nblk = (int)((p.rows + p.blk - 1) / p.blk);
    const int qa = bq0 < nblk ? bq0 : nblk - 1, qb = bq0 + 1 < nblk ? bq0 + 1 : nblk - 1;
    sbA = p.perm ? p.perm[qa] : qa;
    sbB = p.perm ? p.perm[qb] : qb;
    if (p.rowscale) {
      sA = p.scale[sbA];
      zA = p.zero[sbA];
      sB = p.scale[sbB];
      zB = p.zero[sbB];
    }
  }
  // 2-D blocks: (y, x) of offset br0 once; the 16 rows then step x (gw >= 16
  // and blocks of at least 128 rows: at most one row wrap, at most one block
  // boundary, after which (y, x) = (0, br))
  const int gw = (int)p.gw, gwo = (int)p.gwo, gho = (int)p.gho;
  const int gy0 = gw > 0 ? br0 / gw : 0, gx0 = gw > 0 ? br0 - gy0 * gw : 0;
  const int vb = gw > 0 ? gho * gwo : vblk;  // source rows per block
  const int rows = (int)p.rows;
  // source row, scale and zero of row r (row r of the 16 has offset br0 + r)
  auto locate = [&](int r, int& src, float& s, float& z) -> bool {
    int bq = bq0, br = br0 + r;
    const bool wrapped = br >= blk;
    if (wrapped) {
      if constexpr (TWO) {  // blk >= 16: at most one block boundary
        bq += 1;
        br -= blk;
      } else {  // small blocks: stepped
        const int d = br / blk;
        bq += d;
        br -= d * blk;
      }
    }
    bool inside;
    int srow;
    if (gw > 0) {
      int y = wrapped ? 0 : gy0, x = wrapped ? br : gx0 + r;
      if (x >= gw) {
        x -= gw;
        ++y;
      }
      inside = y < gho && x < gwo;
      srow = y * gwo + x;
    } else {
      inside = br < vblk;
      srow = br;
    }
    const bool ok = r0 + r < rows && inside;
    int sb;
    if constexpr (TWO) {
      const bool inb = bq != bq0;
      sb = inb ? sbB : sbA;
      s = inb ? sB : sA;
      z = inb ? zB : zA;
    } else {
      sb = ok ? (p.perm ? p.perm[bq] : bq) : 0;
      s = (p.rowscale && ok) ? p.scale[sb] : s0;
      z = (p.rowscale && ok) ? p.zero[sb] : z0;
    }
    src = sb * vb + srow;
    return ok;
  };
  // ---- phase 1: the 16 rows' loads, issued together (clamped addresses and
  // selects instead of branches around the loads).  Kept for phase 2: the
  // source row (-1 past the end) and, for TWO, a bit per row in block
  // bq0 + 1.
  float g[16][4];
  int32_t src32[16];
  uint32_t inb_mask = 0u;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int src;
    float s, z;
    const bool ok = locate(r, src, s, z);
    src32[r] = ok ? src : -1;
    if (TWO && br0 + r >= blk) inb_mask |= 1u << r;
    if constexpr (VEC) {
      const bool in = ok && full;
      const float4 v = *reinterpret_cast<const float4*>(p.x + (in ? (uint64_t)(uint32_t)src * (uint64_t)p.cols + c0 : 0));
      g[r][0] = in ? v.x : 0.0f;
      g[r][1] = in ? v.y : 0.0f;
      g[r][2] = in ? v.z : 0.0f;
      g[r][3] = in ? v.w : 0.0f;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        g[r][j] = (ok && c0 + j < p.cols) ? p.x[(int64_t)src * p.cols + c0 + j] : 0.0f;
    }
  }
  // ---- phase 2: codes, transposed into words of four rows.  The float4
  // path works in the top-byte form of sr_top / rne_top (offset codes packed
  // by byte permutes); the other path rounds element by element.
  uint32_t tcodes[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int w = 0; w < 4; ++w) tcodes[j][w] = 0u;
  const float Bf = (float)B;
  const uint32_t hoff = (uint32_t)half << 24;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    int src;
    float s, z;
    bool ok;
    if constexpr (TWO) {
      ok = src32[r] >= 0;
      src = ok ? src32[r] : 0;
      const bool inb = (inb_mask >> r) & 1u;
      s = inb ? sB : sA;
      z = inb ? zB : zA;
    } else {
      ok = locate(r, src, s, z);
    }
    if constexpr (VEC) {
      float y[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = s * (g[r][j] - z);
      int32_t t[4];
      if (p.stoch) {
        // Philox block index src * cols / 4 + c0 / 4 (cols % 4 == c0 % 4 == 0)
        const uint64_t pb = (uint64_t)(uint32_t)src * (uint64_t)(p.cols >> 2) + (uint64_t)(c0 >> 2);
        const u32x4 o = philox_of_block(pb, p.seed, p.stream);
        t[0] = sr_top(y[0], o.x, Bf, hoff);
        t[1] = sr_top(y[1], o.y, Bf, hoff);
        t[2] = sr_top(y[2], o.z, Bf, hoff);
        t[3] = sr_top(y[3], o.w, Bf, hoff);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) t[j] = rne_top(y[j], Bf, hoff);
      }
      const bool in = ok && full;
#pragma unroll
      for (int j = 0; j < 4; ++j) tcodes[j][r >> 2] = insert_top(tcodes[j][r >> 2], in ? t[j] : 0, r & 3);
    } else {
      int code[4];
      const uint64_t ebase = (uint64_t)(uint32_t)src * (uint64_t)p.cols + (uint64_t)c0;
      if (p.stoch) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint64_t e = ebase + j;
          const u32x4 o = philox_block(e, p.seed, p.stream);
          code[j] = sr_code(s * (g[r][j] - z), philox_word(o, (int)(e & 3)), B);
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) code[j] = rne_code(s * (g[r][j] - z), B);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int qv = (ok && c0 + j < p.cols) ? code[j] - half : 0;
        tcodes[j][r >> 2] |= (uint32_t)(qv & 255) << (8 * (r & 3));
      }
    }
  }
  const bool tvec = ((p.ldt & 15) == 0) && (r0 + 15 < p.ldt);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t col = c0 + j;
    if (col >= p.cols || r0 >= p.ldt) continue;
    int8_t* dst = p.q_t + col * p.ldt + r0;
    if (tvec) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(tcodes[j][0], tcodes[j][1], tcodes[j][2], tcodes[j][3]);
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (r0 + r < p.ldt) dst[r] = (int8_t)((tcodes[j][r >> 2] >> (8 * (r & 3))) & 255);
    }
  }
}

template <bool TWO, bool VEC>
static hipError_t launch_narrow_lpr(const NarrowQParams& p, int lpr, dim3 grid, hipStream_t s) {
  switch (lpr) {
    case 1: hipLaunchKernelGGL((quant_narrow_t_kernel<1, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    case 2: hipLaunchKernelGGL((quant_narrow_t_kernel<2, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    case 4: hipLaunchKernelGGL((quant_narrow_t_kernel<4, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    case 8: hipLaunchKernelGGL((quant_narrow_t_kernel<8, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    case 16: hipLaunchKernelGGL((quant_narrow_t_kernel<16, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    case 32: hipLaunchKernelGGL((quant_narrow_t_kernel<32, TWO, VEC>), grid, dim3(256), 0, s, p); break;
    default: hipLaunchKernelGGL((quant_narrow_t_kernel<64, TWO, VEC>), grid, dim3(256), 0, s, p); break;
  }
  return hipGetLastError();
}

hipError_t launch_quant_narrow_t(const NarrowQParams& p, hipStream_t s) {
  if (p.blk < 1 || p.vblk < 0 || p.vblk > p.blk) return hipErrorInvalidValue;
  // the kernel keeps row indices in 32 bits
  if (p.ldt + 4096 >= (1ll << 31) || p.rows + p.blk >= (1ll << 31) || p.cols >= (1ll << 31) || p.ldt < p.rows)
    return hipErrorInvalidValue;
  if (p.gw > 0 && (p.gw < 16 || p.blk < 128 || p.gwo > p.gw || p.gho * p.gw > p.blk)) return hipErrorInvalidValue;
  // lanes per row: the smallest power of two covering cols / 4, at most 64
  // (wider rows: column chunks of 256 along grid.y)
  const int64_t need = (p.cols + 3) / 4;
  int lpr = 1;
  while (lpr < need && lpr < 64) lpr <<= 1;
  const int64_t chunks = (need + 63) / 64;
  const int64_t rows_per_block = 4 * (64 / lpr) * 16;
  const int64_t blocks = (p.ldt + rows_per_block - 1) / rows_per_block;
  if (blocks > 0x7FFFFFFF || chunks > 65535) return hipErrorInvalidValue;
  const dim3 grid((unsigned)blocks, (unsigned)chunks);
  const bool two = p.blk >= 16, vec = (p.cols & 3) == 0;
  if (vec) return two ? launch_narrow_lpr<true, true>(p, lpr, grid, s) : launch_narrow_lpr<false, true>(p, lpr, grid, s);
  return two ? launch_narrow_lpr<true, false>(p, lpr, grid, s) : launch_narrow_lpr<false, false>(p, lpr, grid, s);
}

// ---------------------------------------------------------------------------
// W codes [c][(r, s, o)] (deterministic PTQ) and their sums over o per (tap, c)
// ---------------------------------------------------------------------------
// One wave per (tap, channel): lanes over the output channels o.
__global__ __launch_bounds__(256) void conv_wq_kernel(const float* W, ConvGeom g, int bits, const float* scale,
                                                      const float* zero, int8_t* wq_t, int32_t* swq) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int taps = g.kh * g.kw;
  if (t >= (int64_t)taps * g.c) return;  // whole waves
  const int tap = (int)(t / g.c), c = (int)(t % g.c);
  const int B = (1 << bits) - 1, half = 1 << (bits - 1);
  const float s = scale[0], z = zero[0];
  const int64_t K = (int64_t)taps * g.o;
  int sum = 0;
  for (int o = lane; o < g.o; o += 64) {
    const float v = W[((int64_t)o * taps + tap) * g.c + c];
    const int q = rne_code(s * (v - z), B) - half;
    wq_t[(int64_t)c * K + (int64_t)tap * g.o + o] = (int8_t)q;
    sum += q;
  }
  sum = wave_sum4_i(sum);
  if (lane == 0) swq[(int64_t)tap * g.c + c] = sum;
}

// ---------------------------------------------------------------------------
// im2col of the X codes for grad_W: B[(r, s, c)][p] over output pixels p in
// slot order (zero codes on padded taps and for p >= P), plus row sums
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void conv_im2col_w_kernel(ConvGeom g, const int8_t* xq_t, int8_t* bw, int64_t ldb) {
  const int64_t row = blockIdx.y;
  const int tap = (int)(row / g.c), c = (int)(row % g.c);
  const int r = tap / g.kw, s = tap % g.kw;
  const int64_t hw = (int64_t)g.h * g.w, howo = (int64_t)g.ho * g.wo;
  const int64_t p0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 16;
  const int8_t* xc = xq_t + (int64_t)c * g.n * hw;
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  if (p0 < ldb) {
    // (sample, pixel, y, x) of p0 once; the 16 columns then step through x,
    // y and the sample's pitch (columns past ho wo in a pitch are zero)
    int64_t slot = p0 / g.psp;
    int pix = (int)(p0 - slot * g.psp);
    int y = pix / g.wo, x = pix - (pix / g.wo) * g.wo;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      int v = 0;
      if (slot < g.n && pix < howo) {
        const int iy = y * g.stride - g.pad + r, ix = x * g.stride - g.pad + s;
        if (iy >= 0 && iy < g.h && ix >= 0 && ix < g.w) v = xc[slot * hw + iy * g.w + ix];
      }
      w[i >> 2] |= (uint32_t)(v & 255) << (8 * (i & 3));
      ++pix;
      if (++x == g.wo) {
        x = 0;
        ++y;
      }
      if (pix == g.psp) {
        pix = x = y = 0;
        ++slot;
      }
    }
    *reinterpret_cast<uint4*>(bw + row * ldb + p0) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// ---------------------------------------------------------------------------
// masked zero-point sums of Q_b1(G) per (o, tap) and the valid-pixel count of
// each tap: Qs[o][y][x] = sum over samples, then rectangle sums per tap
// ---------------------------------------------------------------------------
// Stride-1 im2col of the activation codes for grad_W, one thread per output
// word: a block takes whole output row segments (sample, y) of one (tap,
// channel) row, and its threads walk the segments' words in order, so loads
// and stores are coalesced along the row.  Output x reads input x + s - pad
// of row iy = y - pad + r; with w and wo multiples of 4 and 4-byte aligned
// rows each output word is a byte funnel shift of two input words, and
// input words outside the row read as zero, which is exactly the padding.
__host__ __device__ inline bool conv_im2col_rows_ok(const ConvGeom& g, const int8_t* xq_t, const int8_t* bw,
                                                    int64_t ldb) {
  return g.stride == 1 && (g.w & 3) == 0 && (g.wo & 3) == 0 && (ldb & 3) == 0 && (((uintptr_t)xq_t) & 3) == 0 &&
         (((uintptr_t)bw) & 3) == 0 && g.wo <= 1024;
}

constexpr int IM2COL_WPT = 8;  // output words per thread (loads in flight together)

__global__ __launch_bounds__(256) void conv_im2col_rows_kernel(ConvGeom g, const int8_t* xq_t, int8_t* bw,
                                                               int64_t ldb, int segs_per_block) {
  const int64_t row = blockIdx.y;
  const int tap = (int)(row / g.c), c = (int)(row % g.c);
  const int r = tap / g.kw, s = tap % g.kw;
  const int64_t hw = (int64_t)g.h * g.w;
  const int nw = g.wo >> 2, iw = g.w >> 2;
  const int64_t nseg = (int64_t)g.n * g.ho;
  const int d = s - g.pad;                              // output x reads input x + d
  const int wq = d >= 0 ? d >> 2 : -((-d + 3) >> 2);   // floor(d / 4)
  const int sh = d - 4 * wq;                            // 0..3
  const int8_t* xc = xq_t + (int64_t)c * g.n * hw;
  int8_t* dst = bw + row * ldb;
  uint32_t lo[IM2COL_WPT], hi[IM2COL_WPT];
  int64_t at[IM2COL_WPT];
  // thread t takes words t, t + 256, ...: a step of 256 words is `sa` whole
  // segments and `sb` words, so (segment, word) and (slot, y) advance
  // without divisions (32-bit: n * ho < 2^31 is checked at launch)
  const int sa = (int)blockDim.x / nw, sb = (int)blockDim.x - sa * nw;
  int ls = threadIdx.x / nw, j = threadIdx.x - ls * nw;
  int seg = (int)blockIdx.x * segs_per_block + ls;
  int slot = seg / g.ho, y = seg - slot * g.ho;
#pragma unroll
  for (int q = 0; q < IM2COL_WPT; ++q) {
    lo[q] = hi[q] = 0u;
    at[q] = -1;
    if (ls < segs_per_block && seg < (int)nseg) {
      const int iy = y - g.pad + r;
      at[q] = (int64_t)slot * g.psp + (int64_t)y * g.wo + 4 * j;
      if (iy >= 0 && iy < g.h) {
        const uint32_t* src = reinterpret_cast<const uint32_t*>(xc + (int64_t)slot * hw + (int64_t)iy * g.w);
        const int k0 = j + wq;
        if (k0 >= 0 && k0 < iw) lo[q] = src[k0];
        if (k0 + 1 >= 0 && k0 + 1 < iw) hi[q] = src[k0 + 1];
      }
    }
    // advance by blockDim.x words
    int step = sa;
    j += sb;
    if (j >= nw) {
      j -= nw;
      ++step;
    }
    ls += step;
    seg += step;
    y += step;
    while (y >= g.ho) {
      y -= g.ho;
      ++slot;
    }
  }
#pragma unroll
  for (int q = 0; q < IM2COL_WPT; ++q)
    if (at[q] >= 0)
      *reinterpret_cast<uint32_t*>(dst + at[q]) =
          sh == 0 ? lo[q] : (uint32_t)((((uint64_t)hi[q] << 32) | lo[q]) >> (8 * sh));
  // the zero tail [P, ldb) of the row: the last block's threads (a pitch
  // longer than ho wo gets its zeros from conv_pitch_zero_kernel)
  if (blockIdx.x == gridDim.x - 1 && g.psp == (int64_t)g.ho * g.wo) {
    const int64_t P = nseg * g.wo;
    for (int64_t t = P + 4 * (int64_t)threadIdx.x; t < ldb; t += 4 * (int64_t)blockDim.x)
      *reinterpret_cast<uint32_t*>(dst + t) = 0u;
  }
}

// The kw shifted copies of the zero-halo activation grid (the implicit
// grad_W form), one thread per 16-byte chunk j of grid row y' of one
// (channel, slot): byte x' of copy s holds input pixel (y' - pad, x' + s -
// pad), zero outside the image.  The thread loads the input words under
// the chunk plus the kw - 1 bytes after it once (word-aligned rows: w % 4
// == 0) and stores each copy's chunk as a byte funnel shift of them.
constexpr int XGRID_MAXKW = 8;
__global__ __launch_bounds__(256) void conv_xgrid_kernel(ConvGeom g, const int8_t* xq_t, int8_t* grid) {
  constexpr int NWD = (16 + XGRID_MAXKW - 1 + 3) / 4 + 1;  // input words a chunk can need
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = (int)(g.gwp >> 4);  // chunks per grid row
  const int64_t rows_per_c = (int64_t)g.n * g.ghp;
  if (t >= (int64_t)g.c * rows_per_c * cpr) return;
  const int j = (int)(t % cpr);
  const int64_t rr = t / cpr;  // (c, slot, y')
  const int yp = (int)(rr % g.ghp);
  const int64_t cs = rr / g.ghp;
  const int slot = (int)(cs % g.n);
  const int c = (int)(cs / g.n);
  const int iy = yp - g.pad;
  const int iw = g.w >> 2;
  // input bytes from x0 = 16 j - pad on: words w0 .. w0 + NWD - 1 with w0 = floor(x0 / 4)
  const int x0 = 16 * j - g.pad;
  const int w0 = x0 >= 0 ? x0 >> 2 : -((-x0 + 3) >> 2);
  const int sh0 = x0 - 4 * w0;  // 0..3
  uint32_t wd[NWD];
  const bool rowin = iy >= 0 && iy < g.h;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(xq_t + ((int64_t)c * g.n + slot) * g.h * g.w +
                                                          (int64_t)(rowin ? iy : 0) * g.w);
#pragma unroll
  for (int k = 0; k < NWD; ++k) {
    const int wi = w0 + k;
    wd[k] = (rowin && wi >= 0 && wi < iw) ? src[wi] : 0u;
  }
  int8_t* dst0 = grid + (int64_t)c * g.ldx + (int64_t)slot * g.psp + (int64_t)yp * g.gwp + 16 * j;
#pragma unroll
  for (int s = 0; s < XGRID_MAXKW; ++s) {
    if (s >= g.kw) break;
    // bytes x0 + s .. x0 + s + 15: word offset (sh0 + s) / 4, byte shift (sh0 + s) % 4
    const int b = sh0 + s, q = b >> 2, sh = b & 3;
    uint32_t o[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint32_t lo = 0u, hi = 0u;
#pragma unroll
      for (int k = 0; k + 1 < NWD; ++k)
        if (k == q + u) {
          lo = wd[k];
          hi = wd[k + 1];
        }
      o[u] = sh == 0 ? lo : (uint32_t)((((uint64_t)hi << 32) | lo) >> (8 * sh));
    }
    *reinterpret_cast<uint4*>(dst0 + (int64_t)s * g.c * g.ldx) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

__device__ __forceinline__ void tap_range(int r, int stride, int pad, int h, int ho, int& lo, int& hi) {
  lo = 0;
  while (lo < ho && lo * stride - pad + r < 0) ++lo;
  hi = ho;
  while (hi > lo && (hi - 1) * stride - pad + r >= h) --hi;
}

// One block per (o, tap): the code sums qs[o] over the tap's valid output
// pixels (a rectangle), spread over the block's threads.
// Code sums of the im2col rows without touching them: xs[c][pix] sums the
// activation codes over samples, and row (tap, c) of the im2col matrix sums
// xs[c] over the input pixels its valid output pixels read (a strided
// rectangle), one block per row.
__global__ void conv_xsum_kernel(ConvGeom g, const int8_t* xq_t, int32_t* xs) {
  const int64_t hw = (int64_t)g.h * g.w;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)g.c * hw) return;
  const int64_t c = t / hw, pix = t % hw;
  const int8_t* col = xq_t + c * g.n * hw + pix;
  int s4[4] = {0, 0, 0, 0};
#pragma unroll 16
  for (int n = 0; n < g.n; ++n) s4[n & 3] += col[(int64_t)n * hw];
  xs[t] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
}

template <typename T>
__global__ __launch_bounds__(256) void conv_xtapsum_kernel(ConvGeom g, const T* xs, T* sumB) {
  const int64_t row = blockIdx.x;  // (tap, c)
  const int tap = (int)(row / g.c), c = (int)(row % g.c);
  const int r = tap / g.kw, s = tap % g.kw;
  int ylo, yhi, xlo, xhi;
  tap_range(r, g.stride, g.pad, g.h, g.ho, ylo, yhi);
  tap_range(s, g.stride, g.pad, g.w, g.wo, xlo, xhi);
  const T* x = xs + (int64_t)c * g.h * g.w;
  const int wx = xhi - xlo, cnt = (yhi - ylo) * wx;
  T sum = 0;
  // eight loads in flight per round: indices past cnt are clamped (their
  // values dropped), so no load sits under a branch
  for (int i0 = threadIdx.x; i0 < cnt; i0 += 8 * blockDim.x) {
    T v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = min(i0 + u * (int)blockDim.x, cnt - 1);
      const int dy = i / wx;
      const int iy = (ylo + dy) * g.stride - g.pad + r, ix = (xlo + i - dy * wx) * g.stride - g.pad + s;
      v[u] = x[(int64_t)iy * g.w + ix];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (i0 + u * (int)blockDim.x < cnt) sum += v[u];
  }
  __shared__ T ssum[4];
  sum = wave_sum_t<T>(sum);
  if ((threadIdx.x & 63) == 0) ssum[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) sumB[row] = ssum[0] + ssum[1] + ssum[2] + ssum[3];
}

__global__ void conv_qsum_kernel(ConvGeom g, const int8_t* q1_t, int64_t ldq, int32_t* qs) {
  const int64_t howo = (int64_t)g.ho * g.wo;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)g.o * howo) return;
  const int64_t o = t / howo, pix = t % howo;
  // slot n's codes start at n psp; grid rows of gwp in the implicit form
  const int64_t off = g.gwp > 0 ? (pix / g.wo) * g.gwp + pix % g.wo : pix;
  const int8_t* row = q1_t + o * ldq + off;
  int s4[4] = {0, 0, 0, 0};
#pragma unroll 16
  for (int n = 0; n < g.n; ++n) s4[n & 3] += row[(int64_t)n * g.psp];
  qs[t] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
}

// valid output rows / columns of tap offset r: y with 0 <= y*stride - pad + r < h
template <typename T>
__global__ __launch_bounds__(256) void conv_tapsum_kernel(ConvGeom g, const T* qs, T* sumA_tap, int32_t* count_tap) {
  const int taps = g.kh * g.kw;
  const int64_t t = blockIdx.x;
  const int o = (int)(t / taps), tap = (int)(t % taps);
  const int r = tap / g.kw, s = tap % g.kw;
  int ylo, yhi, xlo, xhi;
  tap_range(r, g.stride, g.pad, g.h, g.ho, ylo, yhi);
  tap_range(s, g.stride, g.pad, g.w, g.wo, xlo, xhi);
  const T* q = qs + (int64_t)o * g.ho * g.wo;
  const int wx = xhi - xlo, cnt = (yhi - ylo) * wx;
  T sum = 0;
  // eight loads in flight per round (clamped indices, values past cnt dropped)
  for (int i0 = threadIdx.x; i0 < cnt; i0 += 8 * blockDim.x) {
    T v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = min(i0 + u * (int)blockDim.x, cnt - 1);
      const int dy = i / wx;
      v[u] = q[(int64_t)(ylo + dy) * g.wo + xlo + (i - dy * wx)];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (i0 + u * (int)blockDim.x < cnt) sum += v[u];
  }
  __shared__ T ssum[4];
  sum = wave_sum_t<T>(sum);
  if ((threadIdx.x & 63) == 0) ssum[threadIdx.x >> 6] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    sumA_tap[t] = ssum[0] + ssum[1] + ssum[2] + ssum[3];
    if (o == 0) count_tap[tap] = g.n * cnt;
  }
}

// split-K reduction of grad_W with the per-tap masked zero-point expansion:
// out[o][(tap, c)] = dA dB acc + dA zB sumA_tap[o][tap] + zA dB sumB[(tap, c)] + count[tap] zA zB
// A block takes 64 outputs; its wave w sums splits w, w + 4, ... with eight
// loads in flight, and the four wave sums meet in LDS (integers: any order
// gives the same sum).  Lanes past the end load a clamped index and store
// nothing, so the loads sit under no branch.
__global__ __launch_bounds__(256) void conv_gradw_reduce_kernel(GemmParams p, ConvGeom g, const int32_t* sumA_tap,
                                                                const int32_t* count_tap) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t idx = (int64_t)blockIdx.x * 64 + lane;
  const int64_t MN = p.M * p.N;
  const int64_t ic = idx < MN ? idx : MN - 1;
  int64_t s8[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int sp = wave;
  for (; sp + 28 < p.splits; sp += 32)
#pragma unroll
    for (int u = 0; u < 8; ++u) s8[u] += (int64_t)p.part[(int64_t)(sp + 4 * u) * MN + ic];
  for (; sp < p.splits; sp += 4) s8[0] += (int64_t)p.part[(int64_t)sp * MN + ic];
  __shared__ int64_t swave[4][64];
  swave[wave][lane] = ((s8[0] + s8[1]) + (s8[2] + s8[3])) + ((s8[4] + s8[5]) + (s8[6] + s8[7]));
  __syncthreads();
  if (wave != 0 || idx >= MN) return;
  const int64_t sum = (swave[0][lane] + swave[1][lane]) + (swave[2][lane] + swave[3][lane]);
  const int64_t row = idx / p.N, col = idx % p.N;
  const int taps = g.kh * g.kw;
  const int tap = (int)(col / g.c);
  const double dA = 1.0 / (double)p.scaleA[0];
  const double zA = (double)p.zeroA[0] + (double)p.halfA * dA;
  const double dB = 1.0 / (double)p.scaleB[0];
  const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
  const double v = dA * dB * (double)sum + dA * zB * (double)sumA_tap[row * taps + tap] +
                   zA * dB * (double)p.sumB[col] + (double)count_tap[tap] * zA * zB;
  p.out[row * p.ldo + col] = (float)v;
}

// ---------------------------------------------------------------------------
// K-blocked grad_W for a per-sample Q_b1 (Sec. 4.1's per-sample scales on the
// weight-gradient product).  A sample's pixels form one K block, so the
// contraction gives an exact int32 sum per (slot, o, (tap, c)); each is
// scaled by its slot's 1 / s in float64.  With x1 = q dA_n + zA_n for the
// gradient codes of slot n and x2 = q dB + zB on valid taps:
//   grad_W[o][(tap, c)] = dB sum_n dA_n acc_n + zB sum_n dA_n SA_n[o][tap]
//                       + dB sum_n zA_n SB_n[(tap, c)] + zB cnt[tap] sum_n zA_n
// with SA_n, SB_n the code sums of slot n over the tap's valid pixels and
// cnt[tap] their number per sample.
// ---------------------------------------------------------------------------
// zero codes in the pitch tails [n psp + ho wo, (n + 1) psp) of each row
__global__ __launch_bounds__(256) void conv_pitch_zero_kernel(ConvGeom g, int8_t* bw, int64_t ldb) {
  const int64_t howo = (int64_t)g.ho * g.wo, tail = g.psp - howo;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (int64_t)g.n * tail) return;
  const int64_t slot = t / tail;
  bw[(int64_t)blockIdx.y * ldb + slot * g.psp + howo + (t - slot * tail)] = 0;
}

// slot weights dA = 1 / s, zA = z + half / s (slot n holds sample perm[n])
// and sum_n zA_n, one block
__global__ __launch_bounds__(256) void conv_psq_weights_kernel(const float* scale, const float* zero,
                                                               const int32_t* perm, int n, int half, ConvPsqSums ps) {
  double zs = 0.0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int smp = perm ? perm[i] : i;
    const double d = 1.0 / (double)scale[smp];
    const double za = (double)zero[smp] + (double)half * d;
    ps.dA[i] = d;
    ps.zA[i] = za;
    zs += za;
  }
  __shared__ double sw[4];
  zs = wave_sum_t<double>(zs);
  if ((threadIdx.x & 63) == 0) sw[threadIdx.x >> 6] = zs;
  __syncthreads();
  if (threadIdx.x == 0) ps.zsum[0] = (sw[0] + sw[1]) + (sw[2] + sw[3]);
}

// out[ch][pix] = sum over slots i of wt[i] codes[ch ld + i pitch + pix] (float64)
// (rows of rw pixels stored rp apart when rp > 0)
__global__ void conv_wsum_kernel(const int8_t* codes, int64_t ld, int64_t pitch, int64_t npix, int64_t nch, int n,
                                 int64_t rw, int64_t rp, const double* wt, double* out) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= nch * npix) return;
  const int64_t ch = t / npix, pix = t - (t / npix) * npix;
  const int64_t off = rp > 0 ? (pix / rw) * rp + pix % rw : pix;
  const int8_t* col = codes + ch * ld + off;
  double s4[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int i = 0; i < n; ++i) s4[i & 3] += wt[i] * (double)col[(int64_t)i * pitch];
  out[t] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
}

// the reduction over slots (split i = slot i), weighted by dA, plus the
// zero-point terms; layout of the work as in conv_gradw_reduce_kernel
__global__ __launch_bounds__(256) void conv_gradw_psq_reduce_kernel(GemmParams p, ConvGeom g, ConvPsqSums ps,
                                                                    const int32_t* count_tap) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t idx = (int64_t)blockIdx.x * 64 + lane;
  const int64_t MN = p.M * p.N;
  const int64_t ic = idx < MN ? idx : MN - 1;
  double s8[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
  int sp = wave;
  for (; sp + 28 < p.splits; sp += 32)
#pragma unroll
    for (int u = 0; u < 8; ++u) s8[u] += ps.dA[sp + 4 * u] * (double)p.part[(int64_t)(sp + 4 * u) * MN + ic];
  for (; sp < p.splits; sp += 4) s8[0] += ps.dA[sp] * (double)p.part[(int64_t)sp * MN + ic];
  __shared__ double swave[4][64];
  swave[wave][lane] = ((s8[0] + s8[1]) + (s8[2] + s8[3])) + ((s8[4] + s8[5]) + (s8[6] + s8[7]));
  __syncthreads();
  if (wave != 0 || idx >= MN) return;
  const double sum = (swave[0][lane] + swave[1][lane]) + (swave[2][lane] + swave[3][lane]);
  const int64_t row = idx / p.N, col = idx % p.N;
  const int taps = g.kh * g.kw;
  const int tap = (int)(col / g.c);
  const double dB = 1.0 / (double)p.scaleB[0];
  const double zB = (double)p.zeroB[0] + (double)p.halfB * dB;
  const double cnt1 = (double)(count_tap[tap] / g.n);
  const double v = dB * sum + zB * ps.WA[row * taps + tap] + dB * ps.WB[col] + zB * cnt1 * ps.zsum[0];
  p.out[row * p.ldo + col] = (float)v;
}

// ---------------------------------------------------------------------------
// grad_X helpers: S_G[pix][slot] = sum_o Q_b2 codes (pixel-major, so that the
// slots of one output pixel are consecutive words); CT[pix_in][c] = sum of W
// codes over the valid taps of an input pixel, cnt[pix_in] = their number
// ---------------------------------------------------------------------------
__global__ void conv_sg_kernel(ConvGeom g, const int8_t* q2, int32_t* sg) {
  // n * ho * wo < 2^31 (checked by the launcher): thread t = pix * n + slot
  const uint32_t howo = (uint32_t)g.ho * (uint32_t)g.wo;
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (uint32_t)g.n * howo) return;
  // Q_b2 codes are pixel-major [pix][slot][o]: thread t reads the t-th run of o codes
  const int8_t* src = q2 + (int64_t)t * g.o;
  int sum = 0;
  if ((g.o & 15) == 0 && ((uintptr_t)q2 & 15) == 0) {
    // 64 channels (four loads in flight) per step, then 16 at a time
    int o = 0;
    for (; o + 64 <= g.o; o += 64) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const uint4*>(src + o + 16 * u);
#pragma unroll
      for (int u = 0; u < 4; ++u) sum = sum4_i8(v[u].x, sum4_i8(v[u].y, sum4_i8(v[u].z, sum4_i8(v[u].w, sum))));
    }
    for (; o < g.o; o += 16) {
      const uint4 v = *reinterpret_cast<const uint4*>(src + o);
      sum = sum4_i8(v.x, sum4_i8(v.y, sum4_i8(v.z, sum4_i8(v.w, sum))));
    }
  } else {
    for (int o = 0; o < g.o; ++o) sum += src[o];
  }
  sg[t] = sum;
}

// taps (r, s) whose output pixel feeds input pixel (iy, ix)
__device__ __forceinline__ bool tap_hits(const ConvGeom& g, int iy, int ix, int r, int s, int& y, int& x) {
  const int ty = iy + g.pad - r, tx = ix + g.pad - s;
  if (ty < 0 || tx < 0 || ty % g.stride || tx % g.stride) return false;
  y = ty / g.stride;
  x = tx / g.stride;
  return y < g.ho && x < g.wo;
}

// Row sums of the grad_X A rows: rs[pix][slot] = sum of S_G[pixel][slot]
// over the output pixels whose taps reach input pixel pix (slot fastest,
// so a wave reads consecutive words of each tap's S_G run).  Stride 1: the
// taps' loads go out together (missing taps read entry 0 and add nothing).
template <bool S1>
__global__ void conv_rs_kernel(ConvGeom g, const int32_t* sg, int32_t* rs) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= (uint32_t)g.n * (uint32_t)(g.h * g.w)) return;
  const uint32_t pix = t / (uint32_t)g.n, slot = t - pix * (uint32_t)g.n;
  const int iy = (int)(pix / (uint32_t)g.w), ix = (int)pix - iy * g.w;
  int sum = 0;
  if constexpr (S1) {
    constexpr int U = 8;  // taps per round of loads
    const int taps = g.kh * g.kw;
    for (int t0 = 0; t0 < taps; t0 += U) {
      int v[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int tap = t0 + u;
        const int r = tap / g.kw, s = tap - r * g.kw;
        const int y = iy + g.pad - r, x = ix + g.pad - s;
        ok[u] = tap < taps && y >= 0 && y < g.ho && x >= 0 && x < g.wo;
        v[u] = sg[ok[u] ? ((int64_t)y * g.wo + x) * g.n + slot : 0];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) sum += ok[u] ? v[u] : 0;
    }
  } else {
    for (int r = 0; r < g.kh; ++r)
      for (int s = 0; s < g.kw; ++s) {
        int y, x;
        if (tap_hits(g, iy, ix, r, s, y, x)) sum += sg[((int64_t)y * g.wo + x) * g.n + slot];
      }
  }
  rs[t] = sum;
}

template <bool S1>
__global__ void conv_ct_kernel(ConvGeom g, const int32_t* swq, int32_t* ct, int32_t* cnt) {
  const int64_t hw = (int64_t)g.h * g.w;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= hw * g.c) return;
  const int64_t pix = t / g.c;
  const int c = (int)(t % g.c);
  const int iy = (int)(pix / g.w), ix = (int)(pix % g.w);
  int sum = 0, n = 0;
  if constexpr (S1) {
    constexpr int U = 8;
    const int taps = g.kh * g.kw;
    for (int t0 = 0; t0 < taps; t0 += U) {
      int v[U];
      bool ok[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int tap = t0 + u;
        const int r = tap / g.kw, s = tap - r * g.kw;
        const int y = iy + g.pad - r, x = ix + g.pad - s;
        ok[u] = tap < taps && y >= 0 && y < g.ho && x >= 0 && x < g.wo;
        v[u] = swq[ok[u] ? (int64_t)tap * g.c + c : 0];
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        sum += ok[u] ? v[u] : 0;
        n += ok[u] ? 1 : 0;
      }
    }
  } else {
    for (int r = 0; r < g.kh; ++r)
      for (int s = 0; s < g.kw; ++s) {
        int y, x;
        if (tap_hits(g, iy, ix, r, s, y, x)) {
          sum += swq[(int64_t)(r * g.kw + s) * g.c + c];
          ++n;
        }
      }
  }
  ct[t] = sum;
  if (c == 0) cnt[pix] = n;
}

// Implicit im2col rows of grad_X: row m = (input pixel m / npad, slot m % npad);
// column k = (tap k / o, channel k % o).  16-byte chunks of 16 channels.
struct ConvXLoader {
  const int8_t* q2;
  ConvGeom g;
  int64_t M, K, D;
  struct Row {
    const int8_t* base;  // this slot's gradient codes
    int iy, ix;          // input pixel
    bool ok;
  };
  // M < 2^31 (checked at launch): the row splits in 32-bit arithmetic
  __device__ __forceinline__ Row row(int64_t m) const {
    Row rw{q2, 0, 0, false};
    if (m >= M) return rw;
    const uint32_t npad = (uint32_t)g.npad;
    const uint32_t pix = (uint32_t)m / npad, slot = (uint32_t)m - pix * npad;
    if (slot >= (uint32_t)g.n) return rw;
    rw.base = q2 + (int64_t)slot * g.o;  // pixel-major codes: slot offset inside each pixel
    rw.iy = (int)(pix / (uint32_t)g.w);
    rw.ix = (int)pix - rw.iy * g.w;
    rw.ok = true;
    return rw;
  }
  struct KState {
    int o0, r, s;  // channel offset and tap of the chunk column
    bool ok;
  };
  __device__ __forceinline__ KState kstate(int64_t k) const {
    KState ks{0, 0, 0, k < K};
    const int kk = (int)k;
    const int tap = kk / g.o;
    ks.o0 = kk - tap * g.o;
    ks.r = tap / g.kw;
    ks.s = tap - ks.r * g.kw;
    return ks;
  }
  __device__ __forceinline__ Chunk16 load(const Row& rw, const KState& ks) const {
    Chunk16 c{{0u, 0u, 0u, 0u}};
    if (!rw.ok || !ks.ok) return c;
    int y, x;
    if (g.stride == 1) {
      // output pixel (iy + pad - r, ix + pad - s): no divisions
      y = rw.iy + g.pad - ks.r;
      x = rw.ix + g.pad - ks.s;
      if (y < 0 || x < 0 || y >= g.ho || x >= g.wo) return c;
    } else if (!tap_hits(g, rw.iy, rw.ix, ks.r, ks.s, y, x)) {
      return c;
    }
    const uint4 v = *reinterpret_cast<const uint4*>(rw.base + ((int64_t)y * g.wo + x) * g.n * g.o + ks.o0);
    c.w[0] = v.x;
    c.w[1] = v.y;
    c.w[2] = v.z;
    c.w[3] = v.w;
    return c;
  }
};

// Stride-1 grad_X loader with at most 32 taps.  A row maps once to the code
// offset of output pixel (iy + pad, ix + pad) of its slot and a bit mask of
// the taps (r, s) whose output pixel (iy + pad - r, ix + pad - s) exists; a
// stage maps its K offset to a tap and the offset of that tap's channels
// relative to the row's pixel.  A chunk is then a bit test and an add; a
// lane whose tap misses reads a 16-byte block of zeros instead, so no lane
// is masked off around the load.
__device__ __attribute__((aligned(16))) int8_t conv_zero16[16];

struct ConvXLoader1 {
  const int8_t* q2;
  ConvGeom g;
  int64_t M, K, D;
  struct Row {
    int64_t off;    // codes of output pixel (iy + pad, ix + pad) of this slot
    uint32_t mask;  // bit r * kw + s: that tap reaches an output pixel
  };
  __device__ __forceinline__ Row row(int64_t m) const {
    Row rw{0, 0u};
    if (m >= M) return rw;
    const uint32_t npad = (uint32_t)g.npad;
    const uint32_t pix = (uint32_t)m / npad, slot = (uint32_t)m - pix * npad;
    if (slot >= (uint32_t)g.n) return rw;
    const int iy = (int)(pix / (uint32_t)g.w), ix = (int)pix - iy * g.w;
    const int yc = iy + g.pad, xc = ix + g.pad;
    uint32_t mask = 0u;
    for (int r = 0; r < g.kh; ++r)
      for (int s = 0; s < g.kw; ++s)
        if (yc - r >= 0 && yc - r < g.ho && xc - s >= 0 && xc - s < g.wo) mask |= 1u << (r * g.kw + s);
    rw.off = (((int64_t)yc * g.wo + xc) * g.n + slot) * g.o;  // pixel-major codes
    rw.mask = mask;
    return rw;
  }
  struct KState {
    int64_t off;  // channel offset of the tap minus its pixel displacement
    int tap;      // 32 (no tap) past the end of K
  };
  __device__ __forceinline__ KState kstate(int64_t k) const {
    KState ks{0, 32};
    if (k >= K) return ks;
    const int kk = (int)k;
    const int tap = kk / g.o;
    const int o0 = kk - tap * g.o;
    const int r = tap / g.kw, s = tap - r * g.kw;
    ks.off = (int64_t)o0 - ((int64_t)r * g.wo + s) * g.n * g.o;
    ks.tap = tap;
    return ks;
  }
  __device__ __forceinline__ Chunk16 load(const Row& rw, const KState& ks) const {
    const bool hit = ks.tap < 32 && ((rw.mask >> ks.tap) & 1u);
    const int8_t* src = hit ? q2 + (rw.off + ks.off) : conv_zero16;
    const uint4 v = *reinterpret_cast<const uint4*>(src);
    return Chunk16{{v.x, v.y, v.z, v.w}};
  }
};

// B operand of the grad_X contraction: the W codes [c][(r, s, o)] (16-byte
// aligned rows, K a multiple of 16).  Rows past N are clamped to the last
// one (their columns are never stored) and chunks past K come from the zero
// block, so the K loop has no branches around its loads.
struct ConvWLoader {
  const int8_t* B;
  int64_t ldb, N, K;
  __device__ __forceinline__ Chunk16 load(int64_t r, int64_t k) const {
    const int64_t rr = r < N ? r : N - 1;
    const int8_t* src = k < K ? B + rr * ldb + k : conv_zero16;
    const uint4 v = *reinterpret_cast<const uint4*>(src);
    return Chunk16{{v.x, v.y, v.z, v.w}};
  }
};

struct ConvRowStage {
  double rterm;  // zW * (codes summed over the valid taps of the row)
  double hz;     // BHQ group row: half + c_g;  affine row: z + half / s
  double dq;     // 1 / s
  int kind;      // BHQ slot kind (0 affine)
  int orow;      // output pixel row (sample * h * w + pixel), -1 if none
};

using CfgConvX = TileCfg<128, 64, 64, 64, 64>;  // 64-code K stages, 36 KB of LDS: four blocks per CU

// The K stages of a grad_X tile: only the taps that reach one of the tile's
// input pixels (a tile's 128 rows hold the slots of at most two pixels).
// With stride 2 about a quarter of the taps reach a pixel, and pixels with
// none (odd ones of a 1 x 1 stride-2 conv) run no K loop at all.  Stage t
// at K offset 64 st[t]; past the list, K (the loaders load zeros).
constexpr int CONVX_MAXST = 512;
struct KStageList {
  const uint16_t* st;
  int64_t n, K;
  __device__ __forceinline__ int64_t k(int64_t t) const { return t < n ? 64 * (int64_t)st[t] : K; }
};

template <int EPI, int KG, class XLoader>
__global__ __launch_bounds__(256) void conv_gradx_kernel(GemmParams p, ConvGeom g, const int8_t* q2, const int32_t* rs,
                                                          const int32_t* ct, const int32_t* cnt) {
  using C = CfgConvX;
  constexpr int EP_BYTES = C::BM * C::BN * 4 + C::BM * (int)sizeof(ConvRowStage);
  constexpr int BYTES = EP_BYTES > C::OP_BYTES ? EP_BYTES : C::OP_BYTES;
  __shared__ __attribute__((aligned(16))) int8_t lds[BYTES];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
  const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
  const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
  const int64_t tile = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  const int64_t m0 = (tile / tiles_n) * C::BM;
  const int64_t n0 = (tile % tiles_n) * C::BN;
  const int lrow = lane & 31;
  const int h = lane >> 5;
  const int64_t D = (int64_t)g.ho * g.wo * g.o;

  v16i acc[C::IT][C::JT];
#pragma unroll
  for (int i = 0; i < C::IT; ++i)
#pragma unroll
    for (int j = 0; j < C::JT; ++j) acc[i][j] = v16i{0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
  const XLoader aload{q2, g, p.M, p.K, D};
  const int taps = g.kh * g.kw;
  const int spt = g.o / 64;  // K stages per tap
  if (taps <= 64 && g.o % 64 == 0 && taps * spt <= CONVX_MAXST) {
    __shared__ uint16_t s_st[CONVX_MAXST];
    __shared__ int s_nst;
    if (wave == 0) {
      // lane i: does tap i reach an input pixel of this tile?
      const uint32_t npad = (uint32_t)g.npad, hw = (uint32_t)(g.h * g.w);
      const uint32_t pa = (uint32_t)m0 / npad;
      const uint32_t last = (uint32_t)((m0 + C::BM - 1 < p.M ? m0 + C::BM - 1 : p.M - 1));
      const uint32_t pb = last / npad;
      bool hit = false;
      if (lane < taps) {
        const int r = lane / g.kw, s2 = lane - (lane / g.kw) * g.kw;
        int y, x;
        for (uint32_t pix = pa; pix <= pb && pix < hw; ++pix) {
          const int iy = (int)(pix / (uint32_t)g.w), ix = (int)pix - iy * g.w;
          if (tap_hits(g, iy, ix, r, s2, y, x)) hit = true;
        }
      }
      const uint64_t mask = __ballot(hit);
      if (hit) {
        const int before = __popcll(mask & ((1ull << lane) - 1ull));
        for (int j = 0; j < spt; ++j) s_st[before * spt + j] = (uint16_t)(lane * spt + j);
      }
      if (lane == 0) s_nst = __popcll(mask) * spt;
    }
    __syncthreads();
    generic_mainloop_km<C>(p, aload, ConvWLoader{p.B, p.ldb, p.N, p.K}, lds, m0, n0, KStageList{s_st, s_nst, p.K},
                           acc);
  } else {
    generic_mainloop<C>(p, aload, ConvWLoader{p.B, p.ldb, p.N, p.K}, lds, m0, n0, 0, p.K, acc);
  }

  int32_t* sacc = reinterpret_cast<int32_t*>(lds);
  ConvRowStage* srow = reinterpret_cast<ConvRowStage*>(lds + C::BM * C::BN * 4);
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
  // Row terms, one thread per tile row.  M < 2^31 (checked by the launcher),
  // so the row splits into (input pixel, slot) in 32-bit arithmetic; S_G is
  // pixel-major, so the slots of one tap read consecutive words.
  if (tid < C::BM) {
    const int64_t m = m0 + tid;
    ConvRowStage q{};
    q.orow = -1;
    const uint32_t npad = (uint32_t)g.npad;
    const uint32_t pix = (uint32_t)m / npad, slot = (uint32_t)m - pix * npad;
    if (m < p.M && slot < (uint32_t)g.n) {
      const float s = p.rowwiseA ? p.scaleA[slot] : p.scaleA[0];
      const float z = p.rowwiseA ? p.zeroA[slot] : p.zeroA[0];
      q.kind = (EPI == EPI_BHQ) ? bhq_slot_kind(p.L, slot) : (EPI == EPI_BHQT ? (p.slot[slot].size > 1) : 0);
      q.rterm = zW * (double)rs[(int64_t)pix * g.n + slot];
      q.dq = 1.0 / (double)s;
      q.hz = q.kind != 0 ? (double)p.halfA + (double)z : (double)z + (double)p.halfA * q.dq;
      q.orow = (int)((p.perm ? (int64_t)p.perm[slot] : (int64_t)slot) * ((int64_t)g.h * g.w) + pix);
    }
    srow[tid] = q;
  }
  __syncthreads();
  // Wave w owns the 64 tile rows [64 w, 64 w + 64): one run, the slots of one
  // input pixel (npad % 64 == 0), so the column terms are loaded once.  Lane
  // l holds the four columns n0 + 4 (l % 16) .. +3 of row 4 i + l / 16 in
  // step i, so one step covers four rows and stores 16-byte words.  A BHQ
  // group of KG rows (KG <= 64, aligned) lies inside the run; its column sums
  // meet across the four row lanes by xor shuffles, which give every lane of
  // the group the same sum.
  constexpr int WROWS = C::BM / C::WAVES;
  static_assert(C::BN == 64 && WROWS == 64 && KG <= 64, "epilogue wave layout");
  const int r0 = wave * WROWS;
  const int cq = lane & 15, rsub = lane >> 4;
  const int64_t col = n0 + 4 * cq;
  if (col >= p.N || m0 + r0 >= p.M) return;
  const bool vec = col + 3 < p.N && (p.ldo & 3) == 0 && ((uintptr_t)p.out & 15) == 0;
  const int64_t pix = (int64_t)((uint32_t)(m0 + r0) / (uint32_t)g.npad);
  const double kz = (double)cnt[pix] * ((double)g.o * zW);
  double colterm[4];
#pragma unroll
  for (int e = 0; e < 4; ++e)
    colterm[e] = col + e < p.N ? dW * (double)ct[pix * g.c + col + e] + kz : 0.0;
  auto row_acc = [&](int row, double (&a)[4]) {
    const int4 v = *reinterpret_cast<const int4*>(&sacc[row * C::BN + 4 * cq]);
    a[0] = (double)v.x;
    a[1] = (double)v.y;
    a[2] = (double)v.z;
    a[3] = (double)v.w;
  };
  auto store = [&](int orow, const double (&v)[4]) {
    float* dst = p.out + (int64_t)orow * p.ldo + col;
    if (vec) {
      *reinterpret_cast<float4*>(dst) = make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (col + e < p.N) dst[e] = (float)v[e];
    }
  };
  if constexpr (EPI == EPI_BHQ && KG > 1) {
    constexpr int RB = KG > 4 ? KG : 4;  // rows per block of steps
    for (int blk = r0; blk < r0 + WROWS; blk += RB) {
      double S[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
      for (int i = 0; i < RB / 4; ++i) {
        const int row = blk + 4 * i + rsub;
        const ConvRowStage& q = srow[row];
        double a[4];
        row_acc(row, a);
        if (q.kind != 0) {
#pragma unroll
          for (int e = 0; e < 4; ++e) S[e] += dW * a[e] + (q.rterm + q.hz * colterm[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        S[e] += __shfl_xor(S[e], 16);
        if constexpr (KG >= 4) S[e] += __shfl_xor(S[e], 32);
      }
      const int g0 = (blk + rsub) & ~(KG - 1);  // first row of this lane's group
      const ConvRowStage& q0 = srow[g0];
      if (q0.orow < 0 && q0.kind == 0) continue;
      double a0[4], tau[4];
      row_acc(g0, a0);
      const double alpha = q0.kind == 2 ? p.L.inv_sk_p : p.L.inv_sk_k;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double T0 = dW * a0[e] + (q0.rterm + q0.hz * colterm[e]);
        tau[e] = (alpha * S[e] - T0) / (1.0 - alpha);
      }
#pragma unroll 4
      for (int i = 0; i < RB / 4; ++i) {
        const int row = blk + 4 * i + rsub;
        const ConvRowStage& q = srow[row];
        if (q.orow < 0) continue;
        double a[4], v[4];
        row_acc(row, a);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (q.kind != 0) {
            const double T = dW * a[e] + (q.rterm + q.hz * colterm[e]);
            const double Z = (row == g0) ? T + (1.0 - alpha) * tau[e] : T - alpha * tau[e];
            v[e] = Z * q.dq;
          } else {
            v[e] = q.dq * (dW * a[e] + q.rterm) + q.hz * colterm[e];
          }
        }
        store(q.orow, v);
      }
    }
  } else {
#pragma unroll 4
    for (int i = 0; i < WROWS / 4; ++i) {
      const int row = r0 + 4 * i + rsub;
      const ConvRowStage& q = srow[row];
      if (q.orow < 0) continue;
      double a[4], v[4];
      row_acc(row, a);
      if (EPI == EPI_BHQT && q.kind != 0) {
        // a row of a multi-row group of the general plan: its T for the inverse pass
        double* dst = p.tbuf + (m0 + row) * p.ldt + col;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < p.N) dst[e] = dW * a[e] + (q.rterm + q.hz * colterm[e]);
        continue;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = q.dq * (dW * a[e] + q.rterm) + q.hz * colterm[e];
      store(q.orow, v);
    }
  }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_conv_wq(const float* W, const ConvGeom& g, int bits, const float* scale, const float* zero,
                          int8_t* wq_t, int32_t* swq, hipStream_t s) {
  const int64_t n = (int64_t)g.kh * g.kw * g.c;
  hipLaunchKernelGGL(conv_wq_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s, W, g, bits, scale, zero, wq_t,
                     swq);
  return hipGetLastError();
}

hipError_t launch_conv_im2col_w_t(const ConvGeom& gi, const int8_t* xq_t, int8_t* bw, int64_t ldb, int32_t* xs,
                                  int32_t* sumB, const ConvGeom& g, hipStream_t s);

hipError_t launch_conv_im2col_w(const ConvGeom& g, const int8_t* xq_t, int8_t* bw, int64_t ldb, int32_t* xs,
                                int32_t* sumB, hipStream_t s) {
  if (g.gwp > 0) {
    // the kw shifted copies of the zero-halo grid: the im2col kernels on a
    // one-row kernel whose output rows are the ghp grid rows of gwp bytes
    ConvGeom gg = g;
    gg.kh = 1;
    gg.ho = (int)g.ghp;
    gg.wo = (int)g.gwp;
    if (g.stride != 1 || g.ghp != g.h + 2 * g.pad || g.gwp < g.w + 2 * g.pad || (g.gwp & 15) != 0 ||
        g.psp < g.ghp * g.gwp || ldb != g.ldx || g.kw > g.gwp)
      return hipErrorInvalidValue;
    if ((g.w & 3) == 0 && g.kw <= XGRID_MAXKW && (((uintptr_t)xq_t) & 3) == 0 && (((uintptr_t)bw) & 15) == 0) {
      const int64_t nt = (int64_t)g.c * g.n * g.ghp * (g.gwp >> 4);
      if ((nt + 255) / 256 > 0x7FFFFFFF) return hipErrorInvalidValue;
      hipLaunchKernelGGL(conv_xgrid_kernel, dim3((unsigned)((nt + 255) / 256)), dim3(256), 0, s, g, xq_t, bw);
      return launch_conv_im2col_w_t(gg, xq_t, nullptr, ldb, xs, sumB, g, s);
    }
    return launch_conv_im2col_w_t(gg, xq_t, bw, ldb, xs, sumB, g, s);
  }
  return launch_conv_im2col_w_t(g, xq_t, bw, ldb, xs, sumB, g, s);
}

// gi: the geometry the codes are laid out for (im2col, or the grid copies);
// g: the conv's own (for the zero-point sums)
hipError_t launch_conv_im2col_w_t(const ConvGeom& gi, const int8_t* xq_t, int8_t* bw, int64_t ldb, int32_t* xs,
                                  int32_t* sumB, const ConvGeom& g, hipStream_t s) {
  const int64_t rows = (int64_t)gi.kh * gi.kw * gi.c;
  if (rows > 65535 || gi.psp < (int64_t)gi.ho * gi.wo || ldb < (int64_t)gi.n * gi.psp || (ldb & 15) != 0)
    return hipErrorInvalidValue;
  if (!bw) {
    // the codes are laid out already: only the zero-point sums
  } else if (conv_im2col_rows_ok(gi, xq_t, bw, ldb)) {
    // stride 1, rows of 4-byte words: one thread per output word
    const int spb = 256 * IM2COL_WPT / (gi.wo / 4);
    const int64_t blocks = ((int64_t)gi.n * gi.ho + spb - 1) / spb;
    if (spb < 1 || blocks > 0x7FFFFFFF || (int64_t)gi.n * gi.ho + 256 * IM2COL_WPT > 0x7FFFFFFF)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL(conv_im2col_rows_kernel, dim3((unsigned)blocks, (unsigned)rows), dim3(256), 0, s, gi, xq_t, bw,
                       ldb, spb);
    if (gi.psp > (int64_t)gi.ho * gi.wo) {
      const int64_t nt = (int64_t)gi.n * (gi.psp - (int64_t)gi.ho * gi.wo);
      if ((nt + 255) / 256 > 0x7FFFFFFF) return hipErrorInvalidValue;
      hipLaunchKernelGGL(conv_pitch_zero_kernel, dim3((unsigned)((nt + 255) / 256), (unsigned)rows), dim3(256), 0, s,
                         gi, bw, ldb);
    }
  } else {
    const int64_t chunks = (ldb + 16 * 256 - 1) / (16 * 256);
    if (chunks > 0x7FFFFFFF) return hipErrorInvalidValue;
    hipLaunchKernelGGL(conv_im2col_w_kernel, dim3((unsigned)chunks, (unsigned)rows), dim3(256), 0, s, gi, xq_t, bw,
                       ldb);
  }
  if (!xs) return hipGetLastError();  // per-sample Q_b1 forms its own sums
  const int64_t nx = (int64_t)g.c * g.h * g.w;
  hipLaunchKernelGGL(conv_xsum_kernel, dim3((unsigned)((nx + 255) / 256)), dim3(256), 0, s, g, xq_t, xs);
  hipLaunchKernelGGL(conv_xtapsum_kernel<int32_t>, dim3((unsigned)((int64_t)g.kh * g.kw * g.c)), dim3(256), 0, s, g,
                     xs, sumB);
  return hipGetLastError();
}

hipError_t launch_conv_tapsums(const ConvGeom& g, const int8_t* q1_t, int64_t ldq, int32_t* qs, int32_t* sumA_tap,
                               int32_t* count_tap, hipStream_t s) {
  const int64_t n1 = (int64_t)g.o * g.ho * g.wo;
  hipLaunchKernelGGL(conv_qsum_kernel, dim3((unsigned)((n1 + 255) / 256)), dim3(256), 0, s, g, q1_t, ldq, qs);
  const int64_t n2 = (int64_t)g.o * g.kh * g.kw;
  hipLaunchKernelGGL(conv_tapsum_kernel<int32_t>, dim3((unsigned)n2), dim3(256), 0, s, g, qs, sumA_tap, count_tap);
  return hipGetLastError();
}

hipError_t launch_conv_gradw_reduce(const GemmParams& p, const ConvGeom& g, const int32_t* sumA_tap,
                                    const int32_t* count_tap, hipStream_t s) {
  const int64_t MN = p.M * p.N;
  if (MN < 1 || (MN + 63) / 64 > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(conv_gradw_reduce_kernel, dim3((unsigned)((MN + 63) / 64)), dim3(256), 0, s, p, g, sumA_tap,
                     count_tap);
  return hipGetLastError();
}

hipError_t launch_conv_psq_sums(const ConvGeom& g, const float* scale, const float* zero, const int32_t* perm,
                                int half, const int8_t* q1_t, int64_t ldq, const int8_t* xq_t, const ConvPsqSums& ps,
                                int32_t* count_tap, hipStream_t s) {
  const int64_t howo = (int64_t)g.ho * g.wo, hw = (int64_t)g.h * g.w;
  const int64_t taps = (int64_t)g.kh * g.kw;
  const int64_t n1 = (int64_t)g.o * howo, n2 = (int64_t)g.c * hw;
  if ((n1 + 255) / 256 > 0x7FFFFFFF || (n2 + 255) / 256 > 0x7FFFFFFF || g.o * taps > 0x7FFFFFFF ||
      taps * g.c > 65535)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(conv_psq_weights_kernel, dim3(1), dim3(256), 0, s, scale, zero, perm, g.n, half, ps);
  hipLaunchKernelGGL(conv_wsum_kernel, dim3((unsigned)((n1 + 255) / 256)), dim3(256), 0, s, q1_t, ldq, g.psp, howo,
                     (int64_t)g.o, g.n, (int64_t)g.wo, g.gwp, (const double*)ps.dA, ps.qw);
  hipLaunchKernelGGL(conv_wsum_kernel, dim3((unsigned)((n2 + 255) / 256)), dim3(256), 0, s, xq_t, g.n * hw, hw, hw,
                     (int64_t)g.c, g.n, (int64_t)0, (int64_t)0, (const double*)ps.zA, ps.xw);
  hipLaunchKernelGGL(conv_tapsum_kernel<double>, dim3((unsigned)(g.o * taps)), dim3(256), 0, s, g,
                     (const double*)ps.qw, ps.WA, count_tap);
  hipLaunchKernelGGL(conv_xtapsum_kernel<double>, dim3((unsigned)(taps * g.c)), dim3(256), 0, s, g,
                     (const double*)ps.xw, ps.WB);
  return hipGetLastError();
}

hipError_t launch_conv_gradw_psq_reduce(const GemmParams& p, const ConvGeom& g, const ConvPsqSums& ps,
                                        const int32_t* count_tap, hipStream_t s) {
  const int64_t MN = p.M * p.N;
  if (MN < 1 || (MN + 63) / 64 > 0x7FFFFFFF || p.splits != g.n) return hipErrorInvalidValue;
  hipLaunchKernelGGL(conv_gradw_psq_reduce_kernel, dim3((unsigned)((MN + 63) / 64)), dim3(256), 0, s, p, g, ps,
                     count_tap);
  return hipGetLastError();
}

hipError_t launch_conv_gradx_prep(const ConvGeom& g, const int8_t* q2, const int32_t* swq, int32_t* sg, int32_t* rs,
                                  int32_t* ct,
                                  int32_t* cnt, hipStream_t s) {
  const int64_t n1 = (int64_t)g.n * g.ho * g.wo;
  if (n1 > 0x7FFFFFFF) return hipErrorInvalidValue;
  hipLaunchKernelGGL(conv_sg_kernel, dim3((unsigned)((n1 + 255) / 256)), dim3(256), 0, s, g, q2, sg);
  const int64_t nr = (int64_t)g.n * g.h * g.w;
  if (nr > 0x7FFFFFFF) return hipErrorInvalidValue;
  if (g.stride == 1)
    hipLaunchKernelGGL(conv_rs_kernel<true>, dim3((unsigned)((nr + 255) / 256)), dim3(256), 0, s, g, (const int32_t*)sg,
                       rs);
  else
    hipLaunchKernelGGL(conv_rs_kernel<false>, dim3((unsigned)((nr + 255) / 256)), dim3(256), 0, s, g, (const int32_t*)sg,
                       rs);
  const int64_t n2 = (int64_t)g.h * g.w * g.c;
  if (g.stride == 1)
    hipLaunchKernelGGL(conv_ct_kernel<true>, dim3((unsigned)((n2 + 255) / 256)), dim3(256), 0, s, g, swq, ct, cnt);
  else
    hipLaunchKernelGGL(conv_ct_kernel<false>, dim3((unsigned)((n2 + 255) / 256)), dim3(256), 0, s, g, swq, ct, cnt);
  return hipGetLastError();
}

template <int EPI, int KG>
static hipError_t launch_conv_gradx_t(const GemmParams& p, const ConvGeom& g, const int8_t* q2, const int32_t* rs,
                                      const int32_t* ct, const int32_t* cnt, hipStream_t s) {
  const int64_t tiles = ((p.M + CfgConvX::BM - 1) / CfgConvX::BM) * ((p.N + CfgConvX::BN - 1) / CfgConvX::BN);
  if (tiles > 0x7FFFFFFF || p.M > 0x7FFFFFFF || g.npad % 64 != 0) return hipErrorInvalidValue;
  // q2 is a workspace carve (16-byte aligned); o % 16 == 0 keeps every chunk aligned
  if (g.stride == 1 && g.kh * g.kw <= 32)
    hipLaunchKernelGGL((conv_gradx_kernel<EPI, KG, ConvXLoader1>), dim3((unsigned)tiles), dim3(CfgConvX::THREADS), 0,
                       s, p, g, q2, rs, ct, cnt);
  else
    hipLaunchKernelGGL((conv_gradx_kernel<EPI, KG, ConvXLoader>), dim3((unsigned)tiles), dim3(CfgConvX::THREADS), 0,
                       s, p, g, q2, rs, ct, cnt);
  return hipGetLastError();
}

hipError_t launch_conv_gradx(const GemmParams& p, int epi, const ConvGeom& g, const int8_t* q2, const int32_t* rs,
                             const int32_t* ct, const int32_t* cnt, hipStream_t s) {
  if (epi == EPI_ROW) return launch_conv_gradx_t<EPI_ROW, 0>(p, g, q2, rs, ct, cnt, s);
  if (epi == EPI_BHQT)
    return p.slot && p.tbuf ? launch_conv_gradx_t<EPI_BHQT, 0>(p, g, q2, rs, ct, cnt, s) : hipErrorInvalidValue;
  switch (p.L.k) {
    case 1: return launch_conv_gradx_t<EPI_BHQ, 1>(p, g, q2, rs, ct, cnt, s);
    case 2: return launch_conv_gradx_t<EPI_BHQ, 2>(p, g, q2, rs, ct, cnt, s);
    case 4: return launch_conv_gradx_t<EPI_BHQ, 4>(p, g, q2, rs, ct, cnt, s);
    case 8: return launch_conv_gradx_t<EPI_BHQ, 8>(p, g, q2, rs, ct, cnt, s);
    case 16: return launch_conv_gradx_t<EPI_BHQ, 16>(p, g, q2, rs, ct, cnt, s);
    case 32: return launch_conv_gradx_t<EPI_BHQ, 32>(p, g, q2, rs, ct, cnt, s);
    case 64: return launch_conv_gradx_t<EPI_BHQ, 64>(p, g, q2, rs, ct, cnt, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace fqt
