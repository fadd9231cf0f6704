// C ABI of libfqt.so (declared in include/fqt.h): argument checks, workspace
// carving and the launch sequence of each entry point.
#include <string.h>

#include <mutex>

#include "../../include/fqt.h"
#include "fqt_device.h"
#include "fqt_kernels.h"

namespace fqt {
namespace {

constexpr int64_t MAX_K_CHUNK = 65536;  // int32-exact K per contraction split
constexpr int64_t MAX_ROWS = 65535LL * 64;  // quantizer grid limit (64 slots per tile row)

// Bump allocator over the caller's workspace; with base == nullptr it only
// measures.  Every block is 256-byte aligned.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(int64_t count) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += (size_t)count * sizeof(T);
    return p;
  }
};

// Fixed header at the start of every workspace: the status word.
struct Header {
  uint32_t* status;
};
Header take_header(Carver& c) { return Header{c.take<uint32_t>(64)}; }

bool valid_bits(int b) { return b >= 1 && b <= 8; }

// Optional phase markers of fqt_bwd_cfg.trace.
struct Tracer {
  const fqt_trace* t;
  hipStream_t s;
  void begin(int i) const {
    if (t && i < t->count && t->start[i]) (void)hipEventRecord(static_cast<hipEvent_t>(t->start[i]), s);
  }
  void end(int i) const {
    if (t && i < t->count && t->stop[i]) (void)hipEventRecord(static_cast<hipEvent_t>(t->stop[i]), s);
  }
};
// Block sizes the aligned fast path takes (groups inside 64-row tiles); any
// other size, and 0 (App. D), go through the general plan.
bool aligned_block(int k) { return k >= 1 && k <= 64 && (k & (k - 1)) == 0; }
// App. D scores every number of groups, O(rows^2) terms.
constexpr int64_t APPD_MAX_ROWS = 65536;

#define FQT_TRY(expr)                              \
  do {                                             \
    const hipError_t e_ = (expr);                  \
    if (e_ != hipSuccess) return FQT_EDEVICE;      \
  } while (0)

// ---------------------------------------------------------------------------
// standalone quantizers
// ---------------------------------------------------------------------------
// Workspace pieces of a block Householder plan: the sort, and for the
// general plan (App. D, or a block size the aligned path does not take) the
// sorted-position scalars, slot records and the forward transform's
// per-group column term.  group_off / num_groups stand in when the caller
// gives none.
struct BhqWs {
  void* plan;
  bool general;
  AppdWs appd;
  SlotInfo* slot;
  float* tau;
  int32_t* group_off;
  int32_t* num_groups;
};

BhqWs carve_bhq(Carver& c, int64_t rows, int64_t cols, int block_size) {
  BhqWs b{};
  b.plan = c.take<char>((int64_t)bhq_plan_workspace(rows));
  b.general = !aligned_block(block_size);
  b.group_off = c.take<int32_t>(rows + 1);
  b.num_groups = c.take<int32_t>(1);
  if (b.general) {
    void* ap = c.take<char>((int64_t)appd_workspace(rows));
    if (ap) b.appd = appd_carve(ap, rows);
    b.slot = c.take<SlotInfo>(rows);
    b.tau = c.take<float>((rows + 1) / 2 * cols);
  }
  return b;
}

// The plan of a BHQ quantization, asynchronous: perm, per-slot scale / zero,
// group offsets and the number of groups (and the slot records for the
// general plan).  fin: the finalize step to run inside the first launch.
fqt_status plan_bhq(const BhqWs& b, const float* rmin, const float* rmax, int64_t rows, int bits, int block_size,
                    int32_t* perm, float* scale, float* zero, int32_t* group_off, int32_t* num_groups,
                    const FinalizePlan* fin, hipStream_t s) {
  int32_t* goff = group_off ? group_off : b.group_off;
  int32_t* ng = num_groups ? num_groups : b.num_groups;
  if (!b.general) {
    // the aligned layout's group count is known here: stored only when asked for
    const BhqLayout L = bhq_layout(rows, block_size);
    FQT_TRY(launch_bhq_plan(rmin, rmax, L, bits, b.plan, perm, scale, zero, goff, num_groups, fin, s));
    return FQT_OK;
  }
  FQT_TRY(launch_bhq_sort(rmin, rmax, rows, b.plan, b.appd.sigma, fin, s));
  FQT_TRY(launch_general_plan(rmin, rmax, rows, bits, block_size, b.appd, nullptr, perm, scale, zero, goff, b.slot,
                              ng, s));
  return FQT_OK;
}

// Quantizer parameters of a planned BHQ: the aligned layout, or the general
// plan with its per-group column term computed here (after the plan).
fqt_status bhq_params(const BhqWs& b, const float* x, int64_t rows, int64_t cols, int block_size,
                      const int32_t* perm, const float* scale, QuantParams& p, hipStream_t s) {
  if (!b.general) {
    p.L = bhq_layout(rows, block_size);
    return FQT_OK;
  }
  FQT_TRY(launch_bhq_tau(x, rows, cols, perm, scale, b.slot, b.tau, s));
  p.L = BhqLayout{};
  p.L.rows = rows;
  p.L.k = 0;
  p.slot = b.slot;
  p.tau = b.tau;
  return FQT_OK;
}

// Whether a BHQ block size is valid (>= 0) and, for App. D (0), within its rows limit.
fqt_status check_block(int block_size, int64_t rows) {
  if (block_size < 0) return FQT_EINVAL;
  if (block_size == 0 && rows > APPD_MAX_ROWS) return FQT_EUNSUPPORTED;
  return FQT_OK;
}

// ---------------------------------------------------------------------------
// standalone quantizers
// ---------------------------------------------------------------------------
struct QuantWs {
  Header h;
  StatsSeg seg;
  float* rmin;
  float* rmax;
  BhqWs bhq;
  float* tscale;  // FQT_SHIFT: the per-tensor step scale s
};

QuantWs carve_quant(Carver& c, fqt_kind kind, const float* x, int64_t rows, int64_t cols, int block_size = 1) {
  QuantWs w{};
  w.h = take_header(c);
  w.seg = kind == FQT_PTQ ? stats_flat_seg(x, rows * cols) : stats_rows_seg(x, rows, cols);
  w.seg.part = c.take<float2>(stats_partials(w.seg));
  if (kind != FQT_PTQ) {
    w.rmin = c.take<float>(rows);
    w.rmax = c.take<float>(rows);
    stats_direct_rows(w.seg, w.rmin, w.rmax);
  }
  if (kind == FQT_BHQ) w.bhq = carve_bhq(c, rows, cols, block_size);
  if (kind == FQT_SHIFT) w.tscale = c.take<float>(1);
  return w;
}

void add_zero(FinalizePlan& fp, int32_t* p, int64_t n) {
  if (p && n > 0) {
    fp.zero_i32[fp.nzero] = p;
    fp.zero_n[fp.nzero] = n;
    ++fp.nzero;
  }
}

fqt_status check_quant_args(const float* x, int64_t rows, int64_t cols, int bits, const fqt_qtensor* out,
                            bool need_q = true) {
  if (!x || !out || (need_q && !out->q) || !out->scale || !out->zero) return FQT_EINVAL;
  if (rows < 1 || cols < 1 || !valid_bits(bits)) return FQT_EINVAL;
  if (rows > MAX_ROWS || cols > ((int64_t)1 << 40) / rows) return FQT_EUNSUPPORTED;
  return FQT_OK;
}

// nseeds > 0: the seed batch (sums of the codes and of their squares over the
// keys seed .. seed + nseeds - 1 into sum_c / sum_c2) instead of the codes.
fqt_status quantize_common(fqt_kind kind, const float* x, int64_t rows, int64_t cols, int bits, int stochastic,
                           uint64_t seed, uint32_t stream, int transpose, int block_size, const fqt_qtensor* out,
                           void* ws, size_t ws_bytes, hipStream_t s, int nseeds = 0, int32_t* sum_c = nullptr,
                           int32_t* sum_c2 = nullptr) {
  fqt_status st = check_quant_args(x, rows, cols, bits, out, nseeds == 0);
  if (st != FQT_OK) return st;
  if (kind == FQT_BHQ) {
    if (!out->perm) return FQT_EINVAL;
    st = check_block(block_size, rows);
    if (st != FQT_OK) return st;
  }
  if (kind == FQT_SHIFT && !out->shift) return FQT_EINVAL;
  if (!ws) return FQT_EWORKSPACE;
  Carver cs(nullptr);
  carve_quant(cs, kind, x, rows, cols, block_size);
  if (ws_bytes < cs.off) return FQT_EWORKSPACE;
  Carver c(ws);
  QuantWs w = carve_quant(c, kind, x, rows, cols, block_size);

  StatsPlan sp{};
  sp.seg[0] = w.seg;
  sp.nseg = 1;
  FQT_TRY(launch_stats(sp, s));
  FinalizePlan fp{};
  fp.seg[0] = w.seg;
  fp.nseg = 1;
  fp.row_seg = kind == FQT_PTQ ? -1 : 0;
  fp.rmin = w.rmin;
  fp.rmax = w.rmax;
  fp.status = w.h.status;
  if (kind != FQT_BHQ) {
    const int per_row = kind == FQT_SHIFT ? 2 : (kind == FQT_PSQ ? 1 : 0);
    fp.out[0] = ScaleOut{0, bits, per_row, out->scale, out->zero, out->shift, w.tscale};
    fp.nout = 1;
  }
  add_zero(fp, out->code_sum, transpose ? cols : rows);
  if (kind == FQT_BHQ) add_zero(fp, bhq_plan_carve(w.bhq.plan, rows).rank, rows);
  // with row ranges straight from the statistics kernel, the BHQ plan's first
  // launch also runs the finalize step
  const bool fin_in_plan = kind == FQT_BHQ && w.seg.rmin != nullptr;
  if (!fin_in_plan) FQT_TRY(launch_finalize(fp, s));

  QuantParams p{};
  p.x = x;
  p.rows = rows;
  p.cols = cols;
  p.bits = bits;
  p.stoch = stochastic;
  p.seed = seed;
  p.stream = stream;
  p.scale = out->scale;
  p.zero = out->zero;
  if (transpose) {
    p.q_t = out->q;
    p.sum_t = out->code_sum;
  } else {
    p.q_nat = out->q;
    p.sum_nat = out->code_sum;
  }
  int mode = QM_TENSOR;
  if (kind == FQT_PSQ || kind == FQT_SHIFT) {
    mode = QM_ROW;
    if (kind == FQT_SHIFT) p.shift = out->shift;
  } else if (kind == FQT_BHQ) {
    st = plan_bhq(w.bhq, w.rmin, w.rmax, rows, bits, block_size, out->perm, out->scale, out->zero, out->group_off,
                  out->num_groups, fin_in_plan ? &fp : nullptr, s);
    if (st != FQT_OK) return st;
    st = bhq_params(w.bhq, x, rows, cols, block_size, out->perm, out->scale, p, s);
    if (st != FQT_OK) return st;
    p.perm = out->perm;
    mode = QM_BHQ;
  }
  if (nseeds > 0) {
    p.q_nat = nullptr;
    p.sum_nat = nullptr;
    p.nseeds = nseeds;
    p.sum_c = sum_c;
    p.sum_c2 = sum_c2;
    FQT_TRY(launch_quant_seeds(p, mode, s));
    return FQT_OK;
  }
  FQT_TRY(launch_quant(p, mode, s));
  return FQT_OK;
}

// ---------------------------------------------------------------------------
// linear backward
// ---------------------------------------------------------------------------
struct LinearWs {
  Header h;
  StatsSeg sx_seg, sw_seg, sg_seg;
  float *rmin, *rmax;
  int8_t *qx_t, *qw_t, *qg1_t, *qg2;
  int32_t *sum_x, *sum_w, *sum_g1, *sum_g2;
  float *sx, *zx, *sw, *zw, *sg1, *zg1, *sg2, *zg2;
  int32_t* perm;
  BhqWs bhq;
  double* tbuf;      // general BHQ plan: T rows of multi-row groups [N, d_in]
  int32_t* part;
  int splits;
  int8_t* shift1;    // Q_b1 = FQT_SHIFT: per-row shifts, step scale, zero-point terms and column vector
  float* tscale1;
  double* zeta1;
  double* colvec;
  double* colvec_part;
};

int linear_splits(int64_t N) { return (int)((N + MAX_K_CHUNK - 1) / MAX_K_CHUNK); }

LinearWs carve_linear(Carver& c, const float* X, const float* W, const float* G, int64_t N, int64_t d_in,
                      int64_t d_out, const fqt_bwd_cfg& cfg) {
  LinearWs w{};
  w.h = take_header(c);
  w.sx_seg = stats_flat_seg(X, N * d_in);
  w.sw_seg = stats_flat_seg(W, d_out * d_in);
  w.sg_seg = stats_rows_seg(G, N, d_out);
  w.sx_seg.part = c.take<float2>(stats_partials(w.sx_seg));
  w.sw_seg.part = c.take<float2>(stats_partials(w.sw_seg));
  w.sg_seg.part = c.take<float2>(stats_partials(w.sg_seg));
  w.rmin = c.take<float>(N);
  w.rmax = c.take<float>(N);
  stats_direct_rows(w.sg_seg, w.rmin, w.rmax);
  w.qx_t = c.take<int8_t>(d_in * N);
  w.qw_t = c.take<int8_t>(d_in * d_out);
  w.qg1_t = c.take<int8_t>(d_out * N);
  w.qg2 = c.take<int8_t>(N * d_out);
  w.sum_x = c.take<int32_t>(d_in);
  w.sum_w = c.take<int32_t>(d_in);
  w.sum_g1 = c.take<int32_t>(d_out);
  w.sum_g2 = c.take<int32_t>(N);
  w.sx = c.take<float>(1);
  w.zx = c.take<float>(1);
  w.sw = c.take<float>(1);
  w.zw = c.take<float>(1);
  const bool shift = cfg.qb_w.kind == FQT_SHIFT;
  w.sg1 = c.take<float>(shift ? N : 1);
  w.zg1 = c.take<float>(shift ? N : 1);
  if (shift) {
    w.shift1 = c.take<int8_t>(N);
    w.tscale1 = c.take<float>(1);
    w.zeta1 = c.take<double>(N);
    w.colvec = c.take<double>(d_in);
    w.colvec_part = c.take<double>(colvec_splits(N) * (d_in + 1));
  }
  w.sg2 = c.take<float>(N);
  w.zg2 = c.take<float>(N);
  if (cfg.qb_x.kind == FQT_BHQ) {
    w.perm = c.take<int32_t>(N);
    w.bhq = carve_bhq(c, N, d_out, cfg.qb_x.block_size);
    if (w.bhq.general) w.tbuf = c.take<double>(N * d_in);
  }
  w.splits = linear_splits(N);
  if (w.splits > 1) w.part = c.take<int32_t>((int64_t)w.splits * d_out * d_in);
  return w;
}

// ---------------------------------------------------------------------------
// linear forward
// ---------------------------------------------------------------------------
struct ForwardWs {
  Header h;
  StatsSeg sx_seg, sw_seg;
  int8_t *qx, *qw;
  int32_t *sum_x, *sum_w;
  float *sx, *zx, *sw, *zw;
  int32_t* part;
  int splits;
};

ForwardWs carve_forward(Carver& c, const float* X, const float* W, int64_t N, int64_t d_in, int64_t d_out) {
  ForwardWs w{};
  w.h = take_header(c);
  w.sx_seg = stats_flat_seg(X, N * d_in);
  w.sw_seg = stats_flat_seg(W, d_out * d_in);
  w.sx_seg.part = c.take<float2>(stats_partials(w.sx_seg));
  w.sw_seg.part = c.take<float2>(stats_partials(w.sw_seg));
  w.qx = c.take<int8_t>(N * d_in);
  w.qw = c.take<int8_t>(d_out * d_in);
  w.sum_x = c.take<int32_t>(N);
  w.sum_w = c.take<int32_t>(d_out);
  w.sx = c.take<float>(1);
  w.zx = c.take<float>(1);
  w.sw = c.take<float>(1);
  w.zw = c.take<float>(1);
  w.splits = (int)((d_in + MAX_K_CHUNK - 1) / MAX_K_CHUNK);
  if (w.splits > 1) w.part = c.take<int32_t>((int64_t)w.splits * N * d_out);
  return w;
}

fqt_status check_cfg(const fqt_bwd_cfg* cfg) {
  if (!cfg) return FQT_EINVAL;
  if (!valid_bits(cfg->f_bits) || !valid_bits(cfg->theta_bits) || !valid_bits(cfg->qb_w.bits) ||
      !valid_bits(cfg->qb_x.bits))
    return FQT_EINVAL;
  if (cfg->qb_x.kind < FQT_PTQ || cfg->qb_x.kind > FQT_SHIFT || cfg->qb_w.kind < FQT_PTQ ||
      cfg->qb_w.kind > FQT_SHIFT)
    return FQT_EINVAL;
  if (cfg->qb_w.kind == FQT_BHQ || cfg->qb_x.kind == FQT_SHIFT) return FQT_EUNSUPPORTED;
  if (cfg->qb_x.kind == FQT_BHQ && cfg->qb_x.block_size < 0) return FQT_EINVAL;
  if (cfg->relu_input != 0 && cfg->relu_input != 1) return FQT_EINVAL;
  if (cfg->packed_codes != 0 && cfg->packed_codes != 1) return FQT_EINVAL;
  return FQT_OK;
}

// ---------------------------------------------------------------------------
// conv backward
// ---------------------------------------------------------------------------
fqt_status check_conv_shape(const fqt_conv_shape& sh) {
  if (sh.n < 1 || sh.c < 1 || sh.h < 1 || sh.w < 1 || sh.o < 1 || sh.kh < 1 || sh.kw < 1 || sh.stride < 1 ||
      sh.pad < 0)
    return FQT_EINVAL;
  if (sh.ho != (sh.h + 2 * sh.pad - sh.kh) / sh.stride + 1 || sh.wo != (sh.w + 2 * sh.pad - sh.kw) / sh.stride + 1 ||
      sh.ho < 1 || sh.wo < 1)
    return FQT_EINVAL;
  // 16-channel gathers of the gradient codes; row / tap counts within grid limits
  if (sh.o % 16 != 0 || (int64_t)sh.kh * sh.kw * sh.c > 65535 || sh.n > MAX_ROWS) return FQT_EUNSUPPORTED;
  const int64_t P = (int64_t)sh.n * sh.ho * sh.wo;
  if (P > 0x7FFFFFFF / 2 || (int64_t)sh.n * sh.h * sh.w > 0x7FFFFFFF / 2) return FQT_EUNSUPPORTED;
  return FQT_OK;
}

ConvGeom conv_geom(const fqt_conv_shape& sh) {
  ConvGeom g{sh.n, sh.c, sh.h, sh.w, sh.o, sh.kh, sh.kw, sh.stride, sh.pad, sh.ho, sh.wo, 0, 0, 0, 0, 0};
  g.npad = ((int64_t)sh.n + 63) / 64 * 64;
  g.psp = (int64_t)sh.ho * sh.wo;
  return g;
}

// The grad_W layout.  Stride 1: the implicit form on the zero-halo grid
// (rows of gwp = w + 2 pad rounded up to 16 bytes) when a slot's grid pitch
// is at most 1.5 times its output pixels (rounded up to 128 for a per-sample
// Q_b1), else the explicit im2col.  Per-sample Q_b1: each slot's pixels start
// a 128-byte K stage.
ConvGeom conv_geom(const fqt_conv_shape& sh, const fqt_bwd_cfg& cfg) {
  ConvGeom g = conv_geom(sh);
  const bool psq1 = cfg.qb_w.kind == FQT_PSQ;
  const int64_t howo = g.psp;
  const int64_t compact = psq1 ? (howo + 127) / 128 * 128 : howo;
  if (sh.stride == 1) {
    const int64_t gwp = ((int64_t)sh.w + 2 * sh.pad + 15) / 16 * 16, ghp = (int64_t)sh.h + 2 * sh.pad;
    const int64_t gsp = (ghp * gwp + 127) / 128 * 128;
    if (2 * gsp <= 3 * compact && gwp <= 4096 && (!psq1 || gsp <= MAX_K_CHUNK)) {
      g.gwp = gwp;
      g.ghp = ghp;
      g.psp = gsp;
      // copies reach r gwp <= (kh - 1) gwp past the last slot's K range
      g.ldx = ((int64_t)sh.n * gsp + (sh.kh - 1) * gwp + 127) / 128 * 128;
      return g;
    }
  }
  g.psp = compact;
  return g;
}

struct ConvWs {
  Header h;
  StatsSeg sx_seg, sw_seg, sg_seg;
  float *rmin, *rmax;
  int8_t *xq_t, *wq_t, *q2, *q1_t, *bw;
  int32_t *swq, *sumB, *xs, *qs, *sumA_tap, *count_tap, *sg, *rs, *ct, *cnt;
  float *sx, *zx, *sw, *zw, *sg1, *zg1, *sg2, *zg2;
  int32_t* perm;
  BhqWs bhq;
  double* tbuf;      // general BHQ plan: T rows (input pixel, slot) of multi-row groups [h w npad, c]
  ConvPsqSums ps;    // per-sample Q_b1
  int32_t* part;
  int64_t ldq, kchunk;
  int splits;
};

ConvWs carve_conv(Carver& c, const float* X, const float* W, const float* G, const ConvGeom& g,
                  const fqt_bwd_cfg& cfg) {
  ConvWs w{};
  const int64_t N = g.n, hw = (int64_t)g.h * g.w, howo = (int64_t)g.ho * g.wo;
  const int64_t taps = (int64_t)g.kh * g.kw;
  const int64_t P = N * howo;
  w.h = take_header(c);
  w.sx_seg = stats_flat_seg(X, N * hw * g.c);
  w.sw_seg = stats_flat_seg(W, (int64_t)g.o * taps * g.c);
  w.sg_seg = stats_rows_seg(G, N, howo * g.o);
  w.sx_seg.part = c.take<float2>(stats_partials(w.sx_seg));
  w.sw_seg.part = c.take<float2>(stats_partials(w.sw_seg));
  w.sg_seg.part = c.take<float2>(stats_partials(w.sg_seg));
  w.rmin = c.take<float>(N);
  w.rmax = c.take<float>(N);
  stats_direct_rows(w.sg_seg, w.rmin, w.rmax);
  const bool psq1 = cfg.qb_w.kind == FQT_PSQ;
  w.ldq = (psq1 || g.gwp > 0) ? N * g.psp : (P + 127) / 128 * 128;
  w.xq_t = c.take<int8_t>((int64_t)g.c * N * hw);
  w.wq_t = c.take<int8_t>((int64_t)g.c * taps * g.o);
  w.q2 = c.take<int8_t>(N * howo * g.o);
  w.q1_t = c.take<int8_t>((int64_t)g.o * w.ldq);
  // explicit im2col [(tap, c)][ldq], or the kw shifted activation grids [s][c][ldx]
  w.bw = c.take<int8_t>(g.gwp > 0 ? (int64_t)g.kw * g.c * g.ldx : taps * g.c * w.ldq);
  w.swq = c.take<int32_t>(taps * g.c);
  w.sumB = c.take<int32_t>(taps * g.c);
  w.xs = c.take<int32_t>((int64_t)g.c * g.h * g.w);
  w.qs = c.take<int32_t>((int64_t)g.o * howo);
  w.sumA_tap = c.take<int32_t>((int64_t)g.o * taps);
  w.count_tap = c.take<int32_t>(taps);
  w.sg = c.take<int32_t>(N * howo);
  w.rs = c.take<int32_t>(N * hw);
  w.ct = c.take<int32_t>(hw * g.c);
  w.cnt = c.take<int32_t>(hw);
  w.sx = c.take<float>(1);
  w.zx = c.take<float>(1);
  w.sw = c.take<float>(1);
  w.zw = c.take<float>(1);
  w.sg1 = c.take<float>(psq1 ? N : 1);
  w.zg1 = c.take<float>(psq1 ? N : 1);
  w.sg2 = c.take<float>(N);
  w.zg2 = c.take<float>(N);
  if (cfg.qb_x.kind == FQT_BHQ) {
    w.perm = c.take<int32_t>(N);
    w.bhq = carve_bhq(c, N, howo * g.o, cfg.qb_x.block_size);
    if (w.bhq.general) w.tbuf = c.take<double>(hw * g.npad * g.c);
  }
  if (psq1) {
    // one K block per slot: exact int32 partials, weighted in float64
    w.ps.dA = c.take<double>(N);
    w.ps.zA = c.take<double>(N);
    w.ps.zsum = c.take<double>(1);
    w.ps.qw = c.take<double>((int64_t)g.o * howo);
    w.ps.xw = c.take<double>((int64_t)g.c * hw);
    w.ps.WA = c.take<double>((int64_t)g.o * taps);
    w.ps.WB = c.take<double>(taps * g.c);
    w.kchunk = g.psp;
    w.splits = (int)N;
    w.part = c.take<int32_t>(N * g.o * taps * g.c);
    return w;
  }
  // grad_W: split the pixel contraction so that at most 512 blocks run (two
  // full rounds of one block per CU), in a multiple of the XCD count of
  // splits when there are that many, each K chunk a whole number of 128-byte
  // stages and at most 65536
  const int64_t tiles = (g.o <= 64 ? 1 : (g.o + 127) / 128) * ((taps * g.c + 127) / 128);
  int64_t want = 512 / tiles;
  if (want >= NUM_XCD) want = want / NUM_XCD * NUM_XCD;
  const int64_t stages = w.ldq / 128;
  if (want > stages) want = stages;
  if (want < 1) want = 1;
  int64_t kchunk = (stages + want - 1) / want * 128;
  if (kchunk > 65536) kchunk = 65536;
  int64_t splits = (w.ldq + kchunk - 1) / kchunk;
  if (splits >= NUM_XCD && splits % NUM_XCD != 0) {
    // a multiple of the XCD count, so that the contraction keeps each
    // split's tiles on one XCD (trailing splits may be empty: zero partials)
    splits = (splits + NUM_XCD - 1) / NUM_XCD * NUM_XCD;
    kchunk = (stages + splits - 1) / splits * 128;
  }
  w.kchunk = kchunk;
  w.splits = (int)splits;
  w.part = c.take<int32_t>((int64_t)w.splits * g.o * taps * g.c);
  return w;
}

// ---------------------------------------------------------------------------
// Scratch memory of the no-allocation entry point: one array per GPU, held
// until the process ends.  Its device address is taken once per device (with
// that device current) and used wherever host code hands the memory out.
// ---------------------------------------------------------------------------
constexpr size_t NOALLOC_SCRATCH_BYTES = (size_t)4 << 20;
constexpr int NOALLOC_MAX_DEVICES = 64;
static __device__ __align__(256) uint8_t scratch[NOALLOC_SCRATCH_BYTES];
std::mutex scratch_mu;
void* scratch_ptr[NOALLOC_MAX_DEVICES];

fqt_status scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= NOALLOC_MAX_DEVICES) return FQT_EDEVICE;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FQT_EDEVICE;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return FQT_OK;
}

__global__ void copy_status_kernel(const uint32_t* src, uint32_t* dst) {
  if (threadIdx.x < STATUS_WORDS) dst[threadIdx.x] = src[threadIdx.x];
}

}  // namespace
}  // namespace fqt

using namespace fqt;

extern "C" {

fqt_status fqt_quantize_ptq(const float* x, int64_t rows, int64_t cols, int bits, int stochastic, uint64_t seed,
                            uint32_t stream, int transpose, const fqt_qtensor* out, void* ws, size_t ws_bytes,
                            fqt_stream_t s) {
  return quantize_common(FQT_PTQ, x, rows, cols, bits, stochastic ? 1 : 0, seed, stream, transpose ? 1 : 0, 0, out,
                         ws, ws_bytes, s);
}

fqt_status fqt_quantize_shift(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed, uint32_t stream,
                              int transpose, const fqt_qtensor* out, void* ws, size_t ws_bytes, fqt_stream_t s) {
  return quantize_common(FQT_SHIFT, x, rows, cols, bits, 1, seed, stream, transpose, 1, out, ws, ws_bytes, s);
}

fqt_status fqt_quantize_psq(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed, uint32_t stream,
                            const fqt_qtensor* out, void* ws, size_t ws_bytes, fqt_stream_t s) {
  return quantize_common(FQT_PSQ, x, rows, cols, bits, 1, seed, stream, 0, 0, out, ws, ws_bytes, s);
}

fqt_status fqt_quantize_bhq(const float* x, int64_t rows, int64_t cols, int bits, int block_size, uint64_t seed,
                            uint32_t stream, const fqt_qtensor* out, void* ws, size_t ws_bytes, fqt_stream_t s) {
  return quantize_common(FQT_BHQ, x, rows, cols, bits, 1, seed, stream, 0, block_size, out, ws, ws_bytes, s);
}

fqt_status fqt_quantize_psq_noalloc(const float* x, int64_t rows, int64_t cols, int bits, uint64_t seed,
                                    uint32_t stream, const fqt_qtensor* out, uint32_t* status, fqt_stream_t s) {
  fqt_status st = check_quant_args(x, rows, cols, bits, out);
  if (st != FQT_OK) return st;
  Carver cs(nullptr);
  carve_quant(cs, FQT_PSQ, x, rows, cols, 0);
  if (cs.off > NOALLOC_SCRATCH_BYTES) return FQT_EUNSUPPORTED;
  void* ws = nullptr;
  st = scratch_of_current_device(&ws);
  if (st != FQT_OK) return st;
  st = quantize_common(FQT_PSQ, x, rows, cols, bits, 1, seed, stream, 0, 0, out, ws, NOALLOC_SCRATCH_BYTES, s);
  if (st != FQT_OK) return st;
  if (status) {
    hipLaunchKernelGGL(copy_status_kernel, dim3(1), dim3(64), 0, s, static_cast<const uint32_t*>(ws), status);
    FQT_TRY(hipGetLastError());
  }
  return FQT_OK;
}

fqt_status fqt_quantize_seeds(const float* x, int64_t rows, int64_t cols, fqt_kind kind, int bits, int block_size,
                              uint64_t seed, int32_t nseeds, uint32_t stream, const fqt_qtensor* plan,
                              int32_t* sum_code, int32_t* sum_code2, void* ws, size_t ws_bytes, fqt_stream_t s) {
  if (!sum_code || !sum_code2 || !plan) return FQT_EINVAL;
  if (kind != FQT_PTQ && kind != FQT_PSQ && kind != FQT_BHQ) return FQT_EINVAL;
  if (nseeds < 1 || nseeds > 32768) return FQT_EINVAL;
  if (cols % 4 != 0 || ((uintptr_t)x & 15) || ((uintptr_t)sum_code & 15) || ((uintptr_t)sum_code2 & 15))
    return FQT_EUNSUPPORTED;
  return quantize_common(kind, x, rows, cols, bits, 1, seed, stream, 0, kind == FQT_BHQ ? block_size : 0, plan, ws,
                         ws_bytes, s, nseeds, sum_code, sum_code2);
}

size_t fqt_quantize_workspace(fqt_kind kind, int64_t rows, int64_t cols, int block_size) {
  if (rows < 1 || cols < 1) return 0;
  Carver c(nullptr);
  carve_quant(c, kind, nullptr, rows, cols, block_size);
  return c.off;
}

size_t fqt_bhq_adaptive_workspace(int64_t rows, int64_t cols) {
  if (rows < 1 || cols < 1) return 0;
  Carver c(nullptr);
  carve_quant(c, FQT_BHQ, nullptr, rows, cols, 0);
  return c.off;
}

fqt_status fqt_bhq_adaptive_groups(const float* x, int64_t rows, int64_t cols, int bits, int32_t* num_groups,
                                   double* objective, void* ws, size_t ws_bytes, fqt_stream_t s) {
  if (!x || !num_groups) return FQT_EINVAL;
  if (rows < 1 || cols < 1 || !valid_bits(bits)) return FQT_EINVAL;
  if (rows > APPD_MAX_ROWS || cols > ((int64_t)1 << 40) / rows) return FQT_EUNSUPPORTED;
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_bhq_adaptive_workspace(rows, cols)) return FQT_EWORKSPACE;
  Carver c(ws);
  QuantWs w = carve_quant(c, FQT_BHQ, x, rows, cols, 0);
  StatsPlan sp{};
  sp.seg[0] = w.seg;
  sp.nseg = 1;
  FQT_TRY(launch_stats(sp, s));
  FinalizePlan fp{};
  fp.seg[0] = w.seg;
  fp.nseg = 1;
  fp.row_seg = 0;
  fp.rmin = w.rmin;
  fp.rmax = w.rmax;
  fp.status = w.h.status;
  add_zero(fp, bhq_plan_carve(w.bhq.plan, rows).rank, rows);
  FQT_TRY(launch_finalize(fp, s));
  FQT_TRY(launch_bhq_sort(w.rmin, w.rmax, rows, w.bhq.plan, w.bhq.appd.sigma, nullptr, s));
  FQT_TRY(launch_appd_search(w.rmin, w.rmax, rows, bits, w.bhq.appd, objective, num_groups, s));
  return FQT_OK;
}

size_t fqt_linear_backward_workspace(int64_t N, int64_t d_in, int64_t d_out, const fqt_bwd_cfg* cfg) {
  if (!cfg || N < 1 || d_in < 1 || d_out < 1 || cfg->qb_w.kind == FQT_PSQ) return 0;
  Carver c(nullptr);
  carve_linear(c, nullptr, nullptr, nullptr, N, d_in, d_out, *cfg);
  return c.off;
}

fqt_status fqt_linear_backward(const float* X, const float* W, const float* G, int64_t N, int64_t d_in,
                               int64_t d_out, const fqt_bwd_cfg* cfg, float* grad_W, float* grad_X, void* ws,
                               size_t ws_bytes, fqt_stream_t s) {
  if (!X || !W || !G || !grad_W || !grad_X) return FQT_EINVAL;
  if (N < 1 || d_in < 1 || d_out < 1) return FQT_EINVAL;
  fqt_status st = check_cfg(cfg);
  if (st != FQT_OK) return st;
  // a per-sample Q_b1 takes the shift form (Sec. 4.3) on a linear layer
  if (cfg->qb_w.kind == FQT_PSQ) return FQT_EUNSUPPORTED;
  if (N > MAX_ROWS || d_out > MAX_ROWS || d_out > MAX_K_CHUNK || N > 0x7FFFFFFF / 2) return FQT_EUNSUPPORTED;
  if (cfg->qb_x.kind == FQT_BHQ) {
    st = check_block(cfg->qb_x.block_size, N);
    if (st != FQT_OK) return st;
  }
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_linear_backward_workspace(N, d_in, d_out, cfg)) return FQT_EWORKSPACE;
  Carver c(ws);
  LinearWs w = carve_linear(c, X, W, G, N, d_in, d_out, *cfg);
  // caller buffers for the gradient codes (and the BHQ permutation)
  if (cfg->qb2_codes) w.qg2 = cfg->qb2_codes;
  if (cfg->qb1_codes) w.qg1_t = cfg->qb1_codes;
  if (cfg->perm && w.perm) w.perm = cfg->perm;
  const fqt_qspec qx = cfg->qb_x;
  const bool bhq = qx.kind == FQT_BHQ;
  const Tracer tr{cfg->trace, s};

  // statistics of X, W (per tensor) and G (per row), one launch
  tr.begin(0);
  tr.end(0);
  tr.begin(1);
  StatsPlan sp{};
  sp.seg[0] = w.sx_seg;
  sp.seg[1] = w.sw_seg;
  sp.seg[2] = w.sg_seg;
  sp.nseg = 3;
  FQT_TRY(launch_stats(sp, s));
  tr.end(1);
  // scales: Q_f, Q_theta, Q_b1 per tensor; Q_b2 per tensor / per row / BHQ plan
  tr.begin(2);
  FinalizePlan fp{};
  fp.seg[0] = w.sx_seg;
  fp.seg[1] = w.sw_seg;
  fp.seg[2] = w.sg_seg;
  fp.nseg = 3;
  fp.row_seg = 2;
  fp.rmin = w.rmin;
  fp.rmax = w.rmax;
  fp.status = w.h.status;
  fp.out[0] = ScaleOut{0, cfg->f_bits, 0, w.sx, w.zx};
  fp.out[1] = ScaleOut{1, cfg->theta_bits, 0, w.sw, w.zw};
  const bool shift1 = cfg->qb_w.kind == FQT_SHIFT;
  fp.out[2] = ScaleOut{2, cfg->qb_w.bits, shift1 ? 2 : 0, w.sg1, w.zg1, w.shift1, w.tscale1, w.zeta1};
  fp.nout = 3;
  if (qx.kind != FQT_BHQ) fp.out[fp.nout++] = ScaleOut{2, qx.bits, qx.kind == FQT_PSQ ? 1 : 0, w.sg2, w.zg2};
  add_zero(fp, w.sum_x, d_in);
  add_zero(fp, w.sum_w, d_in);
  add_zero(fp, w.sum_g1, d_out);
  add_zero(fp, w.sum_g2, N);
  if (bhq) add_zero(fp, bhq_plan_carve(w.bhq.plan, N).rank, N);
  const bool fin_in_plan = bhq && w.sg_seg.rmin != nullptr;
  if (!fin_in_plan) FQT_TRY(launch_finalize(fp, s));
  int mode = qx.kind == FQT_PSQ ? QM_ROW : QM_TENSOR;
  if (bhq) {
    st = plan_bhq(w.bhq, w.rmin, w.rmax, N, qx.bits, qx.block_size, w.perm, w.sg2, w.zg2, nullptr, nullptr,
                  fin_in_plan ? &fp : nullptr, s);
    if (st != FQT_OK) return st;
    mode = QM_BHQ;
  }
  tr.end(2);

  // Q_f(X): deterministic PTQ, codes [d_in, N] in slot order (rows through perm)
  QuantParams px{};
  px.x = X;
  px.rows = N;
  px.cols = d_in;
  px.perm = w.perm;
  px.bits = cfg->f_bits;
  px.scale = w.sx;
  px.zero = w.zx;
  px.q_t = w.qx_t;
  px.sum_t = w.sum_x;
  // Q_theta(W): deterministic PTQ, codes [d_in, d_out]
  QuantParams pw{};
  pw.x = W;
  pw.rows = d_out;
  pw.cols = d_in;
  pw.bits = cfg->theta_bits;
  pw.scale = w.sw;
  pw.zero = w.zw;
  pw.q_t = w.qw_t;
  pw.sum_t = w.sum_w;
  QuantParams pg{};
  pg.x = G;
  pg.rows = N;
  pg.cols = d_out;
  pg.perm = w.perm;
  pg.bits = qx.bits;
  pg.stoch = 1;
  pg.seed = cfg->seed;
  pg.stream = 1;
  pg.scale = w.sg2;
  pg.zero = w.zg2;
  pg.q_nat = w.qg2;
  pg.sum_nat = w.sum_g2;
  // codes of at most 4 bits are stored two per byte and unpacked by the
  // grad_X contraction's loader
  const bool packed = cfg->packed_codes == 1 && qx.bits <= 4 && d_out % 16 == 0;
  pg.packed = packed ? 1 : 0;
  pg.bits2 = cfg->qb_w.bits;
  pg.stream2 = 0;
  pg.scale2 = w.sg1;
  pg.zero2 = w.zg1;
  pg.shift2 = w.shift1;
  pg.q2_t = w.qg1_t;
  pg.sum2_t = w.sum_g1;
  if (bhq) {
    st = bhq_params(w.bhq, G, N, d_out, qx.block_size, w.perm, w.sg2, pg, s);
    if (st != FQT_OK) return st;
  }
  // Q_b2(G) [N, d_out] slot order (stream 1) and Q_b1(G) [d_out, N] (stream 0)
  // from one read of G, with Q_f(X) and Q_theta(W) in the same launch (phase
  // 5; phases 3 and 4 stay empty)
  tr.begin(3);
  tr.end(3);
  tr.begin(4);
  tr.end(4);
  tr.begin(5);
  FQT_TRY(launch_quant_fused(pg, mode, px, pw, s));
  if (shift1) {
    // Q_b1's per-sample zero points meet X along the contraction: their
    // terms form one float64 vector over d_in
    ColvecParams cv{};
    cv.q_t = w.qx_t;
    cv.rows = N;
    cv.cols = d_in;
    cv.perm = w.perm;
    cv.zeta = w.zeta1;
    cv.scaleX = w.sx;
    cv.zeroX = w.zx;
    cv.halfX = 1 << (cfg->f_bits - 1);
    cv.part = w.colvec_part;
    cv.out = w.colvec;
    FQT_TRY(launch_colvec(cv, s));
  }
  tr.end(5);

  // grad_W [d_out, d_in] = Q_b1(G)^T Q_f(X): contraction over the N samples
  GemmParams gw{};
  gw.A = w.qg1_t;
  gw.B = w.qx_t;
  gw.M = d_out;
  gw.N = d_in;
  gw.K = N;
  gw.lda = N;
  gw.ldb = N;
  gw.splits = w.splits;
  gw.kchunk = w.splits > 1 ? MAX_K_CHUNK : N;
  gw.part = w.part;
  gw.out = grad_W;
  gw.ldo = d_in;
  gw.sumA = w.sum_g1;
  gw.sumB = w.sum_x;
  gw.scaleA = w.sg1;
  gw.zeroA = w.zg1;
  gw.halfA = 1 << (cfg->qb_w.bits - 1);
  if (shift1) {
    // shifted codes count in the common step 1 / (s 2^E), E = min(4, 8 - bits)
    gw.scaleA = w.tscale1;
    gw.expA = cfg->qb_w.bits <= 4 ? 4 : 8 - cfg->qb_w.bits;
    gw.colvec = w.colvec;
  }
  gw.scaleB = w.sx;
  gw.zeroB = w.zx;
  gw.halfB = 1 << (cfg->f_bits - 1);
  tr.begin(6);
  if (w.splits > 1) {
    FQT_TRY(launch_gemm(gw, EPI_RAW_I32, s));
    FQT_TRY(launch_splitk_reduce(gw, nullptr, EPI_TENSOR, s));
  } else {
    FQT_TRY(launch_gemm(gw, EPI_TENSOR, s));
  }
  tr.end(6);
  // grad_X [N, d_in] = Q_b2(G) Q_theta(W): contraction over d_out
  GemmParams gx{};
  gx.A = w.qg2;
  gx.B = w.qw_t;
  gx.M = N;
  gx.N = d_in;
  gx.K = d_out;
  gx.lda = packed ? d_out / 2 : d_out;
  gx.packedA = packed ? 1 : 0;
  gx.ldb = d_out;
  gx.splits = 1;
  gx.kchunk = d_out;
  gx.out = grad_X;
  gx.ldo = d_in;
  gx.perm = w.perm;
  gx.sumA = w.sum_g2;
  gx.sumB = w.sum_w;
  gx.scaleA = w.sg2;
  gx.zeroA = w.zg2;
  gx.rowwiseA = qx.kind != FQT_PTQ;
  gx.halfA = 1 << (qx.bits - 1);
  gx.scaleB = w.sw;
  gx.zeroB = w.zw;
  gx.halfB = 1 << (cfg->theta_bits - 1);
  gx.L = pg.L;
  gx.mask = cfg->relu_input ? X : nullptr;  // [N, d_in], the same layout as grad_X
  tr.begin(7);
  if (bhq && w.bhq.general) {
    // general plan: one-row groups finished in the epilogue, the other rows'
    // T through the inverse pass
    gx.slot = w.bhq.slot;
    gx.tbuf = w.tbuf;
    gx.ldt = d_in;
    FQT_TRY(launch_gemm(gx, EPI_BHQT, s));
    InverseParams ip{};
    ip.T = w.tbuf;
    ip.ldt = d_in;
    ip.tstride = 0;
    ip.nblk = 1;
    ip.rows = N;
    ip.cols = d_in;
    ip.slot = w.bhq.slot;
    ip.perm = w.perm;
    ip.scale = w.sg2;
    ip.out = grad_X;
    ip.ldo = d_in;
    ip.ostride = 1;
    ip.obstride = 0;
    ip.mask = gx.mask;
    FQT_TRY(launch_bhq_inverse(ip, s));
  } else {
    FQT_TRY(launch_gemm(gx, bhq ? EPI_BHQ : EPI_ROW, s));
  }
  tr.end(7);
  return FQT_OK;
}

size_t fqt_linear_forward_workspace(int64_t N, int64_t d_in, int64_t d_out) {
  if (N < 1 || d_in < 1 || d_out < 1) return 0;
  Carver c(nullptr);
  carve_forward(c, nullptr, nullptr, N, d_in, d_out);
  return c.off;
}

fqt_status fqt_linear_forward(const float* X, const float* W, int64_t N, int64_t d_in, int64_t d_out, int f_bits,
                              int theta_bits, int relu, float* Y, void* ws, size_t ws_bytes, fqt_stream_t s) {
  if (!X || !W || !Y) return FQT_EINVAL;
  if (N < 1 || d_in < 1 || d_out < 1 || !valid_bits(f_bits) || !valid_bits(theta_bits)) return FQT_EINVAL;
  if (relu != 0 && relu != 1) return FQT_EINVAL;
  if (N > MAX_ROWS || d_out > MAX_ROWS || N > 65535LL * 128 || (d_in + MAX_K_CHUNK - 1) / MAX_K_CHUNK > 65535)
    return FQT_EUNSUPPORTED;
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_linear_forward_workspace(N, d_in, d_out)) return FQT_EWORKSPACE;
  Carver c(ws);
  ForwardWs w = carve_forward(c, X, W, N, d_in, d_out);

  // ranges of X and W (per tensor), one launch; then scales and zeroed code sums
  StatsPlan sp{};
  sp.seg[0] = w.sx_seg;
  sp.seg[1] = w.sw_seg;
  sp.nseg = 2;
  FQT_TRY(launch_stats(sp, s));
  FinalizePlan fp{};
  fp.seg[0] = w.sx_seg;
  fp.seg[1] = w.sw_seg;
  fp.nseg = 2;
  fp.row_seg = -1;
  fp.status = w.h.status;
  fp.out[0] = ScaleOut{0, f_bits, 0, w.sx, w.zx};
  fp.out[1] = ScaleOut{1, theta_bits, 0, w.sw, w.zw};
  fp.nout = 2;
  add_zero(fp, w.sum_x, N);
  add_zero(fp, w.sum_w, d_out);
  FQT_TRY(launch_finalize(fp, s));
  // Q_f(X) [N, d_in] and Q_theta(W) [d_out, d_in]: natural layout (K = d_in
  // contiguous), with per-row code sums for the zero-point terms
  QuantParams px{};
  px.x = X;
  px.rows = N;
  px.cols = d_in;
  px.bits = f_bits;
  px.scale = w.sx;
  px.zero = w.zx;
  px.q_nat = w.qx;
  px.sum_nat = w.sum_x;
  FQT_TRY(launch_quant(px, QM_TENSOR, s));
  QuantParams pw{};
  pw.x = W;
  pw.rows = d_out;
  pw.cols = d_in;
  pw.bits = theta_bits;
  pw.scale = w.sw;
  pw.zero = w.zw;
  pw.q_nat = w.qw;
  pw.sum_nat = w.sum_w;
  FQT_TRY(launch_quant(pw, QM_TENSOR, s));
  // Y = Q_f(X) Q_theta(W)^T: contraction over d_in, per-tensor epilogue
  GemmParams g{};
  g.A = w.qx;
  g.B = w.qw;
  g.M = N;
  g.N = d_out;
  g.K = d_in;
  g.lda = d_in;
  g.ldb = d_in;
  g.splits = w.splits;
  g.kchunk = w.splits > 1 ? MAX_K_CHUNK : d_in;
  g.part = w.part;
  g.out = Y;
  g.ldo = d_out;
  g.sumA = w.sum_x;
  g.sumB = w.sum_w;
  g.scaleA = w.sx;
  g.zeroA = w.zx;
  g.halfA = 1 << (f_bits - 1);
  g.scaleB = w.sw;
  g.zeroB = w.zw;
  g.halfB = 1 << (theta_bits - 1);
  g.relu = relu;
  if (w.splits > 1) {
    FQT_TRY(launch_gemm(g, EPI_RAW_I32, s));
    FQT_TRY(launch_splitk_reduce(g, nullptr, EPI_TENSOR, s));
  } else {
    FQT_TRY(launch_gemm(g, EPI_TENSOR, s));
  }
  return FQT_OK;
}

size_t fqt_gemm_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || N < 1 || K < 1) return 0;
  const int64_t splits = (K + MAX_K_CHUNK - 1) / MAX_K_CHUNK;
  return (size_t)(splits * M * N * 4) + 256;
}

fqt_status fqt_gemm_s8s8_s64(const int8_t* A, const int8_t* B, int64_t M, int64_t N, int64_t K, int64_t lda,
                             int64_t ldb, int64_t* C, void* ws, size_t ws_bytes, fqt_stream_t s) {
  if (!A || !B || !C) return FQT_EINVAL;
  if (M < 1 || N < 1 || K < 1 || lda < K || ldb < K) return FQT_EINVAL;
  if (M > 65535LL * 128 || (K + MAX_K_CHUNK - 1) / MAX_K_CHUNK > 65535) return FQT_EUNSUPPORTED;
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_gemm_workspace(M, N, K)) return FQT_EWORKSPACE;
  GemmParams g{};
  g.A = A;
  g.B = B;
  g.M = M;
  g.N = N;
  g.K = K;
  g.lda = lda;
  g.ldb = ldb;
  g.splits = (int)((K + MAX_K_CHUNK - 1) / MAX_K_CHUNK);
  g.kchunk = g.splits > 1 ? MAX_K_CHUNK : K;
  g.part = static_cast<int32_t*>(ws);
  FQT_TRY(launch_gemm(g, EPI_RAW_I32, s));
  FQT_TRY(launch_splitk_reduce(g, C, EPI_RAW_I32, s));
  return FQT_OK;
}

// 4-bit codes on the 6-bit float matrix cores: packed operands, exact chunks
constexpr int64_t BF6_K_CHUNK = 131072;  // 64 * K < 2^24 keeps float32 sums exact

struct Bf6Ws {
  Header h;
  int8_t *a6, *b6;
  int32_t* part;
  int64_t Kpad, splits;
};

Bf6Ws carve_bf6(Carver& c, int64_t M, int64_t N, int64_t K) {
  Bf6Ws w{};
  w.h = take_header(c);
  const int64_t rb = bf6_row_bytes(K);
  w.Kpad = rb / 96 * 128;
  w.splits = (w.Kpad + BF6_K_CHUNK - 1) / BF6_K_CHUNK;
  w.a6 = c.take<int8_t>(M * rb);
  w.b6 = c.take<int8_t>(N * rb);
  w.part = c.take<int32_t>(w.splits * M * N);
  return w;
}

size_t fqt_gemm_s4s4_bf6_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || N < 1 || K < 1) return 0;
  Carver c(nullptr);
  carve_bf6(c, M, N, K);
  return c.off;
}

fqt_status fqt_gemm_s4s4_bf6(const int8_t* A, const int8_t* B, int64_t M, int64_t N, int64_t K, int64_t lda,
                             int64_t ldb, int64_t* C, void* ws, size_t ws_bytes, fqt_stream_t s) {
  if (!A || !B || !C) return FQT_EINVAL;
  if (M < 1 || N < 1 || K < 1 || lda < K || ldb < K) return FQT_EINVAL;
  if (M > 65535LL * 128 || (K + BF6_K_CHUNK - 1) / BF6_K_CHUNK > 65535) return FQT_EUNSUPPORTED;
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_gemm_s4s4_bf6_workspace(M, N, K)) return FQT_EWORKSPACE;
  Carver c(ws);
  Bf6Ws w = carve_bf6(c, M, N, K);
  FQT_TRY(launch_status_clear(w.h.status, s));
  FQT_TRY(launch_pack_e3m2(A, M, K, lda, w.a6, w.h.status, s));
  FQT_TRY(launch_pack_e3m2(B, N, K, ldb, w.b6, w.h.status, s));
  Bf6Params p{};
  p.A = w.a6;
  p.B = w.b6;
  p.M = M;
  p.N = N;
  p.Kpad = w.Kpad;
  p.lda = bf6_row_bytes(K);
  p.ldb = p.lda;
  p.kchunk = w.splits > 1 ? BF6_K_CHUNK : w.Kpad;
  p.splits = (int)w.splits;
  p.part = w.part;
  FQT_TRY(launch_gemm_bf6(p, s));
  GemmParams g{};
  g.M = M;
  g.N = N;
  g.splits = (int)w.splits;
  g.part = w.part;
  FQT_TRY(launch_splitk_reduce(g, C, EPI_RAW_I32, s));
  return FQT_OK;
}

fqt_status fqt_conv_backward_im2col(const float* X, const float* W, const float* G, const fqt_conv_shape* shape,
                                    const fqt_bwd_cfg* cfg, float* grad_W, float* grad_X, void* ws,
                                    size_t ws_bytes, fqt_stream_t s) {
  if (!X || !W || !G || !grad_W || !shape) return FQT_EINVAL;
  const bool want_x = grad_X != nullptr;  // NULL: no input gradient
  fqt_status st = check_conv_shape(*shape);
  if (st != FQT_OK) return st;
  st = check_cfg(cfg);
  if (st != FQT_OK) return st;
  if (cfg->relu_input || cfg->qb_w.kind == FQT_SHIFT) return FQT_EUNSUPPORTED;
  // per-sample Q_b1: one int32-exact K block per sample, one split per sample
  if (cfg->qb_w.kind == FQT_PSQ && ((int64_t)shape->ho * shape->wo > MAX_K_CHUNK || shape->n > 65535))
    return FQT_EUNSUPPORTED;
  if (cfg->qb_x.kind == FQT_BHQ) {
    st = check_block(cfg->qb_x.block_size, shape->n);
    if (st != FQT_OK) return st;
  }
  if (!ws) return FQT_EWORKSPACE;
  if (ws_bytes < fqt_conv_backward_workspace(shape, cfg)) return FQT_EWORKSPACE;
  const ConvGeom g = conv_geom(*shape, *cfg);
  const bool psq1 = cfg->qb_w.kind == FQT_PSQ;
  Carver c(ws);
  ConvWs w = carve_conv(c, X, W, G, g, *cfg);
  const fqt_qspec qx = cfg->qb_x;
  // without an input gradient there is no Q_b2, so no BHQ plan: samples stay in order
  const bool bhq = qx.kind == FQT_BHQ && want_x;
  int32_t* const perm = bhq ? w.perm : nullptr;
  const Tracer tr{cfg->trace, s};
  const int64_t N = g.n, D = (int64_t)g.ho * g.wo * g.o;
  const int64_t hw = (int64_t)g.h * g.w, howo = (int64_t)g.ho * g.wo;
  const int64_t taps = (int64_t)g.kh * g.kw;

  tr.begin(0);
  tr.end(0);
  tr.begin(1);
  StatsPlan sp{};
  sp.seg[0] = w.sx_seg;
  sp.seg[1] = w.sw_seg;
  sp.seg[2] = w.sg_seg;
  sp.nseg = 3;
  FQT_TRY(launch_stats(sp, s));
  tr.end(1);
  tr.begin(2);
  FinalizePlan fp{};
  fp.seg[0] = w.sx_seg;
  fp.seg[1] = w.sw_seg;
  fp.seg[2] = w.sg_seg;
  fp.nseg = 3;
  fp.row_seg = 2;
  fp.rmin = w.rmin;
  fp.rmax = w.rmax;
  fp.status = w.h.status;
  fp.out[0] = ScaleOut{0, cfg->f_bits, 0, w.sx, w.zx};
  fp.out[1] = ScaleOut{1, cfg->theta_bits, 0, w.sw, w.zw};
  fp.out[2] = ScaleOut{2, cfg->qb_w.bits, psq1 ? 1 : 0, w.sg1, w.zg1};
  fp.nout = 3;
  if (!bhq && want_x) fp.out[fp.nout++] = ScaleOut{2, qx.bits, qx.kind == FQT_PSQ ? 1 : 0, w.sg2, w.zg2};
  if (!psq1) add_zero(fp, w.sumB, taps * g.c);
  if (bhq) add_zero(fp, bhq_plan_carve(w.bhq.plan, N).rank, N);
  const bool fin_in_plan = bhq && w.sg_seg.rmin != nullptr;
  if (!fin_in_plan) FQT_TRY(launch_finalize(fp, s));
  int mode = qx.kind == FQT_PSQ ? QM_ROW : QM_TENSOR;
  if (bhq) {
    st = plan_bhq(w.bhq, w.rmin, w.rmax, N, qx.bits, qx.block_size, w.perm, w.sg2, w.zg2, nullptr, nullptr,
                  fin_in_plan ? &fp : nullptr, s);
    if (st != FQT_OK) return st;
    mode = QM_BHQ;
  }
  tr.end(2);

  // Q_f(X): codes [c][pixels], samples in slot order
  tr.begin(3);
  NarrowQParams nx{};
  nx.x = X;
  nx.rows = N * hw;
  nx.cols = g.c;
  nx.perm = perm;
  nx.blk = hw;
  nx.bits = cfg->f_bits;
  nx.scale = w.sx;
  nx.zero = w.zx;
  nx.q_t = w.xq_t;
  nx.ldt = N * hw;
  FQT_TRY(launch_quant_narrow_t(nx, s));
  tr.end(3);
  // Q_theta(W): codes [c][(r, s, o)] and their sums over o
  tr.begin(4);
  if (want_x) FQT_TRY(launch_conv_wq(W, g, cfg->theta_bits, w.sw, w.zw, w.wq_t, w.swq, s));
  tr.end(4);
  // Q_b2(G) [slot][(y, x, o)] (stream 1); Q_b1(G) [o][pixels] (stream 0)
  tr.begin(5);
  QuantParams pg{};
  pg.x = G;
  pg.rows = N;
  pg.cols = D;
  pg.perm = w.perm;
  pg.bits = qx.bits;
  pg.stoch = 1;
  pg.seed = cfg->seed;
  pg.stream = 1;
  pg.scale = w.sg2;
  pg.zero = w.zg2;
  pg.q_nat = w.q2;
  pg.pm_o = g.o;  // [output pixel][slot][o]: a grad_X tile's slots of one tap read one contiguous run
  if (bhq) {
    st = bhq_params(w.bhq, G, N, D, qx.block_size, w.perm, w.sg2, pg, s);
    if (st != FQT_OK) return st;
  }
  if (want_x) FQT_TRY(launch_quant(pg, mode, s));
  NarrowQParams n1{};
  n1.x = G;
  n1.rows = N * g.psp;
  n1.cols = g.o;
  n1.perm = perm;
  n1.blk = g.psp;
  n1.vblk = howo;
  n1.rowscale = psq1 ? 1 : 0;
  if (g.gwp > 0) {  // output pixel (y, x) at y gwp + x of its slot's grid
    n1.gw = g.gwp;
    n1.gwo = g.wo;
    n1.gho = g.ho;
  }
  n1.bits = cfg->qb_w.bits;
  n1.stoch = 1;
  n1.seed = cfg->seed;
  n1.stream = 0;
  n1.scale = w.sg1;
  n1.zero = w.zg1;
  n1.q_t = w.q1_t;
  n1.ldt = w.ldq;
  FQT_TRY(launch_quant_narrow_t(n1, s));
  tr.end(5);

  // grad_W [o][(r, s, c)] = Q_b1(G)^T im2col(Q_f(X)), split over output pixels
  tr.begin(6);
  FQT_TRY(launch_conv_im2col_w(g, w.xq_t, w.bw, g.gwp > 0 ? g.ldx : w.ldq, psq1 ? nullptr : w.xs, w.sumB, s));
  if (psq1)
    FQT_TRY(launch_conv_psq_sums(g, w.sg1, w.zg1, perm, 1 << (cfg->qb_w.bits - 1), w.q1_t, w.ldq, w.xq_t, w.ps,
                                 w.count_tap, s));
  else
    FQT_TRY(launch_conv_tapsums(g, w.q1_t, w.ldq, w.qs, w.sumA_tap, w.count_tap, s));
  GemmParams gw{};
  gw.A = w.q1_t;
  gw.B = w.bw;
  gw.M = g.o;
  gw.N = taps * g.c;
  gw.K = w.ldq;
  gw.lda = w.ldq;
  gw.ldb = w.ldq;
  if (g.gwp > 0) {  // tap (r, s), channel c: copy s at K offset r gwp
    gw.ldb = g.ldx;
    gw.bmap_c = g.c;
    gw.bmap_kw = g.kw;
    gw.bmap_wp = g.gwp;
  }
  gw.splits = w.splits;
  gw.kchunk = w.kchunk;
  gw.part = w.part;
  gw.out = grad_W;
  gw.ldo = taps * g.c;
  gw.sumB = w.sumB;
  gw.scaleA = w.sg1;
  gw.zeroA = w.zg1;
  gw.halfA = 1 << (cfg->qb_w.bits - 1);
  gw.scaleB = w.sx;
  gw.zeroB = w.zx;
  gw.halfB = 1 << (cfg->f_bits - 1);
  FQT_TRY(launch_gemm(gw, EPI_RAW_I32, s));
  if (psq1)
    FQT_TRY(launch_conv_gradw_psq_reduce(gw, g, w.ps, w.count_tap, s));
  else
    FQT_TRY(launch_conv_gradw_reduce(gw, g, w.sumA_tap, w.count_tap, s));
  tr.end(6);

  // grad_X [n][h][w][c] = col2im(Q_b2(G) Q_theta(W)), implicit im2col rows
  if (!want_x) {
    tr.begin(7);
    tr.end(7);
    return FQT_OK;
  }
  tr.begin(7);
  FQT_TRY(launch_conv_gradx_prep(g, w.q2, w.swq, w.sg, w.rs, w.ct, w.cnt, s));
  GemmParams gx{};
  gx.B = w.wq_t;
  gx.M = hw * g.npad;
  gx.N = g.c;
  gx.K = taps * g.o;
  gx.ldb = taps * g.o;
  gx.splits = 1;
  gx.kchunk = gx.K;
  gx.out = grad_X;
  gx.ldo = g.c;
  gx.perm = w.perm;
  gx.scaleA = w.sg2;
  gx.zeroA = w.zg2;
  gx.rowwiseA = qx.kind != FQT_PTQ;
  gx.halfA = 1 << (qx.bits - 1);
  gx.scaleB = w.sw;
  gx.zeroB = w.zw;
  gx.halfB = 1 << (cfg->theta_bits - 1);
  gx.L = pg.L;
  if (bhq && w.bhq.general) {
    gx.slot = w.bhq.slot;
    gx.tbuf = w.tbuf;
    gx.ldt = g.c;
    FQT_TRY(launch_conv_gradx(gx, EPI_BHQT, g, w.q2, w.rs, w.ct, w.cnt, s));
    InverseParams ip{};
    ip.T = w.tbuf;
    ip.ldt = g.c;
    ip.tstride = g.npad;
    ip.nblk = hw;
    ip.rows = N;
    ip.cols = g.c;
    ip.slot = w.bhq.slot;
    ip.perm = w.perm;
    ip.scale = w.sg2;
    ip.out = grad_X;
    ip.ldo = g.c;
    ip.ostride = hw;
    ip.obstride = 1;
    FQT_TRY(launch_bhq_inverse(ip, s));
  } else {
    FQT_TRY(launch_conv_gradx(gx, bhq ? EPI_BHQ : EPI_ROW, g, w.q2, w.rs, w.ct, w.cnt, s));
  }
  tr.end(7);
  return FQT_OK;
}

size_t fqt_conv_backward_workspace(const fqt_conv_shape* shape, const fqt_bwd_cfg* cfg) {
  if (!shape || !cfg || check_conv_shape(*shape) != FQT_OK) return 0;
  Carver c(nullptr);
  carve_conv(c, nullptr, nullptr, nullptr, conv_geom(*shape, *cfg), *cfg);
  return c.off;
}

constexpr int64_t PROBE_BLOCKS = 2048;  // 8 blocks of 4 waves per CU

fqt_status fqt_probe_mfma_i8(int64_t iters, int32_t* sink, double* ops, fqt_stream_t s) {
  if (iters < 1 || !sink || !ops) return FQT_EINVAL;
  *ops = (double)PROBE_BLOCKS * 4.0 * 4.0 * (double)iters * (2.0 * 32 * 32 * 32);
  return launch_mfma_probe(PROBE_BLOCKS, iters, sink, s) == hipSuccess ? FQT_OK : FQT_EDEVICE;
}

fqt_status fqt_probe_copy(const void* src, void* dst, size_t bytes, fqt_stream_t s) {
  if (!src || !dst || bytes == 0 || bytes % 16 != 0 || ((uintptr_t)src & 15) || ((uintptr_t)dst & 15))
    return FQT_EINVAL;
  return launch_copy_probe(PROBE_BLOCKS * 4, src, dst, (int64_t)(bytes / 16), s) == hipSuccess ? FQT_OK : FQT_EDEVICE;
}

fqt_status fqt_workspace_status(const void* ws, fqt_stream_t s) {
  if (!ws) return FQT_EINVAL;
  if (hipStreamSynchronize(s) != hipSuccess) return FQT_EDEVICE;
  uint32_t words[STATUS_WORDS] = {};
  if (hipMemcpy(words, ws, sizeof(words), hipMemcpyDeviceToHost) != hipSuccess) return FQT_EDEVICE;
  uint32_t word = 0;
  for (int i = 0; i < STATUS_WORDS; ++i) word |= words[i];
  return (word & STATUS_NONFINITE) ? FQT_ENONFINITE : FQT_OK;
}

const char* fqt_status_str(fqt_status st) {
  switch (st) {
    case FQT_OK: return "ok";
    case FQT_EINVAL: return "invalid argument";
    case FQT_EUNSUPPORTED: return "unsupported configuration";
    case FQT_ENONFINITE: return "non-finite input or range overflow";
    case FQT_EWORKSPACE: return "workspace missing or too small";
    case FQT_EDEVICE: return "HIP runtime error";
  }
  return "unknown status";
}

const char* fqt_version(void) { return "fqt-mi355x 0.1 (gfx950)"; }

}  // extern "C"
