"""ctypes binding of libfqt.so (C ABI in include/fqt.h).

Argument marshalling only: every step of the FQT backward runs in the HIP
library.  Tensors are torch CUDA (ROCm) tensors; the binding passes their
device pointers and the current HIP stream, allocates outputs and the
workspace with torch, and raises on any non-OK status.  There is no CPU
fallback: if the library is not built or cannot load, every call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfqt.so")

FQT_PTQ, FQT_PSQ, FQT_BHQ, FQT_SHIFT = 0, 1, 2, 3
KINDS = {"ptq": FQT_PTQ, "psq": FQT_PSQ, "bhq": FQT_BHQ, "shift": FQT_SHIFT}
STATUS = {0: "FQT_OK", 1: "FQT_EINVAL", 2: "FQT_EUNSUPPORTED", 3: "FQT_ENONFINITE", 4: "FQT_EWORKSPACE",
          5: "FQT_EDEVICE"}


class FqtError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {STATUS.get(code, code)}")
        self.code = code


class QTensor(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("scale", ctypes.c_void_p), ("zero", ctypes.c_void_p),
                ("perm", ctypes.c_void_p), ("group_off", ctypes.c_void_p), ("code_sum", ctypes.c_void_p),
                ("shift", ctypes.c_void_p), ("num_groups", ctypes.c_void_p)]


class QSpec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("bits", ctypes.c_int), ("block_size", ctypes.c_int)]


TRACE_PHASES = 8
PHASE_NAMES = ["init", "stats", "scales_plan", "quant_X", "quant_W", "quant_G", "gemm_gradW", "gemm_gradX"]


class Trace(ctypes.Structure):
    _fields_ = [("start", ctypes.c_void_p * TRACE_PHASES), ("stop", ctypes.c_void_p * TRACE_PHASES),
                ("count", ctypes.c_int)]


class BwdCfg(ctypes.Structure):
    _fields_ = [("qb_w", QSpec), ("qb_x", QSpec), ("f_bits", ctypes.c_int), ("theta_bits", ctypes.c_int),
                ("seed", ctypes.c_uint64), ("trace", ctypes.POINTER(Trace)), ("relu_input", ctypes.c_int),
                ("qb2_codes", ctypes.c_void_p), ("qb1_codes", ctypes.c_void_p), ("perm", ctypes.c_void_p),
                ("packed_codes", ctypes.c_int)]


class ConvShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("n", "c", "h", "w", "o", "kh", "kw", "stride", "pad", "ho", "wo")]


EXPORTS = [
    "fqt_quantize_ptq", "fqt_quantize_psq", "fqt_quantize_psq_noalloc", "fqt_quantize_bhq", "fqt_quantize_shift", "fqt_quantize_workspace",
    "fqt_quantize_seeds",
    "fqt_bhq_adaptive_groups", "fqt_bhq_adaptive_workspace",
    "fqt_linear_backward", "fqt_linear_backward_workspace",
    "fqt_linear_forward", "fqt_linear_forward_workspace",
    "fqt_conv_backward_im2col", "fqt_conv_backward_workspace",
    "fqt_gemm_s8s8_s64", "fqt_gemm_workspace", "fqt_gemm_s4s4_bf6", "fqt_gemm_s4s4_bf6_workspace",
    "fqt_probe_mfma_i8", "fqt_probe_copy",
    "fqt_workspace_status", "fqt_status_str", "fqt_version",
]

_lib = None


def load(path=LIB_PATH):
    """Load libfqt.so once and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2010_14298_amd.build (no CPU fallback)")
    lib = ctypes.CDLL(path)
    vp, i64, i32, u32, u64, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint32,
                                  ctypes.c_uint64, ctypes.c_size_t)
    qtp = ctypes.POINTER(QTensor)
    cfgp = ctypes.POINTER(BwdCfg)
    shp = ctypes.POINTER(ConvShape)
    sig = {
        "fqt_quantize_ptq": ([vp, i64, i64, i32, i32, u64, u32, i32, qtp, vp, sz, vp], i32),
        "fqt_quantize_psq": ([vp, i64, i64, i32, u64, u32, qtp, vp, sz, vp], i32),
        "fqt_quantize_psq_noalloc": ([vp, i64, i64, i32, u64, u32, qtp, vp, vp], i32),
        "fqt_quantize_bhq": ([vp, i64, i64, i32, i32, u64, u32, qtp, vp, sz, vp], i32),
        "fqt_quantize_shift": ([vp, i64, i64, i32, u64, u32, i32, qtp, vp, sz, vp], i32),
        "fqt_quantize_workspace": ([i32, i64, i64, i32], sz),
        "fqt_quantize_seeds": ([vp, i64, i64, i32, i32, i32, u64, i32, u32, qtp, vp, vp, vp, sz, vp], i32),
        "fqt_bhq_adaptive_groups": ([vp, i64, i64, i32, vp, vp, vp, sz, vp], i32),
        "fqt_bhq_adaptive_workspace": ([i64, i64], sz),
        "fqt_linear_backward": ([vp, vp, vp, i64, i64, i64, cfgp, vp, vp, vp, sz, vp], i32),
        "fqt_linear_backward_workspace": ([i64, i64, i64, cfgp], sz),
        "fqt_linear_forward": ([vp, vp, i64, i64, i64, i32, i32, i32, vp, vp, sz, vp], i32),
        "fqt_linear_forward_workspace": ([i64, i64, i64], sz),
        "fqt_conv_backward_im2col": ([vp, vp, vp, shp, cfgp, vp, vp, vp, sz, vp], i32),
        "fqt_conv_backward_workspace": ([shp, cfgp], sz),
        "fqt_gemm_s8s8_s64": ([vp, vp, i64, i64, i64, i64, i64, vp, vp, sz, vp], i32),
        "fqt_gemm_workspace": ([i64, i64, i64], sz),
        "fqt_gemm_s4s4_bf6": ([vp, vp, i64, i64, i64, i64, i64, vp, vp, sz, vp], i32),
        "fqt_gemm_s4s4_bf6_workspace": ([i64, i64, i64], sz),
        "fqt_probe_mfma_i8": ([i64, vp, ctypes.POINTER(ctypes.c_double), vp], i32),
        "fqt_probe_copy": ([vp, vp, sz, vp], i32),
        "fqt_workspace_status": ([vp, vp], i32),
        "fqt_status_str": ([i32], ctypes.c_char_p),
        "fqt_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(fn, code):
    if code != 0:
        raise FqtError(fn, code)


def _f32(x, name):
    if not (x.is_cuda and x.dtype == torch.float32 and x.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous float32 CUDA tensor")
    return x


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def cfg_struct(qb_x=("psq", 8, 0), qb_w=("ptq", 8, 0), f_bits=8, theta_bits=8, seed=0, trace=None,
               relu_input=False):
    return BwdCfg(QSpec(KINDS[qb_w[0]], int(qb_w[1]), int(qb_w[2])),
                  QSpec(KINDS[qb_x[0]], int(qb_x[1]), int(qb_x[2])), int(f_bits), int(theta_bits), int(seed),
                  ctypes.pointer(trace) if trace is not None else None, int(bool(relu_input)))


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ----------------------------------------------------------------------------

def fqt_quantize_workspace(kind, rows, cols, block_size=0):
    return load().fqt_quantize_workspace(KINDS.get(kind, kind), rows, cols, block_size)


def _quant_outputs(x, rows, cols, kind, transpose, code_sum):
    dev = x.device
    shape = (cols, rows) if transpose else (rows, cols)
    n_scale = 1 if kind == "ptq" else rows
    out = dict(q=torch.empty(shape, dtype=torch.int8, device=dev),
               scale=torch.empty(n_scale, dtype=torch.float32, device=dev),
               zero=torch.empty(n_scale, dtype=torch.float32, device=dev))
    if kind == "bhq":
        out["perm"] = torch.empty(rows, dtype=torch.int32, device=dev)
        out["group_off"] = torch.empty(rows + 1, dtype=torch.int32, device=dev)
        out["num_groups"] = torch.empty(1, dtype=torch.int32, device=dev)
    if kind == "shift":
        out["shift"] = torch.empty(rows, dtype=torch.int8, device=dev)
    if code_sum:
        out["code_sum"] = torch.empty(cols if transpose else rows, dtype=torch.int32, device=dev)
    qt = QTensor(out["q"].data_ptr(), out["scale"].data_ptr(), out["zero"].data_ptr(),
                 out["perm"].data_ptr() if "perm" in out else 0,
                 out["group_off"].data_ptr() if "group_off" in out else 0,
                 out["code_sum"].data_ptr() if "code_sum" in out else 0,
                 out["shift"].data_ptr() if "shift" in out else 0,
                 out["num_groups"].data_ptr() if "num_groups" in out else 0)
    return out, qt


def fqt_quantize_ptq(x, bits, stochastic, seed=0, stream=0, transpose=False, code_sum=False, ws=None):
    x = _f32(x, "x")
    rows, cols = x.shape
    out, qt = _quant_outputs(x, rows, cols, "ptq", transpose, code_sum)
    if ws is None:
        ws = _workspace(fqt_quantize_workspace("ptq", rows, cols), x.device)
    rc = load().fqt_quantize_ptq(_ptr(x), rows, cols, bits, int(bool(stochastic)), seed, stream,
                                 int(bool(transpose)), ctypes.byref(qt), _ptr(ws), ws.numel(), _stream())
    _check("fqt_quantize_ptq", rc)
    out["ws"] = ws
    return out


def fqt_quantize_shift(x, bits, seed=0, stream=0, transpose=False, code_sum=False, ws=None):
    x = _f32(x, "x")
    rows, cols = x.shape
    out, qt = _quant_outputs(x, rows, cols, "shift", transpose, code_sum)
    if ws is None:
        ws = _workspace(fqt_quantize_workspace("shift", rows, cols), x.device)
    rc = load().fqt_quantize_shift(_ptr(x), rows, cols, bits, seed, stream, int(bool(transpose)), ctypes.byref(qt),
                                   _ptr(ws), ws.numel(), _stream())
    _check("fqt_quantize_shift", rc)
    out["ws"] = ws
    return out


def fqt_quantize_psq(x, bits, seed=0, stream=0, code_sum=False, ws=None):
    x = _f32(x, "x")
    rows, cols = x.shape
    out, qt = _quant_outputs(x, rows, cols, "psq", False, code_sum)
    if ws is None:
        ws = _workspace(fqt_quantize_workspace("psq", rows, cols), x.device)
    rc = load().fqt_quantize_psq(_ptr(x), rows, cols, bits, seed, stream, ctypes.byref(qt), _ptr(ws), ws.numel(),
                                 _stream())
    _check("fqt_quantize_psq", rc)
    out["ws"] = ws
    return out


def fqt_quantize_seeds(x, kind, bits, nseeds, block_size=0, seed=0, stream=0, ws=None):
    """Seed batch: per element the sum over keys seed .. seed + nseeds - 1 of
    the code and of its square (int32 tensors sum_c, sum_c2), plus the plan."""
    x = _f32(x, "x")
    rows, cols = x.shape
    out, qt = _quant_outputs(x, rows, cols, kind, False, False)
    out.pop("q")
    qt.q = 0
    out["sum_c"] = torch.empty((rows, cols), dtype=torch.int32, device=x.device)
    out["sum_c2"] = torch.empty((rows, cols), dtype=torch.int32, device=x.device)
    if ws is None:
        ws = _workspace(fqt_quantize_workspace(kind, rows, cols, block_size), x.device)
    rc = load().fqt_quantize_seeds(_ptr(x), rows, cols, KINDS[kind], bits, block_size, seed, nseeds, stream,
                                   ctypes.byref(qt), _ptr(out["sum_c"]), _ptr(out["sum_c2"]), _ptr(ws), ws.numel(),
                                   _stream())
    _check("fqt_quantize_seeds", rc)
    out["ws"] = ws
    return out


def fqt_quantize_psq_noalloc(x, bits, seed=0, stream=0, code_sum=False, out=None):
    """fqt_quantize_psq on the library's fixed scratch memory (no workspace).
    `out` may hold preallocated q / scale / zero (/ code_sum) tensors; returns
    them with a device status tensor of 4 uint32 words (as int32)."""
    x = _f32(x, "x")
    rows, cols = x.shape
    fresh, _ = _quant_outputs(x, rows, cols, "psq", False, code_sum)
    out = dict(fresh, **(out or {}))
    qt = QTensor(out["q"].data_ptr(), out["scale"].data_ptr(), out["zero"].data_ptr(), 0, 0,
                 out["code_sum"].data_ptr() if "code_sum" in out else 0, 0, 0)
    status = torch.full((4,), -1, dtype=torch.int32, device=x.device)
    rc = load().fqt_quantize_psq_noalloc(_ptr(x), rows, cols, bits, seed, stream, ctypes.byref(qt), _ptr(status),
                                         _stream())
    _check("fqt_quantize_psq_noalloc", rc)
    out["status"] = status
    return out


def fqt_quantize_bhq(x, bits, block_size, seed=0, stream=0, code_sum=False, ws=None):
    x = _f32(x, "x")
    rows, cols = x.shape
    out, qt = _quant_outputs(x, rows, cols, "bhq", False, code_sum)
    if ws is None:
        ws = _workspace(fqt_quantize_workspace("bhq", rows, cols, block_size), x.device)
    rc = load().fqt_quantize_bhq(_ptr(x), rows, cols, bits, block_size, seed, stream, ctypes.byref(qt), _ptr(ws),
                                 ws.numel(), _stream())
    _check("fqt_quantize_bhq", rc)
    out["ws"] = ws
    return out


def fqt_bhq_adaptive_groups(x, bits, objective=True, ws=None):
    """App. D's number of groups (device int32 [1]) and, with objective=True,
    the score of every G (device float64 [rows]); asynchronous."""
    x = _f32(x, "x")
    rows, cols = x.shape
    if ws is None:
        ws = _workspace(load().fqt_bhq_adaptive_workspace(rows, cols), x.device)
    G = torch.empty(1, dtype=torch.int32, device=x.device)
    obj = torch.empty(rows, dtype=torch.float64, device=x.device) if objective else None
    rc = load().fqt_bhq_adaptive_groups(_ptr(x), rows, cols, bits, _ptr(G), _ptr(obj), _ptr(ws), ws.numel(),
                                        _stream())
    _check("fqt_bhq_adaptive_groups", rc)
    return G, obj, ws


def fqt_linear_backward_workspace(N, d_in, d_out, cfg):
    return load().fqt_linear_backward_workspace(N, d_in, d_out, ctypes.byref(cfg))


def fqt_linear_backward(X, W, G, qb_x=("psq", 8, 0), qb_w=("ptq", 8, 0), f_bits=8, theta_bits=8, seed=0,
                        grad_W=None, grad_X=None, ws=None, trace=None, relu_input=False, codes=None,
                        packed_codes=False):
    """codes: optional dict to receive the gradient codes the contractions read:
    it is filled with qb2 [N, d_out], qb1_t [d_out, N] (int8, slot order) and,
    for BHQ, perm [N]."""
    X, W, G = _f32(X, "X"), _f32(W, "W"), _f32(G, "G")
    N, d_in = X.shape
    d_out = W.shape[0]
    if W.shape != (d_out, d_in) or G.shape != (N, d_out):
        raise ValueError("shapes: X [N, d_in], W [d_out, d_in], G [N, d_out]")
    cfg = cfg_struct(qb_x, qb_w, f_bits, theta_bits, seed, trace, relu_input)
    cfg.packed_codes = int(bool(packed_codes))
    if codes is not None:
        codes["qb2"] = torch.empty((N, d_out), dtype=torch.int8, device=X.device)
        codes["qb1_t"] = torch.empty((d_out, N), dtype=torch.int8, device=X.device)
        cfg.qb2_codes = codes["qb2"].data_ptr()
        cfg.qb1_codes = codes["qb1_t"].data_ptr()
        if KINDS.get(qb_x[0], qb_x[0]) == FQT_BHQ:
            codes["perm"] = torch.empty(N, dtype=torch.int32, device=X.device)
            cfg.perm = codes["perm"].data_ptr()
    if grad_W is None:
        grad_W = torch.empty((d_out, d_in), dtype=torch.float32, device=X.device)
    if grad_X is None:
        grad_X = torch.empty((N, d_in), dtype=torch.float32, device=X.device)
    if ws is None:
        ws = _workspace(fqt_linear_backward_workspace(N, d_in, d_out, cfg), X.device)
    rc = load().fqt_linear_backward(_ptr(X), _ptr(W), _ptr(G), N, d_in, d_out, ctypes.byref(cfg), _ptr(grad_W),
                                    _ptr(grad_X), _ptr(ws), ws.numel(), _stream())
    _check("fqt_linear_backward", rc)
    return grad_W, grad_X, ws


def fqt_linear_forward_workspace(N, d_in, d_out):
    return load().fqt_linear_forward_workspace(N, d_in, d_out)


def fqt_linear_forward(X, W, f_bits=8, theta_bits=8, relu=False, Y=None, ws=None):
    """Y = Q_f(X) Q_theta(W)^T (then max(., 0) when relu); returns (Y, ws)."""
    X, W = _f32(X, "X"), _f32(W, "W")
    N, d_in = X.shape
    d_out = W.shape[0]
    if W.shape != (d_out, d_in):
        raise ValueError("shapes: X [N, d_in], W [d_out, d_in]")
    if Y is None:
        Y = torch.empty((N, d_out), dtype=torch.float32, device=X.device)
    if ws is None:
        ws = _workspace(fqt_linear_forward_workspace(N, d_in, d_out), X.device)
    rc = load().fqt_linear_forward(_ptr(X), _ptr(W), N, d_in, d_out, int(f_bits), int(theta_bits), int(bool(relu)),
                                   _ptr(Y), _ptr(ws), ws.numel(), _stream())
    _check("fqt_linear_forward", rc)
    return Y, ws


def conv_shape(n, c, h, w, o, kh, kw, stride, pad):
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (w + 2 * pad - kw) // stride + 1
    return ConvShape(n, c, h, w, o, kh, kw, stride, pad, ho, wo)


def fqt_conv_backward_workspace(shape, cfg):
    return load().fqt_conv_backward_workspace(ctypes.byref(shape), ctypes.byref(cfg))


def fqt_conv_backward_im2col(X, W, G, stride, pad, qb_x=("bhq", 5, 64), qb_w=("ptq", 8, 0), f_bits=8,
                             theta_bits=8, seed=0, grad_W=None, grad_X=None, ws=None, trace=None, input_grad=True):
    """input_grad=False passes a NULL grad_X (no input gradient); grad_X is then returned as None."""
    X, W, G = _f32(X, "X"), _f32(W, "W"), _f32(G, "G")
    n, h, w, c = X.shape
    o, kh, kw, _ = W.shape
    sh = conv_shape(n, c, h, w, o, kh, kw, stride, pad)
    if tuple(G.shape) != (n, sh.ho, sh.wo, o) or W.shape[3] != c:
        raise ValueError("shapes: X [n,h,w,c], W [o,kh,kw,c], G [n,ho,wo,o]")
    cfg = cfg_struct(qb_x, qb_w, f_bits, theta_bits, seed, trace)
    if grad_W is None:
        grad_W = torch.empty(W.shape, dtype=torch.float32, device=X.device)
    if not input_grad:
        grad_X = None
    elif grad_X is None:
        grad_X = torch.empty(X.shape, dtype=torch.float32, device=X.device)
    if ws is None:
        ws = _workspace(fqt_conv_backward_workspace(sh, cfg), X.device)
    rc = load().fqt_conv_backward_im2col(_ptr(X), _ptr(W), _ptr(G), ctypes.byref(sh), ctypes.byref(cfg),
                                         _ptr(grad_W), _ptr(grad_X), _ptr(ws), ws.numel(), _stream())
    _check("fqt_conv_backward_im2col", rc)
    return grad_W, grad_X, ws


def fqt_gemm_workspace(M, N, K):
    return load().fqt_gemm_workspace(M, N, K)


def fqt_gemm_s8s8_s64(A, B, ws=None):
    """C [M, N] int64 = A [M, K] int8 . B [N, K]^T int8 (exact)."""
    if not (A.is_cuda and B.is_cuda and A.dtype == torch.int8 and B.dtype == torch.int8):
        raise ValueError("A, B must be int8 CUDA tensors")
    M, K = A.shape
    N = B.shape[0]
    if B.shape[1] != K or A.stride(1) != 1 or B.stride(1) != 1:
        raise ValueError("A [M, K], B [N, K], K contiguous")
    C = torch.empty((M, N), dtype=torch.int64, device=A.device)
    if ws is None:
        ws = _workspace(fqt_gemm_workspace(M, N, K), A.device)
    rc = load().fqt_gemm_s8s8_s64(_ptr(A), _ptr(B), M, N, K, A.stride(0), B.stride(0), _ptr(C), _ptr(ws),
                                  ws.numel(), _stream())
    _check("fqt_gemm_s8s8_s64", rc)
    return C


def fqt_gemm_s4s4_bf6_workspace(M, N, K):
    return load().fqt_gemm_s4s4_bf6_workspace(M, N, K)


def fqt_gemm_s4s4_bf6(A, B, ws=None, C=None):
    """C [M, N] int64 = A [M, K] . B [N, K]^T for codes in [-8, 7], on the 6-bit
    float matrix cores (exact).  Returns (C, ws); check fqt_workspace_status(ws)."""
    if not (A.is_cuda and B.is_cuda and A.dtype == torch.int8 and B.dtype == torch.int8):
        raise ValueError("A, B must be int8 CUDA tensors")
    M, K = A.shape
    N = B.shape[0]
    if B.shape[1] != K or A.stride(1) != 1 or B.stride(1) != 1:
        raise ValueError("A [M, K], B [N, K], K contiguous")
    if C is None:
        C = torch.empty((M, N), dtype=torch.int64, device=A.device)
    if ws is None:
        ws = _workspace(fqt_gemm_s4s4_bf6_workspace(M, N, K), A.device)
    rc = load().fqt_gemm_s4s4_bf6(_ptr(A), _ptr(B), M, N, K, A.stride(0), B.stride(0), _ptr(C), _ptr(ws),
                                  ws.numel(), _stream())
    _check("fqt_gemm_s4s4_bf6", rc)
    return C, ws


def fqt_workspace_status(ws):
    return load().fqt_workspace_status(_ptr(ws), _stream())


def fqt_version():
    return load().fqt_version().decode()


# ----------------------------------------------------------------------------
# HIP events for fqt_trace (profiling only)
# ----------------------------------------------------------------------------
_hip = None


def _hiprt():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        _hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        _hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    return _hip


def make_trace():
    """A Trace with freshly created HIP events for every phase."""
    hip = _hiprt()
    t = Trace()
    for i in range(TRACE_PHASES):
        for arr in (t.start, t.stop):
            ev = ctypes.c_void_p()
            if hip.hipEventCreate(ctypes.byref(ev)) != 0:
                raise RuntimeError("hipEventCreate failed")
            arr[i] = ev
    t.count = TRACE_PHASES
    return t


def trace_ms(t):
    """Milliseconds of each phase of a completed traced call."""
    hip = _hiprt()
    out = []
    for i in range(t.count):
        ms = ctypes.c_float()
        if hip.hipEventElapsedTime(ctypes.byref(ms), t.start[i], t.stop[i]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        out.append(ms.value)
    return out


def free_trace(t):
    hip = _hiprt()
    for i in range(t.count):
        hip.hipEventDestroy(t.start[i])
        hip.hipEventDestroy(t.stop[i])


# ----------------------------------------------------------------------------
# multi-layer chain: a ReLU MLP, one library call per layer
# ----------------------------------------------------------------------------
def mlp_forward(X, Ws, f_bits=8, theta_bits=8, ws=None):
    """Layer inputs A_0 = X, A_{i+1} = ReLU(Q_f(A_i) Q_theta(W_i)^T), and the
    top layer's (linear) output.  Returns (acts, Z_top)."""
    acts = [X]
    Z = None
    for i, W in enumerate(Ws):
        last = i == len(Ws) - 1
        need = fqt_linear_forward_workspace(acts[-1].shape[0], W.shape[1], W.shape[0])
        Y, ws = fqt_linear_forward(acts[-1], W, f_bits, theta_bits, relu=not last,
                                   ws=ws if ws is not None and ws.numel() >= need else None)
        if last:
            Z = Y
        else:
            acts.append(Y)
    return acts, Z


def mlp_backward(acts, Ws, G, specs, seeds, qb_w=("ptq", 8, 0), f_bits=8, theta_bits=8):
    """FQT backward of the chain from the top output gradient G: layer i runs
    fqt_linear_backward with quantizer specs[i] and seed seeds[i]; below the
    top, grad_X is masked by the ReLU that produced the layer input.
    Returns (grads_W, dZ) per layer (dZ[i] is layer i's output gradient)."""
    L = len(Ws)
    grads, dZs = [None] * L, [None] * L
    dZ = G
    for i in range(L - 1, -1, -1):
        dZs[i] = dZ
        gW, gX, ws = fqt_linear_backward(acts[i], Ws[i], dZ, qb_x=specs[i], qb_w=qb_w, f_bits=f_bits,
                                         theta_bits=theta_bits, seed=seeds[i], relu_input=i > 0)
        grads[i] = gW
        dZ = gX
    return grads, dZs


# ----------------------------------------------------------------------------
# machine probes (measured peaks)
# ----------------------------------------------------------------------------
def fqt_probe_mfma_i8(iters, sink):
    """Enqueue the int8 matrix-core loop; returns its operation count."""
    ops = ctypes.c_double(0.0)
    _check("fqt_probe_mfma_i8", load().fqt_probe_mfma_i8(int(iters), _ptr(sink), ctypes.byref(ops), _stream()))
    return ops.value


def fqt_probe_copy(src, dst):
    """Enqueue a streaming copy of src into dst (same byte size); returns bytes moved."""
    nbytes = src.numel() * src.element_size()
    _check("fqt_probe_copy", load().fqt_probe_copy(_ptr(src), _ptr(dst), nbytes, _stream()))
    return 2 * nbytes
