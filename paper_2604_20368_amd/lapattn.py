"""ctypes binding of the lapattn C ABI (include/lapattn.h).

Argument marshalling only: tensors are passed as device pointers, the stream is
torch's current HIP stream, and every step of the computation runs in the HIP
library.  If the library is missing the calls raise; there is no fallback.
"""
import ctypes
import os

# LAPATTN_LIB: another build of the same library (the CPU sanitizer run loads an instrumented one)
LIB_PATH = os.environ.get("LAPATTN_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblapattn.so")

LAPATTN_FP32, LAPATTN_BF16 = 0, 1
LAPATTN_NORM_INLINE, LAPATTN_NORM_ROWSUM, LAPATTN_NORM_NONE, LAPATTN_NORM_MSPACE = 0, 1, 2, 3
LAPATTN_OK, LAPATTN_ERR_NULL, LAPATTN_ERR_SHAPE, LAPATTN_ERR_PARAM = 0, 1, 2, 3
LAPATTN_ERR_UNSUPPORTED, LAPATTN_ERR_WORKSPACE, LAPATTN_ERR_HIP, LAPATTN_ERR_ALIGN = 4, 5, 6, 7
LAPATTN_ERR_SCRATCH = 8
LAPATTN_WS_BACKWARD, LAPATTN_WS_DWC = 1, 2

EXPORTS = ("lapattn_workspace_size", "lapattn_forward", "lapattn_backward", "lapattn_status_str",
           "lapattn_timing_enable", "lapattn_timing_read", "lapattn_timing_name", "lapattn_forward_noalloc")


class lapattn_opts(ctypes.Structure):
    _fields_ = [("norm", ctypes.c_int), ("eps", ctypes.c_float), ("grid_w", ctypes.c_int), ("pool_r", ctypes.c_int),
                ("dwc_k", ctypes.c_int), ("dwc_w", ctypes.c_void_p), ("dwc_b", ctypes.c_void_p),
                ("dwc_dw", ctypes.c_void_p), ("dwc_db", ctypes.c_void_p), ("whiten", ctypes.c_void_p),
                ("save", ctypes.c_int)]


class LapattnError(RuntimeError):
    def __init__(self, code, where):
        super().__init__("%s failed: %s (status %d)" % (where, lapattn_status_str(code), code))
        self.code = code


_lib = None


def library():
    """Open liblapattn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("HIP library %s is missing: build it with __graft_entry__.build() "
                           "or python -m paper_2604_20368_amd.build" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, ci, cf, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.lapattn_workspace_size.restype = sz
    lib.lapattn_workspace_size.argtypes = [ci] * 8
    lib.lapattn_forward.restype = ci
    lib.lapattn_forward.argtypes = [vp] * 4 + [ci] * 5 + [cf, ci, ci, ctypes.POINTER(lapattn_opts), vp, sz, vp]
    lib.lapattn_backward.restype = ci
    lib.lapattn_backward.argtypes = [vp] * 7 + [ci] * 5 + [cf, ci, ci, ctypes.POINTER(lapattn_opts), vp, sz, vp]
    lib.lapattn_forward_noalloc.restype = ci
    lib.lapattn_forward_noalloc.argtypes = [vp] * 4 + [ci] * 5 + [cf, ci, ci, ctypes.POINTER(lapattn_opts), vp]
    lib.lapattn_status_str.restype = ctypes.c_char_p
    lib.lapattn_status_str.argtypes = [ci]
    lib.lapattn_timing_enable.restype = ci
    lib.lapattn_timing_enable.argtypes = [ci]
    lib.lapattn_timing_read.restype = ci
    lib.lapattn_timing_read.argtypes = [ctypes.POINTER(ctypes.c_float), ci]
    lib.lapattn_timing_name.restype = ctypes.c_char_p
    lib.lapattn_timing_name.argtypes = [ci]
    _lib = lib
    return lib


# ------------------------------------------------------------------------------ raw C-ABI calls

def lapattn_status_str(code):
    return library().lapattn_status_str(int(code)).decode()


def lapattn_workspace_size(B, H, n, d, m, ns_iters, dtype, flags):
    """flags: LAPATTN_WS_BACKWARD and/or LAPATTN_WS_DWC (a bool counts as the backward flag)."""
    return int(library().lapattn_workspace_size(B, H, n, d, m, ns_iters, dtype, int(flags)))


def _opts(norm, eps, grid=None, dwc=None, whiten=None, save=False):
    gw, r = grid if grid is not None else (0, 0)
    k, w, b, dw, db = dwc if dwc is not None else (0, None, None, None, None)
    return ctypes.byref(lapattn_opts(int(norm), float(eps), int(gw), int(r), int(k), w, b, dw, db, whiten,
                                     int(bool(save))))


def lapattn_forward(Q, K, V, Out, B, H, n, d, m, lam, ns_iters, dtype, norm=LAPATTN_NORM_INLINE, eps=0.0,
                    workspace=0, workspace_bytes=0, stream=0, grid=None, dwc=None, whiten=None, save=False):
    """Raw call with integer device addresses; returns the status code.  grid = (W', r): the
    W'-wide token map, with r x r window landmarks when r > 0 (None: no map, balanced
    segments).  dwc = (k, filters, bias, dfilters, dbias) addresses of the convolution branch;
    whiten the address of the landmark-space whitening."""
    return library().lapattn_forward(Q, K, V, Out, B, H, n, d, m, float(lam), ns_iters, dtype,
                                     _opts(norm, eps, grid, dwc, whiten, save), workspace, workspace_bytes, stream)


def lapattn_forward_noalloc(Q, K, V, Out, B, H, n, d, m, lam, ns_iters, dtype, norm=LAPATTN_NORM_INLINE, eps=0.0,
                            stream=0, grid=None, dwc=None, whiten=None, save=False):
    """Raw call of the forward on the library's static scratch array (no workspace argument)."""
    return library().lapattn_forward_noalloc(Q, K, V, Out, B, H, n, d, m, float(lam), ns_iters, dtype,
                                             _opts(norm, eps, grid, dwc, whiten, save), stream)


def lapattn_backward(Q, K, V, dO, dQ, dK, dV, B, H, n, d, m, lam, ns_iters, dtype, norm=LAPATTN_NORM_INLINE,
                     eps=0.0, workspace=0, workspace_bytes=0, stream=0, grid=None, dwc=None, whiten=None,
                     save=False):
    return library().lapattn_backward(Q, K, V, dO, dQ, dK, dV, B, H, n, d, m, float(lam), ns_iters, dtype,
                                      _opts(norm, eps, grid, dwc, whiten, save), workspace, workspace_bytes, stream)


def lapattn_timing_enable(on):
    return library().lapattn_timing_enable(int(bool(on)))


def lapattn_timing_read(cap=32):
    buf = (ctypes.c_float * cap)()
    k = library().lapattn_timing_read(buf, cap)
    if k < 0:
        raise RuntimeError("lapattn_timing_read failed")
    return [(library().lapattn_timing_name(i).decode(), buf[i]) for i in range(min(k, cap))]


# ------------------------------------------------------------------------------ torch marshalling

def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return LAPATTN_FP32
    if t.dtype == torch.bfloat16:
        return LAPATTN_BF16
    raise TypeError("lapattn takes float32 or bfloat16 tensors, got %s" % t.dtype)


def _check(*ts):
    import torch
    ref = ts[0]
    for t in ts:
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError("lapattn needs device tensors")
        if not t.is_contiguous() or t.shape != ref.shape or t.dtype != ref.dtype or t.device != ref.device:
            raise ValueError("lapattn needs contiguous [B,H,n,d] tensors of one dtype and device")
    if ref.dim() != 4:
        raise ValueError("lapattn needs [B,H,n,d] tensors")


def _stream(t):
    import torch
    return torch.cuda.current_stream(t.device).cuda_stream


def workspace(Q, m, ns_iters, for_backward=False, dwc=False):
    import torch
    B, H, n, d = Q.shape
    flags = (LAPATTN_WS_BACKWARD if for_backward else 0) | (LAPATTN_WS_DWC if dwc else 0)
    nbytes = lapattn_workspace_size(B, H, n, d, m, ns_iters, _dtype_code(Q), flags)
    if nbytes == 0:
        raise ValueError("invalid lapattn sizes")
    return torch.empty(nbytes, dtype=torch.uint8, device=Q.device)


def _dwc_args(Q, dwc, grads=None):
    """(k, filters, bias, dfilters, dbias) addresses for dwc = (filters [H][d][k][k], bias [H][d] or
    None), fp32 device tensors; grads = (dfilters, dbias) or None."""
    import torch
    if dwc is None:
        return None
    w, b = dwc
    H, d = Q.shape[1], Q.shape[3]
    k = w.shape[-1]
    for t, shape in ((w, (H, d, k, k)), (b, (H, d))) + (() if grads is None else ((grads[0], (H, d, k, k)),
                                                                                     (grads[1], (H, d)))):
        if t is None:
            continue
        if (not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != torch.float32 or not t.is_contiguous()
                or tuple(t.shape) != shape or t.device != Q.device):
            raise ValueError("convolution filters and bias are contiguous fp32 device tensors [H][d][k][k] and [H][d]")
    dw, db = (None, None) if grads is None else grads
    ptr = lambda t: None if t is None else t.data_ptr()
    return (k, ptr(w), ptr(b), ptr(dw), ptr(db))


def _whiten_arg(Q, m, whiten):
    import torch
    if whiten is None:
        return None
    if (not isinstance(whiten, torch.Tensor) or not whiten.is_cuda or whiten.dtype != torch.float32
            or not whiten.is_contiguous() or tuple(whiten.shape) != (Q.shape[1], m) or whiten.device != Q.device):
        raise ValueError("the whitening is a contiguous fp32 device tensor [H][m]")
    return whiten.data_ptr()


def forward(Q, K, V, m, lam, ns_iters, norm=LAPATTN_NORM_INLINE, eps=0.0, out=None, ws=None, grid=None, dwc=None,
            whiten=None, save=False):
    """Out = lapattn(Q, K, V) on torch's current stream; grid = (W', r) the token map (r > 0: window
    landmarks), dwc = (filters, bias) adds the convolution branch over that map, whiten [H][m]
    is the diagonal of LAPATTN_NORM_MSPACE; save keeps the internals in ws (a backward-sized
    workspace) for backward(..., save=True, ws=ws)."""
    import torch
    _check(Q, K, V)
    out = torch.empty_like(Q) if out is None else out
    _check(Q, out)
    ws = workspace(Q, m, ns_iters, save, dwc is not None) if ws is None else ws
    B, H, n, d = Q.shape
    rc = lapattn_forward(Q.data_ptr(), K.data_ptr(), V.data_ptr(), out.data_ptr(), B, H, n, d, m, lam, ns_iters,
                         _dtype_code(Q), norm, eps, ws.data_ptr(), ws.numel(), _stream(Q), grid, _dwc_args(Q, dwc),
                         _whiten_arg(Q, m, whiten), save)
    if rc != LAPATTN_OK:
        raise LapattnError(rc, "lapattn_forward")
    return out


def forward_noalloc(Q, K, V, m, lam, ns_iters, norm=LAPATTN_NORM_INLINE, eps=0.0, out=None, grid=None, dwc=None,
                    whiten=None):
    """Out = lapattn(Q, K, V) through lapattn_forward_noalloc: no workspace is allocated (out is
    allocated here unless given)."""
    import torch
    _check(Q, K, V)
    out = torch.empty_like(Q) if out is None else out
    _check(Q, out)
    B, H, n, d = Q.shape
    rc = lapattn_forward_noalloc(Q.data_ptr(), K.data_ptr(), V.data_ptr(), out.data_ptr(), B, H, n, d, m, lam,
                                 ns_iters, _dtype_code(Q), norm, eps, _stream(Q), grid, _dwc_args(Q, dwc),
                                 _whiten_arg(Q, m, whiten))
    if rc != LAPATTN_OK:
        raise LapattnError(rc, "lapattn_forward_noalloc")
    return out


def backward(Q, K, V, dO, m, lam, ns_iters, norm=LAPATTN_NORM_INLINE, eps=0.0, grads=None, ws=None, grid=None,
             dwc=None, dwc_grads=None, whiten=None, save=False):
    """(dQ, dK, dV) of sum(Out * dO) on torch's current stream; with dwc = (filters, bias) also the
    filter and bias gradients: (dQ, dK, dV, dfilters, dbias)."""
    import torch
    _check(Q, K, V, dO)
    dQ, dK, dV = grads if grads is not None else (torch.empty_like(Q), torch.empty_like(Q), torch.empty_like(Q))
    _check(Q, dQ, dK, dV)
    if dwc is not None and dwc_grads is None:
        dwc_grads = (torch.empty_like(dwc[0]), torch.empty((Q.shape[1], Q.shape[3]), dtype=torch.float32,
                                                             device=Q.device))
    ws = workspace(Q, m, ns_iters, True, dwc is not None) if ws is None else ws
    B, H, n, d = Q.shape
    rc = lapattn_backward(Q.data_ptr(), K.data_ptr(), V.data_ptr(), dO.data_ptr(), dQ.data_ptr(), dK.data_ptr(),
                          dV.data_ptr(), B, H, n, d, m, lam, ns_iters, _dtype_code(Q), norm, eps, ws.data_ptr(),
                          ws.numel(), _stream(Q), grid, _dwc_args(Q, dwc, dwc_grads), _whiten_arg(Q, m, whiten),
                          save)
    if rc != LAPATTN_OK:
        raise LapattnError(rc, "lapattn_backward")
    return (dQ, dK, dV) if dwc is None else (dQ, dK, dV) + tuple(dwc_grads)
