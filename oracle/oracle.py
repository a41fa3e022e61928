"""ctypes marshalling for the fp64 oracle in ``lapattn_oracle.c``.

TEST INFRASTRUCTURE ONLY (see the package docstring).  No arithmetic of the
method is done here: every function converts its numpy arguments to contiguous
fp64 buffers and calls the C oracle.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lapattn_oracle.c")
_LIB = os.path.join(_HERE, "liblapattn_oracle.so")

NORM_INLINE, NORM_ROWSUM, NORM_NONE, NORM_MSPACE = 0, 1, 2, 3

_lib = None
_dp = ctypes.POINTER(ctypes.c_double)


def build(force=True):
    """Compile the oracle with gcc (plain -O2, no fp contraction, OpenMP)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
           "-shared", "-std=c11", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.check_call(cmd, cwd=_HERE)
    os.replace(tmp, _LIB)
    return _LIB


def load():
    global _lib
    if _lib is not None:
        return _lib
    if os.environ.get("LAPATTN_ORACLE_LIB"):   # another build of lapattn_oracle.c (the sanitizer run's)
        _lib = _configure(ctypes.CDLL(os.environ["LAPATTN_ORACLE_LIB"]))
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    _lib = _configure(ctypes.CDLL(_LIB))
    return _lib


class using:
    """Context manager: route every call through another build of the oracle
    (the mutation tests compile deliberately broken copies on the CPU)."""

    def __init__(self, path):
        self.lib = _configure(ctypes.CDLL(path))

    def __enter__(self):
        global _lib
        self.prev, _lib = _lib, self.lib
        return self

    def __exit__(self, *exc):
        global _lib
        _lib = self.prev
        return False


def _configure(lib):
    lib.lapattn_oracle_kernel.restype = ctypes.c_double
    lib.lapattn_oracle_kernel.argtypes = [_dp, _dp, ctypes.c_int, ctypes.c_double]
    lib.lapattn_oracle_segments.restype = ctypes.c_int
    lib.lapattn_oracle_segments.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    lib.lapattn_oracle_ns.restype = ctypes.c_double
    lib.lapattn_oracle_ns.argtypes = [_dp, ctypes.c_int, ctypes.c_int, ctypes.c_double, _dp]
    lib.lapattn_oracle_forward.restype = ctypes.c_int
    lib.lapattn_oracle_windows.restype = ctypes.c_int
    lib.lapattn_oracle_windows.argtypes = [ctypes.c_int] * 4 + [ctypes.POINTER(ctypes.c_int)] * 2
    lib.lapattn_oracle_forward.argtypes = ([_dp] * 4 + [ctypes.c_int] * 5 + [ctypes.c_double, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_int] + [_dp] * 9)
    lib.lapattn_oracle_backward.restype = ctypes.c_int
    lib.lapattn_oracle_backward.argtypes = ([_dp] * 7 + [ctypes.c_int] * 5 + [ctypes.c_double, ctypes.c_int,
                                            ctypes.c_int, ctypes.c_double, ctypes.c_int, ctypes.c_int, _dp])
    lib.lapattn_oracle_dwc.restype = ctypes.c_int
    lib.lapattn_oracle_dwc.argtypes = [_dp] * 4 + [ctypes.c_int] * 6
    lib.lapattn_oracle_dwc_backward.restype = ctypes.c_int
    lib.lapattn_oracle_dwc_backward.argtypes = [_dp] * 6 + [ctypes.c_int] * 6
    lib.lapattn_oracle_threads.restype = ctypes.c_int
    lib.lapattn_oracle_threads.argtypes = []
    return lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a):
    return None if a is None else a.ctypes.data_as(_dp)


def threads():
    return load().lapattn_oracle_threads()


def kernel(x, y, lam):
    x, y = _f64(x), _f64(y)
    assert x.shape == y.shape and x.ndim == 1
    return load().lapattn_oracle_kernel(_p(x), _p(y), x.shape[0], float(lam))


def segments(n, m):
    starts = (ctypes.c_int * (m + 1))()
    rc = load().lapattn_oracle_segments(int(n), int(m), starts)
    if rc:
        raise ValueError("bad segment arguments n=%d m=%d" % (n, m))
    return np.array(list(starts), dtype=np.int64)


def windows(n, m, grid=None):
    """(starts, members) of the landmark membership; grid = (W', r) for r x r windows of the
    H' x W' token map, None for the balanced segments."""
    gw, r = grid if grid is not None else (0, 0)
    starts = (ctypes.c_int * (m + 1))()
    members = (ctypes.c_int * n)()
    if load().lapattn_oracle_windows(int(n), int(m), int(gw), int(r), starts, members):
        raise ValueError("bad landmark windows n=%d m=%d grid=%r" % (n, m, grid))
    return np.array(list(starts), dtype=np.int64), np.array(list(members), dtype=np.int64)


def ns(W, T, eps=0.0):
    """Returns (Xs, c): Xs[t] = X_t for t = 0..T, c = the X0 scale."""
    W = _f64(W)
    m = W.shape[0]
    assert W.shape == (m, m)
    Xs = np.empty((T + 1, m, m), dtype=np.float64)
    c = load().lapattn_oracle_ns(_p(W), m, int(T), float(eps), _p(Xs))
    return Xs, c


def _attention_grid(grid):
    """(W', r) of the landmark windows for the attention part: (0, 0) when there are none
    (grid None, or a token map with r = 0 that only the convolution branch uses)."""
    if grid is None or grid[1] == 0:
        return 0, 0
    return grid


def dwc(V, weight, bias, grid_w):
    """DWC(V) of Eq. (7) (R14): weight [H][d][k][k], bias [H][d] or None, over the token map
    of width grid_w.  Returns E [B][H][n][d]."""
    V, weight = _f64(V), _f64(weight)
    B, H, n, d = V.shape
    k = weight.shape[-1]
    assert weight.shape == (H, d, k, k)
    bias = None if bias is None else _f64(bias)
    assert bias is None or bias.shape == (H, d)
    E = np.empty_like(V)
    if load().lapattn_oracle_dwc(_p(V), _p(weight), _p(bias), _p(E), B, H, n, d, int(grid_w), int(k)):
        raise ValueError("oracle dwc rejected its arguments")
    return E


def dwc_backward(V, weight, dE, grid_w):
    """(dV, dweight, dbias) of sum(DWC(V) * dE): the convolution's part of dV only."""
    V, weight, dE = _f64(V), _f64(weight), _f64(dE)
    B, H, n, d = V.shape
    k = weight.shape[-1]
    dV, dW, db = np.empty_like(V), np.empty_like(weight), np.empty((H, d))
    if load().lapattn_oracle_dwc_backward(_p(V), _p(weight), _p(dE), _p(dV), _p(dW), _p(db),
                                          B, H, n, d, int(grid_w), int(k)):
        raise ValueError("oracle dwc backward rejected its arguments")
    return dV, dW, db


def _whiten(whiten, H, m):
    if whiten is None:
        return None
    w = _f64(whiten)
    assert w.shape == (H, m)
    return w


def forward(Q, K, V, m, lam, T, norm=NORM_INLINE, eps=0.0, intermediates=False, grid=None, dwc_branch=None,
            whiten=None):
    """Out = Z V (+ DWC(V) when dwc_branch = (weight, bias) is given, over the token map of width
    grid[0]); grid = (W', r) selects r x r landmark windows when r > 0; whiten [H][m] is the
    diagonal of NORM_MSPACE (None: ones)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    B, H, n, d = Q.shape
    assert K.shape == Q.shape and V.shape == Q.shape
    out = np.empty_like(Q)
    inter = None
    ptrs = [None] * 8
    if intermediates:
        inter = dict(
            Qt=np.empty((B, H, m, d)), Kt=np.empty((B, H, m, d)), W=np.empty((B, H, m, m)),
            Xs=np.empty((B, H, T + 1, m, m)), U=np.empty((B, H, m, d + 1)), M=np.empty((B, H, m, d + 1)),
            Y=np.empty((B, H, n, d + 1)), vbar=np.empty((B, H, d)))
        ptrs = [inter[k] for k in ("Qt", "Kt", "W", "Xs", "U", "M", "Y", "vbar")]
    gw, r = _attention_grid(grid)
    rc = load().lapattn_oracle_forward(_p(Q), _p(K), _p(V), _p(out), B, H, n, d, int(m), float(lam),
                                       int(T), int(norm), float(eps), int(gw), int(r), *[_p(a) for a in ptrs],
                                       _p(_whiten(whiten, H, m)))
    if rc:
        raise ValueError("oracle forward rejected its arguments (code %d)" % rc)
    if dwc_branch is not None:
        if grid is None:
            raise ValueError("the convolution branch needs the token map (grid)")
        out = out + dwc(V, dwc_branch[0], dwc_branch[1], grid[0])
    return (out, inter) if intermediates else out


def backward(Q, K, V, dO, m, lam, T, norm=NORM_INLINE, eps=0.0, grid=None, dwc_branch=None, whiten=None):
    """(dQ, dK, dV), and with dwc_branch = (weight, bias) also (dweight, dbias)."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    B, H, n, d = Q.shape
    dQ, dK, dV = np.empty_like(Q), np.empty_like(Q), np.empty_like(Q)
    gw, r = _attention_grid(grid)
    rc = load().lapattn_oracle_backward(_p(Q), _p(K), _p(V), _p(dO), _p(dQ), _p(dK), _p(dV),
                                        B, H, n, d, int(m), float(lam), int(T), int(norm), float(eps),
                                        int(gw), int(r), _p(_whiten(whiten, H, m)))
    if rc:
        raise ValueError("oracle backward rejected its arguments (code %d)" % rc)
    if dwc_branch is None:
        return dQ, dK, dV
    if grid is None:
        raise ValueError("the convolution branch needs the token map (grid)")
    dVc, dW, db = dwc_backward(V, dwc_branch[0], dO, grid[0])
    return dQ, dK, dV + dVc, dW, db
