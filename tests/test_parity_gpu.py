"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Three metrics per head (b, h), maximum over heads:
  fro  ||O_gpu - O_ref||_F / ||O_ref||_F
  max  max |O_gpu - O_ref| / max |O_ref|
  row  max over rows i of ||o_i - r_i|| / max(||r_i||, ROW_FLOOR * rms_i ||r_i||)
The tolerance of the method applies to fro: 1e-4 for fp32 inputs, 2e-2 for bf16
inputs, on Out and on each of dQ, dK, dV.  fro alone moves by only about 1/sqrt(n)
when one whole row is wrong; max and row see a single bad element, row or tile (a
wrong row scores about 1).  Their bounds (BOUNDS) equal the tolerance except for
the rows of fp32 gradients: a gradient row is a sum over up to n keys of terms of
both signs (and under the landmark-space normalisation a difference of two
landmark sums), and its fp32 rounding error relative to the row's own norm
reaches ~5e-4 while fro stays <= 2e-5, so there row <= 1e-3.  A row whose
reference norm is below ROW_FLOOR times the head's rms row norm is measured
against that floor (its own norm says little about accuracy).  Where
the reference is NaN (a row whose kernel values all underflow under the row-sum
normalisation), the GPU value must be NaN too and is left out of the metrics.
Reduced sizes compare every output and span several tiles plus a ragged tail; the
full workload sizes run exactly the launch configuration the benchmark times and
compare a sample of heads, which the oracle computes independently (every head is
an independent problem).
"""
import math

import numpy as np
import pytest

import oracle
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# (fro, max, row) bounds by input dtype and output kind (module docstring)
BOUNDS = {("fp32", "out"): (1e-4, 1e-4, 1e-4), ("fp32", "grad"): (1e-4, 1e-4, 1e-3),
          ("bf16", "out"): (2e-2, 2e-2, 2e-2), ("bf16", "grad"): (2e-2, 2e-2, 2e-2)}
GRADS = ("dQ", "dK", "dV", "dfilters", "dbias")


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20368_amd import lapattn
    lapattn.library()
    return lapattn


def to_dev(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x)).to("cuda")
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def to_np(t):
    return t.float().cpu().numpy().astype(np.float64)


ROW_FLOOR = 0.1


def metrics(gpu, ref, ref_nan_any=False):
    """(fro, max, row) of the module docstring, each the maximum over heads; arrays are
    [B, H, n, d] or [BH, n, d].  NaN reference entries must be NaN on the GPU as well
    (AssertionError otherwise; with ref_nan_any the GPU may give a number there) and are
    left out."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rows, d = gpu.shape[-2], gpu.shape[-1]
    g = gpu.reshape(-1, rows, d).copy()
    r = ref.reshape(-1, rows, d).copy()
    nan = np.isnan(r)
    assert ref_nan_any or np.array_equal(np.isnan(g) & nan, nan), "reference NaN where the GPU gives a number"
    g[nan] = 0.0
    r[nan] = 0.0
    diff = g - r
    fro = np.linalg.norm(diff.reshape(len(g), -1), axis=1) / np.maximum(np.linalg.norm(r.reshape(len(r), -1), axis=1),
                                                                          1e-300)
    mx = np.abs(diff).reshape(len(g), -1).max(1) / np.maximum(np.abs(r).reshape(len(r), -1).max(1), 1e-300)
    rn = np.linalg.norm(r, axis=2)
    floor = ROW_FLOOR * np.sqrt((rn ** 2).mean(1, keepdims=True))
    row = (np.linalg.norm(diff, axis=2) / np.maximum(np.maximum(rn, floor), 1e-300)).max(1)
    return float(fro.max()), float(mx.max()), float(row.max())


def assert_parity(got, ref, dtype, what="out", ref_nan_any=False):
    """Checks the three metrics against BOUNDS[dtype, kind of `what`] and that the GPU gave no
    NaN or inf where the reference is finite; returns the metrics."""
    m3 = metrics(got, ref, ref_nan_any)
    bounds = BOUNDS[dtype, "grad" if what in GRADS else "out"]
    say("  %s: fro %.3e max %.3e row %.3e" % ((what,) + m3))
    fin = np.isfinite(np.asarray(ref, dtype=np.float64))
    assert np.isfinite(np.asarray(got, dtype=np.float64)[fin]).all(), "%s: non-finite GPU values" % what
    assert all(v <= b for v, b in zip(m3, bounds)), "%s: %s above %s" % (what, m3, bounds)
    return m3


def say(msg):
    print(msg, flush=True)


def dev_dwc(dwc):
    """(filters, bias) numpy -> fp32 device tensors."""
    if dwc is None:
        return None
    return tuple(None if a is None else torch.from_numpy(a).to("cuda") for a in dwc)


def dev_f32(a):
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def run_forward(L, x, w, norm=0, eps=0.0, grid=None, dwc=None, whiten=None):
    Q, K, V = (to_dev(x[k], w.dtype) for k in ("Q", "K", "V"))
    out = L.forward(Q, K, V, w.m, w.lam, w.T, norm=norm, eps=eps, grid=grid, dwc=dev_dwc(dwc), whiten=dev_f32(whiten))
    torch.cuda.synchronize()
    return to_np(out)


def check_forward(L, w, norm=0, eps=0.0, grid=None, dwc=None, whiten=None, x=None, ref_nan_any=False):
    """The forward on w's inputs (or on the given inputs x) against the oracle."""
    say("forward %s B=%d H=%d n=%d d=%d m=%d T=%d %s lambda=%g norm=%d eps=%g grid=%s dwc k=%s whiten=%s dist=%s%s" %
        (w.name, w.B, w.H, w.n, w.d, w.m, w.T, w.dtype, w.lam, norm, eps, grid,
         None if dwc is None else dwc[0].shape[-1], whiten is not None, w.dist, "" if x is None else " (given inputs)"))
    x = W.make_inputs(w, with_grad=False) if x is None else x
    got = run_forward(L, x, w, norm, eps, grid, dwc, whiten)
    ref = oracle.forward(x["Q"], x["K"], x["V"], w.m, w.lam, w.T, norm, eps, grid=grid, dwc_branch=dwc,
                         whiten=None if whiten is None else np.asarray(whiten, dtype=np.float32).astype(np.float64))
    return assert_parity(got, ref, w.dtype, ref_nan_any=ref_nan_any)


# ------------------------------------------------------------------------------ reduced sizes, every output

@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_forward_reduced(L, name):
    w = W.WORKLOADS[name]
    for n in (w.n, 1000):
        check_forward(L, W.small(w, n=n, B=1, H=3))


@pytest.mark.parametrize("norm", [0, 1, 2])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("d", [32, 64])
def test_forward_norms_dtypes(L, norm, dtype, d):
    w = W.Workload("mix", 2, 2, 777, d, 37, 5, dtype, 1 / math.sqrt(d), math.sqrt(d), 7, False)
    check_forward(L, w, norm=norm)


def test_forward_tiny_workload(L):
    check_forward(L, W.WORKLOADS["tiny"])


@pytest.mark.parametrize("nm", [16, 32, 64])
def test_forward_landmarks_equal_tokens(L, nm):
    """m = n: with enough updates the method is exact dense attention; the GPU
    must agree with the oracle at the same T (both converged)."""
    w = W.Workload("dense", 1, 2, nm, 32, nm, 50, "fp32", 1.0, math.sqrt(32), 11, False)
    check_forward(L, w)
    check_forward(L, w.with_(T=6))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("n,m", [(1, 1), (5, 1), (63, 7), (64, 64), (65, 64), (513, 1), (300, 33)])
def test_forward_edge_shapes(L, n, m, dtype):
    w = W.Workload("edge", 1, 2, n, 64, m, 4, dtype, 0.125, 8.0, 12, False)
    check_forward(L, w)
    check_forward(L, w.with_(d=32, sigma=1 / math.sqrt(32), lam=math.sqrt(32)), norm=1)


def test_forward_lambda4_and_eps(L):
    w = W.WORKLOADS["pvt_stage1"].with_(B=2, lam=4.0)
    check_forward(L, w)
    check_forward(L, W.WORKLOADS["deit_small"].with_(B=2), eps=0.05)


def test_forward_deterministic(L):
    w = W.small(W.WORKLOADS["highres"], n=4096, B=1, H=2)
    x = W.make_inputs(w, with_grad=False)
    a = run_forward(L, x, w)
    b = run_forward(L, x, w)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_reused_workspace(L, dtype):
    """One workspace and one output buffer, two different inputs in turn (then the first
    again): every call must see its own tables, never values left by the previous call."""
    w = W.small(W.WORKLOADS["highres"], n=2048, B=1, H=2).with_(dtype=dtype)
    xs = [W.make_inputs(w.with_(seed=s), with_grad=False) for s in (61, 62)]
    devs = [[to_dev(x[k], dtype) for k in ("Q", "K", "V")] for x in xs]
    out = torch.empty_like(devs[0][0])
    ws = L.workspace(devs[0][0], w.m, w.T)
    for i in (0, 1, 0):
        L.forward(*devs[i], w.m, w.lam, w.T, out=out, ws=ws)
        torch.cuda.synchronize()
        ref = oracle.forward(xs[i]["Q"], xs[i]["K"], xs[i]["V"], w.m, w.lam, w.T)
        say("reused workspace %s input %d" % (dtype, i))
        assert_parity(to_np(out), ref, dtype)


def test_forward_nan_propagates(L):
    w = W.Workload("nan", 1, 2, 300, 32, 10, 3, "fp32", 0.2, 4.0, 13, False)
    x = W.make_inputs(w, with_grad=False)
    x["Q"][0, 1, 17, 3] = np.nan
    got = run_forward(L, x, w)
    assert np.isnan(got[0, 1]).any()
    ref = oracle.forward(x["Q"][:, :1], x["K"][:, :1], x["V"][:, :1], w.m, w.lam, w.T)
    assert_parity(got[:, :1], ref, "fp32")


# ------------------------------------------------------------------------------ full workload sizes, sampled heads

@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_forward_full_size_sampled_heads(L, name):
    w = W.WORKLOADS[name]
    say("forward full %s" % name)
    x = W.make_inputs(w, with_grad=False)
    got = run_forward(L, x, w)
    BH = w.BH
    heads = sorted(set([0, BH - 1, BH // 2, (7 * BH) // 11]))
    sub = {k: np.ascontiguousarray(v.reshape(BH, w.n, w.d)[heads][None]) for k, v in x.items()}
    ref = oracle.forward(sub["Q"], sub["K"], sub["V"], w.m, w.lam, w.T)
    say("  heads %s" % heads)
    assert np.isfinite(got).all()
    assert_parity(got.reshape(BH, w.n, w.d)[heads][None], ref, w.dtype)


# ------------------------------------------------------------------------------ backward

def check_backward(L, w, norm=0, eps=0.0, heads=None, grid=None, dwc=None, whiten=None):
    say("backward %s B=%d H=%d n=%d d=%d m=%d T=%d %s norm=%d eps=%g grid=%s dwc k=%s whiten=%s" %
        (w.name, w.B, w.H, w.n, w.d, w.m, w.T, w.dtype, norm, eps, grid, None if dwc is None else dwc[0].shape[-1],
         whiten is not None))
    x = W.make_inputs(w, with_grad=True)
    Q, K, V, dO = (to_dev(x[k], w.dtype) for k in ("Q", "K", "V", "dO"))
    res = L.backward(Q, K, V, dO, w.m, w.lam, w.T, norm=norm, eps=eps, grid=grid, dwc=dev_dwc(dwc),
                     whiten=dev_f32(whiten))
    torch.cuda.synchronize()
    got = [to_np(t) for t in res[:3]]
    BH = w.BH
    if heads is None:
        sub, gsub = x, got
    else:
        sub = {k: np.ascontiguousarray(v.reshape(BH, w.n, w.d)[heads][None]) for k, v in x.items()}
        gsub = [g.reshape(BH, w.n, w.d)[heads][None] for g in got]
    wsub = None
    if whiten is not None:
        wf = np.asarray(whiten, dtype=np.float32).astype(np.float64)
        wsub = wf if heads is None else wf[[hh % w.H for hh in heads]]
    ref = oracle.backward(sub["Q"], sub["K"], sub["V"], sub["dO"], w.m, w.lam, w.T, norm, eps, grid=grid,
                          dwc_branch=dwc, whiten=wsub)
    for g in got:
        assert np.isfinite(g).all()
    for g, r, what in zip(gsub, ref[:3], ("dQ", "dK", "dV")):
        assert_parity(g, r, w.dtype, what)
    if dwc is not None:
        assert heads is None, "the filter gradients sum over every head of the batch"
        gw_, gb_ = (res[3].cpu().numpy().astype(np.float64), res[4].cpu().numpy().astype(np.float64))
        assert np.isfinite(gw_).all() and np.isfinite(gb_).all()
        # filter gradient: per head, one row of k * k taps per channel; bias: one row per head
        Hh, dd, kk = gw_.shape[0], gw_.shape[1], gw_.shape[-1]
        assert_parity(gw_.reshape(Hh, dd, kk * kk), ref[3].reshape(Hh, dd, kk * kk), w.dtype, "dfilters")
        assert_parity(gb_.reshape(1, Hh, dd), ref[4].reshape(1, Hh, dd), w.dtype, "dbias")


@pytest.mark.parametrize("norm", [0, 1, 2])
def test_backward_reduced(L, norm):
    w = W.small(W.WORKLOADS["train"], n=700, B=1, H=2)
    check_backward(L, w, norm=norm)


@pytest.mark.parametrize("d,m,n", [(64, 64, 500), (32, 20, 197), (64, 9, 64), (32, 1, 33)])
def test_backward_shapes(L, d, m, n):
    w = W.Workload("bshape", 1, 2, n, d, m, 4, "fp32", 1 / math.sqrt(d), math.sqrt(d), 14, True)
    check_backward(L, w)


@pytest.mark.parametrize("n,d", [(4096, 32), (16384, 64)])
def test_long_sequence_few_heads(L, n, d):
    """Batch 1, 2 heads, m = 64: the chunk lengths the library picks for a small grid at their
    limit of 64 partial sums per head -- 64-token landmark-major chunks at n = 4096 (256 at
    n = 16384) and 256-key blocks on the key side (16 and 64 partials)."""
    w = W.Workload("long", 1, 2, n, d, 64, 6, "fp32", 1 / math.sqrt(d), math.sqrt(d), 16, True)
    check_forward(L, w)
    check_backward(L, w)


@pytest.mark.parametrize("m", [16, 32, 64])
def test_sweep_shape_saved_path(L, m):
    """The kernel-timing sweep's longest shape (B=1, H=2, d=32, n=16384, fp32, lambda = sqrt(32),
    T = 6, the same seeds) on the path the sweep times -- forward and backward with save on one
    workspace -- against the oracle, output and gradients."""
    w = W.Workload("sweep", 1, 2, 16384, 32, m, 6, "fp32", 1 / math.sqrt(32), math.sqrt(32), 7 + 16384 + m, True)
    say("sweep shape n=%d m=%d, save path" % (w.n, m))
    x = W.make_inputs(w, with_grad=True)
    Q, K, V, dO = (to_dev(x[k], w.dtype) for k in ("Q", "K", "V", "dO"))
    ws = L.workspace(Q, m, w.T, True)
    out = L.forward(Q, K, V, m, w.lam, w.T, ws=ws, save=True)
    g = L.backward(Q, K, V, dO, m, w.lam, w.T, ws=ws, save=True)
    torch.cuda.synchronize()
    assert_parity(to_np(out), oracle.forward(x["Q"], x["K"], x["V"], m, w.lam, w.T), w.dtype)
    ref = oracle.backward(x["Q"], x["K"], x["V"], x["dO"], m, w.lam, w.T)
    for gg, r, what in zip(g[:3], ref[:3], ("dQ", "dK", "dV")):
        assert_parity(to_np(gg), r, w.dtype, what)


def test_backward_eps(L):
    w = W.Workload("beps", 1, 2, 300, 32, 16, 5, "fp32", 0.2, 4.0, 15, True)
    check_backward(L, w, eps=0.1)


def test_backward_full_size_sampled_heads(L):
    w = W.WORKLOADS["train"]
    check_backward(L, w, heads=[0, 37, 91, w.BH - 1])


def test_backward_deterministic(L):
    w = W.small(W.WORKLOADS["train"], n=1000, B=1, H=2)
    x = W.make_inputs(w, with_grad=True)
    Q, K, V, dO = (to_dev(x[k], w.dtype) for k in ("Q", "K", "V", "dO"))
    a = [to_np(t) for t in L.backward(Q, K, V, dO, w.m, w.lam, w.T)]
    b = [to_np(t) for t in L.backward(Q, K, V, dO, w.m, w.lam, w.T)]
    assert all(np.array_equal(p, q) for p, q in zip(a, b))


@pytest.mark.parametrize("norm", [0, 1, 2])
def test_backward_bf16(L, norm):
    """bf16 inputs: the fp32 backward on the widened values, gradients rounded to bf16."""
    w = W.small(W.WORKLOADS["train"], n=700, B=1, H=2).with_(dtype="bf16")
    check_backward(L, w, norm=norm)
    check_backward(L, w.with_(d=64, sigma=0.125, lam=8.0, n=333, m=37), norm=norm)


# ------------------------------------------------------------------------------ r x r window landmarks

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_window_landmarks(L, dtype):
    """Landmarks as 7 x 7 windows of a 56 x 56 token map (m = 64), as on the PVT stage-1 grid,
    and 4 x 4 windows of a 24 x 32 map (m = 48), every normalisation."""
    w = W.WORKLOADS["pvt_stage1"].with_(B=1, H=2, dtype=dtype)
    check_forward(L, w, grid=(56, 7))
    w2 = W.Workload("grid", 1, 2, 24 * 32, 32, 48, 6, dtype, 1 / math.sqrt(32), math.sqrt(32), 31, False)
    for norm in (0, 1, 2):
        check_forward(L, w2, norm=norm, grid=(32, 4))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_window_landmarks(L, dtype):
    w = W.Workload("gridb", 1, 2, 16 * 20, 32, 20, 5, dtype, 1 / math.sqrt(32), math.sqrt(32), 33, True)
    check_backward(L, w, grid=(20, 4))
    check_backward(L, w.with_(d=64, sigma=0.125, lam=8.0), norm=1, grid=(20, 4))
    check_backward(L, w.with_(n=15 * 15, m=25), grid=(15, 3))


# ------------------------------------------------------------------------------ convolution branch of Eq. (7)

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_convolution_branch(L, dtype):
    """Out = Z V + DWC(V): 3 x 3 filters with bias over a 24 x 32 map with window landmarks, 5 x 5
    without bias over the same map with segment landmarks, and 1 x 1 / 7 x 7 filters over a
    7 x 9 map (the 7 x 7 filter is wider than the map's height)."""
    w = W.Workload("conv", 1, 2, 24 * 32, 64, 48, 6, dtype, 0.125, 8.0, 41, False)
    check_forward(L, w, grid=(32, 4), dwc=W.make_dwc(2, 64, 3, seed=1))
    w2 = w.with_(d=32, sigma=1 / math.sqrt(32), lam=math.sqrt(32), m=20)
    check_forward(L, w2, norm=1, grid=(32, 0), dwc=W.make_dwc(2, 32, 5, seed=2, bias=False))
    w3 = W.Workload("conv3", 2, 1, 7 * 9, 64, 7, 4, dtype, 0.125, 8.0, 43, False)
    for k in (1, 7):
        check_forward(L, w3, norm=2, grid=(9, 0), dwc=W.make_dwc(1, 64, k, seed=3 + k))


def test_forward_convolution_branch_full_size(L):
    """The PVT stage-1 shape (B=32, n = 56 x 56, bf16) with 7 x 7 window landmarks and a 3 x 3
    branch; sampled heads (each head's output depends on that head only)."""
    w = W.WORKLOADS["pvt_stage1"]
    dwc = W.make_dwc(w.H, w.d, 3, seed=7)
    say("forward full %s with dwc" % w.name)
    x = W.make_inputs(w, with_grad=False)
    got = run_forward(L, x, w, grid=(56, 7), dwc=dwc)
    heads = [0, 13, w.BH - 1]
    sub = {k: np.ascontiguousarray(v.reshape(w.BH, w.n, w.d)[heads][None]) for k, v in x.items()}
    dsub = (dwc[0][[0]], dwc[1][[0]])   # H = 1: every sampled head uses filter set 0
    ref = oracle.forward(sub["Q"], sub["K"], sub["V"], w.m, w.lam, w.T, grid=(56, 7),
                         dwc_branch=(np.repeat(dsub[0], len(heads), 0), np.repeat(dsub[1], len(heads), 0)))
    say("  heads %s" % heads)
    assert_parity(got.reshape(w.BH, w.n, w.d)[heads][None], ref, w.dtype)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_convolution_branch(L, dtype):
    """dV gains DWC^T(dOut); the filter and bias gradients sum over a batch of two."""
    w = W.Workload("convb", 2, 2, 16 * 20, 32, 20, 5, dtype, 1 / math.sqrt(32), math.sqrt(32), 45, True)
    check_backward(L, w, grid=(20, 4), dwc=W.make_dwc(2, 32, 3, seed=5))
    check_backward(L, w.with_(d=64, sigma=0.125, lam=8.0), norm=1, grid=(20, 0),
                   dwc=W.make_dwc(2, 64, 5, seed=6, bias=False))
    check_backward(L, w.with_(n=6 * 8, m=6, B=1), norm=2, grid=(8, 0), dwc=W.make_dwc(2, 32, 7, seed=8))


# ------------------------------------------------------------------------------ landmark-space normalisation

MSPACE = 3


def rand_whiten(H, m, seed):
    return np.random.default_rng(seed).uniform(0.5, 1.5, size=(H, m)).astype(np.float32)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_mspace(L, dtype):
    """Appendix B's landmark-space embedding with a per-head diagonal whitening: every landmark
    tile of the n = 16384 shape with a ragged tail, an odd m, and the all-ones default."""
    w = W.small(W.WORKLOADS["highres"], n=3000, B=1, H=2).with_(dtype=dtype)
    check_forward(L, w, norm=MSPACE, whiten=rand_whiten(2, 64, 1))
    check_forward(L, w.with_(n=333, m=37), norm=MSPACE, whiten=rand_whiten(2, 37, 2))
    w2 = W.small(W.WORKLOADS["train"], n=700, B=2, H=2).with_(dtype=dtype, m=20)
    check_forward(L, w2, norm=MSPACE)
    check_forward(L, w2, norm=MSPACE, whiten=np.zeros((2, 20), np.float32))


def test_forward_mspace_full_size_sampled_heads(L):
    w = W.WORKLOADS["highres"]
    wh = rand_whiten(w.H, w.m, 3)
    say("forward full %s mspace" % w.name)
    x = W.make_inputs(w, with_grad=False)
    got = run_forward(L, x, w, norm=MSPACE, whiten=wh)
    heads = [0, 5, w.BH - 1]
    sub = {k: np.ascontiguousarray(v.reshape(w.BH, w.n, w.d)[heads][None]) for k, v in x.items()}
    ref = oracle.forward(sub["Q"], sub["K"], sub["V"], w.m, w.lam, w.T, MSPACE,
                         whiten=wh.astype(np.float64)[[hh % w.H for hh in heads]])
    say("  heads %s" % heads)
    assert_parity(got.reshape(w.BH, w.n, w.d)[heads][None], ref, w.dtype)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_mspace(L, dtype):
    w = W.small(W.WORKLOADS["train"], n=700, B=1, H=2).with_(dtype=dtype)
    check_backward(L, w, norm=MSPACE, whiten=rand_whiten(2, 64, 4))
    check_backward(L, w.with_(d=64, sigma=0.125, lam=8.0, n=333, m=37, B=2), norm=MSPACE, whiten=rand_whiten(2, 37, 5))
    check_backward(L, w.with_(m=9, n=64), norm=MSPACE)


def test_backward_mspace_full_size_sampled_heads(L):
    w = W.WORKLOADS["train"]
    check_backward(L, w, norm=MSPACE, heads=[0, 37, w.BH - 1], whiten=rand_whiten(w.H, w.m, 6))


# ------------------------------------------------------------------------------ saved forward state

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_reuses_saved_forward_state(L, dtype):
    """forward(save) then backward(save) on one workspace equals, bit for bit, the calls that
    recompute (the backward skips pool, key-side summary and solve for fp32 inputs; bf16 ignores
    save), for the inline and landmark-space forms and with the convolution branch."""
    w = W.small(W.WORKLOADS["train"], n=56 * 14, B=2, H=2).with_(dtype=dtype)
    x = W.make_inputs(w, with_grad=True)
    Q, K, V, dO = (to_dev(x[k], w.dtype) for k in ("Q", "K", "V", "dO"))
    for kw in (dict(), dict(norm=MSPACE, whiten=dev_f32(rand_whiten(2, w.m, 9))),
               dict(grid=(56, 0), dwc=dev_dwc(W.make_dwc(2, w.d, 3, seed=10)))):
        say("saved state %s %s" % (dtype, sorted(kw)))
        ws = L.workspace(Q, w.m, w.T, True, "dwc" in kw)
        out_s = L.forward(Q, K, V, w.m, w.lam, w.T, ws=ws, save=True, **kw)
        g_s = L.backward(Q, K, V, dO, w.m, w.lam, w.T, ws=ws, save=True, **kw)
        out_r = L.forward(Q, K, V, w.m, w.lam, w.T, **kw)
        g_r = L.backward(Q, K, V, dO, w.m, w.lam, w.T, **kw)
        torch.cuda.synchronize()
        assert torch.equal(out_s, out_r)
        assert all(torch.equal(a, b) for a, b in zip(g_s, g_r))


# ------------------------------------------------------------------------------ options together

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_all_options_together(L, dtype):
    """Window landmarks, the landmark-space normalisation with a whitening, eps > 0, lambda = 4 and
    a 5 x 5 convolution branch at once, forward and backward, against the oracle."""
    w = W.Workload("combo", 2, 2, 24 * 20, 32, 30, 5, dtype, 1 / math.sqrt(32), 4.0, 47, True)
    grid = (20, 4)   # 24 x 20 map, 4 x 4 windows: 6 x 5 = 30 landmarks
    dwc = W.make_dwc(2, 32, 5, seed=12)
    wh = rand_whiten(2, 30, 13)
    check_forward(L, w, norm=MSPACE, eps=0.05, grid=grid, dwc=dwc, whiten=wh)
    check_backward(L, w, norm=MSPACE, eps=0.05, grid=grid, dwc=dwc, whiten=wh)


# ------------------------------------------------------------------------------ edge cases of the method

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("T", [0, 1])
def test_forward_few_ns_updates(L, dtype, T):
    """T = 0 (Algorithm 2's start X_0 = W^T / (||W||_1 ||W||_inf) alone, R9) and T = 1, with and
    without the row-sum normalisation, a ragged n, an odd m and m = 64."""
    for d in (32, 64):
        w = W.Workload("fewT", 1, 2, 777, d, 37, T, dtype, 1 / math.sqrt(d), math.sqrt(d), 17, False)
        for norm in (0, 1):
            check_forward(L, w, norm=norm)
        check_forward(L, w.with_(n=1000, m=64))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_forward_kernel_underflow(L, dtype):
    """lambda = 1e-6: every kernel value underflows, in fp64 as well, so ||W||_1 ||W||_inf = 0 and
    X = 0 (R10).  The inline form then gives v-bar in every row and the plain form exactly 0."""
    w = W.Workload("underflow", 1, 2, 777, 64, 37, 6, dtype, 0.125, 1e-6, 18, False)
    check_forward(L, w, norm=0)
    x = W.make_inputs(w, with_grad=False)
    got = run_forward(L, x, w, norm=2)
    assert not np.any(got), "the plain form must be exactly zero when every kernel value underflows"


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_forward_large_lambda(L, dtype):
    """lambda = 1e8: every kernel value rounds to 1 (fp64 keeps 1 - 1e-8 * distance), W is the
    all-ones matrix, Algorithm 2 stays at its pseudoinverse and every row is about v-bar, the
    lambda -> infinity limit.  The inline output v-bar + sum_j g_ij (v_j - v-bar) has magnitude
    |v-bar| ~ sigma / sqrt(n), while each kernel value carries its own rounding: its relative
    error grows like eps * n, which for fp32 kernel values (eps = 6e-8) reaches the 1e-4 bar
    near n = 800.  The fp32 inline case therefore runs at n = 300 (ragged against both the
    64-token tiles and the 37 segments); the row sums (Y / s, well conditioned) and bf16 run
    at n = 777."""
    w = W.Workload("flat", 1, 2, 777, 64, 37, 6, dtype, 0.125, 1e8, 19, False)
    check_forward(L, w if dtype == "bf16" else w.with_(n=300), norm=0)
    check_forward(L, w, norm=1)


# ------------------------------------------------------------------------------ input distributions (bf16 frame)

@pytest.mark.parametrize("norm", [0, 1])
def test_forward_bf16_heavy_tailed(L, norm):
    """Q and K drawn from Student-t with 3 degrees of freedom: a head's largest |x| lies tens of
    standard deviations out, which sets the range of the fixed-point distance frame."""
    w = W.Workload("t3", 1, 2, 3000, 64, 64, 8, "bf16", 0.125, 8.0, 20, False, dist="t3")
    check_forward(L, w, norm=norm)
    check_forward(L, w.with_(d=32, sigma=1 / math.sqrt(32), lam=math.sqrt(32), m=37, n=777, seed=24), norm=norm)


@pytest.mark.parametrize("m", [32, 64])
def test_forward_bf16_nonfinite_inputs(L, m):
    """A NaN or an infinity in V, or a NaN in Q, of head 1 makes every output of head 1 NaN under
    each normalisation (for m > 48 the value statistics come from the key side, m <= 48 from the
    pooling), and head 0 keeps its parity."""
    w = W.Workload("nonfinite", 1, 2, 1000, 64, m, 6, "bf16", 0.125, 8.0, 27, False)
    for where, val in (("V", np.nan), ("V", np.inf), ("V", -np.inf), ("Q", np.nan)):
        x = W.make_inputs(w, with_grad=False)
        x[where][0, 1, 500, 7] = val
        for norm in (0, 1, 2, 3):
            say("non-finite %s = %s, m = %d, norm %d" % (where, val, m, norm))
            got = run_forward(L, x, w, norm=norm)
            assert np.isnan(got[0, 1]).all(), "head 1 must be NaN everywhere"
            ref = oracle.forward(x["Q"][:, :1], x["K"][:, :1], x["V"][:, :1], w.m, w.lam, w.T, norm)
            assert_parity(got[:, :1], ref, "bf16")


@pytest.mark.parametrize("norm", [0, 1])
def test_forward_bf16_outlier_tokens(L, norm):
    """One query row and one key row of head 0 and one value row of head 1 scaled by 2^10 (exact
    in bf16), then milder ones (2^5), whose kernel values (~1e-11) lie below fp16's range.  The
    far query's inline output is v-bar; under the row-sum normalisation it is the weighted mean
    of the values, which needs its kernel values relative to the row's largest."""
    w = W.Workload("outlier", 1, 2, 3000, 64, 64, 8, "bf16", 0.125, 8.0, 21, False)
    x = W.make_inputs(w, with_grad=False)
    x["Q"][0, 0, 1234] *= 1024.0
    x["K"][0, 0, 777] *= 1024.0
    x["V"][0, 1, 55] *= 1024.0
    # row sums: the far query's kernel values (~e^-800) underflow in fp64, so its reference row
    # is 0/0; the GPU forms them relative to its row's bound and returns the weighted mean
    check_forward(L, w, norm=norm, x=x, ref_nan_any=True)
    # a milder outlier (x 2^5) keeps every kernel value finite
    x = W.make_inputs(w.with_(seed=25), with_grad=False)
    x["Q"][0, 0, 2999] *= 32.0
    x["K"][0, 1, 0] *= 32.0
    check_forward(L, w, norm=norm, x=x)


@pytest.mark.parametrize("norm", [0, 1])
def test_forward_bf16_input_scales(L, norm):
    """Unit-variance Q, K, V (distances eight times the usual ones, kernel values down to about
    1e-4), and values of magnitude ~1e-6 (below fp16's normal range without a prescale)."""
    w = W.Workload("scale", 1, 2, 3000, 64, 64, 8, "bf16", 1.0, 8.0, 22, False)
    check_forward(L, w, norm=norm)
    w2 = w.with_(sigma=0.125, seed=23)
    x = W.make_inputs(w2, with_grad=False)
    x["V"] = W.round_bf16(x["V"] * 1e-5)
    check_forward(L, w2, norm=norm, x=x)


# ------------------------------------------------------------------------------ saved state at more shapes

@pytest.mark.parametrize("d,m", [(64, 17), (64, 33), (32, 37), (64, 37)])
def test_backward_saved_state_shapes(L, d, m):
    """forward(save) + backward(save) equal the recomputing calls bit for bit at d = 64, odd m and
    m in one 32-wide range or past it, for the inline and row-sum forms; window landmarks too."""
    w = W.Workload("saved", 2, 2, 700, d, m, 5, "fp32", 1 / math.sqrt(d), math.sqrt(d), 26, True)
    cases = [(w, dict()), (w, dict(norm=1))]
    if m == 37:   # 4 x 4 windows of a 24 x 20 map: 30 landmarks
        cases.append((w.with_(n=24 * 20, m=30), dict(grid=(20, 4))))
    for wc, kw in cases:
        say("saved state d=%d m=%d n=%d %s" % (wc.d, wc.m, wc.n, sorted(kw.items())))
        x = W.make_inputs(wc, with_grad=True)
        Q, K, V, dO = (to_dev(x[k], wc.dtype) for k in ("Q", "K", "V", "dO"))
        ws = L.workspace(Q, wc.m, wc.T, True)
        out_s = L.forward(Q, K, V, wc.m, wc.lam, wc.T, ws=ws, save=True, **kw)
        g_s = L.backward(Q, K, V, dO, wc.m, wc.lam, wc.T, ws=ws, save=True, **kw)
        out_r = L.forward(Q, K, V, wc.m, wc.lam, wc.T, **kw)
        g_r = L.backward(Q, K, V, dO, wc.m, wc.lam, wc.T, **kw)
        torch.cuda.synchronize()
        assert torch.equal(out_s, out_r)
        assert all(torch.equal(a, b) for a, b in zip(g_s, g_r))


# ------------------------------------------------------------------------------ m up to 128 (64 < m: the
# landmark groups of 64, the Newton-Schulz solve and its backward over many workgroups)

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("d,m,n", [(32, 96, 1000), (64, 128, 1111), (64, 65, 300), (32, 128, 128), (64, 100, 777)])
def test_forward_many_landmarks(L, dtype, d, m, n):
    """m past one group of 64 landmarks, each normalisation, ragged n, m = n at 128."""
    w = W.Workload("bigm", 1, 2, n, d, m, 6, dtype, 1 / math.sqrt(d), math.sqrt(d), 41, False)
    for norm in (0, 1, 2):
        check_forward(L, w, norm=norm)
    check_forward(L, w, norm=MSPACE, whiten=rand_whiten(2, m, 7))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_forward_many_landmarks_windows_and_options(L, dtype):
    """4 x 4 windows of a 32 x 64 token map (m = 128) with eps and the convolution branch;
    Algorithm 2's X0 alone (T = 0), one update, and a kernel that underflows (the c = 0 guard)."""
    w = W.Workload("bigw", 1, 2, 32 * 64, 64, 128, 8, dtype, 1 / 8, 8.0, 43, False)
    check_forward(L, w, grid=(64, 4))
    check_forward(L, w, norm=1, eps=0.05, grid=(64, 4), dwc=W.make_dwc(2, 64, 3, seed=44))
    for T in (0, 1):
        check_forward(L, w.with_(T=T, n=500, m=120))
    check_forward(L, w.with_(n=300, m=99, lam=1e-6))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("d,m,n", [(32, 96, 700), (64, 128, 600), (64, 73, 333)])
def test_backward_many_landmarks(L, dtype, d, m, n):
    """Gradients at m past 64: each normalisation, eps, the landmark-space form."""
    w = W.Workload("bigmb", 1, 2, n, d, m, 5, dtype, 1 / math.sqrt(d), math.sqrt(d), 45, True)
    for norm in (0, 1, 2):
        check_backward(L, w, norm=norm)
    check_backward(L, w, eps=0.1)
    check_backward(L, w, norm=MSPACE, whiten=rand_whiten(2, m, 46))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_many_landmarks_windows(L, dtype):
    """4 x 4 windows of a 32 x 64 map (m = 128), with the convolution branch; T = 0 and T = 1."""
    w = W.Workload("bigwb", 1, 2, 32 * 64, 32, 128, 4, dtype, 1 / math.sqrt(32), math.sqrt(32), 47, True)
    check_backward(L, w, grid=(64, 4))
    check_backward(L, w, norm=1, grid=(64, 4), dwc=W.make_dwc(2, 32, 3, seed=48))
    for T in (0, 1):
        check_backward(L, w.with_(T=T, n=400, m=110))


@pytest.mark.parametrize("d,m", [(32, 96), (64, 128), (64, 81)])
def test_backward_saved_state_many_landmarks(L, d, m):
    """forward(save) + backward(save) equal the recomputing calls bit for bit past 64 landmarks
    (the saved rows of A and B in groups of 64), inline and row-sum forms; windows too."""
    w = W.Workload("savedbig", 2, 2, 700, d, m, 5, "fp32", 1 / math.sqrt(d), math.sqrt(d), 49, True)
    cases = [(w, dict()), (w, dict(norm=1))]
    if m == 128:
        cases.append((w.with_(n=32 * 64), dict(grid=(64, 4))))
    for wc, kw in cases:
        say("saved state d=%d m=%d n=%d %s" % (wc.d, wc.m, wc.n, sorted(kw.items())))
        x = W.make_inputs(wc, with_grad=True)
        Q, K, V, dO = (to_dev(x[k], wc.dtype) for k in ("Q", "K", "V", "dO"))
        ws = L.workspace(Q, wc.m, wc.T, True)
        out_s = L.forward(Q, K, V, wc.m, wc.lam, wc.T, ws=ws, save=True, **kw)
        g_s = L.backward(Q, K, V, dO, wc.m, wc.lam, wc.T, ws=ws, save=True, **kw)
        out_r = L.forward(Q, K, V, wc.m, wc.lam, wc.T, **kw)
        g_r = L.backward(Q, K, V, dO, wc.m, wc.lam, wc.T, **kw)
        torch.cuda.synchronize()
        assert torch.equal(out_s, out_r)
        assert all(torch.equal(a, b) for a, b in zip(g_s, g_r))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_many_landmarks_full_size_sampled_heads(L, dtype):
    """The n = 16384 workload (B=8, H=2, d=64) with m = 128 landmarks, as bench.py times it:
    every output checked finite, four sampled heads against the oracle."""
    w = W.WORKLOADS["highres"].with_(name="highres_m128", m=128, dtype=dtype)
    say("forward full %s %s" % (w.name, dtype))
    x = W.make_inputs(w, with_grad=False)
    got = run_forward(L, x, w)
    BH = w.BH
    heads = sorted(set([0, BH - 1, BH // 2, (7 * BH) // 11]))
    sub = {k: np.ascontiguousarray(v.reshape(BH, w.n, w.d)[heads][None]) for k, v in x.items()}
    ref = oracle.forward(sub["Q"], sub["K"], sub["V"], w.m, w.lam, w.T)
    say("  heads %s" % heads)
    assert np.isfinite(got).all()
    assert_parity(got.reshape(BH, w.n, w.d)[heads][None], ref, w.dtype)


# ------------------------------------------------------------------------------ small heads: the one-launch forward
# fp32 heads with n <= 256, m <= 32 and d in {32, 64} (the DeiT-small shape: 197 tokens, 32
# landmarks) run pooling, K_LL, Algorithm 2, the key side and the query side in one workgroup
# per head.  These cases pin that path against the oracle across its limits.

def launch_names(L, fn):
    """Names of the library launches made by fn() (the library's own launch recorder)."""
    L.lapattn_timing_enable(1)
    try:
        fn()
        torch.cuda.synchronize()
    finally:
        L.lapattn_timing_enable(0)
    return [k for k, _ in L.lapattn_timing_read(cap=256)]


def test_small_forward_is_one_launch(L):
    """The small-head shapes take the one-launch path; one token more, a bf16 input, m past 32
    or the saved-state forward take the others."""
    def names(w, **kw):
        x = W.make_inputs(w, with_grad=False)
        return launch_names(L, lambda: run_forward(L, x, w, **kw))
    w = W.WORKLOADS["deit_small"].with_(B=1, H=2)
    assert names(w) == ["small_forward"]
    assert names(w.with_(n=256, d=32)) == ["small_forward"]
    for other in (w.with_(n=257), w.with_(m=33), w.with_(dtype="bf16")):
        assert "small_forward" not in names(other), other


@pytest.mark.parametrize("d", [32, 64])
@pytest.mark.parametrize("norm", [0, 1, 2])
@pytest.mark.parametrize("n,m", [(1, 1), (2, 2), (31, 7), (64, 17), (197, 32), (256, 32), (256, 1), (32, 32),
                                 (100, 31)])
def test_small_forward_shapes(L, d, norm, n, m):
    """Every normalisation at d = 32 and 64: one token, n = m, a ragged n against the 64-key
    waves, an odd m, m = 1 and m = 32, n = 256 (every thread a live token)."""
    w = W.Workload("small", 2, 3, n, d, m, 6, "fp32", 1 / math.sqrt(d), math.sqrt(d), 51, False)
    check_forward(L, w, norm=norm)


@pytest.mark.parametrize("T", [0, 1, 12])
def test_small_forward_ns_updates(L, T):
    """Algorithm 2's X_0 alone (T = 0), one update and many (the iterate has converged)."""
    for d in (32, 64):
        w = W.Workload("smallT", 1, 2, 197, d, 29, T, "fp32", 1 / math.sqrt(d), math.sqrt(d), 52, False)
        for norm in (0, 1):
            check_forward(L, w, norm=norm)


def test_small_forward_windows_eps_lambda(L):
    """4 x 4 windows of a 16 x 16 map (m = 16) and of a 12 x 16 map (m = 12), eps on the
    diagonal, lambda = 4 and a heavy-tailed input."""
    w = W.Workload("smallw", 1, 2, 256, 64, 16, 6, "fp32", 0.125, 8.0, 53, False)
    for norm in (0, 1, 2):
        check_forward(L, w, norm=norm, grid=(16, 4))
    check_forward(L, w.with_(n=192, m=12, d=32), norm=1, grid=(16, 4))
    check_forward(L, w.with_(m=30, n=200), eps=0.05)
    check_forward(L, w.with_(m=30, n=200, lam=4.0, dist="t3"))


def test_small_forward_degenerate_kernels(L):
    """lambda = 1e-6 (every kernel value underflows: X = 0, the inline form gives v-bar, the
    plain form 0), lambda = 1e8 (every kernel value rounds to 1) and a NaN query entry (its head's
    output NaN, the other head untouched)."""
    w = W.Workload("smallu", 1, 2, 197, 64, 32, 6, "fp32", 0.125, 1e-6, 54, False)
    check_forward(L, w, norm=0)
    x = W.make_inputs(w, with_grad=False)
    assert not np.any(run_forward(L, x, w, norm=2))
    check_forward(L, w.with_(lam=1e8), norm=0)
    check_forward(L, w.with_(lam=1e8), norm=1)
    w = w.with_(lam=8.0)
    x = W.make_inputs(w, with_grad=False)
    x["Q"][0, 1, 17, 3] = np.nan
    got = run_forward(L, x, w)
    assert np.isnan(got[0, 1]).any()
    ref = oracle.forward(x["Q"][:, :1], x["K"][:, :1], x["V"][:, :1], w.m, w.lam, w.T)
    assert_parity(got[:, :1], ref, "fp32")
