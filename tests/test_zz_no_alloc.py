"""lapattn_forward_noalloc, the forward on the library's static scratch array, against
lapattn_forward on a caller-allocated workspace, both called through the C ABI.

The two run the same kernels on the same workspace layout, so the outputs must be equal bit
for bit.  Two calls in a row, the second on a smaller input than the first: the shared array
still holds the first call's contents when the second starts, which must not leak into it.
The second case is also checked against the fp64 oracle."""
import math

import numpy as np
import pytest

import oracle
import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2604_20368_amd import lapattn
    lapattn.library()
    return lapattn


def run_both(L, w, norm):
    print("noalloc %s B=%d H=%d n=%d d=%d m=%d T=%d %s norm=%d" % (w.name, w.B, w.H, w.n, w.d, w.m, w.T, w.dtype,
                                                                   norm), flush=True)
    x = W.make_inputs(w, with_grad=False)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Q, K, V = (torch.from_numpy(x[k]).to("cuda").to(dt) for k in ("Q", "K", "V"))
    code = L.LAPATTN_BF16 if w.dtype == "bf16" else L.LAPATTN_FP32
    ws = L.workspace(Q, w.m, w.T)
    ref = torch.empty_like(Q)
    got = torch.full_like(Q, float("nan"))
    st = torch.cuda.current_stream().cuda_stream
    rc = L.lapattn_forward(Q.data_ptr(), K.data_ptr(), V.data_ptr(), ref.data_ptr(), w.B, w.H, w.n, w.d, w.m, w.lam,
                           w.T, code, norm, 0.0, ws.data_ptr(), ws.numel(), st)
    assert rc == L.LAPATTN_OK, L.lapattn_status_str(rc)
    rc = L.lapattn_forward_noalloc(Q.data_ptr(), K.data_ptr(), V.data_ptr(), got.data_ptr(), w.B, w.H, w.n, w.d,
                                   w.m, w.lam, w.T, code, norm, 0.0, st)
    assert rc == L.LAPATTN_OK, L.lapattn_status_str(rc)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    return x, got


def test_noalloc_equals_forward_on_two_calls(L):
    # first the n = 16384 workload the benchmark times (bf16, 10 MiB of workspace) ...
    run_both(L, W.WORKLOADS["highres"], 0)
    # ... then a smaller fp32 problem with the row-sum normalisation on the same array
    w = W.Workload("noalloc_small", 1, 2, 3000, 32, 37, 6, "fp32", 1 / math.sqrt(32), math.sqrt(32), 51, False)
    x, got = run_both(L, w, 1)
    ref = oracle.forward(x["Q"], x["K"], x["V"], w.m, w.lam, w.T, 1)
    g = got.double().cpu().numpy().reshape(w.B * w.H, -1)
    r = ref.reshape(w.B * w.H, -1)
    err = float((np.linalg.norm(g - r, axis=1) / np.linalg.norm(r, axis=1)).max())
    print("  noalloc fp32 against the oracle: %.3e" % err, flush=True)
    assert err <= 1e-4


def test_noalloc_rejects_oversize_without_launching(L):
    """A call beyond the 32 MiB array returns LAPATTN_ERR_SCRATCH and leaves the output alone."""
    w = W.WORKLOADS["highres"]
    Q = torch.zeros((16, w.H, w.n, w.d), dtype=torch.float32, device="cuda")
    out = torch.full_like(Q, 7.0)
    rc = L.lapattn_forward_noalloc(Q.data_ptr(), Q.data_ptr(), Q.data_ptr(), out.data_ptr(), 16, w.H, w.n, w.d, w.m,
                                   w.lam, w.T, L.LAPATTN_FP32, 0, 0.0, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == L.LAPATTN_ERR_SCRATCH
    assert bool((out == 7.0).all())
