"""HIP graph capture of the C-ABI calls.

The library enqueues only kernel launches on the caller's stream (no memsets, no
allocations, no host synchronisation), so a forward or a backward can be captured into a
graph and replayed.  Each replay follows new inputs copied into the captured buffers, with
eager work and a synchronisation in between, and must equal, bit for bit, an eager call on
the same inputs with its own output and workspace buffers.
"""
import pytest

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


def to_dev(x, dtype):
    t = torch.from_numpy(x).to("cuda")
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def replay_case(L, w, backward, **kw):
    print("graph %s B=%d H=%d n=%d d=%d m=%d %s backward=%s" % (w.name, w.B, w.H, w.n, w.d, w.m, w.dtype, backward),
          flush=True)
    names = ("Q", "K", "V", "dO") if backward else ("Q", "K", "V")
    x = W.make_inputs(w, with_grad=backward)
    bufs = [to_dev(x[k], w.dtype) for k in names]
    ws = L.workspace(bufs[0], w.m, w.T, backward, "dwc" in kw)
    outs = [torch.empty_like(bufs[0]) for _ in range(3 if backward else 1)]

    def run():
        if backward:
            L.backward(*bufs, w.m, w.lam, w.T, grads=outs, ws=ws, **kw)
        else:
            L.forward(*bufs, w.m, w.lam, w.T, out=outs[0], ws=ws, **kw)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for r in range(3):
        xr = W.make_inputs(w.with_(seed=w.seed + 1 + r), with_grad=backward)
        for b, k in zip(bufs, names):
            b.copy_(to_dev(xr[k], w.dtype))
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = [o.clone() for o in outs]
        if backward:
            ref = L.backward(*bufs, w.m, w.lam, w.T, **kw)
        else:
            ref = (L.forward(*bufs, w.m, w.lam, w.T, **kw),)
        torch.cuda.synchronize()
        same = [torch.equal(a, b) for a, b in zip(got, ref)]
        print("  replay %d bitwise equal to eager: %s" % (r, same), flush=True)
        assert all(same)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_graph_replay(L, dtype):
    replay_case(L, W.small(W.WORKLOADS["highres"], n=3000, B=1, H=2).with_(dtype=dtype), backward=False)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_backward_graph_replay(L, dtype):
    replay_case(L, W.small(W.WORKLOADS["train"], n=900, B=1, H=2).with_(dtype=dtype), backward=True)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_forward_graph_replay_with_options(L, dtype):
    """The convolution branch and the landmark-space normalisation under capture."""
    import numpy as np
    w = W.small(W.WORKLOADS["train"], n=24 * 20, B=1, H=2).with_(dtype=dtype, m=30)
    fw, fb = W.make_dwc(2, w.d, 3, seed=21)
    wh = np.random.default_rng(22).uniform(0.5, 1.5, size=(2, 30)).astype(np.float32)
    dev = lambda a: torch.from_numpy(a).to("cuda")
    replay_case(L, w, backward=False, norm=3, grid=(20, 4), dwc=(dev(fw), dev(fb)), whiten=dev(wh))
