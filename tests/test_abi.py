"""The C ABI on the host (no GPU needed): the library loads, exports every entry
point the header declares, and rejects bad arguments before touching the device.
Invalid calls only: a rejected call returns before any HIP call."""
import os
import re

import pytest

from paper_2604_20368_amd import lapattn as L

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "lapattn.h")

FAKE = 0x1000   # non-null address that is never dereferenced: every call below is rejected first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lapattn_\w+)\s*\(", text)))


def test_library_exports_every_declared_function():
    lib = L.library()
    names = declared_functions()
    assert set(names) == set(L.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    for code in range(9):
        assert L.lapattn_status_str(code) and L.lapattn_status_str(code) != "unknown status"
    assert L.lapattn_status_str(99) == "unknown status"


def fwd(**kw):
    args = dict(Q=FAKE, K=FAKE, V=FAKE, Out=FAKE, B=1, H=2, n=100, d=32, m=8, lam=1.0, ns_iters=4, dtype=0,
                norm=0, eps=0.0, workspace=FAKE, workspace_bytes=0)
    args.update(kw)
    return L.lapattn_forward(**args)


def bwd(**kw):
    args = dict(Q=FAKE, K=FAKE, V=FAKE, dO=FAKE, dQ=FAKE, dK=FAKE, dV=FAKE, B=1, H=2, n=100, d=32, m=8, lam=1.0,
                ns_iters=4, dtype=0, norm=0, eps=0.0, workspace=FAKE, workspace_bytes=0)
    args.update(kw)
    return L.lapattn_backward(**args)


@pytest.mark.parametrize("call", [fwd, bwd])
def test_argument_validation(call):
    ptrs = ["Q", "K", "V"] + (["Out"] if call is fwd else ["dO", "dQ", "dK", "dV"])
    for p in ptrs:
        assert call(**{p: 0}) == L.LAPATTN_ERR_NULL
    assert call(B=0) == L.LAPATTN_ERR_SHAPE
    assert call(H=0) == L.LAPATTN_ERR_SHAPE
    assert call(n=0) == L.LAPATTN_ERR_SHAPE
    assert call(m=0) == L.LAPATTN_ERR_SHAPE
    assert call(m=101) == L.LAPATTN_ERR_SHAPE                     # m > n
    assert call(B=1 << 12, H=1 << 10, n=1 << 10, d=32) == L.LAPATTN_ERR_SHAPE   # B*H*n*d >= 2^31
    for p in ptrs:
        assert call(**{p: FAKE + 8}) == L.LAPATTN_ERR_ALIGN       # 16-byte vectors
    assert call(workspace=FAKE + 16) == L.LAPATTN_ERR_ALIGN      # 256-byte slices
    assert call(lam=0.0) == L.LAPATTN_ERR_PARAM
    assert call(lam=-1.0) == L.LAPATTN_ERR_PARAM
    assert call(lam=float("inf")) == L.LAPATTN_ERR_PARAM
    assert call(lam=float("nan")) == L.LAPATTN_ERR_PARAM
    assert call(ns_iters=-1) == L.LAPATTN_ERR_PARAM
    assert call(ns_iters=65) == L.LAPATTN_ERR_PARAM
    assert call(dtype=2) == L.LAPATTN_ERR_PARAM
    assert call(norm=4) == L.LAPATTN_ERR_PARAM
    assert call(eps=-0.1) == L.LAPATTN_ERR_PARAM
    assert call(eps=float("nan")) == L.LAPATTN_ERR_PARAM
    assert call(d=48) == L.LAPATTN_ERR_UNSUPPORTED
    assert call(n=200, m=129) == L.LAPATTN_ERR_UNSUPPORTED      # m up to 128
    assert call(n=200, m=128, workspace_bytes=0) == L.LAPATTN_ERR_WORKSPACE   # a valid m > 64
    assert call(workspace_bytes=0) == L.LAPATTN_ERR_WORKSPACE    # valid sizes, workspace too small
    need = L.lapattn_workspace_size(1, 2, 100, 32, 8, 4, 0, call is bwd)
    assert call(workspace_bytes=need - 1) == L.LAPATTN_ERR_WORKSPACE
    assert call(workspace=0, workspace_bytes=need) == L.LAPATTN_ERR_WORKSPACE


def test_backward_bf16_workspace():
    """The bf16 backward runs the fp32 backward on widened copies of its four inputs and
    rounds the three fp32 gradients: its workspace holds seven more B*H*n*d fp32 arrays, and a
    call given only the fp32 amount is rejected before any launch."""
    f32 = L.lapattn_workspace_size(1, 2, 100, 32, 8, 4, 0, 1)
    b16 = L.lapattn_workspace_size(1, 2, 100, 32, 8, 4, 1, 1)
    assert b16 >= f32 + 7 * (2 * 100 * 32 * 4)
    assert bwd(dtype=1, workspace_bytes=f32) == L.LAPATTN_ERR_WORKSPACE


def test_workspace_size_monotone_and_invalid():
    for bwd_flag in (0, 1):
        sizes = [L.lapattn_workspace_size(2, 2, n, 64, 64, 8, 0, bwd_flag) for n in (64, 197, 512, 3136, 16384)]
        assert all(b >= a > 0 for a, b in zip(sizes, sizes[1:])) and sizes[-1] > sizes[0]
        prev = 0
        for BH in (1, 2, 16, 384):
            s = L.lapattn_workspace_size(BH, 1, 3136, 32, 64, 6, 0, bwd_flag)
            assert s > prev
            prev = s
    assert L.lapattn_workspace_size(1, 1, 10, 32, 11, 4, 0, 0) == 0      # m > n
    assert L.lapattn_workspace_size(1, 1, 10, 40, 4, 4, 0, 0) == 0       # d unsupported
    # the forward workspace is O(n) in the sequence length: no n x m or n x n buffer
    a = L.lapattn_workspace_size(8, 2, 16384, 64, 64, 8, 1, 0)
    b = L.lapattn_workspace_size(8, 2, 4 * 16384, 64, 64, 8, 1, 0)
    assert b < 4.2 * a
    assert a < 16 * 16384 * 64 * 4    # well under one fp32 n x m matrix per head


@pytest.mark.parametrize("call", [fwd, bwd])
def test_window_landmark_options_validated(call):
    """r x r window landmarks (grid = (W', r)): the windows must tile the n-token map and give
    exactly m landmarks; otherwise the call is rejected before any launch."""
    assert call(grid=(10, 5), m=8) == L.LAPATTN_ERR_SHAPE      # 10 x 10 map, r = 5: m must be 4
    assert call(grid=(3, 1), m=8) == L.LAPATTN_ERR_SHAPE       # 100 tokens are not a 3-wide map
    assert call(grid=(20, 3), m=8) == L.LAPATTN_ERR_SHAPE      # r does not divide W' = 20
    assert call(grid=(4, 4), m=8) == L.LAPATTN_ERR_SHAPE       # r does not divide H' = 25
    assert call(grid=(0, 5), m=4) == L.LAPATTN_ERR_PARAM       # windows need the map
    assert call(grid=(3, 0), m=4) == L.LAPATTN_ERR_SHAPE       # a map without windows must still fit n
    assert call(grid=(-10, 5), m=4) == L.LAPATTN_ERR_PARAM
    # valid geometry: the call gets as far as the workspace check
    assert call(grid=(10, 5), m=4) == L.LAPATTN_ERR_WORKSPACE
    assert call(grid=(20, 5), m=4) == L.LAPATTN_ERR_WORKSPACE  # 5 x 20 map, r = 5: 1 x 4 windows
    assert call(grid=(10, 0), m=4) == L.LAPATTN_ERR_WORKSPACE  # a map with segment landmarks


@pytest.mark.parametrize("call", [fwd, bwd])
def test_convolution_options_validated(call):
    """The convolution branch: an odd filter side up to 7, the token map, and the filters."""
    for k in (2, 9, -1, 4):
        assert call(grid=(10, 0), m=4, dwc=(k, FAKE, None, None, None)) == L.LAPATTN_ERR_PARAM
    assert call(m=4, dwc=(3, FAKE, None, None, None)) == L.LAPATTN_ERR_PARAM          # no map
    assert call(grid=(3, 0), m=4, dwc=(3, FAKE, None, None, None)) == L.LAPATTN_ERR_SHAPE
    assert call(grid=(10, 0), m=4, dwc=(3, None, None, None, None)) == L.LAPATTN_ERR_NULL
    for k in (1, 3, 5, 7):
        assert call(grid=(10, 0), m=4, dwc=(k, FAKE, FAKE, FAKE, FAKE)) == L.LAPATTN_ERR_WORKSPACE
        assert call(grid=(10, 5), m=4, dwc=(k, FAKE, None, None, None)) == L.LAPATTN_ERR_WORKSPACE


def test_convolution_workspace():
    """The branch needs one fp32 [B,H,n,d] buffer in the forward and filter-gradient partials in
    the backward, both reported only with LAPATTN_WS_DWC; unknown flags give 0."""
    for dt in (0, 1):
        f0 = L.lapattn_workspace_size(2, 3, 3136, 64, 64, 8, dt, 0)
        f1 = L.lapattn_workspace_size(2, 3, 3136, 64, 64, 8, dt, L.LAPATTN_WS_DWC)
        assert f1 >= f0 + 2 * 3 * 3136 * 64 * 4
        b0 = L.lapattn_workspace_size(2, 3, 3136, 64, 64, 8, dt, L.LAPATTN_WS_BACKWARD)
        b1 = L.lapattn_workspace_size(2, 3, 3136, 64, 64, 8, dt, L.LAPATTN_WS_BACKWARD | L.LAPATTN_WS_DWC)
        assert b1 > b0
        assert L.lapattn_workspace_size(2, 3, 3136, 64, 64, 8, dt, 4) == 0


def test_saved_forward_needs_the_backward_workspace():
    """With save, the forward keeps the backward's internals: a forward-sized workspace is
    rejected (fp32); bf16 ignores save."""
    fsz = L.lapattn_workspace_size(1, 2, 100, 32, 8, 4, 0, 0)
    bsz = L.lapattn_workspace_size(1, 2, 100, 32, 8, 4, 0, L.LAPATTN_WS_BACKWARD)
    assert bsz > fsz
    assert fwd(save=True, workspace_bytes=fsz) == L.LAPATTN_ERR_WORKSPACE
    assert fwd(save=True, workspace_bytes=bsz - 256) == L.LAPATTN_ERR_WORKSPACE
    assert fwd(save=False, workspace_bytes=fsz - 256) == L.LAPATTN_ERR_WORKSPACE


def fwd_noalloc(**kw):
    args = dict(Q=FAKE, K=FAKE, V=FAKE, Out=FAKE, B=1, H=2, n=100, d=32, m=8, lam=1.0, ns_iters=4, dtype=0,
                norm=0, eps=0.0)
    args.update(kw)
    return L.lapattn_forward_noalloc(**args)


def test_forward_noalloc_validation():
    """The allocation-free forward applies the forward's checks, then rejects calls whose workspace
    would exceed its 32 MiB scratch array, and the save option -- all before any HIP call."""
    for p in ("Q", "K", "V", "Out"):
        assert fwd_noalloc(**{p: 0}) == L.LAPATTN_ERR_NULL
    assert fwd_noalloc(m=101) == L.LAPATTN_ERR_SHAPE
    assert fwd_noalloc(lam=0.0) == L.LAPATTN_ERR_PARAM
    assert fwd_noalloc(d=48) == L.LAPATTN_ERR_UNSUPPORTED
    assert fwd_noalloc(Q=FAKE + 4) == L.LAPATTN_ERR_ALIGN
    assert fwd_noalloc(save=True) == L.LAPATTN_ERR_PARAM
    # the n = 16384 workload fits (10 MiB of workspace); the same shape with fp32 inputs at twice
    # the batch (37 MiB), or with the convolution branch (74 MiB), does not
    big = dict(B=8, H=2, n=16384, d=64, m=64, ns_iters=8, dtype=1)
    assert L.lapattn_workspace_size(8, 2, 16384, 64, 64, 8, 1, 0) <= 32 << 20
    assert L.lapattn_workspace_size(16, 2, 16384, 64, 64, 8, 0, 0) > 32 << 20
    assert fwd_noalloc(**dict(big, B=16, dtype=0)) == L.LAPATTN_ERR_SCRATCH
    assert fwd_noalloc(**big, grid=(128, 0), dwc=(3, FAKE, 0, 0, 0)) == L.LAPATTN_ERR_SCRATCH
