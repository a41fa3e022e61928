"""Seeded synthetic workloads for Nystrom-Laplacian attention.

This module only draws inputs: it holds the five workload shapes and a seeded
generator.  It contains none of the method's arithmetic, so both the oracle and
the HIP path can be fed from it.

Inputs stand in for the paper's vision workloads (ImageNet-1K classification and
COCO detection, Sec. 5), which are not used here: the token counts are those of
the architectures it builds on -- 197 = 14x14 patches + a class token (DeiT at
224^2), 3136 = 56x56 (PVT stage 1 at 224^2), 16384 = 128x128 (dense prediction).

Recipe: numpy PCG64 ``default_rng(seed)``; draw ``standard_normal((B,H,n,d))`` for
Q, then K, then V, then (training workload only) dOut; scale Q, K, V by sigma and
dOut by 1; round to fp32 (round-to-nearest-even), then to bf16 (RNE) for the bf16
workloads.  A heavy-tailed variant (``dist="t3"``, a robustness case, not one of the
five workloads) draws Q and K from ``standard_t(3, ...)`` instead, in the same order.
The fp32 arrays returned always hold the exact values the device receives, so the
oracle sees the same numbers widened to fp64.
"""
import math
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    n: int
    d: int
    m: int
    T: int
    dtype: str        # "fp32" or "bf16": the input/output storage type
    sigma: float      # std of Q, K, V entries
    lam: float        # Laplacian scale lambda
    seed: int
    backward: bool    # the workload also runs the backward pass
    dist: str = "normal"   # Q and K entries: "normal", or "t3" (Student-t, 3 degrees of freedom)

    @property
    def BH(self):
        return self.B * self.H

    def with_(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


WORKLOADS = {
    # 1 x 1 head, n=256, d=32, m=16 segments of 16 tokens, lambda = sqrt(d), 6 NS updates
    "tiny": Workload("tiny", 1, 1, 256, 32, 16, 6, "fp32", 1.0, math.sqrt(32), 101, False),
    # DeiT-small-like: 64 x 6 heads, n=197 (14x14 + cls), d=64, m=32 (segments of 6 or 7)
    "deit_small": Workload("deit_small", 64, 6, 197, 64, 32, 6, "fp32", 1 / 8, 8.0, 102, False),
    # PVT stage-1-like: 32 x 1, n=3136 (56x56), d=64, m=64 (segments of 49), 8 NS updates, bf16
    "pvt_stage1": Workload("pvt_stage1", 32, 1, 3136, 64, 64, 8, "bf16", 1 / 8, 8.0, 103, False),
    # High resolution: 8 x 2, n=16384 (128x128), d=64, m=64 (segments of 256), 8 NS updates, bf16
    "highres": Workload("highres", 8, 2, 16384, 64, 64, 8, "bf16", 1 / 8, 8.0, 104, False),
    # Training step: 32 x 4, n=3136, d=32, m=64, 6 NS updates, fp32, forward + backward
    "train": Workload("train", 32, 4, 3136, 32, 64, 6, "fp32", 1 / math.sqrt(32), math.sqrt(32), 105, True),
}


def round_bf16(x32):
    """Round fp32 values to the nearest bf16 (ties to even); returned as fp32."""
    x32 = np.ascontiguousarray(x32, dtype=np.float32)
    b = x32.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    return b.astype(np.uint32).view(np.float32)


def bf16_bits(x32):
    """The 16-bit patterns of fp32 values that are already bf16-representable."""
    x32 = np.ascontiguousarray(x32, dtype=np.float32)
    return (x32.view(np.uint32) >> 16).astype(np.uint16)


def make_inputs(w, with_grad=None, heads=None):
    """Draw Q, K, V (and dOut) for workload ``w``.

    Returns a dict of fp32 numpy arrays [B,H,n,d] holding exactly the values the
    device receives (already bf16-rounded for bf16 workloads).  ``heads``
    optionally keeps only the listed flat head indices (b*H + h) after drawing the
    full tensors, so a sample matches the full workload exactly.
    """
    with_grad = w.backward if with_grad is None else with_grad
    rng = np.random.default_rng(w.seed)
    shape = (w.B, w.H, w.n, w.d)
    out = {}
    for name, scale in (("Q", w.sigma), ("K", w.sigma), ("V", w.sigma)) + ((("dO", 1.0),) if with_grad else ()):
        if w.dist == "t3" and name in ("Q", "K"):
            x = (rng.standard_t(3, shape) * scale).astype(np.float32)
        else:
            x = (rng.standard_normal(shape) * scale).astype(np.float32)
        if w.dtype == "bf16":
            x = round_bf16(x)
        out[name] = x
    if heads is not None:
        heads = list(heads)
        for k in out:
            out[k] = np.ascontiguousarray(out[k].reshape(w.BH, w.n, w.d)[heads][None])
    return out


def small(w, n=None, B=1, H=2, m=None, seed=None):
    """A reduced-size variant of a workload with the same d, T, dtype, lambda and
    value distribution (used where the oracle must cover every output)."""
    n = n if n is not None else w.n
    m = m if m is not None else min(w.m, n)
    return w.with_(name=w.name + "_small", B=B, H=H, n=n, m=m, seed=seed if seed is not None else w.seed + 1000)


def make_dwc(H, d, k, seed, bias=True):
    """Filters [H][d][k][k] ~ N(0, 1/k^2) and a bias [H][d] ~ N(0, 0.1^2) (fp32 numpy arrays;
    bias None when not drawn) for the depth-wise convolution branch."""
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((H, d, k, k)) / k).astype(np.float32)
    b = (0.1 * rng.standard_normal((H, d))).astype(np.float32) if bias else None
    return w, b
