"""Pins for the fp64 oracle (CPU only).

The paper prints no numeric output for any step of the path, so the oracle is
pinned to what the mathematics fixes: hand-derived worked examples
(tests/golden/worked_examples.txt), closed forms, special cases that reduce to
exact dense Laplacian attention or to a library inverse, invariants of the
normalisation, and central finite differences for the backward.  Each check is
chosen so that a plausible slip in the oracle (a dropped term, a sign, a wrong
index, a transposed factor, a wrong norm) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.txt")


# ----------------------------------------------------------------------------- helpers

def parse_golden():
    cases, cur = {}, None
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("["):
                cur = cases.setdefault(line.strip("[]"), {})
                continue
            k, v = (s.strip() for s in line.split("=", 1))
            cur[k] = v
    return cases


def num_rows(s):
    return np.array([[eval(x, {"exp": math.exp}) for x in row.split()] for row in s.split(";")], dtype=np.float64)


def exprs(s):
    return np.array([eval(x, {"exp": math.exp}) for x in s.split(";")], dtype=np.float64)


def dense_laplacian_attention(Q, K, V, lam, norm):
    """Exact O(n^2 d) Laplacian-kernel attention of one head, written from the
    definitions: g_ij = exp(-||q_i - k_j||_1 / lambda) (Sec. 4.1) and
    inline: z_ij = g_ij - mean_j g_ij + 1/n (Eq. (4), Sigma^{-1/2} = I), out = Z V;
    rowsum: Eq. (3); none: G V."""
    G = np.exp(-np.abs(Q[:, None, :] - K[None, :, :]).sum(-1) / lam)
    n = K.shape[0]
    if norm == oracle.NORM_INLINE:
        Z = G - G.mean(axis=1, keepdims=True) + 1.0 / n
        return Z @ V
    if norm == oracle.NORM_ROWSUM:
        return (G @ V) / G.sum(axis=1, keepdims=True)
    return G @ V


def rand_qkv(rng, B, H, n, d, sigma=1.0):
    return [rng.standard_normal((B, H, n, d)) * sigma for _ in range(3)]


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


# ----------------------------------------------------------------------------- kernel

def test_kernel_identity_and_unit_distance(oracle_lib):
    rng = np.random.default_rng(1)
    x = rng.standard_normal(7)
    assert oracle.kernel(x, x, 3.0) == 1.0                       # k(x, x) = 1
    # ||x - y||_1 = lambda gives exactly e^-1 (all terms are exact binary fractions)
    x = np.zeros(4)
    y = np.array([1.0, -1.0, 0.5, -1.5])
    assert oracle.kernel(x, y, 4.0) == pytest.approx(math.exp(-1.0), rel=1e-15)
    y2 = rng.standard_normal(7)
    x2 = rng.standard_normal(7)
    assert oracle.kernel(x2, y2, 2.0) == oracle.kernel(y2, x2, 2.0)   # symmetric


def test_kernel_gradient_norm_appendix_a(oracle_lib):
    """App. A: away from coordinate ties, ||grad_x k||_2 = (sqrt(d)/lambda) k.
    An l2 (Gaussian-like) kernel or a wrong lambda placement fails this."""
    rng = np.random.default_rng(2)
    for d, lam in ((5, 1.0), (32, math.sqrt(32)), (64, 8.0)):
        x, y = rng.standard_normal(d), rng.standard_normal(d)
        h = 1e-7
        g = np.empty(d)
        for c in range(d):
            e = np.zeros(d)
            e[c] = h
            g[c] = (oracle.kernel(x + e, y, lam) - oracle.kernel(x - e, y, lam)) / (2 * h)
        k = oracle.kernel(x, y, lam)
        assert np.linalg.norm(g) == pytest.approx(math.sqrt(d) / lam * k, rel=1e-6)
        # each component is -(1/lambda) sign(x_c - y_c) k (the minus sign of App. A)
        np.testing.assert_allclose(g, -np.sign(x - y) * k / lam, rtol=1e-6, atol=1e-12)


# ----------------------------------------------------------------------------- segments

@pytest.mark.parametrize("n,m", [(197, 32), (256, 16), (3136, 64), (16384, 64), (13, 5), (7, 7), (9, 1)])
def test_segments_balanced_partition(oracle_lib, n, m):
    s = oracle.segments(n, m)
    sizes = np.diff(s)
    assert s[0] == 0 and s[-1] == n and len(s) == m + 1
    assert sizes.min() >= 1 and sizes.max() - sizes.min() <= 1
    assert sizes.sum() == n


def test_segments_deit_shape(oracle_lib):
    sizes = np.diff(oracle.segments(197, 32))
    assert (sizes == 6).sum() == 27 and (sizes == 7).sum() == 5   # 27*6 + 5*7 = 197
    assert list(np.diff(oracle.segments(3136, 64))) == [49] * 64


def test_segments_golden(oracle_lib):
    c = parse_golden()["seg1"]
    assert list(oracle.segments(10, 4)) == [int(x) for x in c["starts_10_4"].split()]
    s = oracle.segments(197, 32)
    assert s[1] == int(c["first_197_32"]) and s[31] == int(c["last_start_197_32"])


def test_forward_permutation_within_hand_stated_segments(oracle_lib):
    """Same invariance with the segment boundaries of the golden file (n=10, m=4)."""
    starts = [int(x) for x in parse_golden()["seg1"]["starts_10_4"].split()]
    rng = np.random.default_rng(12)
    Q, K, V = rand_qkv(rng, 1, 1, 10, 3)
    out = oracle.forward(Q, K, V, 4, 1.3, 4)
    perm = np.concatenate([starts[l] + rng.permutation(starts[l + 1] - starts[l])[::-1] for l in range(4)])
    outp = oracle.forward(Q[:, :, perm], K[:, :, perm], V[:, :, perm], 4, 1.3, 4)
    np.testing.assert_allclose(outp, out[:, :, perm], rtol=1e-12, atol=1e-13)


def test_segments_reject_m_above_n(oracle_lib):
    with pytest.raises(ValueError):
        oracle.segments(4, 5)


# ----------------------------------------------------------------------------- Newton-Schulz

def test_ns_golden_examples(oracle_lib):
    g = parse_golden()
    for key in ("ns1", "ns2"):
        c = g[key]
        Wm = num_rows(c["W"])
        T = int(c["T"])
        eps = float(c.get("eps", "0"))
        Xs, _ = oracle.ns(Wm, T, eps)
        np.testing.assert_allclose(Xs[T], num_rows(c["X1"]), rtol=0, atol=1e-15)


def test_ns_x0_uses_transpose_and_induced_norms(oracle_lib):
    rng = np.random.default_rng(3)
    Wm = rng.random((9, 9)) + np.triu(rng.random((9, 9)))      # nonsymmetric, positive
    Xs, c = oracle.ns(Wm, 0)
    cref = np.linalg.norm(Wm, 1) * np.linalg.norm(Wm, np.inf)
    assert c == pytest.approx(cref, rel=1e-14)
    np.testing.assert_allclose(Xs[0], Wm.T / cref, rtol=1e-14)


@pytest.mark.parametrize("m,T", [(16, 6), (32, 6), (64, 8), (7, 3)])
def test_ns_residual_identity(oracle_lib, m, T):
    """X_{t+1} = X_t (2I - W X_t) gives I - X_{t+1} W = (I - X_t W)^2, hence
    I - X_T W = (I - X0 W)^(2^T) with X0 = W^T/c."""
    rng = np.random.default_rng(10 + m)
    Wm = np.exp(-np.abs(rng.standard_normal((m, 1, 4)) - rng.standard_normal((1, m, 4))).sum(-1) / 2.0)
    Xs, c = oracle.ns(Wm, T)
    R0 = np.eye(m) - Wm.T @ Wm / (np.linalg.norm(Wm, 1) * np.linalg.norm(Wm, np.inf))
    expect = np.linalg.matrix_power(R0, 2 ** T)
    np.testing.assert_allclose(np.eye(m) - Xs[T] @ Wm, expect, rtol=0, atol=1e-12)
    # the closed-form residual bound with sigma_min from the SVD
    smin = np.linalg.svd(Wm, compute_uv=False).min()
    bound = (1 - smin ** 2 / c) ** (2 ** T)
    assert np.linalg.norm(np.eye(m) - Xs[T] @ Wm, 2) <= bound + 1e-12


def test_ns_special_cases(oracle_lib):
    m = 6
    # W = c I: X0 = I/c = W^-1 exactly, and it stays there
    Xs, _ = oracle.ns(3.0 * np.eye(m), 4)
    for t in range(5):
        np.testing.assert_allclose(Xs[t], np.eye(m) / 3.0, rtol=1e-15)
    # diagonal W: x_T = (1 - (1 - w^2/c)^(2^T)) / w elementwise, c = max w^2
    w = np.array([0.3, 1.0, 2.0, 0.7, 1.5, 0.05])
    T = 5
    Xs, c = oracle.ns(np.diag(w), T)
    assert c == pytest.approx(4.0)
    np.testing.assert_allclose(np.diag(Xs[T]), (1 - (1 - w ** 2 / 4.0) ** (2 ** T)) / w, rtol=1e-12)
    assert np.abs(Xs[T] - np.diag(np.diag(Xs[T]))).max() == 0.0
    # all-ones W: X_t = 11^T / m^2 = pinv(W) for every t
    ones = np.ones((m, m))
    Xs, _ = oracle.ns(ones, 5)
    for t in range(6):
        np.testing.assert_allclose(Xs[t], np.linalg.pinv(ones), rtol=1e-13)
    # W = 0: the start scale vanishes and X := 0
    Xs, c = oracle.ns(np.zeros((m, m)), 3)
    assert c == 0.0 and not Xs.any()


@pytest.mark.parametrize("kappa", [2, 10, 50])
@pytest.mark.parametrize("spd", [True, False])
def test_ns_converges_to_inverse(oracle_lib, kappa, spd):
    """Sec. 5.3 runs Newton-Schulz for condition numbers 2..50 and reports stable
    convergence; with X0 = W^T/c the residual contracts for any nonsingular W."""
    m = 24
    rng = np.random.default_rng(kappa * 7 + spd)
    Uo, _ = np.linalg.qr(rng.standard_normal((m, m)))
    Vo, _ = np.linalg.qr(rng.standard_normal((m, m)))
    s = np.geomspace(1.0, kappa, m)
    Wm = Uo @ np.diag(s) @ (Uo if spd else Vo).T
    c = np.linalg.norm(Wm, 1) * np.linalg.norm(Wm, np.inf)
    T = int(math.ceil(math.log2(math.log(1e-16) / math.log(1 - 1.0 / c)))) + 1
    Xs, _ = oracle.ns(Wm, T)
    inv = np.linalg.inv(Wm)
    assert rel(Xs[T], inv) < 1e-11
    res = [np.linalg.norm(np.eye(m) - Xs[t] @ Wm, 2) for t in range(T + 1)]
    assert all(res[t + 1] <= res[t] + 1e-12 for t in range(T))       # monotone contraction


# ----------------------------------------------------------------------------- forward

def test_forward_golden_examples(oracle_lib):
    g = parse_golden()
    for key in ("ex1", "ex2"):
        c = g[key]
        n, d, m, T = int(c["n"]), int(c["d"]), int(c["m"]), int(c["T"])
        lam = float(c["lambda"])
        Q = np.array([float(x) for x in c["Q"].split()]).reshape(1, 1, n, d)
        K = np.array([float(x) for x in c["K"].split()]).reshape(1, 1, n, d)
        V = np.array([float(x) for x in c["V"].split()]).reshape(1, 1, n, d)
        for norm, field in ((oracle.NORM_INLINE, "inline"), (oracle.NORM_ROWSUM, "rowsum"), (oracle.NORM_NONE, "none")):
            out = oracle.forward(Q, K, V, m, lam, T, norm)
            np.testing.assert_allclose(out.reshape(-1), exprs(c[field]), rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("norm", [oracle.NORM_INLINE, oracle.NORM_ROWSUM, oracle.NORM_NONE])
@pytest.mark.parametrize("n,d,lam", [(16, 8, math.sqrt(8)), (40, 4, 4.0), (24, 32, math.sqrt(32))])
def test_forward_landmarks_equal_tokens_is_dense_attention(oracle_lib, norm, n, d, lam):
    """With m = n every segment is one token, K_QL = K_LL = K_LK = G, and once
    Newton-Schulz has converged G^ = G G^-1 G = G: the method reduces to exact
    dense Laplacian attention.  Pins the kernel, the factor orientation and the
    normalisation together."""
    rng = np.random.default_rng(n * 100 + d)
    Q, K, V = rand_qkv(rng, 1, 2, n, d)
    out, it = oracle.forward(Q, K, V, n, lam, 60, norm, intermediates=True)
    for h in range(2):
        Wm = it["W"][0, h]
        floor = 1e-15 * np.linalg.cond(Wm) * n          # fp64 rounding floor of a converged inverse
        assert np.linalg.norm(np.eye(n) - it["Xs"][0, h, -1] @ Wm) < floor   # converged
        ref = dense_laplacian_attention(Q[0, h], K[0, h], V[0, h], lam, norm)
        assert rel(out[0, h], ref) < max(floor, 1e-12)


def test_forward_tiny_workload_m_equals_n(oracle_lib):
    """The tiny workload's shape (n = 256, d = 32, N(0,1)) with m = n: kappa(K_LL)
    is ~3e5, so about 50 updates are needed to converge; then the result is the
    dense attention up to the fp64 rounding floor of a kappa ~ 3e5 inverse."""
    w = W.WORKLOADS["tiny"]
    x = W.make_inputs(w)
    out, it = oracle.forward(x["Q"], x["K"], x["V"], 256, w.lam, 52, intermediates=True)
    Wm = it["W"][0, 0]
    floor = 1e-15 * np.linalg.cond(Wm) * 256
    assert np.linalg.norm(np.eye(256) - it["Xs"][0, 0, -1] @ Wm) < floor
    ref = dense_laplacian_attention(x["Q"][0, 0].astype(np.float64), x["K"][0, 0].astype(np.float64),
                                    x["V"][0, 0].astype(np.float64), w.lam, oracle.NORM_INLINE)
    assert rel(out[0, 0], ref) < floor


def test_forward_one_landmark_closed_form(oracle_lib):
    """m = 1: the landmarks are the global means, K_LL = k(qbar, kbar) is 1x1 and
    X0 = 1/K_LL is already its inverse, so G^_ij = k(q_i, kbar) k(qbar, k_j) / k(qbar, kbar)."""
    rng = np.random.default_rng(5)
    Q, K, V = rand_qkv(rng, 1, 1, 11, 3)
    lam = 1.7
    out = oracle.forward(Q, K, V, 1, lam, 4)[0, 0]
    q, k, v = Q[0, 0], K[0, 0], V[0, 0]
    qb, kb = q.mean(0), k.mean(0)
    lap = lambda a, b: np.exp(-np.abs(a - b).sum(-1) / lam)
    G = lap(q, kb)[:, None] * lap(qb, k)[None, :] / lap(qb, kb)
    Z = G - G.mean(1, keepdims=True) + 1.0 / 11
    np.testing.assert_allclose(out, Z @ v, rtol=1e-13, atol=1e-14)


def test_forward_inline_rows_sum_to_one(oracle_lib):
    """Eq. (4) with Sigma^{-1/2} = I: every row of Z sums to 1, so a constant V is
    reproduced exactly, a translation of V translates the output, and the output
    is linear in V -- whatever X_T is (T = 6, far from converged)."""
    rng = np.random.default_rng(6)
    Q, K, V = rand_qkv(rng, 1, 2, 37, 8)
    m, lam, T = 9, 2.0, 6
    c = rng.standard_normal(8)
    const = np.broadcast_to(c, V.shape).copy()
    out_c = oracle.forward(Q, K, const, m, lam, T)
    np.testing.assert_allclose(out_c, const, rtol=1e-9, atol=1e-9)
    out = oracle.forward(Q, K, V, m, lam, T)
    out_t = oracle.forward(Q, K, V + c, m, lam, T)
    np.testing.assert_allclose(out_t, out + c, rtol=1e-9, atol=1e-9)
    V2 = rng.standard_normal(V.shape)
    out2 = oracle.forward(Q, K, V2, m, lam, T)
    out12 = oracle.forward(Q, K, 2.0 * V - 3.0 * V2, m, lam, T)
    np.testing.assert_allclose(out12, 2.0 * out - 3.0 * out2, rtol=1e-9, atol=1e-9)


def test_forward_permutation_within_segments(oracle_lib):
    """Landmarks are segment means, so permuting tokens jointly inside each
    segment [floor(l n/m), floor((l+1) n/m)) permutes the outputs the same way;
    a permutation across a segment boundary does not."""
    rng = np.random.default_rng(7)
    n, d, m = 29, 5, 6
    Q, K, V = rand_qkv(rng, 1, 1, n, d)
    out = oracle.forward(Q, K, V, m, 1.5, 5)
    s = oracle.segments(n, m)
    perm = np.concatenate([s[l] + rng.permutation(s[l + 1] - s[l]) for l in range(m)])
    outp = oracle.forward(Q[:, :, perm], K[:, :, perm], V[:, :, perm], m, 1.5, 5)
    np.testing.assert_allclose(outp, out[:, :, perm], rtol=1e-12, atol=1e-13)
    swap = np.arange(n)
    swap[[s[1] - 1, s[1]]] = swap[[s[1], s[1] - 1]]         # exchange across the first boundary
    outs = oracle.forward(Q[:, :, swap], K[:, :, swap], V[:, :, swap], m, 1.5, 5)
    assert np.abs(outs - out[:, :, swap]).max() > 1e-6


def test_forward_large_lambda_gives_mean_value(oracle_lib):
    """lambda -> infinity: every kernel value is 1, K_LL = 11^T whose NS iterate
    is its pseudoinverse, G^ = 11^T, s_i = n and out_i = vbar."""
    rng = np.random.default_rng(8)
    Q, K, V = rand_qkv(rng, 1, 1, 20, 4)
    out = oracle.forward(Q, K, V, 5, 1e12, 6)
    np.testing.assert_allclose(out[0, 0], np.broadcast_to(V[0, 0].mean(0), (20, 4)), rtol=1e-9, atol=1e-9)


def test_forward_zero_scale_guard(oracle_lib):
    """Tiny lambda underflows every kernel value: K_LL = 0, X := 0, G^ = 0 and the
    inline output is vbar (rowsum would divide by zero and is not asked)."""
    rng = np.random.default_rng(9)
    Q, K, V = rand_qkv(rng, 1, 1, 12, 3)
    out, it = oracle.forward(Q, K, V, 4, 1e-6, 3, intermediates=True)
    assert not it["Xs"].any()
    np.testing.assert_allclose(out[0, 0], np.broadcast_to(V[0, 0].mean(0), (12, 3)), rtol=1e-12)


def test_forward_factored_equals_explicit_nystrom(oracle_lib):
    """The factored K_QL (X_T (K_LK [V|1])) equals the explicit n x n G^ = K_QL X_T K_LK
    built in numpy from independently computed landmark means."""
    rng = np.random.default_rng(11)
    n, d, m, lam, T = 31, 6, 7, 2.5, 6
    Q, K, V = rand_qkv(rng, 1, 1, n, d)
    out, it = oracle.forward(Q, K, V, m, lam, T, intermediates=True)
    s = oracle.segments(n, m)
    q, k, v = Q[0, 0], K[0, 0], V[0, 0]
    qt = np.stack([q[s[l]:s[l + 1]].mean(0) for l in range(m)])
    kt = np.stack([k[s[l]:s[l + 1]].mean(0) for l in range(m)])
    np.testing.assert_allclose(it["Qt"][0, 0], qt, rtol=1e-14)
    lap = lambda a, b: np.exp(-np.abs(a[:, None] - b[None]).sum(-1) / lam)
    np.testing.assert_allclose(it["W"][0, 0], lap(qt, kt), rtol=1e-14)
    G = lap(q, kt) @ it["Xs"][0, 0, T] @ lap(qt, k)
    Z = G - G.sum(1, keepdims=True) / n + 1.0 / n
    assert rel(out[0, 0], Z @ v) < 1e-12


# ----------------------------------------------------------------------------- backward

def fd_check(Q, K, V, dO, m, lam, T, norm, eps=0.0, h=1e-6, whiten=None):
    dQ, dK, dV = oracle.backward(Q, K, V, dO, m, lam, T, norm, eps, whiten=whiten)
    grads = {"Q": dQ, "K": dK, "V": dV}
    base = {"Q": Q, "K": K, "V": V}
    worst = 0.0
    for name in ("Q", "K", "V"):
        g = np.zeros_like(Q)
        for idx in np.ndindex(Q.shape):
            args = {k: v.copy() for k, v in base.items()}
            args[name][idx] += h
            lp = (oracle.forward(args["Q"], args["K"], args["V"], m, lam, T, norm, eps, whiten=whiten) * dO).sum()
            args[name][idx] -= 2 * h
            lm = (oracle.forward(args["Q"], args["K"], args["V"], m, lam, T, norm, eps, whiten=whiten) * dO).sum()
            g[idx] = (lp - lm) / (2 * h)
        scale = max(np.abs(g).max(), 1e-12)
        worst = max(worst, np.abs(g - grads[name]).max() / scale)
    return worst


@pytest.mark.parametrize("norm", [oracle.NORM_INLINE, oracle.NORM_ROWSUM, oracle.NORM_NONE])
@pytest.mark.parametrize("n,d,m,T,lam", [(13, 3, 5, 4, 1.5), (6, 2, 6, 3, 2.0), (17, 4, 4, 6, 4.0), (9, 5, 1, 2, 3.0)])
def test_backward_matches_finite_differences(oracle_lib, norm, n, d, m, T, lam):
    rng = np.random.default_rng(n * 31 + d * 7 + m + norm)
    Q, K, V = rand_qkv(rng, 1, 1, n, d, 0.7)
    dO = rng.standard_normal(Q.shape)
    assert fd_check(Q, K, V, dO, m, lam, T, norm) < 1e-7


def test_backward_with_perturbation_and_two_heads(oracle_lib):
    rng = np.random.default_rng(21)
    Q, K, V = rand_qkv(rng, 1, 2, 10, 3, 0.5)
    dO = rng.standard_normal(Q.shape)
    assert fd_check(Q, K, V, dO, 4, 1.0, 5, oracle.NORM_INLINE, eps=0.3) < 1e-7


def test_backward_dv_closed_form(oracle_lib):
    """Inline normalisation: out = Z V with Z = G^ - (G^ 1) 1^T/n + 11^T/n and Z
    independent of V, so dV = Z^T dO = G^T dO + (1/n) 1 ((1 - G^ 1)^T dO)."""
    rng = np.random.default_rng(22)
    n, d, m, lam, T = 27, 4, 6, 2.0, 6
    Q, K, V = rand_qkv(rng, 1, 1, n, d)
    dO = rng.standard_normal(Q.shape)
    _, it = oracle.forward(Q, K, V, m, lam, T, intermediates=True)
    q, k = Q[0, 0], K[0, 0]
    lap = lambda a, b: np.exp(-np.abs(a[:, None] - b[None]).sum(-1) / lam)
    G = lap(q, it["Kt"][0, 0]) @ it["Xs"][0, 0, T] @ lap(it["Qt"][0, 0], k)
    s = G.sum(1)
    dv_ref = G.T @ dO[0, 0] + np.outer(np.ones(n), (1 - s) @ dO[0, 0]) / n
    _, _, dV = oracle.backward(Q, K, V, dO, m, lam, T)
    np.testing.assert_allclose(dV[0, 0], dv_ref, rtol=1e-11, atol=1e-12)


def test_backward_scale_term_is_needed(oracle_lib):
    """The X0 scale c = ||W||_1 ||W||_inf depends on the landmarks; the
    finite-difference check above would fail without its gradient.  Here: the
    gradient is not symmetric in a way that hides it -- dQ changes when c is
    perturbed through one landmark only (a smoke check that c enters)."""
    rng = np.random.default_rng(23)
    Q, K, V = rand_qkv(rng, 1, 1, 8, 2)
    dO = rng.standard_normal(Q.shape)
    assert fd_check(Q, K, V, dO, 8, 1.0, 0, oracle.NORM_NONE) < 1e-7   # T = 0: output = A W^T/c B V


def test_backward_sign_decided_on_fp32_landmark_means(oracle_lib):
    """R16: a key coordinate equal to the fp32 rounding of a query-landmark mean is a tie of
    sign(qt - k) for the kernels, which hold landmarks in fp32.  Input A: queries 1 and 1 + 2^-23
    (fp32 neighbours), mean 1 + 2^-24, which rounds (to even) to 1.0; key coordinate 1.0.
    Input B: the second query is 1.0, so the mean is exactly 1.0 and the tie is real.  At a kink
    the central difference gives the average of the one-sided derivatives, i.e. sign(0) = 0
    (R8); the oracle's gradient at A must equal it up to the smooth change of 2^-24, while the
    fp64 decision sign(2^-24) = 1 would differ by a whole one-sided term."""
    lam, T, m = 1.5, 4, 2
    Q = np.array([[1.0, 0.3], [1.0 + 2.0 ** -23, -0.2], [0.5, 0.7], [-0.1, 0.2]])[None, None]
    K = np.array([[0.3, -0.4], [-0.6, 0.1], [1.0, 0.4], [0.2, -0.3]])[None, None]
    rng = np.random.default_rng(41)
    V = rng.standard_normal(Q.shape)
    dO = rng.standard_normal(Q.shape)
    assert np.float32((Q[0, 0, 0, 0] + Q[0, 0, 1, 0]) / 2) == np.float32(1.0)
    QB = Q.copy()
    QB[0, 0, 1, 0] = 1.0
    h = 1e-7
    loss = lambda q, k: (oracle.forward(q, k, V, m, lam, T) * dO).sum()
    kp, km = K.copy(), K.copy()
    kp[0, 0, 2, 0] += h
    km[0, 0, 2, 0] -= h
    fd_b = (loss(QB, kp) - loss(QB, km)) / (2 * h)
    dK_a = oracle.backward(Q, K, V, dO, m, lam, T)[1][0, 0, 2, 0]
    dK_b = oracle.backward(QB, K, V, dO, m, lam, T)[1][0, 0, 2, 0]
    assert abs(dK_b - fd_b) < 1e-6 * max(1.0, abs(fd_b))
    assert abs(dK_a - fd_b) < 1e-5 * max(1.0, abs(fd_b))
    # the one-sided derivatives (above and below the kink) differ from the tie value
    kp2 = K.copy()
    kp2[0, 0, 2, 0] += 2 * h
    right = (loss(QB, kp2) - loss(QB, kp)) / h
    assert abs(right - fd_b) > 1e-3


# ----------------------------------------------------------------------------- 2-D windows

def window_order(hp, wp, r):
    """Token indices of an hp x wp row-major map grouped by r x r window (windows row-major,
    tokens row-major inside a window), built by reshaping the map -- the layout average
    pooling with kernel r and stride r works on (Sec. 4.2)."""
    idx = np.arange(hp * wp).reshape(hp // r, r, wp // r, r)
    return idx.transpose(0, 2, 1, 3).reshape(-1)


@pytest.mark.parametrize("hp,wp,r", [(4, 6, 2), (6, 6, 3), (8, 4, 2), (3, 9, 3)])
def test_windows_landmarks_are_average_pooling(oracle_lib, hp, wp, r):
    """The landmark means of the windowed oracle equal numpy's r x r average pooling of the
    token map, in the row-major order of the pooled map."""
    rng = np.random.default_rng(hp * 100 + wp * 10 + r)
    n, m, d = hp * wp, (hp // r) * (wp // r), 3
    Q, K, V = rand_qkv(rng, 1, 2, n, d)
    _, inter = oracle.forward(Q, K, V, m, 2.0, 3, intermediates=True, grid=(wp, r))
    pool = lambda X: X.reshape(1, 2, hp // r, r, wp // r, r, d).mean(axis=(3, 5)).reshape(1, 2, m, d)
    assert np.allclose(inter["Qt"], pool(Q), rtol=1e-13, atol=1e-14)
    assert np.allclose(inter["Kt"], pool(K), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("norm", [oracle.NORM_INLINE, oracle.NORM_ROWSUM])
def test_windows_equal_segments_of_the_window_ordered_tokens(oracle_lib, norm):
    """Everything after pooling treats tokens alike, so the windowed forward and backward on a
    token map equal the segment forward and backward on the tokens listed window by window
    (each window is then one segment of r^2 consecutive tokens), permuted back."""
    hp, wp, r, d = 6, 8, 2, 3
    n, m = hp * wp, (hp // r) * (wp // r)
    perm = window_order(hp, wp, r)
    rng = np.random.default_rng(77 + norm)
    Q, K, V = rand_qkv(rng, 1, 2, n, d, 0.6)
    dO = rng.standard_normal(Q.shape)
    out2 = oracle.forward(Q, K, V, m, 1.7, 4, norm, grid=(wp, r))
    out1 = oracle.forward(Q[:, :, perm], K[:, :, perm], V[:, :, perm], m, 1.7, 4, norm)
    assert rel(out2[:, :, perm], out1) < 1e-13
    g2 = oracle.backward(Q, K, V, dO, m, 1.7, 4, norm, grid=(wp, r))
    g1 = oracle.backward(Q[:, :, perm], K[:, :, perm], V[:, :, perm], dO[:, :, perm], m, 1.7, 4, norm)
    for a, b in zip(g2, g1):
        assert rel(a[:, :, perm], b) < 1e-12


def test_windows_special_cases_and_rejections(oracle_lib):
    rng = np.random.default_rng(5)
    Q, K, V = rand_qkv(rng, 1, 1, 12, 2)
    # r = 1: every token is a landmark, as segments with m = n
    assert rel(oracle.forward(Q, K, V, 12, 1.0, 5, grid=(4, 1)), oracle.forward(Q, K, V, 12, 1.0, 5)) < 1e-14
    # one window covering the map: the global mean, as one segment
    Q2, K2, V2 = rand_qkv(rng, 1, 1, 9, 2)
    assert rel(oracle.forward(Q2, K2, V2, 1, 1.0, 3, grid=(3, 3)), oracle.forward(Q2, K2, V2, 1, 1.0, 3)) < 1e-14
    # r must divide both sides, n must fill the map, m must match the pooled map
    for grid, m in (((4, 3), 1), ((5, 1), 12), ((4, 2), 4), ((6, 2), 4)):
        with pytest.raises(ValueError):
            oracle.forward(Q, K, V, m, 1.0, 2, grid=grid)


# ----------------------------------------------------------------------------- DWC(V) branch (R14)

def rand_dwc(rng, H, d, k, bias=True):
    w = rng.standard_normal((H, d, k, k))
    return w, (rng.standard_normal((H, d)) if bias else None)


@pytest.mark.parametrize("gh,gw,k", [(5, 7, 3), (4, 4, 1), (3, 8, 5), (6, 5, 7), (2, 9, 3)])
def test_dwc_is_library_cross_correlation(oracle_lib, gh, gw, k):
    """Each channel's map is scipy's zero-filled 'same' cross-correlation with its filter."""
    from scipy.signal import correlate2d
    rng = np.random.default_rng(gh * 100 + gw * 10 + k)
    B, H, d = 2, 2, 3
    V = rng.standard_normal((B, H, gh * gw, d))
    w, b = rand_dwc(rng, H, d, k)
    E = oracle.dwc(V, w, b, gw)
    for bi in range(B):
        for h in range(H):
            for c in range(d):
                ref = correlate2d(V[bi, h, :, c].reshape(gh, gw), w[h, c], mode="same", boundary="fill") + b[h, c]
                np.testing.assert_allclose(E[bi, h, :, c].reshape(gh, gw), ref, rtol=1e-13, atol=1e-13)


def test_dwc_one_hot_filters_shift_the_map(oracle_lib):
    """A filter with a single 1 at tap (u, t) copies the value at offset (u - p, t - p),
    zero off the map; the centre tap is the identity; the bias adds per channel."""
    rng = np.random.default_rng(3)
    gh, gw, k, d = 4, 6, 5, 2
    p = (k - 1) // 2
    V = rng.standard_normal((1, 1, gh * gw, d))
    bias = np.array([[0.25, -1.5]])
    for u, t in ((p, p), (0, 4), (3, 1), (4, 4)):
        w = np.zeros((1, d, k, k))
        w[:, :, u, t] = 1.0
        E = oracle.dwc(V, w, bias, gw)[0, 0].reshape(gh, gw, d)
        grid = V[0, 0].reshape(gh, gw, d)
        for y in range(gh):
            for x in range(gw):
                yy, xx = y + u - p, x + t - p
                want = (grid[yy, xx] if 0 <= yy < gh and 0 <= xx < gw else np.zeros(d)) + bias[0]
                np.testing.assert_array_equal(E[y, x], want)


def test_dwc_backward_matches_finite_differences(oracle_lib):
    """sum(DWC(V) * dE) is linear in V, in the filters and in the bias separately, so central
    differences give every gradient entry up to rounding (brute force over all entries)."""
    rng = np.random.default_rng(4)
    B, H, gh, gw, d, k = 2, 2, 3, 4, 2, 3
    V = rng.standard_normal((B, H, gh * gw, d))
    w, b = rand_dwc(rng, H, d, k)
    dE = rng.standard_normal(V.shape)
    dV, dW, db = oracle.dwc_backward(V, w, dE, gw)
    f = lambda V_, w_, b_: float((oracle.dwc(V_, w_, b_, gw) * dE).sum())
    for arr, grad, name in ((V, dV, "V"), (w, dW, "W"), (b, db, "b")):
        for idx in np.ndindex(arr.shape):
            args = {"V": V.copy(), "W": w.copy(), "b": b.copy()}
            args[name][idx] += 0.5
            fp = f(args["V"], args["W"], args["b"])
            args[name][idx] -= 1.0
            fm = f(args["V"], args["W"], args["b"])
            assert abs((fp - fm) - grad[idx]) < 1e-11, (name, idx)


def test_dwc_in_the_full_path(oracle_lib):
    """Eq. (7): Out = Z V + DWC(V).  The branch adds exactly DWC(V) to the forward; the
    backward adds the branch's dV and gives the filter and bias gradients, checked by central
    differences through the whole path (dQ, dK are unchanged by the branch)."""
    rng = np.random.default_rng(6)
    gh, gw, d, m, T, lam, k = 3, 4, 2, 3, 4, 1.5, 3
    n = gh * gw
    Q, K, V = rand_qkv(rng, 1, 2, n, d, 0.7)
    w, b = rand_dwc(rng, 2, d, k)
    dO = rng.standard_normal(Q.shape)
    base = oracle.forward(Q, K, V, m, lam, T)
    both = oracle.forward(Q, K, V, m, lam, T, grid=(gw, 0), dwc_branch=(w, b))
    np.testing.assert_allclose(both - base, oracle.dwc(V, w, b, gw), rtol=0, atol=1e-14)
    dQ, dK, dV, dW, db = oracle.backward(Q, K, V, dO, m, lam, T, grid=(gw, 0), dwc_branch=(w, b))
    dQ0, dK0, _ = oracle.backward(Q, K, V, dO, m, lam, T)
    assert np.array_equal(dQ, dQ0) and np.array_equal(dK, dK0)
    h = 1e-6
    f = lambda V_, w_, b_: float((oracle.forward(Q, K, V_, m, lam, T, grid=(gw, 0), dwc_branch=(w_, b_)) * dO).sum())
    for arr, grad, name in ((V, dV, "V"), (w, dW, "W"), (b, db, "b")):
        g = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args = {"V": V.copy(), "W": w.copy(), "b": b.copy()}
            args[name][idx] += h
            fp = f(args["V"], args["W"], args["b"])
            args[name][idx] -= 2 * h
            g[idx] = (fp - f(args["V"], args["W"], args["b"])) / (2 * h)
        assert np.abs(g - grad).max() / max(np.abs(g).max(), 1e-12) < 1e-7, name


def test_dwc_rejections(oracle_lib):
    rng = np.random.default_rng(7)
    V = rng.standard_normal((1, 1, 12, 2))
    for gw, k in ((5, 3), (0, 3), (4, 2), (4, 0), (-4, 3)):
        w = np.zeros((1, 2, max(k, 1), max(k, 1))) if k > 0 else np.zeros((1, 2, 0, 0))
        with pytest.raises(ValueError):
            oracle.dwc(V, w, None, gw)


# ----------------------------------------------------------------------------- m-space normalisation (R15)

def dense_whitened_attention(Q, K, V, lam, w):
    """Eq. (4) written out densely with a diagonal whitening over the keys:
    z_ij = w_j (g_ij - mean_j' g_ij') + 1/n, out = Z V."""
    G = np.exp(-np.abs(Q[:, None, :] - K[None, :, :]).sum(-1) / lam)
    n = K.shape[0]
    Z = (G - G.mean(axis=1, keepdims=True)) * w[None, :] + 1.0 / n
    return Z @ V


@pytest.mark.parametrize("n,d,lam", [(16, 8, math.sqrt(8)), (24, 4, 4.0)])
def test_mspace_landmarks_equal_tokens_is_dense_whitened_attention(oracle_lib, n, d, lam):
    """With m = n the landmarks are the keys, M = K_LL^-1 K_LK V = V once Newton-Schulz has
    converged, and the landmark-space embedding of Appendix B with diagonal w is Eq. (4) with
    the whitening diag(w) over the keys; w = 1 gives the inline normalisation."""
    rng = np.random.default_rng(n + d)
    Q, K, V = rand_qkv(rng, 1, 2, n, d)
    w = rng.uniform(0.5, 1.5, size=(2, n))
    out, it = oracle.forward(Q, K, V, n, lam, 60, oracle.NORM_MSPACE, intermediates=True, whiten=w)
    ones = oracle.forward(Q, K, V, n, lam, 60, oracle.NORM_MSPACE)
    inline = oracle.forward(Q, K, V, n, lam, 60, oracle.NORM_INLINE)
    for h in range(2):
        floor = 1e-15 * np.linalg.cond(it["W"][0, h]) * n
        assert rel(out[0, h], dense_whitened_attention(Q[0, h], K[0, h], V[0, h], lam, w[h])) < max(floor, 1e-12)
        assert rel(ones[0, h], dense_laplacian_attention(Q[0, h], K[0, h], V[0, h], lam, oracle.NORM_INLINE)) < max(floor, 1e-12)
        assert rel(ones[0, h], inline[0, h]) < max(floor, 1e-12)


def test_mspace_zero_whitening_gives_the_mean_landmark_row(oracle_lib):
    """w = 0 leaves only the 1/m offset: every output row is the mean of the rows of M[:, :d]."""
    rng = np.random.default_rng(31)
    n, d, m = 30, 3, 7
    Q, K, V = rand_qkv(rng, 2, 1, n, d)
    out, it = oracle.forward(Q, K, V, m, 1.5, 5, oracle.NORM_MSPACE, intermediates=True, whiten=np.zeros((1, m)))
    for b in range(2):
        mean_row = it["M"][b, 0, :, :d].mean(axis=0)
        np.testing.assert_allclose(out[b, 0], np.broadcast_to(mean_row, (n, d)), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("n,d,m,T,lam", [(13, 3, 5, 4, 1.5), (9, 5, 1, 2, 3.0), (12, 2, 12, 3, 2.0)])
def test_mspace_backward_matches_finite_differences(oracle_lib, n, d, m, T, lam):
    rng = np.random.default_rng(n * 7 + m)
    Q, K, V = rand_qkv(rng, 1, 2, n, d, 0.7)
    dO = rng.standard_normal(Q.shape)
    w = rng.uniform(0.3, 1.7, size=(2, m))
    assert fd_check(Q, K, V, dO, m, lam, T, oracle.NORM_MSPACE, whiten=w) < 1e-7
