"""Pins for the fp64 oracle: it is checked against things other than itself.

Each pin is a closed form, an invariant the paper states, brute force on tiny
inputs, exact rational arithmetic, or an independent library routine. The
``check_*`` helpers take the function under test as an argument so that the
mutation tests at the bottom can show that a planted mistake (in a copy of the
oracle, on the CPU) fails at least one pin.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from workloads import CONFIGS, make_custom_inputs, make_layer_inputs

GOLD = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.json")


def rel(a, b):
    a, b = np.asarray(a), np.asarray(b)
    if a.shape != b.shape:
        return float("inf")
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300))


def rand_attn(rng, M, N, Hq, Hkv, dh, kscale=1.0):
    Q = rng.standard_normal((M, Hq, dh))
    K = rng.standard_normal((Hkv, N, dh)) * kscale
    V = rng.standard_normal((Hkv, N, dh))
    return Q, K, V


# --------------------------------------------------------------------------- checks

def brute_attention(Q, K, V, scale):
    """Scalar loops: softmax attention written out term by term."""
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
    grp = Hq // Hkv
    O = [[0.0] * (Hq * dh) for _ in range(M)]
    for m in range(M):
        for h in range(Hq):
            g = h // grp
            s = [scale * sum(Q[m, h, c] * K[g, n, c] for c in range(dh)) for n in range(N)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for c in range(dh):
                O[m][h * dh + c] = sum(e[n] * V[g, n, c] for n in range(N)) / z
    return np.array(O)


def check_attention_bruteforce(attn):
    rng = np.random.default_rng(1)
    worst = 0.0
    for (M, N, Hq, Hkv, dh) in [(3, 5, 4, 2, 4), (2, 7, 6, 3, 3), (4, 1, 2, 1, 5)]:
        Q, K, V = rand_attn(rng, M, N, Hq, Hkv, dh)
        s = 0.37
        worst = max(worst, rel(attn(Q, K, V, s), brute_attention(Q, K, V, s)))
    return worst


def check_attention_sdpa(attn):
    """torch's scaled_dot_product_attention (float64, CPU) with KV heads repeated."""
    rng = np.random.default_rng(2)
    worst = 0.0
    for (M, N, Hq, Hkv, dh) in [(17, 33, 4, 2, 8), (9, 64, 28, 4, 16), (5, 40, 8, 8, 8)]:
        Q, K, V = rand_attn(rng, M, N, Hq, Hkv, dh, kscale=1.5)
        s = 1.0 / math.sqrt(dh)
        q = torch.from_numpy(Q).permute(1, 0, 2)                      # [Hq, M, dh]
        k = torch.from_numpy(K).repeat_interleave(Hq // Hkv, dim=0)   # [Hq, N, dh]
        v = torch.from_numpy(V).repeat_interleave(Hq // Hkv, dim=0)
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=s)
        ref = o.permute(1, 0, 2).reshape(M, Hq * dh).numpy()
        worst = max(worst, rel(attn(Q, K, V, s), ref))
    return worst


def brute_targets(Of, Oc, W, rho):
    M, d = Of.shape
    dout = W.shape[1]
    T = np.zeros((M, dout))
    for i in range(M):
        for j in range(dout):
            acc = 0.0
            for k in range(d):
                acc += W[k, j] * (Of[i, k] - Oc[i, k])
            if rho:
                acc += Of[i, j] - Oc[i, j]
            T[i, j] = acc
    return T


def check_targets(tg):
    rng = np.random.default_rng(3)
    Of, Oc = rng.standard_normal((5, 4)), rng.standard_normal((5, 4))
    W = rng.standard_normal((4, 4))
    return max(rel(tg(Of, Oc, W, r), brute_targets(Of, Oc, W, r)) for r in (0, 1))


def check_normal_equations(ne):
    """Eq. 9: sums of per-token outer products."""
    rng = np.random.default_rng(4)
    X, T = rng.standard_normal((7, 3)), rng.standard_normal((7, 2))
    G, C = ne(X, T)
    Gb = sum(np.outer(X[i], X[i]) for i in range(7))
    Cb = sum(np.outer(X[i], T[i]) for i in range(7))
    return max(rel(G, Gb), rel(C, Cb))


def frac_solve(A, B):
    """Exact Gauss-Jordan elimination over the rationals."""
    n = len(A)
    m = len(B[0])
    A = [row[:] + brow[:] for row, brow in zip(A, B)]
    for c in range(n):
        p = next(r for r in range(c, n) if A[r][c] != 0)
        A[c], A[p] = A[p], A[c]
        piv = A[c][c]
        A[c] = [x / piv for x in A[c]]
        for r in range(n):
            if r != c and A[r][c] != 0:
                f = A[r][c]
                A[r] = [x - f * y for x, y in zip(A[r], A[c])]
    return [row[n:n + m] for row in A]


def check_solve_rational(solve):
    """Eq. 8 on small integer data, solved exactly in rational arithmetic."""
    rng = np.random.default_rng(5)
    worst = 0.0
    for (rows, din, dout, lam) in [(4, 3, 2, Fraction(1, 3)), (2, 4, 3, Fraction(1, 10)),
                                   (6, 2, 5, Fraction(2))]:
        X = rng.integers(-3, 4, size=(rows, din))
        T = rng.integers(-3, 4, size=(rows, dout))
        Xf = [[Fraction(int(v)) for v in r] for r in X]
        Tf = [[Fraction(int(v)) for v in r] for r in T]
        A = [[sum(Xf[k][i] * Xf[k][j] for k in range(rows)) + (lam if i == j else 0)
              for j in range(din)] for i in range(din)]
        Bm = [[sum(Xf[k][i] * Tf[k][j] for k in range(rows)) for j in range(dout)]
              for i in range(din)]
        exact = np.array([[float(v) for v in r] for r in frac_solve(A, Bm)])
        G = X.T.astype(float) @ X
        C = X.T.astype(float) @ T
        worst = max(worst, rel(solve(G, C, float(lam)), exact))
    return worst


def check_solve_lstsq(solve):
    """Ridge = least squares on the augmented system [X; sqrt(lam) I] dW ~ [T; 0]."""
    rng = np.random.default_rng(6)
    worst = 0.0
    for (rows, din, dout, lam) in [(50, 20, 7, 0.3), (10, 30, 30, 1e-2)]:
        X, T = rng.standard_normal((rows, din)), rng.standard_normal((rows, dout))
        A = np.vstack([X, np.sqrt(lam) * np.eye(din)])
        Bm = np.vstack([T, np.zeros((din, dout))])
        ref = np.linalg.lstsq(A, Bm, rcond=None)[0]
        worst = max(worst, rel(solve(X.T @ X, X.T @ T, lam), ref))
    return worst


# --------------------------------------------------------------------------- pins

def test_golden_hand_worked():
    gold = json.load(open(GOLD))
    a = gold["attention_two_keys"]
    O = oracle.attention(np.array(a["Q"]), np.array(a["K"]), np.array(a["V"]), a["scale"])
    assert rel(O, a["O"]) < 1e-15
    t = gold["targets_eq5"]
    T = oracle.targets(np.array(t["Of"]), np.array(t["Oc"]), np.array(t["W"]), t["rho"])
    assert np.array_equal(T, np.array(t["T"]))
    r = gold["ridge_eq8"]
    G, C = oracle.normal_equations(np.array(r["X"]), np.array(r["T"]))
    assert np.array_equal(G, np.array(r["G"])) and np.array_equal(C, np.array(r["C"]))
    assert rel(oracle.solve_patch(G, C, r["lam"]), r["dW"]) < 1e-15
    ad = gold["adaptive_ridge_eq7"]
    assert abs(oracle.ridge_lambda(np.array(ad["G"]), ad["lam0"], "adaptive") - ad["lam"]) < 1e-16


def test_softmax_rows_library_and_sum():
    rng = np.random.default_rng(0)
    S = rng.standard_normal((64, 300)) * 20
    P = oracle.softmax_rows(S)
    assert rel(P, scipy.special.softmax(S, axis=1)) < 1e-14
    assert np.max(np.abs(P.sum(axis=1) - 1.0)) < 1e-15


def test_attention_bruteforce():
    assert check_attention_bruteforce(oracle.attention) < 1e-13


def test_attention_library_sdpa():
    assert check_attention_sdpa(oracle.attention) < 1e-13


def test_attention_closed_forms():
    rng = np.random.default_rng(7)
    M, Hq, Hkv, dh = 6, 4, 2, 8
    # one key: O = its V
    Q, K, V = rand_attn(rng, M, 1, Hq, Hkv, dh)
    O = oracle.attention(Q, K, V).reshape(M, Hq, dh)
    for h in range(Hq):
        assert np.allclose(O[:, h], V[h // 2, 0][None, :], atol=1e-15)
    # zero keys: uniform weights, O = mean of V
    Q, K, V = rand_attn(rng, M, 9, Hq, Hkv, dh)
    O = oracle.attention(Q, 0 * K, V).reshape(M, Hq, dh)
    for h in range(Hq):
        assert np.allclose(O[:, h], V[h // 2].mean(axis=0)[None, :], atol=1e-14)
    # a dominant key: O -> its V
    K = rng.standard_normal((Hkv, 9, dh)) * 1e-3
    Q = np.abs(rng.standard_normal((M, Hq, dh)))
    K[:, 4, :] = 1e3
    O = oracle.attention(Q, K, V).reshape(M, Hq, dh)
    for h in range(Hq):
        assert np.allclose(O[:, h], V[h // 2, 4][None, :], atol=1e-12)


def test_attention_invariances():
    rng = np.random.default_rng(8)
    Q, K, V = rand_attn(rng, 11, 50, 8, 2, 16)
    O = oracle.attention(Q, K, V)
    perm = rng.permutation(50)
    assert rel(oracle.attention(Q, K[:, perm], V[:, perm]), O) < 1e-14
    # GQA == MHA with each KV head repeated for its query heads
    Kr = np.repeat(K, 4, axis=0)
    Vr = np.repeat(V, 4, axis=0)
    assert rel(oracle.attention(Q, Kr, Vr), O) < 1e-15
    # row chunking changes nothing
    assert rel(oracle.attention(Q, K, V, max_score_bytes=8 * 50 * 3), O) == 0.0
    # attention_rows is the row subset
    rows = np.array([0, 5, 10])
    assert rel(oracle.attention_rows(Q, K, V, rows), O[rows]) == 0.0


def test_gather_cache():
    rng = np.random.default_rng(9)
    Q, K, V = rand_attn(rng, 5, 20, 4, 2, 8)
    Kg, Vg = oracle.gather_cache(K, V, np.arange(20))
    assert np.array_equal(Kg, K) and np.array_equal(Vg, V)
    idx = np.array([0, 3, 4, 19])
    Kg, Vg = oracle.gather_cache(K, V, idx)
    for j, n in enumerate(idx):
        assert np.array_equal(Kg[:, j], K[:, n]) and np.array_equal(Vg[:, j], V[:, n])


def test_targets_bruteforce_and_linearity():
    assert check_targets(oracle.targets) < 1e-15
    rng = np.random.default_rng(10)
    Of, Oc = rng.standard_normal((6, 5)), rng.standard_normal((6, 5))
    W1, W2 = rng.standard_normal((5, 5)), rng.standard_normal((5, 5))
    lin = oracle.targets(Of, Oc, W1 + W2, 0) - oracle.targets(Of, Oc, W1, 0) - oracle.targets(Of, Oc, W2, 0)
    assert np.max(np.abs(lin)) < 1e-13
    assert np.array_equal(oracle.targets(Of, Of, W1, 1), np.zeros((6, 5)))


def test_normal_equations_outer_products_and_chunks():
    assert check_normal_equations(oracle.normal_equations) < 1e-15
    rng = np.random.default_rng(11)
    X, T = rng.standard_normal((100, 12)), rng.standard_normal((100, 9))
    G, C = oracle.normal_equations(X, T)
    cuts = [0, 7, 8, 40, 99, 100]
    Gc, Cc = oracle.normal_equations_chunked((X[a:b], T[a:b]) for a, b in zip(cuts, cuts[1:]))
    assert rel(Gc, G) < 1e-14 and rel(Cc, C) < 1e-14
    assert np.array_equal(G, G.T)
    assert np.min(np.linalg.eigvalsh(G)) > -1e-12


def test_solve_rational_exact():
    assert check_solve_rational(oracle.solve_patch) < 1e-14


def test_solve_lstsq_library():
    assert check_solve_lstsq(oracle.solve_patch) < 1e-12


def test_solve_push_through_and_residual():
    rng = np.random.default_rng(12)
    X, T = rng.standard_normal((40, 60)), rng.standard_normal((40, 25))
    lam = 0.05
    G, C = oracle.normal_equations(X, T)
    dW = oracle.solve_patch(G, C, lam)
    push = X.T @ np.linalg.solve(X @ X.T + lam * np.eye(40), T)
    assert rel(dW, push) < 1e-11
    A = G + lam * np.eye(60)
    res = np.linalg.norm(A @ dW - C) / (np.linalg.norm(A) * np.linalg.norm(dW) + np.linalg.norm(C))
    assert res < 1e-15


def test_solve_closed_forms_and_limits():
    rng = np.random.default_rng(13)
    # d_in = 1: dW = sum x t / (sum x^2 + lam)
    x, t = rng.standard_normal((30, 1)), rng.standard_normal((30, 4))
    G, C = oracle.normal_equations(x, t)
    assert rel(oracle.solve_patch(G, C, 0.7), (x.T @ t) / (np.sum(x * x) + 0.7)) < 1e-15
    # diagonal G: dW = C / (diag + lam)
    Gd = np.diag(rng.uniform(0.5, 3.0, 6))
    Cd = rng.standard_normal((6, 3))
    assert rel(oracle.solve_patch(Gd, Cd, 0.2), Cd / (np.diag(Gd)[:, None] + 0.2)) < 1e-15
    # lambda -> infinity: dW -> 0 and lam dW -> C, with O(1/lam) error
    X, T = rng.standard_normal((20, 8)), rng.standard_normal((20, 5))
    G, C = oracle.normal_equations(X, T)
    errs = []
    for lam in (1e4, 1e6, 1e8):
        dW = oracle.solve_patch(G, C, lam)
        errs.append(rel(lam * dW, C))
        assert np.linalg.norm(dW) < 10 * np.linalg.norm(C) / lam
    assert errs[1] < errs[0] / 50 and errs[2] < errs[1] / 50
    # optimality: the ridge objective grows in every random direction
    lam = 0.3
    dW = oracle.solve_patch(G, C, lam)
    J = lambda D: np.sum((X @ D - T) ** 2) + lam * np.sum(D * D)
    for _ in range(5):
        E = rng.standard_normal(dW.shape) * 1e-3
        assert J(dW + E) > J(dW) and J(dW - E) > J(dW)
    assert J(dW) < J(np.zeros_like(dW))


def test_solve_scaling_laws():
    rng = np.random.default_rng(14)
    X, T = rng.standard_normal((30, 10)), rng.standard_normal((30, 4))
    G, C = oracle.normal_equations(X, T)
    dW = oracle.solve_patch(G, C, 0.5)
    a = 3.0
    G2, C2 = oracle.normal_equations(a * X, T)
    assert rel(oracle.solve_patch(G2, C2, a * a * 0.5), dW / a) < 1e-13
    G3, C3 = oracle.normal_equations(X, a * T)
    assert rel(oracle.solve_patch(G3, C3, 0.5), a * dW) < 1e-14
    # adaptive ridge (Eq. 7): dW(aX) = dW(X) / a with lambda_0 fixed
    lam_a = oracle.ridge_lambda(G, 0.1, "adaptive")
    lam_b = oracle.ridge_lambda(G2, 0.1, "adaptive")
    assert abs(lam_b / lam_a - a * a) < 1e-12
    assert rel(oracle.solve_patch(G2, C2, lam_b), oracle.solve_patch(G, C, lam_a) / a) < 1e-13
    # the trace-mean scaling has the same invariance
    lam_a = oracle.ridge_lambda(G, 0.1, "trace_mean")
    lam_b = oracle.ridge_lambda(G2, 0.1, "trace_mean")
    assert abs(lam_b / lam_a - a * a) < 1e-12
    assert rel(oracle.solve_patch(G2, C2, lam_b), oracle.solve_patch(G, C, lam_a) / a) < 1e-13
    with pytest.raises(ValueError):
        oracle.solve_patch(G, C, 0.0)


def test_ridge_scalings_closed_forms():
    """Eq. 7 and the trace mean by hand on a 2 x 2 G; both equal lambda_0 c on G = c I
    (every eigenvalue c: the mean and the eigenvalue-weighted mean coincide)."""
    G = np.array([[2.0, 1.0], [1.0, 4.0]])
    assert oracle.ridge_lambda(G, 0.5, "adaptive") == 0.5 * (4 + 1 + 1 + 16) / 6
    assert oracle.ridge_lambda(G, 0.5, "trace_mean") == 0.5 * 6 / 2
    assert oracle.ridge_lambda(G, 0.5, "absolute") == 0.5
    c, lam0 = 7.0, 0.01
    Gc = c * np.eye(5)
    assert abs(oracle.ridge_lambda(Gc, lam0, "adaptive") - lam0 * c) < 1e-15
    assert abs(oracle.ridge_lambda(Gc, lam0, "trace_mean") - lam0 * c) < 1e-15
    with pytest.raises(ValueError):
        oracle.ridge_lambda(G, 0.5, "spectral")


def test_layer_patch_identity_cache_gives_zero_patch():
    """Compressed cache == full cache => T = 0 => C = 0 => dW = 0 exactly."""
    inp = make_custom_inputs(M=24, N=40, B=40, Hq=4, Hkv=2, dh=8, dtype="bf16",
                             cache="identity", seed=3)
    out = oracle.layer_patch(inp)
    assert np.max(np.abs(out["dW"])) == 0.0
    assert np.max(np.abs(out["T"])) == 0.0


def test_layer_patch_config0_properties():
    cfg = CONFIGS[0]
    inp = make_layer_inputs(cfg)
    out = oracle.layer_patch(inp)
    dW, G, C, lam = out["dW"], out["G"], out["C"], out["lam"]
    assert dW.shape == (cfg.d, cfg.d) and np.all(np.isfinite(dW))
    A = G + lam * np.eye(cfg.d)
    res = np.linalg.norm(A @ dW - C) / (np.linalg.norm(A) * np.linalg.norm(dW) + np.linalg.norm(C))
    assert res < 1e-15
    push = out["Oc"].T @ np.linalg.solve(out["Oc"] @ out["Oc"].T + lam * np.eye(cfg.M), out["T"])
    assert rel(dW, push) < 1e-9
    # chunked accumulation over the reference tokens gives the same patch
    Gc, Cc = oracle.normal_equations_chunked(
        (out["Oc"][a:a + 40], out["T"][a:a + 40]) for a in range(0, cfg.M, 40))
    assert rel(oracle.solve_patch(Gc, Cc, lam), dW) < 1e-10
    # the compressed cache is the sorted eviction subset of the recipe
    idx = inp.idx
    assert idx.shape == (cfg.B,) and np.all(np.diff(idx) > 0)
    assert list(idx[:4]) == [0, 1, 2, 3] and list(idx[-cfg.n_recent:]) == list(range(cfg.N - cfg.n_recent, cfg.N))


def test_synthesized_cache_is_convex_mix():
    inp = make_custom_inputs(M=8, N=100, B=6, Hq=4, Hkv=2, dh=8, dtype="f32",
                             cache="synthesize", n_mix=5, seed=1)
    pos, w = inp.extra["syn_pos"], inp.extra["syn_w"]
    assert np.allclose(w.sum(axis=1), 1.0) and np.all(w > 0)
    assert all(len(set(p)) == 5 for p in pos)
    K = inp.K.astype(np.float64)
    for g in range(2):
        for b in range(6):
            assert np.allclose(inp.Kc[g, b], w[b] @ K[g, pos[b]], rtol=1e-6, atol=1e-6)


# --------------------------------------------------------------------------- mutations

def test_pins_catch_planted_mistakes():
    """Copies of oracle functions with one planted mistake each fail a pin."""
    def attn_wrong_group(Q, K, V, scale=None):
        M, Hq, dh = Q.shape
        Hkv = K.shape[0]
        O = np.empty((M, Hq * dh))
        for h in range(Hq):
            g = h % Hkv                                # wrong GQA mapping
            S = Q[:, h, :] @ K[g].T * scale
            O[:, h * dh:(h + 1) * dh] = oracle.softmax_rows(S) @ V[g]
        return O

    def attn_no_scale(Q, K, V, scale=None):
        return oracle.attention(Q, K, V, 1.0)         # scale dropped

    def targets_no_residual(Of, Oc, W, rho=1):
        return (Of - Oc) @ W                          # residual term dropped

    def targets_transposed(Of, Oc, W, rho=1):
        return (Of - Oc) @ W.T + rho * (Of - Oc)      # transposed operand

    def ne_transposed(X, T):
        return X.T @ X, T.T @ X                        # wrong orientation

    def solve_no_ridge(G, C, lam):
        return np.linalg.lstsq(G, C, rcond=None)[0]   # lambda dropped

    def solve_sign(G, C, lam):
        return np.linalg.solve(G - lam * np.eye(G.shape[0]), C)   # wrong sign

    assert check_attention_bruteforce(attn_wrong_group) > 1e-2
    assert check_attention_bruteforce(attn_no_scale) > 1e-2
    assert check_targets(targets_no_residual) > 1e-2
    assert check_targets(targets_transposed) > 1e-2
    assert check_normal_equations(ne_transposed) > 1e-2
    assert check_solve_rational(solve_no_ridge) > 1e-3
    assert check_solve_rational(solve_sign) > 1e-3


# ------------------------------------------------------- chunked reference set (f2)

def brute_attention_chunk(Q, K, V, Ks, Vs, scale):
    """Scalar loops: query m of the chunk sees every cache entry and its own
    entries 0..m, written out term by term."""
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
    grp = Hq // Hkv
    O = np.zeros((M, Hq * dh))
    for m in range(M):
        for h in range(Hq):
            g = h // grp
            keys = [K[g, n] for n in range(N)] + [Ks[g, j] for j in range(m + 1)]
            vals = [V[g, n] for n in range(N)] + [Vs[g, j] for j in range(m + 1)]
            s = [scale * sum(Q[m, h, c] * k[c] for c in range(dh)) for k in keys]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for c in range(dh):
                O[m, h * dh + c] = sum(e[i] * vals[i][c] for i in range(len(e))) / z
    return O


def rand_chunk(rng, M, N, Hq, Hkv, dh):
    Q, K, V = rand_attn(rng, M, N, Hq, Hkv, dh)
    Ks = rng.standard_normal((Hkv, M, dh))
    Vs = rng.standard_normal((Hkv, M, dh))
    return Q, K, V, Ks, Vs


def check_attention_chunk_bruteforce(fn):
    rng = np.random.default_rng(11)
    worst = 0.0
    for (M, N, Hq, Hkv, dh) in [(4, 5, 4, 2, 3), (3, 0, 2, 1, 4), (5, 2, 6, 3, 2), (1, 3, 2, 2, 3)]:
        Q, K, V, Ks, Vs = rand_chunk(rng, M, N, Hq, Hkv, dh)
        worst = max(worst, rel(fn(Q, K, V, Ks, Vs, 0.41), brute_attention_chunk(Q, K, V, Ks, Vs, 0.41)))
    return worst


def test_attention_chunk_bruteforce():
    assert check_attention_chunk_bruteforce(oracle.attention_chunk) < 1e-13


def test_attention_chunk_empty_cache_is_causal_sdpa():
    """With no cache entries a chunk is plain causal self-attention: torch's
    scaled_dot_product_attention(is_causal=True), float64 on the CPU."""
    rng = np.random.default_rng(12)
    for (M, Hq, Hkv, dh) in [(23, 4, 2, 8), (40, 8, 8, 16)]:
        Q, K, V, Ks, Vs = rand_chunk(rng, M, 0, Hq, Hkv, dh)
        s = 1.0 / math.sqrt(dh)
        q = torch.from_numpy(Q).permute(1, 0, 2)
        k = torch.from_numpy(Ks).repeat_interleave(Hq // Hkv, dim=0)
        v = torch.from_numpy(Vs).repeat_interleave(Hq // Hkv, dim=0)
        o = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True, scale=s)
        ref = o.permute(1, 0, 2).reshape(M, Hq * dh).numpy()
        assert rel(oracle.attention_chunk(Q, K, V, Ks, Vs, s), ref) < 1e-13


def test_attention_chunk_rows_reduce_to_plain_attention():
    """Row m equals the (pinned) unmasked attention of that one query over the
    cache followed by the chunk's entries 0..m."""
    rng = np.random.default_rng(13)
    Q, K, V, Ks, Vs = rand_chunk(rng, 9, 30, 8, 2, 16)
    O = oracle.attention_chunk(Q, K, V, Ks, Vs)
    for m in range(9):
        Kc = np.concatenate([K, Ks[:, :m + 1]], axis=1)
        Vc = np.concatenate([V, Vs[:, :m + 1]], axis=1)
        assert rel(O[m:m + 1], oracle.attention(Q[m:m + 1], Kc, Vc)) < 1e-14


def test_attention_chunk_causality_and_prefix():
    rng = np.random.default_rng(14)
    Q, K, V, Ks, Vs = rand_chunk(rng, 12, 20, 4, 2, 8)
    O = oracle.attention_chunk(Q, K, V, Ks, Vs)
    # own entries after position 5 cannot reach queries 0..5, and do reach the rest
    Ks2, Vs2 = Ks.copy(), Vs.copy()
    Ks2[:, 6:] += 3.0
    Vs2[:, 6:] -= 2.0
    O2 = oracle.attention_chunk(Q, K, V, Ks2, Vs2)
    assert np.array_equal(O2[:6], O[:6])
    assert np.all(np.abs(O2[6:] - O[6:]).max(axis=1) > 1e-6)
    # a chunk's prefix is itself a chunk
    assert rel(oracle.attention_chunk(Q[:7], K, V, Ks[:, :7], Vs[:, :7]), O[:7]) < 1e-15
    # rows sum to one: all-ones values give all-ones outputs
    O1 = oracle.attention_chunk(Q, K, np.ones_like(V), Ks, np.ones_like(Vs))
    assert np.max(np.abs(O1 - 1.0)) < 1e-14


def test_layer_patch_chunked_properties():
    from workloads import make_chunk_inputs
    inp = make_custom_inputs(M=16, N=96, B=96, Hq=4, Hkv=2, dh=16, dtype="f32",
                             cache="identity", lam=1e-2, seed=5)
    chunks = [make_chunk_inputs(inp, j, 16) for j in range(3)]
    triples = [(c.Q, c.Ks, c.Vs) for c in chunks]
    # compressed cache == full cache: teacher and student agree, Delta W = 0 exactly
    out = oracle.layer_patch_chunked(inp, triples)
    assert np.array_equal(out["dW"], np.zeros_like(out["dW"]))
    # eviction cache: the statistics are the sums over chunks of each chunk's own
    # outer products (Eq. 9), and the patch solves the stacked regression
    inp = make_custom_inputs(M=16, N=96, B=40, Hq=4, Hkv=2, dh=16, dtype="f32", lam=1e-2, seed=6)
    chunks = [make_chunk_inputs(inp, j, 16) for j in range(3)]
    out = oracle.layer_patch_chunked(inp, [(c.Q, c.Ks, c.Vs) for c in chunks])
    K, V = oracle.decode(inp.K, "f32"), oracle.decode(inp.V, "f32")
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    W = oracle.decode(inp.W, "f32")
    X, T = [], []
    for c in chunks:
        Q, Ks, Vs = (oracle.decode(a, "f32") for a in (c.Q, c.Ks, c.Vs))
        Of = brute_attention_chunk(Q, K, V, Ks, Vs, inp.scale)
        Oc = brute_attention_chunk(Q, Kc, Vc, Ks, Vs, inp.scale)
        X.append(Oc)
        T.append((Of - Oc) @ W + (Of - Oc))
    X, T = np.vstack(X), np.vstack(T)
    Gs = sum(np.outer(X[i], X[i]) for i in range(X.shape[0]))
    Cs = sum(np.outer(X[i], T[i]) for i in range(X.shape[0]))
    assert rel(out["G"], Gs) < 1e-12 and rel(out["C"], Cs) < 1e-12
    A = np.vstack([X, np.sqrt(1e-2) * np.eye(X.shape[1])])
    Bm = np.vstack([T, np.zeros((X.shape[1], T.shape[1]))])
    assert rel(out["dW"], np.linalg.lstsq(A, Bm, rcond=None)[0]) < 1e-9


def test_chunk_pins_catch_planted_mistakes():
    def no_self(Q, K, V, Ks, Vs, scale=None):           # own prefix excludes the token itself
        M = Q.shape[0]
        O = np.empty((M, Q.shape[1] * Q.shape[2]))
        for m in range(M):
            Kc = np.concatenate([K, Ks[:, :m]], axis=1)
            Vc = np.concatenate([V, Vs[:, :m]], axis=1)
            if Kc.shape[1] == 0:
                Kc, Vc = Ks[:, :1], Vs[:, :1]
            O[m] = oracle.attention(Q[m:m + 1], Kc, Vc, scale)[0]
        return O

    def no_mask(Q, K, V, Ks, Vs, scale=None):           # the whole chunk is visible
        return oracle.attention(Q, np.concatenate([K, Ks], 1), np.concatenate([V, Vs], 1), scale)

    def own_from_cache_values(Q, K, V, Ks, Vs, scale=None):   # own keys paired with wrong values
        return oracle.attention_chunk(Q, K, V, Ks, Vs[:, ::-1], scale)

    assert check_attention_chunk_bruteforce(no_self) > 1e-2
    assert check_attention_chunk_bruteforce(no_mask) > 1e-2
    assert check_attention_chunk_bruteforce(own_from_cache_values) > 1e-2


# ------------------------------------------------------------ MLP-shaped patch (f3)

def brute_mlp_features(Z, Wg, Wu, eps):
    M, d = Z.shape
    d_ff = Wg.shape[1]
    H = np.zeros((M, d_ff))
    for i in range(M):
        r = math.sqrt(sum(Z[i, k] ** 2 for k in range(d)) / d + eps)
        u = [Z[i, k] / r for k in range(d)]
        for j in range(d_ff):
            g = sum(u[k] * Wg[k, j] for k in range(d))
            up = sum(u[k] * Wu[k, j] for k in range(d))
            H[i, j] = g / (1.0 + math.exp(-g)) * up
    return H


def check_mlp_features(fn):
    rng = np.random.default_rng(31)
    Z = rng.standard_normal((5, 6)) * 0.3
    Wg, Wu = rng.standard_normal((6, 7)), rng.standard_normal((6, 7))
    return rel(fn(Z, Wg, Wu, 1e-5), brute_mlp_features(Z, Wg, Wu, 1e-5))


def check_block_targets(fn):
    rng = np.random.default_rng(32)
    Hf, Hc = rng.standard_normal((4, 6)), rng.standard_normal((4, 6))
    Zf, Zc = rng.standard_normal((4, 3)), rng.standard_normal((4, 3))
    W = rng.standard_normal((6, 3))
    ref = np.array([[sum(W[k, j] * (Hf[i, k] - Hc[i, k]) for k in range(6)) + Zf[i, j] - Zc[i, j]
                     for j in range(3)] for i in range(4)])
    return rel(fn(Hf, Hc, W, Zf, Zc), ref)


def test_silu_and_rms_norm_library_and_closed_forms():
    x = np.linspace(-30, 30, 601)
    assert rel(oracle.silu(x), x * scipy.special.expit(x)) < 1e-15
    assert oracle.silu(np.zeros(1))[0] == 0.0
    assert rel(oracle.silu(-x), oracle.silu(x) - x) < 1e-13          # silu(-x) = silu(x) - x
    rng = np.random.default_rng(33)
    Z = rng.standard_normal((9, 40)) * 3
    ref = torch.nn.functional.rms_norm(torch.from_numpy(Z), (40,), eps=1e-5).numpy()
    assert rel(oracle.rms_norm(Z, 1e-5), ref) < 1e-15
    # unit gain: the output's mean square is ms / (ms + eps)
    U = oracle.rms_norm(Z, 1e-5)
    ms = np.mean(Z * Z, axis=1)
    assert np.max(np.abs(np.mean(U * U, axis=1) - ms / (ms + 1e-5))) < 1e-14


def test_mlp_features_bruteforce_and_library():
    assert check_mlp_features(oracle.mlp_features) < 1e-13
    rng = np.random.default_rng(34)
    Z = rng.standard_normal((20, 32))
    Wg, Wu = rng.standard_normal((32, 48)) / 6, rng.standard_normal((32, 48)) / 6
    F = torch.nn.functional
    z = torch.from_numpy(Z)
    u = F.rms_norm(z, (32,), eps=1e-5)
    ref = (F.silu(u @ torch.from_numpy(Wg)) * (u @ torch.from_numpy(Wu))).numpy()
    assert rel(oracle.mlp_features(Z, Wg, Wu), ref) < 1e-14


def test_block_targets_bruteforce():
    assert check_block_targets(oracle.block_targets) < 1e-14


def test_mlp_layer_patch_properties():
    from workloads import make_mlp_weights
    # compressed cache == full cache: no correction, the student already matches
    inp = make_custom_inputs(M=12, N=80, B=80, Hq=4, Hkv=2, dh=8, dtype="f32", cache="identity",
                             lam=1e-2, seed=3)
    mlp = make_mlp_weights(inp, 48)
    out = oracle.mlp_layer_patch(inp, mlp)
    assert np.array_equal(out["dW"], np.zeros((48, 32)))
    assert np.array_equal(out["Y_student"], out["Y_teacher"])
    # fewer tokens than features: the per-token condition (Eq. 4) can be met exactly,
    # so as lambda -> 0 the patched student's output reaches the teacher's, O(lambda)
    inp = make_custom_inputs(M=12, N=80, B=20, Hq=4, Hkv=2, dh=8, dtype="f32", lam=1e-2, seed=4)
    mlp = make_mlp_weights(inp, 48)
    gaps = []
    for lam in (1e-2, 1e-4, 1e-6):
        out = oracle.mlp_layer_patch(inp, mlp, lam=lam)
        gaps.append(rel(out["Y_student"], out["Y_teacher"]))
    assert gaps[0] > gaps[1] > gaps[2] and gaps[2] < 1e-6 and gaps[1] < 2e-2 * gaps[0]
    # the patch solves its normal equations and agrees with the push-through form
    # Hc^T (Hc Hc^T + lambda I)^{-1} T, a different route through the same algebra
    out = oracle.mlp_layer_patch(inp, mlp, lam=1e-2)
    Q, K, V = (oracle.decode(a, "f32") for a in (inp.Q, inp.K, inp.V))
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    Wg, Wu, Wd = (oracle.decode(a, "f32") for a in (mlp.Wg, mlp.Wu, mlp.Wd))
    Of = oracle.attention(Q, K, V, inp.scale)
    Oc = oracle.attention(Q, Kc, Vc, inp.scale)
    Hf, Hc = oracle.mlp_features(Of, Wg, Wu), oracle.mlp_features(Oc, Wg, Wu)
    T = (Hf - Hc) @ Wd + (Of - Oc)
    assert rel(out["G"], Hc.T @ Hc) < 1e-14 and rel(out["C"], Hc.T @ T) < 1e-14
    resid = (out["G"] + 1e-2 * np.eye(48)) @ out["dW"] - out["C"]
    assert np.linalg.norm(resid) / np.linalg.norm(out["C"]) < 1e-12
    push = Hc.T @ np.linalg.solve(Hc @ Hc.T + 1e-2 * np.eye(12), T)
    assert rel(out["dW"], push) < 1e-10
    assert rel(out["Y_student"], Hc @ (Wd + out["dW"]) + Oc) < 1e-15


def test_mlp_pins_catch_planted_mistakes():
    def feats_wrong_sign(Z, Wg, Wu, eps=1e-5):        # silu with e^{+x}
        U = oracle.rms_norm(Z, eps)
        G = U @ Wg
        return G / (1.0 + np.exp(G)) * (U @ Wu)

    def feats_no_norm(Z, Wg, Wu, eps=1e-5):           # RMS norm dropped
        return oracle.silu(Z @ Wg) * (Z @ Wu)

    def feats_swapped(Z, Wg, Wu, eps=1e-5):           # gate and up swapped
        return oracle.mlp_features(Z, Wu, Wg, eps)

    def targets_no_residual(Hf, Hc, W, Zf, Zc):
        return (Hf - Hc) @ W

    def targets_student_weights(Hf, Hc, W, Zf, Zc):   # residual sign flipped
        return (Hf - Hc) @ W - (Zf - Zc)

    assert check_mlp_features(feats_wrong_sign) > 1e-2
    assert check_mlp_features(feats_no_norm) > 1e-2
    assert check_mlp_features(feats_swapped) > 1e-2
    assert check_block_targets(targets_no_residual) > 1e-2
    assert check_block_targets(targets_student_weights) > 1e-2


# ------------------------------------------- compressed-cache formats (f4): bias, MX int

def brute_attention_bias(Q, K, V, scale, bias):
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
    grp = Hq // Hkv
    O = np.zeros((M, Hq * dh))
    for m in range(M):
        for h in range(Hq):
            g = h // grp
            s = [scale * sum(Q[m, h, c] * K[g, n, c] for c in range(dh)) + bias[g, n] for n in range(N)]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            for c in range(dh):
                O[m, h * dh + c] = sum(e[n] * V[g, n, c] for n in range(N)) / sum(e)
    return O


def test_attention_bias_bruteforce_and_closed_forms():
    rng = np.random.default_rng(51)
    Q, K, V = rand_attn(rng, 3, 6, 4, 2, 3)
    bias = rng.standard_normal((2, 6))
    assert rel(oracle.attention(Q, K, V, 0.3, bias=bias), brute_attention_bias(Q, K, V, 0.3, bias)) < 1e-13
    # a bias constant per KV head changes nothing (softmax shift invariance)
    Q, K, V = rand_attn(rng, 7, 20, 8, 2, 8)
    O = oracle.attention(Q, K, V)
    const = np.repeat(np.array([[3.0], [-2.0]]), 20, axis=1)
    assert rel(oracle.attention(Q, K, V, bias=const), O) < 1e-14
    # zero keys: the weights are exactly e^bias, O = the bias-weighted mean of V
    w = rng.random((2, 20)) + 0.1
    Ob = oracle.attention(Q, 0 * K, V, bias=np.log(w)).reshape(7, 8, 8)
    for h in range(8):
        g = h // 4
        ref = (w[g][:, None] * V[g]).sum(0) / w[g].sum()
        assert np.allclose(Ob[:, h], ref[None, :], atol=1e-14)
    # a bias of log(k) on an entry equals k copies of that entry
    b = np.zeros((2, 20))
    b[:, 5] = np.log(3.0)
    K3 = np.concatenate([K, K[:, 5:6], K[:, 5:6]], axis=1)
    V3 = np.concatenate([V, V[:, 5:6], V[:, 5:6]], axis=1)
    assert rel(oracle.attention(Q, K, V, bias=b), oracle.attention(Q, K3, V3)) < 1e-14


def test_dequantize_mx_library_and_exactness():
    from workloads import bf16_bits_to_f32, bf16_round_bits, quantize_mx
    rng = np.random.default_rng(52)
    q = rng.integers(-127, 128, size=(3, 4, 64)).astype(np.int8)
    e = rng.integers(-20, 5, size=(3, 4, 2)).astype(np.int8)
    d = oracle.dequantize_mx(q, e)
    assert np.array_equal(d, np.ldexp(q.astype(np.float64), np.repeat(e, 32, axis=-1).astype(np.int64)))
    # int8 magnitudes times powers of two are bf16 numbers: the round trip is exact
    f = d.astype(np.float32)
    assert np.array_equal(bf16_bits_to_f32(bf16_round_bits(f)), f)
    # the quantizer of the inputs stays within half a step of the value
    x = rng.standard_normal((2, 9, 128)).astype(np.float32) * 3
    for bits in (8, 4):
        qq, ee = quantize_mx(x, bits)
        step = np.exp2(np.repeat(ee.astype(np.float64), 32, axis=-1))
        assert np.all(np.abs(oracle.dequantize_mx(qq, ee) - x) <= 0.5 * step + 1e-12)


# ----------------------------------------------------------- low-rank patch (f4)

def _rrr_case(rng, rows=60, din=24, dout=16, planted=None):
    X = rng.standard_normal((rows, din))
    if planted is None:
        dW = rng.standard_normal((din, dout))
    else:  # a strong rank-`planted` part plus noise: a clear gap after eigenvalue `planted`
        dW = rng.standard_normal((din, planted)) @ rng.standard_normal((planted, dout)) * 3
        dW += 0.01 * rng.standard_normal((din, dout))
    return X, X.T @ X, dW


def check_low_rank(fn):
    """The reduced-rank fit loses exactly the discarded eigenvalues: with Yhat = X dW,
    ||X (dW - dW_r)||_F^2 = sum of the eigenvalues of Yhat^T Yhat past r, the optimum
    over all rank-r output projections (Eckart-Young on the fitted targets)."""
    rng = np.random.default_rng(61)
    X, G, dW = _rrr_case(rng)
    r = 5
    out = fn(G, dW, r)
    s = np.linalg.svd(X @ dW, compute_uv=False)
    lost = np.linalg.norm(X @ (dW - out["dW"])) ** 2
    return abs(lost - np.sum(s[r:] ** 2)) / np.sum(s ** 2)


def test_low_rank_patch_optimal_loss_and_rank():
    assert check_low_rank(oracle.low_rank_patch) < 1e-12
    rng = np.random.default_rng(62)
    X, G, dW = _rrr_case(rng)
    out = oracle.low_rank_patch(G, dW, 5)
    assert np.linalg.matrix_rank(out["dW"], tol=1e-9 * np.linalg.norm(dW)) == 5
    assert rel(out["A"] @ out["U"].T, out["dW"]) < 1e-14
    assert np.max(np.abs(out["U"].T @ out["U"] - np.eye(5))) < 1e-13
    # full rank keeps the patch
    assert rel(oracle.low_rank_patch(G, dW, 16)["dW"], dW) < 1e-13
    # no other rank-5 output projection fits better
    best = np.linalg.norm(X @ (dW - out["dW"])) ** 2
    for _ in range(20):
        P, _ = np.linalg.qr(rng.standard_normal((16, 5)))
        assert np.linalg.norm(X @ (dW - dW @ P @ P.T)) ** 2 >= best * (1 - 1e-12)


def test_low_rank_patch_matches_svd_of_fitted_targets():
    """With a clear gap, the projector is the one of the top right singular vectors
    of the fitted targets X dW (numpy SVD, a different route)."""
    rng = np.random.default_rng(63)
    X, G, dW = _rrr_case(rng, planted=4)
    out = oracle.low_rank_patch(G, dW, 4)
    _, _, Vt = np.linalg.svd(X @ dW)
    P = Vt[:4].T @ Vt[:4]
    assert rel(out["dW"], dW @ P) < 1e-10


def test_low_rank_pins_catch_planted_mistakes():
    def bottom(G, dW, r):                       # smallest eigenvalues kept
        w, V = np.linalg.eigh(dW.T @ G @ dW)
        U = V[:, :r]
        return {"dW": dW @ U @ U.T}

    def no_gram(G, dW, r):                      # S_H dropped: eigenvectors of dW^T dW
        w, V = np.linalg.eigh(dW.T @ dW)
        U = V[:, ::-1][:, :r]
        return {"dW": dW @ U @ U.T}

    def truncated_svd(G, dW, r):                # best rank-r approximation of dW itself
        U, s, Vt = np.linalg.svd(dW, full_matrices=False)
        return {"dW": (U[:, :r] * s[:r]) @ Vt[:r]}

    for f in (bottom, no_gram, truncated_svd):
        assert check_low_rank(f) > 1e-4


# ------------------------------------------- stored-input decoding and block composition

def check_decode_bf16(dec) -> bool:
    """Hand-written bf16 bit patterns decode to their values, and a random array decodes
    as torch's own bfloat16 reinterpretation of the same bits does."""
    cases = [(0x3F80, 1.0), (0xC000, -2.0), (0x3E80, 0.25), (0x4049, 3.140625),
             (0x7F7F, (2.0 - 2.0 ** -7) * 2.0 ** 127),     # largest finite bf16
             (0x0080, 2.0 ** -126),                      # smallest normal
             (0x0001, 2.0 ** -133),                      # smallest subnormal
             (0x8000, -0.0), (0x7F80, math.inf), (0xFF80, -math.inf)]
    bits = np.array([c[0] for c in cases], dtype=np.uint16)
    got = np.asarray(dec(bits, "bf16"), dtype=np.float64)
    want = np.array([c[1] for c in cases])
    ok = got.shape == want.shape and bool(np.array_equal(got, want))
    ok = ok and bool(np.signbit(got[7])) and not bool(np.signbit(got[0]))
    rnd = np.random.default_rng(77).integers(0, 1 << 16, size=4096, dtype=np.uint16)
    rnd = rnd[(rnd & 0x7F80) != 0x7F80]                 # finite values (no inf / NaN)
    ref = torch.from_numpy(rnd.view(np.int16).copy()).view(torch.bfloat16).double().numpy()
    got = np.asarray(dec(rnd, "bf16"), dtype=np.float64)
    return ok and got.shape == ref.shape and bool(np.array_equal(got, ref))


def test_decode_bf16_bit_patterns_and_torch_view():
    assert check_decode_bf16(oracle.decode)
    x = np.random.default_rng(78).standard_normal(257).astype(np.float32)
    assert np.array_equal(oracle.decode(x, "f32"), x.astype(np.float64))


def _torch_decode(a, dtype):
    """Stored input -> float64 through torch's own bf16 type (not the oracle's decode)."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
        return t.double().numpy()
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def _composed_patch(inp, rho):
    """One block's patch composed from independently written pieces (Eq. 4-6):
    scalar-loop attention for both caches, each token's block output y = h W + rho z
    under either cache, the per-token target as the block-output discrepancy of
    Eq. 4 (teacher minus student), and Eq. 6 as a stacked least-squares problem."""
    dt = inp.dtype
    Q, K, V, W = (_torch_decode(a, dt) for a in (inp.Q, inp.K, inp.V, inp.W))
    if inp.idx is not None:
        Kc = np.stack([[K[g, n] for n in inp.idx] for g in range(inp.Hkv)])
        Vc = np.stack([[V[g, n] for n in inp.idx] for g in range(inp.Hkv)])
    else:
        Kc, Vc = _torch_decode(inp.Kc, dt), _torch_decode(inp.Vc, dt)
    Hf = brute_attention(Q, K, V, inp.scale)            # teacher features h (and z)
    Hc = brute_attention(Q, Kc, Vc, inp.scale)          # student features h' (and z')
    Yf = np.array([h @ W + rho * h for h in Hf])        # teacher block outputs
    Yc = np.array([h @ W + rho * h for h in Hc])        # unpatched student block outputs
    T = Yf - Yc
    d = W.shape[0]
    A = np.vstack([Hc, np.sqrt(inp.lam) * np.eye(d)])
    Bm = np.vstack([T, np.zeros((d, W.shape[1]))])
    dW = np.linalg.lstsq(A, Bm, rcond=None)[0]
    return dW, Hc, Yf, Yc, W


def check_layer_patch(fn) -> float:
    """Worst relative error of fn(inp, rho)["dW"] against the composed patch over both
    cache kinds, both input dtypes and rho in {0, 1}; a patch that does not move the
    student's block output toward the teacher's scores inf."""
    worst = 0.0
    for k, (cache, dt) in enumerate([("evict", "bf16"), ("synthesize", "f32"),
                                     ("evict", "f32"), ("synthesize", "bf16")]):
        inp = make_custom_inputs(M=6, N=11, B=4, Hq=4, Hkv=2, dh=4, dtype=dt, cache=cache,
                                 n_mix=3, lam=0.05, seed=40 + k)
        for rho in (0, 1):
            ref, Hc, Yf, Yc, W = _composed_patch(inp, rho)
            got = fn(inp, rho)["dW"]
            worst = max(worst, rel(got, ref))
            patched = Hc @ (W + got) + rho * Hc
            if not np.linalg.norm(patched - Yf) < np.linalg.norm(Yc - Yf):
                return math.inf
    return worst


def test_layer_patch_composed_from_independent_pieces():
    assert check_layer_patch(lambda inp, rho: oracle.layer_patch(inp, rho=rho)) < 1e-10


def test_decode_and_layer_patch_pins_catch_planted_mistakes():
    def decode_shift15(x, dtype):
        a = np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(15)
        with np.errstate(invalid="ignore"):
            return a.view(np.float32).astype(np.float64)    # wrong shift

    def decode_half(x, dtype):
        return np.ascontiguousarray(x, dtype=np.uint16).view(np.float16).astype(np.float64)

    def layer_patch_swapped(inp, rho):
        dt = inp.dtype
        Q, K, V, W = (oracle.decode(a, dt) for a in (inp.Q, inp.K, inp.V, inp.W))
        Kc, Vc = (oracle.gather_cache(K, V, inp.idx) if inp.idx is not None
                  else (oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)))
        Of = oracle.attention(Q, K, V, inp.scale)
        Oc = oracle.attention(Q, Kc, Vc, inp.scale)
        T = oracle.targets(Oc, Of, W, rho)                   # student minus teacher
        G, C = oracle.normal_equations(Oc, T)
        return {"dW": oracle.solve_patch(G, C, inp.lam)}

    def layer_patch_teacher_basis(inp, rho):
        dt = inp.dtype
        Q, K, V, W = (oracle.decode(a, dt) for a in (inp.Q, inp.K, inp.V, inp.W))
        Kc, Vc = (oracle.gather_cache(K, V, inp.idx) if inp.idx is not None
                  else (oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)))
        Of = oracle.attention(Q, K, V, inp.scale)
        Oc = oracle.attention(Q, Kc, Vc, inp.scale)
        T = oracle.targets(Of, Oc, W, rho)
        G, C = oracle.normal_equations(Of, T)                # teacher features as basis
        return {"dW": oracle.solve_patch(G, C, inp.lam)}

    assert not check_decode_bf16(decode_shift15)
    assert not check_decode_bf16(decode_half)
    assert check_layer_patch(layer_patch_swapped) > 1e-2
    assert check_layer_patch(layer_patch_teacher_basis) > 1e-2


# ------------------------------------------------- per-KV-head eviction index sets

def brute_attention_heads(Q, K, V, sets, scale):
    """Scalar loops: KV head g's cache is the rows of K[g], V[g] listed in sets[g]."""
    M, Hq, dh = Q.shape
    Hkv = K.shape[0]
    grp = Hq // Hkv
    O = np.zeros((M, Hq * dh))
    for m in range(M):
        for h in range(Hq):
            g = h // grp
            s = [scale * sum(Q[m, h, c] * K[g, n, c] for c in range(dh)) for n in sets[g]]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            for c in range(dh):
                O[m, h * dh + c] = sum(e[i] * V[g, n, c] for i, n in enumerate(sets[g])) / sum(e)
    return O


def _head_sets_case(rng):
    Q, K, V = rand_attn(rng, 4, 30, 6, 3, 4, kscale=1.5)
    counts = np.array([7, 3, 5], dtype=np.int32)
    idx = np.full((3, 7), -1, dtype=np.int32)
    sets = []
    for g in range(3):
        sg = np.sort(rng.choice(30, size=counts[g], replace=False))
        idx[g, :counts[g]] = sg
        sets.append(list(sg))
    return Q, K, V, idx, counts, sets


def check_per_head_gather(gather) -> float:
    rng = np.random.default_rng(91)
    Q, K, V, idx, counts, sets = _head_sets_case(rng)
    Kc, Vc = gather(K, V, idx, counts)
    return rel(oracle.attention(Q, Kc, Vc, 0.5), brute_attention_heads(Q, K, V, sets, 0.5))


def test_per_head_gather_bruteforce_and_reductions():
    assert check_per_head_gather(oracle.gather_cache) < 1e-13
    rng = np.random.default_rng(92)
    Q, K, V = rand_attn(rng, 5, 40, 8, 4, 8)
    shared = np.sort(rng.choice(40, size=9, replace=False)).astype(np.int32)
    # one set replicated over the heads is the shared set
    Ks, Vs = oracle.gather_cache(K, V, shared)
    Kh, Vh = oracle.gather_cache(K, V, np.tile(shared, (4, 1)))
    assert rel(oracle.attention(Q, Kh, Vh), oracle.attention(Q, Ks, Vs)) < 1e-15
    # counts keep a prefix of each head's set; full counts change nothing
    per = np.stack([np.sort(rng.choice(40, size=9, replace=False)) for _ in range(4)]).astype(np.int32)
    Ka, Va = oracle.gather_cache(K, V, per)
    Kb, Vb = oracle.gather_cache(K, V, per, np.full(4, 9))
    assert rel(oracle.attention(Q, Kb, Vb), oracle.attention(Q, Ka, Va)) < 1e-15
    cnt = np.array([9, 1, 4, 6])
    Kt, Vt = oracle.gather_cache(K, V, per, cnt)
    O = oracle.attention(Q, Kt, Vt)
    for g in range(4):
        Kg, Vg = oracle.gather_cache(K[g:g + 1], V[g:g + 1], per[g, :cnt[g]])
        og = oracle.attention(Q[:, 2 * g:2 * g + 2], Kg, Vg)
        assert rel(O[:, 2 * g * 8:(2 * g + 2) * 8], og) < 1e-15
    # a head keeping one entry returns that entry's value
    assert np.allclose(O[:, 2 * 8:3 * 8], V[1, per[1, 0]][None, :], atol=1e-15)
    # permuting a head's own set leaves its output unchanged
    pp = per.copy()
    pp[2] = pp[2][::-1]
    Kp, Vp = oracle.gather_cache(K, V, pp)
    assert rel(oracle.attention(Q, Kp, Vp), oracle.attention(Q, Ka, Va)) < 1e-14


def test_per_head_gather_pin_catches_planted_mistakes():
    def gather_head0(K, V, idx, counts=None):
        Hkv = K.shape[0]
        s = idx[0][:int(counts[0])]                       # head 0's set for every head
        return [K[g][s] for g in range(Hkv)], [V[g][s] for g in range(Hkv)]

    def gather_no_counts(K, V, idx, counts=None):
        idx = np.where(idx < 0, 0, idx)                   # padding read as row 0
        return [K[g][idx[g]] for g in range(K.shape[0])], [V[g][idx[g]] for g in range(K.shape[0])]

    assert check_per_head_gather(gather_head0) > 1e-2
    assert check_per_head_gather(gather_no_counts) > 1e-2


def test_per_head_eviction_sets_recipe():
    inp = make_custom_inputs(M=4, N=500, B=40, Hq=8, Hkv=4, dh=8, cache="evict_heads",
                             n_sink=4, n_recent=10, seed=5)
    assert inp.idx.shape == (4, inp.B) and inp.counts.shape == (4,)
    assert int(inp.counts.sum()) == 4 * 40 and inp.B == int(inp.counts.max())
    assert len(set(inp.counts.tolist())) > 1                 # the heads' budgets differ
    for g in range(4):
        s = inp.idx[g, :inp.counts[g]]
        assert np.all(np.diff(s) > 0) and np.all(inp.idx[g, inp.counts[g]:] == -1)
        assert list(s[:4]) == [0, 1, 2, 3] and list(s[-10:]) == list(range(490, 500))
    # the whole-block patch over per-head sets: ΔW = 0 for a compressed cache that
    # keeps every token in every head
    full = make_custom_inputs(M=6, N=12, B=12, Hq=4, Hkv=2, dh=4, cache="identity", seed=6)
    full.idx = np.tile(np.arange(12, dtype=np.int32), (2, 1))
    full.counts = np.full(2, 12, dtype=np.int32)
    assert np.max(np.abs(oracle.layer_patch(full)["dW"])) == 0.0
