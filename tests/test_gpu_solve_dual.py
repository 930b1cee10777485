"""GPU parity of the ridge patch solved in the dual form (few rows, wide d_in).

patchkv_solve_patch_dual takes the statistics' inputs X [rows, d_in] and
T [rows, d_out] and returns X^T (X X^T + lambda I)^{-1} T, which equals Eq. 8's
(X^T X + lambda I)^{-1} X^T T for every X and lambda > 0 (push-through identity).
The reference is the oracle's Eq. 8 on G = X^T X, C = X^T T in fp64, so each test
checks the identity and the kernels together.

Tolerances (relative Frobenius error): K = X X^T and X^T Y take both operands as
two bf16 pieces with all four term products (about 2^-16 relative per product), the
rows x rows solve is the FP32-grade solve of the primal path. The forward error is
bounded by kappa(K + lambda I) * s * 2^-16, with s = sigma_max / sigma_min of X (X^T
maps the error of Y into dW), for the default and exact products, and by
kappa * s * 2^-14 for PATCHKV_SOLVE_FAST_BF16 (three products of about 2^-18 each);
every bound is computed from the system at hand and floored at 1e-4.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, rel

pytestmark = pytest.mark.gpu


def _system(rows, din, dout, seed, scale=0.3):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((rows, din)) * scale).astype(np.float32)
    T = rng.standard_normal((rows, dout)).astype(np.float32)
    return X, T


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _reference(X, T, lam, ridge="absolute"):
    X64, T64 = X.astype(np.float64), T.astype(np.float64)
    G, C = oracle.normal_equations(X64, T64)
    lam_used = oracle.ridge_lambda(G, lam, ridge)
    return oracle.solve_patch(G, C, lam_used), lam_used


def _tol(X, lam, products):
    X64 = X.astype(np.float64)
    s = np.linalg.svd(X64, compute_uv=False)
    s = s[s > s[0] * 1e-7] if s[0] > 0 else np.ones(1)
    # K = X X^T has rows - rank(X) zero eigenvalues: then lambda is the smallest of K + lambda I
    smin2 = s[-1] ** 2 if len(s) == X.shape[0] else 0.0
    kappa = (s[0] ** 2 + lam) / (smin2 + lam)
    stretch = s[0] / s[-1]
    per = 2.0 ** -16 if products != "split3" else 2.0 ** -14
    return max(1e-4, kappa * stretch * per)


def _mode(products):
    return {"split6": 0, "exact": pkv.SOLVE_EXACT_F32, "split3": pkv.SOLVE_FAST_BF16}[products]


DUAL_CASES = [
    (64, 512, 32, 0.1),
    (300, 1000, 130, 0.3),     # ragged tiles in every dimension
    (257, 2049, 67, 0.2),      # odd leading dimensions: unvectorised loads and stores
    (1000, 3000, 200, 0.1),
    (500, 300, 100, 0.5),      # more rows than d_in: the identity still holds
    (1, 7, 3, 0.1),            # degenerate: one row, a 1 x 1 system
    (33, 1, 5, 0.1),           # d_in = 1
]


@pytest.mark.parametrize("products", ["split6", "exact", "split3"])
@pytest.mark.parametrize("rows,din,dout,lam", DUAL_CASES)
def test_dual_solve_matches_eq8(rows, din, dout, lam, products):
    X, T = _system(rows, din, dout, rows + din + dout)
    print(f"dual solve rows={rows} d_in={din} d_out={dout} {products}", flush=True)
    dW, info = pkv.solve_patch_dual(_dev(X), _dev(T), lam, mode=_mode(products))
    assert int(info.item()) == 0
    ref, _ = _reference(X, T, lam)
    err, tol = rel(host(dW), ref), _tol(X, lam, products)
    print(f"  err {err:.3e} tol {tol:.3e}", flush=True)
    assert err <= tol


@pytest.mark.parametrize("ridge", ["adaptive", "trace_mean"])
def test_dual_solve_scaled_ridge(ridge):
    """Eq. 7's adaptive coefficient and the trace mean depend on G only through
    ||G||_F and tr G (and d_in), which X X^T shares with X^T X: the dual solve applies
    the primal system's lambda."""
    rows, din, dout, lam0 = 400, 1500, 90, 0.01
    X, T = _system(rows, din, dout, 11)
    base = pkv.RIDGE_ADAPTIVE if ridge == "adaptive" else pkv.RIDGE_TRACE_MEAN
    dW, info = pkv.solve_patch_dual(_dev(X), _dev(T), lam0, mode=base)
    assert int(info.item()) == 0
    X64, T64 = X.astype(np.float64), T.astype(np.float64)
    G, C = oracle.normal_equations(X64, T64)
    lam = oracle.ridge_lambda(G, lam0, ridge)
    ref = oracle.solve_patch(G, C, lam)
    err = rel(host(dW), ref)
    print(f"dual {ridge}: lambda {lam:.4e} err {err:.3e}", flush=True)
    assert err <= _tol(X, lam, "split6")


def test_dual_matches_primal_gpu_path():
    """The dual and the primal GPU paths on the same inputs (statistics + solve on the
    d_in-wide system, then the rows-wide system). With rows < d_in, G = X^T X is
    rank-deficient and G + lambda I has condition number (sigma_max^2 + lambda) /
    lambda, while K + lambda I has (sigma_max^2 + lambda) / (sigma_min^2 + lambda):
    the primal path meets its own, looser bound and the dual path is the more accurate."""
    rows, din, dout, lam = 512, 2048, 256, 0.1
    X, T = _system(rows, din, dout, 5)
    Xd, Td = _dev(X), _dev(T)
    G, C = pkv.accumulate_normal_eq(Xd, Td, acc=pkv.F32)
    dWp, ip = pkv.solve_patch(G, C, lam)
    dWd, idl = pkv.solve_patch_dual(Xd, Td, lam)
    assert int(ip.item()) == 0 and int(idl.item()) == 0
    ref, _ = _reference(X, T, lam)
    ep, ed, epd = rel(host(dWp), ref), rel(host(dWd), ref), rel(host(dWd), host(dWp))
    print(f"primal {ep:.3e} dual {ed:.3e} dual-vs-primal {epd:.3e}", flush=True)
    s0 = np.linalg.norm(X.astype(np.float64), 2)
    tol_primal = max(1e-4, (s0 ** 2 + lam) / lam * 2.0 ** -16)
    assert ed <= _tol(X, lam, "split6") and ep <= tol_primal
    assert ed <= ep and epd <= ep + ed


def test_dual_solve_mlp_shape():
    """The MLP-shaped patch's widths at 1,024 reference rows: X [1024, 14336]
    (SwiGLU features), T [1024, 4096]; 14336-wide primal system vs the 1024-wide dual
    one, checked on 64 sampled output columns of the fp64 reference."""
    rows, din, dout, lam0 = 1024, 14336, 4096, 0.001
    rng = np.random.default_rng(6)
    X = (rng.standard_normal((rows, din)) * 0.05).astype(np.float32)
    T = (rng.standard_normal((rows, dout)) * 0.02).astype(np.float32)
    dW, info = pkv.solve_patch_dual(_dev(X), _dev(T), lam0, mode=pkv.RIDGE_ADAPTIVE)
    assert int(info.item()) == 0
    cols = np.sort(rng.choice(dout, 64, replace=False))
    X64 = X.astype(np.float64)
    K = X64 @ X64.T
    lam = lam0 * float(np.sum(K * K)) / float(np.trace(K))  # = Eq. 7 on X^T X
    # reference columns through Eq. 8 on the primal system would need a 14336-wide
    # factorization; the push-through identity gives the same columns exactly
    Y = np.linalg.solve(K + lam * np.eye(rows), T[:, cols].astype(np.float64))
    ref = X64.T @ Y
    err = rel(host(dW)[:, cols], ref)
    print(f"dual MLP shape: lambda {lam:.4e} err {err:.3e}", flush=True)
    assert err <= 1e-3


def test_dual_solve_reuses_outputs_and_reports_pivots():
    """Caller-provided dW and info are written in place; a NaN in X reaches the
    pivot check (info > 0) rather than a silent result."""
    rows, din, dout = 96, 640, 48
    X, T = _system(rows, din, dout, 8)
    dW = torch.full((din, dout), 7.0, device=DEV)
    info = torch.full((1,), -3, dtype=torch.int32, device=DEV)
    out, inf = pkv.solve_patch_dual(_dev(X), _dev(T), 0.2, dW=dW, info=info)
    assert out.data_ptr() == dW.data_ptr() and inf.data_ptr() == info.data_ptr()
    assert int(info.item()) == 0
    ref, _ = _reference(X, T, 0.2)
    assert rel(host(dW), ref) <= 1e-4
    Xn = X.copy()
    Xn[10, 3] = np.nan
    _, inf2 = pkv.solve_patch_dual(_dev(Xn), _dev(T), 0.2)
    assert int(inf2.item()) > 0
