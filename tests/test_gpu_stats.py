"""GPU parity of targets, sufficient statistics and the ridge solve.

Tolerances (relative Frobenius error):
* fp32 accumulation path: operands split into two bf16 terms (representation
  error ~2^-17 relative) with fp32 accumulation: targets and statistics within
  5e-5.
* fp64 accumulation path: fp64 products of fp32 inputs: 1e-12.
* solve, fp32 with FP32-grade products (the default: three bf16 pieces per operand,
  six MFMA products, about 2^-24 relative per product) or exact fp32 products
  (PATCHKV_SOLVE_EXACT_F32): Cholesky + triangular solves in fp32 on systems with
  condition number kappa <= ~1e2: error ~ kappa * 2^-24 * (growth), bound 1e-4; on
  ill-conditioned systems (kappa 1e4 - 1e5) bound kappa * 2^-20.
* solve, fp32 with PATCHKV_SOLVE_FAST_BF16 (two bf16 pieces, three products): each
  product carries about 3 * 2^-18 relative error (hi/lo representation of both
  operands and the dropped lo*lo term), so the first-order forward error is
  kappa * 3 * 2^-18 times a modest growth factor; bound kappa * 2^-14 (a factor ~5 of
  slack), computed from the system's own kappa.
* solve, fp64: the solve is fp64 but dW is returned in fp32, whose rounding alone
  is ~3e-8 RMS; bound 1e-7.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, rel

pytestmark = pytest.mark.gpu


def randn(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape).astype(np.float32) * np.float32(scale)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("M,din,dout,wdt,rho", [
    (200, 256, 256, "bf16", 1),
    (77, 300, 300, "f32", 1),
    (130, 200, 96, "bf16", 0),       # rectangular, ragged tiles
    (1024, 1024, 1024, "bf16", 1),
    (1, 64, 64, "bf16", 1),          # a single reference token
    (1, 64, 40, "f32", 0),
])
def test_targets(M, din, dout, wdt, rho):
    Of, Oc = randn((M, din), 1, 0.3), randn((M, din), 2, 0.3)
    W = randn((din, dout), 3, 1 / np.sqrt(din))
    if wdt == "bf16":
        Wt = dev(W).to(torch.bfloat16)
        Wref = Wt.float().cpu().numpy().astype(np.float64)
    else:
        Wt = dev(W)
        Wref = W.astype(np.float64)
    T = host(pkv.compute_targets(dev(Of), dev(Oc), Wt, rho=rho))
    ref = oracle.targets(Of.astype(np.float64), Oc.astype(np.float64), Wref, rho)
    assert rel(T, ref) <= 5e-5


@pytest.mark.parametrize("rows,din,dout", [(128, 256, 256), (300, 200, 130), (2048, 1024, 1024),
                                           (5, 64, 33), (1000, 3584, 512), (700, 4096, 256)])
def test_normal_equations_f32(rows, din, dout):
    """G exactly symmetric (mirrored tiles) and both products the same bits every call."""
    X, Yf, Yc = randn((rows, din), 4, 0.2), randn((rows, dout), 5), randn((rows, dout), 6)
    G, C = pkv.accumulate_normal_eq(dev(X), dev(Yf), dev(Yc), acc=pkv.F32)
    Gr, Cr = oracle.normal_equations(X.astype(np.float64), Yf.astype(np.float64) - Yc.astype(np.float64))
    assert rel(host(G), Gr) <= 5e-5
    assert rel(host(C), Cr) <= 5e-5
    g = host(G)
    assert np.array_equal(g, g.T)
    G2, C2 = pkv.accumulate_normal_eq(dev(X), dev(Yf), dev(Yc), acc=pkv.F32)
    assert torch.equal(G2, G) and torch.equal(C2, C)


@pytest.mark.parametrize("acc,din,dout", [("f32", 192, 160), ("f64", 192, 160), ("f32", 600, 300),
                                          ("f64", 600, 300)])
def test_normal_equations_accumulate_chunks(acc, din, dout):
    """Eq. 9: running sums over reference chunks equal the one-shot statistics. With
    d_in = 600 G spans several tiles per side (4 x 4 of the symmetric product's 192-tiles,
    the last one ragged), so the mirrored lower triangle is accumulated too; d_in = 192 is
    exactly one tile."""
    code = pkv.F32 if acc == "f32" else pkv.F64
    rows = 700
    X, Y = randn((rows, din), 7, 0.5), randn((rows, dout), 8)
    Gr, Cr = oracle.normal_equations(X.astype(np.float64), Y.astype(np.float64))
    G = C = None
    for a, b in [(0, 100), (100, 101), (101, 450), (450, 700)]:
        G, C = pkv.accumulate_normal_eq(dev(X[a:b]), dev(Y[a:b]), G=G, C=C, acc=code,
                                        accumulate=a > 0)
    tol = 5e-5 if acc == "f32" else 1e-12
    g = host(G)
    assert np.array_equal(g, g.T)
    assert rel(g, Gr) <= tol and rel(host(C), Cr) <= tol


def test_normal_equations_f64():
    rows, din, dout = 150, 256, 256
    X, Yf, Yc = randn((rows, din), 9, 0.2), randn((rows, dout), 10), randn((rows, dout), 11)
    G, C = pkv.accumulate_normal_eq(dev(X), dev(Yf), dev(Yc), acc=pkv.F64)
    Gr, Cr = oracle.normal_equations(X.astype(np.float64), Yf.astype(np.float64) - Yc.astype(np.float64))
    assert rel(host(G), Gr) <= 1e-12 and rel(host(C), Cr) <= 1e-12


def _spd_system(d, dout, rows, seed, scale=0.3):
    X = randn((rows, d), seed, scale).astype(np.float64)
    T = randn((rows, dout), seed + 1).astype(np.float64)
    return oracle.normal_equations(X, T)


def _mode(products):
    return {"split6": 0, "exact": pkv.SOLVE_EXACT_F32, "split3": pkv.SOLVE_FAST_BF16}[products]


def _solve_tol(acc, products, G, lam):
    if acc == "f64":
        return 1e-7
    if products in ("split6", "exact"):
        return 1e-4
    ev = np.linalg.eigvalsh(G + lam * np.eye(G.shape[0]))
    return float(ev[-1] / ev[0]) * 2.0 ** -14


SOLVE_CASES = [
    (256, 256, 400, "f64", 1e-2),
    (300, 130, 500, "f64", 0.3),     # ragged last block, rectangular right-hand side
    (400, 130, 500, "f64", 0.3),     # short last pair in the backward's block inversion
    (512, 512, 1000, "f32", 0.1),
    (1000, 700, 1500, "f32", 0.5),
    (64, 64, 30, "f32", 1.0),        # single block, rank-deficient X
    (700, 900, 1200, "f32", 0.2),    # d_out > d_in, ragged tiles in both directions
    (301, 67, 500, "f32", 0.3),      # rows not 16-byte aligned: unvectorised loads everywhere
    (257, 33, 400, "f64", 0.3),      # the same in fp64 (odd leading dimension)
    (17, 3, 40, "f32", 0.1),         # one partial block: a full leaf and a 1-wide one
    (1, 1, 5, "f32", 0.1),           # degenerate: a single unknown
    (1, 1, 5, "f64", 0.1),
]


# the fp64 solve has a single arithmetic: its cases run once, under the default mode
SOLVE_RUNS = [c + (p,) for c in SOLVE_CASES
              for p in (("split6", "exact", "split3") if c[3] == "f32" else ("split6",))]


@pytest.mark.parametrize("d,dout,rows,acc,lam,products", SOLVE_RUNS)
def test_solve(d, dout, rows, acc, lam, products):
    G, C = _spd_system(d, dout, rows, d + dout)
    tdt = torch.float64 if acc == "f64" else torch.float32
    mode = pkv.RIDGE_ABSOLUTE | _mode(products)
    dW, info = pkv.solve_patch(dev(G).to(tdt), dev(C).to(tdt), lam, mode=mode)
    assert int(info.item()) == 0
    Gin = G if acc == "f64" else G.astype(np.float32).astype(np.float64)
    Cin = C if acc == "f64" else C.astype(np.float32).astype(np.float64)
    ref = oracle.solve_patch(Gin, Cin, lam)
    err, tol = rel(host(dW), ref), _solve_tol(acc, products, Gin, lam)
    print(f"solve d={d} dout={dout} {acc} {products}: err {err:.3e} tol {tol:.3e}", flush=True)
    assert err <= tol


@pytest.mark.parametrize("ridge", ["adaptive", "trace_mean"])
@pytest.mark.parametrize("acc,products", [("f32", "split6"), ("f32", "exact"), ("f32", "split3"),
                                          ("f64", "split6")])
def test_solve_adaptive_ridge(acc, products, ridge):
    G, C = _spd_system(200, 150, 300, 3)
    tdt = torch.float64 if acc == "f64" else torch.float32
    base = pkv.RIDGE_ADAPTIVE if ridge == "adaptive" else pkv.RIDGE_TRACE_MEAN
    mode = base | _mode(products)
    dW, info = pkv.solve_patch(dev(G).to(tdt), dev(C).to(tdt), 0.01, mode=mode)
    assert int(info.item()) == 0
    Gin = G if acc == "f64" else G.astype(np.float32).astype(np.float64)
    Cin = C if acc == "f64" else C.astype(np.float32).astype(np.float64)
    lam = oracle.ridge_lambda(Gin, 0.01, ridge)
    err = rel(host(dW), oracle.solve_patch(Gin, Cin, lam))
    assert err <= _solve_tol(acc, products, Gin, lam)


@pytest.mark.parametrize("d,dout,kappa", [(512, 256, 1e4), (1000, 300, 1e5), (1536, 200, 3e4)])
def test_solve_fp32_grade_on_ill_conditioned_systems(d, dout, kappa):
    """G + lambda I with eigenvalues log-spaced from 1 down to 1/kappa: the default
    (six-term) products and exact fp32 products both stay within kappa * 2^-20 of the
    fp64 solution, and the six-term error is within a small factor of the exact one
    (FP32 grade), where the three-term products lose about 2^8 more."""
    rng = np.random.default_rng(d + int(kappa))
    U, _ = np.linalg.qr(rng.standard_normal((d, d)))
    ev = np.logspace(0.0, -np.log10(kappa), d)
    lam = 0.5 * ev[-1]
    G = ((U * (ev - lam)) @ U.T).astype(np.float32)
    G = (0.5 * (G + G.T)).astype(np.float32)
    C = rng.standard_normal((d, dout)).astype(np.float32)
    Gin, Cin = G.astype(np.float64), C.astype(np.float64)
    e = np.linalg.eigvalsh(Gin + lam * np.eye(d))
    kap = float(e[-1] / e[0])
    ref = oracle.solve_patch(Gin, Cin, lam)
    errs = {}
    for products in ("split6", "exact", "split3"):
        dW, info = pkv.solve_patch(dev(G), dev(C), lam, mode=pkv.RIDGE_ABSOLUTE | _mode(products))
        assert int(info.item()) == 0
        errs[products] = rel(host(dW), ref)
    print(f"ill-conditioned d={d} kappa={kap:.2e}: " +
          "  ".join(f"{k} {v:.3e}" for k, v in errs.items()), flush=True)
    assert errs["split6"] <= kap * 2.0 ** -20 and errs["exact"] <= kap * 2.0 ** -20
    assert errs["split6"] <= 4.0 * errs["exact"] + 1e-6


@pytest.mark.parametrize("acc", ["f32", "f64"])
def test_solve_reports_non_positive_pivot(acc):
    """A G that is not positive semidefinite gives info = first failing column."""
    d = 300
    G = np.eye(d)
    G[150, 150] = -5.0
    C = np.ones((d, 8))
    tdt = torch.float64 if acc == "f64" else torch.float32
    _, info = pkv.solve_patch(dev(G).to(tdt), dev(C).to(tdt), 1.0)
    assert int(info.item()) == 151


def test_zero_patch_for_identical_caches():
    """O_c == O_f bitwise => T = 0 => C = 0 => dW = 0 exactly."""
    from workloads import make_custom_inputs
    from gpu_util import idx_dev, to_dev
    inp = make_custom_inputs(M=64, N=256, B=256, Hq=4, Hkv=2, dh=64, dtype="bf16",
                             cache="identity", seed=1)
    q, k, v = to_dev(inp.Q, "bf16"), to_dev(inp.K, "bf16"), to_dev(inp.V, "bf16")
    idx = idx_dev(inp.idx)
    O1 = pkv.attend_compressed(q, k, v, idx=idx)
    O2 = pkv.attend_compressed(q, k, v, idx=idx)
    T = pkv.compute_targets(O1, O2, to_dev(inp.W, "bf16"), rho=1)
    G, C = pkv.accumulate_normal_eq(O2, T, acc=pkv.F32)
    dW, info = pkv.solve_patch(G, C, 0.1)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    assert torch.count_nonzero(T).item() == 0
    assert torch.count_nonzero(C).item() == 0
    assert torch.count_nonzero(dW).item() == 0
