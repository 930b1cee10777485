"""GPU parity on seeded random shapes, beyond the hand-picked cases of the other files.

Each case draws its sizes from a fixed seed (the same cases every run) and checks the
library against the fp64 oracle with the tolerances of the per-entry-point tests:
* attention over the full cache and over the gathered compressed cache (bf16: 4e-3
  and 5e-5; fp32: 2e-5), with head_dim 64 or 128, any GQA group and ragged sizes;
* the ridge solve (fp32 split products: kappa 2^-14; fp64: 1e-7), with d and d_out
  ragged against every tile and block width;
* chunked attention with the causal own prefix, the normal equations, and the
  reduced-rank patch with a planted gap.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_chunk_inputs, make_custom_inputs

pytestmark = pytest.mark.gpu

TOL_FULL = {"bf16": 4e-3, "f32": 2e-5}
TOL_COMP = {"bf16": 5e-5, "f32": 2e-5}


def _attention_case(i):
    r = np.random.default_rng([2609, 1, i])
    Hkv = int(r.choice([1, 2, 4, 8]))
    G = int(r.integers(1, 9))
    dh = int(r.choice([64, 128]))
    dt = "bf16" if i % 3 else "f32"
    M = int(r.integers(1, 400))
    N = int(r.integers(1, 6000))
    B = int(r.integers(1, N + 1))
    return M, N, B, G * Hkv, Hkv, dh, dt


@pytest.mark.parametrize("i", range(12))
def test_attention_random_shape(i):
    M, N, B, Hq, Hkv, dh, dt = _attention_case(i)
    print(f"random attention case {i}: M={M} N={N} B={B} Hq={Hq} Hkv={Hkv} dh={dh} {dt}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=1000 + i)
    Q, K, V = (oracle.decode(inp.Q, dt), oracle.decode(inp.K, dt), oracle.decode(inp.V, dt))
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    Of = host(pkv.attend_full(q, k, v))
    assert rel(Of, oracle.attention(Q, K, V, inp.scale)) <= TOL_FULL[dt]
    Oc = host(pkv.attend_compressed(q, k, v, idx=idx_dev(inp.idx)))
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    assert rel(Oc, oracle.attention(Q, Kc, Vc, inp.scale)) <= TOL_COMP[dt]


def _solve_case(i):
    r = np.random.default_rng([2609, 2, i])
    d = int(r.integers(1, 1300))
    dout = int(r.integers(1, 700))
    rows = int(r.integers(max(2, d // 2), 2 * d + 10))
    acc = "f64" if i % 4 == 0 else "f32"
    return d, dout, rows, acc


@pytest.mark.parametrize("i", range(10))
def test_solve_random_shape(i):
    d, dout, rows, acc = _solve_case(i)
    print(f"random solve case {i}: d={d} d_out={dout} rows={rows} {acc}", flush=True)
    r = np.random.default_rng([2609, 3, i])
    X = (0.3 * r.standard_normal((rows, d))).astype(np.float32).astype(np.float64)
    T = r.standard_normal((rows, dout)).astype(np.float32).astype(np.float64)
    G, C = oracle.normal_equations(X, T)
    lam = 0.2
    tdt = torch.float64 if acc == "f64" else torch.float32
    dW, info = pkv.solve_patch(torch.from_numpy(G).to(DEV).to(tdt),
                               torch.from_numpy(C).to(DEV).to(tdt), lam)
    assert int(info.item()) == 0
    Gin = G if acc == "f64" else G.astype(np.float32).astype(np.float64)
    Cin = C if acc == "f64" else C.astype(np.float32).astype(np.float64)
    ref = oracle.solve_patch(Gin, Cin, lam)
    if acc == "f64":
        tol = 1e-7
    else:
        ev = np.linalg.eigvalsh(Gin + lam * np.eye(d))
        tol = float(ev[-1] / ev[0]) * 2.0 ** -14
    err = rel(host(dW), ref)
    print(f"  err {err:.3e} tol {tol:.3e}", flush=True)
    assert err <= tol


TOL_CHUNK = {("bf16", 1): 4e-3, ("bf16", 2): 5e-5, ("f32", 1): 2e-5, ("f32", 2): 2e-5}


@pytest.mark.parametrize("i", range(8))
def test_chunk_attention_random_shape(i):
    """A reference chunk over the full and the evicted cache plus its own causal prefix."""
    r = np.random.default_rng([2609, 4, i])
    Hkv = int(r.choice([1, 2, 4, 8]))
    Hq = Hkv * int(r.integers(1, 8))
    dh = int(r.choice([64, 128]))
    dt = "bf16" if i % 3 else "f32"
    M, N = int(r.integers(1, 300)), int(r.integers(1, 3000))
    B = int(r.integers(1, N + 1))
    print(f"random chunk case {i}: M={M} N={N} B={B} Hq={Hq} Hkv={Hkv} dh={dh} {dt}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=2000 + i)
    ch = make_chunk_inputs(inp, 0, M)
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    Q, Ks, Vs = (oracle.decode(a, dt) for a in (ch.Q, ch.Ks, ch.Vs))
    q, k, v, ks, vs = (to_dev(a, dt) for a in (ch.Q, inp.K, inp.V, ch.Ks, ch.Vs))
    ref_f = oracle.attention_chunk(Q, K, V, Ks, Vs, inp.scale)
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    ref_c = oracle.attention_chunk(Q, Kc, Vc, Ks, Vs, inp.scale)
    pt = 1 + i % 2
    Of = host(pkv.attend_chunk(q, k, v, ks, vs, p_terms=pt))
    Oc = host(pkv.attend_chunk(q, k, v, ks, vs, idx=idx_dev(inp.idx), p_terms=pt))
    assert rel(Of, ref_f) <= TOL_CHUNK[(dt, pt)]
    assert rel(Oc, ref_c) <= TOL_CHUNK[(dt, pt)]


@pytest.mark.parametrize("i", range(8))
def test_normal_equations_random_shape(i):
    """G = X^T X and C = X^T (Yf - Yc) in fp32 (split products, bound 5e-5) and fp64
    (bound 1e-12), G exactly symmetric."""
    r = np.random.default_rng([2609, 5, i])
    rows, din, dout = int(r.integers(1, 1500)), int(r.integers(1, 900)), int(r.integers(1, 900))
    acc = pkv.F64 if i % 4 == 0 else pkv.F32
    print(f"random normal-equation case {i}: rows={rows} d_in={din} d_out={dout} "
          f"{'f64' if acc == pkv.F64 else 'f32'}", flush=True)
    X = (0.2 * r.standard_normal((rows, din))).astype(np.float32)
    Yf, Yc = (r.standard_normal((rows, dout)).astype(np.float32) for _ in range(2))
    G, C = pkv.accumulate_normal_eq(*(torch.from_numpy(a).to(DEV) for a in (X, Yf, Yc)), acc=acc)
    Gr, Cr = oracle.normal_equations(X.astype(np.float64), Yf.astype(np.float64) - Yc.astype(np.float64))
    tol = 1e-12 if acc == pkv.F64 else 5e-5
    g = host(G)
    assert rel(g, Gr) <= tol and rel(host(C), Cr) <= tol
    assert np.array_equal(g, g.T)


@pytest.mark.parametrize("i", range(6))
def test_low_rank_random_shape(i):
    """Reduced-rank patch with a planted spectral gap after the r-th eigenvalue: the
    projected patch matches the oracle element-wise (bound 1e-4)."""
    r = np.random.default_rng([2609, 6, i])
    din, dout = int(r.integers(2, 400)), int(r.integers(2, 400))
    b = min(64, dout) & ~1
    rank = int(r.integers(1, min(b, din) + 1))  # the planted gap sits after eigenvalue r
    print(f"random low-rank case {i}: d_in={din} d_out={dout} r={rank}", flush=True)
    X = r.standard_normal((400, din)).astype(np.float32)
    G = (X.astype(np.float64).T @ X).astype(np.float32)
    dW = (r.standard_normal((din, rank)) @ r.standard_normal((rank, dout)) * 2
          + 0.01 * r.standard_normal((din, dout))).astype(np.float32)
    ref = oracle.low_rank_patch(G.astype(np.float64), dW.astype(np.float64), rank)
    A, U, dWr = pkv.low_rank_patch(torch.from_numpy(G).to(DEV), torch.from_numpy(dW).to(DEV),
                                   r=rank, iters=40)
    assert rel(host(dWr), ref["dW"]) <= 1e-4
