"""GPU parity on seeded random shapes, beyond the hand-picked cases of the other files.

Each case draws its sizes from a fixed seed (the same cases every run) and checks the
library against the fp64 oracle with the tolerances of the per-entry-point tests:
* attention over the full cache and over the gathered compressed cache (bf16: 4e-3
  and 5e-5; fp32: 2e-5), with head_dim 64 or 128, any GQA group and ragged sizes;
* the ridge solve (fp32 split products: kappa 2^-14; fp64: 1e-7), with d and d_out
  ragged against every tile and block width.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_custom_inputs

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
