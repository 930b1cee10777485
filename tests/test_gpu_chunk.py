"""GPU parity of the chunked reference set (a chunk attends over the cache plus its
own causal prefix; statistics summed over chunks) against the fp64 oracle.

Tolerances as for the single-chunk passes: bf16 with P rounded to bf16 (p_terms 1)
4e-3, with the two-term split of P (p_terms 2) 5e-5, fp32 inputs 2e-5; layer patch
dW 2e-2 for bf16 inputs (fp32 statistics) and 1e-4 for fp32 inputs (fp64 statistics).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_chunk_inputs, make_custom_inputs

pytestmark = pytest.mark.gpu

TOL = {("bf16", 1): 4e-3, ("bf16", 2): 5e-5, ("f32", 1): 2e-5, ("f32", 2): 2e-5}

SHAPES = [
    # M, N, B, Hq, Hkv, dh, dtype
    (64, 700, 150, 8, 2, 128, "bf16"),      # ragged cache, own entries in 2 tiles
    (100, 1000, 333, 28, 4, 128, "bf16"),   # GQA group of 7: 7 rows per query position
    (33, 129, 17, 4, 4, 64, "bf16"),        # head_dim 64
    (300, 2049, 260, 32, 8, 128, "bf16"),   # several row tiles, own prefix spans 10 tiles
    (200, 5, 3, 8, 2, 128, "bf16"),         # tiny cache: the own entries dominate
    (1, 40, 7, 4, 2, 128, "bf16"),          # one token: it sees the cache and itself
    (128, 2048, 256, 4, 2, 64, "f32"),
    (70, 333, 100, 8, 2, 128, "f32"),
]


def _chunk(M, N, B, Hq, Hkv, dh, dt, cache="evict", seed=0):
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, cache=cache,
                             seed=seed + M + N, n_mix=min(64, N))
    ch = make_chunk_inputs(inp, 0, M)
    return inp, ch


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_attend_chunk_full_and_evicted(shape):
    M, N, B, Hq, Hkv, dh, dt = shape
    print(f"chunk attention parity M={M} N={N} B={B} Hq={Hq} Hkv={Hkv} dh={dh} {dt}", flush=True)
    inp, ch = _chunk(M, N, B, Hq, Hkv, dh, dt)
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    Q, Ks, Vs = (oracle.decode(a, dt) for a in (ch.Q, ch.Ks, ch.Vs))
    q, k, v, ks, vs = (to_dev(a, dt) for a in (ch.Q, inp.K, inp.V, ch.Ks, ch.Vs))
    ref_f = oracle.attention_chunk(Q, K, V, Ks, Vs, inp.scale)
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    ref_c = oracle.attention_chunk(Q, Kc, Vc, Ks, Vs, inp.scale)
    for pt in (1, 2):
        Of = host(pkv.attend_chunk(q, k, v, ks, vs, p_terms=pt))
        Oc = host(pkv.attend_chunk(q, k, v, ks, vs, idx=idx_dev(inp.idx), p_terms=pt))
        e_f, e_c = rel(Of, ref_f), rel(Oc, ref_c)
        print(f"  p_terms {pt}: O_f {e_f:.3e}  O_c {e_c:.3e}", flush=True)
        assert e_f <= TOL[(dt, pt)] and e_c <= TOL[(dt, pt)]


@pytest.mark.parametrize("shape", [s for s in SHAPES if s[6] == "bf16"],
                         ids=lambda s: "x".join(map(str, s)))
def test_chunk_stored_v_tiles_equal_transposed_tiles(shape):
    """A contiguous cache and the chunk's own entries are read with their V rows as
    stored; with per-head counts (every count = N) the same call goes through the V^T
    pre-pass. Same operands in the same order: equal bit for bit."""
    M, N, B, Hq, Hkv, dh, dt = shape
    inp, ch = _chunk(M, N, B, Hq, Hkv, dh, dt)
    q, k, v, ks, vs = (to_dev(a, dt) for a in (ch.Q, inp.K, inp.V, ch.Ks, ch.Vs))
    counts = torch.full((Hkv,), N, dtype=torch.int32, device=DEV)
    for pt in (1, 2):
        o_nat = pkv.attend_chunk(q, k, v, ks, vs, p_terms=pt)
        o_vt = pkv.attend_chunk(q, k, v, ks, vs, counts=counts, p_terms=pt)
        torch.cuda.synchronize()
        print(f"chunk stored vs transposed V tiles {shape} p_terms {pt}", flush=True)
        assert torch.isfinite(o_nat).all() and torch.equal(o_nat, o_vt)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_attend_chunk_synthesized_and_prefix_of_rows(dt):
    """A synthesized compressed cache (contiguous K_c, V_c), and a cache given as the
    first n_cache rows of a longer buffer."""
    inp, ch = _chunk(90, 600, 80, 8, 2, 128, dt, cache="synthesize")
    Q, Ks, Vs = (oracle.decode(a, dt) for a in (ch.Q, ch.Ks, ch.Vs))
    q, ks, vs = (to_dev(a, dt) for a in (ch.Q, ch.Ks, ch.Vs))
    Kc, Vc = oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)
    O = host(pkv.attend_chunk(q, to_dev(inp.Kc, dt), to_dev(inp.Vc, dt), ks, vs, p_terms=2))
    assert rel(O, oracle.attention_chunk(Q, Kc, Vc, Ks, Vs, inp.scale)) <= TOL[(dt, 2)]
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    O = host(pkv.attend_chunk(q, to_dev(inp.K, dt), to_dev(inp.V, dt), ks, vs, n_cache=257))
    ref = oracle.attention_chunk(Q, K[:, :257], V[:, :257], Ks, Vs, inp.scale)
    assert rel(O, ref) <= TOL[(dt, 1)]


def test_attend_chunk_causality_on_gpu():
    """Changing own entries after position 40 leaves rows 0..40 bitwise unchanged."""
    inp, ch = _chunk(96, 500, 64, 8, 2, 128, "bf16")
    q, k, v, ks, vs = (to_dev(a, "bf16") for a in (ch.Q, inp.K, inp.V, ch.Ks, ch.Vs))
    O1 = host(pkv.attend_chunk(q, k, v, ks, vs))
    ks2, vs2 = ks.clone(), vs.clone()
    ks2[:, 41:] = ks2[:, 41:] * 2 + 1
    vs2[:, 41:] = -vs2[:, 41:]
    O2 = host(pkv.attend_chunk(q, k, v, ks2, vs2))
    assert np.array_equal(O1[:41], O2[:41])
    assert np.all(np.abs(O1[41:] - O2[41:]).max(axis=1) > 1e-4)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_chunked_layer_patch(dt):
    """Three chunks: teacher and student chunk passes, targets, statistics accumulated
    over chunks, one solve; dW against the oracle's layer_patch_chunked."""
    M, N, B, Hq, Hkv, dh = (96, 1500, 200, 4, 2, 64) if dt == "f32" else (128, 3000, 300, 8, 2, 128)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=21,
                             lam=1e-2 if dt == "f32" else 1e-1)
    chunks = [make_chunk_inputs(inp, j, M) for j in range(3)]
    ref = oracle.layer_patch_chunked(inp, [(c.Q, c.Ks, c.Vs) for c in chunks])
    acc = pkv.F64 if dt == "f32" else pkv.F32
    adt = torch.float64 if dt == "f32" else torch.float32
    d = Hq * dh
    k, v, W = to_dev(inp.K, dt), to_dev(inp.V, dt), to_dev(inp.W, dt)
    idx = idx_dev(inp.idx)
    G = torch.empty((d, d), dtype=adt, device=DEV)
    C = torch.empty((d, d), dtype=adt, device=DEV)
    for j, c in enumerate(chunks):
        q, ks, vs = (to_dev(a, dt) for a in (c.Q, c.Ks, c.Vs))
        Of = pkv.attend_chunk(q, k, v, ks, vs, p_terms=1)
        Oc = pkv.attend_chunk(q, k, v, ks, vs, idx=idx, p_terms=2)
        T = pkv.compute_targets(Of, Oc, W, rho=1)
        pkv.accumulate_normal_eq(Oc, T, G=G, C=C, acc=acc, accumulate=j > 0)
    dW, info = pkv.solve_patch(G, C, inp.lam)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    e = rel(host(dW), ref["dW"])
    print(f"chunked layer patch {dt}: dW {e:.3e}", flush=True)
    assert e <= (1e-4 if dt == "f32" else 2e-2)
