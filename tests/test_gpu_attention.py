"""GPU parity of the attention entry points against the fp64 oracle.

Tolerances (relative Frobenius error of O):
* bf16 full-cache pass: P enters the P V product rounded to bf16 (relative
  rounding error <= 2^-9 per weight, RMS ~1.1e-3), Q K^T and the accumulation are
  exact / fp32, so the error of O stays near 1e-3; bound 4e-3.
* bf16 compressed pass: P enters as a two-term bf16 split (error ~2^-17), so only
  fp32 accumulation remains; bound 5e-5.
* fp32 inputs: fp32 dot products, softmax and accumulation; bound 2e-5.
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

SHAPES = [
    # M, N, B, Hq, Hkv, dh, dtype
    (64, 700, 150, 8, 2, 128, "bf16"),      # ragged N (not a multiple of the 32-key tile)
    (100, 1000, 333, 28, 4, 128, "bf16"),   # GQA group of 7, ragged row tiles
    (33, 129, 17, 4, 4, 64, "bf16"),        # head_dim 64, group 1
    (300, 2049, 260, 32, 8, 128, "bf16"),   # several row tiles, ragged tail
    (16, 40000, 4000, 8, 8, 128, "bf16"),   # few rows, long cache: split-key path + merge
    (128, 2048, 256, 4, 2, 64, "f32"),      # tiny fp32 layer shape
    (50, 333, 100, 8, 2, 128, "f32"),
    (8, 20000, 3000, 4, 2, 64, "f32"),      # fp32 split-key path
    (300, 3000, 700, 16, 4, 128, "f32"),    # fp32 MFMA kernel: several row tiles per head, ragged tail
    (1, 1, 1, 4, 2, 64, "bf16"),            # degenerate: one query, one key, one entry
    # one row tile per KV head: the keys split into 32-key ranges, the last one 8 (9)
    # keys long, so a work item's first tile is already past its range's end
    (1, 1000, 7, 4, 2, 128, "bf16"),
    (2, 1001, 9, 8, 2, 64, "bf16"),
    (1, 1, 1, 4, 2, 128, "f32"),
]


def _decode(inp):
    return (oracle.decode(inp.Q, inp.dtype), oracle.decode(inp.K, inp.dtype),
            oracle.decode(inp.V, inp.dtype))


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_attend_full_and_compressed(shape):
    M, N, B, Hq, Hkv, dh, dt = shape
    print(f"attention parity M={M} N={N} B={B} Hq={Hq} Hkv={Hkv} dh={dh} {dt}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=M + N)
    Q, K, V = _decode(inp)
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    Of = host(pkv.attend_full(q, k, v))
    ref = oracle.attention(Q, K, V, inp.scale)
    assert rel(Of, ref) <= TOL_FULL[dt]
    Oc = host(pkv.attend_compressed(q, k, v, idx=idx_dev(inp.idx)))
    Kc, Vc = oracle.gather_cache(K, V, inp.idx)
    assert rel(Oc, oracle.attention(Q, Kc, Vc, inp.scale)) <= TOL_COMP[dt]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_attend_synthesized_cache(dt):
    inp = make_custom_inputs(M=70, N=900, B=120, Hq=8, Hkv=2, dh=128, dtype=dt, cache="synthesize",
                             n_mix=16, seed=5)
    Q = oracle.decode(inp.Q, dt)
    Kc, Vc = oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)
    Oc = host(pkv.attend_compressed(to_dev(inp.Q, dt), to_dev(inp.Kc, dt), to_dev(inp.Vc, dt)))
    assert rel(Oc, oracle.attention(Q, Kc, Vc, inp.scale)) <= TOL_COMP[dt]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_identity_gather_matches_full(dt):
    """idx = 0..N-1 reproduces the full-cache attention."""
    inp = make_custom_inputs(M=40, N=500, B=500, Hq=4, Hkv=2, dh=128, dtype=dt, cache="identity",
                             seed=2)
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    Of = host(pkv.attend_full(q, k, v))
    Oc = host(pkv.attend_compressed(q, k, v, idx=idx_dev(inp.idx)))
    assert rel(Oc, Of) <= TOL_FULL[dt]


GATHER_ID_CASES = [
    # M, N, Hq, Hkv, dh, late-key excess (0: none)
    (300, 2049, 32, 8, 128, 0.0),    # ragged tail, several row tiles
    (16, 40000, 8, 8, 128, 0.0),     # split key ranges + merge
    (33, 129, 4, 4, 64, 0.0),        # head_dim 64
    (64, 2000, 8, 2, 128, 10.0),     # the fixup runs
]


@pytest.mark.parametrize("case", GATHER_ID_CASES, ids=lambda c: "x".join(map(str, c)))
def test_identity_gather_equals_contiguous_bitwise(case):
    """Gathered keys (loaded through registers by row index) and gathered V^T tiles give
    the same MFMA operands in the same order as the contiguous cache read directly, so
    an identity index set (shared, and per KV head) reproduces the contiguous result bit
    for bit, with one- and two-term P."""
    M, N, Hq, Hkv, dh, a = case
    print(f"identity gather vs contiguous: {case}", flush=True)
    rng = np.random.default_rng(N + dh)
    Qf = (rng.standard_normal((M, Hq, dh)) * 0.5 + (1.0 if a else 0.0)).astype(np.float32)
    Kf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    Vf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    if a:
        Kf[:, N * 3 // 4, :] = a
    q, k, v = (torch.from_numpy(x).bfloat16().to(DEV) for x in (Qf, Kf, Vf))
    ident = torch.arange(N, dtype=torch.int32, device=DEV)
    per_head = ident.repeat(Hkv, 1).contiguous()
    for pt in (1, 2):
        ref = pkv.attend_cache(q, k, v, p_terms=pt)
        shared = pkv.attend_cache(q, k, v, idx=ident, p_terms=pt)
        heads = pkv.attend_cache(q, k, v, idx=per_head, p_terms=pt)
        torch.cuda.synchronize()
        assert torch.isfinite(ref).all()
        assert torch.equal(shared, ref) and torch.equal(heads, ref), pt


def test_gather_permutation_and_duplicates():
    """A permuted index set gives the same output; a duplicated entry counts twice."""
    inp = make_custom_inputs(M=30, N=300, B=64, Hq=8, Hkv=4, dh=128, dtype="bf16", seed=4)
    q, k, v = to_dev(inp.Q, "bf16"), to_dev(inp.K, "bf16"), to_dev(inp.V, "bf16")
    base = host(pkv.attend_compressed(q, k, v, idx=idx_dev(inp.idx)))
    perm = np.random.default_rng(0).permutation(inp.idx)
    assert rel(host(pkv.attend_compressed(q, k, v, idx=idx_dev(perm))), base) <= 1e-5
    dup = np.concatenate([inp.idx, inp.idx[:5]])
    Q, K, V = _decode(inp)
    Kc, Vc = oracle.gather_cache(K, V, dup)
    got = host(pkv.attend_compressed(q, k, v, idx=idx_dev(dup)))
    assert rel(got, oracle.attention(Q, Kc, Vc, inp.scale)) <= TOL_COMP["bf16"]


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_single_entry_cache_returns_its_value(dt):
    inp = make_custom_inputs(M=20, N=1, B=1, Hq=4, Hkv=2, dh=64, dtype=dt, cache="identity", seed=9)
    O = host(pkv.attend_full(to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)))
    V = oracle.decode(inp.V, dt)
    ref = np.concatenate([V[h // 2, 0] for h in range(4)])[None, :].repeat(20, axis=0)
    # the softmax weight is exp2 of the fp32 rounding residual of the scaled score,
    # i.e. 1 to within an ulp, so O equals V to fp32 rounding
    assert np.max(np.abs(O - ref)) <= 4e-7 * np.max(np.abs(ref))


def test_attention_deterministic():
    inp = make_custom_inputs(M=64, N=3000, B=100, Hq=8, Hkv=2, dh=128, dtype="bf16", seed=8)
    q, k, v = to_dev(inp.Q, "bf16"), to_dev(inp.K, "bf16"), to_dev(inp.V, "bf16")
    a = pkv.attend_full(q, k, v)
    b = pkv.attend_full(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


NAT_CASES = [
    # M, N, Hq, Hkv, dh, p_terms, late-key excess (0: none)
    (300, 2049, 32, 8, 128, 1, 0.0),    # ragged tail, several row tiles
    (100, 1000, 28, 4, 128, 2, 0.0),    # GQA group of 7, two-term P
    (33, 129, 4, 4, 64, 1, 0.0),        # head_dim 64
    (16, 40000, 8, 8, 128, 1, 0.0),     # split key ranges + merge
    (8, 20000, 8, 2, 64, 2, 0.0),       # split key ranges, head_dim 64, two-term P
    (64, 2000, 8, 2, 128, 1, 10.0),     # scores outgrow the first tile: the fixup runs
    (64, 2000, 8, 2, 128, 2, 10.0),
]


@pytest.mark.parametrize("case", NAT_CASES, ids=lambda c: "x".join(map(str, c)))
def test_stored_v_tiles_equal_transposed_tiles(case):
    """A contiguous bf16 cache is read with its V rows as stored (transposing LDS reads
    of the P V operand); the same cache with per-head counts (every count = n) goes
    through the V^T pre-pass instead. The MFMA operands and their order are the same,
    so the outputs must be equal bit for bit, on the fast path, with split key ranges
    and in the fixup."""
    M, N, Hq, Hkv, dh, pt, a = case
    print(f"stored vs transposed V tiles: {case}", flush=True)
    rng = np.random.default_rng(M + N + dh)
    Qf = (rng.standard_normal((M, Hq, dh)) * 0.5 + (1.0 if a else 0.0)).astype(np.float32)
    Kf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    Vf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    if a:
        Kf[:, N * 3 // 4, :] = a
    q, k, v = (torch.from_numpy(x).bfloat16().to(DEV) for x in (Qf, Kf, Vf))
    counts = torch.full((Hkv,), N, dtype=torch.int32, device=DEV)
    i1 = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    i2 = torch.full((1,), -5, dtype=torch.int32, device=DEV)
    o_nat = pkv.attend_cache(q, k, v, p_terms=pt, info=i1)
    o_vt = pkv.attend_cache(q, k, v, counts=counts, p_terms=pt, info=i2)
    torch.cuda.synchronize()
    assert int(i1.item()) == 0 and int(i2.item()) == 0
    assert torch.isfinite(o_nat).all()
    assert torch.equal(o_nat, o_vt)
    if pt == 1:
        assert torch.equal(o_nat, pkv.attend_full(q, k, v))


@pytest.mark.parametrize("a", [1.0, 3.0, 4.0, 5.0, 8.0, 10.0])
def test_scores_outgrowing_the_first_tile(a):
    """One late key (position 1500 of 2000) scores about 16a - 4 log2 units above the
    first key tile's maximum for every query row. Small excesses stay on the fast
    path's fixed offset; large ones (row sums above 2^64, fp32 overflow of P or O,
    exp2 overflow to inf) send the work item to the lazily rescaled fixup. Every
    case must match the fp64 oracle."""
    M, N, Hq, Hkv, dh, late = 64, 2000, 8, 2, 128, 1500
    print(f"late-key excess a={a}", flush=True)
    rng = np.random.default_rng(int(a * 10))
    Qf = (rng.standard_normal((M, Hq, dh)) * 0.5 + 1.0).astype(np.float32)
    Kf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    Vf = rng.standard_normal((Hkv, N, dh)).astype(np.float32)
    Kf[:, late, :] = a
    q, k, v = (torch.from_numpy(x).bfloat16().to(DEV) for x in (Qf, Kf, Vf))
    Q, K, V = (x.double().cpu().numpy() for x in (q, k, v))
    scale = dh ** -0.5
    Of = host(pkv.attend_full(q, k, v, scale=scale))
    e_f = rel(Of, oracle.attention(Q, K, V, scale))
    idx = np.sort(np.concatenate([np.arange(0, 200), np.arange(1400, 1600)])).astype(np.int32)
    Oc = host(pkv.attend_compressed(q, k, v, idx=idx_dev(idx), scale=scale))
    Kc, Vc = oracle.gather_cache(K, V, idx)
    e_c = rel(Oc, oracle.attention(Q, Kc, Vc, scale))
    # two-term P over every key, contiguous and gathered (an overflowing weight makes
    # the low piece NaN, which must send the work item to the fixup too)
    ref = oracle.attention(Q, K, V, scale)
    O2 = host(pkv.attend_cache(q, k, v, scale=scale, p_terms=2))
    e_2 = rel(O2, ref)
    all_idx = np.arange(N, dtype=np.int32)
    Og = host(pkv.attend_compressed(q, k, v, idx=idx_dev(all_idx), scale=scale))
    e_g = rel(Og, ref)
    print(f"  O_f {e_f:.3e}  O_c {e_c:.3e}  two-term P: contiguous {e_2:.3e} gathered {e_g:.3e}",
          flush=True)
    assert all(np.isfinite(x).all() for x in (Of, Oc, O2, Og))
    assert e_f <= TOL_FULL["bf16"] and e_c <= TOL_COMP["bf16"]
    assert e_2 <= TOL_COMP["bf16"] and e_g <= TOL_COMP["bf16"]
