"""GPU parity of attention over compressed caches in the formats of Sec. 3.1 and
App. C: a per-entry logit bias (attention matching) and block-scaled int8 / int4
entries (quantized KV caches), against the fp64 oracle.

Block-scaled entries are exact in bf16, so the tolerances are those of the plain
passes: bf16 with P rounded to bf16 (p_terms 1) 4e-3, with a two-term P (p_terms
2) 5e-5; fp32 inputs 2e-5. The bf16 kernels read block-scaled entries themselves
(keys expanded when a tile is stored to LDS, values by the V^T pre-pass); since the
expansion is exact, their output must equal, bit for bit, that of the same kernel
variant over the expanded bf16 rows.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_cache_bias, make_custom_inputs, make_quant_cache, pack_int4

pytestmark = pytest.mark.gpu

TOL = {("bf16", 1): 4e-3, ("bf16", 2): 5e-5, ("f32", 1): 2e-5, ("f32", 2): 2e-5}


def _ref(inp, K, V, idx, bias):
    Q = oracle.decode(inp.Q, inp.dtype)
    if idx is not None:
        K, V = oracle.gather_cache(K, V, idx)
    return oracle.attention(Q, K, V, inp.scale, bias=bias)


@pytest.mark.parametrize("dt,M,N,B,Hq,Hkv,dh", [
    ("bf16", 64, 900, 150, 8, 2, 128),
    ("bf16", 300, 2049, 260, 28, 4, 128),   # GQA group of 7, several row tiles
    ("bf16", 16, 30000, 5000, 8, 8, 64),    # few rows, long cache: split keys + merge
    ("f32", 100, 700, 90, 4, 2, 64),
])
def test_attend_cache_bias(dt, M, N, B, Hq, Hkv, dh):
    print(f"bias parity {dt} M={M} N={N} B={B}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=M + B)
    bias = make_cache_bias(inp)
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    b = torch.from_numpy(bias).to(DEV)
    ref_g = _ref(inp, K, V, inp.idx, bias.astype(np.float64))
    ref_c = _ref(inp, K[:, :B], V[:, :B], None, bias.astype(np.float64))
    for pt in (1, 2):
        Og = host(pkv.attend_cache(q, k, v, idx=idx_dev(inp.idx), bias=b, p_terms=pt))
        Oc = host(pkv.attend_cache(q, k, v, n_cache=B, bias=b, p_terms=pt))
        e_g, e_c = rel(Og, ref_g), rel(Oc, ref_c)
        print(f"  p_terms {pt}: gathered {e_g:.3e}  contiguous {e_c:.3e}", flush=True)
        assert e_g <= TOL[(dt, pt)] and e_c <= TOL[(dt, pt)]
    # no bias through the same entry point: the plain compressed pass
    O0 = host(pkv.attend_cache(q, k, v, idx=idx_dev(inp.idx), p_terms=2))
    assert rel(O0, _ref(inp, K, V, inp.idx, None)) <= TOL[(dt, 2)]


@pytest.mark.parametrize("dt,bits", [("bf16", 8), ("bf16", 4), ("f32", 8), ("f32", 4)])
def test_attend_cache_block_scaled(dt, bits):
    M, N, B, Hq, Hkv, dh = 96, 1200, 200, 8, 2, 128
    print(f"MXINT{bits} parity {dt}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype=dt, seed=bits)
    qc = make_quant_cache(inp.K, inp.V, bits, dt)
    Kq = oracle.dequantize_mx(qc.Kq if bits == 8 else _unpack(qc.Kq), qc.Ke)
    Vq = oracle.dequantize_mx(qc.Vq if bits == 8 else _unpack(qc.Vq), qc.Ve)
    bias = make_cache_bias(inp)
    fmt = pkv.KV_MXINT8 if bits == 8 else pkv.KV_MXINT4
    q = to_dev(inp.Q, dt)
    kq, vq = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (qc.Kq, qc.Vq))
    ke, ve = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in (qc.Ke, qc.Ve))
    b = torch.from_numpy(bias).to(DEV)
    for with_bias in (False, True):
        bb = b if with_bias else None
        ref = _ref(inp, Kq, Vq, inp.idx, bias.astype(np.float64) if with_bias else None)
        O = host(pkv.attend_cache(q, kq, vq, kv_format=fmt, Ke=ke, Ve=ve, idx=idx_dev(inp.idx),
                                  bias=bb, p_terms=2))
        e = rel(O, ref)
        print(f"  bias {with_bias}: {e:.3e}", flush=True)
        assert e <= TOL[(dt, 2)]


def _unpack(p):
    lo = (p & 0xF).astype(np.int16)
    hi = (p >> 4).astype(np.int16)
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def test_bias_of_log_k_equals_k_copies_on_gpu():
    """A bias of log(3) on an entry equals three copies of it (bf16, two-term P)."""
    inp = make_custom_inputs(M=80, N=400, B=60, Hq=8, Hkv=2, dh=128, dtype="bf16", seed=9)
    q, k, v = to_dev(inp.Q, "bf16"), to_dev(inp.K, "bf16"), to_dev(inp.V, "bf16")
    bias = np.zeros((2, 60), dtype=np.float32)
    bias[:, 7] = np.log(3.0)
    O1 = host(pkv.attend_cache(q, k, v, n_cache=60, bias=torch.from_numpy(bias).to(DEV)))
    idx3 = np.concatenate([np.arange(60), [7, 7]]).astype(np.int32)
    O3 = host(pkv.attend_cache(q, k, v, idx=idx_dev(idx3)))
    assert rel(O1, O3) <= 5e-5


def _expanded(qc, bits):
    """The block-scaled cache's exact values as bf16 device tensors."""
    K = oracle.dequantize_mx(qc.Kq if bits == 8 else _unpack(qc.Kq), qc.Ke)
    V = oracle.dequantize_mx(qc.Vq if bits == 8 else _unpack(qc.Vq), qc.Ve)
    k = torch.from_numpy(K.astype(np.float32)).to(torch.bfloat16)
    v = torch.from_numpy(V.astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(k.double().numpy(), K) and np.array_equal(v.double().numpy(), V)
    return K, V, k.to(DEV), v.to(DEV)


@pytest.mark.parametrize("bits", [8, 4])
@pytest.mark.parametrize("M,N,B,Hq,Hkv,dh", [
    (96, 1200, 200, 8, 2, 128),
    (40, 3000, 700, 8, 8, 64),      # head_dim 64, few rows: split key ranges + merge
    (300, 2049, 260, 28, 4, 128),   # GQA group of 7, ragged tiles
])
def test_block_scaled_in_kernel_equals_expanded_rows(bits, M, N, B, Hq, Hkv, dh):
    print(f"MXINT{bits} in-kernel vs expanded M={M} N={N} B={B} dh={dh}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype="bf16", seed=bits + dh)
    qc = make_quant_cache(inp.K, inp.V, bits, "bf16")
    K, V, kx, vx = _expanded(qc, bits)
    fmt = pkv.KV_MXINT8 if bits == 8 else pkv.KV_MXINT4
    q = to_dev(inp.Q, "bf16")
    kq, vq, ke, ve = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
                      for a in (qc.Kq, qc.Vq, qc.Ke, qc.Ve))
    idx = idx_dev(inp.idx)
    b = torch.from_numpy(make_cache_bias(inp)).to(DEV)

    def both(**kw):
        Oq = pkv.attend_cache(q, kq, vq, kv_format=fmt, Ke=ke, Ve=ve, **kw)
        Ox = pkv.attend_cache(q, kx, vx, **kw)
        return Oq, Ox

    # same kernel variant on both sides: bitwise
    for kw in (dict(idx=idx, p_terms=1), dict(idx=idx, p_terms=2), dict(n_cache=B, p_terms=2),
               dict(idx=idx, bias=b, p_terms=2)):
        Oq, Ox = both(**kw)
        torch.cuda.synchronize()
        assert torch.equal(Oq, Ox), {k: v for k, v in kw.items() if k == "p_terms"}
    # the whole cache, P rounded to bf16: the expanded rows take the direct-to-LDS kernel
    Oq, Ox = both(p_terms=1)
    assert rel(host(Oq), host(Ox)) <= 1e-6
    assert rel(host(Oq), oracle.attention(oracle.decode(inp.Q, "bf16"), K, V, inp.scale)) <= 4e-3


@pytest.mark.parametrize("bits", [8, 4])
def test_block_scaled_full_context_parity(bits):
    """Quantization as the compression: the student cache is the whole context in
    block-scaled form (no eviction), attended with a two-term P against the oracle."""
    M, N, Hq, Hkv, dh = 200, 9000, 16, 4, 128
    print(f"MXINT{bits} full-context parity N={N}", flush=True)
    inp = make_custom_inputs(M=M, N=N, B=N, Hq=Hq, Hkv=Hkv, dh=dh, dtype="bf16", seed=40 + bits,
                             cache="identity")
    qc = make_quant_cache(inp.K, inp.V, bits, "bf16")
    K, V, _, _ = _expanded(qc, bits)
    fmt = pkv.KV_MXINT8 if bits == 8 else pkv.KV_MXINT4
    kq, vq, ke, ve = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
                      for a in (qc.Kq, qc.Vq, qc.Ke, qc.Ve))
    O = host(pkv.attend_cache(to_dev(inp.Q, "bf16"), kq, vq, kv_format=fmt, Ke=ke, Ve=ve,
                              p_terms=2))
    e = rel(O, oracle.attention(oracle.decode(inp.Q, "bf16"), K, V, inp.scale))
    print(f"  {e:.3e}", flush=True)
    assert e <= 5e-5


@pytest.mark.parametrize("bits", [8, 4])
def test_block_scaled_per_head_sets_and_bad_entries(bits):
    """Per-KV-head index sets with counts, one entry outside the cache: the in-kernel
    expansion reads it as a zero row and reports it, like the plain path."""
    M, N, B, Hq, Hkv, dh = 64, 1500, 300, 8, 4, 128
    inp = make_custom_inputs(M=M, N=N, B=B, Hq=Hq, Hkv=Hkv, dh=dh, dtype="bf16", seed=7 * bits,
                             cache="evict_heads")
    qc = make_quant_cache(inp.K, inp.V, bits, "bf16")
    _, _, kx, vx = _expanded(qc, bits)
    fmt = pkv.KV_MXINT8 if bits == 8 else pkv.KV_MXINT4
    kq, vq, ke, ve = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
                      for a in (qc.Kq, qc.Vq, qc.Ke, qc.Ve))
    idx = np.array(inp.idx, dtype=np.int32)
    assert inp.counts[1] > 5
    idx[1, 5] = N + 3  # outside the cache: flat position 1 * B + 5
    q, it, ct = to_dev(inp.Q, "bf16"), idx_dev(idx), idx_dev(inp.counts)
    iq = torch.zeros(1, dtype=torch.int32, device=DEV)
    ix = torch.zeros(1, dtype=torch.int32, device=DEV)
    for pt in (1, 2):
        Oq = pkv.attend_cache(q, kq, vq, kv_format=fmt, Ke=ke, Ve=ve, idx=it, counts=ct,
                              p_terms=pt, info=iq)
        Ox = pkv.attend_cache(q, kx, vx, idx=it, counts=ct, p_terms=pt, info=ix)
        torch.cuda.synchronize()
        assert torch.equal(Oq, Ox)
        assert int(iq.item()) == int(ix.item()) == -(1 + 1 * idx.shape[1] + 5)


@pytest.mark.parametrize("bits", [8, 4])
def test_block_scaled_extreme_exponents(bits):
    """Exponents far from the workloads' (values down in bf16's subnormal range and up
    near 2^117 for V): the kernels' expansion (ldexp in fp32, then round to nearest even to
    bf16) gives the same bits as the exact values rounded by torch, so the in-kernel
    path equals attention over those rows bit for bit."""
    M, N, Hq, Hkv, dh = 40, 700, 4, 2, 128
    rng = np.random.default_rng(77 + bits)
    qmax = 127 if bits == 8 else 7
    Kq = rng.integers(-qmax, qmax + 1, (Hkv, N, dh)).astype(np.int8)
    Vq = rng.integers(-qmax, qmax + 1, (Hkv, N, dh)).astype(np.int8)
    Ke = rng.integers(-9, -5, (Hkv, N, dh // 32)).astype(np.int8)
    # int8 exponents: the smallest ones put q 2^e (|q| <= 3) below 2^-126, in the
    # subnormal range; the largest reach 127 2^110
    Ve = np.where(rng.random((Hkv, N, dh // 32)) < 0.5, rng.integers(-128, -117, (Hkv, N, dh // 32)),
                  rng.integers(100, 111, (Hkv, N, dh // 32))).astype(np.int8)
    assert (Ve == -128).any() and np.abs(oracle.dequantize_mx(Vq, Ve)).max() < 3e38
    pack = (lambda a: a) if bits == 8 else pack_int4
    fmt = pkv.KV_MXINT8 if bits == 8 else pkv.KV_MXINT4
    K = oracle.dequantize_mx(Kq, Ke)
    V = oracle.dequantize_mx(Vq, Ve)
    kx = torch.from_numpy(K.astype(np.float32)).to(torch.bfloat16).to(DEV)
    vx = torch.from_numpy(V.astype(np.float32)).to(torch.bfloat16).to(DEV)
    q = torch.from_numpy(rng.standard_normal((M, Hq, dh)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    kq, vq, ke, ve = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
                      for a in (pack(Kq), pack(Vq), Ke, Ve))
    for pt in (1, 2):
        Oq = pkv.attend_cache(q, kq, vq, kv_format=fmt, Ke=ke, Ve=ve, n_cache=N, p_terms=pt)
        Ox = pkv.attend_cache(q, kx, vx, n_cache=N, p_terms=pt)
        torch.cuda.synchronize()
        assert torch.isfinite(Ox).all()
        assert torch.equal(Oq, Ox)
