"""GPU parity of attention over compressed caches in the formats of Sec. 3.1 and
App. C: a per-entry logit bias (attention matching) and block-scaled int8 / int4
entries (quantized KV caches), against the fp64 oracle.

Block-scaled entries are exact in bf16, so the tolerances are those of the plain
passes: bf16 with P rounded to bf16 (p_terms 1) 4e-3, with a two-term P (p_terms
2) 5e-5; fp32 inputs 2e-5.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_cache_bias, make_custom_inputs, make_quant_cache

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
