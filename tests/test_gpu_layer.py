"""End-to-end parity of patchkv_compute_layer_patch against the fp64 oracle.

The bar on the patch dW is the relative Frobenius error: <= 1e-4 for fp32 inputs
(fp64 statistics and solve) and <= 2e-2 for bf16 inputs (fp32 statistics and solve).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import host, idx_dev, rel, to_dev
from workloads import CONFIGS, make_custom_inputs, make_layer_inputs

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def run_layer(inp, rho=1, mode=pkv.RIDGE_ABSOLUTE, lam=None):
    dt = inp.dtype
    kw = {}
    if inp.idx is not None:
        kw["idx"] = idx_dev(inp.idx)
    else:
        kw["Kc"], kw["Vc"] = to_dev(inp.Kc, dt), to_dev(inp.Vc, dt)
    dW, info = pkv.compute_layer_patch(to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt),
                                       to_dev(inp.W, dt), lam=inp.lam if lam is None else lam,
                                       scale=inp.scale, rho=rho, mode=mode, **kw)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    return host(dW)


def test_config0_full_size():
    cfg = CONFIGS[0]
    print(f"layer parity {cfg.name}", flush=True)
    inp = make_layer_inputs(cfg)
    ref = oracle.layer_patch(inp, keep=False)["dW"]
    err = rel(run_layer(inp), ref)
    print(f"  rel err {err:.3e}", flush=True)
    assert err <= TOL["f32"]


@pytest.mark.parametrize("case", [
    dict(M=200, N=3000, B=300, Hq=8, Hkv=2, dh=128, dtype="bf16", cache="evict", lam=0.1),
    dict(M=150, N=2000, B=128, Hq=7, Hkv=1, dh=128, dtype="bf16", cache="synthesize", lam=0.05),
    dict(M=64, N=1000, B=200, Hq=4, Hkv=2, dh=128, dtype="f32", cache="evict", lam=0.01),
    dict(M=300, N=1500, B=99, Hq=4, Hkv=4, dh=64, dtype="bf16", cache="evict", lam=0.1),
], ids=["bf16-evict", "bf16-synth-g7", "f32-dh128", "bf16-dh64-mha"])
def test_layer_small(case):
    print(f"layer parity {case}", flush=True)
    inp = make_custom_inputs(seed=21, n_mix=16, **case)
    ref = oracle.layer_patch(inp, keep=False)["dW"]
    err = rel(run_layer(inp), ref)
    print(f"  rel err {err:.3e}", flush=True)
    assert err <= TOL[inp.dtype]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_layer_rho0_and_adaptive(dtype):
    inp = make_custom_inputs(M=128, N=1200, B=200, Hq=4, Hkv=2, dh=64, dtype=dtype, seed=22)
    ref0 = oracle.layer_patch(inp, rho=0, keep=False)["dW"]
    assert rel(run_layer(inp, rho=0), ref0) <= TOL[dtype]
    refa = oracle.layer_patch(inp, mode="adaptive", lam=1e-3, keep=False)["dW"]
    assert rel(run_layer(inp, mode=pkv.RIDGE_ADAPTIVE, lam=1e-3), refa) <= TOL[dtype]
