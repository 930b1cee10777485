"""GPU parity of the MLP-shaped patch (SwiGLU features of the RMS-normed attention
output, targets through the d_ff x d down-projection plus the attention residual,
the d_ff x d patch, student-state propagation) against the fp64 oracle.

Tolerances: features, targets and propagation take fp32 operands as two-term bf16
splits (relative representation error ~2^-17 per operand, fp32 accumulation):
5e-5. The layer patch dW and the propagated student state: 2e-2, the bar for
bf16-input configurations (fp32 statistics and solve, as for the d x d patch).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, idx_dev, rel, to_dev
from workloads import make_custom_inputs, make_mlp_weights

pytestmark = pytest.mark.gpu


def randn(shape, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(shape) * scale).astype(np.float32)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


@pytest.mark.parametrize("wdt,M,d,d_ff", [("bf16", 300, 512, 1024), ("bf16", 77, 320, 700),
                                           ("f32", 130, 256, 516)])
def test_mlp_features(wdt, M, d, d_ff):
    print(f"mlp features {wdt} M={M} d={d} d_ff={d_ff}", flush=True)
    inp = make_custom_inputs(M=8, N=16, B=4, Hq=d // 64, Hkv=1, dh=64, dtype=wdt, seed=M)
    mlp = make_mlp_weights(inp, d_ff)
    Z = randn((M, d), M + 1, 0.05)
    H = host(pkv.mlp_features(dev(Z), to_dev(mlp.Wg, wdt), to_dev(mlp.Wu, wdt)))
    ref = oracle.mlp_features(Z.astype(np.float64), oracle.decode(mlp.Wg, wdt),
                              oracle.decode(mlp.Wu, wdt), mlp.eps)
    e = rel(H, ref)
    print(f"  H {e:.3e}", flush=True)
    assert e <= 5e-5


@pytest.mark.parametrize("wdt", ["bf16", "f32"])
def test_block_targets_and_propagation(wdt):
    M, d, d_ff = 200, 384, 900
    inp = make_custom_inputs(M=8, N=16, B=4, Hq=6, Hkv=1, dh=64, dtype=wdt, seed=5)
    mlp = make_mlp_weights(inp, d_ff)
    Hf, Hc = randn((M, d_ff), 1), randn((M, d_ff), 2)
    Hc = (Hf + 0.05 * Hc).astype(np.float32)          # student features near the teacher's
    Zf, Zc = randn((M, d), 3, 0.1), randn((M, d), 4, 0.1)
    dW = randn((d_ff, d), 6, 1e-2)
    Wd = to_dev(mlp.Wd, wdt)
    T = host(pkv.compute_block_targets(dev(Hf), dev(Hc), Wd, dev(Zf), dev(Zc)))
    W64 = oracle.decode(mlp.Wd, wdt)
    ref_t = oracle.block_targets(Hf.astype(np.float64), Hc.astype(np.float64), W64,
                                 Zf.astype(np.float64), Zc.astype(np.float64))
    Y = host(pkv.propagate_student(dev(Hc), Wd, dev(dW), dev(Zc)))
    ref_y = oracle.propagate_student(Hc.astype(np.float64), W64, dW.astype(np.float64),
                                     Zc.astype(np.float64))
    e_t, e_y = rel(T, ref_t), rel(Y, ref_y)
    print(f"block targets {wdt}: T {e_t:.3e}  Y {e_y:.3e}", flush=True)
    assert e_t <= 5e-5 and e_y <= 5e-5


def _gpu_mlp_patch(inp, mlp, lam, mode):
    dt = inp.dtype
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    Wg, Wu, Wd = to_dev(mlp.Wg, dt), to_dev(mlp.Wu, dt), to_dev(mlp.Wd, dt)
    Of = pkv.attend_full(q, k, v, scale=inp.scale)
    Oc = pkv.attend_compressed(q, k, v, idx=idx_dev(inp.idx), scale=inp.scale)
    Hf = pkv.mlp_features(Of, Wg, Wu, eps=mlp.eps)
    Hc = pkv.mlp_features(Oc, Wg, Wu, eps=mlp.eps)
    T = pkv.compute_block_targets(Hf, Hc, Wd, Of, Oc)
    G, C = pkv.accumulate_normal_eq(Hc, T, acc=pkv.F32)
    code = pkv.RIDGE_ADAPTIVE if mode == "adaptive" else pkv.RIDGE_ABSOLUTE
    dW, info = pkv.solve_patch(G, C, lam, mode=code)
    Y = pkv.propagate_student(Hc, Wd, dW, Oc)
    torch.cuda.synchronize()
    return dW, info, Y


@pytest.mark.parametrize("mode,lam", [("adaptive", 1e-3), ("absolute", 1.0)])
def test_mlp_layer_patch(mode, lam):
    """Attention, features, targets, statistics (d_in = d_ff), solve and
    propagation on a bf16 block, against the oracle's mlp_layer_patch. With
    d_ff = 1408 features and 384 tokens, 1024 directions of G carry only the ridge;
    the ridge is the MLP workload's adaptive one (Eq. 7, lambda_0 = 1e-3, here
    lambda ~ 1.6) or an absolute lambda = 1."""
    inp = make_custom_inputs(M=384, N=3000, B=300, Hq=8, Hkv=2, dh=64, dtype="bf16", seed=41)
    mlp = make_mlp_weights(inp, 1408)
    ref = oracle.mlp_layer_patch(inp, mlp, mode=mode, lam=lam)
    dW, info, Y = _gpu_mlp_patch(inp, mlp, lam, mode)
    assert int(info.item()) == 0
    e_w, e_y = rel(host(dW), ref["dW"]), rel(host(Y), ref["Y_student"])
    gap = rel(ref["Y_student"], ref["Y_teacher"]), rel(host(Y), ref["Y_teacher"])
    print(f"mlp layer patch ({mode}, lambda {ref['lam']:.3g}): dW {e_w:.3e}  Y {e_y:.3e}  student-teacher gap oracle {gap[0]:.3e} "
          f"gpu {gap[1]:.3e}", flush=True)
    assert e_w <= 2e-2 and e_y <= 2e-2


def test_mlp_identity_cache_gives_zero_patch():
    """Identical caches: the features, and so T, G's right-hand side and dW, are
    exactly zero; the propagated student state equals the teacher's block output."""
    inp = make_custom_inputs(M=100, N=500, B=500, Hq=4, Hkv=2, dh=64, dtype="bf16", seed=43,
                             cache="identity")
    mlp = make_mlp_weights(inp, 512)
    dt = inp.dtype
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    Wg, Wu, Wd = to_dev(mlp.Wg, dt), to_dev(mlp.Wu, dt), to_dev(mlp.Wd, dt)
    idx = idx_dev(inp.idx)
    Of = pkv.attend_compressed(q, k, v, idx=idx, scale=inp.scale)
    Oc = pkv.attend_compressed(q, k, v, idx=idx, scale=inp.scale)
    Hf, Hc = pkv.mlp_features(Of, Wg, Wu), pkv.mlp_features(Oc, Wg, Wu)
    T = pkv.compute_block_targets(Hf, Hc, Wd, Of, Oc)
    G, C = pkv.accumulate_normal_eq(Hc, T, acc=pkv.F32)
    dW, info = pkv.solve_patch(G, C, 0.1)
    Y = pkv.propagate_student(Hc, Wd, dW, Oc)
    Yt = pkv.propagate_student(Hf, Wd, torch.zeros_like(dW), Of)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    assert torch.count_nonzero(T).item() == 0 and torch.count_nonzero(dW).item() == 0
    assert torch.equal(Y, Yt)
