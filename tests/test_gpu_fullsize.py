"""Parity at the workloads' full sizes, in the launch sequence bench.py times.

For every stored oracle fixture (written by tests/golden/make_oracle_fixtures.py
from the fp64 oracle alone) the patch dW of the GPU path is compared on
  * 8 sampled rows, element by element (relative Frobenius error of those rows),
  * a seeded random sketch dW @ R (tracks the relative error of the whole matrix),
  * ||dW||_F,
each against the 2e-2 bar for bf16 inputs. Attention outputs are compared on
sampled query rows that the oracle computes one by one. The single-call entry
point patchkv_compute_layer_patch must reproduce the step-by-step result bitwise.
For the chunked workload (4 reference chunks of 5,120 tokens) the sampled attention
rows are those of the last chunk, each computed by the oracle as plain attention of
that token over the cache followed by the chunk's own entries up to it.
"""
import glob
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_39329_amd as pkv
from gpu_util import DEV, host, rel
from workloads import (CONFIGS, make_cache_extras, make_chunk_inputs, make_layer_inputs,
                       make_mlp_weights, unpack_int4)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
from bench import Buffers, LayerDev, chunked_layer_steps, layer_steps  # noqa: E402

sys.path.insert(0, os.path.join(ROOT, "tests", "golden"))
from make_oracle_fixtures import fixture_path, sample_rows, sample_tokens, sketch_matrix  # noqa: E402

pytestmark = pytest.mark.gpu

CASES = [(1, 0), (2, 0), (4, 0), (3, 0), (3, 8), (3, 16), (3, 24), (3, 31), (5, 0), (6, 0), (7, 0),
         (8, 0), (9, 0), (10, 0), (11, 0)]
TOL = 2e-2


@pytest.mark.parametrize("cid,layer", CASES, ids=[f"c{c}-l{l}" for c, l in CASES])
def test_full_size_layer_patch(cid, layer):
    path = fixture_path(cid, layer)
    if not os.path.exists(path):
        pytest.skip(f"oracle fixture {os.path.basename(path)} not generated")
    cfg = CONFIGS[cid]
    print(f"full-size parity: config {cid} ({cfg.name}) layer {layer}", flush=True)
    fx = np.load(path)
    inp = make_layer_inputs(cfg, layer)
    chunks = [make_chunk_inputs(inp, j, cfg.M) for j in range(cfg.chunks)] if cfg.chunks > 1 else ()
    mlp = make_mlp_weights(inp, cfg.d_ff) if cfg.d_ff else None
    qc, cbias = make_cache_extras(cfg, inp)
    L = LayerDev(inp, torch, DEV, chunks, mlp, (qc, cbias))
    bufs = Buffers(cfg, torch, DEV, 1)
    if chunks:
        chunked_layer_steps(pkv, cfg, L, bufs, 0)
    else:
        layer_steps(pkv, cfg, L, bufs, 0)
    torch.cuda.synchronize()
    assert int(bufs.info[0].item()) == 0
    dW = host(bufs.dW[0])

    rows = sample_rows(cid, layer, dW.shape[0])
    assert np.array_equal(rows, fx["rows"])
    e_rows = rel(dW[rows], fx["dW_rows"])
    e_sk = rel(dW @ sketch_matrix(cid, layer, cfg.d), fx["sketch"])
    e_norm = abs(np.linalg.norm(dW) - float(fx["norm"])) / float(fx["norm"])
    print(f"  rows {e_rows:.3e}  sketch {e_sk:.3e}  norm {e_norm:.3e}", flush=True)
    assert e_rows <= TOL and e_sk <= TOL and e_norm <= TOL
    if cfg.rank:  # the reduced-rank factors capture the oracle's top-r energy
        X = bufs.dW[0] @ bufs.U[0]
        energy = float((X * (bufs.G @ X)).sum().item())
        e_en = abs(energy - float(fx["rank_energy"])) / float(fx["rank_energy"])
        print(f"  rank-{cfg.rank} energy {e_en:.3e}", flush=True)
        assert e_en <= TOL
    if cfg.d_ff:  # the propagated student state on sampled tokens
        y_rows = sample_tokens(cid, layer, cfg.M)
        assert np.array_equal(y_rows, fx["y_rows"])
        e_y = rel(host(bufs.Y)[y_rows], fx["Y_rows"])
        print(f"  Y rows {e_y:.3e}", flush=True)
        assert e_y <= TOL

    # attention outputs on sampled query rows, computed by the oracle row by row
    q_rows = np.random.default_rng([cid, layer, 7]).choice(cfg.M, 3, replace=False)
    dt = inp.dtype
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    if qc is not None:
        q = (lambda a: a) if qc.bits == 8 else unpack_int4
        Kc, Vc = oracle.dequantize_mx(q(qc.Kq), qc.Ke), oracle.dequantize_mx(q(qc.Vq), qc.Ve)
    elif inp.idx is not None:
        Kc, Vc = oracle.gather_cache(K, V, inp.idx, inp.counts)
    else:
        Kc, Vc = oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)
    cb = None if cbias is None else cbias.astype(np.float64)
    if chunks:
        last = chunks[-1]
        ref_f, ref_c = [], []
        for m in q_rows:
            q = oracle.decode(last.Q[m:m + 1], dt)
            ks, vs = oracle.decode(last.Ks[:, :m + 1], dt), oracle.decode(last.Vs[:, :m + 1], dt)
            ref_f.append(oracle.attention(q, np.concatenate([K, ks], 1), np.concatenate([V, vs], 1),
                                          inp.scale)[0])
            ref_c.append(oracle.attention(q, np.concatenate([Kc, ks], 1),
                                          np.concatenate([Vc, vs], 1), inp.scale)[0])
        ref_f, ref_c = np.array(ref_f), np.array(ref_c)
    else:
        Q = oracle.decode(inp.Q[q_rows], dt)
        ref_f = oracle.attention(Q, K, V, inp.scale)
        ref_c = oracle.attention(Q, Kc, Vc, inp.scale, bias=cb)
    e_of = rel(host(bufs.Of)[q_rows], ref_f)
    e_oc = rel(host(bufs.Oc)[q_rows], ref_c)
    print(f"  O_f rows {e_of:.3e}  O_c rows {e_oc:.3e}", flush=True)
    assert e_of <= 4e-3 and e_oc <= 5e-5

    if chunks or cfg.d_ff or cfg.rank or qc is not None or cbias is not None:
        return
    # the single-call entry point runs the same kernels in the same order
    dW2, info2 = pkv.compute_layer_patch(L.Q, L.K, L.V, L.W, idx=L.idx, Kc=L.Kc, Vc=L.Vc,
                                         counts=L.counts, lam=cfg.lam, scale=cfg.scale)
    torch.cuda.synchronize()
    assert int(info2.item()) == 0
    assert torch.equal(dW2, bufs.dW[0])
