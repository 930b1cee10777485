"""Benchmark of the PatchKV context-loading path on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input: for
every layer of the workload, attention of the M reference queries over the full
cache and over the compressed cache, targets, normal equations and the ridge
solve (the same five library calls, in the same order, that
patchkv_compute_layer_patch makes). For a chunked reference set: the two
attention passes, targets and statistics of every chunk, then one solve. For the
MLP-shaped patch: both attention passes, the SwiGLU features of both, the block
targets, the ridge solve (in the dual form, rows x rows, when d_ff exceeds the
reference rows) and the student-state propagation.
The default workload is the 32-layer Llama-3-8B-shaped patch build over a
172,032-token context (1 % cache budget, 4,096 reference queries per layer). All
layer inputs are resident in HBM before the timed region starts.

Prints one JSON line: seconds per layer patch (value), attention TFLOP/s and its
fraction of the bf16 MFMA peak, context tokens/s, the roofline of the dominant
kernel (the full-cache attention, timed with HIP events on its stream inside the
timed region) and the fp64 CPU oracle timed on a bounded sample of the same
workload.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--layers L] [--dump-dw DIR]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sec per layer patch + ref-query attention TFLOP/s (% of MFMA peak), 1 MI355X"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 MFMA
PEAK_HBM_GBS = 8000.0


def traffic_profile(cfg) -> str:
    return os.path.join(ROOT, "profiles", f"hbm_traffic__{cfg.name}.md")


def measured_traffic(cfg):
    """HBM bytes per full-cache attention launch (fast path and fixup, and the V^T
    pre-pass of a call that runs one)
    from the committed counter summary of this workload (FETCH_SIZE and WRITE_SIZE,
    calibrated on a plain copy; written by profile_summary.py), or None when there is
    none or a kernel source changed since the counters were taken."""
    import hashlib
    path = traffic_profile(cfg)
    if not os.path.exists(path):
        return None
    hashes, nbytes = [], None
    for line in open(path):
        t = line.split()
        if len(t) == 3 and t[0] == "source_sha256":
            hashes.append((t[1], t[2]))
        elif len(t) == 3 and t[0] == "traffic_bytes_per_launch" and t[1] == "attend_full":
            nbytes = float(t[2])
    if not hashes or nbytes is None:
        return None
    for src, h in hashes:
        with open(os.path.join(ROOT, src), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != h:
                return None
    return nbytes


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--layers", type=int, default=None, help="layers per step (default: all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=256,
                    help="query rows of the oracle sample for the CPU baseline")
    ap.add_argument("--dump-dw", metavar="DIR", default=None,
                    help="after the timed steps, write every layer's patch dW (fp32 .npy) to DIR")
    return ap.parse_args()


class LayerDev:
    """One layer's inputs on the device (and, for a chunked reference set, every
    chunk's queries and own keys and values)."""

    def __init__(self, inp, torch, dev, chunks=(), mlp=None, extras=(None, None)):
        def t(a):
            x = torch.from_numpy(np.ascontiguousarray(a))
            if inp.dtype == "bf16":
                x = x.view(torch.bfloat16)
            return x.to(dev, non_blocking=False)
        self.Q, self.K, self.V, self.W = t(inp.Q), t(inp.K), t(inp.V), t(inp.W)
        self.chunks = [(t(c.Q), t(c.Ks), t(c.Vs)) for c in chunks]
        qc, bias = extras
        self.kv_format, self.Kq = 0, None
        if qc is not None:  # block-scaled compressed cache (MXINT8 = 1, MXINT4 = 2)
            self.kv_format = 1 if qc.bits == 8 else 2
            self.Kq, self.Vq, self.Ke, self.Ve = (torch.from_numpy(np.ascontiguousarray(a)).to(dev)
                                                  for a in (qc.Kq, qc.Vq, qc.Ke, qc.Ve))
        self.bias = torch.from_numpy(bias).to(dev) if bias is not None else None
        self.Wg = self.Wu = self.Wd = None
        if mlp is not None:
            self.Wg, self.Wu, self.Wd, self.eps = t(mlp.Wg), t(mlp.Wu), t(mlp.Wd), mlp.eps
        self.idx = (torch.from_numpy(inp.idx).to(dev) if inp.idx is not None else None)
        # per-KV-head index sets keep different numbers of entries per head
        self.counts = (torch.from_numpy(inp.counts).to(dev) if inp.counts is not None else None)
        self.Kc = t(inp.Kc) if inp.Kc is not None else None
        self.Vc = t(inp.Vc) if inp.Vc is not None else None


def dual_solve(cfg) -> bool:
    """The ridge patch through X^T (X X^T + lambda I)^{-1} T: the MLP-shaped patch whose
    d_ff exceeds the reference rows (and needs no G for a reduced-rank step)."""
    return bool(cfg.d_ff) and not cfg.rank and cfg.M < cfg.d_ff


class Buffers:
    """Per-step device buffers shared by all layers (the stream orders their reuse)."""

    def __init__(self, cfg, torch, dev, nl: int):
        self.acc = 1 if cfg.dtype == "bf16" else 2  # F32 statistics for bf16 inputs, F64 for fp32
        adt = torch.float64 if self.acc == 2 else torch.float32
        M, d = cfg.M, cfg.d
        din = cfg.d_ff or d  # the patched projection's input width
        self.mode = 1 if cfg.ridge == "adaptive" else 0  # RIDGE_ADAPTIVE / RIDGE_ABSOLUTE
        self.Of = torch.empty((M, d), dtype=torch.float32, device=dev)
        self.Oc = torch.empty((M, d), dtype=torch.float32, device=dev)
        self.T = torch.empty((M, d), dtype=torch.float32, device=dev)
        # the MLP-shaped patch with fewer reference rows than d_ff: solved in the dual
        # form (rows x rows) straight from H_c and T, no d_ff x d_ff statistics
        self.dual = dual_solve(cfg)
        if not self.dual:
            self.G = torch.empty((din, din), dtype=adt, device=dev)
            self.C = torch.empty((din, d), dtype=adt, device=dev)
        self.dW = [torch.empty((din, d), dtype=torch.float32, device=dev) for _ in range(nl)]
        self.info = torch.zeros((nl,), dtype=torch.int32, device=dev)
        if cfg.rank:  # reduced-rank factors of every layer's patch
            self.A = [torch.empty((din, cfg.rank), dtype=torch.float32, device=dev) for _ in range(nl)]
            self.U = [torch.empty((d, cfg.rank), dtype=torch.float32, device=dev) for _ in range(nl)]
        if cfg.d_ff:
            self.Hf = torch.empty((M, din), dtype=torch.float32, device=dev)
            self.Hc = torch.empty((M, din), dtype=torch.float32, device=dev)
            self.Y = torch.empty((M, d), dtype=torch.float32, device=dev)


def layer_steps(pkv, cfg, L, bufs, li: int, events=None):
    """One layer patch through the five library calls, in the order
    patchkv_compute_layer_patch makes them (for the MLP-shaped patch: with the
    SwiGLU features of both passes, the block targets and, after the solve, the
    student-state propagation); ``events`` = (start, end) CUDA events recorded
    around the full-cache attention on the current stream."""
    acc = pkv.F32 if bufs.acc == 1 else pkv.F64
    if events is not None:
        events[0].record()
    if cfg.teacher_p_terms == 2:  # the full cache with a two-term P
        pkv.attend_cache(L.Q, L.K, L.V, scale=cfg.scale, p_terms=2, O=bufs.Of)
    else:
        pkv.attend_full(L.Q, L.K, L.V, scale=cfg.scale, O=bufs.Of)
    if events is not None:
        events[1].record()
    if L.Kq is not None:  # block-scaled compressed cache (the compressed entries themselves)
        pkv.attend_cache(L.Q, L.Kq, L.Vq, kv_format=L.kv_format, Ke=L.Ke, Ve=L.Ve, bias=L.bias,
                         scale=cfg.scale, p_terms=2, O=bufs.Oc)
    elif L.bias is not None:
        pkv.attend_cache(L.Q, *((L.K, L.V) if L.idx is not None else (L.Kc, L.Vc)), idx=L.idx,
                         counts=L.counts, bias=L.bias, scale=cfg.scale, p_terms=2, O=bufs.Oc)
    elif L.idx is not None:
        pkv.attend_compressed(L.Q, L.K, L.V, idx=L.idx, counts=L.counts, scale=cfg.scale,
                              O=bufs.Oc)
    else:
        pkv.attend_compressed(L.Q, L.Kc, L.Vc, scale=cfg.scale, O=bufs.Oc)
    if cfg.d_ff:  # MLP-shaped patch
        pkv.mlp_features(bufs.Of, L.Wg, L.Wu, eps=L.eps, H=bufs.Hf)
        pkv.mlp_features(bufs.Oc, L.Wg, L.Wu, eps=L.eps, H=bufs.Hc)
        pkv.compute_block_targets(bufs.Hf, bufs.Hc, L.Wd, bufs.Of, bufs.Oc, T=bufs.T)
        if bufs.dual:
            pkv.solve_patch_dual(bufs.Hc, bufs.T, cfg.lam, mode=bufs.mode, dW=bufs.dW[li],
                                 info=bufs.info[li:li + 1])
        else:
            pkv.accumulate_normal_eq(bufs.Hc, bufs.T, G=bufs.G, C=bufs.C, acc=acc)
    else:
        pkv.compute_targets(bufs.Of, bufs.Oc, L.W, rho=1, T=bufs.T)
        pkv.accumulate_normal_eq(bufs.Oc, bufs.T, G=bufs.G, C=bufs.C, acc=acc)
    if not bufs.dual:
        pkv.solve_patch(bufs.G, bufs.C, cfg.lam, mode=bufs.mode, dW=bufs.dW[li],
                        info=bufs.info[li:li + 1])
    if cfg.d_ff:  # the student state through the patched block
        pkv.propagate_student(bufs.Hc, L.Wd, bufs.dW[li], bufs.Oc, Y=bufs.Y)
    if cfg.rank:  # the reduced-rank factors (A, U): dW_r = A U^T
        pkv.low_rank_patch(bufs.G, bufs.dW[li], r=cfg.rank, A=bufs.A[li], U=bufs.U[li],
                           want_full=False)


def chunked_layer_steps(pkv, cfg, L, bufs, li: int, events=None):
    """One layer patch from a chunked reference set: for each chunk, attention over
    the full cache and over the compressed cache, each plus the chunk's own causal
    prefix, targets and statistics (summed over chunks); then one solve. ``events``
    holds a (start, end) pair per chunk around its full-cache attention."""
    acc = pkv.F32 if bufs.acc == 1 else pkv.F64
    for j, (Q, Ks, Vs) in enumerate(L.chunks):
        if events is not None:
            events[j][0].record()
        pkv.attend_chunk(Q, L.K, L.V, Ks, Vs, scale=cfg.scale, p_terms=1, O=bufs.Of)
        if events is not None:
            events[j][1].record()
        if L.idx is not None:
            pkv.attend_chunk(Q, L.K, L.V, Ks, Vs, idx=L.idx, counts=L.counts, scale=cfg.scale,
                             p_terms=2, O=bufs.Oc)
        else:
            pkv.attend_chunk(Q, L.Kc, L.Vc, Ks, Vs, scale=cfg.scale, p_terms=2, O=bufs.Oc)
        pkv.compute_targets(bufs.Of, bufs.Oc, L.W, rho=1, T=bufs.T)
        pkv.accumulate_normal_eq(bufs.Oc, bufs.T, G=bufs.G, C=bufs.C, acc=acc, accumulate=j > 0)
    pkv.solve_patch(bufs.G, bufs.C, cfg.lam, mode=bufs.mode, dW=bufs.dW[li],
                    info=bufs.info[li:li + 1])


def cpu_baseline(cfg, rows: int) -> dict:
    """The fp64 oracle on a bounded sample of one layer, scaled to s / layer patch.

    Sample: layer 0's attention (full and compressed cache) and statistics for
    ``rows`` of the M reference queries (their cost is linear in M, so it is scaled
    by M / rows), plus the complete d x d ridge solve (independent of M).
    """
    import oracle
    from workloads import (make_cache_extras, make_chunk_inputs, make_layer_inputs,
                           make_mlp_weights, unpack_int4)
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        blas_threads = None
    cores = len(os.sched_getaffinity(0))
    inp = make_layer_inputs(cfg, 0)
    dt = inp.dtype
    ch = make_chunk_inputs(inp, 0, cfg.M) if cfg.chunks > 1 else None
    rows = min(rows, cfg.M)
    sel = np.linspace(0, cfg.M - 1, rows).astype(np.int64)
    t0 = time.perf_counter()
    K, V = oracle.decode(inp.K, dt), oracle.decode(inp.V, dt)
    W = oracle.decode(inp.W, dt)
    qc, cbias = make_cache_extras(cfg, inp)
    cb = None if cbias is None else cbias.astype(np.float64)
    if qc is not None:
        unq = (lambda a: a) if qc.bits == 8 else unpack_int4
        Kc, Vc = oracle.dequantize_mx(unq(qc.Kq), qc.Ke), oracle.dequantize_mx(unq(qc.Vq), qc.Ve)
    elif inp.idx is not None:
        Kc, Vc = oracle.gather_cache(K, V, inp.idx, inp.counts)
    else:
        Kc, Vc = oracle.decode(inp.Kc, dt), oracle.decode(inp.Vc, dt)
    if ch is None:
        Q = oracle.decode(inp.Q[sel], dt)
        Of = oracle.attention(Q, K, V, inp.scale)
        Oc = oracle.attention(Q, Kc, Vc, inp.scale, bias=cb)
    else:
        # the first ``rows`` tokens of chunk 0 (a chunk's prefix is itself a chunk)
        Q = oracle.decode(ch.Q[:rows], dt)
        Ks, Vs = oracle.decode(ch.Ks[:, :rows], dt), oracle.decode(ch.Vs[:, :rows], dt)
        Of = oracle.attention_chunk(Q, K, V, Ks, Vs, inp.scale)
        Oc = oracle.attention_chunk(Q, Kc, Vc, Ks, Vs, inp.scale)
    if cfg.d_ff:
        mlp = make_mlp_weights(inp, cfg.d_ff)
        Wg, Wu, Wd = (oracle.decode(a, dt) for a in (mlp.Wg, mlp.Wu, mlp.Wd))
        Hf, Hc = oracle.mlp_features(Of, Wg, Wu, mlp.eps), oracle.mlp_features(Oc, Wg, Wu, mlp.eps)
        T = oracle.block_targets(Hf, Hc, Wd, Of, Oc)
        G, C = oracle.normal_equations(Hc, T)
    else:
        T = oracle.targets(Of, Oc, W, 1)
        G, C = oracle.normal_equations(Oc, T)
    t_rows = time.perf_counter() - t0
    tokens = cfg.M * cfg.chunks
    # the solve at full size needs a well-posed full-size G: scale the sampled
    # statistics up to all reference tokens' worth of mass (its cost does not
    # depend on G's values)
    t1 = time.perf_counter()
    Gs, Cs = G * (tokens / rows), C * (tokens / rows)
    dW = oracle.solve_patch(Gs, Cs, oracle.ridge_lambda(Gs, cfg.lam, cfg.ridge))
    if cfg.rank:
        oracle.low_rank_patch(Gs, dW, cfg.rank)
    t_solve = time.perf_counter() - t1
    if cfg.d_ff:  # the propagation is linear in the rows, like the rest of the sample
        t2 = time.perf_counter()
        oracle.propagate_student(Hc, Wd, dW, Oc)
        t_rows += time.perf_counter() - t2
    est = t_rows * (tokens / rows) + t_solve
    what = (f"the first {rows} tokens of reference chunk 0 (of {cfg.chunks} chunks x {cfg.M})"
            if ch is not None else f"{rows} of {cfg.M} reference queries")
    return {"value": est, "unit": "s/layer-patch", "cores": cores, "blas_threads": blas_threads,
            "kind": "oracle",
            "sample": f"config {cfg.cid} layer 0: fp64 attention (full + compressed), targets and "
                      f"statistics for {what} ({t_rows:.2f} s, scaled x{tokens / rows:.0f}) + "
                      f"full {G.shape[0]}x{cfg.d} Cholesky solve"
                      f"{' and rank-%d reduction' % cfg.rank if cfg.rank else ''} "
                      f"({t_solve:.2f} s); input decoding included"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2609_39329_amd as pkv
    from workloads import (get_config, make_cache_extras, make_chunk_inputs, make_layer_inputs,
                           make_mlp_weights)

    cfg = get_config(args.config)
    nl = cfg.layers if args.layers is None else min(args.layers, cfg.layers)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t0 = time.perf_counter()
    layers = []
    for layer in range(nl):
        inp = make_layer_inputs(cfg, layer)
        chunks = [make_chunk_inputs(inp, j, cfg.M) for j in range(cfg.chunks)] if cfg.chunks > 1 else ()
        mlp = make_mlp_weights(inp, cfg.d_ff) if cfg.d_ff else None
        layers.append(LayerDev(inp, torch, dev, chunks, mlp, make_cache_extras(cfg, inp)))
        if layer % 8 == 7 or layer == nl - 1:
            log(f"[bench] inputs of {layer + 1}/{nl} layers resident ({time.perf_counter() - t0:.1f} s)")
    torch.cuda.synchronize()

    M, d = cfg.M, cfg.d
    chunked = cfg.chunks > 1
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(cfg.chunks)] for _ in range(nl)]

    bufs = Buffers(cfg, torch, dev, nl)

    def step(timed: bool):
        for li, L in enumerate(layers):
            if chunked:
                chunked_layer_steps(pkv, cfg, L, bufs, li, ev[li] if timed else None)
            else:
                layer_steps(pkv, cfg, L, bufs, li, ev[li][0] if timed else None)

    for w in range(args.warmup):
        step(False)
        torch.cuda.synchronize()
        log(f"[bench] warmup step {w + 1}/{args.warmup} done")
    attn_ms = []
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for s in range(args.steps):
        t0 = time.perf_counter()
        step(True)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        this = [a.elapsed_time(b) for pairs in ev for a, b in pairs]
        attn_ms += this
        log(f"[bench] step {s + 1}/{args.steps} done: {dt * 1e3:.1f} ms, full-cache attention "
            f"{np.mean(this):.3f} ms per call")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    bad = int((bufs.info != 0).sum().item())
    if bad:
        log(f"[bench] WARNING: {bad} layer solve(s) reported a non-positive pivot")

    ms_step = elapsed / args.steps * 1e3
    s_layer = elapsed / (args.steps * nl)
    # per launch; a chunk's own causal prefix adds sum_m (m + 1) = M (M + 1) / 2 keys
    own = M * (M + 1) / 2.0 if chunked else 0.0
    att_flops_full = 4.0 * cfg.Hq * cfg.dh * (M * cfg.N + own)
    att_flops_comp = 4.0 * cfg.Hq * cfg.dh * (M * cfg.B + own)
    launches = cfg.chunks                               # full-cache attention launches per layer
    t_attn = float(np.mean(attn_ms)) * 1e-3            # dominant kernel: full-cache attention
    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = att_flops_full / t_attn / 1e12
    kv_bytes = 2.0 * cfg.Hkv * cfg.N * cfg.dh * (2 if cfg.dtype == "bf16" else 4)
    traffic = measured_traffic(cfg)

    out = {
        "metric": METRIC,
        "value": s_layer,
        "unit": "s/layer-patch",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; shapes and distributions of the workload)",
        "config": {"workload": cfg.name, "config_id": cfg.cid, "layers_per_step": nl,
                   "N": cfg.N, "B": cfg.B, "M": M, "d": d, "Hq": cfg.Hq, "Hkv": cfg.Hkv,
                   "dh": cfg.dh, "lambda": cfg.lam, "compressed_cache": cfg.cache,
                   "reference_chunks": cfg.chunks,
                   "own_causal_prefix": chunked, "ridge": cfg.ridge, "rank": cfg.rank,
                   "kv_format": cfg.kv_format, "cache_bias": cfg.cache_bias,
                   "patch": (f"MLP down-projection {cfg.d_ff}x{d} (SwiGLU features, student "
                             f"propagation)" if cfg.d_ff else f"{d}x{d} projection"),
                   "solve": (f"dual ({M}x{M} system from H_c and T)" if dual_solve(cfg)
                             else f"primal ({cfg.d_ff or d}x{cfg.d_ff or d} normal equations)")},
        "attention_full_ms": t_attn * 1e3,
        "attention_full_tflops": achieved,
        "attention_full_frac_of_peak": achieved / peak,
        "attention_total_tflops_per_layer_time":
            launches * (att_flops_full + att_flops_comp) / s_layer / 1e12,
        "context_tokens_per_s": cfg.N / s_layer,
        "kv_stream_gbs_full_attention": kv_bytes / t_attn / 1e9,
        "kv_stream_frac_of_hbm_peak": kv_bytes / t_attn / 1e9 / PEAK_HBM_GBS,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "kernel": (("patchkv_attend_chunk" if chunked else
                                 "patchkv_attend_cache (full cache, two-term P: 1.5x the MFMA "
                                 "work of the algorithmic flops counted here)"
                                 if cfg.teacher_p_terms == 2 else "patchkv_attend_full")
                                + ((": vt_kernel (V^T tiles of the cache and own entries) + "
                                    "attn_bf16_kernel fast path + fixup" if chunked else
                                    ": attn_bf16_kernel fast path (V tiles as stored) + fixup")
                                   if cfg.dtype == "bf16" else ": attn_f32_kernel")),
                     "flops_per_launch": att_flops_full,
                     "traffic_unit": "HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "traffic_source": os.path.relpath(traffic_profile(cfg), ROOT) if traffic else None,
                     "hbm_gbs": traffic / t_attn / 1e9 if traffic else None,
                     "hbm_frac": traffic / t_attn / 1e9 / PEAK_HBM_GBS if traffic else None},
        "solve_info_nonzero_layers": bad,
    }
    if args.dump_dw:  # the patches are the artefact the method persists (outside the timed region)
        os.makedirs(args.dump_dw, exist_ok=True)
        for li in range(nl):
            np.save(os.path.join(args.dump_dw, f"dW_layer{li:02d}.npy"), bufs.dW[li].cpu().numpy())
            if cfg.rank:
                np.save(os.path.join(args.dump_dw, f"A_layer{li:02d}.npy"), bufs.A[li].cpu().numpy())
                np.save(os.path.join(args.dump_dw, f"U_layer{li:02d}.npy"), bufs.U[li].cpu().numpy())
        log(f"[bench] wrote {nl} layer patch(es) to {args.dump_dw}")
    if not args.no_cpu_baseline:
        log("[bench] timing the fp64 CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(cfg, args.cpu_rows)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
