"""The allocation-free compressed-cache attention (patchkv_attend_compressed_noalloc),
called through the C ABI, against patchkv_attend_compressed on the same inputs: the
same kernels run, so the outputs must agree bitwise, on two calls in a row (the
second smaller, so it runs on what the first left in the fixed scratch), for shared
and per-head index sets, key splits and a synthesized cache. Sizes beyond the fixed
scratch are rejected on the host before anything is enqueued.
"""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_39329_amd as pkv
from paper_2609_39329_amd import binding as B
from gpu_util import DEV, idx_dev, to_dev
from workloads import make_custom_inputs

pytestmark = pytest.mark.gpu


def _noalloc(inp, q, k, v, idx, mode, counts, B_, O, info):
    L = B.lib()
    dt = B.BF16 if inp.dtype == "bf16" else B.F32
    p = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    return L.patchkv_attend_compressed_noalloc(
        dt, p(q), p(k), p(v), p(idx), mode, p(counts), inp.M, inp.N, B_, inp.Hq, inp.Hkv,
        inp.dh, inp.scale, p(O), p(info), torch.cuda.current_stream().cuda_stream)


def _case(cache, dt, **shape):
    inp = make_custom_inputs(dtype=dt, cache=cache, n_mix=8, **shape)
    q, k, v = to_dev(inp.Q, dt), to_dev(inp.K, dt), to_dev(inp.V, dt)
    idx = idx_dev(inp.idx) if inp.idx is not None else None
    counts = idx_dev(inp.counts) if inp.counts is not None else None
    if inp.idx is None:
        k, v = to_dev(inp.Kc, dt), to_dev(inp.Vc, dt)
    mode = B.IDX_PER_HEAD if (inp.idx is not None and inp.idx.ndim == 2) else B.IDX_SHARED
    return inp, q, k, v, idx, mode, counts


CASES = [
    # (first call, second smaller call)
    (("evict_heads", "bf16", dict(M=300, N=5000, B=1500, Hq=32, Hkv=8, dh=128, seed=61)),
     ("evict", "bf16", dict(M=40, N=900, B=100, Hq=8, Hkv=2, dh=64, seed=62))),
    (("evict", "bf16", dict(M=16, N=40000, B=4000, Hq=8, Hkv=8, dh=128, seed=63)),    # key splits
     ("synthesize", "bf16", dict(M=20, N=500, B=60, Hq=4, Hkv=2, dh=128, seed=64))),
    (("evict_heads", "f32", dict(M=8, N=20000, B=3000, Hq=4, Hkv=2, dh=64, seed=65)),
     ("evict", "f32", dict(M=5, N=300, B=40, Hq=4, Hkv=2, dh=64, seed=66))),
]


@pytest.mark.parametrize("first,second", CASES, ids=["heads-then-shared", "split-then-synth",
                                                      "f32"])
def test_noalloc_matches_workspace_entry_point(first, second):
    for cache, dt, shape in (first, second):
        print(f"noalloc parity {cache} {dt} {shape}", flush=True)
        inp, q, k, v, idx, mode, counts = _case(cache, dt, **shape)
        B_ = inp.B if inp.idx is not None else inp.Kc.shape[1]
        need = B.lib().patchkv_attend_workspace_bytes(
            B.BF16 if dt == "bf16" else B.F32, inp.M, B_, inp.Hq, inp.Hkv, inp.dh)
        assert need <= B.NOALLOC_SCRATCH_BYTES
        ref_info = torch.full((1,), 99, dtype=torch.int32, device=DEV)
        ref = pkv.attend_compressed(q, k, v, idx=idx, counts=counts, info=ref_info)
        O = torch.full((inp.M, inp.Hq * inp.dh), float("nan"), dtype=torch.float32, device=DEV)
        info = torch.full((1,), 99, dtype=torch.int32, device=DEV)
        st = _noalloc(inp, q, k, v, idx, mode, counts, B_, O, info)
        assert st == B.OK, B.lib().patchkv_status_string(st)
        torch.cuda.synchronize()
        assert int(info.item()) == int(ref_info.item()) == 0
        assert torch.equal(O, ref)


def test_noalloc_rejects_sizes_beyond_the_fixed_scratch():
    # bf16 V^T tiles alone: 8 heads x 65536 entries x 128 x 2 bytes = 128 MiB > 64 MiB
    need = B.lib().patchkv_attend_workspace_bytes(B.BF16, 64, 65536, 32, 8, 128)
    assert need > B.NOALLOC_SCRATCH_BYTES
    FAKE = 1 << 12
    st = B.lib().patchkv_attend_compressed_noalloc(B.BF16, FAKE, FAKE, FAKE, None, 0, None, 64,
                                                   65536, 65536, 32, 8, 128, 0.1, FAKE, None,
                                                   None)
    assert st == B.E_SCRATCH
