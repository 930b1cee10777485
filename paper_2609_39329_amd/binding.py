"""ctypes binding of libpatchkv (argument marshalling only).

The raw C functions are exposed under their C names through :func:`lib`. The
functions below with the same names minus the ``patchkv_`` prefix take torch
tensors that already live on the GPU, read shapes and dtypes off them, allocate
outputs and workspace with torch (device memory and streams are torch's), and
call the library on the current torch stream. Every step of the computation runs
in the library's HIP kernels; nothing here computes. If the library is missing
the import of this module's functions fails loudly - there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
# PATCHKV_LIBRARY names another build of the same library (the host AddressSanitizer
# build of the C ABI layer, for the CPU validation tests)
LIB_PATH = os.environ.get("PATCHKV_LIBRARY") or os.path.join(HERE, "lib", "libpatchkv.so")

OK, E_NULL, E_SHAPE, E_DTYPE, E_VALUE, E_WORKSPACE, E_UNSUPPORTED, E_HIP, E_SCRATCH = range(9)
NOALLOC_SCRATCH_BYTES = 64 << 20  # fixed scratch of patchkv_attend_compressed_noalloc
F32, BF16, F64 = 0, 1, 2
IDX_SHARED, IDX_PER_HEAD = 0, 1
RIDGE_ABSOLUTE, RIDGE_ADAPTIVE, RIDGE_TRACE_MEAN = 0, 1, 2
# flags OR-ed into a ridge mode for the F32 solve's block products (default: three bf16
# pieces, six products, FP32-grade)
SOLVE_EXACT_F32 = 16  # exact fp32 products on fp32 MFMA
SOLVE_FAST_BF16 = 32  # two bf16 pieces, three products (about 2^-16 per product)

_c_i64 = ctypes.c_int64
_c_int = ctypes.c_int
_c_vp = ctypes.c_void_p
_c_sz = ctypes.c_size_t

# name -> (restype, argtypes)
SIGNATURES = {
    "patchkv_status_string": (ctypes.c_char_p, [_c_int]),
    "patchkv_version": (_c_int, []),
    "patchkv_attend_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_int, _c_int, _c_int]),
    "patchkv_attend_full": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int,
                                     _c_int, ctypes.c_float, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_attend_compressed": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_vp,
                                           _c_i64, _c_i64, _c_i64, _c_int, _c_int, _c_int,
                                           ctypes.c_float, _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_attend_compressed_noalloc": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_int,
                                                   _c_vp, _c_i64, _c_i64, _c_i64, _c_int, _c_int,
                                                   _c_int, ctypes.c_float, _c_vp, _c_vp, _c_vp]),
    "patchkv_attend_chunk_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_int, _c_int,
                                                     _c_int]),
    "patchkv_attend_chunk": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_vp, _c_i64,
                                      _c_i64, _c_vp, _c_vp, _c_i64, _c_int, _c_int, _c_int,
                                      ctypes.c_float, _c_int, _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_attend_cache_workspace_bytes": (_c_sz, [_c_int, _c_int, _c_i64, _c_i64, _c_int,
                                                     _c_int, _c_int]),
    "patchkv_attend_cache": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_int, _c_vp, _c_vp, _c_vp,
                                      _c_int, _c_vp, _c_i64, _c_i64, _c_vp, _c_i64, _c_int, _c_int,
                                      _c_int, ctypes.c_float, _c_int, _c_vp, _c_vp, _c_vp, _c_sz,
                                      _c_vp]),
    "patchkv_targets_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_i64]),
    "patchkv_compute_targets": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_i64,
                                         _c_int, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_mlp_features_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_i64]),
    "patchkv_mlp_features": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_i64,
                                      ctypes.c_float, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_block_targets_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_i64]),
    "patchkv_compute_block_targets": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_i64,
                                               _c_i64, _c_i64, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_propagate_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_i64]),
    "patchkv_propagate_student": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64,
                                           _c_i64, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_normal_eq_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_i64]),
    "patchkv_accumulate_normal_eq": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_i64,
                                              _c_int, _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_solve_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64]),
    "patchkv_solve_patch_dual_workspace_bytes": (_c_sz, [_c_i64, _c_i64, _c_i64]),
    "patchkv_solve_patch_dual": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_i64, ctypes.c_double,
                                          _c_int, _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_solve_patch": (_c_int, [_c_int, _c_vp, _c_vp, _c_i64, _c_i64, ctypes.c_double, _c_int,
                                     _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_low_rank_workspace_bytes": (_c_sz, [_c_i64, _c_i64, _c_int]),
    "patchkv_low_rank_patch": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_vp,
                                        _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_layer_workspace_bytes": (_c_sz, [_c_int, _c_int, _c_i64, _c_i64, _c_i64, _c_int,
                                              _c_int, _c_int]),
    "patchkv_compute_layer_patch": (_c_int, [_c_int, _c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_int,
                                             _c_vp, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_i64,
                                             _c_int, _c_int, _c_int, ctypes.c_float, _c_int,
                                             ctypes.c_double, _c_int, _c_vp, _c_vp, _c_vp, _c_sz,
                                             _c_vp]),
}

_LIB = None


class PatchKVError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = lib().patchkv_status_string(status).decode()
        super().__init__(f"{fn} failed: {msg} (status {status})")


def lib() -> ctypes.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libpatchkv is not built ({LIB_PATH} missing); "
                              "run __graft_entry__.build() or paper_2609_39329_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise PatchKVError(fn, status)


# ------------------------------------------------------------------ torch helpers

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.float64:
        return F64
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _require_gpu(*ts) -> None:
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous and on the GPU")


def _expect(t, name: str, dtypes, shape=None) -> None:
    """Raise before any launch if ``t`` does not have one of ``dtypes`` and ``shape``
    (a tuple whose None entries match any size): the C ABI receives only a pointer
    and would read or write memory of the size the other arguments imply."""
    if t is None:
        return
    if not isinstance(dtypes, (tuple, list)):
        dtypes = (dtypes,)
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if shape is not None:
        if t.dim() != len(shape) or any(w is not None and int(a) != int(w)
                                        for a, w in zip(t.shape, shape)):
            want = "[" + ", ".join("*" if w is None else str(int(w)) for w in shape) + "]"
            raise ValueError(f"{name} must have shape {want}, got {list(t.shape)}")


def _expect_info(info) -> None:
    torch = _torch()
    if info is not None:
        _expect(info, "info", torch.int32)
        if info.numel() < 1:
            raise ValueError("info must hold at least one int32")


def _index_set(idx, counts, Hkv: int):
    """(idx_mode, B) of a compressed cache's index set: idx int32 [B] (shared by every
    KV head) or [Hkv, B] (one set per KV head); counts int32 [Hkv] or None."""
    torch = _torch()
    _expect(idx, "idx", torch.int32)
    _expect(counts, "counts", torch.int32, (Hkv,))
    if idx is None:
        return IDX_SHARED, None
    if idx.dim() == 1:
        return IDX_SHARED, idx.shape[0]
    if idx.dim() == 2 and idx.shape[0] == Hkv:
        return IDX_PER_HEAD, idx.shape[1]
    raise ValueError(f"idx must have shape [B] or [{Hkv}, B], got {list(idx.shape)}")


def _qkv(Q, K, V, name_k: str = "K", name_v: str = "V"):
    """Shapes of Q [M, Hq, dh] and K, V [Hkv, N, dh] of Q's dtype (bf16 or f32)."""
    torch = _torch()
    _expect(Q, "Q", (torch.bfloat16, torch.float32))
    if Q.dim() != 3:
        raise ValueError(f"Q must have shape [M, Hq, dh], got {list(Q.shape)}")
    M, Hq, dh = Q.shape
    _expect(K, name_k, Q.dtype, (None, None, dh))
    Hkv, N, _ = K.shape
    _expect(V, name_v, Q.dtype, (Hkv, N, dh))
    return M, Hq, dh, Hkv, N


def _workspace(nbytes: int, device, stream=None):
    """Scratch for one call, allocated on the stream the call runs on (torch's caching
    allocator may hand the block to later work on that stream once it is freed)."""
    torch = _torch()
    if nbytes == 0:
        return None
    if stream is None:
        return torch.empty(nbytes, dtype=torch.uint8, device=device)
    with torch.cuda.stream(stream):
        return torch.empty(nbytes, dtype=torch.uint8, device=device)


def attend_full(Q, K, V, scale: Optional[float] = None, O=None, stream=None):
    """O [M, Hq*dh] fp32 = attention of Q [M,Hq,dh] over K, V [Hkv,N,dh]."""
    torch = _torch()
    _require_gpu(Q, K, V, O)
    M, Hq, dh, Hkv, N = _qkv(Q, K, V)
    _expect(O, "O", torch.float32, (M, Hq * dh))
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_workspace_bytes(dt, M, N, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_full",
           L.patchkv_attend_full(dt, _ptr(Q), _ptr(K), _ptr(V), M, N, Hq, Hkv, dh, scale,
                                 _ptr(O), _ptr(ws), nb, _stream(stream)))
    return O


def attend_compressed(Q, K, V, idx=None, counts=None, scale: Optional[float] = None, O=None,
                      info=None, stream=None):
    """Attention over the compressed cache. idx int32 [B]: rows idx of every KV head of
    the full cache K, V; idx int32 [Hkv, B]: rows idx[g] of KV head g; idx None: K and V
    are the synthesized cache [Hkv, B, dh]. counts int32 [Hkv] (optional): head g keeps
    only its first counts[g] entries. info (optional int32 tensor): the index-set check
    (0, or a negative code for an out-of-range entry or count)."""
    torch = _torch()
    _require_gpu(Q, K, V, idx, counts, O, info)
    M, Hq, dh, Hkv, N = _qkv(Q, K, V)
    mode, B = _index_set(idx, counts, Hkv)
    if B is None:
        B = N
    _expect(O, "O", torch.float32, (M, Hq * dh))
    _expect_info(info)
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_workspace_bytes(dt, M, B, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_compressed",
           L.patchkv_attend_compressed(dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), mode,
                                       _ptr(counts), M, N, B, Hq, Hkv, dh, scale, _ptr(O),
                                       _ptr(info), _ptr(ws), nb, _stream(stream)))
    return O


def attend_compressed_noalloc(Q, K, V, idx=None, counts=None, scale: Optional[float] = None,
                              O=None, info=None, stream=None):
    """attend_compressed through the library's allocation-free entry point: the scratch
    is the library's fixed device buffer, not a workspace (torch still allocates O
    when it is not given)."""
    torch = _torch()
    _require_gpu(Q, K, V, idx, counts, O, info)
    M, Hq, dh, Hkv, N = _qkv(Q, K, V)
    mode, B = _index_set(idx, counts, Hkv)
    if B is None:
        B = N
    _expect(O, "O", torch.float32, (M, Hq * dh))
    _expect_info(info)
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    _check("patchkv_attend_compressed_noalloc",
           lib().patchkv_attend_compressed_noalloc(dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), mode,
                                                   _ptr(counts), M, N, B, Hq, Hkv, dh, scale,
                                                   _ptr(O), _ptr(info), _stream(stream)))
    return O


def attend_chunk(Q, K, V, Ks, Vs, idx=None, counts=None, n_cache: Optional[int] = None,
                 scale: Optional[float] = None, p_terms: int = 1, O=None, info=None,
                 stream=None):
    """Attention of one reference chunk (queries Q [M,Hq,dh]) over a cache plus the
    chunk's own causal prefix Ks, Vs [Hkv,M,dh]: token m sees the cache and own
    entries 0..m. The cache is K[:, idx], V[:, idx] (idx int32 [n_cache], or
    [Hkv, n_cache] per KV head) or, with idx None, the first n_cache rows of K, V
    (default: all of them). p_terms = 2 forms P V from a two-term bf16 split of P
    (as attend_compressed)."""
    torch = _torch()
    _require_gpu(Q, K, V, Ks, Vs, idx, counts, O, info)
    M, Hq, dh, Hkv, n_src = _qkv(Q, K, V)
    _expect(Ks, "Ks", Q.dtype, (Hkv, M, dh))
    _expect(Vs, "Vs", Q.dtype, (Hkv, M, dh))
    mode, B = _index_set(idx, counts, Hkv)
    if B is not None:
        n_cache = B
    elif n_cache is None:
        n_cache = n_src
    _expect(O, "O", torch.float32, (M, Hq * dh))
    _expect_info(info)
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_chunk_workspace_bytes(dt, M, n_cache, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_chunk",
           L.patchkv_attend_chunk(dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), mode, _ptr(counts),
                                  n_src, n_cache, _ptr(Ks), _ptr(Vs), M, Hq, Hkv, dh, scale,
                                  p_terms, _ptr(O), _ptr(info), _ptr(ws), nb, _stream(stream)))
    return O


def compute_targets(Of, Oc, W, rho: int = 1, T=None, stream=None):
    """T = (Of - Oc) W + rho (Of - Oc), fp32."""
    torch = _torch()
    _require_gpu(Of, Oc, W, T)
    _expect(Of, "Of", torch.float32)
    if Of.dim() != 2:
        raise ValueError(f"Of must have shape [M, d_in], got {list(Of.shape)}")
    M, din = Of.shape
    _expect(Oc, "Oc", torch.float32, (M, din))
    _expect(W, "W", (torch.bfloat16, torch.float32), (din, None))
    dout = W.shape[1]
    _expect(T, "T", torch.float32, (M, dout))
    wdt = _dtype_code(W)
    if T is None:
        T = torch.empty((M, dout), dtype=torch.float32, device=Of.device)
    L = lib()
    nb = L.patchkv_targets_workspace_bytes(wdt, M, din, dout)
    ws = _workspace(nb, Of.device, stream)
    _check("patchkv_compute_targets",
           L.patchkv_compute_targets(wdt, _ptr(Of), _ptr(Oc), _ptr(W), M, din, dout, rho, _ptr(T),
                                     _ptr(ws), nb, _stream(stream)))
    return T


KV_PLAIN, KV_MXINT8, KV_MXINT4 = 0, 1, 2


def attend_cache(Q, K, V, kv_format: int = KV_PLAIN, Ke=None, Ve=None, idx=None, counts=None,
                 n_cache: Optional[int] = None, bias=None, scale: Optional[float] = None,
                 p_terms: int = 2, O=None, info=None, stream=None):
    """Attention over a compressed cache with an optional per-entry logit bias
    bias [Hkv, n_cache] (float32) and K, V stored plain (Q's dtype) or block-scaled:
    KV_MXINT8 (int8 [Hkv, n, dh]) / KV_MXINT4 (uint8 [Hkv, n, dh/2]) with int8
    exponents Ke, Ve [Hkv, n, dh/32]. The cache is rows idx (int32 [n_cache], or
    [Hkv, n_cache] per KV head) or the first n_cache rows (default all); counts int32
    [Hkv] (optional) keeps only each head's first counts[g] entries."""
    torch = _torch()
    _require_gpu(Q, K, V, Ke, Ve, idx, counts, bias, O, info)
    _expect(Q, "Q", (torch.bfloat16, torch.float32))
    if Q.dim() != 3:
        raise ValueError(f"Q must have shape [M, Hq, dh], got {list(Q.shape)}")
    M, Hq, dh = Q.shape
    if K.dim() != 3:
        raise ValueError(f"K must have shape [Hkv, n, *], got {list(K.shape)}")
    Hkv, n_src = K.shape[0], K.shape[1]
    if kv_format == KV_PLAIN:
        _expect(K, "K", Q.dtype, (Hkv, n_src, dh))
        _expect(V, "V", Q.dtype, (Hkv, n_src, dh))
    else:
        width = dh if kv_format == KV_MXINT8 else dh // 2
        qdt = torch.int8 if kv_format == KV_MXINT8 else torch.uint8
        _expect(K, "K", qdt, (Hkv, n_src, width))
        _expect(V, "V", qdt, (Hkv, n_src, width))
        if Ke is None or Ve is None:
            raise ValueError("block-scaled caches need the exponents Ke and Ve")
        _expect(Ke, "Ke", torch.int8, (Hkv, n_src, dh // 32))
        _expect(Ve, "Ve", torch.int8, (Hkv, n_src, dh // 32))
    mode, B = _index_set(idx, counts, Hkv)
    if B is not None:
        n_cache = B
    elif n_cache is None:
        n_cache = n_src
    _expect(bias, "bias", torch.float32, (Hkv, n_cache))
    _expect(O, "O", torch.float32, (M, Hq * dh))
    _expect_info(info)
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_cache_workspace_bytes(dt, kv_format, M, n_cache, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_cache",
           L.patchkv_attend_cache(dt, _ptr(Q), _ptr(K), _ptr(V), kv_format, _ptr(Ke), _ptr(Ve),
                                  _ptr(idx), mode, _ptr(counts), n_src, n_cache, _ptr(bias), M,
                                  Hq, Hkv, dh, scale, p_terms, _ptr(O), _ptr(info), _ptr(ws), nb,
                                  _stream(stream)))
    return O


def mlp_features(Z, Wg, Wu, eps: float = 1e-5, H=None, stream=None):
    """H [M, d_ff] = silu(u Wg) * (u Wu), u = RMS-normed Z [M, d] (unit gain)."""
    torch = _torch()
    _require_gpu(Z, Wg, Wu, H)
    _expect(Z, "Z", torch.float32)
    if Z.dim() != 2:
        raise ValueError(f"Z must have shape [M, d], got {list(Z.shape)}")
    M, d = Z.shape
    _expect(Wg, "Wg", (torch.bfloat16, torch.float32), (d, None))
    d_ff = Wg.shape[1]
    _expect(Wu, "Wu", Wg.dtype, (d, d_ff))
    _expect(H, "H", torch.float32, (M, d_ff))
    wt = _dtype_code(Wg)
    if H is None:
        H = torch.empty((M, d_ff), dtype=torch.float32, device=Z.device)
    L = lib()
    nb = L.patchkv_mlp_features_workspace_bytes(wt, M, d, d_ff)
    ws = _workspace(nb, Z.device, stream)
    _check("patchkv_mlp_features",
           L.patchkv_mlp_features(wt, _ptr(Z), _ptr(Wg), _ptr(Wu), M, d, d_ff, eps, _ptr(H),
                                  _ptr(ws), nb, _stream(stream)))
    return H


def compute_block_targets(Hf, Hc, W, Zf, Zc, T=None, stream=None):
    """T [M, d] = (Hf - Hc) W + (Zf - Zc) for the MLP-shaped block (W [d_ff, d])."""
    torch = _torch()
    _require_gpu(Hf, Hc, W, Zf, Zc, T)
    _expect(Hf, "Hf", torch.float32)
    if Hf.dim() != 2:
        raise ValueError(f"Hf must have shape [M, d_ff], got {list(Hf.shape)}")
    M, d_ff = Hf.shape
    _expect(Hc, "Hc", torch.float32, (M, d_ff))
    _expect(W, "W", (torch.bfloat16, torch.float32), (d_ff, None))
    d = W.shape[1]
    _expect(Zf, "Zf", torch.float32, (M, d))
    _expect(Zc, "Zc", torch.float32, (M, d))
    _expect(T, "T", torch.float32, (M, d))
    wt = _dtype_code(W)
    if T is None:
        T = torch.empty((M, d), dtype=torch.float32, device=Hf.device)
    L = lib()
    nb = L.patchkv_block_targets_workspace_bytes(wt, M, d_ff, d)
    ws = _workspace(nb, Hf.device, stream)
    _check("patchkv_compute_block_targets",
           L.patchkv_compute_block_targets(wt, _ptr(Hf), _ptr(Hc), _ptr(W), _ptr(Zf), _ptr(Zc), M,
                                           d_ff, d, _ptr(T), _ptr(ws), nb, _stream(stream)))
    return T


def propagate_student(Hc, W, dW, Zc, Y=None, stream=None):
    """Y [M, d] = Hc (W + dW) + Zc: the patched block's output on the student side."""
    torch = _torch()
    _require_gpu(Hc, W, dW, Zc, Y)
    _expect(Hc, "Hc", torch.float32)
    if Hc.dim() != 2:
        raise ValueError(f"Hc must have shape [M, d_ff], got {list(Hc.shape)}")
    M, d_ff = Hc.shape
    _expect(W, "W", (torch.bfloat16, torch.float32), (d_ff, None))
    d = W.shape[1]
    _expect(dW, "dW", torch.float32, (d_ff, d))
    _expect(Zc, "Zc", torch.float32, (M, d))
    _expect(Y, "Y", torch.float32, (M, d))
    wt = _dtype_code(W)
    if Y is None:
        Y = torch.empty((M, d), dtype=torch.float32, device=Hc.device)
    L = lib()
    nb = L.patchkv_propagate_workspace_bytes(wt, M, d_ff, d)
    ws = _workspace(nb, Hc.device, stream)
    _check("patchkv_propagate_student",
           L.patchkv_propagate_student(wt, _ptr(Hc), _ptr(W), _ptr(dW), _ptr(Zc), M, d_ff, d,
                                       _ptr(Y), _ptr(ws), nb, _stream(stream)))
    return Y


def accumulate_normal_eq(Xc, Yf, Yc=None, G=None, C=None, acc: int = F32, accumulate: bool = False,
                         stream=None):
    """G (+)= Xc^T Xc and C (+)= Xc^T (Yf - Yc); returns (G, C) of the acc dtype."""
    torch = _torch()
    _require_gpu(Xc, Yf, Yc, G, C)
    if acc not in (F32, F64):
        raise ValueError("acc must be F32 or F64")
    _expect(Xc, "Xc", torch.float32)
    if Xc.dim() != 2:
        raise ValueError(f"Xc must have shape [rows, d_in], got {list(Xc.shape)}")
    rows, din = Xc.shape
    _expect(Yf, "Yf", torch.float32, (rows, None))
    dout = Yf.shape[1]
    _expect(Yc, "Yc", torch.float32, (rows, dout))
    tdt = torch.float64 if acc == F64 else torch.float32
    _expect(G, "G", tdt, (din, din))
    _expect(C, "C", tdt, (din, dout))
    if G is None:
        G = torch.zeros((din, din), dtype=tdt, device=Xc.device)
    if C is None:
        C = torch.zeros((din, dout), dtype=tdt, device=Xc.device)
    L = lib()
    nb = L.patchkv_normal_eq_workspace_bytes(acc, rows, din, dout)
    ws = _workspace(nb, Xc.device, stream)
    _check("patchkv_accumulate_normal_eq",
           L.patchkv_accumulate_normal_eq(acc, _ptr(Xc), _ptr(Yf), _ptr(Yc), rows, din, dout,
                                          int(accumulate), _ptr(G), _ptr(C), _ptr(ws), nb,
                                          _stream(stream)))
    return G, C


def solve_patch(G, C, lam: float, mode: int = RIDGE_ABSOLUTE, dW=None, info=None, stream=None):
    """dW = (G + lam I)^{-1} C (fp32 out); returns (dW, info tensor)."""
    torch = _torch()
    _require_gpu(G, C, dW, info)
    _expect(G, "G", (torch.float32, torch.float64))
    if G.dim() != 2 or G.shape[0] != G.shape[1]:
        raise ValueError(f"G must be square [d_in, d_in], got {list(G.shape)}")
    din = G.shape[0]
    _expect(C, "C", G.dtype, (din, None))
    dout = C.shape[1]
    _expect(dW, "dW", torch.float32, (din, dout))
    _expect_info(info)
    acc = _dtype_code(G)
    if dW is None:
        dW = torch.empty((din, dout), dtype=torch.float32, device=G.device)
    if info is None:
        info = torch.empty((1,), dtype=torch.int32, device=G.device)
    L = lib()
    nb = L.patchkv_solve_workspace_bytes(acc, din, dout)
    ws = _workspace(nb, G.device, stream)
    _check("patchkv_solve_patch",
           L.patchkv_solve_patch(acc, _ptr(G), _ptr(C), din, dout, lam, mode, _ptr(dW), _ptr(info),
                                 _ptr(ws), nb, _stream(stream)))
    return dW, info


def solve_patch_dual(X, T, lam: float, mode: int = RIDGE_ABSOLUTE, dW=None, info=None,
                     stream=None):
    """dW = X^T (X X^T + lam I)^{-1} T, equal to (X^T X + lam I)^{-1} X^T T (X [rows, d_in],
    T [rows, d_out] float32; fp32 out); returns (dW, info tensor)."""
    torch = _torch()
    _require_gpu(X, T, dW, info)
    _expect(X, "X", torch.float32)
    if X.dim() != 2:
        raise ValueError(f"X must have shape [rows, d_in], got {list(X.shape)}")
    rows, din = X.shape
    _expect(T, "T", torch.float32, (rows, None))
    dout = T.shape[1]
    _expect(dW, "dW", torch.float32, (din, dout))
    _expect_info(info)
    if dW is None:
        dW = torch.empty((din, dout), dtype=torch.float32, device=X.device)
    if info is None:
        info = torch.empty((1,), dtype=torch.int32, device=X.device)
    L = lib()
    nb = L.patchkv_solve_patch_dual_workspace_bytes(rows, din, dout)
    if nb == 0:
        raise ValueError(f"unsupported dual solve shape rows={rows} d_in={din} d_out={dout}")
    ws = _workspace(nb, X.device, stream)
    _check("patchkv_solve_patch_dual",
           L.patchkv_solve_patch_dual(_ptr(X), _ptr(T), rows, din, dout, lam, mode, _ptr(dW),
                                      _ptr(info), _ptr(ws), nb, _stream(stream)))
    return dW, info


def layer_workspace_bytes(dtype: int, acc: int, M: int, N: int, B: int, Hq: int, Hkv: int,
                          dh: int) -> int:
    return lib().patchkv_layer_workspace_bytes(dtype, acc, M, N, B, Hq, Hkv, dh)


def low_rank_patch(G, dW, r: int = 32, iters: int = 24, A=None, U=None, dWr=None,
                   want_full: bool = True, stream=None):
    """Reduced-rank patch: (A [d_in, r], U [d_out, r], dW_r = A U^T or None) for the
    projection of dW onto the top-r eigenvectors of dW^T G dW (G, dW float32)."""
    torch = _torch()
    _require_gpu(G, dW, A, U, dWr)
    _expect(dW, "dW", torch.float32)
    if dW.dim() != 2:
        raise ValueError(f"dW must have shape [d_in, d_out], got {list(dW.shape)}")
    din, dout = dW.shape
    _expect(G, "G", torch.float32, (din, din))
    _expect(A, "A", torch.float32, (din, r))
    _expect(U, "U", torch.float32, (dout, r))
    _expect(dWr, "dWr", torch.float32, (din, dout))
    dev = dW.device
    if A is None:
        A = torch.empty((din, r), dtype=torch.float32, device=dev)
    if U is None:
        U = torch.empty((dout, r), dtype=torch.float32, device=dev)
    if dWr is None and want_full:
        dWr = torch.empty((din, dout), dtype=torch.float32, device=dev)
    L = lib()
    nb = L.patchkv_low_rank_workspace_bytes(din, dout, r)
    ws = _workspace(nb, dev, stream)
    _check("patchkv_low_rank_patch",
           L.patchkv_low_rank_patch(_ptr(G), _ptr(dW), din, dout, r, iters, _ptr(A), _ptr(U),
                                    _ptr(dWr), _ptr(ws), nb, _stream(stream)))
    return A, U, dWr


def compute_layer_patch(Q, K, V, W, idx=None, Kc=None, Vc=None, counts=None, lam: float = 0.1,
                        scale: Optional[float] = None, rho: int = 1, acc: Optional[int] = None,
                        mode: int = RIDGE_ABSOLUTE, dW=None, info=None, workspace=None,
                        stream=None):
    """One block's patch dW [d, d] fp32; returns (dW, info). The compressed cache is
    rows idx of K, V (int32 [B] shared, or [Hkv, B] per KV head; counts optional) or
    the synthesized Kc, Vc [Hkv, B, dh]."""
    torch = _torch()
    _require_gpu(Q, K, V, W, idx, Kc, Vc, counts, dW, info, workspace)
    M, Hq, dh, Hkv, N = _qkv(Q, K, V)
    d = Hq * dh
    _expect(W, "W", Q.dtype, (d, d))
    idx_mode, B = _index_set(idx, counts, Hkv)
    if idx is None:
        if Kc is None or Vc is None:
            raise ValueError("pass idx (eviction subset) or Kc and Vc (synthesized cache)")
        _expect(Kc, "Kc", Q.dtype, (Hkv, None, dh))
        B = Kc.shape[1]
        _expect(Vc, "Vc", Q.dtype, (Hkv, B, dh))
    _expect(dW, "dW", torch.float32, (d, d))
    _expect_info(info)
    _expect(workspace, "workspace", torch.uint8)
    dt = _dtype_code(Q)
    if acc is None:
        acc = F64 if dt == F32 else F32
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if dW is None:
        dW = torch.empty((d, d), dtype=torch.float32, device=Q.device)
    if info is None:
        info = torch.empty((1,), dtype=torch.int32, device=Q.device)
    L = lib()
    nb = L.patchkv_layer_workspace_bytes(dt, acc, M, N, B, Hq, Hkv, dh)
    ws = workspace if workspace is not None else _workspace(nb, Q.device, stream)
    wsz = ws.numel() * ws.element_size() if ws is not None else 0
    _check("patchkv_compute_layer_patch",
           L.patchkv_compute_layer_patch(dt, acc, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), idx_mode,
                                         _ptr(counts), _ptr(Kc), _ptr(Vc), _ptr(W), M, N, B, Hq,
                                         Hkv, dh, scale, rho, lam, mode, _ptr(dW), _ptr(info),
                                         _ptr(ws), wsz, _stream(stream)))
    return dW, info
