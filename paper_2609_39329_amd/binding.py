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
LIB_PATH = os.path.join(HERE, "lib", "libpatchkv.so")

OK, E_NULL, E_SHAPE, E_DTYPE, E_VALUE, E_WORKSPACE, E_UNSUPPORTED, E_HIP = range(8)
F32, BF16, F64 = 0, 1, 2
RIDGE_ABSOLUTE, RIDGE_ADAPTIVE, RIDGE_TRACE_MEAN = 0, 1, 2
SOLVE_EXACT_F32 = 16  # flag OR-ed into a ridge mode: exact fp32 products in the F32 solve

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
    "patchkv_attend_compressed": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64,
                                           _c_i64, _c_int, _c_int, _c_int, ctypes.c_float, _c_vp,
                                           _c_vp, _c_sz, _c_vp]),
    "patchkv_attend_chunk_workspace_bytes": (_c_sz, [_c_int, _c_i64, _c_i64, _c_int, _c_int,
                                                     _c_int]),
    "patchkv_attend_chunk": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_i64, _c_i64, _c_vp,
                                      _c_vp, _c_i64, _c_int, _c_int, _c_int, ctypes.c_float,
                                      _c_int, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_attend_cache_workspace_bytes": (_c_sz, [_c_int, _c_int, _c_i64, _c_i64, _c_int,
                                                     _c_int, _c_int]),
    "patchkv_attend_cache": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_int, _c_vp, _c_vp, _c_vp,
                                      _c_i64, _c_i64, _c_vp, _c_i64, _c_int, _c_int, _c_int,
                                      ctypes.c_float, _c_int, _c_vp, _c_vp, _c_sz, _c_vp]),
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
    "patchkv_solve_patch": (_c_int, [_c_int, _c_vp, _c_vp, _c_i64, _c_i64, ctypes.c_double, _c_int,
                                     _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_low_rank_workspace_bytes": (_c_sz, [_c_i64, _c_i64, _c_int]),
    "patchkv_low_rank_patch": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_vp,
                                        _c_vp, _c_vp, _c_sz, _c_vp]),
    "patchkv_layer_workspace_bytes": (_c_sz, [_c_int, _c_int, _c_i64, _c_i64, _c_i64, _c_int,
                                              _c_int, _c_int]),
    "patchkv_compute_layer_patch": (_c_int, [_c_int, _c_int, _c_vp, _c_vp, _c_vp, _c_vp, _c_vp,
                                             _c_vp, _c_vp, _c_i64, _c_i64, _c_i64, _c_int, _c_int,
                                             _c_int, ctypes.c_float, _c_int, ctypes.c_double,
                                             _c_int, _c_vp, _c_vp, _c_vp, _c_sz, _c_vp]),
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
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
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


def attend_compressed(Q, K, V, idx=None, scale: Optional[float] = None, O=None, stream=None):
    """Attention over the compressed cache: K[:, idx], V[:, idx] (idx int32 [B]) or,
    with idx None, K and V are the synthesized cache [Hkv, B, dh]."""
    torch = _torch()
    _require_gpu(Q, K, V, idx, O)
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
    B = idx.shape[0] if idx is not None else N
    if idx is not None and idx.dtype != torch.int32:
        raise TypeError("idx must be int32")
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_workspace_bytes(dt, M, B, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_compressed",
           L.patchkv_attend_compressed(dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), M, N, B, Hq, Hkv,
                                       dh, scale, _ptr(O), _ptr(ws), nb, _stream(stream)))
    return O



def attend_chunk(Q, K, V, Ks, Vs, idx=None, n_cache: Optional[int] = None,
                 scale: Optional[float] = None, p_terms: int = 1, O=None, stream=None):
    """Attention of one reference chunk (queries Q [M,Hq,dh]) over a cache plus the
    chunk's own causal prefix Ks, Vs [Hkv,M,dh]: token m sees the cache and own
    entries 0..m. The cache is K[:, idx], V[:, idx] (idx int32 [n_cache]) or, with
    idx None, the first n_cache rows of K, V (default: all of them). p_terms = 2
    forms P V from a two-term bf16 split of P (as attend_compressed)."""
    torch = _torch()
    _require_gpu(Q, K, V, Ks, Vs, idx, O)
    M, Hq, dh = Q.shape
    Hkv, n_src, _ = K.shape
    if idx is not None:
        if idx.dtype != torch.int32:
            raise TypeError("idx must be int32")
        n_cache = idx.shape[0]
    elif n_cache is None:
        n_cache = n_src
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_chunk_workspace_bytes(dt, M, n_cache, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_chunk",
           L.patchkv_attend_chunk(dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), n_src, n_cache,
                                  _ptr(Ks), _ptr(Vs), M, Hq, Hkv, dh, scale, p_terms, _ptr(O),
                                  _ptr(ws), nb, _stream(stream)))
    return O


def compute_targets(Of, Oc, W, rho: int = 1, T=None, stream=None):
    """T = (Of - Oc) W + rho (Of - Oc), fp32."""
    torch = _torch()
    _require_gpu(Of, Oc, W, T)
    M, din = Of.shape
    dout = W.shape[1]
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


def attend_cache(Q, K, V, kv_format: int = KV_PLAIN, Ke=None, Ve=None, idx=None,
                 n_cache: Optional[int] = None, bias=None, scale: Optional[float] = None,
                 p_terms: int = 2, O=None, stream=None):
    """Attention over a compressed cache with an optional per-entry logit bias
    bias [Hkv, n_cache] (float32) and K, V stored plain (Q's dtype) or block-scaled:
    KV_MXINT8 (int8 [Hkv, n, dh]) / KV_MXINT4 (uint8 [Hkv, n, dh/2]) with int8
    exponents Ke, Ve [Hkv, n, dh/32]. The cache is rows idx (int32 [n_cache]) or the
    first n_cache rows (default all)."""
    torch = _torch()
    _require_gpu(Q, K, V, Ke, Ve, idx, bias, O)
    M, Hq, dh = Q.shape
    Hkv, n_src = K.shape[0], K.shape[1]
    if idx is not None:
        if idx.dtype != torch.int32:
            raise TypeError("idx must be int32")
        n_cache = idx.shape[0]
    elif n_cache is None:
        n_cache = n_src
    dt = _dtype_code(Q)
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    if O is None:
        O = torch.empty((M, Hq * dh), dtype=torch.float32, device=Q.device)
    L = lib()
    nb = L.patchkv_attend_cache_workspace_bytes(dt, kv_format, M, n_cache, Hq, Hkv, dh)
    ws = _workspace(nb, Q.device, stream)
    _check("patchkv_attend_cache",
           L.patchkv_attend_cache(dt, _ptr(Q), _ptr(K), _ptr(V), kv_format, _ptr(Ke), _ptr(Ve),
                                  _ptr(idx), n_src, n_cache, _ptr(bias), M, Hq, Hkv, dh, scale,
                                  p_terms, _ptr(O), _ptr(ws), nb, _stream(stream)))
    return O


def mlp_features(Z, Wg, Wu, eps: float = 1e-5, H=None, stream=None):
    """H [M, d_ff] = silu(u Wg) * (u Wu), u = RMS-normed Z [M, d] (unit gain)."""
    torch = _torch()
    _require_gpu(Z, Wg, Wu, H)
    M, d = Z.shape
    d_ff = Wg.shape[1]
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
    M, d_ff = Hf.shape
    d = W.shape[1]
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
    M, d_ff = Hc.shape
    d = W.shape[1]
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
    rows, din = Xc.shape
    dout = Yf.shape[1]
    tdt = torch.float64 if acc == F64 else torch.float32
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
    din, dout = C.shape
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


def layer_workspace_bytes(dtype: int, acc: int, M: int, N: int, B: int, Hq: int, Hkv: int,
                          dh: int) -> int:
    return lib().patchkv_layer_workspace_bytes(dtype, acc, M, N, B, Hq, Hkv, dh)


def low_rank_patch(G, dW, r: int = 32, iters: int = 24, A=None, U=None, dWr=None,
                   want_full: bool = True, stream=None):
    """Reduced-rank patch: (A [d_in, r], U [d_out, r], dW_r = A U^T or None) for the
    projection of dW onto the top-r eigenvectors of dW^T G dW (G, dW float32)."""
    torch = _torch()
    _require_gpu(G, dW, A, U, dWr)
    din, dout = dW.shape
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


def compute_layer_patch(Q, K, V, W, idx=None, Kc=None, Vc=None, lam: float = 0.1,
                        scale: Optional[float] = None, rho: int = 1, acc: Optional[int] = None,
                        mode: int = RIDGE_ABSOLUTE, dW=None, info=None, workspace=None,
                        stream=None):
    """One block's patch dW [d, d] fp32; returns (dW, info)."""
    torch = _torch()
    _require_gpu(Q, K, V, W, idx, Kc, Vc, dW, info)
    M, Hq, dh = Q.shape
    Hkv, N, _ = K.shape
    B = idx.shape[0] if idx is not None else Kc.shape[1]
    dt = _dtype_code(Q)
    if acc is None:
        acc = F64 if dt == F32 else F32
    scale = 1.0 / dh ** 0.5 if scale is None else scale
    d = Hq * dh
    if dW is None:
        dW = torch.empty((d, d), dtype=torch.float32, device=Q.device)
    if info is None:
        info = torch.empty((1,), dtype=torch.int32, device=Q.device)
    L = lib()
    nb = L.patchkv_layer_workspace_bytes(dt, acc, M, N, B, Hq, Hkv, dh)
    ws = workspace if workspace is not None else _workspace(nb, Q.device, stream)
    wsz = ws.numel() * ws.element_size() if ws is not None else 0
    _check("patchkv_compute_layer_patch",
           L.patchkv_compute_layer_patch(dt, acc, _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), _ptr(Kc),
                                         _ptr(Vc), _ptr(W), M, N, B, Hq, Hkv, dh, scale, rho, lam,
                                         mode, _ptr(dW), _ptr(info), _ptr(ws), wsz,
                                         _stream(stream)))
    return dW, info
