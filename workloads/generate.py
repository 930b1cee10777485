"""Seeded input generation.

Recipe (the same bytes feed the oracle and the GPU path):

* Every random tensor has a tensor id: 0 key scales, 1 K, 2 V, 3 Q, 4 W,
  5 eviction middle positions, 6 synthesis positions, 7 synthesis weights;
  8 MLP gate projection, 9 MLP up projection, 10 MLP down projection,
  11 the compressed cache's per-entry logit bias, 12 the per-head budget shares
  of per-head eviction sets, 13 (block g) the middle positions of KV head g;
  reference chunk j of a chunked reference set: 16 + 4j its queries, 17 + 4j its
  own keys, 18 + 4j its own values.
* Normal tensors are drawn in C order in blocks of ``BLOCK`` elements; block ``b``
  of tensor ``tid`` uses ``Generator(PCG64(SeedSequence([seed, cid, layer, tid, b])))``
  and ``standard_normal(n, dtype=float32)``. Blocks are independent streams, so
  they are drawn on several threads and the result does not depend on the
  thread count.
* Q, V ~ N(0, 1). K = Z * s with a per-(kv head, channel) scale
  s ~ LogNormal(0, 0.5) (float32 product). W = Z * float32(1/sqrt(d)).
  A chunk's queries and own values are N(0, 1); its own keys carry the layer's
  key scales s like the cache keys. MLP weights: gate and up [d, d_ff] are
  Z * float32(1/sqrt(d)), down [d_ff, d] is Z * float32(1/sqrt(d_ff)).
* Attention-matching logit bias of a compressed cache: per (KV head, entry)
  beta = log(n_mix) + 0.25 Z (an entry standing for n_mix originals), float32.
* Block-scaled integer cache (MX-style): per (KV head, entry) and block of 32
  channels, e = ceil(log2(max|x| / q_max)) (q_max 127 for int8, 7 for int4;
  e = 0 for an all-zero block) and q = round-half-even(x / 2^e) clipped to
  [-q_max, q_max]; int8 q as int8, int4 q packed two per byte (even channel in
  the low nibble), e as int8. q * 2^e is exact in bf16.
* bf16 tensors are rounded from those float32 values with round-to-nearest-even
  and stored as their raw uint16 bit patterns; fp32 tensors are stored as is.
* Eviction subset: ``n_sink`` sinks, the last ``n_recent`` tokens, and
  ``n_random`` positions drawn uniformly without replacement from
  [n_sink, N - n_recent), sorted ascending, int32, shared by all KV heads.
* Per-KV-head eviction subsets (standing in for KVzip's global head scoring,
  where heads compete for one budget and keep different tokens): every head keeps
  the sinks and the recent tokens; the Hkv * (B - n_sink - n_recent) middle slots
  of the total budget are shared out over the heads in proportion to a
  LogNormal(0, 0.5) weight per head (largest remainders round; no head takes more
  than the N - n_sink - n_recent middle positions there are), and head g draws its
  share uniformly without replacement from the middle positions. Each head's set
  is sorted; the sets are stored as int32 [Hkv, B_max] padded with -1 past each
  head's count, with the counts as int32 [Hkv].
* Synthesized compressed cache: entry b mixes ``n_mix`` distinct full-cache
  positions (uniform without replacement over [0, N)) with weights u / sum(u),
  u ~ U(0, 1). The mix is formed in float64 from the (already rounded) K and V,
  shared by all KV heads, then rounded to float32 (RNE) and, for bf16, to bf16
  (RNE).
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, field
from typing import Callable, Optional

import numpy as np
from numpy.random import PCG64, Generator, SeedSequence

from .configs import Config

BLOCK = 1 << 22

TID_SCALE, TID_K, TID_V, TID_Q, TID_W, TID_EVICT, TID_SYN_POS, TID_SYN_W = range(8)
TID_GATE, TID_UP, TID_DOWN, TID_BIAS = 8, 9, 10, 11
TID_HEAD_SHARE, TID_HEAD_EVICT = 12, 13
TID_CHUNK = 16  # chunk j: 16 + 4j queries, 17 + 4j own keys, 18 + 4j own values


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _rng(seed: int, cid: int, layer: int, tid: int, block: int = 0) -> Generator:
    return Generator(PCG64(SeedSequence([seed, cid, layer, tid, block])))


def bf16_round_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_tensor(seed: int, cid: int, layer: int, tid: int, shape: tuple,
                   bf16: bool, post: Optional[Callable[[np.ndarray, int], np.ndarray]] = None
                   ) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
    nblk = (n + BLOCK - 1) // BLOCK

    def work(b: int) -> None:
        lo = b * BLOCK
        hi = min(n, lo + BLOCK)
        z = _rng(seed, cid, layer, tid, b).standard_normal(hi - lo, dtype=np.float32)
        if post is not None:
            z = post(z, lo)
        out[lo:hi] = bf16_round_bits(z) if bf16 else z

    if nblk == 1:
        work(0)
    else:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(work, range(nblk)))
    return out.reshape(shape)


@dataclass
class LayerInputs:
    """One layer's inputs. bf16 tensors hold uint16 bit patterns."""
    cid: int
    layer: int
    dtype: str                   # "bf16" or "f32"
    M: int
    N: int
    B: int
    Hq: int
    Hkv: int
    dh: int
    lam: float
    scale: float
    Q: np.ndarray                # [M, Hq, dh]
    K: np.ndarray                # [Hkv, N, dh]
    V: np.ndarray                # [Hkv, N, dh]
    W: np.ndarray                # [d, d]
    idx: Optional[np.ndarray] = None   # [B] or per KV head [Hkv, B] int32 (eviction), or None
    Kc: Optional[np.ndarray] = None    # [Hkv, B, dh] (synthesized) or None
    Vc: Optional[np.ndarray] = None
    counts: Optional[np.ndarray] = None  # [Hkv] int32 entries kept per head (per-head sets)
    extra: dict = field(default_factory=dict)

    @property
    def d(self) -> int:
        return self.Hq * self.dh


def _eviction_idx(rng: Generator, N: int, n_sink: int, n_recent: int, n_random: int) -> np.ndarray:
    if n_sink + n_recent + n_random > N:
        raise ValueError("eviction subset larger than the cache")
    mid = rng.choice(np.arange(n_sink, N - n_recent, dtype=np.int64), size=n_random, replace=False)
    idx = np.concatenate([np.arange(n_sink, dtype=np.int64), mid,
                          np.arange(N - n_recent, N, dtype=np.int64)])
    idx.sort()
    return idx.astype(np.int32)


def _shares(total: int, weights: np.ndarray, cap: int) -> np.ndarray:
    """Split ``total`` slots over the heads in proportion to ``weights`` (largest
    remainders round), no head above ``cap``."""
    n = np.zeros(len(weights), dtype=np.int64)
    open_ = np.ones(len(weights), dtype=bool)
    left = total
    while left > 0 and open_.any():
        w = np.where(open_, weights, 0.0)
        exact = left * w / w.sum()
        add = np.floor(exact).astype(np.int64)
        rem = left - int(add.sum())
        order = np.argsort(-(exact - add), kind="stable")
        add[order[:rem]] += 1
        add = np.minimum(add, cap - n)
        n += add
        left -= int(add.sum())
        open_ &= n < cap
    return n


def _eviction_idx_heads(seed: int, cid: int, layer: int, Hkv: int, N: int, B: int,
                        n_sink: int, n_recent: int):
    if n_sink + n_recent > B or B > N:
        raise ValueError("eviction budget inconsistent with the cache")
    cap = N - n_sink - n_recent
    w = _rng(seed, cid, layer, TID_HEAD_SHARE).lognormal(0.0, 0.5, size=Hkv)
    mids = _shares(Hkv * (B - n_sink - n_recent), w, cap)
    sets = []
    for g in range(Hkv):
        mid = _rng(seed, cid, layer, TID_HEAD_EVICT, g).choice(
            np.arange(n_sink, N - n_recent, dtype=np.int64), size=int(mids[g]), replace=False)
        ig = np.concatenate([np.arange(n_sink, dtype=np.int64), mid,
                             np.arange(N - n_recent, N, dtype=np.int64)])
        ig.sort()
        sets.append(ig)
    counts = np.array([len(x) for x in sets], dtype=np.int32)
    idx = np.full((Hkv, int(counts.max())), -1, dtype=np.int32)
    for g, ig in enumerate(sets):
        idx[g, :len(ig)] = ig
    return idx, counts


def make_custom_inputs(*, M: int, N: int, B: int, Hq: int, Hkv: int, dh: int,
                       dtype: str = "bf16", cache: str = "evict", lam: float = 1e-1,
                       seed: int = 0, cid: int = 100, layer: int = 0,
                       n_sink: Optional[int] = None, n_recent: Optional[int] = None,
                       n_mix: int = 64, key_sigma: float = 0.5,
                       d_out: Optional[int] = None) -> LayerInputs:
    """Draw one layer of inputs of any shape with the recipe above.

    For ``cache == "evict"`` the B kept positions are ``n_sink`` sinks + ``n_recent``
    recent + the rest random (defaults: 4 sinks, half of the remainder recent).
    ``cache == "evict_heads"``: per-KV-head sets with B entries per head on average
    (``idx`` [Hkv, B_max], ``counts`` [Hkv]; the returned ``B`` is B_max).
    ``cache == "identity"`` keeps every position (B = N): the compressed cache equals
    the full cache.
    """
    if dtype not in ("bf16", "f32"):
        raise ValueError(dtype)
    bf16 = dtype == "bf16"
    d = Hq * dh
    d_out = d if d_out is None else d_out

    s = _rng(seed, cid, layer, TID_SCALE).lognormal(mean=0.0, sigma=key_sigma,
                                                    size=(Hkv, dh)).astype(np.float32)

    def scale_k(z: np.ndarray, lo: int) -> np.ndarray:
        rows = np.arange(lo // dh, (lo + z.size) // dh)
        return (z.reshape(-1, dh) * s[rows // N]).reshape(-1)

    K = _normal_tensor(seed, cid, layer, TID_K, (Hkv, N, dh), bf16, scale_k)
    V = _normal_tensor(seed, cid, layer, TID_V, (Hkv, N, dh), bf16)
    Q = _normal_tensor(seed, cid, layer, TID_Q, (M, Hq, dh), bf16)
    wscale = np.float32(1.0 / np.sqrt(d))
    W = _normal_tensor(seed, cid, layer, TID_W, (d, d_out), bf16, lambda z, lo: z * wscale)

    out = LayerInputs(cid=cid, layer=layer, dtype=dtype, M=M, N=N, B=B, Hq=Hq, Hkv=Hkv,
                      dh=dh, lam=lam, scale=1.0 / float(dh) ** 0.5, Q=Q, K=K, V=V, W=W)
    out.extra["seed"] = seed
    out.extra["key_scale"] = s
    if cache == "evict":
        ns = 4 if n_sink is None else n_sink
        ns = min(ns, B)
        nr = (B - ns) // 2 if n_recent is None else n_recent
        out.idx = _eviction_idx(_rng(seed, cid, layer, TID_EVICT), N, ns, nr, B - ns - nr)
    elif cache == "evict_heads":
        ns = min(4 if n_sink is None else n_sink, B)
        nr = (B - ns) // 2 if n_recent is None else n_recent
        out.idx, out.counts = _eviction_idx_heads(seed, cid, layer, Hkv, N, B, ns, nr)
        out.B = int(out.idx.shape[1])
        out.extra["B_mean"] = B
    elif cache == "identity":
        if B != N:
            raise ValueError("identity cache needs B == N")
        out.idx = np.arange(N, dtype=np.int32)
    elif cache == "synthesize":
        rp = _rng(seed, cid, layer, TID_SYN_POS)
        if n_mix > N:
            raise ValueError("n_mix larger than the cache")
        pos = np.stack([rp.choice(N, size=n_mix, replace=False) for _ in range(B)])
        u = _rng(seed, cid, layer, TID_SYN_W).random((B, n_mix))
        w = u / u.sum(axis=1, keepdims=True)
        out.Kc = _mix(K, pos, w, bf16)
        out.Vc = _mix(V, pos, w, bf16)
        out.extra["syn_pos"] = pos
        out.extra["syn_w"] = w
    else:
        raise ValueError(cache)
    return out


@dataclass
class ChunkInputs:
    """One reference chunk: its queries and its own keys and values."""
    chunk: int
    Q: np.ndarray                # [Mc, Hq, dh]
    Ks: np.ndarray               # [Hkv, Mc, dh]
    Vs: np.ndarray               # [Hkv, Mc, dh]


def make_chunk_inputs(inp: LayerInputs, chunk: int, M: int) -> ChunkInputs:
    """Reference chunk ``chunk`` (M tokens) of the layer ``inp``: queries, own keys
    (scaled by the layer's key scales) and own values, drawn with the recipe above."""
    bf16 = inp.dtype == "bf16"
    seed, s = inp.extra["seed"], inp.extra["key_scale"]
    Hq, Hkv, dh = inp.Hq, inp.Hkv, inp.dh
    base = TID_CHUNK + 4 * chunk

    def scale_k(z: np.ndarray, lo: int) -> np.ndarray:
        rows = np.arange(lo // dh, (lo + z.size) // dh)
        return (z.reshape(-1, dh) * s[rows // M]).reshape(-1)

    Q = _normal_tensor(seed, inp.cid, inp.layer, base, (M, Hq, dh), bf16)
    Ks = _normal_tensor(seed, inp.cid, inp.layer, base + 1, (Hkv, M, dh), bf16, scale_k)
    Vs = _normal_tensor(seed, inp.cid, inp.layer, base + 2, (Hkv, M, dh), bf16)
    return ChunkInputs(chunk=chunk, Q=Q, Ks=Ks, Vs=Vs)


@dataclass
class MlpWeights:
    """A SwiGLU MLP of one block: gate and up [d, d_ff], down [d_ff, d] (stored form)."""
    Wg: np.ndarray
    Wu: np.ndarray
    Wd: np.ndarray
    d_ff: int
    eps: float = 1e-5


def make_mlp_weights(inp: LayerInputs, d_ff: int) -> MlpWeights:
    """The MLP weights of the layer ``inp`` with intermediate width d_ff."""
    bf16 = inp.dtype == "bf16"
    seed, d = inp.extra["seed"], inp.d
    sg = np.float32(1.0 / np.sqrt(d))
    sd = np.float32(1.0 / np.sqrt(d_ff))
    Wg = _normal_tensor(seed, inp.cid, inp.layer, TID_GATE, (d, d_ff), bf16, lambda z, lo: z * sg)
    Wu = _normal_tensor(seed, inp.cid, inp.layer, TID_UP, (d, d_ff), bf16, lambda z, lo: z * sg)
    Wd = _normal_tensor(seed, inp.cid, inp.layer, TID_DOWN, (d_ff, d), bf16, lambda z, lo: z * sd)
    return MlpWeights(Wg=Wg, Wu=Wu, Wd=Wd, d_ff=d_ff)


def make_cache_bias(inp: LayerInputs, n_mix: int = 64, sigma: float = 0.25) -> np.ndarray:
    """Per-entry logit bias [Hkv, B] of the layer's compressed cache (float32)."""
    z = _rng(inp.extra["seed"], inp.cid, inp.layer, TID_BIAS).standard_normal(
        (inp.Hkv, inp.B), dtype=np.float32)
    return (np.float32(np.log(n_mix)) + np.float32(sigma) * z).astype(np.float32)


@dataclass
class QuantCache:
    """A block-scaled integer cache: q (int8 [Hkv, n, dh], or uint8 [Hkv, n, dh/2]
    holding two int4 per byte) and e (int8 [Hkv, n, dh/32]) for K and for V."""
    bits: int
    Kq: np.ndarray
    Ke: np.ndarray
    Vq: np.ndarray
    Ve: np.ndarray


def quantize_mx(X: np.ndarray, bits: int, block: int = 32):
    """float array [..., dh] -> (q, e) per the recipe above (q unpacked, int8)."""
    qmax = {8: 127, 4: 7}[bits]
    shp = X.shape
    xb = np.asarray(X, dtype=np.float64).reshape(shp[:-1] + (shp[-1] // block, block))
    amax = np.abs(xb).max(axis=-1)
    with np.errstate(divide="ignore"):
        e = np.where(amax > 0, np.ceil(np.log2(np.where(amax > 0, amax, 1.0) / qmax)), 0.0)
    q = np.clip(np.rint(xb / np.exp2(e)[..., None]), -qmax, qmax)
    return q.reshape(shp).astype(np.int8), e.astype(np.int8)


def pack_int4(q: np.ndarray) -> np.ndarray:
    """int8 values in [-8, 7] [..., dh] -> uint8 [..., dh/2], even channel in the low nibble."""
    u = (q.astype(np.int16) & 0xF).astype(np.uint8)
    return (u[..., 0::2] | (u[..., 1::2] << 4)).astype(np.uint8)


def unpack_int4(p: np.ndarray) -> np.ndarray:
    """uint8 [..., dh/2] (two int4, even channel low) -> int8 [..., dh]."""
    lo = (p & 0xF).astype(np.int16)
    hi = (p >> 4).astype(np.int16)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = np.where(lo >= 8, lo - 16, lo)
    out[..., 1::2] = np.where(hi >= 8, hi - 16, hi)
    return out


def make_cache_extras(cfg, inp: LayerInputs):
    """The compressed cache's storage and bias of a workload config: (QuantCache of
    the compressed entries or None, logit bias [Hkv, B] or None). Quantized caches
    hold the compressed entries themselves (the synthesized K_c, V_c, or the gathered
    rows of an eviction subset)."""
    qc = None
    if cfg.kv_format != "plain":
        bits = {"mxint8": 8, "mxint4": 4}[cfg.kv_format]
        if cfg.cache == "identity":  # the whole context
            Kc, Vc = inp.K, inp.V
        elif inp.idx is not None:
            Kc, Vc = inp.K[:, inp.idx], inp.V[:, inp.idx]
        else:
            Kc, Vc = inp.Kc, inp.Vc
        qc = make_quant_cache(np.ascontiguousarray(Kc), np.ascontiguousarray(Vc), bits, inp.dtype)
    bias = make_cache_bias(inp, n_mix=cfg.n_mix or 64) if cfg.cache_bias else None
    return qc, bias


def make_quant_cache(K: np.ndarray, V: np.ndarray, bits: int, dtype: str) -> QuantCache:
    """Block-scaled integer version of a cache K, V [Hkv, n, dh] (stored form)."""
    kf = bf16_bits_to_f32(K) if dtype == "bf16" else K
    vf = bf16_bits_to_f32(V) if dtype == "bf16" else V
    Kq, Ke = quantize_mx(kf, bits)
    Vq, Ve = quantize_mx(vf, bits)
    if bits == 4:
        Kq, Vq = pack_int4(Kq), pack_int4(Vq)
    return QuantCache(bits=bits, Kq=Kq, Ke=Ke, Vq=Vq, Ve=Ve)


def _mix(X: np.ndarray, pos: np.ndarray, w: np.ndarray, bf16: bool) -> np.ndarray:
    Hkv, _, dh = X.shape
    B = pos.shape[0]
    res = np.empty((Hkv, B, dh), dtype=np.uint16 if bf16 else np.float32)
    for g in range(Hkv):
        xg = bf16_bits_to_f32(X[g]) if bf16 else X[g]
        mixed = np.einsum("bi,bid->bd", w, xg[pos].astype(np.float64)).astype(np.float32)
        res[g] = bf16_round_bits(mixed) if bf16 else mixed
    return res


def make_layer_inputs(cfg: Config, layer: int = 0, seed: int = 0) -> LayerInputs:
    """Inputs of layer ``layer`` of one of the five workload configs."""
    if not 0 <= layer < cfg.layers:
        raise ValueError(f"config {cfg.cid} has {cfg.layers} layer(s)")
    if cfg.cache == "identity":
        return make_custom_inputs(M=cfg.M, N=cfg.N, B=cfg.N, Hq=cfg.Hq, Hkv=cfg.Hkv, dh=cfg.dh,
                                  dtype=cfg.dtype, cache="identity", lam=cfg.lam, seed=seed,
                                  cid=cfg.cid, layer=layer)
    if cfg.cache in ("evict", "evict_heads"):
        return make_custom_inputs(M=cfg.M, N=cfg.N, B=cfg.B, Hq=cfg.Hq, Hkv=cfg.Hkv,
                                  dh=cfg.dh, dtype=cfg.dtype, cache=cfg.cache, lam=cfg.lam,
                                  seed=seed, cid=cfg.cid, layer=layer, n_sink=cfg.n_sink,
                                  n_recent=cfg.n_recent)
    return make_custom_inputs(M=cfg.M, N=cfg.N, B=cfg.B, Hq=cfg.Hq, Hkv=cfg.Hkv, dh=cfg.dh,
                              dtype=cfg.dtype, cache="synthesize", lam=cfg.lam, seed=seed,
                              cid=cfg.cid, layer=layer, n_mix=cfg.n_mix)
