"""fp64 CPU oracle for the PatchKV context-loading path.

TEST INFRASTRUCTURE ONLY. This module is the correctness reference for the GPU
library. Only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import it; the product path never calls it and never falls back to it.
It shares no code with the GPU implementation: it reads the seeded inputs
(raw bf16 bit patterns or float32 values) and decodes them itself.

What it computes, per transformer block (paper, Sec. 2.2-2.3 and Alg. 1):

  (a1) teacher attention: every reference query attends over the full cache;
  (a2) student attention: the same queries over the compressed cache;
  (a3) per-token targets t_i = W (h_i - h'_i) + (z_i - z'_i)            (Eq. 5);
  (a4) sufficient statistics S_H = H'^T H', S_T = T^T H', summed over
       reference chunks starting from zero                              (Eq. 9);
  (a5) ridge patch  Delta W = S_T (S_H + lambda I)^{-1}                 (Eq. 8),
       with lambda absolute or adaptive, lambda_0 ||S_H||_F^2 / tr S_H   (Eq. 7).

and, for a reference set split into chunks (Sec. 2.3, chunked query encoding;
Alg. 1, the loop over reference chunks):

  (f2) each chunk's tokens attend over the cache and over the chunk's own
       causal prefix (cross-chunk attention dropped); the statistics of all
       chunks are summed before the single solve.

and, for the MLP-shaped patch of the paper's own block (Sec. 2.2; Alg. 1):

  (f3) h = SwiGLU features of the normalised attention output, W the
       d_ff x d down-projection, z the attention output; targets
       t = W (h - h') + (z - z'), a d_ff x d patch, and the student state the
       patched block passes on, h' (W + Delta W) + z'.

Readings where the paper is silent (each is also listed in the design notes):

* Row-vector orientation. Activations are rows (one token per row), so with
  X = H' (tokens x d_in) and T (tokens x d_out) the statistics are
  G = X^T X (= S_H) and C = X^T T (= S_T^T), and the returned patch is
  Delta W = (G + lambda I)^{-1} C, the transpose of the paper's column-vector
  Delta W. The patched layer computes X (W + Delta W) (+ rho X).
* Synthetic block: the block has no MLP; the patched projection W is d x d and
  both h and z are the concatenated attention heads O (z is the attention output
  in Sec. 2.2). Eq. 5 then reads T = (O_f - O_c) W + rho (O_f - O_c) with
  rho = 1; rho = 0 gives the pure projection form.
* Attention: every query attends to every cache entry (no mask, RoPE already
  applied), softmax scale 1/sqrt(dh) unless given, GQA query head h reads KV
  head floor(h / (Hq / Hkv)).
* MLP block (f3): the MLP reads the attention output through an RMS norm with
  unit gain and eps = 1e-5, u = z / sqrt(mean(z^2) + eps), then
  h = silu(u W_gate) * (u W_up), silu(x) = x / (1 + e^-x), and the block output
  is y = h W + z (Llama- and Qwen-style SwiGLU; the block's own input and the
  output projection of attention are folded into z).
* Chunked reference set: token m of a chunk also attends to the chunk's own
  tokens 0..m (its causal prefix, itself included), whose keys and values the
  caller supplies. At the first block the teacher's and the student's chunk
  states coincide (both are the token embeddings), so the same own keys and
  values serve both passes there; in general each pass takes its own.

Parity pins for every function live in the CPU test suite (closed forms,
invariants, brute force, library routines, hand-written bf16 bit patterns, and
the whole block composed from independently written pieces).
"""
from __future__ import annotations

import numpy as np
import scipy.linalg

__all__ = [
    "decode", "softmax_rows", "attention", "gather_cache", "targets",
    "normal_equations", "normal_equations_chunked", "ridge_lambda", "solve_patch",
    "layer_patch", "attention_rows", "attention_chunk", "layer_patch_chunked", "rms_norm",
    "silu", "mlp_features", "block_targets", "propagate_student", "mlp_layer_patch",
    "dequantize_mx", "low_rank_patch",
]


def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored input -> float64, exactly.

    ``dtype == "bf16"``: x holds bf16 bit patterns (uint16); the value is the
    float32 whose upper 16 bits are those bits. ``"f32"``: x holds float32.
    """
    if dtype == "bf16":
        a = np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return a.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "f64":
        return np.asarray(x, dtype=np.float64)
    raise ValueError(dtype)


def softmax_rows(S: np.ndarray) -> np.ndarray:
    """Row-wise softmax, two passes: subtract the row max, exponentiate, normalise."""
    S = S - S.max(axis=1, keepdims=True)
    P = np.exp(S)
    P /= P.sum(axis=1, keepdims=True)
    return P


def attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float | None = None,
              max_score_bytes: int = 1 << 28, bias: np.ndarray | None = None) -> np.ndarray:
    """Reference-query attention over one cache (teacher Alg. 1 / student Alg. 1).

    Q [M, Hq, dh], K and V [Hkv, Nk, dh], all float64; K and V may also be
    sequences of Hkv arrays [Nk_g, dh] (a compressed cache whose KV heads keep
    different numbers of entries). Returns O [M, Hq*dh] with
    O[m, h*dh:(h+1)*dh] = softmax(scale * Q[m,h] K[g]^T + bias[g]) V[g],
    g = floor(h / (Hq/Hkv)); ``bias`` [Hkv, Nk] (natural-log units, default none)
    is a per-entry logit bias, as an attention-matching compressed cache carries
    with its entries (Sec. 3.1). Rows are processed in chunks only to bound memory.
    """
    M, Hq, dh = Q.shape
    Hkv = len(K)
    if len(V) != Hkv or Hkv == 0 or Hq % Hkv:
        raise ValueError("shape mismatch")
    for g in range(Hkv):
        if K[g].ndim != 2 or K[g].shape[1] != dh or V[g].shape != K[g].shape:
            raise ValueError("shape mismatch")
    Nk = max(K[g].shape[0] for g in range(Hkv))
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    group = Hq // Hkv
    O = np.empty((M, Hq * dh), dtype=np.float64)
    rows = max(1, min(M, max_score_bytes // (8 * max(Nk, 1))))
    for h in range(Hq):
        g = h // group
        for r0 in range(0, M, rows):
            r1 = min(M, r0 + rows)
            S = (Q[r0:r1, h, :] @ K[g].T) * scale
            if bias is not None:
                S = S + bias[g][None, :]
            O[r0:r1, h * dh:(h + 1) * dh] = softmax_rows(S) @ V[g]
    return O


def dequantize_mx(q: np.ndarray, e: np.ndarray, block: int = 32) -> np.ndarray:
    """A block-scaled integer cache entry (App. C, quantized KV caches) as float64:
    value = q * 2^e, q [..., dh] integers, e [..., dh / block] one power-of-two
    exponent per block of ``block`` consecutive channels."""
    q = np.asarray(q, dtype=np.float64)
    scale = np.exp2(np.repeat(np.asarray(e, dtype=np.float64), block, axis=-1))
    return q * scale


def attention_rows(Q: np.ndarray, K: np.ndarray, V: np.ndarray, rows: np.ndarray,
                   scale: float | None = None) -> np.ndarray:
    """Attention output of a subset of query rows (each row is independent)."""
    return attention(Q[np.asarray(rows)], K, V, scale)


def attention_chunk(Q: np.ndarray, K: np.ndarray, V: np.ndarray, Ks: np.ndarray,
                    Vs: np.ndarray, scale: float | None = None,
                    max_score_bytes: int = 1 << 28) -> np.ndarray:
    """One reference chunk's attention (Sec. 2.3, chunked query encoding; Alg. 1).

    Q [Mc, Hq, dh] are the chunk's queries, K and V [Hkv, Nk, dh] the cache (full
    or compressed), Ks and Vs [Hkv, Mc, dh] the chunk's own keys and values. Query
    m attends over all Nk cache entries and over its own entries 0..m: the own
    entries m+1.. get a score of -inf before the softmax. Returns O [Mc, Hq*dh].
    """
    M, Hq, dh = Q.shape
    Hkv = len(K)
    if len(V) != Hkv or Ks.shape != (Hkv, M, dh) or Vs.shape != Ks.shape:
        raise ValueError("shape mismatch")
    for g in range(Hkv):
        if K[g].ndim != 2 or K[g].shape[1] != dh or V[g].shape != K[g].shape:
            raise ValueError("shape mismatch")
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    if scale is None:
        scale = 1.0 / np.sqrt(dh)
    group = Hq // Hkv
    O = np.empty((M, Hq * dh), dtype=np.float64)
    rows = max(1, min(M, max_score_bytes // (8 * (max(k.shape[0] for k in K) + M))))
    for h in range(Hq):
        g = h // group
        Nk = K[g].shape[0]
        Kall = np.concatenate([K[g], Ks[g]], axis=0)     # [Nk + M, dh]
        Vall = np.concatenate([V[g], Vs[g]], axis=0)
        for r0 in range(0, M, rows):
            r1 = min(M, r0 + rows)
            S = (Q[r0:r1, h, :] @ Kall.T) * scale
            own = np.arange(M)[None, :]                  # own entry index j
            query = np.arange(r0, r1)[:, None]           # query position m
            S[:, Nk:][own > query] = -np.inf
            O[r0:r1, h * dh:(h + 1) * dh] = softmax_rows(S) @ Vall
    return O


def gather_cache(K: np.ndarray, V: np.ndarray, idx: np.ndarray, counts=None):
    """Eviction-style compressed cache: the kept entries of K, V [Hkv, N, dh].

    ``idx`` [B], one set for every KV head: K[:, idx], V[:, idx]. ``idx`` [Hkv, B],
    one set per KV head (KVzip's global head scoring, App. B.1, keeps different
    tokens in different heads): head g keeps rows idx[g, :counts[g]] of K[g], V[g]
    (all B when ``counts`` is None); the result is then a pair of lists of per-head
    arrays, which ``attention`` accepts.
    """
    idx = np.asarray(idx)
    if idx.ndim == 1 and counts is None:
        return K[:, idx, :], V[:, idx, :]
    Hkv = K.shape[0]
    sets = [idx] * Hkv if idx.ndim == 1 else [idx[g] for g in range(Hkv)]
    if counts is not None:
        sets = [sets[g][:int(counts[g])] for g in range(Hkv)]
    return [K[g][sets[g]] for g in range(Hkv)], [V[g][sets[g]] for g in range(Hkv)]


def targets(Of: np.ndarray, Oc: np.ndarray, W: np.ndarray, rho: int = 1) -> np.ndarray:
    """Per-token targets of Eq. 5 in row form: T = (O_f - O_c) W + rho (O_f - O_c).

    h - h' = O_f - O_c enters through the patched projection W; z - z' = O_f - O_c
    is the residual attention-output term (present when rho = 1).
    """
    D = Of - Oc
    T = D @ W
    if rho:
        if W.shape[0] != W.shape[1]:
            raise ValueError("the residual term needs a square W")
        T = T + rho * D
    return T


def normal_equations(Xc: np.ndarray, T: np.ndarray):
    """Sufficient statistics of Eq. 9 in row form: G = Xc^T Xc, C = Xc^T T."""
    return Xc.T @ Xc, Xc.T @ T


def normal_equations_chunked(chunks):
    """Eq. 9 accumulated over reference chunks, starting from zero (Alg. 1).

    ``chunks`` yields (Xc_j, T_j) pairs; each chunk's outer-product sums are added
    to running totals and the chunk is then dropped.
    """
    G = C = None
    for Xj, Tj in chunks:
        if G is None:
            G = np.zeros((Xj.shape[1], Xj.shape[1]))
            C = np.zeros((Xj.shape[1], Tj.shape[1]))
        G += Xj.T @ Xj
        C += Xj.T @ Tj
    return G, C


def ridge_lambda(G0: np.ndarray, lam: float, mode: str = "absolute") -> float:
    """The ridge coefficient: absolute; adaptive per Eq. 7, lambda_0 ||G||_F^2 / tr G; or the
    trace mean lambda_0 tr G / d (the mean eigenvalue, the alternative scaling of the
    paper's ridge-scaling ablation). For the last two, lam is lambda_0."""
    if mode == "absolute":
        return float(lam)
    if mode == "adaptive":
        return float(lam) * float(np.sum(G0 * G0)) / float(np.trace(G0))
    if mode == "trace_mean":
        return float(lam) * float(np.trace(G0)) / G0.shape[0]
    raise ValueError(mode)


def solve_patch(G0: np.ndarray, C: np.ndarray, lam: float) -> np.ndarray:
    """Eq. 8 in row form: Delta W = (G0 + lam I)^{-1} C, via LAPACK Cholesky."""
    if not lam > 0:
        raise ValueError("ridge coefficient must be positive")
    A = G0 + lam * np.eye(G0.shape[0])
    return scipy.linalg.cho_solve(scipy.linalg.cho_factor(A, lower=True), C)


def layer_patch(inp, rho: int = 1, mode: str = "absolute", lam: float | None = None,
                keep: bool = True, cache=None, bias: np.ndarray | None = None) -> dict:
    """One block's patch from a ``workloads`` LayerInputs (all steps in fp64).

    ``cache`` = (Kc, Vc) float64 replaces the layer's own compressed cache (e.g. a
    dequantized one); ``bias`` [Hkv, B] is its per-entry logit bias. Returns a dict
    with dW and, when ``keep``, the intermediates O_f, O_c, T, G (without the
    ridge), C and the lambda used.
    """
    dt = inp.dtype
    Q = decode(inp.Q, dt)
    K = decode(inp.K, dt)
    V = decode(inp.V, dt)
    W = decode(inp.W, dt)
    Of = attention(Q, K, V, inp.scale)
    if cache is not None:
        Kc, Vc = cache
    elif inp.idx is not None:
        Kc, Vc = gather_cache(K, V, inp.idx, inp.counts)
    else:
        Kc, Vc = decode(inp.Kc, dt), decode(inp.Vc, dt)
    del K, V
    Oc = attention(Q, Kc, Vc, inp.scale, bias=bias)
    T = targets(Of, Oc, W, rho)
    G0, C = normal_equations(Oc, T)
    lam_used = ridge_lambda(G0, inp.lam if lam is None else lam, mode)
    dW = solve_patch(G0, C, lam_used)
    out = {"dW": dW, "lam": lam_used}
    if keep:
        out.update(Of=Of, Oc=Oc, T=T, G=G0, C=C)
    return out


def layer_patch_chunked(inp, chunks, rho: int = 1, mode: str = "absolute",
                        lam: float | None = None) -> dict:
    """One block's patch from a reference set split into chunks (Sec. 2.3; Alg. 1).

    ``inp`` is a ``workloads`` LayerInputs (the cache, the compressed cache and W);
    ``chunks`` yields per-chunk (Q, Ks, Vs) in the same stored form. For every chunk
    the teacher pass attends over the full cache and the student pass over the
    compressed cache, both plus the chunk's causal prefix; the chunk's targets and
    statistics are formed and added to running sums that start from zero; one
    ridge solve follows. Returns dW, lambda, G (without the ridge) and C.
    """
    dt = inp.dtype
    K = decode(inp.K, dt)
    V = decode(inp.V, dt)
    W = decode(inp.W, dt)
    if inp.idx is not None:
        Kc, Vc = gather_cache(K, V, inp.idx, inp.counts)
    else:
        Kc, Vc = decode(inp.Kc, dt), decode(inp.Vc, dt)
    G0 = np.zeros((W.shape[0], W.shape[0]))
    C = np.zeros((W.shape[0], W.shape[1]))
    for Qj, Ksj, Vsj in chunks:
        Qj, Ksj, Vsj = decode(Qj, dt), decode(Ksj, dt), decode(Vsj, dt)
        Of = attention_chunk(Qj, K, V, Ksj, Vsj, inp.scale)
        Oc = attention_chunk(Qj, Kc, Vc, Ksj, Vsj, inp.scale)
        T = targets(Of, Oc, W, rho)
        Gj, Cj = normal_equations(Oc, T)
        G0 += Gj
        C += Cj
    lam_used = ridge_lambda(G0, inp.lam if lam is None else lam, mode)
    return {"dW": solve_patch(G0, C, lam_used), "lam": lam_used, "G": G0, "C": C}


def rms_norm(X: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """Row-wise RMS normalisation with unit gain: x / sqrt(mean(x^2) + eps)."""
    return X / np.sqrt(np.mean(X * X, axis=1, keepdims=True) + eps)


def silu(X: np.ndarray) -> np.ndarray:
    """x * sigmoid(x) = x / (1 + e^-x)."""
    return X / (1.0 + np.exp(-X))


def mlp_features(Z: np.ndarray, Wg: np.ndarray, Wu: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """The post-activation MLP intermediate h of Sec. 2.2 for a SwiGLU block whose
    MLP reads the attention output z: u = rms_norm(z), h = silu(u Wg) * (u Wu).
    Z [M, d], Wg and Wu [d, d_ff]; returns H [M, d_ff]."""
    U = rms_norm(Z, eps)
    return silu(U @ Wg) * (U @ Wu)


def block_targets(Hf: np.ndarray, Hc: np.ndarray, W: np.ndarray, Zf: np.ndarray,
                  Zc: np.ndarray) -> np.ndarray:
    """Eq. 5 for the MLP-shaped block, row form: T = (Hf - Hc) W + (Zf - Zc), with
    W [d_ff, d] the down-projection and Z the attention outputs."""
    return (Hf - Hc) @ W + (Zf - Zc)


def propagate_student(Hc: np.ndarray, W: np.ndarray, dW: np.ndarray, Zc: np.ndarray) -> np.ndarray:
    """Student-state propagation (Alg. 1): the patched block's output on the
    student's activations, Hc (W + dW) + Zc, the next block's student input."""
    return Hc @ (W + dW) + Zc


def mlp_layer_patch(inp, mlp, mode: str = "absolute", lam: float | None = None) -> dict:
    """The MLP-shaped patch of one block (Sec. 2.2; Alg. 1), all in fp64.

    ``inp``: a ``workloads`` LayerInputs (queries, caches); ``mlp``: MlpWeights
    with Wg, Wu [d, d_ff] and Wd [d_ff, d] (stored form) and eps. Teacher and
    student attention give z = O_f, O_c; h = mlp_features(z); the patch solves
    Eq. 8 with G = Hc^T Hc, C = Hc^T T; the student state is propagated through
    the patched block. Returns dW [d_ff, d], Y_student, Y_teacher, lambda, G, C.
    """
    dt = inp.dtype
    Q, K, V = decode(inp.Q, dt), decode(inp.K, dt), decode(inp.V, dt)
    Wg, Wu, Wd = decode(mlp.Wg, dt), decode(mlp.Wu, dt), decode(mlp.Wd, dt)
    Of = attention(Q, K, V, inp.scale)
    if inp.idx is not None:
        Kc, Vc = gather_cache(K, V, inp.idx, inp.counts)
    else:
        Kc, Vc = decode(inp.Kc, dt), decode(inp.Vc, dt)
    del K, V
    Oc = attention(Q, Kc, Vc, inp.scale)
    Hf = mlp_features(Of, Wg, Wu, mlp.eps)
    Hc = mlp_features(Oc, Wg, Wu, mlp.eps)
    T = block_targets(Hf, Hc, Wd, Of, Oc)
    G0, C = normal_equations(Hc, T)
    lam_used = ridge_lambda(G0, inp.lam if lam is None else lam, mode)
    dW = solve_patch(G0, C, lam_used)
    return {"dW": dW, "lam": lam_used, "G": G0, "C": C,
            "Y_student": propagate_student(Hc, Wd, dW, Oc), "Y_teacher": Hf @ Wd + Of}


def low_rank_patch(G0: np.ndarray, dW: np.ndarray, r: int) -> dict:
    """The reduced-rank patch (App. C, low-rank weight patches; reduced-rank regression).

    In the paper's column form the ridge patch is projected onto its top-r output
    subspace, U_r U_r^T dW, with U_r the top-r eigenvectors of dW S_H dW^T. In row
    form (dW [d_in, d_out], G0 = S_H) that is dW_r = dW U_r U_r^T with U_r [d_out, r]
    the top-r eigenvectors of dW^T G0 dW, the covariance of the fitted targets.
    Returns dW_r, the factors A = dW U_r [d_in, r] and U_r, and all eigenvalues in
    descending order (LAPACK eigh).
    """
    S = dW.T @ G0 @ dW
    w, V = np.linalg.eigh(S)
    U = V[:, ::-1][:, :r]
    return {"dW": dW @ U @ U.T, "A": dW @ U, "U": U, "eig": w[::-1].copy()}
