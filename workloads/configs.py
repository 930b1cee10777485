"""The synthetic workload shapes.

Each stands in for a setting the paper measures (Sec. 3.1 and App. C): contexts up to
~170K tokens, aggressive cache budgets (down to ~1 % of the context), and one
reference chunk of a few thousand query tokens per block. The model shapes are
those of Llama-3-8B (d=4096, 32 query / 8 KV heads, head_dim 128) and Qwen-2.5-7B
(d=3584, 28 / 4 heads), plus a tiny fp32 layer that a CPU finishes in seconds.

Compressed-cache structure:
  * "evict":      B = n_sink sink tokens + the last n_recent tokens + n_random
                  seeded-random middle positions (sorted), i.e. an eviction subset
                  of the full cache, standing in for KVzip's output.
  * "evict_heads": per-KV-head eviction subsets whose sizes differ between heads
                  (B entries per head on average), standing in for KVzip's global
                  head scoring: sinks and recent tokens in every head, the middle
                  budget shared out over the heads.
  * "synthesize": B synthetic entries, each a seeded-random convex combination of
                  n_mix full-cache entries, standing in for an approximation method
                  (Attention Matching) whose entries are not a subset.
  * "identity":   every position (B = N); with kv_format "mxint8" / "mxint4" the
                  compression is the quantization of the whole context (App. C).
"""
from dataclasses import dataclass


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    d: int            # model width = Hq * dh
    Hq: int
    Hkv: int
    dh: int
    N: int            # full-cache tokens
    B: int            # compressed-cache entries
    M: int            # reference query tokens
    lam: float        # absolute ridge coefficient
    dtype: str        # "f32" or "bf16" (Q, K, V and W)
    layers: int = 1
    cache: str = "evict"     # "evict" | "evict_heads" | "synthesize" | "identity"
    n_sink: int = 0
    n_recent: int = 0
    n_random: int = 0
    n_mix: int = 0           # synthesize: entries mixed per synthetic entry
    chunks: int = 1          # reference chunks per layer (M tokens each, own causal prefix)
    d_ff: int = 0            # > 0: patch the d_ff x d down-projection of a SwiGLU MLP
    ridge: str = "absolute"  # "absolute": lam is lambda; "adaptive": lam is lambda_0 of Eq. 7
    rank: int = 0            # > 0: also the reduced-rank patch of this rank
    kv_format: str = "plain" # compressed cache storage: "plain", "mxint8" or "mxint4"
    cache_bias: bool = False # compressed cache entries carry a logit bias
    # 2: the full-cache (teacher) pass also forms P V from a two-term bf16 split of P.
    # Needed where O_f - O_c is small next to O_f (int8 quantization of the whole
    # context changes O by ~2 %): P rounded to bf16 (~1.6e-3 relative error in O_f)
    # would then be ~8 % of the targets.
    teacher_p_terms: int = 1

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv

    @property
    def scale(self) -> float:
        return 1.0 / float(self.dh) ** 0.5

    @property
    def acc(self) -> str:
        """Accumulation type of the normal equations for this input dtype."""
        return "f64" if self.dtype == "f32" else "f32"


CONFIGS = (
    Config(0, "tiny-fp32", d=256, Hq=4, Hkv=2, dh=64, N=2048, B=256, M=128,
           lam=1e-2, dtype="f32", n_sink=4, n_recent=124, n_random=128),
    Config(1, "llama3-8b-layer-32k", d=4096, Hq=32, Hkv=8, dh=128, N=32768, B=2048,
           M=1024, lam=1e-1, dtype="bf16", n_sink=4, n_recent=1020, n_random=1024),
    Config(2, "llama3-8b-layer-128k", d=4096, Hq=32, Hkv=8, dh=128, N=131072, B=4096,
           M=2048, lam=1e-1, dtype="bf16", n_sink=4, n_recent=2044, n_random=2048),
    Config(3, "llama3-8b-32layer-172k", d=4096, Hq=32, Hkv=8, dh=128, N=172032,
           B=1720, M=4096, lam=1e-1, dtype="bf16", layers=32, n_sink=4, n_recent=860,
           n_random=856),
    Config(4, "qwen2.5-7b-layer-64k-synth", d=3584, Hq=28, Hkv=4, dh=128, N=65536,
           B=1024, M=2048, lam=5e-2, dtype="bf16", cache="synthesize", n_mix=64),
    # chunked reference set: 4 chunks of 5,120 tokens (the paper's default chunk
    # size), each attending over the cache plus its own causal prefix
    Config(5, "llama3-8b-layer-172k-4x5k-chunks", d=4096, Hq=32, Hkv=8, dh=128, N=172032,
           B=1720, M=5120, lam=1e-1, dtype="bf16", chunks=4, n_sink=4, n_recent=860,
           n_random=856),
    # the paper's own block: the patch is the 14336 x 4096 down-projection of
    # Llama-3-8B's SwiGLU MLP, fed by the attention output of config 3's layer, with
    # the paper's adaptive ridge (Eq. 7), lambda_0 = 1e-3
    Config(6, "llama3-8b-mlp-layer-172k", d=4096, Hq=32, Hkv=8, dh=128, N=172032, B=1720,
           M=4096, lam=1e-3, dtype="bf16", d_ff=14336, ridge="adaptive", n_sink=4, n_recent=860,
           n_random=856),
    # config 3's build with every patch also reduced to rank 32 (the paper's low-rank
    # variant: (d + d) * 32 numbers per patch instead of d * d)
    Config(7, "llama3-8b-32layer-172k-rank32", d=4096, Hq=32, Hkv=8, dh=128, N=172032, B=1720,
           M=4096, lam=1e-1, dtype="bf16", layers=32, rank=32, n_sink=4, n_recent=860,
           n_random=856),
    # config 4 with an attention-matching style compressed cache: synthesized entries
    # with a per-entry logit bias, stored as block-scaled int8 (MX-style)
    Config(8, "qwen2.5-7b-layer-64k-synth-bias-mxint8", d=3584, Hq=28, Hkv=4, dh=128, N=65536,
           B=1024, M=2048, lam=5e-2, dtype="bf16", cache="synthesize", n_mix=64,
           kv_format="mxint8", cache_bias=True),
    # config 3's 32-layer build with per-KV-head eviction sets (KVzip's global head
    # scoring): 1,720 entries per head on average, the counts differing between heads
    Config(9, "llama3-8b-32layer-172k-headwise", d=4096, Hq=32, Hkv=8, dh=128, N=172032,
           B=1720, M=4096, lam=1e-1, dtype="bf16", layers=32, cache="evict_heads", n_sink=4,
           n_recent=860, n_random=856),
    # quantization as the compression: the student cache is the whole 172,032-token
    # context in block-scaled int8 (int4), read by the attention kernels as stored
    Config(10, "llama3-8b-layer-172k-context-mxint8", d=4096, Hq=32, Hkv=8, dh=128, N=172032,
           B=172032, M=4096, lam=1e-1, dtype="bf16", cache="identity", kv_format="mxint8",
           teacher_p_terms=2),
    Config(11, "llama3-8b-layer-172k-context-mxint4", d=4096, Hq=32, Hkv=8, dh=128, N=172032,
           B=172032, M=4096, lam=1e-1, dtype="bf16", cache="identity", kv_format="mxint4"),
)


def get_config(cid: int) -> Config:
    return CONFIGS[cid]
