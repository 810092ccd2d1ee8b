"""The fingerprint workloads: layer-stack shapes and request sizes (data only).

Both the oracle and the benchmark read this table; it holds no arithmetic of the
method.  Each workload is a fingerprint of a Llama-2-style model under one of the
compression settings the paper searches over (Sec. 3.2, Table A.1): the number of
hidden layers kept, the layer shape, the weight and KV-cache formats, and one
dummy request of B sequences with a P-token prompt followed by S decode steps
(Sec. 5.3).  The cache holds P + S positions.
"""
from __future__ import annotations

import dataclasses


@dataclasses.dataclass(frozen=True)
class Shape:
    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    max_batch: int
    max_prompt: int
    max_seq: int
    rms_eps: float = 1e-5
    rope_theta: float = 1e4
    vocab: int = 0          # > 0: the fingerprint also holds embedding, final norm and LM head

    @property
    def q_dim(self):
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self):
        return self.n_kv_heads * self.head_dim


def _cfg(L, H, nh, nkv, d, F, wq, kvq, B, P, S):
    return dict(shape=Shape(L, H, nh, nkv, d, F, B, P, P + S), wq=wq, kvq=kvq, B=B, P=P, S=S)


# name: (layers, hidden, heads, kv heads, head_dim, ffn, weights, KV cache, batch, prompt, steps)
CONFIGS = {
    "tiny": _cfg(1, 256, 4, 4, 64, 688, "bf16", "bf16", 1, 32, 16),
    "llama2-7b-bf16": _cfg(2, 4096, 32, 32, 128, 11008, "bf16", "bf16", 1, 512, 100),
    "llama2-7b-int8": _cfg(2, 4096, 32, 32, 128, 11008, "int8", "int8", 16, 512, 100),
    "llama2-13b-int4": _cfg(4, 5120, 40, 40, 128, 13824, "int4", "bf16", 32, 1024, 100),
    "llama2-70b-tp8-int4": _cfg(4, 8192, 8, 1, 128, 3584, "int4", "int8", 64, 2048, 100),
    # 2:4 semi-structured sparse bf16 weights (pruning, Sec. 3.3), the 7B shape at batch 16
    "llama2-7b-sp24": _cfg(2, 4096, 32, 32, 128, 11008, "sp24", "bf16", 16, 512, 100),
}

# The workload the benchmark's headline is quoted on: the largest model, prompt, batch
# and prefill that fits one GPU (a 1/8 tensor-parallel shard of the 70B model).
HEADLINE = "llama2-70b-tp8-int4"

# Llama-2 vocabulary size, for fingerprints that keep the embedding and LM head.
LLAMA2_VOCAB = 32000
