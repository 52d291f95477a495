"""Workload presets: the five batch shapes the verification path is measured on.

Each preset fixes the batch size R, the drafted tree (depth x branching, logit
scale sigma, vocabulary V), the global verification budget B (the cap of
eq. 4, counted in draft nodes), the attention head layout and the KV-prefix
length range.  Vocabulary sizes follow the model table in the paper's
appendix (Llama-3: 128256, Qwen3: 151936).  Tree defaults follow the paper's
configuration protocol (depth 8 / top-k 10 for the large-tree setting).
"""
from dataclasses import dataclass
from typing import Tuple


@dataclass(frozen=True)
class Config:
    name: str
    R: int                 # concurrent requests in the batch
    depth: int             # drafted tree depth D
    branch: int            # children per expanded node (top-k)
    sigma: float           # draft logits ~ N(0,1) * sigma
    vocab: int             # vocabulary size V
    budget: int            # global verification budget B (draft nodes)
    hq: int                # query heads
    hkv: int               # key/value heads
    head_dim: int          # head dimension (128)
    p_lo: int              # KV prefix length, inclusive range
    p_hi: int
    accept: Tuple          # ("const", p) or ("beta", a, b): P(target argmax == draft top-1)

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def nodes_per_request(self) -> int:
        # beam tree: k children of the root, then k expanded nodes per depth
        return self.branch + (self.depth - 1) * self.branch * self.branch

    @property
    def capacity(self) -> int:
        # verify rows at capacity: one root per request + at most B drafts
        return self.R + self.budget

    @property
    def mask_words(self) -> int:
        return (self.budget + 1 + 31) // 32


CONFIGS = {
    "tiny": Config("tiny", 4, 4, 4, 2.0, 32, 16, 8, 8, 128, 256, 256, ("const", 0.7)),
    "l8b": Config("l8b", 32, 6, 8, 3.0, 128256, 128, 32, 8, 128, 512, 2048, ("const", 0.65)),
    "l70b": Config("l70b", 64, 8, 8, 3.0, 128256, 256, 64, 8, 128, 1024, 4096, ("beta", 6.0, 3.0)),
    "q235b": Config("q235b", 128, 8, 10, 3.0, 151936, 256, 64, 4, 128, 1024, 8192, ("beta", 5.0, 4.0)),
    "long": Config("long", 16, 10, 6, 4.0, 151936, 192, 64, 4, 128, 16384, 32768, ("const", 0.75)),
}

ORDER = ["tiny", "l8b", "l70b", "q235b", "long"]

# Shape studies beside the five workloads: narrow GQA groups, where a stream
# has fewer rows than one 16-row matrix tile (G = 1 decode: one row per KV
# head; G = 2 with about one draft per request).  Small drafted trees (the
# shape of the attention, not the tree, is what these measure).
EXTRA_CONFIGS = {
    "g1_decode": Config("g1_decode", 64, 4, 4, 2.0, 32, 0, 8, 8, 128, 1024, 8192, ("const", 0.7)),
    "g1_tree": Config("g1_tree", 64, 4, 4, 2.0, 32, 128, 8, 8, 128, 1024, 8192, ("const", 0.7)),
    "g2_tree": Config("g2_tree", 64, 4, 4, 2.0, 32, 64, 16, 8, 128, 1024, 8192, ("const", 0.7)),
    # the Qwen3-235B-shaped batch at the share one GPU holds under 4-way tensor
    # parallelism over the KV heads: 16 query heads and one KV head
    "q235b_tp4": Config("q235b_tp4", 128, 8, 10, 3.0, 151936, 256, 16, 1, 128, 1024, 8192,
                        ("beta", 5.0, 4.0)),
}
CONFIGS.update(EXTRA_CONFIGS)

DESCRIPTION = {
    "tiny": "batch 4, tree 4x4 over vocab 32, B=16, 8q/8kv heads, prefix 256",
    "l8b": "Llama-3.1-8B-shaped layer: batch 32, tree 6x8, B=128, 32q/8kv, prefix 512-2048",
    "l70b": "Llama-3.3-70B-shaped layer: batch 64, tree 8x8, B=256, 64q/8kv, prefix 1024-4096",
    "q235b": "Qwen3-235B-A22B-shaped layer: batch 128, tree 8x10, B=256, 64q/4kv, prefix 1024-8192",
    "long": "long context: batch 16, tree 10x6, B=192, 64q/4kv, prefix 16384-32768",
    "g1_decode": "GQA group 1, decode only: batch 64, B=0, 8q/8kv, prefix 1024-8192",
    "g1_tree": "GQA group 1: batch 64, tree 4x4, B=128, 8q/8kv, prefix 1024-8192",
    "g2_tree": "GQA group 2: batch 64, tree 4x4, B=64, 16q/8kv, prefix 1024-8192",
    "q235b_tp4": "Qwen3-235B-shaped layer at a TP-4 share: batch 128, tree 8x10, B=256, 16q/1kv, prefix 1024-8192",
}
