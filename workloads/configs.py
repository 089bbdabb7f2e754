"""Model shapes and verification workloads.

Shapes are LLaMA-style decoder-only stacks (the paper's phone targets are
LLaMa2 / Vicuna 7B and 13B, Table 3; its memory-wall table adds 33B, Table 1).
The paper names the layer kinds only generically (embedding, masked
self-attention, norm, linear; §2.1).  The concrete block is RMSNorm, rotary
positions, multi-head attention with as many K/V heads as query heads, a
SwiGLU feed-forward, no biases, an untied LM head.
"""

from dataclasses import dataclass, field


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    weight_std: float = 0.02
    seed: int = 0
    weight_bits: int = 16  # layer matrices: 16 = bf16, 4 = 4-bit codes with a bf16 scale per 128 inputs

    def params(self) -> int:
        d, f, v, l = self.d_model, self.d_ffn, self.vocab, self.n_layers
        return l * (4 * d * d + 3 * d * f + 2 * d) + 2 * v * d + d

    def weight_bytes(self) -> int:
        """Bytes of every weight a pass reads once: the layer matrices (bf16,
        or 4-bit codes plus one bf16 scale per 128 inputs), the norm gains and
        the LM head; the embedding contributes only its gathered rows."""
        d, f, v, l = self.d_model, self.d_ffn, self.vocab, self.n_layers
        mats = 4 * d * d + 3 * d * f
        per_mat = 2 * mats if self.weight_bits == 16 else mats // 2 + 2 * (mats // 128)
        return l * (per_mat + 2 * 2 * d) + 2 * v * d + 2 * d


MODELS = {
    "tiny": ModelShape("tiny", 2, 256, 4, 64, 688, 1024, seed=0x5EED0001),
    "llama7b": ModelShape("llama7b", 32, 4096, 32, 128, 11008, 32000, seed=0x5EED0007),
    "llama13b": ModelShape("llama13b", 40, 5120, 40, 128, 13824, 32000, seed=0x5EED0013),
    "llama30b": ModelShape("llama30b", 60, 6656, 52, 128, 17920, 32000, seed=0x5EED0030),
    # a ~1B draft model for the 7B-class targets (TinyLlama's depth and widths,
    # as many K/V heads as query heads)
    "draft1b": ModelShape("draft1b", 22, 2048, 16, 128, 5632, 32000, seed=0x5EED0001B),
    # 4-bit weight-only targets (the paper's phone models are INT4, §4.1).  The
    # small one has a ragged vocabulary (not a multiple of 16) and more than
    # one scale group per matrix row everywhere.
    "q4small": ModelShape("q4small", 2, 512, 4, 128, 1408, 1998, seed=0x5EED0104, weight_bits=4),
    "llama7b_q4": ModelShape("llama7b_q4", 32, 4096, 32, 128, 11008, 32000, seed=0x5EED0074, weight_bits=4),
}


@dataclass(frozen=True)
class Workload:
    """One verification workload: a model, a prefix length and a tree recipe.

    tree: ("complete", (b1, b2, ...)) -> root plus levels with branching b_k;
          ("random", n, max_parent_depth) -> parent of node i uniform over
          earlier nodes whose depth is at most max_parent_depth;
          ("chain", n) -> a single branch.
    """

    name: str
    model: str
    prefix_len: int
    tree: tuple
    seed: int = 1234
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def shape(self) -> ModelShape:
        return MODELS[self.model]


WORKLOADS = {
    "tiny_p32_n15": Workload("tiny_p32_n15", "tiny", 32, ("complete", (2, 2, 2))),
    "llama7b_p512_n31": Workload("llama7b_p512_n31", "llama7b", 512, ("complete", (2, 2, 2, 2))),
    "llama7b_p2048_n41": Workload("llama7b_p2048_n41", "llama7b", 2048, ("complete", (4, 3, 2))),
    # (the 128-row pass at the 7B shape: the widest tree a pass takes, and the
    # prefill's chunk size)
    "llama7b_p512_n128": Workload("llama7b_p512_n128", "llama7b", 512, ("random", 128, 7)),
    "llama13b_p1024_n41": Workload("llama13b_p1024_n41", "llama13b", 1024, ("complete", (4, 3, 2))),
    "q4small_p96_n15": Workload("q4small_p96_n15", "q4small", 96, ("complete", (2, 2, 2))),
    "llama7b_q4_p512_n31": Workload("llama7b_q4_p512_n31", "llama7b_q4", 512, ("complete", (2, 2, 2, 2))),
    "llama30b_p1024_n1": Workload("llama30b_p1024_n1", "llama30b", 1024, ("random", 1, 7)),
    "llama30b_p1024_n8": Workload("llama30b_p1024_n8", "llama30b", 1024, ("random", 8, 7)),
    "llama30b_p1024_n32": Workload("llama30b_p1024_n32", "llama30b", 1024, ("random", 32, 7)),
    "llama30b_p1024_n128": Workload("llama30b_p1024_n128", "llama30b", 1024, ("random", 128, 7)),
}


def get_workload(name: str) -> Workload:
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    return WORKLOADS[name]
