"""Decoder shapes used by the synthetic workloads.

A Llama-style decoder (RMSNorm, rotary position embedding, grouped-query
attention, SwiGLU MLP, untied LM head).  The paper's target models are
Llama-3.1-8B and Qwen3-8B/4B (App. A, checkpoint table); the shapes below are
random-init stand-ins of the same size class.
"""

from dataclasses import dataclass, asdict, replace


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float
    rms_eps: float = 1e-5
    max_pos: int = 20480          # rotary table length (positions 0..max_pos-1)
    max_draft: int = 64           # longest chain draft (App. A drafting table)
    page_size: int = 16           # tokens per KV page

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def with_layers(self, n_layers: int) -> "ModelConfig":
        return replace(self, n_layers=n_layers, name=f"{self.name}-L{n_layers}")

    def as_dict(self) -> dict:
        return asdict(self)

    def layer_params(self) -> int:
        """Number of weight-matrix parameters in one decoder layer."""
        d = self.d_model
        return d * self.q_dim + 2 * d * self.kv_dim + self.q_dim * d + 3 * d * self.ffn_dim


# 2 layers, d_model 256, 4/4 heads of 64, SwiGLU 1024, vocab 4096, theta 1e4.
TINY = ModelConfig("tiny", 2, 256, 4, 4, 64, 1024, 4096, 1.0e4, max_pos=4096)

# Llama-3-8B shape: 32 layers, d_model 4096, 32 q / 8 kv heads of 128,
# SwiGLU 14336, vocab 128256, theta 5e5.
SHAPE_8B = ModelConfig("8b", 32, 4096, 32, 8, 128, 14336, 128256, 5.0e5)

# 32B shape that fits one GPU: 64 layers, d_model 5120, 64 q / 8 kv heads of
# 128 (q_dim 8192 != d_model), SwiGLU 27648, vocab 152064.  The workload does
# not fix theta; 1e6 is used (it does not change cost).
SHAPE_32B = ModelConfig("32b", 64, 5120, 64, 8, 128, 27648, 152064, 1.0e6)


def config_by_name(name: str) -> ModelConfig:
    table = {c.name: c for c in (TINY, SHAPE_8B, SHAPE_32B)}
    if name in table:
        return table[name]
    base, _, lay = name.partition("-L")
    if base in table and lay.isdigit():
        return table[base].with_layers(int(lay))
    raise KeyError(name)
