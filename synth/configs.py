"""Model shapes for the synthetic decoders.

The shapes follow the dense decoders whose costs the paper tabulates
(Appendix C, Table C1: width, vocabulary, depth) and the readout placements it
studies (Section 5.1 and Table 3: exit at about one third, one half and two
thirds of depth). Weights are random, never trained.

final_norm_gain: with every gain equal to one, random N(0, 0.02^2) weights give
logits of standard deviation 0.02*sqrt(H) (about 0.8 at H=1536), so the
readout's max-probability sits near 1/V for every token and a threshold cannot
separate tokens. The final RMSNorm gain is therefore set to 250/sqrt(H), which
gives logits of standard deviation about 5 and a spread of confidences over
(0, 1). The readout and the full head share this norm, as the paper's readout
passes its output through the model's own final normalisation.
"""
from dataclasses import dataclass, field, replace
import math


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    wdtype: str                 # "f32" or "bf16": storage type of matrices and KV
    readout_layers: tuple       # layers (1-based count of layers run) carrying a readout
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    init_std: float = 0.02
    seed: int = 0

    @property
    def final_norm_gain(self) -> float:
        return 250.0 / math.sqrt(self.hidden)

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def layer_params(self) -> int:
        """Parameters of one decoder layer's seven matrices (norm gains excluded)."""
        H, A, K, D, F = self.hidden, self.n_q_heads, self.n_kv_heads, self.head_dim, self.ffn
        return H * A * D + 2 * H * K * D + A * D * H + 3 * H * F

    @property
    def wbytes(self) -> int:
        return 2 if self.wdtype == "bf16" else 4

    def with_readouts(self, layers) -> "ModelConfig":
        return replace(self, readout_layers=tuple(layers))


CONFIGS = {
    # 4 layers, H=256, 4 q / 2 kv heads of 64, SwiGLU 1024, V=4096, fp32, readout at 2.
    "tiny": ModelConfig("tiny", 4, 256, 4, 2, 64, 1024, 4096, "f32", (2,)),
    # 1.5B-shaped: 28 layers, H=1536, 12 q / 2 kv heads of 128, F=8960, V=151936, bf16.
    "d1p5b": ModelConfig("d1p5b", 28, 1536, 12, 2, 128, 8960, 151936, "bf16", (14,)),
    # Same shape with readouts at one quarter, one half and three quarters of depth.
    "d1p5b_sweep": ModelConfig("d1p5b_sweep", 28, 1536, 12, 2, 128, 8960, 151936, "bf16",
                               (7, 14, 21)),
    # 0.5B-shaped: 24 layers, H=896, 14 q / 2 kv heads of 64, F=4864.
    "d0p5b": ModelConfig("d0p5b", 24, 896, 14, 2, 64, 4864, 151936, "bf16", (12,)),
    # 3B-shaped: 36 layers, H=2048, 16 q / 2 kv heads of 128, F=11008.
    "d3b": ModelConfig("d3b", 36, 2048, 16, 2, 128, 11008, 151936, "bf16", (18,)),
}


def get_config(name: str) -> ModelConfig:
    if name not in CONFIGS:
        raise KeyError(f"unknown model config {name!r}; known: {sorted(CONFIGS)}")
    return CONFIGS[name]

# Test-only variant: the tiny shapes with bf16 storage, to exercise bf16 code at small size.
CONFIGS["tiny_bf16"] = replace(CONFIGS["tiny"], name="tiny_bf16", wdtype="bf16")
