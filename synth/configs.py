"""Model shapes of the five synthetic workloads (Llama-style decoders).

Shapes only.  RMSNorm epsilon and RoPE base are the same for every shape
(1e-5 and 10000): the weights are random, so the published values of the real
models they are shaped after would buy nothing.
"""
from dataclasses import dataclass, asdict


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    weight_seed: int
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    page_size: int = 16

    @property
    def q_dim(self):
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self):
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_dim(self):
        return self.q_dim + 2 * self.kv_dim

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    def with_layers(self, n_layers, name=None):
        d = asdict(self)
        d["n_layers"] = n_layers
        d["name"] = name or f"{self.name}-L{n_layers}"
        return ModelShape(**d)

    def params_per_layer(self):
        d, f = self.d_model, self.ffn_dim
        return d * self.qkv_dim + self.q_dim * d + 3 * d * f


MODELS = {
    # 2 layers, d 256, 4 q-heads / 2 kv-heads of 64, SwiGLU 688, vocab 2048, seed 0
    "tiny": ModelShape("tiny", 2, 256, 4, 2, 64, 688, 2048, weight_seed=0),
    # Llama-3-8B shape, seed 1 (used by the three 8B workloads)
    "llama8b": ModelShape("llama8b", 32, 4096, 32, 8, 128, 14336, 128256, weight_seed=1),
    # Qwen2.5-32B shape, seed 4
    "qwen32b": ModelShape("qwen32b", 64, 5120, 40, 8, 128, 27648, 152064, weight_seed=4),
    # Llama-3.1-70B shape (the model the paper serves), seed 5: 141 GB of bf16 weights, one MI355X
    "llama70b": ModelShape("llama70b", 80, 8192, 64, 8, 128, 28672, 128256, weight_seed=5),
}


def model_shape(name, n_layers=None):
    m = MODELS[name]
    return m if n_layers is None else m.with_layers(n_layers)
