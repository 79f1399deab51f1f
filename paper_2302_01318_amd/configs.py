"""Named model shapes and workloads.

Chinchilla's own shape (d_model 8192, 64 heads, 80 layers) and the paper's
draft shape (d_model 6144, 48 heads, 8 layers) come from the paper's
Hyperparams table; the paper does not give FFN widths, vocabulary or block
design. The 70B-shaped target here uses FFN 32768 = 4 d with a two-matrix
GELU FFN and untied embeddings (65 B parameters, 130 GB in bf16), vocab 32000.
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class ModelShape:
    name: str
    d_model: int
    n_layers: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    ffn: str = "gelu"          # "gelu" or "swiglu"
    dtype: str = "bf16"        # "f32", "bf16" or "fp8" (FP8 E4M3 projections, bf16 activations / KV)
    eps: float = 1e-5
    rope_base: float = 10000.0

    def with_(self, **kw):
        return replace(self, **kw)

    def n_params(self):
        d, F, V, HD = self.d_model, self.d_ff, self.vocab, self.n_heads * self.head_dim
        ffn = (2 if self.ffn == "gelu" else 3) * d * F
        return self.n_layers * (4 * d * HD + ffn + 2 * d) + 2 * V * d + d

    def act_bytes(self):
        """Bytes per element of the embedding, the KV cache and q."""
        return 4 if self.dtype == "f32" else 2

    def weight_bytes(self):
        """Bytes per element of a projection matrix."""
        return {"f32": 4, "bf16": 2, "fp8": 1}[self.dtype]

    def matrix_bytes(self, rows, cols):
        """Bytes a forward streams for one [rows][cols] projection: the
        elements, plus an fp32 scale per row for FP8."""
        return rows * cols * self.weight_bytes() + (4 * rows if self.dtype == "fp8" else 0)

    def matrix_bytes_per_layer(self):
        """Bytes of the projection matrices of one block (what a forward streams)."""
        d, F, HD = self.d_model, self.d_ff, self.n_heads * self.head_dim
        mb = self.matrix_bytes
        ffn = 2 * mb(F, d) + mb(d, F) if self.ffn == "swiglu" else mb(F, d) + mb(d, F)
        return mb(3 * HD, d) + mb(d, HD) + ffn


# Tiny end-to-end pair (fp32): target and draft share the vocabulary.
TINY_TARGET = ModelShape("tiny-target", 256, 4, 4, 64, 1024, 1024, "gelu", "f32")
TINY_DRAFT = ModelShape("tiny-draft", 128, 2, 2, 64, 512, 1024, "gelu", "f32")
# 7B-shaped target (bf16, SwiGLU 11008).
SEVEN_B = ModelShape("7b", 4096, 32, 32, 128, 11008, 32000, "swiglu", "bf16")
# Chinchilla-70B-shaped target and its draft (bf16).
SEVENTY_B = ModelShape("70b", 8192, 80, 64, 128, 32768, 32000, "gelu", "bf16")
DRAFT_70B = ModelShape("70b-draft", 3072, 24, 24, 128, 12288, 32000, "gelu", "bf16")

SHAPES = {s.name: s for s in (TINY_TARGET, TINY_DRAFT, SEVEN_B, SEVENTY_B, DRAFT_70B)}

# Accept/resample-alone grid (vocab 32000).
ACCEPT_GRID = {"V": 32000, "K": (1, 2, 4, 8), "B": (1, 8, 64), "sigma": 2.0, "sigma_pert": 0.5}

# 70B verify sweep.
SWEEP = {"K": (1, 2, 3, 4, 6, 8), "B": (1, 4, 16), "ctx": (2048, 8192),
         "sigma_pert": (0.1, 0.5, 1.0)}

# K trade-off study on a coupled 70B / draft pair: the draft's logits are the
# target's plus N(0, code_pert^2) per entry (the sigma_pert of the accept-stage
# pairs), the logit spread is 2 as there.
K_STUDY = {"K": (1, 2, 3, 4, 6, 8), "layer_std": 0.002, "code_pert": (0.1, 0.5, 1.0), "logit_std": 2.0,
           "rank": 64, "prompt": 256, "n_new": 128, "reps": 10, "pair_seed": 7}
