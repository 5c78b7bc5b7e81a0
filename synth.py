"""Seeded synthetic inputs for the KV-cache repair workloads.

This module only draws numbers: model shapes, random-init weights, token ids,
edit placements and synthetic stale caches. It holds none of the decoder's or
the repair's arithmetic, so both the GPU library's callers and the CPU oracle's
tests can take their inputs from here without sharing any method code.

The paper's benchmark (HotpotQA background paragraphs plus a synthetic record,
trained Llama/Qwen/Mistral checkpoints) is not available; these generators
stand in for its shapes only: contexts of about 5000 tokens, one short
length-preserving in-place edit, a budget of K downstream positions.

Conventions
* Matrices and biases are N(0, 0.02); norm gains are 1 + N(0, 0.02) (a gain
  drawn literally from N(0, 0.02) would make every logit tiny and attention
  uniform, which tests nothing).
* bf16 tensors are drawn in fp32 and rounded to bf16 (round-to-nearest-even);
  the rounded bytes are the canonical values for every consumer.
* Linear weights are stored [out_features][in_features], row-major.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import torch

# Master seeds for the independent streams of a workload.
SEED_WEIGHTS = 0
SEED_TOKENS = 1
SEED_EDIT_POS = 2
SEED_EDIT_IDS = 3
SEED_STALE = 4


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Shape of a Llama-style pre-norm decoder."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float
    rope_theta: float
    qkv_bias: bool = False

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_params(self) -> int:
        d, f = self.d_model, self.d_ffn
        p = d * (self.q_dim + 2 * self.kv_dim) + self.q_dim * d + 3 * d * f + 2 * d
        if self.qkv_bias:
            p += self.q_dim + 2 * self.kv_dim
        return p

    def kv_bytes_per_pos(self, elem_bytes: int) -> int:
        return self.n_layers * 2 * self.kv_dim * elem_bytes


# The five workload shapes.  eps for the Qwen2.5 family is its usual 1e-6;
# the Llama/Mistral shapes use 1e-5 as the tiny configuration does.
TINY = ModelShape("tiny-llama", 2, 256, 4, 4, 64, 688, 1024, 1e-5, 10000.0)
LLAMA3_8B = ModelShape("llama3-8b", 32, 4096, 32, 8, 128, 14336, 128256, 1e-5, 500000.0)
QWEN25_7B = ModelShape("qwen2.5-7b", 28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1000000.0,
                       qkv_bias=True)
MISTRAL_7B = ModelShape("mistral-7b", 32, 4096, 32, 8, 128, 14336, 32768, 1e-5, 1000000.0)

SHAPES = {s.name: s for s in (TINY, LLAMA3_8B, QWEN25_7B, MISTRAL_7B)}


def scaled_shape(base: ModelShape, **overrides) -> ModelShape:
    """A copy of ``base`` with some fields replaced (reduced test models)."""
    return dataclasses.replace(base, **overrides)


def _mix_seed(master: int, *parts: int) -> int:
    """Deterministic 63-bit seed from a master seed and integer labels."""
    x = (master * 0x9E3779B97F4A7C15 + 0x632BE59BD9B4E019) & ((1 << 64) - 1)
    for p in parts:
        x ^= (p + 0x9E3779B97F4A7C15 + ((x << 6) & ((1 << 64) - 1)) + (x >> 2)) & ((1 << 64) - 1)
        x = (x * 0xBF58476D1CE4E5B9) & ((1 << 64) - 1)
    return x & ((1 << 63) - 1)


def _generator(device: str, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _normal(shape, std: float, mean: float, dtype: torch.dtype, device: str, seed: int) -> torch.Tensor:
    g = _generator(device, seed)
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(mean=mean, std=std, generator=g)
    return t.to(dtype)


LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo",
                 "mlp_norm", "w_gate", "w_up", "w_down")


def make_weights(shape: ModelShape, dtype: torch.dtype = torch.bfloat16, device: str = "cpu",
                 seed: int = SEED_WEIGHTS, std: float = 0.02,
                 with_embed: bool = True) -> Dict[str, object]:
    """Random-init weights: {'embed', 'final_norm', 'layers': [dict per layer]}.

    Every tensor has its own seed derived from (seed, layer, tensor index), so
    one layer can be regenerated without drawing the others.
    """
    d, hd = shape.d_model, shape.head_dim
    layers: List[Dict[str, Optional[torch.Tensor]]] = []
    for l in range(shape.n_layers):
        layers.append(make_layer_weights(shape, l, dtype, device, seed, std))
    out: Dict[str, object] = {"layers": layers}
    out["final_norm"] = _normal((d,), std, 1.0, dtype, device, _mix_seed(seed, 1 << 20, 1))
    if with_embed:
        out["embed"] = _normal((shape.vocab, d), std, 0.0, dtype, device, _mix_seed(seed, 1 << 20, 0))
    return out


def make_layer_weights(shape: ModelShape, layer: int, dtype: torch.dtype, device: str,
                       seed: int = SEED_WEIGHTS, std: float = 0.02) -> Dict[str, Optional[torch.Tensor]]:
    d, f = shape.d_model, shape.d_ffn
    qd, kd = shape.q_dim, shape.kv_dim
    dims = {
        "attn_norm": (d,), "wq": (qd, d), "wk": (kd, d), "wv": (kd, d),
        "bq": (qd,), "bk": (kd,), "bv": (kd,), "wo": (d, qd),
        "mlp_norm": (d,), "w_gate": (f, d), "w_up": (f, d), "w_down": (d, f),
    }
    w: Dict[str, Optional[torch.Tensor]] = {}
    for i, name in enumerate(LAYER_TENSORS):
        if name in ("bq", "bk", "bv") and not shape.qkv_bias:
            w[name] = None
            continue
        mean = 1.0 if name.endswith("norm") else 0.0
        w[name] = _normal(dims[name], std, mean, dtype, device, _mix_seed(seed, layer, i))
    return w


def make_lm_head(shape: ModelShape, dtype: torch.dtype = torch.bfloat16, device: str = "cpu",
                 seed: int = SEED_WEIGHTS, std: float = 0.02) -> torch.Tensor:
    """Random-init output projection [vocab][d_model] (untied from the embedding)."""
    return _normal((shape.vocab, shape.d_model), std, 0.0, dtype, device, _mix_seed(seed, 1 << 21, 0))


def make_tokens(n: int, vocab: int, seed: int = SEED_TOKENS, device: str = "cpu") -> torch.Tensor:
    """n uniform token ids in [0, vocab), int32."""
    g = _generator("cpu", _mix_seed(seed, n, vocab))
    return torch.randint(0, vocab, (n,), generator=g, dtype=torch.int64).to(torch.int32).to(device)


def edit_position(lo: int, hi: int, seed: int = SEED_EDIT_POS, label: int = 0) -> int:
    """A seeded edit start, uniform over the integers [lo, hi]."""
    g = _generator("cpu", _mix_seed(seed, label, lo, hi))
    return int(torch.randint(lo, hi + 1, (1,), generator=g).item())


def apply_edit(tokens: torch.Tensor, start: int, length: int, vocab: int,
               seed: int = SEED_EDIT_IDS, label: int = 0) -> torch.Tensor:
    """Length-preserving in-place edit: ids in [start, start+length) redrawn uniformly."""
    out = tokens.clone().cpu()
    g = _generator("cpu", _mix_seed(seed, label, start, length))
    out[start:start + length] = torch.randint(0, vocab, (length,), generator=g,
                                              dtype=torch.int64).to(torch.int32)
    return out.to(tokens.device)


def stale_cache_std(shape: ModelShape) -> float:
    """Typical K/V magnitude of a random-init layer: 0.02 * sqrt(d_model)."""
    return 0.02 * math.sqrt(shape.d_model)


def make_stale_cache(shape: ModelShape, n_cap: int, dtype: torch.dtype = torch.bfloat16,
                     device: str = "cpu", seed: int = SEED_STALE, label: int = 0) -> torch.Tensor:
    """A synthetic stale cache [L][2][H_kv][n_cap][head_dim] of N(0, s^2) values.

    Repair is defined for any stale cache, so a random one is a valid input;
    its magnitude matches what a random-init layer writes.
    """
    return _normal((shape.n_layers, 2, shape.n_kv_heads, n_cap, shape.head_dim),
                   stale_cache_std(shape), 0.0, dtype, device, _mix_seed(seed, label, n_cap))


def doc_lengths(n_docs: int, lo: int, hi: int, seed: int = SEED_TOKENS) -> List[int]:
    """Context lengths uniform over [lo, hi] for a batch of documents."""
    g = _generator("cpu", _mix_seed(seed, n_docs, lo, hi, 7))
    return [int(x) for x in torch.randint(lo, hi + 1, (n_docs,), generator=g)]
