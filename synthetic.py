"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module only draws random numbers and lays them out; it holds none of the
reuse method's arithmetic. Both the HIP path and the CPU oracle receive what it
produces, so that the two sides see identical bytes.

Workload shapes follow the paper's throughput setting (Sec. 4.4: a few
thousand to ~16K tokens per request, tens of retrieved memory units, 10-30 %
recompute) on Llama-style decoders of 3B/7B/32B width. The paper's real
memories (LoCoMo / AMA-Bench dialogues retrieved by A-MEM) and trained weights
are not available; uniform random token ids and N(0, 0.02^2) weights stand in
for them.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch


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
    rope_theta: float
    rms_eps: float = 1e-6
    dtype: str = "bf16"  # "f32" or "bf16": storage type of weights and K/V

    @property
    def kv_width(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def qkv_width(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def with_layers(self, n_layers: int) -> "ModelShape":
        d = dict(self.__dict__)
        d["n_layers"] = n_layers
        return ModelShape(**d)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    chunk_lens: tuple
    query_len: int
    refresh: tuple          # refresh ratios as (num, den) pairs; first one is the headline
    cache_bits: int = 16    # 16 = plain cache; 4 / 2 = group-64 integer, 8 = group-64 FP8 E4M3

    @property
    def n_ctx(self) -> int:
        return int(sum(self.chunk_lens))

    @property
    def n_tokens(self) -> int:
        return self.n_ctx + self.query_len


SHAPES: Dict[str, ModelShape] = {
    "tiny": ModelShape("tiny", 2, 256, 4, 4, 64, 688, 1024, 1.0e4, dtype="f32"),
    "3b": ModelShape("3b", 28, 3072, 24, 8, 128, 8192, 128256, 1.0e6),
    "7b": ModelShape("7b", 28, 3584, 28, 4, 128, 18944, 152064, 1.0e6),
    "32b": ModelShape("32b", 64, 5120, 40, 8, 128, 27648, 152064, 1.0e6),
}


def chunk_lengths(name: str, seed: int = 0) -> tuple:
    """Memory-unit lengths of each workload (the 3B one draws U{192..256})."""
    if name == "tiny":
        return (64,) * 4
    if name == "3b":
        rng = np.random.default_rng(seed + 2)
        return tuple(int(x) for x in rng.integers(192, 257, size=20))
    if name in ("7b", "7b-q4", "7b-q2", "7b-fp8"):
        return (200,) * 40
    if name == "32b":
        return (200,) * 80
    raise KeyError(name)


def workload(name: str, seed: int = 0) -> Workload:
    if name == "tiny":
        return Workload(name, SHAPES["tiny"], chunk_lengths(name, seed), 32, ((1, 5),))
    if name == "3b":
        return Workload(name, SHAPES["3b"], chunk_lengths(name, seed), 64,
                        ((1, 5), (1, 10), (3, 10)))
    if name == "7b":
        return Workload(name, SHAPES["7b"], chunk_lengths(name, seed), 128, ((1, 5),))
    if name == "32b":
        return Workload(name, SHAPES["32b"], chunk_lengths(name, seed), 128,
                        ((1, 10), (3, 10)))
    if name in ("7b-q4", "7b-q2", "7b-fp8"):
        return Workload(name, SHAPES["7b"], chunk_lengths(name, seed), 128, ((1, 5),),
                        cache_bits={"7b-q4": 4, "7b-q2": 2, "7b-fp8": 8}[name])
    raise KeyError(name)


def torch_dtype(shape: ModelShape):
    return torch.float32 if shape.dtype == "f32" else torch.bfloat16


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _normal(shape_, std: float, seed: int, dtype, device) -> torch.Tensor:
    t = torch.empty(shape_, dtype=torch.float32, device=device)
    t.normal_(0.0, std, generator=_gen(seed, device))
    return t.to(dtype)


def make_weights(shape: ModelShape, seed: int = 0, device="cpu", n_layers: Optional[int] = None,
                 std: float = 0.02, embed: bool = True) -> dict:
    """Random-init decoder weights in the library's layout.

    Per layer: attn_norm [D], w_qkv [(Hq+2Hkv)*hd][D] (q rows, then k, then v),
    w_o [D][Hq*hd], mlp_norm [D], w_gate_up [2F][D] (gate rows first), w_down [D][F].
    Plus embed [V][D] and final_norm [D]. Linear weights ~ N(0, std^2), norm gains 1.
    Each tensor has its own seed derived from (seed, layer, slot), so a model truncated
    to fewer layers shares its first layers with the full one. The values depend on
    the device's generator: tensors meant for both the oracle and the GPU are drawn
    on the CPU.
    """
    L = shape.n_layers if n_layers is None else n_layers
    dt = torch_dtype(shape)
    D, F = shape.d_model, shape.ffn_dim
    hqd = shape.n_q_heads * shape.head_dim
    base = 1_000_003 * (seed + 1)
    layers = []
    for l in range(L):
        s = base + 97 * l
        layers.append({
            "attn_norm": torch.ones(D, dtype=dt, device=device),
            "w_qkv": _normal((shape.qkv_width, D), std, s + 1, dt, device),
            "w_o": _normal((D, hqd), std, s + 2, dt, device),
            "mlp_norm": torch.ones(D, dtype=dt, device=device),
            "w_gate_up": _normal((2 * F, D), std, s + 3, dt, device),
            "w_down": _normal((D, F), std, s + 4, dt, device),
        })
    return {
        "embed": _normal((shape.vocab, D), std, base + 11, dt, device) if embed else None,
        "final_norm": torch.ones(D, dtype=dt, device=device),
        "layers": layers,
    }


def make_tokens(n: int, vocab: int, seed: int = 0) -> np.ndarray:
    """Uniform token ids over [0, vocab)."""
    rng = np.random.default_rng(seed + 1)
    return rng.integers(0, vocab, size=n).astype(np.int32)


def random_array(shape_, seed: int, scale: float = 1.0) -> np.ndarray:
    """Plain seeded normal draws (fp64), for kernel-level parity inputs."""
    return np.random.default_rng(seed).standard_normal(shape_) * scale
