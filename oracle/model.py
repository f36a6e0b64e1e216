"""Oracle decoder: a Llama-style pre-norm transformer in plain fp64 NumPy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper evaluates Qwen2.5 / Qwen3 / Mistral decoders (Sec. 4.1 "Models",
App. A.1). Their common structure is written out here: token embedding; per
layer RMSNorm, bias-free Q/K/V projections, rotary position embedding on q and k
(rotate-half pairing of dimension k with k + hd/2), causal grouped-query softmax
attention scaled by 1/sqrt(hd), output projection with residual add, RMSNorm,
SwiGLU MLP with residual add; final RMSNorm. Full recompute (the "no KV reuse"
baseline of Sec. 4.1 "Baselines" and Table 3) is this model run on the whole
concatenated context. Standalone unit caching (Sec. 3.1: a memory unit is
encoded once, when first observed) is this model run on one unit at position 0.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ModelDims:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    rope_theta: float
    rms_eps: float


def dims_from(shape) -> ModelDims:
    """Copy the dimension fields of any object carrying them."""
    return ModelDims(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                     shape.head_dim, shape.ffn_dim, float(shape.rope_theta), float(shape.rms_eps))


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):  # a torch tensor: read its values exactly
        x = x.detach().to("cpu")
        import torch
        x = x.to(torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def split_layer(lw: dict, dims: ModelDims) -> dict:
    """Split one layer's weights from the packed layout into named fp64 matrices.

    Packed layout: w_qkv stacks the q, k, v projection rows; w_gate_up stacks the
    gate rows, then the up rows. Matrices are [out][in].
    """
    hq = dims.n_q_heads * dims.head_dim
    hk = dims.n_kv_heads * dims.head_dim
    qkv = _f64(lw["w_qkv"])
    gu = _f64(lw["w_gate_up"])
    F = dims.ffn_dim
    return {
        "attn_norm": _f64(lw["attn_norm"]),
        "w_q": qkv[:hq], "w_k": qkv[hq:hq + hk], "w_v": qkv[hq + hk:hq + 2 * hk],
        "w_o": _f64(lw["w_o"]),
        "mlp_norm": _f64(lw["mlp_norm"]),
        "w_gate": gu[:F], "w_up": gu[F:2 * F],
        "w_down": _f64(lw["w_down"]),
    }


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x divided by the root of (mean of x^2 over the last axis + eps), times gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope_cos_sin(positions, head_dim: int, theta: float):
    """cos and sin of the rotary angles p * theta^(-2k/hd), k = 0 .. hd/2-1, in fp64."""
    k = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(float(theta), -2.0 * k / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def rotate(x: np.ndarray, positions, theta: float) -> np.ndarray:
    """Rotary embedding of x [n][H][hd] at per-token angles positions[t].

    Dimension k (k < hd/2) is paired with k + hd/2 and the pair is rotated by
    positions[t] * theta^(-2k/hd). A rotation by a then by b equals one by a + b,
    which is what re-encoding a cached key at a new offset relies on (Sec. 2,
    positional re-encoding of reused states).
    """
    hd = x.shape[-1]
    half = hd // 2
    c, s = rope_cos_sin(positions, hd, theta)
    c = c[:, None, :]
    s = s[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, q_pos, k: np.ndarray, v: np.ndarray, k_pos) -> np.ndarray:
    """Causal grouped-query softmax attention.

    q [nq][Hq][hd]; k, v [nk][Hkv][hd]. Query row j (at position q_pos[j]) attends to
    the keys whose position is <= q_pos[j]; query head h reads KV head h // (Hq/Hkv).
    Scores are q.k / sqrt(hd); the softmax is over the allowed keys.
    """
    nq, hq, hd = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    q_pos = np.asarray(q_pos)
    k_pos = np.asarray(k_pos)
    allowed = k_pos[None, :] <= q_pos[:, None]
    out = np.empty((nq, hq, hd), dtype=np.float64)
    scale = 1.0 / np.sqrt(hd)
    for h in range(hq):
        s = (q[:, h, :] @ k[:, h // g, :].T) * scale
        s = np.where(allowed, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, h // g, :]
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def project_qkv(h: np.ndarray, positions, w: dict, dims: ModelDims):
    """q, k, v of the rows h [n][D] at the given positions (RoPE applied to q and k)."""
    n = h.shape[0]
    x = rms_norm(h, w["attn_norm"], dims.rms_eps)
    q = (x @ w["w_q"].T).reshape(n, dims.n_q_heads, dims.head_dim)
    k = (x @ w["w_k"].T).reshape(n, dims.n_kv_heads, dims.head_dim)
    v = (x @ w["w_v"].T).reshape(n, dims.n_kv_heads, dims.head_dim)
    return rotate(q, positions, dims.rope_theta), rotate(k, positions, dims.rope_theta), v


def output_and_mlp(h: np.ndarray, attn: np.ndarray, w: dict, dims: ModelDims) -> np.ndarray:
    """Residual add of the attention output projection, then the SwiGLU MLP block."""
    n = h.shape[0]
    h = h + attn.reshape(n, -1) @ w["w_o"].T
    x = rms_norm(h, w["mlp_norm"], dims.rms_eps)
    return h + (silu(x @ w["w_gate"].T) * (x @ w["w_up"].T)) @ w["w_down"].T


def decoder_layer(h: np.ndarray, positions, w: dict, dims: ModelDims):
    """One layer over rows that attend only to each other (ordinary causal prefill)."""
    q, k, v = project_qkv(h, positions, w, dims)
    o = attention(q, positions, k, v, positions)
    return output_and_mlp(h, o, w, dims), k, v


def embed(weights: dict, tokens) -> np.ndarray:
    e = weights["embed"]
    idx = np.asarray(tokens, dtype=np.int64)
    if hasattr(e, "detach"):
        import torch
        return _f64(e[torch.as_tensor(idx)])
    return np.asarray(e[idx], dtype=np.float64)


def full_prefill(tokens, pos0: int, weights: dict, dims: ModelDims, layers=None):
    """Ordinary causal prefill of `tokens` at positions pos0, pos0+1, ...

    Returns (final-normed hidden states [n][D], K [L][n][Hkv][hd], V [L][n][Hkv][hd]);
    K is stored after RoPE. `layers` may pass pre-split fp64 layer weights.
    """
    n = len(tokens)
    pos = pos0 + np.arange(n)
    if layers is None:
        layers = [split_layer(lw, dims) for lw in weights["layers"][:dims.n_layers]]
    h = embed(weights, tokens)
    ks, vs = [], []
    for w in layers:
        h, k, v = decoder_layer(h, pos, w, dims)
        ks.append(k)
        vs.append(v)
    hf = rms_norm(h, _f64(weights["final_norm"]), dims.rms_eps)
    return hf, np.stack(ks), np.stack(vs)


def cache_units(tokens, chunk_lens, weights: dict, dims: ModelDims, layers=None):
    """Standalone caches: each memory unit prefilled alone at position 0 (Sec. 3.1).

    Returns lists (one entry per unit) of K [L][n_i][Hkv][hd] and V [L][n_i][Hkv][hd].
    """
    if layers is None:
        layers = [split_layer(lw, dims) for lw in weights["layers"][:dims.n_layers]]
    kc, vc = [], []
    s = 0
    for n in chunk_lens:
        _, k, v = full_prefill(tokens[s:s + n], 0, weights, dims, layers)
        kc.append(k)
        vc.append(v)
        s += n
    return kc, vc


def lm_logits(h_final: np.ndarray, weights: dict, lm_head=None) -> np.ndarray:
    """Next-token logits of final-normed rows: h W^T over the vocabulary. W is the output
    embedding; the 3B-class decoders the paper evaluates tie it to the input embedding,
    which is the default here (`lm_head` passes an untied [V][D] table)."""
    w = _f64(lm_head if lm_head is not None else weights["embed"])
    return np.asarray(h_final, dtype=np.float64) @ w.T


def greedy_token(logits: np.ndarray) -> int:
    """The largest logit's index (equal values: the lowest index)."""
    return int(np.argmax(logits))


def decode_step(token: int, k_past, v_past, weights: dict, dims: ModelDims, layers=None,
                lm_head=None):
    """One generated token on top of per-layer past keys/values [L][n][Hkv][hd] at
    positions 0..n-1 (after a reuse prefill: its corrected caches). The token sits at
    position n; in every layer it attends to the n past keys and to its own.

    Returns (final-normed hidden [D], logits [V], k_new [L][Hkv][hd], v_new [L][Hkv][hd]).
    """
    n = np.asarray(k_past[0]).shape[0]
    if layers is None:
        layers = [split_layer(lw, dims) for lw in weights["layers"][:dims.n_layers]]
    h = embed(weights, [token])
    pos = np.array([n])
    key_pos = np.arange(n + 1)
    ks, vs = [], []
    for l, w in enumerate(layers):
        q, k, v = project_qkv(h, pos, w, dims)
        kk = np.concatenate([np.asarray(k_past[l], dtype=np.float64), k])
        vv = np.concatenate([np.asarray(v_past[l], dtype=np.float64), v])
        o = attention(q, pos, kk, vv, key_pos)
        h = output_and_mlp(h, o, w, dims)
        ks.append(k[0])
        vs.append(v[0])
    hf = rms_norm(h, _f64(weights["final_norm"]), dims.rms_eps)
    return hf[0], lm_logits(hf, weights, lm_head)[0], np.stack(ks), np.stack(vs)
