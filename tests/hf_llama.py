"""Independent reference decoder for the oracle pins: the `transformers` Llama model.

Builds a CPU fp64 LlamaModel (eager attention) carrying the same weights as a
library-layout weight dict, so the oracle's decoder can be checked against a
third-party implementation of the same architecture.
"""
import torch
from transformers import LlamaConfig, LlamaModel
from transformers.cache_utils import DynamicCache


def build(weights: dict, dims, vocab: int) -> LlamaModel:
    cfg = LlamaConfig(vocab_size=vocab, hidden_size=dims.d_model, intermediate_size=dims.ffn_dim,
                      num_hidden_layers=dims.n_layers, num_attention_heads=dims.n_q_heads,
                      num_key_value_heads=dims.n_kv_heads, head_dim=dims.head_dim,
                      rms_norm_eps=dims.rms_eps, rope_theta=dims.rope_theta,
                      attention_bias=False, mlp_bias=False, max_position_embeddings=1 << 16)
    cfg._attn_implementation = "eager"
    model = LlamaModel(cfg).double().eval()
    hq = dims.n_q_heads * dims.head_dim
    hk = dims.n_kv_heads * dims.head_dim
    F = dims.ffn_dim
    sd = {"embed_tokens.weight": weights["embed"], "norm.weight": weights["final_norm"]}
    for l in range(dims.n_layers):
        lw = weights["layers"][l]
        p = f"layers.{l}."
        qkv = lw["w_qkv"]
        sd[p + "self_attn.q_proj.weight"] = qkv[:hq]
        sd[p + "self_attn.k_proj.weight"] = qkv[hq:hq + hk]
        sd[p + "self_attn.v_proj.weight"] = qkv[hq + hk:hq + 2 * hk]
        sd[p + "self_attn.o_proj.weight"] = lw["w_o"]
        sd[p + "mlp.gate_proj.weight"] = lw["w_gate_up"][:F]
        sd[p + "mlp.up_proj.weight"] = lw["w_gate_up"][F:]
        sd[p + "mlp.down_proj.weight"] = lw["w_down"]
        sd[p + "input_layernorm.weight"] = lw["attn_norm"]
        sd[p + "post_attention_layernorm.weight"] = lw["mlp_norm"]
    sd = {k: torch.as_tensor(v).to(torch.float64) for k, v in sd.items()}
    model.load_state_dict(sd, strict=True)
    return model


@torch.no_grad()
def prefill(model, tokens, pos0=0):
    """Hidden states (final norm applied) and per-layer K, V as [L][n][Hkv][hd] arrays."""
    ids = torch.as_tensor(tokens, dtype=torch.long)[None]
    pos = (pos0 + torch.arange(ids.shape[1]))[None]
    out = model(input_ids=ids, position_ids=pos, use_cache=True)
    pkv = out.past_key_values
    ks = torch.stack([lay.keys[0].transpose(0, 1) for lay in pkv.layers])
    vs = torch.stack([lay.values[0].transpose(0, 1) for lay in pkv.layers])
    return out.last_hidden_state[0].numpy(), ks.numpy(), vs.numpy()


@torch.no_grad()
def continue_from(model, past_k, past_v, tokens, pos0):
    """Run `tokens` at positions pos0.. on top of given per-layer K/V [L][n][Hkv][hd]."""
    cache = DynamicCache(config=model.config)
    for l in range(len(past_k)):
        k = torch.as_tensor(past_k[l]).transpose(0, 1)[None].contiguous()
        v = torch.as_tensor(past_v[l]).transpose(0, 1)[None].contiguous()
        cache.update(k, v, l)
    ids = torch.as_tensor(tokens, dtype=torch.long)[None]
    pos = (pos0 + torch.arange(ids.shape[1]))[None]
    out = model(input_ids=ids, position_ids=pos, past_key_values=cache, use_cache=True)
    return out.last_hidden_state[0].numpy()


def build_causal_lm(weights: dict, dims, vocab: int):
    """LlamaForCausalLM with the output embedding tied to the input embedding, carrying
    the same weights as a library-layout weight dict (fp64, eager attention)."""
    from transformers import LlamaForCausalLM
    base = build(weights, dims, vocab)
    cfg = base.config
    cfg.tie_word_embeddings = True
    lm = LlamaForCausalLM(cfg).double().eval()
    lm.model.load_state_dict(base.state_dict(), strict=True)
    lm.tie_weights()
    return lm


@torch.no_grad()
def next_token_logits(lm, tokens):
    """Logits [n][vocab] of every position of an ordinary prefill of `tokens`."""
    ids = torch.as_tensor(tokens, dtype=torch.long)[None]
    return lm(input_ids=ids).logits[0].numpy()
