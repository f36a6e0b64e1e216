"""Pins for the oracle decoder: a third-party Llama, brute force, Lemma 1, causality."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from tests import hf_llama
from tests.oracle_fixtures import small_model, context


def close_to(a, ref, rel):
    """max|a - ref| <= rel * max|ref|. The transformers Llama keeps RMSNorm and the
    rotary angles in fp32 even in an fp64 model, so agreement is ~1e-6 relative."""
    err = np.abs(np.asarray(a) - np.asarray(ref)).max()
    assert err <= rel * np.abs(ref).max(), (err, np.abs(ref).max())


def test_full_prefill_matches_transformers_llama():
    dims, w, V = small_model(seed=1)
    toks = context(1, [20], 5, V)
    h, k, v = oracle.full_prefill(toks, 0, w, dims)
    ref_h, ref_k, ref_v = hf_llama.prefill(hf_llama.build(w, dims, V), toks)
    close_to(h, ref_h, 1e-5)
    close_to(k, ref_k, 1e-5)
    close_to(v, ref_v, 1e-5)


def test_full_prefill_at_offset_matches_transformers_llama():
    dims, w, V = small_model(seed=2, hq=6, hkv=2, hd=16, D=48)
    toks = context(2, [13], 0, V)
    h, k, v = oracle.full_prefill(toks, 37, w, dims)
    ref_h, ref_k, ref_v = hf_llama.prefill(hf_llama.build(w, dims, V), toks, pos0=37)
    close_to(h, ref_h, 1e-5)
    close_to(k, ref_k, 1e-5)
    close_to(v, ref_v, 1e-5)


def brute_attention(q, qp, k, v, kp):
    nq, hq, hd = q.shape
    g = hq // k.shape[1]
    out = np.zeros_like(q)
    for j in range(nq):
        for h in range(hq):
            keys = [t for t in range(k.shape[0]) if kp[t] <= qp[j]]
            s = [sum(q[j, h, e] * k[t, h // g, e] for e in range(hd)) / np.sqrt(hd) for t in keys]
            mx = max(s)
            p = [np.exp(x - mx) for x in s]
            z = sum(p)
            for e in range(hd):
                out[j, h, e] = sum(pi * v[t, h // g, e] for pi, t in zip(p, keys)) / z
    return out


def test_attention_brute_force_gqa_sparse_rows():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((5, 4, 4))
    k = rng.standard_normal((9, 2, 4))
    v = rng.standard_normal((9, 2, 4))
    qp = np.array([0, 2, 3, 7, 8])          # sparse, sorted query positions
    kp = np.arange(9)
    np.testing.assert_allclose(oracle.attention(q, qp, k, v, kp), brute_attention(q, qp, k, v, kp),
                               rtol=0, atol=1e-12)


def test_first_unit_cache_is_a_causal_prefix_of_full_prefill():
    dims, w, V = small_model(seed=4)
    lens = [7, 5]
    toks = context(4, lens, 3, V)
    _, kf, vf = oracle.full_prefill(toks, 0, w, dims)
    kc, vc = oracle.cache_units(toks, lens, w, dims)
    np.testing.assert_allclose(kc[0], kf[:, :7], rtol=0, atol=1e-12)
    np.testing.assert_allclose(vc[0], vf[:, :7], rtol=0, atol=1e-12)
    # the second unit was cached out of context: its deeper-layer states differ
    assert np.abs(vc[1][1] - vf[1, 7:12]).max() > 1e-3


@settings(max_examples=60, deadline=None)
@given(seed=st.integers(0, 10_000), n=st.integers(1, 12), d=st.sampled_from([2, 4, 8, 16]),
       dk=st.floats(0.0, 2.0), dv=st.floats(0.0, 2.0))
def test_lemma1_attention_perturbation_bound(seed, n, d, dk, dv):
    """Lemma 1 (App. B): ||y - y*|| <= Vmax ||q|| / sqrt(d) * max||dk_i|| + max||dv_i||.

    The constant is the one in the lemma's statement; the proof's last line halves it,
    which a two-token example violates (see test_lemma1_halved_constant_is_violated).
    """
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((1, 1, d))
    ks = rng.standard_normal((n, 1, d))
    vs = rng.standard_normal((n, 1, d))
    kp = ks + dk * rng.standard_normal((n, 1, d)) / np.sqrt(d)
    vp = vs + dv * rng.standard_normal((n, 1, d)) / np.sqrt(d)
    pos = np.arange(n)
    qpos = np.array([n - 1])
    y = oracle.attention(q, qpos, kp, vp, pos)[0, 0]
    ys = oracle.attention(q, qpos, ks, vs, pos)[0, 0]
    vmax = np.linalg.norm(vs[:, 0], axis=1).max()
    bound = (vmax * np.linalg.norm(q) / np.sqrt(d) * np.linalg.norm((kp - ks)[:, 0], axis=1).max()
             + np.linalg.norm((vp - vs)[:, 0], axis=1).max())
    assert np.linalg.norm(y - ys) <= bound * (1 + 1e-6) + 1e-12


def test_lemma1_halved_constant_is_violated():
    """Two tokens with values +-Vmax and a small symmetric logit shift: the error is
    Vmax ||q|| eps / sqrt(d), twice the bound with the halved constant."""
    d, eps = 4, 1e-3
    q = np.zeros((1, 1, d)); q[0, 0, 0] = 2.0
    ks = np.zeros((2, 1, d))
    vs = np.zeros((2, 1, d)); vs[0, 0, 1] = 1.0; vs[1, 0, 1] = -1.0
    kp = ks.copy(); kp[0, 0, 0] = eps; kp[1, 0, 0] = -eps
    pos = np.arange(2)
    y = oracle.attention(q, [1], kp, vs, pos)[0, 0]
    ys = oracle.attention(q, [1], ks, vs, pos)[0, 0]
    err = np.linalg.norm(y - ys)
    halved = 1.0 * 2.0 / (2 * np.sqrt(d)) * eps
    assert err > 1.9 * halved
    assert err <= 2.0 / np.sqrt(d) * eps * (1 + 1e-6)


def test_decode_step_is_the_next_row_of_a_full_prefill():
    """On the caches of an ordinary prefill, one decode step gives exactly what a prefill
    of one more token gives for that token (hidden row, logits, its K and V)."""
    dims, w, V = small_model(seed=11)
    toks = context(11, [17], 3, V)
    n = len(toks) - 1
    _, k, v = oracle.full_prefill(toks[:n], 0, w, dims)
    h1, logits, kn, vn = oracle.decode_step(int(toks[n]), k, v, w, dims)
    h_all, k_all, v_all = oracle.full_prefill(toks, 0, w, dims)
    np.testing.assert_allclose(h1, h_all[n], rtol=0, atol=1e-12)
    np.testing.assert_allclose(kn, k_all[:, n], rtol=0, atol=1e-12)
    np.testing.assert_allclose(vn, v_all[:, n], rtol=0, atol=1e-12)
    np.testing.assert_allclose(logits, h_all[n] @ np.asarray(w["embed"]).T, rtol=0, atol=1e-10)


def test_decode_step_on_arbitrary_caches_matches_transformers_llama():
    """Past K/V that no prefill produced (as after a reuse prefill): the transformers
    Llama run with them as its cache gives the same hidden row."""
    dims, w, V = small_model(seed=12, hq=6, hkv=2, hd=16, D=48)
    rng = np.random.default_rng(12)
    n = 23
    k = rng.standard_normal((dims.n_layers, n, dims.n_kv_heads, dims.head_dim))
    v = rng.standard_normal((dims.n_layers, n, dims.n_kv_heads, dims.head_dim))
    tok = 5
    h1, logits, _, _ = oracle.decode_step(tok, k, v, w, dims)
    ref = hf_llama.continue_from(hf_llama.build(w, dims, V), k, v, [tok], n)[0]
    close_to(h1, ref, 1e-5)
    assert oracle.greedy_token(logits) == int(np.argmax(ref @ np.asarray(w["embed"]).T))


def test_greedy_token_takes_the_lowest_index_of_equal_maxima():
    assert oracle.greedy_token(np.array([0.5, 2.0, -1.0, 2.0])) == 1


def test_lm_logits_match_transformers_tied_causal_lm():
    """Next-token logits of the final-normed rows with the output embedding tied to the
    input embedding: the transformers LlamaForCausalLM (tie_word_embeddings) gives the same
    logits at every position, and the same greedy token."""
    dims, w, V = small_model(seed=13, hq=4, hkv=2, hd=8, D=32)
    toks = context(13, [9, 6], 4, V)
    h, _, _ = oracle.full_prefill(toks, 0, w, dims)
    ours = oracle.lm_logits(h, w)
    lm = hf_llama.build_causal_lm(w, dims, V)
    assert lm.lm_head.weight.data_ptr() == lm.model.embed_tokens.weight.data_ptr()
    ref = hf_llama.next_token_logits(lm, toks)
    assert ours.shape == ref.shape == (len(toks), V)
    close_to(ours, ref, 1e-5)  # the decoders differ by transformers' fp32 norms / angles
    # the head alone, on transformers' own final hidden states: exact up to fp64 rounding
    import torch
    with torch.no_grad():
        h_hf = lm.model(input_ids=torch.as_tensor(toks, dtype=torch.long)[None]).last_hidden_state[0]
    close_to(oracle.lm_logits(h_hf.numpy(), w), ref, 1e-13)
    assert [oracle.greedy_token(r) for r in ours] == [int(np.argmax(r)) for r in ref]
    # an untied table is used when given
    other = np.random.default_rng(13).standard_normal((V, dims.d_model))
    np.testing.assert_allclose(oracle.lm_logits(h[:2], w, other), h[:2] @ other.T, rtol=1e-13)
