"""First decode step over the corrected caches (akvs_lm_head, akvs_decode_step) against
the oracle: the next-token logits of the last query row, one and two generated tokens
attending to the reuse prefill's corrected keys and values, and the greedy pick."""
import numpy as np
import pytest
import torch

import oracle
import synthetic
from paper_2607_21604_amd.runtime import Engine
from tests.gpu_util import DEV, to_dev, dev_weights, f64, max_rel
from tests.libutil import ensure_built
from tests.test_gpu_e2e import Case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def check_pick(tok_gpu, logits_gpu):
    """The pick is the first index of the largest logit the GPU computed."""
    lg = logits_gpu.cpu().numpy()
    assert int(tok_gpu) == int(np.argmax(lg))


def test_reuse_then_two_decode_steps_tiny():
    c = Case("tiny")
    ref = c.oracle()
    T = len(c.toks)
    out = c.gpu(probes=(ref["probe_k"], ref["probe_v"]), kv_rows=T + 2)
    assert out["k_corr"].shape[1] == T + 2
    # the reuse prefill still writes rows 0..T-1 as before
    assert max_rel(f64(out["k_corr"][:, :T]), ref["k_corr"]) < 1e-4
    # next token from the last query row
    logits0, tok0 = c.eng.lm_head(out["h_query"][-1:].contiguous())
    ref_logits0 = oracle.lm_logits(ref["h_query"][-1:], c.w)
    assert max_rel(f64(logits0), ref_logits0) < 1e-4
    check_pick(tok0[0], logits0[0])
    # decode on the oracle's token so both sides follow the same path
    t0 = oracle.greedy_token(ref_logits0[0])
    k_ref, v_ref = ref["k_corr"], ref["v_corr"]
    tok = to_dev(np.array([t0], np.int32))
    lg1, nt1 = c.eng.decode_step(tok, T, out["k_corr"], out["v_corr"])
    h1, r_lg1, kn, vn = oracle.decode_step(t0, k_ref, v_ref, c.w, c.dims, c.layers)
    assert max_rel(f64(lg1), r_lg1) < 1e-4
    assert max_rel(f64(out["k_corr"][:, T]), kn) < 1e-4
    assert max_rel(f64(out["v_corr"][:, T]), vn) < 1e-4
    check_pick(nt1[0], lg1)
    # a second step sees the first one's key and value
    t1 = oracle.greedy_token(r_lg1)
    lg2, _ = c.eng.decode_step(to_dev(np.array([t1], np.int32)), T + 1, out["k_corr"], out["v_corr"])
    k2 = np.concatenate([k_ref, kn[:, None]], axis=1)
    v2 = np.concatenate([v_ref, vn[:, None]], axis=1)
    _, r_lg2, _, _ = oracle.decode_step(t1, k2, v2, c.w, c.dims, c.layers)
    assert max_rel(f64(lg2), r_lg2) < 1e-4


def test_decode_step_3b_width_bf16():
    """3B width (3 layers, vocab 128256): a step over a full prefill's caches against the
    oracle run on the same (bf16) cache values."""
    c = Case("3b", n_layers=3, n_units=2)
    n = 300
    toks = to_dev(c.toks[:n].astype(np.int32))
    _, k, v = c.eng.full_prefill(toks, 0, want_h=False)
    kc = torch.zeros((3, n + 1) + tuple(k.shape[2:]), dtype=k.dtype, device=DEV)
    vc = torch.zeros_like(kc)
    kc[:, :n].copy_(k)
    vc[:, :n].copy_(v)
    t = int(c.toks[n])
    lg, nt = c.eng.decode_step(to_dev(np.array([t], np.int32)), n, kc, vc)
    torch.cuda.synchronize()
    _, r_lg, kn, vn = oracle.decode_step(t, f64(k), f64(v), c.w, c.dims, c.layers)
    assert max_rel(f64(lg), r_lg) < 2e-2
    assert max_rel(f64(kc[:, n]), kn) < 2e-2
    assert max_rel(f64(vc[:, n]), vn) < 2e-2
    check_pick(nt[0], lg)


def test_greedy_pick_takes_lowest_index_of_equal_maxima():
    """An output embedding whose rows 5 and 9 are equal and give the largest logit."""
    shape = synthetic.SHAPES["tiny"]
    w = synthetic.make_weights(shape, seed=3)
    eng = Engine(shape, dev_weights(w))
    rng = np.random.default_rng(0)
    h = torch.from_numpy(rng.standard_normal((1, shape.d_model)).astype(np.float32)).to(DEV)
    w_out = torch.from_numpy(rng.standard_normal((shape.vocab, shape.d_model)).astype(np.float32) * 0.01)
    w_out[5] = torch.from_numpy(h[0].cpu().numpy())
    w_out[9] = w_out[5]
    logits, tok = eng.lm_head(h, w_out.to(DEV))
    assert int(tok[0]) == 5
    assert float(logits[0, 5]) == float(logits[0, 9]) == float(logits[0].max())


def test_decode_workspace_and_bounds():
    from paper_2607_21604_amd import akvs
    shape = synthetic.SHAPES["tiny"]
    w = synthetic.make_weights(shape, seed=3)
    eng = Engine(shape, dev_weights(w))
    kc = torch.zeros((shape.n_layers, 8, shape.n_kv_heads, shape.head_dim), device=DEV)
    with pytest.raises(akvs.AkvsError):
        eng.decode_step(to_dev(np.array([1], np.int32)), 8, kc, kc.clone())  # no room for row 8


@pytest.mark.parametrize("n_q,n_kv,hd,n", [
    (24, 8, 128, 0), (24, 8, 128, 16), (24, 8, 128, 4516), (28, 4, 128, 1000),
    (40, 8, 128, 16128), (8, 1, 64, 300), (4, 4, 64, 129), (16, 1, 128, 200),
    (16, 1, 128, 3000)])
def test_decode_step_one_row_attention_shapes(n_q, n_kv, hd, n):
    """One decode step of a one-layer bf16 model over random caches of n positions, at the
    query / KV head ratios of the 3B, 7B and 32B shapes and at head dim 64: the one-row
    attention kernel from a single key chunk up to 127 chunks of 128 keys; 16 query heads
    per KV head take the general attention kernel instead (over 3001 keys with its
    12-way key split and the merge's sequential path). Keys are scaled
    so that the softmax is far from uniform. Logits and the new K/V row against the oracle
    run on the same cache values."""
    shape = synthetic.ModelShape("dec", 1, 512, n_q, n_kv, hd, 1024, 2048, 1.0e6)
    w = synthetic.make_weights(shape, seed=7)
    eng = Engine(shape, dev_weights(w))
    dims = oracle.dims_from(shape)
    layers = [oracle.split_layer(lw, dims) for lw in w["layers"]]
    rng = np.random.default_rng(n + n_q)
    k = torch.from_numpy(rng.standard_normal((1, n, n_kv, hd)).astype(np.float32) * 30).bfloat16()
    v = torch.from_numpy(rng.standard_normal((1, n, n_kv, hd)).astype(np.float32)).bfloat16()
    kc = torch.zeros((1, n + 1, n_kv, hd), dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros_like(kc)
    kc[:, :n].copy_(k.to(DEV))
    vc[:, :n].copy_(v.to(DEV))
    t = 77
    lg, nt = eng.decode_step(to_dev(np.array([t], np.int32)), n, kc, vc)
    torch.cuda.synchronize()
    _, r_lg, kn, vn = oracle.decode_step(t, f64(k), f64(v), w, dims, layers)
    assert max_rel(f64(kc[:, n]), kn) < 2e-2
    assert max_rel(f64(vc[:, n]), vn) < 2e-2
    assert max_rel(f64(lg), r_lg) < 2e-2
    check_pick(nt[0], lg)
