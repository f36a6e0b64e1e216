"""Parity at the full size of the benchmark's 3B-class workload (28 layers, width 3072,
24/8 heads of 128, FFN 8192; 20 units of U{192..256} tokens + a 64-token query, T = 4516,
r = 1/5, check layer 1), in the launch configurations the benchmark times.

The oracle cannot run the 28-layer procedure at this size within a test, so the checks
are (a) step entries at full size against the oracle on sampled outputs it computes one
by one (attention rows, GEMM rows) or on whole tensors where that is cheap (selection,
offsets, correction), and (b) properties of the whole call that hold at any size:
bitwise determinism, prefix layers identical to the full prefill, 100 % refresh equal
to the full prefill, the check-layer divergences of every unit token against the oracle,
and valid top-b probe sets.
"""
import numpy as np
import pytest
import torch

import oracle
import synthetic
from paper_2607_21604_amd import akvs
from paper_2607_21604_amd.runtime import Engine
from tests.gpu_util import DEV, to_dev, f64, max_rel, storage_round, check_valid_top_b
from tests.libutil import ensure_built
from tests.test_gpu_steps import (rope, run_select, make_offset_case, gpu_offset_and_correction,
                                  oracle_offset_and_correction)

pytestmark = pytest.mark.gpu

WL = synthetic.workload("3b", 0)
SHAPE = WL.shape
LENS = list(WL.chunk_lens)
Q = WL.query_len
T = WL.n_tokens
TC = WL.n_ctx


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def probe_like_positions(seed):
    """Ascending row positions shaped like the recomputed rows at r = 1/5: per unit
    between b and 2b distinct tokens, then every query token."""
    rng = np.random.default_rng(seed)
    starts = oracle.chunk_starts(LENS)
    pos = []
    for s, n in zip(starts, LENS):
        b = oracle.probe_budget(n, 1, 5)
        k = int(rng.integers(b, min(n, 2 * b) + 1))
        pos.append(s + np.sort(rng.choice(n, size=k, replace=False)))
    pos.append(np.arange(TC, T))
    return np.concatenate(pos).astype(np.int32)


def sample_rows(n_rows, k, seed):
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(n_rows, size=k, replace=False).tolist()) | {0, n_rows - 1, n_rows - Q}
    return np.array(sorted(pick))


def test_fullsize_attention_sampled_rows():
    """M ~ 1400 probe-like rows x 24 heads over T = 4516 keys, with and without the key
    split the reuse prefill uses; 40 sampled rows against per-row oracle attention."""
    hq, hkv, hd = SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.head_dim
    pos = probe_like_positions(1)
    n = len(pos)
    q = storage_round(synthetic.random_array((n, hq, hd), 61), torch.bfloat16)
    k = storage_round(synthetic.random_array((T, hkv, hd), 62), torch.bfloat16)
    v = storage_round(synthetic.random_array((T, hkv, hd), 63), torch.bfloat16)
    m = akvs.model_cfg(SHAPE, n_layers=1)
    ws_bytes = akvs.akvs_attention_workspace_size(m, n, T)
    assert ws_bytes > 0  # this size splits the key range, like the benchmark's probe layers
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    qd, pd, kd, vd = to_dev(q), to_dev(pos), to_dev(k), to_dev(v)
    out_split = torch.empty((n, hq * hd), dtype=torch.bfloat16, device=DEV)
    out_plain = torch.empty_like(out_split)
    akvs.akvs_sparse_query_attention(qd, pd, n, kd, vd, T, m, out_split, ws)
    akvs.akvs_sparse_query_attention(qd, pd, n, kd, vd, T, m, out_plain)
    torch.cuda.synchronize()
    rows = sample_rows(n, 37, 2)
    ref = oracle.attention(f64(q)[rows], pos[rows], f64(k), f64(v), np.arange(T)).reshape(len(rows), -1)
    assert max_rel(f64(out_split)[rows], ref) < 1e-2
    assert max_rel(f64(out_plain)[rows], ref) < 1e-2
    assert max_rel(f64(out_split), f64(out_plain)) < 1e-2


@pytest.mark.parametrize("rows_kind", ["probe", "all"])
def test_fullsize_probe_layer_gemms_sampled_rows(rows_kind):
    """QKV projection and O-proj + MLP at the full 3B width, over M ~ 1400 probe-like rows
    (the probe layers' GEMM shapes) and over all T = 4516 rows (the prefix layers'); the
    two row counts take every block-tile shape of the projection GEMM between them. About
    40 sampled rows, the rows at tile edges among them, against the oracle."""
    pos = probe_like_positions(3) if rows_kind == "probe" else np.arange(T, dtype=np.int32)
    n = len(pos)
    w = synthetic.make_weights(SHAPE, seed=5, n_layers=1, embed=False)
    dims = oracle.dims_from(SHAPE.with_layers(1))
    lw = w["layers"][0]
    m = akvs.model_cfg(SHAPE, n_layers=1)
    lwd = {k: to_dev(t) for k, t in lw.items()}  # kept alive: layer_array holds raw pointers
    lws = akvs.layer_array({"layers": [lwd]})[0]
    hq, hkv, hd = SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.head_dim
    h = (np.random.default_rng(6).standard_normal((n, SHAPE.d_model)) * 0.5).astype(np.float32)
    h_dev = to_dev(h)
    tab = rope(T, hd, SHAPE.rope_theta)
    q = torch.empty((n, hq, hd), dtype=torch.bfloat16, device=DEV)
    kf = torch.empty((n, hkv, hd), dtype=torch.bfloat16, device=DEV)
    vf = torch.empty_like(kf)
    ws = torch.empty(akvs.akvs_step_workspace_size(m, n), dtype=torch.uint8, device=DEV)
    akvs.akvs_probe_qkv(h_dev, n, to_dev(pos), m, lws, tab, T, q, kf, vf, ws)
    att = storage_round(synthetic.random_array((n, hq * hd), 7), torch.bfloat16)
    akvs.akvs_probe_out_mlp(h_dev, n, to_dev(att), m, lws, ws)
    torch.cuda.synchronize()
    edges = [e for e in (95, 96, 127, 128, 191, 192, 255, 256, 1279, 1280, 4479, 4480, n - 1) if e < n]
    rows = np.union1d(sample_rows(n, 29, 4), edges)
    sw = oracle.split_layer(lw, dims)
    h64 = h.astype(np.float64)[rows]
    rq, rk, rv = oracle.model.project_qkv(h64, pos[rows], sw, dims)
    assert max_rel(f64(q)[rows], rq) < 2e-2
    assert max_rel(f64(kf)[rows], rk) < 2e-2
    assert max_rel(f64(vf)[rows], rv) < 2e-2
    ref = oracle.model.output_and_mlp(h64, f64(att)[rows], sw, dims)
    assert max_rel(f64(h_dev)[rows], ref) < 2e-2


@pytest.mark.parametrize("refresh", [(1, 5), (1, 10), (3, 10)])
def test_fullsize_selection_bit_exact(refresh):
    """Probe lists, flags, recomputed rows and weights of the 20-unit context, bit-exact."""
    rng = np.random.default_rng(8)
    d_k = rng.random(TC).astype(np.float32) * 3
    d_v = rng.integers(0, 40, size=TC).astype(np.float32) * 0.1  # ties
    got, sum_b, cap = run_select(d_k, d_v, LENS, Q, refresh)
    starts = oracle.chunk_starts(LENS)
    budgets = [oracle.probe_budget(n, *refresh) for n in LENS]
    sk = [oracle.select_top(d_k[s:s + n], b) + s for s, n, b in zip(starts, LENS, budgets)]
    sv = [oracle.select_top(d_v[s:s + n], b) + s for s, n, b in zip(starts, LENS, budgets)]
    assert list(got["probe_k"][:sum_b]) == [int(x) for x in np.concatenate(sk)]
    assert list(got["probe_v"][:sum_b]) == [int(x) for x in np.concatenate(sv)]
    in_kv = np.zeros(TC, bool)
    in_kv[np.concatenate(sk)] = True
    in_kv[np.concatenate(sv)] = True
    rows = np.concatenate([np.nonzero(in_kv)[0], np.arange(TC, T)])
    assert int(got["n_rows"][0]) == len(rows) <= cap
    np.testing.assert_array_equal(got["rows"][:len(rows)], rows)


def test_fullsize_offsets_and_correction():
    """Per-unit offsets and the corrected K/V of every unit token of the 20-unit context
    (8 KV heads of 128; the helper appends 3 query rows)."""
    cs = make_offset_case("bf16", LENS, SHAPE.n_kv_heads, SHAPE.head_dim, seed=12)
    mu_k, mu_v, k_corr, v_corr = gpu_offset_and_correction(cs, SHAPE.n_kv_heads, SHAPE.head_dim)
    rmk, rmv, rck, rcv = oracle_offset_and_correction(cs)
    assert max_rel(f64(mu_k), rmk) < 1e-5 and max_rel(f64(mu_v), rmv) < 1e-5
    assert max_rel(f64(k_corr), rck) < 4e-3 and max_rel(f64(v_corr), rcv) < 4e-3


@pytest.fixture(scope="module")
def bench_case():
    """The benchmark's call: weights drawn on the device by the seeded generator, unit
    caches from the library's standalone prefill of each unit."""
    w = synthetic.make_weights(SHAPE, seed=0, device=DEV)
    eng = Engine(SHAPE, w, DEV)
    toks = torch.tensor(synthetic.make_tokens(T, SHAPE.vocab, 0), dtype=torch.int32, device=DEV)
    k_cache, v_cache = eng.cache_units(toks, LENS)
    torch.cuda.synchronize()
    return dict(w=w, eng=eng, toks=toks, k=k_cache, v=v_cache)


def run(case, refresh=(1, 5), k=None, v=None):
    out = case["eng"].reuse_prefill(case["toks"], LENS, Q, case["k"] if k is None else k,
                                    case["v"] if v is None else v, refresh, 1, 0)
    torch.cuda.synchronize()
    return out


def test_fullsize_reuse_is_deterministic_and_keeps_prefix_layers(bench_case):
    a = run(bench_case)
    b = run(bench_case)
    n = int(a["n_rows"][0])
    assert n == int(b["n_rows"][0]) and 1000 < n < 2000
    for key in ("h_query", "k_corr", "v_corr", "d_k", "d_v"):
        assert torch.equal(a[key], b[key]), key
    assert torch.equal(a["rows"][:n], b["rows"][:n])
    sb = a["_sum_b"]
    assert torch.equal(a["probe_k"][:sb], b["probe_k"][:sb])
    # layer 0 (before the check layer) is an ordinary prefill of every token: same kernels,
    # same inputs as the full prefill, so the same bits
    _, kf, vf = bench_case["eng"].full_prefill(bench_case["toks"], want_h=False)
    assert torch.equal(a["k_corr"][0], kf[0]) and torch.equal(a["v_corr"][0], vf[0])


def test_fullsize_full_refresh_equals_full_prefill(bench_case):
    out = run(bench_case, refresh=(1, 1))
    h, kf, vf = bench_case["eng"].full_prefill(bench_case["toks"], want_h=True)
    torch.cuda.synchronize()
    assert int(out["n_rows"][0]) == T
    assert max_rel(f64(out["h_query"]), f64(h[TC:])) < 2e-2
    assert max_rel(f64(out["k_corr"]), f64(kf)) < 2e-2
    assert max_rel(f64(out["v_corr"]), f64(vf)) < 2e-2


def test_fullsize_check_layer_divergence_and_probe_sets(bench_case):
    """Random unit caches from the seeded generator (so no oracle input comes from the
    library): the divergences of all 4452 unit tokens at check layer 1 against the oracle
    (prefix layer 0 over all 4516 tokens, then the layer-1 K/V projection), and the GPU's
    probe sets as valid top-b sets of both."""
    L, hkv, hd = SHAPE.n_layers, SHAPE.n_kv_heads, SHAPE.head_dim
    kc = torch.empty((L, TC, hkv, hd), dtype=torch.bfloat16)
    vc = torch.empty_like(kc)
    for l in (0, 1):
        kc[l] = storage_round(synthetic.random_array((TC, hkv, hd), 700 + l), torch.bfloat16)
        vc[l] = storage_round(synthetic.random_array((TC, hkv, hd), 800 + l), torch.bfloat16)
    kc[2:] = kc[1]
    vc[2:] = vc[1]
    out = run(bench_case, k=to_dev(kc), v=to_dev(vc))
    d_k, d_v = f64(out["d_k"]), f64(out["d_v"])

    # oracle: the device-drawn weights of layers 0 and 1 and the token embeddings
    dims = oracle.dims_from(SHAPE.with_layers(2))
    w = bench_case["w"]
    layers = [oracle.split_layer({k: t.cpu() for k, t in w["layers"][l].items()}, dims)
              for l in (0, 1)]
    toks = bench_case["toks"].cpu().numpy()
    h = f64(w["embed"][bench_case["toks"]])
    pos = np.arange(T)
    h, _, _ = oracle.decoder_layer(h, pos, layers[0], dims)
    _, k1, v1 = oracle.model.project_qkv(h[:TC], pos[:TC], layers[1], dims)
    starts = oracle.chunk_starts(LENS)
    kre = np.concatenate([oracle.rerotate(f64(kc[1, s:s + n]), s, SHAPE.rope_theta)
                          for s, n in zip(starts, LENS)])
    ref_k = oracle.divergence(k1, kre)
    ref_v = oracle.divergence(v1, f64(vc[1]))
    assert max_rel(d_k, ref_k) < 2e-2 and max_rel(d_v, ref_v) < 2e-2
    assert len(toks) == T
    budgets = [oracle.probe_budget(n, 1, 5) for n in LENS]
    sb = sum(budgets)
    off = np.concatenate([[0], np.cumsum(budgets)])
    pk = out["probe_k"][:sb].cpu().numpy()
    pv = out["probe_v"][:sb].cpu().numpy()
    slack_k = 2 * np.abs(d_k - ref_k).max()
    slack_v = 2 * np.abs(d_v - ref_v).max()
    check_valid_top_b(ref_k, d_k, [pk[off[i]:off[i + 1]] for i in range(len(LENS))], starts, LENS,
                      budgets, slack_k)
    check_valid_top_b(ref_v, d_v, [pv[off[i]:off[i + 1]] for i in range(len(LENS))], starts, LENS,
                      budgets, slack_v)


@pytest.mark.parametrize("name,n_ctx,rows_kind", [
    ("32b", 2600, "all"), ("32b", 2600, "probe"), ("7b", 4200, "all"), ("7b", 4200, "probe")])
def test_attention_head_layouts_sampled_rows(name, n_ctx, rows_kind):
    """Attention at the 32B (40 query heads over 8 KV heads) and 7B (28 over 4) head
    layouts. All positions of a context: several query heads of one KV head per block,
    sharing each K/V tile (5 and 7 heads per block at these row counts). About 900
    probe-like rows: one head per block with key splits. Sampled rows, the tile edges and
    the last rows among them, against per-row oracle attention, with and without the
    split workspace."""
    shape = synthetic.SHAPES[name]
    hq, hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    if rows_kind == "all":
        pos = np.arange(n_ctx, dtype=np.int32)
    else:
        rng = np.random.default_rng(n_ctx)
        pick = rng.choice(n_ctx - 64, size=900 - 64, replace=False)
        pos = np.sort(np.concatenate([pick, np.arange(n_ctx - 64, n_ctx)])).astype(np.int32)
    n = len(pos)
    q = storage_round(synthetic.random_array((n, hq, hd), 71), torch.bfloat16)
    k = storage_round(synthetic.random_array((n_ctx, hkv, hd), 72) * 3, torch.bfloat16)
    v = storage_round(synthetic.random_array((n_ctx, hkv, hd), 73), torch.bfloat16)
    m = akvs.model_cfg(shape, n_layers=1)
    qd, pd, kd, vd = to_dev(q), to_dev(pos), to_dev(k), to_dev(v)
    out_plain = torch.empty((n, hq * hd), dtype=torch.bfloat16, device=DEV)
    akvs.akvs_sparse_query_attention(qd, pd, n, kd, vd, n_ctx, m, out_plain)
    outs = [out_plain]
    ws_bytes = akvs.akvs_attention_workspace_size(m, n, n_ctx)
    if ws_bytes:
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
        out_split = torch.empty_like(out_plain)
        akvs.akvs_sparse_query_attention(qd, pd, n, kd, vd, n_ctx, m, out_split, ws)
        outs.append(out_split)
    torch.cuda.synchronize()
    edges = [e for e in (31, 32, 63, 64, 127, 128, 159, 160, n - 65, n - 64) if 0 <= e < n]
    rows = np.union1d(sample_rows(n, 29, 3), edges)
    ref = oracle.attention(f64(q)[rows], pos[rows], f64(k), f64(v),
                           np.arange(n_ctx)).reshape(len(rows), -1)
    for o in outs:
        assert max_rel(f64(o)[rows], ref) < 1e-2
    if len(outs) == 2:
        assert max_rel(f64(outs[1]), f64(outs[0])) < 1e-2
