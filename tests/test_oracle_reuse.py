"""Pins for the oracle's reuse procedure: closed forms, invariants, brute force, and
continuations computed by a third-party Llama."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle
from tests import hf_llama
from tests.oracle_fixtures import small_model, context

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_probe_budget_table():
    cases = json.load(open(os.path.join(GOLDEN, "probe_budgets.json")))["cases"]
    for c in cases:
        assert oracle.probe_budget(c["n"], c["num"], c["den"]) == c["b"], c
    # the float form of the same formula gets the 7 % case wrong
    assert int(np.ceil(0.07 * 100)) == 8


def test_divergence_closed_form():
    fresh = np.zeros((2, 2, 2))
    reuse = np.zeros((2, 2, 2))
    fresh[0, 0, 0], fresh[0, 1, 1] = 3.0, 4.0     # 3-4-5 across two heads
    reuse[1] = 1.0
    np.testing.assert_allclose(oracle.divergence(fresh, reuse), [5.0, 2.0])


def brute_top(d, b):
    """Among all b-subsets, the one every member of which outranks every non-member."""
    n = len(d)
    found = []
    for sub in itertools.combinations(range(n), b):
        rest = [k for k in range(n) if k not in sub]
        if all(d[j] > d[k] or (d[j] == d[k] and j < k) for j in sub for k in rest):
            found.append(sub)
    assert len(found) == 1
    return list(found[0])


def test_select_top_brute_force_with_ties():
    rng = np.random.default_rng(0)
    for trial in range(200):
        n = int(rng.integers(1, 9))
        d = rng.integers(0, 4, size=n).astype(float)   # many ties
        b = int(rng.integers(0, n + 1))
        assert list(oracle.select_top(d, b)) == brute_top(d, b)


def test_constant_residual_is_recovered_exactly():
    """Fresh = reused + mu_i per unit with ||mu_i|| >= 1: every weight is 1 and the
    corrected states equal the fresh ones (Sec. 3.4 offset model with zero fluctuation)."""
    rng = np.random.default_rng(1)
    n, H, hd = 30, 2, 8
    reuse = rng.standard_normal((n, H, hd))
    mu = rng.standard_normal((H, hd))
    mu *= 1.5 / np.linalg.norm(mu)
    fresh = reuse + mu
    d = oracle.divergence(fresh, reuse)
    np.testing.assert_allclose(d, 1.5)
    w = oracle.correction_weights(d)
    probes = oracle.select_top(d, 5)
    mu_hat = oracle.probe_offset(fresh[probes], reuse[probes])
    np.testing.assert_allclose(mu_hat, mu, atol=1e-14)
    is_probe = np.isin(np.arange(n), probes)
    corr = oracle.correct_chunk(reuse, fresh, is_probe, w, mu_hat)
    np.testing.assert_allclose(corr, fresh, atol=1e-14)


def test_small_constant_residual_is_scaled_by_its_norm():
    """||mu|| < 1: the weight is ||mu|| and non-probe tokens get reuse + ||mu|| mu."""
    rng = np.random.default_rng(2)
    reuse = rng.standard_normal((10, 1, 4))
    mu = np.array([[0.3, 0.0, -0.4, 0.0]])       # norm 0.5
    fresh = reuse + mu
    w = oracle.correction_weights(oracle.divergence(fresh, reuse))
    np.testing.assert_allclose(w, 0.5)
    is_probe = np.zeros(10, bool)
    is_probe[[2, 7]] = True
    corr = oracle.correct_chunk(reuse, fresh, is_probe, w, oracle.probe_offset(fresh[[2, 7]], reuse[[2, 7]]))
    np.testing.assert_allclose(corr[~is_probe], reuse[~is_probe] + 0.5 * mu, atol=1e-15)
    np.testing.assert_array_equal(corr[is_probe], fresh[is_probe])


def test_empty_probe_set_gives_zero_offset():
    z = oracle.probe_offset(np.zeros((0, 2, 4)), np.zeros((0, 2, 4)))
    assert z.shape == (2, 4) and not z.any()


def test_probe_mean_error_decays_like_inverse_sqrt_b():
    """Residuals mu + xi, probes drawn uniformly with replacement (the setting of Prop. 2):
    the offset error shrinks about as b^(-1/2) (App. C.2)."""
    rng = np.random.default_rng(3)
    n, dim, trials = 400, 16, 400
    mu = rng.standard_normal(dim)
    errs = {}
    for b in (4, 16, 64):
        e = []
        for _ in range(trials):
            resid = mu + rng.standard_normal((n, dim))
            idx = rng.integers(0, n, size=b)
            e.append(np.linalg.norm(oracle.probe_offset(resid[idx], np.zeros((b, dim))) - mu))
        errs[b] = np.mean(e)
    assert 1.6 < errs[4] / errs[16] < 2.5
    assert 1.6 < errs[16] / errs[64] < 2.5


# ---- whole procedure on a small random model ----------------------------------------

LENS = [6, 9, 5]
Q = 4


@pytest.fixture(scope="module")
def small():
    dims, w, V = small_model(seed=11, L=3)
    toks = context(11, LENS, Q, V)
    kc, vc = oracle.cache_units(toks, LENS, w, dims)
    return dims, w, V, toks, kc, vc


def test_full_refresh_equals_full_prefill(small):
    dims, w, V, toks, kc, vc = small
    h, kf, vf = oracle.full_prefill(toks, 0, w, dims)
    for c in (0, 1, 2):
        out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 1), check_layer=c)
        assert len(out["rows"]) == sum(LENS) + Q
        np.testing.assert_allclose(out["h_query"], h[-Q:], atol=1e-10)
        np.testing.assert_allclose(out["k_corr"], kf, atol=1e-10)
        np.testing.assert_allclose(out["v_corr"], vf, atol=1e-10)


def test_full_refresh_matches_transformers_llama(small):
    dims, w, V, toks, kc, vc = small
    ref_h, _, _ = hf_llama.prefill(hf_llama.build(w, dims, V), toks)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 1), check_layer=1)
    err = np.abs(out["h_query"] - ref_h[-Q:]).max()
    assert err <= 1e-5 * np.abs(ref_h).max()


def test_stale_reuse_matches_transformers_continuation(small):
    """Refresh 0 without a check layer: every unit's cached K/V re-rotated to its new
    offset and used as is at every layer; the query continues on top of that cache."""
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(0, 1),
                               flags=oracle.F_NO_PREFIX_RECOMPUTE)
    tc = sum(LENS)
    starts = oracle.chunk_starts(LENS)
    past_k = np.concatenate([np.stack([oracle.rerotate(kc[i][l], starts[i], dims.rope_theta)
                                       for l in range(dims.n_layers)]) for i in range(3)], axis=1)
    past_v = np.concatenate([vc[i] for i in range(3)], axis=1)
    np.testing.assert_allclose(out["k_corr"][:, :tc], past_k, atol=1e-13)
    np.testing.assert_array_equal(out["v_corr"][:, :tc], past_v)
    ref = hf_llama.continue_from(hf_llama.build(w, dims, V), past_k, past_v, toks[tc:], tc)
    err = np.abs(out["h_query"] - ref).max()
    assert err <= 1e-5 * np.abs(ref).max()
    assert list(out["rows"]) == list(range(tc, tc + Q))


def test_no_correction_keeps_probes_fresh_and_the_rest_stale(small):
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                               flags=oracle.F_NO_CORRECTION)
    tc = sum(LENS)
    in_k = np.zeros(tc, bool)
    for p in out["probe_k"]:
        in_k[p] = True
    for l in range(1, dims.n_layers):
        np.testing.assert_array_equal(out["k_corr"][l, :tc][~in_k], out["k_reuse"][l][~in_k])
    # layer 0 precedes the check layer and is fresh for every token
    _, kf, _ = oracle.full_prefill(toks, 0, w, dims)
    np.testing.assert_allclose(out["k_corr"][0], kf[0], atol=1e-12)


def test_probe_sets_sizes_order_and_weights(small):
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    starts = oracle.chunk_starts(LENS)
    for i, n in enumerate(LENS):
        b = oracle.probe_budget(n, 1, 3)
        for side, d in ((out["probe_k"][i], out["d_k"]), (out["probe_v"][i], out["d_v"])):
            assert len(side) == b and np.all(np.diff(side) > 0)
            seg = d[starts[i]:starts[i] + n]
            assert list(side - starts[i]) == brute_top(seg, b)
    np.testing.assert_array_equal(out["w_k"], np.minimum(out["d_k"], 1.0))
    rows = out["rows"]
    assert np.all(np.diff(rows) > 0) and list(rows[-Q:]) == list(range(sum(LENS), sum(LENS) + Q))


def test_first_unit_has_no_residual(small):
    """Unit 1 sits at position 0 with nothing before it: its cache equals its fresh
    states, so its divergence, offset and correction vanish (up to rounding)."""
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    n0 = LENS[0]
    assert np.abs(out["d_k"][:n0]).max() < 1e-12 and np.abs(out["d_v"][:n0]).max() < 1e-12
    _, kf, vf = oracle.full_prefill(toks, 0, w, dims)
    np.testing.assert_allclose(out["k_corr"][:, :n0], kf[:, :n0], atol=1e-12)


def test_check_layer_zero_has_no_value_divergence(small):
    """At the first layer a token's value depends on the token alone, so d_V is 0 up
    to rounding: a check at the very first layer cannot rank values, which is why the
    check layer defaults to the second."""
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=0)
    assert np.abs(out["d_v"]).max() < 1e-12
    assert np.abs(out["d_k"]).max() < 1e-12


def test_fresh_if_recomputed(small):
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                               flags=oracle.F_FRESH_IF_RECOMPUTED)
    base = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    # a token only in the K probe set gets a fresh V here, a corrected V in the default mode
    only_k = [j for p, q in zip(base["probe_k"], base["probe_v"]) for j in p if j not in q]
    assert only_k
    assert np.abs(out["v_corr"][2, only_k] - base["v_corr"][2, only_k]).max() > 1e-6


def test_given_probes_reproduce_own_selection_and_are_validated(small):
    dims, w, V, toks, kc, vc = small
    base = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    again = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                                 probes=(base["probe_k"], base["probe_v"]))
    np.testing.assert_array_equal(again["h_query"], base["h_query"])
    bad = [p.copy() for p in base["probe_k"]]
    bad[1] = bad[1][:-1]
    with pytest.raises(ValueError):
        oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                             probes=(bad, base["probe_v"]))


def test_correction_moves_reuse_towards_fresh_on_a_shifted_model(small):
    """Sanity of direction: the mean corrected error is below the stale error."""
    dims, w, V, toks, kc, vc = small
    _, kf, vf = oracle.full_prefill(toks, 0, w, dims)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 2), check_layer=1,
                               flags=oracle.F_UNIT_WEIGHTS)
    tc = sum(LENS)
    stale = np.abs(out["k_reuse"][1:] - kf[1:, :tc]).mean()
    corr = np.abs(out["k_corr"][1:, :tc] - kf[1:, :tc]).mean()
    assert corr < stale


# ---- variants: pre-RoPE key offsets, asymmetric K/V budgets --------------------------------

def test_pre_rope_offset_recovers_a_constant_pre_rope_shift():
    """Fresh keys that differ from the reused ones by one constant vector before the
    rotary map (after it: a different vector per position) are recovered exactly by the
    pre-RoPE offset, and the corrected keys equal the fresh ones; the post-RoPE mean of
    the same probes does not recover them."""
    rng = np.random.default_rng(21)
    n, H, hd, s0, theta = 24, 2, 8, 37, 10000.0
    pos = np.arange(s0, s0 + n)
    reuse = rng.standard_normal((n, H, hd))
    delta = rng.standard_normal((H, hd))
    delta *= 2.0 / np.linalg.norm(delta)
    shift = oracle.model.rotate(np.broadcast_to(delta, (n, H, hd)).copy(), pos, theta)
    fresh = reuse + shift
    probes = np.array([2, 5, 11, 19])
    mu = oracle.probe_offset_pre_rope(fresh[probes], reuse[probes], pos[probes], theta)
    np.testing.assert_allclose(mu, delta, atol=1e-13)
    w = oracle.correction_weights(oracle.divergence(fresh, reuse))
    np.testing.assert_allclose(w, 1.0)
    is_probe = np.isin(np.arange(n), probes)
    corr = oracle.correct_chunk_pre_rope(reuse, fresh, is_probe, w, mu, pos, theta)
    np.testing.assert_allclose(corr, fresh, atol=1e-13)
    post = oracle.probe_offset(fresh[probes], reuse[probes])
    assert np.abs(oracle.correct_chunk(reuse, fresh, is_probe, w, post) - fresh).max() > 1e-2


def test_pre_rope_offset_at_position_zero_equals_post_rope():
    """With every probe at position 0 the rotary map is the identity: both offsets agree."""
    rng = np.random.default_rng(22)
    f = rng.standard_normal((3, 2, 8))
    r = rng.standard_normal((3, 2, 8))
    np.testing.assert_allclose(oracle.probe_offset_pre_rope(f, r, [0, 0, 0], 1e4),
                               oracle.probe_offset(f, r), atol=1e-15)


def test_asymmetric_budgets_select_per_side(small):
    dims, w, V, toks, kc, vc = small
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                               refresh_v=(2, 3))
    starts = oracle.chunk_starts(LENS)
    for i, n in enumerate(LENS):
        bk, bv = oracle.probe_budget(n, 1, 3), oracle.probe_budget(n, 2, 3)
        assert out["budgets"][i] == bk and out["budgets_v"][i] == bv
        assert list(out["probe_k"][i] - starts[i]) == brute_top(out["d_k"][starts[i]:starts[i] + n], bk)
        assert list(out["probe_v"][i] - starts[i]) == brute_top(out["d_v"][starts[i]:starts[i] + n], bv)
    # equal ratios on both sides reproduce the symmetric call
    a = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                             refresh_v=(1, 3))
    b = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    np.testing.assert_array_equal(a["h_query"], b["h_query"])


def test_full_value_refresh_gives_fresh_values(small):
    """r_V = 1 recomputes every value: the corrected values of every layer from the check
    layer on are the fresh ones of that run, i.e. those of a full prefill when the keys
    are fully refreshed too."""
    dims, w, V, toks, kc, vc = small
    h, kf, vf = oracle.full_prefill(toks, 0, w, dims)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 1), check_layer=1,
                               refresh_v=(1, 1))
    np.testing.assert_allclose(out["v_corr"], vf, atol=1e-10)
    out2 = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(0, 1), check_layer=1,
                                refresh_v=(1, 1))
    assert len(out2["rows"]) == sum(LENS) + Q     # every unit token recomputed for its value
