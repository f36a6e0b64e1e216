"""Exact pins of the oracle's whole reuse procedure (Algorithm 1, Sec. 3.3) at refresh
ratios strictly between 0 and 1.

Construction. Take the full prefill's per-layer keys and values of the concatenated
context and build each unit's cache from them minus a constant of that unit and layer:
cached K_i^l = Rot(-s_i)(K_full^l[unit i] - mu_i^l), cached V_i^l = V_full^l[unit i] - nu_i^l.
Re-rotating by s_i gives K_reuse = K_full - mu_i^l exactly (up to rounding), so the
residual fresh - reused of every token of unit i is the constant mu_i^l (nu_i^l). Then,
by induction over the layers from the check layer on:
  * the recomputed rows carry the full prefill's hidden states, so their fresh keys and
    values are the full prefill's;
  * the probe mean of a unit is mu_i^l exactly ("Mean estimation");
  * with weight 1 the corrected state K_reuse + mu_i^l is K_full ("AgentKVShift
    correction"), so the rows' attention over the corrected cache is the full prefill's
    attention and their next hidden states are the full prefill's.
Hence h_query and every layer's K_corr / V_corr equal the full prefill's. The offsets
differ per layer, so taking a layer's offset from another layer, attending over the
uncorrected cache, applying the correction after the layer's attention, or correcting
with the wrong side's offset or sign all break the equality.

At the check layer itself the same construction with ||mu_i^c|| < 1 gives a closed form
for that layer alone (the weights are w = ||mu_i^c||): a non-probe token holds
K_full - (1 - ||mu_i^c||) mu_i^c, which pins that the check layer corrects its non-probe
tokens rather than taking the fresh states it computed for every token (Alg. 1 keeps the
fresh states of the probes only).
"""
import numpy as np
import pytest

import oracle
from tests.oracle_fixtures import small_model, context

LENS = [7, 11, 5, 9]
Q = 5


def unit_constant_caches(k_full, v_full, lens, theta, rng, norm_k, norm_v, pre_rope=False):
    """Unit caches equal to the full prefill's states minus one constant per unit and layer
    (keys rotated back to the unit's own positions 0..n_i-1). norm_k / norm_v: callables
    layer -> norm of that layer's offsets. pre_rope: the key constant is applied before the
    rotary map (a pre-RoPE shift: Rot(p) delta at position p).

    Returns (k caches, v caches, key constants [L][m][Hkv][hd], value constants)."""
    L, _, hkv, hd = k_full.shape
    starts = oracle.chunk_starts(lens)
    m = len(lens)
    mu = np.empty((L, m, hkv, hd))
    nu = np.empty((L, m, hkv, hd))
    for l in range(L):
        for i in range(m):
            a = rng.standard_normal((hkv, hd))
            b = rng.standard_normal((hkv, hd))
            mu[l, i] = a * (norm_k(l) / np.linalg.norm(a))
            nu[l, i] = b * (norm_v(l) / np.linalg.norm(b))
    kc, vc = [], []
    for i, (s, n) in enumerate(zip(starts, lens)):
        ks, vs = [], []
        for l in range(L):
            seg_k = k_full[l, s:s + n]
            if pre_rope:
                shift = oracle.model.rotate(np.broadcast_to(mu[l, i], (n, hkv, hd)).copy(),
                                            np.arange(s, s + n), theta)
            else:
                shift = mu[l, i][None]
            ks.append(oracle.rerotate(seg_k - shift, -int(s), theta))
            vs.append(v_full[l, s:s + n] - nu[l, i][None])
        kc.append(np.stack(ks))
        vc.append(np.stack(vs))
    return kc, vc, mu, nu


@pytest.fixture(scope="module")
def model():
    dims, w, V = small_model(seed=31, L=4, D=32, hq=4, hkv=2, hd=8, F=40)
    toks = context(31, LENS, Q, V)
    h, k, v = oracle.full_prefill(toks, 0, w, dims)
    return dims, w, toks, h, k, v


def assert_equals_full(out, h, k, v, atol=1e-9):
    np.testing.assert_allclose(out["h_query"], h[-Q:], rtol=0, atol=atol)
    for l in range(k.shape[0]):  # every layer on its own
        np.testing.assert_allclose(out["k_corr"][l], k[l], rtol=0, atol=atol, err_msg=f"K layer {l}")
        np.testing.assert_allclose(out["v_corr"][l], v[l], rtol=0, atol=atol, err_msg=f"V layer {l}")


@pytest.mark.parametrize("refresh", [(1, 4), (1, 2)])
@pytest.mark.parametrize("check_layer", [1, 2])
@pytest.mark.parametrize("weights", ["unit", "min(d,1)"])
def test_per_unit_constant_residual_reproduces_full_prefill(model, refresh, check_layer, weights):
    """Caches = full prefill minus a per-unit, per-layer constant: the reuse prefill at
    0 < r < 1 returns the full prefill's query states and every layer's K/V. With the
    paper's weights min(d, 1) the check-layer constants have norm >= 1, so every weight is
    1 (d of a unit token is the norm of its unit's constant)."""
    dims, w, toks, h, k, v = model
    rng = np.random.default_rng(100 + 10 * check_layer + refresh[1])
    kc, vc, mu, nu = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                          lambda l: 1.5 + 0.5 * l, lambda l: 2.0 + 0.25 * l)
    flags = oracle.F_UNIT_WEIGHTS if weights == "unit" else 0
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=refresh,
                               check_layer=check_layer, flags=flags)
    tc = sum(LENS)
    starts = oracle.chunk_starts(LENS)
    # 0 < r < 1: some but not all unit tokens are recomputed
    assert Q < len(out["rows"]) < tc + Q
    # the check-layer divergence of a unit token is its unit's constant's norm
    for i, (s, n) in enumerate(zip(starts, LENS)):
        np.testing.assert_allclose(out["d_k"][s:s + n], np.linalg.norm(mu[check_layer, i]),
                                   rtol=1e-12)
        np.testing.assert_allclose(out["d_v"][s:s + n], np.linalg.norm(nu[check_layer, i]),
                                   rtol=1e-12)
    np.testing.assert_array_equal(out["w_k"], 1.0)
    assert_equals_full(out, h, k, v)


def test_asymmetric_budgets_and_fresh_if_recomputed_reproduce_full_prefill(model):
    dims, w, toks, h, k, v = model
    rng = np.random.default_rng(7)
    kc, vc, _, _ = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                        lambda l: 1.2, lambda l: 3.0)
    for flags in (oracle.F_UNIT_WEIGHTS, oracle.F_FRESH_IF_RECOMPUTED):
        out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 4),
                                   check_layer=1, flags=flags, refresh_v=(1, 3))
        assert_equals_full(out, h, k, v)


def test_pre_rope_constant_is_recovered_by_pre_rope_offsets(model):
    """A constant shift before the rotary map (Rot(p) delta_i at position p): the pre-RoPE
    offsets reproduce the full prefill exactly; the post-RoPE offsets do not."""
    dims, w, toks, h, k, v = model
    rng = np.random.default_rng(8)
    kc, vc, _, _ = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                        lambda l: 1.5, lambda l: 1.5, pre_rope=True)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1,
                               flags=oracle.F_PRE_ROPE_OFFSETS)
    assert_equals_full(out, h, k, v)
    post = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=1)
    assert np.abs(post["k_corr"][2] - k[2]).max() > 1e-3


def test_check_layer_corrects_its_non_probe_tokens(model):
    """||mu^c|| < 1 at the check layer: weights are ||mu_i^c||, the probes take the fresh
    (= full prefill) states and every other unit token of unit i holds
    K_full - (1 - ||mu_i^c||) mu_i^c at the check layer; layers before it are the full
    prefill's. Taking the check layer's fresh states for every token would give K_full."""
    dims, w, toks, h, k, v = model
    c = 1
    rng = np.random.default_rng(9)
    kc, vc, mu, nu = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                          lambda l: 0.4 if l == c else 2.0,
                                          lambda l: 0.7 if l == c else 2.0)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=c)
    starts = oracle.chunk_starts(LENS)
    for l in range(c):
        np.testing.assert_allclose(out["k_corr"][l], k[l], rtol=0, atol=1e-10)
        np.testing.assert_allclose(out["v_corr"][l], v[l], rtol=0, atol=1e-10)
    for i, (s, n) in enumerate(zip(starts, LENS)):
        nk, nv = np.linalg.norm(mu[c, i]), np.linalg.norm(nu[c, i])
        np.testing.assert_allclose(out["w_k"][s:s + n], nk, rtol=1e-12)
        np.testing.assert_allclose(out["w_v"][s:s + n], nv, rtol=1e-12)
        pk, pv = set(out["probe_k"][i].tolist()), set(out["probe_v"][i].tolist())
        for t in range(s, s + n):
            ek = k[c, t] if t in pk else k[c, t] - (1.0 - nk) * mu[c, i]
            ev = v[c, t] if t in pv else v[c, t] - (1.0 - nv) * nu[c, i]
            np.testing.assert_allclose(out["k_corr"][c, t], ek, rtol=0, atol=1e-10)
            np.testing.assert_allclose(out["v_corr"][c, t], ev, rtol=0, atol=1e-10)
    tc = sum(LENS)
    np.testing.assert_allclose(out["k_corr"][c, tc:], k[c, tc:], rtol=0, atol=1e-10)
    np.testing.assert_allclose(out["v_corr"][c, tc:], v[c, tc:], rtol=0, atol=1e-10)


def test_fresh_if_recomputed_gives_key_only_probes_their_fresh_values(model):
    """Probe sets handed over with S_K != S_V, ||nu^c|| < 1 at the check layer. A token in
    S_K but not S_V is recomputed: with the FRESH_IF_RECOMPUTED flag its value is the
    fresh one (= the full prefill's), by default (per-side membership, Algorithm 1) its
    value is corrected: V_full - (1 - ||nu_i^c||) nu_i^c. Symmetrically for value-only
    probes and their keys."""
    dims, w, toks, h, k, v = model
    c = 1
    rng = np.random.default_rng(10)
    kc, vc, mu, nu = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                          lambda l: 0.5, lambda l: 0.6)
    starts = oracle.chunk_starts(LENS)
    bud = [oracle.probe_budget(n, 1, 3) for n in LENS]
    # keys: the first b positions of each unit, values: the last b (disjoint when b < n/2)
    pk = [np.arange(s, s + b) for s, b in zip(starts, bud)]
    pv = [np.arange(s + n - b, s + n) for s, n, b in zip(starts, LENS, bud)]
    for flags, fresh in ((0, False), (oracle.F_FRESH_IF_RECOMPUTED, True)):
        out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3),
                                   check_layer=c, flags=flags, probes=(pk, pv))
        for i, (s, n) in enumerate(zip(starts, LENS)):
            nk, nv = np.linalg.norm(mu[c, i]), np.linalg.norm(nu[c, i])
            for t in pk[i]:  # key-only probes: their values
                if t in pv[i]:
                    continue
                ev = v[c, t] if fresh else v[c, t] - (1.0 - nv) * nu[c, i]
                np.testing.assert_allclose(out["v_corr"][c, t], ev, rtol=0, atol=1e-10)
                np.testing.assert_allclose(out["k_corr"][c, t], k[c, t], rtol=0, atol=1e-10)
            for t in pv[i]:  # value-only probes: their keys
                if t in pk[i]:
                    continue
                ek = k[c, t] if fresh else k[c, t] - (1.0 - nk) * mu[c, i]
                np.testing.assert_allclose(out["k_corr"][c, t], ek, rtol=0, atol=1e-10)
                np.testing.assert_allclose(out["v_corr"][c, t], v[c, t], rtol=0, atol=1e-10)


def test_layer_zero_check_reproduces_full_prefill_with_unit_weights(model):
    """Check layer 0 (no prefix layer): the invariant still holds (the constants make the
    divergences non-zero even at the first layer)."""
    dims, w, toks, h, k, v = model
    rng = np.random.default_rng(11)
    kc, vc, _, _ = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                        lambda l: 1.0 + l, lambda l: 1.0 + l)
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 2), check_layer=0,
                               flags=oracle.F_UNIT_WEIGHTS)
    assert_equals_full(out, h, k, v)


def test_each_side_averages_over_its_own_probe_set(model):
    """Check layer c with handed-over, disjoint probe sets (keys: the first b tokens of a
    unit, values: the last b). The residual of a token is its unit's constant plus a
    perturbation that vanishes on that side's own probes: fresh - reused = mu_i + delta_t for
    keys (delta_t = 0 on S_K), nu_i + eps_t for values (eps_t = 0 on S_V). The offset of a
    side is the mean over its own probes, hence exactly mu_i / nu_i, and with every weight
    1 (||mu_i + delta_t|| >= 1) a non-probe token of that side holds
    reused + mu_i = K_full - delta_t (V_full - eps_t for values). A mean over the other
    side's probes would pick up the perturbations."""
    dims, w, toks, h, k, v = model
    c = 1
    L, _, hkv, hd = k.shape
    rng = np.random.default_rng(12)
    starts = oracle.chunk_starts(LENS)
    bud = [oracle.probe_budget(n, 1, 3) for n in LENS]
    pk = [np.arange(s, s + b) for s, b in zip(starts, bud)]
    pv = [np.arange(s + n - b, s + n) for s, n, b in zip(starts, LENS, bud)]
    kc, vc, mu, nu = unit_constant_caches(k, v, LENS, dims.rope_theta, rng,
                                          lambda l: 3.0, lambda l: 3.0)
    tc = sum(LENS)
    delta = np.zeros((tc, hkv, hd))
    eps = np.zeros((tc, hkv, hd))
    for i, (s, n) in enumerate(zip(starts, LENS)):
        for t in range(s, s + n):
            if t not in pk[i]:
                delta[t] = 0.5 * rng.standard_normal((hkv, hd)) / np.sqrt(hkv * hd)
            if t not in pv[i]:
                eps[t] = 0.5 * rng.standard_normal((hkv, hd)) / np.sqrt(hkv * hd)
        # the check layer's cache of unit i carries the perturbations too
        kc[i][c] = kc[i][c] - oracle.rerotate(delta[s:s + n], -int(s), dims.rope_theta)
        vc[i][c] = vc[i][c] - eps[s:s + n]
    out = oracle.reuse_prefill(toks, w, dims, LENS, Q, kc, vc, refresh=(1, 3), check_layer=c,
                               probes=(pk, pv))
    np.testing.assert_array_equal(out["w_k"], 1.0)
    np.testing.assert_array_equal(out["w_v"], 1.0)
    for i, (s, n) in enumerate(zip(starts, LENS)):
        for t in range(s, s + n):
            np.testing.assert_allclose(out["k_corr"][c, t], k[c, t] - delta[t], rtol=0, atol=1e-10)
            np.testing.assert_allclose(out["v_corr"][c, t], v[c, t] - eps[t], rtol=0, atol=1e-10)
