"""Step entries of the C ABI against the CPU oracle on identical seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
import synthetic
from paper_2607_21604_amd import akvs
from tests.gpu_util import DEV, to_dev, f64, max_rel, storage_round, oracle_quantized
from tests.libutil import ensure_built

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def rope(n_pos, hd, theta):
    t = torch.empty((n_pos, hd // 2, 2), dtype=torch.float32, device=DEV)
    akvs.akvs_rope_table(n_pos, hd, theta, t)
    return t


def test_rope_table_matches_fp64_angles():
    for hd, theta, n in ((128, 1e6, 16200), (64, 1e4, 300)):
        t = rope(n, hd, theta).cpu().numpy()
        c, s = oracle.rope_cos_sin(np.arange(n), hd, theta)
        assert np.abs(t[..., 0] - c).max() < 2e-7 and np.abs(t[..., 1] - s).max() < 2e-7


def unit_layout(lens):
    starts = oracle.chunk_starts(lens)
    delta = np.concatenate([np.full(n, s) for s, n in zip(starts, lens)]).astype(np.int32)
    return starts, delta


@pytest.mark.parametrize("dtype,hkv,hd", [("bf16", 8, 128), ("f32", 4, 64), ("bf16", 3, 64)])
def test_rerotate_keys(dtype, hkv, hd):
    lens = [37, 1, 64, 130]
    starts, delta = unit_layout(lens)
    n = int(sum(lens))
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    k = storage_round(synthetic.random_array((n, hkv, hd), 1), tdt)
    v = storage_round(synthetic.random_array((n, hkv, hd), 2), tdt)
    tab = rope(n + 10, hd, 1e4)
    kd = torch.empty((n, hkv, hd), dtype=tdt, device=DEV)
    vd = torch.empty_like(kd)
    akvs.akvs_rerotate_keys(akvs.cache_struct(to_dev(k), to_dev(v)), n, hkv, hd, to_dev(delta), tab,
                            n + 10, kd, vd, akvs.dtype_code(kd))
    ref_k = np.concatenate([oracle.rerotate(f64(k)[s:s + m], s, 1e4) for s, m in zip(starts, lens)])
    tol = 4e-3 if dtype == "bf16" else 2e-6
    assert max_rel(f64(kd), ref_k) < tol
    assert torch.equal(vd.cpu(), v)
    # zero offset leaves keys unchanged bit for bit
    akvs.akvs_rerotate_keys(akvs.cache_struct(to_dev(k), to_dev(v)), n, hkv, hd,
                            to_dev(np.zeros(n, np.int32)), tab, n + 10, kd, vd, akvs.dtype_code(kd))
    assert torch.equal(kd.cpu(), k)


@pytest.mark.parametrize("bits", [4, 2, 8])
def test_rerotate_quantised_cache(bits):
    lens = [64, 70]
    starts, delta = unit_layout(lens)
    n, hkv, hd = 134, 4, 128
    x = storage_round(synthetic.random_array((2, n, hkv, hd), 3), torch.bfloat16)
    packed, meta, deq, dt = oracle_quantized(f64(x), bits)
    tab = rope(n, hd, 1e6)
    kd = torch.empty((n, hkv, hd), dtype=torch.bfloat16, device=DEV)
    vd = torch.empty_like(kd)
    cache = akvs.Cache(0, 0, 0, 0, dt)
    kq, vq = to_dev(packed[0]), to_dev(packed[1])
    km, vm = to_dev(meta[0]), to_dev(meta[1])
    cache.k, cache.v, cache.k_meta, cache.v_meta = kq.data_ptr(), vq.data_ptr(), km.data_ptr(), vm.data_ptr()
    akvs.akvs_rerotate_keys(cache, n, hkv, hd, to_dev(delta), tab, n, kd, vd, akvs.AKVS_BF16)
    ref_k = np.concatenate([oracle.rerotate(deq[0][s:s + m], s, 1e6) for s, m in zip(starts, lens)])
    assert max_rel(f64(kd), ref_k) < 4e-3
    assert max_rel(f64(vd), deq[1]) < 4e-3


@pytest.mark.parametrize("fresh_dtype", ["bf16", "f32"])
def test_check_divergence(fresh_dtype):
    lens = [100, 3, 200]
    starts, delta = unit_layout(lens)
    n, hkv, hd = 303, 8, 128
    tdt = torch.bfloat16 if fresh_dtype == "bf16" else torch.float32
    kf = storage_round(synthetic.random_array((n, hkv, hd), 4), tdt)
    vf = storage_round(synthetic.random_array((n, hkv, hd), 5), tdt)
    kc = storage_round(synthetic.random_array((n, hkv, hd), 6), tdt)
    vc = storage_round(synthetic.random_array((n, hkv, hd), 7), tdt)
    tab = rope(n, hd, 1e6)
    dk = torch.empty(n, dtype=torch.float32, device=DEV)
    dv = torch.empty_like(dk)
    akvs.akvs_check_divergence(to_dev(kf), to_dev(vf), akvs.dtype_code(kf),
                               akvs.cache_struct(to_dev(kc), to_dev(vc)), n, hkv, hd, to_dev(delta),
                               tab, n, dk, dv)
    reuse = np.concatenate([oracle.rerotate(f64(kc)[s:s + m], s, 1e6) for s, m in zip(starts, lens)])
    np.testing.assert_allclose(f64(dk), oracle.divergence(f64(kf), reuse), rtol=2e-5)
    np.testing.assert_allclose(f64(dv), oracle.divergence(f64(vf), f64(vc)), rtol=2e-5)


def run_select(d_k, d_v, lens, q, refresh, flags=0, given=None, refresh_v=None):
    cfg = akvs.reuse_cfg(lens, q, refresh, 1, flags, refresh_v)
    meta, (tc, sum_b, cap, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
    out = {
        "probe_k": torch.full((max(sum_b, 1),), -7, dtype=torch.int32, device=DEV),
        "probe_v": torch.full((max(sum_bv, 1),), -7, dtype=torch.int32, device=DEV),
        "w_k": torch.empty(tc, dtype=torch.float32, device=DEV),
        "w_v": torch.empty(tc, dtype=torch.float32, device=DEV),
        "flags": torch.empty(tc, dtype=torch.uint8, device=DEV),
        "chunk_rows": torch.empty(len(lens), dtype=torch.int32, device=DEV),
        "rows": torch.full((t_all,), -7, dtype=torch.int32, device=DEV),
        "n_rows": torch.empty(1, dtype=torch.int32, device=DEV),
        "fresh_row": torch.empty(t_all, dtype=torch.int32, device=DEV),
    }
    if given is not None:
        out["probe_k"][:sum_b] = to_dev(np.concatenate(given[0]).astype(np.int32))
        out["probe_v"][:sum_bv] = to_dev(np.concatenate(given[1]).astype(np.int32))
    akvs.akvs_select_probes(to_dev(d_k.astype(np.float32)), to_dev(d_v.astype(np.float32)), cfg,
                            to_dev(meta), out["probe_k"], out["probe_v"], out["w_k"], out["w_v"],
                            out["flags"], out["chunk_rows"], out["rows"], out["n_rows"],
                            out["fresh_row"])
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, sum_b, cap


@pytest.mark.parametrize("refresh", [(3, 10), (1, 5), (0, 1), (1, 1), (1, 100)])
def test_select_probes_bit_exact(refresh):
    lens = [1, 7, 64, 65, 200, 1000, 2500]
    q = 5
    tc = sum(lens)
    rng = np.random.default_rng(9)
    d_k = rng.integers(0, 20, size=tc).astype(np.float32) * 0.25   # many ties
    d_v = rng.random(tc).astype(np.float32) * 3
    got, sum_b, cap = run_select(d_k, d_v, lens, q, refresh)
    starts = oracle.chunk_starts(lens)
    budgets = [oracle.probe_budget(n, *refresh) for n in lens]
    sk = [oracle.select_top(d_k[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets)]
    sv = [oracle.select_top(d_v[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets)]
    assert list(got["probe_k"][:sum_b]) == [int(x) for x in np.concatenate(sk)]
    assert list(got["probe_v"][:sum_b]) == [int(x) for x in np.concatenate(sv)]
    in_k = np.zeros(tc, bool); in_v = np.zeros(tc, bool)
    for p in sk: in_k[p] = True
    for p in sv: in_v[p] = True
    np.testing.assert_array_equal(got["flags"], in_k.astype(np.uint8) | (in_v.astype(np.uint8) << 1))
    rows = np.concatenate([np.nonzero(in_k | in_v)[0], np.arange(tc, tc + q)])
    assert int(got["n_rows"][0]) == len(rows) <= cap
    np.testing.assert_array_equal(got["rows"][:len(rows)], rows)
    fr = np.full(tc + q, -1); fr[rows] = np.arange(len(rows))
    np.testing.assert_array_equal(got["fresh_row"], fr)
    if refresh[0] > 0:
        np.testing.assert_array_equal(got["w_k"], np.minimum(d_k, np.float32(1)))
        np.testing.assert_array_equal(got["w_v"], np.minimum(d_v, np.float32(1)))


@pytest.mark.parametrize("refresh,refresh_v", [((1, 10), (1, 2)), ((1, 2), (0, 1)), ((0, 1), (3, 10))])
def test_select_probes_value_ratio_bit_exact(refresh, refresh_v):
    lens = [1, 7, 64, 65, 200, 1000]
    q = 4
    tc = sum(lens)
    rng = np.random.default_rng(19)
    d_k = rng.integers(0, 20, size=tc).astype(np.float32) * 0.25
    d_v = rng.random(tc).astype(np.float32) * 3
    got, sum_b, cap = run_select(d_k, d_v, lens, q, refresh, refresh_v=refresh_v)
    starts = oracle.chunk_starts(lens)
    bk = [oracle.probe_budget(n, *refresh) for n in lens]
    bv = [oracle.probe_budget(n, *refresh_v) for n in lens]
    sk = [oracle.select_top(d_k[s:s + n], b) + s for s, n, b in zip(starts, lens, bk)]
    sv = [oracle.select_top(d_v[s:s + n], b) + s for s, n, b in zip(starts, lens, bv)]
    assert list(got["probe_k"][:sum(bk)]) == [int(x) for x in np.concatenate(sk)]
    assert list(got["probe_v"][:sum(bv)]) == [int(x) for x in np.concatenate(sv)]
    in_k = np.zeros(tc, bool); in_v = np.zeros(tc, bool)
    for p in sk: in_k[p] = True
    for p in sv: in_v[p] = True
    rows = np.concatenate([np.nonzero(in_k | in_v)[0], np.arange(tc, tc + q)])
    assert int(got["n_rows"][0]) == len(rows) <= cap
    np.testing.assert_array_equal(got["rows"][:len(rows)], rows)
    wk = np.minimum(d_k, np.float32(1)) if refresh[0] else np.zeros(tc, np.float32)
    wv = np.minimum(d_v, np.float32(1)) if refresh_v[0] else np.zeros(tc, np.float32)
    np.testing.assert_array_equal(got["w_k"], wk)
    np.testing.assert_array_equal(got["w_v"], wv)


def test_select_given_probes_and_unit_weights():
    lens = [50, 80]
    rng = np.random.default_rng(10)
    d_k = rng.random(130).astype(np.float32)
    d_v = rng.random(130).astype(np.float32)
    given = ([np.array([1, 5, 9, 20, 49]) + 0, np.array([50, 51, 60, 70, 71, 90, 100, 129])],
             [np.array([0, 2, 4, 6, 8]), np.array([55, 56, 57, 58, 59, 60, 61, 62])])
    # budgets at r = 1/10: 5 and 8
    got, sum_b, _ = run_select(d_k, d_v, lens, 3, (1, 10),
                               akvs.AKVS_F_GIVEN_PROBES | akvs.AKVS_F_UNIT_WEIGHTS, given)
    assert list(got["probe_k"][:sum_b]) == list(np.concatenate(given[0]))
    union = sorted(set(np.concatenate(given[0])) | set(np.concatenate(given[1])))
    assert list(got["rows"][:int(got["n_rows"][0])]) == union + [130, 131, 132]
    assert np.all(got["w_k"] == 1) and np.all(got["w_v"] == 1)


def make_offset_case(dtype, lens, hkv, hd, seed, flags=0, refresh=(1, 5), refresh_v=None):
    """Random cache, divergences and fresh rows; the probe sets, recomputed rows and weights
    come from the oracle's selection on the same divergences."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    q = 3
    tc = sum(lens)
    starts, delta = unit_layout(lens)
    rng = np.random.default_rng(seed)
    d_k = rng.random(tc).astype(np.float32) * 2
    d_v = rng.random(tc).astype(np.float32) * 2
    budgets = [oracle.probe_budget(n, *refresh) for n in lens]
    budgets_v = [oracle.probe_budget(n, *(refresh_v or refresh)) for n in lens]
    sk = [oracle.select_top(d_k[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets)]
    sv = [oracle.select_top(d_v[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets_v)]
    in_k = np.zeros(tc, bool)
    in_v = np.zeros(tc, bool)
    for p in sk:
        in_k[p] = True
    for p in sv:
        in_v[p] = True
    rows = np.concatenate([np.nonzero(in_k | in_v)[0], np.arange(tc, tc + q)])
    fresh_row = np.full(tc + q, -1)
    fresh_row[rows] = np.arange(len(rows))
    unit = bool(flags & akvs.AKVS_F_UNIT_WEIGHTS)
    w_k = np.ones(tc) if unit else oracle.correction_weights(d_k)
    w_v = np.ones(tc) if unit else oracle.correction_weights(d_v)
    sel = {"probe_k": np.concatenate(sk).astype(np.int32), "probe_v": np.concatenate(sv).astype(np.int32),
           "w_k": w_k.astype(np.float32), "w_v": w_v.astype(np.float32),
           "flags": (in_k.astype(np.uint8) | (in_v.astype(np.uint8) << 1)),
           "fresh_row": fresh_row.astype(np.int32)}
    cap = len(rows)
    kc = storage_round(synthetic.random_array((tc, hkv, hd), seed + 1), tdt)
    vc = storage_round(synthetic.random_array((tc, hkv, hd), seed + 2), tdt)
    kf = storage_round(synthetic.random_array((cap, hkv, hd), seed + 3), tdt)
    vf = storage_round(synthetic.random_array((cap, hkv, hd), seed + 4), tdt)
    return dict(tdt=tdt, q=q, tc=tc, starts=starts, lens=lens, sel=sel, rows=rows, kc=kc, vc=vc,
                kf=kf, vf=vf, refresh=refresh, flags=flags, budgets=budgets, budgets_v=budgets_v,
                refresh_v=refresh_v)


def gpu_offset_and_correction(cs, hkv, hd, theta=1e6):
    lens, q = cs["lens"], cs["q"]
    cfg = akvs.reuse_cfg(lens, q, cs["refresh"], 1, cs["flags"], cs["refresh_v"])
    meta, (tc, sum_b, cap, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
    m = akvs.ModelCfg(1, 64, hkv, hkv, hd, 64, 16, theta, 1e-6, akvs.dtype_code(cs["kc"]))
    tab = rope(t_all, hd, theta)
    sel = {k: to_dev(v) for k, v in cs["sel"].items()}
    kc, vc, kf, vf = (to_dev(cs[k]) for k in ("kc", "vc", "kf", "vf"))
    cache = akvs.cache_struct(kc, vc)
    mu_k = torch.empty((len(lens), hkv, hd), dtype=torch.float32, device=DEV)
    mu_v = torch.empty_like(mu_k)
    akvs.akvs_chunk_offset(kf, vf, sel["fresh_row"], cache, cfg, to_dev(meta), sel["probe_k"],
                           sel["probe_v"], m, tab, t_all, mu_k, mu_v)
    k_corr = torch.empty((t_all, hkv, hd), dtype=cs["tdt"], device=DEV)
    v_corr = torch.empty_like(k_corr)
    akvs.akvs_apply_correction(cache, mu_k, mu_v, sel["w_k"], sel["w_v"], sel["flags"], kf, vf,
                               sel["fresh_row"], cfg, to_dev(meta), m, tab, t_all, k_corr, v_corr)
    torch.cuda.synchronize()
    return mu_k, mu_v, k_corr, v_corr


def oracle_offset_and_correction(cs, theta=1e6):
    """The same step on the CPU oracle from the same inputs."""
    lens, starts, q, tc = cs["lens"], cs["starts"], cs["q"], cs["tc"]
    sel = cs["sel"]
    off = np.concatenate([[0], np.cumsum(cs["budgets"])])
    off_v = np.concatenate([[0], np.cumsum(cs["budgets_v"])])
    kc, vc, kf, vf = (f64(cs[k]) for k in ("kc", "vc", "kf", "vf"))
    reuse_k = np.concatenate([oracle.rerotate(kc[s:s + n], s, theta) for s, n in zip(starts, lens)])
    fresh_k = np.zeros((tc + q,) + kc.shape[1:])
    fresh_v = np.zeros_like(fresh_k)
    fresh_k[cs["rows"]] = kf[:len(cs["rows"])]
    fresh_v[cs["rows"]] = vf[:len(cs["rows"])]
    mus_k, mus_v, ck, cv = [], [], [], []
    flags = cs["flags"]
    for i, (s, n) in enumerate(zip(starts, lens)):
        pk = sel["probe_k"][off[i]:off[i + 1]]
        pv = sel["probe_v"][off_v[i]:off_v[i + 1]]
        pre = bool(flags & oracle.F_PRE_ROPE_OFFSETS)
        if flags & oracle.F_NO_CORRECTION:
            mk = np.zeros(kc.shape[1:]); mv = np.zeros(kc.shape[1:])
        elif pre:
            mk = oracle.probe_offset_pre_rope(fresh_k[pk], reuse_k[pk], pk, theta)
            mv = oracle.probe_offset(fresh_v[pv], vc[pv])
        else:
            mk = oracle.probe_offset(fresh_k[pk], reuse_k[pk])
            mv = oracle.probe_offset(fresh_v[pv], vc[pv])
        mus_k.append(mk); mus_v.append(mv)
        f = sel["flags"][s:s + n]
        any_ = (f != 0) if flags & oracle.F_FRESH_IF_RECOMPUTED else np.zeros(n, bool)
        fk = (f & 1).astype(bool) | any_
        if pre:
            ck.append(oracle.correct_chunk_pre_rope(reuse_k[s:s + n], fresh_k[s:s + n], fk,
                                                    sel["w_k"][s:s + n], mk, np.arange(s, s + n),
                                                    theta))
        else:
            ck.append(oracle.correct_chunk(reuse_k[s:s + n], fresh_k[s:s + n], fk,
                                           sel["w_k"][s:s + n], mk))
        cv.append(oracle.correct_chunk(vc[s:s + n], fresh_v[s:s + n], (f & 2).astype(bool) | any_,
                                       sel["w_v"][s:s + n], mv))
    ck.append(fresh_k[tc:]); cv.append(fresh_v[tc:])
    return np.stack(mus_k), np.stack(mus_v), np.concatenate(ck), np.concatenate(cv)


@pytest.mark.parametrize("dtype,hkv,hd,flags,refresh_v", [
    ("bf16", 8, 128, 0, None), ("f32", 4, 64, 0, None),
    ("bf16", 4, 128, akvs.AKVS_F_FRESH_IF_RECOMPUTED, None),
    ("bf16", 2, 64, akvs.AKVS_F_NO_CORRECTION, None), ("f32", 2, 128, akvs.AKVS_F_UNIT_WEIGHTS, None),
    ("bf16", 8, 128, akvs.AKVS_F_PRE_ROPE_OFFSETS, None), ("f32", 4, 64, akvs.AKVS_F_PRE_ROPE_OFFSETS, None),
    ("bf16", 8, 128, 0, (1, 2)), ("f32", 4, 64, akvs.AKVS_F_PRE_ROPE_OFFSETS, (0, 1))])
def test_chunk_offset_and_correction(dtype, hkv, hd, flags, refresh_v):
    cs = make_offset_case(dtype, [23, 64, 1, 150], hkv, hd, seed=11, flags=flags,
                          refresh_v=refresh_v)
    mu_k, mu_v, k_corr, v_corr = gpu_offset_and_correction(cs, hkv, hd)
    rmk, rmv, rck, rcv = oracle_offset_and_correction(cs)
    tol = 1e-5
    assert max_rel(f64(mu_k), rmk) < tol and max_rel(f64(mu_v), rmv) < tol
    tol = 4e-3 if dtype == "bf16" else 2e-6
    assert max_rel(f64(k_corr), rck) < tol
    assert max_rel(f64(v_corr), rcv) < tol


def test_constant_residual_is_recovered_on_gpu():
    """Fresh = rotated cache + mu_i with every weight 1: the corrected cache equals the
    fresh states (within one bf16 rounding)."""
    lens, hkv, hd, q = [40, 70, 33], 8, 128, 3
    cs = make_offset_case("f32", lens, hkv, hd, seed=21, flags=akvs.AKVS_F_UNIT_WEIGHTS)
    starts, tc = cs["starts"], cs["tc"]
    rng = np.random.default_rng(5)
    mu = rng.standard_normal((len(lens), hkv, hd))
    kc, vc = f64(cs["kc"]), f64(cs["vc"])
    reuse_k = np.concatenate([oracle.rerotate(kc[s:s + n], s, 1e6) for s, n in zip(starts, lens)])
    true_k = reuse_k + np.concatenate([np.broadcast_to(mu[i], (n, hkv, hd)) for i, n in enumerate(lens)])
    true_v = vc + np.concatenate([np.broadcast_to(mu[i], (n, hkv, hd)) for i, n in enumerate(lens)])
    rows = cs["rows"]
    kf = np.zeros((len(rows), hkv, hd)); vf = np.zeros_like(kf)
    kf[:len(rows) - q] = true_k[rows[:-q]]; vf[:len(rows) - q] = true_v[rows[:-q]]
    cs["kf"] = storage_round(kf, torch.float32); cs["vf"] = storage_round(vf, torch.float32)
    mu_k, _, k_corr, v_corr = gpu_offset_and_correction(cs, hkv, hd)
    assert max_rel(f64(mu_k), mu) < 1e-5
    assert max_rel(f64(k_corr)[:tc], true_k) < 1e-5
    assert max_rel(f64(v_corr)[:tc], true_v) < 1e-5


@pytest.mark.parametrize("dtype,hq,hkv,hd,n_rows,n_keys", [
    ("bf16", 6, 2, 128, 77, 300), ("bf16", 28, 4, 128, 130, 1000), ("bf16", 4, 4, 64, 64, 64),
    ("bf16", 24, 8, 128, 600, 2400), ("bf16", 6, 2, 128, 5, 2000), ("bf16", 24, 8, 128, 3, 4096),
    ("bf16", 28, 4, 128, 1700, 2600), ("bf16", 16, 2, 64, 700, 3000),
    ("bf16", 64, 8, 128, 900, 3000), ("bf16", 2, 1, 128, 5000, 6000),
    ("f32", 4, 4, 64, 50, 288), ("f32", 6, 3, 128, 9, 70)])
def test_sparse_query_attention(dtype, hq, hkv, hd, n_rows, n_keys):
    """Against the oracle with and without the key-split workspace. With it, the bf16 calls
    run the planned split: one round of 128-row blocks (600 rows over 2400 keys; hd 64 at
    700 over 3000), one round of 256-row blocks (the few-row cases, up to 8 pieces per tile)
    and two rounds of them (1700 rows over 2600 keys at 28 query heads; 900 over 3000 at 64),
    tiles in one piece writing their rows directly; at 2 query heads one round of forty
    128-row tiles in up to 8 pieces each."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    rng = np.random.default_rng(n_rows)
    pos = np.sort(rng.choice(n_keys, size=n_rows, replace=False)).astype(np.int32)
    q = storage_round(synthetic.random_array((n_rows, hq, hd), 31), tdt)
    k = storage_round(synthetic.random_array((n_keys, hkv, hd), 32), tdt)
    v = storage_round(synthetic.random_array((n_keys, hkv, hd), 33), tdt)
    m = akvs.ModelCfg(1, 64, hq, hkv, hd, 64, 16, 1e4, 1e-6, akvs.dtype_code(q))
    ref = oracle.attention(f64(q), pos, f64(k), f64(v), np.arange(n_keys)).reshape(n_rows, -1)
    nbytes = akvs.akvs_attention_workspace_size(m, n_rows, n_keys)
    # the key-split workspace starts as all-ones bytes (NaN floats): splits whose keys all
    # lie past a row's position must not carry any of it into the merge
    outs = []
    for ws in (None, torch.full((max(nbytes, 1),), 255, dtype=torch.uint8, device=DEV),
               torch.zeros(max(nbytes, 1), dtype=torch.uint8, device=DEV)):
        out = torch.empty((n_rows, hq * hd), dtype=tdt, device=DEV)
        akvs.akvs_sparse_query_attention(to_dev(q), to_dev(pos), n_rows, to_dev(k), to_dev(v), n_keys,
                                         m, out, ws)
        assert max_rel(f64(out), ref) < (1e-2 if dtype == "bf16" else 1e-5)
        outs.append(out)
    assert torch.equal(outs[1], outs[2])


def gemm_case(shape, n_rows, seed):
    w = synthetic.make_weights(shape, seed=seed, n_layers=1, embed=False)
    dims = oracle.dims_from(shape.with_layers(1))
    lw = w["layers"][0]
    rng = np.random.default_rng(seed)
    h = rng.standard_normal((n_rows, shape.d_model)) * 0.5
    return w, dims, lw, h


@pytest.mark.parametrize("name,n_rows", [("3b", 200), ("7b", 129), ("32b", 300), ("tiny", 70),
                                         ("3b", 1), ("3b", 257), ("7b", 700), ("tiny", 1),
                                         ("tiny", 33)])
def test_probe_qkv_and_out_mlp(name, n_rows):
    """Probe-row projections (QKV with the rotary map, output projection and MLP with the
    residual adds) against the oracle. Row counts from 1 to 700 cross the 16-, 32-, 192- and
    256-row tile edges and take both the K-split and the unsplit launches; tiny is the fp32
    path with 64-wide heads."""
    shape = synthetic.SHAPES[name]
    w, dims, lw, h = gemm_case(shape, n_rows, seed=3)
    tdt = synthetic.torch_dtype(shape)
    m = akvs.model_cfg(shape, n_layers=1)
    lwd = {k: to_dev(t) for k, t in lw.items()}
    lws = akvs.layer_array({"layers": [lwd]})[0]
    rng = np.random.default_rng(4)
    pos = np.sort(rng.choice(20000, size=n_rows, replace=False)).astype(np.int32)
    tab = rope(20000, shape.head_dim, shape.rope_theta)
    hq, hkv, hd = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    q = torch.empty((n_rows, hq, hd), dtype=tdt, device=DEV)
    kf = torch.empty((n_rows, hkv, hd), dtype=tdt, device=DEV)
    vf = torch.empty_like(kf)
    ws = torch.empty(akvs.akvs_step_workspace_size(m, n_rows), dtype=torch.uint8, device=DEV)
    h32 = h.astype(np.float32)
    h_dev = to_dev(h32)
    akvs.akvs_probe_qkv(h_dev, n_rows, to_dev(pos), m, lws, tab, 20000, q, kf, vf, ws)
    sw = oracle.split_layer(lw, dims)
    rq, rk, rv = oracle.model.project_qkv(h32.astype(np.float64), pos, sw, dims)
    tol = 2e-2 if shape.dtype == "bf16" else 1e-5
    assert max_rel(f64(q), rq) < tol and max_rel(f64(kf), rk) < tol and max_rel(f64(vf), rv) < tol
    att = storage_round(synthetic.random_array((n_rows, hq * hd), 5), tdt)
    akvs.akvs_probe_out_mlp(h_dev, n_rows, to_dev(att), m, lws, ws)
    ref = oracle.model.output_and_mlp(h32.astype(np.float64), f64(att), sw, dims)
    assert max_rel(f64(h_dev), ref) < tol


def test_e4m3_cache_decodes_every_byte():
    """All 256 E4M3 bytes through the library's cache reader (the V copy of the
    re-rotation entry, scale 1): each gives the value of the format's definition."""
    hkv, hd, n = 1, 128, 2
    codes = np.arange(256, dtype=np.uint8).reshape(n, hkv, hd)
    meta = np.zeros((n, hkv, 2, 2), np.float16)
    meta[..., 0] = 1.0
    cache = akvs.Cache(0, 0, 0, 0, akvs.AKVS_E4M3G64)
    kq, vq, km = to_dev(codes), to_dev(codes), to_dev(meta)
    cache.k, cache.v, cache.k_meta, cache.v_meta = kq.data_ptr(), vq.data_ptr(), km.data_ptr(), km.data_ptr()
    kd = torch.empty((n, hkv, hd), dtype=torch.bfloat16, device=DEV)  # holds E4M3 values exactly
    vd = torch.empty_like(kd)
    akvs.akvs_rerotate_keys(cache, n, hkv, hd, to_dev(np.zeros(n, np.int32)), rope(n, hd, 1e6), n,
                            kd, vd, akvs.AKVS_BF16)
    got = vd.float().cpu().numpy().reshape(-1).astype(np.float64)
    ref = oracle.e4m3_value(np.arange(256))
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    np.testing.assert_array_equal(got[~np.isnan(ref)], ref[~np.isnan(ref)])


def test_quantize_e4m3_bit_exact():
    x = storage_round(synthetic.random_array((300, 128), 48), torch.bfloat16)
    x[7, :64] = 0.0           # all-zero group: scale 0, codes 0
    x[9, 64:] = 1e-3          # constant group
    pos = oracle.e4m3_value(np.arange(0x7F))
    mids = ((pos[:-1] + pos[1:]) / 2)[-63:]     # ties between neighbours, scale exactly 1
    x[11, :64] = torch.from_numpy(np.concatenate([[448.0], mids]))
    x[12, :64] = -x[11, :64]
    codes, meta = oracle.quantize_e4m3_g64(f64(x))
    c = torch.empty((300, 128), dtype=torch.uint8, device=DEV)
    mt = torch.empty((300, 2, 2), dtype=torch.float16, device=DEV)
    akvs.akvs_quantize_cache(to_dev(x), 300, 128, 8, c, mt)
    np.testing.assert_array_equal(c.cpu().numpy(), codes)
    np.testing.assert_array_equal(mt.cpu().numpy().view(np.uint16), meta.view(np.uint16))


@pytest.mark.parametrize("bits", [4, 2])
def test_quantize_cache_bit_exact(bits):
    x = storage_round(synthetic.random_array((300, 128), 40 + bits), torch.bfloat16)
    x[7, :64] = 0.25          # constant group: scale 0
    codes, meta = oracle.quantize_g64(f64(x), bits)
    c = torch.empty((300, 128 * bits // 8), dtype=torch.uint8, device=DEV)
    mt = torch.empty((300, 2, 2), dtype=torch.float16, device=DEV)
    akvs.akvs_quantize_cache(to_dev(x), 300, 128, bits, c, mt)
    np.testing.assert_array_equal(c.cpu().numpy(), oracle.pack_codes(codes, bits))
    np.testing.assert_array_equal(mt.cpu().numpy().view(np.uint16), meta.view(np.uint16))


def test_mfma_busy_loop_runs_and_rejects_bad_arguments():
    """The counter-calibration loop: every thread's sum is finite and the same for every
    block (the inputs depend on the thread index only); negative sizes are rejected."""
    out = torch.full((3 * 256,), float("nan"), dtype=torch.float32, device=DEV)
    akvs.akvs_mfma_busy_loop(3, 5, out)
    torch.cuda.synchronize()
    o = out.view(3, 256).cpu()
    assert torch.isfinite(o).all()
    assert torch.equal(o[0], o[1]) and torch.equal(o[0], o[2])
    with pytest.raises(akvs.AkvsError):
        akvs.akvs_mfma_busy_loop(-1, 5, out)
