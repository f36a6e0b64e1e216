"""Whole-procedure parity at full width and full sequence length, truncated depth.

Every bf16 workload shape is checked with all of its memory units and its query (the 3B
shape: 20 units of U{192..256} + 64, T = 4516; the 7B shape: 40 x 200 + 128, T = 8128, also
with 4-bit and 2-bit unit caches) over three layers (the prefix layer, the check layer and
one layer after it), and the 32B width (D = 5120, 40/8 heads, F = 27648) over three layers
with as many 200-token units as the test time allows. Each layer's corrected keys and
values and the query's final states are compared with the oracle's (Algorithm 1 return
value), the oracle's probe sets handed to the library so that the float comparison
isolates arithmetic; the library's own selection is checked against its own divergences.
The bf16 full prefill (the no-reuse baseline) is compared with the oracle's, and the exact
invariant of the oracle pins (unit caches equal to the full prefill's states minus one
constant per unit and layer reproduce the full prefill) is run on the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
from tests.gpu_util import to_dev, f64, max_rel, check_valid_top_b, oracle_quantized, storage_round
from tests.libutil import ensure_built
from tests.test_gpu_e2e import Case
from tests.test_oracle_alg1 import unit_constant_caches
from paper_2607_21604_amd import akvs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def own_selection_is_valid(case, out, ref):
    """The library's divergences agree with the oracle's, and its probe sets are valid
    top-b sets of its own divergences (and of the oracle's up to twice their difference)."""
    budgets = ref["budgets"]
    for side, key in (("probe_k", "d_k"), ("probe_v", "d_v")):
        d = f64(out[key])
        err = np.abs(d - ref[key]).max()
        assert err <= 2e-2 * np.abs(ref[key]).max(), (key, err)
        p = case.split(out[side].cpu().numpy(), budgets)
        check_valid_top_b(ref[key], d, p, case.starts, case.lens, budgets, 2 * err)


@pytest.fixture(scope="module")
def full3b():
    c = Case("3b", n_layers=3)
    assert sum(c.lens) + c.q == 4516
    c.full = oracle.full_prefill(c.toks, 0, c.w, c.dims, c.layers)
    return c


def test_3b_full_sequence_reuse_prefill(full3b):
    c = full3b
    ref = c.oracle()
    own = c.gpu()
    own_selection_is_valid(c, own, ref)
    errs = c.compare(c.gpu(probes=(ref["probe_k"], ref["probe_v"])), ref)
    print("3b full sequence", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.mark.parametrize("refresh", [(1, 100), (1, 10)])
def test_3b_full_sequence_low_refresh(full3b, refresh):
    """Small probe sets (171 and about 810 recomputed rows): the probe layer's attention
    runs the key split planned on the device from the live rows (8-wave blocks, per-tile
    split counts with end marks for the merge)."""
    c = full3b
    ref = c.oracle(refresh=refresh)
    errs = c.compare(c.gpu(refresh=refresh, probes=(ref["probe_k"], ref["probe_v"])), ref)
    print("3b full sequence r=%d/%d" % refresh, {k: f"{v:.2e}" for k, v in errs.items()})


def test_3b_full_sequence_full_prefill_bf16(full3b):
    """akvs_full_prefill (the speedup's denominator) against the oracle at bf16, 3 layers,
    every layer's keys and values and the final states of every row."""
    c = full3b
    h, k, v = c.eng.full_prefill(c.tok_dev)
    torch.cuda.synchronize()
    rh, rk, rv = c.full
    errs = {"h": max_rel(f64(h), rh)}
    kk, vv = f64(k), f64(v)
    for l in range(rk.shape[0]):
        errs[f"k[{l}]"] = max_rel(kk[l], rk[l])
        errs[f"v[{l}]"] = max_rel(vv[l], rv[l])
    assert all(e <= 2e-2 for e in errs.values()), errs


@pytest.mark.parametrize("flags", [akvs.AKVS_F_UNIT_WEIGHTS, 0])
def test_3b_unit_constant_caches_reproduce_full_prefill(full3b, flags):
    """Unit caches = the oracle's full-prefill states minus one constant per unit and layer
    (norms 1.5-3, so min(d, 1) = 1 too), rounded to bf16: the library's reuse prefill at
    r = 1/4 with its own probe selection returns the full prefill's query states and every
    layer's keys and values, within the bf16 tolerance."""
    c = full3b
    rh, rk, rv = c.full
    rng = np.random.default_rng(41)
    kc, vc, _, _ = unit_constant_caches(rk, rv, c.lens, c.dims.rope_theta, rng,
                                        lambda l: 1.5 + 0.5 * l, lambda l: 2.0 + 0.5 * l)
    k_all = to_dev(torch.cat([storage_round(x, torch.bfloat16) for x in kc], dim=1))
    v_all = to_dev(torch.cat([storage_round(x, torch.bfloat16) for x in vc], dim=1))
    out = c.gpu(refresh=(1, 4), flags=flags, k_cache=k_all, v_cache=v_all)
    n = int(out["n_rows"][0])
    assert c.q < n < len(c.toks)
    assert torch.all(out["d_k"] > 1.0) and torch.all(out["d_v"] > 1.0)
    ref = {"h_query": rh[-c.q:], "k_corr": rk, "v_corr": rv}
    errs = c.compare(out, ref, rows=False)
    print("3b unit-constant invariant", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.fixture(scope="module")
def full7b():
    c = Case("7b", n_layers=3)
    assert sum(c.lens) + c.q == 8128
    return c


def test_7b_full_sequence_reuse_prefill(full7b):
    c = full7b
    ref = c.oracle()
    own = c.gpu()
    own_selection_is_valid(c, own, ref)
    errs = c.compare(c.gpu(probes=(ref["probe_k"], ref["probe_v"])), ref)
    print("7b full sequence", {k: f"{v:.2e}" for k, v in errs.items()})


@pytest.mark.parametrize("bits", [4, 2])
def test_7b_full_sequence_quantised_cache(full7b, bits):
    """4-bit / 2-bit group-64 unit caches (quantised by the oracle): the oracle runs on the
    same codes (dequantised), the library dequantises inside its kernels."""
    c = full7b
    codes_k, meta_k, deq_k, dt = oracle_quantized(f64(c.k_all), bits)
    codes_v, meta_v, deq_v, _ = oracle_quantized(f64(c.v_all), bits)
    kc = [deq_k[:, s:s + n] for s, n in zip(c.starts, c.lens)]
    vc = [deq_v[:, s:s + n] for s, n in zip(c.starts, c.lens)]
    ref = c.oracle(kc=kc, vc=vc)
    out = c.gpu(probes=(ref["probe_k"], ref["probe_v"]),
                k_cache=to_dev(codes_k), v_cache=to_dev(codes_v),
                k_meta=to_dev(meta_k), v_meta=to_dev(meta_v), cache_dtype=dt)
    errs = c.compare(out, ref)
    print(f"7b full sequence {bits}-bit", {k: f"{v:.2e}" for k, v in errs.items()})


def test_32b_width_reuse_prefill():
    """32B width (D = 5120, 40 / 8 heads, F = 27648, vocab 152064), three layers, ten
    200-token units + the 128-token query (T = 2128), at the 32B workload's refresh ratios."""
    c = Case("32b", n_layers=3, n_units=10)
    for refresh in ((1, 10), (3, 10)):
        ref = c.oracle(refresh=refresh)
        own = c.gpu(refresh=refresh)
        own_selection_is_valid(c, own, ref)
        errs = c.compare(c.gpu(refresh=refresh, probes=(ref["probe_k"], ref["probe_v"])), ref)
        print(f"32b width r={refresh}", {k: f"{v:.2e}" for k, v in errs.items()})
