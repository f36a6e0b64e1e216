"""Whole-procedure parity: the library's full prefill and reuse prefill against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synthetic
from paper_2607_21604_amd import akvs
from paper_2607_21604_amd.runtime import Engine
from tests.gpu_util import (DEV, oracle_quantized, to_dev, dev_weights, f64, max_rel, oracle_caches,
                            check_valid_top_b)
from tests.libutil import ensure_built

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


class Case:
    """A model, a context of units + query, oracle-made unit caches and a GPU engine."""

    def __init__(self, name, n_layers=None, n_units=None, seed=0, lens=None):
        wl = synthetic.workload(name, seed)
        self.shape = wl.shape if n_layers is None else wl.shape.with_layers(n_layers)
        self.lens = list(lens) if lens else list(
            wl.chunk_lens[:n_units] if n_units else wl.chunk_lens)
        self.q = wl.query_len
        self.refresh = wl.refresh[0]
        self.tdt = synthetic.torch_dtype(self.shape)
        self.w = synthetic.make_weights(self.shape, seed)
        self.toks = synthetic.make_tokens(sum(self.lens) + self.q, self.shape.vocab, seed)
        self.dims = oracle.dims_from(self.shape)
        self.layers = [oracle.split_layer(lw, self.dims) for lw in self.w["layers"]]
        self.kc, self.vc, self.k_all, self.v_all = oracle_caches(
            self.toks, self.lens, self.w, self.dims, self.tdt, self.layers)
        self.eng = Engine(self.shape, dev_weights(self.w))
        self.tok_dev = to_dev(self.toks)
        self.starts = oracle.chunk_starts(self.lens)
        self.tol = 1e-4 if self.shape.dtype == "f32" else 2e-2

    def oracle(self, refresh=None, check_layer=1, flags=0, probes=None, kc=None, vc=None,
               refresh_v=None):
        return oracle.reuse_prefill(self.toks, self.w, self.dims, self.lens, self.q,
                                    kc if kc is not None else self.kc,
                                    vc if vc is not None else self.vc,
                                    refresh or self.refresh, check_layer, flags, probes,
                                    self.layers, refresh_v=refresh_v)

    def gpu(self, refresh=None, check_layer=1, flags=0, probes=None, **kw):
        given = None
        if probes is not None:
            given = (to_dev(np.concatenate(probes[0]).astype(np.int32)),
                     to_dev(np.concatenate(probes[1]).astype(np.int32)))
            flags |= akvs.AKVS_F_GIVEN_PROBES
        k = kw.pop("k_cache", self.k_all)
        v = kw.pop("v_cache", self.v_all)
        out = self.eng.reuse_prefill(self.tok_dev, self.lens, self.q, k, v, refresh or self.refresh,
                                     check_layer, flags, given_probes=given, **kw)
        torch.cuda.synchronize()
        return out

    def split(self, flat, budgets):
        off = np.concatenate([[0], np.cumsum(budgets)])
        return [flat[off[i]:off[i + 1]] for i in range(len(budgets))]

    def compare(self, out, ref, tol=None, rows=True):
        """h_query and K_corr / V_corr of every layer, each layer against its own largest
        reference value, within tol; the recomputed rows bit-exact."""
        tol = tol or self.tol
        errs = {"h_query": max_rel(f64(out["h_query"]), ref["h_query"])}
        k, v = f64(out["k_corr"]), f64(out["v_corr"])
        for l in range(ref["k_corr"].shape[0]):
            errs[f"k_corr[{l}]"] = max_rel(k[l, :ref["k_corr"].shape[1]], ref["k_corr"][l])
            errs[f"v_corr[{l}]"] = max_rel(v[l, :ref["v_corr"].shape[1]], ref["v_corr"][l])
        assert all(e <= tol for e in errs.values()), errs
        if rows:
            n = int(out["n_rows"][0])
            np.testing.assert_array_equal(out["rows"][:n].cpu().numpy(), ref["rows"])
        return errs


@pytest.fixture(scope="module")
def tiny():
    return Case("tiny")


def test_tiny_full_prefill(tiny):
    h, k, v = tiny.eng.full_prefill(tiny.tok_dev)
    rh, rk, rv = oracle.full_prefill(tiny.toks, 0, tiny.w, tiny.dims, tiny.layers)
    assert max_rel(f64(h), rh) < 1e-4 and max_rel(f64(k), rk) < 1e-4 and max_rel(f64(v), rv) < 1e-4


def test_tiny_unit_caching_matches_oracle(tiny):
    k, v = tiny.eng.cache_units(tiny.tok_dev, tiny.lens)
    assert max_rel(f64(k), f64(tiny.k_all)) < 1e-5 and max_rel(f64(v), f64(tiny.v_all)) < 1e-5


@pytest.mark.parametrize("check_layer", [1, 0])
def test_tiny_reuse_prefill(tiny, check_layer):
    ref = tiny.oracle(check_layer=check_layer)
    own = tiny.gpu(check_layer=check_layer)
    budgets = ref["budgets"]
    d_k, d_v = f64(own["d_k"]), f64(own["d_v"])
    # divergences agree to within the error of the two states they compare: |d - d'| is
    # at most the distance between the GPU's and the oracle's fresh and reused rows, so
    # the bound scales with the size of the check-layer key and value rows
    c = check_layer
    knorm = np.linalg.norm(f64(tiny.k_all)[c].reshape(sum(tiny.lens), -1), axis=1).max()
    vnorm = np.linalg.norm(f64(tiny.v_all)[c].reshape(sum(tiny.lens), -1), axis=1).max()
    assert np.abs(d_k - ref["d_k"]).max() <= 1e-5 * knorm
    assert np.abs(d_v - ref["d_v"]).max() <= 1e-5 * vnorm
    pk = tiny.split(own["probe_k"].cpu().numpy(), budgets)
    pv = tiny.split(own["probe_v"].cpu().numpy(), budgets)
    check_valid_top_b(ref["d_k"], d_k, pk, tiny.starts, tiny.lens, budgets,
                      2 * np.abs(d_k - ref["d_k"]).max())
    check_valid_top_b(ref["d_v"], d_v, pv, tiny.starts, tiny.lens, budgets,
                      2 * np.abs(d_v - ref["d_v"]).max())
    # with the oracle's probe sets, every float output agrees
    given = tiny.gpu(check_layer=check_layer, probes=(ref["probe_k"], ref["probe_v"]))
    tiny.compare(given, ref)


@pytest.mark.parametrize("flags", [akvs.AKVS_F_NO_CORRECTION, akvs.AKVS_F_UNIT_WEIGHTS,
                                   akvs.AKVS_F_FRESH_IF_RECOMPUTED])
def test_tiny_reuse_flags(tiny, flags):
    ref = tiny.oracle(flags=flags)
    tiny.compare(tiny.gpu(flags=flags, probes=(ref["probe_k"], ref["probe_v"])), ref)


def test_tiny_full_refresh_equals_full_prefill(tiny):
    out = tiny.gpu(refresh=(1, 1))
    rh, rk, rv = oracle.full_prefill(tiny.toks, 0, tiny.w, tiny.dims, tiny.layers)
    assert int(out["n_rows"][0]) == tiny.toks.size
    assert max_rel(f64(out["h_query"]), rh[-tiny.q:]) < 1e-4
    assert max_rel(f64(out["k_corr"]), rk) < 1e-4 and max_rel(f64(out["v_corr"]), rv) < 1e-4


def test_tiny_stale_reuse(tiny):
    flags = akvs.AKVS_F_NO_PREFIX_RECOMPUTE
    ref = tiny.oracle(refresh=(0, 1), flags=flags)
    out = tiny.gpu(refresh=(0, 1), flags=flags)
    tiny.compare(out, ref)
    tc = sum(tiny.lens)
    # values are reused bit for bit
    assert torch.equal(out["v_corr"][:, :tc].cpu(), tiny.v_all.cpu())


def test_tiny_is_deterministic(tiny):
    a = tiny.gpu()
    b = tiny.gpu()
    for k in ("h_query", "k_corr", "v_corr", "d_k", "d_v", "probe_k", "probe_v", "n_rows"):
        assert torch.equal(a[k], b[k]), k
    n = int(a["n_rows"][0])
    assert torch.equal(a["rows"][:n], b["rows"][:n])


@pytest.fixture(scope="module")
def w3b():
    return Case("3b", n_layers=3, n_units=6)


def test_3b_width_reuse_prefill(w3b):
    ref = w3b.oracle()
    own = w3b.gpu()
    budgets = ref["budgets"]
    d_k = f64(own["d_k"])
    assert np.abs(d_k - ref["d_k"]).max() <= 2e-2 * np.abs(ref["d_k"]).max()
    pk = w3b.split(own["probe_k"].cpu().numpy(), budgets)
    check_valid_top_b(ref["d_k"], d_k, pk, w3b.starts, w3b.lens, budgets,
                      2 * np.abs(d_k - ref["d_k"]).max())
    errs = w3b.compare(w3b.gpu(probes=(ref["probe_k"], ref["probe_v"])), ref)
    print("3b-width errors", errs)


def test_3b_width_full_refresh_equals_full_prefill(w3b):
    out = w3b.gpu(refresh=(1, 1))
    h, k, v = w3b.eng.full_prefill(w3b.tok_dev)
    assert max_rel(f64(out["h_query"]), f64(h)[-w3b.q:]) < 2e-2
    assert max_rel(f64(out["k_corr"]), f64(k)) < 2e-2


@pytest.mark.parametrize("flags,refresh_v", [
    (akvs.AKVS_F_PRE_ROPE_OFFSETS, None), (0, (1, 2)), (akvs.AKVS_F_PRE_ROPE_OFFSETS, (0, 1))])
def test_tiny_variants_pre_rope_offsets_and_value_ratio(tiny, flags, refresh_v):
    """The pre-RoPE key offsets and a value ratio of its own, whole procedure against the
    oracle (its probe sets handed over)."""
    ref = tiny.oracle(flags=flags, refresh_v=refresh_v)
    out = tiny.gpu(flags=flags, probes=(ref["probe_k"], ref["probe_v"]), refresh_v=refresh_v)
    tiny.compare(out, ref)


def test_3b_width_pre_rope_offsets(w3b):
    ref = w3b.oracle(flags=akvs.AKVS_F_PRE_ROPE_OFFSETS)
    out = w3b.gpu(flags=akvs.AKVS_F_PRE_ROPE_OFFSETS, probes=(ref["probe_k"], ref["probe_v"]))
    w3b.compare(out, ref)


@pytest.fixture(scope="module")
def long_units():
    # a unit longer than one correction segment (512 tokens): its offsets take their own
    # pass and the correction runs over several segments of the unit
    return Case("tiny", lens=[600, 40, 130])


@pytest.mark.parametrize("flags", [0, akvs.AKVS_F_PRE_ROPE_OFFSETS])
def test_tiny_long_unit_reuse_prefill(long_units, flags):
    ref = long_units.oracle(flags=flags)
    out = long_units.gpu(flags=flags, probes=(ref["probe_k"], ref["probe_v"]))
    long_units.compare(out, ref)


@pytest.mark.parametrize("lens", [[1, 2, 70, 1], [50], [1]])
@pytest.mark.parametrize("refresh", [(1, 5), (0, 1)])
def test_tiny_degenerate_unit_lengths(lens, refresh):
    """Units of one and two tokens (whose budget ceil(r n) covers the whole unit on both
    sides at r = 1/5, and nothing at r = 0), a single unit, and a single one-token unit:
    the whole procedure against the oracle on the oracle's probe sets."""
    c = Case("tiny", lens=lens)
    ref = c.oracle(refresh=refresh)
    given = (ref["probe_k"], ref["probe_v"]) if refresh[0] else None  # r = 0: empty sets
    out = c.gpu(refresh=refresh, probes=given)
    c.compare(out, ref)
