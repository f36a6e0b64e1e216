"""Batched reuse prefill (akvs_reuse_prefill_batch): every request of a batch gives what
the single-request call gives on the same inputs. The single call is itself checked
against the oracle elsewhere; here the batch must reproduce it per request: bit for bit
for the fp32 path, whose kernels compute each row independently of the others; for bf16
the layers before the check layer, the divergences and the selections bit for bit (each
request runs them alone, on buffers sized as its single call would size them), the rest
within the bf16 tolerance, since the combined projections' K-split choice depends on the
combined row count."""
import numpy as np
import pytest
import torch

import oracle
import synthetic
from paper_2607_21604_amd import akvs
from paper_2607_21604_amd.runtime import reuse_prefill_batch
from tests.gpu_util import to_dev, f64, max_rel, oracle_caches
from tests.libutil import ensure_built
from tests.test_gpu_e2e import Case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def make_requests(case, specs):
    """Requests over the case's model: (unit lengths, query length, token seed)."""
    reqs = []
    for lens, q, seed in specs:
        toks = synthetic.make_tokens(sum(lens) + q, case.shape.vocab, seed)
        _, _, k, v = oracle_caches(toks, lens, case.w, case.dims, case.tdt, case.layers)
        reqs.append({"tokens": to_dev(np.asarray(toks, dtype=np.int32)), "chunk_lens": list(lens),
                     "query_len": q, "k_cache": k, "v_cache": v})
    return reqs


def single(case, r, refresh, flags=0):
    out = case.eng.reuse_prefill(r["tokens"], r["chunk_lens"], r["query_len"], r["k_cache"],
                                 r["v_cache"], refresh, 1, flags)
    torch.cuda.synchronize()
    return out


def rows_of(out):
    n = int(out["n_rows"][0])
    return out["rows"][:n], n


@pytest.mark.parametrize("refresh", [(1, 5), (1, 1), (0, 1)])
def test_tiny_batch_matches_single_bitwise(refresh):
    c = Case("tiny")
    reqs = make_requests(c, [([64, 64, 64, 64], 32, 0), ([17, 90, 5], 9, 1),
                             ([200], 1, 2), ([33, 33, 33, 33, 33, 33], 50, 3)])
    outs = reuse_prefill_batch(c.eng, reqs, refresh, 1, 0)
    torch.cuda.synchronize()
    for r, o in zip(reqs, outs):
        s = single(c, r, refresh)
        for k in ("h_query", "k_corr", "v_corr", "d_k", "d_v", "n_rows"):
            assert torch.equal(o[k], s[k]), k
        ro, n = rows_of(o)
        rs, _ = rows_of(s)
        assert torch.equal(ro, rs)
        sb = s["_sum_b"]
        assert torch.equal(o["probe_k"][:sb], s["probe_k"][:sb])


def test_tiny_batch_against_oracle():
    """Each request of a batch against the oracle (fp32 tolerance). The oracle's probe sets
    are handed over: the first unit's cached keys equal its fresh ones, so its divergences
    are rounding noise and its top-b set is not unique."""
    c = Case("tiny")
    reqs = make_requests(c, [([17, 90, 5], 9, 1), ([64, 64], 32, 0)])
    refs = []
    for r in reqs:
        toks = r["tokens"].cpu().numpy()
        kc, vc, _, _ = oracle_caches(toks, r["chunk_lens"], c.w, c.dims, c.tdt, c.layers)
        refs.append(oracle.reuse_prefill(toks, c.w, c.dims, r["chunk_lens"], r["query_len"], kc,
                                         vc, (1, 5), 1, 0, None, c.layers))
    outs = reuse_prefill_batch(c.eng, reqs, (1, 5), 1, 0)
    for o, ref in zip(outs, refs):
        for key in ("probe_k", "probe_v"):
            p = np.concatenate(ref[key]).astype(np.int32)
            o[key][:p.size].copy_(torch.from_numpy(p))
    outs = reuse_prefill_batch(c.eng, reqs, (1, 5), 1, akvs.AKVS_F_GIVEN_PROBES, outputs=outs)
    torch.cuda.synchronize()
    for o, ref in zip(outs, refs):
        assert max_rel(f64(o["h_query"]), ref["h_query"]) < 1e-4
        assert max_rel(f64(o["k_corr"]), ref["k_corr"]) < 1e-4
        assert max_rel(f64(o["v_corr"]), ref["v_corr"]) < 1e-4
        n = int(o["n_rows"][0])
        np.testing.assert_array_equal(o["rows"][:n].cpu().numpy(), ref["rows"])


def test_3b_width_batch_matches_single():
    c = Case("3b", n_layers=3, n_units=4)
    reqs = make_requests(c, [([200, 230, 192, 256], 64, 0), ([250, 199], 64, 5),
                             ([211, 240, 197], 32, 6)])
    outs = reuse_prefill_batch(c.eng, reqs, (1, 5), 1, 0)
    torch.cuda.synchronize()
    for r, o in zip(reqs, outs):
        s = single(c, r, (1, 5))
        for k in ("d_k", "d_v", "n_rows"):
            assert torch.equal(o[k], s[k]), k
        assert torch.equal(o["probe_k"][:s["_sum_b"]], s["probe_k"][:s["_sum_b"]])
        ro, n = rows_of(o)
        rs, _ = rows_of(s)
        assert torch.equal(ro, rs)
        assert torch.equal(o["k_corr"][0], s["k_corr"][0])  # prefix layer
        for k in ("h_query", "k_corr", "v_corr"):
            assert max_rel(f64(o[k]), f64(s[k])) < 1e-2, k
