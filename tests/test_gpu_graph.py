"""The reuse prefill captured in a HIP graph: every replay equals the eager call bit for
bit, with eager work and synchronisations between replays, also after new token ids are
written into the captured input buffer."""
import numpy as np
import pytest
import torch

import synthetic
from paper_2607_21604_amd.runtime import ReuseGraph
from tests.gpu_util import to_dev
from tests.libutil import ensure_built
from tests.test_gpu_e2e import Case

pytestmark = pytest.mark.gpu

KEYS = ("h_query", "k_corr", "v_corr", "d_k", "d_v", "n_rows")


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


def snapshot(out):
    n = int(out["n_rows"][0])
    snap = {k: out[k].clone() for k in KEYS}
    snap["rows"] = out["rows"][:n].clone()
    snap["probe_k"] = out["probe_k"][:out["_sum_b"]].clone()
    snap["probe_v"] = out["probe_v"][:out["_sum_b"]].clone()
    return snap


def assert_same(a, b):
    for k in a:
        assert torch.equal(a[k], b[k]), k


@pytest.mark.parametrize("name,n_layers,n_units", [("tiny", None, None), ("3b", 3, 6)])
def test_graph_replays_match_eager(name, n_layers, n_units):
    c = Case(name, n_layers=n_layers, n_units=n_units)
    args = (c.tok_dev, c.lens, c.q, c.k_all, c.v_all, c.refresh, 1, 0)
    eager = snapshot(c.eng.reuse_prefill(*args))
    g = ReuseGraph(c.eng, *args)
    for i in range(3):
        got = snapshot(g.replay())
        torch.cuda.synchronize()
        assert_same(got, eager)
        # eager work of the program between replays, on other buffers; the full refresh
        # needs a larger workspace, so the engine replaces its workspace tensor while the
        # graph keeps the one it was captured with
        other = c.eng.reuse_prefill(c.tok_dev, c.lens, c.q, c.k_all, c.v_all, (1, 1), 1, 0)
        torch.cuda.synchronize()
        assert int(other["n_rows"][0]) == len(c.toks)
        assert c.eng._ws is not g.ws
        assert c.eng._ws.data_ptr() != g.ws.data_ptr()
        # a replay writes nothing into the eager call's outputs or its workspace's results
        before = snapshot(other)
        again = snapshot(g.replay())
        torch.cuda.synchronize()
        assert_same(snapshot(other), before)
        assert_same(again, eager)


def test_graph_replay_with_new_tokens_in_place():
    c = Case("tiny")
    tok = c.tok_dev.clone()
    g = ReuseGraph(c.eng, tok, c.lens, c.q, c.k_all, c.v_all, c.refresh, 1, 0)
    first = snapshot(g.replay())
    new = synthetic.make_tokens(len(c.toks), c.shape.vocab, 7)
    tok.copy_(to_dev(np.asarray(new, dtype=np.int32)))
    torch.cuda.synchronize()
    got = snapshot(g.replay())
    eager = snapshot(c.eng.reuse_prefill(tok, c.lens, c.q, c.k_all, c.v_all, c.refresh, 1, 0))
    torch.cuda.synchronize()
    assert_same(got, eager)
    assert not torch.equal(got["h_query"], first["h_query"])


def test_batch_graph_replays_match_eager():
    """The batched call captured once: each replay equals the eager batch bit for bit,
    with eager single-request work between replays."""
    from paper_2607_21604_amd.runtime import BatchGraph, reuse_prefill_batch
    from tests.test_gpu_batch import make_requests
    c = Case("3b", n_layers=3, n_units=4)
    reqs = make_requests(c, [([200, 230, 192, 256], 64, 0), ([250, 199], 64, 5)])
    eager = [snapshot(o) for o in reuse_prefill_batch(c.eng, reqs, (1, 5), 1, 0)]
    g = BatchGraph(c.eng, reqs, (1, 5), 1, 0)
    for i in range(3):
        got = [snapshot(o) for o in g.replay()]
        torch.cuda.synchronize()
        for a, b in zip(got, eager):
            assert_same(a, b)
        r = reqs[1]
        other = c.eng.reuse_prefill(r["tokens"], r["chunk_lens"], r["query_len"], r["k_cache"],
                                    r["v_cache"], (1, 1), 1, 0)
        torch.cuda.synchronize()
        assert int(other["n_rows"][0]) == sum(r["chunk_lens"]) + r["query_len"]
        before = snapshot(other)
        again = [snapshot(o) for o in g.replay()]
        torch.cuda.synchronize()
        assert_same(snapshot(other), before)
        for a, b in zip(again, eager):
            assert_same(a, b)
