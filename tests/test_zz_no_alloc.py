"""akvs_decode_step_noalloc (the decode step on the library's own scratch array) against
akvs_decode_step with a caller workspace: identical logits, next token and written cache
rows, on two calls in a row of which the second has the smaller input."""
import ctypes

import numpy as np
import pytest
import torch

import synthetic
from paper_2607_21604_amd import akvs
from paper_2607_21604_amd.runtime import Engine
from tests.libutil import ensure_built

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda")


@pytest.fixture(scope="module", autouse=True)
def lib():
    return ensure_built()


@pytest.fixture(scope="module")
def eng3b():
    shape = synthetic.SHAPES["3b"].with_layers(3)
    return Engine(shape, synthetic.make_weights(shape, seed=3, device=DEV), DEV)


def random_caches(eng, rows, seed):
    sh = eng.shape
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    k = torch.randn((eng.n_layers, rows, sh.n_kv_heads, sh.head_dim), generator=g, device=DEV)
    v = torch.randn(k.shape, generator=g, device=DEV)
    return k.to(eng.dtype), v.to(eng.dtype)


def both_steps(eng, n_past, token, seed):
    """(logits, next token, caches) of the workspace entry point and of the no-allocation one,
    each on its own copy of the same caches."""
    k, v = random_caches(eng, n_past + 1, seed)
    k2, v2 = k.clone(), v.clone()
    tok = torch.tensor([token], dtype=torch.int32, device=DEV)
    lg_a, nt_a = eng.decode_step(tok, n_past, k, v)
    lg_b = torch.full_like(lg_a, float("nan"))
    nt_b = torch.full_like(nt_a, -7)
    akvs.akvs_decode_step_noalloc(tok, n_past, eng.weights["embed"], eng.layers,
                                  eng.weights["final_norm"], None, eng.m, k2, v2, n_past + 1,
                                  lg_b, nt_b)
    torch.cuda.synchronize()
    return (lg_a, nt_a, k, v), (lg_b, nt_b, k2, v2)


def assert_identical(a, b, n_past):
    lg_a, nt_a, k, v = a
    lg_b, nt_b, k2, v2 = b
    assert torch.equal(lg_a, lg_b)
    assert int(nt_a[0]) == int(nt_b[0])
    # the step writes the token's key and value into row n_past of every layer
    assert torch.equal(k[:, n_past], k2[:, n_past]) and torch.equal(v[:, n_past], v2[:, n_past])
    assert torch.equal(k, k2) and torch.equal(v, v2)


def test_noalloc_decode_matches_workspace_entry_point_twice(eng3b):
    """3B width, three layers: first over 4516 past tokens (the 3B workload's corrected
    caches plus the token), then over 300."""
    for n_past, token, seed in ((4516, 1234, 1), (300, 99, 2)):
        a, b = both_steps(eng3b, n_past, token, seed)
        assert_identical(a, b, n_past)


def test_noalloc_decode_tiny_fp32_general_attention():
    """fp32 model (the general attention path and its key-split partials in the scratch)."""
    shape = synthetic.SHAPES["tiny"]
    eng = Engine(shape, synthetic.make_weights(shape, seed=4, device=DEV), DEV)
    for n_past, token, seed in ((287, 5, 3), (31, 17, 4)):
        a, b = both_steps(eng, n_past, token, seed)
        assert_identical(a, b, n_past)


def test_noalloc_decode_rejects_a_step_larger_than_its_scratch(eng3b):
    """A past long enough that the attention partials exceed the scratch: ENOSPACE, and
    nothing is written."""
    n_past = 1 << 22
    need = akvs.akvs_decode_workspace_size(eng3b.m, n_past)
    assert need > akvs.AKVS_NOALLOC_SCRATCH_BYTES
    lg = torch.zeros(eng3b.shape.vocab, dtype=torch.float32, device=DEV)
    nt = torch.zeros(1, dtype=torch.int32, device=DEV)
    tok = torch.zeros(1, dtype=torch.int32, device=DEV)
    kc = torch.zeros(8, dtype=torch.bfloat16, device=DEV)  # never touched: rejected first
    with pytest.raises(akvs.AkvsError, match="no-allocation entry point holds"):
        akvs.akvs_decode_step_noalloc(tok, n_past, eng3b.weights["embed"], eng3b.layers,
                                      eng3b.weights["final_norm"], None, eng3b.m, kc, kc,
                                      n_past + 1, lg, nt)
    torch.cuda.synchronize()
    assert not lg.any() and int(nt[0]) == 0
