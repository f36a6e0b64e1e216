"""The C ABI without a GPU: exported symbols, host-only helpers, argument validation."""
import ctypes
import json
import os
import subprocess

import pytest
import torch

import oracle
from paper_2607_21604_amd import akvs
from tests.libutil import ensure_built, declared_functions

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def lib():
    return ensure_built()


def test_every_declared_function_is_exported(lib):
    names = declared_functions()
    assert len(names) >= 20
    out = subprocess.run(["nm", "-D", "--defined-only", akvs.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    # and the binding wraps exactly the declared set
    assert sorted(akvs.EXPORTED) == names


def test_chunk_meta_matches_budget_table(lib):
    cases = json.load(open(os.path.join(GOLDEN, "probe_budgets.json")))["cases"]
    for c in cases:
        if c["num"] > c["den"]:
            continue
        cfg = akvs.reuse_cfg([c["n"], 3], 2, (c["num"], c["den"]), 1, 0)
        meta, tot = akvs.akvs_chunk_meta(cfg)
        assert int(meta[0, 2]) == c["b"]
        assert int(meta[1, 2]) == oracle.probe_budget(3, c["num"], c["den"])
        assert tot[0] == c["n"] + 3 and tot[3] == c["n"] + 5


def test_chunk_meta_offsets_and_row_cap(lib):
    lens = [5, 1, 17, 64]
    cfg = akvs.reuse_cfg(lens, 9, (3, 10), 1, 0)
    meta, (tc, sum_b, cap, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
    b = [oracle.probe_budget(n, 3, 10) for n in lens]
    starts = oracle.chunk_starts(lens)
    m = len(lens)
    assert [int(x) for x in meta[:m, 0]] == list(starts)
    assert [int(x) for x in meta[:m, 2]] == b
    assert [int(x) for x in meta[:m, 3]] == [0, b[0], b[0] + b[1], b[0] + b[1] + b[2]]
    assert (tc, sum_b, t_all, sum_bv) == (87, sum(b), 96, sum(b))
    assert cap == sum(min(n, 2 * bb) for n, bb in zip(lens, b)) + 9
    assert torch.equal(meta[m:], meta[:m])   # the value table equals the key table


def test_chunk_meta_value_side_ratio(lib):
    """A value ratio of its own: the second table carries its budgets and CSR offsets,
    the row cap counts both sides."""
    lens = [5, 1, 17, 64]
    cfg = akvs.reuse_cfg(lens, 9, (1, 10), 1, 0, refresh_v=(1, 2))
    meta, (tc, sum_b, cap, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
    bk = [oracle.probe_budget(n, 1, 10) for n in lens]
    bv = [oracle.probe_budget(n, 1, 2) for n in lens]
    m = len(lens)
    assert [int(x) for x in meta[:m, 2]] == bk and [int(x) for x in meta[m:, 2]] == bv
    assert [int(x) for x in meta[m:, 3]] == [0, bv[0], bv[0] + bv[1], bv[0] + bv[1] + bv[2]]
    assert [int(x) for x in meta[m:, 0]] == list(oracle.chunk_starts(lens))
    assert (sum_b, sum_bv) == (sum(bk), sum(bv))
    assert cap == sum(min(n, a + c) for n, a, c in zip(lens, bk, bv)) + 9


@pytest.mark.parametrize("bad", [
    dict(n_chunks=0), dict(query_len=0), dict(refresh=(6, 5)), dict(refresh=(1, 0)),
    dict(flags=1 << 7), dict(lens=[4, 0, 3]), dict(flags=akvs.AKVS_F_NO_PREFIX_RECOMPUTE),
    dict(refresh_v=(3, 2)), dict(refresh_v=(-1, 2)),
    dict(refresh=(0, 1), refresh_v=(1, 2), flags=akvs.AKVS_F_NO_PREFIX_RECOMPUTE),
])
def test_invalid_reuse_configs_are_rejected(lib, bad):
    lens = bad.get("lens", [4, 5, 3])
    cfg = akvs.reuse_cfg(lens, bad.get("query_len", 2), bad.get("refresh", (1, 5)), 1,
                         bad.get("flags", 0), bad.get("refresh_v"))
    if "n_chunks" in bad:
        cfg.n_chunks = 0
    with pytest.raises(akvs.AkvsError) as e:
        akvs.akvs_chunk_meta(cfg)
    assert e.value.status == akvs.AKVS_EINVAL


class _Shape:
    def __init__(self, **kw):
        d = dict(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688,
                 vocab=1024, rope_theta=1e4, rms_eps=1e-6, dtype="f32")
        d.update(kw)
        self.__dict__.update(d)


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), akvs.AKVS_EUNSUPPORTED),
    (dict(n_q_heads=6, n_kv_heads=4), akvs.AKVS_ESHAPE),
    (dict(n_layers=0), akvs.AKVS_EINVAL),
    (dict(dtype="bf16", ffn_dim=688), akvs.AKVS_EUNSUPPORTED),
])
def test_invalid_models_are_rejected_before_any_launch(lib, kw, status):
    m = akvs.model_cfg(_Shape(**kw))
    assert akvs.akvs_workspace_size(m, None, 16) == 0
    cfg = akvs.reuse_cfg([4, 4], 2, (1, 5), 1, 0)
    layers = (akvs.LayerW * max(m.n_layers, 1))()
    cache = akvs.Cache(16, 16, None, None, akvs.AKVS_F32)
    out = akvs.ReuseOut(16, 16, 16, None, None, None, None, None, None)
    st = lib.akvs_reuse_prefill(16, 16, layers, 16, ctypes.byref(m), ctypes.byref(cfg),
                                ctypes.byref(cache), ctypes.byref(out), 16, 1 << 20, None)
    assert st == status, lib.akvs_last_error()


def _valid_args():
    m = akvs.model_cfg(_Shape())
    cfg = akvs.reuse_cfg([4, 4], 2, (1, 5), 1, 0)
    layers = (akvs.LayerW * 2)(*[akvs.LayerW(*([4096] * 6)) for _ in range(2)])
    cache = akvs.Cache(4096, 4096, None, None, akvs.AKVS_F32)
    out = akvs.ReuseOut(4096, 4096, 4096, None, None, None, None, None, None)
    return m, cfg, layers, cache, out


def test_workspace_too_small_and_misalignment(lib):
    m, cfg, layers, cache, out = _valid_args()
    need = akvs.akvs_workspace_size(m, cfg)
    assert need > 0
    st = lib.akvs_reuse_prefill(4096, 4096, layers, 4096, ctypes.byref(m), ctypes.byref(cfg),
                                ctypes.byref(cache), ctypes.byref(out), 4096, need - 1, None)
    assert st == akvs.AKVS_ENOSPACE
    assert b"workspace" in lib.akvs_last_error()
    cache.k = 4100  # not 16-byte aligned
    st = lib.akvs_reuse_prefill(4096, 4096, layers, 4096, ctypes.byref(m), ctypes.byref(cfg),
                                ctypes.byref(cache), ctypes.byref(out), 4096, need, None)
    assert st == akvs.AKVS_EINVAL


def test_cache_dtype_must_match_model(lib):
    m, cfg, layers, cache, out = _valid_args()
    cache.dtype = akvs.AKVS_U4G64
    st = lib.akvs_reuse_prefill(4096, 4096, layers, 4096, ctypes.byref(m), ctypes.byref(cfg),
                                ctypes.byref(cache), ctypes.byref(out), 4096, 1 << 30, None)
    assert st == akvs.AKVS_EDTYPE


def test_given_probes_need_probe_buffers(lib):
    m, cfg, layers, cache, out = _valid_args()
    cfg.flags = akvs.AKVS_F_GIVEN_PROBES
    st = lib.akvs_reuse_prefill(4096, 4096, layers, 4096, ctypes.byref(m), ctypes.byref(cfg),
                                ctypes.byref(cache), ctypes.byref(out), 4096, 1 << 30, None)
    assert st == akvs.AKVS_EINVAL


def test_status_strings(lib):
    for s in range(7):
        assert lib.akvs_status_string(s)
    assert lib.akvs_status_string(99) == b"unknown status"


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    monkeypatch.setattr(akvs, "_lib", None)
    with pytest.raises(ImportError):
        akvs.load(str(tmp_path / "nope.so"))


def test_attention_workspace(lib):
    """The key-split workspace of the attention step: sized like the reuse prefill's probe
    layers for a bf16 3B-class head layout, 0 for fp32 models, and a short one refused."""
    m = akvs.ModelCfg(1, 3072, 24, 8, 128, 8192, 16, 1e6, 1e-6, akvs.AKVS_BF16)
    need = akvs.akvs_attention_workspace_size(m, 1400, 4516)
    assert need > 0 and need % 256 == 0
    assert akvs.akvs_attention_workspace_size(m, 50000, 4516) == 0  # enough row tiles: no split
    m32 = akvs.ModelCfg(1, 256, 4, 4, 64, 688, 16, 1e4, 1e-6, akvs.AKVS_F32)
    assert akvs.akvs_attention_workspace_size(m32, 1400, 4516) == 0
    st = lib.akvs_sparse_query_attention(4096, 4096, 1400, 4096, 4096, 4516, ctypes.byref(m), 4096,
                                         4096, need - 256, None)
    assert st == akvs.AKVS_ENOSPACE


def test_batch_workspace_and_validation(lib):
    """Batched reuse prefill: the workspace covers each request's single-call buffers;
    requests that disagree on the check layer, and an empty batch, are refused before any
    device work."""
    m = akvs.ModelCfg(4, 3072, 24, 8, 128, 8192, 16, 1e6, 1e-6, akvs.AKVS_BF16)
    a = akvs.reuse_cfg([300, 280, 256], 64, (1, 5), 1, 0)
    b = akvs.reuse_cfg([512, 100], 32, (1, 5), 1, 0)
    ca, _, _ = akvs.batch_arrays([a, b], [], [])
    both = akvs.akvs_batch_workspace_size(m, ca, 2)
    one = akvs.akvs_batch_workspace_size(m, ca, 1)
    assert both > one > 0
    c = akvs.reuse_cfg([512, 100], 32, (1, 5), 2, 0)
    cm, _, _ = akvs.batch_arrays([a, c], [], [])
    assert akvs.akvs_batch_workspace_size(m, cm, 2) == 0
    tp = (ctypes.c_void_p * 2)(4096, 4096)
    lw = (akvs.LayerW * 4)(*[akvs.LayerW(*([4096] * 6)) for _ in range(4)])
    st = lib.akvs_reuse_prefill_batch(tp, 2, 4096, lw, 4096, ctypes.byref(m), cm, None, None,
                                      4096, 1 << 30, None)
    assert st == akvs.AKVS_EINVAL and b"check layer" in lib.akvs_last_error()
    st = lib.akvs_reuse_prefill_batch(tp, 0, 4096, lw, 4096, ctypes.byref(m), ca, None, None,
                                      4096, 1 << 30, None)
    assert st == akvs.AKVS_EINVAL and b"batch 0" in lib.akvs_last_error()


def test_noalloc_decode_scratch_limit(lib):
    """The no-allocation decode step states its scratch size in the header (the binding
    carries the same number) and rejects, before touching the GPU, a step whose workspace
    would exceed it."""
    import re
    from tests.libutil import HEADER
    text = open(HEADER).read()
    mt = re.search(r"#define AKVS_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert mt and int(mt.group(1)) << int(mt.group(2)) == akvs.AKVS_NOALLOC_SCRATCH_BYTES
    m = akvs.ModelCfg(2, 3072, 24, 8, 128, 8192, 128256, 1e6, 1e-6, akvs.AKVS_BF16)
    assert akvs.akvs_decode_workspace_size(m, 16128) <= akvs.AKVS_NOALLOC_SCRATCH_BYTES
    big = 1 << 22
    assert akvs.akvs_decode_workspace_size(m, big) > akvs.AKVS_NOALLOC_SCRATCH_BYTES
    layers = (akvs.LayerW * 2)()
    st = lib.akvs_decode_step_noalloc(None, big, None, layers, None, None, ctypes.byref(m), None,
                                      None, big + 1, None, None, None)
    assert st == akvs.AKVS_ENOSPACE
    assert "no-allocation entry point holds" in lib.akvs_last_error().decode()
