"""Device-memory plumbing around libakvs: allocate outputs and workspaces with torch,
marshal the descriptors, call the C entry points on the current stream.

Nothing here computes any part of the method; every step runs in the library.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import akvs


class Engine:
    """A decoder (weights on one device) and the calls of the library over it."""

    def __init__(self, shape, weights: dict, device="cuda"):
        self.shape = shape
        self.device = torch.device(device)
        self.weights = weights
        self.n_layers = len(weights["layers"])
        self.m = akvs.model_cfg(shape, n_layers=self.n_layers)
        self.layers = akvs.layer_array(weights)
        self.dtype = torch.float32 if self.m.dtype == akvs.AKVS_F32 else torch.bfloat16
        self._ws = None

    def workspace(self, nbytes: int) -> torch.Tensor:
        """The engine's workspace, grown when a call needs more. A grown workspace replaces
        the old tensor; a captured graph keeps its own reference to the tensor it was
        captured with (see ReuseGraph), so replays never run on freed memory."""
        if self._ws is None or self._ws.numel() < nbytes:
            self._ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        return self._ws

    def full_prefill(self, tokens: torch.Tensor, pos0: int = 0, want_h: bool = True):
        n = int(tokens.numel())
        sh = self.shape
        L = self.n_layers
        k = torch.empty((L, n, sh.n_kv_heads, sh.head_dim), dtype=self.dtype, device=self.device)
        v = torch.empty_like(k)
        h = torch.empty((n, sh.d_model), dtype=torch.float32, device=self.device) if want_h else None
        ws = self.workspace(akvs.akvs_workspace_size(self.m, None, n))
        akvs.akvs_full_prefill(tokens, n, pos0, self.weights["embed"], self.layers,
                               self.weights["final_norm"], self.m, h, k, v, ws)
        return h, k, v

    def lm_head(self, h: torch.Tensor, w_out: Optional[torch.Tensor] = None):
        """Logits [n][vocab] fp32 and greedy tokens [n] of final-normed rows h [n][D]
        (w_out None: tied to the input embedding)."""
        n = int(h.shape[0])
        logits = torch.empty((n, self.shape.vocab), dtype=torch.float32, device=self.device)
        toks = torch.empty(n, dtype=torch.int32, device=self.device)
        ws = self.workspace(akvs.akvs_decode_workspace_size(self.m, 0))
        akvs.akvs_lm_head(h.contiguous(), n, w_out if w_out is not None else self.weights["embed"],
                          self.m, logits, toks, ws)
        return logits, toks

    def decode_step(self, token: torch.Tensor, n_past: int, k_cache: torch.Tensor,
                    v_cache: torch.Tensor, w_out: Optional[torch.Tensor] = None, logits=None,
                    next_token=None):
        """One decode step of `token` (device int32 [1]) at position n_past over caches
        [L][cache_rows][Hkv][hd] (rows < n_past valid; row n_past is written). Returns
        (logits [vocab] fp32, next token [1] int32)."""
        if logits is None:
            logits = torch.empty(self.shape.vocab, dtype=torch.float32, device=self.device)
        if next_token is None:
            next_token = torch.empty(1, dtype=torch.int32, device=self.device)
        ws = self.workspace(akvs.akvs_decode_workspace_size(self.m, n_past))
        akvs.akvs_decode_step(token, n_past, self.weights["embed"], self.layers,
                              self.weights["final_norm"], w_out, self.m, k_cache, v_cache,
                              int(k_cache.shape[1]), logits, next_token, ws)
        return logits, next_token

    def cache_units(self, tokens: torch.Tensor, chunk_lens: Sequence[int]):
        """Standalone per-unit caches: each unit prefilled alone at position 0, laid out
        [L][T_c][Hkv][hd] with the units back to back."""
        sh = self.shape
        tc = int(sum(chunk_lens))
        kc = torch.empty((self.n_layers, tc, sh.n_kv_heads, sh.head_dim), dtype=self.dtype,
                         device=self.device)
        vc = torch.empty_like(kc)
        s = 0
        for n in chunk_lens:
            _, k, v = self.full_prefill(tokens[s:s + n], 0, want_h=False)
            kc[:, s:s + n].copy_(k)
            vc[:, s:s + n].copy_(v)
            s += n
        return kc, vc

    def reuse_prefill(self, tokens: torch.Tensor, chunk_lens: Sequence[int], query_len: int,
                      k_cache: torch.Tensor, v_cache: torch.Tensor, refresh=(1, 5),
                      check_layer: int = 1, flags: int = 0, k_meta=None, v_meta=None,
                      cache_dtype: Optional[int] = None, given_probes=None, outputs=None,
                      kv_rows: int = 0, refresh_v=None):
        """Run the reuse prefill. Returns a dict of device tensors (h_query, k_corr, v_corr,
        probe_k, probe_v, d_k, d_v, rows, n_rows). `outputs` may pass a previous result
        dict to reuse its buffers. kv_rows > T sizes k_corr / v_corr [L][kv_rows][Hkv][hd]
        (rows T.. left for decode steps). refresh_v: the value side's own ratio."""
        sh = self.shape
        cfg = akvs.reuse_cfg(chunk_lens, query_len, refresh, check_layer, flags, refresh_v)
        _, (tc, sum_b, row_cap, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
        if outputs is None:
            dev = self.device
            outputs = {
                "h_query": torch.empty((query_len, sh.d_model), dtype=torch.float32, device=dev),
                "k_corr": torch.empty((self.n_layers, max(kv_rows, t_all), sh.n_kv_heads,
                                       sh.head_dim), dtype=self.dtype, device=dev),
                "probe_k": torch.empty(max(sum_b, 1), dtype=torch.int32, device=dev),
                "probe_v": torch.empty(max(sum_bv, 1), dtype=torch.int32, device=dev),
                "d_k": torch.empty(tc, dtype=torch.float32, device=dev),
                "d_v": torch.empty(tc, dtype=torch.float32, device=dev),
                "rows": torch.empty(t_all, dtype=torch.int32, device=dev),
                "n_rows": torch.empty(1, dtype=torch.int32, device=dev),
            }
            outputs["v_corr"] = torch.empty_like(outputs["k_corr"])
        if given_probes is not None:
            outputs["probe_k"][:sum_b].copy_(given_probes[0])
            outputs["probe_v"][:sum_bv].copy_(given_probes[1])
        o = outputs
        out = akvs.ReuseOut(*(akvs.ptr(o[k]) for k in ("h_query", "k_corr", "v_corr", "probe_k",
                                                       "probe_v", "d_k", "d_v", "rows", "n_rows")),
                            int(o["k_corr"].shape[1]))
        cache = akvs.cache_struct(k_cache, v_cache, k_meta, v_meta,
                                  cache_dtype if cache_dtype is not None else akvs.dtype_code(k_cache))
        ws = self.workspace(akvs.akvs_workspace_size(self.m, cfg))
        akvs.akvs_reuse_prefill(tokens, self.weights["embed"], self.layers,
                                self.weights["final_norm"], self.m, cfg, cache, out, ws)
        outputs["_sum_b"] = sum_b
        outputs["_sum_b_v"] = sum_bv
        return outputs


def _reuse_outputs(engine, query_len, tc, sum_b, t_all, sum_bv=None):
    sh, dev = engine.shape, engine.device
    out = {
        "h_query": torch.empty((query_len, sh.d_model), dtype=torch.float32, device=dev),
        "k_corr": torch.empty((engine.n_layers, t_all, sh.n_kv_heads, sh.head_dim),
                              dtype=engine.dtype, device=dev),
        "probe_k": torch.empty(max(sum_b, 1), dtype=torch.int32, device=dev),
        "probe_v": torch.empty(max(sum_b if sum_bv is None else sum_bv, 1), dtype=torch.int32,
                               device=dev),
        "d_k": torch.empty(tc, dtype=torch.float32, device=dev),
        "d_v": torch.empty(tc, dtype=torch.float32, device=dev),
        "rows": torch.empty(t_all, dtype=torch.int32, device=dev),
        "n_rows": torch.empty(1, dtype=torch.int32, device=dev),
    }
    out["v_corr"] = torch.empty_like(out["k_corr"])
    out["_sum_b"] = sum_b
    out["_sum_b_v"] = sum_b if sum_bv is None else sum_bv
    return out


def reuse_prefill_batch(engine: Engine, requests, refresh=(1, 5), check_layer: int = 1,
                        flags: int = 0, outputs=None):
    """Batched reuse prefill (akvs_reuse_prefill_batch). `requests`: list of dicts with
    tokens, chunk_lens, query_len, k_cache, v_cache (and optional k_meta, v_meta,
    cache_dtype). Returns one output dict per request (as Engine.reuse_prefill);
    `outputs` may pass a previous result list to reuse its buffers."""
    cfgs, caches, outs = [], [], []
    if outputs is None:
        outputs = []
        for r in requests:
            cfg = akvs.reuse_cfg(r["chunk_lens"], r["query_len"], refresh, check_layer, flags)
            _, (tc, sum_b, _, t_all, sum_bv) = akvs.akvs_chunk_meta(cfg)
            outputs.append(_reuse_outputs(engine, r["query_len"], tc, sum_b, t_all, sum_bv))
    for r, o in zip(requests, outputs):
        cfgs.append(akvs.reuse_cfg(r["chunk_lens"], r["query_len"], refresh, check_layer, flags))
        dt = r.get("cache_dtype")
        caches.append(akvs.cache_struct(r["k_cache"], r["v_cache"], r.get("k_meta"), r.get("v_meta"),
                                        dt if dt is not None else akvs.dtype_code(r["k_cache"])))
        outs.append(akvs.ReuseOut(*(akvs.ptr(o[k]) for k in ("h_query", "k_corr", "v_corr",
                                                            "probe_k", "probe_v", "d_k", "d_v",
                                                            "rows", "n_rows"))))
    ca, cc, co = akvs.batch_arrays(cfgs, caches, outs)
    ws = engine.workspace(akvs.akvs_batch_workspace_size(engine.m, ca, len(requests)))
    akvs.akvs_reuse_prefill_batch([r["tokens"] for r in requests], engine.weights["embed"],
                                  engine.layers, engine.weights["final_norm"], engine.m, ca, cc,
                                  co, ws)
    return outputs


def cache_dtype_for_bits(bits: int) -> int:
    """Cache dtype code of a group-64 format: 4 / 2-bit integer or 8-bit FP8 E4M3."""
    return {4: akvs.AKVS_U4G64, 2: akvs.AKVS_U2G64, 8: akvs.AKVS_E4M3G64}[bits]


def quantize_cache(x: torch.Tensor, bits: int):
    """Group-64 quantised copy of a cache [..][hd] (codes uint8, meta fp16 (scale, zero));
    bits 4 / 2: integer codes, 8: FP8 E4M3 codes."""
    hd = x.shape[-1]
    rows = x.numel() // hd
    codes = torch.empty(x.shape[:-1] + (hd * bits // 8,), dtype=torch.uint8, device=x.device)
    meta = torch.empty(x.shape[:-1] + (hd // 64, 2), dtype=torch.float16, device=x.device)
    akvs.akvs_quantize_cache(x.contiguous(), rows, hd, bits, codes, meta)
    return codes, meta


class BatchGraph:
    """One batched reuse-prefill call (reuse_prefill_batch) captured in a HIP graph, as
    ReuseGraph does for a single request: an eager call sizes the workspace and allocates
    the outputs, the capture reruns it on the same buffers, replay() reruns every kernel."""

    def __init__(self, engine: Engine, requests, *args, **kw):
        kw.pop("outputs", None)
        self.out = reuse_prefill_batch(engine, requests, *args, **kw)
        torch.cuda.synchronize(engine.device)
        self.ws = engine._ws  # the captured kernels address this workspace: keep it alive
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            reuse_prefill_batch(engine, requests, *args, outputs=self.out, **kw)
        torch.cuda.synchronize(engine.device)
        assert engine._ws is self.ws

    def replay(self):
        self.graph.replay()
        return self.out


class ReuseGraph:
    """One reuse-prefill call captured in a HIP graph (torch.cuda.CUDAGraph).

    The call is made once eagerly (which sizes the workspace and allocates the outputs),
    then captured; replay() reruns every kernel on the same buffers, so new token ids or
    cache contents are written into the captured tensors in place. The library's calls
    are capture-safe: kernel launches only (host tables travel as kernel arguments), no
    allocation, copy, memset or synchronisation. Kernel timing (akvs_profile_enable) must
    be off while capturing."""

    def __init__(self, engine: Engine, *args, **kw):
        kw.pop("outputs", None)
        self.out = engine.reuse_prefill(*args, **kw)
        torch.cuda.synchronize(engine.device)
        self.ws = engine._ws  # the captured kernels address this workspace: keep it alive
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            engine.reuse_prefill(*args, outputs=self.out, **kw)
        torch.cuda.synchronize(engine.device)
        assert engine._ws is self.ws

    def replay(self):
        self.graph.replay()
        return self.out


class FullGraph:
    """akvs_full_prefill over fixed token buffers captured in a HIP graph (the baseline
    counterpart of ReuseGraph); the outputs live in the graph's memory pool."""

    def __init__(self, engine: Engine, tokens: torch.Tensor, pos0: int = 0, want_h: bool = True):
        engine.full_prefill(tokens, pos0, want_h)  # sizes the workspace
        torch.cuda.synchronize(engine.device)
        self.ws = engine._ws  # the captured kernels address this workspace: keep it alive
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.out = engine.full_prefill(tokens, pos0, want_h)
        torch.cuda.synchronize(engine.device)
        assert engine._ws is self.ws

    def replay(self):
        self.graph.replay()
        return self.out
