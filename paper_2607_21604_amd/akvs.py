"""ctypes binding of libakvs (the AgentKVShift reuse-prefill library for MI355X).

Argument marshalling only: tensors are passed as device pointers, descriptors as
ctypes structs, and every computation runs in the library's HIP kernels. Each
function of the C ABI has a wrapper of the same name that raises AkvsError on a
non-zero status. torch provides device memory and the current HIP stream.

Loading fails loudly when the shared library is missing; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libakvs.so")

AKVS_OK, AKVS_EINVAL, AKVS_ESHAPE, AKVS_EDTYPE, AKVS_EUNSUPPORTED, AKVS_ENOSPACE, AKVS_EHIP = range(7)
AKVS_F32, AKVS_BF16, AKVS_U4G64, AKVS_U2G64, AKVS_E4M3G64 = range(5)
AKVS_F_NO_CORRECTION = 1
AKVS_F_UNIT_WEIGHTS = 2
AKVS_F_FRESH_IF_RECOMPUTED = 4
AKVS_F_NO_PREFIX_RECOMPUTE = 8
AKVS_F_GIVEN_PROBES = 16
AKVS_F_PRE_ROPE_OFFSETS = 32
AKVS_NOALLOC_SCRATCH_BYTES = 32 << 20  # scratch array of akvs_decode_step_noalloc (akvs.h)
(AKVS_K_GEMM, AKVS_K_ATTENTION, AKVS_K_CORRECTION, AKVS_K_OFFSET, AKVS_K_DIVERGENCE,
 AKVS_K_SELECT, AKVS_K_NORM, AKVS_K_OTHER, AKVS_K_GEMV) = range(9)
KERNEL_CLASSES = ("gemm", "attention", "correction", "offset", "divergence", "select", "norm",
                  "other")


class AkvsError(RuntimeError):
    def __init__(self, status: int, fn: str, msg: str):
        super().__init__(f"{fn}: status {status}: {msg}")
        self.status = status


class ModelCfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float), ("dtype", ctypes.c_int32)]


class LayerW(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")]


class ReuseCfg(ctypes.Structure):
    _fields_ = [("n_chunks", ctypes.c_int32), ("chunk_len", ctypes.POINTER(ctypes.c_int32)),
                ("query_len", ctypes.c_int32), ("refresh_num", ctypes.c_int32),
                ("refresh_den", ctypes.c_int32), ("check_layer", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("refresh_v_num", ctypes.c_int32),
                ("refresh_v_den", ctypes.c_int32)]


class Cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("k_meta", ctypes.c_void_p),
                ("v_meta", ctypes.c_void_p), ("dtype", ctypes.c_int32)]


class ReuseOut(ctypes.Structure):
    _fields_ = [("h_query", ctypes.c_void_p), ("k_corr", ctypes.c_void_p),
                ("v_corr", ctypes.c_void_p), ("probe_k", ctypes.c_void_p),
                ("probe_v", ctypes.c_void_p), ("d_k", ctypes.c_void_p), ("d_v", ctypes.c_void_p),
                ("rows", ctypes.c_void_p), ("n_rows", ctypes.c_void_p), ("kv_rows", ctypes.c_int32)]


_P = ctypes.c_void_p
_I = ctypes.c_int32
_SIGS = {
    "akvs_version": (_I, []),
    "akvs_status_string": (ctypes.c_char_p, [_I]),
    "akvs_last_error": (ctypes.c_char_p, []),
    "akvs_chunk_meta": (_I, [ctypes.POINTER(ReuseCfg), _P, _P]),
    "akvs_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ModelCfg), ctypes.POINTER(ReuseCfg), _I]),
    "akvs_step_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ModelCfg), _I]),
    "akvs_attention_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ModelCfg), _I, _I]),
    "akvs_rope_table": (_I, [_I, _I, ctypes.c_float, _P, _P]),
    "akvs_rerotate_keys": (_I, [ctypes.POINTER(Cache), _I, _I, _I, _P, _P, _I, _P, _P, _I, _P]),
    "akvs_check_divergence": (_I, [_P, _P, _I, ctypes.POINTER(Cache), _I, _I, _I, _P, _P, _I, _P,
                                   _P, _P]),
    "akvs_select_probes": (_I, [_P, _P, ctypes.POINTER(ReuseCfg), _P, _P, _P, _P, _P, _P, _P, _P,
                                _P, _P, _P]),
    "akvs_probe_qkv": (_I, [_P, _I, _P, ctypes.POINTER(ModelCfg), ctypes.POINTER(LayerW), _P, _I,
                            _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "akvs_chunk_offset": (_I, [_P, _P, _P, ctypes.POINTER(Cache), ctypes.POINTER(ReuseCfg), _P, _P,
                               _P, ctypes.POINTER(ModelCfg), _P, _I, _P, _P, _P]),
    "akvs_apply_correction": (_I, [ctypes.POINTER(Cache), _P, _P, _P, _P, _P, _P, _P, _P,
                                   ctypes.POINTER(ReuseCfg), _P, ctypes.POINTER(ModelCfg), _P, _I,
                                   _P, _P, _P]),
    "akvs_sparse_query_attention": (_I, [_P, _P, _I, _P, _P, _I, ctypes.POINTER(ModelCfg), _P, _P,
                                         ctypes.c_size_t, _P]),
    "akvs_probe_out_mlp": (_I, [_P, _I, _P, ctypes.POINTER(ModelCfg), ctypes.POINTER(LayerW), _P,
                                ctypes.c_size_t, _P]),
    "akvs_quantize_cache": (_I, [_P, _I, _I, _I, _I, _P, _P, _P]),
    "akvs_reuse_prefill": (_I, [_P, _P, ctypes.POINTER(LayerW), _P, ctypes.POINTER(ModelCfg),
                                ctypes.POINTER(ReuseCfg), ctypes.POINTER(Cache),
                                ctypes.POINTER(ReuseOut), _P, ctypes.c_size_t, _P]),
    "akvs_reuse_prefill_batch": (_I, [ctypes.POINTER(ctypes.c_void_p), _I, _P,
                                      ctypes.POINTER(LayerW), _P, ctypes.POINTER(ModelCfg),
                                      ctypes.POINTER(ReuseCfg), ctypes.POINTER(Cache),
                                      ctypes.POINTER(ReuseOut), _P, ctypes.c_size_t, _P]),
    "akvs_batch_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ModelCfg),
                                                    ctypes.POINTER(ReuseCfg), _I]),
    "akvs_full_prefill": (_I, [_P, _I, _I, _P, ctypes.POINTER(LayerW), _P, ctypes.POINTER(ModelCfg),
                               _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "akvs_decode_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(ModelCfg), _I]),
    "akvs_lm_head": (_I, [_P, _I, _P, ctypes.POINTER(ModelCfg), _P, _P, _P, ctypes.c_size_t, _P]),
    "akvs_decode_step": (_I, [_P, _I, _P, ctypes.POINTER(LayerW), _P, _P, ctypes.POINTER(ModelCfg),
                              _P, _P, _I, _P, _P, _P, ctypes.c_size_t, _P]),
    "akvs_decode_step_noalloc": (_I, [_P, _I, _P, ctypes.POINTER(LayerW), _P, _P,
                                      ctypes.POINTER(ModelCfg), _P, _P, _I, _P, _P, _P]),
    "akvs_profile_enable": (_I, [_I]),
    "akvs_profile_read": (_I, [_I, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double)]),
    "akvs_mfma_busy_loop": (_I, [_I, _I, _P, _P]),
}
EXPORTED = tuple(_SIGS)

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libakvs.so (built by paper_2607_21604_amd.build). Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2607_21604_amd.build` "
                          "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, fn: str):
    if status != AKVS_OK:
        raise AkvsError(status, fn, load().akvs_last_error().decode())


def ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    return t.data_ptr()


def stream_handle(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return AKVS_F32
    if t.dtype == torch.bfloat16:
        return AKVS_BF16
    raise ValueError(f"unsupported tensor dtype {t.dtype}")


def model_cfg(shape, dtype: Optional[int] = None, n_layers: Optional[int] = None) -> ModelCfg:
    if dtype is None:
        dtype = AKVS_F32 if shape.dtype == "f32" else AKVS_BF16
    return ModelCfg(shape.n_layers if n_layers is None else n_layers, shape.d_model,
                    shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim, shape.vocab,
                    float(shape.rope_theta), float(shape.rms_eps), dtype)


def layer_array(weights: dict) -> ctypes.Array:
    lays = weights["layers"]
    arr = (LayerW * len(lays))()
    for i, lw in enumerate(lays):
        arr[i] = LayerW(*(ptr(lw[k]) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm",
                                               "w_gate_up", "w_down")))
    return arr


def reuse_cfg(chunk_lens: Sequence[int], query_len: int, refresh=(1, 5), check_layer: int = 1,
              flags: int = 0, refresh_v=None):
    """refresh_v: the value side's own ratio (num, den); None: the key ratio for both."""
    lens = (ctypes.c_int32 * len(chunk_lens))(*[int(n) for n in chunk_lens])
    rv = refresh_v if refresh_v is not None else (0, 0)
    cfg = ReuseCfg(len(chunk_lens), lens, int(query_len), int(refresh[0]), int(refresh[1]),
                   int(check_layer), int(flags), int(rv[0]), int(rv[1]))
    cfg._keep = lens  # the length array must outlive the struct
    return cfg


def cache_struct(k, v, k_meta=None, v_meta=None, dtype: Optional[int] = None) -> Cache:
    """A Cache descriptor; it holds references to its tensors so that they outlive it."""
    if dtype is None:
        dtype = dtype_code(k)
    c = Cache(ptr(k), ptr(v), ptr(k_meta), ptr(v_meta), dtype)
    c._keep = (k, v, k_meta, v_meta)
    return c


# ---- wrappers with the C names -------------------------------------------------------------

def akvs_version() -> int:
    return load().akvs_version()


def akvs_chunk_meta(cfg: ReuseCfg):
    """Returns (meta [2m][4] int32 host tensor: key table then value table,
    totals (T_c, sum b_K, row cap, T, sum b_V))."""
    meta = torch.zeros((2 * cfg.n_chunks, 4), dtype=torch.int32)
    tot = torch.zeros(5, dtype=torch.int32)
    _check(load().akvs_chunk_meta(ctypes.byref(cfg), meta.data_ptr(), tot.data_ptr()),
           "akvs_chunk_meta")
    return meta, tuple(int(x) for x in tot)


def akvs_workspace_size(m: ModelCfg, cfg: Optional[ReuseCfg], n_tokens: int = 0) -> int:
    return load().akvs_workspace_size(ctypes.byref(m), ctypes.byref(cfg) if cfg is not None else None,
                                      int(n_tokens))


def akvs_step_workspace_size(m: ModelCfg, n_rows: int) -> int:
    return load().akvs_step_workspace_size(ctypes.byref(m), int(n_rows))


def akvs_attention_workspace_size(m: ModelCfg, n_rows: int, n_keys: int) -> int:
    return load().akvs_attention_workspace_size(ctypes.byref(m), int(n_rows), int(n_keys))


def akvs_rope_table(n_pos, head_dim, theta, table, stream=None):
    _check(load().akvs_rope_table(n_pos, head_dim, theta, ptr(table), stream_handle(stream)),
           "akvs_rope_table")


def akvs_rerotate_keys(src: Cache, n_tokens, n_kv_heads, head_dim, pos_delta, rope, rope_rows,
                       k_dst, v_dst, dst_dtype, stream=None):
    _check(load().akvs_rerotate_keys(ctypes.byref(src), n_tokens, n_kv_heads, head_dim,
                                     ptr(pos_delta), ptr(rope), rope_rows, ptr(k_dst), ptr(v_dst),
                                     dst_dtype, stream_handle(stream)), "akvs_rerotate_keys")


def akvs_check_divergence(k_fresh, v_fresh, fresh_dtype, cache: Cache, n_tokens, n_kv_heads,
                          head_dim, pos_delta, rope, rope_rows, d_k, d_v, stream=None):
    _check(load().akvs_check_divergence(ptr(k_fresh), ptr(v_fresh), fresh_dtype,
                                        ctypes.byref(cache), n_tokens, n_kv_heads, head_dim,
                                        ptr(pos_delta), ptr(rope), rope_rows, ptr(d_k), ptr(d_v),
                                        stream_handle(stream)), "akvs_check_divergence")


def akvs_select_probes(d_k, d_v, cfg: ReuseCfg, chunk_meta, probe_k, probe_v, w_k, w_v, flags,
                       chunk_rows, rows, n_rows, fresh_row, stream=None):
    _check(load().akvs_select_probes(ptr(d_k), ptr(d_v), ctypes.byref(cfg), ptr(chunk_meta),
                                     ptr(probe_k), ptr(probe_v), ptr(w_k), ptr(w_v), ptr(flags),
                                     ptr(chunk_rows), ptr(rows), ptr(n_rows), ptr(fresh_row),
                                     stream_handle(stream)), "akvs_select_probes")


def akvs_probe_qkv(h, n_rows, positions, m: ModelCfg, lw: LayerW, rope, rope_rows, q, k_fresh,
                   v_fresh, ws, stream=None):
    _check(load().akvs_probe_qkv(ptr(h), n_rows, ptr(positions), ctypes.byref(m), ctypes.byref(lw),
                                 ptr(rope), rope_rows, ptr(q), ptr(k_fresh), ptr(v_fresh), ptr(ws),
                                 ws.numel() * ws.element_size(), stream_handle(stream)),
           "akvs_probe_qkv")


def akvs_chunk_offset(k_fresh, v_fresh, fresh_row, cache: Cache, cfg: ReuseCfg, chunk_meta,
                      probe_k, probe_v, m: ModelCfg, rope, rope_rows, mu_k, mu_v, stream=None):
    _check(load().akvs_chunk_offset(ptr(k_fresh), ptr(v_fresh), ptr(fresh_row), ctypes.byref(cache),
                                    ctypes.byref(cfg), ptr(chunk_meta), ptr(probe_k), ptr(probe_v),
                                    ctypes.byref(m), ptr(rope), rope_rows, ptr(mu_k), ptr(mu_v),
                                    stream_handle(stream)), "akvs_chunk_offset")


def akvs_apply_correction(cache: Cache, mu_k, mu_v, w_k, w_v, flags, k_fresh, v_fresh, fresh_row,
                          cfg: ReuseCfg, chunk_meta, m: ModelCfg, rope, rope_rows, k_corr, v_corr,
                          stream=None):
    _check(load().akvs_apply_correction(ctypes.byref(cache), ptr(mu_k), ptr(mu_v), ptr(w_k),
                                        ptr(w_v), ptr(flags), ptr(k_fresh), ptr(v_fresh),
                                        ptr(fresh_row), ctypes.byref(cfg), ptr(chunk_meta),
                                        ctypes.byref(m), ptr(rope), rope_rows, ptr(k_corr),
                                        ptr(v_corr), stream_handle(stream)), "akvs_apply_correction")


def akvs_sparse_query_attention(q, positions, n_rows, k, v, n_keys, m: ModelCfg, out, ws=None,
                                stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().akvs_sparse_query_attention(ptr(q), ptr(positions), n_rows, ptr(k), ptr(v), n_keys,
                                              ctypes.byref(m), ptr(out), ptr(ws), nbytes,
                                              stream_handle(stream)),
           "akvs_sparse_query_attention")


def akvs_probe_out_mlp(h, n_rows, attn_out, m: ModelCfg, lw: LayerW, ws, stream=None):
    _check(load().akvs_probe_out_mlp(ptr(h), n_rows, ptr(attn_out), ctypes.byref(m), ctypes.byref(lw),
                                     ptr(ws), ws.numel() * ws.element_size(), stream_handle(stream)),
           "akvs_probe_out_mlp")


def akvs_quantize_cache(x, n_rows, head_dim, bits, codes, meta, stream=None):
    _check(load().akvs_quantize_cache(ptr(x), dtype_code(x), n_rows, head_dim, bits, ptr(codes),
                                      ptr(meta), stream_handle(stream)), "akvs_quantize_cache")


def akvs_reuse_prefill(tokens, embed, layers: ctypes.Array, final_norm, m: ModelCfg, cfg: ReuseCfg,
                       cache: Cache, out: ReuseOut, ws, stream=None):
    _check(load().akvs_reuse_prefill(ptr(tokens), ptr(embed), layers, ptr(final_norm),
                                     ctypes.byref(m), ctypes.byref(cfg), ctypes.byref(cache),
                                     ctypes.byref(out), ptr(ws), ws.numel() * ws.element_size(),
                                     stream_handle(stream)), "akvs_reuse_prefill")


def batch_arrays(cfgs, caches, outs):
    """ctypes arrays of per-request descriptors; they keep the descriptors (and what those
    keep alive) referenced."""
    n = len(cfgs)
    ca = (ReuseCfg * n)(*cfgs)
    cc = (Cache * n)(*caches)
    co = (ReuseOut * n)(*outs)
    ca._keep, cc._keep, co._keep = list(cfgs), list(caches), list(outs)
    return ca, cc, co


def akvs_batch_workspace_size(m: ModelCfg, cfgs: ctypes.Array, batch: int) -> int:
    return load().akvs_batch_workspace_size(ctypes.byref(m), cfgs, int(batch))


def akvs_reuse_prefill_batch(tokens, embed, layers: ctypes.Array, final_norm, m: ModelCfg,
                             cfgs: ctypes.Array, caches: ctypes.Array, outs: ctypes.Array, ws,
                             stream=None):
    n = len(tokens)
    tp = (ctypes.c_void_p * n)(*[ptr(t) for t in tokens])
    _check(load().akvs_reuse_prefill_batch(tp, n, ptr(embed), layers, ptr(final_norm),
                                           ctypes.byref(m), cfgs, caches, outs, ptr(ws),
                                           ws.numel() * ws.element_size(), stream_handle(stream)),
           "akvs_reuse_prefill_batch")


def akvs_full_prefill(tokens, n_tokens, pos0, embed, layers: ctypes.Array, final_norm, m: ModelCfg,
                      h_out, k_out, v_out, ws, stream=None):
    _check(load().akvs_full_prefill(ptr(tokens), n_tokens, pos0, ptr(embed), layers, ptr(final_norm),
                                    ctypes.byref(m), ptr(h_out), ptr(k_out), ptr(v_out), ptr(ws),
                                    ws.numel() * ws.element_size(), stream_handle(stream)),
           "akvs_full_prefill")


def akvs_decode_workspace_size(m: ModelCfg, n_past: int) -> int:
    return load().akvs_decode_workspace_size(ctypes.byref(m), int(n_past))


def akvs_lm_head(h, n_rows, w_out, m: ModelCfg, logits, tokens, ws, stream=None):
    _check(load().akvs_lm_head(ptr(h), int(n_rows), ptr(w_out), ctypes.byref(m), ptr(logits),
                               ptr(tokens), ptr(ws), ws.numel() * ws.element_size(),
                               stream_handle(stream)), "akvs_lm_head")


def akvs_decode_step(token, n_past, embed, layers: ctypes.Array, final_norm, w_out, m: ModelCfg,
                     k_cache, v_cache, cache_rows, logits, next_token, ws, stream=None):
    _check(load().akvs_decode_step(ptr(token), int(n_past), ptr(embed), layers, ptr(final_norm),
                                   ptr(w_out), ctypes.byref(m), ptr(k_cache), ptr(v_cache),
                                   int(cache_rows), ptr(logits), ptr(next_token), ptr(ws),
                                   ws.numel() * ws.element_size(), stream_handle(stream)),
           "akvs_decode_step")


def akvs_decode_step_noalloc(token, n_past, embed, layers: ctypes.Array, final_norm, w_out,
                             m: ModelCfg, k_cache, v_cache, cache_rows, logits, next_token,
                             stream=None):
    """akvs_decode_step on the library's own scratch array (no workspace argument)."""
    _check(load().akvs_decode_step_noalloc(ptr(token), int(n_past), ptr(embed), layers,
                                           ptr(final_norm), ptr(w_out), ctypes.byref(m),
                                           ptr(k_cache), ptr(v_cache), int(cache_rows),
                                           ptr(logits), ptr(next_token), stream_handle(stream)),
           "akvs_decode_step_noalloc")


def akvs_profile_enable(class_mask: int):
    """Bit (1 << class) enables event timing of that kernel class; 0 disables."""
    _check(load().akvs_profile_enable(int(class_mask)), "akvs_profile_enable")


def akvs_mfma_busy_loop(n_blocks: int, iters: int, out, stream=None):
    """Counter reference: n_blocks x 256 threads of independent bf16 MFMAs; out fp32 [n_blocks*256]."""
    _check(load().akvs_mfma_busy_loop(int(n_blocks), int(iters), ptr(out), stream_handle(stream)),
           "akvs_mfma_busy_loop")


def akvs_profile_read(kernel_class: int):
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    _check(load().akvs_profile_read(kernel_class, ctypes.byref(n), ctypes.byref(ms)),
           "akvs_profile_read")
    return int(n.value), float(ms.value)
