"""Helpers of the GPU parity tests: device copies, tolerances, oracle-made caches."""
import numpy as np
import torch

import oracle

DEV = torch.device("cuda")


def to_dev(t, dtype=None):
    if isinstance(t, np.ndarray):
        t = torch.from_numpy(np.ascontiguousarray(t))
    return t.to(device=DEV, dtype=dtype if dtype is not None else t.dtype).contiguous()


def dev_weights(w_cpu):
    return {"embed": to_dev(w_cpu["embed"]), "final_norm": to_dev(w_cpu["final_norm"]),
            "layers": [{k: to_dev(t) for k, t in lw.items()} for lw in w_cpu["layers"]]}


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def max_rel(a, ref):
    """max |a - ref| / max |ref| over the whole tensor."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-30))


def storage_round(x: np.ndarray, torch_dtype) -> torch.Tensor:
    """Round fp64 values to the storage dtype (CPU tensor)."""
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch_dtype)


def oracle_caches(toks, lens, w_cpu, dims, torch_dtype, layers=None):
    """Standalone unit caches from the oracle, rounded to the storage dtype.

    Returns (per-unit CPU tensors k, v lists, concatenated device tensors k, v)."""
    kc, vc = oracle.cache_units(toks, lens, w_cpu, dims, layers)
    kc = [storage_round(k, torch_dtype) for k in kc]
    vc = [storage_round(v, torch_dtype) for v in vc]
    k_all = to_dev(torch.cat(kc, dim=1))
    v_all = to_dev(torch.cat(vc, dim=1))
    return kc, vc, k_all, v_all


def check_valid_top_b(d_ref, d_gpu, probes_gpu, starts, lens, budgets, slack):
    """The GPU's probe set of each unit is a top-b set of its own divergences (ties by
    position), and of the reference divergences up to `slack`."""
    for s, n, b, p in zip(starts, lens, budgets, probes_gpu):
        p = np.asarray(p)
        assert len(p) == b and np.all(np.diff(p) > 0) and (b == 0 or (p[0] >= s and p[-1] < s + n))
        if b == 0 or b == n:
            continue
        inside = np.zeros(n, bool)
        inside[p - s] = True
        dg = np.asarray(d_gpu[s:s + n])
        lo_in = dg[inside].min()
        hi_out = dg[~inside].max()
        assert lo_in >= hi_out
        if lo_in == hi_out:  # ties: the earlier positions are taken
            tied_in = np.nonzero(inside & (dg == lo_in))[0]
            tied_out = np.nonzero(~inside & (dg == lo_in))[0]
            assert tied_in.max() < tied_out.min()
        dr = np.asarray(d_ref[s:s + n])
        assert dr[inside].min() >= dr[~inside].max() - slack


def oracle_quantized(x64, bits):
    """A cache quantised by the oracle: (storage bytes, meta, dequantised values, dtype code)
    for bits 4 / 2 (integer groups) or 8 (FP8 E4M3 groups)."""
    from paper_2607_21604_amd import akvs
    if bits == 8:
        codes, meta = oracle.quantize_e4m3_g64(x64)
        return codes, meta, oracle.dequantize_e4m3_g64(codes, meta), akvs.AKVS_E4M3G64
    codes, meta = oracle.quantize_g64(x64, bits)
    return (oracle.pack_codes(codes, bits), meta, oracle.dequantize_g64(codes, meta),
            akvs.AKVS_U4G64 if bits == 4 else akvs.AKVS_U2G64)
