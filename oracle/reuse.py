"""Oracle for the probe-guided residual correction (Sec. 3.3, Algorithm 1).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The method is an approximation of full recompute, not a faster route to it, so
the oracle runs the procedure itself, in the paper's order:

1. Reused states. Unit i starts at s_i = n_0 + ... + n_{i-1} in the concatenated
   context. Its cached keys were rotated at positions 0..n_i-1, so they are
   re-encoded by a further rotation of s_i (Sec. 2, positional re-encoding);
   values are used as stored (Sec. 3.1, direct reuse).
2. Layers before the check layer are computed for every token (they produce the
   fresh check-layer states that Sec. 3.3 "Probe selection" compares against).
3. Check layer: per-token divergences d_K, d_V (the Sec. 3.3 display equation),
   top-b probe sets per unit with b = ceil(r n) (same paragraph), weights
   w = min(d, 1).
4. For every layer from the check layer on (Algorithm 1 loop): recompute the
   probe and query rows, estimate each unit's offset as the mean fresh-minus-reused
   difference over its probes (Sec. 3.3 "Mean estimation"), correct every
   non-probe token by one weighted vector add (Sec. 3.3 "AgentKVShift correction"),
   then run the recomputed rows' attention over the corrected cache and their MLP.
"""
from __future__ import annotations

import numpy as np

from .model import (ModelDims, _f64, embed, split_layer, project_qkv, attention,
                    output_and_mlp, decoder_layer, rotate, rms_norm)

F_NO_CORRECTION = 1        # offsets forced to 0: probes fresh, the rest as reused
F_UNIT_WEIGHTS = 2         # w = 1 for every token instead of min(d, 1)
F_FRESH_IF_RECOMPUTED = 4  # a token recomputed for either side takes fresh K and V
F_NO_PREFIX_RECOMPUTE = 8  # no check layer at all: stale reuse (needs refresh 0)
F_PRE_ROPE_OFFSETS = 32    # key offsets estimated and applied before the rotary map


def probe_budget(n: int, num: int, den: int) -> int:
    """b = ceil(r n) with r = num/den, in exact integer arithmetic (Sec. 3.3)."""
    if den <= 0 or num < 0 or num > den:
        raise ValueError("refresh ratio must satisfy 0 <= num <= den, den > 0")
    return -((-num * n) // den)


def chunk_starts(lens) -> np.ndarray:
    """Start position of each unit in the concatenated context."""
    lens = np.asarray(lens, dtype=np.int64)
    return np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)


def rerotate(k: np.ndarray, delta: int, theta: float) -> np.ndarray:
    """Rotate every key of k [n][H][hd] further by the offset delta."""
    return rotate(k, np.full(k.shape[0], delta, dtype=np.int64), theta)


def divergence(fresh: np.ndarray, reuse: np.ndarray) -> np.ndarray:
    """Per-token L2 distance over all heads and dims (Sec. 3.3, check-layer divergence)."""
    diff = (fresh - reuse).reshape(fresh.shape[0], -1)
    return np.sqrt(np.sum(diff * diff, axis=1))


def select_top(d, b: int) -> np.ndarray:
    """The b tokens of largest d (equal d: the earlier token first), ascending order."""
    d = np.asarray(d)
    order = sorted(range(len(d)), key=lambda j: (-d[j], j))
    return np.array(sorted(order[:b]), dtype=np.int64)


def correction_weights(d) -> np.ndarray:
    """w_j = min(d_j, 1) (Sec. 3.3)."""
    return np.minimum(np.asarray(d, dtype=np.float64), 1.0)


def probe_offset(fresh_probes: np.ndarray, reuse_probes: np.ndarray) -> np.ndarray:
    """Mean of fresh-minus-reused over the probe rows (Sec. 3.3 "Mean estimation").

    Rows may repeat (sampling with replacement); an empty probe set gives 0.
    """
    if fresh_probes.shape[0] == 0:
        return np.zeros(fresh_probes.shape[1:], dtype=np.float64)
    return np.mean(fresh_probes - reuse_probes, axis=0)


def probe_offset_pre_rope(fresh_probes: np.ndarray, reuse_probes: np.ndarray, positions,
                          theta: float) -> np.ndarray:
    """Key offset taken before the rotary map (the pre-RoPE variant of "Mean estimation",
    Sec. 3.3, whose default form averages the differences after the rotary map): every
    probe's fresh-minus-reused difference is rotated back by its own position, then
    averaged. An empty set gives 0."""
    if fresh_probes.shape[0] == 0:
        return np.zeros(fresh_probes.shape[1:], dtype=np.float64)
    diff = fresh_probes - reuse_probes
    return np.mean(rotate(diff, -np.asarray(positions, dtype=np.int64), theta), axis=0)


def correct_chunk_pre_rope(reuse: np.ndarray, fresh: np.ndarray, is_fresh, w, mu_pre,
                           positions, theta: float) -> np.ndarray:
    """correct_chunk with a pre-RoPE key offset: token t gets reuse_t + w_t Rot(t) mu_pre."""
    n = reuse.shape[0]
    mu_t = rotate(np.broadcast_to(mu_pre, (n,) + mu_pre.shape).copy(),
                  np.asarray(positions, dtype=np.int64), theta)
    is_fresh = np.asarray(is_fresh, dtype=bool)
    w = np.asarray(w, dtype=np.float64)
    shape_w = (-1,) + (1,) * (reuse.ndim - 1)
    corrected = reuse + w.reshape(shape_w) * mu_t
    return np.where(is_fresh.reshape(shape_w), fresh, corrected)


def correct_chunk(reuse: np.ndarray, fresh: np.ndarray, is_fresh, w, mu) -> np.ndarray:
    """Corrected states of one unit (Algorithm 1, inner loop).

    Tokens flagged fresh take their recomputed state; every other token j takes
    reuse_j + w_j * mu. Rows of `fresh` that are not flagged are ignored.
    """
    is_fresh = np.asarray(is_fresh, dtype=bool)
    w = np.asarray(w, dtype=np.float64)
    shape_w = (-1,) + (1,) * (reuse.ndim - 1)
    corrected = reuse + w.reshape(shape_w) * mu[None]
    return np.where(is_fresh.reshape(shape_w), fresh, corrected)


def reuse_prefill(tokens, weights: dict, dims: ModelDims, chunk_lens, query_len: int,
                  k_cache, v_cache, refresh=(1, 5), check_layer: int = 1, flags: int = 0,
                  probes=None, layers=None, refresh_v=None) -> dict:
    """The whole reuse prefill over units U_1..U_m followed by the query.

    k_cache[i], v_cache[i]: unit i's standalone cache [L][n_i][Hkv][hd] (keys rotated at
    positions 0..n_i-1), already dequantised if the cache is quantised.
    refresh: r as an integer pair (num, den). refresh_v: the value side's own ratio
    (asymmetric K/V budgets, the Limitations' K-V asymmetry direction); None: the same
    as the keys. check_layer: 0-based layer index.
    probes: optional (list of K-probe position arrays, list of V-probe position arrays),
    global positions per unit, used instead of the top-b selection.

    Returns h_query (final-normed query rows), k_corr / v_corr [L][T][Hkv][hd],
    d_k / d_v [T_c] (None without a check layer), probe_k / probe_v (global positions,
    per unit), rows (recomputed positions, ascending), w_k / w_v.
    """
    num, den = refresh
    lens = [int(n) for n in chunk_lens]
    if any(n < 1 for n in lens):
        raise ValueError("every unit needs at least one token")
    m = len(lens)
    tc = int(sum(lens))
    t_all = tc + int(query_len)
    starts = chunk_starts(lens)
    L, hkv, hd = dims.n_layers, dims.n_kv_heads, dims.head_dim
    if layers is None:
        layers = [split_layer(lw, dims) for lw in weights["layers"][:L]]
    no_prefix = bool(flags & F_NO_PREFIX_RECOMPUTE)
    num_v, den_v = refresh_v if refresh_v is not None else refresh
    if no_prefix and (num != 0 or num_v != 0):
        raise ValueError("stale reuse (no check layer) is defined for refresh 0 only")
    c = 0 if no_prefix else int(check_layer)
    if not 0 <= c < L:
        raise ValueError("check layer out of range")
    pos = np.arange(t_all)

    # 1. reused states at their new positions
    k_reuse = np.empty((L, tc, hkv, hd))
    v_reuse = np.empty((L, tc, hkv, hd))
    for i in range(m):
        s, n = int(starts[i]), lens[i]
        kc, vc = _f64(k_cache[i]), _f64(v_cache[i])
        for l in range(L):
            k_reuse[l, s:s + n] = rerotate(kc[l], s, dims.rope_theta)
            v_reuse[l, s:s + n] = vc[l]

    k_corr = np.empty((L, t_all, hkv, hd))
    v_corr = np.empty((L, t_all, hkv, hd))

    # 2. layers before the check layer, every token
    h = embed(weights, tokens)
    for l in range(c):
        h, k, v = decoder_layer(h, pos, layers[l], dims)
        k_corr[l] = k
        v_corr[l] = v

    # 3. check layer: divergences, probe sets, weights
    budgets = [probe_budget(n, num, den) for n in lens]
    budgets_v = [probe_budget(n, num_v, den_v) for n in lens]
    if no_prefix:
        d_k = d_v = None
        sk = [np.zeros(0, np.int64) for _ in range(m)]
        sv = [np.zeros(0, np.int64) for _ in range(m)]
        w_k = np.zeros(tc)
        w_v = np.zeros(tc)
    else:
        _, kf, vf = project_qkv(h[:tc], pos[:tc], layers[c], dims)
        d_k = divergence(kf, k_reuse[c])
        d_v = divergence(vf, v_reuse[c])
        if probes is None:
            sk = [select_top(d_k[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets)]
            sv = [select_top(d_v[s:s + n], b) + s for s, n, b in zip(starts, lens, budgets_v)]
        else:
            sk = [np.asarray(p, np.int64) for p in probes[0]]
            sv = [np.asarray(p, np.int64) for p in probes[1]]
            for i in range(m):
                for side, bud in ((sk[i], budgets[i]), (sv[i], budgets_v[i])):
                    s, n = int(starts[i]), lens[i]
                    if (len(side) != bud or len(np.unique(side)) != len(side)
                            or (len(side) and (side.min() < s or side.max() >= s + n))):
                        raise ValueError(f"given probe set of unit {i} is not a valid top-b set")
        if flags & F_UNIT_WEIGHTS:
            w_k = np.ones(tc)
            w_v = np.ones(tc)
        else:
            w_k = correction_weights(d_k)
            w_v = correction_weights(d_v)

    in_k = np.zeros(tc, dtype=bool)
    in_v = np.zeros(tc, dtype=bool)
    for i in range(m):
        in_k[sk[i]] = True
        in_v[sv[i]] = True
    rows = np.concatenate([np.nonzero(in_k | in_v)[0], np.arange(tc, t_all)]).astype(np.int64)
    row_of = np.full(t_all, -1, dtype=np.int64)
    row_of[rows] = np.arange(len(rows))
    fresh_k_mask = in_k | in_v if flags & F_FRESH_IF_RECOMPUTED else in_k
    fresh_v_mask = in_k | in_v if flags & F_FRESH_IF_RECOMPUTED else in_v

    # 4. from the check layer on: recompute rows, offsets, correction, attention, MLP
    hr = h[rows]
    for l in range(c, L):
        q, kf, vf = project_qkv(hr, rows, layers[l], dims)
        k_fresh = np.zeros((t_all, hkv, hd))
        v_fresh = np.zeros((t_all, hkv, hd))
        k_fresh[rows] = kf
        v_fresh[rows] = vf
        for i in range(m):
            s, n = int(starts[i]), lens[i]
            if flags & F_NO_CORRECTION:
                mu_k = np.zeros((hkv, hd))
                mu_v = np.zeros((hkv, hd))
            elif flags & F_PRE_ROPE_OFFSETS:
                mu_k = probe_offset_pre_rope(k_fresh[sk[i]], k_reuse[l][sk[i]], sk[i],
                                             dims.rope_theta)
                mu_v = probe_offset(v_fresh[sv[i]], v_reuse[l][sv[i]])
            else:
                mu_k = probe_offset(k_fresh[sk[i]], k_reuse[l][sk[i]])
                mu_v = probe_offset(v_fresh[sv[i]], v_reuse[l][sv[i]])
            seg = slice(s, s + n)
            if flags & F_PRE_ROPE_OFFSETS and not flags & F_NO_CORRECTION:
                k_corr[l, seg] = correct_chunk_pre_rope(k_reuse[l, seg], k_fresh[seg],
                                                        fresh_k_mask[seg], w_k[seg], mu_k,
                                                        np.arange(s, s + n), dims.rope_theta)
            else:
                k_corr[l, seg] = correct_chunk(k_reuse[l, seg], k_fresh[seg], fresh_k_mask[seg],
                                               w_k[seg], mu_k)
            v_corr[l, seg] = correct_chunk(v_reuse[l, seg], v_fresh[seg], fresh_v_mask[seg],
                                           w_v[seg], mu_v)
        k_corr[l, tc:] = k_fresh[tc:]
        v_corr[l, tc:] = v_fresh[tc:]
        o = attention(q, rows, k_corr[l], v_corr[l], pos)
        hr = output_and_mlp(hr, o, layers[l], dims)

    h_query = rms_norm(hr[len(rows) - int(query_len):], _f64(weights["final_norm"]), dims.rms_eps)
    return {
        "h_query": h_query, "k_corr": k_corr, "v_corr": v_corr,
        "d_k": d_k, "d_v": d_v, "probe_k": sk, "probe_v": sv, "rows": rows,
        "w_k": w_k, "w_v": w_v, "k_reuse": k_reuse, "v_reuse": v_reuse,
        "budgets": budgets, "budgets_v": budgets_v, "starts": starts,
    }
