"""Benchmark of the reuse prefill on one MI355X.

One step = one akvs_reuse_prefill call over the whole 3B-class workload (28-layer
decoder of width 3072, 24/8 heads of 128, FFN 8192; 20 memory units of U{192..256}
tokens + a 64-token query, ~4.5K tokens; refresh 20 %, check layer 1), with token ids,
weights and unit caches already resident in HBM. The unit caches are built beforehand
by the library's own full prefill of each unit at position 0 (not timed).

Prints one JSON line: reuse-prefill tokens/s, the full-prefill baseline on the same
tokens and the speedup, the roofline figure of the dominant kernel (the bf16 MFMA GEMM,
timed with HIP events on its launch stream during the timed eager steps) and the CPU
oracle timed on a bounded sample of the same workload. The headline step time is the
whole call replayed from a HIP graph (every kernel runs; only the host launch overhead
of ~300 launches per step is gone); the eager time is reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16
HBM_PEAK_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="3b")
    p.add_argument("--refresh", default="1/5")
    p.add_argument("--refresh-sweep", default="auto",
                   help="extra refresh ratios timed after the headline one, comma separated; "
                        "a ':select' suffix times the select-only mode (offsets forced to 0) "
                        "('auto': the workload's listed ratios, 'none': skip)")
    p.add_argument("--batch-sweep", default="auto",
                   help="comma-separated batch sizes for the batched reuse prefill leg "
                        "(auto: 4,8,16 for 3b; none elsewhere)")
    p.add_argument("--no-decode", action="store_true", help="skip the decode-step leg")
    p.add_argument("--check-layer", type=int, default=1)
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-full", action="store_true", help="skip the full-prefill baseline leg")
    p.add_argument("--no-graph", action="store_true", help="skip the graph-replay leg")
    p.add_argument("--random-caches", action="store_true",
                   help="unit caches drawn at random instead of prefilled (counter runs)")
    p.add_argument("--calibrate-mfma", action="store_true",
                   help="run the library's MFMA-only loop first (reference for MFMA-busy counters)")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="run one 1 GiB read + 1 GiB write kernel first (FETCH/WRITE counter calibration)")
    p.add_argument("--traffic-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="write the GEMM traffic summary from two rocprofv3 --pmc CSVs and exit")
    return p.parse_args()


GEMM_KERNEL = "k_gemm_bf16"
COPY_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_gemm_bf16_traffic_3b_reuse.txt")
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_21604_amd", "csrc", "k_gemm.hip")


def source_hash(path=GEMM_SOURCE):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_summary(fetch_csv, write_csv):
    """HBM bytes per GEMM launch from rocprofv3 FETCH_SIZE / WRITE_SIZE per-dispatch CSVs,
    each scaled by what the counter reads for the 1 GiB read + 1 GiB write elementwise
    calibration kernel (torch.neg) of the same run."""
    import csv

    def per_kernel(path, counter):
        gemm, copy = [], []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"])
            if GEMM_KERNEL in r["Kernel_Name"]:
                gemm.append(v)
            elif "neg_kernel" in r["Kernel_Name"]:
                copy.append(v)
        return gemm, copy

    fg, fc = per_kernel(fetch_csv, "FETCH_SIZE")
    wg, wc = per_kernel(write_csv, "WRITE_SIZE")
    f_scale = COPY_BYTES / max(fc)   # bytes per counter unit (KiB nominal)
    w_scale = COPY_BYTES / max(wc)
    fetch = sum(fg) / len(fg) * f_scale
    write = sum(wg) / len(wg) * w_scale
    lines = [
        "# k_gemm_bf16 HBM traffic, 3B-class reuse prefill (r=1/5), bench.py counter runs",
        "# commands (from the repository root, on the GPU box):",
        "#   rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/fetch -o run -- python3 bench.py --steps 2 "
        "--warmup 1 --no-cpu-baseline --no-full --no-graph --no-decode --refresh-sweep none "
        "--batch-sweep none --random-caches --calibrate-copy",
        "#   rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/write -o run -- python3 bench.py --steps 2 "
        "--warmup 1 --no-cpu-baseline --no-full --no-graph --no-decode --refresh-sweep none "
        "--batch-sweep none --random-caches --calibrate-copy",
        "#   python3 bench.py --traffic-summary OUT/fetch/run_counter_collection.csv "
        "OUT/write/run_counter_collection.csv",
        f"source_sha256_16: {source_hash()}",
        f"gemm_launches: {len(fg)}",
        f"copy_fetch_counter: {max(fc):.1f}  (for {COPY_BYTES} bytes read)",
        f"copy_write_counter: {max(wc):.1f}  (for {COPY_BYTES} bytes written)",
        f"fetch_bytes_per_launch: {fetch:.0f}",
        f"write_bytes_per_launch: {write:.0f}",
        f"traffic_bytes_per_launch: {fetch + write:.0f}",
    ]
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    open(TRAFFIC_FILE, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def measured_traffic():
    """HBM bytes per GEMM launch from the committed counter summary, or None when the
    summary is missing or was taken on a different GEMM source."""
    try:
        kv = dict(l.split(": ", 1) for l in open(TRAFFIC_FILE).read().splitlines()
                  if ": " in l and not l.startswith("#"))
        if kv.get("source_sha256_16") != source_hash():
            return None
        return float(kv["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def gemm_flops(shape, rows_full, t_ctx, m_rows, c):
    """Algorithmic GEMM flops of one reuse-prefill step.

    Per computed row and layer: 2 * (D*(Hq+2Hkv)*hd + Hq*hd*D + 2F*D + F*D); the prefix
    layers compute every row, the check layer adds the K/V projection of every unit
    token, and the layers from the check layer on compute the M recomputed rows."""
    D, F = shape.d_model, shape.ffn_dim
    hqw = shape.n_q_heads * shape.head_dim
    kvw = shape.n_kv_heads * shape.head_dim
    per_row = 2.0 * (D * (hqw + 2 * kvw) + hqw * D + 2 * F * D + F * D)
    return (c * rows_full * per_row + 2.0 * t_ctx * D * 2 * kvw
            + (shape.n_layers - c) * m_rows * per_row)


def full_gemm_flops(shape, n):
    D, F = shape.d_model, shape.ffn_dim
    hqw = shape.n_q_heads * shape.head_dim
    kvw = shape.n_kv_heads * shape.head_dim
    return shape.n_layers * n * 2.0 * (D * (hqw + 2 * kvw) + hqw * D + 2 * F * D + F * D)


def attention_flops(shape, n, t_ctx, row_pos, c):
    """Causal-effective attention flops of one reuse-prefill step: 4*Hq*hd per (row, key)
    pair with key position <= row position; prefix layers over all n rows, probe layers
    over the recomputed rows, the last layer over the query rows."""
    import numpy as np
    per = 4.0 * shape.n_q_heads * shape.head_dim
    full = n * (n + 1) / 2.0
    probe = float(np.sum(row_pos.astype(np.float64) + 1.0))
    last = float(sum(p + 1 for p in range(t_ctx, n)))
    return per * (c * full + (shape.n_layers - c - 1) * probe + last)


def correction_bytes(shape, n, t_ctx, cache_bits):
    """Algorithmic HBM bytes of one re-rotation + correction launch (one layer): read the
    unit cache K and V once (codes + fp16 scale/zero per 64 elements when quantised),
    write K_corr and V_corr for every position."""
    kvw = shape.n_kv_heads * shape.head_dim
    s_in = 2.0 if cache_bits >= 16 else cache_bits / 8.0 + 4.0 / 64.0
    return 2.0 * t_ctx * kvw * s_in + 2.0 * n * kvw * 2.0


def cpu_baseline(wl, refresh, c, seed, m_rows):
    """The oracle, as it stands, on a bounded sample: one prefix layer over all T rows and
    one layer from the check layer on (M recomputed rows + the unit correction) at the
    full width and length of the workload, scaled to the L-layer step. Inputs are fresh
    seeded draws of the same shapes."""
    import numpy as np
    import oracle
    import synthetic

    shape = wl.shape
    dims = oracle.dims_from(shape.with_layers(1))
    w = synthetic.make_weights(shape, seed=seed, n_layers=1, embed=False)
    lw = oracle.split_layer(w["layers"][0], dims)
    T, tc = wl.n_tokens, wl.n_ctx
    rng = np.random.default_rng(seed + 5)
    h = rng.standard_normal((T, shape.d_model)) * 0.02
    pos = np.arange(T)
    t0 = time.perf_counter()
    oracle.decoder_layer(h, pos, lw, dims)
    t_prefix = time.perf_counter() - t0
    rows = np.sort(np.concatenate([rng.choice(tc, size=m_rows - wl.query_len, replace=False),
                                   np.arange(tc, T)]))
    kc = rng.standard_normal((tc, shape.n_kv_heads, shape.head_dim))
    vc = rng.standard_normal((tc, shape.n_kv_heads, shape.head_dim))
    starts = oracle.chunk_starts(wl.chunk_lens)
    # the layer from the check layer on, repeated until the sample holds about 10 s of work
    reps, t_probe_total = 0, 0.0
    while reps == 0 or (t_prefix + t_probe_total < 10.0 and reps < 8):
        t0 = time.perf_counter()
        q, kf, vf = oracle.model.project_qkv(h[rows], rows, lw, dims)
        k_corr = np.empty((T, shape.n_kv_heads, shape.head_dim))
        v_corr = np.empty_like(k_corr)
        for s, n in zip(starts, wl.chunk_lens):
            reuse = oracle.rerotate(kc[s:s + n], s, shape.rope_theta)
            mu = oracle.probe_offset(kf[:8], reuse[:8])
            k_corr[s:s + n] = oracle.correct_chunk(reuse, reuse, np.zeros(n, bool), np.ones(n), mu)
            v_corr[s:s + n] = oracle.correct_chunk(vc[s:s + n], vc[s:s + n], np.zeros(n, bool),
                                                   np.ones(n), mu)
        k_corr[tc:] = kf[-wl.query_len:]
        v_corr[tc:] = vf[-wl.query_len:]
        o = oracle.attention(q, rows, k_corr, v_corr, pos)
        oracle.model.output_and_mlp(h[rows], o, lw, dims)
        t_probe_total += time.perf_counter() - t0
        reps += 1
    t_probe = t_probe_total / reps
    L = shape.n_layers
    t_step = c * t_prefix + (L - c) * t_probe
    try:
        import threadpoolctl
        threads = max(p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()) or 1
    except Exception:
        threads = os.cpu_count() or 1
    return {"value": T / t_step, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"fp64 NumPy oracle at full width and length (T={T}): one prefix layer "
                       f"({t_prefix:.2f} s) and {reps} run(s) of one probe layer with M={m_rows} "
                       f"rows plus the unit correction ({t_probe:.2f} s each), scaled to "
                       f"{c} + {L - c} layers (extrapolated step {t_step:.1f} s)")}


def main():
    args = parse()
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    import synthetic
    from paper_2607_21604_amd import akvs
    from paper_2607_21604_amd.runtime import Engine

    if not os.path.exists(akvs.LIB_PATH):
        from paper_2607_21604_amd import build
        build.build()
    akvs.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    num, den = (int(x) for x in args.refresh.split("/"))
    wl = synthetic.workload(args.workload, args.seed)
    shape = wl.shape
    print(f"# workload {wl.name}: T={wl.n_tokens} ({len(wl.chunk_lens)} units, q={wl.query_len}), "
          f"L={shape.n_layers}, r={num}/{den}", file=sys.stderr, flush=True)

    if args.calibrate_mfma:
        # two blocks of four waves per CU (two waves per SIMD), MFMAs only
        n_blocks = 2 * torch.cuda.get_device_properties(dev).multi_processor_count
        iters = 4000
        buf = torch.empty(n_blocks * 256, dtype=torch.float32, device=dev)
        akvs.akvs_mfma_busy_loop(n_blocks, 16, buf)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        akvs.akvs_mfma_busy_loop(n_blocks, iters, buf)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        tf = n_blocks * 4 * iters * 8 * 32768.0 / dt * 1e-12
        print(f"# MFMA-only loop: {dt * 1e3:.3f} ms, {tf:.0f} TFLOP/s (wall clock, one launch)",
              file=sys.stderr, flush=True)
        del buf
    if args.calibrate_copy:
        # an elementwise kernel that reads and writes COPY_BYTES once each (a same-dtype
        # copy_ may go to the DMA engines and show no kernel dispatch)
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
    w = synthetic.make_weights(shape, seed=args.seed, device=dev)
    eng = Engine(shape, w, dev)
    toks = torch.tensor(synthetic.make_tokens(wl.n_tokens, shape.vocab, args.seed),
                        dtype=torch.int32, device=dev)
    if args.random_caches:
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed + 3)
        k_cache = torch.randn((shape.n_layers, wl.n_ctx, shape.n_kv_heads, shape.head_dim),
                              generator=g, device=dev).to(torch.bfloat16)
        v_cache = torch.randn(k_cache.shape, generator=g, device=dev).to(torch.bfloat16)
    else:
        k_cache, v_cache = eng.cache_units(toks, wl.chunk_lens)
    qkw = {}
    if wl.cache_bits < 16:
        from paper_2607_21604_amd.runtime import cache_dtype_for_bits, quantize_cache
        kq, km = quantize_cache(k_cache, wl.cache_bits)
        vq, vm = quantize_cache(v_cache, wl.cache_bits)
        del k_cache, v_cache
        k_cache, v_cache = kq, vq
        qkw = {"k_meta": km, "v_meta": vm,
               "cache_dtype": cache_dtype_for_bits(wl.cache_bits)}
    torch.cuda.synchronize()
    print("# unit caches built", file=sys.stderr, flush=True)

    def reuse(outputs=None, refresh=(num, den)):
        return eng.reuse_prefill(toks, wl.chunk_lens, wl.query_len, k_cache, v_cache,
                                 refresh, args.check_layer, 0, outputs=outputs, **qkw)

    out = reuse()
    for _ in range(args.warmup):
        reuse(out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    classes = (akvs.AKVS_K_GEMM, akvs.AKVS_K_ATTENTION, akvs.AKVS_K_CORRECTION)
    for cl in classes:
        akvs.akvs_profile_read(cl)
    akvs.akvs_profile_enable(sum(1 << cl for cl in classes))
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(args.steps):
        reuse(out)
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    akvs.akvs_profile_enable(0)
    ms_step = t0.elapsed_time(t1) / args.steps
    g_launches, g_ms = akvs.akvs_profile_read(akvs.AKVS_K_GEMM)
    a_launches, a_ms = akvs.akvs_profile_read(akvs.AKVS_K_ATTENTION)
    c_launches, c_ms = akvs.akvs_profile_read(akvs.AKVS_K_CORRECTION)
    m_rows = int(out["n_rows"].item())
    row_pos = out["rows"][:m_rows].cpu().numpy()
    print(f"# reuse: {ms_step:.3f} ms/step (wall {1e3 * wall / args.steps:.3f}), M={m_rows}",
          file=sys.stderr, flush=True)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(args.steps):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    # The same calls replayed from HIP graphs (the launch overhead of ~300 kernels per step
    # removed): the headline figures. The eager timings above give the per-kernel events.
    from paper_2607_21604_amd.runtime import ReuseGraph, FullGraph
    ms_graph = None
    if not args.no_graph:
        rg = ReuseGraph(eng, toks, wl.chunk_lens, wl.query_len, k_cache, v_cache, (num, den),
                        args.check_layer, 0, **qkw)
        ms_graph = timed(rg.replay)
        print(f"# reuse (graph replay): {ms_graph:.3f} ms/step", file=sys.stderr, flush=True)
        del rg

    # full-prefill baseline on the same tokens (same kernels)
    ms_full = ms_full_graph = None
    if not args.no_full:
        eng.full_prefill(toks, want_h=True)
        ms_full = timed(lambda: eng.full_prefill(toks, want_h=True))
        print(f"# full prefill: {ms_full:.3f} ms/step", file=sys.stderr, flush=True)
        if not args.no_graph:
            fg = FullGraph(eng, toks)
            ms_full_graph = timed(fg.replay)
            print(f"# full prefill (graph replay): {ms_full_graph:.3f} ms/step", file=sys.stderr,
                  flush=True)
            del fg

    sweep = {}
    extra = args.refresh_sweep
    if extra == "auto":
        extra = {"3b": "1/100,1/20,1/10,3/10,1/2,3/4,1/5:select",
                 "32b": "1/10,3/10"}.get(wl.name, "none")
    full_ref = ms_full_graph or ms_full
    for r in ([] if extra == "none" else extra.split(",")):
        ratio, _, mode = r.partition(":")
        rn, rd = (int(x) for x in ratio.split("/"))
        fl = akvs.AKVS_F_NO_CORRECTION if mode == "select" else 0
        if args.no_graph:
            o2 = eng.reuse_prefill(toks, wl.chunk_lens, wl.query_len, k_cache, v_cache, (rn, rd),
                                   args.check_layer, fl, **qkw)
            ms_r = timed(lambda: eng.reuse_prefill(toks, wl.chunk_lens, wl.query_len, k_cache,
                                                   v_cache, (rn, rd), args.check_layer, fl,
                                                   outputs=o2, **qkw))
        else:
            rg = ReuseGraph(eng, toks, wl.chunk_lens, wl.query_len, k_cache, v_cache, (rn, rd),
                            args.check_layer, fl, **qkw)
            o2 = rg.out
            ms_r = timed(rg.replay)
            del rg
        m_r = int(o2["n_rows"].item())
        sweep[r] = {"tokens_per_s": wl.n_tokens / (ms_r * 1e-3), "ms_per_step": ms_r,
                    "recomputed_rows": m_r,
                    "speedup_vs_full_prefill": full_ref / ms_r if full_ref else None}
        print(f"# reuse at r={r}: {ms_r:.3f} ms/step, M={m_r}", file=sys.stderr, flush=True)
        del o2

    # first decode step over the corrected caches: the next token from the last query row,
    # then one generated token through every layer (weights read once: HBM-bound)
    decode = None
    if not args.no_decode:
        T = wl.n_tokens
        out_d = eng.reuse_prefill(toks, wl.chunk_lens, wl.query_len, k_cache, v_cache, (num, den),
                                  args.check_layer, 0, kv_rows=T + 1, **qkw)
        _, tok0 = eng.lm_head(out_d["h_query"][-1:].contiguous())
        lg_buf = torch.empty(shape.vocab, dtype=torch.float32, device=dev)
        nt_buf = torch.empty(1, dtype=torch.int32, device=dev)

        def dstep():
            eng.decode_step(tok0, T, out_d["k_corr"], out_d["v_corr"], logits=lg_buf,
                            next_token=nt_buf)

        dstep()
        torch.cuda.synchronize()
        ms_dec_eager = timed(dstep)
        ms_dec = None
        if not args.no_graph:
            g_dec = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_dec):
                dstep()
            ms_dec = timed(g_dec.replay)
            del g_dec
        ms_d = ms_dec or ms_dec_eager
        D, F = shape.d_model, shape.ffn_dim
        w_bytes = 2.0 * (shape.n_layers * (shape.qkv_width * D + D * shape.n_q_heads * shape.head_dim
                                           + 3 * F * D) + shape.vocab * D)
        kv_bytes = 2.0 * 2 * shape.n_layers * (T + 1) * shape.kv_width
        decode = {"ms_per_token": ms_d, "ms_per_token_eager": ms_dec_eager,
                  "timing": "HIP-graph replay" if ms_dec else "eager calls",
                  "hbm_bytes_per_token": w_bytes + kv_bytes,
                  "achieved_GBps": (w_bytes + kv_bytes) / (ms_d * 1e-3) / 1e9,
                  "peak_GBps": HBM_PEAK_GBS,
                  "frac": (w_bytes + kv_bytes) / (ms_d * 1e-3) / 1e9 / HBM_PEAK_GBS,
                  "note": "weights of every layer and the tied output embedding read once, plus "
                          "the corrected keys and values of all T tokens"}
        print(f"# decode step over the corrected caches: {ms_d:.3f} ms/token "
              f"({decode['achieved_GBps']:.0f} GB/s)", file=sys.stderr, flush=True)
        del out_d

    # batched reuse prefill: B requests of this workload's shape (same unit lengths, their
    # own token ids and unit caches) in one call, whose projections run over all requests'
    # recomputed rows at once
    batch = {}
    bs = args.batch_sweep
    if bs == "auto":
        bs = {"3b": "4,8,16"}.get(wl.name, "none")
    if bs != "none" and wl.cache_bits == 16 and not args.random_caches:
        from paper_2607_21604_amd.runtime import BatchGraph, reuse_prefill_batch
        sizes = [int(x) for x in bs.split(",")]
        reqs = [{"tokens": toks, "chunk_lens": wl.chunk_lens, "query_len": wl.query_len,
                 "k_cache": k_cache, "v_cache": v_cache}]
        for i in range(1, max(sizes)):
            ti = torch.tensor(synthetic.make_tokens(wl.n_tokens, shape.vocab, args.seed + 100 + i),
                              dtype=torch.int32, device=dev)
            ki, vi = eng.cache_units(ti, wl.chunk_lens)
            reqs.append({"tokens": ti, "chunk_lens": wl.chunk_lens, "query_len": wl.query_len,
                         "k_cache": ki, "v_cache": vi})
        one = ms_graph or ms_step
        for B in sizes:
            if args.no_graph:
                ob = reuse_prefill_batch(eng, reqs[:B], (num, den), args.check_layer, 0)
                ms_b = timed(lambda: reuse_prefill_batch(eng, reqs[:B], (num, den),
                                                         args.check_layer, 0, outputs=ob))
            else:
                bg = BatchGraph(eng, reqs[:B], (num, den), args.check_layer, 0)
                ms_b = timed(bg.replay)
                del bg
            batch[str(B)] = {"tokens_per_s": B * wl.n_tokens / (ms_b * 1e-3), "ms_per_step": ms_b,
                             "throughput_vs_single": B * one / ms_b}
            print(f"# batch of {B}: {ms_b:.3f} ms/step ({B * one / ms_b:.2f}x the one-request "
                  f"rate)", file=sys.stderr, flush=True)
        del reqs

    flops_step = gemm_flops(shape, wl.n_tokens, wl.n_ctx, m_rows, args.check_layer)
    achieved = flops_step * args.steps / (g_ms * 1e-3) / 1e12 if g_ms > 0 else None
    per_launch = flops_step * args.steps / max(g_launches, 1)
    roofline = {"bound": "mfma", "kernel": "k_gemm_bf16",
                "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / MFMA_BF16_PEAK_TFLOPS if achieved else None,
                "traffic": measured_traffic(), "traffic_unit": "HBM bytes per launch",
                "launches": g_launches,
                "avg_launch_us": 1e3 * g_ms / max(g_launches, 1),
                "algorithmic_flops_per_launch": per_launch,
                "gemm_share_of_step": g_ms / args.steps / ms_step}
    # the other two kernels the method is measured on: attention (MFMA) and the fused
    # re-rotation + correction (HBM), each from its own HIP-event class
    attn_f = attention_flops(shape, wl.n_tokens, wl.n_ctx, row_pos, args.check_layer)
    corr_b = correction_bytes(shape, wl.n_tokens, wl.n_ctx, wl.cache_bits) * c_launches / args.steps
    kernels = {
        "k_attn_bf16": {"bound": "mfma", "unit": "TFLOP/s", "peak": MFMA_BF16_PEAK_TFLOPS,
                        "achieved": attn_f * args.steps / (a_ms * 1e-3) / 1e12 if a_ms else None,
                        "launches": a_launches, "avg_launch_us": 1e3 * a_ms / max(a_launches, 1),
                        "note": "causal-effective flops 4*Hq*hd*sum(p+1); time includes the "
                                "key-split merge"},
        "k_correction": {"bound": "hbm", "unit": "GB/s", "peak": HBM_PEAK_GBS,
                         "achieved": corr_b * args.steps / (c_ms * 1e-3) / 1e9 if c_ms else None,
                         "launches": c_launches, "avg_launch_us": 1e3 * c_ms / max(c_launches, 1),
                         "algorithmic_bytes_per_launch": corr_b * args.steps / max(c_launches, 1)},
    }
    for k in kernels.values():
        k["frac"] = k["achieved"] / k["peak"] if k["achieved"] else None
    cpu = None
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, (num, den), args.check_layer, args.seed, m_rows)
    T = wl.n_tokens
    ms_head = ms_graph or ms_step
    full_head = ms_full_graph or ms_full
    line = {
        "metric": "reuse-prefill tokens/s at 20% refresh + speedup vs full prefill, 1 GPU",
        "value": T / (ms_head * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_head,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: uniform token ids, N(0,0.02^2) random-init weights, unit caches "
                "from the library's standalone prefill of each unit",
        "config": {"workload": f"{wl.name}-class reuse prefill: {shape.n_layers} layers, "
                               f"d_model {shape.d_model}, {shape.n_q_heads}/{shape.n_kv_heads} "
                               f"heads x {shape.head_dim}, FFN {shape.ffn_dim}; "
                               f"{len(wl.chunk_lens)} units + {wl.query_len} query tokens",
                   "tokens": T, "context_tokens": wl.n_ctx, "query_tokens": wl.query_len,
                   "refresh": f"{num}/{den}", "check_layer": args.check_layer,
                   "recomputed_rows": m_rows, "recomputed_fraction": m_rows / T},
        "timing": "HIP-graph replay of the whole call" if ms_graph else "eager calls",
        "ms_per_step_eager": ms_step,
        "speedup_vs_full_prefill": full_head / ms_head if full_head else None,
        "full_prefill_tokens_per_s": T / (full_head * 1e-3) if full_head else None,
        "ms_full_prefill": full_head,
        "ms_full_prefill_eager": ms_full,
        "roofline": roofline,
        "kernels": kernels,
        "refresh_sweep": sweep,
        "batch_sweep": batch,
        "decode_step": decode,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
