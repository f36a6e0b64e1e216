"""Benchmark of the reuse prefill on one MI355X.

One step = one akvs_reuse_prefill call over the whole 32B-class workload (64-layer
decoder of width 5120, 40/8 heads of 128, FFN 27648; 80 memory units of 200 tokens + a
128-token query, T = 16128; refresh 20 %, check layer 1), with token ids, weights and
unit caches already resident in HBM. The unit caches are built beforehand by the
library's own full prefill of each unit at position 0 (not timed).

Prints one JSON line: reuse-prefill tokens/s, the full-prefill baseline on the same
tokens and the speedup, the roofline figure of the dominant kernel (the bf16 MFMA GEMM,
timed with HIP events on its launch stream during the timed eager steps) and the CPU
oracle timed on a bounded sample of the same workload. The headline step time is the
whole call replayed from a HIP graph (every kernel runs; only the host launch overhead
of the ~700 launches per step is gone); the eager time is reported beside it. Extra keys
hold the workload's other refresh ratios (1/10, 3/10) and the other workloads (7B-class
at r = 1/5 with bf16, 4-bit and 2-bit unit caches; the 3B-class refresh sweep, batch
sweep and first decode step), each timed the same way with fewer repetitions.
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
    p.add_argument("--workload", default="32b")
    p.add_argument("--refresh", default="1/5")
    p.add_argument("--refresh-sweep", default="auto",
                   help="extra refresh ratios timed after the headline one, comma separated; "
                        "a ':select' suffix times the select-only mode (offsets forced to 0) "
                        "('auto': the workload's listed ratios, 'none': skip)")
    p.add_argument("--batch-sweep", default="auto",
                   help="comma-separated batch sizes for the batched reuse prefill leg "
                        "(auto: 4,8,16 for 3b; none elsewhere)")
    p.add_argument("--no-decode", action="store_true", help="skip the decode-step legs")
    p.add_argument("--extra-workloads", default="auto",
                   help="comma-separated workloads timed after the headline one (auto: "
                        "7b,7b-q4,7b-q2,3b for the 32b headline; none: skip)")
    p.add_argument("--extra-steps", type=int, default=5,
                   help="timed repetitions of every leg other than the headline one")
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
                   help="write the GEMM traffic summary of --workload from two rocprofv3 --pmc "
                        "CSVs and exit")
    p.add_argument("--trace-summary", metavar="KERNEL_TRACE_CSV",
                   help="print per-kernel durations of the reuse calls in a rocprofv3 "
                        "--kernel-trace CSV of this script and exit")
    return p.parse_args()


GEMM_KERNEL = "k_gemm_bf16"
COPY_BYTES = 1 << 30
GEMM_SOURCE = os.path.join(ROOT, "paper_2607_21604_amd", "csrc", "k_gemm.hip")
PROFILE_FLAGS = ("--no-cpu-baseline --no-full --no-graph --no-decode --refresh-sweep none "
                 "--batch-sweep none --extra-workloads none")


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"k_gemm_bf16_traffic_{workload}_reuse.txt")


def source_hash(path=GEMM_SOURCE):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_summary(fetch_csv, write_csv, workload, refresh):
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
    run = (f"python3 bench.py --workload {workload} --refresh {refresh} --steps 2 --warmup 1 "
           f"{PROFILE_FLAGS} --random-caches --calibrate-copy")
    lines = [
        f"# k_gemm_bf16 HBM traffic, {workload}-class reuse prefill (r={refresh}), bench.py "
        "counter runs",
        "# commands (from the repository root):",
        f"#   rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/fetch -o run -- {run}",
        f"#   rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/write -o run -- {run}",
        f"#   python3 bench.py --workload {workload} --refresh {refresh} --traffic-summary "
        "OUT/fetch/run_counter_collection.csv OUT/write/run_counter_collection.csv",
        f"source_sha256_16: {source_hash()}",
        f"gemm_launches: {len(fg)}",
        f"copy_fetch_counter: {max(fc):.1f}  (for {COPY_BYTES} bytes read)",
        f"copy_write_counter: {max(wc):.1f}  (for {COPY_BYTES} bytes written)",
        f"fetch_bytes_per_launch: {fetch:.0f}",
        f"write_bytes_per_launch: {write:.0f}",
        f"traffic_bytes_per_launch: {fetch + write:.0f}",
    ]
    path = traffic_file(workload)
    os.makedirs(os.path.dirname(path), exist_ok=True)
    open(path, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def measured_traffic(workload):
    """HBM bytes per GEMM launch from the committed counter summary of the workload, or
    None when the summary is missing or was taken on a different GEMM source."""
    try:
        kv = dict(l.split(": ", 1) for l in open(traffic_file(workload)).read().splitlines()
                  if ": " in l and not l.startswith("#"))
        if kv.get("source_sha256_16") != source_hash():
            return None
        return float(kv["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


KERNEL_CLASSES = (("k_gemm_bf16", "GEMM (every k_gemm_bf16* kernel, fixup excluded)"),
                  ("k_attn_bf16", "attention (without the split merge)"),
                  ("k_attn_combine", "attention split merge"),
                  ("k_correction", "re-rotation + correction"),
                  ("k_chunk_offset", "per-unit offsets"),
                  ("k_rmsnorm", "RMSNorm"))


def trace_summary(path, n_last):
    """Per-kernel durations of a rocprofv3 --kernel-trace CSV of this script: the reuse
    calls are the dispatch runs that start at a rotary-table dispatch and hold a probe
    selection; one call's table, then each kernel class averaged over the last n_last calls
    (the timed steps of a run with --steps n_last)."""
    import collections
    import csv
    import re
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))

    def short(n):
        return re.sub(r"\(.*\)$", "", n).replace("void ", "")

    def dur(r):
        return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    starts = [i for i, r in enumerate(rows) if "k_rope_table" in r["Kernel_Name"]]
    segs = [rows[a:b] for a, b in zip(starts, starts[1:] + [len(rows)])]
    reuse = [sg for sg in segs if any("k_select_rank" in r["Kernel_Name"] for r in sg)]
    last = reuse[-n_last:]
    seg = last[-1]
    t0 = int(seg[0]["Start_Timestamp"])
    t1 = max(int(r["End_Timestamp"]) for r in seg)
    agg = collections.OrderedDict()
    for r in seg:
        c = agg.setdefault(short(r["Kernel_Name"]), [0, 0.0])
        c[0] += 1
        c[1] += dur(r)
    out = [f"reuse calls in the trace: {len(reuse)}; the table is the last one, the class "
           f"averages are over the last {len(last)}",
           "",
           f"{len(seg)} dispatches, first start to last end {(t1 - t0) / 1e6:.3f} ms, kernel busy "
           f"{sum(v[1] for v in agg.values()) / 1e3:.3f} ms",
           "",
           "| kernel | calls | total us | avg us |",
           "|---|---:|---:|---:|"]
    for k, (n, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| {k} | {n} | {t:.1f} | {t / n:.1f} |")
    out.append("")
    for name, what in KERNEL_CLASSES:
        d = [dur(r) for sg in last for r in sg if name in r["Kernel_Name"]]
        if d:
            out.append(f"{name} ({what}): {len(d)} dispatches over {len(last)} calls, "
                       f"avg {sum(d) / len(d):.2f} us, total per call {sum(d) / len(last):.1f} us")
    print("\n".join(out))


def gemm_flops(shape, rows_full, t_ctx, m_rows, c, query_len):
    """Algorithmic GEMM flops of one reuse-prefill step, counted as the step runs them.

    Per computed row and layer: 2 * (D*(Hq+2Hkv)*hd + Hq*hd*D + 2F*D + F*D). The prefix
    layers compute every row; the check layer adds the K/V projection of every unit token;
    the layers from the check layer on compute the M recomputed rows, except that the last
    layer's output projection and MLP only run on the q query rows (the recomputed unit rows
    of the last layer only supply that layer's fresh keys and values)."""
    D, F = shape.d_model, shape.ffn_dim
    hqw = shape.n_q_heads * shape.head_dim
    kvw = shape.n_kv_heads * shape.head_dim
    qkv = 2.0 * D * (hqw + 2 * kvw)
    rest = 2.0 * (hqw * D + 2 * F * D + F * D)
    L = shape.n_layers
    return (c * rows_full * (qkv + rest) + 2.0 * t_ctx * D * 2 * kvw
            + (L - c - 1) * m_rows * (qkv + rest) + m_rows * qkv + query_len * rest)


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


def cpu_baseline(wl, c, seed, m_rows):
    """The oracle, as it stands, on a bounded sample of the workload: one layer from the
    check layer on at the workload's full width and length (the M recomputed rows' QKV,
    the per-unit offsets and the correction of every unit token, the rows' attention over
    all T keys, their output projection and MLP), timed once. The step is that layer times
    the L - c layers that run it, plus c prefix layers over all T rows, each estimated from
    the same run: its projection/MLP part scaled by T/M rows, its attention part by the
    number of (row, key) pairs the oracle evaluates (T*T against M*T). Inputs are fresh
    seeded draws of the workload's shapes."""
    import numpy as np
    import oracle
    import synthetic

    shape = wl.shape
    dims = oracle.dims_from(shape.with_layers(1))
    w = synthetic.make_weights(shape, seed=seed, n_layers=1, embed=False)
    lw = oracle.split_layer(w["layers"][0], dims)
    del w
    T, tc = wl.n_tokens, wl.n_ctx
    rng = np.random.default_rng(seed + 5)
    rows = np.sort(np.concatenate([rng.choice(tc, size=m_rows - wl.query_len, replace=False),
                                   np.arange(tc, T)]))
    h = rng.standard_normal((m_rows, shape.d_model)) * 0.02
    kc = rng.standard_normal((tc, shape.n_kv_heads, shape.head_dim))
    vc = rng.standard_normal((tc, shape.n_kv_heads, shape.head_dim))
    starts = oracle.chunk_starts(wl.chunk_lens)
    pos = np.arange(T)
    t0 = time.perf_counter()
    q, kf, vf = oracle.model.project_qkv(h, rows, lw, dims)
    t_qkv = time.perf_counter() - t0
    t0 = time.perf_counter()
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
    t_corr = time.perf_counter() - t0
    t0 = time.perf_counter()
    o = oracle.attention(q, rows, k_corr, v_corr, pos)
    t_attn = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.model.output_and_mlp(h, o, lw, dims)
    t_mlp = time.perf_counter() - t0
    t_probe = t_qkv + t_corr + t_attn + t_mlp
    t_prefix = (t_qkv + t_mlp) * T / m_rows + t_attn * T / m_rows
    L = shape.n_layers
    t_step = c * t_prefix + (L - c) * t_probe
    blas = None
    try:
        import threadpoolctl
        blas = max(p.get("num_threads", 1) for p in threadpoolctl.threadpool_info())
    except Exception:
        pass
    host = os.cpu_count() or 1
    return {"value": T / t_step, "unit": "tokens/s", "cores": int(blas or 1), "kind": "oracle",
            "host_cpus": host, "blas_threads": blas,
            "sample": (f"fp64 NumPy oracle, one layer from the check layer on at full width and "
                       f"length (T={T}, M={m_rows} recomputed rows): QKV {t_qkv:.2f} s, offsets "
                       f"+ correction of {tc} unit tokens {t_corr:.2f} s, attention "
                       f"{t_attn:.2f} s, output + MLP {t_mlp:.2f} s; prefix layer estimated "
                       f"from it ({t_prefix:.1f} s: rows x T/M); step = {c} prefix + "
                       f"{L - c} such layers = {t_step:.1f} s (extrapolated)")}


def main():
    args = parse()
    num, den = (int(x) for x in args.refresh.split("/"))
    if args.traffic_summary:
        traffic_summary(*args.traffic_summary, args.workload, args.refresh)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary, args.steps)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "one GPU only: this build measures the reuse prefill on a "
                                   "single MI355X and has no multi-GPU path; run with --gpus 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    from paper_2607_21604_amd import akvs

    if not os.path.exists(akvs.LIB_PATH):
        from paper_2607_21604_amd import build
        build.build()
    akvs.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibrate_mfma:
        calibrate_mfma(dev)
    if args.calibrate_copy:
        # an elementwise kernel that reads and writes COPY_BYTES once each (a same-dtype
        # copy_ may go to the DMA engines and show no kernel dispatch)
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    head = Leg(args, args.workload, dev)
    line = head.headline((num, den))
    extra = args.extra_workloads
    if extra == "auto":
        extra = "7b,7b-q4,7b-q2,3b" if args.workload == "32b" else "none"
    if extra != "none":
        head.free()
        line["workloads"] = {}
        for name in extra.split(","):
            leg = Leg(args, name, dev)
            line["workloads"][name] = leg.extra()
            leg.free()
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(head.wl, args.check_layer, args.seed,
                                            line["config"]["recomputed_rows"])
    print(json.dumps(line))


def calibrate_mfma(dev):
    import torch
    from paper_2607_21604_amd import akvs
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


class Leg:
    """One workload on the GPU: weights, token ids and unit caches resident in HBM, and the
    timed calls over them."""

    def __init__(self, args, name, dev):
        import torch
        import synthetic
        from paper_2607_21604_amd.runtime import Engine
        self.args, self.dev = args, dev
        self.wl = wl = synthetic.workload(name, args.seed)
        self.shape = shape = wl.shape
        print(f"# workload {wl.name}: T={wl.n_tokens} ({len(wl.chunk_lens)} units, "
              f"q={wl.query_len}), L={shape.n_layers}", file=sys.stderr, flush=True)
        self.w = synthetic.make_weights(shape, seed=args.seed, device=dev)
        self.eng = Engine(shape, self.w, dev)
        self.toks = torch.tensor(synthetic.make_tokens(wl.n_tokens, shape.vocab, args.seed),
                                 dtype=torch.int32, device=dev)
        if args.random_caches:
            g = torch.Generator(device=dev)
            g.manual_seed(args.seed + 3)
            self.k_cache = torch.randn((shape.n_layers, wl.n_ctx, shape.n_kv_heads, shape.head_dim),
                                       generator=g, device=dev).to(torch.bfloat16)
            self.v_cache = torch.randn(self.k_cache.shape, generator=g, device=dev).to(torch.bfloat16)
        else:
            self.k_cache, self.v_cache = self.eng.cache_units(self.toks, wl.chunk_lens)
        self.qkw = {}
        if wl.cache_bits < 16:
            from paper_2607_21604_amd.runtime import cache_dtype_for_bits, quantize_cache
            kq, km = quantize_cache(self.k_cache, wl.cache_bits)
            vq, vm = quantize_cache(self.v_cache, wl.cache_bits)
            self.k_cache, self.v_cache = kq, vq
            self.qkw = {"k_meta": km, "v_meta": vm,
                        "cache_dtype": cache_dtype_for_bits(wl.cache_bits)}
        torch.cuda.synchronize()
        print("# unit caches built", file=sys.stderr, flush=True)

    def free(self):
        import torch
        for k in ("eng", "w", "toks", "k_cache", "v_cache", "qkw"):
            if hasattr(self, k):
                delattr(self, k)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()

    def reuse(self, refresh, flags=0, outputs=None, **kw):
        return self.eng.reuse_prefill(self.toks, self.wl.chunk_lens, self.wl.query_len,
                                      self.k_cache, self.v_cache, refresh, self.args.check_layer,
                                      flags, outputs=outputs, **self.qkw, **kw)

    def timed(self, fn, reps, warmup):
        import torch
        stream = torch.cuda.current_stream()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def graph_time(self, refresh, flags, reps, warmup):
        """(ms per replayed call, recomputed rows) of one reuse call captured in a graph."""
        from paper_2607_21604_amd.runtime import ReuseGraph
        rg = ReuseGraph(self.eng, self.toks, self.wl.chunk_lens, self.wl.query_len, self.k_cache,
                        self.v_cache, refresh, self.args.check_layer, flags, **self.qkw)
        ms = self.timed(rg.replay, reps, warmup)
        m = int(rg.out["n_rows"].item())
        del rg
        return ms, m

    def full_time(self, reps, warmup):
        """ms per full prefill of the same tokens (graph replay unless --no-graph)."""
        from paper_2607_21604_amd.runtime import FullGraph
        if self.args.no_graph:
            self.eng.full_prefill(self.toks, want_h=True)
            return self.timed(lambda: self.eng.full_prefill(self.toks, want_h=True), reps, warmup)
        fg = FullGraph(self.eng, self.toks)
        ms = self.timed(fg.replay, reps, warmup)
        del fg
        return ms

    def ratio_legs(self, ratios, full_ms):
        """Each refresh ratio (a ':select' suffix: offsets forced to 0) timed as a graph."""
        from paper_2607_21604_amd import akvs
        a = self.args
        out = {}
        for r in ratios:
            ratio, _, mode = r.partition(":")
            rn, rd = (int(x) for x in ratio.split("/"))
            fl = akvs.AKVS_F_NO_CORRECTION if mode == "select" else 0
            if a.no_graph:
                o = self.reuse((rn, rd), fl)
                ms = self.timed(lambda: self.reuse((rn, rd), fl, outputs=o), a.extra_steps, 1)
                m = int(o["n_rows"].item())
                del o
            else:
                ms, m = self.graph_time((rn, rd), fl, a.extra_steps, 1)
            out[r] = {"tokens_per_s": self.wl.n_tokens / (ms * 1e-3), "ms_per_step": ms,
                      "recomputed_rows": m,
                      "speedup_vs_full_prefill": full_ms / ms if full_ms else None}
            print(f"# {self.wl.name} reuse at r={r}: {ms:.3f} ms/step, M={m}", file=sys.stderr,
                  flush=True)
        return out

    def decode(self, refresh):
        """First decode step over the corrected caches: the next token from the last query
        row, then one generated token through every layer (weights read once: HBM-bound)."""
        import torch
        a, shape, T = self.args, self.shape, self.wl.n_tokens
        out_d = self.reuse(refresh, kv_rows=T + 1)
        _, tok0 = self.eng.lm_head(out_d["h_query"][-1:].contiguous())
        lg_buf = torch.empty(shape.vocab, dtype=torch.float32, device=self.dev)
        nt_buf = torch.empty(1, dtype=torch.int32, device=self.dev)

        def dstep():
            self.eng.decode_step(tok0, T, out_d["k_corr"], out_d["v_corr"], logits=lg_buf,
                                 next_token=nt_buf)

        dstep()
        torch.cuda.synchronize()
        ms_eager = self.timed(dstep, max(a.extra_steps, 5), 1)
        ms_graph = None
        if not a.no_graph:
            g_dec = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_dec):
                dstep()
            ms_graph = self.timed(g_dec.replay, max(a.extra_steps, 5), 1)
            del g_dec
        ms = ms_graph or ms_eager
        D, F = shape.d_model, shape.ffn_dim
        w_bytes = 2.0 * (shape.n_layers * (shape.qkv_width * D + D * shape.n_q_heads * shape.head_dim
                                           + 3 * F * D) + shape.vocab * D)
        kv_bytes = 2.0 * 2 * shape.n_layers * (T + 1) * shape.kv_width
        gbps = (w_bytes + kv_bytes) / (ms * 1e-3) / 1e9
        print(f"# {self.wl.name} decode step over the corrected caches: {ms:.3f} ms/token "
              f"({gbps:.0f} GB/s)", file=sys.stderr, flush=True)
        return {"ms_per_token": ms, "ms_per_token_eager": ms_eager,
                "timing": "HIP-graph replay" if ms_graph else "eager calls",
                "hbm_bytes_per_token": w_bytes + kv_bytes, "achieved_GBps": gbps,
                "peak_GBps": HBM_PEAK_GBS, "frac": gbps / HBM_PEAK_GBS,
                "note": "weights of every layer and the tied output embedding read once, plus "
                        "the corrected keys and values of all T tokens"}

    def batch(self, refresh, sizes):
        """B requests of this workload's shape (same unit lengths, their own token ids and
        unit caches) in one batched call, whose projections run over all requests' rows."""
        import torch
        import synthetic
        from paper_2607_21604_amd.runtime import BatchGraph, reuse_prefill_batch
        a, wl = self.args, self.wl
        reqs = [{"tokens": self.toks, "chunk_lens": wl.chunk_lens, "query_len": wl.query_len,
                 "k_cache": self.k_cache, "v_cache": self.v_cache}]
        for i in range(1, max(sizes)):
            ti = torch.tensor(synthetic.make_tokens(wl.n_tokens, self.shape.vocab, a.seed + 100 + i),
                              dtype=torch.int32, device=self.dev)
            ki, vi = self.eng.cache_units(ti, wl.chunk_lens)
            reqs.append({"tokens": ti, "chunk_lens": wl.chunk_lens, "query_len": wl.query_len,
                         "k_cache": ki, "v_cache": vi})
        one, _ = self.graph_time(refresh, 0, a.extra_steps, 1) if not a.no_graph else (None, 0)
        out = {}
        for B in sizes:
            if a.no_graph:
                ob = reuse_prefill_batch(self.eng, reqs[:B], refresh, a.check_layer, 0)
                ms = self.timed(lambda: reuse_prefill_batch(self.eng, reqs[:B], refresh,
                                                            a.check_layer, 0, outputs=ob),
                                a.extra_steps, 1)
                if B == 1:
                    one = ms
            else:
                bg = BatchGraph(self.eng, reqs[:B], refresh, a.check_layer, 0)
                ms = self.timed(bg.replay, a.extra_steps, 1)
                del bg
            out[str(B)] = {"tokens_per_s": B * wl.n_tokens / (ms * 1e-3), "ms_per_step": ms,
                           "throughput_vs_single": B * one / ms if one else None}
            print(f"# {wl.name} batch of {B}: {ms:.3f} ms/step", file=sys.stderr, flush=True)
        del reqs
        return out

    def extra(self):
        """A workload other than the headline: its listed refresh ratios (graph replay), the
        full prefill, and for the 3B shape the refresh sweep, batch sweep and decode step."""
        a, wl = self.args, self.wl
        full_ms = None if a.no_full else self.full_time(a.extra_steps, 1)
        ratios = [f"{n}/{d}" for n, d in wl.refresh]
        if wl.name == "3b" and a.refresh_sweep == "auto":
            ratios += ["1/100", "1/20", "1/2", "3/4", "1/5:select"]
        res = {"workload": self.describe(), "tokens": wl.n_tokens,
               "full_prefill_ms": full_ms,
               "full_prefill_tokens_per_s": wl.n_tokens / (full_ms * 1e-3) if full_ms else None,
               "refresh": self.ratio_legs(ratios, full_ms)}
        if wl.name == "3b":
            if a.batch_sweep != "none" and not a.random_caches:
                sizes = [4, 8, 16] if a.batch_sweep == "auto" else [int(x) for x in
                                                                    a.batch_sweep.split(",")]
                res["batch_sweep"] = self.batch((1, 5), sizes)
            if not a.no_decode:
                res["decode_step"] = self.decode((1, 5))
        return res

    def describe(self):
        sh, wl = self.shape, self.wl
        bits = {16: "bf16", 4: "4-bit group-64", 2: "2-bit group-64", 8: "FP8-E4M3 group-64"}
        return (f"{wl.name}-class reuse prefill: {sh.n_layers} layers, d_model {sh.d_model}, "
                f"{sh.n_q_heads}/{sh.n_kv_heads} heads x {sh.head_dim}, FFN {sh.ffn_dim}, vocab "
                f"{sh.vocab}; {len(wl.chunk_lens)} units ({min(wl.chunk_lens)}-"
                f"{max(wl.chunk_lens)} tokens) + {wl.query_len} query tokens, T={wl.n_tokens}; "
                f"{bits[wl.cache_bits]} unit caches")

    def headline(self, refresh):
        """The timed steps of the metric: K eager calls with per-kernel HIP events, then the
        same call replayed K times from a HIP graph (the headline time), the full prefill,
        the workload's other refresh ratios and the decode step."""
        import torch
        from paper_2607_21604_amd import akvs
        a, wl, shape = self.args, self.wl, self.shape
        out = self.reuse(refresh)
        for _ in range(a.warmup):
            self.reuse(refresh, outputs=out)
        torch.cuda.synchronize()
        classes = (akvs.AKVS_K_GEMM, akvs.AKVS_K_ATTENTION, akvs.AKVS_K_CORRECTION)
        for cl in classes:
            akvs.akvs_profile_read(cl)
        akvs.akvs_profile_enable(sum(1 << cl for cl in classes))
        stream = torch.cuda.current_stream()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        wall0 = time.perf_counter()
        e0.record(stream)
        for _ in range(a.steps):
            self.reuse(refresh, outputs=out)
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - wall0
        akvs.akvs_profile_enable(0)
        ms_eager = e0.elapsed_time(e1) / a.steps
        g_launches, g_ms = akvs.akvs_profile_read(akvs.AKVS_K_GEMM)
        a_launches, a_ms = akvs.akvs_profile_read(akvs.AKVS_K_ATTENTION)
        c_launches, c_ms = akvs.akvs_profile_read(akvs.AKVS_K_CORRECTION)
        m_rows = int(out["n_rows"].item())
        row_pos = out["rows"][:m_rows].cpu().numpy()
        del out
        print(f"# reuse: {ms_eager:.3f} ms/step eager (wall {1e3 * wall / a.steps:.3f}), "
              f"M={m_rows}", file=sys.stderr, flush=True)
        ms_graph = None
        if not a.no_graph:
            ms_graph, _ = self.graph_time(refresh, 0, a.steps, a.warmup)
            print(f"# reuse (graph replay): {ms_graph:.3f} ms/step", file=sys.stderr, flush=True)
        full_ms = None
        if not a.no_full:
            full_ms = self.full_time(min(a.steps, a.extra_steps), 1)
            print(f"# full prefill: {full_ms:.3f} ms/step", file=sys.stderr, flush=True)
        rs = f"{refresh[0]}/{refresh[1]}"
        sweep = {}
        if a.refresh_sweep != "none":
            ratios = ([f"{n}/{d}" for n, d in wl.refresh] if a.refresh_sweep == "auto"
                      else a.refresh_sweep.split(","))
            sweep = self.ratio_legs([r for r in ratios if r != rs], full_ms)
        decode = None if a.no_decode else self.decode(refresh)

        T = wl.n_tokens
        flops_step = gemm_flops(shape, T, wl.n_ctx, m_rows, a.check_layer, wl.query_len)
        per_launch = flops_step * a.steps / max(g_launches, 1)
        achieved = per_launch / (g_ms / max(g_launches, 1) * 1e-3) / 1e12 if g_ms > 0 else None
        roofline = {"bound": "mfma", "kernel": "k_gemm_bf16",
                    "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / MFMA_BF16_PEAK_TFLOPS if achieved else None,
                    "traffic": measured_traffic(wl.name), "traffic_unit": "HBM bytes per launch",
                    "launches": g_launches,
                    "avg_launch_us": 1e3 * g_ms / max(g_launches, 1),
                    "algorithmic_flops_per_launch": per_launch,
                    "gemm_share_of_step": g_ms / a.steps / ms_eager,
                    "timing": "HIP events around every GEMM launch on its stream, timed eager "
                              "steps"}
        attn_f = attention_flops(shape, T, wl.n_ctx, row_pos, a.check_layer)
        corr_b = correction_bytes(shape, T, wl.n_ctx, wl.cache_bits) * c_launches / a.steps
        kernels = {
            "k_attn_bf16": {"bound": "mfma", "unit": "TFLOP/s", "peak": MFMA_BF16_PEAK_TFLOPS,
                            "achieved": attn_f * a.steps / (a_ms * 1e-3) / 1e12 if a_ms else None,
                            "launches": a_launches,
                            "avg_launch_us": 1e3 * a_ms / max(a_launches, 1),
                            "note": "causal-effective flops 4*Hq*hd*sum(p+1); time includes "
                                    "the key-split merge"},
            "k_correction": {"bound": "hbm", "unit": "GB/s", "peak": HBM_PEAK_GBS,
                             "achieved": corr_b * a.steps / (c_ms * 1e-3) / 1e9 if c_ms else None,
                             "launches": c_launches,
                             "avg_launch_us": 1e3 * c_ms / max(c_launches, 1),
                             "algorithmic_bytes_per_launch":
                                 corr_b * a.steps / max(c_launches, 1)},
        }
        for k in kernels.values():
            k["frac"] = k["achieved"] / k["peak"] if k["achieved"] else None
        ms_head = ms_graph or ms_eager
        return {
            "metric": "reuse-prefill tokens/s at 20% refresh + speedup vs full prefill, 1 GPU",
            "value": T / (ms_head * 1e-3), "unit": "tokens/s", "n_gpus": 1,
            "steps": a.steps, "warmup": a.warmup, "ms_per_step": ms_head,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic: uniform token ids, N(0,0.02^2) random-init weights, unit caches "
                    "from the library's standalone prefill of each unit",
            "config": {"workload": self.describe(), "tokens": T, "context_tokens": wl.n_ctx,
                       "query_tokens": wl.query_len, "refresh": rs,
                       "check_layer": a.check_layer, "recomputed_rows": m_rows,
                       "recomputed_fraction": m_rows / T},
            "timing": "HIP-graph replay of the whole call" if ms_graph else "eager calls",
            "ms_per_step_eager": ms_eager,
            "speedup_vs_full_prefill": full_ms / ms_head if full_ms else None,
            "full_prefill_tokens_per_s": T / (full_ms * 1e-3) if full_ms else None,
            "ms_full_prefill": full_ms,
            "roofline": roofline,
            "kernels": kernels,
            "refresh_sweep": sweep,
            "decode_step": decode,
            "cpu_baseline": None,
        }


if __name__ == "__main__":
    main()
