"""Benchmark of the derived-operator hot path on one MI355X.

One step = one pass of the whole path over one batch of the four measured workloads,
through the public entry points, inputs already resident in HBM:
  derived_conv2d            ResNet conv3x3, N=16, C=K=256, 14x14            (GEMM + OffsetAdd)
  derived_conv_transpose2d  DCGAN convT 4x4 s2, N=16, 512->256, 8x8 -> 16x16 (GEMM + selective add)
  derived_dilated_conv2d    CSRNet dilated conv3x3 d2, C=K=512, 96x128       (GEMM + dilated OffsetAdd)
  banded_bmm                Longformer band, B=96, L=4096, d=64, w=256, dil 2 (fused G2BMM/softmax/GBMM)
Each convolution runs the derived program variant that is faster for it (PATHS below);
both variants are timed and reported.

`value` is the step's algorithmic TFLOP/s (all GEMM-stage and band contractions over
the step time).  Per workload it also reports the GEMM stage in TFLOP/s and % of the
bf16 MFMA peak (and, since its fp32 Y makes it HBM-bound on these shapes, its HBM
GB/s and % of the roofline that binds it; the same stage with a bf16 Y appears warm as
gemm_ybf16_*), the eOperator stage in GB/s and % of the HBM peak, the fused kernel in
TFLOP/s, and for the band also the three stages of its staged form (G2BMM, softmax
eOperator, GBMM) in GB/s and % of the HBM peak, each measured two ways:
  warm     HIP events around a HIP graph of back-to-back launches of that kernel (host
           launch gaps do not count), on the stream it runs on.  Operands and the staged
           scope stay in the 256 MB MALL between such launches, so warm eOperator rates
           are MALL-assisted (named *_mall_assisted), not HBM fractions;
  cold     ("cold" block, the reference figures) the kernel's duration after a 512 MB
           read that evicts L2 and the MALL, from HIP graphs of 20 (flush, kernel),
           (flush, fill) and (flush, fill, fill) sequences (fill: a one-element fill),
           combined so that the flush, the fill and the event overhead cancel.
`roofline` covers the kernel with the largest share of a step (warm; frac_cold from the
cold duration).

`cpu_baseline` times the CPU oracle on a bounded sample of the same workloads.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
       python bench.py --stage NAME [--steps K] [--cold]   (launch one stage kernel K
       times, for profiling; NAME is gemm:<cfg>, eop:<cfg>, op:<cfg>, fused:<cfg> for cfg
       2-4, fusedres:4 (the dilated workload as residue sub-image convolutions),
       band_fused, band_g2bmm, band_softmax, band_gbmm, srcnn_direct_fused,
       srcnn_split3x3, srcnn_split3x3_chain, srcnn_direct_staged (the SRCNN conv5x5
       workload), or copy = a plain 256 MiB device copy; --cold puts a 512 MB read
       before every launch)
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

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E

# derived-program variant per convolution workload: "staged" = GEMM stage + eOperator
# through the Y scope, "fused" = the fused expression (no Y), "residues" = the fused
# expression of the dilated convolution as non-dilated convolutions over its residue
# sub-images (the dilated workload only)
PATHS = {2: "fused", 3: "fused", 4: "fused"}


def traffic_record(kernel_key):
    """HBM bytes per launch of `kernel_key` ("name[workload]") from its rocprofv3 PMC
    record in profiles/, or None when there is none or the kernel source has changed
    since the counters were taken (the record stores the source's sha256)."""
    import hashlib
    kname, wl = kernel_key[:-1].split("[")
    path = os.path.join(ROOT, "profiles", f"{kname}__{wl}__traffic.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line:
            key, val = line.split(":", 1)
            rec[key.strip()] = val.strip().split()[0] if val.strip() else ""
    src = os.path.join(ROOT, rec.get("kernel_source", ""))
    if not os.path.isfile(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    return int(rec["traffic_bytes_per_launch"])


def cold_trace_record():
    """Cold kernel durations (ms) by stage name ("gemm:2", "band_softmax", ...) from the
    rocprofv3 kernel-trace record profiles/cold_stages__all_workloads__kernel_trace.txt,
    for the stages whose kernel source still has the sha256 recorded with it."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "cold_stages__all_workloads__kernel_trace.txt")
    rec = {}
    if not os.path.exists(path):
        return rec
    for line in open(path):
        f = line.split()
        if len(f) < 8 or not f[1].isdigit() or not f[5].startswith("paper_2208_02025_amd/"):
            continue
        src = os.path.join(ROOT, f[5])
        if os.path.isfile(src) and hashlib.sha256(open(src, "rb").read()).hexdigest() == f[6]:
            rec[f[0]] = float(f[2]) * 1e-3
    return rec


def valid_taps_1d(n_in, n_out, r, stride, pad, dil, transposed):
    """Number of (output position, tap) pairs that read a real input position."""
    cnt = 0
    for o in range(n_out):
        for t in range(r):
            if transposed:
                th = o + pad - t * dil
                if th >= 0 and th % stride == 0 and th // stride < n_in:
                    cnt += 1
            else:
                i = o * stride - pad + t * dil
                if 0 <= i < n_in:
                    cnt += 1
    return cnt


def conv_costs(wl, ho, wo, y_bytes=4, out_bytes=4):
    m = wl.n * wl.h * wl.w
    nc = wl.r * wl.s * wl.k
    flops = 2.0 * m * wl.c * nc
    taps = wl.n * valid_taps_1d(wl.h, ho, wl.r, wl.stride[0], wl.pad[0], wl.dil[0], wl.transposed) \
        * valid_taps_1d(wl.w, wo, wl.s, wl.stride[1], wl.pad[1], wl.dil[1], wl.transposed)
    eop_bytes = taps * wl.k * y_bytes + wl.n * ho * wo * wl.k * out_bytes
    return flops, eop_bytes


def srcnn_calls(dev):
    """The SRCNN conv5x5 workload's inputs in HBM and its three derived programs, each
    with preallocated outputs and workspaces: direct fused, split into 3x3 blocks
    (fused 3x3 stage), direct GEMM + OffsetAdd."""
    import torch
    import paper_2208_02025_amd as ol
    import synth
    wl = synth.WORKLOADS[6]
    x, wt = (t.to(dev) for t in synth.conv_inputs(wl))
    desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), wl.stride, wl.pad, 1, 0, x.dtype,
                        torch.float32)
    out = torch.empty((wl.n, wl.h, wl.w, wl.k), dtype=torch.float32, device=dev)

    def ws(flags):
        return torch.empty(max(ol.conv_workspace_bytes(desc, False, flags), 16),
                           dtype=torch.uint8, device=dev)
    ws_split = ws(ol.CONV_SPLIT_3X3 | ol.FUSE_EPILOGUE)
    ws_chain = ws(ol.CONV_SPLIT_3X3)
    ws_staged = ws(0)
    fns = {
        "direct_fused": lambda: ol.derived_conv2d(x, wt, wl.stride, wl.pad, out=out, fuse=True),
        "split3x3": lambda: ol.derived_conv2d(x, wt, wl.stride, wl.pad, out=out, ws=ws_split,
                                              fuse=True, split3x3=True),
        # the split form through the 3x3 stage's GEMM and its two eOperators fused into
        # one kernel (the intermediate Z is never formed)
        "split3x3_chain": lambda: ol.derived_conv2d(x, wt, wl.stride, wl.pad, out=out,
                                                    ws=ws_chain, split3x3=True),
        "direct_staged": lambda: ol.derived_conv2d(x, wt, wl.stride, wl.pad, out=out,
                                                   ws=ws_staged),
    }
    return wl, fns


def band_flops(wl):
    return 2 * 2.0 * wl.b * wl.l * (2 * wl.w + 1) * wl.d


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--stage", default=None, help="launch only this stage kernel")
    ap.add_argument("--cold", action="store_true",
                    help="with --stage: a 512 MB read before every launch (cold caches)")
    ap.add_argument("--streams", type=int, default=1, choices=[1, 2, 4],
                    help="streams the step's independent operators are spread over: 1 = "
                         "all in order on one stream, 2 = the band beside the three "
                         "convolutions, 4 = one stream per operator")
    ap.add_argument("--dilated-path", default=None, choices=["staged", "fused", "residues"],
                    help="derived-program variant of the dilated workload (default: PATHS)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this library has no multi-GPU path "
              "(batch/head sharding needs no communication; see the design notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2208_02025_amd as ol
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    # ---------------------------------------------------------------- inputs in HBM
    conv_ops = []
    for cfg, entry in ((2, ol.derived_conv2d), (3, ol.derived_conv_transpose2d),
                       (4, ol.derived_dilated_conv2d)):
        wl = synth.WORKLOADS[cfg]
        x, wt = synth.conv_inputs(wl)
        x, wt = x.to(dev), wt.to(dev)
        desc = ol.conv_desc(tuple(x.shape), tuple(wt.shape), wl.stride, wl.pad, wl.dil,
                            wl.out_pad, x.dtype, torch.float32)
        ho, wo = ol.conv_out_hw(desc, wl.transposed)
        out = torch.empty((wl.n, ho, wo, wl.k), dtype=torch.float32, device=dev)
        ws = torch.empty(ol.conv_workspace_bytes(desc, wl.transposed), dtype=torch.uint8,
                         device=dev)
        kw = dict(stride=wl.stride, padding=wl.pad, out=out, ws=ws)
        path = PATHS[cfg] if cfg != 4 or not args.dilated_path else args.dilated_path
        fused = path != "staged"
        if path == "residues":
            kw["residues"] = True
        if cfg == 3:
            kw["output_padding"] = wl.out_pad
        if cfg == 4:
            kw["dilation"] = wl.dil
        flops, eop_bytes = conv_costs(wl, ho, wo)
        conv_ops.append(dict(cfg=cfg, wl=wl, entry=entry, x=x, wt=wt, kw=kw, desc=desc, ws=ws,
                             path=path,
                             out=out, flops=flops, eop_bytes=eop_bytes, fused=fused,
                             m=wl.n * wl.h * wl.w, nc=wl.r * wl.s * wl.k))
    bwl = synth.WORKLOADS[5]
    q, k, v = (t.to(dev) for t in synth.band_inputs(bwl))
    o = torch.empty(tuple(q.shape), dtype=torch.float32, device=dev)
    bflops = band_flops(bwl)

    def band_call():
        ol.banded_bmm(q, k, v, bwl.w, bwl.dilation, bwl.scale, mask_invalid=bwl.mask_invalid,
                      out=o)

    if args.stage:
        run_stage(args, conv_ops, bwl, q, k, v, o, stream)
        return

    def conv_call(op):
        op["entry"](op["x"], op["wt"], **dict(op["kw"], fuse=op["fused"]))

    # the four operators are independent: with --streams > 1 they are forked from the
    # current stream onto side streams (default priority) and joined back each step
    groups = {1: [conv_ops + ["band"]], 2: [conv_ops, ["band"]],
              4: [[op] for op in conv_ops] + [["band"]]}[args.streams]
    side = [torch.cuda.Stream(dev) for _ in groups[1:]]

    def run_group(group):
        for op in group:
            band_call() if op == "band" else conv_call(op)

    def step():
        if not side:
            run_group(groups[0])
            return
        main = torch.cuda.current_stream(dev)
        fork = torch.cuda.Event()
        fork.record(main)
        joins = []
        for s_, group in zip(side, groups[1:]):
            s_.wait_event(fork)
            with torch.cuda.stream(s_):
                run_group(group)
                ev = torch.cuda.Event()
                ev.record(s_)
                joins.append(ev)
        run_group(groups[0])
        for ev in joins:
            main.wait_event(ev)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ----------------------------------------------------------------- timed steps
    # K steps launched back to back: the host stays ahead of the GPU, so the kernels of
    # consecutive steps run without gaps.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_per_step = (time.perf_counter() - t0) * 1e3 / args.steps
    # The same step captured once into a HIP graph and replayed K times (for callers that
    # replay a graph per batch); each replay adds the graph launch latency between steps.
    step_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(step_graph):
        step()
    step_graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step_graph.replay()
    torch.cuda.synchronize()
    graph_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    total_flops = sum(op["flops"] for op in conv_ops) + bflops
    value = total_flops / (ms_per_step * 1e-3) / 1e12

    # ------------------------------------------------ per-kernel timing (HIP events)
    def time_kernel(fn, reps):
        """Average duration of one launch: `reps` launches captured in a HIP graph,
        replayed between two events on the current stream."""
        fn()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(reps):
                fn()
        graph.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        graph.replay()
        e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) / reps   # ms per launch

    # Cold: before every launch a 512 MB buffer is read (outside the events), which
    # evicts L2 (4 MB per XCD) and the 256 MB MALL with clean lines; the median of the
    # launches is kept.  (Writing the buffer instead leaves dirty lines whose write-back
    # then runs inside the timed launch.)
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
    flush_sink = torch.empty((), dtype=torch.float32, device=dev)

    def time_kernel_cold(fn, reps):
        fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(reps)]
        for i in range(reps):
            torch.amax(flush, dim=0, out=flush_sink)
            evs[i][0].record(stream)
            fn()
            evs[i][1].record(stream)
        torch.cuda.synchronize()
        d = sorted(a.elapsed_time(b) for a, b in evs)
        return d[len(d) // 2] if len(d) % 2 else 0.5 * (d[len(d) // 2 - 1] + d[len(d) // 2])

    # Cold kernel durations without the launch and event overhead, from HIP graphs of
    # `reps` repetitions replayed three times between events (medians):
    #   A = (flush, kernel),  C = (flush, tiny),  D = (flush, tiny, tiny)
    # with `tiny` a one-element kernel.  Per repetition A - C = kernel - tiny and
    # D - C = tiny + one launch gap, so (A + D - 2C) / reps is the kernel's duration
    # after a flush plus one gap between graph nodes (about 1.5-2 us on this chip): the
    # flush, the tiny kernel and the event overhead cancel.  The rocprofv3 kernel-trace
    # durations of the same pairs (bench.py --stage NAME --cold), when their record in
    # profiles/ matches the current kernel sources, are reported beside them
    # ("cold_trace"): the kernel alone.
    noop = lambda: flush_sink.add_(1.0)      # a one-element kernel (no memset node)

    def seq_graph_ms(seq, reps):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                for f in seq:
                    f()
        g.replay()
        torch.cuda.synchronize()
        times = []
        for _ in range(3):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            g.replay()
            e1.record(stream)
            e1.synchronize()
            times.append(e0.elapsed_time(e1))
        del g
        return sorted(times)[1]

    flush_fn = lambda: torch.amax(flush, dim=0, out=flush_sink)
    reps = max(args.steps, 10)
    reps_cold = max(args.steps, 30)
    reps_pair = 20
    base_c_ms = seq_graph_ms([flush_fn, noop], reps_pair)
    base_d_ms = seq_graph_ms([flush_fn, noop, noop], reps_pair)

    def time_kernel_cold_dur(fn):
        fn()
        torch.cuda.synchronize()
        a_ms = seq_graph_ms([flush_fn, fn], reps_pair)
        return max((a_ms + base_d_ms - 2 * base_c_ms) / reps_pair, 0.0)

    # what a single launch costs between its events on this stream: a one-element fill,
    # timed like the event-bracketed cold launches (part of each such figure)
    event_floor = time_kernel_cold(noop, reps_cold)
    per_cfg = {}
    trace_rec = cold_trace_record()
    kernels = []   # (name, ms per launch, bound, achieved, peak, unit, algorithmic work)
    for op in conv_ops:
        y = op["ws"][:op["m"] * op["nc"] * 4].view(torch.float32).view(op["m"], op["nc"])
        a = op["x"].view(op["m"], op["wl"].c)
        b = op["wt"].view(op["nc"], op["wl"].c)
        g_fn = lambda: ol.gemm_nt(a, b, out=y)
        e_fn = lambda: ol.eop_gather(op["desc"], op["wl"].transposed, y, out=op["out"])
        kw_f = {k_: v_ for k_, v_ in op["kw"].items() if k_ != "residues"}
        f_fn = lambda: op["entry"](op["x"], op["wt"], **dict(kw_f, ws=None, fuse=True))
        g_ms = time_kernel(g_fn, reps)
        # the same GEMM stage with its scope Y held in bf16 (OLLIE_Y_BF16): half of Y's
        # bytes; a variant reported beside the fp32 default, never the headline
        yb = op["ws"][:op["m"] * op["nc"] * 2].view(torch.bfloat16).view(op["m"], op["nc"])
        gb_ms = time_kernel(lambda: ol.gemm_nt(a, b, y_dtype=torch.bfloat16, out=yb), reps)
        e_ms = time_kernel(e_fn, reps)
        f_ms = time_kernel(f_fn, reps)
        g_cold = time_kernel_cold_dur(g_fn)
        e_cold = time_kernel_cold_dur(e_fn)
        f_cold = time_kernel_cold_dur(f_fn)
        e_cold_ev = time_kernel_cold(e_fn, reps_cold)
        r_ms = None
        if op["cfg"] == 4:   # the dilated workload also in the residue sub-image form
            r_ms = time_kernel(lambda: op["entry"](op["x"], op["wt"],
                                                   **dict(kw_f, ws=None, residues=True)),
                               reps)
        k_ms = r_ms if op["path"] == "residues" else f_ms   # the fused kernel the step runs
        k_tf = op["flops"] / (k_ms * 1e-3) / 1e12
        g_tf = op["flops"] / (g_ms * 1e-3) / 1e12
        e_gb = op["eop_bytes"] / (e_ms * 1e-3) / 1e9
        f_tf = op["flops"] / (f_ms * 1e-3) / 1e12
        # the GEMM stage's HBM bytes: Y written once, A and B read once
        g_bytes = op["m"] * op["nc"] * 4 + (op["m"] + op["nc"]) * op["wl"].c * 2
        g_gb = g_bytes / (g_ms * 1e-3) / 1e9
        t_mfma = op["flops"] / (PEAK_BF16_TFLOPS * 1e12)
        t_hbm = g_bytes / (PEAK_HBM_GBS * 1e9)
        g_bound = "hbm" if t_hbm > t_mfma else "mfma"
        name = op["wl"].name
        per_cfg[name] = {
            "path": op["path"],
            "op_ms": round(k_ms if op["fused"] else g_ms + e_ms, 5),
            "gemm_ms": round(g_ms, 5), "gemm_tflops": round(g_tf, 2),
            "gemm_pct_mfma_peak": round(100 * g_tf / PEAK_BF16_TFLOPS, 2),
            "gemm_hbm_gbs": round(g_gb, 1), "gemm_pct_hbm_peak": round(100 * g_gb / PEAK_HBM_GBS, 2),
            "gemm_bound": g_bound,
            "gemm_pct_roofline": round(100 * max(t_mfma, t_hbm) / (g_ms * 1e-3), 2),
            "gemm_ybf16_ms": round(gb_ms, 5),
            "gemm_ybf16_tflops": round(op["flops"] / (gb_ms * 1e-3) / 1e12, 2),
            "gemm_ybf16_pct_mfma_peak": round(100 * t_mfma / (gb_ms * 1e-3), 2),
            "eop_ms": round(e_ms, 5), "eop_gbs_mall_assisted": round(e_gb, 1),
            "eop_pct_hbm_peak_mall_assisted": round(100 * e_gb / PEAK_HBM_GBS, 2),
            "fused_ms": round(f_ms, 5), "fused_tflops": round(f_tf, 2),
            "fused_pct_mfma_peak": round(100 * f_tf / PEAK_BF16_TFLOPS, 2),
            "gemm_gflop": round(op["flops"] / 1e9, 4), "gemm_mbytes": round(g_bytes / 1e6, 3),
            "eop_mbytes": round(op["eop_bytes"] / 1e6, 3),
        }
        t_g = max(t_mfma, t_hbm)
        per_cfg[name].update({
            "cold": {"gemm_ms": round(g_cold, 5),
                     "gemm_tflops": round(op["flops"] / (g_cold * 1e-3) / 1e12, 2),
                     "gemm_pct_mfma_peak": round(100 * t_mfma / (g_cold * 1e-3), 2),
                     "gemm_pct_roofline": round(100 * t_g / (g_cold * 1e-3), 2),
                     "eop_ms": round(e_cold, 5),
                     "eop_gbs": round(op["eop_bytes"] / (e_cold * 1e-3) / 1e9, 1),
                     "eop_pct_hbm_peak": round(100 * op["eop_bytes"] / (e_cold * 1e-3)
                                               / (PEAK_HBM_GBS * 1e9), 2),
                     "eop_event_bracketed_ms": round(e_cold_ev, 5),
                     "fused_ms": round(f_cold, 5),
                     "fused_tflops": round(op["flops"] / (f_cold * 1e-3) / 1e12, 2),
                     "fused_pct_mfma_peak": round(100 * t_mfma / (f_cold * 1e-3), 2)},
        })
        if r_ms is not None:
            per_cfg[name]["fused_residue_form_ms"] = round(r_ms, 5)
        ct = {}
        for kind in ("gemm", "eop", "fused"):
            ms = trace_rec.get(f"{kind}:{op['cfg']}")
            if ms is None:
                continue
            ct[f"{kind}_ms"] = round(ms, 5)
            if kind == "eop":
                ct["eop_gbs"] = round(op["eop_bytes"] / (ms * 1e-3) / 1e9, 1)
                ct["eop_pct_hbm_peak"] = round(100 * op["eop_bytes"] / (ms * 1e-3)
                                               / (PEAK_HBM_GBS * 1e9), 2)
            else:
                ct[f"{kind}_pct_mfma_peak"] = round(100 * t_mfma / (ms * 1e-3), 2)
                if kind == "gemm":
                    ct["gemm_pct_roofline"] = round(100 * t_g / (ms * 1e-3), 2)
        if ct:
            per_cfg[name]["cold_trace"] = ct
        if op["fused"]:
            kernels.append((f"conv_fused[{name}]", k_ms, "mfma", k_tf, PEAK_BF16_TFLOPS,
                            "TFLOP/s", op["flops"]))
        else:
            if g_bound == "hbm":
                kernels.append((f"gemm_nt[{name}]", g_ms, "hbm", g_gb, PEAK_HBM_GBS, "GB/s",
                                g_bytes))
            else:
                kernels.append((f"gemm_nt[{name}]", g_ms, "mfma", g_tf, PEAK_BF16_TFLOPS,
                                "TFLOP/s", op["flops"]))
            kernels.append((f"eop_gather[{name}]", e_ms, "hbm", e_gb, PEAK_HBM_GBS, "GB/s",
                            op["eop_bytes"]))
    b_ms = time_kernel(band_call, reps)
    b_cold = time_kernel_cold_dur(band_call)
    b_tf = bflops / (b_ms * 1e-3) / 1e12
    per_cfg[bwl.name] = {"path": "fused", "op_ms": round(b_ms, 5), "fused_ms": round(b_ms, 5),
                         "band_tflops": round(b_tf, 2),
                         "band_pct_mfma_peak": round(100 * b_tf / PEAK_BF16_TFLOPS, 2),
                         "band_gflop": round(bflops / 1e9, 3),
                         "cold": {"fused_ms": round(b_cold, 5),
                                  "band_tflops": round(bflops / (b_cold * 1e-3) / 1e12, 2),
                                  "band_pct_mfma_peak": round(
                                      100 * bflops / (b_cold * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                                      2)}}
    # the staged band (OLLIE_BAND_STAGED): G2BMM -> softmax eOperator -> GBMM through S
    # (fp32) and P (bf16), each an HBM-bound stage with algorithmic bytes
    #   G2BMM: Q + K read, S written;  softmax: S read, P written;  GBMM: P + V read, O written
    nbnd = 2 * bwl.w + 1
    rows = bwl.b * bwl.l
    s_st = torch.empty((bwl.b, bwl.l, nbnd), dtype=torch.float32, device=dev)
    p_st = torch.empty((bwl.b, bwl.l, nbnd), dtype=torch.bfloat16, device=dev)
    ol.band_g2bmm(q, k, bwl.w, bwl.dilation, bwl.scale, s=s_st)
    ol.band_softmax(s_st, bwl.w, bwl.dilation, bwl.mask_invalid, p=p_st)
    qkv_bytes = rows * bwl.d * 2
    stages = {
        "g2bmm": (lambda: ol.band_g2bmm(q, k, bwl.w, bwl.dilation, bwl.scale, s=s_st),
                  2 * qkv_bytes + rows * nbnd * 4),
        "softmax_eop": (lambda: ol.band_softmax(s_st, bwl.w, bwl.dilation, bwl.mask_invalid,
                                                p=p_st), rows * nbnd * (4 + 2)),
        "gbmm": (lambda: ol.band_gbmm(p_st, v, bwl.w, bwl.dilation, o=o),
                 rows * nbnd * 2 + qkv_bytes + rows * bwl.d * 4),
    }
    staged = {}
    for nm, (fn, nbytes) in stages.items():
        w_ms = time_kernel(fn, reps)
        c_ms = time_kernel_cold_dur(fn)
        staged[nm] = {"warm_ms": round(w_ms, 5), "cold_ms": round(c_ms, 5),
                      "mbytes": round(nbytes / 1e6, 2),
                      "gbs": round(nbytes / (c_ms * 1e-3) / 1e9, 1),
                      "pct_hbm_peak": round(100 * nbytes / (c_ms * 1e-3) / (PEAK_HBM_GBS * 1e9),
                                            2)}
    for nm, key in (("g2bmm", "band_g2bmm"), ("softmax_eop", "band_softmax"),
                    ("gbmm", "band_gbmm")):
        ms = trace_rec.get(key)
        if ms is not None:
            staged[nm]["cold_trace_ms"] = round(ms, 5)
            staged[nm]["pct_hbm_peak_trace"] = round(
                100 * stages[nm][1] / (ms * 1e-3) / (PEAK_HBM_GBS * 1e9), 2)
    ms = trace_rec.get("band_fused")
    if ms is not None:
        per_cfg[bwl.name]["cold_trace"] = {
            "fused_ms": round(ms, 5),
            "band_pct_mfma_peak": round(100 * bflops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2)}
    staged["op_ms"] = round(sum(staged[n]["warm_ms"] for n in stages), 5)
    per_cfg[bwl.name]["staged"] = staged
    per_cfg[bwl.name]["eop_ms"] = staged["softmax_eop"]["cold_ms"]
    per_cfg[bwl.name]["eop_pct_hbm_peak"] = staged["softmax_eop"]["pct_hbm_peak"]
    del s_st, p_st
    kernels.append((f"band_fused[{bwl.name}]", b_ms, "mfma", b_tf, PEAK_BF16_TFLOPS, "TFLOP/s",
                    bflops))
    # ------------------------- the Conv5x5 -> Conv3x3 derived form (a workload of its own,
    # not part of the step): the SRCNN layer direct (fused over its 25 taps), in the
    # split form (weight split + fused 3x3 stage with 4K channels + block OffsetAdd),
    # and direct through GEMM + OffsetAdd; rates use the direct form's flops
    next_rows = {}
    swl, s_fns = srcnn_calls(dev)
    s_flops = conv_costs(swl, swl.h, swl.w)[0]
    row = {"row": "Conv5x5 -> Conv3x3 derived form", "gflop": round(s_flops / 1e9, 3),
           "split_mfma_work_ratio": round(9 * ((swl.r + 2) // 3) * ((swl.s + 2) // 3)
                                          / (swl.r * swl.s), 4)}
    for nm, fn in s_fns.items():
        w_ms = time_kernel(fn, reps)
        c_ms = time_kernel_cold_dur(fn)
        row[f"{nm}_ms"] = round(w_ms, 5)
        row[f"{nm}_tflops"] = round(s_flops / (w_ms * 1e-3) / 1e12, 2)
        row[f"{nm}_cold_ms"] = round(c_ms, 5)
    next_rows[swl.name] = row

    # The roofline entry covers the kernel with the largest share of a step (warm
    # back-to-back launches, whose average rocprofv3's kernel trace of the same run
    # shows); frac_cold is the same fraction from the cold median.
    cold_ms = {f"band_fused[{bwl.name}]": b_cold}
    for op in conv_ops:
        c = per_cfg[op["wl"].name]["cold"]
        if op["fused"]:
            cold_ms[f"conv_fused[{op['wl'].name}]"] = c["fused_ms"]
        else:
            cold_ms[f"gemm_nt[{op['wl'].name}]"] = c["gemm_ms"]
            cold_ms[f"eop_gather[{op['wl'].name}]"] = c["eop_ms"]
    timed = kernels
    dom = max(timed, key=lambda t: t[1])
    roofline = {"kernel": dom[0], "bound": dom[2], "achieved": round(dom[3], 3),
                "peak": dom[4], "unit": dom[5], "frac": round(dom[3] / dom[4], 4),
                "traffic": traffic_record(dom[0]), "avg_launch_ms": round(dom[1], 5),
                "algorithmic_per_launch": dom[6],
                "cold_launch_ms": round(cold_ms[dom[0]], 5),
                "frac_cold": round(dom[6] / (cold_ms[dom[0]] * 1e-3)
                                   / (1e12 if dom[5] == "TFLOP/s" else 1e9) / dom[4], 4)}

    # ---------------------------------------------------------------- CPU baseline
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(conv_ops, bwl)

    line = {
        "metric": "GEMM TFLOP/s (% MFMA peak) + eOperator GB/s (% HBM peak), per config, 1 GPU",
        "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "graph_replay_ms_per_step": round(graph_ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "derived conv3x3 (N16 C256 14x14) + convT4x4s2 (N16 512->256 "
                               "8x8) + dilated conv3x3 d2 (C512 96x128) + band (B96 L4096 d64 "
                               "w256 dil2), bf16 in, fp32 accumulate/out",
                   "parallelism": "single GPU",
                   "launch": "stream" if args.streams == 1 else
                             f"{args.streams} streams (independent operators side by side)",
                   "paths": {op["wl"].name: op["path"] for op in conv_ops}},
        "per_config": per_cfg,
        "next_rows": next_rows,
        "cold_event_floor_ms": round(event_floor, 5),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def run_stage(args, conv_ops, bwl, q, k, v, o, stream):
    """Launch one stage kernel `steps` times after `warmup` launches; print its
    HIP-event average (for rocprofv3 runs that should see a single kernel/workload)."""
    import torch
    import paper_2208_02025_amd as ol

    name = args.stage
    fn = None
    if ":" in name:
        kind, cfg = name.split(":")
        op = next(o_ for o_ in conv_ops if o_["cfg"] == int(cfg))
        y = op["ws"][:op["m"] * op["nc"] * 4].view(torch.float32).view(op["m"], op["nc"])
        a = op["x"].view(op["m"], op["wl"].c)
        b = op["wt"].view(op["nc"], op["wl"].c)
        if kind == "gemm":
            fn = lambda: ol.gemm_nt(a, b, out=y)
        elif kind == "eop":
            ol.gemm_nt(a, b, out=y)
            fn = lambda: ol.eop_gather(op["desc"], op["wl"].transposed, y, out=op["out"])
        elif kind == "op":
            fn = lambda: op["entry"](op["x"], op["wt"], **op["kw"])
        elif kind == "fused":
            fn = lambda: op["entry"](op["x"], op["wt"], **dict(op["kw"], fuse=True))
        elif kind == "fusedres":
            fn = lambda: op["entry"](op["x"], op["wt"], **dict(op["kw"], ws=None, residues=True))
    elif name in ("srcnn_direct_fused", "srcnn_split3x3", "srcnn_split3x3_chain",
                  "srcnn_direct_staged"):
        fn = srcnn_calls(q.device)[1][name[len("srcnn_"):]]
    elif name == "band_fused":
        fn = lambda: ol.banded_bmm(q, k, v, bwl.w, bwl.dilation, bwl.scale,
                                   mask_invalid=bwl.mask_invalid, out=o)
    elif name in ("band_g2bmm", "band_softmax", "band_gbmm"):
        s = ol.band_g2bmm(q, k, bwl.w, bwl.dilation, bwl.scale)
        p = ol.band_softmax(s, bwl.w, bwl.dilation, bwl.mask_invalid)
        fn = {"band_g2bmm": lambda: ol.band_g2bmm(q, k, bwl.w, bwl.dilation, bwl.scale, s=s),
              "band_softmax": lambda: ol.band_softmax(s, bwl.w, bwl.dilation,
                                                      bwl.mask_invalid, p=p),
              "band_gbmm": lambda: ol.band_gbmm(p, v, bwl.w, bwl.dilation, o=o)}[name]
    elif name == "copy":
        # plain device copy of 256 MiB: the reference for scaling HBM traffic counters
        src = torch.empty(64 << 20, dtype=torch.float32, device=q.device).fill_(1.0)
        dst = torch.empty_like(src)
        fn = lambda: dst.copy_(src)
    if fn is None:
        raise SystemExit(f"unknown stage {name}")
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    # a HIP graph of `steps` launches, replayed between two events: kernel time only,
    # no host launch gaps (the same method as the main benchmark's per-kernel figures);
    # with --cold each launch follows a 512 MB read that evicts L2 and the MALL (the
    # pairs of the benchmark's cold figures, so a kernel trace of this run gives the
    # cold kernel durations directly)
    flush = torch.ones(128 << 20, dtype=torch.float32, device=q.device) if args.cold else None
    sink = torch.empty((), dtype=torch.float32, device=q.device)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(args.steps):
            if flush is not None:
                torch.amax(flush, dim=0, out=sink)
            fn()
    graph.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    graph.replay()
    e1.record(stream)
    e1.synchronize()
    print(json.dumps({"stage": name, "launches": args.steps, "cold": bool(args.cold),
                      "avg_ms_incl_flush" if args.cold else "avg_ms":
                          round(e0.elapsed_time(e1) / args.steps, 5)}), flush=True)


def cpu_baseline(conv_ops, bwl):
    """The oracle (as it stands) on whole steps of the same workloads: every output of
    the three convolutions and every row of the band, repeated until about 10 s of CPU
    time (at most 8 steps); value = the steps' algorithmic flops / CPU time."""
    import oracle
    import synth

    inputs = [(op, synth.conv_inputs(op["wl"])) for op in conv_ops]
    qkv = synth.band_inputs(bwl)
    flops = 0.0
    secs = 0.0
    steps = 0
    while steps == 0 or (secs < 10.0 and steps < 8):
        for op, (x, wt) in inputs:
            wl = op["wl"]
            t0 = time.perf_counter()
            if wl.transposed:
                oracle.conv_transpose2d(x, wt, wl.stride, wl.pad, wl.dil, wl.out_pad)
            else:
                oracle.conv2d(x, wt, wl.stride, wl.pad, wl.dil)
            secs += time.perf_counter() - t0
            flops += op["flops"]
        t0 = time.perf_counter()
        oracle.band(*qkv, bwl.w, bwl.dilation, bwl.scale, bwl.mask_invalid, want_s=False,
                    want_p=False)
        secs += time.perf_counter() - t0
        flops += band_flops(bwl)
        steps += 1
    return {"value": round(flops / secs / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds": round(secs, 2),
            "sample": f"{steps} whole step(s), repeated until at least 10 s of CPU time: all "
                      "outputs of the conv3x3, convT and dilated conv workloads and all "
                      "393216 band rows"}


if __name__ == "__main__":
    main()
