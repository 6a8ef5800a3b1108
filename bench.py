"""Benchmark of one layer's QCFuse fusion step on one MI355X.

A step is the whole hot path over one batch: re-positioning, query-row
rotation and the probe buffer (one fused launch), anchor probe attention,
critical-layer scores, per-chunk top-k, scatter of the recomputed rows and
their causal attention.
The default workload is the largest single-GPU one: a long-context layer shaped
like a 70B GQA model (32 chunks x 1024 tokens + a 128-token query, H_q=64,
H_kv=8, d=128, bf16, rho=30%), seeded synthetic data; ``--config c2`` / ``c5``
run the Llama-3-8B-shaped layer and the ragged 16-request batch.
Inputs are resident in HBM before the timed region; several buffer sets are
rotated so the 256 MB last-level cache does not hold the previous step's data.

Prints one JSON line:  metric = selected-token fused-prefill tokens/s per layer
(|R| recomputed rows / step time), with the attention call's roofline
fraction (algorithmic FLOPs per launch / its average HIP-event duration), its
measured HBM traffic (the committed counter record, while the attention
source is unchanged) and the CPU oracle's throughput on a bounded sample of
the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def attention_code_digest():
    """sha256 of the attention source with its comments and blank lines removed: a counter
    record stays valid while the kernel code it measured is unchanged."""
    import hashlib
    import re
    src = open(os.path.join(ROOT, "paper_2606_05875_amd", "csrc", "attention.hip"),
               encoding="utf-8").read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    code = "\n".join(line.rstrip() for line in src.splitlines() if line.strip())
    return hashlib.sha256(code.encode()).hexdigest()


def measured_traffic(config, kv_row_stride):
    """HBM bytes per attention call from the committed counter record of this workload, or
    None when there is none or the attention code or the cache row stride has changed
    since the counters were taken."""
    rec_path = os.path.join(ROOT, "profiles", f"attention_{config}_hbm_traffic.md")
    try:
        rec = None
        for line in open(rec_path):
            if line.startswith("{"):
                rec = json.loads(line)
        digest = attention_code_digest()
    except (OSError, ValueError):
        return None
    if (not rec or rec.get("attention_code_sha256") != digest
            or rec.get("kv_row_stride") != kv_row_stride):
        return None
    return rec["bytes_per_call"]


def attn_flops(step, R_pos):
    """Algorithmic FLOPs of the causal row attention: 4*H_q*d*sum(pos+1) over recomputed rows."""
    w = step.w
    return 4.0 * w.n_q_heads * w.head_dim * float(np.sum(R_pos.astype(np.float64) + 1.0))


def assemble_bytes(step):
    """Algorithmic HBM bytes of qcf_assemble: every chunk row's K and V read and written once;
    each query row reads q/k/v and writes k/v twice (cache, probe) and q once; each anchor
    reads its stored K/V row and writes it into the probe buffer."""
    w, p = step.w, step.plan
    e = 2 if w.dtype == "bf16" else 4
    kv = w.n_kv_heads * w.head_dim * e
    qb = w.n_q_heads * w.head_dim * e
    n_ctx = int(w.seg_len.sum())
    n_q = int(p.u_idx.size)
    n_anchor = int(p.probe_idx.size) - n_q
    return 4.0 * kv * n_ctx + n_q * (2 * qb + 6 * kv) + 4.0 * kv * n_anchor


def scatter_bytes(step):
    """Fresh rows of R: k, v read, rotated k plus v written (and q read, rotated q written when
    the attention does not rotate the queries itself)."""
    w = step.w
    n = int(step.R_idx.numel())
    es = step.k.element_size()
    nq = 0 if step.rot_in_attn else 2 * w.n_q_heads
    return n * (nq + 4 * w.n_kv_heads) * w.head_dim * es


def probe_attn_flops(step):
    w, p = step.w, step.plan
    tot = 0.0
    for b in range(w.batch):
        na = int(p.cu_probe[b + 1] - p.cu_probe[b]) - int(w.q_lens[b])
        nq = int(w.q_lens[b])
        tot += sum(na + i + 1 for i in range(nq))
    return 4.0 * w.n_q_heads * w.head_dim * tot


def stack_study(args):
    """c3: the 36-layer stack.  Times the selector with the compact view (anchors, critical
    layers) and with the full view (every context token, every layer), the recompute of
    every layer, and the overlap of the two selections (the paper's requirement
    T_select(C_A, L*) < T_select(C, L) and the coverage it trades for it)."""
    import torch
    from paper_2606_05875_amd.stack import FusionStack
    from paper_2606_05875_amd.workloads import full_view, make_stack_workload

    torch.cuda.set_device(0)
    sw = make_stack_workload("c3")
    res = {}
    for view, w in (("anchors", sw), ("full", full_view(sw))):
        st = FusionStack(w)
        st.build_pic()
        for _ in range(max(1, args.warmup)):
            st.run()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        t_sel, t_rec = [], []
        for _ in range(args.steps):
            ev[0].record()
            st.select()
            ev[1].record()
            st.recompute()
            ev[2].record()
            torch.cuda.synchronize()
            t_sel.append(ev[0].elapsed_time(ev[1]))
            t_rec.append(ev[1].elapsed_time(ev[2]))
        out = st.results()
        res[view] = dict(select_ms=float(np.median(t_sel)), recompute_ms=float(np.median(t_rec)),
                         P=np.concatenate(out["P"]), n_R=int(out["R"].size))
        del st
        torch.cuda.empty_cache()
    # recompute-ratio sweep on the compact view (the PIC caches and inputs shared); 100% is a
    # full prefill of every token through the same kernels
    sweep = {}
    base = FusionStack(sw)
    base.build_pic()
    for rho in (1500, 3000, 5000, 10000):
        st = FusionStack(sw, rho_bp=rho, share=base)
        for _ in range(max(1, args.warmup)):
            st.run()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        t_sel, t_rec = [], []
        torch.cuda.synchronize()
        for _ in range(args.steps):
            ev[0].record()
            st.select()
            ev[1].record()
            st.recompute()
            ev[2].record()
            torch.cuda.synchronize()
            t_sel.append(ev[0].elapsed_time(ev[1]))
            t_rec.append(ev[1].elapsed_time(ev[2]))
        n_R = int(st.R_idx.numel())
        sel, rec = float(np.median(t_sel)), float(np.median(t_rec))
        sweep[rho] = dict(recomputed_rows=n_R, select_ms=sel, recompute_ms=rec,
                          tokens_per_s=n_R * sw.n_layers / ((sel + rec) * 1e-3))
        del st
    # full prefill = every token through every layer with no selection: the 100% recompute
    full = sweep[10000]["recompute_ms"]
    for rho, r in sweep.items():
        if rho != 10000:
            r["speedup_vs_full_prefill"] = full / (r["select_ms"] + r["recompute_ms"])
    del base
    torch.cuda.empty_cache()
    a, f = res["anchors"], res["full"]
    overlap = np.intersect1d(a["P"], f["P"]).size / max(f["P"].size, 1)
    L = sw.n_layers
    print(json.dumps({
        "metric": "c3 stack: selected-token fused-prefill tokens/s per layer", "unit": "tokens/s",
        "value": a["n_R"] * L / ((a["select_ms"] + a["recompute_ms"]) * 1e-3),
        "recompute_only_value": a["n_R"] * L / (a["recompute_ms"] * 1e-3),
        "steps": args.steps, "warmup": args.warmup, "dtype": "bf16", "data": "synthetic (seeded, random weights)",
        "config": {"workload": "c3: " + sw.meta["desc"], "recomputed_rows": a["n_R"], "layers": L,
                   "rho_bp": sw.rho_bp},
        "select_ms": {"anchors_critical_layers": a["select_ms"], "full_view_all_layers": f["select_ms"]},
        "recompute_ms": a["recompute_ms"],
        "select_speedup": f["select_ms"] / a["select_ms"],
        "P_overlap_with_full_view": overlap,
        "ratio_sweep": {f"{rho / 100:g}%": r for rho, r in sweep.items()},
        "full_prefill_ms": full}), flush=True)


def recompute_study(args):
    """c3 at rho 30%: the recompute of every layer alone (selection done once before), timed over
    ``--steps`` runs.  Under a kernel trace the run holds only recompute launches, so its
    statistics split a layer between libqcf's kernels and the stack's glue (RMSNorm, the
    projections and the residual product)."""
    import torch
    from paper_2606_05875_amd.stack import FusionStack
    from paper_2606_05875_amd.workloads import make_stack_workload

    torch.cuda.set_device(0)
    sw = make_stack_workload("c3")
    st = FusionStack(sw)
    st.build_pic()
    st.select()
    for _ in range(max(1, args.warmup)):
        st.recompute()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(args.steps):
        st.recompute()
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    n_R = int(st.R_idx.numel())
    print(json.dumps({"study": "c3 recompute alone", "rho_bp": st.rho_bp, "layers": sw.n_layers,
                      "recomputed_rows": n_R, "runs": args.steps, "warmup": args.warmup,
                      "ms_per_recompute": ms, "us_per_layer": ms * 1e3 / sw.n_layers}), flush=True)


def pipeline_study(args):
    """c3 with the PIC caches in pinned host memory: each layer's cache loads on a copy
    stream while earlier layers compute (Section 3.5).  Reports the copy-only time, the
    compute-only time (caches resident in HBM), the overlapped time and the overlap
    efficiency (t_copy + t_compute - t_overlapped) / min(t_copy, t_compute)."""
    import torch
    from paper_2606_05875_amd.stack import FusionStack, HostPicPipeline
    from paper_2606_05875_amd.workloads import make_stack_workload

    torch.cuda.set_device(0)
    sw = make_stack_workload("c3")
    st = FusionStack(sw)
    st.build_pic()
    pipe = HostPicPipeline(st, slots=args.slots)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn):
        for _ in range(max(1, args.warmup)):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(args.steps):
            ev[0].record()
            fn()
            ev[1].record()
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
        return float(np.median(ts))

    t_compute = timed(lambda: st.run())
    t_copy = timed(lambda: pipe.copy_only())
    t_over = timed(lambda: st.run(pipe.begin()))
    # the part of the shorter phase hidden under the longer one
    eff = (t_copy + t_compute - t_over) / min(t_copy, t_compute)
    print(json.dumps({
        "metric": "c3 stack with host-resident PIC caches: selected-token fused-prefill tokens/s per layer",
        "unit": "tokens/s", "value": int(st.R_idx.numel()) * sw.n_layers / (t_over * 1e-3),
        "steps": args.steps, "warmup": args.warmup, "dtype": "bf16", "data": "synthetic (seeded, random weights)",
        "config": {"workload": "c3: " + sw.meta["desc"], "recomputed_rows": int(st.R_idx.numel()),
                   "layers": sw.n_layers, "rho_bp": sw.rho_bp},
        "host_to_device_bytes": pipe.bytes, "copy_only_ms": t_copy,
        "copy_GBs": pipe.bytes / (t_copy * 1e-3) / 1e9, "compute_only_ms": t_compute,
        "overlapped_ms": t_over, "overlap_efficiency": eff, "staging_slots": pipe.n_slots}), flush=True)


def anchor_profile(args):
    """Recall@10% (eq. profile_recall_at10) of planted evidence on the c3 stack: the query
    probe with no anchors, Sink and Knorm anchors at several retained ratios, the full
    view, and scoring at one layer at a time.  The evidence is a mechanism demonstration:
    context duplicates of query tokens plus key heads that match their group's first query
    head (the workload generator's ``evidence``); it is not the paper's span-labelled data."""
    import dataclasses
    import torch
    from paper_2606_05875_amd.anchors import anchors_knorm, anchors_sink
    from paper_2606_05875_amd.stack import FusionStack
    from paper_2606_05875_amd.workloads import make_stack_workload

    torch.cuda.set_device(0)
    sw = make_stack_workload("c3", evidence=(2, 64))
    E = sw.meta["evidence_rows"]
    base = FusionStack(sw, rho_bp=1000)
    base.build_pic()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def recall(anchor_local, layers):
        sv = dataclasses.replace(sw, anchor_local=[np.asarray(a, np.int32) for a in anchor_local],
                                 critical_layers=tuple(layers))
        st = FusionStack(sv, rho_bp=1000, share=base)
        st.select()
        torch.cuda.synchronize()
        ev[0].record()
        st.select()
        ev[1].record()
        torch.cuda.synchronize()
        P = st.R_idx.cpu().numpy()[:int(st.plan.n_P.sum())]
        return float(np.isin(E, P).mean()), ev[0].elapsed_time(ev[1])

    Lstar = sw.critical_layers
    rows = []
    r, t = recall([np.zeros(0, np.int32)] * sw.n_chunks, Lstar)
    rows.append(dict(view="query only (r_a = 0)", recall=r, select_ms=t))
    for ra in (500, 1000, 2000, 5000):
        for name, fn in (("sink", lambda ra=ra: anchors_sink(sw.seg_len, ra)),
                         ("knorm", lambda ra=ra: anchors_knorm(base.k_pic, sw.seg_start, sw.seg_len, ra))):
            r, t = recall(fn(), Lstar)
            rows.append(dict(view=f"{name} r_a = {ra / 10000:g}", recall=r, select_ms=t))
    r, t = recall([np.arange(n) for n in sw.seg_len], Lstar)
    rows.append(dict(view="full context (r_a = 1)", recall=r, select_ms=t))
    kn = anchors_knorm(base.k_pic, sw.seg_start, sw.seg_len, 1000)
    per_layer = [recall(kn, (l,))[0] for l in range(sw.n_layers)]
    best = sorted(range(sw.n_layers), key=lambda l: -per_layer[l])[:3]
    r_best, t_best = recall(kn, tuple(sorted(best)))
    r_all, t_all = recall(kn, tuple(range(sw.n_layers)))
    print(json.dumps({
        "metric": "c3 stack: Recall@10% of planted evidence", "workload": "c3: " + sw.meta["desc"],
        "evidence_rows": int(E.size), "scoring_layers_for_anchor_rows": list(Lstar),
        "anchor_views": rows, "per_layer_recall_knorm10": per_layer,
        "top3_layers": sorted(best), "top3_layers_recall": r_best, "top3_select_ms": t_best,
        "all_layers_recall": r_all, "all_layers_select_ms": t_all}), flush=True)


def rerope_rate(steps, hkv, d, reps=40):
    """qcf_rerope (keys re-positioned, values stitched) alone: HIP events around back-to-back
    calls, (a) on the step's own context, cycling through the buffer sets, and (b) on a
    32 x 1024-token context (268 MB per call, three sets cycled so that no call finds its inputs
    in the 256 MB last-level cache).
    Algorithmic bytes: each context row's K and V read once and written once."""
    import torch
    from paper_2606_05875_amd import qcf
    from paper_2606_05875_amd.step import kv_buffer

    def timed(calls):
        for c in calls[:4]:
            c()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for i in range(reps):
            calls[i % len(calls)]()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    out = {}
    ctx = int(steps[0].w.ctx_len.sum())
    t = timed([st.stage_rerope for st in steps])
    nbytes = 4 * ctx * hkv * d * 2
    out["step_context"] = {"rows": ctx, "bytes_per_call": nbytes, "us_per_call": t * 1e6,
                           "GBs": nbytes / t / 1e9, "hbm_frac": nbytes / t / 1e9 / PEAK_HBM_GBS}
    n_seg, seg = 32, 1024
    T = n_seg * seg
    dev = steps[0].device
    i32 = lambda a: torch.tensor(a, dtype=torch.int32, device=dev)
    starts, lens = i32([s * seg for s in range(n_seg)]), i32([seg] * n_seg)
    calls = []
    for _ in range(3):  # three sets (~800 MB): a call never finds its inputs still cached
        k_in = (torch.randn((T, hkv * d), device=dev) * 0.1).to(torch.bfloat16).view(T, hkv, d)
        v_in = torch.randn_like(k_in)
        k_out = kv_buffer(T, hkv, d, torch.bfloat16, dev)
        v_out = kv_buffer(T, hkv, d, torch.bfloat16, dev)
        calls.append(qcf.prepare(qcf.qcf_rerope, k_out, k_in, starts, lens, starts, seg, 5e5,
                                 v_out=v_out, v_in=v_in))
    t = timed(calls)
    nbytes = 4 * T * hkv * d * 2
    out["context_32x1024"] = {"rows": T, "bytes_per_call": nbytes, "us_per_call": t * 1e6,
                              "GBs": nbytes / t / 1e9, "hbm_frac": nbytes / t / 1e9 / PEAK_HBM_GBS}
    return out


def memory_study(args):
    """The HBM-bound kernels alone on the c2 step (a few buffer sets cycled): qcf_assemble,
    qcf_rerope, qcf_scatter_kv; plus qcf_rerope on a 32 x 1024-token context.  One JSON line
    (events around back-to-back calls); run it under rocprofv3 for kernel durations."""
    import torch
    from paper_2606_05875_amd.step import FusionStep
    from paper_2606_05875_amd.workloads import make_workload

    torch.cuda.set_device(0)
    w = make_workload("c2")
    steps = [FusionStep(w) for _ in range(5)]
    for st in steps:
        st.run()
    torch.cuda.synchronize()
    out = {"study": "HBM-bound kernels", "workload": "c2: " + w.meta["desc"]}
    for name, nbytes in (("assemble", assemble_bytes(steps[0])),
                         ("scatter", scatter_bytes(steps[0]))):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for i in range(args.steps):
            getattr(steps[i % len(steps)], "stage_" + name)()
        b.record()
        torch.cuda.synchronize()
        t = a.elapsed_time(b) / args.steps * 1e-3
        out[name] = {"bytes_per_call": nbytes, "us_per_call": t * 1e6, "GBs": nbytes / t / 1e9,
                     "hbm_frac": nbytes / t / 1e9 / PEAK_HBM_GBS}
    out["rerope"] = rerope_rate(steps, w.n_kv_heads, w.head_dim, reps=args.steps)
    # for scale: a plain device copy with the long-context re-position's bytes (134 MB each way)
    pairs = []
    for _ in range(3):  # three sets, as for the re-position
        src = torch.empty(32 * 1024 * w.n_kv_heads * w.head_dim, dtype=torch.float32, device="cuda")
        src.uniform_()
        pairs.append((src, torch.empty_like(src)))
    for i in range(4):
        pairs[i % 3][1].copy_(pairs[i % 3][0])
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for i in range(args.steps):
        pairs[i % 3][1].copy_(pairs[i % 3][0])
    b.record()
    torch.cuda.synchronize()
    t = a.elapsed_time(b) / args.steps * 1e-3
    nbytes = 2 * pairs[0][0].numel() * 4
    out["device_copy"] = {"bytes_per_call": nbytes, "us_per_call": t * 1e6, "GBs": nbytes / t / 1e9,
                          "hbm_frac": nbytes / t / 1e9 / PEAK_HBM_GBS}
    print(json.dumps(out), flush=True)


def topk_study(args):
    """qcf_select_topk alone: per-chunk selection and global (one segment per request)
    selection on the contexts of the workloads, HIP events around 200 back-to-back calls."""
    import torch
    from paper_2606_05875_amd import qcf
    from paper_2606_05875_amd.workloads import make_workload

    torch.cuda.set_device(0)
    rows = []
    for name in ("c2", "c4", "c5"):
        w = make_workload(name)
        rng = np.random.default_rng(3)
        sc = torch.from_numpy(rng.exponential(3.0, w.n_rows).astype(np.float32)).cuda()
        for mode in ("chunk", "global"):
            if mode == "chunk":
                starts, lens, req = w.seg_start, w.seg_len, w.seg_req
            else:
                starts, lens, req = w.cu_kv[:-1], w.ctx_len, np.arange(w.batch)
            ks = (int(w.rho_bp) * np.asarray(lens, np.int64)) // 10000
            outs = np.concatenate([[0], np.cumsum(ks)[:-1]])
            d = lambda a: torch.from_numpy(np.ascontiguousarray(np.asarray(a, np.int32))).cuda()
            out = torch.empty(int(ks.sum()), dtype=torch.int32, device="cuda")
            call = qcf.prepare(qcf.qcf_select_topk, out, sc, d(starts), d(lens), d(ks), d(outs),
                               int(max(lens)))
            for _ in range(10):
                call()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record()
            for _ in range(args.steps):
                call()
            b.record()
            torch.cuda.synchronize()
            rows.append({"workload": name, "selection": mode, "segments": int(len(lens)),
                         "max_segment": int(max(lens)), "selected": int(ks.sum()),
                         "us_per_call": a.elapsed_time(b) / args.steps * 1e3})
    print(json.dumps({"study": "qcf_select_topk per-chunk vs global", "rho_bp": "per workload",
                      "scores": "seeded exponential", "calls": args.steps, "rows": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c4", help="workload: c4 (the headline), c2 or c5")
    ap.add_argument("--sets", type=int, default=0, help="buffer sets rotated (0: enough for 512 MB)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the c2 and c5 summaries that the default c4 line carries")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a 256 MiB device-to-device copy 20 times (HBM counter calibration)")
    ap.add_argument("--stack", action="store_true",
                    help="the c3 multi-layer stack instead: selection (anchor view vs full view) and "
                         "recompute times, one JSON line (not the headline metric)")
    ap.add_argument("--recompute-only", action="store_true",
                    help="with --stack: time the recompute of every layer alone (c3, rho 30%%)")
    ap.add_argument("--pipeline", action="store_true",
                    help="with --stack: the stored chunk caches stream layer by layer from pinned host "
                         "memory (copy-only, compute-only and overlapped times)")
    ap.add_argument("--slots", type=int, default=3, help="with --pipeline: device staging slots")
    ap.add_argument("--memory-study", action="store_true",
                    help="the HBM-bound kernels alone (assemble, rerope, scatter on c2; rerope on a "
                         "32 x 1024-token context), one JSON line; not the headline metric")
    ap.add_argument("--topk-study", action="store_true",
                    help="time qcf_select_topk alone, per-chunk vs global selection, on the c2/c4/c5 "
                         "contexts (one JSON line; not the headline metric)")
    ap.add_argument("--anchor-profile", action="store_true",
                    help="with --stack: Recall@10%% of planted evidence over anchor rules/ratios and "
                         "single scoring layers (a mechanism demonstration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the fusion step has no multi-GPU path; it would "
              "shard by request or by KV-head group, one process per GPU", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        # a plain copy of known size: 256 MiB read + 256 MiB written per launch
        x = torch.empty(64 << 20, dtype=torch.float32, device="cuda").uniform_()
        y = torch.empty_like(x)
        for _ in range(20):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": x.numel() * 4, "bytes_written": y.numel() * 4,
                          "launches": 20}), flush=True)
        return
    if args.topk_study:
        return topk_study(args)
    if args.memory_study:
        return memory_study(args)
    if args.stack:
        if args.anchor_profile:
            return anchor_profile(args)
        if args.recompute_only:
            return recompute_study(args)
        return pipeline_study(args) if args.pipeline else stack_study(args)
    from paper_2606_05875_amd.step import FusionStep
    from paper_2606_05875_amd.workloads import make_workload

    torch.cuda.set_device(0)
    w = make_workload(args.config)
    first = FusionStep(w)
    per_set = sum(t.numel() * t.element_size() for t in (first.k_pic, first.v_pic, first.q_new,
                                                         first.k_new, first.v_new, first.k, first.v))
    n_sets = args.sets or max(1, math.ceil(512e6 / per_set))
    steps = [first] + [FusionStep(w) for _ in range(n_sets - 1)]
    torch.cuda.synchronize()

    for i in range(args.warmup):
        steps[i % n_sets].run()
    torch.cuda.synchronize()

    # headline: K whole steps between two events (events inside the loop would add
    # their own cost to every step)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        steps[i % n_sets].run()
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps

    # the same steps in the fused-scores flow (scores straight from the stored chunk keys,
    # re-positioning on a second stream), for comparison
    for st in steps:
        st.fused = True
    for i in range(args.warmup):
        steps[i % n_sets].run()
    torch.cuda.synchronize()
    t_start.record()
    for i in range(args.steps):
        steps[i % n_sets].run()
    t_end.record()
    torch.cuda.synchronize()
    ms_step_fused = t_start.elapsed_time(t_end) / args.steps
    for st in steps:
        st.fused = False

    # roofline: the same steps again, with events on the launch stream around every
    # recomputed-row attention call
    n_ev = min(args.steps, 100)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n_ev)]
    torch.cuda.synchronize()
    for i in range(n_ev):
        s = steps[i % n_sets]
        s.run_front()
        ev[i][0].record()
        s.stage_attn()
        ev[i][1].record()
        s.join()
    torch.cuda.synchronize()
    attn_all = np.array([a.elapsed_time(b) for a, b in ev])
    attn_ms = float(np.mean(attn_all))

    R_pos = first.R_pos.cpu().numpy()
    n_R = int(R_pos.size)
    flops = attn_flops(first, R_pos)
    achieved = flops / (attn_ms * 1e-3) / 1e12

    # per-stage breakdown (separate, untimed for the headline): events around each stage
    stage_ms = {}
    for name in ("assemble", "scores", "rope_table", "rerope", "query_assemble", "scores_pic",
                 "probe_attn", "select", "scores_select", "scatter", "attn"):
        reps = 20
        # one untimed call per buffer set first: a stage outside the step's own flow
        # marshals its call on first use
        for st in steps:
            getattr(st, "stage_" + name)()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for i in range(reps):
            getattr(steps[i % n_sets], "stage_" + name)()
        b.record()
        torch.cuda.synchronize()
        stage_ms[name] = a.elapsed_time(b) / reps
    asm_gbs = assemble_bytes(first) / (stage_ms["assemble"] * 1e-3) / 1e9
    rerope = rerope_rate(steps, w.n_kv_heads, w.head_dim)

    out = {
        "metric": "selected-token fused-prefill tokens/s per layer",
        "value": n_R / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded; shapes of the paper's 512-token-chunk RAG requests)",
        "config": {"workload": f"{args.config}: {w.meta['desc']}", "recomputed_rows": n_R,
                   "rho_bp": w.rho_bp, "tokens": w.n_rows, "buffer_sets": n_sets},
        "roofline": {"kernel": "qcf_sparse_prefill_attn, recomputed rows (attn_w8_kernel + "
                               "attn_stream_merge_kernel)",
                     "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic(args.config, int(first.k.stride(0))),
                     "traffic_unit": "bytes per launch (HBM, calibrated rocprofv3 FETCH_SIZE + WRITE_SIZE)",
                     "flops_per_launch": flops, "avg_launch_ms": attn_ms,
                     "launch_ms_p10_p50_p90": [float(np.percentile(attn_all, q)) for q in (10, 50, 90)]},
        "ms_per_step_fused_scores_flow": ms_step_fused,
        # the step split as fusion kernels (re-position, fresh-row scatter, row attention) and
        # selector (probe attention, scores + top-k in the one call the step makes), from the
        # per-stage timings below
        "fusion_kernels_ms": stage_ms["rerope"] + stage_ms["scatter"] + stage_ms["attn"],
        "fusion_kernels_tokens_per_s": n_R / ((stage_ms["rerope"] + stage_ms["scatter"]
                                               + stage_ms["attn"]) * 1e-3),
        "selector_ms": stage_ms["probe_attn"] + stage_ms["scores_select"],
        "stage_ms": stage_ms,
        "paper_context": {
            "ttft_speedup_vs_full_prefill": 1.7, "ttft_speedup_vs_prophetkv": 1.5,
            "hardware": "2x NVIDIA H20 (SGLang, BF16, Triton recompute kernel)",
            "note": "end-to-end time-to-first-token ratios at matched quality from the paper's "
                    "evaluation; context only, not this metric"},
        "assemble_GBs": asm_gbs,
        "assemble_hbm_frac": asm_gbs / PEAK_HBM_GBS,
        "rerope_hbm": rerope,
    }

    if args.config == "c4" and not args.no_others:
        out["other_workloads"] = {name: workload_summary(name) for name in ("c2", "c5")}
        out["achievable"] = achievable_peaks()
        out["roofline"]["frac_of_achievable"] = achieved / out["achievable"]["mfma_bf16_loop"]["tflops"]
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def achievable_peaks(iters=10000):
    """What this part reaches on plain loops, beside the published peaks: the attention's bf16
    product instruction (v_mfma_f32_32x32x16_bf16) in a loop at the attention's occupancy, two
    waves per SIMD, on random operands (qcf_mfma_loop), with the clock of one block per XCD read
    from its counters; and a 512 MiB device-to-device copy."""
    import torch
    from paper_2606_05875_amd import qcf
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = 2 * n_cu
    ops = torch.randn(1 << 20, device="cuda").to(torch.bfloat16)
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(32, dtype=torch.int64, device="cuda")
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    qcf.qcf_mfma_loop(ops, sink, clocks, blocks, max(1, iters // 10))
    torch.cuda.synchronize()
    times = []
    for _ in range(3):
        a.record()
        qcf.qcf_mfma_loop(ops, sink, clocks, blocks, iters)
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
    ms = float(np.median(times))
    flops = blocks * 4 * iters * 16 * 32768
    tflops = flops / (ms * 1e-3) / 1e12
    c = clocks.view(8, 4).cpu().numpy().astype(np.float64)
    ghz = (c[:, 3] - c[:, 1]) / ((c[:, 2] - c[:, 0]) / 100e6) / 1e9
    x = torch.empty(128 << 20, dtype=torch.float32, device="cuda").uniform_()
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    a.record()
    for _ in range(10):
        y.copy_(x)
    b.record()
    torch.cuda.synchronize()
    gbs = 2 * x.numel() * 4 * 10 / (a.elapsed_time(b) * 1e-3) / 1e9
    del x, y
    return {"mfma_bf16_loop": {"tflops": tflops, "frac_of_peak": tflops / PEAK_BF16_TFLOPS, "ms": ms,
                               "clock_ghz_min_median_max": [float(ghz.min()), float(np.median(ghz)),
                                                            float(ghz.max())],
                               "occupancy": "2 waves per SIMD, 4 accumulators per wave, random bf16"},
            "device_copy": {"GBs": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS, "bytes": 2 * (512 << 20)}}


def workload_summary(name, steps=100, warmup=10):
    """Step time, selected tokens/s and recomputed-row attention share of the bf16 peak of one
    more workload, measured the headline's way (rotated buffer sets up to 512 MB, K whole steps
    between two events; the attention over events on its launch stream)."""
    import torch
    from paper_2606_05875_amd.step import FusionStep
    from paper_2606_05875_amd.workloads import make_workload

    w = make_workload(name)
    first = FusionStep(w)
    per_set = sum(t.numel() * t.element_size() for t in (first.k_pic, first.v_pic, first.q_new,
                                                         first.k_new, first.v_new, first.k, first.v))
    sets = [first] + [FusionStep(w) for _ in range(max(1, math.ceil(512e6 / per_set)) - 1)]
    for i in range(warmup):
        sets[i % len(sets)].run()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for i in range(steps):
        sets[i % len(sets)].run()
    b.record()
    torch.cuda.synchronize()
    ms_step = a.elapsed_time(b) / steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
    for i, (x, y) in enumerate(ev):
        s = sets[i % len(sets)]
        s.run_front()
        x.record()
        s.stage_attn()
        y.record()
        s.join()
    torch.cuda.synchronize()
    attn_ms = float(np.mean([x.elapsed_time(y) for x, y in ev]))
    R_pos = first.R_pos.cpu().numpy()
    achieved = attn_flops(first, R_pos) / (attn_ms * 1e-3) / 1e12
    res = {"workload": w.meta["desc"], "ms_per_step": ms_step,
           "tokens_per_s": int(R_pos.size) / (ms_step * 1e-3), "attn_ms": attn_ms,
           "attn_frac_bf16_peak": achieved / PEAK_BF16_TFLOPS, "buffer_sets": len(sets)}
    del sets, first
    torch.cuda.empty_cache()
    return res


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, budget_s):
    """The oracle's step on the host cores, on a bounded sample of the same workload.

    One oracle step without any attention row (re-position, probe, scores, selection,
    fused cache) plus one with the attention of m evenly spaced rows of R; the attention
    part is scaled to all of R by the visible-key count (its cost is proportional to it).
    m grows from 16 until the sampled step takes about ``budget_s`` / 2."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    t = time.perf_counter()
    base = oracle.fusion_step(w, attn_rows=np.zeros(0, np.int64))
    t_fixed = time.perf_counter() - t
    R = np.concatenate(base["R"])
    R_pos = np.concatenate(base["R_pos"]).astype(np.float64)
    m = 16
    while True:
        idx = np.unique(np.linspace(0, R.size - 1, min(m, R.size)).round().astype(np.int64))
        t = time.perf_counter()
        oracle.fusion_step(w, attn_rows=R[idx])
        t_sample = time.perf_counter() - t
        if t_sample > budget_s / 2 or idx.size == R.size or m >= 4096:
            break
        m *= 2
    t_attn = max(t_sample - t_fixed, 0.0) * float(np.sum(R_pos + 1)) / float(np.sum(R_pos[idx] + 1))
    sec = t_fixed + t_attn
    return {"value": R.size / sec, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"one oracle step without attention ({t_fixed:.2f} s) and one with the attention "
                       f"of {idx.size} of {R.size} recomputed rows ({t_sample:.2f} s); attention time "
                       f"scaled by visible keys to all rows: {sec:.1f} s per step"),
            "host_cpus": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
            "cpu_model": _cpu_model()}


if __name__ == "__main__":
    main()
