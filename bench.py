#!/usr/bin/env python3
"""Throughput of the STCA forward under request level batching on one MI355X.

One step = one stca_forward over the whole batch (per layer: the history K/V
projection fused into the multi-target attention, then the target update),
inputs already resident in HBM.  Prints one JSON line: targets scored per
second over the K timed steps of the headline workload (128 requests x 32
targets, L = 10240), the dominant kernel against its roofline (HIP events
recorded on the library's stream around every launch, in a second pass of K
steps so that the events stay out of the timed region), and the fp64 CPU
oracle timed on a bounded sample of the same workload.  Sub-records of the
same line: `ablation` (the headline batch in the instance-wise, non-RLB
layout, one target per request, materialised K/V, many targets per
request), `train_step` (forward + backward at the training window, with its
own roofline and CPU baseline) and `configs` (every workload: throughput,
roofline fraction and the non-RLB ablation).

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--quick]
                    [--backward [--sl]] [--paper]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2511_06077_amd import accounting, stca  # noqa: E402
from paper_2511_06077_amd import workload as W  # noqa: E402

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def reordered_requests(b: W.Batch, attn_form: int) -> np.ndarray:
    """Requests the library runs in the reordered form (its per-request rule,
    host offsets given, d_h = 32): every one when the form is forced or no
    request has more than 32 / h targets; otherwise, in the automatic choice,
    those with at most 32 / h targets; none in the standard form."""
    wl = b.wl
    m = b.n_tgt
    if attn_form == stca.STCA_ATTN_STANDARD or wl.d_model // wl.n_heads != 32:
        return np.zeros(m.shape, dtype=bool)
    cap = 32 // wl.n_heads
    live = m > 0
    if attn_form == stca.STCA_ATTN_REORDERED or (m[live] <= cap).all():
        return live
    return live & (m <= cap)


def kernel_work(label: str, b: W.Batch, es: int, attn_form: int = stca.STCA_ATTN_AUTO):
    """Algorithmic (flop, bytes) of one launch of a kernel, from the method's
    compulsory work (accounting.stage_costs) divided over launches."""
    wl = b.wl
    c = accounting.stage_costs(b.hist_len, b.n_tgt, wl.d_model, wl.n_layers, es)
    n = wl.n_layers
    d = wl.d_model
    L = b.hist_len.astype(np.float64)
    m = b.n_tgt.astype(np.float64)
    reord = reordered_requests(b, attn_form)
    if label == "proj":
        # all layers in one launch; rows of requests without targets still count
        Ls = float(b.hist_len.sum())
        return 4.0 * Ls * wl.d_model ** 2 * n, es * Ls * wl.d_model * (1 + 2 * n)
    if label == "attn":
        return c["attn"]["flop"] / n, c["attn"]["bytes"] / n
    if label in ("fused", "fused_wide"):
        # one layer: project the rows of the requests this launch serves
        # (X read once) and attend; units with up to 32 targets go to "fused"
        sel = (m > 0) & ~reord & ((m <= 32) if label == "fused" else (m > 32))
        return (4.0 * L[sel].sum() * d * d + 4.0 * (m[sel] * L[sel]).sum() * d,
                es * L[sel].sum() * d)
    if label == "reord_attn":
        # one layer of the reordered form (Eq. attn-optimized): scores X U^T and
        # P^T X over the m h (target, head) rows of each request, X read once
        return (4.0 * (L[reord] * m[reord]).sum() * d * wl.n_heads, es * L[reord].sum() * d)
    if label == "update":
        return c["update"]["flop"] / n, 0.0
    return 0.0, 0.0


def roofline_entry(label, ms, flop, byts, peak_tf):
    t_mfma = flop / (peak_tf * 1e12) if flop else 0.0
    t_hbm = byts / (PEAK_HBM_GBS * 1e9) if byts else 0.0
    if t_mfma >= t_hbm:
        ach = flop / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": ach, "peak": peak_tf, "unit": "TFLOP/s", "frac": ach / peak_tf,
                "traffic": None}
    ach = byts / (ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": ach, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": ach / PEAK_HBM_GBS,
            "traffic": None}


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE scaled by a plain copy's readings), or
    None when no summary covers this workload or the kernel source changed
    since the counters were taken."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.json")):
        rec = json.load(open(path))
        if rec.get("workload") != workload or kernel not in rec.get("kernels", {}):
            continue
        for src, sha in rec["sources"].items():
            if hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest() != sha:
                return None
        return rec["kernels"][kernel]["bytes"]
    return None


def cpu_baseline(wl: W.Workload, budget_s: float, backward: bool = False):
    """The fp64 oracle, as it is, on requests of the same workload taken in
    order until the time budget is spent: its forward, or (backward) its
    forward and hand-derived backward (all gradients)."""
    from oracle import stca_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    L, m = W.request_shapes(wl)
    done_t, done_r, spent = 0, 0, 0.0
    for r in range(wl.n_requests):
        sub = W.make_batch(wl, requests=[r], with_grad=backward, threads=1)
        inp = sub.f64()
        t0 = time.perf_counter()
        if backward:
            O.backward(inp, inp["grad_out"])
        else:
            O.forward(inp, keep=False)
        spent += time.perf_counter() - t0
        done_t += int(m[r])
        done_r += 1
        if spent >= budget_s:
            break
    what = "forward + backward" if backward else "forward"
    return {"value": done_t / spent, "unit": "targets trained/s" if backward else "targets/s", "cores": int(cores),
            "kind": "oracle",
            "sample": f"{what} of the first {done_r} of {wl.n_requests} requests of {wl.name} ({done_t} targets), "
                      f"{spent:.1f} s of fp64 CPU work"}


def settle(run, seconds: float) -> int:
    """Untimed steps for `seconds` of wall time before the warm-up proper: the
    GPU clock ramps up over the first tens of milliseconds of sustained work,
    which a few warm-up steps do not cover."""
    import torch
    n, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(8):
            run()
        n += 8
        torch.cuda.synchronize()
    return n


def plain_forward(db, steps: int, warmup: int) -> float:
    """The same K steps without per-kernel events: total milliseconds."""
    import torch
    stream = torch.cuda.current_stream(db.device)
    for _ in range(warmup):
        db.forward()
    torch.cuda.synchronize(db.device)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        db.forward()
    end.record(stream)
    torch.cuda.synchronize(db.device)
    return start.elapsed_time(end)


def timed_forward(db, steps: int, warmup: int):
    import torch
    dev = db.device
    stream = torch.cuda.current_stream(dev)
    for _ in range(warmup):
        db.forward()
    torch.cuda.synchronize(dev)
    nl = stca.stca_forward_launch_count(db.dims, db.batch)
    evs = [stca.HipEvents(nl + 1) for _ in range(steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize(dev)
    start.record(stream)
    for k in range(steps):
        stca.stca_forward_profiled(db.dims, db.batch, db.hist, db.tgt, db.weights, db.out, None, db.ws,
                                   db.ws_bytes, stream.cuda_stream, evs[k].ev, evs[k].labels)
    end.record(stream)
    torch.cuda.synchronize(dev)
    total_ms = start.elapsed_time(end)
    per = {}
    for e in evs:
        for k in range(nl):
            lab = e.label(k)
            per.setdefault(lab, []).append(e.elapsed_ms(k, k + 1))
    for e in evs:
        e.close()
    return total_ms, per


def kernel_table(per: dict, b, steps: int, es: int, peak_tf: float, attn_form: int = stca.STCA_ATTN_AUTO) -> dict:
    """Per-kernel durations (HIP events) with their algorithmic rates."""
    kernels = {}
    for lab, v in per.items():
        launches = len(v) // steps
        ms = float(np.mean(v))
        flop, byts = kernel_work(lab, b, es, attn_form)
        ent = {"launches_per_step": launches, "ms_per_launch": ms, "ms_per_step": ms * launches}
        if flop or byts:
            ent.update({"tflops": flop / (ms * 1e-3) / 1e12, "gbs": byts / (ms * 1e-3) / 1e9,
                        "mfma_frac": flop / (ms * 1e-3) / 1e12 / peak_tf,
                        "hbm_frac": byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS})
        kernels[lab] = ent
    return kernels


def design_bound_ms(b, es: int, peak_tf: float) -> float:
    """The fused design's own bound: per layer X read once and the K/V
    projection plus attention at the matrix-core peak (K and V never reach
    HBM), plus the target update at peak."""
    wl = b.wl
    L = b.hist_len[b.n_tgt > 0].astype(np.float64)
    m = b.n_tgt[b.n_tgt > 0].astype(np.float64)
    dm = wl.d_model
    c = accounting.stage_costs(b.hist_len, b.n_tgt, dm, wl.n_layers, es)
    fused_flop = wl.n_layers * (4.0 * L.sum() * dm * dm + 4.0 * (m * L).sum() * dm)
    fused_bytes = wl.n_layers * es * L.sum() * dm
    return (max(fused_flop / (peak_tf * 1e12), fused_bytes / (PEAK_HBM_GBS * 1e9))
            + c["update"]["flop"] / (peak_tf * 1e12)) * 1e3


def measure_forward(db, steps: int, warmup: int, settle_s: float, events: bool = True) -> dict:
    """Settling steps, W warm-up steps, K timed plain steps (the value), then
    (events) K more steps with a HIP event around every launch for the
    per-kernel table and the dominant kernel's roofline."""
    b, wl = db.b, db.b.wl
    es = 2 if wl.dtype == "bf16" else 4
    peak_tf = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    n_settle = settle(db.forward, settle_s) if settle_s > 0 else 0
    ms = plain_forward(db, steps, warmup) / steps
    out = {"workload": wl.name, "requests": int(b.n_requests), "targets": int(b.n_tgt_total),
           "history_rows": int(b.n_hist), "ms_per_step": ms, "targets_per_s": b.n_tgt_total / (ms * 1e-3),
           "settle_steps": n_settle, "launches": stca.stca_forward_launch_count(db.dims, db.batch)}
    if not events:
        return out
    ev_total, per = timed_forward(db, steps, 1)
    af = db.dims.attn_form
    kernels = kernel_table(per, b, steps, es, peak_tf, af)
    dom = max((k for k in kernels if kernel_work(k, b, es, af) != (0.0, 0.0)),
              key=lambda k: kernels[k]["ms_per_step"])
    flop, byts = kernel_work(dom, b, es, af)
    roof = roofline_entry(dom, kernels[dom]["ms_per_launch"], flop, byts, peak_tf)
    roof["kernel"] = dom
    roof["traffic"] = measured_traffic(wl.name, dom)
    c = accounting.stage_costs(b.hist_len, b.n_tgt, wl.d_model, wl.n_layers, es)
    path_ms = sum(max(v["flop"] / (peak_tf * 1e12), v["bytes"] / (PEAK_HBM_GBS * 1e9)) for v in c.values()) * 1e3
    dms = design_bound_ms(b, es, peak_tf)
    out.update({"roofline": roof, "kernels": kernels, "ms_per_step_with_kernel_events": ev_total / steps,
                "path_roofline": {"ms": path_ms, "frac": path_ms / ms,
                                  "targets_per_s": b.n_tgt_total / (path_ms * 1e-3)},
                "fused_design_roofline": {"ms": dms, "frac": dms / ms,
                                          "targets_per_s": b.n_tgt_total / (dms * 1e-3)}})
    return out


def instance_wise(db, backward: bool = False, **forms):
    """The same samples in the instance-wise layout of App. A.3: every target
    becomes a request of its own carrying a copy of its request's history
    (the non-RLB layout, history re-encoded per target).  Built on the GPU by
    a row gather from the request-level batch; targets (and upstream
    gradients) keep their order."""
    import torch
    from paper_2511_06077_amd.device import DeviceBatch
    b = db.b
    reps = b.n_tgt.astype(np.int64)
    L = np.repeat(b.hist_len.astype(np.int64), reps)
    ones = np.ones(int(reps.sum()), dtype=np.int64)
    hoff = W.offsets(L)
    shift = np.repeat(b.hist_off[:-1].astype(np.int64), reps) - hoff[:-1].astype(np.int64)
    dev = db.device
    idx = torch.arange(int(hoff[-1]), device=dev, dtype=torch.int64)
    idx += torch.repeat_interleave(torch.from_numpy(shift).to(dev), torch.from_numpy(L).to(dev))
    hist = db.hist.index_select(0, idx)
    del idx
    nb = W.Batch(b.wl, np.repeat(b.requests, reps), L, ones, hoff, W.offsets(ones), None, None, b.weights, None)
    return DeviceBatch.from_tensors(nb, hist, db.tgt, db.w, device=dev, backward=backward, **forms)


def non_rlb_forward(db, steps: int) -> dict:
    """The instance-wise layout of the same batch, timed with the same
    kernels (standard attention form) and with the form chosen automatically
    (one target per request: the reordered attention)."""
    import torch
    out = {}
    for key, attn in (("standard_form", "standard"), ("auto_form", "auto")):
        nb = instance_wise(db, attn=attn)
        ms = plain_forward(nb, steps, 2) / steps
        out[key] = {"requests": int(nb.b.n_requests), "history_rows": int(nb.b.n_hist), "ms_per_step": ms,
                    "targets_per_s": nb.b.n_tgt_total / (ms * 1e-3),
                    "launches": stca.stca_forward_launch_count(nb.dims, nb.batch)}
        del nb
        torch.cuda.empty_cache()
    return out


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=W.HEADLINE, choices=sorted(W.WORKLOADS))
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget per baseline (0: skip)")
    ap.add_argument("--settle-seconds", type=float, default=1.0,
                    help="untimed steps for this long before the warm-up (GPU clock ramp)")
    ap.add_argument("--quick", action="store_true",
                    help="only the headline record (no ablation, training-step or per-config sub-records)")
    ap.add_argument("--backward", action="store_true",
                    help="instead: forward + backward steps (the training window workload by default)")
    ap.add_argument("--sl", action="store_true",
                    help="with --backward: a stochastic-length batch (Beta lengths, alpha 0.02, L_avg 2048 of 10240)")
    ap.add_argument("--paper", action="store_true",
                    help="instead: the paper-exact stack (stca_forward_paper: SwiGLU + LayerNorm history transform "
                         "per layer, query fusion, head token z) on the same workload")
    ap.add_argument("--kv", default="auto", choices=["auto", "fused", "materialize"],
                    help="history K/V form of the headline record (auto: the library's choice)")
    ap.add_argument("--attn", default="auto", choices=["auto", "standard", "reordered"],
                    help="attention form of the headline record (auto: the library's choice)")
    ap.add_argument("--bwd", default="auto", choices=["auto", "fused", "reordered", "generic"],
                    help="with --backward: the backward form (auto: the library's choice)")
    ap.add_argument("--copy-gib", type=float, default=0.0,
                    help="instead: time a plain device-to-device copy of this many GiB (HBM counter calibration)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (the STCA path needs no collectives; requests shard with "
              f"zero communication); got --gpus {args.gpus}, WORLD_SIZE={world}", file=sys.stderr)
        return 2

    import torch
    if args.copy_gib > 0:
        return copy_calibration(args)
    if args.backward:
        rec = train_record(args, W.WORKLOADS[args.workload if args.workload != W.HEADLINE
                                             else "train_bf16_R256_m16_L2048_d256"], args.steps, args.warmup,
                           sl=args.sl)
        print(json.dumps(rec), flush=True)
        return 0
    if args.paper:
        return paper_step(args)
    from paper_2511_06077_amd.device import DeviceBatch
    wl = W.WORKLOADS[args.workload]
    t0 = time.time()
    b = W.make_batch(wl, with_grad=False)
    log(f"[bench] generated {wl.name}: {b.n_hist} history rows, {b.n_tgt_total} targets ({time.time() - t0:.1f} s)")
    db = DeviceBatch(b, device="cuda:0", kv=args.kv, attn=args.attn)
    log(f"[bench] workspace {db.ws_bytes / 2**30:.2f} GiB; path {stca.stca_path(db.dims)}")
    # the timed region: W warm-up steps, then exactly K plain steps; per-kernel
    # durations come from the same K steps again with a HIP event recorded on
    # the library's stream around every launch (the events themselves add a
    # few microseconds per launch, so they stay out of the timed region)
    head = measure_forward(db, args.steps, args.warmup, args.settle_seconds)
    ms_step = head["ms_per_step"]
    log(f"[bench] {args.steps} steps: {ms_step:.3f} ms/step; {head['ms_per_step_with_kernel_events']:.3f} "
        f"with per-kernel events")
    rec = {
        "metric": "targets scored/sec, STCA forward",
        "value": head["targets_per_s"],
        "unit": "targets/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "requests": wl.n_requests,
                   "targets_per_request": wl.n_targets or list(wl.tgt_range),
                   "hist_len": wl.hist_len or list(wl.hist_range), "d_model": wl.d_model,
                   "heads": wl.n_heads, "layers": wl.n_layers, "ffn_hidden": wl.ffn_hidden,
                   **({"kv_form": args.kv} if args.kv != "auto" else {}),
                   **({"attn_form": args.attn} if args.attn != "auto" else {})},
        "roofline": head["roofline"],
        "path_roofline": head["path_roofline"],
        "fused_design_roofline": head["fused_design_roofline"],
        "kernels": head["kernels"],
        "ms_per_step_with_kernel_events": head["ms_per_step_with_kernel_events"],
        "settle_steps": head["settle_steps"],
    }
    sub_steps = max(5, args.steps // 5)
    if not args.quick:
        log("[bench] ablation")
        rec["ablation"] = ablation(db, args, sub_steps)
    del db
    torch.cuda.empty_cache()
    if not args.quick:
        log("[bench] training step")
        rec["train_step"] = train_record(args, W.WORKLOADS["train_bf16_R256_m16_L2048_d256"], sub_steps,
                                         max(2, args.warmup // 2), with_non_rlb=True)
        log("[bench] per-configuration records")
        rec["configs"] = config_records(args, rec, sub_steps)
    if args.cpu_seconds > 0:
        log("[bench] timing the CPU oracle")
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(rec), flush=True)
    return 0


def config_records(args, rec: dict, steps: int) -> dict:
    """Every workload: throughput, the dominant kernel's roofline fraction,
    the fused design's bound, and the same batch in the instance-wise
    (non-RLB) layout.  The headline and training-window entries restate the
    line's own measurements."""
    import torch
    from paper_2511_06077_amd.device import DeviceBatch
    out = {}
    for name in ("tiny_f32_R4_m4_L256_d64", "uniform_bf16_R64_m16_L1024_d128",
                 "ragged_bf16_R256_L512-10240_m1-64_d256"):
        wl = W.WORKLOADS[name]
        db = DeviceBatch(W.make_batch(wl, with_grad=False), device="cuda:0")
        r = measure_forward(db, steps, 3, 0.2)
        r.pop("kernels")
        nr = instance_wise(db, attn="standard")
        ms = plain_forward(nr, steps, 2) / steps
        r["non_rlb"] = {"requests": int(nr.b.n_requests), "history_rows": int(nr.b.n_hist), "ms_per_step": ms,
                        "targets_per_s": nr.b.n_tgt_total / (ms * 1e-3), "form": "standard attention, same kernels"}
        r["rlb_gain"] = ms / r["ms_per_step"]
        out[name] = r
        del db, nr
        torch.cuda.empty_cache()
        log(f"[bench] {name}: {r['ms_per_step']:.3f} ms/step, non-RLB {ms:.3f} ms/step")
    head = {k: rec[k] for k in ("ms_per_step", "roofline", "path_roofline", "fused_design_roofline")}
    head["targets_per_s"] = rec["value"]
    nr = rec["ablation"]["non_rlb"]["standard_form"]
    head["non_rlb"] = dict(nr, form="standard attention, same kernels")
    head["rlb_gain"] = nr["ms_per_step"] / rec["ms_per_step"]
    out[rec["config"]["workload"]] = head
    t = rec["train_step"]
    out[t["config"]["workload"]] = dict({k: t[k] for k in ("ms_per_step", "roofline", "non_rlb", "rlb_gain")},
                                        targets_per_s=t["value"], step="forward + backward")
    return out


def paper_kernel_work(label: str, b: W.Batch):
    """Algorithmic (flop, bytes) of one launch of a kernel of the paper-exact
    stack: swiglu_ln = one layer's SwiGLU block (u, v and o products, 6 d F
    flop per history row) and LayerNorm over every history row, reading X and
    writing the transformed history once (bf16); fused = that layer's K/V
    projection of the transformed history and the attention (as the standard
    stack's fused kernel)."""
    wl = b.wl
    d, F = wl.d_model, wl.ffn_hidden
    Lall = float(b.hist_len.sum())
    L = b.hist_len.astype(np.float64)
    m = b.n_tgt.astype(np.float64)
    sel = (m > 0) & (m <= 32)
    if label == "swiglu_ln":
        return 6.0 * Lall * d * F, 2.0 * Lall * d * 2
    if label == "fused":
        return 4.0 * L[sel].sum() * d * d + 4.0 * (m[sel] * L[sel]).sum() * d, 2.0 * L[sel].sum() * d
    return 0.0, 0.0


def paper_step(args) -> int:
    """The paper-exact stack's forward (stca_forward_paper) on the workload:
    per layer the history's SwiGLU + LayerNorm transform (fused MFMA kernel),
    the fused projection + attention over it, and the target side (query
    fusion with W_C, SwiGLU + LayerNorm, head token z).  Same timing protocol
    as the standard stack: settling steps, W warm-up, K timed plain steps,
    then K steps with per-kernel HIP events."""
    import torch
    from paper_2511_06077_amd.device import PaperDeviceBatch
    wl = W.WORKLOADS[args.workload]
    b = W.make_batch(wl, with_grad=False)
    db = PaperDeviceBatch(b, W.make_paper_weights(wl), device="cuda:0")
    log(f"[bench] paper stack {wl.name}: workspace {db.ws_bytes / 2**30:.2f} GiB")
    n_settle = settle(db.forward, args.settle_seconds)
    ms_step = plain_forward(db, args.steps, args.warmup) / args.steps
    dev = db.device
    stream = torch.cuda.current_stream(dev)
    nl = stca.stca_paper_launch_count(db.dims, db.batch)
    evs = [stca.HipEvents(nl + 1) for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    for k in range(args.steps):
        stca.stca_forward_paper_profiled(db.dims, db.batch, db.hist, db.tgt, db.weights, db.z, None, db.ws,
                                         db.ws_bytes, stream.cuda_stream, evs[k].ev, evs[k].labels)
    torch.cuda.synchronize(dev)
    per = {}
    for e in evs:
        for k in range(nl):
            per.setdefault(e.label(k), []).append(e.elapsed_ms(k, k + 1))
        e.close()
    log(f"[bench] paper stack {args.steps} steps: {ms_step:.3f} ms/step")
    kernels = {}
    for lab, v in per.items():
        launches = len(v) // args.steps
        ms = float(np.mean(v))
        flop, byts = paper_kernel_work(lab, b)
        ent = {"launches_per_step": launches, "ms_per_launch": ms, "ms_per_step": ms * launches}
        if flop or byts:
            ent.update({"tflops": flop / (ms * 1e-3) / 1e12, "gbs": byts / (ms * 1e-3) / 1e9,
                        "mfma_frac": flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                        "hbm_frac": byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS})
        kernels[lab] = ent
    dom = max((k for k in kernels if paper_kernel_work(k, b) != (0.0, 0.0)), key=lambda k: kernels[k]["ms_per_step"])
    flop, byts = paper_kernel_work(dom, b)
    roof = roofline_entry(dom, kernels[dom]["ms_per_launch"], flop, byts, PEAK_BF16_TFLOPS)
    roof["kernel"] = dom
    roof["traffic"] = None
    n = wl.n_layers
    bound_ms = sum(max(paper_kernel_work(k, b)[0] / (PEAK_BF16_TFLOPS * 1e12),
                       paper_kernel_work(k, b)[1] / (PEAK_HBM_GBS * 1e9)) for k in ("swiglu_ln", "fused")) * n * 1e3
    rec = {"metric": "targets scored/sec, STCA forward (paper-exact stack)",
           "value": b.n_tgt_total / (ms_step * 1e-3), "unit": "targets/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if wl.dtype == "bf16" else "f32", "data": "synthetic",
           "config": {"workload": wl.name + "_paper", "requests": wl.n_requests,
                      "targets_per_request": wl.n_targets or list(wl.tgt_range),
                      "hist_len": wl.hist_len or list(wl.hist_range), "d_model": wl.d_model, "heads": wl.n_heads,
                      "layers": n, "ffn_hidden": wl.ffn_hidden},
           "roofline": roof,
           "history_side_roofline": {"ms": bound_ms, "frac": bound_ms / ms_step},
           "kernels": kernels, "settle_steps": n_settle}
    print(json.dumps(rec), flush=True)
    return 0


def backward_phase_work(label: str, b: W.Batch, fused: bool, reordered: bool = False):
    """Algorithmic (flop, bytes, peak TFLOP/s) of one occurrence of a backward
    phase (stca_backward_profiled's markers), as the kernels are designed.

    reordered (d = 128/256, at most 128 / n_heads targets per request): per
    layer one pass over X forms S = X U^T, dP = X H^T, Z = dE^T X and
    Y = P^T X over the request's m H (target, head) pairs (8 L m H d flop)
    and writes [ln2 dE | P] (bf16, 4 L m H bytes); dq, dW_K, dW_V come from Z
    and Y (6 m d^2 flop); dX = E W_r after the layers (4 n L m H d flop,
    reads every layer's E, writes dX in fp32).

    fused (requests of at most 32 targets): the recomputed attention and the
    attention backward each project the history inside the kernel (X read
    once per layer; K/V projection 4 L d^2 flop), on the bf16 matrix cores;
    the attention backward writes dK | dV once, row-major bf16 (read as they
    are by both history-side products after the layers); the target
    side (recomputation and gradients) runs on bf16 operands.  Otherwise:
    the K|V product with fp32 output, the exact fp32 attention on the fp32
    MFMA (157.3 TFLOP/s), target-side products in fp32 where they decide ReLU
    gates.  Either way every layer's [dW_K | dW_V] and dX are formed once
    after the layers."""
    wl = b.wl
    d, F, n = wl.d_model, wl.ffn_hidden, wl.n_layers
    Ls = float(b.hist_len[b.n_tgt > 0].sum())
    mL = float((b.n_tgt.astype(np.float64) * b.hist_len).sum())
    mt = float(b.n_tgt.sum())
    H = wl.n_heads
    if reordered:
        if label == "attn_bwd":
            return 8 * H * mL * d, 2 * Ls * d + 4 * H * mL, PEAK_BF16_TFLOPS
        if label == "kv_grads":
            return 6 * mt * d * d, 4 * H * mt * d + 8 * mt * d, PEAK_BF16_TFLOPS
        if label == "dx":
            return 4 * n * H * mL * d, n * 4 * H * mL + 4 * Ls * d, PEAK_BF16_TFLOPS
    if label == "kv_gemm":
        return 4 * Ls * d * d, 2 * Ls * d + 8 * Ls * d, PEAK_BF16_TFLOPS
    if label == "dw_kv":  # X (or X^T) read once, every layer's dK | dV (or its transpose)
        return n * 4 * Ls * d * d, 2 * Ls * d + n * 4 * Ls * d, PEAK_BF16_TFLOPS
    if label == "dx":  # every layer's dK | dV read, dX written once (fp32)
        return n * 4 * Ls * d * d, n * 4 * Ls * d + 4 * Ls * d, PEAK_BF16_TFLOPS
    if label == "attn_fwd":
        if fused:
            return 4 * Ls * d * d + 4 * mL * d, 2 * Ls * d, PEAK_BF16_TFLOPS
        return 4 * mL * d, 8 * Ls * d, PEAK_FP32_TFLOPS
    if label == "attn_bwd":
        if fused:
            return 4 * Ls * d * d + 10 * mL * d, 2 * Ls * d + 4 * Ls * d, PEAK_BF16_TFLOPS
        return 10 * mL * d, 8 * Ls * d + 8 * Ls * d, PEAK_FP32_TFLOPS
    if label == "target_gemm":
        if fused:
            # per layer: the recomputation (W_O, W_1, W_2, W_Q) and the
            # gradient products (dW2, dH, dW1, du, dWo, da, dWq, ds), over
            # 13 markers for 4 layers (one initial, two per layer after)
            per_layer = 2 * mt * (2 * d * d + 2 * d * F) + 2 * mt * (4 * d * F + 4 * d * d)
            return per_layer * n / (1 + 3 * n), 0.0, PEAK_BF16_TFLOPS
        # per layer over 4 markers: fp32 products q, o (d x d) and FFN1, FFN2
        # (d x F); bf16 products dW2, dH, dW1, du (d x F) and dWo, da, dWq, ds
        # (d x d), counted at the fp32 peak by their time ratio
        f32 = 2 * mt * (2 * d * d + 2 * d * F)
        b16 = 2 * mt * (4 * d * F + 4 * d * d)
        return (f32 + b16 * PEAK_FP32_TFLOPS / PEAK_BF16_TFLOPS) / 4, 0.0, PEAK_FP32_TFLOPS
    return 0.0, 0.0, 0.0


def train_record(args, wl: W.Workload, steps: int, warmup: int, sl: bool = False,
                 with_non_rlb: bool = False) -> dict:
    """Forward + backward of the training window: one step = the forward then
    the backward (all gradients) over the whole batch, inputs resident
    (stca_forward_train + stca_backward_record where the batch qualifies,
    else stca_forward + stca_backward).  The phases are then timed with HIP
    events in a pass of the recomputing backward (stca_backward_profiled),
    whose attention-backward phase is the same kernels on the same inputs as
    in the two-call step; that phase's roofline is the record's `roofline`.
    The CPU baseline is the oracle's forward and hand-derived backward."""
    import torch
    from paper_2511_06077_amd.device import DeviceBatch, to_device
    sl_info = None
    if sl:
        # stochastic-length batch: full histories of L_infer = 10240 rows cut
        # to Beta-sampled temporal suffixes (alpha = 0.02, L_avg = 2048)
        from paper_2511_06077_amd import sl as SL
        full_wl = W.Workload(wl.name + "_L10240", wl.n_requests, wl.d_model, wl.n_heads, wl.n_layers, wl.dtype,
                             wl.seed, hist_len=10240, n_targets=wl.n_targets, backward=True)
        t0 = time.time()
        full = W.make_batch(full_wl, with_grad=True)
        b, sl_info = SL.sl_batch(full, wl.seed, alpha=0.02, l_min=8, l_avg=2048, l_max=10240)
        del full
        log(f"[bench] stochastic-length batch: {b.n_hist} of {wl.n_requests * 10240} rows kept "
            f"({time.time() - t0:.1f} s)")
        wl = b.wl
    else:
        b = W.make_batch(wl, with_grad=True)
    db = DeviceBatch(b, device="cuda:0", backward=True, bwd=getattr(args, "bwd", "auto"))
    dout = to_device(b.grad_out, "cuda:0")

    def timed_step(dbx, k, w):
        use_rec = dbx.record is not None

        def fwd():
            dbx.forward_train() if use_rec else dbx.forward()

        def bwd():
            dbx.backward(dout, use_record=use_rec)
        for _ in range(w):
            fwd()
            bwd()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        # forward and backward timed separately (each backward reads the record
        # of the last forward_train, which stays valid across backward calls)
        e[0].record(stream)
        for _ in range(k):
            fwd()
        e[1].record(stream)
        for _ in range(k):
            bwd()
        e[2].record(stream)
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / k, e[1].elapsed_time(e[2]) / k, use_rec

    settle(lambda: (db.forward(), db.backward(dout)), args.settle_seconds)
    fwd, bwd, use_rec = timed_step(db, steps, warmup)
    ms = fwd + bwd
    stream = torch.cuda.current_stream()
    # the recomputing backward (what stca_backward alone costs), for reference
    e2 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    e2[0].record(stream)
    for _ in range(steps):
        db.backward(dout)
    e2[1].record(stream)
    torch.cuda.synchronize()
    bwd_recompute = e2[0].elapsed_time(e2[1]) / steps
    # phases of the recomputing backward (stca_backward_profiled), timed on
    # the library's stream
    g = db.backward(dout)
    dw = stca.wgrads(g["dwq"], g["dwk"], g["dwv"], g["dwo"], g["dw1"], g["dw2"])
    nl = stca.stca_backward_launch_count(db.dims, db.batch)
    per = {}
    for _ in range(steps):
        ev = stca.HipEvents(nl + 1)
        stca.stca_backward_profiled(db.dims, db.batch, db.hist, db.tgt, db.weights, dout, g["dhist"], g["dtgt"],
                                    dw, db.bws, db.bws_bytes, stream.cuda_stream, ev.ev, ev.labels)
        torch.cuda.synchronize()
        for k in range(nl):
            per.setdefault(ev.label(k), []).append(ev.elapsed_ms(k, k + 1))
        ev.close()
    fused = "kv_gemm" not in per  # the attention kernels project the history themselves
    reordered = "kv_grads" in per  # the reordered form: no K, V, dK, dV
    phases = {}
    for lab, v in per.items():
        occ = len(v) // steps
        t = float(np.mean(v))
        ent = {"per_step": occ, "ms_each": t, "ms_per_step": t * occ}
        flop, byts, peak = backward_phase_work(lab, b, fused, reordered)
        if flop:
            ent.update({"tflops": flop / (t * 1e-3) / 1e12, "gbs": byts / (t * 1e-3) / 1e9,
                        "mfma_frac": flop / (t * 1e-3) / 1e12 / peak, "hbm_frac": byts / (t * 1e-3) / 1e9 / PEAK_HBM_GBS})
        phases[lab] = ent
    dom = max((k for k in phases if backward_phase_work(k, b, fused, reordered)[0]), key=lambda k: phases[k]["ms_per_step"])
    flop, byts, peak = backward_phase_work(dom, b, fused, reordered)
    roof = roofline_entry(dom, phases[dom]["ms_each"], flop, byts, peak)
    roof["kernel"] = dom
    roof["traffic"] = measured_traffic(wl.name, dom) if not sl else None
    bound_ms = sum(max(f / (pk * 1e12), by / (PEAK_HBM_GBS * 1e9)) * phases[k]["per_step"] * 1e3
                   for k in phases for f, by, pk in [backward_phase_work(k, b, fused, reordered)] if f)
    rec = {
        "metric": "targets trained/sec, STCA forward+backward", "value": b.n_tgt_total / (ms * 1e-3),
        "unit": "targets/s", "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": wl.name, "requests": wl.n_requests, "targets_per_request": wl.n_targets,
                   "hist_len": wl.hist_len, "d_model": wl.d_model, "heads": wl.n_heads, "layers": wl.n_layers,
                   **({"bwd_form": args.bwd} if getattr(args, "bwd", "auto") != "auto" else {})},
        "stochastic_length": sl_info,
        "training_record": use_rec, "forward_ms": fwd, "backward_ms": bwd,
        "backward_recomputing_ms": bwd_recompute, "roofline": roof,
        "backward_phase_bound_ms": bound_ms, "backward_phase_bound_frac": bound_ms / bwd_recompute,
        "backward_phases": phases}
    if with_non_rlb:
        nr = instance_wise(db, backward=True)
        f2, b2, rec2 = timed_step(nr, max(2, steps // 4), 1)
        rec["non_rlb"] = {"requests": int(nr.b.n_requests), "history_rows": int(nr.b.n_hist),
                          "ms_per_step": f2 + b2, "forward_ms": f2, "backward_ms": b2, "training_record": rec2,
                          "targets_per_s": nr.b.n_tgt_total / ((f2 + b2) * 1e-3)}
        rec["rlb_gain"] = (f2 + b2) / ms
        del nr
    del db
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0 and not sl:
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds, backward=True)
    return rec


def copy_calibration(args) -> int:
    """A plain copy of known size: reads and writes args.copy_gib GiB per
    launch, so HBM byte counters read on it give their scale."""
    import torch
    n = int(args.copy_gib * 2**30) // 4
    src = torch.randn(n, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    print(json.dumps({"copy_bytes_each_way": n * 4, "ms_per_copy": ms,
                      "gbs_read_plus_write": 2 * n * 4 / (ms * 1e-3) / 1e9}), flush=True)
    return 0


def ablation(db, args, steps: int) -> dict:
    """The headline batch in other layouts and forms: (a) the instance-wise
    (non-RLB) layout, every target its own request with a copy of the
    history (App. A.3), with the same kernels and with the automatic form;
    (b) one target per request, reordered (App. A.2.2) and standard form;
    (c) K/V materialised by one GEMM and streamed, and the whole batch in the
    reordered form (Eq. attn-optimized, units of up to 256 rows (t, j));
    (d) the same number of targets as 16 requests of 256 (K/V written once,
    read once per 128 targets) against the fused form."""
    import torch
    from paper_2511_06077_amd.device import DeviceBatch
    wl = db.b.wl
    out = {"non_rlb": non_rlb_forward(db, max(3, steps // 2))}
    out["rlb_gain"] = out["non_rlb"]["standard_form"]["ms_per_step"] / (plain_forward(db, steps, 2) / steps)
    for key, forms in (("materialized_kv", {"kv": "materialize"}), ("reordered_form", {"attn": "reordered"})):
        try:
            dm = DeviceBatch(db.b, device="cuda:0", **forms)
        except stca.StcaError as e:  # a form the batch does not admit
            out[key] = {"unsupported": str(e)}
            continue
        ms, per = timed_forward(dm, steps, 1)
        ms /= steps
        out[key] = {"ms_per_step": ms, "targets_per_s": dm.b.n_tgt_total / (ms * 1e-3),
                    "kernels_ms_per_step": {k: float(np.sum(v)) / steps for k, v in per.items()}}
        del dm
        torch.cuda.empty_cache()
    if wl.n_targets > 1 and wl.hist_range is None:
        one = W.Workload(wl.name + "_m1", wl.n_requests, wl.d_model, wl.n_heads, wl.n_layers, wl.dtype, wl.seed,
                         hist_len=wl.hist_len, n_targets=1)
        bo = W.make_batch(one)
        for key, mode in (("one_target_per_request", "auto"), ("one_target_per_request_standard", "standard")):
            d1 = DeviceBatch(bo, device="cuda:0", attn=mode)
            ms = plain_forward(d1, steps, 2) / steps
            out[key] = {"ms_per_step": ms, "targets_per_s": one.n_requests / (ms * 1e-3),
                        "launches": stca.stca_forward_launch_count(d1.dims, d1.batch)}
            del d1
            torch.cuda.empty_cache()
        many = W.Workload(wl.name + "_m256", max(1, wl.n_requests * wl.n_targets // 256), wl.d_model, wl.n_heads,
                          wl.n_layers, wl.dtype, wl.seed, hist_len=wl.hist_len, n_targets=256)
        bm = W.make_batch(many)
        for key, mode in (("many_targets_per_request", "auto"), ("many_targets_per_request_fused", "fused")):
            d2 = DeviceBatch(bm, device="cuda:0", kv=mode)
            ms = plain_forward(d2, steps, 2) / steps
            out[key] = {"requests": many.n_requests, "targets": bm.n_tgt_total, "ms_per_step": ms,
                        "targets_per_s": bm.n_tgt_total / (ms * 1e-3),
                        "launches": stca.stca_forward_launch_count(d2.dims, d2.batch)}
            del d2
            torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    sys.exit(main())
