#!/usr/bin/env python3
"""LinSimp forward + backward throughput on one MI355X.

Workload: the 16k-context layer (B=2, H=16, n=16384, d=m=128, w=64; bf16
inputs, float32 state), synthetic seeded inputs resident in HBM.  One step is
the whole hot path: forward (key feature map, chunk states, chunk scan,
anchor-window readout) and backward (query sweeps, state sweep, reverse scan,
key side) on the same batch; the backward reuses the boundary states the
forward left in the shared workspace.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--head | --decode] [--workload NAME]

With --head the step is the full head instead of the core: L2 normalisation
and query temperature, core, gated RMSNorm (per-head gate), and the backward
of all three; the line then also reports the streaming head kernels against
the HBM peak (`head_streams`).

--workload runs the same step on another forward + backward workload of
paper_2608_09307_amd/workloads.py (the 64k stress shape, or the 2k-token layer
the paper times); the default line is the 16k layer.

With --decode the line is the autoregressive path instead (256 sequences x
16 heads, d = m = 128, w = 64, after an 8192-token prefix): decode steps per
second over all sequences, the decode kernel against the HBM peak, and the
prefill and 16-token chunked decode times.  The default line carries the same
measurements as its `decode` object, taken in the same run after the timed
forward + backward steps (--no-decode leaves them out).

Prints one JSON line.  `value` is tokens/s (B*n per step time).  `roofline`
reports the dominant kernel (largest share of the timed region) against the
bf16 matrix-core peak, from HIP events recorded around every library kernel
on its stream during the timed steps.  `cpu_baseline` times the float64 oracle
on host cores on a causal prefix of one (batch, head) sequence, and in `extra`
on the single f32 head, the 2k-token layer's forward and the decode step.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

WORKLOAD = "layer16k_bf16"
PEAK_BF16_TFLOPS = 2500.0          # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0              # MI355X HBM3E peak
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_layer16k_bf16.json")
DECODE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_decode_s256_h16.json")


def anchor_rows(n, w):
    """sum_i min(i+1, w): (row, anchor) pairs of one sequence."""
    if n <= w:
        return n * (n + 1) // 2
    return w * (w + 1) // 2 + (n - w) * w


def kernel_flops(wl):
    """Algorithmic matrix-core flops per launch of each hot kernel (2 flops per
    multiply-add).  Forward readout: logits (D) + readout (Dv + 1 for the
    normaliser) per (row, anchor) pair and feature; backward: the five anchor
    contractions (logits, readout, dpsi, dz, dM) = 2D + 3Dv, split across the
    kernels that perform them."""
    ar = wl.B * wl.H * anchor_rows(wl.n, wl.w)
    f = 2 * wl.m * ar
    return {
        "fwd_readout": f * (wl.D + wl.Dv + 1),
        "bwd_du": f * (wl.D + wl.Dv),
        "bwd_dqdr": f * (wl.Dv + wl.D),
        "bwd_state": f * wl.Dv,
    }


def decode_step_bytes(wl, es=2):
    """Algorithmic HBM bytes of one decode step over all (sequence, head)
    pairs: M and a read and written (float32) with the frame, both anchor
    rings read and one slot of each written, the token's q, k, v, r, u in and
    the output row out."""
    D, Dv, m, w = wl.D, wl.Dv, wl.m, wl.w
    per = (2 * 4 * m * Dv + 2 * 4 * m + 2 * 4 + w * (D + Dv) * es + (D + Dv) * es
           + (3 * D + 2 * Dv) * es + Dv * es)
    return wl.B * wl.H * per


def measure_decode(steps, warmup, torch, L, dev):
    """The autoregressive path at 256 sequences x 16 heads after an
    8192-token prefix: the median of three timed prefills (after an untimed
    one), `steps` timed single decode steps (after `warmup` untimed ones) and
    one timed 16-token chunked call, all on the current stream.  Returns the
    measurements as a dict."""
    from paper_2608_09307_amd.workloads import WORKLOADS, make_decode_inputs
    wl = WORKLOADS["decode_s256_h16"]
    x = make_decode_inputs(wl, device=dev)
    pre, tok = x["prefix"], x["token"]
    st = L.prefill(pre["k"], pre["v"], pre["r"], pre["u"], x["omega"], wl.w)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    prefill_ms = []
    for _ in range(3):
        st = None                # each timed call takes its outputs from the allocator's cache
        ev[0].record(stream)
        st = L.prefill(pre["k"], pre["v"], pre["r"], pre["u"], x["omega"], wl.w)
        ev[1].record(stream)
        torch.cuda.synchronize()
        prefill_ms.append(ev[0].elapsed_time(ev[1]))
    for _ in range(warmup):
        L.decode_step(st, tok["q"], tok["k"], tok["v"], tok["r"], tok["u"], x["omega"], wl.w)
    torch.cuda.synchronize()
    L.timing_enable(True)
    L.timing_read()
    ev[2].record(stream)
    for _ in range(steps):
        L.decode_step(st, tok["q"], tok["k"], tok["v"], tok["r"], tok["u"], x["omega"], wl.w)
    ev[3].record(stream)
    torch.cuda.synchronize()
    kt = L.timing_read()
    L.timing_enable(False)
    T = 16
    chunk = {nm: tok[nm][:, :, None, :].expand(wl.B, wl.H, T, tok[nm].shape[-1]).contiguous()
             for nm in ("q", "k", "v", "r", "u")}
    L.decode_chunk(st, *(chunk[nm] for nm in ("q", "k", "v", "r", "u")), x["omega"], wl.w)
    torch.cuda.synchronize()
    ev[4].record(stream)
    L.decode_chunk(st, *(chunk[nm] for nm in ("q", "k", "v", "r", "u")), x["omega"], wl.w)
    ev[5].record(stream)
    torch.cuda.synchronize()
    ms = ev[2].elapsed_time(ev[3]) / steps
    chunk_ms = ev[4].elapsed_time(ev[5])
    roofline = None
    if "decode" in kt:
        avg_ms = kt["decode"][0] / kt["decode"][1]
        gbs = decode_step_bytes(wl) / (avg_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic_for("decode", DECODE_TRAFFIC_FILE),
                    "kernel": "decode",
                    "avg_ms": round(avg_ms, 4), "bytes": decode_step_bytes(wl)}
    del x, pre, tok, st, chunk
    return {
        "metric": "LinSimp decode tokens/s (256 sequences x 16 heads, 8192-token prefix)",
        "value": round(wl.B / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms, 4),
        "config": {"workload": "decode_s256_h16", "S": wl.B, "H": wl.H, "prefix": wl.n_prefix,
                   "d": wl.D, "m": wl.m, "w": wl.w},
        "roofline": roofline,
        "prefill_ms": round(sorted(prefill_ms)[1], 3),
        "chunk16": {"ms_per_call": round(chunk_ms, 4), "us_per_token_step": round(chunk_ms * 1e3 / T, 2),
                    "tokens_per_s": round(wl.B * T / (chunk_ms * 1e-3), 1)},
    }


def run_decode(args, torch, L, dev):
    """Decode-mode line (--decode): the measurements of measure_decode as the
    line itself."""
    m = measure_decode(args.steps, args.warmup, torch, L, dev)
    line = {
        "metric": m["metric"], "value": m["value"], "unit": m["unit"], "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": m["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1)*d^-1/4 prefix and tokens, N(0,1) feature bank)",
        "config": m["config"], "roofline": m["roofline"], "prefill_ms": m["prefill_ms"],
        "chunk16": m["chunk16"],
    }
    print(json.dumps(line), flush=True)


def head_stream_bytes(wl, es=2):
    """Algorithmic HBM bytes per launch of the streaming head kernels (each
    row read and written once; per-row float32 scalars included)."""
    rows = wl.B * wl.H * wl.n
    D, Dv = wl.D, wl.Dv
    return {
        "head_prenorm": rows * 6 * D * es,                        # q, k, r in; q', k', r' out
        "head_gate": rows * (2 * Dv * es + 4),                    # o~ in; y, rho out
        "head_gate_bwd": rows * (3 * Dv * es + 2 * 4),            # o~, dy in; d o~ out; rho in, part out
        "head_prenorm_bwd": rows * (9 * D * es + 4),              # q, k, r, core grads in; grads out
    }


HEADERS = ["common.h", "keyfeat.h", "linsimp_internal.h", "prof.h"]
KERNEL_FILES = {"fwd_readout": ["fwd.hip"] + HEADERS, "bwd_du": ["bwd.hip"] + HEADERS,
                "bwd_dqdr": ["bwd.hip"] + HEADERS, "bwd_state": ["bwd.hip"] + HEADERS,
                "bwd_keys": ["bwd.hip"] + HEADERS, "decode": ["decode.hip"] + HEADERS}


def src_digest(files=None):
    """sha256 prefix of the named kernel sources (all of csrc/ by default) and
    of the build script that holds their compiler flags."""
    h = hashlib.sha256()
    pkg = os.path.join(ROOT, "paper_2608_09307_amd")
    csrc = os.path.join(pkg, "csrc")
    names = sorted(files) if files else sorted(os.listdir(csrc))
    for name in names:
        if name.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(csrc, name), "rb") as fh:
                h.update(name.encode())
                h.update(fh.read())
    with open(os.path.join(pkg, "build.py"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SYMBOLS = {"fwd_readout": "k_readout", "bwd_du": "k_bwd_du", "bwd_dqdr": "k_bwd_dqdr",
                  "bwd_state": "k_bwd_state", "bwd_keys": "k_bwd_keys", "decode": "k_decode"}


def traffic_for(kernel, path=TRAFFIC_FILE):
    """Calibrated HBM bytes (FETCH_SIZE + WRITE_SIZE) per launch of `kernel`
    from the committed counter runs, if they were taken on the kernel's
    current sources (its .hip file and the headers it includes); else None."""
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    per = t.get("per_kernel", {}).get(KERNEL_SYMBOLS.get(kernel, ""))
    if per is None or kernel not in KERNEL_FILES:
        return None
    if per.get("src_sha") != src_digest(KERNEL_FILES[kernel]):
        return None
    return per["fetch_bytes"] + per["write_bytes"]


def host_info():
    """Host cores this process may run on, BLAS threads and the CPU model."""
    cores = len(os.sched_getaffinity(0))
    blas = None
    try:
        from threadpoolctl import threadpool_info
        blas = max([int(p.get("num_threads", 1)) for p in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        pass
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return cores, blas, model


def cpu_baseline(x, wl, budget_s, dev):
    """Time the float64 oracle on host cores.  The headline value: forward +
    backward on the first rows of one (batch, head) sequence of the step's
    workload (rows are causal, so a prefix is a complete sub-problem), scaled
    to the full job as tokens/s = rows/s / H.  `extra` times the oracle on the
    other workloads: the single f32 head in full, the 2k-token layer's
    forward on two of its 32 (batch, head) pairs, and the decode step on 32
    of the 4096 (sequence, head) pairs of the 256 x 16 decode workload (state
    prefilled by the oracle outside the timed region), each scaled to its
    whole job.  Inputs come from the seeded generators on `dev` (the values
    the GPU path is measured on); only the sampled slices are copied to the
    host."""
    import numpy as np
    from oracle import linsimp as O
    from paper_2608_09307_amd.workloads import WORKLOADS, make_decode_inputs, make_inputs

    cores, blas, model = host_info()

    def f64(t):
        return t.detach().float().cpu().double().numpy()

    b, h = 0, 0
    q, k, v, r, u = (f64(x[nm][b, h]) for nm in ("q", "k", "v", "r", "u"))
    om, dO = f64(x["omega"][h]), f64(x["dO"][b, h])

    def run(rows):
        t0 = time.perf_counter()
        O.forward_recurrent(q[:rows], k[:rows], v[:rows], r[:rows], u[:rows], om, wl.w)
        O.backward(q[:rows], k[:rows], v[:rows], r[:rows], u[:rows], om, wl.w, dO[:rows])
        return time.perf_counter() - t0

    cal_rows = 256
    t_cal = run(cal_rows)
    rows = int(min(wl.n, max(cal_rows, cal_rows * budget_s / max(t_cal, 1e-6))))
    rows = max(cal_rows, rows)
    t = run(rows) if rows != cal_rows else t_cal
    rate = rows / t / wl.H
    extra = {}
    # the single f32 head (1 x 1 x 256, d = m = 32), forward, in full
    w1 = WORKLOADS["head_f32_n256"]
    x1 = make_inputs(w1, device=dev)
    a1 = [f64(x1[nm][0, 0]) for nm in ("q", "k", "v", "r", "u")] + [f64(x1["omega"][0])]
    t0 = time.perf_counter()
    O.forward_recurrent(*a1, w1.w)
    t1 = time.perf_counter() - t0
    extra["head_f32_n256_fwd"] = {"value": round(w1.n / t1, 1), "unit": "tokens/s",
                                  "sample": f"the whole workload ({w1.n} rows) in {t1:.3f} s"}
    # the 2k-token layer forward (4 x 8 x 2048, d = m = 64) on two (batch, head) pairs
    w2 = WORKLOADS["layer2k_bf16"]
    x2 = make_inputs(w2, device=dev)
    t0 = time.perf_counter()
    for bb, hh in ((0, 0), (3, 7)):
        O.forward_recurrent(*(f64(x2[nm][bb, hh]) for nm in ("q", "k", "v", "r", "u")),
                            f64(x2["omega"][hh]), w2.w)
    t2 = time.perf_counter() - t0
    extra["layer2k_bf16_fwd"] = {
        "value": round(2 * w2.n / t2 / w2.H, 1), "unit": "tokens/s",
        "sample": (f"forward of 2 of the {w2.B * w2.H} (batch, head) pairs in {t2:.2f} s; "
                   f"full-job tokens/s = rows/s / H (H={w2.H})")}
    # the decode step (256 x 16 after 8192 tokens) on 32 (sequence, head) pairs
    w4 = WORKLOADS["decode_s256_h16"]
    x4 = make_decode_inputs(w4, device=dev)
    pre, tok = x4["prefix"], x4["token"]
    picks = [(7 * j % w4.B, j % w4.H) for j in range(32)]
    states = [O.prefill_state(*(f64(pre[nm][s_, h_]) for nm in ("k", "v", "r", "u")),
                              f64(x4["omega"][h_]), w4.w) for s_, h_ in picks]
    toks = [[f64(tok[nm][s_, h_]) for nm in ("q", "k", "v", "r", "u")] for s_, h_ in picks]
    oms = [f64(x4["omega"][h_]) for _, h_ in picks]
    t0 = time.perf_counter()
    for st_, tk, om4 in zip(states, toks, oms):
        O.decode_step(st_, *tk, om4, w4.w)
    t4 = time.perf_counter() - t0
    del x4, pre, tok
    pairs = w4.B * w4.H
    extra["decode_s256_h16_step"] = {
        "value": round(w4.B / (t4 * pairs / len(picks)), 2), "unit": "tokens/s",
        "sample": (f"one decode step of {len(picks)} of the {pairs} (sequence, head) pairs in "
                   f"{t4 * 1e3:.1f} ms (prefill excluded); a whole step over all pairs scaled "
                   f"as {pairs}/{len(picks)} times that; tokens/s = sequences / step time")}
    return {"value": rate, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "blas_threads": blas, "cpu_model": model,
            "sample": (f"float64 oracle forward+backward of the first {rows} rows of one "
                       f"(batch, head) of the {wl.n}-token layer in {t:.1f} s; full-job "
                       f"tokens/s = rows/s / H (H={wl.H})"),
            "extra": extra}


def copy_calibration(torch, dev, nbytes=1 << 30, reps=3):
    """A plain device-to-device copy of `nbytes` (read nbytes, write nbytes) run
    `reps` times: the reference for scaling FETCH_SIZE / WRITE_SIZE counters."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the oracle timing on host cores")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (for scaling HBM counters)")
    ap.add_argument("--head", action="store_true",
                    help="time the full head (normalisation, core, gated RMSNorm) instead of the core")
    ap.add_argument("--decode", action="store_true",
                    help="time prefill, decode steps and chunked decode (256 x 16 sequences)")
    ap.add_argument("--no-decode", action="store_true",
                    help="leave the decode measurement out of the forward + backward line")
    ap.add_argument("--workload", default=WORKLOAD,
                    help="forward + backward workload of the step (default: the 16k layer); "
                         "e.g. stress64k_m256 or layer2k_h6_d64_m128")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the LinSimp core here runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_09307_amd import linsimp as L
    from paper_2608_09307_amd.workloads import WORKLOADS, make_head_params, make_inputs

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(torch, dev)
        return
    if args.decode:
        run_decode(args, torch, L, dev)
        return
    if args.workload not in WORKLOADS or WORKLOADS[args.workload].mode != "fwdbwd":
        print(f"--workload must be a forward + backward workload, not {args.workload}", file=sys.stderr)
        sys.exit(2)
    wl = WORKLOADS[args.workload]
    x = make_inputs(wl, device=dev, with_grad=True)
    d = L.dims_of(x["q"], x["v"], x["omega"], wl.w)
    ws_b = L.alloc_workspace(d, True, dev)
    out = torch.empty_like(x["v"])
    stats = torch.empty(x["q"].shape[:3] + (2,), dtype=torch.float32, device=dev)
    grads = tuple(torch.empty_like(x[nm]) for nm in ("q", "k", "v", "r", "u"))

    def step():
        # the forward writes its boundary states into the backward-sized
        # workspace and the backward reuses them (LINSIMP_BWD_REUSE_STATES)
        L.fwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, out=out, stats=stats,
              workspace=ws_b)
        L.bwd(x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, out, stats, x["dO"],
              grads=grads, workspace=ws_b, reuse_states=True)

    if args.head:
        import ctypes
        hp = make_head_params(wl, device=dev)
        hargs = (x["q"], x["k"], x["v"], x["r"], x["u"], x["omega"], wl.w, hp["tau"], hp["gate"])
        del ws_b
        hws = L._aligned_bytes(int(L.lib().linsimp_head_workspace_size(ctypes.byref(d), 1)), dev)
        y, saved = L.head_fwd(*hargs, workspace=hws)

        def step():  # noqa: F811  (the full head instead of the core)
            L.head_fwd(*hargs, y=y, saved=saved, workspace=hws)
            L.head_bwd(*hargs, saved, x["dO"], workspace=hws, reuse_states=True)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    L.timing_enable(True)
    L.timing_read()
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    L.timing_enable(False)
    kt = L.timing_read()
    ms = e0.elapsed_time(e1) / args.steps

    tokens = wl.B * wl.n
    kf = kernel_flops(wl)
    fwd_flops = kf["fwd_readout"]
    bwd_flops = kf["bwd_du"] + kf["bwd_dqdr"] + kf["bwd_state"]
    step_tflops = (fwd_flops + bwd_flops) / (ms * 1e-3) / 1e12
    dominant = max(kt, key=lambda k: kt[k][0]) if kt else None
    kernels_ms = {k: round(v[0] / max(v[1], 1), 4) for k, v in sorted(kt.items(), key=lambda kv: -kv[1][0])}
    roofline = None
    if dominant is not None:
        tot, cnt = kt[dominant]
        avg_s = tot / cnt * 1e-3
        if dominant in kf:
            achieved = kf[dominant] / avg_s / 1e12
            roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                        "traffic": traffic_for(dominant) if args.workload == WORKLOAD else None,
                        "kernel": dominant,
                        "avg_ms": round(tot / cnt, 4)}
    head_streams = None
    if args.head:
        hb = head_stream_bytes(wl)
        head_streams = {}
        for k, b in hb.items():
            if k in kt:
                gbs = b / (kt[k][0] / kt[k][1] * 1e-3) / 1e9
                head_streams[k] = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                                   "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                                   "bytes": b, "avg_ms": round(kt[k][0] / kt[k][1], 4)}
    line = {
        "metric": ("LinSimp head fwd+bwd tokens/s at n=16k" if args.head else
                   "LinSimp fwd+bwd tokens/s at n=16k; % of MI355X bf16 MFMA peak" if args.workload == WORKLOAD else
                   f"LinSimp fwd+bwd tokens/s ({args.workload})"),
        "value": round(tokens / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1)*d^-1/4 streams, N(0,1) feature bank and dO)",
        "config": {"workload": args.workload + ("_head" if args.head else ""), "B": wl.B, "H": wl.H,
                   "n": wl.n, "d": wl.D, "m": wl.m, "w": wl.w},
        "mfma_frac_step": round(step_tflops / PEAK_BF16_TFLOPS, 4),
        "algorithmic_tflops_step": round(step_tflops, 2),
        "roofline": roofline,
        "kernels_avg_ms": kernels_ms,
    }
    if head_streams is not None:
        line["head_streams"] = head_streams
    if not args.no_decode and not args.head and args.workload == WORKLOAD:
        # the HBM-bound path, measured in the same run after the timed steps
        del x, ws_b, out, stats, grads
        torch.cuda.empty_cache()
        line["decode"] = measure_decode(args.steps, args.warmup, torch, L, dev)
        x = make_inputs(wl, device=dev, with_grad=True) if not args.no_cpu_baseline else None
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(x, wl, args.cpu_seconds, dev)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
