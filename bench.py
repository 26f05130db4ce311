#!/usr/bin/env python3
"""Benchmark of the DASC state-checkpoint hot path on one MI355X.

One step = one pass of the whole device path over one batch of synthetic input:
    pack     64 Kimi-Linear-shaped KDA layer states (32 heads, 128x128 fp32,
             1556 of 4096 rows kept = 38%) into ragged checkpoints,
    restore  the 64 checkpoints into fresh active states (omitted rows = +0.0),
    refresh  16 of them by replaying W = 1024 suffix tokens of the gated delta
             rule and overwriting only the omitted rows.
The selection plan is built once on the host before timing (the paper builds it
offline); its host time is reported separately.

Prints one JSON line.  `value` is suffix tokens refreshed per second of whole-step
time (n_req * W / step time); per-kernel rates are in `kernels`.  All inputs are
resident in HBM before the timed region starts.

    python bench.py [--steps K] [--warmup W] [--workload kimi_headline|kimi_model|qwen_gdn]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak
# Chunked WY form at 32-token chunks, dk = dv = 128, per head-token: the three 16x16
# A tiles (3*16*16*128 MAC), K_G S (32*128*128), T'(V - K_G S) (32*32*128)
# and K_H^T U (128*32*128), per 32 tokens, 2 FLOP per MAC.
WY_FLOP_PER_HEAD_TOKEN = 2.0 * (3 * 16 * 16 * 128 + 32 * 128 * 128 + 32 * 32 * 128 + 128 * 32 * 128) / 32
METRIC = "pack/restore GB/s + suffix-refresh tokens/s (KDA 32h x 128x128, W=1024)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    # From idle, the clock takes about 25 back-to-back steps to settle under this load: the
    # refresh launch time climbs from 295 to 350 us and comes back to 300 us over the
    # first 23 launches of a run, then stays at 280-300 us.
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default="kimi_headline",
                    choices=["kimi_headline", "kimi_model", "qwen_gdn"])
    ap.add_argument("--W", type=int, default=1024)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-windows", action="store_true",
                    help="time the refresh at the headline window only (counter runs average "
                         "every dispatch of a kernel, so the other windows would mix in)")
    ap.add_argument("--copy-calib", action="store_true",
                    help="run only a plain device copy of known size (counter calibration)")
    ap.add_argument("--copy-bw", action="store_true",
                    help="time only torch's device copy of 4 GiB (the box's plain-copy rate)")
    return ap.parse_args()


def kernel_source_hash() -> str:
    """Digest of everything that decides the device code: the kernel sources and headers,
    and the build script with its compiler flags."""
    h = hashlib.sha256()
    for f in ("pack_restore.hip", "quant.hip", "refresh.hip", "refresh_wy.hip", "refresh_wy_gdn.hip",
              "ckpt_layout.h", "refresh_kernels.h", "launch_common.h", "wy_ops.h"):
        with open(os.path.join(ROOT, "paper_2608_30386_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "paper_2608_30386_amd", "build.py"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()[:16]


def _counter_summary():
    """The committed counter summary, if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return {}
    with open(path) as fh:
        t = json.load(fh)
    return t if t.get("source_hash") == kernel_source_hash() else {}


def measured_traffic(key: str):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled), or None."""
    return _counter_summary().get("kernels", {}).get(key)


def measured_util(key: str, what: str):
    """MFMA-busy or VALU-active fraction of the kernel's SIMD cycles, or None."""
    return _counter_summary().get("utilisation", {}).get(key, {}).get(what)


class KernelTimer:
    """HIP events around launches on the stream the library is given."""

    def __init__(self, torch):
        self.torch = torch
        self.spans = {}

    def run(self, name, fn):
        ev0 = self.torch.cuda.Event(enable_timing=True)
        ev1 = self.torch.cuda.Event(enable_timing=True)
        ev0.record()
        fn()
        ev1.record()
        self.spans.setdefault(name, []).append((ev0, ev1))

    def mean_ms(self, name):
        return float(np.mean([a.elapsed_time(b) for a, b in self.spans[name]]))


def copy_calibration(torch):
    n = 1 << 28  # 1 GiB of fp32
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "launches": 3}))


def copy_bandwidth(torch, args):
    """torch's device-to-device copy of 4 GiB of fp32: the plain-copy rate of the GPU, the
    secondary reference for the pack and restore rates (bytes read + written per second)."""
    n = 1 << 30
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    print(json.dumps({"copy_bytes": 2 * n * 4, "ms": ms, "GBps": 2 * n * 4 / ms / 1e6,
                      "steps": args.steps, "warmup": args.warmup}))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(the checkpoint kernels run on one device). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_calib:
        copy_calibration(torch)
        return
    if args.copy_bw:
        copy_bandwidth(torch, args)
        return
    if args.workload == "kimi_headline":
        out = bench_headline(torch, args)
    elif args.workload == "kimi_model":
        out = bench_pack_restore_only(torch, args, "kimi_model")
    else:
        out = bench_gdn(torch, args)
    print(json.dumps(out))


# ---------------------------------------------------------------------------------------

def timed_steps(torch, fn, args) -> float:
    """Warm up, then wall-clock exactly args.steps calls between two synchronisations (ms
    per call)."""
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / args.steps


def _setup_plan(wl):
    import paper_2608_30386_amd as D
    from workloads import log_lambda

    sh = D.Shape(wl.arch, wl.n_layers, wl.n_heads, wl.n_qk_heads, wl.dk, wl.dv)
    t0 = time.perf_counter()
    plan = D.dasc_plan(sh, D.dasc_static_log_decay(log_lambda(wl)), wl.keep_mode, wl.keep_k,
                       wl.w_max, wl.n_ranks, wl.eps)
    return sh, plan, time.perf_counter() - t0


def _i32(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def _bf16(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def bench_headline(torch, args):
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS, log_lambda, refresh_inputs, states_host

    wl = WORKLOADS["kimi_layer"]
    W = args.W
    n_ckpt, n_req = wl.n_ckpt, wl.n_req
    sh, plan, plan_s = _setup_plan(wl)
    R = int(plan["n_rows"])
    rows, dv = sh.rows, sh.dv

    states_np = states_host(wl, n_ckpt)
    inp = refresh_inputs(wl, W, log_lambda(wl)[0])
    states = torch.from_numpy(states_np).cuda()
    ckpt = torch.empty((n_ckpt, R, dv), dtype=torch.float32, device="cuda")
    active = torch.empty_like(states)
    unit_row, inv_row = _i32(torch, plan["unit_row"]), _i32(torch, plan["inv_row"])
    ids = _i32(torch, np.arange(n_ckpt))
    req = _i32(torch, np.arange(n_req))
    k, v = _bf16(torch, inp["k"]), _bf16(torch, inp["v"])
    g, beta = torch.from_numpy(inp["g"]).cuda(), torch.from_numpy(inp["beta"]).cuda()
    torch.cuda.synchronize()

    timer = KernelTimer(torch)

    def plain_step():
        D.dasc_pack(sh, states, ids, unit_row, ckpt, ids)
        D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R)
        D.dasc_refresh(sh, 0, inv_row, active, req, k, v, g, beta, W)

    def step():
        timer.run("pack", lambda: D.dasc_pack(sh, states, ids, unit_row, ckpt, ids))
        timer.run("restore", lambda: D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R))
        timer.run("refresh", lambda: D.dasc_refresh(sh, 0, inv_row, active, req, k, v, g, beta, W))

    # the timed steps are plain launches; events around each launch add about 10 us of
    # GPU-side gap per kernel, so the per-kernel durations come from a second pass.
    # (A HIP graph of the three launches replays slower here: 0.405 vs 0.357 ms.)
    ms_step = timed_steps(torch, plain_step, args)

    # per-kernel durations: HIP events around each launch, on the library's stream
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    timer.spans.clear()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()

    # Load with refresh of the refreshed requests: dasc_restore + dasc_refresh (two launches)
    # against the fused dasc_restore_refresh (one launch, the same result bit for bit)
    def load_wr():
        timer.run("restore_req", lambda: D.dasc_restore(sh, ckpt, req, inv_row, active, req, n_rows=R))
        timer.run("refresh_req", lambda: D.dasc_refresh(sh, 0, inv_row, active, req, k, v, g, beta, W))
        timer.run("restore_refresh", lambda: D.dasc_restore_refresh(
            sh, 0, ckpt, req, inv_row, active, req, k, v, g, beta, W, n_rows=R))

    load_wr()
    torch.cuda.synchronize()
    for name in ("restore_req", "refresh_req", "restore_refresh"):
        timer.spans[name].clear()
    for _ in range(args.steps):
        load_wr()
    torch.cuda.synchronize()

    omitted = (plan["inv_row"] < 0).reshape(sh.n_heads, sh.dk)
    heads_refreshed = int(omitted.any(axis=1).sum())
    bytes_pack = 2 * R * dv * 4 * n_ckpt
    bytes_restore = (R + rows) * dv * 4 * n_ckpt

    def refresh_bytes(w):
        # refresh reads k, v, g, beta and the restored state of every refreshed head, and
        # writes the omitted rows
        per_head = (2 * w * sh.dk + 2 * w * dv + 4 * w * sh.dk + 4 * w + 4 * sh.dk * dv)
        return per_head, n_req * (heads_refreshed * per_head + int(omitted.sum()) * dv * 4)

    per_head, bytes_refresh = refresh_bytes(W)
    flops_refresh = WY_FLOP_PER_HEAD_TOKEN * W * n_req * heads_refreshed

    # the serving shape's other replay windows (refresh alone, same requests and state)
    by_window = {}
    for w2 in wl.windows:
        if w2 == W or args.no_other_windows:
            continue
        inp2 = refresh_inputs(wl, w2, log_lambda(wl)[0], salt=w2)
        k2, v2 = _bf16(torch, inp2["k"]), _bf16(torch, inp2["v"])
        g2, b2 = torch.from_numpy(inp2["g"]).cuda(), torch.from_numpy(inp2["beta"]).cuda()
        name = f"refresh_W{w2}"
        run2 = lambda: D.dasc_refresh(sh, 0, inv_row, active, req, k2, v2, g2, b2, w2)  # noqa: E731
        for _ in range(args.warmup):
            run2()
        torch.cuda.synchronize()
        for _ in range(args.steps):
            timer.run(name, run2)
        torch.cuda.synchronize()
        ms2 = timer.mean_ms(name)
        by_window[str(w2)] = {"ms": ms2, "tokens_per_s": n_req * w2 / (ms2 / 1e3),
                              "GBps": refresh_bytes(w2)[1] / ms2 / 1e6,
                              "hbm_frac": refresh_bytes(w2)[1] / ms2 / 1e6 / HBM_PEAK_GBPS}
        del k2, v2, g2, b2

    t = {n: timer.mean_ms(n) for n in ("pack", "restore", "refresh", "restore_req", "refresh_req",
                                       "restore_refresh")}
    # fused: suffix inputs of every refreshed head, each kept row read once, every row of
    # the layer written once
    bytes_fused = n_req * (heads_refreshed * (per_head - 4 * sh.dk * dv) + R * dv * 4 + rows * dv * 4)
    kernels = {
        "pack": {"ms": t["pack"], "GBps": bytes_pack / t["pack"] / 1e6,
                 "hbm_frac": bytes_pack / t["pack"] / 1e6 / HBM_PEAK_GBPS, "bytes": bytes_pack},
        "restore": {"ms": t["restore"], "GBps": bytes_restore / t["restore"] / 1e6,
                    "hbm_frac": bytes_restore / t["restore"] / 1e6 / HBM_PEAK_GBPS,
                    "bytes": bytes_restore},
        "refresh": {"ms": t["refresh"], "tokens_per_s": n_req * W / (t["refresh"] / 1e3),
                    "GBps": bytes_refresh / t["refresh"] / 1e6,
                    "TFLOPs": flops_refresh / t["refresh"] / 1e9, "bytes": bytes_refresh,
                    "flops": flops_refresh, "heads": n_req * heads_refreshed},
        "restore_refresh_fused": {
            "ms": t["restore_refresh"], "unfused_ms": t["restore_req"] + t["refresh_req"],
            "requests": n_req, "GBps": bytes_fused / t["restore_refresh"] / 1e6,
            "bytes": bytes_fused},
        "refresh_by_window": by_window,
    }
    achieved = bytes_refresh / t["refresh"] / 1e6          # GB/s
    traffic = measured_traffic("kimi_headline/refresh")
    out = {
        "metric": METRIC,
        "value": n_req * W / (ms_step / 1e3),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"KDA layer 32h x 128x128 fp32: pack+restore {n_ckpt} checkpoints "
                        f"(R={R} of {rows} rows kept), refresh {n_req} requests W={W}",
            "n_checkpoints": n_ckpt, "n_requests": n_req, "W": W, "rows_kept": R,
            "inputs": "k,v bf16; g,beta fp32; state fp32",
        },
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": traffic, "kernel": "refresh",
                     "work_per_launch": f"{bytes_refresh} B = per refreshed head: k, v (bf16), g, "
                                        "beta (fp32), restored state read, omitted rows written",
                     "mfma_frac": flops_refresh / (t["refresh"] / 1e3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
                     "mfma_busy": measured_util("kimi_headline/refresh", "mfma_busy"),
                     "valu_active": measured_util("kimi_headline/refresh", "valu_active")},
        "kernels": kernels,
        "pack_restore_GBps": (bytes_pack + bytes_restore) / (t["pack"] + t["restore"]) / 1e6,
        "plan_host_ms": plan_s * 1e3,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_headline(wl, plan, states_np, inp, W, n_req)
    return out


def cpu_baseline_headline(wl, plan, states_np, inp, W, n_req):
    """The oracle, as it stands, on a bounded sample of the same step."""
    from threadpoolctl import threadpool_limits

    from oracle import pack as OK
    from oracle import recurrence as OR

    n_s, req_s = wl.n_ckpt, n_req // 2        # all checkpoints, half the requests
    R = int(plan["n_rows"])
    words = states_np.reshape(states_np.shape[0], -1, wl.dv).view(np.uint32)
    with threadpool_limits(1):
        t0 = time.perf_counter()
        ck = OK.pack(words, list(range(n_s)), plan["unit_row"],
                     np.zeros((1, n_s, R, wl.dv), np.uint32), list(range(n_s)))
        t_pack = time.perf_counter() - t0
        t0 = time.perf_counter()
        back = OK.restore(ck, list(range(n_s)), plan["unit_row"], np.zeros_like(words[:n_s]),
                          list(range(n_s)))
        t_restore = time.perf_counter() - t0
        layer = back.view(np.float32).reshape(n_s, wl.n_heads, wl.dk, wl.dv)
        pairs = [(n, h) for n in range(req_s) for h in range(wl.n_heads)]
        sub = {key: val[:req_s] for key, val in inp.items()}
        t0 = time.perf_counter()
        OR.refresh(layer[:req_s], plan["inv_row"], sub["k"], sub["v"], sub["g"], sub["beta"],
                   wl.n_qk_heads, pairs=pairs)
        t_ref = time.perf_counter() - t0
    scale_ck = wl.n_ckpt / n_s
    step_s = (t_pack + t_restore) * scale_ck + t_ref * n_req / req_s
    return {"value": n_req * W / step_s, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"pack+restore all {n_s} checkpoints, refresh {req_s} of {n_req} requests "
                      f"x 32 heads at W={W} (fp64 per-token form, vectorised over heads); the "
                      "refresh time is scaled to all requests",
            "sample_seconds": t_pack + t_restore + t_ref,
            "host_cpus": os.cpu_count()}


def bench_pack_restore_only(torch, args, name):
    """GB-scale pack + restore (full-model KDA set) for the HBM roofline."""
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS, states_device

    wl = WORKLOADS[name]
    sh, plan, plan_s = _setup_plan(wl)
    R, rows, dv, n = int(plan["n_rows"]), sh.rows, sh.dv, wl.n_ckpt
    T, C = wl.n_ranks, int(plan["slice_rows"])
    states = states_device(wl, n, "cuda")
    ckpt = torch.empty((T, n, C, dv), dtype=torch.float32, device="cuda")
    active = torch.empty_like(states)
    unit_row, inv_row = _i32(torch, plan["unit_row"]), _i32(torch, plan["inv_row"])
    ids = _i32(torch, np.arange(n))
    timer = KernelTimer(torch)

    def plain_step():
        D.dasc_pack(sh, states, ids, unit_row, ckpt, ids, n_ranks=T, slice_rows=C)
        D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R, n_ranks=T, slice_rows=C)

    def step():
        timer.run("pack", lambda: D.dasc_pack(sh, states, ids, unit_row, ckpt, ids, n_ranks=T,
                                              slice_rows=C))
        timer.run("restore", lambda: D.dasc_restore(sh, ckpt, ids, inv_row, active, ids,
                                                    n_rows=R, n_ranks=T, slice_rows=C))

    ms_step = timed_steps(torch, plain_step, args)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    timer.spans.clear()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    bp = 2 * R * dv * 4 * n
    br = (R + rows) * dv * 4 * n
    t = {k_: timer.mean_ms(k_) for k_ in ("pack", "restore")}
    gbps = (bp + br) / (t["pack"] + t["restore"]) / 1e6
    dom = "restore" if t["restore"] >= t["pack"] else "pack"
    dom_bytes = br if dom == "restore" else bp
    ach = dom_bytes / t[dom] / 1e6

    # INT8 checkpoints (App. E.1) on the same states, flat layout, timed separately
    del ckpt
    q = torch.empty((n, R, dv), dtype=torch.int8, device="cuda")
    s = torch.empty((n, R), dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        D.dasc_pack_q8(sh, states, ids, unit_row, q, s, ids)
        D.dasc_restore_q8(sh, q, s, ids, inv_row, active, ids, n_rows=R)
    torch.cuda.synchronize()
    timer.spans.clear()
    for _ in range(args.steps):
        timer.run("pack_q8", lambda: D.dasc_pack_q8(sh, states, ids, unit_row, q, s, ids))
        timer.run("restore_q8", lambda: D.dasc_restore_q8(sh, q, s, ids, inv_row, active, ids,
                                                          n_rows=R))
    torch.cuda.synchronize()
    tq = {k_: timer.mean_ms(k_) for k_ in ("pack_q8", "restore_q8")}
    bpq = R * n * (dv * 4 + dv + 4)               # read fp32 rows, write int8 rows + scales
    brq = n * (R * (dv + 4) + rows * dv * 4)      # read int8 rows + scales, write fp32 states

    # padded layout (App. B Scheme 1, the comparison layout): same rows moved, L * R_max
    # rows reserved per checkpoint
    del q, s
    r_max = int(plan["r_max_rows"])
    off = _i32(torch, plan["layer_off_rows"])
    ck_pad = torch.empty((sh.n_layers, n, r_max, dv), dtype=torch.float32, device="cuda")
    for _ in range(args.warmup):
        D.dasc_pack_padded(sh, states, ids, unit_row, off, ck_pad, ids)
        D.dasc_restore_padded(sh, ck_pad, ids, off, inv_row, active, ids, n_rows=R)
    torch.cuda.synchronize()
    timer.spans.clear()
    for _ in range(args.steps):
        timer.run("pack_padded", lambda: D.dasc_pack_padded(sh, states, ids, unit_row, off, ck_pad,
                                                            ids))
        timer.run("restore_padded", lambda: D.dasc_restore_padded(sh, ck_pad, ids, off, inv_row,
                                                                  active, ids, n_rows=R))
    torch.cuda.synchronize()
    del ck_pad
    tp = {k_: timer.mean_ms(k_) for k_ in ("pack_padded", "restore_padded")}
    return {
        "metric": "pack+restore GB/s (full-model KDA checkpoint set)", "value": gbps, "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": f"{wl.n_layers} KDA layers x 32h x 128x128 fp32, {n} checkpoints, "
                               f"R={R} of {rows} rows kept, T={T} rank slices"},
        "roofline": {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBPS, "traffic": measured_traffic(f"{name}/{dom}"),
                     "kernel": dom},
        "kernels": {k_: {"ms": tt[k_], "GBps": b / tt[k_] / 1e6,
                         "hbm_frac": b / tt[k_] / 1e6 / HBM_PEAK_GBPS, "bytes": b}
                    for tt, k_, b in ((t, "pack", bp), (t, "restore", br),
                                      (tq, "pack_q8", bpq), (tq, "restore_q8", brq),
                                      (tp, "pack_padded", bp), (tp, "restore_padded", br))},
        "q8_checkpoint_bytes": R * (dv + 4), "fp32_checkpoint_bytes": R * dv * 4,
        "padded_checkpoint_bytes": sh.n_layers * r_max * dv * 4,
        "tp_stage1": tp_stage1(D, sh, plan, T),
        "plan_host_ms": plan_s * 1e3,
    }


def tp_stage1(D, sh, plan, T):
    """Stage-1 head-bundle permutation on this plan (host): retained rows of the worst
    rank before and after, and the rows stage 2 must move off over-full ranks to reach
    the balanced slot width C (rows a rank owns beyond C)."""
    res = D.dasc_tp_permutation(sh, plan["unit_count"], T)
    C = -(-int(plan["n_rows"]) // T)
    over = lambda rows: int(np.maximum(rows - C, 0).sum())  # noqa: E731
    return {"worst_rank_rows_identity": int(res["rank_rows_identity"].max()),
            "worst_rank_rows_permuted": int(res["rank_rows"].max()), "balanced_rows": C,
            "moved_rows_identity": over(res["rank_rows_identity"]),
            "moved_rows_permuted": over(res["rank_rows"])}


def bench_gdn(torch, args):
    """Qwen-GDN shape: pack/restore 128 checkpoints, refresh 8 requests x 36 layers."""
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS, log_lambda, refresh_inputs, states_device

    wl = WORKLOADS["qwen_gdn"]
    sh, plan, plan_s = _setup_plan(wl)
    R, rows, dv, n, W = int(plan["n_rows"]), sh.rows, sh.dv, wl.n_ckpt, args.W
    states = states_device(wl, n, "cuda")
    ckpt = torch.empty((n, R, dv), dtype=torch.float32, device="cuda")
    active = torch.empty_like(states)
    unit_row, inv_row = _i32(torch, plan["unit_row"]), _i32(torch, plan["inv_row"])
    ids, req = _i32(torch, np.arange(n)), _i32(torch, np.arange(wl.n_req))
    lam = log_lambda(wl)
    layers = []
    for l in range(wl.n_layers):
        inp = refresh_inputs(wl, W, lam[l], salt=l)
        layers.append((_bf16(torch, inp["k"]), _bf16(torch, inp["v"]),
                       torch.from_numpy(inp["g"]).cuda(), torch.from_numpy(inp["beta"]).cuda()))
    # the per-chunk WY factors of the two-launch GDN kernel, allocated once
    ws = torch.empty(D.dasc_refresh_workspace_bytes(sh, wl.n_req, W), dtype=torch.uint8,
                     device="cuda")
    timer = KernelTimer(torch)

    def ref():
        for l, (k, v, g, b) in enumerate(layers):
            D.dasc_refresh(sh, l, inv_row, active, req, k, v, g, b, W, workspace=ws)

    def plain_step():
        D.dasc_pack(sh, states, ids, unit_row, ckpt, ids)
        D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R)
        ref()

    def step():
        timer.run("pack", lambda: D.dasc_pack(sh, states, ids, unit_row, ckpt, ids))
        timer.run("restore", lambda: D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R))
        timer.run("refresh_all_layers", ref)

    ms_step = timed_steps(torch, plain_step, args)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    timer.spans.clear()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()

    # Load with refresh of the 8 requests: dasc_restore of their states + the 36 layer
    # refreshes, against one dasc_restore_refresh per layer (each restores its own layer;
    # the same bits)
    def load_wr():
        timer.run("restore_req", lambda: D.dasc_restore(sh, ckpt, req, inv_row, active, req, n_rows=R))
        timer.run("refresh_req", ref)

        def fused():
            for l, (k, v, g, b) in enumerate(layers):
                D.dasc_restore_refresh(sh, l, ckpt, req, inv_row, active, req, k, v, g, b, W, n_rows=R,
                                       workspace=ws)
        timer.run("restore_refresh", fused)

    load_wr()
    torch.cuda.synchronize()
    for name in ("restore_req", "refresh_req", "restore_refresh"):
        timer.spans[name].clear()
    for _ in range(args.steps):
        load_wr()
    torch.cuda.synchronize()
    t = {k_: timer.mean_ms(k_) for k_ in ("pack", "restore", "refresh_all_layers", "restore_req",
                                          "refresh_req", "restore_refresh")}
    bp, br = 2 * R * dv * 4 * n, (R + rows) * dv * 4 * n
    omitted = (plan["inv_row"].reshape(sh.n_layers, sh.n_heads, sh.dk) < 0).all(axis=2)
    om_heads = int(omitted.sum())
    heads = wl.n_req * om_heads
    # key heads some omitted v-head of their layer reads (v-heads of a group share one)
    key_heads = wl.n_req * sum(len(set(np.flatnonzero(o) // (sh.n_heads // sh.n_qk_heads)))
                               for o in omitted)
    # per refreshed head: v (bf16), g, beta (fp32), the restored head read and written; per
    # key head read: k (bf16)
    per_head = 2 * W * dv + 4 * W + 4 * W + 2 * 4 * sh.dk * dv
    bytes_ref = heads * per_head + key_heads * 2 * W * sh.dk
    ach = bytes_ref / (t["refresh_all_layers"] / 1e3) / 1e9          # GB/s
    flops = 5.0 * sh.dk * dv * W * heads
    return {
        "metric": "GDN pack/restore GB/s + refresh tokens/s (36 layers)",
        "value": wl.n_req * W / (t["refresh_all_layers"] / 1e3), "unit": "tokens/s (all 36 layers)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"Qwen-GDN 36 layers 16 qk / 32 v heads 128x128: pack+restore {n} "
                               f"checkpoints (12 of 32 heads kept), refresh {wl.n_req} requests x "
                               f"{om_heads} omitted heads W={W}"},
        "roofline": {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBPS, "traffic": measured_traffic("qwen_gdn/refresh"),
                     "kernel": "refresh",
                     "work_per_launch": f"{bytes_ref // wl.n_layers} B per layer launch "
                                        f"({heads // wl.n_layers} heads, "
                                        f"{key_heads / wl.n_layers:.1f} key heads)",
                     "recurrence_TFLOPs": flops / (t["refresh_all_layers"] / 1e3) / 1e12,
                     "mfma_busy": measured_util("qwen_gdn/refresh", "mfma_busy"),
                     "valu_active": measured_util("qwen_gdn/refresh", "valu_active")},
        "kernels": {"pack": {"ms": t["pack"], "GBps": bp / t["pack"] / 1e6},
                    "restore": {"ms": t["restore"], "GBps": br / t["restore"] / 1e6},
                    "refresh_all_layers": {"ms": t["refresh_all_layers"], "GBps": ach,
                                           "launches": 2 * wl.n_layers, "bytes": bytes_ref},
                    "restore_refresh_fused": {"ms": t["restore_refresh"], "launches": 2 * wl.n_layers,
                                              "unfused_ms": t["restore_req"] + t["refresh_req"],
                                              "requests": wl.n_req}},
        "plan_host_ms": plan_s * 1e3,
    }


if __name__ == "__main__":
    main()
