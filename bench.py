#!/usr/bin/env python3
"""Benchmark of the DASC state-checkpoint hot path on one MI355X.

One step = one pass of the whole device path over one batch of synthetic input:
    Store    pack 64 Kimi-Linear-shaped KDA layer states (32 heads, 128x128 fp32,
             1556 of 4096 rows kept = 38%) into ragged checkpoints;
    Load     restore the 64 checkpoints into fresh active states (omitted rows = +0.0),
             16 of them with refresh: replay W = 1024 suffix tokens of the gated delta
             rule and overwrite only the omitted rows.  The 16 take the fused Load with
             refresh (restore and replay in one launch, bit-identical to the two), the
             other 48 the plain restore; --unfused-step restores all 64, then refreshes.
The selection plan is built once on the host before timing (the paper builds it
offline); its host time is reported separately.

Prints one JSON line.  `value` is suffix tokens refreshed per second of whole-step
time (n_req * W / step time); per-kernel rates are in `kernels`.  All inputs are
resident in HBM before any timed region starts.

Order of work on the GPU:
  0. the headline measurement below taken as the very first GPU work of the process,
     reported as `first_pass_ms_per_step`;
  1. per-kernel durations of the step's kernels, from HIP events around batches of
     back-to-back launches of one kernel (median over batches);
  2. the headline: --warmup untimed steps, then exactly --steps timed steps between
     two synchronisations.  The refresh kernel's own duration follows the GPU's clock,
     which drops under sudden sustained load and recovers, so the same steps measured
     first thing (step 0) read 5-20% slower per step than here, after step 1;
  3. the other configurations, as extra keys: the full-model KDA checkpoint set (24
     layers, 256 checkpoints, T = 8 rank slices) pack/restore, and the Qwen-GDN refresh
     of 8 requests x 36 layers (`extra`);
  4. the CPU baseline (the oracle on the host cores, at 1 thread and at all of them).

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
MAX_POOL_THREADS = 16           # the host CPU share of one GPU on the benchmark machines


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default="kimi_headline",
                    choices=["kimi_headline", "kimi_model", "qwen_gdn"])
    ap.add_argument("--W", type=int, default=1024)
    ap.add_argument("--batches", type=int, default=10,
                    help="per-kernel timing: batches of back-to-back launches (median over them)")
    ap.add_argument("--per-batch", type=int, default=10, help="launches per timing batch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="headline only: skip the full-model KDA and Qwen-GDN extra keys")
    ap.add_argument("--unfused-step", action="store_true",
                    help="restore every checkpoint, then refresh (two launches for the refreshed "
                         "requests) instead of the fused Load with refresh")
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
              "refresh_noalloc.hip", "ckpt_layout.h", "refresh_kernels.h", "launch_common.h",
              "wy_ops.h"):
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


BATCHES, PER_BATCH = 10, 10   # set from --batches / --per-batch


def batched_ms(torch, fn, batches: int | None = None, per_batch: int | None = None,
               warm: int = 3) -> float:
    """Duration of one call of `fn` on the GPU (ms): HIP events on torch's current stream
    (the stream the library launches on) around `batches` runs of `per_batch`
    back-to-back calls, the median over the batches of elapsed / per_batch.  Events around
    whole batches add no per-launch gap."""
    batches = BATCHES if batches is None else min(batches, BATCHES)
    per_batch = PER_BATCH if per_batch is None else min(per_batch, PER_BATCH)
    for _ in range(warm):
        fn()
    spans = []
    for _ in range(batches):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(per_batch):
            fn()
        e1.record()
        spans.append((e0, e1))
    torch.cuda.synchronize()
    return float(np.median([a.elapsed_time(b) / per_batch for a, b in spans]))


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
    ms = batched_ms(torch, lambda: dst.copy_(src), batches=5, per_batch=max(args.steps // 5, 1))
    print(json.dumps({"copy_bytes": 2 * n * 4, "ms": ms, "GBps": 2 * n * 4 / ms / 1e6,
                      "steps": args.steps}))


def main():
    global BATCHES, PER_BATCH
    args = parse()
    BATCHES, PER_BATCH = max(1, args.batches), max(1, args.per_batch)
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
        out = bench_full_model(torch, args)
    else:
        out = bench_gdn(torch, args)
    print(json.dumps(out))


# ---------------------------------------------------------------------------------------

def timed_steps(torch, fn, args) -> float:
    """args.warmup untimed calls, then wall-clock exactly args.steps calls between two
    synchronisations (ms per call)."""
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


def _rate(ms, nbytes):
    return {"ms": ms, "GBps": nbytes / ms / 1e6, "hbm_frac": nbytes / ms / 1e6 / HBM_PEAK_GBPS,
            "bytes": nbytes}


def kda_refresh_bytes(sh, plan, n_req, W):
    """Algorithmic bytes of one KDA refresh launch: per refreshed head k, v (bf16), g,
    beta (fp32) and the restored state read; the omitted rows written."""
    omitted = (plan["inv_row"] < 0).reshape(sh.n_heads, sh.dk)
    heads = int(omitted.any(axis=1).sum())
    per_head = 2 * W * sh.dk + 2 * W * sh.dv + 4 * W * sh.dk + 4 * W + 4 * sh.dk * sh.dv
    return per_head, heads, n_req * (heads * per_head + int(omitted.sum()) * sh.dv * 4)


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

    def pack():
        D.dasc_pack(sh, states, ids, unit_row, ckpt, ids)

    def restore():
        D.dasc_restore(sh, ckpt, ids, inv_row, active, ids, n_rows=R)

    def refresh():
        D.dasc_refresh(sh, 0, inv_row, active, req, k, v, g, beta, W)

    # The Load of the step: the refreshed requests take the fused Load with refresh (restore
    # and replay in one launch, bit-identical to restore then refresh), the other checkpoints
    # the plain restore.  --unfused-step restores every checkpoint, then refreshes.
    ids_rest = _i32(torch, np.arange(n_req, n_ckpt))

    def restore_rest():
        D.dasc_restore(sh, ckpt, ids_rest, inv_row, active, ids_rest, n_rows=R)

    def load_refresh():
        D.dasc_restore_refresh(sh, 0, ckpt, req, inv_row, active, req, k, v, g, beta, W, n_rows=R)

    def step():
        pack()
        if args.unfused_step:
            restore()
            refresh()
        else:
            restore_rest()
            load_refresh()

    # the headline measurement as the first GPU work of the process (cold clock)
    first_ms = timed_steps(torch, step, args)

    # 1. per-kernel durations
    t = {"pack": batched_ms(torch, pack), "restore": batched_ms(torch, restore),
         "refresh": batched_ms(torch, refresh)}
    # Load with refresh of the refreshed requests: dasc_restore + dasc_refresh (two launches)
    # against the fused dasc_restore_refresh (the same result bit for bit)
    t["restore_req"] = batched_ms(torch, lambda: D.dasc_restore(sh, ckpt, req, inv_row, active, req,
                                                                n_rows=R))
    t["refresh_req"] = batched_ms(torch, refresh)
    t["restore_refresh"] = batched_ms(torch, load_refresh)
    t["restore_rest"] = batched_ms(torch, restore_rest)

    per_head, heads, bytes_refresh = kda_refresh_bytes(sh, plan, n_req, W)
    bytes_pack = 2 * R * dv * 4 * n_ckpt
    bytes_restore = (R + rows) * dv * 4 * n_ckpt
    flops_refresh = WY_FLOP_PER_HEAD_TOKEN * W * n_req * heads

    # the serving shape's other replay windows (refresh alone, same requests and state)
    by_window = {}
    for w2 in wl.windows:
        if w2 == W or args.no_other_windows:
            continue
        inp2 = refresh_inputs(wl, w2, log_lambda(wl)[0], salt=w2)
        k2, v2 = _bf16(torch, inp2["k"]), _bf16(torch, inp2["v"])
        g2, b2 = torch.from_numpy(inp2["g"]).cuda(), torch.from_numpy(inp2["beta"]).cuda()
        ms2 = batched_ms(torch, lambda: D.dasc_refresh(sh, 0, inv_row, active, req, k2, v2, g2, b2, w2))
        b_w2 = kda_refresh_bytes(sh, plan, n_req, w2)[2]
        by_window[str(w2)] = {"tokens_per_s": n_req * w2 / (ms2 / 1e3), **_rate(ms2, b_w2)}
        del k2, v2, g2, b2

    # fused: suffix inputs of every refreshed head, each kept row read once, every row of
    # the layer written once
    bytes_fused = n_req * (heads * (per_head - 4 * sh.dk * dv) + R * dv * 4 + rows * dv * 4)
    kernels = {
        "pack": _rate(t["pack"], bytes_pack),
        "restore": _rate(t["restore"], bytes_restore),
        "refresh": {"tokens_per_s": n_req * W / (t["refresh"] / 1e3),
                    "TFLOPs": flops_refresh / t["refresh"] / 1e9, "flops": flops_refresh,
                    "heads": n_req * heads, **_rate(t["refresh"], bytes_refresh)},
        "restore_refresh_fused": {
            "ms": t["restore_refresh"], "unfused_ms": t["restore_req"] + t["refresh_req"],
            "requests": n_req, "tokens_per_s": n_req * W / (t["restore_refresh"] / 1e3),
            **_rate(t["restore_refresh"], bytes_fused)},
        "restore_rest": {"checkpoints": n_ckpt - n_req,
                         **_rate(t["restore_rest"], (R + rows) * dv * 4 * (n_ckpt - n_req))},
        "refresh_by_window": by_window,
        "timing": "HIP events around 10 batches of 10 back-to-back launches, median",
    }

    # 2. the headline: warmup, then exactly args.steps timed steps
    ms_step = timed_steps(torch, step, args)

    # 3. the other configurations
    extra = {}
    if not args.no_extra:
        extra["kimi_model"] = full_model_keys(torch, args, layouts=("ragged",))
        torch.cuda.empty_cache()
        extra["qwen_gdn"] = gdn_refresh_keys(torch, args)
        torch.cuda.empty_cache()

    # roofline of the step's dominant kernel: the fused Load with refresh (or, with
    # --unfused-step, the refresh)
    if args.unfused_step:
        rk, r_ms, r_bytes = "refresh", t["refresh"], bytes_refresh
        r_what = (f"{bytes_refresh} B = per refreshed head: k, v (bf16), g, beta (fp32), restored "
                  "state read, omitted rows written")
    else:
        rk, r_ms, r_bytes = "restore_refresh", t["restore_refresh"], bytes_fused
        r_what = (f"{bytes_fused} B = per refreshed head: k, v (bf16), g, beta (fp32); per request: "
                  "each kept row of the checkpoint read once, every row of the layer written once")
    achieved = r_bytes / r_ms / 1e6          # GB/s
    step_desc = (f"pack {n_ckpt} checkpoints, restore {n_ckpt}, refresh {n_req} requests W={W}"
                 if args.unfused_step else
                 f"pack {n_ckpt} checkpoints, restore {n_ckpt - n_req}, Load with refresh of "
                 f"{n_req} requests W={W} (restore + replay in one launch)")
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
            "workload": f"KDA layer 32h x 128x128 fp32 (R={R} of {rows} rows kept): {step_desc}",
            "n_checkpoints": n_ckpt, "n_requests": n_req, "W": W, "rows_kept": R,
            "inputs": "k,v bf16; g,beta fp32; state fp32",
        },
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(f"kimi_headline/{rk}"), "kernel": rk,
                     "work_per_launch": r_what,
                     "mfma_frac": flops_refresh / (r_ms / 1e3) / 1e12 / BF16_MFMA_PEAK_TFLOPS,
                     "mfma_busy": measured_util(f"kimi_headline/{rk}", "mfma_busy"),
                     "valu_active": measured_util(f"kimi_headline/{rk}", "valu_active")},
        "first_pass_ms_per_step": first_ms,
        "kernels": kernels,
        "pack_restore_GBps": (bytes_pack + bytes_restore) / (t["pack"] + t["restore"]) / 1e6,
        "extra": extra,
        "plan_host_ms": plan_s * 1e3,
    }
    # 4. the oracle on the host cores
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_headline(wl, plan, states_np, inp, W, n_req)
    return out


# ---- CPU baseline: the oracle, as it stands ---------------------------------------------

def _oracle_sample(wl, plan, states_np, inp, W, n_req, threads):
    """Seconds the oracle takes on the bounded sample (pack and restore of every
    checkpoint, refresh of half the requests), its work split over `threads` host threads:
    checkpoints and (request, head) pairs are dealt to the threads, each of which calls the
    oracle's own functions on its share (numpy releases the interpreter lock inside its
    array loops, so the shares run in parallel)."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import pack as OK
    from oracle import recurrence as OR

    n_s, req_s = wl.n_ckpt, n_req // 2
    R = int(plan["n_rows"])
    words = states_np.reshape(states_np.shape[0], -1, wl.dv).view(np.uint32)
    ck_parts = [list(range(n_s))[i::threads] for i in range(threads)]
    pairs = [(n, h) for n in range(req_s) for h in range(wl.n_heads)]
    pair_parts = [pairs[i::threads] for i in range(threads)]
    sub = {key: val[:req_s] for key, val in inp.items()}

    def pack_restore(ids):
        ck = OK.pack(words, ids, plan["unit_row"], np.zeros((1, len(ids), R, wl.dv), np.uint32),
                     list(range(len(ids))))
        back = OK.restore(ck, list(range(len(ids))), plan["unit_row"],
                          np.zeros((len(ids),) + words.shape[1:], np.uint32), list(range(len(ids))))
        return back

    layer = np.ascontiguousarray(
        pack_restore(list(range(req_s))).view(np.float32).reshape(req_s, wl.n_heads, wl.dk, wl.dv))

    def refresh(ps):
        return OR.refresh(layer, plan["inv_row"], sub["k"], sub["v"], sub["g"], sub["beta"],
                          wl.n_qk_heads, pairs=ps)

    with ThreadPoolExecutor(threads) as ex:
        t0 = time.perf_counter()
        list(ex.map(pack_restore, [p for p in ck_parts if p]))
        t_pr = time.perf_counter() - t0
        t0 = time.perf_counter()
        list(ex.map(refresh, [p for p in pair_parts if p]))
        t_ref = time.perf_counter() - t0
    return t_pr, t_ref


def cpu_baseline_headline(wl, plan, states_np, inp, W, n_req):
    """The oracle, as it stands, on a bounded sample of the same step, timed on one host
    thread and on every host core this process may run on (at most MAX_POOL_THREADS)."""
    from threadpoolctl import threadpool_limits

    affinity = len(os.sched_getaffinity(0))
    n_all = max(1, min(affinity, MAX_POOL_THREADS))
    res = {}
    with threadpool_limits(1):              # no BLAS threads on top of the pool
        for threads in sorted({1, n_all}):
            t_pr, t_ref = _oracle_sample(wl, plan, states_np, inp, W, n_req, threads)
            step_s = t_pr + t_ref * n_req / (n_req // 2)
            res[threads] = {"value": n_req * W / step_s, "sample_seconds": t_pr + t_ref}
    best = res[n_all]
    return {"value": best["value"], "unit": "tokens/s", "cores": n_all, "kind": "oracle",
            "sample": f"pack+restore all {wl.n_ckpt} checkpoints, refresh {n_req // 2} of {n_req} "
                      f"requests x 32 heads at W={W} (fp64 per-token form); the refresh time is "
                      f"scaled to all requests; work dealt to {n_all} host threads",
            "sample_seconds": best["sample_seconds"],
            "one_thread": {"value": res[1]["value"], "sample_seconds": res[1]["sample_seconds"]},
            "host_cpus": os.cpu_count(), "affinity_cpus": affinity}


# ---- full-model KDA checkpoint set --------------------------------------------------------

def full_model_keys(torch, args, layouts=("ragged", "q8", "padded")):
    """Pack/restore of the full-model KDA set (24 layers x 32 heads, 256 checkpoints, T = 8
    rank slices), per-kernel durations by batched HIP events; GB-scale, so the rates are
    HBM rates."""
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS, states_device

    wl = WORKLOADS["kimi_model"]
    sh, plan, plan_s = _setup_plan(wl)
    R, rows, dv, n = int(plan["n_rows"]), sh.rows, sh.dv, wl.n_ckpt
    T, C = wl.n_ranks, int(plan["slice_rows"])
    states = states_device(wl, n, "cuda")
    active = torch.empty_like(states)
    unit_row, inv_row = _i32(torch, plan["unit_row"]), _i32(torch, plan["inv_row"])
    ids = _i32(torch, np.arange(n))
    bp = 2 * R * dv * 4 * n
    br = (R + rows) * dv * 4 * n
    kern = {}
    if "ragged" in layouts:
        ckpt = torch.empty((T, n, C, dv), dtype=torch.float32, device="cuda")
        kern["pack"] = _rate(batched_ms(torch, lambda: D.dasc_pack(
            sh, states, ids, unit_row, ckpt, ids, n_ranks=T, slice_rows=C), batches=5), bp)
        kern["restore"] = _rate(batched_ms(torch, lambda: D.dasc_restore(
            sh, ckpt, ids, inv_row, active, ids, n_rows=R, n_ranks=T, slice_rows=C), batches=5), br)
        del ckpt
    if "q8" in layouts:
        q = torch.empty((n, R, dv), dtype=torch.int8, device="cuda")
        s = torch.empty((n, R), dtype=torch.float32, device="cuda")
        kern["pack_q8"] = _rate(batched_ms(torch, lambda: D.dasc_pack_q8(
            sh, states, ids, unit_row, q, s, ids), batches=5), R * n * (dv * 4 + dv + 4))
        kern["restore_q8"] = _rate(batched_ms(torch, lambda: D.dasc_restore_q8(
            sh, q, s, ids, inv_row, active, ids, n_rows=R), batches=5), n * (R * (dv + 4) + rows * dv * 4))
        del q, s
    if "padded" in layouts:
        r_max = int(plan["r_max_rows"])
        off = _i32(torch, plan["layer_off_rows"])
        ck_pad = torch.empty((sh.n_layers, n, r_max, dv), dtype=torch.float32, device="cuda")
        kern["pack_padded"] = _rate(batched_ms(torch, lambda: D.dasc_pack_padded(
            sh, states, ids, unit_row, off, ck_pad, ids), batches=5), bp)
        kern["restore_padded"] = _rate(batched_ms(torch, lambda: D.dasc_restore_padded(
            sh, ck_pad, ids, off, inv_row, active, ids, n_rows=R), batches=5), br)
        del ck_pad
    del states, active
    return {"workload": f"{wl.n_layers} KDA layers x 32h x 128x128 fp32, {n} checkpoints, "
                        f"R={R} of {rows} rows kept, T={T} rank slices",
            "kernels": kern,
            "pack_restore_GBps": (bp + br) / (kern["pack"]["ms"] + kern["restore"]["ms"]) / 1e6
            if "ragged" in layouts else None,
            "checkpoint_bytes": {"fp32": R * dv * 4, "q8": R * (dv + 4),
                                 "padded": sh.n_layers * int(plan["r_max_rows"]) * dv * 4},
            "plan_host_ms": plan_s * 1e3}


def bench_full_model(torch, args):
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS

    res = full_model_keys(torch, args)
    wl_sh, plan, _ = _setup_plan(WORKLOADS["kimi_model"])
    k = res["kernels"]
    dom = "restore" if k["restore"]["ms"] >= k["pack"]["ms"] else "pack"
    return {
        "metric": "pack+restore GB/s (full-model KDA checkpoint set)",
        "value": res["pack_restore_GBps"], "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": k["pack"]["ms"] + k["restore"]["ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32",
        "data": "synthetic", "config": {"workload": res["workload"]},
        "roofline": {"bound": "hbm", "achieved": k[dom]["GBps"], "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": k[dom]["GBps"] / HBM_PEAK_GBPS,
                     "traffic": measured_traffic(f"kimi_model/{dom}"), "kernel": dom},
        "kernels": k, "checkpoint_bytes": res["checkpoint_bytes"],
        "tp_stage1": tp_stage1(D, wl_sh, plan, 8), "plan_host_ms": res["plan_host_ms"],
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


# ---- Qwen-GDN ------------------------------------------------------------------------------

def gdn_refresh_keys(torch, args, with_pack_restore=False, with_fused=False):
    """Refresh of the omitted v-heads of 8 requests over all 36 GDN layers at W = 1024
    (each layer: the factor launch and the recurrence launch), per-layer durations by
    batched HIP events.  Inputs are drawn on the device."""
    import paper_2608_30386_amd as D
    from workloads import WORKLOADS, log_lambda, refresh_inputs_device, states_device

    wl = WORKLOADS["qwen_gdn"]
    sh, plan, plan_s = _setup_plan(wl)
    R, rows, dv, W, n_req = int(plan["n_rows"]), sh.rows, sh.dv, args.W, wl.n_req
    n_pool = wl.n_ckpt if with_pack_restore else n_req
    states = states_device(wl, n_pool, "cuda")
    active = states.clone()
    inv_row = _i32(torch, plan["inv_row"])
    req = _i32(torch, np.arange(n_req))
    lam = log_lambda(wl)
    layers = [refresh_inputs_device(wl, W, lam[l], "cuda", salt=l) for l in range(wl.n_layers)]
    ws = torch.empty(D.dasc_refresh_workspace_bytes(sh, n_req, W), dtype=torch.uint8, device="cuda")

    def ref_all():
        for l, x in enumerate(layers):
            D.dasc_refresh(sh, l, inv_row, active, req, x["k"], x["v"], x["g"], x["beta"], W,
                           workspace=ws)

    ms_all = batched_ms(torch, ref_all, batches=5, per_batch=4)
    omitted = (plan["inv_row"].reshape(sh.n_layers, sh.n_heads, sh.dk) < 0).all(axis=2)
    heads = n_req * int(omitted.sum())
    # key heads some omitted v-head of their layer reads (v-heads of a group share one)
    key_heads = n_req * sum(len(set(np.flatnonzero(o) // (sh.n_heads // sh.n_qk_heads)))
                            for o in omitted)
    # per refreshed head: v (bf16), g, beta (fp32), the restored head read and written; per
    # key head read: k (bf16)
    per_head = 2 * W * dv + 4 * W + 4 * W + 2 * 4 * sh.dk * dv
    bytes_ref = heads * per_head + key_heads * 2 * W * sh.dk
    out = {"workload": f"Qwen-GDN 36 layers, 16 qk / 32 v heads 128x128: refresh {n_req} requests "
                       f"x {heads // n_req // wl.n_layers} omitted heads per layer, W={W}",
           "refresh_all_layers": {"tokens_per_s": n_req * W / (ms_all / 1e3), "launches": 2 * wl.n_layers,
                                  "per_layer_ms": ms_all / wl.n_layers, **_rate(ms_all, bytes_ref)},
           "bytes_per_layer": bytes_ref // wl.n_layers,
           "recurrence_TFLOPs": 5.0 * sh.dk * dv * W * heads / (ms_all / 1e3) / 1e12,
           "plan_host_ms": plan_s * 1e3}
    if with_fused:
        ckpt = torch.empty((n_pool, R, dv), dtype=torch.float32, device="cuda")
        ids = _i32(torch, np.arange(n_pool))
        D.dasc_pack(sh, states, ids, _i32(torch, plan["unit_row"]), ckpt, ids)

        def fused():
            for l, x in enumerate(layers):
                D.dasc_restore_refresh(sh, l, ckpt, req, inv_row, active, req, x["k"], x["v"], x["g"],
                                       x["beta"], W, n_rows=R, workspace=ws)
        t_restore = batched_ms(torch, lambda: D.dasc_restore(sh, ckpt, req, inv_row, active, req,
                                                             n_rows=R), batches=5)
        out["restore_refresh_fused"] = {"ms": batched_ms(torch, fused, batches=5, per_batch=4),
                                        "unfused_ms": t_restore + ms_all, "requests": n_req}
    if with_pack_restore:
        ckpt = torch.empty((n_pool, R, dv), dtype=torch.float32, device="cuda")
        ids = _i32(torch, np.arange(n_pool))
        unit_row = _i32(torch, plan["unit_row"])
        out["pack"] = _rate(batched_ms(torch, lambda: D.dasc_pack(sh, states, ids, unit_row, ckpt, ids),
                                       batches=5), 2 * R * dv * 4 * n_pool)
        out["restore"] = _rate(batched_ms(torch, lambda: D.dasc_restore(
            sh, ckpt, ids, inv_row, active, ids, n_rows=R), batches=5), (R + rows) * dv * 4 * n_pool)
    del states, active, layers, ws
    return out


def bench_gdn(torch, args):
    """Qwen-GDN shape: refresh 8 requests x 36 layers, fused Load, pack/restore 128
    checkpoints."""
    res = gdn_refresh_keys(torch, args, with_pack_restore=True, with_fused=True)
    r = res["refresh_all_layers"]
    return {
        "metric": "GDN refresh tokens/s (36 layers) + pack/restore GB/s",
        "value": r["tokens_per_s"], "unit": "tokens/s (all 36 layers)",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": r["ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic", "config": {"workload": res["workload"]},
        "roofline": {"bound": "hbm", "achieved": r["GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": r["hbm_frac"], "traffic": measured_traffic("qwen_gdn/refresh"),
                     "kernel": "refresh (factor + recurrence per layer)",
                     "mfma_busy": measured_util("qwen_gdn/refresh", "mfma_busy"),
                     "valu_active": measured_util("qwen_gdn/refresh", "valu_active")},
        "kernels": res,
    }


if __name__ == "__main__":
    main()
