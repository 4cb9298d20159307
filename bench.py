#!/usr/bin/env python
"""Throughput of the pruned RNN-T loss (forward + backward) on one MI355X.

One step is the whole path on one batch resident in HBM:
  trivial joiner + full-lattice forward/backward + d am, d lm (simple loss,
  scaled 0.5 as in Sec. 3.3), pruning bounds, the full joiner on the pruned
  (t, u) pairs, the pruned recursion, the joiner backward to d enc, d dec,
  dW, db, and the training loss (0.5 simple + pruned, summed).
No [N, T, S, V] array is kept: the joiner's forward reduces its logits to
lse and the target / blank log-probs, and the backward recomputes them in
chunks of rows whose size does not depend on N or T.
The headline workload is the BPE-sized batch (N=16, T ~ U[150,250],
U ~ U[20,60], V=500, S=5, J=512, fp32), synthetic and seeded; frames = sum of
valid T_n.

Prints one JSON line: frames/s, peak HBM bytes, the roofline of the dominant
contraction (HIP events recorded by the library on the launch stream around
that kernel only, during the timed steps), a per-kernel census from a short
untimed pass with every launch bracketed, the same step with the logits kept
between forward and backward (`kept_logits`), the long-batch workload (bf16
joiner, V=500, S=5) measured the same way (`long`), and the CPU oracle's
throughput on the host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}  # MI355X dense MFMA
PEAK_HBM_GBS = 8000.0

WORKLOAD_TEXT = {
    "bpe": "bpe: N=16, T~U[150,250], U~U[20,60], V=500, S=5, J=512, fp32 joiner",
    "long": "long: N=32, T~U[300,500], U~U[50,100], V=500, S=5, J=512, bf16 joiner",
    "largev": "largev: N=16, T~U[200,300], U~U[40,80], V=5000 (Zipf 1.1 symbols), S=5, J=512, fp32 joiner",
    "stress": "stress: N=8, T~U[800,1000], U~U[200,300] (25% U=T/3), V=8000, S=10, J=768, bf16 joiner",
}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "joiner_hbm_traffic_bpe.md")
BRACKET_EVERY = 4  # timed steps per step whose dominant kernel is bracketed by HIP events


def _traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed FETCH_SIZE / WRITE_SIZE
    runs (scaled by the copy calibration), or None when they were not taken on
    this workload or the kernel's sources changed since."""
    import hashlib
    import re
    if workload != "bpe" or not os.path.exists(TRAFFIC_FILE):
        return None
    m = re.search(r"```json\n(.*?)```", open(TRAFFIC_FILE).read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    h = hashlib.sha256()
    for f in rec["sources"]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    k = rec["kernels"].get(kernel)
    if h.hexdigest() != rec["sources_sha256"] or k is None:
        return None
    return int(1024 * (k["fetch_kib"] * rec["fetch_scale"] + k["write_kib"] * rec["write_scale"]))


def _unpruned(P, batch, enc, dec, W, bias, frames, dev, steps: int = 5) -> dict:
    """The unpruned loss with the same joiner at every (t, u), its (N, T, U+1, V)
    logits kept (as a framework materialising them would), on the same batch:
    the comparison of the method's speed and memory claims (Sec. 1, Sec. 3.2)."""
    import torch
    N, T, U = batch.N, batch.T, batch.U
    J, V = int(W.shape[0]), int(W.shape[1])
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated(dev)
    torch.cuda.reset_peak_memory_stats(dev)
    f32 = dict(dtype=torch.float32, device=dev)
    bufs = dict(loss=torch.empty(N, **f32), enc_grad=torch.empty(N, T, J, **f32),
                dec_grad=torch.empty(N, U + 1, J, **f32), W_grad=torch.empty(J, V, **f32),
                bias_grad=torch.empty(V, **f32), logits=torch.empty(N, T, U + 1, V, **f32))
    ws = torch.empty(P.full_loss_workspace_size(N, T, U, J, V, P._jdtype(W)), dtype=torch.uint8, device=dev)
    P.rnnt_full_loss(batch, enc, dec, W, bias, workspace=ws, **bufs)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        P.rnnt_full_loss(batch, enc, dec, W, bias, workspace=ws, **bufs)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    peak = torch.cuda.max_memory_allocated(dev) - base
    del bufs, ws
    torch.cuda.empty_cache()
    return {"what": "unpruned RNN-T loss + gradients, same joiner at every (t, u), logits [N,T,U+1,V] kept",
            "ms_per_step": round(ms, 4), "frames_per_s": round(frames / (ms / 1000.0), 1),
            "peak_hbm_bytes_excl_inputs": int(peak), "steps": steps}


def _band_algorithms(P, batch, S, out, reps: int = 20) -> dict:
    """The pruned recursion alone (loss and band occupations), each algorithm
    on this workload's own band log-probs and bounds from one step: the
    anti-diagonal wavefront (depth T_n + U_n) and the chunked scan over frames
    (depth about 2C + T_n / C)."""
    import torch
    px, py, rg = out["px"], out["py"], out["ranges"]
    N, T, U = batch.N, batch.T, batch.U
    res = {}
    for alg, chunk in (("wavefront", 0), ("scan", 0)):
        nbytes = P.pruned_loss_workspace_size(N, T, U, S, alg, chunk)
        if nbytes == 0:
            continue  # S beyond what the algorithm supports
        ws = torch.empty(nbytes, dtype=torch.uint8, device=px.device)
        loss = torch.empty(N, dtype=torch.float32, device=px.device)
        gx, gy = torch.empty_like(px), torch.empty_like(px)
        run = lambda: P.rnnt_pruned_loss(batch, S, px, py, rg, loss=loss, px_occ=gx, py_occ=gy, workspace=ws,
                                         algorithm=alg, chunk=chunk)
        for _ in range(3):
            run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        torch.cuda.synchronize()
        res[alg] = {"us_per_call": round(1000 * e0.elapsed_time(e1) / reps, 1), "workspace_bytes": nbytes}
    res["auto"] = "scan" if S <= 16 else "wavefront"
    res["reps"] = reps
    return res


_CPU_BATCH = None


def _cpu_worker_init():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _cpu_one(n):
    """The oracle's whole path on utterance n of the batch (stages 1-4 with gradients)."""
    import numpy as np

    import oracle as O
    b = _CPU_BATCH
    sl = slice(n, n + 1)
    S = b.wl.S
    s1 = O.simple_stage(b.am[sl], b.lm[sl], b.symbols[sl], b.t_len[sl], b.u_len[sl], b.wl.blank,
                        scale=np.full(1, 0.5))
    r = O.prune_ranges(s1["gx"], s1["gy"], b.t_len[sl], b.u_len[sl], S)
    O.pruned_stage(b.enc[sl], b.dec[sl], b.W, b.bias, r, b.symbols[sl], b.t_len[sl], b.u_len[sl], b.wl.blank)
    return int(b.t_len[n])


def _cpu_baseline(b, budget_s: float) -> dict:
    """The CPU oracle (as is) on the utterances of the same batch, one
    utterance per task over a pool of worker processes (one BLAS thread
    each, one per host core up to 16), in whole passes over the batch for
    about budget_s seconds. Run before the GPU is touched (the workers are
    forked)."""
    import multiprocessing as mp
    global _CPU_BATCH
    _CPU_BATCH = b
    workers = max(1, min(16, os.cpu_count() or 1))
    ctx = mp.get_context("fork")
    frames = done = 0
    with ctx.Pool(workers, initializer=_cpu_worker_init) as pool:
        t0 = time.perf_counter()
        while True:
            frames += sum(pool.map(_cpu_one, list(range(b.N)) * max(1, workers // b.N), chunksize=1))
            done += b.N * max(1, workers // b.N)
            if time.perf_counter() - t0 > budget_s:
                break
        dt = time.perf_counter() - t0
    return {"value": round(frames / dt, 2), "unit": "frames/s", "cores": workers, "kind": "oracle",
            "sample": f"{done} utterance runs over the {b.N} utterances of the same batch ({frames} frames), "
                      f"full oracle path (trivial joiner, lattice, am/lm grads, bounds, pruned joiner, pruned "
                      f"lattice, joiner grads), fp64 NumPy, {workers} processes with 1 BLAS thread each, "
                      f"{dt:.1f} s"}


def _measure(P, _native, b, args, keep_logits: bool, roofline: bool, census: bool, spread: bool,
             settle_s: float = 0.0) -> dict:
    """One workload's step on the GPU: warm-up, optionally a census pass with
    every kernel bracketed, then the timed steps (the dominant contraction
    bracketed by HIP events on every BRACKET_EVERY-th step when `roofline`)."""
    import ctypes

    import numpy as np
    import torch

    dev = torch.device("cuda:0")
    bf = b.wl.joiner_dtype == "bf16"
    S, J, V = b.wl.S, b.wl.J, b.V
    frames = b.frames
    M = S * frames
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev)
    jt = (lambda a: f32(a).to(torch.bfloat16)) if bf else f32
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats(dev)
    base_mem = torch.cuda.memory_allocated(dev)
    batch = P.Batch(i32(b.t_len), i32(b.u_len), i32(b.symbols), b.T, b.U, b.wl.blank)
    am, lm = f32(b.am), f32(b.lm)
    enc, dec, W, bias = jt(b.enc), jt(b.dec), jt(b.W), jt(b.bias)
    inputs_mem = torch.cuda.memory_allocated(dev) - base_mem
    step = P.PrunedRnntLoss(S, simple_scale=0.5, keep_logits=keep_logits)
    run = lambda: step.step(batch, am, lm, enc, dec, W, bias)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    if settle_s > 0:
        # untimed steps until the device has run busy for settle_s seconds:
        # after a long idle phase (the CPU baseline) the first ~0.5 s of work
        # run measurably slower than steady state
        t_end = time.perf_counter() + settle_s
        while time.perf_counter() < t_end:
            for _ in range(10):
                run()
            torch.cuda.synchronize()
    L = _native.lib()

    def kernel_table(nsteps):
        buf = ctypes.create_string_buffer(4096)
        L.rnnt_profile_names(buf, 4096)
        out = {}
        for name in [x for x in buf.value.decode().split(",") if x]:
            n = ctypes.c_int32()
            tot = ctypes.c_double()
            _native.check(L.rnnt_profile_query(name.encode(), ctypes.byref(n), ctypes.byref(tot)))
            out[name] = {"launches": n.value, "avg_us": round(1000 * tot.value / max(n.value, 1), 2),
                         "us_per_step": round(1000 * tot.value / nsteps, 2)}
        return out

    res = {}
    kernels = None
    if census or roofline:
        if args.copy_mib > 0 and census:
            src = torch.ones(args.copy_mib << 18, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            torch.cuda.synchronize()
            dst.copy_(src)
            torch.cuda.synchronize()
            del src, dst
        # census: every kernel bracketed by events, outside the timed region
        # (the event packets themselves cost ~5 us per launch)
        census_steps = max(1, min(args.steps, 5))
        L.rnnt_profile_reset()
        L.rnnt_profile_select(None)
        L.rnnt_profile_enable(1)
        for _ in range(census_steps):
            run()
        torch.cuda.synchronize()
        L.rnnt_profile_enable(0)
        kernels = kernel_table(census_steps)
        L.rnnt_profile_reset()
        if census:
            res["kernels"] = kernels
            res["kernels_census_steps"] = census_steps
    # the dominant contraction among the joiner GEMMs, algorithmic work per
    # step: 2 M J V for the forward, for dh and for dW; the recomputed
    # path's pipelined backward launches ("joiner_bwd": the next chunk's
    # recomputed logits with the current chunk's dh and dW) do dh and dW,
    # 4 M J V per step (the recomputation is overhead: time, not work)
    work = {"joiner_fwd": 2.0 * M * J * V, "joiner_dh": 2.0 * M * J * V, "joiner_dw": 2.0 * M * J * V,
            "joiner_bwd": 4.0 * M * J * V}
    dom = None
    if roofline:
        dom = max((k for k in work if k in kernels), key=lambda k: kernels[k]["us_per_step"])
        L.rnnt_profile_select(dom.encode())
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        if roofline:
            L.rnnt_profile_enable(1 if i % BRACKET_EVERY == BRACKET_EVERY - 1 or args.steps < BRACKET_EVERY else 0)
        run()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    L.rnnt_profile_enable(0)
    ms_total = ev0.elapsed_time(ev1)
    peak = torch.cuda.max_memory_allocated(dev) - base_mem
    res.update({"value": round(frames * args.steps / (ms_total / 1000.0), 1),
                "ms_per_step": round(ms_total / args.steps, 4), "peak_hbm_bytes": int(peak),
                "peak_hbm_bytes_excl_inputs": int(peak - inputs_mem), "wall_s_timed": round(wall, 3),
                "frames": frames, "rows_M": M, "dtype": "bf16" if bf else "f32"})
    if roofline:
        timed = kernel_table(args.steps)[dom]
        L.rnnt_profile_reset()
        L.rnnt_profile_select(None)
        per_launch_flops = work[dom] / (kernels[dom]["launches"] / res.get("kernels_census_steps", 5))
        achieved = per_launch_flops / (timed["avg_us"] * 1e-6) / 1e12
        dt = res["dtype"]
        res["roofline"] = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS[dt],
                           "unit": "TFLOP/s", "frac": round(achieved / PEAK_TFLOPS[dt], 4),
                           "traffic": _traffic(dom, b.wl.name),
                           "algorithmic_flops_per_launch": per_launch_flops, "avg_launch_us": timed["avg_us"],
                           "launches_timed": timed["launches"],
                           "bracketed_steps": f"every {BRACKET_EVERY}th timed step"}
    if spread:
        # step-time spread (after the timed region): each step bracketed on its own
        per_step = []
        for _ in range(args.steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            run()
            e1.record(stream)
            e1.synchronize()
            per_step.append(e0.elapsed_time(e1))
        q = np.percentile(np.asarray(per_step), [10, 50, 90])
        res["ms_per_step_spread"] = {"p10": round(float(q[0]), 4), "median": round(float(q[1]), 4),
                                     "p90": round(float(q[2]), 4), "steps": len(per_step),
                                     "note": "each step bracketed by its own events, after the timed region"}
    res["_ctx"] = (step, batch, enc, dec, W, bias, run)
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="bpe", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--keep-logits", action="store_true",
                    help="headline step with the [N,T,S,V] logits kept between forward and backward")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unpruned", action="store_true",
                    help="skip the comparison with the unpruned loss (same joiner at every (t, u))")
    ap.add_argument("--no-band-algorithms", action="store_true",
                    help="skip timing the pruned recursion's algorithms one by one")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the kept-logits step and the long-batch workload")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="before the census, run one device-to-device copy of this many MiB (a plain copy "
                         "kernel of known size that scales rocprofv3's FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the loss is per utterance, "
              "so a batch shards over GPUs by utterance with no communication in the loss itself). "
              "Run with --gpus 1.",
              file=sys.stderr)
        return 2

    from workloads import make_batch
    b = make_batch(args.workload, seed=0)
    # the CPU baseline first, in forked workers, before anything touches the GPU
    cpu = None if args.no_cpu_baseline else _cpu_baseline(b, args.cpu_budget)

    import torch

    import paper_2206_13236_amd as P
    from paper_2206_13236_amd import _native

    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch.zeros(1, device=dev)
    torch.cuda.synchronize()

    head = _measure(P, _native, b, args, keep_logits=args.keep_logits, roofline=True, census=True, spread=True,
                    settle_s=0.5)
    step, batch, enc, dec, W, bias, run = head.pop("_ctx")
    band = None if args.no_band_algorithms else _band_algorithms(P, batch, b.wl.S, run())
    unpruned = None if args.no_unpruned else _unpruned(P, batch, enc, dec, W, bias, b.frames, dev)
    del step, batch, enc, dec, W, bias, run
    extra = {}
    if not args.no_extra:
        # the same workload with the logits kept (one GEMM less, [N,T,S,V] more memory)
        k = _measure(P, _native, b, args, keep_logits=not args.keep_logits, roofline=False, census=False,
                     spread=False)
        k.pop("_ctx")
        extra["kept_logits" if not args.keep_logits else "recomputed_logits"] = {
            "what": "same step with the [N,T,S,V] logits " + ("kept" if not args.keep_logits else "not kept"),
            **{key: k[key] for key in ("value", "ms_per_step", "peak_hbm_bytes", "peak_hbm_bytes_excl_inputs")}}
        if args.workload != "long":
            bl = make_batch("long", seed=0)
            lg = _measure(P, _native, bl, args, keep_logits=args.keep_logits, roofline=True, census=False,
                          spread=False)
            lg.pop("_ctx")
            extra["long"] = {"workload": WORKLOAD_TEXT["long"], "frames_per_step": bl.frames,
                             **{key: lg[key] for key in ("value", "ms_per_step", "peak_hbm_bytes",
                                                         "peak_hbm_bytes_excl_inputs", "dtype", "roofline")}}
    S, J, V = b.wl.S, b.wl.J, b.V
    line = {
        "metric": "pruned RNN-T loss fwd+bwd frames/sec at V=500,S=5; peak HBM bytes",
        "value": head["value"],
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "ms_per_step_spread": head["ms_per_step_spread"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "frames_per_step": b.frames, "rows_M": head["rows_M"],
                   "N": b.N, "T": b.T, "U": b.U, "V": V, "S": S, "J": J, "seed": 0,
                   "logits_kept": bool(args.keep_logits)},
        "peak_hbm_bytes": head["peak_hbm_bytes"],
        "peak_hbm_bytes_excl_inputs": head["peak_hbm_bytes_excl_inputs"],
        "wall_s_timed": head["wall_s_timed"],
        "roofline": head["roofline"],
        **extra,
        "band_algorithms": band,
        "unpruned": unpruned,
        "kernels": head["kernels"],
        "kernels_census_steps": head["kernels_census_steps"],
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
