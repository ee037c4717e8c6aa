#!/usr/bin/env python3
"""Benchmark of one frame of the read-sparse readout + store-sparse commit.

One step = select_queries + readout + commit for every object of one frame,
on synthetic inputs already resident in HBM, against a bank in steady state.
Default workload: 64x64 token grid, d_model 256, one head of 256, bank k/v
width 64, bf16, bank of 1 pinned conditioning frame + 6 recent frames pruned
to in-mask tokens, read keep ratio rho ~ U[0.15, 0.30] per frame.

Prints ONE JSON line (rank 0) with frames/s, the attention kernel's roofline
fraction (kernel durations from HIP events around its launches, live) and the
fp64 oracle's frames/s on this host as a reported CPU baseline.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "readout+commit frames/s at 64x64 grid, 7-frame bank; MFMA util %, HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
N_DISTINCT = 40   # distinct resident input frames cycled through by the steps


def _describe(cfg) -> str:
    obj = "1 object" if cfg.n_obj == 1 else "%d objects on one shared grid" % cfg.n_obj
    rho = ("rho %.2f" % cfg.rho) if cfg.rho is not None else ("rho ~ U[%.2f, %.2f]" % (cfg.rho_lo, cfg.rho_hi))
    return ("%s: %dx%d grid, %s, d_model %d, %d head(s) x %d, k/v %d, %s, bank %d pinned + %d recent frames "
            "(mask area %.2f-%.2f), %s" % (cfg.name, cfg.m, cfg.n, obj, cfg.C, cfg.H, cfg.d_h, cfg.d_kv, cfg.dtype,
                                           cfg.n_pin, cfg.f_max - cfg.n_pin, cfg.area_lo, cfg.area_hi, rho))


# ---------------------------------------------------------------------------
# CPU baseline (child process, fp64 oracle, one thread)
# ---------------------------------------------------------------------------
def cpu_child(workload: str, frames: int, rope_theta: float = 0.0, write_dw: int = -1):
    import numpy as np  # noqa: F401  (threads pinned by the parent's env)
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle
    from harness import OraclePipeline
    from workloads import CONFIGS, make_frame, make_sequence, make_weights
    cfg = CONFIGS[workload]
    n_pre = cfg.f_max
    seq = make_sequence(cfg, n_frames=n_pre + frames + 1)
    W = make_weights(cfg)
    orc = OraclePipeline(cfg, W, rope=oracle.axial_table(cfg.m, cfg.n, cfg.d_h, rope_theta) if rope_theta else None)
    keep = None
    if write_dw >= 0:
        from workloads import fall_counts
        lo, hi = fall_counts("0.05", "0.95", cfg.mn)
        keep = oracle.write_keepset(seq.masks[0], cfg.s, cfg.m, cfg.n, write_dw, lo, hi)[0].reshape(-1).astype(np.uint8)

    def commit(fr, t, pin):
        if keep is None:
            orc.commit(fr.Kmem, fr.Vmem, seq.masks[t], t, pin)
        else:
            for o in range(cfg.n_obj):
                orc.banks[o].commit(fr.Kmem[o], fr.Vmem[o], keep, t, pin)

    for t in range(n_pre):
        commit(make_frame(cfg, t), t, t < cfg.n_pin)
    t0 = time.perf_counter()
    for t in range(n_pre, n_pre + frames):
        fr = make_frame(cfg, t)
        sel, _ = orc.select(seq.read_mask(cfg, t), fr.X, seq.k[t])
        for o in range(cfg.n_obj):
            g = 0 if cfg.union_objects else o
            orc.readout_rows(fr.X, o, sel[g])
        commit(fr, t, False)
    dt = time.perf_counter() - t0
    print(json.dumps({"seconds": dt, "frames": frames, "prefill": n_pre}))


def cpu_baseline(workload: str, frames: int, rope_theta: float = 0.0, write_dw: int = -1):
    env = dict(os.environ)
    for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "NUMEXPR_NUM_THREADS"):
        env[v] = "1"
    env["HIP_VISIBLE_DEVICES"] = ""
    p = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-child", "--workload", workload,
                        "--cpu-frames", str(frames), "--rope", str(rope_theta), "--write-dw", str(write_dw)], stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True,
                       env=env, timeout=600)
    if p.returncode != 0:
        return {"value": None, "unit": "frames/s", "cores": 1, "kind": "oracle", "error": p.stderr[-500:]}
    r = json.loads(p.stdout.strip().splitlines()[-1])
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": r["frames"] / r["seconds"], "unit": "frames/s", "cores": 1, "kind": "oracle",
            "sample": "%d frames (select + readout of every selected row + commit) after a %d-frame prefill, "
                      "fp64 NumPy, 1 thread; host %s with %d cores available"
                      % (r["frames"], r.get("prefill", 0), cpu, len(os.sched_getaffinity(0))),
            "seconds": r["seconds"]}


# ---------------------------------------------------------------------------
# GPU run
# ---------------------------------------------------------------------------
def _kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("readout.hip", "device_util.h", "rs3_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2608_22526_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def _traffic(kernel: str):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.txt" % kernel)
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != _kernel_source_hash():
        return None
    return d.get("bytes_per_launch")


def _absorb(cfg, layer: str) -> bool:
    """Single-head layers with a narrower bank run the attention on the raw
    bank rows (W_k folded into the query, W_v into the output projection)."""
    if layer == "absorbed":
        return True
    if layer == "projected":
        return False
    return cfg.H == 1 and cfg.d_kv < cfg.D


def made_events(torch, n, timing=False):
    """n events whose HIP objects exist already: torch creates an event's HIP
    object on its first record, which costs 10-40 us of host time, so every
    event a timed region records is recorded once here, before it starts."""
    evs = [torch.cuda.Event(enable_timing=timing) for _ in range(n)]
    for e in evs:
        e.record()
    torch.cuda.synchronize()
    return evs


class QueueWindow:
    """Keeps at most about `window` frames queued ahead of the GPU: every
    `every` frames an event is recorded, and before queueing more the host
    waits for the event from `window` frames earlier.  The GPU always has
    work queued; the host never runs into the runtime's slow path for a full
    launch queue (hundreds of queued launches with large argument blocks)."""

    def __init__(self, torch, window=48, every=8):
        self.torch, self.window, self.every = torch, window, every
        self.events = {}
        # events are made here, outside any timed region, and reused
        self.pool = made_events(torch, window // every + 2)

    def before(self, i):
        if i % self.every == 0:
            ev = self.events.pop(i - self.window, None)
            if ev is not None:
                ev.synchronize()
                self.pool.append(ev)

    def after(self, i):
        if i % self.every == 0:
            ev = self.pool.pop() if self.pool else self.torch.cuda.Event()
            ev.record()
            self.events[i] = ev


def _fixed_keepset(torch, rs3, sess, cfg, seed_masks, D_w):
    """The paper's write keep-set K_w (Eq. 8) from the first frame's masks,
    once per sequence, as the commit mask of every object (grid stride 1).
    Returns (keep [n_obj][mn] u8 on the device, |K_w|, kernel us)."""
    from workloads import fall_counts
    if cfg.s != 1:
        raise SystemExit("the fixed write keep-set workloads use stride-1 grids")
    lo, hi = fall_counts("0.05", "0.95", cfg.mn)
    keep = torch.zeros((cfg.n_obj, cfg.mn), dtype=torch.uint8, device="cuda")
    counts = torch.zeros(2, dtype=torch.int32, device="cuda")
    ev = made_events(torch, 2, timing=True)
    rs3.write_keepset(sess.grid, cfg.n_obj, seed_masks, D_w, lo, hi, cfg.n_obj, keep, counts)   # warm
    ev[0].record()
    for _ in range(10):
        rs3.write_keepset(sess.grid, cfg.n_obj, seed_masks, D_w, lo, hi, cfg.n_obj, keep, counts)
    ev[1].record()
    torch.cuda.synchronize()
    return keep, int(counts[1].item()), 1000.0 * ev[0].elapsed_time(ev[1]) / 10


def gpu_run(args):
    import numpy as np
    import torch
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device
    from workloads import CONFIGS, make_frame, make_sequence, make_weights

    cfg = CONFIGS[args.workload]
    if args.objects:
        # that many objects per call, each on a grid of its own
        from dataclasses import replace
        cfg = replace(cfg, n_obj=args.objects, shared_x=False, union_objects=False)
    dev = "cuda"
    n_pre = cfg.f_max
    seq = make_sequence(cfg, n_frames=n_pre + N_DISTINCT)
    W = make_weights(cfg)
    k_all = [max(ks) for ks in seq.k]
    absorb = _absorb(cfg, args.layer) and not args.rope
    sess = Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype,
                   n_obj=cfg.n_obj, shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap,
                   f_max=cfg.f_max, n_pin=cfg.n_pin, weights=W, r_s=cfg.r_s, c=cfg.c, max_sel=max(k_all),
                   n_splits=args.splits, absorb=absorb, rope_theta=args.rope or None)
    # resident inputs
    frames = []
    for t in range(n_pre + N_DISTINCT):
        fr = make_frame(cfg, t)
        frames.append(dict(X=to_device(fr.X), K=to_device(fr.Kmem), V=to_device(fr.Vmem),
                           mask=to_device(seq.masks[t]), rmask=to_device(seq.read_mask(cfg, t)), k=seq.k[t],
                           max_sel=max(seq.k[t])))
    in_place = cfg.n_obj == 1
    Y = None if in_place else torch.empty((cfg.n_obj, cfg.mn, cfg.C), dtype=frames[0]["X"].dtype, device=dev)
    fixed = None
    if args.write_dw >= 0:
        keep, kw, kw_us = _fixed_keepset(torch, rs3, sess, cfg, frames[0]["mask"], args.write_dw)
        fixed = {"D_w": args.write_dw, "keep_cells": kw, "keepset_kernel_us": kw_us}
        for f in frames:
            f["mask"] = keep
    for t in range(n_pre):
        f = frames[t]
        sess.commit(f["K"], f["V"], f["mask"], t, t < cfg.n_pin)

    step_t = [n_pre]
    main = torch.cuda.current_stream()
    two = args.streams == 2
    calls = "separate" if (two or args.separate) else args.calls
    fused = calls == "readout_commit"
    side = torch.cuda.Stream() if two else main
    ev_read = torch.cuda.Event()
    ev_commit = torch.cuda.Event()
    ev_commit.record(main)

    def step(record=None):
        # The selection of frame t needs only frame t's read mask and tokens,
        # so it runs while frame t-1's commit is still in flight on the side
        # stream; the readout waits for that commit (its bank must hold frame
        # t-1), and frame t's commit waits for the readout.
        t = step_t[0]
        f = frames[n_pre + (t - n_pre) % N_DISTINCT]
        if calls == "frame":
            # the whole frame in one call (rs3_frame)
            if record is not None:
                nk = [b.info()["n_keys"] for b in sess.banks]
            sess.frame(f["rmask"], f["X"], f["k"], f["X"] if in_place else Y, f["K"], f["V"], f["mask"], t, False,
                       max_sel=f["max_sel"])
            if record is not None:
                cnt = sess.sel_count.cpu().numpy()
                g = [0 if cfg.union_objects else o for o in range(cfg.n_obj)]
                record.append(dict(sel=[int(cnt[g[o]]) for o in range(cfg.n_obj)], n_keys=nk))
            step_t[0] += 1
            return
        sess.select(f["rmask"], f["X"], f["k"])
        if two:
            main.wait_event(ev_commit)
        if record is not None:
            cnt = sess.sel_count.cpu().numpy()
            nk = [b.info()["n_keys"] for b in sess.banks]
            g = [0 if cfg.union_objects else o for o in range(cfg.n_obj)]
            record.append(dict(sel=[int(cnt[g[o]]) for o in range(cfg.n_obj)], n_keys=nk))
        if fused:
            # readout and commit in one call (the split merge and the commit
            # share one launch)
            sess.readout_commit(f["X"], f["X"] if in_place else Y, f["K"], f["V"], f["mask"], t, False,
                                max_sel=f["max_sel"])
            step_t[0] += 1
            return
        if in_place:
            sess.readout(f["X"], f["X"], max_sel=f["max_sel"])
        else:
            sess.readout(f["X"], Y, max_sel=f["max_sel"])
        if two:
            ev_read.record(main)
            side.wait_event(ev_read)
            sess.commit(f["K"], f["V"], f["mask"], t, False, stream=side.cuda_stream)
            ev_commit.record(side)
        else:
            sess.commit(f["K"], f["V"], f["mask"], t, False)
        step_t[0] += 1

    if args.copy_probe_mb > 0:
        # kernels of known traffic that calibrate the HBM byte counters: a fill
        # (writes nb bytes), a sum (reads nb bytes) and a device copy (both)
        nb = args.copy_probe_mb << 20
        src_t = torch.ones(nb // 4, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        float(src_t.sum())
        dst_t = torch.empty_like(src_t)
        dst_t.copy_(src_t)
        torch.cuda.synchronize()
        del src_t, dst_t
    for i in range(args.warmup):
        if i % 8 == 7:
            torch.cuda.synchronize()
        step()
    torch.cuda.synchronize()
    # pass A: frames/s, no instrumentation
    ev0, ev1 = made_events(torch, 2, timing=True)
    qw = QueueWindow(torch)
    enq = []
    torch.cuda.synchronize()
    ev0.record(main)
    h0 = time.perf_counter()
    for i in range(args.steps):
        qw.before(i)
        t_in = time.perf_counter()
        step()
        enq.append(time.perf_counter() - t_in)
        qw.after(i)
    host_loop_us = (time.perf_counter() - h0) * 1e6 / args.steps
    main.wait_event(ev_commit)
    ev1.record(main)
    torch.cuda.synchronize()
    host_us = float(np.median(enq)) * 1e6   # (after the end event: numpy's first call can take tens of ms)
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / args.steps
    fps = 1000.0 / ms_step
    graph = _graph_pass(torch, step, args.steps) if not two and args.graph else None
    # pass B: per-kernel durations from HIP events around each launch
    rs3.profile_enable(True, 16 * args.steps + 64)
    rs3.profile_reset()
    recs = []
    for _ in range(args.steps):
        step(record=recs)   # synchronises every frame (records its sizes)
    torch.cuda.synchronize()
    rep = rs3.profile_report()
    rs3.profile_enable(False)
    errs = [b.error() for b in sess.banks]

    # algorithmic attention flops (the method's work: QK^T and PV at the model
    # width D = H*d_h, whatever width the kernel runs at) and executed flops
    # (QK^T and PV at the kernel's attention width, plus the query projection
    # when the attention kernel does it)
    Da = cfg.d_kv if absorb else cfg.D
    attn_ms, attn_n = rep["attn"]
    alg_flops = sum(4.0 * r["sel"][o] * r["n_keys"][o] * cfg.D for r in recs for o in range(cfg.n_obj))
    exec_flops = sum(4.0 * r["sel"][o] * r["n_keys"][o] * Da for r in recs for o in range(cfg.n_obj))
    sel_tot = sum(sum(r["sel"]) for r in recs)
    # the frame call of a single 64-wide head at d_model 256 projects every
    # cell's query in the energy launch; otherwise launches without a separate
    # projection kernel project their queries inside the attention
    pre_projected = calls == "frame" and cfg.dtype == "bf16" and absorb and Da == 64 and cfg.C == 256 \
        and not args.rope and rep.get("qproj", (0.0, 0))[1] == 0
    if pre_projected:
        proj_share = 0.0
    else:
        proj_share = 1.0 - (rep.get("qproj", (0.0, 0))[1] / attn_n if attn_n else 0.0)
    exec_flops += proj_share * sum(2.0 * r["sel"][o] * cfg.C * Da for r in recs for o in range(cfg.n_obj))
    avg_attn_s = attn_ms / 1000.0 / max(attn_n, 1)
    alg_per_launch = alg_flops / max(attn_n, 1)
    exec_per_launch = exec_flops / max(attn_n, 1)
    achieved_tflops = alg_per_launch / avg_attn_s / 1e12 if attn_n else 0.0
    exec_tflops = exec_per_launch / avg_attn_s / 1e12 if attn_n else 0.0
    kernels = {}
    for name, (ms, n) in rep.items():
        if n and not name.startswith("_"):
            kernels[name] = {"launches": n, "avg_us": 1000.0 * ms / n, "us_per_step": 1000.0 * ms / args.steps}
    kernel_sum_us = sum(v["us_per_step"] for v in kernels.values())
    traffic = _traffic("attn_%s_%s" % (cfg.name, "absorbed" if absorb else "projected"))
    out = {
        "metric": METRIC,
        "value": fps,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": _describe(cfg), "grid": "%dx%d" % (cfg.m, cfg.n), "n_obj": cfg.n_obj,
                   "bank_frames": cfg.f_max, "d_model": cfg.C, "heads": cfg.H, "d_head": cfg.d_h,
                   "d_kv": cfg.d_kv, "eager_launches": True, "streams": args.streams,
                   "calls": {"separate": "select + readout + commit", "readout_commit": "select + readout_commit",
                             "frame": "rs3_frame (select + readout + commit in one call)"}[calls],
                   "readout": "in place" if in_place else "out of place",
                   "attention": ("absorbed: one head of width d_kv=%d on the raw bank rows" % cfg.d_kv) if absorb
                   else ("projected: %d head(s) of width %d%s" % (cfg.H, cfg.d_h,
                         ", axial rotary table (theta %g) on queries and keys" % args.rope if args.rope else ""))},
        "roofline": {"bound": "mfma", "achieved": achieved_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved_tflops / PEAK_BF16_TFLOPS,
                     "traffic": traffic,
                     "kernel": ("k_attn_g2 (split-KV attention, heads of 64; queries projected by the energy launch)"
                                if pre_projected else "k_attn (split-KV attention)"),
                     "flops_per_launch": alg_per_launch,
                     "flops_basis": "algorithmic: 4 * selected queries * bank keys * D (D = H * d_h = %d), the "
                                    "method's QK^T and PV at the model width" % cfg.D,
                     "executed_flops_per_launch": exec_per_launch,
                     "executed_achieved": exec_tflops,
                     "executed_frac": exec_tflops / PEAK_BF16_TFLOPS,
                     "executed_basis": ("4 * selected * keys * %d (the kernel's attention width%s)%s"
                                        % (Da, ", absorbed" if absorb else "",
                                           "" if proj_share == 0.0 else
                                           " + 2 * selected * d_model * width for the query projection inside"
                                           " the kernel (%.0f%% of launches)" % (100.0 * proj_share))),
                     "avg_launch_us": avg_attn_s * 1e6},
        "extra": {
            "query_tokens_per_s": sel_tot / args.steps * fps,
            "grid_tokens_per_s": cfg.n_obj * cfg.mn * fps,
            "mean_selected_per_frame": sel_tot / args.steps,
            "mean_bank_keys": sum(sum(r["n_keys"]) for r in recs) / len(recs) / cfg.n_obj,
            "kernels": kernels,
            "kernel_sum_us_per_step": kernel_sum_us,
            "bank_errors": errs,
            "splits": sess.n_splits,
            "host_enqueue_us_per_step": host_us,
            "host_enqueue_basis": "median host time inside one frame's calls (argument marshalling, validation and "
                                  "the kernel launches), without the waits of the bounded queue",
            "host_loop_us_per_step": host_loop_us,
            "hip_graph": graph,
            "fixed_write_keepset": fixed,
            "copy_bandwidth": copy_bandwidth() if args.copy_bw else None,
            "read_bandwidth": read_bandwidth() if args.copy_bw else None,
        },
    }
    return out


# ---------------------------------------------------------------------------
# The L-layer memory-attention stack (rs3_stack_readout) in the frame
# ---------------------------------------------------------------------------
STACK_F = 2048
STACK_METRIC = "select + L-layer memory-attention stack + commit frames/s at 64x64 grid, 7-frame bank"


def _stack_flops(n, N, L, C, F, d_kv):
    """Algorithmic flops of one stack call on n kept rows and N bank keys:
    (matrix products, self-attention, cross-attention)."""
    gemm = 2.0 * n * C * (3 * C) + 2.0 * n * C * C + 2.0 * n * C * d_kv + 2.0 * n * d_kv * C + 4.0 * n * C * F
    return L * gemm, L * 4.0 * n * n * C, L * 4.0 * n * N * d_kv


def cpu_child_stack(workload: str, frames: int, n_layers: int, H_s: int):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    from harness import OraclePipeline
    from oracle import stack as ostack
    from workloads import CONFIGS, make_frame, make_sequence, make_stack_weights, make_weights, storage_to_f64
    cfg = CONFIGS[workload]
    n_pre = cfg.f_max
    seq = make_sequence(cfg, n_frames=n_pre + frames + 1)
    orc = OraclePipeline(cfg, make_weights(cfg))
    ws = [{k: (storage_to_f64(v, "bf16") if v.dtype == np.uint16 else v.astype(np.float64)) for k, v in w.items()}
          for w in make_stack_weights(cfg.C, cfg.d_kv, STACK_F, n_layers, "bf16", seed=0)]
    for t in range(n_pre):
        orc.commit(make_frame(cfg, t).Kmem, make_frame(cfg, t).Vmem, seq.masks[t], t, t < cfg.n_pin)
    t0 = time.perf_counter()
    for t in range(n_pre, n_pre + frames):
        fr = make_frame(cfg, t)
        sel, _ = orc.select(seq.read_mask(cfg, t), fr.X, seq.k[t])
        K, V, _ = orc.banks[0].key_rows()
        ostack.stack(storage_to_f64(fr.X[0], cfg.dtype), sel[0], storage_to_f64(K, cfg.dtype),
                     storage_to_f64(V, cfg.dtype), ws, H_s, 1)
        orc.commit(fr.Kmem, fr.Vmem, seq.masks[t], t, False)
    dt = time.perf_counter() - t0
    print(json.dumps({"seconds": dt, "frames": frames, "prefill": n_pre}))


def cpu_baseline_stack(workload: str, frames: int, n_layers: int, H_s: int):
    env = dict(os.environ)
    for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "NUMEXPR_NUM_THREADS"):
        env[v] = "1"
    env["HIP_VISIBLE_DEVICES"] = ""
    p = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-child", "--workload", workload,
                        "--cpu-frames", str(frames), "--stack", str(n_layers), "--stack-heads", str(H_s)],
                       stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, env=env, timeout=600)
    if p.returncode != 0:
        return {"value": None, "unit": "frames/s", "cores": 1, "kind": "oracle", "error": p.stderr[-500:]}
    r = json.loads(p.stdout.strip().splitlines()[-1])
    return {"value": r["frames"] / r["seconds"], "unit": "frames/s", "cores": 1, "kind": "oracle",
            "sample": "%d frame(s) (select + the %d-layer stack row by row on the kept rows + commit) after a "
                      "%d-frame prefill, fp64 NumPy, 1 thread" % (r["frames"], n_layers, r.get("prefill", 0)),
            "seconds": r["seconds"]}


def gpu_run_stack(args):
    import numpy as np
    import torch
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device
    from workloads import CONFIGS, make_frame, make_sequence, make_stack_weights, make_weights

    cfg = CONFIGS[args.workload]
    if cfg.dtype != "bf16" or cfg.C != 256 or cfg.d_kv != 64 or cfg.n_obj != 1:
        raise SystemExit("--stack runs single-object bf16 workloads of d_model 256 and bank rows of 64")
    L, H_s = args.stack, args.stack_heads
    n_pre = cfg.f_max
    seq = make_sequence(cfg, n_frames=n_pre + N_DISTINCT)
    k_all = [max(ks) for ks in seq.k]
    sess = Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=1,
                   shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap, f_max=cfg.f_max,
                   n_pin=cfg.n_pin, weights=make_weights(cfg), r_s=cfg.r_s, c=cfg.c, max_sel=max(k_all),
                   absorb=True)
    stack = rs3.Stack(make_stack_weights(cfg.C, cfg.d_kv, STACK_F, L, "bf16", seed=0), H_s=H_s, F=STACK_F)
    ws = torch.empty(stack.workspace_size(max(k_all), args.splits), dtype=torch.uint8, device="cuda")
    Y = torch.empty((cfg.mn, cfg.C), dtype=torch.bfloat16, device="cuda")
    frames = []
    for t in range(n_pre + N_DISTINCT):
        fr = make_frame(cfg, t)
        frames.append(dict(X=to_device(fr.X), K=to_device(fr.Kmem), V=to_device(fr.Vmem),
                           mask=to_device(seq.masks[t]), rmask=to_device(seq.read_mask(cfg, t)), k=seq.k[t],
                           max_sel=max(seq.k[t])))
    for t in range(n_pre):
        f = frames[t]
        sess.commit(f["K"], f["V"], f["mask"], t, t < cfg.n_pin)
    step_t = [n_pre]
    bank = sess.banks[0]

    def step(record=None):
        t = step_t[0]
        f = frames[n_pre + (t - n_pre) % N_DISTINCT]
        sess.select(f["rmask"], f["X"], f["k"])
        if record is not None:
            record.append(dict(sel=int(sess.sel_count.cpu()[0]), n_keys=bank.info()["n_keys"]))
        stack.readout(sess.grid, f["X"], bank, sess.sel_idx, sess.sel_count, f["max_sel"], Y, 0, ws, args.splits)
        sess.commit(f["K"], f["V"], f["mask"], t, False)
        step_t[0] += 1

    for i in range(args.warmup):
        if i % 8 == 7:
            torch.cuda.synchronize()
        step()
    torch.cuda.synchronize()
    main = torch.cuda.current_stream()
    ev0, ev1 = made_events(torch, 2, timing=True)
    qw = QueueWindow(torch, window=16, every=4)
    enq = []
    torch.cuda.synchronize()
    ev0.record(main)
    h0 = time.perf_counter()
    for i in range(args.steps):
        qw.before(i)
        t_in = time.perf_counter()
        step()
        enq.append(time.perf_counter() - t_in)
        qw.after(i)
    host_loop_us = (time.perf_counter() - h0) * 1e6 / args.steps
    ev1.record(main)
    torch.cuda.synchronize()
    host_us = float(np.median(enq)) * 1e6   # (after the end event: numpy's first call can take tens of ms)
    ms_step = ev0.elapsed_time(ev1) / args.steps
    fps = 1000.0 / ms_step
    graph = _graph_pass(torch, step, args.steps) if args.graph else None
    rs3.profile_enable(True, (8 * L + 8) * args.steps + 64)
    rs3.profile_reset()
    recs = []
    for _ in range(args.steps):
        step(record=recs)
    torch.cuda.synchronize()
    rep = rs3.profile_report()
    rs3.profile_enable(False)
    fl = [_stack_flops(r["sel"], r["n_keys"], L, cfg.C, STACK_F, cfg.d_kv) for r in recs]
    gemm_fl, sa_fl, ca_fl = (sum(f[i] for f in fl) for i in range(3))
    kernels = {}
    for name, (ms, n) in rep.items():
        if n and not name.startswith("_"):
            kernels[name] = {"launches": n, "avg_us": 1000.0 * ms / n, "us_per_step": 1000.0 * ms / args.steps}
    g_ms, g_n = rep["stack_gemm"]
    a_ms, a_n = rep["attn"]
    gemm_tf = gemm_fl / (g_ms / 1000.0) / 1e12 if g_ms else 0.0
    attn_tf = (sa_fl + ca_fl) / (a_ms / 1000.0) / 1e12 if a_ms else 0.0
    dom = "stack_gemm" if g_ms >= a_ms else "attn"
    ach = gemm_tf if dom == "stack_gemm" else attn_tf
    per_launch = (gemm_fl / max(g_n, 1)) if dom == "stack_gemm" else ((sa_fl + ca_fl) / max(a_n, 1))
    sel_mean = sum(r["sel"] for r in recs) / len(recs)
    return {
        "metric": STACK_METRIC,
        "value": fps,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": _describe(cfg) + "; memory attention: %d-layer stack on the kept rows "
                   "(self-attention %d head(s) of %d, cross-attention one absorbed head on the raw bank rows, "
                   "MLP %d hidden), fp32 residual stream, bf16 output out of place" % (L, H_s, cfg.C // H_s,
                                                                                      STACK_F),
                   "grid": "%dx%d" % (cfg.m, cfg.n), "layers": L, "d_model": cfg.C, "self_heads": H_s,
                   "mlp_hidden": STACK_F, "d_kv": cfg.d_kv, "bank_frames": cfg.f_max},
        "roofline": {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": ach / PEAK_BF16_TFLOPS, "traffic": None,
                     "kernel": "k_stk_gemm (all products of the stack)" if dom == "stack_gemm"
                     else "k_attn (self- and cross-attention of the stack)",
                     "flops_per_launch": per_launch,
                     "flops_basis": "algorithmic: per layer 2n*C*(3C + C + 2 d_kv) + 4n*C*F for the products, "
                                    "4n^2*C self-attention, 4n*N*d_kv cross-attention (n kept rows, N bank keys)",
                     "avg_launch_us": 1000.0 * (g_ms / max(g_n, 1) if dom == "stack_gemm" else a_ms / max(a_n, 1))},
        "extra": {
            "mean_selected_per_frame": sel_mean,
            "mean_bank_keys": sum(r["n_keys"] for r in recs) / len(recs),
            "stack_gemm_TFLOP_s": gemm_tf,
            "attention_TFLOP_s": attn_tf,
            "flops_per_frame": {"products": gemm_fl / len(recs), "self_attention": sa_fl / len(recs),
                                "cross_attention": ca_fl / len(recs)},
            "kernels": kernels,
            "kernel_sum_us_per_step": sum(v["us_per_step"] for v in kernels.values()),
            "bank_errors": [bank.error()],
            "host_enqueue_us_per_step": host_us,
            "host_loop_us_per_step": host_loop_us,
            "hip_graph": graph,
        },
    }


def _graph_pass(torch, step, steps):
    """Frames/s with the frame sequence replayed from one captured HIP graph
    (the N_DISTINCT resident input frames, one graph launch each pass): the
    same kernels with the per-launch host work removed."""
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for _ in range(N_DISTINCT):
            step()
    torch.cuda.synchronize()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    reps = max(1, -(-steps // N_DISTINCT))
    e0, e1 = made_events(torch, 2, timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / (reps * N_DISTINCT)
    del g
    return {"frames_per_s": 1000.0 / ms, "ms_per_step": ms, "frames_timed": reps * N_DISTINCT,
            "frames_per_graph": N_DISTINCT}


# ---------------------------------------------------------------------------
# Report mode: every workload, the 128x128 keep-ratio sweep, the bank-length
# curve of the long video and the object-count sweep (one JSON file).
# ---------------------------------------------------------------------------
def _algo_bytes(cfg, absorb, rec):
    """Algorithmic bytes per frame of each kernel for one recorded frame:
    what the step must move (split partials are implementation traffic and
    are not counted), not what the kernel happens to move."""
    b = 2 if cfg.dtype == "bf16" else 4
    Da = cfg.d_kv if absorb else cfg.D
    n_x = 1 if cfg.shared_x else cfg.n_obj
    sel, kept, nk = rec["sel"], rec["kept"], rec["n_keys"]
    mn, C, dkv = cfg.mn, cfg.C, cfg.d_kv
    return {
        "energy": n_x * mn * (C * b + 8),
        "select": cfg.n_obj * mn * cfg.s * cfg.s + 8 * mn * len(set(rec["groups"])) + 4 * sum(sel),
        "qproj": sum(q * (C * b + Da * 2) for q in sel) + Da * C * 2,
        "attn": sum(n * Da * 2 * 2 + q * Da * 2 * 2 for q, n in zip(sel, nk)),
        "combine": sum(q * (Da * 2 + 2 * C * b) for q in sel) + C * Da * 2,
        "commit": cfg.n_obj * mn + sum(k * (4 + 4 * dkv * b + 2 * Da * 2) for k in kept),
        # the split merge with the scatter and the commit in one launch
        "merge_commit": sum(q * (Da * 2 + 2 * C * b) for q in sel) + C * Da * 2
                        + cfg.n_obj * mn + sum(k * (4 + 4 * dkv * b + 2 * Da * 2) for k in kept),
    }


def run_workload(cfg, *, absorb, steps, warmup, commit=True, prefill=None, splits=0, rope_theta=None,
                 write_dw=-1, separate=False):
    """Steady-state frames of `cfg` (objects beyond 64 run as several calls per
    frame).  separate: select, readout and commit as three calls (the split
    merge with the scatter, and the commit, then run as launches of their own).
    Returns frame timing percentiles, per-kernel times and rates."""
    import numpy as np
    import torch
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import Session, to_device
    from workloads import make_frame, make_sequence, make_weights

    n_pre = cfg.f_max if prefill is None else prefill
    # distinct resident input frames: fewer when every object has its own grid
    n_gen = 2 if cfg.n_obj > 64 else n_pre + (8 if cfg.n_obj > 8 else N_DISTINCT)
    n_dist = n_gen if cfg.n_obj > 64 else n_gen - n_pre
    seq = make_sequence(cfg, n_frames=n_pre + n_dist)
    W = make_weights(cfg)
    chunks = [(o0, min(64, cfg.n_obj - o0)) for o0 in range(0, cfg.n_obj, 64)]
    max_sel = max(max(ks) for ks in seq.k)
    sessions = [Session(m=cfg.m, n=cfg.n, s=cfg.s, C=cfg.C, H=cfg.H, d_kv=cfg.d_kv, dtype=cfg.dtype, n_obj=no,
                        shared_x=cfg.shared_x, union_objects=cfg.union_objects, cap=cfg.cap, f_max=cfg.f_max,
                        n_pin=cfg.n_pin, weights=W, r_s=cfg.r_s, c=cfg.c, max_sel=max_sel, n_splits=splits,
                        absorb=absorb, rope_theta=rope_theta) for _, no in chunks]
    frames = []
    for t in range(n_gen):
        fr = make_frame(cfg, t)
        per = []
        for (o0, no) in chunks:
            xs = slice(0, 1) if cfg.shared_x else slice(o0, o0 + no)
            per.append(dict(X=to_device(fr.X[xs]), K=to_device(fr.Kmem[o0:o0 + no]), V=to_device(fr.Vmem[o0:o0 + no]),
                            mask=to_device(seq.masks[t][o0:o0 + no]),
                            rmask=to_device(seq.read_mask(cfg, t)[o0:o0 + no]),
                            k=seq.k[t] if cfg.union_objects else seq.k[t][o0:o0 + no]))
        frames.append(dict(per=per, max_sel=max(seq.k[t])))
    keep_cells = None
    if write_dw >= 0:
        if len(sessions) != 1:
            raise SystemExit("the fixed write keep-set workloads run one call per frame")
        keep, keep_cells, _ = _fixed_keepset(torch, rs3, sessions[0], cfg, frames[0]["per"][0]["mask"], write_dw)
        for fr_ in frames:
            fr_["per"][0]["mask"] = keep
    outs = [None if no == 1 else
            torch.empty((no, cfg.mn, cfg.C), dtype=frames[0]["per"][0]["X"].dtype, device="cuda") for _, no in chunks]
    def frame_of(t):
        return t % n_gen if cfg.n_obj > 64 else (t if t < n_pre else n_pre + (t - n_pre) % n_dist)

    for t in range(n_pre):
        for ci, sess in enumerate(sessions):
            f = frames[frame_of(t)]["per"][ci]
            sess.commit(f["K"], f["V"], f["mask"], t, t < cfg.n_pin)
    step_t = [n_pre]

    def step():
        t = step_t[0]
        fi = frame_of(t)
        for ci, sess in enumerate(sessions):
            f = frames[fi]["per"][ci]
            Y = outs[ci]
            if commit and separate:
                sess.select(f["rmask"], f["X"], f["k"])
                sess.readout(f["X"], f["X"] if Y is None else Y, max_sel=frames[fi]["max_sel"])
                sess.commit(f["K"], f["V"], f["mask"], t, False)
            elif commit:   # the whole frame in one call
                sess.frame(f["rmask"], f["X"], f["k"], f["X"] if Y is None else Y, f["K"], f["V"], f["mask"], t,
                           False, max_sel=frames[fi]["max_sel"])
            else:
                sess.select(f["rmask"], f["X"], f["k"])
                sess.readout(f["X"], f["X"] if Y is None else Y, max_sel=frames[fi]["max_sel"])
        if commit:
            step_t[0] += 1

    for i in range(warmup):
        if i % 8 == 7:
            torch.cuda.synchronize()
        step()
    torch.cuda.synchronize()
    ev = made_events(torch, steps + 1, timing=True)
    ev[0].record()
    for i in range(steps):
        if i >= 48:
            ev[i - 48].synchronize()   # bounded queue (see QueueWindow)
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per_frame = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]) * 1e3
    total_ms = ev[0].elapsed_time(ev[steps])
    rs3.profile_enable(True, 16 * steps * len(sessions) + 64)
    rs3.profile_reset()
    for i in range(steps):
        if i % 16 == 15:
            torch.cuda.synchronize()
        step()
    torch.cuda.synchronize()
    rep = rs3.profile_report()
    rs3.profile_enable(False)
    # frame contents (selected, kept, bank keys) on a few frames
    recs = []
    for _ in range(3):
        step()
        torch.cuda.synchronize()
        sel, kept, nks, groups = [], [], [], []
        for sess in sessions:
            cnt = sess.sel_count.cpu().numpy()
            for o in range(sess.n_obj):
                g = 0 if cfg.union_objects else o
                sel.append(int(cnt[g]))
                groups.append((id(sess), g))
            kept += [int(v) for v in sess.kept_count.cpu().numpy()] if commit else [0] * sess.n_obj
            nks += [b.info()["n_keys"] for b in sess.banks]
        recs.append(dict(sel=sel, kept=kept, n_keys=nks, groups=groups))
    Da = cfg.d_kv if absorb else cfg.D
    fps = 1000.0 * steps / total_ms
    kern = {}
    byt = [_algo_bytes(cfg, absorb, r) for r in recs]
    for name, (ms, n) in rep.items():
        if not n:
            continue
        launches_per_frame = n / steps
        avg_us = 1000.0 * ms / n
        d = {"avg_us": avg_us, "launches_per_frame": launches_per_frame}
        if name in byt[0]:
            bytes_frame = sum(b_[name] for b_ in byt) / len(byt)
            d["algo_bytes_per_frame"] = bytes_frame
            d["GB_s"] = bytes_frame / launches_per_frame / (avg_us * 1e-6) / 1e9
            d["frac_hbm"] = d["GB_s"] / PEAK_HBM_GBS
        kern[name] = d
    attn_flops = sum(4.0 * q * n * Da for r in recs for q, n in zip(r["sel"], r["n_keys"])) / len(recs)
    alg_flops = sum(4.0 * q * n * cfg.D for r in recs for q, n in zip(r["sel"], r["n_keys"])) / len(recs)
    if "attn" in kern:
        # executed: QK^T and PV at the kernel's attention width; algorithmic:
        # the same at the model width D (what the method computes)
        a = kern["attn"]
        a["flops_per_frame"] = attn_flops
        a["TFLOP_s"] = attn_flops / a["launches_per_frame"] / (a["avg_us"] * 1e-6) / 1e12
        a["frac_mfma"] = a["TFLOP_s"] / PEAK_BF16_TFLOPS
        a["algorithmic_flops_per_frame"] = alg_flops
        a["TFLOP_s_algorithmic"] = alg_flops / a["launches_per_frame"] / (a["avg_us"] * 1e-6) / 1e12
        a["frac_mfma_algorithmic"] = a["TFLOP_s_algorithmic"] / PEAK_BF16_TFLOPS
    q_frame = sum(sum(r["sel"]) for r in recs) / len(recs)
    k_frame = sum(sum(r["kept"]) for r in recs) / len(recs)
    return {
        "frames_per_s": fps, "ms_per_frame": total_ms / steps,
        "frame_us_p10_p50_p90": [float(np.percentile(per_frame, q)) for q in (10, 50, 90)],
        "query_tokens_per_s": q_frame * fps, "committed_tokens_per_s": k_frame * fps,
        "grid_tokens_per_s": cfg.n_obj * cfg.mn * fps,
        "selected_per_frame": q_frame, "kept_per_frame": k_frame,
        "bank_keys_mean": sum(sum(r["n_keys"]) for r in recs) / len(recs) / cfg.n_obj,
        "kernels": kern, "attention_width": Da, "objects": cfg.n_obj, "calls_per_frame": len(sessions),
        "fixed_write_keep_cells": keep_cells,
    }


def read_bandwidth(mib: int = 512, reps: int = 10):
    """Rate of the library's read-only streaming kernel (rs3_stream_read: 16-byte
    loads, xor-reduced per thread) over `mib` MiB, larger than the 256 MB
    Infinity Cache: the reference for kernels that mostly read (the energies
    read every grid row once).  Returns GB/s of bytes read."""
    import torch
    import paper_2608_22526_amd as rs3
    nb = mib << 20
    src = torch.ones(nb // 4, dtype=torch.int32, device="cuda")
    out = torch.empty(rs3.RS3_STREAM_READ_THREADS, dtype=torch.int32, device="cuda")
    rs3.stream_read(src, nb, out)
    torch.cuda.synchronize()
    ev = made_events(torch, 2, timing=True)
    ev[0].record()
    for _ in range(reps):
        rs3.stream_read(src, nb, out)
    ev[1].record()
    torch.cuda.synchronize()
    s_per = ev[0].elapsed_time(ev[1]) / 1000.0 / reps
    # every word is 1: each thread xors an even or odd number of them
    x = out.cpu().numpy()
    ok = bool(((x == 0) | (x == 1)).all())
    return {"GB_s": nb / s_per / 1e9, "bytes_read": float(nb), "us_per_read": s_per * 1e6, "result_ok": ok,
            "kernel": "rs3_stream_read (16-byte loads, four in flight per thread, %d threads)"
                      % rs3.RS3_STREAM_READ_THREADS}


def copy_bandwidth(mib: int = 512, reps: int = 10):
    """Bandwidth of the library's own grid copy kernel (the out-of-place
    readout's X -> Y copy: a readout with no selected row launches only that
    copy) on `mib` MiB read and `mib` MiB written: 64 per-object bf16 grids of
    d_model 256, larger than the 256 MB Infinity Cache together.  Returns
    GB/s of bytes read + written."""
    import numpy as np
    import torch
    import paper_2608_22526_amd as rs3
    n_obj = 64
    mn = mib * (1 << 20) // (n_obj * 256 * 2)
    m = 1
    while m * m < mn:
        m *= 2
    n = mn // m
    C = 256
    w = np.zeros((C, C), np.uint16)
    wk = np.zeros((64, C), np.uint16)
    layer = rs3.Layer(C, 1, 64, rs3.RS3_BF16, w, wk, wk, w, absorb=True)
    banks = [rs3.Bank(layer, 64, 2, 0) for _ in range(n_obj)]
    X = torch.empty((n_obj, m * n, C), dtype=torch.bfloat16, device="cuda").fill_(1.0)
    Y = torch.empty_like(X)
    sel = torch.zeros((n_obj, m * n), dtype=torch.int32, device="cuda")
    cnt = torch.zeros(n_obj, dtype=torch.int32, device="cuda")
    ws = torch.zeros(256, dtype=torch.uint8, device="cuda")

    def once():
        rs3.readout(layer, (m, n, 1), n_obj, X, m * n * C, banks, sel, cnt, m * n, 0, 0, Y, m * n * C, ws=ws)
    once()
    torch.cuda.synchronize()
    ev = made_events(torch, 2, timing=True)
    ev[0].record()
    for _ in range(reps):
        once()
    ev[1].record()
    torch.cuda.synchronize()
    s_per = ev[0].elapsed_time(ev[1]) / 1000.0 / reps
    moved = 2.0 * X.numel() * 2
    ok = bool(torch.equal(X, Y))
    del X, Y
    return {"GB_s": moved / s_per / 1e9, "bytes_read_plus_written": moved, "us_per_copy": s_per * 1e6,
            "copy_exact": ok, "kernel": "k_copy_grid16 (16-byte vectors, grid-stride)"}


def run_post(n_obj, H, W, k=9, reps=50):
    """The closure and palette step on decoder logits of n_obj x H x W (bf16):
    time per call and algorithmic bandwidth (logits read once, closed masks
    and palette written once)."""
    import torch
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import to_device
    from workloads import make_decoder_logits
    L = to_device(make_decoder_logits(n_obj, H, W, seed=1))
    ws = torch.zeros(rs3.close_workspace_size(n_obj, H, W), dtype=torch.uint8, device="cuda")
    closed = torch.empty((n_obj, H, W), dtype=torch.uint8, device="cuda")
    pal = torch.empty((H, W), dtype=torch.uint8, device="cuda")
    for _ in range(5):
        rs3.close_masks(n_obj, H, W, L, rs3.RS3_BF16, k, closed, pal, ws)
    ev = made_events(torch, 2, timing=True)
    ev[0].record()
    for _ in range(reps):
        rs3.close_masks(n_obj, H, W, L, rs3.RS3_BF16, k, closed, pal, ws)
    ev[1].record()
    torch.cuda.synchronize()
    us = 1000.0 * ev[0].elapsed_time(ev[1]) / reps
    algo = n_obj * H * W * 2 + n_obj * H * W + H * W
    return {"us_per_call": us, "algo_bytes": algo, "GB_s": algo / (us * 1e-6) / 1e9,
            "frac_hbm": algo / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}


def report(args):
    from dataclasses import replace
    from workloads import CONFIGS
    out = {"device": "one MI355X", "steps": args.steps}

    def log(tag, r):
        print("%-34s %9.0f frames/s  p50 %7.1f us  attn %s" % (
            tag, r["frames_per_s"], r["frame_us_p10_p50_p90"][1],
            ("%.1f us %.1f TF/s" % (r["kernels"]["attn"]["avg_us"], r["kernels"]["attn"]["TFLOP_s"]))
            if "attn" in r["kernels"] else "-"), flush=True)

    # the runtime's one-time launch-argument pool growth happens here, untimed
    run_workload(CONFIGS["sam2_single"], absorb=True, steps=8, warmup=400)
    for name in ("tiny_f32", "sam2_single", "multi_obj8", "long_video", "highres"):
        cfg = CONFIGS[name]
        for mode in (("absorbed", "projected") if cfg.H == 1 and cfg.dtype == "bf16" else ("projected",)):
            r = run_workload(cfg, absorb=mode == "absorbed", steps=args.steps, warmup=args.warmup)
            out["%s/%s" % (name, mode)] = r
            log("%s/%s" % (name, mode), r)
    # rotary positions on the gathered subset (Eq. 7): projected layers only
    for name in ("sam2_single", "highres"):
        cfg = CONFIGS[name]
        r = run_workload(cfg, absorb=False, steps=args.steps, warmup=args.warmup, rope_theta=10000.0)
        out["%s/projected+rope" % name] = r
        log("%s/projected+rope" % name, r)
    # closure of the decoded masks and the palette (Sec. 3.3), 9x9
    for (no, H, W) in ((1, 256, 256), (8, 256, 256), (1, 1024, 1024), (8, 1024, 1024)):
        r = run_post(no, H, W)
        out["post/%dx%dx%d" % (no, H, W)] = r
        print("post %d x %dx%d: %.1f us, %.0f GB/s" % (no, H, W, r["us_per_call"], r["GB_s"]), flush=True)
    # the paper's own write rule (Eq. 8): every frame written at the fixed
    # keep-set of the first frame's mask, default and aggressive radius
    for D_w in (24, 12):
        for name in ("sam2_single", "long_video"):
            r = run_workload(CONFIGS[name], absorb=True, steps=args.steps, warmup=args.warmup, write_dw=D_w)
            out["%s/absorbed+fixed_write%d" % (name, D_w)] = r
            log("%s/absorbed fixed write D_w=%d" % (name, D_w), r)
    hr = CONFIGS["highres"]
    for rho in ("0.1", "0.25", "0.5", "1.0"):
        cfg = replace(hr, rho=float(rho))
        r = run_workload(cfg, absorb=False, steps=max(5, args.steps // 4), warmup=3)
        out["highres_rho/%s" % rho] = r
        log("highres rho=%s" % rho, r)
    lv = CONFIGS["long_video"]
    for L in (1, 2, 4, 8, 16, 32, 64):
        for mode in ("absorbed", "projected"):
            r = run_workload(lv, absorb=mode == "absorbed", steps=max(5, args.steps // 4), warmup=3, commit=False,
                             prefill=L)
            out["long_video_bank/%d/%s" % (L, mode)] = r
            log("long_video L=%d %s" % (L, mode), r)
    base = CONFIGS["multi_obj8"]
    for B in (1, 8, 64, 512):
        cfg = replace(base, n_obj=B, shared_x=False, union_objects=False)
        r = run_workload(cfg, absorb=True, steps=max(3, args.steps // 8), warmup=2)
        out["objects/%d" % B] = r
        log("objects B=%d (per-object grids)" % B, r)
    # the scatter (split merge + W_o + residual) and the commit as launches of
    # their own, with the library's copy kernel as the bandwidth reference
    out["copy_bandwidth"] = copy_bandwidth()
    print("copy kernel: %.0f GB/s" % out["copy_bandwidth"]["GB_s"], flush=True)
    out["read_bandwidth"] = read_bandwidth()
    print("read-only stream: %.0f GB/s" % out["read_bandwidth"]["GB_s"], flush=True)
    for B in (1, 8, 64, 512):
        cfg = replace(base, n_obj=B, shared_x=False, union_objects=False) if B > 1 else CONFIGS["sam2_single"]
        r = run_workload(cfg, absorb=True, steps=max(3, args.steps // 8) if B > 8 else args.steps, warmup=2 if B > 8
                         else args.warmup, separate=True)
        out["separate/%d" % B] = r
        log("separate launches B=%d" % B, r)
        print("   " + ", ".join("%s %.0f GB/s" % (k, v["GB_s"]) for k, v in r["kernels"].items() if "GB_s" in v),
              flush=True)
    with open(args.report, "w") as fh:
        json.dump(out, fh, indent=1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=400,
                    help="untimed frames first; the HIP runtime grows its launch-argument pool once "
                         "(a stall of tens of ms) after the first thousand-odd launches of a process")
    ap.add_argument("--workload", default="sam2_single")
    ap.add_argument("--objects", type=int, default=0,
                    help="objects per call (at most 64), each on a grid of its own; 0 keeps the workload's")
    ap.add_argument("--splits", type=int, default=0)
    ap.add_argument("--write-dw", type=int, default=-1,
                    help="write every frame at the fixed keep-set K_w of this dilation radius (Eq. 8), built "
                         "from the first frame's masks; -1 = each frame's own mask")
    ap.add_argument("--rope", type=float, default=0.0,
                    help="axial rotary table with this theta on a projected layer (0 = none)")
    ap.add_argument("--layer", choices=["auto", "projected", "absorbed"], default="auto")
    ap.add_argument("--streams", type=int, choices=[1, 2], default=1,
                    help="2: frame t's commit overlaps frame t+1's selection on a second stream")
    ap.add_argument("--separate", action="store_true",
                    help="select, readout and commit as three calls (same as --calls separate)")
    ap.add_argument("--calls", choices=["frame", "readout_commit", "separate"], default="frame",
                    help="frame: one rs3_frame call per frame (default); readout_commit: rs3_select_queries + "
                         "rs3_readout_commit; separate: select, readout and commit")
    ap.add_argument("--no-graph", dest="graph", action="store_false",
                    help="skip the HIP-graph replay pass (reported beside the eager frames/s)")
    ap.add_argument("--cpu-frames", type=int, default=40)
    ap.add_argument("--copy-probe-mb", type=int, default=0)
    ap.add_argument("--no-copy-bw", dest="copy_bw", action="store_false",
                    help="skip the measurement of the library's copy-kernel bandwidth (512 MiB each way)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-child", action="store_true")
    ap.add_argument("--report", default="", help="write the full measurement report (JSON) to this path")
    ap.add_argument("--post-only", action="store_true", help="time only the closure and palette step")
    ap.add_argument("--stack", type=int, default=0,
                    help="run the frame with an L-layer memory-attention stack on the kept rows (rs3_stack_readout) "
                         "in place of the single readout layer; 0 = the single layer")
    ap.add_argument("--stack-heads", type=int, default=1, help="self-attention heads of the stack")
    args = ap.parse_args()
    if args.cpu_child:
        if args.stack:
            cpu_child_stack(args.workload, args.cpu_frames, args.stack, args.stack_heads)
        else:
            cpu_child(args.workload, args.cpu_frames, args.rope, args.write_dw)
        return
    if args.rope and args.layer == "absorbed":
        print("--rope needs a projected layer: the rotation sits between the projections that absorption "
              "folds together", file=sys.stderr)
        sys.exit(2)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one MI355X: the path runs on a single GPU (objects or bank frames would be "
              "sharded across GPUs with no exchange, which this benchmark does not launch). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    if args.objects and (args.objects > 64 or args.stack or not args.no_cpu_baseline):
        print("--objects takes 1 to 64 objects per call, without --stack, with --no-cpu-baseline (the oracle "
              "baseline times the workload's own objects)", file=sys.stderr)
        sys.exit(2)
    if args.post_only:
        for (no, H, W) in ((1, 256, 256), (8, 256, 256), (1, 1024, 1024), (8, 1024, 1024)):
            print(json.dumps({"post": [no, H, W], **run_post(no, H, W)}), flush=True)
        return
    if args.report:
        report(args)
        return
    if args.stack:
        out = gpu_run_stack(args)
        if not args.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline_stack(args.workload, 2, args.stack, args.stack_heads)
        print(json.dumps(out))
        return
    out = gpu_run(args)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_frames, args.rope, args.write_dw)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
