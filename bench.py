#!/usr/bin/env python3
"""Benchmark of OctreeNCA inference on one MI355X.

One step = one whole octree inference (octree_nca_infer: pyramid, coarsest
seed, per level upsample + inject and the level's NCA steps, readout) over one
synthetic input already resident in HBM.  Default workload: the 184.5 MP
pathology-scale 2D image (16384 x 11264 RGB, 6 levels, 20 steps per level,
fp32 state).

Prints one JSON line with
* value = NCA cell-steps per second (sum over levels of cells x steps, per
  second of wall time of the timed passes);
* roofline of the dominant kernel (the fused NCA step): algorithmic FLOP per
  cell-step x cell-steps of all timed step launches / their summed duration,
  timed with HIP events on the launch stream, against the peak of the
  arithmetic the kernel runs on;
* cpu_baseline: the CPU oracle timed on a bounded sample of the same workload;
* peak device memory;
* under "workloads", the same record (value, ms per pass, roofline, peak
  memory) for further workloads timed in the same run (default: the one-minute
  2D+t video, 1800 x 240 x 432 RGB, fp16 states, 5 levels, 16 steps each; the
  320 x 320 x 24 volume, fp32 states, 3 levels; the 1024 x 1024 2D image,
  4 levels).
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

# MI355X published peaks
HBM_PEAK_GBS = 8000.0
FP32_VECTOR_PEAK_TFLOPS = 157.3      # packed fp32 FMA
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0     # dense
FP16_MFMA_PEAK_TFLOPS = 2500.0     # dense
# The library is built without packed fp32 VALU instructions: one fp32 FMA per
# lane per clock, 256 CUs x 4 SIMDs x 16 lanes x 2 FLOP x 2.4 GHz.
FP32_SCALAR_FMA_PEAK_TFLOPS = 256 * 4 * 16 * 2 * 2.4e9 / 1e12


def algorithmic_flop_per_cell_step(wl) -> int:
    """Multiply-adds the method itself needs per cell and step, x2, plus the
    bias, ReLU and residual adds: perception C*taps MACs + C bias adds;
    first linear 2C*H MACs + H bias adds + H ReLU; second linear
    H*(C-n_in) MACs; residual (C-n_in) adds."""
    c, h, taps, hid = wl.channels, wl.hidden, wl.taps(), wl.channels - wl.n_in
    return 2 * (c * taps + 2 * c * h + h * hid) + c + h + h + hid


def algorithmic_train_flop_per_cell_step(wl) -> int:
    """Forward and backward of one training step per cell: the forward
    (algorithmic_flop_per_cell_step) twice (once in the forward pass, once
    recomputed by the backward), then W2^T gu (2 H (C-n_in)), the ReLU mask
    (H), W1^T ga (2 H 2C), dW1 += ga f^T (2 H 2C), dW2 += gu h^T (2 (C-n_in) H),
    db1 (H), dconv_b (C), dconv_w (2 C taps), the transposed convolution
    (2 C taps) and the state-gradient adds (2 C)."""
    c, h, taps, hid = wl.channels, wl.hidden, wl.taps(), wl.channels - wl.n_in
    bwd = 2 * h * hid + h + 2 * h * 2 * c + 2 * h * 2 * c + 2 * hid * h + h + c + \
        2 * c * taps + 2 * c * taps + 2 * c
    return 2 * algorithmic_flop_per_cell_step(wl) + bwd


def algorithmic_train_bytes_per_cell_step(wl) -> int:
    """fp32 state of C channels: the forward reads a state and writes the next
    (kept), the backward reads that state and dL/dS' and writes dL/dS."""
    return 5 * wl.channels * 4


def algorithmic_bytes_per_cell_step(wl) -> int:
    """Read C channels, write the C - n_in hidden channels."""
    eb = 2 if wl.dtype == "f16" else 4
    return (wl.channels + wl.channels - wl.n_in) * eb


def step_kernel_arithmetic(wl, kernel: str):
    """(kernel name, arithmetic of its MLP contraction, that arithmetic's
    MI355X peak in TFLOP/s) for a step-kernel name of ``Model(kernel=...)``."""
    names = set(kernel.split(","))
    if "valu" in names:
        return "nca_step_valu", "fp32 vector FMA", FP32_SCALAR_FMA_PEAK_TFLOPS
    if "mfma_f32" in names:
        return "nca_step_mfma / fp32 MFMA", "fp32 MFMA", FP32_MFMA_PEAK_TFLOPS
    if "mfma_f16" in names or (wl.dtype == "f16" and "mfma_bf16x3" not in names):
        return "nca_step_mfma / fp16 MFMA", "fp16 MFMA", FP16_MFMA_PEAK_TFLOPS
    if "mfma_bf16x3" in names:
        return "nca_step_mfma / split-bf16 MFMA", "bf16 MFMA (3 products per fp32 product)", \
            BF16_MFMA_PEAK_TFLOPS
    return "nca_step_mfma / scaled-fp16 MFMA", \
        "fp16 MFMA (fp16 activations x split fp16 weights, 2 products per fp32 product)", \
        FP16_MFMA_PEAK_TFLOPS


def arithmetic_label(wl, kernel: str) -> str:
    """What the step computes in, beside the storage type ``dtype``."""
    names = set(kernel.split(","))
    store = "fp16 state" if wl.dtype == "f16" else "fp32 state"
    if "valu" in names:
        return f"{store}; perception and MLP fp32 FMA on the vector ALUs"
    if "mfma_f32" in names:
        return f"{store}; perception fp32 FMA; MLP fp32 MFMA, fp32 accumulate"
    if "mfma_bf16x3" in names:
        return f"{store}; perception fp32 FMA; MLP split-bf16 MFMA (3 products), fp32 accumulate"
    if wl.dtype == "f16":
        pk = "packed fp16 FMA" if wl.ndim == 3 else "fp32 FMA"
        return f"{store}; perception {pk}; MLP fp16 MFMA, fp32 accumulate"
    return (f"{store}; perception fp32 FMA; MLP fp16 MFMA on activations scaled by 2^-8 and "
            "rounded to fp16 x weights split into fp16 hi + lo, fp32 accumulate")


STEP_SOURCES = ("paper_2508_06993_amd/csrc/step_mfma.hip", "paper_2508_06993_amd/csrc/device_common.h")
HOST_MARKER = "// ==== host side"


def step_source_sha256() -> str:
    """Hash of the step kernels' device code: device_common.h and the part of
    step_mfma.hip before its host-side launch code."""
    import hashlib
    h = hashlib.sha256()
    for rel in STEP_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            text = f.read()
        cut = text.find(HOST_MARKER.encode())
        h.update(text if cut < 0 else text[:cut])
    return h.hexdigest()


def measured_traffic(wl, selector: str):
    """HBM bytes per step launch from the profiler's FETCH_SIZE / WRITE_SIZE
    counters (each scaled by what it reads for a plain copy of known size),
    recorded in profiles/ together with the hash of the step kernel's sources;
    None when no record matches this workload, selector and source."""
    path = os.path.join(ROOT, "profiles", f"step_kernel_traffic_{wl.name}.md")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if ":" in line and line.strip().startswith("- `"):
            k, v = line.strip()[3:].split("`:", 1)
            rec[k.strip()] = v.strip().strip("`")
    if rec.get("source_sha256") != step_source_sha256() or rec.get("kernel_selector") != selector:
        return None
    return float(rec["traffic_bytes_per_launch"])


def blas_info():
    """(numpy version, BLAS library and version, BLAS threads) of this process."""
    import numpy as np
    libs, threads = [], 1
    try:
        from threadpoolctl import threadpool_info
        for p in threadpool_info():
            if p.get("user_api") == "blas":
                libs.append(f"{p.get('internal_api')} {p.get('version')}")
                threads = max(threads, int(p.get("num_threads", 1)))
    except Exception:   # pragma: no cover
        pass
    return np.__version__, ", ".join(libs) or "unknown", threads


def cpu_baseline(wl, seconds_hint=10.0, max_steps=200):
    """Time the CPU oracle on a crop of the finest level (random state, the
    workload's level-0 weights): consecutive NCA steps in one process (no
    band-parallel driver) until about `seconds_hint` seconds of CPU work (at
    least 4 steps, at most max_steps)."""
    import numpy as np
    import oracle
    from synthetic import make_weights, storage_dtype
    npver, blas, threads = blas_info()
    rng = np.random.default_rng(0)
    if wl.ndim == 2:
        shape = (1, 512, 1024)
    else:
        shape = (16, 128, 256)
    dt = storage_dtype(wl)
    state = rng.normal(0, 1, shape + (wl.channels,)).astype(dt)
    w = make_weights(wl)[0]
    steps = 0
    t0 = time.perf_counter()
    while steps < max_steps and (steps < 4 or time.perf_counter() - t0 < seconds_hint):
        state = oracle.nca_step(state, w, wl.n_in, wl.ndim, 0, steps, wl.seed, wl.fire_rate, dt)
        steps += 1
    dt_s = time.perf_counter() - t0
    cells = shape[0] * shape[1] * shape[2]
    return {"value": cells * steps / dt_s, "unit": "cell-steps/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{steps} NCA steps of the finest level on a {shape[0]}x{shape[1]}x"
                      f"{shape[2]} crop ({cells * steps} cell-steps, {dt_s:.1f} s), "
                      f"numpy float64 arithmetic, BLAS threads={threads}, "
                      f"affinity={len(os.sched_getaffinity(0))} cpus",
            "numpy": npver, "blas": blas, "blas_threads": int(threads),
            "affinity_cpus": len(os.sched_getaffinity(0)), "band_parallel": False}


def cpu_train_baseline(wl, seconds_hint=10.0):
    """Time the CPU oracle's training step (forward keeping every state, the
    readout MSE, backward through all steps and levels) on the workload's
    structure at a reduced extent, repeated until about `seconds_hint` s."""
    import numpy as np
    import oracle
    from synthetic import make_image, make_target, make_weights, scaled
    npver, blas, threads = blas_info()
    small = scaled(wl, (1, 160, 160)) if wl.ndim == 2 else scaled(wl, wl.extent)
    image = make_image(small)
    target = make_target(small, image)
    ws = make_weights(small)
    kw = dict(ndim=small.ndim, n_in=small.n_in, factors=small.factors, seed=small.seed,
              fire_rate=small.fire_rate)
    runs = 0
    t0 = time.perf_counter()
    while runs < 1 or time.perf_counter() - t0 < seconds_hint:
        tape = oracle.train_forward(image, ws, channels=small.channels, steps=small.steps,
                                    dtype=np.float32, **kw)
        _, g = oracle.readout_mse(tape.final, target)
        oracle.train_backward(tape, ws, g_final=g, **kw)
        runs += 1
    dt_s = time.perf_counter() - t0
    cs = small.cell_steps()
    return {"value": cs * runs / dt_s, "unit": "cell-steps/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{runs} training step(s) (forward + backward) of the workload's structure "
                      f"at {small.extent[1]}x{small.extent[2]} ({cs} cell-steps each, "
                      f"{dt_s:.1f} s), numpy float64, BLAS threads={threads}, "
                      f"affinity={len(os.sched_getaffinity(0))} cpus",
            "numpy": npver, "blas": blas, "blas_threads": int(threads),
            "affinity_cpus": len(os.sched_getaffinity(0)), "band_parallel": False}


def train_bench(args):
    """--train: the fused training step (octree_nca_train_step) on a training
    workload; one step = forward keeping every state + loss + backward."""
    import numpy as np
    import torch
    import paper_2508_06993_amd as octnca
    from paper_2508_06993_amd.runtime import upload_weights
    from synthetic import TRAIN_WORKLOADS, make_image, make_target, make_weights

    wl = TRAIN_WORKLOADS[args.train_workload]
    torch.cuda.set_device(0)
    octnca.lib()
    print(f"# training workload {wl.name}: extent {wl.extent}, levels {wl.levels}, "
          f"steps {wl.steps}", file=sys.stderr, flush=True)
    model = octnca.Model(ndim=wl.ndim, n_in=wl.n_in)
    image_np = make_image(wl)
    image = torch.from_numpy(image_np).cuda()
    target = torch.from_numpy(make_target(wl, image_np)).cuda()
    wts = make_weights(wl)
    weights = upload_weights(wts)
    grads = [{k: torch.zeros(np.shape(getattr(w, k)), dtype=torch.float32, device="cuda")
              for k in ("conv_w", "conv_b", "w1", "b1", "w2")} for w in wts]
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    torch.cuda.reset_peak_memory_stats()
    work = torch.empty(octnca.octree_nca_train_workspace_bytes(model, wl.extent, wl.factors,
                                                               wl.steps),
                       dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()

    def one():
        octnca.octree_nca_train_step(model, image, wl.factors, weights, wl.steps, wl.fire_rate,
                                     wl.seed, target, work, grads, loss, stream=stream)

    for _ in range(args.warmup):
        one()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        one()
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = sum(a.elapsed_time(b) for a, b in ev)
    cs = wl.cell_steps()
    flop = algorithmic_train_flop_per_cell_step(wl) * cs * args.steps
    byts = algorithmic_train_bytes_per_cell_step(wl) * cs * args.steps
    tflops = flop / (gpu_ms * 1e-3) / 1e12
    gbs = byts / (gpu_ms * 1e-3) / 1e9
    # the backward, most of the FLOPs and of the time, runs on fp32 MFMA
    t_mfma = flop / (FP32_MFMA_PEAK_TFLOPS * 1e12)
    t_hbm = byts / (HBM_PEAK_GBS * 1e9)
    if t_mfma >= t_hbm:
        bound, achieved, peak, unit = "mfma", tflops, FP32_MFMA_PEAK_TFLOPS, "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", gbs, HBM_PEAK_GBS, "GB/s"
    out = {
        "metric": "NCA training cell-steps/sec",
        "value": cs * args.steps / wall,
        "unit": "cell-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "extent_dhw": list(wl.extent), "levels": wl.levels,
                   "steps_per_level": list(wl.steps), "cells_per_level": wl.cells_per_level(),
                   "cell_steps_per_step": cs, "channels": wl.channels, "hidden": wl.hidden,
                   "n_in": wl.n_in, "fire_rate": wl.fire_rate, "loss": "readout MSE",
                   "parallelism": "single GPU"},
        "roofline": {"kernel": "octree_nca_train_step (forward split-bf16 MFMA, backward fp32 MFMA)",
                     "bound": bound, "achieved": round(achieved, 3), "peak": round(peak, 1),
                     "unit": unit, "frac": round(achieved / peak, 4), "traffic": None,
                     "achieved_tflops": round(tflops, 3), "achieved_hbm_gbs": round(gbs, 1),
                     "gpu_ms_per_step": round(gpu_ms / args.steps, 3),
                     "flop_per_cell_step": algorithmic_train_flop_per_cell_step(wl),
                     "bytes_per_cell_step": algorithmic_train_bytes_per_cell_step(wl)},
        "peak_vram_gb": round(torch.cuda.max_memory_allocated() / 1e9, 3),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_train_baseline(wl)
    print(json.dumps(out), flush=True)
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="pathology184mp")
    ap.add_argument("--extra", default="video2dt,volume3d,medium2d",
                    help="comma-separated further workloads timed in the same run and reported "
                         "under 'workloads' in the same JSON line ('' for none)")
    ap.add_argument("--model", default="c16h64", choices=sorted(MODEL_SIZES),
                    help="model size C/H: the paper's 16/64 or the ablation's 12/48, 20/100")
    ap.add_argument("--kernel", default="mfma",
                    help="step kernel, a name accepted by Model(kernel=...), e.g. mfma, "
                         "mfma_1step, mfma_f32, valu")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--train", action="store_true",
                    help="time the fused training step instead of the inference")
    ap.add_argument("--train-workload", default="pathology_train320")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized device buffer 3 times (calibrates the HBM "
                         "byte counters of a profiler against a kernel of known traffic)")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for --gpus {args.gpus}); the octree "
              "inference of one image runs on a single MI355X. Use --gpus 1.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if args.train:
        return train_bench(args)
    if args.copy_probe:
        n = args.copy_probe * (1 << 20)
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 3}))
        return 0

    from synthetic import WORKLOADS
    import paper_2508_06993_amd as octnca
    octnca.lib()   # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    wl = with_model(WORKLOADS[args.workload], args.model)
    out = inference_record(wl, args.kernel, args.steps, args.warmup)
    extras = [w for w in (args.extra.split(",") if args.extra else []) if w and w != wl.name]
    if extras:
        out["workloads"] = {}
        for name in extras:
            out["workloads"][name] = inference_record(with_model(WORKLOADS[name], args.model),
                                                      args.kernel, args.steps, args.warmup,
                                                      sub=True)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)
    return 0


MODEL_SIZES = {"c16h64": (16, 64), "c12h48": (12, 48), "c20h100": (20, 100)}


def with_model(wl, model: str):
    """The workload with another of the ablation's model sizes (supplement
    S10): C state channels and H hidden units, the same image and octree."""
    import dataclasses
    c, h = MODEL_SIZES[model]
    if (c, h) == (wl.channels, wl.hidden):
        return wl
    return dataclasses.replace(wl, channels=c, hidden=h, name=f"{wl.name}_{model}")


def inference_record(wl, kernel: str, steps: int, warmup: int, sub: bool = False) -> dict:
    """Time `steps` whole inferences of workload `wl` (after `warmup` untimed
    ones) with the image resident in HBM; the bench record of that workload."""
    import gc
    import torch
    import paper_2508_06993_amd as octnca
    from paper_2508_06993_amd.runtime import Inference, upload_weights, to_device_image
    from synthetic import make_weights
    from synthetic.cache import cached_image

    print(f"# workload {wl.name}: extent {wl.extent}, levels {wl.levels}, steps {wl.steps}, "
          f"kernel {kernel}", file=sys.stderr, flush=True)
    model = octnca.Model(ndim=wl.ndim, n_in=wl.n_in, dtype=wl.dtype, channels=wl.channels,
                         hidden=wl.hidden, kernel=kernel)
    image_np = cached_image(wl)
    image = to_device_image(image_np, model)
    del image_np
    weights = upload_weights(make_weights(wl))
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    run = Inference(model, wl.extent, wl.factors)
    stream = torch.cuda.current_stream()
    L = wl.levels

    def one_pass(events=None):
        run(image, weights, wl.steps, wl.fire_rate, wl.seed,
            level_events=[e.cuda_event for e in events] if events else None, stream=stream)

    for _ in range(warmup):
        one_pass()
    torch.cuda.synchronize()
    print(f"# {wl.name}: warmup done", file=sys.stderr, flush=True)

    # events: created (first record) before the timed region
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * L)] for _ in range(steps)]
    for row in ev:
        for e in row:
            e.record(stream)
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for k in range(steps):
        one_pass(ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print(f"# {wl.name}: timed passes done", file=sys.stderr, flush=True)

    cells = wl.cells_per_level()
    cell_steps = wl.cell_steps()
    step_ms = 0.0
    for row in ev:
        for l in range(L):
            if wl.steps[l] > 0:
                step_ms += row[2 * l].elapsed_time(row[2 * l + 1])
    # step-kernel launches of a pass as the library enqueues them (a launch
    # runs one step, or two on large 2D fp32 levels)
    launches = steps * sum(octnca.octree_nca_infer_launches(model, wl.extent, wl.factors,
                                                            wl.steps))
    avg_launch_ms = step_ms / launches
    flop = algorithmic_flop_per_cell_step(wl) * cell_steps * steps
    byts = algorithmic_bytes_per_cell_step(wl) * cell_steps * steps
    achieved_tflops = flop / (step_ms * 1e-3) / 1e12
    achieved_gbs = byts / (step_ms * 1e-3) / 1e9
    kname, arith, arith_peak = step_kernel_arithmetic(wl, kernel)
    # binding roof: the larger of the two floors (bytes at HBM peak, FLOPs at
    # the peak of the arithmetic the kernel's contraction runs on)
    t_hbm = byts / (HBM_PEAK_GBS * 1e9)
    t_arith = flop / (arith_peak * 1e12)
    if t_arith >= t_hbm:
        bound = "alu" if arith == "fp32 vector FMA" else "mfma"
        achieved, peak, unit = achieved_tflops, arith_peak, "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", achieved_gbs, HBM_PEAK_GBS, "GB/s"
    roofline = {
        "kernel": kname,
        "bound": bound,
        "achieved": round(achieved, 3),
        "peak": round(peak, 1),
        "unit": unit,
        "frac": round(achieved / peak, 4),
        "traffic": measured_traffic(wl, kernel),
        "traffic_unit": "bytes per launch (HBM, profiler counters)",
        "arithmetic": arith,
        "achieved_tflops": round(achieved_tflops, 3),
        "arith_peak_tflops": round(arith_peak, 1),
        "arith_frac": round(achieved_tflops / arith_peak, 4),
        "achieved_hbm_gbs": round(achieved_gbs, 1),
        "hbm_frac": round(achieved_gbs / HBM_PEAK_GBS, 4),
        "avg_launch_ms": round(avg_launch_ms, 4),
        "launches": launches,
        "flop_per_cell_step": algorithmic_flop_per_cell_step(wl),
        "bytes_per_cell_step": algorithmic_bytes_per_cell_step(wl),
    }
    peak_vram = torch.cuda.max_memory_allocated() / 1e9
    out = {
        "metric": "NCA cell-steps/sec",
        "value": cell_steps * steps / wall,
        "unit": "cell-steps/s",
    }
    if not sub:
        out.update({"n_gpus": 1, "steps": steps, "warmup": warmup})
    out.update({
        "ms_per_step": wall / steps * 1e3,
    })
    if not sub:
        out.update({"higher_is_better": True, "scaling": "weak", "vs_baseline": None})
    out.update({
        "dtype": "f16" if wl.dtype == "f16" else "f32",
        "arithmetic": arithmetic_label(wl, kernel),
        "data": "synthetic",
        "config": {"workload": wl.name, "extent_dhw": list(wl.extent), "levels": wl.levels,
                   "steps_per_level": list(wl.steps), "cells_per_level": cells,
                   "cell_steps_per_pass": cell_steps, "channels": wl.channels,
                   "hidden": wl.hidden, "n_in": wl.n_in, "fire_rate": wl.fire_rate,
                   "kernel": kernel, "parallelism": "single GPU"},
        "roofline": roofline,
        "peak_vram_gb": round(peak_vram, 3),
        "step_kernel_ms_per_pass": round(step_ms / steps, 3),
    })
    del run, image, weights
    gc.collect()
    torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    sys.exit(main())
