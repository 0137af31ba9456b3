#!/usr/bin/env python3
"""Throughput of one draft step of FOVEA's retrieval + fusion on one MI355X.

A step is one fovea_retrieve_fuse call over the whole batch: query projection, scoring
of every valid key, cumulative-mass selection, renormalised gather, correction MLPs,
gated residual and RMSNorm.  Default workload: the batched serving shape (32 requests,
each with its own 576-entry memory, 60 draft-tree nodes per request, d = 4096,
d_m = 1024, k_max = 64, tau per request in [0.6, 0.95]), synthetic seeded inputs.

Protocol: inputs are resident in HBM; the timed loop rotates over several copies of
the inputs (more bytes than the 256 MB Infinity Cache) so each step reads its keys,
values and hidden states from HBM; W warm-up steps, then exactly K steps between two
HIP events after a device synchronisation.  A second, profiled pass brackets every
kernel with HIP events for the per-kernel roofline.  The fp64 oracle is timed on the
host cores on a bounded sample as the CPU baseline.

--backward times fovea_retrieve_fuse_backward (fp32 context, the selection of one
forward run held fixed, dL/dh_hat synthetic) on the workload's shapes instead.

--lm-head vicuna7b|qwen2_5_7b extends every step by the drafter's LM head over the
corrected states and the top-K_c (--kc, default 6) candidate extraction
(fovea_lm_topk), with a synthetic head of that vocabulary; the CPU baseline is then
skipped.

Prints one JSON line.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0    # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3     # dense fp32
PROFILES = os.path.join(ROOT, "profiles")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="batched_b32")
    ap.add_argument("--copies", type=int, default=6, help="input copies rotated in the timed loop")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--lm-head", default=None, choices=["vicuna7b", "qwen2_5_7b"],
                    help="extend the step by the drafter's LM head and top-K_c candidates")
    ap.add_argument("--kc", type=int, default=6, help="candidates per node with --lm-head")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward of the step (fp32) instead of the forward")
    ap.add_argument("--build-memory", action="store_true",
                    help="time the one-off memory build (every request's visual tokens -> keys "
                         "and values) of the workload instead of the draft step")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of known size (counter calibration)")
    return ap.parse_args()


def source_hash() -> str:
    """Hash of the library sources; counter readings are valid for this hash only."""
    import hashlib

    h = hashlib.sha256()
    for sub in ("include", os.path.join("paper_2608_22883_amd", "csrc")):
        base = os.path.join(ROOT, sub)
        for name in sorted(os.listdir(base)):
            with open(os.path.join(base, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, run: str):
    """HBM bytes per launch of `kernel` in run `run` (a workload name, with a suffix for
    the other modes) from the committed counter summary profiles/traffic_<run>.txt
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy's readings), or None when the
    summary is missing or was taken on other sources."""
    try:
        with open(os.path.join(PROFILES, f"traffic_{run}.txt")) as f:
            rows = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    rows = {k.strip(): v.strip() for k, v in rows.items()}
    if rows.get("source_hash") != source_hash():
        return None
    v = rows.get(f"traffic_bytes {kernel}")
    return int(float(v)) if v else None


def copy_calibration():
    """A plain device-to-device copy of 256 MiB, ten times: the reference dispatch for
    scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch

    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(10):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps(dict(copy_bytes_read=n, copy_bytes_written=n, dispatches=10)), flush=True)


def kernel_model(wl, case, union_rows, k_sum, lm=None, kc=0):
    """Algorithmic bytes and flops per launch of each kernel (storage dtype es)."""
    import numpy as np

    es = 2 if wl.dtype == "bf16" else 4
    n, d, d_m, d_c = case.n_nodes, wl.d, wl.d_m, wl.d_c
    Ms = np.diff(case.mem_off).astype(np.int64)
    Ts = np.diff(case.node_off).astype(np.int64)
    pairs = int((Ms * Ts).sum())
    n_mem = int(Ms.sum())
    k = {}
    k["row_stats"] = dict(bytes=n * d * es + n * 8, flops=3 * n * d)
    k["hq"] = dict(bytes=n * d * es + (d_m + 2 * d_c) * d * es + n * d_m * 4 + n * 2 * d_c * 4,
                   flops=2 * n * d * (d_m + 2 * d_c))
    k["score"] = dict(bytes=n_mem * d_m * es + n * d_m * 4 + pairs * 4, flops=2 * pairs * d_m)
    k["select_gather"] = dict(bytes=pairs * 4 + union_rows * d_m * es + n * d_m * es,
                              flops=2 * int(k_sum) * d_m)
    k["corr1"] = dict(bytes=n * d_m * es + 2 * d_c * d_m * es + n * 2 * d_c * 4 + n * d_c * es,
                      flops=2 * n * d_m * 2 * d_c)
    k["corr2"] = dict(bytes=n * d_c * es + d * d_c * es + 2 * n * d * es, flops=2 * n * d_c * d)
    k["rms"] = dict(bytes=2 * n * d * es, flops=3 * n * d)
    if lm is not None:
        cand = n * ((lm["vocab"] + 127) // 128) * kc * 8
        k["lm_head"] = dict(bytes=lm["vocab"] * d * es + n * d * es + cand,
                            flops=2 * n * d * lm["vocab"])
        k["lm_merge"] = dict(bytes=cand + n * kc * 8, flops=0)
    # the retrieval as one operation: every key, q, the selected value rows, r
    retrieval = dict(bytes=n_mem * d_m * es + n * d_m * 4 + union_rows * d_m * es + n * d_m * es,
                     flops=2 * pairs * d_m + 2 * int(k_sum) * d_m)
    return k, retrieval


def cpu_baseline(case, budget_s):
    """The fp64 oracle, as it stands, on the host cores: whole steps of the same workload
    repeated until the time budget is used (at least one)."""
    import numpy as np  # noqa: F401

    import oracle
    from threadpoolctl import threadpool_info

    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    t0 = time.perf_counter()
    reps = 0
    while True:
        oracle.retrieve_fuse(case.weights, case.mem_off, case.keys, case.values, case.valid,
                             case.node_off, case.h, case.depth, case.tau, case.k_min, case.k_max,
                             gain_rounding="bf16" if case.workload.dtype == "bf16" else None)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or el / reps * (reps + 1) > 2.5 * budget_s:
            break
    return dict(value=case.n_nodes * reps / el, unit="states/s", cores=int(threads), kind="oracle",
                sample=f"{reps} full step(s) of the same workload ({case.n_nodes} draft states each), "
                       f"{el:.1f} s wall, fp64 NumPy, BLAS threads={threads}, "
                       f"affinity cpus={len(os.sched_getaffinity(0))}")


def backward_main(args):
    """One step = one fovea_retrieve_fuse_backward call over the whole batch (fp32)."""
    import numpy as np
    import torch

    import paper_2608_22883_amd as F
    from synth import WORKLOADS, make_case, make_output_grad

    wl = WORKLOADS[args.workload].with_(dtype="f32")
    log(f"[bench] generating {wl.name} (fp32) ...")
    case = make_case(wl)
    W = case.weights
    dev = torch.device("cuda:0")
    dims = dict(d=wl.d, d_v=wl.d, d_m=wl.d_m, d_c=wl.d_c, n_depth=wl.n_depth, dtype=0,
                ln_eps=W["ln_eps"], rms_eps=W["rms_eps"])
    fv = F.Fovea(dims, W, device=dev)

    def dev_t(x, d=torch.float32):
        return torch.tensor(np.asarray(x), dtype=d, device=dev)

    inp = dict(mem_off=torch.tensor(case.mem_off, dtype=torch.int64, device=dev),
               keys=dev_t(case.keys), values=dev_t(case.values), valid=None,
               node_off=torch.tensor(case.node_off, dtype=torch.int32, device=dev),
               h=dev_t(case.h), depth=torch.tensor(case.depth, dtype=torch.int32, device=dev),
               tau=dev_t(case.tau), m_max=case.m_max, t_max=case.t_max, k_min=case.k_min,
               k_max=case.k_max)
    out = fv.retrieve_fuse(inp, debug=True)
    torch.cuda.synchronize()
    K, idx = out.k, out.idx
    n, d, d_m, d_c = case.n_nodes, wl.d, wl.d_m, wl.d_c
    dh_hat = dev_t(make_output_grad(n, d, wl.seed + 17))
    grads = fv.retrieve_fuse_backward(inp, K, idx, dh_hat)  # allocates the outputs once
    dh, dkeys, dvalues = grads.pop("dh"), grads.pop("dkeys"), grads.pop("dvalues")
    g = {k[1:]: v for k, v in grads.items()}
    B = wl.B
    ws = torch.empty(F.fovea_retrieve_fuse_backward_workspace(fv.ctx, B, n, case.m_max, case.k_max),
                     dtype=torch.uint8, device=dev)

    def step():
        F.fovea_retrieve_fuse_backward(
            fv.ctx, fv.params, fv.b_g2, B, inp["mem_off"], inp["keys"].shape[0], case.m_max,
            inp["keys"], inp["values"], inp["node_off"], n, case.t_max, inp["h"], inp["depth"],
            K, idx, case.k_max, dh_hat, dh, dkeys, dvalues, g, ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"[bench] backward, {args.steps} steps: {ms * 1e3:.1f} us/step")
    F.fovea_profile(fv.ctx, True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = F.fovea_profile_read(fv.ctx, 32)
    F.fovea_profile(fv.ctx, False)
    npad = (n + 63) // 64 * 64
    gemm_flops = 2 * n * (d * d_m + (d + d_m) * 2 * d_c + d_c * d + d * d_c + 2 * d_c * (d + d_m)
                          + d_m * d) + 2 * npad * (d * d_c + 2 * d_c * (d + d_m) + d_m * d)
    kernels = []
    for name, (tot, cnt) in prof.items():
        per_step_us = tot / args.steps * 1e3
        e = dict(name=name, us_per_step=round(per_step_us, 2), timed_regions_per_step=cnt // args.steps)
        if name == "bwd_gemm":
            # fp32-accurate products as bf16 GEMMs over a tripled K (hi/lo planes): the
            # matrix cores issue three times the products' flops
            e["TFLOPs"] = round(gemm_flops / (per_step_us * 1e-6) / 1e12, 2)
            e["MFMA_TFLOPs"] = round(3 * gemm_flops / (per_step_us * 1e-6) / 1e12, 2)
        kernels.append(e)
        log(f"[bench] {name:14s} {per_step_us:9.2f} us/step  ({cnt // args.steps} timed regions)")
    kernels.sort(key=lambda k: -k["us_per_step"])
    gk = next(k for k in kernels if k["name"] == "bwd_gemm")
    line = dict(
        metric="draft states/sec for the backward of retrieve+fuse (fp32, selection held fixed)",
        value=round(n / (ms * 1e-3), 1), unit="states/s", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(ms, 5), higher_is_better=True, scaling="weak",
        vs_baseline=None, dtype="f32", data="synthetic",
        config=dict(workload=wl.name, mode="backward", B=wl.B, T=wl.T, M=wl.M, d=d, d_m=d_m,
                    d_c=d_c, k_max=wl.k_max, states_per_step=n),
        roofline=dict(bound="mfma", achieved=gk["MFMA_TFLOPs"], peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                      frac=round(gk["MFMA_TFLOPs"] / PEAK_BF16_TFLOPS, 4), traffic=None,
                      kernel="bwd_gemm (all GEMM launches of a step; bf16 matrix cores, K tripled "
                             "by the hi/lo planes of the fp32 operands)"),
        kernels=kernels)
    fv.close()
    print(json.dumps(line), flush=True)


def build_main(args):
    """One step = one fovea_build_memory call over every request's visual tokens (the
    workload's B memories of M rows: LayerNorm over d_v, then W_K and W_U)."""
    import numpy as np
    import torch

    import oracle
    import paper_2608_22883_amd as F
    from synth import WORKLOADS, make_memory_case

    wl = WORKLOADS[args.workload]
    n_rows = wl.B * wl.M
    log(f"[bench] generating {n_rows} visual tokens of width {wl.d} ...")
    V, W = make_memory_case(wl, n_rows)
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    dims = dict(d=wl.d, d_v=wl.d, d_m=wl.d_m, d_c=wl.d_c, n_depth=wl.n_depth,
                dtype=1 if wl.dtype == "bf16" else 0, ln_eps=W["ln_eps"], rms_eps=W["rms_eps"])
    fv = F.Fovea(dims, W, device=dev)
    Vd = torch.tensor(V, dtype=dt, device=dev)
    # copies at distinct addresses so that consecutive calls cannot hit in the 256 MB MALL
    sets = [Vd] + [Vd.clone() for _ in range(args.copies - 1)]
    keys = torch.empty(n_rows, wl.d_m, dtype=dt, device=dev)
    values = torch.empty_like(keys)
    ws = torch.empty(max(F.fovea_build_memory_workspace(fv.ctx, n_rows), 256), dtype=torch.uint8,
                     device=dev)

    def step(i):
        F.fovea_build_memory(fv.ctx, sets[i % len(sets)], keys, values, ws)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"[bench] build_memory, {args.steps} calls: {ms * 1e3:.1f} us/call")
    F.fovea_profile(fv.ctx, True)
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    prof = F.fovea_profile_read(fv.ctx)
    F.fovea_profile(fv.ctx, False)
    es = 2 if wl.dtype == "bf16" else 4
    d_v, d_m = wl.d, wl.d_m
    model = dict(mem_row_stats=dict(bytes=n_rows * d_v * es + n_rows * 8, flops=3 * n_rows * d_v),
                 mem_proj=dict(bytes=n_rows * d_v * es + 2 * d_m * d_v * es + 2 * n_rows * d_m * es,
                               flops=2 * n_rows * d_v * 2 * d_m))
    peak_fl = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    kernels = []
    for name, (tot, cnt) in prof.items():
        avg_ms = tot / cnt
        m = model.get(name, dict(bytes=0, flops=0))
        gbs = m["bytes"] / (avg_ms * 1e-3) / 1e9
        tfl = m["flops"] / (avg_ms * 1e-3) / 1e12
        mfma = name == "mem_proj"
        kernels.append(dict(name=name, avg_us=round(avg_ms * 1e3, 2), launches=cnt,
                            alg_bytes=m["bytes"], alg_flops=m["flops"], GBs=round(gbs, 1),
                            TFLOPs=round(tfl, 2), bound="mfma" if mfma else "hbm",
                            frac=round(tfl / peak_fl if mfma else gbs / PEAK_HBM_GBS, 4)))
        log(f"[bench] {name:14s} {avg_ms * 1e3:8.2f} us  {gbs:8.1f} GB/s  {tfl:7.2f} TFLOP/s")
    kernels.sort(key=lambda k: -k["avg_us"])
    pk = next(k for k in kernels if k["name"] == "mem_proj")
    line = dict(
        metric="visual-memory rows/sec for build_memory (LayerNorm, W_K and W_U)",
        value=round(n_rows / (ms * 1e-3), 1), unit="rows/s", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(ms, 5), higher_is_better=True, scaling="weak",
        vs_baseline=None, dtype=wl.dtype, data="synthetic",
        config=dict(workload=wl.name, mode="build_memory", rows=n_rows, images=wl.B,
                    rows_per_image=wl.M, d_v=d_v, d_m=d_m, input_copies=len(sets)),
        roofline=dict(bound="mfma", achieved=pk["TFLOPs"], peak=peak_fl, unit="TFLOP/s",
                      frac=pk["frac"], traffic=measured_traffic("mem_proj", wl.name + "_build"),
                      kernel="mem_proj"),
        kernels=kernels)
    if not args.no_cpu_baseline:
        # the oracle on whole images (M rows each) within the time budget
        from threadpoolctl import threadpool_info

        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        t0 = time.perf_counter()
        reps = 0
        while True:
            r0 = (reps % wl.B) * wl.M
            oracle.build_memory(V[r0:r0 + wl.M], W["mem_ln_g"], W["mem_ln_b"], W["W_K"], W["W_U"],
                                W["ln_eps"], gain_rounding="bf16" if wl.dtype == "bf16" else None)
            reps += 1
            el = time.perf_counter() - t0
            if el >= args.cpu_seconds or el / reps * (reps + 1) > 2.5 * args.cpu_seconds:
                break
        line["cpu_baseline"] = dict(
            value=reps * wl.M / el, unit="rows/s", cores=int(threads), kind="oracle",
            sample=f"{reps} image(s) of {wl.M} rows, {el:.1f} s wall, fp64 NumPy, BLAS threads={threads}")
    fv.close()
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the retrieval of each request is independent, "
              "so more GPUs would each run this same single-GPU step on their share of the "
              "requests; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.backward:
        backward_main(args)
        return
    if args.build_memory:
        build_main(args)
        return

    import numpy as np
    import torch

    from paper_2608_22883_amd import Fovea, fovea_profile, fovea_profile_read
    from synth import WORKLOADS, make_case
    sys.path.insert(0, os.path.join(ROOT, "tests"))

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = WORKLOADS[args.workload]
    log(f"[bench] generating {wl.name} ...")
    case = make_case(wl)
    W = case.weights
    dev = torch.device("cuda:0")
    dims = dict(d=wl.d, d_v=wl.d, d_m=wl.d_m, d_c=wl.d_c, n_depth=wl.n_depth,
                dtype=1 if wl.dtype == "bf16" else 0, ln_eps=W["ln_eps"], rms_eps=W["rms_eps"])
    fv = Fovea(dims, W, device=dev)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    def dev_t(x, d=dt):
        return torch.tensor(np.asarray(x), dtype=d, device=dev)

    base = dict(mem_off=torch.tensor(case.mem_off, dtype=torch.int64, device=dev),
                keys=dev_t(case.keys), values=dev_t(case.values), valid=None,
                node_off=torch.tensor(case.node_off, dtype=torch.int32, device=dev),
                h=dev_t(case.h), depth=torch.tensor(case.depth, dtype=torch.int32, device=dev),
                tau=dev_t(case.tau, torch.float32), m_max=case.m_max, t_max=case.t_max,
                k_min=case.k_min, k_max=case.k_max)
    # copies at distinct addresses so that consecutive steps cannot hit in the 256 MB MALL
    sets = [base] + [dict(base, keys=base["keys"].clone(), values=base["values"].clone(),
                          h=base["h"].clone()) for _ in range(args.copies - 1)]
    per_set = sum(base[k].numel() * base[k].element_size() for k in ("keys", "values", "h"))
    out = fv.alloc_outputs(case.n_nodes, case.k_max, wl.d, wl.d_m)
    lm = None
    if args.lm_head:
        from synth import LM_HEADS, make_lm_case

        lm = dict(LM_HEADS[args.lm_head], name=args.lm_head)
        if lm["d"] != wl.d:
            log(f"[bench] {args.lm_head} has d={lm['d']}, the workload d={wl.d}")
            sys.exit(2)
        _, W_lm = make_lm_case(1, wl.d, lm["vocab"], wl.dtype, seed=wl.seed + 31)
        W_lm = dev_t(W_lm)
        lm_idx = torch.empty(case.n_nodes, args.kc, dtype=torch.int32, device=dev)

    def step(i, debug=False):
        fv.retrieve_fuse(sets[i % len(sets)], out, debug=debug)
        if lm is not None:
            fv.lm_topk(out.h_out, W_lm, args.kc, idx=lm_idx, want_logits=False)

    # one debug run: selected sets (for the algorithmic gather bytes) and a sanity check
    fv.retrieve_fuse(base, out, debug=True)
    torch.cuda.synchronize()
    K = out.k.cpu().numpy()
    idx = out.idx.cpu().numpy()
    union_rows = 0
    for b in range(wl.B):
        t0, t1 = case.node_off[b], case.node_off[b + 1]
        sel = idx[t0:t1]
        union_rows += len(np.unique(sel[sel >= 0]))
    log(f"[bench] K min/median/max {K.min()}/{np.median(K)}/{K.max()}, union rows {union_rows}")

    # whole-step timing
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        step(i)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"[bench] {args.steps} steps: {ms * 1e3:.1f} us/step")

    # distribution of single-step times (events around every step, a separate pass so
    # that the timed region above holds nothing but the steps)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for i in range(args.steps):
        evs[i][0].record()
        step(i)
        evs[i][1].record()
    torch.cuda.synchronize()
    per = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])
    pct = dict(p10=round(float(np.percentile(per, 10)), 2), median=round(float(np.median(per)), 2),
               p90=round(float(np.percentile(per, 90)), 2), mean=round(float(per.mean()), 2))
    log(f"[bench] single steps: p10 {pct['p10']} us, median {pct['median']} us, p90 {pct['p90']} us")

    # per-kernel timing (events around each kernel, on the library's stream)
    fovea_profile(fv.ctx, True)
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    prof = fovea_profile_read(fv.ctx)
    fovea_profile(fv.ctx, False)

    kmodel, retrieval = kernel_model(wl, case, union_rows, int(K.sum()), lm, args.kc)
    peak_fl = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    kernels = []
    for name, (tot, cnt) in prof.items():
        avg_ms = tot / cnt
        m = kmodel.get(name, dict(bytes=0, flops=0))
        gbs = m["bytes"] / (avg_ms * 1e-3) / 1e9
        tfl = m["flops"] / (avg_ms * 1e-3) / 1e12
        mfma = name in ("hq", "corr1", "corr2") or (
            name == "lm_head" and m["flops"] / m["bytes"] > peak_fl / PEAK_HBM_GBS * 1e3)
        kernels.append(dict(
            name=name, avg_us=round(avg_ms * 1e3, 2), launches=cnt, alg_bytes=m["bytes"],
            alg_flops=m["flops"], GBs=round(gbs, 1), TFLOPs=round(tfl, 2),
            bound="mfma" if mfma else "hbm",
            frac=round((tfl / peak_fl) if mfma else (gbs / PEAK_HBM_GBS), 4)))
        log(f"[bench] {name:14s} {avg_ms * 1e3:8.2f} us  {gbs:8.1f} GB/s  {tfl:7.2f} TFLOP/s")
    kernels.sort(key=lambda k: -k["avg_us"])
    dom = kernels[0]
    run = wl.name if lm is None else f"{wl.name}_{lm['name']}"
    if dom["bound"] == "mfma":
        roof = dict(bound="mfma", achieved=dom["TFLOPs"],
                    peak=PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS,
                    unit="TFLOP/s", frac=dom["frac"], traffic=measured_traffic(dom["name"], run),
                    kernel=dom["name"])
    else:
        roof = dict(bound="hbm", achieved=dom["GBs"], peak=PEAK_HBM_GBS, unit="GB/s",
                    frac=dom["frac"], traffic=measured_traffic(dom["name"], run), kernel=dom["name"])
    ret_names = [k["name"] for k in kernels if k["name"] in ("score", "select_gather")]
    ret_us = sum(k["avg_us"] for k in kernels if k["name"] in ret_names)
    ret_gbs = retrieval["bytes"] / (ret_us * 1e-6) / 1e9 if ret_us else 0.0

    metric = "draft states/sec for retrieve+fuse (M=576, d=4096); % of peak HBM GB/s"
    if lm is not None:
        metric = (f"draft states/sec for retrieve+fuse + LM head ({lm['name']}, vocab "
                  f"{lm['vocab']}) top-{args.kc} candidates")
    line = dict(
        metric=metric,
        value=round(case.n_nodes / (ms * 1e-3), 1), unit="states/s", n_gpus=1,
        steps=args.steps, warmup=args.warmup, ms_per_step=round(ms, 5), higher_is_better=True,
        scaling="weak", vs_baseline=None, dtype=wl.dtype, data="synthetic",
        config=dict(workload=wl.name, description=wl.description, B=wl.B, T=wl.T, M=wl.M,
                    d=wl.d, d_m=wl.d_m, d_c=wl.d_c, k_max=wl.k_max,
                    states_per_step=case.n_nodes, input_copies=len(sets),
                    rotated_bytes=per_set * len(sets),
                    **({} if lm is None else dict(lm_head=lm["name"], vocab=lm["vocab"],
                                                  kc=args.kc))),
        roofline=roof,
        step_us=pct,
        retrieval=dict(kernels=ret_names, us=round(ret_us, 2),
                       alg_bytes=retrieval["bytes"], GBs=round(ret_gbs, 1),
                       frac=round(ret_gbs / PEAK_HBM_GBS, 4)),
        kernels=kernels,
        K=dict(min=int(K.min()), median=float(np.median(K)), max=int(K.max()),
               union_value_rows=int(union_rows)),
    )
    if not args.no_cpu_baseline and lm is None:
        log("[bench] timing the oracle on the host ...")
        line["cpu_baseline"] = cpu_baseline(case, args.cpu_seconds)
    fv.close()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
