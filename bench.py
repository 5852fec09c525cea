"""Benchmark of the RingAda stage hot path on one MI355X.

One step = the whole per-stage path on one batch of synthetic input resident
in HBM: forward through the 12-block BERT-base-shaped stage, the initiator's
[CLS]-head loss and head update, the backward stopped at block 8, and the
update of the unfrozen adapters.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "stage fine-tune samples/sec (fwd+early-stop bwd); % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, published
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, published
GEMM_PREFIX = "gemm_"
CSRC = os.path.join(ROOT, "paper_2502_19864_amd", "csrc")
# source files that define each family of named kernels
KERNEL_SOURCES = {"gemm_": ("k_gemm.hip", "attn_core.h", "common.h", "kernels.h"),
                  "attn_": ("k_attention.hip", "attn_core.h", "common.h", "kernels.h"),
                  "adapter_": ("k_adapter.hip", "k_misc.hip", "common.h", "kernels.h")}


def kernel_source_hash(name):
    """sha256 over the sources that define the kernel family of `name`."""
    files = next((f for pre, f in KERNEL_SOURCES.items() if name.startswith(pre)), None)
    if files is None:
        return None
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_trace_us(name, workload):
    """Average duration (us) of kernel `name` in the committed rocprofv3 kernel
    trace of `workload`, if one exists and was taken on the current sources of
    that kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"kernel_trace_{workload}.md")
    if not os.path.exists(path):
        return None
    want = kernel_source_hash(name)
    for line in open(path):
        m = re.match(r"\s*trace:\s+kernel=(\S+)\s+avg_us=([0-9.]+)\s+source_sha256=([0-9a-f]+)", line)
        if m and m.group(1) == name and m.group(3) == want:
            return float(m.group(2))
    return None


def recorded_traffic(name, workload):
    """HBM bytes per launch of kernel `name` on `workload`, from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary, if one exists and was taken on
    the current sources of that kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    want = kernel_source_hash(name)
    for line in open(path):
        m = re.match(r"\s*traffic:\s+kernel=(\S+)\s+bytes_per_launch=(\d+)\s+source_sha256=([0-9a-f]+)", line)
        if m and m.group(1) == name and m.group(3) == want:
            return int(m.group(2))
    return None


def copy_calibration(torch, mib, reps=5):
    """A plain elementwise copy (dst = -src, float32) of `mib` MiB read and
    `mib` MiB written per launch: the known-size kernel that scales the
    FETCH_SIZE / WRITE_SIZE counters to bytes."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    log(f"[bench] copy calibration: {reps} launches of neg() over {mib} MiB float32 in, {mib} MiB out")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _f64(v):
    """float64 copies of every array in a nest of lists, tuples and dicts."""
    if isinstance(v, dict):
        return {k: _f64(x) for k, x in v.items()}
    if isinstance(v, (list, tuple)):
        return type(v)(_f64(x) for x in v)
    if isinstance(v, np.ndarray) and v.dtype.kind == "f":
        return v.astype(np.float64)
    return v


def cpu_baseline(w, inp, min_seconds=10.0, max_steps=8):
    """The oracle as the tests run it (numpy, float64) timed on this host: full
    steps (forward, head loss, early-stopped backward, SGD) on every sample of
    the workload, repeated until about min_seconds of CPU work have run."""
    import oracle as O
    from threadpoolctl import threadpool_info
    from paper_2502_19864_amd.workloads import adapters_as_computed
    desc = O.make_desc(w.arch, w.n_blocks, w.d_model, w.n_heads, w.d_ffn, w.d_adapter, placement=w.placement)
    W = _f64(inp["weights"])
    A = _f64(adapters_as_computed(w, inp["adapters"]))
    x = _f64(inp["x"])
    t0 = time.perf_counter()
    steps = 0
    while steps < max_steps and (steps == 0 or time.perf_counter() - t0 < min_seconds):
        y, caches = O.stage_forward(desc, W, A, x)
        if w.loss == "cls_ce":
            _, dy, _, _ = O.cls_head_ce(y, _f64(inp["w_h"]), _f64(inp["b_h"]), inp["labels"])
        elif w.loss == "mse":
            _, dy = O.mse_loss(y, _f64(inp["target"]))
        else:
            dy = _f64(inp["dy"])
        _, grads = O.stage_backward(desc, W, A, caches, dy, w.lowest_unfrozen)
        O.sgd_step(A, grads, 1e-3)
        steps += 1
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {"value": round(steps * w.batch / dt, 3), "unit": "samples/s", "cores": len(os.sched_getaffinity(0)),
            "blas_threads": int(threads), "kind": "oracle", "impl": "numpy float64 oracle (tests' reference)",
            "sample": f"{steps} full step(s) (forward, head loss, backward to block {w.lowest_unfrozen}, SGD) of "
                      f"the {w.name} workload, all {w.batch} samples each, numpy float64 oracle, {dt:.2f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="bert_base")
    ap.add_argument("--lowest-unfrozen", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch every kernel from the host each step instead of replaying a HIP graph")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="after the bench, run a plain copy kernel of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs one ring stage on one GPU; --gpus {args.gpus} is not supported "
              f"(the multi-GPU ring is not part of it)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2502_19864_amd import binding as B
    from paper_2502_19864_amd.stage import Stage
    from paper_2502_19864_amd.workloads import WORKLOADS, make_inputs

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    B.lib()
    w = WORKLOADS[args.workload]
    if args.lowest_unfrozen is not None:
        w = w.replace(lowest_unfrozen=args.lowest_unfrozen)
    c = w.lowest_unfrozen
    log(f"[bench] workload {w.name}: generating inputs")
    inp = make_inputs(w)
    st = Stage(w, inp)
    dev = st.dev
    x = st.upload(inp["x"])
    y = st.empty(*inp["x"].shape)
    dy = st.empty(*inp["x"].shape)
    dx = st.empty(*inp["x"].shape) if c < 0 else None
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    if w.loss == "cls_ce":
        # the head's weight and bias in one buffer (and their gradients in
        # another), so that one SGD launch updates both
        nwh = inp["w_h"].size
        hp = st.f32(np.concatenate([inp["w_h"].ravel(), inp["b_h"].ravel()]))
        hg = torch.zeros_like(hp)
        wh, bh = hp[:nwh].view(inp["w_h"].shape), hp[nwh:]
        gwh, gbh = hg[:nwh].view(inp["w_h"].shape), hg[nwh:]
        labels = torch.from_numpy(inp["labels"]).to(dev)
    elif w.loss == "mse":
        target = st.upload(inp["target"])
    else:
        dy = st.upload(inp["dy"])
    stash_bytes, scratch_bytes = st.ensure_workspace(w.batch, w.seq, c)
    lr = 1e-4

    def step():
        s = st.sptr
        st.forward(x, y, c)
        if w.loss == "cls_ce":
            B.ringada_head_ce(s, st.desc.dtype, y, w.batch, w.seq, w.d_model, wh, bh, 2, labels, dy, gwh, gbh, loss)
            B.ringada_sgd_f32(s, hp, hg, hp.numel(), lr)
        elif w.loss == "mse":
            B.ringada_loss_mse(s, st.desc.dtype, y, target, y.numel(), dy, loss)
        if c < w.n_blocks:
            st.backward(dy, c, dx)
            st.step(c, lr)

    log(f"[bench] warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if not args.no_graph:
        # one step captured into a HIP graph (every launch of the step is
        # stream-ordered on the capturing stream), replayed each step
        graph = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            step()  # one eager step on the capture stream first
        torch.cuda.current_stream().wait_stream(cap)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            step()
        torch.cuda.synchronize()
        run = graph.replay
        for _ in range(2):
            run()
        torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps ({'HIP graph replay' if run is not step else 'eager launches'})")
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms = 1e3 * elapsed / args.steps
    value = w.batch * args.steps / elapsed

    # per-kernel durations: HIP events around every launch, same steps again
    log("[bench] per-kernel event timing")
    B.ringada_prof_begin(st.handle)
    for _ in range(args.steps):
        step()
    prof = B.ringada_prof_end(st.handle, 128)
    torch.cuda.synchronize()
    prof.sort(key=lambda e: -e["total_ms"])
    for e in prof:
        log("[bench]   %-18s %5d launches %9.3f ms total %8.2f us avg  %7.1f TFLOP/s  %7.1f GB/s" % (
            e["name"], e["launches"], e["total_ms"], 1e3 * e["total_ms"] / e["launches"],
            e["flops"] / (e["total_ms"] * 1e-3) / 1e12 if e["total_ms"] else 0,
            e["bytes"] / (e["total_ms"] * 1e-3) / 1e9 if e["total_ms"] else 0))
    gemms = [e for e in prof if e["name"].startswith(GEMM_PREFIX)]
    gemm_flops = sum(e["flops"] for e in gemms)
    gemm_ms = sum(e["total_ms"] for e in gemms)
    # the projection FLOPs alone: the fused QKV projection + attention kernel also
    # counts the attention's 4 B H S^2 d_head per launch, which is not GEMM work
    attn_in_gemm = sum(e["launches"] * 4.0 * w.batch * w.n_heads * w.seq * w.seq * (w.d_model // w.n_heads)
                       for e in gemms if e["name"] == "gemm_qkv_attn_fwd")
    all_flops = sum(e["flops"] for e in prof)
    dom = prof[0]
    dom_avg_s = dom["total_ms"] * 1e-3 / dom["launches"]
    if dom["name"].startswith(("gemm_", "attn_")):  # dense contractions; the rest is HBM-bound
        achieved = dom["flops"] / dom["launches"] / dom_avg_s / 1e12
        roof = {"kernel": dom["name"], "bound": "mfma", "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": None, "avg_us": round(dom_avg_s * 1e6, 2), "launches_per_step": dom["launches"] // args.steps}
    else:
        achieved = dom["bytes"] / dom["launches"] / dom_avg_s / 1e9
        roof = {"kernel": dom["name"], "bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                "avg_us": round(dom_avg_s * 1e6, 2), "launches_per_step": dom["launches"] // args.steps}

    roof["traffic"] = recorded_traffic(dom["name"], w.name)
    # the same kernel's average duration in the committed rocprofv3 kernel trace
    # (null if its sources changed since), and the fraction that duration gives
    traced = recorded_trace_us(dom["name"], w.name)
    roof["traced_avg_us"] = traced
    roof["frac_traced"] = (round(dom["flops" if roof["bound"] == "mfma" else "bytes"] / dom["launches"] / (traced * 1e-6)
                                 / (1e12 if roof["bound"] == "mfma" else 1e9) / roof["peak"], 4) if traced else None)
    cpu = None if args.no_cpu_baseline else cpu_baseline(w, inp)
    st.close()
    if args.copy_calib_mib:
        copy_calibration(torch, args.copy_calib_mib)
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "samples/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.n_blocks} {'post-LN' if w.arch == 'bert' else 'pre-RMSNorm'} "
                               f"blocks, d={w.d_model}, {w.n_heads} heads, FFN {w.d_ffn}, "
                               + ("one adapter/block after the FFN" if w.placement == "ffn" else "two adapters/block")
                               + f" m={w.d_adapter}, seq {w.seq}, batch {w.batch}, lowest unfrozen block {c}",
                   "batch": w.batch, "seq_len": w.seq, "n_blocks": w.n_blocks, "lowest_unfrozen": c,
                   "placement": w.placement,
                   "parallelism": "one ring stage on one GPU"},
        "tokens_per_s": round(value * w.seq, 1),
        "gemm_mfma_frac": (round((gemm_flops - attn_in_gemm) / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
                           if gemm_ms else None),
        "gemm_attn_mfma_frac": round(gemm_flops / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4) if gemm_ms else None,
        "stage_mfma_frac": round(all_flops / args.steps / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "stash_bytes": stash_bytes, "scratch_bytes": scratch_bytes,
        "launch": "hip_graph" if run is not step else "eager",
        "roofline": roof, "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
