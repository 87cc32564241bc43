#!/usr/bin/env python3
"""Benchmark of the folded MoE layer on one MI355X.

Default workload: the Mixtral-8x7B-shaped layer (bf16, hidden 4096, 8 experts,
top-2, intermediate 14336).  One step = one prefill forward (4096 tokens,
K'=1 token-level folding) + one decode forward (32 tokens, pool of 4 of 8
experts), each the whole folded layer: router, Top-K, selection, fold,
permutation, grouped SwiGLU GEMMs, combine.  Inputs are seeded synthetic data
resident in HBM before the timed region; the projector tables are seeded
stand-ins (their values only steer selection, not the amount of work).

Prints ONE JSON line: value = prefill TFLOP/s (algorithmic flops / mean
prefill-layer time), with the decode layer's us/layer and HBM GB/s, the
roofline of the dominant kernel (the prefill gate/up GEMM, timed live with
HIP events on its stream), the CPU oracle timed on a bounded sample (folded
and unfolded), and a `secondary` block: the Qwen3-30B-A3B-shaped layer's
prefill (8192 tokens, K'=4) and decode (128 tokens, D=16), folded and
unfolded, timed in the same run.  The
timed steps record HIP events only at the layer boundaries and around the
dominant kernel; the per-stage breakdown in the line comes from a second,
fully instrumented run of the same steps after the timed region.  `clock`
holds the GFX clock the driver reports for each XCD (amd-smi, three readings)
while prefill forwards run back to back after the timed region, and the peak
fractions against the dense peak at that clock (null without amd-smi, and null
with `plausible` false when the reading is below the clock that the measured
gate/up rate needs).

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--workload mixtral|qwen3|glm|qwen3-decode]

Two helper modes serve the committed profile summaries:

    python bench.py --copy-calibration          # one 1 GiB device copy (counter scale)
    python bench.py --prof-summary DIR          # markdown summary of the rocprofv3 runs in DIR

`roofline.traffic` is read from the committed traffic summary of the dominant
kernel, and only when the kernel sources still hash to what was profiled
(otherwise it is null).
"""

from __future__ import annotations

import argparse
import csv
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_24938_amd.measure import (PEAK_BF16_TFLOPS, PEAK_HBM_GBS, HipEvents,  # noqa: E402
                                          decode_bytes, make_layer, prefill_flops)

METRIC = "folded MoE layer: prefill TFLOP/s + %MFMA peak; decode µs/layer + HBM GB/s"
COPY_BYTES = 1 << 30        # size of the calibration copy
# the dominant launch: the prefill gate/up GEMM with fused SiLU*up (256x256 tiles) and the fixup of its
# split remainder (both inside the gate/up stage the events time)
DOMINANT = ("expert_gate_up_wide", "expert_wide_fixup<true, false>")
KERNEL_SOURCES = ["paper_2608_24938_amd/csrc/k_gemm.hip", "paper_2608_24938_amd/csrc/common.hpp",
                  "paper_2608_24938_amd/csrc/kernels.hpp", "paper_2608_24938_amd/build.py"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "expert_gemm_gate_up_mixtral_prefill_traffic.md")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_sources_sha256():
    """Hash of the sources that define the dominant kernel and its compile flags."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(workload):
    """Scaled HBM bytes per launch of the dominant kernel from the committed summary, or None when the
    summary is absent, covers another workload or was taken from different kernel sources."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    m = re.search(r"^traffic-record: (\{.*\})\s*$", text, re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("sources_sha256") != kernel_sources_sha256() or rec.get("workload") != workload:
        return None
    return rec


def run_phase(X, layer, x, phase, budget, tables, warmup, dbg=None):
    """Output and workspace of one phase, after `warmup` untimed forwards."""
    import torch
    S, L, h = tables
    y = torch.empty_like(x)
    ws = torch.empty(X.moe_workspace_size(layer, x.shape[0], phase, budget), dtype=torch.uint8, device="cuda")
    for _ in range(warmup):
        X.moe_forward(layer, x, phase, budget, S, L, h, y=y, workspace=ws, debug=dbg)
    torch.cuda.synchronize()
    return y, ws


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="mixtral", choices=["mixtral", "qwen3", "glm", "qwen3-decode"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the Qwen3-shaped prefill and decode timed after the main workload")
    ap.add_argument("--no-clock", action="store_true",
                    help="skip the amd-smi clock readings (for runs under a profiler, whose preloaded "
                         "library must not reach the amd-smi child process)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one plain 1 GiB device copy (the scale for the FETCH_SIZE/WRITE_SIZE counters)")
    ap.add_argument("--prof-summary", metavar="DIR",
                    help="print a markdown summary of the rocprofv3 runs under DIR (trace/, fetch/, write/, "
                         "copyfetch/, copywrite/) and exit")
    args = ap.parse_args()
    if args.prof_summary:
        print(prof_summary(args.prof_summary, args.workload, args.steps))
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the folded layer is measured "
              f"on a single MI355X and no multi-GPU path is built.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2608_24938_amd import exfold as X
    from paper_2608_24938_amd import synth

    X.lib()  # fail loudly if the library is missing
    torch.cuda.init()
    props = torch.cuda.get_device_properties(0)
    log(f"device: {props.name} CUs={props.multi_processor_count}")

    if args.workload == "mixtral":
        shape = synth.MIXTRAL
        prefill = (4096, 1)
        decode = (32, 4)
        workload = "mixtral-8x7b-shaped MoE layer (d=4096, 8 experts, top-2, I=14336, bf16): " \
                   "prefill 4096 tokens K'=1 + decode 32 tokens pool D=4"
    elif args.workload == "qwen3":
        shape = synth.QWEN3
        prefill = (8192, 4)
        decode = (64, 32)
        workload = "qwen3-30b-a3b-shaped MoE layer (d=2048, 128 experts, top-8, I=768, skewed router, bf16): " \
                   "prefill 8192 tokens K'=4 + decode 64 tokens pool D=32"
    elif args.workload == "glm":
        shape = synth.GLM45
        prefill = (4096, 4)
        decode = (64, 32)
        workload = "glm-4.5-air-shaped MoE layer (d=4096, 128 experts + 1 shared, top-8, I=1408, bf16): " \
                   "prefill 4096 tokens K'=4 + decode 64 tokens pool D=32"
    else:
        shape = synth.QWEN3_DECODE
        prefill = (512, 4)
        decode = (128, 16)
        workload = "qwen3-30b-a3b-shaped MoE layer (bf16): prefill 512 tokens K'=4 + decode 128 tokens pool D=16"

    t0 = time.time()
    layer, host, dev = make_layer(shape, seed=0)
    T, kp = prefill
    B, D = decode
    xs_p = synth.tokens(shape, T, seed=0)
    xs_d = synth.tokens(shape, B, seed=1)
    x_p, x_d = dev(xs_p), dev(xs_d)
    S_np, L_np, h_np = synth.synthetic_tables(shape.n_experts, seed=0)
    tables = (dev(S_np), dev(L_np), dev(h_np))
    torch.cuda.synchronize()
    log(f"inputs ready in {time.time() - t0:.1f}s")

    stream = torch.cuda.current_stream()
    sptr = ctypes.c_void_p(stream.cuda_stream)
    ev = HipEvents()
    dbg_d = {"pool_size": torch.empty(1, dtype=torch.int32, device="cuda")}
    S, L, h = tables
    y_p, ws_p = run_phase(X, layer, x_p, "prefill", kp, tables, args.warmup)
    y_d, ws_d = run_phase(X, layer, x_d, "decode", D, tables, args.warmup, dbg_d)
    names = X.EVENT_NAMES
    START, PERMUTE, GATE_UP, END = (names.index(n) for n in ("start", "permute", "gate_up", "end"))

    def sparse(idx):
        """Per-step event arrays that record only the stage boundaries in idx (NULL entries are skipped)."""
        out = []
        for _ in range(args.steps):
            full = ev.array(X.N_EVENTS)
            arr = (ctypes.c_void_p * X.N_EVENTS)()
            for i in idx:
                arr[i] = full[i]
            out.append(arr)
        return out

    # timed steps: the layer boundaries, plus the gate/up GEMM launch of the prefill forward (the
    # dominant kernel); no other events inside the layer
    ev_p, ev_d = sparse((START, PERMUTE, GATE_UP, END)), sparse((START, END))
    edge = ev.array(2)
    torch.cuda.synchronize()
    # ---- timed region: exactly `steps` steps, synchronised on both sides ----
    ev.record(edge[0], sptr)
    for k in range(args.steps):
        X.moe_forward(layer, x_p, "prefill", kp, S, L, h, y=y_p, workspace=ws_p, events=ev_p[k])
        X.moe_forward(layer, x_d, "decode", D, S, L, h, y=y_d, workspace=ws_d, events=ev_d[k], debug=dbg_d)
    ev.record(edge[1], sptr)
    torch.cuda.synchronize()
    total_ms = ev.ms(edge[0], edge[1])

    def mean_us(arrs, a, b):
        return float(np.mean([ev.ms(x[a], x[b]) for x in arrs])) * 1e3

    layer_p, layer_d = mean_us(ev_p, START, END), mean_us(ev_d, START, END)
    gate_up_us = mean_us(ev_p, PERMUTE, GATE_UP)

    # stage breakdown (informational): a separate run with an event at every stage boundary
    st_ev_p, st_ev_d = [ev.array(X.N_EVENTS) for _ in range(args.steps)], [ev.array(X.N_EVENTS) for _ in range(args.steps)]
    for k in range(args.steps):
        X.moe_forward(layer, x_p, "prefill", kp, S, L, h, y=y_p, workspace=ws_p, events=st_ev_p[k])
        X.moe_forward(layer, x_d, "decode", D, S, L, h, y=y_d, workspace=ws_d, events=st_ev_d[k], debug=dbg_d)
    torch.cuda.synchronize()

    def stages(arrs):
        out = {}
        for i in range(1, len(names)):
            out[names[i]] = mean_us(arrs, i - 1, i)
        out["layer"] = mean_us(arrs, 0, len(names) - 1)
        return out

    st_p, st_d = stages(st_ev_p), stages(st_ev_d)
    touched = int(dbg_d["pool_size"].item())
    flops_p = prefill_flops(shape, T, kp)
    tflops = flops_p / (layer_p * 1e-6) / 1e12
    gu_flops = 4 * shape.d * shape.inter * (T * kp + (T if shape.shared_inter else 0))
    gu_tflops = gu_flops / (gate_up_us * 1e-6) / 1e12
    bytes_d = decode_bytes(shape, B, touched)
    gbs_d = bytes_d / (layer_d * 1e-6) / 1e9
    log(f"prefill stages (us): {json.dumps({k: round(v, 1) for k, v in st_p.items()})}")
    log(f"decode stages (us): {json.dumps({k: round(v, 1) for k, v in st_d.items()})}")

    # algorithmic bytes of one gate/up launch: the touched experts' gate/up weights, the gathered
    # activations and the H it writes
    esz = 2 if shape.dtype == "bf16" else 4
    gu_rows = T * kp + (T if shape.shared_inter else 0)
    n_groups = shape.n_experts + (1 if shape.shared_inter else 0)
    gu_bytes = (2 * shape.inter * shape.d * n_groups + gu_rows * shape.d + gu_rows * shape.inter) * esz
    traffic = recorded_traffic(args.workload)
    clock = None if args.no_clock else measured_gfx_clock(
        lambda: X.moe_forward(layer, x_p, "prefill", kp, S, L, h, y=y_p, workspace=ws_p))
    if clock is not None:
        # a reading is used only if the measured gate/up rate fits under the dense MFMA rate at
        # that clock (a lower reading cannot have held while the kernel ran)
        scale = NOMINAL_SCLK_MHZ / clock["mean_mhz"]
        pf, rf = tflops / PEAK_BF16_TFLOPS * scale, gu_tflops / PEAK_BF16_TFLOPS * scale
        clock["plausible"] = rf <= 1.0
        clock["prefill_frac_at_measured_clock"] = round(pf, 4) if rf <= 1.0 else None
        clock["roofline_frac_at_measured_clock"] = round(rf, 4) if rf <= 1.0 else None

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(shape, host, xs_p, (S_np, L_np, h_np), kp)

    secondary = None
    if args.workload == "mixtral" and not args.no_secondary:
        del layer, host, x_p, x_d, y_p, y_d, ws_p, ws_d
        torch.cuda.empty_cache()
        secondary = secondary_configs(X, ev, args.steps, args.warmup)

    rec = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) tokens, N(0,0.02^2) weights, seeded stand-in projector tables)",
        "config": {"workload": workload, "prefill_tokens": T, "k_pre": kp, "decode_tokens": B, "pool_budget": D},
        "prefill": {"us_per_layer": round(layer_p, 1), "tflops": round(tflops, 2),
                    "frac_mfma_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
                    "algorithmic_gflop": round(flops_p / 1e9, 2),
                    "stages_us_instrumented": {k: round(v, 1) for k, v in st_p.items()}},
        "decode": {"us_per_layer": round(layer_d, 1), "hbm_gbs": round(gbs_d, 1),
                   "frac_hbm_peak": round(gbs_d / PEAK_HBM_GBS, 4), "experts_touched": touched,
                   "algorithmic_mb": round(bytes_d / 1e6, 2),
                   "stages_us_instrumented": {k: round(v, 1) for k, v in st_d.items()}},
        "roofline": {"bound": "mfma", "achieved": round(gu_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(gu_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": None if traffic is None else traffic["bytes_per_launch"],
                     "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                     "algorithmic_bytes": gu_bytes,
                     "kernel": " + ".join(DOMINANT) + " (prefill gate/up GEMM, fused SiLU*up)",
                     "per_launch_gflop": round(gu_flops / 1e9, 2), "avg_launch_us": round(gate_up_us, 1)},
        "cpu_baseline": cpu,
        "secondary": secondary,
        "clock": clock,
    }
    ev.close()
    print(json.dumps(rec), flush=True)


NOMINAL_SCLK_MHZ = 2400  # the clock of the dense peak figure


def measured_gfx_clock(fwd, seconds=2.0, samples=3):
    """The GFX clock of each XCD as the driver reports it (`amd-smi metric -c`), sampled `samples`
    times while fwd() runs back to back (the first 0.5 s into the load, then one about every 0.3 s
    after the previous reading returns); None where amd-smi is missing or fails.  mean_mhz is the
    median over the samples of their mean over the XCDs."""
    import shutil
    import subprocess
    import threading
    import numpy as np
    import torch
    exe = shutil.which("amd-smi")
    if exe is None:
        return None
    texts = []

    def sample():
        time.sleep(0.5)
        for _ in range(samples):
            try:
                texts.append(subprocess.run([exe, "metric", "-c"], capture_output=True, text=True, timeout=10).stdout)
            except (OSError, subprocess.SubprocessError):
                pass
            time.sleep(0.3)

    th = threading.Thread(target=sample)
    t0 = time.time()
    th.start()
    while (th.is_alive() or time.time() - t0 < seconds) and time.time() - t0 < 40:
        for _ in range(10):
            fwd()
        torch.cuda.synchronize()
    th.join(timeout=15)
    per = [[int(v) for v in re.findall(r"GFX_\d+:\s+CLK:\s+(\d+)\s*MHz", t)] for t in texts]
    per = [m for m in per if m]
    if not per:
        return None
    means = [float(np.mean(m)) for m in per]
    return {"source": "amd-smi metric -c, sampled during back-to-back prefill forwards", "gfx_mhz": per,
            "sample_mean_mhz": [round(v, 1) for v in means], "mean_mhz": round(float(np.median(means)), 1),
            "nominal_mhz": NOMINAL_SCLK_MHZ}


def secondary_configs(X, ev, steps, warmup):
    """The Qwen3-30B-A3B-shaped layer (d=2048, 128 experts, top-8, I=768, skewed router), timed in the
    same run as the main workload: a prefill of 8192 tokens with K'=4 and a decode batch of 128 tokens
    with a pool of D=16, each folded and unfolded (every Top-K route executed), `steps` forwards
    after `warmup`, HIP events at each forward's start and end on the library's stream."""
    import numpy as np
    import torch
    from paper_2608_24938_amd import synth
    shape = synth.QWEN3
    layer, _, dev = make_layer(shape, seed=0)
    tables = tuple(dev(a) for a in synth.synthetic_tables(shape.n_experts, seed=0))
    sptr = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    out = {}
    for key, phase, T, budget, seed in (("qwen3_prefill", "prefill", 8192, 4, 0),
                                        ("qwen3_decode", "decode", 128, 16, 1)):
        x = dev(synth.tokens(shape, T, seed=seed))
        y = torch.empty_like(x)
        ws = torch.empty(max(X.moe_workspace_size(layer, T, phase, budget), X.moe_workspace_size(layer, T, "dense", 0)),
                         dtype=torch.uint8, device="cuda")
        dbg = {"offsets": torch.empty(shape.n_experts + 2, dtype=torch.int32, device="cuda")}

        def timed(ph, bud):
            for _ in range(warmup):
                X.moe_forward(layer, x, ph, bud, *tables, y=y, workspace=ws)
            torch.cuda.synchronize()
            arrs = [ev.array(2) for _ in range(steps)]
            for a in arrs:
                ev.record(a[0], sptr)
                X.moe_forward(layer, x, ph, bud, *tables, y=y, workspace=ws)
                ev.record(a[1], sptr)
            torch.cuda.synchronize()
            return float(np.mean([ev.ms(a[0], a[1]) for a in arrs])) * 1e3

        us = timed(phase, budget)
        us_dense = timed("dense", 0)
        X.moe_forward(layer, x, phase, budget, *tables, y=y, workspace=ws, debug=dbg)
        counts = np.diff(dbg["offsets"].cpu().numpy()[: shape.n_experts + 1])
        touched = int((counts > 0).sum())
        rec = {"us_per_layer": round(us, 1), "unfolded_us_per_layer": round(us_dense, 1), "experts_touched": touched}
        if phase == "prefill":
            flops = prefill_flops(shape, T, budget)
            wbytes = 3 * shape.d * shape.inter * 2 * touched + 2 * T * shape.d * 2
            rec.update(workload=f"qwen3-30b-a3b-shaped MoE layer (d=2048, 128 experts, top-8, I=768, skewed router, "
                                f"bf16): prefill {T} tokens K'={budget}",
                       tflops=round(flops / (us * 1e-6) / 1e12, 2),
                       frac_mfma_peak=round(flops / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4),
                       algorithmic_gflop=round(flops / 1e9, 2),
                       hbm_gbs=round(wbytes / (us * 1e-6) / 1e9, 1),
                       frac_hbm_peak=round(wbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                       max_rows_per_expert=int(counts.max()), mean_rows_per_expert=round(float(counts[counts > 0].mean()), 1))
        else:
            nbytes = decode_bytes(shape, T, touched)
            rec.update(workload=f"qwen3-30b-a3b-shaped MoE layer (bf16): decode {T} tokens, pool D={budget}",
                       hbm_gbs=round(nbytes / (us * 1e-6) / 1e9, 1),
                       frac_hbm_peak=round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
                       algorithmic_mb=round(nbytes / 1e6, 2))
        out[key] = rec
        log(f"{key}: {json.dumps(rec)}")
    return out


def cpu_baseline(shape, host, xs_p, tables, kp, target_s=15.0, probe_tokens=64):
    """The oracle, as it stands, on a bounded prefix of the prefill batch (folded layer).  The prefix
    grows 4x per run (from probe_tokens) until a run takes target_s/2 or covers the whole batch; the
    last run is the one reported."""
    import numpy as np
    from oracle import exfold_oracle as O
    from paper_2608_24938_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [os.cpu_count()])
    except Exception:
        threads = os.cpu_count()
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{blas.get('name')} {blas.get('version')}"
    except Exception:
        blas = "unknown"
    widen = synth.widen
    ref = O.Layer(w_router=widen(host["wr"]), w_gate_up=lambda e: widen(host["gu"][e]),
                  w_down=lambda e: widen(host["dn"][e]), router_bias=host["bias"],
                  ws_gate_up=None if host["sgu"] is None else widen(host["sgu"]),
                  ws_down=None if host["sdn"] is None else widen(host["sdn"]))
    S, L, h = tables

    def timed(n, phase="prefill"):
        x = widen(xs_p[:n])
        t0 = time.perf_counter()
        O.moe_forward(ref, x, shape.top_k, phase, kp, S, L, h)
        return time.perf_counter() - t0

    n_tokens = min(probe_tokens, xs_p.shape[0])
    dt = timed(n_tokens)
    while dt < target_s / 2 and n_tokens < xs_p.shape[0]:
        log(f"cpu oracle: {n_tokens} tokens in {dt:.2f}s")
        n_tokens = min(xs_p.shape[0], 4 * n_tokens)
        dt = timed(n_tokens)
    flops = prefill_flops(shape, n_tokens, kp)
    log(f"cpu oracle: {n_tokens} tokens in {dt:.2f}s")
    dt_dense = timed(n_tokens, "dense")
    log(f"cpu oracle, unfolded: {n_tokens} tokens in {dt_dense:.2f}s")
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n_tokens} of the {xs_p.shape[0]} prefill tokens, folded layer (float64 NumPy), "
                      f"{dt:.2f} s wall", "seconds": round(dt, 3), "unfolded_seconds": round(dt_dense, 3),
            "host_cpus": os.cpu_count(), "blas": blas, "blas_threads": int(threads)}


def copy_calibration():
    """One plain device-to-device copy of COPY_BYTES (after a warm-up copy): the kernel whose FETCH_SIZE and
    WRITE_SIZE counter values scale the counters of the other kernels to bytes."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(2):
        torch.mul(src, 1.0, out=dst)   # an elementwise kernel: reads COPY_BYTES, writes COPY_BYTES
    torch.cuda.synchronize()
    log(f"copied {COPY_BYTES} bytes twice")


def _counters(path):
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            key = (r["Kernel_Name"], int(r["Grid_Size"]))
            out.setdefault(key, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return out


def _find(dirname, suffix):
    for root, _, files in os.walk(dirname):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    raise FileNotFoundError(f"no *{suffix} under {dirname}")


def prof_summary(d, workload, steps):
    """Markdown summary of the rocprofv3 runs under d; `steps` is the --steps of the traced run.  Each
    kernel's launches end with the `steps` timed steps and then the `steps` steps of the instrumented
    stage breakdown, so the timed launches are the `steps` before the last `steps`."""
    mean = lambda v: sum(v) / len(v)
    cf = _counters(_find(os.path.join(d, "copyfetch"), "counter_collection.csv"))
    cw = _counters(_find(os.path.join(d, "copywrite"), "counter_collection.csv"))
    # the calibration copy is the launch that reads the most (the buffer fill before it only writes)
    ck = max(cf, key=lambda k: mean(cf[k]["FETCH_SIZE"]))
    fetch_kib = mean(cf[ck]["FETCH_SIZE"])
    write_kib = mean(cw[ck]["WRITE_SIZE"])
    f_fac = COPY_BYTES / (fetch_kib * 1024)
    w_fac = COPY_BYTES / (write_kib * 1024)
    lines = [f"copy calibration: kernel `{ck[0]}` copying {COPY_BYTES} B reads FETCH_SIZE {fetch_kib:.0f} KiB and "
             f"WRITE_SIZE {write_kib:.0f} KiB per dispatch -> scale FETCH_SIZE x{f_fac:.4f}, WRITE_SIZE x{w_fac:.4f}",
             ""]
    trace = _find(os.path.join(d, "trace"), "kernel_trace.csv")
    durs = {}
    with open(trace) as f:
        for r in csv.DictReader(f):
            grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
            key = (r["Kernel_Name"], grid)
            durs.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    fe = _counters(_find(os.path.join(d, "fetch"), "counter_collection.csv"))
    wr = _counters(_find(os.path.join(d, "write"), "counter_collection.csv"))
    lines.append("| kernel | grid (work-items) | launches | avg us | avg us, timed steps | min us | "
                 "HBM read MB/launch | HBM write MB/launch |")
    lines.append("|---|---|---|---|---|---|---|---|")
    record = None
    dom = {"avg_us": 0.0, "timed": 0.0, "rd": 0.0, "wt": 0.0, "grids": [], "found": 0}
    for key, v in sorted(durs.items(), key=lambda kv: -sum(kv[1])):
        name = key[0].replace("exfold::", "").replace("(GemmKArgs)", "").replace("void ", "")
        rd = mean(fe[key]["FETCH_SIZE"]) * 1024 * f_fac if key in fe else None
        wt = mean(wr[key]["WRITE_SIZE"]) * 1024 * w_fac if key in wr else None
        fmt = lambda b: "-" if b is None else f"{b / 1e6:.1f}"
        timed = mean(v[-2 * steps:-steps]) if len(v) >= 2 * steps else mean(v)
        lines.append(f"| `{name[:80]}` | {key[1]} | {len(v)} | {mean(v):.1f} | {timed:.1f} | {min(v):.1f} | "
                     f"{fmt(rd)} | {fmt(wt)} |")
        part = next((i for i, n in enumerate(DOMINANT) if n in key[0]), None)
        if part is not None and rd is not None and wt is not None and not dom["found"] & (1 << part):
            dom["found"] |= 1 << part
            dom["avg_us"] += mean(v)
            dom["timed"] += timed
            dom["rd"] += rd
            dom["wt"] += wt
            dom["grids"].append(key[1])
    if dom["found"] == (1 << len(DOMINANT)) - 1:
        record = {"workload": workload, "kernel": " + ".join(DOMINANT), "grid": dom["grids"],
                  "avg_us": round(dom["avg_us"], 1), "avg_us_timed_steps": round(dom["timed"], 1),
                  "fetch_bytes": round(dom["rd"]), "write_bytes": round(dom["wt"]),
                  "bytes_per_launch": round(dom["rd"] + dom["wt"]),
                  "fetch_scale": round(f_fac, 4), "write_scale": round(w_fac, 4),
                  "sources_sha256": kernel_sources_sha256()}
    lines.append("")
    if record is not None:
        lines.append("The dominant launch is the prefill gate/up GEMM and the fixup of its split remainder (the "
                     "gate/up stage); their traffic (read + write, scaled) per launch, summed:")
        lines.append("")
        lines.append("traffic-record: " + json.dumps(record))
    return "\n".join(lines)


if __name__ == "__main__":
    main()
