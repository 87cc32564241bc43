"""Timing sweep of the folded layer over the synthetic workload configurations.

For each configuration (``synth.WORKLOADS``: the tiny fp32 layer, the
Mixtral-, Qwen3- and GLM-shaped prefill and decode cases) on one GPU:

* folded forward (``exfold_moe_forward`` in the configuration's phase) and the
  unfolded forward (dense phase: every Top-K route executed) on the same tokens,
  each timed with HIP events around the single forward;
* cold cache by default: a 1 GiB scratch buffer is read before every timed
  forward, so no weight stays in the L2 or the 256 MB Infinity Cache (a read,
  not a write: dirty scratch lines would charge their write-back to the
  forward); warm numbers (no scratch read) are reported beside them;
* the same forward captured once in a HIP graph and replayed (warm), which
  removes the host's launch overhead between the layer's kernels;
* median, p10 and p90 over the repetitions; the spread of the median over eight
  further token batches (the pool and the routes change with the tokens; each
  batch gets two untimed forwards first);
* the stage breakdown of one instrumented forward, and the folding overhead:
  router + Top-K/selection/fold + permutation as a share of the layer;
* experts touched and rows per expert (max / mean over touched experts);
* prefill: algorithmic TFLOP/s and % of the dense bf16 MFMA peak; decode:
  algorithmic HBM bytes (touched experts' weights, router, x, y) in GB/s and %
  of the HBM peak;
* decode: the same batch on a static pool of the same budget (tables formed
  once), with the front-end µs it saves against the batch pool.

    python -m paper_2608_24938_amd.sweep [--only NAME ...] [--reps-prefill 20] [--reps-decode 100]
                                         [--md FILE] [--ceilings]

Prints one JSON line per configuration; --md also writes a markdown table.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import sys

import numpy as np

from . import synth
from .measure import PEAK_BF16_TFLOPS, PEAK_HBM_GBS, HipEvents, decode_bytes, make_layer, prefill_flops

SCRATCH_BYTES = 1 << 30
N_BATCHES = 8


def _pct(v, q):
    return float(np.percentile(np.asarray(v), q))


def _time(X, ev, stream, fwd, reps, scratch):
    """Per-rep µs of fwd() between two events on the library's stream."""
    sptr = ctypes.c_void_p(stream.cuda_stream)
    pairs = [ev.array(2) for _ in range(reps)]
    for a in pairs:
        if scratch is not None:
            scratch.sum()
        ev.record(a[0], sptr)
        fwd()
        ev.record(a[1], sptr)
    stream.synchronize()
    return [ev.ms(a[0], a[1]) * 1e3 for a in pairs]


def _capture(fwd):
    """fwd captured in a HIP graph (warmed up on a side stream first, as torch requires)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fwd()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fwd()
    torch.cuda.synchronize()
    return g


def _stages(X, ev, stream, fwd, reps=5):
    """Median µs of every stage from fully instrumented forwards."""
    arrs = [ev.array(X.N_EVENTS) for _ in range(reps)]
    for a in arrs:
        fwd(a)
    stream.synchronize()
    names = X.EVENT_NAMES
    out = {}
    for i in range(1, len(names)):
        out[names[i]] = float(np.median([ev.ms(a[i - 1], a[i]) for a in arrs])) * 1e3
    out["layer"] = float(np.median([ev.ms(a[0], a[len(names) - 1]) for a in arrs])) * 1e3
    return out


def run_config(name, wl, layer, dev, args, ev, stream, scratch):
    import torch
    from . import exfold as X

    shape, phase, T, budget = wl.shape, wl.phase, wl.tokens, wl.budget
    S, L, h = (dev(a) for a in synth.synthetic_tables(shape.n_experts, seed=0))
    x = dev(synth.tokens(shape, T, seed=1))
    y = torch.empty_like(x)
    ws = torch.empty(X.moe_workspace_size(layer, T, phase, budget), dtype=torch.uint8, device="cuda")
    ws_dense = torch.empty(X.moe_workspace_size(layer, T, "dense", shape.top_k), dtype=torch.uint8,
                           device="cuda")
    dbg = X.debug_buffers(layer, T, phase, budget, "cuda")
    reps = args.reps_prefill if phase == "prefill" else args.reps_decode

    def folded(xx=x, events=None, debug=None):
        X.moe_forward(layer, xx, phase, budget, S, L, h, y=y, workspace=ws, events=events, debug=debug)

    def dense():
        X.moe_forward(layer, x, "dense", shape.top_k, y=y, workspace=ws_dense)

    for _ in range(args.warmup):
        folded()
        dense()
    folded(debug=dbg)
    stream.synchronize()
    offs = dbg["offsets"].cpu().numpy()[: shape.n_experts + 1].astype(np.int64)
    rows = np.diff(offs)
    touched = int((rows > 0).sum())

    cold = _time(X, ev, stream, folded, reps, scratch)
    warm = _time(X, ev, stream, folded, reps, None)
    cold_dense = _time(X, ev, stream, dense, max(5, reps // 2), scratch)
    # the further batches are drawn and copied to the device before any of them is timed: drawing one
    # leaves the GPU idle long enough for its clock to drop, which the next forwards would pay
    xb = [dev(synth.tokens(shape, T, seed=100 + i)) for i in range(N_BATCHES)]
    batch_medians = []
    for xi in xb:
        for _ in range(args.warmup):  # untimed: the first forwards on a new batch pay one-time costs
            folded(xi)
        batch_medians.append(float(np.median(_time(X, ev, stream, lambda: folded(xi), max(5, reps // 4),
                                                   scratch))))
    del xb
    st = _stages(X, ev, stream, lambda a: folded(events=a))
    graph = _capture(folded)
    graph_warm = _time(X, ev, stream, graph.replay, reps, None)

    t = float(np.median(cold))
    rec = {
        "config": name, "shape": shape.name, "phase": phase, "tokens": T, "budget": budget,
        "dtype": shape.dtype, "reps": reps,
        "us_cold": {"median": round(t, 1), "p10": round(_pct(cold, 10), 1), "p90": round(_pct(cold, 90), 1)},
        "us_warm_median": round(float(np.median(warm)), 1),
        "us_graph_warm_median": round(float(np.median(graph_warm)), 1),
        "us_unfolded_cold_median": round(float(np.median(cold_dense)), 1),
        "us_median_over_8_batches": {"min": round(min(batch_medians), 1), "max": round(max(batch_medians), 1)},
        # the median over all nine batches (this one and the eight further ones)
        "us_median_over_9_batches": round(float(np.median(batch_medians + [t])), 1),
        "experts_touched": touched,
        "rows_per_touched_expert": {"max": int(rows.max()), "mean": round(float(rows[rows > 0].mean()), 1)},
        "stages_us": {k: round(v, 1) for k, v in st.items()},
        "fold_overhead_share": round((st["router"] + st["fold"] + st["permute"]) / st["layer"], 4),
    }
    if phase == "prefill" and shape.dtype == "bf16":
        k_out = min(budget, shape.top_k)
        fl = prefill_flops(shape, T, k_out)
        rec["tflops"] = round(fl / (t * 1e-6) / 1e12, 1)
        rec["frac_mfma_peak"] = round(fl / (t * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)
        rec["unfolded_tflops_equiv"] = round(prefill_flops(shape, T, shape.top_k) /
                                             (rec["us_unfolded_cold_median"] * 1e-6) / 1e12, 1)
    elif phase.startswith("decode"):
        by = decode_bytes(shape, T, touched)
        rec["algorithmic_mb"] = round(by / 1e6, 1)
        rec["hbm_gbs"] = round(by / (t * 1e-6) / 1e9, 1)
        rec["frac_hbm_peak"] = round(by / (t * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)
    if phase == "decode":
        rec["static"] = static_pool_timing(X, ev, stream, layer, x, y, budget, (S, L, h), reps, scratch, st, args)
    return rec


def static_pool_timing(X, ev, stream, layer, x, y, budget, tables, reps, scratch, st_dyn, args):
    """The same batch on a static pool of the same budget (the D experts of largest h, per-source tables
    formed once, Eq. appendix_decode_static_budget): cold and graph µs, experts touched, and the
    front-end µs (Top-K, pool, tables, remap and permutation: the router-to-fold stages) against the
    batch pool's."""
    import torch
    S, L, h = tables
    _, _, tgt, scl = X.static_pool(h, budget, S, L)
    ws = torch.empty(X.moe_workspace_size(layer, x.shape[0], "decode_static", budget), dtype=torch.uint8,
                     device="cuda")
    dbg = X.debug_buffers(layer, x.shape[0], "decode_static", budget, "cuda")

    def fwd(events=None, debug=None):
        X.moe_forward(layer, x, "decode_static", budget, S, L, h, y=y, workspace=ws, events=events,
                      debug=debug, static_tables=(tgt, scl))

    for _ in range(args.warmup):
        fwd()
    fwd(debug=dbg)
    stream.synchronize()
    rows = np.diff(dbg["offsets"].cpu().numpy()[: layer.n_experts + 1].astype(np.int64))
    cold = _time(X, ev, stream, fwd, reps, scratch)
    st = _stages(X, ev, stream, lambda a: fwd(events=a))
    g = _capture(fwd)
    graph = _time(X, ev, stream, g.replay, reps, None)
    front = lambda q: q["fold"] + q["permute"]
    return {"us_cold_median": round(float(np.median(cold)), 1), "us_graph_warm_median": round(float(np.median(graph)), 1),
            "experts_touched": int((rows > 0).sum()), "front_us": round(front(st), 1),
            "front_us_batch_pool": round(front(st_dyn), 1), "front_us_saved": round(front(st_dyn) - front(st), 1),
            "stages_us": {k: round(v, 1) for k, v in st.items()}}


def ceilings(ev, stream):
    """Context for the fractions: large plain bf16 GEMMs through torch (hipBLASLt) with the weights
    stored as the layer stores them ([N_out, K], the product x W^T) and as [K, N_out] (x W), one
    Mixtral-shaped expert (512 x 28672 x 4096, x W^T), a streaming read of 4 GiB through torch's
    reduction and a 2 GiB device copy (read + write bytes), each the median of 10 timed calls."""
    import torch
    out = {}
    n = 8192
    a = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    for name, f in (("bf16_gemm_8192_xwT_tflops", lambda: a @ b.t()), ("bf16_gemm_8192_xw_tflops", lambda: a @ b)):
        for _ in range(3):
            f()
        us = _time(None, ev, stream, f, 10, None)
        out[name] = round(2 * n ** 3 / (float(np.median(us)) * 1e-6) / 1e12, 1)
    del a, b
    m, nn, k = 512, 28672, 4096
    a = torch.randn(m, k, device="cuda").to(torch.bfloat16)
    b = torch.randn(nn, k, device="cuda").to(torch.bfloat16)
    for _ in range(3):
        a @ b.t()
    us = _time(None, ev, stream, lambda: a @ b.t(), 10, None)
    out["bf16_gemm_mixtral_expert_xwT_tflops"] = round(2 * m * nn * k / (float(np.median(us)) * 1e-6) / 1e12, 1)
    del a, b
    big = torch.ones(1 << 30, dtype=torch.float32, device="cuda")  # 4 GiB
    for _ in range(2):
        big.sum()
    us = _time(None, ev, stream, lambda: big.sum(), 10, None)
    out["stream_read_4gib_gbs"] = round(big.numel() * 4 / (float(np.median(us)) * 1e-6) / 1e9, 1)
    half = big[: big.numel() // 2]
    dst = torch.empty_like(half)
    dst.copy_(half)
    us = _time(None, ev, stream, lambda: dst.copy_(half), 10, None)
    out["stream_copy_2gib_read_plus_write_gbs"] = round(2 * half.numel() * 4 / (float(np.median(us)) * 1e-6) / 1e9, 1)
    del big, half, dst
    torch.cuda.empty_cache()
    return out


def markdown_static(recs):
    rows = [r for r in recs if "static" in r]
    if not rows:
        return ""
    lines = ["", "| config | batch pool: µs cold / graph, touched, front µs | static pool: µs cold / graph, touched, "
             "front µs | front µs saved |", "|---|---|---|---|"]
    for r in rows:
        s = r["static"]
        lines.append(f"| {r['config']} | {r['us_cold']['median']} / {r['us_graph_warm_median']}, {r['experts_touched']}, "
                     f"{s['front_us_batch_pool']} | {s['us_cold_median']} / {s['us_graph_warm_median']}, "
                     f"{s['experts_touched']}, {s['front_us']} | {s['front_us_saved']} |")
    return "\n".join(lines) + "\n"


def markdown(recs):
    lines = ["| config | µs cold (p10–p90) | µs warm | µs graph | µs unfolded | 9 batches: median (8 more: min–max) | touched | "
             "rows max/mean | fold overhead | rate | % peak |", "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in recs:
        c = r["us_cold"]
        if "tflops" in r:
            rate, frac = f"{r['tflops']} TFLOP/s", f"{100 * r['frac_mfma_peak']:.1f}% MFMA"
        elif "hbm_gbs" in r:
            rate, frac = f"{r['hbm_gbs'] / 1000:.2f} TB/s", f"{100 * r['frac_hbm_peak']:.1f}% HBM"
        else:
            rate, frac = "—", "—"
        b = r["us_median_over_8_batches"]
        rp = r["rows_per_touched_expert"]
        lines.append(f"| {r['config']} | {c['median']} ({c['p10']}–{c['p90']}) | {r['us_warm_median']} | "
                     f"{r['us_graph_warm_median']} | {r['us_unfolded_cold_median']} | "
                     f"{r['us_median_over_9_batches']} ({b['min']}–{b['max']}) | {r['experts_touched']} | "
                     f"{rp['max']}/{rp['mean']} | {100 * r['fold_overhead_share']:.1f}% | {rate} | {frac} |")
    return "\n".join(lines) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--only", nargs="*", help="configuration names (default: all)")
    ap.add_argument("--reps-prefill", type=int, default=20)
    ap.add_argument("--reps-decode", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--md", help="also write a markdown table here")
    ap.add_argument("--ceilings", action="store_true",
                    help="also time a plain 8192^3 bf16 GEMM, a 4 GiB streaming read and a 2 GiB copy (context)")
    args = ap.parse_args(argv)

    import torch
    from . import exfold as X

    X.lib()  # fail loudly if the library is missing
    names = args.only or list(synth.WORKLOADS)
    unknown = [n for n in names if n not in synth.WORKLOADS]
    if unknown:
        sys.exit(f"unknown configurations: {unknown}")
    stream = torch.cuda.current_stream()
    ev = HipEvents()
    scratch = torch.empty(SCRATCH_BYTES // 4, dtype=torch.float32, device="cuda")
    recs = []
    if args.ceilings:
        print(json.dumps({"ceilings": ceilings(ev, stream)}), flush=True)
    # one layer per shape, configurations of a shape in a row
    by_shape = {}
    for n in names:
        by_shape.setdefault(synth.WORKLOADS[n].shape.name + str(synth.WORKLOADS[n].shape.router_bias), []).append(n)
    for group in by_shape.values():
        shape = synth.WORKLOADS[group[0]].shape
        layer, _, dev = make_layer(shape, seed=0)
        for n in group:
            rec = run_config(n, synth.WORKLOADS[n], layer, dev, args, ev, stream, scratch)
            print(json.dumps(rec), flush=True)
            recs.append(rec)
        del layer
        torch.cuda.empty_cache()
    ev.close()
    if args.md:
        with open(args.md, "w") as f:
            f.write(markdown(recs))
            f.write(markdown_static(recs))


if __name__ == "__main__":
    main()
