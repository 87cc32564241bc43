"""Synthetic quality demo of expert folding on a stack of MoE layers.

Layers with directionally aligned experts (synth.aligned_expert_weights) are
calibrated on the GPU (exfold_calibrate_projectors, layer by layer on the
dense residual stream of the calibration tokens), then run three ways on the
same tokens, every layer through libexfold:

* dense:   the unfolded layer on the router's Top-K routes;
* direct:  the same budget with every omitted route dropped (S = 0: Direct
           Top-K' in prefill, pool-only routes in decode);
* exfold:  the same budget with omitted routes folded through the calibrated
           scalar projectors (prefill: Eq. prefill_fold; decode: Eq. decode_remap).

Reported, per phase: the relative L2 error of each layer's output against the
dense layer on the dense stream's input (per-layer error), and of the stack's
total MoE contribution sum_l y_l after each method ran on its own stream
(accumulated error), each as the mean and max over tokens.  The residual
stream h_{l+1} = h_l + y_l is the harness around the layer (plain torch).

    python -m paper_2608_24938_amd.quality [--layers 4] [--sigma 0.3] ...
"""

from __future__ import annotations

import argparse
import json

import torch

from . import exfold as X
from . import synth


def _dev(a):
    import numpy as np
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(a).to("cuda")


def make_layers(shape, n_layers, seed, sigma, spread):
    layers = []
    for l in range(n_layers):
        gu, dn = synth.aligned_expert_weights(shape, seed + l, sigma, spread)
        layers.append(X.Layer(w_router=_dev(synth.router_weight(shape, seed + l)), w_gate_up=_dev(gu),
                              w_down=_dev(dn), top_k=shape.top_k,
                              router_bias=_dev(synth.router_bias(shape, seed + l))))
    return layers


def calibrate_stack(layers, x_cal, lam=1e-3, clip=4.0):
    """(S, L, h) of every layer, calibrated on its input along the dense stream."""
    tables = []
    h = x_cal
    for layer in layers:
        tables.append(X.calibrate_projectors(layer, h, lam=lam, clip=clip))
        h = (h.float() + X.moe_forward(layer, h, "dense").float()).to(h.dtype)
    return tables


def _layer(layer, tab, x, method, phase, budget):
    if method == "dense":
        return X.moe_forward(layer, x, "dense")
    S, L, h = tab
    if method == "direct":
        S = torch.zeros_like(S)
    return X.moe_forward(layer, x, phase, budget, S, L, h)


def _rel(a, b):
    a, b = a.double(), b.double()
    e = (a - b).norm(dim=1) / b.norm(dim=1).clamp_min(1e-30)
    return {"mean": float(e.mean()), "max": float(e.max())}


def evaluate(layers, tables, x, phase, budget):
    """Per-layer and accumulated errors of direct and exfold against dense."""
    out = {}
    streams = {m: x for m in ("dense", "direct", "exfold")}
    contrib = {m: torch.zeros_like(x, dtype=torch.float32) for m in streams}
    per_layer = {"direct": [], "exfold": []}
    for layer, tab in zip(layers, tables):
        y_ref = _layer(layer, tab, streams["dense"], "dense", phase, budget)
        for m in ("direct", "exfold"):
            per_layer[m].append(_rel(_layer(layer, tab, streams["dense"], m, phase, budget).float(),
                                     y_ref.float()))
        for m in streams:
            y = y_ref if m == "dense" else _layer(layer, tab, streams[m], m, phase, budget)
            contrib[m] += y.float()
            streams[m] = (streams[m].float() + y.float()).to(x.dtype)
    for m in ("direct", "exfold"):
        out[m] = {"per_layer": per_layer[m], "stack": _rel(contrib[m], contrib["dense"])}
    return out


def run(shape=synth.QWEN3, n_layers=4, seed=0, sigma=0.3, spread=3.0, t_prefill=512, k_pre=4,
        b_decode=64, d_pool=64, m_cal=4096):
    layers = make_layers(shape, n_layers, seed, sigma, spread)
    x_cal = _dev(synth.calibration_tokens(shape, m_cal, seed))
    tables = calibrate_stack(layers, x_cal)
    xp = _dev(synth.tokens(shape, t_prefill, seed))
    xd = _dev(synth.tokens(shape, b_decode, seed + 1))
    return {
        "workload": f"{n_layers} stacked {shape.name}-shaped layers (d={shape.d}, N={shape.n_experts}, "
                    f"K={shape.top_k}, I={shape.inter}), aligned experts sigma={sigma}, scale spread {spread}x, "
                    f"calibrated on {m_cal} tokens",
        "prefill": {"tokens": t_prefill, "k_pre": k_pre, **evaluate(layers, tables, xp, "prefill", k_pre)},
        "decode": {"tokens": b_decode, "pool": d_pool, **evaluate(layers, tables, xd, "decode", d_pool)},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--layers", type=int, default=4)
    ap.add_argument("--sigma", type=float, default=0.3)
    ap.add_argument("--spread", type=float, default=3.0)
    ap.add_argument("--prefill-tokens", type=int, default=512)
    ap.add_argument("--k-pre", type=int, default=4)
    ap.add_argument("--decode-tokens", type=int, default=64)
    ap.add_argument("--pool", type=int, default=64)
    ap.add_argument("--m-cal", type=int, default=4096)
    a = ap.parse_args()
    X.lib()
    print(json.dumps(run(n_layers=a.layers, sigma=a.sigma, spread=a.spread, t_prefill=a.prefill_tokens,
                         k_pre=a.k_pre, b_decode=a.decode_tokens, d_pool=a.pool, m_cal=a.m_cal)))


if __name__ == "__main__":
    main()
