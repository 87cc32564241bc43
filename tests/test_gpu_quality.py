"""The synthetic quality demo: on directionally aligned experts, folding
through calibrated projectors recovers the omitted experts' contributions that
dropping them (Direct Top-K', pool-only decode) loses."""

import numpy as np
import pytest
import torch

from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import quality as Q
from paper_2608_24938_amd import synth

from .gpu_common import to_dev

pytestmark = pytest.mark.gpu

SHAPE = synth.LayerShape("quality-bf16", d=256, inter=128, n_experts=32, top_k=8, dtype="bf16", m_cal=2048)


def _stack(sigma, scales=None, n_layers=2, seed=11, lam=1e-3):
    layers = []
    for l in range(n_layers):
        gu, dn = synth.aligned_expert_weights(SHAPE, seed + l, sigma, 3.0, scales=scales)
        layers.append(X.Layer(w_router=to_dev(synth.router_weight(SHAPE, seed + l)), w_gate_up=to_dev(gu),
                              w_down=to_dev(dn), top_k=SHAPE.top_k))
    tables = Q.calibrate_stack(layers, to_dev(synth.calibration_tokens(SHAPE, 2048, seed)), lam=lam)
    return layers, tables


@pytest.mark.parametrize("sigma", [0.1, 0.3])
def test_folding_beats_dropping_on_aligned_experts(sigma):
    layers, tables = _stack(sigma)
    xp = to_dev(synth.tokens(SHAPE, 256, 11))
    xd = to_dev(synth.tokens(SHAPE, 64, 12))
    for x, phase, budget in ((xp, "prefill", 4), (xd, "decode", 8)):
        r = Q.evaluate(layers, tables, x, phase, budget)
        direct, exfold = r["direct"]["stack"]["mean"], r["exfold"]["stack"]["mean"]
        print(phase, sigma, "direct", round(direct, 4), "exfold", round(exfold, 4), flush=True)
        assert direct > 0.05                      # the budget really drops mass
        assert exfold < 0.5 * direct, (phase, direct, exfold)
        for d_, e_ in zip(r["direct"]["per_layer"], r["exfold"]["per_layer"]):
            assert e_["mean"] < d_["mean"]


def test_exact_multiples_fold_to_the_full_output():
    # sigma = 0 and power-of-two scales: every expert output is an exact multiple
    # of the base expert's, so lambda = 0 calibrates exact scalars and folding
    # reproduces the dense layer up to the bf16 rounding of H and y
    scales = np.array([0.5, 1.0, 2.0, 1.0] * (SHAPE.n_experts // 4))
    layers, tables = _stack(0.0, scales=scales, n_layers=1, lam=0.0)
    x = to_dev(synth.tokens(SHAPE, 128, 13))
    for phase, budget in (("prefill", 2), ("decode", 4)):
        r = Q.evaluate(layers, tables, x, phase, budget)
        assert r["exfold"]["stack"]["max"] <= 2e-2, (phase, r["exfold"]["stack"])
        assert r["direct"]["stack"]["mean"] > 0.1
