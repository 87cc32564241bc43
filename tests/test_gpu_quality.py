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


def test_stack_matches_oracle_layer_by_layer():
    """The stacked demo against the oracle, layer by layer: each layer is calibrated on the same
    dense-stream input bytes by the device and by the oracle (pair counts bit-exact, S, L and h
    within 1e-2), then dense, direct and ExFold run on the device and in the oracle with the
    device's tables; every token's output agrees within the bf16 tolerance, and so do the demo's
    per-layer errors of direct and ExFold against dense."""
    from oracle import exfold_oracle as O

    from .gpu_common import DEV, from_dev, per_token_rel_l2

    sigma, seed, K = 0.3, 11, SHAPE.top_k
    layers, refs = [], []
    for l in range(2):
        gu, dn = synth.aligned_expert_weights(SHAPE, seed + l, sigma, 3.0)
        wr = synth.router_weight(SHAPE, seed + l)
        layers.append(X.Layer(w_router=to_dev(wr), w_gate_up=to_dev(gu), w_down=to_dev(dn), top_k=K))
        refs.append(O.Layer(w_router=synth.widen(wr), w_gate_up=synth.widen(gu), w_down=synth.widen(dn)))

    def logits_of(layer, x):
        dbg = X.debug_buffers(layer, x.shape[0], "dense", 0, DEV)
        X.moe_forward(layer, x, "dense", 0, debug=dbg)
        return dbg["logits"].cpu().numpy()

    h_cal = to_dev(synth.calibration_tokens(SHAPE, 2048, seed))
    tables = Q.calibrate_stack(layers, h_cal)
    # the calibration inputs along the dense stream, as calibrate_stack forms them
    cal_in = [h_cal]
    for layer in layers[:-1]:
        cal_in.append((cal_in[-1].float() + X.moe_forward(layer, cal_in[-1], "dense").float()).to(h_cal.dtype))
    for l, (layer, ref, tab, xin) in enumerate(zip(layers, refs, tables, cal_in)):
        S, L, h = (t.cpu().numpy() for t in tab)
        rS, rL, rh, rst = O.calibrate(ref, from_dev(xin), K, logits=logits_of(layer, xin))
        obs = rst["n"] > 0
        np.testing.assert_allclose(S, rS, rtol=1e-2, atol=1e-2 * max(1.0, np.abs(rS).max()))
        np.testing.assert_array_equal(L[~obs], rL[~obs])
        np.testing.assert_allclose(L[obs], rL[obs], rtol=1e-2, atol=1e-2)
        np.testing.assert_allclose(h, rh, rtol=1e-2)
        assert np.abs(S[obs]).max() > 0.5, "aligned experts should calibrate large scalars"

    xp = to_dev(synth.tokens(SHAPE, 256, 11))
    xd = to_dev(synth.tokens(SHAPE, 64, 12))
    for x, phase, budget in ((xp, "prefill", 4), (xd, "decode", 8)):
        demo = Q.evaluate(layers, tables, x, phase, budget)
        s_in = x
        for l, (layer, ref, tab) in enumerate(zip(layers, refs, tables)):
            S, L, h = (t.cpu().numpy() for t in tab)
            xl = from_dev(s_in)
            lg = logits_of(layer, s_in)
            y_dev, y_ref = {}, {}
            for m in ("dense", "direct", "exfold"):
                y_dev[m] = from_dev(Q._layer(layer, tab, s_in, m, phase, budget))
                if m == "dense":
                    y_ref[m] = O.moe_forward(ref, xl, K, "dense", 0, logits=lg)[0]
                else:
                    Sm = np.zeros_like(S) if m == "direct" else S
                    y_ref[m] = O.moe_forward(ref, xl, K, phase, budget, Sm, L, h, logits=lg)[0]
                err = per_token_rel_l2(y_dev[m], y_ref[m])
                assert err.max() <= 2e-2, (phase, l, m, err.max())
            for m in ("direct", "exfold"):
                e_ref = per_token_rel_l2(y_ref[m], y_ref["dense"]).mean()
                e_demo = demo[m]["per_layer"][l]["mean"]
                print(f"{phase} layer {l} {m}: demo {e_demo:.4f} oracle {e_ref:.4f}", flush=True)
                assert abs(e_demo - e_ref) <= 0.01 + 0.02 * e_ref, (phase, l, m, e_demo, e_ref)
            s_in = (s_in.float() + Q._layer(layer, tab, s_in, "dense", phase, budget).float()).to(x.dtype)
