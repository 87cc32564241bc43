"""Parity at the full layer sizes, in the launch configuration the benchmark times.

Each case runs one folded forward of a full-size layer (Mixtral-, Qwen3- and
GLM-shaped) through the C-ABI with a caller workspace, then checks, against
the oracle:

* every router logit within the float32 rounding bound of its float64 value;
* Top-K ids (bit-exact) and softmax weights (one float32 ulp) recomputed from
  the device's logits;
* the keep mask / pool (dynamic, or static with its per-source tables), the folded ids and weights and the permutation,
  bit-exact, recomputed from the device's routes;
* the oracle's own routing from x (float64 logits) on every token: equal
  except at a near-tie of the logits;
* y of every token, per-token rel-L2 within the bf16 tolerance, from the
  device's folded routes.

The Qwen3-shaped layer is also calibrated on the device (4096 co-routed
tokens, lambda 1e-3, clip 4) and checked against the oracle's calibration;
its prefill and decode forwards then fold with those calibrated tables.
"""

import numpy as np
import pytest
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import DEV, TOL_Y, LayerPair, from_dev, logits_bound, per_token_rel_l2, sync, to_dev, topk_near_tie

pytestmark = pytest.mark.gpu

_LAYERS = {}


def _layer(shape):
    """One seeded full-size layer per shape for the whole module (weights are GBs)."""
    if shape.name not in _LAYERS or _LAYERS[shape.name].shape is not shape:
        _LAYERS.clear()
        torch.cuda.empty_cache()
        _LAYERS[shape.name] = LayerPair(shape, seed=0, lazy_oracle=True)
    return _LAYERS[shape.name]


def _check(shape, T, phase, budget, seed, tables=None):
    lp = _layer(shape)
    N, K = shape.n_experts, shape.top_k
    print(f"full size: {shape.name} {phase} T={T} budget={budget} seed={seed}", flush=True)
    xs = synth.tokens(shape, T, seed=seed)
    S, L, h = synth.synthetic_tables(N, seed=seed) if tables is None else tables
    x = to_dev(xs)
    ws = torch.empty(X.moe_workspace_size(lp.dev, T, phase, budget), dtype=torch.uint8, device=DEV)
    dbg = X.debug_buffers(lp.dev, T, phase, budget, DEV)
    if phase == "decode_static":
        # the static pool and its per-source tables on the device, bit-exact against the oracle's
        pool, psize, tgt, scl = X.static_pool(to_dev(h), budget, to_dev(S), to_dev(L))
        sync()
        s_pool = O.select_static_pool(h, budget)
        assert int(psize.item()) == len(s_pool) and pool.cpu().numpy().tolist() == s_pool
        rt, rs = O.decode_tables(s_pool, S, L, N)
        np.testing.assert_array_equal(tgt.cpu().numpy(), rt)
        np.testing.assert_array_equal(scl.cpu().numpy().view(np.uint32), rs.view(np.uint32))
        y = X.moe_forward(lp.dev, x, phase, budget, debug=dbg, workspace=ws, static_tables=(tgt, scl))
    else:
        y = X.moe_forward(lp.dev, x, phase, budget, to_dev(S), to_dev(L), to_dev(h), debug=dbg, workspace=ws)
    sync()
    g = {k: v.cpu().numpy() for k, v in dbg.items()}
    y = from_dev(y)

    # router logits: every entry within the float32 rounding bound
    xf = synth.widen(xs)
    ref_logits = O.router_logits(xf, lp.ref.w_router, lp.ref.router_bias)
    bound = logits_bound(xf, lp.ref.w_router, lp.ref.router_bias, shape.d)
    assert np.all(np.abs(g["logits"].astype(np.float64) - ref_logits) <= bound)

    # Top-K and softmax from the device's logits
    r_ids, r_w = O.route(g["logits"], K)
    np.testing.assert_array_equal(g["topk_ids"], r_ids)
    np.testing.assert_allclose(g["topk_w"], r_w, rtol=2 ** -22, atol=0)

    # selection and fold from the device's routes: bit-exact
    ids, w = g["topk_ids"], g["topk_w"]
    if phase == "prefill":
        keep = O.select_prefill(ids, w, h, budget)
        np.testing.assert_array_equal(g["keep"].astype(bool), keep)
        f_ids, f_w = O.fold_prefill(ids, w, keep, S, L)
        k_out = min(budget, K)
    elif phase == "decode_static":
        f_ids, f_w, _, _ = O.fold_decode(ids, w, s_pool, S, L, N)
        assert set(np.unique(g["fold_ids"]).tolist()) <= set(s_pool)
        k_out = K
    else:
        pool, cand = O.select_decode_pool(ids, w, h, N, budget)
        n = int(g["pool_size"][0])
        assert n == len(pool) == min(budget, len(cand))
        assert g["pool"][:n].tolist() == pool
        f_ids, f_w, _, _ = O.fold_decode(ids, w, pool, S, L, N)
        assert len(np.unique(g["fold_ids"])) <= budget
        k_out = K
    np.testing.assert_array_equal(g["fold_ids"], f_ids)
    np.testing.assert_array_equal(g["fold_w"].view(np.uint32), f_w.view(np.uint32))

    # permutation of the executed routes
    _, offsets, row_slot = O.permute_routes(g["fold_ids"], N)
    np.testing.assert_array_equal(g["offsets"][: N + 1], offsets)
    np.testing.assert_array_equal(g["row_slot"][: T * k_out], row_slot)

    # the oracle's own routing from x on every token: equal except at near-ties
    tie = topk_near_tie(ref_logits, bound, K)
    o_ids, _ = O.route(ref_logits, K)
    same = np.all(o_ids == ids, axis=1)
    assert np.all(same | tie), "routing differs from the oracle away from a near-tie"

    # y of every token from the device's folded routes
    y_ref = O.moe_output(lp.ref, xf, g["fold_ids"], g["fold_w"])
    err = per_token_rel_l2(y, y_ref)
    assert err.max() <= TOL_Y[shape.dtype], (err.max(), int(np.argmax(err)))
    assert np.isfinite(y).all()
    print(f"{shape.name} {phase} T={T} budget={budget}: max rel-L2 {err.max():.2e} over all {T} tokens, "
          f"routes differing from the oracle's own {int((~same).sum())} (within the rounding bound of a "
          f"tie: {int(tie.sum())})", flush=True)
    return g


def test_mixtral_prefill_4096_kp1():
    _check(synth.MIXTRAL, 4096, "prefill", 1, seed=0)


def test_mixtral_decode_32_d4():
    g = _check(synth.MIXTRAL, 32, "decode", 4, seed=1)
    assert int(g["pool_size"][0]) == 4


def test_qwen3_prefill_8192_kp4_skewed():
    g = _check(synth.QWEN3, 8192, "prefill", 4, seed=0)
    load = np.bincount(g["fold_ids"].reshape(-1), minlength=synth.QWEN3.n_experts)
    assert load.max() > 2 * load.mean(), "the biased router should give an imbalanced load"


@pytest.mark.parametrize("B", [16, 64, 256])
@pytest.mark.parametrize("D", [32, 64])
def test_glm_decode(B, D):
    _check(synth.GLM45, B, "decode", D, seed=B + D)


# (128, 16), (256, 32): 128x128 tiles for both projections; (512, 16), (512, 32): wide tiles for both
@pytest.mark.parametrize("B,D", [(1, 16), (8, 16), (64, 16), (128, 16), (512, 16), (128, 32), (256, 32), (512, 32),
                                 (1, 64), (64, 64), (512, 64)])
def test_qwen3_decode_sweep(B, D):
    _check(synth.QWEN3_DECODE, B, "decode", D, seed=3 * B + D)


@pytest.mark.parametrize("shape,B,D", [(synth.QWEN3_DECODE, 128, 16), (synth.QWEN3_DECODE, 1, 64),
                                       (synth.GLM45, 64, 32), (synth.MIXTRAL, 32, 4)])
def test_static_decode(shape, B, D):
    """Static decode pool (TopK of the norm proxy, tables precomputed once) at the full sizes."""
    _check(shape, B, "decode_static", D, seed=5 * B + D)


CAL_TOL = 1e-2   # bf16 expert outputs: H rounded to bf16 before the down projection


def test_qwen3_calibration_then_fold_with_calibrated_tables():
    """Calibration at the Qwen3-shaped configuration (d=2048, 128 experts, top-8, I=768, skewed
    router; 4096 co-routed calibration tokens, lambda 1e-3, clip 4) against the oracle, then a
    prefill (8192 tokens, K'=4) and a decode (128 tokens, D=16) forward folding with the device's
    calibrated tables, checked like the other full-size cases."""
    shape = synth.QWEN3
    lp = _layer(shape)
    N, K, m = shape.n_experts, shape.top_k, 4096
    print(f"calibration: {shape.name} m={m}", flush=True)
    xc = synth.calibration_tokens(shape, m, seed=0)
    xcd = to_dev(xc)
    # the device's router logits of the calibration tokens (the kernels calibration routes with)
    # feed the oracle's routing, so both sides evaluate the same expert pairs
    dbg = X.debug_buffers(lp.dev, m, "dense", 0, DEV)
    X.moe_forward(lp.dev, xcd, "dense", 0, debug=dbg)
    S, L, h, st = X.calibrate_projectors(lp.dev, xcd, lam=1e-3, clip=4.0, mode="corouted", with_stats=True)
    sync()
    g_logits = dbg["logits"].cpu().numpy()
    xf = synth.widen(xc)
    bound = logits_bound(xf, lp.ref.w_router, lp.ref.router_bias, shape.d)
    ref_logits = O.router_logits(xf, lp.ref.w_router, lp.ref.router_bias)
    assert np.all(np.abs(g_logits.astype(np.float64) - ref_logits) <= bound)
    rS, rL, rh, rst = O.calibrate(lp.ref, xf, K, lam=1e-3, clip=4.0, mode="corouted", logits=g_logits)
    st = st.cpu().numpy()
    np.testing.assert_array_equal(st[..., 3], rst["n"])
    obs = rst["n"] > 0
    assert obs.sum() > N * (N - 1) // 4, "too few co-routed pairs for a meaningful check"
    np.testing.assert_allclose(st[..., 0][obs], rst["A"][obs], rtol=CAL_TOL, atol=CAL_TOL * np.abs(rst["A"]).max())
    np.testing.assert_allclose(st[..., 1][obs], rst["V"][obs], rtol=CAL_TOL)
    np.testing.assert_allclose(st[..., 2][obs], rst["C"][obs], rtol=CAL_TOL)
    Sg, Lg, hg = S.cpu().numpy(), L.cpu().numpy(), h.cpu().numpy()
    np.testing.assert_allclose(Sg, rS, rtol=CAL_TOL, atol=CAL_TOL * max(1.0, np.abs(rS).max()))
    np.testing.assert_array_equal(Lg[~obs], rL[~obs])
    np.testing.assert_allclose(Lg[obs], rL[obs], rtol=CAL_TOL, atol=CAL_TOL)
    np.testing.assert_allclose(hg, rh, rtol=CAL_TOL)
    print(f"calibration: {int(obs.sum())} observed pairs, max |S| {np.abs(Sg[obs]).max():.3f}, "
          f"max S error {np.abs(Sg - rS).max():.2e}, max rel h error {np.abs(hg / rh - 1).max():.2e}", flush=True)
    tables = (Sg, Lg, hg)
    _check(shape, 8192, "prefill", 4, seed=5, tables=tables)
    _check(shape, 128, "decode", 16, seed=6, tables=tables)
