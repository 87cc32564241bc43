"""Parity at the full layer sizes, in the launch configuration the benchmark times.

Each case runs one folded forward of a full-size layer (Mixtral-, Qwen3- and
GLM-shaped) through the C-ABI with a caller workspace, then checks, against
the oracle:

* every router logit within the float32 rounding bound of its float64 value;
* Top-K ids (bit-exact) and softmax weights (one float32 ulp) recomputed from
  the device's logits;
* the keep mask / pool, the folded ids and weights and the permutation,
  bit-exact, recomputed from the device's routes;
* the oracle's own routing from x (float64 logits) on a token sample: equal
  except at a near-tie of the logits;
* y of a token sample (all tokens for small decode batches), per-token
  rel-L2 within the bf16 tolerance, from the device's folded routes.
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


def _sample(T, n, rng):
    if T <= n:
        return np.arange(T)
    mid = rng.choice(np.arange(1, T - 1), size=n - 2, replace=False)
    return np.sort(np.concatenate([[0, T - 1], mid]))


def _check(shape, T, phase, budget, seed, n_sample):
    lp = _layer(shape)
    N, K = shape.n_experts, shape.top_k
    xs = synth.tokens(shape, T, seed=seed)
    S, L, h = synth.synthetic_tables(N, seed=seed)
    x = to_dev(xs)
    ws = torch.empty(X.moe_workspace_size(lp.dev, T, phase, budget), dtype=torch.uint8, device=DEV)
    dbg = X.debug_buffers(lp.dev, T, phase, budget, DEV)
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

    rng = np.random.default_rng(seed)
    smp = _sample(T, n_sample, rng)
    # the oracle's own routing from x on the sample: equal except at near-ties
    tie = topk_near_tie(ref_logits[smp], bound[smp], K)
    o_ids, _ = O.route(ref_logits[smp], K)
    same = np.all(o_ids == ids[smp], axis=1)
    assert np.all(same | tie), "routing differs from the oracle away from a near-tie"

    # y of the sampled tokens from the device's folded routes
    y_ref = O.moe_output(lp.ref, xf[smp], g["fold_ids"][smp], g["fold_w"][smp])
    err = per_token_rel_l2(y[smp], y_ref)
    assert err.max() <= TOL_Y[shape.dtype], (err.max(), smp[np.argmax(err)])
    print(f"{shape.name} {phase} T={T} budget={budget}: max rel-L2 {err.max():.2e} over {len(smp)} tokens, "
          f"routes differing from the oracle's own {int((~same).sum())} (within the rounding bound of a "
          f"tie: {int(tie.sum())})", flush=True)
    return g


def test_mixtral_prefill_4096_kp1():
    _check(synth.MIXTRAL, 4096, "prefill", 1, seed=0, n_sample=48)


def test_mixtral_decode_32_d4():
    g = _check(synth.MIXTRAL, 32, "decode", 4, seed=1, n_sample=32)
    assert int(g["pool_size"][0]) == 4


def test_qwen3_prefill_8192_kp4_skewed():
    g = _check(synth.QWEN3, 8192, "prefill", 4, seed=0, n_sample=64)
    load = np.bincount(g["fold_ids"].reshape(-1), minlength=synth.QWEN3.n_experts)
    assert load.max() > 2 * load.mean(), "the biased router should give an imbalanced load"


@pytest.mark.parametrize("B", [16, 64, 256])
@pytest.mark.parametrize("D", [32, 64])
def test_glm_decode(B, D):
    _check(synth.GLM45, B, "decode", D, seed=B + D, n_sample=256)


@pytest.mark.parametrize("B,D", [(1, 16), (8, 16), (64, 16), (512, 16), (128, 32), (1, 64), (64, 64), (512, 64)])
def test_qwen3_decode_sweep(B, D):
    _check(synth.QWEN3_DECODE, B, "decode", D, seed=3 * B + D, n_sample=128)
