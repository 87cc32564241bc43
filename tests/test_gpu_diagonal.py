"""Diagonal projectors on the GPU (Appendix B, Eq. appendix_diagonal_projector;
the unfused reconstruction path): calibration of the per-dimension maps and
their loss, and the prefill forward that applies them element-wise."""

import numpy as np
import pytest
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import DEV, TOL_Y, LayerPair, from_dev, per_token_rel_l2, sync, to_dev

pytestmark = pytest.mark.gpu

SMALL_F32 = synth.LayerShape("diag-f32", d=128, inter=64, n_experts=8, top_k=3, dtype="f32")
SMALL_BF16 = synth.LayerShape("diag-bf16", d=256, inter=128, n_experts=16, top_k=4, dtype="bf16",
                              router_bias=True)
SHARED_BF16 = synth.LayerShape("diag-shared", d=128, inter=64, n_experts=12, top_k=4, shared_inter=64,
                               dtype="bf16")


@pytest.mark.parametrize("shape,m,mode,lam", [(SMALL_F32, 200, "corouted", 1e-3), (SMALL_F32, 64, "common", 0.1),
                                              (SMALL_BF16, 300, "corouted", 1e-3), (SMALL_BF16, 1, "corouted", 1e-3)])
def test_diagonal_calibration_matches_oracle(shape, m, mode, lam):
    lp = LayerPair(shape, seed=21)
    xs = synth.calibration_tokens(shape, m, seed=21)
    Dg, Ld = X.calibrate_diagonal(lp.dev, to_dev(xs), lam=lam, mode=mode)
    sync()
    Dg, Ld = Dg.cpu().numpy(), Ld.cpu().numpy()
    # the oracle on the device's routes (the router's float32 logits decide them)
    S_, L_, h_, st = O.calibrate(lp.ref, synth.widen(xs), shape.top_k, lam=lam, clip=0.0, mode=mode)
    rD, rL, rst = O.calibrate_diagonal(lp.ref, synth.widen(xs), shape.top_k, lam=lam, mode=mode)
    obs = rst["n"] > 0
    N = shape.n_experts
    eye = np.eye(N, dtype=bool)
    assert np.all(Dg[eye] == 1.0) and np.all(Ld[eye] == 0.0)
    assert np.all(Ld[~obs & ~eye] == np.float32(1e30)) and np.all(Dg[~obs & ~eye] == 0.0)
    tol = 1e-4 if shape.dtype == "f32" else 2e-2
    sel = obs & ~eye
    scale = np.abs(rD[sel]).max()
    np.testing.assert_allclose(Dg[sel], rD[sel], rtol=tol, atol=tol * max(1.0, scale))
    np.testing.assert_allclose(Ld[sel], rL[sel], rtol=tol, atol=tol)


@pytest.mark.parametrize("shape,T,kp", [(SMALL_F32, 64, 1), (SMALL_BF16, 200, 2), (SHARED_BF16, 77, 2),
                                        (SMALL_BF16, 1, 3)])
def test_diagonal_forward_matches_oracle(shape, T, kp):
    lp = LayerPair(shape, seed=22)
    Dg, Ld = X.calibrate_diagonal(lp.dev, to_dev(synth.calibration_tokens(shape, 256, seed=22)))
    _, _, h = synth.synthetic_tables(shape.n_experts, seed=22)
    xs = synth.tokens(shape, T, seed=23)
    dbg = X.debug_buffers(lp.dev, T, "prefill", kp, DEV)
    y = X.moe_forward(lp.dev, to_dev(xs), "prefill_diag", kp, None, Ld, to_dev(h), debug=dbg, diag=Dg)
    sync()
    ids, w = dbg["topk_ids"].cpu().numpy(), dbg["topk_w"].cpu().numpy()
    keep = O.select_prefill(ids, w, h, kp)
    np.testing.assert_array_equal(dbg["keep"].cpu().numpy().astype(bool), keep)
    oi, ow, folds = O.fold_prefill_diagonal(ids, w, keep, Ld.cpu().numpy())
    np.testing.assert_array_equal(dbg["fold_ids"].cpu().numpy(), oi)
    ref = O.diagonal_output(lp.ref, synth.widen(xs), oi, ow, folds, Dg.cpu().numpy())
    err = per_token_rel_l2(from_dev(y), ref)
    assert err.max() <= TOL_Y[shape.dtype], err.max()


def test_diagonal_fold_reproduces_per_dimension_multiples():
    # experts 4..7 copy gate/up of experts 0..3 and scale their down projection per
    # hidden dimension by powers of two: the calibrated diagonal maps (lambda = 0)
    # fold them exactly, so the folded layer matches the dense one
    shape = synth.LayerShape("diag-twins", d=128, inter=64, n_experts=8, top_k=2, dtype="f32")
    lp = LayerPair(shape, seed=24)
    rng = np.random.default_rng(24)
    gu = lp.dev.w_gate_up.clone()
    dn = lp.dev.w_down.clone()
    for j in range(4):
        c = torch.tensor(2.0 ** rng.integers(-1, 2, size=shape.d), dtype=torch.float32, device=DEV)
        gu[4 + j] = gu[j]
        dn[4 + j] = dn[j] * c[:, None]
    # routes: every token on one of (j, 4 + j) pairs, made certain by the router
    wr = torch.zeros_like(lp.dev.w_router)
    layer = X.Layer(w_router=wr, w_gate_up=gu, w_down=dn, top_k=2)
    x = to_dev(synth.tokens(shape, 96, seed=25))
    bias = torch.full((8,), -10.0, device=DEV)
    ys = []
    for j in range(4):
        b = bias.clone()
        b[j], b[4 + j] = 1.0, 0.5
        lj = X.Layer(w_router=wr, w_gate_up=gu, w_down=dn, top_k=2, router_bias=b)
        Dg, Ld = X.calibrate_diagonal(lj, x, lam=0.0, mode="common")
        h = torch.ones(8, device=DEV)
        y0 = X.moe_forward(lj, x, "dense", 0)
        yd = X.moe_forward(lj, x, "prefill_diag", 1, None, Ld, h, diag=Dg)
        ys.append((y0, yd))
    sync()
    for y0, yd in ys:
        err = per_token_rel_l2(from_dev(yd), from_dev(y0).astype(np.float64))
        assert err.max() <= 1e-4, err.max()
