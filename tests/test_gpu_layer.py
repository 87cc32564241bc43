"""Layer-level parity of the HIP path with the oracle: expert execution on
given routes, the full folded forward in every phase, the identity budgets,
exact-multiple folding, calibration and determinism."""

import numpy as np
import pytest
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import (DEV, TOL_Y, LayerPair, from_dev, logits_bound, per_token_rel_l2, sync, to_dev,
                         topk_near_tie)

pytestmark = pytest.mark.gpu

SMALL_BF16 = synth.LayerShape("small-bf16", d=256, inter=512, n_experts=8, top_k=2, dtype="bf16", m_cal=512)
WIDE_BF16 = synth.LayerShape("wide-bf16", d=256, inter=128, n_experts=128, top_k=8, dtype="bf16",
                             router_bias=True, m_cal=1024)
SHARED_BF16 = synth.LayerShape("shared-bf16", d=384, inter=192, n_experts=64, top_k=6, shared_inter=192,
                               dtype="bf16", m_cal=512)
WIDE_F32 = synth.LayerShape("wide-f32", d=128, inter=64, n_experts=64, top_k=8, dtype="f32", router_bias=True)
# few experts (bf16, <= 32): the router, Top-K and fold in one kernel, one workgroup a token
ROUTER24_BF16 = synth.LayerShape("router-24", d=512, inter=256, n_experts=24, top_k=4, dtype="bf16",
                                 router_bias=True)
ROUTER8_BF16 = synth.LayerShape("router-8", d=1024, inter=256, n_experts=8, top_k=2, dtype="bf16")
ROUTER48_BF16 = synth.LayerShape("router-48", d=768, inter=128, n_experts=48, top_k=4, dtype="bf16")
# the largest routing the library takes: 256 experts, top-16 (decode front end at its expert limit)
MAX_BF16 = synth.LayerShape("max-experts", d=128, inter=128, n_experts=256, top_k=16, dtype="bf16",
                            router_bias=True)
# 1024+ tokens and a multiple of 128 experts: the router as a plain tiled GEMM whose
# reduction is split in four (partial sums added in order by the Top-K kernel)
ROUTER_SPLIT_BF16 = synth.LayerShape("router-split", d=1024, inter=128, n_experts=128, top_k=8, dtype="bf16",
                                     router_bias=True)


@pytest.mark.parametrize("shape,T,k_out", [(synth.TINY, 64, 2), (synth.TINY, 1, 1), (SMALL_BF16, 200, 2),
                                           (WIDE_BF16, 300, 8), (SHARED_BF16, 77, 3), (WIDE_F32, 150, 5),
                                           (SMALL_BF16, 513, 1)])
def test_execute_matches_oracle(shape, T, k_out):
    lp = LayerPair(shape, seed=1)
    rng = np.random.default_rng(T)
    ids = rng.integers(0, shape.n_experts, size=(T, k_out)).astype(np.int32)   # duplicates allowed
    w = rng.standard_normal((T, k_out)).astype(np.float32)
    xs = synth.tokens(shape, T, seed=1)
    y = X.moe_execute(lp.dev, to_dev(xs), to_dev(ids), to_dev(w))
    sync()
    ref = O.moe_output(lp.ref, synth.widen(xs), ids, w)
    err = per_token_rel_l2(from_dev(y), ref)
    assert err.max() <= TOL_Y[shape.dtype], err.max()


def _forward_case(shape, T, phase, budget, seed=2):
    lp = LayerPair(shape, seed=seed)
    xs = synth.tokens(shape, T, seed=seed)
    S, L, h = synth.synthetic_tables(shape.n_experts, seed=seed)
    dbg = X.debug_buffers(lp.dev, T, phase, budget, DEV)
    y = X.moe_forward(lp.dev, to_dev(xs), phase, budget, to_dev(S), to_dev(L), to_dev(h), debug=dbg)
    sync()
    return lp, xs, (S, L, h), dbg, from_dev(y)


@pytest.mark.parametrize("shape,T,phase,budget", [
    (synth.TINY, 64, "prefill", 1), (synth.TINY, 64, "dense", 0), (synth.TINY, 64, "decode", 4),
    (SMALL_BF16, 300, "prefill", 1), (SMALL_BF16, 32, "decode", 4), (SMALL_BF16, 129, "dense", 0),
    (WIDE_BF16, 500, "prefill", 4), (WIDE_BF16, 64, "decode", 16), (WIDE_BF16, 256, "decode", 32),
    (SHARED_BF16, 100, "prefill", 2), (SHARED_BF16, 48, "decode", 8), (WIDE_F32, 90, "prefill", 3),
    (WIDE_F32, 33, "decode", 5),
    # 1024+ tokens: the router's many-token layouts (32 tokens a workgroup for
    # 33-127 experts, d in chunks of 256: three for the 48-expert shape; 128 x
    # 128 MFMA tiles for multiples of 128 experts), with a ragged last tile
    (SHARED_BF16, 1100, "prefill", 2), (WIDE_BF16, 1500, "prefill", 4), (SMALL_BF16, 1030, "prefill", 1),
    (ROUTER48_BF16, 1050, "prefill", 2), (ROUTER_SPLIT_BF16, 1100, "prefill", 3), (MAX_BF16, 1030, "prefill", 5),
    # small decode batches: Top-K and softmax inside the one-workgroup front end
    (synth.TINY, 16, "decode", 4), (WIDE_BF16, 16, "decode", 16), (WIDE_F32, 20, "decode", 5),
    (SHARED_BF16, 3, "decode", 8),
    # 256 experts, top-16: prefill fold, decode pools below and above the candidate count, dense
    (MAX_BF16, 90, "prefill", 5), (MAX_BF16, 24, "decode", 40), (MAX_BF16, 40, "decode", 256),
    (MAX_BF16, 33, "dense", 0),
    # route_small_kernel (router, Top-K and fold in one kernel) for few experts
    (ROUTER24_BF16, 21, "decode", 6), (ROUTER24_BF16, 1, "decode", 2), (ROUTER8_BF16, 64, "decode", 4),
    (ROUTER8_BF16, 37, "dense", 0), (ROUTER24_BF16, 90, "decode", 10), (ROUTER24_BF16, 300, "prefill", 2),
    # beyond 1024 tokens: one workgroup per 16 tokens (logits over all of d, then routing), ragged last block
    (ROUTER24_BF16, 1100, "prefill", 2), (ROUTER24_BF16, 1040, "decode", 10), (ROUTER8_BF16, 2050, "dense", 0),
])
def test_forward_matches_oracle(shape, T, phase, budget):
    lp, xs, (S, L, h), dbg, y = _forward_case(shape, T, phase, budget)
    N, K = shape.n_experts, shape.top_k
    x = synth.widen(xs)
    g = {k: v.cpu().numpy() for k, v in dbg.items()}
    # router logits within the float32 rounding bound
    ref_logits = O.router_logits(x, lp.ref.w_router, lp.ref.router_bias)
    bound = logits_bound(x, lp.ref.w_router, lp.ref.router_bias, shape.d)
    assert np.all(np.abs(g["logits"].astype(np.float64) - ref_logits) <= bound)

    # stage by stage from the device's own logits and routes: discrete results bit-exact
    ids, w = g["topk_ids"], g["topk_w"]
    r_ids, r_w = O.route(g["logits"], K)
    np.testing.assert_array_equal(ids, r_ids)
    np.testing.assert_allclose(w, r_w, rtol=2 ** -22, atol=0)
    if phase == "prefill":
        keep = O.select_prefill(ids, w, h, budget)
        np.testing.assert_array_equal(g["keep"].astype(bool), keep)
        f_ids, f_w = O.fold_prefill(ids, w, keep, S, L)
    elif phase == "decode":
        pool, _ = O.select_decode_pool(ids, w, h, N, budget)
        n = int(g["pool_size"][0])
        assert g["pool"][:n].tolist() == pool
        f_ids, f_w, _, _ = O.fold_decode(ids, w, pool, S, L, N)
    else:
        f_ids, f_w = ids, w
    ex_ids = g["fold_ids"] if phase != "dense" else ids
    ex_w = g["fold_w"] if phase != "dense" else w
    np.testing.assert_array_equal(ex_ids, f_ids)
    np.testing.assert_array_equal(ex_w.view(np.uint32), f_w.view(np.uint32))

    # end to end from x: the oracle's own float64 routing, selection and fold
    y_ref, info = O.moe_forward(lp.ref, x, K, phase, budget, S, L, h)
    tie = topk_near_tie(ref_logits, bound, K)
    same_routes = np.all(ids == info["topk_ids"], axis=1)
    assert np.all(same_routes | tie), "route mismatch away from a near-tie"
    same_exec = np.all(ex_ids == info["fold_ids"], axis=1)
    allowed = max(2, T // 50)
    if phase == "prefill":
        # equal routes, different selection: only where the oracle's scores w*h tie within
        # the one-ulp difference of the two softmax weights
        for i in np.nonzero(same_routes & ~same_exec)[0]:
            sc = np.sort(info["topk_w"][i].astype(np.float64) * h[info["topk_ids"][i]].astype(np.float64))[::-1]
            kp = min(budget, K)
            assert sc[kp - 1] - sc[kp] <= 1e-5 * sc[0], ("selection differs away from a near-tie", i)
    elif phase == "decode":
        g_pool = g["pool"][: int(g["pool_size"][0])].tolist()
        assert len(g_pool) == len(info["pool"])
        if g_pool != info["pool"]:
            # only a near-tie of the batch scores may change the pool: check the margin
            wr = info["topk_w"].astype(np.float64)
            score = np.zeros(N)
            np.add.at(score, info["topk_ids"].reshape(-1), wr.reshape(-1))
            score *= h.astype(np.float64)
            diff = sorted(set(g_pool) ^ set(info["pool"]))
            assert np.ptp(score[diff]) <= 1e-5 * score.max(), "pool differs away from a near-tie"
            allowed = T      # a changed pool moves every token routed to the experts that changed
    # every token's y: against the oracle's own output where the executed routes agree, and
    # against the oracle on the device's executed routes where a near-tie changed them
    y_cmp = y_ref.copy()
    moved = np.nonzero(~same_exec)[0]
    if moved.size:
        y_cmp[moved] = O.moe_output(lp.ref, x[moved], ex_ids[moved], ex_w[moved])
    err = per_token_rel_l2(y, y_cmp)
    assert err.max() <= TOL_Y[shape.dtype], (err.max(), int(np.argmax(err)))
    assert moved.size <= allowed, f"{moved.size} of {T} tokens left the oracle's routes"
    print(f"{shape.name} {phase} T={T}: max rel-L2 {err.max():.2e}, tokens on other routes {moved.size}",
          flush=True)


@pytest.mark.parametrize("shape,T,K_id,D_id", [(WIDE_F32, 64, 8, 64), (WIDE_BF16, 200, 8, 128),
                                              (SHARED_BF16, 60, 6, 64)])
def test_identity_budgets_are_bitwise_dense(shape, T, K_id, D_id):
    lp = LayerPair(shape, seed=4)
    xs = to_dev(synth.tokens(shape, T, seed=4))
    S, L, h = (to_dev(a) for a in synth.synthetic_tables(shape.n_experts, seed=4))
    y0 = X.moe_forward(lp.dev, xs, "dense", 0)
    yp = X.moe_forward(lp.dev, xs, "prefill", K_id, S, L, h)
    yp2 = X.moe_forward(lp.dev, xs, "prefill", K_id + 5, S, L, h)
    yd = X.moe_forward(lp.dev, xs, "decode", D_id, S, L, h)
    sync()
    bits = lambda y: y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32)
    for y in (yp, yp2, yd):
        assert torch.equal(bits(y), bits(y0))
    # |candidates| <= D < N: the routes are bitwise unchanged.  The expert GEMMs are planned on
    # the host before the pool exists, from the D busy experts a decode pool allows at most; where
    # that plan equals the dense one (the same kernels, splits and grids) y is bitwise dense, and
    # where it differs the down projection's sums may be split differently, so y agrees within
    # the tolerance
    for Tn in (3, 16):
        xn = xs[:Tn].contiguous()
        dbg0 = X.debug_buffers(lp.dev, Tn, "dense", 0, DEV)
        yn = X.moe_forward(lp.dev, xn, "dense", 0, debug=dbg0)
        sync()
        n_cand = len(np.unique(dbg0["topk_ids"].cpu().numpy()))
        D = n_cand if Tn == 16 else D_id - 1
        assert n_cand <= D < shape.n_experts
        dbg = X.debug_buffers(lp.dev, Tn, "decode", D, DEV)
        ydn = X.moe_forward(lp.dev, xn, "decode", D, S, L, h, debug=dbg)
        sync()
        assert int(dbg["pool_size"].item()) == n_cand
        assert torch.equal(dbg["fold_ids"], dbg["topk_ids"])
        assert torch.equal(dbg["fold_w"].view(torch.int32), dbg["topk_w"].view(torch.int32))
        rows, groups = Tn * shape.top_k, shape.n_experts
        same_plan = _plan(lp.dev, rows, min(D, rows)) == _plan(lp.dev, rows, min(groups, rows))
        print(f"{shape.name} T={Tn} D={D} (candidates {n_cand}): plans equal {same_plan}", flush=True)
        if same_plan:
            assert torch.equal(bits(ydn), bits(yn))
        else:
            err = per_token_rel_l2(from_dev(ydn), from_dev(yn).astype(np.float64))
            assert err.max() <= TOL_Y[shape.dtype]


def _plan(layer, rows, active):
    """The expert-GEMM plan of the library for `rows` rows and `active` busy groups."""
    import ctypes
    ls = layer.struct()
    out = (ctypes.c_int32 * 10)()
    shared = 1 if layer.ws_down is not None else 0
    cu = torch.cuda.get_device_properties(0).multi_processor_count
    assert X.lib().exfold_gemm_plan(ctypes.byref(ls), rows + shared * (rows // layer.top_k), active + shared,
                                    cu, out) == X.OK
    return list(out)


def _twin_layer(dtype, seed=5):
    """Experts 4+j copy gate/up of expert j and scale its down projection by c_j (a power of two);
    the router ranks every base expert just above its twin."""
    c = (0.5, -2.0, 2.0, -0.5)   # no c = -1: twin logits differ by 1e-4, so E_j - E_tw would cancel
    shape = synth.LayerShape("twin", d=256, inter=128, n_experts=8, top_k=2, dtype=dtype)
    lp = LayerPair(shape, seed=seed)
    gu, dn, wr = lp.storage["gu"].copy(), lp.storage["dn"].copy(), lp.storage["wr"].copy()
    gu[4:] = gu[:4]
    wr[4:] = wr[:4]
    scaled = synth.widen(dn[:4]) * np.array(c, np.float32)[:, None, None]
    dn[4:] = synth._bf16_bits_inplace(scaled.copy()) if dtype == "bf16" else scaled
    bias = np.array([0, 0, 0, 0, -1e-4, -1e-4, -1e-4, -1e-4], np.float32)
    dev = X.Layer(w_router=to_dev(wr), w_gate_up=to_dev(gu), w_down=to_dev(dn), top_k=2, router_bias=to_dev(bias))
    ref = O.Layer(w_router=synth.widen(wr), w_gate_up=synth.widen(gu), w_down=synth.widen(dn), router_bias=bias)
    return shape, dev, ref, c


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_exact_multiples_fold_reproduces_full_output(dtype):
    shape, dev, ref, c = _twin_layer(dtype)
    xc = to_dev(synth.calibration_tokens(shape, 256, seed=5))
    S, L, h = X.calibrate_projectors(dev, xc, lam=0.0, clip=4.0, mode="common")
    sync()
    S_, L_ = S.cpu().numpy(), L.cpu().numpy()
    for j, cj in enumerate(c):
        if dtype == "f32":
            # float32 experts: u = c v holds bit for bit, so s = c and l = 0 exactly
            assert S_[4 + j, j] == np.float32(cj) and S_[j, 4 + j] == np.float32(1.0 / cj)
            assert L_[4 + j, j] == 0.0 and L_[j, 4 + j] == 0.0
        else:
            # bf16 MFMA products: the scaled twin agrees to the last float32 bits
            assert abs(S_[4 + j, j] - cj) <= 1e-6 * abs(cj) and abs(S_[j, 4 + j] - 1 / cj) <= 1e-6 / abs(cj)
            assert L_[4 + j, j] <= 1e-6 and L_[j, 4 + j] <= 1e-6
    T = 96
    xs = synth.tokens(shape, T, seed=6)
    x = to_dev(xs)
    y_full = O.moe_forward(ref, synth.widen(xs), 2, "dense", 0)[0]
    dbg = X.debug_buffers(dev, T, "prefill", 1, DEV)
    yp = X.moe_forward(dev, x, "prefill", 1, S, L, h, debug=dbg)
    hd = to_dev(np.array([10, 10, 10, 10, 1, 1, 1, 1], np.float32))
    dbgd = X.debug_buffers(dev, T, "decode", 4, DEV)
    yd = X.moe_forward(dev, x, "decode", 4, S, L, hd, debug=dbgd)
    sync()
    ids = dbg["topk_ids"].cpu().numpy()
    twin = (ids[:, 0] % 4) == (ids[:, 1] % 4)
    assert twin.mean() > 0.95
    assert sorted(dbgd["pool"].cpu().numpy().tolist()) == [0, 1, 2, 3]
    for y in (yp, yd):
        err = per_token_rel_l2(from_dev(y), y_full)[twin]
        assert err.max() <= TOL_Y[dtype], err.max()


# 4096 calibration tokens x 2 routes: both GEMMs on the wide tiles, the per-row
# outputs kept in float32 for the statistics
CAL_WIDE = synth.LayerShape("cal-wide", d=2048, inter=512, n_experts=8, top_k=2, dtype="bf16")


@pytest.mark.parametrize("shape,m,mode,lam,clip", [(synth.TINY, 512, "corouted", 1e-3, 4.0),
                                                   (synth.TINY, 200, "common", 1e-3, 0.0),
                                                   (WIDE_F32, 300, "corouted", 1e-2, 4.0),
                                                   (SMALL_BF16, 512, "corouted", 1e-3, 4.0),
                                                   (CAL_WIDE, 4096, "corouted", 1e-3, 4.0)])
def test_calibration_matches_oracle(shape, m, mode, lam, clip):
    lp = LayerPair(shape, seed=7)
    xs = synth.calibration_tokens(shape, m, seed=7)
    S, L, h, st = X.calibrate_projectors(lp.dev, to_dev(xs), lam=lam, clip=clip, mode=mode, with_stats=True)
    sync()
    rS, rL, rh, rst = O.calibrate(lp.ref, synth.widen(xs), shape.top_k, lam=lam, clip=clip, mode=mode)
    st = st.cpu().numpy()
    np.testing.assert_array_equal(st[..., 3], rst["n"])
    tol = 1e-4 if shape.dtype == "f32" else 1e-2
    obs = rst["n"] > 0
    np.testing.assert_allclose(st[..., 0][obs], rst["A"][obs], rtol=tol, atol=tol * np.abs(rst["A"]).max())
    np.testing.assert_allclose(st[..., 1][obs], rst["V"][obs], rtol=tol)
    np.testing.assert_allclose(st[..., 2][obs], rst["C"][obs], rtol=tol)
    S, L, h = S.cpu().numpy(), L.cpu().numpy(), h.cpu().numpy()
    np.testing.assert_allclose(S, rS, rtol=tol, atol=tol * max(1.0, np.abs(rS).max()))
    np.testing.assert_array_equal(L[~obs], rL[~obs])                  # 1e30 and the zero diagonal exactly
    np.testing.assert_allclose(L[obs], rL[obs], rtol=tol, atol=tol)
    np.testing.assert_allclose(h, rh, rtol=tol)


@pytest.mark.parametrize("shape,T,phase,budget", [(WIDE_BF16, 700, "prefill", 4), (WIDE_BF16, 64, "decode", 16),
                                                  (SHARED_BF16, 100, "decode", 8)])
def test_forward_is_deterministic(shape, T, phase, budget):
    lp = LayerPair(shape, seed=8)
    xs = to_dev(synth.tokens(shape, T, seed=8))
    S, L, h = (to_dev(a) for a in synth.synthetic_tables(shape.n_experts, seed=8))
    a = X.moe_forward(lp.dev, xs, phase, budget, S, L, h)
    b = X.moe_forward(lp.dev, xs, phase, budget, S, L, h)
    sync()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_zero_tokens_is_a_noop():
    lp = LayerPair(synth.TINY, seed=9)
    x = torch.empty((0, 256), dtype=torch.float32, device=DEV)
    S, L, h = (to_dev(a) for a in synth.synthetic_tables(8, seed=9))
    y = X.moe_forward(lp.dev, x, "prefill", 1, S, L, h)
    sync()
    assert y.shape == (0, 256)


# Rows per active group select the expert kernel: <= 8, <= 24, <= 64 rows stream
# the weights (16/32/64-row chunks); <= 384 use 128x128 LDS tiles; more use the
# 256x256 direct-to-LDS tiles.  Group sizes are skewed so every path also sees
# ragged groups, empty groups and partial tiles.
PATH_SHAPES = {
    "bf16-256x512": synth.LayerShape("paths", d=256, inter=512, n_experts=8, top_k=2, dtype="bf16"),
    "bf16-384x192": synth.LayerShape("paths-odd", d=384, inter=192, n_experts=8, top_k=2, dtype="bf16"),
    # at 8192 tokens: the wide gate/up tile with six 64-wide reduction stages and one pair of
    # 128-column gate/up slices (below that the skinny tile)
    "bf16-384x256": synth.LayerShape("paths-384", d=384, inter=256, n_experts=8, top_k=2, dtype="bf16"),
}


@pytest.mark.parametrize("shape_name", sorted(PATH_SHAPES))
@pytest.mark.parametrize("T,k_out", [(48, 1), (150, 1), (400, 1), (1900, 1), (4096, 1), (2100, 2), (8192, 1)])
def test_execute_every_kernel_path(shape_name, T, k_out):
    shape = PATH_SHAPES[shape_name]
    lp = LayerPair(shape, seed=11)
    rng = np.random.default_rng(T + k_out)
    p = np.array([0.3, 0.2, 0.15, 0.12, 0.1, 0.08, 0.05, 0.0])   # expert 7 stays empty
    ids = rng.choice(shape.n_experts, size=(T, k_out), p=p).astype(np.int32)
    w = rng.standard_normal((T, k_out)).astype(np.float32)
    xs = synth.tokens(shape, T, seed=11)
    dbg = {"offsets": torch.empty(shape.n_experts + 2, dtype=torch.int32, device=DEV)}
    y = X.moe_execute(lp.dev, to_dev(xs), to_dev(ids), to_dev(w), debug=dbg)
    sync()
    counts = np.diff(dbg["offsets"].cpu().numpy()[: shape.n_experts + 1])
    np.testing.assert_array_equal(counts, np.bincount(ids.reshape(-1), minlength=shape.n_experts))
    ref = O.moe_output(lp.ref, synth.widen(xs), ids, w)
    err = per_token_rel_l2(from_dev(y), ref)
    assert err.max() <= TOL_Y["bf16"], err.max()


# Wide tiles for both GEMMs (2 rows >= 3 x 256 per expert and at least one
# round of down tiles): whole rounds of one tile per CU, then a short last
# round whose tiles are split along the reduction and finished by the fixup
# kernel.  The wide tile list counts rows in 128-row units u_g = ceil(rows_g /
# 128) per pair of n-tiles (gate/up: inter / 256 pairs, down: d / 512); a
# group whose last tile holds at most 128 rows ends in one 128 x 512 tail tile
# per pair.
SPLIT_SHAPE = synth.LayerShape("wide-split", d=2048, inter=1024, n_experts=8, top_k=2, dtype="bf16")


def _routes_with_counts(counts, k_out, rng):
    """[T, k_out] routes in which expert e appears counts[e] times, distinct within a token."""
    labels = np.repeat(np.arange(len(counts)), counts).astype(np.int32)
    T = labels.size // k_out
    ids = labels.reshape(k_out, T).T.copy()   # every block of one label is shorter than T
    return ids[rng.permutation(T)]


def _wide_split(tiles, G, KT):
    """(whole tiles, remainder tiles, split) of a wide launch of `tiles` tiles in rounds of G."""
    rem = tiles % G
    s = min(G // rem, 16, KT // 4) if rem else 1
    return (tiles - rem, rem, s) if rem and s >= 2 else (tiles, 0, 1)


# units (sum of ceil(rows / 128)) -> route counts; 4 units per pair of n-tiles
# for both GEMMs: 75 units = 300 tiles (44 split 5 ways for gate/up, 4 for
# down; tails of each kind), 96 = 384 (128 split twice, the largest split
# remainder), 100 = 400 (144 left whole)
SPLIT_COUNTS = {32: [512] * 8,   # 128 tiles: no whole round, every tile split in two
                75: [1300, 1200, 1100, 1000, 1400, 1024, 1100, 1100],
                96: [1500, 1500, 1537, 1538, 1290, 1300, 1400, 1540],
                100: [1500, 1500, 1537, 1538, 1290, 1300, 1400, 2101]}


@pytest.mark.parametrize("units,k_out", [(32, 2), (75, 1), (75, 2), (96, 1), (100, 2)])
def test_execute_wide_split_remainder(units, k_out):
    shape = SPLIT_SHAPE
    counts = np.array(SPLIT_COUNTS[units])
    assert int(np.ceil(counts / 128).sum()) == units
    G = torch.cuda.get_device_properties(0).multi_processor_count
    tiles = units * (shape.inter // 256)          # = units * (d // 512) for the down GEMM
    print(f"wide split: {units} units, k_out={k_out}, G={G}: whole/rem/split gate/up "
          f"{_wide_split(tiles, G, shape.d // 64)}, down {_wide_split(tiles, G, shape.inter // 64)}", flush=True)
    lp = LayerPair(shape, seed=17)
    rng = np.random.default_rng(units * 10 + k_out)
    ids = _routes_with_counts(counts, k_out, rng)
    T = ids.shape[0]
    w = rng.standard_normal((T, k_out)).astype(np.float32)
    xs = synth.tokens(shape, T, seed=17)
    y = from_dev(X.moe_execute(lp.dev, to_dev(xs), to_dev(ids), to_dev(w)))
    sync()
    # sampled tokens: the ends, a random spread, and every token routed to the
    # last rows of each expert (the tail tiles)
    order = np.argsort(ids[:, 0], kind="stable")
    ends = np.cumsum(np.bincount(ids[:, 0], minlength=shape.n_experts))
    tails = np.concatenate([order[max(0, e - 8):e] for e in ends])
    smp = np.unique(np.concatenate([[0, T - 1], rng.choice(np.arange(1, T - 1), 254, replace=False), tails]))
    ref = O.moe_output(lp.ref, synth.widen(xs[smp]), ids[smp], w[smp])
    err = per_token_rel_l2(y[smp], ref)
    assert err.max() <= TOL_Y["bf16"], err.max()
    # every token was written: a tile left out of the fixup would leave stale or zero rows
    assert np.isfinite(y).all()
    assert (np.linalg.norm(y, axis=1) > 0).all()
    # the result does not depend on the run (fixed summation order of the split partials)
    y2 = from_dev(X.moe_execute(lp.dev, to_dev(xs), to_dev(ids), to_dev(w)))
    sync()
    np.testing.assert_array_equal(y, y2)


# A shared expert on the wide tiles: its rows form the last group (weights from
# the shared tensors), with a 128-row tail tile at 4096 + 96 tokens.
SHARED_WIDE = synth.LayerShape("shared-wide", d=2048, inter=512, n_experts=8, top_k=2, shared_inter=512,
                               dtype="bf16")


@pytest.mark.parametrize("T,k_out", [(4096, 2), (4192, 1)])
def test_execute_wide_with_shared_expert(T, k_out):
    shape = SHARED_WIDE
    lp = LayerPair(shape, seed=19)
    rng = np.random.default_rng(T)
    ids = np.stack([rng.permutation(shape.n_experts)[:k_out] for _ in range(T)]).astype(np.int32)
    w = rng.standard_normal((T, k_out)).astype(np.float32)
    xs = synth.tokens(shape, T, seed=19)
    y = from_dev(X.moe_execute(lp.dev, to_dev(xs), to_dev(ids), to_dev(w)))
    sync()
    smp = np.unique(np.concatenate([[0, T - 1], np.arange(T - 100, T), rng.choice(T, 200, replace=False)]))
    ref = O.moe_output(lp.ref, synth.widen(xs[smp]), ids[smp], w[smp])
    err = per_token_rel_l2(y[smp], ref)
    assert err.max() <= TOL_Y["bf16"], err.max()
    assert np.isfinite(y).all()
