"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle by a route other than its own code: closed forms,
brute force on tiny inputs, special cases that reduce to a textbook or
library routine, invariants the paper states, a hand-worked example with
dyadic numbers, and the storage figure the projector ablation table prints.
"""

import itertools
import math
import os

import numpy as np
import pytest
from scipy.special import expit

from oracle import exfold_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))


def rand_layer(rng, n=8, d=16, inter=8, shared=0, scale=0.3):
    gu = (rng.standard_normal((n, 2 * inter, d)) * scale).astype(np.float32)
    dn = (rng.standard_normal((n, d, inter)) * scale).astype(np.float32)
    wr = (rng.standard_normal((n, d)) * scale).astype(np.float32)
    sh = {}
    if shared:
        sh = dict(ws_gate_up=(rng.standard_normal((2 * shared, d)) * scale).astype(np.float32),
                  ws_down=(rng.standard_normal((d, shared)) * scale).astype(np.float32))
    return O.Layer(w_router=wr, w_gate_up=gu, w_down=dn, **sh)


# ---------------------------------------------------------------- experts (Eq. gated_expert)

def test_expert_scalar_closed_form():
    rng = np.random.default_rng(1)
    for _ in range(20):
        wg, wu, wd, x = rng.standard_normal(4) * 2
        gu = np.array([[wg], [wu]], dtype=np.float64)
        dn = np.array([[wd]])
        got = O.expert_forward(np.array([[x]]), gu, dn)[0, 0]
        z = wg * x
        want = wd * (z / (1.0 + math.exp(-z))) * (wu * x)
        assert got == pytest.approx(want, rel=1e-14, abs=1e-300)


def test_expert_diagonal_reduces_to_silu_times_x():
    # W_gate = diag(a), W_up = I, W_down = I  =>  E(x) = SiLU(a*x) * x, SiLU = z * sigmoid(z)
    rng = np.random.default_rng(2)
    d = 6
    a = rng.standard_normal(d)
    gu = np.concatenate([np.diag(a), np.eye(d)])
    x = rng.standard_normal((5, d)) * 3
    got = O.expert_forward(x, gu, np.eye(d))
    want = (a * x) * expit(a * x) * x
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-15)
    # gate and up are not interchangeable: swapping them changes the output
    swapped = O.expert_forward(x, np.concatenate([np.eye(d), np.diag(a)]), np.eye(d))
    assert not np.allclose(swapped, want)


def test_expert_zero_and_down_linearity():
    rng = np.random.default_rng(3)
    gu = rng.standard_normal((8, 5))
    dn = rng.standard_normal((5, 4))
    assert np.all(O.expert_forward(np.zeros((2, 5)), gu, dn) == 0)
    x = rng.standard_normal((3, 5))
    np.testing.assert_array_equal(O.expert_forward(x, gu, 4.0 * dn), 4.0 * O.expert_forward(x, gu, dn))


# ---------------------------------------------------------------- router (Eq. topk_gate)

def test_router_logits_unit_vectors():
    rng = np.random.default_rng(4)
    wr = rng.standard_normal((5, 7))
    b = rng.standard_normal(5)
    got = O.router_logits(np.eye(7), wr, b)
    np.testing.assert_array_equal(got, wr.T + b[None, :])


def _check_topk_property(logits, ids):
    n = logits.shape[1]
    for i in range(logits.shape[0]):
        row = logits[i].astype(np.float64)
        sel = [int(e) for e in ids[i]]
        assert len(set(sel)) == len(sel)
        for a, b in zip(sel, sel[1:]):
            assert row[a] > row[b] or (row[a] == row[b] and a < b)
        last = sel[-1]
        for e in range(n):
            if e not in sel:
                assert row[e] < row[last] or (row[e] == row[last] and e > last)


def test_topk_order_property_with_ties():
    rng = np.random.default_rng(5)
    logits = rng.standard_normal((200, 16)).astype(np.float32)
    logits[:, 3] = logits[:, 9]                  # exact ties between ids 3 and 9
    logits[::7, :] = np.round(logits[::7, :])    # many ties on some rows
    logits[5] = 0.0                              # all tied: ids 0..K-1
    logits[6, 4] = -0.0                          # -0 ties +0
    for k in (1, 2, 5, 16):
        ids = O.topk_ids(logits, k)
        _check_topk_property(logits, ids)
        assert list(ids[5]) == list(range(k))


def test_softmax_closed_forms():
    rng = np.random.default_rng(6)
    logits = rng.standard_normal((100, 10)).astype(np.float32) * 3
    ids, w = O.route(logits, 4)
    w64 = w.astype(np.float64)
    np.testing.assert_allclose(w64.sum(axis=1), 1.0, atol=4 * 2.0 ** -24)
    for i in range(0, 100, 9):
        for a in range(4):
            for b in range(4):
                ratio = math.exp(float(logits[i, ids[i, a]]) - float(logits[i, ids[i, b]]))
                assert w64[i, a] / w64[i, b] == pytest.approx(ratio, rel=4 * 2.0 ** -24)
    # equal logits give uniform weights; K=1 gives exactly 1
    _, wu = O.route(np.zeros((2, 8), np.float32), 4)
    assert np.all(wu == np.float32(0.25))
    _, w1 = O.route(logits, 1)
    assert np.all(w1 == 1.0)


# ---------------------------------------------------------------- prefill selection (Eq. prefill_budget)

def test_prefill_select_bruteforce_subsets():
    rng = np.random.default_rng(7)
    for k, kp in [(4, 1), (4, 2), (6, 3), (8, 4), (8, 7)]:
        ids = np.stack([rng.permutation(16)[:k] for _ in range(50)]).astype(np.int32)
        w = rng.random((50, k)).astype(np.float32)
        h = (rng.random(16) + 0.1).astype(np.float32)
        keep = O.select_prefill(ids, w, h, kp)
        for i in range(50):
            score = [float(w[i, j]) * float(h[ids[i, j]]) for j in range(k)]
            best = max(itertools.combinations(range(k), kp), key=lambda c: sum(score[j] for j in c))
            assert set(np.nonzero(keep[i])[0]) == set(best)


def test_prefill_select_constant_h_is_direct_topk():
    rng = np.random.default_rng(8)
    logits = rng.standard_normal((40, 12)).astype(np.float32)
    ids, w = O.route(logits, 6)
    keep = O.select_prefill(ids, w, np.full(12, 0.7, np.float32), 3)
    assert np.all(keep[:, :3]) and not np.any(keep[:, 3:])
    # all scores tied -> first K' route positions
    keep = O.select_prefill(ids, np.full_like(w, 0.25), np.ones(12, np.float32), 2)
    assert np.all(keep[:, :2]) and not np.any(keep[:, 2:])


# ---------------------------------------------------------------- prefill fold (Eq. prefill_fold)

def test_prefill_fold_hand_worked_example():
    # routes (5, 2, 7, 0), w = (1/2, 1/4, 1/8, 1/8); h5=1, h2=4, h7=2, h0=1
    # scores (1/2, 1, 1/4, 1/8) -> K'=2 keeps ids 5 and 2, listed in route order.
    # omitted 7: L[7,5]=1/2 > L[7,2]=1/4 -> target 2, S[7,2]=2: w~2 = 1/4 + 1/8*2 = 1/2
    # omitted 0: L[0,5] = L[0,2] -> first in route order -> 5, S[0,5]=-1: w~5 = 1/2 - 1/8 = 3/8
    n = 8
    ids = np.array([[5, 2, 7, 0]], np.int32)
    w = np.array([[0.5, 0.25, 0.125, 0.125]], np.float32)
    h = np.ones(n, np.float32)
    h[2], h[7] = 4.0, 2.0
    S = np.zeros((n, n), np.float32)
    L = np.ones((n, n), np.float32)
    L[7, 5], L[7, 2], S[7, 2] = 0.5, 0.25, 2.0
    L[0, 5], L[0, 2], S[0, 5] = 0.1, 0.1, -1.0
    keep = O.select_prefill(ids, w, h, 2)
    assert keep.tolist() == [[True, True, False, False]]
    out_ids, out_w = O.fold_prefill(ids, w, keep, S, L)
    assert out_ids.tolist() == [[5, 2]]
    assert out_w.tolist() == [[0.375, 0.5]]


def test_prefill_fold_properties():
    rng = np.random.default_rng(9)
    n, k, kp, t = 16, 8, 3, 60
    ids = np.stack([rng.permutation(n)[:k] for _ in range(t)]).astype(np.int32)
    w = rng.random((t, k)).astype(np.float32)
    h = rng.random(n).astype(np.float32)
    S = rng.standard_normal((n, n)).astype(np.float32)
    L = rng.random((n, n)).astype(np.float32)
    L[:, 3] = L[:, 5]                                   # ties in the loss table
    keep = O.select_prefill(ids, w, h, kp)
    out_ids, out_w = O.fold_prefill(ids, w, keep, S, L)
    assert out_ids.shape == (t, kp)
    for i in range(t):
        ret = [j for j in range(k) if keep[i, j]]
        assert out_ids[i].tolist() == [int(ids[i, j]) for j in ret]       # route order
        expect = {j: float(w[i, j]) for j in ret}
        for j in range(k):
            if keep[i, j]:
                continue
            s = int(ids[i, j])
            cand = [int(ids[i, r]) for r in ret]
            tpos = int(np.argmin(L[s, cand]))                           # numpy: first minimum
            expect[ret[tpos]] += float(w[i, j]) * float(S[s, cand[tpos]])
        np.testing.assert_array_equal(out_w[i], np.array([expect[j] for j in ret], np.float32))
    # S == 0: direct Top-K' drop, weights not renormalised
    _, w0 = O.fold_prefill(ids, w, keep, np.zeros_like(S), L)
    np.testing.assert_array_equal(w0, np.stack([w[i][keep[i]] for i in range(t)]))
    # S == 1: routed mass conserved
    _, w1 = O.fold_prefill(ids, w, keep, np.ones_like(S), L)
    np.testing.assert_allclose(w1.astype(np.float64).sum(1), w.astype(np.float64).sum(1), rtol=1e-6)


def test_prefill_identity_budget_is_bitwise():
    rng = np.random.default_rng(10)
    logits = rng.standard_normal((30, 12)).astype(np.float32)
    ids, w = O.route(logits, 4)
    for kp in (4, 5, 100):
        keep = O.select_prefill(ids, w, rng.random(12).astype(np.float32), kp)
        oi, ow = O.fold_prefill(ids, w, keep, rng.random((12, 12)), rng.random((12, 12)))
        assert np.array_equal(oi, ids) and np.array_equal(ow.view(np.uint32), w.view(np.uint32))


# ---------------------------------------------------------------- decode pool (Eq. decode_budget)

def test_decode_hand_worked_example():
    # token0 (1, 3) w (3/4, 1/4); token1 (3, 0) w (1/2, 1/2); token2 (2, 1) w (1/2, 1/2); h = (1, 1, 2, 1)
    # sum_w: e0 1/2, e1 5/4, e2 1/2, e3 3/4 -> scores 1/2, 5/4, 1, 3/4 -> D=2 pool (1, 2)
    # source 0: L[0,1]=.3 > L[0,2]=.2 -> 2, S=1/2;  source 3: L[3,1] = L[3,2] -> pool order -> 1, S=3
    ids = np.array([[1, 3], [3, 0], [2, 1]], np.int32)
    w = np.array([[0.75, 0.25], [0.5, 0.5], [0.5, 0.5]], np.float32)
    h = np.array([1, 1, 2, 1], np.float32)
    pool, cand = O.select_decode_pool(ids, w, h, 4, 2)
    assert pool == [1, 2] and cand == [0, 1, 2, 3]
    S = np.zeros((4, 4), np.float32)
    L = np.ones((4, 4), np.float32)
    L[0, 1], L[0, 2], S[0, 2] = 0.3, 0.2, 0.5
    L[3, 1], L[3, 2], S[3, 1] = 0.4, 0.4, 3.0
    ni, nw, tgt, scl = O.fold_decode(ids, w, pool, S, L, 4)
    assert ni.tolist() == [[1, 1], [1, 2], [2, 1]]
    assert nw.tolist() == [[0.75, 0.75], [1.5, 0.25], [0.5, 0.5]]
    assert tgt.tolist() == [2, 1, 2, 1] and scl.tolist() == [0.5, 1.0, 1.0, 3.0]


def test_decode_pool_bruteforce_and_fixed_point_bound():
    rng = np.random.default_rng(11)
    n, k = 10, 3
    for trial in range(30):
        b = int(rng.integers(1, 6))
        ids = np.stack([rng.permutation(n)[:k] for _ in range(b)]).astype(np.int32)
        w = rng.random((b, k)).astype(np.float32)
        h = (rng.random(n) + 0.05).astype(np.float32)
        dd = int(rng.integers(1, 7))
        pool, cand = O.select_decode_pool(ids, w, h, n, dd)
        assert cand == sorted(set(ids.reshape(-1).tolist()))
        assert len(pool) == min(dd, len(cand)) and set(pool) <= set(cand)
        real = {e: sum(float(w[i, j]) for i in range(b) for j in range(k) if ids[i, j] == e) * float(h[e])
                for e in cand}
        best = max(itertools.combinations(cand, len(pool)), key=lambda c: sum(real[e] for e in c))
        assert set(pool) == set(best)
        # pool order is descending real-valued score
        assert all(real[a] >= real[c] for a, c in zip(pool, pool[1:]))
        # R6 deviation bound: |fixed-point score - real score| <= slots * 2^-41 * h
        scale = 2.0 ** 40
        for e in cand:
            fx = sum(int(np.rint(float(w[i, j]) * scale)) for i in range(b) for j in range(k) if ids[i, j] == e)
            assert abs(fx / scale * float(h[e]) - real[e]) <= b * 2.0 ** -41 * float(h[e]) + 1e-15


def test_decode_pool_ties_lower_id():
    ids = np.array([[0, 1], [2, 3]], np.int32)
    w = np.full((2, 2), 0.5, np.float32)
    pool, _ = O.select_decode_pool(ids, w, np.ones(4, np.float32), 4, 3)
    assert pool == [0, 1, 2]


def test_decode_fold_invariants_and_identity():
    rng = np.random.default_rng(12)
    n, k = 32, 4
    S = rng.standard_normal((n, n)).astype(np.float32)
    L = rng.random((n, n)).astype(np.float32)
    for b in (1, 3, 17, 64):
        logits = rng.standard_normal((b, n)).astype(np.float32)
        ids, w = O.route(logits, k)
        h = rng.random(n).astype(np.float32)
        for dd in (1, 2, 5, 16, n):
            pool, cand = O.select_decode_pool(ids, w, h, n, dd)
            ni, nw, tgt, scl = O.fold_decode(ids, w, pool, S, L, n)
            assert ni.shape == ids.shape and nw.shape == w.shape
            assert len(set(ni.reshape(-1).tolist())) <= dd
            assert set(ni.reshape(-1).tolist()) <= set(pool)
            kept = np.isin(ids, pool)
            assert np.array_equal(ni[kept], ids[kept])
            assert np.array_equal(nw[kept].view(np.uint32), w[kept].view(np.uint32))
            # remapped weight == float32 multiply (numpy float32 arithmetic)
            moved = ~kept
            np.testing.assert_array_equal(nw[moved], (w * S[ids, ni])[moved])
            for s in range(n):
                if s not in pool:
                    assert tgt[s] == pool[int(np.argmin(L[s, pool]))]
            if dd >= len(cand):
                assert np.array_equal(ni, ids) and np.array_equal(nw.view(np.uint32), w.view(np.uint32))


def test_static_pool():
    h = np.array([0.5, 2.0, 2.0, 1.0, 0.1], np.float32)
    assert O.select_static_pool(h, 3) == [1, 2, 3]
    assert sorted(O.select_static_pool(h, 5)) == list(range(5))
    # D = N: every source is in the pool, the remap is the identity
    ids = np.array([[4, 0], [2, 1]], np.int32)
    w = np.array([[0.6, 0.4], [0.7, 0.3]], np.float32)
    ni, nw, _, _ = O.fold_decode(ids, w, O.select_static_pool(h, 5), np.zeros((5, 5)), np.ones((5, 5)), 5)
    assert np.array_equal(ni, ids) and np.array_equal(nw, w)


# ---------------------------------------------------------------- permutation

def test_permutation_matches_stable_argsort():
    rng = np.random.default_rng(13)
    for shape, n in [((64, 1), 8), ((100, 8), 128), ((1, 3), 4), ((0, 4), 5), ((37, 2), 3)]:
        ids = rng.integers(0, n, size=shape).astype(np.int32)
        counts, offsets, row_slot = O.permute_routes(ids, n)
        flat = ids.reshape(-1)
        np.testing.assert_array_equal(counts, np.bincount(flat, minlength=n))
        np.testing.assert_array_equal(offsets, np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=n))]))
        np.testing.assert_array_equal(row_slot, np.argsort(flat, kind="stable"))


# ---------------------------------------------------------------- layer output (Eq. moe_output)

def test_moe_output_equals_dense_masked_sum():
    """All N experts evaluated on every token, combined through a dense [T, N] gate matrix."""
    rng = np.random.default_rng(14)
    layer = rand_layer(rng, n=8, d=12, inter=6, shared=5)
    x = rng.standard_normal((9, 12)).astype(np.float32)
    ids = rng.integers(0, 8, size=(9, 3)).astype(np.int32)     # duplicates allowed (decode remap)
    w = rng.standard_normal((9, 3)).astype(np.float32)
    alpha = np.zeros((9, 8))
    for i in range(9):
        for j in range(3):
            alpha[i, ids[i, j]] += float(w[i, j])
    dense = sum(alpha[:, e:e + 1] * O.expert_forward(x, *layer.expert(e)) for e in range(8))
    dense = dense + O.expert_forward(x, layer.ws_gate_up, layer.ws_down)
    np.testing.assert_allclose(O.moe_output(layer, x, ids, w), dense, rtol=1e-12, atol=1e-13)


def test_identity_budgets_give_bitwise_dense_output():
    rng = np.random.default_rng(15)
    layer = rand_layer(rng, n=8, d=12, inter=6)
    x = rng.standard_normal((20, 12)).astype(np.float32)
    S = rng.standard_normal((8, 8)).astype(np.float32)
    L = rng.random((8, 8)).astype(np.float32)
    h = rng.random(8).astype(np.float32)
    y0, _ = O.moe_forward(layer, x, 3, "dense", 0)
    yp, _ = O.moe_forward(layer, x, 3, "prefill", 3, S, L, h)
    yd, info = O.moe_forward(layer, x, 3, "decode", 8, S, L, h)
    assert np.array_equal(y0, yp) and np.array_equal(y0, yd)


def test_fold_then_execute_equals_definition():
    """Eq. folded_moe term by term vs coalesced prefill fold and in-place decode remap."""
    rng = np.random.default_rng(16)
    n = 8
    layer = rand_layer(rng, n=n, d=10, inter=6, shared=4)
    x = rng.standard_normal((15, 10)).astype(np.float32)
    S = rng.standard_normal((n, n)).astype(np.float32)
    L = rng.random((n, n)).astype(np.float32)
    h = rng.random(n).astype(np.float32)
    logits = O.router_logits(x, layer.w_router)
    ids, w = O.route(logits, 4)
    # prefill, K' = 2
    y_fold, info = O.moe_forward(layer, x, 4, "prefill", 2, S, L, h)
    sets = [[int(ids[i, j]) for j in range(4) if info["keep"][i, j]] for i in range(15)]
    y_def = O.folded_output_by_definition(layer, x, ids, w, sets, S, L)
    np.testing.assert_allclose(y_fold, y_def, rtol=1e-6, atol=1e-7)  # w~ is stored as float32
    # decode, D = 3
    y_fold, info = O.moe_forward(layer, x, 4, "decode", 3, S, L, h)
    y_def = O.folded_output_by_definition(layer, x, ids, w, [info["pool"]] * 15, S, L)
    np.testing.assert_allclose(y_fold, y_def, rtol=1e-6, atol=1e-7)


# ---------------------------------------------------------------- calibration (Eq. scalar_projector, projection_loss)

def twin_layer(rng, d=16, inter=8, c=(0.5, -1.0, 2.0, -0.5)):
    """Experts 4+j copy gate/up of expert j and scale its down projection by c_j (a power of two)."""
    base = rand_layer(rng, n=4, d=d, inter=inter)
    gu = np.concatenate([base.w_gate_up, base.w_gate_up])
    dn = np.concatenate([base.w_down, np.stack([np.float32(cj) * base.w_down[j] for j, cj in enumerate(c)])])
    wr = (rng.standard_normal((8, d)) * 0.3).astype(np.float32)
    return O.Layer(w_router=wr, w_gate_up=gu, w_down=dn)


def test_exact_multiples_calibrate_to_exact_scalars_and_fold_exactly():
    rng = np.random.default_rng(17)
    c = (0.5, -1.0, 2.0, -0.5)
    layer = twin_layer(rng, c=c)
    xc = rng.standard_normal((40, 16)).astype(np.float32)
    S, L, h, st = O.calibrate(layer, xc, 2, lam=0.0, clip=4.0, mode="common")
    for j, cj in enumerate(c):
        assert st["S64"][4 + j, j] == cj and st["S64"][j, 4 + j] == 1.0 / cj
        assert st["L64"][4 + j, j] == 0.0 and st["L64"][j, 4 + j] == 0.0
    off = [(s, t) for s in range(8) for t in range(8) if s != t and abs(s - t) != 4]
    assert min(st["L64"][s, t] for s, t in off) > 0.0
    x = rng.standard_normal((24, 16)).astype(np.float32)
    # prefill: every token routes one twin pair; K' = 1
    j = rng.integers(0, 4, 24)
    flip = rng.random(24) < 0.5
    ids = np.stack([np.where(flip, j + 4, j), np.where(flip, j, j + 4)], 1).astype(np.int32)
    w = rng.random((24, 2)).astype(np.float32)
    keep = O.select_prefill(ids, w, h, 1)
    fi, fw = O.fold_prefill(ids, w, keep, S, L)
    y = O.moe_output(layer, x, ids, w)
    np.testing.assert_allclose(O.moe_output(layer, x, fi, fw), y, rtol=1e-6, atol=1e-9)  # fp32 metadata
    # same in float64 metadata: exact up to float64 rounding
    fw64 = np.array([float(w[i, keep[i]][0]) + float(w[i, ~keep[i]][0]) *
                     float(S[ids[i, ~keep[i]][0], fi[i, 0]]) for i in range(24)])[:, None]
    np.testing.assert_allclose(O.moe_output(layer, x, fi, fw64), y, rtol=1e-12, atol=1e-14)
    # decode: pool of the four base experts (large h), every twin folds onto its base
    hd = np.array([10, 10, 10, 10, 1, 1, 1, 1], np.float32)
    ids4 = np.concatenate([ids, ids[::-1]], 1)
    w4 = rng.random((24, 4)).astype(np.float32)
    pool, _ = O.select_decode_pool(ids4, w4, hd, 8, 4)
    assert sorted(pool) == [0, 1, 2, 3]
    ni, nw, tgt, scl = O.fold_decode(ids4, w4, pool, S, L, 8)
    assert tgt.tolist()[4:] == [0, 1, 2, 3] and scl.tolist()[4:] == list(c)
    np.testing.assert_allclose(O.moe_output(layer, x, ni, nw), O.moe_output(layer, x, ids4, w4),
                               rtol=1e-12, atol=1e-14)


def _pair_samples(layer, xc, top_k, mode):
    logits = O.router_logits(xc, layer.w_router)
    ids = O.topk_ids(logits, top_k)
    outs = np.stack([O.expert_forward(xc, *layer.expert(e)) for e in range(layer.n_experts)])
    ev = [list(map(int, ids[i])) if mode == "corouted" else list(range(layer.n_experts))
          for i in range(xc.shape[0])]
    return outs, ev


@pytest.mark.parametrize("mode", ["corouted", "common"])
def test_scalar_projector_is_weighted_ridge_least_squares(mode):
    rng = np.random.default_rng(18)
    layer = rand_layer(rng, n=5, d=8, inter=6)
    xc = rng.standard_normal((30, 8)).astype(np.float32)
    lam = 0.37
    S, L, h, st = O.calibrate(layer, xc, 2, lam=lam, clip=0.0, mode=mode)
    outs, ev = _pair_samples(layer, xc, 2, mode)
    checked = 0
    for s in range(5):
        for t in range(5):
            toks = [i for i in range(30) if s in ev[i] and t in ev[i]]
            if s == t or not toks:
                continue
            rows = [math.sqrt(np.linalg.norm(outs[s, i])) * outs[t, i] for i in toks]
            rhs = [math.sqrt(np.linalg.norm(outs[s, i])) * outs[s, i] for i in toks]
            M = np.concatenate(rows + [np.array([math.sqrt(lam)])])[:, None]
            r = np.concatenate(rhs + [np.array([0.0])])
            sol = np.linalg.lstsq(M, r, rcond=None)[0][0]
            assert st["S64"][s, t] == pytest.approx(sol, rel=1e-10, abs=1e-14)
            # Eq. projection_loss evaluated directly from the samples
            wts = [np.linalg.norm(outs[s, i]) for i in toks]
            num = sum(wi * np.sum((outs[s, i] - sol * outs[t, i]) ** 2) for wi, i in zip(wts, toks))
            den = sum(wi * np.sum(outs[s, i] ** 2) for wi, i in zip(wts, toks)) + O.EPSILON
            assert st["L64"][s, t] == pytest.approx(num / den, rel=1e-9, abs=1e-12)
            checked += 1
    assert checked > 0


def test_calibration_edge_cases():
    rng = np.random.default_rng(19)
    layer = rand_layer(rng, n=8, d=8, inter=4)
    xc = rng.standard_normal((3, 8)).astype(np.float32)          # few tokens: most pairs unobserved
    S, L, h, st = O.calibrate(layer, xc, 2)
    assert np.all(np.diag(S) == 1.0) and np.all(np.diag(L) == 0.0)
    unobs = (st["n"] == 0) & ~np.eye(8, dtype=bool)
    assert unobs.any()
    assert np.all(S[unobs] == 0.0) and np.all(L[unobs] == np.float32(1e30))
    assert np.all(np.abs(S) <= 4.0)
    # h: mean output norm over tokens routed to the expert; unrouted experts get the mean of observed
    outs, ev = _pair_samples(layer, xc, 2, "corouted")
    seen = sorted(set(e for row in ev for e in row))
    for e in seen:
        want = np.mean([np.linalg.norm(outs[e, i]) for i in range(3) if e in ev[i]])
        assert float(h[e]) == pytest.approx(want, rel=1e-6)
    for e in set(range(8)) - set(seen):
        assert float(h[e]) == pytest.approx(np.mean([float(st["h64"][s]) for s in seen]), rel=1e-6)


def test_clipped_scalar_defines_the_loss():
    # E_s = 8 E_t: unclipped s = 8; clipped to 4, the loss is ||8v - 4v||^2 / ||8v||^2 = 1/4
    rng = np.random.default_rng(20)
    layer = twin_layer(rng, c=(8.0, 1.0, 1.0, 1.0))
    xc = rng.standard_normal((10, 16)).astype(np.float32)
    S, L, h, st = O.calibrate(layer, xc, 2, lam=0.0, clip=4.0, mode="common")
    assert st["S64"][4, 0] == 4.0
    assert st["L64"][4, 0] == pytest.approx(0.25, rel=1e-12)
    _, _, _, st0 = O.calibrate(layer, xc, 2, lam=0.0, clip=0.0, mode="common")
    assert st0["S64"][4, 0] == 8.0 and st0["L64"][4, 0] == 0.0


def test_storage_matches_projector_ablation_table():
    rows = {}
    with open(os.path.join(HERE, "golden", "projector_storage.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                fam, val, unit = line.split()
                rows[fam] = (float(val), unit)
    units = {"B": 1, "MiB": 2 ** 20}
    for fam, (val, unit) in rows.items():
        got = O.table_storage_bytes(48, 128, fam) / units[unit]
        assert f"{got:.2f}" == f"{val:.2f}", fam


# ---------------------------------------------------------------- fold safeguards (Appendix C; Eq. dsv4_confidence)

def _safeguard_case():
    """Three routes of one token: experts 0, 1, 2 with w = (1/2, 1/4, 1/4); the
    first two are retained.  Source 2: L[2,0] = 3/4, L[2,1] = 1/2, S[2,1] = 2."""
    ids = np.array([[0, 1, 2]], np.int32)
    w = np.array([[0.5, 0.25, 0.25]], np.float32)
    keep = np.array([[True, True, False]])
    S = np.zeros((3, 3), np.float32)
    S[2, 0], S[2, 1] = 4.0, 2.0
    L = np.ones((3, 3), np.float32)
    L[2, 0], L[2, 1] = 0.75, 0.5
    return ids, w, keep, S, L


def test_safeguards_off_equal_the_main_fold():
    rng = np.random.default_rng(31)
    T, N, K, kp = 60, 16, 6, 2
    ids = np.stack([rng.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
    w = rng.random((T, K)).astype(np.float32)
    S = rng.standard_normal((N, N)).astype(np.float32)
    L = rng.random((N, N)).astype(np.float32)
    keep = O.select_prefill(ids, w, rng.random(N).astype(np.float32), kp)
    ref = O.fold_prefill(ids, w, keep, S, L)
    for kw in ({}, {"loss_cap": float(L.max())}, {"confidence": True}):
        L_ = np.zeros_like(L) if kw.get("confidence") else L     # c_s = 1 when every loss is 0
        ref_ = O.fold_prefill(ids, w, keep, S, L_)
        got = O.fold_prefill_safeguarded(ids, w, keep, S, L_, **kw)
        np.testing.assert_array_equal(got[0], ref_[0])
        np.testing.assert_array_equal(got[1].view(np.uint32), ref_[1].view(np.uint32))
    np.testing.assert_array_equal(O.fold_prefill_safeguarded(ids, w, keep, S, L)[1], ref[1])


def test_confidence_split_hand_worked():
    ids, w, keep, S, L = _safeguard_case()
    # target: expert 1 (loss 1/2 < 3/4); c = 1/2; target gets 1/4 * 1/2 * 2 = 1/4;
    # the rest 1/8 goes 2:1 to the retained routes (router weights 1/2 : 1/4)
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, confidence=True)
    np.testing.assert_array_equal(fw, np.float32([[0.5 + 1 / 12, 0.5 + 1 / 24]]))
    # with renormalisation the weights sum to the router total 1 (folded total 9/8)
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, confidence=True, renorm=True)
    np.testing.assert_allclose(fw, [[(7 / 12) * 8 / 9, (13 / 24) * 8 / 9]], rtol=2 ** -23)
    # a loss above 1 gives c = 0: nothing moves to the target, all of w_s is spread
    L2 = L.copy()
    L2[2, 0], L2[2, 1] = 3.0, 1.5
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L2, confidence=True)
    np.testing.assert_array_equal(fw, np.float32([[0.5 + 1 / 6, 0.25 + 1 / 12]]))


def test_loss_cap_hand_worked():
    ids, w, keep, S, L = _safeguard_case()
    # cap 0.6 excludes (2, 0) only: the target stays expert 1 -> w1 += 1/4 * 2
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=0.6)
    np.testing.assert_array_equal(fw, np.float32([[0.5, 0.75]]))
    # a loss equal to the cap is admissible
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=0.5)
    np.testing.assert_array_equal(fw, np.float32([[0.5, 0.75]]))
    # cap below every loss: the omitted route is dropped (Direct Top-K'), and the
    # renormalised weights keep the router's 2:1 ratio and sum to 1
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=0.4)
    np.testing.assert_array_equal(fw, np.float32([[0.5, 0.25]]))
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=0.4, renorm=True)
    np.testing.assert_allclose(fw, [[2 / 3, 1 / 3]], rtol=2 ** -23)
    # cap 0.7 excludes the cheaper pair's rival only; cap 0.8 keeps both: same target
    for cap in (0.7, 0.8):
        _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=cap)
        np.testing.assert_array_equal(fw, np.float32([[0.5, 0.75]]))
    # swap the losses: the target becomes expert 0 unless the cap excludes it
    L3 = L.copy()
    L3[2, 0], L3[2, 1] = 0.5, 0.75
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L3)
    np.testing.assert_array_equal(fw, np.float32([[1.5, 0.25]]))
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L3, loss_cap=0.4)
    np.testing.assert_array_equal(fw, np.float32([[0.5, 0.25]]))


def test_renormalisation_preserves_the_routed_weight_sum():
    rng = np.random.default_rng(32)
    T, N, K, kp = 80, 32, 8, 3
    ids = np.stack([rng.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
    w = rng.dirichlet(np.ones(K), size=T).astype(np.float32)
    S = rng.random((N, N)).astype(np.float32) * 2            # positive scalars: positive totals
    L = rng.random((N, N)).astype(np.float32)
    keep = O.select_prefill(ids, w, rng.random(N).astype(np.float32), kp)
    for kw in ({"renorm": True}, {"renorm": True, "confidence": True}, {"renorm": True, "loss_cap": 0.5}):
        _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, **kw)
        np.testing.assert_allclose(fw.astype(np.float64).sum(1), w.astype(np.float64).sum(1), rtol=K * 2 ** -23)
    # the confidence split conserves sum_t w_t + sum_s w_s (c_s S[s, t*] + 1 - c_s)
    _, fw = O.fold_prefill_safeguarded(ids, w, keep, S, L, confidence=True)
    for i in range(T):
        ret = [j for j in range(K) if keep[i, j]]
        exp = sum(float(w[i, j]) for j in ret)
        for j in range(K):
            if keep[i, j]:
                continue
            s = ids[i, j]
            lt = [float(L[s, ids[i, q]]) for q in ret]
            q = ret[int(np.argmin(lt))]
            c = min(1.0, max(0.0, 1.0 - min(lt)))
            exp += float(w[i, j]) * (c * float(S[s, ids[i, q]]) + 1.0 - c)
        assert abs(float(fw[i].astype(np.float64).sum()) - exp) <= 1e-6 * max(1.0, abs(exp))


# ---------------------------------------------------------------- diagonal projector (Eq. appendix_diagonal_projector)

def _diag_layer(rng, n=4, d=6, inter=5, shared_gate=False):
    gu = rng.standard_normal((n, 2 * inter, d)) * 0.5
    if shared_gate:
        gu[:] = gu[0]
    dn = rng.standard_normal((n, d, inter)) * 0.5
    wr = rng.standard_normal((n, d)) * 0.5
    return O.Layer(w_router=wr, w_gate_up=gu, w_down=dn)


def test_diagonal_projector_is_per_dimension_weighted_ridge():
    rng = np.random.default_rng(41)
    layer = _diag_layer(rng)
    x = rng.standard_normal((40, 6))
    lam = 0.3
    Dg, Ld, st = O.calibrate_diagonal(layer, x, top_k=3, lam=lam, mode="common")
    U = np.stack([O.expert_forward(x, *layer.expert(e)) for e in range(4)])      # [N, m, d]
    s, t = 2, 0
    wv = np.linalg.norm(U[s], axis=1)
    for nd in range(6):
        # minimise sum_i w_i (u_in - c v_in)^2 + lam c^2 as a stacked least-squares problem
        a = np.concatenate([np.sqrt(wv) * U[t][:, nd], [np.sqrt(lam)]])[:, None]
        b = np.concatenate([np.sqrt(wv) * U[s][:, nd], [0.0]])
        c = np.linalg.lstsq(a, b, rcond=None)[0][0]
        assert abs(st["D64"][s, t, nd] - c) <= 1e-10 * max(1.0, abs(c))
    # the loss is the weighted residual of the diagonal map, normalised by the source energy
    resid = float((wv * ((U[s] - st["D64"][s, t] * U[t]) ** 2).sum(1)).sum())
    energy = float((wv * (U[s] ** 2).sum(1)).sum())
    assert abs(st["L64"][s, t] - resid / (energy + O.EPSILON)) <= 1e-9 * max(1.0, st["L64"][s, t])
    assert np.all(Dg[np.arange(4), np.arange(4)] == 1.0) and np.all(Ld[np.arange(4), np.arange(4)] == 0.0)


def test_diagonal_recovers_per_dimension_scales_exactly():
    # target outputs scaled per hidden dimension: u = c . v (c a vector of powers of two):
    # with lambda = 0 the diagonal projector is exactly c with zero loss, while the
    # scalar projector cannot represent it (positive loss)
    rng = np.random.default_rng(42)
    layer = _diag_layer(rng, shared_gate=True)
    cvec = np.array([0.5, 2.0, -1.0, 4.0, 0.25, -2.0])
    layer.w_down[1] = cvec[:, None] * layer.w_down[0]
    x = rng.standard_normal((30, 6))
    Dg, Ld, _ = O.calibrate_diagonal(layer, x, top_k=4, lam=0.0, mode="common")
    np.testing.assert_array_equal(Dg[1, 0], cvec.astype(np.float32))
    assert Ld[1, 0] <= 1e-12
    S, L, _, _ = O.calibrate(layer, x, top_k=4, lam=0.0, clip=0.0, mode="common")
    assert L[1, 0] > 0.1


def test_diagonal_fold_reproduces_the_full_output_for_exact_maps():
    # experts 2 and 3 are exact per-dimension multiples of experts 0 and 1: with the
    # calibrated diagonal maps, folding them onto 0 and 1 gives the full output
    rng = np.random.default_rng(43)
    layer = _diag_layer(rng)
    c2 = np.array([0.5, 2.0, 1.0, -1.0, 0.25, 4.0])
    c3 = np.array([2.0, -0.5, 1.0, 0.5, 1.0, 2.0])
    layer.w_gate_up[2] = layer.w_gate_up[0]
    layer.w_gate_up[3] = layer.w_gate_up[1]
    layer.w_down[2] = c2[:, None] * layer.w_down[0]
    layer.w_down[3] = c3[:, None] * layer.w_down[1]
    x = rng.standard_normal((30, 6))
    Dg, Ld, _ = O.calibrate_diagonal(layer, x, top_k=4, lam=0.0, mode="common")
    ids = np.array([[0, 1, 2, 3]] * 30, np.int32)
    w = np.tile(np.float32([0.4, 0.3, 0.2, 0.1]), (30, 1))
    keep = np.array([[True, True, False, False]] * 30)
    oi, ow, folds = O.fold_prefill_diagonal(ids, w, keep, Ld)
    assert [(s, q) for s, _, q in folds[0]] == [(2, 0), (3, 1)]
    y = O.diagonal_output(layer, x, oi, ow, folds, Dg)
    ref = O.moe_output(layer, x, ids, w)
    assert np.abs(y - ref).max() <= 1e-6 * np.abs(ref).max()


def test_diagonal_with_uniform_maps_equals_the_scalar_fold():
    # a diagonal map c . 1 acts like the scalar c: same targets (same loss table),
    # same output as Eq. prefill_fold
    rng = np.random.default_rng(44)
    layer = _diag_layer(rng, n=6, d=5, inter=4)
    x = rng.standard_normal((20, 5))
    S = rng.standard_normal((6, 6)).astype(np.float32)
    L = rng.random((6, 6)).astype(np.float32)
    Dg = np.repeat(S[:, :, None], 5, axis=2)
    lg = O.router_logits(x, layer.w_router)
    ids, w = O.route(lg, 4)
    keep = O.select_prefill(ids, w, rng.random(6).astype(np.float32), 2)
    oi, ow, folds = O.fold_prefill_diagonal(ids, w, keep, L)
    y = O.diagonal_output(layer, x, oi, ow, folds, Dg)
    fi, fw = O.fold_prefill(ids, w, keep, S, L)
    np.testing.assert_array_equal(oi, fi)
    ref = O.moe_output(layer, x, fi, fw)
    assert np.abs(y - ref).max() <= 1e-6 * np.abs(ref).max()
