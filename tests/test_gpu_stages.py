"""Stage-wise parity of the HIP kernels with the oracle on identical input bytes.

Discrete outputs (Top-K ids, keep masks, pools, decode tables, folded ids,
permutations) and the folded weights must be bit-exact: both sides take every
decision on the same float32 values with exact float64 products or exact
integer sums.  Softmax weights are float64 on both sides, rounded once.
"""

import numpy as np
import pytest
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X

from .gpu_common import DEV, from_dev, to_dev, sync

pytestmark = pytest.mark.gpu

rng_cases = [
    # (T, N, K, budget)
    (1, 8, 2, 1), (64, 8, 2, 1), (333, 128, 8, 4), (1000, 128, 8, 2), (257, 256, 16, 7), (5, 16, 16, 15),
    (100, 64, 6, 3), (77, 128, 8, 8), (31, 128, 8, 12),
]


def rand_logits(rng, T, N, ties=False):
    lg = (rng.standard_normal((T, N)) * 1.5).astype(np.float32)
    if ties:
        lg[::3] = np.round(lg[::3])          # many exact ties
        lg[1::5, : N // 2] = lg[1::5, N // 2: 2 * (N // 2)]
    return lg


@pytest.mark.parametrize("T,N,K,kp", rng_cases)
@pytest.mark.parametrize("ties", [False, True])
def test_topk_softmax_and_prefill_select(T, N, K, kp, ties):
    rng = np.random.default_rng(T * 7 + N + K + ties)
    lg = rand_logits(rng, T, N, ties)
    h = (rng.random(N) + 0.05).astype(np.float32)
    if ties:
        h[::2] = 1.0
    ids, w, keep = X.select_prefill(to_dev(h), kp, logits=to_dev(lg), top_k=K)
    sync()
    ref_ids, ref_w = O.route(lg, K)
    np.testing.assert_array_equal(ids.cpu().numpy(), ref_ids)
    np.testing.assert_allclose(w.cpu().numpy(), ref_w, rtol=2 ** -22, atol=0)
    # selection on identical route bytes: bit-exact
    ref_keep = O.select_prefill(ids.cpu().numpy(), w.cpu().numpy(), h, kp)
    np.testing.assert_array_equal(keep.cpu().numpy().astype(bool), ref_keep)


@pytest.mark.parametrize("T,N,K,kp", rng_cases)
def test_prefill_fold(T, N, K, kp):
    rng = np.random.default_rng(1000 + T + N)
    ids = np.stack([rng.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
    w = rng.random((T, K)).astype(np.float32)
    h = rng.random(N).astype(np.float32)
    S = rng.standard_normal((N, N)).astype(np.float32)
    L = rng.random((N, N)).astype(np.float32)
    L[:, 1] = L[:, 0]                                                         # loss ties
    L[:, 5:8] = L[:, 4:5]
    L[rng.random((N, N)) < 0.1] = np.float32(1e30)                            # unobserved pairs
    d_ids, d_w = to_dev(ids), to_dev(w)
    _, _, keep = X.select_prefill(to_dev(h), kp, topk_ids=d_ids, topk_w=d_w)
    out_ids, out_w = X.fold_gates("prefill", kp, d_ids, d_w, to_dev(S), to_dev(L), keep=keep)
    sync()
    ref_keep = O.select_prefill(ids, w, h, kp)
    np.testing.assert_array_equal(keep.cpu().numpy().astype(bool), ref_keep)
    ri, rw = O.fold_prefill(ids, w, ref_keep, S, L)
    np.testing.assert_array_equal(out_ids.cpu().numpy(), ri)
    np.testing.assert_array_equal(out_w.cpu().numpy().view(np.uint32), rw.view(np.uint32))


@pytest.mark.parametrize("B,N,K,D", [(1, 8, 2, 4), (32, 8, 2, 4), (16, 128, 8, 32), (64, 128, 8, 32),
                                     (256, 128, 8, 64), (512, 128, 8, 16), (3, 128, 8, 64), (40, 256, 16, 100),
                                     (7, 16, 4, 16), (128, 128, 8, 128)])
def test_decode_pool_and_remap(B, N, K, D):
    rng = np.random.default_rng(B * 31 + N + D)
    lg = rand_logits(rng, B, N)
    h = (rng.random(N) + 0.05).astype(np.float32)
    S = rng.standard_normal((N, N)).astype(np.float32)
    L = rng.random((N, N)).astype(np.float32)
    L[rng.random((N, N)) < 0.05] = np.float32(1e30)
    ids, w, pool, psize = X.select_decode_pool(to_dev(h), D, logits=to_dev(lg), top_k=K)
    sync()
    ref_ids, ref_w = O.route(lg, K)
    np.testing.assert_array_equal(ids.cpu().numpy(), ref_ids)
    gi, gw = ids.cpu().numpy(), w.cpu().numpy()
    ref_pool, cand = O.select_decode_pool(gi, gw, h, N, D)
    n = int(psize.cpu().numpy()[0])
    assert n == len(ref_pool)
    got_pool = pool.cpu().numpy()
    assert got_pool[:n].tolist() == ref_pool
    assert np.all(got_pool[n:] == -1)
    out_ids, out_w, tgt, scl = X.fold_gates("decode", D, ids, w, to_dev(S), to_dev(L), pool=pool,
                                            pool_size=psize, tables=True)
    sync()
    ri, rw, rt, rs = O.fold_decode(gi, gw, ref_pool, S, L, N)
    np.testing.assert_array_equal(tgt.cpu().numpy(), rt)
    np.testing.assert_array_equal(scl.cpu().numpy().view(np.uint32), rs.view(np.uint32))
    np.testing.assert_array_equal(out_ids.cpu().numpy(), ri)
    np.testing.assert_array_equal(out_w.cpu().numpy().view(np.uint32), rw.view(np.uint32))
    assert len(set(out_ids.cpu().numpy().reshape(-1).tolist())) <= D


def test_decode_pool_ties_and_fixed_point():
    # equal weight sums and equal h: pool order falls back to the lower id
    N, K, B = 16, 2, 8
    ids = np.array([[i % N, (i + 8) % N] for i in range(B)], np.int32)
    w = np.full((B, K), 0.5, np.float32)
    h = np.ones(N, np.float32)
    _, _, pool, ps = X.select_decode_pool(to_dev(h), 5, topk_ids=to_dev(ids), topk_w=to_dev(w))
    sync()
    ref, _ = O.select_decode_pool(ids, w, h, N, 5)
    assert pool.cpu().numpy()[: int(ps.item())].tolist() == ref == [0, 1, 2, 3, 4]
    # tiny weights exercise the rint(w * 2^40) rounding
    w2 = np.array([[3e-13, 1 - 3e-13]] * B, np.float32)
    _, _, pool, ps = X.select_decode_pool(to_dev(h), 3, topk_ids=to_dev(ids), topk_w=to_dev(w2))
    sync()
    ref, _ = O.select_decode_pool(ids, w2, h, N, 3)
    assert pool.cpu().numpy()[: int(ps.item())].tolist() == ref


def test_decode_empty_batch_and_identity():
    N, K = 32, 4
    h = torch.ones(N, device=DEV)
    ids = torch.empty((0, K), dtype=torch.int32, device=DEV)
    w = torch.empty((0, K), dtype=torch.float32, device=DEV)
    _, _, pool, ps = X.select_decode_pool(h, 8, topk_ids=ids, topk_w=w)
    sync()
    assert int(ps.item()) == 0 and np.all(pool.cpu().numpy() == -1)


@pytest.mark.parametrize("T,k_out,N,shared", [(64, 1, 8, False), (1000, 4, 128, False), (333, 8, 128, True),
                                              (1, 2, 8, False), (2500, 3, 256, True), (17, 8, 128, False),
                                              # at and just past the one-workgroup capacity (4096 slots)
                                              (1024, 4, 128, True), (4097, 1, 8, False)])
def test_permutation_is_stable_counting_sort(T, k_out, N, shared):
    from .gpu_common import LayerPair
    from paper_2608_24938_amd import synth
    rng = np.random.default_rng(T + k_out)
    # skewed ids with empty groups and duplicates within a token
    p = rng.dirichlet(np.full(N, 0.3))
    ids = rng.choice(N, size=(T, k_out), p=p).astype(np.int32)
    w = rng.standard_normal((T, k_out)).astype(np.float32)
    shape = synth.LayerShape("perm", d=128, inter=64, n_experts=N, top_k=min(8, N),
                             shared_inter=64 if shared else 0, dtype="bf16")
    lp = LayerPair(shape, seed=3)
    x = to_dev(synth.tokens(shape, T, seed=3))
    dbg = {"offsets": torch.empty(N + 2, dtype=torch.int32, device=DEV),
           "row_slot": torch.empty(T * k_out + (T if shared else 0), dtype=torch.int32, device=DEV)}
    X.moe_execute(lp.dev, x, to_dev(ids), to_dev(w), debug=dbg)
    sync()
    counts, offsets, row_slot = O.permute_routes(ids, N)
    got_off = dbg["offsets"].cpu().numpy()
    np.testing.assert_array_equal(got_off[: N + 1], offsets)
    assert got_off[N + 1] == T * k_out + (T if shared else 0)
    got_rs = dbg["row_slot"].cpu().numpy()
    np.testing.assert_array_equal(got_rs[: T * k_out], row_slot)
    if shared:
        assert np.all(got_rs[T * k_out:] == -1)
