"""Prefill fold safeguards on the GPU against the oracle: the loss cap, the
renormalisation and the confidence split (Appendix C; Appendix F, Eq.
dsv4_confidence), alone and combined, on the fold stage and in the forward."""

import numpy as np
import pytest
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import DEV, TOL_Y, LayerPair, from_dev, per_token_rel_l2, sync, to_dev

pytestmark = pytest.mark.gpu

OPTS = [dict(loss_cap=0.99), dict(renorm=True), dict(confidence=True), dict(loss_cap=0.5, renorm=True),
        dict(confidence=True, renorm=True), dict(loss_cap=0.7, confidence=True, renorm=True),
        dict(loss_cap=-1.0), dict(loss_cap=-1.0, renorm=True)]


@pytest.mark.parametrize("T,N,K,kp", [(64, 8, 2, 1), (333, 128, 8, 4), (200, 64, 6, 3), (50, 16, 16, 5),
                                      (17, 256, 16, 1)])
@pytest.mark.parametrize("opts", OPTS, ids=lambda o: "-".join(f"{k}={v}" for k, v in o.items()))
def test_safeguarded_fold_matches_oracle(T, N, K, kp, opts):
    rng = np.random.default_rng(T + N + K + len(opts))
    ids = np.stack([rng.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
    w = rng.dirichlet(np.ones(K), size=T).astype(np.float32)
    h = rng.random(N).astype(np.float32)
    S = (rng.standard_normal((N, N)) * 1.5).astype(np.float32)
    L = (rng.random((N, N)) * 1.3).astype(np.float32)            # some losses above 1: c_s = 0
    L[:, 1] = L[:, 0]                                            # loss ties
    L[rng.random((N, N)) < 0.1] = np.float32(1e30)               # unobserved pairs
    L[rng.random((N, N)) < 0.05] = np.float32(0.5)               # exactly at a cap
    d_ids, d_w = to_dev(ids), to_dev(w)
    _, _, keep = X.select_prefill(to_dev(h), kp, topk_ids=d_ids, topk_w=d_w)
    out_ids, out_w = X.fold_gates("prefill", kp, d_ids, d_w, to_dev(S), to_dev(L), keep=keep, **opts)
    sync()
    ref_keep = O.select_prefill(ids, w, h, kp)
    np.testing.assert_array_equal(keep.cpu().numpy().astype(bool), ref_keep)
    ri, rw = O.fold_prefill_safeguarded(ids, w, ref_keep, S, L, **opts)
    np.testing.assert_array_equal(out_ids.cpu().numpy(), ri)
    np.testing.assert_array_equal(out_w.cpu().numpy().view(np.uint32), rw.view(np.uint32))


def test_safeguards_off_equal_the_main_fold():
    rng = np.random.default_rng(5)
    T, N, K, kp = 256, 128, 8, 4
    ids = np.stack([rng.permutation(N)[:K] for _ in range(T)]).astype(np.int32)
    w = rng.dirichlet(np.ones(K), size=T).astype(np.float32)
    S = rng.standard_normal((N, N)).astype(np.float32)
    L = rng.random((N, N)).astype(np.float32)
    keep = to_dev(O.select_prefill(ids, w, rng.random(N).astype(np.float32), kp).astype(np.uint8))
    a = X.fold_gates("prefill", kp, to_dev(ids), to_dev(w), to_dev(S), to_dev(L), keep=keep)
    b = X.fold_gates("prefill", kp, to_dev(ids), to_dev(w), to_dev(S), to_dev(L), keep=keep,
                     loss_cap=float(L.max()))
    sync()
    assert (a[0] == b[0]).all()
    assert (a[1].view(torch.int32) == b[1].view(torch.int32)).all()


WIDE_BF16 = synth.LayerShape("wide-bf16", d=256, inter=128, n_experts=128, top_k=8, dtype="bf16",
                             router_bias=True)


@pytest.mark.parametrize("shape,T,kp,opts", [(WIDE_BF16, 300, 4, dict(loss_cap=0.99, renorm=True)),
                                             (WIDE_BF16, 200, 2, dict(confidence=True)),
                                             (synth.TINY, 64, 1, dict(confidence=True, renorm=True))])
def test_safeguarded_forward_matches_oracle(shape, T, kp, opts):
    lp = LayerPair(shape, seed=9)
    xs = synth.tokens(shape, T, seed=9)
    S, L, h = synth.synthetic_tables(shape.n_experts, seed=9)
    dbg = X.debug_buffers(lp.dev, T, "prefill", kp, DEV)
    y = X.moe_forward(lp.dev, to_dev(xs), "prefill", kp, to_dev(S), to_dev(L), to_dev(h), debug=dbg,
                      safeguards=opts)
    sync()
    ids, w = dbg["topk_ids"].cpu().numpy(), dbg["topk_w"].cpu().numpy()
    keep = O.select_prefill(ids, w, h, kp)
    ri, rw = O.fold_prefill_safeguarded(ids, w, keep, S, L, **opts)
    np.testing.assert_array_equal(dbg["fold_ids"].cpu().numpy(), ri)
    np.testing.assert_array_equal(dbg["fold_w"].cpu().numpy().view(np.uint32), rw.view(np.uint32))
    ref = O.moe_output(lp.ref, synth.widen(xs), ri, rw)
    err = per_token_rel_l2(from_dev(y), ref)
    assert err.max() <= TOL_Y[shape.dtype], err.max()
