"""exfold_moe_forward_scratch (the forward for callers that cannot allocate)
against exfold_moe_forward with a caller workspace: the same kernels on the
library's static scratch, so every output is bit-identical.  Two calls in a
row per phase, the second with fewer tokens (the scratch keeps the first
call's contents)."""

import numpy as np
import pytest
import torch

from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import DEV, LayerPair, sync, to_dev

pytestmark = pytest.mark.gpu

SHAPE = synth.LayerShape("scratch-bf16", d=512, inter=256, n_experts=64, top_k=6, shared_inter=256,
                         dtype="bf16", router_bias=True)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32) \
        if t.dtype in (torch.float32, torch.int32) else t


@pytest.mark.parametrize("phase,budget,sizes", [("decode", 16, (256, 40)), ("prefill", 3, (1500, 300)),
                                                ("dense", 0, (700, 1)), ("decode_static", 8, (96, 7))])
def test_scratch_forward_matches_workspace_forward(phase, budget, sizes):
    lp = LayerPair(SHAPE, seed=21)
    S, L, h = (to_dev(a) for a in synth.synthetic_tables(SHAPE.n_experts, seed=21))
    static = None
    if phase == "decode_static":
        _, _, tgt, scl = X.static_pool(h, budget, S, L)
        static = (tgt, scl)
    for T in sizes:
        assert X.moe_workspace_size(lp.dev, T, phase, budget) <= X.SCRATCH_BYTES
        print(f"scratch forward: {phase} T={T} budget={budget}", flush=True)
        x = to_dev(synth.tokens(SHAPE, T, seed=T))
        dbg_a = X.debug_buffers(lp.dev, T, phase, budget, DEV)
        dbg_b = X.debug_buffers(lp.dev, T, phase, budget, DEV)
        for v in (*dbg_a.values(), *dbg_b.values()):
            v.fill_(7)           # entries a phase does not write stay equal
        ya = X.moe_forward(lp.dev, x, phase, budget, S, L, h, debug=dbg_a, static_tables=static)
        yb = torch.full_like(x, float("nan"))
        X.moe_forward_scratch(lp.dev, x, phase, budget, S, L, h, y=yb, debug=dbg_b, static_tables=static)
        sync()
        assert torch.equal(_bits(ya), _bits(yb)), f"y differs ({phase}, T={T})"
        keys = ["logits", "topk_ids", "topk_w", "fold_ids", "fold_w", "offsets", "row_slot"]
        if phase == "prefill":
            keys.append("keep")
        if phase == "decode":
            keys += ["pool", "pool_size", "tgt_ids", "tgt_scale"]
        for k in keys:
            assert torch.equal(_bits(dbg_a[k]), _bits(dbg_b[k])), f"{k} differs ({phase}, T={T})"
        assert np.isfinite(yb.float().cpu().numpy()).all()
