"""The folded forward captured in a HIP graph replays bit-for-bit.

exfold_moe_forward allocates nothing and issues no memset or host
synchronisation, so a caller can capture it (torch.cuda.graph records the
library's launches on the capture stream).  Each case captures one forward,
then replays the graph several times with the program's own eager work (new
inputs copied in, an eager forward, synchronisations) between the replays, and
checks every replay against the eager forward on the same inputs, bitwise.
"""

import numpy as np
import pytest
import torch

from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

from .gpu_common import LayerPair, sync, to_dev

pytestmark = pytest.mark.gpu

WIDE_BF16 = synth.LayerShape("wide-bf16", d=256, inter=128, n_experts=128, top_k=8, dtype="bf16",
                             router_bias=True, m_cal=1024)
SHARED_BF16 = synth.LayerShape("shared-bf16", d=384, inter=192, n_experts=64, top_k=6, shared_inter=192,
                               dtype="bf16", m_cal=512)
# 4096 tokens on 8 experts: the gate/up GEMM takes the wide tile loaded straight into LDS
DEEP_BF16 = synth.LayerShape("deep-bf16", d=256, inter=512, n_experts=8, top_k=2, dtype="bf16")


@pytest.mark.parametrize("shape,T,phase,budget", [(WIDE_BF16, 300, "prefill", 4), (WIDE_BF16, 48, "decode", 16),
                                                  (SHARED_BF16, 40, "decode", 8), (synth.TINY, 64, "prefill", 1),
                                                  (WIDE_BF16, 48, "dense", 8), (DEEP_BF16, 4096, "prefill", 1)])
def test_graph_replays_match_eager(shape, T, phase, budget):
    lp = LayerPair(shape, seed=21)
    S, L, h = (to_dev(a) for a in synth.synthetic_tables(shape.n_experts, seed=21))
    x_in = to_dev(synth.tokens(shape, T, seed=21))
    y_out = torch.empty_like(x_in)
    ws = torch.empty(X.moe_workspace_size(lp.dev, T, phase, budget), dtype=torch.uint8, device=x_in.device)
    key = "topk_ids" if phase == "dense" else "fold_ids"   # the routes the layer executed
    fold_ids = X.debug_buffers(lp.dev, T, phase, budget, x_in.device)[key]

    def fwd():
        X.moe_forward(lp.dev, x_in, phase, budget, S, L, h, y=y_out, workspace=ws, debug={key: fold_ids})

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fwd()
    torch.cuda.current_stream().wait_stream(side)
    sync()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fwd()
    sync()

    for rep in range(4):
        xs = to_dev(synth.tokens(shape, T, seed=100 + rep))
        ref = X.moe_forward(lp.dev, xs, phase, budget, S, L, h)          # eager, own buffers
        ref_ids = torch.empty_like(fold_ids)
        X.moe_forward(lp.dev, xs, phase, budget, S, L, h, debug={key: ref_ids})
        sync()
        x_in.copy_(xs)
        y_out.fill_(0)
        g.replay()
        sync()
        assert torch.equal(y_out.view(torch.int16) if y_out.dtype == torch.bfloat16 else y_out.view(torch.int32),
                           ref.view(torch.int16) if ref.dtype == torch.bfloat16 else ref.view(torch.int32)), \
            f"replay {rep} differs from the eager forward"
        np.testing.assert_array_equal(fold_ids.cpu().numpy(), ref_ids.cpu().numpy())
    print(f"{shape.name} {phase} T={T}: 4 graph replays bitwise equal to eager", flush=True)
