"""The measurement arithmetic (algorithmic flops and bytes) against closed forms.

Pinned to the sizes of the layer shapes: a prefill layer executes 2·d·N flops
of router GEMM per token and 6·d·I per executed route (4·d·I gate/up, 2·d·I
down); a decode layer reads the three weight matrices of every touched expert
once (3·d·I elements), plus the shared expert, the router weights, x and y.
"""

import pytest

from paper_2608_24938_amd import synth
from paper_2608_24938_amd.measure import decode_bytes, prefill_flops


def test_mixtral_prefill_flops():
    # 4096 tokens, K'=1: 2*4096*8*4096 + 6*4096*14336*4096
    assert prefill_flops(synth.MIXTRAL, 4096, 1) == 2 * 4096 * 8 * 4096 + 6 * 4096 * 14336 * 4096
    assert prefill_flops(synth.MIXTRAL, 4096, 1) == pytest.approx(1.44338e12, rel=1e-5)


def test_prefill_flops_linear_in_routes():
    base = prefill_flops(synth.QWEN3, 8192, 0)
    per_route = 6 * 2048 * 768 * 8192
    for k in (1, 4, 8):
        assert prefill_flops(synth.QWEN3, 8192, k) == base + k * per_route


def test_shared_expert_counts_once_per_token():
    no_routes = prefill_flops(synth.GLM45, 100, 0)
    assert no_routes == 2 * 4096 * 128 * 100 + 6 * 4096 * 1408 * 100


def test_mixtral_decode_bytes():
    # four experts of 3*4096*14336 bf16 weights, router 8x4096, x and y 32x4096, routes 32*2*16 B
    want = 4 * 3 * 4096 * 14336 * 2 + 8 * 4096 * 2 + 2 * 32 * 4096 * 2 + 32 * 2 * 16
    assert decode_bytes(synth.MIXTRAL, 32, 4) == want
    assert decode_bytes(synth.MIXTRAL, 32, 4) == pytest.approx(1.4099e9, rel=1e-4)


def test_glm_decode_bytes_include_shared_expert():
    touched = 32
    w = (touched + 1) * 3 * 4096 * 1408 * 2
    assert decode_bytes(synth.GLM45, 64, touched) == w + 128 * 4096 * 2 + 2 * 64 * 4096 * 2 + 64 * 8 * 16
