"""Expert-GEMM plans (host logic, no GPU): the kernel family each workload shape
takes, and launch grids that cover every split of the rows into expert groups
(a grid short of the device-side tile count would leave tiles uncomputed)."""

import ctypes

import numpy as np
import pytest

from paper_2608_24938_amd import exfold as X

FAKE = 0x10000  # weights are never dereferenced by the planner
SIMT, TILE, SKINNY, WIDE = range(4)


def layer(d, inter, n, k, shared=0, dtype=X.BF16):
    return X._Layer(d, inter, n, k, shared, dtype, 0, FAKE, None, FAKE, FAKE,
                    FAKE if shared else None, FAKE if shared else None)


def plan(ly, rows, active, cu=256):
    out = (ctypes.c_int32 * 10)()
    assert X.lib().exfold_gemm_plan(ctypes.byref(ly), rows, active, cu, out) == X.OK
    v = list(out)
    return dict(zip(("kind", "bm", "bn", "ksplit", "grid"), v[:5])), dict(zip(("kind", "bm", "bn", "ksplit", "grid"), v[5:]))


MIXTRAL = dict(d=4096, inter=14336, n=8, k=2)
QWEN3 = dict(d=2048, inter=768, n=128, k=8)
GLM = dict(d=4096, inter=1408, n=128, k=8, shared=1408)


@pytest.mark.parametrize("shape,rows,active,gu_kind,dn_kind", [
    (MIXTRAL, 4096, 8, WIDE, WIDE),          # prefill, 4096 tokens, K' = 1
    (MIXTRAL, 8192, 8, WIDE, WIDE),
    (MIXTRAL, 64, 4, SKINNY, SKINNY),        # decode, 32 tokens, pool of 4
    (QWEN3, 32768, 128, WIDE, WIDE),         # prefill, 8192 tokens, K' = 4
    (QWEN3, 1024, 16, TILE, TILE),           # decode, 128 tokens, pool of 16 (64 rows per expert)
    (QWEN3, 1024, 64, SKINNY, SKINNY),       # decode, 128 tokens, pool of 64 (16 rows per expert)
    (QWEN3, 4096, 32, WIDE, WIDE),           # decode, 512 tokens, pool of 32 (wide down without a full round)
    (QWEN3, 2048, 16, TILE, TILE),           # 128 rows per expert but 48 wide tiles, under a quarter round
    (QWEN3, 2048, 32, TILE, TILE),           # 64 rows per expert: 128x128 down tiles above 48 rows
    (QWEN3, 1024, 32, TILE, SKINNY),         # 32 rows per expert: skinny down tiles up to 48 rows
    (QWEN3, 512, 16, TILE, SKINNY),          # 32 rows per expert: 128x128 gate/up tiles above 24 rows
    (QWEN3, 384, 16, SKINNY, SKINNY),        # 24 rows per expert: skinny gate/up tiles
    (GLM, 64 * 8 + 64, 33, SKINNY, SKINNY),  # decode with the shared expert
    (GLM, 4096 * 4 + 4096, 129, TILE, TILE),  # I = 1408 splits into no 256-wide pairs
])
def test_kernel_family(shape, rows, active, gu_kind, dn_kind):
    gu, dn = plan(layer(**shape), rows, active)
    assert (gu["kind"], dn["kind"]) == (gu_kind, dn_kind), (gu, dn)


def test_float32_layers_take_the_simt_kernels():
    gu, dn = plan(layer(256, 512, 8, 2, dtype=X.F32), 64, 8)
    assert gu["kind"] == dn["kind"] == SIMT


def test_query_validation():
    ly = layer(**MIXTRAL)
    out = (ctypes.c_int32 * 10)()
    L = X.lib()
    assert L.exfold_gemm_plan(ctypes.byref(ly), 64, 4, 256, None) == X.ERR_NULL
    assert L.exfold_gemm_plan(ctypes.byref(ly), -1, 4, 256, out) == X.ERR_SHAPE
    assert L.exfold_gemm_plan(ctypes.byref(ly), 64, 0, 256, out) == X.ERR_SHAPE
    assert L.exfold_gemm_plan(ctypes.byref(ly), 64, 4, 0, out) == X.ERR_SHAPE
    bad = layer(**MIXTRAL, dtype=7)
    assert L.exfold_gemm_plan(ctypes.byref(bad), 64, 4, 256, out) == X.ERR_DTYPE


def _tiles(p, sizes, out_cols, gate_up):
    """Tiles the device-side list holds for these group sizes under plan p."""
    if p["kind"] == SIMT:
        return 0
    n_tiles = out_cols // (p["bn"] // 2 if gate_up else p["bn"])
    if p["kind"] == WIDE:       # 128-row units, one tile per unit and pair of n-tiles
        return int(sum(-(-r // 128) for r in sizes)) * (n_tiles // 2)
    return int(sum(-(-r // p["bm"]) for r in sizes)) * n_tiles * p["ksplit"]


def _splits(rows, groups, rng):
    yield [rows] + [0] * (groups - 1)                     # one busy group
    q, r = divmod(rows, groups)
    yield [q + (i < r) for i in range(groups)]           # even
    if rows >= 129 * groups:                              # every group one row past a 128-row unit
        base = [128 * ((rows // groups - 1) // 128) + 1] * groups
        base[0] += rows - sum(base)
        yield base
    for _ in range(20):
        yield list(rng.multinomial(rows, rng.dirichlet(np.full(groups, 0.3))))


@pytest.mark.parametrize("shape,rows,active", [
    (MIXTRAL, 4096, 8), (MIXTRAL, 20000, 8), (MIXTRAL, 64, 4), (QWEN3, 32768, 128), (QWEN3, 1024, 16),
    (GLM, 4096 * 4 + 4096, 129), (GLM, 64 * 8 + 64, 33),
    (dict(d=384, inter=256, n=8, k=2), 8192, 8), (dict(d=2048, inter=1024, n=8, k=2), 9000, 8),
])
def test_grids_cover_every_split(shape, rows, active):
    ly = layer(**shape)
    groups = shape["n"] + (1 if shape.get("shared") else 0)
    gu, dn = plan(ly, rows, active)
    rng = np.random.default_rng(rows)
    for sizes in _splits(rows, groups, rng):
        assert sum(sizes) == rows
        for p, cols, gate_up in ((gu, shape["inter"], True), (dn, shape["d"], False)):
            need = _tiles(p, sizes, cols, gate_up) + (256 if p["kind"] == WIDE else 0)
            assert p["grid"] >= need, (p, sizes)
