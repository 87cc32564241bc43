"""Projector-table files: exact round trip, the storage arithmetic, and rejection of bad files."""

import numpy as np
import pytest

from oracle import exfold_oracle as O
from paper_2608_24938_amd import synth
from paper_2608_24938_amd.tables import LayerTables, load_tables, save_tables, table_bytes


def _layers(n_layers, n, d=0, seed=0):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n_layers):
        S = rng.standard_normal((n, n)).astype(np.float32)
        L = rng.random((n, n)).astype(np.float32)
        L[0, 1] = np.float32(1e30)                     # an unobserved pair survives as is
        h = rng.random(n).astype(np.float32)
        Dg = rng.standard_normal((n, n, d)).astype(np.float32) if d else None
        out.append(LayerTables(S, L, h, Dg))
    return out


@pytest.mark.parametrize("d", [0, 16])
def test_round_trip_is_bitwise(tmp_path, d):
    layers = _layers(3, 8, d)
    path = tmp_path / "t.bin"
    nbytes = save_tables(str(path), layers, lam=1e-3, clip=4.0, mode="common")
    assert path.stat().st_size == nbytes
    back, meta = load_tables(str(path))
    assert meta == {"lambda": np.float32(1e-3), "clip": 4.0, "mode": "common", "n_experts": 8, "d": d}
    for a, b in zip(layers, back):
        for f in ("S", "L", "h"):
            np.testing.assert_array_equal(getattr(a, f).view(np.uint32), getattr(b, f).view(np.uint32))
        if d:
            np.testing.assert_array_equal(a.Dg.view(np.uint32), b.Dg.view(np.uint32))
        else:
            assert b.Dg is None


def test_storage_matches_the_two_table_arithmetic():
    # 48 layers of N = 128: two N x N float32 tables per layer are 6.00 MiB (the oracle's storage
    # count); the file adds h (N floats per layer) and a fixed header
    n_layers, n = 48, 128
    tables_only = O.table_storage_bytes(n_layers, n, "pair")
    assert tables_only == 6 * 1024 * 1024
    assert table_bytes(n_layers, n) == tables_only + n_layers * n * 4 + 36


def test_oracle_calibration_round_trips(tmp_path):
    shape = synth.TINY
    gu, dn = synth.all_expert_weights(shape, 0)
    layer = O.Layer(w_router=synth.router_weight(shape, 0), w_gate_up=gu, w_down=dn)
    x = synth.widen(synth.calibration_tokens(shape, 64, 0))
    S, L, h = O.calibrate(layer, x, shape.top_k)[:3]
    path = tmp_path / "cal.bin"
    save_tables(str(path), [(S, L, h)])
    (t,), _ = load_tables(str(path))
    np.testing.assert_array_equal(t.S, np.asarray(S, dtype=np.float32))
    np.testing.assert_array_equal(t.L, np.asarray(L, dtype=np.float32))


@pytest.mark.parametrize("damage", ["magic", "version", "truncated", "extra"])
def test_bad_files_are_rejected(tmp_path, damage):
    path = tmp_path / "t.bin"
    save_tables(str(path), _layers(2, 4))
    raw = bytearray(path.read_bytes())
    if damage == "magic":
        raw[0:4] = b"XXXX"
    elif damage == "version":
        raw[4] = 9
    elif damage == "truncated":
        raw = raw[:-4]
    else:
        raw += b"\0\0\0\0"
    path.write_bytes(bytes(raw))
    with pytest.raises(ValueError):
        load_tables(str(path))


def test_inconsistent_layers_are_rejected(tmp_path):
    a, b = _layers(1, 4)[0], _layers(1, 5)[0]
    with pytest.raises(ValueError):
        save_tables(str(tmp_path / "t.bin"), [a, b])
    with pytest.raises(ValueError):
        save_tables(str(tmp_path / "t.bin"), [a], mode="other")


def test_mode_names_are_the_bindings(tmp_path):
    # the calibration mode strings of exfold.calibrate_projectors are accepted as they are
    from paper_2608_24938_amd import exfold as X
    for mode in X.CAL_MODE:
        save_tables(str(tmp_path / "m.bin"), _layers(1, 4), mode=mode)
        assert load_tables(str(tmp_path / "m.bin"))[1]["mode"] == mode
    save_tables(str(tmp_path / "m.bin"), _layers(1, 4), mode="common_input")
    assert load_tables(str(tmp_path / "m.bin"))[1]["mode"] == "common"


@pytest.mark.gpu
def test_calibrate_save_load_forward(tmp_path):
    """Tables calibrated on the device, written, read back and used: the forward with the loaded
    tables is bit-identical to the forward with the tables as calibrated."""
    import torch
    from paper_2608_24938_amd import exfold as X

    from .gpu_common import LayerPair, sync, to_dev
    shape = synth.LayerShape("tables-bf16", d=256, inter=128, n_experts=32, top_k=4, dtype="bf16")
    lp = LayerPair(shape, seed=3)
    for mode in X.CAL_MODE:
        S, L, h = X.calibrate_projectors(lp.dev, to_dev(synth.calibration_tokens(shape, 512, 3)), mode=mode)
        path = tmp_path / f"{mode}.bin"
        save_tables(str(path), [(S, L, h)], mode=mode)
        (t,), meta = load_tables(str(path))
        assert meta["mode"] == mode
        x = to_dev(synth.tokens(shape, 200, 3))
        for phase, budget in (("prefill", 2), ("decode", 8)):
            y0 = X.moe_forward(lp.dev, x, phase, budget, S, L, h)
            y1 = X.moe_forward(lp.dev, x, phase, budget, to_dev(t.S), to_dev(t.L), to_dev(t.h))
            sync()
            assert torch.equal(y0.view(torch.int16), y1.view(torch.int16)), (mode, phase)
