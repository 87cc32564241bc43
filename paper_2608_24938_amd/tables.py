"""Persistence of calibrated projector tables.

The projector tables are computed once per model on calibration tokens and then
kept fixed (Sec. 4.2; the calibrated state is two N x N float32 tables per MoE
layer, Table 3's storage arithmetic, plus the per-expert output norms h).  This
module writes and reads them as one little-endian file:

    header  magic b"EXFT", version u32, n_layers u32, n_experts u32,
            lambda f32, clip f32, mode u32 (0 co-routed, 1 common input),
            flags u32 (bit 0: diagonal maps present), d u32 (diagonal maps only)
    per layer: S [N, N] f32, L [N, N] f32, h [N] f32
               (+ Dg [N, N, d] f32 with the diagonal flag)

Everything is plain host memory (numpy); device tensors are copied to the host
first.  Reading checks the magic, version, sizes and the file length, and
raises ValueError on any mismatch.
"""

from __future__ import annotations

import struct
from dataclasses import dataclass

import numpy as np

MAGIC = b"EXFT"
VERSION = 1
_HEADER = struct.Struct("<4sIIIffIII")
MODES = {"corouted": 0, "common": 1}          # the binding's calibration mode names
_ALIASES = {"common_input": "common", "co-routed": "corouted"}


@dataclass
class LayerTables:
    S: np.ndarray            # [N, N] float32, row = source expert
    L: np.ndarray            # [N, N] float32
    h: np.ndarray            # [N] float32
    Dg: np.ndarray | None = None  # [N, N, d] float32 diagonal maps, or None


def _host(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def table_bytes(n_layers: int, n_experts: int, d: int = 0) -> int:
    """File size: header + per layer two N x N tables, h, and optionally the diagonal maps."""
    per = 2 * n_experts * n_experts * 4 + n_experts * 4 + n_experts * n_experts * d * 4
    return _HEADER.size + n_layers * per


def save_tables(path: str, layers, lam: float = 1e-3, clip: float = 4.0, mode: str = "corouted") -> int:
    """Write the tables of every layer (a list of LayerTables or (S, L, h[, Dg]) tuples); returns bytes."""
    rows = [t if isinstance(t, LayerTables) else LayerTables(*t) for t in layers]
    if not rows:
        raise ValueError("no layers")
    n = _host(rows[0].S).shape[0]
    diag = rows[0].Dg is not None
    d = _host(rows[0].Dg).shape[2] if diag else 0
    mode = _ALIASES.get(mode, mode)
    if mode not in MODES:
        raise ValueError(f"unknown calibration mode {mode!r}")
    with open(path, "wb") as f:
        f.write(_HEADER.pack(MAGIC, VERSION, len(rows), n, float(lam), float(clip), MODES[mode], int(diag), d))
        for i, t in enumerate(rows):
            S, L, h = _host(t.S), _host(t.L), _host(t.h)
            if S.shape != (n, n) or L.shape != (n, n) or h.shape != (n,):
                raise ValueError(f"layer {i}: shapes {S.shape}, {L.shape}, {h.shape} for N = {n}")
            if (t.Dg is not None) != diag:
                raise ValueError(f"layer {i}: diagonal maps present in some layers only")
            f.write(S.astype("<f4").tobytes())
            f.write(L.astype("<f4").tobytes())
            f.write(h.astype("<f4").tobytes())
            if diag:
                Dg = _host(t.Dg)
                if Dg.shape != (n, n, d):
                    raise ValueError(f"layer {i}: diagonal maps {Dg.shape}, expected {(n, n, d)}")
                f.write(Dg.astype("<f4").tobytes())
    return table_bytes(len(rows), n, d)


def load_tables(path: str):
    """Read a table file: (list of LayerTables, metadata dict)."""
    with open(path, "rb") as f:
        raw = f.read()
    if len(raw) < _HEADER.size:
        raise ValueError("file shorter than the header")
    magic, version, n_layers, n, lam, clip, mode, flags, d = _HEADER.unpack_from(raw, 0)
    if magic != MAGIC:
        raise ValueError("not a projector table file")
    if version != VERSION:
        raise ValueError(f"unsupported table file version {version}")
    diag = bool(flags & 1)
    if len(raw) != table_bytes(n_layers, n, d if diag else 0):
        raise ValueError(f"file length {len(raw)} does not match {n_layers} layers of N = {n}")
    off = _HEADER.size
    out = []

    def take(count, shape):
        nonlocal off
        a = np.frombuffer(raw, dtype="<f4", count=count, offset=off).reshape(shape).astype(np.float32)
        off += count * 4
        return a

    for _ in range(n_layers):
        S = take(n * n, (n, n))
        L = take(n * n, (n, n))
        h = take(n, (n,))
        Dg = take(n * n * d, (n, n, d)) if diag else None
        out.append(LayerTables(S, L, h, Dg))
    inv = {v: k for k, v in MODES.items()}
    return out, {"lambda": lam, "clip": clip, "mode": inv.get(mode, mode), "n_experts": n, "d": d}
