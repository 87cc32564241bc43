"""Seeded synthetic inputs for the folded MoE layer.

This module only draws random numbers and rounds them to the storage dtype.
It holds none of the layer's arithmetic, so both the device library (through
the tests and the benchmark) and the CPU oracle can be fed the same bytes.

Recipe (all configs):
* Generator: numpy ``PCG64`` seeded through ``SeedSequence``; normal draws in
  float32 (``standard_normal(dtype=float32)``), scaled, then rounded to the
  storage dtype (bf16 by round-to-nearest-even, or kept as float32).
* Sub-seeds from the base seed ``s``: weights ``16*s + 0`` (router with
  spawn key (0,); routed expert ``e``: gate/up (1, e, 0), down (1, e, 1);
  shared expert: gate/up (2, 0), down (2, 1)), tokens ``16*s + 1``,
  calibration tokens ``16*s + 2``, router bias ``16*s + 3``.
* Storage format: bf16 tensors are returned as uint16 bit patterns (what the
  device reads); ``widen`` gives the exact float32 values the oracle reads.
* Values: tokens x ~ N(0, 1); every weight ~ N(0, 0.02^2); the skewed router
  adds a per-expert logit bias b ~ N(0, 1) (float32).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

WEIGHT_STD = 0.02


@dataclass(frozen=True)
class LayerShape:
    name: str
    d: int                  # hidden size
    inter: int              # expert intermediate size I
    n_experts: int          # routed experts N
    top_k: int              # router Top-K
    shared_inter: int = 0   # shared-expert intermediate size (0: none)
    dtype: str = "bf16"     # storage dtype of x, y and all weights: "bf16" or "f32"
    router_bias: bool = False
    m_cal: int = 4096       # calibration tokens


@dataclass(frozen=True)
class Workload:
    shape: LayerShape
    phase: str              # "prefill" | "decode" | "dense"
    tokens: int             # T (prefill) or B (decode)
    budget: int             # K' (prefill) or D (decode)
    seed: int = 0
    tags: tuple = field(default_factory=tuple)


TINY = LayerShape("tiny", d=256, inter=512, n_experts=8, top_k=2, dtype="f32", m_cal=512)
MIXTRAL = LayerShape("mixtral-8x7b", d=4096, inter=14336, n_experts=8, top_k=2)
QWEN3 = LayerShape("qwen3-30b-a3b", d=2048, inter=768, n_experts=128, top_k=8, router_bias=True)
QWEN3_DECODE = LayerShape("qwen3-30b-a3b", d=2048, inter=768, n_experts=128, top_k=8)
GLM45 = LayerShape("glm-4.5-air", d=4096, inter=1408, n_experts=128, top_k=8, shared_inter=1408)

WORKLOADS = {
    "tiny_prefill": Workload(TINY, "prefill", 64, 1),
    "mixtral_prefill": Workload(MIXTRAL, "prefill", 4096, 1),
    "mixtral_decode": Workload(MIXTRAL, "decode", 32, 4),
    "qwen3_prefill": Workload(QWEN3, "prefill", 8192, 4),
    **{f"glm_decode_b{b}_d{dd}": Workload(GLM45, "decode", b, dd)
       for b in (16, 64, 256) for dd in (32, 64)},
    **{f"qwen3_decode_b{b}_d{dd}": Workload(QWEN3_DECODE, "decode", b, dd)
       for b in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512) for dd in (16, 32, 64)},
}


def _rng(entropy: int, spawn_key=()) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy, spawn_key=spawn_key)))


_CHUNK = 1 << 22


def _bf16_bits_inplace(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (ties to even) and return the bf16 bit patterns (uint16)."""
    flat = a.reshape(-1).view(np.uint32)
    out = np.empty(flat.size, dtype=np.uint16)
    tmp = np.empty(min(_CHUNK, flat.size), dtype=np.uint32)
    for lo in range(0, flat.size, _CHUNK):
        u = flat[lo:lo + _CHUNK]
        t = tmp[: u.size]
        np.right_shift(u, 16, out=t)
        np.bitwise_and(t, 1, out=t)
        t += np.uint32(0x7FFF)
        u += t
        np.right_shift(u, 16, out=u)
        out[lo:lo + u.size] = u
    return out.reshape(a.shape)


def widen(a: np.ndarray) -> np.ndarray:
    """Storage array -> float32 values (bf16 bit patterns are widened exactly)."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return np.asarray(a, dtype=np.float32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Nearest bf16 values (ties to even) of float32 data, as float32."""
    return widen(_bf16_bits_inplace(np.array(a, dtype=np.float32, copy=True)))


def _draw(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) draws in the storage format: uint16 bf16 bit patterns, or float32."""
    a = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return _bf16_bits_inplace(a) if dtype == "bf16" else a


def router_weight(shape: LayerShape, seed: int = 0) -> np.ndarray:
    """[N, d] router weight in storage format."""
    return _draw(_rng(16 * seed + 0, (0,)), (shape.n_experts, shape.d), WEIGHT_STD, shape.dtype)


def router_bias(shape: LayerShape, seed: int = 0):
    """[N] float32 per-expert logit bias (skewed router), or None."""
    if not shape.router_bias:
        return None
    return _rng(16 * seed + 3).standard_normal(size=shape.n_experts, dtype=np.float32)


def expert_gate_up(shape: LayerShape, e: int, seed: int = 0) -> np.ndarray:
    """[2I, d] (gate rows then up rows) of routed expert e, storage format."""
    return _draw(_rng(16 * seed + 0, (1, e, 0)), (2 * shape.inter, shape.d), WEIGHT_STD, shape.dtype)


def expert_down(shape: LayerShape, e: int, seed: int = 0) -> np.ndarray:
    """[d, I] down projection of routed expert e, storage format."""
    return _draw(_rng(16 * seed + 0, (1, e, 1)), (shape.d, shape.inter), WEIGHT_STD, shape.dtype)


def expert_weights(shape: LayerShape, e: int, seed: int = 0):
    return expert_gate_up(shape, e, seed), expert_down(shape, e, seed)


def shared_weights(shape: LayerShape, seed: int = 0):
    """([2I_s, d], [d, I_s]) of the shared expert in storage format, or (None, None)."""
    if not shape.shared_inter:
        return None, None
    gu = _draw(_rng(16 * seed + 0, (2, 0)), (2 * shape.shared_inter, shape.d), WEIGHT_STD, shape.dtype)
    dn = _draw(_rng(16 * seed + 0, (2, 1)), (shape.d, shape.shared_inter), WEIGHT_STD, shape.dtype)
    return gu, dn


def tokens(shape: LayerShape, n: int, seed: int = 0) -> np.ndarray:
    """[n, d] tokens x ~ N(0, 1), storage format."""
    return _draw(_rng(16 * seed + 1), (n, shape.d), 1.0, shape.dtype)


def calibration_tokens(shape: LayerShape, m: int | None = None, seed: int = 0) -> np.ndarray:
    """[m, d] calibration tokens ~ N(0, 1), storage format."""
    return _draw(_rng(16 * seed + 2), (m or shape.m_cal, shape.d), 1.0, shape.dtype)


def all_expert_weights(shape: LayerShape, seed: int = 0, threads: int = 8):
    """Stacked ([N, 2I, d], [N, d, I]) in storage format, drawn in parallel threads."""
    from concurrent.futures import ThreadPoolExecutor
    sdt = np.uint16 if shape.dtype == "bf16" else np.float32
    gu = np.empty((shape.n_experts, 2 * shape.inter, shape.d), dtype=sdt)
    dn = np.empty((shape.n_experts, shape.d, shape.inter), dtype=sdt)

    def job(arg):
        e, part = arg
        if part == 0:
            gu[e] = expert_gate_up(shape, e, seed)
        else:
            dn[e] = expert_down(shape, e, seed)

    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(job, [(e, p) for e in range(shape.n_experts) for p in (0, 1)]))
    return gu, dn


def synthetic_tables(n_experts: int, seed: int = 0):
    """Seeded stand-in projector tables (S, L [N, N], h [N], float32) for speed and parity runs:
    S ~ N(0, 0.5^2), L ~ U(0, 1) with a zero diagonal and S = 1 on it, h ~ U(0.5, 2)."""
    rng = _rng(16 * seed + 4)
    S = (rng.standard_normal((n_experts, n_experts), dtype=np.float32) * np.float32(0.5))
    L = rng.random((n_experts, n_experts), dtype=np.float32)
    np.fill_diagonal(S, 1.0)
    np.fill_diagonal(L, 0.0)
    h = (np.float32(0.5) + np.float32(1.5) * rng.random(n_experts, dtype=np.float32)).astype(np.float32)
    return S, L, h


# ---------------------------------------------------------------------------
# Directionally aligned experts (a synthetic stand-in for the alignment of
# expert outputs that the paper observes in trained MoE layers): every routed
# expert is one base expert with its own output scale c_e and a perturbation,
#   W_gu[e] = W_gu_base + sigma * N_e,   W_down[e] = c_e * (W_down_base + sigma * M_e),
# with c_e log-uniform in [1/sqrt(spread), sqrt(spread)] (output norms spread
# by the factor `spread`).  sigma = 0 gives exact scalar multiples up to the
# bf16 rounding.  Spawn keys: bases (3, 0) and (3, 1), perturbations (4, e, 0)
# and (4, e, 1), scales (5,).
# ---------------------------------------------------------------------------

def aligned_scales(shape: LayerShape, seed: int = 0, spread: float = 3.0) -> np.ndarray:
    """[N] float64 output scales c_e of the aligned experts."""
    u = _rng(16 * seed + 0, (5,)).random(shape.n_experts)
    return np.exp((u - 0.5) * np.log(spread))


def aligned_expert_weights(shape: LayerShape, seed: int = 0, sigma: float = 0.3, spread: float = 3.0,
                           scales=None):
    """(w_gate_up [N, 2I, d], w_down [N, d, I]) of aligned experts, storage format.

    scales: optional [N] output scales replacing the log-uniform draw."""
    n, d, inter = shape.n_experts, shape.d, shape.inter
    base_gu = _rng(16 * seed + 0, (3, 0)).standard_normal((2 * inter, d), dtype=np.float32) * WEIGHT_STD
    base_dn = _rng(16 * seed + 0, (3, 1)).standard_normal((d, inter), dtype=np.float32) * WEIGHT_STD
    c = aligned_scales(shape, seed, spread) if scales is None else np.asarray(scales, dtype=np.float64)
    gu = np.empty((n, 2 * inter, d), dtype=np.uint16 if shape.dtype == "bf16" else np.float32)
    dn = np.empty((n, d, inter), dtype=gu.dtype)
    for e in range(n):
        g = base_gu + np.float32(sigma * WEIGHT_STD) * _rng(16 * seed + 0, (4, e, 0)).standard_normal(
            base_gu.shape, dtype=np.float32)
        w = (base_dn + np.float32(sigma * WEIGHT_STD) * _rng(16 * seed + 0, (4, e, 1)).standard_normal(
            base_dn.shape, dtype=np.float32)) * np.float32(c[e])
        gu[e] = _bf16_bits_inplace(g) if shape.dtype == "bf16" else g
        dn[e] = _bf16_bits_inplace(w) if shape.dtype == "bf16" else w
    return gu, dn
