"""Shared helpers of the GPU parity tests: device copies of the seeded inputs,
tolerances derived from the arithmetic, and near-tie accounting."""

from __future__ import annotations

import numpy as np
import torch

from oracle import exfold_oracle as O
from paper_2608_24938_amd import exfold as X
from paper_2608_24938_amd import synth

DEV = "cuda:0"
U32 = 2.0 ** -24          # float32 unit roundoff
TOL_Y = {"f32": 1e-4, "bf16": 2e-2}   # max per-token rel-L2 of y


def to_dev(a: np.ndarray) -> torch.Tensor:
    """Storage array -> device tensor (uint16 bf16 bit patterns become torch.bfloat16)."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def from_dev(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return synth.widen(t.view(torch.int16).cpu().numpy().view(np.uint16))
    return t.cpu().numpy()


class LayerPair:
    """The same seeded layer on the device (binding) and for the oracle (float32 views)."""

    def __init__(self, shape: synth.LayerShape, seed: int = 0, lazy_oracle: bool = False):
        self.shape = shape
        wr = synth.router_weight(shape, seed)
        bias = synth.router_bias(shape, seed)
        gu, dn = synth.all_expert_weights(shape, seed)
        sgu, sdn = synth.shared_weights(shape, seed)
        self.dev = X.Layer(w_router=to_dev(wr), w_gate_up=to_dev(gu), w_down=to_dev(dn), top_k=shape.top_k,
                           router_bias=None if bias is None else to_dev(bias),
                           ws_gate_up=None if sgu is None else to_dev(sgu),
                           ws_down=None if sdn is None else to_dev(sdn))
        self.storage = dict(wr=wr, gu=gu, dn=dn, bias=bias, sgu=sgu, sdn=sdn)
        widen = synth.widen
        self.ref = O.Layer(w_router=widen(wr),
                           w_gate_up=(lambda e: widen(gu[e])) if lazy_oracle else widen(gu),
                           w_down=(lambda e: widen(dn[e])) if lazy_oracle else widen(dn),
                           router_bias=bias,
                           ws_gate_up=None if sgu is None else widen(sgu),
                           ws_down=None if sdn is None else widen(sdn))


def logits_bound(x: np.ndarray, w_router: np.ndarray, bias, d: int) -> np.ndarray:
    """Rounding bound of a float32 dot product of length d plus a bias add:
    gamma_{d+2} * (sum |x_j w_j| + |b|), valid for any summation order."""
    n = d + 2
    gamma = n * U32 / (1 - n * U32)
    mag = np.abs(x.astype(np.float64)) @ np.abs(w_router.astype(np.float64)).T
    if bias is not None:
        mag = mag + np.abs(bias.astype(np.float64))[None, :]
    return gamma * mag


def per_token_rel_l2(y: np.ndarray, ref: np.ndarray) -> np.ndarray:
    y = y.astype(np.float64)
    ref = ref.astype(np.float64)
    return np.linalg.norm(y - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)


def topk_near_tie(logits64: np.ndarray, bound: np.ndarray, k: int) -> np.ndarray:
    """Tokens whose Top-K set or order is decided by a margin within the rounding bound."""
    t, n = logits64.shape
    out = np.zeros(t, dtype=bool)
    for i in range(t):
        order = np.lexsort((np.arange(n), -logits64[i]))
        r = logits64[i][order]
        b = bound[i][order]
        lim = min(k + 1, n)
        gaps = r[: lim - 1] - r[1:lim]
        out[i] = np.any(gaps <= b[: lim - 1] + b[1:lim])
    return out


def sync():
    torch.cuda.synchronize()
