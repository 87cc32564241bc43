"""ctypes binding of libexfold (the C-ABI in include/exfold.h).

Argument marshalling only: torch supplies device memory and the current
stream; every step of the layer runs in the library's HIP kernels.  The
library is loaded on first use; a missing library raises ``RuntimeError``
(there is no fallback path).
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libexfold.so")
_lib = None

(OK, ERR_NULL, ERR_SHAPE, ERR_BUDGET, ERR_DTYPE, ERR_WORKSPACE, ERR_DEVICE, ERR_UNSUPPORTED, ERR_ARG, ERR_ALIGN,
 ERR_SCRATCH) = range(11)
SCRATCH_BYTES = 64 << 20   # EXFOLD_SCRATCH_BYTES
F32, BF16 = 0, 1
PHASE = {"dense": 0, "prefill": 1, "decode": 2, "decode_static": 3, "prefill_diag": 4}
CAL_MODE = {"corouted": 0, "common": 1}

EXPORTED = [
    "exfold_select_prefill", "exfold_select_decode_pool", "exfold_fold_gates", "exfold_static_pool",
    "exfold_moe_workspace_size", "exfold_moe_forward", "exfold_moe_forward_scratch",
    "exfold_execute_workspace_size",
    "exfold_moe_execute", "exfold_calibrate_workspace_size", "exfold_calibrate_projectors",
    "exfold_calibrate_diagonal",
    "exfold_status_str", "exfold_gemm_plan",
]


class ExfoldError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: status {status} ({status_str(status)})")


class _Layer(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int64), ("inter", ctypes.c_int64), ("n_experts", ctypes.c_int64),
                ("top_k", ctypes.c_int64), ("shared_inter", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("w_router", ctypes.c_void_p), ("router_bias", ctypes.c_void_p),
                ("w_gate_up", ctypes.c_void_p), ("w_down", ctypes.c_void_p),
                ("ws_gate_up", ctypes.c_void_p), ("ws_down", ctypes.c_void_p)]


class _Tables(ctypes.Structure):
    _fields_ = [("S", ctypes.c_void_p), ("L", ctypes.c_void_p), ("h", ctypes.c_void_p),
                ("tgt", ctypes.c_void_p), ("scl", ctypes.c_void_p), ("loss_cap", ctypes.c_float),
                ("fold_flags", ctypes.c_int32), ("Dg", ctypes.c_void_p)]


FOLD_LOSS_CAP, FOLD_RENORM, FOLD_CONFIDENCE = 1, 2, 4


def fold_opts(loss_cap=None, renorm=False, confidence=False):
    """(loss_cap, fold_flags) of the prefill fold safeguards (EXFOLD_FOLD_* in the header)."""
    flags = (FOLD_LOSS_CAP if loss_cap is not None else 0) | (FOLD_RENORM if renorm else 0) | \
        (FOLD_CONFIDENCE if confidence else 0)
    return (0.0 if loss_cap is None else float(loss_cap)), flags


_DEBUG_FIELDS = ["logits", "topk_ids", "topk_w", "keep", "pool", "pool_size", "tgt_ids", "tgt_scale",
                 "fold_ids", "fold_w", "offsets", "row_slot"]


N_EVENTS = 7
EVENT_NAMES = ["start", "router", "fold", "permute", "gate_up", "down", "end"]


class _Debug(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _DEBUG_FIELDS] + [("events", ctypes.c_void_p)]


def lib() -> ctypes.CDLL:
    """Load libexfold.so (built in-tree by paper_2608_24938_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"libexfold.so is not built ({_LIB_PATH}); run paper_2608_24938_amd.build")
        L = ctypes.CDLL(_LIB_PATH)
        i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
        dbl = ctypes.c_double
        sig = {
            "exfold_select_prefill": (i32, [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp]),
            "exfold_select_decode_pool": (i32, [vp, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp]),
            "exfold_fold_gates": (i32, [i32, i64, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                        ctypes.c_float, i32, vp]),
            "exfold_static_pool": (i32, [vp, i64, i64, vp, vp, vp, vp, vp, vp, vp]),
            "exfold_moe_workspace_size": (sz, [vp, i64, i32, i64]),
            "exfold_moe_forward": (i32, [vp, vp, vp, i64, i32, i64, vp, vp, vp, sz, vp]),
            "exfold_moe_forward_scratch": (i32, [vp, vp, vp, i64, i32, i64, vp, vp, vp]),
            "exfold_execute_workspace_size": (sz, [vp, i64, i64]),
            "exfold_moe_execute": (i32, [vp, vp, i64, i64, vp, vp, vp, vp, vp, sz, vp]),
            "exfold_calibrate_workspace_size": (sz, [vp, i64, i32]),
            "exfold_calibrate_projectors": (i32, [vp, vp, i64, dbl, dbl, i32, vp, vp, vp, vp, vp, sz, vp]),
            "exfold_calibrate_diagonal": (i32, [vp, vp, i64, dbl, i32, vp, vp, vp, sz, vp]),
            "exfold_status_str": (ctypes.c_char_p, [i32]),
            "exfold_gemm_plan": (i32, [vp, i64, i64, i32, vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_str(status: int) -> str:
    return lib().exfold_status_str(status).decode()


def _check(status: int, where: str):
    if status != OK:
        raise ExfoldError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t, dtype, shape, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)} on the GPU, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


@dataclass
class Layer:
    """Device weights of one MoE layer (bf16 weights are torch.bfloat16 tensors)."""
    w_router: torch.Tensor          # [N, d]
    w_gate_up: torch.Tensor         # [N, 2I, d]
    w_down: torch.Tensor            # [N, d, I]
    top_k: int
    router_bias: torch.Tensor | None = None   # [N] float32
    ws_gate_up: torch.Tensor | None = None    # [2I_s, d]
    ws_down: torch.Tensor | None = None       # [d, I_s]

    @property
    def n_experts(self):
        return self.w_router.shape[0]

    @property
    def d(self):
        return self.w_router.shape[1]

    @property
    def inter(self):
        return self.w_down.shape[2]

    @property
    def dtype(self):
        return self.w_router.dtype

    def struct(self) -> _Layer:
        code = {torch.bfloat16: BF16, torch.float32: F32}[self.dtype]
        return _Layer(self.d, self.inter, self.n_experts, self.top_k,
                      0 if self.ws_down is None else self.ws_down.shape[1], code, 0,
                      self.w_router.data_ptr(), None if self.router_bias is None else self.router_bias.data_ptr(),
                      self.w_gate_up.data_ptr(), self.w_down.data_ptr(),
                      None if self.ws_gate_up is None else self.ws_gate_up.data_ptr(),
                      None if self.ws_down is None else self.ws_down.data_ptr())


def _workspace(nbytes: int, device, stream=None) -> torch.Tensor:
    """Temporary workspace for one call.  torch's caching allocator returns 256-byte aligned
    blocks (512 in practice).  When the call runs on another stream than the current one, the
    block is tied to that stream too (record_stream), so the allocator does not hand it out
    again while the call's kernels may still use it."""
    ws = torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)
    if stream is not None:
        ws.record_stream(stream)
    return ws


def select_prefill(h, k_pre, logits=None, topk_ids=None, topk_w=None, top_k=None, stream=None):
    """Top-K routes (from logits, or given) and the prefill keep mask. Returns (ids, w, keep)."""
    if logits is not None:
        T, N = logits.shape
        K = top_k
        topk_ids = torch.empty((T, K), dtype=torch.int32, device=logits.device)
        topk_w = torch.empty((T, K), dtype=torch.float32, device=logits.device)
    else:
        T, K = topk_ids.shape
        N = h.shape[0]
    keep = torch.empty((T, K), dtype=torch.uint8, device=h.device)
    _check(lib().exfold_select_prefill(_ptr(logits), T, N, K, k_pre, _ptr(h), _ptr(topk_ids), _ptr(topk_w),
                                       _ptr(keep), _stream(stream)), "exfold_select_prefill")
    return topk_ids, topk_w, keep


def select_decode_pool(h, budget, logits=None, topk_ids=None, topk_w=None, top_k=None, stream=None):
    """Top-K routes (from logits, or given) and the decode pool. Returns (ids, w, pool, pool_size)."""
    N = h.shape[0]
    if logits is not None:
        B = logits.shape[0]
        K = top_k
        topk_ids = torch.empty((B, K), dtype=torch.int32, device=logits.device)
        topk_w = torch.empty((B, K), dtype=torch.float32, device=logits.device)
    else:
        B, K = topk_ids.shape
    pool = torch.empty((min(budget, N),), dtype=torch.int32, device=h.device)
    pool_size = torch.empty((1,), dtype=torch.int32, device=h.device)
    _check(lib().exfold_select_decode_pool(_ptr(logits), B, N, K, budget, _ptr(h), _ptr(topk_ids), _ptr(topk_w),
                                           _ptr(pool), _ptr(pool_size), _stream(stream)),
           "exfold_select_decode_pool")
    return topk_ids, topk_w, pool, pool_size


def fold_gates(phase, budget, topk_ids, topk_w, S, L, keep=None, pool=None, pool_size=None, tables=False,
               stream=None, loss_cap=None, renorm=False, confidence=False):
    """Fold route metadata. Returns (out_ids, out_w) or (out_ids, out_w, tgt, scl) with tables=True.

    loss_cap/renorm/confidence: the prefill safeguards (see fold_opts)."""
    T, K = topk_ids.shape
    N = S.shape[0]
    ph = PHASE[phase]
    k_out = min(budget, K) if phase == "prefill" else K
    dev = S.device
    out_ids = torch.empty((T, k_out), dtype=torch.int32, device=dev)
    out_w = torch.empty((T, k_out), dtype=torch.float32, device=dev)
    tgt = torch.empty((N,), dtype=torch.int32, device=dev) if tables else None
    scl = torch.empty((N,), dtype=torch.float32, device=dev) if tables else None
    _check(lib().exfold_fold_gates(ph, T, N, K, budget, _ptr(topk_ids), _ptr(topk_w), _ptr(keep), _ptr(pool),
                                   _ptr(pool_size), _ptr(S), _ptr(L), _ptr(out_ids), _ptr(out_w), _ptr(tgt),
                                   _ptr(scl), *fold_opts(loss_cap, renorm, confidence), _stream(stream)),
           "exfold_fold_gates")
    return (out_ids, out_w, tgt, scl) if tables else (out_ids, out_w)


def static_pool(h, budget, S, L, stream=None):
    """Static decode pool TopK(h, D) and its per-source tables. Returns (pool, pool_size, tgt, scl)."""
    N = h.shape[0]
    dev = h.device
    pool = torch.empty((min(budget, N),), dtype=torch.int32, device=dev)
    pool_size = torch.empty((1,), dtype=torch.int32, device=dev)
    tgt = torch.empty((N,), dtype=torch.int32, device=dev)
    scl = torch.empty((N,), dtype=torch.float32, device=dev)
    _check(lib().exfold_static_pool(_ptr(h), N, budget, _ptr(S), _ptr(L), _ptr(pool), _ptr(pool_size), _ptr(tgt),
                                    _ptr(scl), _stream(stream)), "exfold_static_pool")
    return pool, pool_size, tgt, scl


def moe_workspace_size(layer: Layer, T: int, phase: str, budget: int) -> int:
    ls = layer.struct()
    n = lib().exfold_moe_workspace_size(ctypes.byref(ls), T, PHASE[phase], budget)
    if n == 0 and T > 0:
        raise ValueError("invalid layer/shape for exfold_moe_forward")
    return n


def debug_buffers(layer: Layer, T: int, phase: str, budget: int, device) -> dict:
    """Device buffers for every intermediate of the forward (see exfold_debug)."""
    N, K = layer.n_experts, layer.top_k
    k_out = min(budget, K) if phase == "prefill" else K
    R = T * k_out
    i32, f32 = torch.int32, torch.float32
    return {
        "logits": torch.empty((T, N), dtype=f32, device=device),
        "topk_ids": torch.empty((T, K), dtype=i32, device=device),
        "topk_w": torch.empty((T, K), dtype=f32, device=device),
        "keep": torch.empty((T, K), dtype=torch.uint8, device=device),
        "pool": torch.empty((max(1, min(budget, N)),), dtype=i32, device=device),
        "pool_size": torch.empty((1,), dtype=i32, device=device),
        "tgt_ids": torch.empty((N,), dtype=i32, device=device),
        "tgt_scale": torch.empty((N,), dtype=f32, device=device),
        "fold_ids": torch.empty((T, k_out), dtype=i32, device=device),
        "fold_w": torch.empty((T, k_out), dtype=f32, device=device),
        "offsets": torch.empty((N + 2,), dtype=i32, device=device),
        "row_slot": torch.empty((R + (T if layer.ws_down is not None else 0),), dtype=i32, device=device),
    }


def moe_forward(layer: Layer, x, phase: str = "dense", budget: int = 0, S=None, L=None, h=None, y=None,
                debug: dict | None = None, workspace=None, stream=None, events=None, static_tables=None,
                safeguards: dict | None = None, diag=None):
    """Folded MoE layer forward; returns y [T, d] (dtype of the layer).

    static_tables: (tgt, scl) from static_pool, for phase "decode_static".
    safeguards: prefill fold safeguards, keyword arguments of fold_opts.
    diag: [N, N, d] diagonal maps from calibrate_diagonal, for phase "prefill_diag" (L is then the
    diagonal loss table).
    events: optional ctypes array of N_EVENTS hipEvent_t handles recorded at the stage boundaries."""
    T = x.shape[0]
    _need(x, layer.dtype, (T, layer.d), "x")
    if y is None:
        y = torch.empty_like(x)
    ls = layer.struct()
    tgt, scl = static_tables if static_tables is not None else (None, None)
    cap, flags = fold_opts(**(safeguards or {}))
    tb = _Tables(_ptr(S), _ptr(L), _ptr(h), _ptr(tgt), _ptr(scl), cap, flags, _ptr(diag)) \
        if (S is not None or L is not None or tgt is not None) else None
    dbg = None
    if debug is not None or events is not None:
        debug = debug or {}
        dbg = _Debug(*[_ptr(debug.get(f)) for f in _DEBUG_FIELDS],
                     None if events is None else ctypes.cast(events, ctypes.c_void_p))
    need = lib().exfold_moe_workspace_size(ctypes.byref(ls), T, PHASE[phase], budget)
    if workspace is None:
        workspace = _workspace(need, x.device, stream)
    _check(lib().exfold_moe_forward(ctypes.byref(ls), None if tb is None else ctypes.byref(tb), _ptr(x), T,
                                    PHASE[phase], budget, _ptr(y), None if dbg is None else ctypes.byref(dbg),
                                    _ptr(workspace), workspace.numel(), _stream(stream)), "exfold_moe_forward")
    return y


def moe_forward_scratch(layer: Layer, x, phase: str = "dense", budget: int = 0, S=None, L=None, h=None, y=None,
                        debug: dict | None = None, stream=None, static_tables=None,
                        safeguards: dict | None = None, diag=None):
    """moe_forward on the library's static scratch (exfold_moe_forward_scratch): no workspace is
    allocated; y must be given by callers that cannot allocate (otherwise it is created here)."""
    T = x.shape[0]
    _need(x, layer.dtype, (T, layer.d), "x")
    if y is None:
        y = torch.empty_like(x)
    ls = layer.struct()
    tgt, scl = static_tables if static_tables is not None else (None, None)
    cap, flags = fold_opts(**(safeguards or {}))
    tb = _Tables(_ptr(S), _ptr(L), _ptr(h), _ptr(tgt), _ptr(scl), cap, flags, _ptr(diag)) \
        if (S is not None or L is not None or tgt is not None) else None
    dbg = None
    if debug is not None:
        dbg = _Debug(*[_ptr(debug.get(f)) for f in _DEBUG_FIELDS], None)
    _check(lib().exfold_moe_forward_scratch(ctypes.byref(ls), None if tb is None else ctypes.byref(tb), _ptr(x), T,
                                            PHASE[phase], budget, _ptr(y),
                                            None if dbg is None else ctypes.byref(dbg), _stream(stream)),
           "exfold_moe_forward_scratch")
    return y


def moe_execute(layer: Layer, x, route_ids, route_w, y=None, debug: dict | None = None, stream=None):
    """Run the experts on given routes [T, K_out] and combine; returns y."""
    T, k_out = route_ids.shape
    if y is None:
        y = torch.empty_like(x)
    ls = layer.struct()
    dbg = None
    if debug is not None:
        dbg = _Debug(*[_ptr(debug.get(f)) for f in _DEBUG_FIELDS], None)
    need = lib().exfold_execute_workspace_size(ctypes.byref(ls), T, k_out)
    ws = _workspace(need, x.device, stream)
    _check(lib().exfold_moe_execute(ctypes.byref(ls), _ptr(x), T, k_out, _ptr(route_ids), _ptr(route_w), _ptr(y),
                                    None if dbg is None else ctypes.byref(dbg), _ptr(ws), ws.numel(),
                                    _stream(stream)), "exfold_moe_execute")
    return y


def calibrate_projectors(layer: Layer, x_cal, lam: float = 1e-3, clip: float = 4.0, mode: str = "corouted",
                         with_stats: bool = False, stream=None):
    """Projector calibration; returns (S, L, h) float32 device tensors (+ stats [N,N,4] float64)."""
    m = x_cal.shape[0]
    N = layer.n_experts
    dev = x_cal.device
    ls = layer.struct()
    S = torch.empty((N, N), dtype=torch.float32, device=dev)
    L = torch.empty((N, N), dtype=torch.float32, device=dev)
    h = torch.empty((N,), dtype=torch.float32, device=dev)
    stats = torch.empty((N, N, 4), dtype=torch.float64, device=dev) if with_stats else None
    need = lib().exfold_calibrate_workspace_size(ctypes.byref(ls), m, CAL_MODE[mode])
    ws = _workspace(need, dev, stream)
    _check(lib().exfold_calibrate_projectors(ctypes.byref(ls), _ptr(x_cal), m, lam, clip, CAL_MODE[mode], _ptr(S),
                                             _ptr(L), _ptr(h), _ptr(stats), _ptr(ws), ws.numel(), _stream(stream)),
           "exfold_calibrate_projectors")
    return (S, L, h, stats) if with_stats else (S, L, h)


def calibrate_diagonal(layer: Layer, x_cal, lam: float = 1e-3, mode: str = "corouted", stream=None):
    """Diagonal projector calibration; returns (Dg [N, N, d], Ld [N, N]) float32 device tensors."""
    m = x_cal.shape[0]
    N, d = layer.n_experts, layer.d
    dev = x_cal.device
    ls = layer.struct()
    Dg = torch.empty((N, N, d), dtype=torch.float32, device=dev)
    Ld = torch.empty((N, N), dtype=torch.float32, device=dev)
    need = lib().exfold_calibrate_workspace_size(ctypes.byref(ls), m, CAL_MODE[mode])
    ws = _workspace(need, dev, stream)
    _check(lib().exfold_calibrate_diagonal(ctypes.byref(ls), _ptr(x_cal), m, lam, CAL_MODE[mode], _ptr(Dg), _ptr(Ld),
                                           _ptr(ws), ws.numel(), _stream(stream)), "exfold_calibrate_diagonal")
    return Dg, Ld
