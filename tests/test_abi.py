"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and host-side validation returns the documented status codes
before anything is enqueued (no compute call is made here)."""

import ctypes
import os
import re

import pytest

from paper_2608_24938_amd import exfold as X

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "exfold.h")

FAKE = 0x10000  # never dereferenced: every call below fails validation first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(exfold_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = X.lib()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert sorted(names) == sorted(X.EXPORTED)


def test_status_strings():
    for code in range(11):
        assert X.status_str(code)
    assert X.status_str(0) == "ok"


def layer(**kw):
    base = dict(d=256, inter=512, n_experts=8, top_k=2, shared_inter=0, dtype=X.F32)
    base.update(kw)
    ptrs = dict(w_router=FAKE, router_bias=None, w_gate_up=FAKE, w_down=FAKE, ws_gate_up=None, ws_down=None)
    ptrs.update({k: v for k, v in kw.items() if k in ptrs})
    return X._Layer(base["d"], base["inter"], base["n_experts"], base["top_k"], base["shared_inter"],
                    base["dtype"], 0, ptrs["w_router"], ptrs["router_bias"], ptrs["w_gate_up"], ptrs["w_down"],
                    ptrs["ws_gate_up"], ptrs["ws_down"])


def ws_size(ly, T=64, phase=1, budget=1):
    return X.lib().exfold_moe_workspace_size(ctypes.byref(ly), T, phase, budget)


def forward(ly, T=64, phase=1, budget=1, tables=True, ws_bytes=None, x=FAKE, y=FAKE, ws=FAKE * 16,
            static=(FAKE, FAKE), flags=(0.0, 0), diag=FAKE):
    tb = X._Tables(FAKE, FAKE, FAKE, *static, *flags, diag)
    if ws_bytes is None:
        ws_bytes = 0
    return X.lib().exfold_moe_forward(ctypes.byref(ly), ctypes.byref(tb) if tables else None, x, T, phase,
                                      budget, y, None, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), X.ERR_DTYPE),
    (dict(w_router=None), X.ERR_NULL),
    (dict(w_down=None), X.ERR_NULL),
    (dict(top_k=9), X.ERR_SHAPE),
    (dict(top_k=0), X.ERR_SHAPE),
    (dict(d=-128), X.ERR_SHAPE),
    (dict(n_experts=300, top_k=2), X.ERR_UNSUPPORTED),
    (dict(n_experts=32, top_k=17), X.ERR_UNSUPPORTED),
    (dict(d=200), X.ERR_UNSUPPORTED),
    (dict(inter=100), X.ERR_UNSUPPORTED),
    (dict(shared_inter=512), X.ERR_NULL),
    (dict(shared_inter=256, ws_gate_up=FAKE, ws_down=FAKE), X.ERR_UNSUPPORTED),
    (dict(w_gate_up=FAKE + 8), X.ERR_ALIGN),
    (dict(w_router=FAKE + 2), X.ERR_ALIGN),
    (dict(shared_inter=512, ws_gate_up=FAKE, ws_down=FAKE + 4), X.ERR_ALIGN),
])
def test_layer_validation(kw, code):
    ly = layer(**kw)
    assert forward(ly) == code
    assert ws_size(ly) == 0


def test_forward_validation_codes():
    ly = layer()
    assert forward(ly, phase=5) == X.ERR_ARG
    assert forward(ly, budget=0) == X.ERR_BUDGET
    assert forward(ly, phase=2, budget=0) == X.ERR_BUDGET
    assert forward(ly, T=-1) == X.ERR_SHAPE
    assert forward(ly, tables=False) == X.ERR_NULL
    assert forward(ly, x=None) == X.ERR_NULL
    assert forward(ly, x=FAKE + 8) == X.ERR_ALIGN        # 16-byte vectors move x and y
    assert forward(ly, y=FAKE + 2) == X.ERR_ALIGN
    need = ws_size(ly)
    assert need > 0
    assert forward(ly, ws_bytes=need - 1) == X.ERR_WORKSPACE
    assert forward(ly, ws_bytes=need, ws=FAKE * 16 + 8) == X.ERR_WORKSPACE   # misaligned
    assert forward(ly, ws_bytes=need, ws=None) == X.ERR_NULL
    assert forward(ly, T=0) == X.OK                                           # empty batch: no-op
    # dense phase needs no tables
    assert forward(ly, phase=0, tables=False, ws_bytes=0) == X.ERR_WORKSPACE
    # the static decode phase needs the precomputed per-source tables
    assert forward(ly, phase=3, budget=4, static=(None, None)) == X.ERR_NULL
    assert forward(ly, phase=3, budget=4, static=(FAKE, None)) == X.ERR_NULL
    assert forward(ly, phase=3, budget=0) == X.ERR_BUDGET
    assert forward(ly, phase=3, budget=4, ws_bytes=0) == X.ERR_WORKSPACE
    # unknown safeguard bits or a NaN loss cap
    assert forward(ly, flags=(0.0, 16)) == X.ERR_ARG
    assert forward(ly, flags=(float("nan"), 1)) == X.ERR_ARG
    assert forward(ly, flags=(0.99, 7), ws_bytes=0) == X.ERR_WORKSPACE
    # the diagonal phase needs the maps
    assert forward(ly, phase=4, budget=1, diag=None) == X.ERR_NULL
    assert forward(ly, phase=4, budget=0) == X.ERR_BUDGET
    assert forward(ly, phase=4, budget=1, ws_bytes=0) == X.ERR_WORKSPACE
    assert ws_size(ly, phase=4, budget=1) > ws_size(ly, phase=1, budget=1)


def test_workspace_grows_with_tokens_and_budget():
    ly = layer(dtype=X.BF16)
    a, b = ws_size(ly, T=64), ws_size(ly, T=128)
    assert 0 < a < b
    assert ws_size(ly, T=64, phase=1, budget=1) < ws_size(ly, T=64, phase=1, budget=2)
    assert ws_size(ly, T=0) > 0


def test_select_and_fold_validation():
    L = X.lib()
    f = FAKE
    assert L.exfold_select_prefill(f, 4, 8, 9, 1, f, f, f, f, None) == X.ERR_SHAPE
    assert L.exfold_select_prefill(f, 4, 8, 2, 0, f, f, f, f, None) == X.ERR_BUDGET
    assert L.exfold_select_prefill(f, 4, 8, 2, 1, None, f, f, f, None) == X.ERR_NULL
    assert L.exfold_select_prefill(f, 4, 512, 2, 1, f, f, f, f, None) == X.ERR_UNSUPPORTED
    assert L.exfold_select_prefill(f, 0, 8, 2, 1, f, f, f, f, None) == X.OK
    assert L.exfold_select_decode_pool(f, 4, 8, 2, 0, f, f, f, f, f, None) == X.ERR_BUDGET
    assert L.exfold_select_decode_pool(f, 4, 8, 2, 3, f, f, f, None, f, None) == X.ERR_NULL
    assert L.exfold_fold_gates(7, 4, 8, 2, 1, f, f, f, f, f, f, f, f, f, None, None, 0.0, 0, None) == X.ERR_ARG
    assert L.exfold_fold_gates(1, 4, 8, 2, 0, f, f, f, f, f, f, f, f, f, None, None, 0.0, 0, None) == X.ERR_BUDGET
    assert L.exfold_fold_gates(1, 4, 8, 2, 1, f, f, None, f, f, f, f, f, f, None, None, 0.0, 0, None) == X.ERR_NULL
    assert L.exfold_fold_gates(2, 4, 8, 2, 1, f, f, None, None, f, f, f, f, f, None, None, 0.0, 0, None) == X.ERR_NULL
    assert L.exfold_fold_gates(2, 4, 8, 2, 1, f, f, None, f, f, None, f, f, f, None, None, 0.0, 0, None) == X.ERR_NULL
    assert L.exfold_fold_gates(3, 4, 8, 2, 1, f, f, None, f, f, f, f, f, f, None, None, 0.0, 0, None) == X.ERR_ARG
    assert L.exfold_fold_gates(1, 4, 8, 2, 1, f, f, f, f, f, f, f, f, f, None, None, 0.5, 8, None) == X.ERR_ARG
    assert L.exfold_fold_gates(1, 4, 8, 2, 1, f, f, f, f, f, f, f, f, f, None, None, float("nan"), 1,
                               None) == X.ERR_ARG
    assert L.exfold_static_pool(f, 8, 0, f, f, f, f, f, f, None) == X.ERR_BUDGET
    assert L.exfold_static_pool(f, 0, 4, f, f, f, f, f, f, None) == X.ERR_SHAPE
    assert L.exfold_static_pool(f, 512, 4, f, f, f, f, f, f, None) == X.ERR_UNSUPPORTED
    assert L.exfold_static_pool(f, 8, 4, f, f, f, f, None, f, None) == X.ERR_NULL
    assert L.exfold_static_pool(None, 8, 4, f, f, f, f, f, f, None) == X.ERR_NULL


def test_calibrate_validation():
    L = X.lib()
    ly = layer()
    f = FAKE
    n = L.exfold_calibrate_workspace_size(ctypes.byref(ly), 512, 0)
    assert n > 0 and L.exfold_calibrate_workspace_size(ctypes.byref(ly), 512, 1) > n
    assert L.exfold_calibrate_workspace_size(ctypes.byref(ly), 512, 4) == 0
    call = lambda **kw: L.exfold_calibrate_projectors(
        ctypes.byref(ly), kw.get("x", f), kw.get("m", 512), kw.get("lam", 1e-3), kw.get("clip", 4.0),
        kw.get("mode", 0), kw.get("S", f), f, f, None, f * 16, kw.get("ws", 0), None)
    assert call(mode=3) == X.ERR_ARG
    assert call(lam=-1.0) == X.ERR_ARG
    assert call(clip=float("nan")) == X.ERR_ARG
    assert call(S=None) == X.ERR_NULL
    dcall = lambda **kw: L.exfold_calibrate_diagonal(ctypes.byref(ly), kw.get("x", f), 512, kw.get("lam", 1e-3),
                                                     kw.get("mode", 0), kw.get("D", f), f, f * 16, 0, None)
    assert dcall(mode=3) == X.ERR_ARG
    assert dcall(lam=-1.0) == X.ERR_ARG
    assert dcall(D=None) == X.ERR_NULL
    assert dcall() == X.ERR_WORKSPACE
    assert call(x=None) == X.ERR_NULL
    assert call(ws=n - 1) == X.ERR_WORKSPACE


def test_execute_validation():
    L = X.lib()
    ly = layer()
    f = FAKE
    assert L.exfold_execute_workspace_size(ctypes.byref(ly), 64, 0) == 0
    n = L.exfold_execute_workspace_size(ctypes.byref(ly), 64, 2)
    assert n > 0
    assert L.exfold_moe_execute(ctypes.byref(ly), f, 64, 2, None, f, f, None, f * 16, n, None) == X.ERR_NULL
    assert L.exfold_moe_execute(ctypes.byref(ly), f + 8, 64, 2, f, f, f, None, f * 16, n, None) == X.ERR_ALIGN
    assert L.exfold_moe_execute(ctypes.byref(ly), f, 64, 2, f, f, f, None, f * 16, n - 1, None) == X.ERR_WORKSPACE


def test_scratch_forward_validation():
    # exfold_moe_forward_scratch: the forward's validation codes, then the scratch limit, all
    # before any device call
    L = X.lib()
    ly = layer(dtype=X.BF16)
    tb = X._Tables(FAKE, FAKE, FAKE, FAKE, FAKE, 0.0, 0, FAKE)
    call = lambda T=64, phase=1, budget=1, tables=True, x=FAKE, y=FAKE: L.exfold_moe_forward_scratch(
        ctypes.byref(ly), ctypes.byref(tb) if tables else None, x, T, phase, budget, y, None, None)
    assert call(phase=5) == X.ERR_ARG
    assert call(budget=0) == X.ERR_BUDGET
    assert call(T=-1) == X.ERR_SHAPE
    assert call(tables=False) == X.ERR_NULL
    assert call(x=None) == X.ERR_NULL
    assert call(y=FAKE + 2) == X.ERR_ALIGN
    assert call(T=0) == X.OK
    big = 1
    while ws_size(ly, T=big, phase=2, budget=4) <= X.SCRATCH_BYTES:
        big *= 2
    assert call(T=big, phase=2, budget=4) == X.ERR_SCRATCH
    assert X.status_str(X.ERR_SCRATCH).startswith("request needs more than the static scratch")
