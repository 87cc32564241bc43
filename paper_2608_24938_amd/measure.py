"""Measurement helpers shared by bench.py and the sweep: HIP events on the
library's stream, seeded full-size layers, and the algorithmic work of a layer
(flops of a prefill forward, HBM bytes of a decode forward).
"""

from __future__ import annotations

import ctypes
import os

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


class HipEvents:
    """hipEvent_t handles from the HIP runtime torch has loaded (one runtime per process)."""

    def __init__(self):
        import torch
        path = os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so")
        self.hip = ctypes.CDLL(path if os.path.exists(path) else "libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.owned = []

    def array(self, n):
        arr = (ctypes.c_void_p * n)()
        for i in range(n):
            ev = ctypes.c_void_p()
            assert self.hip.hipEventCreate(ctypes.byref(ev)) == 0
            arr[i] = ev.value
            self.owned.append(ev.value)
        return arr

    def record(self, ev, stream):
        assert self.hip.hipEventRecord(ev, stream) == 0

    def ms(self, a, b):
        out = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(out), a, b) == 0
        return float(out.value)

    def close(self):
        for ev in self.owned:
            self.hip.hipEventDestroy(ev)
        self.owned = []


def make_layer(shape, seed=0):
    """Seeded synthetic layer of `shape` on the device: (exfold.Layer, host arrays, host-to-device copier)."""
    import numpy as np
    import torch
    from . import exfold as X
    from . import synth

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)
        return torch.from_numpy(a).to("cuda")

    wr = synth.router_weight(shape, seed)
    gu, dn = synth.all_expert_weights(shape, seed, threads=16)
    sgu, sdn = synth.shared_weights(shape, seed)
    layer = X.Layer(w_router=dev(wr), w_gate_up=dev(gu), w_down=dev(dn), top_k=shape.top_k,
                    router_bias=dev(synth.router_bias(shape, seed)), ws_gate_up=dev(sgu), ws_down=dev(sdn))
    host = dict(wr=wr, gu=gu, dn=dn, sgu=sgu, sdn=sdn, bias=synth.router_bias(shape, seed))
    return layer, host, dev


def prefill_flops(shape, T, k_out):
    """Algorithmic flops of one prefill layer: router GEMM + gate/up (4dI) and down (2dI) per executed route."""
    shared = 6 * shape.d * shape.shared_inter * T
    return 2 * shape.d * shape.n_experts * T + 6 * shape.d * shape.inter * T * k_out + shared


def decode_bytes(shape, B, touched):
    """Algorithmic HBM bytes of one decode layer: weights of the touched experts (+ shared), router, x and y."""
    esz = 2 if shape.dtype == "bf16" else 4
    w = 3 * shape.d * shape.inter * esz * touched + 3 * shape.d * shape.shared_inter * esz
    return w + shape.n_experts * shape.d * esz + 2 * B * shape.d * esz + B * shape.top_k * 16
