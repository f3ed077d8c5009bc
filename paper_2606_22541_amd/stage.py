"""Convenience wrapper over the C ABI for torch callers (tests, bench, smoke).

Holds a stage handle built from :class:`inputs.ExpertWeights` on the GPU and
turns micro-batch tensors into ``moe_microbatch`` structs.  All work runs in
the HIP library; this module only marshals arguments and copies workspace
views back to the host for inspection.
"""
from __future__ import annotations

import ctypes
from typing import Dict, Optional

import numpy as np
import torch

from . import moe_stage as C

_hip = None


def _hip_lib():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    return _hip


def device_to_numpy(ptr: int, count: int, dtype) -> np.ndarray:
    """Synchronous copy of ``count`` elements at device address ``ptr``."""
    out = np.empty(max(count, 0), dtype=dtype)
    if count > 0:
        rc = _hip_lib().hipMemcpy(out.ctypes.data, ptr, out.nbytes, 2)  # device -> host
        if rc != 0:
            raise RuntimeError("hipMemcpy failed (%d)" % rc)
    return out


class ExpertStage:
    """One device's share of experts, created from generator weights (one
    ExpertWeights, or a list of them: one per layer)."""

    def __init__(self, cfg, weights, n_slots: int = 1, max_tokens: Optional[int] = None):
        self.cfg = cfg
        self.fp8 = cfg.dtype == "fp8"
        self.max_tokens = cfg.max_tokens if max_tokens is None else max_tokens
        layers = list(weights) if isinstance(weights, (list, tuple)) else [weights]
        self.n_layers = len(layers)
        self.n_slots = n_slots
        self.desc = C.make_desc(cfg.d, cfg.f, cfg.E, cfg.e0, cfg.E_loc, cfg.k, self.max_tokens,
                                n_slots, C.MOE_DTYPE_FP8_E4M3_B128 if self.fp8 else C.MOE_DTYPE_BF16,
                                int(cfg.has_shared), self.n_layers)
        wts = [C.make_weights(w.w_gate, w.w_up, w.w_down, w.s_gate, w.s_up, w.s_down,
                              w.sh_gate, w.sh_up, w.sh_down, w.sh_s_gate, w.sh_s_up, w.sh_s_down)
               for w in layers]
        torch.cuda.synchronize()
        self.handle = C.moe_stage_create(self.desc, wts)
        self._keep = {}

    def microbatch(self, x, ids, w, out, x_scales=None, mode=C.MOE_COMBINE_OVERWRITE,
                   layer_id=None):
        return C.make_microbatch(ids.shape[0], x, ids, w, out, x_scales, mode, layer_id)

    def submit(self, mb, stream=None) -> int:
        return C.moe_stage_submit_microbatch(self.handle, mb, stream)

    def dispatch(self, slot, mb, stream=None):
        C.moe_dispatch(self.handle, slot, mb, stream)

    def expert_ffn(self, slot, stream=None):
        C.moe_expert_ffn(self.handle, slot, stream)

    def expert_ffn_grouped(self, slot, rows, counts, y, row_scales=None, layer_id=None,
                           stream=None):
        """Expert FFN of rows already grouped by local expert (counts: device
        int32 [E_loc]); y receives one bf16 row per input row."""
        gb = C.make_grouped_batch(rows.shape[0], rows, counts, y, row_scales, layer_id)
        C.moe_expert_ffn_grouped(self.handle, slot, gb, stream)

    def combine(self, slot, stream=None):
        C.moe_combine(self.handle, slot, stream)

    def sync(self):
        C.moe_stage_sync(self.handle)

    def view(self, slot: int, rows: bool = True) -> Dict[str, np.ndarray]:
        """Host copies of a slot's dispatch results and intermediate rows."""
        v = C.moe_stage_query(self.handle, slot)
        cfg = self.cfg
        T = v.n_tokens
        res = dict(counts=device_to_numpy(v.counts, cfg.E, np.int32),
                   offsets=device_to_numpy(v.offsets, cfg.E_loc + 1, np.int32))
        n = int(res["offsets"][-1])
        res["n_loc"] = n
        res["slot_of_row"] = device_to_numpy(v.slot_of_row, n, np.int32)
        res["row_of_slot"] = device_to_numpy(v.row_of_slot, T * cfg.k, np.int32)
        if rows:
            eb = np.uint8 if self.fp8 else np.uint16
            if v.x_perm:          # NULL: the row gather is fused into the gate/up GEMM
                res["x_perm"] = device_to_numpy(v.x_perm, n * cfg.d, eb).reshape(n, cfg.d)
            res["h"] = device_to_numpy(v.h, n * cfg.f, eb).reshape(n, cfg.f)
            res["y_perm"] = device_to_numpy(v.y_perm, n * cfg.d, np.uint16).reshape(n, cfg.d)
            if self.fp8:   # scales are stored transposed: [groups][capacity_rows]
                cap = v.capacity_rows
                xs = device_to_numpy(v.x_perm_scales, cap * cfg.d // 128, np.float32)
                res["x_perm_scales"] = xs.reshape(cfg.d // 128, cap)[:, :n].T.copy()
                hs = device_to_numpy(v.h_scales, cap * cfg.f // 128, np.float32)
                res["h_scales"] = hs.reshape(cfg.f // 128, cap)[:, :n].T.copy()
            if cfg.has_shared:
                res["y_shared"] = device_to_numpy(v.y_shared, T * cfg.d, np.uint16).reshape(T, cfg.d)
        return res

    def close(self):
        if self.handle:
            C.moe_stage_destroy(self.handle)
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def to_device_routing(ids: np.ndarray, w: np.ndarray, device="cuda"):
    return (torch.from_numpy(np.ascontiguousarray(ids, np.int32)).to(device),
            torch.from_numpy(np.ascontiguousarray(w, np.float32)).to(device))


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def quantize_fp8(x: torch.Tensor, stream=None):
    """Runs the stage's sender-side quantiser on a [T, d] bf16 tensor."""
    T, d = x.shape
    xq = torch.empty((T, d), dtype=torch.uint8, device=x.device)
    xs = torch.empty((T, d // 128), dtype=torch.float32, device=x.device)
    C.moe_quantize_fp8(x, T, d, xq, xs, stream)
    return xq, xs
