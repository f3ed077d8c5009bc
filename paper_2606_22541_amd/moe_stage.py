"""Python binding of the MoE expert stage's C ABI (``include/moe_stage.h``).

Argument marshalling only: every step of the stage runs in the HIP kernels of
``libmoe_stage.so``.  Functions carry the C names.  Pointers may be given as
torch tensors (their ``data_ptr()``) or integers; streams as
``torch.cuda.Stream`` objects, raw ``hipStream_t`` integers, or None (torch's
current stream).  A non-OK status raises :class:`MoEStageError`.

There is no fallback: if the library is not built, importing the functions
works but every call raises, naming the build step.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe_stage.so")

MOE_OK = 0
MOE_EINVAL = -1
MOE_ENOMEM = -2
MOE_EHIP = -3
MOE_EBADID = -4
MOE_EUNSUPPORTED = -5
MOE_EBUSY = -6
MOE_EBADLAYER = -7
MOE_ETIMEOUT = -8
MOE_EBADCOUNT = -9
MOE_DTYPE_BF16 = 0
MOE_DTYPE_FP8_E4M3_B128 = 1
MOE_COMBINE_OVERWRITE = 0
MOE_COMBINE_ACCUMULATE = 1

# Every entry point the header declares.
EXPORTS = (
    "moe_stage_create", "moe_stage_destroy", "moe_dispatch", "moe_expert_ffn", "moe_combine",
    "moe_stage_submit_microbatch", "moe_quantize_fp8", "moe_stage_query", "moe_stage_sync",
    "moe_stage_workspace_bytes", "moe_status_string", "moe_stage_profile",
    "moe_stage_profile_read", "moe_ingest_wait", "moe_ingest_signal", "moe_expert_ffn_grouped",
    "moe_stage_poll", "moe_dispatch_index_noalloc", "moe_stream_create_cu_masked",
    "moe_stream_destroy",
)
MOE_PROF_KINDS = 6
PROF_KIND_NAMES = ("dispatch_index", "gather", "gemm_gate_up_swiglu", "gemm_down", "combine",
                   "quantize_h")


class moe_stage_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "d_model", "d_ff", "n_experts", "first_local_expert", "n_local_experts", "top_k",
        "max_tokens", "n_slots", "dtype", "has_shared_expert", "n_layers")]


class moe_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "w_gate", "w_up", "w_down", "s_gate", "s_up", "s_down",
        "sh_gate", "sh_up", "sh_down", "sh_s_gate", "sh_s_up", "sh_s_down")]


class moe_microbatch(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int32), ("x", ctypes.c_void_p), ("x_scales", ctypes.c_void_p),
                ("topk_ids", ctypes.c_void_p), ("topk_w", ctypes.c_void_p), ("out", ctypes.c_void_p),
                ("combine_mode", ctypes.c_int32), ("layer_id", ctypes.c_void_p)]


class moe_grouped_batch(ctypes.Structure):
    _fields_ = [("n_rows_max", ctypes.c_int32), ("rows", ctypes.c_void_p),
                ("row_scales", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("layer_id", ctypes.c_void_p)]


class moe_dispatch_view(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "counts", "offsets", "slot_of_row", "row_of_slot", "x_perm", "x_perm_scales", "h",
        "h_scales", "y_perm", "h_shared", "h_shared_scales", "y_shared")] + [
        ("capacity_rows", ctypes.c_int32), ("n_tokens", ctypes.c_int32)]


class MoEStageError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (what, _status_text(status), status))


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("%s is not built; run __graft_entry__.build() "
                           "(or python -m paper_2606_22541_amd.build)" % path)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    st = ctypes.c_int32
    sig = {
        "moe_stage_create": (st, [ctypes.POINTER(moe_stage_desc), ctypes.POINTER(moe_weights),
                                  ctypes.POINTER(P)]),
        "moe_stage_destroy": (None, [P]),
        "moe_dispatch": (st, [P, ctypes.c_int32, ctypes.POINTER(moe_microbatch), P]),
        "moe_expert_ffn": (st, [P, ctypes.c_int32, P]),
        "moe_combine": (st, [P, ctypes.c_int32, P]),
        "moe_stage_submit_microbatch": (st, [P, ctypes.POINTER(moe_microbatch), P,
                                             ctypes.POINTER(ctypes.c_int32)]),
        "moe_quantize_fp8": (st, [P, ctypes.c_int32, ctypes.c_int32, P, P, P]),
        "moe_stage_query": (st, [P, ctypes.c_int32, ctypes.POINTER(moe_dispatch_view)]),
        "moe_stage_sync": (st, [P]),
        "moe_stage_poll": (st, [P, ctypes.c_int32]),
        "moe_stream_create_cu_masked": (st, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(P)]),
        "moe_stream_destroy": (st, [P]),
        "moe_dispatch_index_noalloc": (st, [P] + [ctypes.c_int32] * 5 + [P] * 6),
        "moe_stage_workspace_bytes": (st, [ctypes.POINTER(moe_stage_desc),
                                           ctypes.POINTER(ctypes.c_int64)]),
        "moe_status_string": (ctypes.c_char_p, [st]),
        "moe_stage_profile": (st, [P, ctypes.c_int32]),
        "moe_stage_profile_read": (st, [P, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int32)]),
        "moe_ingest_wait": (st, [P, P, ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint32, P]),
        "moe_ingest_signal": (st, [P, ctypes.c_uint32, P]),
        "moe_expert_ffn_grouped": (st, [P, ctypes.c_int32, ctypes.POINTER(moe_grouped_batch), P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _status_text(status: int) -> str:
    try:
        return load_library().moe_status_string(status).decode()
    except Exception:  # the library may be what is missing
        return "status"


def _check(status: int, what: str):
    if status != MOE_OK:
        raise MoEStageError(status, what)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if hasattr(t, "data_ptr"):
        return t.data_ptr() or None
    return int(t)


def _stream(s) -> Optional[int]:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream or None
    return int(s) or None


def make_desc(d_model, d_ff, n_experts, first_local_expert, n_local_experts, top_k, max_tokens,
              n_slots=1, dtype=MOE_DTYPE_BF16, has_shared_expert=0, n_layers=1) -> moe_stage_desc:
    return moe_stage_desc(d_model, d_ff, n_experts, first_local_expert, n_local_experts, top_k,
                          max_tokens, n_slots, dtype, int(has_shared_expert), int(n_layers))


def make_weights(w_gate, w_up, w_down, s_gate=None, s_up=None, s_down=None, sh_gate=None,
                 sh_up=None, sh_down=None, sh_s_gate=None, sh_s_up=None,
                 sh_s_down=None) -> moe_weights:
    return moe_weights(*[_ptr(t) for t in (w_gate, w_up, w_down, s_gate, s_up, s_down, sh_gate,
                                           sh_up, sh_down, sh_s_gate, sh_s_up, sh_s_down)])


def make_microbatch(n_tokens, x, topk_ids, topk_w, out, x_scales=None,
                    combine_mode=MOE_COMBINE_OVERWRITE, layer_id=None) -> moe_microbatch:
    """layer_id: device int32 (tensor or address) naming the layer, or None."""
    return moe_microbatch(int(n_tokens), _ptr(x), _ptr(x_scales), _ptr(topk_ids), _ptr(topk_w),
                          _ptr(out), int(combine_mode), _ptr(layer_id))


def moe_stage_create(desc: moe_stage_desc, weights) -> int:
    """weights: one moe_weights, or a sequence of desc.n_layers of them."""
    if isinstance(weights, moe_weights):
        weights = [weights]
    arr = (moe_weights * len(weights))(*weights)
    h = ctypes.c_void_p()
    _check(load_library().moe_stage_create(ctypes.byref(desc), arr, ctypes.byref(h)),
           "moe_stage_create")
    return h.value


def moe_stage_destroy(stage: int) -> None:
    load_library().moe_stage_destroy(stage)


def moe_dispatch(stage: int, slot: int, mb: moe_microbatch, stream=None) -> None:
    _check(load_library().moe_dispatch(stage, slot, ctypes.byref(mb), _stream(stream)),
           "moe_dispatch")


def moe_expert_ffn(stage: int, slot: int, stream=None) -> None:
    _check(load_library().moe_expert_ffn(stage, slot, _stream(stream)), "moe_expert_ffn")


def make_grouped_batch(n_rows_max, rows, counts, y, row_scales=None,
                       layer_id=None) -> moe_grouped_batch:
    """counts: device int32 [n_local_experts]; layer_id as in make_microbatch."""
    return moe_grouped_batch(int(n_rows_max), _ptr(rows), _ptr(row_scales), _ptr(counts), _ptr(y),
                             _ptr(layer_id))


def moe_expert_ffn_grouped(stage: int, slot: int, gb: moe_grouped_batch, stream=None) -> None:
    _check(load_library().moe_expert_ffn_grouped(stage, slot, ctypes.byref(gb), _stream(stream)),
           "moe_expert_ffn_grouped")


def moe_combine(stage: int, slot: int, stream=None) -> None:
    _check(load_library().moe_combine(stage, slot, _stream(stream)), "moe_combine")


def moe_stage_submit_microbatch(stage: int, mb: moe_microbatch, stream=None) -> int:
    slot = ctypes.c_int32(-1)
    _check(load_library().moe_stage_submit_microbatch(stage, ctypes.byref(mb), _stream(stream),
                                                      ctypes.byref(slot)),
           "moe_stage_submit_microbatch")
    return slot.value


def moe_quantize_fp8(x_bf16, n_tokens: int, d_model: int, x_q, x_s, stream=None) -> None:
    _check(load_library().moe_quantize_fp8(_ptr(x_bf16), n_tokens, d_model, _ptr(x_q), _ptr(x_s),
                                           _stream(stream)), "moe_quantize_fp8")


def moe_stage_query(stage: int, slot: int) -> moe_dispatch_view:
    v = moe_dispatch_view()
    _check(load_library().moe_stage_query(stage, slot, ctypes.byref(v)), "moe_stage_query")
    return v


def moe_stage_poll(stage: int, slot: int) -> int:
    """MOE_OK when the slot's last work has completed, MOE_EBUSY while it is
    in flight (raises on any other status)."""
    r = load_library().moe_stage_poll(stage, slot)
    if r not in (MOE_OK, MOE_EBUSY):
        raise MoEStageError(r, "moe_stage_poll")
    return r


def moe_dispatch_index_noalloc(topk_ids, n_tokens: int, top_k: int, n_experts: int,
                               first_local_expert: int, n_local_experts: int, counts, offsets,
                               slot_of_row, row_of_slot, err=None, stream=None) -> None:
    """The dispatch index into caller-owned outputs, with no allocation."""
    _check(load_library().moe_dispatch_index_noalloc(
        _ptr(topk_ids), n_tokens, top_k, n_experts, first_local_expert, n_local_experts,
        _ptr(counts), _ptr(offsets), _ptr(slot_of_row), _ptr(row_of_slot), _ptr(err),
        _stream(stream)), "moe_dispatch_index_noalloc")


def moe_stream_create_cu_masked(first_cu: int, n_cus: int) -> int:
    """A hipStream_t (as an int) restricted to CUs [first_cu, first_cu + n_cus)."""
    h = ctypes.c_void_p()
    _check(load_library().moe_stream_create_cu_masked(first_cu, n_cus, ctypes.byref(h)),
           "moe_stream_create_cu_masked")
    return h.value


def moe_stream_destroy(stream: int) -> None:
    _check(load_library().moe_stream_destroy(stream), "moe_stream_destroy")


def moe_stage_sync(stage: int) -> None:
    _check(load_library().moe_stage_sync(stage), "moe_stage_sync")


def moe_stage_sync_status(stage: int) -> int:
    """moe_stage_sync returning the status instead of raising."""
    return load_library().moe_stage_sync(stage)


def moe_stage_workspace_bytes(desc: moe_stage_desc) -> int:
    b = ctypes.c_int64(0)
    _check(load_library().moe_stage_workspace_bytes(ctypes.byref(desc), ctypes.byref(b)),
           "moe_stage_workspace_bytes")
    return b.value


def moe_status_string(status: int) -> str:
    return load_library().moe_status_string(status).decode()


def moe_stage_profile(stage: int, enable: bool) -> None:
    _check(load_library().moe_stage_profile(stage, int(bool(enable))), "moe_stage_profile")


def moe_stage_profile_read(stage: int):
    """Returns {kind name: (total ms, launches)} and clears the records."""
    ms = (ctypes.c_double * MOE_PROF_KINDS)()
    n = (ctypes.c_int32 * MOE_PROF_KINDS)()
    _check(load_library().moe_stage_profile_read(stage, ms, n), "moe_stage_profile_read")
    return {PROF_KIND_NAMES[i]: (ms[i], n[i]) for i in range(MOE_PROF_KINDS)}


def moe_ingest_wait(stage: int, ready, n_words: int, epoch: int, spin_limit: int = 0,
                    stream=None) -> None:
    _check(load_library().moe_ingest_wait(stage, _ptr(ready), int(n_words), epoch & 0xFFFFFFFF,
                                          int(spin_limit), _stream(stream)), "moe_ingest_wait")


def moe_ingest_signal(word, epoch: int, stream=None) -> None:
    _check(load_library().moe_ingest_signal(_ptr(word), epoch & 0xFFFFFFFF, _stream(stream)),
           "moe_ingest_signal")

