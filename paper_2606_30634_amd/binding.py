"""ctypes binding of the stage library's C ABI (include/asyncstage.h): argument marshalling only.

Device memory and streams come from PyTorch; every step of the path runs in the library's HIP
kernels.  Importing this module fails loudly when the built library is missing."""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libasyncstage.so")

STAGE_OK, STAGE_EINVAL, STAGE_ENOSPACE, STAGE_EHIP, STAGE_ESTATE, STAGE_ENONFINITE = 0, -1, -2, -3, -4, -5
DT_F32, DT_BF16, DT_I32 = 0, 1, 2

EXPORTS = ["stage_required_bytes", "stage_init", "stage_num_tensors", "stage_tensor",
           "stage_tensor_by_name", "stage_sync_weights", "stage_forward", "stage_backward",
           "delayed_update", "delayed_update_flat", "stage_embed_indices", "stage_poll_nonfinite",
           "stage_grad_norm", "stage_profile_enable", "stage_profile_read", "stage_last_error",
           "stage_destroy", "stage_set_update_overlap", "stage_join_update", "stage_resume",
           "grad_norm_flat_workspace_bytes", "grad_norm_flat", "hbm_stream_copy", "delayed_update_flat_adan",
           "grad_norm_flat_noalloc"]
PROF_GEMM, PROF_ATTN_FWD, PROF_ATTN_BWD, PROF_UPDATE, PROF_NORM, PROF_OTHER, PROF_NS = range(7)


class StageShape(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("n_blocks", "d_model", "n_heads", "n_kv_heads", "head_dim",
                                         "d_ffn", "vocab", "first_stage", "last_stage",
                                         "tie_embedding", "seq_len", "micro_batch", "max_inflight",
                                         "dtype")] + [("rms_eps", C.c_float), ("rope_theta", C.c_float),
                                                      ("optimizer", C.c_int32), ("max_delay", C.c_int32)]


class UpdateHParams(C.Structure):
    _fields_ = [(n, C.c_float) for n in ("lr", "beta1", "beta2", "eps", "weight_decay", "clip_norm",
                                         "ef_lambda")] + [("delay", C.c_int32), ("optimizer", C.c_int32),
                                                          ("momentum", C.c_float), ("update_rms", C.c_float),
                                                          ("ns_steps", C.c_int32), ("predict", C.c_int32),
                                                          ("nadam_psi", C.c_float), ("beta3", C.c_float)]


class StageError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} -> {code}: {msg}")
        self.code = code


def _load():
    # One HIP runtime per process: torch ships its own libamdhip64 with the same soname as ROCm's.
    # Loading torch first makes this library bind to that runtime; loading this library first would
    # bring a second HIP/HSA runtime into the process, which then sees no device.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    lib = C.CDLL(LIB_PATH)
    vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "stage_required_bytes": (sz, [C.POINTER(StageShape)]),
        "stage_init": (C.c_int, [C.POINTER(StageShape), vp, sz, vp, C.POINTER(vp)]),
        "stage_num_tensors": (C.c_int, [vp, C.POINTER(i32)]),
        "stage_tensor": (C.c_int, [vp, i32, C.POINTER(C.c_char_p), C.POINTER(vp), C.POINTER(i64), C.POINTER(i32)]),
        "stage_tensor_by_name": (C.c_int, [vp, C.c_char_p, C.POINTER(vp), C.POINTER(i64), C.POINTER(i32)]),
        "stage_sync_weights": (C.c_int, [vp]),
        "stage_forward": (C.c_int, [vp, i32, i64, vp, vp, vp, vp, vp]),
        "stage_backward": (C.c_int, [vp, i32, vp, vp, i32]),
        "delayed_update": (C.c_int, [vp, i64, C.POINTER(UpdateHParams)]),
        "delayed_update_flat": (C.c_int, [i64, vp, vp, i32, vp, vp, vp, vp, i32, i64,
                                          C.POINTER(UpdateHParams), vp, vp]),
        "stage_embed_indices": (C.c_int, [vp, i32, vp, vp, vp]),
        "stage_poll_nonfinite": (C.c_int, [vp, C.POINTER(i64)]),
        "stage_grad_norm": (C.c_int, [vp, i32, vp]),
        "stage_profile_enable": (C.c_int, [vp, i32]),
        "stage_set_update_overlap": (C.c_int, [vp, i32]),
        "stage_join_update": (C.c_int, [vp]),
        "stage_resume": (C.c_int, [vp, i64, i32]),
        "grad_norm_flat_workspace_bytes": (sz, []),
        "grad_norm_flat": (C.c_int, [i64, vp, i32, C.c_float, vp, vp, vp, sz, vp]),
        "hbm_stream_copy": (C.c_int, [vp, vp, sz, vp]),
        "grad_norm_flat_noalloc": (C.c_int, [i64, vp, i32, C.c_float, vp, vp, vp]),
        "delayed_update_flat_adan": (C.c_int, [i64, vp, vp, i32, vp, vp, vp, vp, vp, vp, i32, i64,
                                               C.POINTER(UpdateHParams), vp, vp]),
        "stage_profile_read": (C.c_int, [vp, i32, C.POINTER(C.c_double), C.POINTER(i64), C.POINTER(C.c_double)]),
        "stage_last_error": (C.c_char_p, []),
        "stage_destroy": (None, [vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


LIB = _load()


def last_error() -> str:
    return LIB.stage_last_error().decode()


def check(fn: str, rc: int) -> int:
    if rc != STAGE_OK:
        raise StageError(fn, rc, last_error())
    return rc


def _call(fn: str, *args) -> int:
    return check(fn, getattr(LIB, fn)(*args))


def stage_required_bytes(shape: StageShape) -> int:
    return LIB.stage_required_bytes(C.byref(shape))


def stage_init(shape: StageShape, arena_ptr: int, arena_bytes: int, stream_ptr: int) -> int:
    out = C.c_void_p()
    _call("stage_init", C.byref(shape), arena_ptr, arena_bytes, stream_ptr, C.byref(out))
    return out.value


def stage_num_tensors(s: int) -> int:
    n = C.c_int32()
    _call("stage_num_tensors", s, C.byref(n))
    return n.value


def stage_tensor(s: int, idx: int):
    name, ptr, numel, dt = C.c_char_p(), C.c_void_p(), C.c_int64(), C.c_int32()
    _call("stage_tensor", s, idx, C.byref(name), C.byref(ptr), C.byref(numel), C.byref(dt))
    return name.value.decode(), ptr.value, numel.value, dt.value


def stage_tensor_by_name(s: int, name: str):
    ptr, numel, dt = C.c_void_p(), C.c_int64(), C.c_int32()
    _call("stage_tensor_by_name", s, name.encode(), C.byref(ptr), C.byref(numel), C.byref(dt))
    return ptr.value, numel.value, dt.value


def stage_sync_weights(s: int) -> None:
    _call("stage_sync_weights", s)


def stage_forward(s: int, slot: int, step: int, tokens=None, x_in=None, targets=None, y_out=None,
                  loss_dev=None) -> None:
    _call("stage_forward", s, slot, step, tokens, x_in, targets, y_out, loss_dev)


def stage_backward(s: int, slot: int, dy=None, dx_out=None, microbatches_per_step: int = 1) -> None:
    _call("stage_backward", s, slot, dy, dx_out, microbatches_per_step)


def delayed_update(s: int, t: int, hp: UpdateHParams) -> None:
    _call("delayed_update", s, t, C.byref(hp))


def delayed_update_flat(n, x, g_prev, g_is_bf16, m, v, u_prev, x_shadow, shadow_is_bf16, t,
                        hp: UpdateHParams, clip_scale_dev, stream) -> None:
    _call("delayed_update_flat", n, x, g_prev, int(g_is_bf16), m, v, u_prev, x_shadow,
          int(shadow_is_bf16), t, C.byref(hp), clip_scale_dev, stream)


def delayed_update_flat_adan(n, x, g_prev, g_is_bf16, m, v, d, g_last, u_prev, x_shadow, shadow_is_bf16, t,
                             hp: UpdateHParams, clip_scale_dev, stream) -> None:
    _call("delayed_update_flat_adan", n, x, g_prev, int(g_is_bf16), m, v, d, g_last, u_prev, x_shadow,
          int(shadow_is_bf16), t, C.byref(hp), clip_scale_dev, stream)


def grad_norm_flat_workspace_bytes() -> int:
    return LIB.grad_norm_flat_workspace_bytes()


def grad_norm_flat(n, g, g_is_bf16, clip_norm, out_dev, nonfinite_dev, workspace, workspace_bytes, stream) -> None:
    _call("grad_norm_flat", n, g, int(g_is_bf16), clip_norm, out_dev, nonfinite_dev, workspace,
          workspace_bytes, stream)


def grad_norm_flat_noalloc(n, g, g_is_bf16, clip_norm, out_dev, nonfinite_dev, stream) -> None:
    _call("grad_norm_flat_noalloc", n, g, int(g_is_bf16), clip_norm, out_dev, nonfinite_dev, stream)


def hbm_stream_copy(dst, src, nbytes, stream) -> None:
    _call("hbm_stream_copy", dst, src, nbytes, stream)


def stage_embed_indices(s: int, slot: int, ids, counts, n_unique) -> None:
    _call("stage_embed_indices", s, slot, ids, counts, n_unique)


def stage_poll_nonfinite(s: int):
    k = C.c_int64()
    rc = LIB.stage_poll_nonfinite(s, C.byref(k))
    if rc not in (STAGE_OK, STAGE_ENONFINITE):
        check("stage_poll_nonfinite", rc)
    return rc, k.value


def stage_grad_norm(s: int, which: int, norm_dev) -> None:
    _call("stage_grad_norm", s, which, norm_dev)


def stage_set_update_overlap(s: int, mode: int) -> None:
    _call("stage_set_update_overlap", s, int(mode))


def stage_join_update(s: int) -> None:
    _call("stage_join_update", s)


def stage_resume(s: int, next_t: int, delay: int) -> None:
    _call("stage_resume", s, next_t, delay)


def stage_profile_enable(s: int, on: bool) -> None:
    _call("stage_profile_enable", s, int(on))


def stage_profile_read(s: int, cls: int):
    """(milliseconds, launches, algorithmic work) of one kernel class since the last read."""
    ms, n, work = C.c_double(), C.c_int64(), C.c_double()
    _call("stage_profile_read", s, cls, C.byref(ms), C.byref(n), C.byref(work))
    return ms.value, n.value, work.value


def stage_destroy(s: int) -> None:
    LIB.stage_destroy(s)
