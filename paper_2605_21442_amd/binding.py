"""ctypes binding of liblce.so: the C ABI of include/lce.h, same names, argument marshalling only.

Every function here forwards plain integers (device pointers, sizes, a stream
handle) to the library and turns a non-zero status into ``LceError``. Nothing
is computed in Python. The library is loaded on first use from this package's
directory; if it was not built, loading raises instead of falling back to
anything else.

The pointers and streams come from PyTorch, whose wheel carries its own HIP runtime. torch is
imported before the library is loaded, so that the library's HIP runtime dependency resolves to
that same, already loaded runtime: loaded first, the library would bring the system's runtime
into the process beside torch's, and its launches would then find no device.
"""
from __future__ import annotations

import ctypes
import os
import threading

LIB_NAME = "liblce.so"
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

LCE_OK = 0
LCE_ERR_NULL = 1
LCE_ERR_SHAPE = 2
LCE_ERR_ALIGN = 3
LCE_ERR_UNSUPPORTED = 4
LCE_ERR_WORKSPACE = 5
LCE_ERR_HIP = 6
LCE_ERR_ARG = 7

LCE_REDUCE_MEAN = 0
LCE_REDUCE_SUM = 1
LCE_REDUCE_NONE = 2
LCE_STATUS_TARGET_OUT_OF_RANGE = 1
LCE_FLAG_ACCUMULATE_DW = 1
LCE_FLAG_REUSE_FORWARD = 2

REDUCTIONS = {"mean": LCE_REDUCE_MEAN, "sum": LCE_REDUCE_SUM, "none": LCE_REDUCE_NONE}

# every symbol include/lce.h declares
EXPORTED = ("lce_workspace_size", "lce_forward", "lce_backward", "lce_status_string",
            "lce_timing_enable", "lce_timing_kernel_count", "lce_timing_kernel_name",
            "lce_timing_read", "lce_adamw_step", "lce_backward_adamw", "lce_forward_shard",
            "lce_combine_shards", "lce_backward_shard", "lce_kd_workspace_size", "lce_kd_forward",
            "lce_kd_backward", "lce_kd_workspace_size_fused", "lce_kd_forward_backward", "lce_plan_info",
            "lce_forward_noalloc")


class LceError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {lce_status_string(code)} (status {code})")


class LceProblem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("d", ctypes.c_int64), ("v", ctypes.c_int64),
                ("ld_h", ctypes.c_int64), ("ld_w", ctypes.c_int64),
                ("ignore_index", ctypes.c_int32), ("reduction", ctypes.c_int32),
                ("target_bytes", ctypes.c_int32), ("flags", ctypes.c_int32)]


class LceAdamW(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float), ("step", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class LceKdProblem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("ds", ctypes.c_int64), ("dt", ctypes.c_int64), ("v", ctypes.c_int64),
                ("ld_hs", ctypes.c_int64), ("ld_ws", ctypes.c_int64), ("ld_ht", ctypes.c_int64),
                ("ld_wt", ctypes.c_int64), ("temperature", ctypes.c_float), ("ignore_index", ctypes.c_int32),
                ("reduction", ctypes.c_int32), ("target_bytes", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


def kd_problem(n: int, ds: int, dt: int, v: int, *, ld_hs: int = 0, ld_ws: int = 0, ld_ht: int = 0,
               ld_wt: int = 0, temperature: float = 1.0, ignore_index: int = -100,
               reduction: str | int = "mean", target_bytes: int = 4, flags: int = 0) -> LceKdProblem:
    red = REDUCTIONS[reduction] if isinstance(reduction, str) else int(reduction)
    return LceKdProblem(n, ds, dt, v, ld_hs, ld_ws, ld_ht, ld_wt, temperature, ignore_index, red, target_bytes,
                        flags, 0)


class LcePlanInfo(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int64) for k in (
        "npad", "rows_g", "vc", "nslab", "dh_kz", "part_rows", "fwd_gathers", "fwd_one_launch",
        "o_idx", "o_pos", "o_nv", "o_hv", "o_pm", "o_ps", "o_terms", "fwd_bytes",
        "o_g", "o_dh32", "o_dh32b", "bwd_bytes")]


class LceShard(ctypes.Structure):
    _fields_ = [("v_total", ctypes.c_int64), ("v_begin", ctypes.c_int64)]


def problem(n: int, d: int, v: int, *, ld_h: int = 0, ld_w: int = 0, ignore_index: int = -100,
            reduction: str | int = "mean", target_bytes: int = 4, flags: int = 0) -> LceProblem:
    red = REDUCTIONS[reduction] if isinstance(reduction, str) else int(reduction)
    return LceProblem(n, d, v, ld_h, ld_w, ignore_index, red, target_bytes, flags)


def adamw(lr: float, beta1: float, beta2: float, eps: float, weight_decay: float, step: int) -> LceAdamW:
    return LceAdamW(lr, beta1, beta2, eps, weight_decay, step, 0)


_lib = None
_lock = threading.Lock()


def load() -> ctypes.CDLL:
    """Load liblce.so once; raise if it is missing (there is no other implementation)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; "
                               f"g.build()'` from the repository root")
        import torch  # noqa: F401  (its HIP runtime first: see the module docstring)
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(LceProblem)
        vp, sz = ctypes.c_void_p, ctypes.c_size_t
        lib.lce_workspace_size.argtypes = [P, ctypes.POINTER(sz), ctypes.POINTER(sz)]
        lib.lce_forward.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_backward.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        A = ctypes.POINTER(LceAdamW)
        lib.lce_adamw_step.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, vp, vp, vp, vp, vp, A, vp]
        lib.lce_backward_adamw.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, A, vp, sz, vp]
        S = ctypes.POINTER(LceShard)
        lib.lce_forward_shard.argtypes = [P, S, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_combine_shards.argtypes = [P, ctypes.c_int32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_backward_shard.argtypes = [P, S, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        KP = ctypes.POINTER(LceKdProblem)
        lib.lce_kd_workspace_size.argtypes = [KP, ctypes.POINTER(sz), ctypes.POINTER(sz)]
        lib.lce_kd_forward.argtypes = [KP, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_kd_backward.argtypes = [KP, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_kd_workspace_size_fused.argtypes = [KP, ctypes.POINTER(sz)]
        lib.lce_kd_forward_backward.argtypes = [KP, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        lib.lce_plan_info.argtypes = [P, ctypes.POINTER(LcePlanInfo)]
        lib.lce_forward_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.lce_status_string.argtypes = [ctypes.c_int]
        lib.lce_status_string.restype = ctypes.c_char_p
        lib.lce_timing_enable.argtypes = [ctypes.c_int]
        lib.lce_timing_kernel_count.argtypes = []
        lib.lce_timing_kernel_name.argtypes = [ctypes.c_int]
        lib.lce_timing_kernel_name.restype = ctypes.c_char_p
        lib.lce_timing_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_int64)]
        for name in ("lce_workspace_size", "lce_forward", "lce_backward", "lce_timing_enable",
                     "lce_timing_read", "lce_timing_kernel_count", "lce_adamw_step", "lce_backward_adamw",
                     "lce_forward_shard", "lce_combine_shards", "lce_backward_shard", "lce_kd_workspace_size",
                     "lce_kd_forward", "lce_kd_backward", "lce_kd_workspace_size_fused", "lce_kd_forward_backward",
                     "lce_plan_info", "lce_forward_noalloc"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
        return lib


def _check(code: int, where: str) -> None:
    if code != LCE_OK:
        raise LceError(code, where)


def lce_status_string(code: int) -> str:
    return load().lce_status_string(int(code)).decode()


def lce_workspace_size(p: LceProblem) -> tuple[int, int]:
    f, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(load().lce_workspace_size(ctypes.byref(p), ctypes.byref(f), ctypes.byref(b)),
           "lce_workspace_size")
    return f.value, b.value


def lce_plan_info(p: LceProblem) -> dict:
    """The workspace layout the library carves for problem p (host only)."""
    out = LcePlanInfo()
    _check(load().lce_plan_info(ctypes.byref(p), ctypes.byref(out)), "lce_plan_info")
    return {k: getattr(out, k) for k, _ in LcePlanInfo._fields_}


LCE_NOALLOC_SCRATCH_BYTES = 256 * 1024 * 1024


def lce_forward_noalloc(p: LceProblem, H: int, W: int, targets: int, loss: int, lse: int, n_valid: int,
                        dev_status: int, stream: int) -> None:
    _check(load().lce_forward_noalloc(ctypes.byref(p), H, W, targets, loss, lse, n_valid, dev_status or None,
                                      stream or None), "lce_forward_noalloc")


def lce_forward(p: LceProblem, H: int, W: int, targets: int, loss: int, lse: int, n_valid: int,
                dev_status: int, workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(load().lce_forward(ctypes.byref(p), H, W, targets, loss, lse, n_valid, dev_status or None,
                              workspace, workspace_bytes, stream or None), "lce_forward")


def lce_backward(p: LceProblem, H: int, W: int, targets: int, lse: int, n_valid: int, grad_loss: int,
                 dH: int, dW: int, workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(load().lce_backward(ctypes.byref(p), H, W, targets, lse, n_valid, grad_loss, dH, dW,
                               workspace, workspace_bytes, stream or None), "lce_backward")


def lce_adamw_step(v: int, d: int, ld_w: int, W: int, dW: int, exp_avg: int, exp_avg_sq: int,
                   W_master: int, opt: LceAdamW, stream: int) -> None:
    _check(load().lce_adamw_step(v, d, ld_w, W, dW or None, exp_avg, exp_avg_sq, W_master or None,
                                 ctypes.byref(opt), stream or None), "lce_adamw_step")


def lce_backward_adamw(p: LceProblem, H: int, W: int, targets: int, lse: int, n_valid: int,
                       grad_loss: int, dH: int, exp_avg: int, exp_avg_sq: int, W_master: int,
                       opt: LceAdamW, workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(load().lce_backward_adamw(ctypes.byref(p), H, W, targets, lse, n_valid, grad_loss, dH, exp_avg,
                                     exp_avg_sq, W_master or None, ctypes.byref(opt), workspace,
                                     workspace_bytes, stream or None), "lce_backward_adamw")


def lce_forward_shard(p: LceProblem, shard: LceShard, H: int, W: int, targets: int, lse_part: int,
                      tgt_part: int, n_valid: int, dev_status: int, workspace: int, workspace_bytes: int,
                      stream: int) -> None:
    _check(load().lce_forward_shard(ctypes.byref(p), ctypes.byref(shard), H, W, targets, lse_part, tgt_part,
                                    n_valid, dev_status or None, workspace, workspace_bytes, stream or None),
           "lce_forward_shard")


def lce_combine_shards(p: LceProblem, n_shards: int, lse_parts: int, tgt_parts: int, targets: int, loss: int,
                       lse: int, n_valid: int, dev_status: int, workspace: int, workspace_bytes: int,
                       stream: int) -> None:
    _check(load().lce_combine_shards(ctypes.byref(p), n_shards, lse_parts, tgt_parts, targets, loss, lse,
                                     n_valid, dev_status or None, workspace, workspace_bytes, stream or None),
           "lce_combine_shards")


def lce_backward_shard(p: LceProblem, shard: LceShard, H: int, W: int, targets: int, lse: int, n_valid: int,
                       grad_loss: int, dH_part: int, dW: int, workspace: int, workspace_bytes: int,
                       stream: int) -> None:
    _check(load().lce_backward_shard(ctypes.byref(p), ctypes.byref(shard), H, W, targets, lse, n_valid,
                                     grad_loss, dH_part, dW, workspace, workspace_bytes, stream or None),
           "lce_backward_shard")


def lce_kd_workspace_size(p: LceKdProblem) -> tuple[int, int]:
    f, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    _check(load().lce_kd_workspace_size(ctypes.byref(p), ctypes.byref(f), ctypes.byref(b)), "lce_kd_workspace_size")
    return f.value, b.value


def lce_kd_forward(p: LceKdProblem, Hs: int, Ws: int, Ht: int, Wt: int, targets: int, loss: int, lse_s: int,
                   lse_t: int, n_valid: int, dev_status: int, workspace: int, workspace_bytes: int,
                   stream: int) -> None:
    _check(load().lce_kd_forward(ctypes.byref(p), Hs, Ws, Ht, Wt, targets, loss, lse_s, lse_t, n_valid,
                                 dev_status or None, workspace, workspace_bytes, stream or None), "lce_kd_forward")


def lce_kd_backward(p: LceKdProblem, Hs: int, Ws: int, Ht: int, Wt: int, targets: int, lse_s: int, lse_t: int,
                    n_valid: int, grad_loss: int, dHs: int, dWs: int, workspace: int, workspace_bytes: int,
                    stream: int) -> None:
    _check(load().lce_kd_backward(ctypes.byref(p), Hs, Ws, Ht, Wt, targets, lse_s, lse_t, n_valid, grad_loss,
                                  dHs, dWs, workspace, workspace_bytes, stream or None), "lce_kd_backward")


def lce_kd_workspace_size_fused(p: LceKdProblem) -> int:
    b = ctypes.c_size_t(0)
    _check(load().lce_kd_workspace_size_fused(ctypes.byref(p), ctypes.byref(b)), "lce_kd_workspace_size_fused")
    return b.value


def lce_kd_forward_backward(p: LceKdProblem, Hs: int, Ws: int, Ht: int, Wt: int, targets: int, grad_loss: int,
                            loss: int, lse_s: int, lse_t: int, n_valid: int, dev_status: int, dHs: int, dWs: int,
                            workspace: int, workspace_bytes: int, stream: int) -> None:
    _check(load().lce_kd_forward_backward(ctypes.byref(p), Hs, Ws, Ht, Wt, targets, grad_loss, loss, lse_s, lse_t,
                                          n_valid, dev_status or None, dHs, dWs, workspace, workspace_bytes,
                                          stream or None), "lce_kd_forward_backward")


def lce_timing_enable(on: bool) -> None:
    _check(load().lce_timing_enable(1 if on else 0), "lce_timing_enable")


def lce_timing_kernel_names() -> list[str]:
    lib = load()
    return [lib.lce_timing_kernel_name(k).decode() for k in range(lib.lce_timing_kernel_count())]


def lce_timing_read(k: int) -> tuple[float, int]:
    ms, cnt = ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(load().lce_timing_read(k, ctypes.byref(ms), ctypes.byref(cnt)), "lce_timing_read")
    return ms.value, cnt.value
