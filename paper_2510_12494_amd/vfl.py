"""ctypes binding of libvfl.so (include/vfl.h): same names, argument
marshalling only.  Every step of the training path runs in the library's
gfx950 kernels; there is no Python or CPU fallback: importing the binding
without a built library raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvfl.so")

VFL_OK, VFL_E_INVALID, VFL_E_NOMEM, VFL_E_HIP, VFL_E_NOT_READY, VFL_E_STALE, VFL_E_STATE = range(7)
VFL_F32, VFL_BF16 = 0, 1
VFL_PARTY_A, VFL_PARTY_B, VFL_TOP = 0, 1, 2
VFL_PARAM_W, VFL_PARAM_B, VFL_PARAM_TABLE = 0, 1, 2
VFL_NOISE_EMB, VFL_NOISE_GRAD, VFL_CLIP_EMB, VFL_CLIP_GRAD = 1, 2, 4, 8
VFL_FIFO_DISCARD, VFL_LOSS_MSE = 16, 32
VFL_MAX_LAYERS = 16
VFL_GRAPH_CYCLES = 4
VFL_STATIC_WORKSPACE_BYTES = 64 << 20
VFL_TIMED_EVERY = 4       # vfl_run times the launches of every 4th tick of a captured cycle
STATUS_NAMES = {0: "VFL_OK", 1: "VFL_E_INVALID", 2: "VFL_E_NOMEM", 3: "VFL_E_HIP",
                4: "VFL_E_NOT_READY", 5: "VFL_E_STALE", 6: "VFL_E_STATE"}

EXPORTS = ("vfl_workspace_size", "vfl_create", "vfl_create_static", "vfl_set_param", "vfl_get_param",
           "vfl_bottom_forward", "vfl_publish", "vfl_top_step", "vfl_bottom_backward",
           "vfl_step", "vfl_get_message", "vfl_get_trace", "vfl_schedule_tick", "vfl_check",
           "vfl_philox", "vfl_timing_enable", "vfl_timing_read", "vfl_bind_dataset", "vfl_run",
           "vfl_state_size", "vfl_get_state", "vfl_set_state", "vfl_discard", "vfl_plan", "vfl_fit_delay",
           "vfl_sync_interval", "vfl_replica_average",
           "vfl_last_error", "vfl_destroy")
KERNEL_CLASSES = ("fwd", "active", "bwd", "dw", "reduce", "cast", "emb_sgd", "gemm", "dwt", "avg")


class vfl_plan_party(C.Structure):
    _fields_ = [("lambda_", C.c_double), ("gamma", C.c_double), ("phi", C.c_double),
                ("beta", C.c_double), ("lambda_top", C.c_double), ("gamma_top", C.c_double),
                ("phi_top", C.c_double), ("beta_top", C.c_double), ("cores", C.c_double),
                ("w_min", C.c_int32), ("w_max", C.c_int32), ("mem_base", C.c_double),
                ("mem_coef", C.c_double), ("mem_cap", C.c_double)]


class vfl_plan_link(C.Structure):
    _fields_ = [("emb_bytes_per_row", C.c_double), ("grad_bytes_per_row", C.c_double),
                ("bandwidth", C.c_double), ("chi", C.c_double)]


class vfl_bottom_spec(C.Structure):
    _fields_ = [("dense_in", C.c_int32), ("n_cat", C.c_int32), ("vocab", C.c_int32),
                ("emb_dim", C.c_int32), ("n_layers", C.c_int32),
                ("widths", C.c_int32 * VFL_MAX_LAYERS), ("relu_mask", C.c_uint32)]


class vfl_top_spec(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("widths", C.c_int32 * VFL_MAX_LAYERS),
                ("relu_mask", C.c_uint32)]


class vfl_opts(C.Structure):
    _fields_ = [("dtype", C.c_int), ("batch", C.c_int32), ("staleness", C.c_int32),
                ("replicas", C.c_int32), ("lr", C.c_float), ("clip_c", C.c_float),
                ("sigma", C.c_float), ("seed", C.c_uint64), ("flags", C.c_uint32)]


class vfl_batch(C.Structure):
    _fields_ = [("dense", C.c_void_p), ("ld", C.c_int64), ("ids", C.c_void_p),
                ("labels", C.c_void_p), ("rows", C.c_int32), ("row0", C.c_int64)]


class vfl_dataset(C.Structure):
    _fields_ = [("dense", C.c_void_p), ("ld", C.c_int64), ("ids", C.c_void_p),
                ("labels", C.c_void_p)]


class VflError(RuntimeError):
    def __init__(self, status: int, where: str, text: str = ""):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)} {text}".strip())


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2510_12494_amd/build.py "
                          "(there is no fallback implementation)")
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, U32, U64, SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_size_t
    BS, TS, OP, BA = (C.POINTER(vfl_bottom_spec), C.POINTER(vfl_top_spec), C.POINTER(vfl_opts),
                      C.POINTER(vfl_batch))
    sig = {
        "vfl_workspace_size": [BS, BS, TS, OP, C.POINTER(SZ)],
        "vfl_create": [BS, BS, TS, OP, P, SZ, P, P, C.POINTER(P)],
        "vfl_create_static": [BS, BS, TS, OP, P, P, C.POINTER(P)],
        "vfl_set_param": [P, C.c_int, I32, I32, P, SZ, I32],
        "vfl_get_param": [P, C.c_int, I32, I32, P, SZ, I32],
        "vfl_bottom_forward": [P, C.c_int, I64, BA, I32],
        "vfl_publish": [P, I64],
        "vfl_top_step": [P, I64, P],
        "vfl_bottom_backward": [P, C.c_int, I64],
        "vfl_step": [P, I64, BA, I32, BA, I32, P],
        "vfl_get_message": [P, I32, I64, P, SZ, C.POINTER(I32)],
        "vfl_get_trace": [P, C.POINTER(I64), SZ, C.POINTER(SZ)],
        "vfl_schedule_tick": [I64, I32, I64, C.POINTER(I64)],
        "vfl_sync_interval": [I32, I64, C.POINTER(I32)],
        "vfl_replica_average": [C.POINTER(P), I32, U32],
        "vfl_check": [P, C.POINTER(U32), C.POINTER(U32)],
        "vfl_philox": [U64, U32, U32, U32, I32, I32, P, P],
        "vfl_timing_enable": [P, U32],
        "vfl_timing_read": [P, I32, C.POINTER(C.c_double), C.POINTER(I64), C.POINTER(C.c_double)],
        "vfl_bind_dataset": [P, C.POINTER(vfl_dataset), C.POINTER(vfl_dataset), I64],
        "vfl_run": [P, I64, I64, P, I64],
        "vfl_state_size": [P, C.POINTER(SZ)],
        "vfl_discard": [P, I64],
        "vfl_plan": [C.POINTER(vfl_plan_party), C.POINTER(vfl_plan_party), C.POINTER(vfl_plan_link),
                     C.POINTER(I32), I32, C.POINTER(I32), C.POINTER(C.c_double)],
        "vfl_fit_delay": [C.POINTER(C.c_double), C.POINTER(C.c_double), I32, C.POINTER(C.c_double),
                          C.POINTER(C.c_double)],
        "vfl_get_state": [P, P, SZ],
        "vfl_set_state": [P, P, SZ],
        "vfl_destroy": [P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.vfl_last_error.argtypes = [P]
    lib.vfl_last_error.restype = C.c_char_p
    return lib


_lib = _load()


def _chk(st: int, where: str, ctx=None):
    if st != VFL_OK:
        # without a context the text is the calling thread's last
        # vfl_workspace_size / vfl_create failure
        raw = _lib.vfl_last_error(ctx)
        text = raw.decode() if raw else ""
        raise VflError(st, where, text)


def _batches(bs):
    if not bs:
        return None, 0
    arr = (vfl_batch * len(bs))(*bs)
    return arr, len(bs)


# ---------------------------------------------------------------- the ABI
def vfl_workspace_size(a: vfl_bottom_spec, b: vfl_bottom_spec, top: vfl_top_spec,
                       o: vfl_opts) -> int:
    n = C.c_size_t(0)
    _chk(_lib.vfl_workspace_size(C.byref(a), C.byref(b), C.byref(top), C.byref(o), C.byref(n)),
         "vfl_workspace_size")
    return n.value


def vfl_create(a, b, top, o, workspace_ptr: int, nbytes: int, stream_a: int, stream_b: int):
    h = C.c_void_p()
    _chk(_lib.vfl_create(C.byref(a), C.byref(b), C.byref(top), C.byref(o), C.c_void_p(workspace_ptr),
                         nbytes, C.c_void_p(stream_a), C.c_void_p(stream_b), C.byref(h)),
         "vfl_create")
    return h


def vfl_create_static(a, b, top, o, stream_a: int, stream_b: int):
    h = C.c_void_p()
    _chk(_lib.vfl_create_static(C.byref(a), C.byref(b), C.byref(top), C.byref(o), C.c_void_p(stream_a),
                                C.c_void_p(stream_b), C.byref(h)),
         "vfl_create_static")
    return h


def vfl_set_param(ctx, party: int, layer: int, kind: int, src_ptr: int, nbytes: int, on_device: bool):
    _chk(_lib.vfl_set_param(ctx, party, layer, kind, C.c_void_p(src_ptr), nbytes, int(on_device)),
         "vfl_set_param", ctx)


def vfl_get_param(ctx, party: int, layer: int, kind: int, dst_ptr: int, nbytes: int, on_device: bool):
    _chk(_lib.vfl_get_param(ctx, party, layer, kind, C.c_void_p(dst_ptr), nbytes, int(on_device)),
         "vfl_get_param", ctx)


def vfl_bottom_forward(ctx, party: int, group: int, batches):
    arr, n = _batches(batches)
    _chk(_lib.vfl_bottom_forward(ctx, party, group, arr, n), "vfl_bottom_forward", ctx)


def vfl_publish(ctx, group: int):
    _chk(_lib.vfl_publish(ctx, group), "vfl_publish", ctx)


def vfl_top_step(ctx, group: int, loss_ptr: int = 0):
    _chk(_lib.vfl_top_step(ctx, group, C.c_void_p(loss_ptr or None)), "vfl_top_step", ctx)


def vfl_bottom_backward(ctx, party: int, group: int):
    _chk(_lib.vfl_bottom_backward(ctx, party, group), "vfl_bottom_backward", ctx)


def vfl_step(ctx, t: int, a_batches, b_batches, loss_ptr: int = 0):
    aa, na = _batches(a_batches)
    bb, nb = _batches(b_batches)
    _chk(_lib.vfl_step(ctx, t, aa, na, bb, nb, C.c_void_p(loss_ptr or None)), "vfl_step", ctx)


def vfl_get_message(ctx, which: int, group: int, dst_ptr: int, nbytes: int):
    hdr = (C.c_int32 * 3)()
    _chk(_lib.vfl_get_message(ctx, which, group, C.c_void_p(dst_ptr), nbytes, hdr),
         "vfl_get_message", ctx)
    return tuple(hdr)


def vfl_get_trace(ctx):
    n = C.c_size_t(0)
    _chk(_lib.vfl_get_trace(ctx, None, 0, C.byref(n)), "vfl_get_trace", ctx)
    buf = (C.c_int64 * (7 * n.value))()
    _chk(_lib.vfl_get_trace(ctx, buf, n.value, C.byref(n)), "vfl_get_trace", ctx)
    return [tuple(buf[7 * i:7 * i + 7]) for i in range(n.value)]


def vfl_schedule_tick(t: int, s: int, n_groups: int):
    out = (C.c_int64 * 7)()
    _chk(_lib.vfl_schedule_tick(t, s, n_groups, out), "vfl_schedule_tick")
    return tuple(out)


def vfl_sync_interval(dt0: int, t: int) -> int:
    v = C.c_int32(0)
    _chk(_lib.vfl_sync_interval(dt0, t, C.byref(v)), "vfl_sync_interval")
    return v.value


def vfl_replica_average(ctxs, parties: int):
    arr = (C.c_void_p * len(ctxs))(*[h.value if isinstance(h, C.c_void_p) else h for h in ctxs])
    _chk(_lib.vfl_replica_average(arr, len(ctxs), parties), "vfl_replica_average", ctxs[0] if ctxs else None)


def vfl_check(ctx):
    """(header mismatches, out-of-range ids read) since the context's creation."""
    v, b = C.c_uint32(0), C.c_uint32(0)
    _chk(_lib.vfl_check(ctx, C.byref(v), C.byref(b)), "vfl_check", ctx)
    return v.value, b.value


def vfl_philox(seed: int, step: int, tag: int, row0: int, rows: int, groups: int, out_ptr: int,
               stream: int = 0):
    _chk(_lib.vfl_philox(seed, step, tag, row0, rows, groups, C.c_void_p(out_ptr),
                         C.c_void_p(stream or None)), "vfl_philox")


def vfl_timing_enable(ctx, mask: int):
    _chk(_lib.vfl_timing_enable(ctx, mask), "vfl_timing_enable", ctx)


def vfl_timing_read(ctx, cls: int):
    """(milliseconds, launches, algorithmic work) summed over the class."""
    ms, n, wk = C.c_double(0), C.c_int64(0), C.c_double(0)
    _chk(_lib.vfl_timing_read(ctx, cls, C.byref(ms), C.byref(n), C.byref(wk)), "vfl_timing_read", ctx)
    return ms.value, n.value, wk.value


def vfl_bind_dataset(ctx, a: vfl_dataset, b: vfl_dataset, n_rows: int):
    _chk(_lib.vfl_bind_dataset(ctx, C.byref(a), C.byref(b), n_rows), "vfl_bind_dataset", ctx)


def vfl_run(ctx, t0: int, n: int, loss_ptr: int = 0, loss_len: int = 0):
    _chk(_lib.vfl_run(ctx, t0, n, C.c_void_p(loss_ptr or None), loss_len), "vfl_run", ctx)


def vfl_plan(a: vfl_plan_party, p: vfl_plan_party, link: vfl_plan_link, batches):
    """Returns ((w_a, w_p, B), cost)."""
    arr = (C.c_int32 * len(batches))(*batches)
    out = (C.c_int32 * 3)()
    cost = C.c_double(0.0)
    _chk(_lib.vfl_plan(C.byref(a), C.byref(p), C.byref(link), arr, len(batches), out, C.byref(cost)),
         "vfl_plan")
    return (out[0], out[1], out[2]), cost.value


def vfl_fit_delay(batches, seconds):
    """Returns (coef, exp) of T = coef * B**exp fitted to the measured pairs."""
    n = len(batches)
    xb = (C.c_double * n)(*batches)
    xt = (C.c_double * n)(*seconds)
    coef, expo = C.c_double(0.0), C.c_double(0.0)
    _chk(_lib.vfl_fit_delay(xb, xt, n, C.byref(coef), C.byref(expo)), "vfl_fit_delay")
    return coef.value, expo.value


def vfl_discard(ctx, group: int):
    _chk(_lib.vfl_discard(ctx, group), "vfl_discard", ctx)


def vfl_state_size(ctx) -> int:
    n = C.c_size_t(0)
    _chk(_lib.vfl_state_size(ctx, C.byref(n)), "vfl_state_size", ctx)
    return n.value


def vfl_get_state(ctx) -> np.ndarray:
    """The context's state image (uint8 host array of vfl_state_size bytes)."""
    buf = np.empty(vfl_state_size(ctx), dtype=np.uint8)
    _chk(_lib.vfl_get_state(ctx, buf.ctypes.data, buf.nbytes), "vfl_get_state", ctx)
    return buf


def vfl_set_state(ctx, image: np.ndarray):
    a = np.ascontiguousarray(image, dtype=np.uint8)
    _chk(_lib.vfl_set_state(ctx, a.ctypes.data, a.nbytes), "vfl_set_state", ctx)


def vfl_last_error(ctx) -> str:
    raw = _lib.vfl_last_error(ctx)
    return raw.decode() if raw else ""


def vfl_destroy(ctx):
    _chk(_lib.vfl_destroy(ctx), "vfl_destroy")


def library():
    """The loaded ctypes library (for symbol checks)."""
    return _lib
