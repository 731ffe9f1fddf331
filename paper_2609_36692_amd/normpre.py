"""ctypes binding of libnormpre (include/normpre.h), same names as the C ABI.

Argument marshalling only: every numerical step runs in the library's gfx950
kernels.  There is no fallback: if the shared library is missing or cannot
be loaded, every entry point raises.  Tensors are passed as raw device
pointers; the stream defaults to torch's current stream.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libnormpre.so")

NORMPRE_OK = 0
NORMPRE_ERR_INVALID_ARG = -1
NORMPRE_ERR_UNSUPPORTED = -2
NORMPRE_ERR_OOM = -3
NORMPRE_ERR_HIP = -4
NORMPRE_ERR_NOT_INITIALIZED = -5

NORMPRE_VARIANT_G = 0
NORMPRE_VARIANT_L = 1
NORMPRE_VARIANT_MUON = 2
NORMPRE_VARIANT_NORMALIZE_ONLY = 3
VARIANTS = {"G": NORMPRE_VARIANT_G, "L": NORMPRE_VARIANT_L, "MUON": NORMPRE_VARIANT_MUON,
            "NORM": NORMPRE_VARIANT_NORMALIZE_ONLY}
NORMPRE_ORIENT_ALTERNATING = 0
NORMPRE_ORIENT_ROW = 1
NORMPRE_ORIENT_COL = 2
NORMPRE_ORIENT_BOTH = 3
NORMPRE_FLAG_DEBUG = 1
NORMPRE_FLAG_TIME_KERNELS = 2
NORMPRE_FLAG_TANGENT_NONE = 4
NORMPRE_FLAG_TANGENT_STRICT = 8
NORMPRE_FLAG_L_EXACT = 16
NORMPRE_FLAG_SOURCE_X = 32
NORMPRE_FLAG_CHECK_FINITE = 64

NORMPRE_NOALLOC_SCRATCH_BYTES = 256 << 20

NORMPRE_SPECTRUM_GAMMA = 0
NORMPRE_SPECTRUM_GX = 1

NORMPRE_DEBUG_PSI = 0
NORMPRE_DEBUG_T = 1
NORMPRE_DEBUG_RITZ = 2
NORMPRE_DEBUG_NSEL = 3
NORMPRE_DEBUG_ELL = 4
NORMPRE_DEBUG_TNORM2 = 5
NORMPRE_DEBUG_ORIENT = 6

NORMPRE_KCLASS_NORMALIZE = 0
NORMPRE_KCLASS_NS_GRAM = 1
NORMPRE_KCLASS_NS_POLY = 2
NORMPRE_KCLASS_NS_COMBINE = 3
NORMPRE_KCLASS_G_UPDATE = 4
NORMPRE_KCLASS_SK_STREAM = 5
NORMPRE_KCLASS_SK_SMALL = 6
NORMPRE_KCLASS_L_APPLY = 7
NORMPRE_KCLASS_EIGEN = 8
NORMPRE_KCLASS_NORMALIZE_COL = 9
NORMPRE_KCLASS_COUNT = 10
KCLASS_NAMES = ["normalize", "ns_gram", "ns_poly", "ns_combine", "g_update",
                "sk_stream", "sk_small", "l_apply", "eigen", "normalize_col"]


class NormPreError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"normpre error {code}: {msg}")
        self.code = code


class normpre_hparams(ctypes.Structure):
    _fields_ = [
        ("lr", ctypes.c_float),
        ("momentum", ctypes.c_float),
        ("weight_decay", ctypes.c_float),
        ("target_rms", ctypes.c_float),
        ("ns_iters", ctypes.c_int32),
        ("ns_coeffs", ctypes.c_float * 3),
        ("ns_eps", ctypes.c_float),
        ("rank", ctypes.c_int32),
        ("oversample", ctypes.c_int32),
        ("power_iters", ctypes.c_int32),
        ("orientation", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("step", ctypes.c_int64),
        ("norm_eps", ctypes.c_float),
        ("flags", ctypes.c_uint32),
    ]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libnormpre.so (once).  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i64p = ctypes.POINTER(ctypes.c_int64)
    hpp = ctypes.POINTER(normpre_hparams)
    sig = {
        "normpre_default_hparams": (ctypes.c_int, [hpp]),
        "normpre_init": (ctypes.c_int, [ctypes.POINTER(P), ctypes.c_int]),
        "normpre_destroy": (None, [P]),
        "normpre_last_error": (ctypes.c_char_p, [P]),
        "normpre_validate": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, i64p, hpp, ctypes.c_char_p, ctypes.c_int]),
        "normpre_step": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int, ctypes.POINTER(P), ctypes.POINTER(P),
                                        ctypes.POINTER(P), i64p, hpp, P]),
        "normpre_debug_fetch": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int, P, ctypes.c_int64, i64p]),
        "normpre_sketch_omega": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int64,
                                                ctypes.c_int32, P, P]),
        "normpre_kernel_stats": (ctypes.c_int, [P, ctypes.c_int, i64p, ctypes.POINTER(ctypes.c_double),
                                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                                ctypes.POINTER(ctypes.c_double), ctypes.c_int]),
        "normpre_version": (ctypes.c_char_p, []),
        "normpre_spectrum": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, P, P, hpp,
                                            ctypes.POINTER(ctypes.c_double), P]),
        "normpre_energy_split": (ctypes.c_int, [ctypes.POINTER(ctypes.c_double), ctypes.c_int64, ctypes.c_int32,
                                                ctypes.POINTER(ctypes.c_double)]),
        "normpre_descent_alignment": (ctypes.c_int, [P, ctypes.c_int, ctypes.POINTER(P), ctypes.POINTER(P),
                                                     ctypes.POINTER(P), i64p, ctypes.c_float, ctypes.c_float,
                                                     ctypes.POINTER(ctypes.c_double),
                                                     ctypes.POINTER(ctypes.c_double), P]),
        "normpre_nonfinite_counts": (ctypes.c_int, [P, i64p, ctypes.c_int]),
        "normpre_stream_ceiling": (ctypes.c_int, [ctypes.c_int, ctypes.c_int64, P, P, P, P, P, P]),
        "normpre_workspace_size": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, i64p, hpp, i64p]),
        "normpre_reserve": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int, i64p, hpp, P]),
        "normpre_workspace_bytes": (ctypes.c_int, [P, i64p]),
        "normpre_step_noalloc": (ctypes.c_int, [P, ctypes.c_int, ctypes.c_int, ctypes.POINTER(P), ctypes.POINTER(P),
                                                ctypes.POINTER(P), i64p, hpp, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(code: int, ctx=None):
    if code != NORMPRE_OK:
        raise NormPreError(code, normpre_last_error(ctx))


def _ptr(x) -> int:
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream_handle(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------- entry points
def normpre_version() -> str:
    return load_library().normpre_version().decode()


def normpre_default_hparams(**overrides) -> normpre_hparams:
    hp = normpre_hparams()
    _check(load_library().normpre_default_hparams(ctypes.byref(hp)))
    for k, v in overrides.items():
        if k == "ns_coeffs":
            hp.ns_coeffs = (ctypes.c_float * 3)(*v)
        else:
            setattr(hp, k, v)
    return hp


def normpre_init(device: int = 0):
    ctx = ctypes.c_void_p()
    _check(load_library().normpre_init(ctypes.byref(ctx), int(device)))
    return ctx


def normpre_destroy(ctx) -> None:
    if ctx:
        load_library().normpre_destroy(ctx)


def normpre_last_error(ctx=None) -> str:
    s = load_library().normpre_last_error(ctx)
    return s.decode() if s else ""


def _shapes_array(shapes: Sequence[Sequence[int]]):
    flat = [int(v) for mn in shapes for v in mn]
    return (ctypes.c_int64 * max(1, len(flat)))(*flat)


def normpre_validate(variant: int, shapes, hp: normpre_hparams):
    """Host-only check; returns (code, message)."""
    buf = ctypes.create_string_buffer(512)
    arr = _shapes_array(shapes) if shapes is not None else None
    code = load_library().normpre_validate(int(variant), 0 if shapes is None else len(shapes), arr,
                                           ctypes.byref(hp) if hp is not None else None, buf, 512)
    return code, buf.value.decode()


def _step_args(params, grads, momentum, shapes):
    n = len(params)
    if shapes is None:
        shapes = [tuple(p.shape) for p in params]
    P = ctypes.c_void_p
    pw = (P * max(1, n))(*[_ptr(x) for x in params])
    pg = (P * max(1, n))(*[_ptr(x) for x in grads])
    pm = (P * max(1, n))(*[_ptr(x) for x in momentum])
    return n, pw, pg, pm, _shapes_array(shapes)


def normpre_step(ctx, variant: int, params, grads, momentum, hp: normpre_hparams, stream=None,
                 shapes=None) -> None:
    """One NormPre step on lists of fp32 device tensors (or raw pointers + shapes)."""
    n, pw, pg, pm, sh = _step_args(params, grads, momentum, shapes)
    code = load_library().normpre_step(ctx, int(variant), n, pw, pg, pm, sh, ctypes.byref(hp),
                                       _stream_handle(stream))
    _check(code, ctx)


def normpre_step_noalloc(ctx, variant: int, params, grads, momentum, hp: normpre_hparams, stream=None,
                         shapes=None) -> None:
    """normpre_step through the library's static scratch array (no allocation)."""
    n, pw, pg, pm, sh = _step_args(params, grads, momentum, shapes)
    code = load_library().normpre_step_noalloc(ctx, int(variant), n, pw, pg, pm, sh, ctypes.byref(hp),
                                               _stream_handle(stream))
    _check(code, ctx)


def normpre_nonfinite_counts(ctx, num_mats: int) -> np.ndarray:
    """Per-matrix non-finite entry counts of the last step made with
    NORMPRE_FLAG_CHECK_FINITE."""
    out = np.zeros(max(1, num_mats), dtype=np.int64)
    _check(load_library().normpre_nonfinite_counts(ctx, out.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                                    int(num_mats)), ctx)
    return out[:num_mats]


def normpre_stream_ceiling(mix: int, a, b, c, out32, out16, stream=None) -> None:
    """Streaming reference kernel with a normalization pass's byte mix
    (fp32 tensors a, b, c, out32 and an fp16 out16 of the same length)."""
    n = a.numel()
    vp = lambda x: ctypes.c_void_p(_ptr(x)) if x is not None else None  # noqa: E731
    _check(load_library().normpre_stream_ceiling(int(mix), n, vp(a), vp(b), vp(c), vp(out32), vp(out16),
                                                 _stream_handle(stream)))


def normpre_workspace_size(variant: int, shapes, hp: normpre_hparams) -> int:
    out = ctypes.c_int64()
    _check(load_library().normpre_workspace_size(int(variant), len(shapes), _shapes_array(shapes),
                                                 ctypes.byref(hp), ctypes.byref(out)))
    return out.value


def normpre_reserve(ctx, variant: int, shapes, hp: normpre_hparams, stream=None) -> None:
    code = load_library().normpre_reserve(ctx, int(variant), len(shapes), _shapes_array(shapes), ctypes.byref(hp),
                                          _stream_handle(stream))
    _check(code, ctx)


def normpre_workspace_bytes(ctx) -> int:
    out = ctypes.c_int64()
    _check(load_library().normpre_workspace_bytes(ctx, ctypes.byref(out)), ctx)
    return out.value


def normpre_debug_fetch(ctx, index: int, what: int, count: int, dtype=np.float32) -> np.ndarray:
    out = np.empty(count, dtype=dtype)
    written = ctypes.c_int64()
    code = load_library().normpre_debug_fetch(ctx, int(index), int(what), out.ctypes.data_as(ctypes.c_void_p),
                                              out.nbytes, ctypes.byref(written))
    _check(code, ctx)
    return out[: written.value // out.itemsize]


def normpre_sketch_omega(seed: int, step: int, matrix_id: int, b: int, ell: int, out, stream=None) -> None:
    code = load_library().normpre_sketch_omega(ctypes.c_uint64(seed), int(step), int(matrix_id), int(b), int(ell),
                                               ctypes.c_void_p(_ptr(out)), _stream_handle(stream))
    _check(code)


def normpre_kernel_stats(ctx, kclass: int, reset: bool = False) -> dict:
    launches = ctypes.c_int64()
    ms, flops, xflops, nbytes = ctypes.c_double(), ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    code = load_library().normpre_kernel_stats(ctx, int(kclass), ctypes.byref(launches), ctypes.byref(ms),
                                               ctypes.byref(flops), ctypes.byref(xflops), ctypes.byref(nbytes),
                                               int(bool(reset)))
    _check(code, ctx)
    return {"launches": launches.value, "ms": ms.value, "flops": flops.value, "exec_flops": xflops.value,
            "bytes": nbytes.value}


def normpre_spectrum(ctx, which: int, w, m, hp: normpre_hparams, stream=None) -> np.ndarray:
    """Eigenvalues (descending) of Gamma or of the trace-matched G_X of one
    matrix in hp's active orientation; w, m: 2-D fp32 device tensors."""
    rows, cols = (int(v) for v in w.shape)
    a = rows if (hp.orientation == NORMPRE_ORIENT_ROW or
                 (hp.orientation == NORMPRE_ORIENT_ALTERNATING and hp.step % 2 == 0)) else cols
    out = np.empty(a, dtype=np.float64)
    code = load_library().normpre_spectrum(ctx, int(which), rows, cols, ctypes.c_void_p(_ptr(w)),
                                           ctypes.c_void_p(_ptr(m)), ctypes.byref(hp),
                                           out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                           _stream_handle(stream))
    _check(code, ctx)
    return out


def normpre_descent_alignment(ctx, grads, w_before, w_after, lr: float, weight_decay: float, stream=None):
    """(per-matrix cosines, mean) of App. A's descent alignment; lists of 2-D
    fp32 device tensors (gradients, weights before and after the step)."""
    n = len(grads)
    P = ctypes.c_void_p
    shapes = [tuple(g.shape) for g in grads]
    pg = (P * max(1, n))(*[_ptr(x) for x in grads])
    pb = (P * max(1, n))(*[_ptr(x) for x in w_before])
    pa = (P * max(1, n))(*[_ptr(x) for x in w_after])
    cos = np.zeros(max(1, n), dtype=np.float64)
    mean = ctypes.c_double()
    code = load_library().normpre_descent_alignment(ctx, n, pg, pb, pa, _shapes_array(shapes), float(lr),
                                                    float(weight_decay),
                                                    cos.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                                    ctypes.byref(mean), _stream_handle(stream))
    _check(code, ctx)
    return cos[:n], mean.value


def normpre_energy_split(eigs, count: int, rank: int) -> np.ndarray:
    """[E_top, E_remain, E_sub, E_global] of the first `count` eigenvalues."""
    e = np.ascontiguousarray(np.asarray(eigs, dtype=np.float64))
    if count > e.size:
        raise ValueError("count exceeds the number of eigenvalues")
    out = np.zeros(4, dtype=np.float64)
    code = load_library().normpre_energy_split(e.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), int(count),
                                               int(rank), out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    _check(code)
    return out


class NormPre:
    """Small stateful wrapper: one context, momentum buffers and step counter
    for a list of 2-D fp32 CUDA/HIP tensors (the hidden weight matrices)."""

    def __init__(self, params, variant: str = "G", device: int | None = None, **hparams):
        import torch
        self.params = list(params)
        self.variant = VARIANTS[variant.upper()]
        dev = self.params[0].device.index if device is None else device
        self.ctx = normpre_init(0 if dev is None else dev)
        self.hp = normpre_default_hparams(**hparams)
        self.momentum = [torch.zeros_like(p) for p in self.params]
        self.t = int(hparams.get("step", 0))

    def step(self, grads, stream=None):
        self.hp.step = self.t
        normpre_step(self.ctx, self.variant, self.params, grads, self.momentum, self.hp, stream)
        self.t += 1

    def close(self):
        normpre_destroy(self.ctx)
        self.ctx = None

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                self.close()
        except Exception:
            pass
