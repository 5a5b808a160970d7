"""Python binding of ``libxcache.so`` (the C ABI in ``include/xcache.h``).

Argument marshalling only: every step of the cached chunk forward runs in the
library's HIP kernels.  Device buffers are passed as raw addresses (for
example ``tensor.data_ptr()`` of a CUDA/HIP PyTorch tensor) and the stream as
a ``hipStream_t`` handle (``torch.cuda.current_stream().cuda_stream``).
If the library has not been built, loading raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxcache.so")

XC_OK, XC_ERR_INVALID_ARG, XC_ERR_STATE, XC_ERR_OOM, XC_ERR_HIP, XC_ERR_UNSUPPORTED = range(6)
XC_F32, XC_BF16 = 0, 1
XC_STEP0_OFF, XC_STEP0_FORCE, XC_STEP0_STRICT = 0, 1, 2
XC_FP_GRID3D, XC_FP_LINSPACE1D = 0, 1
XC_FP_REFRESH_EVERY, XC_FP_REFRESH_ON_COMPUTE = 0, 1
XC_FORCE_FULL = 1
XC_DEC_COMPUTE, XC_DEC_SKIP, XC_DEC_FORCED, XC_DEC_NONE = 0, 1, 2, 255
XC_CACHE_RESIDUAL, XC_CACHE_KEYS, XC_CACHE_VALUES = 0, 1, 2
XC_MAX_GROUPS = 8
(XC_KERN_ATTENTION, XC_KERN_GEMM_QKV, XC_KERN_GEMM_OPROJ, XC_KERN_GEMM_UP, XC_KERN_GEMM_DOWN,
 XC_KERN_GATE, XC_KERN_GATE_DECIDE, XC_KERN_SKIP_ADD, XC_KERN_LN_MOD, XC_KERN_QK_NORM, XC_KERN_ADALN,
 XC_KERN_CROSS_Q, XC_KERN_CROSS_ATTENTION, XC_KERN_CROSS_O, XC_KERN_COUNT) = range(15)

KERNEL_NAMES = ["attention", "gemm_qkv", "gemm_oproj", "gemm_up", "gemm_down", "gate", "gate_decide", "skip_add",
                "ln_mod", "qk_norm", "adaln", "cross_q", "cross_attention", "cross_o"]

EXPORTED = ["xc_status_string", "xc_init", "xc_forward_chunk", "xc_forward_chunk_noalloc", "xc_kv_update",
            "xc_set_condition", "xc_read_cache", "xc_stats",
            "xc_reset", "xc_destroy", "xc_axpby", "xc_fingerprint_rows", "xc_profile", "xc_kernel_times",
            "xc_mfma_rate", "xc_lds_dma_rate"]


class ViewGroupC(ctypes.Structure):
    _fields_ = [("views", ctypes.c_int32), ("frames", ctypes.c_int32),
                ("height", ctypes.c_int32), ("width", ctypes.c_int32)]


class ModelConfigC(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("mlp_hidden", ctypes.c_int32), ("temb_dim", ctypes.c_int32),
                ("action_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("n_steps", ctypes.c_int32),
                ("kv_window", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("groups", ViewGroupC * XC_MAX_GROUPS), ("rope", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("cond_len", ctypes.c_int32)]


class GateConfigC(ctypes.Structure):
    _fields_ = [("enabled", ctypes.c_int32), ("fp_budget", ctypes.c_int32), ("warmup", ctypes.c_int32),
                ("front_anchors", ctypes.c_int32), ("back_anchors", ctypes.c_int32),
                ("adaptive", ctypes.c_int32), ("tau_floor", ctypes.c_float), ("margin", ctypes.c_float),
                ("alpha", ctypes.c_float), ("tau_cos_fixed", ctypes.c_float), ("tau_dev", ctypes.c_float),
                ("eps", ctypes.c_float), ("max_stale", ctypes.c_int32), ("step0_mode", ctypes.c_int32),
                ("tau_strict0", ctypes.c_float), ("kv_protect", ctypes.c_int32), ("fp_mode", ctypes.c_int32),
                ("fp_refresh", ctypes.c_int32)]


class StatsC(ctypes.Structure):
    _fields_ = [("generations", ctypes.c_int64), ("evals_post_warmup", ctypes.c_int64),
                ("gated_evals", ctypes.c_int64), ("skips", ctypes.c_int64),
                ("kv_block_evals", ctypes.c_int64), ("last_step", ctypes.c_int32)]


class XCacheError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what} failed: {xc_status_string(status)}")


_lib: Optional[ctypes.CDLL] = None


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load ``libxcache.so`` (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with `python -m paper_2604_20289_amd.build` "
                           "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(p)
    vp, i32, u32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "xc_status_string": (ctypes.c_char_p, [i32]),
        "xc_init": (i32, [P(ModelConfigC), P(GateConfigC), vp, sz, vp, P(vp)]),
        "xc_forward_chunk": (i32, [vp, i32, f32, vp, vp, vp, u32]),
        "xc_forward_chunk_noalloc": (i32, [vp, i32, f32, vp, vp, vp, u32]),
        "xc_kv_update": (i32, [vp, f32, vp, vp, vp]),
        "xc_set_condition": (i32, [vp, vp, i32]),
        "xc_read_cache": (i32, [vp, i32, i32, i32, vp, sz]),
        "xc_stats": (i32, [vp, P(StatsC), vp, vp, vp, vp, vp, vp]),
        "xc_reset": (i32, [vp]),
        "xc_destroy": (i32, [vp]),
        "xc_axpby": (i32, [vp, f32, vp, f32, vp, vp, sz]),
        "xc_fingerprint_rows": (i32, [P(ModelConfigC), P(GateConfigC), vp, sz, P(sz)]),
        "xc_profile": (i32, [vp, i32]),
        "xc_kernel_times": (i32, [vp, i32, P(ctypes.c_int64), P(ctypes.c_double), i32]),
        "xc_mfma_rate": (i32, [i32, i32, vp, P(ctypes.c_double)]),
        "xc_lds_dma_rate": (i32, [i32, vp, P(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def xc_status_string(status: int) -> str:
    return load_library().xc_status_string(status).decode()


def _check(status: int, what: str):
    if status != XC_OK:
        raise XCacheError(status, what)


def model_config(model) -> ModelConfigC:
    """Marshal a model description (attributes as in ``xc_model_config``;
    ``dtype`` may be "f32"/"bf16" or XC_F32/XC_BF16; ``groups`` a sequence of
    objects with views/frames/height/width)."""
    c = ModelConfigC()
    c.n_blocks, c.hidden, c.n_heads = model.n_blocks, model.hidden, model.n_heads
    c.head_dim, c.mlp_hidden = model.head_dim, model.mlp_hidden
    c.temb_dim, c.action_dim = model.temb_dim, model.action_dim
    dt = model.dtype
    c.dtype = {"f32": XC_F32, "bf16": XC_BF16}.get(dt, dt) if isinstance(dt, str) else int(dt)
    c.n_steps, c.kv_window = model.n_steps, model.kv_window
    groups = list(model.groups)
    c.n_groups = len(groups)
    for i, g in enumerate(groups[:XC_MAX_GROUPS]):
        c.groups[i] = ViewGroupC(g.views, g.frames, g.height, g.width)
    c.rope = getattr(model, "rope", 0)
    c.rope_theta = getattr(model, "rope_theta", 10000.0)
    c.cond_len = getattr(model, "cond_len", 0)
    return c


def gate_config(gate) -> GateConfigC:
    """Marshal gate hyper-parameters (attributes as in ``xc_gate_config``)."""
    c = GateConfigC()
    for name, _ in GateConfigC._fields_:
        setattr(c, name, getattr(gate, name))
    return c


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)}")


def xc_init(model, gate, weights: np.ndarray, stream: int = 0) -> int:
    lib = load_library()
    w = np.ascontiguousarray(weights, dtype=np.float32)
    h = ctypes.c_void_p()
    mc, gc = model_config(model), gate_config(gate)
    _check(lib.xc_init(ctypes.byref(mc), ctypes.byref(gc), w.ctypes.data, w.nbytes, stream or None,
                       ctypes.byref(h)), "xc_init")
    return h.value


def xc_forward_chunk(h: int, step: int, timestep: float, action: np.ndarray, x_in, x_out, flags: int = 0):
    a = np.ascontiguousarray(action, dtype=np.float32)
    _check(load_library().xc_forward_chunk(h, step, timestep, a.ctypes.data, _ptr(x_in), _ptr(x_out), flags),
           "xc_forward_chunk")


def xc_forward_chunk_noalloc(h: int, step: int, timestep: float, action: np.ndarray, x_in, x_out, flags: int = 0):
    a = np.ascontiguousarray(action, dtype=np.float32)
    _check(load_library().xc_forward_chunk_noalloc(h, step, timestep, a.ctypes.data, _ptr(x_in), _ptr(x_out), flags),
           "xc_forward_chunk_noalloc")


def xc_kv_update(h: int, timestep: float, action: np.ndarray, x_clean, x_out=None):
    a = np.ascontiguousarray(action, dtype=np.float32)
    _check(load_library().xc_kv_update(h, timestep, a.ctypes.data, _ptr(x_clean), _ptr(x_out)), "xc_kv_update")


def xc_set_condition(h: int, cond: np.ndarray):
    c = np.ascontiguousarray(cond, dtype=np.float32)
    if c.ndim != 2:
        raise ValueError("condition tokens must be [n_tokens, hidden]")
    _check(load_library().xc_set_condition(h, c.ctypes.data, c.shape[0]), "xc_set_condition")


def xc_read_cache(h: int, kind: int, step: int, block: int, out, n_floats: int):
    _check(load_library().xc_read_cache(h, kind, step, block, _ptr(out), n_floats), "xc_read_cache")


def xc_stats(h: int, n_steps: int, n_blocks: int) -> dict:
    st = StatsC()
    counts = np.zeros(n_steps * n_blocks, np.int32)
    dec = np.zeros(n_blocks, np.uint8)
    cos = np.zeros(n_blocks, np.float32)
    dev = np.zeros(n_blocks, np.float32)
    tau = np.zeros(n_blocks, np.float32)
    ema = np.zeros(n_steps * n_blocks, np.float32)
    _check(load_library().xc_stats(h, ctypes.byref(st), counts.ctypes.data, dec.ctypes.data, cos.ctypes.data,
                                   dev.ctypes.data, tau.ctypes.data, ema.ctypes.data), "xc_stats")
    return {"generations": st.generations, "evals_post_warmup": st.evals_post_warmup,
            "gated_evals": st.gated_evals, "skips": st.skips, "kv_block_evals": st.kv_block_evals,
            "last_step": st.last_step, "skip_counts": counts.reshape(n_steps, n_blocks),
            "last_decision": dec, "last_cos": cos, "last_dev": dev, "last_tau": tau,
            "ema": ema.reshape(n_steps, n_blocks)}


def xc_reset(h: int):
    _check(load_library().xc_reset(h), "xc_reset")


def xc_destroy(h: int):
    _check(load_library().xc_destroy(h), "xc_destroy")


def xc_axpby(h: int, a: float, x, b: float, y, out, n: int):
    _check(load_library().xc_axpby(h, a, _ptr(x), b, _ptr(y), _ptr(out), n), "xc_axpby")


def xc_fingerprint_rows(model, gate) -> np.ndarray:
    lib = load_library()
    mc, gc = model_config(model), gate_config(gate)
    n = ctypes.c_size_t()
    _check(lib.xc_fingerprint_rows(ctypes.byref(mc), ctypes.byref(gc), None, 0, ctypes.byref(n)),
           "xc_fingerprint_rows")
    rows = np.zeros(n.value, np.int32)
    _check(lib.xc_fingerprint_rows(ctypes.byref(mc), ctypes.byref(gc), rows.ctypes.data, rows.size,
                                   ctypes.byref(n)), "xc_fingerprint_rows")
    return rows


def xc_profile(h: int, enable: bool):
    _check(load_library().xc_profile(h, 1 if enable else 0), "xc_profile")


def xc_kernel_times(h: int, kind: int, clear: bool = False):
    n = ctypes.c_int64()
    ms = ctypes.c_double()
    _check(load_library().xc_kernel_times(h, kind, ctypes.byref(n), ctypes.byref(ms), 1 if clear else 0),
           "xc_kernel_times")
    return n.value, ms.value


def xc_mfma_rate(shape: int, random_operands: bool, stream: Optional[int] = None) -> float:
    """TFLOP/s of the bf16 MFMA loop: shape 0 32x32x16, 1 16x16x32 (operands in registers); 2-4 the
    attention loop's mix at its occupancy (2 + LDS operand reads, 3 + softmax VALU, 4 both)."""
    t = ctypes.c_double()
    _check(load_library().xc_mfma_rate(shape, 1 if random_operands else 0, stream or None, ctypes.byref(t)),
           "xc_mfma_rate")
    return t.value


def xc_lds_dma_rate(row_bytes: int, stream: Optional[int] = None) -> float:
    """TB/s of the global -> LDS request stream with row_bytes (64, 128, 256) per row and request."""
    t = ctypes.c_double()
    _check(load_library().xc_lds_dma_rate(row_bytes, stream or None, ctypes.byref(t)), "xc_lds_dma_rate")
    return t.value


class XCache:
    """Owns one library handle bound to a HIP stream.

    ``x_in``/``x_out`` are float32 device tensors of shape [L, C].
    """

    def __init__(self, model, gate, weights: np.ndarray, stream: int = 0):
        self.model = model
        self.gate = gate
        self.S, self.B = model.n_steps, model.n_blocks
        self.h = xc_init(model, gate, weights, stream)

    def forward_chunk(self, step: int, timestep: float, action, x_in, x_out, flags: int = 0):
        xc_forward_chunk(self.h, step, timestep, action, x_in, x_out, flags)

    def forward_chunk_noalloc(self, step: int, timestep: float, action, x_in, x_out, flags: int = 0):
        xc_forward_chunk_noalloc(self.h, step, timestep, action, x_in, x_out, flags)

    def set_condition(self, cond):
        xc_set_condition(self.h, cond)

    def kv_update(self, timestep: float, action, x_clean, x_out=None):
        xc_kv_update(self.h, timestep, action, x_clean, x_out)

    def stats(self) -> dict:
        return xc_stats(self.h, self.S, self.B)

    def read_cache(self, kind: int, step: int, block: int, out):
        """Copy a cache into the float32 device tensor ``out`` (see xc_read_cache)."""
        xc_read_cache(self.h, kind, step, block, out, out.numel())

    def reset(self):
        xc_reset(self.h)

    def axpby(self, a, x, b, y, out, n):
        xc_axpby(self.h, a, x, b, y, out, n)

    def profile(self, enable: bool):
        xc_profile(self.h, enable)

    def kernel_times(self, kind: int, clear: bool = False):
        return xc_kernel_times(self.h, kind, clear)

    def close(self):
        if self.h:
            xc_destroy(self.h)
            self.h = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
