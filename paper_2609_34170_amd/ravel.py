"""Thin ctypes binding of libravel (include/ravel.h).

Argument marshalling only: every step of the rolling denoise path runs in the
HIP kernels of libravel.so.  Device buffers are torch tensors on the GPU (used
for memory and streams only); host arrays are numpy arrays.  The library must
be built first (``paper_2609_34170_amd.build.build()``); importing this module
without it raises immediately -- there is no CPU fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Tuple

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libravel.so")

F32, BF16 = 0, 1
TRANSFORMER, ANALYTIC_OT, ANALYTIC_LINEAR = 0, 1, 2
OPT_SYNC_CONTEXT, OPT_USE_GRAPH, OPT_DEBUG, OPT_PERSISTENT, OPT_FAIL_LAYERS = 1, 2, 3, 4, 5
Q_GRAPHS, Q_PERSISTENT, Q_PHASES, Q_STEPS = 1, 2, 3, 4

_STATUS = {0: "OK", -1: "E_INVALID", -2: "E_NOMEM", -3: "E_HIP", -4: "E_SHAPE", -5: "E_STATE"}


class RavelError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class RavelConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "layers", "width", "n_q_heads", "n_kv_heads", "head_dim", "mlp_dim", "horizon", "action_dim",
        "prefix_len", "n_fop", "fop_obs_dim", "fop_stride", "dtype", "model_kind")] + [
        ("delta_bias", ctypes.c_float), ("rms_eps", ctypes.c_float), ("offset_mode", ctypes.c_int32),
        ("rope_base", ctypes.c_float)]


class RavelTensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("dtype", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("dims", ctypes.c_int64 * 4), ("data", ctypes.c_void_p)]


class KernelRecord(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("bytes", ctypes.c_double), ("flops", ctypes.c_double),
                ("ms", ctypes.c_float)]


SYMBOLS = [
    "ravel_create", "ravel_destroy", "ravel_model_weight_bytes", "ravel_buffer_create",
    "ravel_buffer_destroy", "ravel_buffer_set_option", "ravel_context_acquire", "ravel_set_context",
    "ravel_step", "ravel_step_state", "ravel_set_relative_dims", "ravel_full_denoise", "ravel_train_loss",
    "ravel_fop_encode", "ravel_fop_encode_noalloc", "ravel_buffer_sync", "ravel_debug_state",
    "ravel_publish_log", "ravel_buffer_query",
    "ravel_buffer_save", "ravel_buffer_load", "ravel_profile_step", "ravel_last_error",
]

_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2609_34170_amd.build.build()")
    lib = ctypes.CDLL(path)
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    sig = {
        "ravel_create": ([ctypes.POINTER(RavelConfig), ctypes.POINTER(RavelTensor), i32, ctypes.POINTER(vp)], i32),
        "ravel_destroy": ([vp], None),
        "ravel_model_weight_bytes": ([vp], i64),
        "ravel_buffer_create": ([vp, i32, u64, ctypes.POINTER(vp)], i32),
        "ravel_buffer_destroy": ([vp], None),
        "ravel_buffer_set_option": ([vp, i32, i64], i32),
        "ravel_context_acquire": ([vp, i32, ctypes.POINTER(vp), ctypes.POINTER(vp), vp], i32),
        "ravel_set_context": ([vp, i32, vp, vp, i64, vp], i32),
        "ravel_step": ([vp, vp, vp, vp], i32),
        "ravel_full_denoise": ([vp, i32, vp, vp, vp, vp], i32),
        "ravel_train_loss": ([vp, vp, vp, vp, vp, vp, vp, vp], i32),
        "ravel_set_relative_dims": ([vp, vp], i32),
        "ravel_step_state": ([vp, vp, vp, vp, vp], i32),
        "ravel_fop_encode": ([vp, vp, vp, vp], i32),
        "ravel_fop_encode_noalloc": ([vp, i32, vp, vp, vp], i32),
        "ravel_buffer_sync": ([vp], i32),
        "ravel_debug_state": ([vp, vp, vp, vp], i32),
        "ravel_publish_log": ([vp, vp, ctypes.POINTER(i32)], i32),
        "ravel_buffer_query": ([vp, i32, ctypes.POINTER(i64)], i32),
        "ravel_buffer_save": ([vp, vp, ctypes.POINTER(ctypes.c_size_t)], i32),
        "ravel_buffer_load": ([vp, vp, ctypes.c_size_t], i32),
        "ravel_profile_step": ([vp, vp, vp, vp, ctypes.POINTER(KernelRecord), ctypes.POINTER(i32)], i32),
        "ravel_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        msg = load_library().ravel_last_error().decode(errors="replace")
        raise RavelError(status, msg)


def _ptr(x) -> Optional[int]:
    """Device/host address of a torch tensor, numpy array or raw int (None -> NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("host arrays must be C-contiguous")
        return x.ctypes.data
    if hasattr(x, "data_ptr"):
        if not x.is_contiguous():
            raise ValueError("tensors must be contiguous")
        return x.data_ptr()
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_config(shape) -> RavelConfig:
    c = RavelConfig()
    for f, _ in RavelConfig._fields_:
        setattr(c, f, getattr(shape, f))
    return c


class Model:
    """A model on the current HIP device (ravel_create)."""

    def __init__(self, shape, weights: Dict[str, np.ndarray]):
        lib = load_library()
        self.shape = shape
        self.cfg = make_config(shape)
        keep: List[np.ndarray] = []
        arr = (RavelTensor * max(len(weights), 1))()
        for i, (name, a) in enumerate(weights.items()):
            a = np.ascontiguousarray(a, dtype=np.float32)
            keep.append(a)
            t = arr[i]
            t.name = name.encode()
            t.dtype = F32
            t.rank = a.ndim
            for d in range(a.ndim):
                t.dims[d] = a.shape[d]
            t.data = a.ctypes.data
        h = ctypes.c_void_p()
        _check(lib.ravel_create(ctypes.byref(self.cfg), arr, len(weights), ctypes.byref(h)))
        self.h = h

    def fop_encode_noalloc(self, batch: int, obs, fop_tokens, stream=None):
        """The FOP encoder without a buffer and without allocating (fixed device scratch)."""
        _check(load_library().ravel_fop_encode_noalloc(self.h, int(batch), _ptr(obs), _ptr(fop_tokens),
                                                        _stream(stream)))

    @property
    def weight_bytes(self) -> int:
        return int(load_library().ravel_model_weight_bytes(self.h))

    def close(self):
        if getattr(self, "h", None):
            load_library().ravel_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Buffer:
    """Rolling state of B environments (ravel_buffer_create)."""

    def __init__(self, model: Model, batch: int, seed: int = 0):
        lib = load_library()
        self.model = model
        self.B = batch
        self.seed = seed
        h = ctypes.c_void_p()
        _check(lib.ravel_buffer_create(model.h, batch, seed, ctypes.byref(h)))
        self.h = h

    # -- options -----------------------------------------------------------
    def set_option(self, option: int, value: int):
        _check(load_library().ravel_buffer_set_option(self.h, option, int(value)))

    # -- context plane -------------------------------------------------------
    def acquire(self, env: int, stream=None) -> Tuple[int, int]:
        k, v = ctypes.c_void_p(), ctypes.c_void_p()
        _check(load_library().ravel_context_acquire(self.h, env, ctypes.byref(k), ctypes.byref(v),
                                                    _stream(stream)))
        return k.value, v.value

    def set_context(self, env: int, k, v, t_obs: int, stream=None):
        _check(load_library().ravel_set_context(self.h, env, _ptr(k), _ptr(v), int(t_obs), _stream(stream)))

    # -- hot path ----------------------------------------------------------
    def step(self, fop_tokens, action_out, stream=None):
        _check(load_library().ravel_step(self.h, _ptr(fop_tokens), _ptr(action_out), _stream(stream)))

    def set_relative_dims(self, mask):
        m = None
        if mask is not None:
            m = np.ascontiguousarray(np.asarray(mask, dtype=np.int32))
            self._mask = m
        _check(load_library().ravel_set_relative_dims(self.h, None if m is None else m.ctypes.data))

    def step_state(self, fop_tokens, state, action_out, stream=None):
        _check(load_library().ravel_step_state(self.h, _ptr(fop_tokens), _ptr(state), _ptr(action_out),
                                               _stream(stream)))

    def full_denoise(self, steps: int, fop_tokens, noise, chunk_out, stream=None):
        _check(load_library().ravel_full_denoise(self.h, int(steps), _ptr(fop_tokens), _ptr(noise), _ptr(chunk_out),
                                                 _stream(stream)))

    def train_loss(self, target, noise, ages, fop_tokens, loss_out, v_out=None, stream=None):
        _check(load_library().ravel_train_loss(self.h, _ptr(target), _ptr(noise), _ptr(ages), _ptr(fop_tokens),
                                               _ptr(loss_out), _ptr(v_out), _stream(stream)))

    def fop_encode(self, obs, fop_tokens, stream=None):
        _check(load_library().ravel_fop_encode(self.h, _ptr(obs), _ptr(fop_tokens), _stream(stream)))

    def profile_step(self, fop_tokens, action_out, stream=None, capacity: int = 4096):
        recs = (KernelRecord * capacity)()
        n = ctypes.c_int32(capacity)
        _check(load_library().ravel_profile_step(self.h, _ptr(fop_tokens), _ptr(action_out), _stream(stream),
                                                 recs, ctypes.byref(n)))
        return [(recs[i].name.decode(), recs[i].bytes, recs[i].flops, recs[i].ms) for i in range(n.value)]

    # -- inspection --------------------------------------------------------
    def sync(self):
        _check(load_library().ravel_buffer_sync(self.h))

    def debug_state(self):
        s = self.model.shape
        X = np.zeros((self.B, s.horizon, s.action_dim), dtype=np.float32)
        t = ctypes.c_int64()
        t_obs = np.zeros(self.B, dtype=np.int64)
        _check(load_library().ravel_debug_state(self.h, X.ctypes.data, ctypes.addressof(t), t_obs.ctypes.data))
        return X, int(t.value), t_obs

    def publish_log(self) -> List[Tuple[int, int, int]]:
        lib = load_library()
        n = ctypes.c_int32(0)
        _check(lib.ravel_publish_log(self.h, None, ctypes.byref(n)))
        cap = max(n.value, 1)
        buf = np.zeros((cap, 3), dtype=np.int64)
        n = ctypes.c_int32(cap)
        _check(lib.ravel_publish_log(self.h, buf.ctypes.data, ctypes.byref(n)))
        return [tuple(int(x) for x in buf[i]) for i in range(n.value)]

    def query(self, key: int) -> int:
        v = ctypes.c_int64(0)
        _check(load_library().ravel_buffer_query(self.h, int(key), ctypes.byref(v)))
        return int(v.value)

    def save(self) -> bytes:
        lib = load_library()
        n = ctypes.c_size_t(0)
        _check(lib.ravel_buffer_save(self.h, None, ctypes.byref(n)))
        blob = np.zeros(n.value, dtype=np.uint8)
        _check(lib.ravel_buffer_save(self.h, blob.ctypes.data, ctypes.byref(n)))
        return blob.tobytes()

    def load(self, blob: bytes):
        a = np.frombuffer(blob, dtype=np.uint8).copy()
        _check(load_library().ravel_buffer_load(self.h, a.ctypes.data, a.size))

    def close(self):
        if getattr(self, "h", None):
            load_library().ravel_buffer_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
