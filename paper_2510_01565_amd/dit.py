"""Python binding of the C ABI in ``include/dit.h`` (ctypes; argument
marshalling only -- every step runs in the HIP library).

Device buffers are passed as torch tensors (their data pointers) or raw
integers; streams as torch streams, raw ``hipStream_t`` integers, or None for
torch's current stream.  The library must be built (``build.py``); importing
this module does not load it, the first call does, and fails loudly when the
shared library is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdit_mi355x.so")

DIT_OK, DIT_ERR_INVALID_ARG, DIT_ERR_UNSUPPORTED, DIT_ERR_WORKSPACE, DIT_ERR_HIP = range(5)
DIT_F32, DIT_BF16 = 0, 1
DIT_MAX_REQUESTS = 16
DIT_MAX_GRID = 256
DIT_FLAG_BATCH_INVARIANT = 1
DIT_NOALLOC_SCRATCH_BYTES = 256 << 20

EXPORTED = ("dit_weight_count", "dit_weight_manifest", "dit_workspace_size", "dit_step", "dit_step_noalloc",
            "dit_block_forward", "euler_update", "dit_attention_workspace_size", "dit_attention", "dit_linear",
            "dit_profile_start", "dit_profile_stop", "dit_profile_entry", "dit_last_error")


class DitError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"dit status {status}: {msg}")
        self.status = status


class dit_config(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int), ("heads", ctypes.c_int), ("head_dim", ctypes.c_int),
                ("mlp_ratio", ctypes.c_int), ("n_double", ctypes.c_int), ("n_single", ctypes.c_int),
                ("in_channels", ctypes.c_int), ("text_dim", ctypes.c_int), ("time_freq_dim", ctypes.c_int),
                ("tie_streams", ctypes.c_int), ("rope_theta", ctypes.c_float), ("ln_eps", ctypes.c_float),
                ("dtype", ctypes.c_int), ("flags", ctypes.c_int)]


class dit_batch(ctypes.Structure):
    _fields_ = [("n_req", ctypes.c_int), ("grid_h", ctypes.POINTER(ctypes.c_int)),
                ("grid_w", ctypes.POINTER(ctypes.c_int)), ("n_txt", ctypes.POINTER(ctypes.c_int)),
                ("t", ctypes.POINTER(ctypes.c_float))]


class dit_weights(ctypes.Structure):
    _fields_ = [("tensors", ctypes.POINTER(ctypes.c_void_p)), ("n_tensors", ctypes.c_int)]


_lib = None


def lib() -> ctypes.CDLL:
    """Loads the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing (run paper_2510_01565_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        vp, ip, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        L.dit_last_error.restype = ctypes.c_char_p
        L.dit_weight_count.argtypes = [ctypes.POINTER(dit_config), ctypes.POINTER(ctypes.c_int)]
        L.dit_weight_manifest.argtypes = [ctypes.POINTER(dit_config), ip, ctypes.POINTER(ctypes.c_char_p),
                                          ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_int)]
        L.dit_workspace_size.argtypes = [ctypes.POINTER(dit_config), ctypes.POINTER(dit_batch),
                                         ctypes.POINTER(ctypes.c_size_t)]
        L.dit_step.argtypes = [ctypes.POINTER(dit_config), ctypes.POINTER(dit_weights), ctypes.POINTER(dit_batch),
                               vp, vp, vp, vp, sz, vp]
        L.dit_step_noalloc.argtypes = [ctypes.POINTER(dit_config), ctypes.POINTER(dit_weights),
                                       ctypes.POINTER(dit_batch), vp, vp, vp, vp]
        L.dit_block_forward.argtypes = [ctypes.POINTER(dit_config), ctypes.POINTER(dit_weights), ip, ip,
                                        ctypes.POINTER(dit_batch), vp, vp, vp, sz, vp]
        L.euler_update.argtypes = [ctypes.POINTER(dit_batch), ip, ip, vp, vp, ctypes.POINTER(ctypes.c_float), vp]
        L.dit_attention_workspace_size.argtypes = [ctypes.POINTER(dit_batch), ip, ip, ip,
                                                   ctypes.POINTER(ctypes.c_size_t)]
        L.dit_attention.argtypes = [ctypes.POINTER(dit_batch), ip, ip, ip, vp, vp, vp, vp, vp, sz, vp]
        L.dit_linear.argtypes = [ip, ip, ip, ip, vp, vp, vp, vp, ip, vp]
        L.dit_profile_start.argtypes = []
        L.dit_profile_stop.argtypes = [ctypes.POINTER(ctypes.c_int)]
        L.dit_profile_entry.argtypes = [ip, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_long),
                                        ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                        ctypes.POINTER(ctypes.c_double)]
        for name in EXPORTED:
            if name != "dit_last_error":
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(st: int) -> None:
    if st != DIT_OK:
        raise DitError(st, lib().dit_last_error().decode())


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def make_config(shape, flags: int = 0) -> dit_config:
    """dit_config from a ``workloads.ModelShape``-like object; ``flags``: DIT_FLAG_* bits."""
    return dit_config(shape.hidden, shape.heads, shape.head_dim, shape.mlp_ratio, shape.n_double, shape.n_single,
                      shape.in_channels, shape.text_dim, shape.time_freq_dim, 1 if shape.tie_streams else 0,
                      float(shape.rope_theta), float(shape.ln_eps), DIT_BF16 if shape.dtype == "bf16" else DIT_F32,
                      flags)


class Batch:
    """Owns the host arrays of a dit_batch."""

    def __init__(self, grid_h: Sequence[int], grid_w: Sequence[int], n_txt: Sequence[int],
                 t: Optional[Sequence[float]] = None):
        n = len(grid_h)
        self.n = n
        self._gh = (ctypes.c_int * n)(*grid_h)
        self._gw = (ctypes.c_int * n)(*grid_w)
        self._nt = (ctypes.c_int * n)(*n_txt)
        self._t = (ctypes.c_float * n)(*t) if t is not None else None
        self.c = dit_batch(n, self._gh, self._gw, self._nt,
                           ctypes.cast(self._t, ctypes.POINTER(ctypes.c_float)) if self._t is not None else None)


class Weights:
    """Owns the pointer array of a dit_weights (tensors must stay alive)."""

    def __init__(self, tensors: Sequence):
        self.tensors = list(tensors)
        self._arr = (ctypes.c_void_p * len(tensors))(*[_ptr(t) for t in tensors])
        self.c = dit_weights(self._arr, len(tensors))


def weight_count(cfg: dit_config) -> int:
    n = ctypes.c_int()
    _check(lib().dit_weight_count(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def weight_manifest(cfg: dit_config) -> List[Tuple[str, Tuple[int, ...]]]:
    out = []
    for i in range(weight_count(cfg)):
        name = ctypes.c_char_p()
        shape = (ctypes.c_int * 2)()
        nd = ctypes.c_int()
        _check(lib().dit_weight_manifest(ctypes.byref(cfg), i, ctypes.byref(name), shape, ctypes.byref(nd)))
        out.append((name.value.decode(), tuple(shape[:nd.value])))
    return out


def workspace_size(cfg: dit_config, batch: Batch) -> int:
    n = ctypes.c_size_t()
    _check(lib().dit_workspace_size(ctypes.byref(cfg), ctypes.byref(batch.c), ctypes.byref(n)))
    return n.value


def dit_step(cfg: dit_config, w: Weights, batch: Batch, latents, text_emb, velocity, ws, ws_bytes: int,
             stream=None) -> None:
    _check(lib().dit_step(ctypes.byref(cfg), ctypes.byref(w.c), ctypes.byref(batch.c), _ptr(latents),
                          _ptr(text_emb), _ptr(velocity), _ptr(ws), ws_bytes, _stream(stream)))


def dit_step_noalloc(cfg: dit_config, w: Weights, batch: Batch, latents, text_emb, velocity, stream=None) -> None:
    _check(lib().dit_step_noalloc(ctypes.byref(cfg), ctypes.byref(w.c), ctypes.byref(batch.c), _ptr(latents),
                                  _ptr(text_emb), _ptr(velocity), _stream(stream)))


def dit_block_forward(cfg: dit_config, w: Weights, kind: int, index: int, batch: Batch, hidden, cond, ws,
                      ws_bytes: int, stream=None) -> None:
    _check(lib().dit_block_forward(ctypes.byref(cfg), ctypes.byref(w.c), kind, index, ctypes.byref(batch.c),
                                   _ptr(hidden), _ptr(cond), _ptr(ws), ws_bytes, _stream(stream)))


def euler_update(batch: Batch, channels: int, dtype: int, latents, velocity, dt: Sequence[float],
                 stream=None) -> None:
    arr = (ctypes.c_float * len(dt))(*dt)
    _check(lib().euler_update(ctypes.byref(batch.c), channels, dtype, _ptr(latents), _ptr(velocity), arr,
                              _stream(stream)))


def attention_workspace_size(batch: Batch, heads: int, head_dim: int, dtype: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().dit_attention_workspace_size(ctypes.byref(batch.c), heads, head_dim, dtype, ctypes.byref(n)))
    return n.value


def dit_attention(batch: Batch, heads: int, head_dim: int, dtype: int, q, k, v, o, ws, ws_bytes: int,
                  stream=None) -> None:
    _check(lib().dit_attention(ctypes.byref(batch.c), heads, head_dim, dtype, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                               _ptr(ws), ws_bytes, _stream(stream)))


def dit_linear(M: int, N: int, K: int, dtype: int, x, w, b, y, out_dtype: int, stream=None) -> None:
    _check(lib().dit_linear(M, N, K, dtype, _ptr(x), _ptr(w), _ptr(b), _ptr(y), out_dtype, _stream(stream)))


def profile_start() -> None:
    _check(lib().dit_profile_start())


def profile_stop() -> dict:
    """Stops kernel timing; returns {family: {launches, ms, flops, bytes}}."""
    n = ctypes.c_int()
    _check(lib().dit_profile_stop(ctypes.byref(n)))
    out = {}
    for i in range(n.value):
        name = ctypes.c_char_p()
        cnt = ctypes.c_long()
        ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        _check(lib().dit_profile_entry(i, ctypes.byref(name), ctypes.byref(cnt), ctypes.byref(ms), ctypes.byref(fl),
                                       ctypes.byref(by)))
        out[name.value.decode()] = {"launches": cnt.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}
    return out
