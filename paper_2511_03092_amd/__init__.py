"""SnapStream hot path on MI355X: Python binding of libsnapstream.so.

Argument marshalling only.  Every step of compression and decoding runs in the
HIP kernels of ``libsnapstream.so`` (built in-tree by ``build.py``); torch is
used for device memory and the current stream.  If the library is missing the
first call raises -- there is no other implementation behind these names.

Functions keep the C names (include/snapstream.h):
    snap_compress, snap_prefill, snap_prefill_attn, snap_cache_append, snap_decode_attn, snap_decode_step,
    snap_decode_step_noalloc, snap_advance, snap_debug_checks,
    snap_compress_workspace, snap_prefill_workspace, snap_decode_workspace, snap_status_str
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsnapstream.so")
# the same library built with the device-side invariant checks (build.py --debug)
DEBUG_LIB_PATH = os.path.join(_HERE, "libsnapstream_debug.so")

SNAP_OK, SNAP_ERR_INVALID_ARG, SNAP_ERR_UNSUPPORTED, SNAP_ERR_WORKSPACE, SNAP_ERR_HIP = range(5)
SNAP_F32, SNAP_BF16, SNAP_FP8_E4M3 = 0, 1, 2
SNAP_POOL_MAX, SNAP_POOL_AVG = 0, 1
SNAP_NORM_CAND, SNAP_NORM_ROW = 0, 1
SNAP_FP8_SCALES_GIVEN, SNAP_FP8_SCALES_AMAX = 0, 1
SNAP_KV_AUTO, SNAP_KV_STREAM, SNAP_KV_KEEP = 0, 1, 2

EXPORTED = ["snap_compress_workspace", "snap_decode_workspace", "snap_prefill_workspace", "snap_compress",
            "snap_prefill", "snap_prefill_attn", "snap_cache_append",
            "snap_decode_attn", "snap_decode_step", "snap_decode_step_noalloc", "snap_advance", "snap_debug_checks",
            "snap_status_str", "snap_last_error"]


class SnapParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_q_heads", "n_kv_heads", "d_qk", "d_v", "v_in_k", "sink", "recent", "topk",
        "obs_window", "pool_kernel", "pool", "norm", "in_dtype", "kv_dtype")] + [("sm_scale", ctypes.c_float),
                                                                                  ("fp8_scales", ctypes.c_int32),
                                                                                  ("fp8_qk", ctypes.c_int32),
                                                                                  ("kv_reuse", ctypes.c_int32)]


class SnapCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("k_scale", ctypes.c_void_p),
                ("v_scale", ctypes.c_void_p), ("n_slots", ctypes.c_int32)]


class SnapError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"snapstream: {msg} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


def use_library(path: str) -> ctypes.CDLL:
    """Route every call of this module to the library at `path` (the release
    or the debug build); returns the library that was in use."""
    global _lib
    prev = lib()
    _lib = load(path)
    return prev


def load(path: str) -> ctypes.CDLL:
    """Load one build of the library and declare its entry points."""
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2511_03092_amd.build` "
                          "(there is no fallback implementation)")
    # torch first: its HIP runtime is then the process's libamdhip64.so.7, and
    # the library binds to that same runtime (the one that owns the device
    # memory passed in).  Loaded before torch, the library would bring in the
    # system's runtime beside torch's, and its launches would not see torch's
    # device state.
    import torch  # noqa: F401
    L = ctypes.CDLL(path)
    P, vp, i32, sz = ctypes.POINTER(SnapParams), ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    C = ctypes.POINTER(SnapCache)
    L.snap_compress_workspace.argtypes = [P, i32, i32]
    L.snap_compress_workspace.restype = sz
    L.snap_decode_workspace.argtypes = [P, i32]
    L.snap_decode_workspace.restype = sz
    L.snap_compress.argtypes = [P, C, vp, vp, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
    L.snap_compress.restype = ctypes.c_int
    L.snap_prefill_workspace.argtypes = [P, i32, i32]
    L.snap_prefill_workspace.restype = sz
    L.snap_prefill.argtypes = [P, C, vp, vp, i32, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.snap_prefill.restype = ctypes.c_int
    L.snap_prefill_attn.argtypes = [P, i32, vp, i32, vp, vp, vp, vp, vp, sz, vp]
    L.snap_prefill_attn.restype = ctypes.c_int
    L.snap_cache_append.argtypes = [P, C, vp, i32, vp, vp, vp, vp]
    L.snap_cache_append.restype = ctypes.c_int
    L.snap_decode_attn.argtypes = [P, C, vp, vp, i32, vp, vp, vp, i32, vp, sz, vp]
    L.snap_decode_attn.restype = ctypes.c_int
    L.snap_decode_step.argtypes = [P, C, vp, vp, i32, vp, vp, vp, vp, vp, i32, vp, sz, vp]
    L.snap_decode_step.restype = ctypes.c_int
    L.snap_decode_step_noalloc.argtypes = [P, C, vp, vp, i32, vp, vp, vp, vp, vp, i32, vp]
    L.snap_decode_step_noalloc.restype = ctypes.c_int
    L.snap_advance.argtypes = [vp, i32, i32, vp, vp]
    L.snap_advance.restype = ctypes.c_int
    L.snap_status_str.argtypes = [ctypes.c_int]
    L.snap_status_str.restype = ctypes.c_char_p
    L.snap_last_error.argtypes = []
    L.snap_last_error.restype = ctypes.c_char_p
    L.snap_debug_checks.argtypes = [ctypes.POINTER(ctypes.c_uint32), i32]
    L.snap_debug_checks.restype = ctypes.c_int
    return L


@dataclass
class Params:
    """Hyper-parameters (snap_params); dtypes use the SNAP_* codes."""
    n_q_heads: int
    n_kv_heads: int
    d_qk: int
    d_v: int
    sink: int
    recent: int
    topk: int
    obs_window: int
    pool_kernel: int
    pool: int = SNAP_POOL_MAX
    norm: int = SNAP_NORM_CAND
    v_in_k: bool = False
    in_dtype: int = SNAP_BF16
    kv_dtype: int = SNAP_BF16
    sm_scale: float = 0.0
    fp8_scales: int = SNAP_FP8_SCALES_GIVEN
    fp8_qk: int = 0
    kv_reuse: int = SNAP_KV_AUTO

    @property
    def budget(self) -> int:
        return self.sink + self.recent + self.topk

    def c(self) -> SnapParams:
        return SnapParams(self.n_q_heads, self.n_kv_heads, self.d_qk, self.d_v, int(self.v_in_k), self.sink,
                          self.recent, self.topk, self.obs_window, self.pool_kernel, self.pool, self.norm,
                          self.in_dtype, self.kv_dtype, float(self.sm_scale), int(self.fp8_scales),
                          int(self.fp8_qk), int(self.kv_reuse))


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(status: int):
    if status != SNAP_OK:
        L = lib()
        raise SnapError(status, (L.snap_last_error() or b"").decode() or L.snap_status_str(status).decode())


def cache_struct(k, v=None, k_scale=None, v_scale=None) -> SnapCache:
    return SnapCache(_ptr(k), _ptr(v), _ptr(k_scale), _ptr(v_scale), int(k.shape[0]))


def snap_status_str(status: int) -> str:
    return lib().snap_status_str(status).decode()


def snap_compress_workspace(p: Params, n_seq: int, max_len: int) -> int:
    return int(lib().snap_compress_workspace(ctypes.byref(p.c()), n_seq, max_len))


def snap_decode_workspace(p: Params, n: int) -> int:
    return int(lib().snap_decode_workspace(ctypes.byref(p.c()), n))


def snap_compress(p: Params, cache: SnapCache, pos, n_topk, slot_ids, lengths, q_obs, k, v, workspace,
                  sel_out=None, pooled_out=None, stream=None):
    n_seq, max_len = int(k.shape[0]), int(k.shape[2])
    _check(lib().snap_compress(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), _ptr(n_topk), n_seq,
                               _ptr(slot_ids), _ptr(lengths), max_len, _ptr(q_obs), _ptr(k), _ptr(v),
                               _ptr(sel_out), _ptr(pooled_out), _ptr(workspace),
                               workspace.numel() * workspace.element_size(), _stream(stream)))


def snap_prefill_workspace(p: Params, n_seq: int, max_len: int) -> int:
    return int(lib().snap_prefill_workspace(ctypes.byref(p.c()), n_seq, max_len))


def snap_prefill(p: Params, cache: SnapCache, pos, n_topk, slot_ids, lengths, q, k, v, out, workspace,
                 sel_out=None, pooled_out=None, stream=None):
    n_seq, max_len = int(k.shape[0]), int(k.shape[2])
    _check(lib().snap_prefill(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), _ptr(n_topk), n_seq,
                              _ptr(slot_ids), _ptr(lengths), max_len, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                              _ptr(sel_out), _ptr(pooled_out), _ptr(workspace),
                              workspace.numel() * workspace.element_size(), _stream(stream)))


def snap_prefill_attn(p: Params, lengths, q, k, v, out, workspace, stream=None):
    n_seq, max_len = int(k.shape[0]), int(k.shape[2])
    _check(lib().snap_prefill_attn(ctypes.byref(p.c()), n_seq, _ptr(lengths), max_len, _ptr(q), _ptr(k), _ptr(v),
                                   _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _stream(stream)))


def snap_cache_append(p: Params, cache: SnapCache, pos, slot_ids, k_new, v_new=None, stream=None):
    _check(lib().snap_cache_append(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), int(k_new.shape[0]),
                                   _ptr(slot_ids), _ptr(k_new), _ptr(v_new), _stream(stream)))


def snap_decode_attn(p: Params, cache: SnapCache, pos, n_topk, slot_ids, q, out, workspace, stream=None):
    import torch
    out_dtype = SNAP_BF16 if out.dtype == torch.bfloat16 else SNAP_F32
    _check(lib().snap_decode_attn(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), _ptr(n_topk),
                                  int(q.shape[0]), _ptr(slot_ids), _ptr(q), _ptr(out), out_dtype,
                                  _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def snap_decode_step(p: Params, cache: SnapCache, pos, n_topk, slot_ids, q, k_new, v_new, out, workspace,
                     stream=None):
    import torch
    out_dtype = SNAP_BF16 if out.dtype == torch.bfloat16 else SNAP_F32
    _check(lib().snap_decode_step(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), _ptr(n_topk),
                                  int(q.shape[0]), _ptr(slot_ids), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(out),
                                  out_dtype, _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def snap_decode_step_noalloc(p: Params, cache: SnapCache, pos, n_topk, slot_ids, q, k_new, v_new, out, stream=None):
    import torch
    out_dtype = SNAP_BF16 if out.dtype == torch.bfloat16 else SNAP_F32
    _check(lib().snap_decode_step_noalloc(ctypes.byref(p.c()), ctypes.byref(cache), _ptr(pos), _ptr(n_topk),
                                          int(q.shape[0]), _ptr(slot_ids), _ptr(q), _ptr(k_new), _ptr(v_new),
                                          _ptr(out), out_dtype, _stream(stream)))


def snap_advance(pos, slot_ids, stream=None):
    _check(lib().snap_advance(_ptr(pos), int(pos.shape[0]), int(slot_ids.shape[0]), _ptr(slot_ids),
                              _stream(stream)))


def snap_debug_checks(reset: bool = True) -> int:
    """The invariant bits the debug build's kernels recorded (waits for the
    device); raises SnapError on a release build."""
    flags = ctypes.c_uint32(0)
    _check(lib().snap_debug_checks(ctypes.byref(flags), int(reset)))
    return int(flags.value)


def workspace(nbytes: int, device="cuda"):
    """A 256-byte aligned device buffer (torch's allocator aligns to 512)."""
    import torch
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
