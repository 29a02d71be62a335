"""Thin Python binding of libfsx (include/fsx.h): argument marshalling only.

Every step of the expert tick runs in the HIP library; this module only turns
torch tensors / numpy arrays into the raw pointers and sizes the C ABI takes,
and turns non-zero status codes into exceptions.  If the library has not been
built, loading it raises -- there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfsx.so")

F32, BF16, FP8_E4M3 = 0, 1, 2
APPEND_RING, APPEND_ERROR = 0, 1
CACHE_HEAD_MAJOR, CACHE_TOKEN_MAJOR, CACHE_SHARED = 0, 1, 2
FLAG_GENERIC, FLAG_MULTI_LAUNCH, FLAG_TRACE = 1, 2, 4
HEAD_MEAN_LINEAR, HEAD_QUERY_MLP = 0, 1
MAX_BATCH = 64
STATUS = {0: "FSX_OK", 1: "FSX_E_INVALID", 2: "FSX_E_UNSUPPORTED", 3: "FSX_E_CAPACITY", 4: "FSX_E_OOM",
          5: "FSX_E_HIP"}
SYMBOLS = ("fsx_expert_create", "fsx_expert_forward", "fsx_cache_append_rows", "fsx_expert_status",
           "fsx_expert_trace", "fsx_expert_destroy", "fsx_last_error", "fsx_expert_info", "fsx_version",
           "fsx_probe_hbm_read", "fsx_expert_forward_noalloc", "fsx_cache_append_rows_quantize",
           "fsx_loop_create", "fsx_loop_tick", "fsx_loop_append", "fsx_loop_sync", "fsx_loop_destroy",
           "fsx_loop_last_error", "fsx_backbone_create", "fsx_backbone_append", "fsx_backbone_info",
           "fsx_backbone_destroy")


class FsxError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class ExpertCfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("n_expert_tokens", ctypes.c_int32),
                ("n_out", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_frame_tokens", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("flags", ctypes.c_int32), ("tick_timeout_us", ctypes.c_int32), ("head_kind", ctypes.c_int32),
                ("head_hidden", ctypes.c_int32)]


class HeadWeights(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("b", ctypes.c_void_p), ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "attn_norm", "ffn_norm")]


class BackboneCfg(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("max_new_rows", ctypes.c_int32),
                ("max_batch", ctypes.c_int32), ("dtype", ctypes.c_int32), ("rope_base", ctypes.c_float),
                ("rms_eps", ctypes.c_float)]


class LoopTickInfo(ctypes.Structure):
    _fields_ = [("tick", ctypes.c_int64), ("published", ctypes.c_int32), ("staleness", ctypes.c_int32),
                ("start", ctypes.c_int64 * MAX_BATCH), ("len", ctypes.c_int64 * MAX_BATCH),
                ("pos", ctypes.c_int64 * MAX_BATCH)]


class CacheDescC(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("batch", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("capacity", ctypes.c_int64), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("k_scale", ctypes.c_void_p), ("v_scale", ctypes.c_void_p),
                ("start", ctypes.POINTER(ctypes.c_int64)), ("len", ctypes.POINTER(ctypes.c_int64)),
                ("pos", ctypes.POINTER(ctypes.c_int64))]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libfsx.so (built by ``paper_2607_15621_amd.build``); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_15621_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.fsx_expert_create.argtypes = [ctypes.POINTER(ExpertCfg), ctypes.POINTER(LayerWeights), vp,
                                        ctypes.POINTER(HeadWeights), vp, ctypes.POINTER(vp)]
        L.fsx_expert_forward.argtypes = [vp, ctypes.POINTER(CacheDescC), vp, i32, i32, vp, vp, vp]
        L.fsx_cache_append_rows.argtypes = [ctypes.POINTER(CacheDescC), vp, vp, i32, i32, vp]
        L.fsx_expert_status.argtypes = [vp, vp]
        L.fsx_expert_trace.argtypes = [vp, ctypes.POINTER(ctypes.c_uint64), i64, ctypes.POINTER(i32),
                                       ctypes.POINTER(i32), vp]
        L.fsx_expert_destroy.argtypes = [vp]
        L.fsx_expert_destroy.restype = None
        L.fsx_last_error.restype = ctypes.c_char_p
        L.fsx_expert_info.argtypes = [vp, ctypes.POINTER(i32), ctypes.POINTER(i64), ctypes.POINTER(i64)]
        L.fsx_version.restype = ctypes.c_char_p
        L.fsx_probe_hbm_read.argtypes = [vp, i64, i32, vp, vp]
        L.fsx_expert_forward_noalloc.argtypes = [vp, ctypes.POINTER(CacheDescC), vp, i32, i32, vp, vp, vp]
        L.fsx_expert_forward_noalloc.restype = ctypes.c_int
        L.fsx_cache_append_rows_quantize.argtypes = [ctypes.POINTER(CacheDescC), vp, vp, i32, i32, i32, vp]
        L.fsx_loop_create.argtypes = [vp, ctypes.POINTER(CacheDescC), i32, i32, vp, vp, ctypes.POINTER(vp)]
        L.fsx_loop_tick.argtypes = [vp, vp, i32, i32, vp, vp, ctypes.POINTER(LoopTickInfo)]
        L.fsx_loop_append.argtypes = [vp, vp, vp, i32, i32]
        L.fsx_loop_sync.argtypes = [vp, ctypes.POINTER(CacheDescC)]
        L.fsx_loop_destroy.argtypes = [vp]
        L.fsx_loop_destroy.restype = None
        L.fsx_loop_last_error.restype = ctypes.c_char_p
        for n in ("fsx_cache_append_rows_quantize", "fsx_loop_create", "fsx_loop_tick", "fsx_loop_append",
                  "fsx_loop_sync"):
            getattr(L, n).restype = ctypes.c_int
        L.fsx_backbone_create.argtypes = [ctypes.POINTER(BackboneCfg), ctypes.POINTER(LayerWeights), vp,
                                          ctypes.POINTER(vp)]
        L.fsx_backbone_append.argtypes = [vp, ctypes.POINTER(CacheDescC), vp, i32, i32, vp, i32, vp]
        L.fsx_backbone_info.argtypes = [vp, ctypes.POINTER(i64), ctypes.POINTER(i64)]
        L.fsx_backbone_destroy.argtypes = [vp]
        L.fsx_backbone_destroy.restype = None
        for n in ("fsx_backbone_create", "fsx_backbone_append", "fsx_backbone_info"):
            getattr(L, n).restype = ctypes.c_int
        for n in ("fsx_expert_create", "fsx_expert_forward", "fsx_cache_append_rows", "fsx_expert_info",
                  "fsx_expert_status", "fsx_expert_trace", "fsx_probe_hbm_read"):
            getattr(L, n).restype = ctypes.c_int
        _lib = L
    return _lib


def last_error() -> str:
    return lib().fsx_last_error().decode()


def version() -> str:
    return lib().fsx_version().decode()


def _check(code: int):
    if code != 0:
        raise FsxError(code, last_error())


def _ptr(t) -> int:
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def _stream(stream) -> int:
    if stream is None:
        import torch

        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def make_cfg(n_layers, d_model, n_heads, head_dim, d_ffn, n_expert_tokens=10, n_out=10, max_batch=1,
             max_frame_tokens=0, dtype=BF16, rope_base=10000.0, rms_eps=1e-6, flags=0,
             tick_timeout_us=0, head_kind=HEAD_MEAN_LINEAR, head_hidden=0) -> ExpertCfg:
    return ExpertCfg(n_layers, d_model, n_heads, head_dim, d_ffn, n_expert_tokens, n_out, max_batch,
                     max_frame_tokens, dtype, rope_base, rms_eps, flags, tick_timeout_us, head_kind, head_hidden)


class Expert:
    """Handle returned by fsx_expert_create; fsx_expert_destroy runs on close()."""

    def __init__(self, handle: int, cfg: ExpertCfg):
        self.handle = handle
        self.cfg = cfg

    def close(self):
        if self.handle:
            lib().fsx_expert_destroy(ctypes.c_void_p(self.handle))
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def expert_create(cfg: ExpertCfg, layers: Sequence[dict], final_norm, head, stream=None) -> Expert:
    """fsx_expert_create.  layers: per layer a dict of device tensors (wq, wk, wv, wo, w_gate, w_up,
    w_down, attn_norm, ffn_norm) in nn.Linear layout.  head: the mean-pool head's weight [n_out][d], or a dict
    w1, b1, w2, b2 of device tensors for the query head."""
    arr = (LayerWeights * len(layers))()
    for i, lw in enumerate(layers):
        arr[i] = LayerWeights(*[_ptr(lw[n]) for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
                                                        "attn_norm", "ffn_norm")])
    if isinstance(head, dict):
        hw = HeadWeights(_ptr(head["w1"]), _ptr(head["b1"]), _ptr(head["w2"]), _ptr(head["b2"]))
    else:
        hw = HeadWeights(_ptr(head), None, None, None)
    out = ctypes.c_void_p(0)
    _check(lib().fsx_expert_create(ctypes.byref(cfg), arr if len(layers) else None, _ptr(final_norm),
                                   ctypes.byref(hw), _stream(stream), ctypes.byref(out)))
    return Expert(out.value, cfg)


def expert_info(ex: Expert):
    path, wb, wsb = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().fsx_expert_info(ctypes.c_void_p(ex.handle), ctypes.byref(path), ctypes.byref(wb),
                                 ctypes.byref(wsb)))
    return {"path": path.value, "weight_bytes": wb.value, "workspace_bytes": wsb.value}


class CacheDesc:
    """fsx_cache_desc: device K/V tensors, [batch][n_layers][H][capacity][Dh] (layout CACHE_HEAD_MAJOR) or
    [batch][n_layers][capacity][H][Dh] (CACHE_TOKEN_MAJOR), plus host ring state.

    start / len / pos are numpy int64 arrays that the C side reads, and updates in place on append.
    """

    def __init__(self, k, v, dtype: int, n_layers: int, n_heads: int, head_dim: int, capacity: int,
                 lengths, positions=None, starts=None, k_scale=None, v_scale=None, layout: int = CACHE_HEAD_MAJOR):
        self.k, self.v, self.k_scale, self.v_scale = k, v, k_scale, v_scale
        batch = len(lengths)
        self.len = np.ascontiguousarray(np.asarray(lengths, dtype=np.int64))
        self.pos = np.ascontiguousarray(np.asarray(lengths if positions is None else positions, dtype=np.int64))
        self.start = np.ascontiguousarray(np.zeros(batch, np.int64) if starts is None else
                                          np.asarray(starts, dtype=np.int64))
        P = ctypes.POINTER(ctypes.c_int64)
        self.layout = layout
        self.c = CacheDescC(dtype, batch, n_layers, n_heads, head_dim, layout, capacity, _ptr(k), _ptr(v),
                            _ptr(k_scale), _ptr(v_scale), self.start.ctypes.data_as(P),
                            self.len.ctypes.data_as(P), self.pos.ctypes.data_as(P))


def expert_forward(ex: Expert, cache: CacheDesc, tokens, batch: int, n_frame_tokens: int, waypoints,
                   hidden=None, stream=None):
    """fsx_expert_forward: one tick for `batch` agents (enqueued on `stream`)."""
    _check(lib().fsx_expert_forward(ctypes.c_void_p(ex.handle), ctypes.byref(cache.c), _ptr(tokens), batch,
                                    n_frame_tokens, _ptr(waypoints), _ptr(hidden), _stream(stream)))


def expert_forward_noalloc(ex: Expert, cache: CacheDesc, tokens, batch: int, n_frame_tokens: int, waypoints,
                           hidden=None, stream=None):
    """fsx_expert_forward_noalloc: the same tick, its workspace in the library's static device array."""
    _check(lib().fsx_expert_forward_noalloc(ctypes.c_void_p(ex.handle), ctypes.byref(cache.c), _ptr(tokens), batch,
                                            n_frame_tokens, _ptr(waypoints), _ptr(hidden), _stream(stream)))


def expert_status(ex: Expert, stream=None):
    """fsx_expert_status: synchronise the stream; raise if a tick of this handle timed out."""
    _check(lib().fsx_expert_status(ctypes.c_void_p(ex.handle), _stream(stream)))


def expert_trace(ex: Expert, n_wg_max: int = 1024, stream=None) -> np.ndarray:
    """fsx_expert_trace: [n_wg][n_events] real-time stamps (100 MHz) of the last tick."""
    n_layers = ex.cfg.n_layers
    cap = n_wg_max * (2 + 16 * n_layers + 1)
    buf = np.zeros(cap, np.uint64)
    nw, ne = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().fsx_expert_trace(ctypes.c_void_p(ex.handle), buf.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)),
                                  cap, ctypes.byref(nw), ctypes.byref(ne), _stream(stream)))
    return buf[: nw.value * ne.value].reshape(nw.value, ne.value)


def cache_append_rows(cache: CacheDesc, k_rows, v_rows, n_rows: int, policy: int = APPEND_RING, stream=None):
    """fsx_cache_append_rows: enqueue the row copy; host ring state is updated on return."""
    _check(lib().fsx_cache_append_rows(ctypes.byref(cache.c), _ptr(k_rows), _ptr(v_rows), n_rows, policy,
                                       _stream(stream)))


def probe_hbm_read(buf, nbytes: int, mode: int, sink, stream=None):
    """fsx_probe_hbm_read: enqueue one read-only pass over nbytes of buf (measurement helper)."""
    _check(lib().fsx_probe_hbm_read(_ptr(buf), nbytes, mode, _ptr(sink), _stream(stream)))


def cache_append_rows_quantize(cache: CacheDesc, k_rows, v_rows, rows_dtype: int, n_rows: int,
                               policy: int = APPEND_RING, stream=None):
    """fsx_cache_append_rows_quantize: bf16 / fp32 rows encoded into an fp8 cache with its scales."""
    _check(lib().fsx_cache_append_rows_quantize(ctypes.byref(cache.c), _ptr(k_rows), _ptr(v_rows), rows_dtype,
                                                n_rows, policy, _stream(stream)))


class Loop:
    """fsx_loop: the asynchronous deployment loop (expert every tick, appends on a second stream)."""

    def __init__(self, ex: Expert, cache: CacheDesc, append_every: int, expert_stream, append_stream,
                 policy: int = APPEND_RING):
        self.ex, self.cache = ex, cache  # the loop reads their device buffers
        out = ctypes.c_void_p(0)
        self._check(lib().fsx_loop_create(ctypes.c_void_p(ex.handle), ctypes.byref(cache.c), append_every, policy,
                                          _stream(expert_stream), _stream(append_stream), ctypes.byref(out)))
        self.handle = out.value

    @staticmethod
    def _check(code):
        if code != 0:
            raise FsxError(code, lib().fsx_loop_last_error().decode())

    def tick(self, tokens, batch: int, n_frame_tokens: int, waypoints, hidden=None) -> dict:
        info = LoopTickInfo()
        self._check(lib().fsx_loop_tick(ctypes.c_void_p(self.handle), _ptr(tokens), batch, n_frame_tokens,
                                        _ptr(waypoints), _ptr(hidden), ctypes.byref(info)))
        return {"tick": info.tick, "published": info.published, "staleness": info.staleness,
                "start": list(info.start[:batch]), "len": list(info.len[:batch]), "pos": list(info.pos[:batch])}

    def append(self, k_rows, v_rows, rows_dtype: int, n_rows: int):
        self._check(lib().fsx_loop_append(ctypes.c_void_p(self.handle), _ptr(k_rows), _ptr(v_rows), rows_dtype,
                                          n_rows))

    def sync(self, cache_out: Optional[CacheDesc] = None):
        self._check(lib().fsx_loop_sync(ctypes.c_void_p(self.handle),
                                        ctypes.byref(cache_out.c) if cache_out is not None else None))

    def close(self):
        if self.handle:
            lib().fsx_loop_destroy(ctypes.c_void_p(self.handle))
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Backbone:
    """fsx_backbone: the backbone's incremental forward that produces the appended cache rows."""

    def __init__(self, cfg: BackboneCfg, layers: Sequence[dict], stream=None):
        arr = (LayerWeights * len(layers))()
        for i, lw in enumerate(layers):
            arr[i] = LayerWeights(*[_ptr(lw[n]) for n in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
                                                            "attn_norm", "ffn_norm")])
        out = ctypes.c_void_p(0)
        _check(lib().fsx_backbone_create(ctypes.byref(cfg), arr, _stream(stream), ctypes.byref(out)))
        self.handle, self.cfg = out.value, cfg

    def append(self, cache: CacheDesc, tokens, batch: int, n_rows: int, hidden=None, policy: int = APPEND_RING,
               stream=None):
        _check(lib().fsx_backbone_append(ctypes.c_void_p(self.handle), ctypes.byref(cache.c), _ptr(tokens), batch,
                                         n_rows, _ptr(hidden), policy, _stream(stream)))

    def info(self):
        wb, wsb = ctypes.c_int64(), ctypes.c_int64()
        _check(lib().fsx_backbone_info(ctypes.c_void_p(self.handle), ctypes.byref(wb), ctypes.byref(wsb)))
        return {"weight_bytes": wb.value, "workspace_bytes": wsb.value}

    def close(self):
        if self.handle:
            lib().fsx_backbone_destroy(ctypes.c_void_p(self.handle))
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
