"""Seeded synthetic inputs for the action-expert tick, shared by the oracle side and the GPU side.

This module holds NO arithmetic of the method: it only draws random numbers,
rounds them to the stored dtype, and encodes the fp8 form of the stored cache
(the cache is produced by the backbone, upstream of the expert; its fp8
encoding is part of how the input is stored, not of what the expert computes).
Both the oracle harness and the GPU harness call it; neither the oracle nor the
HIP library imports it.

Every array is drawn from its own keyed stream
``numpy.random.default_rng([workload_id, tag, *index])`` so any slab (one
agent, one layer, K or V) can be regenerated independently and in parallel.

Distributions (the paper trains on driving logs and ships no weights; these
synthetic stand-ins have the shapes of its model, Sec. 3.1, and of its
deployment cache, Sec. 3.3):

* weights ~ N(0, 0.02^2), norm gains = 1;
* expert tokens and current-frame tokens ~ N(0, 1);
* cached backbone K/V rows ~ N(0, 1), taken as already rotated;
* appended K/V rows ~ N(0, 1).

Values are returned as float32 arrays whose values are exactly representable
in the workload's dtype (bf16 values are rounded to nearest-even here), so the
fp64 oracle and the GPU see bit-identical inputs.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

# stream tags
TAG_WEIGHT, TAG_TOKEN, TAG_CACHE_K, TAG_CACHE_V, TAG_APPEND_K, TAG_APPEND_V = 1, 2, 3, 4, 5, 6
WEIGHT_NAMES = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")
E4M3_MAX = 448.0


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: model sizes, batch, cache lengths and dtypes."""

    name: str
    wid: int  # seed key
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    n_expert_tokens: int
    n_frame_tokens: int
    batch: int
    lengths: tuple  # valid cache rows per agent
    dtype: str  # "f32" | "bf16": weights, tokens, expert activations
    cache_dtype: str  # "f32" | "bf16" | "fp8"
    capacity: int  # rows per (agent, layer) allocated in the ring
    n_out: int = 10
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    append_rows: int = 0  # rows appended per (agent, layer) by the append step
    head_kind: int = 0  # 0: mean-pool + linear head; 1: two-layer head over the waypoint queries
    head_hidden: int = 0  # hidden width of the two-layer head
    stress_keys: bool = False  # cached keys with outlier channels, a growing scale and a sink row (stress_keys())

    @property
    def seq(self) -> int:
        return self.n_expert_tokens + self.n_frame_tokens

    @property
    def attn_width(self) -> int:
        return self.n_heads * self.head_dim

    def positions(self) -> List[int]:
        """Position of expert token 0 for each agent: right after its cached rows."""
        return [int(x) for x in self.lengths]

    def replace(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


def _ragged_lengths(seed: int, n: int, lo: int, hi: int) -> tuple:
    return tuple(int(x) for x in np.random.default_rng(seed).integers(lo, hi + 1, n))


# The five workloads: a tiny fp32 expert; the full-size expert (32 layers, width 512, 32 heads x 128,
# SwiGLU 2048) on one agent at a 40-frame history (64 instruction rows + 4 rows x 40 frames = 224), on
# one agent with a long history plus 64 current-frame tokens, on 16 agents sharing the weights, and on
# 8 agents with ragged histories held as an fp8 cache.
FULL = dict(n_layers=32, d_model=512, n_heads=32, head_dim=128, d_ffn=2048, n_expert_tokens=10)
WORKLOADS = {
    "tiny_fp32_L40": Workload(
        name="tiny_fp32_L40", wid=0, n_layers=2, d_model=64, n_heads=4, head_dim=32, d_ffn=256,
        n_expert_tokens=10, n_frame_tokens=0, batch=1, lengths=(40,), dtype="f32", cache_dtype="f32",
        capacity=40),
    "single_bf16_L224": Workload(
        name="single_bf16_L224", wid=1, n_frame_tokens=0, batch=1, lengths=(224,), dtype="bf16",
        cache_dtype="bf16", capacity=224, **FULL),
    "long_bf16_L4096_F64": Workload(
        name="long_bf16_L4096_F64", wid=2, n_frame_tokens=64, batch=1, lengths=(4096,), dtype="bf16",
        cache_dtype="bf16", capacity=4096, **FULL),
    "batched_bf16_B16_L1024": Workload(
        name="batched_bf16_B16_L1024", wid=3, n_frame_tokens=0, batch=16, lengths=(1024,) * 16,
        dtype="bf16", cache_dtype="bf16", capacity=1040, append_rows=4, **FULL),
    "ragged_fp8_B8": Workload(
        name="ragged_fp8_B8", wid=4, n_frame_tokens=0, batch=8, lengths=_ragged_lengths(4, 8, 256, 16384),
        dtype="bf16", cache_dtype="fp8", capacity=16384, **FULL),
}


# ----------------------------------------------------------------------------- rounding helpers

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = ((u + r) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return out.view(np.float32)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype in ("bf16", "fp8"):  # the fp8 cache is encoded from a bf16 source
        return round_bf16(x)
    raise ValueError(dtype)


def _normal(key, shape, std=1.0) -> np.ndarray:
    g = np.random.default_rng(key)
    a = g.standard_normal(int(np.prod(shape)), dtype=np.float32).reshape(shape)
    if std != 1.0:
        a *= np.float32(std)
    return a


# ----------------------------------------------------------------------------- weights and tokens

def make_weights(wl: Workload):
    """Per-layer weight dicts (nn.Linear [out][in] layout) + final norm gain + the head: its weight [n_out][d], or
    for the two-layer head a dict w1 [hidden][d], b1 [hidden], w2 [2][hidden], b2 [2] (biases ~N(0, 0.02^2), fp32)."""
    d, A, F = wl.d_model, wl.attn_width, wl.d_ffn
    shapes = {"wq": (A, d), "wk": (A, d), "wv": (A, d), "wo": (d, A),
              "w_gate": (F, d), "w_up": (F, d), "w_down": (d, F)}
    layers = []
    for layer in range(wl.n_layers):
        lw = {}
        for i, name in enumerate(WEIGHT_NAMES):
            lw[name] = round_to(_normal([wl.wid, TAG_WEIGHT, layer, i], shapes[name], 0.02), wl.dtype)
        lw["attn_norm"] = np.ones(d, np.float32)
        lw["ffn_norm"] = np.ones(d, np.float32)
        layers.append(lw)
    final_norm = np.ones(d, np.float32)
    if wl.head_kind == 1:
        hid = wl.head_hidden
        head = {"w1": round_to(_normal([wl.wid, TAG_WEIGHT, wl.n_layers, 0], (hid, d), 0.02), wl.dtype),
                "b1": _normal([wl.wid, TAG_WEIGHT, wl.n_layers, 1], (hid,), 0.02),
                "w2": round_to(_normal([wl.wid, TAG_WEIGHT, wl.n_layers, 2], (2, hid), 0.02), wl.dtype),
                "b2": _normal([wl.wid, TAG_WEIGHT, wl.n_layers, 3], (2,), 0.02)}
        return layers, final_norm, head
    head_w = round_to(_normal([wl.wid, TAG_WEIGHT, wl.n_layers, 0], (wl.n_out, d), 0.02), wl.dtype)
    return layers, final_norm, head_w


def make_tokens(wl: Workload) -> np.ndarray:
    """[B][S][d]: rows < T are expert tokens, the rest current-frame tokens; ~N(0,1)."""
    out = np.empty((wl.batch, wl.seq, wl.d_model), np.float32)
    for b in range(wl.batch):
        out[b] = round_to(_normal([wl.wid, TAG_TOKEN, b], (wl.seq, wl.d_model)), wl.dtype)
    return out


# ----------------------------------------------------------------------------- cache slabs

def cache_slab(wl: Workload, b: int, layer: int, kind: str, rows: Optional[int] = None) -> np.ndarray:
    """Source values of the cached rows of (agent b, layer, 'k'|'v'): [L_b][H][Dh] float32.

    For bf16 and fp8 caches these are bf16-rounded; for an fp8 cache they are the
    values the fp8 codes encode (see ``fp8_encode``).
    """
    L = wl.lengths[b] if rows is None else rows
    tag = TAG_CACHE_K if kind == "k" else TAG_CACHE_V
    a = _normal([wl.wid, tag, b, layer], (L, wl.n_heads, wl.head_dim))
    if kind == "k" and wl.stress_keys:
        a = stress_keys(a)
    return round_to(a, wl.cache_dtype)


def stress_keys(a: np.ndarray) -> np.ndarray:
    """Keys [L][H][Dh] made hard for an online softmax: channels 0-3 of every head 8x (outlier channels, as in
    the caches of large language models), row i scaled by 1 + 3 i / L (scores grow along the sequence, so a query's
    running maximum keeps moving), and row floor(2L/3) a further 8x (a sink row far past the first tiles)."""
    L = a.shape[0]
    a = a.astype(np.float32).copy()
    a[:, :, :4] *= 8.0
    a *= (1.0 + 3.0 * np.arange(L, dtype=np.float32) / max(L, 1))[:, None, None]
    if L > 0:
        a[(2 * L) // 3] *= 8.0
    return a


def append_rows(wl: Workload, step: int, kind: str, n_rows: int) -> np.ndarray:
    """New rows appended at append step `step`: [B][n_layers][n][H][Dh] float32 (bf16-rounded)."""
    tag = TAG_APPEND_K if kind == "k" else TAG_APPEND_V
    a = _normal([wl.wid, tag, step], (wl.batch, wl.n_layers, n_rows, wl.n_heads, wl.head_dim))
    return round_to(a, wl.cache_dtype if wl.cache_dtype != "fp8" else "bf16")


def fp8_encode(src: np.ndarray):
    """Encode a [L][H][Dh] slab as OCP E4M3 codes with one fp32 scale per head.

    scale_h = amax over the slab's rows of head h / 448; code = RNE(clamp(x / scale_h, +-448)).
    Returns (codes uint8 [L][H][Dh], scales float32 [H]).
    """
    import torch

    src = np.ascontiguousarray(src, np.float32)
    amax = np.abs(src).max(axis=(0, 2)) if src.shape[0] else np.zeros(src.shape[1], np.float32)
    scale = (amax.astype(np.float32) / np.float32(E4M3_MAX)).astype(np.float32)
    scale = np.where(scale > 0, scale, np.float32(1.0)).astype(np.float32)
    y = np.clip(src / scale[None, :, None], -E4M3_MAX, E4M3_MAX).astype(np.float32)
    codes = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes, scale


def parallel_map(fn, items, workers: Optional[int] = None):
    """Run fn over items on a thread pool (NumPy's generators release the GIL)."""
    if workers is None:
        workers = min(16, len(os.sched_getaffinity(0)))
    with ThreadPoolExecutor(max(1, workers)) as ex:
        return list(ex.map(fn, items))
