"""GPU-side plumbing: seeded synthetic inputs -> device tensors and libfsx handles.

Imports nothing from the oracle; ``harness.py`` adds the oracle side.
"""

from __future__ import annotations

import numpy as np
import torch

import synth
from paper_2607_15621_amd import fsx

NORMS = ("attn_norm", "ffn_norm")


def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def fsx_dtype(name: str) -> int:
    return {"f32": fsx.F32, "bf16": fsx.BF16, "fp8": fsx.FP8_E4M3}[name]


class Model:
    """Weights of a workload on the host (float32 arrays holding dtype-exact values)."""

    def __init__(self, wl: synth.Workload):
        self.wl = wl
        self.layers, self.final_norm, self.head_w = synth.make_weights(wl)

    def create(self, max_batch=None, max_frame_tokens=None, flags=0, device="cuda", tick_timeout_us=0) -> fsx.Expert:
        wl = self.wl
        td = torch_dtype(wl.dtype)
        self.dev_layers = []
        for lw in self.layers:
            self.dev_layers.append({k: torch.from_numpy(v).to(device=device, dtype=torch.float32 if k in NORMS else td)
                                    for k, v in lw.items()})
        self.dev_final = torch.from_numpy(self.final_norm).to(device)
        if isinstance(self.head_w, dict):
            self.dev_head = {k: torch.from_numpy(v).to(device=device, dtype=td if k in ("w1", "w2") else torch.float32)
                             for k, v in self.head_w.items()}
        else:
            self.dev_head = torch.from_numpy(self.head_w).to(device=device, dtype=td)
        cfg = fsx.make_cfg(wl.n_layers, wl.d_model, wl.n_heads, wl.head_dim, wl.d_ffn, wl.n_expert_tokens, wl.n_out,
                           max_batch or wl.batch, wl.n_frame_tokens if max_frame_tokens is None else max_frame_tokens,
                           fsx_dtype(wl.dtype), wl.rope_base, wl.rms_eps, flags, tick_timeout_us, wl.head_kind,
                           wl.head_hidden)
        ex = fsx.expert_create(cfg, self.dev_layers, self.dev_final, self.dev_head)
        torch.cuda.synchronize()
        # the library packed its own copy; the caller's tensors may go
        del self.dev_layers, self.dev_final, self.dev_head
        return ex


class Cache:
    """A device cache filled from the generator, plus the fsx descriptor over it.

    starts: optional ring start slot per agent (rows i sit at (start + i) mod capacity).
    """

    def __init__(self, wl: synth.Workload, lengths=None, starts=None, capacity=None, device="cuda",
                 fill_workers=None, layout=fsx.CACHE_HEAD_MAJOR):
        self.wl = wl
        self.layout = layout
        self.lengths = list(wl.lengths if lengths is None else lengths)
        B = len(self.lengths)
        cap = wl.capacity if capacity is None else capacity
        self.capacity = cap
        self.starts = [0] * B if starts is None else list(starts)
        if layout == fsx.CACHE_TOKEN_MAJOR:
            shape = (B, wl.n_layers, cap, wl.n_heads, wl.head_dim)  # a slot holds every head of one token
        else:
            shape = (B, wl.n_layers, wl.n_heads, cap, wl.head_dim)  # head-major rings
        if wl.cache_dtype == "fp8":
            self.k = torch.zeros(shape, dtype=torch.uint8, device=device)
            self.v = torch.zeros(shape, dtype=torch.uint8, device=device)
            self.k_scale = torch.ones((B, wl.n_layers, wl.n_heads), dtype=torch.float32, device=device)
            self.v_scale = torch.ones((B, wl.n_layers, wl.n_heads), dtype=torch.float32, device=device)
            self.scales = {}
        else:
            td = torch_dtype(wl.cache_dtype)
            self.k = torch.zeros(shape, dtype=td, device=device)
            self.v = torch.zeros(shape, dtype=td, device=device)
            self.k_scale = self.v_scale = None
        jobs = [(b, l) for b in range(B) for l in range(wl.n_layers) if self.lengths[b] > 0]
        synth.parallel_map(self._fill, jobs, fill_workers)
        torch.cuda.synchronize()
        self.desc = fsx.CacheDesc(self.k, self.v, fsx_dtype(wl.cache_dtype), wl.n_layers, wl.n_heads, wl.head_dim,
                                  cap, self.lengths, positions=self.lengths, starts=self.starts,
                                  k_scale=self.k_scale, v_scale=self.v_scale, layout=layout)

    def _slots(self, b, n):
        return (self.starts[b] + np.arange(n)) % self.capacity

    def _fill(self, job):
        b, l = job
        L = self.lengths[b]
        idx = torch.from_numpy(self._slots(b, L))
        for kind, dst in (("k", self.k), ("v", self.v)):
            src = synth.cache_slab(self.wl, b, l, kind, rows=L)
            if self.wl.cache_dtype == "fp8":
                codes, scale = synth.fp8_encode(src)
                self.scales[(b, l, kind)] = scale
                (self.k_scale if kind == "k" else self.v_scale)[b, l] = torch.from_numpy(scale).to(dst.device)
                t = torch.from_numpy(codes)
            else:
                t = torch.from_numpy(src).to(dst.dtype)
            if self.layout == fsx.CACHE_TOKEN_MAJOR:  # generator slab [L][H][Dh] = slots of the ring
                dst[b, l].index_copy_(0, idx.to(dst.device), t.to(dst.device, non_blocking=False))
            else:  # generator slab [L][H][Dh] -> head-major [H][L][Dh] rows of the ring
                t = t.permute(1, 0, 2).contiguous()
                dst[b, l].index_copy_(1, idx.to(dst.device), t.to(dst.device, non_blocking=False))

    def slot_rows(self, b, l, kind, slots):
        """Device rows [len(slots)][H][Dh] of (agent b, layer l) at the given ring slots, whatever the layout."""
        t = self.k if kind == "k" else self.v
        idx = torch.as_tensor(np.asarray(slots), device=t.device)
        if self.layout == fsx.CACHE_TOKEN_MAJOR:
            return t[b, l].index_select(0, idx)
        return t[b, l].index_select(1, idx).permute(1, 0, 2)

    def rows_for_append(self, rows: np.ndarray, dtype):
        """Generator rows [B][n_layers][n][H][Dh] -> the device layout fsx_cache_append_rows takes for this cache."""
        if self.layout == fsx.CACHE_TOKEN_MAJOR:
            return torch.from_numpy(np.ascontiguousarray(rows)).to("cuda", dtype)
        return head_major_rows(rows, dtype)


def head_major_rows(rows: np.ndarray, dtype, device="cuda"):
    """Appended rows [B][n_layers][n][H][Dh] (generator order) -> device [B][n_layers][H][n][Dh]."""
    return torch.from_numpy(np.ascontiguousarray(rows.transpose(0, 1, 3, 2, 4))).to(device, dtype)


def tokens_for(wl: synth.Workload, device="cuda"):
    host = synth.make_tokens(wl)
    return host, torch.from_numpy(host).to(device=device, dtype=torch_dtype(wl.dtype))


def rel_err(got, want) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    return float(np.abs(got - want).max() / max(np.abs(want).max(), 1e-30))


def run_forward(ex, cache: Cache, tok_dev, batch, n_frame, with_hidden=False):
    wl = cache.wl
    S = wl.n_expert_tokens + n_frame
    wp = torch.full((batch, wl.n_out), float("nan"), device=tok_dev.device)
    hid = None
    if with_hidden:
        hid = torch.full((wl.n_layers, batch, S, wl.d_model), float("nan"), device=tok_dev.device)
    fsx.expert_forward(ex, cache.desc, tok_dev, batch, n_frame, wp, hid)
    torch.cuda.synchronize()
    return wp.cpu().numpy(), (hid.cpu().numpy() if with_hidden else None)
