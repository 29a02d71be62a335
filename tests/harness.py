"""Test harness: the GPU plumbing of ``gpu_inputs`` plus the fp64 oracle on the same seeded inputs.

The GPU side receives the generator's arrays converted to torch device tensors;
the oracle receives the same arrays upcast to float64.  Nothing flows from the
GPU result into the oracle.
"""

from __future__ import annotations

import numpy as np

import oracle
import synth
from gpu_inputs import Cache as _Cache
from gpu_inputs import Model as _Model
from gpu_inputs import head_major_rows, rel_err, run_forward, tokens_for  # noqa: F401


def shape_of(wl: synth.Workload) -> oracle.ExpertShape:
    return oracle.ExpertShape(n_layers=wl.n_layers, d_model=wl.d_model, n_heads=wl.n_heads, head_dim=wl.head_dim,
                              d_ffn=wl.d_ffn, n_expert_tokens=wl.n_expert_tokens, n_out=wl.n_out,
                              rope_base=wl.rope_base, rms_eps=wl.rms_eps)


class Model(_Model):
    def oracle_agent(self, tokens_b, cache_rows, pos):
        """fp64 oracle for one agent: cache_rows(l) -> (K, V) float arrays [L][H][Dh]."""
        return oracle.expert_forward(shape_of(self.wl), self.layers, self.final_norm, self.head_w, tokens_b,
                                     cache_rows, pos)


class Cache(_Cache):
    def oracle_rows(self, b, decoded=False):
        """cache_rows(l) for the oracle: the generator's source values (or the fp8 decode if decoded)."""
        wl = self.wl

        def rows(l):
            out = []
            for kind in ("k", "v"):
                src = synth.cache_slab(wl, b, l, kind, rows=self.lengths[b]).astype(np.float64)
                if decoded and wl.cache_dtype == "fp8":
                    codes, scale = synth.fp8_encode(src.astype(np.float32))
                    src = oracle.e4m3fn_decode(codes) * scale.astype(np.float64)[None, :, None]
                out.append(src)
            return out[0], out[1]

        return rows
