"""fp64 reference of the backbone's incremental forward (Sec. 3.3: every K ticks the current frame's tokens are
appended to the backbone's KV cache through an incremental forward pass whose cost does not depend on the history
length).

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Imports nothing but NumPy and the expert oracle's pinned
building blocks (RMSNorm, rotary encoding, SwiGLU).

The backbone is LLaMA-7B (Sec. 3: a frozen LLaMA-7B consumes [text | f1 | f2 | ...]): decoder layers of pre-norm
RMSNorm, q/k/v projections d -> H*Dh with rotary encoding, causal attention, output projection, pre-norm SwiGLU.
One incremental forward takes the n new tokens of a frame at positions pos .. pos+n-1 and, at every layer, attends
from each new token to every cached row of that layer and to the new rows up to itself; the new tokens' keys (rotated)
and values are the rows appended to the cache.

Readings (the paper gives the model only by name): LLaMA's layer as published -- RMSNorm eps 1e-6, rotate-half
rotary pairs (j, j + Dh/2) with base 10^4, scale 1/sqrt(Dh), full multi-head attention (no grouping), SwiGLU
FFN without biases.  Cached keys are stored rotated at their own positions, which is what makes the append exact.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Sequence

import numpy as np

from .expert import apply_rope, rmsnorm, swiglu_ffn


@dataclass(frozen=True)
class BackboneShape:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-6


def causal_cache_attention(q, k_new, v_new, k_cache, v_cache) -> np.ndarray:
    """Attention of n new tokens: query i over [cached rows ; new rows 0..i], one softmax per (query, head), scale
    1/sqrt(Dh).  q, k_new, v_new: [n][H][Dh]; k_cache, v_cache: [L][H][Dh].  Returns [n][H][Dh]."""
    q = np.asarray(q, np.float64)
    n, H, Dh = q.shape
    L = np.asarray(k_cache).shape[0]
    keys = np.concatenate([np.asarray(k_cache, np.float64), np.asarray(k_new, np.float64)], axis=0)
    vals = np.concatenate([np.asarray(v_cache, np.float64), np.asarray(v_new, np.float64)], axis=0)
    allow = np.arange(L + n)[None, :] < (L + np.arange(n) + 1)[:, None]  # [n][L + n]
    sc = np.einsum("ihc,rhc->hir", q, keys) / np.sqrt(np.float64(Dh))
    sc = np.where(allow[None], sc, -np.inf)
    sc = sc - sc.max(axis=-1, keepdims=True)
    p = np.exp(sc)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.einsum("hir,rhc->ihc", p, vals)


def backbone_layer(h, lw: dict, k_cache, v_cache, positions, shape: BackboneShape):
    """One decoder layer over the new tokens h [n][d].  lw: wq, wk, wv [H*Dh][d], wo [d][H*Dh], w_gate, w_up
    [d_ffn][d], w_down [d][d_ffn], attn_norm, ffn_norm [d].  Returns (h_out [n][d], k_new, v_new [n][H][Dh])."""
    h = np.asarray(h, np.float64)
    n = h.shape[0]
    H, Dh = shape.n_heads, shape.head_dim
    x = rmsnorm(h, lw["attn_norm"], shape.rms_eps)
    q = (x @ np.asarray(lw["wq"], np.float64).T).reshape(n, H, Dh)
    k = (x @ np.asarray(lw["wk"], np.float64).T).reshape(n, H, Dh)
    v = (x @ np.asarray(lw["wv"], np.float64).T).reshape(n, H, Dh)
    q = apply_rope(q, positions, shape.rope_base)
    k = apply_rope(k, positions, shape.rope_base)
    a = causal_cache_attention(q, k, v, k_cache, v_cache).reshape(n, H * Dh)
    h = h + a @ np.asarray(lw["wo"], np.float64).T
    x = rmsnorm(h, lw["ffn_norm"], shape.rms_eps)
    return h + swiglu_ffn(x, lw["w_gate"], lw["w_up"], lw["w_down"]), k, v


def backbone_incremental_forward(shape: BackboneShape, layers: Sequence[dict], tokens,
                                 cache_rows: Callable[[int], tuple], pos: int):
    """The incremental forward of n new tokens (embeddings [n][d]) at positions pos .. pos+n-1 over a cache whose
    layer l holds cache_rows(l) -> (K, V) [L][H][Dh] (keys rotated at their own positions).
    Returns (k_rows, v_rows [n_layers][n][H][Dh] -- the rows to append, keys rotated -- and hidden [n_layers][n][d])."""
    h = np.asarray(tokens, np.float64)
    positions = pos + np.arange(h.shape[0], dtype=np.float64)
    ks, vs, hidden = [], [], []
    for layer, lw in enumerate(layers):
        kc, vc = cache_rows(layer)
        h, k, v = backbone_layer(h, lw, kc, vc, positions, shape)
        ks.append(k)
        vs.append(v)
        hidden.append(h)
    return np.stack(ks), np.stack(vs), np.stack(hidden)
