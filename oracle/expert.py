"""fp64 reference of the action-expert forward (Sec. 3.1, Eq. (1); Sec. 3.3).

TEST INFRASTRUCTURE ONLY -- see the package docstring.  Imports nothing but
NumPy.

The expert is a stack of transformer layers that reads the frozen backbone's
per-layer key/value cache.  At layer l it projects its own tokens into the
backbone's attention geometry (H heads of width Dh, so A = H*Dh) with
rectangular projections W_q, W_k, W_v (A x d), runs ONE attention over the
concatenation [cached backbone keys ; its own keys] and the matching values
(Eq. (1)), projects back to width d with W_o, and applies a SwiGLU feed-forward
block (Sec. 3.1).  The backbone never attends to expert tokens, so the cache is
an input that the forward only reads (Sec. 3.1, Sec. 3.3).  Waypoints are
regressed from the expert tokens (Sec. 3.1, per-frame token list).

Readings of what the paper leaves open (each is also listed in the design
notes; the GPU path implements the same readings):

* Normalisation: pre-norm RMSNorm before attention and before the FFN, with
  residual adds, eps = 1e-6, and a final RMSNorm before the head.  The paper
  names neither the norm nor its placement.
* Positional encoding: rotary encoding of q and k of every expert-sequence
  token at positions pos, pos+1, ..., pos+S-1, pairing channel j with
  j + Dh/2, angle p * base^(-2j/Dh).  The paper's own expert uses learned
  positional embeddings and no rotary encoding (Sec. 3.1); ``rope_base = 0``
  reproduces that form (learned embeddings are then part of the input
  tokens).  Cached backbone keys are used as stored: they already carry the
  rotary phases they were cached with (Sec. 3.1).
* Attention scale 1/sqrt(Dh), no mask: every expert-sequence token (expert
  tokens and optional current-frame tokens) attends to every cached row and
  to every expert-sequence token.
* Full multi-head attention: q, k and v all have H heads (the paper gives the
  backbone's 32-head, 128-wide geometry and no grouping).
* FFN: z = (silu(x W_g^T) * (x W_u^T)) W_d^T with silu(u) = u / (1 + e^-u).
* Head (workload form, ``head_kind = 0``): final RMSNorm, mean over the first
  T (expert) tokens, then a linear d -> n_out map without bias; outputs
  ordered x0, y0, ..., x4, y4.
* Head (the paper's form, ``head_kind = 1``, Sec. 3.1): the five learnable
  waypoint queries are decoded to five (x, y) waypoints by a two-layer head.
  The paper gives neither the width nor the activation; reading: the queries
  are the LAST n_out/2 of the T expert tokens (the per-frame token list puts
  the state token and the four visual tokens first), each query row goes
  through the final RMSNorm, Linear(d -> hidden) with bias, GELU in its exact
  erf form, Linear(hidden -> 2) with bias; query i gives (x_i, y_i).
* Staleness-augmented training form (Sec. 3.2): frames are numbered from 1;
  frame j's block sees the prefix up to frame j - delta (text alone when
  j <= delta); blocks do not see each other (per-block masks).
* Precision: no intermediate rounding anywhere -- everything is float64.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable, Sequence

import numpy as np


@dataclass(frozen=True)
class ExpertShape:
    """Sizes of the expert (Sec. 3.1: 32 layers, width 512, 32 heads x 128)."""

    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    n_expert_tokens: int = 10
    n_out: int = 10
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    head_kind: int = 0  # 0: mean-pool + linear; 1: two-layer head over the waypoint queries
    head_hidden: int = 0  # width of the two-layer head's hidden layer (head_kind 1)

    @property
    def attn_width(self) -> int:
        return self.n_heads * self.head_dim


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm: x / sqrt(mean(x^2) + eps) * gain (reading: LLaMA pre-norm)."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def rope_cos_sin(positions: np.ndarray, head_dim: int, base: float):
    """cos/sin of the rotary angles p * base^(-2j/Dh), j < Dh/2, in float64.

    Returns two arrays of shape [len(positions)][Dh/2].
    """
    half = head_dim // 2
    j = np.arange(half, dtype=np.float64)
    theta = np.power(np.float64(base), -2.0 * j / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate channel pairs (j, j+Dh/2) of x[S][H][Dh] by the angle of each row's position.

    (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin).  base <= 0 means no rotation.
    """
    x = np.asarray(x, dtype=np.float64)
    if base <= 0:
        return x.copy()
    dh = x.shape[-1]
    half = dh // 2
    cos, sin = rope_cos_sin(positions, dh, base)
    cos = cos[:, None, :]
    sin = sin[:, None, :]
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def joint_attention(q, k_self, v_self, k_cache, v_cache) -> np.ndarray:
    """Eq. (1): Attn(Q_ae, [K_vlm; K_ae], [V_vlm; V_ae]) for every head.

    q, k_self, v_self: [S][H][Dh]; k_cache, v_cache: [L][H][Dh] (L may be 0).
    One softmax per (query, head) over all L + S keys, scale 1/sqrt(Dh).
    Returns [S][H][Dh].
    """
    q = np.asarray(q, dtype=np.float64)
    dh = q.shape[-1]
    keys = np.concatenate([np.asarray(k_cache, np.float64), np.asarray(k_self, np.float64)], axis=0)
    vals = np.concatenate([np.asarray(v_cache, np.float64), np.asarray(v_self, np.float64)], axis=0)
    # head-major views: qh [H][S][Dh], kh/vh [H][L+S][Dh]
    qh = np.ascontiguousarray(q.transpose(1, 0, 2))
    kh = np.ascontiguousarray(keys.transpose(1, 0, 2))
    vh = np.ascontiguousarray(vals.transpose(1, 0, 2))
    scores = np.matmul(qh, kh.transpose(0, 2, 1)) / np.sqrt(np.float64(dh))  # [H][S][L+S]
    scores = scores - scores.max(axis=-1, keepdims=True)
    p = np.exp(scores)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.matmul(p, vh).transpose(1, 0, 2)  # [S][H][Dh]


def silu(u: np.ndarray) -> np.ndarray:
    return u / (1.0 + np.exp(-u))


def swiglu_ffn(x, w_gate, w_up, w_down) -> np.ndarray:
    """SwiGLU feed-forward block (Sec. 3.1): (silu(x Wg^T) * (x Wu^T)) Wd^T."""
    x = np.asarray(x, dtype=np.float64)
    g = x @ np.asarray(w_gate, np.float64).T
    u = x @ np.asarray(w_up, np.float64).T
    return (silu(g) * u) @ np.asarray(w_down, np.float64).T


def expert_layer(h, lw: dict, k_cache, v_cache, positions, shape: ExpertShape) -> np.ndarray:
    """One expert layer (Sec. 3.1): pre-norm joint attention + O-proj, pre-norm SwiGLU.

    h: [S][d] residual stream.  lw: dict with wq, wk, wv ([A][d]), wo ([d][A]),
    w_gate, w_up ([d_ffn][d]), w_down ([d][d_ffn]), attn_norm, ffn_norm ([d]).
    k_cache, v_cache: this layer's cached backbone rows [L][H][Dh].
    """
    h = np.asarray(h, dtype=np.float64)
    S = h.shape[0]
    H, Dh = shape.n_heads, shape.head_dim
    x = rmsnorm(h, lw["attn_norm"], shape.rms_eps)
    q = (x @ np.asarray(lw["wq"], np.float64).T).reshape(S, H, Dh)
    k = (x @ np.asarray(lw["wk"], np.float64).T).reshape(S, H, Dh)
    v = (x @ np.asarray(lw["wv"], np.float64).T).reshape(S, H, Dh)
    q = apply_rope(q, positions, shape.rope_base)
    k = apply_rope(k, positions, shape.rope_base)
    a = joint_attention(q, k, v, k_cache, v_cache).reshape(S, H * Dh)
    h = h + a @ np.asarray(lw["wo"], np.float64).T
    x = rmsnorm(h, lw["ffn_norm"], shape.rms_eps)
    return h + swiglu_ffn(x, lw["w_gate"], lw["w_up"], lw["w_down"])


def waypoint_head(h, final_norm, head_w, n_expert_tokens: int, eps: float) -> np.ndarray:
    """Final RMSNorm, mean over the expert tokens (rows < T), linear d -> n_out."""
    x = rmsnorm(np.asarray(h, np.float64)[:n_expert_tokens], final_norm, eps)
    return x.mean(axis=0) @ np.asarray(head_w, np.float64).T


def gelu(u: np.ndarray) -> np.ndarray:
    """GELU in its exact form u * Phi(u) = u / 2 * (1 + erf(u / sqrt(2)))."""
    u = np.asarray(u, dtype=np.float64)
    erf = np.vectorize(math.erf, otypes=[np.float64])
    return 0.5 * u * (1.0 + erf(u / math.sqrt(2.0)))


def query_head(h, final_norm, w1, b1, w2, b2, n_expert_tokens: int, n_queries: int, eps: float) -> np.ndarray:
    """The paper's waypoint head (Sec. 3.1): n_queries waypoint-query tokens, each decoded by a two-layer head.

    The queries are rows T - n_queries .. T - 1 of the residual stream (the last expert tokens).  Each row is
    final-normalised, mapped by Linear(d -> hidden) + b1, GELU, Linear(hidden -> 2) + b2.  Returns
    [x0, y0, x1, y1, ...] (query i gives waypoint i).
    """
    h = np.asarray(h, np.float64)
    x = rmsnorm(h[n_expert_tokens - n_queries:n_expert_tokens], final_norm, eps)
    u = gelu(x @ np.asarray(w1, np.float64).T + np.asarray(b1, np.float64))
    y = u @ np.asarray(w2, np.float64).T + np.asarray(b2, np.float64)
    return y.reshape(-1)


def apply_head(shape: "ExpertShape", h, final_norm, head) -> np.ndarray:
    """The head of ``shape.head_kind``: head is W_head [n_out][d] (kind 0) or a dict w1, b1, w2, b2 (kind 1)."""
    if shape.head_kind == 1:
        return query_head(h, final_norm, head["w1"], head["b1"], head["w2"], head["b2"], shape.n_expert_tokens,
                          shape.n_out // 2, shape.rms_eps)
    return waypoint_head(h, final_norm, head, shape.n_expert_tokens, shape.rms_eps)


def expert_forward(
    shape: ExpertShape,
    layers: Sequence[dict],
    final_norm,
    head_w,
    tokens,
    cache_rows: Callable[[int], tuple],
    pos: int,
):
    """One tick of the expert for ONE agent (agents are independent).

    tokens: [S][d] expert-sequence embeddings (rows < T expert tokens, the rest
    optional current-frame tokens).  cache_rows(l) -> (K, V), each [L][H][Dh],
    the valid cached rows of layer l in any order (attention is invariant to
    the order of cache rows).  pos: position of token 0.
    head_w: the head's parameters (see ``apply_head``).
    Returns (waypoints [n_out], hidden [n_layers][S][d]).
    """
    h = np.asarray(tokens, dtype=np.float64)
    S = h.shape[0]
    positions = pos + np.arange(S, dtype=np.float64)
    hidden = []
    for layer, lw in enumerate(layers):
        kc, vc = cache_rows(layer)
        h = expert_layer(h, lw, kc, vc, positions, shape)
        hidden.append(h)
    wp = apply_head(shape, h, final_norm, head_w)
    return wp, np.stack(hidden)


# ----------------------------------------------------------------------------- staleness-augmented training form

def staleness_visible_rows(n_text: int, rows_per_frame: int, n_frames: int, delta: int) -> np.ndarray:
    """Backbone prefix rows visible to the expert block of each frame j = 1..n_frames (Sec. 3.2): the prefix ends at
    frame j - delta, or at the instruction text alone when j < delta (frames are numbered from 1, so j = delta also
    sees the text alone).  Returns [n_frames] row counts."""
    j = np.arange(1, n_frames + 1)
    return n_text + rows_per_frame * np.maximum(0, j - delta)


def masked_multiblock_forward(shape: ExpertShape, layers: Sequence[dict], final_norm, head, block_tokens,
                              prefix_rows: Callable[[int], tuple], visible, positions):
    """All expert blocks of a training clip in ONE forward (Sec. 3.2): the clip's sequence is [backbone prefix ;
    block 0 ; block 1 ; ...]; at every layer one attention runs over it with a per-block mask -- a query of block j
    sees prefix rows < visible[j] and the rows of block j, nothing else (the backbone rows never attend to expert
    rows, so the prefix is an input).  The MLP acts per token and the head per block.

    block_tokens: [J][S][d]; prefix_rows(l) -> (K, V) [L][H][Dh] (the whole prefix of layer l, rows in order);
    visible: [J] rows of the prefix block j sees; positions: [J] position of block j's token 0.
    Returns waypoints [J][n_out] and hidden [n_layers][J][S][d].
    """
    blocks = np.asarray(block_tokens, np.float64)
    J, S, d = blocks.shape
    H, Dh = shape.n_heads, shape.head_dim
    h = blocks.reshape(J * S, d)
    pos = (np.asarray(positions, np.float64)[:, None] + np.arange(S)[None, :]).reshape(J * S)
    blk = np.repeat(np.arange(J), S)
    hidden = []
    for layer, lw in enumerate(layers):
        kc, vc = (np.asarray(a, np.float64) for a in prefix_rows(layer))
        L = kc.shape[0]
        x = rmsnorm(h, lw["attn_norm"], shape.rms_eps)
        q = apply_rope((x @ np.asarray(lw["wq"], np.float64).T).reshape(J * S, H, Dh), pos, shape.rope_base)
        k = apply_rope((x @ np.asarray(lw["wk"], np.float64).T).reshape(J * S, H, Dh), pos, shape.rope_base)
        v = (x @ np.asarray(lw["wv"], np.float64).T).reshape(J * S, H, Dh)
        keys = np.concatenate([kc, k], axis=0)  # [L + J S][H][Dh]
        vals = np.concatenate([vc, v], axis=0)
        # mask [J S][L + J S]: prefix row r visible to block j iff r < visible[j]; expert row visible iff same block
        allow = np.concatenate([np.arange(L)[None, :] < np.asarray(visible)[blk][:, None],
                                blk[:, None] == blk[None, :]], axis=1)
        sc = np.einsum("thc,rhc->htr", q, keys) / np.sqrt(np.float64(Dh))
        sc = np.where(allow[None], sc, -np.inf)
        sc = sc - sc.max(axis=-1, keepdims=True)
        p = np.exp(sc)
        p = p / p.sum(axis=-1, keepdims=True)
        a = np.einsum("htr,rhc->thc", p, vals).reshape(J * S, H * Dh)
        h = h + a @ np.asarray(lw["wo"], np.float64).T
        x = rmsnorm(h, lw["ffn_norm"], shape.rms_eps)
        h = h + swiglu_ffn(x, lw["w_gate"], lw["w_up"], lw["w_down"])
        hidden.append(h.reshape(J, S, d))
    wp = np.stack([apply_head(shape, h.reshape(J, S, d)[j], final_norm, head) for j in range(J)])
    return wp, np.stack(hidden)
