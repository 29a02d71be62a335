"""Pins of the backbone oracle (incremental forward, Sec. 3.3) against things other than itself (CPU only).

The golden test of the paper (monolithic against incremental prefill) is a pin here: a sequence run at once from an
empty cache and the same sequence appended frame by frame, each step reading the rows the previous steps appended,
give the same rows and hidden states.  Then a scalar-loop layer, causality, the single-token case against the
pinned unmasked joint attention, and torch's causal scaled-dot-product attention; planted mistakes must be caught.
"""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import backbone as ob
from oracle import expert as ox


def _rng(*key):
    return np.random.default_rng(list(key))


def _layers(r, n_layers=2, d=8, H=2, Dh=4, F=12):
    A = H * Dh
    out = []
    for _ in range(n_layers):
        out.append({"wq": r.standard_normal((A, d)) * 0.3, "wk": r.standard_normal((A, d)) * 0.3,
                    "wv": r.standard_normal((A, d)) * 0.3, "wo": r.standard_normal((d, A)) * 0.3,
                    "w_gate": r.standard_normal((F, d)) * 0.3, "w_up": r.standard_normal((F, d)) * 0.3,
                    "w_down": r.standard_normal((d, F)) * 0.3,
                    "attn_norm": 1 + 0.1 * r.standard_normal(d), "ffn_norm": 1 + 0.1 * r.standard_normal(d)})
    return out, ob.BackboneShape(n_layers=n_layers, d_model=d, n_heads=H, head_dim=Dh, d_ffn=F, rope_base=100.0)


@pytest.mark.parametrize("split", [(12,), (4, 4, 4), (1, 3, 8), (5, 7)])
def test_monolithic_equals_incremental_prefill(split):
    # Sec. 3.3: rotary phases make append-only caching exact; the paper's golden test compares monolithic against
    # incremental prefill.  The rows each step appends are the rows the monolithic pass produces for those tokens.
    r = _rng(30)
    layers, sh = _layers(r)
    toks = r.standard_normal((12, sh.d_model))
    empty = lambda l: (np.zeros((0, sh.n_heads, sh.head_dim)),) * 2
    k_mono, v_mono, h_mono = ob.backbone_incremental_forward(sh, layers, toks, empty, 0)
    kc = [np.zeros((0, sh.n_heads, sh.head_dim)) for _ in layers]
    vc = [np.zeros((0, sh.n_heads, sh.head_dim)) for _ in layers]
    hs, t0 = [], 0
    for n in split:
        k, v, h = ob.backbone_incremental_forward(sh, layers, toks[t0:t0 + n], lambda l: (kc[l], vc[l]), t0)
        for l in range(sh.n_layers):
            kc[l] = np.concatenate([kc[l], k[l]])
            vc[l] = np.concatenate([vc[l], v[l]])
        hs.append(h)
        t0 += n
    np.testing.assert_allclose(np.stack(kc), k_mono, rtol=0, atol=1e-12)
    np.testing.assert_allclose(np.stack(vc), v_mono, rtol=0, atol=1e-12)
    np.testing.assert_allclose(np.concatenate(hs, axis=1), h_mono, rtol=0, atol=1e-12)


def brute_force_backbone_layer(h, lw, kc, vc, pos, sh):
    """Scalar-loop transcription of one causal decoder layer over new tokens with a cache."""
    n, d = h.shape
    H, Dh, F = sh.n_heads, sh.head_dim, sh.d_ffn

    def norm(row, g):
        ms = sum(v * v for v in row) / len(row)
        return [row[i] / math.sqrt(ms + sh.rms_eps) * g[i] for i in range(len(row))]

    def lin(row, W):
        return [sum(W[o][i] * row[i] for i in range(len(row))) for o in range(len(W))]

    def rot(vec, p):
        out = list(vec)
        for j in range(Dh // 2):
            ang = p * sh.rope_base ** (-2 * j / Dh)
            c, s = math.cos(ang), math.sin(ang)
            out[j] = vec[j] * c - vec[j + Dh // 2] * s
            out[j + Dh // 2] = vec[j + Dh // 2] * c + vec[j] * s
        return out

    xs = [norm(list(h[t]), lw["attn_norm"]) for t in range(n)]
    q, k, v = [lin(x, lw["wq"]) for x in xs], [lin(x, lw["wk"]) for x in xs], [lin(x, lw["wv"]) for x in xs]
    att = [[0.0] * (H * Dh) for _ in range(n)]
    for hd in range(H):
        sl = slice(hd * Dh, (hd + 1) * Dh)
        for t in range(n):
            qt = rot(q[t][sl], pos + t)
            keys = [list(kc[r, hd]) for r in range(kc.shape[0])] + [rot(k[j][sl], pos + j) for j in range(t + 1)]
            vals = [list(vc[r, hd]) for r in range(vc.shape[0])] + [v[j][sl] for j in range(t + 1)]
            sc = [sum(a * b for a, b in zip(qt, kk)) / math.sqrt(Dh) for kk in keys]
            mx = max(sc)
            e = [math.exp(s - mx) for s in sc]
            z = sum(e)
            for c in range(Dh):
                att[t][hd * Dh + c] = sum(e[i] / z * vals[i][c] for i in range(len(vals)))
    out = []
    for t in range(n):
        h1 = [h[t][i] + lin(att[t], lw["wo"])[i] for i in range(d)]
        x = norm(h1, lw["ffn_norm"])
        g, u = lin(x, lw["w_gate"]), lin(x, lw["w_up"])
        z = [g[i] / (1 + math.exp(-g[i])) * u[i] for i in range(F)]
        dn = lin(z, lw["w_down"])
        out.append([h1[i] + dn[i] for i in range(d)])
    return np.array(out)


@pytest.mark.parametrize("L", [0, 5])
def test_backbone_layer_matches_brute_force(L):
    r = _rng(31, L)
    layers, sh = _layers(r, n_layers=1)
    h = r.standard_normal((4, sh.d_model))
    kc, vc = r.standard_normal((L, sh.n_heads, sh.head_dim)), r.standard_normal((L, sh.n_heads, sh.head_dim))
    got, _, _ = ob.backbone_layer(h, layers[0], kc, vc, 7 + np.arange(4.0), sh)
    np.testing.assert_allclose(got, brute_force_backbone_layer(h, layers[0], kc, vc, 7, sh), rtol=0, atol=1e-12)


def test_new_tokens_do_not_see_later_tokens():
    r = _rng(32)
    layers, sh = _layers(r)
    toks = r.standard_normal((6, sh.d_model))
    kc = r.standard_normal((2, 5, sh.n_heads, sh.head_dim))
    rows = lambda l: (kc[l], kc[l] * 0.5)
    k1, v1, h1 = ob.backbone_incremental_forward(sh, layers, toks, rows, 5)
    toks2 = toks.copy()
    toks2[3:] += 10 * r.standard_normal((3, sh.d_model))
    k2, v2, h2 = ob.backbone_incremental_forward(sh, layers, toks2, rows, 5)
    np.testing.assert_array_equal(h2[:, :3], h1[:, :3])
    np.testing.assert_array_equal(k2[:, :3], k1[:, :3])
    assert np.abs(h2[:, 3:] - h1[:, 3:]).max() > 1e-3


def test_single_new_token_equals_unmasked_joint_attention_and_library_causal_attention():
    r = _rng(33)
    H, Dh, L = 3, 8, 6
    q, k, v = (r.standard_normal((1, H, Dh)) for _ in range(3))
    kc, vc = r.standard_normal((L, H, Dh)), r.standard_normal((L, H, Dh))
    np.testing.assert_allclose(ob.causal_cache_attention(q, k, v, kc, vc), ox.joint_attention(q, k, v, kc, vc),
                               rtol=0, atol=1e-13)
    n = 5  # no cache: torch's causal attention over the new tokens alone
    q, k, v = (r.standard_normal((n, H, Dh)) for _ in range(3))
    empty = np.zeros((0, H, Dh))
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a.transpose(1, 0, 2)))
    want = torch.nn.functional.scaled_dot_product_attention(T(q), T(k), T(v), is_causal=True).numpy()
    np.testing.assert_allclose(ob.causal_cache_attention(q, k, v, empty, empty), want.transpose(1, 0, 2),
                               rtol=1e-12, atol=1e-12)


MUTANTS = ("no_causal_mask", "keys_not_rotated", "cache_ignored")


def _mutant(kind, orig_attn, orig_layer):
    if kind == "no_causal_mask":
        return "causal_cache_attention", lambda q, kn, vn, kc, vc: ox.joint_attention(q, kn, vn, kc, vc)
    if kind == "keys_not_rotated":
        def layer(h, lw, kc, vc, positions, shape):
            s0 = ob.BackboneShape(**{**shape.__dict__, "rope_base": 0.0})
            out, k, v = orig_layer(h, lw, kc, vc, positions, shape)
            _, k0, _ = orig_layer(h, lw, kc, vc, positions, s0)
            return out, k0, v
        return "backbone_layer", layer
    return "causal_cache_attention", lambda q, kn, vn, kc, vc: orig_attn(q, kn, vn, kc[:0], vc[:0])


@pytest.mark.parametrize("kind", MUTANTS)
def test_planted_mistakes_are_caught(kind, monkeypatch):
    name, fn = _mutant(kind, ob.causal_cache_attention, ob.backbone_layer)
    monkeypatch.setattr(ob, name, fn)
    caught = 0
    for t in (lambda: test_monolithic_equals_incremental_prefill((4, 4, 4)), lambda: test_backbone_layer_matches_brute_force(5),
              test_new_tokens_do_not_see_later_tokens,
              test_single_new_token_equals_unmasked_joint_attention_and_library_causal_attention):
        try:
            t()
        except AssertionError:
            caught += 1
    assert caught >= 1, kind
