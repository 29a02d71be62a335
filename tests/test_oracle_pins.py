"""Pins of the fp64 oracle against things other than itself (CPU only).

Each test ties one oracle function to a brute-force construction, a library
routine applied to a case it covers, a closed form, an invariant the paper
states, or a value the format specification prints.  ``test_planted_mistakes``
then plants plausible mistakes in the oracle (on the CPU) and checks that at
least one pin catches each.
"""

from __future__ import annotations

import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import expert as ox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(*key):
    return np.random.default_rng(list(key))


# ----------------------------------------------------------------------------- attention, Eq. (1)

def brute_force_joint_attention(q, k_self, v_self, k_cache, v_cache):
    """Full-sequence masked softmax attention written with scalar loops.

    The sequence is [cached backbone rows ; expert rows].  Backbone rows may not
    attend to expert rows (the asymmetry of Sec. 3.1), expert rows attend to
    everything.  Backbone queries get arbitrary values: with the mask they can
    not influence expert outputs.  Returns the expert rows of the output.
    """
    L, H, Dh = k_cache.shape
    S = q.shape[0]
    n = L + S
    rng = _rng(99)
    q_all = np.concatenate([rng.standard_normal((L, H, Dh)), q], axis=0)
    k_all = np.concatenate([k_cache, k_self], axis=0)
    v_all = np.concatenate([v_cache, v_self], axis=0)
    out = np.zeros((n, H, Dh))
    for h in range(H):
        for i in range(n):
            logits = []
            for j in range(n):
                allowed = not (i < L and j >= L)  # backbone never attends to expert tokens
                if allowed:
                    s = 0.0
                    for c in range(Dh):
                        s += q_all[i, h, c] * k_all[j, h, c]
                    logits.append((j, s / math.sqrt(Dh)))
            mx = max(s for _, s in logits)
            w = [(j, math.exp(s - mx)) for j, s in logits]
            tot = sum(x for _, x in w)
            for j, x in w:
                out[i, h, :] += (x / tot) * v_all[j, h, :]
    return out[L:]


@pytest.mark.parametrize("L,S,H,Dh", [(0, 1, 1, 4), (5, 3, 2, 4), (7, 4, 3, 8), (1, 10, 2, 6)])
def test_attention_matches_brute_force_masked_softmax(L, S, H, Dh):
    r = _rng(1, L, S, H, Dh)
    q, ks, vs = (r.standard_normal((S, H, Dh)) for _ in range(3))
    kc, vc = (r.standard_normal((L, H, Dh)) for _ in range(2))
    got = ox.joint_attention(q, ks, vs, kc, vc)
    want = brute_force_joint_attention(q, ks, vs, kc, vc)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_softmax_rows_sum_to_one():
    # With every value vector equal to ones, each output element is the row sum of P.
    r = _rng(2)
    S, L, H, Dh = 6, 11, 3, 8
    q, ks = r.standard_normal((S, H, Dh)) * 3, r.standard_normal((S, H, Dh))
    kc = r.standard_normal((L, H, Dh)) * 2
    out = ox.joint_attention(q, ks, np.ones((S, H, Dh)), kc, np.ones((L, H, Dh)))
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-13)


def test_attention_invariant_to_cache_row_permutation():
    r = _rng(3)
    S, L, H, Dh = 5, 37, 4, 16
    q, ks, vs = (r.standard_normal((S, H, Dh)) for _ in range(3))
    kc, vc = (r.standard_normal((L, H, Dh)) for _ in range(2))
    perm = r.permutation(L)
    a = ox.joint_attention(q, ks, vs, kc, vc)
    b = ox.joint_attention(q, ks, vs, kc[perm], vc[perm])
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)


def test_empty_cache_reduces_to_textbook_self_attention():
    # L = 0: Eq. (1) is plain multi-head self-attention; torch's SDPA (float64, CPU) is the textbook form.
    r = _rng(4)
    S, H, Dh = 9, 4, 16
    q, k, v = (r.standard_normal((S, H, Dh)) for _ in range(3))
    got = ox.joint_attention(q, k, v, np.zeros((0, H, Dh)), np.zeros((0, H, Dh)))
    t = lambda a: torch.from_numpy(a).permute(1, 0, 2).unsqueeze(0)  # [1][H][S][Dh]
    want = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_cache_attention_equals_library_attention_over_concatenation():
    # L > 0 as one library attention over the concatenated keys (no mask for expert queries).
    r = _rng(5)
    S, L, H, Dh = 4, 23, 2, 32
    q, ks, vs = (r.standard_normal((S, H, Dh)) for _ in range(3))
    kc, vc = (r.standard_normal((L, H, Dh)) for _ in range(2))
    got = ox.joint_attention(q, ks, vs, kc, vc)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).permute(1, 0, 2).unsqueeze(0)
    want = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(np.concatenate([kc, ks])), t(np.concatenate([vc, vs])))[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_split_rows_log_sum_exp_merge_equals_one_softmax():
    # Split-K ("flash-decode") algebra: per-chunk (max, sum, unnormalised output) merged by
    # log-sum-exp rescaling reproduces the single softmax of Eq. (1).
    r = _rng(6)
    S, L, H, Dh = 3, 50, 2, 8
    q, ks, vs = (r.standard_normal((S, H, Dh)) for _ in range(3))
    kc, vc = (r.standard_normal((L, H, Dh)) * 2 for _ in range(2))
    keys = np.concatenate([kc, ks])
    vals = np.concatenate([vc, vs])
    cuts = [0, 7, 8, 30, 49, L + S]
    parts = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        s = np.einsum("shd,rhd->shr", q, keys[a:b]) / math.sqrt(Dh)
        m = s.max(-1)
        p = np.exp(s - m[..., None])
        parts.append((m, p.sum(-1), np.einsum("shr,rhd->shd", p, vals[a:b])))
    M = np.max([p[0] for p in parts], axis=0)
    l = sum(p[1] * np.exp(p[0] - M) for p in parts)
    o = sum(p[2] * np.exp(p[0] - M)[..., None] for p in parts)
    np.testing.assert_allclose(o / l[..., None], ox.joint_attention(q, ks, vs, kc, vc), rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- rotary encoding

def test_rope_equals_complex_multiplication():
    # Pair (x_j, x_{j+Dh/2}) as the complex number x_j + i x_{j+Dh/2}; rotation by angle p*theta_j
    # is multiplication by exp(i p theta_j), theta_j = base^(-2j/Dh).
    r = _rng(7)
    S, H, Dh, base = 5, 3, 16, 10000.0
    x = r.standard_normal((S, H, Dh))
    pos = np.array([0, 1, 17, 4096, 16383], np.float64)
    got = ox.apply_rope(x, pos, base)
    half = Dh // 2
    want = np.empty_like(x)
    for s in range(S):
        for j in range(half):
            w = complex(math.cos(pos[s] * base ** (-2 * j / Dh)), math.sin(pos[s] * base ** (-2 * j / Dh)))
            z = (x[s, :, j] + 1j * x[s, :, j + half]) * w
            want[s, :, j], want[s, :, j + half] = z.real, z.imag
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)


def test_rope_relative_position_and_identity():
    r = _rng(8)
    Dh, base = 32, 10000.0
    q, k = r.standard_normal((1, 1, Dh)), r.standard_normal((1, 1, Dh))
    dots = []
    for shift in (0.0, 5.0, 1000.0):
        qr = ox.apply_rope(q, np.array([12.0 + shift]), base)
        kr = ox.apply_rope(k, np.array([3.0 + shift]), base)
        dots.append(float((qr * kr).sum()))
    np.testing.assert_allclose(dots, dots[0], rtol=0, atol=1e-10)
    np.testing.assert_allclose(ox.apply_rope(q, np.array([0.0]), base), q, rtol=0, atol=0)
    np.testing.assert_allclose(ox.apply_rope(q, np.array([7.0]), 0.0), q, rtol=0, atol=0)  # base 0: no rotary


# ----------------------------------------------------------------------------- norm, FFN, head

def test_rmsnorm_matches_library_and_unit_rms():
    r = _rng(9)
    x = r.standard_normal((7, 64)) * 5
    g = r.standard_normal(64)
    got = ox.rmsnorm(x, g, 1e-6)
    want = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), 1e-6).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)
    unit = ox.rmsnorm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt((unit ** 2).mean(-1)), 1.0, rtol=1e-14)


def test_swiglu_matches_library():
    r = _rng(10)
    x = r.standard_normal((6, 32))
    wg, wu, wd = r.standard_normal((48, 32)), r.standard_normal((48, 32)), r.standard_normal((32, 48))
    T = lambda a: torch.from_numpy(a)
    F = torch.nn.functional
    want = F.linear(F.silu(F.linear(T(x), T(wg))) * F.linear(T(x), T(wu)), T(wd)).numpy()
    np.testing.assert_allclose(ox.swiglu_ffn(x, wg, wu, wd), want, rtol=1e-13, atol=1e-13)


def test_waypoint_head_pools_only_expert_tokens():
    r = _rng(11)
    T, S, d = 10, 14, 16
    h = r.standard_normal((S, d))
    w = r.standard_normal((10, d))
    a = ox.waypoint_head(h, np.ones(d), w, T, 1e-6)
    h2 = h.copy()
    h2[T:] = r.standard_normal((S - T, d)) * 100  # frame-token rows are not pooled
    np.testing.assert_array_equal(a, ox.waypoint_head(h2, np.ones(d), w, T, 1e-6))
    # closed form for one token: head(rmsnorm(h_0)) with T = 1
    b = ox.waypoint_head(h, np.ones(d), w, 1, 0.0)
    x0 = h[0] / np.sqrt((h[0] ** 2).mean())
    np.testing.assert_allclose(b, w @ x0, rtol=1e-13, atol=1e-13)


def loop_mean_pool_head(h, g, w, T, eps):
    """Scalar-loop transcription of the workload head: for each of the first T rows its RMSNorm times the gain,
    averaged over those rows, then the linear map (no bias)."""
    d = h.shape[1]
    pooled = [0.0] * d
    for t in range(T):
        ms = sum(h[t][i] * h[t][i] for i in range(d)) / d
        for i in range(d):
            pooled[i] += h[t][i] / math.sqrt(ms + eps) * g[i] / T
    return np.array([sum(w[o][i] * pooled[i] for i in range(d)) for o in range(w.shape[0])])


@pytest.mark.parametrize("T,S", [(3, 5), (10, 10), (10, 14)])
def test_waypoint_head_mean_pool_matches_loop(T, S):
    # T > 1 with a non-unit final gain: the pooling is a mean (not a sum) of rows normalised one by one (the norm comes
    # before the pooling), and the rows past T (frame tokens) are not pooled.
    r = _rng(17, T, S)
    d = 12
    h = r.standard_normal((S, d)) * (1 + np.arange(S))[:, None]  # rows of different scales
    g = 1 + 0.5 * r.standard_normal(d)
    w = r.standard_normal((10, d))
    got = ox.waypoint_head(h, g, w, T, 1e-6)
    np.testing.assert_allclose(got, loop_mean_pool_head(h, g, w, T, 1e-6), rtol=0, atol=1e-12)


def loop_query_head(h, g, w1, b1, w2, b2, T, nq, eps):
    """Scalar-loop transcription of the two-layer query head: rows T-nq .. T-1, each RMSNorm times the gain, then
    hidden_j = GELU(sum_i w1[j][i] x_i + b1[j]) with GELU(u) = u (1 + erf(u / sqrt 2)) / 2, then out_c = sum_j
    w2[c][j] hidden_j + b2[c]; query q gives outputs 2q, 2q + 1."""
    d = h.shape[1]
    out = []
    for t in range(T - nq, T):
        ms = sum(h[t][i] * h[t][i] for i in range(d)) / d
        x = [h[t][i] / math.sqrt(ms + eps) * g[i] for i in range(d)]
        hid = []
        for j in range(w1.shape[0]):
            u = sum(w1[j][i] * x[i] for i in range(d)) + b1[j]
            hid.append(u * (1.0 + math.erf(u / math.sqrt(2.0))) / 2.0)
        for c in range(2):
            out.append(sum(w2[c][j] * hid[j] for j in range(len(hid))) + b2[c])
    return np.array(out)


def _query_head_inputs(seed=18, T=10, S=12, d=16, hidden=24, nq=5):
    r = _rng(seed)
    h = r.standard_normal((S, d)) * 2
    g = 1 + 0.3 * r.standard_normal(d)
    w1, b1 = r.standard_normal((hidden, d)) * 0.5, r.standard_normal(hidden)
    w2, b2 = r.standard_normal((2, hidden)) * 0.5, r.standard_normal(2)
    return h, g, w1, b1, w2, b2, T, nq


def test_query_head_matches_loop():
    h, g, w1, b1, w2, b2, T, nq = _query_head_inputs()
    got = ox.query_head(h, g, w1, b1, w2, b2, T, nq, 1e-6)
    np.testing.assert_allclose(got, loop_query_head(h, g, w1, b1, w2, b2, T, nq, 1e-6), rtol=0, atol=1e-12)


def test_query_head_matches_library_and_reads_only_the_query_rows():
    h, g, w1, b1, w2, b2, T, nq = _query_head_inputs(seed=19)
    F = torch.nn.functional
    x = torch.from_numpy(h[T - nq:T])
    x = F.rms_norm(x, (h.shape[1],), weight=torch.from_numpy(g), eps=1e-6)
    want = F.linear(F.gelu(F.linear(x, torch.from_numpy(w1), torch.from_numpy(b1))), torch.from_numpy(w2),
                    torch.from_numpy(b2)).numpy().reshape(-1)
    got = ox.query_head(h, g, w1, b1, w2, b2, T, nq, 1e-6)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    h2 = h.copy()
    h2[:T - nq] = 50 * _rng(20).standard_normal((T - nq, h.shape[1]))  # state and visual tokens
    h2[T:] = 50 * _rng(21).standard_normal((h.shape[0] - T, h.shape[1]))  # frame tokens
    np.testing.assert_array_equal(ox.query_head(h2, g, w1, b1, w2, b2, T, nq, 1e-6), got)


def test_gelu_special_values():
    # GELU(0) = 0; GELU(u) - GELU(-u) = u (Phi(u) + Phi(-u) = 1); Phi(1) from its series closed form
    u = np.array([0.0, 0.5, 1.0, 3.0])
    np.testing.assert_allclose(ox.gelu(u) - ox.gelu(-u), u, rtol=0, atol=1e-15)
    assert ox.gelu(np.array([0.0]))[0] == 0.0
    phi1 = 0.5 + sum((-1) ** n / (math.factorial(n) * (2 * n + 1) * 2 ** n) for n in range(40)) / math.sqrt(2 * math.pi)
    np.testing.assert_allclose(ox.gelu(np.array([1.0]))[0], phi1, rtol=1e-15)


# ----------------------------------------------------------------------------- one layer, brute force

def _tiny_layer(r, d=8, H=2, Dh=4, F=12):
    A = H * Dh
    lw = {"wq": r.standard_normal((A, d)) * 0.3, "wk": r.standard_normal((A, d)) * 0.3,
          "wv": r.standard_normal((A, d)) * 0.3, "wo": r.standard_normal((d, A)) * 0.3,
          "w_gate": r.standard_normal((F, d)) * 0.3, "w_up": r.standard_normal((F, d)) * 0.3,
          "w_down": r.standard_normal((d, F)) * 0.3,
          "attn_norm": 1 + 0.1 * r.standard_normal(d), "ffn_norm": 1 + 0.1 * r.standard_normal(d)}
    return lw, ox.ExpertShape(n_layers=1, d_model=d, n_heads=H, head_dim=Dh, d_ffn=F, n_expert_tokens=3,
                              rope_base=100.0)


def brute_force_layer(h, lw, kc, vc, pos, sh):
    """Scalar-loop transcription of one pre-norm layer on tiny inputs."""
    S, d = h.shape
    H, Dh, F = sh.n_heads, sh.head_dim, sh.d_ffn

    def norm(row, g):
        ms = sum(v * v for v in row) / len(row)
        return [row[i] / math.sqrt(ms + sh.rms_eps) * g[i] for i in range(len(row))]

    def lin(row, W):
        return [sum(W[o][i] * row[i] for i in range(len(row))) for o in range(len(W))]

    def rot(vec, p):  # vec: list of Dh for one head
        out = list(vec)
        for j in range(Dh // 2):
            ang = p * sh.rope_base ** (-2 * j / Dh)
            c, s = math.cos(ang), math.sin(ang)
            out[j] = vec[j] * c - vec[j + Dh // 2] * s
            out[j + Dh // 2] = vec[j + Dh // 2] * c + vec[j] * s
        return out

    xs = [norm(list(h[t]), lw["attn_norm"]) for t in range(S)]
    q = [lin(x, lw["wq"]) for x in xs]
    k = [lin(x, lw["wk"]) for x in xs]
    v = [lin(x, lw["wv"]) for x in xs]
    att = [[0.0] * (H * Dh) for _ in range(S)]
    for hd in range(H):
        sl = slice(hd * Dh, (hd + 1) * Dh)
        qh = [rot(q[t][sl], pos + t) for t in range(S)]
        keys = [list(kc[r, hd]) for r in range(kc.shape[0])] + [rot(k[t][sl], pos + t) for t in range(S)]
        vals = [list(vc[r, hd]) for r in range(vc.shape[0])] + [v[t][sl] for t in range(S)]
        for t in range(S):
            sc = [sum(a * b for a, b in zip(qh[t], kk)) / math.sqrt(Dh) for kk in keys]
            mx = max(sc)
            e = [math.exp(s - mx) for s in sc]
            z = sum(e)
            for c in range(Dh):
                att[t][hd * Dh + c] = sum(e[r] / z * vals[r][c] for r in range(len(vals)))
    h1 = [[h[t][i] + lin(att[t], lw["wo"])[i] for i in range(d)] for t in range(S)]
    out = []
    for t in range(S):
        x = norm(h1[t], lw["ffn_norm"])
        g, u = lin(x, lw["w_gate"]), lin(x, lw["w_up"])
        z = [g[i] / (1 + math.exp(-g[i])) * u[i] for i in range(F)]
        dn = lin(z, lw["w_down"])
        out.append([h1[t][i] + dn[i] for i in range(d)])
    return np.array(out)


@pytest.mark.parametrize("L", [0, 1, 6])
def test_layer_matches_brute_force(L):
    r = _rng(12, L)
    lw, sh = _tiny_layer(r)
    S = 4
    h = r.standard_normal((S, sh.d_model))
    kc = r.standard_normal((L, sh.n_heads, sh.head_dim))
    vc = r.standard_normal((L, sh.n_heads, sh.head_dim))
    pos = 5.0
    got = ox.expert_layer(h, lw, kc, vc, pos + np.arange(S), sh)
    np.testing.assert_allclose(got, brute_force_layer(h, lw, kc, vc, pos, sh), rtol=0, atol=1e-12)


def test_layer_with_zero_output_projections_is_identity():
    r = _rng(13)
    lw, sh = _tiny_layer(r)
    lw["wo"] = np.zeros_like(lw["wo"])
    lw["w_down"] = np.zeros_like(lw["w_down"])
    h = r.standard_normal((3, sh.d_model))
    kc = r.standard_normal((4, sh.n_heads, sh.head_dim))
    np.testing.assert_array_equal(ox.expert_layer(h, lw, kc, kc, np.arange(3.0), sh), h)


# ----------------------------------------------------------------------------- forward-level invariants

def _tiny_forward_inputs(seed=14, L=9, S=5, n_layers=2):
    r = _rng(seed)
    layers = []
    for _ in range(n_layers):
        lw, sh = _tiny_layer(r)
        layers.append(lw)
    sh = ox.ExpertShape(n_layers=n_layers, d_model=sh.d_model, n_heads=sh.n_heads, head_dim=sh.head_dim,
                        d_ffn=sh.d_ffn, n_expert_tokens=3, rope_base=100.0)
    toks = r.standard_normal((S, sh.d_model))
    kc = r.standard_normal((n_layers, L, sh.n_heads, sh.head_dim))
    vc = r.standard_normal((n_layers, L, sh.n_heads, sh.head_dim))
    head_w = r.standard_normal((10, sh.d_model))
    return sh, layers, toks, kc, vc, head_w


def test_forward_leaves_cache_untouched_and_is_order_invariant():
    # The backbone never attends to expert tokens, so the cache is read-only for the expert (Sec. 3.1).
    sh, layers, toks, kc, vc, hw = _tiny_forward_inputs()
    kc0, vc0 = kc.copy(), vc.copy()
    wp, hid = ox.expert_forward(sh, layers, np.ones(sh.d_model), hw, toks, lambda l: (kc[l], vc[l]), pos=9)
    np.testing.assert_array_equal(kc, kc0)
    np.testing.assert_array_equal(vc, vc0)
    perm = np.random.default_rng(0).permutation(kc.shape[1])
    wp2, hid2 = ox.expert_forward(sh, layers, np.ones(sh.d_model), hw, toks,
                                  lambda l: (kc[l][perm], vc[l][perm]), pos=9)
    np.testing.assert_allclose(wp2, wp, rtol=0, atol=1e-12)
    assert hid.shape == (sh.n_layers, toks.shape[0], sh.d_model)


def test_forward_is_composition_of_layers_and_head():
    sh, layers, toks, kc, vc, hw = _tiny_forward_inputs(n_layers=3)
    fn = np.ones(sh.d_model)
    wp, hid = ox.expert_forward(sh, layers, fn, hw, toks, lambda l: (kc[l], vc[l]), pos=9)
    pos = 9 + np.arange(toks.shape[0])
    h = toks
    for l in range(3):
        h = brute_force_layer(h, layers[l], kc[l], vc[l], 9.0, sh)
        np.testing.assert_allclose(hid[l], h, rtol=0, atol=1e-11)
    np.testing.assert_allclose(wp, ox.waypoint_head(h, fn, hw, 3, sh.rms_eps), rtol=0, atol=1e-11)
    assert pos[0] == 9


def test_forward_with_empty_cache_depends_only_on_relative_positions():
    # Rotary encoding makes every score depend on the difference of positions only (Sec. 3.1 reading): with no cached
    # rows, moving token 0 from position 9 to 9 + 1000 leaves the forward unchanged; with cached rows (whose keys keep
    # the phases they were cached with) the same move changes it.
    sh, layers, toks, kc, vc, hw = _tiny_forward_inputs(seed=15, L=7)
    fn = np.ones(sh.d_model)
    empty = lambda l: (kc[l][:0], vc[l][:0])
    full = lambda l: (kc[l], vc[l])
    wp0, hid0 = ox.expert_forward(sh, layers, fn, hw, toks, empty, pos=9)
    wp1, hid1 = ox.expert_forward(sh, layers, fn, hw, toks, empty, pos=1009)
    np.testing.assert_allclose(hid1, hid0, rtol=0, atol=1e-10)
    np.testing.assert_allclose(wp1, wp0, rtol=0, atol=1e-10)
    wf0, _ = ox.expert_forward(sh, layers, fn, hw, toks, full, pos=9)
    wf1, _ = ox.expert_forward(sh, layers, fn, hw, toks, full, pos=1009)
    assert np.abs(wf1 - wf0).max() > 1e-3


def test_expert_sequence_attention_is_unmasked():
    # No mask among the expert-sequence tokens (expert and frame tokens see each other, Sec. 3.1 reading): without the
    # rotary encoding (rope_base 0, the learned-embedding form) the layers are equivariant to any permutation of the
    # sequence's rows, and the waypoints, pooled over the first T rows, are invariant to permutations inside the
    # expert rows and inside the frame rows.  A causal or block mask breaks both.
    sh, layers, toks, kc, vc, hw = _tiny_forward_inputs(seed=16, L=5, S=7)
    sh0 = ox.ExpertShape(n_layers=sh.n_layers, d_model=sh.d_model, n_heads=sh.n_heads, head_dim=sh.head_dim,
                         d_ffn=sh.d_ffn, n_expert_tokens=3, rope_base=0.0)
    fn = np.ones(sh.d_model)
    rows = lambda l: (kc[l], vc[l])
    wp, hid = ox.expert_forward(sh0, layers, fn, hw, toks, rows, pos=5)
    perm = np.array([6, 2, 4, 0, 5, 1, 3])  # mixes expert rows (0..2) and frame rows (3..6)
    _, hidp = ox.expert_forward(sh0, layers, fn, hw, toks[perm], rows, pos=5)
    np.testing.assert_allclose(hidp, hid[:, perm], rtol=0, atol=1e-11)
    inside = np.array([2, 0, 1, 5, 6, 3, 4])  # permutes inside the expert rows and inside the frame rows
    wpi, _ = ox.expert_forward(sh0, layers, fn, hw, toks[inside], rows, pos=5)
    np.testing.assert_allclose(wpi, wp, rtol=0, atol=1e-11)
    # a causal mask (row t sees the cache and rows <= t) fails the equivariance
    def causal(q, k_self, v_self, k_cache, v_cache):
        S = q.shape[0]
        return np.stack([ox_joint(q[t:t + 1], k_self[:t + 1], v_self[:t + 1], k_cache, v_cache)[0] for t in range(S)])
    ox_joint = ox.joint_attention
    try:
        ox.joint_attention = causal
        _, hc = ox.expert_forward(sh0, layers, fn, hw, toks, rows, pos=5)
        _, hcp = ox.expert_forward(sh0, layers, fn, hw, toks[perm], rows, pos=5)
    finally:
        ox.joint_attention = ox_joint
    assert np.abs(hcp - hc[:, perm]).max() > 1e-3


def test_append_only_cache_is_exact():
    # Sec. 3.3: with pre-rotated keys, a cache grown by appends equals one built at once; only the
    # set of rows matters.  Appending rows in any split order gives the same forward.
    sh, layers, toks, kc, vc, hw = _tiny_forward_inputs(L=12)
    fn = np.ones(sh.d_model)
    mono = ox.expert_forward(sh, layers, fn, hw, toks, lambda l: (kc[l], vc[l]), pos=12)[0]
    pieces = [slice(8, 12), slice(0, 4), slice(4, 8)]  # appended out of order, as in a wrapped ring
    inc = ox.expert_forward(sh, layers, fn, hw, toks,
                            lambda l: (np.concatenate([kc[l][p] for p in pieces]),
                                       np.concatenate([vc[l][p] for p in pieces])), pos=12)[0]
    np.testing.assert_allclose(inc, mono, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- staleness-augmented training form

def test_staleness_visible_rows_closed_form():
    # Sec. 3.2: the prefix visible to frame j's block ends at frame j - delta, or at the text alone when j < delta
    n_text, per = 64, 4
    v = ox.staleness_visible_rows(n_text, per, 6, 2)
    assert list(v) == [64, 64, 68, 72, 76, 80]  # frames 1, 2 (j < delta and j = delta): text only; frame 3 sees frame 1
    assert list(ox.staleness_visible_rows(n_text, per, 3, 0)) == [68, 72, 76]  # no staleness: up to the frame itself
    assert list(ox.staleness_visible_rows(10, 4, 2, 5)) == [10, 10]


def _multiblock_inputs(seed=23, J=4, S=3, n_text=5, per=2, rope=100.0):
    r = _rng(seed)
    layers = []
    for _ in range(2):
        lw, sh = _tiny_layer(r)
        layers.append(lw)
    sh = ox.ExpertShape(n_layers=2, d_model=sh.d_model, n_heads=sh.n_heads, head_dim=sh.head_dim, d_ffn=sh.d_ffn,
                        n_expert_tokens=3, rope_base=rope)
    L = n_text + per * J
    kc = r.standard_normal((2, L, sh.n_heads, sh.head_dim))
    vc = r.standard_normal((2, L, sh.n_heads, sh.head_dim))
    toks = r.standard_normal((J, S, sh.d_model))
    hw = r.standard_normal((10, sh.d_model))
    return sh, layers, toks, kc, vc, hw


@pytest.mark.parametrize("delta,rope", [(0, 100.0), (2, 100.0), (1, 0.0)])
def test_multiblock_masked_forward_equals_independent_blocks(delta, rope):
    # One masked attention over the whole clip equals running each block alone over its truncated prefix -- the
    # equivalence that lets the blocks run as a batch of agents sharing one cache.
    sh, layers, toks, kc, vc, hw = _multiblock_inputs(rope=rope)
    J = toks.shape[0]
    vis = ox.staleness_visible_rows(5, 2, J, delta)
    pos = vis + 100
    fn = 1 + 0.2 * _rng(24).standard_normal(sh.d_model)
    wp, hid = ox.masked_multiblock_forward(sh, layers, fn, hw, toks, lambda l: (kc[l], vc[l]), vis, pos)
    for j in range(J):
        wj, hj = ox.expert_forward(sh, layers, fn, hw, toks[j], lambda l, j=j: (kc[l][:vis[j]], vc[l][:vis[j]]),
                                   pos=pos[j])
        np.testing.assert_allclose(wp[j], wj, rtol=0, atol=1e-11)
        np.testing.assert_allclose(hid[:, j], hj, rtol=0, atol=1e-11)


def test_multiblock_masked_forward_matches_brute_force_layer():
    # one layer of the clip through the scalar-loop layer of each block over its own visible prefix
    sh, layers, toks, kc, vc, hw = _multiblock_inputs(seed=25, J=3)
    sh1 = ox.ExpertShape(n_layers=1, d_model=sh.d_model, n_heads=sh.n_heads, head_dim=sh.head_dim, d_ffn=sh.d_ffn,
                         n_expert_tokens=3, rope_base=sh.rope_base)
    vis = np.array([5, 7, 9])
    pos = np.array([9.0, 11.0, 13.0])
    _, hid = ox.masked_multiblock_forward(sh1, layers[:1], np.ones(sh.d_model), hw, toks,
                                          lambda l: (kc[l], vc[l]), vis, pos)
    for j in range(3):
        want = brute_force_layer(toks[j], layers[0], kc[0][:vis[j]], vc[0][:vis[j]], pos[j], sh1)
        np.testing.assert_allclose(hid[0, j], want, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------- fp8

def test_e4m3_decode_exhaustive_against_library():
    codes = np.arange(256, dtype=np.uint8)
    got = oracle.e4m3fn_decode(codes)
    lib = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(lib)
    assert nan.sum() == 2 and np.array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], lib[~nan])


def test_e4m3_encode_against_library():
    # round-to-nearest-even onto the E4M3 grid after the clamp: torch's float8_e4m3fn cast, on values already
    # clamped to the finite range (torch itself turns values >= 480 into NaN, hence the clamp), including every
    # midpoint between neighbouring grid values (ties), the subnormal range and the clamp boundaries
    r = _rng(22)
    grid = oracle.e4m3fn_decode(np.arange(0x7F, dtype=np.uint8))
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)
    vals = np.concatenate([r.standard_normal(50000).astype(np.float32) * 40, mids, -mids, grid.astype(np.float32),
                           np.float32([448, -448, 464, 479.9, 1e6, -1e6, 0.0, -0.0, 2.0 ** -10, 3 * 2.0 ** -11])])
    for scale in (np.float32(1.0), np.float32(0.0123)):
        got = oracle.e4m3fn_encode(vals * scale, scale)
        y = np.clip(vals * scale / scale, -448, 448).astype(np.float32)
        want = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        np.testing.assert_array_equal(got, want)


def test_e4m3_encode_is_inverse_of_decode_on_the_grid():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    vals = oracle.e4m3fn_decode(codes).astype(np.float32)
    got = oracle.e4m3fn_encode(vals, np.float32(1.0))
    np.testing.assert_array_equal(got, codes)


def test_e4m3_decode_spec_points():
    for line in open(os.path.join(GOLDEN, "e4m3_spec_points.txt")):
        if line.startswith("#") or not line.strip():
            continue
        code, val = line.split()
        got = float(oracle.e4m3fn_decode(np.array([int(code, 16)], np.uint8))[0])
        if val == "nan":
            assert math.isnan(got)
        else:
            assert got == float(val) and math.copysign(1, got) == math.copysign(1, float(val)), (code, got)


# ----------------------------------------------------------------------------- paper sizes

def test_workload_sizes_follow_the_paper():
    import synth

    g = {}
    for line in open(os.path.join(GOLDEN, "expert_shape.txt")):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            g[k] = int(v)
    wl = synth.WORKLOADS["single_bf16_L224"]
    assert (wl.n_layers, wl.d_model, wl.n_heads, wl.head_dim) == (g["n_layers"], g["d_ae"], g["n_heads"],
                                                                   g["head_dim"])
    assert wl.attn_width == g["qkv_proj_rows"] and wl.d_model == g["qkv_proj_cols"]
    assert wl.n_expert_tokens == g["expert_tokens_per_frame"]
    assert wl.n_out == g["waypoints"] * g["values_per_waypoint"]
    # 40-frame history at 4 backbone rows per frame plus a 64-token instruction
    assert wl.lengths[0] == 64 + g["backbone_tokens_per_frame"] * 40
    b = synth.WORKLOADS["batched_bf16_B16_L1024"]
    assert b.append_rows == g["backbone_tokens_per_frame"]


# ----------------------------------------------------------------------------- planted mistakes

MUTANTS = {
    "attention_scale_1_over_Dh": ("joint_attention", "scale"),
    "rope_sign_flipped": ("apply_rope", "sign"),
    "self_keys_dropped": ("joint_attention", "noself"),
    "gate_up_swapped": ("swiglu_ffn", "swap"),
    "rms_without_sqrt": ("rmsnorm", "nosqrt"),
    "head_sum_instead_of_mean": ("waypoint_head", "headsum"),
    "head_norm_after_pool": ("waypoint_head", "poolnorm"),
    "query_head_tanh_gelu": ("gelu", "tanhgelu"),
    "query_head_bias_dropped": ("query_head", "nobias"),
    "query_head_first_rows": ("query_head", "firstrows"),
    "e4m3_encode_truncates": ("e4m3fn_encode", "trunc"),
    "staleness_off_by_one": ("staleness_visible_rows", "vis_off1"),
    "multiblock_blocks_see_each_other": ("masked_multiblock_forward", "blockleak"),
    "e4m3_encode_ties_toward_zero": ("e4m3fn_encode", "tieslow"),
}


def _mutant(kind):
    if kind == "scale":
        def f(q, ks, vs, kc, vc):
            return ORIG["joint_attention"](np.asarray(q) / math.sqrt(q.shape[-1]), ks, vs, kc, vc)
    elif kind == "noself":
        def f(q, ks, vs, kc, vc):
            if len(kc) == 0:
                return ORIG["joint_attention"](q, ks, vs, kc, vc)
            s = np.einsum("shd,rhd->hsr", q, kc) / math.sqrt(q.shape[-1])
            p = np.exp(s - s.max(-1, keepdims=True))
            p /= p.sum(-1, keepdims=True)
            return np.einsum("hsr,rhd->shd", p, vc)
    elif kind == "sign":
        def f(x, positions, base):
            return ORIG["apply_rope"](x, -np.asarray(positions, np.float64), base)
    elif kind == "swap":
        def f(x, wg, wu, wd):
            return ORIG["swiglu_ffn"](x, wu, wg, wd)
    elif kind == "nosqrt":
        def f(x, gain, eps):
            x = np.asarray(x, np.float64)
            return x / (np.mean(x * x, -1, keepdims=True) + eps) * gain
    elif kind == "headsum":
        def f(h, g, w, T, eps):
            return ORIG["waypoint_head"](h, g, w, T, eps) * T
    elif kind == "poolnorm":
        def f(h, g, w, T, eps):
            x = np.asarray(h, np.float64)[:T].mean(axis=0, keepdims=True)
            return ox.rmsnorm(x, g, eps)[0] @ np.asarray(w, np.float64).T
    elif kind == "tanhgelu":
        def f(u):
            u = np.asarray(u, np.float64)
            return 0.5 * u * (1 + np.tanh(math.sqrt(2 / math.pi) * (u + 0.044715 * u ** 3)))
    elif kind == "nobias":
        def f(h, g, w1, b1, w2, b2, T, nq, eps):
            return ORIG["query_head"](h, g, w1, np.zeros_like(b1), w2, b2, T, nq, eps)
    elif kind == "firstrows":
        def f(h, g, w1, b1, w2, b2, T, nq, eps):
            return ORIG["query_head"](h, g, w1, b1, w2, b2, nq, nq, eps)
    elif kind == "vis_off1":
        def f(n_text, per, n_frames, delta):
            j = np.arange(1, n_frames + 1)
            return n_text + per * np.maximum(0, j - delta + 1)
    elif kind == "blockleak":
        def f(shape, layers, final_norm, head, block_tokens, prefix_rows, visible, positions):
            # every block also attends to the other blocks' rows: one block holding all the clip's expert tokens
            # would be the unmasked form; emulate with the first block seeing the second block's tokens
            bt = np.asarray(block_tokens, np.float64)
            wp, hid = ORIG["masked_multiblock_forward"](shape, layers, final_norm, head, bt, prefix_rows, visible,
                                                        positions)
            if bt.shape[0] > 1:
                both = np.concatenate([bt[0], bt[1]], axis=0)[None]
                sh2 = ox.ExpertShape(**{**shape.__dict__})
                w2, h2 = ORIG["masked_multiblock_forward"](sh2, layers, final_norm, head, both, prefix_rows,
                                                           np.asarray(visible)[:1], np.asarray(positions)[:1])
                hid = hid.copy()
                hid[:, 0] = h2[:, 0, :bt.shape[1]]
                wp = wp.copy()
                wp[0] = w2[0]
            return wp, hid
    elif kind == "trunc":
        def f(x, scale):
            y = np.clip(np.asarray(x, np.float32) / np.float32(scale), -448, 448).astype(np.float64)
            grid = oracle.e4m3fn_decode(np.arange(0x7F, dtype=np.uint8))
            idx = np.searchsorted(grid, np.abs(y), side="right") - 1
            return np.where(np.signbit(y), idx | 0x80, idx).astype(np.uint8)
    elif kind == "tieslow":
        def f(x, scale):
            y = np.clip(np.asarray(x, np.float32) / np.float32(scale), -448, 448).astype(np.float64)
            grid = oracle.e4m3fn_decode(np.arange(0x7F, dtype=np.uint8))
            a = np.abs(y)
            idx = np.argmin(np.abs(grid[None, :] - a.reshape(-1, 1)), axis=1)  # first (smaller) of two nearest
            return np.where(np.signbit(y).reshape(-1), idx | 0x80, idx).astype(np.uint8).reshape(np.shape(x))
    return f


ORIG = {n: getattr(ox, n) for n in ("joint_attention", "apply_rope", "swiglu_ffn", "rmsnorm", "waypoint_head",
                                    "query_head", "gelu")}
ORIG["e4m3fn_encode"] = oracle.fp8.e4m3fn_encode
ORIG["staleness_visible_rows"] = ox.staleness_visible_rows
ORIG["masked_multiblock_forward"] = ox.masked_multiblock_forward
PIN_TESTS = [
    lambda: test_attention_matches_brute_force_masked_softmax(5, 3, 2, 4),
    lambda: test_cache_attention_equals_library_attention_over_concatenation(),
    lambda: test_rope_equals_complex_multiplication(),
    lambda: test_swiglu_matches_library(),
    lambda: test_rmsnorm_matches_library_and_unit_rms(),
    lambda: test_layer_matches_brute_force(6),
    lambda: test_waypoint_head_mean_pool_matches_loop(3, 5),
    lambda: test_query_head_matches_loop(),
    lambda: test_query_head_matches_library_and_reads_only_the_query_rows(),
    lambda: test_e4m3_encode_against_library(),
    lambda: test_staleness_visible_rows_closed_form(),
    lambda: test_multiblock_masked_forward_equals_independent_blocks(2, 100.0),
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    fn_name, kind = MUTANTS[name]
    if fn_name == "e4m3fn_encode":
        monkeypatch.setattr(oracle.fp8, fn_name, _mutant(kind))
        monkeypatch.setattr(oracle, fn_name, _mutant(kind))
    else:
        monkeypatch.setattr(ox, fn_name, _mutant(kind))
    caught = 0
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            caught += 1
    assert caught >= 1, f"no pin caught the planted mistake {name}"
