"""GPU forms of the append-only golden test (Sec. 3.3: a cache grown by incremental appends equals one written at
once), the token-major cache layout, and the expert without rotary encoding (the paper's own positional form,
Sec. 3.1).

* A ring built by appends of 4 rows (one frame per append) from empty must hold exactly the bytes of a ring into
  which the same rows were written in one go, and the forwards over the two must give bitwise-identical waypoints;
  also when the appends wrap the ring.
* Every forward path reads a token-major cache ([capacity][H][Dh] per layer) as it reads a head-major one.
* rope_base = 0 (no rotary encoding on the expert tokens) matches the oracle on the tick kernel and on the per-phase
  launches, for one and for several query tiles per agent.
"""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import synth
from harness import Cache, Model, record, rel_err, run_forward, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

TOL = 2e-2
LAYOUTS = {"head-major": fsx.CACHE_HEAD_MAJOR, "token-major": fsx.CACHE_TOKEN_MAJOR}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small(wid, lengths, capacity, n_frame=0, n_heads=4, n_layers=2, rope_base=10000.0, cache_dtype="bf16"):
    return synth.Workload(name=f"golden{wid}", wid=wid, n_layers=n_layers, d_model=128, n_heads=n_heads, head_dim=128,
                          d_ffn=256, n_expert_tokens=10, n_frame_tokens=n_frame, batch=len(lengths),
                          lengths=tuple(lengths), dtype="bf16", cache_dtype=cache_dtype, capacity=capacity,
                          rope_base=rope_base)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


@pytest.mark.parametrize("layout", sorted(LAYOUTS))
@pytest.mark.parametrize("capacity", [48, 32])  # 40 rows: no wrap, and a wrap by 8 rows
def test_appended_ring_equals_bulk_written_ring(layout, capacity):
    lay = LAYOUTS[layout]
    n_app, n = 10, 4  # ten frames of four rows
    wl = small(200, lengths=(0, 0), capacity=capacity)
    say(f"case golden append-vs-bulk {layout} capacity {capacity}")
    steps = [(synth.append_rows(wl, s, "k", n), synth.append_rows(wl, s, "v", n)) for s in range(n_app)]
    # incremental: appends of 4 rows from an empty ring
    inc = Cache(wl, layout=lay)
    for k_new, v_new in steps:
        fsx.cache_append_rows(inc.desc, inc.rows_for_append(k_new, torch.bfloat16),
                              inc.rows_for_append(v_new, torch.bfloat16), n, fsx.APPEND_RING)
    torch.cuda.synchronize()
    total = n_app * n
    kept = min(total, capacity)
    assert list(inc.desc.len) == [kept] * wl.batch and list(inc.desc.pos) == [total] * wl.batch
    first = total - kept  # oldest row still held
    assert list(inc.desc.start) == [first % capacity] * wl.batch
    # monolithic: the same rows written at once at their slots
    allk = np.concatenate([s[0] for s in steps], axis=2)[:, :, first:]  # [B][layers][kept][H][Dh]
    allv = np.concatenate([s[1] for s in steps], axis=2)[:, :, first:]
    mono = Cache(wl, layout=lay)
    slots = torch.as_tensor((first + np.arange(kept)) % capacity, device="cuda")
    for b in range(wl.batch):
        for l in range(wl.n_layers):
            for dst, src in ((mono.k, allk), (mono.v, allv)):
                rows = torch.from_numpy(np.ascontiguousarray(src[b, l])).to("cuda", torch.bfloat16)  # [kept][H][Dh]
                if lay == fsx.CACHE_TOKEN_MAJOR:
                    dst[b, l].index_copy_(0, slots, rows)
                else:
                    dst[b, l].index_copy_(1, slots, rows.permute(1, 0, 2).contiguous())
    mono.desc.len[:] = kept
    mono.desc.start[:] = first % capacity
    mono.desc.pos[:] = total
    torch.cuda.synchronize()
    assert torch.equal(_bits(inc.k), _bits(mono.k)) and torch.equal(_bits(inc.v), _bits(mono.v)), "cache bytes differ"
    model = Model(wl)
    ex = model.create()
    host_tok, tok = tokens_for(wl)
    wp_inc, _ = run_forward(ex, inc, tok, wl.batch, 0)
    wp_mono, _ = run_forward(ex, mono, tok, wl.batch, 0)
    assert np.array_equal(wp_inc, wp_mono), "waypoints over the appended and the bulk-written ring differ"
    for b in range(wl.batch):
        def rows(l, b=b):
            return allk[b, l].astype(np.float64), allv[b, l].astype(np.float64)
        ref, _ = model.oracle_agent(host_tok[b], rows, total)
        record(b, rel_err(wp_inc[b], ref), TOL)
    ex.close()


@pytest.mark.parametrize("path", ["tick", "per-phase", "generic"])
@pytest.mark.parametrize("n_frame", [0, 64])
def test_token_major_cache_matches_oracle(path, n_frame):
    flags = {"tick": 0, "per-phase": fsx.FLAG_MULTI_LAUNCH, "generic": fsx.FLAG_GENERIC}[path]
    wl = small(210 + n_frame, lengths=(300, 0, 77), capacity=320, n_frame=n_frame, n_heads=16)
    say(f"case token-major {path} n_frame={n_frame}")
    model = Model(wl)
    cache = Cache(wl, starts=(100, 0, 310), layout=fsx.CACHE_TOKEN_MAJOR)
    head = Cache(wl, starts=(100, 0, 310), layout=fsx.CACHE_HEAD_MAJOR)
    host_tok, tok = tokens_for(wl)
    ex = model.create(flags=flags)
    wp, hid = run_forward(ex, cache, tok, wl.batch, n_frame, with_hidden=True)
    wph, _ = run_forward(ex, head, tok, wl.batch, n_frame)
    assert np.array_equal(wp, wph), "token-major and head-major caches give different waypoints"
    for b in range(wl.batch):
        ref, ref_hid = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), TOL, extra={"L": wl.lengths[b]})
        record(b, max(rel_err(hid[l, b], ref_hid[l]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    ex.close()


def test_token_major_fp8_cache_matches_oracle():
    wl = small(220, lengths=(500, 33), capacity=512, cache_dtype="fp8", n_heads=16)
    say("case token-major fp8")
    model = Model(wl)
    cache = Cache(wl, starts=(400, 500), layout=fsx.CACHE_TOKEN_MAJOR)
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), 6e-2, what="waypoints vs bf16 source, max|d| / max|ref|")
        record(b, rel_err(wp[b], refd), TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")
    ex.close()


def test_token_major_append_is_bit_exact():
    wl = small(230, lengths=(30, 64), capacity=64)
    cache = Cache(wl, layout=fsx.CACHE_TOKEN_MAJOR)
    before_k = cache.k.clone()
    n = 4
    k_new = synth.append_rows(wl, 0, "k", n)
    v_new = synth.append_rows(wl, 0, "v", n)
    kd = cache.rows_for_append(k_new, torch.bfloat16)  # [B][layers][n][H][Dh]
    vd = cache.rows_for_append(v_new, torch.bfloat16)
    fsx.cache_append_rows(cache.desc, kd, vd, n, fsx.APPEND_RING)
    torch.cuda.synchronize()
    assert list(cache.desc.len) == [34, 64] and list(cache.desc.start) == [0, 4]
    for l in range(wl.n_layers):
        assert torch.equal(_bits(cache.k[0, l, 30:34]), _bits(kd[0, l]))
        assert torch.equal(_bits(cache.k[1, l, 0:4]), _bits(kd[1, l]))
        assert torch.equal(_bits(cache.v[1, l, 0:4]), _bits(vd[1, l]))
        assert torch.equal(_bits(cache.k[0, l, :30]), _bits(before_k[0, l, :30]))
        assert torch.equal(_bits(cache.k[1, l, 4:]), _bits(before_k[1, l, 4:]))
        assert torch.equal(_bits(cache.k[0, l, 34:]), _bits(before_k[0, l, 34:]))


@pytest.mark.parametrize("path", ["tick", "per-phase"])
@pytest.mark.parametrize("n_frame", [0, 30])
def test_expert_without_rotary_encoding_matches_oracle(path, n_frame):
    """rope_base = 0: learned positional embeddings are part of the input tokens, the expert's q and k are not
    rotated (Sec. 3.1)."""
    flags = {"tick": 0, "per-phase": fsx.FLAG_MULTI_LAUNCH}[path]
    wl = small(240 + n_frame, lengths=(150, 257), capacity=300, n_frame=n_frame, n_heads=16, rope_base=0.0)
    say(f"case no rotary {path} n_frame={n_frame}")
    model = Model(wl)
    cache = Cache(wl, starts=(290, 3))
    host_tok, tok = tokens_for(wl)
    ex = model.create(flags=flags)
    wp, hid = run_forward(ex, cache, tok, wl.batch, n_frame, with_hidden=True)
    for b in range(wl.batch):
        ref, ref_hid = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), TOL)
        record(b, max(rel_err(hid[l, b], ref_hid[l]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    ex.close()
