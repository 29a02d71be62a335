"""The allocation-free tick (fsx_expert_forward_noalloc, workspace in the library's static device array) against
fsx_expert_forward on the same handle and inputs, on two calls in a row, the second smaller than the first (fewer
agents, fewer frame tokens, shorter caches), so the second call runs over what the first left in the array.  Both
results are also held to the oracle at the bf16 tolerance.  Calls that need more than the array, or handles that do
not run the tick kernel, are refused before any GPU work."""

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


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def wl_of(wid, lengths, n_frame):
    return synth.Workload(name=f"noalloc{wid}", wid=wid, n_layers=2, d_model=256, n_heads=16, head_dim=128, d_ffn=512,
                          n_expert_tokens=10, n_frame_tokens=n_frame, batch=len(lengths), lengths=tuple(lengths),
                          dtype="bf16", cache_dtype="bf16", capacity=640)


def noalloc_forward(ex, cache, tok, batch, n_frame, with_hidden=True):
    wl = cache.wl
    S = wl.n_expert_tokens + n_frame
    wp = torch.full((batch, wl.n_out), float("nan"), device="cuda")
    hid = torch.full((wl.n_layers, batch, S, wl.d_model), float("nan"), device="cuda") if with_hidden else None
    fsx.expert_forward_noalloc(ex, cache.desc, tok, batch, n_frame, wp, hid)
    torch.cuda.synchronize()
    return wp.cpu().numpy(), (hid.cpu().numpy() if with_hidden else None)


def test_noalloc_tick_matches_forward_on_two_calls():
    big = wl_of(300, lengths=(600, 37, 250), n_frame=30)
    model = Model(big)
    ex = model.create(max_batch=3, max_frame_tokens=30)
    calls = [(big, (5, 0, 300)), (wl_of(301, lengths=(120,), n_frame=0), (100,))]
    for i, (wl, starts) in enumerate(calls):
        say(f"case noalloc call {i}: {wl.batch} agents, {wl.n_frame_tokens} frame tokens, L={wl.lengths}")
        cache = Cache(wl, starts=starts)
        host_tok, tok = tokens_for(wl)
        wp_na, hid_na = noalloc_forward(ex, cache, tok, wl.batch, wl.n_frame_tokens)
        wp, hid = run_forward(ex, cache, tok, wl.batch, wl.n_frame_tokens, with_hidden=True)
        assert np.array_equal(wp_na, wp), "waypoints differ from fsx_expert_forward"
        assert np.array_equal(hid_na, hid), "hidden states differ from fsx_expert_forward"
        for b in range(wl.batch):
            ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
            record(b, rel_err(wp_na[b], ref), TOL, what=f"call {i} waypoints, max|d| / max|ref|")
    ex.close()


def test_noalloc_refuses_what_does_not_fit():
    # full widths, one layer, 64 agents of 10 tokens: the workspace exceeds the static array
    wl = synth.Workload(name="noalloc_big", wid=302, n_layers=1, d_model=512, n_heads=32, head_dim=128, d_ffn=2048,
                        n_expert_tokens=10, n_frame_tokens=0, batch=64, lengths=(16,) * 64, dtype="bf16",
                        cache_dtype="bf16", capacity=16)
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    _, tok = tokens_for(wl)
    wp = torch.zeros((wl.batch, wl.n_out), device="cuda")
    with pytest.raises(fsx.FsxError) as e:
        fsx.expert_forward_noalloc(ex, cache.desc, tok, wl.batch, 0, wp)
    assert e.value.code == 3 and "bytes" in str(e.value)
    ex.close()
    small = wl_of(303, lengths=(40,), n_frame=0)
    m2 = Model(small)
    ex2 = m2.create(flags=fsx.FLAG_MULTI_LAUNCH)
    c2 = Cache(small)
    _, t2 = tokens_for(small)
    with pytest.raises(fsx.FsxError) as e:
        fsx.expert_forward_noalloc(ex2, c2.desc, t2, 1, 0, torch.zeros((1, small.n_out), device="cuda"))
    assert e.value.code == 2
    ex2.close()
