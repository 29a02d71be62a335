"""The persistent tick kernel: agreement with the per-phase launch path, consecutive ticks with new inputs,
per-layer hidden outputs, and the bounded-wait failure path (forced from the host by a tiny wait limit)."""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import synth
from harness import Cache, Model, oracle_agents, record, rel_err, run_forward, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small(wid, lengths, n_frame=0, capacity=400, n_layers=3, d_model=128, n_heads=4, d_ffn=256):
    return synth.Workload(name=f"tick{wid}", wid=wid, n_layers=n_layers, d_model=d_model, n_heads=n_heads,
                          head_dim=128, d_ffn=d_ffn, n_expert_tokens=10, n_frame_tokens=n_frame,
                          batch=len(lengths), lengths=tuple(lengths), dtype="bf16", cache_dtype="bf16",
                          capacity=capacity)


# n_frame 30, 50, 90: 3, 4 and 7 query tiles per agent (7: more than one attention pass over the cache)
@pytest.mark.parametrize("n_frame", [0, 30, 50, 90])
def test_tick_kernel_and_per_phase_launches_match_oracle(n_frame):
    wl = small(70 + n_frame, lengths=(17, 0, 250, 399), n_frame=n_frame)
    say(f"case tick vs per-phase, n_frame={n_frame}")
    model = Model(wl)
    cache = Cache(wl, starts=(390, 0, 200, 1))
    host_tok, tok = tokens_for(wl)
    outs = {}
    for name, flags in (("tick", 0), ("per-phase", fsx.FLAG_MULTI_LAUNCH)):
        ex = model.create(flags=flags)
        wp, hid = run_forward(ex, cache, tok, wl.batch, n_frame, with_hidden=True)
        outs[name] = (wp, hid)
        ex.close()
    for b in range(wl.batch):
        ref, ref_hid = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        for name, (wp, hid) in outs.items():
            record(b, rel_err(wp[b], ref), TOL, what=f"{name} waypoints, max|d| / max|ref|")
            record(b, max(rel_err(hid[l, b], ref_hid[l]) for l in range(wl.n_layers)), TOL,
                   what=f"{name} worst layer hidden, max|d| / max|ref|")
    assert rel_err(outs["tick"][0], outs["per-phase"][0]) <= 1e-2


@pytest.mark.parametrize("lengths", [(150,), (0,), (333,)])
def test_single_agent_small_matches_oracle(lengths):
    """One agent, one query tile, 2 heads per XCD (one attention workgroup per head, no partial states), per-layer
    hidden outputs included; cache lengths 150 (ragged last tile), 0 (own rows only) and 333."""
    wl = small(96 + lengths[0] % 7, lengths=lengths, capacity=400, n_layers=3, d_model=256, n_heads=16)
    say(f"case single agent, L={lengths[0]}")
    model = Model(wl)
    cache = Cache(wl, starts=(123,))
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp, hid = run_forward(ex, cache, tok, 1, 0, with_hidden=True)
    ref, ref_hid = model.oracle_agent(host_tok[0], cache.oracle_rows(0), cache.desc.pos[0])
    record(0, rel_err(wp[0], ref), TOL)
    record(0, max(rel_err(hid[l, 0], ref_hid[l]) for l in range(wl.n_layers)), TOL,
           what="worst layer hidden, max|d| / max|ref|")
    ex.close()


# 32 heads (4 per XCD, 96 Q units per XCD), one workgroup per attention segment: with 2 agents the 24 other
# workgroups of an XCD have exactly one wave per Q unit and take them all; with 3 agents the 20 others are too few
# and every workgroup takes Q units
@pytest.mark.parametrize("lengths", [(200, 37), (90, 0, 150)])
def test_attention_workgroups_with_and_without_q_units_match_oracle(lengths):
    wl = small(120 + len(lengths), lengths=lengths, capacity=256, n_layers=2, d_model=128, n_heads=32)
    say(f"case {len(lengths)} agents of 32 heads, L={lengths}")
    model = Model(wl)
    cache = Cache(wl, starts=tuple(31 * (b + 1) for b in range(len(lengths))))
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp, hid = run_forward(ex, cache, tok, wl.batch, 0, with_hidden=True)
    for b in range(wl.batch):
        ref, ref_hid = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), TOL, extra={"L": lengths[b]})
        record(b, max(rel_err(hid[l, b], ref_hid[l]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    ex.close()


def test_maximum_batch_of_agents_matches_oracle():
    """64 agents (the batch limit) of 32 heads: 256 attention segments per XCD (the plan's limit), 640 rows in eight
    row blocks; ragged cache lengths (0 included) in rings with different starts.  Every agent is checked."""
    rng = np.random.default_rng(7)
    lengths = tuple(int(x) for x in rng.integers(0, 121, 64))
    lengths = (0,) + lengths[1:]
    wl = small(90, lengths=lengths, capacity=128, n_layers=2, d_model=128, n_heads=32)
    say("case 64 agents")
    model = Model(wl)
    cache = Cache(wl, starts=tuple(int(x) for x in rng.integers(0, 128, 64)))
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    pos = [int(p) for p in cache.desc.pos]
    refs = oracle_agents(model, range(wl.batch),
                         lambda b: model.oracle_agent(host_tok[b], cache.oracle_rows(b), pos[b])[0])
    for b in range(wl.batch):
        record(b, rel_err(wp[b], refs[b]), TOL, extra={"L": lengths[b]})
    assert np.isfinite(wp).all()
    ex.close()


@pytest.mark.parametrize("n_frame", [30, 64])
def test_many_query_slices_across_agents_match_oracle(n_frame):
    """Several query tiles per agent with enough cache rows that every workgroup takes an equal slice of the XCD's
    tiles: slices cut segments of different agents and leave partial states merged per query tile."""
    wl = small(110 + n_frame, lengths=(3000, 2500, 3100), capacity=3200, n_layers=2, d_model=128, n_heads=16,
               n_frame=n_frame)
    say(f"case many-query slices, n_frame={n_frame}")
    model = Model(wl)
    cache = Cache(wl, starts=(3000, 17, 900))
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp, _ = run_forward(ex, cache, tok, wl.batch, n_frame)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), TOL)
    ex.close()


def test_consecutive_ticks_with_new_inputs():
    """Each tick must see its own inputs: forward A, then B (new tokens and cache), then A again."""
    wl_a = small(80, lengths=(64, 120))
    wl_b = wl_a.replace(wid=81)  # other tokens and cache; the weights stay those of A
    model = Model(wl_a)
    ex = model.create()
    cache_a = Cache(wl_a)
    cache_b = Cache(wl_b)
    host_a, tok_a = tokens_for(wl_a)
    host_b, tok_b = tokens_for(wl_b)
    for rnd, (cache, host, tok) in enumerate(((cache_a, host_a, tok_a), (cache_b, host_b, tok_b),
                                              (cache_a, host_a, tok_a))):
        wp, _ = run_forward(ex, cache, tok, wl_a.batch, 0)
        for b in range(wl_a.batch):
            ref, _ = model.oracle_agent(host[b], cache.oracle_rows(b), cache.desc.pos[b])
            record(b, rel_err(wp[b], ref), TOL, what=f"round {rnd} waypoints, max|d| / max|ref|")


def test_many_ticks_are_bitwise_reproducible():
    wl = small(82, lengths=(300,), n_layers=2)
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    _, tok = tokens_for(wl)
    first, _ = run_forward(ex, cache, tok, 1, 0)
    wp = torch.empty((1, wl.n_out), device="cuda")
    for _ in range(50):
        fsx.expert_forward(ex, cache.desc, tok, 1, 0, wp)
    torch.cuda.synchronize()
    fsx.expert_status(ex)
    assert np.array_equal(wp.cpu().numpy(), first)


def test_wait_limit_failure_is_reported_and_poisons_waypoints():
    """A 1 us bound on every wait makes the tick give up: waypoints NaN, status reports it once."""
    wl = small(83, lengths=(200, 50), n_layers=2)
    model = Model(wl)
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    ex_lim = model.create(tick_timeout_us=1)
    wp, _ = run_forward(ex_lim, cache, tok, wl.batch, 0)
    assert np.isnan(wp).all()
    with pytest.raises(fsx.FsxError) as e:
        fsx.expert_status(ex_lim)
    assert e.value.code == 5 and "timed out" in str(e.value)
    fsx.expert_status(ex_lim)  # reported once
    ex_lim.close()
    ex = model.create()  # an expert with the default bound works on the same inputs
    wp2, _ = run_forward(ex, cache, tok, wl.batch, 0)
    fsx.expert_status(ex)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        assert rel_err(wp2[b], ref) <= TOL
