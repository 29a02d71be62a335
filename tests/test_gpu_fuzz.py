"""Seeded random shapes through the whole forward, every agent against the fp64 oracle.

Each case draws its configuration from its own seed (so a failure names a reproducible shape): 1-3 layers, width
128-512, 4-32 heads of 128, SwiGLU width 256-2048, 8-16 expert tokens, 0-70 frame tokens (one to six query tiles),
1-6 agents with lengths 0-400 (some empty) on rings that wrap at random rows, a bf16 or fp8 cache in either layout,
and the persistent tick kernel or the per-phase launches.  The shapes stay inside what the tick kernel takes (at
most 4 heads and 512 FFN columns per XCD).
"""

from __future__ import annotations

import sys

import numpy as np
import pytest

import synth
from harness import Cache, Model, record, rel_err, run_forward, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
FP8_TOL = 6e-2
N_CASES = 24


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def draw(case: int):
    """The configuration of one case, from its own seed."""
    rng = np.random.default_rng([7919, case])
    B = int(rng.integers(1, 7))
    lengths = [int(x) for x in rng.integers(0, 401, B)]
    if B > 1 and rng.random() < 0.5:
        lengths[int(rng.integers(0, B))] = 0  # an agent with an empty cache
    capacity = max(max(lengths), 1) + int(rng.integers(0, 41))
    starts = [int(x) for x in rng.integers(0, capacity, B)]
    wl = synth.Workload(
        name=f"fuzz{case}", wid=300 + case, n_layers=int(rng.integers(1, 4)),
        d_model=int(rng.choice([128, 256, 384, 512])), n_heads=int(rng.choice([4, 8, 16, 24, 32])), head_dim=128,
        d_ffn=int(rng.choice([256, 512, 768, 1024, 2048])), n_expert_tokens=int(rng.choice([8, 10, 16])),
        n_frame_tokens=int(rng.choice([0, 0, 7, 30, 70])), batch=B, lengths=tuple(lengths), dtype="bf16",
        cache_dtype=str(rng.choice(["bf16", "fp8"])), capacity=capacity)
    layout = fsx.CACHE_TOKEN_MAJOR if rng.random() < 0.5 else fsx.CACHE_HEAD_MAJOR
    flags = fsx.FLAG_MULTI_LAUNCH if rng.random() < 0.3 else 0
    return wl, starts, layout, flags


def test_draws_cover_the_intended_space():
    """The seeded draws reach the kinds of case the fuzz is for (checked on the configurations alone)."""
    cases = [draw(c) for c in range(N_CASES)]
    assert any(wl.cache_dtype == "fp8" for wl, *_ in cases) and any(wl.cache_dtype == "bf16" for wl, *_ in cases)
    assert any(lay == fsx.CACHE_TOKEN_MAJOR for _, _, lay, _ in cases)
    assert any(fl == fsx.FLAG_MULTI_LAUNCH for *_, fl in cases) and any(fl == 0 for *_, fl in cases)
    assert any(wl.seq > 16 for wl, *_ in cases) and any(wl.seq <= 16 for wl, *_ in cases)
    assert any(0 in wl.lengths for wl, *_ in cases)


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_shape_matches_oracle(case):
    wl, starts, layout, flags = draw(case)
    say(f"case fuzz {case}: layers {wl.n_layers}, d {wl.d_model}, heads {wl.n_heads}, ffn {wl.d_ffn}, "
        f"T {wl.n_expert_tokens}, F {wl.n_frame_tokens}, lengths {list(wl.lengths)}, capacity {wl.capacity}, "
        f"starts {starts}, cache {wl.cache_dtype}, "
        f"{'token' if layout == fsx.CACHE_TOKEN_MAJOR else 'head'}-major, "
        f"{'per-phase' if flags else 'tick kernel'}")
    model = Model(wl)
    ex = model.create(flags=flags)
    cache = Cache(wl, starts=starts, layout=layout)
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, wl.n_frame_tokens)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        if wl.cache_dtype == "fp8":
            record(b, rel_err(wp[b], ref), FP8_TOL, what="waypoints vs bf16 source, max|d| / max|ref|")
            refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
            record(b, rel_err(wp[b], refd), BF16_TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")
        else:
            record(b, rel_err(wp[b], ref), BF16_TOL)
    ex.close()
