"""GPU parity of the HIP expert tick against the fp64 oracle (same seeded inputs).

Tolerances:
  fp32 expert      : max-abs waypoint error <= 1e-4, per-layer hidden max-abs error <= 1e-3
  bf16 expert      : max |wp - wp_ref| / max |wp_ref| <= 2e-2 per agent
  fp8-stored cache : same relative form, <= 6e-2 (graded against the bf16 source values)
  append           : bit-exact
The bf16 per-layer hidden bound (2e-2 of the layer's max magnitude) is derived from bf16 rounding of the
projection inputs (relative 2^-9 per element, accumulated over 32 layers), see the design notes.
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

BF16_WP_TOL = 2e-2
FP8_WP_TOL = 6e-2
BF16_HID_TOL = 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small_bf16(name="small_bf16", wid=10, lengths=(0, 40, 333), n_frame=0, capacity=400, n_layers=2):
    return synth.Workload(name=name, wid=wid, n_layers=n_layers, d_model=128, n_heads=4, head_dim=128, d_ffn=256,
                          n_expert_tokens=10, n_frame_tokens=n_frame, batch=len(lengths), lengths=tuple(lengths),
                          dtype="bf16", cache_dtype="bf16", capacity=capacity)


def check_agents(model, cache, host_tok, wp, hid, agents, wp_tol, hid_tol=None, absolute=False, decoded=False):
    for b in agents:
        ref_wp, ref_hid = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=decoded), cache.desc.pos[b])
        if absolute:
            err = float(np.abs(wp[b] - ref_wp).max())
        else:
            err = rel_err(wp[b], ref_wp)
        record(b, err, wp_tol, what="waypoints, max|d|" if absolute else "waypoints, max|d| / max|ref|",
               extra={"L": cache.lengths[b]})
        if hid is not None and hid_tol is not None:
            worst = 0.0
            for l in range(ref_hid.shape[0]):
                if absolute:
                    e = float(np.abs(hid[l, b] - ref_hid[l]).max())
                else:
                    e = rel_err(hid[l, b], ref_hid[l])
                worst = max(worst, e)
            record(b, worst, hid_tol, what="worst layer hidden, max|d|" if absolute else
                   "worst layer hidden, max|d| / max|ref|")


def test_tiny_fp32_expert_matches_oracle():
    wl = synth.WORKLOADS["tiny_fp32_L40"]
    say("case tiny_fp32_L40")
    model = Model(wl)
    ex = model.create()
    assert fsx.expert_info(ex)["path"] == 1
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    wp, hid = run_forward(ex, cache, tok, 1, 0, with_hidden=True)
    check_agents(model, cache, host_tok, wp, hid, [0], 1e-4, 1e-3, absolute=True)


@pytest.mark.parametrize("n_frame", [0, 22])
def test_small_bf16_fused_path_matches_oracle(n_frame):
    wl = small_bf16(lengths=(0, 40, 333), n_frame=n_frame, wid=10 + n_frame)
    say(f"case small_bf16 n_frame={n_frame}")
    model = Model(wl)
    ex = model.create()
    assert fsx.expert_info(ex)["path"] == 0
    cache = Cache(wl, starts=(0, 390, 7))  # agent 1 wraps around the ring end
    host_tok, tok = tokens_for(wl)
    wp, hid = run_forward(ex, cache, tok, wl.batch, n_frame, with_hidden=True)
    check_agents(model, cache, host_tok, wp, hid, range(wl.batch), BF16_WP_TOL, BF16_HID_TOL)


def test_small_bf16_generic_path_matches_oracle():
    wl = small_bf16(lengths=(5, 70), n_frame=3, wid=30)
    say("case small_bf16 generic path")
    model = Model(wl)
    ex = model.create(flags=fsx.FLAG_GENERIC)
    assert fsx.expert_info(ex)["path"] == 1
    cache = Cache(wl, starts=(398, 0))
    host_tok, tok = tokens_for(wl)
    wp, hid = run_forward(ex, cache, tok, wl.batch, 3, with_hidden=True)
    check_agents(model, cache, host_tok, wp, hid, range(wl.batch), BF16_WP_TOL, BF16_HID_TOL)


def test_full_single_agent_L224_matches_oracle_and_leaves_cache_untouched():
    wl = synth.WORKLOADS["single_bf16_L224"]
    say("case single_bf16_L224")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    k0, v0 = cache.k.clone(), cache.v.clone()
    host_tok, tok = tokens_for(wl)
    wp, hid = run_forward(ex, cache, tok, 1, 0, with_hidden=True)
    check_agents(model, cache, host_tok, wp, hid, [0], BF16_WP_TOL, BF16_HID_TOL)
    assert torch.equal(cache.k, k0) and torch.equal(cache.v, v0), "forward wrote the cache"
    wp2, _ = run_forward(ex, cache, tok, 1, 0)
    assert np.array_equal(wp, wp2), "two forwards differ bitwise"


def test_full_long_history_with_frame_tokens_matches_oracle():
    wl = synth.WORKLOADS["long_bf16_L4096_F64"]
    say("case long_bf16_L4096_F64")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, 1, wl.n_frame_tokens)
    check_agents(model, cache, host_tok, wp, None, [0], BF16_WP_TOL)


def test_small_permuted_cache_rows_give_same_waypoints():
    wl = small_bf16(lengths=(200,), wid=40, capacity=256)
    say("case permutation invariance")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, 1, 0)
    perm = torch.randperm(200, generator=torch.Generator().manual_seed(0)).to(cache.k.device)
    cache.k[0, :, :, :200] = cache.k[0, :, :, :200][:, :, perm]
    cache.v[0, :, :, :200] = cache.v[0, :, :, :200][:, :, perm]
    torch.cuda.synchronize()
    wp2, _ = run_forward(ex, cache, tok, 1, 0)
    assert rel_err(wp2, wp) <= 1e-2
