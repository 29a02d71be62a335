"""The paper's own expert form (Sec. 3.1) on every path: no rotary encoding on the expert tokens (learned positional
embeddings, here a seeded table added to the token embeddings before the call, so both sides receive the same
folded tokens) and the two-layer head that decodes the last five expert tokens (the waypoint queries) to five
(x, y) waypoints.  Reference: the oracle with the same head (query_head)."""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import synth
from harness import Cache, Model, record, rel_err, run_forward
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def paper_form(wl: synth.Workload, hidden: int) -> synth.Workload:
    return wl.replace(rope_base=0.0, head_kind=1, head_hidden=hidden)


def folded_tokens(wl):
    """Token embeddings plus a learned positional embedding per sequence slot (a seeded table, bf16-rounded sum)."""
    tok = synth.make_tokens(wl)
    pe = np.random.default_rng([wl.wid, 77]).standard_normal((wl.seq, wl.d_model)).astype(np.float32) * 0.5
    host = synth.round_to(tok + pe[None], wl.dtype)
    td = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    return host, torch.from_numpy(host).to("cuda", td)


@pytest.mark.parametrize("path", ["tick", "per-phase", "generic"])
@pytest.mark.parametrize("n_frame", [0, 30])
def test_paper_form_small_matches_oracle(path, n_frame):
    flags = {"tick": 0, "per-phase": fsx.FLAG_MULTI_LAUNCH, "generic": fsx.FLAG_GENERIC}[path]
    wl = paper_form(synth.Workload(name="paper_small", wid=500 + n_frame, n_layers=2, d_model=256, n_heads=16,
                                   head_dim=128, d_ffn=512, n_expert_tokens=10, n_frame_tokens=n_frame, batch=3,
                                   lengths=(200, 0, 77), dtype="bf16", cache_dtype="bf16", capacity=256), hidden=256)
    say(f"case paper form {path} n_frame={n_frame}")
    model = Model(wl)
    ex = model.create(flags=flags)
    cache = Cache(wl, starts=(100, 0, 250))
    host_tok, tok = folded_tokens(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, n_frame)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), 2e-2)
    ex.close()


def test_paper_form_tiny_fp32_matches_oracle():
    wl = paper_form(synth.WORKLOADS["tiny_fp32_L40"], hidden=48)
    say("case paper form tiny fp32")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = folded_tokens(wl)
    wp, _ = run_forward(ex, cache, tok, 1, 0)
    ref, _ = model.oracle_agent(host_tok[0], cache.oracle_rows(0), cache.desc.pos[0])
    record(0, float(np.abs(wp[0] - ref).max()), 1e-4, what="waypoints, max|d|")
    ex.close()


@pytest.mark.slow
def test_paper_form_full_40_frame_shape_matches_oracle():
    """The full-size expert (32 layers, width 512, 32 x 128 heads) at the 40-frame history, in the paper's form."""
    wl = paper_form(synth.WORKLOADS["single_bf16_L224"], hidden=512)
    say("case paper form single_bf16_L224")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = folded_tokens(wl)
    wp, hid = run_forward(ex, cache, tok, 1, 0, with_hidden=True)
    ref, ref_hid = model.oracle_agent(host_tok[0], cache.oracle_rows(0), cache.desc.pos[0])
    record(0, rel_err(wp[0], ref), 2e-2)
    record(0, max(rel_err(hid[l, 0], ref_hid[l]) for l in range(wl.n_layers)), 2e-2,
           what="worst layer hidden, max|d| / max|ref|")
    ex.close()


def test_query_head_arguments_are_validated():
    wl = paper_form(synth.Workload(name="paper_bad", wid=510, n_layers=1, d_model=128, n_heads=4, head_dim=128,
                                   d_ffn=256, n_expert_tokens=4, n_frame_tokens=0, batch=1, lengths=(8,),
                                   dtype="bf16", cache_dtype="bf16", capacity=8), hidden=64)
    model = Model(wl)
    with pytest.raises(fsx.FsxError) as e:  # five waypoint queries do not fit into four expert tokens
        model.create()
    assert e.value.code == 1
