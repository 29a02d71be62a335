"""GPU tests of the cache side: append (bit-exact, ring wrap, error policy), batched agents, the fp8 cache.

Append is checked byte for byte against host slicing of the generator's rows; forwards after an append
are checked against the oracle over the rows the ring then holds.
"""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from harness import Cache, Model, head_major_rows, oracle_agents, record, rel_err, run_forward, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

BF16_WP_TOL = 2e-2
FP8_WP_TOL = 6e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small(wid, lengths, capacity, cache_dtype="bf16", n_layers=2):
    return synth.Workload(name=f"small{wid}", wid=wid, n_layers=n_layers, d_model=128, n_heads=4, head_dim=128,
                          d_ffn=256, n_expert_tokens=10, n_frame_tokens=0, batch=len(lengths),
                          lengths=tuple(lengths), dtype="bf16", cache_dtype=cache_dtype, capacity=capacity)


def rows_after_append(wl, b, l, kind, new_rows, capacity, start_len):
    """The multiset of rows the ring holds after appending new_rows to the generator's slab (oldest evicted)."""
    old = synth.cache_slab(wl, b, l, kind, rows=start_len)
    allr = np.concatenate([old, new_rows], axis=0)
    return allr[max(0, allr.shape[0] - capacity):]


def test_append_is_bit_exact_and_wraps_the_ring():
    wl = small(50, lengths=(30, 64), capacity=64)
    say("case append ring")
    cache = Cache(wl)
    before_k = cache.k.clone()
    n = 4
    k_new = synth.append_rows(wl, 0, "k", n)
    v_new = synth.append_rows(wl, 0, "v", n)
    kd = head_major_rows(k_new, torch.bfloat16)
    vd = head_major_rows(v_new, torch.bfloat16)
    fsx.cache_append_rows(cache.desc, kd, vd, n, fsx.APPEND_RING)
    torch.cuda.synchronize()
    # agent 0: rows 30..33 written, start 0, len 34; agent 1: full ring, slots 0..3 overwritten, start 4
    assert list(cache.desc.len) == [34, 64] and list(cache.desc.start) == [0, 4] and list(cache.desc.pos) == [34, 68]
    for l in range(wl.n_layers):
        assert torch.equal(cache.k[0, l, :, 30:34].view(torch.int16), kd[0, l].view(torch.int16))
        assert torch.equal(cache.k[1, l, :, 0:4].view(torch.int16), kd[1, l].view(torch.int16))
        assert torch.equal(cache.v[1, l, :, 0:4].view(torch.int16), vd[1, l].view(torch.int16))
        # the bytes are the generator's rows of that (layer, head)
        assert torch.equal(cache.k[1, l, 2, 0:4].float().cpu(), torch.from_numpy(k_new[1, l, :, 2]))
        # untouched rows keep their bytes
        assert torch.equal(cache.k[0, l, :, :30].view(torch.int16), before_k[0, l, :, :30].view(torch.int16))
        assert torch.equal(cache.k[1, l, :, 4:].view(torch.int16), before_k[1, l, :, 4:].view(torch.int16))
        assert torch.equal(cache.k[0, l, :, 34:].view(torch.int16), before_k[0, l, :, 34:].view(torch.int16))


def test_append_error_policy_rejects_and_writes_nothing():
    wl = small(51, lengths=(60,), capacity=62)
    cache = Cache(wl)
    before = cache.k.clone()
    kd = torch.zeros((1, wl.n_layers, wl.n_heads, 4, wl.head_dim), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(fsx.FsxError) as e:
        fsx.cache_append_rows(cache.desc, kd, kd, 4, fsx.APPEND_ERROR)
    assert e.value.code == 3
    torch.cuda.synchronize()
    assert torch.equal(cache.k, before) and list(cache.desc.len) == [60]
    with pytest.raises(fsx.FsxError) as e:
        fsx.cache_append_rows(cache.desc, kd, kd, 63, fsx.APPEND_RING)  # more rows than the ring holds
    assert e.value.code == 3


def test_forward_after_wrapping_append_matches_oracle():
    wl = small(52, lengths=(64, 20), capacity=64)
    say("case forward after wrap")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    n = 6
    k_new = synth.append_rows(wl, 0, "k", n)
    v_new = synth.append_rows(wl, 0, "v", n)
    fsx.cache_append_rows(cache.desc, head_major_rows(k_new, torch.bfloat16), head_major_rows(v_new, torch.bfloat16), n)
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    for b in range(wl.batch):
        def rows(l, b=b):
            return (rows_after_append(wl, b, l, "k", k_new[b, l], 64, wl.lengths[b]).astype(np.float64),
                    rows_after_append(wl, b, l, "v", v_new[b, l], 64, wl.lengths[b]).astype(np.float64))
        ref, _ = model.oracle_agent(host_tok[b], rows, cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), BF16_WP_TOL)


@pytest.mark.slow
def test_batched_agents_then_append_match_oracle():
    """16 agents x 1024 cached rows sharing the weights, then 4 rows appended per agent and layer; every agent is
    compared with the oracle before and after the append."""
    wl = synth.WORKLOADS["batched_bf16_B16_L1024"]
    say("case batched_bf16_B16_L1024")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    pos0 = [int(p) for p in cache.desc.pos]
    refs = oracle_agents(model, range(wl.batch),
                         lambda b: model.oracle_agent(host_tok[b], cache.oracle_rows(b), pos0[b])[0])
    for b in range(wl.batch):
        record(b, rel_err(wp[b], refs[b]), BF16_WP_TOL)
    n = wl.append_rows
    k_new = synth.append_rows(wl, 0, "k", n)
    v_new = synth.append_rows(wl, 0, "v", n)
    kd = head_major_rows(k_new, torch.bfloat16)
    vd = head_major_rows(v_new, torch.bfloat16)
    fsx.cache_append_rows(cache.desc, kd, vd, n)
    torch.cuda.synchronize()
    assert all(int(x) == 1028 for x in cache.desc.len)
    assert torch.equal(cache.k[:, :, :, 1024:1028].view(torch.int16), kd.view(torch.int16))
    assert torch.equal(cache.v[:, :, :, 1024:1028].view(torch.int16), vd.view(torch.int16))
    wp2, _ = run_forward(ex, cache, tok, wl.batch, 0)
    pos1 = [int(p) for p in cache.desc.pos]

    def after(b):
        def rows(l):
            return (rows_after_append(wl, b, l, "k", k_new[b, l], wl.capacity, 1024).astype(np.float64),
                    rows_after_append(wl, b, l, "v", v_new[b, l], wl.capacity, 1024).astype(np.float64))
        return model.oracle_agent(host_tok[b], rows, pos1[b])[0]

    refs = oracle_agents(model, range(wl.batch), after)
    for b in range(wl.batch):
        record(b, rel_err(wp2[b], refs[b]), BF16_WP_TOL, what="waypoints after append, max|d| / max|ref|")


def test_fp8_decode_of_every_code_on_the_gpu():
    """All 254 finite E4M3 codes stored in the cache decode as the OCP definition says (both paths)."""
    wl = small(60, lengths=(2,), capacity=2, cache_dtype="fp8", n_layers=1)
    model = Model(wl)
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    H, Dh = wl.n_heads, wl.head_dim
    block = np.resize(codes, (2, H, Dh))
    host_tok, tok = tokens_for(wl)
    results = []
    for flags in (0, fsx.FLAG_GENERIC):
        ex = model.create(flags=flags)
        cache = Cache(wl)
        for kind, t in (("k", cache.k), ("v", cache.v)):
            rows = block if kind == "v" else np.flip(block, 0)
            t[0, 0].copy_(torch.from_numpy(np.ascontiguousarray(rows.transpose(1, 0, 2))))  # [H][rows][Dh]
        cache.k_scale.fill_(1.0 / 64)
        cache.v_scale.fill_(1.0 / 32)
        torch.cuda.synchronize()
        wp, _ = run_forward(ex, cache, tok, 1, 0)
        results.append(wp[0])
    dec = oracle.e4m3fn_decode(block)
    kv = (np.flip(dec, 0) / 64.0, dec / 32.0)
    ref, _ = model.oracle_agent(host_tok[0], lambda l: kv, 2)
    for wp in results:
        assert rel_err(wp, ref) <= BF16_WP_TOL, rel_err(wp, ref)


def test_small_fp8_cache_matches_oracle():
    wl = small(61, lengths=(300, 45, 0), capacity=320, cache_dtype="fp8")
    say("case small fp8")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl, starts=(100, 310, 0))
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), FP8_WP_TOL, what="waypoints vs bf16 source, max|d| / max|ref|")
        record(b, rel_err(wp[b], refd), BF16_WP_TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")


# Equal lengths on power-of-two rings: with 16 heads (2 per XCD) and 4 agents every (agent, head) attention unit
# takes its whole range and streams from tile (5h + 3b) mod n of its n tiles, wrapping around; 100 rows make four
# tiles, the last one partial, and the rings wrap at different rows.  30 frame tokens: the many-query unit.
@pytest.mark.parametrize("cache_dtype,n_frame", [("bf16", 0), ("fp8", 0), ("bf16", 30), ("fp8", 30)])
def test_whole_range_units_on_power_of_two_rings_match_oracle(cache_dtype, n_frame):
    wl = synth.Workload(name="whole", wid=64, n_layers=2, d_model=256, n_heads=16, head_dim=128, d_ffn=512,
                        n_expert_tokens=10, n_frame_tokens=n_frame, batch=4, lengths=(100,) * 4, dtype="bf16",
                        cache_dtype=cache_dtype, capacity=128)
    say(f"case whole-range units, {cache_dtype}, {n_frame} frame tokens, capacity 128")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl, starts=(120, 64, 0, 127))
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, n_frame)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        if cache_dtype == "fp8":
            refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
            record(b, rel_err(wp[b], ref), FP8_WP_TOL, what="waypoints vs bf16 source, max|d| / max|ref|")
            record(b, rel_err(wp[b], refd), BF16_WP_TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")
        else:
            record(b, rel_err(wp[b], ref), BF16_WP_TOL)
    ex.close()


# Stress keys (outlier channels, keys growing along the sequence, a sink row two thirds in; synth.stress_keys): the
# scores reach ~15 in log2 units, so queries' running maxima jump by more than 2^8 after their first tiles and the
# accumulators are rescaled in the middle of a range.  fp8: compared with the decoded codes (the outliers make the
# per-head scale coarse for the other rows, an input property rather than a kernel error).
@pytest.mark.parametrize("cache_dtype,n_frame", [("bf16", 0), ("fp8", 0), ("bf16", 30), ("fp8", 30)])
def test_stress_keys_rescale_within_a_range_match_oracle(cache_dtype, n_frame):
    wl = small(66, lengths=(700, 333, 90), capacity=720, cache_dtype=cache_dtype).replace(
        n_frame_tokens=n_frame, stress_keys=True)
    say(f"case stress keys, {cache_dtype}, {n_frame} frame tokens")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl, starts=(15, 700, 0))
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, n_frame)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), BF16_WP_TOL,
               what="waypoints vs decoded fp8, max|d| / max|ref|" if cache_dtype == "fp8" else "waypoints, max|d| / max|ref|")
    ex.close()


# 30, 64, 90 frame tokens: 3, 5 and 7 query tiles per agent (key-split jobs only; four whole jobs and one
# key-split; two passes over the cache)
@pytest.mark.parametrize("n_frame", [30, 64, 90])
def test_small_fp8_cache_with_frame_tokens_matches_oracle(n_frame):
    """fp8 cache rows with several query tiles per agent (10 expert + n_frame frame tokens)."""
    wl = small(62, lengths=(290, 64), capacity=300, cache_dtype="fp8").replace(n_frame_tokens=n_frame)
    say(f"case small fp8 with {n_frame} frame tokens")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl, starts=(250, 7))
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, wl.n_frame_tokens)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), FP8_WP_TOL, what="waypoints vs bf16 source, max|d| / max|ref|")
        record(b, rel_err(wp[b], refd), BF16_WP_TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")


def test_fp8_many_query_slices_across_agents_match_oracle():
    """fp8 cache, 5 query tiles per agent (64 frame tokens) and enough rows that slices cut the segments of several
    agents: key-split jobs, whole jobs and partial states merged per query tile, with the fp8 output layout."""
    wl = synth.Workload(name="small_fp8_mq", wid=64, n_layers=2, d_model=128, n_heads=16, head_dim=128, d_ffn=256,
                        n_expert_tokens=10, n_frame_tokens=64, batch=3, lengths=(3000, 2600, 3100), dtype="bf16",
                        cache_dtype="fp8", capacity=3200)
    say("case fp8 many-query slices")
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl, starts=(3100, 5, 700))
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, wl.n_frame_tokens)
    for b in range(wl.batch):
        ref, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b), cache.desc.pos[b])
        refd, _ = model.oracle_agent(host_tok[b], cache.oracle_rows(b, decoded=True), cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), FP8_WP_TOL, what="waypoints vs bf16 source, max|d| / max|ref|")
        record(b, rel_err(wp[b], refd), BF16_WP_TOL, what="waypoints vs decoded fp8, max|d| / max|ref|")


@pytest.mark.slow
def test_ragged_fp8_agents_match_oracle():
    """8 agents with ragged histories (256..16384 rows) in an fp8 cache; every agent vs the oracle (the longest
    agents run the deepest split-K schedules)."""
    wl = synth.WORKLOADS["ragged_fp8_B8"]
    say("case ragged_fp8_B8", wl.lengths)
    model = Model(wl)
    ex = model.create()
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    wp, _ = run_forward(ex, cache, tok, wl.batch, 0)
    assert np.isfinite(wp).all()
    pos = [int(p) for p in cache.desc.pos]
    refs = oracle_agents(model, range(wl.batch),
                         lambda b: model.oracle_agent(host_tok[b], cache.oracle_rows(b), pos[b])[0], workers=8)
    for b in range(wl.batch):
        record(b, rel_err(wp[b], refs[b]), FP8_WP_TOL, what="waypoints vs bf16 source, max|d| / max|ref|",
               extra={"L": wl.lengths[b]})
