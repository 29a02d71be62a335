"""The backbone's incremental forward on the GPU (Sec. 3.3): the slow system's producer of the appended rows.

* The rows the call writes into the ring (rotated keys, values), and the hidden states of every layer, match the
  oracle's incremental forward over the rows the ring held; the other rows keep their bytes; the ring state advances.
* The paper's golden test on the GPU: 8 tokens appended at once from an empty ring and the same tokens appended as
  4 + 4 give the same rows (within the bf16 tolerance) -- rotary phases make append-only caching exact.
* An fp8 cache receives the rows encoded with its scales.
* Full LLaMA-7B widths (d 4096, 32 heads x 128, SwiGLU 11008) on two layers.
* The expert's tick over a cache the backbone extended matches the oracle over the same rows.
"""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from harness import Cache, Model, record, rel_err, run_forward, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bb_workload(wid, lengths, n_new, capacity, d=512, H=4, F=1024, n_layers=2, cache_dtype="bf16"):
    return synth.Workload(name=f"bb{wid}", wid=wid, n_layers=n_layers, d_model=d, n_heads=H, head_dim=128, d_ffn=F,
                          n_expert_tokens=n_new, n_frame_tokens=0, batch=len(lengths), lengths=tuple(lengths),
                          dtype="bf16", cache_dtype=cache_dtype, capacity=capacity)


class BB:
    """The backbone's weights (synthetic, seeded) on the host and in the library."""

    def __init__(self, wl):
        self.wl = wl
        self.layers, _, _ = synth.make_weights(wl)
        dev = [{k: torch.from_numpy(v).to("cuda", torch.float32 if k in ("attn_norm", "ffn_norm") else torch.bfloat16)
                for k, v in lw.items()} for lw in self.layers]
        cfg = fsx.BackboneCfg(wl.n_layers, wl.d_model, wl.n_heads, wl.head_dim, wl.d_ffn, wl.n_expert_tokens,
                              wl.batch, fsx.BF16, wl.rope_base, wl.rms_eps)
        self.bb = fsx.Backbone(cfg, dev)
        torch.cuda.synchronize()
        del dev
        self.shape = oracle.BackboneShape(n_layers=wl.n_layers, d_model=wl.d_model, n_heads=wl.n_heads,
                                          head_dim=wl.head_dim, d_ffn=wl.d_ffn, rope_base=wl.rope_base,
                                          rms_eps=wl.rms_eps)

    def oracle(self, tokens_b, cache_rows, pos):
        return oracle.backbone_incremental_forward(self.shape, self.layers, tokens_b, cache_rows, pos)


def appended(cache, b, first, n):
    """Device rows [layers][n][H][Dh] of agent b at slots first .. first+n-1 (mod capacity), as float."""
    wl = cache.wl
    slots = [(first + j) % cache.capacity for j in range(n)]
    out = []
    for kind in ("k", "v"):
        out.append(np.stack([cache.slot_rows(b, l, kind, slots).float().cpu().numpy() for l in range(wl.n_layers)]))
    return out


@pytest.mark.parametrize("layout", [fsx.CACHE_HEAD_MAJOR, fsx.CACHE_TOKEN_MAJOR])
def test_backbone_append_matches_oracle(layout):
    wl = bb_workload(700, lengths=(37, 0, 200), n_new=4, capacity=256)
    say(f"case backbone append layout {layout}")
    bb = BB(wl)
    cache = Cache(wl, starts=(250, 0, 9), layout=layout)
    before_k = cache.k.clone()
    host_tok, tok = tokens_for(wl)
    first = [int((cache.desc.start[b] + cache.desc.len[b]) % wl.capacity) for b in range(wl.batch)]
    pos0 = [int(p) for p in cache.desc.pos]
    hid = torch.full((wl.n_layers, wl.batch, 4, wl.d_model), float("nan"), device="cuda")
    bb.bb.append(cache.desc, tok, wl.batch, 4, hid)
    torch.cuda.synchronize()
    assert list(cache.desc.len) == [41, 4, 204] and list(cache.desc.pos) == [p + 4 for p in pos0]
    hid = hid.cpu().numpy()
    for b in range(wl.batch):
        k_ref, v_ref, h_ref = bb.oracle(host_tok[b], cache.oracle_rows(b), pos0[b])
        k_got, v_got = appended(cache, b, first[b], 4)
        record(b, rel_err(k_got, k_ref), TOL, what="appended keys (rotated), max|d| / max|ref|")
        record(b, rel_err(v_got, v_ref), TOL, what="appended values, max|d| / max|ref|")
        record(b, max(rel_err(hid[l, b], h_ref[l]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    # rows outside the appended slots keep their bytes
    mask = torch.ones_like(cache.k, dtype=torch.bool)
    for b in range(wl.batch):
        for j in range(4):
            slot = (first[b] + j) % wl.capacity
            if layout == fsx.CACHE_TOKEN_MAJOR:
                mask[b, :, slot] = False
            else:
                mask[b, :, :, slot] = False
    assert torch.equal(cache.k[mask].view(torch.int16), before_k[mask].view(torch.int16))
    bb.bb.close()


def test_backbone_golden_monolithic_vs_incremental_prefill():
    wl8 = bb_workload(710, lengths=(0,), n_new=8, capacity=64)
    say("case backbone golden test")
    bb = BB(wl8)
    host_tok, tok = tokens_for(wl8)
    mono = Cache(wl8)
    bb.bb.append(mono.desc, tok, 1, 8)
    inc = Cache(wl8)
    t4a = tok[:, :4].contiguous()
    t4b = tok[:, 4:].contiguous()
    bb.bb.append(inc.desc, t4a, 1, 4)
    bb.bb.append(inc.desc, t4b, 1, 4)
    torch.cuda.synchronize()
    assert list(mono.desc.len) == list(inc.desc.len) == [8] and list(inc.desc.pos) == [8]
    km, vm = appended(mono, 0, 0, 8)
    ki, vi = appended(inc, 0, 0, 8)
    record(0, rel_err(ki, km), TOL, what="keys incremental vs monolithic, max|d| / max|ref|")
    record(0, rel_err(vi, vm), TOL, what="values incremental vs monolithic, max|d| / max|ref|")
    k_ref, v_ref, _ = bb.oracle(host_tok[0], lambda l: (np.zeros((0, 4, 128)),) * 2, 0)
    record(0, rel_err(ki, k_ref), TOL, what="keys incremental vs oracle, max|d| / max|ref|")
    bb.bb.close()


def test_backbone_append_into_fp8_cache():
    wl = bb_workload(720, lengths=(60,), n_new=4, capacity=80, cache_dtype="fp8")
    bb = BB(wl)
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    bb.bb.append(cache.desc, tok, 1, 4)
    torch.cuda.synchronize()
    rows = cache.oracle_rows(0, decoded=True)
    k_ref, v_ref, _ = bb.oracle(host_tok[0], rows, 60)
    codes = [np.stack([cache.slot_rows(0, l, kind, list(range(60, 64))).contiguous().cpu().numpy()
                       for l in range(wl.n_layers)]) for kind in ("k", "v")]
    for kind, ref, sc, cd in (("k", k_ref, cache.k_scale, codes[0]), ("v", v_ref, cache.v_scale, codes[1])):
        s = sc[0].cpu().numpy()  # [layers][H]
        dec = oracle.e4m3fn_decode(cd) * s[:, None, :, None]
        record(0, rel_err(dec, ref), 6e-2, what=f"appended {kind} (fp8 decoded), max|d| / max|ref|")
    bb.bb.close()


@pytest.mark.slow
def test_backbone_full_llama_widths():
    wl = bb_workload(730, lengths=(224,), n_new=4, capacity=256, d=4096, H=32, F=11008, n_layers=2)
    say("case backbone at LLaMA-7B widths, 2 layers")
    bb = BB(wl)
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    hid = torch.full((wl.n_layers, 1, 4, wl.d_model), float("nan"), device="cuda")
    bb.bb.append(cache.desc, tok, 1, 4, hid)
    torch.cuda.synchronize()
    k_ref, v_ref, h_ref = bb.oracle(host_tok[0], cache.oracle_rows(0), 224)
    k_got, v_got = appended(cache, 0, 224, 4)
    record(0, rel_err(k_got, k_ref), TOL, what="appended keys, max|d| / max|ref|")
    record(0, rel_err(v_got, v_ref), TOL, what="appended values, max|d| / max|ref|")
    hid = hid.cpu().numpy()
    record(0, max(rel_err(hid[l, 0], h_ref[l]) for l in range(wl.n_layers)), TOL,
           what="worst layer hidden, max|d| / max|ref|")
    bb.bb.close()


@pytest.mark.slow
@pytest.mark.parametrize("batch", [8, 16])
def test_backbone_batched_llama_widths(batch):
    # 32 or 64 new rows at LLaMA-7B widths: the projections take the several-column-tiles-per-workgroup kernel
    lengths = tuple(40 + 17 * b for b in range(batch))
    wl = bb_workload(760 + batch, lengths=lengths, n_new=4, capacity=320, d=4096, H=32, F=11008, n_layers=2)
    say(f"case backbone at LLaMA-7B widths, {batch} agents, 2 layers")
    bb = BB(wl)
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    first = [int((cache.desc.start[b] + cache.desc.len[b]) % wl.capacity) for b in range(wl.batch)]
    pos0 = [int(p) for p in cache.desc.pos]
    hid = torch.full((wl.n_layers, wl.batch, 4, wl.d_model), float("nan"), device="cuda")
    bb.bb.append(cache.desc, tok, wl.batch, 4, hid)
    torch.cuda.synchronize()
    hid = hid.cpu().numpy()
    got = [appended(cache, b, first[b], 4) for b in range(wl.batch)]
    refs = synth.parallel_map(lambda b: bb.oracle(host_tok[b], cache.oracle_rows(b), pos0[b]), list(range(wl.batch)))
    for b, (k_ref, v_ref, h_ref) in enumerate(refs):
        record(b, rel_err(got[b][0], k_ref), TOL, what="appended keys (rotated), max|d| / max|ref|")
        record(b, rel_err(got[b][1], v_ref), TOL, what="appended values, max|d| / max|ref|")
        record(b, max(rel_err(hid[l, b], h_ref[l]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    bb.bb.close()


def test_expert_tick_over_rows_the_backbone_appended():
    # producer -> consumer: the backbone extends the cache, then the expert reads it
    wl = bb_workload(740, lengths=(100, 64), n_new=4, capacity=128, d=512, H=16, F=1024)
    ewl = synth.Workload(name="bb_expert", wid=741, n_layers=2, d_model=256, n_heads=16, head_dim=128, d_ffn=512,
                         n_expert_tokens=10, n_frame_tokens=0, batch=2, lengths=(100, 64), dtype="bf16",
                         cache_dtype="bf16", capacity=128)
    bb = BB(wl)
    cache = Cache(wl)
    host_tok, tok = tokens_for(wl)
    pos0 = [int(p) for p in cache.desc.pos]
    bb.bb.append(cache.desc, tok, 2, 4)
    model = Model(ewl)
    ex = model.create()
    e_host, e_tok = tokens_for(ewl)
    wp, _ = run_forward(ex, cache, e_tok, 2, 0)
    for b in range(2):
        k_new, v_new, _ = bb.oracle(host_tok[b], cache.oracle_rows(b), pos0[b])
        base_k, base_v = (synth.cache_slab(wl, b, 0, kd, rows=wl.lengths[b]) for kd in ("k", "v"))

        def rows(l, b=b, k_new=k_new, v_new=v_new):
            return (np.concatenate([synth.cache_slab(wl, b, l, "k", rows=wl.lengths[b]).astype(np.float64), k_new[l]]),
                    np.concatenate([synth.cache_slab(wl, b, l, "v", rows=wl.lengths[b]).astype(np.float64), v_new[l]]))
        ref, _ = model.oracle_agent(e_host[b], rows, cache.desc.pos[b])
        record(b, rel_err(wp[b], ref), TOL, what="expert waypoints after the backbone's append, max|d| / max|ref|")
    ex.close()
    bb.bb.close()
