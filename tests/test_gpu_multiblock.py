"""GPU form of the staleness-augmented training forward (Sec. 3.2): every frame's expert block of a training clip in
one call, block j seeing the clip's backbone prefix only up to frame j - delta.  The blocks run as a batch of agents
over ONE shared cache (FSX_CACHE_SHARED): agent j's ring state is (start 0, len = visible rows of block j).  The
reference is the oracle's clip-level forward with one masked attention over the whole clip per layer."""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from harness import Cache, Model, record, rel_err, tokens_for
from paper_2607_15621_amd import fsx

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("layout", [fsx.CACHE_HEAD_MAJOR, fsx.CACHE_TOKEN_MAJOR])
@pytest.mark.parametrize("delta,rope,n_layers,d_model,n_heads", [(2, 0.0, 2, 256, 16), (0, 10000.0, 2, 256, 16),
                                                                 (2, 0.0, 3, 512, 32)])
def test_clip_blocks_over_shared_cache_match_masked_oracle(layout, delta, rope, n_layers, d_model, n_heads):
    n_text, per, J = 64, 4, 12
    L = n_text + per * J
    vis = oracle.staleness_visible_rows(n_text, per, J, delta)
    wl = synth.Workload(name="clip", wid=400 + delta + n_heads, n_layers=n_layers, d_model=d_model, n_heads=n_heads,
                        head_dim=128, d_ffn=2 * d_model, n_expert_tokens=10, n_frame_tokens=0, batch=J,
                        lengths=(L,) * J, dtype="bf16", cache_dtype="bf16", capacity=L, rope_base=rope)
    say(f"case clip J={J} delta={delta} rope={rope} layout={layout} heads={n_heads}")
    model = Model(wl)
    one = Cache(wl.replace(batch=1, lengths=(L,)), layout=layout)  # the clip's prefix: one agent's rings
    desc = fsx.CacheDesc(one.k, one.v, fsx.BF16, wl.n_layers, wl.n_heads, wl.head_dim, L, vis, positions=vis,
                         layout=layout | fsx.CACHE_SHARED)
    host_tok, tok = tokens_for(wl)
    ex = model.create()
    wp = torch.full((J, wl.n_out), float("nan"), device="cuda")
    hid = torch.full((wl.n_layers, J, wl.seq, wl.d_model), float("nan"), device="cuda")
    fsx.expert_forward(ex, desc, tok, J, 0, wp, hid)
    torch.cuda.synchronize()
    wp, hid = wp.cpu().numpy(), hid.cpu().numpy()
    rows = one.oracle_rows(0)
    ref, ref_hid = oracle.masked_multiblock_forward(
        oracle.ExpertShape(n_layers=wl.n_layers, d_model=wl.d_model, n_heads=wl.n_heads, head_dim=wl.head_dim,
                           d_ffn=wl.d_ffn, rope_base=rope), model.layers, model.final_norm, model.head_w, host_tok,
        rows, vis, vis)
    for j in range(J):
        record(j, rel_err(wp[j], ref[j]), TOL, extra={"L": int(vis[j])})
        record(j, max(rel_err(hid[l, j], ref_hid[l, j]) for l in range(wl.n_layers)), TOL,
               what="worst layer hidden, max|d| / max|ref|")
    ex.close()


def test_shared_cache_refuses_append():
    wl = synth.Workload(name="clip_app", wid=420, n_layers=1, d_model=128, n_heads=4, head_dim=128, d_ffn=256,
                        n_expert_tokens=10, n_frame_tokens=0, batch=1, lengths=(8,), dtype="bf16", cache_dtype="bf16",
                        capacity=16)
    one = Cache(wl)
    desc = fsx.CacheDesc(one.k, one.v, fsx.BF16, 1, 4, 128, 16, [8, 4], layout=fsx.CACHE_SHARED)
    rows = torch.zeros((2, 1, 4, 4, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(fsx.FsxError) as e:
        fsx.cache_append_rows(desc, rows, rows, 4)
    assert e.value.code == 2
