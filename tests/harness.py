"""Test harness: the GPU plumbing of ``gpu_inputs`` plus the fp64 oracle on the same seeded inputs.

The GPU side receives the generator's arrays converted to torch device tensors;
the oracle receives the same arrays upcast to float64.  Nothing flows from the
GPU result into the oracle.
"""

from __future__ import annotations

import json
import os
import tempfile
import threading

import numpy as np

import oracle
import synth
from gpu_inputs import Cache as _Cache
from gpu_inputs import Model as _Model
from gpu_inputs import head_major_rows, rel_err, run_forward, tokens_for  # noqa: F401


def shape_of(wl: synth.Workload) -> oracle.ExpertShape:
    return oracle.ExpertShape(n_layers=wl.n_layers, d_model=wl.d_model, n_heads=wl.n_heads, head_dim=wl.head_dim,
                              d_ffn=wl.d_ffn, n_expert_tokens=wl.n_expert_tokens, n_out=wl.n_out,
                              rope_base=wl.rope_base, rms_eps=wl.rms_eps, head_kind=wl.head_kind,
                              head_hidden=wl.head_hidden)


class Model(_Model):
    def oracle_agent(self, tokens_b, cache_rows, pos):
        """fp64 oracle for one agent: cache_rows(l) -> (K, V) float arrays [L][H][Dh]."""
        return oracle.expert_forward(shape_of(self.wl), self.layers, self.final_norm, self.head_w, tokens_b,
                                     cache_rows, pos)


class Cache(_Cache):
    def oracle_rows(self, b, decoded=False):
        """cache_rows(l) for the oracle: the generator's source values (or the fp8 decode if decoded)."""
        wl = self.wl

        def rows(l):
            out = []
            for kind in ("k", "v"):
                src = synth.cache_slab(wl, b, l, kind, rows=self.lengths[b]).astype(np.float64)
                if decoded and wl.cache_dtype == "fp8":
                    codes, scale = synth.fp8_encode(src.astype(np.float32))
                    src = oracle.e4m3fn_decode(codes) * scale.astype(np.float64)[None, :, None]
                out.append(src)
            return out[0], out[1]

        return rows


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the parity log (one JSON line per comparison; profiles/parity_errors.md is made from it): FSX_PARITY_LOG, else a
# file in the system's temporary directory
ERR_LOG = os.environ.get("FSX_PARITY_LOG") or os.path.join(tempfile.gettempdir(), "fsx_parity_errors.jsonl")
_log_lock = threading.Lock()


def record(agent, err, tol, what="waypoints, max|d| / max|ref|", extra=None):
    """Print the observed error of one comparison and append it to the parity log (one JSON line per check), then
    assert it is within tol."""
    case = os.environ.get("PYTEST_CURRENT_TEST", "?").rsplit(" ", 1)[0]
    line = {"case": case, "agent": agent, "what": what, "err": float(err), "tol": float(tol),
            "ok": bool(err <= tol)}
    if extra:
        line.update(extra)
    print(f"  {case} agent {agent} {what}: {err:.3e} (tol {tol})", flush=True)
    try:
        with _log_lock:
            os.makedirs(os.path.dirname(ERR_LOG), exist_ok=True)
            with open(ERR_LOG, "a") as f:
                f.write(json.dumps(line) + "\n")
    except OSError:
        pass
    assert err <= tol, line


def oracle_agents(model, agents, job, workers=None):
    """Run job(b) -> oracle result for several agents on a thread pool (NumPy's generators and BLAS release the
    GIL), BLAS limited to one thread per worker; returns {b: result}."""
    from threadpoolctl import threadpool_limits

    agents = list(agents)
    with threadpool_limits(1):
        res = synth.parallel_map(job, agents, workers)
    return dict(zip(agents, res))
