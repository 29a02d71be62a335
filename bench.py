"""Benchmark of the expert tick on one MI355X (ticks/s, µs/tick, fraction of the HBM roofline).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME[,NAME...]] [--no-cpu-baseline]

By default every full-size workload is timed in one run: the 40-frame single agent (the headline line), the
4096-row history with 64 frame tokens, 16 batched agents with their 4-row append, and 8 ragged agents on an fp8
cache; the one JSON line carries the headline workload's fields plus a `workloads` object with each workload's
µs/tick, ticks/s, roofline fraction, HBM traffic and a variant with the 256 MB Infinity Cache flushed before every
tick, an `append` object, the backbone's incremental forward that produces the appended rows at LLaMA-7B shapes
(`backbone_append`) and the device's measured HBM read ceiling (`hbm_read_ceiling`).

Measurement helpers (used by the commands recorded in profiles/):
    python bench.py --copy-calibration BYTES      plain device copies of BYTES (counter calibration)
    python bench.py --summarize-trace DIR --workload NAME --bench-line FILE
        writes profiles/tick_kernel_<NAME>.md from a rocprofv3 --kernel-trace --stats output directory
    python bench.py --summarize-traffic FETCH_DIR WRITE_DIR CFETCH_DIR CWRITE_DIR --workload NAME --copy-bytes B
        writes profiles/traffic_<NAME>.json/.md from four rocprofv3 --pmc output directories (FETCH_SIZE and
        WRITE_SIZE of the tick, then of the calibration copy)

Headline workload: the full-size expert (32 layers, width 512, 32 heads x 128, SwiGLU 2048) on one agent
with a 224-row cache per layer (a 40-frame history at 4 rows per frame plus 64 instruction rows), bf16.
Inputs are seeded synthetic arrays, resident in HBM before the timed region: weights and tokens from the
seeded generators of `synth`, cache rows drawn on the GPU from a seeded torch generator with the same
distributions (N(0, 1), bf16; the fp8 cache encoded per (agent, layer, K/V, head) with scale amax / 448).
Prints ONE JSON line.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
PAPER_EXPERT_MS = 7.5  # paper, Table 3: action expert per tick at a 40-frame history (RTX 3090 Ti)
METRIC = "expert µs/tick and ticks/s at L=224/4096/B=16; achieved HBM GB/s vs peak"
HEADLINE = "single_bf16_L224"
ALL_WORKLOADS = ("single_bf16_L224", "long_bf16_L4096_F64", "batched_bf16_B16_L1024", "ragged_fp8_B8")


def algorithmic_bytes(wl, weight_bytes: int) -> int:
    """Bytes one tick must read: packed weight matrices + the valid cache rows (K and V)."""
    es = {"bf16": 2, "fp8": 1, "f32": 4}[wl.cache_dtype]
    return int(weight_bytes) + sum(wl.lengths) * 2 * wl.n_layers * wl.attn_width * es


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_15621_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, key: str = "bytes_per_launch"):
    """HBM bytes per launch from rocprofv3 counters (FETCH_SIZE + WRITE_SIZE, or with key "dram_bytes_per_launch"
    the EA read/write requests destined for DRAM), if they were taken on these sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except Exception:
        return None
    if d.get("source_hash") != source_hash():
        return None
    return d.get(key)


def cpu_baseline(wl, budget_s: float = 15.0):
    """The fp64 oracle on the host cores: as many full single-agent ticks as fit in ~budget_s."""
    cores = len(os.sched_getaffinity(0))
    for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ.setdefault(v, str(cores))
    from harness import Model  # noqa: E402  (oracle is imported only on this leg)
    import synth  # noqa: E402

    one = wl.replace(batch=1, lengths=wl.lengths[:1])
    model = Model(one)
    tokens = synth.make_tokens(one)
    slabs = {}
    for l in range(one.n_layers):
        slabs[l] = (synth.cache_slab(one, 0, l, "k").astype("float64"), synth.cache_slab(one, 0, l, "v").astype("float64"))
    n, t0 = 0, time.perf_counter()
    while True:
        model.oracle_agent(tokens[0], lambda l: slabs[l], one.lengths[0])
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or (n >= 1 and el * (n + 1) / n > 2 * budget_s):
            break
    return {"value": round(n / el, 4), "unit": "ticks/s", "cores": cores, "kind": "oracle",
            "sample": f"{n} full fp64 oracle tick(s) of one agent ({one.n_layers} layers, L={one.lengths[0]}, "
                      f"S={one.seq}) in {el:.1f} s"}


def _csv_rows(d: str, suffix: str):
    import csv
    import glob
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    return list(csv.DictReader(open(files[0])))


def copy_calibration(nbytes: int, reps: int = 5):
    """Plain device-to-device copies of nbytes (the kernel whose byte counters calibrate FETCH_SIZE/WRITE_SIZE)."""
    import torch

    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


def summarize_trace(d: str, workload: str, bench_line: str, command: str, name: str = ""):
    """profiles/tick_kernel_<workload>.md (or profiles/<name>.md) from a rocprofv3 --kernel-trace --stats
    directory."""
    rows = _csv_rows(d, "kernel_stats.csv")
    line = json.loads(open(bench_line).read().strip().splitlines()[-1])
    title = f"tick kernel, workload `{workload}`" if not name else f"`{name}` (bench.py run of workload `{workload}`)"
    out = [f"# Kernel trace: {title}", "", "Command (from the repository root, on one MI355X):",
           "", "```", command, "```", "", "| kernel | calls | total ms | avg µs | min µs | max µs |",
           "|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        out.append(f"| `{r['Name'][:70]}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.3f} | "
                   f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    out += ["", f"bench.py line of the same run: {line['us_per_tick']} µs/tick (HIP events over {line['steps']} "
                f"back-to-back ticks), {line['value']} agent-ticks/s, algorithmic bytes "
                f"{line['roofline']['algorithmic_bytes_per_launch']:,} per launch, achieved "
                f"{line['roofline']['achieved']} GB/s = {line['roofline']['frac']} of 8000 GB/s.", ""]
    if line.get("backbone_append"):
        out += [f"Backbone incremental forward of the same run: {json.dumps(line['backbone_append'])}", ""]
    path = os.path.join(ROOT, "profiles", f"{name}.md" if name else f"tick_kernel_{workload}.md")
    open(path, "w").write("\n".join(out))
    print(path)


def summarize_traffic(dirs, workload: str, copy_bytes: int, commands, dram: bool = False):
    """profiles/traffic_<workload>.json: HBM bytes per tick-kernel launch from two counters, each scaled by what the
    same counter reads for a plain device copy of copy_bytes.  Default: FETCH_SIZE / WRITE_SIZE (L2 <-> fabric
    traffic, Infinity Cache hits included); with dram: TCC_EA0_RDREQ_DRAM_sum / TCC_EA0_WRREQ_DRAM_sum (requests
    the L2 sends towards DRAM).  dirs: read counter of the tick, write counter of the tick, then the same two for
    the copy.  Both sets live in the same file; each is kept only while the kernel sources match."""
    def mean_counter(d, counter, pick):
        vals = [float(r["Counter_Value"]) for r in _csv_rows(d, "counter_collection.csv")
                if r["Counter_Name"] == counter and pick(r["Kernel_Name"])]
        if not vals:
            raise SystemExit(f"no {counter} rows in {d}")
        return vals

    rd, wr = ("TCC_EA0_RDREQ_DRAM_sum", "TCC_EA0_WRREQ_DRAM_sum") if dram else ("FETCH_SIZE", "WRITE_SIZE")
    tick = lambda n: "k_tick" in n
    copyk = lambda n: "copy" in n.lower() or "elementwise" in n.lower()
    f_tick = mean_counter(dirs[0], rd, tick)
    w_tick = mean_counter(dirs[1], wr, tick)
    f_copy = max(mean_counter(dirs[2], rd, copyk))
    w_copy = max(mean_counter(dirs[3], wr, copyk))
    kf, kw = copy_bytes / f_copy, copy_bytes / w_copy  # bytes per counter unit
    fetch = sum(f_tick) / len(f_tick) * kf
    write = sum(w_tick) / len(w_tick) * kw
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    d = {}
    if os.path.exists(path):
        d = json.load(open(path))
        if d.get("source_hash") != source_hash():
            d = {}
    d.update({"workload": workload, "source_hash": source_hash()})
    pre = "dram_" if dram else ""
    d.update({f"{pre}read_bytes_per_launch" if dram else "fetch_bytes_per_launch": int(fetch),
              f"{pre}write_bytes_per_launch": int(write), f"{pre}bytes_per_launch": int(fetch + write),
              f"{pre}calibration": {"copy_bytes": copy_bytes, "read_counter": rd, "write_counter": wr,
                                    "copy_read_count": f_copy, "copy_write_count": w_copy,
                                    "bytes_per_read_unit": kf, "bytes_per_write_unit": kw},
              f"{pre}dispatches": {"read": len(f_tick), "write": len(w_tick)}, f"{pre}commands": commands})
    json.dump(d, open(path, "w"), indent=1)
    print(path, json.dumps({k: v for k, v in d.items() if k.endswith("bytes_per_launch")}))


INSTR_COUNTERS = ("SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_INSTS_SALU", "SQ_INSTS_VMEM",
                  "SQ_LDS_BANK_CONFLICT", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES")


def summarize_counters(dirs, workloads, commands):
    """profiles/instructions_tick.md: instruction counts of one tick-kernel launch per workload (wave-level
    instructions summed over the device), LDS bank-conflict cycles and the MFMA busy fraction, from rocprofv3 --pmc
    runs (dirs: for each workload in turn, one directory per pass)."""
    per = len(dirs) // len(workloads)
    out = ["# Instruction mix of the tick kernel", "",
           "One tick-kernel launch per workload, counters summed over the device and averaged over the profiled "
           "launches: wave-level instructions by kind, LDS bank-conflict cycles, and the busy cycles of the MFMA "
           "units against those of the shader sequencers (SQ_VALU_MFMA_BUSY_CYCLES / SQ_BUSY_CYCLES; the counters "
           "count in different units per block, so the ratio compares launches, not an absolute utilisation).", "",
           "Commands (from the repository root, on one MI355X, one pass each):", "", "```"] + list(commands) + \
          ["```", "", "| workload | " + " | ".join(c.replace("SQ_", "") for c in INSTR_COUNTERS) + " |",
           "|---|" + "---:|" * len(INSTR_COUNTERS)]
    for i, w in enumerate(workloads):
        vals = {}
        for d in dirs[i * per:(i + 1) * per]:
            for r in _csv_rows(d, "counter_collection.csv"):
                if "k_tick" in r["Kernel_Name"]:
                    vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
        cells = [f"{sum(vals[c]) / len(vals[c]):,.0f}" if c in vals else "–" for c in INSTR_COUNTERS]
        out.append(f"| `{w}` | " + " | ".join(cells) + " |")
    path = os.path.join(ROOT, "profiles", "instructions_tick.md")
    open(path, "w").write("\n".join(out) + "\n")
    print(path)


def summarize_parity(log: str, command: str):
    """profiles/parity_errors.md from the JSON lines the GPU parity tests append (one per comparison): per test, the
    number of comparisons and the worst error against its tolerance; then every comparison of the full-size
    workloads."""
    rows = [json.loads(l) for l in open(log) if l.strip()]
    by = {}
    for r in rows:
        by.setdefault(r["case"], []).append(r)
    out = ["# GPU parity against the fp64 oracle: observed errors", "",
           "Every comparison of a GPU result with the oracle (or with a second GPU path) appends one line to the log",
           "this summary is made from. Command (from the repository root, on one MI355X):", "", "```", command, "```", "",
           f"{len(rows)} comparisons in {len(by)} tests, all within tolerance: "
           f"{all(r['ok'] for r in rows)}.", "",
           "| test | comparisons | worst error | tolerance | measure |", "|---|---|---|---|---|"]
    for case, v in by.items():
        w = max(v, key=lambda r: r["err"] / r["tol"] if r["tol"] > 0 else (0.0 if r["err"] == 0 else float("inf")))
        out.append(f"| `{case.split('::', 1)[-1]}` | {len(v)} | {w['err']:.2e} | {w['tol']:g} | {w['what'].replace('|', chr(92) + '|')} |")
    full = [r for r in rows if any(k in r["case"] for k in ("batched", "ragged", "full_", "maximum_batch"))]
    out += ["", "Every comparison of the full-size workloads (and of the 64-agent case):", "",
            "| test | agent | cache rows | error | tolerance | measure |", "|---|---|---|---|---|---|"]
    for r in full:
        out.append(f"| `{r['case'].split('::', 1)[-1]}` | {r['agent']} | {r.get('L', '')} | {r['err']:.2e} | "
                   f"{r['tol']:g} | {r['what'].replace('|', chr(92) + '|')} |")
    path = os.path.join(ROOT, "profiles", "parity_errors.md")
    open(path, "w").write("\n".join(out) + "\n")
    print(path)


def gpu_cache(wl, seed: int):
    """A head-major device cache of the workload's lengths, rows drawn on the GPU (seeded torch generator): bf16
    N(0, 1), or fp8 codes of such rows with one scale amax / 448 per (agent, layer, K/V, head)."""
    import torch

    from paper_2607_15621_amd import fsx

    B, nl, H, Dh, cap = wl.batch, wl.n_layers, wl.n_heads, wl.head_dim, wl.capacity
    fp8 = wl.cache_dtype == "fp8"
    shape = (B, nl, H, cap, Dh)
    dt = torch.uint8 if fp8 else torch.bfloat16
    k = torch.zeros(shape, dtype=dt, device="cuda")
    v = torch.zeros(shape, dtype=dt, device="cuda")
    ks = torch.ones((B, nl, H), dtype=torch.float32, device="cuda") if fp8 else None
    vs = torch.ones((B, nl, H), dtype=torch.float32, device="cuda") if fp8 else None
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    for b in range(B):
        L = wl.lengths[b]
        if L == 0:
            continue  # no rows (and scales of 1)
        for l in range(nl):
            for t, sc in ((k, ks), (v, vs)):
                x = torch.randn((H, L, Dh), generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
                if fp8:
                    x = x.float()
                    scale = x.abs().amax(dim=(1, 2)) / 448.0
                    scale = torch.where(scale > 0, scale, torch.ones_like(scale))
                    sc[b, l] = scale
                    x = (x / scale[:, None, None]).clamp(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8)
                t[b, l, :, :L] = x
    torch.cuda.synchronize()
    desc = fsx.CacheDesc(k, v, fsx.FP8_E4M3 if fp8 else fsx.BF16, nl, H, Dh, cap, wl.lengths, positions=wl.lengths,
                         k_scale=ks, v_scale=vs)
    return desc, (k, v, ks, vs)


def time_launches(fn, stream, steps: int, warmup: int) -> float:
    """Seconds per call of fn over `steps` back-to-back calls on `stream`, HIP events around the whole run."""
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3 / steps


def time_each(fn, stream, steps: int):
    """Seconds of each of `steps` back-to-back calls of fn on `stream` (an event pair around every call, one
    synchronisation at the end): (10th percentile, median, 90th percentile)."""
    import numpy as np
    import torch

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in ev:
        e0.record(stream)
        fn()
        e1.record(stream)
    torch.cuda.synchronize()
    t = np.array([e0.elapsed_time(e1) / 1e3 for e0, e1 in ev])
    return tuple(float(x) for x in np.percentile(t, [10, 50, 90]))


def time_cold(fn, stream, steps: int, flush) -> float:
    """Seconds per call with the Infinity Cache (256 MB) flushed before each call: a 1 GiB write runs before each
    call, outside its event pair; the per-call event times are averaged."""
    import torch

    tot = 0.0
    for _ in range(steps):
        flush()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        tot += e0.elapsed_time(e1) / 1e3
    return tot / steps


def hbm_ceiling(stream, nbytes: int = 4 << 30, reps: int = 10):
    """GB/s of one read-only pass over nbytes with the library's probe kernel (register loads / direct LDS loads)."""
    import torch

    from paper_2607_15621_amd import fsx

    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(3)
    sink = torch.zeros(1024, dtype=torch.int32, device="cuda")
    out = {"bytes": nbytes}
    for mode, name in ((0, "register_loads_gbs"), (1, "lds_direct_loads_gbs")):
        t = time_launches(lambda: fsx.probe_hbm_read(buf, nbytes, mode, sink, stream), stream, reps, 2)
        out[name] = round(nbytes / t / 1e9, 1)
    # a 128 MiB pass (direct loads) right after a pass over the same bytes (held in the 256 MB Infinity Cache)
    # against one after a pass over 1 GiB of other bytes: what the cache gives a re-read
    small = 128 << 20
    part, rest = buf[:small], buf[small:small + (1 << 30)]

    def one_pass(before):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fsx.probe_hbm_read(before, before.numel(), 1, sink, stream)
        e0.record(stream)
        fsx.probe_hbm_read(part, small, 1, sink, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3

    for name, before in (("reread_128MiB_gbs", part), ("after_other_1GiB_128MiB_gbs", rest)):
        t = sorted(one_pass(before) for _ in range(7))[3]
        out[name] = round(small / t / 1e9, 1)
    del buf, part, rest
    torch.cuda.empty_cache()
    return out


def run_workload(name: str, steps: int, warmup: int, multi_launch: bool, cold_steps: int, flush):
    import torch

    import synth
    from gpu_inputs import Model, tokens_for
    from paper_2607_15621_amd import fsx

    wl = synth.WORKLOADS[name]
    model = Model(wl)
    ex = model.create(flags=fsx.FLAG_MULTI_LAUNCH if multi_launch else 0)
    info = fsx.expert_info(ex)
    desc, keep = gpu_cache(wl, seed=1000 + wl.wid)
    _, tok = tokens_for(wl)
    wp = torch.zeros(wl.batch, wl.n_out, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        fsx.expert_forward(ex, desc, tok, wl.batch, wl.n_frame_tokens, wp, None, stream)

    per_tick = time_launches(step, stream, steps, warmup)
    fsx.expert_status(ex, stream)
    assert torch.isfinite(wp).all(), f"non-finite waypoints ({name})"
    nbytes = algorithmic_bytes(wl, info["weight_bytes"])
    achieved = nbytes / per_tick / 1e9
    r = {"us_per_tick": round(per_tick * 1e6, 2), "ticks_per_s": round(wl.batch / per_tick, 3),
         "agents": wl.batch, "cache_rows": list(wl.lengths), "frame_tokens": wl.n_frame_tokens,
         "cache_dtype": wl.cache_dtype, "algorithmic_bytes": nbytes, "achieved_gbs": round(achieved, 1),
         "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(wl.name),
         "dram_traffic": measured_traffic(wl.name, "dram_bytes_per_launch")}
    # the spread of single ticks (a separate pass, so the back-to-back figure above has no events between calls)
    p10, p50, p90 = time_each(step, stream, steps)
    r.update({"us_per_tick_p10": round(p10 * 1e6, 2), "us_per_tick_median": round(p50 * 1e6, 2),
              "us_per_tick_p90": round(p90 * 1e6, 2)})
    if cold_steps > 0:
        cold = time_cold(step, stream, cold_steps, flush)
        r["us_per_tick_mall_flushed"] = round(cold * 1e6, 2)
        r["frac_mall_flushed"] = round(nbytes / cold / 1e9 / HBM_PEAK_GBS, 4)
    extra = {}
    if wl.append_rows:
        # the append of the batched workload: n rows per (agent, layer), K and V, read once and written once
        n = wl.append_rows
        g = torch.Generator(device="cuda")
        g.manual_seed(7)
        shp = (wl.batch, wl.n_layers, wl.n_heads, n, wl.head_dim)
        kr = torch.randn(shp, generator=g, device="cuda").to(torch.bfloat16)
        vr = torch.randn(shp, generator=g, device="cuda").to(torch.bfloat16)
        ta = time_launches(lambda: fsx.cache_append_rows(desc, kr, vr, n, fsx.APPEND_RING, stream), stream, steps,
                           warmup)
        moved = 2 * 2 * kr.numel() * 2  # K and V, read + write, bf16
        extra = {"workload": name, "rows_per_agent_layer": n, "us_per_append": round(ta * 1e6, 2),
                 "bytes_moved": moved, "achieved_gbs": round(moved / ta / 1e9, 1)}
    ex.close()
    del keep, desc
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return wl, r, extra


def run_backbone(batches=(1, 16), n_new: int = 4, steps: int = 10, warmup: int = 2):
    """The backbone's incremental forward (the producer of the appended rows) at LLaMA-7B shapes -- 32 layers, width
    4096, 32 x 128 heads, SwiGLU 11008, synthetic weights N(0, 0.02^2) drawn on the GPU -- appending n_new tokens per
    agent: one agent over a 224-row cache (the 40-frame history) and 16 agents over 1024-row caches (the batched
    workload's append).  ms per append and the bandwidth of the bytes one call must read (packed weights + cached
    rows)."""
    import torch

    from paper_2607_15621_amd import fsx

    nl, d, H, Dh, F = 32, 4096, 32, 128, 11008
    g = torch.Generator(device="cuda")
    g.manual_seed(2024)
    bf = torch.bfloat16

    def w(*shape):
        return (torch.randn(shape, generator=g, device="cuda") * 0.02).to(bf)

    layers = []
    for _ in range(nl):
        layers.append({"wq": w(H * Dh, d), "wk": w(H * Dh, d), "wv": w(H * Dh, d), "wo": w(d, H * Dh),
                       "w_gate": w(F, d), "w_up": w(F, d), "w_down": w(d, F),
                       "attn_norm": torch.ones(d, device="cuda"), "ffn_norm": torch.ones(d, device="cuda")})
    cfg = fsx.BackboneCfg(nl, d, H, Dh, F, n_new, max(batches), fsx.BF16, 10000.0, 1e-6)
    bb = fsx.Backbone(cfg, layers)
    torch.cuda.synchronize()
    del layers
    torch.cuda.empty_cache()
    wbytes = bb.info()["weight_bytes"]
    stream = torch.cuda.current_stream()
    out = {"model": "LLaMA-7B shapes (32 layers, d 4096, 32 x 128 heads, SwiGLU 11008), synthetic weights",
           "new_tokens_per_agent": n_new, "weight_bytes": wbytes, "paper_ms_per_append_rtx3090ti": 21.1}
    for B in batches:
        L = 224 if B == 1 else 1024
        cap = L + n_new
        k = torch.randn((B, nl, H, cap, Dh), generator=g, device="cuda").to(bf)
        v = torch.randn((B, nl, H, cap, Dh), generator=g, device="cuda").to(bf)
        desc = fsx.CacheDesc(k, v, fsx.BF16, nl, H, Dh, cap, [L] * B)
        tok = torch.randn((B, n_new, d), generator=g, device="cuda").to(bf)
        torch.cuda.synchronize()
        t = time_launches(lambda: bb.append(desc, tok, B, n_new, None, fsx.APPEND_RING, stream), stream, steps, warmup)
        nbytes = wbytes + B * L * nl * 2 * H * Dh * 2
        out[f"agents_{B}"] = {"cache_rows": L, "ms_per_append": round(t * 1e3, 3), "bytes_read": nbytes,
                              "achieved_gbs": round(nbytes / t / 1e9, 1),
                              "frac": round(nbytes / t / 1e9 / HBM_PEAK_GBS, 4)}
        del k, v, desc, tok
        torch.cuda.empty_cache()
    bb.close()
    torch.cuda.empty_cache()
    return out


# Tick time across cache lengths (one agent) and agent counts (1,024 rows each) of the full-size expert, bf16 cache,
# no frame tokens: the shapes of Sec. 4.4's latency discussion, at the history lengths the cache can hold.
SWEEP_LENGTHS = (0, 104, 224, 464, 1024, 2048, 4096, 8192, 16384)
SWEEP_BATCHES = (1, 2, 4, 8, 16, 32)


PHASE_NAMES = ("Q", "A", "O + R1", "F1", "D + R2")


def attention_tail(tr, nl: int, t0: int, nx: int = 8):
    """Over every layer after the first, from a tick's phase trace (rows: workgroups, w on XCD w mod nx; words
    2 + 16 l + e: end of phase e of layer l, 2 + 16 l + 5 + 4: end of the first attention unit, 100 MHz): each
    XCD's latest attention end (µs after the previous layer's end) averaged over the layers, the latest of all
    averaged over the layers, and each slot's attention end against the median of its XCD, averaged over the layers
    and XCDs (slot k of an XCD is workgroup nx k + XCD; its slice of the attention is the same in every layer).
    These tell an XCD that is slow from slices that the plan weighs wrongly."""
    import numpy as np

    per_x, rel = [], []
    for l in range(1, nl):
        base = tr[:, 2 + 16 * (l - 1) + 4].max()
        a_end = (tr[:, 2 + 16 * l + 1] - base) / 100.0
        ran = tr[:, 2 + 16 * l + 5 + 4] >= t0  # ran an attention unit in this tick
        per_x.append([float(a_end[x::nx][ran[x::nx]].max()) if ran[x::nx].any() else float(a_end[x::nx].max())
                      for x in range(nx)])
        r = np.zeros_like(a_end)
        for x in range(nx):
            r[x::nx] = a_end[x::nx] - np.median(a_end[x::nx])
        rel.append(r)
    per_x, rel = np.array(per_x), np.array(rel)
    n_slot = tr.shape[0] // nx
    slot_mean = [float(rel[:, nx * k:nx * k + nx].mean()) for k in range(n_slot)]
    return [float(v) for v in per_x.mean(0)], float(per_x.max(1).mean()), slot_mean


def run_phase_trace(names, out_md: str, command: str, layers=(8, 16), ticks: int = 4):
    """Per-phase times of the tick kernel from its own timestamps (FSX_FLAG_TRACE: every workgroup stamps the end of
    each phase of each layer with the 100 MHz real-time counter).  For each workload and layer: each phase's end,
    median and latest over the workgroups, relative to the latest end of the previous layer; a phase's time is the
    difference of consecutive median ends (the attention also to its latest end)."""
    import numpy as np
    import torch

    import synth
    from gpu_inputs import Model, tokens_for
    from paper_2607_15621_amd import fsx

    stream = torch.cuda.current_stream()
    out = ["# Tick phases from the kernel's own timestamps", "",
           "Each workgroup of the persistent tick kernel stamps the end of every phase of every layer "
           "(`FSX_FLAG_TRACE`, 100 MHz real-time counter); the last of " + str(ticks) + " back-to-back ticks is read. "
           "Ends are µs after the latest workgroup's end of the previous layer (median / latest over the workgroups; "
           "for the attention over those that ran an attention unit); a phase's time is the difference of "
           "consecutive median ends (attention: also to its latest end).", "", f"Command: `{command}`", ""]
    for name in names:
        wl = synth.WORKLOADS[name]
        model = Model(wl)
        ex = model.create(flags=fsx.FLAG_TRACE)
        desc, keep = gpu_cache(wl, seed=1000 + wl.wid)
        _, tok = tokens_for(wl)
        wp = torch.zeros(wl.batch, wl.n_out, device="cuda")
        for _ in range(ticks):
            fsx.expert_forward(ex, desc, tok, wl.batch, wl.n_frame_tokens, wp, None, stream)
        torch.cuda.synchronize()
        fsx.expert_status(ex, stream)
        tr = fsx.expert_trace(ex).astype(np.int64)
        nl = wl.n_layers
        t0 = tr[:, 0].min()
        pre = (tr[:, 1].max() - t0) / 100.0  # registration, attention plan, embedding: every workgroup done
        post = (tr[:, 2 + 16 * nl].max() - tr[:, 2 + 16 * (nl - 1) + 4].max()) / 100.0  # the head
        out += [f"## `{name}`: tick {(tr[:, 2 + 16 * nl].max() - t0) / 100.0:.1f} µs "
                f"(before the first layer {pre:.1f} µs, after the last {post:.1f} µs)", "",
                "| layer | phase | end, median | end, latest | time |", "|---:|---|---:|---:|---:|"]
        xcd_notes = []
        for l in layers:
            base = tr[:, 2 + 16 * (l - 1) + 4].max()
            prev = 0.0
            # workgroups that ran an attention unit in this tick (their first unit's mark is from this tick): with
            # few segments only those stream the cache, the others end the phase at once
            att = tr[:, 2 + 16 * l + 5 + 4] >= t0
            for e, ph in enumerate(PHASE_NAMES):
                v = tr[:, 2 + 16 * l + e]
                if ph == "A" and att.any():
                    v = v[att]
                v = (v[v >= t0] - base) / 100.0
                med, last = float(np.median(v)), float(v.max())
                t = f"{med - prev:.1f}" + (f" / {last - prev:.1f}" if ph == "A" else "")
                out.append(f"| {l} | {ph} | {med:.1f} | {last:.1f} | {t} |")
                prev = med
            out.append(f"| {l} | layer | | {(tr[:, 2 + 16 * l + 4].max() - base) / 100.0:.1f} | |")
            # the attention's latest end on each XCD (workgroup w runs on XCD w mod 8, as the create-time probe
            # measures on this device)
            a_end = (tr[:, 2 + 16 * l + 1] - base) / 100.0
            per_x = [float(a_end[x::8][att[x::8]].max()) if att[x::8].any() else float(a_end[x::8].max())
                     for x in range(8)]
            xcd_notes.append(f"layer {l}: " + ", ".join(f"{v:.1f}" for v in per_x) +
                             f" (spread {max(per_x) - min(per_x):.1f} µs)")
        out += ["", "Latest attention end per XCD (µs, XCD 0..7):", ""] + [f"* {n}" for n in xcd_notes]
        px, latest, slot_mean = attention_tail(tr, nl, t0)
        out += ["", f"Layers 2..{nl}: latest attention end per XCD, mean over the layers (µs, XCD 0..7): " +
                ", ".join(f"{v:.1f}" for v in px) + f"; the latest of all, mean over the layers: {latest:.1f}.", "",
                "Attention end of each slot against the median of its XCD, mean over the layers and XCDs (µs, slot "
                "0..): " + ", ".join(f"{v:+.1f}" for v in slot_mean) + "."]
        out.append("")
        print(f"# phases {name}: done", file=sys.stderr, flush=True)
        ex.close()
        del keep, desc
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    with open(out_md, "w") as f:
        f.write("\n".join(out))


def run_sweep(steps: int, warmup: int, out_md: str, command: str, cache_dtype: str = "bf16"):
    import torch

    import synth
    from gpu_inputs import Model, tokens_for
    from paper_2607_15621_amd import fsx

    points = [(1, L) for L in SWEEP_LENGTHS] + [(B, 1024) for B in SWEEP_BATCHES if B != 1]
    rows = []
    stream = torch.cuda.current_stream()
    for i, (B, L) in enumerate(points):
        wl = synth.Workload(name=f"sweep_B{B}_L{L}", wid=100 + i, n_frame_tokens=0, batch=B, lengths=(L,) * B,
                            dtype="bf16", cache_dtype=cache_dtype, capacity=max(L, 1), **synth.FULL)
        model = Model(wl)
        ex = model.create()
        info = fsx.expert_info(ex)
        desc, keep = gpu_cache(wl, seed=2000 + i)
        _, tok = tokens_for(wl)
        wp = torch.zeros(wl.batch, wl.n_out, device="cuda")
        per_tick = time_launches(lambda: fsx.expert_forward(ex, desc, tok, B, 0, wp, None, stream), stream, steps,
                                 warmup)
        fsx.expert_status(ex, stream)
        assert torch.isfinite(wp).all(), f"non-finite waypoints ({wl.name})"
        nbytes = algorithmic_bytes(wl, info["weight_bytes"])
        gbs = nbytes / per_tick / 1e9
        rows.append({"agents": B, "cache_rows": L, "us_per_tick": round(per_tick * 1e6, 1),
                     "agent_ticks_per_s": round(B / per_tick, 1), "algorithmic_mb": round(nbytes / 1e6, 1),
                     "achieved_gbs": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)})
        print(f"# sweep B={B} L={L}: {rows[-1]['us_per_tick']} us/tick, frac {rows[-1]['frac']}", file=sys.stderr,
              flush=True)
        ex.close()
        del keep, desc
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    out = ["# Tick time across cache lengths and agent counts", "",
           "Full-size expert (32 layers, width 512, 32 heads x 128, SwiGLU 2048, 10 expert tokens), bf16 weights, "
           f"{'fp8 (E4M3, a scale per agent, layer and head for K and for V)' if cache_dtype == 'fp8' else 'bf16'} cache, no frame tokens, seeded "
           "synthetic inputs; one persistent tick-kernel launch per tick, "
           f"{steps} back-to-back launches timed with HIP events after {warmup} warm-up launches. `frac` is the "
           "algorithmic bytes (weights once, every cached K/V row once) per tick over 8 TB/s.", "",
           f"Command: `{command}`", "",
           "| agents | cache rows per agent | µs/tick | agent-ticks/s | algorithmic MB | GB/s | frac |",
           "|---:|---:|---:|---:|---:|---:|---:|"]
    for r in rows:
        out.append(f"| {r['agents']} | {r['cache_rows']} | {r['us_per_tick']} | {r['agent_ticks_per_s']} | "
                   f"{r['algorithmic_mb']} | {r['achieved_gbs']} | {r['frac']} |")
    with open(out_md, "w") as f:
        f.write("\n".join(out) + "\n")
    print(json.dumps({"sweep": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=",".join(ALL_WORKLOADS),
                    help="comma-separated workloads; the first is the headline line")
    ap.add_argument("--cold-steps", type=int, default=10, help="ticks timed with the Infinity Cache flushed (0: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-hbm-probe", action="store_true")
    ap.add_argument("--no-backbone", action="store_true", help="skip the backbone's incremental forward")
    ap.add_argument("--multi-launch", action="store_true", help="one launch per phase instead of the tick kernel")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES")
    ap.add_argument("--summarize-trace", metavar="DIR")
    ap.add_argument("--bench-line", metavar="FILE")
    ap.add_argument("--trace-name", default="", help="with --summarize-trace: write profiles/<NAME>.md")
    ap.add_argument("--summarize-traffic", nargs=4, metavar="DIR")
    ap.add_argument("--dram", action="store_true", help="with --summarize-traffic: the directories hold "
                    "TCC_EA0_RDREQ_DRAM_sum / TCC_EA0_WRREQ_DRAM_sum runs")
    ap.add_argument("--copy-bytes", type=int, default=0)
    ap.add_argument("--summarize-parity", metavar="JSONL", help="write profiles/parity_errors.md from the parity log")
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR", help="write profiles/instructions_tick.md from "
                    "rocprofv3 --pmc runs of the workloads (in --workload order, the same number of passes each)")
    ap.add_argument("--command", action="append", default=[], help="command recorded in a summary")
    ap.add_argument("--sweep", metavar="MD", help="time the tick across cache lengths and agent counts and write "
                    "the table to MD")
    ap.add_argument("--sweep-cache", choices=("bf16", "fp8"), default="bf16", help="cache element type of --sweep")
    ap.add_argument("--phase-trace", metavar="MD", help="per-phase times of the workloads' ticks from the kernel's "
                    "timestamps, written to MD")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.workload, args.bench_line, " && ".join(args.command), args.trace_name)
        return
    if args.summarize_parity:
        summarize_parity(args.summarize_parity, " && ".join(args.command))
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, [n for n in args.workload.split(",") if n], args.command)
        return
    if args.summarize_traffic:
        summarize_traffic(args.summarize_traffic, args.workload, args.copy_bytes, args.command, args.dram)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    torch.cuda.set_device(0)
    if args.phase_trace:
        argv = [os.path.basename(x) if x == args.phase_trace else x for x in sys.argv[1:]]
        run_phase_trace([n for n in args.workload.split(",") if n], args.phase_trace,
                        " ".join(["python", "bench.py"] + argv))
        return
    if args.sweep:
        # the recorded command names the output file by its base name (the directory is the caller's choice)
        argv = [os.path.basename(x) if x == args.sweep else x for x in sys.argv[1:]]
        run_sweep(args.steps, args.warmup, args.sweep, " ".join(["python", "bench.py"] + argv), args.sweep_cache)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        return
    stream = torch.cuda.current_stream()
    names = [n for n in args.workload.split(",") if n]
    flush_buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda") if args.cold_steps > 0 else None
    flush = (lambda: flush_buf.fill_(0)) if flush_buf is not None else None
    t_start = time.perf_counter()
    results, append = {}, None
    head_wl = None
    for i, name in enumerate(names):
        wl, r, extra = run_workload(name, args.steps, args.warmup, args.multi_launch, args.cold_steps, flush)
        results[name] = r
        if extra:
            append = extra
        if i == 0:
            head_wl = wl
        print(f"# {name}: {r['us_per_tick']} us/tick, frac {r['frac']} (single ticks p10 / median / p90: "
              f"{r['us_per_tick_p10']} / {r['us_per_tick_median']} / {r['us_per_tick_p90']} us)", file=sys.stderr,
              flush=True)
    del flush_buf
    torch.cuda.empty_cache()
    ceiling = None if args.no_hbm_probe else hbm_ceiling(stream)
    backbone = None if args.no_backbone else run_backbone()
    wl = head_wl
    h = results[names[0]]
    per_tick = h["us_per_tick"] / 1e6
    value = wl.batch / per_tick  # agent-ticks per second
    if ceiling:
        best = max(ceiling["register_loads_gbs"], ceiling["lds_direct_loads_gbs"])
        for r in results.values():
            r["frac_of_ceiling"] = round(r["achieved_gbs"] / best, 4)
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "ticks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(per_tick * 1e3, 5),
        "us_per_tick": h["us_per_tick"],
        "higher_is_better": True,
        "scaling": "weak",
        # the paper's expert tick (another machine) is quoted for the 40-frame history only
        "vs_baseline": round(value / (1000.0 / PAPER_EXPERT_MS), 3) if wl.name == "single_bf16_L224" else None,
        "dtype": "bf16" if wl.cache_dtype != "fp8" else "bf16 (fp8-e4m3 cache)",
        "data": "synthetic (seeded N(0,1) tokens and cache, N(0,0.02^2) weights)",
        "config": {"workload": wl.name, "agents": wl.batch, "cache_rows": list(wl.lengths)[:8],
                   "layers": wl.n_layers, "d_model": wl.d_model, "heads": wl.n_heads, "head_dim": wl.head_dim,
                   "d_ffn": wl.d_ffn, "expert_tokens": wl.n_expert_tokens, "frame_tokens": wl.n_frame_tokens,
                   "launch": "multi" if args.multi_launch else "tick-kernel"},
        "roofline": {"bound": "hbm", "achieved": h["achieved_gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": h["frac"], "traffic": h["traffic"], "algorithmic_bytes_per_launch": h["algorithmic_bytes"]},
        "workloads": results,
        "append": append,
        "backbone_append": backbone,
        "hbm_read_ceiling": ceiling,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    out["bench_wall_s"] = round(time.perf_counter() - t_start, 1)
    print(json.dumps(out), flush=True)
    # every device allocation is released here, before the interpreter's exit handlers (and a profiler's) run
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
