#!/usr/bin/env python3
"""Benchmark of the batched kernel-latency evaluator on one MI355X.

One benchmark step = one ks_eval_steps call: every stage of the path (record
stream, exact counts, waves, roofline, features, efficiency head on MFMA,
launch floor, per-step sums, all-reduce and step assembly) for every
(spec vector, record) pair of the workload.  Inputs are resident in HBM
before the timed region; only the library call is timed (HIP events on the
stream it launches on).

Default workload: the capacity-planning grid — the Llama-7B trace (1000
steps) plus the first 345 steps of the six-shape S2 trace, 390,050 kernel
records x 256 hypothetical spec vectors = 99.9 M latency predictions per
step, bf16 16->128->128->1 heads.

Prints one JSON line (see the keys below)."""
from __future__ import annotations

import argparse
import json
import os
import platform
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "kernel latency predictions/sec and step evals/sec at 1 GPU; % of HBM/MFMA peak"
PEAK = {"bf16": 2.5e15, "f32": 157.3e12, "hbm": 8.0e12}


C5_BATCH_STEPS = 88_640      # 88,640 steps x 722 kernels = 64.0 M records


def _workload(name: str):
    """(workload, description, oracle sample, batch traces) for each benchmark
    workload.  The oracle sample bounds the CPU baseline to ~10-30 s of
    work; the traces are the batch descriptors the records come from."""
    from workload import gen
    if name == "c4":
        return (gen.config4(), "c4-capacity-grid: llama-7b c1 trace + S2 trace prefix, 256 specs",
                {"specs": 16, "steps": None},
                [gen.trace_c1(), gen.trace_c2(1).slice(0, gen.C4_GRID_STEPS)])
    if name == "c1":
        return (gen.config1(), "c1-llama7b: 1000 steps, 2 datasheet specs, fp32 heads", {"specs": 2, "steps": None},
                [gen.trace_c1()])
    if name == "c3":
        wl = gen.config3()
        return (wl, "c3-mixtral-moe: the whole 200k-step trace (8 experts top-2, Dirichlet(0.5) routing, ragged "
                    "grouped GEMMs) in one call, 2 datasheet specs, bf16 16-128-128-1 heads",
                {"specs": 2, "steps": 200}, [])
    if name == "c5-batch":
        wl = gen.config5(0, C5_BATCH_STEPS)
        return (wl, f"c5-70b-prefix: one 64M-record batch (steps 0..{C5_BATCH_STEPS}), 2 datasheet specs, "
                    "bf16 32-256-256 heads", {"specs": 2, "steps": 300},
                [gen.trace_c5().slice(0, C5_BATCH_STEPS)])
    raise SystemExit(f"unknown workload {name}")


def expand_bytes(n_records: int, n_steps: int, with_mult: bool) -> float:
    """Algorithmic HBM bytes of the expansion's record writer: six u32 fields
    per record (seven with the multiplicity) written, and per step the token
    count, the prefill flag and the request offset it reads."""
    return n_records * 4.0 * (7 if with_mult else 6) + n_steps * 9.0


def kernel_source_hash() -> str:
    """SHA-256 of the GPU kernels' sources with comments and blank lines
    taken out, so that the recorded counters follow the code, not its
    commentary."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in ("ks_kernels.hip", "ks_expand.hip", "ks_internal.h", "ks_sched.inc"):
        with open(os.path.join(ROOT, "paper_2606_28565_amd", "csrc", f)) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        code = [line.rstrip() for line in text.splitlines() if line.strip()]
        h.update(("\n".join(code) + "\n").encode())
    return h.hexdigest()


def recorded_traffic(key: str):
    """HBM bytes per launch of the evaluation kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE summary, scaled by the copy-kernel
    calibration; None if absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh).get(key)
    if not rec or rec.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return rec["hbm_bytes_per_launch"]


def traffic_key(args) -> str:
    """The traffic.json entry of a benchmark configuration (the flags that
    change the evaluation kernel or its inputs)."""
    k = args.workload
    if getattr(args, "eta_one", False):
        k += "-eta1"
    if getattr(args, "kernels", False):
        k += "-kernels"
    elif getattr(args, "per_pair", False):
        k += "-pair"
    if getattr(args, "bounded", "none") != "none":
        k += "-bounded-" + args.bounded
    if getattr(args, "grid", "none") != "none":
        k += "-grid-" + args.grid
    if getattr(args, "expand", "none") != "none":
        k += "-expand-" + args.expand
    return k


def copy_calibration(nbytes: int, reps: int) -> None:
    """A plain device-to-device copy of nbytes, reps times: the reference
    whose FETCH_SIZE / WRITE_SIZE counters scale the evaluation kernel's."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}), flush=True)


# record fields each family's latency formula reads (4 bytes each)
FIELDS_USED = {0: 4, 1: 4, 2: 5, 3: 4, 4: 4, 5: 3, 6: 4, 7: 3, 8: 4, 9: 3}


def stream_bytes(wl, n_specs: int, sums: bool = True, pair_outputs: int = 0) -> float:
    """Algorithmic HBM bytes of one evaluation-kernel launch: the record
    fields each family uses, the per-expert row counts of grouped records,
    the per-step attention work (4 x u64 per step), and the writes: with
    step sums one range (2 x u32) per (family, step) and one fp64 partial
    per (spec, family, step); pair_outputs fp32 values per (spec, record)."""
    import numpy as np
    d = wl.desc
    rows = np.diff(d.fam_off)
    b = float(sum(int(rows[f]) * 4 * FIELDS_USED[f] for f in range(len(rows))))
    g0, g1 = int(d.fam_off[2]), int(d.fam_off[3])
    b += 4.0 * float(d.a[g0:g1].astype(np.int64).sum())
    b += 32.0 * d.n_steps
    if sums:
        segs = sum(len(np.unique(d.step[d.fam_off[f]:d.fam_off[f + 1]])) for f in range(len(rows)))
        b += segs * (8.0 + 8.0 * n_specs)
    b += 4.0 * pair_outputs * d.n_rows * n_specs
    return b


def head_flops_per_pair(in_dim: int, hidden: int) -> int:
    """Algorithmic MLP FLOPs of one prediction: 2 (in h + h h + h)."""
    return 2 * (in_dim * hidden + hidden * hidden + hidden)


def host_threads() -> int:
    """Host threads this process may run on (its CPU affinity), i.e. all the
    host cores the box gives it."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(wl, sample: dict, eta_one: bool, threads: int, bounded=None, grid=None):
    """The oracle as it stands, on a bounded sample of the same workload:
    the first sample["specs"] spec vectors and, if sample["steps"] is set,
    only the records of the first sample["steps"] steps."""
    from threadpoolctl import threadpool_limits
    from oracle import ks_oracle as o
    spec_ids = list(range(min(sample["specs"], wl.n_specs)))
    rows = None
    if sample["steps"] is not None:
        import numpy as np
        rows = np.nonzero(wl.desc.step < sample["steps"])[0]
    with threadpool_limits(limits=threads):
        t = time.perf_counter()
        k = o.eval_kernels(wl.desc, wl.specs, None if eta_one else wl.heads, eta_one=eta_one,
                           spec_ids=spec_ids, rows=rows, bounded=bounded, grid=grid)
        if rows is None:
            o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, spec_ids=spec_ids, kern=k)
        dt = time.perf_counter() - t
    n = wl.desc.n_rows if rows is None else len(rows)
    pairs = n * len(spec_ids)
    what = f"all {n} records" if rows is None else f"the {n} records of steps 0..{sample['steps']}"
    return {"value": pairs / dt, "unit": "predictions/s", "cores": threads, "kind": "oracle",
            "os_cpu_count": os.cpu_count(), "pairs": pairs, "seconds": dt,
            "sample": f"{what} x {len(spec_ids)} of {wl.n_specs} spec vectors "
                      f"({pairs} predictions, {dt:.1f} s, fp64 numpy, {threads} BLAS threads)"}


def _print_expand_only(args, wl, wdesc, db, ms, k_ms) -> int:
    hom = args.expand == "homogeneous"
    eb = expand_bytes(db.fam_off[-1], db.desc.n_steps, hom)
    out = {
        "metric": "kernel records expanded/s", "value": db.fam_off[-1] / (ms * 1e-3), "unit": "records/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": wdesc + " (batch expansion only, "
                               + ("homogeneous" if hom else "per-layer") + " records)",
                   "records": db.fam_off[-1], "serving_steps": db.desc.n_steps},
        "roofline": {"bound": "hbm", "achieved": eb / (k_ms * 1e-3) / 1e9, "peak": PEAK["hbm"] / 1e9,
                     "unit": "GB/s", "frac": eb / (k_ms * 1e-3) / PEAK["hbm"],
                     "traffic": None if hom else recorded_traffic(f"{args.workload}-expand"),
                     "kernel_ms": k_ms,
                     "note": "achieved = record bytes written (+ per-step inputs read) by the record "
                             "writer / its mean HIP-event duration"},
    }
    print(json.dumps(out), flush=True)
    return 0


def nearest_rank(x, p):
    """P_p = x_(k), k = ceil(p/100 n) over the ascending sample (the paper's
    percentile definition)."""
    import math
    xs = sorted(float(v) for v in x)
    if not xs:
        return None
    return xs[max(1, math.ceil(p / 100.0 * len(xs))) - 1]


SIM_SCHED = dict(max_num_seqs=256, max_batched_tokens=8192, block_tokens=16, prefix_cache=1,
                 kv_blocks=12_500)   # about 100 GB of bf16 KV for the Llama-7B shape


SIM_GRID_SEED = 20260602 + 300


def _sim_inputs(n, rate, n_specs=1):
    """Requests, spec table (the GB200 datasheet row, then n_specs - 1
    hypothetical GPUs of the capacity-planning grid), heads, host constants
    and scheduler of the serving simulation."""
    from workload import gen
    from paper_2606_28565_amd import abi
    import numpy as np
    import torch
    reqs = gen.make_requests(n, rate)
    ds = gen.specs_datasheet()
    table = {k: np.asarray(v[:1]) for k, v in ds.items()}
    if n_specs > 1:
        grid = gen.specs_grid(n_specs - 1, SIM_GRID_SEED)
        table = {k: np.concatenate([table[k], np.asarray(grid[k], table[k].dtype)]) for k in table}
    h = gen.make_heads(16, 64, "f32")
    hd = abi.ks_heads()
    hd.in_dim, hd.hidden, hd.precision, hd.mode = 16, 64, abi.KS_F32, abi.KS_ETA_MLP
    keep = {}
    for name in ("w1", "w2", "b2", "w3", "b3"):
        keep[name] = torch.from_numpy(np.ascontiguousarray(h.storage[name]).reshape(-1).copy()).cuda()
        setattr(hd, name, keep[name].data_ptr())
    hc = gen.HostConsts()
    host = abi.ks_host(hc.c_disp, hc.ell, hc.c_ovl, hc.c_tail, hc.body_scale)
    sched = abi.ks_sched(*(SIM_SCHED[k] for k, _ in abi.ks_sched._fields_))
    return reqs, table, hd, keep, host, sched, h


def _serving_summary(reqs, res):
    import numpy as np
    fin = res["state"] == 2
    out_tok = int(np.asarray(reqs["output"])[fin].sum())
    span = float(np.max((res["e2e"] + reqs["arrival"])[fin]) - reqs["arrival"][0]) if fin.any() else 0.0
    return {"finished": int(fin.sum()), "preemptions": res["preemptions"], "simulated_steps": res["n_steps"],
            "simulated_seconds": res["clock"],
            "output_tokens_per_s": out_tok / span if span > 0 else None,
            "ttft_s": {f"p{p}": nearest_rank(res["ttft"][fin], p) for p in (50, 90, 99)},
            "tpot_s": {f"p{p}": nearest_rank(res["tpot"][fin & (np.asarray(reqs["output"]) > 1)], p)
                       for p in (50, 90, 99)}}


def _bench_simulate(args) -> int:
    """Serving simulation: the host scheduler forms every step's batch, the
    GPU path prices it, the clock advances by its t_step; with --sim-specs
    S, S simulations (one per spec vector) run in lockstep and each round's
    steps are priced by one expansion and one evaluation call.  value =
    simulated steps (all simulations) per wall-clock second of the whole
    ks_simulate call."""
    import torch
    from workload import gen
    from paper_2606_28565_amd import abi
    S = args.sim_specs
    reqs, table, hd, keep, host, sched, h = _sim_inputs(args.simulate, args.rate, S)
    warm = {k: v[:min(50, len(v))] for k, v in reqs.items()}
    abi.simulate_many(gen.LLAMA7B, table, hd, host, sched, warm, step_cap=1 << 16, entry_cap=1 << 20)
    torch.cuda.synchronize()
    t = time.perf_counter()
    many = abi.simulate_many(gen.LLAMA7B, table, hd, host, sched, reqs, step_cap=1 << 16, entry_cap=1 << 20)
    wall = time.perf_counter() - t
    steps = sum(r["n_steps"] for r in many)
    rounds = max(r["n_steps"] for r in many)
    spec_desc = "GB200 datasheet row" + (f" + {S - 1} capacity-grid GPUs (seed {SIM_GRID_SEED})" if S > 1 else "")
    line = {
        "metric": "simulated serving steps/s (scheduler in the loop, each step priced on the GPU)",
        "value": steps / wall, "unit": "steps/s", "n_gpus": 1, "steps": 1, "warmup": 1,
        "ms_per_step": wall * 1e3, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"serving simulation: {args.simulate} Poisson requests at {args.rate}/s, "
                               f"llama-7b shape, {S} spec vector(s) in lockstep ({spec_desc}), "
                               "fp32 16-64-64-1 heads",
                   "scheduler": SIM_SCHED, "simulations": S},
        "simulated_steps": steps, "rounds": rounds, "wall_ms_per_round": wall * 1e3 / max(rounds, 1),
        "wall_ms_per_simulated_step": wall * 1e3 / max(steps, 1),
        "serving": _serving_summary(reqs, many[0]),
        "roofline": None,
        "note": "launch- and round-trip-bound by design: every round waits for its latencies before the "
                "schedulers form the next steps",
    }
    if S > 1:
        line["per_spec"] = [{"peak_flops": float(table["peak_flops"][i]), "hbm_bw": float(table["hbm_bw"][i]),
                             **{k: v for k, v in _serving_summary(reqs, r).items()
                                if k in ("simulated_steps", "output_tokens_per_s", "preemptions")},
                             "ttft_p50_s": nearest_rank(r["ttft"][r["state"] == 2], 50)}
                            for i, r in enumerate(many[:16])]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = _sim_cpu_baseline(reqs, h, min(args.simulate, 120))
    print(json.dumps(line), flush=True)
    return 0


def _sim_cpu_baseline(reqs, h, n):
    """The oracle's scheduler with the oracle latency model on the first n
    requests."""
    import numpy as np
    from oracle import ks_expand as ox
    from oracle import ks_oracle as o
    from oracle import ks_sim as osim
    from workload import gen
    u = lambda x: np.asarray(x, np.uint32)
    specs = {k: np.asarray(v[:1]) for k, v in gen.specs_datasheet().items()}
    hc = gen.HostConsts()

    def lat(batch, prefill):
        q = [b[0] for b in batch]
        hh = [b[1] for b in batch]
        e = ox.expand(gen.LLAMA7B, [0, len(q)], q, [prefill], homogeneous=True)
        d = gen.Desc(e["fam_off"], *(u(e[k]) for k in ("step", "m", "n", "k", "a", "b")), u([0, len(q)]),
                     u(q), u(hh), u([]), 2, u(e["mult"]))
        rec = gen.StepRec(*(u(e[k]) for k in ("layers", "hidden", "tp", "n_launch")))
        return float(o.eval_steps(d, rec, specs, hc, h)["t_step"][0, 0])
    lst = [{k: (float(reqs[k][i]) if k == "arrival" else int(reqs[k][i])) for k in reqs} for i in range(n)]
    cfg = osim.SchedCfg(SIM_SCHED["max_num_seqs"], SIM_SCHED["max_batched_tokens"], SIM_SCHED["block_tokens"],
                        SIM_SCHED["kv_blocks"], bool(SIM_SCHED["prefix_cache"]))
    t = time.perf_counter()
    r = osim.simulate(lst, cfg, lat)
    dt = time.perf_counter() - t
    return {"value": len(r.steps) / dt, "unit": "steps/s", "cores": 1, "kind": "oracle",
            "sample": f"the first {n} requests ({len(r.steps)} steps, {dt:.1f} s, Python scheduler with the "
                      "fp64 numpy latency model per step)"}



# --------------------------------------------------------------------------
# sweeps: several evaluation calls per benchmark step
# --------------------------------------------------------------------------
FAMILY_FIELDS_USED = FIELDS_USED


def layout_stream_bytes(fam_off, n_steps: int, n_prefill: int, n_specs: int, with_mult: bool) -> float:
    """stream_bytes for the records of a dense decoder's batch expansion,
    from its family offsets alone: every non-attention family with records
    has them in every step, the attention records of a step sit in one of
    the two attention families."""
    rows = [int(fam_off[f + 1] - fam_off[f]) for f in range(len(fam_off) - 1)]
    b = float(sum(rows[f] * 4 * (FIELDS_USED[f] + (1 if with_mult else 0)) for f in range(len(rows))))
    b += 32.0 * n_steps
    segs = 0
    for f, r in enumerate(rows):
        if r == 0:
            continue
        segs += n_prefill if f == 3 else (n_steps - n_prefill if f == 4 else n_steps)
    b += segs * (8.0 + 8.0 * n_specs)
    return b


def _bench_sweep(args) -> int:
    """c2: the six dense shapes of the six-shape workload (TP 1 to 8), each
    its whole 100k-step trace in one ks_eval_steps call; c5: the whole
    500k-step 70B trace in 64M-record step-aligned batches, each expanded
    on the GPU from its batch descriptors (ks_expand) and evaluated
    (ks_eval_steps).  One benchmark step is the whole sweep; inputs (records
    for c2, batch descriptors for c5) are resident in HBM before the timed
    region.  For c5 a second measurement times the sweep with every batch's
    descriptors uploaded from pinned host memory on a second stream, each
    batch's upload overlapping the previous batch's work (not `value`)."""
    import numpy as np
    import torch
    from paper_2606_28565_amd import abi
    from workload import gen

    stream = abi.current_stream()
    mode = abi.KS_ETA_ONE if args.eta_one else abi.KS_ETA_MLP
    parts, keep = [], []
    if args.workload == "c2":
        in_dim, hidden = 16, 128
        for i in range(len(gen.DENSE_SHAPES)):
            print(f"[bench] c2 shape {gen.DENSE_SHAPES[i].name}", file=sys.stderr, flush=True)
            wl = gen.config2(i)
            di = abi.DeviceInputs(wl)
            heads = di.make_heads("bf16", in_dim, hidden, mode)
            so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
            keep += [so_t]
            parts.append({"name": gen.DENSE_SHAPES[i].name, "tp": gen.DENSE_SHAPES[i].tp, "di": di, "db": None,
                          "desc": di.desc, "steps": di.steps, "heads": heads, "so": so, "ws_ptr": di.ws_ptr,
                          "ws_bytes": di.ws_bytes, "rows": wl.desc.n_rows, "eval_rows": wl.desc.n_rows,
                          "n_steps": wl.desc.n_steps,
                          "bytes": stream_bytes(wl, di.n_specs) if args.eta_one else None})
            del wl
        n_specs = parts[0]["di"].n_specs
        wdesc = ("c2-six-shapes: S1..S6 (hidden 2048..8192, 24..80 layers, GQA, TP 1..8), each shape's whole "
                 "100k-step trace in one call, 2 datasheet specs, bf16 16-128-128-1 heads")
        specs_ptr, host = None, None
    else:
        in_dim, hidden = 32, 256
        expand_mode = abi.KS_EXPAND_HOMOGENEOUS if args.expand == "homogeneous" else abi.KS_EXPAND_PER_LAYER
        tr = gen.trace_c5()
        small = gen.config5(0, 2)
        di0 = abi.DeviceInputs(small)
        keep.append(di0)
        heads = di0.make_heads("bf16", in_dim, hidden, mode)
        n_specs = di0.n_specs
        specs_ptr, host = di0.specs_ptr, di0.host
        bounds = list(range(0, tr.n_steps, C5_BATCH_STEPS)) + [tr.n_steps]
        per_layer_rows = 0
        for lo, hi in zip(bounds[:-1], bounds[1:]):
            print(f"[bench] c5 batch steps {lo}..{hi}", file=sys.stderr, flush=True)
            sl = tr.slice(lo, hi)
            db = abi.DeviceBatch(sl, expand_mode)
            ws_bytes = abi.ks_workspace_bytes(db.desc, n_specs)
            ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device="cuda")
            so_t, so = abi.step_outputs(hi - lo, n_specs)
            keep += [ws, so_t]
            n_pre = int(np.count_nonzero(sl.prefill))
            _, pl = abi.ks_expand_layout(db.model, hi - lo, n_pre, abi.KS_EXPAND_PER_LAYER)
            per_layer_rows += pl[-1]
            parts.append({"name": f"steps {lo}..{hi}", "di": None, "db": db, "desc": db.desc, "steps": db.steps,
                          "heads": heads, "so": so, "ws_ptr": ws.data_ptr() + (-ws.data_ptr()) % 256,
                          "ws_bytes": ws_bytes, "rows": pl[-1], "eval_rows": db.fam_off[-1], "n_steps": hi - lo,
                          "bytes": (layout_stream_bytes(db.fam_off, hi - lo, n_pre, n_specs,
                                                        expand_mode == abi.KS_EXPAND_HOMOGENEOUS)
                                    if args.eta_one else None),
                          "trace": sl})
        del tr
        wdesc = (f"c5-70b-prefix-full: the whole 500k-step trace in {len(parts)} step-aligned batches of "
                 f"<= {C5_BATCH_STEPS} steps (64M records), each expanded on the GPU from its batch "
                 f"descriptors ({'homogeneous' if expand_mode == abi.KS_EXPAND_HOMOGENEOUS else 'per-layer'} "
                 "records) and evaluated, 2 datasheet specs, bf16 32-256-256-1 heads")

    def run_part(pt, timed_ev=None):
        if pt["db"] is not None:
            pt["db"].expand(stream)
        if timed_ev is not None:
            abi.ks_set_timing_events(*timed_ev)
        sp = specs_ptr if pt["di"] is None else pt["di"].specs_ptr
        hs = host if pt["di"] is None else pt["di"].host
        abi.ks_eval_steps(pt["desc"], pt["steps"], sp, n_specs, pt["heads"], hs, pt["so"], None,
                          pt["ws_ptr"], pt["ws_bytes"], stream)
        if timed_ev is not None:
            abi.ks_set_timing_events(None, None)

    def step():
        for pt in parts:
            run_part(pt)

    print(f"[bench] {len(parts)} calls per step; warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for pt in parts:
        abi.ks_device_status(pt["ws_ptr"], pt["ws_bytes"], stream)
        if pt["db"] is not None:
            abi.ks_device_status(pt["db"].ws_ptr, pt["db"].ws_bytes, stream)
    cs = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(cs)
    for _ in range(args.steps):
        step()
    ev1.record(cs)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)

    # each call's evaluation kernel (and record writer), from HIP events the
    # library records around those launches on the stream
    reps = max(3, min(args.steps, 10))
    ev = abi.HipEvents(2 * reps * len(parts))
    try:
        k = 0
        for _ in range(reps):
            for pt in parts:
                run_part(pt, (ev.ev[k], ev.ev[k + 1]))
                k += 2
        torch.cuda.synchronize()
        for i, pt in enumerate(parts):
            pt["kernel_ms"] = sum(ev.elapsed_ms(2 * (r * len(parts) + i), 2 * (r * len(parts) + i) + 1)
                                  for r in range(reps)) / reps
        if parts[0]["db"] is not None:
            k = 0
            for _ in range(reps):
                for pt in parts:
                    abi.ks_set_timing_events(ev.ev[k], ev.ev[k + 1])
                    pt["db"].expand(stream)
                    abi.ks_set_timing_events(None, None)
                    k += 2
            torch.cuda.synchronize()
            for i, pt in enumerate(parts):
                pt["expand_ms"] = sum(ev.elapsed_ms(2 * (r * len(parts) + i), 2 * (r * len(parts) + i) + 1)
                                      for r in range(reps)) / reps
    finally:
        abi.ks_set_timing_events(None, None)
        ev.close()
    k_ms = sum(pt["kernel_ms"] for pt in parts)

    pcie = None
    if parts[0]["db"] is not None:
        pcie = _c5_upload_sweep(parts, run_part, stream, reps)

    dispatch_rows = sum(pt["rows"] for pt in parts)
    eval_rows = sum(pt["eval_rows"] for pt in parts)
    pairs = dispatch_rows * n_specs
    n_steps_total = sum(pt["n_steps"] for pt in parts)
    if args.eta_one:
        alg = sum(pt["bytes"] for pt in parts)
        bound, unit, peak, dtype = "hbm", "GB/s", PEAK["hbm"] / 1e9, "f32"
        achieved = alg / (k_ms * 1e-3) / 1e9
    else:
        alg = float(eval_rows) * n_specs * head_flops_per_pair(in_dim, hidden)
        bound, unit, peak, dtype = "mfma", "TFLOP/s", PEAK["bf16"] / 1e12, "bf16"
        achieved = alg / (k_ms * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": pairs / (ms * 1e-3), "unit": "predictions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": wdesc, "records": dispatch_rows, "evaluated_records": eval_rows,
                   "spec_vectors": n_specs, "serving_steps": n_steps_total, "calls_per_step": len(parts),
                   "predictions_per_step": pairs,
                   "head": "eta=1" if args.eta_one else f"bf16 {in_dim}-{hidden}-{hidden}-1",
                   "input": ("batch descriptors, expanded on the GPU every step" if parts[0]["db"] is not None
                             else "kernel records")},
        "step_evals_per_s": n_steps_total * n_specs / (ms * 1e-3),
        "roofline": {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                     "traffic": recorded_traffic(traffic_key(args)), "kernel_ms": k_ms,
                     "note": "achieved = algorithmic work of the sweep's evaluation-kernel launches (head "
                             "FLOPs over the records evaluated, or the bytes the model reads and writes) / "
                             "the sum of those kernels' mean durations from HIP events around each launch; "
                             "traffic = HBM bytes of those launches per sweep (counters)"},
        "calls": [{"name": pt["name"], "records": pt["rows"], "kernel_ms": pt["kernel_ms"],
                   **({"expand_ms": pt["expand_ms"]} if "expand_ms" in pt else {}),
                   **({"tp": pt["tp"]} if "tp" in pt else {})} for pt in parts],
    }
    if pcie is not None:
        out["pcie_inclusive"] = pcie
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = _sweep_cpu_baseline(args)
    print(json.dumps(out), flush=True)
    return 0


def _c5_upload_sweep(parts, run_part, stream, reps):
    """The c5 sweep with every batch's descriptors (request offsets, query
    and history tokens, prefill flags) copied from pinned host memory on a
    second stream: all uploads are queued at once, and each batch's
    expansion waits for its own upload (an event), so batch b + 1's upload
    overlaps batch b's work.  Returns the whole-sweep time and the upload
    bytes; the resident-input figure stays `value`."""
    import numpy as np
    import torch
    host = []
    nbytes = 0
    for pt in parts:
        tr = pt["trace"]
        arrs = {"req_off": np.ascontiguousarray(tr.req_off, np.uint32).view(np.int32),
                "req_q": np.ascontiguousarray(tr.req_q, np.uint32).view(np.int32),
                "req_h": np.ascontiguousarray(tr.req_h, np.uint32).view(np.int32),
                "prefill": np.ascontiguousarray(tr.prefill, np.uint8)}
        pin = {k: torch.from_numpy(v).pin_memory() for k, v in arrs.items()}
        nbytes += sum(v.numel() * v.element_size() for v in pin.values())
        host.append(pin)
    copy = torch.cuda.Stream()
    comp = torch.cuda.current_stream()
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(comp)
        copy.wait_event(e0)
        done = []
        with torch.cuda.stream(copy):
            for pt, pin in zip(parts, host):
                for k, v in pin.items():
                    pt["db"].t[k].copy_(v, non_blocking=True)
                ev = torch.cuda.Event()
                ev.record(copy)
                done.append(ev)
        for pt, ev in zip(parts, done):
            comp.wait_event(ev)
            run_part(pt)
        e1.record(comp)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return {"ms_per_sweep": sum(times) / len(times), "upload_bytes": nbytes,
            "note": "whole sweep with the batch descriptors uploaded from pinned host memory on a second "
                    "stream, overlapped with the previous batch's expansion and evaluation; not `value` "
                    "(value has the inputs resident in HBM)"}


def _sweep_cpu_baseline(args):
    """The oracle on a bounded sample of the sweep: c2, the records of the
    first 40 steps of each of the six shapes; c5, those of the first 300
    steps; every spec vector."""
    from workload import gen
    threads = args.cpu_threads or host_threads()
    if args.workload == "c2":
        wls = [gen.config2(i, 0, 40) for i in range(len(gen.DENSE_SHAPES))]
        what = "the records of steps 0..40 of each of the six shapes"
    else:
        wls = [gen.config5(0, 300)]
        what = "the records of steps 0..300"
    pairs, secs = 0, 0.0
    for wl in wls:
        r = cpu_baseline(wl, {"specs": wl.n_specs, "steps": None}, args.eta_one, threads)
        pairs += r["pairs"]
        secs += r["seconds"]
    return {"value": pairs / secs, "unit": "predictions/s", "cores": threads, "kind": "oracle",
            "os_cpu_count": os.cpu_count(),
            "sample": f"{what} x 2 spec vectors ({pairs} predictions, {secs:.1f} s, fp64 numpy, "
                      f"{threads} BLAS threads)"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=15)
    ap.add_argument("--workload", default="c4", choices=["c4", "c1", "c3", "c5-batch", "c2", "c5"],
                    help="c4: the capacity grid (default); c1; c3: the whole MoE trace in one call; c5-batch: "
                         "one 64M-record batch of the 70B trace; c2: the six dense shapes, each its whole "
                         "100k-step trace in one call; c5: the whole 500k-step 70B trace in 64M-record "
                         "batches, each expanded on the GPU from its batch descriptors and evaluated")
    ap.add_argument("--eta-one", action="store_true", help="eta = 1 (pure roofline) mode")
    ap.add_argument("--per-pair", action="store_true",
                    help="also write each pair's latency t_kernel (ks_eval_steps with per-pair outputs)")
    ap.add_argument("--kernels", action="store_true",
                    help="per-kernel latencies only: ks_eval_kernels writing t_kernel for every pair, no step sums")
    ap.add_argument("--bounded", default="none", choices=["none", "mixed", "all"],
                    help="families on the bounded analytical head: none; the GEMMs, embedding and "
                         "KV writes (mixed, the rest on the MLP or eta = 1); or all")
    ap.add_argument("--grid", default="none", choices=["none", "all"],
                    help="Tier B: a measured eta grid (8x8x8 over features x1, x2, x6, 8%% of the nodes "
                         "unmeasured) on every family, the head of the mode where a pair falls outside")
    ap.add_argument("--expand", default="none", choices=["none", "per-layer", "homogeneous"],
                    help="start from the batch descriptors: each step runs ks_expand (one record "
                         "per dispatched kernel, or layer-identical kernels as one record of "
                         "multiplicity L) and then ks_eval_steps on its records")
    ap.add_argument("--expand-only", action="store_true",
                    help="time ks_expand alone (the records are not evaluated)")
    ap.add_argument("--simulate", type=int, default=0, metavar="N",
                    help="serving simulation of N requests (Llama-7B shape, GB200 datasheet row, fp32 "
                         "16-64 heads) with the scheduler in the loop; reports simulated steps/s")
    ap.add_argument("--rate", type=float, default=40.0, help="request arrival rate of --simulate (1/s)")
    ap.add_argument("--sim-specs", type=int, default=1, metavar="S",
                    help="--simulate: S simulations in lockstep, one per spec vector (1 .. 256)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build evaluates on one GPU only (the path shards by step ranges "
              "or spec vectors with no exchange; see the design notes); run with --gpus 1",
              file=sys.stderr)
        return 2

    import torch
    from paper_2606_28565_amd import abi

    if not os.path.exists(abi.LIB_PATH):
        from paper_2606_28565_amd import build as b
        b.build()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(args.steps, 1))
        return 0

    if args.simulate:
        return _bench_simulate(args)
    if args.workload in ("c2", "c5"):
        return _bench_sweep(args)

    print(f"[bench] generating workload {args.workload}", file=sys.stderr, flush=True)
    wl, wdesc, sample, traces = _workload(args.workload)
    from workload import gen
    bmask = {"none": 0, "mixed": gen.BOUNDED_MIXED, "all": gen.BOUNDED_ALL}[args.bounded]
    bounded = gen.make_bounded(bmask) if bmask else None
    grid = gen.make_grid(gen.GRID_ALL) if args.grid == "all" else None
    di = abi.DeviceInputs(wl)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden,
                          abi.KS_ETA_ONE if args.eta_one else abi.KS_ETA_MLP, bounded, grid)
    head_pairs = None
    if grid is not None:
        # where each pair's eta comes from (one untimed call): only the pairs
        # left to the head count as its work
        src_t, src_o = abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=False, t_roof=False, eta=False,
                                          t_kernel=False, source=True)
        so0_t, so0 = abi.step_outputs(wl.desc.n_steps, di.n_specs)
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so0, src_o,
                          di.ws_ptr, di.ws_bytes, abi.current_stream())
        torch.cuda.synchronize()
        head_pairs = int((src_t["source"] == 0).sum().item())
        routed_frac = float((src_t["source"] == 2).float().mean().item())
        del src_t, so0_t
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    if args.per_pair or args.kernels:
        ko_t, ko = abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=False, t_roof=False, eta=False)
    else:
        ko = None
    stream = abi.current_stream()
    db = None
    if args.expand != "none" or args.expand_only:
        if len(traces) != 1:
            raise SystemExit("--expand needs a single-model workload (c1 or c5-batch)")
        if args.per_pair and args.expand == "homogeneous":
            raise SystemExit("--per-pair outputs follow one record per dispatch; not with --expand homogeneous")
        mode = abi.KS_EXPAND_HOMOGENEOUS if args.expand == "homogeneous" else abi.KS_EXPAND_PER_LAYER
        db = abi.DeviceBatch(traces[0], mode)
        ews = torch.empty(abi.ks_workspace_bytes(db.desc, di.n_specs) + 256, dtype=torch.uint8,
                          device="cuda")
        ews_ptr = ews.data_ptr() + (-ews.data_ptr()) % 256
        ews_bytes = abi.ks_workspace_bytes(db.desc, di.n_specs)

    def step():
        if db is not None:
            db.expand(stream)
            if args.expand_only:
                return
            abi.ks_eval_steps(db.desc, db.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                              ews_ptr, ews_bytes, stream)
            return
        if args.kernels:
            abi.ks_eval_kernels(di.desc, di.specs_ptr, di.n_specs, heads, ko, di.ws_ptr, di.ws_bytes, stream)
            return
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                          di.ws_ptr, di.ws_bytes, stream)

    def kernel_ms(n: int) -> float:
        """Mean duration of the call's main kernel (the evaluation kernel, or
        the expansion's record writer with --expand-only) over n calls, from
        HIP events the library records around that launch on the stream."""
        ev = abi.HipEvents(2 * n)
        try:
            for i in range(n):
                if db is not None and not args.expand_only:
                    db.expand(stream)       # untimed: the hook brackets the evaluation kernel
                    abi.ks_set_timing_events(ev.ev[2 * i], ev.ev[2 * i + 1])
                    abi.ks_eval_steps(db.desc, db.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                                      ews_ptr, ews_bytes, stream)
                else:
                    abi.ks_set_timing_events(ev.ev[2 * i], ev.ev[2 * i + 1])
                    step()
                abi.ks_set_timing_events(None, None)
            abi.ks_set_timing_events(None, None)
            torch.cuda.synchronize()
            return sum(ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n
        finally:
            abi.ks_set_timing_events(None, None)
            ev.close()

    def expand_kernel_ms(n: int) -> float:
        ev = abi.HipEvents(2 * n)
        try:
            for i in range(n):
                abi.ks_set_timing_events(ev.ev[2 * i], ev.ev[2 * i + 1])
                db.expand(stream)
            abi.ks_set_timing_events(None, None)
            torch.cuda.synchronize()
            return sum(ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(n)) / n
        finally:
            abi.ks_set_timing_events(None, None)
            ev.close()

    print(f"[bench] {wl.desc.n_rows} records x {di.n_specs} specs; warmup {args.warmup}",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    abi.ks_device_status(di.ws_ptr, di.ws_bytes, stream)
    cs = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(cs)
    for _ in range(args.steps):
        step()
    ev1.record(cs)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    print(f"[bench] {args.steps} steps: {ms:.3f} ms/step", file=sys.stderr, flush=True)
    if db is not None:
        abi.ks_device_status(db.ws_ptr, db.ws_bytes, stream)
    # the main kernel alone, in a second pass of as many calls (the timed
    # region above has no extra event records)
    k_ms = kernel_ms(args.steps)
    print(f"[bench] main kernel: {k_ms:.3f} ms/launch", file=sys.stderr, flush=True)

    if args.expand_only:
        return _print_expand_only(args, wl, wdesc, db, ms, k_ms)
    exp = None
    if db is not None:
        e_ms = expand_kernel_ms(args.steps)
        hom = args.expand == "homogeneous"
        eb = expand_bytes(db.fam_off[-1], db.desc.n_steps, hom)
        exp = {"form": args.expand, "records": db.fam_off[-1], "records_kernel_ms": e_ms,
               "roofline": {"bound": "hbm", "achieved": eb / (e_ms * 1e-3) / 1e9, "peak": PEAK["hbm"] / 1e9,
                            "unit": "GB/s", "frac": eb / (e_ms * 1e-3) / PEAK["hbm"], "traffic": None}}
    pairs = wl.desc.n_rows * di.n_specs
    value = pairs / (ms * 1e-3)
    step_evals = wl.desc.n_steps * di.n_specs / (ms * 1e-3)
    # records on the MLP: the families outside the bounded mask
    import numpy as np
    on_mlp = ((bmask >> wl.desc.family()) & 1) == 0
    eval_desc = db.desc if db is not None else None
    if db is not None and args.expand == "homogeneous":
        # the evaluation sees the homogeneous records (one per layer-identical
        # kernel): its work is per record, while value counts dispatches
        n_eval = db.fam_off[-1]
        on_mlp_n = n_eval - sum(db.fam_off[f + 1] - db.fam_off[f] for f in range(gen.NFAM) if (bmask >> f) & 1)
    else:
        n_eval = wl.desc.n_rows
        on_mlp_n = int(np.count_nonzero(on_mlp))
    mlp_pairs = on_mlp_n * di.n_specs if head_pairs is None else head_pairs
    if args.eta_one or bmask == gen.BOUNDED_ALL:
        alg = (stream_bytes(wl, di.n_specs, sums=not args.kernels,
                            pair_outputs=1 if (args.per_pair or args.kernels) else 0)
               if eval_desc is None or args.expand != "homogeneous" else None)
        bound, unit, peak = "hbm", "GB/s", PEAK["hbm"] / 1e9
        achieved = alg / (k_ms * 1e-3) / 1e9 if alg is not None else None
        dtype = "f32"
    else:
        per_pair = head_flops_per_pair(wl.heads.in_dim, wl.heads.hidden)
        alg = float(mlp_pairs) * per_pair
        bf16 = wl.heads.precision == "bf16"
        bound, unit = "mfma", "TFLOP/s"
        peak = (PEAK["bf16"] if bf16 else PEAK["f32"]) / 1e12
        achieved = alg / (k_ms * 1e-3) / 1e12
        dtype = "bf16" if bf16 else "f32"

    out = {
        "metric": METRIC, "value": value, "unit": "predictions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic",
        "config": {"workload": wdesc, "records": wl.desc.n_rows, "spec_vectors": di.n_specs,
                   "serving_steps": wl.desc.n_steps, "predictions_per_step": pairs,
                   "head": ("eta=1" if args.eta_one else
                            f"{wl.heads.precision} {wl.heads.in_dim}-{wl.heads.hidden}-{wl.heads.hidden}-1")
                           + ("" if not bmask else f"; bounded head on families 0x{bmask:03x}")
                           + ("" if grid is None else f"; Tier B grid on every family, {100 * routed_frac:.1f}% of "
                                                      f"the pairs routed to it"),
                   "per_pair_outputs": bool(args.per_pair or args.kernels),
                   "step_sums": not args.kernels,
                   "input": ("batch descriptors, expanded on the GPU every step ("
                             + args.expand + " records)") if db is not None else "kernel records"},
        "step_evals_per_s": step_evals,
        "roofline": {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": achieved / peak if achieved is not None else None,
                     "traffic": recorded_traffic(traffic_key(args)),
                     "kernel_ms": k_ms, "evaluated_records": n_eval,
                     "note": "achieved = algorithmic work of one evaluation-kernel launch (FLOPs of the "
                             "head over the records it evaluates, or the bytes the model reads and "
                             "writes) / that kernel's mean duration from HIP events recorded around "
                             "its launch on the call's stream"},
    }
    if exp is not None:
        out["expand"] = exp
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or host_threads()
        print(f"[bench] cpu baseline: oracle on {sample}, {threads} threads", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, sample, args.eta_one, threads, bounded, grid)
        try:
            model = subprocess.run(["lscpu"], capture_output=True, text=True).stdout
            model = [l.split(":", 1)[1].strip() for l in model.splitlines() if l.startswith("Model name")]
            out["cpu_baseline"]["cpu_model"] = model[0] if model else platform.processor()
        except OSError:
            pass
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
