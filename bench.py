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
    import hashlib
    h = hashlib.sha256()
    for f in ("ks_kernels.hip", "ks_expand.hip", "ks_internal.h"):
        with open(os.path.join(ROOT, "paper_2606_28565_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
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


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=15)
    ap.add_argument("--workload", default="c4", choices=["c4", "c1", "c5-batch"])
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
                     "traffic": (recorded_traffic(f"{args.workload}{'-eta1' if args.eta_one else ''}"
                                                  f"{'-kernels' if args.kernels else ('-pair' if args.per_pair else '')}")
                                 if not bmask and db is None and grid is None else None),
                     "kernel_ms": k_ms, "evaluated_records": n_eval,
                     "note": "achieved = algorithmic work of one evaluation-kernel launch (FLOPs of the "
                             "head over the records it evaluates, or the bytes the model reads and "
                             "writes) / that kernel's mean duration from HIP events recorded around "
                             "its launch on the call's stream"},
    }
    if exp is not None:
        out["expand"] = exp
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
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
