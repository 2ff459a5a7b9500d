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
    """(workload, description, oracle sample) for each benchmark workload.
    The oracle sample bounds the CPU baseline to ~10-30 s of work."""
    from workload import gen
    if name == "c4":
        return (gen.config4(), "c4-capacity-grid: llama-7b c1 trace + S2 trace prefix, 256 specs",
                {"specs": 16, "steps": None})
    if name == "c1":
        return gen.config1(), "c1-llama7b: 1000 steps, 2 datasheet specs, fp32 heads", {"specs": 2, "steps": None}
    if name == "c5-batch":
        wl = gen.config5(0, C5_BATCH_STEPS)
        return (wl, f"c5-70b-prefix: one 64M-record batch (steps 0..{C5_BATCH_STEPS}), 2 datasheet specs, "
                    "bf16 32-256-256 heads", {"specs": 2, "steps": 300})
    raise SystemExit(f"unknown workload {name}")


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ("ks_kernels.hip", "ks_internal.h"):
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


def stream_bytes(wl, n_specs: int) -> float:
    """Algorithmic HBM bytes of one evaluation-kernel launch: the record
    fields each family uses, the per-expert row counts of grouped records,
    the per-step attention work (4 x u64 per step), and the writes: one
    range (2 x u32) per (family, step) and one fp64 partial per (spec,
    family, step)."""
    import numpy as np
    d = wl.desc
    rows = np.diff(d.fam_off)
    b = float(sum(int(rows[f]) * 4 * FIELDS_USED[f] for f in range(len(rows))))
    g0, g1 = int(d.fam_off[2]), int(d.fam_off[3])
    b += 4.0 * float(d.a[g0:g1].astype(np.int64).sum())
    b += 32.0 * d.n_steps
    segs = sum(len(np.unique(d.step[d.fam_off[f]:d.fam_off[f + 1]])) for f in range(len(rows)))
    b += segs * (8.0 + 8.0 * n_specs)
    return b


def head_flops_per_pair(in_dim: int, hidden: int) -> int:
    """Algorithmic MLP FLOPs of one prediction: 2 (in h + h h + h)."""
    return 2 * (in_dim * hidden + hidden * hidden + hidden)


def cpu_baseline(wl, sample: dict, eta_one: bool, threads: int, bounded=None):
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
                           spec_ids=spec_ids, rows=rows, bounded=bounded)
        if rows is None:
            o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, spec_ids=spec_ids, kern=k)
        dt = time.perf_counter() - t
    n = wl.desc.n_rows if rows is None else len(rows)
    pairs = n * len(spec_ids)
    what = f"all {n} records" if rows is None else f"the {n} records of steps 0..{sample['steps']}"
    return {"value": pairs / dt, "unit": "predictions/s", "cores": threads, "kind": "oracle",
            "sample": f"{what} x {len(spec_ids)} of {wl.n_specs} spec vectors "
                      f"({pairs} predictions, {dt:.1f} s, fp64 numpy, {threads} BLAS threads)"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=15)
    ap.add_argument("--workload", default="c4", choices=["c4", "c1", "c5-batch"])
    ap.add_argument("--eta-one", action="store_true", help="eta = 1 (pure roofline) mode")
    ap.add_argument("--per-pair", action="store_true", help="also write per-pair t_roof/eta/t_kernel")
    ap.add_argument("--bounded", default="none", choices=["none", "mixed", "all"],
                    help="families on the bounded analytical head: none; the GEMMs, embedding and "
                         "KV writes (mixed, the rest on the MLP or eta = 1); or all")
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

    print(f"[bench] generating workload {args.workload}", file=sys.stderr, flush=True)
    wl, wdesc, sample = _workload(args.workload)
    from workload import gen
    bmask = {"none": 0, "mixed": gen.BOUNDED_MIXED, "all": gen.BOUNDED_ALL}[args.bounded]
    bounded = gen.make_bounded(bmask) if bmask else None
    di = abi.DeviceInputs(wl)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden,
                          abi.KS_ETA_ONE if args.eta_one else abi.KS_ETA_MLP, bounded)
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    if args.per_pair:
        ko_t, ko = abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=False)
    else:
        ko = None
    stream = abi.current_stream()

    def step():
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                          di.ws_ptr, di.ws_bytes, stream)

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

    pairs = wl.desc.n_rows * di.n_specs
    value = pairs / (ms * 1e-3)
    step_evals = wl.desc.n_steps * di.n_specs / (ms * 1e-3)
    # records on the MLP: the families outside the bounded mask
    import numpy as np
    on_mlp = ((bmask >> wl.desc.family()) & 1) == 0
    if args.eta_one or bmask == gen.BOUNDED_ALL:
        alg = stream_bytes(wl, di.n_specs)
        bound, unit, peak = "hbm", "GB/s", PEAK["hbm"] / 1e9
        achieved = alg / (ms * 1e-3) / 1e9
        dtype = "f32"
    else:
        per_pair = head_flops_per_pair(wl.heads.in_dim, wl.heads.hidden)
        alg = float(int(np.count_nonzero(on_mlp)) * di.n_specs) * per_pair
        bf16 = wl.heads.precision == "bf16"
        bound, unit = "mfma", "TFLOP/s"
        peak = (PEAK["bf16"] if bf16 else PEAK["f32"]) / 1e12
        achieved = alg / (ms * 1e-3) / 1e12
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
                           + ("" if not bmask else f"; bounded head on families 0x{bmask:03x}"),
                   "per_pair_outputs": bool(args.per_pair)},
        "step_evals_per_s": step_evals,
        "roofline": {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": achieved / peak,
                     "traffic": (recorded_traffic(f"{args.workload}{'-eta1' if args.eta_one else ''}")
                                 if not bmask else None),
                     "note": "achieved = algorithmic work of the evaluation kernel per call "
                             "(FLOPs of the head, or the bytes the model reads and writes) / HIP-event "
                             "time of the whole call (all of its kernels)"},
    }
    if not args.no_cpu_baseline:
        threads = args.cpu_threads or min(16, os.cpu_count() or 1)
        print(f"[bench] cpu baseline: oracle on {sample}, {threads} threads", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, sample, args.eta_one, threads, bounded)
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
