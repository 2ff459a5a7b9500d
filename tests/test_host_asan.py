"""The library's host code (argument checks, workspace layouts, the batch
expansion's plan, the serving simulator's scheduler) built with g++ under
AddressSanitizer and UndefinedBehaviorSanitizer and run on the CPU, the
launches replaced by host stand-ins (tests/host/fake_device.cpp).

* Argument checks: every entry point's status on valid and invalid calls
  (null pointers, inconsistent family offsets, bad heads, grids, workspace
  size and alignment, models the expansion refuses, unsorted or empty
  requests) as the header documents them.
* Scheduler: with a stand-in step latency (a function of the step's query
  tokens, its prefill flag and the spec index, computed alike on both
  sides), the library's simulator and the oracle's scheduler (Sec. 4.1-4.2,
  5.8) form the same batches at the same clock and give the same
  per-request metrics, bit for bit, under KV pressure with preemption,
  prefix caching with eviction, and several simulations in lockstep.

A sanitizer report aborts the driver (nonzero exit), which fails the test."""
from __future__ import annotations

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import ks_sim as osim
from workload import gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_28565_amd", "csrc")
HOST = os.path.join(ROOT, "tests", "host")
ROCM_INCLUDE = "/opt/rocm/include"

SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=1:halt_on_error=1",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.isdir(ROCM_INCLUDE):
        pytest.skip("g++ or the HIP runtime headers are not available")
    exe = str(tmp_path_factory.mktemp("host") / "ks_host_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-ffp-contract=off",
           "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE, "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "ks_api.cpp"), os.path.join(CSRC, "ks_sim.cpp"),
           os.path.join(HOST, "fake_device.cpp"), os.path.join(HOST, "host_driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return exe


def _run(exe, mode, stdin=""):
    env = dict(os.environ, **SAN_ENV)
    r = subprocess.run([exe, mode], input=stdin, capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.returncode, r.stderr[-4000:])
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-4000:]
    return r.stdout


KS_OK, KS_EINVAL, KS_ERANGE, KS_EHIP, KS_EWORKSPACE = 0, 1, 2, 3, 4

EXPECTED = {
    "workspace_bytes_positive": 0, "workspace_bytes_null": 0,
    "eval_steps_valid": KS_OK, "eval_kernels_valid": KS_OK, "eval_kernels_null_out": KS_EINVAL,
    "validate_valid": KS_OK, "device_status_small_ws": KS_EWORKSPACE,
    "eval_steps_null_desc": KS_EINVAL, "fam_off_decreasing": KS_EINVAL, "fam_off_end_mismatch": KS_EINVAL,
    "n_rows_negative": KS_ERANGE, "record_array_null": KS_EINVAL, "elem_bytes_zero": KS_ERANGE,
    "n_specs_zero": KS_EINVAL, "specs_null": KS_EINVAL, "ws_null": KS_EWORKSPACE, "ws_small": KS_EWORKSPACE,
    "ws_misaligned": KS_EWORKSPACE, "heads_mode_unknown": KS_EINVAL, "heads_in_dim_17": KS_EINVAL,
    "heads_bf16_hidden_96": KS_EINVAL, "heads_weight_null": KS_EINVAL, "heads_bf16_16_128_valid": KS_OK,
    "bounded_mask_beyond": KS_EINVAL, "bounded_null": KS_EINVAL, "grid_valid": KS_OK, "grid_n_1": KS_EINVAL,
    "grid_empty_range": KS_EINVAL, "grid_axis_15": KS_EINVAL, "grid_too_many_nodes": KS_EINVAL,
    "steps_count_mismatch": KS_EINVAL, "steps_array_null": KS_EINVAL, "host_null": KS_EINVAL,
    "step_out_null": KS_EINVAL, "empty_call": KS_OK,
    "expand_layout_valid": KS_OK, "expand_layout_homogeneous": KS_OK, "expand_layout_null_fam_off": KS_EINVAL,
    "expand_layout_prefill_gt_steps": KS_EINVAL, "expand_layout_mode_unknown": KS_EINVAL,
    "expand_layout_hidden_0": KS_EINVAL, "expand_layout_tp_not_dividing": KS_EINVAL,
    "expand_layout_top_k_above_experts": KS_EINVAL, "expand_layout_moe_valid": KS_OK,
    "expand_layout_n_too_wide": KS_ERANGE, "expand_ws_negative": 0,
    "expand_valid": KS_OK, "expand_ws_small": KS_EWORKSPACE, "expand_batch_null": KS_EINVAL,
    "expand_n_prefill_above_steps": KS_EINVAL,
    "simulate_unsorted_arrivals": KS_EINVAL, "simulate_zero_prompt": KS_ERANGE, "simulate_n_specs_0": KS_EINVAL,
    "simulate_moe_rejected": KS_EINVAL, "simulate_block_tokens_0": KS_EINVAL, "simulate_ws_small": KS_EWORKSPACE,
    "simulate_group_without_prefix": KS_EINVAL, "simulate_valid": KS_OK,
    # 10 steps of a 4-layer dense decoder: 9 kernels per layer plus the
    # embedding and the LM head per step; the homogeneous form keeps one
    # record per layer-identical kernel; the mixture of experts has 10
    # kernels per layer
    "expand_layout_records": 10 * (9 * 4 + 2), "expand_layout_homogeneous_records": 10 * (9 + 2),
    "expand_layout_moe_records": 10 * (10 * 4 + 2),
}


def test_host_argument_checks(driver):
    out = _run(driver, "args")
    got = {}
    for line in out.splitlines():
        name, val = line.split()
        assert val != "empty-message", f"{name}: failing status without a message"
        got[name] = int(val)
    missing = set(EXPECTED) - set(got)
    assert not missing, missing
    for k, v in EXPECTED.items():
        assert got[k] == v, (k, got[k], v)
    assert got["simulate_valid_steps"] > 0


def stand_in_latency(spec_index):
    """The host stand-in's step latency for simulation `spec_index`, in the
    same order of operations."""
    def lat(batch, prefill):
        q = sum(b[0] for b in batch)
        t = 1e-3 + 2e-7 * float(q)
        t += 1e-4 * float(spec_index)
        t += 5e-4 * (1.0 if prefill else 0.0)
        return t
    return lat


SMALL_MODEL = (512, 4, 8, 8, 64, 1376, 32000, 1)   # hidden, layers, heads, kv heads, head dim, ffn, vocab, tp

# (scheduler, simulations, requests, arrival rate)
CASES = {
    "roomy": (osim.SchedCfg(max_num_seqs=64, max_batched_tokens=2048, block_tokens=16, kv_blocks=8192), 1, 80, 50.0),
    # KV pressure (a burst of arrivals): preemption by recompute and prefix eviction
    "tight": (osim.SchedCfg(max_num_seqs=32, max_batched_tokens=1024, block_tokens=16, kv_blocks=300), 1, 80,
              5000.0),
    "noprefix": (osim.SchedCfg(max_num_seqs=16, max_batched_tokens=512, block_tokens=16, kv_blocks=8192,
                               prefix_cache=False), 1, 60, 200.0),
    # three simulations in lockstep, each under its own latency
    "lockstep": (osim.SchedCfg(max_num_seqs=32, max_batched_tokens=1024, block_tokens=32, kv_blocks=400), 3, 60,
                 2000.0),
}


def _parse_sim(out):
    lines = out.splitlines()
    assert lines[0].split()[:2] == ["status", "0"], lines[0]
    sims, cur = [], None
    for line in lines[1:]:
        t = line.split()
        if t[0] == "sim":
            cur = {"n_steps": int(t[2]), "preemptions": int(t[3]), "clock": float.fromhex(t[4]), "steps": [],
                   "req": []}
            sims.append(cur)
        elif t[0] == "step":
            entries = [tuple(int(v) for v in e.split(":")) for e in t[4:]]
            cur["steps"].append((float.fromhex(t[1]), float.fromhex(t[2]), bool(int(t[3])), entries))
        else:
            cur["req"].append((int(t[1]), float.fromhex(t[2]), float.fromhex(t[3]), float.fromhex(t[4])))
    return sims


@pytest.mark.parametrize("case", list(CASES))
def test_host_simulator_matches_oracle_scheduler(driver, case):
    cfg, n_specs, n_req, rate = CASES[case]
    reqs = gen.make_requests(n_req, rate=rate, seed=31 + n_req, prompt_median=320, output_median=40,
                             prefix_lo=64, prefix_hi=512)
    lines = [" ".join(str(v) for v in SMALL_MODEL),
             f"{cfg.max_num_seqs} {cfg.max_batched_tokens} {cfg.block_tokens} {int(cfg.prefix_cache)} "
             f"{cfg.kv_blocks}", f"{n_specs} {n_req}"]
    for i in range(n_req):
        lines.append(f"{float(reqs['arrival'][i]).hex()} {int(reqs['prompt'][i])} {int(reqs['output'][i])} "
                     f"{int(reqs['group'][i])} {int(reqs['prefix'][i])}")
    sims = _parse_sim(_run(driver, "sim", "\n".join(lines) + "\n"))
    assert len(sims) == n_specs
    as_list = [{k: (float(reqs[k][i]) if k == "arrival" else int(reqs[k][i])) for k in reqs} for i in range(n_req)]
    for s, got in enumerate(sims):
        ref = osim.simulate(as_list, cfg, stand_in_latency(s))
        assert got["n_steps"] == len(ref.steps) and got["n_steps"] == len(got["steps"])
        assert got["preemptions"] == ref.preemptions
        for i, (g, r) in enumerate(zip(got["steps"], ref.steps)):
            start, latency, prefill, entries = g
            assert start == r[0], (s, i)
            assert latency == r[1], (s, i)
            assert entries == [tuple(e) for e in r[2]], (s, i)
            assert prefill == r[3], (s, i)
        assert [x[0] for x in got["req"]] == list(ref.state)
        np.testing.assert_array_equal([x[1] for x in got["req"]], ref.ttft)
        np.testing.assert_array_equal([x[2] for x in got["req"]], ref.tpot)
        np.testing.assert_array_equal([x[3] for x in got["req"]], ref.e2e)
    if case in ("tight", "lockstep"):
        assert sims[0]["preemptions"] > 0
