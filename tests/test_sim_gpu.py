"""Parity of the serving simulation (ks_simulate, through the C ABI) with
the oracle's scheduler and latency model.

* Replay: the oracle's scheduler, fed the GPU run's step latencies in
  order, must form exactly the batches the GPU run recorded (requests,
  q, h, prefill flag) and give the same per-request metrics bit for bit
  (both add the same fp64 latencies to the clock in the same order).
* Latency: each recorded step's latency against the oracle model of that
  batch: 1e-5 relative (eta = 1, fp32 heads), 1e-2 (bf16 heads).
* End to end: the oracle's scheduler with the oracle model against the GPU
  run: metrics within 1e-5 relative (eta = 1, fp32 heads), when no
  scheduling decision sits within rounding of a tie (asserted by the
  replay matching first).
* Lockstep: several simulations (one per spec vector) priced together each
  round; every one replays exactly against the oracle's scheduler, its
  latencies follow the oracle model under its own spec vector, and they
  agree with a lone run of the same spec to the rounding order of the
  per-step sums."""
import numpy as np
import pytest
import torch  # noqa: F401

from oracle import ks_expand as ox
from oracle import ks_oracle as o
from oracle import ks_sim as osim
from workload import gen
from paper_2606_28565_amd import abi

pytestmark = pytest.mark.gpu

u32 = lambda x: np.asarray(x, np.uint32)


def spec_row(i=0):
    s = gen.specs_datasheet()
    return {k: (int(v[i]) if k == "n_cu" else float(v[i])) for k, v in s.items()}


def one_spec(i=0):
    return {k: np.asarray([v]) for k, v in spec_row(i).items()}


def device_heads(kind):
    """(ks_heads, keep-alive tensors, gen.Heads or None, eta_one)"""
    hd = abi.ks_heads()
    if kind == "eta1":
        hd.mode = abi.KS_ETA_ONE
        return hd, {}, None, True
    h = gen.make_heads(16, 64, "f32") if kind == "f32" else gen.make_heads(16, 128, "bf16")
    keep = {}
    hd.in_dim, hd.hidden = h.in_dim, h.hidden
    hd.precision = abi.KS_BF16 if h.precision == "bf16" else abi.KS_F32
    hd.mode = abi.KS_ETA_MLP
    for name in ("w1", "w2", "b2", "w3", "b3"):
        arr = np.ascontiguousarray(h.storage[name])
        arr = arr.view(np.int16) if arr.dtype == np.uint16 else arr
        keep[name] = torch.from_numpy(arr.reshape(-1).copy()).cuda()
        setattr(hd, name, keep[name].data_ptr())
    return hd, keep, h, False


def host_struct():
    hc = gen.HostConsts()
    return abi.ks_host(hc.c_disp, hc.ell, hc.c_ovl, hc.c_tail, hc.body_scale)


def sched_struct(cfg):
    return abi.ks_sched(cfg.max_num_seqs, cfg.max_batched_tokens, cfg.block_tokens, int(cfg.prefix_cache),
                        cfg.kv_blocks)


def oracle_latency(shape, heads, eta_one, spec_i=0, table=None):
    specs = one_spec(spec_i) if table is None else {k: np.asarray(v)[spec_i:spec_i + 1] for k, v in table.items()}
    hostc = gen.HostConsts()

    def f(batch, prefill):
        q = [b[0] for b in batch]
        h = [b[1] for b in batch]
        e = ox.expand(shape, [0, len(q)], q, [prefill], homogeneous=True)
        d = gen.Desc(e["fam_off"], *(u32(e[k]) for k in ("step", "m", "n", "k", "a", "b")),
                     u32([0, len(q)]), u32(q), u32(h), u32([]), 2, u32(e["mult"]))
        rec = gen.StepRec(*(u32(e[k]) for k in ("layers", "hidden", "tp", "n_launch")))
        return float(o.eval_steps(d, rec, specs, hostc, heads, eta_one)["t_step"][0, 0])
    return f


def as_list(reqs):
    return [{k: (float(reqs[k][i]) if k == "arrival" else int(reqs[k][i])) for k in reqs}
            for i in range(len(reqs["arrival"]))]


def run_gpu(shape, reqs, cfg, kind, spec_i=0):
    hd, keep, h, eta_one = device_heads(kind)
    res = abi.simulate(shape, spec_row(spec_i), hd, host_struct(), sched_struct(cfg), reqs)
    return res, h, eta_one


def gpu_steps(res):
    off = res["step_entry_off"]
    return [[(int(res["entry_req"][j]), int(res["entry_q"][j]), int(res["entry_h"][j]))
             for j in range(off[i], off[i + 1])] for i in range(res["n_steps"])]


def replay(reqs, cfg, res):
    """The oracle's scheduler driven by the GPU run's latencies; asserts the
    same batch at every step."""
    steps = gpu_steps(res)
    it = iter(range(res["n_steps"]))

    def lat(batch, prefill):
        i = next(it)
        assert [(q, h) for (_, q, h) in steps[i]] == list(batch), f"step {i} differs"
        assert bool(res["step_prefill"][i]) == prefill, f"step {i} prefill flag"
        return float(res["step_latency"][i])
    r = osim.simulate(as_list(reqs), cfg, lat)
    assert len(r.steps) == res["n_steps"]
    for i, s in enumerate(r.steps):
        assert s[2] == steps[i], f"step {i} requests"
        assert s[0] == res["step_start"][i]
    return r


CFGS = {
    "roomy": osim.SchedCfg(max_num_seqs=64, max_batched_tokens=2048, block_tokens=16, kv_blocks=8192),
    "tight": osim.SchedCfg(max_num_seqs=32, max_batched_tokens=1024, block_tokens=16, kv_blocks=700),
    "noprefix": osim.SchedCfg(max_num_seqs=32, max_batched_tokens=512, block_tokens=16, kv_blocks=8192,
                              prefix_cache=False),
}


@pytest.mark.parametrize("kind", ["eta1", "f32", "bf16"])
@pytest.mark.parametrize("cfg_name", list(CFGS))
def test_replay_and_step_latencies(cfg_name, kind):
    cfg = CFGS[cfg_name]
    reqs = gen.make_requests(60, rate=40.0, seed=11, prompt_median=384, output_median=48)
    res, h, eta_one = run_gpu(gen.LLAMA7B, reqs, cfg, kind)
    assert res["n_steps"] > 0 and (res["state"] == osim.FINISHED).all()
    r = replay(reqs, cfg, res)
    np.testing.assert_array_equal(res["ttft"], r.ttft)
    np.testing.assert_array_equal(res["tpot"], r.tpot)
    np.testing.assert_array_equal(res["e2e"], r.e2e)
    assert res["preemptions"] == r.preemptions
    if cfg_name == "tight":
        assert res["preemptions"] > 0
    # every step's latency against the oracle model of its batch
    f = oracle_latency(gen.LLAMA7B, h, eta_one)
    tol = 1e-2 if kind == "bf16" else 1e-5
    steps = gpu_steps(res)
    idx = np.unique(np.linspace(0, res["n_steps"] - 1, 40).astype(int))
    for i in idx:
        want = f([(q, hh) for (_, q, hh) in steps[i]], bool(res["step_prefill"][i]))
        assert abs(res["step_latency"][i] - want) <= tol * want, (i, res["step_latency"][i], want)


@pytest.mark.parametrize("kind", ["eta1", "f32"])
def test_end_to_end_against_the_oracle(kind):
    cfg = CFGS["tight"]
    reqs = gen.make_requests(40, rate=30.0, seed=12, prompt_median=256, output_median=32)
    res, h, eta_one = run_gpu(gen.LLAMA7B, reqs, cfg, kind)
    r = osim.simulate(as_list(reqs), cfg, oracle_latency(gen.LLAMA7B, h, eta_one))
    assert len(r.steps) == res["n_steps"]
    for key in ("ttft", "tpot", "e2e"):
        got, want = np.asarray(res[key]), np.asarray(getattr(r, key))
        np.testing.assert_allclose(got, want, rtol=1e-5, atol=0, err_msg=key)
    thr_gpu = sum(int(x) for x in reqs["output"]) / (max(res["e2e"] + reqs["arrival"]) - reqs["arrival"][0])
    assert thr_gpu == pytest.approx(osim.throughput(as_list(reqs), r), rel=1e-5)


def test_tensor_parallel_shape_and_second_spec():
    # a TP-4 shard with its all-reduce term, on the H100 row of the table
    cfg = CFGS["roomy"]
    reqs = gen.make_requests(30, rate=20.0, seed=13, prompt_median=300, output_median=24)
    shape = gen.DENSE_SHAPES[3]
    res, h, eta_one = run_gpu(shape, reqs, cfg, "eta1", spec_i=1)
    replay(reqs, cfg, res)
    f = oracle_latency(shape, None, True, spec_i=1)
    steps = gpu_steps(res)
    for i in range(0, res["n_steps"], max(1, res["n_steps"] // 20)):
        want = f([(q, hh) for (_, q, hh) in steps[i]], bool(res["step_prefill"][i]))
        assert abs(res["step_latency"][i] - want) <= 1e-5 * want


def test_degenerate_runs():
    cfg = osim.SchedCfg(max_num_seqs=4, max_batched_tokens=64, block_tokens=16, kv_blocks=8)
    empty = {"arrival": np.zeros(0), "prompt": u32([]), "output": u32([])}
    res, _, _ = run_gpu(gen.LLAMA7B, empty, cfg, "eta1")
    assert res["n_steps"] == 0 and res["clock"] == 0.0
    # one request that can never fit the cache, one that runs alone
    reqs = {"arrival": np.array([0.0, 0.1]), "prompt": u32([200, 20]), "output": u32([1, 3])}
    res, _, _ = run_gpu(gen.LLAMA7B, reqs, cfg, "eta1")
    assert list(res["state"]) == [osim.REJECTED, osim.FINISHED]
    assert res["ttft"][0] == 0.0 and res["e2e"][1] > 0
    replay(reqs, cfg, res)


def test_prefix_cache_saves_prefill_tokens():
    reqs = gen.make_requests(50, rate=25.0, seed=14, prompt_median=200, output_median=16, group_frac=0.9)
    on = run_gpu(gen.LLAMA7B, reqs, CFGS["roomy"], "eta1")[0]
    off_cfg = osim.SchedCfg(max_num_seqs=64, max_batched_tokens=2048, block_tokens=16, kv_blocks=8192,
                            prefix_cache=False)
    off = run_gpu(gen.LLAMA7B, reqs, off_cfg, "eta1")[0]
    assert on["entry_q"].sum() < off["entry_q"].sum()
    assert np.median(on["ttft"]) <= np.median(off["ttft"])


def _lockstep(kind, cfg, reqs, table, shape=gen.LLAMA7B):
    hd, keep, h, eta_one = device_heads(kind)
    many = abi.simulate_many(shape, table, hd, host_struct(), sched_struct(cfg), reqs)
    return many, hd, keep, h, eta_one


def _rows(table, rows):
    return {k: np.asarray(v)[rows] for k, v in table.items()}


@pytest.mark.parametrize("kind", ["eta1", "bf16"])
def test_lockstep_simulations_each_follow_their_own_spec(kind):
    # six hypothetical GPUs of the capacity-planning grid and the two
    # datasheet rows, all fed the same requests
    cfg = CFGS["tight"]
    reqs = gen.make_requests(50, rate=35.0, seed=15, prompt_median=320, output_median=40)
    grid, ds = gen.specs_grid(6, 7), gen.specs_datasheet()
    table = {k: np.concatenate([np.asarray(grid[k]), np.asarray(ds[k])]) for k in ds}
    many, hd, keep, h, eta_one = _lockstep(kind, cfg, reqs, table)
    assert len(many) == 8
    tol = 1e-2 if kind == "bf16" else 1e-5
    for i, res in enumerate(many):
        assert res["n_steps"] > 0 and (res["state"] == osim.FINISHED).all()
        r = replay(reqs, cfg, res)
        np.testing.assert_array_equal(res["ttft"], r.ttft)
        np.testing.assert_array_equal(res["e2e"], r.e2e)
        f = oracle_latency(gen.LLAMA7B, h, eta_one, spec_i=i, table=table)
        steps = gpu_steps(res)
        for j in np.unique(np.linspace(0, res["n_steps"] - 1, 12).astype(int)):
            want = f([(q, hh) for (_, q, hh) in steps[j]], bool(res["step_prefill"][j]))
            assert abs(res["step_latency"][j] - want) <= tol * want, (i, j, res["step_latency"][j], want)
    # the spec vectors differ, so the runs do: distinct clocks and step counts
    assert len({res["clock"] for res in many}) == len(many)
    assert len({res["n_steps"] for res in many}) > 1


def test_lockstep_agrees_with_lone_runs():
    cfg = CFGS["roomy"]
    reqs = gen.make_requests(40, rate=30.0, seed=16, prompt_median=256, output_median=32)
    table = gen.specs_grid(3, 8)
    many, hd, keep, h, eta_one = _lockstep("f32", cfg, reqs, table)
    for i, res in enumerate(many):
        lone = abi.simulate_many(gen.LLAMA7B, _rows(table, [i]), hd, host_struct(), sched_struct(cfg), reqs)[0]
        assert lone["n_steps"] == res["n_steps"]
        np.testing.assert_array_equal(lone["entry_q"], res["entry_q"])
        np.testing.assert_array_equal(lone["entry_h"], res["entry_h"])
        np.testing.assert_allclose(res["step_latency"], lone["step_latency"], rtol=1e-6, atol=0)
        np.testing.assert_allclose(res["e2e"], lone["e2e"], rtol=1e-6, atol=0)


def test_lockstep_with_a_repeated_spec_and_an_empty_run():
    # the same spec twice gives the same schedule twice, with latencies equal
    # up to where each step sits in the round's batch (the rounding order of
    # its sums); no requests leaves every simulation empty
    cfg = CFGS["noprefix"]
    reqs = gen.make_requests(20, rate=20.0, seed=17, prompt_median=128, output_median=16)
    ds = gen.specs_datasheet()
    many = _lockstep("eta1", cfg, reqs, _rows(ds, [1, 1]))[0]
    np.testing.assert_array_equal(many[0]["entry_q"], many[1]["entry_q"])
    np.testing.assert_array_equal(many[0]["entry_h"], many[1]["entry_h"])
    np.testing.assert_allclose(many[0]["step_latency"], many[1]["step_latency"], rtol=1e-6, atol=0)
    np.testing.assert_allclose(many[0]["e2e"], many[1]["e2e"], rtol=1e-6, atol=0)
    empty = {"arrival": np.zeros(0), "prompt": u32([]), "output": u32([])}
    for res in _lockstep("eta1", cfg, empty, _rows(ds, [0, 1, 0]))[0]:
        assert res["n_steps"] == 0 and res["clock"] == 0.0
