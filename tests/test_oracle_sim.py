"""Pins of the serving-simulation oracle (oracle/ks_sim.py).

Hand-traced scenarios with a constant step latency (closed forms for
chunked prefill and decode, budget sharing, arrival gaps, a prefix-cache
hit, a forced preemption), and invariants of the token-budget loop on a
random run (budget, sequence and KV limits, token accounting, FCFS order,
metric definitions of Sec. 2.1)."""
import numpy as np
import pytest

from oracle import ks_sim as sim


def const(L=1.0):
    return lambda batch, prefill: L


def req(arrival, prompt, output, group=0, prefix=0):
    return {"arrival": arrival, "prompt": prompt, "output": output, "group": group, "prefix": prefix}


def test_single_request_closed_form():
    # P = 100 over a budget of 32: chunks 32, 32, 32, 4, then O - 1 decodes;
    # TTFT = ceil(P / B) L, TPOT = L, E2E = (ceil(P / B) + O - 1) L
    cfg = sim.SchedCfg(max_batched_tokens=32, block_tokens=16, kv_blocks=64)
    r = sim.simulate([req(0.0, 100, 5)], cfg, const(2.0))
    assert [s[2] for s in r.steps] == [[(0, 32, 0)], [(0, 32, 32)], [(0, 32, 64)], [(0, 4, 96)],
                                       [(0, 1, 100)], [(0, 1, 101)], [(0, 1, 102)], [(0, 1, 103)]]
    assert [s[3] for s in r.steps] == [True] * 4 + [False] * 4
    assert r.ttft == [8.0] and r.tpot == [2.0] and r.e2e == [16.0]
    assert [s[0] for s in r.steps] == [2.0 * i for i in range(8)]


def test_two_requests_share_the_budget():
    # budget 64: A (P 100) takes the whole first step; step 2: A's 36 tokens,
    # then B (P 10) is admitted with 10; from step 3 both decode together
    cfg = sim.SchedCfg(max_batched_tokens=64, block_tokens=16, kv_blocks=64)
    r = sim.simulate([req(0.0, 100, 2), req(0.0, 10, 3)], cfg, const(1.0))
    assert [s[2] for s in r.steps] == [[(0, 64, 0)], [(0, 36, 64), (1, 10, 0)],
                                       [(0, 1, 100), (1, 1, 10)], [(1, 1, 11)]]
    assert r.ttft == [2.0, 2.0] and r.e2e == [3.0, 4.0]
    assert r.tpot == [1.0, 1.0]


def test_arrival_gap_and_max_num_seqs():
    cfg = sim.SchedCfg(max_num_seqs=1, max_batched_tokens=64, block_tokens=16, kv_blocks=64)
    # B arrives while A runs but waits for the only sequence slot; C arrives
    # after everything finished, so the clock jumps to its arrival
    r = sim.simulate([req(0.0, 8, 2), req(0.5, 8, 1), req(10.0, 4, 1)], cfg, const(1.0))
    assert [s[0] for s in r.steps] == [0.0, 1.0, 2.0, 10.0]
    assert [s[2] for s in r.steps] == [[(0, 8, 0)], [(0, 1, 8)], [(1, 8, 0)], [(2, 4, 0)]]
    assert r.ttft == [1.0, 2.5, 1.0]


def test_prefix_hit_skips_the_cached_blocks():
    # group 7 shares S = 64 tokens = 4 blocks of 16; A computes them and
    # caches them; B (arriving after A's prefill) starts at 64 computed
    cfg = sim.SchedCfg(max_batched_tokens=256, block_tokens=16, kv_blocks=64)
    r = sim.simulate([req(0.0, 100, 3, 7, 64), req(5.0, 90, 2, 7, 64)], cfg, const(1.0))
    b_steps = [(s[0], q) for s in r.steps for q in s[2] if q[0] == 1]
    assert b_steps[0] == (5.0, (1, 90 - 64, 64))
    # without prefix caching B computes its whole prompt
    cfg.prefix_cache = False
    r2 = sim.simulate([req(0.0, 100, 3, 7, 64), req(5.0, 90, 2, 7, 64)], cfg, const(1.0))
    assert [q for s in r2.steps for q in s[2] if q[0] == 1][0] == (1, 90, 0)
    # a hit never covers the last prompt token: P = 64 starts at 48 computed
    r3 = sim.simulate([req(0.0, 100, 3, 7, 64), req(5.0, 64, 2, 7, 64)],
                      sim.SchedCfg(max_batched_tokens=256, block_tokens=16, kv_blocks=64), const(1.0))
    assert [q for s in r3.steps for q in s[2] if q[0] == 1][0] == (1, 16, 48)


def test_preemption_by_recompute():
    # 4-token blocks, 6 blocks.  A (P 8, O 16) and B (P 8, O 12) prefill
    # together and decode in lockstep; at 12 computed tokens each holds 3
    # blocks.  The next step A needs a 4th block: nothing is free and no
    # prefix is cached, so B (the last admitted) is preempted, and A decodes
    # alone.  B returns when A has finished and recomputes its 8 prompt
    # tokens plus the 5 it had generated, in one chunk.
    cfg = sim.SchedCfg(max_batched_tokens=64, block_tokens=4, kv_blocks=6)
    r = sim.simulate([req(0.0, 8, 16), req(0.0, 8, 12)], cfg, const(1.0))
    assert r.preemptions == 1
    assert r.state == [sim.FINISHED, sim.FINISHED]
    steps = [s[2] for s in r.steps]
    assert steps[0] == [(0, 8, 0), (1, 8, 0)]
    assert steps[4] == [(0, 1, 11), (1, 1, 11)]
    assert steps[5] == [(0, 1, 12)]                    # B preempted
    a_done = max(i for i, st in enumerate(steps) if any(q[0] == 0 for q in st))
    assert steps[a_done + 1] == [(1, 13, 0)]           # recompute: 8 + 5 tokens
    assert r.e2e[0] == 16.0                            # A: 1 prefill + 15 decodes
    assert r.ttft[1] == 1.0


def test_request_that_never_fits_is_rejected():
    cfg = sim.SchedCfg(max_batched_tokens=64, block_tokens=16, kv_blocks=4)
    r = sim.simulate([req(0.0, 60, 10), req(0.0, 8, 2)], cfg, const(1.0))
    assert r.state == [sim.REJECTED, sim.FINISHED]


def _random_requests(n, seed, groups=4, gap=0.002):
    rng = np.random.Generator(np.random.PCG64(seed))
    t = np.cumsum(rng.exponential(gap, n))
    pre = rng.integers(32, 400, groups + 1)
    out = []
    for i in range(n):
        g = int(rng.integers(0, groups + 1)) if rng.random() < 0.5 else 0
        P = int(rng.integers(8, 700))
        S = min(int(pre[g]), P) if g else 0
        out.append(req(float(t[i]), max(P, S), int(rng.integers(1, 60)), g, S))
    return out


@pytest.mark.parametrize("kv", [4096, 120])
def test_invariants_on_a_random_run(kv):
    reqs = _random_requests(120, 5)
    cfg = sim.SchedCfg(max_num_seqs=16, max_batched_tokens=512, block_tokens=16, kv_blocks=kv)
    lat = lambda batch, prefill: 1e-3 + 2e-6 * sum(q for q, _ in batch) + (5e-4 if prefill else 0.0)
    r = sim.simulate(reqs, cfg, lat)
    assert all(s == sim.FINISHED for s in r.state)
    last_h = {}
    for (t0, L, batch, prefill) in r.steps:
        assert sum(q for _, q, _ in batch) <= cfg.max_batched_tokens
        assert len(batch) <= cfg.max_num_seqs
        assert len({i for i, _, _ in batch}) == len(batch)
        for (i, q, h) in batch:
            assert q >= 1
            last_h[i] = h + q
    # every request ends having computed its prompt and all but its last token
    for i, rq in enumerate(reqs):
        assert last_h[i] == rq["prompt"] + rq["output"] - 1
    # the clock only moves forward by the step latencies (or to arrivals)
    starts = [s[0] for s in r.steps]
    assert all(b >= a + s[1] - 1e-12 for a, b, s in zip(starts, starts[1:], r.steps))
    for i, rq in enumerate(reqs):
        assert r.ttft[i] > 0 and r.e2e[i] >= r.ttft[i]
        if rq["output"] > 1:
            assert r.tpot[i] > 0
    if kv == 4096:
        assert r.preemptions == 0
        # FCFS: requests are first scheduled in arrival order
        first = []
        for s in r.steps:
            for (i, _, _) in s[2]:
                if i not in first:
                    first.append(i)
        assert first == sorted(first)
    else:
        assert r.preemptions > 0


def test_throughput_definition():
    reqs = [req(1.0, 16, 4), req(1.0, 16, 4)]
    cfg = sim.SchedCfg(max_batched_tokens=64, block_tokens=16, kv_blocks=64)
    r = sim.simulate(reqs, cfg, const(0.5))
    # both finish after 1 prefill + 3 decode steps = 2 s: 8 tokens / 2 s
    assert sim.throughput(reqs, r) == pytest.approx(4.0)
