"""CPU oracle of the serving simulation: the scheduler in the loop.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this module; only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the library's simulator.

What it computes, and where the paper states it (KernelSight-LM):

* Sec. 4.1-4.2: a discrete-event simulator; requests arrive, the scheduler
  forms a batch, the predictor prices it, and the simulation clock advances
  by the predicted step time.
* Sec. 5.8 ("Faithful vLLM v1 scheduling"): one token-budget loop advances
  every request's computed-token count toward its target, which covers
  continuous batching, chunked prefill and prefix-cache-aware admission,
  with FCFS queueing and preemption by recompute under KV pressure;
  ("Hierarchical prefix caching"): a prefix hit reuses cached KV blocks, so
  only the uncached suffix is computed.
* Sec. 2.1: TTFT (submission to first token), TPOT (mean time between
  output tokens after the first) and output throughput (tokens/s).

Readings (the paper gives the behaviour, not the parameters or data
structures; the library's simulator takes the same ones):

* A request has an arrival time, P prompt tokens, O >= 1 output tokens and
  optionally a prefix group g whose first S_g tokens all its requests share.
  Its target is P + (tokens generated so far); `computed` counts tokens whose
  KV is in the cache.  When computed reaches the target the step samples a
  token: generated += 1 (the first one sets TTFT), the target grows by one;
  at O generated tokens the request finishes.
* Each step starts at the clock: arrivals up to it join the waiting queue.
  Budget = max_batched_tokens.  Running requests, in admission order, get
  n = min(target - computed, budget) tokens; if the KV cache cannot hold
  their blocks, cached prefixes nobody uses are evicted (least recently used
  first), then the most recently admitted running request is preempted (its
  blocks freed, computed reset to 0, back to the front of the waiting
  queue) until it fits or the request itself was preempted.  Without a
  preemption in the step, waiting requests are then admitted FCFS while the
  budget is positive and fewer than max_num_seqs run: a prefix hit of c
  cached blocks starts computed at min(c, floor((target - 1) / b)) * b, and
  the request gets n = min(target - computed, budget) if its blocks fit
  (after evicting unused prefixes), else admission stops.
* KV blocks of b tokens: a running request holds ceil(computed_after_step
  / b) blocks minus the prefix blocks it shares.  When a request's computed
  count first covers its group's floor(S_g / b) full prefix blocks and the
  group has no cached prefix, those blocks become the group's cache entry
  (moved from the request, which now shares them).  An entry lives until
  evicted; a request admitted with a hit shares it.
* The step's batch descriptor: request r with q_r = n tokens over h_r =
  computed history; the step carries a prefill chunk if some scheduled
  request has more than one token left to compute (target - computed > 1).
  Its latency is the model's t_step (Eq. 2-4) for that batch.
* A waiting request whose whole sequence (P + O tokens) needs more blocks
  than the cache has is rejected at admission.  A pass that schedules
  nothing (every running request preempted) schedules again at the same
  clock, when the running set is empty and every cached prefix evictable.
* Metrics: TTFT = first-token time - arrival; TPOT = (last-token time -
  first-token time) / (O - 1), 0 for O = 1; E2E = finish - arrival; output
  throughput = sum O / (last finish - first arrival).
"""
from __future__ import annotations

from dataclasses import dataclass, field

WAITING, RUNNING, FINISHED, REJECTED = 0, 1, 2, 3


@dataclass
class SchedCfg:
    max_num_seqs: int = 256
    max_batched_tokens: int = 8192
    block_tokens: int = 16
    kv_blocks: int = 8192
    prefix_cache: bool = True


@dataclass
class _Req:
    idx: int
    arrival: float
    prompt: int
    output: int
    group: int
    prefix: int
    generated: int = 0
    computed: int = 0
    held: int = 0          # blocks held outside a shared cache entry
    shared: int = 0        # blocks shared from the group's cache entry
    state: int = WAITING
    first: float = -1.0
    last: float = -1.0
    finish: float = -1.0
    admitted_at: int = -1  # admission sequence number (preemption order)

    @property
    def target(self) -> int:
        return self.prompt + self.generated


@dataclass
class SimResult:
    ttft: list
    tpot: list
    e2e: list
    state: list
    steps: list = field(default_factory=list)   # (start, latency, [(req, q, h)], prefill)
    preemptions: int = 0


def _ceil(a, b):
    return -(-a // b)


def simulate(requests, cfg: SchedCfg, step_latency, max_steps=10_000_000):
    """requests: list of dicts with arrival, prompt, output, group, prefix
    (sorted by arrival).  step_latency(batch, prefill) -> seconds, where
    batch is the list of (q, h) of the step's requests in schedule order."""
    reqs = [_Req(i, float(r["arrival"]), int(r["prompt"]), int(r["output"]),
                 int(r.get("group", 0)), int(r.get("prefix", 0))) for i, r in enumerate(requests)]
    b = cfg.block_tokens
    cache = {}         # group -> [blocks, refcount, last_use]
    waiting, running = [], []
    nxt, clock, admit_seq = 0, 0.0, 0
    out = SimResult([0.0] * len(reqs), [0.0] * len(reqs), [0.0] * len(reqs), [0] * len(reqs))
    use_clock = [0]    # LRU stamp: incremented per use

    def used_blocks():
        return sum(r.held for r in running) + sum(e[0] for e in cache.values())

    def free_blocks():
        return cfg.kv_blocks - used_blocks()

    def evict_until(need):
        # least recently used entries that no running request shares
        while free_blocks() < need:
            idle = [(e[2], g) for g, e in cache.items() if e[1] == 0]
            if not idle:
                return False
            _, g = min(idle)
            del cache[g]
        return True

    def release(r):
        if r.shared and r.group in cache:
            cache[r.group][1] -= 1
        r.held = r.shared = 0

    def touch(g):
        use_clock[0] += 1
        cache[g][2] = use_clock[0]

    steps = idle = 0
    while True:
        while nxt < len(reqs) and reqs[nxt].arrival <= clock:
            waiting.append(reqs[nxt])
            nxt += 1
        if not running and not waiting:
            if nxt >= len(reqs):
                break
            clock = max(clock, reqs[nxt].arrival)
            continue
        budget = cfg.max_batched_tokens
        sched = []          # (req, n, computed before)
        preempted = False
        i = 0
        while i < len(running) and budget > 0:
            r = running[i]
            n = min(r.target - r.computed, budget)
            need = _ceil(r.computed + n, b) - r.shared - r.held
            while need > free_blocks() and not evict_until(need):
                victim = running.pop()          # most recently admitted
                release(victim)
                victim.computed = 0
                victim.state = WAITING
                waiting.insert(0, victim)
                out.preemptions += 1
                preempted = True
                if victim is r:
                    break
            if r.state != RUNNING:
                break
            r.held += max(need, 0)
            sched.append((r, n, r.computed))
            budget -= n
            i += 1
        if not preempted:
            while waiting and budget > 0 and len(running) < cfg.max_num_seqs:
                r = waiting[0]
                hit = 0
                if cfg.prefix_cache and r.group and r.group in cache:
                    hit = min(cache[r.group][0], (r.target - 1) // b)
                if _ceil(r.prompt + r.output, b) > cfg.kv_blocks:
                    waiting.pop(0)          # can never hold its whole sequence
                    r.state = REJECTED
                    continue
                n = min(r.target - hit * b, budget)
                need = _ceil(hit * b + n, b) - hit
                if need > free_blocks() and not evict_until(need):
                    break
                if hit and r.group not in cache:
                    hit = 0         # the entry was evicted to make room
                    n = min(r.target, budget)
                    need = _ceil(n, b)
                    if need > free_blocks() and not evict_until(need):
                        break
                waiting.pop(0)
                r.state = RUNNING
                r.computed = hit * b
                r.shared = hit
                r.held = need
                if hit:
                    cache[r.group][1] += 1
                    touch(r.group)
                r.admitted_at = admit_seq
                admit_seq += 1
                running.append(r)
                sched.append((r, n, r.computed))
                budget -= n
        if not sched:
            # every running request was preempted (the next pass admits
            # from an emptied cache) or the waiting ones were rejected
            idle += 1
            if idle > 2:
                raise RuntimeError("no progress: nothing schedulable")
            continue
        idle = 0
        batch = [(n, h) for (_, n, h) in sched]
        prefill = any(r.target - h > 1 for (r, _, h) in sched)
        lat = float(step_latency(batch, prefill))
        out.steps.append((clock, lat, [(r.idx, n, h) for (r, n, h) in sched], prefill))
        assert used_blocks() <= cfg.kv_blocks
        clock += lat
        steps += 1
        if steps > max_steps:
            raise RuntimeError("step limit")
        done = []
        for (r, n, _) in sched:
            r.computed += n
            pb = r.prefix // b
            if (cfg.prefix_cache and r.group and pb > 0 and r.shared == 0 and r.computed >= pb * b
                    and r.group not in cache):
                cache[r.group] = [pb, 1, 0]
                touch(r.group)
                r.shared = pb
                r.held -= pb
            if r.computed == r.target:
                r.generated += 1
                if r.generated == 1:
                    r.first = clock
                r.last = clock
                if r.generated == r.output:
                    r.finish = clock
                    done.append(r)
        for r in done:
            running.remove(r)
            release(r)
            r.state = FINISHED
    for r in reqs:
        out.state[r.idx] = r.state
        if r.state == FINISHED:
            out.ttft[r.idx] = r.first - r.arrival
            out.tpot[r.idx] = (r.last - r.first) / (r.output - 1) if r.output > 1 else 0.0
            out.e2e[r.idx] = r.finish - r.arrival
    return out


def throughput(requests, res: SimResult):
    """Output tokens per second over the whole run (first arrival to last
    finish), counting finished requests."""
    fin = [i for i, s in enumerate(res.state) if s == FINISHED]
    if not fin:
        return 0.0
    first = min(float(requests[i]["arrival"]) for i in range(len(requests)))
    last = max(float(requests[i]["arrival"]) + res.e2e[i] for i in fin)
    return sum(int(requests[i]["output"]) for i in fin) / (last - first)
