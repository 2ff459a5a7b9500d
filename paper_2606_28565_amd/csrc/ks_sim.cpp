// Serving simulation with the scheduler in the loop (the C ABI's
// ks_simulate): a host discrete-event loop (Sec. 4.1-4.2) running the
// token-budget scheduler of Sec. 5.8 (continuous batching, chunked prefill,
// prefix-cache-aware FCFS admission, preemption by recompute), pricing every
// step it forms with the library's GPU path (batch expansion in the
// homogeneous form, then the evaluation kernels for one spec vector) and
// advancing its clock by the step's t_step (Eq. 4).
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <deque>
#include <unordered_map>
#include <vector>

#include "ks.h"
#include "ks_internal.h"

namespace {

constexpr size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

enum : int32_t { kWaiting = 0, kRunning = 1, kFinished = 2, kRejected = 3 };

struct Req {
  double arrival = 0, first = -1, last = -1, finish = -1;
  uint32_t prompt = 0, output = 0, group = 0, prefix = 0;
  uint32_t generated = 0, computed = 0;
  int64_t held = 0, shared = 0;   // blocks of its own, blocks of its group's cache entry
  int32_t state = kWaiting;
  uint32_t target() const { return prompt + generated; }
};

struct Entry {
  int64_t blocks = 0, refs = 0;
  uint64_t last_use = 0;
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Device workspace of the simulator (every region 256-byte aligned):
//   stage   : req_off[2], req_q[S], req_h[S] (u32), prefill flag (u8)
//   records : step, m, n, k, a, b, mult (u32 [R] each) and the four
//             per-step arrays (u32 [1] each), R = records of one step
//   expand  : ks_expand's workspace for one step
//   eval    : ks_eval_steps' workspace for one step and one spec
//   outputs : t_body, t_gpu, t_step (f64)
struct SimLayout {
  size_t stage, rec, expand, eval, outs, total;
  size_t expand_bytes, eval_bytes;
  int64_t R;
  int32_t S;
};

bool sim_layout(const ks_model *md, const ks_sched *sc, SimLayout *L) {
  int64_t fo_p[KS_NFAM + 1], fo_d[KS_NFAM + 1];
  if (ks_expand_layout(md, 1, 1, KS_EXPAND_HOMOGENEOUS, fo_p) != KS_OK) return false;
  if (ks_expand_layout(md, 1, 0, KS_EXPAND_HOMOGENEOUS, fo_d) != KS_OK) return false;
  L->R = fo_p[KS_NFAM] > fo_d[KS_NFAM] ? fo_p[KS_NFAM] : fo_d[KS_NFAM];
  L->S = sc->max_num_seqs;
  // the evaluation workspace depends on the family layout; take the larger
  size_t ev = 0;
  for (const int64_t *fo : {fo_p, fo_d}) {
    const size_t b = ks::eval_workspace_bytes(fo, 1, 1);
    if (b > ev) ev = b;
  }
  L->eval_bytes = ev;
  L->expand_bytes = ks_expand_workspace_bytes(1);
  size_t off = 0;
  L->stage = off;
  off += align256((2 + 2 * (size_t)L->S) * sizeof(uint32_t) + 4);
  L->rec = off;
  off += align256((7 * (size_t)L->R + 4) * sizeof(uint32_t));
  L->expand = off;
  off += align256(L->expand_bytes);
  L->eval = off;
  off += align256(L->eval_bytes);
  L->outs = off;
  off += align256(3 * sizeof(double));
  L->total = off;
  return true;
}

ks_status check_sched(const ks_model *md, const ks_sched *sc) {
  if (!md || !sc) return ks::set_error(KS_EINVAL, "model or sched is NULL");
  if (md->experts != 0) return ks::set_error(KS_EINVAL, "the simulator takes dense decoders only (experts = 0)");
  if (sc->max_num_seqs < 1 || sc->max_num_seqs > (1 << 20))
    return ks::set_error(KS_EINVAL, "sched.max_num_seqs %d outside 1 .. 2^20", sc->max_num_seqs);
  if (sc->max_batched_tokens < 1 || sc->max_batched_tokens >= (1 << 24))
    return ks::set_error(KS_ERANGE, "sched.max_batched_tokens %d outside 1 .. 2^24 - 1", sc->max_batched_tokens);
  if (sc->block_tokens < 1) return ks::set_error(KS_EINVAL, "sched.block_tokens %d below 1", sc->block_tokens);
  if (sc->prefix_cache != 0 && sc->prefix_cache != 1)
    return ks::set_error(KS_EINVAL, "sched.prefix_cache %d not 0 or 1", sc->prefix_cache);
  if (sc->kv_blocks < 1) return ks::set_error(KS_EINVAL, "sched.kv_blocks %lld below 1", (long long)sc->kv_blocks);
  return KS_OK;
}

}  // namespace

extern "C" {

size_t ks_simulate_workspace_bytes(const ks_model *model, const ks_sched *sched) {
  if (check_sched(model, sched) != KS_OK) return 0;
  SimLayout L;
  if (!sim_layout(model, sched, &L)) return 0;
  return L.total;
}

ks_status ks_simulate(const ks_model *model, const ks_spec *spec, const ks_heads *heads, const ks_host *host,
                      const ks_sched *sched, const ks_requests *rq, ks_sim_out *out, void *ws, size_t ws_bytes,
                      hipStream_t stream) {
  ks_status st = check_sched(model, sched);
  if (st != KS_OK) return st;
  if (!spec || !heads || !host || !rq || !out) return ks::set_error(KS_EINVAL, "a pointer argument is NULL");
  SimLayout L;
  if (!sim_layout(model, sched, &L)) return ks::set_error(KS_EINVAL, "model rejected by the expansion");
  if (!ws) return ks::set_error(KS_EWORKSPACE, "workspace is NULL");
  if (ws_bytes < L.total) return ks::set_error(KS_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, L.total);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return ks::set_error(KS_EWORKSPACE, "workspace not 256-byte aligned");
  const int64_t n = rq->n;
  if (n < 0 || n >= (int64_t(1) << 32)) return ks::set_error(KS_ERANGE, "requests.n %lld outside [0, 2^32)", (long long)n);
  if (n > 0 && (!rq->arrival || !rq->prompt || !rq->output))
    return ks::set_error(KS_EINVAL, "a request array is NULL");
  if (rq->group && !rq->prefix) return ks::set_error(KS_EINVAL, "requests.prefix is NULL with groups");
  if (out->step_cap < 0 || out->entry_cap < 0) return ks::set_error(KS_EINVAL, "negative record capacity");
  if (out->step_cap > 0 && (!out->step_start || !out->step_latency || !out->step_prefill || !out->step_entry_off))
    return ks::set_error(KS_EINVAL, "a step record array is NULL with step_cap > 0");
  if (out->entry_cap > 0 && (!out->entry_req || !out->entry_q || !out->entry_h))
    return ks::set_error(KS_EINVAL, "an entry record array is NULL with entry_cap > 0");

  std::vector<Req> R((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    Req &r = R[(size_t)i];
    r.arrival = rq->arrival[i];
    r.prompt = rq->prompt[i];
    r.output = rq->output[i];
    r.group = rq->group ? rq->group[i] : 0;
    r.prefix = r.group ? rq->prefix[i] : 0;
    if (!std::isfinite(r.arrival) || (i > 0 && r.arrival < R[(size_t)i - 1].arrival))
      return ks::set_error(KS_EINVAL, "request %lld: arrivals not finite and non-decreasing", (long long)i);
    if (r.prompt < 1 || r.output < 1 || r.prompt >= (1u << 24) || r.output >= (1u << 24))
      return ks::set_error(KS_ERANGE, "request %lld: prompt and output must be in 1 .. 2^24 - 1", (long long)i);
    if (r.prefix > r.prompt) return ks::set_error(KS_EINVAL, "request %lld: prefix longer than the prompt", (long long)i);
  }

  char *w = static_cast<char *>(ws);
  uint32_t *d_stage = reinterpret_cast<uint32_t *>(w + L.stage);
  uint32_t *d_req_off = d_stage, *d_req_q = d_stage + 2, *d_req_h = d_stage + 2 + L.S;
  uint8_t *d_prefill = reinterpret_cast<uint8_t *>(d_stage + 2 + 2 * L.S);
  uint32_t *d_rec = reinterpret_cast<uint32_t *>(w + L.rec);
  ks_records rec;
  rec.step = d_rec;
  rec.m = d_rec + L.R;
  rec.n = d_rec + 2 * L.R;
  rec.k = d_rec + 3 * L.R;
  rec.a = d_rec + 4 * L.R;
  rec.b = d_rec + 5 * L.R;
  rec.mult = d_rec + 6 * L.R;
  rec.layers = d_rec + 7 * L.R;
  rec.hidden = rec.layers + 1;
  rec.tp = rec.layers + 2;
  rec.n_launch = rec.layers + 3;
  double *d_out = reinterpret_cast<double *>(w + L.outs);
  ks_step_out so = {d_out, d_out + 1, d_out + 2};
  ks_steps steps = {1, rec.layers, rec.hidden, rec.tp, rec.n_launch};
  const int64_t b = sched->block_tokens;

  std::vector<uint32_t> stage(2 + 2 * (size_t)L.S + 1);
  std::deque<int64_t> waiting;
  std::vector<int64_t> running;
  std::unordered_map<uint32_t, Entry> cache;
  int64_t used = 0;              // blocks held by running requests plus cache entries
  uint64_t use_clock = 0;
  int64_t next = 0, n_steps = 0, n_entries = 0, preemptions = 0, idle = 0;
  double clock = 0.0;
  if (out->step_cap > 0) out->step_entry_off[0] = 0;

  auto evict_until = [&](int64_t need) {
    while (sched->kv_blocks - used < need) {
      uint32_t victim = 0;
      uint64_t best = UINT64_MAX;
      bool found = false;
      for (const auto &kv : cache)
        if (kv.second.refs == 0 && kv.second.last_use < best) {
          best = kv.second.last_use;
          victim = kv.first;
          found = true;
        }
      if (!found) return false;
      used -= cache[victim].blocks;
      cache.erase(victim);
    }
    return true;
  };
  auto release = [&](Req &r) {
    if (r.shared) {
      auto it = cache.find(r.group);
      if (it != cache.end()) it->second.refs -= 1;
    }
    used -= r.held;
    r.held = r.shared = 0;
  };
  auto touch = [&](uint32_t g) { cache[g].last_use = ++use_clock; };

  struct Sched {
    int64_t r;
    uint32_t q, h;
  };
  std::vector<Sched> sch;
  while (true) {
    while (next < n && R[(size_t)next].arrival <= clock) waiting.push_back(next++);
    if (running.empty() && waiting.empty()) {
      if (next >= n) break;
      clock = std::fmax(clock, R[(size_t)next].arrival);
      continue;
    }
    int64_t budget = sched->max_batched_tokens;
    sch.clear();
    bool preempted = false;
    for (size_t i = 0; i < running.size() && budget > 0; ++i) {
      Req &r = R[(size_t)running[i]];
      const int64_t q = std::min<int64_t>((int64_t)r.target() - r.computed, budget);
      const int64_t need = ceil_div((int64_t)r.computed + q, b) - r.shared - r.held;
      while (need > sched->kv_blocks - used && !evict_until(need)) {
        const int64_t v = running.back();   // the most recently admitted
        running.pop_back();
        Req &vr = R[(size_t)v];
        release(vr);
        vr.computed = 0;
        vr.state = kWaiting;
        waiting.push_front(v);
        ++preemptions;
        preempted = true;
        if (&vr == &r) break;
      }
      if (r.state != kRunning) break;
      if (need > 0) {
        r.held += need;
        used += need;
      }
      sch.push_back({running[i], (uint32_t)q, r.computed});
      budget -= q;
    }
    if (!preempted) {
      while (!waiting.empty() && budget > 0 && (int64_t)running.size() < sched->max_num_seqs) {
        const int64_t idx = waiting.front();
        Req &r = R[(size_t)idx];
        if (ceil_div((int64_t)r.prompt + r.output, b) > sched->kv_blocks) {
          waiting.pop_front();      // can never hold its whole sequence
          r.state = kRejected;
          continue;
        }
        int64_t hit = 0;
        if (sched->prefix_cache && r.group) {
          auto it = cache.find(r.group);
          if (it != cache.end()) hit = std::min<int64_t>(it->second.blocks, ((int64_t)r.target() - 1) / b);
        }
        int64_t q = std::min<int64_t>((int64_t)r.target() - hit * b, budget);
        int64_t need = ceil_div(hit * b + q, b) - hit;
        if (need > sched->kv_blocks - used && !evict_until(need)) break;
        if (hit && cache.find(r.group) == cache.end()) {
          hit = 0;                  // the entry was evicted to make room
          q = std::min<int64_t>(r.target(), budget);
          need = ceil_div(q, b);
          if (need > sched->kv_blocks - used && !evict_until(need)) break;
        }
        waiting.pop_front();
        r.state = kRunning;
        r.computed = (uint32_t)(hit * b);
        r.shared = hit;
        r.held = need;
        used += need;
        if (hit) {
          cache[r.group].refs += 1;
          touch(r.group);
        }
        running.push_back(idx);
        sch.push_back({idx, (uint32_t)q, r.computed});
        budget -= q;
      }
    }
    if (sch.empty()) {
      // every running request was preempted: schedule again at this clock
      if (++idle > 2) return ks::set_error(KS_EINVAL, "simulation made no progress at t = %g", clock);
      continue;
    }
    idle = 0;

    // price the step: batch descriptor -> device, expansion, evaluation
    const int64_t nq = (int64_t)sch.size();
    bool prefill = false;
    uint64_t pairs = 0;
    stage[0] = 0;
    stage[1] = (uint32_t)nq;
    for (int64_t i = 0; i < nq; ++i) {
      const Req &r = R[(size_t)sch[i].r];
      stage[2 + i] = sch[i].q;
      stage[2 + L.S + i] = sch[i].h;
      prefill = prefill || (r.target() - sch[i].h > 1);
      const uint64_t q = sch[i].q, h = sch[i].h;
      pairs += q * h + q * (q + 1) / 2;
    }
    if (pairs >= (uint64_t(1) << 40))
      return ks::set_error(KS_ERANGE, "step at t = %g: causal pairs at or above 2^40", clock);
    uint8_t pre = prefill ? 1 : 0;
    std::memcpy(&stage[2 + 2 * L.S], &pre, 1);
    hipError_t e = hipMemcpyAsync(d_stage, stage.data(), stage.size() * sizeof(uint32_t), hipMemcpyHostToDevice,
                                  stream);
    if (e != hipSuccess) return ks::set_error(KS_EHIP, "batch copy: %s", hipGetErrorString(e));
    ks_batch bt = {1, d_req_off, d_req_q, nq, d_prefill, prefill ? 1 : 0};
    int64_t fo[KS_NFAM + 1];
    st = ks_expand_layout(model, 1, bt.n_prefill, KS_EXPAND_HOMOGENEOUS, fo);
    if (st != KS_OK) return st;
    st = ks_expand(model, &bt, KS_EXPAND_HOMOGENEOUS, &rec, w + L.expand, L.expand_bytes, stream);
    if (st != KS_OK) return st;
    ks_desc d;
    std::memset(&d, 0, sizeof d);
    d.n_rows = fo[KS_NFAM];
    for (int f = 0; f <= KS_NFAM; ++f) d.fam_off[f] = fo[f];
    d.step = rec.step;
    d.m = rec.m;
    d.n = rec.n;
    d.k = rec.k;
    d.a = rec.a;
    d.b = rec.b;
    d.mult = rec.mult;
    d.n_steps = 1;
    d.req_off = d_req_off;
    d.req_q = d_req_q;
    d.req_h = d_req_h;
    d.n_req = nq;
    d.elem_bytes = 2;
    st = ks_eval_steps(&d, &steps, spec, 1, heads, host, &so, nullptr, w + L.eval, L.eval_bytes, stream);
    if (st != KS_OK) return st;
    double lat = 0.0;
    e = hipMemcpyAsync(&lat, d_out + 2, sizeof lat, hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return ks::set_error(KS_EHIP, "step latency readback: %s", hipGetErrorString(e));

    if (n_steps < out->step_cap && n_entries + nq <= out->entry_cap) {
      out->step_start[n_steps] = clock;
      out->step_latency[n_steps] = lat;
      out->step_prefill[n_steps] = pre;
      for (int64_t i = 0; i < nq; ++i) {
        out->entry_req[n_entries + i] = (uint32_t)sch[i].r;
        out->entry_q[n_entries + i] = sch[i].q;
        out->entry_h[n_entries + i] = sch[i].h;
      }
      n_entries += nq;
      out->step_entry_off[n_steps + 1] = n_entries;
    }
    clock += lat;
    ++n_steps;

    std::vector<int64_t> done;
    for (const Sched &s : sch) {
      Req &r = R[(size_t)s.r];
      r.computed += s.q;
      const int64_t pb = (int64_t)r.prefix / b;
      if (sched->prefix_cache && r.group && pb > 0 && r.shared == 0 && (int64_t)r.computed >= pb * b &&
          cache.find(r.group) == cache.end()) {
        Entry en;
        en.blocks = pb;
        en.refs = 1;
        cache[r.group] = en;
        touch(r.group);
        r.shared = pb;
        r.held -= pb;               // the blocks move from the request to the entry
      }
      if (r.computed == r.target()) {
        r.generated += 1;
        if (r.generated == 1) r.first = clock;
        r.last = clock;
        if (r.generated == r.output) {
          r.finish = clock;
          done.push_back(s.r);
        }
      }
    }
    for (int64_t idx : done) {
      for (size_t i = 0; i < running.size(); ++i)
        if (running[i] == idx) {
          running.erase(running.begin() + (ptrdiff_t)i);
          break;
        }
      release(R[(size_t)idx]);
      R[(size_t)idx].state = kFinished;
    }
  }
  for (int64_t i = 0; i < n; ++i) {
    const Req &r = R[(size_t)i];
    const bool fin = r.state == kFinished;
    if (out->state) out->state[i] = r.state;
    if (out->ttft) out->ttft[i] = fin ? r.first - r.arrival : 0.0;
    if (out->tpot) out->tpot[i] = fin && r.output > 1 ? (r.last - r.first) / (double)(r.output - 1) : 0.0;
    if (out->e2e) out->e2e[i] = fin ? r.finish - r.arrival : 0.0;
  }
  out->n_steps = n_steps;
  out->n_entries = n_entries;
  out->preemptions = preemptions;
  out->clock = clock;
  return KS_OK;
}

}  // extern "C"
