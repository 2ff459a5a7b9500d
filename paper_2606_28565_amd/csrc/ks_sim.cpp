// Serving simulation with the scheduler in the loop (the C ABI's
// ks_simulate): host discrete-event loops (Sec. 4.1-4.2) running the
// token-budget scheduler of Sec. 5.8 (continuous batching, chunked prefill,
// prefix-cache-aware FCFS admission, preemption by recompute), one per spec
// vector, in lockstep: each round every unfinished simulation forms its next
// step, the round's steps are priced together by the library's GPU path
// (batch expansion in the homogeneous form, then the evaluation kernels for
// all spec vectors, each step keeping its own simulation's t_step, Eq. 4),
// and each simulation advances its clock by its step's latency.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdint>
#include <algorithm>
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

// Device workspace of the simulator for S simulations (every region
// 256-byte aligned):
//   stage   : a round's batch, packed: req_off[A + 1], req_q, req_h (at
//             most S Q entries each, Q = max_num_seqs), each step's own spec
//             [A] (u32), prefill flags [A] (u8); A <= S steps
//   records : step, m, n, k, a, b, mult (u32 [S R] each) and the four
//             per-step arrays (u32 [S] each), R = records of one step
//   expand  : ks_expand's workspace for S steps
//   eval    : ks_eval_steps' workspace for S steps and S specs
//   outputs : t_body, t_gpu, t_step (f64 [S][S]), each step's own latency (f64 [S])
struct SimLayout {
  size_t stage, rec, expand, eval, outs, lat, total;
  size_t expand_bytes, eval_bytes;
  int64_t R, S, Q;
};

bool sim_layout(const ks_model *md, const ks_sched *sc, int32_t n_sims, SimLayout *L) {
  int64_t fo_p[KS_NFAM + 1], fo_d[KS_NFAM + 1];
  if (ks_expand_layout(md, 1, 1, KS_EXPAND_HOMOGENEOUS, fo_p) != KS_OK) return false;
  if (ks_expand_layout(md, 1, 0, KS_EXPAND_HOMOGENEOUS, fo_d) != KS_OK) return false;
  L->R = fo_p[KS_NFAM] > fo_d[KS_NFAM] ? fo_p[KS_NFAM] : fo_d[KS_NFAM];
  L->S = n_sims;
  L->Q = sc->max_num_seqs;
  // an upper bound of the evaluation workspace for any round: every family
  // at S steps' records (both attention families at S each)
  int64_t fo[KS_NFAM + 1];
  fo[0] = 0;
  for (int f = 0; f < KS_NFAM; ++f) {
    const int64_t per = std::max(fo_p[f + 1] - fo_p[f], fo_d[f + 1] - fo_d[f]);
    fo[f + 1] = fo[f] + per * L->S;
  }
  L->eval_bytes = ks::eval_workspace_bytes(fo, L->S, n_sims);
  L->expand_bytes = ks_expand_workspace_bytes(L->S);
  const size_t S = (size_t)L->S, Q = (size_t)L->Q;
  size_t off = 0;
  L->stage = off;
  off += align256((S + 1 + 2 * S * Q + S + (S + 3) / 4) * sizeof(uint32_t));
  L->rec = off;
  off += align256((7 * (size_t)L->R * S + 4 * S) * sizeof(uint32_t));
  L->expand = off;
  off += align256(L->expand_bytes);
  L->eval = off;
  off += align256(L->eval_bytes);
  L->outs = off;
  off += align256(3 * S * S * sizeof(double));
  L->lat = off;
  off += align256(S * sizeof(double));
  L->total = off;
  return true;
}

ks_status check_sched(const ks_model *md, const ks_sched *sc, int32_t n_sims) {
  if (!md || !sc) return ks::set_error(KS_EINVAL, "model or sched is NULL");
  if (md->experts != 0) return ks::set_error(KS_EINVAL, "the simulator takes dense decoders only (experts = 0)");
  if (n_sims < 1 || n_sims > 256) return ks::set_error(KS_EINVAL, "n_specs %d outside 1 .. 256", n_sims);
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

struct Sched {
  int64_t r;
  uint32_t q, h;
};

// One simulation's scheduler state; next() forms the next step's batch at
// the clock, advance() applies its latency.
class Sim {
 public:
  Sim(const ks_sched *sc, const std::vector<Req> &reqs) : sc_(sc), R_(reqs) {}

  // 1: a step in `sch` (prefill flag in `prefill`), 0: every request done,
  // -1: no progress possible
  int next(std::vector<Sched> &sch, bool &prefill) {
    const int64_t n = (int64_t)R_.size(), b = sc_->block_tokens;
    for (int idle = 0;;) {
      while (next_ < n && R_[(size_t)next_].arrival <= clock) waiting_.push_back(next_++);
      if (running_.empty() && waiting_.empty()) {
        if (next_ >= n) return 0;
        clock = std::fmax(clock, R_[(size_t)next_].arrival);
        continue;
      }
      int64_t budget = sc_->max_batched_tokens;
      sch.clear();
      bool preempted = false;
      for (size_t i = 0; i < running_.size() && budget > 0; ++i) {
        Req &r = R_[(size_t)running_[i]];
        const int64_t q = std::min<int64_t>((int64_t)r.target() - r.computed, budget);
        const int64_t need = ceil_div((int64_t)r.computed + q, b) - r.shared - r.held;
        while (need > sc_->kv_blocks - used_ && !evict_until(need)) {
          const int64_t v = running_.back();   // the most recently admitted
          running_.pop_back();
          Req &vr = R_[(size_t)v];
          release(vr);
          vr.computed = 0;
          vr.state = kWaiting;
          waiting_.push_front(v);
          ++preemptions;
          preempted = true;
          if (&vr == &r) break;
        }
        if (r.state != kRunning) break;
        if (need > 0) {
          r.held += need;
          used_ += need;
        }
        sch.push_back({running_[i], (uint32_t)q, r.computed});
        budget -= q;
      }
      if (!preempted) {
        while (!waiting_.empty() && budget > 0 && (int64_t)running_.size() < sc_->max_num_seqs) {
          const int64_t idx = waiting_.front();
          Req &r = R_[(size_t)idx];
          if (ceil_div((int64_t)r.prompt + r.output, b) > sc_->kv_blocks) {
            waiting_.pop_front();      // can never hold its whole sequence
            r.state = kRejected;
            continue;
          }
          int64_t hit = 0;
          if (sc_->prefix_cache && r.group) {
            auto it = cache_.find(r.group);
            if (it != cache_.end()) hit = std::min<int64_t>(it->second.blocks, ((int64_t)r.target() - 1) / b);
          }
          int64_t q = std::min<int64_t>((int64_t)r.target() - hit * b, budget);
          int64_t need = ceil_div(hit * b + q, b) - hit;
          if (need > sc_->kv_blocks - used_ && !evict_until(need)) break;
          if (hit && cache_.find(r.group) == cache_.end()) {
            hit = 0;                   // the entry was evicted to make room
            q = std::min<int64_t>(r.target(), budget);
            need = ceil_div(q, b);
            if (need > sc_->kv_blocks - used_ && !evict_until(need)) break;
          }
          waiting_.pop_front();
          r.state = kRunning;
          r.computed = (uint32_t)(hit * b);
          r.shared = hit;
          r.held = need;
          used_ += need;
          if (hit) {
            cache_[r.group].refs += 1;
            touch(r.group);
          }
          running_.push_back(idx);
          sch.push_back({idx, (uint32_t)q, r.computed});
          budget -= q;
        }
      }
      if (sch.empty()) {
        // every running request was preempted: schedule again at this clock
        if (++idle > 2) return -1;
        continue;
      }
      prefill = false;
      for (const Sched &e : sch) prefill = prefill || (R_[(size_t)e.r].target() - e.h > 1);
      return 1;
    }
  }

  void advance(const std::vector<Sched> &sch, double lat, bool prefill, ks_sim_out *out) {
    const int64_t nq = (int64_t)sch.size(), b = sc_->block_tokens;
    if (n_steps < out->step_cap && n_entries + nq <= out->entry_cap) {
      out->step_start[n_steps] = clock;
      out->step_latency[n_steps] = lat;
      out->step_prefill[n_steps] = prefill ? 1 : 0;
      for (int64_t i = 0; i < nq; ++i) {
        out->entry_req[n_entries + i] = (uint32_t)sch[(size_t)i].r;
        out->entry_q[n_entries + i] = sch[(size_t)i].q;
        out->entry_h[n_entries + i] = sch[(size_t)i].h;
      }
      n_entries += nq;
      out->step_entry_off[n_steps + 1] = n_entries;
    }
    clock += lat;
    ++n_steps;
    done_.clear();
    for (const Sched &e : sch) {
      Req &r = R_[(size_t)e.r];
      r.computed += e.q;
      const int64_t pb = (int64_t)r.prefix / b;
      if (sc_->prefix_cache && r.group && pb > 0 && r.shared == 0 && (int64_t)r.computed >= pb * b &&
          cache_.find(r.group) == cache_.end()) {
        Entry en;
        en.blocks = pb;
        en.refs = 1;
        cache_[r.group] = en;
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
          done_.push_back(e.r);
        }
      }
    }
    for (int64_t idx : done_) {
      for (size_t i = 0; i < running_.size(); ++i)
        if (running_[i] == idx) {
          running_.erase(running_.begin() + (ptrdiff_t)i);
          break;
        }
      release(R_[(size_t)idx]);
      R_[(size_t)idx].state = kFinished;
    }
  }

  void finish(ks_sim_out *out) const {
    for (size_t i = 0; i < R_.size(); ++i) {
      const Req &r = R_[i];
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
  }

  double clock = 0.0;
  int64_t n_steps = 0, n_entries = 0, preemptions = 0;

 private:
  bool evict_until(int64_t need) {
    while (sc_->kv_blocks - used_ < need) {
      uint32_t victim = 0;
      uint64_t best = UINT64_MAX;
      bool found = false;
      for (const auto &kv : cache_)
        if (kv.second.refs == 0 && kv.second.last_use < best) {
          best = kv.second.last_use;
          victim = kv.first;
          found = true;
        }
      if (!found) return false;
      used_ -= cache_[victim].blocks;
      cache_.erase(victim);
    }
    return true;
  }
  void release(Req &r) {
    if (r.shared) {
      auto it = cache_.find(r.group);
      if (it != cache_.end()) it->second.refs -= 1;
    }
    used_ -= r.held;
    r.held = r.shared = 0;
  }
  void touch(uint32_t g) { cache_[g].last_use = ++use_clock_; }

  const ks_sched *sc_;
  std::vector<Req> R_;
  std::deque<int64_t> waiting_;
  std::vector<int64_t> running_, done_;
  std::unordered_map<uint32_t, Entry> cache_;
  int64_t used_ = 0, next_ = 0;    // used_: blocks held by running requests plus cache entries
  uint64_t use_clock_ = 0;
};

}  // namespace

extern "C" {

size_t ks_simulate_workspace_bytes(const ks_model *model, const ks_sched *sched, int32_t n_specs) {
  if (check_sched(model, sched, n_specs) != KS_OK) return 0;
  SimLayout L;
  if (!sim_layout(model, sched, n_specs, &L)) return 0;
  return L.total;
}

ks_status ks_simulate(const ks_model *model, const ks_spec *specs, int32_t n_specs, const ks_heads *heads,
                      const ks_host *host, const ks_sched *sched, const ks_requests *rq, ks_sim_out *outs,
                      void *ws, size_t ws_bytes, hipStream_t stream) {
  ks_status st = check_sched(model, sched, n_specs);
  if (st != KS_OK) return st;
  if (!specs || !heads || !host || !rq || !outs) return ks::set_error(KS_EINVAL, "a pointer argument is NULL");
  SimLayout L;
  if (!sim_layout(model, sched, n_specs, &L)) return ks::set_error(KS_EINVAL, "model rejected by the expansion");
  if (!ws) return ks::set_error(KS_EWORKSPACE, "workspace is NULL");
  if (ws_bytes < L.total) return ks::set_error(KS_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, L.total);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return ks::set_error(KS_EWORKSPACE, "workspace not 256-byte aligned");
  const int64_t n = rq->n;
  if (n < 0 || n >= (int64_t(1) << 32)) return ks::set_error(KS_ERANGE, "requests.n %lld outside [0, 2^32)", (long long)n);
  if (n > 0 && (!rq->arrival || !rq->prompt || !rq->output))
    return ks::set_error(KS_EINVAL, "a request array is NULL");
  if (rq->group && !rq->prefix) return ks::set_error(KS_EINVAL, "requests.prefix is NULL with groups");
  for (int32_t s = 0; s < n_specs; ++s) {
    const ks_sim_out *out = &outs[s];
    if (out->step_cap < 0 || out->entry_cap < 0) return ks::set_error(KS_EINVAL, "negative record capacity");
    if (out->step_cap > 0 && (!out->step_start || !out->step_latency || !out->step_prefill || !out->step_entry_off))
      return ks::set_error(KS_EINVAL, "a step record array is NULL with step_cap > 0");
    if (out->entry_cap > 0 && (!out->entry_req || !out->entry_q || !out->entry_h))
      return ks::set_error(KS_EINVAL, "an entry record array is NULL with entry_cap > 0");
  }

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

  const int64_t S = n_specs;
  char *w = static_cast<char *>(ws);
  uint32_t *d_stage = reinterpret_cast<uint32_t *>(w + L.stage);
  uint32_t *d_rec = reinterpret_cast<uint32_t *>(w + L.rec);
  const int64_t RS = L.R * S;
  ks_records rec;
  rec.step = d_rec;
  rec.m = d_rec + RS;
  rec.n = d_rec + 2 * RS;
  rec.k = d_rec + 3 * RS;
  rec.a = d_rec + 4 * RS;
  rec.b = d_rec + 5 * RS;
  rec.mult = d_rec + 6 * RS;
  rec.layers = d_rec + 7 * RS;
  rec.hidden = rec.layers + S;
  rec.tp = rec.layers + 2 * S;
  rec.n_launch = rec.layers + 3 * S;
  double *d_out = reinterpret_cast<double *>(w + L.outs);
  double *d_lat = reinterpret_cast<double *>(w + L.lat);

  std::vector<Sim> sims;
  sims.reserve((size_t)S);
  for (int64_t s = 0; s < S; ++s) {
    sims.emplace_back(sched, R);
    if (outs[s].step_cap > 0) outs[s].step_entry_off[0] = 0;
  }
  std::vector<std::vector<Sched>> batch((size_t)S);
  std::vector<uint8_t> pre((size_t)S), live((size_t)S, 1);
  std::vector<int64_t> who;             // the simulation of each step of the round
  std::vector<uint32_t> h_off, h_q, h_h, h_spec;
  std::vector<uint8_t> h_pre;
  // the round's packed batch and its latencies cross PCIe through pinned
  // host buffers (asynchronous DMA rather than a staged pageable copy),
  // sized like the workspace's stage region; each round's synchronization
  // ends its copies before the buffers are reused
  struct Pinned {
    void *p = nullptr;
    ~Pinned() {
      if (p) (void)hipHostFree(p);
    }
  } pin_stage, pin_lat;
  const size_t stage_words = (size_t)(S + 1 + 2 * S * L.Q + S + (S + 3) / 4);
  hipError_t e = hipHostMalloc(&pin_stage.p, stage_words * sizeof(uint32_t), 0);
  if (e == hipSuccess) e = hipHostMalloc(&pin_lat.p, (size_t)S * sizeof(double), 0);
  if (e != hipSuccess) return ks::set_error(KS_EHIP, "pinned staging buffers: %s", hipGetErrorString(e));
  uint32_t *h_stage = static_cast<uint32_t *>(pin_stage.p);
  double *lat = static_cast<double *>(pin_lat.p);
  while (true) {
    // every unfinished simulation forms its next step
    who.clear();
    for (int64_t s = 0; s < S; ++s) {
      if (!live[(size_t)s]) continue;
      bool p = false;
      const int r = sims[(size_t)s].next(batch[(size_t)s], p);
      if (r < 0) return ks::set_error(KS_EINVAL, "simulation %lld made no progress at t = %g", (long long)s,
                                       sims[(size_t)s].clock);
      if (r == 0) {
        live[(size_t)s] = 0;
        continue;
      }
      pre[(size_t)s] = p ? 1 : 0;
      who.push_back(s);
    }
    const int64_t A = (int64_t)who.size();
    if (A == 0) break;

    // the round's steps as one batch: step i is simulation who[i]
    h_off.assign(1, 0);
    h_q.clear();
    h_h.clear();
    h_spec.clear();
    h_pre.clear();
    int64_t n_pre = 0;
    for (int64_t i = 0; i < A; ++i) {
      const std::vector<Sched> &sb = batch[(size_t)who[(size_t)i]];
      uint64_t pairs = 0;
      for (const Sched &e : sb) {
        h_q.push_back(e.q);
        h_h.push_back(e.h);
        pairs += (uint64_t)e.q * e.h + (uint64_t)e.q * (e.q + 1) / 2;
      }
      if (pairs >= (uint64_t(1) << 40))
        return ks::set_error(KS_ERANGE, "simulation %lld: a step's causal pairs at or above 2^40", (long long)who[(size_t)i]);
      h_off.push_back((uint32_t)h_q.size());
      h_spec.push_back((uint32_t)who[(size_t)i]);
      h_pre.push_back(pre[(size_t)who[(size_t)i]]);
      n_pre += pre[(size_t)who[(size_t)i]];
    }
    // one host-to-device copy of the round's batch, packed:
    // req_off[A + 1], req_q[nq], req_h[nq], own spec[A] (u32), prefill[A] (u8)
    const int64_t nq = (int64_t)h_q.size();
    uint32_t *d_req_off = d_stage, *d_req_q = d_req_off + (A + 1), *d_req_h = d_req_q + nq;
    uint32_t *d_own = d_req_h + nq;
    uint8_t *d_prefill = reinterpret_cast<uint8_t *>(d_own + A);
    size_t words = 0;
    for (const std::vector<uint32_t> *v : {&h_off, &h_q, &h_h, &h_spec}) {
      std::memcpy(h_stage + words, v->data(), v->size() * sizeof(uint32_t));
      words += v->size();
    }
    const size_t pre_words = (size_t)(A + 3) / 4;
    std::memset(h_stage + words, 0, pre_words * sizeof(uint32_t));
    std::memcpy(h_stage + words, h_pre.data(), (size_t)A);
    words += pre_words;
    e = hipMemcpyAsync(d_stage, h_stage, words * sizeof(uint32_t), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return ks::set_error(KS_EHIP, "batch copy: %s", hipGetErrorString(e));
    ks_batch bt = {A, d_req_off, d_req_q, nq, d_prefill, n_pre};
    int64_t fo[KS_NFAM + 1];
    st = ks_expand_layout(model, A, n_pre, KS_EXPAND_HOMOGENEOUS, fo);
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
    d.n_steps = A;
    d.req_off = d_req_off;
    d.req_q = d_req_q;
    d.req_h = d_req_h;
    d.n_req = nq;
    d.elem_bytes = 2;
    ks_steps stp = {A, rec.layers, rec.hidden, rec.tp, rec.n_launch};
    ks_step_out so = {d_out, d_out + S * A, d_out + 2 * S * A};
    // every step against every spec (all pairs); each simulation keeps its own
    // (and each step's latency under its own simulation's spec, in the same
    // launches)
    st = ks::eval_steps_own(&d, &stp, specs, n_specs, heads, host, &so, w + L.eval, L.eval_bytes, d_own, d_lat,
                            stream);
    if (st != KS_OK) return st;
    e = hipMemcpyAsync(lat, d_lat, A * sizeof(double), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return ks::set_error(KS_EHIP, "step latency readback: %s", hipGetErrorString(e));
    for (int64_t i = 0; i < A; ++i) {
      const int64_t s = who[(size_t)i];
      sims[(size_t)s].advance(batch[(size_t)s], lat[i], pre[(size_t)s] != 0, &outs[s]);
    }
  }
  for (int64_t s = 0; s < S; ++s) sims[(size_t)s].finish(&outs[s]);
  return KS_OK;
}

}  // extern "C"
