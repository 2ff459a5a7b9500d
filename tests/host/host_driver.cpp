// CPU driver of the library's host code, built with g++ under AddressSanitizer
// and UndefinedBehaviorSanitizer against host stand-ins of the launches
// (fake_device.cpp).  TEST INFRASTRUCTURE ONLY.
//
//   host_driver args   every entry point's argument checks: one line
//                      "<case> <status>" per call (valid calls included)
//   host_driver sim    reads a model, a scheduler configuration, a spec
//                      count and requests on stdin and runs ks_simulate
//                      with the stand-in step latency; prints each
//                      simulation's steps and per-request metrics with
//                      exact (hexadecimal) floats
#include <hip/hip_runtime_api.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "ks.h"

namespace {

// 256-byte aligned host buffer standing in for device memory
struct Buf {
  void *p = nullptr;
  size_t n = 0;
  explicit Buf(size_t bytes) : n(bytes) {
    p = std::aligned_alloc(256, (bytes + 255) / 256 * 256 + 256);
    std::memset(p, 0, (bytes + 255) / 256 * 256 + 256);
  }
  ~Buf() { std::free(p); }
  Buf(const Buf &) = delete;
  Buf &operator=(const Buf &) = delete;
};

void report(const char *name, ks_status st) {
  std::printf("%s %d\n", name, (int)st);
  if (st != KS_OK && std::strlen(ks_last_error()) == 0) std::printf("%s empty-message\n", name);
}

// Three GEMM records over two steps, one decode request per step.
struct Small {
  std::vector<uint32_t> step{0, 0, 1}, m{1, 2, 3}, n{128, 256, 512}, k{64, 64, 64}, a{0, 0, 0}, b{0, 0, 0};
  std::vector<uint32_t> req_off{0, 1, 2}, req_q{1, 1}, req_h{100, 200};
  std::vector<uint32_t> layers{2, 2}, hidden{64, 64}, tp{1, 2}, n_launch{0, 2};
  ks_desc d;
  ks_steps s;
  ks_spec spec[2];
  ks_host host{4e-6, 0.0, 0.0, 0.0, 1.0};
  std::vector<double> out;
  ks_step_out so;
  Small() : out(6 * 2) {
    std::memset(&d, 0, sizeof d);
    d.n_rows = 3;
    for (int f = 1; f <= KS_NFAM; ++f) d.fam_off[f] = 3;
    d.step = step.data();
    d.m = m.data();
    d.n = n.data();
    d.k = k.data();
    d.a = a.data();
    d.b = b.data();
    d.n_steps = 2;
    d.req_off = req_off.data();
    d.req_q = req_q.data();
    d.req_h = req_h.data();
    d.n_req = 2;
    d.elem_bytes = 2;
    s = ks_steps{2, layers.data(), hidden.data(), tp.data(), n_launch.data()};
    for (int i = 0; i < 2; ++i) spec[i] = ks_spec{1e15, 4e12, 3e-6, 5e7, 8e-6, 2e-6, 3e11, 64u + i, 0u};
    so = ks_step_out{out.data(), out.data() + 4, out.data() + 8};
  }
};

ks_heads eta_one() {
  ks_heads h;
  std::memset(&h, 0, sizeof h);
  h.mode = KS_ETA_ONE;
  return h;
}

ks_model llama_like() {
  ks_model m;
  std::memset(&m, 0, sizeof m);
  m.hidden = 256;
  m.layers = 4;
  m.q_heads = 8;
  m.kv_heads = 2;
  m.head_dim = 32;
  m.ffn = 688;
  m.vocab = 1000;
  m.tp = 1;
  return m;
}

int run_args() {
  Small x;
  const ks_heads h1 = eta_one();
  const size_t wsb = ks_workspace_bytes(&x.d, 2);
  std::printf("workspace_bytes_positive %d\n", wsb > 0 ? 0 : 1);
  std::printf("workspace_bytes_null %d\n", ks_workspace_bytes(nullptr, 2) == 0 ? 0 : 1);
  Buf ws(wsb);
  report("eval_steps_valid", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  {
    std::vector<float> tk(2 * 3), tr(2 * 3), eta(2 * 3);
    std::vector<uint64_t> F(3), Bt(3), B(3);
    ks_kernel_out ko;
    std::memset(&ko, 0, sizeof ko);
    ko.flops = F.data();
    ko.bytes = Bt.data();
    ko.blocks = B.data();
    ko.t_roof = tr.data();
    ko.eta = eta.data();
    ko.t_kernel = tk.data();
    report("eval_kernels_valid", ks_eval_kernels(&x.d, x.spec, 2, &h1, &ko, ws.p, wsb, nullptr));
    report("eval_kernels_null_out", ks_eval_kernels(&x.d, x.spec, 2, &h1, nullptr, ws.p, wsb, nullptr));
  }
  report("validate_valid", ks_validate(&x.d, &x.s, x.spec, 2, ws.p, wsb, nullptr));
  report("device_status_small_ws", ks_device_status(ws.p, 16, nullptr));
  report("eval_steps_null_desc", ks_eval_steps(nullptr, &x.s, x.spec, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  {
    Small y;
    y.d.fam_off[3] = 1;   // decreases after family 2 (3 -> 1)
    y.d.fam_off[2] = 3;
    report("fam_off_decreasing", ks_eval_steps(&y.d, &y.s, y.spec, 2, &h1, &y.host, &y.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    Small y;
    y.d.fam_off[KS_NFAM] = 2;
    report("fam_off_end_mismatch", ks_eval_steps(&y.d, &y.s, y.spec, 2, &h1, &y.host, &y.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    Small y;
    y.d.n_rows = -1;
    report("n_rows_negative", ks_eval_steps(&y.d, &y.s, y.spec, 2, &h1, &y.host, &y.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    Small y;
    y.d.k = nullptr;
    report("record_array_null", ks_eval_steps(&y.d, &y.s, y.spec, 2, &h1, &y.host, &y.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    Small y;
    y.d.elem_bytes = 0;
    report("elem_bytes_zero", ks_eval_steps(&y.d, &y.s, y.spec, 2, &h1, &y.host, &y.so, nullptr, ws.p, wsb, nullptr));
  }
  report("n_specs_zero", ks_eval_steps(&x.d, &x.s, x.spec, 0, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  report("specs_null", ks_eval_steps(&x.d, &x.s, nullptr, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  report("ws_null", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, &x.host, &x.so, nullptr, nullptr, wsb, nullptr));
  report("ws_small", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb - 8, nullptr));
  report("ws_misaligned", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, &x.host, &x.so, nullptr,
                                        static_cast<char *>(ws.p) + 8, wsb, nullptr));
  {
    ks_heads h = eta_one();
    h.mode = 7;
    report("heads_mode_unknown", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  }
  std::vector<float> wts(1 << 16, 0.0f);
  {
    ks_heads h = eta_one();
    h.mode = KS_ETA_MLP;
    h.precision = KS_F32;
    h.in_dim = 17;
    h.hidden = 64;
    h.w1 = h.w2 = h.b2 = h.w3 = h.b3 = wts.data();
    report("heads_in_dim_17", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.in_dim = 16;
    h.precision = KS_BF16;
    h.hidden = 96;
    report("heads_bf16_hidden_96", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.hidden = 128;
    h.w3 = nullptr;
    report("heads_weight_null", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.w3 = wts.data();
    report("heads_bf16_16_128_valid", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    ks_heads h = eta_one();
    h.bounded_mask = 1u << KS_NFAM;
    h.bounded = wts.data();
    report("bounded_mask_beyond", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.bounded_mask = 1;
    h.bounded = nullptr;
    report("bounded_null", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    ks_heads h = eta_one();
    h.grid_mask = 1;
    h.grid = wts.data();
    for (int d = 0; d < 3; ++d) {
      h.grid_axis[d] = d;
      h.grid_n[d] = 4;
      h.grid_lo[d] = 0.0;
      h.grid_hi[d] = 1.0;
    }
    report("grid_valid", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.grid_n[1] = 1;
    report("grid_n_1", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.grid_n[1] = 4;
    h.grid_hi[2] = h.grid_lo[2];
    report("grid_empty_range", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.grid_hi[2] = 1.0;
    h.grid_axis[0] = 15;
    report("grid_axis_15", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    h.grid_axis[0] = 0;
    h.grid_n[0] = h.grid_n[1] = h.grid_n[2] = 16;
    report("grid_too_many_nodes", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
  }
  {
    ks_steps s = x.s;
    s.n_steps = 3;
    report("steps_count_mismatch", ks_eval_steps(&x.d, &s, x.spec, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    s = x.s;
    s.tp = nullptr;
    report("steps_array_null", ks_eval_steps(&x.d, &s, x.spec, 2, &h1, &x.host, &x.so, nullptr, ws.p, wsb, nullptr));
    report("host_null", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, nullptr, &x.so, nullptr, ws.p, wsb, nullptr));
    ks_step_out so = x.so;
    so.t_gpu = nullptr;
    report("step_out_null", ks_eval_steps(&x.d, &x.s, x.spec, 2, &h1, &x.host, &so, nullptr, ws.p, wsb, nullptr));
  }
  {
    // an empty record set over no steps is a valid (empty) call
    ks_desc d;
    std::memset(&d, 0, sizeof d);
    d.req_off = x.req_off.data();
    d.elem_bytes = 2;
    ks_steps s{0, nullptr, nullptr, nullptr, nullptr};
    ks_step_out so{nullptr, nullptr, nullptr};
    const size_t eb = ks_workspace_bytes(&d, 1);
    Buf w(eb);
    report("empty_call", ks_eval_steps(&d, &s, x.spec, 1, &h1, &x.host, &so, nullptr, w.p, eb, nullptr));
  }
  // batch expansion: layouts and plans
  {
    int64_t fo[KS_NFAM + 1];
    ks_model m = llama_like();
    report("expand_layout_valid", ks_expand_layout(&m, 10, 3, KS_EXPAND_PER_LAYER, fo));
    // 9 kernels per layer + embedding + LM head per step
    std::printf("expand_layout_records %lld\n", (long long)fo[KS_NFAM]);
    report("expand_layout_homogeneous", ks_expand_layout(&m, 10, 3, KS_EXPAND_HOMOGENEOUS, fo));
    std::printf("expand_layout_homogeneous_records %lld\n", (long long)fo[KS_NFAM]);
    report("expand_layout_null_fam_off", ks_expand_layout(&m, 10, 3, KS_EXPAND_PER_LAYER, nullptr));
    report("expand_layout_prefill_gt_steps", ks_expand_layout(&m, 10, 11, KS_EXPAND_PER_LAYER, fo));
    report("expand_layout_mode_unknown", ks_expand_layout(&m, 10, 3, 5, fo));
    ks_model b = m;
    b.hidden = 0;
    report("expand_layout_hidden_0", ks_expand_layout(&b, 10, 3, KS_EXPAND_PER_LAYER, fo));
    b = m;
    b.tp = 3;
    report("expand_layout_tp_not_dividing", ks_expand_layout(&b, 10, 3, KS_EXPAND_PER_LAYER, fo));
    b = m;
    b.experts = 8;
    b.top_k = 9;
    b.expert_ffn = 512;
    report("expand_layout_top_k_above_experts", ks_expand_layout(&b, 10, 3, KS_EXPAND_PER_LAYER, fo));
    b.top_k = 2;
    report("expand_layout_moe_valid", ks_expand_layout(&b, 10, 3, KS_EXPAND_PER_LAYER, fo));
    std::printf("expand_layout_moe_records %lld\n", (long long)fo[KS_NFAM]);
    b = m;
    b.ffn = 1u << 20;
    report("expand_layout_n_too_wide", ks_expand_layout(&b, 10, 3, KS_EXPAND_PER_LAYER, fo));
    std::printf("expand_ws_negative %d\n", ks_expand_workspace_bytes(-1) == 0 ? 0 : 1);

    // a two-step batch expanded into host records
    std::vector<uint32_t> off{0, 2, 3}, q{5, 1, 1};
    std::vector<uint8_t> pre{1, 0};
    ks_batch bt{2, off.data(), q.data(), 3, pre.data(), 1};
    ks_expand_layout(&m, 2, 1, KS_EXPAND_PER_LAYER, fo);
    const size_t R = (size_t)fo[KS_NFAM];
    std::vector<uint32_t> rec(7 * R + 8);
    ks_records out{rec.data(), rec.data() + R, rec.data() + 2 * R, rec.data() + 3 * R, rec.data() + 4 * R,
                   rec.data() + 5 * R, nullptr, rec.data() + 6 * R, rec.data() + 6 * R + 2,
                   rec.data() + 6 * R + 4, rec.data() + 6 * R + 6};
    const size_t eb = ks_expand_workspace_bytes(2);
    Buf w(eb);
    report("expand_valid", ks_expand(&m, &bt, KS_EXPAND_PER_LAYER, &out, w.p, eb, nullptr));
    report("expand_ws_small", ks_expand(&m, &bt, KS_EXPAND_PER_LAYER, &out, w.p, eb - 4, nullptr));
    report("expand_batch_null", ks_expand(&m, nullptr, KS_EXPAND_PER_LAYER, &out, w.p, eb, nullptr));
    ks_batch bad = bt;
    bad.n_prefill = 3;
    report("expand_n_prefill_above_steps", ks_expand(&m, &bad, KS_EXPAND_PER_LAYER, &out, w.p, eb, nullptr));
  }
  // serving simulation: argument checks
  {
    ks_model m = llama_like();
    ks_sched sc{8, 256, 16, 1, 4096};
    std::vector<double> arr{0.0, 0.5, 0.25};
    std::vector<uint32_t> prompt{10, 20, 30}, output{2, 3, 4};
    ks_requests rq{3, arr.data(), prompt.data(), output.data(), nullptr, nullptr};
    ks_sim_out so;
    std::memset(&so, 0, sizeof so);
    const size_t sb = ks_simulate_workspace_bytes(&m, &sc, 1);
    Buf w(sb);
    ks_host host{4e-6, 0.0, 0.0, 0.0, 1.0};
    report("simulate_unsorted_arrivals", ks_simulate(&m, x.spec, 1, &h1, &host, &sc, &rq, &so, w.p, sb, nullptr));
    arr[2] = 1.0;
    prompt[1] = 0;
    report("simulate_zero_prompt", ks_simulate(&m, x.spec, 1, &h1, &host, &sc, &rq, &so, w.p, sb, nullptr));
    prompt[1] = 20;
    report("simulate_n_specs_0", ks_simulate(&m, x.spec, 0, &h1, &host, &sc, &rq, &so, w.p, sb, nullptr));
    ks_model moe = m;
    moe.experts = 8;
    moe.top_k = 2;
    moe.expert_ffn = 512;
    report("simulate_moe_rejected", ks_simulate(&moe, x.spec, 1, &h1, &host, &sc, &rq, &so, w.p, sb, nullptr));
    ks_sched bad = sc;
    bad.block_tokens = 0;
    report("simulate_block_tokens_0", ks_simulate(&m, x.spec, 1, &h1, &host, &bad, &rq, &so, w.p, sb, nullptr));
    report("simulate_ws_small", ks_simulate(&m, x.spec, 1, &h1, &host, &sc, &rq, &so, w.p, sb - 256, nullptr));
    std::vector<uint32_t> group{1, 1, 0};
    ks_requests rg = rq;
    rg.group = group.data();
    report("simulate_group_without_prefix", ks_simulate(&m, x.spec, 1, &h1, &host, &sc, &rg, &so, w.p, sb, nullptr));
    report("simulate_valid", ks_simulate(&m, x.spec, 1, &h1, &host, &sc, &rq, &so, w.p, sb, nullptr));
    std::printf("simulate_valid_steps %lld\n", (long long)so.n_steps);
  }
  return 0;
}

int run_sim() {
  ks_model m;
  std::memset(&m, 0, sizeof m);
  ks_sched sc;
  int n_specs = 0;
  long long n = 0;
  if (std::scanf("%u %u %u %u %u %u %u %u", &m.hidden, &m.layers, &m.q_heads, &m.kv_heads, &m.head_dim, &m.ffn,
                 &m.vocab, &m.tp) != 8)
    return 2;
  long long kv_blocks = 0;
  if (std::scanf("%d %d %d %d %lld", &sc.max_num_seqs, &sc.max_batched_tokens, &sc.block_tokens, &sc.prefix_cache,
                 &kv_blocks) != 5)
    return 2;
  sc.kv_blocks = kv_blocks;
  if (std::scanf("%d %lld", &n_specs, &n) != 2 || n_specs < 1 || n < 0) return 2;
  std::vector<double> arrival((size_t)n);
  std::vector<uint32_t> prompt((size_t)n), output((size_t)n), group((size_t)n), prefix((size_t)n);
  char tok[64];
  for (long long i = 0; i < n; ++i) {
    if (std::scanf("%63s %u %u %u %u", tok, &prompt[(size_t)i], &output[(size_t)i], &group[(size_t)i],
                   &prefix[(size_t)i]) != 5)
      return 2;
    arrival[(size_t)i] = std::strtod(tok, nullptr);   // hexadecimal floats are exact
  }
  ks_requests rq{n, arrival.data(), prompt.data(), output.data(), group.data(), prefix.data()};
  std::vector<ks_spec> specs((size_t)n_specs);
  for (int s = 0; s < n_specs; ++s) specs[(size_t)s] = ks_spec{1e15, 4e12, 3e-6, 5e7, 8e-6, 2e-6, 3e11, 132u, 0u};
  const ks_heads h = eta_one();
  ks_host host{4e-6, 0.0, 0.0, 0.0, 1.0};
  const int64_t cap = 1 << 16, ecap = 1 << 20;
  struct Out {
    std::vector<double> ttft, tpot, e2e, start, lat;
    std::vector<int32_t> state;
    std::vector<uint8_t> pre;
    std::vector<int64_t> off;
    std::vector<uint32_t> er, eq, eh;
  };
  std::vector<Out> o((size_t)n_specs);
  std::vector<ks_sim_out> so((size_t)n_specs);
  for (int s = 0; s < n_specs; ++s) {
    Out &x = o[(size_t)s];
    x.ttft.resize((size_t)n);
    x.tpot.resize((size_t)n);
    x.e2e.resize((size_t)n);
    x.state.resize((size_t)n);
    x.start.resize(cap);
    x.lat.resize(cap);
    x.pre.resize(cap);
    x.off.resize(cap + 1);
    x.er.resize(ecap);
    x.eq.resize(ecap);
    x.eh.resize(ecap);
    so[(size_t)s] = ks_sim_out{x.ttft.data(), x.tpot.data(), x.e2e.data(), x.state.data(), cap, ecap,
                               x.start.data(), x.lat.data(), x.pre.data(), x.off.data(), x.er.data(),
                               x.eq.data(), x.eh.data(), 0, 0, 0, 0.0};
  }
  const size_t wsb = ks_simulate_workspace_bytes(&m, &sc, n_specs);
  if (!wsb) {
    std::printf("status %d %s\n", (int)KS_EINVAL, ks_last_error());
    return 0;
  }
  Buf ws(wsb);
  const ks_status st = ks_simulate(&m, specs.data(), n_specs, &h, &host, &sc, &rq, so.data(), ws.p, wsb, nullptr);
  std::printf("status %d\n", (int)st);
  if (st != KS_OK) return 0;
  for (int s = 0; s < n_specs; ++s) {
    const ks_sim_out &r = so[(size_t)s];
    const Out &x = o[(size_t)s];
    std::printf("sim %d %lld %lld %a\n", s, (long long)r.n_steps, (long long)r.preemptions, r.clock);
    for (int64_t i = 0; i < r.n_steps && i < cap; ++i) {
      std::printf("step %a %a %d", x.start[(size_t)i], x.lat[(size_t)i], (int)x.pre[(size_t)i]);
      for (int64_t j = x.off[(size_t)i]; j < x.off[(size_t)i + 1]; ++j)
        std::printf(" %u:%u:%u", x.er[(size_t)j], x.eq[(size_t)j], x.eh[(size_t)j]);
      std::printf("\n");
    }
    for (long long i = 0; i < n; ++i)
      std::printf("req %d %a %a %a\n", x.state[(size_t)i], x.ttft[(size_t)i], x.tpot[(size_t)i], x.e2e[(size_t)i]);
  }
  return 0;
}

}  // namespace

int main(int argc, char **argv) {
  if (argc == 2 && std::string(argv[1]) == "args") return run_args();
  if (argc == 2 && std::string(argv[1]) == "sim") return run_sim();
  std::fprintf(stderr, "usage: host_driver args|sim\n");
  return 2;
}
