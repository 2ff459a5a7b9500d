"""Pins of the fp64 oracle against what the paper and the mathematics fix:
the paper's worked example, closed forms, brute-force enumeration on tiny
inputs, and special cases that reduce to textbook results."""
import math
import os

import numpy as np
import pytest

from oracle import ks_oracle as o
from oracle import metrics
from workload import gen
from tests import brute
from tests.helpers import make_desc, spec, steprec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [line.split() for line in f if line.strip() and not line.startswith("#")]


# ---------------------------------------------------------------- waves ----
def test_wave_quantization_worked_example():
    (B, N, W, idle, un, ud), = [[int(v) for v in r] for r in _golden("wave_quantization.txt")]
    Wo, u = o.waves(np.array([B], np.uint64), N)
    assert int(Wo[0]) == W
    assert u[0] == pytest.approx(un / ud, rel=0, abs=1e-15)
    bw, bidle = brute.dispatch_waves(B, N)
    assert (bw, bidle) == (W, idle)


@pytest.mark.parametrize("B,N", [(1, 4), (4, 4), (5, 4), (100, 7), (128, 132), (133, 132), (1000, 148)])
def test_waves_match_dispatch_simulation(B, N):
    W, u = o.waves(np.array([B], np.uint64), N)
    bw, _ = brute.dispatch_waves(B, N)
    assert int(W[0]) == bw
    assert u[0] == pytest.approx(bw * N / B, rel=1e-15)
    assert u[0] >= 1.0


def test_waves_zero_blocks():
    W, u = o.waves(np.array([0], np.uint64), 132)
    assert int(W[0]) == 0 and u[0] == 1.0


# ---------------------------------------------------------------- counts ---
@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (3, 5, 7), (130, 2, 3), (2, 129, 4)])
def test_gemm_counts_brute(M, N, K):
    d = make_desc([(gen.GEMM, 0, M, N, K, 0, 0), (gen.LM_HEAD, 0, M, N, K, 0, 0)], [[(1, 0)]])
    c = o.kernel_counts(d)
    F, Bt = brute.gemm_work(M, N, K, 2)
    assert [int(v) for v in c["F"]] == [F, F]
    assert [int(v) for v in c["Bt"]] == [Bt, Bt]
    assert int(c["B"][0]) == brute.tiles_2d(M, N, 128)
    assert int(c["F"][0]) == 2 * M * N * K          # closed form GEMM FLOPs = 2MNK


def test_gemm_flops_closed_form_large():
    M, N, K = 4096, 11008, 4096
    d = make_desc([(gen.GEMM, 0, M, N, K, 0, 0)], [[(1, 0)]])
    assert int(o.kernel_counts(d)["F"][0]) == 2 * M * N * K


REQ_CASES = [
    [(1, 0)],
    [(1, 5)],
    [(3, 0)],
    [(4, 2), (1, 7), (1, 0)],
    [(130, 3), (1, 9)],
    [(257, 0)],
]


@pytest.mark.parametrize("reqs", REQ_CASES)
@pytest.mark.parametrize("fam", [gen.ATTN_PREFILL, gen.ATTN_DECODE])
def test_attention_counts_brute(reqs, fam):
    H, Hkv, dd = 3, 2, 2
    d = make_desc([(fam, 0, 0, H, dd, Hkv, 0)], [reqs])
    c = o.kernel_counts(d)
    F, Bt, B, pairs = brute.attention_work(reqs, H, Hkv, dd, 2)
    assert int(c["F"][0]) == F
    assert int(c["Bt"][0]) == Bt
    assert int(c["B"][0]) == B
    assert int(o.attention_work(d.req_off, d.req_q, d.req_h)["PAIRS"][0]) == pairs
    assert int(c["M"][0]) == sum(q for q, _ in reqs)


def test_attention_uses_own_step_requests():
    reqs = [[(1, 10)], [(5, 0), (1, 3)]]
    d = make_desc([(gen.ATTN_DECODE, 0, 0, 2, 4, 1, 0), (gen.ATTN_PREFILL, 1, 0, 2, 4, 1, 0)], reqs)
    c = o.kernel_counts(d)
    # family-major: PREFILL (step 1) comes before DECODE (step 0)
    F1, _, _, _ = brute.attention_work(reqs[1], 2, 1, 4, 2)
    F0, _, _, _ = brute.attention_work(reqs[0], 2, 1, 4, 2)
    assert [int(v) for v in c["F"]] == [F1, F0]


def test_grouped_gemm_counts_brute():
    experts = [5, 0, 130, 1]          # ragged M_e, one empty expert
    N, K = 3, 4
    d = make_desc([(gen.GROUPED_GEMM, 0, 0, N, K, len(experts), 2)], [[(1, 0)]],
                  expert_rows=[9, 9] + experts)
    c = o.kernel_counts(d)
    F = Bt = B = 0
    for me in experts:                 # one GEMM per non-empty expert
        if me == 0:
            continue
        f, bt = brute.gemm_work(me, N, K, 2)
        F += f
        Bt += bt
        B += brute.tiles_2d(me, N, 128)
    assert int(c["F"][0]) == F
    assert int(c["Bt"][0]) == Bt
    assert int(c["B"][0]) == B
    assert int(c["M"][0]) == sum(experts)


_ELEMENTWISE_BRUTE = {
    gen.RMSNORM: lambda m, n, k: brute.rmsnorm_work(m, n, 2),
    gen.ROPE: lambda m, n, k: brute.rope_work(m, n, k, 2),
    gen.SILU_MUL: lambda m, n, k: brute.silu_mul_work(m, n, 2),
    gen.KV_WRITE: lambda m, n, k: brute.kv_write_work(m, n, k, 2),
    gen.EMBED: lambda m, n, k: brute.embed_work(m, n, 2),
}


@pytest.mark.parametrize("fam", [gen.RMSNORM, gen.ROPE, gen.SILU_MUL, gen.KV_WRITE, gen.EMBED])
@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (7, 3, 2), (300, 5, 3), (37, 29, 4)])
def test_elementwise_counts_brute(fam, m, n, k):
    """F, Bt and B of the norm, rotary, activation, KV-write and embedding
    records against their kernels enumerated element by element (the
    operations of each element's expression, the distinct elements read and
    written, the blocks the grid mapping touches).  (300, 5) and (37, 29)
    span several 1024-element SiLU blocks with a ragged last one."""
    d = make_desc([(fam, 0, m, n, k, 0, 0)], [[(1, 0)]])
    c = o.kernel_counts(d)
    F, Bt, B = _ELEMENTWISE_BRUTE[fam](m, n, k)
    assert (int(c["F"][0]), int(c["Bt"][0]), int(c["B"][0])) == (F, Bt, B)


def test_unused_k_is_ignored_by_the_features():
    """Norm, activation and embedding records carry no K: whatever their k
    field holds, feature x12 (the K shape feature) is 0 and their latency is
    the same as with k = 0; the families that have a K (GEMM, LM head,
    grouped GEMM, attention, RoPE, KV write) take log2(1 + k) / 24 from it
    (Sec. 5.3: shape features per family)."""
    k = 77
    rows = [(gen.GEMM, 0, 5, 9, k, 0, 0), (gen.LM_HEAD, 0, 2, 9, k, 0, 0),
            (gen.GROUPED_GEMM, 0, 0, 9, k, 2, 0), (gen.ATTN_DECODE, 0, 0, 4, k, 2, 0),
            (gen.RMSNORM, 0, 5, 64, k, 0, 0), (gen.ROPE, 0, 5, 6, k, 0, 0),
            (gen.SILU_MUL, 0, 5, 64, k, 0, 0), (gen.KV_WRITE, 0, 5, 2, k, 0, 0),
            (gen.EMBED, 0, 5, 64, k, 0, 0)]
    d = make_desc(rows, [[(1, 30), (1, 4)]], expert_rows=[3, 2])
    heads = gen.make_heads(16, 8, "f32")
    sp = spec()
    r = o.eval_kernels(d, sp, heads, keep_features=True)
    fam = d.family()
    unused = np.isin(fam, [gen.RMSNORM, gen.SILU_MUL, gen.EMBED])
    assert unused.sum() == 3 and (~unused).sum() == 6
    x12 = r["x"][0, :, 12]
    assert (x12[unused] == 0.0).all()
    np.testing.assert_allclose(x12[~unused], math.log2(1 + k) / 24, rtol=1e-15)
    # the same records with k = 0 where it is unused: identical predictions
    rows0 = [rw if rw[0] not in (gen.RMSNORM, gen.SILU_MUL, gen.EMBED) else rw[:4] + (0,) + rw[5:]
             for rw in rows]
    r0 = o.eval_kernels(make_desc(rows0, [[(1, 30), (1, 4)]], expert_rows=[3, 2]), sp, heads)
    np.testing.assert_array_equal(r["z"], r0["z"])
    np.testing.assert_array_equal(r["t"], r0["t"])
    # and a K that the family has does change its prediction
    rows1 = [rw if rw[0] != gen.ROPE else rw[:4] + (3,) + rw[5:] for rw in rows]
    r1 = o.eval_kernels(make_desc(rows1, [[(1, 30), (1, 4)]], expert_rows=[3, 2]), sp, heads)
    rope = fam == gen.ROPE
    assert (r1["z"][:, rope] != r["z"][:, rope]).all()
    np.testing.assert_array_equal(r1["z"][:, ~rope], r["z"][:, ~rope])


# ---------------------------------------------------------------- roofline -
def test_roofline_textbook_when_waves_full():
    """eta = 1, t0 = 0 and B a multiple of N: t = max(F/P, Bt/BW)."""
    M = N = 128 * 4
    K = 256
    d = make_desc([(gen.GEMM, 0, M, N, K, 0, 0)], [[(1, 0)]])
    sp = spec(P=1e15, BW=4e12, n_cu=16, t0=0.0)
    k = o.eval_kernels(d, sp, eta_one=True)
    F = 2 * M * N * K
    Bt = 2 * (M * K + K * N + M * N)
    assert k["t"][0, 0] == pytest.approx(max(F / 1e15, Bt / 4e12), rel=1e-15)


def test_roofline_partial_wave_inflates_compute_only():
    d = make_desc([(gen.GEMM, 0, 128 * 9, 128, 4096, 0, 0),      # 9 blocks
                   (gen.RMSNORM, 0, 9, 64, 0, 0, 0)], [[(1, 0)]])  # 9 blocks, memory-bound
    sp = spec(P=1e12, BW=1e15, n_cu=4, t0=0.0)
    k = o.eval_kernels(d, sp, eta_one=True)
    F = 2 * 128 * 9 * 128 * 4096
    assert k["t_comp"][0, 0] == pytest.approx(F / 1e12 * 12 / 9, rel=1e-15)
    Bt_norm = 2 * (2 * 9 * 64 + 64)
    assert k["t_mem"][0, 1] == pytest.approx(Bt_norm / 1e15, rel=1e-15)


def test_launch_floor_after_eta():
    """t = max(t_roof eta, t0): with eta = 2 and t_roof = 0.75 t0 the floor
    does not bind (1.5 t0); flooring before scaling would give 2 t0."""
    t0 = 1e-6
    assert o.kernel_latency(0.75 * t0, 2.0, t0) == pytest.approx(1.5 * t0)
    assert o.kernel_latency(0.25 * t0, 2.0, t0) == t0


def test_zero_work_kernel_pays_floor():
    d = make_desc([(gen.EMBED, 0, 0, 64, 0, 0, 0)], [[(1, 0)]])
    sp = spec(t0=3e-6)
    k = o.eval_kernels(d, sp, heads=gen.make_heads(16, 8, "f32"))
    assert k["t"][0, 0] == 3e-6


# ---------------------------------------------------------------- features -
def test_features_hand_example():
    """GEMM 128^3, dt = 2, P = 2^50, BW = 2^40, N = 4, L2 = 2^20, t0 = 2^-20:
    F = 2^22, Bt = 3 2^15, B = 1, W = 1, u = 4, AI = 2^7/3,
    t_comp = 2^-26, t_mem = 3 2^-25."""
    d = make_desc([(gen.GEMM, 0, 128, 128, 128, 0, 0)], [[(1, 0)]])
    sp = o.spec_at(spec(), 0)
    c = o.kernel_counts(d)
    rf = o.roofline(c["F"], c["Bt"], c["B"], sp)
    x = o.features(c, d.n, d.k, rf, sp)[0]
    l3 = math.log2(3)
    want = [(7 - l3) / 16, (-3 - l3) / 16, math.log2(5 / 4) / 16, 1 / 4, 1 / 16, 1.0,
            (l3 - 5) / 16, 1 / 7, math.log2(1 + 2 ** 22) / 64, math.log2(1 + 98304) / 48,
            math.log2(129) / 24, math.log2(129) / 24, math.log2(129) / 24,
            math.log2(1 + 2 ** 22) / 48, math.log2(1 + 98304) / 40, 1.0]
    np.testing.assert_allclose(x, want, rtol=1e-14, atol=1e-15)
    x32 = o.features(c, d.n, d.k, rf, sp, in_dim=32)[0]
    np.testing.assert_allclose(x32[16:], np.square(want), rtol=1e-14, atol=1e-15)


def test_features_zero_work_limits():
    d = make_desc([(gen.EMBED, 0, 0, 64, 0, 0, 0)], [[(1, 0)]])
    sp = o.spec_at(spec(), 0)
    c = o.kernel_counts(d)
    rf = o.roofline(c["F"], c["Bt"], c["B"], sp)
    x = o.features(c, d.n, o.effective_k(d, np.arange(1)), rf, sp)[0]
    assert x[0] == -10 / 16 and x[1] == -20 / 16 and x[6] == -20 / 16
    assert x[3] == 1.0 and x[4] == 0.0 and x[5] == 1.0 and x[7] == 0.0


# ---------------------------------------------------------------- head -----
def test_head_zero_weights_closed_form():
    """All weights zero: z = b3 and eta = 1 + e^-b3; sigma = 1/eta in (0, 1]."""
    H = 8
    x = np.random.default_rng(0).normal(size=(5, 16))
    for b3 in (-2.0, 0.0, 0.7):
        z = o.head_forward(x, np.zeros((H, 16)), np.zeros((H, H)), np.zeros(H), np.zeros(H), b3)
        np.testing.assert_array_equal(z, b3)
        eta = o.eta_from_z(z)
        assert eta[0] == pytest.approx(1 + math.exp(-b3), rel=1e-15)
        assert 0 < 1 / eta[0] <= 1


def test_head_hand_example():
    """in 2, hidden 2: W1 = [[1, -1], [2, 0]], x = (3, 1) -> h1 = (2, 6);
    W2 = [[1, 1], [-1, 0]], b2 = (0.5, 1) -> h2 = relu(8.5, -1) = (8.5, 0);
    w3 = (0.25, 9), b3 = -1 -> z = 1.125."""
    z = o.head_forward(np.array([[3.0, 1.0]]), np.array([[1.0, -1.0], [2.0, 0.0]]),
                       np.array([[1.0, 1.0], [-1.0, 0.0]]), np.array([0.5, 1.0]),
                       np.array([0.25, 9.0]), -1.0)
    assert z[0] == 1.125


@pytest.mark.parametrize("precision,in_dim,hidden", [("f32", 16, 64), ("bf16", 16, 128), ("bf16", 32, 16)])
def test_head_matches_scalar_loops(precision, in_dim, hidden):
    heads = gen.make_heads(in_dim, hidden, precision, std=0.5)
    rng = np.random.default_rng(1)
    x = rng.normal(size=(3, in_dim))
    f = 4
    emu = precision == "bf16"
    z = o.head_forward(x, heads.w1[f], heads.w2[f], heads.b2[f], heads.w3[f], heads.b3[f], emu)
    rnd = brute.bf16_scalar if emu else (lambda v: v)
    for i in range(3):
        zb = brute.mlp_scalar(list(x[i]), heads.w1[f].tolist(), heads.w2[f].tolist(),
                              heads.b2[f].tolist(), heads.w3[f].tolist(), float(heads.b3[f]), rnd)
        assert z[i] == pytest.approx(zb, rel=1e-12, abs=1e-12)


def test_bf16_rounding_ties_and_library():
    import torch
    # hand-worked ties: 1 + 2^-8 sits halfway between 1 and 1 + 2^-7 -> even (1);
    # 1 + 3 2^-8 sits halfway between 1 + 2^-7 and 1 + 2^-6 -> even (1 + 2^-6)
    assert o.round_bf16(1 + 2 ** -8) == 1.0
    assert o.round_bf16(1 + 3 * 2 ** -8) == 1 + 2 ** -6
    assert o.round_bf16(-(1 + 3 * 2 ** -8)) == -(1 + 2 ** -6)
    assert o.round_bf16(1 + 2 ** -8 + 2 ** -30) == 1 + 2 ** -7
    # float32-representable values: agree with torch's float32 -> bfloat16
    v = np.random.default_rng(2).normal(scale=3.0, size=20000).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(o.round_bf16(v.astype(np.float64)), ref)
    for val in v[:200]:
        assert o.round_bf16(float(val)) == brute.bf16_scalar(float(val))


# ---------------------------------------------------------------- steps ----
def test_allreduce_closed_forms():
    S, beta, a0, al = 1 << 20, 100e9, 5e-6, 1e-6
    assert o.allreduce_time(1, S, a0, al, beta) == 0.0
    assert o.allreduce_time(2, S, a0, al, beta) == pytest.approx(a0 + al + S / beta, rel=1e-15)
    big = 1 << 20
    t = o.allreduce_time(big, S, 0.0, 0.0, beta)
    assert t == pytest.approx(2 * S / beta, rel=1e-5)
    for P in (2, 3, 4, 8, 16):
        sent = brute.ring_allreduce_bytes(P, S)
        assert o.allreduce_time(P, S, 0.0, 0.0, beta) == pytest.approx(sent / beta, rel=1e-14)


def test_assembly_closed_forms():
    g = np.array([1e-3, 5e-3])
    np.testing.assert_array_equal(o.step_assembly(g, np.array([3.0, 0.0]), 0, 0, 0, 0), g)
    # host overlap floor above the GPU body: c_ovl + n c_disp + c_tail
    t = o.step_assembly(np.array([1e-3]), np.array([2.0]), 1e-5, 0.0, 4e-3, 2e-4)
    assert t[0] == pytest.approx(1e-3 + 2e-5 + 3e-3 + 2e-4)
    # host floor l binds
    t = o.step_assembly(np.array([1e-4]), np.array([0.0]), 0.0, 2e-3, 0.0, 0.0)
    assert t[0] == 2e-3


def test_assembly_not_above_additive():
    rng = np.random.default_rng(3)
    g = rng.uniform(0, 1e-2, 1000)
    n = rng.integers(0, 80, 1000).astype(float)
    cd, ell, co, ct = 4e-6, 1.5e-3, 2.5e-3, 3e-4
    t = o.step_assembly(g, n, cd, ell, co, ct)
    assert (t <= g + n * cd + ell + co + ct + 1e-18).all()


def test_step_body_equals_loop_sum():
    w = gen.config1(0, 12)
    k = o.eval_kernels(w.desc, w.specs, w.heads)
    s = o.eval_steps(w.desc, w.steps, w.specs, w.host, w.heads, kern=k)
    for si in range(2):
        acc = [0.0] * w.desc.n_steps
        for i in range(w.desc.n_rows):
            acc[int(w.desc.step[i])] += float(k["t"][si, i])
        np.testing.assert_allclose(s["t_body"][si], acc, rtol=1e-13)
        # t_gpu = body_scale * body (TP 1: no all-reduce)
        np.testing.assert_allclose(s["t_gpu"][si], w.host.body_scale * np.array(acc), rtol=1e-13)


def test_step_comm_two_allreduces_per_layer():
    reqs = [[(5, 10), (1, 3)]]
    d = make_desc([(gen.EMBED, 0, 6, 64, 0, 0, 0)], reqs)
    sp = spec(t0=0.0)
    rec = steprec(1, layers=3, hidden=64, tp=4)
    host = gen.HostConsts(0.0, 0.0, 0.0, 0.0, 1.0)
    s = o.eval_steps(d, rec, sp, host, eta_one=True)
    S = 6 * 64 * 2
    t_ar = 8e-6 + 2e-6 * 2 + 2 * 3 / 4 * S / 300e9
    assert s["t_comm"][0, 0] == pytest.approx(2 * 3 * t_ar, rel=1e-14)
    assert s["t_step"][0, 0] == pytest.approx(s["t_body"][0, 0] + 2 * 3 * t_ar, rel=1e-14)


# ---------------------------------------------------------------- metrics --
def test_metrics_appendix():
    assert metrics.mape([110, 90], [100, 100]) == pytest.approx(10.0)
    np.testing.assert_allclose(metrics.abs_pct_err([1.5], [1.0]), [50.0])
    e = [5, 1, 4, 2, 3]
    assert metrics.percentile_nearest_rank(e, 50) == 3      # k = ceil(2.5) = 3
    assert metrics.percentile_nearest_rank(e, 90) == 5      # k = ceil(4.5) = 5
    assert metrics.percentile_nearest_rank(e, 20) == 1      # k = 1


# ---------------------------------------- bounded analytical head (Sec. 5.3) --
def test_bounded_head_zero_weights_closed_form():
    """g = a = 0: gamma = 1/2, alpha = 1/4, so eta = 1/(1/2 - 1/(4W)): 4 at
    one wave, 8/3 at two, toward 2 (= 1/gamma) as the waves grow; a record
    without blocks counts as one wave."""
    x = np.random.default_rng(0).normal(size=(4, 16))
    z = np.zeros(16)
    eta = o.bounded_eta(x, np.array([1, 2, 4, 0]), z, z)
    np.testing.assert_allclose(eta, [4.0, 8.0 / 3.0, 1.0 / (0.5 - 1.0 / 16), 4.0], rtol=1e-15)
    assert abs(o.bounded_eta(x[:1], np.array([10 ** 12]), z, z)[0] - 2.0) < 1e-11


def test_bounded_head_hand_example():
    """Only the constant feature x15 = 1 and g15 = ln 3: gamma = 3/4; a = 0:
    alpha = 3/8; at W = 3 the utilization is 3/4 - 1/8 = 5/8, eta = 1.6."""
    x = np.zeros((1, 16))
    x[0, 15] = 1.0
    g = np.zeros(16)
    g[15] = math.log(3.0)
    eta = o.bounded_eta(x, np.array([3]), g, np.zeros(16))
    assert abs(eta[0] - 1.6) < 1e-15


def test_bounded_head_monotone_and_bounded():
    """Random heads: eta >= 1 / gamma > 1, and eta falls as the wave count
    grows (the monotone wave-quantization prior the form imposes)."""
    rng = np.random.default_rng(5)
    x = rng.normal(size=(200, 16))
    g, a = rng.normal(size=16), rng.normal(size=16)
    gamma = 1.0 / (1.0 + np.exp(-(x @ g)))
    prev = None
    for w in (1, 2, 3, 7, 100, 10 ** 6):
        eta = o.bounded_eta(x, np.full(200, w), g, a)
        assert (eta >= 1.0 / gamma - 1e-12).all() and (eta > 1.0).all()
        if prev is not None:
            assert (eta < prev).all()
        prev = eta


def test_bounded_mask_selects_per_family():
    """Families in the mask take the bounded head, the others keep theirs
    (the MLP, or eta = 1), bit for bit."""
    wl = gen.config1(0, 30)
    bd = gen.make_bounded(gen.BOUNDED_MIXED)
    fam = wl.desc.family()
    on = ((gen.BOUNDED_MIXED >> fam) & 1).astype(bool)
    assert on.any() and (~on).any()
    for eta_one in (False, True):
        plain = o.eval_kernels(wl.desc, wl.specs, wl.heads, eta_one=eta_one)
        mixed = o.eval_kernels(wl.desc, wl.specs, wl.heads, eta_one=eta_one, bounded=bd)
        np.testing.assert_array_equal(mixed["eta"][:, ~on], plain["eta"][:, ~on])
        np.testing.assert_array_equal(mixed["t_roof"], plain["t_roof"])
        assert (mixed["eta"][:, on] > 1.0).all()
        # zero-weight bounded heads on the same families: the closed form
        zero = gen.Bounded(gen.BOUNDED_MIXED, np.zeros((gen.NFAM, 16)), np.zeros((gen.NFAM, 16)),
                           np.zeros((gen.NFAM, 2, 16), np.float32))
        z = o.eval_kernels(wl.desc, wl.specs, wl.heads, eta_one=eta_one, bounded=zero)
        w = np.maximum(z["W"][:, on].astype(np.float64), 1.0)
        np.testing.assert_allclose(z["eta"][:, on], 1.0 / (0.5 - 0.25 / w), rtol=1e-15)


# ------------------------------------------ Tier B grid interpolation (Sec. 5.5) --
def _grid(values, lo=(-1.0, 0.0, -0.5), hi=(0.5, 0.4, 0.7), axes=(1, 2, 6)):
    v = np.asarray(values, np.float32)
    full = np.broadcast_to(v, (gen.NFAM,) + v.shape).copy()
    return gen.Grid(gen.GRID_ALL, axes, np.asarray(lo, np.float64), np.asarray(hi, np.float64),
                    v.shape, full)


def _coords_to_x16(c, axes=(1, 2, 6)):
    x = np.random.default_rng(1).normal(size=(len(c), 16))
    x[:, list(axes)] = c
    return x


def test_grid_reproduces_node_values():
    """At a node every weight but one vanishes: the node's value."""
    v = np.random.default_rng(2).uniform(1.0, 3.0, size=(4, 5, 3)).astype(np.float32)
    gr = _grid(v)
    idx = np.array(np.meshgrid(*[np.arange(s) for s in v.shape], indexing="ij")).reshape(3, -1).T
    c = gr.lo + idx * (gr.hi - gr.lo) / (np.array(v.shape) - 1)
    eta, routed = o.grid_eta(_coords_to_x16(c), gr, 0)
    assert routed.all()
    np.testing.assert_allclose(eta, v[tuple(idx.T)].astype(np.float64), rtol=1e-14)


def test_grid_reproduces_multilinear_functions():
    """Trilinear interpolation is exact for (a0 + b0 c0)(a1 + b1 c1)(a2 + b2 c2)
    and for sums of such terms (here an affine function plus c0 c1 c2), at any
    point of the box: a dropped weight or a swapped axis fails this."""
    gr0 = _grid(np.zeros((6, 4, 5)))
    n = np.array(gr0.n)
    node = [np.linspace(gr0.lo[d], gr0.hi[d], n[d]) for d in range(3)]
    C = np.meshgrid(*node, indexing="ij")

    def f(c0, c1, c2):
        return 1.5 + 0.7 * c0 - 0.3 * c1 + 0.2 * c2 + 0.9 * c0 * c1 * c2 + 0.4 * c0 * c2

    vals = f(*C)
    gr = gen.Grid(gen.GRID_ALL, gr0.axes, gr0.lo, gr0.hi, gr0.n,
                  np.broadcast_to(vals, (gen.NFAM,) + vals.shape).copy())   # float64 nodes
    rng = np.random.default_rng(3)
    c = gr.lo + rng.uniform(size=(500, 3)) * (gr.hi - gr.lo)
    eta, routed = o.grid_eta(_coords_to_x16(c), gr, 3)
    assert routed.all()
    np.testing.assert_allclose(eta, f(c[:, 0], c[:, 1], c[:, 2]), rtol=1e-13, atol=1e-13)


def test_grid_matches_regular_grid_interpolator():
    """Random node values with unmeasured (NaN) nodes against scipy's
    RegularGridInterpolator: same values where routed, and routed exactly
    where scipy's linear interpolation is not NaN (a NaN corner reaches the
    result whatever its weight)."""
    from scipy.interpolate import RegularGridInterpolator
    rng = np.random.default_rng(4)
    v = rng.uniform(1.0, 4.0, size=(7, 6, 8))
    v[rng.uniform(size=v.shape) < 0.1] = np.nan
    gr = gen.Grid(gen.GRID_ALL, (0, 3, 12), np.array([-0.6, 0.2, 0.1]), np.array([0.0, 1.0, 0.3]), v.shape,
                  np.broadcast_to(v, (gen.NFAM,) + v.shape).copy())
    node = [np.linspace(gr.lo[d], gr.hi[d], v.shape[d]) for d in range(3)]
    ref = RegularGridInterpolator(node, v, method="linear", bounds_error=False, fill_value=np.nan)
    c = gr.lo + rng.uniform(size=(4000, 3)) * (gr.hi - gr.lo)
    eta, routed = o.grid_eta(_coords_to_x16(c, gr.axes), gr, 7)
    r = ref(c)
    np.testing.assert_array_equal(routed, ~np.isnan(r))
    assert 0.2 < routed.mean() < 0.8
    np.testing.assert_allclose(eta[routed], r[routed], rtol=1e-13)


def test_grid_outside_box_or_unmeasured_falls_back():
    """Outside the box, or in a cell with an unmeasured corner, nothing is
    routed; one unmeasured node blocks exactly the (up to 8) cells around it."""
    v = np.full((5, 5, 5), 2.0)
    v[2, 2, 2] = np.nan
    gr = _grid(v)
    n = np.array(v.shape)
    step = (gr.hi - gr.lo) / (n - 1)
    # cell centres: blocked iff the cell touches node (2, 2, 2)
    idx = np.array(np.meshgrid(*[np.arange(4)] * 3, indexing="ij")).reshape(3, -1).T
    c = gr.lo + (idx + 0.5) * step
    _, routed = o.grid_eta(_coords_to_x16(c), gr, 0)
    blocked = np.all((idx == 1) | (idx == 2), axis=1)
    np.testing.assert_array_equal(routed, ~blocked)
    # just outside each face
    for d in range(3):
        for side in (-1, 1):
            p = (gr.lo + gr.hi) / 2
            p[d] = (gr.lo[d] if side < 0 else gr.hi[d]) + side * 1e-9
            _, r = o.grid_eta(_coords_to_x16(p[None]), gr, 0)
            assert not r[0]
    # on the faces themselves: routed (the box is closed)
    _, r = o.grid_eta(_coords_to_x16(np.array([gr.lo, gr.hi])), gr, 0)
    assert r.all()


def test_grid_routing_in_eval_kernels():
    """Per family: routed records take the interpolated eta of their own
    features, the rest keep the family's other head bit for bit (MLP, eta = 1
    or the bounded head); routing does not depend on that other head; an
    all-NaN grid routes nothing."""
    wl = gen.config1(0, 30)
    gr = gen.make_grid(gen.GRID_ALL ^ (1 << gen.GEMM))
    fam = wl.desc.family()
    res = []
    for kw in ({}, {"eta_one": True}, {"bounded": gen.make_bounded(gen.BOUNDED_MIXED)}):
        heads = None if kw.get("eta_one") else wl.heads
        plain = o.eval_kernels(wl.desc, wl.specs, heads, **kw)
        mixed = o.eval_kernels(wl.desc, wl.specs, heads, grid=gr, keep_features=not kw, **kw)
        r = mixed["routed"]
        assert r.any() and (~r).any() and not r[:, fam == gen.GEMM].any()
        np.testing.assert_array_equal(mixed["eta"][~r], plain["eta"][~r])
        np.testing.assert_array_equal(mixed["t_roof"], plain["t_roof"])
        t0 = wl.specs["t0"][:, None]
        np.testing.assert_array_equal(mixed["t"], np.maximum(mixed["t_roof"] * mixed["eta"], t0))
        if not kw:
            for s in range(wl.n_specs):
                for f in np.unique(fam[r[s]]):
                    sel = r[s] & (fam == f)
                    e, rr = o.grid_eta(mixed["x"][s][sel][:, :16], gr, f)
                    assert rr.all()
                    np.testing.assert_array_equal(mixed["eta"][s, sel], e)
        res.append(mixed)
    for m in res[1:]:
        np.testing.assert_array_equal(m["routed"], res[0]["routed"])
        np.testing.assert_array_equal(m["eta"][m["routed"]], res[0]["eta"][m["routed"]])
    empty = gen.Grid(gr.mask, gr.axes, gr.lo, gr.hi, gr.n, np.full_like(gr.values, np.nan))
    a = o.eval_kernels(wl.desc, wl.specs, wl.heads, grid=empty)
    b = o.eval_kernels(wl.desc, wl.specs, wl.heads)
    assert not a["routed"].any()
    np.testing.assert_array_equal(a["eta"], b["eta"])
