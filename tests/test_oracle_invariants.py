"""Property checks of the oracle: invariants the paper states or that follow
from the definitions."""
import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import ks_oracle as o
from workload import gen
from tests.helpers import make_desc, spec

reqs_st = st.lists(st.tuples(st.integers(1, 3000), st.integers(0, 200000)), min_size=1, max_size=12)


def _attn_eval(reqs, sp):
    d = make_desc([(gen.ATTN_PREFILL, 0, 0, 32, 128, 8, 0)], [reqs])
    k = o.eval_kernels(d, sp, eta_one=True)
    c = k["counts"]
    return int(c["F"][0]), int(c["Bt"][0]), k["t_roof"][0, 0]


@settings(max_examples=150, deadline=None)
@given(reqs_st, st.integers(0, 11), st.integers(1, 500), st.booleans())
def test_attention_monotone_in_kv_and_chunk(reqs, which, extra, grow_q):
    """F and Bt do not decrease when a request's history or chunk grows, and
    neither does t_roof when the history grows (the grid is unchanged).  A
    longer chunk can add query blocks and so lower the wave-quantization
    factor u: t_roof need not grow with the chunk (e.g. q 126 -> 129 doubles
    the blocks).  Counts and roofline only: the paper calls the attention
    efficiency surface itself non-monotone."""
    sp = spec(P=2.25e15, BW=8e12, n_cu=148)
    base = _attn_eval(reqs, sp)
    i = which % len(reqs)
    q, h = reqs[i]
    more = list(reqs)
    more[i] = (q + extra, h) if grow_q else (q, h + extra)
    bigger = _attn_eval(more, sp)
    assert bigger[0] >= base[0] and bigger[1] >= base[1]
    if not grow_q:
        assert bigger[2] >= base[2]


@settings(max_examples=100, deadline=None)
@given(reqs_st, st.randoms(use_true_random=False))
def test_attention_request_order_irrelevant(reqs, rnd):
    a = o.attention_work(*_req_arrays(reqs))
    shuffled = list(reqs)
    rnd.shuffle(shuffled)
    b = o.attention_work(*_req_arrays(shuffled))
    for key in a:
        assert int(a[key][0]) == int(b[key][0])


def _req_arrays(reqs):
    return (np.array([0, len(reqs)]), np.array([q for q, _ in reqs]), np.array([h for _, h in reqs]))


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2 ** 20), st.integers(1, 400))
def test_waves_bounds(B, N):
    W, u = o.waves(np.array([B], np.uint64), N)
    assert u[0] >= 1.0
    if B:
        assert (int(W[0]) - 1) * N < B <= int(W[0]) * N


def test_latency_bounds_on_c1_sample():
    w = gen.config1(0, 30)
    k = o.eval_kernels(w.desc, w.specs, w.heads)
    assert (k["eta"] >= 1.0).all()
    assert (k["u"] >= 1.0).all()
    for s in range(2):
        assert (k["t"][s] >= w.specs["t0"][s]).all()
        assert (k["t"][s] >= k["t_roof"][s] * k["eta"][s] * (1 - 1e-15)).all()


def test_step_body_invariant_to_row_order_within_family():
    w = gen.config1(0, 20)
    k = o.eval_kernels(w.desc, w.specs, w.heads)
    body = o.step_body(k["t"][0], w.desc.step, w.desc.n_steps)
    perm = np.random.default_rng(5).permutation(w.desc.n_rows)
    body2 = o.step_body(k["t"][0][perm], w.desc.step[perm], w.desc.n_steps)
    np.testing.assert_allclose(body, body2, rtol=1e-13)


def test_bf16_emulation_gap_is_small():
    """The emulated-bf16 head stays close to the exact float64 head: the gap
    bounds the effect of the rounding points on eta."""
    w = gen.config4(n_specs=2, grid_steps=5, c1_steps=5)
    a = o.eval_kernels(w.desc, w.specs, w.heads, emulate_bf16=True)
    b = o.eval_kernels(w.desc, w.specs, w.heads, emulate_bf16=False)
    rel = np.abs(a["eta"] / b["eta"] - 1)
    assert rel.max() < 1e-2
