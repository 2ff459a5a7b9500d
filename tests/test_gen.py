"""Seeded workload generators: determinism, sizes and layout."""
import numpy as np
import pytest

from workload import gen


def test_c1_size_and_layout():
    w = gen.config1()
    d = w.desc
    assert d.n_rows == 1000 * (32 * 9 + 2) == 290_000
    assert d.n_steps == 1000
    fam = d.family()
    for f in range(gen.NFAM):
        s = d.step[d.fam_off[f]:d.fam_off[f + 1]]
        assert (np.diff(s.astype(np.int64)) >= 0).all(), gen.FAMILIES[f]
    # every step has exactly one LM head and one embedding record
    assert np.array_equal(np.bincount(d.step[fam == gen.LM_HEAD], minlength=1000), np.ones(1000))
    assert d.n_rows - d.fam_off[gen.KV_WRITE + 1] + d.fam_off[gen.KV_WRITE] == d.n_rows
    assert w.n_specs == 2 and w.heads.precision == "f32" and w.heads.hidden == 64


def test_deterministic():
    a, b = gen.config1(0, 50), gen.config1(0, 50)
    for name in ("step", "m", "n", "k", "a", "b", "req_q", "req_h", "req_off"):
        np.testing.assert_array_equal(getattr(a.desc, name), getattr(b.desc, name))
    np.testing.assert_array_equal(a.heads.w2, b.heads.w2)


def test_slice_is_prefix_of_full_trace():
    full = gen.config1()
    part = gen.config1(0, 40)
    n = part.desc.n_steps
    r = int(part.desc.req_off[-1])
    np.testing.assert_array_equal(part.desc.req_q, full.desc.req_q[:r])
    np.testing.assert_array_equal(part.desc.req_h, full.desc.req_h[:r])
    assert n == 40


def test_c4_grid_size():
    w = gen.config4()
    assert w.desc.n_steps == 1345
    assert w.desc.n_rows == 1345 * 290 == 390_050
    assert w.n_specs * w.desc.n_rows > 0.99e8
    assert w.heads.precision == "bf16" and w.heads.hidden == 128


def test_moe_routing_sums_to_top2_tokens():
    w = gen.config3(0, 40)
    d = w.desc
    ex = d.expert_rows.reshape(40, 32, 8).astype(np.int64)
    tokens = np.add.reduceat(d.req_q.astype(np.int64), d.req_off[:-1].astype(np.int64))
    np.testing.assert_array_equal(ex.sum(-1), 2 * tokens[:, None].repeat(32, 1))
    assert d.n_rows == 40 * (32 * 10 + 2)
    g = d.fam_off[gen.GROUPED_GEMM], d.fam_off[gen.GROUPED_GEMM + 1]
    assert (d.a[g[0]:g[1]] == 8).all()
    assert (d.b[g[0]:g[1]].astype(np.int64) + 8 <= len(d.expert_rows)).all()
    # a later step range draws the same routing as the full trace would
    w2 = gen.config3(1020, 1030)
    w3 = gen.config3(1000, 1030)
    np.testing.assert_array_equal(w2.desc.expert_rows, w3.desc.expert_rows[20 * 256:])


def test_c5_prefix_hits_shorten_chunks():
    w = gen.config5(0, 300)
    d = w.desc
    q = d.req_q.astype(np.int64)
    assert q.max() <= 2048 and q.min() >= 1
    assert d.req_h.max() <= 131072 + 2048 and d.req_h.min() >= 512
    assert w.heads.in_dim == 32 and w.heads.hidden == 256


@pytest.mark.parametrize("i", range(6))
def test_c2_shapes(i):
    w = gen.config2(i, 0, 20)
    s = gen.DENSE_SHAPES[i]
    assert w.desc.n_rows == 20 * (9 * s.layers + 2)
    assert (w.steps.tp == s.tp).all()


def test_head_parameters_rounded_once():
    h = gen.make_heads(16, 128, "bf16")
    bits = h.storage["w2"]
    assert bits.dtype == np.uint16
    back = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    np.testing.assert_array_equal(back, h.w2)
    hf = gen.make_heads(16, 64, "f32")
    np.testing.assert_array_equal(hf.storage["w1"].astype(np.float64), hf.w1)
