"""Pins of the batch -> kernel expansion oracle (oracle/ks_expand.py).

Pinned by: hand-derived record lists of tiny models (tests/golden/,
each with its citation); the per-step kernel counts the workloads state
(9 kernels per layer plus embedding and LM head); an independent
implementation of the same record layout (the record builder that hands the
workloads to the library); the homogeneous form's defining property (the
same step bodies as one record per dispatch, Sec. 5.7); and degenerate
batches."""
import os
from types import SimpleNamespace

import numpy as np
import pytest

from oracle import ks_expand as ox
from oracle import ks_oracle as o
from workload import gen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FAM = {name: i for i, name in enumerate(gen.FAMILIES)}


def load_fixture(name):
    model, steps, recs, n_launch, homog = None, [], [], None, 0
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            head, *rest = line.split()
            if head == "model":
                kv = dict(x.split("=") for x in rest)
                model = SimpleNamespace(**{k: int(v) for k, v in kv.items()})
            elif head == "step":
                reqs = [tuple(int(v) for v in x.split(":")) for x in rest[0].split(",")]
                steps.append((reqs, int(rest[1].split("=")[1])))
            elif head == "homogeneous":
                homog = int(rest[0])
            elif head == "n_launch":
                n_launch = [int(v) for v in rest]
            else:
                recs.append((FAM[head],) + tuple(int(v) for v in rest))
    req_off = np.cumsum([0] + [len(r) for r, _ in steps])
    req_q = [q for r, _ in steps for q, _ in r]
    req_h = [h for r, _ in steps for _, h in r]
    prefill = [p for _, p in steps]
    return model, req_off, req_q, req_h, prefill, bool(homog), recs, n_launch


def as_rows(e):
    fam = np.repeat(np.arange(gen.NFAM), np.diff(e["fam_off"]))
    return [(int(fam[i]),) + tuple(int(e[f][i]) for f in ox.FIELDS) for i in range(len(fam))]


@pytest.mark.parametrize("name", ["expand_tiny_dense.txt", "expand_tiny_moe_homogeneous.txt"])
def test_hand_derived_records(name):
    model, req_off, req_q, _, prefill, homog, recs, n_launch = load_fixture(name)
    e = ox.expand(model, req_off, req_q, prefill, homogeneous=homog)
    assert as_rows(e) == recs
    assert list(e["n_launch"]) == n_launch
    assert list(e["layers"]) == [model.layers] * len(prefill)
    assert list(e["hidden"]) == [model.hidden] * len(prefill)
    assert list(e["tp"]) == [model.tp] * len(prefill)


def test_llama7b_workload_count():
    # 1000 steps of 32 layers x 9 kernels plus the embedding and LM head
    tr = gen.trace_c1()
    e = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill)
    assert e["fam_off"][-1] == 1000 * (32 * 9 + 2) == 290_000
    assert (e["mult"] == 1).all()
    # attention records split by the step's prefill flag, one per layer
    n_pre = int(tr.prefill.sum())
    assert np.diff(e["fam_off"])[gen.ATTN_PREFILL] == 32 * n_pre
    assert np.diff(e["fam_off"])[gen.ATTN_DECODE] == 32 * (1000 - n_pre)


def test_moe_per_step_count():
    # the mixture replaces the 3 MLP kernels by router, 2 grouped GEMMs and
    # SiLU x mul: 10 kernels per layer
    w = gen.config3(0, 30)
    tr = gen.trace_c3().slice(0, 30)
    e = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill)
    assert e["fam_off"][-1] == 30 * (32 * 10 + 2)
    assert np.diff(e["fam_off"])[gen.GROUPED_GEMM] == 30 * 32 * 2
    assert w.desc.n_rows == e["fam_off"][-1]


@pytest.mark.parametrize("homog", [False, True])
def test_closed_form_family_counts(homog):
    for shape in (gen.LLAMA7B, gen.MIXTRAL, gen.DENSE_SHAPES[5],
                  gen.ModelShape("kvw", 1024, 3, 8, 2, 64, 4096, kv_write=True)):
        prefill = [1, 0, 0, 1, 0]
        req_off = [0, 2, 3, 5, 6, 8]
        req_q = [7, 1, 1, 1, 1, 40, 1, 1]
        e = ox.expand(shape, req_off, req_q, prefill, homogeneous=homog)
        c = ox.family_counts(shape, 5, 2, homog)
        np.testing.assert_array_equal(np.diff(e["fam_off"]), c)
        # every dispatched kernel is accounted for exactly once
        per_step = shape.layers * (9 + (1 if shape.experts else 0) + (1 if shape.kv_write else 0)) + 2
        assert int(e["mult"].sum()) == 5 * per_step


def _trace_cases():
    cases = [("c1", gen.trace_c1().slice(0, 120))]
    for i in range(6):
        cases.append((f"c2-{i}", gen.trace_c2(i).slice(0, 12)))
    tr3 = gen.trace_c3().slice(0, 25)
    tr3.experts = gen.route_tokens(gen.trace_c3(), gen.SEED + 3, 0, 25)
    cases.append(("c3", tr3))
    cases.append(("c5", gen.trace_c5().slice(0, 15)))
    kvw = gen.ModelShape("kvw", 2048, 5, 16, 4, 128, 5632, tp=2, kv_write=True)
    cases.append(("kvw", gen.trace_uniform(kvw, 40, 7, bmax=8)))
    # fewer KV heads than GPUs: each GPU keeps a replica of one KV head
    rep = gen.ModelShape("kvrep", 2048, 3, 16, 2, 128, 5632, tp=4, kv_write=True)
    cases.append(("kvrep", gen.trace_uniform(rep, 30, 8, bmax=8)))
    return cases


@pytest.mark.parametrize("name,tr", _trace_cases(), ids=[c[0] for c in _trace_cases()])
def test_matches_record_builder(name, tr):
    """The generator's record builder lays the same workloads out with numpy
    tables; the oracle enumerates kernels step by step.  Both must agree
    bit for bit."""
    desc, rec = gen.build([tr])
    e = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill)
    np.testing.assert_array_equal(desc.fam_off, e["fam_off"])
    for f in ("step", "m", "n", "k", "a", "b"):
        np.testing.assert_array_equal(getattr(desc, f).astype(np.int64), e[f], err_msg=f)
    for f in ("layers", "hidden", "tp", "n_launch"):
        np.testing.assert_array_equal(getattr(rec, f).astype(np.int64), e[f], err_msg=f)


def _desc_from(e, tr):
    u = lambda x: np.asarray(x, np.uint32)
    experts = u(tr.experts.reshape(-1)) if tr.experts is not None else u([])
    return gen.Desc(e["fam_off"], u(e["step"]), u(e["m"]), u(e["n"]), u(e["k"]), u(e["a"]),
                    u(e["b"]), u(tr.req_off), u(tr.req_q), u(tr.req_h), experts, 2, u(e["mult"]))


@pytest.mark.parametrize("case", ["c1", "c3", "kvw"])
def test_homogeneous_same_step_bodies(case):
    """Sec. 5.7: t_gpu = L t_layer + t_lm_head + t_embed.  One record of
    multiplicity L per layer-identical kernel gives the same step terms as
    one record per dispatched kernel."""
    tr = dict(_trace_cases())[case]
    full = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill)
    hom = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill, homogeneous=True)
    assert hom["fam_off"][-1] < full["fam_off"][-1]
    specs = gen.specs_datasheet()
    host = gen.HostConsts()
    rec = gen.StepRec(*(np.asarray(full[f], np.uint32) for f in ("layers", "hidden", "tp", "n_launch")))
    for heads, eta_one in ((None, True), (gen.make_heads(16, 64, "f32"), False)):
        rf = o.eval_steps(_desc_from(full, tr), rec, specs, host, heads, eta_one)
        rh = o.eval_steps(_desc_from(hom, tr), rec, specs, host, heads, eta_one)
        for key in ("t_body", "t_gpu", "t_step"):
            np.testing.assert_allclose(rh[key], rf[key], rtol=1e-12, err_msg=key)


def test_homogeneous_body_is_explicit_weighted_sum():
    """Brute force: the oracle's body of a multiplicity record set equals an
    explicit loop adding each record's latency mult times."""
    tr = dict(_trace_cases())["c3"]
    hom = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill, homogeneous=True)
    d = _desc_from(hom, tr)
    k = o.eval_kernels(d, gen.specs_datasheet(), eta_one=True)
    rec = gen.StepRec(*(np.asarray(hom[f], np.uint32) for f in ("layers", "hidden", "tp", "n_launch")))
    body = o.eval_steps(d, rec, gen.specs_datasheet(), gen.HostConsts(), eta_one=True, kern=k)["t_body"]
    for s in range(2):
        ref = [0.0] * d.n_steps
        for i in range(d.n_rows):
            for _ in range(int(d.mult[i])):
                ref[int(d.step[i])] += float(k["t"][s, i])
        np.testing.assert_allclose(body[s], ref, rtol=1e-13)


def test_degenerate_batches():
    m = gen.LLAMA7B
    e = ox.expand(m, [0], [], [])
    assert e["fam_off"][-1] == 0 and len(e["n_launch"]) == 0
    # a step without requests still dispatches its kernels, over 0 tokens
    e = ox.expand(m, [0, 0], [], [0])
    assert e["fam_off"][-1] == 32 * 9 + 2
    assert (e["m"] == 0).all()
    # a one-layer model: the homogeneous form equals the plain one
    one = gen.ModelShape("one", 256, 1, 4, 4, 64, 512)
    a = ox.expand(one, [0, 1, 3], [9, 1, 1], [1, 0])
    b = ox.expand(one, [0, 1, 3], [9, 1, 1], [1, 0], homogeneous=True)
    for f in ("fam_off",) + ox.FIELDS:
        np.testing.assert_array_equal(a[f], b[f])
