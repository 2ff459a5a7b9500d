"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Tolerances (design notes, "Oracle and parity"): counts bit-exact; t_roof and
fp32-head outputs 1e-5 relative; bf16-head eta 1e-2 relative and z within
ZTOL absolute; given the GPU's eta, t = max(t_roof eta, t0) to 1e-5; step
outputs 1e-5 (fp32 heads, eta = 1) and 1e-2 (bf16 heads)."""
import numpy as np
import pytest
import torch  # noqa: F401  (runtime loads at collection, not inside a timed test)

from oracle import ks_oracle as o
from workload import gen
from tests import gpu_helpers as g
from tests.helpers import make_desc, spec, steprec, sub_desc
from paper_2606_28565_amd import abi

pytestmark = pytest.mark.gpu

REL = 1e-5
REL_BF16 = 1e-2
# |z_gpu - z_oracle| for std-0.1 bf16 heads: a flipped bf16 rounding of one
# hidden activation moves z by about |w3| 2^-8 |h2| ~ 0.1 * 2e-4; even all
# 256 activations of both layers flipping the same way stay below 5e-3.
ZTOL = 5e-3


def _z_from_eta(eta):
    return -np.log(np.asarray(eta, np.float64) - 1.0)


def z_error_bound(wl, ref):
    """First-order bound on |z_gpu - z_oracle| from the arithmetic, per pair.
    With magnitudes m1 = |W1||x|, m2 = |W2| m1' + |b2|, where ' marks the
    relu-active inputs of the next layer, the terms of z sum to
    s3 = |w3||h2| + |b3|, s2 = |w3||W2||h1| and s1 = |w3||W2||W1||x|.
    fp32: each length-n dot product errs by at most n 2^-24 times its
    absolute term sum (Higham's gamma_n), so |dz| <= 2^-24 (128 s3 + K2 s2 +
    K1 s1) plus the feature error (a few ulps of each x).  bf16: the two
    sides may round an activation to neighbouring bf16 values (one ulp,
    2^-7 relative), so |dz| <= 2^-7 (s3 + s2 + s1)."""
    fam = wl.desc.family()[ref["rows"]]
    x = ref["x"]                                    # [spec, row, in]
    h = wl.heads
    bound = np.zeros(x.shape[:2])
    for f in np.unique(fam):
        sel = fam == f
        xf = np.abs(x[:, sel, :])
        a1 = xf @ np.abs(h.w1[f]).T                 # |W1||x|
        h1 = np.maximum(x[:, sel, :] @ h.w1[f].T, 0.0)
        act1 = h1 > 0
        a2 = (a1 * act1) @ np.abs(h.w2[f]).T        # |W2||W1||x| over active units
        h2 = np.maximum(h1 @ h.w2[f].T + h.b2[f], 0.0)
        act2 = h2 > 0
        w3 = np.abs(h.w3[f])
        s3 = np.abs(h2) @ w3 + abs(h.b3[f])
        s2 = ((np.abs(h1) @ np.abs(h.w2[f]).T + np.abs(h.b2[f])) * act2) @ w3
        s1 = (a2 * act2) @ w3
        if h.precision == "bf16":
            bound[:, sel] = 2.0 ** -7 * (s3 + s2 + s1)
        else:
            k1, k2 = h.in_dim, h.hidden
            bound[:, sel] = 2.0 ** -24 * (h.hidden * s3 + k2 * s2 + (k1 + 16) * s1)
    return bound


def _check_kernels(wl, gpu, ref, bf16, eta_one=False, ztol=ZTOL):
    c = ref["counts"]
    if "flops" in gpu:
        np.testing.assert_array_equal(gpu["flops"], c["F"])
        np.testing.assert_array_equal(gpu["bytes"], c["Bt"])
        np.testing.assert_array_equal(gpu["blocks"], c["B"])
    assert g.rel_err(gpu["t_roof"], ref["t_roof"]).max() <= REL
    if eta_one:
        assert (gpu["eta"] == 1.0).all()
        assert g.rel_err(gpu["t_kernel"], ref["t"]).max() <= REL
        return
    t0 = wl.specs["t0"][: gpu["eta"].shape[0], None]
    cond = np.maximum(ref["t_roof"] * gpu["eta"].astype(np.float64), t0)
    assert g.rel_err(gpu["t_kernel"], cond).max() <= REL
    if bf16:
        assert g.rel_err(gpu["eta"], ref["eta"]).max() <= REL_BF16
        dz = np.abs(_z_from_eta(gpu["eta"]) - ref["z"])
        assert dz.max() <= ztol, dz.max()
        assert g.rel_err(gpu["t_kernel"], ref["t"]).max() <= REL_BF16
    else:
        assert g.rel_err(gpu["eta"], ref["eta"]).max() <= REL
        assert g.rel_err(gpu["t_kernel"], ref["t"]).max() <= REL


def _check_steps(wl, gpu, ref_steps, bf16, n_specs):
    tol = REL_BF16 if bf16 else REL
    for key in ("t_body", "t_gpu", "t_step"):
        e = g.rel_err(gpu[key], ref_steps[key][:n_specs])
        assert e.max() <= tol, (key, e.max())


def _steps_given_eta(wl, gpu, ref_k, n_specs):
    """Oracle step terms with the GPU's eta substituted: isolates the
    aggregation and assembly from the head."""
    t0 = wl.specs["t0"][:n_specs, None]
    t = np.maximum(ref_k["t_roof"][:n_specs] * gpu["eta"].astype(np.float64), t0)
    kern = dict(ref_k)
    kern["t"] = t
    return o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, spec_ids=range(n_specs), kern=kern)


# ------------------------------------------------------------------- c1 ----
@pytest.fixture(scope="module")
def c1():
    wl = gen.config1()
    return wl, o.eval_kernels(wl.desc, wl.specs, wl.heads)


def test_c1_kernels_fp32_head(c1):
    wl, ref = c1
    gpu = g.eval_kernels(wl)
    _check_kernels(wl, gpu, ref, bf16=False)


def test_c1_steps_fp32_head(c1):
    wl, ref = c1
    gpu = g.eval_steps(wl)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, wl.heads, kern=ref)
    _check_steps(wl, gpu, rs, bf16=False, n_specs=2)
    _check_kernels(wl, gpu, ref, bf16=False)


def test_c1_eta_one():
    wl = gen.config1()
    ref = o.eval_kernels(wl.desc, wl.specs, eta_one=True)
    gpu = g.eval_steps(wl, eta_one=True)
    _check_kernels(wl, gpu, ref, bf16=False, eta_one=True)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, eta_one=True, kern=ref)
    _check_steps(wl, gpu, rs, bf16=False, n_specs=2)


def test_c1_deterministic():
    wl = gen.config1(0, 200)
    a = g.eval_steps(wl)
    b = g.eval_steps(wl)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])


# ------------------------------------------------------------ bf16 heads ----
def _bf16_case(wl, n_specs=None, counts=True):
    """counts=False: no per-record counts written, so the kernel forms F, Bt
    and the row-count feature in fp32 (the path of calls without count
    outputs, e.g. the benchmark's)."""
    n_specs = n_specs or wl.n_specs
    ref = o.eval_kernels(wl.desc, wl.specs, wl.heads, spec_ids=range(n_specs))
    gpu = g.eval_steps(wl, n_specs=n_specs, counts=counts)
    _check_kernels(wl, gpu, ref, bf16=True)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, wl.heads, spec_ids=range(n_specs), kern=ref)
    _check_steps(wl, gpu, rs, bf16=True, n_specs=n_specs)
    ge = _steps_given_eta(wl, gpu, ref, n_specs)
    _check_steps(wl, gpu, ge, bf16=False, n_specs=n_specs)
    return gpu, ref


def test_c4_subset_bf16_16_128():
    _bf16_case(gen.config4(n_specs=24, grid_steps=25, c1_steps=40))


@pytest.mark.parametrize("n_specs", [1, 2, 3, 7])
def test_spec_loop_counts_for_the_16_128_head(n_specs):
    """The 16-128 head evaluates its spec loop software-pipelined (each
    spec's epilogue and tail ride in the next spec's groups, its features in
    the previous one's): any number of spec vectors against the oracle, and
    every spec's outputs bit-identical to those of a call with only the
    spec vectors up to it (a spec's results do not depend on its neighbours
    in the loop)."""
    wl = gen.config4(n_specs=8, grid_steps=12, c1_steps=20)
    gpu, ref = _bf16_case(wl, n_specs=n_specs)
    if n_specs > 1:
        fewer = g.eval_steps(wl, n_specs=n_specs - 1)
        for k in ("t_roof", "eta", "t_kernel", "t_body", "t_step"):
            np.testing.assert_array_equal(gpu[k][:n_specs - 1], fewer[k], err_msg=k)


@pytest.mark.parametrize("counts", [True, False])
def test_c3_moe_subset(counts):
    _bf16_case(gen.config3(0, 30), counts=counts)


@pytest.mark.parametrize("counts", [True, False])
def test_c5_subset_bf16_32_256(counts):
    _bf16_case(gen.config5(0, 24), counts=counts)


@pytest.mark.parametrize("shape_idx", range(6))
@pytest.mark.parametrize("counts", [True, False])
def test_c2_shape_subsets_with_tp(shape_idx, counts):
    _bf16_case(gen.config2(shape_idx, 0, 12), counts=counts)


def test_c4_full_size_sampled():
    """The 256-spec capacity grid at full size, in the launch configuration
    the benchmark times; sampled (spec, step) outputs against the oracle run
    on just those steps' records."""
    wl = gen.config4()
    gpu = g.eval_steps(wl)
    rng = np.random.default_rng(11)
    steps = np.unique(np.concatenate([[0, 999, 1000, wl.desc.n_steps - 1],
                                      rng.integers(0, wl.desc.n_steps, 4)]))
    specs = np.unique(np.concatenate([[0, wl.n_specs - 1], rng.integers(0, wl.n_specs, 4)]))
    rows = np.nonzero(np.isin(wl.desc.step, steps))[0]
    ref = o.eval_kernels(wl.desc, wl.specs, wl.heads, spec_ids=specs, rows=rows)
    ge = np.maximum(ref["t_roof"] * gpu["eta"][specs][:, rows], wl.specs["t0"][specs, None])
    assert g.rel_err(gpu["t_kernel"][specs][:, rows], ge).max() <= REL
    assert g.rel_err(gpu["eta"][specs][:, rows], ref["eta"]).max() <= REL_BF16
    c = ref["counts"]
    np.testing.assert_array_equal(gpu["flops"][rows], c["F"][rows])
    for si, s in enumerate(specs):
        body = np.bincount(wl.desc.step[rows], weights=ref["t"][si], minlength=wl.desc.n_steps)[steps]
        body_ge = np.bincount(wl.desc.step[rows], weights=ge[si], minlength=wl.desc.n_steps)[steps]
        assert g.rel_err(gpu["t_body"][s, steps], body).max() <= REL_BF16
        assert g.rel_err(gpu["t_body"][s, steps], body_ge).max() <= REL


# --------------------------------------------------------------- all kinds --
KINDS = [("f32", 16, 64), ("f32", 16, 128), ("f32", 32, 64), ("f32", 32, 128),
         ("bf16", 16, 64), ("bf16", 16, 128), ("bf16", 16, 256),
         ("bf16", 32, 64), ("bf16", 32, 128), ("bf16", 32, 256)]


@pytest.mark.parametrize("precision,in_dim,hidden", KINDS)
@pytest.mark.parametrize("counts", [True, False])
def test_every_head_kind(precision, in_dim, hidden, counts):
    """counts=False: the fp32 count path (no per-record count output)."""
    wl = gen.config1(0, 6).with_heads(gen.make_heads(in_dim, hidden, precision))
    ref = o.eval_kernels(wl.desc, wl.specs, wl.heads)
    gpu = g.eval_kernels(wl, counts=counts)
    _check_kernels(wl, gpu, ref, bf16=precision == "bf16")
    assert ("flops" in gpu) == counts


@pytest.mark.parametrize("precision,in_dim,hidden", KINDS)
def test_every_head_kind_stress(precision, in_dim, hidden):
    """Heads with std-0.25 weights: eta spans 1 .. 1e5 and many relu units
    switch.  Larger weights make the layer sums cancel more, so z is checked
    against the arithmetic's own error bound (plus the resolution of z that
    an fp32 eta near 1 keeps: -log(eta - 1) moves by ~2^-23 eta/(eta - 1)
    per ulp, and the exponential adds a few more ulps), and eta against the
    bf16 bar."""
    wl = gen.config1(0, 6).with_heads(gen.make_heads(in_dim, hidden, precision, std=0.25))
    ref = o.eval_kernels(wl.desc, wl.specs, wl.heads, keep_features=True)
    gpu = g.eval_kernels(wl)
    np.testing.assert_array_equal(gpu["flops"], ref["counts"]["F"])
    t0 = wl.specs["t0"][:, None]
    cond = np.maximum(ref["t_roof"] * gpu["eta"].astype(np.float64), t0)
    assert g.rel_err(gpu["t_kernel"], cond).max() <= REL
    eta = gpu["eta"].astype(np.float64)
    resolved = eta > 1.0
    dz = np.abs(_z_from_eta(eta[resolved]) - ref["z"][resolved])
    bound = z_error_bound(wl, ref)[resolved] + 2.0 ** -20 * eta[resolved] / (eta[resolved] - 1.0)
    assert (dz <= bound).all(), (dz.max(), (dz / bound).max())
    assert (ref["z"][~resolved] > 15).all()      # eta rounds to 1 only when e^-z < 2^-24
    assert g.rel_err(gpu["eta"], ref["eta"]).max() <= REL_BF16


@pytest.mark.parametrize("in_dim,hidden", [(16, 128), (32, 256), (16, 64)])
def test_bf16_weights_at_unaligned_addresses(in_dim, hidden):
    """The bf16 heads stage W2 into LDS by 16-byte row chunks when its
    address allows, else element by element: W1 and W2 passed two bytes past
    a 16-byte boundary give outputs bit-identical to the aligned call."""
    import torch
    wl = gen.config1(0, 4).with_heads(gen.make_heads(in_dim, hidden, "bf16"))
    di = abi.DeviceInputs(wl)

    def run(heads):
        so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
        ko_t, ko = abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=False)
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                          di.ws_ptr, di.ws_bytes, abi.current_stream())
        torch.cuda.synchronize()
        abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
        return {k: v.cpu().numpy() for k, v in list(so_t.items()) + list(ko_t.items())}

    aligned = run(di.make_heads("bf16", in_dim, hidden, abi.KS_ETA_MLP))
    heads = di.make_heads("bf16", in_dim, hidden, abi.KS_ETA_MLP)
    keep = []
    for name in ("w1", "w2"):
        t = di.heads_t[name]
        buf = torch.zeros(t.numel() + 16, dtype=t.dtype, device=t.device)
        base = (-buf.data_ptr() % 16) // t.element_size() + 1   # one element past a 16-byte boundary
        buf[base:base + t.numel()] = t
        keep.append(buf)
        ptr = buf.data_ptr() + base * t.element_size()
        assert ptr % 16 == 2
        setattr(heads, name, ptr)
    unaligned = run(heads)
    for k in aligned:
        np.testing.assert_array_equal(unaligned[k], aligned[k], err_msg=k)


# ------------------------------------------------------------- edge cases --
def _wl(desc, n_steps, heads=None, tp=1, layers=1, specs=None):
    return gen.Workload("edge", desc, steprec(n_steps, layers=layers, hidden=64, tp=tp, n_launch=1),
                        specs or spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6),
                        heads or gen.make_heads(16, 64, "f32"), gen.HostConsts())


def _edge_check(wl):
    ref = o.eval_kernels(wl.desc, wl.specs, wl.heads)
    gpu = g.eval_steps(wl)
    _check_kernels(wl, gpu, ref, bf16=wl.heads.precision == "bf16")
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, wl.heads, kern=ref)
    _check_steps(wl, gpu, rs, bf16=wl.heads.precision == "bf16", n_specs=wl.n_specs)


def test_single_record():
    _edge_check(_wl(make_desc([(gen.GEMM, 0, 77, 300, 129, 0, 0)], [[(1, 5)]]), 1))


def test_zero_work_and_empty_request_step():
    rows = [(gen.EMBED, 0, 0, 64, 0, 0, 0), (gen.ATTN_DECODE, 1, 0, 8, 128, 2, 0),
            (gen.ATTN_DECODE, 0, 0, 8, 128, 2, 0), (gen.SILU_MUL, 1, 0, 10, 0, 0, 0)]
    _edge_check(_wl(make_desc(rows, [[], [(3, 7)]]), 2))


def test_ragged_segments_crossing_tiles():
    """One family whose step segments straddle 64-record tiles in every way:
    lengths 1, 63, 64, 65, 130, 200 and single records between them."""
    rows, reqs = [], []
    lens = [1, 63, 64, 65, 1, 130, 1, 200, 2, 64]
    for j, L in enumerate(lens):
        reqs.append([(1 + j, 100 * j)])
        rows += [(gen.GEMM, j, 3 + i, 128 + i, 64, 0, 0) for i in range(L)]
        rows.append((gen.RMSNORM, j, 5 + j, 4096, 0, 0, 0))
    _edge_check(_wl(make_desc(rows, reqs), len(lens)))


def test_steps_missing_from_families_and_tp_comm():
    rows = [(gen.GEMM, 0, 4, 4096, 4096, 0, 0), (gen.GEMM, 2, 9, 4096, 4096, 0, 0),
            (gen.ATTN_PREFILL, 1, 0, 8, 128, 1, 0), (gen.LM_HEAD, 3, 2, 8000, 4096, 0, 0)]
    reqs = [[(4, 0)], [(300, 5), (1, 9)], [(9, 1)], [(1, 1), (1, 2)]]
    _edge_check(_wl(make_desc(rows, reqs), 4, tp=4, layers=3))


def test_grouped_gemm_with_empty_experts():
    rows = [(gen.GROUPED_GEMM, 0, 0, 256, 512, 4, 0), (gen.GROUPED_GEMM, 0, 0, 512, 256, 4, 4),
            (gen.GROUPED_GEMM, 1, 0, 256, 512, 3, 8)]
    experts = [0, 5, 0, 300, 0, 0, 0, 0, 129, 1, 0]
    _edge_check(_wl(make_desc(rows, [[(3, 1)], [(5, 2)]], expert_rows=experts), 2,
                    heads=gen.make_heads(16, 128, "bf16")))


def test_many_specs_single_step():
    rng = np.random.default_rng(4)
    n = 37
    sp = gen.specs_grid(n, 99)
    rows = [(gen.GEMM, 0, int(m), 4096, 4096, 0, 0) for m in rng.integers(1, 5000, 70)]
    _edge_check(_wl(make_desc(rows, [[(5, 9)]]), 1, specs=sp, heads=gen.make_heads(16, 128, "bf16")))


# ---------------------------------------------- eta = 1 stream, wave count ----
def _eta1_case(wl, counts):
    ref = o.eval_kernels(wl.desc, wl.specs, eta_one=True)
    gpu = g.eval_steps(wl, eta_one=True, counts=counts)
    assert ("flops" in gpu) == counts
    _check_kernels(wl, gpu, ref, bf16=False, eta_one=True)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, eta_one=True, kern=ref)
    _check_steps(wl, gpu, rs, bf16=False, n_specs=wl.n_specs)
    steps_only = g.eval_steps(wl, eta_one=True, per_pair=False)
    _check_steps(wl, steps_only, rs, bf16=False, n_specs=wl.n_specs)


def test_eta_one_without_count_outputs():
    """Without per-record count outputs the eta = 1 stream forms F and Bt in
    fp32; t_roof, t and the step sums keep the 1e-5 bar."""
    _eta1_case(gen.config1(0, 120), counts=False)
    _eta1_case(gen.config3(0, 40), counts=False)


def _run_workload(seed, n_steps, max_run, n_specs):
    """Per family, each step's records in one run of U{1..max_run} records
    (some families skip steps), so that runs start and end at every one of
    a lane's four records, at 16-lane row (64-record tile) edges and at
    256-record workgroup-tile edges; family sizes are not multiples of 4."""
    rng = np.random.default_rng(seed)
    rows, reqs = [], []
    for j in range(n_steps):
        reqs.append([(int(rng.integers(1, 40)), int(rng.integers(0, 5000)))
                     for _ in range(int(rng.integers(1, 4)))])
    shape = {gen.GEMM: lambda: (int(rng.integers(1, 3000)), int(rng.integers(64, 9000)), int(rng.integers(64, 9000)), 0, 0),
             gen.ATTN_DECODE: lambda: (0, 8 * int(rng.integers(1, 9)), 128, int(rng.integers(1, 9)), 0),
             gen.RMSNORM: lambda: (int(rng.integers(1, 3000)), 4096, 0, 0, 0),
             gen.SILU_MUL: lambda: (int(rng.integers(1, 3000)), int(rng.integers(1, 30000)), 0, 0, 0),
             gen.EMBED: lambda: (int(rng.integers(1, 3000)), 8192, 0, 0, 0)}
    for f, mk in shape.items():
        for j in range(n_steps):
            if rng.uniform() < 0.1:
                continue
            run = int(rng.integers(1, max_run + 1)) if rng.uniform() < 0.7 else int(rng.integers(1, 6))
            rows += [(f, j) + mk() for _ in range(run)]
    sp = gen.specs_grid(n_specs, 7) if n_specs > 1 else spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6)
    return _wl(make_desc(rows, reqs), n_steps, specs=sp)


@pytest.mark.parametrize("seed,n_steps,max_run,n_specs", [(1, 40, 9, 1), (2, 60, 70, 3), (3, 30, 300, 5),
                                                           (4, 400, 200, 2)])
def test_eta_one_step_sums_runs_at_every_offset(seed, n_steps, max_run, n_specs):
    """The eta = 1 step sums without per-pair outputs (each lane sums four
    consecutive records, a row scan joins the lanes) against the oracle, and
    against the same call with per-pair outputs (one record per lane)."""
    wl = _run_workload(seed, n_steps, max_run, n_specs)
    ref = o.eval_kernels(wl.desc, wl.specs, eta_one=True)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, eta_one=True, kern=ref)
    steps_only = g.eval_steps(wl, eta_one=True, per_pair=False)
    _check_steps(wl, steps_only, rs, bf16=False, n_specs=wl.n_specs)
    per_pair = g.eval_steps(wl, eta_one=True, counts=False)
    _check_kernels(wl, per_pair, ref, bf16=False, eta_one=True)
    for key in ("t_body", "t_gpu", "t_step"):
        assert g.rel_err(steps_only[key], per_pair[key]).max() <= 2 * REL
    again = g.eval_steps(wl, eta_one=True, per_pair=False)
    for key in ("t_body", "t_gpu", "t_step"):
        np.testing.assert_array_equal(again[key], steps_only[key])


def _multi_spec(n_cus):
    n = len(n_cus)
    rng = np.random.default_rng(11)
    return {"peak_flops": rng.uniform(0.5e15, 5e15, n), "hbm_bw": rng.uniform(2e12, 1e13, n),
            "t0": np.full(n, 2e-6), "l2_bytes": np.full(n, 64.0 * 2 ** 20),
            "ar_alpha0": np.full(n, 8e-6), "ar_alpha_log2p": np.full(n, 2e-6),
            "ar_beta": np.full(n, 300e9), "n_cu": np.asarray(n_cus, np.int64)}


def _block_count_workload(heads=None):
    """Block counts that are exact multiples of the CU counts, and one off,
    in a first SiLU tile that stays below 2^23; then a SiLU tile that
    crosses it (2^23 - 1, 2^23, 2^23 + 1, a multiple of 148 just above,
    2^24 - 1 and about 2^32).  A SiLU record (T, I) has B = ceil(T I / 1024),
    so (T, 1024) gives B = T."""
    n_cus = [148, 132, 256, 97, 1, 65535]
    rows = []
    for n in n_cus[:4]:                      # GEMM: B = ceil(M/128) ceil(N/128)
        for k in (1, 3, 7):
            for d in (-1, 0, 1):
                bb = k * n + d
                rows.append((gen.GEMM, 0, 128 * bb, 128, 64, 0, 0))
                rows.append((gen.GEMM, 0, 128 * bb - 5, 100, 64, 0, 0))
    small = [148 * k + d for k in (1, 50, 5000, 56679) for d in (-1, 0, 1)]
    small += [132 * k + d for k in (1, 63550) for d in (-1, 0, 1)]
    small += [256 * k + d for k in (1, 32767) for d in (-1, 0, 1)]
    small += [97 * k + d for k in (1, 86479) for d in (-1, 0, 1)]
    small += [65535 * k + d for k in (1, 128) for d in (-1, 0, 1)]
    assert max(small) < (1 << 23) and len(small) <= 64
    rows += [(gen.SILU_MUL, 0, v, 1024, 0, 0, 0) for v in small]
    rows += [(gen.SILU_MUL, 0, 3 * 1024 + 7, 1, 0, 0, 0)] * (64 - len(small))
    big = [(1 << 23) - 1, 1 << 23, (1 << 23) + 1, 148 * 56680, (1 << 24) - 1]
    rows += [(gen.SILU_MUL, 0, v, 1024, 0, 0, 0) for v in big]
    rows += [(gen.SILU_MUL, 0, (1 << 24) - 1, (1 << 18) - 1, 0, 0, 0), (gen.SILU_MUL, 0, 5, 7, 0, 0, 0)]
    d = make_desc(rows, [[(1, 1)]])
    return _wl(d, 1, specs=_multi_spec(n_cus), heads=heads)


def _stream_block_count_workload():
    """SiLU block counts k N - 1, k N and k N + 1 just below 2^22 for every
    CU count, all in the first 256-record tile (so the stream's fp32 wave
    count, exact below 2^22, takes them), then a tile with counts from
    2^22 - 1 up (its fp64 path)."""
    n_cus = [148, 132, 256, 97, 1, 65535]
    near = []
    for n in n_cus:
        k = ((1 << 22) - 2) // n
        near += [v for v in (k * n - 1, k * n, k * n + 1) if v < (1 << 22)]
    rows = [(gen.SILU_MUL, 0, v, 1024, 0, 0, 0) for v in near]
    rows += [(gen.SILU_MUL, 0, 1000 + i, 1024, 0, 0, 0) for i in range(256 - len(rows))]
    rows += [(gen.SILU_MUL, 0, v, 1024, 0, 0, 0)
             for v in ((1 << 22) - 1, 1 << 22, (1 << 22) + 1, (1 << 23) + 1, (1 << 24) - 1)]
    d = make_desc(rows, [[(1, 1)]])
    return _wl(d, 1, specs=_multi_spec(n_cus))


@pytest.mark.parametrize("bounded", [False, True])
def test_stream_wave_count_just_below_2_22(bounded):
    wl = _stream_block_count_workload()
    bd = gen.make_bounded(gen.BOUNDED_ALL) if bounded else None
    ref = o.eval_kernels(wl.desc, wl.specs, None, eta_one=True, bounded=bd)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, eta_one=True, kern=ref)
    steps_only = g.eval_steps(wl, eta_one=True, per_pair=False, bounded=bd)
    _check_steps(wl, steps_only, rs, bf16=False, n_specs=wl.n_specs)
    gpu = g.eval_steps(wl, eta_one=True, counts=False, bounded=bd)
    for k, r in (("t_roof", "t_roof"), ("eta", "eta"), ("t_kernel", "t")):
        assert g.rel_err(gpu[k], ref[r]).max() <= REL, k


def test_block_counts_around_the_fp32_wave_path():
    wl = _block_count_workload()
    b = o.kernel_counts(wl.desc)["B"]
    assert (b >= (1 << 23)).any() and (b < (1 << 23)).any()
    _eta1_case(wl, counts=True)
    _eta1_case(wl, counts=False)


def test_block_counts_around_the_fp32_wave_path_bf16_head():
    _edge_check(_block_count_workload(heads=gen.make_heads(16, 128, "bf16")))


def test_n_cu_above_limit_flagged():
    sp = spec(n_cu=70000)
    wl = _wl(make_desc([(gen.GEMM, 0, 77, 300, 129, 0, 0)], [[(1, 5)]]), 1, specs=sp)
    with pytest.raises(abi.KsError) as e:
        g.eval_kernels(wl, eta_one=True)
    assert e.value.status == abi.KS_ERANGE


# ------------------------------------------------------------ maximum size --
C5_BATCH_STEPS = 88_640      # steps 0 .. 88,640 of the 70B trace: 63,998,080 records


_sub_desc = sub_desc


def test_max_size_batch_sampled():
    """The benchmark's 70B batch (the largest single call of that workload:
    88,640 steps of the prefix-cache trace, 63,998,080 records, prefill steps
    with prefix-shortened chunks and decode steps) in the launch
    configuration the benchmark times, bf16 32-256 heads and eta = 1:
    sampled prefill and decode steps against the oracle, bf16 eta also
    against the plain fp64 definition (no bf16 rounding points); the eta = 1
    step sums of the streaming kernel against the per-pair path on every
    step."""
    import torch
    wl = gen.config5(0, C5_BATCH_STEPS)
    d = wl.desc
    assert d.n_rows == 63_998_080
    fam = d.family()
    pre_steps = np.unique(d.step[fam == gen.ATTN_PREFILL])
    dec_steps = np.unique(d.step[fam == gen.ATTN_DECODE])
    assert len(pre_steps) > 0 and len(dec_steps) > 0
    rng = np.random.default_rng(3)
    steps = np.unique(np.concatenate([[0, d.n_steps - 1], rng.choice(pre_steps, 4), rng.choice(dec_steps, 4)]))
    rows = np.nonzero(np.isin(d.step, steps))[0]
    assert (fam[rows] == gen.ATTN_PREFILL).any() and (fam[rows] == gen.ATTN_DECODE).any()
    rows_t = torch.as_tensor(rows, device="cuda")
    sub = _sub_desc(d, rows)
    for eta_one in (False, True):
        print(f"[max batch] eta_one={eta_one}", flush=True)
        di = abi.DeviceInputs(wl)
        heads = di.make_heads("bf16", 32, 256, abi.KS_ETA_ONE if eta_one else abi.KS_ETA_MLP)
        so_t, so = abi.step_outputs(d.n_steps, di.n_specs)
        ko_t, ko = abi.kernel_outputs(d.n_rows, di.n_specs, counts=False)
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                          di.ws_ptr, di.ws_bytes, abi.current_stream())
        torch.cuda.synchronize()
        abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
        gpu = {key: ko_t[key][:, rows_t].cpu().numpy() for key in ("t_roof", "eta", "t_kernel")}
        body_all = so_t["t_body"].cpu().numpy()
        body = body_all[:, steps]
        del ko_t
        stream = None
        if eta_one:
            # the same call without per-pair outputs: the eta = 1 streaming
            # kernel, in the launch configuration the benchmark times
            abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, None,
                              di.ws_ptr, di.ws_bytes, abi.current_stream())
            torch.cuda.synchronize()
            abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
            stream = so_t["t_body"].cpu().numpy()
            assert g.rel_err(stream, body_all).max() <= 2 * REL
        del di, so_t
        torch.cuda.empty_cache()
        ref = o.eval_kernels(sub, wl.specs, None if eta_one else wl.heads, eta_one=eta_one)
        assert g.rel_err(gpu["t_roof"], ref["t_roof"]).max() <= REL
        if eta_one:
            assert (gpu["eta"] == 1.0).all()
            assert g.rel_err(gpu["t_kernel"], ref["t"]).max() <= REL
        else:
            assert g.rel_err(gpu["eta"], ref["eta"]).max() <= REL_BF16
            dz = np.abs(_z_from_eta(gpu["eta"]) - ref["z"])
            assert dz.max() <= ZTOL, dz.max()
            assert g.rel_err(gpu["t_kernel"], ref["t"]).max() <= REL_BF16
            pure = o.eval_kernels(sub, wl.specs, wl.heads, emulate_bf16=False)
            assert g.rel_err(gpu["eta"], pure["eta"]).max() <= REL_BF16
            assert g.rel_err(gpu["t_kernel"], pure["t"]).max() <= REL_BF16
        t_ge = np.maximum(ref["t_roof"] * gpu["eta"], wl.specs["t0"][:, None])
        assert g.rel_err(gpu["t_kernel"], t_ge).max() <= REL
        for s in range(wl.n_specs):
            ref_body = np.bincount(d.step[rows], weights=t_ge[s], minlength=d.n_steps)[steps]
            assert g.rel_err(body[s], ref_body).max() <= REL
            if stream is not None:
                assert g.rel_err(stream[s, steps], ref_body).max() <= REL


# ------------------------------------------ bf16 heads vs the plain definition --
@pytest.mark.parametrize("which", ["c4", "c5"])
def test_bf16_heads_against_the_unrounded_definition(which):
    """bf16 heads against the model's plain fp64 definition (no bf16 rounding
    points at all, the oracle's emulate_bf16=False), not only against the
    emulation of the kernel's rounding: eta, t_kernel and the step outputs
    within the 1e-2 bar."""
    wl = (gen.config4(n_specs=24, grid_steps=25, c1_steps=40) if which == "c4" else gen.config5(0, 24))
    gpu = g.eval_steps(wl)
    pure = o.eval_kernels(wl.desc, wl.specs, wl.heads, emulate_bf16=False)
    assert g.rel_err(gpu["eta"], pure["eta"]).max() <= REL_BF16
    assert g.rel_err(gpu["t_kernel"], pure["t"]).max() <= REL_BF16
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, wl.heads, kern=pure)
    _check_steps(wl, gpu, rs, bf16=True, n_specs=wl.n_specs)


# ------------------------------------------------- K fields the model ignores --
@pytest.mark.parametrize("precision,in_dim,hidden", [("f32", 16, 64), ("bf16", 16, 128)])
def test_unused_k_fields_are_ignored(precision, in_dim, hidden):
    """Norm, activation and embedding records carry no K: garbage in their k
    field changes nothing (their K feature is 0 on both sides), while the
    other families' k still counts."""
    wl = gen.config1(0, 40).with_heads(gen.make_heads(in_dim, hidden, precision))
    d = wl.desc
    fam = d.family()
    unused = np.isin(fam, [gen.RMSNORM, gen.SILU_MUL, gen.EMBED])
    k = d.k.copy()
    k[unused] = np.random.default_rng(9).integers(1, 1 << 17, int(unused.sum())).astype(np.uint32)
    dk = gen.Desc(d.fam_off, d.step, d.m, d.n, k, d.a, d.b, d.req_off, d.req_q, d.req_h, d.expert_rows,
                  d.elem_bytes)
    wk = gen.Workload(wl.name, dk, wl.steps, wl.specs, wl.heads, wl.host)
    ref = o.eval_kernels(dk, wl.specs, wl.heads)
    gpu = g.eval_steps(wk)
    _check_kernels(wk, gpu, ref, bf16=precision == "bf16")
    base = g.eval_steps(wl)
    for key in ("eta", "t_kernel", "t_body", "t_step"):
        np.testing.assert_array_equal(gpu[key], base[key], err_msg=key)
    eta1 = g.eval_steps(wk, eta_one=True, per_pair=False)
    eta1_base = g.eval_steps(wl, eta_one=True, per_pair=False)
    np.testing.assert_array_equal(eta1["t_body"], eta1_base["t_body"])


# -------------------------------------------------- bounded analytical head --
def _bounded_case(wl, bd, eta_one=False, n_specs=None, null_mlp=False, counts=True):
    """Families in bd.mask: fp32 bounded head at 1e-5; the others keep the
    MLP bar of their precision (or eta = 1 exactly).  counts=False: no
    per-record count outputs (F and Bt formed in fp32)."""
    n_specs = n_specs or wl.n_specs
    heads = None if eta_one else wl.heads
    ref = o.eval_kernels(wl.desc, wl.specs, heads, eta_one=eta_one, spec_ids=range(n_specs), bounded=bd)
    gpu = g.eval_steps(wl, eta_one=eta_one, n_specs=n_specs, bounded=bd, null_mlp=null_mlp, counts=counts)
    c = ref["counts"]
    if counts:
        np.testing.assert_array_equal(gpu["flops"], c["F"])
    assert g.rel_err(gpu["t_roof"], ref["t_roof"]).max() <= REL
    on = ((bd.mask >> wl.desc.family()) & 1).astype(bool)
    assert g.rel_err(gpu["eta"][:, on], ref["eta"][:, on]).max() <= REL
    assert g.rel_err(gpu["t_kernel"][:, on], ref["t"][:, on]).max() <= REL
    bf16 = not eta_one and wl.heads.precision == "bf16"
    if (~on).any():
        tol = REL_BF16 if bf16 else REL
        assert g.rel_err(gpu["eta"][:, ~on], ref["eta"][:, ~on]).max() <= tol
    t0 = wl.specs["t0"][:n_specs, None]
    assert g.rel_err(gpu["t_kernel"], np.maximum(ref["t_roof"] * gpu["eta"].astype(np.float64), t0)).max() <= REL
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, heads, eta_one=eta_one,
                      spec_ids=range(n_specs), kern=ref)
    _check_steps(wl, gpu, rs, bf16=bf16 and (~on).any(), n_specs=n_specs)
    _check_steps(wl, gpu, _steps_given_eta(wl, gpu, ref, n_specs), bf16=False, n_specs=n_specs)


def test_bounded_mixed_with_bf16_mlp():
    _bounded_case(gen.config4(n_specs=12, grid_steps=20, c1_steps=30), gen.make_bounded(gen.BOUNDED_MIXED))


def test_bounded_mixed_with_fp32_mlp_and_moe():
    _bounded_case(gen.config1(0, 60), gen.make_bounded(gen.BOUNDED_MIXED))
    _bounded_case(gen.config3(0, 20), gen.make_bounded(gen.BOUNDED_MIXED | (1 << gen.ATTN_DECODE)))


def test_bounded_only():
    """Every family bounded: through eta = 1 mode, and through MLP mode with
    NULL MLP weights (both run the head-less kernel)."""
    wl = gen.config1(0, 60)
    bd = gen.make_bounded(gen.BOUNDED_ALL)
    _bounded_case(wl, bd, eta_one=True)
    _bounded_case(wl, bd, null_mlp=True)
    _bounded_case(wl, bd, eta_one=True, counts=False)
    # some families bounded, the rest at eta = 1
    _bounded_case(wl, gen.make_bounded(gen.BOUNDED_MIXED), eta_one=True)
    _bounded_case(wl, gen.make_bounded(gen.BOUNDED_MIXED), eta_one=True, counts=False)


@pytest.mark.parametrize("seed,n_steps,max_run,n_specs", [(1, 40, 9, 1), (3, 30, 300, 5), (4, 400, 200, 2)])
@pytest.mark.parametrize("mask", [gen.BOUNDED_ALL, gen.BOUNDED_MIXED])
def test_bounded_stream_step_sums_runs_at_every_offset(seed, n_steps, max_run, n_specs, mask):
    """Calls without an MLP family take the stream (four records per lane)
    with the bounded head on its families: step sums alone, and with
    per-pair outputs, against the oracle over runs ending at every lane,
    row and tile offset."""
    wl = _run_workload(seed, n_steps, max_run, n_specs)
    bd = gen.make_bounded(mask)
    ref = o.eval_kernels(wl.desc, wl.specs, None, eta_one=True, bounded=bd)
    rs = o.eval_steps(wl.desc, wl.steps, wl.specs, wl.host, eta_one=True, kern=ref)
    steps_only = g.eval_steps(wl, eta_one=True, per_pair=False, bounded=bd)
    _check_steps(wl, steps_only, rs, bf16=False, n_specs=wl.n_specs)
    per_pair = g.eval_steps(wl, eta_one=True, counts=False, bounded=bd)
    assert g.rel_err(per_pair["eta"], ref["eta"]).max() <= REL
    assert g.rel_err(per_pair["t_kernel"], ref["t"]).max() <= REL
    assert g.rel_err(per_pair["t_roof"], ref["t_roof"]).max() <= REL
    for key in ("t_body", "t_gpu", "t_step"):
        assert g.rel_err(steps_only[key], per_pair[key]).max() <= 2 * REL


def test_bounded_with_block_counts_around_2_23():
    wl = _block_count_workload(heads=gen.make_heads(32, 256, "bf16"))
    _bounded_case(wl, gen.make_bounded(gen.BOUNDED_ALL ^ (1 << gen.GEMM)))


# ------------------------------------------- Tier B measured grids (Sec. 5.5) --
GRID_EPS = 1e-5   # node units: fp32 coordinates may sit on either side of a face this close


def _grid_eta_check(wl, gr, ref, plain, gpu_eta, n_specs, fallback_tol):
    """Pairs with every coordinate farther than GRID_EPS from a cell face are
    routed as the oracle routes them and match its eta (REL when routed, the
    fallback head's bar otherwise).  Pairs that close to a face match the
    fallback or the grid at one of the nearby points on either side."""
    fam = wl.desc.family()
    on = ((gr.mask >> fam) & 1).astype(bool)
    ax = list(gr.axes)
    n = np.asarray(gr.n, np.float64)
    step = (gr.hi - gr.lo) / (n - 1)
    n_amb = 0
    amb_all = np.zeros((n_specs, len(fam)), bool)
    for s in range(n_specs):
        x = ref["x16"][s]
        t = (x[:, ax] - gr.lo) / step
        amb = on & (np.abs(t - np.round(t)) < GRID_EPS).any(axis=1)
        amb_all[s] = amb
        n_amb += int(amb.sum())
        routed = ref["routed"][s] & ~amb
        rest = ~routed & ~amb
        assert g.rel_err(gpu_eta[s, routed], ref["eta"][s, routed]).max(initial=0) <= REL
        assert g.rel_err(gpu_eta[s, rest], ref["eta"][s, rest]).max(initial=0) <= fallback_tol
        for r in np.nonzero(amb)[0]:
            cands = [plain["eta"][s, r]]
            for sg in np.array(np.meshgrid(*[[-2, 0, 2]] * 3)).reshape(3, -1).T:
                xn = x[r].copy()
                xn[ax] += sg * GRID_EPS * step
                e, rr = o.grid_eta(xn[None], gr, fam[r])
                if rr[0]:
                    cands.append(e[0])
            tol = max(REL * 4, fallback_tol)
            assert min(g.rel_err(gpu_eta[s, r], c) for c in cands) <= tol, (s, r, gpu_eta[s, r], cands)
    assert n_amb <= 0.01 * on.sum() * n_specs
    return amb_all


def _grid_case(wl, gr, eta_one=False, bounded=None, null_mlp=False, n_specs=None, expect_routed=True):
    n_specs = n_specs or wl.n_specs
    heads = None if eta_one else wl.heads
    kw = dict(eta_one=eta_one, spec_ids=range(n_specs), bounded=bounded)
    ref = o.eval_kernels(wl.desc, wl.specs, heads, grid=gr, **kw)
    plain = o.eval_kernels(wl.desc, wl.specs, heads, **kw)
    gpu = g.eval_steps(wl, eta_one=eta_one, n_specs=n_specs, bounded=bounded, grid=gr, null_mlp=null_mlp,
                       source=True)
    if expect_routed:
        assert ref["routed"].any() and (~ref["routed"]).any()
    np.testing.assert_array_equal(gpu["flops"], ref["counts"]["F"])
    assert g.rel_err(gpu["t_roof"], ref["t_roof"]).max() <= REL
    bf16 = not eta_one and wl.heads.precision == "bf16"
    fam = wl.desc.family()
    on_b = ((bounded.mask if bounded is not None else 0) >> fam) & 1
    mlp_fallback = bf16 and not (on_b.astype(bool)).all()
    amb = _grid_eta_check(wl, gr, ref, plain, gpu["eta"], n_specs, REL_BF16 if mlp_fallback else REL)
    # where each pair's eta came from: the grid where the oracle routes it
    # (pairs within GRID_EPS of a cell face may go either way), else the
    # bounded head for its families, else the mode's head
    fallback = np.broadcast_to(np.where(on_b.astype(bool), 1, 0)[None, :], ref["routed"].shape)
    want = np.where(ref["routed"], 2, fallback)
    src = gpu["source"].astype(np.int64)
    np.testing.assert_array_equal(src[~amb], want[~amb])
    assert ((src[amb] == 2) | (src[amb] == fallback[amb])).all()
    t0 = wl.specs["t0"][:n_specs, None]
    assert g.rel_err(gpu["t_kernel"], np.maximum(ref["t_roof"] * gpu["eta"].astype(np.float64), t0)).max() <= REL
    _check_steps(wl, gpu, _steps_given_eta(wl, gpu, ref, n_specs), bf16=False, n_specs=n_specs)
    return ref, gpu


def _quantile_grid(wl, mask, axes, q=(0.1, 0.9), n=(6, 5, 7), holes=0.08, seed=gen.GRID_SEED):
    """A grid over the central quantiles of the workload's own features
    (taken from the oracle), so part of the records fall inside."""
    x = o.eval_kernels(wl.desc, wl.specs, None, eta_one=True,
                       grid=gen.make_grid(0, axes=axes))["x16"].reshape(-1, 16)[:, list(axes)]
    lo, hi = np.quantile(x, q[0], axis=0), np.quantile(x, q[1], axis=0)
    hi = np.maximum(hi, lo + 1e-3)
    # off the features' recurring exact values (x4 = 1/16 at one wave, ...)
    w = hi - lo
    lo, hi = lo - 0.0137 * w, hi + 0.0191 * w
    return gen.make_grid(mask, axes=axes, lo=lo, hi=hi, n=n, holes=holes, seed=seed)


def test_grid_with_fp32_mlp():
    wl = gen.config1(0, 60)
    _grid_case(wl, gen.make_grid(gen.GRID_ALL ^ (1 << gen.GEMM)))


def test_grid_with_bf16_mlp():
    """bf16 MLP fallback; the head is skipped for waves with every record on
    the grid."""
    wl = gen.config4(n_specs=12, grid_steps=20, c1_steps=30)
    _grid_case(wl, _quantile_grid(wl, gen.GRID_ALL, (1, 2, 6)))


def test_grid_eta_one_and_bounded_fallbacks():
    wl = gen.config1(0, 60)
    gr = gen.make_grid(gen.GRID_ALL)
    _grid_case(wl, gr, eta_one=True)
    bd = gen.make_bounded(gen.BOUNDED_MIXED)
    _grid_case(wl, gr, bounded=bd)
    _grid_case(wl, gr, eta_one=True, bounded=bd)
    _grid_case(wl, gr, bounded=gen.make_bounded(gen.BOUNDED_ALL), null_mlp=True)


@pytest.mark.parametrize("axes", [(0, 3, 4), (5, 7, 8), (9, 10, 11), (12, 13, 14), (2, 1, 6)])
def test_grid_every_feature_axis(axes):
    wl = gen.config3(0, 20)
    _grid_case(wl, _quantile_grid(wl, gen.GRID_ALL, axes), expect_routed=False)


def test_grid_sizes_and_degenerate_grids():
    """The largest grid (2048 nodes), the smallest (2 x 2 x 2), a grid with
    no holes, one with no measured node (routes nothing: the plain result)."""
    wl = gen.config1(0, 40)
    _grid_case(wl, _quantile_grid(wl, gen.GRID_ALL, (1, 2, 6), n=(16, 16, 8)))
    _grid_case(wl, _quantile_grid(wl, gen.GRID_ALL, (1, 2, 6), n=(2, 2, 2), holes=0.0))
    _grid_case(wl, _quantile_grid(wl, gen.GRID_ALL, (1, 2, 6), n=(9, 3, 4), holes=0.0))
    ref, gpu = _grid_case(wl, gen.make_grid(gen.GRID_ALL, holes=1.0), expect_routed=False)
    assert not ref["routed"].any()
    plain = g.eval_steps(wl)
    np.testing.assert_array_equal(gpu["eta"], plain["eta"])
    np.testing.assert_array_equal(gpu["t_step"], plain["t_step"])


@pytest.mark.parametrize("bounded_mask", [0, gen.BOUNDED_MIXED, gen.BOUNDED_ALL])
def test_eta_source_without_grid(bounded_mask):
    """Without a grid every pair's eta comes from its family's head: the
    bounded head for the families in the mask, the MLP for the others."""
    wl = gen.config1(0, 30)
    bd = gen.make_bounded(bounded_mask) if bounded_mask else None
    gpu = g.eval_steps(wl, bounded=bd, source=True)
    want = ((bounded_mask >> wl.desc.family()) & 1).astype(np.uint8)
    np.testing.assert_array_equal(gpu["source"], np.broadcast_to(want, gpu["source"].shape))
