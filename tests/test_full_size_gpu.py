"""The six-shape and mixture-of-experts workloads at full size, in the
launch configuration the benchmark times (each shape's whole 100k-step
trace, the whole 200k-step MoE trace, in one call): sampled prefill and
decode steps against the oracle, which prices just those steps' records.
Counts bit-exact; t_roof and, given the GPU's eta, t and the step outputs
within 1e-5; bf16 eta against the oracle's emulation of the bf16 rounding
points and against the plain fp64 definition within 1e-2."""
import numpy as np
import pytest
import torch  # noqa: F401  (runtime loads at collection, not inside a timed test)

from oracle import ks_oracle as o
from paper_2606_28565_amd import abi
from tests import gpu_helpers as g
from tests.helpers import sub_desc
from workload import gen

pytestmark = pytest.mark.gpu

REL = 1e-5
REL_BF16 = 1e-2


def _sampled_check(wl, seed):
    import torch
    d = wl.desc
    fam = d.family()
    pre = np.unique(d.step[fam == gen.ATTN_PREFILL])
    dec = np.unique(d.step[fam == gen.ATTN_DECODE])
    assert len(pre) and len(dec)
    rng = np.random.default_rng(seed)
    steps = np.unique(np.concatenate([[0, d.n_steps - 1], rng.choice(pre, 3), rng.choice(dec, 3)]))
    rows = np.nonzero(np.isin(d.step, steps))[0]
    print(f"[full size] {wl.name}: {d.n_rows} records, {d.n_steps} steps; steps {steps.tolist()}", flush=True)
    di = abi.DeviceInputs(wl)
    so_t, so = abi.step_outputs(d.n_steps, di.n_specs)
    ko_t, ko = abi.kernel_outputs(d.n_rows, di.n_specs)
    abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, di.heads, di.host, so, ko,
                      di.ws_ptr, di.ws_bytes, abi.current_stream())
    torch.cuda.synchronize()
    abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
    rows_t = torch.as_tensor(rows, device="cuda")
    gpu = {k: ko_t[k][:, rows_t].cpu().numpy() for k in ("t_roof", "eta", "t_kernel")}
    cnt = {k: ko_t[k][rows_t].cpu().numpy().view(np.uint64) for k in ("flops", "bytes", "blocks")}
    step_out = {k: so_t[k].cpu().numpy()[:, steps] for k in ("t_body", "t_gpu", "t_step")}
    del ko_t
    # the benchmark's launch: step outputs only (no per-pair or count
    # outputs, so F, Bt and the row-count feature are formed in fp32)
    abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, di.heads, di.host, so, None,
                      di.ws_ptr, di.ws_bytes, abi.current_stream())
    torch.cuda.synchronize()
    abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
    bench_out = {k: so_t[k].cpu().numpy()[:, steps] for k in ("t_body", "t_gpu", "t_step")}
    del so_t, di
    torch.cuda.empty_cache()

    sd = sub_desc(d, rows)
    ref = o.eval_kernels(sd, wl.specs, wl.heads)
    c = ref["counts"]
    np.testing.assert_array_equal(cnt["flops"], c["F"])
    np.testing.assert_array_equal(cnt["bytes"], c["Bt"])
    np.testing.assert_array_equal(cnt["blocks"], c["B"])
    assert g.rel_err(gpu["t_roof"], ref["t_roof"]).max() <= REL
    assert g.rel_err(gpu["eta"], ref["eta"]).max() <= REL_BF16
    pure = o.eval_kernels(sd, wl.specs, wl.heads, emulate_bf16=False)
    assert g.rel_err(gpu["eta"], pure["eta"]).max() <= REL_BF16
    t0 = wl.specs["t0"][:, None]
    t_ge = np.maximum(ref["t_roof"] * gpu["eta"].astype(np.float64), t0)
    assert g.rel_err(gpu["t_kernel"], t_ge).max() <= REL
    # step outputs: the oracle's step terms over the sampled steps' records,
    # with the GPU's eta (1e-5) and end to end (1e-2)
    kern = dict(ref)
    kern["t"] = t_ge
    ge = o.eval_steps(sd, wl.steps, wl.specs, wl.host, spec_ids=range(wl.n_specs), kern=kern)
    e2e = o.eval_steps(sd, wl.steps, wl.specs, wl.host, spec_ids=range(wl.n_specs), kern=ref)
    for k in ("t_body", "t_gpu", "t_step"):
        assert g.rel_err(step_out[k], ge[k][:, steps]).max() <= REL, k
        assert g.rel_err(step_out[k], e2e[k][:, steps]).max() <= REL_BF16, k
        assert g.rel_err(bench_out[k], e2e[k][:, steps]).max() <= REL_BF16, k
        assert g.rel_err(bench_out[k], step_out[k]).max() <= REL_BF16, k


@pytest.mark.parametrize("shape_idx", range(6))
def test_six_shape_workload_full_trace(shape_idx):
    """Each dense shape (hidden 2048..8192, TP 1..8: the all-reduce term of
    Eq. 3 in every step) over its whole trace."""
    _sampled_check(gen.config2(shape_idx), 40 + shape_idx)


def test_moe_workload_full_trace():
    """The Mixtral-like decoder's whole trace: ragged grouped GEMMs (experts
    with no routed rows included) over 51.2M routed row counts."""
    wl = gen.config3()
    assert (wl.desc.expert_rows == 0).any()
    _sampled_check(wl, 7)
