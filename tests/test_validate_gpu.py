"""Bad device data is reported, never faulted on: every index the kernels
derive from device data is bounds-checked in the kernel (out-of-range
records are skipped and flagged), and ks_validate names the problem.
The conditions are forced from the host by writing bad values into
correctly sized arrays."""
import numpy as np
import pytest

from paper_2606_28565_amd import abi
from workload import gen
from tests.helpers import make_desc, spec, steprec

pytestmark = pytest.mark.gpu


def _wl(rows, reqs, experts=(), specs=None):
    d = make_desc(rows, reqs, expert_rows=experts)
    return gen.Workload("bad", d, steprec(len(reqs)), specs or spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6),
                        gen.make_heads(16, 64, "f32"), gen.HostConsts())


GOOD_ROWS = [(gen.GEMM, 0, 4, 64, 64, 0, 0), (gen.GEMM, 1, 4, 64, 64, 0, 0),
             (gen.GROUPED_GEMM, 1, 0, 64, 64, 2, 0), (gen.ATTN_DECODE, 0, 0, 8, 128, 2, 0)]
GOOD_REQS = [[(1, 10)], [(2, 20)]]


def _validate(wl):
    import torch
    di = abi.DeviceInputs(wl)
    st = abi.ks_validate(di.desc, di.steps, di.specs_ptr, di.n_specs, di.ws_ptr, di.ws_bytes,
                         abi.current_stream(), check=False)
    torch.cuda.synchronize()
    return st, abi.ks_last_error()


def _eval_status(wl):
    import torch
    di = abi.DeviceInputs(wl)
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, di.heads, di.host, so, None,
                      di.ws_ptr, di.ws_bytes, abi.current_stream())
    st = abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream(), check=False)
    torch.cuda.synchronize()
    return st, abi.ks_last_error(), {k: v.cpu().numpy() for k, v in so_t.items()}


def _eval_status_eta_one(wl):
    """eta = 1 step sums without per-pair outputs (the streaming kernel)."""
    import torch
    di = abi.DeviceInputs(wl)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden, abi.KS_ETA_ONE)
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, None,
                      di.ws_ptr, di.ws_bytes, abi.current_stream())
    st = abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream(), check=False)
    torch.cuda.synchronize()
    return st, abi.ks_last_error(), {k: v.cpu().numpy() for k, v in so_t.items()}


def test_eta_one_stream_flags_and_skips_bad_records():
    """A record whose step is out of range, and a grouped GEMM whose expert
    offsets run past the table, are flagged by the eta = 1 stream; the other
    records' step sums are those of the input without the bad records."""
    good = GOOD_ROWS[:2] + [(gen.ATTN_DECODE, 0, 0, 8, 128, 2, 0)]
    st, msg, ref = _eval_status_eta_one(_wl(good, GOOD_REQS))
    assert st == abi.KS_OK, msg
    st, msg, out = _eval_status_eta_one(_wl(good + [(gen.GEMM, 7, 4, 64, 64, 0, 0)], GOOD_REQS))
    assert st == abi.KS_EINVAL and "step" in msg
    np.testing.assert_array_equal(out["t_body"], ref["t_body"])
    st, msg, _ = _eval_status_eta_one(_wl([(gen.GROUPED_GEMM, 0, 0, 64, 64, 4, 3)], [[(1, 1)]],
                                          experts=[1, 2, 3, 4]))
    assert st == abi.KS_EINVAL and "expert" in msg


def test_good_input_validates():
    st, msg = _validate(_wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0]))
    assert st == abi.KS_OK, msg


def test_step_out_of_range_flagged_and_skipped():
    rows = GOOD_ROWS[:1] + [(gen.GEMM, 7, 4, 64, 64, 0, 0)]      # step 7 >= n_steps 2
    st, msg, out = _eval_status(_wl(rows, GOOD_REQS))
    assert st == abi.KS_EINVAL and "step" in msg
    assert np.isfinite(out["t_step"]).all()
    st, msg = _validate(_wl(rows, GOOD_REQS))
    assert st == abi.KS_EINVAL and "step" in msg


def test_unsorted_steps_detected():
    wl = _wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0])
    wl.desc.step[:2] = [1, 0]                                   # GEMM segment decreases
    st, msg = _validate(wl)
    assert st == abi.KS_EINVAL and "decrease" in msg


def test_expert_offset_out_of_range_flagged():
    rows = [(gen.GROUPED_GEMM, 0, 0, 64, 64, 4, 3)]             # needs rows 3..6 of 4
    st, msg, _ = _eval_status(_wl(rows, [[(1, 1)]], experts=[1, 2, 3, 4]))
    assert st == abi.KS_EINVAL and "expert" in msg


def test_request_offsets_out_of_range_flagged():
    wl = _wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0])
    wl.desc.req_off[2] = 50                                      # beyond n_req = 2
    st, msg, _ = _eval_status(wl)
    assert st == abi.KS_EINVAL and "request" in msg


def test_shape_limits_flagged():
    rows = [(gen.GEMM, 0, 1 << 24, 64, 64, 0, 0)]
    st, msg = _validate(_wl(rows, [[(1, 1)]]))
    assert st == abi.KS_ERANGE and "limits" in msg


def test_bad_spec_flagged():
    sp = spec()
    sp["n_cu"][:] = 0
    st, msg = _validate(_wl(GOOD_ROWS[:1], GOOD_REQS[:1], specs=sp))
    assert st == abi.KS_ERANGE and "spec" in msg


@pytest.mark.parametrize("n_specs", [3, 1024, 1025, 1100])
def test_bad_spec_flagged_by_evaluation(n_specs):
    """A spec vector whose n_cu lies outside 1 .. 65535 is flagged by the
    evaluation call itself: with few specs their constants are formed in the
    clear kernel right after the flag word is reset, with many (1100) by a
    grid of their own.  The next call with good specs reports clean."""
    sp = {k: np.repeat(v, n_specs) for k, v in spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6).items()}
    for bad in (0, 70000):
        sp["n_cu"][n_specs - 1] = bad
        st, msg, _ = _eval_status(_wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0], specs=sp))
        assert st == abi.KS_ERANGE and "spec" in msg, (bad, msg)
    sp["n_cu"][n_specs - 1] = 132
    st, msg, _ = _eval_status(_wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0], specs=sp))
    assert st == abi.KS_OK, msg


@pytest.mark.parametrize("n", [1024, 1025, 1100])
def test_many_specs_match_single_spec_calls(n):
    """n distinct spec vectors in one call (spec constants formed in the
    clear kernel up to 1024 specs, by a grid of their own beyond) give, spec
    by spec, the step latencies of a one-spec call, bit for bit."""
    base = spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6)
    sp = {k: np.repeat(v, n) for k, v in base.items()}
    sp["peak_flops"] = 1e15 * (1.0 + np.arange(n) / n)
    sp["hbm_bw"] = 4e12 * (1.0 + 0.5 * np.cos(np.arange(n)))
    sp["n_cu"] = (64 + np.arange(n) % 200).astype(np.int64)
    st, msg, many = _eval_status(_wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0], specs=sp))
    assert st == abi.KS_OK, msg
    for i in sorted({0, 1, 1023, min(1024, n - 1), n - 1}):
        one = {k: v[i:i + 1].copy() for k, v in sp.items()}
        st, msg, out = _eval_status(_wl(GOOD_ROWS, GOOD_REQS, experts=[3, 0], specs=one))
        assert st == abi.KS_OK, msg
        for k in ("t_body", "t_gpu", "t_step"):
            np.testing.assert_array_equal(many[k].reshape(n, -1)[i], out[k].reshape(1, -1)[0], err_msg=f"{k} {i}")
