"""The allocation-free entry point ks_eval_steps_static against ks_eval_steps
with a caller-provided workspace: the same kernels, so the same outputs bit
for bit, on consecutive calls that leave the shared device array behind
(the second smaller than the first); the size limit is refused on the host
before any launch."""
import ctypes as C

import numpy as np
import pytest

from paper_2606_28565_amd import abi
from tests.helpers import make_desc, spec, steprec
from workload import gen


def _run(wl, eta_one=False, per_pair=True, static=False, bad=False):
    import torch
    di = abi.DeviceInputs(wl)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden,
                          abi.KS_ETA_ONE if eta_one else abi.KS_ETA_MLP)
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    ko_t, ko = (abi.kernel_outputs(wl.desc.n_rows, di.n_specs) if per_pair else ({}, None))
    stream = abi.current_stream()
    flags = None
    if static:
        flags = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        abi.ks_eval_steps_static(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                                 flags.data_ptr(), stream)
    else:
        abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                          di.ws_ptr, di.ws_bytes, stream)
        if not bad:
            abi.ks_device_status(di.ws_ptr, di.ws_bytes, stream)
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in so_t.items()}
    out.update({k: v.cpu().numpy() for k, v in ko_t.items()})
    if flags is not None:
        out["flags"] = int(flags.cpu().numpy()[0])
    return out


def _same(a, b):
    assert a.keys() - {"flags"} == b.keys() - {"flags"}
    for k in b:
        if k != "flags":
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


@pytest.mark.gpu
def test_static_entry_matches_workspace_entry_on_consecutive_calls():
    """Capacity-grid subset (bf16 16-128 heads, 64 spec vectors), then a
    smaller Llama-7B slice (fp32 heads), then the eta = 1 step sums of a
    70B slice (the streaming kernel): each call of the static entry point
    against the workspace entry point's outputs, bit for bit."""
    big = gen.config4(n_specs=64, grid_steps=60, c1_steps=300)
    small = gen.config1(0, 50)
    cases = [(big, False, True), (small, False, True), (gen.config5(0, 30), True, False)]
    for wl, eta_one, per_pair in cases:
        print(f"[static] {wl.name} {wl.desc.n_rows} records x {wl.n_specs} specs eta_one={eta_one}", flush=True)
        ref = _run(wl, eta_one=eta_one, per_pair=per_pair)
        got = _run(wl, eta_one=eta_one, per_pair=per_pair, static=True)
        assert got["flags"] == 0
        _same(got, ref)
    # the first case again after the smaller ones: the array holds the last
    # call's contents, and nothing of them leaks into this call
    again = _run(big, static=True)
    assert again["flags"] == 0
    _same(again, _run(big))


@pytest.mark.gpu
def test_static_entry_reports_bad_data_flags():
    """A record whose step is beyond n_steps: skipped and flagged; the flag
    word reaches the caller's device pointer and the step sums are those of
    the workspace entry point on the same input."""
    rows = [(gen.GEMM, 0, 4, 64, 64, 0, 0), (gen.GEMM, 7, 4, 64, 64, 0, 0)]
    wl = gen.Workload("bad", make_desc(rows, [[(1, 10)], [(2, 20)]]), steprec(2),
                      spec(P=1e15, BW=4e12, n_cu=132, t0=2e-6), gen.make_heads(16, 64, "f32"), gen.HostConsts())
    got = _run(wl, per_pair=False, static=True)
    assert got["flags"] != 0
    ref = _run(wl, per_pair=False, bad=True)
    np.testing.assert_array_equal(got["t_body"], ref["t_body"])
    good = _run(gen.config1(0, 5), per_pair=False, static=True)
    assert good["flags"] == 0


def test_static_entry_refuses_calls_beyond_its_array():
    """A call needing more workspace than the static array is refused with
    KS_ERANGE on the host, before any launch (fake device pointers: nothing
    is dereferenced)."""
    d = abi.ks_desc()
    n_rows = 1 << 20
    d.n_rows = n_rows
    for f in range(abi.NFAM + 1):
        d.fam_off[f] = 0 if f == 0 else n_rows
    for name in ("step", "m", "n", "k", "a", "b", "req_off", "req_q", "req_h"):
        setattr(d, name, 0x1000)
    d.n_steps = 1 << 20
    d.n_req = 3
    d.elem_bytes = 2
    n_specs = 64
    need = abi.ks_workspace_bytes(d, n_specs)
    assert need > abi.KS_STATIC_SCRATCH_BYTES
    st = abi.ks_steps()
    st.n_steps = d.n_steps
    for name in ("layers", "hidden", "tp", "n_launch"):
        setattr(st, name, 0x1000)
    h = abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_ONE)
    host = abi.ks_host(0, 0, 0, 0, 1)
    so = abi.ks_step_out(0x3000, 0x3000, 0x3000)
    rc = abi.ks_eval_steps_static(d, st, 0x2000, n_specs, h, host, so, None, None, None, check=False)
    assert rc == abi.KS_ERANGE
    assert "static scratch" in abi.ks_last_error()
    # bad arguments get the evaluation's own message
    rc = abi.ks_eval_steps_static(d, st, 0x2000, 0, h, host, so, None, None, None, check=False)
    assert rc == abi.KS_EINVAL and "n_specs" in abi.ks_last_error()
