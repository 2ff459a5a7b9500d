"""The C-ABI library: loads, exports every declared symbol, matches the
header's struct layout, and rejects bad host arguments before any launch.
CPU only (no compute call reaches a GPU)."""
import ctypes as C
import os
import re
import subprocess

import pytest

from paper_2606_28565_amd import abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ks.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\**\s+\**(ks_\w+)\s*\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    lib = abi.load()
    names = _declared_functions()
    assert {"ks_eval_kernels", "ks_eval_steps", "ks_workspace_bytes", "ks_validate",
            "ks_device_status", "ks_last_error", "ks_version", "ks_expand", "ks_expand_layout",
            "ks_expand_workspace_bytes", "ks_simulate", "ks_simulate_workspace_bytes",
            "ks_set_timing_events"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert abi.ks_version().startswith("ks ")


def test_struct_layout_matches_header(tmp_path):
    """Compile a C probe of offsetof/sizeof against include/ks.h and compare
    with the ctypes mirrors."""
    structs = {"ks_desc": abi.ks_desc, "ks_spec": abi.ks_spec, "ks_heads": abi.ks_heads,
               "ks_steps": abi.ks_steps, "ks_host": abi.ks_host,
               "ks_kernel_out": abi.ks_kernel_out, "ks_step_out": abi.ks_step_out,
               "ks_model": abi.ks_model, "ks_batch": abi.ks_batch, "ks_records": abi.ks_records,
               "ks_sched": abi.ks_sched, "ks_requests": abi.ks_requests, "ks_sim_out": abi.ks_sim_out}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ks.h"', "int main(void){"]
    for s, cls in structs.items():
        lines.append(f'printf("{s} size %zu\\n", sizeof({s}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{s} {f} %zu\\n", offsetof({s}, {f}));')
    lines.append("return 0;}")
    c = tmp_path / "probe.c"
    c.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", str(c), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {}
    for line in out:
        if line:
            s, f, v = line.split()
            got[(s, f)] = int(v)
    for s, cls in structs.items():
        assert got[(s, "size")] == C.sizeof(cls), s
        for f, _ in cls._fields_:
            assert got[(s, f)] == getattr(cls, f).offset, (s, f)


def _desc(n_rows=10, n_steps=2):
    d = abi.ks_desc()
    d.n_rows = n_rows
    for f in range(abi.NFAM + 1):
        d.fam_off[f] = 0 if f == 0 else n_rows
    for name in ("step", "m", "n", "k", "a", "b", "req_off", "req_q", "req_h"):
        setattr(d, name, 0x1000)
    d.n_steps = n_steps
    d.n_req = 3
    d.elem_bytes = 2
    return d


def _call_eval(d, n_specs=1, heads=None, out=True, ws=0x100000, ws_bytes=1 << 30, specs=0x2000):
    h = heads or abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_ONE)
    o = abi.ks_kernel_out()
    return abi.ks_eval_kernels(d, specs, n_specs, h, o if out else None, ws, ws_bytes, None, check=False) \
        if out else abi.load().ks_eval_kernels(C.byref(d), specs, n_specs, C.byref(h), None, ws, ws_bytes, None)


@pytest.mark.parametrize("mutate,status,needle", [
    (lambda d: setattr(d, "step", None), abi.KS_EINVAL, "record array"),
    (lambda d: d.fam_off.__setitem__(3, 1), abi.KS_EINVAL, "fam_off"),
    (lambda d: [d.fam_off.__setitem__(i, 9) for i in range(1, abi.NFAM + 1)], abi.KS_EINVAL, "!= n_rows"),
    (lambda d: setattr(d, "req_off", None), abi.KS_EINVAL, "req_off"),
    (lambda d: setattr(d, "elem_bytes", 0), abi.KS_ERANGE, "elem_bytes"),
    (lambda d: setattr(d, "n_rows", -1), abi.KS_ERANGE, "n_rows"),
    (lambda d: setattr(d, "n_steps", 0), abi.KS_EINVAL, "n_steps"),
])
def test_bad_descriptor_rejected_on_host(mutate, status, needle):
    d = _desc()
    mutate(d)
    assert _call_eval(d) == status
    assert needle in abi.ks_last_error()


def test_bad_specs_heads_workspace_rejected_on_host():
    d = _desc()
    assert _call_eval(d, n_specs=0) == abi.KS_EINVAL
    assert _call_eval(d, specs=None) == abi.KS_EINVAL
    assert _call_eval(d, ws=None) == abi.KS_EWORKSPACE
    assert _call_eval(d, ws_bytes=16) == abi.KS_EWORKSPACE
    assert _call_eval(d, ws=0x100010) == abi.KS_EWORKSPACE     # misaligned
    bad_heads = [abi.ks_heads(24, 64, abi.KS_F32, abi.KS_ETA_MLP, 1, 1, 1, 1, 1),
                 abi.ks_heads(16, 256, abi.KS_F32, abi.KS_ETA_MLP, 1, 1, 1, 1, 1),
                 abi.ks_heads(16, 96, abi.KS_BF16, abi.KS_ETA_MLP, 1, 1, 1, 1, 1),
                 abi.ks_heads(16, 64, 7, abi.KS_ETA_MLP, 1, 1, 1, 1, 1),
                 abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_MLP, 1, None, 1, 1, 1),
                 abi.ks_heads(16, 64, abi.KS_F32, 5),
                 # bounded-head mask beyond the families, or without parameters
                 abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_ONE, bounded_mask=1 << 10, bounded=0x1000),
                 abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_ONE, bounded_mask=3, bounded=None),
                 # MLP mode with a family left for the MLP but no MLP weights
                 abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_MLP, bounded_mask=3, bounded=0x1000)]
    for h in bad_heads:
        assert _call_eval(d, heads=h) == abi.KS_EINVAL, abi.ks_last_error()
    # Tier B grids: each field outside its documented range
    good = dict(grid_mask=3, grid=0x1000, grid_axis=(1, 2, 6), grid_n=(4, 4, 4),
                grid_lo=(0.0, 0.0, 0.0), grid_hi=(1.0, 1.0, 1.0))
    for key, val, needle in (("grid_mask", 1 << 10, "grid_mask"), ("grid", None, "grid is NULL"),
                             ("grid_axis", (1, 15, 6), "grid_axis[1]"), ("grid_axis", (-1, 2, 6), "grid_axis[0]"),
                             ("grid_n", (4, 1, 4), "grid_n[1]"), ("grid_n", (16, 16, 16), "nodes"),
                             ("grid_hi", (1.0, 1.0, 0.0), "grid_lo/hi[2]"),
                             ("grid_lo", (float("nan"), 0.0, 0.0), "grid_lo/hi[0]"),
                             ("grid_hi", (1e39, 1.0, 1.0), "grid_lo/hi[0]"),
                             ("grid_hi", (1e-40, 1.0, 1.0), "grid_lo/hi[0]")):
        for mode in (abi.KS_ETA_ONE, abi.KS_ETA_MLP):
            kw = dict(good, **{key: val})
            h = abi.ks_heads(16, 64, abi.KS_F32, mode, 1, 1, 1, 1, 1, **kw)
            assert _call_eval(d, heads=h) == abi.KS_EINVAL, (key, val)
            assert needle in abi.ks_last_error(), (needle, abi.ks_last_error())
    assert abi.load().ks_eval_kernels(C.byref(d), 0x2000, 1, C.byref(abi.ks_heads(16, 64, 0, 1)),
                                      None, 0x100000, 1 << 30, None) == abi.KS_EINVAL


def test_eval_steps_host_checks():
    d = _desc()
    lib = abi.load()
    st = abi.ks_steps(3, 0x10, 0x10, 0x10, 0x10)      # n_steps mismatch
    h = abi.ks_heads(16, 64, abi.KS_F32, abi.KS_ETA_ONE)
    host = abi.ks_host(0, 0, 0, 0, 1)
    so = abi.ks_step_out(0x10, 0x10, 0x10)
    r = lib.ks_eval_steps(C.byref(d), C.byref(st), 0x2000, 1, C.byref(h), C.byref(host),
                          C.byref(so), None, 0x100000, 1 << 30, None)
    assert r == abi.KS_EINVAL and "n_steps" in abi.ks_last_error()
    st.n_steps = 2
    so.t_gpu = None
    r = lib.ks_eval_steps(C.byref(d), C.byref(st), 0x2000, 1, C.byref(h), C.byref(host),
                          C.byref(so), None, 0x100000, 1 << 30, None)
    assert r == abi.KS_EINVAL and "step output" in abi.ks_last_error()


def test_workspace_bytes_grows_with_specs():
    d = _desc(n_rows=1000, n_steps=10)
    a, b = abi.ks_workspace_bytes(d, 1), abi.ks_workspace_bytes(d, 64)
    assert 0 < a < b and a % 256 == 0 and b % 256 == 0
    assert abi.ks_workspace_bytes(d, 0) == 0


def test_missing_library_fails_loudly(tmp_path):
    with pytest.raises(RuntimeError, match="no fallback"):
        abi._lib, saved = None, abi._lib
        try:
            abi.load(str(tmp_path / "nope.so"))
        finally:
            abi._lib = saved


# ---- batch expansion (host side only)
def _model(**kw):
    from workload import gen
    base = dict(hidden=4096, layers=32, q_heads=32, kv_heads=8, head_dim=128, ffn=11008, vocab=32000,
                tp=1, experts=0, top_k=0, expert_ffn=0, kv_write=0)
    base.update(kw)
    return abi.ks_model(*(base[n] for n in abi.MODEL_FIELDS))


def test_expand_layout_closed_form_counts():
    """Record counts per family for a dense and an MoE model, both modes,
    against the oracle's closed form (host arithmetic only)."""
    from types import SimpleNamespace
    from oracle import ks_expand as ox
    cases = [dict(), dict(kv_write=1, tp=4), dict(experts=8, top_k=2, expert_ffn=14336, ffn=0),
             dict(kv_heads=2, tp=8, q_heads=64, ffn=28672, layers=80, hidden=8192)]
    for kw in cases:
        md = _model(**kw)
        shape = SimpleNamespace(**{n: getattr(md, n) for n in abi.MODEL_FIELDS})
        for mode in (abi.KS_EXPAND_PER_LAYER, abi.KS_EXPAND_HOMOGENEOUS):
            for S, npre in ((0, 0), (1, 1), (1000, 297), (88_640, 26_000)):
                _, fo = abi.ks_expand_layout(md, S, npre, mode)
                want = ox.family_counts(shape, S, npre, mode == abi.KS_EXPAND_HOMOGENEOUS)
                assert [fo[f + 1] - fo[f] for f in range(abi.NFAM)] == list(want), (kw, mode, S)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(tp=3), abi.KS_EINVAL, "q_heads"),
    (dict(vocab=32001, tp=2, q_heads=32), abi.KS_EINVAL, "vocab"),
    (dict(ffn=11007, tp=2), abi.KS_EINVAL, "ffn"),
    (dict(layers=0), abi.KS_EINVAL, "layers"),
    (dict(experts=2000, top_k=2, expert_ffn=64), abi.KS_ERANGE, "experts"),
    (dict(experts=8, top_k=9, expert_ffn=64), abi.KS_EINVAL, "top_k"),
    (dict(ffn=300000), abi.KS_ERANGE, "2^18"),
    (dict(head_dim=4096), abi.KS_ERANGE, "2^12"),
    (dict(kv_write=2), abi.KS_EINVAL, "kv_write"),
])
def test_expand_layout_rejects_bad_models(kw, status, needle):
    st, _ = abi.ks_expand_layout(_model(**kw), 10, 2, 0, check=False)
    assert st == status and needle in abi.ks_last_error()


def test_expand_layout_rejects_bad_counts():
    md = _model()
    assert abi.ks_expand_layout(md, 10, 11, 0, check=False)[0] == abi.KS_EINVAL
    assert abi.ks_expand_layout(md, -1, 0, 0, check=False)[0] == abi.KS_ERANGE
    assert abi.ks_expand_layout(md, 10, 2, 7, check=False)[0] == abi.KS_EINVAL
    # more records than the u32 record index allows
    assert abi.ks_expand_layout(md, 20_000_000, 0, 0, check=False)[0] == abi.KS_ERANGE
    # MoE routed-row offsets must fit u32
    moe = _model(experts=1024, top_k=2, expert_ffn=1024, ffn=0, layers=80)
    assert abi.ks_expand_layout(moe, 60_000, 0, 1, check=False)[0] == abi.KS_ERANGE
    assert abi.ks_expand_workspace_bytes(-1) == 0
    assert abi.ks_expand_workspace_bytes(5000) >= 256 + 2 * 4 * 5000


def test_expand_host_checks():
    md = _model()
    out = abi.ks_records()
    ws = C.create_string_buffer(1 << 16)
    wsp = (C.addressof(ws) + 255) & ~255
    b = abi.ks_batch(4, None, None, 0, None, 1)
    assert abi.ks_expand(md, b, 0, out, wsp, 1 << 15, None, check=False) == abi.KS_EINVAL
    assert "req_off" in abi.ks_last_error()
    b.req_off = 16
    assert abi.ks_expand(md, b, 0, out, wsp, 1 << 15, None, check=False) == abi.KS_EINVAL
    assert "prefill" in abi.ks_last_error()
    b.prefill = 16
    assert abi.ks_expand(md, b, 0, out, wsp, 1 << 15, None, check=False) == abi.KS_EINVAL
    assert "record output" in abi.ks_last_error()
    for name in ("step", "m", "n", "k", "a", "b"):
        setattr(out, name, 16)
    assert abi.ks_expand(md, b, 1, out, wsp, 1 << 15, None, check=False) == abi.KS_EINVAL
    assert "mult" in abi.ks_last_error()
    assert abi.ks_expand(md, b, 0, out, wsp, 1 << 15, None, check=False) == abi.KS_EINVAL
    assert "per-step" in abi.ks_last_error()
    for name in ("layers", "hidden", "tp", "n_launch"):
        setattr(out, name, 16)
    assert abi.ks_expand(md, b, 0, out, wsp, 8, None, check=False) == abi.KS_EWORKSPACE
    assert abi.ks_expand(md, b, 0, out, wsp + 8, 1 << 15, None, check=False) == abi.KS_EWORKSPACE
    # the record writer's index arithmetic: a family with 2^16 or more
    # records per step (20,000 layers x 4 GEMMs) is refused before any launch
    deep = _model(layers=20_000)
    assert abi.ks_expand(deep, b, 0, out, wsp, 1 << 15, None, check=False) == abi.KS_ERANGE
    assert "limits" in abi.ks_last_error()


# ---- serving simulation (host side only)
def _sched(**kw):
    base = dict(max_num_seqs=64, max_batched_tokens=4096, block_tokens=16, prefix_cache=1, kv_blocks=4096)
    base.update(kw)
    return abi.ks_sched(*(base[n] for n, _ in abi.ks_sched._fields_))


@pytest.mark.parametrize("kw,needle", [
    (dict(max_num_seqs=0), "max_num_seqs"),
    (dict(max_batched_tokens=1 << 24), "max_batched_tokens"),
    (dict(block_tokens=0), "block_tokens"),
    (dict(prefix_cache=2), "prefix_cache"),
    (dict(kv_blocks=0), "kv_blocks"),
])
def test_simulate_rejects_bad_schedulers(kw, needle):
    assert abi.ks_simulate_workspace_bytes(_model(), _sched(**kw)) == 0
    assert needle in abi.ks_last_error()


def test_simulate_workspace_and_model_checks():
    assert abi.ks_simulate_workspace_bytes(_model(), _sched()) > 0
    # the workspace grows with the number of simulations run in lockstep
    one, many = (abi.ks_simulate_workspace_bytes(_model(), _sched(), s) for s in (1, 8))
    assert many > one
    for bad in (0, 257):
        assert abi.ks_simulate_workspace_bytes(_model(), _sched(), bad) == 0
        assert "n_specs" in abi.ks_last_error()
    assert abi.ks_simulate_workspace_bytes(_model(experts=8, top_k=2, expert_ffn=1024, ffn=0), _sched()) == 0
    assert "dense" in abi.ks_last_error()


def _sim_call(arrival, prompt, output, ws_bytes=1 << 22, group=None, prefix=None):
    import numpy as np
    arr = {"a": np.ascontiguousarray(arrival, np.float64), "p": np.ascontiguousarray(prompt, np.uint32),
           "o": np.ascontiguousarray(output, np.uint32)}
    g = np.ascontiguousarray(group, np.uint32) if group is not None else None
    x = np.ascontiguousarray(prefix, np.uint32) if prefix is not None else None
    rq = abi.ks_requests(len(arrival), arr["a"].ctypes.data, arr["p"].ctypes.data, arr["o"].ctypes.data,
                         g.ctypes.data if g is not None else None, x.ctypes.data if x is not None else None)
    out = abi.ks_sim_out()
    ws = C.create_string_buffer(ws_bytes + 256)
    wsp = (C.addressof(ws) + 255) & ~255
    st = abi.ks_simulate(_model(), 16, 1, abi.ks_heads(), abi.ks_host(), _sched(), rq, out, wsp, ws_bytes,
                         None, check=False)
    return st, abi.ks_last_error()


def test_simulate_rejects_bad_requests_on_host():
    # every case fails before any device call (the spec pointer is a dummy)
    assert _sim_call([1.0, 0.5], [10, 10], [2, 2]) == (abi.KS_EINVAL, _sim_call([1.0, 0.5], [10, 10], [2, 2])[1])
    assert "non-decreasing" in _sim_call([1.0, 0.5], [10, 10], [2, 2])[1]
    assert _sim_call([0.0], [0], [2])[0] == abi.KS_ERANGE
    assert _sim_call([0.0], [5], [0])[0] == abi.KS_ERANGE
    assert _sim_call([0.0], [5], [2], group=[1], prefix=[9])[0] == abi.KS_EINVAL
    assert _sim_call([0.0], [5], [2], group=[1])[0] == abi.KS_EINVAL
    assert _sim_call([0.0], [5], [2], ws_bytes=64)[0] == abi.KS_EWORKSPACE
