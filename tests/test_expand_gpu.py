"""Parity of the batch expansion (ks_expand, through the C ABI) with the
oracle's enumeration of the kernels each step dispatches, and of the step
terms evaluated on its records.

Records are integers: bit-exact.  Step terms on the expanded records: the
same tolerances as on any record set (1e-5 relative with eta = 1 and fp32
heads); the homogeneous form (multiplicity L) against one record per
dispatch: 1e-5 relative (fp32 step sums of m t instead of m separate t)."""
import numpy as np
import pytest
import torch

from oracle import ks_expand as ox
from oracle import ks_oracle as o
from workload import gen
from tests import gpu_helpers as g
from tests.test_oracle_expand import load_fixture
from paper_2606_28565_amd import abi

pytestmark = pytest.mark.gpu

FIELDS = ("step", "m", "n", "k", "a", "b")


def _u32(t):
    return t.cpu().numpy().view(np.uint32).astype(np.int64)


def run_expand(tr, mode=abi.KS_EXPAND_PER_LAYER, n_prefill=None, check=True):
    db = abi.DeviceBatch(tr, mode)
    if n_prefill is not None:
        db.batch.n_prefill = n_prefill
    torch.cuda.synchronize()
    st = db.expand(abi.current_stream(), check)
    torch.cuda.synchronize()
    return db, st


def check_against_oracle(tr, homogeneous):
    mode = abi.KS_EXPAND_HOMOGENEOUS if homogeneous else abi.KS_EXPAND_PER_LAYER
    db, _ = run_expand(tr, mode)
    abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream())
    ref = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill, homogeneous=homogeneous)
    assert list(db.fam_off) == list(ref["fam_off"])
    for f in FIELDS:
        np.testing.assert_array_equal(_u32(db.t[f]), ref[f], err_msg=f)
    if homogeneous:
        np.testing.assert_array_equal(_u32(db.t["mult"]), ref["mult"])
    for f in ("layers", "hidden", "tp", "n_launch"):
        np.testing.assert_array_equal(_u32(db.t["s_" + f]), ref[f], err_msg=f)
    return db, ref


def _cases():
    cases = [("c1", gen.trace_c1().slice(0, 160))]
    for i in range(6):
        cases.append((f"c2-{i}", gen.trace_c2(i).slice(0, 10)))
    tr3 = gen.trace_c3().slice(0, 24)
    tr3.experts = gen.route_tokens(gen.trace_c3(), gen.SEED + 3, 0, 24)
    cases.append(("c3", tr3))
    cases.append(("c5", gen.trace_c5().slice(0, 12)))
    cases.append(("kvw", gen.trace_uniform(gen.ModelShape("kvw", 2048, 5, 16, 4, 128, 5632, tp=2,
                                                             kv_write=True), 40, 7, bmax=8)))
    cases.append(("kvrep", gen.trace_uniform(gen.ModelShape("kvrep", 2048, 3, 16, 2, 128, 5632, tp=4,
                                                               kv_write=True), 30, 8, bmax=8)))
    # several 1024-step blocks of the prefill rank scan, ragged tail
    one = gen.ModelShape("one-layer", 512, 1, 8, 8, 64, 1024)
    cases.append(("blocks", gen.trace_uniform(one, 2 * 1024 + 317, 9, bmax=3, p_prefill=0.5)))
    return cases


CASES = _cases()


@pytest.mark.parametrize("homog", [False, True], ids=["per-layer", "homogeneous"])
@pytest.mark.parametrize("name,tr", CASES, ids=[c[0] for c in CASES])
def test_expand_matches_oracle(name, tr, homog):
    check_against_oracle(tr, homog)


class _Tr:
    """A hand-made batch in the trace interface ks_expand's binding reads."""

    def __init__(self, shape, reqs, prefill, experts=None):
        self.shape = shape
        self.req_off = np.cumsum([0] + [len(r) for r in reqs]).astype(np.int64)
        self.req_q = np.array([q for r in reqs for q, _ in r], np.int64)
        self.req_h = np.array([h for r in reqs for _, h in r], np.int64)
        self.prefill = np.asarray(prefill, bool)
        self.experts = experts

    @property
    def n_steps(self):
        return len(self.prefill)


@pytest.mark.parametrize("name", ["expand_tiny_dense.txt", "expand_tiny_moe_homogeneous.txt"])
def test_expand_hand_derived(name):
    model, req_off, req_q, req_h, prefill, homog, recs, n_launch = load_fixture(name)
    reqs = [list(zip(req_q[req_off[j]:req_off[j + 1]], req_h[req_off[j]:req_off[j + 1]]))
            for j in range(len(prefill))]
    tr = _Tr(model, reqs, prefill)
    db, _ = run_expand(tr, abi.KS_EXPAND_HOMOGENEOUS if homog else abi.KS_EXPAND_PER_LAYER)
    abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream())
    fam = np.repeat(np.arange(gen.NFAM), np.diff(db.fam_off))
    mult = _u32(db.t["mult"]) if homog else np.ones(len(fam), np.int64)
    got = [(int(fam[i]),) + tuple(int(_u32(db.t[f])[i]) for f in FIELDS) + (int(mult[i]),)
           for i in range(len(fam))]
    assert got == recs
    assert list(_u32(db.t["s_n_launch"])) == n_launch


@pytest.mark.parametrize("prefill", [[1] * 37, [0] * 37, [0] * 1024 + [1], [1] + [0] * 1500])
def test_expand_all_or_no_prefill_and_block_edges(prefill):
    shape = gen.ModelShape("s", 256, 2, 4, 2, 64, 512)
    reqs = [[(1 + (j % 5), 10 + j)] * (1 + j % 3) for j in range(len(prefill))]
    check_against_oracle(_Tr(shape, reqs, prefill), False)


# A batch of at most 1024 steps (one block of the prefill rank scan) and at
# most 64 chunks of 256 items takes the one-workgroup expansion: 1024 steps
# of a one-layer model (about 45 chunks) sit on its edge; 1025 steps, or the
# same steps of a two-layer model (about 80 chunks), take the multi-kernel
# path.
@pytest.mark.parametrize("layers,n_steps", [(1, 1024), (1, 1025), (2, 1024)])
def test_expand_one_workgroup_path_edges(layers, n_steps):
    shape = gen.ModelShape("edge", 256, layers, 4, 2, 64, 512)
    prefill = [(j % 7) == 3 for j in range(n_steps)]
    reqs = [[(1 + (j % 5), 10 + j)] * (1 + j % 3) for j in range(n_steps)]
    check_against_oracle(_Tr(shape, reqs, prefill), False)
    check_against_oracle(_Tr(shape, reqs, prefill), True)


def test_expand_empty_steps_and_empty_batch():
    shape = gen.ModelShape("s", 256, 2, 4, 2, 64, 512)
    # steps without requests still dispatch their kernels over 0 tokens
    tr = _Tr(shape, [[], [(3, 4)], [], []], [0, 1, 0, 0])
    db, ref = check_against_oracle(tr, False)
    assert (_u32(db.t["m"])[ref["step"] != 1] == 0).all()
    db, _ = run_expand(_Tr(shape, [], []))
    assert db.fam_off[-1] == 0


def test_expand_wrong_prefill_count_is_flagged():
    tr = gen.trace_c1().slice(0, 50)
    n = int(tr.prefill.sum())
    for wrong in (n - 1, n + 1):
        db, _ = run_expand(tr, n_prefill=wrong)
        st = abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream(), check=False)
        assert st == abi.KS_EINVAL and "prefill" in abi.ks_last_error()
    # the flag clears on the next good call
    db, _ = run_expand(tr)
    abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream())


def test_expand_bad_request_offsets_are_flagged():
    shape = gen.ModelShape("s", 256, 2, 4, 2, 64, 512)
    tr = _Tr(shape, [[(3, 4)], [(1, 2)]], [1, 0])
    tr.req_off = np.array([0, 5, 2], np.int64)     # out of order and beyond n_req
    db, _ = run_expand(tr)
    st = abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream(), check=False)
    assert st == abi.KS_EINVAL and "request" in abi.ks_last_error()


def test_expand_token_limit_is_flagged():
    moe = gen.ModelShape("m", 256, 2, 4, 2, 64, 0, experts=4, top_k=2, expert_ffn=256)
    # top_k T = 2 * 2^23 reaches the 2^24 limit of a record's m
    tr = _Tr(moe, [[(1 << 23, 0)]], [1], experts=np.zeros((1, 2, 4), np.int64))
    db, _ = run_expand(tr)
    st = abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream(), check=False)
    assert st == abi.KS_ERANGE and "limits" in abi.ks_last_error()


def _eval_on(db, wl_specs, heads_wl, eta_one):
    di_specs = torch.from_numpy(abi.pack_specs(wl_specs).view(np.uint8).copy()).cuda()
    n_specs = len(wl_specs["peak_flops"])
    hd = abi.ks_heads()
    heads_t = {}
    if not eta_one:
        h = heads_wl
        hd.in_dim, hd.hidden = h.in_dim, h.hidden
        hd.precision = abi.KS_BF16 if h.precision == "bf16" else abi.KS_F32
        for name in ("w1", "w2", "b2", "w3", "b3"):
            arr = np.ascontiguousarray(h.storage[name])
            arr = arr.view(np.int16) if arr.dtype == np.uint16 else arr
            heads_t[name] = torch.from_numpy(arr.reshape(-1).copy()).cuda()
            setattr(hd, name, heads_t[name].data_ptr())
    hd.mode = abi.KS_ETA_ONE if eta_one else abi.KS_ETA_MLP
    hc = gen.HostConsts()
    host = abi.ks_host(hc.c_disp, hc.ell, hc.c_ovl, hc.c_tail, hc.body_scale)
    S = db.desc.n_steps
    so_t, so = abi.step_outputs(S, n_specs)
    wsb = abi.ks_workspace_bytes(db.desc, n_specs)
    ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
    wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
    abi.ks_eval_steps(db.desc, db.steps, di_specs.data_ptr(), n_specs, hd, host, so, None, wsp, wsb,
                      abi.current_stream())
    torch.cuda.synchronize()
    abi.ks_device_status(wsp, wsb, abi.current_stream())
    return {k: v.cpu().numpy() for k, v in so_t.items()}


@pytest.mark.parametrize("case", ["c1", "c3", "kvw"])
@pytest.mark.parametrize("eta_one", [True, False], ids=["eta1", "fp32-mlp"])
def test_steps_on_expanded_records(case, eta_one):
    """ks_expand -> ks_eval_steps in both forms against the oracle's step
    terms on its own expansion (one record per dispatch)."""
    tr = dict(CASES)[case]
    heads = gen.make_heads(16, 64, "f32")
    specs = gen.specs_datasheet()
    full = ox.expand(tr.shape, tr.req_off, tr.req_q, tr.prefill)
    u = lambda x: np.asarray(x, np.uint32)
    experts = u(tr.experts.reshape(-1)) if tr.experts is not None else u([])
    desc = gen.Desc(full["fam_off"], *(u(full[f]) for f in FIELDS), u(tr.req_off), u(tr.req_q),
                    u(tr.req_h), experts, 2)
    rec = gen.StepRec(*(u(full[f]) for f in ("layers", "hidden", "tp", "n_launch")))
    ref = o.eval_steps(desc, rec, specs, gen.HostConsts(), None if eta_one else heads, eta_one)
    for mode in (abi.KS_EXPAND_PER_LAYER, abi.KS_EXPAND_HOMOGENEOUS):
        db, _ = run_expand(tr, mode)
        got = _eval_on(db, specs, heads, eta_one)
        for key in ("t_body", "t_gpu", "t_step"):
            err = g.rel_err(got[key], ref[key]).max()
            assert err <= 1e-5, (mode, key, err)


def test_full_size_batch_sampled():
    """The 70B prefix-cache workload's 64M-record batch (88,640 steps):
    the expansion equals the record builder's layout bit for bit, and
    sampled steps equal the oracle's kernel list at their positions."""
    S = 88_640
    tr = gen.trace_c5().slice(0, S)
    db, _ = run_expand(tr)
    abi.ks_device_status(db.ws_ptr, db.ws_bytes, abi.current_stream())
    desc, rec = gen.build([tr])
    assert list(db.fam_off) == list(desc.fam_off)
    for f in FIELDS:
        want = torch.from_numpy(getattr(desc, f).view(np.int32)).cuda()
        assert torch.equal(db.t[f], want), f
    pos_pre = np.cumsum(np.concatenate([[0], tr.prefill.astype(np.int64)]))
    fo = db.fam_off
    L = tr.shape.layers
    per = {gen.GEMM: 4 * L, gen.LM_HEAD: 1, gen.RMSNORM: 2 * L, gen.ROPE: L, gen.SILU_MUL: L, gen.EMBED: 1}
    rng = np.random.Generator(np.random.PCG64(11))
    idx, want = [], []
    for j in sorted(rng.choice(S, 24, replace=False)) + [0, S - 1]:
        T = int(tr.req_q[tr.req_off[j]:tr.req_off[j + 1]].sum())
        R = int(tr.req_off[j + 1] - tr.req_off[j])
        ks = ox.step_kernels(tr.shape, int(j), T, R, bool(tr.prefill[j]))
        seen = {}
        for (f, layer, m, n, k, a, b) in ks:
            q = seen.get(f, 0)
            seen[f] = q + 1
            if f in (gen.ATTN_PREFILL, gen.ATTN_DECODE):
                rank = pos_pre[j] if f == gen.ATTN_PREFILL else j - pos_pre[j]
                i = fo[f] + rank * L + q
            else:
                i = fo[f] + j * per[f] + q
            idx.append(int(i))
            want.append((int(j), m, n, k, a, b))
    sel = torch.tensor(idx, dtype=torch.int64, device="cuda")
    got = np.stack([_u32(db.t[f][sel]) for f in FIELDS], axis=1)
    np.testing.assert_array_equal(got, np.array(want, np.int64))


@pytest.mark.parametrize("variant", ["bf16", "bf16-grid", "bounded"])
def test_homogeneous_matches_per_layer_on_gpu(variant):
    """Both forms price the same kernels with the same per-record latency;
    the step sums differ only in fp32 summation order (m t once against t
    added m times), for the MFMA head, the grid-routed variant and the
    bounded head alike."""
    tr = gen.trace_c1().slice(0, 120)
    wl = gen.config1(0, 120).with_heads(gen.make_heads(16, 128, "bf16"))
    bounded = gen.make_bounded(gen.BOUNDED_MIXED) if variant == "bounded" else None
    grid = gen.make_grid(gen.GRID_ALL) if variant == "bf16-grid" else None
    res = {}
    for mode in (abi.KS_EXPAND_PER_LAYER, abi.KS_EXPAND_HOMOGENEOUS):
        db, _ = run_expand(tr, mode)
        di = abi.DeviceInputs(wl)
        heads = di.make_heads("bf16", 16, 128, abi.KS_ETA_MLP, bounded, grid)
        so_t, so = abi.step_outputs(db.desc.n_steps, di.n_specs)
        wsb = abi.ks_workspace_bytes(db.desc, di.n_specs)
        ws = torch.empty(wsb + 256, dtype=torch.uint8, device="cuda")
        wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
        abi.ks_eval_steps(db.desc, db.steps, di.specs_ptr, di.n_specs, heads, di.host, so, None, wsp, wsb,
                          abi.current_stream())
        torch.cuda.synchronize()
        abi.ks_device_status(wsp, wsb, abi.current_stream())
        res[mode] = {k: v.cpu().numpy() for k, v in so_t.items()}
    for key in ("t_body", "t_gpu", "t_step"):
        err = g.rel_err(res[abi.KS_EXPAND_HOMOGENEOUS][key], res[abi.KS_EXPAND_PER_LAYER][key]).max()
        assert err <= 1e-5, (key, err)
