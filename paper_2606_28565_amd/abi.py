"""ctypes binding of the C ABI in include/ks.h (libks.so).

Argument marshalling only: every stage of the evaluation runs in the HIP
kernels of libks.so.  torch owns the device memory and supplies the stream.
There is no fallback: if the library is missing or fails to load, the
import of the entry points raises."""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libks.so")

NFAM = 10
KS_OK, KS_EINVAL, KS_ERANGE, KS_EHIP, KS_EWORKSPACE = range(5)
KS_F32, KS_BF16 = 0, 1
KS_ETA_MLP, KS_ETA_ONE = 0, 1
KS_STATIC_SCRATCH_BYTES = 64 << 20   # the allocation-free entry point's device array
STATUS_NAMES = {0: "KS_OK", 1: "KS_EINVAL", 2: "KS_ERANGE", 3: "KS_EHIP", 4: "KS_EWORKSPACE"}

P = C.c_void_p


class ks_desc(C.Structure):
    _fields_ = [("n_rows", C.c_int64), ("fam_off", C.c_int64 * (NFAM + 1)),
                ("step", P), ("m", P), ("n", P), ("k", P), ("a", P), ("b", P),
                ("n_steps", C.c_int64), ("req_off", P), ("req_q", P), ("req_h", P),
                ("n_req", C.c_int64), ("expert_rows", P), ("n_expert_rows", C.c_int64),
                ("elem_bytes", C.c_uint32), ("reserved", C.c_uint32), ("mult", P)]


class ks_spec(C.Structure):
    _fields_ = [("peak_flops", C.c_double), ("hbm_bw", C.c_double), ("t0", C.c_double),
                ("l2_bytes", C.c_double), ("ar_alpha0", C.c_double),
                ("ar_alpha_log2p", C.c_double), ("ar_beta", C.c_double),
                ("n_cu", C.c_uint32), ("reserved", C.c_uint32)]


class ks_heads(C.Structure):
    _fields_ = [("in_dim", C.c_int32), ("hidden", C.c_int32), ("precision", C.c_int32),
                ("mode", C.c_int32), ("w1", P), ("w2", P), ("b2", P), ("w3", P), ("b3", P),
                ("bounded_mask", C.c_uint32), ("grid_mask", C.c_uint32), ("bounded", P),
                ("grid_axis", C.c_int32 * 3), ("grid_n", C.c_int32 * 3),
                ("grid_lo", C.c_double * 3), ("grid_hi", C.c_double * 3), ("grid", P)]


class ks_steps(C.Structure):
    _fields_ = [("n_steps", C.c_int64), ("layers", P), ("hidden", P), ("tp", P), ("n_launch", P)]


class ks_host(C.Structure):
    _fields_ = [("c_disp", C.c_double), ("ell", C.c_double), ("c_ovl", C.c_double),
                ("c_tail", C.c_double), ("body_scale", C.c_double)]


class ks_kernel_out(C.Structure):
    _fields_ = [("flops", P), ("bytes", P), ("blocks", P),
                ("t_roof", P), ("eta", P), ("t_kernel", P), ("source", P)]


class ks_step_out(C.Structure):
    _fields_ = [("t_body", P), ("t_gpu", P), ("t_step", P)]


MODEL_FIELDS = ("hidden", "layers", "q_heads", "kv_heads", "head_dim", "ffn", "vocab", "tp",
                "experts", "top_k", "expert_ffn", "kv_write")


class ks_model(C.Structure):
    _fields_ = [(name, C.c_uint32) for name in MODEL_FIELDS]


class ks_batch(C.Structure):
    _fields_ = [("n_steps", C.c_int64), ("req_off", P), ("req_q", P), ("n_req", C.c_int64),
                ("prefill", P), ("n_prefill", C.c_int64)]


class ks_records(C.Structure):
    _fields_ = [(name, P) for name in ("step", "m", "n", "k", "a", "b", "mult",
                                       "layers", "hidden", "tp", "n_launch")]


KS_EXPAND_PER_LAYER, KS_EXPAND_HOMOGENEOUS = 0, 1


class ks_sched(C.Structure):
    _fields_ = [("max_num_seqs", C.c_int32), ("max_batched_tokens", C.c_int32),
                ("block_tokens", C.c_int32), ("prefix_cache", C.c_int32), ("kv_blocks", C.c_int64)]


class ks_requests(C.Structure):
    _fields_ = [("n", C.c_int64), ("arrival", P), ("prompt", P), ("output", P), ("group", P),
                ("prefix", P)]


class ks_sim_out(C.Structure):
    _fields_ = [("ttft", P), ("tpot", P), ("e2e", P), ("state", P), ("step_cap", C.c_int64),
                ("entry_cap", C.c_int64), ("step_start", P), ("step_latency", P), ("step_prefill", P),
                ("step_entry_off", P), ("entry_req", P), ("entry_q", P), ("entry_h", P),
                ("n_steps", C.c_int64), ("n_entries", C.c_int64), ("preemptions", C.c_int64),
                ("clock", C.c_double)]


assert C.sizeof(ks_spec) == 64


class KsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load libks.so (built by ``paper_2606_28565_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2606_28565_amd.build` (there is no fallback)")
    lib = C.CDLL(path)
    pd, pst, psp, ph, phost, pko, pso = (C.POINTER(ks_desc), C.POINTER(ks_steps),
                                          P, C.POINTER(ks_heads), C.POINTER(ks_host),
                                          C.POINTER(ks_kernel_out), C.POINTER(ks_step_out))
    lib.ks_workspace_bytes.argtypes = [pd, C.c_int32]
    lib.ks_workspace_bytes.restype = C.c_size_t
    lib.ks_eval_kernels.argtypes = [pd, psp, C.c_int32, ph, pko, P, C.c_size_t, P]
    lib.ks_eval_kernels.restype = C.c_int
    lib.ks_eval_steps.argtypes = [pd, pst, psp, C.c_int32, ph, phost, pso, pko, P, C.c_size_t, P]
    lib.ks_eval_steps.restype = C.c_int
    lib.ks_eval_steps_static.argtypes = [pd, pst, psp, C.c_int32, ph, phost, pso, pko, P, P]
    lib.ks_eval_steps_static.restype = C.c_int
    lib.ks_validate.argtypes = [pd, pst, psp, C.c_int32, P, C.c_size_t, P]
    lib.ks_validate.restype = C.c_int
    lib.ks_device_status.argtypes = [P, C.c_size_t, P]
    lib.ks_device_status.restype = C.c_int
    lib.ks_expand_layout.argtypes = [C.POINTER(ks_model), C.c_int64, C.c_int64, C.c_int32,
                                     C.POINTER(C.c_int64)]
    lib.ks_expand_layout.restype = C.c_int
    lib.ks_expand_workspace_bytes.argtypes = [C.c_int64]
    lib.ks_expand_workspace_bytes.restype = C.c_size_t
    lib.ks_expand.argtypes = [C.POINTER(ks_model), C.POINTER(ks_batch), C.c_int32,
                              C.POINTER(ks_records), P, C.c_size_t, P]
    lib.ks_expand.restype = C.c_int
    lib.ks_simulate_workspace_bytes.argtypes = [C.POINTER(ks_model), C.POINTER(ks_sched), C.c_int32]
    lib.ks_simulate_workspace_bytes.restype = C.c_size_t
    lib.ks_simulate.argtypes = [C.POINTER(ks_model), P, C.c_int32, C.POINTER(ks_heads), C.POINTER(ks_host),
                                C.POINTER(ks_sched), C.POINTER(ks_requests), C.POINTER(ks_sim_out), P,
                                C.c_size_t, P]
    lib.ks_simulate.restype = C.c_int
    lib.ks_set_timing_events.argtypes = [P, P]
    lib.ks_set_timing_events.restype = C.c_int
    lib.ks_last_error.argtypes = []
    lib.ks_last_error.restype = C.c_char_p
    lib.ks_version.argtypes = []
    lib.ks_version.restype = C.c_char_p
    _lib = lib
    return lib


def _check(st: int) -> int:
    if st != KS_OK:
        raise KsError(st, load().ks_last_error().decode())
    return st


# --------------------------------------------------------------------------
# the entry points, same names as the C ABI; arguments are ctypes structs
# and raw device addresses
# --------------------------------------------------------------------------
def ks_workspace_bytes(desc: ks_desc, n_specs: int) -> int:
    return load().ks_workspace_bytes(C.byref(desc), n_specs)


def ks_eval_kernels(desc, specs_ptr, n_specs, heads, out, ws_ptr, ws_bytes, stream, check=True):
    st = load().ks_eval_kernels(C.byref(desc), specs_ptr, n_specs, C.byref(heads), C.byref(out),
                                ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_eval_steps(desc, steps, specs_ptr, n_specs, heads, host, out, kout, ws_ptr, ws_bytes,
                  stream, check=True):
    st = load().ks_eval_steps(C.byref(desc), C.byref(steps), specs_ptr, n_specs, C.byref(heads),
                              C.byref(host), C.byref(out),
                              C.byref(kout) if kout is not None else None,
                              ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_eval_steps_static(desc, steps, specs_ptr, n_specs, heads, host, out, kout, flags_ptr, stream,
                         check=True):
    st = load().ks_eval_steps_static(C.byref(desc), C.byref(steps), specs_ptr, n_specs, C.byref(heads),
                                     C.byref(host), C.byref(out),
                                     C.byref(kout) if kout is not None else None, flags_ptr, stream)
    return _check(st) if check else st


def ks_validate(desc, steps, specs_ptr, n_specs, ws_ptr, ws_bytes, stream, check=True):
    st = load().ks_validate(C.byref(desc), C.byref(steps) if steps is not None else None,
                            specs_ptr, n_specs, ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_device_status(ws_ptr, ws_bytes, stream, check=True):
    st = load().ks_device_status(ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_expand_layout(model: ks_model, n_steps: int, n_prefill: int, mode: int, check=True):
    """Returns (status, fam_off as a list of NFAM + 1 ints)."""
    arr = (C.c_int64 * (NFAM + 1))()
    st = load().ks_expand_layout(C.byref(model), n_steps, n_prefill, mode, arr)
    if check:
        _check(st)
    return st, list(arr)


def ks_expand_workspace_bytes(n_steps: int) -> int:
    return load().ks_expand_workspace_bytes(n_steps)


def ks_expand(model, batch, mode, out, ws_ptr, ws_bytes, stream, check=True):
    st = load().ks_expand(C.byref(model), C.byref(batch), mode, C.byref(out), ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_simulate_workspace_bytes(model: ks_model, sched: ks_sched, n_specs: int = 1) -> int:
    return load().ks_simulate_workspace_bytes(C.byref(model), C.byref(sched), n_specs)


def ks_simulate(model, specs_ptr, n_specs, heads, host, sched, requests, outs, ws_ptr, ws_bytes, stream,
                check=True):
    """outs: a ks_sim_out, or a ctypes array of n_specs of them."""
    st = load().ks_simulate(C.byref(model), specs_ptr, n_specs, C.byref(heads), C.byref(host), C.byref(sched),
                            C.byref(requests), outs if isinstance(outs, C.Array) else C.byref(outs),
                            ws_ptr, ws_bytes, stream)
    return _check(st) if check else st


def ks_set_timing_events(before, after, check=True):
    """before, after: raw hipEvent_t handles (see HipEvents), or None."""
    st = load().ks_set_timing_events(before, after)
    return _check(st) if check else st


class HipEvents:
    """A pool of timing-enabled HIP events, created and read through the HIP
    runtime directly (for ks_set_timing_events)."""

    def __init__(self, n: int):
        import torch  # noqa: F401  (initialises the runtime)
        self.rt = C.CDLL("libamdhip64.so")
        self.rt.hipEventCreate.argtypes = [C.POINTER(C.c_void_p)]
        self.rt.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.rt.hipEventDestroy.argtypes = [C.c_void_p]
        self.ev = []
        for _ in range(n):
            h = C.c_void_p()
            if self.rt.hipEventCreate(C.byref(h)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev.append(h.value)

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = C.c_float()
        if self.rt.hipEventElapsedTime(C.byref(ms), self.ev[a], self.ev[b]) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for h in self.ev:
            self.rt.hipEventDestroy(h)
        self.ev = []


def ks_last_error() -> str:
    return load().ks_last_error().decode()


def ks_version() -> str:
    return load().ks_version().decode()


# --------------------------------------------------------------------------
# marshalling helpers: host arrays -> torch device tensors -> ctypes structs
# --------------------------------------------------------------------------
SPEC_DTYPE = np.dtype([("peak_flops", "<f8"), ("hbm_bw", "<f8"), ("t0", "<f8"),
                       ("l2_bytes", "<f8"), ("ar_alpha0", "<f8"), ("ar_alpha_log2p", "<f8"),
                       ("ar_beta", "<f8"), ("n_cu", "<u4"), ("reserved", "<u4")])
assert SPEC_DTYPE.itemsize == 64


def pack_specs(specs: dict) -> np.ndarray:
    """Spec vectors (dict of equal-length arrays) -> ks_spec records."""
    n = len(specs["peak_flops"])
    rec = np.zeros(n, SPEC_DTYPE)
    for name in SPEC_DTYPE.names:
        if name != "reserved":
            rec[name] = specs[name]
    return rec


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


class DeviceInputs:
    """The inputs of one evaluation, resident in device memory (torch
    tensors), and the ctypes structs that point at them."""

    def __init__(self, wl, device="cuda", n_specs: int | None = None):
        import torch
        dev = torch.device(device)

        def u32(x):
            return torch.from_numpy(np.ascontiguousarray(x, np.uint32).view(np.int32)).to(dev)

        d = wl.desc
        self.t = {name: u32(getattr(d, name)) for name in
                  ("step", "m", "n", "k", "a", "b", "req_off", "req_q", "req_h", "expert_rows")}
        sr = wl.steps
        for name in ("layers", "hidden", "tp", "n_launch"):
            self.t["s_" + name] = u32(getattr(sr, name))
        rec = pack_specs(wl.specs)
        if n_specs is not None:
            rec = rec[:n_specs]
        self.n_specs = len(rec)
        self.t["specs"] = torch.from_numpy(rec.view(np.uint8).copy()).to(dev)
        h = wl.heads
        self.heads_t = {}
        for name in ("w1", "w2", "b2", "w3", "b3"):
            arr = np.ascontiguousarray(h.storage[name])
            if arr.dtype == np.uint16:
                arr = arr.view(np.int16)
            self.heads_t[name] = torch.from_numpy(arr.reshape(-1).copy()).to(dev)

        self.desc = ks_desc()
        self.desc.n_rows = d.n_rows
        for f in range(NFAM + 1):
            self.desc.fam_off[f] = int(d.fam_off[f])
        for name in ("step", "m", "n", "k", "a", "b", "req_off", "req_q", "req_h"):
            setattr(self.desc, name, _ptr(self.t[name]) if self.t[name].numel() else None)
        self.desc.n_steps = d.n_steps
        self.desc.n_req = len(d.req_q)
        self.desc.expert_rows = _ptr(self.t["expert_rows"]) if len(d.expert_rows) else None
        self.desc.n_expert_rows = len(d.expert_rows)
        self.desc.elem_bytes = d.elem_bytes
        if getattr(d, "mult", None) is not None:
            self.t["mult"] = u32(d.mult)
            self.desc.mult = _ptr(self.t["mult"]) if self.t["mult"].numel() else None

        self.steps = ks_steps()
        self.steps.n_steps = d.n_steps
        for name in ("layers", "hidden", "tp", "n_launch"):
            t = self.t["s_" + name]
            setattr(self.steps, name, _ptr(t) if t.numel() else None)

        self.heads = self.make_heads(h.precision, h.in_dim, h.hidden, KS_ETA_MLP)
        hc = wl.host
        self.host = ks_host(hc.c_disp, hc.ell, hc.c_ovl, hc.c_tail, hc.body_scale)
        self.ws_bytes = ks_workspace_bytes(self.desc, self.n_specs)
        if self.ws_bytes == 0:
            raise KsError(KS_EINVAL, ks_last_error() or "bad descriptor")
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
        off = (-self.ws.data_ptr()) % 256
        self.ws_ptr = self.ws.data_ptr() + off

    def make_heads(self, precision, in_dim, hidden, mode, bounded=None, grid=None) -> ks_heads:
        """bounded: a ``workload.gen.Bounded`` (its mask and parameters), or
        None for no bounded-head family.  grid: a ``workload.gen.Grid``
        (Tier B measured grids), or None."""
        hd = ks_heads()
        hd.in_dim, hd.hidden = in_dim, hidden
        hd.precision = KS_BF16 if precision == "bf16" else KS_F32
        hd.mode = mode
        for name in ("w1", "w2", "b2", "w3", "b3"):
            setattr(hd, name, _ptr(self.heads_t[name]))
        if bounded is not None and bounded.mask:
            import torch
            self.t["bounded"] = torch.from_numpy(np.ascontiguousarray(bounded.storage, np.float32)
                                                 .reshape(-1).copy()).to(self.t["step"].device)
            hd.bounded_mask = bounded.mask
            hd.bounded = _ptr(self.t["bounded"])
        if grid is not None and grid.mask:
            import torch
            self.t["grid"] = torch.from_numpy(np.ascontiguousarray(grid.values, np.float32)
                                              .reshape(-1).copy()).to(self.t["step"].device)
            hd.grid_mask = grid.mask
            hd.grid = _ptr(self.t["grid"])
            for d in range(3):
                hd.grid_axis[d] = int(grid.axes[d])
                hd.grid_n[d] = int(grid.n[d])
                hd.grid_lo[d] = float(grid.lo[d])
                hd.grid_hi[d] = float(grid.hi[d])
        return hd

    @property
    def specs_ptr(self) -> int:
        return self.t["specs"].data_ptr()


def kernel_outputs(n_rows: int, n_specs: int, device="cuda", counts=True, t_roof=True,
                   eta=True, t_kernel=True, source=False):
    """Allocate per-record / per-pair output tensors and the struct."""
    import torch
    dev = torch.device(device)
    o = {}
    if counts:
        for name in ("flops", "bytes", "blocks"):
            o[name] = torch.empty(n_rows, dtype=torch.int64, device=dev)
    for name, want in (("t_roof", t_roof), ("eta", eta), ("t_kernel", t_kernel)):
        if want:
            o[name] = torch.empty((n_specs, n_rows), dtype=torch.float32, device=dev)
    if source:
        o["source"] = torch.empty((n_specs, n_rows), dtype=torch.uint8, device=dev)
    s = ks_kernel_out()
    for name in ("flops", "bytes", "blocks", "t_roof", "eta", "t_kernel", "source"):
        setattr(s, name, _ptr(o.get(name)) if name in o and o[name].numel() else None)
    return o, s


def step_outputs(n_steps: int, n_specs: int, device="cuda"):
    import torch
    dev = torch.device(device)
    o = {name: torch.empty((n_specs, n_steps), dtype=torch.float64, device=dev)
         for name in ("t_body", "t_gpu", "t_step")}
    s = ks_step_out(*(_ptr(o[n]) for n in ("t_body", "t_gpu", "t_step")))
    return o, s


def current_stream() -> int:
    import torch
    return torch.cuda.current_stream().cuda_stream


# --------------------------------------------------------------------------
# batch expansion: batch descriptors on the device -> records on the device
# --------------------------------------------------------------------------
def model_of(shape) -> ks_model:
    """A decoder shape (any object with the ks_model field names, e.g.
    ``workload.gen.ModelShape``) -> ks_model."""
    return ks_model(*(int(getattr(shape, name)) for name in MODEL_FIELDS))


class DeviceBatch:
    """One batch of steps (request lists, prefill flags and, for a mixture of
    experts, the [steps][layers][experts] routing counts) resident on the
    device, the record arrays ks_expand writes, and a ks_desc / ks_steps
    pair over them for the evaluation entry points."""

    def __init__(self, trace, mode=KS_EXPAND_PER_LAYER, device="cuda", elem_bytes=2):
        import torch
        dev = torch.device(device)

        def u32(x):
            return torch.from_numpy(np.ascontiguousarray(x, np.uint32).view(np.int32)).to(dev)

        self.mode = mode
        self.model = model_of(trace.shape)
        S = int(trace.n_steps)
        n_pre = int(np.count_nonzero(trace.prefill))
        self.t = {"req_off": u32(trace.req_off), "req_q": u32(trace.req_q), "req_h": u32(trace.req_h),
                  "prefill": torch.from_numpy(np.ascontiguousarray(trace.prefill, np.uint8)).to(dev)}
        route = trace.experts if trace.experts is not None else np.zeros(0, np.uint32)
        self.t["route"] = u32(np.asarray(route).reshape(-1))
        self.batch = ks_batch(S, _ptr(self.t["req_off"]),
                              _ptr(self.t["req_q"]) if self.t["req_q"].numel() else None,
                              int(len(trace.req_q)), _ptr(self.t["prefill"]) if S else None, n_pre)
        _, fam_off = ks_expand_layout(self.model, S, n_pre, mode)
        self.fam_off = fam_off
        n = fam_off[-1]
        # the per-layer form has no multiplicities: its records are written
        # without them (NULL), and the descriptor carries none
        fields = ("step", "m", "n", "k", "a", "b") + (("mult",) if mode == KS_EXPAND_HOMOGENEOUS else ())
        for name in fields:
            self.t[name] = torch.empty(n, dtype=torch.int32, device=dev)
        for name in ("layers", "hidden", "tp", "n_launch"):
            self.t["s_" + name] = torch.empty(S, dtype=torch.int32, device=dev)
        self.out = ks_records(*(_ptr(self.t[name]) if n and name in self.t else None
                                for name in ("step", "m", "n", "k", "a", "b", "mult")),
                              *(_ptr(self.t["s_" + name]) if S else None
                                for name in ("layers", "hidden", "tp", "n_launch")))
        self.ws_bytes = ks_expand_workspace_bytes(S)
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
        self.ws_ptr = self.ws.data_ptr() + (-self.ws.data_ptr()) % 256

        self.desc = ks_desc()
        self.desc.n_rows = n
        for f in range(NFAM + 1):
            self.desc.fam_off[f] = fam_off[f]
        for name in ("step", "m", "n", "k", "a", "b"):
            setattr(self.desc, name, _ptr(self.t[name]) if n else None)
        self.desc.mult = _ptr(self.t["mult"]) if n and mode == KS_EXPAND_HOMOGENEOUS else None
        self.desc.n_steps = S
        self.desc.req_off = _ptr(self.t["req_off"])
        self.desc.req_q = self.batch.req_q
        self.desc.req_h = _ptr(self.t["req_h"]) if self.t["req_h"].numel() else None
        self.desc.n_req = self.batch.n_req
        self.desc.expert_rows = _ptr(self.t["route"]) if self.t["route"].numel() else None
        self.desc.n_expert_rows = int(self.t["route"].numel())
        self.desc.elem_bytes = elem_bytes
        self.steps = ks_steps(S, *(_ptr(self.t["s_" + name]) if S else None
                                   for name in ("layers", "hidden", "tp", "n_launch")))

    def expand(self, stream, check=True):
        return ks_expand(self.model, self.batch, self.mode, self.out, self.ws_ptr, self.ws_bytes,
                         stream, check)


# --------------------------------------------------------------------------
# serving simulation: host arrays in, host arrays out
# --------------------------------------------------------------------------
def simulate_many(shape, specs: dict, heads: ks_heads, host: ks_host, sched: ks_sched, requests: dict,
                  step_cap: int = 1 << 20, entry_cap: int = 1 << 22, device="cuda", check=True):
    """Runs ks_simulate with one simulation per spec vector.  shape: a
    decoder shape (ks_model field names); specs: dict of arrays [n_specs];
    requests: dict of arrays arrival, prompt, output and optionally group,
    prefix.  Returns one dict per spec vector of numpy arrays (per request
    and per step) and the counters."""
    import torch
    model = model_of(shape)
    rec = pack_specs({k: np.atleast_1d(np.asarray(v)) for k, v in specs.items()})
    S = len(rec)
    spec_t = torch.from_numpy(rec.view(np.uint8).copy()).to(device)
    n = len(requests["arrival"])
    arr = {"arrival": np.ascontiguousarray(requests["arrival"], np.float64)}
    for k in ("prompt", "output", "group", "prefix"):
        if k in requests:
            arr[k] = np.ascontiguousarray(requests[k], np.uint32)
    rq = ks_requests(n, arr["arrival"].ctypes.data, arr["prompt"].ctypes.data, arr["output"].ctypes.data,
                     arr["group"].ctypes.data if "group" in arr else None,
                     arr["prefix"].ctypes.data if "group" in arr else None)
    results = []
    outs = (ks_sim_out * S)()
    for s in range(S):
        res = {"ttft": np.zeros(n), "tpot": np.zeros(n), "e2e": np.zeros(n), "state": np.zeros(n, np.int32),
               "step_start": np.zeros(step_cap), "step_latency": np.zeros(step_cap),
               "step_prefill": np.zeros(step_cap, np.uint8),
               "step_entry_off": np.zeros(step_cap + 1, np.int64),
               "entry_req": np.zeros(entry_cap, np.uint32), "entry_q": np.zeros(entry_cap, np.uint32),
               "entry_h": np.zeros(entry_cap, np.uint32)}
        outs[s] = ks_sim_out(res["ttft"].ctypes.data, res["tpot"].ctypes.data, res["e2e"].ctypes.data,
                             res["state"].ctypes.data, step_cap, entry_cap, res["step_start"].ctypes.data,
                             res["step_latency"].ctypes.data, res["step_prefill"].ctypes.data,
                             res["step_entry_off"].ctypes.data, res["entry_req"].ctypes.data,
                             res["entry_q"].ctypes.data, res["entry_h"].ctypes.data, 0, 0, 0, 0.0)
        results.append(res)
    wsb = ks_simulate_workspace_bytes(model, sched, S)
    if wsb == 0:
        raise KsError(KS_EINVAL, ks_last_error())
    ws = torch.empty(wsb + 256, dtype=torch.uint8, device=device)
    wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
    st = ks_simulate(model, spec_t.data_ptr(), S, heads, host, sched, rq, outs, wsp, wsb, current_stream(),
                     check)
    for s, res in enumerate(results):
        out = outs[s]
        ns, ne = int(out.n_steps), int(out.n_entries)
        for k in ("step_start", "step_latency", "step_prefill"):
            res[k] = res[k][:min(ns, step_cap)]
        res["step_entry_off"] = res["step_entry_off"][:min(ns, step_cap) + 1]
        for k in ("entry_req", "entry_q", "entry_h"):
            res[k] = res[k][:ne]
        res.update(status=st, n_steps=ns, n_entries=ne, preemptions=int(out.preemptions),
                   clock=float(out.clock))
    return results


def simulate(shape, spec_row: dict, heads: ks_heads, host: ks_host, sched: ks_sched, requests: dict,
             step_cap: int = 1 << 20, entry_cap: int = 1 << 22, device="cuda", check=True):
    """ks_simulate for one spec vector (dict of scalars); one result dict."""
    return simulate_many(shape, {k: np.asarray([v]) for k, v in spec_row.items()}, heads, host, sched,
                         requests, step_cap, entry_cap, device, check)[0]
