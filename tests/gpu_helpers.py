"""Run the HIP path through the C ABI on synthetic workloads (GPU tests)."""
from __future__ import annotations

import numpy as np

from paper_2606_28565_amd import abi


def eval_kernels(wl, eta_one=False, n_specs=None, counts=True, bounded=None, grid=None):
    import torch
    di = abi.DeviceInputs(wl, n_specs=n_specs)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden,
                          abi.KS_ETA_ONE if eta_one else abi.KS_ETA_MLP, bounded, grid)
    o, so = abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=counts)
    abi.ks_eval_kernels(di.desc, di.specs_ptr, di.n_specs, heads, so, di.ws_ptr, di.ws_bytes,
                        abi.current_stream())
    torch.cuda.synchronize()
    abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
    out = {k: v.cpu().numpy() for k, v in o.items()}
    for k in ("flops", "bytes", "blocks"):
        if k in out:
            out[k] = out[k].view(np.uint64)
    return out


def eval_steps(wl, eta_one=False, n_specs=None, per_pair=True, counts=True, bounded=None,
               null_mlp=False, grid=None, source=False):
    """counts=False asks for per-pair outputs without the per-record counts
    (the eta = 1 stream then forms F and Bt in fp32).  bounded: a
    ``workload.gen.Bounded``; grid: a ``workload.gen.Grid``; null_mlp
    passes NULL MLP weights."""
    import torch
    di = abi.DeviceInputs(wl, n_specs=n_specs)
    heads = di.make_heads(wl.heads.precision, wl.heads.in_dim, wl.heads.hidden,
                          abi.KS_ETA_ONE if eta_one else abi.KS_ETA_MLP, bounded, grid)
    if null_mlp:
        heads.w1 = heads.w2 = heads.b2 = heads.w3 = heads.b3 = None
    so_t, so = abi.step_outputs(wl.desc.n_steps, di.n_specs)
    ko_t, ko = (abi.kernel_outputs(wl.desc.n_rows, di.n_specs, counts=counts, source=source) if per_pair
                else ({}, None))
    abi.ks_eval_steps(di.desc, di.steps, di.specs_ptr, di.n_specs, heads, di.host, so, ko,
                      di.ws_ptr, di.ws_bytes, abi.current_stream())
    torch.cuda.synchronize()
    abi.ks_device_status(di.ws_ptr, di.ws_bytes, abi.current_stream())
    out = {k: v.cpu().numpy() for k, v in so_t.items()}
    for k, v in ko_t.items():
        out[k] = v.cpu().numpy()
        if k in ("flops", "bytes", "blocks"):
            out[k] = out[k].view(np.uint64)
    return out


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return np.abs(a - b) / np.maximum(np.abs(b), 1e-300)
