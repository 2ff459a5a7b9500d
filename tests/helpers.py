"""Hand-built inputs for small tests."""
from __future__ import annotations

import numpy as np

from workload import gen


def make_desc(rows, reqs, expert_rows=(), elem_bytes=2):
    """rows: iterable of (family, step, m, n, k, a, b); reqs: per step, a list
    of (q, h).  Records are laid out family-major, step order kept."""
    rows = sorted(rows, key=lambda r: (r[0], r[1]))
    fam_off = np.zeros(gen.NFAM + 1, np.int64)
    for r in rows:
        fam_off[r[0] + 1] += 1
    fam_off = np.cumsum(fam_off)
    cols = list(zip(*rows)) if rows else [()] * 7
    u = lambda c: np.asarray(c, np.uint32)
    req_off = np.zeros(len(reqs) + 1, np.uint32)
    req_off[1:] = np.cumsum([len(r) for r in reqs])
    q = u([x[0] for r in reqs for x in r])
    h = u([x[1] for r in reqs for x in r])
    return gen.Desc(fam_off, u(cols[1]), u(cols[2]), u(cols[3]), u(cols[4]),
                    u(cols[5]), u(cols[6]), req_off, q, h, u(list(expert_rows)),
                    elem_bytes)


def spec(P=2.0 ** 50, BW=2.0 ** 40, n_cu=4, l2=2.0 ** 20, t0=2.0 ** -20,
         alpha0=8e-6, alpha_log2p=2e-6, beta=300e9):
    return {"peak_flops": np.array([P]), "hbm_bw": np.array([BW]),
            "t0": np.array([t0]), "l2_bytes": np.array([l2]),
            "ar_alpha0": np.array([alpha0]), "ar_alpha_log2p": np.array([alpha_log2p]),
            "ar_beta": np.array([beta]), "n_cu": np.array([n_cu], np.int64)}


def steprec(n_steps, layers=1, hidden=64, tp=1, n_launch=0):
    full = lambda v: np.full(n_steps, v, np.uint32)
    return gen.StepRec(full(layers), full(hidden), full(tp), full(n_launch))


def sub_desc(d, rows):
    """The records `rows` (sorted) of d, with d's request lists and expert
    table: the oracle then prices only those records."""
    fam = d.family()[rows]
    fam_off = np.zeros(gen.NFAM + 1, np.int64)
    fam_off[1:] = np.cumsum(np.bincount(fam, minlength=gen.NFAM))
    mult = None if getattr(d, "mult", None) is None else d.mult[rows]
    return gen.Desc(fam_off, d.step[rows], d.m[rows], d.n[rows], d.k[rows], d.a[rows], d.b[rows],
                    d.req_off, d.req_q, d.req_h, d.expert_rows, d.elem_bytes, mult)
