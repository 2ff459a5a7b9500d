"""fp64 CPU oracle of the batched kernel-latency model.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this module; only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the HIP library: it reads
the seeded inputs produced by ``workload.gen`` and computes everything else
itself, plainly and slowly, in float64 (integer counts as exact uint64 with
asserted input limits that rule out overflow).

What it computes, and where the paper states it (KernelSight-LM):

* per dispatched kernel: FLOPs F and bytes Bt from its shapes; the roofline
  operands of Eq. 2 (Sec. 5.3), with the arithmetic intensity of Eq. 1
  (Sec. 2.3);
* wave quantization u = ceil(B/N) N / B on the compute term (Sec. 2.2,
  Fig. "wave quantization"; Sec. 5.3);
* t_roof = max(F u / P, Bt / BW) (Eq. 2);
* a per-family efficiency head on dimensionless features (Sec. 5.3,
  "Per-family heads on dimensionless features"); its output is a
  utilization sigma in (0, 1] and the efficiency factor is eta = 1/sigma >= 1
  (Sec. 5.3, Fig. "efficiency factor" caption);
* per family, instead of that head, the bounded analytical head
  eta = 1/(gamma - alpha/W) (Sec. 5.3, the efficiency-factor figure);
* Tier B (Sec. 5.5): eta interpolated over a grid of measured values in
  three feature coordinates where the query lies in the measured region,
  the family's other head elsewhere ("density-routed");
* t = max(t_roof eta, t0), the launch floor applied after eta (Eq. 2);
* per-step body: the sum of the step's kernels (Sec. 5.7), which with one
  record per dispatched kernel equals L t_layer + t_lm_head + t_embed;
* ring all-reduce t_ar = alpha0 + 2(P-1)/P S/beta, two per layer (Eq. 3,
  Sec. 5.6);
* step assembly t_step = max(t_gpu + n c_disp, l) + max(0, c_ovl - t_gpu)
  + c_tail (Eq. 4, Sec. 5.7).

The per-family count formulas, the feature list, the head's activation and
the meaning of n and l in Eq. 4 are not given by the paper; the readings
taken here are the ones the library implements and are listed with the
design notes.  Parity unpinned: the absolute eta values (the heads are
seeded stand-ins for trained ones, and the paper prints no worked example
of a full prediction).
"""
from __future__ import annotations

import numpy as np

from workload.gen import (NFAM, GEMM, LM_HEAD, GROUPED_GEMM, ATTN_PREFILL,
                          ATTN_DECODE, RMSNORM, ROPE, SILU_MUL, KV_WRITE, EMBED)

TILE = 128          # output tile edge of GEMM and attention query blocks
EW_BLOCK = 1024     # elements per block of the SiLU-and-multiply kernel

U64 = np.uint64

# input limits under which every count below fits in 63 bits
LIM_M = 1 << 24
LIM_NK = 1 << 18
LIM_ATTN_NK = 1 << 12
LIM_REQ = 1 << 24        # q_r, h_r
LIM_PAIRS = 1 << 40      # per-step causal pairs


# --------------------------------------------------------------------------
# attention work of a step (Sec. 5.8, "Mixed prefill-decode steps")
# --------------------------------------------------------------------------
def attention_work(req_off, req_q, req_h):
    """Per step, over its requests r with q_r new query tokens and h_r cached
    history: each decode attends over its cached context, a prefill chunk over
    its history plus its own causal triangle (diagonal included).

    Returns uint64 arrays Q = sum q_r, KV = sum (h_r + q_r),
    PAIRS = sum (q_r h_r + q_r (q_r + 1) / 2), TILES = sum ceil(q_r / 128)."""
    req_off = np.asarray(req_off, np.int64)
    q = np.asarray(req_q, np.int64)
    h = np.asarray(req_h, np.int64)
    assert q.size == 0 or (q.max() < LIM_REQ and h.max() < LIM_REQ)
    n_steps = len(req_off) - 1
    out = {}
    per_req = {
        "Q": q.astype(U64),
        "KV": (h + q).astype(U64),
        "PAIRS": (q.astype(U64) * h.astype(U64) + q.astype(U64) * (q.astype(U64) + U64(1)) // U64(2)),
        "TILES": ((q + TILE - 1) // TILE).astype(U64),
    }
    nz = np.diff(req_off) > 0
    for key, v in per_req.items():
        acc = np.zeros(n_steps, U64)
        if nz.any():
            acc[nz] = np.add.reduceat(v, req_off[:-1][nz])
        out[key] = acc
    assert (out["PAIRS"] < U64(LIM_PAIRS)).all()
    return out


# --------------------------------------------------------------------------
# FLOPs, bytes and thread blocks of each dispatched kernel
# --------------------------------------------------------------------------
def kernel_counts(desc):
    """F (FLOPs), Bt (bytes moved) and B (thread blocks) of every record, and
    the effective row count M that the shape features use.  F and Bt are the
    F_comp and F_mem of Eq. 2; B feeds the wave count of Sec. 2.2.

    GEMM / LM head (M, N, K):   F = 2MNK, Bt = dt(MK + KN + MN),
                                B = ceil(M/128) ceil(N/128)
    grouped GEMM, experts M_e:  M = sum M_e, A = #{M_e > 0},
                                F = 2MNK, Bt = dt(MK + A KN + MN),
                                B = sum_e ceil(M_e/128) ceil(N/128)
    attention (H heads n, d = k, Hkv = a) over the step's requests:
                                F = 4 H d PAIRS, Bt = dt(2 H d Q + 2 Hkv d KV),
                                B = H TILES, M = Q
    RMSNorm (T, D):             F = 4TD, Bt = dt(2TD + D), B = T
    RoPE (T, heads, d):         F = 3 T heads d, Bt = dt(2 T heads d + T d), B = T
    SiLU x mul (T, I):          F = 5TI, Bt = 3 dt T I, B = ceil(TI/1024)
    KV write (T, Hkv, d):       F = 0, Bt = 4 dt T Hkv d, B = T
    embedding (T, D):           F = 0, Bt = 2 dt T D + 4T, B = T
    """
    n_rows = desc.n_rows
    dt = U64(desc.elem_bytes)
    F = np.zeros(n_rows, U64)
    Bt = np.zeros(n_rows, U64)
    B = np.zeros(n_rows, U64)
    M = np.zeros(n_rows, U64)
    agg = attention_work(desc.req_off, desc.req_q, desc.req_h)
    one = U64(1)
    t = U64(TILE)
    for f in range(NFAM):
        lo, hi = int(desc.fam_off[f]), int(desc.fam_off[f + 1])
        if hi == lo:
            continue
        s = slice(lo, hi)
        m = desc.m[s].astype(U64)
        n = desc.n[s].astype(U64)
        k = desc.k[s].astype(U64)
        a = desc.a[s].astype(U64)
        assert m.max() < LIM_M and n.max() < LIM_NK and k.max() < LIM_NK
        if f in (GEMM, LM_HEAD):
            F[s] = U64(2) * m * n * k
            Bt[s] = dt * (m * k + k * n + m * n)
            B[s] = ((m + t - one) // t) * ((n + t - one) // t)
            M[s] = m
        elif f == GROUPED_GEMM:
            E = desc.a[s].astype(np.int64)
            base = desc.b[s].astype(np.int64)
            idx = np.repeat(base, E) + (np.arange(E.sum()) - np.repeat(np.cumsum(E) - E, E))
            me = desc.expert_rows[idx].astype(U64)
            starts = np.cumsum(E) - E
            Msum = np.zeros(hi - lo, U64)
            act = np.zeros(hi - lo, U64)
            tiles = np.zeros(hi - lo, U64)
            nzr = E > 0
            if nzr.any():
                Msum[nzr] = np.add.reduceat(me, starts[nzr])
                act[nzr] = np.add.reduceat((me > 0).astype(U64), starts[nzr])
                tiles[nzr] = np.add.reduceat((me + t - one) // t, starts[nzr])
            assert Msum.max() < LIM_M
            F[s] = U64(2) * Msum * n * k
            Bt[s] = dt * (Msum * k + act * k * n + Msum * n)
            B[s] = tiles * ((n + t - one) // t)
            M[s] = Msum
        elif f in (ATTN_PREFILL, ATTN_DECODE):
            assert n.max() < LIM_ATTN_NK and k.max() < LIM_ATTN_NK and a.max() < LIM_ATTN_NK
            st = desc.step[s].astype(np.int64)
            Q, KV, P, TL = agg["Q"][st], agg["KV"][st], agg["PAIRS"][st], agg["TILES"][st]
            F[s] = U64(4) * n * k * P
            Bt[s] = dt * (U64(2) * n * k * Q + U64(2) * a * k * KV)
            B[s] = n * TL
            M[s] = Q
        elif f == RMSNORM:
            F[s] = U64(4) * m * n
            Bt[s] = dt * (U64(2) * m * n + n)
            B[s] = m
            M[s] = m
        elif f == ROPE:
            F[s] = U64(3) * m * n * k
            Bt[s] = dt * (U64(2) * m * n * k + m * k)
            B[s] = m
            M[s] = m
        elif f == SILU_MUL:
            F[s] = U64(5) * m * n
            Bt[s] = U64(3) * dt * m * n
            B[s] = (m * n + U64(EW_BLOCK - 1)) // U64(EW_BLOCK)
            M[s] = m
        elif f == KV_WRITE:
            F[s] = U64(0)
            Bt[s] = U64(4) * dt * m * n * k
            B[s] = m
            M[s] = m
        elif f == EMBED:
            F[s] = U64(0)
            Bt[s] = U64(2) * dt * m * n + U64(4) * m
            B[s] = m
            M[s] = m
    return {"F": F, "Bt": Bt, "B": B, "M": M}


# --------------------------------------------------------------------------
# roofline with wave quantization (Sec. 2.2; Eq. 2)
# --------------------------------------------------------------------------
def waves(B, n_cu):
    """W = ceil(B / N) scheduling waves and u = W N / B >= 1 (Sec. 2.2).
    A kernel with no blocks has W = 0 and u = 1."""
    B = np.asarray(B, U64)
    N = U64(n_cu)
    W = (B + N - U64(1)) // N
    u = np.ones(B.shape, np.float64)
    nz = B > 0
    u[nz] = (W[nz] * N).astype(np.float64) / B[nz].astype(np.float64)
    return W, u


def roofline(F, Bt, B, spec):
    """t_roof = max(F u / P_peak, Bt / BW_peak), u on the compute term only
    (Eq. 2, Sec. 5.3)."""
    W, u = waves(B, spec["n_cu"])
    t_comp = np.asarray(F, U64).astype(np.float64) * u / spec["peak_flops"]
    t_mem = np.asarray(Bt, U64).astype(np.float64) / spec["hbm_bw"]
    return {"W": W, "u": u, "t_comp": t_comp, "t_mem": t_mem,
            "t_roof": np.maximum(t_comp, t_mem)}


# --------------------------------------------------------------------------
# dimensionless features (Sec. 5.3, "Per-family heads on dimensionless
# features": arithmetic intensity and its position relative to the ridge,
# per-SM work and occupancy, wave count, L2 residency)
# --------------------------------------------------------------------------
K_UNUSED = (RMSNORM, SILU_MUL, EMBED)    # families whose records carry no K


def features(cnt, n, k, rf, spec, in_dim=16):
    """k: the records' K field, already zeroed for the families that carry
    no K (see effective_k)."""
    F = cnt["F"].astype(np.float64)
    Bt = cnt["Bt"].astype(np.float64)
    B = cnt["B"].astype(np.float64)
    M = cnt["M"].astype(np.float64)
    W = rf["W"].astype(np.float64)
    N = float(spec["n_cu"])
    P, BW = spec["peak_flops"], spec["hbm_bw"]
    ai = F / np.maximum(Bt, 1.0)                       # Eq. 1
    x = np.empty((len(F), 16), np.float64)
    x[:, 0] = np.log2(np.maximum(ai, 2.0 ** -10)) / 16          # intensity
    x[:, 1] = np.log2(np.maximum(ai * BW / P, 2.0 ** -20)) / 16  # vs ridge P/BW
    x[:, 2] = np.log2(1.0 + B / N) / 16                          # blocks per SM
    x[:, 3] = 1.0 / rf["u"]                                      # last-wave occupancy
    x[:, 4] = np.log2(1.0 + W) / 16                              # wave count
    x[:, 5] = np.minimum(1.0, spec["l2_bytes"] / np.maximum(Bt, 1.0))  # L2 residency
    x[:, 6] = np.log2(np.maximum(rf["t_roof"] / max(spec["t0"], 1e-9), 2.0 ** -20)) / 16
    den = rf["t_comp"] + rf["t_mem"]
    x[:, 7] = np.where(den > 0, rf["t_comp"] / np.where(den > 0, den, 1.0), 0.0)
    x[:, 8] = np.log2(1.0 + F) / 64
    x[:, 9] = np.log2(1.0 + Bt) / 48
    x[:, 10] = np.log2(1.0 + M) / 24
    x[:, 11] = np.log2(1.0 + np.asarray(n, np.float64)) / 24
    x[:, 12] = np.log2(1.0 + np.asarray(k, np.float64)) / 24
    x[:, 13] = np.log2(1.0 + F / np.maximum(B, 1.0)) / 48          # work per block
    x[:, 14] = np.log2(1.0 + Bt / np.maximum(B, 1.0)) / 40         # bytes per block
    x[:, 15] = 1.0
    if in_dim == 16:
        return x
    assert in_dim == 32
    return np.concatenate([x, x * x], axis=1)


# --------------------------------------------------------------------------
# efficiency head (Sec. 5.3; eta = 1/sigma, Fig. "efficiency factor")
# --------------------------------------------------------------------------
def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (8 significant bits),
    ties to even.  Normal range only."""
    x = np.asarray(x, np.float64)
    mant, ex = np.frexp(x)                  # x = mant 2^ex, 0.5 <= |mant| < 1
    tiny = (x != 0) & (np.abs(x) < 2.0 ** -126)
    assert not tiny.any(), "bf16 subnormal range is outside the model's use"
    return np.ldexp(np.rint(np.ldexp(mant, 8)), ex - 8)


def head_forward(x, w1, w2, b2, w3, b3, emulate_bf16=False):
    """z = w3 . relu(W2 relu(W1 x) + b2) + b3 for the rows of x (one family's
    parameters).  With emulate_bf16 the inputs of the two matrix layers, x
    and h1, are rounded to bfloat16 before their products (the layers the
    bf16 heads run as bfloat16 matrix products); the last layer, a dot
    product with w3, takes relu(h2) unrounded.  Products and sums stay
    float64."""
    r = round_bf16 if emulate_bf16 else (lambda v: v)
    h1 = np.maximum(r(x) @ w1.T, 0.0)
    h2 = np.maximum(r(h1) @ w2.T + b2, 0.0)
    return h2 @ w3 + b3


def bounded_eta(x16, W, g, a):
    """The bounded analytical head (Sec. 5.3, "A diverse, low-capacity head
    family", and the efficiency-factor figure): utilization gamma - alpha/W
    rising with the wave count W toward its peak gamma, eta its reciprocal.
    Reading: gamma(x) = sigma(g . x) and alpha(x) = gamma(x) sigma(a . x),
    so 0 < alpha < gamma < 1 and the utilization lies in (0, 1) for W >= 1;
    a record without blocks (W = 0) counts as one wave."""
    x16 = np.asarray(x16, np.float64)
    gamma = 1.0 / (1.0 + np.exp(-(x16 @ g)))
    alpha = gamma / (1.0 + np.exp(-(x16 @ a)))
    w = np.maximum(np.asarray(W, np.float64), 1.0)
    return 1.0 / (gamma - alpha / w)


def grid_eta(x16, grid, f):
    """Tier B (Sec. 5.5, "Tier B: Target-Measured Prediction"): eta
    interpolated over a grid of measured values in feature coordinates.
    Reading: a regular grid over three of the base features, multilinear
    interpolation of eta in the cell holding the query.  The query is routed
    to the grid only inside the grid's box and only if all eight corners of
    its cell were measured (NaN marks a missing node): the "dense interior"
    of the measured points.  Returns (eta, routed); where routed is False
    the family's learned head applies."""
    x16 = np.asarray(x16, np.float64)
    lo, hi, n = np.asarray(grid.lo), np.asarray(grid.hi), np.asarray(grid.n)
    c = x16[:, list(grid.axes)]
    t = (c - lo) / (hi - lo) * (n - 1)                       # node coordinates
    inside = np.all((t >= 0.0) & (t <= n - 1), axis=1)
    i = np.clip(np.floor(t), 0, n - 2).astype(np.int64)
    fr = t - i
    v = grid.values[f].astype(np.float64)
    eta = np.zeros(len(c))
    known = np.ones(len(c), bool)
    for corner in range(8):
        b = [(corner >> d) & 1 for d in range(3)]
        idx = tuple(np.clip(i[:, d] + b[d], 0, n[d] - 1) for d in range(3))
        w = np.prod([fr[:, d] if b[d] else 1.0 - fr[:, d] for d in range(3)], axis=0)
        val = v[idx]
        known &= ~np.isnan(val)
        eta += w * np.where(np.isnan(val), 0.0, val)
    routed = inside & known
    return np.where(routed, eta, np.nan), routed


def eta_from_z(z):
    """sigma = 1/(1 + e^-z) in (0, 1]; eta = 1/sigma = 1 + e^-z >= 1."""
    return 1.0 + np.exp(-z)


def kernel_latency(t_roof, eta, t0):
    """t = max(t_roof eta, t0): the launch floor is a hard lower bound applied
    after eta, never scaled by it (Eq. 2)."""
    return np.maximum(t_roof * eta, t0)


# --------------------------------------------------------------------------
# per-kernel evaluation for every spec vector
# --------------------------------------------------------------------------
def effective_k(desc, rows):
    """K as the features use it: the record's k, or 0 for families without K."""
    k = desc.k[rows].astype(np.int64)
    fam = desc.family()[rows]
    return np.where(np.isin(fam, K_UNUSED), 0, k)


def spec_at(specs, s):
    return {key: (int(v[s]) if key == "n_cu" else float(v[s])) for key, v in specs.items()}


def eval_kernels(desc, specs, heads=None, eta_one=False, emulate_bf16=None,
                 spec_ids=None, rows=None, keep_features=False, bounded=None, grid=None):
    """Per-kernel latency model for every (spec, record) pair.

    heads: a ``workload.gen.Heads``; eta_one forces eta = 1 (pure roofline).
    bounded: a ``workload.gen.Bounded``; the families in its mask take eta
    from the bounded analytical head instead (of the MLP or of eta = 1).
    grid: a ``workload.gen.Grid`` (Tier B); for the families in its mask,
    records routed to the grid take the interpolated eta ("routed" output;
    "x16": the base features of every pair when a grid is given).
    emulate_bf16 defaults to True for bf16 heads.  spec_ids / rows restrict
    the evaluation to a subset (counts are still exact per record).
    keep_features also returns the feature vectors ("x").
    Returns counts (per record) and float64 arrays [n_spec_ids, n_sel_rows]."""
    cnt = kernel_counts(desc)
    n_specs = len(specs["peak_flops"])
    spec_ids = list(range(n_specs)) if spec_ids is None else list(spec_ids)
    rows = np.arange(desc.n_rows) if rows is None else np.asarray(rows, np.int64)
    fam = desc.family()[rows]
    sub = {key: v[rows] for key, v in cnt.items()}
    if emulate_bf16 is None:
        emulate_bf16 = heads is not None and heads.precision == "bf16"
    out = {key: np.zeros((len(spec_ids), len(rows))) for key in
           ("t_roof", "eta", "t", "z", "t_comp", "t_mem", "u")}
    out["W"] = np.zeros((len(spec_ids), len(rows)), U64)
    out["routed"] = np.zeros((len(spec_ids), len(rows)), bool)
    if keep_features and not eta_one:
        out["x"] = np.zeros((len(spec_ids), len(rows), heads.in_dim))
    if grid is not None:
        out["x16"] = np.zeros((len(spec_ids), len(rows), 16))
    for si, s in enumerate(spec_ids):
        sp = spec_at(specs, s)
        rf = roofline(sub["F"], sub["Bt"], sub["B"], sp)
        mask = bounded.mask if bounded is not None else 0
        on_b = ((mask >> fam) & 1).astype(bool)
        if eta_one:
            z = np.full(len(rows), np.inf)
            eta = np.ones(len(rows))
        else:
            x = features(sub, desc.n[rows], effective_k(desc, rows), rf, sp, heads.in_dim)
            if keep_features:
                out["x"][si] = x
            z = np.zeros(len(rows))
            for f in np.unique(fam[~on_b]):
                sel = fam == f
                z[sel] = head_forward(x[sel], heads.w1[f], heads.w2[f], heads.b2[f],
                                      heads.w3[f], heads.b3[f], emulate_bf16)
            eta = eta_from_z(z)
        if on_b.any():
            x16 = features(sub, desc.n[rows], effective_k(desc, rows), rf, sp, 16)
            for f in np.unique(fam[on_b]):
                sel = fam == f
                eta[sel] = bounded_eta(x16[sel], rf["W"][sel], bounded.g[f], bounded.a[f])
                z[sel] = -np.log(eta[sel] - 1.0)
        gmask = grid.mask if grid is not None else 0
        on_g = ((gmask >> fam) & 1).astype(bool)
        if grid is not None:
            x16 = features(sub, desc.n[rows], effective_k(desc, rows), rf, sp, 16)
            out["x16"][si] = x16
            for f in np.unique(fam[on_g]):
                sel = np.nonzero(fam == f)[0]
                eg, routed = grid_eta(x16[sel], grid, f)
                eta[sel[routed]] = eg[routed]
                z[sel[routed]] = -np.log(np.maximum(eg[routed] - 1.0, 1e-300))
                out["routed"][si, sel] = routed
        out["t_roof"][si] = rf["t_roof"]
        out["t_comp"][si] = rf["t_comp"]
        out["t_mem"][si] = rf["t_mem"]
        out["u"][si] = rf["u"]
        out["W"][si] = rf["W"]
        out["z"][si] = z
        out["eta"][si] = eta
        out["t"][si] = kernel_latency(rf["t_roof"], eta, sp["t0"])
    out["counts"] = cnt
    out["rows"] = rows
    return out


# --------------------------------------------------------------------------
# step terms (Sec. 5.6, Eq. 3; Sec. 5.7, Eq. 4)
# --------------------------------------------------------------------------
def step_body(t, step, n_steps, mult=None):
    """Sum of the latencies of each step's kernels (Sec. 5.7); a record of
    multiplicity m stands for m dispatches of the same kernel (the L
    homogeneous layers of t_gpu = L t_layer + ...) and adds m t."""
    w = t if mult is None else t * np.asarray(mult, np.float64)
    return np.bincount(np.asarray(step, np.int64), weights=w, minlength=n_steps)


def allreduce_time(P, S, alpha0, alpha_log2p, beta):
    """Ring all-reduce (Eq. 3): t_ar = alpha0(P) + 2(P-1)/P S / beta_eff with
    alpha0(P) = alpha0 + alpha_log2p log2 P (startup growing weakly with P).
    A single shard (P = 1) issues no all-reduce."""
    P = np.asarray(P, np.float64)
    S = np.asarray(S, np.float64)
    t = alpha0 + alpha_log2p * np.log2(np.maximum(P, 1.0)) + 2.0 * (P - 1.0) / P * S / beta
    return np.where(P > 1, t, 0.0)


def step_assembly(t_gpu, n_launch, c_disp, ell, c_ovl, c_tail):
    """Eq. 4: t_step = max(t_gpu + n c_disp, l) + max(0, c_ovl - t_gpu) + c_tail."""
    return (np.maximum(t_gpu + n_launch * c_disp, ell)
            + np.maximum(0.0, c_ovl - t_gpu) + c_tail)


def eval_steps(desc, steprec, specs, host, heads=None, eta_one=False,
               emulate_bf16=None, spec_ids=None, kern=None, bounded=None, grid=None):
    """Per (spec, step): t_body, t_comm, t_gpu, t_step.  Every step's records
    must be present in desc (the body sums them).  ``kern`` may pass a result
    of eval_kernels over all rows to reuse."""
    if kern is None:
        kern = eval_kernels(desc, specs, heads, eta_one, emulate_bf16, spec_ids, bounded=bounded, grid=grid)
    n_steps = desc.n_steps
    spec_ids = list(range(len(specs["peak_flops"]))) if spec_ids is None else list(spec_ids)
    tokens = attention_work(desc.req_off, desc.req_q, desc.req_h)["Q"].astype(np.float64)
    S = tokens * steprec.hidden.astype(np.float64) * desc.elem_bytes   # activation bytes
    L = steprec.layers.astype(np.float64)
    out = {key: np.zeros((len(spec_ids), n_steps)) for key in ("t_body", "t_comm", "t_gpu", "t_step")}
    for si, s in enumerate(spec_ids):
        sp = spec_at(specs, s)
        mult = None if getattr(desc, "mult", None) is None else desc.mult[kern["rows"]]
        body = step_body(kern["t"][si], desc.step[kern["rows"]], n_steps, mult)
        t_ar = allreduce_time(steprec.tp, S, sp["ar_alpha0"], sp["ar_alpha_log2p"], sp["ar_beta"])
        comm = 2.0 * L * t_ar                       # two all-reduces per layer
        gpu = host.body_scale * body + comm
        out["t_body"][si] = body
        out["t_comm"][si] = comm
        out["t_gpu"][si] = gpu
        out["t_step"][si] = step_assembly(gpu, steprec.n_launch.astype(np.float64),
                                          host.c_disp, host.ell, host.c_ovl, host.c_tail)
    return out
