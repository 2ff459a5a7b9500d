"""Seeded synthetic workloads for the batched kernel-latency evaluator.

This module only produces inputs.  It draws batch compositions (per-request
query and history lengths), per-layer expert token counts, hardware spec
vectors, efficiency-head parameters and host constants, and lays the
dispatched kernels of every serving step out as shape records.  It computes
no part of the latency model: no FLOP, byte, block or pair counts, no
roofline, no features, no head, no sums.  Both the CPU oracle and the HIP
path read what it returns.

The batch descriptor follows the paper's statement of the predictor input
(Sec. 4.1 "System Overview" and Sec. 5.8 "Mixed prefill-decode steps"): per
step, the decode tokens, the prefill-chunk lengths and every request's
KV-cache length.  One kernel record is emitted per dispatched kernel; the
dense kernels of a step run over all of its tokens, and one attention kernel
per layer covers all of the step's requests.

All randomness uses ``numpy.random.Generator(PCG64(seed))``.
"""
from __future__ import annotations

import dataclasses
import functools
from dataclasses import dataclass, field

import numpy as np

SEED = 20260602
HEAD_SEED = SEED + 100

FAMILIES = ("GEMM", "LM_HEAD", "GROUPED_GEMM", "ATTN_PREFILL", "ATTN_DECODE",
            "RMSNORM", "ROPE", "SILU_MUL", "KV_WRITE", "EMBED")
NFAM = len(FAMILIES)
(GEMM, LM_HEAD, GROUPED_GEMM, ATTN_PREFILL, ATTN_DECODE,
 RMSNORM, ROPE, SILU_MUL, KV_WRITE, EMBED) = range(NFAM)


# --------------------------------------------------------------------------
# model shapes
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelShape:
    """Decoder shape; TP shards are modelled as per-GPU shapes."""
    name: str
    hidden: int          # D
    layers: int          # L
    q_heads: int         # Hq, whole model
    kv_heads: int        # Hkv, whole model
    head_dim: int        # d
    ffn: int             # FFN width, whole model (dense MLP)
    vocab: int = 32000   # V
    tp: int = 1          # P
    experts: int = 0     # E (0: dense MLP)
    top_k: int = 0
    expert_ffn: int = 0  # per-expert FFN width, whole model
    kv_write: bool = False  # emit a KV-cache write kernel per layer

    # per-GPU shard sizes (KV heads replicate when there are fewer than P)
    @property
    def h(self) -> int:
        return self.q_heads // self.tp

    @property
    def hkv(self) -> int:
        return -(-self.kv_heads // self.tp)

    @property
    def i(self) -> int:
        return self.ffn // self.tp

    @property
    def ie(self) -> int:
        return self.expert_ffn // self.tp

    @property
    def v(self) -> int:
        return self.vocab // self.tp


LLAMA7B = ModelShape("llama-7b", 4096, 32, 32, 32, 128, 11008)
DENSE_SHAPES = (
    ModelShape("S1", 2048, 24, 16, 8, 128, 5632, tp=1),
    ModelShape("S2", 4096, 32, 32, 32, 128, 11008, tp=1),
    ModelShape("S3", 4096, 32, 32, 8, 128, 14336, tp=2),
    ModelShape("S4", 5120, 40, 40, 8, 128, 13824, tp=4),
    ModelShape("S5", 8192, 48, 64, 8, 128, 22016, tp=4),
    ModelShape("S6", 8192, 80, 64, 8, 128, 28672, tp=8),
)
MIXTRAL = ModelShape("mixtral-8x7b", 4096, 32, 32, 8, 128, 0, experts=8,
                     top_k=2, expert_ffn=14336)
LLAMA70B = ModelShape("70b", 8192, 80, 64, 8, 128, 28672)


# --------------------------------------------------------------------------
# kernel templates: which kernels a layer / a step dispatches, in order
# --------------------------------------------------------------------------
# m source: "T" tokens of the step, "2T" routed token copies (top-2),
# "R" requests of the step (LM head), "0" unused (attention, grouped GEMM).
@dataclass(frozen=True)
class _Tpl:
    fam: int          # family; ATTN_PREFILL stands for "the step's attention"
    m_src: str
    n: int
    k: int
    a: int = 0
    grouped: bool = False


def _layer_templates(s: ModelShape) -> list[_Tpl]:
    d, D = s.head_dim, s.hidden
    t = [_Tpl(GEMM, "T", (s.h + 2 * s.hkv) * d, D),        # QKV projection
         _Tpl(ROPE, "T", s.h + s.hkv, d)]                  # rotary on q and k
    if s.kv_write:
        t.append(_Tpl(KV_WRITE, "T", s.hkv, d))            # KV-cache write
    t += [_Tpl(ATTN_PREFILL, "0", s.h, d, s.hkv),          # attention
          _Tpl(GEMM, "T", D, s.h * d),                     # O projection
          _Tpl(RMSNORM, "T", D, 0),
          _Tpl(RMSNORM, "T", D, 0)]
    if s.experts == 0:
        t += [_Tpl(GEMM, "T", 2 * s.i, D),                 # gate/up
              _Tpl(SILU_MUL, "T", s.i, 0),
              _Tpl(GEMM, "T", D, s.i)]                     # down
    else:
        t += [_Tpl(GEMM, "T", s.experts, D),               # router
              _Tpl(GROUPED_GEMM, "0", 2 * s.ie, D, s.experts, True),
              _Tpl(SILU_MUL, "2T", s.ie, 0),
              _Tpl(GROUPED_GEMM, "0", D, s.ie, s.experts, True)]
    return t


def _step_templates(s: ModelShape) -> list[_Tpl]:
    return [_Tpl(EMBED, "T", s.hidden, 0),
            _Tpl(LM_HEAD, "R", s.v, s.hidden)]


def kernels_per_step(s: ModelShape) -> int:
    return s.layers * len(_layer_templates(s)) + len(_step_templates(s))


# --------------------------------------------------------------------------
# batch traces
# --------------------------------------------------------------------------
@dataclass
class Trace:
    """Per-step batch descriptors for one model shape."""
    shape: ModelShape
    req_off: np.ndarray        # int64 [S+1]
    req_q: np.ndarray          # int64 [R]  query tokens of each request
    req_h: np.ndarray          # int64 [R]  cached history of each request
    prefill: np.ndarray        # bool  [S]  step carries a prefill chunk
    experts: np.ndarray | None = None   # int64 [S, L, E] routed token copies

    @property
    def n_steps(self) -> int:
        return len(self.prefill)

    def slice(self, lo: int, hi: int) -> "Trace":
        r0, r1 = int(self.req_off[lo]), int(self.req_off[hi])
        return Trace(self.shape, self.req_off[lo:hi + 1] - r0,
                     self.req_q[r0:r1].copy(), self.req_h[r0:r1].copy(),
                     self.prefill[lo:hi].copy(),
                     None if self.experts is None else self.experts[lo:hi].copy())


def step_tokens(tr: "Trace") -> np.ndarray:
    """Query tokens per step (the batch's token count)."""
    out = np.zeros(tr.n_steps, np.int64)
    nz = np.diff(tr.req_off) > 0
    if nz.any():
        out[nz] = np.add.reduceat(tr.req_q, tr.req_off[:-1][nz])
    return out


def _requests(batch, prefill, q_first, ctx, h_first_extra=None):
    req_off = np.zeros(len(batch) + 1, np.int64)
    np.cumsum(batch, out=req_off[1:])
    q = np.ones(int(req_off[-1]), np.int64)
    h = ctx.astype(np.int64)
    first = req_off[:-1][prefill]
    q[first] = q_first[prefill]
    if h_first_extra is not None:
        h[first] += h_first_extra[prefill]
    return req_off, q, h


def trace_uniform(shape, n_steps, seed, bmax=64, ctx_lo=128, ctx_hi=4096,
                  p_prefill=0.3, chunk_lo=64, chunk_hi=2048):
    """Batch ~U{1..bmax}, context ~U{ctx_lo..ctx_hi}; a step carries a prefill
    chunk ~U{chunk_lo..chunk_hi} with probability p_prefill (request 0 then
    prefills that chunk over its context; the others decode one token)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    batch = rng.integers(1, bmax, size=n_steps, endpoint=True)
    prefill = rng.random(n_steps) < p_prefill
    chunk = rng.integers(chunk_lo, chunk_hi, size=n_steps, endpoint=True)
    ctx = rng.integers(ctx_lo, ctx_hi, size=int(batch.sum()), endpoint=True)
    req_off, q, h = _requests(batch, prefill, chunk, ctx)
    return Trace(shape, req_off, q, h, prefill)


def trace_lognormal(shape, n_steps, seed, bmax=256, median=1024, sigma=1.0,
                    ctx_max=32768, p_prefill=0.3, chunk_lo=64, chunk_hi=2048):
    """Batch ~U{1..bmax}; context = min(ctx_max, max(1, floor(LogNormal)))."""
    rng = np.random.Generator(np.random.PCG64(seed))
    batch = rng.integers(1, bmax, size=n_steps, endpoint=True)
    prefill = rng.random(n_steps) < p_prefill
    chunk = rng.integers(chunk_lo, chunk_hi, size=n_steps, endpoint=True)
    ln = rng.lognormal(np.log(median), sigma, size=int(batch.sum()))
    ctx = np.minimum(ctx_max, np.maximum(1, np.floor(ln))).astype(np.int64)
    req_off, q, h = _requests(batch, prefill, chunk, ctx)
    return Trace(shape, req_off, q, h, prefill)


def trace_pareto_prefix(shape, n_steps, seed, bmax=64, alpha=1.2, ctx_min=512,
                        ctx_max=131072, p_prefill=0.3, chunk_lo=64,
                        chunk_hi=2048, hit_max=0.9):
    """Pareto(alpha, ctx_min) contexts capped at ctx_max.  A prefill step's
    chunk c0 loses its prefix-cache hit fraction f ~ U[0, hit_max]: only
    max(1, round(c0 (1-f))) tokens are computed, and the cached part joins
    the request's history."""
    rng = np.random.Generator(np.random.PCG64(seed))
    batch = rng.integers(1, bmax, size=n_steps, endpoint=True)
    prefill = rng.random(n_steps) < p_prefill
    chunk = rng.integers(chunk_lo, chunk_hi, size=n_steps, endpoint=True)
    u = 1.0 - rng.random(int(batch.sum()))          # (0, 1]
    ctx = np.minimum(ctx_max, np.floor(ctx_min * u ** (-1.0 / alpha))).astype(np.int64)
    hit = rng.uniform(0.0, hit_max, size=n_steps)
    computed = np.maximum(1, np.rint(chunk * (1.0 - hit))).astype(np.int64)
    req_off, q, h = _requests(batch, prefill, computed, ctx, chunk - computed)
    return Trace(shape, req_off, q, h, prefill)


ROUTE_BLOCK = 1024


def route_tokens(tr: Trace, seed: int, step_lo=0, step_hi=None, alpha=0.5) -> np.ndarray:
    """Per (step, layer): expert shares p ~ Dirichlet(alpha 1_E) and routed
    copies M ~ Multinomial(top_k T, p).  Drawn in blocks of ROUTE_BLOCK steps
    from generators seeded by (seed, block), so any step range [step_lo,
    step_hi) of the full trace is cheap and identical to the full draw."""
    s = tr.shape
    step_hi = tr.n_steps if step_hi is None else step_hi
    tokens = step_tokens(tr)
    out = np.empty((step_hi - step_lo, s.layers, s.experts), np.int64)
    b_lo = step_lo // ROUTE_BLOCK
    for blk in range(b_lo * ROUTE_BLOCK, step_hi, ROUTE_BLOCK):
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence([seed, blk // ROUTE_BLOCK])))
        j1 = min(tr.n_steps, blk + ROUTE_BLOCK)
        n_t = np.repeat(s.top_k * tokens[blk:j1], s.layers)
        p = rng.dirichlet(np.full(s.experts, alpha), size=len(n_t))
        m = rng.multinomial(n_t, p).reshape(j1 - blk, s.layers, s.experts)
        lo, hi = max(blk, step_lo), min(j1, step_hi)
        if hi > lo:
            out[lo - step_lo:hi - step_lo] = m[lo - blk:hi - blk]
    return out


# --------------------------------------------------------------------------
# kernel records (family-major structure of arrays)
# --------------------------------------------------------------------------
@dataclass
class Desc:
    """Dispatched-kernel records, family-major and step-sorted per family."""
    fam_off: np.ndarray        # int64 [NFAM+1]
    step: np.ndarray           # uint32 [n_rows]
    m: np.ndarray
    n: np.ndarray
    k: np.ndarray
    a: np.ndarray
    b: np.ndarray
    req_off: np.ndarray        # uint32 [n_steps+1]
    req_q: np.ndarray          # uint32 [n_req]
    req_h: np.ndarray          # uint32 [n_req]
    expert_rows: np.ndarray    # uint32 [n_expert_rows]
    elem_bytes: int = 2
    mult: np.ndarray | None = None   # uint32 [n_rows]: dispatches per record (None: 1)

    @property
    def n_rows(self) -> int:
        return int(self.fam_off[-1])

    @property
    def n_steps(self) -> int:
        return len(self.req_off) - 1

    def family(self) -> np.ndarray:
        return np.repeat(np.arange(NFAM, dtype=np.int64), np.diff(self.fam_off))


@dataclass
class StepRec:
    """Per-step model record."""
    layers: np.ndarray         # uint32 [n_steps]
    hidden: np.ndarray         # uint32
    tp: np.ndarray             # uint32
    n_launch: np.ndarray       # uint32: host launches priced by c_disp


def build(traces: list[Trace]) -> tuple[Desc, StepRec]:
    """Lay the traces (consecutive step ranges) out as kernel records."""
    per_fam = [[] for _ in range(NFAM)]
    req_off, req_q, req_h, experts = [0], [], [], []
    layers, hidden, tp, n_launch = [], [], [], []
    step0, r0, e0 = 0, 0, 0
    for tr in traces:
        s, S = tr.shape, tr.n_steps
        steps = np.arange(S, dtype=np.int64)
        nreq = np.diff(tr.req_off)
        tokens = step_tokens(tr)
        msrc = {"T": tokens, "2T": s.top_k * tokens, "R": nreq, "0": np.zeros(S, np.int64)}
        for v in msrc.values():
            assert v.size == 0 or (v.min() >= 0 and v.max() < 2 ** 32), "m does not fit u32"
        assert step0 + S < 2 ** 32
        msrc32 = {key: v.astype(np.uint32) for key, v in msrc.items()}
        lt = _layer_templates(s)
        attn_fam = np.where(tr.prefill, ATTN_PREFILL, ATTN_DECODE)
        for f in range(NFAM):
            if f in (ATTN_PREFILL, ATTN_DECODE):
                tpls = [t for t in lt if t.fam == ATTN_PREFILL]
                sel = steps[attn_fam == f]
                per_layer = True
            else:
                tpls = [t for t in lt if t.fam == f]
                per_layer = bool(tpls)
                if not tpls:
                    tpls = [t for t in _step_templates(s) if t.fam == f]
                sel = steps
            if not tpls or len(sel) == 0:
                continue
            nt = len(tpls)
            reps = s.layers if per_layer else 1
            cnt = reps * nt
            ns = len(sel)
            # (step, slot) tables; slot = layer * nt + template
            slot_tpl = [tpls[q % nt] for q in range(cnt)]
            u32 = np.uint32
            st = np.repeat((sel + step0).astype(u32), cnt)
            n_arr = np.tile(np.array([t.n for t in slot_tpl], u32), ns)
            k_arr = np.tile(np.array([t.k for t in slot_tpl], u32), ns)
            a_arr = np.tile(np.array([t.a for t in slot_tpl], u32), ns)
            m2 = np.empty((ns, cnt), u32)
            for q, t in enumerate(slot_tpl):
                m2[:, q] = msrc32[t.m_src][sel]
            m_arr = m2.reshape(-1)
            b2 = np.zeros((ns, cnt), u32)
            for q, t in enumerate(slot_tpl):
                if t.grouped:
                    v = e0 + (sel * s.layers + q // nt) * s.experts
                    assert v.size == 0 or (v.min() >= 0 and v.max() + s.experts <= 2 ** 32)
                    b2[:, q] = v
            b_arr = b2.reshape(-1)
            per_fam[f].append((st, m_arr, n_arr, k_arr, a_arr, b_arr))
        req_off.append(tr.req_off[1:] + r0)
        req_q.append(tr.req_q)
        req_h.append(tr.req_h)
        if tr.experts is not None:
            experts.append(tr.experts.reshape(-1))
            e0 += tr.experts.size
        layers.append(np.full(S, s.layers))
        hidden.append(np.full(S, s.hidden))
        tp.append(np.full(S, s.tp))
        # prefill steps run eagerly: one host launch charge per layer;
        # pure decode steps replay a captured graph (no per-kernel launch).
        n_launch.append(np.where(tr.prefill, s.layers, 0))
        step0 += S
        r0 += int(tr.req_off[-1])

    fam_off = np.zeros(NFAM + 1, np.int64)
    cols = [[] for _ in range(6)]
    for f in range(NFAM):
        for part in per_fam[f]:
            for c, arr in zip(cols, part):
                c.append(arr)
        fam_off[f + 1] = fam_off[f] + sum(len(p[0]) for p in per_fam[f])

    def cat(xs, dt=np.uint32):
        if not xs:
            return np.zeros(0, dt)
        if all(x.dtype == dt for x in xs):
            return np.concatenate(xs) if len(xs) > 1 else xs[0]
        x = np.concatenate(xs)
        if x.size:
            assert x.min() >= 0 and x.max() < 2 ** 32, "field does not fit u32"
        return x.astype(dt)

    step, m, n, k, a, b = (cat(c) for c in cols)
    desc = Desc(fam_off, step, m, n, k, a, b,
                cat([np.array([0])] + req_off[1:]) if len(req_off) > 1 else np.zeros(1, np.uint32),
                cat(req_q), cat(req_h), cat(experts))
    rec = StepRec(cat(layers), cat(hidden), cat(tp), cat(n_launch))
    return desc, rec


# --------------------------------------------------------------------------
# hardware spec vectors, heads, host constants
# --------------------------------------------------------------------------
SPEC_FIELDS = ("peak_flops", "hbm_bw", "t0", "l2_bytes", "ar_alpha0",
               "ar_alpha_log2p", "ar_beta", "n_cu")


def specs_datasheet() -> dict:
    """Two datasheet spec vectors: dense BF16 peak and HBM bandwidth of the
    GB200 and H100-80GB rows of the paper's GPU table (Appendix, Table
    "GPUs used").  SM count and L2 size are public datasheet values the paper
    does not list; t0 is the portable launch floor, and the all-reduce
    constants are synthetic."""
    return {
        "peak_flops": np.array([2.25e15, 9.89e14]),
        "hbm_bw": np.array([8.0e12, 3.35e12]),
        "t0": np.array([3.0e-6, 3.0e-6]),
        "l2_bytes": np.array([126.0 * 2 ** 20, 50.0 * 2 ** 20]),
        "ar_alpha0": np.array([8.0e-6, 8.0e-6]),
        "ar_alpha_log2p": np.array([2.0e-6, 2.0e-6]),
        "ar_beta": np.array([300e9, 300e9]),
        "n_cu": np.array([148, 132], np.int64),
    }


def specs_grid(n: int, seed: int) -> dict:
    """Hypothetical GPUs: P ~ logU[0.5, 5] PFLOP/s, BW ~ logU[2, 10] TB/s,
    N_cu ~ U{64..320}, L2 ~ logU[32, 256] MiB, t0 ~ logU[1, 5] us,
    beta ~ logU[100, 900] GB/s."""
    rng = np.random.Generator(np.random.PCG64(seed))

    def logu(lo, hi):
        return np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))
    p = logu(0.5e15, 5e15)
    bw = logu(2e12, 10e12)
    ncu = rng.integers(64, 320, size=n, endpoint=True)
    l2 = logu(32 * 2 ** 20, 256 * 2 ** 20)
    t0 = logu(1e-6, 5e-6)
    beta = logu(100e9, 900e9)
    return {"peak_flops": p, "hbm_bw": bw, "t0": t0, "l2_bytes": l2,
            "ar_alpha0": np.full(n, 8.0e-6), "ar_alpha_log2p": np.full(n, 2.0e-6),
            "ar_beta": beta, "n_cu": ncu.astype(np.int64)}


def _f32_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Storage conversion of drawn parameters: round-to-nearest-even of the
    float32 bit pattern to its upper 16 bits (finite inputs only)."""
    u = x32.astype(np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@dataclass
class Heads:
    """Per-family efficiency heads: z = w3 . relu(W2 relu(W1 x) + b2) + b3.
    The first layer has no separate bias: the constant feature x15 = 1 carries
    it through W1's matching column."""
    in_dim: int
    hidden: int
    precision: str             # "f32" or "bf16"
    w1: np.ndarray             # float64 [NFAM, H, in]  exact parameter values
    w2: np.ndarray             # [NFAM, H, H]
    b2: np.ndarray             # [NFAM, H]
    w3: np.ndarray             # [NFAM, H]
    b3: np.ndarray             # [NFAM]
    storage: dict = field(default_factory=dict)   # name -> float32 / uint16 bits


def make_heads(in_dim: int, hidden: int, precision: str, seed: int = HEAD_SEED,
               std: float = 0.1) -> Heads:
    """Family f draws W1, W2, b2, w3, b3 (row-major [out][in]) in that order
    from PCG64(seed + f), all N(0, std^2).  Values are rounded once to the
    head's storage precision; those rounded values are the parameters."""
    shapes = {"w1": (hidden, in_dim), "w2": (hidden, hidden), "b2": (hidden,),
              "w3": (hidden,), "b3": ()}
    vals = {k: [] for k in shapes}
    stor = {k: [] for k in shapes}
    for f in range(NFAM):
        rng = np.random.Generator(np.random.PCG64(seed + f))
        for name, shp in shapes.items():
            x32 = rng.normal(0.0, std, size=shp).astype(np.float32)
            if precision == "f32":
                stor[name].append(x32)
                vals[name].append(x32.astype(np.float64))
            elif precision == "bf16":
                bits = _f32_to_bf16_bits(np.atleast_1d(x32)).reshape(shp)
                stor[name].append(bits)
                vals[name].append(_bf16_bits_to_f64(np.atleast_1d(bits)).reshape(shp))
            else:
                raise ValueError(precision)
    v = {k: np.stack(x) for k, x in vals.items()}
    s = {k: np.ascontiguousarray(np.stack(x)) for k, x in stor.items()}
    return Heads(in_dim, hidden, precision, v["w1"], v["w2"], v["b2"], v["w3"],
                 v["b3"], s)


@dataclass
class Bounded:
    """Per-family bounded analytical heads (the form NeuSight uses, kept by
    the paper as one admissible head): gamma and alpha are logistic-linear
    in the 16 base features.  mask bit f: family f uses this head instead of
    the MLP (or instead of eta = 1)."""
    mask: int
    g: np.ndarray              # float64 [NFAM, 16]  exact parameter values (fp32)
    a: np.ndarray              # float64 [NFAM, 16]
    storage: np.ndarray        # float32 [NFAM, 2, 16]: g then a


BOUNDED_SEED = HEAD_SEED + 50


def make_bounded(mask: int, seed: int = BOUNDED_SEED, std: float = 0.5) -> Bounded:
    """Family f draws g then a (16 each) from PCG64(seed + f), N(0, std^2),
    rounded to float32 (the rounded values are the parameters)."""
    st = np.zeros((NFAM, 2, 16), np.float32)
    for f in range(NFAM):
        rng = np.random.Generator(np.random.PCG64(seed + f))
        st[f, 0] = rng.normal(0.0, std, 16).astype(np.float32)
        st[f, 1] = rng.normal(0.0, std, 16).astype(np.float32)
    v = st.astype(np.float64)
    return Bounded(int(mask), v[:, 0].copy(), v[:, 1].copy(), np.ascontiguousarray(st))


# the families whose head the mixed configuration switches to the bounded
# form: compute-bound GEMMs and the smooth memory-bound writes (Sec. 5.3)
BOUNDED_MIXED = (1 << GEMM) | (1 << LM_HEAD) | (1 << GROUPED_GEMM) | (1 << KV_WRITE) | (1 << EMBED)
BOUNDED_ALL = (1 << NFAM) - 1


@dataclass
class Grid:
    """Tier-B measured efficiency grids (synthetic stand-ins): per family a
    regular grid over three of the 16 base features, eta at each node, NaN
    where the node was not measured.  mask bit f: family f has a grid."""
    mask: int
    axes: tuple                # three feature indices
    lo: np.ndarray             # float64 [3]
    hi: np.ndarray             # float64 [3]
    n: tuple                   # nodes per axis
    values: np.ndarray         # float32 [NFAM, n0, n1, n2]; the float32 values are the data


GRID_SEED = HEAD_SEED + 60


def make_grid(mask: int, axes=(1, 2, 6), lo=(-0.8, 0.0, -0.4), hi=(0.2, 0.4, 0.6), n=(8, 8, 8),
              holes: float = 0.08, seed: int = GRID_SEED) -> Grid:
    """A smooth efficiency surface over the grid's coordinates (c0, c1, c2),
    eta = 1 + 0.6 sigma(3 c0 + 2) + 0.8 c1 + 0.3 cos(3 c2) + N(0, 0.02^2)
    (kept >= 1), different per family by a seeded offset; a seeded fraction
    `holes` of the nodes is left unmeasured (NaN)."""
    lo, hi = np.asarray(lo, np.float64), np.asarray(hi, np.float64)
    c = [np.linspace(lo[d], hi[d], n[d]) for d in range(3)]
    C0, C1, C2 = np.meshgrid(*c, indexing="ij")
    vals = np.zeros((NFAM,) + tuple(n), np.float32)
    for f in range(NFAM):
        rng = np.random.Generator(np.random.PCG64(seed + f))
        off = rng.uniform(0.0, 0.5)
        eta = (1.0 + off + 0.6 / (1.0 + np.exp(-(3.0 * C0 + 2.0))) + 0.8 * C1 + 0.3 * np.cos(3.0 * C2)
               + rng.normal(0.0, 0.02, C0.shape))
        eta = np.maximum(eta, 1.0)
        eta[rng.uniform(size=C0.shape) < holes] = np.nan
        vals[f] = eta.astype(np.float32)
    return Grid(int(mask), tuple(axes), lo, hi, tuple(n), vals)


GRID_ALL = (1 << NFAM) - 1


@dataclass(frozen=True)
class HostConsts:
    """Host terms of the step assembly (synthetic calibration values)."""
    c_disp: float = 4.0e-6       # per host launch
    ell: float = 1.5e-3          # host floor of a step
    c_ovl: float = 2.5e-3        # host overlap floor
    c_tail: float = 3.0e-4       # serial tail
    body_scale: float = 1.04     # microbenchmark-to-serving body scale


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------
@dataclass
class Workload:
    name: str
    desc: Desc
    steps: StepRec
    specs: dict
    heads: Heads
    host: HostConsts
    info: dict = field(default_factory=dict)

    @property
    def n_specs(self) -> int:
        return len(self.specs["peak_flops"])

    def with_heads(self, heads: Heads) -> "Workload":
        return dataclasses.replace(self, heads=heads)


C1_STEPS, C2_STEPS, C3_STEPS, C4_GRID_STEPS, C5_STEPS = 1000, 100_000, 200_000, 345, 500_000


# Full traces are drawn at their configured length and then sliced, so a step
# range is always a slice of the same trace.
@functools.lru_cache(maxsize=2)
def trace_c1() -> Trace:
    return trace_uniform(LLAMA7B, C1_STEPS, SEED + 1)


@functools.lru_cache(maxsize=2)
def trace_c2(shape_idx: int) -> Trace:
    return trace_lognormal(DENSE_SHAPES[shape_idx], C2_STEPS, SEED + 2 + 10 * (shape_idx + 1))


@functools.lru_cache(maxsize=1)
def trace_c3() -> Trace:
    return trace_uniform(MIXTRAL, C3_STEPS, SEED + 3)


@functools.lru_cache(maxsize=1)
def trace_c5() -> Trace:
    return trace_pareto_prefix(LLAMA70B, C5_STEPS, SEED + 5)


def _wl(name, traces, specs, heads, info=None):
    desc, rec = build(traces)
    return Workload(name, desc, rec, specs, heads, HostConsts(), info or {})


def config1(step_lo=0, step_hi=C1_STEPS) -> Workload:
    """Llama-7B shape, 1000 steps, batch U{1..64}, context U{128..4096},
    30% prefill steps with chunk U{64..2048}; 2 datasheet spec vectors;
    fp32 16->64->64->1 heads."""
    tr = trace_c1().slice(step_lo, step_hi)
    return _wl("c1-llama7b", [tr], specs_datasheet(), make_heads(16, 64, "f32"),
               {"steps": (step_lo, step_hi)})


def config2(shape_idx: int, step_lo=0, step_hi=C2_STEPS) -> Workload:
    """One of six dense shapes (TP as per-GPU shards), lognormal contexts
    (median 1024, max 32768), batch U{1..256}; bf16 16->128->128->1 heads."""
    tr = trace_c2(shape_idx).slice(step_lo, step_hi)
    return _wl(f"c2-{DENSE_SHAPES[shape_idx].name}", [tr], specs_datasheet(),
               make_heads(16, 128, "bf16"), {"steps": (step_lo, step_hi)})


def config3(step_lo=0, step_hi=C3_STEPS) -> Workload:
    """Mixtral-like MoE (8 experts, top-2), Dirichlet(0.5) routing per step
    and layer; bf16 16->128->128->1 heads."""
    full = trace_c3()
    tr = full.slice(step_lo, step_hi)
    tr.experts = route_tokens(full, SEED + 3, step_lo, step_hi)
    return _wl("c3-mixtral", [tr], specs_datasheet(), make_heads(16, 128, "bf16"),
               {"steps": (step_lo, step_hi)})


def config4(n_specs=256, grid_steps=C4_GRID_STEPS, c1_steps=C1_STEPS) -> Workload:
    """Capacity-planning grid: the config-1 trace followed by the first
    grid_steps steps of the config-2 S2 trace, against n_specs hypothetical
    GPUs; bf16 16->128->128->1 heads."""
    traces = [trace_c1().slice(0, c1_steps), trace_c2(1).slice(0, grid_steps)]
    return _wl("c4-grid", traces, specs_grid(n_specs, SEED + 4),
               make_heads(16, 128, "bf16"), {"n_specs": n_specs})


def config5(step_lo=0, step_hi=C5_STEPS) -> Workload:
    """70B shape, Pareto contexts (alpha 1.2, min 512, max 131072) with a
    prefix-cache hit fraction U[0, 0.9] on prefill chunks; bf16
    32->256->256->1 heads."""
    tr = trace_c5().slice(step_lo, step_hi)
    return _wl("c5-70b-prefix", [tr], specs_datasheet(), make_heads(32, 256, "bf16"),
               {"steps": (step_lo, step_hi)})


# --------------------------------------------------------------------------
# serving requests for the simulator (synthetic arrival process)
# --------------------------------------------------------------------------
REQ_SEED = SEED + 200


def make_requests(n: int, rate: float, seed: int = REQ_SEED, prompt_median=512, prompt_sigma=1.0,
                  prompt_max=8192, output_median=128, output_sigma=0.8, output_max=2048,
                  groups=8, group_frac=0.5, prefix_lo=256, prefix_hi=2048) -> dict:
    """n requests from a Poisson process of `rate` requests/s; prompt and
    output lengths lognormal (clipped to [1, max]); a fraction group_frac of
    the requests carries one of `groups` shared system prompts, whose
    lengths are U{prefix_lo..prefix_hi} (a request's prompt is at least its
    prefix).  Stand-in for the paper's production conversation trace, which
    is not available."""
    rng = np.random.Generator(np.random.PCG64(seed))
    arrival = np.cumsum(rng.exponential(1.0 / rate, n))
    prompt = np.clip(np.floor(rng.lognormal(np.log(prompt_median), prompt_sigma, n)), 1, prompt_max)
    output = np.clip(np.floor(rng.lognormal(np.log(output_median), output_sigma, n)), 1, output_max)
    plen = rng.integers(prefix_lo, prefix_hi, groups + 1, endpoint=True)
    group = np.where(rng.random(n) < group_frac, rng.integers(1, groups + 1, n), 0)
    prefix = np.where(group > 0, plen[group], 0)
    prompt = np.maximum(prompt, prefix)
    return {"arrival": arrival, "prompt": prompt.astype(np.uint32), "output": output.astype(np.uint32),
            "group": group.astype(np.uint32), "prefix": prefix.astype(np.uint32)}
