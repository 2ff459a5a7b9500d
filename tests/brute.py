"""Brute-force counters for tiny inputs: they enumerate the work a kernel
does instead of using a closed form, so they pin the oracle's formulas.
Plain Python loops; only usable on very small shapes."""
from __future__ import annotations

import math


def gemm_work(M, N, K, dt):
    """Enumerate C[i, j] += A[i, l] B[l, j]; count MACs and distinct touched
    elements of A, B and C."""
    macs = 0
    a_el, b_el, c_el = set(), set(), set()
    for i in range(M):
        for j in range(N):
            for l in range(K):
                macs += 1
                a_el.add((i, l))
                b_el.add((l, j))
            c_el.add((i, j))
    return 2 * macs, dt * (len(a_el) + len(b_el) + len(c_el))


def tiles_2d(M, N, tile):
    """Distinct (row-tile, col-tile) pairs that own at least one output."""
    return len({(i // tile, j // tile) for i in range(M) for j in range(N)})


def attention_work(reqs, H, Hkv, d, dt):
    """reqs: list of (q, h).  Query token i of a request sits at position
    h + i and attends to keys 0 .. h + i.  Per head and (query, key) pair:
    d MACs for q.k and d MACs for p.v.  Bytes: Q read and O written (H d per
    query token), K and V read (Hkv d per cached or new token)."""
    pairs = 0
    q_el, o_el, k_el, v_el = set(), set(), set(), set()
    tiles = set()
    for r, (q, h) in enumerate(reqs):
        for i in range(q):
            pos = h + i
            tiles.add((r, i // 128))
            for key in range(pos + 1):
                pairs += 1
            for hh in range(H):
                for c in range(d):
                    q_el.add((r, i, hh, c))
                    o_el.add((r, i, hh, c))
        for pos in range(h + q):
            for hh in range(Hkv):
                for c in range(d):
                    k_el.add((r, pos, hh, c))
                    v_el.add((r, pos, hh, c))
    flops = 2 * (2 * d * pairs) * H
    nbytes = dt * (len(q_el) + len(o_el) + len(k_el) + len(v_el))
    return flops, nbytes, H * len(tiles), pairs


def dispatch_waves(B, N):
    """Round-robin dispatch of B equal blocks onto N SMs; returns the number
    of waves and the idle SM slots in the last wave."""
    if B == 0:
        return 0, 0
    busy_until = [0] * N
    waves = 0
    for blk in range(B):
        sm = min(range(N), key=lambda s: (busy_until[s], s))
        busy_until[sm] += 1
        waves = max(waves, busy_until[sm])
    last = sum(1 for s in range(N) if busy_until[s] == waves)
    return waves, N - last


def ring_allreduce_bytes(P, S):
    """Bytes each rank sends in a ring all-reduce of S bytes over P ranks:
    P - 1 reduce-scatter steps and P - 1 all-gather steps, one chunk of S/P
    per step."""
    if P == 1:
        return 0.0
    chunk = S / P
    sent = [0.0] * P
    for _phase in range(2):
        for _step in range(P - 1):
            for r in range(P):
                sent[r] += chunk
    assert all(abs(s - sent[0]) < 1e-9 * max(1.0, S) for s in sent)
    return sent[0]


def mlp_scalar(x, w1, w2, b2, w3, b3, rnd=lambda v: v):
    """z for one feature vector, with explicit [out][in] indexing; rnd
    rounds the inputs of the two matrix layers (x and h1), the last layer
    takes relu(h2) as it is."""
    H, I = len(w1), len(x)
    xr = [rnd(v) for v in x]
    h1 = []
    for o in range(H):
        s = 0.0
        for i in range(I):
            s += w1[o][i] * xr[i]
        h1.append(rnd(max(s, 0.0)))
    h2 = []
    for o in range(H):
        s = b2[o]
        for i in range(H):
            s += w2[o][i] * h1[i]
        h2.append(max(s, 0.0))
    z = b3
    for i in range(H):
        z += w3[i] * h2[i]
    return z


def bf16_scalar(v):
    """Round to 8 significant bits, ties to even, by exhaustive search over
    the two neighbouring bfloat16 values."""
    if v == 0.0:
        return 0.0
    e = math.floor(math.log2(abs(v)))
    # guard log2 rounding at exact powers of two
    while abs(v) >= 2.0 ** (e + 1):
        e += 1
    while abs(v) < 2.0 ** e:
        e -= 1
    ulp = 2.0 ** (e - 7)
    lo = math.floor(abs(v) / ulp) * ulp
    hi = lo + ulp
    d_lo, d_hi = abs(v) - lo, hi - abs(v)
    if d_lo < d_hi:
        r = lo
    elif d_hi < d_lo:
        r = hi
    else:
        r = lo if int(round(lo / ulp)) % 2 == 0 else hi
    return math.copysign(r, v)


# ---------------------------------------------------------------------------
# elementwise and memory kernels: each kernel written out as the loop it runs
# over its elements, counting the arithmetic operations of every element's
# expression and collecting the distinct elements it reads and writes, and
# the thread blocks its grid mapping touches.  Returns (F, Bt, B).

def rmsnorm_work(T, D, dt):
    """y[t, i] = x[t, i] * rsqrt(mean_i x[t, i]^2) * w[i], one block per token
    row: per element a square and an accumulate (the mean), the scale by the
    row's reciprocal root and the weight multiply."""
    ops = 0
    x_rd, w_rd, y_wr, blocks = set(), set(), set(), set()
    for t in range(T):
        for i in range(D):                       # pass 1: sum of squares
            ops += 2                             # x * x, acc += .
            x_rd.add((t, i))
        for i in range(D):                       # pass 2: normalise, weight
            ops += 2                             # * r, * w[i]
            x_rd.add((t, i))
            w_rd.add(i)
            y_wr.add((t, i))
        blocks.add(t)
    return ops, dt * (len(x_rd) + len(w_rd) + len(y_wr)), len(blocks)


def rope_work(T, heads, d, dt):
    """x'[t, h, c] = x[t, h, c] cos[t, c] + rot(x)[t, h, c] sin[t, c] in place
    over the rotated heads, one block per token: per element two multiplies
    and one add; the position's cos/sin table holds d values (cos for one half
    of the rotation pairs' slots, sin for the other)."""
    ops = 0
    x_rd, x_wr, tab, blocks = set(), set(), set(), set()
    for t in range(T):
        for h in range(heads):
            for c in range(d):
                ops += 3
                x_rd.add((t, h, c))
                x_wr.add((t, h, c))
                tab.add((t, c))
        blocks.add(t)
    return ops, dt * (len(x_rd) + len(x_wr) + len(tab)), len(blocks)


def silu_mul_work(T, I, dt, block=1024):
    """out[t, i] = g / (1 + exp(-g)) * u with g = gate[t, i], u = up[t, i]:
    negate, exponentiate, add one, divide, multiply by u (five operations);
    flat blocks of `block` elements."""
    ops = 0
    g_rd, u_rd, o_wr, blocks = set(), set(), set(), set()
    for t in range(T):
        for i in range(I):
            ops += 5
            g_rd.add((t, i))
            u_rd.add((t, i))
            o_wr.add((t, i))
            blocks.add((t * I + i) // block)
    return ops, dt * (len(g_rd) + len(u_rd) + len(o_wr)), len(blocks)


def kv_write_work(T, Hkv, d, dt):
    """cache_k[slot(t), h, c] = k[t, h, c] and the same for v: a copy, no
    arithmetic; one block per token."""
    k_rd, v_rd, ck_wr, cv_wr, blocks = set(), set(), set(), set(), set()
    for t in range(T):
        for h in range(Hkv):
            for c in range(d):
                k_rd.add((t, h, c))
                v_rd.add((t, h, c))
                ck_wr.add((t, h, c))
                cv_wr.add((t, h, c))
        blocks.add(t)
    return 0, dt * (len(k_rd) + len(v_rd) + len(ck_wr) + len(cv_wr)), len(blocks)


def embed_work(T, D, dt, id_bytes=4):
    """out[t, i] = table[id[t], i]: read the token's id (a 4-byte integer),
    gather its table row and write the output row; no arithmetic; one block
    per token.  Token ids are taken distinct (the gathered rows do not
    repeat: the bytes a kernel moves, not a cache's hits)."""
    ids, tab, out, blocks = set(), set(), set(), set()
    for t in range(T):
        ids.add(t)
        for i in range(D):
            tab.add((t, i))                      # row id[t] = t (distinct ids)
            out.add((t, i))
        blocks.add(t)
    return 0, id_bytes * len(ids) + dt * (len(tab) + len(out)), len(blocks)
