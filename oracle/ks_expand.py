"""CPU oracle of the batch -> dispatched-kernel expansion.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this module; only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the HIP library (nor with
the record builder of ``workload.gen``): it reads the seeded batch
descriptors and enumerates, with plain Python loops, the kernels each step
dispatches.

What it computes, and where the paper states it (KernelSight-LM):

* Sec. 4.1 (system overview): for every step the scheduler hands the
  predictor a batch descriptor (decode tokens, prefill-chunk lengths,
  per-request KV lengths) and the predictor prices each kernel the step
  dispatches.  Here the descriptor is the step's request list (q_r query
  tokens over h_r cached tokens), a prefill flag and, for a mixture of
  experts, the routed token copies of every (layer, expert).
* Sec. 5.8 (mixed prefill-decode steps): the dense GEMMs, norms and
  activations run over the step's concatenated tokens T = sum q_r, and
  attention prices every request of the step (one attention kernel per
  layer whose family follows the step's prefill flag).
* Sec. 5.7: the step's GPU body is L t_layer + t_lm_head + t_embed: one
  embedding and one LM head per step, L homogeneous layers.  The
  homogeneous expansion keeps that form literally: a kernel that is the
  same in every layer is one record standing for L dispatches
  (multiplicity L); kernels that differ between layers (a mixture of
  experts' grouped GEMMs, whose per-expert rows follow each layer's
  routing) stay one record per layer.

Readings (the paper names the kernel kinds but not every shape; the
library's record layout follows the same readings):

* per layer, in dispatch order: QKV GEMM (T, (H + 2 Hkv) d, D); RoPE
  (T, H + Hkv, d); the KV-cache write (T, Hkv, d) if the model writes one;
  attention (H, d, Hkv over the step's requests); O GEMM (T, D, H d); two
  RMSNorms (T, D); then either the dense MLP (gate/up GEMM (T, 2I, D),
  SiLU x mul (T, I), down GEMM (T, D, I)) or the mixture of experts
  (router GEMM (T, E, D), grouped gate/up (2 I_e, D over E experts), SiLU x
  mul (k T, I_e), grouped down (D, I_e over E experts));
* per step: the embedding (T, D) first and the LM head (R, V, D) last, R
  the step's request count (one logit row per request);
* tensor parallelism P shards the shapes: H = Hq / P, Hkv = ceil(Hkv / P)
  (KV heads replicate when there are fewer than P), I = FFN / P,
  I_e = FFN_e / P, V / P;
* a grouped GEMM record of layer l in step j points at that layer's E
  routed row counts: b = (j L + l) E in the [step][layer][expert] routing
  array, a = E;
* the host launch count n of Eq. 4 is L for a step with a prefill chunk
  (run eagerly, one launch charge per layer, Sec. 5.8) and 0 otherwise
  (a captured decode graph);
* records are family-major and, within a family, ordered by step, then
  layer, then dispatch order.
"""
from __future__ import annotations

import numpy as np

from workload.gen import (NFAM, GEMM, LM_HEAD, GROUPED_GEMM, ATTN_PREFILL,
                          ATTN_DECODE, RMSNORM, ROPE, SILU_MUL, KV_WRITE, EMBED)

FIELDS = ("step", "m", "n", "k", "a", "b", "mult")


def shard(model):
    """Per-GPU sizes under tensor parallelism P (whole-model sizes / P; KV
    heads are replicated when the model has fewer than P of them)."""
    P = int(model.tp)
    return {
        "D": int(model.hidden),
        "L": int(model.layers),
        "d": int(model.head_dim),
        "H": int(model.q_heads) // P,
        "Hkv": -(-int(model.kv_heads) // P),
        "I": int(model.ffn) // P,
        "Ie": int(model.expert_ffn) // P,
        "V": int(model.vocab) // P,
        "E": int(model.experts),
        "topk": int(model.top_k),
        "P": P,
    }


def layer_kernels(model, T, attn_family, route_base):
    """The kernels one decoder layer dispatches for a step of T tokens, in
    dispatch order, as (family, m, n, k, a, b) tuples.  route_base: offset of
    this layer's E routed row counts (mixture of experts only)."""
    s = shard(model)
    D, d, H, Hkv = s["D"], s["d"], s["H"], s["Hkv"]
    ks = [(GEMM, T, (H + 2 * Hkv) * d, D, 0, 0),          # QKV projection
          (ROPE, T, H + Hkv, d, 0, 0)]                     # rotary on q and k
    if model.kv_write:
        ks.append((KV_WRITE, T, Hkv, d, 0, 0))             # KV-cache write
    ks += [(attn_family, 0, H, d, Hkv, 0),                 # attention over the requests
           (GEMM, T, D, H * d, 0, 0),                      # O projection
           (RMSNORM, T, D, 0, 0, 0),
           (RMSNORM, T, D, 0, 0, 0)]
    if s["E"] == 0:
        I = s["I"]
        ks += [(GEMM, T, 2 * I, D, 0, 0),                  # gate/up
               (SILU_MUL, T, I, 0, 0, 0),
               (GEMM, T, D, I, 0, 0)]                      # down
    else:
        E, Ie = s["E"], s["Ie"]
        ks += [(GEMM, T, E, D, 0, 0),                      # router
               (GROUPED_GEMM, 0, 2 * Ie, D, E, route_base),
               (SILU_MUL, s["topk"] * T, Ie, 0, 0, 0),
               (GROUPED_GEMM, 0, D, Ie, E, route_base)]
    return ks


def step_kernels(model, j, T, R, prefill):
    """Every kernel step j dispatches, in dispatch order, as (family, layer,
    m, n, k, a, b); layer is -1 for the per-step kernels."""
    s = shard(model)
    L, E = s["L"], s["E"]
    attn = ATTN_PREFILL if prefill else ATTN_DECODE
    out = [(EMBED, -1, T, s["D"], 0, 0, 0)]
    for layer in range(L):
        for (f, m, n, k, a, b) in layer_kernels(model, T, attn, (j * L + layer) * E):
            out.append((f, layer, m, n, k, a, b))
    out.append((LM_HEAD, -1, R, s["V"], s["D"], 0, 0))
    return out


def expand(model, req_off, req_q, prefill, homogeneous=False):
    """Records of every kernel of steps 0 .. S-1 (S = len(prefill)).

    Returns a dict: fam_off (int64 [NFAM+1]), the record fields step, m, n,
    k, a, b, mult (int64 [n_rows], family-major), and the per-step arrays
    layers, hidden, tp, n_launch (int64 [S]).  With homogeneous=True the
    L records of a kernel that is identical in every layer of a step become
    one record of multiplicity L (Sec. 5.7); otherwise every dispatched
    kernel is one record of multiplicity 1."""
    req_off = [int(v) for v in req_off]
    q = [int(v) for v in req_q]
    S = len(prefill)
    assert len(req_off) == S + 1
    s = shard(model)
    L = s["L"]
    per_fam = [[] for _ in range(NFAM)]
    for j in range(S):
        T = sum(q[req_off[j]:req_off[j + 1]])
        R = req_off[j + 1] - req_off[j]
        ks = step_kernels(model, j, T, R, bool(prefill[j]))
        if not homogeneous:
            for (f, layer, m, n, k, a, b) in ks:
                per_fam[f].append((j, m, n, k, a, b, 1))
            continue
        # group the per-layer kernels by their position in the layer; a
        # position whose L records are all equal collapses into one
        per_layer = [kk for kk in ks if kk[1] >= 0]
        n_pos = len(per_layer) // L
        collapsed = {}
        for p in range(n_pos):
            recs = [per_layer[layer * n_pos + p] for layer in range(L)]
            collapsed[p] = all(r[0:1] + r[2:] == recs[0][0:1] + recs[0][2:] for r in recs)
        for (f, layer, m, n, k, a, b) in ks:
            if layer < 0:
                per_fam[f].append((j, m, n, k, a, b, 1))
        # family order within a step: per family, collapsed positions in
        # layer order, then the per-layer records by (layer, position)
        for p in range(n_pos):
            if collapsed[p]:
                f, _, m, n, k, a, b = per_layer[p]
                per_fam[f].append((j, m, n, k, a, b, L))
        for layer in range(L):
            for p in range(n_pos):
                if not collapsed[p]:
                    f, _, m, n, k, a, b = per_layer[layer * n_pos + p]
                    per_fam[f].append((j, m, n, k, a, b, 1))
    out = {"fam_off": np.zeros(NFAM + 1, np.int64)}
    cols = {name: [] for name in FIELDS}
    for f in range(NFAM):
        # the step loop appended each family's records by step, then layer,
        # then dispatch order
        recs = per_fam[f]
        for r in recs:
            for name, v in zip(FIELDS, r):
                cols[name].append(v)
        out["fam_off"][f + 1] = out["fam_off"][f] + len(recs)
    for name in FIELDS:
        out[name] = np.array(cols[name], np.int64)
    out["layers"] = np.full(S, L, np.int64)
    out["hidden"] = np.full(S, s["D"], np.int64)
    out["tp"] = np.full(S, s["P"], np.int64)
    out["n_launch"] = np.array([L if p else 0 for p in prefill], np.int64)
    return out


def family_counts(model, n_steps, n_prefill, homogeneous=False):
    """Records per family, in closed form: per step one embedding and one LM
    head; per layer the kernels above (attention in the family of the
    step's prefill flag).  Homogeneous: each layer-identical kernel once."""
    s = shard(model)
    L, E = s["L"], s["E"]
    rep = 1 if homogeneous else L
    c = np.zeros(NFAM, np.int64)
    c[EMBED] = c[LM_HEAD] = n_steps
    c[GEMM] = (3 if E else 4) * rep * n_steps
    c[ROPE] = rep * n_steps
    c[KV_WRITE] = rep * n_steps if model.kv_write else 0
    c[RMSNORM] = 2 * rep * n_steps
    c[SILU_MUL] = rep * n_steps
    c[GROUPED_GEMM] = 2 * L * n_steps if E else 0
    c[ATTN_PREFILL] = rep * n_prefill
    c[ATTN_DECODE] = rep * (n_steps - n_prefill)
    return c
