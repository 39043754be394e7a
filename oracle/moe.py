"""The routed mixture-of-experts layer, written out in fp64 (numpy).

Test infrastructure: see the package docstring.

The layer (paper: System and model context / Execution structure and
Fig. architecture): a router picks the top-k routed experts of every token;
each picked expert runs gate/up -> activation -> down on FP4 block-scaled
weights; an always-on shared expert runs beside them; the partial outputs join
in a sum. The steps, in order, each cite what fixes them:

1. ``router_logits``   -- logits = x . Wr^T (the "Router" box of the figure).
2. ``route_topk``      -- k largest logits, ties to the lower expert id,
                          selected positions in a fixed order (Correctness
                          recovery / Later numerical and integration repairs:
                          membership ties broken by logical id, fixed order;
                          Remaining risks and next steps, item 2); softmax
                          weights renormalised over the k picks.
3. ``permute``         -- stable token->expert grouping of the assignments (the
                          expert sorter of Prefill optimization / From
                          per-assignment scalar work to CDNA2 MFMA, item 8).
4. ``mx_quantize`` (x) -- per-32 activation quantisation before gate/up
                          (Historical TP4 decode optimization / Parallel
                          decomposition; module ``mx``).
5. ``expert_ffn``      -- gate/up projection, SwiGLU, per-32 re-quantisation of
                          the intermediate, down projection (Historical
                          down-consumer pilot: the intermediate is quantised
                          per 32 again before the down projection).
6. ``combine``         -- every (token, slot) keeps its own partial and the
                          weighted partials are summed in a fixed order
                          (Current TP8 native-AR results / Accepted large-prefill
                          configuration: unique-slot stores and a fixed-order
                          FP32 top-k reduction). The oracle sums in fp64 and
                          rounds once to bf16.

The BF16 contract (``fmt='bf16'``, the paper's accepted large-prefill
arithmetic: Large-M CK and the meaning of the earlier 6.42k result; Accepted
large-prefill configuration) replaces steps 4 and 5's per-32 quantisation:
x enters unquantised and h is rounded once to bf16 before the down
projection; weights, partials and combine are unchanged.

Readings where the paper is silent: softmax scoring
with renormalisation over the k picks and routed scale 1; SwiGLU
h = silu(gate) * up; rows 0..I-1 of W13 are gate, I..2I-1 are up; the shared
expert is expert index E with weight 1, added after the routed slots.

Pins for every function are in tests/test_oracle_*.py.
"""
from __future__ import annotations

import numpy as np

from . import mx


def router_logits(x_bits, wr_bits) -> np.ndarray:
    """logits[t, e] = sum_h x[t, h] * Wr[e, h] in fp64 (x, Wr are bf16 bits)."""
    return mx.bf16_to_f64(x_bits) @ mx.bf16_to_f64(wr_bits).T


def route_topk(logits, k: int, n_shared: int = 0):
    """Top-k routing of every token.

    ``logits`` [T, E] (fp32 values are widened exactly to fp64). Experts are
    ordered by (logit descending, expert id ascending); the first k are kept in
    that order. Weights are the softmax renormalised over the k picks:
    w_j = exp(l_j - l_0) / sum_i exp(l_i - l_0). With ``n_shared`` = 1 an extra
    column holds expert id E with weight 1.

    Returns (ids int32 [T, k + n_shared], w fp64 [T, k + n_shared]).
    """
    lg = np.asarray(logits).astype(np.float64)
    t, e = lg.shape
    if not 1 <= k <= e:
        raise ValueError("need 1 <= k <= E")
    # a stable sort of -logit keeps equal logits in ascending id order
    order = np.argsort(-lg, axis=1, kind="stable")[:, :k]
    sel = np.take_along_axis(lg, order, axis=1)
    ex = np.exp(sel - sel[:, :1])
    w = ex / ex.sum(axis=1, keepdims=True)
    ids = order.astype(np.int32)
    if n_shared:
        ids = np.concatenate([ids, np.full((t, 1), e, np.int32)], axis=1)
        w = np.concatenate([w, np.ones((t, 1))], axis=1)
    return ids, w


def route_topk_ex(logits, k: int, n_shared: int = 0, score: str = "softmax", bias=None,
                  n_group: int = 1, topk_group: int = 1, renorm: bool = True,
                  scale: float = 1.0):
    """Routing variants (readings: the paper fixes top-k and a deterministic
    order but not the scoring; these follow DeepSeek's published router).

    Scores s: softmax over the E logits, or the logistic sigmoid of each.
    Selection key: s + bias (bias steers selection only), or the logit itself
    without a bias (same order as s). With ``n_group`` > 1 the experts form
    n_group groups of E / n_group consecutive ids; a group scores the sum of
    its two largest values of s + bias (its single value for one-expert
    groups); the ``topk_group`` best groups (ties to the lower group) stay and
    the other experts are excluded. Picks: the k largest keys, ordered by (key
    descending, id ascending). Weights: s of the picks, divided by their sum
    if ``renorm``, times ``scale``. The shared column is as in route_topk.

    Returns (ids int32 [T, k + n_shared], w fp64 [T, k + n_shared]).
    """
    lg = np.asarray(logits).astype(np.float64)
    t, e = lg.shape
    if not 1 <= k <= e:
        raise ValueError("need 1 <= k <= E")
    if n_group < 1 or e % n_group or not 1 <= topk_group <= n_group:
        raise ValueError("bad grouping")
    if score == "softmax":
        z = np.exp(lg - lg.max(axis=1, keepdims=True))
        s = z / z.sum(axis=1, keepdims=True)
    elif score == "sigmoid":
        s = 1.0 / (1.0 + np.exp(-lg))
    else:
        raise ValueError(f"score: {score!r}")
    b = None if bias is None else np.asarray(bias, np.float64)
    key = lg.copy() if b is None else s + b
    if n_group > 1:
        gs = e // n_group
        v = (s if b is None else s + b).reshape(t, n_group, gs)
        top = -np.sort(-v, axis=2)
        gscore = top[:, :, 0] if gs == 1 else top[:, :, 0] + top[:, :, 1]
        gkeep = np.argsort(-gscore, axis=1, kind="stable")[:, :topk_group]
        allowed = np.zeros((t, n_group), bool)
        np.put_along_axis(allowed, gkeep, True, axis=1)
        key = np.where(np.repeat(allowed, gs, axis=1), key, -np.inf)
    order = np.argsort(-key, axis=1, kind="stable")[:, :k]
    w = np.take_along_axis(s, order, axis=1)
    if renorm:
        w = w / w.sum(axis=1, keepdims=True)
    w = w * scale
    ids = order.astype(np.int32)
    if n_shared:
        ids = np.concatenate([ids, np.full((t, 1), e, np.int32)], axis=1)
        w = np.concatenate([w, np.ones((t, 1))], axis=1)
    return ids, w


def permute(ids, n_experts_total: int):
    """Stable counting sort of the assignments a = t*k_total + j by expert id.

    Returns counts [NE], offsets [NE+1] (exclusive prefix sum), sorted [A]
    (assignments grouped by expert, increasing a inside each expert) and its
    inverse pos [A] (sorted[pos[a]] == a); all int32.
    """
    flat = np.asarray(ids).reshape(-1).astype(np.int64)
    if flat.size and (flat.min() < 0 or flat.max() >= n_experts_total):
        raise ValueError("expert id out of range")
    counts = np.bincount(flat, minlength=n_experts_total)
    offsets = np.zeros(n_experts_total + 1, np.int64)
    offsets[1:] = np.cumsum(counts)
    srt = np.argsort(flat, kind="stable")
    pos = np.empty_like(srt)
    pos[srt] = np.arange(flat.size)
    return (counts.astype(np.int32), offsets.astype(np.int32),
            srt.astype(np.int32), pos.astype(np.int32))


def swiglu(g, u) -> np.ndarray:
    """h = silu(g) * u = g * u / (1 + exp(-g)) in fp64."""
    with np.errstate(over="ignore"):
        return g * u / (1.0 + np.exp(-g))


def expert_ffn(a, w13_packed, w13_scales, w2_packed, w2_scales, fmt):
    """One expert on its rows.

    a: fp64 [M, H] activations as the expert sees them (already dequantised
    from their MX codes when ``fmt`` is set). W13 [2I, H] holds gate rows
    0..I-1 then up rows I..2I-1; W2 is [H, I]. With ``fmt`` set, the
    intermediate h is quantised per 32 along I before the down projection;
    ``fmt`` None skips that (the unquantised reading used for reporting only).

    ``fmt`` 'bf16' is the BF16 contract (Large-M CK and the meaning of the
    earlier 6.42k result; Historical down-consumer pilot): no per-32
    quantisation; h is rounded once to bf16 (nearest, ties to even) and the
    down projection consumes that rounded intermediate.

    Returns dict(g, u, h, hq, hs, hd, p): gate, up, intermediate, its codes and
    scale bytes (None without fmt; for 'bf16' hq holds the bf16 bits and hs
    is None), the intermediate the down projection consumes, and the partial
    outputs p [M, H].
    """
    w13 = mx.dequant_fp4(w13_packed, w13_scales)
    w2 = mx.dequant_fp4(w2_packed, w2_scales)
    i = w13.shape[0] // 2
    g = a @ w13[:i].T
    u = a @ w13[i:].T
    h = swiglu(g, u)
    if fmt is None:
        hq = hs = None
        hd = h
    elif fmt == "bf16":
        hq, hs = mx.f64_to_bf16(h), None
        hd = mx.bf16_to_f64(hq)
    else:
        hq, hs = mx.mx_quantize(h, fmt)
        hd = mx.mx_dequantize(hq, hs, fmt)
    p = hd @ w2.T
    return dict(g=g, u=u, h=h, hq=hq, hs=hs, hd=hd, p=p)


def combine(p_slots, w) -> np.ndarray:
    """out[t] = sum_j w[t, j] * P[t, j] in fp64 (P [T, k_total, H], w [T, k_total])."""
    return np.einsum("tj,tjh->th", np.asarray(w, np.float64), p_slots)


def layer(x_bits, w13, w13s, w2, w2s, *, k, n_shared=0, logits=None, wr_bits=None,
          fmt="e4m3", tokens=None, keep=False):
    """The whole layer for the tokens in ``tokens`` (default: all).

    x_bits uint16 [T, H]; w13/w13s/w2/w2s are indexable by expert (arrays
    [NE, ...] or any object whose ``[e]`` returns that expert's arrays), with
    NE = E + n_shared and the shared expert at index E. Give either fp32
    ``logits`` [T, E] or bf16 router weights ``wr_bits`` [E, H].
    ``fmt``: activation element format ('e4m3', 'e2m3', 'e2m1'), 'bf16' for
    the BF16 contract (x exact, h rounded to bf16; see expert_ffn) or None
    for no activation quantisation.

    Returns a dict with ``out`` (bf16 bits [len(tokens), H]), ``out_f64`` and
    the routing and permutation arrays for all T tokens; with ``keep`` also the
    quantised x of the subset, per expert the expert_ffn intermediates of its
    rows (``rows`` are positions in the sorted order), and the partials
    ``p_slots`` [len(tokens), k_total, H].
    """
    t_all, hdim = np.asarray(x_bits).shape
    if logits is None:
        if wr_bits is None:
            raise ValueError("need logits or router weights")
        lg64 = router_logits(x_bits, wr_bits)
        logits = lg64.astype(np.float32)
    else:
        lg64 = None
    e = np.asarray(logits).shape[1]
    ids, w = route_topk(logits, k, n_shared)
    k_total = k + n_shared
    ne = e + n_shared
    counts, offsets, srt, pos = permute(ids, ne)

    tokens = np.arange(t_all) if tokens is None else np.asarray(tokens, np.int64)
    slot_of = np.full(t_all, -1, np.int64)          # token -> row of the subset
    slot_of[tokens] = np.arange(tokens.size)

    # activations are quantised per token row, so the subset is exact
    x64 = mx.bf16_to_f64(np.asarray(x_bits)[tokens])
    if fmt is None or fmt == "bf16":
        xq = xs = None
        xd = x64
    else:
        xq, xs = mx.mx_quantize(x64, fmt)
        xd = mx.mx_dequantize(xq, xs, fmt)

    p_slots = np.zeros((tokens.size, k_total, hdim))
    per_expert = {}
    for ex in range(ne):
        rows = np.arange(offsets[ex], offsets[ex + 1])
        a_idx = srt[rows].astype(np.int64)
        sub = slot_of[a_idx // k_total]
        sel = sub >= 0
        if not sel.any():
            continue
        rows, a_idx, sub = rows[sel], a_idx[sel], sub[sel]
        r = expert_ffn(xd[sub], w13[ex], w13s[ex], w2[ex], w2s[ex], fmt)
        p_slots[sub, a_idx % k_total] = r["p"]
        if keep:
            r["rows"] = rows
            per_expert[ex] = r
    out64 = combine(p_slots, w[tokens])
    res = dict(out=mx.f64_to_bf16(out64), out_f64=out64, ids=ids, w=w, counts=counts,
               offsets=offsets, sorted=srt, pos=pos, logits=logits, logits_f64=lg64,
               tokens=tokens)
    if keep:
        res.update(xq=xq, xs=xs, per_expert=per_expert, p_slots=p_slots)
    return res
