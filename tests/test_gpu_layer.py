"""GPU parity of the whole layer (route -> permute -> grouped GEMM -> combine)
against the fp64 oracle, through the C ABI, in the launch configuration the
benchmark times.

Bar (bf16 output): max over tokens of max_h |y - y*| / max_h |y*| <= 1e-2,
against the oracle with the same activation quantisation, for every named
workload and every MXFP8 case; route ids and the permutation bit-exact;
activation codes bit-exact; stage 2 alone (from the GPU's own h codes) at the
same bar; ten repeated runs bit-identical.

On the small synthetic shapes (few h values per token) one h code that the
GPU's fp32 h puts on the other side of a rounding midpoint than the
oracle's fp64 h (a valid rounding: check_hq_codes bounds it to one grid step)
can move a token's row by more than 1e-2. There a token may miss the bar
against the oracle only if one of its rows holds such a code, and it must
then meet the bar against the oracle evaluated on the GPU's h codes (the
other correct result). The named workloads get no such allowance."""
import numpy as np
import pytest
import torch

import synth
from oracle import moe as omoe
from oracle import mx
from tests import gpu_common as gc
from tests.gpu_common import log

pytestmark = pytest.mark.gpu

TOL = 1e-2


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


def run_layer(m, cfg, x_dev, weights, logits=None, wr=None, fmt="e4m3", fused=False):
    """The default (unfused) path is the one the benchmark times."""
    layer = m.MoELayer(cfg.T, cfg.H, cfg.E, cfg.k, cfg.I, cfg.n_shared, fmt, fused=fused)
    lg = None if logits is None else torch.from_numpy(logits).cuda()
    out = layer.forward(x_dev, weights, logits=lg, w_router=wr)
    torch.cuda.synchronize()
    return layer, out


# Element grid of each MX activation format: (largest value, exponent of the
# smallest normal, mantissa bits).
GRID = {"e4m3": (448.0, -6, 3), "e2m3": (7.5, 0, 3), "e2m1": (6.0, 0, 1)}


def gpu_hq_rows(layer, cfg, rows, fmt):
    """The GPU's h codes (one code per element) and scale bytes of sorted rows
    ``rows``, copied from the grouped GEMM's workspace."""
    rb = m_ws_bytes(cfg.I, fmt)
    hq = layer.workspace_view(2)[: cfg.A * rb].view(cfg.A, rb)
    hs = layer.workspace_view(3)[: cfg.A * cfg.I // 32].view(cfg.A, cfg.I // 32)
    idx = torch.from_numpy(np.asarray(rows, np.int64)).cuda()
    q = gc.ws_codes(hq.index_select(0, idx).cpu().numpy(), fmt)
    return q, hs.index_select(0, idx).cpu().numpy()


def m_ws_bytes(K, fmt):
    """Workspace bytes of K activation codes (e2m3 blocks in 32-byte slots)."""
    return K * {"e4m3": 8, "e2m3": 8, "e2m1": 4}[fmt] // 8


def check_hq_codes(layer, cfg, ref, fmt):
    """The h codes the GPU fed to the down projection against the oracle's.

    The GPU's h carries the fp32 / matrix-core accumulation error of G and U,
    which is relative to the largest products, not to h itself: an element
    can take a neighbouring grid value (when it sits near a rounding
    midpoint), and elements far below their block's maximum can move a few
    subnormal steps. Bound, on dequantised values: |v_gpu - v_oracle| <= one
    grid step at the larger magnitude + 1e-4 of the block's scaled maximum
    (the format's largest value times the larger block scale). Differing codes
    must be rare (at most 1e-3 of the codes).

    Block scales follow the block maximum: when the oracle's maximum sits
    within a relative 1e-4 of the boundary maxval * 2^X between two scales,
    the GPU's fp32 maximum may fall on the other side, and its scale is one
    off. Only such blocks may differ in scale, and only rarely (at most 1e-3
    of the blocks)."""
    maxval, emin, mbits = GRID[fmt]
    flips = total = moved = blocks = 0
    flipped = set()  # sorted rows holding a differing code
    for r in ref["per_expert"].values():
        g, sg = gpu_hq_rows(layer, cfg, r["rows"], fmt)
        g, sg = g.astype(np.int64), sg.astype(np.int64)
        o, so = r["hq"].astype(np.int64), r["hs"].astype(np.int64)
        ds = sg != so
        if ds.any():
            amax = np.abs(r["h"]).reshape(len(r["rows"]), -1, 32).max(2)
            bound = maxval * np.ldexp(1.0, np.minimum(sg, so) - 127)
            near = (np.abs(sg - so) == 1) & (np.abs(amax - bound) <= 1e-4 * bound)
            assert (near | ~ds).all(), "h block scales differ away from a scale boundary"
        moved += int(ds.sum())
        blocks += ds.size
        eg = np.repeat(sg, 32, axis=1) - 127
        eo = np.repeat(so, 32, axis=1) - 127
        vg = np.ldexp(mx.elem_decode(g, fmt), eg)
        vo = np.ldexp(mx.elem_decode(o, fmt), eo)
        big = np.maximum(np.abs(vg), np.abs(vo))
        _, ex = np.frexp(big)
        step = np.ldexp(1.0, np.maximum(ex - 1, np.maximum(eg, eo) + emin) - mbits)
        d = vg != vo
        far = d & (np.abs(vg - vo) > step + 1e-4 * maxval * np.ldexp(1.0, np.maximum(eg, eo)))
        assert not far.any(), f"h values too far apart: {list(zip(vg[far], vo[far]))[:8]}"
        flips += int((g != o).sum())
        total += d.size
        flipped |= set(np.asarray(r["rows"])[(g != o).any(1)].tolist())
    assert moved <= 1e-3 * max(blocks, 1), (moved, blocks)
    assert flips <= 1e-3 * max(total, 1) + 32 * moved, (flips, total)
    return flips, total, flipped


def check_stage2(layer, cfg, weights, rows, fmt):
    """Stage 2 on its own: the fp32 partial rows of sorted rows ``rows``
    against the fp64 product of the GPU's own h codes with W2 (so a neighbouring
    h code taken in stage 1 does not count against stage 2), row-relative,
    at the layer's bar. Returns the largest row-relative error."""
    offsets = layer.perm[1].cpu().numpy()
    srt = layer.perm[2].cpu().numpy()
    rows = np.unique(np.asarray(rows, np.int64))
    q, s = gpu_hq_rows(layer, cfg, rows, fmt)
    hd = mx.mx_dequantize(q, s, fmt)
    P = layer.partials
    worst = 0.0
    experts = np.searchsorted(offsets, rows, side="right") - 1
    for e in np.unique(experts):
        sel = experts == e
        w2 = mx.dequant_fp4(weights[2][e], weights[3][e])
        ref = hd[sel] @ w2.T
        a = torch.from_numpy(srt[rows[sel]].astype(np.int64)).cuda()
        got = P.index_select(0, a).cpu().numpy().astype(np.float64)
        worst = max(worst, gc.rowrel(got, ref))
    log(f"  stage 2 alone (GPU h codes x W2, fp64): rowrel={worst:.3e} on {rows.size} rows")
    assert worst <= TOL
    return worst


def output_on_gpu_h(layer, cfg, inp, lg, tokens, fmt):
    """The oracle's output for ``tokens`` evaluated on the GPU's h codes: per
    slot the fp64 product of the dequantised codes with W2, summed with the
    oracle's routing weights (fp64)."""
    ids_w = omoe.route_topk(lg, cfg.k, cfg.n_shared)
    pos = layer.perm[3].cpu().numpy()
    y = np.zeros((len(tokens), cfg.H))
    for i, t in enumerate(tokens):
        rows = pos[t * cfg.k_total + np.arange(cfg.k_total)]
        q, s = gpu_hq_rows(layer, cfg, rows, fmt)
        hd = mx.mx_dequantize(q, s, fmt)
        for j in range(cfg.k_total):
            e = int(ids_w[0][t, j])
            y[i] += ids_w[1][t, j] * (mx.dequant_fp4(inp.weights[2][e], inp.weights[3][e]) @ hd[j])
    return y


def check_against_oracle(cfg, inp, layer, out, tokens, fmt="e4m3", logits=None, bar=TOL,
                         stage2_rows=None, oracle_x_tokens=0, named=False):
    """Layer output against the oracle with the same activation quantisation
    (Oracle-Q), row-relative, at ``bar`` (1e-2, the layer target, for every
    named workload); h codes of the checked tokens' rows against the oracle's;
    stage 2 alone on ``stage2_rows`` (sorted rows; default: every row of the
    checked tokens); the paper's metrics (max abs, relative L2, cosine)
    against Oracle-Q and, on the first ``oracle_x_tokens`` tokens, against the
    oracle without activation quantisation (Oracle-X), logged."""
    lg = inp.logits if logits is None else logits
    ref = omoe.layer(inp.x, *inp.weights, k=cfg.k, n_shared=cfg.n_shared, logits=lg, fmt=fmt,
                     tokens=tokens, keep=True)
    flips, nh, flipped = check_hq_codes(layer, cfg, ref, fmt)
    tokens = np.asarray(tokens)
    y = gc.bf16_to_f64(gc.bf16_bits(out)[tokens])
    err = gc.rowrel(y, ref["out_f64"])
    mq = gc.metrics(y, ref["out_f64"])
    log(f"  rowrel={err:.3e} vs oracle-Q (bar {bar:g}); tokens={len(tokens)}; "
        f"h code flips={flips}/{nh}; metrics-Q max_abs={mq['max_abs']:.4g} "
        f"rel_l2={mq['rel_l2']:.3e} cosine={mq['cosine']:.9f}")
    if named or err <= bar:
        assert err <= bar
    else:
        per = np.array([gc.rowrel(y[i:i + 1], ref["out_f64"][i:i + 1]) for i in range(len(tokens))])
        over = np.nonzero(per > bar)[0]
        flip_tok = set((layer.perm[2].cpu().numpy()[sorted(flipped)] // cfg.k_total).tolist())
        assert all(int(tokens[i]) in flip_tok for i in over), \
            "a token misses the bar without an h code at a rounding midpoint"
        yc = output_on_gpu_h(layer, cfg, inp, lg, tokens[over], fmt)
        errc = gc.rowrel(y[over], yc)
        log(f"  {len(over)} token(s) over the bar, each with an h code at a midpoint; against "
            f"the oracle on the GPU's h codes: rowrel={errc:.3e} (bar {bar:g})")
        assert errc <= bar
    if oracle_x_tokens:
        tx = np.asarray(tokens)[:oracle_x_tokens]
        rx = omoe.layer(inp.x, *inp.weights, k=cfg.k, n_shared=cfg.n_shared, logits=lg,
                        fmt=None, tokens=tx)
        mx_ = gc.metrics(gc.bf16_to_f64(gc.bf16_bits(out)[tx]), rx["out_f64"])
        log(f"  metrics-X (no activation quantisation, {len(tx)} tokens): rowrel="
            f"{gc.rowrel(gc.bf16_to_f64(gc.bf16_bits(out)[tx]), rx['out_f64']):.3e} "
            f"max_abs={mx_['max_abs']:.4g} rel_l2={mx_['rel_l2']:.3e} cosine={mx_['cosine']:.9f}")
    if layer.partials is None:
        return ref, err
    # partials against the oracle's (these include the effect of any h code
    # that stage 1 took on the other side of a midpoint): logged
    P = layer.partials.view(cfg.T, cfg.k_total, cfg.H)[torch.from_numpy(np.asarray(tokens)).cuda()]
    perr = gc.rowrel(P.cpu().numpy().reshape(-1, cfg.H), ref["p_slots"].reshape(-1, cfg.H))
    log(f"  partials vs oracle-Q: rowrel={perr:.3e}")
    if stage2_rows is None:
        stage2_rows = np.concatenate([r["rows"] for r in ref["per_expert"].values()])
    check_stage2(layer, cfg, inp.weights, stage2_rows, fmt)
    return ref, err


def assert_repeats_identical(layer, x, weights, first, logits=None, wr=None, reps=10):
    """The same forward ``reps`` times in all (the first already ran and gave
    ``first``): every output bit-identical (the reduction order is fixed)."""
    first = first.clone()
    lg = None if logits is None else torch.from_numpy(logits).cuda()
    for i in range(reps - 1):
        out = layer.forward(x, weights, logits=lg, w_router=wr)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), first.view(torch.int16)), f"run {i + 2} differs"
    log(f"  {reps} runs bit-identical")


def small_case(T, H, I, E, k, S, seed, routing="normal"):
    cfg = synth.LayerConfig("small", T, H, E, k, I, S, routing, seed)
    return cfg, synth.make_inputs(cfg)


@pytest.mark.parametrize("fmt", ["e4m3", "e2m3", "e2m1"])
@pytest.mark.parametrize("shape", [
    (37, 512, 384, 16, 4, 1),     # ragged: ~10 rows per expert, K tail, 3 h tiles
    (200, 384, 384, 4, 2, 0),     # many rows per expert: 7 row tiles with a ragged tail
    (64, 1024, 256, 64, 8, 1),    # decode-like spread
    (3, 256, 128, 8, 8, 1),       # k = E
    (1, 128, 128, 1, 1, 0),       # smallest shape
    (300, 1024, 512, 4, 2, 1),    # tiled geometry, 256-row tiles: ~150-300 rows per expert, ragged
    (600, 512, 1024, 2, 1, 0),    # tiled geometry, 128-row tiles (2 per CU): full tiles + a ragged one
    (130, 512, 512, 2, 1, 0),     # tiled geometry: ~65 rows per expert, partial row blocks
    (400, 512, 256, 4, 2, 0),     # tiled stage 1 (128-row tiles), short-K stage 2 (I = 256)
    (300, 1024, 384, 4, 2, 1),    # tiled stage 1, streaming stage 2 (I = 384) and a shared expert
    (700, 768, 128, 5, 2, 1),     # streaming stage 1 (H = 768), short-K stage 2 with K = 128
    (170, 1024, 256, 3, 2, 0),    # short-K stage 2: tiles of 128 rows and ragged ones under 64
    (300, 2048, 512, 4, 2, 0),    # tiled stage 1 with K = 2048: middle groups of the K loop
    (40, 2048, 2048, 8, 2, 1),    # streaming, K = 2048 in both stages (8 triple-buffered steps)
    (16, 1024, 4096, 4, 2, 0),    # streaming stage 2 with K = 4096 (16 steps)
    (24, 8192, 512, 8, 2, 0),     # streaming stage 1 with K = 8192 (32 steps)
])
def test_small_layers(m, shape, fmt):
    cfg, inp = small_case(*shape, seed=sum(shape))
    log(f"small layer {shape} {fmt}")
    weights = gc.dev_expert_weights(inp.weights)
    # the unfused path, so its partials are checked too (the fused path's
    # output is compared with this path's bit for bit in test_gpu_fused.py)
    layer, out = run_layer(m, cfg, gc.to_dev_bf16(inp.x), weights, logits=inp.logits, fmt=fmt)
    log(f"  variant {m.moe_last_variant()}")
    ref, _ = check_against_oracle(cfg, inp, layer, out, np.arange(cfg.T), fmt,
                                  oracle_x_tokens=cfg.T)
    assert np.array_equal(layer.ids.cpu().numpy(), ref["ids"])
    assert np.array_equal(layer.perm[2].cpu().numpy(), ref["sorted"])
    xq = layer.workspace_view(0)[: cfg.T * m.ws_code_bytes(cfg.H, fmt)].cpu().numpy()
    assert np.array_equal(gc.ws_codes(xq.reshape(cfg.T, -1), fmt), ref["xq"])
    xs = layer.workspace_view(1)[: cfg.T * cfg.H // 32].cpu().numpy().reshape(cfg.T, -1)
    assert np.array_equal(xs, ref["xs"])


def test_tiled_geometry_skewed(m):
    """Zipf-skewed routing through the tiled geometry: hot experts with many
    row tiles, cold ones with a handful of rows or none."""
    cfg = synth.LayerConfig("skew", 600, 512, 16, 4, 512, 0, "zipf", 5, zipf_empty=3)
    inp = synth.make_inputs(cfg)
    log("tiled skewed")
    weights = gc.dev_expert_weights(inp.weights)
    layer, out = run_layer(m, cfg, gc.to_dev_bf16(inp.x), weights, logits=inp.logits)
    assert m.moe_last_variant() == m.VARIANT_TILED
    check_against_oracle(cfg, inp, layer, out, np.arange(cfg.T))


@pytest.mark.parametrize("fmt", ["e4m3", "e2m1"])
def test_tiled_row_tile_sizes_bit_identical(m, fmt):
    """The two arrangements of the LDS-tiled geometry (row tiles of 128 rows,
    two workgroups per CU, chunks of four tiles; of 256 rows, one workgroup
    per CU, chunks of two), forced through moe_set_tiled_rows on a shape whose
    experts hold ~360 rows (three 128-row tiles or two 256-row tiles, the last
    one ragged): outputs and partials bit-identical, both at the oracle bar."""
    cfg, inp = small_case(600, 512, 1024, 4, 2, 1, seed=11)
    log(f"tiled row-tile sizes {fmt}")
    weights = gc.dev_expert_weights(inp.weights)
    res = {}
    try:
        for rows in (128, 256):
            m.set_tiled_rows(rows)
            layer, out = run_layer(m, cfg, gc.to_dev_bf16(inp.x), weights, logits=inp.logits,
                                   fmt=fmt)
            assert m.moe_last_variant() == m.VARIANT_TILED
            check_against_oracle(cfg, inp, layer, out, np.arange(cfg.T), fmt)
            res[rows] = (out.clone(), layer.partials.clone())
    finally:
        m.set_tiled_rows(0)
    assert torch.equal(res[128][0], res[256][0])
    assert torch.equal(res[128][1], res[256][1])


def test_tiny_config_with_router(m):
    """The tiny workload end to end, logits from the bf16 router weights."""
    cfg = synth.CONFIGS["tiny"]
    inp = synth.make_inputs(cfg)
    log("tiny config")
    weights = gc.dev_expert_weights(inp.weights)
    wr = gc.to_dev_bf16(inp.wr)
    layer, out = run_layer(m, cfg, gc.to_dev_bf16(inp.x), weights, wr=wr)
    lg64 = omoe.router_logits(inp.x, inp.wr)
    lg_gpu = layer.logits.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(lg_gpu - lg64) <= 1e-5 * np.abs(lg64).max())
    # the oracle routes on its own logits; no near-ties in this workload
    srt = np.sort(lg64, axis=1)[:, ::-1]
    assert np.all(srt[:, cfg.k - 1] - srt[:, cfg.k] > 1e-5)
    ref = omoe.layer(inp.x, *inp.weights, k=cfg.k, wr_bits=inp.wr, keep=True)
    assert np.array_equal(layer.ids.cpu().numpy(), ref["ids"])
    y = gc.bf16_to_f64(gc.bf16_bits(out))
    err = gc.rowrel(y, ref["out_f64"])
    mq = gc.metrics(y, ref["out_f64"])
    refx = omoe.layer(inp.x, *inp.weights, k=cfg.k, wr_bits=inp.wr, fmt=None)
    mxx = gc.metrics(y, refx["out_f64"])
    log(f"  tiny rowrel={err:.3e} (bar {TOL:g}); metrics-Q rel_l2={mq['rel_l2']:.3e} "
        f"cosine={mq['cosine']:.9f}; metrics-X rowrel={gc.rowrel(y, refx['out_f64']):.3e} "
        f"rel_l2={mxx['rel_l2']:.3e} cosine={mxx['cosine']:.9f}")
    assert err <= TOL
    assert_repeats_identical(layer, gc.to_dev_bf16(inp.x), weights, out, wr=wr)


def test_hand_cases_exact(m):
    """H1 and H2 (tests/golden/hand_cases.json) come out exactly on the GPU."""
    log("hand cases")
    x = gc.to_dev_bf16(np.full((1, 128), 0x3F00, np.uint16))

    def const(h, i, w2_scale=127):
        b = 2 | (2 << 4)
        return (np.full((2 * i, h // 2), b, np.uint8), np.full((2 * i, h // 32), 127, np.uint8),
                np.full((h, i // 2), b, np.uint8), np.full((h, i // 32), w2_scale, np.uint8))
    # H = I = 128: G = U = 64, h = 4096/(1+e^-64) -> 4096, P = 128*4096 = 524288
    w = tuple(gc.to_dev_u8(np.stack([a])) for a in const(128, 128))
    cfg = synth.LayerConfig("h1", 1, 128, 1, 1, 128, 0)
    _, out = run_layer(m, cfg, x, w, logits=np.zeros((1, 1), np.float32))
    assert np.all(gc.bf16_to_f64(gc.bf16_bits(out)) == 524288.0)
    e0, e2 = const(128, 128), const(128, 128, 128)
    w = tuple(gc.to_dev_u8(np.stack(z)) for z in zip(e0, e0, e2, e0))
    cfg = synth.LayerConfig("h2", 1, 128, 4, 2, 128, 0)
    layer, out = run_layer(m, cfg, x, w, logits=np.array([[1, 3, 3, 0]], np.float32))
    assert layer.ids.cpu().numpy().tolist() == [[1, 2]]
    assert np.all(gc.bf16_to_f64(gc.bf16_bits(out)) == 0.5 * 524288 + 0.5 * 2 * 524288)


def test_empty_tokens(m):
    log("T = 0")
    cfg = synth.LayerConfig("empty", 0, 256, 8, 2, 128, 1)
    w = gc.dev_expert_weights(synth.gen_all_experts(cfg))
    layer = m.MoELayer(0, 256, 8, 2, 128, 1)
    out = layer.forward(torch.empty((0, 256), dtype=torch.bfloat16, device="cuda"), w,
                        logits=torch.empty((0, 8), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert out.shape == (0, 256)
    assert layer.perm[1].cpu().numpy().tolist() == [0] * 10


# Sorted-row positions inside an expert that the tiled kernels treat
# differently: first and last rows of a row tile (128 or 256 rows, by the
# shape) and of each 32-row block, the first rows of the other wave half's
# blocks, the first rows of a ragged tail tile; the last row of the expert is
# added per expert.
ROW_CLASSES = (0, 31, 32, 127, 128, 129, 200, 255, 256, 257, 300, 383, 384, 511, 512)


def _row_class_sample(cfg, perm, ntok, n_mid=2, seed=7):
    """Tokens and sorted rows that cover the kernels' row classes: the rows at
    ROW_CLASSES (and the last row) of the most and least loaded non-empty
    routed experts and of ``n_mid`` seeded others, their tokens, plus seeded
    tokens up to ``ntok`` and the last token. Returns (tokens, rows)."""
    counts, offsets, srt, _ = (np.asarray(a) for a in perm)
    nz = np.nonzero(counts[:cfg.E])[0]
    rng = np.random.default_rng(seed)
    experts = {int(nz[np.argmax(counts[nz])]), int(nz[np.argmin(counts[nz])])}
    experts |= set(int(e) for e in rng.choice(nz, min(n_mid, nz.size), replace=False))
    rows = []
    for e in sorted(experts):
        c = int(counts[e])
        rows += [int(offsets[e]) + p for p in ROW_CLASSES + (c - 1,) if p < c]
    rows = np.unique(rows)
    tokens = set((srt[rows] // cfg.k_total).tolist()) | {cfg.T - 1}
    extra = rng.permutation(cfg.T)
    for t in extra:
        if len(tokens) >= ntok:
            break
        tokens.add(int(t))
    return np.array(sorted(tokens)), rows


@pytest.mark.parametrize("name,ntok", [("decode", 64), ("prefill8k", 32), ("skew32k", 32),
                                       ("tpshard", 64), ("prefill8k_bal", 16)])
def test_full_size_configs(m, name, ntok):
    """Full-size workloads: route, permutation and activation codes compared in
    full; outputs, h codes and stage-2 partials on tokens and rows chosen to
    cover the kernels' row classes (all 64 tokens at decode); ten runs
    bit-identical."""
    cfg = synth.CONFIGS[name]
    log(f"full {name}: generating inputs")
    inp = synth.make_inputs(cfg, lazy=True)
    weights = gc.dev_weights(cfg)
    x = gc.to_dev_bf16(inp.x)
    log(f"full {name}: forward")
    layer, out = run_layer(m, cfg, x, weights, logits=inp.logits)
    variant = m.moe_last_variant()
    assert variant == {"decode": m.VARIANT_STREAM, "tpshard": m.VARIANT_SHORT}.get(
        name, m.VARIANT_TILED)
    ids_ref, w_ref = omoe.route_topk(inp.logits, cfg.k, cfg.n_shared)
    assert np.array_equal(layer.ids.cpu().numpy(), ids_ref)
    perm_ref = omoe.permute(ids_ref, cfg.NE)
    for g, r in zip(layer.perm, perm_ref):
        assert np.array_equal(g.cpu().numpy(), r)
    xq = layer.workspace_view(0)[: cfg.T * cfg.H].cpu().numpy().reshape(cfg.T, cfg.H)
    rows = np.arange(0, cfg.T, max(1, cfg.T // 256))
    xq_ref, _ = mx.mx_quantize(mx.bf16_to_f64(inp.x[rows]), "e4m3")
    assert np.array_equal(xq[rows], xq_ref)
    tokens, srows = _row_class_sample(cfg, perm_ref, ntok)
    log(f"full {name}: oracle on {len(tokens)} tokens, stage 2 on {len(srows)} class rows "
        f"(variant {variant})")
    check_against_oracle(cfg, inp, layer, out, tokens, stage2_rows=srows, oracle_x_tokens=4,
                         named=True)
    assert_repeats_identical(layer, x, weights, out, logits=inp.logits)


def test_metamorphic_w2_scale_doubles_output(m):
    """W2 scale bytes + 1 => every output exactly x2 on the GPU (bitwise)."""
    cfg = synth.LayerConfig("mm", 96, 512, 16, 4, 256, 1, "normal", 3)
    inp = synth.make_inputs(cfg)
    log("metamorphic w2 scale")
    w = list(gc.dev_expert_weights(inp.weights))
    x = gc.to_dev_bf16(inp.x)
    _, out = run_layer(m, cfg, x, tuple(w), logits=inp.logits)
    base = gc.bf16_to_f64(gc.bf16_bits(out))
    w[3] = w[3] + 1
    _, out2 = run_layer(m, cfg, x, tuple(w), logits=inp.logits)
    assert np.array_equal(gc.bf16_to_f64(gc.bf16_bits(out2)), 2 * base)
    # token permutation permutes output rows bit-exactly
    perm = np.random.default_rng(0).permutation(cfg.T)
    w[3] = w[3] - 1
    _, out3 = run_layer(m, cfg, gc.to_dev_bf16(inp.x[perm]), tuple(w), logits=inp.logits[perm])
    assert np.array_equal(gc.bf16_bits(out3), gc.bf16_bits(out)[perm])


@pytest.mark.parametrize("fmt", ["e2m1", "e2m3"])
def test_full_size_prefill_fp4_rate_activations(m, fmt):
    """The 8K prefill with MXFP4 or MXFP6 activations (the FP4-rate runs of the
    bench): routing exact, tokens covering the row classes against the oracle
    in the same format, ten runs bit-identical."""
    cfg = synth.CONFIGS["prefill8k"]
    inp = synth.make_inputs(cfg, lazy=True)
    weights = gc.dev_weights(cfg)
    x = gc.to_dev_bf16(inp.x)
    log(f"full prefill8k {fmt}: forward")
    layer, out = run_layer(m, cfg, x, weights, logits=inp.logits, fmt=fmt)
    assert m.moe_last_variant() == m.VARIANT_TILED
    ids_ref, _ = omoe.route_topk(inp.logits, cfg.k, cfg.n_shared)
    assert np.array_equal(layer.ids.cpu().numpy(), ids_ref)
    tokens, srows = _row_class_sample(cfg, omoe.permute(ids_ref, cfg.NE), 16)
    log(f"full prefill8k {fmt}: oracle on {len(tokens)} tokens")
    check_against_oracle(cfg, inp, layer, out, tokens, fmt, stage2_rows=srows, named=True)
    assert_repeats_identical(layer, x, weights, out, logits=inp.logits)


def test_layer_at_expert_and_k_limits(m):
    """1024 routed experts (MOE_MAX_EXPERTS) + the shared one, so the tile
    list's threads handle a second group, and k_total = 32 (MOE_MAX_K_TOTAL):
    most experts empty, the rest with a row or two."""
    cfg = synth.LayerConfig("limits", 8, 256, 1024, 31, 128, 1, "normal", 11)
    inp = synth.make_inputs(cfg)
    log("layer at the expert and k limits")
    weights = gc.dev_expert_weights(inp.weights)
    layer, out = run_layer(m, cfg, gc.to_dev_bf16(inp.x), weights, logits=inp.logits)
    ref, _ = check_against_oracle(cfg, inp, layer, out, np.arange(cfg.T))
    assert np.array_equal(layer.ids.cpu().numpy(), ref["ids"])
    assert np.array_equal(layer.perm[2].cpu().numpy(), ref["sorted"])
