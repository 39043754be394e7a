"""GPU routing variants (moe_route_topk_ex) against the oracle's route_topk_ex.

Without a bias, keys are raw logits on both sides, so picks must match bit
for bit (ties included). With a bias or groups, keys and group scores are
fp32 sums on the GPU and fp64 in the oracle: a pick may differ only where the
oracle's keys (or group scores) of the two candidates lie within a relative
1e-5 of each other; everything else must match. Weights: relative 1e-5."""
import numpy as np
import pytest
import torch

from oracle import moe as omoe
from tests.gpu_common import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def m():
    from paper_2609_15627_amd import moe
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return moe


def _keys(lg, score, bias):
    lg = lg.astype(np.float64)
    if score == "softmax":
        z = np.exp(lg - lg.max(axis=1, keepdims=True))
        s = z / z.sum(axis=1, keepdims=True)
    else:
        s = 1 / (1 + np.exp(-lg))
    return s if bias is None else s + bias


def _run(m, lg, k, S, **o):
    bias = o.get("bias")
    dev_bias = None if bias is None else torch.from_numpy(bias).cuda()
    ids, w = m.moe_route_topk(torch.from_numpy(lg).cuda(), k, S, **{**o, "bias": dev_bias})
    torch.cuda.synchronize()
    return ids.cpu().numpy(), w.cpu().numpy().astype(np.float64)


def _check(m, lg, k, S, **o):
    ids_ref, w_ref = omoe.route_topk_ex(lg, k, S, **o)
    ids, w = _run(m, lg, k, S, **o)
    exact = o.get("bias") is None and o.get("n_group", 1) == 1
    diff = (ids != ids_ref).any(axis=1)
    if exact:
        assert not diff.any(), np.nonzero(diff)[0][:5]
    else:
        key = _keys(lg, o.get("score", "softmax"), o.get("bias"))
        for t in np.nonzero(diff)[0]:
            a = set(ids[t, :k]) ^ set(ids_ref[t, :k])
            if a:  # different sets: every swapped key ties the last kept one
                kk = key[t, list(a)]
                last = key[t, ids_ref[t, k - 1]]
                assert np.all(np.abs(kk - last) <= 1e-5 * np.abs(last)), (t, ids[t], ids_ref[t])
            else:  # same set, order differs: neighbouring keys tie
                kk = key[t, ids[t, :k]]
                assert np.allclose(np.sort(kk), np.sort(key[t, ids_ref[t, :k]]), rtol=1e-5)
        assert diff.mean() <= 1e-2, diff.mean()
    same = ~diff
    assert np.all(np.abs(w[same] - w_ref[same]) <= 1e-5 * np.abs(w_ref[same]) + 1e-7)
    return diff.sum()


OPTS = [
    ("softmax_norenorm", 8, 1, dict(renorm=False)),
    ("sigmoid_top6_scale", 6, 0, dict(score="sigmoid", scale=2.5)),
    ("sigmoid_top6_norenorm", 6, 1, dict(score="sigmoid", renorm=False)),
    ("softmax_groups", 8, 1, dict(n_group=8, topk_group=4)),
    ("sigmoid_bias_groups", 8, 1, dict(score="sigmoid", n_group=8, topk_group=4, scale=2.5,
                                       bias=True)),
    ("softmax_bias", 6, 0, dict(bias=True)),
]


@pytest.mark.parametrize("name,k,S,opts", OPTS, ids=[o[0] for o in OPTS])
def test_route_variants(m, name, k, S, opts):
    rng = np.random.default_rng(abs(hash(name)) % 2**31)
    lg = rng.standard_normal((4096, 256)).astype(np.float32)
    o = dict(opts)
    if o.pop("bias", None):
        o["bias"] = (0.1 * rng.standard_normal(256)).astype(np.float32)
    log(f"route variant {name}")
    n = _check(m, lg, k, S, **o)
    log(f"  near-tie differences: {n}")


def test_route_variant_ties_and_small_groups(m):
    rng = np.random.default_rng(9)
    lg = rng.integers(-2, 2, (300, 64)).astype(np.float32)    # many exact ties
    log("route variant ties")
    _check(m, lg, 4, 0, score="sigmoid", renorm=False)
    _check(m, lg, 4, 1, n_group=64, topk_group=8)              # groups of one expert


def test_route_variant_default_is_bitwise_route_topk(m):
    lg = np.random.default_rng(10).standard_normal((500, 256)).astype(np.float32)
    a = m.moe_route_topk(torch.from_numpy(lg).cuda(), 8, 1)
    # an option set equal to the defaults but sent through the variant kernel
    b = m.moe_route_topk(torch.from_numpy(lg).cuda(), 8, 1, n_group=2, topk_group=2)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_route_variant_rejects(m):
    lg = torch.zeros((4, 16), dtype=torch.float32, device="cuda")
    for bad in (dict(n_group=3), dict(n_group=4, topk_group=5), dict(n_group=4, topk_group=1)):
        with pytest.raises(m.MoeError):
            m.moe_route_topk(lg, 6, 0, **bad)


# ----------------------------------------------------------- fused router (f1)
def _router_case(T, H, E, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H)).astype(np.float32)
    wr = (0.02 * rng.standard_normal((E, H))).astype(np.float32)
    xb = (x.view(np.uint32) >> 16).astype(np.uint16)       # truncation to bf16 bits
    wb = (wr.view(np.uint32) >> 16).astype(np.uint16)
    return xb, wb


@pytest.mark.parametrize("T,H,E,k,S,opts", [
    (8192, 4096, 256, 8, 1, {}),                                   # prefill-sized, defaults
    (64, 4096, 256, 6, 0, dict(score="sigmoid", scale=2.5)),       # decode, the model's top-6
    (100, 1024, 256, 8, 1, dict(score="sigmoid", n_group=8, topk_group=4, bias=True)),
    (37, 256, 8, 2, 0, {}),                                        # ragged token block, E < 64
    (1500, 512, 64, 4, 0, dict(score="sigmoid")),                  # fused path, ragged last block
    (65, 512, 100, 7, 1, dict(renorm=False)),                      # E not a multiple of 64
    (1024, 512, 300, 6, 0, {}),                                    # fused, two expert chunks
    (1100, 256, 1024, 8, 1, dict(score="sigmoid", n_group=8, topk_group=4, bias=True)),
    (2048, 1024, 384, 8, 1, {}),                                   # fused, E = 384
])
def test_router_topk_fused(m, T, H, E, k, S, opts):
    xb, wb = _router_case(T, H, E, T + H + E)
    o = dict(opts)
    if o.pop("bias", None):
        o["bias"] = (0.05 * np.random.default_rng(1).standard_normal(E)).astype(np.float32)
    log(f"fused router T={T} H={H} E={E} k={k} opts={sorted(o)}")
    x = torch.from_numpy(xb.view(np.int16)).cuda().view(torch.bfloat16)
    wr = torch.from_numpy(wb.view(np.int16)).cuda().view(torch.bfloat16)
    bias = None if "bias" not in o else torch.from_numpy(o["bias"]).cuda()
    ids, w, lg = m.moe_router_topk(x, wr, k, S, want_logits=True, **{**o, "bias": bias})
    torch.cuda.synchronize()
    ids, w, lg = ids.cpu().numpy(), w.cpu().numpy().astype(np.float64), lg.cpu().numpy()
    # logits: exact bf16 products summed in fp32, H / 16 accumulation steps of
    # the matrix core, each rounding by at most 2^-24 of a partial sum bounded
    # by sum_h |x_h w_h|
    ref = omoe.router_logits(xb, wb)
    mag = np.abs(omoe.mx.bf16_to_f64(xb)) @ np.abs(omoe.mx.bf16_to_f64(wb)).T
    assert np.all(np.abs(lg - ref) <= (H / 16 + 16) * 2.0 ** -24 * mag + 1e-30)
    # routing of the GPU's own logits must match the oracle's routing of them exactly
    # where the keys are logits, and within near ties otherwise
    ids_ref, w_ref = omoe.route_topk_ex(lg, k, S, **o)
    diff = (ids != ids_ref).any(axis=1)
    if "bias" not in o and o.get("n_group", 1) == 1:
        assert not diff.any()
    else:
        assert diff.mean() <= 1e-2
    same = ~diff
    assert np.all(np.abs(w[same] - w_ref[same]) <= 1e-5 * np.abs(w_ref[same]) + 1e-7)
    # and against the fp64 logits: picks differ only at logit near-ties
    ids64, _ = omoe.route_topk_ex(ref, k, S, **o)
    d64 = (ids[:, :k] != ids64[:, :k]).any(axis=1)
    log(f"  picks differing from fp64-logit routing: {int(d64.sum())} of {T}")
    assert d64.mean() <= 1e-2


def test_router_topk_rejects(m):
    x = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(m.MoeError):  # more experts than MOE_MAX_EXPERTS
        m.moe_router_topk(torch.zeros((4, 128), dtype=torch.bfloat16, device="cuda"),
                          torch.zeros((1025, 128), dtype=torch.bfloat16, device="cuda"), 2)
    with pytest.raises(m.MoeError):
        m.moe_router_topk(torch.zeros((4, 96), dtype=torch.bfloat16, device="cuda"),
                          torch.zeros((16, 96), dtype=torch.bfloat16, device="cuda"), 2)
    with pytest.raises(m.MoeError):
        m.moe_router_topk(torch.zeros((4, 192), dtype=torch.bfloat16, device="cuda"),
                          torch.zeros((16, 192), dtype=torch.bfloat16, device="cuda"), 2)
