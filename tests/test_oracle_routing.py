"""Pins of the routing variants of the oracle (route_topk_ex): hand-computed
cases, special cases that reduce to the pinned route_topk, and invariants.
Every expected value below is derived by hand or from a closed form, not from
the function under test."""
import math

import numpy as np
import pytest

from oracle import moe as omoe


def _logits(t, e, seed):
    return np.random.default_rng(seed).standard_normal((t, e)).astype(np.float32)


def test_defaults_are_route_topk():
    lg = _logits(64, 256, 1)
    for k, s in ((8, 1), (6, 0), (1, 0)):
        i0, w0 = omoe.route_topk(lg, k, s)
        i1, w1 = omoe.route_topk_ex(lg, k, s)
        assert np.array_equal(i0, i1)
        assert np.allclose(w0, w1, rtol=1e-14, atol=0)


def test_model_top6_order():
    # the model routes each token to 6 experts: the 6 largest logits, by
    # (logit descending, id ascending); ties at 0.5 go to the lower id
    lg = np.array([[0.5, 3.0, 0.5, -1.0, 2.0, 0.5, 7.0, 0.5, 1.0]], np.float32)
    ids, w = omoe.route_topk_ex(lg, 6)
    assert ids.tolist() == [[6, 1, 4, 8, 0, 2]]
    ex = np.exp(np.array([7.0, 3.0, 2.0, 1.0, 0.5, 0.5]) - 7.0)
    assert np.allclose(w[0], ex / ex.sum(), rtol=1e-15)


def test_sigmoid_bias_hand_case():
    # s = sigmoid(l) = [s(2), s(1), 1/2, s(-1)]; key = s + bias = [s(2), s(1), 1.1, s(-1)]:
    # the bias lifts expert 2 above expert 0; weights use s (not the bias)
    lg = np.array([[2.0, 1.0, 0.0, -1.0]], np.float32)
    bias = np.array([0.0, 0.0, 0.6, 0.0], np.float32)
    ids, w = omoe.route_topk_ex(lg, 2, score="sigmoid", bias=bias)
    assert ids.tolist() == [[2, 0]]
    s2 = 1.0 / (1.0 + math.exp(-2.0))
    assert np.allclose(w[0], [0.5 / (0.5 + s2), s2 / (0.5 + s2)], rtol=1e-12)
    ids, w = omoe.route_topk_ex(lg, 2, score="sigmoid", bias=bias, renorm=False, scale=2.5)
    assert np.allclose(w[0], [1.25, 2.5 * s2], rtol=1e-12)


def test_group_limited_hand_case():
    # 4 groups of 2: softmax masses exp(l) per group: g0 e^5 + e^-5, g1 2 e^3.5 (66.2),
    # g2 e^4 + e^-5 (54.6), g3 2. Top-2 groups: g0, g1, so expert 4 (logit 4) is
    # excluded and the second pick is expert 2 (tie with 3 at 3.5: lower id).
    lg = np.array([[5.0, -5.0, 3.5, 3.5, 4.0, -5.0, 0.0, 0.0]], np.float32)
    ids, w = omoe.route_topk_ex(lg, 2, n_group=4, topk_group=2)
    assert ids.tolist() == [[0, 2]]
    r = math.exp(-1.5)
    assert np.allclose(w[0], [1 / (1 + r), r / (1 + r)], rtol=1e-12)
    ids, _ = omoe.route_topk_ex(lg, 2)
    assert ids.tolist() == [[0, 4]]  # without groups expert 4 is second


def test_group_reductions():
    lg = _logits(200, 64, 2)
    base = omoe.route_topk_ex(lg, 6, score="sigmoid")
    for ng, tg in ((1, 1), (8, 8), (4, 4)):
        ids, w = omoe.route_topk_ex(lg, 6, score="sigmoid", n_group=ng, topk_group=tg)
        assert np.array_equal(ids, base[0]) and np.allclose(w, base[1], rtol=1e-15)


def test_group_selection_properties():
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((300, 64)).astype(np.float32)
    bias = (0.05 * rng.standard_normal(64)).astype(np.float32)
    ng, tg, k = 8, 3, 6
    ids, _ = omoe.route_topk_ex(lg, k, score="sigmoid", bias=bias, n_group=ng, topk_group=tg)
    s = 1 / (1 + np.exp(-lg.astype(np.float64)))
    key = s + bias
    gsc = np.sort(key.reshape(-1, ng, 8), axis=2)[:, :, -2:].sum(axis=2)
    for t in range(len(lg)):
        groups = set(ids[t] // 8)
        assert len(groups) <= tg
        # a group holding a pick is beaten by fewer than tg groups
        for g in groups:
            assert (gsc[t] > gsc[t, g]).sum() < tg
        # no expert of a kept group outranks the last pick
        kept = np.argsort(-gsc[t], kind="stable")[:tg]
        cand = np.concatenate([np.arange(8 * g, 8 * g + 8) for g in kept])
        rest = np.setdiff1d(cand, ids[t])
        assert key[t, rest].max() <= key[t, ids[t][-1]]


def test_sigmoid_without_bias_picks_like_softmax():
    lg = _logits(100, 256, 4)
    i0, _ = omoe.route_topk(lg, 8)
    i1, w1 = omoe.route_topk_ex(lg, 8, score="sigmoid")
    assert np.array_equal(i0, i1)
    s = 1 / (1 + np.exp(-np.take_along_axis(lg.astype(np.float64), i1, axis=1)))
    assert np.allclose(w1, s / s.sum(axis=1, keepdims=True), rtol=1e-14)


def test_renorm_and_scale():
    lg = _logits(50, 32, 5)
    _, w = omoe.route_topk_ex(lg, 4, score="sigmoid", scale=2.5)
    assert np.allclose(w.sum(axis=1), 2.5, rtol=1e-14)
    ids, w = omoe.route_topk_ex(lg, 4, renorm=False)
    full = np.exp(lg.astype(np.float64))
    full /= full.sum(axis=1, keepdims=True)
    assert np.allclose(w, np.take_along_axis(full, ids, axis=1), rtol=1e-13)
    assert (w.sum(axis=1) < 1).all()


def test_shared_column_kept():
    lg = _logits(5, 16, 6)
    ids, w = omoe.route_topk_ex(lg, 3, 1, score="sigmoid", scale=2.5)
    assert (ids[:, 3] == 16).all() and (w[:, 3] == 1.0).all()


@pytest.mark.parametrize("bad", [dict(n_group=3), dict(n_group=4, topk_group=5),
                                 dict(score="relu")])
def test_rejects_bad_options(bad):
    with pytest.raises(ValueError):
        omoe.route_topk_ex(_logits(2, 16, 7), 2, **bad)


def test_balanced_routing_gives_equal_loads():
    """The 'balanced' synthetic routing (the prefill8k_bal measurement
    companion) gives every routed expert exactly T*k/E assignments and token t
    the experts (t*k + j) % E in pick order j."""
    import synth
    cfg = synth.CONFIGS["prefill8k_bal"]
    ids, w = omoe.route_topk(synth.gen_logits(cfg), cfg.k, cfg.n_shared)
    t = np.arange(cfg.T)[:, None]
    assert np.array_equal(ids[:, :cfg.k], (t * cfg.k + np.arange(cfg.k)[None, :]) % cfg.E)
    counts = np.bincount(ids.ravel(), minlength=cfg.NE)
    assert (counts[:cfg.E] == cfg.T * cfg.k // cfg.E).all() and counts[cfg.E] == cfg.T
