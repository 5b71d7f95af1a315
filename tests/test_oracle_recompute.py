"""Pins of the recompute oracle (App. C.2) against closed forms, library
routines and invariants, so that a dropped term, a wrong sign or index, or a
transposed operand in it fails here."""
import math

import numpy as np
import pytest
from scipy.special import expit, softmax

from oracle import kara_recompute as rc


def test_rms_norm_closed_forms():
    g = np.array([1.0, 2.0, -1.0, 0.5])
    # a constant vector c has mean square c^2: the result is sign(c) * g (eps = 0)
    np.testing.assert_allclose(rc.rms_norm(np.full((1, 4), -3.0), g, 0.0)[0], -g)
    # [3, 4, 0, 0]: mean square 25/4, norm factor 2/5
    np.testing.assert_allclose(rc.rms_norm(np.array([[3.0, 4.0, 0.0, 0.0]]), np.ones(4), 0.0)[0],
                               [1.2, 1.6, 0.0, 0.0])
    # eps sits inside the square root
    np.testing.assert_allclose(rc.rms_norm(np.array([[1.0, 1.0]]), np.ones(2), 3.0)[0], [0.5, 0.5])
    # scale invariance
    h = np.random.default_rng(0).normal(size=(3, 16))
    np.testing.assert_allclose(rc.rms_norm(7.5 * h, np.ones(16), 0.0), rc.rms_norm(h, np.ones(16), 0.0))


def test_rope_closed_forms_and_invariants():
    # d = 2: one pair, inverse frequency theta^0 = 1, rotation by `pos` radians
    x = np.array([[[1.0, 0.0]], [[1.0, 0.0]], [[0.0, 2.0]]])
    y = rc.rope(x, np.array([0, 1, 3]), 10000.0)
    np.testing.assert_allclose(y[0, 0], [1.0, 0.0])
    np.testing.assert_allclose(y[1, 0], [math.cos(1.0), math.sin(1.0)], atol=1e-15)
    np.testing.assert_allclose(y[2, 0], [-2.0 * math.sin(3.0), 2.0 * math.cos(3.0)], atol=1e-15)
    # d = 4: pairs (0, 2) and (1, 3); the second pair turns at theta^(-1/2)
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    y = rc.rope(x, np.array([5]), 100.0)[0, 0]
    a = 5 * 100.0 ** -0.5
    np.testing.assert_allclose(y, [0.0, math.cos(a), 0.0, math.sin(a)], atol=1e-15)
    rng = np.random.default_rng(1)
    q, k = rng.normal(size=(1, 1, 64)), rng.normal(size=(1, 1, 64))
    # norms are preserved, and q(m).k(n) depends only on m - n
    qm = rc.rope(q, np.array([17]), 10000.0)
    np.testing.assert_allclose(np.linalg.norm(qm), np.linalg.norm(q))
    dots = [float(rc.rope(q, np.array([m]), 1e4)[0, 0] @ rc.rope(k, np.array([m - 5]), 1e4)[0, 0])
            for m in (5, 40, 1000)]
    np.testing.assert_allclose(dots, dots[0], rtol=1e-12)
    # position 0 is the identity
    np.testing.assert_allclose(rc.rope(q, np.array([0]), 1e4), q)


def test_silu_matches_library():
    x = np.linspace(-30, 30, 101)
    np.testing.assert_allclose(rc.silu(x), x * expit(x), rtol=1e-14, atol=1e-300)
    assert rc.silu(np.array([0.0]))[0] == 0.0


def test_attention_closed_forms():
    rng = np.random.default_rng(2)
    d = 8
    k = rng.normal(size=(6, 1, d))
    v = rng.normal(size=(6, 1, d))
    q = rng.normal(size=(3, 1, d))
    # p0 = 0: the first window token sees only cache row 0, whose value it returns
    o = rc.causal_window_attention(q, k, v, 0, 1.0)
    np.testing.assert_allclose(o[0, 0], v[0, 0])
    # equal keys: the mean of the visible values
    ke = np.repeat(k[:1], 6, axis=0)
    o = rc.causal_window_attention(q, ke, v, 2, 1.0)
    for w in range(3):
        np.testing.assert_allclose(o[w, 0], v[:3 + w, 0].mean(axis=0))
    # a row against scipy's softmax over exactly the visible rows
    o = rc.causal_window_attention(q, k, v, 2, 0.3)
    p = softmax(0.3 * (k[:4, 0] @ q[1, 0]))
    np.testing.assert_allclose(o[1, 0], p @ v[:4, 0])


def test_attention_is_causal_and_grouped():
    rng = np.random.default_rng(3)
    Hq, Hkv, d = 4, 2, 8
    k = rng.normal(size=(10, Hkv, d))
    v = rng.normal(size=(10, Hkv, d))
    q = rng.normal(size=(4, Hq, d))
    base = rc.causal_window_attention(q, k, v, 5, 0.5)
    # rows after p0 + w do not reach token w
    k2, v2 = k.copy(), v.copy()
    k2[7:], v2[7:] = 50.0, -50.0
    got = rc.causal_window_attention(q, k2, v2, 5, 0.5)
    np.testing.assert_allclose(got[:2], base[:2])
    assert not np.allclose(got[2:], base[2:])
    # query heads 0, 1 read KV head 0; heads 2, 3 read KV head 1
    k3 = k.copy()
    k3[:, 1] = rng.normal(size=(10, d))
    got = rc.causal_window_attention(q, k3, v, 5, 0.5)
    np.testing.assert_allclose(got[:, :2], base[:, :2])
    assert not np.allclose(got[:, 2:], base[:, 2:])


def _layer_weights(rng, D, Hq, d, F, zero_out=False):
    s = 1.0 / math.sqrt(D)
    return dict(w_q=rng.normal(size=(D, Hq * d)) * s, w_o=np.zeros((Hq * d, D)) if zero_out else
                rng.normal(size=(Hq * d, D)) * s, w_gate=rng.normal(size=(D, F)) * s, w_up=rng.normal(size=(D, F)) * s,
                w_down=np.zeros((F, D)) if zero_out else rng.normal(size=(F, D)) / math.sqrt(F),
                g_attn=1.0 + 0.1 * rng.normal(size=D), g_ffn=1.0 + 0.1 * rng.normal(size=D))


def test_layer_structure():
    rng = np.random.default_rng(4)
    D, Hq, Hkv, d, F, W, p0 = 32, 4, 2, 8, 48, 5, 3
    dims = dict(n_q_heads=Hq, head_dim=d, rms_eps=1e-6, rope_theta=10000.0)
    h = rng.normal(size=(W, D))
    k = rng.normal(size=(p0 + W, Hkv, d))
    v = rng.normal(size=(p0 + W, Hkv, d))
    # with W_o = W_down = 0 the residual stream passes through unchanged and
    # the queries are RoPE(RMSNorm(h) g W_q) at positions rope_pos0 + w
    wt = _layer_weights(rng, D, Hq, d, F, zero_out=True)
    q, h2, o = rc.recompute_layer(h, wt, k, v, p0, 100, dims)
    np.testing.assert_allclose(h2, h)
    want = rc.rope((rc.rms_norm(h, wt["g_attn"], 1e-6) @ wt["w_q"]).reshape(W, Hq, d), 100 + np.arange(W), 1e4)
    np.testing.assert_allclose(q, want)
    # the two residual branches add: attention only, then the feed-forward block
    wt = _layer_weights(rng, D, Hq, d, F)
    q, h2, o = rc.recompute_layer(h, wt, k, v, p0, 100, dims)
    h_att = h + o.reshape(W, -1) @ wt["w_o"]
    x2 = rc.rms_norm(h_att, wt["g_ffn"], 1e-6)
    np.testing.assert_allclose(h2, h_att + (rc.silu(x2 @ wt["w_gate"]) * (x2 @ wt["w_up"])) @ wt["w_down"])
    # the window token at w attends to cache rows 0 .. p0 + w: brute force on one head
    logits = k[:p0 + 3, 1] @ q[2, 3] / math.sqrt(d)
    np.testing.assert_allclose(o[2, 3], softmax(logits) @ v[:p0 + 3, 1])


@pytest.mark.parametrize("bs", [1, 3, 16])
def test_cache_rows_follow_the_block_table(bs):
    rng = np.random.default_rng(5)
    pool = rng.normal(size=(12, 2, bs, 4))
    table = rng.permutation(12)[:6]
    rows = rc.cache_rows(pool, table, 5, bs, lambda a: a)
    for pos in range(5):
        np.testing.assert_array_equal(rows[pos], pool[table[pos // bs], :, pos % bs, :])
