"""Pins for the oracle's window scoring, Eq. (4) (Kara Sec. 4.1).

Each test fixes a fact the paper or the mathematics determines, chosen so a
plausible slip (causal mask, softmax over the wrong axis, dropped scale,
buffer keys in the denominator, one GQA head only) fails one of them.
"""
import math

import numpy as np
import pytest
from scipy.special import softmax as scipy_softmax

import oracle

LN3 = math.log(3.0)


def test_closed_form_two_tokens():
    # W=2, U=0, d=1, scale 1.  Row 0 logits [0,0] -> [1/2,1/2]; row 1 logits
    # [0, ln 3] -> [1/4, 3/4]; colsum -> [3/4, 5/4].  A causal mask would give
    # [5/4, 3/4]; a softmax over queries would give [1, 1].
    q = np.array([[0.0], [LN3]])
    k = np.array([[0.0], [1.0]])
    a = oracle.window_scores(q, k, 1.0)
    np.testing.assert_allclose(a, [0.75, 1.25], rtol=0, atol=1e-15)


def test_buffer_keys_excluded_from_denominator():
    # Same window with U=1: only key 0 is compressible, both queries score it,
    # each row's softmax has one entry, so A = [2] (= number of query rows).
    # Keeping the buffer key in the denominator would give 1/2 + 1/4.
    q = np.array([[0.0], [LN3]])
    k = np.array([[0.0]])
    np.testing.assert_allclose(oracle.window_scores(q, k, 1.0), [2.0], atol=1e-15)


def test_scale_is_one_over_sqrt_d():
    # d=4: q=[ln3, ln3, 0, 0], keys 0 and [1,1,0,0]: logits [0, 2 ln 3] * 1/2
    # -> softmax [1/4, 3/4].  Without the scale it would be [1/10, 9/10].
    p = dict(head_dim=4, scale=0.0)
    s = oracle.scale_of(p)
    assert s == 0.5
    q = np.array([[LN3, LN3, 0.0, 0.0]])
    k = np.array([[0.0, 0.0, 0.0, 0.0], [1.0, 1.0, 0.0, 0.0]])
    np.testing.assert_allclose(oracle.window_scores(q, k, s), [0.25, 0.75], atol=1e-15)


def test_single_query_reduces_to_softmax():
    # One query row: the colsum is that row's softmax (library routine).
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 16))
    k = rng.standard_normal((37, 16))
    want = scipy_softmax(q[0] @ k.T / 4.0)
    np.testing.assert_allclose(oracle.window_scores(q, k, 0.25), want, rtol=1e-13)


@pytest.mark.parametrize("case", ["zero_q", "equal_k", "one_key"])
def test_special_cases(case):
    rng = np.random.default_rng(1)
    R, N, d = 24, 10, 8
    q = rng.standard_normal((R, d))
    k = rng.standard_normal((N, d))
    if case == "zero_q":
        q[:] = 0.0
        want = np.full(N, R / N)
    elif case == "equal_k":
        k[:] = k[0]
        want = np.full(N, R / N)
    else:
        k = k[:1]
        want = np.array([float(R)])
    np.testing.assert_allclose(oracle.window_scores(q, k, 0.3), want, rtol=1e-13)


def test_invariants_random():
    rng = np.random.default_rng(2)
    R, N, d = 40, 29, 16
    q = rng.standard_normal((R, d)) * 2
    k = rng.standard_normal((N, d))
    a = oracle.window_scores(q, k, 0.25)
    # every softmax row sums to 1, so the scores sum to the number of rows
    assert abs(a.sum() - R) < 1e-11
    assert np.all(a > 0)
    # the query rows are summed: their order does not matter
    a2 = oracle.window_scores(q[rng.permutation(R)], k, 0.25)
    np.testing.assert_allclose(a2, a, rtol=1e-12)
    # permuting keys permutes the scores
    perm = rng.permutation(N)
    a3 = oracle.window_scores(q, k[perm], 0.25)
    np.testing.assert_allclose(a3, a[perm], rtol=1e-12)


def _pool_case(G, Hkv, W, d, dtype, seed):
    rng = np.random.default_rng(seed)
    Hq = G * Hkv
    q = rng.standard_normal((1, 1, W, Hq, d)).astype(np.float32)
    bs, pages = 4, 16
    pool = rng.standard_normal((pages, Hkv, bs, d)).astype(np.float32)
    table = rng.permutation(pages)[None, :].astype(np.int64)
    return q, pool, table, bs


def test_gqa_groups_all_query_heads_of_a_kv_head():
    # Hq=4, Hkv=2 (G=2): KV head 1 is scored by query heads 2 and 3 over all
    # W window tokens, i.e. 2*W rows; its scores sum to 2*W.
    G, Hkv, W, d = 2, 2, 6, 8
    q, pool, table, bs = _pool_case(G, Hkv, W, d, "f32", 3)
    p = dict(window=W, buffer=0, block_size=bs, n_q_heads=G * Hkv, n_kv_heads=Hkv,
             head_dim=d, dtype="f32", scale=0.0)
    p0 = 3
    rows = oracle.unit_queries(q, p, 0, 0, 1)
    assert rows.shape == (W * G, d)
    np.testing.assert_array_equal(rows[0::2], q[0, 0, :, 2, :].astype(np.float64))
    np.testing.assert_array_equal(rows[1::2], q[0, 0, :, 3, :].astype(np.float64))
    keys = oracle.unit_keys(pool, p, table[0], p0, 1)
    for j in range(W):
        pos = p0 + j
        np.testing.assert_array_equal(keys[j], pool[table[0, pos // bs], 1, pos % bs].astype(np.float64))
    a = oracle.score_units(p, [0], q, [pool], table, np.array([p0]), [(0, 0, 1)])[0]
    assert abs(a.sum() - G * W) < 1e-11
    # equals the sum of each query head's own colsum (one softmax per row)
    scale = 1 / math.sqrt(d)
    per_head = sum(oracle.window_scores(q[0, 0, :, h, :].astype(np.float64), keys, scale) for h in (2, 3))
    np.testing.assert_allclose(a, per_head, rtol=1e-12)


def test_bf16_widening_exact():
    vals = np.array([1.0, -2.5, 0.0078125, 2.0 ** 127, -0.0, 1.5 * 2.0 ** -130], dtype=np.float32)
    bits = (vals.view(np.uint32) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(oracle.bf16_bits_to_f64(bits), vals.astype(np.float64))


def test_round_scores_is_nearest_even():
    x = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24])
    r = oracle.round_scores(x)
    assert r[0] == np.float32(1.0) and r[1] == np.float32(1.0 + 2.0 ** -22)


def test_scoring_queries_split_rows_additively():
    # Column sums of per-row softmaxes add over disjoint query sets: scoring
    # with the first W-U positions' queries plus scoring with the last U
    # (the buffer alone, the ablation without bidirectional attention of
    # Sec. 5.3) gives Kara's score with all W.  A slip that took the wrong
    # rows for the narrowed set, or normalised over the query subset, breaks
    # the identity; each part also sums to its own number of rows.
    G, Hkv, W, U, d = 2, 2, 10, 3, 8
    q, pool, table, bs = _pool_case(G, Hkv, W, d, "f32", 5)
    p = dict(window=W, buffer=U, block_size=bs, n_q_heads=G * Hkv, n_kv_heads=Hkv,
             head_dim=d, dtype="f32", scale=0.0)
    p0 = 1
    full = oracle.score_units(p, [0], q, [pool], table, np.array([p0]), [(0, 0, 1)])[0]
    tail = oracle.score_units(dict(p, score_queries=U), [0], np.ascontiguousarray(q[:, :, W - U:]), [pool],
                              table, np.array([p0]), [(0, 0, 1)])[0]
    keys = oracle.unit_keys(pool, p, table[0], p0, 1)
    front = sum(oracle.window_scores(q[0, 0, :W - U, h, :].astype(np.float64), keys, 1 / math.sqrt(d))
                for h in (2, 3))
    np.testing.assert_allclose(front + tail, full, rtol=1e-12)
    assert abs(tail.sum() - G * U) < 1e-12
    # the buffer rows are the ones scoring: position W-1's query head 3
    # alone, as a single softmax row, is one term of the tail score
    last = oracle.window_scores(q[0, 0, W - 1:, 3, :].astype(np.float64), keys, 1 / math.sqrt(d))
    assert (tail >= last - 1e-15).all()


def test_scoring_queries_shape_checked():
    G, Hkv, W, d = 1, 1, 6, 8
    q, pool, table, bs = _pool_case(G, Hkv, W, d, "f32", 2)
    p = dict(window=W, buffer=2, block_size=bs, n_q_heads=1, n_kv_heads=1, head_dim=d, dtype="f32",
             scale=0.0, score_queries=2)
    with pytest.raises(ValueError):
        oracle.unit_queries(q, p, 0, 0, 0)
