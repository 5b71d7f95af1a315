"""Pins for the oracle's selection: discrete TopK, Eq. (5); Token2Chunk,
Eq. (6)-(8); and the fill rule of App. C.3 (Kara Sec. 4.1-4.2)."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "token2chunk_examples.json")


def _beats(a, i, j):
    """i ranks before j: larger score, or equal score and lower index."""
    return a[i] > a[j] or (a[i] == a[j] and i < j)


def _brute_topk(a, k):
    """The unique k-subset whose every member ranks before every non-member."""
    n = len(a)
    winners = []
    for sub in itertools.combinations(range(n), k):
        s = set(sub)
        if all(_beats(a, i, j) for i in s for j in range(n) if j not in s):
            winners.append(sorted(sub))
    assert len(winners) == 1
    return winners[0]


def _brute_chunks(a, disc, alpha, gamma):
    """Chunk choice by exhaustive search over subsets of the candidates."""
    cands = []
    for k in range(len(disc) - 1):
        lo, hi = disc[k], disc[k + 1]
        interior = list(range(lo + 1, hi))
        if 1 <= len(interior) and (hi - lo + 1) <= gamma:    # endpoints included
            score = (float(a[lo]) + float(a[hi])) * len(interior)
            cands.append((k, score, interior))
    want = min(alpha // (gamma - 2), len(cands))
    best = None
    for sub in itertools.combinations(range(len(cands)), want):
        inside = set(sub)
        ok = all(
            cands[c][1] > cands[o][1] or (cands[c][1] == cands[o][1] and cands[c][0] < cands[o][0])
            for c in inside for o in range(len(cands)) if o not in inside)
        if ok:
            assert best is None
            best = sub
    assert best is not None
    chosen = sorted(cands[c][0] for c in best)
    added = sorted(x for c in best for x in cands[c][2])
    return chosen, added


def test_ranking_example():
    g = json.load(open(GOLD))
    a = np.array(g["scores_12"], dtype=np.float32)
    assert list(oracle.rank_order(a)) == g["ranking_12"]


@pytest.mark.parametrize("ex", json.load(open(GOLD))["examples"], ids=lambda e: e["name"])
def test_hand_examples(ex):
    g = json.load(open(GOLD))
    a = np.array(g[ex["scores"]] if isinstance(ex["scores"], str) else ex["scores"], dtype=np.float32)
    disc = oracle.discrete_topk(a, ex["budget"] - ex["alpha"])
    assert list(disc) == ex["discrete"]
    cands = oracle.chunk_candidates(a, disc, ex["gamma"])
    assert sorted((k, r) for r, k in cands) == [tuple(c) for c in ex["candidates"]]
    chosen, added = oracle.token2chunk(a, disc, ex["alpha"], ex["gamma"])
    assert list(chosen) == ex["chosen"] and list(added) == ex["added"]
    disc2, kept = oracle.kept_set(a, ex["budget"], ex["alpha"], ex["gamma"])
    assert list(disc2) == ex["discrete"]
    assert list(kept) == ex["kept"]
    fill = sorted(set(kept) - set(disc) - set(added))
    assert fill == ex["fill"]


@pytest.mark.parametrize("seed", range(40))
def test_topk_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 10))
    a = rng.integers(0, 4, n).astype(np.float32)      # many ties
    k = int(rng.integers(0, n + 1))
    assert list(oracle.discrete_topk(a, k)) == _brute_topk(a, k)


@pytest.mark.parametrize("seed", range(60))
def test_token2chunk_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(4, 22))
    a = (rng.integers(0, 6, n) / 8.0).astype(np.float32)
    budget = int(rng.integers(2, n + 1))
    alpha = int(rng.integers(0, budget))
    gamma = int(rng.integers(3, 9))
    disc = list(oracle.discrete_topk(a, budget - alpha))
    chosen, added = oracle.token2chunk(a, np.array(disc), alpha, gamma)
    bchosen, badded = _brute_chunks(a, disc, alpha, gamma)
    assert list(chosen) == bchosen and list(added) == badded


@pytest.mark.parametrize("seed", range(60))
def test_kept_set_invariants(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(2, 300))
    if seed % 3 == 0:
        a = rng.integers(0, 5, n).astype(np.float32)
    else:
        a = rng.random(n).astype(np.float32)
    budget = int(rng.integers(1, n + 1))
    alpha = int(rng.integers(0, budget))
    gamma = int(rng.integers(3, 12))
    disc, kept = oracle.kept_set(a, budget, alpha, gamma)
    assert len(disc) == budget - alpha
    assert len(kept) == budget and len(set(kept.tolist())) == budget
    assert kept.min() >= 0 and kept.max() < n
    assert np.all(np.diff(kept) > 0) and np.all(np.diff(disc) > 0)
    assert set(disc.tolist()) <= set(kept.tolist())
    chosen, added = oracle.token2chunk(a, disc, alpha, gamma)
    assert len(chosen) <= alpha // (gamma - 2)
    assert len(added) <= alpha
    for k in chosen:
        lo, hi = disc[k], disc[k + 1]
        assert 2 <= hi - lo <= gamma - 1           # interior of at most gamma-2
    # every added position lies strictly between two consecutive discrete ones
    for x in added:
        j = np.searchsorted(disc, x)
        assert 0 < j < len(disc) and disc[j - 1] < x < disc[j]
    # fill: each filled position ranks before every position left out
    fill = sorted(set(kept.tolist()) - set(disc.tolist()) - set(added.tolist()))
    assert len(fill) == alpha - len(added)
    out = sorted(set(range(n)) - set(kept.tolist()))
    for f in fill:
        for o in out:
            assert _beats(a, f, o)


def test_alpha_zero_is_plain_topk():
    rng = np.random.default_rng(9)
    a = rng.random(64).astype(np.float32)
    disc, kept = oracle.kept_set(a, 13, 0, 8)
    np.testing.assert_array_equal(kept, disc)
    np.testing.assert_array_equal(kept, np.sort(np.argsort(-a, kind="stable")[:13]))


def test_all_equal_scores_keep_lowest_indices():
    a = np.full(50, 0.25, dtype=np.float32)
    for alpha, gamma in [(0, 3), (4, 4), (16, 8)]:
        _, kept = oracle.kept_set(a, 20, alpha, gamma)
        assert list(kept) == list(range(20))


def test_chunk_length_limit_counts_both_endpoints():
    # gamma is the maximum chunk length with both endpoints included (Eq. (7):
    # I[k+1]-I[k] < gamma): with gamma=5 the span 0..4 (5 positions) is a
    # candidate, the span 0..5 (6 positions) is not.
    a = np.array([1, 0, 0, 0, 1, 1], dtype=np.float32)
    assert oracle.chunk_candidates(a, np.array([0, 4]), 5) == [(2.0 * 3, 0)]
    assert oracle.chunk_candidates(a, np.array([0, 5]), 5) == []
    assert oracle.chunk_candidates(a, np.array([0, 1]), 5) == []      # empty interior
