"""The parity checkers themselves, on the CPU: what they must accept and what
they must reject.  Mistakes are planted in oracle-made results, never run on
a GPU.

P3 (tests/kara_check.p3_unit) replays each selection stage of Eq. (5)-(8)
and App. C.3 with the oracle's scores on the GPU's previous-stage result and
accepts a difference only as swaps across that stage's boundary within the
propagated score tolerance.  The cases are built on a ten-position window
with budget 5, alpha 2, gamma 4 (k = 3 discrete positions, n_c = 1 chunk,
fill up to 2).

The recompute attention check (kara_check.check_attention) must accept an
output carrying exactly the kernel's rounding (bf16 weights, normalised by
their own sum, bf16 store) and reject one key dropped or read twice at the
2048-entry block-table segment switch.
"""
import numpy as np
import pytest
import torch

import kara_check as kc
import oracle
from oracle import kara_recompute as rc

P = dict(budget=5, chunk_budget=2, max_chunk_len=4)


def _base():
    # discrete top-3 = {0, 2, 4}; candidates (0,2) R = 1.7 and (2,4) R = 1.4;
    # the chunk (0,2) adds 1; the fill then takes 6 (0.5)
    return np.array([0.9, 0.1, 0.8, 0.1, 0.6, 0.01, 0.5, 0.01, 0.02, 0.01], dtype=np.float32)


def _gpu_from(a_gpu):
    """What a correct GPU returns on its own scores a_gpu (P2 holds)."""
    d, k = oracle.kept_set(a_gpu, P["budget"], P["chunk_budget"], P["max_chunk_len"])
    return d, k


def test_p1_rejects_non_finite_and_out_of_tolerance_scores():
    rng = np.random.default_rng(3)
    ora = rng.uniform(0.0, 4.0, size=(2, 64)).astype(np.float32)
    ora[0, 5] = 0.0
    kc.check_p1(ora.copy(), ora)
    near = ora * np.float32(1 + 1.5e-3)
    kc.check_p1(near, ora)
    for planted in (np.nan, np.inf, -np.inf):
        got = ora.copy()
        got[1, 7] = planted
        with pytest.raises(AssertionError):
            kc.check_p1(got, ora)
    got = ora.copy()
    got[0, 5] = 2e-5          # past the 1e-5 absolute tolerance of a zero score
    with pytest.raises(AssertionError):
        kc.check_p1(got, ora)
    got = ora.copy()
    got[1, 9] *= np.float32(1.003)
    with pytest.raises(AssertionError):
        kc.check_p1(got, ora)


def test_base_case_is_what_the_comments_say():
    d, k = _gpu_from(_base())
    assert d.tolist() == [0, 2, 4] and k.tolist() == [0, 1, 2, 4, 6]


def test_identical_results_pass_and_count_zero():
    a = _base()
    d, k = _gpu_from(a)
    assert kc.p3_unit(a, a, d, k, P) is False


def test_discrete_near_tie_swap_accepted():
    a = _base()
    a[6] = np.float32(0.5999)                       # 4 (0.6) and 6 within tolerance
    g = a.copy()
    g[6], g[4] = np.float32(0.6001), np.float32(0.5999)
    d, k = _gpu_from(g)
    assert d.tolist() == [0, 2, 6]
    kc.p3_unit(a, g, d, k, P)                       # accepted (kept sets may or may not differ)


def test_discrete_swap_away_from_the_boundary_rejected():
    a = _base()
    d = np.array([0, 2, 8])                         # 8 (0.02) in place of 4 (0.6)
    _, added = oracle.token2chunk(a, d, P["chunk_budget"], P["max_chunk_len"])
    taken = np.zeros(len(a), bool)
    taken[d] = True
    taken[added] = True
    fill = oracle.fill_positions(a, taken, P["chunk_budget"] - len(added))
    taken[fill] = True
    with pytest.raises(AssertionError, match="discrete set"):
        kc.p3_unit(a, a, d, np.flatnonzero(taken), P)


def test_chunk_tie_swap_accepted():
    a = _base()
    a[4] = np.float32(0.9)                          # (0,2) and (2,4) both R = 1.7: a tie
    g = a.copy()
    g[0] = np.float32(0.8999)                       # the GPU's scores put (2,4) first
    d, k = _gpu_from(g)
    _, k_ora = _gpu_from(a)
    assert not np.array_equal(k, k_ora)
    assert kc.p3_unit(a, g, d, k, P) is True


def test_chunk_choice_away_from_the_boundary_rejected():
    a = _base()
    g = a.copy()
    g[0] = np.float32(0.59)                         # discrete set unchanged, (2,4) now first
    d, k = _gpu_from(g)
    assert d.tolist() == [0, 2, 4] and 3 in k
    with pytest.raises(AssertionError, match="chunk choice"):
        kc.p3_unit(a, g, d, k, P)


def test_fill_near_tie_swap_accepted():
    a = _base()
    a[8] = np.float32(0.4999)
    g = a.copy()
    g[8] = np.float32(0.5001)
    d, k = _gpu_from(g)
    assert 8 in k and 6 not in k
    assert kc.p3_unit(a, g, d, k, P) is True


def test_fill_away_from_the_boundary_rejected():
    a = _base()
    d, k = _gpu_from(a)
    planted = np.sort(np.concatenate([k[k != 6], [7]]))     # 7 (0.01) in place of 6 (0.5)
    with pytest.raises(AssertionError, match="fill"):
        kc.p3_unit(a, a, d, planted, P)


def test_kept_set_not_made_of_the_stages_rejected():
    a = _base()
    d, k = _gpu_from(a)
    planted = np.sort(np.concatenate([k[k != 1], [3]]))     # drop the chunk interior
    with pytest.raises(AssertionError):
        kc.p3_unit(a, a, d, planted, P)


def test_random_units_with_in_tolerance_noise_pass():
    """Scores perturbed within the P1 tolerance: whatever the GPU's selection
    does with them, P3 accepts it."""
    rng = np.random.default_rng(3)
    p = dict(budget=52, chunk_budget=16, max_chunk_len=8)
    differ = 0
    for _ in range(40):
        a = (rng.random(256) ** 3).astype(np.float32)
        a[rng.integers(256, size=20)] = a[rng.integers(256, size=20)]       # exact ties
        g = (a.astype(np.float64) + rng.uniform(-1, 1, 256) * 0.9 * kc.tol(a)).astype(np.float32)
        d, k = oracle.kept_set(g, p["budget"], p["chunk_budget"], p["max_chunk_len"])
        differ += kc.p3_unit(a, g, d, k, p)
    assert differ > 0          # the noise did move some decisions


# ---- recompute attention ----

def _bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


def _kernel_model(q, k_rows, v_rows, p0, scale, drop=None, dup=None):
    """Attention with the kernel's roundings: bf16 weights normalised by their
    own sum, bf16 output.  drop: a key position left out; dup: (a, b) key b
    read in place of key a."""
    W, Hq, d = q.shape
    G = Hq // k_rows.shape[1]
    out = np.zeros((W, Hq, d))
    for w in range(W):
        n = p0 + w + 1
        idx = np.arange(n)
        if drop is not None:
            idx = idx[idx != drop]
        if dup is not None:
            idx = np.where(idx == dup[0], dup[1], idx)
        for hq in range(Hq):
            h = hq // G
            x = (k_rows[idx, h, :] @ q[w, hq, :]) * scale
            e = _bf16(np.exp2((x - x.max()) * np.log2(np.e)))
            out[w, hq] = e @ v_rows[idx, h, :] / e.sum()
    return _bf16(out)


@pytest.fixture(scope="module")
def attn_case():
    rng = np.random.default_rng(5)
    W, Hq, Hkv, d, p0 = 6, 4, 2, 64, 2050
    bf = lambda a: _bf16(a)
    q = bf(rng.standard_normal((W, Hq, d)))
    k = bf(rng.standard_normal((p0 + W, Hkv, d)))
    v = bf(rng.standard_normal((p0 + W, Hkv, d)))
    scale = 1.0 / np.sqrt(d)
    o = rc.causal_window_attention(q, k, v, p0, scale)
    spread = kc.attention_spread(q, k, v, p0, scale, o)
    return dict(q=q, k=k, v=v, p0=p0, scale=scale, o=o, spread=spread)


def test_attention_check_accepts_the_kernels_rounding(attn_case):
    c = attn_case
    got = _kernel_model(c["q"], c["k"], c["v"], c["p0"], c["scale"])
    kc.check_attention(got, c["o"], c["spread"], "rounding model")


@pytest.mark.parametrize("planted,key", [("drop", 2048), ("drop", 2049), ("drop", 2050), ("dup", 2048)])
def test_attention_check_rejects_one_key_wrong_at_the_segment_switch(attn_case, planted, key):
    c = attn_case
    kw = dict(drop=key) if planted == "drop" else dict(dup=(key, key - 1))
    got = _kernel_model(c["q"], c["k"], c["v"], c["p0"], c["scale"], **kw)
    with pytest.raises(AssertionError, match="out of tolerance"):
        kc.check_attention(got, c["o"], c["spread"], planted)

