"""Pins for the oracle's prefill-time compression (App. C.2).

Windows of the prompt are compressed all at once (oracle.compress_prefill).
The paper's decoding-time step compresses one window and advances by
|W|-|U|; compressing the same windows one after another with the
single-window step must leave the same cache, because a window's contents
are untouched by the compaction of earlier windows (they only shift down).
That identity, and the one-window case, pin the multi-window composition:
a wrong window offset, a window's kept rows applied to another window, or a
wrong length or block release breaks one of them.
"""
import copy

import numpy as np
import pytest

import oracle


def _case(seed, W, U, nw, bs, L=2, Hkv=2, G=2, d=8, n_seqs=3):
    rng = np.random.default_rng(seed)
    N = W - U
    p = dict(window=W, buffer=U, budget=5, chunk_budget=2, max_chunk_len=4, head_dim=d, n_q_heads=G * Hkv,
             n_kv_heads=Hkv, block_size=bs, dtype="f32", scale=0.0)
    p0 = np.array([0, 7, 3])[:n_seqs]
    tail = np.array([2, 0, 5])[:n_seqs]
    lens = p0 + (nw - 1) * N + W + tail
    max_blocks = int(-(-lens.max() // bs))
    pages = n_seqs * max_blocks + 4
    perm = rng.permutation(pages)
    table = np.full((n_seqs, max_blocks), -1, dtype=np.int64)
    c = 0
    for s in range(n_seqs):
        nb = -(-int(lens[s]) // bs)
        table[s, :nb] = perm[c:c + nb]
        c += nb
    p.update(num_pages=pages, max_blocks_per_seq=max_blocks)
    kp = [rng.standard_normal((pages, Hkv, bs, d)).astype(np.float32) for _ in range(L)]
    vp = [rng.standard_normal((pages, Hkv, bs, d)).astype(np.float32) for _ in range(L)]
    trig = np.array([2, 0, 1]) if n_seqs == 3 else np.arange(n_seqs)
    q = rng.standard_normal((L, n_seqs, nw, W, G * Hkv, d)).astype(np.float32)
    return p, trig, q, kp, vp, table, lens.astype(np.int64), p0.astype(np.int64)


def _rows(pool, table_row, n, h, bs):
    return oracle.read_rows(pool, table_row, np.arange(n), h, bs)


@pytest.mark.parametrize("W,U,nw,bs", [(16, 0, 3, 5), (16, 3, 3, 5), (12, 4, 4, 4), (16, 3, 1, 6)])
def test_prefill_equals_windows_one_after_another(W, U, nw, bs):
    p, trig, q, kp, vp, table, lens, p0 = _case(W * 100 + U * 10 + nw, W, U, nw, bs)
    N = W - U
    # all windows at once
    kp_a, vp_a = copy.deepcopy(kp), copy.deepcopy(vp)
    tab_a, len_a = table.copy(), lens.copy()
    out = oracle.compress_prefill(p, trig, nw, q, kp_a, vp_a, tab_a, len_a, p0)
    assert (out["status"] == 0).all()
    # one window at a time: window w starts at p0 + w*budget once the earlier
    # windows have been compressed (w*(N-budget) positions fewer before it)
    kp_b, vp_b = copy.deepcopy(kp), copy.deepcopy(vp)
    tab_b, len_b = table.copy(), lens.copy()
    freed_b = [[] for _ in trig]
    for w in range(nw):
        starts = p0 + w * p["budget"]
        o = oracle.compress(p, trig, np.ascontiguousarray(q[:, :, w]), kp_b, vp_b, tab_b, len_b, starts)
        assert (o["status"] == 0).all()
        np.testing.assert_array_equal(o["scores"], out["scores"][:, :, w])
        np.testing.assert_array_equal(o["kept"], out["kept"][:, :, w])
        for t in range(len(trig)):
            freed_b[t] += o["freed"][t]
    np.testing.assert_array_equal(len_a, len_b)
    np.testing.assert_array_equal(tab_a, tab_b)
    np.testing.assert_array_equal(len_a[trig], lens[trig] - nw * (N - p["budget"]))
    for t, s in enumerate(trig):
        assert sorted(out["freed"][t]) == sorted(freed_b[t])
        for l in range(len(kp)):
            for h in range(p["n_kv_heads"]):
                for A, B in ((kp_a, kp_b), (vp_a, vp_b)):
                    np.testing.assert_array_equal(_rows(A[l], tab_a[s], len_a[s], h, p["block_size"]),
                                                  _rows(B[l], tab_b[s], len_b[s], h, p["block_size"]))


def test_prefill_layout_and_short_prompt():
    # the cache after compression: window 0's kept rows, window 1's kept rows
    # (offset by N), then the last window's buffer and the rest, in order
    W, U, nw, bs = 10, 2, 2, 4
    p, trig, q, kp, vp, table, lens, p0 = _case(5, W, U, nw, bs, L=1, Hkv=1, G=1, n_seqs=1)
    N = W - U
    s = int(trig[0])
    before = _rows(kp[0], table[s], int(lens[s]), 0, bs)
    out = oracle.compress_prefill(p, trig, nw, q, kp, vp, table, lens, p0)
    k0, k1 = out["kept"][0, 0, 0, 0], out["kept"][0, 0, 1, 0]
    a = int(p0[s])
    want = np.concatenate([before[:a], before[a + k0], before[a + N + k1], before[a + 2 * N:]])
    np.testing.assert_array_equal(_rows(kp[0], table[s], int(lens[s]), 0, bs), want)
    # a prompt one token too short for its windows is flagged and untouched
    p, trig, q, kp, vp, table, lens, p0 = _case(6, W, U, nw, bs, L=1, Hkv=1, G=1, n_seqs=1)
    s = int(trig[0])
    lens[s] = p0[s] + (nw - 1) * N + W - 1
    out = oracle.compress_prefill(p, trig, nw, q, kp, vp, table, lens, p0)
    assert out["status"][0] == oracle.SEQ_BAD_WINDOW
