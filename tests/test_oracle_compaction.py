"""Pins for the oracle's window gather, Eq. (9), and the memory compaction,
block release and metadata update of Algorithm 1 (Kara App. C.4)."""
import json
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "compaction_example.json")


def _params(**kw):
    p = dict(window=8, buffer=0, budget=3, chunk_budget=0, max_chunk_len=3, head_dim=2,
             n_q_heads=1, n_kv_heads=1, block_size=4, num_pages=8, max_blocks_per_seq=6,
             dtype="f32", scale=0.0)
    p.update(kw)
    return p


def _position_pool(p, table, seq_lens, n_heads=1, seed=None):
    """Pool whose row at (seq, pos, head) holds (seq*1000 + pos, head)."""
    pool = np.full((p["num_pages"], n_heads, p["block_size"], 2), -1.0, dtype=np.float32)
    for s in range(table.shape[0]):
        for pos in range(seq_lens[s]):
            pg = table[s, pos // p["block_size"]]
            for h in range(n_heads):
                pool[pg, h, pos % p["block_size"]] = (s * 1000 + pos, h)
    return pool


def test_hand_example():
    g = json.load(open(GOLD))
    p = _params(window=g["window"], buffer=g["buffer"], budget=g["budget"], block_size=g["block_size"])
    N = p["window"] - p["buffer"]
    table = np.array([[5, 2, 7, 0, -1, -1]], dtype=np.int64)
    seq_lens = np.array([g["seq_len"]])
    win = np.array([g["window_start"]])
    k_pool = _position_pool(p, table, seq_lens)
    v_pool = k_pool.copy()
    scores = np.zeros((1, 1, 1, N), dtype=np.float32)
    scores[0, 0, 0, g["kept"]] = 1.0
    q = np.zeros((1, 1, p["window"], 1, 2), dtype=np.float32)
    out = oracle.compress(p, [0], q, [k_pool], [v_pool], table, seq_lens, win, score_override=scores)
    assert list(out["kept"][0, 0, 0]) == g["kept"]
    assert list(oracle.compaction_map(np.array(g["kept"]), p["window"], p["buffer"], 3)) == g["map"]
    assert seq_lens[0] == g["new_len"]
    assert list(np.flatnonzero(table[0] == -1)) == [3, 4, 5]
    assert out["freed"][0] == [0] and out["n_freed"][0] == 1
    live = oracle.read_rows(k_pool, table[0], np.arange(g["new_len"]), 0, p["block_size"])[:, 0]
    want = [0, 1] + [g["window_start"] + m for m in g["map"]]
    assert list(live) == want
    np.testing.assert_array_equal(k_pool, v_pool)


def test_full_budget_moves_nothing():
    p = _params(budget=8, window=8)
    table = np.array([[3, 1, 6, 0, 2, -1]], dtype=np.int64)
    seq_lens = np.array([19])
    win = np.array([5])
    pool = _position_pool(p, table, seq_lens)
    before = pool.copy()
    scores = np.random.default_rng(0).random((1, 1, 1, 8)).astype(np.float32)
    q = np.zeros((1, 1, 8, 1, 2), dtype=np.float32)
    out = oracle.compress(p, [0], q, [pool], [pool.copy()], table, seq_lens, win, score_override=scores)
    np.testing.assert_array_equal(pool, before)
    assert seq_lens[0] == 19 and out["n_freed"][0] == 0 and list(table[0]) == [3, 1, 6, 0, 2, -1]


@pytest.mark.parametrize("seed", range(12))
def test_random_invariants(seed):
    rng = np.random.default_rng(seed)
    bs = int(rng.choice([2, 4, 16]))
    W = int(rng.integers(4, 40))
    U = int(rng.integers(0, W))
    N = W - U
    budget = int(rng.integers(1, N + 1))
    H = int(rng.integers(1, 3))
    B = 4
    maxb = 40
    lens, wins = [], []
    for s in range(B):
        p0 = int(rng.integers(0, 50))
        tail = int(rng.integers(0, 20))
        wins.append(p0)
        lens.append(p0 + W + tail)
    need = sum(-(-L // bs) for L in lens)
    num_pages = need + 5
    perm = rng.permutation(num_pages)
    table = np.full((B, maxb), -1, dtype=np.int64)
    c = 0
    for s in range(B):
        nb = -(-lens[s] // bs)
        table[s, :nb] = perm[c:c + nb]
        c += nb
    p = _params(window=W, buffer=U, budget=budget, chunk_budget=0, block_size=bs,
                num_pages=num_pages, max_blocks_per_seq=maxb, n_kv_heads=H, n_q_heads=H)
    seq_lens = np.array(lens)
    win = np.array(wins)
    kp = _position_pool(p, table, seq_lens, H)
    vp = kp + 0.5
    orig_k, orig_table, orig_lens = kp.copy(), table.copy(), seq_lens.copy()
    trig = [2, 0]
    scores = rng.random((1, 2, H, N)).astype(np.float32)
    q = np.zeros((1, 2, W, H, 2), dtype=np.float32)
    out = oracle.compress(p, trig, q, [kp], [vp], table, seq_lens, win, score_override=scores)
    for t, s in enumerate(trig):
        new_len = orig_lens[s] - (N - budget)
        assert seq_lens[s] == new_len
        old_b, new_b = -(-orig_lens[s] // bs), -(-new_len // bs)
        assert out["n_freed"][t] == old_b - new_b
        assert out["freed"][t] == list(orig_table[s, new_b:old_b])
        assert np.all(table[s, new_b:] == -1)
        np.testing.assert_array_equal(table[s, :new_b], orig_table[s, :new_b])
        tail = orig_lens[s] - win[s] - W
        for h in range(H):
            live = oracle.read_rows(kp, table[s], np.arange(new_len), h, bs)
            before = oracle.read_rows(orig_k, orig_table[s], np.arange(orig_lens[s]), h, bs)
            np.testing.assert_array_equal(live[:win[s]], before[:win[s]])       # prefix untouched
            m = oracle.compaction_map(out["kept"][0, t, h], W, U, tail)
            np.testing.assert_array_equal(live[win[s]:], before[win[s] + m])
            np.testing.assert_array_equal(oracle.read_rows(vp, table[s], np.arange(new_len), h, bs), live + 0.5)
    for s in (1, 3):   # sequences not triggered are untouched
        for h in range(H):
            a = oracle.read_rows(kp, table[s], np.arange(seq_lens[s]), h, bs)
            b = oracle.read_rows(orig_k, orig_table[s], np.arange(orig_lens[s]), h, bs)
            np.testing.assert_array_equal(a, b)
    # pages are conserved: what the tables still hold plus what was freed
    held = set(table[table >= 0].tolist()) | {x for f in out["freed"] for x in f}
    assert held == set(orig_table[orig_table >= 0].tolist())


def test_validation_flags_and_leaves_flagged_untouched():
    p = _params(window=8, budget=3, num_pages=20, max_blocks_per_seq=6)
    table = np.array([[0, 1, 2, 3, -1, -1],
                      [4, 5, 6, 7, -1, -1],
                      [8, 9, 99, 10, -1, -1],
                      [11, 12, 13, 14, -1, -1]], dtype=np.int64)
    seq_lens = np.array([13, 13, 13, 5])
    win = np.array([2, 2, 2, 0])
    trig = [0, 1, 2, 3, 1, 7]
    st = oracle.validate(p, np.array(trig), table, seq_lens, win)
    assert list(st) == [0, oracle.SEQ_DUP_TRIGGER, oracle.SEQ_BAD_PAGE, oracle.SEQ_BAD_WINDOW,
                        oracle.SEQ_DUP_TRIGGER, oracle.SEQ_BAD_INDEX]
    pool = _position_pool(p, np.where(table >= 20, 0, table), seq_lens)
    before = pool.copy()
    tb = table.copy()
    scores = np.random.default_rng(1).random((1, 2, 1, 8)).astype(np.float32)
    q = np.zeros((1, 2, 8, 1, 2), dtype=np.float32)
    out = oracle.compress(p, [2, 3], q, [pool], [pool.copy()], table, seq_lens, win, score_override=scores)
    assert list(out["status"]) == [oracle.SEQ_BAD_PAGE, oracle.SEQ_BAD_WINDOW]
    np.testing.assert_array_equal(pool, before)
    np.testing.assert_array_equal(table, tb)
    assert list(seq_lens) == [13, 13, 13, 5]



def test_validation_flags_a_page_mapped_twice():
    """R-PAGES: a page compaction writes may hold no other block of the same
    sequence.  Sequence 0 maps page 5 twice inside its window; sequence 1 maps
    its prefix page again at the window's last block; sequence 2 repeats a
    page inside the prefix only, which compaction never writes; sequence 3
    has an out-of-pool page and a duplicate (both bits)."""
    p = _params(window=8, budget=3, num_pages=40, max_blocks_per_seq=6)
    table = np.array([[0, 1, 5, 5, -1, -1],
                      [6, 7, 8, 6, -1, -1],
                      [9, 9, 10, 11, -1, -1],
                      [12, 13, 99, 13, -1, -1]], dtype=np.int64)
    seq_lens = np.array([13, 13, 16, 13])
    win = np.array([4, 4, 8, 4])
    st = oracle.validate(p, np.arange(4), table, seq_lens, win)
    assert list(st) == [oracle.SEQ_DUP_PAGE, oracle.SEQ_DUP_PAGE, 0,
                        oracle.SEQ_BAD_PAGE | oracle.SEQ_DUP_PAGE]
    # flagged sequences are neither compacted nor committed
    pool = _position_pool(p, np.where(table >= 40, 0, table), seq_lens)
    before, tb = pool.copy(), table.copy()
    scores = np.random.default_rng(2).random((1, 2, 1, 8)).astype(np.float32)
    q = np.zeros((1, 2, 8, 1, 2), dtype=np.float32)
    out = oracle.compress(p, [0, 1], q, [pool], [pool.copy()], table, seq_lens, win, score_override=scores)
    assert list(out["status"]) == [oracle.SEQ_DUP_PAGE, oracle.SEQ_DUP_PAGE]
    np.testing.assert_array_equal(pool, before)
    np.testing.assert_array_equal(table, tb)

def test_device_compaction_checker_on_the_oracle():
    """The all-units compaction check of the full-size GPU test, run on the
    CPU: it accepts the oracle's compaction and rejects a swapped row, a row
    of the wrong head and a changed row before the window."""
    torch = pytest.importorskip("torch")
    import kara_check as kc
    import kara_inputs as ki

    cfg = ki.workload("batch8", n_seqs=3, n_layers=2, buffer=32, budget=199, prefix=(40, 300), tail=(0, 15),
                      num_pages=512)
    geom = ki.make_geometry(cfg)
    p = geom.params()
    L, nt, H, bs = cfg["n_layers"], len(geom.trig), p["n_kv_heads"], p["block_size"]
    W, U, N = p["window"], p["buffer"], p["window"] - p["buffer"]
    kp, vp = zip(*(ki.make_pools(geom, l, "cpu") for l in range(L)))
    kp, vp = list(kp), list(vp)
    # rows before the window carry data too, so that a write there shows
    for pools in (kp, vp):
        for pool in pools:
            pool.add_(torch.randn(pool.shape, generator=torch.Generator().manual_seed(5)).to(pool.dtype))
    snap = kc.WindowSnapshot(geom, kp, vp)

    rng = np.random.default_rng(3)
    kept = np.zeros((L, nt, H, p["budget"]), dtype=np.int32)
    for l in range(L):
        for t, s in enumerate(geom.trig):
            p0, old = int(geom.win_start[s]), int(geom.seq_lens[s])
            pos = np.arange(p0, old)
            pg, sl = geom.block_table[s, pos // bs], pos % bs
            for h in range(H):
                a = rng.random(N).astype(np.float32)
                _, kept[l, t, h] = oracle.kept_set(a, p["budget"], p["chunk_budget"], p["max_chunk_len"])
                for pool in (kp[l], vp[l]):
                    rows = pool[pg, h, sl, :].view(torch.int16).numpy()     # raw bf16 bits
                    moved = oracle.gather_rows(rows, kept[l, t, h], W, U)
                    pool[pg[:len(moved)], h, sl[:len(moved)], :] = torch.from_numpy(moved).view(torch.bfloat16)
    kept_t = torch.from_numpy(kept)
    snap.check(geom, p, kept_t, kp, vp)

    s0 = int(geom.trig[1])
    p0 = int(geom.win_start[s0])
    page, slot = lambda x: int(geom.block_table[s0, x // bs]), lambda x: x % bs

    # a swapped pair of kept rows (layer 1, head 0, destinations 3 and 4)
    a_, b_ = p0 + 3, p0 + 4
    ra, rb = vp[1][page(a_), 0, slot(a_)].clone(), vp[1][page(b_), 0, slot(b_)].clone()
    vp[1][page(a_), 0, slot(a_)], vp[1][page(b_), 0, slot(b_)] = rb, ra
    with pytest.raises(AssertionError, match="V kept rows of layer 1"):
        snap.check(geom, p, kept_t, kp, vp)
    vp[1][page(a_), 0, slot(a_)], vp[1][page(b_), 0, slot(b_)] = ra, rb

    # a buffer row taken from the neighbouring head
    d_ = p0 + p["budget"] + 2
    r0 = kp[0][page(d_), 1, slot(d_)].clone()
    kp[0][page(d_), 1, slot(d_)] = kp[0][page(d_), 0, slot(d_)]
    with pytest.raises(AssertionError, match="K buffer/tail rows of layer 0"):
        snap.check(geom, p, kept_t, kp, vp)
    kp[0][page(d_), 1, slot(d_)] = r0

    # a row before the window overwritten
    x = p0 - 1
    kp[1][page(x), 2, slot(x), 5] += 1
    with pytest.raises(AssertionError, match="rows before the window, layer 1"):
        snap.check(geom, p, kept_t, kp, vp)
