"""GPU parity of each C-ABI entry point on its own, fed the oracle's output
of the previous stage: kara_score_window (tolerance), kara_select and
kara_token2chunk and kara_select_kept (bit-exact on given scores, including ties, negative
values and -0), kara_compact_pages and kara_commit_tables (bit-exact), plus
the library's handling of malformed caller input."""
import numpy as np
import pytest

import kara_inputs as ki
import oracle

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(scope="module")
def case():
    import kara_check as kc
    _need_gpu()
    return kc.setup(ki.workload("qwen14b", n_seqs=3, n_layers=2, window=512, budget=103, prefix=(17, 300)))


def test_score_window_matches_oracle(case):
    import kara_check as kc
    from paper_2607_01237_amd import kara
    p = case.p
    L, nt, H = len(case.kp), case.trig.numel(), p["n_kv_heads"]
    N = p["window"] - p["buffer"]
    ws = torch.empty(kara.workspace_size(case.params, nt, L), dtype=torch.uint8, device="cuda")
    scores = torch.full((L, nt, H, N), float("nan"), device="cuda")
    status = torch.full((nt,), -1, dtype=torch.int32, device="cuda")
    for _ in range(2):       # the split counters must be reusable call after call
        kara.score_window(case.params, case.trig, case.q, case.kp, case.bt, case.seq_lens, case.win_start,
                          scores, status, ws)
    torch.cuda.synchronize()
    ora, st = kc.oracle_scores(case)
    assert np.array_equal(status.cpu().numpy(), st)
    rep = kc.check_p1(scores.cpu().numpy(), ora)
    print("score_window", rep)


def _select_cases():
    rng = np.random.default_rng(7)
    yield "random", rng.random((6, 300)).astype(np.float32)
    yield "ties", rng.integers(0, 4, (6, 300)).astype(np.float32)
    a = rng.standard_normal((6, 300)).astype(np.float32)
    a[:, ::7] = -0.0
    a[:, 3::7] = 0.0
    yield "signed", a
    yield "equal", np.full((2, 300), 0.5, dtype=np.float32)
    # past 2048 positions the 16-position instance runs: ties and equal
    # scores there too, at a ragged length and at the largest one
    yield "ties_2049", rng.integers(0, 4, (3, 2049)).astype(np.float32)
    yield "ties_4096", rng.integers(0, 4, (3, 4096)).astype(np.float32)
    yield "equal_4096", np.full((2, 4096), 0.25, dtype=np.float32)
    yield "random_4096", rng.random((3, 4096)).astype(np.float32)


@pytest.mark.parametrize("name,scores", list(_select_cases()), ids=lambda x: x if isinstance(x, str) else "")
def test_select_and_token2chunk_bit_exact(name, scores):
    from paper_2607_01237_amd import kara
    _need_gpu()
    N = scores.shape[1]
    for budget, alpha, gamma in [(60, 16, 8), (60, 0, 8), (61, 20, 3), (300, 5, 4), (1, 0, 3)]:
        p = dict(window=N, buffer=0, budget=budget, chunk_budget=alpha, max_chunk_len=gamma, head_dim=128,
                 n_q_heads=8, n_kv_heads=8, block_size=16, num_pages=64, max_blocks_per_seq=64, dtype="bf16",
                 scale=0.0)
        par = kara.make_params(p, 1)
        sc = _dev(scores)
        disc = torch.full((scores.shape[0], budget - alpha), -9, dtype=torch.int32, device="cuda")
        kept = torch.full((scores.shape[0], budget), -9, dtype=torch.int32, device="cuda")
        kara.select(par, sc, disc)
        kara.token2chunk(par, sc, disc, kept)
        # the one-launch form the fused step runs
        disc1, kept1 = torch.full_like(disc, -9), torch.full_like(kept, -9)
        kara.select_kept(par, sc, disc1, kept1)
        torch.cuda.synchronize()
        d, k = disc.cpu().numpy(), kept.cpu().numpy()
        d1, k1 = disc1.cpu().numpy(), kept1.cpu().numpy()
        for u in range(scores.shape[0]):
            wd, wk = oracle.kept_set(scores[u], budget, alpha, gamma)
            assert np.array_equal(d[u], wd), (name, budget, alpha, gamma, u)
            assert np.array_equal(k[u], wk), (name, budget, alpha, gamma, u)
            assert np.array_equal(d1[u], wd), ("one launch", name, budget, alpha, gamma, u)
            assert np.array_equal(k1[u], wk), ("one launch", name, budget, alpha, gamma, u)


def test_token2chunk_rejects_bad_discrete():
    from paper_2607_01237_amd import kara
    _need_gpu()
    p = dict(window=64, buffer=0, budget=10, chunk_budget=4, max_chunk_len=4, head_dim=64, n_q_heads=1,
             n_kv_heads=1, block_size=16, num_pages=8, max_blocks_per_seq=8, dtype="f32", scale=0.0)
    par = kara.make_params(p, 1)
    sc = _dev(np.random.default_rng(0).random((3, 64)).astype(np.float32))
    disc = _dev(np.array([[0, 1, 2, 3, 4, 5], [5, 4, 3, 2, 1, 0], [0, 1, 2, 3, 4, 64]], dtype=np.int32))
    kept = torch.zeros((3, 10), dtype=torch.int32, device="cuda")
    kara.token2chunk(par, sc, disc, kept)
    k = kept.cpu().numpy()
    assert (k[0] >= 0).all() and (k[1] == -1).all() and (k[2] == -1).all()


def test_compact_and_commit_bit_exact(case):
    import kara_check as kc
    from paper_2607_01237_amd import kara
    p = case.p
    L, nt, H = len(case.kp), case.trig.numel(), p["n_kv_heads"]
    N = p["window"] - p["buffer"]
    rng = np.random.default_rng(3)
    scores = rng.random((L, nt, H, N)).astype(np.float32)
    kept = np.zeros((L, nt, H, p["budget"]), dtype=np.int32)
    for idx in np.ndindex(L, nt, H):
        kept[idx] = oracle.kept_set(scores[idx], p["budget"], p["chunk_budget"], p["max_chunk_len"])[1]
    status = torch.full((nt,), -1, dtype=torch.int32, device="cuda")
    freed = torch.full((nt, p["max_blocks_per_seq"]), -9, dtype=torch.int32, device="cuda")
    n_freed = torch.full((nt,), -9, dtype=torch.int32, device="cuda")
    # an event starts with a status-resetting call; then compact layer by
    # layer and commit once (the per-layer calling pattern)
    kara.validate(case.params, case.trig, case.bt, case.seq_lens, case.win_start, status)
    kg = _dev(kept)
    for l in range(L):
        kara.compact_pages(case.params, case.trig, kg[l:l + 1].contiguous(), case.kp[l:l + 1], case.vp[l:l + 1],
                           case.bt, case.seq_lens, case.win_start, status)
    kara.commit_tables(case.params, case.trig, case.bt, case.seq_lens, case.win_start, freed, n_freed, status)
    torch.cuda.synchronize()
    gpu = dict(scores=scores, kept=kept, status=status.cpu().numpy(), bt=case.bt.cpu().numpy(),
               seq_lens=case.seq_lens.cpu().numpy(), freed=freed.cpu().numpy(), n_freed=n_freed.cpu().numpy())
    kc.check_p4(case, gpu, commit=True)


def test_compact_rejects_bad_kept():
    import kara_check as kc
    from paper_2607_01237_amd import kara
    _need_gpu()
    c = kc.setup(ki.workload("batch8", n_seqs=2, window=256, budget=52))
    p = c.p
    nt, H = c.trig.numel(), p["n_kv_heads"]
    kept = np.tile(np.arange(p["budget"], dtype=np.int32), (1, nt, H, 1))
    kept[0, 1, 3, 5] = kept[0, 1, 3, 4]          # not strictly ascending in sequence 1
    before = [ki.raw_numpy(t) for t in c.kp]
    status = torch.full((nt,), -1, dtype=torch.int32, device="cuda")
    kara.validate(c.params, c.trig, c.bt, c.seq_lens, c.win_start, status)
    kara.compact_pages(c.params, c.trig, _dev(kept), c.kp, c.vp, c.bt, c.seq_lens, c.win_start, status)
    torch.cuda.synchronize()
    st = status.cpu().numpy()
    assert st[0] == 0 and st[1] == kara.SEQ_BAD_KEPT
    after = ki.raw_numpy(c.kp[0])
    s1 = int(c.geom.trig[1])
    pos = np.arange(c.geom.win_start[s1], c.geom.seq_lens[s1])
    pg = c.geom.block_table[s1, pos // p["block_size"]]
    assert np.array_equal(after[pg, :, pos % p["block_size"]], before[0][pg, :, pos % p["block_size"]])


def test_bad_kept_in_a_later_layer_stops_the_commit():
    """Per-layer compaction: a bad kept set found in layer 1's call keeps the
    sequence flagged through the commit, which then leaves its table,
    length and freed list alone; the other sequence commits normally."""
    import kara_check as kc
    from paper_2607_01237_amd import kara
    _need_gpu()
    c = kc.setup(ki.workload("batch8", n_seqs=2, n_layers=2, window=256, budget=52))
    p = c.p
    nt, H, L = c.trig.numel(), p["n_kv_heads"], 2
    kept = np.tile(np.arange(p["budget"], dtype=np.int32) * 2, (L, nt, H, 1))
    kept[1, 1, 2, 7] = kept[1, 1, 2, 6]          # layer 1, sequence 1: not strictly ascending
    bt0, sl0 = c.bt.cpu().numpy().copy(), c.seq_lens.cpu().numpy().copy()
    status = torch.full((nt,), -1, dtype=torch.int32, device="cuda")
    freed = torch.full((nt, p["max_blocks_per_seq"]), -9, dtype=torch.int32, device="cuda")
    n_freed = torch.full((nt,), -9, dtype=torch.int32, device="cuda")
    kara.validate(c.params, c.trig, c.bt, c.seq_lens, c.win_start, status)
    kg = _dev(kept)
    for l in range(L):
        kara.compact_pages(c.params, c.trig, kg[l:l + 1].contiguous(), c.kp[l:l + 1], c.vp[l:l + 1], c.bt,
                           c.seq_lens, c.win_start, status)
    kara.commit_tables(c.params, c.trig, c.bt, c.seq_lens, c.win_start, freed, n_freed, status)
    torch.cuda.synchronize()
    st, bt, sl = status.cpu().numpy(), c.bt.cpu().numpy(), c.seq_lens.cpu().numpy()
    fr, nf = freed.cpu().numpy(), n_freed.cpu().numpy()
    s0, s1 = int(c.geom.trig[0]), int(c.geom.trig[1])
    assert st[0] == 0 and st[1] == kara.SEQ_BAD_KEPT, st
    assert np.array_equal(bt[s1], bt0[s1]) and sl[s1] == sl0[s1]
    assert nf[1] == 0 and (fr[1] == -1).all()
    N = p["window"] - p["buffer"]
    assert sl[s0] == sl0[s0] - (N - p["budget"]) and nf[0] > 0


def test_page_mapped_twice_is_flagged():
    """A window whose block table maps one page at two blocks is flagged
    KARA_SEQ_DUP_PAGE and left untouched; the others compress as the
    oracle does (P1-P4)."""
    import kara_check as kc
    _need_gpu()
    cfg = ki.workload("batch8", n_seqs=3, window=256, budget=52)
    geom = ki.make_geometry(cfg)
    bt = geom.block_table.copy()
    s = int(geom.trig[1])
    b0 = int(geom.win_start[s]) // geom.params()["block_size"]
    bt[s, b0 + 3] = bt[s, b0 + 1]
    case = kc.setup(cfg, block_table=bt)
    rep, gpu = kc.full_check(case)
    assert gpu["status"][1] == oracle.SEQ_DUP_PAGE and gpu["status"][0] == 0 and gpu["status"][2] == 0
    print("dup page", rep)
