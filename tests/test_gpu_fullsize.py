"""Parity at full size, in the launch configuration bench.py times.

The whole workload -- 64 sequences x 40 layers of the Qwen3-14B shape with
W = 2048, and the 256-sequence, 36-layer ragged one -- goes through one
kara_compress_window call over all layers, exactly as the bench runs it.
The oracle then checks what it can compute one unit at a time:
  P1  scores of at least 64 sampled units covering every layer and KV
      head, fp64, against the GPU's;
  P2  the oracle's selection on the GPU's scores, for every unit;
  P3  the oracle's end-to-end kept set of the P1 units (swaps across a
      near-tie boundary excepted);
  P4  the compacted K/V rows of the P1 units, and the block tables, lengths
      and freed lists of every sequence.
Only the sampled units' rows are copied to the host (the pools are ~140 GB).
For every unit, compaction is also checked on the device against its
definition: each row written equals, bit for bit, the row the compaction
map names in a device snapshot of [p0, seq_len) taken before the call, and
the rows before p0 keep their checksums.  That check uses torch indexing
only, not the library.
"""
import numpy as np
import pytest

import kara_inputs as ki
import oracle

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _units_sample(rng, L, nt, H, n):
    """At least n units: the corners, one unit of every layer (its head
    cycling through every KV head, a random trigger), then random ones."""
    units = {(0, 0, 0), (L - 1, nt - 1, H - 1), (L // 2, nt // 2, H // 2), (L - 1, 0, H - 1)}
    for l in range(L):
        units.add((l, int(rng.integers(nt)), l % H))
    for h in range(H):
        units.add((int(rng.integers(L)), int(rng.integers(nt)), h))
    while len(units) < n:
        units.add((int(rng.integers(L)), int(rng.integers(nt)), int(rng.integers(H))))
    return sorted(units)


def _rows(pool, table_row, positions, head, bs):
    """One head's rows at logical positions, as raw host values."""
    pg = torch.from_numpy(table_row[positions // bs].astype(np.int64)).to(pool.device)
    sl = torch.from_numpy((positions % bs).astype(np.int64)).to(pool.device)
    return ki.raw_numpy(pool[pg, head, sl, :])


@pytest.mark.parametrize("name,n_p1", [("qwen14b", 64), ("ragged", 64)])
def test_fullsize_sampled(name, n_p1):
    import kara_check as kc
    from paper_2607_01237_amd import kara
    _need_gpu()
    torch.cuda.empty_cache()          # the pools take most of the card
    dev = torch.device("cuda:0")
    cfg = ki.workload(name)
    geom = ki.make_geometry(cfg)
    p = geom.params()
    L, nt, H = cfg["n_layers"], len(geom.trig), p["n_kv_heads"]
    W, U, N, bs = p["window"], p["buffer"], p["window"] - p["buffer"], p["block_size"]
    G = p["n_q_heads"] // H
    print(f"\n[case] {name} full size: {L} layers x {nt} triggered x {H} heads, W={W}", flush=True)

    dt = ki.torch_dtype(cfg)
    q = torch.empty((L, nt, ki.scoring_queries(cfg), p["n_q_heads"], p["head_dim"]), dtype=dt, device=dev)
    kp, vp = [], []
    for l in range(L):
        q[l] = ki.make_queries(geom, l, dev)
        k_, v_ = ki.make_pools(geom, l, dev)
        kp.append(k_)
        vp.append(v_)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bt, seq_lens, win_start, trig = T(geom.block_table), T(geom.seq_lens), T(geom.win_start), T(geom.trig)
    params = kara.make_params(p, geom.block_table.shape[0])

    rng = np.random.default_rng(11)
    p1_units = _units_sample(rng, L, nt, H, n_p1)
    # host copies, before the call, of what the oracle needs for the P1 units
    before = {}
    for (l, t, h) in p1_units:
        s = int(geom.trig[t])
        pos = np.arange(int(geom.seq_lens[s]))
        before[(l, t, h)] = dict(
            q=ki.raw_numpy(q[l, t, :, h * G:(h + 1) * G, :]),
            k=_rows(kp[l], geom.block_table[s], pos, h, bs),
            v=_rows(vp[l], geom.block_table[s], pos, h, bs))

    # device snapshot of every triggered sequence's [p0, seq_len), checksums of [0, p0)
    snap = kc.WindowSnapshot(geom, kp, vp)

    ws = torch.empty(kara.workspace_size(params, nt, L), dtype=torch.uint8, device=dev)
    scores = torch.empty((L, nt, H, N), dtype=torch.float32, device=dev)
    disc = torch.empty((L, nt, H, p["budget"] - p["chunk_budget"]), dtype=torch.int32, device=dev)
    kept = torch.empty((L, nt, H, p["budget"]), dtype=torch.int32, device=dev)
    freed = torch.full((nt, p["max_blocks_per_seq"]), -7, dtype=torch.int32, device=dev)
    n_freed = torch.full((nt,), -7, dtype=torch.int32, device=dev)
    status = torch.full((nt,), -7, dtype=torch.int32, device=dev)
    kara.compress_window(params, trig, q, kp, vp, bt, seq_lens, win_start, True, status, ws, scores=scores,
                         discrete=disc, kept=kept, freed=freed, n_freed=n_freed)
    torch.cuda.synchronize()
    st = status.cpu().numpy()
    assert (st == 0).all(), st
    print("[case] step done; checking", flush=True)

    # P2 on every unit: the oracle's selection on the GPU's own scores
    sc_all, di_all, ke_all = scores.cpu().numpy(), disc.cpu().numpy(), kept.cpu().numpy()
    n_units = 0
    for l in range(L):
        for t in range(nt):
            for h in range(H):
                d, k = oracle.kept_set(sc_all[l, t, h], p["budget"], p["chunk_budget"], p["max_chunk_len"])
                assert np.array_equal(d, di_all[l, t, h]), f"P2 discrete at {(l, t, h)}"
                assert np.array_equal(k, ke_all[l, t, h]), f"P2 kept at {(l, t, h)}"
                n_units += 1
        if l % 10 == 9:
            print(f"[case] P2 through layer {l}", flush=True)
    sc_h, kept_h = {}, {}
    for u in p1_units:
        sc_h[u], kept_h[u] = sc_all[u], ke_all[u]

    # compaction of every unit against its definition, on the device
    snap.check(geom, p, kept, kp, vp)
    del snap

    # P1 and P3 on the sampled units (fp64 scores from the host copies)
    from concurrent.futures import ThreadPoolExecutor
    scale = oracle.scale_of(p)

    def ora(u):
        b = before[u]
        s = int(geom.trig[u[1]])
        qa = oracle.to_f64(b["q"].reshape(-1, b["q"].shape[-1]), p["dtype"])
        p0 = int(geom.win_start[s])
        ka = oracle.to_f64(b["k"][p0:p0 + N], p["dtype"])
        return oracle.round_scores(oracle.window_scores(qa, ka, scale))

    with ThreadPoolExecutor(16) as ex:
        ora_sc = dict(zip(p1_units, ex.map(ora, p1_units)))
    worst = 0.0
    differ = 0
    layers_seen, heads_seen = set(), set()
    for u in p1_units:
        a = ora_sc[u]
        err = np.abs(sc_h[u].astype(np.float64) - a.astype(np.float64))
        assert (err <= kc.tol(a.astype(np.float64))).all(), f"P1 at {u}: max err {err.max()}"
        worst = max(worst, float((err / (np.abs(a) + 1e-12)).max()))
        differ += kc.p3_unit(a, sc_h[u], di_all[u], kept_h[u], p)
        layers_seen.add(u[0])
        heads_seen.add(u[2])
    assert layers_seen == set(range(L)) and heads_seen == set(range(H))

    # P4: tables of every sequence, rows of the sampled units
    bt_h, sl_h = bt.cpu().numpy(), seq_lens.cpu().numpy()
    fr_h, nf_h = freed.cpu().numpy(), n_freed.cpu().numpy()
    want_bt = geom.block_table.copy()
    want_sl = geom.seq_lens.copy()
    for t, s in enumerate(geom.trig):
        s = int(s)
        old = int(geom.seq_lens[s])
        new = old - (N - p["budget"])
        rel = oracle.released_blocks(old, new, bs)
        want_fr = np.full(p["max_blocks_per_seq"], -1, dtype=np.int32)
        want_fr[:len(rel)] = geom.block_table[s, rel]
        assert nf_h[t] == len(rel) and np.array_equal(fr_h[t], want_fr), f"P4 freed list of trigger {t}"
        want_bt[s, rel] = -1
        want_sl[s] = new
    assert np.array_equal(bt_h, want_bt), "P4 block tables"
    assert np.array_equal(sl_h, want_sl), "P4 sequence lengths"
    for u in p1_units:
        l, t, h = u
        s = int(geom.trig[t])
        p0 = int(geom.win_start[s])
        old = int(geom.seq_lens[s])
        new = int(want_sl[s])
        for name_, src, pool in (("K", before[u]["k"], kp[l]), ("V", before[u]["v"], vp[l])):
            want = np.concatenate([src[:p0], oracle.gather_rows(src[p0:old], kept_h[u], W, U)])
            got = _rows(pool, bt_h[s], np.arange(new), h, bs)
            assert want.shape == got.shape
            assert np.array_equal(want.view(np.uint8), got.view(np.uint8)), f"P4 {name_} rows of {u}"
    print(f"[case] ok: P1 max rel err {worst:.2e} over {len(p1_units)} units, P2 and compaction over {n_units} units, "
          f"P3 near-tie differences {differ}", flush=True)
    del q, kp, vp, ws, scores, disc, kept
    torch.cuda.empty_cache()
