"""The decode-loop soak at its stated shape, checked against the oracle.

128 sequences x 40 layers of the Qwen3-14B shape (40/8 heads, d = 128,
bf16), W = 1024, budget 205, a 1K-token prompt and 31 intervals of 1024
generated tokens (appended 128 at a time, one decode step after each
append), each ending in a compression event over every sequence and layer
(Algorithm 1; App. C.4).  The pool holds the peak need plus 1 %, handed out
from a shuffled free list, so the block tables are fragmented and reused.

Every event (paper_2607_01237_amd/soak.py, Soak.settle): the device's
lengths, block tables and freed-page lists equal the host's page-pool model
for all 128 sequences -- the freed pages are exactly the trailing blocks the
new length no longer covers -- and no page is lost or mapped twice.

Events 1, 16 and 31, in addition:
  P2  the oracle's selection on the GPU's scores equals the GPU's discrete
      and kept sets, for all 40,960 units;
  compaction of every unit, on the device, against its definition (each
      written row equals the snapshot row the compaction map names; rows
      before the window keep their checksums);
  P1  fp64 oracle scores of 16 sampled units (host copies taken before the
      call) within 1e-5 + 2e-3 |A|;
  P3  the oracle's end-to-end kept sets of those units, near-tie swaps
      across a decision boundary excepted.
"""
import time

import numpy as np
import pytest

import kara_inputs as ki
import oracle

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

CHECK_EVENTS = (0, 15, 30)      # events 1, 16 and 31


class _SoakGeom:
    """The view of the soak's state that the device compaction check reads."""

    def __init__(self, sk):
        self.trig = np.arange(sk.n, dtype=np.int32)
        self.win_start = sk.p0.copy()
        self.seq_lens = sk.pool.lens.copy()
        self.block_table = sk.pool.table.copy()
        self._p = dict(sk.p)

    def params(self):
        return self._p


def test_soak_full_shape():
    import kara_check as kc
    from paper_2607_01237_amd.soak import Soak
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    torch.cuda.empty_cache()
    dev = torch.device("cuda:0")
    cfg = ki.workload("soak")
    geom = ki.soak_geometry(cfg)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg["seed"])
    sk = Soak(cfg, geom, dev, gen)
    p = sk.p
    W, N, G, H, L, n = sk.W, sk.W - p["buffer"], sk.Hq // sk.Hkv, sk.Hkv, sk.L, sk.n
    assert (n, L, sk.Hq, H, sk.d, W, p["budget"], cfg["n_intervals"]) == (128, 40, 40, 8, 128, 1024, 205, 31)
    print(f"\n[case] soak full shape: {n} x {L} layers, pool {geom.num_pages} pages, "
          f"{cfg['n_intervals']} events", flush=True)
    t0 = time.perf_counter()
    sk.prompt()
    rng = np.random.default_rng(17)
    scale = oracle.scale_of(p)
    n_dec = W // sk.chunk
    total_differ = 0
    for ev in range(cfg["n_intervals"]):
        for _ in range(n_dec):
            sk.append(sk.chunk)
            sk.decode()
        check = ev in CHECK_EVENTS
        if not check:
            sk.compress()
            sk.settle()
            continue
        sk.draw_queries()
        torch.cuda.synchronize()
        sg = _SoakGeom(sk)
        # host copies of the sampled units' queries and window keys, and a
        # device snapshot of every window and tail, before the call
        units = {(int(rng.integers(L)), int(rng.integers(n)), int(h)) for h in range(H)}
        while len(units) < 16:
            units.add((int(rng.integers(L)), int(rng.integers(n)), int(rng.integers(H))))
        units = sorted(units)
        host = {}
        for (l, s, h) in units:
            pos = np.arange(sg.win_start[s], sg.win_start[s] + N)
            pg = torch.from_numpy(sg.block_table[s, pos // sk.bs].astype(np.int64)).to(dev)
            sl = torch.from_numpy((pos % sk.bs).astype(np.int64)).to(dev)
            host[(l, s, h)] = (ki.raw_numpy(sk.q[l, s, :, h * G:(h + 1) * G, :]).reshape(W * G, -1),
                               ki.raw_numpy(sk.kp[l][pg, h, sl, :]))
        snap = kc.WindowSnapshot(sg, sk.kp, sk.vp)
        sk.compress(want_scores=True, fresh_q=False)
        sk.settle()
        snap.check(sg, p, sk.kept, sk.kp, sk.vp)
        del snap
        sc, di, ke = sk.scores.cpu().numpy(), sk.disc.cpu().numpy(), sk.kept.cpu().numpy()
        for u in np.ndindex(L, n, H):
            d_, k_ = oracle.kept_set(sc[u], p["budget"], p["chunk_budget"], p["max_chunk_len"])
            assert np.array_equal(d_, di[u]), f"event {ev + 1}: P2 discrete at {u}"
            assert np.array_equal(k_, ke[u]), f"event {ev + 1}: P2 kept at {u}"
        worst = 0.0
        for u in units:
            qa, ka = (oracle.to_f64(x, p["dtype"]) for x in host[u])
            a = oracle.round_scores(oracle.window_scores(qa, ka, scale))
            err = np.abs(sc[u].astype(np.float64) - a.astype(np.float64))
            assert (err <= kc.tol(a.astype(np.float64))).all(), f"event {ev + 1}: P1 at {u}, max err {err.max()}"
            worst = max(worst, float((err / (np.abs(a) + 1e-12)).max()))
            total_differ += kc.p3_unit(a, sc[u], di[u], ke[u], p)
        print(f"[case] event {ev + 1}: P2 and compaction over {L * n * H} units, P1 max rel err {worst:.2e} "
              f"over {len(units)} units, {sk.reclaimed} pages reclaimed so far, "
              f"{time.perf_counter() - t0:.0f} s", flush=True)
    assert sk.reclaimed > 0
    print(f"[case] ok: {cfg['n_intervals']} events, {sk.reclaimed} pages reclaimed, P3 units differing "
          f"{total_differ}", flush=True)
    del sk
    torch.cuda.empty_cache()
