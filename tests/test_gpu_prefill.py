"""GPU parity of prefill-time compression (kara_compress_prefill, App. C.2)
against the oracle's compress_prefill on the same seeded inputs:

  P1  every window's scores within the score tolerance;
  P2  the oracle's selection on the GPU's scores equals the GPU's index sets;
  P3  the oracle's end-to-end kept sets equal the GPU's, or differ only by
      swaps across a near-tie decision boundary (every window);
  P4  the oracle's compaction with those index sets equals the GPU's cache
      (bit-exact rows), block tables, lengths and freed pages.
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


def _check(cfg):
    import kara_check as kc
    from paper_2607_01237_amd import kara
    _need_gpu()
    dev = torch.device("cuda:0")
    nw = cfg["n_windows"]
    print(f"\n[case] prefill {nw} windows W={cfg['window']} U={cfg['buffer']} bs={cfg['block_size']}", flush=True)
    geom = ki.make_geometry(cfg)
    p = geom.params()
    L, nt, H = cfg["n_layers"], len(geom.trig), p["n_kv_heads"]
    W, U, N, bs = p["window"], p["buffer"], p["window"] - p["buffer"], p["block_size"]
    q = torch.stack([ki.make_queries(geom, l, dev) for l in range(L)]).contiguous()
    pools = [ki.make_pools(geom, l, dev) for l in range(L)]
    kp, vp = [x[0] for x in pools], [x[1] for x in pools]
    # the oracle takes [L, nt, n_windows, Wq, Hq, d]; one window has no axis of its own on the device
    host = dict(q=ki.raw_numpy(q).reshape((L, nt, nw) + tuple(q.shape[-3:])), kp=[ki.raw_numpy(t) for t in kp], vp=[ki.raw_numpy(t) for t in vp],
                bt=geom.block_table.copy(), lens=geom.seq_lens.copy())
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    bt, lens, ws0, trig = T(geom.block_table), T(geom.seq_lens), T(geom.win_start), T(geom.trig)
    params = kara.make_params(p, geom.block_table.shape[0])
    ws = torch.empty(kara.workspace_size(params, nt * nw, L), dtype=torch.uint8, device=dev)
    scores = torch.full((L, nt, nw, H, N), float("nan"), dtype=torch.float32, device=dev)
    disc = torch.full((L, nt, nw, H, p["budget"] - p["chunk_budget"]), -7, dtype=torch.int32, device=dev)
    kept = torch.full((L, nt, nw, H, p["budget"]), -7, dtype=torch.int32, device=dev)
    freed = torch.full((nt, p["max_blocks_per_seq"]), -7, dtype=torch.int32, device=dev)
    n_freed = torch.full((nt,), -7, dtype=torch.int32, device=dev)
    status = torch.full((nt,), -7, dtype=torch.int32, device=dev)
    kara.compress_prefill(params, trig, nw, q, kp, vp, bt, lens, ws0, True, status, ws, scores=scores,
                          discrete=disc, kept=kept, freed=freed, n_freed=n_freed)
    torch.cuda.synchronize()
    st = status.cpu().numpy()
    sc, di, ke = scores.cpu().numpy(), disc.cpu().numpy(), kept.cpu().numpy()

    # P1: the oracle's own scores
    ora = oracle.compress_prefill(p, geom.trig, nw, host["q"], [k.copy() for k in host["kp"]],
                                  [v.copy() for v in host["vp"]], host["bt"].copy(), host["lens"].copy(),
                                  geom.win_start, commit=True, threads=8)
    assert np.array_equal(ora["status"], st), (ora["status"], st)
    ok = st == 0
    a = ora["scores"][:, ok].astype(np.float64)
    err = np.abs(sc[:, ok].astype(np.float64) - a)
    assert (err <= kc.tol(a)).all(), f"P1: max err {err.max():.3e}"
    # P2 and P4: the oracle's selection and compaction on the GPU's scores
    kp_o, vp_o = [k.copy() for k in host["kp"]], [v.copy() for v in host["vp"]]
    bt_o, lens_o = host["bt"].copy(), host["lens"].copy()
    ref = oracle.compress_prefill(p, geom.trig, nw, host["q"], kp_o, vp_o, bt_o, lens_o, geom.win_start,
                                  commit=True, score_override=np.nan_to_num(sc))
    assert np.array_equal(ref["discrete"][:, ok], di[:, ok]), "P2 discrete"
    assert np.array_equal(ref["kept"][:, ok], ke[:, ok]), "P2 kept"
    # P3: every window of every valid sequence, stage by stage on oracle scores
    differ = 0
    for l in range(L):
        for t in np.flatnonzero(ok):
            for w in range(nw):
                for h in range(H):
                    differ += kc.p3_unit(ora["scores"][l, t, w, h], sc[l, t, w, h], di[l, t, w, h],
                                         ke[l, t, w, h], p)
    assert np.array_equal(bt.cpu().numpy(), bt_o), "P4 block tables"
    assert np.array_equal(lens.cpu().numpy(), lens_o), "P4 lengths"
    fr, nf = freed.cpu().numpy(), n_freed.cpu().numpy()
    for t in range(nt):
        want = ref["freed"][t]
        assert nf[t] == len(want) and list(fr[t, :nf[t]]) == want, f"P4 freed of trigger {t}"
        assert (fr[t, nf[t]:] == -1).all()
    for l in range(L):
        for name, dev_pool, ora_pool in (("K", kp[l], kp_o[l]), ("V", vp[l], vp_o[l])):
            got = ki.raw_numpy(dev_pool)
            assert np.array_equal(got.view(np.uint8), ora_pool.view(np.uint8)), f"P4 {name} pool of layer {l}"
    assert (lens_o[geom.trig[ok]] == host["lens"][geom.trig[ok]] - nw * (N - p["budget"])).all()
    print(f"[case] ok: P1 max abs err {err.max():.2e}, P3 units differing {differ}", flush=True)


@pytest.mark.parametrize("window,buffer,n_windows,block_size,dtype,head_dim", [
    (256, 0, 3, 16, "bf16", 128),
    (256, 32, 3, 7, "bf16", 128),
    (200, 9, 4, 16, "bf16", 64),
    (96, 16, 5, 16, "f32", 64),
    (512, 0, 1, 16, "bf16", 128),
])
def test_prefill_parity(window, buffer, n_windows, block_size, dtype, head_dim):
    N = window - buffer
    budget = -(-N // 5)
    cfg = ki.workload("prefill", n_seqs=3, n_layers=2, window=window, buffer=buffer, n_windows=n_windows,
                      block_size=block_size, dtype=dtype, head_dim=head_dim, budget=budget,
                      chunk_budget=min(8, budget - 1), max_chunk_len=5, prefix=(0, 40), tail=(0, 30),
                      n_q_heads=8, n_kv_heads=2)
    _check(cfg)
