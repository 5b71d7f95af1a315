"""Soak invariants: the compression step inside a decode loop, scaled down.

A small batch runs several intervals of (append, decode) ending in a
compression event, through the same driver the benchmark uses.  The host
keeps its own copy of every sequence's K/V rows: appended rows go in as
drawn, and after each event the window is replaced by the oracle's gather of
its kept set.  Checked on every event:
  * the device cache equals the host copy bit for bit, before and after
    compression (append, compaction and the block-table rewrite);
  * the kept sets are the oracle's selection on the GPU's own scores, and a
    sample of the scores matches the oracle's fp64 scores;
  * decode attention over the compressed cache equals softmax attention in
    fp64 over the host copy;
  * the page pool is conserved (checked by the driver against the device's
    freed lists and block table).
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


def _f64(raw, dtype):
    return oracle.to_f64(raw, dtype)


def _device_rows(sk, l, s, h, n_tok):
    pos = np.arange(n_tok)
    pg = torch.from_numpy(sk.pool.table[s, pos // sk.bs].astype(np.int64)).to(sk.dev)
    sl = torch.from_numpy((pos % sk.bs).astype(np.int64)).to(sk.dev)
    return ki.raw_numpy(sk.kp[l][pg, h, sl]), ki.raw_numpy(sk.vp[l][pg, h, sl])


def _check_cache(sk, host_k, host_v, what):
    for l in range(sk.L):
        for s in range(sk.n):
            n_tok = int(sk.pool.lens[s])
            for h in range(sk.Hkv):
                k, v = _device_rows(sk, l, s, h, n_tok)
                assert len(host_k[l][s][h]) == n_tok
                assert np.array_equal(k.view(np.uint8), np.asarray(host_k[l][s][h]).view(np.uint8)), \
                    f"{what}: K rows of layer {l} seq {s} head {h}"
                assert np.array_equal(v.view(np.uint8), np.asarray(host_v[l][s][h]).view(np.uint8)), \
                    f"{what}: V rows of layer {l} seq {s} head {h}"


def _check_decode(sk, host_k, host_v, dtype):
    sk.decode()
    torch.cuda.synchronize()
    got = sk.out.cpu().numpy()
    qh = _f64(ki.raw_numpy(sk.q_dec), dtype)
    G = sk.Hq // sk.Hkv
    scale = 1.0 / np.sqrt(sk.d)
    for l in range(sk.L):
        for s in range(sk.n):
            for hq in range(sk.Hq):
                K = _f64(np.asarray(host_k[l][s][hq // G]), dtype)
                V = _f64(np.asarray(host_v[l][s][hq // G]), dtype)
                x = scale * (K @ qh[l, s, hq])
                w = np.exp(x - x.max())
                want = (w / w.sum()) @ V
                err = np.abs(got[l, s, hq] - want)
                assert (err <= 1e-4 + 1e-4 * np.abs(want)).all(), ("decode", l, s, hq, float(err.max()))


@pytest.mark.parametrize("dtype,head_dim,prompt", [("bf16", 128, 70), ("f32", 64, 48)])
def test_soak_invariants(dtype, head_dim, prompt):
    from paper_2607_01237_amd.soak import Soak
    _need_gpu()
    dev = torch.device("cuda:0")
    cfg = ki.workload("soak", n_seqs=4, n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=head_dim, dtype=dtype,
                      window=256, budget=52, chunk_budget=16, max_chunk_len=8, prefix=(prompt, prompt),
                      n_intervals=3, append_chunk=64)
    print(f"\n[case] soak {dtype} d={head_dim} prompt={prompt}", flush=True)
    geom = ki.soak_geometry(cfg)
    gen = torch.Generator(device=dev)
    gen.manual_seed(123)
    sk = Soak(cfg, geom, dev, gen)
    p = sk.p
    W, U = p["window"], p["buffer"]
    N = W - U
    G = sk.Hq // sk.Hkv
    host_k = [[[[] for _ in range(sk.Hkv)] for _ in range(sk.n)] for _ in range(sk.L)]
    host_v = [[[[] for _ in range(sk.Hkv)] for _ in range(sk.n)] for _ in range(sk.L)]

    def append(n_tok):
        k_new, v_new = sk.append(n_tok)
        kn, vn = ki.raw_numpy(k_new), ki.raw_numpy(v_new)
        for l in range(sk.L):
            for s in range(sk.n):
                for h in range(sk.Hkv):
                    host_k[l][s][h].extend(kn[l, s, :, h])
                    host_v[l][s][h].extend(vn[l, s, :, h])

    left = prompt
    while left > 0:
        append(min(sk.chunk, left))
        left -= min(sk.chunk, left)
    sk.p0[:] = prompt
    scale = oracle.scale_of(p)
    rng = np.random.default_rng(0)
    for event in range(cfg["n_intervals"]):
        for c in range(W // sk.chunk):
            append(sk.chunk)
            if c == 0:
                _check_decode(sk, host_k, host_v, dtype)
        torch.cuda.synchronize()
        _check_cache(sk, host_k, host_v, f"event {event} before compression")
        p0 = sk.p0.copy()
        sk.compress(want_scores=True)
        sk.settle()                                   # page-pool checks
        scores = sk.scores.cpu().numpy()
        kept = sk.kept.cpu().numpy()
        q_raw = ki.raw_numpy(sk.q)
        sample = {(int(rng.integers(sk.L)), int(rng.integers(sk.n)), int(rng.integers(sk.Hkv))) for _ in range(3)}
        for l in range(sk.L):
            for s in range(sk.n):
                for h in range(sk.Hkv):
                    a = scores[l, s, h]
                    _, k_ora = oracle.kept_set(a, p["budget"], p["chunk_budget"], p["max_chunk_len"])
                    assert np.array_equal(k_ora, kept[l, s, h]), f"event {event}: kept set of {(l, s, h)}"
                    if (l, s, h) in sample:
                        qa = _f64(q_raw[l, s, :, h * G:(h + 1) * G, :].reshape(W * G, -1), dtype)
                        ka = _f64(np.asarray(host_k[l][s][h][p0[s]:p0[s] + N]), dtype)
                        want = oracle.round_scores(oracle.window_scores(qa, ka, scale)).astype(np.float64)
                        err = np.abs(a.astype(np.float64) - want)
                        assert (err <= 1e-5 + 2e-3 * np.abs(want)).all(), f"event {event}: scores of {(l, s, h)}"
                    for rows in (host_k[l][s][h], host_v[l][s][h]):
                        arr = np.asarray(rows)
                        new = np.concatenate([arr[:p0[s]], oracle.gather_rows(arr[p0[s]:], kept[l, s, h], W, U)])
                        rows[:] = list(new)
        _check_cache(sk, host_k, host_v, f"event {event} after compression")
        _check_decode(sk, host_k, host_v, dtype)
        print(f"[case] event {event}: ok, {sk.reclaimed} pages reclaimed so far", flush=True)
    assert sk.reclaimed > 0
