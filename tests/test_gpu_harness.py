"""The decoding-side helpers (include/kara_harness.h) against plain CPU
references: token append into the paged cache (bit-exact rows, lengths and
status bits) and decode attention of one query per (layer, sequence, query
head) over the whole cache (fp64 softmax attention on the host).

These kernels are not part of the compression step; they let a long-running
workload append, decode and compress on the GPU.  Their references are the
definitions (a row copy; softmax(scale q.K) V), written out here in numpy.
"""
import numpy as np
import pytest

import kara_inputs as ki

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _geom(rng, n_seqs, Hq, Hkv, d, dtype, bs, lens, max_blocks, extra_pages=8):
    need = [min(max_blocks, -(-int(L) // bs)) for L in lens]
    num_pages = int(sum(need)) + extra_pages
    perm = rng.permutation(num_pages)
    table = np.full((n_seqs, max_blocks), -1, dtype=np.int32)
    c = 0
    for s in range(n_seqs):
        table[s, :need[s]] = perm[c:c + need[s]]
        c += need[s]
    p = dict(window=64, buffer=0, budget=16, chunk_budget=4, max_chunk_len=4, head_dim=d, n_q_heads=Hq,
             n_kv_heads=Hkv, block_size=bs, num_pages=num_pages, max_blocks_per_seq=max_blocks, dtype=dtype,
             scale=0.0)
    return p, table, perm[c:].astype(np.int32)


def _f64(a, dtype):
    if dtype == "bf16":
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


@pytest.mark.parametrize("dtype,Hq,Hkv,d", [("f32", 4, 1, 64), ("bf16", 32, 8, 128), ("bf16", 40, 8, 128),
                                             ("bf16", 16, 1, 64), ("f32", 8, 2, 128)])
def test_decode_attention(dtype, Hq, Hkv, d):
    from paper_2607_01237_amd import kara
    _need_gpu()
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(Hq * 131 + d)
    bs, L = 16, 2
    lens = np.array([1, 255, 256, 257, 700, 0, 900, 33], dtype=np.int32)
    max_len = 800                               # the 900-token sequence is over it: zero rows
    p, table, _ = _geom(rng, len(lens), Hq, Hkv, d, dtype, bs, lens, max_blocks=64)
    print(f"\n[case] decode {dtype} Hq={Hq} Hkv={Hkv} d={d}", flush=True)
    params = kara.make_params(p, len(lens))
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device="cpu").manual_seed(5)
    kp = [torch.randn((p["num_pages"], Hkv, bs, d), generator=g).to(dt) for _ in range(L)]
    vp = [torch.randn((p["num_pages"], Hkv, bs, d), generator=g).to(dt) for _ in range(L)]
    # seq 7 is not listed; len(lens) and -1 are indices outside the table (zero rows)
    seqs = np.array([5, 0, 3, 1, 4, 2, 6, len(lens), -1], dtype=np.int32)
    n = len(seqs)
    q = torch.randn((L, n, Hq, d), generator=g).to(dt)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    out = torch.full((L, n, Hq, d), float("nan"), dtype=torch.float32, device=dev)
    ws = torch.empty(kara.decode_workspace_size(params, n, L, max_len), dtype=torch.uint8, device=dev)
    kpd, vpd = [t.to(dev) for t in kp], [t.to(dev) for t in vp]
    kara.decode_attention(params, T(seqs), q.to(dev), kpd, vpd, T(table), T(lens), max_len, out, ws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()

    G = Hq // Hkv
    scale = 1.0 / np.sqrt(d)
    qh = _f64(ki.raw_numpy(q), dtype)
    worst = 0.0
    for l in range(L):
        kh, vh = _f64(ki.raw_numpy(kp[l]), dtype), _f64(ki.raw_numpy(vp[l]), dtype)
        for j, s in enumerate(seqs):
            if s < 0 or s >= len(lens):
                assert (got[l, j] == 0).all(), f"sequence index {s} is outside the table: zero rows"
                continue
            n_tok = int(lens[s])
            if n_tok == 0 or n_tok > max_len:
                assert (got[l, j] == 0).all(), f"seq {s} should give zero rows"
                continue
            pos = np.arange(n_tok)
            pg, sl = table[s, pos // bs], pos % bs
            for hq in range(Hq):
                K, V = kh[pg, hq // G, sl], vh[pg, hq // G, sl]
                x = scale * (K @ qh[l, j, hq])
                w = np.exp(x - x.max())
                want = (w / w.sum()) @ V
                err = np.abs(got[l, j, hq] - want)
                worst = max(worst, float(err.max()))
                assert (err <= 1e-4 + 1e-4 * np.abs(want)).all(), (l, j, hq, float(err.max()))
    print(f"[case] ok: max abs err {worst:.2e}", flush=True)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_kv_append(dtype, d):
    from paper_2607_01237_amd import kara
    _need_gpu()
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(17)
    bs, L, Hkv, n_new, max_blocks = 16, 2, 2, 37, 12
    lens = np.array([0, 15, 16, 100, 150, 40, 3, 160], dtype=np.int32)
    # map the blocks the appended tokens need, except where a case says not to
    p, table, spare = _geom(rng, len(lens), 4 * Hkv, Hkv, d, dtype, bs, lens + n_new, max_blocks)
    print(f"\n[case] append {dtype} d={d}", flush=True)
    table[5, (40 + n_new - 1) // bs] = -1          # sequence 5: last new position unmapped
    # sequence 7: 160 + 37 > 12 * 16 tokens
    seqs = np.array([3, 0, 5, 9, 1, 6, 6, 7, 2, 4], dtype=np.int32)
    want_status = np.array([0, 0, kara.SEQ_BAD_PAGE, kara.SEQ_BAD_INDEX, 0, kara.SEQ_DUP_TRIGGER,
                            kara.SEQ_DUP_TRIGGER, kara.SEQ_BAD_WINDOW, 0, 0], dtype=np.int32)
    params = kara.make_params(p, len(lens))
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    g = torch.Generator(device="cpu").manual_seed(9)
    kp = [torch.randn((p["num_pages"], Hkv, bs, d), generator=g).to(dt) for _ in range(L)]
    vp = [torch.randn((p["num_pages"], Hkv, bs, d), generator=g).to(dt) for _ in range(L)]
    n = len(seqs)
    k_new = torch.randn((L, n, n_new, Hkv, d), generator=g).to(dt)
    v_new = torch.randn((L, n, n_new, Hkv, d), generator=g).to(dt)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    kpd, vpd = [t.to(dev) for t in kp], [t.to(dev) for t in vp]
    sl_d, st_d = T(lens), torch.full((n,), -7, dtype=torch.int32, device=dev)
    kara.kv_append(params, T(seqs), k_new.to(dev), v_new.to(dev), kpd, vpd, T(table), sl_d, st_d)
    torch.cuda.synchronize()
    st = st_d.cpu().numpy()
    assert np.array_equal(st, want_status), st

    want_lens = lens.copy()
    want_k = [ki.raw_numpy(t).copy() for t in kp]
    want_v = [ki.raw_numpy(t).copy() for t in vp]
    kn, vn = ki.raw_numpy(k_new), ki.raw_numpy(v_new)
    for j, s in enumerate(seqs):
        if want_status[j] != 0:
            continue
        pos = lens[s] + np.arange(n_new)
        pg, slot = table[s, pos // bs], pos % bs
        for l in range(L):
            for h in range(Hkv):
                want_k[l][pg, h, slot] = kn[l, j, :, h]
                want_v[l][pg, h, slot] = vn[l, j, :, h]
        want_lens[s] += n_new
    assert np.array_equal(sl_d.cpu().numpy(), want_lens)
    for l in range(L):
        assert np.array_equal(ki.raw_numpy(kpd[l]).view(np.uint8), want_k[l].view(np.uint8)), f"K pool {l}"
        assert np.array_equal(ki.raw_numpy(vpd[l]).view(np.uint8), want_v[l].view(np.uint8)), f"V pool {l}"
    print("[case] ok", flush=True)
