"""Test harness: runs libkara on a seeded workload and checks it against the
CPU oracle (parity procedure P1-P4).

P1  scores within |A_gpu - A_ora| <= 1e-5 + 2e-3 |A_ora| (fp32 accumulation
    against fp64; the tolerance the step is specified with).
P2  the oracle's selection run on the GPU's own scores reproduces the GPU's
    discrete and kept sets bit for bit (same fp32 inputs, same decisions).
P3  end to end, the GPU's kept sets equal the oracle's, or differ only by
    swaps across a decision boundary (k-th score, n_c-th chunk score, fill
    score) where the oracle's values are within the propagated tolerance.
P4  compaction: the oracle's gather, run with the GPU's kept sets on a host
    snapshot, equals the GPU's live cache rows bit for bit, and the block
    tables, lengths and freed-page lists match exactly.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
import torch

import kara_inputs as ki
import oracle
from paper_2607_01237_amd import kara

RTOL, ATOL = 2e-3, 1e-5


def tol(a):
    return ATOL + RTOL * np.abs(a)


@dataclass
class Case:
    geom: ki.Geometry
    p: dict
    params: kara.KaraParams
    q: torch.Tensor
    kp: list
    vp: list
    bt: torch.Tensor
    seq_lens: torch.Tensor
    win_start: torch.Tensor
    trig: torch.Tensor
    host: dict


def setup(cfg: dict, device="cuda", trig=None, seq_lens=None, win_start=None, block_table=None) -> Case:
    geom = ki.make_geometry(cfg)
    if trig is not None:
        geom.trig = np.asarray(trig, dtype=np.int32)
    if seq_lens is not None:
        geom.seq_lens = np.asarray(seq_lens, dtype=np.int32)
    if win_start is not None:
        geom.win_start = np.asarray(win_start, dtype=np.int32)
    if block_table is not None:
        geom.block_table = np.asarray(block_table, dtype=np.int32)
    p = geom.params()
    L = cfg["n_layers"]
    q = torch.stack([ki.make_queries(geom, l, device) for l in range(L)]).contiguous()
    pools = [ki.make_pools(geom, l, device) for l in range(L)]
    kp = [x[0] for x in pools]
    vp = [x[1] for x in pools]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    case = Case(geom=geom, p=p, params=kara.make_params(p, geom.block_table.shape[0]), q=q, kp=kp, vp=vp,
                bt=dev(geom.block_table), seq_lens=dev(geom.seq_lens), win_start=dev(geom.win_start),
                trig=dev(geom.trig), host={})
    case.host = snapshot(case)
    return case


def snapshot(case: Case) -> dict:
    return dict(q=ki.raw_numpy(case.q), kp=[ki.raw_numpy(t) for t in case.kp], vp=[ki.raw_numpy(t) for t in case.vp],
                bt=case.bt.cpu().numpy().copy(), seq_lens=case.seq_lens.cpu().numpy().copy(),
                win_start=case.win_start.cpu().numpy().copy(), trig=case.trig.cpu().numpy().copy())


def n_units(case: Case) -> int:
    return len(case.kp) * case.trig.numel() * case.p["n_kv_heads"]


def run_compress(case: Case, commit=True):
    """One kara_compress_window call; returns host copies of every output."""
    p, dev = case.p, case.q.device
    L, nt, H = len(case.kp), case.trig.numel(), p["n_kv_heads"]
    N = p["window"] - p["buffer"]
    ws = torch.empty(kara.workspace_size(case.params, nt, L), dtype=torch.uint8, device=dev)
    out = dict(
        scores=torch.full((L, nt, H, N), float("nan"), dtype=torch.float32, device=dev),
        discrete=torch.full((L, nt, H, p["budget"] - p["chunk_budget"]), -7, dtype=torch.int32, device=dev),
        kept=torch.full((L, nt, H, p["budget"]), -7, dtype=torch.int32, device=dev),
        freed=torch.full((nt, p["max_blocks_per_seq"]), -7, dtype=torch.int32, device=dev),
        n_freed=torch.full((nt,), -7, dtype=torch.int32, device=dev),
        status=torch.full((nt,), -7, dtype=torch.int32, device=dev),
    )
    kara.compress_window(case.params, case.trig, case.q, case.kp, case.vp, case.bt, case.seq_lens, case.win_start,
                         commit, out["status"], ws, scores=out["scores"], discrete=out["discrete"], kept=out["kept"],
                         freed=out["freed"], n_freed=out["n_freed"])
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res["bt"] = case.bt.cpu().numpy()
    res["seq_lens"] = case.seq_lens.cpu().numpy()
    return res


# ------------------------------------------------------------------ checks
def oracle_scores(case: Case, units=None, threads=8):
    """fp32-rounded oracle scores [L, nt, H, N] (NaN where not computed)."""
    h = case.host
    p = case.p
    L, nt, H = len(h["kp"]), len(h["trig"]), p["n_kv_heads"]
    N = p["window"] - p["buffer"]
    st = oracle.validate(p, h["trig"], h["bt"], h["seq_lens"], h["win_start"])
    if units is None:
        units = [(l, t, hh) for l in range(L) for t in range(nt) for hh in range(H)]
    out = np.full((L, nt, H, N), np.nan, dtype=np.float32)
    ok = [u for u in units if st[u[1]] == 0]
    for u, a in zip(ok, oracle.score_units(p, h["trig"], h["q"], h["kp"], h["bt"], h["win_start"], ok, threads)):
        out[u] = oracle.round_scores(a)
    for u in units:
        if st[u[1]] != 0:
            out[u] = 0.0
    return out, st


def check_p1(gpu_scores, ora_scores):
    m = ~np.isnan(ora_scores)
    err = np.abs(gpu_scores[m].astype(np.float64) - ora_scores[m].astype(np.float64))
    # (written so that a NaN or infinite GPU score fails)
    bad = ~(err <= tol(ora_scores[m].astype(np.float64)))
    assert not bad.any(), f"P1: {bad.sum()} scores out of tolerance (or not finite), max err {np.nanmax(err):.3e}"
    rel = err / np.maximum(np.abs(ora_scores[m]), 1e-30)
    return dict(max_abs=float(err.max()) if err.size else 0.0, max_rel=float(rel.max()) if rel.size else 0.0,
                checked=int(m.sum()))


def check_p2(p, gpu):
    """Oracle selection on the GPU's scores == the GPU's index sets."""
    L, nt, H, _ = gpu["scores"].shape
    for l in range(L):
        for t in range(nt):
            for h in range(H):
                d, k = oracle.kept_set(gpu["scores"][l, t, h], p["budget"], p["chunk_budget"], p["max_chunk_len"])
                assert np.array_equal(d, gpu["discrete"][l, t, h]), f"P2 discrete mismatch at unit {(l, t, h)}"
                assert np.array_equal(k, gpu["kept"][l, t, h]), f"P2 kept mismatch at unit {(l, t, h)}"


def _swap_ok(entered, left, lo, hi):
    """Set `entered` replaced set `left` (same size) in a top-k decision.
    Valid only as swaps across the decision boundary within tolerance: some
    threshold c has every entered item able to reach c (hi >= c) and every
    item that left able to fall to it (lo <= c), i.e.
    max(lo[left]) <= min(hi[entered])."""
    if len(entered) != len(left):
        return False
    if not len(entered):
        return True
    return max(lo[i] for i in left) <= min(hi[i] for i in entered)


def p3_unit(a_ora, a_gpu, disc_gpu, kept_gpu, p):
    """P3 for one unit (Eq. (5)-(8), App. C.3).  The GPU's decisions were
    taken on its own scores (P2 checks that); here each stage is replayed
    with the oracle's fp32 scores on the GPU's previous-stage result, and any
    difference must consist only of swaps across that stage's boundary:
      discrete top-k: scores within tol_a + tol_b of each other;
      chunk top-n_c:  R within (gap-1)(tol_a + tol_b) summed over both
                      candidates, the tolerance of Eq. (6) propagated from
                      its two endpoint scores;
      fill:           scores within tol_a + tol_b.
    Raises AssertionError on any other difference; returns True when the
    unit's final kept set differs from the oracle's own end-to-end one."""
    budget, alpha, gamma = p["budget"], p["chunk_budget"], p["max_chunk_len"]
    a = a_ora.astype(np.float64)
    t = tol(a)
    lo, hi = a - t, a + t
    k = budget - alpha
    disc_gpu = np.asarray(disc_gpu, dtype=np.int64)
    kept_gpu = np.asarray(kept_gpu, dtype=np.int64)
    # stage 1: discrete top-k on the whole window
    d_ora = oracle.discrete_topk(a_ora, k)
    ent, lft = np.setdiff1d(disc_gpu, d_ora), np.setdiff1d(d_ora, disc_gpu)
    assert _swap_ok(ent, lft, lo, hi), \
        f"P3: discrete set differs beyond the k-th boundary (in {ent[:4]}, out {lft[:4]})"
    # stage 2: chunk choice among the candidates of the GPU's discrete set
    chosen_gpu, added_gpu = oracle.token2chunk(a_gpu, disc_gpu, alpha, gamma)
    cands = oracle.chunk_candidates(a_ora, disc_gpu, gamma)
    n_c = alpha // (gamma - 2)
    if cands:
        r = {i: rv for rv, i in cands}
        tr = {i: (int(disc_gpu[i + 1]) - int(disc_gpu[i]) - 1) * (t[disc_gpu[i]] + t[disc_gpu[i + 1]])
              for _, i in cands}
        chosen_ora, _ = oracle.token2chunk(a_ora, disc_gpu, alpha, gamma)
        ent_c = sorted(set(chosen_gpu) - set(chosen_ora))
        lft_c = sorted(set(chosen_ora) - set(chosen_gpu))
        lo_c = {i: r[i] - tr[i] for i in r}
        hi_c = {i: r[i] + tr[i] for i in r}
        assert _swap_ok(ent_c, lft_c, lo_c, hi_c), \
            f"P3: chunk choice differs beyond the n_c-th boundary (in {ent_c}, out {lft_c}; n_c={n_c})"
    # stage 3: fill among the positions the GPU left unselected
    taken = np.zeros(len(a), bool)
    taken[disc_gpu] = True
    taken[added_gpu] = True
    fill_gpu = np.setdiff1d(kept_gpu, np.flatnonzero(taken))
    f = alpha - len(added_gpu)
    assert len(fill_gpu) == f and not np.setdiff1d(np.flatnonzero(taken), kept_gpu).size, \
        "P3: the GPU's kept set is not discrete + chunks + fill (P2 should have caught this)"
    fill_ora = oracle.fill_positions(a_ora, taken, f)
    ent_f, lft_f = np.setdiff1d(fill_gpu, fill_ora), np.setdiff1d(fill_ora, fill_gpu)
    assert _swap_ok(ent_f, lft_f, lo, hi), \
        f"P3: fill differs beyond the fill boundary (in {ent_f[:4]}, out {lft_f[:4]})"
    _, kept_ora = oracle.kept_set(a_ora, budget, alpha, gamma)
    return not np.array_equal(kept_ora, kept_gpu)


def check_p3(p, gpu, ora_scores):
    """P3 over every unit the oracle scored; returns the number of units
    whose kept set differs from the oracle's (near-tie swaps only)."""
    lead = gpu["scores"].shape[:-1]
    differ = 0
    for u in np.ndindex(*lead):
        a = ora_scores[u]
        if np.isnan(a).any():
            continue
        differ += p3_unit(a, gpu["scores"][u], gpu["discrete"][u], gpu["kept"][u], p)
    return differ


def live_rows(pools, bt, seq_lens, trig_or_all, p):
    """Every live row (position < seq_len) of the listed sequences, per layer."""
    bs = p["block_size"]
    out = []
    for pool in pools:
        rows = []
        for s in trig_or_all:
            pos = np.arange(int(seq_lens[s]))
            rows.append(oracle.read_rows(pool, bt[s], pos, slice(None), bs) if len(pos) else
                        np.zeros((0,) + pool.shape[1:2] + pool.shape[3:], pool.dtype))
        out.append(rows)
    return out


def gpu_live_rows(t_pool, bt, seq_lens, seqs, p):
    bs = p["block_size"]
    pages, slots = [], []
    for s in seqs:
        pos = np.arange(int(seq_lens[s]))
        pages.append(bt[s, pos // bs])
        slots.append(pos % bs)
    pg = torch.from_numpy(np.concatenate(pages).astype(np.int64)).to(t_pool.device)
    sl = torch.from_numpy(np.concatenate(slots).astype(np.int64)).to(t_pool.device)
    rows = t_pool[pg, :, sl, :]
    return ki.raw_numpy(rows)


def check_p4(case: Case, gpu, commit=True):
    """Oracle compaction with the GPU's kept sets on the host snapshot."""
    h = case.host
    p = case.p
    kp = [x.copy() for x in h["kp"]]
    vp = [x.copy() for x in h["vp"]]
    bt = h["bt"].copy()
    sl = h["seq_lens"].copy()
    ora = oracle.compress(p, h["trig"], h["q"], kp, vp, bt, sl, h["win_start"], commit=commit,
                          score_override=gpu["scores"])
    assert np.array_equal(ora["status"], gpu["status"]), "P4: status differs"
    assert np.array_equal(ora["kept"], gpu["kept"]), "P4: kept differs (P2 should have caught this)"
    assert np.array_equal(bt, gpu["bt"]), "P4: block table differs"
    assert np.array_equal(sl, gpu["seq_lens"]), "P4: seq_lens differ"
    if commit:
        assert np.array_equal(ora["n_freed"], gpu["n_freed"]), "P4: n_freed differs"
        for t, fr in enumerate(ora["freed"]):
            want = np.full(p["max_blocks_per_seq"], -1, dtype=np.int32)
            want[:len(fr)] = fr
            assert np.array_equal(want, gpu["freed"][t]), f"P4: freed list of trigger {t} differs"
    seqs = list(range(bt.shape[0]))
    seqs = [s for s in seqs if sl[s] > 0]
    for l in range(len(kp)):
        for name, opools, tpools in (("K", kp, case.kp), ("V", vp, case.vp)):
            want = np.concatenate([oracle.read_rows(opools[l], bt[s], np.arange(sl[s]), slice(None), p["block_size"])
                                   for s in seqs])
            got = gpu_live_rows(tpools[l], bt, sl, seqs, p)
            assert want.shape == got.shape
            if not np.array_equal(want.view(np.uint8), got.view(np.uint8)):
                bad = np.argwhere(np.any(want != got, axis=tuple(range(1, want.ndim))))
                raise AssertionError(f"P4: {name} layer {l}: {len(bad)} live rows differ (first {bad[:3].ravel()})")
    return ora


def full_check(case: Case, commit=True, units=None):
    """Runs the fused step and P1-P4; returns a small report."""
    ora_scores, st = oracle_scores(case, units)
    gpu = run_compress(case, commit=commit)
    assert np.array_equal(st, gpu["status"]), f"status {gpu['status']} != oracle {st}"
    rep = check_p1(gpu["scores"], ora_scores)
    check_p2(case.p, gpu)
    rep["p3_units_differing"] = check_p3(case.p, gpu, ora_scores)
    check_p4(case, gpu, commit)
    rep["units"] = n_units(case)
    return rep, gpu


# ---- compaction of every unit, checked on the device against its definition ----
# At full size the pools do not fit on the host.  Before the call, every
# triggered sequence's rows [p0, seq_len) are copied on the device; after it,
# each row compaction wrote must equal, bit for bit, the snapshot row the
# compaction map names (kept ++ [N, W + tail), window-relative), and the rows
# before p0 must keep their checksums.  Plain torch indexing, not the library.

def positions(geom, lo, hi):
    """Concatenated (page, slot) of logical positions [lo(s), hi(s)) of every
    triggered sequence s, and each sequence's offset in the concatenation."""
    bs = geom.params()["block_size"]
    pg, sl, off = [], [], [0]
    for s in geom.trig:
        pos = np.arange(lo(int(s)), hi(int(s)), dtype=np.int64)
        pg.append(geom.block_table[s, pos // bs].astype(np.int64))
        sl.append(pos % bs)
        off.append(off[-1] + len(pos))
    return np.concatenate(pg), np.concatenate(sl), np.array(off[:-1], dtype=np.int64)


def checksum(rows, chunk=1 << 26):
    """Order-sensitive checksum of 16-bit rows (exact integer arithmetic, in
    chunks to bound the temporaries)."""
    x = rows.reshape(-1).view(torch.int16)
    s1 = s2 = 0
    for a in range(0, x.numel(), chunk):
        xc = x[a:a + chunk].to(torch.int64)
        w = torch.arange(a, a + xc.numel(), device=x.device, dtype=torch.int64) % 65521 + 1
        s1 += int(xc.sum())
        s2 += int((xc * w).sum())
    return s1, s2


class WindowSnapshot:
    """Device copy of the rows a compression may read or move, taken before
    the call; check() verifies every unit's compaction afterwards."""

    def __init__(self, geom, kp, vp):
        dev = kp[0].device
        T = lambda a: torch.from_numpy(a).to(dev)
        w_pg, w_sl, self.off = positions(geom, lambda s: int(geom.win_start[s]), lambda s: int(geom.seq_lens[s]))
        w_pg, w_sl = T(w_pg), T(w_sl)
        pre_pg, pre_sl, _ = positions(geom, lambda s: 0, lambda s: int(geom.win_start[s]))
        self.pre_pg, self.pre_sl = T(pre_pg), T(pre_sl)
        self.rows = [(k[w_pg, :, w_sl, :], v[w_pg, :, w_sl, :]) for k, v in zip(kp, vp)]
        self.pre = [self._prefix_sums(k, v) for k, v in zip(kp, vp)]

    def _prefix_sums(self, k, v):
        return checksum(k[self.pre_pg, :, self.pre_sl, :]), checksum(v[self.pre_pg, :, self.pre_sl, :])

    def check(self, geom, p, kept, kp, vp):
        """kept: [L, n_trig, Hkv, budget] (one window per sequence)."""
        dev = kp[0].device
        W, N, B, bs, H = p["window"], p["window"] - p["buffer"], p["budget"], p["block_size"], p["n_kv_heads"]
        nt = len(geom.trig)
        trig = geom.trig.astype(np.int64)
        p0s = geom.win_start[trig].astype(np.int64)
        tails = geom.seq_lens[trig].astype(np.int64) - p0s - W
        # destination j < B takes kept[j]; j >= B takes window-relative N + (j - B)
        kt, kj = np.repeat(np.arange(nt), B), np.tile(np.arange(B), nt)
        ex_t = np.concatenate([np.full(W + tl - N, t, dtype=np.int64) for t, tl in enumerate(tails)])
        ex_rel = np.concatenate([np.arange(N, W + tl, dtype=np.int64) for tl in tails])
        ex_j = ex_rel - N + B

        def dst(t_idx, j):
            pos = p0s[t_idx] + j
            return (torch.from_numpy(geom.block_table[trig[t_idx], pos // bs].astype(np.int64)).to(dev),
                    torch.from_numpy(pos % bs).to(dev))

        k_pg, k_sl = dst(kt, kj)
        e_pg, e_sl = dst(ex_t, ex_j)
        e_src = torch.from_numpy(self.off[ex_t] + ex_rel).to(dev)
        off = torch.from_numpy(self.off).to(dev).view(nt, 1, 1)
        hv = torch.arange(H, device=dev).view(H, 1)
        for l, (k, v) in enumerate(zip(kp, vp)):
            src = (kept[l].to(dev).to(torch.int64) + off).permute(1, 0, 2).reshape(H, -1)    # [H, nt*B]
            for name, pool, snap in (("K", k, self.rows[l][0]), ("V", v, self.rows[l][1])):
                want, got = snap[src, hv], pool[k_pg.view(1, -1), hv, k_sl.view(1, -1)]
                assert torch.equal(want.view(torch.int16), got.view(torch.int16)), \
                    f"compaction: {name} kept rows of layer {l}"
                want, got = snap[e_src.view(1, -1), hv], pool[e_pg.view(1, -1), hv, e_sl.view(1, -1)]
                assert torch.equal(want.view(torch.int16), got.view(torch.int16)), \
                    f"compaction: {name} buffer/tail rows of layer {l}"
            assert self._prefix_sums(k, v) == self.pre[l], f"compaction: rows before the window, layer {l}"


# ---- recompute attention: tolerance from the kernel's rounding model ----
# The kernel forms fp32 logits from bf16 operands (exact products, fp32
# sums), rounds each softmax weight to bf16 (relative error delta_j, |delta_j|
# <= u = 2^-8, of effectively random sign) and divides the weighted value sum
# by the sum of the same rounded weights; the output is stored as bf16.
# With normalised weights p_j the error is, to first order,
#     sum_j p_j delta_j (v_j - o) + (output rounding, <= u |o|),
# a sum of independent terms with standard deviation at most
# u/sqrt(3) * sqrt(sum_j p_j^2 (v_j - o)^2).  The bound allows five times
# u times that root (about 8.7 standard deviations), u |o| for the store and
# 2^-16 for the fp32 accumulation.  Dropping or duplicating one of n keys
# moves o by about |v_j - o| / n, which at n = 2048 is several times larger.

ATTN_U = 2.0 ** -8


def attention_spread(q, k_rows, v_rows, p0, scale, o):
    """sqrt(sum_j p_j^2 (v_j - o)^2) per output element [W, Hq, d], with p the
    causal softmax weights of window token w over cache rows [0, p0 + w]."""
    W, Hq, d = q.shape
    G = Hq // k_rows.shape[1]
    out = np.zeros((W, Hq, d))
    for w in range(W):
        n = p0 + w + 1
        for hq in range(Hq):
            h = hq // G
            x = (k_rows[:n, h, :] @ q[w, hq, :]) * scale
            pw = np.exp(x - x.max())
            pw /= pw.sum()
            dv = v_rows[:n, h, :] - o[w, hq][None, :]
            out[w, hq] = np.sqrt((pw[:, None] ** 2 * dv ** 2).sum(axis=0))
    return out


def attention_tol(o, spread):
    return ATTN_U * np.abs(o) + 5.0 * ATTN_U * spread + 2.0 ** -16


def check_attention(got, want, spread, what=""):
    err = np.abs(got - want)
    bad = err > attention_tol(want, spread)
    assert not bad.any(), f"attention {what}: {int(bad.sum())} elements out of tolerance, max err {err.max():.3e}"
    return float(err.max())
