"""CPU oracle for Kara's sliding-window KV-cache compression step.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check and
the benchmark's CPU-baseline leg may import it; the product path never calls
it and shares no code with it.

What it computes (Kara, Sec. 4 and App. C):

* window scoring, Eq. (4): A = colsum(softmax(Q_W K_{W\\U}^T / sqrt(d)));
* discrete top-k, Eq. (5): I = TopK(A, ceil(r(|W|-|U|)) - alpha);
* Token2Chunk, Eq. (6)-(8), plus the fill rule of App. C.3;
* the window gather, Eq. (9), applied to a paged cache, followed by the
  memory compaction, block release and metadata update of Algorithm 1
  (App. C.4).

Everything floating point is fp64 (scores are rounded to fp32 once, at the
end of Eq. (4)); selection works on those fp32 scores; Token2Chunk's chunk
scores are formed in fp64 from them.  No blocking, fusion or reordering: each
function follows the paper's definition step by step so it can be read
against the equations.  Arrays are numpy; bf16 is carried as raw uint16.

Readings taken where the paper is silent or ambiguous (each one is tagged at
the place it is used):

* R-GQA: with grouped-query attention the G query heads that share a KV head
  all act as queries of that head: one colsum over the G*|W| query rows.
* R-DENOM: the softmax runs over the compressible keys only (Eq. (4) as
  written); buffer keys take no part.
* R-TIE: every ranking is by (value descending, index ascending).
* R-GAP1: a candidate chunk must have a non-empty interior
  (2 <= I[k+1]-I[k] <= gamma-1).
* R-ORDER: after compaction the window holds the kept rows in ascending
  original order, then the buffer, then the tokens after the window.
* R-PAGES: compaction is in place in the window's own pages; the trailing
  logical blocks no longer needed are released in ascending order.
* R-PREFILL: prompt windows advance by |W|-|U| like decode-time windows, so
  consecutive windows share the |U| buffer positions (queries of both,
  compressible keys of the later one); all windows are scored and selected
  independently and at once.
* R-QSUBSET: scoring with part of the window's queries (the ablation that
  uses the buffer's queries only, Sec. 5.3) keeps Eq. (4)'s softmax over the
  compressible keys and column sum, over fewer rows.
"""

from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

# per-sequence status bits (same meaning as the library's)
SEQ_OK = 0
SEQ_BAD_WINDOW = 1
SEQ_BAD_PAGE = 2
SEQ_DUP_TRIGGER = 4
SEQ_BAD_INDEX = 8
SEQ_DUP_PAGE = 32


# ---------------------------------------------------------------- elements
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of raw bf16 bit patterns (uint16) to fp64."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def to_f64(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored elements ('bf16' as uint16 bits, or 'f32')."""
    if dtype == "bf16":
        return bf16_bits_to_f64(raw)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


# ------------------------------------------------------------- Eq. (4)
def window_scores(q: np.ndarray, k: np.ndarray, scale: float) -> np.ndarray:
    """Importance of each compressible KV pair, Eq. (4), in fp64.

    q: [R, d] every query row of the window (all |W| window tokens -- the
       buffer's included -- and, under R-GQA, every query head of the group);
    k: [N, d] keys of the compressible region W\\U (N = |W|-|U|);
    scale: the 1/sqrt(d) of Eq. (1).

    Logits are unmasked (bidirectional, Sec. 4.1); the softmax runs over the
    key dimension (R-DENOM: compressible keys only); colsum sums over every
    query row.
    """
    logits = (q @ k.T) * scale                    # [R, N], no causal mask
    m = logits.max(axis=1, keepdims=True)         # row-wise shift (exactness only)
    e = np.exp(logits - m)
    p = e / e.sum(axis=1, keepdims=True)          # softmax over keys
    return p.sum(axis=0)                          # colsum over all queries


def round_scores(a: np.ndarray) -> np.ndarray:
    """Scores are handed to selection as fp32 (round to nearest even)."""
    return np.asarray(a, dtype=np.float64).astype(np.float32)


# ------------------------------------------------------------- rankings
def rank_order(values: np.ndarray, positions: np.ndarray | None = None) -> np.ndarray:
    """Positions sorted by (value descending, position ascending) (R-TIE)."""
    v = np.asarray(values)
    if positions is None:
        positions = np.arange(v.shape[0])
    positions = np.asarray(positions, dtype=np.int64)
    key = v[positions].astype(np.float64)
    order = np.lexsort((positions, -key))         # last key is primary
    return positions[order]


# ------------------------------------------------------------- Eq. (5)
def discrete_topk(a32: np.ndarray, k: int) -> np.ndarray:
    """I = TopK(A, k), Eq. (5); returned sorted ascending as Eq. (6) needs."""
    if not 0 <= k <= a32.shape[0]:
        raise ValueError("k out of range")
    return np.sort(rank_order(a32)[:k])


# ------------------------------------------------------------- Eq. (6)-(8)
def chunk_candidates(a32: np.ndarray, disc: np.ndarray, gamma: int):
    """Candidate chunks between consecutive discrete indices, Eq. (6)-(7).

    Returns a list of (R_k, k) for every k whose span is within the maximum
    chunk length (I[k+1]-I[k] < gamma, endpoints included, Eq. (7)) and whose
    interior is non-empty (R-GAP1).  R_k is Eq. (6) in fp64 from fp32 scores.
    """
    out = []
    for k in range(len(disc) - 1):
        gap = int(disc[k + 1]) - int(disc[k])
        if gap < 2 or gap >= gamma:
            continue
        r = (float(a32[disc[k]]) + float(a32[disc[k + 1]])) * float(gap - 1)
        out.append((r, k))
    return out


def token2chunk(a32: np.ndarray, disc: np.ndarray, alpha: int, gamma: int):
    """Chunks chosen by Eq. (7) and the positions they add, Eq. (8).

    At most floor(alpha/(gamma-2)) chunks are taken, best (R desc, k asc)
    first.  Returns (chosen chunk ids ascending, added positions ascending).
    """
    n_chunks = alpha // (gamma - 2)
    cands = chunk_candidates(a32, disc, gamma)
    cands.sort(key=lambda rk: (-rk[0], rk[1]))
    chosen = sorted(k for _, k in cands[:n_chunks])
    added = []
    for k in chosen:
        added.extend(range(int(disc[k]) + 1, int(disc[k + 1])))
    return chosen, np.asarray(added, dtype=np.int64)


def fill_positions(a32: np.ndarray, taken: np.ndarray, count: int) -> np.ndarray:
    """Fill rule, App. C.3: top up with the best-scored unselected positions."""
    free = np.flatnonzero(~taken)
    return np.sort(rank_order(a32, free)[:count])


def kept_set(a32: np.ndarray, budget: int, alpha: int, gamma: int):
    """Final retained set I-hat of one (sequence, layer, KV head).

    Returns (I ascending, I-hat ascending).  |I-hat| == budget always.
    """
    n = a32.shape[0]
    if not (1 <= budget <= n and 0 <= alpha < budget and gamma >= 3):
        raise ValueError("bad selection parameters")
    disc = discrete_topk(a32, budget - alpha)                 # Eq. (5)
    _, added = token2chunk(a32, disc, alpha, gamma)           # Eq. (6)-(8)
    taken = np.zeros(n, dtype=bool)
    taken[disc] = True
    taken[added] = True
    fill = fill_positions(a32, taken, alpha - len(added))     # App. C.3
    taken[fill] = True
    kept = np.flatnonzero(taken)
    assert kept.shape[0] == budget
    return disc, kept


# ------------------------------------------------------- Eq. (9) + App. C.4
def compaction_map(kept: np.ndarray, window: int, buffer: int, tail: int) -> np.ndarray:
    """Window-relative source of each destination row after compaction.

    Eq. (9) keeps the rows of I-hat; the buffer rows and the tokens after the
    window follow them (R-ORDER).
    """
    return np.concatenate([
        np.asarray(kept, dtype=np.int64),
        np.arange(window - buffer, window, dtype=np.int64),
        np.arange(window, window + tail, dtype=np.int64),
    ])


def gather_rows(rows: np.ndarray, kept: np.ndarray, window: int, buffer: int) -> np.ndarray:
    """Rows [window + tail, ...] before compaction -> rows after (a gather)."""
    tail = rows.shape[0] - window
    return rows[compaction_map(kept, window, buffer, tail)].copy()


def released_blocks(seq_len: int, new_len: int, block_size: int):
    """Logical blocks released after compaction (UpdateMetadata)."""
    old_b = -(-seq_len // block_size)
    new_b = -(-new_len // block_size)
    return list(range(new_b, old_b))


# -------------------------------------------------------- paged cache model
def window_positions(p0: int, count: int) -> np.ndarray:
    return p0 + np.arange(count, dtype=np.int64)


def read_rows(pool: np.ndarray, table_row: np.ndarray, positions: np.ndarray, head: int,
              block_size: int) -> np.ndarray:
    """Rows of one KV head at logical positions, read through the block table."""
    pages = table_row[positions // block_size]
    slots = positions % block_size
    return pool[pages, head, slots, :]


def write_rows(pool: np.ndarray, table_row: np.ndarray, positions: np.ndarray, head: int,
               block_size: int, rows: np.ndarray) -> None:
    pages = table_row[positions // block_size]
    slots = positions % block_size
    pool[pages, head, slots, :] = rows


def validate(p: dict, trig: np.ndarray, block_table: np.ndarray, seq_lens: np.ndarray,
             win_start: np.ndarray) -> np.ndarray:
    """Per-trigger status word: which windows cannot be compressed."""
    n_seqs = block_table.shape[0]
    status = np.zeros(len(trig), dtype=np.int32)
    W, bs = p["window"], p["block_size"]
    for t, s in enumerate(trig):
        if not 0 <= s < n_seqs:
            status[t] |= SEQ_BAD_INDEX
            continue
        if np.count_nonzero(trig == s) > 1:
            status[t] |= SEQ_DUP_TRIGGER
        p0, L = int(win_start[s]), int(seq_lens[s])
        if p0 < 0 or p0 + W > L or L > p["max_blocks_per_seq"] * bs:
            status[t] |= SEQ_BAD_WINDOW
            continue
        pages = block_table[s, p0 // bs: -(-L // bs)]
        if np.any(pages < 0) or np.any(pages >= p["num_pages"]):
            status[t] |= SEQ_BAD_PAGE
        # R-PAGES: compaction rewrites the window's pages in place, so each
        # page it writes must hold no other block of the sequence
        row = block_table[s, :-(-L // bs)]
        for b in range(p0 // bs, len(row)):
            if 0 <= row[b] < p["num_pages"] and np.any(row[:b] == row[b]):
                status[t] |= SEQ_DUP_PAGE
                break
    return status


def scoring_queries(p: dict) -> int:
    """Wq: the window positions whose queries score (the last Wq).  Every
    position for Kara's Eq. (4); the buffer's alone for the ablation without
    bidirectional attention (Sec. 5.3), read here as the same softmax over
    the compressible keys and column sum, over fewer query rows."""
    return int(p.get("score_queries", 0) or p["window"])


def unit_queries(q_raw: np.ndarray, p: dict, layer: int, t: int, head: int) -> np.ndarray:
    """All query rows scoring KV head `head` (R-GQA): [Wq*G, d] in fp64.
    q_raw holds the Wq scoring positions' queries."""
    if q_raw.shape[2] != scoring_queries(p):
        raise ValueError(f"q has {q_raw.shape[2]} positions, the parameters score with {scoring_queries(p)}")
    G = p["n_q_heads"] // p["n_kv_heads"]
    rows = q_raw[layer, t, :, head * G:(head + 1) * G, :]     # [W, G, d]
    return to_f64(rows.reshape(-1, rows.shape[-1]), p["dtype"])


def unit_keys(k_pool: np.ndarray, p: dict, table_row: np.ndarray, p0: int, head: int) -> np.ndarray:
    n = p["window"] - p["buffer"]
    pos = window_positions(p0, n)
    return to_f64(read_rows(k_pool, table_row, pos, head, p["block_size"]), p["dtype"])


def scale_of(p: dict) -> float:
    s = float(p.get("scale", 0.0) or 0.0)
    return s if s > 0.0 else 1.0 / math.sqrt(p["head_dim"])


def score_units(p: dict, trig, q_raw, k_pools, block_table, win_start, units, threads: int = 0):
    """fp64 Eq. (4) scores for the listed (layer, trigger, head) units."""
    scale = scale_of(p)

    def one(u):
        l, t, h = u
        s = int(trig[t])
        qa = unit_queries(q_raw, p, l, t, h)
        ka = unit_keys(k_pools[l], p, block_table[s], int(win_start[s]), h)
        return window_scores(qa, ka, scale)

    units = list(units)
    if threads and threads > 1 and len(units) > 1:
        with ThreadPoolExecutor(threads) as ex:
            return list(ex.map(one, units))
    return [one(u) for u in units]


def compress(p: dict, trig, q_raw, k_pools, v_pools, block_table, seq_lens, win_start,
             commit: bool = True, threads: int = 0, score_override=None):
    """The whole step on host copies of the paged cache (mutated in place).

    Returns dict with status, scores (fp32, [L, n_trig, Hkv, N]), discrete,
    kept, freed lists and n_freed.  `score_override`, if given, replaces the
    scores (fp32 array of the same shape) before selection: used to run this
    oracle's selection on another implementation's scores.
    """
    trig = np.asarray(trig, dtype=np.int64)
    L = len(k_pools)
    nt = len(trig)
    H = p["n_kv_heads"]
    W, U, bs = p["window"], p["buffer"], p["block_size"]
    N = W - U
    budget, alpha, gamma = p["budget"], p["chunk_budget"], p["max_chunk_len"]
    status = validate(p, trig, block_table, seq_lens, win_start)

    scores = np.zeros((L, nt, H, N), dtype=np.float32)
    disc = np.zeros((L, nt, H, budget - alpha), dtype=np.int32)
    kept = np.zeros((L, nt, H, budget), dtype=np.int32)
    units = [(l, t, h) for l in range(L) for t in range(nt) for h in range(H) if status[t] == 0]
    if score_override is not None:
        scores[...] = score_override
    else:
        for u, a in zip(units, score_units(p, trig, q_raw, k_pools, block_table, win_start, units, threads)):
            scores[u] = round_scores(a)
    for (l, t, h) in [(l, t, h) for l in range(L) for t in range(nt) for h in range(H)]:
        d_, k_ = kept_set(scores[l, t, h], budget, alpha, gamma)
        disc[l, t, h] = d_
        kept[l, t, h] = k_

    freed, n_freed = [], np.zeros(nt, dtype=np.int32)
    for t in range(nt):
        if status[t] != 0:
            freed.append([])
            continue
        s = int(trig[t])
        p0, sl = int(win_start[s]), int(seq_lens[s])
        tail = sl - p0 - W
        pos = window_positions(p0, W + tail)
        for l in range(L):
            for pool in (k_pools[l], v_pools[l]):
                for h in range(H):
                    before = read_rows(pool, block_table[s], pos, h, bs)
                    after = gather_rows(before, kept[l, t, h], W, U)
                    write_rows(pool, block_table[s], pos[:after.shape[0]], h, bs, after)
        if commit:
            new_len = sl - (N - budget)
            blocks = released_blocks(sl, new_len, bs)
            freed.append([int(block_table[s, b]) for b in blocks])
            n_freed[t] = len(blocks)
            block_table[s, blocks] = -1
            seq_lens[s] = new_len
        else:
            freed.append([])
    return dict(status=status, scores=scores, discrete=disc, kept=kept, freed=freed, n_freed=n_freed)


def compress_prefill(p: dict, trig, n_windows: int, q_raw, k_pools, v_pools, block_table, seq_lens,
                     win_start, commit: bool = True, threads: int = 0, score_override=None):
    """Prefill-time compression (App. C.2) on host copies (mutated in place).

    The prompt of sequence s = trig[t] is split into n_windows windows,
    window w covering [p0 + w*(W-U), p0 + w*(W-U) + W) with p0 = win_start[s]
    (the window advances by W-U, as it does during decoding).  Each window is
    scored by its own queries q_raw[l, t, w] (Eq. (4)) and selected on its
    own (Eq. (5)-(8), App. C.3), all windows at once.  The cache then holds,
    in order, each window's kept rows and everything after the last window's
    compressible region (R-ORDER applied window by window), and the sequence
    is n_windows * (W-U-budget) shorter.

    q_raw: [L, n_trig, n_windows, Wq, Hq, d]; scores, discrete and kept gain
    the window axis after the trigger.
    """
    trig = np.asarray(trig, dtype=np.int64)
    L = len(k_pools)
    nt = len(trig)
    H = p["n_kv_heads"]
    W, U, bs = p["window"], p["buffer"], p["block_size"]
    N = W - U
    nw = int(n_windows)
    budget, alpha, gamma = p["budget"], p["chunk_budget"], p["max_chunk_len"]
    # the windows together span (nw-1)*N + W positions from p0
    status = validate(dict(p, window=(nw - 1) * N + W), trig, block_table, seq_lens, win_start)

    scores = np.zeros((L, nt, nw, H, N), dtype=np.float32)
    disc = np.zeros((L, nt, nw, H, budget - alpha), dtype=np.int32)
    kept = np.zeros((L, nt, nw, H, budget), dtype=np.int32)
    if score_override is not None:
        scores[...] = score_override
    else:
        for w in range(nw):
            starts = np.asarray(win_start, dtype=np.int64) + w * N
            units = [(l, t, h) for l in range(L) for t in range(nt) for h in range(H) if status[t] == 0]
            res = score_units(p, trig, q_raw[:, :, w], k_pools, block_table, starts, units, threads)
            for (l, t, h), a in zip(units, res):
                scores[l, t, w, h] = round_scores(a)
    for l in range(L):
        for t in range(nt):
            for w in range(nw):
                for h in range(H):
                    d_, k_ = kept_set(scores[l, t, w, h], budget, alpha, gamma)
                    disc[l, t, w, h] = d_
                    kept[l, t, w, h] = k_

    freed, n_freed = [], np.zeros(nt, dtype=np.int32)
    for t in range(nt):
        if status[t] != 0:
            freed.append([])
            continue
        s = int(trig[t])
        p0, sl = int(win_start[s]), int(seq_lens[s])
        pos = window_positions(p0, sl - p0)
        for l in range(L):
            for pool in (k_pools[l], v_pools[l]):
                for h in range(H):
                    before = read_rows(pool, block_table[s], pos, h, bs)
                    parts = [before[w * N + kept[l, t, w, h]] for w in range(nw)] + [before[nw * N:]]
                    after = np.concatenate(parts)
                    write_rows(pool, block_table[s], pos[:after.shape[0]], h, bs, after)
        if commit:
            new_len = sl - nw * (N - budget)
            blocks = released_blocks(sl, new_len, bs)
            freed.append([int(block_table[s, b]) for b in blocks])
            n_freed[t] = len(blocks)
            block_table[s, blocks] = -1
            seq_lens[s] = new_len
        else:
            freed.append([])
    return dict(status=status, scores=scores, discrete=disc, kept=kept, freed=freed, n_freed=n_freed)
