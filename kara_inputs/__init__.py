"""Seeded synthetic workloads for the KV-compression step.

This module only draws random numbers and lays out paged-cache geometry
(block tables, window starts, sequence lengths).  It holds none of the
method's arithmetic and is shared by the tests, the benchmark and the
oracle-side checks, which all receive the same bytes from it.

The paper measures on reasoning benchmarks run through trained models
(Kara Sec. 5); neither datasets nor weights are used here.  Instead every
workload below draws Q/K/V with the shapes of the models the paper serves
(Qwen3-8B: 32 query / 8 KV heads, head dim 128; Qwen3-14B: 40 / 8, 128) and
the window hyper-parameters of App. B.

Workloads (name -> what it is):

* ``tiny``      1 sequence, 1 layer, 4/1 heads, d=64, fp32; W=128, budget 26
                (20 %), gamma=4, alpha=4; block 16, 32 pages, shuffled table.
* ``batch8``    8 sequences, 1 layer, 32/8 heads, d=128, bf16; W=1024,
                budget 205; 2 % of the window positions of each (sequence,
                KV head) have keys scaled by 4 (heavy hitters).
* ``qwen14b``   64 sequences, 40 layers, 40/8 heads, d=128, bf16; W=2048,
                budget 410; 4K-16K tokens of earlier context resident;
                keys carry a random rank-8 component per (layer, head).
* ``ragged``    256 sequences, 36 layers, 32/8 heads, bf16; W=1024; each
                sequence's uncompressed fill drawn from 0..W+127, so only the
                sequences with a full window trigger; pool ~90 % occupied,
                pages handed out from a shuffled free list.
* ``buffer_only``  the ``qwen14b`` batch with a 64-token buffer whose queries
                alone score the compressible 1984 keys (the ablation without
                bidirectional attention, Sec. 5.3); budget ceil(0.2*1984).
* ``threshold_topk`` the whole-cache top-k of Eq. (2)-(3) as a baseline:
                128 sequences, R1-Llama-8B shape (32 layers, 32/8 heads),
                cache at the threshold C_max = 1280 tokens compressed to
                1025 (the vLLM+SnapKV setting of App. B.1): the window is the
                whole cache, its last 32 tokens (observation queries) are
                kept and score the other 1248, 993 of which are kept by
                plain top-k (no chunks).
* ``prefill``   16 prompts of 16K-17K tokens, Qwen3-8B shape (36 layers,
                32/8 heads), compressed before decoding in 16 windows of
                W=1024 each (App. C.2), budget 205 per window; the prompt's
                last 0-1023 tokens (short of a window) stay uncompressed.
* ``soak``      128 sequences, 40 layers, 40/8 heads; a 1K prompt, then 31
                intervals of W=1024 generated tokens (appended 128 at a time,
                one decode step per append) each ending in a compression
                event, so contexts grow to 32K logical tokens; fresh N(0,1)
                Q/K/V every interval; pool = peak need + 1 %, pages handed out
                from a shuffled free list (``soak_geometry``).

Every workload uses U=0 unless a variant sets ``buffer``: the tiny case's
"budget 26 of W=128 (20 %)" equals ceil(0.2*128) only with no buffer.
"""

from __future__ import annotations

import copy
from dataclasses import dataclass, field

import numpy as np

BASE = {
    "tiny": dict(n_seqs=1, n_layers=1, n_q_heads=4, n_kv_heads=1, head_dim=64, dtype="f32",
                 window=128, buffer=0, budget=26, max_chunk_len=4, chunk_budget=4,
                 block_size=16, num_pages=32, seed=0, prefix=(64, 64), tail=(5, 5),
                 pool_slack=None, key_mode="normal"),
    "batch8": dict(n_seqs=8, n_layers=1, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                   window=1024, buffer=0, budget=205, max_chunk_len=8, chunk_budget=16,
                   block_size=16, num_pages=4096, seed=1, prefix=(0, 2047), tail=(0, 15),
                   pool_slack=None, key_mode="heavy"),
    "qwen14b": dict(n_seqs=64, n_layers=40, n_q_heads=40, n_kv_heads=8, head_dim=128, dtype="bf16",
                    window=2048, buffer=0, budget=410, max_chunk_len=8, chunk_budget=16,
                    block_size=16, num_pages=None, seed=2, prefix=(4096, 16384), tail=(0, 15),
                    pool_slack=0.10, key_mode="lowrank"),
    "ragged": dict(n_seqs=256, n_layers=36, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                   window=1024, buffer=0, budget=205, max_chunk_len=8, chunk_budget=16,
                   block_size=16, num_pages=None, seed=3, prefix=(0, 4096), tail=None,
                   pool_slack="occupancy90", key_mode="normal", fill_max=1024 + 127),
    "buffer_only": dict(n_seqs=64, n_layers=40, n_q_heads=40, n_kv_heads=8, head_dim=128, dtype="bf16",
                        window=2048, buffer=64, budget=397, max_chunk_len=8, chunk_budget=16,
                        block_size=16, num_pages=None, seed=5, prefix=(4096, 16384), tail=(0, 15),
                        pool_slack=0.10, key_mode="lowrank", score_queries=64),
    "threshold_topk": dict(n_seqs=128, n_layers=32, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                           window=1280, buffer=32, budget=993, max_chunk_len=8, chunk_budget=0,
                           block_size=16, num_pages=None, seed=6, prefix=(0, 0), tail=(0, 0),
                           pool_slack=0.10, key_mode="normal", score_queries=32),
    "prefill": dict(n_seqs=16, n_layers=36, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                    window=1024, buffer=0, budget=205, max_chunk_len=8, chunk_budget=16,
                    block_size=16, num_pages=None, seed=7, prefix=(0, 0), tail=(0, 1023),
                    pool_slack=0.10, key_mode="normal", n_windows=16),
    "recompute": dict(n_seqs=16, n_layers=36, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16",
                      window=1024, buffer=0, budget=205, max_chunk_len=8, chunk_budget=16,
                      block_size=16, num_pages=None, seed=9, prefix=(3072, 15360), tail=(0, 15),
                      pool_slack=0.05, key_mode="normal", hidden=4096, ffn=12288, rope_theta=1e6,
                      rms_eps=1e-6),
    "soak": dict(n_seqs=128, n_layers=40, n_q_heads=40, n_kv_heads=8, head_dim=128, dtype="bf16",
                 window=1024, buffer=0, budget=205, max_chunk_len=8, chunk_budget=16,
                 block_size=16, num_pages=None, seed=4, prefix=(1024, 1024), tail=(0, 0),
                 pool_slack=0.01, key_mode="normal", n_intervals=31, append_chunk=128, n_dec=8),
}


def workload(name: str, **over) -> dict:
    """A workload description, optionally with fields overridden (for the
    scaled-down variants that the tests run against the full oracle)."""
    cfg = copy.deepcopy(BASE[name])
    cfg.update(over)
    cfg["name"] = name
    return cfg


@dataclass
class Geometry:
    """Host-side metadata of one batch (numpy, int32)."""
    cfg: dict
    trig: np.ndarray
    seq_lens: np.ndarray
    win_start: np.ndarray
    block_table: np.ndarray
    num_pages: int
    max_blocks: int
    extra: dict = field(default_factory=dict)

    def params(self) -> dict:
        c = self.cfg
        return dict(window=c["window"], buffer=c["buffer"], budget=c["budget"],
                    chunk_budget=c["chunk_budget"], max_chunk_len=c["max_chunk_len"],
                    head_dim=c["head_dim"], n_q_heads=c["n_q_heads"], n_kv_heads=c["n_kv_heads"],
                    block_size=c["block_size"], num_pages=self.num_pages,
                    max_blocks_per_seq=self.max_blocks, dtype=c["dtype"], scale=0.0,
                    n_layers=c["n_layers"], score_queries=c.get("score_queries", 0))


def _blocks(n_tokens: int, bs: int) -> int:
    return -(-n_tokens // bs)


def make_geometry(cfg: dict) -> Geometry:
    """Sequence lengths, window starts, triggers and a shuffled page table."""
    rng = np.random.default_rng(cfg["seed"])
    B, W, bs = cfg["n_seqs"], cfg["window"], cfg["block_size"]
    lo, hi = cfg["prefix"]
    prefix = rng.integers(lo, hi + 1, B)
    if cfg.get("fill_max") is not None:
        # ragged serving: uncompressed fill per sequence; only full windows fire
        fill = rng.integers(0, cfg["fill_max"] + 1, B)
        trig = np.flatnonzero(fill >= W)
        seq_lens = prefix + fill
        win_start = np.where(fill >= W, prefix, 0)
    else:
        tlo, thi = cfg["tail"]
        tail = rng.integers(tlo, thi + 1, B)
        trig = np.arange(B)
        # n_windows consecutive windows (prefill) advance by W - U
        nw = cfg.get("n_windows", 1)
        seq_lens = prefix + (nw - 1) * (W - cfg["buffer"]) + W + tail
        win_start = prefix
    need = np.array([_blocks(int(L), bs) for L in seq_lens])
    max_blocks = int(cfg.get("max_blocks") or need.max())
    used = int(need.sum())
    if cfg["num_pages"] is not None:
        num_pages = int(cfg["num_pages"])
    elif cfg["pool_slack"] == "occupancy90":
        num_pages = int(np.ceil(used / 0.90))
    else:
        num_pages = int(np.ceil(used * (1.0 + cfg["pool_slack"])))
    if used > num_pages:
        raise ValueError("pool too small for the batch")
    free_list = rng.permutation(num_pages)          # fragmented free list
    table = np.full((B, max_blocks), -1, dtype=np.int32)
    c = 0
    for s in range(B):
        table[s, :need[s]] = free_list[c:c + need[s]]
        c += need[s]
    return Geometry(cfg=cfg, trig=trig.astype(np.int32), seq_lens=seq_lens.astype(np.int32),
                    win_start=win_start.astype(np.int32), block_table=table,
                    num_pages=num_pages, max_blocks=max_blocks,
                    extra=dict(free_pages=free_list[c:].astype(np.int32)))


@dataclass
class SoakGeometry:
    """Sizes of the decode-loop soak: the longest physical length any
    sequence reaches, the block-table width, the pool, and the initial
    (shuffled) free list."""
    max_tokens: int
    max_blocks: int
    num_pages: int
    free_list: np.ndarray


def soak_geometry(cfg: dict) -> SoakGeometry:
    """Each interval appends W tokens; the event then leaves `budget` of them
    (no buffer, U = 0), so before the last event a sequence holds
    prompt + (n-1)*budget + W."""
    if cfg["buffer"] != 0:
        raise ValueError("the soak runs with U = 0")
    bs, W = cfg["block_size"], cfg["window"]
    prompt = cfg["prefix"][0]
    max_tokens = prompt + (cfg["n_intervals"] - 1) * cfg["budget"] + W
    max_blocks = _blocks(max_tokens, bs)
    num_pages = int(np.ceil(cfg["n_seqs"] * max_blocks * (1.0 + cfg["pool_slack"])))
    rng = np.random.default_rng(cfg["seed"])
    return SoakGeometry(max_tokens=max_tokens, max_blocks=max_blocks, num_pages=num_pages,
                        free_list=rng.permutation(num_pages).astype(np.int32))


# ---------------------------------------------------------------- serving
# The serving analogue of the paper's KvLLM runs (App. B.1): an 8B-class
# decoder (32 layers, 32/8 heads, d=128, bf16), 256-token blocks, windows of
# three blocks (768) with a 32-token buffer, 257 tokens retained per window
# (budget 225 plus the buffer), an event every 128 steps compressing at most
# 30 sequences.  A batch of requests with short prompts and reasoning-length
# generations arrives at once, against a pool that holds about 37 % of what
# the batch would need uncompressed, so admission is memory bound.
SERVE = dict(
    shape=dict(n_layers=32, n_q_heads=32, n_kv_heads=8, head_dim=128, dtype="bf16", chunk_budget=16,
               max_chunk_len=8),
    sched=dict(n_slots=256, block_size=256, window=768, buffer=32, budget=225, period=128, max_per_event=30,
               max_running=256, reserve_pages=4, protect_prompt=0),
    n_requests=128, prompt=(64, 256), gen=(1024, 3072), pool_frac=0.37, seed=8,
)


def serve_setup(cfg: dict = None, **over):
    """(shape, scheduler config without `compress`, prompts, generation
    lengths, initial free list) of a serving run.  Lengths are uniform in the
    stated closed ranges; the pool is pool_frac of the batch's uncompressed
    demand, rounded up to whole pages."""
    c = copy.deepcopy(SERVE if cfg is None else cfg)
    c.update(over)
    rng = np.random.default_rng(c["seed"])
    n = c["n_requests"]
    prompts = rng.integers(c["prompt"][0], c["prompt"][1] + 1, n).astype(np.int32)
    gens = rng.integers(c["gen"][0], c["gen"][1] + 1, n).astype(np.int32)
    sc = dict(c["sched"])
    bs = sc["block_size"]
    sc["max_blocks_per_seq"] = _blocks(int((prompts + gens).max()), bs)
    sc["num_pages"] = _blocks(int(np.ceil(c["pool_frac"] * float((prompts + gens).sum()))), bs)
    order = rng.permutation(sc["num_pages"]).astype(np.int32)
    return dict(c["shape"]), sc, prompts, gens, order


# ---------------------------------------------------------------- tensors
def torch_dtype(cfg):
    import torch
    return torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32


def _gen(device, seed):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def scoring_queries(cfg: dict) -> int:
    """Number of window positions whose queries score (the last ones)."""
    return cfg.get("score_queries", 0) or cfg["window"]


def make_queries(geom: Geometry, layer: int, device="cpu"):
    """Scoring queries of one layer: [n_trig, Wq, Hq, d] ~ N(0,1), Wq the
    scoring positions (the whole window unless the workload narrows it)."""
    import torch
    c = geom.cfg
    g = _gen(device, c["seed"] * 1_000_003 + 7919 * layer + 1)
    shape = (len(geom.trig), scoring_queries(c), c["n_q_heads"], c["head_dim"])
    if c.get("n_windows", 1) > 1:       # prefill: [n_trig, n_windows, Wq, Hq, d]
        shape = (shape[0], c["n_windows"]) + shape[1:]
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch_dtype(c))


def _row_index(geom: Geometry, seqs=None):
    """(page, slot) of every window and tail token of the triggered sequences."""
    bs = geom.cfg["block_size"]
    pages, slots, owner, pos_all = [], [], [], []
    seqs = geom.trig if seqs is None else seqs
    for t, s in enumerate(seqs):
        pos = np.arange(geom.win_start[s], geom.seq_lens[s])
        pages.append(geom.block_table[s, pos // bs])
        slots.append(pos % bs)
        owner.append(np.full(pos.shape, t))
        pos_all.append(pos)
    return (np.concatenate(pages), np.concatenate(slots), np.concatenate(owner), np.concatenate(pos_all))


def make_pools(geom: Geometry, layer: int, device="cpu"):
    """K and V pools of one layer, [num_pages, Hkv, bs, d].

    Window and tail tokens of the triggered sequences get random rows; the
    rest of the pool (earlier context, free pages) stays zero -- the step
    never reads it.
    """
    import torch
    c = geom.cfg
    Hkv, d, bs = c["n_kv_heads"], c["head_dim"], c["block_size"]
    dt = torch_dtype(c)
    kp = torch.zeros((geom.num_pages, Hkv, bs, d), dtype=dt, device=device)
    vp = torch.zeros_like(kp)
    pages, slots, owner, pos = _row_index(geom)
    n = pages.shape[0]
    g = _gen(device, c["seed"] * 1_000_003 + 7919 * layer + 2)
    kr = torch.randn((n, Hkv, d), generator=g, device=device, dtype=torch.float32)
    vr = torch.randn((n, Hkv, d), generator=g, device=device, dtype=torch.float32)
    if c["key_mode"] == "heavy":
        # 2 % of each (sequence, KV head)'s window positions get 4x key norm
        rng = np.random.default_rng(c["seed"] * 7 + layer)
        W = c["window"]
        scale = np.ones((n, Hkv), dtype=np.float32)
        starts = np.concatenate([[0], np.cumsum(np.bincount(owner, minlength=len(geom.trig)))])
        n_heavy = max(1, int(round(0.02 * W)))
        for t in range(len(geom.trig)):
            for h in range(Hkv):
                sel = rng.choice(W, n_heavy, replace=False)
                scale[starts[t] + sel, h] = 4.0
        kr = kr * torch.from_numpy(scale).to(device)[:, :, None]
    elif c["key_mode"] == "lowrank":
        # K = Z + B_{l,h} c_t with B ~ N(0, 1/8) per (layer, head), c_t ~ N(0,1)^8
        r = 8
        B = torch.randn((Hkv, d, r), generator=g, device=device, dtype=torch.float32) / np.sqrt(r)
        ct = torch.randn((n, r), generator=g, device=device, dtype=torch.float32)
        low = torch.matmul(ct[None], B.transpose(1, 2).contiguous())      # [Hkv, n, d]
        kr = kr + low.permute(1, 0, 2)
    pg = torch.from_numpy(pages.astype(np.int64)).to(device)
    sl = torch.from_numpy(slots.astype(np.int64)).to(device)
    kp[pg, :, sl, :] = kr.to(dt)
    vp[pg, :, sl, :] = vr.to(dt)
    return kp, vp


def raw_numpy(t):
    """Host copy of a tensor's stored bytes: bf16 as uint16 bits, fp32 as is."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()
