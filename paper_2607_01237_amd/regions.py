"""Survivors per region of the original sequence under repeated compression.

The paper contrasts a threshold-triggered policy, which compresses the whole
cache again each time it reaches its limit (Sec. 3, Eq. (2)-(3)), with
Kara's sliding window, which compresses each window once (Sec. 4, App.
C.4): under the first, early parts of the sequence keep losing tokens at
every event; under the second, a region keeps what its window kept.  This
module runs both policies on the GPU through kara_compress_window over a
long synthetic generation and counts, after every event, how many tokens of
each region of the original sequence (fixed-size spans of token indices)
are still cached, averaged over layers and KV heads.

Which original token a cache row holds is tracked twice: on the host, by
applying every event's kept sets to per-(layer, head) lists of token
indices, and on the device, where every V row carries its token's index in
its first two entries (index // 256 and index % 256, exact in bf16; V does
not take part in scoring).  check() compares the two.
"""

from __future__ import annotations

import numpy as np

from . import kara

KARA, THRESHOLD = "kara", "threshold"


class Regions:
    def __init__(self, shape: dict, policy: str, geo: dict, n_seqs: int, max_tokens: int, device, seed: int):
        import torch

        self.torch = torch
        self.dev = device
        self.policy = policy
        self.L, self.Hq, self.Hkv, self.d = shape["n_layers"], shape["n_q_heads"], shape["n_kv_heads"], shape["head_dim"]
        self.n = n_seqs
        self.W, self.U, self.budget = geo["window"], geo["buffer"], geo["budget"]
        self.N = self.W - self.U
        self.bs = geo["block_size"]
        self.Wq = geo.get("score_queries", 0) or self.W
        self.max_tokens = max_tokens
        self.max_blocks = -(-max_tokens // self.bs)
        num_pages = n_seqs * self.max_blocks
        p = dict(window=self.W, buffer=self.U, budget=self.budget, chunk_budget=geo["chunk_budget"],
                 max_chunk_len=geo["max_chunk_len"], head_dim=self.d, n_q_heads=self.Hq, n_kv_heads=self.Hkv,
                 block_size=self.bs, num_pages=num_pages, max_blocks_per_seq=self.max_blocks, dtype="bf16",
                 scale=0.0, score_queries=geo.get("score_queries", 0))
        self.params = kara.make_params(p, n_seqs)
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        shape_p = (num_pages, self.Hkv, self.bs, self.d)
        self.kp = [torch.zeros(shape_p, dtype=torch.bfloat16, device=device) for _ in range(self.L)]
        self.vp = [torch.zeros(shape_p, dtype=torch.bfloat16, device=device) for _ in range(self.L)]
        # sequence s owns pages s*max_blocks .. for the whole run: the trailing
        # blocks a commit releases are mapped again (to the same pages) before
        # the next append
        bt = np.arange(num_pages, dtype=np.int32).reshape(n_seqs, self.max_blocks)
        self.bt0 = torch.from_numpy(bt).to(device)
        self.bt = self.bt0.clone()
        self.lens = torch.zeros(n_seqs, dtype=torch.int32, device=device)
        self.win_start = torch.zeros(n_seqs, dtype=torch.int32, device=device)
        self.seqs = torch.arange(n_seqs, dtype=torch.int32, device=device)
        self.app_status = torch.zeros(n_seqs, dtype=torch.int32, device=device)
        self.status = torch.zeros(n_seqs, dtype=torch.int32, device=device)
        self.kept = torch.empty((self.L, n_seqs, self.Hkv, self.budget), dtype=torch.int32, device=device)
        self.freed = torch.empty((n_seqs, self.max_blocks), dtype=torch.int32, device=device)
        self.n_freed = torch.empty(n_seqs, dtype=torch.int32, device=device)
        self.ws = torch.empty(kara.workspace_size(self.params, n_seqs, self.L), dtype=torch.uint8, device=device)
        self.generated = 0               # tokens generated per sequence (all sequences in step)
        self.p0 = 0                      # window start (all sequences alike)
        # host: original token index of every cache row, per (sequence, layer, head)
        self.ids = [[[np.zeros(0, dtype=np.int64) for _ in range(self.Hkv)] for _ in range(self.L)]
                    for _ in range(n_seqs)]
        self.events = 0

    def append(self, n_tok):
        torch = self.torch
        shape = (self.L, self.n, n_tok, self.Hkv, self.d)
        k_new = torch.randn(shape, generator=self.gen, device=self.dev).to(torch.bfloat16)
        v_new = torch.randn(shape, generator=self.gen, device=self.dev).to(torch.bfloat16)
        idx = torch.arange(self.generated, self.generated + n_tok, device=self.dev)
        v_new[..., 0] = (idx // 256).to(torch.bfloat16).view(1, 1, n_tok, 1)
        v_new[..., 1] = (idx % 256).to(torch.bfloat16).view(1, 1, n_tok, 1)
        kara.kv_append(self.params, self.seqs, k_new, v_new, self.kp, self.vp, self.bt, self.lens, self.app_status)
        new = np.arange(self.generated, self.generated + n_tok, dtype=np.int64)
        for s in range(self.n):
            for l in range(self.L):
                for h in range(self.Hkv):
                    self.ids[s][l][h] = np.concatenate([self.ids[s][l][h], new])
        self.generated += n_tok

    def length(self):
        return len(self.ids[0][0][0])

    def due(self):
        """Kara: a whole uncompressed window exists; threshold: the cache reached the window (its limit)."""
        if self.policy == KARA:
            return self.length() - self.p0 >= self.W
        return self.length() >= self.W

    def compress(self):
        torch = self.torch
        self.win_start.fill_(self.p0)
        q = torch.randn((self.L, self.n, self.Wq, self.Hq, self.d), generator=self.gen, device=self.dev).to(
            torch.bfloat16)
        kara.compress_window(self.params, self.seqs, q, self.kp, self.vp, self.bt, self.lens, self.win_start, True,
                             self.status, self.ws, kept=self.kept, freed=self.freed, n_freed=self.n_freed)
        st = self.status.cpu().numpy()
        if (st != 0).any():
            raise RuntimeError(f"compression flagged {st.tolist()}")
        self.bt.copy_(self.bt0)
        kept = self.kept.cpu().numpy()
        p0, N = self.p0, self.N
        for s in range(self.n):
            for l in range(self.L):
                for h in range(self.Hkv):
                    ids = self.ids[s][l][h]
                    self.ids[s][l][h] = np.concatenate([ids[:p0], ids[p0 + kept[l, s, h]], ids[p0 + N:]])
        if self.policy == KARA:
            self.p0 += self.budget
        self.events += 1

    def survivors(self, region: int, n_regions: int) -> np.ndarray:
        """Mean cached tokens per region of `region` original tokens, over
        sequences, layers and KV heads."""
        out = np.zeros(n_regions)
        for s in range(self.n):
            for l in range(self.L):
                for h in range(self.Hkv):
                    out += np.bincount(self.ids[s][l][h] // region, minlength=n_regions)[:n_regions]
        return out / (self.n * self.L * self.Hkv)

    def check(self):
        """The device cache's token indices (from V) equal the host's lists."""
        torch = self.torch
        n = self.length()
        pos = torch.arange(n, device=self.dev)
        for s in range(self.n):
            pages = self.bt[s, pos // self.bs].long()
            slots = (pos % self.bs).long()
            if int(self.lens[s]) != n:
                raise RuntimeError(f"sequence {s}: device length {int(self.lens[s])} != {n}")
            for l in range(self.L):
                rows = self.vp[l][pages, :, slots, :2].float()                   # [n, Hkv, 2]
                got = (rows[..., 0] * 256 + rows[..., 1]).long().cpu().numpy()   # [n, Hkv]
                for h in range(self.Hkv):
                    if not np.array_equal(got[:, h], self.ids[s][l][h]):
                        raise RuntimeError(f"sequence {s} layer {l} head {h}: cached tokens differ")


def run(shape, geos: dict, n_seqs, n_tokens, chunk, region, device, seed, check_every=0):
    """Both policies over the same generation length; returns per-event
    survivor tables {policy: [(tokens generated, [survivors per region])]}."""
    n_regions = -(-n_tokens // region)
    out = {}
    for policy, geo in geos.items():
        r = Regions(shape, policy, geo, n_seqs, n_tokens, device, seed)
        rows = []
        while r.generated < n_tokens:
            r.append(min(chunk, n_tokens - r.generated))
            while r.due():
                r.compress()
                rows.append((r.generated, r.survivors(region, n_regions).tolist()))
                if check_every and r.events % check_every == 0:
                    r.check()
        if check_every:
            r.check()
        out[policy] = dict(events=rows, final=r.survivors(region, n_regions).tolist(), cache_len=r.length())
    return out
