"""Decode-loop soak driver: the compression step inside a running decode loop.

Per interval of W generated tokens, for every sequence of the batch:
  1. map the blocks the next tokens need, from a host free list of pages;
  2. append fresh K/V rows (kara_harness_kv_append), `append_chunk` tokens at
     a time, each append followed by one decode step (one query per sequence,
     layer and query head over the whole cache, kara_harness_decode_attention);
  3. compress the window [p0, p0 + W) of every sequence in every layer
     (kara_compress_window, with the metadata commit);
  4. put the pages the commit freed back on the free list; p0 += budget.

The host keeps a model of the page pool (free list, block tables, lengths)
and checks it against what the device returns after every event: the freed
pages must be exactly the trailing blocks the new length no longer covers,
and no page may be mapped twice or lost.  All arithmetic on K/V runs in the
library's kernels; this module only draws inputs, moves page ids and times.
"""

from __future__ import annotations

import numpy as np

from . import kara


class PagePool:
    """Host model of the paged pool: free list, block tables, lengths."""

    def __init__(self, n_seqs, num_pages, max_blocks, block_size, free_list):
        self.num_pages = num_pages
        self.bs = block_size
        self.free = [int(x) for x in free_list[::-1]]      # pop() hands out free_list in order
        self.table = np.full((n_seqs, max_blocks), -1, dtype=np.int32)
        self.lens = np.zeros(n_seqs, dtype=np.int32)

    def reserve(self, seqs, n_new):
        """Maps every block that positions [len, len + n_new) of the listed
        sequences need and that is not mapped yet."""
        for s in seqs:
            first = -(-int(self.lens[s]) // self.bs)
            last = -(-(int(self.lens[s]) + n_new) // self.bs)
            if last > self.table.shape[1]:
                raise RuntimeError(f"sequence {s} outgrows its block table")
            for b in range(first, last):
                if not self.free:
                    raise RuntimeError("page pool exhausted")
                self.table[s, b] = self.free.pop()

    def release(self, seqs, new_lens, freed, n_freed):
        """Applies one commit: the blocks past each new length go back to the
        free list; returns the number of pages reclaimed.  Raises if the
        device's freed list is not exactly those blocks' pages."""
        total = 0
        for t, s in enumerate(seqs):
            old, new = int(self.lens[s]), int(new_lens[t])
            blocks = np.arange(-(-new // self.bs), -(-old // self.bs))
            want = self.table[s, blocks]
            got = freed[t, :int(n_freed[t])]
            if not np.array_equal(want, got):
                raise RuntimeError(f"sequence {s}: freed pages {got.tolist()} != trailing blocks {want.tolist()}")
            self.free.extend(int(x) for x in want)
            self.table[s, blocks] = -1
            self.lens[s] = new
            total += len(blocks)
        return total

    def check(self):
        mapped = self.table[self.table >= 0]
        if len(np.unique(mapped)) != len(mapped):
            raise RuntimeError("a page is mapped twice")
        if len(mapped) + len(self.free) != self.num_pages or len(set(self.free)) != len(self.free):
            raise RuntimeError("pages lost or duplicated")
        if np.isin(np.asarray(self.free, dtype=np.int64), mapped).any():
            raise RuntimeError("a free page is still mapped")


class Soak:
    """State of one soak run on one GPU: pools, host pool model, inputs."""

    def __init__(self, cfg, geom, device, generator):
        import torch

        self.torch = torch
        self.cfg = cfg
        self.dev = device
        self.gen = generator
        c = cfg
        self.L, self.n = c["n_layers"], c["n_seqs"]
        self.W, self.budget, self.chunk = c["window"], c["budget"], c["append_chunk"]
        if self.W % self.chunk != 0:
            raise ValueError("append_chunk must divide the window")
        self.Hq, self.Hkv, self.d, self.bs = c["n_q_heads"], c["n_kv_heads"], c["head_dim"], c["block_size"]
        self.dt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
        self.max_len = geom.max_tokens
        p = dict(window=self.W, buffer=c["buffer"], budget=self.budget, chunk_budget=c["chunk_budget"],
                 max_chunk_len=c["max_chunk_len"], head_dim=self.d, n_q_heads=self.Hq, n_kv_heads=self.Hkv,
                 block_size=self.bs, num_pages=geom.num_pages, max_blocks_per_seq=geom.max_blocks,
                 dtype=c["dtype"], scale=0.0)
        self.p = p
        self.params = kara.make_params(p, self.n)
        self.pool = PagePool(self.n, geom.num_pages, geom.max_blocks, self.bs, geom.free_list)
        shape = (geom.num_pages, self.Hkv, self.bs, self.d)
        # rows are written by the append before anything reads them
        self.kp = [torch.empty(shape, dtype=self.dt, device=device) for _ in range(self.L)]
        self.vp = [torch.empty(shape, dtype=self.dt, device=device) for _ in range(self.L)]
        n, L = self.n, self.L
        self.seqs = torch.arange(n, dtype=torch.int32, device=device)
        self.bt = torch.from_numpy(self.pool.table).to(device)
        self.lens = torch.zeros(n, dtype=torch.int32, device=device)
        self.win_start = torch.zeros(n, dtype=torch.int32, device=device)
        self.k_new = torch.empty((L, n, self.chunk, self.Hkv, self.d), dtype=self.dt, device=device)
        self.v_new = torch.empty_like(self.k_new)
        self.q_dec = torch.empty((L, n, self.Hq, self.d), dtype=self.dt, device=device)
        self.out = torch.empty((L, n, self.Hq, self.d), dtype=torch.float32, device=device)
        self.dec_ws = torch.empty(kara.decode_workspace_size(self.params, n, L, self.max_len), dtype=torch.uint8,
                                  device=device)
        self.q = torch.empty((L, n, self.W, self.Hq, self.d), dtype=self.dt, device=device)
        self.ws = torch.empty(kara.workspace_size(self.params, n, L), dtype=torch.uint8, device=device)
        self.status = torch.zeros(n, dtype=torch.int32, device=device)
        self.app_status = torch.zeros(n, dtype=torch.int32, device=device)
        self.app_bad = torch.zeros((), dtype=torch.bool, device=device)
        self.freed = torch.empty((n, geom.max_blocks), dtype=torch.int32, device=device)
        self.n_freed = torch.empty(n, dtype=torch.int32, device=device)
        self.kept = torch.empty((L, n, self.Hkv, self.budget), dtype=torch.int32, device=device)
        self.disc = torch.empty((L, n, self.Hkv, self.budget - c["chunk_budget"]), dtype=torch.int32,
                                device=device)
        self.scores = torch.empty((L, n, self.Hkv, self.W - c["buffer"]), dtype=torch.float32, device=device)
        self.p0 = np.zeros(n, dtype=np.int32)
        self.reclaimed = 0

    def page_bytes(self):
        """K+V bytes of one page over all layers."""
        return 2 * self.L * self.Hkv * self.bs * self.d * (2 if self.dt == self.torch.bfloat16 else 4)

    def append(self, n_tok):
        """Maps pages and appends n_tok fresh N(0,1) rows to every sequence."""
        self.pool.reserve(range(self.n), n_tok)
        self.bt.copy_(self.torch.from_numpy(self.pool.table))
        k_new, v_new = self.k_new[:, :, :n_tok], self.v_new[:, :, :n_tok]
        if n_tok != self.chunk:
            k_new, v_new = k_new.contiguous(), v_new.contiguous()
        k_new.normal_(generator=self.gen)
        v_new.normal_(generator=self.gen)
        kara.kv_append(self.params, self.seqs, k_new, v_new, self.kp, self.vp, self.bt, self.lens,
                       self.app_status)
        self.app_bad |= (self.app_status != 0).any()
        self.pool.lens += n_tok
        return k_new, v_new

    def decode(self, events=None):
        """One decode step with fresh queries; HIP events bracket the call."""
        self.q_dec.normal_(generator=self.gen)
        if events:
            events[0].record()
        kara.decode_attention(self.params, self.seqs, self.q_dec, self.kp, self.vp, self.bt, self.lens,
                              self.max_len, self.out, self.dec_ws)
        if events:
            events[1].record()

    def draw_queries(self):
        """Fresh N(0,1) window queries for the next event; sets the window starts."""
        self.q.normal_(generator=self.gen)
        self.win_start.copy_(self.torch.from_numpy(self.p0))

    def compress(self, events=None, want_scores=False, fresh_q=True):
        """One compression event over every sequence and layer (with the
        queries draw_queries() left when fresh_q is False)."""
        if fresh_q:
            self.draw_queries()
        if events:
            events[0].record()
        kara.compress_window(self.params, self.seqs, self.q, self.kp, self.vp, self.bt, self.lens, self.win_start,
                             True, self.status, self.ws, scores=self.scores if want_scores else None,
                             discrete=self.disc if want_scores else None, kept=self.kept, freed=self.freed,
                             n_freed=self.n_freed)
        if events:
            events[1].record()

    def settle(self):
        """After an event: check the device against the host pool model and
        reclaim the freed pages.  Returns the pages reclaimed."""
        torch = self.torch
        torch.cuda.synchronize()
        if bool(self.app_bad):
            raise RuntimeError("an append flagged a sequence")
        st = self.status.cpu().numpy()
        if (st != 0).any():
            raise RuntimeError(f"per-sequence status {st}")
        lens = self.lens.cpu().numpy()
        want = self.pool.lens - (self.W - self.cfg["buffer"] - self.budget)
        if not np.array_equal(lens, want):
            raise RuntimeError("device lengths differ from the pool model")
        got = self.pool.release(range(self.n), lens, self.freed.cpu().numpy(), self.n_freed.cpu().numpy())
        if not np.array_equal(self.bt.cpu().numpy(), self.pool.table):
            raise RuntimeError("device block table differs from the pool model")
        self.pool.check()
        self.p0 += self.budget
        self.reclaimed += got
        return got

    def prompt(self):
        """The uncompressed prompt, appended in chunks (not timed)."""
        left = self.cfg["prefix"][0]
        while left > 0:
            self.append(min(self.chunk, left))
            left -= min(self.chunk, left)
        self.p0[:] = self.cfg["prefix"][0]
