"""Serving loop on one GPU under the periodic compression policy.

The scheduler (include/kara_sched.h, C++) decides every step; this module
moves its decisions to the GPU and back:

  1. step_begin: preemptions, pages for each running sequence's next token,
     admissions.  The host block table and lengths are copied to the device
     when they changed.
  2. Admitted sequences prefill their prompt (or, after a preemption, their
     whole context) with fresh N(0,1) K/V rows (kara_harness_kv_append).
  3. Every decoding sequence appends one fresh K/V row and runs one decode
     step: one N(0,1) query per layer and query head over its paged cache
     (kara_harness_decode_attention).
  4. step_end: the counter g advances; at an event the triggered sequences'
     windows are compressed in every layer (kara_compress_window, with the
     metadata commit) using fresh N(0,1) window queries, and the scheduler
     takes the device's freed-page list back (kara_sched_event_commit checks
     it against its own).

There are no model weights: token contents and queries are synthetic, so a
step costs what the cache costs (appends, attention over the live context,
compression), which is the part of serving the policy changes.
"""

from __future__ import annotations

import numpy as np

from . import kara


class Serve:
    def __init__(self, shape: dict, sched_cfg: dict, device, seed: int, page_order=None, check=False):
        import torch

        self.torch = torch
        self.dev = device
        self.check = check
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        c = dict(kara.Scheduler.CONFIG_DEFAULTS, **sched_cfg)
        self.c = c
        self.sched = kara.Scheduler(c, page_order)
        self.L, self.Hq, self.Hkv, self.d = shape["n_layers"], shape["n_q_heads"], shape["n_kv_heads"], shape["head_dim"]
        self.dt = torch.bfloat16 if shape["dtype"] == "bf16" else torch.float32
        self.n_slots, self.mb, self.bs = c["n_slots"], c["max_blocks_per_seq"], c["block_size"]
        self.W, self.U, self.budget = c["window"], c["buffer"], c["budget"]
        self.max_len = self.mb * self.bs
        p = dict(window=self.W, buffer=self.U, budget=self.budget, chunk_budget=shape["chunk_budget"],
                 max_chunk_len=shape["max_chunk_len"], head_dim=self.d, n_q_heads=self.Hq, n_kv_heads=self.Hkv,
                 block_size=self.bs, num_pages=c["num_pages"], max_blocks_per_seq=self.mb, dtype=shape["dtype"],
                 scale=0.0)
        self.p = p
        self.params = kara.make_params(p, self.n_slots)
        pshape = (c["num_pages"], self.Hkv, self.bs, self.d)
        # every row is written by an append before anything reads it
        self.kp = [torch.empty(pshape, dtype=self.dt, device=device) for _ in range(self.L)]
        self.vp = [torch.empty(pshape, dtype=self.dt, device=device) for _ in range(self.L)]
        self.bt = torch.full((self.n_slots, self.mb), -1, dtype=torch.int32, device=device)
        self.lens = torch.zeros(self.n_slots, dtype=torch.int32, device=device)
        self.win_start = torch.zeros(self.n_slots, dtype=torch.int32, device=device)
        self.app_status = torch.zeros(self.n_slots, dtype=torch.int32, device=device)
        self.app_bad = torch.zeros((), dtype=torch.bool, device=device)
        self.dec_ws = torch.empty(kara.decode_workspace_size(self.params, self.n_slots, self.L, self.max_len),
                                  dtype=torch.uint8, device=device)
        self.outbuf = torch.empty(self.L * self.n_slots * self.Hq * self.d, dtype=torch.float32, device=device)
        m = c["max_per_event"]
        self.qbuf = torch.empty(self.L * m * self.W * self.Hq * self.d, dtype=self.dt, device=device)
        self.ws = torch.empty(kara.workspace_size(self.params, m, self.L), dtype=torch.uint8, device=device)
        self.status = torch.zeros(m, dtype=torch.int32, device=device)
        self.freed = torch.empty((m, self.mb), dtype=torch.int32, device=device)
        self.n_freed = torch.empty(m, dtype=torch.int32, device=device)
        self.history = []      # per step: running, waiting, decoded, free pages, event size
        self.n_submitted = 0

    def submit(self, prompt_len, max_new):
        rid = self.sched.submit(prompt_len, max_new)
        self.n_submitted += 1
        return rid

    def _upload(self):
        bt, lens = self.sched.tables()
        self.bt.copy_(self.torch.from_numpy(bt))
        self.lens.copy_(self.torch.from_numpy(lens))

    def _rand(self, shape):
        t = self.torch.empty(shape, dtype=self.dt, device=self.dev)
        t.normal_(generator=self.gen)
        return t

    def _append(self, slots, n_new):
        torch = self.torch
        seqs = torch.from_numpy(np.asarray(slots, dtype=np.int32)).to(self.dev)
        shape = (self.L, len(slots), n_new, self.Hkv, self.d)
        kara.kv_append(self.params, seqs, self._rand(shape), self._rand(shape), self.kp, self.vp, self.bt,
                       self.lens, self.app_status)
        self.app_bad |= (self.app_status[:len(slots)] != 0).any()
        return seqs

    def step(self):
        """One step of the serving loop; returns the event's triggered slots."""
        torch = self.torch
        st = self.sched.step_begin()
        if st["tables_changed"]:
            self._upload()
        for slot, n in zip(st["admitted"], st["prefill_len"]):
            self._append([int(slot)], int(n))
        nd = len(st["decode"])
        if nd:
            seqs = self._append(st["decode"], 1)
            q = self._rand((self.L, nd, self.Hq, self.d))
            out = self.outbuf[:self.L * nd * self.Hq * self.d].view(self.L, nd, self.Hq, self.d)
            kara.decode_attention(self.params, seqs, q, self.kp, self.vp, self.bt, self.lens, self.max_len, out,
                                  self.dec_ws)
        finished = self.sched.stats()["finished"]
        trig, ws = self.sched.step_end()
        if self.sched.stats()["finished"] != finished:
            # finished sequences left the tables; the device follows now, so
            # its tables equal the scheduler's at every step boundary
            self._upload()
        nt = len(trig)
        if nt:
            self.win_start.copy_(torch.from_numpy(ws))
            tdev = torch.from_numpy(trig).to(self.dev)
            q = self.qbuf[:self.L * nt * self.W * self.Hq * self.d].view(self.L, nt, self.W, self.Hq, self.d)
            q.normal_(generator=self.gen)
            kara.compress_window(self.params, tdev, q, self.kp, self.vp, self.bt, self.lens, self.win_start, True,
                                 self.status[:nt], self.ws, freed=self.freed[:nt], n_freed=self.n_freed[:nt])
            status = self.status[:nt].cpu().numpy()
            if (status != 0).any():
                raise RuntimeError(f"compression flagged slots {trig[status != 0].tolist()}: {status.tolist()}")
            self.sched.commit(self.freed[:nt].cpu().numpy(), self.n_freed[:nt].cpu().numpy())
        if self.check:
            self.verify()
        s = self.sched.stats()
        self.history.append((s["running"], s["waiting"], nd, s["free_pages"], nt))
        return trig

    def verify(self):
        """The device's tables equal the scheduler's and no append was flagged."""
        self.torch.cuda.synchronize()
        if bool(self.app_bad):
            raise RuntimeError("an append flagged a sequence")
        bt, lens = self.sched.tables()
        if not np.array_equal(self.lens.cpu().numpy(), lens):
            raise RuntimeError("device lengths differ from the scheduler's")
        if not np.array_equal(self.bt.cpu().numpy(), bt):
            raise RuntimeError("device block table differs from the scheduler's")

    def run(self, max_steps):
        """Steps until every submitted request finished (or max_steps)."""
        for i in range(max_steps):
            self.step()
            if self.sched.stats()["finished"] == self.n_submitted:
                return i + 1
        return max_steps
