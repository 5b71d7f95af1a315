"""Plain model of KvLLM's periodic compression policy (Algorithm 1, App. C.4).

TEST INFRASTRUCTURE: only tests/, the package's smoke check and the bench's
CPU baseline use this module; the product's scheduler is the C++ runtime
behind include/kara_sched.h, which shares nothing with it.

Algorithm 1 in plain Python, a loop over lists:
  while the running queue is not empty:
      run one decoding step for every running sequence (the K/V cache grows
      by one token each);
      g += 1;
      if g > |W| and g mod delta == 0:
          Q' = Select(Q): sequences whose trailing |W| tokens are uncompressed;
          for each e in Q': compress the window, compact the memory, update
          the metadata (length, block table, released blocks).

Around it, the serving loop of a paged-attention engine: a waiting queue,
admission when pages and slots allow, a page per block of tokens, and
preemption when a decoding sequence finds no free page.  Where the paper
leaves these open, the model takes the readings stated in kara_sched.h's
policy: preemption of the most recently admitted sequence (recompute: it is
readmitted later with its whole context uncompressed), admission only in
steps without preemption, first come first served; the Select condition
p0 + |W| <= block_size * (ceil(len / block_size) - 1), so the last,
possibly partial, block stays out of every window; candidates in queue
order, at most max_per_event; after compression the length drops by
|W| - |U| - budget, trailing blocks are released in ascending order and p0
advances by budget (the buffer re-enters the next window, App. C.2).
The free page list is first in, first out.

Parity pins (tests/test_sched.py) do not rest on this model alone: closed
forms for one sequence without memory pressure (event steps, lengths, pages
reclaimed) and invariants (page conservation, Select's condition, the event
rule of Algorithm 1) check it first.
"""

from __future__ import annotations

from collections import deque


def _blocks(n, bs):
    return -(-n // bs)


class SchedModel:
    def __init__(self, cfg: dict, page_order=None):
        d = dict(reserve_pages=0, compress=1, protect_prompt=0)
        d.update(cfg)
        self.c = d
        n, mb = d["n_slots"], d["max_blocks_per_seq"]
        self.table = [[-1] * mb for _ in range(n)]
        self.lens = [0] * n
        self.p0 = [0] * n
        self.owner = [-1] * n
        pages = list(range(d["num_pages"])) if page_order is None else [int(x) for x in page_order]
        self.free = deque(pages)
        self.free_slots = list(range(n - 1, -1, -1))   # pop() gives slot 0 first
        self.waiting = deque()
        self.running = []
        self.reqs = []
        self.g = 0
        self.pending = []
        self.stats = dict(events=0, compressed=0, pages_reclaimed=0, preemptions=0, tokens_decoded=0,
                          tokens_prefilled=0, finished=0, peak_running=0)
        self._step = None

    # ---- requests
    def submit(self, prompt_len, max_new):
        bs, c = self.c["block_size"], self.c
        need = _blocks(prompt_len + max_new, bs)
        if prompt_len < 1 or max_new < 1 or need > c["max_blocks_per_seq"] or need > c["num_pages"] - c["reserve_pages"]:
            raise ValueError("request does not fit")
        self.reqs.append(dict(prompt=prompt_len, max_new=max_new, gen=0, state=0, slot=-1, comp=0, pre=0,
                              prefill=prompt_len))
        rid = len(self.reqs) - 1
        self.waiting.append(rid)
        return rid

    # ---- pages
    def _mapped(self, slot):
        row = self.table[slot]
        n = 0
        while n < len(row) and row[n] >= 0:
            n += 1
        return n

    def _map(self, slot, n_tokens):
        for b in range(_blocks(n_tokens, self.c["block_size"])):
            if self.table[slot][b] < 0:
                self.table[slot][b] = self.free.popleft()

    def _vacate(self, slot):
        for b, pg in enumerate(self.table[slot]):
            if pg < 0:
                break
            self.free.append(pg)
            self.table[slot][b] = -1
        self.lens[slot] = 0
        self.p0[slot] = 0
        self.owner[slot] = -1
        self.free_slots.append(slot)

    def _preempt_last(self, out):
        rid = self.running.pop()
        r = self.reqs[rid]
        slot = r["slot"]
        r.update(prefill=r["prompt"] + r["gen"], state=0, slot=-1, pre=r["pre"] + 1)
        self.stats["preemptions"] += 1
        self._vacate(slot)
        out["preempted"].append(slot)
        self.waiting.appendleft(rid)

    # ---- one step of the serving loop
    def step_begin(self):
        assert self._step is None and not self.pending
        c, bs = self.c, self.c["block_size"]
        out = dict(preempted=[], decode=[], admitted=[], prefill_len=[], admitted_id=[])
        i = 0
        while i < len(self.running):
            rid = self.running[i]
            slot = self.reqs[rid]["slot"]
            need = _blocks(self.lens[slot] + 1, bs)
            gone = False
            while self._mapped(slot) < need and not self.free:
                victim = self.running[-1]
                self._preempt_last(out)
                if victim == rid:
                    gone = True
                    break
            if gone:
                break
            self._map(slot, self.lens[slot] + 1)
            out["decode"].append(slot)
            i += 1
        if not out["preempted"]:
            while self.waiting and self.free_slots and len(self.running) < c["max_running"]:
                rid = self.waiting[0]
                r = self.reqs[rid]
                if len(self.free) < _blocks(r["prefill"], bs) + c["reserve_pages"]:
                    break
                self.waiting.popleft()
                slot = self.free_slots.pop()
                r.update(state=1, slot=slot)
                self.owner[slot] = rid
                self.lens[slot] = 0
                self.p0[slot] = r["prompt"] if c["protect_prompt"] else 0
                self._map(slot, r["prefill"])
                self.running.append(rid)
                out["admitted"].append(slot)
                out["prefill_len"].append(r["prefill"])
                out["admitted_id"].append(rid)
        self.stats["peak_running"] = max(self.stats["peak_running"], len(self.running))
        self._step = out
        return out

    def step_end(self):
        out = self._step
        assert out is not None
        self._step = None
        c, bs = self.c, self.c["block_size"]
        for slot, n in zip(out["admitted"], out["prefill_len"]):
            self.lens[slot] = n
            self.stats["tokens_prefilled"] += n
        for slot in out["decode"]:
            self.lens[slot] += 1
            self.reqs[self.owner[slot]]["gen"] += 1
            self.stats["tokens_decoded"] += 1
        keep = []
        for rid in self.running:
            r = self.reqs[rid]
            if r["gen"] >= r["max_new"]:
                r["state"] = 2
                self._vacate(r["slot"])
                r["slot"] = -1
                self.stats["finished"] += 1
            else:
                keep.append(rid)
        self.running = keep
        # Algorithm 1: the counter, then the periodic event
        self.g += 1
        trig = []
        if c["compress"] and self.g > c["window"] and self.g % c["period"] == 0:
            for rid in self.running:
                if len(trig) == c["max_per_event"]:
                    break
                slot = self.reqs[rid]["slot"]
                last_block_start = bs * (_blocks(self.lens[slot], bs) - 1)
                if self.p0[slot] + c["window"] <= last_block_start:
                    trig.append(slot)
        self.pending = trig
        return list(trig), list(self.p0)

    def commit(self):
        """The metadata update of every sequence of the pending event; returns
        each one's released pages in ascending logical-block order."""
        c, bs = self.c, self.c["block_size"]
        shrink = c["window"] - c["buffer"] - c["budget"]
        released = []
        for slot in self.pending:
            old = self.lens[slot]
            new = old - shrink
            pages = []
            for b in range(_blocks(new, bs), _blocks(old, bs)):
                pages.append(self.table[slot][b])
                self.free.append(self.table[slot][b])
                self.table[slot][b] = -1
            released.append(pages)
            self.stats["pages_reclaimed"] += len(pages)
            self.lens[slot] = new
            self.p0[slot] += c["budget"]
            self.reqs[self.owner[slot]]["comp"] += 1
        if self.pending:
            self.stats["events"] += 1
            self.stats["compressed"] += len(self.pending)
        self.pending = []
        return released

    # ---- reports
    def snapshot(self):
        return dict(steps=self.g, running=len(self.running), waiting=len(self.waiting), free_pages=len(self.free),
                    pages_in_use=self.c["num_pages"] - len(self.free), **self.stats)
