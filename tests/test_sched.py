"""The periodic compression policy (Algorithm 1, App. C.4): the C++ runtime
behind include/kara_sched.h against a hand-derived example, invariants, and
step by step against the plain Python model in oracle/.  Host code only."""
import numpy as np
import pytest

from oracle.kara_sched_model import SchedModel
from paper_2607_01237_amd import kara


def _cfg(**over):
    c = dict(n_slots=8, num_pages=64, block_size=4, max_blocks_per_seq=32, window=8, buffer=0, budget=2, period=4,
             max_per_event=30, max_running=8, reserve_pages=0, compress=1, protect_prompt=0)
    c.update(over)
    return c


def _drive(run, n_steps):
    """Runs a scheduler-like object (model or C++) through n_steps steps;
    returns per-step records of every decision."""
    recs = []
    for _ in range(n_steps):
        st = run.step_begin()
        trig, ws = run.step_end()
        rec = dict(pre=list(st["preempted"]), dec=list(st["decode"]), adm=list(st["admitted"]),
                   pl=list(st["prefill_len"]), trig=list(trig), ws=[int(ws[s]) for s in trig])
        if len(trig):
            rec["released"] = run.commit()
        recs.append(rec)
    return recs


class CppRun:
    """The C++ scheduler with the model's step interface; commit returns the
    released pages read back from the tables before and after."""

    def __init__(self, cfg, page_order=None):
        self.s = kara.Scheduler(cfg, page_order)
        self.cfg = cfg
        self.pending = []

    def step_begin(self):
        return self.s.step_begin()

    def step_end(self):
        trig, ws = self.s.step_end()
        self.pending = list(trig)
        return trig, ws

    def commit(self):
        bt0, _ = self.s.tables()
        self.s.commit()
        bt1, _ = self.s.tables()
        out = []
        for slot in self.pending:
            gone = np.nonzero((bt0[slot] >= 0) & (bt1[slot] < 0))[0]
            out.append([int(bt0[slot, b]) for b in gone])
        return out


# ---------------------------------------------------------------- pins
def test_single_sequence_hand_derived():
    """One sequence, no memory pressure: bs=4, |W|=8, |U|=0, budget 2,
    delta=4, prompt 4, 40 new tokens.  The prefill step is g=1, decoding steps
    g=2..41, so the length at the end of step g is g+3 until the first event.
    Events need g > 8 and g mod 4 == 0, and p0 + 8 <= 4*(ceil(len/4) - 1):
      g=12 len 15 p0 0: 8 <= 12  -> len 9,  p0 2, block 3 released
      g=16 len 13 p0 2: 10 <= 12 -> len 7,  p0 4, blocks 2,3 released
      g=20 len 11 p0 4: 12 > 8   -> no event
      g=24 len 15 p0 4: 12 <= 12 -> len 9,  p0 6, block 3 released
      g=28 len 13 p0 6: 14 > 12  -> no event
      g=32 len 17 p0 6: 14 <= 16 -> len 11, p0 8, blocks 3,4 released
      g=36 len 15 p0 8: 16 > 12  -> no event
      g=40 len 19 p0 8: 16 <= 16 -> len 13, p0 10, block 4 released
    and at g=41 the 40th token finishes the sequence."""
    want_g = [12, 16, 24, 32, 40]
    want_pre = [15, 13, 15, 17, 19]
    want_post = [9, 7, 9, 11, 13]
    want_released = [1, 2, 1, 2, 1]
    for run in (SchedModel(_cfg()), CppRun(_cfg())):
        run_s = run.s if isinstance(run, CppRun) else None
        (run if run_s is None else run_s).submit(4, 40)
        got_g, got_pre, got_post, got_rel = [], [], [], []
        for g in range(1, 42):
            run.step_begin()
            trig, ws = run.step_end()
            if len(trig):
                lens = run.lens if run_s is None else run_s.tables()[1]
                got_g.append(g)
                got_pre.append(int(lens[trig[0]]))
                rel = run.commit()
                got_rel.append(len(rel[0]))
                lens = run.lens if run_s is None else run_s.tables()[1]
                got_post.append(int(lens[trig[0]]))
        assert (got_g, got_pre, got_post, got_rel) == (want_g, want_pre, want_post, want_released)
        stats = run.snapshot() if run_s is None else run_s.stats()
        assert stats["finished"] == 1 and stats["tokens_decoded"] == 40 and stats["pages_reclaimed"] == 7
        assert stats["free_pages"] == 64


def test_no_event_before_window_or_off_period():
    """Algorithm 1 fires only when g > |W| and g mod delta == 0, whatever the
    lengths: with delta = 5 and |W| = 8 the only steps that may fire are 10,
    15, 20, ..."""
    cfg = _cfg(period=5, block_size=1, budget=1, max_blocks_per_seq=128, num_pages=400)
    s = kara.Scheduler(cfg)
    for _ in range(4):
        s.submit(20, 60)
    for g in range(1, 61):
        s.step_begin()
        trig, _ = s.step_end()
        if len(trig):
            assert g > 8 and g % 5 == 0
            s.commit()
    assert s.stats()["events"] > 0


def test_compression_off_never_fires():
    s = kara.Scheduler(_cfg(compress=0))
    for _ in range(3):
        s.submit(10, 50)
    for _ in range(60):
        s.step_begin()
        trig, _ = s.step_end()
        assert len(trig) == 0
    assert s.stats()["pages_reclaimed"] == 0


def _check_invariants(s: kara.Scheduler, cfg):
    bt, lens = s.tables()
    st = s.stats()
    mapped = bt[bt >= 0]
    assert len(np.unique(mapped)) == len(mapped), "a page is mapped twice"
    assert len(mapped) + st["free_pages"] == cfg["num_pages"], "pages lost or duplicated"
    bs = cfg["block_size"]
    for slot in range(cfg["n_slots"]):
        nb = int((bt[slot] >= 0).sum())
        assert (bt[slot, :nb] >= 0).all(), "holes in a block-table row"
        assert nb == -(-int(lens[slot]) // bs), f"slot {slot}: {nb} blocks for length {lens[slot]}"
    assert st["running"] <= cfg["max_running"]


@pytest.mark.parametrize("seed,over", [
    (0, {}),
    (1, dict(buffer=2, budget=3, window=10)),
    (2, dict(num_pages=40, max_running=6)),           # tight pool (compression avoids preemption)
    (3, dict(protect_prompt=1, block_size=3, period=3)),
    (4, dict(compress=0, num_pages=48)),              # uncompressed: preemptions
    (5, dict(max_per_event=1, block_size=1, window=6, budget=1, num_pages=300, max_blocks_per_seq=80)),
    (6, dict(num_pages=30, reserve_pages=2, buffer=1, window=9, budget=2, period=2)),
])
def test_runtime_matches_model(seed, over):
    """Every decision of the C++ runtime (preemptions, decoding slots,
    admissions, events, window starts, released pages, tables, statistics)
    equals the model's, step by step, on a seeded stream of requests; the
    runtime's page accounting holds after every step."""
    cfg = _cfg(**over)
    rng = np.random.default_rng(seed)
    order = rng.permutation(cfg["num_pages"]).astype(np.int32)
    model, cpp = SchedModel(cfg, order), CppRun(cfg, order)
    n_req = 14
    prompts = rng.integers(1, 12, n_req)
    news = rng.integers(5, 60, n_req)
    arrive = np.sort(rng.integers(0, 60, n_req))
    k = 0
    for step in range(260):
        while k < n_req and arrive[k] <= step:
            assert model.submit(int(prompts[k]), int(news[k])) == cpp.s.submit(int(prompts[k]), int(news[k]))
            k += 1
        a = _drive(model, 1)[0]
        b = _drive(cpp, 1)[0]
        assert a == b, f"step {step}: model {a} != runtime {b}"
        bt, lens = cpp.s.tables()
        assert np.array_equal(bt, np.array(model.table, dtype=np.int32)), f"step {step}: block tables differ"
        assert np.array_equal(lens, np.array(model.lens, dtype=np.int32)), f"step {step}: lengths differ"
        _check_invariants(cpp.s, cfg)
        st, ms = cpp.s.stats(), model.snapshot()
        for key in ms:
            assert st[key] == ms[key], f"step {step}: {key} {st[key]} != {ms[key]}"
    assert cpp.s.stats()["finished"] == n_req
    for rid in range(n_req):
        info = cpp.s.request(rid)
        assert info["state"] == kara.REQ_FINISHED and info["generated"] == news[rid]


def test_preemption_happens_and_recovers():
    """A pool too small for every sequence uncompressed: the runtime preempts,
    readmits with the whole context, and still finishes every request."""
    cfg = _cfg(num_pages=24, max_running=8, compress=0)
    s = kara.Scheduler(cfg)
    for _ in range(6):
        s.submit(6, 50)
    for _ in range(2000):
        s.step_begin()
        trig, _ = s.step_end()
        _check_invariants(s, cfg)
        if s.stats()["finished"] == 6:
            break
    st = s.stats()
    assert st["finished"] == 6 and st["preemptions"] > 0
    assert st["tokens_decoded"] >= 6 * 50
    # a readmitted request prefilled its generated tokens again
    assert st["tokens_prefilled"] > 6 * 6


def test_compression_raises_concurrency():
    """The point of the policy: with the same constrained pool, compressing
    keeps more sequences running and finishes the same requests in fewer
    steps than the uncompressed baseline."""
    res = {}
    for comp in (0, 1):
        cfg = _cfg(num_pages=60, max_running=16, n_slots=16, block_size=4, window=16, budget=4, period=8,
                   compress=comp, max_blocks_per_seq=64)
        s = kara.Scheduler(cfg)
        for _ in range(16):
            s.submit(8, 120)
        running = []
        for step in range(5000):
            s.step_begin()
            trig, _ = s.step_end()
            if len(trig):
                s.commit()
            running.append(s.stats()["running"])
            if s.stats()["finished"] == 16:
                break
        res[comp] = (step + 1, float(np.mean(running)), s.stats()["preemptions"])
    assert res[1][0] < res[0][0], res
    assert res[1][1] > res[0][1], res


def test_commit_checks_device_freed_list():
    cfg = _cfg()
    s = kara.Scheduler(cfg)
    s.submit(4, 40)
    for _ in range(12):
        s.step_begin()
        trig, _ = s.step_end()
    assert list(trig) == [0]
    bt, lens = s.tables()
    freed = np.full((1, cfg["max_blocks_per_seq"]), -1, dtype=np.int32)
    freed[0, 0] = bt[0, 3] + 1 if bt[0, 3] + 1 < cfg["num_pages"] else 0   # wrong page
    with pytest.raises(kara.KaraError) as e:
        s.commit(freed, np.array([1], dtype=np.int32))
    assert e.value.code == kara.ERR_SCHED_MISMATCH
    # the host state was updated from its own computation anyway
    assert s.tables()[1][0] == 9
    # and a correct list passes at the next event
    for _ in range(4):
        s.step_begin()
        trig, _ = s.step_end()
    assert list(trig) == [0]
    bt, lens = s.tables()
    freed = np.full((1, cfg["max_blocks_per_seq"]), -1, dtype=np.int32)
    freed[0, :2] = bt[0, 2:4]
    s.commit(freed, np.array([2], dtype=np.int32))


def test_bad_config_and_calls_rejected():
    for over in (dict(budget=0), dict(budget=9), dict(buffer=8), dict(period=0), dict(max_per_event=0),
                 dict(max_running=9), dict(reserve_pages=64), dict(window=5000, budget=10), dict(block_size=0)):
        with pytest.raises(kara.KaraError):
            kara.Scheduler(_cfg(**over))
    with pytest.raises(kara.KaraError):
        kara.Scheduler(_cfg(), page_order=np.zeros(64, dtype=np.int32))      # not a permutation
    s = kara.Scheduler(_cfg())
    with pytest.raises(kara.KaraError):
        s.submit(0, 5)
    with pytest.raises(kara.KaraError):
        s.submit(100, 100)                                                   # outgrows the block table
    with pytest.raises(kara.KaraError):
        s.step_end()                                                         # no step begun
    s.submit(4, 40)
    s.step_begin()
    with pytest.raises(kara.KaraError):
        s.step_begin()                                                       # step begun twice
    s.step_end()
    with pytest.raises(kara.KaraError):
        s.commit()                                                           # no event pending
    for _ in range(11):
        s.step_begin()
        trig, _ = s.step_end()
    assert len(trig) == 1
    with pytest.raises(kara.KaraError):
        s.step_begin()                                                       # event not committed
    s.commit()
    s.step_begin()
