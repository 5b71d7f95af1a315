"""Benchmark of one Kara compression event on one MI355X.

A step is the whole path -- validation, window scoring, discrete TopK,
Token2Chunk + fill, in-place compaction of K and V, metadata commit -- for
every triggered sequence, layer and KV head of one batch, through
kara_compress_window.  Inputs are resident in HBM before timing starts.
Before every step (warm-up, timed and staged alike) the block table, the
sequence lengths and every K/V row compaction can overwrite are restored
from a device backup, outside the timed region, so every step compresses
the same fresh input; HIP events on the launch stream bracket the
compression call alone.

Prints one JSON line.  `value` is window tokens compressed per second
(triggered sequences x windows x window length per step / step time).  `roofline`
covers the dominant kernel (scoring) from a staged pass that times each
stage with HIP events on the launch stream; `roofline_select_compact` covers
the HBM-bound stages.  `cpu_baseline` times the CPU oracle on a bounded
sample of units on this host.

    python bench.py [--steps K] [--warmup W] [--workload qwen14b|batch8|ragged|buffer_only|threshold_topk|prefill]
    python bench.py --workload soak [--intervals n] [--warmup W]
    python bench.py --workload serve [--requests n]
    python bench.py --workload recompute [--steps K] [--warmup W]
    python bench.py --workload regions

The soak runs the compression step inside a decode loop (append, decode
attention, compress, reclaim pages; paper_2607_01237_amd/soak.py) and reports
per-event compression latency, per-step decode latency and pages reclaimed;
its `value` averages the events after the first W.  The serve workload runs
a batch of requests through the periodic policy's serving loop
(paper_2607_01237_amd/serve.py) with and without compression on the same
memory-bound pool and reports generated tokens/s of each.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 (matrix and vector)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen14b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--intervals", type=int, default=0, help="soak only: number of compression intervals "
                                                             "(default: the workload's 31)")
    ap.add_argument("--requests", type=int, default=0, help="serve only: number of requests (default: the "
                                                           "workload's 128)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="rough budget of the CPU-oracle sample")
    ap.add_argument("--copy-calibration-gib", type=float, default=0.0,
                    help="run one plain streaming kernel (bf16 negation) over this many GiB before the steps, as "
                         "the reference for rocprofv3 FETCH_SIZE / WRITE_SIZE counts")
    ap.add_argument("--summarize-counters", nargs="+", metavar="CSV",
                    help="print the per-kernel mean per dispatch of every counter in rocprofv3 --pmc CSVs, and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print the HBM-traffic summary of two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) "
                         "of this script with --copy-calibration-gib, and exit")
    return ap.parse_args()


# ---- HBM traffic from hardware counters ----
# The counters come from two separate rocprofv3 --pmc runs of this script
# (one counter block each).  Each counter is scaled by what it reads for a
# plain streaming kernel of known size in the same run, and the result is
# stored in profiles/ together with a hash of the kernel sources it was taken
# on; a changed source makes the stored figure stale and the JSON reports null.

TRAFFIC_SOURCES = {
    "score": ["paper_2607_01237_amd/csrc/kara_score.hip"],
    "select_compact": ["paper_2607_01237_amd/csrc/kara_select.hip", "paper_2607_01237_amd/csrc/kara_pages.hip"],
}
TRAFFIC_KERNELS = {"score": ["score1_kernel", "score_kernel", "split_sum_kernel"],
                   "select_compact": ["compact_kernel", "select_kernel"]}


def scoring_kernel_name(p):
    """Which scoring kernel the library runs for these parameters (the rule
    of its plan_score: the single-sweep kernel for bf16, d = 128 and
    512 < N <= 2048 with pools and query blocks addressable by 32-bit
    offsets; the two-sweep kernel otherwise)."""
    n = p["window"] - p["buffer"]
    pool = p["num_pages"] * p["n_kv_heads"] * p["block_size"] * p["head_dim"] * 2
    qblk = (p.get("score_queries") or p["window"]) * p["n_q_heads"] * p["head_dim"] * 2
    if p["dtype"] == "bf16" and p["head_dim"] == 128 and 512 < n <= 2048 and pool < 2**32 and qblk < 2**32:
        return "score1_kernel (single-sweep window scoring, Eq. 4)"
    return "score_kernel (two-sweep window scoring, Eq. 4)"
CALIBRATION_KERNEL = "neg_kernel"


def sources_sha256(paths):
    import hashlib
    h = hashlib.sha256()
    for rel in paths:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_path(workload):
    return os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")


def load_traffic(workload):
    """Stored per-launch HBM bytes of each stage, or None where stale/absent."""
    out = {"score": None, "select_compact": None}
    path = traffic_path(workload)
    if not os.path.exists(path):
        return out
    text = open(path).read()
    if "```json" not in text:
        return out
    blob = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    for stage in out:
        rec = blob.get(stage)
        if rec and rec.get("sources_sha256") == sources_sha256(TRAFFIC_SOURCES[stage]):
            out[stage] = rec["hbm_bytes_per_launch"]
    return out


def _pmc_per_dispatch(csv_path, counter):
    import csv
    per = {}
    names = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        d = r["Dispatch_Id"]
        per[d] = per.get(d, 0.0) + float(r["Counter_Value"])
        names[d] = r["Kernel_Name"]
    return per, names


def summarize_pmc(fetch_csv, write_csv, workload, calib_gib):
    fetch, names = _pmc_per_dispatch(fetch_csv, "FETCH_SIZE")
    write, wnames = _pmc_per_dispatch(write_csv, "WRITE_SIZE")
    true_bytes = calib_gib * 2**30

    def total_of(per, nm, key):
        vals = [v * 1024.0 for d, v in per.items() if key in nm[d]]   # counters are KiB per dispatch
        return float(np.sum(vals)), len(vals)

    # torch splits the negation of more than 2^31 elements into several
    # dispatches: the calibration is the total over all of them
    cf, ncf = total_of(fetch, names, CALIBRATION_KERNEL)
    cw, ncw = total_of(write, wnames, CALIBRATION_KERNEL)
    if not ncf or not ncw:
        raise SystemExit("the calibration kernel is missing from the counter runs (use --copy-calibration-gib)")
    sf, sw = true_bytes / cf, true_bytes / cw
    lines = [f"# HBM traffic from rocprofv3 counters: {workload} workload", "",
             "Two counter runs of the same command, one per counter block:", "", "```",
             f"cd /tmp && export TMPDIR=/tmp && rocprofv3 --pmc FETCH_SIZE -d $OUT/pmc_fetch -o pmc "
             f"--output-format csv -- python3 $REPO/bench.py --workload {workload} --steps 1 --warmup 0 "
             f"--no-cpu-baseline --copy-calibration-gib {calib_gib:g}",
             "(the same with --pmc WRITE_SIZE and -d $OUT/pmc_write; $OUT is any output directory)",
             f"python3 bench.py --workload {workload} --copy-calibration-gib {calib_gib:g} "
             "--summarize-pmc <fetch csv> <write csv>", "```", "",
             f"Calibration: one bf16 negation over {calib_gib:g} GiB ({ncf} dispatches) reads and writes "
             f"{true_bytes / 1e9:.3f} GB; the "
             f"counters read {cf / 1e9:.3f} GB fetched and {cw / 1e9:.3f} GB written, so FETCH_SIZE is scaled by "
             f"{sf:.4f} and WRITE_SIZE by {sw:.4f}.", "",
             "| kernel | dispatches | FETCH (GB, scaled) | WRITE (GB, scaled) |", "|---|---|---|---|"]
    blob = {"workload": workload, "calibration_gib": calib_gib, "fetch_scale": sf, "write_scale": sw}
    for stage, kernels in TRAFFIC_KERNELS.items():
        total = 0.0
        passes = None
        for k in kernels:
            f_b, n = total_of(fetch, names, k)
            w_b, _ = total_of(write, wnames, k)
            if n == 0:
                continue
            passes = n if passes is None else passes
            lines.append(f"| {k} | {n} | {f_b * sf / n / 1e9:.3f} | {w_b * sw / n / 1e9:.3f} |")
            total += f_b * sf + w_b * sw
        # per pass of the stage: the first kernel of the stage runs once per pass
        blob[stage] = {"kernels": kernels, "hbm_bytes_per_launch": total / passes if passes else None,
                       "sources_sha256": sources_sha256(TRAFFIC_SOURCES[stage])}
    lines += ["", "The table gives the average per dispatch.  Per pass of a stage (one scoring launch; one "
              "selection-and-compaction pass, selection being one launch in the staged pass and in the fused step "
              "alike):", "", "```json", json.dumps(blob, indent=1), "```"]
    return "\n".join(lines)


def summarize_counters(paths):
    """Markdown table: for every kernel (name up to its argument list), the
    number of dispatches and the mean per dispatch of each counter found."""
    import csv
    vals, disp = {}, {}
    for path in paths:
        per = {}
        for r in csv.DictReader(open(path)):
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").split("(", 1)[0].replace("void ", "")
            name = name if len(name) <= 60 else name[:57] + "..."
            key = (path, r["Dispatch_Id"])
            d = per.setdefault(key, {"name": name})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        for (p, _), d in per.items():
            name = d.pop("name")
            for c, v in d.items():
                vals.setdefault(name, {}).setdefault(c, []).append(v)
            disp.setdefault(name, {}).setdefault(p, 0)
            disp[name][p] += 1
    counters = sorted({c for k in vals.values() for c in k})
    lines = ["| kernel | dispatches | " + " | ".join(counters) + " |", "|---|---|" + "---|" * len(counters)]
    for name in sorted(vals):
        n = max(disp[name].values())
        cells = [f"{np.mean(vals[name][c]):.6g}" if c in vals[name] else "" for c in counters]
        lines.append(f"| {name} | {n} | " + " | ".join(cells) + " |")
    return "\n".join(lines)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def setup(cfg, device):
    import torch

    import kara_inputs as ki
    from paper_2607_01237_amd import kara

    geom = ki.make_geometry(cfg)
    p = geom.params()
    L, nt = cfg["n_layers"], len(geom.trig)
    dt = ki.torch_dtype(cfg)
    nw = cfg.get("n_windows", 1)
    q = torch.empty((L, nt) + ((nw,) if nw > 1 else ()) + (ki.scoring_queries(cfg), cfg["n_q_heads"],
                                                            cfg["head_dim"]), dtype=dt, device=device)
    kp, vp = [], []
    for l in range(L):
        q[l] = ki.make_queries(geom, l, device)
        k_, v_ = ki.make_pools(geom, l, device)
        kp.append(k_)
        vp.append(v_)
        if (l + 1) % 10 == 0:
            log(f"layer {l + 1}/{L} generated")
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    meta = dict(bt=dev(geom.block_table), seq_lens=dev(geom.seq_lens), win_start=dev(geom.win_start),
                trig=dev(geom.trig))
    meta["bt0"] = meta["bt"].clone()
    meta["seq_lens0"] = meta["seq_lens"].clone()
    params = kara.make_params(p, geom.block_table.shape[0])
    return geom, p, params, q, kp, vp, meta


def moved_rows(kept, p, tails):
    """Rows that change place in one step, per (layer, trigger, head): kept
    rows not already at their destination plus the rows after the last
    window's compressible region (its buffer and the tail), which shift down.
    kept: [L, nt, n_windows, H, budget]; tails: rows after the last window."""
    budget, W, U = p["budget"], p["window"], p["buffer"]
    N = W - U
    nw = kept.shape[2]
    w = np.arange(nw)[:, None]
    j = np.arange(budget)
    in_place = (kept.transpose(0, 1, 3, 2, 4) + w * N == w * budget + j).sum(axis=(-2, -1))   # [L, nt, H]
    shift = nw * (N - budget)                                # positions the buffer/tail move by
    extra = (U + tails[None, :, None]) * (1 if shift > 0 else 0)
    return (nw * budget - in_place) + extra


def dest_rows(geom, p, n_windows):
    """(page, slot) of every row a compression of the triggered sequences
    may overwrite: per sequence the destination range [p0, p0 + n_dst) of
    compaction, n_dst = seq_len - p0 - n_windows * (N - budget)."""
    N, bs = p["window"] - p["buffer"], p["block_size"]
    pages, slots = [], []
    for s in geom.trig:
        p0 = int(geom.win_start[s])
        pos = np.arange(p0, int(geom.seq_lens[s]) - n_windows * (N - p["budget"]), dtype=np.int64)
        pages.append(geom.block_table[s, pos // bs].astype(np.int64))
        slots.append(pos % bs)
    return np.concatenate(pages), np.concatenate(slots)


def cpu_baseline(geom, p, q, kp, vp, budget_s, n_windows=1, threads=None):
    """The oracle, as it stands, on whole units of the workload.

    Units in layer order (sequence by sequence, window by window, every KV
    head, then the next layer) are copied to the host in batches and run through the oracle's scoring,
    selection, Token2Chunk, fill and K/V gather until `budget_s` seconds have
    passed.  With one window a unit's rows are its window and the tail after
    it; with several, the unit's own window.
    """
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    if threads is None:
        # one GPU's share of the host: the GPU machines allot 16 cores per GPU,
        # whatever the affinity mask shows
        threads = min(16, len(os.sched_getaffinity(0)))
    W, U = p["window"], p["buffer"]
    N = W - U
    scale = oracle.scale_of(p)

    def one(args):
        qa, ka, va = args
        a = oracle.round_scores(oracle.window_scores(qa, ka[:N], scale))
        _, kept = oracle.kept_set(a, p["budget"], p["chunk_budget"], p["max_chunk_len"])
        oracle.gather_rows(ka, kept, W, U)
        oracle.gather_rows(va, kept, W, U)
        return 1

    H = p["n_kv_heads"]
    # layer by layer until the time budget is spent
    all_units = [(l, t, w, h) for l in range(len(kp)) for t in range(len(geom.trig)) for w in range(n_windows)
                 for h in range(H)]
    done, busy = 0, 0.0
    # one BLAS thread per worker, so that `threads` is the number of cores used
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=1), ThreadPoolExecutor(threads) as ex:
        for i in range(0, len(all_units), threads):
            batch = all_units[i:i + threads]
            hq, hk, hv = host_units(geom, p, q, kp, vp, batch, n_windows)
            t0 = time.perf_counter()
            done += sum(ex.map(one, [(hq[u], hk[u], hv[u]) for u in batch]))
            busy += time.perf_counter() - t0
            if busy > budget_s:
                break
    return done, busy, threads


def host_units(geom, p, q, kp, vp, units, n_windows=1):
    """Host fp64 copies of the listed (layer, trigger, window, head) units'
    queries and K/V rows (window and tail with one window, else the window)."""
    import torch

    import kara_inputs as ki
    import oracle

    H, G, W = p["n_kv_heads"], p["n_q_heads"] // p["n_kv_heads"], p["window"]
    N, bs = W - p["buffer"], p["block_size"]
    out_q, out_k, out_v = {}, {}, {}
    for (l, t, w, h) in units:
        s = int(geom.trig[t])
        p0 = int(geom.win_start[s]) + w * N
        qw = q[l, t] if n_windows == 1 else q[l, t, w]
        rows = qw[:, h * G:(h + 1) * G, :].reshape(-1, q.shape[-1])
        out_q[(l, t, w, h)] = oracle.to_f64(ki.raw_numpy(rows), p["dtype"])
        pos = np.arange(p0, int(geom.seq_lens[s]) if n_windows == 1 else p0 + W)
        pg = torch.from_numpy(geom.block_table[s, pos // bs].astype(np.int64)).to(q.device)
        sl = torch.from_numpy((pos % bs).astype(np.int64)).to(q.device)
        out_k[(l, t, w, h)] = oracle.to_f64(ki.raw_numpy(kp[l][pg, h, sl, :]), p["dtype"])
        out_v[(l, t, w, h)] = oracle.to_f64(ki.raw_numpy(vp[l][pg, h, sl, :]), p["dtype"])
    return out_q, out_k, out_v


def run_soak(args):
    """The decode-loop soak: intervals of appends and decode steps, each
    ending in one timed compression event over every sequence and layer."""
    import torch

    import kara_inputs as ki
    from paper_2607_01237_amd import kara
    from paper_2607_01237_amd.soak import Soak

    kara.load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    cfg = ki.workload("soak")
    if args.intervals:
        cfg["n_intervals"] = args.intervals
    geom = ki.soak_geometry(cfg)
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg["seed"])
    sk = Soak(cfg, geom, device, gen)
    log(f"soak: {sk.n} sequences x {sk.L} layers, {cfg['n_intervals']} intervals, pool {geom.num_pages} pages "
        f"({geom.num_pages * sk.page_bytes() / 1e9:.1f} GB K+V), mem {torch.cuda.memory_allocated() / 2**30:.1f} GiB")
    sk.prompt()
    torch.cuda.synchronize()
    n_int = cfg["n_intervals"]
    n_dec = cfg["window"] // cfg["append_chunk"]
    p = sk.p
    N = p["window"] - p["buffer"]
    G = p["n_q_heads"] // p["n_kv_heads"]
    flops = 2.0 * sk.L * sk.n * p["n_kv_heads"] * G * p["window"] * N * p["head_dim"]
    ev = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    comp_ms, dec_ms, reclaimed, resident, logical = [], [], [], [], []
    score_ms = []
    t0 = time.perf_counter()
    for i in range(n_int):
        dec = []
        for _ in range(n_dec):
            sk.append(cfg["append_chunk"])
            e = ev()
            sk.decode(e)
            dec.append(e)
        if i >= n_int - 3:
            # the scoring kernel alone on this event's inputs (reads only)
            sk.q.normal_(generator=gen)
            sk.win_start.copy_(torch.from_numpy(sk.p0))
            e = ev()
            e[0].record()
            kara.score_window(sk.params, sk.seqs, sk.q, sk.kp, sk.bt, sk.lens, sk.win_start, sk.scores, sk.status,
                              sk.ws)
            e[1].record()
            torch.cuda.synchronize()
            score_ms.append(e[0].elapsed_time(e[1]))
        ce = ev()
        sk.compress(ce)
        got = sk.settle()
        comp_ms.append(ce[0].elapsed_time(ce[1]))
        dec_ms.append([a.elapsed_time(b) for a, b in dec])
        reclaimed.append(got)
        mapped = int((sk.pool.table >= 0).sum())
        resident.append(mapped)
        logical.append(cfg["prefix"][0] + (i + 1) * cfg["window"])
        log(f"event {i + 1}/{n_int}: compress {comp_ms[-1]:.2f} ms, decode {np.mean(dec_ms[-1]):.2f} ms/step, "
            f"reclaimed {got} pages, resident {mapped * sk.page_bytes() / 1e9:.1f} GB, "
            f"{time.perf_counter() - t0:.0f} s")
    timed = comp_ms[args.warmup:] if len(comp_ms) > args.warmup else comp_ms
    ms = float(np.mean(timed))
    win_tokens = sk.n * sk.W
    tok_bytes = sk.page_bytes() // sk.bs
    ach = flops / (np.mean(score_ms) * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if p["dtype"] == "bf16" else PEAK_F32_TFLOPS
    result = {
        "metric": "window tokens compressed/s (score+select+compact); % MFMA peak / % HBM GB/s",
        "value": win_tokens / (ms * 1e-3),
        "unit": "window tokens/s",
        "n_gpus": 1,
        "steps": len(timed),
        "warmup": len(comp_ms) - len(timed),
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": p["dtype"],
        "data": "synthetic (fresh seeded N(0,1) Q/K/V every interval; no model weights or datasets)",
        "config": {
            "workload": "soak", "sequences": sk.n, "layers": sk.L, "q_heads": p["n_q_heads"],
            "kv_heads": p["n_kv_heads"], "head_dim": p["head_dim"], "window": p["window"], "budget": p["budget"],
            "prompt": cfg["prefix"][0], "intervals": n_int, "append_chunk": cfg["append_chunk"],
            "decode_steps_per_interval": n_dec, "pages": geom.num_pages,
        },
        "roofline": {
            "kernel": scoring_kernel_name(p),
            "bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak, "traffic": None,
            "flop_per_launch": flops, "avg_launch_ms": float(np.mean(score_ms)),
        },
        "soak": {
            "compress_ms_per_event": comp_ms,
            "decode_ms_per_step_mean_per_event": [float(np.mean(x)) for x in dec_ms],
            "pages_reclaimed_per_event": reclaimed,
            "pages_reclaimed_total": int(sum(reclaimed)),
            "logical_tokens_per_sequence": logical,
            "resident_GB_per_event": [r * sk.page_bytes() / 1e9 for r in resident],
            "uncompressed_GB_at_end": sk.n * logical[-1] * tok_bytes / 1e9,
            "decode_ms_per_step_last_interval": float(np.mean(dec_ms[-1])),
        },
    }
    print(json.dumps(result), flush=True)


def run_recompute(args):
    """A compression event with its query recomputation (App. C.2): the
    window recompute pass over every layer (query projection, rotary
    embedding, causal attention over the cached prefix, feed-forward) writes
    the scoring queries, then kara_compress_window compresses every window
    with them.  Synthetic weights of the named shape.  Reports window tokens
    per second of the whole event, the recompute's share, and the roofline of
    the attention kernel (timed one layer per launch through
    kara_recompute_attention, HIP events on the launch stream)."""
    import torch

    import kara_inputs as ki
    from paper_2607_01237_amd import kara

    kara.load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    cfg = ki.workload("recompute")
    geom, p, params, q_unused, kp, vp, meta = setup(cfg, device)
    del q_unused
    L, nt, H = cfg["n_layers"], len(geom.trig), p["n_kv_heads"]
    W, N, d, Hq = p["window"], p["window"] - p["buffer"], p["head_dim"], p["n_q_heads"]
    D, F = cfg["hidden"], cfg["ffn"]
    G = Hq // H
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg["seed"] + 1)

    def w(shape, fan_in):
        return (torch.randn(shape, generator=gen, device=device) / fan_in ** 0.5).to(torch.bfloat16)

    wts = [dict(w_q=w((D, Hq * d), D), w_o=w((Hq * d, D), Hq * d), w_gate=w((D, F), D), w_up=w((D, F), D),
                w_down=w((F, D), F), g_attn=torch.ones(D, dtype=torch.bfloat16, device=device),
                g_ffn=torch.ones(D, dtype=torch.bfloat16, device=device)) for _ in range(L)]
    model = kara.make_model(D, F, cfg["rope_theta"], cfg["rms_eps"])
    h0 = torch.randn((nt, W, D), generator=gen, device=device)
    h1 = torch.empty_like(h0)
    q = torch.empty((L, nt, W, Hq, d), dtype=torch.bfloat16, device=device)
    rope_pos0 = meta["win_start"].clone()
    rws = torch.empty(kara.recompute_workspace_size(params, model, nt), dtype=torch.uint8, device=device)
    cws = torch.empty(kara.workspace_size(params, nt, L), dtype=torch.uint8, device=device)
    status = torch.empty(nt, dtype=torch.int32, device=device)
    rstatus = torch.empty(nt, dtype=torch.int32, device=device)
    freed = torch.empty((nt, p["max_blocks_per_seq"]), dtype=torch.int32, device=device)
    n_freed = torch.empty(nt, dtype=torch.int32, device=device)
    stream = torch.cuda.current_stream()
    log(f"recompute: {nt} sequences x {L} layers, D={D} F={F}, mem {torch.cuda.memory_allocated() / 2**30:.1f} GiB")

    def restore():
        meta["bt"].copy_(meta["bt0"], non_blocking=True)
        meta["seq_lens"].copy_(meta["seq_lens0"], non_blocking=True)

    def event(evs=None):
        restore()
        if evs:
            evs[0].record(stream)
        kara.recompute_queries(params, model, meta["trig"], wts, h0, h1, kp, vp, meta["bt"], meta["seq_lens"],
                               meta["win_start"], rope_pos0, q, rstatus, rws, stream=stream)
        if evs:
            evs[1].record(stream)
        kara.compress_window(params, meta["trig"], q, kp, vp, meta["bt"], meta["seq_lens"], meta["win_start"], True,
                             status, cws, freed=freed, n_freed=n_freed, stream=stream)
        if evs:
            evs[2].record(stream)

    for _ in range(args.warmup):
        event()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        event(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert (rstatus.cpu().numpy() == 0).all() and (status.cpu().numpy() == 0).all()
    rec_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in evs]))
    comp_ms = float(np.mean([b.elapsed_time(c) for _, b, c in evs]))
    ms = wall * 1e3 / args.steps

    # the attention kernel alone, one layer per launch
    restore()
    att_out = torch.empty((nt, W, Hq, d), dtype=torch.bfloat16, device=device)
    att_ms = []
    for rep in range(2):
        for l in range(L):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record(stream)
            kara.recompute_attention(params, meta["trig"], q[l], kp[l], vp[l], meta["bt"], meta["seq_lens"],
                                     meta["win_start"], att_out, rstatus, stream=stream)
            e[1].record(stream)
            torch.cuda.synchronize()
            if rep:
                att_ms.append(e[0].elapsed_time(e[1]))
    att_ms = float(np.mean(att_ms))
    p0 = geom.win_start[geom.trig].astype(np.float64)
    # QK^T and PV over the causal extent: query w sees p0 + w + 1 keys
    att_flops = float(sum(4.0 * G * H * d * (W * (p0_ + 1) + W * (W - 1) / 2) for p0_ in p0))
    att_ach = att_flops / (att_ms * 1e-3) / 1e12
    gemm_flops = 2.0 * nt * W * (2 * D * Hq * d + 3 * D * F) * L
    win_tokens = nt * W
    result = {
        "metric": "window tokens compressed/s, compression event with query recomputation",
        "value": win_tokens / (ms * 1e-3),
        "unit": "window tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) hidden states, K/V and weights of the named shape; no checkpoint)",
        "config": {"workload": "recompute", "sequences": nt, "layers": L, "q_heads": Hq, "kv_heads": H,
                   "head_dim": d, "hidden": D, "ffn": F, "window": W, "budget": p["budget"],
                   "context_tokens_mean": float(geom.seq_lens[geom.trig].mean())},
        "roofline": {"kernel": "attn_kernel (recompute causal attention)", "bound": "mfma", "achieved": att_ach,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": att_ach / PEAK_BF16_TFLOPS,
                     "traffic": None, "flop_per_launch": att_flops, "avg_launch_ms": att_ms},
        "recompute": {"recompute_ms": rec_ms, "compress_ms": comp_ms, "attention_ms_total": att_ms * L,
                      "attention_tflop_total": att_flops * L / 1e12, "gemm_tflop_total": gemm_flops / 1e12,
                      "rest_ms": rec_ms - att_ms * L,
                      "gemm_and_rest_tflops": gemm_flops / ((rec_ms - att_ms * L) * 1e-3) / 1e12},
    }
    print(json.dumps(result), flush=True)


def run_regions(args):
    """Survivors per region of the original sequence under Kara's windows and
    under the threshold-triggered whole-cache top-k (the analogue of the
    paper's Fig. 2), at the serving settings of App. B.1: windows of 768
    tokens with a 32-token buffer keeping 257, against compressing the whole
    cache to 1025 tokens whenever it reaches 1280 (32 observation tokens).
    4 sequences x 4 layers of an 8B shape, 8192 generated tokens each."""
    import torch

    from paper_2607_01237_amd import kara, regions

    kara.load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    shape = dict(n_layers=4, n_q_heads=32, n_kv_heads=8, head_dim=128)
    geos = {
        "kara": dict(window=768, buffer=32, budget=225, chunk_budget=16, max_chunk_len=8, block_size=16),
        "threshold": dict(window=1280, buffer=32, budget=993, chunk_budget=0, max_chunk_len=8, block_size=16,
                          score_queries=32),
    }
    n_tok, region = 8192, 512
    t0 = time.perf_counter()
    out = regions.run(shape, geos, n_seqs=4, n_tokens=n_tok, chunk=128, region=region, device=device, seed=12,
                      check_every=4)
    wall = time.perf_counter() - t0
    rows = {pol: [dict(tokens=g, survivors=[round(x, 1) for x in row]) for g, row in v["events"]]
            for pol, v in out.items()}
    result = {
        "metric": "cached tokens per 512-token region of the original sequence after repeated compression",
        "value": out["kara"]["final"][0], "unit": "tokens of region 0 still cached (Kara)",
        "n_gpus": 1, "steps": len(rows["kara"]), "warmup": 0, "ms_per_step": wall * 1e3 / max(1, len(rows["kara"])),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) K/V and queries; V rows carry their token index)",
        "config": {"workload": "regions", "sequences": 4, "layers": 4, "q_heads": 32, "kv_heads": 8, "head_dim": 128,
                   "generated_tokens": n_tok, "region": region, **{f"{p}_{k}": v for p, g in geos.items()
                                                                   for k, v in g.items()}},
        "regions": {pol: {"events": len(rows[pol]), "final": [round(x, 1) for x in out[pol]["final"]],
                          "cache_len": out[pol]["cache_len"], "per_event": rows[pol]} for pol in out},
    }
    print(json.dumps(result), flush=True)


def run_serve(args):
    """The serving analogue of the paper's throughput runs (App. B.1): a batch
    of requests served to completion by the periodic policy on a memory-bound
    pool, then by the same loop with compression switched off (the
    uncompressed baseline), same requests and pool.  Reports generated tokens
    per second of each, mean concurrency and preemptions."""
    import torch

    import kara_inputs as ki
    from paper_2607_01237_amd import kara
    from paper_2607_01237_amd.serve import Serve

    kara.load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    over = {"n_requests": args.requests} if args.requests else {}
    shape, sc, prompts, gens, order = ki.serve_setup(**over)
    runs = {}
    for comp in (1, 0):
        srv = Serve(shape, dict(sc, compress=comp), device, ki.SERVE["seed"], page_order=order)
        for p_, g_ in zip(prompts, gens):
            srv.submit(int(p_), int(g_))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        steps, chunk = 0, 500
        while True:
            done = srv.run(chunk)
            steps += done
            st = srv.sched.stats()
            log(f"serve compress={comp}: {steps} steps, finished {st['finished']}/{len(prompts)}, running "
                f"{st['running']}, events {st['events']}, preemptions {st['preemptions']}, "
                f"{time.perf_counter() - t0:.0f} s")
            if st["finished"] == len(prompts) or steps >= 50000:
                break
        srv.verify()
        wall = time.perf_counter() - t0
        st = srv.sched.stats()
        hist = np.array(srv.history)
        runs[comp] = dict(steps=steps, wall_s=wall, tokens_decoded=st["tokens_decoded"],
                          tokens_per_s=st["tokens_decoded"] / wall, ms_per_step=wall * 1e3 / steps,
                          mean_running=float(hist[:, 0].mean()), peak_running=st["peak_running"],
                          preemptions=st["preemptions"], tokens_prefilled=st["tokens_prefilled"],
                          events=st["events"], sequences_compressed=st["compressed"],
                          pages_reclaimed=st["pages_reclaimed"], finished=st["finished"])
        del srv
        torch.cuda.empty_cache()
    on, off = runs[1], runs[0]
    page_gb = 2 * shape["n_layers"] * shape["n_kv_heads"] * sc["block_size"] * shape["head_dim"] * 2 / 1e9
    result = {
        "metric": "generated tokens/s, serving loop under the periodic compression policy (synthetic tokens)",
        "value": on["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": on["steps"],
        "warmup": 0,
        "ms_per_step": on["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": shape["dtype"],
        "data": "synthetic (seeded N(0,1) K/V and queries; no model weights, datasets or sampling)",
        "config": {
            "workload": "serve", "requests": len(prompts), "layers": shape["n_layers"],
            "q_heads": shape["n_q_heads"], "kv_heads": shape["n_kv_heads"], "head_dim": shape["head_dim"],
            "prompt_range": list(ki.SERVE["prompt"]), "gen_range": list(ki.SERVE["gen"]),
            "pool_pages": sc["num_pages"], "pool_GB": sc["num_pages"] * page_gb, **{k: sc[k] for k in (
                "block_size", "window", "buffer", "budget", "period", "max_per_event", "max_running")},
        },
        "serve": {"kara": on, "uncompressed": off, "speedup": on["tokens_per_s"] / off["tokens_per_s"]},
    }
    print(json.dumps(result), flush=True)


def main():
    args = parse()
    if args.summarize_counters:
        print(summarize_counters(args.summarize_counters))
        return
    if args.summarize_pmc:
        print(summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.workload,
                            args.copy_calibration_gib or 1.0))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; --gpus must be 1 (the step needs no "
                                   "communication: sequences or KV heads would be split across GPUs, not built here)"}))
        sys.exit(2)
    if args.workload == "soak":
        run_soak(args)
        return
    if args.workload == "serve":
        run_serve(args)
        return
    if args.workload == "recompute":
        run_recompute(args)
        return
    if args.workload == "regions":
        run_regions(args)
        return
    import torch

    import kara_inputs as ki
    from paper_2607_01237_amd import kara

    kara.load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    cfg = ki.workload(args.workload)
    t_setup = time.perf_counter()
    geom, p, params, q, kp, vp, meta = setup(cfg, device)
    torch.cuda.synchronize()
    L, nt, H = cfg["n_layers"], len(geom.trig), p["n_kv_heads"]
    W, U, N = p["window"], p["buffer"], p["window"] - p["buffer"]
    G = p["n_q_heads"] // H
    nw = cfg.get("n_windows", 1)
    units = L * nt * H
    log(f"setup {time.perf_counter() - t_setup:.1f}s: {args.workload} units={units} pages={geom.num_pages} "
        f"mem={torch.cuda.memory_allocated() / 2**30:.1f} GiB")

    stream = torch.cuda.current_stream()
    ws_bytes = kara.workspace_size(params, nt * nw, L)
    status = torch.empty(nt, dtype=torch.int32, device=device)
    freed = torch.empty((nt, p["max_blocks_per_seq"]), dtype=torch.int32, device=device)
    n_freed = torch.empty(nt, dtype=torch.int32, device=device)
    # [L, trigger, window, head, ...]: with one window the same memory as [L, trigger, head, ...]
    scores = torch.empty((L, nt * nw, H, N), dtype=torch.float32, device=device)
    disc = torch.empty((L, nt * nw, H, p["budget"] - p["chunk_budget"]), dtype=torch.int32, device=device)
    kept = torch.empty((L, nt * nw, H, p["budget"]), dtype=torch.int32, device=device)

    def restore():
        meta["bt"].copy_(meta["bt0"], non_blocking=True)
        meta["seq_lens"].copy_(meta["seq_lens0"], non_blocking=True)

    # Device backup of the rows compaction overwrites, taken before any step:
    # every step below starts from the same pools and tables (restored
    # outside its events), so every step compresses the same input.
    pg, sl = (torch.from_numpy(a).to(device) for a in dest_rows(geom, p, nw))
    backup = [(k[pg, :, sl, :], v[pg, :, sl, :]) for k, v in zip(kp, vp)]
    log(f"pool backup: {len(pg)} rows per layer, {sum(b.numel() * b.element_size() for kv in backup for b in kv) / 1e9:.2f} GB")

    def restore_pools():
        for (bk, bv), k, v in zip(backup, kp, vp):
            k[pg, :, sl, :] = bk
            v[pg, :, sl, :] = bv

    def compress():
        if nw == 1:
            kara.compress_window(params, meta["trig"], q, kp, vp, meta["bt"], meta["seq_lens"], meta["win_start"],
                                 True, status, ws, kept=kept, freed=freed, n_freed=n_freed, stream=stream)
        else:
            kara.compress_prefill(params, meta["trig"], nw, q, kp, vp, meta["bt"], meta["seq_lens"],
                                  meta["win_start"], True, status, ws, kept=kept, freed=freed, n_freed=n_freed,
                                  stream=stream)


    # The staged pass times scoring and selection through the single-window
    # entry points.  Prefill's windows are scored as separate sequences then:
    # window w of sequence s becomes a sequence of its own that shares s's
    # block-table row and length and starts its window w*(W-U) later, so the
    # scoring launch covers the same (layer, trigger, window, head) units in
    # the same order over the same queries.
    if nw == 1:
        sv = dict(params=params, trig=meta["trig"], bt=meta["bt"], seq_lens=meta["seq_lens"],
                  win_start=meta["win_start"], status=status)
    else:
        tr = geom.trig.astype(np.int64)
        rep = lambda a: torch.from_numpy(np.ascontiguousarray(np.repeat(a, nw, axis=0))).to(device)
        ws_v = np.repeat(geom.win_start[tr], nw) + np.tile(np.arange(nw, dtype=np.int32) * N, nt)
        sv = dict(params=kara.make_params(p, nt * nw), trig=torch.arange(nt * nw, dtype=torch.int32, device=device),
                  bt=rep(geom.block_table[tr]), seq_lens=rep(geom.seq_lens[tr]),
                  win_start=torch.from_numpy(ws_v.astype(np.int32)).to(device),
                  status=torch.empty(nt * nw, dtype=torch.int32, device=device))
    q_v = q.view((L, nt * nw) + tuple(q.shape[-3:]))
    ws = torch.empty(max(ws_bytes, kara.workspace_size(sv["params"], nt * nw, L)), dtype=torch.uint8, device=device)

    if args.copy_calibration_gib > 0:
        n = int(args.copy_calibration_gib * 2**30) // 2
        src = torch.ones(n, dtype=torch.bfloat16, device=device)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    es = 2 if p["dtype"] == "bf16" else 4
    row_bytes = p["head_dim"] * es
    tails = (geom.seq_lens[geom.trig] - geom.win_start[geom.trig] - (nw - 1) * N - W).astype(np.int64)

    def moved_gb():
        """Compaction's algorithmic bytes of the step just run, each way."""
        rows = moved_rows(kept.cpu().numpy().reshape(L, nt, nw, H, p["budget"]), p, tails).sum()
        return float(rows) * row_bytes * 2 / 1e9

    for _ in range(args.warmup):
        restore()
        restore_pools()
        compress()
    torch.cuda.synchronize()
    log("warmup done")

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    step_gb = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        restore()
        restore_pools()
        ev[i][0].record(stream)
        compress()
        ev[i][1].record(stream)
        torch.cuda.synchronize()
        step_gb.append(moved_gb())
    wall = time.perf_counter() - t0
    step_ms = [a.elapsed_time(b) for a, b in ev]
    st = status.cpu().numpy()
    assert (st == 0).all(), f"unexpected status {st}"
    assert len(set(round(x, 6) for x in step_gb)) == 1, f"steps moved different bytes: {step_gb}"
    log(f"timed {args.steps} steps: events mean {np.mean(step_ms):.3f} ms, median {np.median(step_ms):.3f} ms; "
        f"compaction moved {step_gb[0]:.4f} GB each way in every step; wall incl. restores "
        f"{wall * 1e3 / args.steps:.3f} ms/step")

    # staged pass: the same path through the per-stage entry points, with HIP
    # events between stages on the launch stream.  With several windows the
    # compaction and commit have no entry points of their own: the whole
    # prefill call is timed after the staged scoring and selection, and
    # compact+commit is its time less theirs.
    stages = ["score", "select_t2c", "compact", "commit"]
    times = {s: [] for s in stages}
    moved = []
    n_stage = max(3, args.steps)
    for i in range(n_stage + 1):
        restore()
        restore_pools()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        e[0].record(stream)
        kara.score_window(sv["params"], sv["trig"], q_v, kp, sv["bt"], sv["seq_lens"], sv["win_start"], scores,
                          sv["status"], ws, stream=stream)
        e[1].record(stream)
        # selection as the fused step runs it: discrete set and Token2Chunk in one launch
        kara.select_kept(params, scores, disc, kept, stream=stream)
        e[2].record(stream)
        if nw == 1:
            kara.compact_pages(params, meta["trig"], kept, kp, vp, meta["bt"], meta["seq_lens"], meta["win_start"],
                               status, stream=stream)
            e[3].record(stream)
            kara.commit_tables(params, meta["trig"], meta["bt"], meta["seq_lens"], meta["win_start"], freed,
                               n_freed, status, stream=stream)
        else:
            compress()
            e[3].record(stream)
        e[4].record(stream)
        torch.cuda.synchronize()
        if i == 0:
            continue   # first pass warms the staged entry points
        for k, s in enumerate(stages):
            times[s].append(e[k].elapsed_time(e[k + 1]))
        # rows this pass moved (the same input every pass)
        moved.append(float(moved_rows(kept.cpu().numpy().reshape(L, nt, nw, H, p["budget"]), p, tails).sum()))
    avg = {s: float(np.mean(v)) for s, v in times.items()}
    if nw > 1:
        avg["compact"] = max(0.0, avg["compact"] - avg["score"] - avg["select_t2c"])
    st_v = sv["status"].cpu().numpy()
    assert (st_v == 0).all(), f"unexpected staged status {st_v}"
    log("staged ms: " + ", ".join(f"{s}={avg[s]:.3f}" for s in stages))

    # algorithmic work
    Wq = ki.scoring_queries(cfg)
    flops = 2.0 * units * nw * G * Wq * N * p["head_dim"]
    peak = PEAK_BF16_TFLOPS if p["dtype"] == "bf16" else PEAK_F32_TFLOPS
    ach = flops / (avg["score"] * 1e-3) / 1e12
    # read + write, K and V, averaged over the passes timed
    compact_bytes = float(np.mean(moved)) * row_bytes * 2 * 2
    log("compaction algorithmic GB per staged pass (read = write): "
        + ", ".join(f"{m * row_bytes * 2 / 1e9:.4f}" for m in moved))
    select_bytes = float(units * nw) * (N * 4 + p["budget"] * 4 + (p["budget"] - p["chunk_budget"]) * 4 * 2)
    sc_ms = avg["select_t2c"] + avg["compact"]
    sc_gbs = (compact_bytes + select_bytes) / (sc_ms * 1e-3) / 1e9

    ms = float(np.mean(step_ms))
    win_tokens = nt * nw * W
    traffic = load_traffic(args.workload)
    result = {
        "metric": "window tokens compressed/s (score+select+compact); % MFMA peak / % HBM GB/s",
        "value": win_tokens / (ms * 1e-3),
        "unit": "window tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_events_median": float(np.median(step_ms)),
        "ms_per_step_wall_incl_restores": wall * 1e3 / args.steps,
        "compaction_gb_each_way_per_step": step_gb,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": p["dtype"],
        "data": "synthetic (seeded N(0,1) Q/K/V of the named shape; no model weights or datasets)",
        "config": {
            "workload": args.workload, "sequences": int(nt), "layers": L, "q_heads": p["n_q_heads"],
            "kv_heads": H, "head_dim": p["head_dim"], "window": W, "buffer": U, "budget": p["budget"],
            "chunk_budget": p["chunk_budget"], "max_chunk_len": p["max_chunk_len"], "block_size": p["block_size"],
            "pages": int(geom.num_pages), "units_per_step": int(units * nw), "windows_per_sequence": nw,
        },
        "roofline": {
            "kernel": scoring_kernel_name(p),
            "bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak,
            "traffic": traffic["score"], "flop_per_launch": flops, "avg_launch_ms": avg["score"],
        },
        "roofline_select_compact": {
            "bound": "hbm", "achieved": sc_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": sc_gbs / PEAK_HBM_GBS,
            "bytes_per_step": compact_bytes + select_bytes, "avg_ms": sc_ms, "traffic": traffic["select_compact"],
            # several windows: compaction has no entry point of its own, and its
            # time is the fused call's less the staged scoring and selection,
            # which overstates the stage's bandwidth; a kernel trace gives it
            "compact_ms_derived": nw > 1,
        },
        "stage_ms": avg,
        "layer_window_tokens_per_s": win_tokens * L / (ms * 1e-3),
    }

    if not args.no_cpu_baseline:
        done, dt_cpu, threads = cpu_baseline(geom, p, q, kp, vp, args.cpu_seconds, nw)
        # units per window token: every window token is compressed in L*H units
        rate = done / dt_cpu * W / (L * H)
        # the same oracle on one thread, over a quarter of the time
        done1, dt1, _ = cpu_baseline(geom, p, q, kp, vp, args.cpu_seconds / 4, nw, threads=1)
        result["cpu_baseline"] = {
            "value": rate, "unit": "window tokens/s", "cores": threads, "kind": "oracle",
            "host_cpus_visible": len(os.sched_getaffinity(0)), "host_cpu_count": os.cpu_count(),
            "cores_note": "16 worker threads, one BLAS thread each: the host share one GPU is allotted",
            "sample": f"{done} whole (layer, sequence, window, KV head) units of this workload, in layer order: fp64 scoring, "
                      f"selection, Token2Chunk, fill and K/V gather in {dt_cpu:.1f} s of oracle time; one window "
                      f"token is compressed in layers*kv_heads units, so rate = units/s * W/(layers*kv_heads)",
            "value_one_core": done1 / dt1 * W / (L * H),
            "sample_one_core": f"{done1} units on one thread in {dt1:.1f} s",
        }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
