"""GPU parity of the fused step (kara_compress_window) against the CPU oracle,
on every workload shape at sizes the oracle finishes in seconds, plus the
edge cases of the method (ragged compressible length, buffer, full budget,
alpha = 0, gamma = 3, unaligned windows, flagged sequences)."""
import sys

import numpy as np
import pytest

import kara_inputs as ki

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _run(cfg, **kw):
    import kara_check as kc
    _need_gpu()
    print(f"\n[case] {cfg['name']} {({k: cfg[k] for k in ('n_seqs', 'n_layers', 'window', 'buffer', 'budget')})}",
          flush=True)
    case = kc.setup(cfg, **kw)
    rep, gpu = kc.full_check(case)
    print(f"[case] ok {rep}", flush=True)
    return case, rep, gpu


def test_tiny_full():
    _run(ki.workload("tiny"))


def test_batch8_full():
    _, rep, _ = _run(ki.workload("batch8"))
    assert rep["units"] == 64


def test_qwen14b_shape_reduced():
    # the 64 x 40-layer batch at its real per-unit shape (W=2048, G=5), fewer units
    _run(ki.workload("qwen14b", n_seqs=2, n_layers=2, prefix=(4096, 6000)))


def test_qwen14b_buffer_ragged_tiles():
    # U=32: N=2016 is not a multiple of the 16-key tile; budget ceil(0.2*2016)=404
    _run(ki.workload("qwen14b", n_seqs=2, n_layers=1, buffer=32, budget=404, prefix=(100, 3000)))


def test_ragged_reduced():
    case, rep, gpu = _run(ki.workload("ragged", n_seqs=24, n_layers=2, prefix=(0, 1500)))
    assert len(case.geom.trig) < 24


def test_odd_geometry_and_flags():
    # N = 193 (ragged), d=64 bf16, block 7, unaligned starts, G=3; one
    # sequence triggered twice, one with a window past its end
    cfg = ki.workload("batch8", n_seqs=5, n_layers=2, n_q_heads=6, n_kv_heads=2, head_dim=64, window=200,
                      buffer=7, budget=39, chunk_budget=5, max_chunk_len=3, block_size=7, num_pages=600,
                      prefix=(0, 90), tail=(0, 20), key_mode="normal")
    g = ki.make_geometry(cfg)
    lens = g.seq_lens.copy()
    lens[4] = g.win_start[4] + 150          # window overruns the sequence
    _run(cfg, trig=[0, 1, 2, 3, 4, 2], seq_lens=lens)


@pytest.mark.parametrize("window,head_dim", [(40, 128), (150, 128), (330, 128), (150, 64), (1000, 64)])
def test_chunk_counts(window, head_dim):
    # 64-key chunks: one (N=40), odd counts whose last chunk is partial
    # (150 -> 3, 1000 -> 16 with d=64), and 330 -> 6 with a 10-key tail;
    # G*W not a multiple of the 512 rows of a workgroup
    budget = max(2, (window + 4) // 5)
    cfg = ki.workload("batch8", n_seqs=2, n_layers=1, window=window, budget=budget, chunk_budget=min(4, budget - 1),
                      max_chunk_len=4, head_dim=head_dim, prefix=(0, 70), tail=(0, 12), num_pages=256)
    _run(cfg)


def test_fp32_head128_mha():
    cfg = ki.workload("tiny", n_seqs=3, n_q_heads=2, n_kv_heads=2, head_dim=128, window=96, budget=20,
                      chunk_budget=6, max_chunk_len=5, num_pages=64, prefix=(3, 40), tail=(0, 9))
    _run(cfg)


@pytest.mark.parametrize("head_dim,window", [(64, 1024), (128, 512)])
def test_fp32_at_its_largest_window(head_dim, window):
    # fp32 windows hold at most 64K head-dim elements of keys: 1024 keys at
    # d = 64, 512 at d = 128 (two query heads per KV head)
    cfg = ki.workload("tiny", n_seqs=2, n_q_heads=4, n_kv_heads=2, head_dim=head_dim, window=window,
                      budget=window // 5, chunk_budget=8, max_chunk_len=6, num_pages=256, prefix=(3, 90), tail=(0, 9))
    _run(cfg)


def test_more_layers_than_one_launch_takes():
    # 66 layers: scoring and compaction each run as two launches (64 + 2
    # layers' pool pointers), the scores and kept rows laid out across both
    cfg = ki.workload("batch8", n_seqs=2, n_layers=66, n_q_heads=2, n_kv_heads=1, window=128, budget=26,
                      chunk_budget=4, max_chunk_len=4, prefix=(0, 40), tail=(0, 7), num_pages=64)
    _run(cfg)


@pytest.mark.parametrize("budget,alpha,gamma", [(1024, 16, 8), (205, 0, 8), (300, 64, 3), (1, 0, 3)])
def test_selection_extremes(budget, alpha, gamma):
    cfg = ki.workload("batch8", n_seqs=2, budget=budget, chunk_budget=alpha, max_chunk_len=gamma)
    _run(cfg)


def test_deterministic():
    import kara_check as kc
    _need_gpu()
    cfg = ki.workload("batch8", n_seqs=3)
    a = kc.run_compress(kc.setup(cfg))
    b = kc.run_compress(kc.setup(cfg))
    for k in ("scores", "discrete", "kept", "bt", "seq_lens", "freed", "n_freed", "status"):
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


def test_bf16_long_window():
    # N = 2500: 40 64-key chunks with a 4-key tail; G=2, one KV head
    cfg = ki.workload("batch8", n_seqs=2, n_layers=1, n_q_heads=2, n_kv_heads=1, window=2500, budget=500,
                      prefix=(0, 100), tail=(0, 5), num_pages=512, key_mode="normal")
    _run(cfg)


@pytest.mark.parametrize("window,buffer", [(4096, 0), (4128, 32)])
def test_maximum_compressible_window(window, buffer):
    # N = 4096, the largest compressible length the library takes: 64 chunks
    # of 64 keys in each scoring sweep, the 16-position selection instance
    # at its limit; with a buffer, the buffer queries score as well
    cfg = ki.workload("batch8", n_seqs=2, n_layers=1, n_q_heads=2, n_kv_heads=1, window=window, buffer=buffer,
                      budget=820, prefix=(0, 100), tail=(0, 5), num_pages=1024, key_mode="normal")
    _run(cfg)



@pytest.mark.parametrize("window", [600, 1000, 1300, 1536, 2048])
def test_single_sweep_instances(window):
    # bf16, d = 128: every instance of the single-sweep scoring kernel, by
    # key tiles per wave (16, 24, 32) and whole or ragged tiles: N = 600 and
    # 1000 (16, ragged), 1300 (24, ragged), 1536 (24, whole), 2048 (32, whole)
    cfg = ki.workload("batch8", n_seqs=2, n_layers=1, n_q_heads=4, n_kv_heads=1, window=window,
                      budget=window // 5, prefix=(0, 100), tail=(0, 9), num_pages=600, key_mode="normal")
    _run(cfg)


@pytest.mark.parametrize("pos,scale", [(700, 16.0), (300, 16.0), (40, 16.0), (700, -16.0)])
def test_outlier_keys(pos, scale):
    # One window key per (sequence, head) scaled by 16 (exact in bf16).
    # Positive: its logits lie far above the maximum of the row's first keys,
    # where the scoring kernel takes its reference, and it takes nearly all
    # the probability of the rows it agrees with.  Its fp16 weights overflow
    # in roughly a third of the rows of every row tile, so the row sums' selector
    # products meet infinities (0 * inf: whole row tiles of NaN sums) and the
    # overflow redo has to take NaN as overflow.  Negative: its probabilities
    # sit tens of binades below the row maxima.
    import kara_check as kc
    _need_gpu()
    cfg = ki.workload("batch8", n_seqs=2, n_layers=1, key_mode="normal")
    print(f"\n[case] outlier key at window position {pos}, scale {scale}", flush=True)
    case = kc.setup(cfg)
    bs = case.p["block_size"]
    for t, s_ in enumerate(case.geom.trig):
        j = int(case.geom.win_start[s_]) + pos
        page = int(case.geom.block_table[s_, j // bs])
        case.kp[0][page, :, j % bs, :] *= scale
    case.host = kc.snapshot(case)
    rep, gpu = kc.full_check(case)
    print(f"[case] ok {rep}", flush=True)
    if scale > 0:
        # the outlier takes nearly all the probability of the rows whose dot
        # product with it is positive, about half of the G*W rows
        w = gpu["scores"][0, :, :, pos]
        assert (w > 0.25 * case.p["n_q_heads"] // case.p["n_kv_heads"] * case.p["window"]).all()


def test_buffer_only_scoring():
    # the ablation without bidirectional attention: only the 64 buffer
    # queries score the 960 compressible keys (q holds those 64 positions)
    _run(ki.workload("buffer_only", n_seqs=3, n_layers=2, window=1024, budget=192, prefix=(0, 300)))


def test_threshold_topk_baseline():
    # Eq. (2)-(3): the whole cache (1280 tokens at the threshold) is the
    # window, its last 32 tokens score and are kept, plain top-k of 993
    case, rep, gpu = _run(ki.workload("threshold_topk", n_seqs=3, n_layers=2))
    assert (gpu["seq_lens"][case.geom.trig] == 1025).all()


def test_kvllm_serving_geometry():
    # the serving runs' geometry (App. B.1): 256-token blocks, a window of
    # three blocks with a 32-token buffer, 225 kept + 32 buffer = 257 retained
    _run(ki.workload("batch8", n_seqs=3, n_layers=2, block_size=256, window=768, buffer=32, budget=225,
                     prefix=(0, 600), tail=(0, 255), num_pages=40))


def test_wide_block_table():
    # a block-table row wider than compaction stages in LDS (8,192 words with
    # the kept rows): the instance that reads the kept indices and the table
    # from global memory for every tile
    _, rep, _ = _run(ki.workload("batch8", n_seqs=2, n_layers=2, max_blocks=8400))
