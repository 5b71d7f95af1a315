"""Survivors per region under Kara's windowed policy and under the
threshold-triggered whole-cache top-k (Sec. 3 Eq. (2)-(3) against Sec. 4):
after every event the device cache holds exactly the original tokens the
host bookkeeping says it does (token indices carried in V), and the two
policies show their structure -- a region loses tokens once under Kara's
windows, again and again under whole-cache re-selection."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

SHAPE = dict(n_layers=2, n_q_heads=8, n_kv_heads=2, head_dim=64)
GEOS = {
    "kara": dict(window=192, buffer=16, budget=48, chunk_budget=8, max_chunk_len=8, block_size=16),
    "threshold": dict(window=320, buffer=16, budget=240, chunk_budget=0, max_chunk_len=8, block_size=16,
                      score_queries=16),
}


def test_survivors_per_region():
    from paper_2607_01237_amd import regions
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("\n[case] regions: 2 sequences, 2000 tokens, both policies", flush=True)
    region = 64
    out = regions.run(SHAPE, GEOS, n_seqs=2, n_tokens=2000, chunk=32, region=region, device=torch.device("cuda:0"),
                      seed=11, check_every=1)
    k, t = out["kara"], out["threshold"]
    for pol in (k, t):
        assert abs(sum(pol["final"]) - pol["cache_len"]) < 1e-9
        for _, row in pol["events"]:
            assert max(row) <= region
    # Kara (U = 16): the windows slide by W - U = 176 tokens; once a region
    # lies wholly before the next window's start its count never changes
    ev = k["events"]
    assert len(ev) >= 8
    for i in range(1, len(ev)):
        settled = (i * (192 - 16)) // region - 1          # regions wholly before window i's compressible start
        for r in range(max(0, settled)):
            assert ev[i][1][r] == ev[i - 1][1][r], (i, r)
    # threshold: whole-cache re-selection keeps thinning the first region
    tv = [row[0] for _, row in t["events"]]
    assert all(b <= a for a, b in zip(tv, tv[1:]))
    assert tv[-1] < 0.5 * tv[0]
    assert k["events"][-1][1][0] > 2 * t["events"][-1][1][0]
    print(f"[case] ok: kara {len(ev)} events, region 0 keeps {ev[-1][1][0]:.1f}; threshold {len(tv)} events, "
          f"region 0 keeps {tv[-1]:.1f}", flush=True)
