"""CPU oracle for Kara's KV compression step -- test infrastructure only.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this package; the product path never imports it.  See kara_oracle.py.
"""
from .kara_oracle import *  # noqa: F401,F403
from .kara_oracle import (  # noqa: F401
    SEQ_OK, SEQ_BAD_WINDOW, SEQ_BAD_PAGE, SEQ_DUP_TRIGGER, SEQ_BAD_INDEX, SEQ_DUP_PAGE,
    bf16_bits_to_f64, to_f64, window_scores, round_scores, rank_order, discrete_topk,
    chunk_candidates, token2chunk, fill_positions, kept_set, compaction_map, gather_rows,
    released_blocks, read_rows, write_rows, validate, scoring_queries, unit_queries, unit_keys, scale_of,
    score_units, compress, compress_prefill,
)
