"""MI355X (gfx950) implementation of Kara's sliding-window KV-cache
compression step: window scoring, budgeted top-k, Token2Chunk and in-place
paged compaction, behind the C ABI of include/kara.h (libkara.so)."""
from . import kara  # noqa: F401
from .kara import KaraError, KaraParams, make_params  # noqa: F401
