"""ctypes binding of libkara (include/kara.h): argument marshalling only.

Every function takes torch tensors that already live on the GPU and passes
their device pointers, plus the current HIP stream, to the C ABI of the same
name.  All computation happens in the library's HIP kernels; nothing here
falls back to the CPU.  A missing or unloadable library raises KaraError.
"""

from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
# the in-tree library; KARA_LIBRARY names another build of the same sources
# (the host-sanitized one the CPU tests load)
LIB_PATH = os.environ.get("KARA_LIBRARY") or os.path.join(_PKG, "libkara.so")
HEADERS = [os.path.join(os.path.dirname(_PKG), "include", h)
           for h in ("kara.h", "kara_harness.h", "kara_sched.h", "kara_recompute.h")]

BF16, F32 = 0, 1
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP, ERR_SCHED_MISMATCH, ERR_SCHED_NOMEM = 0, -1, -2, -3, -4, -5, -6
ERR_SCRATCH_LIMIT = -7
NOALLOC_SCRATCH_BYTES = 64 << 20      # KARA_NOALLOC_SCRATCH_BYTES
SEQ_OK, SEQ_BAD_WINDOW, SEQ_BAD_PAGE, SEQ_DUP_TRIGGER, SEQ_BAD_INDEX, SEQ_BAD_KEPT, SEQ_DUP_PAGE = \
    0, 1, 2, 4, 8, 16, 32
MAX_COMPRESSIBLE = 4096
REQ_WAITING, REQ_RUNNING, REQ_FINISHED = 0, 1, 2


class KaraError(RuntimeError):
    def __init__(self, fn, code, msg):
        super().__init__(f"{fn}: {msg} ({code})")
        self.code = code


class KaraParams(ctypes.Structure):
    _fields_ = [
        ("window", ctypes.c_int32),
        ("buffer", ctypes.c_int32),
        ("budget", ctypes.c_int32),
        ("chunk_budget", ctypes.c_int32),
        ("max_chunk_len", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_pages", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("n_seqs", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("score_queries", ctypes.c_int32),
    ]


class KaraModel(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w_q", "w_o", "w_gate", "w_up", "w_down", "g_attn", "g_ffn")]


class SchedConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_slots", "num_pages", "block_size", "max_blocks_per_seq", "window", "buffer", "budget", "period",
        "max_per_event", "max_running", "reserve_pages", "compress", "protect_prompt")]


_P32 = ctypes.POINTER(ctypes.c_int32)
_P64 = ctypes.POINTER(ctypes.c_int64)


class SchedStep(ctypes.Structure):
    _fields_ = [("n_preempted", ctypes.c_int32), ("preempted", _P32), ("n_decode", ctypes.c_int32),
                ("decode", _P32), ("n_admitted", ctypes.c_int32), ("admitted", _P32), ("prefill_len", _P32),
                ("admitted_id", _P64), ("tables_changed", ctypes.c_int32)]


class SchedEvent(ctypes.Structure):
    _fields_ = [("n_trig", ctypes.c_int32), ("trig", _P32), ("win_start", _P32)]


class SchedStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("steps", "events", "compressed", "pages_reclaimed", "preemptions",
                                              "tokens_decoded", "tokens_prefilled")] + \
               [(n, ctypes.c_int32) for n in ("running", "waiting", "finished", "free_pages", "peak_running",
                                              "pages_in_use")]


class SchedRequest(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("state", "slot", "len", "win_start", "generated", "compressions",
                                              "preemptions")]


def make_params(p: dict, n_seqs: int) -> KaraParams:
    """KaraParams from a geometry dict (the field names of kara_params_t)."""
    dt = p["dtype"]
    dt = BF16 if dt in ("bf16", BF16) else F32 if dt in ("f32", F32) else dt
    return KaraParams(p["window"], p["buffer"], p["budget"], p["chunk_budget"], p["max_chunk_len"],
                      p["head_dim"], p["n_q_heads"], p["n_kv_heads"], p["block_size"], p["num_pages"],
                      p["max_blocks_per_seq"], n_seqs, dt, float(p.get("scale", 0.0) or 0.0),
                      int(p.get("score_queries", 0) or 0))


_VP = ctypes.c_void_p
_I32 = ctypes.c_int32
_PP = ctypes.POINTER(ctypes.c_void_p)
_PAR = ctypes.POINTER(KaraParams)

_SIGS = {
    "kara_status_string": (ctypes.c_char_p, [_I32]),
    "kara_abi_version": (_I32, []),
    "kara_source_hash": (ctypes.c_char_p, []),
    "kara_last_hip_error": (ctypes.c_char_p, []),
    "kara_workspace_size": (_I32, [_PAR, _I32, _I32, ctypes.POINTER(ctypes.c_size_t)]),
    "kara_validate": (_I32, [_PAR, _I32, _VP, _VP, _VP, _VP, _VP, _VP]),
    "kara_score_window": (_I32, [_PAR, _I32, _VP, _I32, _VP, _PP, _VP, _VP, _VP, _VP, _VP, _VP,
                                 ctypes.c_size_t, _VP]),
    "kara_select": (_I32, [_PAR, ctypes.c_int64, _VP, _VP, _VP]),
    "kara_token2chunk": (_I32, [_PAR, ctypes.c_int64, _VP, _VP, _VP, _VP]),
    "kara_select_kept": (_I32, [_PAR, ctypes.c_int64, _VP, _VP, _VP, _VP]),
    "kara_compact_pages": (_I32, [_PAR, _I32, _VP, _I32, _VP, _PP, _PP, _VP, _VP, _VP, _VP, _VP]),
    "kara_commit_tables": (_I32, [_PAR, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "kara_compress_window": (_I32, [_PAR, _I32, _VP, _I32, _VP, _PP, _PP, _VP, _VP, _VP, _I32, _VP, _VP,
                                    _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP]),
    "kara_compress_window_noalloc": (_I32, [_PAR, _I32, _VP, _I32, _VP, _PP, _PP, _VP, _VP, _VP, _I32, _VP, _VP,
                                            _VP, _VP, _VP, _VP, _VP]),
    "kara_compress_prefill": (_I32, [_PAR, _I32, _VP, _I32, _I32, _VP, _PP, _PP, _VP, _VP, _VP, _I32, _VP, _VP,
                                     _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP]),
    "kara_harness_kv_append": (_I32, [_PAR, _I32, _VP, _I32, _I32, _VP, _VP, _PP, _PP, _VP, _VP, _VP, _VP]),
    "kara_harness_decode_workspace_size": (_I32, [_PAR, _I32, _I32, _I32, ctypes.POINTER(ctypes.c_size_t)]),
    "kara_harness_decode_attention": (_I32, [_PAR, _I32, _VP, _I32, _VP, _PP, _PP, _VP, _VP, _I32, _VP, _VP,
                                             ctypes.c_size_t, _VP]),
    "kara_recompute_attention": (_I32, [_PAR, _I32, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    "kara_recompute_workspace_size": (_I32, [_PAR, ctypes.POINTER(KaraModel), _I32,
                                             ctypes.POINTER(ctypes.c_size_t)]),
    "kara_recompute_queries": (_I32, [_PAR, ctypes.POINTER(KaraModel), _I32, _VP, _I32, ctypes.POINTER(LayerWeights),
                                      _VP, _VP, _PP, _PP, _VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_size_t, _VP]),
    "kara_sched_create": (_I32, [ctypes.POINTER(SchedConfig), _P32, ctypes.POINTER(ctypes.c_void_p)]),
    "kara_sched_destroy": (_I32, [_VP]),
    "kara_sched_submit": (_I32, [_VP, _I32, _I32, _P64]),
    "kara_sched_step_begin": (_I32, [_VP, ctypes.POINTER(SchedStep)]),
    "kara_sched_step_end": (_I32, [_VP, ctypes.POINTER(SchedEvent)]),
    "kara_sched_event_commit": (_I32, [_VP, _P32, _P32]),
    "kara_sched_tables": (_I32, [_VP, ctypes.POINTER(_P32), ctypes.POINTER(_P32)]),
    "kara_sched_stats": (_I32, [_VP, ctypes.POINTER(SchedStats)]),
    "kara_sched_request": (_I32, [_VP, ctypes.c_int64, ctypes.POINTER(SchedRequest)]),
}

_lib = None


def header_functions() -> list[str]:
    """Names of the functions include/kara.h and include/kara_harness.h declare."""
    names = set()
    for h in HEADERS:
        names |= set(re.findall(r"^\S.*?\b(kara_\w+)\s*\(", open(h).read(), flags=re.M))
    return sorted(names)


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise KaraError("load", ERR_HIP, f"{path} is not built; run paper_2607_01237_amd.build")
    # torch ships its own copy of the HIP runtime.  It must be the one loaded
    # when the library resolves libamdhip64, or the library would start a
    # second runtime that cannot see torch's memory and streams.
    import torch  # noqa: F401
    try:
        lib = ctypes.CDLL(path)
    except OSError as e:
        raise KaraError("load", ERR_HIP, f"cannot load {path}: {e}") from e
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    # refuse a library built from other sources than the ones beside it
    from .build import source_hash
    built, here = lib.kara_source_hash().decode(), source_hash()
    if built != here:
        raise KaraError("load", ERR_HIP, f"{path} was built from other sources (library {built[:12]}, sources "
                                         f"{here[:12]}); rebuild with python -m paper_2607_01237_amd.build")
    _lib = lib
    return lib


def status_string(code: int) -> str:
    return load().kara_status_string(code).decode()


def _check(fn: str, code: int):
    if code != OK:
        msg = status_string(code)
        if code == ERR_HIP:
            msg += f" [{load().kara_last_hip_error().decode()}]"
        raise KaraError(fn, code, msg)


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise KaraError("marshal", ERR_INVALID_ARG, "tensor is not on the GPU")
    if not t.is_contiguous():
        raise KaraError("marshal", ERR_INVALID_ARG, "tensor is not contiguous")
    return ctypes.c_void_p(t.data_ptr())


# ---- host-side shape checks: the library takes bare pointers and cannot
# tell a short or mistyped tensor from a right one

def _need(name, t, n, dtype=None):
    """t (a GPU tensor, or None) holds at least n elements of dtype."""
    if t is None:
        return
    if dtype is not None and t.dtype != dtype:
        raise KaraError("marshal", ERR_INVALID_ARG, f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.numel() < n:
        raise KaraError("marshal", ERR_INVALID_ARG, f"{name}: {t.numel()} elements, at least {n} needed")


def _dt(p):
    import torch
    return torch.bfloat16 if p.dtype == BF16 else torch.float32


def _i32():
    import torch
    return torch.int32


def _f32():
    import torch
    return torch.float32


def _tables(p, block_table, seq_lens, win_start=None):
    _need("block_table", block_table, p.n_seqs * p.max_blocks_per_seq, _i32())
    _need("seq_lens", seq_lens, p.n_seqs, _i32())
    _need("win_start", win_start, p.n_seqs, _i32())


def _pools(p, pools, name):
    for i, t in enumerate(pools):
        _need(f"{name}[{i}]", t, p.num_pages * p.n_kv_heads * p.block_size * p.head_dim, _dt(p))


def _units(p, n_layers, n_trig, n_windows=1):
    return n_layers * n_trig * n_windows * p.n_kv_heads


def _step_outputs(p, units, scores, discrete, kept):
    _need("scores", scores, units * (p.window - p.buffer), _f32())
    _need("discrete", discrete, units * (p.budget - p.chunk_budget), _i32())
    _need("kept", kept, units * p.budget, _i32())


def _ptr_array(tensors):
    arr = (ctypes.c_void_p * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = _ptr(t).value
    return arr


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def abi_version() -> int:
    return int(load().kara_abi_version())


def workspace_size(p: KaraParams, n_trig: int, n_layers: int) -> int:
    out = ctypes.c_size_t(0)
    _check("kara_workspace_size", load().kara_workspace_size(ctypes.byref(p), n_trig, n_layers, ctypes.byref(out)))
    return int(out.value)


def validate(p, trig, block_table, seq_lens, win_start, status, stream=None):
    _need("trig", trig, 0, _i32())
    _need("status", status, trig.numel(), _i32())
    _tables(p, block_table, seq_lens, win_start)
    _check("kara_validate", load().kara_validate(ctypes.byref(p), trig.numel(), _ptr(trig), _ptr(block_table),
                                                 _ptr(seq_lens), _ptr(win_start), _ptr(status), _stream(stream)))


def score_window(p, trig, q, k_pools, block_table, seq_lens, win_start, scores, status, workspace,
                 stream=None):
    nt, L = trig.numel(), len(k_pools)
    _need("trig", trig, 0, _i32())
    _need("q", q, L * nt * (p.score_queries or p.window) * p.n_q_heads * p.head_dim, _dt(p))
    _pools(p, k_pools, "k_pools")
    _tables(p, block_table, seq_lens, win_start)
    _step_outputs(p, _units(p, L, nt), scores, None, None)
    _need("status", status, nt, _i32())
    _check("kara_score_window", load().kara_score_window(
        ctypes.byref(p), trig.numel(), _ptr(trig), len(k_pools), _ptr(q), _ptr_array(k_pools),
        _ptr(block_table), _ptr(seq_lens), _ptr(win_start), _ptr(scores), _ptr(status),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream)))


def select(p, scores, discrete, stream=None):
    n_units = scores.numel() // (p.window - p.buffer)
    _step_outputs(p, n_units, scores, discrete, None)
    _check("kara_select", load().kara_select(ctypes.byref(p), n_units, _ptr(scores), _ptr(discrete),
                                             _stream(stream)))


def token2chunk(p, scores, discrete, kept, stream=None):
    n_units = scores.numel() // (p.window - p.buffer)
    _step_outputs(p, n_units, scores, discrete, kept)
    _check("kara_token2chunk", load().kara_token2chunk(ctypes.byref(p), n_units, _ptr(scores), _ptr(discrete),
                                                       _ptr(kept), _stream(stream)))


def select_kept(p, scores, discrete, kept, stream=None):
    n_units = scores.numel() // (p.window - p.buffer)
    _step_outputs(p, n_units, scores, discrete, kept)
    _check("kara_select_kept", load().kara_select_kept(ctypes.byref(p), n_units, _ptr(scores), _ptr(discrete),
                                                       _ptr(kept), _stream(stream)))


def compact_pages(p, trig, kept, k_pools, v_pools, block_table, seq_lens, win_start, status, stream=None):
    nt, L = trig.numel(), len(k_pools)
    _need("trig", trig, 0, _i32())
    _step_outputs(p, _units(p, L, nt), None, None, kept)
    _pools(p, k_pools, "k_pools")
    _pools(p, v_pools, "v_pools")
    _tables(p, block_table, seq_lens, win_start)
    _need("status", status, nt, _i32())
    _check("kara_compact_pages", load().kara_compact_pages(
        ctypes.byref(p), trig.numel(), _ptr(trig), len(k_pools), _ptr(kept), _ptr_array(k_pools),
        _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(win_start), _ptr(status), _stream(stream)))


def commit_tables(p, trig, block_table, seq_lens, win_start, freed, n_freed, status, stream=None):
    nt = trig.numel()
    _need("trig", trig, 0, _i32())
    _tables(p, block_table, seq_lens, win_start)
    _need("freed", freed, nt * p.max_blocks_per_seq, _i32())
    _need("n_freed", n_freed, nt, _i32())
    _need("status", status, nt, _i32())
    _check("kara_commit_tables", load().kara_commit_tables(
        ctypes.byref(p), trig.numel(), _ptr(trig), _ptr(block_table), _ptr(seq_lens), _ptr(win_start),
        _ptr(freed), _ptr(n_freed), _ptr(status), _stream(stream)))


def _compress_checks(p, trig, n_windows, q, k_pools, v_pools, block_table, seq_lens, win_start, status,
                     scores, discrete, kept, freed, n_freed):
    nt, L = trig.numel(), len(k_pools)
    _need("trig", trig, 0, _i32())
    _need("q", q, L * nt * n_windows * (p.score_queries or p.window) * p.n_q_heads * p.head_dim, _dt(p))
    _pools(p, k_pools, "k_pools")
    _pools(p, v_pools, "v_pools")
    _tables(p, block_table, seq_lens, win_start)
    _step_outputs(p, _units(p, L, nt, n_windows), scores, discrete, kept)
    _need("freed", freed, nt * p.max_blocks_per_seq, _i32())
    _need("n_freed", n_freed, nt, _i32())
    _need("status", status, nt, _i32())


def compress_window(p, trig, q, k_pools, v_pools, block_table, seq_lens, win_start, commit, status,
                    workspace, scores=None, discrete=None, kept=None, freed=None, n_freed=None, stream=None):
    _compress_checks(p, trig, 1, q, k_pools, v_pools, block_table, seq_lens, win_start, status, scores, discrete,
                     kept, freed, n_freed)
    _check("kara_compress_window", load().kara_compress_window(
        ctypes.byref(p), trig.numel(), _ptr(trig), len(k_pools), _ptr(q), _ptr_array(k_pools),
        _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(win_start), int(bool(commit)),
        _ptr(scores), _ptr(discrete), _ptr(kept), _ptr(freed), _ptr(n_freed), _ptr(status), _ptr(workspace),
        workspace.numel() * workspace.element_size() if workspace is not None else 0, _stream(stream)))



def compress_window_noalloc(p, trig, q, k_pools, v_pools, block_table, seq_lens, win_start, commit, status,
                            scores=None, discrete=None, kept=None, freed=None, n_freed=None, stream=None):
    """kara_compress_window without a workspace: the library's static
    per-device scratch (NOALLOC_SCRATCH_BYTES) holds it."""
    _compress_checks(p, trig, 1, q, k_pools, v_pools, block_table, seq_lens, win_start, status, scores, discrete,
                     kept, freed, n_freed)
    _check("kara_compress_window_noalloc", load().kara_compress_window_noalloc(
        ctypes.byref(p), trig.numel(), _ptr(trig), len(k_pools), _ptr(q), _ptr_array(k_pools),
        _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(win_start), int(bool(commit)),
        _ptr(scores), _ptr(discrete), _ptr(kept), _ptr(freed), _ptr(n_freed), _ptr(status), _stream(stream)))

def compress_prefill(p, trig, n_windows, q, k_pools, v_pools, block_table, seq_lens, win_start, commit, status,
                     workspace, scores=None, discrete=None, kept=None, freed=None, n_freed=None, stream=None):
    """n_windows consecutive windows of every listed sequence at once (App. C.2)."""
    _compress_checks(p, trig, int(n_windows), q, k_pools, v_pools, block_table, seq_lens, win_start, status, scores,
                     discrete, kept, freed, n_freed)
    _check("kara_compress_prefill", load().kara_compress_prefill(
        ctypes.byref(p), trig.numel(), _ptr(trig), int(n_windows), len(k_pools), _ptr(q), _ptr_array(k_pools),
        _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(win_start), int(bool(commit)),
        _ptr(scores), _ptr(discrete), _ptr(kept), _ptr(freed), _ptr(n_freed), _ptr(status), _ptr(workspace),
        workspace.numel() * workspace.element_size() if workspace is not None else 0, _stream(stream)))


# ---- decoding-side helpers (include/kara_harness.h)

def kv_append(p, seqs, k_new, v_new, k_pools, v_pools, block_table, seq_lens, status, stream=None):
    """Appends k_new / v_new [n_layers][n][n_new][Hkv][d] after each listed sequence's tokens."""
    n, L = seqs.numel(), len(k_pools)
    _need("seqs", seqs, 0, _i32())
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _need(name, t, L * n * k_new.shape[2] * p.n_kv_heads * p.head_dim, _dt(p))
    _pools(p, k_pools, "k_pools")
    _pools(p, v_pools, "v_pools")
    _tables(p, block_table, seq_lens)
    _need("status", status, n, _i32())
    _check("kara_harness_kv_append", load().kara_harness_kv_append(
        ctypes.byref(p), seqs.numel(), _ptr(seqs), k_new.shape[2], len(k_pools), _ptr(k_new), _ptr(v_new),
        _ptr_array(k_pools), _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(status),
        _stream(stream)))


def decode_workspace_size(p, n, n_layers, max_len) -> int:
    out = ctypes.c_size_t(0)
    _check("kara_harness_decode_workspace_size", load().kara_harness_decode_workspace_size(
        ctypes.byref(p), n, n_layers, max_len, ctypes.byref(out)))
    return int(out.value)


def decode_attention(p, seqs, q, k_pools, v_pools, block_table, seq_lens, max_len, out, workspace,
                     stream=None):
    """One query per (layer, sequence, query head) over the paged cache; fp32 out of q's shape."""
    n, L = seqs.numel(), len(k_pools)
    _need("seqs", seqs, 0, _i32())
    _need("q", q, L * n * p.n_q_heads * p.head_dim, _dt(p))
    _need("out", out, L * n * p.n_q_heads * p.head_dim, _f32())
    _pools(p, k_pools, "k_pools")
    _pools(p, v_pools, "v_pools")
    _tables(p, block_table, seq_lens)
    _check("kara_harness_decode_attention", load().kara_harness_decode_attention(
        ctypes.byref(p), seqs.numel(), _ptr(seqs), len(k_pools), _ptr(q), _ptr_array(k_pools),
        _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), max_len, _ptr(out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


# ---- window recompute pass (include/kara_recompute.h)

def recompute_attention(p, trig, q, k_pool, v_pool, block_table, seq_lens, win_start, out, status, stream=None):
    """Causal attention of q [n_trig][W][Hq][d] (bf16) over one layer's paged cache into out."""
    nt = trig.numel()
    _need("trig", trig, 0, _i32())
    for name, t in (("q", q), ("out", out)):
        _need(name, t, nt * p.window * p.n_q_heads * p.head_dim, _dt(p))
    _pools(p, [k_pool], "k_pool")
    _pools(p, [v_pool], "v_pool")
    _tables(p, block_table, seq_lens, win_start)
    _need("status", status, nt, _i32())
    _check("kara_recompute_attention", load().kara_recompute_attention(
        ctypes.byref(p), trig.numel(), _ptr(trig), _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_table),
        _ptr(seq_lens), _ptr(win_start), _ptr(out), _ptr(status), _stream(stream)))


def make_model(hidden, ffn, rope_theta=1e6, rms_eps=1e-6) -> KaraModel:
    return KaraModel(int(hidden), int(ffn), float(rope_theta), float(rms_eps))


def recompute_workspace_size(p, m: KaraModel, n_trig: int) -> int:
    out = ctypes.c_size_t(0)
    _check("kara_recompute_workspace_size", load().kara_recompute_workspace_size(
        ctypes.byref(p), ctypes.byref(m), int(n_trig), ctypes.byref(out)))
    return int(out.value)


def recompute_queries(p, m: KaraModel, trig, weights, hidden_in, hidden_out, k_pools, v_pools, block_table,
                      seq_lens, win_start, rope_pos0, q_out, status, workspace, stream=None):
    """The window recompute pass over len(weights) layers; weights: one dict
    per layer of bf16 tensors w_q, w_o, w_gate, w_up, w_down, g_attn, g_ffn."""
    n, nt = len(weights), trig.numel()
    D, F, HD = m.hidden, m.ffn, p.n_q_heads * p.head_dim
    _need("trig", trig, 0, _i32())
    for name, t in (("hidden_in", hidden_in), ("hidden_out", hidden_out)):
        _need(name, t, nt * p.window * D, _f32())
    _need("q_out", q_out, n * nt * p.window * HD, _dt(p))
    _need("rope_pos0", rope_pos0, p.n_seqs, _i32())
    _pools(p, k_pools, "k_pools")
    _pools(p, v_pools, "v_pools")
    _tables(p, block_table, seq_lens, win_start)
    _need("status", status, nt, _i32())
    sizes = dict(w_q=D * HD, w_o=HD * D, w_gate=D * F, w_up=D * F, w_down=F * D, g_attn=D, g_ffn=D)
    for i, w in enumerate(weights):
        for f, size in sizes.items():
            _need(f"weights[{i}].{f}", w[f], size, _dt(p))
    arr = (LayerWeights * n)()
    for i, w in enumerate(weights):
        arr[i] = LayerWeights(*[_ptr(w[f]).value for f, _ in LayerWeights._fields_])
    _check("kara_recompute_queries", load().kara_recompute_queries(
        ctypes.byref(p), ctypes.byref(m), trig.numel(), _ptr(trig), n, arr, _ptr(hidden_in), _ptr(hidden_out),
        _ptr_array(k_pools), _ptr_array(v_pools), _ptr(block_table), _ptr(seq_lens), _ptr(win_start),
        _ptr(rope_pos0), _ptr(q_out), _ptr(status), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


# ---- periodic compression policy (include/kara_sched.h): host runtime

def _host_i32(a):
    """Host int32 pointer of a contiguous numpy array (or None)."""
    import numpy as np
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(_P32)


def _view(ptr, n, dtype):
    import numpy as np
    if n <= 0:
        return np.zeros(0, dtype=dtype)
    return np.ctypeslib.as_array(ptr, shape=(n,)).copy()


class Scheduler:
    """The host scheduler of include/kara_sched.h; every decision is made by
    the library, this class only converts its outputs to numpy arrays."""

    CONFIG_DEFAULTS = dict(reserve_pages=0, compress=1, protect_prompt=0)

    def __init__(self, cfg: dict, page_order=None):
        import numpy as np
        vals = dict(self.CONFIG_DEFAULTS, **cfg)
        self.cfg = SchedConfig(**{name: int(vals[name]) for name, _ in SchedConfig._fields_})
        self._lib = load()
        self._h = ctypes.c_void_p()
        po = _host_i32(page_order)
        _check("kara_sched_create", self._lib.kara_sched_create(ctypes.byref(self.cfg), po[1] if po else None,
                                                                  ctypes.byref(self._h)))
        self.n_slots, self.max_blocks = self.cfg.n_slots, self.cfg.max_blocks_per_seq
        self._np = np

    def close(self):
        if self._h:
            self._lib.kara_sched_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def submit(self, prompt_len: int, max_new: int) -> int:
        rid = ctypes.c_int64(-1)
        _check("kara_sched_submit", self._lib.kara_sched_submit(self._h, int(prompt_len), int(max_new),
                                                                  ctypes.byref(rid)))
        return int(rid.value)

    def step_begin(self) -> dict:
        st = SchedStep()
        _check("kara_sched_step_begin", self._lib.kara_sched_step_begin(self._h, ctypes.byref(st)))
        i32, i64 = self._np.int32, self._np.int64
        return dict(preempted=_view(st.preempted, st.n_preempted, i32), decode=_view(st.decode, st.n_decode, i32),
                    admitted=_view(st.admitted, st.n_admitted, i32),
                    prefill_len=_view(st.prefill_len, st.n_admitted, i32),
                    admitted_id=_view(st.admitted_id, st.n_admitted, i64), tables_changed=bool(st.tables_changed))

    def step_end(self):
        """(triggered slots, window start of every slot)."""
        ev = SchedEvent()
        _check("kara_sched_step_end", self._lib.kara_sched_step_end(self._h, ctypes.byref(ev)))
        return _view(ev.trig, ev.n_trig, self._np.int32), _view(ev.win_start, self.n_slots, self._np.int32)

    def commit(self, freed=None, n_freed=None):
        """Applies the pending event; freed / n_freed (host arrays) are checked
        against the scheduler's own release when given."""
        f, n = _host_i32(freed), _host_i32(n_freed)
        _check("kara_sched_event_commit", self._lib.kara_sched_event_commit(self._h, f[1] if f else None,
                                                                              n[1] if n else None))

    def tables(self):
        """Copies of the host block table [n_slots, max_blocks] and lengths [n_slots]."""
        bt, ln = _P32(), _P32()
        _check("kara_sched_tables", self._lib.kara_sched_tables(self._h, ctypes.byref(bt), ctypes.byref(ln)))
        return (_view(bt, self.n_slots * self.max_blocks, self._np.int32).reshape(self.n_slots, self.max_blocks),
                _view(ln, self.n_slots, self._np.int32))

    def stats(self) -> dict:
        s = SchedStats()
        _check("kara_sched_stats", self._lib.kara_sched_stats(self._h, ctypes.byref(s)))
        return {name: int(getattr(s, name)) for name, _ in SchedStats._fields_}

    def request(self, rid: int) -> dict:
        r = SchedRequest()
        _check("kara_sched_request", self._lib.kara_sched_request(self._h, int(rid), ctypes.byref(r)))
        return {name: int(getattr(r, name)) for name, _ in SchedRequest._fields_}
