// Host side of libkara's C ABI: argument checks, workspace carving and the
// launch sequence of one compression event (Kara Algorithm 1, App. C.4).
#include <cmath>
#include <cstdint>

#include "kara_internal.h"

using namespace kara;

namespace kara {

constexpr int kMaxWindow = 1 << 16;

kara_status_t make_geom(const kara_params_t* p, int32_t n_trig, Geom* g) {
  if (!p || n_trig < 0) return KARA_ERR_INVALID_ARG;
  const int W = p->window, U = p->buffer;
  if (W < 1 || W > kMaxWindow || U < 0 || U >= W) return KARA_ERR_INVALID_ARG;
  const int N = W - U;
  if (N > KARA_MAX_COMPRESSIBLE) return KARA_ERR_UNSUPPORTED;
  // fp32 windows: at most 64K head-dim elements of keys (1024 keys at d=64, 512 at d=128)
  if (p->dtype == KARA_F32 && (int64_t)N * p->head_dim > 65536) return KARA_ERR_UNSUPPORTED;
  if (p->budget < 1 || p->budget > N) return KARA_ERR_INVALID_ARG;
  if (p->chunk_budget < 0 || p->chunk_budget >= p->budget) return KARA_ERR_INVALID_ARG;
  if (p->max_chunk_len < 3) return KARA_ERR_INVALID_ARG;
  if (p->head_dim < 1 || p->n_q_heads < 1 || p->n_kv_heads < 1) return KARA_ERR_INVALID_ARG;
  if (p->n_q_heads % p->n_kv_heads != 0) return KARA_ERR_INVALID_ARG;
  if (p->block_size < 1 || p->num_pages < 1 || p->max_blocks_per_seq < 1 || p->n_seqs < 1)
    return KARA_ERR_INVALID_ARG;
  if ((int64_t)p->max_blocks_per_seq * p->block_size > INT32_MAX) return KARA_ERR_INVALID_ARG;
  if ((int64_t)p->n_q_heads / p->n_kv_heads * W > INT32_MAX / 2) return KARA_ERR_INVALID_ARG;
  if (p->dtype != KARA_BF16 && p->dtype != KARA_F32) return KARA_ERR_INVALID_ARG;
  if (p->score_queries < 0 || p->score_queries > W) return KARA_ERR_INVALID_ARG;
  if (std::isinf(p->scale)) return KARA_ERR_INVALID_ARG;
  if (p->head_dim != 64 && p->head_dim != 128) return KARA_ERR_UNSUPPORTED;
  // the scoring kernel addresses key rows by 32-bit offsets in 16-byte units
  if ((int64_t)p->num_pages * p->n_kv_heads * p->block_size * p->head_dim *
          (p->dtype == KARA_BF16 ? 2 : 4) / 16 > (int64_t)UINT32_MAX)
    return KARA_ERR_UNSUPPORTED;
  g->W = W;
  g->U = U;
  g->N = N;
  g->Wq = p->score_queries > 0 ? p->score_queries : W;
  g->n_win = 1;
  g->budget = p->budget;
  g->alpha = p->chunk_budget;
  g->gamma = p->max_chunk_len;
  g->k_disc = p->budget - p->chunk_budget;
  g->n_chunks = p->chunk_budget / (p->max_chunk_len - 2);
  g->d = p->head_dim;
  g->Hq = p->n_q_heads;
  g->Hkv = p->n_kv_heads;
  g->G = p->n_q_heads / p->n_kv_heads;
  g->bs = p->block_size;
  g->num_pages = p->num_pages;
  g->max_blocks = p->max_blocks_per_seq;
  g->n_seqs = p->n_seqs;
  g->dtype = p->dtype;
  g->esize = p->dtype == KARA_BF16 ? 2 : 4;
  g->scale = (p->scale > 0.f) ? p->scale : (float)(1.0 / std::sqrt((double)p->head_dim));
  g->n_trig = n_trig;
  return KARA_OK;
}

// the last HIP error a call on this thread failed with (hipSuccess: none)
thread_local hipError_t t_last_hip_error = hipSuccess;

kara_status_t hip_status(hipError_t e) {
  if (e == hipSuccess) return KARA_OK;
  t_last_hip_error = e;
  return KARA_ERR_HIP;
}

bool pools_ok(const void* const* pools, int n_layers) {
  if (!pools) return false;
  for (int i = 0; i < n_layers; ++i)
    if (!pools[i]) return false;
  return true;
}

}  // namespace kara

namespace {

inline size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct WsLayout {
  size_t partials, scores, discrete, kept, total;
};

WsLayout ws_layout(const Geom& g, int n_layers, const ScorePlan& sp) {
  const int64_t units = (int64_t)n_layers * g.n_trig * g.n_win * g.Hkv;
  WsLayout w{};
  size_t off = 0;
  w.partials = off;
  off = align_up(off + (sp.n_splits > 1 ? (size_t)units * sp.n_splits * g.N * sizeof(float) : 0));
  w.scores = off;
  off = align_up(off + (size_t)units * g.N * sizeof(float));
  w.discrete = off;
  off = align_up(off + (size_t)units * g.k_disc * sizeof(int32_t));
  w.kept = off;
  off = align_up(off + (size_t)units * g.budget * sizeof(int32_t));
  w.total = off;
  return w;
}


// Runs fn(layer0, count, pool-pointer structs) over chunks of at most
// kMaxLayersPerLaunch layers.
template <typename Fn>
hipError_t for_layer_chunks(int n_layers, const void* const* k_pools, const void* const* v_pools,
                            Fn fn) {
  for (int l0 = 0; l0 < n_layers; l0 += kMaxLayersPerLaunch) {
    const int cnt = n_layers - l0 < kMaxLayersPerLaunch ? n_layers - l0 : kMaxLayersPerLaunch;
    PoolPtrs kp{}, vp{};
    for (int i = 0; i < cnt; ++i) {
      kp.p[i] = const_cast<void*>(k_pools[l0 + i]);
      if (v_pools) vp.p[i] = const_cast<void*>(v_pools[l0 + i]);
    }
    hipError_t e = fn(l0, cnt, kp, vp);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}


// Window scores of every layer.
hipError_t run_score(const Geom& g, const ScorePlan& sp, int n_layers, const void* q,
                     const void* const* k_pools, const int32_t* trig, const int32_t* bt,
                     const int32_t* win_start, const int32_t* status, float* partials,
                     float* scores, hipStream_t stream) {
  const int64_t q_layer = (int64_t)g.n_trig * g.n_win * g.Wq * g.Hq * g.d * g.esize;
  const int64_t units_layer = (int64_t)g.n_trig * g.n_win * g.Hkv;
  return for_layer_chunks(n_layers, k_pools, nullptr, [&](int l0, int cnt, const PoolPtrs& kp, const PoolPtrs&) {
    return launch_score(g, sp, cnt, (const char*)q + l0 * q_layer, kp, trig, bt, win_start, status,
                        partials + l0 * units_layer * sp.n_splits * g.N, scores + l0 * units_layer * g.N,
                        stream);
  });
}

hipError_t run_compact(const Geom& g, int n_layers, const int32_t* trig, const int32_t* kept,
                       void* const* k_pools, void* const* v_pools, const int32_t* bt,
                       const int32_t* seq_lens, const int32_t* win_start, const int32_t* status,
                       hipStream_t stream) {
  const int64_t k_layer = (int64_t)g.n_trig * g.n_win * g.Hkv * g.budget;
  return for_layer_chunks(n_layers, (const void* const*)k_pools, (const void* const*)v_pools,
                          [&](int l0, int cnt, const PoolPtrs& kp, const PoolPtrs& vp) {
                            return launch_compact(g, cnt, trig, kept + l0 * k_layer, kp, vp, bt,
                                                  seq_lens, win_start, status, stream);
                          });
}

}  // namespace

namespace kara {

size_t compress_workspace_bytes(const Geom& g, int32_t n_layers) {
  const ScorePlan sp = plan_score(g, (int64_t)n_layers * g.n_trig * g.n_win * g.Hkv);
  return ws_layout(g, n_layers, sp).total;
}

// One compression event over n_win consecutive windows (stride W - U) of
// each listed sequence: validation, scoring, selection, compaction and, if
// asked, the metadata commit.
kara_status_t compress(const kara_params_t* p, int32_t n_trig, const int32_t* trig, int32_t n_win,
                       int32_t n_layers, const void* q, void* const* k_pools, void* const* v_pools,
                       int32_t* block_table, int32_t* seq_lens, const int32_t* win_start, int32_t commit,
                       float* scores, int32_t* discrete, int32_t* kept, int32_t* freed, int32_t* n_freed,
                       int32_t* status, void* workspace, size_t workspace_bytes, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_layers < 1 || n_win < 1) return KARA_ERR_INVALID_ARG;
  if ((int64_t)(n_win - 1) * g.N + g.W > (int64_t)g.max_blocks * g.bs) return KARA_ERR_INVALID_ARG;
  g.n_win = n_win;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !q || !block_table || !seq_lens || !win_start || !status ||
      !pools_ok((const void* const*)k_pools, n_layers) || !pools_ok((const void* const*)v_pools, n_layers))
    return KARA_ERR_INVALID_ARG;
  if (commit && (!freed || !n_freed)) return KARA_ERR_INVALID_ARG;
  const int64_t units = (int64_t)n_layers * n_trig * n_win * g.Hkv;
  if (units > INT32_MAX) return KARA_ERR_INVALID_ARG;
  const ScorePlan sp = plan_score(g, units);
  const WsLayout wl = ws_layout(g, n_layers, sp);
  if (!workspace || workspace_bytes < wl.total) return KARA_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  float* partials = (float*)(ws + wl.partials);
  float* scores_buf = scores ? scores : (float*)(ws + wl.scores);
  int32_t* kept_buf = kept ? kept : (int32_t*)(ws + wl.kept);
  hipStream_t s = (hipStream_t)stream;

  hipError_t e = launch_validate(g, trig, block_table, seq_lens, win_start, status, false, s);
  if (e == hipSuccess)
    e = run_score(g, sp, n_layers, q, (const void* const*)k_pools, trig, block_table, win_start, status,
                  partials, scores_buf, s);
  if (e == hipSuccess)
    e = launch_select(g, units, kSelectDiscrete | kSelectKept, scores_buf, nullptr, discrete, kept_buf, s);
  if (e == hipSuccess)
    e = run_compact(g, n_layers, trig, kept_buf, k_pools, v_pools, block_table, seq_lens, win_start,
                    status, s);
  if (e == hipSuccess && commit)
    e = launch_commit(g, trig, block_table, seq_lens, win_start, freed, n_freed, status, s);
  return hip_status(e);
}

}  // namespace kara

extern "C" {

const char* kara_status_string(int32_t s) {
  switch (s) {
    case KARA_OK: return "KARA_OK";
    case KARA_ERR_INVALID_ARG: return "KARA_ERR_INVALID_ARG: a parameter is out of range or a pointer is NULL";
    case KARA_ERR_UNSUPPORTED: return "KARA_ERR_UNSUPPORTED: valid parameters libkara does not support";
    case KARA_ERR_WORKSPACE: return "KARA_ERR_WORKSPACE: workspace missing or too small";
    case KARA_ERR_HIP: return "KARA_ERR_HIP: the HIP runtime rejected a launch";
    case -5: return "KARA_ERR_SCHED_MISMATCH: the device's freed pages differ from the scheduler's";
    case -6: return "KARA_ERR_SCHED_NOMEM: host memory for the scheduler could not be allocated";
    case KARA_ERR_SCRATCH_LIMIT:
      return "KARA_ERR_SCRATCH_LIMIT: the call needs more scratch than the allocation-free entry point holds "
             "(KARA_NOALLOC_SCRATCH_BYTES per device), or its scratch could not be resolved on this device";
    default: return "unknown kara status";
  }
}

int32_t kara_abi_version(void) { return KARA_ABI_VERSION; }

#ifndef KARA_SOURCE_HASH
#define KARA_SOURCE_HASH "unknown"
#endif
const char* kara_source_hash(void) { return KARA_SOURCE_HASH; }

const char* kara_last_hip_error(void) {
  return t_last_hip_error == hipSuccess ? "no HIP error" : hipGetErrorString(t_last_hip_error);
}

kara_status_t kara_workspace_size(const kara_params_t* p, int32_t n_trig, int32_t n_layers,
                                  size_t* bytes) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (!bytes || n_layers < 1) return KARA_ERR_INVALID_ARG;
  const ScorePlan sp = plan_score(g, (int64_t)n_layers * n_trig * g.Hkv);
  *bytes = ws_layout(g, n_layers, sp).total;
  return KARA_OK;
}

kara_status_t kara_validate(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                            const int32_t* block_table, const int32_t* seq_lens,
                            const int32_t* win_start, int32_t* status, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !block_table || !seq_lens || !win_start || !status) return KARA_ERR_INVALID_ARG;
  return hip_status(
      launch_validate(g, trig, block_table, seq_lens, win_start, status, false, (hipStream_t)stream));
}

kara_status_t kara_score_window(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                int32_t n_layers, const void* q, const void* const* k_pools,
                                const int32_t* block_table, const int32_t* seq_lens,
                                const int32_t* win_start, float* scores, int32_t* status,
                                void* workspace, size_t workspace_bytes, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_layers < 1) return KARA_ERR_INVALID_ARG;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !q || !block_table || !seq_lens || !win_start || !scores || !status ||
      !pools_ok(k_pools, n_layers))
    return KARA_ERR_INVALID_ARG;
  const int64_t units = (int64_t)n_layers * n_trig * g.Hkv;
  const ScorePlan sp = plan_score(g, units);
  const WsLayout wl = ws_layout(g, n_layers, sp);
  if (!workspace || workspace_bytes < wl.total) return KARA_ERR_WORKSPACE;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  hipError_t e = launch_validate(g, trig, block_table, seq_lens, win_start, status, false, s);
  if (e == hipSuccess)
    e = run_score(g, sp, n_layers, q, k_pools, trig, block_table, win_start, status, (float*)(ws + wl.partials),
                  scores, s);
  return hip_status(e);
}

kara_status_t kara_select(const kara_params_t* p, int64_t n_units, const float* scores,
                          int32_t* discrete, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, 0, &g);
  if (st != KARA_OK) return st;
  if (n_units < 0 || n_units > INT32_MAX) return KARA_ERR_INVALID_ARG;
  if (n_units == 0) return KARA_OK;
  if (!scores || !discrete) return KARA_ERR_INVALID_ARG;
  return hip_status(launch_select(g, n_units, kSelectDiscrete, scores, nullptr, discrete, nullptr,
                                  (hipStream_t)stream));
}

kara_status_t kara_token2chunk(const kara_params_t* p, int64_t n_units, const float* scores,
                               const int32_t* discrete, int32_t* kept, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, 0, &g);
  if (st != KARA_OK) return st;
  if (n_units < 0 || n_units > INT32_MAX) return KARA_ERR_INVALID_ARG;
  if (n_units == 0) return KARA_OK;
  if (!scores || !discrete || !kept) return KARA_ERR_INVALID_ARG;
  return hip_status(launch_select(g, n_units, kSelectKept, scores, discrete, nullptr, kept,
                                  (hipStream_t)stream));
}

kara_status_t kara_select_kept(const kara_params_t* p, int64_t n_units, const float* scores,
                               int32_t* discrete, int32_t* kept, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, 0, &g);
  if (st != KARA_OK) return st;
  if (n_units < 0 || n_units > INT32_MAX) return KARA_ERR_INVALID_ARG;
  if (n_units == 0) return KARA_OK;
  if (!scores || !discrete || !kept) return KARA_ERR_INVALID_ARG;
  return hip_status(launch_select(g, n_units, kSelectDiscrete | kSelectKept, scores, nullptr, discrete, kept,
                                  (hipStream_t)stream));
}

kara_status_t kara_compact_pages(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                 int32_t n_layers, const int32_t* kept, void* const* k_pools,
                                 void* const* v_pools, const int32_t* block_table,
                                 const int32_t* seq_lens, const int32_t* win_start,
                                 int32_t* status, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_layers < 1) return KARA_ERR_INVALID_ARG;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !kept || !block_table || !seq_lens || !win_start || !status ||
      !pools_ok((const void* const*)k_pools, n_layers) || !pools_ok((const void* const*)v_pools, n_layers))
    return KARA_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_validate(g, trig, block_table, seq_lens, win_start, status, true, s);
  if (e == hipSuccess) e = launch_check_kept(g, n_layers, kept, status, s);
  if (e == hipSuccess)
    e = run_compact(g, n_layers, trig, kept, k_pools, v_pools, block_table, seq_lens, win_start, status, s);
  return hip_status(e);
}

kara_status_t kara_commit_tables(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                 int32_t* block_table, int32_t* seq_lens,
                                 const int32_t* win_start, int32_t* freed, int32_t* n_freed,
                                 int32_t* status, void* stream) {
  Geom g;
  kara_status_t st = make_geom(p, n_trig, &g);
  if (st != KARA_OK) return st;
  if (n_trig == 0) return KARA_OK;
  if (!trig || !block_table || !seq_lens || !win_start || !freed || !n_freed || !status)
    return KARA_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_validate(g, trig, block_table, seq_lens, win_start, status, true, s);
  if (e == hipSuccess) e = launch_commit(g, trig, block_table, seq_lens, win_start, freed, n_freed, status, s);
  return hip_status(e);
}

kara_status_t kara_compress_window(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                   int32_t n_layers, const void* q, void* const* k_pools,
                                   void* const* v_pools, int32_t* block_table, int32_t* seq_lens,
                                   const int32_t* win_start, int32_t commit, float* scores,
                                   int32_t* discrete, int32_t* kept, int32_t* freed,
                                   int32_t* n_freed, int32_t* status, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  return compress(p, n_trig, trig, 1, n_layers, q, k_pools, v_pools, block_table, seq_lens, win_start, commit,
                  scores, discrete, kept, freed, n_freed, status, workspace, workspace_bytes, stream);
}

kara_status_t kara_compress_prefill(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                    int32_t n_windows, int32_t n_layers, const void* q,
                                    void* const* k_pools, void* const* v_pools, int32_t* block_table,
                                    int32_t* seq_lens, const int32_t* win_start, int32_t commit,
                                    float* scores, int32_t* discrete, int32_t* kept, int32_t* freed,
                                    int32_t* n_freed, int32_t* status, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  return compress(p, n_trig, trig, n_windows, n_layers, q, k_pools, v_pools, block_table, seq_lens, win_start,
                  commit, scores, discrete, kept, freed, n_freed, status, workspace, workspace_bytes, stream);
}

}  // extern "C"
