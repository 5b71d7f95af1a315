// Internal declarations shared by libkara's host API and its gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kara.h"

namespace kara {

// Most layers one launch addresses (their pool pointers travel as kernel
// arguments); larger calls are split into several launches.
constexpr int kMaxLayersPerLaunch = 64;

// Geometry as the kernels see it (derived once on the host).
struct Geom {
  int W, U, N;          // window, buffer, compressible length N = W - U
  int Wq;               // scoring queries per unit (the window's last Wq positions)
  int n_win;            // windows per listed sequence: 1, or consecutive prefill windows
                        // at stride N (units = layers x n_trig x n_win x Hkv)
  int budget, alpha, gamma;
  int k_disc;           // budget - alpha, Eq. (5)
  int n_chunks;         // floor(alpha / (gamma - 2)), Eq. (7)
  int d, Hq, Hkv, G;    // head dim, query heads, KV heads, group size
  int bs, num_pages, max_blocks, n_seqs;
  int dtype;            // KARA_BF16 | KARA_F32
  int esize;            // element bytes
  float scale;          // logit scale of Eq. (1)
  int n_trig;
};

struct PoolPtrs {
  void* p[kMaxLayersPerLaunch];
};

// Host helpers shared by the API files (kara_api.cpp): parameter checks into
// a Geom (n_trig: the count of listed sequences), HIP status mapping that
// remembers the error for kara_last_hip_error, pool-array check.
kara_status_t make_geom(const kara_params_t* p, int32_t n_trig, Geom* g);
kara_status_t hip_status(hipError_t e);
bool pools_ok(const void* const* pools, int n_layers);

// Validation kernel (kara_pages.hip).  keep_kept: a KARA_SEQ_BAD_KEPT bit
// already in status survives (staged per-layer compaction and the commit).
hipError_t launch_validate(const Geom& g, const int32_t* trig, const int32_t* block_table,
                           const int32_t* seq_lens, const int32_t* win_start, int32_t* status,
                           bool keep_kept, hipStream_t stream);

// Scoring (kara_score.hip): per unit, n_splits workgroups each write a
// partial column sum into `partials`, and a second kernel adds them in split
// order into `scores` (with one split the workgroup writes `scores` directly).
struct ScorePlan {
  int rows_wg;          // query rows per workgroup
  int n_splits;         // row splits (workgroups) per unit
  int single_nt;        // key tiles per wave of the single-sweep kernel; 0: two sweeps
};
ScorePlan plan_score(const Geom& g, int64_t n_units);
hipError_t launch_score(const Geom& g, const ScorePlan& sp, int n_layers, const void* q,
                        const PoolPtrs& k_pools, const int32_t* trig, const int32_t* block_table,
                        const int32_t* win_start, const int32_t* status, float* partials,
                        float* scores, hipStream_t stream);

// Selection (kara_select.hip).  mode bit 1: discrete top-k; bit 2: Token2Chunk
// + fill (from discrete_in when bit 1 is clear).
enum { kSelectDiscrete = 1, kSelectKept = 2 };
hipError_t launch_select(const Geom& g, int64_t n_units, int mode, const float* scores,
                         const int32_t* discrete_in, int32_t* discrete_out, int32_t* kept_out,
                         hipStream_t stream);

// Compaction and metadata (kara_pages.hip).
hipError_t launch_check_kept(const Geom& g, int n_layers, const int32_t* kept, int32_t* status,
                             hipStream_t stream);
hipError_t launch_compact(const Geom& g, int n_layers, const int32_t* trig, const int32_t* kept,
                          const PoolPtrs& k_pools, const PoolPtrs& v_pools,
                          const int32_t* block_table, const int32_t* seq_lens,
                          const int32_t* win_start, const int32_t* status, hipStream_t stream);
hipError_t launch_commit(const Geom& g, const int32_t* trig, int32_t* block_table,
                         int32_t* seq_lens, const int32_t* win_start, int32_t* freed,
                         int32_t* n_freed, const int32_t* status, hipStream_t stream);

// One compression event (kara_api.cpp): the body of kara_compress_window
// (n_win = 1) and kara_compress_prefill, workspace supplied by the caller.
kara_status_t compress(const kara_params_t* p, int32_t n_trig, const int32_t* trig, int32_t n_win,
                       int32_t n_layers, const void* q, void* const* k_pools, void* const* v_pools,
                       int32_t* block_table, int32_t* seq_lens, const int32_t* win_start, int32_t commit,
                       float* scores, int32_t* discrete, int32_t* kept, int32_t* freed, int32_t* n_freed,
                       int32_t* status, void* workspace, size_t workspace_bytes, void* stream);
// Workspace bytes compress() needs for g (g.n_trig, g.n_win set) and n_layers.
size_t compress_workspace_bytes(const Geom& g, int32_t n_layers);

// Window recompute pass (kara_attn.hip, kara_recompute_ops.hip).
// Validation of the listed sequences for the recompute pass: index, duplicate,
// window inside the sequence, pages of [0, p0 + W) inside the pool.
hipError_t launch_recompute_validate(const Geom& g, const int32_t* trig, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* win_start, int32_t* status,
                                     hipStream_t stream);
// Causal attention of q [n_trig][W][Hq][d] over one layer's cache; skips
// sequences whose status is non-zero.
hipError_t launch_recompute_attention(const Geom& g, const void* q, const void* k_pool, const void* v_pool,
                                      const int32_t* trig, const int32_t* block_table, const int32_t* win_start,
                                      void* out, const int32_t* status, hipStream_t stream);

hipError_t launch_rmsnorm(const float* h, const void* gamma, void* x, int64_t n_tok, int D, float eps,
                          hipStream_t stream);
hipError_t launch_rope(const void* qraw, void* q_out, int n_trig, int W, int Hq, int d, float theta,
                       const int32_t* trig, const int32_t* rope_pos0, const int32_t* status, hipStream_t stream);
hipError_t launch_swiglu(void* gate, const void* up, int64_t n, hipStream_t stream);

}  // namespace kara
