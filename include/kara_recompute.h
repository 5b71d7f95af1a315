/*
 * kara_recompute.h -- the window recompute pass of Kara (App. C.2).
 *
 * The window queries Q_W that Eq. (4) scores with are not kept while
 * decoding.  At a compression event one extra forward pass over the |W|
 * window tokens of each triggered sequence recomputes them, layer by layer:
 * only the query projection, causal attention against the K/V rows already
 * in the cache, and the feed-forward block run; no key or value is
 * recomputed.  With h the residual stream of the window tokens (fp32):
 *
 *   x   = RMSNorm(h) * g_attn
 *   q   = RoPE(x W_q) at rotary positions rope_pos0[s] + w
 *                          -> this layer's scoring queries
 *   o_w = softmax(q_w K[0 : p0+w+1]^T * scale) V[0 : p0+w+1]
 *                          window token w sits at cache position p0 + w,
 *                          p0 = win_start[s]; query head hq reads KV head
 *                          hq / G
 *   h  += concat_heads(o) W_o
 *   x'  = RMSNorm(h) * g_ffn
 *   h  += (silu(x' W_gate) * (x' W_up)) W_down
 *
 * The architecture is that of the decoders the paper evaluates (Qwen3 /
 * Llama family): pre-norm RMSNorm, rotary embedding in the rotate-half form
 * on the queries (cached keys carry theirs), SwiGLU feed-forward, no biases.
 *
 * Conventions are those of kara.h: device pointers owned by the caller,
 * nothing synchronised, argument errors as return codes with nothing
 * enqueued, per-sequence problems in status[t] (KARA_SEQ_*): index out of
 * range, listed twice, window past the sequence end (p0 + window >
 * seq_len), or a page of [0, p0 + window) outside the pool.  A flagged
 * sequence's attention output and scoring queries are left unwritten;
 * kara_recompute_queries runs the matrix products over every listed row, so
 * a flagged sequence's hidden_out rows are unspecified.  bf16 only
 * (params.dtype = KARA_BF16, else KARA_ERR_UNSUPPORTED), head_dim 64 or 128.
 * Device arrays are 16-byte aligned.
 *
 * Allocation.  The matrix products run on rocBLAS.  Their scratch is a
 * 32 MiB slice of the caller's workspace, handed to rocBLAS
 * (rocblas_set_workspace) after a size query has confirmed the products fit
 * in it (else KARA_ERR_WORKSPACE), so rocBLAS allocates no workspace of its
 * own.  The one thing the library creates on this path is the rocBLAS
 * handle: kara_recompute_queries makes one per device on its first call
 * there (rocblas_create_handle: rocBLAS's host state and whatever device
 * memory the handle takes for itself) and keeps it until the process ends;
 * later calls allocate nothing.  Each call binds that handle to its stream
 * and workspace, so calls on one device from several host threads at once
 * must be serialised by the caller.
 *
 * Layouts (row-major)
 *   q, out (attention)  [n_trig][window][n_q_heads][head_dim] bf16
 *   q_out               [n_layers][n_trig][window][n_q_heads][head_dim] bf16:
 *                       the scoring queries, the q argument of
 *                       kara_compress_window for the same trig list
 *   hidden_in/out       [n_trig][window][hidden] fp32
 *   weights             bf16, multiplied from the right: w_q [hidden][n_q_heads*
 *                       head_dim], w_o [n_q_heads*head_dim][hidden], w_gate and
 *                       w_up [hidden][ffn], w_down [ffn][hidden]; g_attn and
 *                       g_ffn [hidden]
 *   rope_pos0           [n_seqs] int32: rotary position of each window's first token
 */
#ifndef KARA_RECOMPUTE_H
#define KARA_RECOMPUTE_H

#include <stddef.h>
#include <stdint.h>

#include "kara.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kara_model {
  int32_t hidden;      /* model width D, a multiple of 4 */
  int32_t ffn;         /* feed-forward width F, a multiple of 8 */
  float rope_theta;    /* rotary base */
  float rms_eps;       /* RMSNorm epsilon (inside the square root) */
} kara_model_t;

typedef struct kara_layer_weights {
  const void* w_q;
  const void* w_o;
  const void* w_gate;
  const void* w_up;
  const void* w_down;
  const void* g_attn;
  const void* g_ffn;
} kara_layer_weights_t;

/* Causal attention of one layer's window queries over the paged cache
 * (the attention step above).  k_pool, v_pool: that layer's pools
 * [num_pages][n_kv_heads][block_size][head_dim].  Validates every listed
 * sequence into status first. */
kara_status_t kara_recompute_attention(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                       const void* q, const void* k_pool, const void* v_pool,
                                       const int32_t* block_table, const int32_t* seq_lens,
                                       const int32_t* win_start, void* out, int32_t* status, void* stream);

/* Bytes of workspace kara_recompute_queries needs for n_trig sequences. */
kara_status_t kara_recompute_workspace_size(const kara_params_t* p, const kara_model_t* m, int32_t n_trig,
                                            size_t* bytes);

/* The whole pass over n_layers layers: weights, k_pools, v_pools are host
 * arrays of n_layers entries (device pointers).  Writes every layer's
 * scoring queries to q_out and the residual stream after the last layer to
 * hidden_out (may equal hidden_in).  The matrix products run on rocBLAS on
 * `stream`. */
kara_status_t kara_recompute_queries(const kara_params_t* p, const kara_model_t* m, int32_t n_trig,
                                     const int32_t* trig, int32_t n_layers, const kara_layer_weights_t* weights,
                                     const float* hidden_in, float* hidden_out, const void* const* k_pools,
                                     const void* const* v_pools, const int32_t* block_table,
                                     const int32_t* seq_lens, const int32_t* win_start, const int32_t* rope_pos0,
                                     void* q_out, int32_t* status, void* workspace, size_t workspace_bytes,
                                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KARA_RECOMPUTE_H */
