/*
 * kara_harness.h -- decoding-side helpers of libkara for driving the
 * compression step over many events (token appends between events, and
 * attention of one new query per sequence over the compressed cache).
 *
 * These are not part of Kara's compression step.  They exist so that a
 * long-running workload -- append a window of tokens, decode, compress,
 * reuse the freed pages, repeat -- runs entirely on the GPU with the same
 * paged layout as the step (kara.h): pools [num_pages][n_kv_heads]
 * [block_size][head_dim] per layer, block table [n_seqs][max_blocks_per_seq]
 * int32 (-1 = none), seq_lens [n_seqs].  Same conventions as kara.h: device
 * pointers unless stated, the caller owns all memory, nothing synchronises,
 * host-checkable argument errors come back as KARA_ERR_* and nothing is
 * launched, per-sequence problems set status bits and leave the sequence
 * untouched.
 */
#ifndef KARA_HARNESS_H
#define KARA_HARNESS_H

#include "kara.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Query heads per KV head the decode attention supports. */
#define KARA_HARNESS_MAX_GROUP 16
/* Keys per split of the decode attention. */
#define KARA_HARNESS_SPLIT_KEYS 256

/*
 * Appends n_new tokens to each of the n sequences seqs[0..n) (distinct) in
 * every one of n_layers layers: K/V row of token i, KV head h, layer l goes to
 * logical position seq_lens[s] + i of sequence s = seqs[j], taken from
 * k_new / v_new [n_layers][n][n_new][n_kv_heads][head_dim] (p->dtype).  Then
 * seq_lens[s] += n_new.  The caller maps the logical blocks covering the new
 * positions in block_table beforehand.  status[j]: KARA_SEQ_BAD_INDEX (s
 * outside [0, n_seqs)), KARA_SEQ_DUP_TRIGGER (s listed twice),
 * KARA_SEQ_BAD_WINDOW (the new length exceeds max_blocks_per_seq *
 * block_size), KARA_SEQ_BAD_PAGE (a new position maps to no page of the
 * pool); flagged sequences are not written.  The window-related fields of p
 * (window, budget, ...) must be valid but are not used.
 */
kara_status_t kara_harness_kv_append(const kara_params_t* p, int32_t n, const int32_t* seqs,
                                     int32_t n_new, int32_t n_layers, const void* k_new,
                                     const void* v_new, void* const* k_pools, void* const* v_pools,
                                     const int32_t* block_table, int32_t* seq_lens,
                                     int32_t* status, void* stream);

/*
 * Bytes of device workspace kara_harness_decode_attention needs for n
 * sequences, n_layers layers and sequences of at most max_len tokens (written
 * to *bytes, a HOST pointer).
 */
kara_status_t kara_harness_decode_workspace_size(const kara_params_t* p, int32_t n, int32_t n_layers,
                                                 int32_t max_len, size_t* bytes);

/*
 * Attention of one query per (layer, sequence, query head) over the whole
 * paged cache of its sequence: out[l][j][hq][:] = softmax_k(scale * q . K_k)
 * V_k over positions k in [0, seq_lens[s]) of KV head hq / G (s = seqs[j],
 * G = n_q_heads / n_kv_heads <= KARA_HARNESS_MAX_GROUP; scale = p->scale, or
 * 1/sqrt(head_dim)).  q: [n_layers][n][n_q_heads][head_dim] (p->dtype); out:
 * fp32, same shape.  Sequences must be at most max_len tokens long (the
 * value the workspace was sized for); longer ones, empty ones and sequence
 * indices outside [0, n_seqs) give zero output rows.  Pages are not checked:
 * the block table must map every position below seq_len to a page of the
 * pool.
 */
kara_status_t kara_harness_decode_attention(const kara_params_t* p, int32_t n, const int32_t* seqs,
                                            int32_t n_layers, const void* q,
                                            const void* const* k_pools, const void* const* v_pools,
                                            const int32_t* block_table, const int32_t* seq_lens,
                                            int32_t max_len, float* out, void* workspace,
                                            size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KARA_HARNESS_H */
