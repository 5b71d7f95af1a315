/*
 * kara.h -- C ABI of libkara, the MI355X (gfx950) implementation of Kara's
 * sliding-window KV-cache compression step (Kara, Sec. 4 and App. C).
 *
 * One compression event, for every triggered sequence, every layer and every
 * KV head ("unit"), runs:
 *   1. window scoring, Eq. (4): bidirectional (unmasked) attention of the
 *      |W| window queries over the |W|-|U| compressible window keys, softmax
 *      over keys, column sum over queries.  With grouped-query attention the
 *      G = n_q_heads / n_kv_heads query heads sharing a KV head are all
 *      queries of that head (G*|W| query rows per unit).  The query set can
 *      be narrowed to the window's trailing positions (score_queries);
 *   2. discrete top-k, Eq. (5): budget - alpha positions;
 *   3. Token2Chunk, Eq. (6)-(8), then the fill rule of App. C.3: exactly
 *      `budget` kept positions per unit;
 *   4. the window gather, Eq. (9), done in place in the paged cache (memory
 *      compaction of Algorithm 1), and the metadata update: trailing pages
 *      released, block table and sequence length rewritten.
 *
 * Conventions
 *   - Every array pointer is DEVICE memory owned by the caller, except the
 *     `k_pools` / `v_pools` arrays themselves, which are HOST arrays of
 *     `n_layers` device pointers.  The library allocates nothing.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls only enqueue
 *     work; none synchronises.
 *   - Return codes report host-checkable argument errors only; on error
 *     nothing is enqueued.  Data-dependent problems of a triggered sequence
 *     (window outside the sequence, page id outside the pool, a page mapped
 *     twice, the sequence triggered twice, sequence index out of range) are
 *     written to the device array `status[t]` (KARA_SEQ_* bits); such a
 *     sequence gets zero scores and is neither compacted nor committed.
 *   - Page ownership: compaction moves rows in place, so the pages holding a
 *     triggered sequence's window and tail must belong to that sequence
 *     alone.  A page mapped twice inside one sequence is flagged
 *     (KARA_SEQ_DUP_PAGE); a page shared between two sequences is not
 *     checked and must not occur (no prefix sharing of window pages).
 *   - status lifetime within one event: kara_validate, kara_score_window,
 *     kara_compress_window and kara_compress_prefill rewrite status[t]
 *     from scratch.  kara_compact_pages and kara_commit_tables keep a
 *     KARA_SEQ_BAD_KEPT bit already set, so a bad kept set found in any
 *     layer's compaction call stops the commit of that sequence; start an
 *     event with one of the former calls.
 *   - kara_token2chunk writes -1 to every kept entry of a unit whose discrete
 *     row is not strictly ascending inside [0, window - buffer).
 *   - Ordering: every ranking is by (value descending, index ascending).
 *
 * Layouts (row-major, contiguous)
 *   q            [n_layers][n_trig][Wq][n_q_heads][head_dim]   bf16|f32,
 *                the queries of the last Wq window positions (Wq = window
 *                unless kara_params_t.score_queries says otherwise);
 *                query head hq = kv_head * G + g belongs to KV head kv_head.
 *   pools        per layer [num_pages][n_kv_heads][block_size][head_dim]
 *   block_table  [n_seqs][max_blocks_per_seq] int32, -1 = no page
 *   seq_lens, win_start  [n_seqs] int32; the window of sequence s covers
 *                logical positions [win_start[s], win_start[s] + window);
 *                positions [win_start+window, seq_len) are the tail that
 *                follows the window.  win_start need not be block aligned.
 *   trig         [n_trig] int32 sequence indices compressed by this call
 *   scores       [n_layers][n_trig][n_kv_heads][window - buffer]    f32
 *   discrete     [n_layers][n_trig][n_kv_heads][budget - chunk_budget] int32,
 *                ascending window-relative positions
 *   kept         [n_layers][n_trig][n_kv_heads][budget] int32, ascending
 *   status       [n_trig] int32
 *   freed        [n_trig][max_blocks_per_seq] int32 page ids released, in
 *                ascending logical-block order, -1 after the last one
 *   n_freed      [n_trig] int32
 *
 * Unit u = (layer * n_trig + t) * n_kv_heads + kv_head.
 */
#ifndef KARA_H
#define KARA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KARA_ABI_VERSION 3

/* Largest compressible region |W|-|U| one call supports. */
#define KARA_MAX_COMPRESSIBLE 4096

typedef enum kara_dtype {
  KARA_BF16 = 0, /* raw bfloat16, 2 bytes */
  KARA_F32 = 1   /* IEEE binary32 */
} kara_dtype_t;

typedef enum kara_status {
  KARA_OK = 0,
  KARA_ERR_INVALID_ARG = -1, /* a parameter is out of range or a pointer is NULL */
  KARA_ERR_UNSUPPORTED = -2, /* valid but not built (e.g. head_dim not 64/128) */
  KARA_ERR_WORKSPACE = -3,   /* workspace missing or smaller than kara_workspace_size() */
  KARA_ERR_HIP = -4,         /* the HIP runtime rejected a launch */
  KARA_ERR_SCRATCH_LIMIT = -7 /* kara_compress_window_noalloc: the call needs more than
                                 KARA_NOALLOC_SCRATCH_BYTES of scratch, or the scratch
                                 could not be resolved on the current device */
} kara_status_t;

/* Per-sequence device status bits. */
#define KARA_SEQ_OK 0
#define KARA_SEQ_BAD_WINDOW 1   /* win_start < 0, win_start + window > seq_len, or seq_len > table capacity */
#define KARA_SEQ_BAD_PAGE 2     /* a page id of the window or tail is outside [0, num_pages) */
#define KARA_SEQ_DUP_TRIGGER 4  /* the sequence appears more than once in trig */
#define KARA_SEQ_BAD_INDEX 8    /* trig[t] outside [0, n_seqs) */
#define KARA_SEQ_BAD_KEPT 16    /* kara_compact_pages: a kept row not ascending or outside [0, window-buffer) */
#define KARA_SEQ_DUP_PAGE 32    /* a page of the blocks compaction writes ([win_start/block_size,
                                   ceil(seq_len/block_size))) appears twice among the sequence's
                                   blocks [0, ceil(seq_len/block_size)) */

/*
 * Window and cache geometry (Kara Sec. 4.1, Eq. (5) and (7); App. C.4).
 *   window          |W| >= 1
 *   buffer          |U|, 0 <= U < W; window - buffer <= KARA_MAX_COMPRESSIBLE
 *   budget          ceil(r (|W|-|U|)): positions kept per unit, 1..W-U
 *   chunk_budget    alpha, 0 <= alpha < budget
 *   max_chunk_len   gamma >= 3, chunk length counting both endpoints
 *   head_dim        d, 64 or 128
 *   n_q_heads, n_kv_heads   n_q_heads a multiple of n_kv_heads
 *   block_size      tokens per page, >= 1
 *   num_pages       pages in each pool
 *   max_blocks_per_seq, n_seqs   block-table shape
 *   dtype           KARA_BF16 or KARA_F32 (q and the pools)
 *   scale           logit scale; <= 0 means 1/sqrt(head_dim) (Eq. (1))
 *   score_queries   Wq, the number of window queries that score the
 *                   compressible keys -- those of the last Wq window
 *                   positions -- with the same softmax over the compressible
 *                   keys and column sum as Eq. (4).  0 or window: every
 *                   window query (Kara's bidirectional scoring).  buffer: the
 *                   buffer's queries only (the ablation without bidirectional
 *                   attention, Sec. 5.3).  With the window spanning the whole
 *                   cache and chunk_budget 0, the whole-cache top-k of
 *                   Eq. (2)-(3) scored by a trailing observation window.
 *                   1 <= Wq <= window otherwise.
 */
typedef struct kara_params {
  int32_t window;
  int32_t buffer;
  int32_t budget;
  int32_t chunk_budget;
  int32_t max_chunk_len;
  int32_t head_dim;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t block_size;
  int32_t num_pages;
  int32_t max_blocks_per_seq;
  int32_t n_seqs;
  int32_t dtype;
  float scale;
  int32_t score_queries;
} kara_params_t;

/* Human-readable name of a kara_status_t value.  Never NULL. */
const char* kara_status_string(int32_t status);

/* KARA_ABI_VERSION of the loaded library. */
int32_t kara_abi_version(void);

/*
 * Build provenance (not part of the method): hex SHA-256 over the sources,
 * headers and compile options this library was built from, or "unknown".
 * A caller holding the sources can recompute it to make sure the loaded
 * binary is current.  Static storage; never freed by the caller.
 */
const char* kara_source_hash(void);

/*
 * Text of the HIP error behind the most recent KARA_ERR_HIP returned on the
 * calling thread ("no HIP error" if there was none).  Static storage; never
 * freed by the caller.
 */
const char* kara_last_hip_error(void);

/*
 * Bytes of device workspace kara_score_window / kara_compress_window need for
 * this geometry, n_trig triggered sequences and n_layers layers (written to
 * *bytes, a HOST pointer).  Holds partial column sums of Eq. (4) and, for
 * outputs the caller does not request, the scores and index sets.
 */
kara_status_t kara_workspace_size(const kara_params_t* p, int32_t n_trig, int32_t n_layers,
                                  size_t* bytes);

/*
 * Checks every triggered sequence's window against its length and block
 * table and writes status[t] (KARA_SEQ_* bits).  Reads block_table,
 * seq_lens, win_start; writes status.
 */
kara_status_t kara_validate(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                            const int32_t* block_table, const int32_t* seq_lens,
                            const int32_t* win_start, int32_t* status, void* stream);

/*
 * Window scoring, Eq. (4), for n_layers layers: writes scores (fp32) and
 * status.  The key states are read from k_pools through the block table.
 * Reductions run in a fixed order, so results are bit-reproducible.
 */
kara_status_t kara_score_window(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                int32_t n_layers, const void* q, const void* const* k_pools,
                                const int32_t* block_table, const int32_t* seq_lens,
                                const int32_t* win_start, float* scores, int32_t* status,
                                void* workspace, size_t workspace_bytes, void* stream);

/*
 * Discrete top-k, Eq. (5): for each of n_units score rows (window - buffer
 * fp32 values), writes the budget - chunk_budget best positions, ascending.
 */
kara_status_t kara_select(const kara_params_t* p, int64_t n_units, const float* scores,
                          int32_t* discrete, void* stream);

/*
 * Token2Chunk, Eq. (6)-(8), and the fill rule of App. C.3: from each unit's
 * scores and ascending discrete set, writes the `budget` kept positions,
 * ascending.  Chunk scores are formed in fp64 from the fp32 scores.
 */
kara_status_t kara_token2chunk(const kara_params_t* p, int64_t n_units, const float* scores,
                               const int32_t* discrete, int32_t* kept, void* stream);

/*
 * Eq. (5)-(8) and the fill rule of App. C.3 in one launch, as
 * kara_compress_window runs them: writes both the discrete set (as
 * kara_select) and the kept positions (as kara_token2chunk), bit for bit
 * the two calls' results, with one pass over each unit's scores.
 */
kara_status_t kara_select_kept(const kara_params_t* p, int64_t n_units, const float* scores,
                               int32_t* discrete, int32_t* kept, void* stream);

/*
 * Window gather, Eq. (9), in place in the paged pools of n_layers layers:
 * window-relative row j receives row kept[j] for j < budget, then the buffer
 * rows, then the tail rows (each K and V head independently).  Writes status
 * (validation runs first; a KARA_SEQ_BAD_KEPT bit already in status[t] is
 * kept, and a sequence with any bit set is not compacted).  Does not touch
 * block_table or seq_lens: call kara_commit_tables once after every layer
 * has been compacted.  Compacting the same layer twice before committing is
 * a caller error.  When layers are compacted one call at a time and a later
 * call finds a bad kept set, the layers compacted by earlier calls stay
 * compacted and the commit skips the sequence: its cache is then
 * inconsistent and must be rebuilt by the caller (the check of all layers'
 * kept sets before any compaction is one call over all layers).
 */
kara_status_t kara_compact_pages(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                 int32_t n_layers, const int32_t* kept, void* const* k_pools,
                                 void* const* v_pools, const int32_t* block_table,
                                 const int32_t* seq_lens, const int32_t* win_start,
                                 int32_t* status, void* stream);

/*
 * Metadata update of Algorithm 1: new seq_len = seq_len - (window - buffer -
 * budget); the logical blocks no longer covered are released (page ids into
 * freed[t][*] in ascending block order, table entries set to -1).  Writes
 * status (validation runs first, keeping a KARA_SEQ_BAD_KEPT bit set by this
 * event's kara_compact_pages calls); flagged sequences are left unchanged.
 */
kara_status_t kara_commit_tables(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                 int32_t* block_table, int32_t* seq_lens,
                                 const int32_t* win_start, int32_t* freed, int32_t* n_freed,
                                 int32_t* status, void* stream);

/*
 * The whole step (Kara Sec. 4, Algorithm 1) for n_layers layers: validation,
 * scoring, selection, Token2Chunk + fill, in-place compaction and -- when
 * `commit` is non-zero -- the metadata update.  scores, discrete and kept are
 * optional outputs (NULL: kept in the workspace).  freed/n_freed are needed
 * only when commit is non-zero.
 */
kara_status_t kara_compress_window(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                   int32_t n_layers, const void* q, void* const* k_pools,
                                   void* const* v_pools, int32_t* block_table, int32_t* seq_lens,
                                   const int32_t* win_start, int32_t commit, float* scores,
                                   int32_t* discrete, int32_t* kept, int32_t* freed,
                                   int32_t* n_freed, int32_t* status, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * Prefill-time compression (App. C.2): the prompt's KV pairs compressed
 * window by window, all windows at once.  Sequence s = trig[t] holds
 * n_windows consecutive windows starting at win_start[s], window w covering
 * [win_start + w*(W-U), win_start + w*(W-U) + W): consecutive windows share
 * the U buffer positions, whose queries score both and whose keys belong to
 * the next window's compressible region.  Each window is one unit per layer
 * and KV head, scored by its own queries (Eq. (4)) and selected on its own
 * (Eq. (5)-(8), App. C.3).  Compaction then leaves, in order, every window's
 * `budget` kept rows and everything after the last window's compressible
 * region (its buffer and the rest of the sequence); the commit shortens the
 * sequence by n_windows * (window - buffer - budget).  One window is
 * kara_compress_window.  The next decode-time window of a compressed
 * sequence starts at win_start + n_windows * budget.
 *
 * Layouts gain a window index after the trigger:
 *   q       [n_layers][n_trig][n_windows][Wq][n_q_heads][head_dim]
 *   scores  [n_layers][n_trig][n_windows][n_kv_heads][window - buffer]
 *   discrete, kept  [n_layers][n_trig][n_windows][n_kv_heads][...]
 * The workspace is sized by kara_workspace_size(p, n_trig * n_windows,
 * n_layers).  A sequence too short for its windows is flagged
 * KARA_SEQ_BAD_WINDOW.  n_windows < 1, or windows longer than a block-table
 * row, is KARA_ERR_INVALID_ARG.
 */
kara_status_t kara_compress_prefill(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                    int32_t n_windows, int32_t n_layers, const void* q,
                                    void* const* k_pools, void* const* v_pools, int32_t* block_table,
                                    int32_t* seq_lens, const int32_t* win_start, int32_t commit,
                                    float* scores, int32_t* discrete, int32_t* kept, int32_t* freed,
                                    int32_t* n_freed, int32_t* status, void* workspace,
                                    size_t workspace_bytes, void* stream);

/*
 * Allocation-free variant of kara_compress_window, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments and results as
 * kara_compress_window without the workspace: the partial column sums, and
 * the scores and index sets the caller does not request, live in a static
 * device array of KARA_NOALLOC_SCRATCH_BYTES that the library holds on every
 * GPU it runs on until the process ends.  The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine).
 *
 * Limit: the workspace kara_workspace_size() reports for (p, n_trig,
 * n_layers) must fit in KARA_NOALLOC_SCRATCH_BYTES, else the call returns
 * KARA_ERR_SCRATCH_LIMIT and enqueues nothing.  64 MiB holds about 3,000
 * units of a 32/8-head, W = 1024 model with scores and index sets left to
 * the library (22 KB each): 53 sequences x 7 layers, or one layer of 380
 * sequences.  The array's device address is resolved once per
 * device, on the first call with that device current.
 *
 * Every call on one GPU shares that GPU's array and leaves its contents
 * there; nothing in it needs to start at zero.  Calls that overlap on one
 * GPU (other streams or host threads without ordering) race on the array:
 * the caller serialises them.
 */
#define KARA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

kara_status_t kara_compress_window_noalloc(const kara_params_t* p, int32_t n_trig, const int32_t* trig,
                                           int32_t n_layers, const void* q, void* const* k_pools,
                                           void* const* v_pools, int32_t* block_table, int32_t* seq_lens,
                                           const int32_t* win_start, int32_t commit, float* scores,
                                           int32_t* discrete, int32_t* kept, int32_t* freed,
                                           int32_t* n_freed, int32_t* status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KARA_H */
