/*
 * kara_sched.h -- host runtime of the periodic compression policy of
 * KvLLM (Kara, Sec. 4.3; App. C.4, Algorithm 1): continuous batching of a
 * running queue over a paged KV pool, a global decoding-step counter g, and
 * every `period` steps a compression event that picks the sequences whose
 * trailing context holds a whole uncompressed window and hands them to
 * kara_compress_window (include/kara.h).  Pages the compression releases go
 * back to the pool, where waiting sequences pick them up.
 *
 * This is host code only: it makes no HIP call and owns only host memory.
 * It keeps the block table, the sequence lengths and each sequence's window
 * start; the caller copies them to the device (kara_sched_tables) and runs
 * the GPU work of each step itself:
 *
 *     kara_sched_step_begin(s, &step)
 *         upload the tables when step.tables_changed
 *         prefill step.admitted[i] with step.prefill_len[i] tokens
 *         append one token to, and decode, every sequence in step.decode
 *     kara_sched_step_end(s, &event)
 *     if (event.n_trig > 0)
 *         kara_compress_window(trig = event.trig, win_start = event.win_start,
 *                              commit = 1, ...)
 *         kara_sched_event_commit(s, freed, n_freed)   (host copies)
 *
 * A sequence occupies one slot, the row of the block table the device calls
 * its sequence index, from admission until it finishes or is preempted.
 * Vacated slots are reused last-vacated first (slot 0 first at the start).
 *
 * Policy (where Algorithm 1 and App. C.4 leave a choice, the reading taken):
 *   - Step order: sequences already running get the page their next token
 *     needs first, in running-queue order.  When the pool is empty, the most
 *     recently admitted running sequence is preempted (its pages return to
 *     the pool; it goes back to the head of the waiting queue and, when
 *     readmitted, prefills its whole context so far, uncompressed) -- this
 *     may be the sequence that needed the page.  Only if nothing was
 *     preempted in this step are waiting sequences admitted, first come
 *     first served, while a slot is free, fewer than max_running run and
 *     the pool holds the prompt's pages plus reserve_pages.  Admitted
 *     sequences only prefill in their first step; the others decode one
 *     token each.
 *   - The counter: g is incremented once per step_end.  An event fires when
 *     g > window and g mod period == 0 (and compress is set).
 *   - Select: a running sequence with length len and window start p0 is a
 *     candidate when the window [p0, p0 + window) ends before the start of
 *     the sequence's last block, p0 + window <= block_size * (ceil(len /
 *     block_size) - 1): its trailing window is uncompressed and the last,
 *     possibly partial, block is never compressed.  Candidates are taken
 *     in running-queue order, at most max_per_event of them.
 *   - After an event each triggered sequence is window - buffer - budget
 *     tokens shorter, the blocks past its new length are released in
 *     ascending logical order (appended to the free list), and p0 advances
 *     by budget: the buffer re-enters the next window, which has thus slid
 *     by window - buffer over the uncompressed context.
 *   - p0 starts at 0 (the whole context, prompt included, is windowed) or,
 *     with protect_prompt, at the end of the prompt.
 *   - The free list is first in, first out: pages are handed out from its
 *     head and released pages join its tail.  It starts as page_order.
 *
 * Errors: every function returns a kara_status_t (include/kara.h).
 * Argument errors give KARA_ERR_INVALID_ARG and change nothing.  Calls out
 * of order (step_begin twice, step_end without step_begin, commit with no
 * event pending, step_begin with an event pending) give
 * KARA_ERR_INVALID_ARG.  kara_sched_event_commit returns
 * KARA_ERR_SCHED_MISMATCH when the device's freed list differs from the
 * host's; the host state is updated from its own computation either way.
 * KARA_ERR_SCHED_NOMEM reports that host memory for the scheduler's tables
 * or queues could not be allocated; the scheduler is then in an unspecified
 * state and may only be destroyed.
 * Pointers returned in the step / event / tables structs point into the
 * scheduler and stay valid until the next call on it.  A scheduler must not
 * be used from two threads at once.
 */
#ifndef KARA_SCHED_H
#define KARA_SCHED_H

#include <stdint.h>

#include "kara.h"

#ifdef __cplusplus
extern "C" {
#endif

/* The device's freed-page list differs from the host's model of it. */
#define KARA_ERR_SCHED_MISMATCH (-5)
/* Host memory for the scheduler could not be allocated. */
#define KARA_ERR_SCHED_NOMEM (-6)

typedef struct kara_sched kara_sched_t;

typedef struct kara_sched_config {
  int32_t n_slots;            /* rows of the block table (>= max_running) */
  int32_t num_pages;          /* pages in the pool */
  int32_t block_size;         /* tokens per page */
  int32_t max_blocks_per_seq; /* columns of the block table */
  int32_t window;             /* |W| */
  int32_t buffer;             /* |U| */
  int32_t budget;             /* kept positions per window, 1..window-buffer */
  int32_t period;             /* delta: decoding steps between events, >= 1 */
  int32_t max_per_event;      /* sequences compressed per event, >= 1 */
  int32_t max_running;        /* running-queue capacity, >= 1 */
  int32_t reserve_pages;      /* pages kept free at admission, >= 0 */
  int32_t compress;           /* 0: never fire (the uncompressed baseline) */
  int32_t protect_prompt;     /* 1: windows start after the prompt */
} kara_sched_config_t;

typedef struct kara_sched_step {
  int32_t n_preempted;
  const int32_t* preempted;   /* slots vacated by preemption this step */
  int32_t n_decode;
  const int32_t* decode;      /* slots that append and decode one token, queue order */
  int32_t n_admitted;
  const int32_t* admitted;    /* slots admitted this step (length 0, pages mapped) */
  const int32_t* prefill_len; /* tokens each admitted slot prefills */
  const int64_t* admitted_id; /* request id of each admitted slot */
  int32_t tables_changed;     /* the block table, or a length other than by the
                                 appends the previous step scheduled, changed
                                 since the previous step_begin */
} kara_sched_step_t;

typedef struct kara_sched_event {
  int32_t n_trig;
  const int32_t* trig;        /* triggered slots, queue order */
  const int32_t* win_start;   /* [n_slots]: window start of every slot */
} kara_sched_event_t;

typedef struct kara_sched_stats {
  int64_t steps;              /* g */
  int64_t events;             /* events that compressed at least one sequence */
  int64_t compressed;         /* sequences compressed, summed over events */
  int64_t pages_reclaimed;    /* pages released by compression */
  int64_t preemptions;
  int64_t tokens_decoded;     /* tokens generated by decoding steps */
  int64_t tokens_prefilled;   /* prompt (and recomputed) tokens prefilled */
  int32_t running, waiting, finished;
  int32_t free_pages;
  int32_t peak_running;       /* most sequences running after a step_begin */
  int32_t pages_in_use;       /* pages mapped by running sequences */
} kara_sched_stats_t;

/* Request states reported by kara_sched_request. */
#define KARA_REQ_WAITING 0
#define KARA_REQ_RUNNING 1
#define KARA_REQ_FINISHED 2

typedef struct kara_sched_request_info {
  int32_t state;              /* KARA_REQ_* */
  int32_t slot;               /* -1 unless running */
  int32_t len;                /* physical length (tokens in the cache) */
  int32_t win_start;          /* p0 */
  int32_t generated;          /* tokens generated so far */
  int32_t compressions;       /* events that compressed it */
  int32_t preemptions;
} kara_sched_request_info_t;

/* Creates a scheduler.  page_order: num_pages distinct page ids (host), the
 * initial free list; NULL = 0, 1, ..., num_pages - 1.  The configuration
 * needs budget <= window - buffer, window - buffer <= KARA_MAX_COMPRESSIBLE,
 * max_running <= n_slots and positive sizes. */
kara_status_t kara_sched_create(const kara_sched_config_t* cfg, const int32_t* page_order,
                                kara_sched_t** out);
kara_status_t kara_sched_destroy(kara_sched_t* s);

/* Queues a request of prompt_len >= 1 prompt tokens that generates
 * max_new >= 1 tokens; its id (0, 1, ... in submission order) goes to *id.
 * prompt_len + max_new must fit the block table uncompressed. */
kara_status_t kara_sched_submit(kara_sched_t* s, int32_t prompt_len, int32_t max_new, int64_t* id);

/* Preemptions, page mapping and admissions of the next step (see Policy). */
kara_status_t kara_sched_step_begin(kara_sched_t* s, kara_sched_step_t* out);

/* Ends the step: lengths advance by what step_begin scheduled, finished
 * sequences release their slot and pages, g increments, and the event (if
 * any) is selected.  With n_trig > 0 the event is pending until
 * kara_sched_event_commit. */
kara_status_t kara_sched_step_end(kara_sched_t* s, kara_sched_event_t* out);

/* Applies the pending event's metadata update.  freed / n_freed: host
 * copies of kara_compress_window's outputs ([n_trig][max_blocks_per_seq],
 * [n_trig]) to check against, or both NULL. */
kara_status_t kara_sched_event_commit(kara_sched_t* s, const int32_t* freed, const int32_t* n_freed);

/* Host block table [n_slots][max_blocks_per_seq] and lengths [n_slots]. */
kara_status_t kara_sched_tables(const kara_sched_t* s, const int32_t** block_table, const int32_t** seq_lens);

kara_status_t kara_sched_stats(const kara_sched_t* s, kara_sched_stats_t* out);

kara_status_t kara_sched_request(const kara_sched_t* s, int64_t id, kara_sched_request_info_t* out);

#ifdef __cplusplus
}
#endif

#endif /* KARA_SCHED_H */
