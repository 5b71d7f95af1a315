// Host runtime of the periodic compression policy (Algorithm 1, App. C.4):
// continuous batching over a paged pool, the global step counter and the
// selection of compression events.  Pure host code; the GPU work of each
// step is the caller's (include/kara_sched.h).
#include <cstring>
#include <deque>
#include <memory>
#include <vector>

#include "kara.h"
#include "kara_sched.h"

namespace {

struct Request {
  int32_t prompt_len = 0;
  int32_t max_new = 0;
  int32_t generated = 0;
  int32_t state = KARA_REQ_WAITING;
  int32_t slot = -1;
  int32_t compressions = 0;
  int32_t preemptions = 0;
  int32_t prefill_len = 0;  // tokens to prefill at the next admission
};

int32_t ceil_div(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }

}  // namespace

struct kara_sched {
  kara_sched_config_t cfg{};
  std::vector<int32_t> table;   // [n_slots][max_blocks]
  std::vector<int32_t> lens;    // [n_slots]
  std::vector<int32_t> p0;      // [n_slots]
  std::vector<int64_t> owner;   // [n_slots] request id, -1 when free
  std::deque<int32_t> free_pages;
  std::deque<int64_t> waiting;  // request ids, head first
  std::vector<int64_t> running; // request ids, admission order
  std::vector<int32_t> free_slots;  // stack: the last slot vacated is reused first; 0 first at start
  std::vector<Request> reqs;

  // per-step outputs
  std::vector<int32_t> preempted, decode, admitted, prefill;
  std::vector<int64_t> admitted_id;
  std::vector<int32_t> trig;
  bool in_step = false;
  bool event_pending = false;
  bool changed = true;

  kara_sched_stats_t st{};

  int32_t mapped(int32_t slot) const {
    const int32_t* row = &table[(size_t)slot * cfg.max_blocks_per_seq];
    int32_t n = 0;
    while (n < cfg.max_blocks_per_seq && row[n] >= 0) ++n;
    return n;
  }

  void release_row(int32_t slot) {
    int32_t* row = &table[(size_t)slot * cfg.max_blocks_per_seq];
    for (int32_t b = 0; b < cfg.max_blocks_per_seq && row[b] >= 0; ++b) {
      free_pages.push_back(row[b]);
      row[b] = -1;
    }
    lens[slot] = 0;
    p0[slot] = 0;
    owner[slot] = -1;
    free_slots.push_back(slot);
    changed = true;
  }

  // Maps blocks of `slot` until it covers n_tokens; the caller has checked
  // that enough pages are free.
  void map_to(int32_t slot, int32_t n_tokens) {
    int32_t* row = &table[(size_t)slot * cfg.max_blocks_per_seq];
    const int32_t need = ceil_div(n_tokens, cfg.block_size);
    for (int32_t b = 0; b < need; ++b)
      if (row[b] < 0) {
        row[b] = free_pages.front();
        free_pages.pop_front();
        changed = true;
      }
  }

  void preempt_last() {
    const int64_t id = running.back();
    running.pop_back();
    Request& r = reqs[(size_t)id];
    const int32_t slot = r.slot;
    // recompute on readmission: the whole context so far, uncompressed
    r.prefill_len = r.prompt_len + r.generated;
    r.state = KARA_REQ_WAITING;
    r.slot = -1;
    r.preemptions += 1;
    st.preemptions += 1;
    release_row(slot);
    preempted.push_back(slot);
    waiting.push_front(id);
  }
};

namespace {

// Every entry point runs its body through guarded(): the C ABI lets no
// exception through, and the containers below can only throw on allocation.
template <typename F>
kara_status_t guarded(F&& body) {
  try {
    return body();
  } catch (...) {
    return (kara_status_t)KARA_ERR_SCHED_NOMEM;
  }
}

bool config_ok(const kara_sched_config_t& c) {
  if (c.n_slots < 1 || c.num_pages < 1 || c.block_size < 1 || c.max_blocks_per_seq < 1) return false;
  if (c.window < 1 || c.buffer < 0 || c.buffer >= c.window) return false;
  if (c.window - c.buffer > KARA_MAX_COMPRESSIBLE) return false;
  if (c.budget < 1 || c.budget > c.window - c.buffer) return false;
  if (c.period < 1 || c.max_per_event < 1 || c.max_running < 1 || c.max_running > c.n_slots) return false;
  if (c.reserve_pages < 0 || c.reserve_pages >= c.num_pages) return false;
  if ((int64_t)c.n_slots * c.max_blocks_per_seq > ((int64_t)1 << 31)) return false;
  return true;
}

}  // namespace

extern "C" {

kara_status_t kara_sched_create(const kara_sched_config_t* cfg, const int32_t* page_order, kara_sched_t** out) {
  return guarded([&]() -> kara_status_t {
    if (!cfg || !out || !config_ok(*cfg)) return KARA_ERR_INVALID_ARG;
    if (page_order) {
      std::vector<char> seen((size_t)cfg->num_pages, 0);
      for (int32_t i = 0; i < cfg->num_pages; ++i) {
        const int32_t p = page_order[i];
        if (p < 0 || p >= cfg->num_pages || seen[(size_t)p]) return KARA_ERR_INVALID_ARG;
        seen[(size_t)p] = 1;
      }
    }
    std::unique_ptr<kara_sched> s(new kara_sched());   // freed if an allocation below throws
    s->cfg = *cfg;
    s->table.assign((size_t)cfg->n_slots * cfg->max_blocks_per_seq, -1);
    s->lens.assign((size_t)cfg->n_slots, 0);
    s->p0.assign((size_t)cfg->n_slots, 0);
    s->owner.assign((size_t)cfg->n_slots, -1);
    for (int32_t i = 0; i < cfg->num_pages; ++i) s->free_pages.push_back(page_order ? page_order[i] : i);
    for (int32_t i = cfg->n_slots - 1; i >= 0; --i) s->free_slots.push_back(i);
    s->st.free_pages = cfg->num_pages;
    *out = s.release();
    return KARA_OK;
  });
}

kara_status_t kara_sched_destroy(kara_sched_t* s) {
  return guarded([&]() -> kara_status_t {
    delete s;
    return KARA_OK;
  });
}

kara_status_t kara_sched_submit(kara_sched_t* s, int32_t prompt_len, int32_t max_new, int64_t* id) {
  return guarded([&]() -> kara_status_t {
    if (!s || prompt_len < 1 || max_new < 1) return KARA_ERR_INVALID_ARG;
    const int64_t total = (int64_t)prompt_len + max_new;
    const int64_t blocks = (total + s->cfg.block_size - 1) / s->cfg.block_size;
    // the whole context must fit the block table, and the pool, uncompressed
    // (a preempted sequence is readmitted uncompressed)
    if (blocks > s->cfg.max_blocks_per_seq || blocks > s->cfg.num_pages - s->cfg.reserve_pages)
      return KARA_ERR_INVALID_ARG;
    Request r;
    r.prompt_len = prompt_len;
    r.max_new = max_new;
    r.prefill_len = prompt_len;
    s->reqs.push_back(r);
    const int64_t rid = (int64_t)s->reqs.size() - 1;
    s->waiting.push_back(rid);
    if (id) *id = rid;
    return KARA_OK;
  });
}

kara_status_t kara_sched_step_begin(kara_sched_t* s, kara_sched_step_t* out) {
  return guarded([&]() -> kara_status_t {
    if (!s || !out || s->in_step || s->event_pending) return KARA_ERR_INVALID_ARG;
    const kara_sched_config_t& c = s->cfg;
    s->preempted.clear();
    s->decode.clear();
    s->admitted.clear();
    s->prefill.clear();
    s->admitted_id.clear();

    // 1. the next token of every running sequence, in queue order
    for (size_t i = 0; i < s->running.size(); ++i) {
      const int64_t id = s->running[i];
      const int32_t slot = s->reqs[(size_t)id].slot;
      const int32_t need = ceil_div((int64_t)s->lens[(size_t)slot] + 1, c.block_size);
      bool self_preempted = false;
      while (s->mapped(slot) < need && s->free_pages.empty()) {
        const bool self = s->running.back() == id;
        s->preempt_last();
        if (self) {
          self_preempted = true;
          break;
        }
      }
      if (self_preempted) break;  // it was the last in the queue
      s->map_to(slot, s->lens[(size_t)slot] + 1);
      s->decode.push_back(slot);
    }

    // 2. admissions, only if nothing was preempted
    if (s->preempted.empty()) {
      while (!s->waiting.empty() && !s->free_slots.empty() && (int32_t)s->running.size() < c.max_running) {
        const int64_t id = s->waiting.front();
        Request& r = s->reqs[(size_t)id];
        const int32_t pages = ceil_div(r.prefill_len, c.block_size);
        if ((int64_t)s->free_pages.size() < (int64_t)pages + c.reserve_pages) break;
        s->waiting.pop_front();
        const int32_t slot = s->free_slots.back();
        s->free_slots.pop_back();
        r.state = KARA_REQ_RUNNING;
        r.slot = slot;
        s->owner[(size_t)slot] = id;
        s->lens[(size_t)slot] = 0;
        s->p0[(size_t)slot] = c.protect_prompt ? r.prompt_len : 0;
        s->map_to(slot, r.prefill_len);
        s->running.push_back(id);
        s->admitted.push_back(slot);
        s->prefill.push_back(r.prefill_len);
        s->admitted_id.push_back(id);
        s->changed = true;
      }
    }

    if ((int32_t)s->running.size() > s->st.peak_running) s->st.peak_running = (int32_t)s->running.size();
    out->n_preempted = (int32_t)s->preempted.size();
    out->preempted = s->preempted.data();
    out->n_decode = (int32_t)s->decode.size();
    out->decode = s->decode.data();
    out->n_admitted = (int32_t)s->admitted.size();
    out->admitted = s->admitted.data();
    out->prefill_len = s->prefill.data();
    out->admitted_id = s->admitted_id.data();
    out->tables_changed = s->changed ? 1 : 0;
    s->changed = false;
    s->in_step = true;
    return KARA_OK;
  });
}

kara_status_t kara_sched_step_end(kara_sched_t* s, kara_sched_event_t* out) {
  return guarded([&]() -> kara_status_t {
    if (!s || !out || !s->in_step) return KARA_ERR_INVALID_ARG;
    const kara_sched_config_t& c = s->cfg;
    s->in_step = false;
    for (size_t i = 0; i < s->admitted.size(); ++i) {
      s->lens[(size_t)s->admitted[i]] = s->prefill[i];
      s->st.tokens_prefilled += s->prefill[i];
    }
    for (int32_t slot : s->decode) {
      s->lens[(size_t)slot] += 1;
      s->reqs[(size_t)s->owner[(size_t)slot]].generated += 1;
      s->st.tokens_decoded += 1;
    }
    // finished sequences leave the running queue
    std::vector<int64_t> still;
    still.reserve(s->running.size());
    for (int64_t id : s->running) {
      Request& r = s->reqs[(size_t)id];
      if (r.generated >= r.max_new) {
        r.state = KARA_REQ_FINISHED;
        s->release_row(r.slot);
        r.slot = -1;
        s->st.finished += 1;
      } else {
        still.push_back(id);
      }
    }
    s->running.swap(still);
    s->st.steps += 1;

    s->trig.clear();
    const int64_t g = s->st.steps;
    if (c.compress && g > c.window && g % c.period == 0) {
      for (int64_t id : s->running) {
        if ((int32_t)s->trig.size() >= c.max_per_event) break;
        const int32_t slot = s->reqs[(size_t)id].slot;
        const int64_t len = s->lens[(size_t)slot];
        const int64_t last_block_start = (int64_t)c.block_size * (ceil_div(len, c.block_size) - 1);
        if ((int64_t)s->p0[(size_t)slot] + c.window <= last_block_start) s->trig.push_back(slot);
      }
    }
    s->event_pending = !s->trig.empty();
    out->n_trig = (int32_t)s->trig.size();
    out->trig = s->trig.data();
    out->win_start = s->p0.data();
    return KARA_OK;
  });
}

kara_status_t kara_sched_event_commit(kara_sched_t* s, const int32_t* freed, const int32_t* n_freed) {
  return guarded([&]() -> kara_status_t {
    if (!s || !s->event_pending || (!freed) != (!n_freed)) return KARA_ERR_INVALID_ARG;
    const kara_sched_config_t& c = s->cfg;
    const int32_t shrink = c.window - c.buffer - c.budget;
    bool mismatch = false;
    for (size_t t = 0; t < s->trig.size(); ++t) {
      const int32_t slot = s->trig[t];
      const int32_t len = s->lens[(size_t)slot];
      const int32_t new_len = len - shrink;
      const int32_t b0 = ceil_div(new_len, c.block_size), b1 = ceil_div(len, c.block_size);
      int32_t* row = &s->table[(size_t)slot * c.max_blocks_per_seq];
      if (n_freed && n_freed[t] != b1 - b0) mismatch = true;
      for (int32_t b = b0; b < b1; ++b) {
        if (freed && (n_freed[t] != b1 - b0 || freed[t * (size_t)c.max_blocks_per_seq + (b - b0)] != row[b]))
          mismatch = true;
        s->free_pages.push_back(row[b]);
        row[b] = -1;
      }
      s->st.pages_reclaimed += b1 - b0;
      s->lens[(size_t)slot] = new_len;
      s->p0[(size_t)slot] += c.budget;
      s->reqs[(size_t)s->owner[(size_t)slot]].compressions += 1;
    }
    s->st.events += 1;
    s->st.compressed += (int64_t)s->trig.size();
    s->event_pending = false;
    s->changed = true;
    return mismatch ? (kara_status_t)KARA_ERR_SCHED_MISMATCH : KARA_OK;
  });
}

kara_status_t kara_sched_tables(const kara_sched_t* s, const int32_t** block_table, const int32_t** seq_lens) {
  return guarded([&]() -> kara_status_t {
    if (!s || !block_table || !seq_lens) return KARA_ERR_INVALID_ARG;
    *block_table = s->table.data();
    *seq_lens = s->lens.data();
    return KARA_OK;
  });
}

kara_status_t kara_sched_stats(const kara_sched_t* s, kara_sched_stats_t* out) {
  return guarded([&]() -> kara_status_t {
    if (!s || !out) return KARA_ERR_INVALID_ARG;
    *out = s->st;
    out->running = (int32_t)s->running.size();
    out->waiting = (int32_t)s->waiting.size();
    out->free_pages = (int32_t)s->free_pages.size();
    out->pages_in_use = s->cfg.num_pages - out->free_pages;
    return KARA_OK;
  });
}

kara_status_t kara_sched_request(const kara_sched_t* s, int64_t id, kara_sched_request_info_t* out) {
  return guarded([&]() -> kara_status_t {
    if (!s || !out || id < 0 || id >= (int64_t)s->reqs.size()) return KARA_ERR_INVALID_ARG;
    const Request& r = s->reqs[(size_t)id];
    out->state = r.state;
    out->slot = r.slot;
    out->len = r.slot >= 0 ? s->lens[(size_t)r.slot] : 0;
    out->win_start = r.slot >= 0 ? s->p0[(size_t)r.slot] : 0;
    out->generated = r.generated;
    out->compressions = r.compressions;
    out->preemptions = r.preemptions;
    return KARA_OK;
  });
}

}  // extern "C"
