// Explicit-release dual-pool page allocator (host).
//
// "KVCache Dual-Pool Design": the FULL pool holds every position of a sequence
// and the SWA pool only what the window needs; admission checks both
// capacities; the FULL index (logical page of a position) is authoritative and
// the SWA table maps the same logical pages to SWA pages.
// "SWA-Aware Prefix Cache Tree": out-of-window SWA pages are released when a
// prefill chunk completes, when the request ends and every N decode tokens, so
// SWA usage stays at window (or chunk) magnitude instead of growing with the
// sequence.
//
// The tables this allocator fills are the block tables of a FULL layer and of
// an HSWA_LAYER_SWA_PAGED layer: logical page i of sequence b (positions
// i*PG .. i*PG+PG-1) -> physical page, -1 where nothing is held.
#include <stdint.h>

#include <new>
#include <vector>

#include "hswa.h"

struct hswa_allocator {
  struct Seq {
    bool used = false;
    int64_t len = 0;             // positions 0 .. len-1 exist
    std::vector<int32_t> full;   // logical page -> FULL page
    std::vector<int32_t> swa;    // logical page -> SWA page or -1
    int32_t swa_lo = 0;          // no SWA page is held below this logical page
    int32_t steps = 0;           // decode steps since the last SWA release
  };
  hswa_allocator_config cfg{};
  std::vector<int32_t> free_full, free_swa;  // stacks; the back is handed out next
  std::vector<Seq> seqs;
};

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// First logical page that must stay in the SWA pool once a sequence of
// length len has been processed: the page of position len - W + 1, where the
// window of the next query (at position len) starts.
int64_t swa_keep_from(const hswa_allocator_config &c, int64_t len) {
  const int64_t first_pos = len - c.window + 1;
  return first_pos <= 0 ? 0 : first_pos / c.page_size;
}

bool valid_seq(const hswa_allocator *a, int32_t seq) {
  return a && seq >= 0 && seq < a->cfg.max_seqs && a->seqs[seq].used;
}

}  // namespace

extern "C" {

hswa_status hswa_allocator_create(const hswa_allocator_config *cfg, hswa_allocator **out) {
  if (!cfg || !out) return HSWA_ERR_INVALID_ARG;
  *out = nullptr;
  if (cfg->page_size < 1 || cfg->window < 1 || cfg->full_pages < 0 || cfg->swa_pages < 0 ||
      cfg->max_seqs < 1 || cfg->table_stride < 1 || cfg->release_every < 1 ||
      cfg->full_pages > INT32_MAX || cfg->swa_pages > INT32_MAX)
    return HSWA_ERR_INVALID_ARG;
  hswa_allocator *a = new (std::nothrow) hswa_allocator();
  if (!a) return HSWA_ERR_CAPACITY;
  try {
    a->cfg = *cfg;
    a->free_full.reserve(cfg->full_pages);
    a->free_swa.reserve(cfg->swa_pages);
    for (int64_t p = cfg->full_pages - 1; p >= 0; --p) a->free_full.push_back((int32_t)p);
    for (int64_t p = cfg->swa_pages - 1; p >= 0; --p) a->free_swa.push_back((int32_t)p);
    a->seqs.resize(cfg->max_seqs);
  } catch (...) {
    delete a;
    return HSWA_ERR_CAPACITY;
  }
  *out = a;
  return HSWA_OK;
}

void hswa_allocator_destroy(hswa_allocator *a) { delete a; }

hswa_status hswa_allocator_admit(hswa_allocator *a, int32_t seq, int64_t len, int32_t chunk) {
  if (!a || seq < 0 || seq >= a->cfg.max_seqs || len < 0 || chunk < 1) return HSWA_ERR_INVALID_ARG;
  if (a->seqs[seq].used) return HSWA_ERR_INVALID_ARG;
  const hswa_allocator_config &c = a->cfg;
  const int64_t full_need = ceil_div(len, c.page_size);
  const int64_t span = len < (int64_t)c.window + chunk ? len : (int64_t)c.window + chunk;
  const int64_t swa_need = len == 0 ? 0 : ceil_div(span, c.page_size) + 1;
  if (full_need > c.table_stride) return HSWA_ERR_CAPACITY;
  if (full_need > (int64_t)a->free_full.size() || swa_need > (int64_t)a->free_swa.size())
    return HSWA_ERR_CAPACITY;
  hswa_allocator::Seq &s = a->seqs[seq];
  s = hswa_allocator::Seq();
  s.used = true;
  return HSWA_OK;
}

hswa_status hswa_allocator_extend(hswa_allocator *a, int32_t seq, int64_t new_len) {
  if (!valid_seq(a, seq)) return HSWA_ERR_INVALID_ARG;
  hswa_allocator::Seq &s = a->seqs[seq];
  const hswa_allocator_config &c = a->cfg;
  if (new_len < s.len) return HSWA_ERR_INVALID_ARG;
  if (new_len == s.len) return HSWA_OK;
  const int64_t pages = ceil_div(new_len, c.page_size);
  if (pages > c.table_stride) return HSWA_ERR_CAPACITY;
  // FULL: every new logical page. SWA: the pages of positions
  // [max(len, new_len - W), new_len) not held yet. The last new token's query
  // (a decode step reads it back from the pool) needs keys from new_len - W
  // on, the next query from new_len - W + 1; earlier new positions are read
  // by nobody from the pool (a prefill chunk takes its own keys from its
  // inputs) and are not stored.
  const int64_t full_have = (int64_t)s.full.size();
  const int64_t lo_pos = new_len - c.window > s.len ? new_len - c.window : s.len;
  const int64_t swa_from = lo_pos / c.page_size;
  int64_t swa_new = 0;
  for (int64_t i = swa_from; i < pages; ++i)
    if (i >= (int64_t)s.swa.size() || s.swa[i] < 0) ++swa_new;
  if (pages - full_have > (int64_t)a->free_full.size() || swa_new > (int64_t)a->free_swa.size())
    return HSWA_ERR_CAPACITY;
  try {
    s.full.reserve(pages);
    s.swa.resize(pages, -1);
  } catch (...) {
    return HSWA_ERR_CAPACITY;
  }
  for (int64_t i = full_have; i < pages; ++i) {
    s.full.push_back(a->free_full.back());
    a->free_full.pop_back();
  }
  for (int64_t i = swa_from; i < pages; ++i) {
    if (s.swa[i] < 0) {
      s.swa[i] = a->free_swa.back();
      a->free_swa.pop_back();
    }
  }
  s.len = new_len;
  return HSWA_OK;
}

hswa_status hswa_allocator_step_end(hswa_allocator *a, int32_t seq, int32_t decode_step, int32_t *released) {
  if (!valid_seq(a, seq)) return HSWA_ERR_INVALID_ARG;
  hswa_allocator::Seq &s = a->seqs[seq];
  int32_t n = 0;
  bool release = true;
  if (decode_step) {
    s.steps += 1;
    release = s.steps >= a->cfg.release_every;
  }
  if (release) {
    s.steps = 0;
    const int64_t keep = swa_keep_from(a->cfg, s.len);
    for (int64_t i = s.swa_lo; i < keep && i < (int64_t)s.swa.size(); ++i) {
      if (s.swa[i] >= 0) {
        a->free_swa.push_back(s.swa[i]);
        s.swa[i] = -1;
        ++n;
      }
    }
    if (keep > s.swa_lo) s.swa_lo = (int32_t)keep;
  }
  if (released) *released = n;
  return HSWA_OK;
}

hswa_status hswa_allocator_free(hswa_allocator *a, int32_t seq) {
  if (!valid_seq(a, seq)) return HSWA_ERR_INVALID_ARG;
  hswa_allocator::Seq &s = a->seqs[seq];
  for (int32_t p : s.full) a->free_full.push_back(p);
  for (int32_t p : s.swa)
    if (p >= 0) a->free_swa.push_back(p);
  s = hswa_allocator::Seq();
  return HSWA_OK;
}

hswa_status hswa_allocator_tables(const hswa_allocator *a, int32_t *full_table, int32_t *swa_table) {
  if (!a) return HSWA_ERR_INVALID_ARG;
  const int64_t stride = a->cfg.table_stride;
  for (int32_t b = 0; b < a->cfg.max_seqs; ++b) {
    const hswa_allocator::Seq &s = a->seqs[b];
    for (int64_t i = 0; i < stride; ++i) {
      if (full_table) full_table[b * stride + i] = i < (int64_t)s.full.size() ? s.full[i] : -1;
      if (swa_table) swa_table[b * stride + i] = i < (int64_t)s.swa.size() ? s.swa[i] : -1;
    }
  }
  return HSWA_OK;
}

hswa_status hswa_allocator_usage(const hswa_allocator *a, int32_t seq, int64_t *full_used, int64_t *swa_used,
                                 int64_t *full_free, int64_t *swa_free) {
  if (!a) return HSWA_ERR_INVALID_ARG;
  int64_t fu = 0, su = 0;
  if (seq >= 0) {
    if (!valid_seq(a, seq)) return HSWA_ERR_INVALID_ARG;
    const hswa_allocator::Seq &s = a->seqs[seq];
    fu = (int64_t)s.full.size();
    for (int32_t p : s.swa) su += p >= 0;
  } else {
    fu = a->cfg.full_pages - (int64_t)a->free_full.size();
    su = a->cfg.swa_pages - (int64_t)a->free_swa.size();
  }
  if (full_used) *full_used = fu;
  if (swa_used) *swa_used = su;
  if (full_free) *full_free = (int64_t)a->free_full.size();
  if (swa_free) *swa_free = (int64_t)a->free_swa.size();
  return HSWA_OK;
}

}  // extern "C"
