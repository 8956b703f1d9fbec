// Host-only C entry points over HostState, built with the system C++ compiler
// (no HIP) so the page allocator and verify/commit state machine can be
// tested on a machine without a GPU.
#include <stdint.h>

#include <cstring>

#include "host_state.h"

using hvd::HostState;

extern "C" {

void* hvdh_create(int32_t max_seqs, int32_t n_pages, int32_t max_pos, int32_t max_draft, int32_t vocab) {
  return new HostState(max_seqs, n_pages, 16, max_pos, max_draft, vocab);
}
void hvdh_destroy(void* h) { delete (HostState*)h; }
int hvdh_prefill(void* h, int32_t id, const int32_t* toks, int32_t n) { return ((HostState*)h)->begin_prefill(id, toks, n); }
int hvdh_begin_verify(void* h, int32_t batch, const int32_t* ids, const int32_t* ctx, const int32_t* draft,
                      const int32_t* lens) {
  return ((HostState*)h)->begin_verify(batch, ids, ctx, draft, lens);
}
void hvdh_finish_verify(void* h, int32_t batch, const int32_t* ids, const int32_t* draft, const int32_t* lens,
                        const int32_t* acc, const int32_t* next) {
  ((HostState*)h)->finish_verify(batch, ids, draft, lens, acc, next);
}
void hvdh_abort_verify(void* h, int32_t batch, const int32_t* ids) { ((HostState*)h)->abort_verify(batch, ids); }
int hvdh_commit(void* h, int32_t batch, const int32_t* ids, const int32_t* keep) {
  return ((HostState*)h)->commit(batch, ids, keep);
}
int hvdh_begin_async(void* h, int32_t batch, const int32_t* ids, const int32_t* ctx, const int32_t* lens,
                     int32_t max_steps) {
  return ((HostState*)h)->begin_async(batch, ids, ctx, lens, max_steps);
}
void hvdh_end_async(void* h, int32_t batch, const int32_t* ids, const int32_t* ctx, const int32_t* pend) {
  ((HostState*)h)->end_async(batch, ids, ctx, pend);
}
int hvdh_truncate(void* h, int32_t id, int32_t ctx, int32_t pend) { return ((HostState*)h)->truncate(id, ctx, pend); }
int hvdh_free_seq(void* h, int32_t id) { return ((HostState*)h)->free_seq(id); }
int32_t hvdh_free_pages(void* h) { return ((HostState*)h)->free_pages(); }
// ctx, pending, verify_pending, number of pages; -1 if not live
int hvdh_seq(void* h, int32_t id, int32_t* out4) {
  const HostState* s = (const HostState*)h;
  if (id < 0 || id >= s->max_seqs() || !s->seq(id).live) return -1;
  const auto& q = s->seq(id);
  out4[0] = q.ctx;
  out4[1] = q.pending;
  out4[2] = q.verify_pending ? 1 : 0;
  out4[3] = (int32_t)q.pages.size();
  return 0;
}
// copies up to cap page ids of seq id; returns the count
int32_t hvdh_pages(void* h, int32_t id, int32_t* out, int32_t cap) {
  const auto& q = ((HostState*)h)->seq(id);
  int32_t n = (int32_t)q.pages.size();
  for (int32_t i = 0; i < n && i < cap; ++i) out[i] = q.pages[i];
  return n;
}
const char* hvdh_error(void* h) { return ((HostState*)h)->error().c_str(); }
}
