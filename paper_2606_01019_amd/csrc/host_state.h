// Host-side state of a KV cache: the page pool, per-sequence page lists and
// the verify/commit state machine.  Pure C++ (no HIP), so it can be built and
// tested without a GPU.
//
// A sequence holds its committed prefix as ctx (tokens whose K/V is cached,
// positions 0..ctx-1) plus the pending token (the last committed token, whose
// K/V the next verify writes at position ctx).  A verify of k draft tokens
// needs K/V slots for positions 0..ctx+k; commit keeps ctx' = ctx + keep + 1
// cached positions and the pages covering positions 0..ctx' (room for the new
// pending token); pages wholly past that return to the pool.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

namespace hvd {

enum HostStatus { HS_OK = 0, HS_ARG = -1, HS_STATE = -2, HS_OOM = -3, HS_RANGE = -4 };

struct PageUpdate {
  int32_t slot, index, page;
};

struct SeqSlot {
  bool live = false;
  int32_t ctx = 0;
  int32_t pending = 0;
  std::vector<int32_t> pages;
  // last verify, waiting for commit
  bool verify_pending = false;
  int32_t k = 0, accepted = 0, next = 0;
  std::vector<int32_t> draft;
  // inside a device-resident verify loop: ctx and pending live on the device
  // until the loop ends, so every host-side call on the sequence is refused
  bool in_async = false;
};

class HostState {
 public:
  HostState(int32_t max_seqs, int32_t n_pages, int32_t page_size, int32_t max_pos, int32_t max_draft,
            int32_t vocab);

  int32_t max_seqs() const { return (int32_t)seqs_.size(); }
  int32_t pages_per_seq() const { return pages_per_seq_; }
  int32_t free_pages() const { return (int32_t)free_.size(); }
  const SeqSlot& seq(int32_t id) const { return seqs_[id]; }
  const std::string& error() const { return err_; }

  // Start a sequence from a prompt of n >= 1 tokens (pages for positions
  // 0..n-1 are reserved: the prompt body plus the pending token).
  int begin_prefill(int32_t id, const int32_t* tokens, int32_t n);
  // Undo a begin_prefill whose device work failed.
  void abort_prefill(int32_t id);

  // Validate a verify batch and reserve the pages it needs (all or nothing).
  int begin_verify(int32_t batch, const int32_t* ids, const int32_t* ctx_lens, const int32_t* draft,
                   const int32_t* draft_lens);
  // Record the device results of a verify begun with begin_verify.
  void finish_verify(int32_t batch, const int32_t* ids, const int32_t* draft, const int32_t* draft_lens,
                     const int32_t* accepted, const int32_t* next);
  // Undo a begin_verify whose device work failed (releases extra pages).
  void abort_verify(int32_t batch, const int32_t* ids);

  int commit(int32_t batch, const int32_t* ids, const int32_t* keep);

  // Device-resident loop of up to max_steps verify+commit steps with fixed
  // draft lengths: validate, and reserve the pages of the longest possible
  // outcome (every draft accepted), ctx + max_steps * (k + 1) positions plus
  // the pending token's (all or nothing).
  int begin_async(int32_t batch, const int32_t* ids, const int32_t* ctx_lens, const int32_t* draft_lens,
                  int32_t max_steps);
  // Loop ended: take the device's ctx and pending tokens, release the pages
  // past the new pending position.
  void end_async(int32_t batch, const int32_t* ids, const int32_t* ctx, const int32_t* pending);
  int truncate(int32_t id, int32_t new_ctx, int32_t pending);
  int free_seq(int32_t id);

  // Page-table entries changed since the last call (slot, index, page).
  std::vector<PageUpdate> take_updates();

 private:
  int fail(int code, const std::string& msg);
  int32_t pages_for(int32_t positions) const { return (positions + page_size_ - 1) / page_size_; }
  void shrink_to(int32_t id, int32_t n_pages);
  bool grow_to(int32_t id, int32_t n_pages);

  std::vector<SeqSlot> seqs_;
  std::vector<int32_t> free_;
  std::vector<PageUpdate> updates_;
  int32_t page_size_, max_pos_, max_draft_, vocab_, pages_per_seq_;
  std::string err_;
};

}  // namespace hvd
