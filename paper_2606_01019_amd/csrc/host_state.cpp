#include "host_state.h"

#include <algorithm>
#include <set>

namespace hvd {

HostState::HostState(int32_t max_seqs, int32_t n_pages, int32_t page_size, int32_t max_pos,
                     int32_t max_draft, int32_t vocab)
    : seqs_(max_seqs), page_size_(page_size), max_pos_(max_pos), max_draft_(max_draft), vocab_(vocab) {
  pages_per_seq_ = pages_for(max_pos + 1);
  free_.reserve(n_pages);
  // Hand out low page ids first (free list used as a stack).
  for (int32_t p = n_pages - 1; p >= 0; --p) free_.push_back(p);
}

int HostState::fail(int code, const std::string& msg) {
  err_ = msg;
  return code;
}

void HostState::shrink_to(int32_t id, int32_t n) {
  SeqSlot& s = seqs_[id];
  while ((int32_t)s.pages.size() > n) {
    free_.push_back(s.pages.back());
    s.pages.pop_back();
  }
}

bool HostState::grow_to(int32_t id, int32_t n) {
  SeqSlot& s = seqs_[id];
  int32_t need = n - (int32_t)s.pages.size();
  if (need <= 0) return true;
  if ((int32_t)free_.size() < need) return false;
  for (int32_t i = 0; i < need; ++i) {
    int32_t p = free_.back();
    free_.pop_back();
    updates_.push_back({id, (int32_t)s.pages.size(), p});
    s.pages.push_back(p);
  }
  return true;
}

int HostState::begin_prefill(int32_t id, const int32_t* tokens, int32_t n) {
  if (id < 0 || id >= max_seqs()) return fail(HS_ARG, "seq_id out of range");
  if (seqs_[id].live) return fail(HS_ARG, "seq_id already in use");
  if (n < 1 || tokens == nullptr) return fail(HS_ARG, "prefill needs n >= 1 tokens");
  if (n - 1 >= max_pos_) return fail(HS_RANGE, "prompt longer than the rotary table");
  for (int32_t i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= vocab_) return fail(HS_RANGE, "token id outside [0, vocab)");
  int32_t need = pages_for(n);
  if ((int32_t)free_.size() < need) return fail(HS_OOM, "page pool exhausted");
  SeqSlot& s = seqs_[id];
  s = SeqSlot();
  s.live = true;
  grow_to(id, need);
  s.ctx = n - 1;
  s.pending = tokens[n - 1];
  return HS_OK;
}

void HostState::abort_prefill(int32_t id) {
  shrink_to(id, 0);
  seqs_[id] = SeqSlot();
}

int HostState::begin_verify(int32_t batch, const int32_t* ids, const int32_t* ctx_lens, const int32_t* draft,
                            const int32_t* draft_lens) {
  if (batch < 1 || batch > max_seqs()) return fail(HS_ARG, "batch must be in [1, max_seqs]");
  if (!ids || !ctx_lens || !draft_lens) return fail(HS_ARG, "null argument");
  std::set<int32_t> seen;
  int64_t off = 0;
  int64_t extra_pages = 0;
  for (int32_t b = 0; b < batch; ++b) {
    int32_t id = ids[b];
    if (id < 0 || id >= max_seqs() || !seqs_[id].live) return fail(HS_ARG, "unknown seq_id");
    if (!seen.insert(id).second) return fail(HS_ARG, "duplicate seq_id in batch");
    const SeqSlot& s = seqs_[id];
    if (s.in_async) return fail(HS_STATE, "sequence is in a device-resident verify loop");
    if (s.verify_pending) return fail(HS_STATE, "previous verify not committed");
    if (ctx_lens[b] != s.ctx) return fail(HS_STATE, "ctx_lens disagrees with the library");
    int32_t k = draft_lens[b];
    if (k < 0 || k > max_draft_) return fail(HS_RANGE, "draft length outside [0, max_draft]");
    if ((int64_t)s.ctx + k >= max_pos_) return fail(HS_RANGE, "position beyond the rotary table");
    if (k > 0 && !draft) return fail(HS_ARG, "null draft_tokens");
    for (int32_t i = 0; i < k; ++i) {
      int32_t t = draft[off + i];
      if (t < 0 || t >= vocab_) return fail(HS_RANGE, "token id outside [0, vocab)");
    }
    off += k;
    int32_t need = pages_for(s.ctx + k + 1);
    extra_pages += std::max<int32_t>(0, need - (int32_t)s.pages.size());
  }
  if (extra_pages > (int64_t)free_.size()) return fail(HS_OOM, "page pool exhausted");
  for (int32_t b = 0; b < batch; ++b) {
    int32_t id = ids[b];
    grow_to(id, pages_for(seqs_[id].ctx + draft_lens[b] + 1));
  }
  return HS_OK;
}

void HostState::finish_verify(int32_t batch, const int32_t* ids, const int32_t* draft, const int32_t* draft_lens,
                              const int32_t* accepted, const int32_t* next) {
  int64_t off = 0;
  for (int32_t b = 0; b < batch; ++b) {
    SeqSlot& s = seqs_[ids[b]];
    int32_t k = draft_lens[b];
    s.verify_pending = true;
    s.k = k;
    s.accepted = accepted[b];
    s.next = next[b];
    s.draft.assign(draft + off, draft + off + k);
    off += k;
  }
}

void HostState::abort_verify(int32_t batch, const int32_t* ids) {
  for (int32_t b = 0; b < batch; ++b) {
    SeqSlot& s = seqs_[ids[b]];
    shrink_to(ids[b], pages_for(s.ctx + 1));
  }
}

int HostState::commit(int32_t batch, const int32_t* ids, const int32_t* keep) {
  if (batch < 1 || batch > max_seqs() || !ids) return fail(HS_ARG, "bad batch");
  std::set<int32_t> seen;
  for (int32_t b = 0; b < batch; ++b) {
    int32_t id = ids[b];
    if (id < 0 || id >= max_seqs() || !seqs_[id].live) return fail(HS_ARG, "unknown seq_id");
    if (!seen.insert(id).second) return fail(HS_ARG, "duplicate seq_id in batch");
    const SeqSlot& s = seqs_[id];
    if (s.in_async) return fail(HS_STATE, "sequence is in a device-resident verify loop");
    if (!s.verify_pending) return fail(HS_STATE, "commit without a verify");
    if (keep && (keep[b] < 0 || keep[b] > s.accepted)) return fail(HS_ARG, "keep outside [0, accepted]");
  }
  for (int32_t b = 0; b < batch; ++b) {
    SeqSlot& s = seqs_[ids[b]];
    int32_t kp = keep ? keep[b] : s.accepted;
    int32_t pend = kp < s.accepted ? s.draft[kp] : s.next;
    s.ctx += kp + 1;
    s.pending = pend;
    s.verify_pending = false;
    s.draft.clear();
    shrink_to(ids[b], pages_for(s.ctx + 1));
  }
  return HS_OK;
}

int HostState::begin_async(int32_t batch, const int32_t* ids, const int32_t* ctx_lens, const int32_t* draft_lens,
                           int32_t max_steps) {
  if (batch < 1 || batch > max_seqs()) return fail(HS_ARG, "batch must be in [1, max_seqs]");
  if (!ids || !ctx_lens || !draft_lens) return fail(HS_ARG, "null argument");
  if (max_steps < 1) return fail(HS_ARG, "max_steps must be >= 1");
  std::set<int32_t> seen;
  int64_t extra_pages = 0;
  for (int32_t b = 0; b < batch; ++b) {
    int32_t id = ids[b];
    if (id < 0 || id >= max_seqs() || !seqs_[id].live) return fail(HS_ARG, "unknown seq_id");
    if (!seen.insert(id).second) return fail(HS_ARG, "duplicate seq_id in batch");
    const SeqSlot& s = seqs_[id];
    if (s.in_async) return fail(HS_STATE, "sequence is in a device-resident verify loop");
    if (s.verify_pending) return fail(HS_STATE, "previous verify not committed");
    if (ctx_lens[b] != s.ctx) return fail(HS_STATE, "ctx_lens disagrees with the library");
    const int32_t k = draft_lens[b];
    if (k < 0 || k > max_draft_) return fail(HS_RANGE, "draft length outside [0, max_draft]");
    // the last step writes positions up to ctx + max_steps * (k + 1) - 1
    const int64_t span = (int64_t)max_steps * (k + 1);
    if ((int64_t)s.ctx + span - 1 >= max_pos_) return fail(HS_RANGE, "position beyond the rotary table");
    const int64_t need = ((int64_t)s.ctx + span + 1 + page_size_ - 1) / page_size_;
    extra_pages += std::max<int64_t>(0, need - (int64_t)s.pages.size());
  }
  if (extra_pages > (int64_t)free_.size()) return fail(HS_OOM, "page pool exhausted");
  for (int32_t b = 0; b < batch; ++b) {
    SeqSlot& s = seqs_[ids[b]];
    grow_to(ids[b], pages_for(s.ctx + max_steps * (draft_lens[b] + 1) + 1));
    s.in_async = true;
  }
  return HS_OK;
}

void HostState::end_async(int32_t batch, const int32_t* ids, const int32_t* ctx, const int32_t* pending) {
  for (int32_t b = 0; b < batch; ++b) {
    SeqSlot& s = seqs_[ids[b]];
    s.in_async = false;
    s.ctx = ctx[b];
    s.pending = pending[b];
    shrink_to(ids[b], pages_for(s.ctx + 1));
  }
}

int HostState::truncate(int32_t id, int32_t new_ctx, int32_t pending) {
  if (id < 0 || id >= max_seqs() || !seqs_[id].live) return fail(HS_ARG, "unknown seq_id");
  SeqSlot& s = seqs_[id];
  if (s.in_async) return fail(HS_STATE, "sequence is in a device-resident verify loop");
  if (new_ctx < 0 || new_ctx > s.ctx) return fail(HS_ARG, "new_ctx_len outside [0, ctx_len]");
  if (pending < 0 || pending >= vocab_) return fail(HS_RANGE, "token id outside [0, vocab)");
  s.ctx = new_ctx;
  s.pending = pending;
  s.verify_pending = false;
  s.draft.clear();
  shrink_to(id, pages_for(new_ctx + 1));
  return HS_OK;
}

int HostState::free_seq(int32_t id) {
  if (id < 0 || id >= max_seqs() || !seqs_[id].live) return fail(HS_ARG, "unknown seq_id");
  if (seqs_[id].in_async) return fail(HS_STATE, "sequence is in a device-resident verify loop");
  shrink_to(id, 0);
  seqs_[id] = SeqSlot();
  return HS_OK;
}

std::vector<PageUpdate> HostState::take_updates() {
  std::vector<PageUpdate> out;
  out.swap(updates_);
  return out;
}

}  // namespace hvd
