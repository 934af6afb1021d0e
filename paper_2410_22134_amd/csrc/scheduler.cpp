#include "scheduler.hpp"

#include <algorithm>

namespace promoe {

Prefetcher::Prefetcher(int n_layers, int slots, int n_experts, size_t chunk_bytes, size_t sub_bytes,
                       int window, uint8_t* cache_base, CopyEngine* engine, size_t high_merge_bytes)
    : L_(n_layers), C_(slots), E_(n_experts), chunk_bytes_(chunk_bytes),
      sub_bytes_(std::min(sub_bytes, chunk_bytes)), window_(window < 1 ? 1 : window), merge_(high_merge_bytes),
      cache_(cache_base), eng_(engine), host_((size_t)n_layers * n_experts, nullptr),
      slots_((size_t)n_layers * slots) {
  n_sub_ = (int)((chunk_bytes_ + sub_bytes_ - 1) / sub_bytes_);
}

void Prefetcher::set_host(int layer, int expert, const uint8_t* p) { host_[layer * E_ + expert] = p; }

int64_t Prefetcher::pending_bytes() const {
  int64_t b = 0;
  for (int64_t q : q_bytes_) b += q;
  for (const LowTask& t : low_) b += (int64_t)chunk_bytes_ - (int64_t)slot_(t.layer, t.slot).ch[t.chunk].n_issued * (int64_t)sub_bytes_;
  return b;
}

void Prefetcher::assign(int layer, int slot, int expert) {
  Slot& s = slot_(layer, slot);
  // cancel queued low-priority work aimed at this slot (it belongs to the old expert)
  for (auto it = low_.begin(); it != low_.end();) {
    if (it->layer == layer && it->slot == slot) it = low_.erase(it);
    else ++it;
  }
  // an earlier copy into the slot may still be in flight (also one of an owner
  // before the current one, whose chunk records were reset when it was evicted)
  if (s.last_copy < retired_) s.queue = pick_queue();
  s.expert = expert;
  for (auto& c : s.ch) c = Chunk();
}

int Prefetcher::pick_queue() {
  const int nq = eng_->queues();
  if ((int)q_bytes_.size() < nq) q_bytes_.resize(nq, 0);
  int best = q_next_ % nq;
  for (int i = 1; i < nq; ++i) {
    const int q = (q_next_ + i) % nq;
    if (q_bytes_[q] < q_bytes_[best]) best = q;
  }
  q_next_ = best + 1;
  return best;
}

void Prefetcher::mark_resident(int layer, int slot, int expert) {
  assign(layer, slot, expert);
  for (auto& c : slot_(layer, slot).ch) {
    c.n_issued = n_sub_;
    c.last = -1;
  }
}

void Prefetcher::push_low(int layer, int slot) {
  Slot& s = slot_(layer, slot);
  if (s.expert < 0) return;
  for (int c = 0; c < kChunks; ++c) {
    Chunk& ch = s.ch[c];
    if (ch.queued || ch.n_issued == n_sub_) continue;  // dedupe: queued, in flight or copied
    ch.queued = true;
    low_.push_back(LowTask{layer, slot, c, s.expert});
  }
}

void Prefetcher::purge_low(int layer) {
  for (auto it = low_.begin(); it != low_.end();) {
    if (it->layer == layer) {
      Chunk& ch = slot_(it->layer, it->slot).ch[it->chunk];
      st_.low_purged += n_sub_ - ch.n_issued;
      ch.queued = false;
      it = low_.erase(it);
    } else {
      ++it;
    }
  }
}

void Prefetcher::issue_sub(int layer, int slot, int chunk, Prio prio, int64_t after_compute) {
  Slot& s = slot_(layer, slot);
  Chunk& ch = s.ch[chunk];
  const size_t off = (size_t)ch.n_issued * sub_bytes_;
  const size_t bytes = std::min(sub_bytes_, chunk_bytes_ - off);
  const size_t slot_off = ((size_t)layer * C_ + slot) * (kChunks * chunk_bytes_) + chunk * chunk_bytes_ + off;
  const uint8_t* src = host_[layer * E_ + s.expert] + chunk * chunk_bytes_ + off;
  // write-after-read: the fill must follow every compute that read the old contents
  int64_t after = std::max(after_compute, s.last_read);
  while (next_seq_ - retired_ >= eng_->capacity()) {  // keep the engine's event ring from wrapping
    eng_->wait(retired_);
    retire();
  }
  int64_t seq = next_seq_++;
  const int q = queue_of(layer, slot);
  note_issued(prio, q, (int64_t)bytes);
  eng_->issue(seq, cache_ + slot_off, src, bytes, after, q);
  ch.n_issued++;
  ch.last = seq;
  s.last_copy = seq;
  st_.copies[prio]++;
  st_.bytes[prio] += (int64_t)bytes;
}

void Prefetcher::issue_pending(int layer, int slot, int64_t after_compute, Prio prio) {
  Slot& s = slot_(layer, slot);
  const size_t expert_bytes = kChunks * chunk_bytes_;
  bool first = true;
  for (int c = 0; c < kChunks;) {
    Chunk& ch = s.ch[c];
    if (ch.queued) {  // promote: drop the queued low-priority task for this chunk
      for (auto it = low_.begin(); it != low_.end(); ++it)
        if (it->layer == layer && it->slot == slot && it->chunk == c) { low_.erase(it); break; }
      ch.queued = false;
    }
    if (ch.n_issued == n_sub_) { ++c; continue; }
    if (merge_ == 0) {
      issue_sub(layer, slot, c, prio, first ? after_compute : -1);
      first = false;
      continue;
    }
    // one copy from the first pending byte of chunk c over every following pending
    // sub-copy that is contiguous with it (a later chunk joins only if none of it
    // was issued yet), in whole sub-copies, up to merge_ bytes
    const size_t start = (size_t)c * chunk_bytes_ + (size_t)ch.n_issued * sub_bytes_;
    size_t end = start;
    for (int cc = c; cc < kChunks; ++cc) {
      Chunk& k = s.ch[cc];
      if (k.n_issued == n_sub_) break;
      if (k.queued) {
        for (auto it = low_.begin(); it != low_.end(); ++it)
          if (it->layer == layer && it->slot == slot && it->chunk == cc) { low_.erase(it); break; }
        k.queued = false;
      }
      const size_t cend = (size_t)(cc + 1) * chunk_bytes_;
      const size_t cstart = (size_t)cc * chunk_bytes_ + (size_t)k.n_issued * sub_bytes_;
      if (cstart != end) break;  // not contiguous with the run
      const size_t budget = start + merge_ - end;
      size_t take = cend - cstart;
      if (take > budget) {
        take = budget / sub_bytes_ * sub_bytes_;
        if (take == 0) {
          if (end != start) break;
          take = std::min(sub_bytes_, cend - cstart);
        }
        end = cstart + take;
        break;
      }
      end = cend;
    }
    const int64_t after = std::max(first ? after_compute : -1, s.last_read);
    while (next_seq_ - retired_ >= eng_->capacity()) {
      eng_->wait(retired_);
      retire();
    }
    const int64_t seq = next_seq_++;
    const int q = queue_of(layer, slot);
    note_issued(prio, q, (int64_t)(end - start));
    const size_t slot_off = ((size_t)layer * C_ + slot) * expert_bytes;
    eng_->issue(seq, cache_ + slot_off + start, host_[layer * E_ + s.expert] + start, end - start, after, q);
    s.last_copy = seq;
    st_.copies[prio]++;
    st_.bytes[prio] += (int64_t)(end - start);
    first = false;
    // mark the covered sub-copies of every chunk in [start, end)
    for (int k = 0; k < kChunks; ++k) {
      const size_t c0 = (size_t)k * chunk_bytes_;
      if (end <= c0 || start >= c0 + chunk_bytes_) continue;
      Chunk& kk = s.ch[k];
      const size_t upto = std::min(end, c0 + chunk_bytes_) - c0;
      const int n_done = upto >= chunk_bytes_ ? n_sub_ : (int)(upto / sub_bytes_);
      if (n_done > kk.n_issued) {
        kk.n_issued = n_done;
        kk.last = seq;
      }
    }
  }
}

void Prefetcher::issue_high(int layer, int slot) {
  if (slot_(layer, slot).expert < 0) return;
  issue_pending(layer, slot, -1, HIGH);
}

void Prefetcher::issue_high_after(int layer, int slot, int64_t after_compute) {
  Slot& s = slot_(layer, slot);
  if (s.expert < 0) return;
  st_.deferred++;
  issue_pending(layer, slot, after_compute, HIGH);
}

int Prefetcher::pump() {
  int n = 0;
  retire();
  while (!low_.empty() && low_in_flight_ < window_) {
    LowTask t = low_.front();
    Slot& s = slot_(t.layer, t.slot);
    Chunk& ch = s.ch[t.chunk];
    if (s.expert != t.expert || ch.n_issued == n_sub_) {  // stale or already served
      ch.queued = false;
      low_.pop_front();
      continue;
    }
    if (whole_low_) {  // drops every queued task of the slot, this one included
      issue_pending(t.layer, t.slot, -1, LOW);
      ++n;
      continue;
    }
    issue_sub(t.layer, t.slot, t.chunk, LOW, -1);
    ++n;
    if (ch.n_issued == n_sub_) {
      ch.queued = false;
      low_.pop_front();
    }
  }
  return n;
}

void Prefetcher::note_issued(Prio prio, int queue, int64_t bytes) {
  inflight_.push_back(InFlight{(uint8_t)prio, (uint8_t)queue, bytes});
  if ((int)q_bytes_.size() <= queue) q_bytes_.resize(queue + 1, 0);
  q_bytes_[queue] += bytes;
  if (prio == LOW) ++low_in_flight_;
}

void Prefetcher::retire() {
  while (retired_ < next_seq_ && eng_->done(retired_)) {
    const InFlight& f = inflight_.front();
    if (f.prio == LOW) --low_in_flight_;
    q_bytes_[f.queue] -= f.bytes;
    inflight_.pop_front();
    ++retired_;
  }
}

int64_t Prefetcher::ready_seq(int layer, int slot, int upto_chunk) const {
  const Slot& s = slot_(layer, slot);
  int64_t need = -1;
  for (int c = 0; c <= upto_chunk; ++c) {
    const Chunk& ch = s.ch[c];
    if (ch.n_issued < n_sub_) return -2;
    if (ch.last >= retired_) need = std::max(need, ch.last);
  }
  return need;
}

void Prefetcher::set_last_read(int layer, int slot, int64_t tok) {
  Slot& s = slot_(layer, slot);
  s.last_read = std::max(s.last_read, tok);
}

std::vector<int> head_readers(const std::vector<FillWait>& waits, const std::vector<char>& arriving, int max_head) {
  std::vector<int> head;
  for (const auto& w : waits) {
    if ((int)head.size() >= max_head) break;
    if (w.after < 0 || !w.fill) continue;
    const int p = w.after;
    bool busy = p < (int)arriving.size() && arriving[p];
    for (const auto& o : waits) busy = busy || o.pos == p;
    if (busy || std::find(head.begin(), head.end(), p) != head.end()) continue;
    head.push_back(p);
  }
  return head;
}

std::vector<std::vector<int>> resident_groups(const std::vector<int>& ready, const std::vector<FillWait>& waits,
                                              int group) {
  size_t last = 0;  // one past the last ready position a fill waits for
  for (const auto& w : waits)
    for (size_t i = 0; i < ready.size(); ++i)
      if (ready[i] == w.after) last = std::max(last, i + 1);
  std::vector<std::vector<int>> out;
  const size_t g = group < 1 ? 1 : (size_t)group;
  for (size_t g0 = 0; g0 < ready.size();) {
    const size_t g1 = g0 < last ? std::min(ready.size(), g0 + g) : ready.size();
    out.emplace_back(ready.begin() + g0, ready.begin() + g1);
    g0 = g1;
  }
  return out;
}

}  // namespace promoe
