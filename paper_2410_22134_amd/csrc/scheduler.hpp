// Copy scheduler of the expert cache: the physical side of the prefetcher
// (ProMoE Sec. "Coordination of Prefetching and Inference": a task queue with
// two priorities served by a worker; "Chunked Prefetching": one task per
// expert matrix; "Early Preemption": a route drops the layer's pending
// low-priority tasks; Alg. 1 and Alg. 2).
//
// The logical state (which expert owns which slot, LRU order, counters) is
// decided on the device by the plan kernels.  This class only tracks what has
// been copied into each slot and issues copies, one FIFO queue, so that:
//   * high-priority copies are issued at once, in the order the route returns;
//   * low-priority copies are issued one sub-copy at a time, at most `window`
//     low-priority sub-copies in flight, so a high-priority copy waits for at
//     most `window` of them; high-priority copies in flight do not hold them
//     back (a prefetch then queues right behind the misses, keeping the link
//     busy through the compute that follows);
//   * a copy into a slot waits for the last compute that read the slot
//     (write-after-read), and compute waits for the copy of the chunk it reads
//     (read-after-write) -- see ready_seq();
//   * copies into a slot go to one engine queue while any of them may be in
//     flight (a slot refilled with nothing in flight moves to the queue with
//     the fewest bytes outstanding), so copies into one slot never overtake
//     each other and the latest copy of a slot completes after all earlier
//     ones (the engine may run several queues at once).
//
// No HIP here: the physical queue is a CopyEngine (HIP streams and events in
// the library, a simulated clock in the CPU tests).  Not thread-safe; the
// owner serialises calls.
#pragma once

#include <cstddef>
#include <cstdint>
#include <climits>
#include <deque>
#include <vector>

namespace promoe {

class CopyEngine {
 public:
  virtual ~CopyEngine() = default;
  // Enqueue copy number `seq` (consecutive from 0) on ordered queue `queue`
  // (< queues()): wait for compute token `after_compute` (-1 none), then copy
  // `bytes` from src to dst.  Copies of one queue complete in issue order;
  // copies of different queues may overlap.
  virtual void issue(int64_t seq, void* dst, const void* src, size_t bytes, int64_t after_compute, int queue) = 0;
  virtual int queues() const { return 1; }
  virtual bool done(int64_t seq) = 0;  // non-blocking completion test
  virtual void wait(int64_t seq) = 0;  // block until copy `seq` completed
  // Most copies that may be in flight at once (bounded by the engine's event ring).
  virtual int64_t capacity() const { return INT64_MAX; }
};

enum Prio { LOW = 0, HIGH = 1 };

struct PhysStats {
  int64_t copies[2] = {0, 0};
  int64_t bytes[2] = {0, 0};
  int64_t low_purged = 0;
  int64_t deferred = 0;
};

class Prefetcher {
 public:
  static constexpr int kChunks = 3;

  // high_merge_bytes > 0: high-priority copies of a slot coalesce contiguous
  // pending sub-copies into copies of up to that many bytes (nothing preempts
  // them, and larger DMA transfers run closer to the link rate).
  Prefetcher(int n_layers, int slots, int n_experts, size_t chunk_bytes, size_t sub_bytes, int window,
             uint8_t* cache_base, CopyEngine* engine, size_t high_merge_bytes = 0);

  void set_host(int layer, int expert, const uint8_t* p);
  const uint8_t* host(int layer, int expert) const { return host_[layer * E_ + expert]; }

  // A plan gave `slot` of `layer` to `expert`: forget the old contents and
  // cancel queued copies aimed at the slot.
  void assign(int layer, int slot, int expert);
  // Warm start: the slot already holds the expert's bytes.
  void mark_resident(int layer, int slot, int expert);

  // Queue the slot's chunks that are neither copied, in flight nor queued, at
  // low priority (Alg. 2 PushPredictedExperts: chunks from ready_chunk on).
  void push_low(int layer, int slot);
  // Drop the layer's queued low-priority work (early preemption).
  void purge_low(int layer);
  // Issue every remaining sub-copy of the slot's chunks now, high priority.
  void issue_high(int layer, int slot);
  // Issue the slot's chunks at high priority after compute token `after`.
  void issue_high_after(int layer, int slot, int64_t after_compute);

  // Without chunked prefetching a low-priority task is the whole expert: once
  // started, every pending sub-copy of the slot is issued at once (so a
  // high-priority copy may wait for a whole expert).
  void set_whole_expert_low(bool on) { whole_low_ = on; }

  // Issue low-priority sub-copies while fewer than `window` of them are in
  // flight.  Returns the number of tasks started.
  int pump();
  // Note completed copies (in FIFO order).
  void retire();

  bool has_low() const { return !low_.empty(); }
  // Bytes issued and not yet known complete, plus the bytes of queued
  // low-priority tasks: what the link must still carry before anything new.
  int64_t pending_bytes() const;
  int64_t in_flight() const { return next_seq_ - retired_; }
  int64_t low_in_flight() const { return low_in_flight_; }
  int64_t oldest_in_flight() const { return retired_ < next_seq_ ? retired_ : -1; }
  int64_t issued() const { return next_seq_; }
  int window() const { return window_; }

  // Copy sequence number that a reader of chunks [0, upto] of the slot must
  // wait for (on the slot's queue), -1 if they are all known complete, or -2 if
  // some sub-copy has not been issued yet.
  int64_t ready_seq(int layer, int slot, int upto_chunk) const;
  // Record that compute token `tok` reads the slot.
  void set_last_read(int layer, int slot, int64_t tok);
  int expert_in(int layer, int slot) const { return slot_(layer, slot).expert; }
  // Engine queue of the copies into the slot.  A slot keeps its queue while any
  // copy into it may be in flight (so copies into one slot stay ordered); when
  // it is given a new expert with nothing in flight it moves to the queue with
  // the fewest bytes outstanding, so fills spread over the queues and the link
  // never waits on one queue's per-copy gap while another has work.
  int queue_of(int layer, int slot) const {
    const int q = slot_(layer, slot).queue;
    return q >= 0 ? q : (layer * C_ + slot) % eng_->queues();
  }

  const PhysStats& stats() const { return st_; }
  void reset_stats() { st_ = PhysStats(); }
  int subs_per_chunk() const { return n_sub_; }

 private:
  struct Chunk {
    int n_issued = 0;    // sub-copies issued
    int64_t last = -1;   // seq of the latest issued sub-copy
    bool queued = false; // a low-priority task for it is queued
  };
  struct Slot {
    int expert = -1;
    int queue = -1;  // engine queue (-1: not chosen yet)
    int64_t last_read = -1;
    int64_t last_copy = -1;  // seq of the latest copy into the slot, whichever expert it carried
    Chunk ch[kChunks];
  };
  struct InFlight {
    uint8_t prio, queue;
    int64_t bytes;
  };
  struct LowTask {
    int layer, slot, chunk, expert;
  };

  Slot& slot_(int l, int s) { return slots_[l * C_ + s]; }
  const Slot& slot_(int l, int s) const { return slots_[l * C_ + s]; }
  void issue_sub(int layer, int slot, int chunk, Prio prio, int64_t after_compute);
  void note_issued(Prio prio, int queue, int64_t bytes);
  int pick_queue();
  // Issue every pending sub-copy of the slot (coalesced when merge_ > 0),
  // dropping its queued low-priority tasks.
  void issue_pending(int layer, int slot, int64_t after_compute, Prio prio);

  int L_, C_, E_;
  size_t chunk_bytes_, sub_bytes_;
  int n_sub_, window_;
  size_t merge_;
  bool whole_low_ = false;
  uint8_t* cache_;
  CopyEngine* eng_;
  std::vector<const uint8_t*> host_;
  std::vector<Slot> slots_;
  std::deque<LowTask> low_;
  int64_t next_seq_ = 0;
  int64_t retired_ = 0;  // copies [0, retired_) are known complete
  std::deque<InFlight> inflight_;  // each copy in [retired_, next_seq_)
  std::vector<int64_t> q_bytes_;   // bytes in flight per engine queue
  int q_next_ = 0;                 // tie-break rotation for pick_queue
  int64_t low_in_flight_ = 0;
  PhysStats st_;
};

// ---- launch order of one FFN call (host logic, no HIP) ----

// A route position whose copies wait for an earlier position's compute.
struct FillWait {
  int pos;    // the waiting position
  int after;  // position whose launch must precede its copies (-1: none)
  bool fill;  // the position's slot changes expert (a write after read)
};

// The resident readers of the victim slots of the first `max_head` fills, in
// fill order, each once: positions that a fill waits for, skipping positions
// that wait themselves (listed in `waits`, or arriving[p]: chunks still being
// copied).  Launching them first starts the link on those fills.
std::vector<int> head_readers(const std::vector<FillWait>& waits, const std::vector<char>& arriving, int max_head);

// Launch groups for the resident positions `ready` (route order) of a step
// larger than decode: groups of `group` positions up to the last one a fill
// waits for, so those fills are released group by group; then every later
// position in one group (they release nothing).
std::vector<std::vector<int>> resident_groups(const std::vector<int>& ready, const std::vector<FillWait>& waits,
                                              int group);

}  // namespace promoe
