// CPU tests of the copy scheduler (Prefetcher) against a copy engine with a
// simulated clock: one FIFO queue, copies take bytes / bandwidth time units,
// a copy may wait for a compute token that completes at a given time.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <random>
#include <string>
#include <vector>

#include "../../paper_2410_22134_amd/csrc/scheduler.hpp"

using namespace promoe;

namespace {

int failures = 0;
#define CHECK(cond)                                                        \
  do {                                                                     \
    if (!(cond)) {                                                         \
      std::printf("FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);          \
      ++failures;                                                          \
    }                                                                      \
  } while (0)

struct FakeEngine : CopyEngine {
  double now = 0.0;
  double bw = 1.0;  // bytes per time unit
  int64_t cap = INT64_MAX;
  struct Copy {
    double start, end;
    uint8_t* dst;
    size_t bytes;
    int64_t after;
    double issued;  // host time of the issue call
  };
  std::vector<Copy> log;
  std::map<int64_t, double> compute_done;  // compute token -> completion time
  int nq = 1;                      // queues reported to the scheduler (all run as one FIFO here)
  std::vector<int> queue_of_copy;  // queue each copy was issued on
  int queues() const override { return nq; }
  void issue(int64_t seq, void* dst, const void*, size_t bytes, int64_t after, int queue) override {
    queue_of_copy.push_back(queue);
    double start = now;
    if (!log.empty()) start = std::max(start, log.back().end);
    if (after >= 0) {
      auto it = compute_done.find(after);
      start = std::max(start, it == compute_done.end() ? 1e30 : it->second);
    }
    if ((int64_t)log.size() != seq) std::abort();
    log.push_back({start, start + (double)bytes / bw, static_cast<uint8_t*>(dst), bytes, after, now});
  }
  bool done(int64_t seq) override { return log[seq].end <= now + 1e-12; }
  void wait(int64_t seq) override { now = std::max(now, log[seq].end); }
  int64_t capacity() const override { return cap; }
  void advance(double t) { now = std::max(now, t); }
};

// Memory layout helpers: one layer, C slots, experts of 3 chunks.
struct Rig {
  FakeEngine eng;
  std::vector<uint8_t> host, cache;
  Prefetcher* pf;
  size_t chunk;
  Rig(int L, int C, int E, size_t chunk_bytes, size_t sub, int window, size_t merge = 0) : chunk(chunk_bytes) {
    host.resize((size_t)L * E * 3 * chunk_bytes);
    cache.resize((size_t)L * C * 3 * chunk_bytes);
    pf = new Prefetcher(L, C, E, chunk_bytes, sub, window, cache.data(), &eng, merge);
    for (int l = 0; l < L; ++l)
      for (int e = 0; e < E; ++e) pf->set_host(l, e, host.data() + ((size_t)l * E + e) * 3 * chunk_bytes);
  }
  ~Rig() { delete pf; }
  // start time of the first copy into (layer, slot) issued at or after log index `from`
  double first_start_into(int layer, int slot, int C, size_t from = 0) {
    uint8_t* lo = cache.data() + ((size_t)layer * C + slot) * 3 * chunk;
    for (size_t i = from; i < eng.log.size(); ++i)
      if (eng.log[i].dst >= lo && eng.log[i].dst < lo + 3 * chunk) return eng.log[i].start;
    return -1.0;
  }
  // the worker's behaviour between host events: issue, wait for the oldest, repeat, up to time t
  void worker_until(double t) {
    for (;;) {
      pf->pump();
      const int64_t o = pf->oldest_in_flight();
      if (o < 0 || eng.log[o].end > t) break;
      eng.wait(o);
      pf->retire();
    }
    eng.advance(t);
    pf->retire();
    pf->pump();
  }
};

// Chunked prefetching and early preemption, the paper's worked example
// (expert of three chunks copied at low priority; a miss arrives during the
// second chunk, or -- with early preemption -- while the first one copies).
void example(double* chunked, double* unchunked, double* early) {
  for (int variant = 0; variant < 3; ++variant) {
    const bool chunking = variant != 1;
    const size_t unit = 100;  // bytes of one matrix; bw 100 B / unit time -> 1 time unit per chunk
    Rig r(1, 4, 8, unit, unit, 1);
    r.pf->set_whole_expert_low(!chunking);  // without chunking the low task is the whole expert
    r.eng.bw = 100.0;
    r.pf->assign(0, 0, 1);  // predicted expert 1 -> slot 0
    r.pf->push_low(0, 0);
    const double miss_at = variant == 2 ? 0.5 : 1.5;  // during chunk 0 (gate end) or chunk 1 (access)
    r.worker_until(miss_at);
    const size_t mark = r.eng.log.size();
    r.pf->purge_low(0);
    r.pf->assign(0, 1, 2);  // missing expert 2 -> slot 1, high priority
    r.pf->issue_high(0, 1);
    double start = r.first_start_into(0, 1, 4, mark);
    if (variant == 0) *chunked = start;
    if (variant == 1) *unchunked = start;
    if (variant == 2) *early = start;
  }
}

void test_example() {
  double a, b, c;
  example(&a, &b, &c);
  CHECK(std::fabs(a - 2.0) < 1e-9);  // right after the second chunk
  CHECK(std::fabs(b - 3.0) < 1e-9);  // after the whole expert without chunking
  CHECK(std::fabs(c - 1.0) < 1e-9);  // early preemption: before the second chunk starts
}

// Whole-expert low-priority tasks: a started task issues all of its expert's
// sub-copies at once (past the window), coalesced when merging is on, and a
// task dropped by a route never starts.
void test_whole_expert_low() {
  for (size_t merge : {(size_t)0, (size_t)1000}) {
    Rig r(2, 4, 8, 100, 50, 1, merge);  // 2 sub-copies per chunk
    r.eng.bw = 100.0;
    r.pf->set_whole_expert_low(true);
    r.pf->assign(1, 0, 3);
    r.pf->push_low(1, 0);
    r.pf->assign(1, 1, 4);
    r.pf->push_low(1, 1);
    CHECK(r.pf->pump() == 1);                       // one task: expert 3 whole
    CHECK(r.eng.log.size() == (merge ? 1u : 6u));
    size_t bytes = 0;
    for (auto& c : r.eng.log) bytes += c.bytes;
    CHECK(bytes == 300);
    CHECK(r.pf->ready_seq(1, 0, 2) >= 0);          // every chunk issued
    CHECK(r.pf->ready_seq(1, 1, 0) == -2);         // the next task has not started
    r.pf->purge_low(1);
    CHECK(r.pf->stats().low_purged == 6);          // expert 4: 3 chunks x 2 sub-copies
    r.worker_until(100.0);
    CHECK(r.pf->stats().bytes[LOW] == 300 && r.pf->stats().copies[HIGH] == 0);
  }
}

// With several engine queues, copies into one slot stay ordered: a copy goes to
// another queue than the slot's previous copy only once that copy completed.
// Slots given new experts spread over the queues.
void test_queue_per_slot() {
  Rig r(2, 4, 8, 100, 50, 2, 1000);
  r.eng.nq = 2;
  r.eng.bw = 100.0;
  for (int s = 0; s < 4; ++s) {
    r.pf->assign(0, s, s);
    r.pf->push_low(0, s);
  }
  r.worker_until(2.0);
  r.pf->assign(0, 1, 6);  // reassign slot 1 while its old copies may be queued
  r.pf->issue_high(0, 1);
  r.pf->assign(1, 2, 5);
  r.pf->issue_high(1, 2);
  r.worker_until(100.0);
  r.pf->assign(0, 1, 7);  // everything completed: the slot may move
  r.pf->issue_high(0, 1);
  r.worker_until(200.0);
  std::map<uint8_t*, size_t> last_into;  // slot base -> index of its latest copy
  bool used[2] = {false, false};
  for (size_t i = 0; i < r.eng.log.size(); ++i) {
    const size_t off = r.eng.log[i].dst - r.cache.data();
    uint8_t* slot_base = r.cache.data() + off / (3 * r.chunk) * (3 * r.chunk);
    const int q = r.eng.queue_of_copy[i];
    CHECK(q == 0 || q == 1);
    used[q] = true;
    auto it = last_into.find(slot_base);
    if (it != last_into.end() && r.eng.queue_of_copy[it->second] != q)
      CHECK(r.eng.log[it->second].end <= r.eng.log[i].issued + 1e-12);
    last_into[slot_base] = i;
  }
  CHECK(used[0] && used[1]);
}

// A slot given a second new expert before anything was copied for the first
// keeps the queue of the copies still in flight from before: the latest expert's
// copies must not overtake them (they would land under the old bytes).
void test_queue_kept_over_uncopied_owner() {
  Rig r(1, 2, 8, 100, 50, 4, 1000);
  r.eng.nq = 2;
  r.eng.bw = 1.0;  // copies stay in flight
  r.pf->assign(0, 0, 1);
  r.pf->push_low(0, 0);
  r.pf->pump();  // expert 1's first sub-copies go out
  CHECK(r.pf->in_flight() > 0);
  const int q_old = r.eng.queue_of_copy.back();
  const size_t n_old = r.eng.log.size();
  r.pf->assign(0, 0, 2);  // queued only, never copied
  r.pf->purge_low(0);
  r.pf->assign(0, 0, 3);
  r.pf->issue_high(0, 0);
  CHECK(r.eng.log.size() > n_old);
  for (size_t i = n_old; i < r.eng.log.size(); ++i) CHECK(r.eng.queue_of_copy[i] == q_old);
}

// Fills issued one after another alternate between two queues: each goes to
// the queue with fewer bytes in flight.
void test_fills_balance_queues() {
  Rig r(1, 6, 8, 100, 100, 2, 1000);
  r.eng.nq = 2;
  r.eng.bw = 100.0;
  for (int s = 0; s < 6; ++s) {
    r.pf->assign(0, s, s);
    r.pf->issue_high(0, s);
  }
  CHECK(r.eng.log.size() == 6u);
  for (int s = 0; s < 6; ++s) CHECK(r.pf->queue_of(0, s) == s % 2);
  for (size_t i = 0; i < r.eng.log.size(); ++i) CHECK(r.eng.queue_of_copy[i] == (int)(i % 2));
}

// Launch order of a large step.  Fills wait for the resident experts whose
// slots they take (position p's fill after position p - 30 in a 60-expert step
// over 30 slots); the head is the first two such readers.
void test_head_readers() {
  std::vector<FillWait> w;
  for (int j = 0; j < 30; ++j) w.push_back(FillWait{30 + j, j, true});
  std::vector<char> arriving(60, 0);
  CHECK((head_readers(w, arriving, 2) == std::vector<int>{0, 1}));
  // a reader whose own chunks are still arriving, and fills that wait on nothing
  // or are not fills, are skipped; each reader appears once
  arriving[0] = 1;
  std::vector<FillWait> w2 = {{40, -1, true}, {41, 0, true}, {42, 2, false}, {43, 1, true}, {44, 1, true}, {45, 3, true}};
  CHECK((head_readers(w2, arriving, 2) == std::vector<int>{1, 3}));
  // a reader that itself waits (listed as a waiting position) is skipped
  std::vector<FillWait> w3 = {{5, 4, true}, {4, 2, true}, {6, 1, true}};
  CHECK((head_readers(w3, std::vector<char>(8, 0), 3) == std::vector<int>{2, 1}));
  CHECK(head_readers(w, std::vector<char>(60, 0), 0).empty());
}

void test_resident_groups() {
  std::vector<int> ready;
  for (int p = 2; p < 30; ++p) ready.push_back(p);  // 0 and 1 ran with the route
  std::vector<FillWait> w;
  for (int j = 0; j < 30; ++j) w.push_back(FillWait{30 + j, j, true});
  auto g = resident_groups(ready, w, 8);
  CHECK(g.size() == 4u);
  CHECK(g.size() == 4u && g[0].front() == 2 && g[0].back() == 9 && g[1].front() == 10 && g[3].back() == 29 &&
        g[3].size() == 4u);
  // nothing waits: one launch
  g = resident_groups(ready, {}, 8);
  CHECK(g.size() == 1u && g[0] == ready);
  // only position 3 is waited for: one group of eight through it, the rest together
  g = resident_groups(ready, {{40, 3, true}}, 8);
  CHECK(g.size() == 2u && g[0].size() == 8u && g[1].size() == ready.size() - 8);
  // waited position in the third group: groups of eight through it, then the rest
  g = resident_groups(ready, {{40, 20, true}}, 8);
  CHECK(g.size() == 4u && g[0].size() == 8u && g[1].size() == 8u && g[2].front() == 18 && g[2].back() == 25 &&
        g[3].front() == 26 && g[3].back() == 29);
  // every position appears exactly once, in order
  std::vector<int> flat;
  for (const auto& x : resident_groups(ready, w, 3)) flat.insert(flat.end(), x.begin(), x.end());
  CHECK(flat == ready);
  CHECK(resident_groups({}, w, 8).empty());
}

// High-priority copies in flight do not count against the low-priority window:
// a prefetch queues right behind the misses, so the link has no idle gap
// between them, and a later miss still waits for at most `window` of them.
void test_low_queues_behind_high() {
  Rig r(2, 4, 8, 100, 100, 2);
  r.eng.bw = 100.0;
  for (int s = 0; s < 3; ++s) {
    r.pf->assign(0, s, s);
    r.pf->issue_high(0, s);  // 9 chunks of misses, 9 time units
  }
  r.pf->assign(1, 0, 5);
  r.pf->push_low(1, 0);
  CHECK(r.pf->pump() == 2);  // two prefetch chunks queue behind the misses at once
  CHECK(r.eng.log.size() == 11);
  CHECK(std::fabs(r.eng.log[9].start - r.eng.log[8].end) < 1e-9);  // no gap after the misses
  CHECK(r.pf->low_in_flight() == 2);
  r.worker_until(100.0);
  CHECK(r.pf->low_in_flight() == 0 && r.eng.log.size() == 12);
}

// pending_bytes(): bytes issued and not yet retired, plus the unissued bytes of
// queued low-priority chunks (what the link must carry before a new copy).
void test_pending_bytes() {
  Rig r(2, 4, 8, 300, 100, 1);  // chunks of 3 sub-copies of 100 bytes
  r.eng.bw = 100.0;
  CHECK(r.pf->pending_bytes() == 0);
  r.pf->assign(0, 0, 0);
  r.pf->issue_high(0, 0);  // 3 chunks = 900 bytes in flight
  CHECK(r.pf->pending_bytes() == 900);
  r.pf->assign(1, 0, 5);
  r.pf->push_low(1, 0);    // 3 chunks queued, none issued yet
  CHECK(r.pf->pending_bytes() == 1800);
  CHECK(r.pf->pump() == 1);  // window 1: one 100-byte sub-copy of the first low chunk
  CHECK(r.pf->pending_bytes() == 1800);  // moved from queued to in flight
  r.eng.advance(9.0);        // the misses (9 units) are done, the low sub-copy (10th unit) not yet
  r.pf->retire();
  CHECK(r.pf->pending_bytes() == 900);
  r.pf->purge_low(1);        // early preemption drops the unissued 800 bytes
  CHECK(r.pf->pending_bytes() == 100);
  r.eng.advance(20.0);
  r.pf->retire();
  CHECK(r.pf->pending_bytes() == 0);
}

// A high-priority copy waits for at most `window` already-issued low-priority
// sub-copies (earlier high-priority copies are drained before each miss).
void test_window_bound() {
  for (int window = 1; window <= 3; ++window) {
    Rig r(2, 8, 16, 1600, 100, window);  // 16 sub-copies per chunk of 1 time unit each
    r.eng.bw = 100.0;
    for (int s = 0; s < 8; ++s) {
      r.pf->assign(1, s, 8 + s);
      r.pf->push_low(1, s);
    }
    double t = 0.37;
    double max_delay = 0.0;
    for (int trial = 0; trial < 4; ++trial) {
      r.worker_until(t);
      const size_t mark = r.eng.log.size();
      const int slot = trial;
      r.pf->assign(0, slot, slot);
      r.pf->issue_high(0, slot);
      const double start = r.first_start_into(0, slot, 8, mark);
      max_delay = std::max(max_delay, start - r.eng.now);
      CHECK(start - r.eng.now <= window * 1.0 + 1e-9);
      t = r.eng.log.back().end + 0.61;  // next miss after this one's copies are done
    }
    CHECK(max_delay > 0.0);  // low-priority work really was in flight
  }
}

void test_purge_dedupe_and_priority() {
  Rig r(3, 4, 8, 100, 100, 1);
  r.eng.bw = 100.0;
  r.pf->assign(1, 0, 5);
  r.pf->push_low(1, 0);
  r.pf->push_low(1, 0);  // dedupe: chunks already queued
  r.pf->assign(2, 0, 6);
  r.pf->push_low(2, 0);
  r.pf->pump();  // window 1: only the first LOW sub-copy issues
  CHECK(r.eng.log.size() == 1);
  r.pf->purge_low(1);  // drops layer 1's remaining two chunks only
  CHECK(r.pf->stats().low_purged == 2);
  CHECK(r.pf->has_low());
  // high priority goes next, in issue order, regardless of queued low work
  r.pf->assign(0, 1, 3);
  r.pf->issue_high(0, 1);
  CHECK(r.eng.log.size() == 4);
  r.worker_until(100.0);
  CHECK(r.eng.log.size() == 7);  // layer 2's three chunks follow
  CHECK(r.pf->stats().copies[LOW] == 4 && r.pf->stats().copies[HIGH] == 3);
  // re-push after a purge continues from what was issued (no duplicate bytes)
  r.pf->issue_high(1, 0);
  CHECK(r.eng.log.size() == 9);
}

void test_ready_and_war() {
  Rig r(1, 2, 4, 100, 50, 2);  // 2 sub-copies per chunk
  r.eng.bw = 100.0;
  r.pf->mark_resident(0, 0, 0);
  CHECK(r.pf->ready_seq(0, 0, 2) == -1);  // warm slot: nothing to wait for
  // a reader of slot 0 (compute token 7, completes at t = 5)
  r.pf->set_last_read(0, 0, 7);
  r.eng.compute_done[7] = 5.0;
  r.pf->assign(0, 0, 3);
  CHECK(r.pf->ready_seq(0, 0, 0) == -2);  // not issued yet
  r.pf->issue_high(0, 0);
  CHECK(r.eng.log[0].after == 7 && r.eng.log[0].start >= 5.0);  // write-after-read
  const int64_t need01 = r.pf->ready_seq(0, 0, 1), need2 = r.pf->ready_seq(0, 0, 2);
  CHECK(need01 == 3 && need2 == 5);  // last sub-copy of chunk 1 / chunk 2
  r.worker_until(100.0);
  CHECK(r.pf->ready_seq(0, 0, 2) == -1);
}

void test_deferred_fill() {
  // streaming through a too-small cache: the fill into slot 0 waits for the
  // compute that reads slot 0's previous expert (token 3 completes at t = 9)
  Rig r(1, 1, 8, 100, 100, 2);
  r.eng.bw = 100.0;
  r.pf->mark_resident(0, 0, 0);
  r.eng.compute_done[3] = 9.0;
  r.pf->assign(0, 0, 4);
  r.pf->issue_high_after(0, 0, 3);
  CHECK(r.eng.log.size() == 3 && r.eng.log[0].start >= 9.0 && r.pf->stats().deferred == 1);
}

void test_assign_cancels_stale_low() {
  Rig r(1, 2, 8, 100, 100, 1);
  r.pf->assign(0, 0, 1);
  r.pf->push_low(0, 0);
  r.pf->assign(0, 0, 2);  // the slot changes hands before its low tasks ran
  r.pf->pump();
  CHECK(r.eng.log.empty());
  CHECK(!r.pf->has_low());
}

void test_capacity_wrap() {
  Rig r(1, 4, 8, 100, 10, 1);
  r.eng.cap = 4;
  for (int s = 0; s < 3; ++s) {
    r.pf->assign(0, s, s);
    r.pf->issue_high(0, s);  // 3 chunks x 10 sub-copies each, at most 4 outstanding
  }
  CHECK(r.pf->in_flight() <= 4);
  CHECK(r.eng.log.size() == 90);
}

void test_high_merge() {
  // chunk 100 B, sub 25 B: a fresh slot at high priority is one 300 B copy (merge 1000)
  {
    FakeEngine eng;
    std::vector<uint8_t> host(8 * 300), cache(2 * 300);
    Prefetcher pf(1, 2, 8, 100, 25, 2, cache.data(), &eng, 1000);
    for (int e = 0; e < 8; ++e) pf.set_host(0, e, host.data() + e * 300);
    pf.assign(0, 1, 3);
    pf.issue_high(0, 1);
    CHECK(eng.log.size() == 1 && eng.log[0].bytes == 300 && eng.log[0].dst == cache.data() + 300);
    CHECK(pf.ready_seq(0, 1, 0) == 0 && pf.ready_seq(0, 1, 2) == 0);
  }
  // partial low progress: chunk 0 half issued at low priority, the rest merges
  // into one run from the first pending byte; merge cap splits at sub boundaries
  {
    FakeEngine eng;
    eng.bw = 1.0;
    std::vector<uint8_t> host(8 * 300), cache(2 * 300);
    Prefetcher pf(1, 2, 8, 100, 25, 2, cache.data(), &eng, 120);
    for (int e = 0; e < 8; ++e) pf.set_host(0, e, host.data() + e * 300);
    pf.assign(0, 0, 5);
    pf.push_low(0, 0);
    pf.pump();  // window 2: two 25 B low sub-copies of chunk 0
    CHECK(eng.log.size() == 2);
    pf.purge_low(0);
    pf.issue_high(0, 0);
    // pending bytes [50, 300) in runs of <= 120 B cut at 25 B boundaries
    size_t covered = 0;
    for (size_t i = 2; i < eng.log.size(); ++i) {
      CHECK(eng.log[i].bytes <= 120 && eng.log[i].bytes % 25 == 0);
      CHECK(eng.log[i].dst == cache.data() + 50 + covered);
      covered += eng.log[i].bytes;
    }
    CHECK(covered == 250);
    CHECK(pf.ready_seq(0, 0, 2) == (int64_t)eng.log.size() - 1);
    CHECK(pf.stats().bytes[HIGH] == 250 && pf.stats().bytes[LOW] == 50);
  }
}

// Every combination of chunk / sub-copy / merge size and low-priority progress:
// the high-priority runs copy each remaining byte of the slot exactly once,
// stay inside the slot, respect the merge cap, and leave every chunk ready.
void test_high_merge_exhaustive() {
  struct Rec : CopyEngine {
    struct C { size_t off, bytes; };
    std::vector<C> log;
    uint8_t* base = nullptr;
    void issue(int64_t, void* d, const void*, size_t b, int64_t, int) override {
      log.push_back({(size_t)(static_cast<uint8_t*>(d) - base), b});
    }
    bool done(int64_t) override { return true; }
    void wait(int64_t) override {}
  };
  for (size_t chunk : {7, 30, 100, 128})
    for (size_t sub : {1, 3, 25, 30, 64, 200})
      for (size_t merge : {0, 1, 29, 64, 120, 1000})
        for (int pre0 = 0; pre0 < 5; ++pre0)
          for (int pre1 = 0; pre1 < 3; ++pre1) {
            const size_t sb = std::min(sub, chunk);
            const int nsub = (int)((chunk + sb - 1) / sb);
            if (merge && merge < sb) continue;
            const int p0 = std::min(pre0, nsub), p1 = std::min(pre1, nsub);
            const int low = p0 + (p0 == nsub ? p1 : 0);
            Rec e;
            std::vector<uint8_t> host(4 * 3 * chunk), cache(2 * 3 * chunk);
            e.base = cache.data();
            Prefetcher pf(1, 2, 4, chunk, sub, std::max(1, low), cache.data(), &e, merge);
            for (int x = 0; x < 4; ++x) pf.set_host(0, x, host.data() + x * 3 * chunk);
            pf.assign(0, 1, 2);
            pf.push_low(0, 1);
            if (low) pf.pump();
            const size_t n_low = e.log.size();
            pf.purge_low(0);
            pf.issue_high(0, 1);
            std::vector<int> cov(3 * chunk, 0);
            bool ok = true;
            for (size_t i = 0; i < e.log.size(); ++i) {
              const auto& c = e.log[i];
              if (c.off < 3 * chunk || c.off + c.bytes > 6 * chunk) { ok = false; break; }
              for (size_t b = 0; b < c.bytes; ++b) cov[c.off - 3 * chunk + b]++;
              if (i >= n_low && merge && c.bytes > std::max(merge, sb)) ok = false;
            }
            for (int v : cov) ok = ok && v == 1;
            ok = ok && pf.ready_seq(0, 1, 2) != -2;
            CHECK(ok);
          }
}


// A copy engine with several independent FIFO queues whose copies take random
// times, moving the bytes when a copy completes: what a reader finds in a slot
// is what has landed by the time it reads.
struct DataEngine : CopyEngine {
  int nq = 2;
  double now = 0.0;
  std::mt19937_64 rng;
  struct Copy {
    double end;
    uint8_t* dst;
    const uint8_t* src;
    size_t bytes;
    bool landed;
  };
  std::vector<Copy> log;
  std::vector<double> q_end;
  std::map<int64_t, double> compute_done;
  explicit DataEngine(int queues, uint64_t seed) : nq(queues), rng(seed), q_end(queues, 0.0) {}
  int queues() const override { return nq; }
  void issue(int64_t seq, void* dst, const void* src, size_t bytes, int64_t after, int queue) override {
    if ((int64_t)log.size() != seq || queue < 0 || queue >= nq) std::abort();
    double start = std::max(now, q_end[queue]);
    if (after >= 0) {
      auto it = compute_done.find(after);
      start = std::max(start, it == compute_done.end() ? 1e30 : it->second);
    }
    const double end = start + 0.05 + std::uniform_real_distribution<double>(0.0, 1.0)(rng) * (double)bytes / 4.0;
    q_end[queue] = end;
    log.push_back({end, static_cast<uint8_t*>(dst), static_cast<const uint8_t*>(src), bytes, false});
  }
  // move the bytes of every copy that has completed by time t, in completion order
  void land(double t) {
    std::vector<size_t> due;
    for (size_t i = 0; i < log.size(); ++i)
      if (!log[i].landed && log[i].end <= t) due.push_back(i);
    std::sort(due.begin(), due.end(), [&](size_t a, size_t b) {
      return log[a].end < log[b].end || (log[a].end == log[b].end && a < b);
    });
    for (size_t i : due) {
      std::memcpy(log[i].dst, log[i].src, log[i].bytes);
      log[i].landed = true;
    }
  }
  bool done(int64_t seq) override {
    land(now);
    return log[seq].end <= now;
  }
  void wait(int64_t seq) override {
    now = std::max(now, log[seq].end);
    land(now);
  }
};

// The library's protocol over random plans and timings: speculative plans
// (assign + push_low), the worker's pumping, and routes that read the layer's
// routed slots -- at once when no copy into them is pending (the early resident
// launch), else after the host has purged the layer's low work, issued the
// rest at high priority and waited, on each queue, for the latest copy
// ready_seq names (the compute stream's event waits).  Every read must find the
// bytes of the expert the plan put in the slot, and no copy may land in a slot
// before a read of its previous contents that the plan ordered first.
void test_random_protocol() {
  const int L = 2, C = 3, E = 6;
  const size_t chunk = 8, sub = 4;
  for (uint64_t seed = 1; seed <= 300; ++seed) {
    const int window = 1 + (int)(seed % 2);
    const size_t merge = seed % 3 == 0 ? 16 : 0;
    DataEngine eng(1 + (int)(seed % 3 != 1), seed);
    std::vector<uint8_t> host((size_t)L * E * 3 * chunk), cache((size_t)L * C * 3 * chunk, 0xEE);
    for (size_t i = 0; i < host.size(); ++i) host[i] = (uint8_t)(i * 7 + 3);
    Prefetcher pf(L, C, E, chunk, sub, window, cache.data(), &eng, merge);
    for (int l = 0; l < L; ++l)
      for (int e = 0; e < E; ++e) pf.set_host(l, e, host.data() + ((size_t)l * E + e) * 3 * chunk);
    std::vector<std::vector<int>> owner(L, std::vector<int>(C));
    for (int l = 0; l < L; ++l)
      for (int s2 = 0; s2 < C; ++s2) {
        owner[l][s2] = s2;
        std::memcpy(cache.data() + ((size_t)l * C + s2) * 3 * chunk, pf.host(l, s2), 3 * chunk);
        pf.mark_resident(l, s2, s2);
      }
    std::mt19937_64& rng = eng.rng;
    auto rnd = [&](int n) { return (int)(rng() % (uint64_t)n); };
    int64_t tok = 0;
    double gpu = 0.0;  // the compute stream's clock
    bool bad = false;
    auto slot_of = [&](int l, int e) {
      for (int s2 = 0; s2 < C; ++s2)
        if (owner[l][s2] == e) return s2;
      return -1;
    };
    auto read = [&](int l, int s2, double t) {
      eng.land(t);
      const uint8_t* got = cache.data() + ((size_t)l * C + s2) * 3 * chunk;
      if (std::memcmp(got, pf.host(l, owner[l][s2]), 3 * chunk) != 0 && !bad) {
        std::printf("  seed %llu: layer %d slot %d read at %.3f does not hold expert %d\n",
                    (unsigned long long)seed, l, s2, t, owner[l][s2]);
        bad = true;
      }
    };
    for (int step = 0; step < 60 && !bad; ++step) {
      // a speculative plan for a random layer
      const int lt = rnd(L);
      std::vector<int> pred;
      for (int n = 1 + rnd(2); (int)pred.size() < n;) {
        const int e = rnd(E);
        if (std::find(pred.begin(), pred.end(), e) == pred.end()) pred.push_back(e);
      }
      for (int e : pred) {
        int s2 = slot_of(lt, e);
        if (s2 < 0) {
          std::vector<int> cand;
          for (int v = 0; v < C; ++v)
            if (std::find(pred.begin(), pred.end(), owner[lt][v]) == pred.end()) cand.push_back(v);
          if (cand.empty()) continue;
          s2 = cand[rnd((int)cand.size())];
          owner[lt][s2] = e;
          pf.assign(lt, s2, e);
        }
        pf.push_low(lt, s2);
      }
      // the worker runs for a while
      for (int k = rnd(4); k > 0; --k) {
        pf.pump();
        eng.now += 0.3 * rnd(4);
        pf.retire();
      }
      // a route of a random layer
      const int lr = rnd(L);
      std::vector<int> routed;
      for (int n = 1 + rnd(2); (int)routed.size() < n;) {
        const int e = rnd(E);
        if (std::find(routed.begin(), routed.end(), e) == routed.end()) routed.push_back(e);
      }
      pf.retire();
      std::vector<int> early_slots, late_slots;
      for (int e : routed) {
        const int s2 = slot_of(lr, e);
        if (s2 >= 0 && pf.ready_seq(lr, s2, 2) == -1) early_slots.push_back(s2);
      }
      const double t_early = std::max(gpu, eng.now);
      for (int s2 : early_slots) read(lr, s2, t_early);
      if (!early_slots.empty()) gpu = t_early + 0.01;
      pf.purge_low(lr);
      for (int e : routed) {
        int s2 = slot_of(lr, e);
        if (s2 >= 0 && std::find(early_slots.begin(), early_slots.end(), s2) != early_slots.end()) continue;
        if (s2 < 0) {
          std::vector<int> cand;
          for (int v = 0; v < C; ++v) {
            bool used = false;
            for (int r2 : routed) used = used || owner[lr][v] == r2;
            if (!used) cand.push_back(v);
          }
          s2 = cand[rnd((int)cand.size())];
          owner[lr][s2] = e;
          pf.assign(lr, s2, e);
        }
        pf.issue_high(lr, s2);
        late_slots.push_back(s2);
      }
      // the early launch's reads are recorded once the plan is read (after the fills above)
      if (!early_slots.empty()) {
        eng.compute_done[tok] = gpu;
        for (int s2 : early_slots) pf.set_last_read(lr, s2, tok);
        ++tok;
      }
      if (!late_slots.empty()) {
        std::vector<int64_t> need(eng.nq, -1);
        for (int s2 : late_slots) {
          const int64_t n = pf.ready_seq(lr, s2, 2);
          CHECK(n != -2);
          const int q = pf.queue_of(lr, s2);
          need[q] = std::max(need[q], n);
        }
        double t = std::max(gpu, eng.now);
        for (int q = 0; q < eng.nq; ++q)
          if (need[q] >= 0) t = std::max(t, eng.log[need[q]].end);
        for (int s2 : late_slots) read(lr, s2, t);
        gpu = t + 0.01;
        eng.compute_done[tok] = gpu;
        for (int s2 : late_slots) pf.set_last_read(lr, s2, tok);
        ++tok;
      }
      eng.now += 0.2 * rnd(3);
      pf.retire();
    }
    CHECK(!bad);
  }
}
}  // namespace

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "example") == 0) {
    double a, b, c;
    example(&a, &b, &c);
    std::printf("%.6f %.6f %.6f\n", a, b, c);
    return 0;
  }
  test_example();
  test_whole_expert_low();
  test_low_queues_behind_high();
  test_pending_bytes();
  test_queue_per_slot();
  test_fills_balance_queues();
  test_queue_kept_over_uncopied_owner();
  test_head_readers();
  test_resident_groups();
  test_window_bound();
  test_purge_dedupe_and_priority();
  test_ready_and_war();
  test_deferred_fill();
  test_assign_cancels_stale_low();
  test_capacity_wrap();
  test_high_merge();
  test_high_merge_exhaustive();
  test_random_protocol();
  std::printf(failures ? "FAILED %d\n" : "ALL OK\n", failures);
  return failures ? 1 : 0;
}
