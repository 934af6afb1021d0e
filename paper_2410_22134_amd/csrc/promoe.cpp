// Host runtime and C ABI of the expert cache (see include/promoe.h).
//
// Split of responsibilities
//  * logical cache state (slot tables, LRU stamps, counters) lives on the
//    device and changes only inside the plan kernels, in stream order;
//  * the plan kernels write a record per plan into host-mapped memory;
//  * the host ingests records in program order into the copy scheduler
//    (Prefetcher), which tracks what each slot physically holds and issues the
//    copies on the library's copy stream;
//  * speculative records are ingested by a worker thread (the prefetch worker
//    of Alg. 1) that waits on the plan's event, so promoe_predict never blocks;
//    a route synchronises once on its own plan and issues its high-priority
//    copies itself, in the returned order, right behind at most `window`
//    in-flight low-priority sub-copies;
//  * compute waits on copy events only for the chunks it reads (gate/up pass
//    after chunks 0-1, down pass after chunk 2); copies into a slot wait on the
//    event of the last launch that read it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/promoe.h"
#include "common.hpp"
#include "kernels.hpp"
#include "scheduler.hpp"

using namespace promoe;

namespace {

thread_local std::string g_last_error;

constexpr int kRecRing = 64;
constexpr int kStallClass = 99;
constexpr size_t kHighMergeBytes = (size_t)64 << 20;  // high-priority copies coalesce up to this size
constexpr size_t kOneQueueChunkBytes = (size_t)24 << 20;  // chunks this large use one copy queue
constexpr int kMaxSplit = 8;  // split-K slices of the shared expert's down GEMM
constexpr int kCopyRing = 4096;
constexpr int kComputeRing = 4096;

// Scratch of promoe_expert_ffn_noalloc: one file-scope device array per GPU
// (each device that loads the library holds its own copy until the process
// ends).  Host code never uses the array's name as an address: the per-device
// address comes from hipGetSymbolAddress, taken once per device at context
// creation with that device current.
constexpr size_t kNoAllocScratchBytes = (size_t)8 << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxDevices] = {};

struct ProfEntry {
  hipEvent_t a, b;
  int cls;  // 0..5 kernel classes, kStallClass copy waits
  double bytes, flops;
};

// Host-to-device copies on two streams (two DMA queues keep the link busy
// through each copy's setup: measured 52 -> 57 GB/s for 5.5 MiB copies).
constexpr int kCopyStreams = 2;
// Fills whose victims' readers run ahead of the other resident experts (one per
// copy queue keeps every queue busy from the start).
constexpr int kHeadFills = kCopyStreams;
// Experts per FFN launch while copies arrive, for steps larger than decode.
constexpr int kArrivalGroup = kCopyStreams;
// Resident experts per FFN launch, for steps larger than decode (as many as
// one 4-bit staging batch).
constexpr int kResidentGroup = 8;
// Expert jobs with at least this many token pairs run on the MFMA GEMM.
constexpr int kGemmMinTokens = 16;

class HipEngine : public CopyEngine {
 public:
  hipStream_t stream[kCopyStreams] = {};
  std::vector<hipEvent_t> ev;
  std::vector<hipEvent_t>* compute_ev = nullptr;
  std::vector<hipStream_t>* compute_stream = nullptr;  // stream each compute token was recorded on
  hipError_t err = hipSuccess;
  // Latest compute token each queue is known to follow (it waited for it, or
  // the token had completed when a copy was queued), and that token's stream.
  int64_t followed[kCopyStreams];
  hipStream_t followed_on[kCopyStreams] = {};
  HipEngine() {
    for (auto& f : followed) f = -1;
  }

  void issue(int64_t seq, void* dst, const void* src, size_t bytes, int64_t after, int queue) override {
    hipStream_t s = stream[queue];
    hipError_t e = hipSuccess;
    // A wait on a compute event costs the copy queue a barrier and a poll even
    // when the event has completed; wait only on compute still running that
    // the queue does not already follow (tokens of one compute stream complete
    // in order, so following a later token of the same stream suffices).
    if (after >= 0) {
      hipEvent_t ce = (*compute_ev)[after % kComputeRing];
      hipStream_t cs = (*compute_stream)[after % kComputeRing];
      const bool covered = followed[queue] >= after && followed_on[queue] == cs;
      if (!covered) {
        if (hipEventQuery(ce) != hipSuccess) e = hipStreamWaitEvent(s, ce, 0);
        if (e == hipSuccess && (after > followed[queue] || followed_on[queue] != cs)) {
          followed[queue] = after;
          followed_on[queue] = cs;
        }
      }
    }
    if (e == hipSuccess) e = hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipEventRecord(ev[seq % kCopyRing], s);
    if (e != hipSuccess && err == hipSuccess) err = e;
  }
  int nq = kCopyStreams;  // queues in use (1 for large chunks)
  int queues() const override { return nq; }
  bool done(int64_t seq) override { return hipEventQuery(ev[seq % kCopyRing]) == hipSuccess; }
  void wait(int64_t seq) override {
    hipError_t e = hipEventSynchronize(ev[seq % kCopyRing]);
    if (e != hipSuccess && err == hipSuccess) err = e;
  }
  hipEvent_t event(int64_t seq) { return ev[seq % kCopyRing]; }
  int64_t capacity() const override { return kCopyRing - 1; }
};

// The copies a launch must wait for: the latest one needed on each engine
// queue (a queue completes in order; queues do not order each other).
struct CopyWait {
  int64_t seq[kCopyStreams];
  CopyWait() { for (auto& q : seq) q = -1; }
  void add(int queue, int64_t s) { seq[queue] = std::max(seq[queue], s); }
};

struct LayerW {
  const void *wg = nullptr, *pw1 = nullptr, *pw2 = nullptr, *shared = nullptr, *sgate = nullptr, *attn = nullptr;
  const float* bias = nullptr;
  bool planned = false;
};

// A position whose copies wait for an earlier position's compute: a fill of a
// slot that an earlier position reads (write after read), or, without early
// preemption, any copy still to issue when the position is reached.
struct Deferred {
  int pos, slot, expert, after;
  bool fill;  // the slot changes expert (else only pending chunks are issued)
};

}  // namespace

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

struct promoe_ctx {
  promoe_config cfg{};
  int dev = 0;
  int L, H, E, K, I, Ish, C, D, Ph, maxT, dt, eb;
  bool q4 = false;  // routed experts stored as 4-bit codes
  bf16_t* d_stage = nullptr;  // 4-bit experts expanded for the MFMA GEMM (kStageExperts)
  size_t chunk_bytes, expert_bytes;
  uint8_t* cache = nullptr;

  // device memory
  void* dmem = nullptr;
  CacheState st{};
  float* d_logits = nullptr;
  int ld_logits = 0;
  int pred_col = 0;  // first predictor column of d_logits (after gate and shared-gate columns)
  float* d_predq = nullptr;
  int32_t* d_pred_ids = nullptr;
  int32_t* d_order_slot = nullptr;
  int32_t* d_offsets = nullptr;
  int32_t* d_perm = nullptr;
  int32_t* d_pos_of = nullptr;
  int32_t* d_warm = nullptr;
  int32_t* d_npos = nullptr;  // resident positions of the latest precise plan (device)
  void* d_act = nullptr;
  float* d_Y = nullptr;
  void* d_act_sh = nullptr;
  float* d_Ysh = nullptr;
  void* d_u = nullptr;
  uint8_t* noalloc_scratch = nullptr;  // this device's address of `scratch`
  bool noalloc_call = false;           // inside promoe_expert_ffn_noalloc: no profiling, no staging

  std::vector<LayerW> lw;

  // gate logits computed by predict, reused by route
  int gate_layer = -1;
  const void* gate_x = nullptr;
  int gate_T = 0;

  // plan records
  PlanRecord* rec_h = nullptr;  // host view
  PlanRecord* rec_d = nullptr;  // device view
  hipEvent_t rec_ev[kRecRing];
  int rec_kind[kRecRing];
  int rec_prio[kRecRing];
  int64_t rec_next = 0, rec_pub = 0, rec_ingested = 0;  // reserved / event recorded / ingested
  std::vector<PlanRecord> last_spec, last_precise;

  // route -> ffn hand-over
  int route_layer = -1;
  int route_T = 0;
  const void* route_x = nullptr;  // input of the latest route (its gate logits are in d_logits)
  int last_route_layer = -1;      // layer of the latest route, kept after its FFN call
  std::vector<char> ffn_started;  // per route position: launched by the route itself
  bool shared_started = false;    // the shared expert too
  // mean interval between consecutive routes (PROMOE_FLAG_FILL_BY_DEADLINE)
  std::chrono::steady_clock::time_point last_route_t{};
  bool have_route_t = false;
  double route_dt_ema = 0.0;
  uint64_t early_busy = 0;        // slots the route's early launch skipped
  size_t early_prof0 = 0, early_nprof = 0;  // its profiling entries (bytes filled in by the route)
  hipStream_t route_stream = nullptr;  // stream of the latest route
  hipEvent_t route_done = nullptr;     // recorded on it after the route's last launch
  // The predictor's kernels after its first rows (second layer, top-k, spec
  // plan) run on a side stream of the library, forked from the caller's stream
  // once those rows are written and joined back into it at the end of the
  // predict call: they overlap the layer's expert launches queued before them.
  hipStream_t pred_stream = nullptr;
  hipEvent_t pred_in = nullptr, pred_done = nullptr;
  bool pred_nojoin = true;            // no prediction's side-stream work needs a device join
  bool pred_pending = false;          // else: pred_done recorded, no stream has waited for it yet
  hipStream_t pred_joined = nullptr;  // or the latest stream that did
  // A prediction launched by promoe_route_predict ends with its spec plan,
  // record pred_host_rec: the next call that could touch what it reads or
  // writes first waits on the host for that record (no device-side join).
  int64_t pred_host_rec = -1;
  // Every expert of every layer resident (as many slots as experts, and each
  // layer's initial cache holds all of them): no plan can fill a slot, so a
  // decode-sized route whose resident launch covers the whole step need not
  // wait for its plan on the host ("lazy" route); its record is taken in
  // later, once complete.
  std::vector<char> layer_full;
  int n_full_layers = 0;
  bool all_resident() const { return C == E && n_full_layers == L; }
  bool rec_lazy[kRecRing] = {};            // record of a lazy route, not yet taken in
  int lazy_T[kRecRing] = {};                // its step's tokens
  size_t lazy_prof0[kRecRing] = {}, lazy_nprof[kRecRing] = {};  // its launch's profiling entries
  bool route_lazy = false;                  // the latest route is lazy
  int64_t n_lazy_routes = 0;
  // promoe_stack_step: the FFN call's combine also adds y into fuse_h, and
  // the route computes x = q(rms(x_from_h)) inside its gate GEMV (batch 1)
  float* fuse_h = nullptr;
  const float* x_from_h = nullptr;
  float* d_h2 = nullptr;  // second residual buffer of the batch-1 layer loop
  // defer_combine: the FFN call leaves its combine (into fuse_h) pending for
  // the next layer's attention GEMV to fold in
  bool defer_combine = false, has_pending = false;
  CombineArgs pending{};
  float* pending_h = nullptr;
  // a lazy batch-1 route's prediction, to ride in its resident gate/up launch
  bool ride_pred = false;
  PredictPlanArgs ride{};
  // first predictor rows computed by a route's gate launch (layer, input, T)
  int pred_rows_layer = -1;
  const void* pred_rows_x = nullptr;
  int pred_rows_T = 0;
  PlanRecord route_rec{};
  std::vector<int64_t> need01, need2;  // copy seq each position waits for (-1 none)
  std::vector<int> need_q;             // engine queue of those copies
  std::vector<uint64_t> pred_host;     // per layer: experts of the last ingested prediction
  int64_t pred_in_time = 0;
  std::vector<Deferred> deferred;

  // scheduler and worker
  HipEngine eng;
  Prefetcher* pf = nullptr;
  std::mutex mu;
  std::condition_variable cv;
  std::thread worker;
  bool stop = false;

  std::vector<hipEvent_t> cev;
  std::vector<hipStream_t> cstream;
  int64_t cnext = 0;
  hipStream_t last_stream = nullptr;

  // profiling: FFN launches timed by the start and end events the launch
  // itself records (kernel execution time), copy-wait stalls by event pairs
  // around the waits
  bool profile = false;
  std::vector<ProfEntry> prof_pending;
  std::vector<hipEvent_t> prof_free;
  static constexpr int kClasses = 6;
  int64_t k_launches[kClasses] = {};
  double k_ms[kClasses] = {}, k_bytes[kClasses] = {}, k_flops[kClasses] = {};
  double stall_ms = 0.0;
};

namespace {

int fail_hip(hipError_t e, const char* what) {
  g_last_error = std::string(what) + ": " + hipGetErrorString(e);
  return PROMOE_EHIP;
}
#define HIPCHK(x)                                 \
  do {                                            \
    hipError_t _e = (x);                          \
    if (_e != hipSuccess) return fail_hip(_e, #x); \
  } while (0)
#define LAUNCHCHK(what)                               \
  do {                                                \
    hipError_t _e = hipGetLastError();                \
    if (_e != hipSuccess) return fail_hip(_e, what);  \
  } while (0)

// This device's address of `scratch` (the current device must be `dev`).
int scratch_address(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) {
    g_last_error = "device index beyond the scratch table";
    return PROMOE_EUNSUP;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return fail_hip(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[dev] = static_cast<uint8_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return PROMOE_OK;
}

hipEvent_t prof_event(promoe_ctx* c) {
  if (!c->prof_free.empty()) {
    hipEvent_t e = c->prof_free.back();
    c->prof_free.pop_back();
    return e;
  }
  // timing-only events: no system-scope fence on completion (it would add a
  // cache writeback/invalidate to every measured interval)
  hipEvent_t e = nullptr;
  hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
  return e;
}

void prof_resolve(promoe_ctx* c) {
  for (auto& p : c->prof_pending) {
    hipEventSynchronize(p.b);
    float ms = 0.0f;
    hipEventElapsedTime(&ms, p.a, p.b);
    if (p.cls < promoe_ctx::kClasses) {
      c->k_launches[p.cls]++;
      c->k_ms[p.cls] += ms;
      c->k_bytes[p.cls] += p.bytes;
      c->k_flops[p.cls] += p.flops;
    } else {
      c->stall_ms += ms;
    }
    c->prof_free.push_back(p.a);
    c->prof_free.push_back(p.b);
  }
  c->prof_pending.clear();
}

// Ingest record r (spec kind) into the copy scheduler.  Caller holds mu and
// knows the record's plan kernel has completed.
void ingest_spec(promoe_ctx* c, int64_t r) {
  const PlanRecord& rec = c->rec_h[r % kRecRing];
  const int layer = rec.layer;
  c->last_spec[layer] = rec;
  if (rec.predicted) {
    uint64_t m = 0;
    for (int i = 0; i < rec.n; ++i) m |= 1ull << rec.expert[i];
    c->pred_host[layer] = m;
  }
  if (!(c->cfg.flags & PROMOE_FLAG_NO_PREFETCH)) {
    const bool high = c->rec_prio[r % kRecRing] == PROMOE_PRIO_HIGH;
    for (int i = 0; i < rec.n; ++i) {
      if (rec.slot[i] < 0) continue;  // skipped: over the fill limit
      if (rec.flag[i]) c->pf->assign(layer, rec.slot[i], rec.expert[i]);
      if (high) c->pf->issue_high(layer, rec.slot[i]);
      else c->pf->push_low(layer, rec.slot[i]);
    }
  }
  c->rec_ingested = r + 1;
}

// Bytes and flops of a resident launch's profiling entries, from its plan: the
// positions it ran (resident, slot not in busy) and the shared expert.
void early_prof_bytes(promoe_ctx* c, const PlanRecord& rec, int T, uint64_t busy, size_t prof0, size_t nprof) {
  double routed_bytes = 0.0, routed_flops = 0.0;
  const double melems = (double)c->I * c->H;
  for (int p = 0; p < rec.n_hit; ++p) {
    if ((busy >> rec.slot[p]) & 1ull) continue;
    routed_bytes += c->q4 ? (double)c->chunk_bytes : melems * c->eb;
    routed_flops += 2.0 * rec.count[p] * melems;
  }
  const double sh_elems = (double)c->Ish * c->H;
  const double sh_bytes = sh_elems * c->eb, sh_flops = 2.0 * T * sh_elems;
  for (size_t i = 0; i < nprof; ++i) {
    ProfEntry& pe = c->prof_pending[prof0 + i];
    const double k = pe.cls == 0 ? 2.0 : 1.0;
    // dense: [shared + routed] x 2 passes; 4-bit: [shared] x 2, then [routed] x 2
    const bool shared_part = c->q4 ? i < 2 && c->Ish > 0 : true;
    const bool routed_part = c->q4 ? !(i < 2 && c->Ish > 0) : true;
    pe.bytes = k * ((shared_part ? sh_bytes : 0.0) + (routed_part ? routed_bytes : 0.0));
    pe.flops = k * ((shared_part ? sh_flops : 0.0) + (routed_part ? routed_flops : 0.0));
  }
}

// Take in the (complete) record r of a lazy route: what the route does with its
// plan once on the host, less the copies (there are none).  Caller holds mu.
void consume_lazy_route(promoe_ctx* c, int64_t r) {
  const int i = (int)(r % kRecRing);
  const PlanRecord& rec = c->rec_h[i];
  const int layer = rec.layer;
  c->last_precise[layer] = rec;
  if (!(c->cfg.flags & PROMOE_FLAG_NO_PREEMPT)) c->pf->purge_low(layer);
  // every predicted expert that was routed was resident in time
  const uint64_t predicted = c->pred_host[layer];
  c->pred_host[layer] = 0ull;
  for (int p = 0; p < rec.n; ++p)
    if ((predicted >> rec.expert[p]) & 1ull) c->pred_in_time++;
  if (c->profile) early_prof_bytes(c, rec, c->lazy_T[i], 0ull, c->lazy_prof0[i], c->lazy_nprof[i]);
  c->rec_lazy[i] = false;
  c->rec_ingested = r + 1;
}

// Records the host takes in without a route waiting on them: spec plans and
// the plans of lazy routes.
bool ingestable(const promoe_ctx* c, int64_t r) {
  return c->rec_kind[r % kRecRing] == 0 || c->rec_lazy[r % kRecRing];
}

// Take in record r (complete, ingestable).  Caller holds mu.
void ingest_rec(promoe_ctx* c, int64_t r) {
  if (c->rec_lazy[r % kRecRing]) consume_lazy_route(c, r);
  else ingest_spec(c, r);
}

void worker_main(promoe_ctx* c) {
  hipSetDevice(c->dev);
  std::unique_lock<std::mutex> lk(c->mu);
  while (!c->stop) {
    while (c->rec_ingested < c->rec_pub && c->rec_kind[c->rec_ingested % kRecRing] == 0 &&
           hipEventQuery(c->rec_ev[c->rec_ingested % kRecRing]) == hipSuccess)
      ingest_spec(c, c->rec_ingested);
    c->pf->pump();
    const bool head_spec = c->rec_ingested < c->rec_pub && c->rec_kind[c->rec_ingested % kRecRing] == 0;
    if (c->pf->has_low() && c->pf->low_in_flight() >= c->pf->window()) {
      const int64_t seq = c->pf->oldest_in_flight();
      hipEvent_t e = c->eng.event(seq);
      lk.unlock();
      hipEventSynchronize(e);
      lk.lock();
      continue;
    }
    if (head_spec) {
      hipEvent_t e = c->rec_ev[c->rec_ingested % kRecRing];
      lk.unlock();
      hipEventSynchronize(e);
      lk.lock();
      continue;
    }
    c->cv.wait(lk);
  }
}

// Reserve a plan record slot (waiting for / ingesting the oldest if the ring is full).
int new_record(promoe_ctx* c, int kind, int prio, int64_t* out) {
  std::unique_lock<std::mutex> lk(c->mu);
  while (c->rec_next - c->rec_ingested >= kRecRing) {
    const int64_t r = c->rec_ingested;
    if (!ingestable(c, r)) {
      g_last_error = "plan record ring blocked by an unconsumed route";
      return PROMOE_ESTATE;
    }
    if (r >= c->rec_pub) {
      g_last_error = "plan record ring full of unpublished records";
      return PROMOE_ESTATE;
    }
    hipEvent_t e = c->rec_ev[r % kRecRing];
    lk.unlock();
    HIPCHK(hipEventSynchronize(e));
    lk.lock();
    if (c->rec_ingested == r) ingest_rec(c, r);
  }
  const int64_t r = c->rec_next++;
  c->rec_kind[r % kRecRing] = kind;
  c->rec_prio[r % kRecRing] = prio;
  c->rec_lazy[r % kRecRing] = false;
  std::memset(&c->rec_h[r % kRecRing], 0, sizeof(PlanRecord));
  *out = r;
  return PROMOE_OK;
}

// Record r's plan event has been recorded (or the plan was abandoned): the
// worker may now look at it.
void publish(promoe_ctx* c, int64_t r) {
  {
    std::lock_guard<std::mutex> lk(c->mu);
    if (c->rec_pub < r + 1) c->rec_pub = r + 1;
  }
  c->cv.notify_all();
}

// Wait until plan record r is readable on the host.  The plan kernel writes
// the record's `done` word last, after a system-scope fence, before the kernel
// ends; polling that word sees the plan sooner than the kernel's completion
// event.  Every 256 polls the event is queried: it ends the wait if the kernel
// has completed, and reports a failed stream instead of spinning on.
hipError_t wait_record(promoe_ctx* c, int64_t r) {
  const volatile int32_t* done = &c->rec_h[r % kRecRing].done;
  for (uint32_t i = 1;; ++i) {
    if (*done) break;
    if ((i & 255) == 0) {
      const hipError_t q = hipEventQuery(c->rec_ev[r % kRecRing]);
      if (q == hipSuccess) break;
      if (q != hipErrorNotReady) return q;
    }
    __builtin_ia32_pause();
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return hipSuccess;
}

// Take in the ingestable records at the head of the ring whose plans have
// completed (block: waiting for each in turn instead of stopping).
hipError_t drain_records(promoe_ctx* c, bool block) {
  std::unique_lock<std::mutex> lk(c->mu);
  while (c->rec_ingested < c->rec_pub && ingestable(c, c->rec_ingested)) {
    const int64_t r = c->rec_ingested;
    const volatile int32_t* done = &c->rec_h[r % kRecRing].done;
    if (!*done) {
      if (!block && hipEventQuery(c->rec_ev[r % kRecRing]) != hipSuccess) break;
      lk.unlock();
      const hipError_t e = wait_record(c, r);
      lk.lock();
      if (e != hipSuccess) return e;
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    if (c->rec_ingested == r) ingest_rec(c, r);
  }
  return hipSuccess;
}

int64_t record_compute(promoe_ctx* c, hipStream_t s) {
  const int64_t tok = c->cnext++;
  hipEventRecord(c->cev[tok % kComputeRing], s);
  c->cstream[tok % kComputeRing] = s;
  return tok;
}

PlanArgs plan_args(promoe_ctx* c, int layer, const int32_t* ids, int T, int64_t r) {
  PlanArgs a{};
  a.st = c->st;
  a.layer = layer;
  a.C = c->C;
  a.E = c->E;
  a.ids = ids;
  a.T = T;
  a.k = c->K;
  // fills allowed in a predictor-driven speculative plan (-1: no limit)
  const int lim = c->cfg.spec_fill_limit;
  a.fill_budget = lim == 0 ? -1 : (lim < 0 ? 0 : lim);
  a.reorder = (c->cfg.flags & PROMOE_FLAG_NO_REORDER) ? 0 : 1;
  a.pinned = (c->cfg.flags & PROMOE_FLAG_STATIC) ? c->C - 2 : 0;
  a.rec = c->rec_d + (r % kRecRing);
  a.d_order_slot = c->d_order_slot;
  a.d_offsets = c->d_offsets;
  a.d_perm = c->d_perm;
  a.d_pos_of = c->d_pos_of;
  a.d_npos = c->d_npos;
  a.host_done = 1;
  return a;
}

// PROMOE_FLAG_FILL_BY_DEADLINE: slots a predictor-driven plan may fill, the
// whole experts the link can still copy before the target layer's route
// (lookahead routes from now at the mean interval between routes) after what
// is already queued or in flight.
int deadline_fill_budget(promoe_ctx* c) {
  const int lim = c->cfg.spec_fill_limit;
  if (lim < 0 || c->D <= 0 || c->route_dt_ema <= 0.0) return 0;
  const int cap = lim > 0 ? lim : 64;
  int64_t pending;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    c->pf->retire();
    pending = c->pf->pending_bytes();
  }
  const double rate = (c->cfg.link_gb_per_s > 0.0f ? c->cfg.link_gb_per_s : 56.0) * 1e9;
  const double room = rate * c->D * c->route_dt_ema - (double)pending;
  if (room <= 0.0) return 0;
  return (int)std::min<double>(cap, std::floor(room / (double)c->expert_bytes));
}

int check_tokens(promoe_ctx* c, int T) {
  if (T < 1 || T > c->maxT) {
    g_last_error = "T out of range";
    return PROMOE_EINVAL;
  }
  return PROMOE_OK;
}

// Gate (+ shared-gate row) (+ predictor first layer) rows over x, one launch:
// columns [0, E) gate logits, E shared-gate logit (if any), then predictor rows.
// Gate rows (and the shared-gate row) of `layer` into d_logits columns
// [0, pred_col), and with `with_pred` the predictor's first rows from column
// pred_col; `gate` = false computes the predictor rows only (the gate columns
// already hold this input's logits).
int launch_gate_rows(promoe_ctx* c, int layer, const void* d_x, int T, bool with_pred, hipStream_t s,
                     bool gate = true) {
  const LayerW& w = c->lw[layer];
  RowsArgs a{};
  a.w[0] = gate ? w.wg : nullptr;
  a.nrows[0] = gate ? c->E : 0;
  a.w[1] = gate ? w.sgate : nullptr;
  a.nrows[1] = gate && w.sgate ? 1 : 0;
  a.w[2] = with_pred ? w.pw1 : nullptr;
  a.nrows[2] = with_pred ? (c->Ph > 0 ? c->Ph : c->E) : 0;
  a.K = c->H;
  a.x = d_x;
  a.ldx = c->H;
  a.x_off = 0;
  a.T = T;
  a.out = c->d_logits;
  a.ldo = c->ld_logits;
  a.o_off = gate ? 0 : c->pred_col;  // the row groups land in consecutive columns
  if (a.nrows[0] + a.nrows[1] + a.nrows[2] == 0) return PROMOE_OK;
  if (c->x_from_h) {
    // x = q(rms(h)) for this input: in the gate GEMV where it can be (batch 1,
    // bf16), else first on its own
    const float* h = c->x_from_h;
    c->x_from_h = nullptr;
    if (c->dt == PROMOE_BF16 && launch_rows_gemv_norm(a, h, nullptr, const_cast<void*>(d_x), s)) {
      LAUNCHCHK("gate rows");
      return PROMOE_OK;
    }
    launch_rmsnorm_quant(h, const_cast<void*>(d_x), T, c->H, c->dt, s);
  }
  if (c->dt == PROMOE_BF16 && T >= 64 && c->H % 64 == 0) {
    // prefill-sized: gate and predictor rows on MFMA, the single shared-gate row as a GEMV
    RowsGemmArgs g{};
    g.w = w.wg;
    g.N = c->E;
    g.K = c->H;
    g.x = d_x;
    g.ldx = c->H;
    g.T = T;
    g.out = c->d_logits;
    g.ldo = c->ld_logits;
    if (gate) launch_gemm_rows(g, s);
    if (a.nrows[1]) {
      RowsArgs r = a;
      r.w[0] = w.sgate;
      r.nrows[0] = 1;
      r.nrows[1] = r.nrows[2] = 0;
      r.o_off = c->E;
      launch_rows_gemv(r, c->dt, c->dt, s);
    }
    if (with_pred) {
      g.w = w.pw1;
      g.N = a.nrows[2];
      g.o_off = c->pred_col;
      launch_gemm_rows(g, s);
    }
  } else {
    launch_rows_gemv(a, c->dt, c->dt, s);
  }
  LAUNCHCHK("gate rows");
  return PROMOE_OK;
}

}  // namespace

// =====================================================================
extern "C" {

const char* promoe_strerror(int err) {
  switch (err) {
    case PROMOE_OK: return "ok";
    case PROMOE_EINVAL: return "invalid argument";
    case PROMOE_ENOMEM: return "out of memory";
    case PROMOE_EHIP: return "HIP runtime error";
    case PROMOE_ESTATE: return "call order violated";
    case PROMOE_EUNSUP: return "unsupported shape";
    default: return "unknown error";
  }
}

const char* promoe_last_error_string(void) { return g_last_error.c_str(); }

// Bytes of one stored expert matrix (I x H elements).
static size_t matrix_bytes(const promoe_config* cfg) {
  const size_t n = (size_t)cfg->inter * (size_t)cfg->hidden;
  if (cfg->weight_format == PROMOE_WEIGHTS_INT4) return n / 2 + (n / kInt4Group) * 2;
  return n * (cfg->dtype == PROMOE_BF16 ? 2 : 4);
}

size_t promoe_expert_bytes(const promoe_config* cfg) {
  if (!cfg) return 0;
  return 3 * matrix_bytes(cfg);
}

int promoe_host_alloc(size_t bytes, void** out) {
  if (!out || !bytes) return PROMOE_EINVAL;
  void* p = nullptr;
  hipError_t e = hipHostMalloc(&p, bytes, hipHostMallocDefault);
  if (e != hipSuccess) return fail_hip(e, "hipHostMalloc");
  *out = p;
  return PROMOE_OK;
}

int promoe_host_free(void* p) {
  if (!p) return PROMOE_EINVAL;
  HIPCHK(hipHostFree(p));
  return PROMOE_OK;
}

int promoe_create(const promoe_config* cfg, void* d_cache, size_t cache_bytes, promoe_ctx** out) {
  if (!cfg || !d_cache || !out) return PROMOE_EINVAL;
  const promoe_config& g = *cfg;
  if (g.n_layers < 1 || g.hidden < 8 || g.inter < 8 || g.n_experts < 1 || g.top_k < 1 ||
      g.slots_per_layer < 1 || g.max_tokens < 1 || g.lookahead < 0 || g.pred_hidden < 0 || g.shared_inter < 0 ||
      (g.dtype != PROMOE_F32 && g.dtype != PROMOE_BF16) || g.top_k > g.n_experts || g.spec_fill_limit < -1 ||
      g.spec_fill_limit > 64 || ((g.flags & PROMOE_FLAG_STATIC) && g.slots_per_layer < 3) ||
      (g.weight_format != PROMOE_WEIGHTS_DENSE && g.weight_format != PROMOE_WEIGHTS_INT4)) {
    g_last_error = "invalid config";
    return PROMOE_EINVAL;
  }
  if (g.n_experts > kMaxE || g.slots_per_layer > 64 || g.top_k > kMaxK || g.hidden % 8 || g.inter % 8 ||
      g.shared_inter % 8 || g.pred_hidden % 8 || (int64_t)g.max_tokens * g.top_k > 8192 ||
      (g.weight_format == PROMOE_WEIGHTS_INT4 &&
       (g.dtype != PROMOE_BF16 || g.hidden % kInt4Group || g.inter % kInt4Group))) {
    g_last_error = "unsupported shape";
    return PROMOE_EUNSUP;
  }
  const size_t ebytes = promoe_expert_bytes(cfg);
  if (cache_bytes < (size_t)g.n_layers * g.slots_per_layer * ebytes) {
    g_last_error = "cache region too small";
    return PROMOE_EINVAL;
  }
  promoe_ctx* c = new (std::nothrow) promoe_ctx();
  if (!c) return PROMOE_ENOMEM;
  c->cfg = g;
  c->L = g.n_layers; c->H = g.hidden; c->E = g.n_experts; c->K = g.top_k; c->I = g.inter;
  c->Ish = g.shared_inter; c->C = g.slots_per_layer; c->D = g.lookahead; c->Ph = g.pred_hidden;
  c->maxT = g.max_tokens; c->dt = g.dtype; c->eb = g.dtype == PROMOE_BF16 ? 2 : 4;
  c->q4 = g.weight_format == PROMOE_WEIGHTS_INT4;
  c->chunk_bytes = matrix_bytes(&g);
  c->expert_bytes = 3 * c->chunk_bytes;
  c->cache = static_cast<uint8_t*>(d_cache);
  c->profile = (g.flags & PROMOE_FLAG_PROFILE) != 0;
  c->lw.resize(c->L);
  c->last_spec.resize(c->L);
  c->pred_host.assign(c->L, 0ull);
  c->layer_full.assign(c->L, 0);
  c->last_precise.resize(c->L);
  hipGetDevice(&c->dev);
  {
    const int rc = scratch_address(c->dev, &c->noalloc_scratch);
    if (rc) {
      delete c;
      return rc;
    }
  }

  // ---- device memory (one allocation, 256-byte aligned pieces)
  const int L = c->L, C = c->C, E = c->E, T = c->maxT, Kk = c->K, H = c->H;
  c->pred_col = E + ((c->Ish > 0 && g.shared_gate) ? 1 : 0);
  c->ld_logits = c->pred_col + std::max(c->Ph, E);
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
  const size_t o_se = take(sizeof(int32_t) * L * C), o_so = take(sizeof(int32_t) * L * E),
               o_stamp = take(sizeof(uint32_t) * L * C), o_fs = take(sizeof(uint32_t) * L * C),
               o_su = take(sizeof(int32_t) * L * C), o_clock = take(sizeof(uint32_t) * L),
               o_fseq = take(sizeof(uint32_t) * L), o_cnt = take(sizeof(int64_t) * L * kCounters),
               o_pmask = take(sizeof(uint64_t) * L),
               o_pxq = take(sizeof(float) * L * kFusedPredMaxT * kMaxE), o_pxc = take(sizeof(uint32_t) * L),
               o_logits = take(sizeof(float) * (size_t)T * c->ld_logits), o_predq = take(sizeof(float) * (size_t)T * E),
               o_pids = take(sizeof(int32_t) * (size_t)T * Kk), o_oslot = take(sizeof(int32_t) * 64),
               o_offs = take(sizeof(int32_t) * 65), o_perm = take(sizeof(int32_t) * (size_t)T * Kk),
               o_posof = take(sizeof(int32_t) * 64), o_warm = take(sizeof(int32_t) * 64),
               o_npos = take(sizeof(int32_t) * 4),
               o_act = take((size_t)c->eb * T * Kk * c->I), o_Y = take(sizeof(float) * (size_t)T * Kk * H),
               o_actsh = take((size_t)c->eb * T * std::max(c->Ish, 1)),
               o_Ysh = take(sizeof(float) * (size_t)kMaxSplit * T * H),
               o_u = take((size_t)c->eb * T * H), o_h2 = take(sizeof(float) * (size_t)T * H);
  hipError_t e = hipMalloc(&c->dmem, off);
  if (e != hipSuccess) {
    delete c;
    return fail_hip(e, "hipMalloc");
  }
  uint8_t* b = static_cast<uint8_t*>(c->dmem);
  c->st.slot_expert = reinterpret_cast<int32_t*>(b + o_se);
  c->st.slot_of = reinterpret_cast<int32_t*>(b + o_so);
  c->st.stamp = reinterpret_cast<uint32_t*>(b + o_stamp);
  c->st.fetch_seq = reinterpret_cast<uint32_t*>(b + o_fs);
  c->st.spec_unused = reinterpret_cast<int32_t*>(b + o_su);
  c->st.clock = reinterpret_cast<uint32_t*>(b + o_clock);
  c->st.fseq = reinterpret_cast<uint32_t*>(b + o_fseq);
  c->st.counters = reinterpret_cast<int64_t*>(b + o_cnt);
  c->st.pred_mask = reinterpret_cast<uint64_t*>(b + o_pmask);
  c->st.pred_xq = reinterpret_cast<float*>(b + o_pxq);
  c->st.pred_xcnt = reinterpret_cast<uint32_t*>(b + o_pxc);
  c->d_logits = reinterpret_cast<float*>(b + o_logits);
  c->d_predq = reinterpret_cast<float*>(b + o_predq);
  c->d_pred_ids = reinterpret_cast<int32_t*>(b + o_pids);
  c->d_order_slot = reinterpret_cast<int32_t*>(b + o_oslot);
  c->d_offsets = reinterpret_cast<int32_t*>(b + o_offs);
  c->d_perm = reinterpret_cast<int32_t*>(b + o_perm);
  c->d_pos_of = reinterpret_cast<int32_t*>(b + o_posof);
  c->d_warm = reinterpret_cast<int32_t*>(b + o_warm);
  c->d_npos = reinterpret_cast<int32_t*>(b + o_npos);
  c->d_act = b + o_act;
  c->d_Y = reinterpret_cast<float*>(b + o_Y);
  c->d_act_sh = b + o_actsh;
  c->d_Ysh = reinterpret_cast<float*>(b + o_Ysh);
  c->d_u = b + o_u;
  c->d_h2 = reinterpret_cast<float*>(b + o_h2);
  if (c->q4 && gemm_supported(c->I, c->H) && gemm_supported(c->H, c->I)) {
    e = hipMalloc(&c->d_stage, (size_t)kStageExperts * 3 * c->I * c->H * sizeof(bf16_t));
    if (e != hipSuccess) {
      hipFree(c->dmem);
      delete c;
      return fail_hip(e, "hipMalloc(stage)");
    }
  }

  launch_state_init(c->st, L, C, E, nullptr);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    hipFree(c->dmem);
    delete c;
    return fail_hip(e, "state init");
  }

  // ---- plan records in host-mapped memory
  void* rh = nullptr;
  e = hipHostMalloc(&rh, sizeof(PlanRecord) * kRecRing, hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    hipFree(c->dmem);
    delete c;
    return fail_hip(e, "hipHostMalloc(records)");
  }
  std::memset(rh, 0, sizeof(PlanRecord) * kRecRing);
  void* rd = nullptr;
  e = hipHostGetDevicePointer(&rd, rh, 0);
  if (e != hipSuccess) {
    hipHostFree(rh);
    hipFree(c->dmem);
    delete c;
    return fail_hip(e, "hipHostGetDevicePointer");
  }
  c->rec_h = static_cast<PlanRecord*>(rh);
  c->rec_d = static_cast<PlanRecord*>(rd);
  for (int i = 0; i < kRecRing; ++i) hipEventCreateWithFlags(&c->rec_ev[i], hipEventDisableTiming);
  hipEventCreateWithFlags(&c->route_done, hipEventDisableTiming);
  hipEventCreateWithFlags(&c->pred_in, hipEventDisableTiming);
  hipEventCreateWithFlags(&c->pred_done, hipEventDisableTiming);
  hipStreamCreateWithFlags(&c->pred_stream, hipStreamNonBlocking);

  // ---- copy engine + scheduler
  for (auto& cs : c->eng.stream) hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  c->eng.ev.resize(kCopyRing);
  for (auto& ev : c->eng.ev) hipEventCreateWithFlags(&ev, hipEventDisableTiming);
  c->cev.resize(kComputeRing);
  for (auto& ev : c->cev) hipEventCreateWithFlags(&ev, hipEventDisableTiming);
  c->eng.compute_ev = &c->cev;
  c->cstream.assign(kComputeRing, nullptr);
  c->eng.compute_stream = &c->cstream;
  const size_t sub = g.copy_subchunk_bytes > 0 ? (size_t)g.copy_subchunk_bytes : ((size_t)16 << 20);
  const int window = g.copy_window > 0 ? g.copy_window : 2;
  // A second queue only hides the per-copy setup gap, which copies of this size
  // amortise; on one queue copies land in issue order, so the first fill of a
  // step lands first instead of sharing the link until all land together.
  if (c->chunk_bytes >= kOneQueueChunkBytes) c->eng.nq = 1;
  c->pf = new Prefetcher(L, C, E, c->chunk_bytes, sub, window, c->cache, &c->eng, std::max(sub, kHighMergeBytes));
  c->pf->set_whole_expert_low((g.flags & PROMOE_FLAG_NO_CHUNK) != 0);
  if (c->profile) {
    // timing events for the first steps, so few are created inside a timed region
    for (int i = 0; i < 512; ++i) {
      hipEvent_t e = nullptr;
      if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) == hipSuccess) c->prof_free.push_back(e);
    }
  }
  c->worker = std::thread(worker_main, c);
  *out = c;
  return PROMOE_OK;
}

static int pred_host_join(promoe_ctx* c);

int promoe_sync(promoe_ctx* c) {
  if (!c) return PROMOE_EINVAL;
  const int jrc = pred_host_join(c);
  if (jrc) return jrc;
  {
    std::unique_lock<std::mutex> lk(c->mu);
    // flush speculative records and low-priority work, then wait for every copy
    for (;;) {
      while (c->rec_ingested < c->rec_pub && ingestable(c, c->rec_ingested)) {
        hipEvent_t e = c->rec_ev[c->rec_ingested % kRecRing];
        const int64_t r = c->rec_ingested;
        lk.unlock();
        hipEventSynchronize(e);
        lk.lock();
        if (c->rec_ingested == r) ingest_rec(c, r);
      }
      c->pf->pump();
      if (!c->pf->has_low() && c->pf->in_flight() == 0) break;
      const int64_t seq = c->pf->oldest_in_flight();
      if (seq >= 0) {
        hipEvent_t e = c->eng.event(seq);
        lk.unlock();
        hipEventSynchronize(e);
        lk.lock();
      }
      c->pf->retire();
    }
    if (c->eng.err != hipSuccess) return fail_hip(c->eng.err, "copy engine");
  }
  HIPCHK(hipStreamSynchronize(c->pred_stream));
  if (c->last_stream) HIPCHK(hipStreamSynchronize(c->last_stream));
  HIPCHK(hipStreamSynchronize(nullptr));
  if (c->profile) prof_resolve(c);
  return PROMOE_OK;
}

int promoe_destroy(promoe_ctx* c) {
  if (!c) return PROMOE_EINVAL;
  {
    std::lock_guard<std::mutex> lk(c->mu);
    c->stop = true;
  }
  c->cv.notify_all();
  if (c->worker.joinable()) c->worker.join();
  for (auto& cs : c->eng.stream) hipStreamSynchronize(cs);
  hipStreamSynchronize(c->pred_stream);
  hipDeviceSynchronize();
  if (c->profile) prof_resolve(c);
  for (auto& e : c->prof_free) hipEventDestroy(e);
  for (auto& e : c->eng.ev) hipEventDestroy(e);
  for (auto& e : c->cev) hipEventDestroy(e);
  for (int i = 0; i < kRecRing; ++i) hipEventDestroy(c->rec_ev[i]);
  hipEventDestroy(c->route_done);
  hipEventDestroy(c->pred_in);
  hipEventDestroy(c->pred_done);
  hipStreamDestroy(c->pred_stream);
  for (auto& cs : c->eng.stream) hipStreamDestroy(cs);
  hipHostFree(c->rec_h);
  hipFree(c->dmem);
  if (c->d_stage) hipFree(c->d_stage);
  delete c->pf;
  delete c;
  return PROMOE_OK;
}

int promoe_set_layer(promoe_ctx* c, int layer, const void* d_wgate, const float* d_bias, const void* d_pw1,
                     const void* d_pw2, const void* d_shared, const void* d_shared_gate) {
  if (!c || layer < 0 || layer >= c->L || !d_wgate) return PROMOE_EINVAL;
  if (c->cfg.router_bias && !d_bias) return PROMOE_EINVAL;
  if (c->Ish > 0 && !d_shared) return PROMOE_EINVAL;
  if (c->Ish > 0 && c->cfg.shared_gate && !d_shared_gate) return PROMOE_EINVAL;
  if (d_pw1 && c->Ph > 0 && !d_pw2) return PROMOE_EINVAL;
  LayerW& w = c->lw[layer];
  w.wg = d_wgate;
  w.bias = c->cfg.router_bias ? d_bias : nullptr;
  w.pw1 = d_pw1;
  w.pw2 = c->Ph > 0 ? d_pw2 : nullptr;
  w.shared = c->Ish > 0 ? d_shared : nullptr;
  w.sgate = (c->Ish > 0 && c->cfg.shared_gate) ? d_shared_gate : nullptr;
  return PROMOE_OK;
}

int promoe_set_attn(promoe_ctx* c, int layer, const void* d_wattn) {
  if (!c || layer < 0 || layer >= c->L || !d_wattn) return PROMOE_EINVAL;
  c->lw[layer].attn = d_wattn;
  return PROMOE_OK;
}

int promoe_set_expert_host(promoe_ctx* c, int layer, int expert, const void* h_pinned) {
  if (!c || layer < 0 || layer >= c->L || expert < 0 || expert >= c->E || !h_pinned) return PROMOE_EINVAL;
  std::lock_guard<std::mutex> lk(c->mu);
  c->pf->set_host(layer, expert, static_cast<const uint8_t*>(h_pinned));
  return PROMOE_OK;
}

int promoe_set_initial_cache(promoe_ctx* c, int layer, const int32_t* h_experts, int n) {
  if (!c || layer < 0 || layer >= c->L || n < 0 || n > c->C || (n && !h_experts)) return PROMOE_EINVAL;
  if (c->lw[layer].planned) {
    g_last_error = "initial cache after the first plan";
    return PROMOE_ESTATE;
  }
  std::vector<int> seen(c->E, 0);
  for (int i = 0; i < n; ++i) {
    if (h_experts[i] < 0 || h_experts[i] >= c->E || seen[h_experts[i]]++) return PROMOE_EINVAL;
    if (!c->pf->host(layer, h_experts[i])) {
      g_last_error = "expert host buffer not set";
      return PROMOE_ESTATE;
    }
  }
  for (int i = 0; i < n; ++i) {
    uint8_t* dst = c->cache + ((size_t)layer * c->C + i) * c->expert_bytes;
    HIPCHK(hipMemcpy(dst, c->pf->host(layer, h_experts[i]), c->expert_bytes, hipMemcpyHostToDevice));
  }
  HIPCHK(hipMemcpy(c->d_warm, h_experts, sizeof(int32_t) * n, hipMemcpyHostToDevice));
  launch_warm(c->st, layer, c->C, c->E, c->d_warm, n, nullptr);
  LAUNCHCHK("warm");
  HIPCHK(hipDeviceSynchronize());
  const bool full = c->C == c->E && n == c->E;
  if (full != (c->layer_full[layer] != 0)) {
    c->layer_full[layer] = full;
    c->n_full_layers += full ? 1 : -1;
  }
  std::lock_guard<std::mutex> lk(c->mu);
  for (int i = 0; i < n; ++i) c->pf->mark_resident(layer, i, h_experts[i]);
  return PROMOE_OK;
}

static int predict_tail(promoe_ctx* c, int layer, int target, int T, int32_t* d_pred_ids, int32_t* h_q,
                        int32_t* n_q, hipStream_t s, int64_t* rec_out);
static int finish_spec(promoe_ctx* c, int target, int64_t r, hipStream_t s, int32_t* h_q, int32_t* n_q,
                       int64_t* rec_out);

// The host waits for the spec plan that ends a prediction of promoe_route_predict:
// the side stream's kernels before it are then complete too.
static int pred_host_join(promoe_ctx* c) {
  if (c->pred_host_rec < 0) return PROMOE_OK;
  const int64_t r = c->pred_host_rec;
  c->pred_host_rec = -1;
  const hipError_t e = wait_record(c, r);
  return e == hipSuccess ? PROMOE_OK : fail_hip(e, "prediction");
}

// Order stream s after the predictor's side-stream work (its reads of the
// predictor rows in d_logits, its writes of the predicted ids and of the
// target layer's cache state), unless s already waited for it.
static hipError_t pred_join(promoe_ctx* c, hipStream_t s) {
  if (c->pred_nojoin || (!c->pred_pending && c->pred_joined == s)) return hipSuccess;
  const hipError_t e = hipStreamWaitEvent(s, c->pred_done, 0);
  if (e == hipSuccess) {
    c->pred_pending = false;
    c->pred_joined = s;
  }
  return e;
}

// The prediction of `layer` on stream s (routed: no route will need this
// layer's gate logits on this input any more, so only predictor rows are
// computed).  join_now: s waits for the side stream before the call returns;
// else, with host_join, the next call that needs it waits on the host for the
// spec plan's record, and without, the layer's FFN call joins it on the device
// (after its last launch).
static int predict_launch(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_pred_ids, int32_t* h_q,
                          int32_t* n_q, hipStream_t s, bool routed, bool join_now, bool host_join = true) {
  int rc = pred_host_join(c);
  if (rc) return rc;
  HIPCHK(pred_join(c, s));
  const int target = layer + c->D;
  const bool has_pred = target < c->L && c->lw[layer].pw1 != nullptr;
  const bool rows_ready =
      has_pred && c->pred_rows_layer == layer && c->pred_rows_x == d_x && c->pred_rows_T == T;
  c->pred_rows_layer = -1;
  if (!rows_ready) {
    rc = launch_gate_rows(c, layer, d_x, T, has_pred, s, !routed);
    if (rc) return rc;
    if (!routed) {
      c->gate_layer = layer;
      c->gate_x = d_x;
      c->gate_T = T;
    }
  }
  if (n_q) *n_q = 0;
  if (!has_pred) return PROMOE_OK;
  // Fork: the rest reads the predictor rows (and the cache state of the target
  // layer, which no launch on s touches before the join below).
  if (!rows_ready) HIPCHK(hipEventRecord(c->pred_in, s));
  hipStream_t ps = c->pred_stream;
  HIPCHK(hipStreamWaitEvent(ps, c->pred_in, 0));
  int64_t spec_rec;
  rc = predict_tail(c, layer, target, T, d_pred_ids, h_q, n_q, ps, &spec_rec);
  if (!rc && !join_now && host_join && spec_rec >= 0) {
    // the spec plan's record marks the end of the side stream's work (earlier
    // side-stream work was joined at the top of this call)
    c->pred_host_rec = spec_rec;
    c->pred_nojoin = true;
    return PROMOE_OK;
  }
  // Join: whatever s runs after it (the caller's reads of the predicted ids, the
  // next gate launch over d_logits, the target layer's route) follows it.
  hipError_t je = hipEventRecord(c->pred_done, ps);
  if (je == hipSuccess) {
    c->pred_nojoin = false;
    c->pred_pending = true;
    c->pred_joined = nullptr;
    if (join_now) je = pred_join(c, s);
  }
  if (rc) return rc;
  if (je != hipSuccess) return fail_hip(je, "predictor join");
  return PROMOE_OK;
}

int promoe_predict(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_pred_ids, int32_t* h_q,
                   int32_t* n_q, void* stream) {
  if (!c || layer < 0 || layer >= c->L || !d_x || !c->lw[layer].wg) return PROMOE_EINVAL;
  int rc = check_tokens(c, T);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  c->last_stream = s;
  const int target = layer + c->D;
  if (target < c->L && c->lw[layer].pw1 && c->route_layer == target) {
    g_last_error = "prediction for a layer whose route is not consumed";
    return PROMOE_ESTATE;
  }
  // After route(layer) on the same input (its FFN call done or not) no route
  // needs this layer's gate logits any more.
  const bool routed = c->last_route_layer == layer && c->route_x == d_x && c->route_T == T;
  return predict_launch(c, layer, d_x, T, d_pred_ids, h_q, n_q, s, routed, true);
}

static int predict_tail(promoe_ctx* c, int layer, int target, int T, int32_t* d_pred_ids, int32_t* h_q,
                        int32_t* n_q, hipStream_t s, int64_t* rec_out) {
  int rc;
  *rec_out = -1;
  int32_t* pids = d_pred_ids ? d_pred_ids : c->d_pred_ids;
  const bool plan = !(c->cfg.flags & PROMOE_FLAG_NO_PREFETCH);
  // Decode-sized steps: the predictor's second layer, top-k and the spec plan
  // in one launch.
  const bool fused = plan && T <= kFusedPredMaxT && c->Ph <= kFusedPredMaxHidden &&
                     (c->Ph == 0 || reinterpret_cast<uintptr_t>(c->lw[layer].pw2) % 16 == 0);
  if (fused) {
    int64_t r;
    rc = new_record(c, 0, PROMOE_PRIO_LOW, &r);
    if (rc) return rc;
    PredictPlanArgs pp{};
    pp.plan = plan_args(c, target, pids, T, r);
    if (c->cfg.flags & PROMOE_FLAG_FILL_BY_DEADLINE) pp.plan.fill_budget = deadline_fill_budget(c);
    pp.h = c->d_logits + c->pred_col;
    pp.ldh = c->ld_logits;
    pp.Ph = c->Ph;
    pp.w2 = c->lw[layer].pw2;
    pp.w2_bf16 = c->dt == PROMOE_BF16;
    pp.pred_ids = pids;
    launch_predict_plan(pp, s);
    return finish_spec(c, target, r, s, h_q, n_q, rec_out);
  }
  TopkArgs tk{};
  if (c->Ph > 0) {
    RowsArgs a{};
    a.w[0] = c->lw[layer].pw2;
    a.nrows[0] = c->E;
    a.K = c->Ph;
    a.x = c->d_logits;
    a.ldx = c->ld_logits;
    a.x_off = c->pred_col;
    a.T = T;
    a.out = c->d_predq;
    a.ldo = c->E;
    a.relu_in = 1;
    launch_rows_gemv(a, c->dt, PROMOE_F32, s);
    tk.logits = c->d_predq;
    tk.ld = c->E;
  } else {
    tk.logits = c->d_logits + c->pred_col;
    tk.ld = c->ld_logits;
  }
  tk.E = c->E;
  tk.k = c->K;
  tk.T = T;
  tk.ids = pids;
  tk.want_weights = 0;
  tk.sgate_col = -1;
  launch_topk(tk, s);
  LAUNCHCHK("predictor");
  if (!plan) return PROMOE_OK;
  int64_t r;
  rc = new_record(c, 0, PROMOE_PRIO_LOW, &r);
  if (rc) return rc;
  PlanArgs pa = plan_args(c, target, pids, T, r);
  if (c->cfg.flags & PROMOE_FLAG_FILL_BY_DEADLINE) pa.fill_budget = deadline_fill_budget(c);
  launch_plan_spec(pa, s);
  return finish_spec(c, target, r, s, h_q, n_q, rec_out);
}

// After a spec plan's launch on s: its record's event, publication, and the
// optional host copy of the list.
static int finish_spec(promoe_ctx* c, int target, int64_t r, hipStream_t s, int32_t* h_q, int32_t* n_q,
                       int64_t* rec_out) {
  hipError_t le = hipGetLastError();
  if (le == hipSuccess) le = hipEventRecord(c->rec_ev[r % kRecRing], s);
  publish(c, r);
  if (le != hipSuccess) return fail_hip(le, "plan_spec");
  *rec_out = r;
  c->lw[target].planned = true;
  if (h_q || n_q) {
    HIPCHK(hipEventSynchronize(c->rec_ev[r % kRecRing]));
    const PlanRecord& rec = c->rec_h[r % kRecRing];
    if (n_q) *n_q = rec.n;
    if (h_q)
      for (int i = 0; i < rec.n; ++i) h_q[i] = rec.expert[i];
  }
  return PROMOE_OK;
}

int promoe_prefetch(promoe_ctx* c, int target_layer, const int32_t* h_ids, int n, int prio, void* stream) {
  if (!c || target_layer < 0 || target_layer >= c->L || n < 0 || n > c->C || (n && !h_ids)) return PROMOE_EINVAL;
  if (prio != PROMOE_PRIO_LOW && prio != PROMOE_PRIO_HIGH) return PROMOE_EINVAL;
  std::vector<int> seen(c->E, 0);
  for (int i = 0; i < n; ++i)
    if (h_ids[i] < 0 || h_ids[i] >= c->E || seen[h_ids[i]]++) return PROMOE_EINVAL;
  if (c->route_layer == target_layer) {
    g_last_error = "prefetch for a layer whose route is not consumed";
    return PROMOE_ESTATE;
  }
  if (c->cfg.flags & PROMOE_FLAG_NO_PREFETCH) return PROMOE_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  c->last_stream = s;
  // a prediction may still be planning on the side stream
  int rc = pred_host_join(c);
  if (rc) return rc;
  HIPCHK(pred_join(c, s));
  int64_t r;
  rc = new_record(c, 0, prio, &r);
  if (rc) return rc;
  PlanRecord& rec = c->rec_h[r % kRecRing];
  rec.n_q_in = n;
  for (int i = 0; i < n; ++i) rec.q_in[i] = h_ids[i];
  launch_plan_spec(plan_args(c, target_layer, nullptr, 0, r), s);
  hipError_t le = hipGetLastError();
  if (le == hipSuccess) le = hipEventRecord(c->rec_ev[r % kRecRing], s);
  publish(c, r);
  if (le != hipSuccess) return fail_hip(le, "plan_spec");
  c->lw[target_layer].planned = true;
  return PROMOE_OK;
}

static int launch_route_head(promoe_ctx* c, int layer, const void* d_x, int T, hipStream_t s);
static int early_resident_launch(promoe_ctx* c, int layer, const void* d_x, int T, hipStream_t s, int64_t r,
                                 bool* launched);
static void early_resident_release(promoe_ctx* c, int layer, int T, hipStream_t s);

// The route of `layer`; with_pred: also the layer's prediction, launched while
// the host waits for the precise plan.
static int route_impl(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                      float* d_shared_scale, int32_t* h_order, int32_t* n_order, hipStream_t s, bool with_predict,
                      int32_t* d_pred_ids);

int promoe_route(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                 float* d_shared_scale, int32_t* h_order, int32_t* n_order, void* stream) {
  return route_impl(c, layer, d_x, T, d_ids, d_w, d_shared_scale, h_order, n_order,
                    static_cast<hipStream_t>(stream), false, nullptr);
}

int promoe_route_predict(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                         float* d_shared_scale, int32_t* d_pred_ids, int32_t* h_order, int32_t* n_order,
                         void* stream) {
  if (c && c->D == 0) {
    g_last_error = "promoe_route_predict needs a look-ahead of at least 1";
    return PROMOE_EINVAL;
  }
  return route_impl(c, layer, d_x, T, d_ids, d_w, d_shared_scale, h_order, n_order,
                    static_cast<hipStream_t>(stream), true, d_pred_ids);
}

static int route_impl(promoe_ctx* c, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                      float* d_shared_scale, int32_t* h_order, int32_t* n_order, hipStream_t s, bool with_predict,
                      int32_t* d_pred_ids) {
  if (!c || layer < 0 || layer >= c->L || !d_x || !d_ids || !d_w || !c->lw[layer].wg) return PROMOE_EINVAL;
  if (c->cfg.shared_gate && c->Ish > 0 && !d_shared_scale) return PROMOE_EINVAL;
  int rc = check_tokens(c, T);
  if (rc) return rc;
  if (c->route_layer >= 0) {
    g_last_error = "previous route not consumed by promoe_expert_ffn";
    return PROMOE_ESTATE;
  }
  c->last_stream = s;
  rc = pred_host_join(c);
  if (rc) return rc;
  HIPCHK(pred_join(c, s));
  // plans of earlier lazy routes that have completed
  if (c->all_resident()) HIPCHK(drain_records(c, false));
  {
    const auto now = std::chrono::steady_clock::now();
    if (c->have_route_t) {
      const double dt = std::chrono::duration<double>(now - c->last_route_t).count();
      if (dt < 1.0) c->route_dt_ema = c->route_dt_ema > 0.0 ? 0.8 * c->route_dt_ema + 0.2 * dt : dt;
    }
    c->last_route_t = now;
    c->have_route_t = true;
  }
  if (c->x_from_h && c->gate_layer == layer && c->gate_x == d_x && c->gate_T == T) {
    // gate logits already computed on this input: x itself still to be formed
    launch_rmsnorm_quant(c->x_from_h, const_cast<void*>(d_x), T, c->H, c->dt, s);
    c->x_from_h = nullptr;
  }
  // A route that will not wait for its plan (lazy, below) has the host take the
  // record in on the plan's event: the kernel skips the fence and done word
  // that a host poll needs, which sit on the path to the expert launches.  A
  // decode-sized route that brings its layer's prediction runs it as a second
  // block of the plan kernel: no side stream to fork and join, and the host
  // still sees the precise plan as soon as its block has written it.
  const bool in_order = (c->cfg.flags & (PROMOE_FLAG_NO_REORDER | PROMOE_FLAG_NO_PREEMPT)) != 0;
  const bool lazy_plan = c->all_resident() && !h_order && !n_order && !in_order && (int64_t)T * c->K <= 64 &&
                         T < kGemmMinTokens && !c->noalloc_call;
  const int target = layer + c->D;
  const bool pred_in_plan = with_predict && c->D > 0 && target < c->L && c->lw[layer].pw1 &&
                            !(c->cfg.flags & PROMOE_FLAG_NO_PREFETCH) && T <= kFusedPredMaxT &&
                            c->Ph <= kFusedPredMaxHidden &&
                            (c->Ph == 0 || reinterpret_cast<uintptr_t>(c->lw[layer].pw2) % 16 == 0) &&
                            (int64_t)T * c->K <= kFusedRouteMaxPairs;
  if (!(c->gate_layer == layer && c->gate_x == d_x && c->gate_T == T)) {
    // With a look-ahead the layer's prediction follows its route on the same
    // input: its first predictor rows ride in the gate launch, and the side
    // stream of the predictor starts from this point.
    const bool with_pred = c->D > 0 && layer + c->D < c->L && c->lw[layer].pw1 &&
                           !(c->cfg.flags & PROMOE_FLAG_NO_PREFETCH);
    rc = launch_gate_rows(c, layer, d_x, T, with_pred, s);
    if (rc) return rc;
    c->pred_rows_layer = -1;
    if (with_pred && !pred_in_plan) {
      HIPCHK(hipEventRecord(c->pred_in, s));
      c->pred_rows_layer = layer;
      c->pred_rows_x = d_x;
      c->pred_rows_T = T;
    }
  }
  c->gate_layer = -1;
  TopkArgs tk{};
  tk.logits = c->d_logits;
  tk.ld = c->ld_logits;
  tk.E = c->E;
  tk.k = c->K;
  tk.T = T;
  tk.bias = c->lw[layer].bias;
  tk.renorm = c->cfg.renorm;
  tk.want_weights = 1;
  tk.ids = d_ids;
  tk.w = d_w;
  const bool sg = c->cfg.shared_gate && c->Ish > 0;
  tk.sgate_col = sg ? c->E : -1;
  tk.sscale = sg ? d_shared_scale : nullptr;
  int64_t r, r_spec = -1;
  rc = new_record(c, 1, PROMOE_PRIO_HIGH, &r);
  if (rc) return rc;
  if (pred_in_plan && (rc = new_record(c, 0, PROMOE_PRIO_LOW, &r_spec))) {
    publish(c, r);
    return rc;
  }
  // A lazy one-token route (every expert resident, nobody waiting on the plan)
  // has its prediction ride in the resident gate/up launch that follows the
  // plan kernel, beside that launch's row tiles, instead of in the plan
  // kernel, where the prediction's chain outlasts the plan's and holds back
  // the expert launches.
  const bool ride = pred_in_plan && lazy_plan && T == 1 && c->dt == PROMOE_BF16 && !c->q4;
  if (pred_in_plan) {
    PlanArgs pa = plan_args(c, layer, d_ids, T, r);
    pa.host_done = lazy_plan ? 0 : 1;
    PredictPlanArgs pp{};
    int32_t* pids = d_pred_ids ? d_pred_ids : c->d_pred_ids;
    pp.plan = plan_args(c, target, pids, T, r_spec);
    pp.plan.host_done = lazy_plan ? 0 : 1;
    if (c->cfg.flags & PROMOE_FLAG_FILL_BY_DEADLINE) pp.plan.fill_budget = deadline_fill_budget(c);
    pp.h = c->d_logits + c->pred_col;
    pp.ldh = c->ld_logits;
    pp.Ph = c->Ph;
    pp.w2 = c->lw[layer].pw2;
    pp.w2_bf16 = c->dt == PROMOE_BF16;
    pp.pred_ids = pids;
    if (ride) {
      launch_route_plan(tk, pa, s);
      c->ride = pp;
      c->ride_pred = true;
    } else {
      launch_route_plan_predict(tk, pa, pp, s);
    }
    c->pred_rows_layer = -1;
  } else if ((int64_t)T * c->K <= kFusedRouteMaxPairs) {
    PlanArgs pa = plan_args(c, layer, d_ids, T, r);
    pa.host_done = lazy_plan ? 0 : 1;
    launch_route_plan(tk, pa, s);
  } else {
    launch_topk(tk, s);
    launch_plan_precise(plan_args(c, layer, d_ids, T, r), s);
  }
  hipError_t le = hipGetLastError();
  if (le == hipSuccess) le = hipEventRecord(c->rec_ev[r % kRecRing], s);
  if (r_spec >= 0 && !ride) {
    // the prediction's record completes with the same kernel
    if (le == hipSuccess) le = hipEventRecord(c->rec_ev[r_spec % kRecRing], s);
    publish(c, r_spec);
    c->lw[target].planned = true;
  }
  bool early_ffn = false, lazy = false;
  if (le == hipSuccess) {
    rc = early_resident_launch(c, layer, d_x, T, s, r, &early_ffn);
    if (ride && !rc) {
      // the resident launch carried the prediction, or it runs on its own now;
      // its record completes with that launch
      if (c->ride_pred) launch_predict_plan(c->ride, s);
      c->ride_pred = false;
      le = hipGetLastError();
      if (le == hipSuccess) le = hipEventRecord(c->rec_ev[r_spec % kRecRing], s);
      if (le != hipSuccess) rc = fail_hip(le, "prediction");
    }
  }
  if (ride) {
    c->ride_pred = false;
    publish(c, r_spec);
    c->lw[target].planned = true;
  }
  if (le == hipSuccess) {
    // every expert resident: the resident launch covers the step, and the
    // caller does not ask for the order, so the plan is taken in later
    lazy = !rc && early_ffn && c->all_resident() && !h_order && !n_order;
    // the prediction's launches (on the side stream) fill the host's wait for the plan
    if (!rc && with_predict && !pred_in_plan)
      rc = predict_launch(c, layer, d_x, T, d_pred_ids, nullptr, nullptr, s, true, false, !lazy);
    if (rc) {
      publish(c, r);
      return rc;
    }
  }
  if (lazy) {
    {
      std::lock_guard<std::mutex> lk(c->mu);
      const int i = (int)(r % kRecRing);
      c->rec_lazy[i] = true;
      c->lazy_T[i] = T;
      c->lazy_prof0[i] = c->early_prof0;
      c->lazy_nprof[i] = c->early_nprof;
      c->early_nprof = 0;
      // its resident launch ran every position and the shared expert: the FFN
      // call has no position to launch
      c->ffn_started.clear();
      c->deferred.clear();
      c->need01.clear();
      c->need2.clear();
      c->need_q.clear();
      c->shared_started = c->Ish > 0;
    }
    publish(c, r);
    c->lw[layer].planned = true;
    HIPCHK(hipEventRecord(c->route_done, s));
    c->route_stream = s;
    c->route_lazy = true;
    c->n_lazy_routes++;
    c->route_layer = layer;
    c->last_route_layer = layer;
    c->route_T = T;
    c->route_x = d_x;
    return PROMOE_OK;
  }
  if (le == hipSuccess) le = wait_record(c, r);
  publish(c, r);
  if (le != hipSuccess) return fail_hip(le, "plan_precise");
  c->lw[layer].planned = true;

  std::unique_lock<std::mutex> lk(c->mu);
  while (c->rec_ingested < r) {  // earlier plans on the same stream: complete
    HIPCHK(wait_record(c, c->rec_ingested));
    ingest_rec(c, c->rec_ingested);
  }
  const PlanRecord rec = c->rec_h[r % kRecRing];
  c->rec_ingested = r + 1;
  c->last_precise[layer] = rec;
  const bool early = !(c->cfg.flags & PROMOE_FLAG_NO_PREEMPT);
  if (early) c->pf->purge_low(layer);
  c->pf->retire();  // completions so far, for the in-time count below
  const uint64_t predicted = c->pred_host[layer];
  c->pred_host[layer] = 0ull;
  c->need01.assign(rec.n, -1);
  c->need2.assign(rec.n, -1);
  c->need_q.assign(rec.n, 0);
  c->deferred.clear();
  for (int pos = 0; pos < rec.n; ++pos) {
    const int slot = rec.slot[pos];
    const bool fill = rec.flag[pos] != 0;
    // Without early preemption a copy starts when its position is reached, after
    // the previous position's compute (positions then run in order, so this also
    // follows any earlier reader of the slot).
    if (!early && pos > 0 && (fill || c->pf->ready_seq(layer, slot, 2) == -2)) {
      c->deferred.push_back(Deferred{pos, slot, rec.expert[pos], pos - 1, fill});
      continue;
    }
    if (fill && rec.after[pos] >= 0) {
      c->deferred.push_back(Deferred{pos, slot, rec.expert[pos], rec.after[pos], true});
      continue;
    }
    if (fill) c->pf->assign(layer, slot, rec.expert[pos]);
    c->pf->issue_high(layer, slot);
    c->need01[pos] = c->pf->ready_seq(layer, slot, 1);
    c->need2[pos] = c->pf->ready_seq(layer, slot, 2);
    c->need_q[pos] = c->pf->queue_of(layer, slot);
    if (((predicted >> rec.expert[pos]) & 1ull) && c->need01[pos] == -1 && c->need2[pos] == -1) c->pred_in_time++;
  }
  c->route_rec = rec;
  c->ffn_started.assign(rec.n, 0);
  c->shared_started = false;
  if (early_ffn) early_resident_release(c, layer, T, s);
  rc = launch_route_head(c, layer, d_x, T, s);
  if (rc) return rc;
  if (c->eng.err != hipSuccess) return fail_hip(c->eng.err, "copy engine");
  // the FFN call reads what the route's kernels wrote (ids, weights, the plan's
  // slots and permutation): one on another stream waits for this event
  HIPCHK(hipEventRecord(c->route_done, s));
  c->route_stream = s;
  lk.unlock();
  c->cv.notify_all();
  c->route_layer = layer;
  c->last_route_layer = layer;
  c->route_T = T;
  c->route_x = d_x;
  c->route_rec = rec;
  if (h_order)
    for (int i = 0; i < rec.n; ++i) h_order[i] = rec.expert[i];
  if (n_order) *n_order = rec.n;
  return PROMOE_OK;
}

namespace {

// Launch the gate/up and down passes over a list of jobs (route positions, or
// kSharedJob), waiting first for copies `wait01` (chunks 0-1 of every job) and
// then `wait2` (chunk 2).  Jobs with >= kGemmMinTokens pairs go to the MFMA
// GEMM (bf16, tile-aligned shapes), the rest to the GEMV kernels.

int ffn_launch_one(promoe_ctx* c, FfnArgs a, const std::vector<int>& jobs, hipStream_t s, const CopyWait& wait01,
                   const CopyWait& wait2, bool gemm, const bf16_t* stage = nullptr) {
  const PlanRecord& rec = c->route_rec;
  int maxc = 1;
  double wbytes = 0, flops = 0;
  a.n_jobs = (int)jobs.size();
  for (size_t i = 0; i < jobs.size(); ++i) {
    const bool sh = jobs[i] == kSharedJob;
    FfnJob& jb = a.jobs[i];
    jb.pos = jobs[i];
    jb.r0 = 0;
    jb.pad = 0;
    if (sh) {
      jb.w = a.shared_w;
      jb.q0 = 0;
      jb.q1 = a.T;
      jb.I = c->Ish;
    } else {
      jb.w = stage ? static_cast<const void*>(stage + i * 3 * (size_t)c->I * c->H)
                   : static_cast<const void*>(c->cache + ((size_t)a.layer * c->C + rec.slot[jobs[i]]) * c->expert_bytes);
      jb.q0 = rec.offset[jobs[i]];
      jb.q1 = rec.offset[jobs[i] + 1];
      jb.I = c->I;
    }
    const int cnt = sh ? a.T : rec.count[jobs[i]];
    const double melems = (double)(sh ? c->Ish : c->I) * c->H;
    maxc = std::max(maxc, cnt);
    wbytes += (a.q4 && !stage) ? (double)c->chunk_bytes : melems * c->eb;  // bytes the kernel reads
    flops += 2.0 * cnt * melems;
  }
  for (int pass = 0; pass < 2; ++pass) {
    const CopyWait& w = pass == 0 ? wait01 : wait2;
    bool any = false;
    for (int64_t q : w.seq) any = any || q >= 0;
    if (any) {
      hipEvent_t pa = nullptr, pb = nullptr;
      const bool prof = c->profile && !c->noalloc_call;
      if (prof) { pa = prof_event(c); pb = prof_event(c); hipEventRecord(pa, s); }
      for (int64_t q : w.seq)
        if (q >= 0) HIPCHK(hipStreamWaitEvent(s, c->eng.event(q), 0));
      if (prof) { hipEventRecord(pb, s); c->prof_pending.push_back(ProfEntry{pa, pb, kStallClass, 0, 0}); }
    }
    const double k = pass == 0 ? 2.0 : 1.0;  // gate and up, or down
    const bool shared_only = jobs.size() == 1 && jobs[0] == kSharedJob;
    const int cls = (gemm ? (shared_only ? 4 : 2) : 0) + pass;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (c->profile && !c->noalloc_call) {
      e0 = prof_event(c);
      e1 = prof_event(c);
      c->prof_pending.push_back(ProfEntry{e0, e1, cls, k * wbytes, k * flops});
    }
    if (gemm) launch_gemm(a, pass, maxc, s, e0, e1);
    else launch_ffn(a, pass, maxc, c->dt, s, e0, e1);
    LAUNCHCHK("ffn");
  }
  return PROMOE_OK;
}

bool use_gemm(promoe_ctx* c, int tokens, bool shared) {
  if (c->dt != PROMOE_BF16 || tokens < kGemmMinTokens) return false;
  const int I = shared ? c->Ish : c->I;
  return gemm_supported(I, c->H) && gemm_supported(c->H, I);
}

int ffn_launch(promoe_ctx* c, FfnArgs a, const std::vector<int>& jobs, hipStream_t s, const CopyWait& wait01,
               const CopyWait& wait2) {
  // split by kernel family; the shared expert (M = T) gets its own GEMM launch
  // so the routed groups can use the small-M tile
  // 4-bit routed experts go to the dequantising GEMV, or -- with enough tokens --
  // are expanded to bf16 and run on the MFMA GEMM (the shared expert stays dense)
  std::vector<int> gv, gm, sh, gq, gqm;
  for (int p : jobs) {
    const bool is_sh = p == kSharedJob;
    const int cnt = is_sh ? a.T : c->route_rec.count[p];
    if (c->q4 && !is_sh) (c->d_stage && !c->noalloc_call && use_gemm(c, cnt, false) ? gqm : gq).push_back(p);
    else if (!use_gemm(c, cnt, is_sh)) gv.push_back(p);
    else if (is_sh) sh.push_back(p);
    else gm.push_back(p);
  }
  int rc = PROMOE_OK;
  if (!sh.empty() && (rc = ffn_launch_one(c, a, sh, s, wait01, wait2, true))) return rc;
  if (!gm.empty() && (rc = ffn_launch_one(c, a, gm, s, wait01, wait2, true))) return rc;
  if (!gv.empty() && (rc = ffn_launch_one(c, a, gv, s, wait01, wait2, false))) return rc;
  if (!gq.empty()) {
    FfnArgs q = a;
    q.q4 = 1;
    if ((rc = ffn_launch_one(c, q, gq, s, wait01, wait2, false))) return rc;
  }
  // staged: every copy of the batch before the expansion, then two GEMM passes
  for (size_t b0 = 0; b0 < gqm.size(); b0 += kStageExperts) {
    const std::vector<int> batch(gqm.begin() + b0, gqm.begin() + std::min(gqm.size(), b0 + kStageExperts));
    CopyWait w;
    for (int q = 0; q < kCopyStreams; ++q) w.seq[q] = std::max(wait01.seq[q], wait2.seq[q]);
    for (int64_t q : w.seq)
      if (q >= 0) HIPCHK(hipStreamWaitEvent(s, c->eng.event(q), 0));
    DequantArgs d{};
    d.dst = c->d_stage;
    d.n = (int)batch.size();
    d.inter = c->I;
    d.hidden = c->H;
    for (size_t i = 0; i < batch.size(); ++i)
      d.src[i] = c->cache + ((size_t)a.layer * c->C + c->route_rec.slot[batch[i]]) * c->expert_bytes;
    launch_dequant_q4(d, s);
    LAUNCHCHK("dequant");
    if ((rc = ffn_launch_one(c, a, batch, s, CopyWait(), CopyWait(), true, c->d_stage))) return rc;
  }
  return PROMOE_OK;
}

}  // namespace

namespace {

FfnArgs ffn_args(promoe_ctx* c, int layer, const void* d_x, int T) {
  FfnArgs a{};
  a.cache = c->cache;
  a.expert_bytes = (int64_t)c->expert_bytes;
  a.layer = layer;
  a.slots = c->C;
  a.order_slot = c->d_order_slot;
  a.offsets = c->d_offsets;
  a.perm = c->d_perm;
  a.hidden = c->H;
  a.inter = c->I;
  a.top_k = c->K;
  a.T = T;
  a.x = d_x;
  a.act = c->d_act;
  a.Y = c->d_Y;
  a.shared_inter = c->Ish;
  a.shared_w = c->lw[layer].shared;
  a.act_sh = c->d_act_sh;
  a.Ysh = c->d_Ysh;
  // The shared expert's down GEMM has few output tiles; split its reduction so
  // the launch covers the CUs (gemm_shared_down_split).  Slices write separate
  // partial outputs that the combine adds in slice order (deterministic).
  a.ksplit = 1;
  a.ysh_split_stride = (int64_t)T * c->H;
  if (c->Ish > 0 && use_gemm(c, T, true))
    a.ksplit = std::max(1, std::min(std::min(gemm_shared_down_split(T, c->H), kMaxSplit), c->Ish / 64 / 4));
  return a;
}

// A launch reading route positions `jobs` was enqueued on s: it becomes the
// last read of their slots, and the fills that waited for it are issued.
// Caller holds c->mu.  Returns the launch's compute token.
int64_t release_after_launch(promoe_ctx* c, int layer, const std::vector<int>& jobs, hipStream_t s) {
  const PlanRecord& rec = c->route_rec;
  const int64_t tok = record_compute(c, s);
  for (int p : jobs)
    if (p != kSharedJob) c->pf->set_last_read(layer, rec.slot[p], tok);
  for (auto it = c->deferred.begin(); it != c->deferred.end();) {
    const Deferred d = *it;
    if (std::find(jobs.begin(), jobs.end(), d.after) == jobs.end()) {
      ++it;
      continue;
    }
    if (d.fill) c->pf->assign(layer, d.slot, d.expert);
    c->pf->issue_high_after(layer, d.slot, tok);
    c->need01[d.pos] = c->pf->ready_seq(layer, d.slot, 1);
    c->need2[d.pos] = c->pf->ready_seq(layer, d.slot, 2);
    c->need_q[d.pos] = c->pf->queue_of(layer, d.slot);
    it = c->deferred.erase(it);
  }
  return tok;
}

std::vector<FillWait> fill_waits(const promoe_ctx* c) {
  std::vector<FillWait> w;
  w.reserve(c->deferred.size());
  for (const auto& d : c->deferred) w.push_back(FillWait{d.pos, d.after, d.fill});
  return w;
}

}  // namespace

// Decode-sized steps: the FFN of the resident positions and the shared expert
// is enqueued right behind the precise plan, before the host has seen the plan,
// with every route position resolved on the device (FfnJob::w == null): the
// reordered plan puts the resident experts first and writes their count, slots
// and pair ranges to device memory.  Only slots with no copy pending can be
// read that early, so the spec plans queued for the layer must all have been
// ingested (their plan kernels done) and the slots whose bytes are not all
// known to have landed are passed as busy_mask and skipped; the host replays
// the same rule once the plan is known (early_resident_release).  The route's
// host round trip then overlaps the experts' compute instead of preceding it.
static int early_resident_launch(promoe_ctx* c, int layer, const void* d_x, int T, hipStream_t s, int64_t r,
                                 bool* launched) {
  *launched = false;
  const bool in_order = (c->cfg.flags & (PROMOE_FLAG_NO_REORDER | PROMOE_FLAG_NO_PREEMPT)) != 0;
  if (in_order || (int64_t)T * c->K > 64 || T >= kGemmMinTokens || c->noalloc_call) return PROMOE_OK;
  uint64_t busy = 0;
  if (!c->all_resident()) {
    // Earlier plans must be on the host first (their fills decide which slots
    // are busy): they are speculative ones (a precise one would still await its
    // FFN call), and a spec plan published before this route was queued ahead
    // of it, so waiting for it costs at most the wait for this route's plan.
    // (With every expert resident no plan fills a slot and none is busy.)
    std::unique_lock<std::mutex> lk(c->mu);
    const int64_t first = c->rec_ingested;
    for (int64_t rr = first; rr < r; ++rr)
      if (!ingestable(c, rr) || rr >= c->rec_pub) return PROMOE_OK;
    lk.unlock();
    for (int64_t rr = first; rr < r; ++rr) {
      const hipError_t e = wait_record(c, rr);
      if (e != hipSuccess) return fail_hip(e, "spec plan");
    }
    lk.lock();
    while (c->rec_ingested < r) ingest_rec(c, c->rec_ingested);
    c->pf->retire();
    for (int slot = 0; slot < c->C; ++slot)
      if (c->pf->ready_seq(layer, slot, 2) != -1) busy |= 1ull << slot;
  }
  FfnArgs a = ffn_args(c, layer, d_x, T);
  a.npos = c->d_npos;
  a.busy_mask = busy;
  const size_t prof0 = c->prof_pending.size();
  // dense experts: one launch of the shared expert and the positions; 4-bit
  // experts: the dense shared expert, then the positions on the 4-bit GEMV
  for (int part = 0; part < 2; ++part) {
    const bool routed_q4 = part == 1;
    if (part == 1 && !c->q4) break;
    int n = 0;
    if (c->Ish > 0 && part == 0) {
      FfnJob& j = a.jobs[n++];
      j.w = a.shared_w;
      j.q0 = 0;
      j.q1 = T;
      j.I = c->Ish;
      j.r0 = 0;
      j.pos = kSharedJob;
      j.pad = 0;
    }
    if (c->q4 == routed_q4) {
      const int P = std::min(c->E, T * c->K);
      for (int p = 0; p < P; ++p) {
        FfnJob& j = a.jobs[n++];
        j.w = nullptr;
        j.q0 = j.q1 = 0;
        j.I = c->I;
        j.r0 = 0;
        j.pos = p;
        j.pad = 0;
      }
    }
    if (n == 0) continue;
    a.n_jobs = n;
    a.q4 = routed_q4 ? 1 : 0;
    for (int pass = 0; pass < 2; ++pass) {
      hipEvent_t e0 = nullptr, e1 = nullptr;
      if (c->profile) {
        e0 = prof_event(c);
        e1 = prof_event(c);
        c->prof_pending.push_back(ProfEntry{e0, e1, pass, 0.0, 0.0});
      }
      if (pass == 0 && c->ride_pred && launch_ffn_gateup_pred(a, c->ride, c->dt, s, e0, e1))
        c->ride_pred = false;
      else
        launch_ffn(a, pass, T, c->dt, s, e0, e1);
      LAUNCHCHK("early ffn");
    }
  }
  c->early_busy = busy;
  c->early_prof0 = prof0;
  c->early_nprof = c->prof_pending.size() - prof0;
  *launched = true;
  return PROMOE_OK;
}

// The plan is known: the positions the early launch computed (resident, slot not
// busy) are marked started, their slots' last reader becomes that launch (its
// compute token is recorded now: nothing was enqueued on s since), fills that
// wait for them are released, and the launch's profiling entries get their bytes.
static void early_resident_release(promoe_ctx* c, int layer, int T, hipStream_t s) {
  const PlanRecord& rec = c->route_rec;
  std::vector<int> jobs;
  for (int p = 0; p < rec.n_hit; ++p) {
    if ((c->early_busy >> rec.slot[p]) & 1ull) continue;
    c->ffn_started[p] = 1;
    jobs.push_back(p);
  }
  if (c->Ish > 0) {
    c->shared_started = true;
    jobs.push_back(kSharedJob);
  }
  release_after_launch(c, layer, jobs, s);
  if (c->profile && c->early_nprof) early_prof_bytes(c, rec, T, c->early_busy, c->early_prof0, c->early_nprof);
  c->early_nprof = 0;
}

// Steps larger than decode: a fill whose victim slot is read by a resident
// expert of the same step waits for that read.  The route launches the readers
// of the first fills' victims itself, right behind its plan, so the link
// starts on those fills while the caller runs the predictor and the FFN call
// computes the rest.  Caller holds c->mu; c->route_rec is this route's plan.
static int launch_route_head(promoe_ctx* c, int layer, const void* d_x, int T, hipStream_t s) {
  const bool in_order = (c->cfg.flags & (PROMOE_FLAG_NO_REORDER | PROMOE_FLAG_NO_PREEMPT)) != 0;
  if ((int64_t)T * c->K <= 64 || in_order) return PROMOE_OK;
  std::vector<char> arriving(c->route_rec.n);
  for (int p = 0; p < c->route_rec.n; ++p) arriving[p] = c->need01[p] != -1 || c->need2[p] != -1;
  const std::vector<int> head = head_readers(fill_waits(c), arriving, kHeadFills);
  if (head.empty()) return PROMOE_OK;
  const int rc = ffn_launch(c, ffn_args(c, layer, d_x, T), head, s, CopyWait(), CopyWait());
  if (rc) return rc;
  release_after_launch(c, layer, head, s);
  for (int p : head) c->ffn_started[p] = 1;
  return PROMOE_OK;
}

// Argument checks shared by promoe_expert_ffn and its allocation-free variant.
static int check_ffn_call(promoe_ctx* c, int layer, const void* d_x, int T, const int32_t* d_ids, const float* d_w,
                          const float* d_shared_scale, const void* d_y) {
  if (!c || layer < 0 || layer >= c->L || !d_x || !d_ids || !d_w || !d_y) return PROMOE_EINVAL;
  if (c->route_layer != layer || c->route_T != T) {
    g_last_error = "expert_ffn without a matching route";
    return PROMOE_ESTATE;
  }
  if (c->cfg.shared_gate && c->Ish > 0 && !d_shared_scale) return PROMOE_EINVAL;
  return PROMOE_OK;
}

// The FFN of the routed layer with the activations and expert outputs in the
// buffers `a` names (the context's, or the allocation-free scratch).
static int expert_ffn_run(promoe_ctx* c, int layer, int T, const float* d_w, const float* d_shared_scale,
                          void* d_y, hipStream_t s, const FfnArgs& a) {
  c->last_stream = s;
  const PlanRecord& rec = c->route_rec;

  std::unique_lock<std::mutex> lk(c->mu);
  const bool lazy = c->route_lazy;
  c->route_lazy = false;
  const int n = lazy ? 0 : rec.n;
  // On another stream than the route's, order this call after everything the
  // route enqueued: its top-k and plan (ids, weights, slots, permutation) and
  // the readers of the first fills' victim slots it may have started.
  if (c->route_stream != s) HIPCHK(hipStreamWaitEvent(s, c->route_done, 0));
  // Outputs the route's own launches wrote into the context's buffers, when this
  // call keeps its expert outputs elsewhere (the allocation-free variant): every
  // pair's row is carried over, and the launches below overwrite the rest.
  const bool any_started = lazy || c->shared_started ||
                           std::find(c->ffn_started.begin(), c->ffn_started.end(), 1) != c->ffn_started.end();
  if (any_started && a.Y != c->d_Y) {
    HIPCHK(hipMemcpyAsync(a.Y, c->d_Y, sizeof(float) * (size_t)T * c->K * c->H, hipMemcpyDeviceToDevice, s));
    if (c->shared_started)
      HIPCHK(hipMemcpyAsync(a.Ysh, c->d_Ysh, sizeof(float) * a.ksplit * (size_t)a.ysh_split_stride,
                            hipMemcpyDeviceToDevice, s));
  }
  std::vector<char> done(c->ffn_started), is_def(n, 0);
  for (const auto& d : c->deferred) is_def[d.pos] = 1;

  auto after_launch = [&](const std::vector<int>& jobs) {
    release_after_launch(c, layer, jobs, s);
    for (int p : jobs)
      if (p != kSharedJob) done[p] = 1;
    for (int p = 0; p < n; ++p) is_def[p] = 0;
    for (const auto& d : c->deferred) is_def[d.pos] = 1;
  };

  // Reordered inference runs every ready expert first; without it (or without
  // early preemption, where a later position's copy starts only when it is
  // reached) positions run strictly in the route order.
  const bool in_order = (c->cfg.flags & (PROMOE_FLAG_NO_REORDER | PROMOE_FLAG_NO_PREEMPT)) != 0;
  // 1. the shared expert and every routed expert whose chunks are already in HBM.
  // Decode-sized steps run them in one launch.  Larger steps run the resident
  // experts that fills wait for kResidentGroup at a time in the route order,
  // so those fills (victims in the same order) are released group by group
  // instead of behind all of them; then the other resident experts in one
  // launch, and the shared expert last.
  std::vector<int> ready;
  for (int p = 0; p < n; ++p) {
    if (done[p]) continue;
    if (!is_def[p] && c->need01[p] < 0 && c->need2[p] < 0) ready.push_back(p);
    else if (in_order) break;
  }
  int rc = PROMOE_OK;
  const bool batch = (int64_t)T * c->K <= 64;
  std::vector<int> jobs;
  if (batch) {
    if (c->Ish > 0 && !c->shared_started) jobs.push_back(kSharedJob);
    jobs.insert(jobs.end(), ready.begin(), ready.end());
    if (!jobs.empty()) {
      rc = ffn_launch(c, a, jobs, s, CopyWait(), CopyWait());
      if (rc) return rc;
      after_launch(jobs);
    }
  } else {
    // groups only up to the last resident expert that a fill waits for; the
    // rest release nothing and run in one launch (fewer, fuller GEMMs)
    for (const auto& g : resident_groups(ready, fill_waits(c), kResidentGroup)) {
      rc = ffn_launch(c, a, g, s, CopyWait(), CopyWait());
      if (rc) return rc;
      after_launch(g);
    }
    if (c->Ish > 0) {
      jobs.assign(1, kSharedJob);
      rc = ffn_launch(c, a, jobs, s, CopyWait(), CopyWait());
      if (rc) return rc;
      after_launch(jobs);
    }
  }
  // 2. experts still arriving.  Decode-sized steps batch them into one launch
  // behind the last copy (a GEMV is ~1% of a copy, so per-expert launches buy no
  // overlap); larger steps launch in the route order, kArrivalGroup experts at
  // a time, so compute follows the copies: consecutive fills run on different
  // copy queues and arrive together, and a launch of one expert's few tokens
  // leaves most CUs idle, so two experts cost about what one does.  Fills
  // deferred behind an earlier expert's read are released as it is launched,
  // so an expert that such a fill waits for is launched as soon as it has
  // arrived, without waiting for a second one (with few slots per layer every
  // fill waits for the previous occupant of its slot).
  auto releases_fill = [&](int p) {
    for (const auto& d : c->deferred)
      if (d.after == p) return true;
    return false;
  };
  for (;;) {
    jobs.clear();
    CopyWait w01, w2;
    for (int p = 0; p < n; ++p) {
      if (done[p]) continue;
      if (is_def[p]) {
        if (in_order) break;
        continue;
      }
      jobs.push_back(p);
      w01.add(c->need_q[p], c->need01[p]);
      w2.add(c->need_q[p], c->need2[p]);
      if (!batch && ((int)jobs.size() == kArrivalGroup || releases_fill(p))) break;
    }
    if (jobs.empty()) break;
    rc = ffn_launch(c, a, jobs, s, w01, w2);
    if (rc) return rc;
    after_launch(jobs);
  }
  for (int p = 0; p < n; ++p)
    if (!done[p]) {
      g_last_error = "expert_ffn: unreleased position";
      return PROMOE_ESTATE;
    }
  if (c->eng.err != hipSuccess) return fail_hip(c->eng.err, "copy engine");
  lk.unlock();
  c->cv.notify_all();

  CombineArgs ca{};
  ca.Y = a.Y;
  ca.w = d_w;
  ca.Ysh = c->Ish > 0 ? a.Ysh : nullptr;
  ca.ysh_split = a.ksplit;
  ca.ysh_split_stride = a.ysh_split_stride;
  ca.sscale = (c->Ish > 0 && c->cfg.shared_gate) ? d_shared_scale : nullptr;
  ca.y = d_y;
  ca.hidden = c->H;
  ca.top_k = c->K;
  if (c->fuse_h && c->defer_combine) {
    // the layer loop folds this combine into the next layer's first kernel
    c->pending = ca;
    c->pending_h = c->fuse_h;
    c->has_pending = true;
  } else if (c->fuse_h) {
    launch_combine_residual(ca, c->fuse_h, T, c->dt, s);
  } else {
    launch_combine(ca, T, c->dt, s);
  }
  LAUNCHCHK("combine");
  // a prediction the route launched on the side stream: later work on s follows it
  HIPCHK(pred_join(c, s));
  c->route_layer = -1;
  if (c->profile && !c->noalloc_call && c->prof_pending.size() > 4096) {
    HIPCHK(hipStreamSynchronize(s));
    HIPCHK(drain_records(c, true));  // lazy routes' plans give their launches' bytes
    prof_resolve(c);
  }
  return PROMOE_OK;
}

int promoe_expert_ffn(promoe_ctx* c, int layer, const void* d_x, int T, const int32_t* d_ids, const float* d_w,
                      const float* d_shared_scale, void* d_y, void* stream) {
  const int rc = check_ffn_call(c, layer, d_x, T, d_ids, d_w, d_shared_scale, d_y);
  if (rc) return rc;
  return expert_ffn_run(c, layer, T, d_w, d_shared_scale, d_y, static_cast<hipStream_t>(stream),
                        ffn_args(c, layer, d_x, T));
}

int promoe_expert_ffn_noalloc(promoe_ctx* c, int layer, const void* d_x, int T, const int32_t* d_ids,
                              const float* d_w, const float* d_shared_scale, void* d_y, void* stream) {
  int rc = check_ffn_call(c, layer, d_x, T, d_ids, d_w, d_shared_scale, d_y);
  if (rc) return rc;
  if ((int64_t)T * c->K > 64) {
    g_last_error = "expert_ffn_noalloc: more than 64 routed pairs (T * top_k) in the step";
    return PROMOE_EINVAL;
  }
  // Scratch layout: activations [T*k x I], expert outputs [T*k x H] fp32,
  // shared activations [T x I_sh], shared partial outputs [ksplit x T x H] fp32,
  // each piece 256-byte aligned.  Every byte the kernels read is written
  // earlier in the same call, so nothing needs clearing.
  FfnArgs a = ffn_args(c, layer, d_x, T);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off += (bytes + 255) & ~(size_t)255; return o; };
  const size_t pairs = (size_t)T * c->K;
  const size_t o_act = take(pairs * c->I * c->eb), o_Y = take(pairs * c->H * sizeof(float)),
               o_actsh = take((size_t)T * std::max(c->Ish, 1) * c->eb),
               o_Ysh = take((size_t)a.ksplit * T * c->H * sizeof(float));
  if (off > kNoAllocScratchBytes) {
    g_last_error = "expert_ffn_noalloc: the step needs " + std::to_string(off) + " bytes of scratch, more than the " +
                   std::to_string(kNoAllocScratchBytes) + " of the allocation-free call";
    return PROMOE_EINVAL;
  }
  uint8_t* base = c->noalloc_scratch;
  a.act = base + o_act;
  a.Y = reinterpret_cast<float*>(base + o_Y);
  a.act_sh = base + o_actsh;
  a.Ysh = reinterpret_cast<float*>(base + o_Ysh);
  c->noalloc_call = true;
  rc = expert_ffn_run(c, layer, T, d_w, d_shared_scale, d_y, static_cast<hipStream_t>(stream), a);
  c->noalloc_call = false;
  return rc;
}

int promoe_cache_stats(promoe_ctx* c, int layer, promoe_stats* out) {
  if (!c || !out || layer < -1 || layer >= c->L) return PROMOE_EINVAL;
  int rc = promoe_sync(c);
  if (rc) return rc;
  std::vector<int64_t> cnt((size_t)c->L * kCounters);
  HIPCHK(hipMemcpy(cnt.data(), c->st.counters, sizeof(int64_t) * cnt.size(), hipMemcpyDeviceToHost));
  std::memset(out, 0, sizeof(*out));
  int64_t* dst = &out->prec_access;
  for (int l = 0; l < c->L; ++l) {
    if (layer >= 0 && l != layer) continue;
    for (int i = 0; i < kCounters; ++i) dst[i] += cnt[(size_t)l * kCounters + i];
  }
  std::lock_guard<std::mutex> lk(c->mu);
  const PhysStats& ps = c->pf->stats();
  out->copies_low = ps.copies[0];
  out->copies_high = ps.copies[1];
  out->bytes_low = ps.bytes[0];
  out->bytes_high = ps.bytes[1];
  out->low_purged = ps.low_purged;
  out->deferred = ps.deferred;
  out->pred_in_time = c->pred_in_time;
  out->lazy_routes = c->n_lazy_routes;
  for (int i = 0; i < promoe_ctx::kClasses; ++i) {
    out->k_launches[i] = c->k_launches[i];
    out->k_ms[i] = c->k_ms[i];
    out->k_bytes[i] = c->k_bytes[i];
    out->k_flops[i] = c->k_flops[i];
  }
  out->stall_ms = c->stall_ms;
  return PROMOE_OK;
}

int promoe_reset_stats(promoe_ctx* c) {
  if (!c) return PROMOE_EINVAL;
  int rc = promoe_sync(c);
  if (rc) return rc;
  if (c->profile) prof_resolve(c);
  HIPCHK(hipMemset(c->st.counters, 0, sizeof(int64_t) * kCounters * c->L));
  HIPCHK(hipDeviceSynchronize());
  std::lock_guard<std::mutex> lk(c->mu);
  c->pf->reset_stats();
  c->pred_in_time = 0;
  c->n_lazy_routes = 0;
  for (int i = 0; i < promoe_ctx::kClasses; ++i) c->k_launches[i] = 0, c->k_ms[i] = c->k_bytes[i] = c->k_flops[i] = 0.0;
  c->stall_ms = 0.0;
  return PROMOE_OK;
}

int promoe_slot_table(promoe_ctx* c, int layer, int32_t* h_slot_of) {
  if (!c || !h_slot_of || layer < 0 || layer >= c->L) return PROMOE_EINVAL;
  int rc = promoe_sync(c);
  if (rc) return rc;
  HIPCHK(hipMemcpy(h_slot_of, c->st.slot_of + (size_t)layer * c->E, sizeof(int32_t) * c->E, hipMemcpyDeviceToHost));
  return PROMOE_OK;
}

int promoe_last_plan(promoe_ctx* c, int layer, int kind, promoe_plan* out) {
  if (!c || !out || layer < 0 || layer >= c->L || (kind != 0 && kind != 1)) return PROMOE_EINVAL;
  int rc = promoe_sync(c);
  if (rc) return rc;
  std::lock_guard<std::mutex> lk(c->mu);
  const PlanRecord& r = kind == 0 ? c->last_spec[layer] : c->last_precise[layer];
  out->n = r.n;
  out->fill_budget = r.fill_budget;
  for (int i = 0; i < 64; ++i) {
    out->expert[i] = r.expert[i];
    out->slot[i] = r.slot[i];
    out->flag[i] = r.flag[i];
    out->victim[i] = r.victim[i];
    out->after[i] = r.after[i];
    out->count[i] = r.count[i];
  }
  return PROMOE_OK;
}

int promoe_stack_step(promoe_ctx* c, float* d_h, int T, void* d_x, void* d_y, int32_t* d_ids, float* d_w,
                      float* d_shared_scale, int32_t* d_pred_ids, int predict, void* stream) {
  if (!c || !d_h || !d_x || !d_y || !d_ids || !d_w) return PROMOE_EINVAL;
  int rc = check_tokens(c, T);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // Batch 1: the two RMSNorms of a layer run inside the attention surrogate's
  // GEMV and the gate GEMV (bit for bit the separate kernels), the attention
  // GEMV writing the updated residual into the other of two buffers.
  const bool fold = T == 1 && c->dt == PROMOE_BF16 && !(predict && c->D == 0);
  float* hb[2] = {d_h, c->d_h2};
  int cur = 0;
  // a pending combine, launched on its own (adding into its residual buffer)
  auto flush_combine = [&]() {
    if (!c->has_pending) return;
    launch_combine_residual(c->pending, c->pending_h, T, c->dt, s);
    c->has_pending = false;
  };
  c->has_pending = false;
  for (int l = 0; l < c->L; ++l) {
    if (fold) {
      c->last_stream = s;
      bool x_ready = false;
      if (c->lw[l].attn) {
        RowsArgs a{};
        a.w[0] = c->lw[l].attn;
        a.nrows[0] = c->H;
        a.K = c->H;
        a.T = T;
        a.out = hb[cur ^ 1];
        a.ldo = c->H;
        // the previous layer's combine folded in when it is pending on hb[cur]
        const bool cmb = c->has_pending && c->pending_h == hb[cur];
        if (!cmb) flush_combine();
        if (launch_rows_gemv_norm(a, hb[cur], hb[cur], nullptr, s, cmb ? &c->pending : nullptr)) {
          LAUNCHCHK("attn surrogate");
          cur ^= 1;
          c->has_pending = false;
        } else {
          flush_combine();
          if ((rc = promoe_attn_surrogate(c, l, hb[cur], T, d_x, stream))) return rc;
          x_ready = true;
        }
      }
      flush_combine();
      if (!x_ready) c->x_from_h = hb[cur];
    } else if ((rc = promoe_attn_surrogate(c, l, d_h, T, d_x, stream))) {
      return rc;
    }
    if (predict && c->D == 0) {
      if ((rc = promoe_predict(c, l, d_x, T, d_pred_ids, nullptr, nullptr, stream))) return rc;
      rc = route_impl(c, l, d_x, T, d_ids, d_w, d_shared_scale, nullptr, nullptr, s, false, nullptr);
    } else {
      rc = route_impl(c, l, d_x, T, d_ids, d_w, d_shared_scale, nullptr, nullptr, s, predict != 0, d_pred_ids);
    }
    c->x_from_h = nullptr;
    if (rc) return rc;
    // the combine also does the residual add; with a next layer whose
    // attention GEMV can fold it in, it is left pending for that launch
    c->fuse_h = hb[cur];
    c->defer_combine = fold && l + 1 < c->L && c->lw[l + 1].attn != nullptr;
    rc = promoe_expert_ffn(c, l, d_x, T, d_ids, d_w, d_shared_scale, d_y, stream);
    c->fuse_h = nullptr;
    c->defer_combine = false;
    if (rc) {
      c->has_pending = false;
      return rc;
    }
  }
  flush_combine();
  if (cur) HIPCHK(hipMemcpyAsync(d_h, c->d_h2, sizeof(float) * (size_t)T * c->H, hipMemcpyDeviceToDevice, s));
  return PROMOE_OK;
}

int promoe_attn_surrogate(promoe_ctx* c, int layer, float* d_h, int T, void* d_x_out, void* stream) {
  if (!c || layer < 0 || layer >= c->L || !d_h || !d_x_out) return PROMOE_EINVAL;
  int rc = check_tokens(c, T);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  c->last_stream = s;
  if (c->lw[layer].attn) {
    launch_rmsnorm_quant(d_h, c->d_u, T, c->H, c->dt, s);
    RowsArgs a{};
    a.w[0] = c->lw[layer].attn;
    a.nrows[0] = c->H;
    a.K = c->H;
    a.x = c->d_u;
    a.ldx = c->H;
    a.T = T;
    a.out = d_h;
    a.ldo = c->H;
    a.add = 1;
    if (c->dt == PROMOE_BF16 && T >= 64 && c->H % 64 == 0) {
      RowsGemmArgs g{};
      g.w = c->lw[layer].attn;
      g.N = c->H;
      g.K = c->H;
      g.x = c->d_u;
      g.ldx = c->H;
      g.T = T;
      g.out = d_h;
      g.ldo = c->H;
      g.add = 1;
      launch_gemm_rows(g, s);
    } else {
      launch_rows_gemv(a, c->dt, c->dt, s);
    }
  }
  launch_rmsnorm_quant(d_h, d_x_out, T, c->H, c->dt, s);
  LAUNCHCHK("attn surrogate");
  return PROMOE_OK;
}

int promoe_residual_add(promoe_ctx* c, float* d_h, const void* d_y, int T, void* stream) {
  if (!c || !d_h || !d_y) return PROMOE_EINVAL;
  int rc = check_tokens(c, T);
  if (rc) return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  c->last_stream = s;
  launch_residual_add(d_h, d_y, T * c->H, c->dt, s);
  LAUNCHCHK("residual");
  return PROMOE_OK;
}

}  // extern "C"
