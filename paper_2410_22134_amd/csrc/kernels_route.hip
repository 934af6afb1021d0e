// Routing and cache-plan kernels for gfx950 (wave64).
//
//  * k_topk          -- per token one wave, one lane per expert (E <= 64):
//                       softmax and top-k by (logit desc, id asc) from k rounds
//                       of a DPP wave max over order-preserving logit bits and a
//                       ballot of the lanes holding it (lowest id first),
//                       renormalised weights, the shared expert's sigmoid gate.
//                       Used by the router and, ids only, by the predictor.
//  * k_plan_spec     -- speculative plan of a target layer (Alg. 2
//                       PushPredictedExperts): integer vote over the tokens'
//                       predicted ids, then the LRU plan: the list's resident
//                       experts touched, then its others filled (optionally
//                       only the first few), never evicting a predicted expert.
//  * k_plan_precise  -- precise plan of the routed layer (Alg. 2
//                       PushPreciseExperts, Sec. "Reordered Inference"):
//                       hit/miss, order, victim slots, counters, followed by the
//                       token permutation grouping (t, r) pairs by position;
//                       k_route_plan runs the top-k first in the same block.
//
// Both plans run in one workgroup: the counting phases use all 256 threads,
// the sequential LRU walk runs in wave 0 with one lane per slot (for slot
// state) and one lane per expert (for slot_of), so every victim search is one
// wave-wide argmin and every lookup one scalar lane read.  The plans write a
// record into host-mapped memory for the copy scheduler.  k_predict_plan and
// k_route_plan_predict spread the predictor's second layer over several
// blocks, the last of which to finish runs the top-k and the spec plan.
#include "common.hpp"
#include "kernels.hpp"

namespace promoe {

enum {
  CNT_PREC = 0, CNT_HIT, CNT_MISS, CNT_SPEC_ISSUED, CNT_SPEC_RESIDENT, CNT_SPEC_USED, CNT_SPEC_WASTED, CNT_EVICT,
  CNT_PRED_N, CNT_PRED_CORRECT
};

// ============================================================ top-k
// Token t by one wave (lane = expert); ids_copy (LDS, may be null) also gets the ids.
__device__ __forceinline__ void topk_token(const TopkArgs& a, int t, int lane, int32_t* ids_copy) {
  const bool valid = lane < a.E;
  float z = -INFINITY;
  if (valid) z = a.logits[(size_t)t * a.ld + lane] + (a.bias ? a.bias[lane] : 0.0f);
  const uint32_t key = f32_order_key(z);
  bool cand = valid;
  int myrank = -1;
  for (int r = 0; r < a.k; ++r) {
    const int e = wave_pick_max(key, cand);
    if (lane == e) myrank = r;
    if (lane == 0) {
      a.ids[t * a.k + r] = e;
      if (ids_copy) ids_copy[t * a.k + r] = e;
    }
  }
  if (a.want_weights) {
    const float zmax = wave_max(valid ? z : -INFINITY);
    const float ez = valid ? expf(z - zmax) : 0.0f;
    const float denom = a.renorm ? wave_sum(myrank >= 0 ? ez : 0.0f) : wave_sum(ez);
    if (myrank >= 0) a.w[t * a.k + myrank] = ez / denom;
    if (a.sgate_col >= 0 && lane == 0) {
      const float u = a.logits[(size_t)t * a.ld + a.sgate_col];
      a.sscale[t] = 1.0f / (1.0f + expf(-u));
    }
  }
}

__global__ __launch_bounds__(256) void k_topk(TopkArgs a) {
  const int t = blockIdx.x * 4 + threadIdx.x / kWave;
  if (t >= a.T) return;
  topk_token(a, t, threadIdx.x % kWave, nullptr);
}

// ============================================================ plan helpers
struct WaveState {
  int slot_expert;  // lane = slot
  uint32_t stamp, fetch;
  int spec_unused;
  int slot_of;      // lane = expert
};

__device__ __forceinline__ void load_state(const PlanArgs& a, int lane, WaveState& w, uint32_t& clock, uint32_t& fseq,
                                           int64_t (&cnt)[kCounters]) {
  const int bc = a.layer * a.C, be = a.layer * a.E;
  w.slot_expert = lane < a.C ? a.st.slot_expert[bc + lane] : -1;
  w.stamp = lane < a.C ? a.st.stamp[bc + lane] : 0u;
  w.fetch = lane < a.C ? a.st.fetch_seq[bc + lane] : 0u;
  w.spec_unused = lane < a.C ? a.st.spec_unused[bc + lane] : 0;
  w.slot_of = lane < a.E ? a.st.slot_of[be + lane] : -1;
  clock = a.st.clock[a.layer];
  fseq = a.st.fseq[a.layer];
#pragma unroll
  for (int i = 0; i < kCounters; ++i) cnt[i] = a.st.counters[a.layer * kCounters + i];
}

__device__ __forceinline__ void store_state(const PlanArgs& a, int lane, const WaveState& w, uint32_t clock,
                                            uint32_t fseq, const int64_t (&cnt)[kCounters]) {
  const int bc = a.layer * a.C, be = a.layer * a.E;
  if (lane < a.C) {
    a.st.slot_expert[bc + lane] = w.slot_expert;
    a.st.stamp[bc + lane] = w.stamp;
    a.st.fetch_seq[bc + lane] = w.fetch;
    a.st.spec_unused[bc + lane] = w.spec_unused;
  }
  if (lane < a.E) a.st.slot_of[be + lane] = w.slot_of;
  if (lane == 0) {
    a.st.clock[a.layer] = clock;
    a.st.fseq[a.layer] = fseq;
#pragma unroll
    for (int i = 0; i < kCounters; ++i) a.st.counters[a.layer * kCounters + i] = cnt[i];
  }
}

// A layer's cache state as wave 0 of a plan holds it, loaded at the start of
// a kernel so that its loads overlap the work before the plan (the top-k, the
// predictor's second layer) instead of following it.
struct PlanState {
  WaveState w;
  uint32_t clock, fseq;
  int64_t cnt[kCounters];
  uint64_t pred_mask;
};

__device__ __forceinline__ void load_plan_state(const PlanArgs& a, int lane, PlanState& ps) {
  load_state(a, lane, ps.w, ps.clock, ps.fseq, ps.cnt);
  ps.pred_mask = a.st.pred_mask[a.layer];
}

// Lowest-index free slot, else the least recently stamped one (stamps are
// unique), among the slots that are not pinned.
__device__ __forceinline__ int victim_slot(const PlanArgs& a, int lane, const WaveState& w) {
  uint64_t key = ~0ull;
  if (lane < a.C && lane >= a.pinned) key = w.slot_expert < 0 ? (uint64_t)lane : ((1ull << 40) | (uint64_t)w.stamp);
  key = (key << 6) | (uint64_t)lane;
  return (int)(wave_min_u64(key) & 63ull);
}

// victim_slot among the slots whose expert is not in `spare` (a bit per
// expert); -1 when every candidate slot holds such an expert.
__device__ __forceinline__ int spare_victim_slot(const PlanArgs& a, int lane, const WaveState& w, uint64_t spare) {
  uint64_t key = ~0ull;
  if (lane < a.C && lane >= a.pinned) {
    if (w.slot_expert < 0) key = (uint64_t)lane;
    else if (!((spare >> w.slot_expert) & 1ull)) key = (1ull << 40) | (uint64_t)w.stamp;
  }
  key = (key << 6) | (uint64_t)lane;
  const uint64_t m = wave_min_u64(key);
  return m >= (1ull << 47) ? -1 : (int)(m & 63ull);
}

// Give slot v to expert e: evict its occupant (counted), fill, stamp.
__device__ __forceinline__ int fill_slot(const PlanArgs& a, int lane, WaveState& w, int e, int v, bool speculative,
                                         uint32_t& clock, uint32_t& fseq, int64_t (&cnt)[kCounters]) {
  const int old = lane_value(w.slot_expert, v);
  const int old_unused = lane_value(w.spec_unused, v);
  if (old >= 0) {
    cnt[CNT_EVICT]++;
    if (old_unused) cnt[CNT_SPEC_WASTED]++;
    if (lane == old) w.slot_of = -1;
  }
  ++fseq;
  ++clock;
  if (lane == v) {
    w.slot_expert = e;
    w.fetch = fseq;
    w.stamp = clock;
    w.spec_unused = speculative ? 1 : 0;
  }
  if (lane == e) w.slot_of = v;
  return old;
}

// ============================================================ spec plan
struct SpecLds {
  int votes[kMaxE], best[kMaxE], Q[kMaxE];
  int nq;
};

// The spec plan over the predicted ids `ids` [T x k] (global or LDS; a.ids
// non-null marks the plan as a prediction), or over the caller's list in the
// record when a.ids is null.  All 256 threads of the block enter.
__device__ __forceinline__ void plan_spec_body(const PlanArgs& a, const int32_t* ids, SpecLds& sh,
                                               const PlanState* pre = nullptr) {
  int* votes = sh.votes;
  int* best = sh.best;
  int* Q = sh.Q;
  int& nq = sh.nq;
  const int tid = threadIdx.x, lane = tid % kWave;
  if (tid < kMaxE) { votes[tid] = 0; best[tid] = kMaxK; }
  __syncthreads();
  uint64_t voted = 0, listed = 0;  // wave 0: experts voted for; the list's members (prediction)
  if (a.ids) {
    const int n = a.T * a.k;
    for (int i = tid; i < n; i += 256) {
      const int e = ids[i];
      atomicAdd(&votes[e], 1);
      atomicMin(&best[e], i % a.k);
    }
  }
  __syncthreads();
  if (a.ids) {
    // rank of each voted expert by (votes desc, best rank asc, id asc): one
    // wave, lane = expert, counting the larger keys (key order = that order)
    if (tid < kWave) {
      const int ve = lane < a.E ? votes[lane] : 0, be = lane < a.E ? best[lane] : kMaxK;
      const uint32_t key = ve > 0 ? ((uint32_t)ve << 12) | ((uint32_t)(15 - be) << 6) | (uint32_t)(63 - lane) : 0u;
      // only voted lanes can hold a larger key (the others' key is 0)
      voted = __ballot(ve > 0);
      int rank = 0;
      for (uint64_t m = voted; m; m &= m - 1) rank += lane_value(key, __builtin_ctzll(m)) > key ? 1 : 0;
      if (ve > 0 && rank < a.C) Q[rank] = lane;
      listed = __ballot(ve > 0 && rank < a.C);  // the first min(voted, C): Q
      if (lane == 0) nq = min(__popcll(voted), a.C);
    }
  } else if (tid == 0) {
    nq = a.rec->n_q_in;
    for (int i = 0; i < nq; ++i) Q[i] = a.rec->q_in[i];
  }
  __syncthreads();
  if (tid >= kWave) return;

  WaveState w;
  uint32_t clock, fseq;
  int64_t cnt[kCounters];
  if (pre) {
    w = pre->w;
    clock = pre->clock;
    fseq = pre->fseq;
#pragma unroll
    for (int i = 0; i < kCounters; ++i) cnt[i] = pre->cnt[i];
  } else {
    load_state(a, lane, w, clock, fseq, cnt);
  }
  PlanRecord* rec = a.rec;
  // Host-given lists are never limited; a predicted plan fills at most fill_budget slots.
  const int budget = a.ids ? a.fill_budget : -1;
  if (a.ids) {  // a prediction: remembered until the layer's route scores it
    if (lane == 0) a.st.pred_mask[a.layer] = listed;
    cnt[CNT_PRED_N] += nq;
  }
  // Experts no fill may evict: every expert the prediction votes for (of which
  // Q is the first C), or the caller's whole list.
  uint64_t spare = voted;
  if (!a.ids) {
    for (int i = 0; i < nq; ++i) spare |= 1ull << Q[i];
  }
  // The list's hits first (Alg. 2 counts them as it pushes the list), then its
  // fills (the worker of Alg. 1 replaces a slot only when a copy starts): no
  // fill evicts a member of the list.
  // lane i keeps list member i's record entries, stored at the end one
  // coalesced store per field (the record lives in host memory)
  int my_e = 0, my_s = -1, my_f = 0, my_v = -1;
  const int q_lane = lane < nq ? Q[lane] : 0;  // list member i in lane i
  for (int i = 0; i < nq; ++i) {
    const int e = lane_value(q_lane, i);
    const int s_res = lane_value(w.slot_of, e);
    if (s_res >= 0) {
      ++clock;
      if (lane == s_res) w.stamp = clock;
      cnt[CNT_SPEC_RESIDENT]++;
      if (lane == i) { my_e = e; my_s = s_res; my_f = 0; my_v = -1; }
    }
  }
  int fills = 0;
  for (int i = 0; i < nq; ++i) {
    const int e = lane_value(q_lane, i);
    if (lane_value(w.slot_of, e) >= 0) continue;
    const int v = (budget >= 0 && fills >= budget) ? -1 : spare_victim_slot(a, lane, w, spare);
    if (v < 0) {
      if (lane == i) { my_e = e; my_s = -1; my_f = 0; my_v = -1; }
      continue;
    }
    ++fills;
    const int old = fill_slot(a, lane, w, e, v, true, clock, fseq, cnt);
    cnt[CNT_SPEC_ISSUED]++;
    if (lane == i) { my_e = e; my_s = v; my_f = 1; my_v = old; }
  }
  store_state(a, lane, w, clock, fseq, cnt);
  if (lane < nq) {
    rec->expert[lane] = my_e;
    rec->slot[lane] = my_s;
    rec->flag[lane] = my_f;
    rec->victim[lane] = my_v;
    rec->after[lane] = -1;
  }
  if (lane == 0) {
    rec->kind = 0;
    rec->layer = a.layer;
    rec->n = nq;
    rec->n_hit = 0;
    rec->predicted = a.ids ? 1 : 0;
    rec->fill_budget = budget;
    if (a.host_done) {
      __threadfence_system();
      rec->done = 1;
    }
  }
}

__global__ __launch_bounds__(256) void k_plan_spec(PlanArgs a) {
  __shared__ SpecLds sh;
  plan_spec_body(a, a.ids, sh);
}

// ============================================================ predictor tail + spec plan
// For a step of at most kFusedPredMaxT tokens: the predictor's second layer
// q[t][e] = W2[e] . relu(h[t]) (fp32 accumulation; or q = h when the
// predictor is one layer), each token's top-k by (q desc, id asc) as k_topk
// orders them, written out and kept in LDS, then the spec plan of the vote.
//
// The rows of W2 are spread over pred_blocks(E, Ph) blocks of
// kPredExpertsPerBlock experts each, so that their loads run on that many CUs
// (one CU alone streams the ~128 KB of a 64 x 1024 bf16 W2 at a few tens of
// GB/s).  Each block writes its logits to the target layer's exchange buffer
// and counts itself in with a device-scope atomic after a release fence; the
// block that counts last acquires, reads every logit back, resets the count
// and runs the top-k and the plan.  No block waits on another.
constexpr int kPredThreadsPerExpert = 256 / kPredExpertsPerBlock;  // 32: lanes of one wave

struct PredictLds {
  float hs[kFusedPredMaxT * kFusedPredMaxHidden];
  float qs[kFusedPredMaxT * kMaxE];
  int32_t ids_l[kFusedPredMaxT * kMaxK];
  SpecLds sh;
  int last;
};

// blk: this block's index among the prediction's pred_blocks(E, Ph) blocks.
__device__ __forceinline__ void predict_plan_body(const PredictPlanArgs& p, PredictLds& L, int blk) {
  float* hs = L.hs;
  float* qs = L.qs;
  int32_t* ids_l = L.ids_l;
  const PlanArgs& a = p.plan;
  const int tid = threadIdx.x, lane = tid % kWave, wv = tid / kWave;
  PlanState ps;  // used by the block that runs the plan; loaded early by every block
  if (tid < kWave) load_plan_state(a, lane, ps);
  const int T = a.T, E = a.E, k = a.k, Ph = p.Ph;
  const int nblk = pred_blocks(E, Ph);
  if (Ph > 0) {
    // kPredThreadsPerExpert threads per expert: thread q of expert e takes
    // the 16-byte chunks q, q + 32, ... of its row; with bf16 weights every
    // chunk is loaded before the hidden activations are staged
    const int n8 = Ph / 8;  // Ph % 8 == 0
    const int el = tid / kPredThreadsPerExpert, q = tid % kPredThreadsPerExpert;
    const int e = blk * kPredExpertsPerBlock + el;
    constexpr int kChunks = kFusedPredMaxHidden / 8 / kPredThreadsPerExpert;
    uint4 wq[kChunks];
    if (p.w2_bf16) {
      const uint4* row = reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(p.w2) + (size_t)(e < E ? e : 0) * Ph);
#pragma unroll
      for (int u = 0; u < kChunks; ++u) {
        const int j8 = q + kPredThreadsPerExpert * u;
        wq[u] = (e < E && j8 < n8) ? row[j8] : make_uint4(0, 0, 0, 0);
      }
    }
    {
      // every load of the hidden activations is issued before the first LDS store
      constexpr int kPer = kFusedPredMaxT * kFusedPredMaxHidden / 256;
      const int n = T * Ph;
      float hv[kPer];
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        hv[u] = 0.0f;
        if (i < n) {
          const int t = i / Ph, j = i - t * Ph;
          hv[u] = p.h[(size_t)t * p.ldh + j];
        }
      }
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int i = tid + 256 * u;
        if (i < n) hs[i] = fmaxf(hv[u], 0.0f);
      }
    }
    __syncthreads();
    float acc[kFusedPredMaxT];
#pragma unroll
    for (int t = 0; t < kFusedPredMaxT; ++t) acc[t] = 0.0f;
    if (e < E) {
      if (p.w2_bf16) {
#pragma unroll
        for (int u = 0; u < kChunks; ++u) {
          const int j8 = q + kPredThreadsPerExpert * u;
          if (j8 >= n8) break;
          const uint32_t q4[4] = {wq[u].x, wq[u].y, wq[u].z, wq[u].w};
          float wj[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            wj[2 * i] = __uint_as_float(q4[i] << 16);
            wj[2 * i + 1] = __uint_as_float(q4[i] & 0xFFFF0000u);
          }
#pragma unroll
          for (int t = 0; t < kFusedPredMaxT; ++t) {
            if (t < T) {
              const float* h = hs + t * Ph + j8 * 8;
#pragma unroll
              for (int i = 0; i < 8; ++i) acc[t] = fmaf(wj[i], h[i], acc[t]);
            }
          }
        }
      } else {
        for (int j8 = q; j8 < n8; j8 += kPredThreadsPerExpert) {
          const float* w = static_cast<const float*>(p.w2) + (size_t)e * Ph + j8 * 8;
          float wj[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) wj[i] = w[i];
#pragma unroll
          for (int t = 0; t < kFusedPredMaxT; ++t) {
            if (t < T) {
              const float* h = hs + t * Ph + j8 * 8;
#pragma unroll
              for (int i = 0; i < 8; ++i) acc[t] = fmaf(wj[i], h[i], acc[t]);
            }
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < kFusedPredMaxT; ++t) {
      if (t < T) {
        float v = acc[t];
#pragma unroll
        for (int o = 1; o < kPredThreadsPerExpert; o <<= 1) v += __shfl_xor(v, o, kWave);
        if (q == 0 && e < E) qs[t * kMaxE + e] = v;
      }
    }
    __syncthreads();
    if (nblk > 1) {
      float* xq = a.st.pred_xq + (size_t)a.layer * kFusedPredMaxT * kMaxE;
      uint32_t* xcnt = a.st.pred_xcnt + a.layer;
      if (tid < kWave) {
        for (int i = lane; i < T * kPredExpertsPerBlock; i += kWave) {
          const int t = i / kPredExpertsPerBlock, ee = blk * kPredExpertsPerBlock + i % kPredExpertsPerBlock;
          if (ee < E) xq[t * kMaxE + ee] = qs[t * kMaxE + ee];
        }
        __threadfence();  // release: this wave's logit stores before the count
        uint32_t prev = 0;
        if (lane == 0) prev = atomicAdd(xcnt, 1u);
        prev = lane_value(prev, 0);
        if (lane == 0) L.last = prev == (uint32_t)(nblk - 1) ? 1 : 0;
      }
      __syncthreads();
      if (!L.last) return;
      if (tid < kWave) {
        __threadfence();  // acquire: every block's logits
        for (int i = lane; i < T * E; i += kWave) {
          const int t = i / E, ee = i - t * E;
          qs[t * kMaxE + ee] = xq[t * kMaxE + ee];
        }
        if (lane == 0) atomicExch(xcnt, 0u);  // every block has counted: ready for the next launch
      }
      __syncthreads();
    }
  } else {
    for (int i = tid; i < T * E; i += 256) {
      const int t = i / E, e = i - t * E;
      qs[t * kMaxE + e] = p.h[(size_t)t * p.ldh + e];
    }
    __syncthreads();
  }
  for (int t = wv; t < T; t += 4) {
    bool cand = lane < E;
    const uint32_t key = cand ? f32_order_key(qs[t * kMaxE + lane]) : 0u;
    for (int r = 0; r < k; ++r) {
      const int e = wave_pick_max(key, cand);
      if (lane == 0) {
        ids_l[t * k + r] = e;
        p.pred_ids[t * k + r] = e;
      }
    }
  }
  __syncthreads();
  plan_spec_body(a, ids_l, L.sh, &ps);
}

__global__ __launch_bounds__(256) void k_predict_plan(PredictPlanArgs p) {
  __shared__ PredictLds L;
  predict_plan_body(p, L, blockIdx.x);
}

// ============================================================ precise plan + permutation
struct PreciseLds {
  int cnt_e[kMaxE], pos_of[kMaxE], order[kMaxE], offs[kMaxE + 1], fill[kMaxE];
  int n_pos;
  int wave_cnt[4][kMaxE];
};

// The precise plan over the routed ids `ids` [T x k] (global, or LDS when the
// top-k ran in the same block).  All 256 threads of the block enter.
__device__ __forceinline__ void plan_precise_body(const PlanArgs& a, const int32_t* ids, PreciseLds& sh,
                                                  const PlanState* pre = nullptr) {
  int* cnt_e = sh.cnt_e;
  int* pos_of = sh.pos_of;
  int* order = sh.order;
  int* offs = sh.offs;
  int* fill = sh.fill;
  int& n_pos = sh.n_pos;
  const int tid = threadIdx.x, lane = tid % kWave;
  const int npairs = a.T * a.k;
  if (tid < kMaxE) { cnt_e[tid] = 0; fill[tid] = 0; }
  __syncthreads();
  for (int i = tid; i < npairs; i += 256) atomicAdd(&cnt_e[ids[i]], 1);
  __syncthreads();

  WaveState w;
  uint32_t clock, fseq;
  int64_t cnt[kCounters];
  if (tid < kWave) {
    uint64_t pred_mask;
    if (pre) {
      w = pre->w;
      clock = pre->clock;
      fseq = pre->fseq;
#pragma unroll
      for (int i = 0; i < kCounters; ++i) cnt[i] = pre->cnt[i];
      pred_mask = pre->pred_mask;
    } else {
      load_state(a, lane, w, clock, fseq, cnt);
      pred_mask = a.st.pred_mask[a.layer];
    }
    const bool used = lane < a.E && cnt_e[lane] > 0;
    const bool res = used && w.slot_of >= 0;
    const uint32_t fs = __shfl(w.fetch, w.slot_of >= 0 ? w.slot_of : 0, kWave);
    const uint64_t hmask = __ballot(res);
    const uint64_t mmask = __ballot(used && !res);
    cnt[CNT_PRED_CORRECT] += __popcll(pred_mask & (hmask | mmask));
    const int nh = __popcll(hmask), np = nh + __popcll(mmask);
    // rank among the hits by (fetch sequence, id): one scalar read per hit
    int hit_rank = 0;
    for (uint64_t m = hmask; m; m &= m - 1) {
      const int j = __builtin_ctzll(m);
      const uint32_t fj = lane_value(fs, j);
      if (fj < fs || (fj == fs && j < lane)) ++hit_rank;
    }
    int rank = -1;
    if (!a.reorder) {
      // id order; every member is classified at its turn in the walk below
      const uint64_t umask = __ballot(used);
      if (used) rank = __popcll(umask & ((1ull << lane) - 1ull));
    } else if (res) {
      rank = hit_rank;
    } else if (used) {
      rank = nh + __popcll(mmask & ((1ull << lane) - 1ull));
    }
    pos_of[lane] = rank;
    if (rank >= 0) order[rank] = lane;
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();

    // lane `pos` keeps position pos's record entries; they are stored at the
    // end, one coalesced store per field (the record lives in host memory)
    PlanRecord* rec = a.rec;
    int n_hit = 0;
    int my_e = 0, my_s = 0, my_f = 0, my_v = -1, my_a = -1;
    const int ord_lane = lane < np ? order[lane] : 0;  // the expert at position lane
    for (int pos = 0; pos < np; ++pos) {
      const int e = lane_value(ord_lane, pos);
      // reordered: positions below nh are the resident members; id order: resident now
      const int s = lane_value(w.slot_of, e);
      if (s >= 0) {
        ++n_hit;
        ++clock;
        const int was_spec = lane_value(w.spec_unused, s);
        if (lane == s) { w.stamp = clock; w.spec_unused = 0; }
        cnt[CNT_HIT]++;
        if (was_spec) cnt[CNT_SPEC_USED]++;
        if (lane == pos) { my_e = e; my_s = s; my_f = 0; my_v = -1; my_a = -1; }
      } else {
        const int v = victim_slot(a, lane, w);
        const int old = fill_slot(a, lane, w, e, v, false, clock, fseq, cnt);
        cnt[CNT_MISS]++;
        // an earlier member must finish reading the slot; a later one was never read
        const int po = old >= 0 ? lane_value(rank, old) : -1;
        const int after = po < pos ? po : -1;
        if (lane == pos) { my_e = e; my_s = v; my_f = 1; my_v = old; my_a = after; }
      }
    }
    cnt[CNT_PREC] += np;
    store_state(a, lane, w, clock, fseq, cnt);
    if (lane == 0) a.st.pred_mask[a.layer] = 0ull;
    // pair offsets of the positions: an exclusive prefix sum over the np positions
    const int my_c = lane < np ? cnt_e[ord_lane] : 0;
    int excl = 0, total = 0;
    for (int j = 0; j < np; ++j) {
      const int c = lane_value(my_c, j);
      if (j < lane) excl += c;
      total += c;
    }
    if (lane < np) {
      rec->expert[lane] = my_e;
      rec->slot[lane] = my_s;
      rec->flag[lane] = my_f;
      rec->victim[lane] = my_v;
      rec->after[lane] = my_a;
      rec->count[lane] = my_c;
      rec->offset[lane] = excl;
      a.d_order_slot[lane] = my_s;
      a.d_offsets[lane] = excl;
      offs[lane] = excl;
    }
    if (lane == 0) {
      offs[np] = total;
      rec->offset[np] = total;
      a.d_offsets[np] = total;
      rec->kind = 1;
      rec->layer = a.layer;
      rec->n = np;
      rec->n_hit = n_hit;
      a.d_npos[0] = n_hit;
      n_pos = np;
    }
  }
  __syncthreads();

  // Permutation: pairs in (t, r) order are placed into their position's range,
  // keeping (t, r) order inside a range.  Tiles of 256 pairs; inside a wave the
  // lanes with the same position are found with six ballots (one per bit of the
  // position), which gives each pair its rank among the earlier lanes; the waves'
  // counts are then prefixed through LDS.
  int (&wave_cnt)[4][kMaxE] = sh.wave_cnt;
  const int wave = tid / kWave;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int base = 0; base < npairs; base += 256) {
    const int i = base + tid;
    const int pos = i < npairs ? pos_of[ids[i]] : -1;
    for (int e = tid; e < 4 * kMaxE; e += 256) (&wave_cnt[0][0])[e] = 0;
    uint64_t same = __ballot(pos >= 0);
#pragma unroll
    for (int bit = 0; bit < 6; ++bit) {
      const bool on = pos >= 0 && ((pos >> bit) & 1);
      const uint64_t bal = __ballot(on);
      same &= on ? bal : ~bal;
    }
    const int rank_in_wave = __popcll(same & lt_mask);
    __syncthreads();
    if (pos >= 0 && rank_in_wave == 0) wave_cnt[wave][pos] = __popcll(same);
    __syncthreads();
    if (pos >= 0) {
      int before = fill[pos];
      for (int w = 0; w < wave; ++w) before += wave_cnt[w][pos];
      a.d_perm[offs[pos] + before + rank_in_wave] = i;
    }
    __syncthreads();
    if (tid < kMaxE) fill[tid] += wave_cnt[0][tid] + wave_cnt[1][tid] + wave_cnt[2][tid] + wave_cnt[3][tid];
    __syncthreads();
  }
  if (tid == 0 && a.host_done) {
    __threadfence_system();
    a.rec->done = 1;
  }
}

__global__ __launch_bounds__(256) void k_plan_precise(PlanArgs a) {
  __shared__ PreciseLds sh;
  plan_precise_body(a, a.ids, sh);
}

// Decode-sized steps: the router's top-k and the precise plan in one block
// (one launch and no global round trip between them).  T * k <= kFusedRouteMaxPairs.
__global__ __launch_bounds__(256) void k_route_plan(TopkArgs tk, PlanArgs a) {
  __shared__ int32_t ids_l[kFusedRouteMaxPairs];
  __shared__ PreciseLds sh;
  PlanState ps;
  if (threadIdx.x < kWave) load_plan_state(a, threadIdx.x, ps);
  for (int t = threadIdx.x / kWave; t < tk.T; t += 4) topk_token(tk, t, threadIdx.x % kWave, ids_l);
  __syncthreads();
  plan_precise_body(a, ids_l, sh, &ps);
}

// The same, with the layer's prediction in blocks 1 .. pred_blocks(E, Ph): its
// second layer, top-k and the spec plan of the target layer (disjoint cache
// state; the plan records are the route's and the prediction's), so the
// prediction needs no launch or stream of its own.
union RoutePredictLds {
  struct {
    int32_t ids_l[kFusedRouteMaxPairs];
    PreciseLds sh;
  } route;
  PredictLds pred;
};

__global__ __launch_bounds__(256) void k_route_plan_predict(TopkArgs tk, PlanArgs a, PredictPlanArgs p) {
  __shared__ RoutePredictLds L;
  if (blockIdx.x >= 1) {
    predict_plan_body(p, L.pred, blockIdx.x - 1);
    return;
  }
  PlanState ps;
  if (threadIdx.x < kWave) load_plan_state(a, threadIdx.x, ps);
  for (int t = threadIdx.x / kWave; t < tk.T; t += 4) topk_token(tk, t, threadIdx.x % kWave, L.route.ids_l);
  __syncthreads();
  plan_precise_body(a, L.route.ids_l, L.route.sh, &ps);
}

// ============================================================ state init / warm start
__global__ void k_state_init(CacheState st, int L, int C, int E) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < L * C) { st.slot_expert[i] = -1; st.stamp[i] = 0u; st.fetch_seq[i] = 0u; st.spec_unused[i] = 0; }
  if (i < L * E) st.slot_of[i] = -1;
  if (i < L) { st.clock[i] = (uint32_t)(C - 1); st.fseq[i] = 0u; st.pred_mask[i] = 0ull; st.pred_xcnt[i] = 0u; }
  if (i < L * kCounters) st.counters[i] = 0;
}

__global__ void k_warm(CacheState st, int layer, int C, int E, const int32_t* experts, int n) {
  const int s = threadIdx.x;
  if (s < n) {
    const int e = experts[s];
    st.slot_expert[layer * C + s] = e;
    st.slot_of[layer * E + e] = s;
    st.stamp[layer * C + s] = (uint32_t)s;
    st.fetch_seq[layer * C + s] = 0u;
    st.spec_unused[layer * C + s] = 0;
  }
}

// ============================================================ launchers
void launch_topk(const TopkArgs& a, hipStream_t s) {
  k_topk<<<(a.T + 3) / 4, 256, 0, s>>>(a);
}
void launch_plan_spec(const PlanArgs& a, hipStream_t s) { k_plan_spec<<<1, 256, 0, s>>>(a); }
void launch_predict_plan(const PredictPlanArgs& p, hipStream_t s) {
  k_predict_plan<<<pred_blocks(p.plan.E, p.Ph), 256, 0, s>>>(p);
}
void launch_plan_precise(const PlanArgs& a, hipStream_t s) { k_plan_precise<<<1, 256, 0, s>>>(a); }
void launch_route_plan(const TopkArgs& tk, const PlanArgs& a, hipStream_t s) { k_route_plan<<<1, 256, 0, s>>>(tk, a); }
void launch_route_plan_predict(const TopkArgs& tk, const PlanArgs& a, const PredictPlanArgs& p, hipStream_t s) {
  k_route_plan_predict<<<1 + pred_blocks(p.plan.E, p.Ph), 256, 0, s>>>(tk, a, p);
}
void launch_state_init(CacheState st, int L, int C, int E, hipStream_t s) {
  int n = L * (C > E ? C : E);
  if (n < L * kCounters) n = L * kCounters;
  k_state_init<<<(n + 255) / 256, 256, 0, s>>>(st, L, C, E);
}
void launch_warm(CacheState st, int layer, int C, int E, const int32_t* d_experts, int n, hipStream_t s) {
  k_warm<<<1, 64, 0, s>>>(st, layer, C, E, d_experts, n);
}

}  // namespace promoe
