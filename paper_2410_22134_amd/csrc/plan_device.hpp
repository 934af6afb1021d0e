// Device-side cache-plan and prediction code shared by the plan kernels and
// the expert GEMV launch that can carry a prediction: the LRU wave state, the
// spec plan (Alg. 2 PushPredictedExperts) and the predictor's second layer
// with its top-k, spread over blocks with a last-block handoff.
#pragma once
#include "common.hpp"
#include "kernels.hpp"

namespace promoe {

enum {
  CNT_PREC = 0, CNT_HIT, CNT_MISS, CNT_SPEC_ISSUED, CNT_SPEC_RESIDENT, CNT_SPEC_USED, CNT_SPEC_WASTED, CNT_EVICT,
  CNT_PRED_N, CNT_PRED_CORRECT
};

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

// MAXT: the most tokens a step may have (LDS and registers are sized for it).
template <int MAXT>
struct PredictLds {
  float hs[MAXT * kFusedPredMaxHidden];
  float qs[MAXT * kMaxE];
  int32_t ids_l[MAXT * kMaxK];
  SpecLds sh;
  int last;
};

// blk: this block's index among the prediction's pred_blocks(E, Ph) blocks;
// T <= MAXT.
template <int MAXT>
__device__ __forceinline__ void predict_plan_body(const PredictPlanArgs& p, PredictLds<MAXT>& L, int blk) {
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
      constexpr int kPer = MAXT * kFusedPredMaxHidden / 256;
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
    float acc[MAXT];
#pragma unroll
    for (int t = 0; t < MAXT; ++t) acc[t] = 0.0f;
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
          for (int t = 0; t < MAXT; ++t) {
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
          for (int t = 0; t < MAXT; ++t) {
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
    for (int t = 0; t < MAXT; ++t) {
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

}  // namespace promoe
