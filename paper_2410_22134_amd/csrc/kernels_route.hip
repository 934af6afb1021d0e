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
#include "plan_device.hpp"

namespace promoe {

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

// ============================================================ spec plan, prediction (bodies: plan_device.hpp)
__global__ __launch_bounds__(256) void k_plan_spec(PlanArgs a) {
  __shared__ SpecLds sh;
  plan_spec_body(a, a.ids, sh);
}

__global__ __launch_bounds__(256) void k_predict_plan(PredictPlanArgs p) {
  __shared__ PredictLds<kFusedPredMaxT> L;
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
    if (npairs <= kWave) {
      // every pair in one lane of this wave: its rank among the earlier pairs of
      // its position (six ballots, as below) and the position's offset from the
      // lane that holds it; the same places as the tiled loop below
      const int pos = lane < npairs ? pos_of[ids[lane]] : -1;
      const int off = __shfl(excl, pos >= 0 ? pos : 0, kWave);
      uint64_t same = __ballot(pos >= 0);
#pragma unroll
      for (int bit = 0; bit < 6; ++bit) {
        const bool on = pos >= 0 && ((pos >> bit) & 1);
        const uint64_t bal = __ballot(on);
        same &= on ? bal : ~bal;
      }
      if (pos >= 0) a.d_perm[off + __popcll(same & ((1ull << lane) - 1ull))] = lane;
    }
  }
  if (npairs > kWave) __syncthreads();

  // Permutation: pairs in (t, r) order are placed into their position's range,
  // keeping (t, r) order inside a range.  Tiles of 256 pairs; inside a wave the
  // lanes with the same position are found with six ballots (one per bit of the
  // position), which gives each pair its rank among the earlier lanes; the waves'
  // counts are then prefixed through LDS.
  int (&wave_cnt)[4][kMaxE] = sh.wave_cnt;
  const int wave = tid / kWave;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int base = 0; npairs > kWave && base < npairs; base += 256) {
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
  PredictLds<kFusedPredMaxT> pred;
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
