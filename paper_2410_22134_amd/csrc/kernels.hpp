// Launch-argument structs and host launchers of the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace promoe {

// Rows GEMV: out[t][o_off + j] (=|+=) sum_k W_j[k] * f(x[t][x_off + k]),
// rows j from up to three sources (w[i], nrows[i]) concatenated.
struct RowsArgs {
  const void* w[3];
  int nrows[3];
  int K;
  const void* x;
  int ldx, x_off;
  int T;
  float* out;
  int ldo, o_off;
  int add;      // 1: accumulate into out
  int relu_in;  // 1: f = relu, else identity
};

// Expert FFN launch: a list of jobs (route positions, or the shared expert),
// each job split into row tiles; block b runs tile b - job_tile0[j] of the job
// j with job_tile0[j] <= b < job_tile0[j + 1].
constexpr int kInt4Group = 128;  // 4-bit expert storage: codes per bf16 scale
constexpr int kMaxJobs = 80;  // 64 route positions + pieces of the shared expert
constexpr uint8_t kSharedJob = 255;
// One expert job of an FFN launch (a route position, the shared expert, or a
// piece of the shared expert's rows), 32 bytes: a block reads it with one
// scalar load.
struct alignas(16) FfnJob {
  const void* w;   // expert weights [Wg | Wu | Wd] (slot or resident shared expert); null: a route
                   // position resolved on the device (GEMV kernels; see FfnArgs::npos)
  int32_t q0, q1;  // pair range [q0, q1) (token range for the shared expert)
  int32_t I;       // intermediate size of the expert
  int32_t r0;      // GEMV: first row of the job's piece
  int32_t pos;     // route position, or kSharedJob
  int32_t pad;
};
static_assert(sizeof(FfnJob) == 32, "FfnJob layout");

struct FfnArgs {
  const uint8_t* cache;
  int64_t expert_bytes;
  int layer, slots;
  const int32_t* order_slot;  // [n_pos] slot each position computes from
  const int32_t* offsets;     // [n_pos + 1] pair offsets of each position
  const int32_t* perm;        // [T*k] pair q -> t*k + r
  int hidden, inter, top_k, T;
  const void* x;              // [T x H]
  void* act;                  // [T*k x I] permuted activations
  float* Y;                   // [T*k x H] by (t, r)
  int shared_inter;
  const void* shared_w;       // resident shared expert [Wg | Wu | Wd], I = shared_inter
  void* act_sh;               // [T x I_sh]
  float* Ysh;                 // [T x H]
  int n_jobs;
  int piece_rows;             // GEMV: rows per piece; the shared expert spans several pieces
  int q4;                     // routed experts stored as 4-bit codes (then bf16 scales)
  int ksplit;                   // split-K slices of the shared expert's down GEMM (>= 1)
  int64_t ysh_split_stride;     // elements between the slices' partial outputs in Ysh
  // Jobs with w == null are route positions `pos` resolved on the device from the
  // plan: computed only when pos < npos[0] (the resident positions, which the
  // reordered plan puts first) and the position's slot is not in busy_mask;
  // weights from the slot order_slot[pos], pairs offsets[pos] .. offsets[pos + 1].
  const int32_t* npos;
  uint64_t busy_mask;
  int tail_block0;              // GEMM gate/up of one job: first block of the half-height tail tiles
  int tail_n0;                  // first n-tile (of 128 columns) the tail covers
  int32_t job_tile0[kMaxJobs + 1];  // GEMM: first block of each job in the 1-D grid
  FfnJob jobs[kMaxJobs];
};

struct CombineArgs {
  const float* Y;       // [T*k x H]
  const float* w;       // [T x k]
  const float* Ysh;     // [ysh_split x T x H] partial outputs, summed in slice order, or null
  int ysh_split;
  int64_t ysh_split_stride;
  const float* sscale;  // [T] or null (weight 1)
  void* y;              // [T x H]
  int hidden, top_k;
};

constexpr int kCounters = 10;

// Per-layer logical cache state on the device.
constexpr int kFusedPredMaxT = 8;
constexpr int kFusedPredMaxHidden = 1024;

struct CacheState {
  int32_t* slot_expert;  // [L*C]
  int32_t* slot_of;      // [L*E]
  uint32_t* stamp;       // [L*C]
  uint32_t* fetch_seq;   // [L*C]
  int32_t* spec_unused;  // [L*C]
  uint32_t* clock;       // [L]
  uint32_t* fseq;        // [L]
  int64_t* counters;     // [L*kCounters]: prec_access hit miss spec_issued spec_resident spec_used
                         // spec_wasted evict pred_n pred_correct
  uint64_t* pred_mask;   // [L]: experts of the layer's last prediction not yet routed
  float* pred_xq;        // [L * kFusedPredMaxT * kMaxE]: predictor logits of a target layer, passed
                         // between the blocks of a fused prediction
  uint32_t* pred_xcnt;   // [L]: blocks of that prediction finished (0 between launches)
};

// Plan record written by the plan kernels into host-mapped memory.
struct PlanRecord {
  int32_t kind;   // 0 spec, 1 precise
  int32_t layer;
  int32_t n;
  int32_t n_hit;
  int32_t predicted;  // spec plan from the predictor (not a caller's list)
  int32_t expert[64], slot[64], flag[64], victim[64], after[64], count[64];
  int32_t offset[65];
  int32_t q_in[64];  // host-provided list for promoe_prefetch
  int32_t n_q_in;
  int32_t fill_budget;  // spec plan: most slots it could fill (-1: no limit)
  int32_t done;
};

struct TopkArgs {
  const float* logits;  // [T x ld]; gate logits at column 0..E-1
  int ld;
  int E, k, T;
  const float* bias;    // [E] or null
  int renorm;
  int want_weights;     // 0: ids only (predictor)
  int32_t* ids;         // [T x k]
  float* w;             // [T x k]
  int sgate_col;        // column of the shared-gate logit, -1 none
  float* sscale;        // [T]
};

struct PlanArgs {
  CacheState st;
  int layer, C, E;
  const int32_t* ids;   // [T x k] (precise) or per-token predicted ids (spec); null = use rec->q_in
  int T, k;
  int fill_budget;      // spec plan from ids: most slots filled, -1 = no limit
  int reorder;          // precise plan: 1 hits first (reordered inference), 0 id order
  int pinned;           // slots [0, pinned) are never victims (static cache)
  PlanRecord* rec;      // host-mapped
  int32_t* d_order_slot; // [64]
  int32_t* d_offsets;    // [65]
  int32_t* d_perm;       // [T*k]
  int32_t* d_pos_of;     // [64] scratch
  int32_t* d_npos;       // [1] precise plan: resident positions (reordered: they come first)
  int host_done;         // 1: end with a system-scope fence and the record's done word (the
                         // host polls it); 0: neither (the host waits on the plan's event)
};

// Predictor tail and spec plan in one launch (steps of at most kFusedPredMaxT
// tokens, predictor hidden width at most kFusedPredMaxHidden, a multiple of 8):
// the second layer's rows are spread over blocks of kPredExpertsPerBlock
// experts; the block that finishes last runs the top-k and the spec plan.
constexpr int kPredExpertsPerBlock = 8;
__host__ __device__ inline int pred_blocks(int E, int Ph) { return Ph > 0 ? (E + kPredExpertsPerBlock - 1) / kPredExpertsPerBlock : 1; }
struct PredictPlanArgs {
  PlanArgs plan;        // plan.ids: the predicted-ids output (marks a prediction)
  const float* h;       // [T x ldh] first-layer outputs before relu, or the logits when Ph == 0
  int ldh;
  int Ph;               // hidden width (0: one-layer predictor)
  const void* w2;       // [E x Ph], 16-byte aligned rows
  int w2_bf16;          // 1: bf16 weights, 0: fp32
  int32_t* pred_ids;    // [T x k] out
};
void launch_predict_plan(const PredictPlanArgs& p, hipStream_t s);
// launch_route_plan with the prediction of predict_plan in blocks 1 .. pred_blocks(E, Ph)
void launch_route_plan_predict(const TopkArgs& tk, const PlanArgs& a, const PredictPlanArgs& p, hipStream_t s);

// Expand 4-bit experts into dense bf16 [Wg | Wu | Wd] copies (the MFMA GEMM's
// operand type: each weight (code - 8) * scale is rounded to bf16).
struct DequantArgs {
  const uint8_t* src[8];  // stored experts (cache slots)
  bf16_t* dst;            // n consecutive dense experts
  int n, inter, hidden;
};
constexpr int kStageExperts = 8;
void launch_dequant_q4(const DequantArgs& a, hipStream_t s);

void launch_rows_gemv(const RowsArgs& a, int wdtype, int xdtype, hipStream_t s);
// Batch-1 bf16 rows GEMV over x = q(rms(h)) computed in the kernel, bit for bit
// launch_rmsnorm_quant then launch_rows_gemv; out = (add_src ? add_src : 0) +
// dot; x_out (or null) receives x.  a.x is unused.  Returns false, launching
// nothing, where the separate kernels would not take their register paths.
// With ca (batch 1, bf16, H <= 2048, one shared slice), h is the residual
// before the previous layer's MoE output: the kernel forms y = combine(ca) and
// h' = h + q(y) as launch_combine_residual would, uses h' in place of h and
// of add_src, and stores y to ca->y; h' is not written.
bool launch_rows_gemv_norm(const RowsArgs& a, const float* h, const float* add_src, void* x_out, hipStream_t s,
                           const CombineArgs* ca = nullptr);
// Launches one pass of the GEMV kernels over the jobs (a copy of `a` is
// adjusted per pass; `a` is unchanged).  max_tokens = most pairs of any job.
// With ev0/ev1 set, the launch records them itself at the kernel's start and
// end (hipExtLaunchKernelGGL: kernel execution time, as a profiler sees it).
void launch_ffn(const FfnArgs& a, int pass, int max_tokens, int dtype, hipStream_t s, hipEvent_t ev0 = nullptr,
                hipEvent_t ev1 = nullptr);
// launch_ffn's gate/up pass of a one-token step (dense bf16 experts) with the
// blocks of launch_predict_plan(p) in front of its row tiles; false, launching
// nothing, when the step or the prediction is not of that kind.
bool launch_ffn_gateup_pred(const FfnArgs& a, const PredictPlanArgs& p, int dtype, hipStream_t s,
                            hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Grouped MFMA GEMM (bf16) for the same passes; needs N % 128 == 0 and K % 64 == 0.
bool gemm_supported(int N, int K);
int gemm_shared_down_split(int T, int H);  // split-K slices of the shared down GEMM
// MFMA rows product: out[t][o_off + n] (=|+=) sum_k W[n][k] x[t][k], bf16 in, fp32 out; K % 64 == 0.
struct RowsGemmArgs {
  const void* w;
  int N, K;
  const void* x;
  int ldx, T;
  float* out;
  int ldo, o_off, add;
};
void launch_gemm_rows(const RowsGemmArgs& a, hipStream_t s);
void launch_gemm(FfnArgs& a, int pass, int max_tokens, hipStream_t s, hipEvent_t ev0 = nullptr,
                 hipEvent_t ev1 = nullptr);
void launch_combine(const CombineArgs& a, int T, int dtype, hipStream_t s);
// combine, then h += y, in one launch
void launch_combine_residual(const CombineArgs& a, float* h, int T, int dtype, hipStream_t s);
void launch_rmsnorm_quant(const float* h, void* out, int T, int H, int dtype, hipStream_t s);
void launch_residual_add(float* h, const void* y, int n, int dtype, hipStream_t s);
void launch_topk(const TopkArgs& a, hipStream_t s);
void launch_plan_spec(const PlanArgs& a, hipStream_t s);
void launch_plan_precise(const PlanArgs& a, hipStream_t s);
// the router's top-k and the precise plan in one launch (T * k <= kFusedRouteMaxPairs)
constexpr int kFusedRouteMaxPairs = 64;
void launch_route_plan(const TopkArgs& tk, const PlanArgs& a, hipStream_t s);
void launch_state_init(CacheState st, int L, int C, int E, hipStream_t s);
void launch_warm(CacheState st, int layer, int C, int E, const int32_t* d_experts, int n, hipStream_t s);

}  // namespace promoe
