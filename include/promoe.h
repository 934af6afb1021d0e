/*
 * promoe.h -- C ABI of an MI355X (gfx950) proactive expert cache for
 * Mixture-of-Experts inference, after ProMoE (arXiv 2410.22134, "ProMoE: Fast
 * MoE-based LLM Serving using Proactive Caching").
 *
 * One MoE layer step is   promoe_route
 *                      -> promoe_predict (optional)
 *                      -> promoe_expert_ffn
 * on one stream (with lookahead 0 promoe_predict comes first: it plans the
 * layer the route then uses).  promoe_predict may also precede the route at
 * any lookahead; after it, the low-priority copies it queues for layer
 * l+lookahead go behind layer l's high-priority ones.  With lookahead >= 1 it
 * may also follow promoe_expert_ffn (while d_x still holds layer l's input).
 * The predictor of layer
 * l scores the experts of layer l+lookahead and queues their missing chunks as
 * low-priority copies (the paper's PushPredictedExperts, Alg. 2); the route
 * call gates layer l, drops the layer's remaining low-priority work, queues
 * its missing experts at high priority and returns the reordered expert list
 * (PushPreciseExperts, Alg. 2, "Early Preemption", "Reordered Inference"); the
 * FFN call computes the experts in that order, each waiting only for its own
 * chunks (the dependency mechanism of Sec. "System Integration").
 *
 * Conventions
 *  - Every call returns an int: 0 (PROMOE_OK) or a negative promoe_err.
 *    No C++ exception crosses this boundary.
 *  - d_* arguments are device pointers, h_* host pointers; a `stream`
 *    argument is a hipStream_t passed as void* (NULL = the null stream).
 *  - A token count T must be 1..max_tokens; otherwise (an empty step
 *    included) the call returns PROMOE_EINVAL before any device work.
 *  - Matrices are row-major with the reduction dimension contiguous.
 *    Element type is the config dtype: fp32, or bf16 (raw 16-bit words).
 *  - A routed expert is stored as [Wg (I x H) | Wu (I x H) | Wd (H x I)],
 *    3*I*H elements, in pinned host memory and in cache slots alike; the three
 *    matrices are the expert's three copy chunks (Sec. "Chunked Prefetching").
 *  - Ownership: the caller owns every d_* / h_* buffer, the cache region and
 *    the streams; buffers given to set_* calls must outlive the context.  The
 *    library owns its copy streams, events, worker thread, slot tables,
 *    counters and scratch buffers (allocated in promoe_create).
 *  - One context per GPU; calls on a context come from one host thread.
 *    Asynchronous kernel faults surface as PROMOE_EHIP at the next call that
 *    synchronises.
 */
#ifndef PROMOE_H
#define PROMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct promoe_ctx promoe_ctx;

typedef enum {
  PROMOE_OK = 0,
  PROMOE_EINVAL = -1,  /* bad argument: null pointer, index or size out of range */
  PROMOE_ENOMEM = -2,  /* a library allocation failed */
  PROMOE_EHIP = -3,    /* a HIP runtime call failed (see promoe_last_error_string) */
  PROMOE_ESTATE = -4,  /* call order violated (e.g. expert_ffn without route) */
  PROMOE_EUNSUP = -5   /* shape outside what the kernels support */
} promoe_err;

enum { PROMOE_F32 = 0, PROMOE_BF16 = 1 };
enum { PROMOE_WEIGHTS_DENSE = 0, PROMOE_WEIGHTS_INT4 = 1 };
enum { PROMOE_PRIO_LOW = 0, PROMOE_PRIO_HIGH = 1 };

/* flags.  The NO_* switches turn off one technique each, for the paper's
   ablation (Sec. "Evaluation", ablation study: the LRU baseline plus prefetch,
   chunked prefetch, early preemption and reordered inference in turn) and its
   baselines.  All of them leave the outputs unchanged. */
#define PROMOE_FLAG_PROFILE 1      /* time expert launches on the device clock and copy
                                      stalls with HIP events */
#define PROMOE_FLAG_NO_PREFETCH 2  /* predictions update nothing (Sec. "Expert Prefetching" off) */
#define PROMOE_FLAG_NO_CHUNK 4     /* a low-priority task is a whole expert: once started,
                                      all its bytes are queued at once (Sec. "Chunked
                                      Prefetching" off) */
#define PROMOE_FLAG_NO_PREEMPT 8   /* a route neither drops the layer's queued low-priority
                                      work nor issues its copies: each expert that is not
                                      fully issued is fetched on access, after the compute
                                      of the previous position (Sec. "Early Preemption" off) */
#define PROMOE_FLAG_NO_REORDER 16  /* experts run in ascending id order and the precise
                                      plan classifies each at its turn, so an earlier miss
                                      may evict a later routed expert (Sec. "Reordered
                                      Inference" off) */
#define PROMOE_FLAG_STATIC 32      /* static cache baseline: the first C-2 slots keep their
                                      initial experts for good, misses rotate through the
                                      last 2 (LRU among them).  Needs C >= 3. */
#define PROMOE_FLAG_FILL_BY_DEADLINE 64  /* a predictor-driven plan fills only as many slots
                                      as the host link can copy before the target layer's
                                      route: floor((link rate x lookahead x mean interval
                                      between routes - bytes already queued or in flight)
                                      / expert bytes), at most spec_fill_limit when that is
                                      > 0.  The paper's prefetcher replaces a slot only when
                                      the copy starts and drops what has not started when
                                      the route comes (Alg. 1, "Early Preemption"); a fill
                                      that cannot land in time would only move mispredicted
                                      bytes and evict.  Plans depend on host timing; each
                                      records the budget it used. */

typedef struct promoe_config {
  int32_t n_layers;          /* L */
  int32_t hidden;            /* H, multiple of 8 */
  int32_t n_experts;         /* E routed experts per layer, 1..64 */
  int32_t top_k;             /* k, 1..min(E, 8) */
  int32_t inter;             /* I of a routed expert, multiple of 8 */
  int32_t shared_inter;      /* total I of the resident shared expert(s); 0 = none.
                                Several shared experts are passed as one: gate/up rows
                                stacked, down columns stacked. */
  int32_t shared_gate;       /* 0: shared output weight 1; 1: sigmoid(w_sg . x) */
  int32_t renorm;            /* 1: renormalise the top-k gate weights to sum 1 */
  int32_t router_bias;       /* 1: an fp32 per-expert bias is added to the gate logits */
  int32_t slots_per_layer;   /* C cache slots per layer, 1..64 */
  int32_t lookahead;         /* d: the predictor of layer l targets layer l+d (d >= 0) */
  int32_t pred_hidden;       /* 0: predictor is one GEMV Wp [E x H];
                                else a 2-layer MLP: W1 [pred_hidden x H], W2 [E x pred_hidden];
                                a multiple of 8 */
  int32_t max_tokens;        /* T limit of every call (1..8192 / top_k) */
  int32_t dtype;             /* PROMOE_F32 or PROMOE_BF16 */
  int64_t copy_subchunk_bytes; /* copy issue unit; 0 = 16 MiB */
  int32_t copy_window;       /* low-priority sub-copies kept in flight; 0 = 2 */
  int32_t flags;             /* PROMOE_FLAG_* */
  int32_t spec_fill_limit;   /* Slots a predictor-driven plan (promoe_predict) may fill
                                (Alg. 2 PushPredictedExperts).  0: no limit, every
                                predicted expert that is not resident takes a slot;
                                n > 0: only the first n non-resident experts of the
                                vote order take one, the rest are skipped; -1: none,
                                the plan only refreshes the LRU stamps of resident
                                predicted experts.  The paper's worker replaces a slot
                                only when a copy starts; a limit models how few
                                low-priority copies start before the layer's route
                                when the host link is the bottleneck.  Lists passed to
                                promoe_prefetch are never limited.  -1..64. */
  int32_t weight_format;     /* Storage of the routed experts (host copies and cache
                                slots alike).  PROMOE_WEIGHTS_DENSE: dtype elements.
                                PROMOE_WEIGHTS_INT4: 4-bit codes for models quantised to
                                four bits (the paper's larger models, Sec. "Evaluation"):
                                each matrix of R rows and reduction length K is R x K/2
                                bytes of codes, row-major, two per byte (even k in the
                                low nibble), then R x K/128 bf16 scales, row-major; the
                                weight at (r, k) is (code - 8) * scale[r][k / 128].
                                Needs dtype bf16 and hidden, inter multiples of 128.
                                Gates, predictors and shared experts stay in dtype. */
  float link_gb_per_s;       /* host-to-device rate assumed by PROMOE_FLAG_FILL_BY_DEADLINE,
                                GB/s; 0 = 56 (PCIe Gen5 x16 as measured on MI355X) */
} promoe_config;

typedef struct promoe_stats {
  /* Logical counters, decided on the device in program order; exact. */
  int64_t prec_access;    /* distinct experts routed, summed over route calls */
  int64_t hit;            /* routed experts already slot-assigned */
  int64_t miss;           /* routed experts given a slot at route time */
  int64_t spec_issued;    /* predicted experts given a slot */
  int64_t spec_resident;  /* predicted experts already resident (touched) */
  int64_t spec_used;      /* speculatively filled slots later hit */
  int64_t spec_wasted;    /* speculatively filled slots evicted unused */
  int64_t evict;          /* slot reassignments that displaced an expert */
  int64_t pred_n;         /* experts in predictor-driven plans (|Q| summed) */
  int64_t pred_correct;   /* of those, routed at the layer's next route: accuracy =
                             pred_correct / pred_n (Sec. "A New Prediction Metric:
                             GoodPred"; per token when T = 1) */
  /* Physical counters (host side). */
  int64_t copies_high, copies_low;  /* sub-copies issued per priority */
  int64_t bytes_high, bytes_low;    /* bytes issued per priority */
  int64_t low_purged;               /* queued low-priority sub-copies dropped by route */
  int64_t deferred;                 /* high copies held behind an earlier position's
                                       compute: the slot's previous reader (write after
                                       read), or the previous position (NO_PREEMPT) */
  int64_t pred_in_time;             /* correctly predicted experts whose bytes had all
                                       landed in HBM when the route ran: FetchRate =
                                       pred_in_time / pred_correct */
  /* Timing, PROMOE_FLAG_PROFILE only.  Expert launches are timed by start and
     end events that the launch itself records (kernel execution time); classes:
     [0] GEMV gate/up, [1] GEMV down, [2] GEMM gate/up (routed experts),
     [3] GEMM down (routed), [4] GEMM gate/up (shared expert), [5] GEMM down (shared). */
  int64_t k_launches[6];
  double k_ms[6];         /* summed launch time */
  double k_bytes[6];      /* summed algorithmic weight bytes */
  double k_flops[6];      /* summed algorithmic flops */
  double stall_ms;        /* compute stream time spent waiting on copies (HIP events) */
  double copy_ms;         /* reserved (0) */
  int64_t lazy_routes;    /* decode routes that returned without waiting for their plan
                             on the host: every expert of every layer resident (slots ==
                             experts, each layer's initial cache full), the resident launch
                             covering the step, and no order asked for; their plans are
                             taken in once complete (stats, sync and later routes).  At
                             one token such a route's prediction runs in front of the
                             row tiles of its resident gate/up launch, which the gate/up
                             launch timing (k_ms[0]) then includes */
} promoe_stats;

typedef struct promoe_plan {
  /* The last plan of a layer, as decided on the device.
     kind 0 (spec):    expert[i], slot[i], flag[i] = 1 if newly assigned, victim[i].
     kind 1 (precise): expert[i] = order, slot[i] = slot the position computes from,
                       flag[i] = 1 for a miss, victim[i], after[i] = earlier position whose
                       compute must finish before the fill (-1 none), count[i] = tokens. */
  int32_t n;
  int32_t expert[64], slot[64], flag[64], victim[64], after[64], count[64];
  int32_t fill_budget;  /* kind 0: most slots the plan could fill (-1: no limit) */
} promoe_plan;

/* ---- lifetime ------------------------------------------------------------ */

/* Create a context on the current HIP device (Sec. "Cache Implementation": a
 * per-layer LRU cache of experts whose storage is one contiguous region
 * allocated up front).  d_cache is the caller's cache region of at least
 * n_layers*slots_per_layer*expert_bytes bytes (slot s of layer l at offset
 * (l*C+s)*expert_bytes).  All slots start free.
 * Errors: EINVAL (null/size), EUNSUP (E > 64, C > 64, k > 8, H, I,
 * shared_inter or pred_hidden not a multiple of 8), ENOMEM, EHIP. */
int promoe_create(const promoe_config* cfg, void* d_cache, size_t cache_bytes, promoe_ctx** out);

/* Drain all copies, stop the worker and free library resources. */
int promoe_destroy(promoe_ctx* ctx);

/* ---- weights ------------------------------------------------------------- */

/* Resident weights of a layer (device pointers, caller-owned):
 *  d_wgate [E x H]; d_bias [E] fp32 (router_bias only, else NULL);
 *  d_pw1, d_pw2: predictor owned by this layer, targeting layer+lookahead
 *    (Sec. "Learning-based Predictor"): Wp [E x H] (pred_hidden == 0, d_pw2 NULL)
 *    or W1 [pred_hidden x H], W2 [E x pred_hidden]; NULL when the layer has none;
 *  d_shared: [Wg | Wu | Wd] of the shared expert(s) with I = shared_inter, or NULL;
 *  d_shared_gate [H] (shared_gate only). */
int promoe_set_layer(promoe_ctx* ctx, int layer, const void* d_wgate, const float* d_bias,
                     const void* d_pw1, const void* d_pw2, const void* d_shared,
                     const void* d_shared_gate);

/* Host copy of routed expert `expert` of `layer`: pinned memory (e.g. from
 * promoe_host_alloc) holding [Wg | Wu | Wd]. */
int promoe_set_expert_host(promoe_ctx* ctx, int layer, int expert, const void* h_pinned);

/* Warm start: experts h_experts[0..n) are copied (synchronously) into slots
 * 0..n) of the layer and become resident with LRU order = slot order.  Not
 * counted.  Must precede the layer's first plan.  n <= slots_per_layer. */
int promoe_set_initial_cache(promoe_ctx* ctx, int layer, const int32_t* h_experts, int n);

/* ---- the hot path -------------------------------------------------------- */

/* Look-ahead prediction (Sec. "Learning-based Predictor", "Stride Prefetching";
 * Alg. 2 PushPredictedExperts).  One fused pass over d_x [T x H] computes the
 * gate logits of `layer` (reused by the next promoe_route of that layer on the
 * same d_x; skipped when the latest route was of this layer on the same d_x
 * and T, before or after its promoe_expert_ffn) and the
 * predictor of layer+lookahead; per-token top-k of the
 * predictor output; an integer vote merges the tokens' picks into a list Q of
 * at most slots_per_layer experts (votes desc, best rank asc, id asc); the
 * target layer's cache is planned on the device: first every resident member
 * of Q is touched (Alg. 2 counts these hits as it pushes the list), then each
 * other member, in Q order, takes the lowest free slot or the least recently
 * used one whose expert the prediction does not vote for (the worker of
 * Alg. 1 replaces a slot only when a copy starts, after the list is pushed;
 * trading one predicted expert for another only adds copies), and its three
 * chunks are queued at low priority, copied by the library's worker thread;
 * a member with no such slot, or past cfg.spec_fill_limit, is skipped.
 * The kernels after the predictor's first rows run on a side stream of the
 * library, forked from `stream` once those rows are written and joined back
 * into it before the call returns: they overlap expert work already queued
 * on `stream`, and everything queued on `stream` later follows them.
 * Optional outputs: d_pred_ids [T x k] per-token predicted ids; h_q/n_q the
 * list Q (requesting it synchronises the stream).  When layer+lookahead is
 * past the last layer only the gate logits are computed and *n_q = 0. */
int promoe_predict(promoe_ctx* ctx, int layer, const void* d_x, int T, int32_t* d_pred_ids,
                   int32_t* h_q, int32_t* n_q, void* stream);

/* Route `layer` (Background "MoE based LLMs"; "Early Preemption";
 * "Reordered Inference"; Alg. 2 PushPreciseExperts).  Gate logits
 * (+bias), softmax, top-k by (logit desc, id asc), weights renormalised over
 * the k if cfg.renorm -> d_ids [T x k] int32, d_w [T x k] fp32, and for a gated
 * shared expert d_shared_scale [T] = sigmoid(w_sg . x) (else may be NULL).
 * Then the precise plan: pending low-priority copies of the layer are dropped,
 * order = resident experts by fill order then missing experts by id; missing
 * experts get slots and are copied at high priority.  A missing expert whose
 * slot a resident one of the same step must read first is copied after that
 * read; for steps of more than 64 routed tokens (T * k) the route itself
 * enqueues the FFN of the readers of the first two such slots, right behind
 * the plan, so those copies start while the caller goes on (the FFN call
 * computes the rest; d_x must keep its contents until then, as for the FFN
 * call).  Synchronises with the stream once.  h_order [>= E] receives the
 * order, *n_order its length. */
int promoe_route(promoe_ctx* ctx, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                 float* d_shared_scale, int32_t* h_order, int32_t* n_order, void* stream);

/* promoe_route of `layer` followed by promoe_predict of the same layer on the
 * same input (d_pred_ids as there; Q is not returned), in one call: the
 * predictor's first rows ride in the gate launch.  For steps of up to 8 tokens
 * whose routed pairs (T * k) number at most 64 (and predictor width at most
 * 1024), the rest of the prediction -- second layer, top-k and the spec plan
 * of layer+lookahead -- runs in further blocks of the route's plan kernel on
 * `stream` (the second layer's rows spread over them, the block that finishes
 * last taking the top-k and the plan): the host still reads the precise plan as soon as its block has
 * written it, and d_pred_ids is complete when that kernel is.  Otherwise the
 * predictor's other kernels run on the library's side stream, launched while
 * the host waits for the precise plan, with no device-side join: the spec
 * plan that ends them is awaited on the host by the context's next
 * promoe_route, promoe_route_predict, promoe_predict, promoe_prefetch or
 * promoe_sync call, before that call queues anything (without a spec plan,
 * e.g. with PROMOE_FLAG_NO_PREFETCH, the layer's promoe_expert_ffn call joins
 * the side stream into `stream` after its last launch); there d_pred_ids is
 * complete once such a call has returned.
 * Needs cfg.lookahead >= 1 (with 0 the prediction plans the routed layer
 * itself and must come first), else PROMOE_EINVAL.  Results are those of the
 * two calls made in that order. */
int promoe_route_predict(promoe_ctx* ctx, int layer, const void* d_x, int T, int32_t* d_ids, float* d_w,
                         float* d_shared_scale, int32_t* d_pred_ids, int32_t* h_order, int32_t* n_order,
                         void* stream);

/* External push of a list of experts for `target_layer` (Alg. 2
 * PushPredictedExperts with a caller-chosen list): the same device plan as a
 * prediction; prio selects the copy queue. */
int promoe_prefetch(promoe_ctx* ctx, int target_layer, const int32_t* h_ids, int n, int prio,
                    void* stream);

/* Expert FFN of the routed layer (Background; Sec. "Reordered Inference"):
 * for every (t, r): Y = Wd (bf16|fp32)(silu(Wg x_t) * (Wu x_t)) with the
 * expert read from its cache slot, experts computed in the route order and
 * each launch waiting only on its own chunks; plus the shared expert;
 * d_y [T x H] = sum_r d_w[t,r] Y[t,r] (fixed r order) + s_t Y_shared[t],
 * rounded once to the config dtype.  d_x, d_ids, d_w, d_shared_scale must be
 * the ones passed to promoe_route for this layer. */
int promoe_expert_ffn(promoe_ctx* ctx, int layer, const void* d_x, int T, const int32_t* d_ids,
                      const float* d_w, const float* d_shared_scale, void* d_y, void* stream);

/* Allocation-free variant of promoe_expert_ffn, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same contract, arguments and result as
 * promoe_expert_ffn (the outputs are the same values), but the activations
 * and expert outputs its kernels exchange live in a file-scope device array of
 * PROMOE_NOALLOC_SCRATCH_BYTES (8 MiB) that each GPU the library runs on holds
 * until the process ends, not in the context's buffers.  The call itself
 * allocates no device memory and is never timed (PROMOE_FLAG_PROFILE does not
 * apply to it); 4-bit experts always take the dequantising GEMV.
 * Limits: at most 64 routed pairs (T * top_k <= 64, the decode sizes), and a
 * scratch need of at most 8 MiB: T*k*I*s + T*k*H*4 + T*I_sh*s + n*T*H*4 bytes
 * (s = bytes per element of the config dtype, n = split-K slices of the shared
 * expert's down product, 1 unless T >= 16), each term rounded up to 256.
 * Beyond either limit the call returns PROMOE_EINVAL before any device work
 * (the route stays pending; promoe_expert_ffn may then consume it).  Every
 * call on one GPU shares that GPU's array: calls that overlap on one GPU (two
 * contexts, or two streams of one context) race.  Nothing in the array needs
 * to start at zero: every byte a kernel reads is written earlier in the same
 * call. */
#define PROMOE_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)
int promoe_expert_ffn_noalloc(promoe_ctx* ctx, int layer, const void* d_x, int T, const int32_t* d_ids,
                              const float* d_w, const float* d_shared_scale, void* d_y, void* stream);

/* ---- state and statistics ------------------------------------------------ */

/* Counters behind the paper's metrics (Sec. "A New Prediction Metric: GoodPred":
 * Accuracy = pred_correct / pred_n, FetchRate = pred_in_time / pred_correct,
 * GoodPred = Accuracy x FetchRate; Sec. "Evaluation": hit and miss counts, bytes
 * copied per priority, the stall of compute on copies).  Logical counters of
 * one layer, or of all layers summed (layer = -1); the physical counters and
 * timings always cover all layers.  Synchronises.  Errors: EINVAL (null out,
 * layer out of range), EHIP (a copy or kernel failed). */
int promoe_cache_stats(promoe_ctx* ctx, int layer, promoe_stats* out);
int promoe_reset_stats(promoe_ctx* ctx);
/* h_slot_of [E]: slot of each expert of the layer, -1 if not resident.  Synchronises. */
int promoe_slot_table(promoe_ctx* ctx, int layer, int32_t* h_slot_of);
/* Last spec (kind 0) or precise (kind 1) plan of a layer.  Synchronises. */
int promoe_last_plan(promoe_ctx* ctx, int layer, int kind, promoe_plan* out);
/* Wait for all queued copies and compute issued through the context. */
int promoe_sync(promoe_ctx* ctx);

/* ---- harness (the layer around the MoE block) ---------------------------- */

/* Attention surrogate weight Wa [H x H] of a layer. */
int promoe_set_attn(promoe_ctx* ctx, int layer, const void* d_wattn);
/* d_h [T x H] fp32 residual stream: h += Wa q(rms(h)); d_x_out = q(rms(h)),
 * rms(v) = v / sqrt(mean(v^2) + 1e-6), q = dtype rounding. */
int promoe_attn_surrogate(promoe_ctx* ctx, int layer, float* d_h, int T, void* d_x_out,
                          void* stream);
/* d_h [T x H] fp32 += d_y [T x H] (config dtype). */
int promoe_residual_add(promoe_ctx* ctx, float* d_h, const void* d_y, int T, void* stream);

/* One step of the whole layer stack in one call, the loop a caller would
 * otherwise drive layer by layer: for each layer l, promoe_attn_surrogate(l)
 * into d_x, then (predict != 0) the prediction and the route as the layer loop
 * orders them (look-ahead 0: promoe_predict then promoe_route; else
 * promoe_route_predict), or the route alone (predict == 0), then
 * promoe_expert_ffn into d_y and promoe_residual_add(d_h, d_y).  The buffers
 * are the caller's and those calls' (d_x, d_y [T x H] dtype; d_ids, d_w [T x
 * k]; d_shared_scale [T], may be NULL without a gated shared expert;
 * d_pred_ids [T x k] or NULL); on return d_h holds the stack's output and the
 * other buffers the last layer's values.  Results equal those of the separate
 * calls made in that order; the first failing call's error is returned and
 * the remaining layers are not run. */
int promoe_stack_step(promoe_ctx* ctx, float* d_h, int T, void* d_x, void* d_y, int32_t* d_ids, float* d_w,
                      float* d_shared_scale, int32_t* d_pred_ids, int predict, void* stream);

/* ---- measurement (not part of the method) --------------------------------
 * Achievable peaks of this GPU; the kernels' rooflines are reported against
 * the nominal peaks and against these.  Both launch asynchronously on `stream`
 * (a hipStream_t; NULL = the null stream) and return PROMOE_EINVAL for a null
 * pointer or a size out of range, PROMOE_EHIP if the launch fails.  The caller
 * owns every buffer. */
/* Reads `bytes` (> 0, a multiple of 16) at d_buf once with 16-byte
 * non-temporal loads, `blocks` blocks of 256 threads, each streaming one
 * contiguous piece of ceil(bytes / blocks) bytes (16-128 KiB pieces read
 * fastest); writes one float per block to d_sink (>= blocks floats). */
int promoe_peak_hbm_read(const void* d_buf, size_t bytes, float* d_sink, int blocks, void* stream);
/* `blocks` blocks of 512 threads; each wave runs `iters` rounds of 32
 * independent v_mfma_f32_16x16x32_bf16 on register operands, i.e.
 * blocks * 8 * iters * 32 * 16384 flops.  Writes blocks * 512 floats to d_sink. */
int promoe_peak_mfma_bf16(float* d_sink, int blocks, int iters, void* stream);

/* ---- utilities ----------------------------------------------------------- */

/* Pinned host memory for expert weights (hipHostMalloc); free with promoe_host_free. */
int promoe_host_alloc(size_t bytes, void** out);
int promoe_host_free(void* p);
size_t promoe_expert_bytes(const promoe_config* cfg);
const char* promoe_strerror(int err);
/* Text of the last HIP error seen by the library in this thread. */
const char* promoe_last_error_string(void);

#ifdef __cplusplus
}
#endif
#endif /* PROMOE_H */
