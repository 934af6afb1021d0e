// Skinny matrix-vector kernels for gfx950 (wave64):
//  * k_rows_gemv   -- gate logits + predictor rows in one pass over x, the
//                     predictor's second layer, the attention surrogate
//                     (k_rows_gemv_reg for groups of up to four tokens);
//  * k_ffn_gateup  -- expert pass 1: gate and up rows of the experts of a
//                     launch segment read together, act = q(silu(a) * b);
//  * k_ffn_down    -- expert pass 2: Y = Wd act, scattered to (token, rank);
//  * k_combine     -- y = sum_r w Y + s Ysh, fixed r order, one rounding
//                     (k_combine_residual also adds y into the residual);
//  * k_rmsnorm_quant(_reg), k_residual_add -- the layer around the MoE block.
//
// Every GEMV lets a wave own R weight rows, with every lane streaming 16-byte
// pieces of them (global_load_dwordx4, coalesced across the wave), accumulating
// in fp32, and the wave reducing at the end.  The rows kernel for larger token
// groups stages the tokens in LDS as fp32 K-slabs shared by the block's four
// waves; the expert GEMVs and the decode rows kernel keep each lane's token
// pieces in registers instead.  Weight bytes are read once per token group of
// up to MT tokens, which is what bounds decode (HBM) throughput.
#include <hip/hip_ext.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "plan_device.hpp"

namespace promoe {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kSlabFloats = 8192;  // LDS slab: MT * KS fp32 = 32 KiB

// Stage x[m][k0 .. k0+ks) for m < mt into LDS as fp32.
template <typename TX, int MT>
__device__ __forceinline__ void stage_slab(float* xs, int ks_stride, const TX* const (&xrow)[MT], int mt, int k0,
                                           int ks, bool relu) {
  const int n = mt * ks;
  for (int idx = threadIdx.x; idx < n; idx += kThreads) {
    const int m = idx / ks, kk = idx - m * ks;
    float v = Elem<TX>::load(xrow[m], k0 + kk);
    xs[m * ks_stride + kk] = relu ? fmaxf(v, 0.0f) : v;
  }
}

// acc[r][m] += sum over the slab of row_r[k] * xs[m][k]; rows already offset to the slab start.
template <typename TW, int R, int MT, int U>
__device__ __forceinline__ void wave_dot_slab(const TW* const (&rows)[R], const bool (&rvalid)[R], const float* xs,
                                              int ks_stride, int mt, int nch, int lane, float (&acc)[R][MT]) {
  constexpr int EPC = Elem<TW>::kPer16B;
  for (int c0 = lane; c0 < nch; c0 += kWave * U) {
    uint4 wc[U][R];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * kWave;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (c < nch && rvalid[r]) wc[u][r] = *reinterpret_cast<const uint4*>(rows[r] + (size_t)c * EPC);
        else wc[u][r] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = c0 + u * kWave;
      if (c >= nch) break;
      float xv[MT][EPC];
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if (m < mt) {
#pragma unroll
          for (int e = 0; e < EPC; e += 4) {
            float4 v = *reinterpret_cast<const float4*>(xs + m * ks_stride + c * EPC + e);
            xv[m][e] = v.x; xv[m][e + 1] = v.y; xv[m][e + 2] = v.z; xv[m][e + 3] = v.w;
          }
        } else {
#pragma unroll
          for (int e = 0; e < EPC; ++e) xv[m][e] = 0.0f;
        }
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float w[EPC];
        unpack16(wc[u][r], w);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[r][m] = fmaf(w[e], xv[m][e], acc[r][m]);
        }
      }
    }
  }
}

// ============================================================ k_rows_gemv
// out[t][o_off + j] (=|+=) sum_k W_j[k] x'[t][k], rows j from up to three sources.
template <typename TW, typename TX, int MT>
__global__ __launch_bounds__(kThreads) void k_rows_gemv(RowsArgs a) {
  constexpr int R = 4, U = 2;
  __shared__ __attribute__((aligned(16))) float xs[kSlabFloats];
  const int ks_max = kSlabFloats / MT;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
  const int row0 = (blockIdx.x * kWaves + wave) * R;
  const int t0 = blockIdx.y * MT;
  const int mt = min(MT, a.T - t0);
  if (mt <= 0) return;
  const TX* xrow[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) xrow[m] = reinterpret_cast<const TX*>(a.x) + (size_t)(t0 + min(m, mt - 1)) * a.ldx + a.x_off;
  const TW* rbase[R];
  bool rvalid[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    int j = row0 + r;
    rvalid[r] = j < ntot;
    int src = 0;
    if (j >= a.nrows[0]) { j -= a.nrows[0]; src = 1; if (j >= a.nrows[1]) { j -= a.nrows[1]; src = 2; } }
    rbase[r] = rvalid[r] ? reinterpret_cast<const TW*>(a.w[src]) + (size_t)j * a.K : nullptr;
  }
  float acc[R][MT];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
  for (int k0 = 0; k0 < a.K; k0 += ks_max) {
    const int ks = min(ks_max, a.K - k0);
    __syncthreads();
    stage_slab<TX, MT>(xs, ks_max, xrow, mt, k0, ks, a.relu_in != 0);
    __syncthreads();
    const TW* rows[R];
#pragma unroll
    for (int r = 0; r < R; ++r) rows[r] = rvalid[r] ? rbase[r] + k0 : nullptr;
    wave_dot_slab<TW, R, MT, U>(rows, rvalid, xs, ks_max, mt, ks / Elem<TW>::kPer16B, lane, acc);
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[r][m] = wave_sum(acc[r][m]);
  if (lane < R * MT) {
    const int r = lane % R, m = lane / R;
    float v = 0.0f;
#pragma unroll
    for (int rr = 0; rr < R; ++rr)
#pragma unroll
      for (int mm = 0; mm < MT; ++mm)
        if (rr == r && mm == m) v = acc[rr][mm];
    if (m < mt && rvalid[r]) {
      float* o = a.out + (size_t)(t0 + m) * a.ldo + a.o_off + row0 + r;
      *o = a.add ? *o + v : v;
    }
  }
}

// ============================================================ expert FFN
// Decode-shaped expert GEMVs.  No LDS and no block barrier: every lane holds the
// token vectors' 16-byte pieces for its own k positions in registers and issues
// all of its weight loads (RWxNCH rows x 16 B, about 16 per lane) before the
// first FMA, so each wave keeps ~16 KiB of weights in flight.  A block is four
// independent waves.  The grid is (row tile, job): every job -- a route
// position, or a piece of the shared expert's rows -- spans the same number of
// row tiles, and a block finds its job's fields with independent scalar loads
// from the kernel arguments, so its first weight load waits for one round trip
// only (a search over the jobs, or a byte-sized field read through the vector
// memory path, would chain several before any weight is requested).
constexpr int kBlockWaves = 4;

template <typename TW>
struct Job {
  const TW* W;
  int I, q0, q1, r0, r1;  // rows [r0, r1) of this job's piece
  int pos;                // route position, or kSharedJob
};

// Everything a block needs from the kernel arguments, read before any branch so
// the scalar loads issue together.
template <typename TW>
__device__ __forceinline__ Job<TW> job_of(const FfnArgs& a, int nrows, int by) {
  const FfnJob jd = a.jobs[by];
  Job<TW> jb;
  jb.pos = jd.pos;
  jb.W = reinterpret_cast<const TW*>(jd.w);
  jb.I = jd.I;
  jb.q0 = jd.q0;
  jb.q1 = jd.q1;
  jb.r0 = jd.r0;
  jb.r1 = min(jd.r0 + a.piece_rows, nrows < 0 ? jd.I : nrows);
  if (jd.w == nullptr) {
    // a route position resolved from the plan on the device (one round trip of
    // independent loads); positions that are not resident, or whose slot may
    // still be receiving copies, run no rows
    const int nh = a.npos[0];
    const int slot = a.order_slot[jd.pos];
    const int q0 = a.offsets[jd.pos], q1 = a.offsets[jd.pos + 1];
    const bool run = jd.pos < nh && slot >= 0 && slot < a.slots && !((a.busy_mask >> slot) & 1ull);
    jb.W = reinterpret_cast<const TW*>(a.cache + ((size_t)a.layer * a.slots + (run ? slot : 0)) * a.expert_bytes);
    jb.q0 = q0;
    jb.q1 = run ? q1 : q0;
    if (!run) jb.r1 = jb.r0;
  }
  return jb;
}

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Weights are streamed once per launch: non-temporal loads keep them from
// displacing the token vectors and activations in the caches (measured faster
// on gfx950 for the decode GEMVs).
template <typename TW>
__device__ __forceinline__ uint4 ld16_stream(const TW* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
template <typename TW>
__device__ __forceinline__ uint4 ld16(const TW* p) {
  return *reinterpret_cast<const uint4*>(p);
}

// acc[r][m] += <rows[r], xs[m]> over k; rows/xs point at element 0 of the row
// (xs at the token's vector).  nch = K / EPC chunks of 16 bytes.
template <typename TW, int R, int MT, int NCH>
__device__ __forceinline__ void wave_rows_dot(const TW* const (&rows)[R], const bool (&rv)[R],
                                              const TW* const (&xs)[MT], int mt, int nch, int lane,
                                              float (&acc)[R][MT]) {
  constexpr int EPC = Elem<TW>::kPer16B;
  for (int cb = 0; cb < nch; cb += kWave * NCH) {
    uint4 wr[R][NCH];
    uint4 xr[MT][NCH];
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = cb + lane + u * kWave;
#pragma unroll
      for (int r = 0; r < R; ++r) wr[r][u] = (c < nch && rv[r]) ? ld16_stream(rows[r] + (size_t)c * EPC) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int m = 0; m < MT; ++m) xr[m][u] = (c < nch && m < mt) ? ld16(xs[m] + (size_t)c * EPC) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      float xf[MT][EPC];
#pragma unroll
      for (int m = 0; m < MT; ++m) unpack16(xr[m][u], xf[m]);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        float wf[EPC];
        unpack16(wr[r][u], wf);
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
          for (int e = 0; e < EPC; ++e) acc[r][m] = fmaf(wf[e], xf[m][e], acc[r][m]);
      }
    }
  }
}

// pass 1: act[q][i] = q(silu(Wg[i] . x_t) * (Wu[i] . x_t)) for the wave's RW rows i
// (row tile bx of job by)
template <typename TW, int MT, int NCH, int RW>
__device__ __forceinline__ void ffn_gateup_body(const FfnArgs& a, int bx, int by) {
  constexpr int R = 2 * RW;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const Job<TW> jb = job_of<TW>(a, -1, by);
  const int H = a.hidden, I = jb.I, T = a.T, top_k = a.top_k;
  const int32_t* perm = a.perm;
  void* act_r = a.act;
  void* act_s = a.act_sh;
  const TW* xb = reinterpret_cast<const TW*>(a.x);
  // materialise every argument here, so all of their loads issue together
  asm volatile("" ::"s"(H), "s"(T), "s"(top_k), "s"(perm), "s"(act_r), "s"(act_s), "s"(xb), "s"(jb.W), "s"(jb.I),
               "s"(jb.q0), "s"(jb.q1), "s"(jb.r1), "s"(jb.pos));
  const bool shared = jb.pos == kSharedJob;
  TW* act = reinterpret_cast<TW*>(shared ? act_s : act_r);
  const int i0 = jb.r0 + (bx * kBlockWaves + wave) * RW;
  if (i0 >= jb.r1) return;
  const TW* rows[R];
  bool rv[R];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const bool v = i0 + r < jb.r1;
    rv[2 * r] = rv[2 * r + 1] = v;
    rows[2 * r] = jb.W + (size_t)(v ? i0 + r : 0) * H;          // gate row
    rows[2 * r + 1] = jb.W + (size_t)(v ? I + i0 + r : 0) * H;  // up row
  }
  for (int g = jb.q0; g < jb.q1; g += MT) {
    const int mt = min(MT, jb.q1 - g);
    const TW* xs[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int q = g + min(m, mt - 1);
      const int t = (shared || T == 1) ? (shared ? q : 0) : perm[q] / top_k;
      xs[m] = xb + (size_t)t * H;
    }
    float acc[R][MT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    wave_rows_dot<TW, R, MT, NCH>(rows, rv, xs, mt, H / Elem<TW>::kPer16B, lane, acc);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = wave_sum(acc[r][m]);
    if (lane < RW * MT) {
      const int r = lane % RW, m = lane / RW;
      float ga = 0.0f, ub = 0.0f;
#pragma unroll
      for (int rr = 0; rr < RW; ++rr)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          if (rr == r && mm == m) { ga = acc[2 * rr][mm]; ub = acc[2 * rr + 1][mm]; }
      if (m < mt && i0 + r < jb.r1) Elem<TW>::store(act, (g + m) * I + i0 + r, silu(ga) * ub);
    }
  }
}

template <typename TW, int MT, int NCH, int RW>
__global__ __launch_bounds__(kThreads) void k_ffn_gateup(FfnArgs a) {
  ffn_gateup_body<TW, MT, NCH, RW>(a, blockIdx.x, blockIdx.y);
}

// The resident gate/up launch of a batch-1 route whose plan the host does not
// wait for, carrying that route's prediction: blocks [0, pred_blocks) run the
// predictor's second layer, top-k and spec plan as k_predict_plan's blocks do
// (dispatched first, beside the GEMV's row tiles), the rest are the row tiles
// of k_ffn_gateup<bf16, 1, NCH, 1>, numbered row tile fastest.  The
// prediction then no longer lengthens the chain of dependent launches.
template <int NCH>
__global__ __launch_bounds__(kThreads) void k_ffn_gateup_pred(FfnArgs a, PredictPlanArgs p, int tiles_x) {
  __shared__ PredictLds<1> L;
  const int nblk = pred_blocks(p.plan.E, p.Ph);
  const int b = blockIdx.x;
  if (b < nblk) {
    predict_plan_body<1>(p, L, b);
    return;
  }
  const int g = b - nblk;
  ffn_gateup_body<bf16_t, 1, NCH, 1>(a, g % tiles_x, g / tiles_x);
}

// pass 2: Y[pair][n] = Wd[n] . act[q] for the wave's RW rows n
template <typename TW, int MT, int NCH, int RW>
__global__ __launch_bounds__(kThreads) void k_ffn_down(FfnArgs a) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const Job<TW> jb = job_of<TW>(a, a.hidden, blockIdx.y);
  const int H = a.hidden, I = jb.I;
  const void* act_r = a.act;
  const void* act_s = a.act_sh;
  float* y_r = a.Y;
  float* y_s = a.Ysh;
  const int32_t* perm = a.perm;
  // materialise every argument here, so all of their loads issue together
  asm volatile("" ::"s"(H), "s"(act_r), "s"(act_s), "s"(y_r), "s"(y_s), "s"(perm), "s"(jb.W), "s"(jb.I), "s"(jb.q0),
               "s"(jb.q1), "s"(jb.r1), "s"(jb.pos));
  const bool shared = jb.pos == kSharedJob;
  const TW* actb = reinterpret_cast<const TW*>(shared ? act_s : act_r);
  float* Yb = shared ? y_s : y_r;
  const int n0 = jb.r0 + (blockIdx.x * kBlockWaves + wave) * RW;
  if (n0 >= jb.r1) return;
  const TW* Wd = jb.W + (size_t)2 * I * H;
  const TW* rows[RW];
  bool rv[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    rv[r] = n0 + r < jb.r1;
    rows[r] = Wd + (size_t)(rv[r] ? n0 + r : 0) * I;
  }
  for (int g = jb.q0; g < jb.q1; g += MT) {
    const int mt = min(MT, jb.q1 - g);
    const TW* xs[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) xs[m] = actb + (size_t)(g + min(m, mt - 1)) * I;
    float acc[RW][MT];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    wave_rows_dot<TW, RW, MT, NCH>(rows, rv, xs, mt, I / Elem<TW>::kPer16B, lane, acc);
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = wave_sum(acc[r][m]);
    if (lane < RW * MT) {
      const int r = lane % RW, m = lane / RW;
      float v = 0.0f;
#pragma unroll
      for (int rr = 0; rr < RW; ++rr)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          if (rr == r && mm == m) v = acc[rr][mm];
      if (m < mt && rv[r]) {
        const int q = g + m;
        float* Y = Yb + (size_t)(shared ? q : perm[q]) * H;
        Y[n0 + r] = v;
      }
    }
  }
}

// ============================================================ 4-bit experts
// Dequantising GEMVs for experts stored as 4-bit codes: a matrix of R rows and
// reduction length K is R x K/2 bytes of codes (two per byte, even k in the low
// nibble) followed by R x K/128 bf16 scales; weight (r, k) = (code - 8) *
// scale[r][k / 128].  A lane takes 16-byte pieces of a row (32 weights, a
// quarter of a scale group); per piece and token it forms sum((128 + code) x)
// and sum(x) with bf16 dot2 instructions (128 + code is exact in bf16) and adds
// scale * (sum((128 + code) x) - 136 sum(x)) to the row's accumulator.

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

// c + a.lo * b.lo + a.hi * b.hi over two bf16 pairs packed in 32-bit words.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}

struct Q4Row {
  const uint8_t* codes;  // row start in the code block
  const bf16_t* scales;  // row start in the scale block
};

__device__ __forceinline__ Q4Row q4_row(const uint8_t* mat, int rows, int K, int r) {
  Q4Row q;
  q.codes = mat + (size_t)r * (K / 2);
  q.scales = reinterpret_cast<const bf16_t*>(mat + (size_t)rows * (K / 2)) + (size_t)r * (K / kInt4Group);
  return q;
}

// acc[r][m] += <row r, xs[m]> over K for R rows of one matrix; each lane has
// NCH pieces of every row (and the matching token pieces) in flight at once.
template <int R, int MT, int NCH>
__device__ __forceinline__ void wave_rows_dot_q4(const Q4Row (&rows)[R], const bool (&rv)[R],
                                                 const bf16_t* const (&xs)[MT], int mt, int K, int lane,
                                                 float (&acc)[R][MT]) {
  const int np = K / 32;  // 16-byte pieces per row
  for (int cb = 0; cb < np; cb += kWave * NCH) {
    uint4 wq[R][NCH];
    float scq[R][NCH];
    uint4 xq[MT][NCH][4];
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = cb + lane + u * kWave;
      const bool in = c < np;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        // a piece past the row, or of a row past the job: code 8 (weight 0), scale 0
        wq[r][u] = (in && rv[r]) ? ld16_stream(rows[r].codes + (size_t)c * 16)
                                 : make_uint4(0x88888888u, 0x88888888u, 0x88888888u, 0x88888888u);
        scq[r][u] = (in && rv[r]) ? bf16_to_f32(rows[r].scales[c / 4]) : 0.0f;
      }
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        const uint4* xp = reinterpret_cast<const uint4*>(xs[m] + (size_t)c * 32);
#pragma unroll
        for (int v = 0; v < 4; ++v) xq[m][u][v] = (in && m < mt) ? xp[v] : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      // token pieces: 32 bf16 = 16 words; word j holds elements 2j (low half)
      // and 2j+1; sum(x) by dot2 against (1, 1)
      uint32_t xw[MT][16];
      float sx[MT];
#pragma unroll
      for (int m = 0; m < MT; ++m) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const uint4 q = xq[m][u][v];
          xw[m][4 * v] = q.x; xw[m][4 * v + 1] = q.y; xw[m][4 * v + 2] = q.z; xw[m][4 * v + 3] = q.w;
        }
        float s = 0.0f;
#pragma unroll
        for (int j = 0; j < 16; ++j) s = dot2_bf16(0x3F803F80u, xw[m][j], s);
        sx[m] = s;
      }
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint4 wr = wq[r][u];
        const uint32_t ww[4] = {wr.x, wr.y, wr.z, wr.w};
        float t[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) t[m] = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          // byte b of a code word holds elements 2b (low nibble) and 2b+1: the
          // bf16 pair (128 + lo, 128 + hi), exact (0x4300 is 128, the mantissa
          // step there is 1)
          const uint32_t cw = ww[i];
          const uint32_t pr[4] = {0x43004300u | (cw & 0xFu) | ((cw & 0xF0u) << 12),
                                  0x43004300u | ((cw >> 8) & 0xFu) | ((cw & 0xF000u) << 4),
                                  0x43004300u | ((cw >> 16) & 0xFu) | ((cw >> 4) & 0xF0000u),
                                  0x43004300u | ((cw >> 24) & 0xFu) | ((cw >> 12) & 0xF0000u)};
#pragma unroll
          for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int b = 0; b < 4; ++b) t[m] = dot2_bf16(pr[b], xw[m][4 * i + b], t[m]);
        }
        // sum((128 + code) x) - 136 sum(x) = sum((code - 8) x)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[r][m] = fmaf(scq[r][u], t[m] - 136.0f * sx[m], acc[r][m]);
      }
    }
  }
}

// pass 1, 4-bit experts: act[q][i] for the wave's RW rows i (gate rows, up rows)
template <int MT, int RW, int NCH>
__global__ __launch_bounds__(kThreads) void k_ffn_gateup_q4(FfnArgs a) {
  constexpr int R = 2 * RW;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const Job<bf16_t> jb = job_of<bf16_t>(a, -1, blockIdx.y);
  const int H = a.hidden, I = jb.I, T = a.T, top_k = a.top_k;
  const int32_t* perm = a.perm;
  bf16_t* act = reinterpret_cast<bf16_t*>(a.act);
  const bf16_t* xb = reinterpret_cast<const bf16_t*>(a.x);
  // materialise every argument here, so all of their loads issue together
  asm volatile("" ::"s"(H), "s"(T), "s"(top_k), "s"(perm), "s"(act), "s"(xb), "s"(jb.W), "s"(jb.I), "s"(jb.q0),
               "s"(jb.q1), "s"(jb.r1));
  const int i0 = jb.r0 + (blockIdx.x * kBlockWaves + wave) * RW;
  if (i0 >= jb.r1) return;
  const uint8_t* base = reinterpret_cast<const uint8_t*>(jb.W);
  const size_t mat = (size_t)I * H / 2 + (size_t)I * (H / kInt4Group) * 2;
  Q4Row rows[R];
  bool rv[R];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const bool v = i0 + r < jb.r1;
    rv[2 * r] = rv[2 * r + 1] = v;
    rows[2 * r] = q4_row(base, I, H, v ? i0 + r : 0);            // gate row
    rows[2 * r + 1] = q4_row(base + mat, I, H, v ? i0 + r : 0);  // up row
  }
  for (int g = jb.q0; g < jb.q1; g += MT) {
    const int mt = min(MT, jb.q1 - g);
    const bf16_t* xs[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int q = g + min(m, mt - 1);
      const int t = T == 1 ? 0 : perm[q] / top_k;
      xs[m] = xb + (size_t)t * H;
    }
    float acc[R][MT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    wave_rows_dot_q4<R, MT, NCH>(rows, rv, xs, mt, H, lane, acc);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = wave_sum(acc[r][m]);
    if (lane < RW * MT) {
      const int r = lane % RW, m = lane / RW;
      float ga = 0.0f, ub = 0.0f;
#pragma unroll
      for (int rr = 0; rr < RW; ++rr)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          if (rr == r && mm == m) { ga = acc[2 * rr][mm]; ub = acc[2 * rr + 1][mm]; }
      if (m < mt && i0 + r < jb.r1) Elem<bf16_t>::store(act, (g + m) * I + i0 + r, silu(ga) * ub);
    }
  }
}

// pass 2, 4-bit experts: Y[pair][n] = Wd[n] . act[q] for the wave's RW rows n
template <int MT, int RW, int NCH>
__global__ __launch_bounds__(kThreads) void k_ffn_down_q4(FfnArgs a) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const Job<bf16_t> jb = job_of<bf16_t>(a, a.hidden, blockIdx.y);
  const int H = a.hidden, I = jb.I;
  const bf16_t* actb = reinterpret_cast<const bf16_t*>(a.act);
  float* Y = a.Y;
  const int32_t* perm = a.perm;
  // materialise every argument here, so all of their loads issue together
  asm volatile("" ::"s"(H), "s"(actb), "s"(Y), "s"(perm), "s"(jb.W), "s"(jb.I), "s"(jb.q0), "s"(jb.q1), "s"(jb.r1));
  const int n0 = jb.r0 + (blockIdx.x * kBlockWaves + wave) * RW;
  if (n0 >= jb.r1) return;
  const uint8_t* base = reinterpret_cast<const uint8_t*>(jb.W);
  const size_t mat = (size_t)I * H / 2 + (size_t)I * (H / kInt4Group) * 2;
  Q4Row rows[RW];
  bool rv[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    rv[r] = n0 + r < jb.r1;
    rows[r] = q4_row(base + 2 * mat, H, I, rv[r] ? n0 + r : 0);
  }
  for (int g = jb.q0; g < jb.q1; g += MT) {
    const int mt = min(MT, jb.q1 - g);
    const bf16_t* xs[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) xs[m] = actb + (size_t)(g + min(m, mt - 1)) * I;
    float acc[RW][MT];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    wave_rows_dot_q4<RW, MT, NCH>(rows, rv, xs, mt, I, lane, acc);
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = wave_sum(acc[r][m]);
    if (lane < RW * MT) {
      const int r = lane % RW, m = lane / RW;
      float v = 0.0f;
#pragma unroll
      for (int rr = 0; rr < RW; ++rr)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          if (rr == r && mm == m) v = acc[rr][mm];
      if (m < mt && rv[r]) Y[(size_t)perm[g + m] * H + n0 + r] = v;
    }
  }
}

// Dequantise whole experts for the MFMA GEMM: block (r, e) expands weight row r
// of expert e (gate rows, then up rows, then down rows); each thread turns 8
// weights (4 code bytes, low nibble first) into one 16-byte store of bf16, so
// a wave writes 1 KB contiguously.
__global__ __launch_bounds__(kThreads) void k_dequant_q4(DequantArgs a) {
  const int I = a.inter, H = a.hidden;
  int r = blockIdx.x, mtx = 0;
  if (r >= I) { r -= I; mtx = 1; }
  if (mtx == 1 && r >= I) { r -= I; mtx = 2; }
  const int K = mtx < 2 ? H : I, R = mtx < 2 ? I : H;
  const uint8_t* mat = a.src[blockIdx.y] + (size_t)mtx * ((size_t)I * H / 2 + (size_t)I * (H / kInt4Group) * 2);
  const Q4Row q = q4_row(mat, R, K, r);
  uint4* dst = reinterpret_cast<uint4*>(a.dst + (size_t)blockIdx.y * 3 * I * H + (size_t)mtx * I * H + (size_t)r * K);
  for (int c = threadIdx.x; c < K / 8; c += kThreads) {  // 8-weight chunks of the row
    const uint32_t w = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(q.codes) + c);
    const float sc = bf16_to_f32(q.scales[c / (kInt4Group / 8)]);
    uint32_t out[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const float e0 = ((float)((w >> (8 * b)) & 0xFu) - 8.0f) * sc;
      const float e1 = ((float)((w >> (8 * b + 4)) & 0xFu) - 8.0f) * sc;
      out[b] = (uint32_t)f32_to_bf16(e0) | ((uint32_t)f32_to_bf16(e1) << 16);
    }
    dst[c] = make_uint4(out[0], out[1], out[2], out[3]);
  }
}

void launch_dequant_q4(const DequantArgs& a, hipStream_t s) {
  k_dequant_q4<<<dim3(2 * a.inter + a.hidden, a.n), kThreads, 0, s>>>(a);  // one block per weight row
}

// ============================================================ combine
// y[t][n] = sum_r w[t][r] Y[t][r][n] + s[t] sum_k Ysh[k][t][n], r and k in
// order, one rounding.  Every operand of the element is loaded before the
// first product (up to kMaxK ranks and 8 split-K slices), so the kernel waits
// for one memory round trip instead of one per term.
constexpr int kSplitRegs = 8;
// The combine's arithmetic over operands already loaded: y = sum_r w[r] Y[r]
// (r < top_k, in order), then, with a shared expert, y += s * ysh where ysh
// sums the slices sv[k < min(split, kSplitRegs)] in order and `more` adds any
// later slices.  Every combine goes through here, so all of them round alike.
template <typename More>
__device__ __forceinline__ float combine_terms(const float (&wv)[kMaxK], const float (&yv)[kMaxK], int top_k,
                                               bool has_sh, const float (&sv)[kSplitRegs], int split, float s,
                                               More more) {
  float y = 0.0f;
#pragma unroll
  for (int r = 0; r < kMaxK; ++r)
    if (r < top_k) y += wv[r] * yv[r];
  if (has_sh) {
    float ysh = 0.0f;
#pragma unroll
    for (int k = 0; k < kSplitRegs; ++k)
      if (k < split) ysh += sv[k];
    ysh = more(ysh);
    y += s * ysh;
  }
  return y;
}

__device__ __forceinline__ float combine_value(const CombineArgs& a, int t, int n) {
  float wv[kMaxK], yv[kMaxK], sv[kSplitRegs];
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    const bool in = r < a.top_k;
    wv[r] = in ? a.w[t * a.top_k + r] : 0.0f;
    yv[r] = in ? a.Y[((size_t)t * a.top_k + r) * a.hidden + n] : 0.0f;
  }
  const int split = a.Ysh ? a.ysh_split : 0;
#pragma unroll
  for (int k = 0; k < kSplitRegs; ++k)
    sv[k] = k < split ? a.Ysh[(size_t)k * a.ysh_split_stride + (size_t)t * a.hidden + n] : 0.0f;
  const float s = a.Ysh && a.sscale ? a.sscale[t] : 1.0f;
  return combine_terms(wv, yv, a.top_k, a.Ysh != nullptr, sv, split, s, [&](float ysh) {
    for (int k = kSplitRegs; k < split; ++k) ysh += a.Ysh[(size_t)k * a.ysh_split_stride + (size_t)t * a.hidden + n];
    return ysh;
  });
}

template <typename TY>
__global__ __launch_bounds__(kThreads) void k_combine(CombineArgs a) {
  const int t = blockIdx.y;
  const int n = blockIdx.x * kThreads + threadIdx.x;
  if (n >= a.hidden) return;
  Elem<TY>::store(reinterpret_cast<TY*>(a.y), t * a.hidden + n, combine_value(a, t, n));
}

// Combine and residual add in one launch (the layer loop's combine -> h += y):
// y as k_combine rounds it, h += y as k_residual_add adds it.
template <typename TY>
__global__ __launch_bounds__(kThreads) void k_combine_residual(CombineArgs a, float* h) {
  const int t = blockIdx.y;
  const int n = blockIdx.x * kThreads + threadIdx.x;
  if (n >= a.hidden) return;
  const float y = combine_value(a, t, n);
  Elem<TY>::store(reinterpret_cast<TY*>(a.y), t * a.hidden + n, y);
  h[(size_t)t * a.hidden + n] += Elem<TY>::quant(y);
}

// ============================================================ decode rows GEMV
// Token groups of up to four with weights and tokens of one type: the FFN
// GEMVs' scheme instead of the LDS slab -- one row per wave, each lane holding
// its 16-byte pieces of the token vectors in registers and issuing all of its
// weight loads before the first FMA, so a launch is one memory round trip
// deep (the slab kernel waits for the tokens to reach LDS first, and its four
// rows per wave leave most CUs idle on a 2048-row matrix).
template <typename TW, int MT, int NCH>
__global__ __launch_bounds__(kThreads) void k_rows_gemv_reg(RowsArgs a) {
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
  const int row = blockIdx.x * kWaves + wave;
  const int t0 = blockIdx.y * MT;
  const int mt = min(MT, a.T - t0);
  if (mt <= 0 || row >= ntot) return;
  const TW* xs[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) xs[m] = reinterpret_cast<const TW*>(a.x) + (size_t)(t0 + min(m, mt - 1)) * a.ldx + a.x_off;
  int j = row, src = 0;
  if (j >= a.nrows[0]) { j -= a.nrows[0]; src = 1; if (j >= a.nrows[1]) { j -= a.nrows[1]; src = 2; } }
  const TW* const rows[1] = {reinterpret_cast<const TW*>(a.w[src]) + (size_t)j * a.K};
  const bool rv[1] = {true};
  float acc[1][MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[0][m] = 0.0f;
  wave_rows_dot<TW, 1, MT, NCH>(rows, rv, xs, mt, a.K / Elem<TW>::kPer16B, lane, acc);
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[0][m] = wave_sum(acc[0][m]);
  if (lane < MT) {
    float v = 0.0f;
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (m == lane) v = acc[0][m];
    if (lane < mt) {
      float* o = a.out + (size_t)(t0 + lane) * a.ldo + a.o_off + row;
      *o = a.add ? *o + v : v;
    }
  }
}

// ============================================================ batch-1 rows GEMV over q(rms(h))
// The RMSNorm that feeds a batch-1 rows GEMV folded into it.  Each block forms
// x = q(rms(h)) once, as k_rmsnorm_quant_reg does (thread t sums the squares of
// its VPT pieces t + 256 u in order, the waves' sums -- lane 0's -- are added in
// order, each thread stores its pieces of x rounded to bf16), but into LDS; its
// waves then take their x pieces from there and form the dot in
// k_rows_gemv_reg's order (pieces lane + 64 u, u ascending).  The result is bit
// for bit the two kernels', with one launch and one dependent kernel fewer; the
// weight loads are issued first and overlap the norm.  add_src: out = add_src
// + dot (a second residual buffer, so no block reads a row of h that another
// has already updated); x_out: block 0 also stores x.
//
// CMB: h is the residual before the previous layer's MoE output is added; each
// block first forms that output y = combine(ca) and h' = h + q(y) for the
// whole token, as k_combine_residual would (same operands, same arithmetic),
// then works on h' as above, with out = h' + dot; block 0 stores y to ca.y.
// The combine launch and its dependent-launch gap are gone; h' itself is
// never written (only out, which is h' plus the GEMV).
template <int VPT, int NCH, bool CMB>
__global__ __launch_bounds__(kThreads) void k_rows_gemv_norm(RowsArgs a, const float* h, float eps,
                                                             const float* add_src, bf16_t* x_out, CombineArgs ca) {
  __shared__ __attribute__((aligned(16))) bf16_t xs[4 * VPT * kThreads];
  __shared__ __attribute__((aligned(16))) float hs[CMB ? 4 * VPT * kThreads : 4];
  __shared__ float red[kWaves];
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
  const int row = blockIdx.x * kWaves + wave;
  const bool has_row = row < ntot;
  const int H = a.K, nch = H / 8, n4 = H / 4;
  uint4 wr[NCH];
  if (has_row) {
    int j = row, src = 0;
    if (j >= a.nrows[0]) { j -= a.nrows[0]; src = 1; if (j >= a.nrows[1]) { j -= a.nrows[1]; src = 2; } }
    const bf16_t* wrow = reinterpret_cast<const bf16_t*>(a.w[src]) + (size_t)j * H;
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = lane + u * kWave;
      wr[u] = c < nch ? ld16_stream(wrow + (size_t)c * 8) : make_uint4(0, 0, 0, 0);
    }
  }
  const float4* h4 = reinterpret_cast<const float4*>(h);
  float4 r[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int i = tid + u * kThreads;
    r[u] = i < n4 ? h4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  if constexpr (CMB) {
    // batch 1: Y rows r * H, one shared slice (the launcher checks both)
    const bool has_sh = ca.Ysh != nullptr;
    float wv[kMaxK];
#pragma unroll
    for (int k = 0; k < kMaxK; ++k) wv[k] = k < ca.top_k ? ca.w[k] : 0.0f;
    const float sc = has_sh && ca.sscale ? ca.sscale[0] : 1.0f;
    float4 yq[VPT][kMaxK], sq4[VPT];
    const float4* Y4 = reinterpret_cast<const float4*>(ca.Y);
    const float4* S4 = reinterpret_cast<const float4*>(ca.Ysh);
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int i = tid + u * kThreads;
#pragma unroll
      for (int k = 0; k < kMaxK; ++k)
        yq[u][k] = i < n4 && k < ca.top_k ? Y4[(size_t)k * n4 + i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      sq4[u] = i < n4 && has_sh ? S4[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int i = tid + u * kThreads;
      if (i >= n4) continue;
      float hv[4] = {r[u].x, r[u].y, r[u].z, r[u].w};
      bf16_t yb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float yv[kMaxK], sv[kSplitRegs];
#pragma unroll
        for (int k = 0; k < kMaxK; ++k) yv[k] = c == 0 ? yq[u][k].x : c == 1 ? yq[u][k].y : c == 2 ? yq[u][k].z : yq[u][k].w;
        sv[0] = c == 0 ? sq4[u].x : c == 1 ? sq4[u].y : c == 2 ? sq4[u].z : sq4[u].w;
#pragma unroll
        for (int k = 1; k < kSplitRegs; ++k) sv[k] = 0.0f;
        const float y = combine_terms(wv, yv, ca.top_k, has_sh, sv, 1, sc, [](float v) { return v; });
        yb[c] = f32_to_bf16(y);
        hv[c] += Elem<bf16_t>::quant(y);
      }
      r[u] = make_float4(hv[0], hv[1], hv[2], hv[3]);
      *reinterpret_cast<float4*>(&hs[4 * i]) = r[u];
      if (blockIdx.x == 0)
        *reinterpret_cast<uint2*>(static_cast<bf16_t*>(ca.y) + 4 * (size_t)i) =
            make_uint2((uint32_t)yb[0] | ((uint32_t)yb[1] << 16), (uint32_t)yb[2] | ((uint32_t)yb[3] << 16));
    }
  }
  float sq = 0.0f;
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    sq = fmaf(r[u].x, r[u].x, sq);
    sq = fmaf(r[u].y, r[u].y, sq);
    sq = fmaf(r[u].z, r[u].z, sq);
    sq = fmaf(r[u].w, r[u].w, sq);
  }
  sq = wave_sum(sq);
  if (lane == 0) red[wave] = sq;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int i = tid + u * kThreads;
    if (i < n4) {
      const bf16_t q0 = f32_to_bf16(r[u].x * inv), q1 = f32_to_bf16(r[u].y * inv);
      const bf16_t q2 = f32_to_bf16(r[u].z * inv), q3 = f32_to_bf16(r[u].w * inv);
      const uint2 q = make_uint2((uint32_t)q0 | ((uint32_t)q1 << 16), (uint32_t)q2 | ((uint32_t)q3 << 16));
      *reinterpret_cast<uint2*>(&xs[4 * i]) = q;
      if (x_out && blockIdx.x == 0) *reinterpret_cast<uint2*>(x_out + 4 * (size_t)i) = q;
    }
  }
  __syncthreads();
  if (!has_row) return;
  float acc = 0.0f;
#pragma unroll
  for (int u = 0; u < NCH; ++u) {
    const int c = lane + u * kWave;
    float xf[8], wf[8];
    const uint4 xq = c < nch ? *reinterpret_cast<const uint4*>(&xs[8 * c]) : make_uint4(0, 0, 0, 0);
    unpack16(xq, xf);
    unpack16(wr[u], wf);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(wf[e], xf[e], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) {
    float* o = a.out + a.o_off + row;
    if constexpr (CMB) *o = hs[row] + acc;
    else *o = add_src ? add_src[row] + acc : acc;
  }
}

// ============================================================ harness ops
// RMSNorm of one token per block with the row held in registers: each thread
// loads its VPT 16-byte pieces at once (one memory round trip, where a strided
// loop waits for every element in turn), sums their squares in piece order,
// and the waves reduce in a fixed order.  H % 4 == 0, H <= 4 * VPT * kThreads.
template <typename TQ, int VPT>
__global__ __launch_bounds__(kThreads) void k_rmsnorm_quant_reg(const float* h, void* out, int H, float eps) {
  const int t = blockIdx.x;
  const float4* v = reinterpret_cast<const float4*>(h + (size_t)t * H);
  const int n4 = H / 4;
  __shared__ float red[kWaves];
  float4 r[VPT];
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int i = threadIdx.x + u * kThreads;
    r[u] = i < n4 ? v[i] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  }
  float s = 0.0f;
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    s = fmaf(r[u].x, r[u].x, s);
    s = fmaf(r[u].y, r[u].y, s);
    s = fmaf(r[u].z, r[u].z, s);
    s = fmaf(r[u].w, r[u].w, s);
  }
  s = wave_sum(s);
  if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = s;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  TQ* o = reinterpret_cast<TQ*>(out) + (size_t)t * H;
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int i = threadIdx.x + u * kThreads;
    if (i >= n4) continue;
    Elem<TQ>::store(o, 4 * i, r[u].x * inv);
    Elem<TQ>::store(o, 4 * i + 1, r[u].y * inv);
    Elem<TQ>::store(o, 4 * i + 2, r[u].z * inv);
    Elem<TQ>::store(o, 4 * i + 3, r[u].w * inv);
  }
}

template <typename TQ>
__global__ __launch_bounds__(kThreads) void k_rmsnorm_quant(const float* h, void* out, int H, float eps) {
  const int t = blockIdx.x;
  const float* v = h + (size_t)t * H;
  __shared__ float red[kWaves];
  float s = 0.0f;
  for (int i = threadIdx.x; i < H; i += kThreads) s += v[i] * v[i];
  s = wave_sum(s);
  if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = s;
  __syncthreads();
  float tot = 0.0f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) tot += red[w];
  const float inv = 1.0f / sqrtf(tot / (float)H + eps);
  for (int i = threadIdx.x; i < H; i += kThreads) Elem<TQ>::store(reinterpret_cast<TQ*>(out), t * H + i, v[i] * inv);
}

template <typename TY>
__global__ __launch_bounds__(kThreads) void k_residual_add(float* h, const void* y, int n) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < n) h[i] += Elem<TY>::load(reinterpret_cast<const TY*>(y), i);
}

// ============================================================ launchers
template <typename TW, int MT>
static void rows_reg_launch(const RowsArgs& a, int ntot, hipStream_t s) {
  const dim3 grid((ntot + kWaves - 1) / kWaves, (a.T + MT - 1) / MT);
  const int pieces = a.K / Elem<TW>::kPer16B;
  if (pieces <= kWave) k_rows_gemv_reg<TW, MT, 1><<<grid, kThreads, 0, s>>>(a);
  else if (pieces <= 2 * kWave) k_rows_gemv_reg<TW, MT, 2><<<grid, kThreads, 0, s>>>(a);
  else k_rows_gemv_reg<TW, MT, 4><<<grid, kThreads, 0, s>>>(a);
}

template <typename TW, typename TX>
static void rows_dispatch(const RowsArgs& a, hipStream_t s) {
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
  if constexpr (std::is_same<TW, TX>::value) {
    // decode-sized groups over 16-byte aligned rows and tokens: registers, no LDS
    constexpr int EPC = Elem<TW>::kPer16B;
    bool aligned = a.K % EPC == 0 && a.ldx % EPC == 0 && a.x_off % EPC == 0 &&
                   reinterpret_cast<uintptr_t>(a.x) % 16 == 0;
    for (int i = 0; i < 3; ++i)
      if (a.nrows[i] > 0) aligned = aligned && reinterpret_cast<uintptr_t>(a.w[i]) % 16 == 0;
    if (aligned && a.relu_in == 0 && a.T <= 4 && ntot > 0) {
      if (a.T >= 4) rows_reg_launch<TW, 4>(a, ntot, s);
      else if (a.T >= 2) rows_reg_launch<TW, 2>(a, ntot, s);
      else rows_reg_launch<TW, 1>(a, ntot, s);
      return;
    }
  }
  const int rows_per_block = kWaves * 4;
  const int mt = a.T >= 4 ? 4 : (a.T >= 2 ? 2 : 1);
  dim3 grid((ntot + rows_per_block - 1) / rows_per_block, (a.T + mt - 1) / mt);
  if (mt == 4) k_rows_gemv<TW, TX, 4><<<grid, kThreads, 0, s>>>(a);
  else if (mt == 2) k_rows_gemv<TW, TX, 2><<<grid, kThreads, 0, s>>>(a);
  else k_rows_gemv<TW, TX, 1><<<grid, kThreads, 0, s>>>(a);
}

void launch_rows_gemv(const RowsArgs& a, int wdtype, int xdtype, hipStream_t s) {
  if (wdtype == 1 && xdtype == 1) rows_dispatch<bf16_t, bf16_t>(a, s);
  else if (wdtype == 1 && xdtype == 0) rows_dispatch<bf16_t, float>(a, s);
  else rows_dispatch<float, float>(a, s);
}

// (MT, NCH) pairs keep the registers per lane bounded: MT x NCH x 16 B of token
// pieces plus R x NCH x 16 B of weights in flight.
// Every job of a GEMV launch covers `piece_rows` rows: in pass 1 all H output
// rows; in pass 0 the routed expert's I rows, the shared expert being split into
// as many pieces of that size as the job table allows.
static int gemv_jobs(const FfnArgs& in, int pass, FfnArgs& a) {
  a = in;
  if (pass == 1) {
    for (int j = 0; j < a.n_jobs; ++j) a.jobs[j].r0 = 0;
    a.piece_rows = a.hidden;
    return a.n_jobs;
  }
  int n_routed = 0;
  for (int j = 0; j < in.n_jobs; ++j) n_routed += in.jobs[j].pos != kSharedJob;
  const bool has_shared = n_routed < in.n_jobs;
  int P = n_routed ? in.inter : in.shared_inter;
  int pieces = has_shared ? (in.shared_inter + P - 1) / P : 0;
  if (pieces > kMaxJobs - n_routed) {
    pieces = kMaxJobs - n_routed;
    P = (in.shared_inter + pieces - 1) / pieces;
  }
  int n = 0;
  for (int j = 0; j < in.n_jobs; ++j) {
    const int np = in.jobs[j].pos == kSharedJob ? pieces : 1;
    for (int p = 0; p < np; ++p, ++n) {
      a.jobs[n] = in.jobs[j];
      a.jobs[n].r0 = p * P;
    }
  }
  a.n_jobs = n;
  a.piece_rows = P;
  return n;
}

// 4-bit experts (routed jobs only): rows per wave shrink as the token group grows,
// keeping registers bounded (token pieces MT x 16 words, accumulators R x MT).
// NCH pieces in flight per lane and row.  One: with more, the registers they
// take lower the waves per SIMD, and the one-token launches measured slower
// (Mixtral-8x7B int4 gate/up 30 us at 4 pieces against 23 us at one).
template <int MT, int NCH>
static void ffn_launch_q4(const FfnArgs& a, int pass, const dim3& grid, hipStream_t s, hipEvent_t ev0,
                          hipEvent_t ev1) {
  constexpr int RWG = MT <= 2 ? 2 : (MT == 4 ? 2 : 1), RWD = 2 * RWG;
  if (pass == 0) hipExtLaunchKernelGGL((k_ffn_gateup_q4<MT, RWG, NCH>), grid, dim3(kThreads), 0, s, ev0, ev1, 0, a);
  else hipExtLaunchKernelGGL((k_ffn_down_q4<MT, RWD, NCH>), grid, dim3(kThreads), 0, s, ev0, ev1, 0, a);
}

template <int MT>
static void ffn_dispatch_q4(const FfnArgs& in, int pass, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  constexpr int RWG = MT <= 2 ? 2 : (MT == 4 ? 2 : 1), RWD = 2 * RWG;
  const int rows_per_block = kBlockWaves * (pass == 0 ? RWG : RWD);
  FfnArgs a;
  if (gemv_jobs(in, pass, a) == 0 || a.piece_rows <= 0) return;
  const dim3 grid((a.piece_rows + rows_per_block - 1) / rows_per_block, a.n_jobs);
  ffn_launch_q4<MT, 1>(a, pass, grid, s, ev0, ev1);
}

// One launch of pass `pass` with NCH 16-byte chunks per lane and row in flight.
template <typename TW, int MT, int NCH>
static void ffn_launch_nch(const FfnArgs& a, int pass, const dim3& grid, hipStream_t s, hipEvent_t ev0,
                           hipEvent_t ev1) {
  constexpr int RWG = 1, RWD = 2;
  if (ev0) {
    if (pass == 0) hipExtLaunchKernelGGL(k_ffn_gateup<TW, MT, NCH, RWG>, grid, dim3(kThreads), 0, s, ev0, ev1, 0, a);
    else hipExtLaunchKernelGGL(k_ffn_down<TW, MT, NCH, RWD>, grid, dim3(kThreads), 0, s, ev0, ev1, 0, a);
  } else if (pass == 0) {
    k_ffn_gateup<TW, MT, NCH, RWG><<<grid, kThreads, 0, s>>>(a);
  } else {
    k_ffn_down<TW, MT, NCH, RWD><<<grid, kThreads, 0, s>>>(a);
  }
}

template <typename TW, int MT>
static void ffn_dispatch(const FfnArgs& in, int pass, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  constexpr int RWG = 1, RWD = 2;
  const int rows_per_block = kBlockWaves * (pass == 0 ? RWG : RWD);
  FfnArgs a;
  if (gemv_jobs(in, pass, a) == 0 || a.piece_rows <= 0) return;
  const dim3 grid((a.piece_rows + rows_per_block - 1) / rows_per_block, a.n_jobs);
  if constexpr (MT == 1) {
    // Single-token rows: as many chunks per lane as cover the row in one round
    // when that is at most 4 (a 1408-wide down row is 176 chunks: 3 per lane
    // leaves 16 lanes idle where 4 leave 80, measured 10.9 -> 9.5 us for 46 MB).
    // The lane -> chunk map of one round does not depend on NCH, so the sums
    // are the same bit for bit.
    const int K = pass == 0 ? a.hidden : a.inter;
    const int per_lane = (K / Elem<TW>::kPer16B + kWave - 1) / kWave;
    if (per_lane <= 1) ffn_launch_nch<TW, MT, 1>(a, pass, grid, s, ev0, ev1);
    else if (per_lane == 2) ffn_launch_nch<TW, MT, 2>(a, pass, grid, s, ev0, ev1);
    else if (per_lane == 3) ffn_launch_nch<TW, MT, 3>(a, pass, grid, s, ev0, ev1);
    else ffn_launch_nch<TW, MT, 4>(a, pass, grid, s, ev0, ev1);
  } else {
    constexpr int NCH = MT == 2 ? 4 : (MT == 4 ? 2 : 1);
    ffn_launch_nch<TW, MT, NCH>(a, pass, grid, s, ev0, ev1);
  }
}

template <int NCH>
static void ffn_launch_pred(const FfnArgs& a, const PredictPlanArgs& p, int tiles_x, int grid, hipStream_t s,
                            hipEvent_t ev0, hipEvent_t ev1) {
  if (ev0) hipExtLaunchKernelGGL(k_ffn_gateup_pred<NCH>, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, a, p, tiles_x);
  else k_ffn_gateup_pred<NCH><<<grid, kThreads, 0, s>>>(a, p, tiles_x);
}

bool launch_ffn_gateup_pred(const FfnArgs& in, const PredictPlanArgs& p, int dtype, hipStream_t s, hipEvent_t ev0,
                            hipEvent_t ev1) {
  // batch-1 dense bf16 gate/up rows only, and a prediction of one token
  if (in.q4 || dtype != 1 || in.T != 1 || p.plan.T != 1 || p.Ph > kFusedPredMaxHidden) return false;
  FfnArgs a;
  if (gemv_jobs(in, 0, a) == 0 || a.piece_rows <= 0) return false;
  const int tiles_x = (a.piece_rows + kBlockWaves - 1) / kBlockWaves;  // one row pair per wave
  const int grid = pred_blocks(p.plan.E, p.Ph) + tiles_x * a.n_jobs;
  // as ffn_dispatch<bf16_t, 1> picks NCH for the gate/up pass
  const int per_lane = (a.hidden / Elem<bf16_t>::kPer16B + kWave - 1) / kWave;
  if (per_lane <= 1) ffn_launch_pred<1>(a, p, tiles_x, grid, s, ev0, ev1);
  else if (per_lane == 2) ffn_launch_pred<2>(a, p, tiles_x, grid, s, ev0, ev1);
  else if (per_lane == 3) ffn_launch_pred<3>(a, p, tiles_x, grid, s, ev0, ev1);
  else ffn_launch_pred<4>(a, p, tiles_x, grid, s, ev0, ev1);
  return true;
}

void launch_ffn(const FfnArgs& a, int pass, int max_tokens, int dtype, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int mt = max_tokens >= 8 ? 8 : (max_tokens >= 4 ? 4 : (max_tokens >= 2 ? 2 : 1));
  if (a.q4) {
    if (mt == 8) ffn_dispatch_q4<8>(a, pass, s, ev0, ev1);
    else if (mt == 4) ffn_dispatch_q4<4>(a, pass, s, ev0, ev1);
    else if (mt == 2) ffn_dispatch_q4<2>(a, pass, s, ev0, ev1);
    else ffn_dispatch_q4<1>(a, pass, s, ev0, ev1);
    return;
  }
  if (dtype == 1) {
    if (mt == 8) ffn_dispatch<bf16_t, 8>(a, pass, s, ev0, ev1);
    else if (mt == 4) ffn_dispatch<bf16_t, 4>(a, pass, s, ev0, ev1);
    else if (mt == 2) ffn_dispatch<bf16_t, 2>(a, pass, s, ev0, ev1);
    else ffn_dispatch<bf16_t, 1>(a, pass, s, ev0, ev1);
  } else {
    if (mt == 8) ffn_dispatch<float, 8>(a, pass, s, ev0, ev1);
    else if (mt == 4) ffn_dispatch<float, 4>(a, pass, s, ev0, ev1);
    else if (mt == 2) ffn_dispatch<float, 2>(a, pass, s, ev0, ev1);
    else ffn_dispatch<float, 1>(a, pass, s, ev0, ev1);
  }
}

void launch_combine(const CombineArgs& a, int T, int dtype, hipStream_t s) {
  dim3 grid((a.hidden + kThreads - 1) / kThreads, T);
  if (dtype == 1) k_combine<bf16_t><<<grid, kThreads, 0, s>>>(a);
  else k_combine<float><<<grid, kThreads, 0, s>>>(a);
}

void launch_combine_residual(const CombineArgs& a, float* h, int T, int dtype, hipStream_t s) {
  dim3 grid((a.hidden + kThreads - 1) / kThreads, T);
  if (dtype == 1) k_combine_residual<bf16_t><<<grid, kThreads, 0, s>>>(a, h);
  else k_combine_residual<float><<<grid, kThreads, 0, s>>>(a, h);
}

template <int VPT, bool CMB>
static void rows_norm_launch(const RowsArgs& a, int ntot, int pieces, const float* h, const float* add_src,
                             bf16_t* x_out, const CombineArgs& ca, hipStream_t s) {
  const dim3 grid((ntot + kWaves - 1) / kWaves);
  if (pieces <= kWave) k_rows_gemv_norm<VPT, 1, CMB><<<grid, kThreads, 0, s>>>(a, h, 1e-6f, add_src, x_out, ca);
  else if (pieces <= 2 * kWave)
    k_rows_gemv_norm<VPT, 2, CMB><<<grid, kThreads, 0, s>>>(a, h, 1e-6f, add_src, x_out, ca);
  else if (pieces <= 4 * kWave)
    k_rows_gemv_norm<VPT, 4, CMB><<<grid, kThreads, 0, s>>>(a, h, 1e-6f, add_src, x_out, ca);
  else k_rows_gemv_norm<VPT, 8, CMB><<<grid, kThreads, 0, s>>>(a, h, 1e-6f, add_src, x_out, ca);
}

bool launch_rows_gemv_norm(const RowsArgs& a, const float* h, const float* add_src, void* x_out, hipStream_t s,
                           const CombineArgs* ca) {
  // exactly the cases where the separate kernels take their register paths
  // (launch_rmsnorm_quant and rows_dispatch), so the results agree bit for bit
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
  const int H = a.K, n4 = H / 4, pieces = H / 8;
  auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
  bool ok = a.T == 1 && ntot > 0 && H % 8 == 0 && n4 <= 4 * kThreads && a.relu_in == 0 && al16(h) &&
            (!x_out || al16(x_out));
  for (int i = 0; i < 3; ++i)
    if (a.nrows[i] > 0) ok = ok && al16(a.w[i]);
  // the combine folded in: bf16 y, one shared slice, the token held in at most
  // two float4 pieces per thread (its Y rows in registers)
  if (ca)
    ok = ok && n4 <= 2 * kThreads && ca->hidden == H && ca->top_k >= 1 && ca->top_k <= kMaxK && al16(ca->Y) &&
         (!ca->Ysh || (ca->ysh_split == 1 && al16(ca->Ysh))) && reinterpret_cast<uintptr_t>(ca->y) % 8 == 0;
  if (!ok) return false;
  bf16_t* xo = static_cast<bf16_t*>(x_out);
  const CombineArgs none{};
  if (ca) {
    if (n4 <= kThreads) rows_norm_launch<1, true>(a, ntot, pieces, h, add_src, xo, *ca, s);
    else rows_norm_launch<2, true>(a, ntot, pieces, h, add_src, xo, *ca, s);
  } else if (n4 <= kThreads) {
    rows_norm_launch<1, false>(a, ntot, pieces, h, add_src, xo, none, s);
  } else if (n4 <= 2 * kThreads) {
    rows_norm_launch<2, false>(a, ntot, pieces, h, add_src, xo, none, s);
  } else {
    rows_norm_launch<4, false>(a, ntot, pieces, h, add_src, xo, none, s);
  }
  return true;
}

template <typename TQ>
static void rmsnorm_dispatch(const float* h, void* out, int T, int H, hipStream_t s) {
  const int n4 = H / 4;
  if (H % 4 == 0 && reinterpret_cast<uintptr_t>(h) % 16 == 0 && n4 <= 4 * kThreads) {
    if (n4 <= kThreads) k_rmsnorm_quant_reg<TQ, 1><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
    else if (n4 <= 2 * kThreads) k_rmsnorm_quant_reg<TQ, 2><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
    else k_rmsnorm_quant_reg<TQ, 4><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
  } else {
    k_rmsnorm_quant<TQ><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
  }
}

void launch_rmsnorm_quant(const float* h, void* out, int T, int H, int dtype, hipStream_t s) {
  if (dtype == 1) rmsnorm_dispatch<bf16_t>(h, out, T, H, s);
  else rmsnorm_dispatch<float>(h, out, T, H, s);
}

void launch_residual_add(float* h, const void* y, int n, int dtype, hipStream_t s) {
  dim3 grid((n + kThreads - 1) / kThreads);
  if (dtype == 1) k_residual_add<bf16_t><<<grid, kThreads, 0, s>>>(h, y, n);
  else k_residual_add<float><<<grid, kThreads, 0, s>>>(h, y, n);
}

}  // namespace promoe
