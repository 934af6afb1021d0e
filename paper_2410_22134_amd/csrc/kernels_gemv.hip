// Skinny matrix-vector kernels for gfx950 (wave64):
//  * k_rows_gemv   -- gate logits + predictor rows in one pass over x, the
//                     predictor's second layer, the attention surrogate;
//  * k_ffn_gateup  -- expert pass 1: gate and up rows of the experts of a
//                     launch segment read together, act = q(silu(a) * b);
//  * k_ffn_down    -- expert pass 2: Y = Wd act, scattered to (token, rank);
//  * k_combine     -- y = sum_r w Y + s Ysh, fixed r order, one rounding;
//  * k_rmsnorm_quant, k_residual_add -- the layer around the MoE block.
//
// All GEMVs share one scheme: a wave owns R weight rows; every lane streams
// 16-byte pieces of those rows (global_load_dwordx4, coalesced across the
// wave, U pieces per row in flight); the token vectors are staged in LDS as
// fp32 in K-slabs shared by the block's four waves; each lane accumulates in
// fp32 and the wave reduces at the end.  Weight bytes are read once per token
// group of up to MT tokens, which is what bounds decode (HBM) throughput.
#include "common.hpp"
#include "kernels.hpp"

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
// Token pairs of position p: q in [off[p], off[p+1]) of the permuted pair list
// (pair q is token perm[q] / k, rank perm[q] % k).  The shared expert uses
// q = token.
template <typename TW>
__device__ __forceinline__ const TW* expert_weights(const FfnArgs& a, int p) {
  if (a.shared) return reinterpret_cast<const TW*>(a.shared_w);
  const int slot = a.order_slot[p];
  return reinterpret_cast<const TW*>(a.cache + ((size_t)a.layer * a.slots + slot) * a.expert_bytes);
}

template <typename TW, int MT>
__global__ __launch_bounds__(kThreads) void k_ffn_gateup(FfnArgs a) {
  constexpr int RP = 2, R = 2 * RP, U = 2;  // RP (gate, up) row pairs per wave
  __shared__ __attribute__((aligned(16))) float xs[kSlabFloats];
  const int ks_max = kSlabFloats / MT;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int p = a.shared ? 0 : a.pos_list[blockIdx.y];
  const int I = a.shared ? a.shared_inter : a.inter;
  const int H = a.hidden;
  const TW* W = expert_weights<TW>(a, p);
  const int q0 = a.shared ? 0 : a.offsets[p];
  const int q1 = a.shared ? a.T : a.offsets[p + 1];
  const int i0 = (blockIdx.x * kWaves + wave) * RP;
  const TW* rbase[R];
  bool rvalid[R];
#pragma unroll
  for (int j = 0; j < RP; ++j) {
    const bool v = i0 + j < I;
    rvalid[2 * j] = rvalid[2 * j + 1] = v;
    rbase[2 * j] = v ? W + (size_t)(i0 + j) * H : nullptr;            // gate row
    rbase[2 * j + 1] = v ? W + (size_t)(I + i0 + j) * H : nullptr;    // up row
  }
  using TX = TW;
  for (int g = q0; g < q1; g += MT) {
    const int mt = min(MT, q1 - g);
    const TX* xrow[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const int q = g + min(m, mt - 1);
      const int t = a.shared ? q : a.perm[q] / a.top_k;
      xrow[m] = reinterpret_cast<const TX*>(a.x) + (size_t)t * H;
    }
    float acc[R][MT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    for (int k0 = 0; k0 < H; k0 += ks_max) {
      const int ks = min(ks_max, H - k0);
      __syncthreads();
      stage_slab<TX, MT>(xs, ks_max, xrow, mt, k0, ks, false);
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
    if (lane < RP * MT) {
      const int j = lane % RP, m = lane / RP;
      float ga = 0.0f, ub = 0.0f;
#pragma unroll
      for (int jj = 0; jj < RP; ++jj)
#pragma unroll
        for (int mm = 0; mm < MT; ++mm)
          if (jj == j && mm == m) { ga = acc[2 * jj][mm]; ub = acc[2 * jj + 1][mm]; }
      if (m < mt && i0 + j < I) {
        TW* act = reinterpret_cast<TW*>(a.shared ? a.act_sh : a.act);
        Elem<TW>::store(act, (g + m) * I + i0 + j, silu(ga) * ub);
      }
    }
  }
}

template <typename TW, int MT>
__global__ __launch_bounds__(kThreads) void k_ffn_down(FfnArgs a) {
  constexpr int R = 4, U = 2;
  __shared__ __attribute__((aligned(16))) float xs[kSlabFloats];
  const int ks_max = kSlabFloats / MT;
  const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  const int p = a.shared ? 0 : a.pos_list[blockIdx.y];
  const int I = a.shared ? a.shared_inter : a.inter;
  const int H = a.hidden;
  const TW* Wd = expert_weights<TW>(a, p) + (size_t)2 * I * H;
  const int q0 = a.shared ? 0 : a.offsets[p];
  const int q1 = a.shared ? a.T : a.offsets[p + 1];
  const int n0 = (blockIdx.x * kWaves + wave) * R;
  const TW* rbase[R];
  bool rvalid[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    rvalid[r] = n0 + r < H;
    rbase[r] = rvalid[r] ? Wd + (size_t)(n0 + r) * I : nullptr;
  }
  const TW* actb = reinterpret_cast<const TW*>(a.shared ? a.act_sh : a.act);
  for (int g = q0; g < q1; g += MT) {
    const int mt = min(MT, q1 - g);
    const TW* xrow[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) xrow[m] = actb + (size_t)(g + min(m, mt - 1)) * I;
    float acc[R][MT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[r][m] = 0.0f;
    for (int k0 = 0; k0 < I; k0 += ks_max) {
      const int ks = min(ks_max, I - k0);
      __syncthreads();
      stage_slab<TW, MT>(xs, ks_max, xrow, mt, k0, ks, false);
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
        const int q = g + m;
        float* Y = a.shared ? a.Ysh + (size_t)q * H : a.Y + (size_t)a.perm[q] * H;
        Y[n0 + r] = v;
      }
    }
  }
}

// ============================================================ combine
template <typename TY>
__global__ __launch_bounds__(kThreads) void k_combine(CombineArgs a) {
  const int t = blockIdx.y;
  const int n = blockIdx.x * kThreads + threadIdx.x;
  if (n >= a.hidden) return;
  float y = 0.0f;
  for (int r = 0; r < a.top_k; ++r) y += a.w[t * a.top_k + r] * a.Y[((size_t)t * a.top_k + r) * a.hidden + n];
  if (a.Ysh) {
    const float s = a.sscale ? a.sscale[t] : 1.0f;
    y += s * a.Ysh[(size_t)t * a.hidden + n];
  }
  Elem<TY>::store(reinterpret_cast<TY*>(a.y), t * a.hidden + n, y);
}

// ============================================================ harness ops
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
template <typename TW, typename TX>
static void rows_dispatch(const RowsArgs& a, hipStream_t s) {
  const int ntot = a.nrows[0] + a.nrows[1] + a.nrows[2];
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

template <typename TW, int MT>
static void ffn_dispatch(const FfnArgs& a, int pass, int n_pos, hipStream_t s) {
  const int I = a.shared ? a.shared_inter : a.inter;
  if (pass == 0) {
    dim3 grid((I + kWaves * 2 - 1) / (kWaves * 2), n_pos);
    k_ffn_gateup<TW, MT><<<grid, kThreads, 0, s>>>(a);
  } else {
    dim3 grid((a.hidden + kWaves * 4 - 1) / (kWaves * 4), n_pos);
    k_ffn_down<TW, MT><<<grid, kThreads, 0, s>>>(a);
  }
}

void launch_ffn(const FfnArgs& a, int pass, int n_pos, int max_tokens_per_pos, int dtype, hipStream_t s) {
  const int mt = max_tokens_per_pos >= 8 ? 8 : (max_tokens_per_pos >= 4 ? 4 : (max_tokens_per_pos >= 2 ? 2 : 1));
  if (dtype == 1) {
    if (mt == 8) ffn_dispatch<bf16_t, 8>(a, pass, n_pos, s);
    else if (mt == 4) ffn_dispatch<bf16_t, 4>(a, pass, n_pos, s);
    else if (mt == 2) ffn_dispatch<bf16_t, 2>(a, pass, n_pos, s);
    else ffn_dispatch<bf16_t, 1>(a, pass, n_pos, s);
  } else {
    if (mt == 8) ffn_dispatch<float, 8>(a, pass, n_pos, s);
    else if (mt == 4) ffn_dispatch<float, 4>(a, pass, n_pos, s);
    else if (mt == 2) ffn_dispatch<float, 2>(a, pass, n_pos, s);
    else ffn_dispatch<float, 1>(a, pass, n_pos, s);
  }
}

void launch_combine(const CombineArgs& a, int T, int dtype, hipStream_t s) {
  dim3 grid((a.hidden + kThreads - 1) / kThreads, T);
  if (dtype == 1) k_combine<bf16_t><<<grid, kThreads, 0, s>>>(a);
  else k_combine<float><<<grid, kThreads, 0, s>>>(a);
}

void launch_rmsnorm_quant(const float* h, void* out, int T, int H, int dtype, hipStream_t s) {
  if (dtype == 1) k_rmsnorm_quant<bf16_t><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
  else k_rmsnorm_quant<float><<<T, kThreads, 0, s>>>(h, out, H, 1e-6f);
}

void launch_residual_add(float* h, const void* y, int n, int dtype, hipStream_t s) {
  dim3 grid((n + kThreads - 1) / kThreads);
  if (dtype == 1) k_residual_add<bf16_t><<<grid, kThreads, 0, s>>>(h, y, n);
  else k_residual_add<float><<<grid, kThreads, 0, s>>>(h, y, n);
}

}  // namespace promoe
