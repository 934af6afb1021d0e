// Grouped expert GEMMs for prefill on gfx950 MFMA (bf16 in, fp32 accumulate).
//
// Both passes are "NT" products C[m][n] = sum_k A[m][k] B[n][k] with the
// reduction dimension contiguous in both operands:
//   gate/up: A = token rows of x (gathered through the pair permutation),
//            B = Wg rows and Wu rows of the expert (dual B), epilogue
//            act = bf16(silu(A.Wg^T) * (A.Wu^T));
//   down:    A = activation rows, B = Wd rows (two adjacent 128-row ranges
//            when H % 256 == 0), epilogue writes fp32 rows of Y scattered
//            back to (token, rank).
// One launch covers a list of jobs (route positions or the shared expert);
// block b takes tile b of the flat job x m-tile x n-tile list, remapped so the
// m-tiles that share an n-tile (the same weight rows) run on the same XCD and
// meet in its L2.
//
// Block = 4 or 8 waves (two per SIMD for 8), tile BM x 128 x 64 (k).  A and B
// tiles go global -> LDS directly (global_load_lds_dwordx4: each wave
// instruction fills 8 rows of 128 bytes, no staging registers) through a 2- or
// 3-stage ring.  Each wave double-buffers its MFMA fragments in registers: the
// MFMAs of one 32-wide k step run while the fragments of the next are read
// from LDS, and the DMA of a later k-tile is spread over the same MFMA stream
// (one load per row block) instead of being issued in a burst.  LDS rows are
// unpadded and their 16-byte chunks are XOR-swizzled by (row >> 1) & 7, so the
// 16 rows read by one ds_read_b128 phase fall in distinct banks.  Lane l of an
// MFMA supplies A[l % 16][8*(l/16)..+8] and B[l % 16][8*(l/16)..+8] and
// receives C[4*(l/16) + i][l % 16], i < 4.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace promoe {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef unsigned int gu32x4_t __attribute__((ext_vector_type(4)));

constexpr int kBN = 128;
constexpr int kBK = 64;

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ uint4 gload16_stream(const bf16_t* p) {
  const gu32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const gu32x4_t*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ int gemm_find_job(const FfnArgs& a, int bid) {
  int lo = 0, hi = a.n_jobs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.job_tile0[mid] <= bid) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* gbl_ptr_t;

// Chunk (16 bytes) swizzle of LDS row r: logical chunk c lives at c ^ swz(r).
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4] = 7, lgkmcnt [11:8] = 15).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Main loop shared by the expert and rows GEMMs: C[BM x 128] (+= NB of them)
// over k-tiles [kt0, kt1) of 64.  src[i] is this lane's DMA source row pointer
// (already offset to its swizzled 16-byte chunk) for DMA load i; LDS rows
// 0..BM-1 hold A, then NB x 128 rows of B.
template <int BM, int WM, int WN, int NB, int STAGES>
struct GemmTile {
  static constexpr int NW = WM * WN;
  static constexpr int WTM = BM / WM, WTN = kBN / WN;
  static constexpr int TM = WTM / 16, TN = WTN / 16;
  static constexpr int ROWS = BM + NB * kBN;
  static constexpr int STAGE = ROWS * kBK;
  static constexpr int NLD = ROWS / 8 / NW;
  static_assert(ROWS % (8 * NW) == 0 && BM % 16 == 0 && TM >= 1 && TN >= 1, "tile shape");
  static_assert(STAGES == 2 || STAGES == 3, "stages");

  // Fragments of one 32-wide k step: lane l holds A[l % 16][8*(l/16)..+8] of
  // each 16-row A block and B[l % 16][..] of each 16-row B block.
  struct Frag {
    bf16x8_t a[TM];
    bf16x8_t b[NB][TN];
  };

  __device__ static bf16x8_t lds_frag(const bf16_t* L, int r, int c) {
    return as_bf16x8(*reinterpret_cast<const uint4*>(&L[r * kBK + (c ^ swz(r)) * 8]));
  }

  // One k step's MFMAs on f, row block by row block, while the next k step's
  // fragments are read into g: its B blocks after f's first row block, and A
  // block i right after the MFMAs of f's A block i (so g.a[i] can take
  // f.a[i]'s registers).  L is the stage that holds g's k-tile, s2 its k step.
  // With DMA, the loads of a later k-tile (source offset k0, LDS stage dst) are
  // spread over the row blocks too, so no wave stalls on a burst of them
  // before its MFMAs.
  template <bool DMA>
  __device__ static void step(const Frag& f, Frag& g, const bf16_t* L, int s2, f32x4_t (&acc)[NB][TM][TN],
                              int wm, int wn, int lr, int lg, const bf16_t* const (&src)[NLD], int k0,
                              bf16_t* dst, int wave) {
    const int c = s2 * 4 + lg;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int h = 0; h < NB; ++h)
#pragma unroll
        for (int jn = 0; jn < TN; ++jn)
          acc[h][i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[i], f.b[h][jn], acc[h][i][jn], 0, 0, 0);
      if (i == 0) {
#pragma unroll
        for (int h = 0; h < NB; ++h)
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) g.b[h][jn] = lds_frag(L, BM + h * kBN + wn * WTN + jn * 16 + lr, c);
      }
      g.a[i] = lds_frag(L, wm * WTM + i * 16 + lr, c);
      if (DMA) {
#pragma unroll
        for (int d = i * NLD / TM; d < (i + 1) * NLD / TM; ++d)
          __builtin_amdgcn_global_load_lds((gbl_ptr_t)(src[d] + k0), (lds_ptr_t)(dst + 8 * (NW * d + wave) * kBK),
                                           16, 0, 0);
      }
    }
    sched_rows<0, DMA>();
  }

  template <int I, bool DMA>
  __device__ static void sched_rows() {
    if constexpr (I < TM) {
      __builtin_amdgcn_sched_group_barrier(0x008, NB * TN, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, I == 0 ? NB * TN + 1 : 1, 0);
      constexpr int nd = DMA ? (I + 1) * NLD / TM - I * NLD / TM : 0;
      if constexpr (nd > 0) __builtin_amdgcn_sched_group_barrier(0x010, nd, 0);
      sched_rows<I + 1, DMA>();
    }
  }

  __device__ static void first(Frag& g, const bf16_t* L, int wm, int wn, int lr, int lg) {
#pragma unroll
    for (int h = 0; h < NB; ++h)
#pragma unroll
      for (int jn = 0; jn < TN; ++jn) g.b[h][jn] = lds_frag(L, BM + h * kBN + wn * WTN + jn * 16 + lr, lg);
#pragma unroll
    for (int i = 0; i < TM; ++i) g.a[i] = lds_frag(L, wm * WTM + i * 16 + lr, lg);
  }

  __device__ static void last(const Frag& f, f32x4_t (&acc)[NB][TM][TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int h = 0; h < NB; ++h)
#pragma unroll
        for (int jn = 0; jn < TN; ++jn)
          acc[h][i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(f.a[i], f.b[h][jn], acc[h][i][jn], 0, 0, 0);
  }

  __device__ static void barrier() {
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __asm__ volatile("" ::: "memory");
  }

  __device__ static void run(const bf16_t* const (&src)[NLD], int kt0, int kt1, bf16_t* lds,
                             f32x4_t (&acc)[NB][TM][TN], int wave, int lane) {
    const int wm = wave / WN, wn = wave % WN;
    const int lr = lane % 16, lg = lane / 16;
#pragma unroll
    for (int h = 0; h < NB; ++h)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int jn = 0; jn < TN; ++jn) acc[h][i][jn] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // k-tile kt lives in stage (kt - kt0) % STAGES.  A tile's stage is
    // refilled as soon as every wave has read both of its k steps into
    // registers: the barrier between the two k steps of tile t follows each
    // wave's wait for its own reads of tile t and its own DMA of tile t + 1,
    // so after it tile t + 1 is visible to all waves and tile t + STAGES may
    // overwrite tile t's stage; its DMA is spread over the next k step.  Every
    // iteration issues one tile (past the last tile, the last tile again, into
    // a stage that is not read any more), so exactly STAGES - 2 later tiles
    // may be in flight when tile t + 1 must have landed.
    const int nk = kt1 - kt0;
    if (nk <= 0) return;
#pragma unroll
    for (int st = 0; st < STAGES; ++st) {
      bf16_t* dst = lds + st * STAGE;
      const int k0 = (kt0 + min(st, nk - 1)) * kBK;
#pragma unroll
      for (int i = 0; i < NLD; ++i)
        __builtin_amdgcn_global_load_lds((gbl_ptr_t)(src[i] + k0), (lds_ptr_t)(dst + 8 * (NW * i + wave) * kBK),
                                         16, 0, 0);
    }
    wait_vmcnt<(STAGES - 1) * NLD < 64 ? (STAGES - 1) * NLD : 63>();
    barrier();
    Frag f0, f1;
    first(f0, lds, wm, wn, lr, lg);
    for (int t = 0; t + 1 < nk; ++t) {
      step<false>(f0, f1, lds + (t % STAGES) * STAGE, 1, acc, wm, wn, lr, lg, src, 0, lds, wave);
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's reads of tile t are done
      wait_vmcnt<(STAGES - 2) * NLD>();
      barrier();
      step<true>(f1, f0, lds + ((t + 1) % STAGES) * STAGE, 0, acc, wm, wn, lr, lg, src,
                 (kt0 + min(t + STAGES, nk - 1)) * kBK, lds + (t % STAGES) * STAGE, wave);
    }
    step<false>(f0, f1, lds + ((nk - 1) % STAGES) * STAGE, 1, acc, wm, wn, lr, lg, src, 0, lds, wave);
    last(f1, acc);
    wait_vmcnt<0>();  // no DMA may land in LDS after the block has left it
  }
};

__device__ __forceinline__ int xcd_grouped(int b, int nblk) {
  // block b runs on XCD b % 8: give each XCD a contiguous range of tiles
  return (nblk & 7) == 0 ? (b & 7) * (nblk >> 3) + (b >> 3) : b;
}

// One output tile of job jd: rows m0 .. m0+BM-1 of its token range, columns
// n0 .. n0+127 (per B), k-tiles [kt0, kt1), split-K slice ks (down pass of
// the shared expert).  PASS 0: gate/up (dual B: Wg and Wu rows of one column
// range), PASS 1: down over columns n0 .. n0+127, PASS 2: down over columns
// n0 .. n0+255 (two B blocks).
template <int BM, int WM, int WN, int PASS, int STAGES>
__device__ __forceinline__ void ffn_tile(const FfnArgs& a, bf16_t* lds, const FfnJob& jd, int m0, int n0, int ks,
                                         int kt0, int kt1, int wave, int lane) {
  constexpr int NB = PASS == 1 ? 1 : 2;  // PASS 2: down over two adjacent 128-column ranges
  using G = GemmTile<BM, WM, WN, NB, STAGES>;
  const int wm = wave / WN, wn = wave % WN;
  const bool shared = jd.pos == kSharedJob;
  const int I = jd.I;
  const int H = a.hidden;
  const int K = PASS == 0 ? H : I;
  const int q0 = jd.q0, M = jd.q1 - q0;
  const bf16_t* W = reinterpret_cast<const bf16_t*>(jd.w);

  // DMA sources.  Load i of this wave fills LDS rows 8*(NW*i + wave) .. +8;
  // lane L writes row 8*(NW*i + wave) + L/8, physical chunk L%8, so it fetches
  // logical chunk (L%8) ^ swz(row) of that row.
  const bf16_t* src[G::NLD];
#pragma unroll
  for (int i = 0; i < G::NLD; ++i) {
    const int r = 8 * (G::NW * i + wave) + lane / 8;
    const int c = (lane % 8) ^ swz(r);
    if (r < BM) {
      const int m = min(m0 + r, M - 1);  // rows past M load a valid row; results are discarded
      const bf16_t* row;
      if (PASS == 0) {
        const int q = q0 + m;
        const int t = shared ? q : a.perm[q] / a.top_k;
        row = reinterpret_cast<const bf16_t*>(a.x) + (size_t)t * H;
      } else {
        row = reinterpret_cast<const bf16_t*>(shared ? a.act_sh : a.act) + (size_t)(q0 + m) * I;
      }
      src[i] = row + c * 8;
    } else {
      const int rb = r - BM;
      const int which = rb / kBN, n = n0 + (PASS == 2 ? which * kBN : 0) + rb % kBN;
      const bf16_t* base = PASS == 0 ? W + (size_t)which * I * H : W + (size_t)2 * I * H;  // Wg | Wu, or Wd
      src[i] = base + (size_t)n * K + c * 8;
    }
  }
  f32x4_t acc[NB][G::TM][G::TN];
  G::run(src, kt0, kt1, lds, acc, wave, lane);

  // ---- epilogue
  const int lr = lane % 16, row_in = 4 * (lane / 16);
#pragma unroll
  for (int i = 0; i < G::TM; ++i) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * G::WTM + i * 16 + row_in + r;
      if (m >= M) continue;
      const int q = q0 + m;
      if (PASS == 0) {
        bf16_t* act = reinterpret_cast<bf16_t*>(shared ? a.act_sh : a.act);
#pragma unroll
        for (int jn = 0; jn < G::TN; ++jn) {
          const int n = n0 + wn * G::WTN + jn * 16 + lr;
          act[(size_t)q * I + n] = f32_to_bf16(silu(acc[0][i][jn][r]) * acc[1][i][jn][r]);
        }
      } else {
        float* Y = shared ? a.Ysh + (size_t)ks * a.ysh_split_stride + (size_t)q * H : a.Y + (size_t)a.perm[q] * H;
#pragma unroll
        for (int h = 0; h < NB; ++h)
#pragma unroll
          for (int jn = 0; jn < G::TN; ++jn) Y[n0 + h * kBN + wn * G::WTN + jn * 16 + lr] = acc[h][i][jn][r];
      }
    }
  }
}

// Tail tiles of a one-job gate/up launch: 128 rows, 3 stages.
using TailTile = GemmTile<128, 2, 4, 2, 3>;

// Block b < tail_block0 takes tile b of the flat job x m-tile x n-tile list;
// blocks from tail_block0 on (gate/up of one job only) take tiles of half the
// height over the job's n-tiles from tail_n0, so the launch's last round is
// made of half-size tiles instead of a part-filled round of full ones.
template <int BM, int WM, int WN, int PASS, int STAGES>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_ffn(FfnArgs a) {
  constexpr int NB = PASS == 1 ? 1 : 2;
  using G = GemmTile<BM, WM, WN, NB, STAGES>;
  constexpr bool TAIL = PASS == 0 && BM == 256 && WM * WN == 8;
  constexpr int LDS = TAIL && 3 * TailTile::STAGE > STAGES * G::STAGE ? 3 * TailTile::STAGE : STAGES * G::STAGE;
  __shared__ __attribute__((aligned(1024))) bf16_t lds[LDS];

  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  if constexpr (TAIL) {
    if ((int)blockIdx.x >= a.tail_block0) {
      const int bt = xcd_grouped(blockIdx.x - a.tail_block0, gridDim.x - a.tail_block0);
      const FfnJob jd = a.jobs[0];
      const int mt = (jd.q1 - jd.q0 + 127) / 128;
      ffn_tile<128, 2, 4, PASS, 3>(a, lds, jd, (bt % mt) * 128, (a.tail_n0 + bt / mt) * kBN, 0, 0,
                                   a.hidden / kBK, wave, lane);
      return;
    }
  }
  const int b = xcd_grouped(blockIdx.x, min((int)gridDim.x, a.tail_block0));
  const int j = gemm_find_job(a, b);
  int jt = b - a.job_tile0[j];
  const FfnJob jd = a.jobs[j];
  const bool shared = jd.pos == kSharedJob;
  const int N = PASS == 0 ? jd.I : a.hidden;
  const int K = PASS == 0 ? a.hidden : jd.I;
  const int M = jd.q1 - jd.q0;
  const int mtiles = (M + BM - 1) / BM;
  const int ntiles = N / (PASS == 2 ? 2 * kBN : kBN);
  // split-K (shared down pass only): slice ks of S writes its own partial output
  const int S = (PASS != 0 && shared) ? a.ksplit : 1;
  const int ks = jt / (mtiles * ntiles);
  jt -= ks * mtiles * ntiles;
  const int nk = K / kBK;
  ffn_tile<BM, WM, WN, PASS, STAGES>(a, lds, jd, (jt % mtiles) * BM, (jt / mtiles) * kBN * (PASS == 2 ? 2 : 1), ks, ks * nk / S,
                                     (ks + 1) * nk / S, wave, lane);
}

// out[t][o_off + n] (=|+=) sum_k W[n][k] x[t][k] for n < N (rows past N load the
// last row; their results are discarded).
template <int BM, int WM, int WN, int STAGES>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_rows(RowsGemmArgs a) {
  using G = GemmTile<BM, WM, WN, 1, STAGES>;
  __shared__ __attribute__((aligned(1024))) bf16_t lds[STAGES * G::STAGE];
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const int wm = wave / WN, wn = wave % WN;
  const int b = xcd_grouped(blockIdx.x, gridDim.x);
  const int mtiles = (a.T + BM - 1) / BM;
  const int m0 = (b % mtiles) * BM;
  const int n0 = (b / mtiles) * kBN;
  const bf16_t* X = reinterpret_cast<const bf16_t*>(a.x);
  const bf16_t* W = reinterpret_cast<const bf16_t*>(a.w);
  const bf16_t* src[G::NLD];
#pragma unroll
  for (int i = 0; i < G::NLD; ++i) {
    const int r = 8 * (G::NW * i + wave) + lane / 8;
    const int c = (lane % 8) ^ swz(r);
    if (r < BM) src[i] = X + (size_t)min(m0 + r, a.T - 1) * a.ldx + c * 8;
    else src[i] = W + (size_t)min(n0 + r - BM, a.N - 1) * a.K + c * 8;
  }
  f32x4_t acc[1][G::TM][G::TN];
  G::run(src, 0, a.K / kBK, lds, acc, wave, lane);
  const int lr = lane % 16, row_in = 4 * (lane / 16);
#pragma unroll
  for (int i = 0; i < G::TM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + wm * G::WTM + i * 16 + row_in + r;
      if (m >= a.T) continue;
#pragma unroll
      for (int jn = 0; jn < G::TN; ++jn) {
        const int n = n0 + wn * G::WTN + jn * 16 + lr;
        if (n >= a.N) continue;
        float* o = a.out + (size_t)m * a.ldo + a.o_off + n;
        *o = a.add ? *o + acc[0][i][jn][r] : acc[0][i][jn][r];
      }
    }
}

// Down pass over pairs of adjacent 128-column ranges (PASS 2): a 256 x 256
// output tile, the same reuse of each loaded row as the dual-B gate/up tile.
static bool down_pair(int H) { return H % (2 * kBN) == 0; }

template <int BM, int WM, int WN, int S>
static void gemm_dispatch(FfnArgs& a, int pass, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const bool down2 = pass == 1 && down_pair(a.hidden);
  int tiles = 0;
  for (int j = 0; j < a.n_jobs; ++j) {
    a.job_tile0[j] = tiles;
    const bool sh = a.jobs[j].pos == kSharedJob;
    const int N = pass == 0 ? a.jobs[j].I : a.hidden;
    const int M = a.jobs[j].q1 - a.jobs[j].q0;
    const int split = (pass == 1 && sh) ? a.ksplit : 1;
    tiles += ((M + BM - 1) / BM) * (N / (pass == 1 && down2 ? 2 * kBN : kBN)) * split;
  }
  a.job_tile0[a.n_jobs] = tiles;
  if (tiles == 0) return;
  int grid = tiles;
  a.tail_block0 = tiles;
  a.tail_n0 = 0;
  if (pass == 0 && BM == 256 && WM * WN == 8 && a.n_jobs == 1 && tiles % 256 != 0 && tiles > 256) {
    // whole rounds of full tiles over the 256 CUs, then half-height tiles
    const int M = a.jobs[0].q1 - a.jobs[0].q0;
    const int mtiles = (M + BM - 1) / BM, ntiles = a.jobs[0].I / kBN;
    const int full = tiles / 256 * 256;
    if (full % mtiles == 0) {
      a.tail_n0 = full / mtiles;
      a.tail_block0 = full;
      a.job_tile0[1] = full;
      grid = full + (ntiles - a.tail_n0) * ((M + 127) / 128);
    }
  }
  const dim3 g(grid), b(64 * WM * WN);
  if (pass == 0) hipExtLaunchKernelGGL((k_gemm_ffn<BM, WM, WN, 0, S>), g, b, 0, s, ev0, ev1, 0, a);
  else if (down2) hipExtLaunchKernelGGL((k_gemm_ffn<BM, WM, WN, 2, S>), g, b, 0, s, ev0, ev1, 0, a);
  else hipExtLaunchKernelGGL((k_gemm_ffn<BM, WM, WN, 1, S>), g, b, 0, s, ev0, ev1, 0, a);
}

bool gemm_supported(int N, int K) { return N % kBN == 0 && K % kBK == 0; }

// Tile height: the tallest of 256 / 128 / 64 rows whose count of 128-column
// tiles still covers the 256 CUs (most reuse of each weight tile while filling
// the machine; a down pass over column pairs then runs half as many blocks of
// twice the work, which measured faster than the next smaller height).
static int pick_bm(const FfnArgs& a, int pass, int max_tokens) {
  const int cands[3] = {256, 128, 64};
  for (int ci = 0; ci < 3; ++ci) {
    const int bm = cands[ci];
    if (bm == 256 && max_tokens < 512) continue;
    if (bm == 128 && max_tokens <= 64) continue;
    int tiles = 0;
    for (int j = 0; j < a.n_jobs; ++j) {
      const bool sh = a.jobs[j].pos == kSharedJob;
      const int N = pass == 0 ? a.jobs[j].I : a.hidden;
      const int M = a.jobs[j].q1 - a.jobs[j].q0;
      tiles += ((M + bm - 1) / bm) * (N / kBN) * ((pass == 1 && sh) ? a.ksplit : 1);
    }
    if (tiles >= 256 || bm == 64) return bm;
  }
  return 64;
}

// Split-K slices of the shared expert's down GEMM, which has only (T / BM) x
// (H / 256) output tiles.  Over column pairs: as many slices as fit in one
// round of blocks over the 256 CUs (Qwen2-57B shape, 56 tiles: split 4 at
// 140 us against 150 / 162 / 150 us for splits 2 / 7 / 8).  Over single
// columns: the smallest split giving at least 1.5 rounds (112 tiles: split 4
// at 195 us against 242 / 250 / 238 / 209 us for splits 2 / 3 / 5 / 6).
int gemm_shared_down_split(int T, int H) {
  const int bm = T >= 512 ? 256 : (T > 64 ? 128 : 64);
  const int mt = (T + bm - 1) / bm;
  if (down_pair(H)) return std::max(1, 256 / (mt * (H / (2 * kBN))));
  const int tiles = mt * (H / kBN);
  return (384 + tiles - 1) / tiles;
}

void launch_gemm_rows(const RowsGemmArgs& a, hipStream_t s) {
  const int ntiles = (a.N + kBN - 1) / kBN;
  if (a.T >= 256) {
    k_gemm_rows<128, 2, 4, 3><<<((a.T + 127) / 128) * ntiles, 512, 0, s>>>(a);
  } else {
    k_gemm_rows<64, 1, 4, 3><<<((a.T + 63) / 64) * ntiles, 256, 0, s>>>(a);
  }
}

void launch_gemm(FfnArgs& a, int pass, int max_tokens, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
  const int bm = pick_bm(a, pass, max_tokens);
  if (bm == 256) gemm_dispatch<256, 2, 4, 2>(a, pass, s, ev0, ev1);
  else if (bm == 128) gemm_dispatch<128, 2, 4, 3>(a, pass, s, ev0, ev1);
  else gemm_dispatch<64, 1, 4, 3>(a, pass, s, ev0, ev1);
}

}  // namespace promoe
