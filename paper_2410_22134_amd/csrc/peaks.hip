// Achievable-peak probes of the GPU (measurement only, not part of the
// method): the kernels' rooflines are reported against the nominal peaks and
// against these measured ones.
//  * k_peak_hbm_read -- each block streams one contiguous piece of a buffer
//                       with 16-byte non-temporal loads, XOR-folded into one
//                       float per block.
//  * k_peak_mfma     -- 8 waves per block, each running rounds of 32
//                       independent v_mfma_f32_16x16x32_bf16 on register
//                       operands (two waves per SIMD keep the matrix core fed).
#include "common.hpp"
#include "promoe.h"

namespace promoe {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef unsigned int gu32x4_t __attribute__((ext_vector_type(4)));

constexpr int kPeakReadThreads = 256;
constexpr int kPeakMfmaThreads = 512;
constexpr int kPeakAcc = 32;

// Each block streams one contiguous piece of the buffer, eight 16-byte loads in
// flight per thread (a wave reads 1 KiB per instruction).  Contiguous pieces of
// 16-128 KiB per block measured 7.2-7.3 TB/s over 4 GiB on gfx950, against
// 6.3-6.9 TB/s for a grid-stride stream over the whole buffer.
constexpr int kPeakReadUnroll = 8;
__global__ __launch_bounds__(kPeakReadThreads) void k_peak_hbm_read(const gu32x4_t* buf, size_t n16, size_t per_block,
                                                                     float* sink) {
  const size_t b0 = (size_t)blockIdx.x * per_block;
  const size_t b1 = b0 + per_block < n16 ? b0 + per_block : n16;
  uint32_t x = 0;
  for (size_t i = b0 + threadIdx.x; i < b1; i += (size_t)kPeakReadUnroll * kPeakReadThreads) {
    gu32x4_t v[kPeakReadUnroll];
#pragma unroll
    for (int u = 0; u < kPeakReadUnroll; ++u) {
      const size_t j = i + (size_t)u * kPeakReadThreads;
      v[u] = j < b1 ? __builtin_nontemporal_load(buf + j) : gu32x4_t{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kPeakReadUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  // one value per block: lanes fold through a wave reduction, lane 0 of wave 0 writes
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if (threadIdx.x == 0) sink[blockIdx.x] = (float)(x & 0xFFFFu);
}

__global__ __launch_bounds__(kPeakMfmaThreads) void k_peak_mfma(float* sink, int iters) {
  bf16x8_t a, b;
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)((threadIdx.x & 63) * 0.0009765625f + j);
    b[j] = (__bf16)(j * 0.5f);
  }
  f32x4_t c[kPeakAcc];
#pragma unroll
  for (int i = 0; i < kPeakAcc; ++i) c[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kPeakAcc; ++i) c[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c[i], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kPeakAcc; ++i) s += c[i][0] + c[i][1] + c[i][2] + c[i][3];
  sink[(size_t)blockIdx.x * kPeakMfmaThreads + threadIdx.x] = s;
}

}  // namespace promoe

using namespace promoe;

extern "C" int promoe_peak_hbm_read(const void* d_buf, size_t bytes, float* d_sink, int blocks, void* stream) {
  if (!d_buf || !d_sink || bytes == 0 || bytes % 16 != 0 || blocks <= 0) return PROMOE_EINVAL;
  const size_t n16 = bytes / 16, per_block = (n16 + blocks - 1) / blocks;
  k_peak_hbm_read<<<blocks, kPeakReadThreads, 0, (hipStream_t)stream>>>(
      reinterpret_cast<const gu32x4_t*>(d_buf), n16, per_block, d_sink);
  return hipGetLastError() == hipSuccess ? PROMOE_OK : PROMOE_EHIP;
}

extern "C" int promoe_peak_mfma_bf16(float* d_sink, int blocks, int iters, void* stream) {
  if (!d_sink || blocks <= 0 || iters <= 0) return PROMOE_EINVAL;
  k_peak_mfma<<<blocks, kPeakMfmaThreads, 0, (hipStream_t)stream>>>(d_sink, iters);
  return hipGetLastError() == hipSuccess ? PROMOE_OK : PROMOE_EHIP;
}
