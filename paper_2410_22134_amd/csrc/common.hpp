// Shared device helpers and launch-argument structs for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace promoe {

typedef uint16_t bf16_t;  // raw bfloat16 bits (upper half of an IEEE-754 binary32)

constexpr int kWave = 64;
constexpr int kMaxE = 64;
constexpr int kMaxK = 8;

// ---------------------------------------------------------------- numerics
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even; NaN kept quiet.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kPer16B = 4;
  __device__ static float load(const float* p, int i) { return p[i]; }
  __device__ static void store(float* p, int i, float v) { p[i] = v; }
  __device__ static float quant(float v) { return v; }
};
template <> struct Elem<bf16_t> {
  static constexpr int kPer16B = 8;
  __device__ static float load(const bf16_t* p, int i) { return bf16_to_f32(p[i]); }
  __device__ static void store(bf16_t* p, int i, float v) { p[i] = f32_to_bf16(v); }
  __device__ static float quant(float v) { return bf16_to_f32(f32_to_bf16(v)); }
};

// 16 bytes of weights -> fp32 values
__device__ __forceinline__ void unpack16(const uint4& c, float (&w)[8]) {
  w[0] = bf16_lo(c.x); w[1] = bf16_hi(c.x); w[2] = bf16_lo(c.y); w[3] = bf16_hi(c.y);
  w[4] = bf16_lo(c.z); w[5] = bf16_hi(c.z); w[6] = bf16_lo(c.w); w[7] = bf16_hi(c.w);
}
__device__ __forceinline__ void unpack16(const uint4& c, float (&w)[4]) {
  w[0] = __uint_as_float(c.x); w[1] = __uint_as_float(c.y);
  w[2] = __uint_as_float(c.z); w[3] = __uint_as_float(c.w);
}

__device__ __forceinline__ float silu(float u) { return u / (1.0f + expf(-u)); }

// ---------------------------------------------------------------- wave ops
// Wave-wide max / min through DPP row operations (no LDS round trips): quad
// permutations and row rotations reduce each row of 16 lanes, two row
// broadcasts carry rows 0-2 into row 3, and lane 63's result is read out as a
// scalar, so every lane gets it.  The whole wave must be active.  Max and min
// are exact in any order, so the result equals a butterfly's.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  // lanes outside the row mask, or whose source is invalid, keep their own value
  return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t v) {
  return ((uint64_t)dpp_u32<kCtrl, kRowMask>((uint32_t)(v >> 32)) << 32) | dpp_u32<kCtrl, kRowMask>((uint32_t)v);
}
__device__ __forceinline__ uint64_t lane63_u64(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}
enum : int {
  kDppQuadXor1 = 0xB1,  // quad_perm [1,0,3,2]
  kDppQuadXor2 = 0x4E,  // quad_perm [2,3,0,1]
  kDppRowRor4 = 0x124,
  kDppRowRor8 = 0x128,
  kDppRowBcast15 = 0x142,  // lane 15 of a row into the next row (rows 1 and 3 by mask 0xa)
  kDppRowBcast31 = 0x143,  // lane 31 into rows 2 and 3 (mask 0xc)
};
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  uint64_t t;
  t = dpp_u64<kDppQuadXor1, 0xf>(v); v = t < v ? t : v;
  t = dpp_u64<kDppQuadXor2, 0xf>(v); v = t < v ? t : v;
  t = dpp_u64<kDppRowRor4, 0xf>(v); v = t < v ? t : v;
  t = dpp_u64<kDppRowRor8, 0xf>(v); v = t < v ? t : v;
  t = dpp_u64<kDppRowBcast15, 0xa>(v); v = t < v ? t : v;
  t = dpp_u64<kDppRowBcast31, 0xc>(v); v = t < v ? t : v;
  return lane63_u64(v);
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
  uint32_t t;
  t = dpp_u32<kDppQuadXor1, 0xf>(v); v = t > v ? t : v;
  t = dpp_u32<kDppQuadXor2, 0xf>(v); v = t > v ? t : v;
  t = dpp_u32<kDppRowRor4, 0xf>(v); v = t > v ? t : v;
  t = dpp_u32<kDppRowRor8, 0xf>(v); v = t > v ? t : v;
  t = dpp_u32<kDppRowBcast15, 0xa>(v); v = t > v ? t : v;
  t = dpp_u32<kDppRowBcast31, 0xc>(v); v = t > v ? t : v;
  return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
// One round of a wave's top-k: among the candidate lanes, the one with the
// largest key, ties to the lower lane (a 64-bit key (key << 32 | 63 - lane)
// orders them the same way); it stops being a candidate.  At least one lane
// must be a candidate.
__device__ __forceinline__ int wave_pick_max(uint32_t key, bool& cand) {
  const uint32_t kmax = wave_max_u32(cand ? key : 0u);
  const uint64_t tie = __ballot(cand && key == kmax);
  const int e = (int)__builtin_ctzll(tie);
  if ((int)(threadIdx.x % kWave) == e) cand = false;
  return e;
}
__device__ __forceinline__ float wave_max(float v) {
  float t;
  t = __uint_as_float(dpp_u32<kDppQuadXor1, 0xf>(__float_as_uint(v))); v = fmaxf(v, t);
  t = __uint_as_float(dpp_u32<kDppQuadXor2, 0xf>(__float_as_uint(v))); v = fmaxf(v, t);
  t = __uint_as_float(dpp_u32<kDppRowRor4, 0xf>(__float_as_uint(v))); v = fmaxf(v, t);
  t = __uint_as_float(dpp_u32<kDppRowRor8, 0xf>(__float_as_uint(v))); v = fmaxf(v, t);
  t = __uint_as_float(dpp_u32<kDppRowBcast15, 0xa>(__float_as_uint(v))); v = fmaxf(v, t);
  t = __uint_as_float(dpp_u32<kDppRowBcast31, 0xc>(__float_as_uint(v))); v = fmaxf(v, t);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
// Wave-wide sum in a fixed order: quads, then pairs of quads, then the whole
// row of 16 (row rotations), then rows 0+1 into row 1 and rows 0..3 into row 3
// (row broadcasts, lanes outside the row mask adding 0); lane 63's sum is
// returned to every lane, so all lanes hold the same bits.  The whole wave
// must be active.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_f32_or0(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, kRowMask, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += dpp_f32_or0<kDppQuadXor1, 0xf>(v);
  v += dpp_f32_or0<kDppQuadXor2, 0xf>(v);
  v += dpp_f32_or0<kDppRowRor4, 0xf>(v);
  v += dpp_f32_or0<kDppRowRor8, 0xf>(v);
  v += dpp_f32_or0<kDppRowBcast15, 0xa>(v);
  v += dpp_f32_or0<kDppRowBcast31, 0xc>(v);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
// Value of lane j (j wave-uniform) as a scalar; v_readlane ignores EXEC.
__device__ __forceinline__ int lane_value(int v, int j) { return __builtin_amdgcn_readlane(v, j); }
__device__ __forceinline__ uint32_t lane_value(uint32_t v, int j) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, j);
}

// Order-preserving map of an fp32 to uint32 (larger float -> larger key).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

}  // namespace promoe
