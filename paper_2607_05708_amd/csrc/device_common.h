// Device helpers shared by the libmemattn kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace memattn {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Order-preserving map from fp32 to uint32: a < b (as floats, no NaN)
// exactly when f2ord(a) < f2ord(b).
__device__ __forceinline__ uint32_t f2ord(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float ord2f(uint32_t o) {
  return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

// Selection key: larger key = better candidate (score descending, then id
// ascending).  Key 0 marks an empty slot and is below every real candidate,
// including a score of -inf.
__device__ __forceinline__ uint64_t make_key(float s, uint32_t idx) {
  return (static_cast<uint64_t>(f2ord(s)) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - idx);
}
__device__ __forceinline__ float key_score(uint64_t k) { return ord2f(static_cast<uint32_t>(k >> 32)); }

__device__ __forceinline__ uint32_t key_idx(uint64_t k) { return 0xFFFFFFFFu - static_cast<uint32_t>(k); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// Hardware base-2 exponential (v_exp_f32): exp2(-inf) = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Write one selected key (slot r of query q) as id, score and probability;
// an empty key (fewer candidates than k) becomes id -1, score -inf, p 0.
__device__ __forceinline__ void write_selected(uint64_t key, float c2, float lse2, int64_t at, int32_t* idx,
                                               float* score, float* prob) {
  const bool have = key != 0;
  const float s = have ? key_score(key) : -INFINITY;
  idx[at] = have ? static_cast<int32_t>(key_idx(key)) : -1;
  if (score) score[at] = s;
  if (prob) prob[at] = have ? fast_exp2(s * c2 - lse2) : 0.f;
}

// Running softmax state in the log2 domain: m = max of x = scale*log2e*s
// seen so far, sum = sum of exp2(x - m).
struct SoftmaxState {
  float m;
  float sum;
};

// Largest of a fully active wave's 64 keys, returned to every lane.  DPP
// steps combine each 16-lane row (swaps within quads, then the half-row and
// row mirrors), and the four row maxima are read out as scalars: a few VALU
// and scalar instructions instead of six dependent cross-lane permutes
// through the LDS unit.
template <int CTRL>
__device__ __forceinline__ uint64_t dpp_max_u64(uint64_t x) {
  const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(x)), CTRL, 0xF, 0xF, false);
  const int hi =
      __builtin_amdgcn_update_dpp(0, static_cast<int>(static_cast<uint32_t>(x >> 32)), CTRL, 0xF, 0xF, false);
  const uint64_t o = (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
  return o > x ? o : x;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
  x = dpp_max_u64<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
  x = dpp_max_u64<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
  x = dpp_max_u64<0x141>(x);  // row_half_mirror: the other quad of the half row
  x = dpp_max_u64<0x140>(x);  // row_mirror: the other half of the row
  uint64_t r = 0;
#pragma unroll
  for (int row = 0; row < 4; ++row) {
    const int lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x)), 16 * row);
    const int hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x >> 32)), 16 * row);
    const uint64_t v = (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
    r = v > r ? v : r;
  }
  return r;
}

}  // namespace memattn
