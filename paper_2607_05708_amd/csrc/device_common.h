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

// Descending bitonic sort of `n` (a power of two, n == 2 * blockDim.x) keys
// in LDS; every thread of the block must call it.
__device__ __forceinline__ void block_bitonic_sort_desc(uint64_t* buf, int n) {
  const int tid = threadIdx.x;
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      const int i = 2 * tid - (tid & (stride - 1));
      const int j = i + stride;
      const bool desc = (i & size) == 0;
      const uint64_t a = buf[i];
      const uint64_t b = buf[j];
      if ((a < b) == desc) {
        buf[i] = b;
        buf[j] = a;
      }
      __syncthreads();
    }
  }
}

}  // namespace memattn
