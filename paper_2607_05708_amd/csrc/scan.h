// Device exclusive scan (three launches: per-workgroup sums, one workgroup
// scanning those sums, per-workgroup scans plus offsets) and a fill kernel,
// shared by the kernels that lay out variable-sized work on the device.
// Internal to the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace memattn {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 4;
constexpr int kScanBlock = kScanThreads * kScanItems;  // elements per scan workgroup

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// Exclusive scan of the 1024 values of workgroup `blk` (v[j] for thread t =
// element blk*1024 + t*4 + j); returns this thread's exclusive prefix and
// the workgroup total through `total`.
__device__ __forceinline__ int64_t block_exclusive(int64_t mine, int64_t* red, int64_t& total) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  int64_t inc = mine;
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t o = __shfl_up(inc, off);
    if (lane >= off) inc += o;
  }
  if (lane == 63) red[wave] = inc;
  __syncthreads();
  int64_t before = 0;
  for (int w = 0; w < wave; ++w) before += red[w];
  total = red[0] + red[1] + red[2] + red[3];
  __syncthreads();
  return before + inc - mine;
}

template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(Op op, int64_t n, int64_t* __restrict__ bsum) {
  __shared__ int64_t red[4];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x * kScanItems;
  int64_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j)
    if (base + j < n) s += op(base + j);
  int64_t total;
  block_exclusive(s, red, total);
  if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

// One workgroup: exclusive scan of bsum[0 .. nb) in place, bsum[nb] = total.
__global__ __launch_bounds__(kScanThreads) void scan_bsum_kernel(int64_t* __restrict__ bsum, int64_t nb) {
  __shared__ int64_t red[4];
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += kScanBlock) {
    const int64_t base = b0 + threadIdx.x * kScanItems;
    int64_t v[kScanItems];
    int64_t s = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      v[j] = base + j < nb ? bsum[base + j] : 0;
      s += v[j];
    }
    int64_t total;
    int64_t ex = block_exclusive(s, red, total) + carry;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
      if (base + j < nb) bsum[base + j] = ex;
      ex += v[j];
    }
    carry += total;
  }
  if (threadIdx.x == 0) bsum[nb] = carry;
}

template <class Op>
__global__ __launch_bounds__(kScanThreads) void scan_apply_kernel(Op op, int64_t n, const int64_t* __restrict__ bsum,
                                                                  int64_t* __restrict__ out) {
  __shared__ int64_t red[4];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanBlock + threadIdx.x * kScanItems;
  int64_t v[kScanItems];
  int64_t s = 0;
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    v[j] = base + j < n ? op(base + j) : 0;
    s += v[j];
  }
  int64_t total;
  int64_t ex = block_exclusive(s, red, total) + bsum[blockIdx.x];
#pragma unroll
  for (int j = 0; j < kScanItems; ++j) {
    if (base + j < n) out[base + j] = ex;
    ex += v[j];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) out[n] = bsum[gridDim.x];  // the total, after the last element
}

template <class Op>
hipError_t exclusive_scan(const Op& op, int64_t n, int64_t* bsum, int64_t* out, hipStream_t stream) {
  const int64_t nb = (n + kScanBlock - 1) / kScanBlock;
  const unsigned grid = static_cast<unsigned>(nb > 0 ? nb : 1);
  scan_reduce_kernel<<<grid, kScanThreads, 0, stream>>>(op, n, bsum);
  scan_bsum_kernel<<<1, kScanThreads, 0, stream>>>(bsum, grid);
  scan_apply_kernel<<<grid, kScanThreads, 0, stream>>>(op, n, bsum, out);
  return hipGetLastError();
}

unsigned blocks256(int64_t n) { return static_cast<unsigned>((n + 255) / 256 > 0 ? (n + 255) / 256 : 1); }
}  // namespace
}  // namespace memattn
