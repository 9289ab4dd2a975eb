// Device-side payload generator for large synthetic page pools, plus two
// measurement probes (a streaming copy and a register-only MFMA loop) that
// give the bandwidth and matrix-core rates this GPU actually sustains.  Input
// generation and measurement only; no part of the retrieval method.  Physical page
// table[c, p] receives the SplitMix64 stream (Steele, Lea and Flood, OOPSLA
// 2014) seeded with `key`, words (c*ppc + p)*wpp .. +wpp-1, where output i
// of the stream is mix(key + (i + 1) * 0x9E3779B97F4A7C15).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <limits.h>

namespace {

__device__ __forceinline__ uint64_t splitmix64_at(uint64_t key, uint64_t i) {
  uint64_t z = key + (i + 1u) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One workgroup per (chunk, page); pages whose table entry is out of range
// are skipped.
__global__ __launch_bounds__(256) void fill_payload_kernel(uint64_t* __restrict__ pool, int64_t n_pages,
                                                           int64_t wpp, const int32_t* __restrict__ table,
                                                           int64_t chunk0, int ppc, uint64_t key) {
  const int64_t cp = static_cast<int64_t>(blockIdx.x) + chunk0 * ppc;  // global (chunk, page) index
  const int32_t phys = table[cp];
  if (phys < 0 || phys >= n_pages) return;
  uint64_t* dst = pool + static_cast<int64_t>(phys) * wpp;
  const uint64_t base = static_cast<uint64_t>(cp) * static_cast<uint64_t>(wpp);
  for (int64_t w = threadIdx.x; w < wpp; w += 256) dst[w] = splitmix64_at(key, base + static_cast<uint64_t>(w));
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Streaming copy: each workgroup of 1,024 threads moves one contiguous
// 128 KiB chunk in two rounds of four non-temporal 16-byte loads in flight
// per lane (the fastest of the copy shapes tried: 256 to 1,024 threads, 4 to
// 16 loads in flight, 64 KiB to 1 MiB per workgroup, plain or non-temporal).
constexpr int kCopyThreads = 1024;
constexpr int kCopyInFlight = 4;
constexpr int kCopyRounds = 2;
constexpr int64_t kCopyChunk = int64_t{kCopyThreads} * kCopyInFlight * kCopyRounds * 16;
__global__ __launch_bounds__(kCopyThreads) void copy_probe_kernel(const u32x4* __restrict__ src,
                                                                  u32x4* __restrict__ dst) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * (kCopyChunk / 16);
  for (int r = 0; r < kCopyRounds; ++r) {
    const int64_t o = base + static_cast<int64_t>(r) * kCopyThreads * kCopyInFlight + threadIdx.x;
    u32x4 v[kCopyInFlight];
#pragma unroll
    for (int u = 0; u < kCopyInFlight; ++u) v[u] = __builtin_nontemporal_load(src + o + u * kCopyThreads);
#pragma unroll
    for (int u = 0; u < kCopyInFlight; ++u) __builtin_nontemporal_store(v[u], dst + o + u * kCopyThreads);
  }
}

// MFMA issue rate with operands in registers: 8 waves per workgroup, each
// with 8 independent 32x32 accumulators, `iters` x 8 v_mfma_f32_32x32x16_bf16.
__global__ __attribute__((amdgpu_flat_work_group_size(512, 512), amdgpu_waves_per_eu(2, 2))) void mfma_probe_kernel(
    int iters, float* __restrict__ out) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x + i) & 7) * 0.125f);
    b[i] = static_cast<__bf16>(static_cast<float>((threadIdx.x * 3 + i) & 7) * 0.125f);
  }
  f32x16 acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  float t = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
#pragma unroll
    for (int r = 0; r < 16; ++r) t += acc[j][r];
  }
  out[static_cast<int64_t>(blockIdx.x) * 512 + threadIdx.x] = t;
}

}  // namespace

// Copies `bytes` (a positive multiple of 128 KiB) from src to dst.
extern "C" __attribute__((visibility("default"))) int meminputs_copy_probe(const void* src, void* dst, int64_t bytes,
                                                                         void* stream) {
  if (!src || !dst || bytes <= 0 || bytes % kCopyChunk != 0 || bytes / kCopyChunk > INT32_MAX) return -1;
  copy_probe_kernel<<<dim3(static_cast<unsigned>(bytes / kCopyChunk)), kCopyThreads, 0,
                      static_cast<hipStream_t>(stream)>>>(
      static_cast<const u32x4*>(src), static_cast<u32x4*>(dst));
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// Runs `blocks` workgroups of the MFMA loop; out holds blocks * 512 floats.
// Flops = blocks * 8 waves * iters * 8 * 2 * 32 * 32 * 16.
extern "C" __attribute__((visibility("default"))) int meminputs_mfma_probe(int32_t blocks, int32_t iters, float* out,
                                                                         void* stream) {
  if (!out || blocks < 1 || iters < 1) return -1;
  mfma_probe_kernel<<<dim3(static_cast<unsigned>(blocks)), 512, 0, static_cast<hipStream_t>(stream)>>>(iters, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" __attribute__((visibility("default"))) int meminputs_fill_payload(void* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                                      int64_t n_chunks, int32_t ppc, uint64_t key, void* stream) {
  if (!pool || !table || page_bytes <= 0 || page_bytes % 8 != 0 || ppc < 1 || n_chunks < 0) return -1;
  const int64_t wpp = page_bytes / 8;
  const int64_t per_launch = (int64_t{1} << 30) / ppc;  // keep grid.x below 2^31
  for (int64_t c0 = 0; c0 < n_chunks; c0 += per_launch) {
    const int64_t cn = (n_chunks - c0) < per_launch ? (n_chunks - c0) : per_launch;
    fill_payload_kernel<<<dim3(static_cast<unsigned>(cn * ppc)), 256, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<uint64_t*>(pool), n_pages, wpp, table, c0, ppc, key);
    if (hipGetLastError() != hipSuccess) return -4;
  }
  return 0;
}
