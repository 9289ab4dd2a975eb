// Device-side payload generator for large synthetic page pools (input
// generation only; no part of the retrieval method).  Physical page
// table[c, p] receives the SplitMix64 stream (Steele, Lea and Flood, OOPSLA
// 2014) seeded with `key`, words (c*ppc + p)*wpp .. +wpp-1, where output i
// of the stream is mix(key + (i + 1) * 0x9E3779B97F4A7C15).
#include <hip/hip_runtime.h>
#include <stdint.h>

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

}  // namespace

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
