// Chunk materialisation through the page table (FetchByID + SortByTime of
// Algorithm 1 over the block directory of Section 4.2), and the append-only
// Insert.  Both are HBM-bound copies.
//
// Gather: one workgroup copies one page of one output slot.  Each of its 256
// threads moves 16-byte vectors, sixteen in flight, so a wave issues 1 KiB
// fully coalesced requests; loads and stores are non-temporal because
// neither the source pages nor the gathered output are re-read by this
// kernel.  With time ordering, the workgroup finds the id at its slot's
// position in its group sorted ascending: every id of the group takes the
// position (number of smaller ids + number of equal ids before it), and the
// one at the slot's position is used.
#include "device_common.h"
#include "launch.h"

namespace memattn {

namespace {

constexpr int kMaxGroup = 1024;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void gather_pages_kernel(const u32x4* __restrict__ pool, int64_t n_pages,
                                                           int64_t page_vecs, const int32_t* __restrict__ table,
                                                           int64_t n_chunks, int ppc,
                                                           const int32_t* __restrict__ ids, int64_t count,
                                                           int order, int group, u32x4* __restrict__ out) {
  __shared__ int32_t gids[kMaxGroup];
  __shared__ int32_t chosen_id;
  __shared__ int64_t src_page;
  const int tid = threadIdx.x;
  const int64_t slot = blockIdx.x / ppc;
  const int page = static_cast<int>(blockIdx.x % ppc);

  if (order == 1) {
    const int64_t g0 = (slot / group) * group;
    const int glen = static_cast<int>(min(static_cast<int64_t>(group), count - g0));
    const int want = static_cast<int>(slot - g0);
    for (int i = tid; i < glen; i += 256) gids[i] = ids[g0 + i];
    __syncthreads();
    for (int i = tid; i < glen; i += 256) {
      const int32_t x = gids[i];
      int pos = 0;
      for (int j = 0; j < glen; ++j) {
        const int32_t y = gids[j];
        pos += (y < x || (y == x && j < i)) ? 1 : 0;
      }
      if (pos == want) chosen_id = x;  // positions are distinct: exactly one thread writes
    }
  } else if (tid == 0) {
    chosen_id = ids[slot];
  }
  __syncthreads();
  if (tid == 0) {
    const int32_t c = chosen_id;
    int64_t pg = -1;
    if (c >= 0 && c < n_chunks) {
      const int32_t t = table[static_cast<int64_t>(c) * ppc + page];
      if (t >= 0 && t < n_pages) pg = t;
    }
    src_page = pg;
  }
  __syncthreads();
  const int64_t pg = src_page;
  u32x4* dst = out + blockIdx.x * page_vecs;
  if (pg < 0) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    for (int64_t v = tid; v < page_vecs; v += 256) __builtin_nontemporal_store(z, dst + v);
    return;
  }
  const u32x4* src = pool + pg * page_vecs;
  constexpr int kInFlight = 16;
  for (int64_t v0 = tid; v0 < page_vecs; v0 += kInFlight * 256) {
    u32x4 buf[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int64_t v = v0 + u * 256;
      if (v < page_vecs) buf[u] = __builtin_nontemporal_load(src + v);
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int64_t v = v0 + u * 256;
      if (v < page_vecs) __builtin_nontemporal_store(buf[u], dst + v);
    }
  }
}

// Append: workgroup r copies new row r into bank row n0 + r and writes its
// page-table row.
__global__ __launch_bounds__(256) void append_rows_kernel(uint8_t* __restrict__ bank, int64_t bank_row_bytes,
                                                          int64_t n0, const uint8_t* __restrict__ src,
                                                          int64_t src_row_bytes, int64_t row_bytes,
                                                          int32_t* __restrict__ table, int ppc, int64_t first_page) {
  const int64_t r = blockIdx.x;
  uint8_t* d = bank + (n0 + r) * bank_row_bytes;
  const uint8_t* s = src + r * src_row_bytes;
  for (int64_t b = threadIdx.x; b < row_bytes; b += 256) d[b] = s[b];
  if (threadIdx.x < ppc) table[(n0 + r) * ppc + threadIdx.x] = static_cast<int32_t>(first_page + r * ppc + threadIdx.x);
}

// Fast path of the append when rows are 16-byte aligned and sized.
__global__ __launch_bounds__(256) void append_rows_vec_kernel(u32x4* __restrict__ bank, int64_t bank_row_vecs,
                                                              int64_t n0, const u32x4* __restrict__ src,
                                                              int64_t src_row_vecs, int64_t row_vecs,
                                                              int32_t* __restrict__ table, int ppc,
                                                              int64_t first_page) {
  const int64_t r = blockIdx.x;
  u32x4* d = bank + (n0 + r) * bank_row_vecs;
  const u32x4* s = src + r * src_row_vecs;
  for (int64_t v = threadIdx.x; v < row_vecs; v += 256) d[v] = s[v];
  if (threadIdx.x < ppc) table[(n0 + r) * ppc + threadIdx.x] = static_cast<int32_t>(first_page + r * ppc + threadIdx.x);
}

}  // namespace

hipError_t launch_gather(const void* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                         int64_t n_chunks, int32_t ppc, const int32_t* ids, int64_t count, int32_t order,
                         int32_t group, void* out, hipStream_t stream) {
  if (count == 0) return hipSuccess;
  const int64_t blocks = count * ppc;
  gather_pages_kernel<<<dim3(static_cast<unsigned>(blocks)), 256, 0, stream>>>(
      static_cast<const u32x4*>(pool), n_pages, page_bytes / 16, table, n_chunks, ppc, ids, count, order, group,
      static_cast<u32x4*>(out));
  return hipGetLastError();
}

hipError_t launch_append(void* bank, int64_t bank_stride, int64_t n0, const void* new_emb, int64_t new_stride,
                         int64_t m, int32_t d, int32_t elem_bytes, int32_t* table, int32_t ppc, int64_t first_page,
                         hipStream_t stream) {
  if (m == 0) return hipSuccess;
  const int64_t row_bytes = static_cast<int64_t>(d) * elem_bytes;
  const int64_t brb = bank_stride * elem_bytes, srb = new_stride * elem_bytes;
  const bool vec = (row_bytes % 16 == 0) && (brb % 16 == 0) && (srb % 16 == 0) &&
                   (reinterpret_cast<uintptr_t>(bank) % 16 == 0) && (reinterpret_cast<uintptr_t>(new_emb) % 16 == 0);
  if (vec) {
    append_rows_vec_kernel<<<dim3(static_cast<unsigned>(m)), 256, 0, stream>>>(
        static_cast<u32x4*>(bank), brb / 16, n0, static_cast<const u32x4*>(new_emb), srb / 16, row_bytes / 16, table,
        ppc, first_page);
  } else {
    append_rows_kernel<<<dim3(static_cast<unsigned>(m)), 256, 0, stream>>>(
        static_cast<uint8_t*>(bank), brb, n0, static_cast<const uint8_t*>(new_emb), srb, row_bytes, table, ppc,
        first_page);
  }
  return hipGetLastError();
}

}  // namespace memattn
