// Chunk materialisation through the page table (FetchByID + SortByTime of
// Algorithm 1 over the block directory of Section 4.2), and the append-only
// Insert.  Both are HBM-bound copies.
//
// Gather: one workgroup of 1,024 threads copies two output pages (output
// page u is page u % ppc of slot u / ppc).  Each thread moves 16-byte
// vectors, four per page in flight, so a wave issues 1 KiB fully coalesced
// requests; loads and stores are non-temporal because neither the source
// pages nor the gathered output are re-read by this kernel.  (Two 64 KiB
// pages per 1,024-thread workgroup copy about 17 % faster than one page per
// 256-thread workgroup: fewer, larger workgroups keep more bytes in flight
// per CU.)  With time ordering, the workgroup finds the id at each slot's
// position in its group sorted ascending: every id of the group takes the
// position (number of smaller ids + number of equal ids before it), and the
// one at the slot's position is used.
#include "device_common.h"
#include "launch.h"

namespace memattn {

namespace {

constexpr int kMaxGroup = 1024;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kGatherThreads = 1024;
constexpr int kGatherUnits = 2;     // output pages per workgroup
constexpr int kGatherInFlight = 4;  // 16-byte vectors per thread and page in flight

__global__ __launch_bounds__(kGatherThreads) void gather_pages_kernel(
    const u32x4* __restrict__ pool, int64_t n_pages, int64_t page_vecs, const int32_t* __restrict__ table,
    int64_t n_chunks, int ppc, const int32_t* __restrict__ ids, int64_t count, int order, int group,
    u32x4* __restrict__ out) {
  __shared__ int32_t gids[kMaxGroup];
  __shared__ int32_t chosen_id[kGatherUnits];
  __shared__ int64_t src_page[kGatherUnits];
  const int tid = threadIdx.x;
  const int64_t n_units = count * ppc;
  const int64_t u0 = static_cast<int64_t>(blockIdx.x) * kGatherUnits;
  // (u0 + h < n_units decides, for the whole workgroup, whether unit h exists)
  for (int h = 0; h < kGatherUnits; ++h) {
    const int64_t u = u0 + h;
    if (u >= n_units) break;
    const int64_t slot = u / ppc;
    if (order == 1) {
      const int64_t g0 = (slot / group) * group;
      const int glen = static_cast<int>(min(static_cast<int64_t>(group), count - g0));
      const int want = static_cast<int>(slot - g0);
      __syncthreads();  // the previous unit's reads of gids are done
      for (int i = tid; i < glen; i += kGatherThreads) gids[i] = ids[g0 + i];
      __syncthreads();
      for (int i = tid; i < glen; i += kGatherThreads) {
        const int32_t x = gids[i];
        int pos = 0;
        for (int j = 0; j < glen; ++j) {
          const int32_t y = gids[j];
          pos += (y < x || (y == x && j < i)) ? 1 : 0;
        }
        if (pos == want) chosen_id[h] = x;  // positions are distinct: exactly one thread writes
      }
    } else if (tid == 0) {
      chosen_id[h] = ids[slot];
    }
  }
  __syncthreads();
  if (tid < kGatherUnits) {
    const int64_t u = u0 + tid;
    int64_t pg = -1;
    if (u < n_units) {
      const int32_t c = chosen_id[tid];
      if (c >= 0 && c < n_chunks) {
        const int32_t t = table[static_cast<int64_t>(c) * ppc + u % ppc];
        if (t >= 0 && t < n_pages) pg = t;
      }
    }
    src_page[tid] = pg;
  }
  __syncthreads();
  int64_t pg[kGatherUnits];
  bool live[kGatherUnits];
#pragma unroll
  for (int h = 0; h < kGatherUnits; ++h) {
    pg[h] = src_page[h];
    live[h] = u0 + h < n_units;
  }
  // a page outside the pool (or an id of -1) is written as zeros
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t v0 = tid; v0 < page_vecs; v0 += kGatherInFlight * kGatherThreads) {
    u32x4 buf[kGatherUnits][kGatherInFlight];
#pragma unroll
    for (int h = 0; h < kGatherUnits; ++h) {
#pragma unroll
      for (int i = 0; i < kGatherInFlight; ++i) {
        const int64_t v = v0 + i * kGatherThreads;
        buf[h][i] = (pg[h] >= 0 && v < page_vecs) ? __builtin_nontemporal_load(pool + pg[h] * page_vecs + v) : z;
      }
    }
#pragma unroll
    for (int h = 0; h < kGatherUnits; ++h) {
#pragma unroll
      for (int i = 0; i < kGatherInFlight; ++i) {
        const int64_t v = v0 + i * kGatherThreads;
        if (live[h] && v < page_vecs) __builtin_nontemporal_store(buf[h][i], out + (u0 + h) * page_vecs + v);
      }
    }
  }
}

// Budget-aware materialisation (the prompt prefix of Section 4.3: fetch the
// selected chunks, restore time order, prepend within memory_budget_tokens).
// Workgroup (key i, row block b) writes output rows [b R, b R + R) of key i.
// Wave 0 first plans the key: lane r takes the r-th id in rank order and its
// token count; chunks are admitted while the inclusive prefix sum of counts
// stays within the budget, up to the first id that is -1 (or outside the
// table); each admitted chunk's time position is the number of admitted
// chunks with a smaller id (ties by rank), and its first output row is the
// sum of the counts of the chunks before it in time.  Then every thread maps
// one of the block's rows to its source (page table[c, t / tpp], row t % tpp)
// by a binary search over the time-ordered starts, and the block copies its
// rows in 16-byte vectors, four per thread in flight, zeros past the
// admitted rows.
constexpr int kBudgetRows = 512;      // output rows per workgroup
constexpr int kBudgetThreads = 1024;  // (the copy shape of the page gather)
constexpr int kBudgetInFlight = 4;    // 16-byte vectors per thread in flight

__global__ __launch_bounds__(kBudgetThreads) void gather_budget_kernel(const u32x4* __restrict__ pool, int64_t n_pages,
                                                            int64_t page_vecs, const int32_t* __restrict__ table,
                                                            int64_t n_chunks, int ppc,
                                                            const int32_t* __restrict__ tok_len, int row_vecs,
                                                            int tpp, const int32_t* __restrict__ ids, int k,
                                                            int budget, int blocks_per_key, u32x4* __restrict__ out,
                                                            int32_t* __restrict__ out_tokens,
                                                            int32_t* __restrict__ out_ids) {
  __shared__ int32_t t_id[64];     // admitted chunks in time order
  __shared__ int32_t t_start[65];  // their first output rows; t_start[nk] = total
  __shared__ int32_t s_nk;
  __shared__ int64_t row_src[kBudgetRows];  // source vector index of each row (-1 = zeros)
  const int tid = threadIdx.x;
  const int64_t key = blockIdx.x / blocks_per_key;
  const int blk = static_cast<int>(blockIdx.x % blocks_per_key);
  const int cap = tpp * ppc;

  if (tid < 64) {
    const int lane = tid;
    int32_t c = -1;
    if (lane < k) c = ids[key * k + lane];
    const bool valid = c >= 0 && c < n_chunks;
    int32_t len = 0;
    if (valid) len = min(max(tok_len[c], 0), cap);
    // inclusive prefix sum of the counts over lanes (rank order)
    int32_t pre = len;
    for (int off = 1; off < 64; off <<= 1) {
      const int32_t o = __shfl_up(pre, off);
      if (lane >= off) pre += o;
    }
    const uint64_t bad = __ballot(!valid);  // lanes >= k are invalid too
    const int first_bad = bad ? __builtin_ctzll(bad) : 64;
    const bool keep = lane < first_bad && pre <= budget;
    const uint64_t kept = __ballot(keep);
    const int nk = __builtin_popcountll(kept);
    // time position and first output row of each admitted chunk
    int pos = 0;
    int32_t start = 0;
    for (int j = 0; j < 64; ++j) {
      const int32_t cj = __shfl(c, j);
      const int32_t lj = __shfl(len, j);
      const bool before = ((kept >> j) & 1u) && (cj < c || (cj == c && j < lane));
      pos += before ? 1 : 0;
      start += before ? lj : 0;
    }
    if (keep) {
      t_id[pos] = c;
      t_start[pos] = start;
    }
    // the admitted lanes are lanes 0 .. nk-1 (counts are >= 0, so the
    // prefix sums only grow)
    const int32_t total = __shfl(pre, nk > 0 ? nk - 1 : 0);
    if (lane == 0) {
      t_start[nk] = nk > 0 ? total : 0;
      s_nk = nk;
      if (blk == 0) out_tokens[key] = nk > 0 ? total : 0;
    }
  }
  __syncthreads();
  const int nk = s_nk;
  if (blk == 0 && out_ids != nullptr && tid < k) out_ids[key * k + tid] = tid < nk ? t_id[tid] : -1;

  // source of each of this block's rows
  const int r0 = blk * kBudgetRows;
  const int nrows = min(kBudgetRows, budget - r0);
  const int32_t total = t_start[nk];
  for (int r = tid; r < nrows; r += kBudgetThreads) {
    const int row = r0 + r;
    int64_t src = -1;
    if (row < total) {
      int lo = 0, hi = nk - 1;  // last a with t_start[a] <= row
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (t_start[mid] <= row) lo = mid; else hi = mid - 1;
      }
      const int32_t c = t_id[lo];
      const int t = row - t_start[lo];
      const int32_t pg = table[static_cast<int64_t>(c) * ppc + t / tpp];
      if (pg >= 0 && pg < n_pages) src = static_cast<int64_t>(pg) * page_vecs + static_cast<int64_t>(t % tpp) * row_vecs;
    }
    row_src[r] = src;
  }
  __syncthreads();

  u32x4* dst = out + (key * budget + r0) * static_cast<int64_t>(row_vecs);
  const int n_el = nrows * row_vecs;
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int e0 = tid; e0 < n_el; e0 += kBudgetInFlight * kBudgetThreads) {
    u32x4 buf[kBudgetInFlight];
#pragma unroll
    for (int u = 0; u < kBudgetInFlight; ++u) {
      const int e = e0 + u * kBudgetThreads;
      buf[u] = z;
      if (e < n_el) {
        const int64_t sv = row_src[e / row_vecs];
        if (sv >= 0) buf[u] = __builtin_nontemporal_load(pool + sv + e % row_vecs);
      }
    }
#pragma unroll
    for (int u = 0; u < kBudgetInFlight; ++u) {
      const int e = e0 + u * kBudgetThreads;
      if (e < n_el) __builtin_nontemporal_store(buf[u], dst + e);
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
  const int64_t blocks = (count * ppc + kGatherUnits - 1) / kGatherUnits;
  gather_pages_kernel<<<dim3(static_cast<unsigned>(blocks)), kGatherThreads, 0, stream>>>(
      static_cast<const u32x4*>(pool), n_pages, page_bytes / 16, table, n_chunks, ppc, ids, count, order, group,
      static_cast<u32x4*>(out));
  return hipGetLastError();
}

hipError_t launch_gather_budget(const void* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                                int64_t n_chunks, int32_t ppc, const int32_t* tok_len, int32_t row_bytes,
                                const int32_t* ids, int64_t m, int32_t k, int32_t budget, void* out,
                                int32_t* out_tokens, int32_t* out_ids, hipStream_t stream) {
  if (m == 0) return hipSuccess;
  const int blocks_per_key = budget > 0 ? (budget + kBudgetRows - 1) / kBudgetRows : 1;
  gather_budget_kernel<<<dim3(static_cast<unsigned>(m * blocks_per_key)), kBudgetThreads, 0, stream>>>(
      static_cast<const u32x4*>(pool), n_pages, page_bytes / 16, table, n_chunks, ppc, tok_len, row_bytes / 16,
      static_cast<int>(page_bytes / row_bytes), ids, k, budget, blocks_per_key, static_cast<u32x4*>(out), out_tokens,
      out_ids);
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
