// Background block compaction (Section 4.2, Eq. 2; the background stage of
// Algorithm 2) over the page pool and its directory.
//
// Blocks are P consecutive pages; pages below the allocator frontier have
// been written.  The live chunks are those of the per-namespace chunk tables
// T[u][s] (CSR over namespaces, ascending ids within one); element i = e*ppc
// + p stands for page p of the e-th listed chunk.
//   1. live_kernel: live pages per block (atomic counts).
//   2. phi_kernel: phi(B) = (written(B) - live(B)) / P in fp64, and the
//      compaction flag phi >= theta for blocks wholly below the frontier.
//   3. Exclusive scan of "element i moves" (its page lies in a flagged
//      block) in CSR order: the rank of each moving page within all moving
//      pages, i.e. in (namespace, chunk, page) order.
//   4. Exclusive scan over namespaces of their moving-page counts rounded up
//      to whole blocks: each namespace's first fresh page, so no fresh block
//      mixes namespaces.
//   5. (host: the totals come back and the pool's capacity is checked)
//   6. list_kernel: each moving element's (old page, fresh page, entry).
//   7. move_kernel: one workgroup per moving page copies it (16-byte
//      non-temporal loads and stores, sixteen in flight) and points the
//      directory entry at the fresh page.
// The scans are three launches each: per-block sums, one workgroup scanning
// the block sums, and per-block scans plus the block offset.
#include "device_common.h"
#include "launch.h"

namespace memattn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kScanThreads = 256;
constexpr int kScanItems = 4;
constexpr int kScanBlock = kScanThreads * kScanItems;  // elements per scan workgroup

struct CompactArgs {
  const int32_t* table;
  int64_t n_chunks;
  int ppc;
  const int32_t* offsets;
  const int32_t* chunks;
  int n_ns;
  int64_t n_elems;  // entries * ppc
  int P;
  int64_t next_free;
  const uint8_t* cand;
  const int64_t* pos;  // exclusive scan of moving elements, [n_elems + 1]
};

// page of element i (-1 for a chunk id outside the table)
__device__ __forceinline__ int32_t page_of(const CompactArgs& a, int64_t i) {
  const int32_t c = a.chunks[i / a.ppc];
  if (c < 0 || c >= a.n_chunks) return -1;
  return a.table[static_cast<int64_t>(c) * a.ppc + static_cast<int>(i % a.ppc)];
}

// 1 when element i's page lies in a block being compacted
struct MovingOp {
  CompactArgs a;
  __device__ int64_t operator()(int64_t i) const {
    const int32_t pg = page_of(a, i);
    return (pg >= 0 && pg < a.next_free && a.cand[pg / a.P]) ? 1 : 0;
  }
};

// namespace u's moving pages rounded up to whole blocks
struct PaddedOp {
  CompactArgs a;
  __device__ int64_t operator()(int64_t u) const {
    const int64_t cnt = a.pos[static_cast<int64_t>(a.offsets[u + 1]) * a.ppc] - a.pos[static_cast<int64_t>(a.offsets[u]) * a.ppc];
    return (cnt + a.P - 1) / a.P * a.P;
  }
};

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void live_kernel(CompactArgs a, int32_t* __restrict__ live) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= a.n_elems) return;
  const int32_t pg = page_of(a, i);
  if (pg >= 0 && pg < a.next_free) atomicAdd(live + pg / a.P, 1);
}

__global__ __launch_bounds__(256) void phi_kernel(const int32_t* __restrict__ live, int64_t n_blocks, int P,
                                                  int64_t next_free, double theta, uint8_t* __restrict__ cand,
                                                  float* __restrict__ phi_out, uint8_t* __restrict__ released,
                                                  int32_t* __restrict__ n_cand) {
  const int64_t b = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (b >= n_blocks) return;
  const int64_t left = next_free - b * P;
  const int64_t written = left < P ? left : P;
  const double phi = static_cast<double>(written - live[b]) / static_cast<double>(P);
  const uint8_t c = ((b + 1) * P <= next_free && phi >= theta) ? 1 : 0;
  cand[b] = c;
  if (c) atomicAdd(n_cand, 1);
  if (phi_out) phi_out[b] = static_cast<float>(phi);
  if (released) released[b] = c;
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

struct Move {
  int64_t entry;  // index into the table ([n_chunks, ppc] flattened)
  int32_t old_page;
  int32_t new_page;
};

__global__ __launch_bounds__(256) void list_kernel(CompactArgs a, const int64_t* __restrict__ ns_base,
                                                   int64_t first_new, Move* __restrict__ moves) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= a.n_elems) return;
  const int32_t pg = page_of(a, i);
  if (!(pg >= 0 && pg < a.next_free && a.cand[pg / a.P])) return;
  // namespace of element i: last u with offsets[u] * ppc <= i
  const int64_t e = i / a.ppc;
  int lo = 0, hi = a.n_ns - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.offsets[mid] <= e) lo = mid; else hi = mid - 1;
  }
  const int64_t rank = a.pos[i] - a.pos[static_cast<int64_t>(a.offsets[lo]) * a.ppc];
  const int32_t c = a.chunks[e];
  Move mv;
  mv.entry = static_cast<int64_t>(c) * a.ppc + static_cast<int>(i % a.ppc);
  mv.old_page = pg;
  mv.new_page = static_cast<int32_t>(first_new + ns_base[lo] + rank);
  moves[a.pos[i]] = mv;
}

__global__ __launch_bounds__(256) void move_kernel(u32x4* __restrict__ pool, int64_t page_vecs,
                                                   int32_t* __restrict__ table, const Move* __restrict__ moves) {
  const Move mv = moves[blockIdx.x];
  const u32x4* src = pool + static_cast<int64_t>(mv.old_page) * page_vecs;
  u32x4* dst = pool + static_cast<int64_t>(mv.new_page) * page_vecs;
  constexpr int kInFlight = 16;
  for (int64_t v0 = threadIdx.x; v0 < page_vecs; v0 += kInFlight * 256) {
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
  if (threadIdx.x == 0) table[mv.entry] = mv.new_page;
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

CompactLayout compact_layout(int64_t next_free, int32_t P, int64_t n_entries, int32_t ppc, int32_t n_ns) {
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  CompactLayout L{};
  L.n_blocks = (next_free + P - 1) / P;
  const int64_t n_elems = n_entries * ppc;
  const int64_t nb_e = (n_elems + kScanBlock - 1) / kScanBlock + 1;
  const int64_t nb_u = (static_cast<int64_t>(n_ns) + kScanBlock - 1) / kScanBlock + 1;
  size_t o = 0;
  L.live = o;   o += al(static_cast<size_t>(L.n_blocks) * 4);
  L.cand = o;   o += al(static_cast<size_t>(L.n_blocks));
  L.pos = o;    o += al(static_cast<size_t>(n_elems + 1) * 8);
  L.bsum = o;   o += al(static_cast<size_t>((nb_e > nb_u ? nb_e : nb_u) + 1) * 8);
  L.ns_base = o; o += al(static_cast<size_t>(n_ns + 1) * 8);
  L.moves = o;  o += al(static_cast<size_t>(n_elems > 0 ? n_elems : 1) * sizeof(Move));
  L.counter = o; o += al(8);
  L.bytes = o;
  return L;
}

hipError_t launch_compact_plan(const CompactLayout& L, const int32_t* table, int64_t n_chunks, int32_t ppc,
                               const int32_t* offsets,
                               const int32_t* chunks, int32_t n_ns, int64_t n_entries, int32_t P,
                               int64_t next_free, double theta, float* phi_out, uint8_t* released, void* ws,
                               int64_t* totals_host, hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* live = reinterpret_cast<int32_t*>(w + L.live);
  auto* cand = reinterpret_cast<uint8_t*>(w + L.cand);
  auto* pos = reinterpret_cast<int64_t*>(w + L.pos);
  auto* bsum = reinterpret_cast<int64_t*>(w + L.bsum);
  auto* ns_base = reinterpret_cast<int64_t*>(w + L.ns_base);
  auto* n_cand = reinterpret_cast<int32_t*>(w + L.counter);
  CompactArgs a{table, n_chunks, ppc, offsets, chunks, n_ns, n_entries * ppc, P, next_free, cand, pos};
  fill_i32_kernel<<<blocks256(L.n_blocks), 256, 0, stream>>>(live, L.n_blocks, 0);
  fill_i32_kernel<<<1, 256, 0, stream>>>(n_cand, 1, 0);
  if (a.n_elems > 0) live_kernel<<<blocks256(a.n_elems), 256, 0, stream>>>(a, live);
  if (L.n_blocks > 0)
    phi_kernel<<<blocks256(L.n_blocks), 256, 0, stream>>>(live, L.n_blocks, P, next_free, theta, cand, phi_out,
                                                          released, n_cand);
  hipError_t e = exclusive_scan(MovingOp{a}, a.n_elems, bsum, pos, stream);
  if (e != hipSuccess) return e;
  e = exclusive_scan(PaddedOp{a}, n_ns, bsum, ns_base, stream);
  if (e != hipSuccess) return e;
  // totals: moving pages and fresh pages (namespaces rounded to blocks)
  e = hipMemcpyAsync(totals_host, pos + a.n_elems, sizeof(int64_t), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  e = hipMemcpyAsync(totals_host + 1, ns_base + n_ns, sizeof(int64_t), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  e = hipMemcpyAsync(totals_host + 2, n_cand, sizeof(int32_t), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(stream);
}

hipError_t launch_compact_move(const CompactLayout& L, void* pool, int64_t page_bytes, int32_t* table,
                               int64_t n_chunks, int32_t ppc,
                               const int32_t* offsets, const int32_t* chunks, int32_t n_ns, int64_t n_entries,
                               int32_t P, int64_t next_free, int64_t first_new, int64_t moved, void* ws,
                               hipStream_t stream) {
  if (moved == 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  auto* cand = reinterpret_cast<uint8_t*>(w + L.cand);
  auto* pos = reinterpret_cast<int64_t*>(w + L.pos);
  auto* ns_base = reinterpret_cast<int64_t*>(w + L.ns_base);
  auto* moves = reinterpret_cast<Move*>(w + L.moves);
  CompactArgs a{table, n_chunks, ppc, offsets, chunks, n_ns, n_entries * ppc, P, next_free, cand, pos};
  list_kernel<<<blocks256(a.n_elems), 256, 0, stream>>>(a, ns_base, first_new, moves);
  move_kernel<<<dim3(static_cast<unsigned>(moved)), 256, 0, stream>>>(static_cast<u32x4*>(pool), page_bytes / 16,
                                                                      table, moves);
  return hipGetLastError();
}

}  // namespace memattn
