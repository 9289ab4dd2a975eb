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
//   5. (host: the totals come back in one copy, gathered by totals_kernel,
//      and the pool's capacity is checked)
//   6. list_kernel: each moving element's (old page, fresh page, entry).
//   7. move_kernel: one workgroup of 1,024 threads per two moving pages
//      copies them (16-byte non-temporal loads and stores, four per thread
//      and page in flight) and points the directory entries at the fresh
//      pages.
// The scans are the three-launch device scans of scan.h.
//
// Association-aware relocation (the online stage of Algorithm 2, with the
// dense relation score standing in for the model's co-location choice):
//   1. claim_kernel (one wave per key): lane r holds the key's r-th selected
//      id; the group G_i is the ids scoring >= tau, and it qualifies when it
//      has at least min_group entries; each qualifying group claims its
//      chunks with an atomic min of the key index, so a chunk goes to the
//      first key whose group holds it (as if keys were served in order).
//   2. keep_kernel (one wave per key): the chunks the key won, each at its
//      time position (the number of won chunks with smaller ids).
//   3. Exclusive scan over keys of the won counts: the key's first fresh
//      chunk slot.  (host: totals back, capacity checked)
//   4. reloc_move_kernel: one workgroup per two moved pages copies each to
//      frontier + slot * ppc + page and updates its directory entry; the old
//      copy is left behind as an invalid page.
#include "device_common.h"
#include "launch.h"
#include "scan.h"

namespace memattn {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// namespace u's entry range, clamped to the table (a malformed table is
// rejected before anything moves; the clamp keeps the plan's reads in bounds)
__device__ __forceinline__ int64_t entry_off(const CompactArgs& a, int64_t u) {
  const int64_t n_entries = a.n_elems / a.ppc;
  return min(max(static_cast<int64_t>(a.offsets[u]), int64_t{0}), n_entries);
}

// namespace u's moving pages rounded up to whole blocks
struct PaddedOp {
  CompactArgs a;
  __device__ int64_t operator()(int64_t u) const {
    const int64_t lo = entry_off(a, u);
    const int64_t hi = max(entry_off(a, u + 1), lo);
    const int64_t cnt = a.pos[hi * a.ppc] - a.pos[lo * a.ppc];
    return (cnt + a.P - 1) / a.P * a.P;
  }
};

// Flags (bit 0) a malformed chunk table: offsets not starting at 0, falling,
// or not ending at n_entries, or a chunk id outside the directory or not
// above its predecessor in the same namespace.
__global__ __launch_bounds__(256) void check_tables_kernel(CompactArgs a, int32_t* __restrict__ bad) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t n_entries = a.n_elems / a.ppc;
  bool wrong = false;
  if (i <= a.n_ns) {
    const int32_t o = a.offsets[i];
    if (i == 0 && o != 0) wrong = true;
    if (i == a.n_ns && o != n_entries) wrong = true;
    if (i > 0 && o < a.offsets[i - 1]) wrong = true;
    if (o < 0 || o > n_entries) wrong = true;
  }
  if (i < n_entries) {
    const int32_t c = a.chunks[i];
    if (c < 0 || c >= a.n_chunks) wrong = true;
    // a namespace starts at entry i when some offset equals i; otherwise the
    // previous entry must hold a smaller id
    if (i > 0 && c <= a.chunks[i - 1]) {
      int lo = 0, hi = a.n_ns;  // is i one of the offsets?
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (a.offsets[mid] < i) lo = mid + 1; else hi = mid;
      }
      if (!(lo <= a.n_ns && a.offsets[lo] == i)) wrong = true;
    }
  }
  if (wrong) atomicOr(bad, 1);
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
  const int64_t rank = a.pos[i] - a.pos[entry_off(a, lo) * a.ppc];
  const int32_t c = a.chunks[e];
  Move mv;
  mv.entry = static_cast<int64_t>(c) * a.ppc + static_cast<int>(i % a.ppc);
  mv.old_page = pg;
  mv.new_page = static_cast<int32_t>(first_new + ns_base[lo] + rank);
  moves[a.pos[i]] = mv;
}

// Page copies of the move phases: a workgroup of 1,024 threads copies two
// pages, four 16-byte vectors per thread and page in flight (the copy shape
// that streams HBM fastest on this GPU); src and dst are pool pages (a
// negative src writes zeros), and the two units of a workgroup never
// overlap (sources lie below the frontier, destinations at or above it).
constexpr int kMoveThreads = 1024;
constexpr int kMoveUnits = 2;
constexpr int kMoveInFlight = 4;
__device__ __forceinline__ void copy_pages(u32x4* __restrict__ pool, int64_t page_vecs,
                                           const int64_t (&src)[kMoveUnits], const int64_t (&dst)[kMoveUnits],
                                           const bool (&live)[kMoveUnits]) {
  for (int64_t v0 = threadIdx.x; v0 < page_vecs; v0 += kMoveInFlight * kMoveThreads) {
    u32x4 buf[kMoveUnits][kMoveInFlight];
#pragma unroll
    for (int h = 0; h < kMoveUnits; ++h) {
#pragma unroll
      for (int i = 0; i < kMoveInFlight; ++i) {
        const int64_t v = v0 + i * kMoveThreads;
        if (live[h] && v < page_vecs)
          buf[h][i] = src[h] >= 0 ? __builtin_nontemporal_load(pool + src[h] * page_vecs + v) : u32x4{0u, 0u, 0u, 0u};
      }
    }
#pragma unroll
    for (int h = 0; h < kMoveUnits; ++h) {
#pragma unroll
      for (int i = 0; i < kMoveInFlight; ++i) {
        const int64_t v = v0 + i * kMoveThreads;
        if (live[h] && v < page_vecs) __builtin_nontemporal_store(buf[h][i], pool + dst[h] * page_vecs + v);
      }
    }
  }
}

// Moves kMoveUnits planned pages per workgroup and points their directory
// entries at the new pages.
__global__ __launch_bounds__(kMoveThreads) void move_kernel(u32x4* __restrict__ pool, int64_t page_vecs,
                                                            int32_t* __restrict__ table,
                                                            const Move* __restrict__ moves, int64_t n_moves) {
  const int64_t m0 = static_cast<int64_t>(blockIdx.x) * kMoveUnits;
  Move mv[kMoveUnits];
  int64_t src[kMoveUnits], dst[kMoveUnits];
  bool live[kMoveUnits];
#pragma unroll
  for (int h = 0; h < kMoveUnits; ++h) {
    live[h] = m0 + h < n_moves;
    mv[h] = live[h] ? moves[m0 + h] : Move{0, 0, 0};
    src[h] = mv[h].old_page;
    dst[h] = mv[h].new_page;
  }
  copy_pages(pool, page_vecs, src, dst, live);
#pragma unroll
  for (int h = 0; h < kMoveUnits; ++h)
    if (threadIdx.x == h && live[h]) table[mv[h].entry] = mv[h].new_page;
}

constexpr int32_t kNoOwner = 0x7FFFFFFF;

struct ColocArgs {
  const int32_t* ids;
  const float* scores;
  int64_t m;
  int k;
  double tau;
  int min_group;
  int64_t n_chunks;
};

// Group membership of lane r's id (valid id, score >= tau), whether it is
// the first occurrence of that id among members, and whether the group
// qualifies.  Every lane of the wave must call it.
__device__ __forceinline__ void coloc_lane(const ColocArgs& a, int64_t key, int lane, int32_t& c, bool& first,
                                           bool& qualifies) {
  c = -1;
  bool member = false;
  if (lane < a.k) {
    c = a.ids[key * a.k + lane];
    member = c >= 0 && c < a.n_chunks && static_cast<double>(a.scores[key * a.k + lane]) >= a.tau;
  }
  const uint64_t mem = __ballot(member);
  qualifies = __builtin_popcountll(mem) >= a.min_group;
  first = member;
  for (int j = 0; j < 64; ++j) {
    const int32_t cj = __shfl(c, j);
    if (((mem >> j) & 1u) && j < lane && cj == c) first = false;
  }
}

__global__ __launch_bounds__(256) void claim_kernel(ColocArgs a, int32_t* __restrict__ owner) {
  const int64_t key = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (key >= a.m) return;  // whole waves
  const int lane = threadIdx.x & 63;
  int32_t c;
  bool first, qualifies;
  coloc_lane(a, key, lane, c, first, qualifies);
  if (qualifies && first) atomicMin(owner + c, static_cast<int32_t>(key));
}

__global__ __launch_bounds__(256) void keep_kernel(ColocArgs a, const int32_t* __restrict__ owner,
                                                   int32_t* __restrict__ klist, int64_t* __restrict__ cnt,
                                                   int32_t* __restrict__ n_groups) {
  const int64_t key = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (key >= a.m) return;  // whole waves
  const int lane = threadIdx.x & 63;
  int32_t c;
  bool first, qualifies;
  coloc_lane(a, key, lane, c, first, qualifies);
  const bool keep = qualifies && first && owner[c] == static_cast<int32_t>(key);
  const uint64_t kept = __ballot(keep);
  int pos = 0;
  for (int j = 0; j < 64; ++j) {
    const int32_t cj = __shfl(c, j);
    if (((kept >> j) & 1u) && cj < c) ++pos;  // kept ids are distinct
  }
  if (keep) klist[key * a.k + pos] = c;
  if (lane == 0) {
    cnt[key] = __builtin_popcountll(kept);
    if (kept) atomicAdd(n_groups, 1);
  }
}

struct CountOp {
  const int64_t* cnt;
  __device__ int64_t operator()(int64_t i) const { return cnt[i]; }
};

// Relocation copies: unit u (kMoveUnits per workgroup) is page u % ppc of
// moved chunk u / ppc, taken in (key, time) order; it goes to page
// next_free + u, and its directory entry follows.  An entry outside
// [0, n_pages) is not read: its fresh page is written as zeros.
__global__ __launch_bounds__(kMoveThreads) void reloc_move_kernel(u32x4* __restrict__ pool, int64_t page_vecs,
                                                                  int32_t* __restrict__ table, int ppc,
                                                                  const int32_t* __restrict__ klist, int k,
                                                                  const int64_t* __restrict__ kbase, int64_t m,
                                                                  int64_t next_free, int64_t n_units,
                                                                  int64_t n_pages) {
  __shared__ int32_t s_old[kMoveUnits];
  __shared__ int64_t s_entry[kMoveUnits];
  const int64_t u0 = static_cast<int64_t>(blockIdx.x) * kMoveUnits;
  const int h0 = threadIdx.x;
  if (h0 < kMoveUnits && u0 + h0 < n_units) {
    const int64_t t = (u0 + h0) / ppc;  // moved chunk
    const int p = static_cast<int>((u0 + h0) % ppc);
    int64_t lo = 0, hi = m - 1;  // last key with kbase <= t
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (kbase[mid] <= t) lo = mid; else hi = mid - 1;
    }
    const int32_t c = klist[lo * k + (t - kbase[lo])];
    s_entry[h0] = static_cast<int64_t>(c) * ppc + p;
    s_old[h0] = table[s_entry[h0]];
  }
  __syncthreads();
  int64_t src[kMoveUnits], dst[kMoveUnits];
  bool live[kMoveUnits];
#pragma unroll
  for (int h = 0; h < kMoveUnits; ++h) {
    live[h] = u0 + h < n_units;
    src[h] = (live[h] && s_old[h] >= 0 && s_old[h] < n_pages) ? s_old[h] : -1;
    dst[h] = next_free + u0 + h;
  }
  copy_pages(pool, page_vecs, src, dst, live);
#pragma unroll
  for (int h = 0; h < kMoveUnits; ++h)
    if (threadIdx.x == h && live[h]) table[s_entry[h]] = static_cast<int32_t>(dst[h]);
}


// A plan's results for the host, gathered so that one copy brings them back:
// out = the int64 values at t.s64[0 .. n64), then the int32 values at
// t.s32[0 .. n32).
struct TotalsSrc {
  const int64_t* s64[2];
  const int32_t* s32[2];
};
__global__ __launch_bounds__(64) void totals_kernel(TotalsSrc t, int n64, int n32, int64_t* __restrict__ out) {
  if (threadIdx.x != 0) return;
  for (int i = 0; i < n64; ++i) out[i] = *t.s64[i];
  for (int j = 0; j < n32; ++j) out[n64 + j] = *t.s32[j];
}

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
  L.flags = o;   o += al(8);
  L.totals = o;  o += al(4 * 8);
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
  auto* bad = reinterpret_cast<int32_t*>(w + L.flags);
  fill_i32_kernel<<<1, 256, 0, stream>>>(bad, 1, 0);
  if (n_ns > 0) {
    const int64_t span = (a.n_elems / ppc > n_ns + 1) ? a.n_elems / ppc : n_ns + 1;
    check_tables_kernel<<<blocks256(span), 256, 0, stream>>>(a, bad);
  }
  if (a.n_elems > 0) live_kernel<<<blocks256(a.n_elems), 256, 0, stream>>>(a, live);
  if (L.n_blocks > 0)
    phi_kernel<<<blocks256(L.n_blocks), 256, 0, stream>>>(live, L.n_blocks, P, next_free, theta, cand, phi_out,
                                                          released, n_cand);
  hipError_t e = exclusive_scan(MovingOp{a}, a.n_elems, bsum, pos, stream);
  if (e != hipSuccess) return e;
  e = exclusive_scan(PaddedOp{a}, n_ns, bsum, ns_base, stream);
  if (e != hipSuccess) return e;
  // totals: moving pages, fresh pages (namespaces rounded to blocks),
  // compacted blocks and the malformed-table flag, in one copy
  auto* out = reinterpret_cast<int64_t*>(w + L.totals);
  totals_kernel<<<1, 64, 0, stream>>>(TotalsSrc{{pos + a.n_elems, ns_base + n_ns}, {n_cand, bad}}, 2, 2, out);
  e = hipMemcpyAsync(totals_host, out, 4 * sizeof(int64_t), hipMemcpyDeviceToHost, stream);
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
  move_kernel<<<dim3(static_cast<unsigned>((moved + kMoveUnits - 1) / kMoveUnits)), kMoveThreads, 0, stream>>>(
      static_cast<u32x4*>(pool), page_bytes / 16, table, moves, moved);
  return hipGetLastError();
}

ColocLayout coloc_layout(int64_t m, int32_t k, int64_t n_chunks) {
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  ColocLayout L{};
  const int64_t nb = (m + kScanBlock - 1) / kScanBlock + 1;
  size_t o = 0;
  L.owner = o;  o += al(static_cast<size_t>(n_chunks > 0 ? n_chunks : 1) * 4);
  L.klist = o;  o += al(static_cast<size_t>(m * k > 0 ? m * k : 1) * 4);
  L.cnt = o;    o += al(static_cast<size_t>(m > 0 ? m : 1) * 8);
  L.kbase = o;  o += al(static_cast<size_t>(m + 1) * 8);
  L.bsum = o;   o += al(static_cast<size_t>(nb + 1) * 8);
  L.counter = o; o += al(8);
  L.totals = o;  o += al(2 * 8);
  L.bytes = o;
  return L;
}

hipError_t launch_coloc_plan(const ColocLayout& L, const int32_t* ids, const float* scores, int64_t m, int32_t k,
                             double tau, int32_t min_group, int64_t n_chunks, void* ws, int64_t* totals_host,
                             hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* owner = reinterpret_cast<int32_t*>(w + L.owner);
  auto* klist = reinterpret_cast<int32_t*>(w + L.klist);
  auto* cnt = reinterpret_cast<int64_t*>(w + L.cnt);
  auto* kbase = reinterpret_cast<int64_t*>(w + L.kbase);
  auto* bsum = reinterpret_cast<int64_t*>(w + L.bsum);
  auto* n_groups = reinterpret_cast<int32_t*>(w + L.counter);
  ColocArgs a{ids, scores, m, k, tau, min_group, n_chunks};
  fill_i32_kernel<<<blocks256(n_chunks), 256, 0, stream>>>(owner, n_chunks, kNoOwner);
  fill_i32_kernel<<<1, 256, 0, stream>>>(n_groups, 1, 0);
  const unsigned grid = static_cast<unsigned>((m + 3) / 4 > 0 ? (m + 3) / 4 : 1);
  if (m > 0) {
    claim_kernel<<<grid, 256, 0, stream>>>(a, owner);
    keep_kernel<<<grid, 256, 0, stream>>>(a, owner, klist, cnt, n_groups);
  }
  hipError_t e = exclusive_scan(CountOp{cnt}, m, bsum, kbase, stream);
  if (e != hipSuccess) return e;
  // moved chunks and groups, in one copy
  auto* out = reinterpret_cast<int64_t*>(w + L.totals);
  totals_kernel<<<1, 64, 0, stream>>>(TotalsSrc{{kbase + m, nullptr}, {n_groups, nullptr}}, 1, 1, out);
  e = hipMemcpyAsync(totals_host, out, 2 * sizeof(int64_t), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(stream);
}

hipError_t launch_coloc_move(const ColocLayout& L, void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table,
                             int32_t ppc, int64_t m, int32_t k, int64_t next_free, int64_t moved, void* ws,
                             hipStream_t stream) {
  if (moved == 0) return hipSuccess;
  char* w = static_cast<char*>(ws);
  const int64_t units = moved * ppc;
  reloc_move_kernel<<<dim3(static_cast<unsigned>((units + kMoveUnits - 1) / kMoveUnits)), kMoveThreads, 0, stream>>>(
      static_cast<u32x4*>(pool), page_bytes / 16, table, ppc, reinterpret_cast<const int32_t*>(w + L.klist), k,
      reinterpret_cast<const int64_t*>(w + L.kbase), m, next_free, units, n_pages);
  return hipGetLastError();
}

}  // namespace memattn
