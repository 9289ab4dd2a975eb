// Matrix-core selection path (bf16 embeddings, fp32 accumulation) for gfx950.
//
// Dense-only relevance (Section 5.5) applied to LLMSelect of Algorithm 1:
// s_ij = <q_i, b_j> for a 256-query tile against a split of the bank,
// 256 bank rows per step, fused with the softmax normaliser and a per-query
// running top-k; the score matrix never leaves registers.
//
// Workgroup (main shape): 8 waves (two per SIMD), 256 queries x 256 bank
// rows per step; narrower shapes for fewer queries are described at Shape.
// Wave w owns bank rows [128h, 128h+128) (h = w & 1) and queries
// [64u, 64u+64) (u = w >> 1), i.e. 4 x 2 blocks of v_mfma_f32_32x32x16_bf16
// with the bank tile as the A operand (rows) and the queries as the B operand
// (columns), so each accumulator lane holds one query column.  With two waves
// per SIMD, one wave's load issue or epilogue overlaps the other's MFMAs.  K
// is staged through LDS 32 elements at a time in a ring of four stage buffers
// filled by direct-to-LDS buffer loads issued three stages ahead (across tile
// boundaries) and interleaved with the MFMAs; the fragment reads of one
// k-step overlap the MFMAs of the previous one.  Staged rows are 64 B with an
// XOR swizzle of their 16-byte chunks so fragment reads are bank-conflict
// free.
//
// Epilogue (per bank tile, per 16-row half block): lanes l and l^32 exchange
// (v_permlane32_swap) the rows that belong to the other's query, so lane L
// then owns query L of its wave with every row of the wave's half tile.  The
// lane keeps
//   - (M, sum): running max of x = scale*log2e*s and sum exp2(x - M);
//   - a sorted list of its query's best KCAP keys (score desc, id asc) among
//     its half of the split's rows, in its own partial-output slot of the
//     workspace, with T = the list's last score in a register as a filter.
// Scores above T are appended to a lane-private LDS stash of 8 entries; only
// when some lane's stash would overflow (and once at the end) is the list
// loaded into registers, the stash inserted (the wave runs as many insertion
// rounds as its busiest lane needs) and the list stored back.  After the
// first tiles T is high and merges are rare.  At the end the waves that
// share a query combine their lists and (M, sum) through LDS, so the merge
// kernel sees one partial per split.
//
// Modes (template flags): SAMPLE scores only the first tiles of sampled
// splits and writes 16-bit score keys (a lower bound on each query's k-th
// best comes from them); SCOPED masks rows outside the query's namespace and
// tombstoned rows; GROUPED takes (namespace, query tile, split) work items
// and gathers the rows of the namespace's chunk table.
#include <type_traits>

#include "device_common.h"
#include "launch.h"
#include "scan.h"

namespace memattn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBK = 32;                       // K elements per stage
constexpr int kRowVec = kBK / 8;              // 16-byte chunks per staged row
constexpr int kRing = 4;                      // LDS stage buffers (loads run kRing - 1 stages ahead)
constexpr int kWaveRows = 128;                // bank rows per wave and tile
constexpr int kBlk = kWaveRows / 32;          // 32-row MFMA blocks per wave
constexpr int kHalfBlocks = kWaveRows / 16;   // 16-row epilogue half blocks per wave
static_assert(kRing >= 3, "the pipeline needs three stage buffers");

// Workgroup shape.  Every wave scores 128 bank rows of a tile against 64
// queries; QW query groups of 64 and BW = kWaves / QW bank parts per tile.
//   QW = 4 (wide): 8 waves (two per SIMD), 256 queries x 256 bank rows;
//   QW = 2: 4 waves, 128 queries x 256 rows (65 to 128 queries);
//   QW = 1 (narrow): 4 waves, 64 queries x 512 rows (at most 64 queries),
//   so a few queries do not pay for a 256-query tile.
template <int QW>
struct Shape {
  static_assert(QW == 1 || QW == 2 || QW == 4, "64, 128 or 256 queries per workgroup");
  static constexpr int kWaves = QW == 4 ? 8 : 4;
  static constexpr int kWavesPerEU = kWaves / 4;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int kBW = kWaves / QW;                 // bank parts per tile (partials per split)
  static constexpr int kTileB = kWaveRows * kBW;          // bank rows per tile
  static constexpr int kTileQ = 64 * QW;                  // queries per workgroup
  static constexpr int kStageRows = kTileB + kTileQ;      // staged rows: bank rows, then query rows
  static constexpr int kStageVec = kStageRows * kRowVec;  // 16-byte chunks per stage
  static constexpr int kRowsPerWave = kStageRows / kWaves;
  static constexpr int kLoads = kRowsPerWave / 16;        // 16-row loads per wave and stage
  static constexpr int kLoads0 = (kLoads + 1) / 2;        // of which issued during k-step 0
  static constexpr int kCap = 8;                          // stash entries per lane
  static constexpr int kGroup = kCap < 16 ? kCap : 16;    // scores offered to the stash at a time
  static_assert(kRowsPerWave % 16 == 0 && kTileB % 16 == 0, "loads cover whole 16-row blocks");
  static_assert(kRing * kStageVec * 16 + kCap * kThreads * 8 <= 160 * 1024, "fits the 160 KiB of LDS");
};
static_assert(Shape<4>::kTileB == kMfmaTile && Shape<4>::kTileQ == kMfmaTile, "wide shape matches the plan");
static_assert(Shape<1>::kTileB == 512 && Shape<2>::kTileB == 256, "tile rows as in the plan");
// Buffer descriptor word 3 for raw (untyped) buffer loads on gfx950.
constexpr int kBufferFlags = 0x00020000;

// LDS chunk slot of 16-byte chunk c of staged row `row`.  The XOR swizzle
// makes the fragment reads (8 or 16 consecutive lanes = consecutive rows,
// same chunk) and the staging writes (4 chunks of 2 or 4 consecutive rows)
// hit distinct LDS banks with 64-byte rows.
__device__ __forceinline__ int slot(int row, int c) { return row * kRowVec + (c ^ (((row >> 1) ^ (row >> 2)) & 3)); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Byte offset of a __shared__ object within the workgroup's LDS allocation.
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) void*)p));
}

// Direct-to-LDS 16-byte buffer load: lane l's 16 bytes at byte offset
// voffset + soffset of the descriptor's range land at LDS byte address
// lds_addr + 16 * l (out-of-range lanes land zeros).  Issued through inline
// assembly so that the compiler, which does not see these LDS writes, adds
// no conservative waits; the kernel orders them itself with stage_barrier()
// and wait_all_loads().  M0 is written here without a clobber (the compiler
// reserves it); no compiler-generated code of this file reads or writes M0,
// which a host test checks in the generated assembly.
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t rsrc, uint32_t voffset, int soffset,
                                          uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voffset), "s"(rsrc), "s"(__builtin_amdgcn_readfirstlane(soffset)),
                 "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory");
}
// The same with the non-temporal hint: the line is marked for early
// eviction once read.
__device__ __forceinline__ void lds_dma16_nt(__amdgpu_buffer_rsrc_t rsrc, uint32_t voffset, int soffset,
                                             uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %3\n\tbuffer_load_dwordx4 %0, %1, %2 offen nt lds"
               :
               : "v"(voffset), "s"(rsrc), "s"(__builtin_amdgcn_readfirstlane(soffset)),
                 "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory");
}
// End of a stage: this wave's loads of the next stage have landed (at most
// the newest N of its loads, all for later stages, may still be in flight),
// its LDS reads are done, then the workgroup meets.
template <int N>
__device__ __forceinline__ void stage_barrier() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_all_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Grouped selection: where the work items, chunk tables and grouped queries
// are (all device memory).
struct GroupArgs {
  const int32_t* ns_off;    // [n_ns + 1] chunk-table entry offsets
  const int64_t* q_off;     // [n_ns + 1] grouped-query offsets
  const int64_t* item_off;  // [n_ns + 1] work-item offsets
  const int32_t* perm;      // grouped (or, whole-bank selection, clustered) position -> query index
  int n_ns;
  int S;                    // splits per namespace
  uint32_t bank_bytes;      // bytes of the bank seen by the descriptor (< 2^32)
  int64_t n_entries;        // table entries (offsets are clamped to [0, n_entries])
};

// Which tiles of its split a full-pass launch covers, and how it starts
// and ends.  A split may be scored in two launches: the first covers its
// first tiles and leaves each lane's list (in the workspace) and softmax
// state (lane_ms) behind; the second resumes from them with a tighter bound
// on every query's k-th best score and, being final, combines the parts.
struct PhaseArgs {
  int lo, hi;       // tile offsets within the split: [lo, min(hi, tiles_per_split))
  int resume;       // start from the list and softmax state a previous launch left
  int final_pass;   // combine the bank parts and write the split's partials
  float2* lane_ms;  // per-slot (max, sum) state between launches
};
constexpr PhaseArgs kWholeSplit{0, 0x7FFFFFFF, 0, 1, nullptr};

// A wave-uniform 64-bit value moved to scalar registers (values loaded from
// memory at a uniform address may sit in vector registers).
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(x) >> 32));
  return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// Bubble key x into a descending list; returns the key pushed out of the end.
template <int N>
__device__ __forceinline__ uint64_t list_insert(uint64_t (&list)[N], uint64_t x) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const uint64_t a = list[i];
    const bool gt = x > a;
    list[i] = gt ? x : a;
    x = gt ? a : x;
  }
  return x;
}

// Scores of half block hb (rows 16*hb .. 16*hb+15 of the wave's 128 rows) for the
// query this lane owns, in row order.  Before the exchange, lane l holds rows
// {8*(r/4) + 4*(l/32) + r%4} of both query blocks (qb = 0, 1).
// v_permlane32_swap(x, y) returns (x in lanes 0-31 | y's lanes 0-31 in lanes
// 32-63, x's lanes 32-63 in lanes 0-31 | y in lanes 32-63); with x = qb 0 and
// y = qb 1 every lane L receives query L's rows of half 0 in the first result
// and of half 1 in the second.  With hb a compile-time constant every
// accumulator index is static.
__device__ __forceinline__ void extract_half(const f32x16 (&acc)[kBlk][2], int hb, float (&v)[16]) {
  const int blk = hb >> 1;
  const int r0 = (hb & 1) * 8;
#pragma unroll
  for (int rr = 0; rr < 8; ++rr) {
    const int r = r0 + rr;
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[blk][0][r]),
                                                     __float_as_uint(acc[blk][1][r]), false, false);
    const int j0 = (r >> 2) * 8 + (r & 3) - (hb & 1) * 16;
    v[j0] = __uint_as_float(sw[0]);
    v[j0 + 4] = __uint_as_float(sw[1]);
  }
}

// SAMPLE = true: score only the first `ns` tiles of each split and write
// every score, rounded down to a 16-bit order key, to samp[q][n_samp]; the
// k-th largest of a query's sample is then a lower bound on its k-th best
// score over the whole bank.  SAMPLE = false: the full pass, with each
// query's list threshold starting at that bound t0[q] (inclusive).
// SCOPED = true: row j is a candidate of query q only if row_ns[j] >= 0 (a
// live row) and row_ns[j] == key_ns[q] (the query's namespace); other rows
// score -inf, which keeps them out of the softmax, the sample and the lists.
// GROUPED = true: the workgroup takes one work item (namespace u, 64-query
// tile of u's queries, split of u's chunk table): it scores only the bank
// rows listed in u's chunk table (gathered through per-lane load offsets)
// against queries grouped by namespace (`queries` then holds them in
// grouped order, g.perm maps a grouped position to the query's index).
template <int KCAP, bool SAMPLE, int QW, bool SCOPED, bool GROUPED>
__global__ __attribute__((amdgpu_flat_work_group_size(Shape<QW>::kThreads, Shape<QW>::kThreads),
                          amdgpu_waves_per_eu(Shape<QW>::kWavesPerEU, Shape<QW>::kWavesPerEU))) void
topk_mfma_kernel(const uint16_t* __restrict__ bank, int64_t bank_stride, int64_t n,
                 const uint16_t* __restrict__ queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                 int64_t self_base, int q_tiles, int n_splits, int tiles_per_split,
                 uint64_t* __restrict__ part_keys, float2* __restrict__ part_ms, int ns, int samp_stride,
                 uint16_t* __restrict__ samp, int64_t n_samp, const float* __restrict__ t0_in,
                 uint32_t* __restrict__ thr_shared, const int32_t* __restrict__ row_ns,
                 const int32_t* __restrict__ key_ns, const int32_t* __restrict__ grows, GroupArgs g,
                 PhaseArgs ph) {
  using S = Shape<QW>;
  constexpr int kThreads = S::kThreads;
  constexpr int kTileB = S::kTileB;
  constexpr int kTileQ = S::kTileQ;
  constexpr int kStageVec = S::kStageVec;
  constexpr int kLoadsPerWave = S::kLoads;
  constexpr int kCap = S::kCap;
  constexpr int kGroup = S::kGroup;
  __shared__ u32x4 tiles[kRing][kStageVec];      // 128 KiB (wide) / 144 KiB (narrow)
  __shared__ uint64_t stash[kCap * kThreads];     // 32 KiB / 16 KiB

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = wave % S::kBW;  // bank part: rows [128 half, 128 half + 128) of every tile
  const int qsub = wave / S::kBW;  // queries [64 qsub, 64 qsub + 64) of the query tile

  // XCD-aware placement: workgroups b, b+8, b+16, ... run on one XCD; give
  // consecutive logical ids (the query tiles of one bank split) to one XCD
  // so the split's bank tiles are shared through that XCD's L2.  Grouped
  // items keep the launch order: their grid is an upper bound whose unused
  // tail exits at once, and remapping would pile that tail onto the last
  // XCD while the others run an extra round of real items.
  // Where the query tiles are a multiple of 8 (a relation build's 128, the
  // streaming rounds' 16), an XCD instead takes q_tiles / 8 query tiles with
  // every split of each: a tile's workgroups then read the same query rows
  // at about the same time and share them through L2 as well.
  const int G = gridDim.x;
  const int b = blockIdx.x;
  int L = (!GROUPED && G % 8 == 0) ? (b % 8) * (G / 8) + b / 8 : b;
  if (!GROUPED && !SAMPLE && G % 8 == 0 && q_tiles % 8 == 0 && G % q_tiles == 0) {
    const int sp = G / q_tiles;  // splits in this launch
    const int i = b / 8;         // position on the XCD
    L = (i % sp) * q_tiles + (b % 8) * (q_tiles / 8) + i / sp;
  }
  // the sample pass runs one workgroup per query tile and sampled split
  int samp_slot, split;
  int64_t seg_lo = 0, seg_n = n;  // scanned rows: the bank, or (grouped) entries of one chunk table
  int64_t q_base, q_lim;          // first query of the tile and queries in it
  int64_t tps = tiles_per_split;
  if constexpr (GROUPED) {
    // work item L: namespace u = the last with item_off[u] <= L (items past
    // the total exit here, before any barrier)
    if (L >= uniform64(g.item_off[g.n_ns])) return;
    int lo = 0, hi = g.n_ns - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform64(g.item_off[mid]) <= L) lo = mid; else hi = mid - 1;
    }
    lo = __builtin_amdgcn_readfirstlane(lo);
    const int64_t local = L - uniform64(g.item_off[lo]);
    const int qt = static_cast<int>(local / g.S);
    samp_slot = split = static_cast<int>(local % g.S);
    // the sample pass scores the first tile of each table: split 0's items
    if (SAMPLE && split != 0) return;
    // (offsets are clamped so a malformed table cannot send reads past it)
    seg_lo = min(max(static_cast<int64_t>(__builtin_amdgcn_readfirstlane(g.ns_off[lo])), int64_t{0}), g.n_entries);
    const int64_t seg_end =
        min(max(static_cast<int64_t>(__builtin_amdgcn_readfirstlane(g.ns_off[lo + 1])), seg_lo), g.n_entries);
    seg_n = seg_end - seg_lo;
    const int64_t qg0 = uniform64(g.q_off[lo]);
    q_base = qg0 + static_cast<int64_t>(qt) * kTileQ;
    q_lim = min(static_cast<int64_t>(kTileQ), uniform64(g.q_off[lo + 1]) - q_base);
    q_base = uniform64(q_base);
    q_lim = uniform64(q_lim);
    const int64_t seg_tiles = (seg_n + kTileB - 1) / kTileB;
    tps = (seg_tiles + g.S - 1) / g.S;
  } else {
    const int qt = L % q_tiles;
    samp_slot = L / q_tiles;
    split = SAMPLE ? samp_slot * samp_stride : samp_slot;
    q_base = static_cast<int64_t>(qt) * kTileQ;
    q_lim = min(static_cast<int64_t>(kTileQ), m - q_base);
  }
  const int64_t n_tiles = (seg_n + kTileB - 1) / kTileB;
  const int64_t split_t0 = static_cast<int64_t>(split) * tps;
  const int64_t t0 = split_t0 + ph.lo;
  // A sample pass always covers `ns` tiles per split; tiles past the bank
  // read as zeros and are masked, so every sample slot is written.
  const int64_t t1 = SAMPLE ? t0 + ns : max(t0, min(n_tiles, split_t0 + min(tps, static_cast<int64_t>(ph.hi))));
  const int nk = d / kBK;
  // Stage s (0 <= s < n_stages) = one k-block of bank tile t0 + s / nk.
  const int64_t n_stages = (t1 - t0) * nk;

  // Global -> LDS staging by direct-to-LDS buffer loads.  Wave w moves stage
  // rows [R w, R w + R) (R = kRowsPerWave; stage rows 0 .. kTileB-1 are bank
  // rows, the rest query rows), 16 rows per instruction; lane l lands at LDS
  // chunk slot l of the instruction's 16-row block, i.e. row (l >> 2),
  // physical chunk l & 3, which holds logical chunk (l & 3) ^ swizzle(row)
  // (the swizzle depends on row bits 1-3 only, the same for every block).
  // Descriptors end at the last valid row, so rows past n (or m) land as
  // zeros.  Offsets are 32-bit (a tile spans at most 512 rows of at most
  // 64 Ki elements).
  const int wrow0 = S::kRowsPerWave * wave;  // first stage row of this wave
  const int lrow = lane >> 2;
  const int lchunk = (lane & 3) ^ (((lrow >> 1) ^ (lrow >> 2)) & 3);
  const uint32_t voff_b = static_cast<uint32_t>((lrow * bank_stride + lchunk * 8) * 2);
  const uint32_t voff_q = static_cast<uint32_t>((lrow * q_stride + lchunk * 8) * 2);
  // LDS byte address of this wave's first 16-row block in ring slot 0
  const uint32_t lds_block =
      __builtin_amdgcn_readfirstlane(lds_offset(&tiles[0][0]) + static_cast<uint32_t>(wrow0) * (kRowVec * 16));
  const int q_rows = static_cast<int>(q_lim);
  const __amdgpu_buffer_rsrc_t q_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(queries + q_base * q_stride), 0, static_cast<int>(q_rows * q_stride * 2), kBufferFlags);
  // Loads of the stage (ld_tile, ld_kb) into ring slot ld_slot = stage %
  // kRing: issue_load(i) moves the wave's rows [16i, 16i + 16); next_stage()
  // advances to the following stage.  Stages past the last re-read the last
  // one (into their own free slot), so every stage issues the same number of
  // loads and the vmcnt arithmetic stays exact.  The row offset goes into the
  // per-lane offset and only the column offset into the scalar one, so the
  // descriptor's range check sees each row's own offset whether or not it
  // counts the scalar offset.
  int64_t ld_tile = t0;
  int ld_kb = 0;
  int ld_slot = 0;
  int ld_dir = 1;  // k-block direction of the tile being loaded (see next_stage)
  auto bank_rsrc = [&]() {
    const int b_rows = static_cast<int>(max(int64_t{0}, min(static_cast<int64_t>(kTileB), n - ld_tile * kTileB)));
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(bank + ld_tile * kTileB * bank_stride), 0,
                                             static_cast<int>(b_rows * bank_stride * 2), kBufferFlags);
  };
  __amdgpu_buffer_rsrc_t ld_rsrc = GROUPED ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(bank), 0,
                                                                                static_cast<int>(g.bank_bytes),
                                                                                kBufferFlags)
                                           : bank_rsrc();
  // Grouped: byte offset of the lane's row for each of the wave's bank loads
  // of tile ld_tile (lane l loads row l >> 2 of the load's 16), and the same
  // for the tile after it.  Each lane reads its own row ids, for tile
  // ld_tile + 1 at the start of every compute tile (outside the k loop); the
  // compiler's wait for those reads, at the tile change, also waits for the
  // staging loads issued before it (loads complete in order): one drain per
  // tile.  The loads run at most one tile ahead because a tile has at least
  // 3 k-blocks (the host requires d >= 96).  Rows past the chunk table or
  // outside the bank get an offset past the descriptor's range, so they land
  // as zeros.
  uint32_t gvoff[kLoadsPerWave], gnext[kLoadsPerWave];
  auto tile_offsets = [&](int64_t t, uint32_t (&o)[kLoadsPerWave]) {
#pragma unroll
    for (int i = 0; i < kLoadsPerWave; ++i) {
      const int r0 = wrow0 + 16 * i;
      o[i] = 0xFFFFFFF0u;
      if (r0 < kTileB) {
        const int64_t e = t * kTileB + r0 + lrow;  // the lane's table entry
        const int32_t rid = e < seg_n ? grows[seg_lo + e] : -1;
        if (rid >= 0 && rid < n)
          o[i] = static_cast<uint32_t>(rid) * static_cast<uint32_t>(bank_stride * 2) + static_cast<uint32_t>(lchunk * 16);
      }
    }
  };
  if constexpr (GROUPED) {
    tile_offsets(t0, gvoff);
    tile_offsets(t0 + 1, gnext);
  }
  auto issue_load = [&](int i) {
    const int r0 = wrow0 + 16 * i;  // first stage row of this load (uniform)
    const uint32_t lds = lds_block + static_cast<uint32_t>(ld_slot) * (kStageVec * 16) +
                         static_cast<uint32_t>(i * 16 * kRowVec * 16);
    // bank or query rows: a uniform choice, made with selects rather than a branch
    const bool is_bank = r0 < kTileB;
    const __amdgpu_buffer_rsrc_t rsrc = is_bank ? ld_rsrc : q_rsrc;
    uint32_t voff_bank;
    if constexpr (GROUPED) {
      voff_bank = gvoff[i];
    } else {
      voff_bank = voff_b + static_cast<uint32_t>(r0 * bank_stride * 2);
    }
    const uint32_t voff = is_bank ? voff_bank : voff_q + static_cast<uint32_t>((r0 - kTileB) * q_stride * 2);
    // With at most 64 queries (one query tile) no other workgroup reads a
    // bank line, and the two 64-byte halves of a row's 128-byte line are
    // read one stage apart: the read of the second half marks the line for
    // early eviction, so that it does not push out lines whose second half
    // is still to come (the full pass over the 1M bank 10 us faster for 64
    // queries; with several query tiles the line's other readers would
    // miss, and the short sample pass gains nothing).
    if constexpr (QW == 1 && !GROUPED && !SAMPLE) {
      if (is_bank && (((ld_kb & 1) != 0) == (ld_dir > 0))) {
        lds_dma16_nt(rsrc, voff, ld_kb * kBK * 2, lds);
        return;
      }
    }
    lds_dma16(rsrc, voff, ld_kb * kBK * 2, lds);
  };
  // K-blocks run up in one tile and down in the next, so the query columns
  // read last in a tile are read first in the next one, while still in L2
  // (the accumulation order differs between tiles; every score is still a
  // full fp32 dot product).
  auto next_stage = [&]() {
    ld_slot = ld_slot + 1 == kRing ? 0 : ld_slot + 1;
    const int nkb = ld_kb + ld_dir;
    if (nkb >= 0 && nkb < nk) {
      ld_kb = nkb;
    } else if (ld_tile + 1 < t1) {
      ld_dir = -ld_dir;
      ++ld_tile;
      if constexpr (GROUPED) {
#pragma unroll
        for (int i = 0; i < kLoadsPerWave; ++i) gvoff[i] = gnext[i];
      } else {
        ld_rsrc = bank_rsrc();
      }
    }
  };

  const bool q_valid = qsub * 64 + lane < q_lim;
  int64_t my_q = q_base + qsub * 64 + lane;  // the query this lane owns
  // queries held in grouped or clustered order: g.perm maps the position to
  // the query's index, which keys everything the lane reads and writes
  if (GROUPED || g.perm != nullptr) my_q = q_valid ? g.perm[my_q] : 0;
  // the query's own bank row (relation build), -1 if none; bank rows fit in
  // int32 (n < 2^31 - 1)
  const int32_t self_row = (!GROUPED && self_base >= 0) ? static_cast<int32_t>(self_base + my_q) : -1;
  // the query's namespace (scoped selection); padding lanes match no row
  int32_t my_ns = -1;
  if constexpr (SCOPED) {
    my_ns = q_valid ? key_ns[my_q] : -1;
    my_ns = my_ns < 0 ? -1 : my_ns;
    asm volatile("" ::"v"(my_ns));  // consumed before the staging loads start
  }
  // partial-output slot of (query, split, half); the merge sees 2 per split
  const int64_t out_slot = (my_q * n_splits + split) * S::kBW + half;
  // The lane's sorted list of its query's best KCAP keys lives in its partial
  // output slot in the workspace; it is read and written only at merges.
  if (!SAMPLE && q_valid && !ph.resume) {
#pragma unroll
    for (int i = 0; i < KCAP; ++i) part_keys[out_slot * KCAP + i] = 0;
  }
  // Scores > thr are kept.  thr starts a little below the sampled lower bound
  // on the query's k-th best score (so scores equal to the bound are kept;
  // the margin only admits a few extra candidates, which the list's exact
  // key comparisons then sort out) and rises to the list's last score; within
  // a lane, rows arrive in ascending order, so a later score equal to the
  // list's last one is the worse of the two and is rightly dropped.  Padding
  // lanes (query >= m) keep nothing.
  float thr;
  float run_m = -INFINITY;
  float run_s = 0.f;
  {
    const float t0v = (!SAMPLE && t0_in != nullptr && q_valid) ? t0_in[my_q] : -INFINITY;
    thr = !q_valid ? INFINITY : t0v - (fabsf(t0v) * 1e-6f + 1e-30f);
    // A resumed lane continues from its list (the rows of this launch come
    // after the list's rows, so the list's last score is a strict bound)
    // and from its softmax state.
    if (!SAMPLE && ph.resume && q_valid) {
      const uint64_t last = part_keys[out_slot * KCAP + KCAP - 1];
      if (last != 0) thr = fmaxf(thr, key_score(last));
      const float2 st = ph.lane_ms[out_slot];
      run_m = st.x;
      run_s = st.y;
    }
    // consume the loads here, before any staging load is in flight, so their
    // wait does not also wait for those
    asm volatile("" ::"v"(thr), "v"(run_m), "v"(run_s));
  }
  int cnt = 0;  // stash entries of this lane
  // Insert the stash into the lane's list and raise the threshold.  The list
  // is processed in chunks of up to 16 keys to bound register use: each stash
  // key bubbles through a chunk and the key it pushes out replaces it in the
  // stash, to be offered to the next chunk -- the same result as one bubble
  // pass over the whole list.  The wave runs as many rounds as its busiest
  // lane needs.
  //
  // Every partial of a query (all splits and both halves) also shares its
  // list's last score through thr_shared[q] (an atomic max of order keys):
  // each published score is the k-th best of a subset of the bank, hence a
  // lower bound on the query's k-th best overall, so rows scoring below it
  // cannot be selected.  A row scoring exactly the bound may still win on
  // its lower index, so the shared bound is applied inclusively (the filter
  // keeps v > the next float below it).  Stale reads are still valid bounds.
  auto merge = [&]() {
    constexpr int CH = KCAP < 16 ? KCAP : 16;
    uint64_t* lst = part_keys + out_slot * KCAP;
    uint32_t shared_ord =
        q_valid ? __hip_atomic_load(thr_shared + my_q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
    uint64_t last = 0;
#pragma unroll
    for (int c0 = 0; c0 < KCAP; c0 += CH) {
      uint64_t chunk[CH];
#pragma unroll
      for (int i = 0; i < CH; ++i) chunk[i] = q_valid ? lst[c0 + i] : 0;
      for (int r = 0; __ballot(r < cnt) != 0; ++r) {
        if (r < cnt) stash[r * kThreads + tid] = list_insert<CH>(chunk, stash[r * kThreads + tid]);
      }
      if (q_valid) {
#pragma unroll
        for (int i = 0; i < CH; ++i) lst[c0 + i] = chunk[i];
      }
      last = chunk[CH - 1];
    }
    if (last != 0) {
      const uint32_t own = static_cast<uint32_t>(last >> 32);
      thr = fmaxf(thr, ord2f(own));
      if (q_valid && own > shared_ord) atomicMax(thr_shared + my_q, own);
    }
    if (shared_ord > 0) thr = fmaxf(thr, ord2f(shared_ord - 1));
    cnt = 0;
  };

  // MFMA operand fragments of one 16-deep k-step: the wave's 4 bank blocks
  // and 2 query blocks.
  const int frag_row = lane & 31;
  const int frag_part = lane >> 5;
  struct Frag {
    bf16x8 a[kBlk];
    bf16x8 b[2];
  };
  auto load_frags = [&](int slot_idx, int ks, Frag& f) {
    const u32x4* st = tiles[slot_idx];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
      f.b[qb] = as_bf16x8(st[slot(kTileB + qsub * 64 + qb * 32 + frag_row, ks * 2 + frag_part)]);
#pragma unroll
    for (int blk = 0; blk < kBlk; ++blk)
      f.a[blk] = as_bf16x8(st[slot(half * kWaveRows + blk * 32 + frag_row, ks * 2 + frag_part)]);
  };
  f32x16 acc[kBlk][2];
  // The 8 MFMAs of one k-step, with loads [first, first + cnt) of a later
  // stage issued right after the first MFMA block (early enough to run ahead
  // of the pipeline, late enough that the MFMA pipe is busy meanwhile).
  auto mma = [&](const Frag& f, int first, int cnt) {
#pragma unroll
    for (int blk = 0; blk < kBlk; ++blk) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        acc[blk][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[blk], f.b[qb], acc[blk][qb], 0, 0, 0);
      if (blk == 0 && cnt > 0) {  // compile-time after unrolling
#pragma unroll
        for (int i = 0; i < cnt; ++i) issue_load(first + i);
        __builtin_amdgcn_sched_barrier(0);  // keep the MFMAs on their side of the loads
      }
    }
  };

  // Software pipeline over stages (R = kRing slots, L = kLoadsPerWave):
  //   - the loads of stage s are issued during stage s-(R-1) into ring slot
  //     s % R, the first half during its k-step 0 MFMAs, the second half
  //     during its k-step 1 MFMAs after the barrier ending that stage; slot
  //     s % R was last read during stage s-R, which every wave finished
  //     before the barrier ending stage s-R;
  //   - before the barrier ending stage s, each wave waits until its loads of
  //     stage s+1 have landed: issued after them are the loads of stages
  //     s+2 .. s+R-2 and the first half of stage s+R-1, (R-3)L + L/2 loads
  //     ((R-2)L after the prologue's R-1 stages); its own LDS reads are done
  //     too;
  //   - k-step 1 fragments of a stage are read before its k-step 0 MFMAs, and
  //     k-step 0 fragments of the next stage right after the barrier (after
  //     the epilogue when the next stage starts a new tile).
  Frag f0, f1;
  // (the plan never produces an empty split; an empty one still writes its
  // empty partial list below)
  if (n_stages > 0) {
#pragma unroll 1
    for (int st = 0; st < kRing - 1; ++st) {
#pragma unroll
      for (int i = 0; i < kLoadsPerWave; ++i) issue_load(i);
      next_stage();
    }
    stage_barrier<(kRing - 2) * kLoadsPerWave>();
    int rd_slot = 0;  // ring slot of the current stage
    load_frags(rd_slot, 0, f0);

    for (int64_t tile = t0; tile < t1; ++tile) {
      if constexpr (GROUPED) tile_offsets(ld_tile + 1, gnext);
#pragma unroll
      for (int i = 0; i < kBlk; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
      }
      for (int kb = 0; kb < nk; ++kb) {
        const int nx_slot = rd_slot + 1 == kRing ? 0 : rd_slot + 1;
        load_frags(rd_slot, 1, f1);
        mma(f0, 0, S::kLoads0);
        stage_barrier<(kRing - 3) * kLoadsPerWave + S::kLoads0>();
        // (the next tile's first fragments are read after the epilogue, so
        // they do not occupy registers during it)
        if (kb + 1 < nk) load_frags(nx_slot, 0, f0);
        mma(f1, S::kLoads0, kLoadsPerWave - S::kLoads0);
        next_stage();
        rd_slot = nx_slot;
      }

      // ---------------- epilogue for bank tile `tile`, this wave's half
      const int32_t row_base = static_cast<int32_t>(tile * kTileB) + half * kWaveRows;
      // rows >= n (ragged tail) and the query's own row (relation build) are
      // removed from the candidates by setting their score to -inf
      const int lim = static_cast<int>(max(int64_t{0}, min(static_cast<int64_t>(kWaveRows), seg_n - row_base)));
      const int self_local = (self_row >= row_base && self_row < row_base + kWaveRows) ? self_row - row_base : -1;
      const bool mask_any = __ballot(lim < kWaveRows || self_local >= 0) != 0;
      // Half blocks are visited in a rolled loop; the switch keeps every
      // accumulator index static while bounding register live ranges.
      // Grouped: the bank row ids of half block hb (uniform, scalar loads);
      // -1 past the chunk table.
      auto load_rids = [&](int hb, int32_t (&rid)[16]) {
        const int64_t e0 = seg_lo + row_base + hb * 16;
        if (hb * 16 + 16 <= lim) {
#pragma unroll
          for (int j = 0; j < 16; ++j) rid[j] = grows[e0 + j];
        } else {
#pragma unroll
          for (int j = 0; j < 16; ++j) rid[j] = hb * 16 + j < lim ? grows[e0 + j] : -1;
        }
      };
      auto load_half = [&](int hb, float (&v)[16], const int32_t (&rid)[16]) {
        switch (hb) {
#define MEMATTN_HALF(H)        \
  case H:                      \
    extract_half(acc, H, v);   \
    break;
          MEMATTN_HALF(0) MEMATTN_HALF(1) MEMATTN_HALF(2) MEMATTN_HALF(3)
          MEMATTN_HALF(4) MEMATTN_HALF(5) MEMATTN_HALF(6) MEMATTN_HALF(7)
#undef MEMATTN_HALF
        }
        if (mask_any) {
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int jl = hb * 16 + j;
            if (jl >= lim || jl == self_local) v[j] = -INFINITY;
          }
        }
        if constexpr (SCOPED) {
          // the 16 rows of a half block are the same for every lane: their
          // namespaces come in through scalar loads, which do not wait
          // behind the staging loads in flight
          const int32_t r0 = row_base + hb * 16;
          int32_t rn[16];
          if (hb * 16 + 16 <= lim) {
#pragma unroll
            for (int j = 0; j < 16; ++j) rn[j] = row_ns[r0 + j];
          } else {
#pragma unroll
            for (int j = 0; j < 16; ++j) rn[j] = hb * 16 + j < lim ? row_ns[r0 + j] : -1;
          }
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            if (rn[j] < 0 || rn[j] != my_ns) v[j] = -INFINITY;
          }
        }
        if constexpr (GROUPED) {
          // a table entry outside the bank is not a candidate
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            if (rid[j] < 0 || rid[j] >= n) v[j] = -INFINITY;
          }
        }
      };
      static_assert(kHalfBlocks == 8, "switch above covers 8 half blocks");
      if constexpr (SAMPLE) {
        const int64_t base =
            my_q * n_samp + static_cast<int64_t>(samp_slot) * ns * kTileB + (tile - t0) * kTileB + half * kWaveRows;
#pragma unroll 1
        for (int hb = 0; hb < kHalfBlocks; ++hb) {
          float v[16];
          int32_t rid[16] = {};
          if constexpr (GROUPED) load_rids(hb, rid);
          load_half(hb, v, rid);
          if (q_valid) {
            uint32_t w[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = (f2ord(v[2 * j]) >> 16) | (f2ord(v[2 * j + 1]) & 0xFFFF0000u);
            u32x4* dst = reinterpret_cast<u32x4*>(samp + base + hb * 16);
            dst[0] = u32x4{w[0], w[1], w[2], w[3]};
            dst[1] = u32x4{w[4], w[5], w[6], w[7]};
          }
        }
        load_frags(rd_slot, 0, f0);
        continue;
      }
      // One pass over the half blocks: softmax normaliser, and scores above
      // the threshold appended to the stash (merged into the list only when
      // the stash would overflow, so a merge usually serves several tiles).
      // A half block's 16 scores are offered in groups of kGroup <= kCap, so
      // after a merge a group always fits the emptied stash.
#pragma unroll 1
      for (int hb = 0; hb < kHalfBlocks; ++hb) {
        float v[16];
        int32_t rid[16] = {};
        if constexpr (GROUPED) load_rids(hb, rid);
        load_half(hb, v, rid);
        float hm = v[0];
#pragma unroll
        for (int j = 1; j < 16; ++j) hm = fmaxf(hm, v[j]);
        // scoped: a half block holding no candidate of any of the wave's
        // queries adds nothing
        if ((SCOPED || GROUPED) && __ballot(hm != -INFINITY) == 0) continue;
        const float xm = hm * c2;
        if (xm > run_m) {
          run_s *= fast_exp2(run_m - xm);
          run_m = xm;
        }
        const float msafe = run_m == -INFINITY ? 0.f : run_m;
        float part = 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) part += fast_exp2(fmaf(v[j], c2, -msafe));
        run_s += part;

        if (__ballot(hm > thr) != 0) {
#pragma unroll
          for (int g8 = 0; g8 < 16; g8 += kGroup) {
            int c = 0;
#pragma unroll
            for (int j = 0; j < kGroup; ++j) c += v[g8 + j] > thr ? 1 : 0;
            if (__ballot(cnt + c > kCap) != 0) merge();
#pragma unroll
            for (int j = 0; j < kGroup; ++j) {
              if (v[g8 + j] > thr) {
                const uint32_t id = GROUPED ? static_cast<uint32_t>(rid[g8 + j])
                                            : static_cast<uint32_t>(row_base + hb * 16 + g8 + j);
                stash[cnt * kThreads + tid] = make_key(v[g8 + j], id);
                ++cnt;
              }
            }
          }
        }
      }
      load_frags(rd_slot, 0, f0);  // this stage (landed at the last barrier) starts the next tile
    }
  }
  // No load may still be writing LDS when the workgroup ends.
  wait_all_loads();
  if constexpr (!SAMPLE) {
    // The lane's final list: its list in the workspace with the stash merged
    // in, in registers (the accumulators are dead here), read with all its
    // loads in flight; the combine below takes it from here rather than
    // from the workspace.
    uint64_t fl[KCAP];
    {
      const uint64_t* lst = part_keys + out_slot * KCAP;
#pragma unroll
      for (int i = 0; i < KCAP; ++i) fl[i] = q_valid ? lst[i] : 0;
      for (int r = 0; __ballot(r < cnt) != 0; ++r) {
        if (r < cnt) (void)list_insert<KCAP>(fl, stash[r * kThreads + tid]);
      }
    }
    if (!ph.final_pass) {
      // (uniform: the whole workgroup leaves here) the next launch resumes
      // from the list, its last key and the softmax state
      if (q_valid) {
        uint64_t* lst = part_keys + out_slot * KCAP;
#pragma unroll
        for (int i = 0; i < KCAP; ++i) lst[i] = fl[i];
        const uint32_t own = static_cast<uint32_t>(fl[KCAP - 1] >> 32);
        if (own > 0) atomicMax(thr_shared + my_q, own);
        ph.lane_ms[out_slot] = make_float2(run_m, run_s);
      }
      return;
    }
    // Combine the kBW partials of each query (one per bank part) into one per
    // split, through LDS: the stage ring and the stash are free once every
    // wave has passed the barrier below (all loads have landed).  The wave of
    // part 0 of each query group merges the sorted lists (a kBW-way merge,
    // heads in registers) and writes the split's list to its own slot (the
    // merge kernel reads every kBW-th list slot) and the split's softmax
    // partials to part_ms[q][split].
    static_assert(S::kWaves * KCAP * 64 * 8 <= kRing * kStageVec * 16, "lists fit the ring");
    static_assert(S::kWaves * 64 * 8 <= kCap * kThreads * 8, "partials fit the stash");
    __syncthreads();
    uint64_t* cl = reinterpret_cast<uint64_t*>(&tiles[0][0]);  // [kWaves][KCAP][64]
    float2* cm = reinterpret_cast<float2*>(stash);              // [kWaves][64]
#pragma unroll
    for (int i = 0; i < KCAP; ++i) cl[(wave * KCAP + i) * 64 + lane] = q_valid ? fl[i] : 0;
    cm[wave * 64 + lane] = make_float2(run_m, run_s);
    __syncthreads();
    if (half == 0) {
      constexpr int BW = S::kBW;
      const int w0 = wave;  // waves w0 .. w0 + BW - 1 hold this query group's parts
      uint64_t h[BW];
      int pos[BW];
#pragma unroll
      for (int j = 0; j < BW; ++j) {
        pos[j] = 0;
        h[j] = cl[((w0 + j) * KCAP) * 64 + lane];
      }
      uint64_t* dst = part_keys + out_slot * KCAP;  // part 0's slot (this wave's)
      for (int i = 0; i < KCAP; ++i) {
        int jm = 0;
        uint64_t best = h[0];
#pragma unroll
        for (int j = 1; j < BW; ++j) {
          if (h[j] > best) {
            best = h[j];
            jm = j;
          }
        }
        if (q_valid) dst[i] = best;
#pragma unroll
        for (int j = 0; j < BW; ++j) {
          if (j == jm) {
            ++pos[j];
            h[j] = pos[j] < KCAP ? cl[((w0 + j) * KCAP + pos[j]) * 64 + lane] : 0;
          }
        }
      }
      // softmax partials: common max, rescaled sums
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < BW; ++j) mx = fmaxf(mx, cm[(w0 + j) * 64 + lane].x);
      float sum = 0.f;
#pragma unroll
      for (int j = 0; j < BW; ++j) {
        const float2 v = cm[(w0 + j) * 64 + lane];
        if (v.x != -INFINITY) sum += v.y * fast_exp2(v.x - mx);
      }
      if (q_valid) part_ms[my_q * n_splits + split] = make_float2(mx, sum);  // compact [m, n_splits]
    }
  }
}

// The k-th search over a query's sample.  Every thread (or lane) first keeps
// the kSampleKeep largest of the keys it reads; the k-th largest of those
// kept keys is then found by deciding its 16 bits from the top, a candidate
// bit staying set when at least k kept keys are >= the candidate (counts
// from ballots).  The result equals the sample's k-th largest key unless one
// thread's keys hold more than kSampleKeep of the sample's top k; otherwise
// it is smaller.  Either way it is at most the sample's k-th largest key,
// which is all the bound needs.  Sample positions are bank rows in bank
// order, unrelated to which rows score high, so a thread (8 consecutive
// positions per 16-byte piece) rarely holds more than 4 of the top k: 4 are
// kept (the keep step is most of the search's time).  The search between
// the two launches of a split (prefix_kth) reads sorted lists instead, whose
// heads fall to a few threads, so it keeps kKthKeep.
constexpr int kKthKeep = 8;
constexpr int kSampleKeep = 4;

// t[0] >= t[1] >= ... : the R largest keys offered so far (start at 0,
// which ranks below every key).
template <int R>
__device__ __forceinline__ void keep_largest(uint32_t (&t)[R], uint32_t x) {
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t hi = max(t[r], x);
    x = min(t[r], x);
    t[r] = hi;
  }
}

// Largest 16-bit t with at least k of the wave's keys (R per lane) >= t;
// with SHIFT = 16 the keys sit in the upper half of each word.
template <int R, int SHIFT = 0>
__device__ __forceinline__ uint32_t wave_kth_key(const uint32_t (&key)[R], int k) {
  uint32_t t = 0;
  for (int b = 15; b >= 0; --b) {
    const uint32_t cand = t | (1u << b);
    int c = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) c += __builtin_popcountll(__ballot(key[j] >= (cand << SHIFT)));
    if (c >= k) t = cand;
  }
  return t;
}

// The bound from a query's sample: the k-th search's key decoded to the
// largest float that does not exceed any sample score it stands for; -inf
// when the sample holds fewer than k finite scores (keys below 0x0080 are
// -inf, i.e. masked rows).
__device__ __forceinline__ float sample_bound(uint32_t t, int64_t n_samp, int k) {
  const bool none = n_samp < k || t < 0x0080u;
  return none ? -INFINITY : ord2f(t << 16);
}

// A sample key and its position in one word, so that the larger word is the
// larger key and, among equal keys, the earlier position (positions are
// below 2^16: a sample holds at most 32,768 scores).
__device__ __forceinline__ uint32_t key_at(uint32_t key16, uint32_t pos) { return (key16 << 16) | (0xFFFFu - pos); }
__device__ __forceinline__ uint32_t wave_max(uint32_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = max(x, static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), o)));
  return x;
}
// The query's best sampled position from the largest key_at word, -1 when
// every sampled score is -inf.
__device__ __forceinline__ int32_t best_position(uint32_t best) {
  return (best >> 16) < 0x0080u ? -1 : static_cast<int32_t>(0xFFFFu - (best & 0xFFFFu));
}

// Keys kept for the k-th search: with NEAR, key_at words (the same keys
// rank the same way, and the largest word names the best sampled position),
// else the 16-bit keys themselves.
template <bool NEAR>
__device__ __forceinline__ uint32_t kept_key(uint32_t key16, uint32_t pos) {
  return NEAR ? key_at(key16, pos) : key16;
}

// One workgroup per query, for samples of any size: 256 threads keep 4 keys
// each, one wave searches the 1,024 kept keys.  NEAR: the query's best
// sampled position is written to near_out as well.
template <bool NEAR>
__global__ __launch_bounds__(256) void sample_kth_kernel(const uint16_t* __restrict__ samp, int64_t n_samp, int k,
                                                         float* __restrict__ t0_out, uint32_t* __restrict__ thr_out,
                                                         int32_t* __restrict__ near_out) {
  __shared__ uint32_t kept[256 * kSampleKeep];
  const int tid = threadIdx.x;
  const int64_t q = blockIdx.x;
  const u32x4* row = reinterpret_cast<const u32x4*>(samp + q * n_samp);
  const int64_t n_vec = n_samp / 8;  // n_samp is a multiple of 8 (whole tiles)
  uint32_t top[kSampleKeep];
#pragma unroll
  for (int r = 0; r < kSampleKeep; ++r) top[r] = 0u;
  constexpr int kUnroll = 4;  // 16-byte loads in flight per thread
  for (int64_t i0 = tid; i0 < n_vec; i0 += kUnroll * 256) {
    u32x4 w[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = i0 + u * 256;
      w[u] = i < n_vec ? row[i] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t pos = static_cast<uint32_t>((i0 + u * 256) * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        keep_largest(top, kept_key<NEAR>(w[u][e] & 0xFFFFu, pos + 2 * e));
        keep_largest(top, kept_key<NEAR>(w[u][e] >> 16, pos + 2 * e + 1));
      }
    }
  }
#pragma unroll
  for (int r = 0; r < kSampleKeep; ++r) kept[r * 256 + tid] = top[r];
  __syncthreads();
  if (tid < 64) {
    constexpr int kPerLane = 256 * kSampleKeep / 64;
    uint32_t key[kPerLane];
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) key[j] = kept[j * 64 + tid];
    const uint32_t t = wave_kth_key<kPerLane, NEAR ? 16 : 0>(key, k);
    // every thread's largest word is among key[0 .. 3] of some lane
    const uint32_t best = NEAR ? wave_max(max(max(key[0], key[1]), max(key[2], key[3]))) : 0u;
    if (tid == 0) {
      t0_out[q] = sample_bound(t, n_samp, k);
      if (thr_out) thr_out[q] = 0u;  // the shared bound starts empty (saves the bound-init launch)
      if (NEAR) near_out[q] = best_position(best);
    }
  }
}

// Small samples (n_samp <= 64 * kWaveKthPerLane): one wave per query reads
// the whole sample into registers, each lane keeps its 4 largest keys, and
// the wave searches the 256 kept keys.
constexpr int kWaveKthPerLane = 32;
static_assert(kWaveKthPerLane % 8 == 0, "whole 16-byte pieces per lane");

// With NEAR and top_out set, the kept words at or above the k-th key (each
// a 16-bit key and its sample position) also go to top_out[q][0, kSampleTop),
// zeros after the last (at most kSampleTop of them; any left out only make
// the bound built from them lower).
constexpr int kSampleTop = 64;
template <bool NEAR>
__global__ __launch_bounds__(256) void sample_kth_wave_kernel(const uint16_t* __restrict__ samp, int64_t n_samp,
                                                              int64_t m, int k, float* __restrict__ t0_out,
                                                              uint32_t* __restrict__ thr_out,
                                                              int32_t* __restrict__ near_out,
                                                              uint32_t* __restrict__ top_out) {
  const int lane = threadIdx.x & 63;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (q >= m) return;  // whole waves only; no workgroup barrier below
  // n_samp is a multiple of 8 (whole tiles), so the sample row is read in
  // 16-byte pieces of 8 keys; the order of the keys does not matter
  const u32x4* row = reinterpret_cast<const u32x4*>(samp + q * n_samp);
  u32x4 w[kWaveKthPerLane / 8];
#pragma unroll
  for (int j = 0; j < kWaveKthPerLane / 8; ++j) {
    const int64_t v = static_cast<int64_t>(j) * 64 + lane;
    w[j] = v * 8 < n_samp ? row[v] : u32x4{0u, 0u, 0u, 0u};  // padding keys (0) rank below every key
  }
  uint32_t top[kSampleKeep];
#pragma unroll
  for (int r = 0; r < kSampleKeep; ++r) top[r] = 0u;
#pragma unroll
  for (int j = 0; j < kWaveKthPerLane / 8; ++j) {
    const uint32_t pos = static_cast<uint32_t>((j * 64 + lane) * 8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      keep_largest(top, kept_key<NEAR>(w[j][e] & 0xFFFFu, pos + 2 * e));
      keep_largest(top, kept_key<NEAR>(w[j][e] >> 16, pos + 2 * e + 1));
    }
  }
  const uint32_t t = wave_kth_key<kSampleKeep, NEAR ? 16 : 0>(top, k);
  const uint32_t best = NEAR ? wave_max(top[0]) : 0u;
  if (lane == 0) {
    t0_out[q] = sample_bound(t, n_samp, k);
    if (thr_out) thr_out[q] = 0u;  // the shared bound starts empty (saves the bound-init launch)
    if (NEAR) near_out[q] = best_position(best);
  }
  if (NEAR && top_out != nullptr) {
    uint32_t* dst = top_out + q * kSampleTop;
    const bool finite = sample_bound(t, n_samp, k) != -INFINITY;
    int base = 0;
#pragma unroll
    for (int r = 0; r < kSampleKeep; ++r) {
      const bool sel = finite && (top[r] >> 16) >= t;
      const uint64_t bal = __ballot(sel);
      const int at = base + static_cast<int>(__popcll(bal & ((uint64_t{1} << lane) - 1)));
      if (sel && at < kSampleTop) dst[at] = top[r];
      base += static_cast<int>(__popcll(bal));
    }
    if (lane >= base) dst[lane] = 0u;  // (kSampleTop == 64: one slot per lane)
  }
}

// Between the two launches of a split: a lower bound on each query's k-th
// best score over the rows its lane lists have seen (the union of the lists
// holds the query's best k of those rows), by the sample's keep-then-ballot
// search keeping kKthKeep, on the lists' full 32-bit score order keys: the
// scores are the full pass's own, so the bound needs no rounding down, and
// a 16-bit key would round it down by up to 2^-7 relative, which on the 1M
// retrieval admits over twice the rows in the second launch.  t0[q] keeps
// the larger of this bound and the one it holds.  A query's lists are n_keys
// consecutive keys.  One wave per query (four per workgroup) for up to
// 64 * kWaveKthPerLane keys, else one workgroup per query.

// Largest 32-bit t with at least k of the wave's keys (R per lane) >= t.
template <int R>
__device__ __forceinline__ uint32_t wave_kth_key32(const uint32_t (&key)[R], int k) {
  uint32_t t = 0;
  for (int b = 31; b >= 0; --b) {
    const uint32_t cand = t | (1u << b);
    int c = 0;
#pragma unroll
    for (int j = 0; j < R; ++j) c += __builtin_popcountll(__ballot(key[j] >= cand));
    if (c >= k) t = cand;
  }
  return t;
}
// The bound from the lists' k-th key: -inf when fewer than k finite scores
// were listed (empty list slots hold key 0; order keys below 0x00800000 are
// -inf scores).
__device__ __forceinline__ float prefix_bound(uint32_t t, int64_t n_keys, int k) {
  return (n_keys < k || t < 0x00800000u) ? -INFINITY : ord2f(t);
}
// R keys kept per lane: kKthKeep, or every key when a query has at most
// 64 * R of them (the search is then exact and runs R ballots per bit).
template <int R>
__global__ __launch_bounds__(256) void prefix_kth_wave_kernel(const uint64_t* __restrict__ keys, int64_t n_keys,
                                                              int64_t m, int k, float* __restrict__ t0) {
  const int lane = threadIdx.x & 63;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (q >= m) return;  // whole waves only; no workgroup barrier below
  const uint64_t* row = keys + q * n_keys;
  uint32_t top[R];
#pragma unroll
  for (int r = 0; r < R; ++r) top[r] = 0u;
#pragma unroll
  for (int j = 0; j < kWaveKthPerLane; ++j) {
    const int64_t i = static_cast<int64_t>(j) * 64 + lane;
    if (i < n_keys) keep_largest(top, static_cast<uint32_t>(row[i] >> 32));
  }
  const uint32_t t = wave_kth_key32(top, k);
  if (lane == 0) t0[q] = fmaxf(t0[q], prefix_bound(t, n_keys, k));
}

__global__ __launch_bounds__(256) void prefix_kth_kernel(const uint64_t* __restrict__ keys, int64_t n_keys, int k,
                                                         float* __restrict__ t0) {
  __shared__ uint32_t kept[256 * kKthKeep];
  const int tid = threadIdx.x;
  const int64_t q = blockIdx.x;
  const uint64_t* row = keys + q * n_keys;
  uint32_t top[kKthKeep];
#pragma unroll
  for (int r = 0; r < kKthKeep; ++r) top[r] = 0u;
  constexpr int kUnroll = 4;  // loads in flight per thread
  for (int64_t i0 = tid; i0 < n_keys; i0 += kUnroll * 256) {
    uint64_t w[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t i = i0 + u * 256;
      w[u] = i < n_keys ? row[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) keep_largest(top, static_cast<uint32_t>(w[u] >> 32));
  }
#pragma unroll
  for (int r = 0; r < kKthKeep; ++r) kept[r * 256 + tid] = top[r];
  __syncthreads();
  if (tid < 64) {
    constexpr int kPerLane = 256 * kKthKeep / 64;
    uint32_t key[kPerLane];
#pragma unroll
    for (int j = 0; j < kPerLane; ++j) key[j] = kept[j * 64 + tid];
    const uint32_t t = wave_kth_key32(key, k);
    if (tid == 0) t0[q] = fmaxf(t0[q], prefix_bound(t, n_keys, k));
  }
}

// Query order for the full pass.  A wave's 64 lanes are 64 queries, and a
// 16-row block costs the whole wave the candidate code as soon as one lane
// has a candidate in it; when the 64 queries lie in one region of the bank
// (share their best rows) far fewer blocks do.  Each query's best sampled
// row is a cheap stand-in for its region.  In a relation build the sampled
// rows are queries as well, so sampled positions are further joined along
// their own best-sampled-row links: label(s) = the smallest position
// reachable from s along them (the fixed point of label(s) = min(label(s),
// label(next(s)), label(label(s))), which does not depend on update order).
// Queries are then counting-sorted by the label of their best sampled
// position.  The order inside one label is arbitrary: every query's lists,
// softmax partials and bounds are its own, so results do not depend on it.
// Four launches: the labels (one workgroup, in LDS), the per-label counts
// (one thread per query, which also keeps its rank among its label's
// queries), their exclusive scan (one workgroup), and the scatter of every
// query to its label's first position plus its rank, together with the copy
// of its row.
constexpr int kOrderThreads = 1024;
constexpr int kOrderMaxIters = 64;  // label rounds (a cut-off still leaves a valid order)

__device__ __forceinline__ int32_t block_exclusive_1024(int32_t mine, int32_t* red, int32_t& total) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  int32_t inc = mine;
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t o = __shfl_up(inc, off);
    if (lane >= off) inc += o;
  }
  if (lane == 63) red[wave] = inc;
  __syncthreads();
  int32_t before = 0;
  total = 0;
  for (int w = 0; w < kOrderThreads / 64; ++w) {
    before += w < wave ? red[w] : 0;
    total += red[w];
  }
  __syncthreads();
  return before + inc - mine;
}

// Labels of the first n_lab (<= kOrderMaxSample) sampled positions to
// lab_out[], and the per-label counts cleared.  Sampled position s holds
// bank row (s / run) * split_rows + s % run (run = sampled rows per sampled
// split, split_rows = bank rows from one sampled split to the next); query i
// is bank row i.
__global__ __launch_bounds__(kOrderThreads) void order_labels_kernel(const int32_t* __restrict__ near, int64_t m,
                                                                     int32_t n_lab, int64_t run, int64_t split_rows,
                                                                     int32_t* __restrict__ lab_out,
                                                                     int32_t* __restrict__ cnt) {
  __shared__ int32_t lab[kOrderMaxSample];
  constexpr int kPerThread = kOrderMaxSample / kOrderThreads;  // positions s = tid + j * kOrderThreads
  const int tid = threadIdx.x;
  // each of the thread's positions and where its link leads (itself if none)
  int32_t nx[kPerThread];
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const int32_t s = tid + j * kOrderThreads;
    nx[j] = s;
    if (s < n_lab) {
      const int64_t row = (s / run) * split_rows + s % run;
      const int32_t t = row < m ? near[row] : -1;
      nx[j] = (t >= 0 && t < n_lab) ? t : s;
    }
  }
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const int32_t s = tid + j * kOrderThreads;
    if (s < n_lab) lab[s] = min(s, nx[j]);
  }
  __syncthreads();
  for (int it = 0; it < kOrderMaxIters; ++it) {
    int changed = 0;
#pragma unroll
    for (int j = 0; j < kPerThread; ++j) {
      const int32_t s = tid + j * kOrderThreads;
      if (s < n_lab) {
        const int32_t l = lab[s];
        int32_t l2 = min(l, lab[nx[j]]);
        l2 = min(l2, lab[l2]);
        if (l2 < l) {
          lab[s] = l2;
          changed = 1;
        }
      }
    }
    if (!__syncthreads_or(changed)) break;
  }
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const int32_t s = tid + j * kOrderThreads;
    if (s < n_lab) {
      lab_out[s] = lab[s];
      cnt[s] = 0;
    }
  }
}

// near[q] <- the label of query q's best sampled position (label 0 without
// one), counted per label; rank[q] <- the count before q's own.
__global__ __launch_bounds__(256) void order_count_kernel(int32_t* __restrict__ near, int64_t m, int32_t n_lab,
                                                          const int32_t* __restrict__ lab,
                                                          int32_t* __restrict__ cnt, int32_t* __restrict__ rank) {
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (q >= m) return;
  const int32_t t = near[q];
  const int32_t key = (t >= 0 && t < n_lab) ? lab[t] : 0;
  near[q] = key;
  rank[q] = atomicAdd(cnt + key, 1);
}

// Per-label counts -> first positions, in place (one workgroup; each thread
// scans a run of consecutive labels).
__global__ __launch_bounds__(kOrderThreads) void order_scan_kernel(int32_t* __restrict__ cnt, int32_t n_lab) {
  __shared__ int32_t red[kOrderThreads / 64];
  const int32_t per = (n_lab + kOrderThreads - 1) / kOrderThreads;
  const int32_t s0 = static_cast<int32_t>(threadIdx.x) * per;
  int32_t sum = 0;
  for (int32_t j = 0; j < per; ++j)
    if (s0 + j < n_lab) sum += cnt[s0 + j];
  int32_t total;
  int32_t ex = block_exclusive_1024(sum, red, total);
  for (int32_t j = 0; j < per; ++j) {
    if (s0 + j < n_lab) {
      const int32_t c = cnt[s0 + j];
      cnt[s0 + j] = ex;
      ex += c;
    }
  }
}

// One wave per query: its position is its label's first position plus its
// rank within the label; record it in perm and copy the query's row there
// (16-byte vectors).
__global__ __launch_bounds__(256) void order_scatter_kernel(const int32_t* __restrict__ key,
                                                            const int32_t* __restrict__ rank, int64_t m,
                                                            const int32_t* __restrict__ start,
                                                            const u32x4* __restrict__ queries,
                                                            int64_t q_vecs_stride, int row_vecs,
                                                            int32_t* __restrict__ perm, u32x4* __restrict__ qbuf) {
  const int lane = threadIdx.x & 63;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (q >= m) return;  // whole waves only; no workgroup barrier below
  const int32_t pos = start[key[q]] + rank[q];
  if (lane == 0) perm[pos] = static_cast<int32_t>(q);
  for (int v = lane; v < row_vecs; v += 64)
    qbuf[static_cast<int64_t>(pos) * row_vecs + v] = queries[q * q_vecs_stride + v];
}

// A tighter bound for a relation build in clustered order.  The keys at
// clustered positions near a key are mostly of its own region of the bank,
// and every one of them is a bank row, i.e. one of the key's candidates; the
// k-th best of the key's scores against them is therefore a lower bound on
// its k-th best over the bank.  One workgroup per 64-key tile at positions
// [a, a + 64) scores the tile against the band of positions [a - 32,
// a + 96) (the keys themselves are band rows 32..95, so the band is staged
// once), each score lowered by twice the fp32 accumulation bound of a
// length-d dot product, 2 d 2^-24 ||q|| ||b|| (this kernel and the full pass
// may each be off by that much), so the bound never exceeds the full pass's
// own k-th best.  The key itself and positions outside [0, m) are left out.
// t0[key] keeps the larger of this bound and the one it holds.
constexpr int kBandKeys = 64;
constexpr int kBandRows = 128;          // band rows per tile (32 before, 64 keys, 32 after)
constexpr int kBandChunk = 32;          // K elements per staged chunk
constexpr int kBandPitch = 40;          // staged row pitch in bf16 (80 B: spreads LDS banks)
constexpr int kBandAhead = 4;           // chunks whose global loads are in flight
__global__ __launch_bounds__(256) void band_bound_kernel(const uint16_t* __restrict__ rows, int64_t m, int32_t d,
                                                         int k, const int32_t* __restrict__ perm,
                                                         const uint32_t* __restrict__ samp_top, int64_t run,
                                                         int64_t split_rows, float* __restrict__ t0) {
  __shared__ __attribute__((aligned(16))) uint16_t st[kBandRows * kBandPitch];
  __shared__ float sc[kBandKeys][kBandRows + 1];
  __shared__ float nrm[kBandRows];
  __shared__ uint8_t sampled[kBandRows];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t a = static_cast<int64_t>(blockIdx.x) * kBandKeys;  // first key position of the tile
  const int64_t b0 = a - 32;                                        // first band position
  const int nk = d / kBandChunk;
  // each thread stages 2 of the 512 16-byte pieces of a chunk: band row
  // (tid >> 2) + 64 h, piece tid & 3
  auto load = [&](int c, u32x4 (&v)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = (tid >> 2) + 64 * h;
      const int64_t pos = b0 + r;
      v[h] = (pos >= 0 && pos < m && c < nk)
                 ? *reinterpret_cast<const u32x4*>(rows + pos * d + c * kBandChunk + (tid & 3) * 8)
                 : u32x4{0u, 0u, 0u, 0u};
    }
  };
  u32x4 buf[kBandAhead][2];
#pragma unroll
  for (int u = 0; u < kBandAhead; ++u) load(u, buf[u]);
  f32x16 acc[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[qb][r] = 0.f;
  float sq = 0.f;  // squared norm of band row tid (tid < 128)
  const int frow = lane & 31;
  const int fpart = lane >> 5;
  for (int c0 = 0; c0 < nk; c0 += kBandAhead) {
#pragma unroll
    for (int u = 0; u < kBandAhead; ++u) {
      const int c = c0 + u;
      if (c < nk) {  // uniform
        __syncthreads();  // the previous chunk's LDS reads are done
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int r = (tid >> 2) + 64 * h;
          *reinterpret_cast<u32x4*>(&st[r * kBandPitch + (tid & 3) * 8]) = buf[u][h];
        }
        load(c + kBandAhead, buf[u]);  // the slot just stored takes a later chunk
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const bf16x8 fa =
              as_bf16x8(*reinterpret_cast<const u32x4*>(&st[(32 * wave + frow) * kBandPitch + ks * 16 + fpart * 8]));
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const bf16x8 fb = as_bf16x8(
                *reinterpret_cast<const u32x4*>(&st[(32 + 32 * qb + frow) * kBandPitch + ks * 16 + fpart * 8]));
            acc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb, acc[qb], 0, 0, 0);
          }
        }
        if (tid < kBandRows) {
#pragma unroll
          for (int e = 0; e < kBandChunk; ++e) {
            const float x = __uint_as_float(static_cast<uint32_t>(st[tid * kBandPitch + e]) << 16);
            sq = fmaf(x, x, sq);
          }
        }
      }
    }
  }
  // scores to LDS as sc[key][band row]: lane l holds key column l % 32 of
  // key block qb and band rows 8 (r / 4) + 4 (l / 32) + r % 4 of its wave's 32
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      sc[32 * qb + frow][32 * wave + 8 * (r >> 2) + 4 * fpart + (r & 3)] = acc[qb][r];
  if (tid < kBandRows) {
    nrm[tid] = sqrtf(sq);
    // whether the band row is a sampled row (its score then counts through
    // the sample's own keys, never twice)
    const int64_t pos = b0 + tid;
    bool smp = false;
    if (samp_top != nullptr && pos >= 0 && pos < m) smp = (perm[pos] % split_rows) < run;
    sampled[tid] = smp ? 1 : 0;
  }
  __syncthreads();
  // four threads per key, 32 band rows and 16 of the sample's top keys each;
  // the largest 16-bit order key with at least k of the lowered band scores
  // and the sample's scores at or above it, decided from the top
  const int key = tid >> 2;
  const int part = tid & 3;
  const int64_t kp = a + key;
  const float margin = 2.f * static_cast<float>(d) * 5.9604645e-8f * nrm[32 + key];  // 2 d 2^-24 ||q||
  uint32_t kk[32];
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int r = 32 * part + j;
    const int64_t pos = b0 + r;
    const bool ok = kp < m && pos >= 0 && pos < m && r != 32 + key && sampled[r] == 0;
    const float v = sc[key][r] - (margin * nrm[r] + 1e-30f);
    kk[j] = ok ? (f2ord(v) >> 16) : 0u;
  }
  // the sample pass scores its rows exactly as the full pass does, so its
  // (rounded-down) keys need no margin
  uint32_t sk[kSampleTop / 4];
  const int32_t q = kp < m ? perm[kp] : 0;
  const uint32_t* top_q = (samp_top != nullptr && kp < m)
                              ? samp_top + static_cast<int64_t>(q) * kSampleTop + part * (kSampleTop / 4)
                              : nullptr;
#pragma unroll
  for (int j = 0; j < kSampleTop / 4; ++j) sk[j] = top_q != nullptr ? top_q[j] >> 16 : 0u;
  uint32_t t = 0;
  for (int bit = 15; bit >= 0; --bit) {
    const uint32_t cand = t | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < 32; ++j) cnt += kk[j] >= cand ? 1 : 0;
#pragma unroll
    for (int j = 0; j < kSampleTop / 4; ++j) cnt += sk[j] >= cand ? 1 : 0;
    cnt += __shfl_xor(cnt, 1);
    cnt += __shfl_xor(cnt, 2);
    if (cnt >= k) t = cand;
  }
  if (part == 0 && kp < m && t >= 0x0080u) t0[q] = fmaxf(t0[q], ord2f(t << 16));
}

// Grouped selection, preparation.  Queries are counted per namespace,
// their offsets and the work items per namespace (64-query tiles x S splits)
// come from two scans, and the queries are scattered to grouped positions
// (the order inside a namespace does not matter: every query's partials
// are its own).  A query without a namespace gets empty partials here, as no
// work item covers it.
__global__ __launch_bounds__(256) void group_count_kernel(const int32_t* __restrict__ key_ns, int64_t m, int n_ns,
                                                          int32_t* __restrict__ q_cnt) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= m) return;
  const int32_t u = key_ns[i];
  if (u >= 0 && u < n_ns) atomicAdd(q_cnt + u, 1);
}

struct QCountOp {
  const int32_t* cnt;
  __device__ int64_t operator()(int64_t u) const { return cnt[u]; }
};
struct ItemOp {
  const int32_t* cnt;
  int S;
  __device__ int64_t operator()(int64_t u) const { return (static_cast<int64_t>(cnt[u]) + 63) / 64 * S; }
};

__global__ __launch_bounds__(256) void group_scatter_kernel(const int32_t* __restrict__ key_ns, int64_t m, int n_ns,
                                                            const int64_t* __restrict__ q_off,
                                                            int32_t* __restrict__ fill, int32_t* __restrict__ perm,
                                                            uint64_t* __restrict__ part_keys,
                                                            float2* __restrict__ part_ms, int S, int lists_per_split,
                                                            int kcap) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= m) return;
  const int32_t u = key_ns[i];
  if (u >= 0 && u < n_ns) {
    perm[q_off[u] + atomicAdd(fill + u, 1)] = static_cast<int32_t>(i);
  } else {
    const int64_t nl = static_cast<int64_t>(S) * lists_per_split * kcap;
    for (int64_t j = 0; j < nl; ++j) part_keys[i * nl + j] = 0;
    for (int s = 0; s < S; ++s) part_ms[i * S + s] = make_float2(-INFINITY, 0.f);
  }
}

// The same preparation in one workgroup for up to kPrepNs namespaces and
// kPrepM queries (counts and fill positions in LDS): count, both exclusive
// scans, scatter, empty partials for queries without a namespace and the
// shared bounds, in one launch instead of nine.
constexpr int kPrepNs = 4096;
constexpr int64_t kPrepM = 16384;
__global__ __launch_bounds__(256) void group_prep_kernel(const int32_t* __restrict__ key_ns, int64_t m, int n_ns,
                                                         int S, int64_t* __restrict__ q_off,
                                                         int64_t* __restrict__ item_off, int32_t* __restrict__ perm,
                                                         uint64_t* __restrict__ part_keys,
                                                         float2* __restrict__ part_ms, int lists_per_split, int kcap,
                                                         uint32_t* __restrict__ thr) {
  __shared__ int32_t cnt[kPrepNs];
  __shared__ int32_t pos[kPrepNs];
  __shared__ int64_t red[4];
  constexpr int kPer = kPrepNs / 256;  // namespaces per thread in the scans
  const int tid = threadIdx.x;
  for (int u = tid; u < n_ns; u += 256) cnt[u] = 0;
  __syncthreads();
  for (int64_t i = tid; i < m; i += 256) {
    const int32_t u = key_ns[i];
    if (u >= 0 && u < n_ns) atomicAdd(&cnt[u], 1);
  }
  __syncthreads();
  const int u0 = tid * kPer;
  int64_t sq = 0, si = 0;
  for (int j = 0; j < kPer; ++j) {
    const int u = u0 + j;
    if (u < n_ns) {
      sq += cnt[u];
      si += (cnt[u] + 63) / 64 * S;
    }
  }
  int64_t tq, ti;
  int64_t eq = block_exclusive(sq, red, tq);
  int64_t ei = block_exclusive(si, red, ti);
  for (int j = 0; j < kPer; ++j) {
    const int u = u0 + j;
    if (u < n_ns) {
      const int c = cnt[u];
      q_off[u] = eq;
      item_off[u] = ei;
      pos[u] = static_cast<int32_t>(eq);
      eq += c;
      ei += (c + 63) / 64 * S;
    }
  }
  if (tid == 0) {
    q_off[n_ns] = tq;
    item_off[n_ns] = ti;
  }
  __syncthreads();
  const int64_t nl = static_cast<int64_t>(S) * lists_per_split * kcap;
  for (int64_t i = tid; i < m; i += 256) {
    const int32_t u = key_ns[i];
    if (u >= 0 && u < n_ns) {
      perm[atomicAdd(&pos[u], 1)] = static_cast<int32_t>(i);
    } else {
      for (int64_t j = 0; j < nl; ++j) part_keys[i * nl + j] = 0;
      for (int s = 0; s < S; ++s) part_ms[i * S + s] = make_float2(-INFINITY, 0.f);
    }
    thr[i] = 0u;
  }
}

// qbuf[pos] = queries[perm[pos]] for the grouped positions, 16-byte vectors.
__global__ __launch_bounds__(256) void group_queries_kernel(const u32x4* __restrict__ queries, int64_t q_vecs_stride,
                                                            const int32_t* __restrict__ perm,
                                                            const int64_t* __restrict__ n_grouped, int row_vecs,
                                                            u32x4* __restrict__ qbuf) {
  const int64_t pos = blockIdx.x;
  if (pos >= *n_grouped) return;
  const int64_t q = perm[pos];
  for (int v = threadIdx.x; v < row_vecs; v += 256) qbuf[pos * row_vecs + v] = queries[q * q_vecs_stride + v];
}

// Shared per-query bounds start empty (order key 0 is below every score).
__global__ __launch_bounds__(256) void thr_init_kernel(uint32_t* __restrict__ thr, int64_t m) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < m) thr[i] = 0u;
}

}  // namespace

GroupLayout group_layout(int64_t m, int32_t n_ns, int32_t d, size_t base) {
  auto al = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  GroupLayout L{};
  const int64_t nb = (static_cast<int64_t>(n_ns) + kScanBlock - 1) / kScanBlock + 1;
  size_t o = base;
  L.q_cnt = o;    o += al(static_cast<size_t>(n_ns > 0 ? n_ns : 1) * 4);
  L.fill = o;     o += al(static_cast<size_t>(n_ns > 0 ? n_ns : 1) * 4);
  L.q_off = o;    o += al(static_cast<size_t>(n_ns + 1) * 8);
  L.item_off = o; o += al(static_cast<size_t>(n_ns + 1) * 8);
  L.bsum = o;     o += al(static_cast<size_t>(nb + 1) * 8);
  L.perm = o;     o += al(static_cast<size_t>(m > 0 ? m : 1) * 4);
  L.qbuf = o;     o += al(static_cast<size_t>(m > 0 ? m : 1) * d * 2);
  L.bytes = o;
  return L;
}

hipError_t launch_topk_grouped(const Plan& p, const GroupLayout& G, const uint16_t* bank, int64_t bank_stride,
                               int64_t n, const uint16_t* queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                               int32_t k, const int32_t* ns_off, const int32_t* rows, int32_t n_ns,
                               int64_t n_entries, const int32_t* key_ns, void* ws, hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* samp = reinterpret_cast<uint16_t*>(w + p.ws_samp);
  auto* t0 = reinterpret_cast<float*>(w + p.ws_t0);
  auto* keys = reinterpret_cast<uint64_t*>(w + p.ws_part_keys);
  auto* ms = reinterpret_cast<float2*>(w + p.ws_part_ms);
  auto* thr = reinterpret_cast<uint32_t*>(w + p.ws_thr);
  auto* q_cnt = reinterpret_cast<int32_t*>(w + G.q_cnt);
  auto* fill = reinterpret_cast<int32_t*>(w + G.fill);
  auto* q_off = reinterpret_cast<int64_t*>(w + G.q_off);
  auto* item_off = reinterpret_cast<int64_t*>(w + G.item_off);
  auto* bsum = reinterpret_cast<int64_t*>(w + G.bsum);
  auto* perm = reinterpret_cast<int32_t*>(w + G.perm);
  auto* qbuf = reinterpret_cast<uint16_t*>(w + G.qbuf);
  const int S = p.n_splits;
  if (n_ns <= kPrepNs && m <= kPrepM) {
    group_prep_kernel<<<1, 256, 0, stream>>>(key_ns, m, n_ns, S, q_off, item_off, perm, keys, ms, p.part_stride,
                                             p.kcap, thr);
  } else {
    fill_i32_kernel<<<blocks256(n_ns), 256, 0, stream>>>(q_cnt, n_ns, 0);
    fill_i32_kernel<<<blocks256(n_ns), 256, 0, stream>>>(fill, n_ns, 0);
    group_count_kernel<<<blocks256(m), 256, 0, stream>>>(key_ns, m, n_ns, q_cnt);
    hipError_t e = exclusive_scan(QCountOp{q_cnt}, n_ns, bsum, q_off, stream);
    if (e != hipSuccess) return e;
    e = exclusive_scan(ItemOp{q_cnt, S}, n_ns, bsum, item_off, stream);
    if (e != hipSuccess) return e;
    group_scatter_kernel<<<blocks256(m), 256, 0, stream>>>(key_ns, m, n_ns, q_off, fill, perm, keys, ms, S,
                                                           p.part_stride, p.kcap);
    thr_init_kernel<<<dim3(static_cast<unsigned>((m + 255) / 256)), 256, 0, stream>>>(thr, m);
  }
  group_queries_kernel<<<dim3(static_cast<unsigned>(m)), 256, 0, stream>>>(
      reinterpret_cast<const u32x4*>(queries), q_stride / 8, perm, q_off + n_ns, d / 8, reinterpret_cast<u32x4*>(qbuf));
  // items: at most (ceil(m / 64) + min(m, n_ns)) query tiles, S splits each
  const int64_t bound = ((m + 63) / 64 + (m < n_ns ? m : n_ns)) * S;
  const GroupArgs ga{ns_off, q_off, item_off, perm, n_ns, S, static_cast<uint32_t>(n * bank_stride * 2), n_entries};
  // When the plan asks for it, a sample pass over the first tile of every
  // table (the split-0 items) bounds each query's k-th best from below, as
  // for the whole bank; the full pass starts its thresholds there.
  auto run = [&](auto kcap_tag) -> hipError_t {
    constexpr int KC = decltype(kcap_tag)::value;
    const dim3 grid(static_cast<unsigned>(bound));
    const float* t0_arg = nullptr;
    if (p.ns > 0) {
      topk_mfma_kernel<KC, true, 1, false, true><<<grid, Shape<1>::kThreads, 0, stream>>>(
          bank, bank_stride, n, qbuf, d, m, d, c2, -1, 0, S, 0, keys, ms, p.ns, 1, samp, p.n_samp, nullptr, nullptr,
          nullptr, nullptr, rows, ga, kWholeSplit);
      sample_kth_wave_kernel<false><<<dim3(static_cast<unsigned>((m + 3) / 4)), 256, 0, stream>>>(
          samp, p.n_samp, m, k, t0, nullptr, nullptr, nullptr);
      t0_arg = t0;
    }
    topk_mfma_kernel<KC, false, 1, false, true><<<grid, Shape<1>::kThreads, 0, stream>>>(
        bank, bank_stride, n, qbuf, d, m, d, c2, -1, 0, S, 0, keys, ms, 0, 1, nullptr, 0, t0_arg, thr, nullptr,
        nullptr, rows, ga, kWholeSplit);
    return hipGetLastError();
  };
  switch (p.kcap) {
    case 8:
      return run(std::integral_constant<int, 8>{});
    case 16:
      return run(std::integral_constant<int, 16>{});
    case 32:
      return run(std::integral_constant<int, 32>{});
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_topk_mfma(const Plan& p, const uint16_t* bank, int64_t bank_stride, int64_t n,
                            const uint16_t* queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                            int64_t self_base, int32_t k, const Scope& scope, bool relation, void* ws,
                            hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* keys = reinterpret_cast<uint64_t*>(w + p.ws_part_keys);
  auto* ms = reinterpret_cast<float2*>(w + p.ws_part_ms);
  auto* samp = reinterpret_cast<uint16_t*>(w + p.ws_samp);
  auto* t0 = reinterpret_cast<float*>(w + p.ws_t0);
  auto* thr = reinterpret_cast<uint32_t*>(w + p.ws_thr);
  auto* lane_ms = reinterpret_cast<float2*>(w + p.ws_lane_ms);
  const dim3 grid(static_cast<unsigned>(p.q_tiles * p.n_splits));
  const dim3 samp_grid(static_cast<unsigned>(p.q_tiles * p.n_samp_splits));
  auto run = [&](auto kcap_tag, auto qw_tag, auto scoped_tag) -> hipError_t {
    constexpr int KC = decltype(kcap_tag)::value;
    constexpr int QW = decltype(qw_tag)::value;
    constexpr bool SC = decltype(scoped_tag)::value;
    constexpr int T = Shape<QW>::kThreads;
    const float* t0_arg = nullptr;
    // the full pass takes the queries in clustered order where the plan has
    // room for it (relation builds, no scope)
    const bool ordered = p.order && relation && !SC;
    int32_t* near = ordered ? reinterpret_cast<int32_t*>(w + p.ws_near) : nullptr;
    // the sample's top keys per query, for the band bound (only from the
    // one-wave k-th search, i.e. samples of at most 2,048 keys)
    uint32_t* stop =
        (ordered && p.n_samp <= 64 * kWaveKthPerLane) ? reinterpret_cast<uint32_t*>(w + p.ws_stop) : nullptr;
    if (p.ns > 0) {
      topk_mfma_kernel<KC, true, QW, SC, false><<<samp_grid, T, 0, stream>>>(
          bank, bank_stride, n, queries, q_stride, m, d, c2, self_base, p.q_tiles, p.n_splits, p.tiles_per_split,
          keys, ms, p.ns, p.samp_stride, samp, p.n_samp, nullptr, nullptr, scope.row_ns, scope.key_ns, nullptr,
          GroupArgs{}, kWholeSplit);
      const dim3 wave_grid(static_cast<unsigned>((m + 3) / 4)), wg_grid(static_cast<unsigned>(m));
      if (p.n_samp <= 64 * kWaveKthPerLane) {
        if (near)
          sample_kth_wave_kernel<true><<<wave_grid, 256, 0, stream>>>(samp, p.n_samp, m, k, t0, thr, near, stop);
        else
          sample_kth_wave_kernel<false><<<wave_grid, 256, 0, stream>>>(samp, p.n_samp, m, k, t0, thr, nullptr,
                                                                         nullptr);
      } else {
        if (near)
          sample_kth_kernel<true><<<wg_grid, 256, 0, stream>>>(samp, p.n_samp, k, t0, thr, near);
        else
          sample_kth_kernel<false><<<wg_grid, 256, 0, stream>>>(samp, p.n_samp, k, t0, thr, nullptr);
      }
      t0_arg = t0;
    } else {
      thr_init_kernel<<<dim3(static_cast<unsigned>((m + 255) / 256)), 256, 0, stream>>>(thr, m);
    }
    const uint16_t* fq = queries;  // the queries as the full pass reads them
    int64_t fq_stride = q_stride;
    GroupArgs fg{};
    if (ordered && p.ns > 0) {
      auto* perm = reinterpret_cast<int32_t*>(w + p.ws_perm);
      auto* olab = reinterpret_cast<int32_t*>(w + p.ws_olab);
      auto* ocnt = reinterpret_cast<int32_t*>(w + p.ws_ocnt);
      auto* orank = reinterpret_cast<int32_t*>(w + p.ws_orank);
      auto* qbuf = reinterpret_cast<uint16_t*>(w + p.ws_qbuf);
      const int64_t run = static_cast<int64_t>(p.ns) * p.tile_rows;
      const int64_t split_rows = static_cast<int64_t>(p.samp_stride) * p.tiles_per_split * p.tile_rows;
      const int32_t n_lab = static_cast<int32_t>(p.n_samp < kOrderMaxSample ? p.n_samp : kOrderMaxSample);
      order_labels_kernel<<<1, kOrderThreads, 0, stream>>>(near, m, n_lab, run, split_rows, olab, ocnt);
      order_count_kernel<<<blocks256(m), 256, 0, stream>>>(near, m, n_lab, olab, ocnt, orank);
      order_scan_kernel<<<1, kOrderThreads, 0, stream>>>(ocnt, n_lab);
      order_scatter_kernel<<<dim3(static_cast<unsigned>((m + 3) / 4)), 256, 0, stream>>>(
          near, orank, m, ocnt, reinterpret_cast<const u32x4*>(queries), q_stride / 8, d / 8, perm,
          reinterpret_cast<u32x4*>(qbuf));
      band_bound_kernel<<<dim3(static_cast<unsigned>((m + kBandKeys - 1) / kBandKeys)), 256, 0, stream>>>(
          qbuf, m, d, k, perm, stop, run, split_rows, t0);
      fq = qbuf;
      fq_stride = d;
      fg.perm = perm;
    }
    auto full = [&](const float* t0p, PhaseArgs pa) {
      topk_mfma_kernel<KC, false, QW, SC, false><<<grid, T, 0, stream>>>(
          bank, bank_stride, n, fq, fq_stride, m, d, c2, self_base, p.q_tiles, p.n_splits, p.tiles_per_split,
          keys, ms, p.ns, 1, samp, p.n_samp, t0p, thr, scope.row_ns, scope.key_ns, nullptr, fg, pa);
    };
    if (p.ph_split > 0) {
      // the first tiles of every split, then the k-th-best bound from the
      // lists they left (at least the sampled one), then the rest
      full(t0_arg, PhaseArgs{0, p.ph_split, 0, 0, lane_ms});
      const int64_t n_keys = static_cast<int64_t>(p.n_splits) * p.part_stride * KC;
      if (n_keys <= 64 * 2)
        prefix_kth_wave_kernel<2><<<dim3(static_cast<unsigned>((m + 3) / 4)), 256, 0, stream>>>(keys, n_keys, m, k, t0);
      else if (n_keys <= 64 * kWaveKthPerLane)
        prefix_kth_wave_kernel<kKthKeep><<<dim3(static_cast<unsigned>((m + 3) / 4)), 256, 0, stream>>>(keys, n_keys, m,
                                                                                                      k, t0);
      else
        prefix_kth_kernel<<<dim3(static_cast<unsigned>(m)), 256, 0, stream>>>(keys, n_keys, k, t0);
      full(t0, PhaseArgs{p.ph_split, 0x7FFFFFFF, 1, 1, lane_ms});
    } else {
      full(t0_arg, kWholeSplit);
    }
    return hipGetLastError();
  };
  auto run_q = [&](auto kcap_tag, auto scoped_tag) -> hipError_t {
    switch (p.qw) {
      case 1:
        return run(kcap_tag, std::integral_constant<int, 1>{}, scoped_tag);
      case 2:
        return run(kcap_tag, std::integral_constant<int, 2>{}, scoped_tag);
      default:
        return run(kcap_tag, std::integral_constant<int, 4>{}, scoped_tag);
    }
  };
  auto run_k = [&](auto kcap_tag) -> hipError_t {
    return scope.row_ns ? run_q(kcap_tag, std::true_type{}) : run_q(kcap_tag, std::false_type{});
  };
  switch (p.kcap) {
    case 8:
      return run_k(std::integral_constant<int, 8>{});
    case 16:
      return run_k(std::integral_constant<int, 16>{});
    case 32:
      return run_k(std::integral_constant<int, 32>{});
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace memattn
