// Matrix-core selection path (bf16 embeddings, fp32 accumulation) for gfx950.
//
// Dense-only relevance (Section 5.5) applied to LLMSelect of Algorithm 1:
// s_ij = <q_i, b_j> for a 256-query tile against a split of the bank,
// 256 bank rows per step, fused with the softmax normaliser and a per-query
// running top-k; the score matrix never leaves registers.
//
// Workgroup: 4 waves, 256 queries x 256 bank rows per step.  Wave w owns
// queries [64w, 64w+64) and all 256 bank rows, i.e. 8 x 2 blocks of
// v_mfma_f32_32x32x16_bf16 with the bank tile as the A operand (rows) and the
// queries as the B operand (columns), so each accumulator lane holds one
// query column.  K is staged through LDS 32 elements at a time, double
// buffered, with the next stage's global loads in flight during the current
// stage's MFMAs (and across tile boundaries).  Staged rows are 64 B with an
// XOR swizzle of their 16-byte chunks so fragment reads are bank-conflict
// free.
//
// Epilogue (per bank tile, per 32-row block): lanes l and l^32 exchange the
// half of the block that belongs to the other's query, so lane L then owns
// query L of its wave with all 32 rows of the block.  The lane keeps
//   - (M, sum): running max of x = scale*log2e*s and sum exp2(x - M);
//   - a sorted list of its query's best KCAP keys (score desc, id asc) in a
//     lane-private LDS column, with T = the list's last score in a register
//     as a filter.
// Scores above T (per half block of 16 rows) are appended to a lane-private
// LDS stash; the list is then loaded into registers, the stash inserted (the
// wave runs as many insertion rounds as its busiest lane needs) and the list
// stored back.  After the first tiles T is high and this path is rare.  At the end each lane writes its query's list and
// (M, sum) to the split partials merged by the merge kernel.
#include "device_common.h"
#include "launch.h"

namespace memattn {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTile = kMfmaTile;              // 256
constexpr int kBK = 32;                       // K elements per stage
constexpr int kRowVec = kBK / 8;              // 16-byte chunks per staged row
constexpr int kStageRows = 2 * kTile;         // bank rows then query rows
constexpr int kStageVec = kStageRows * kRowVec;
constexpr int kLoadsPerThread = kStageRows * kRowVec / 256;  // 8 x 16 B
constexpr int kCap = 16;                      // stash entries per lane (half a block)

// LDS chunk slot of 16-byte chunk c of staged row `row`.  The XOR swizzle
// makes the fragment reads (8 or 16 consecutive lanes = consecutive rows,
// same chunk) and the staging writes (4 chunks of 2 or 4 consecutive rows)
// hit distinct LDS banks with 64-byte rows.
__device__ __forceinline__ int slot(int row, int c) { return row * kRowVec + (c ^ (((row >> 1) ^ (row >> 2)) & 3)); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int KCAP>
__device__ __forceinline__ void list_insert(uint64_t (&list)[KCAP], uint64_t x) {
#pragma unroll
  for (int i = 0; i < KCAP; ++i) {
    const uint64_t a = list[i];
    const bool gt = x > a;
    list[i] = gt ? x : a;
    x = gt ? a : x;
  }
}

// Scores of half block hb (bank rows 16*hb .. 16*hb+15 of the tile) for the
// query this lane owns, in row order.  Before the exchange, lane l holds
// rows {8*(r/4) + 4*(l/32) + r%4} of both query blocks; lanes l and l^32
// swap the block that belongs to the other lane's query.  With hb a
// compile-time constant every accumulator index is static.
__device__ __forceinline__ void extract_half(const f32x16 (&acc)[8][2], int hb, bool lo, float (&v)[16]) {
  const int blk = hb >> 1;
  const int r0 = (hb & 1) * 8;
#pragma unroll
  for (int rr = 0; rr < 8; ++rr) {
    const int r = r0 + rr;
    const float mine = lo ? acc[blk][0][r] : acc[blk][1][r];
    const float send = lo ? acc[blk][1][r] : acc[blk][0][r];
    const float recv = __shfl_xor(send, 32);
    const int j0 = (r >> 2) * 8 + (r & 3) - (hb & 1) * 16;
    v[j0] = lo ? mine : recv;
    v[j0 + 4] = lo ? recv : mine;
  }
}

template <int KCAP>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1))) void
topk_mfma_kernel(const uint16_t* __restrict__ bank, int64_t bank_stride, int64_t n,
                 const uint16_t* __restrict__ queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                 int64_t self_base, int q_tiles, int n_splits, int tiles_per_split,
                 uint64_t* __restrict__ part_keys, float2* __restrict__ part_ms) {
  __shared__ u32x4 tiles[2][kStageVec];          // 64 KiB
  __shared__ uint64_t stash[kCap * 256];          // 32 KiB
  __shared__ uint64_t lists[KCAP * 256];          // up to 64 KiB

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // XCD-aware placement: workgroups b, b+8, b+16, ... run on one XCD; give
  // consecutive logical ids (the query tiles of one bank split) to one XCD
  // so the split's bank tiles are shared through that XCD's L2.
  const int G = gridDim.x;
  const int b = blockIdx.x;
  const int L = (G % 8 == 0) ? (b % 8) * (G / 8) + b / 8 : b;
  const int qt = L % q_tiles;
  const int split = L / q_tiles;
  const int64_t n_tiles = (n + kTile - 1) / kTile;
  const int64_t t0 = static_cast<int64_t>(split) * tiles_per_split;
  const int64_t t1 = min(n_tiles, t0 + tiles_per_split);
  const int64_t q_base = static_cast<int64_t>(qt) * kTile;

  const int nk = d / kBK;

  // Global -> LDS staging: thread tid moves 16-byte part (tid & 3) of rows
  // (tid >> 2) + 64*i, i = 0..7; rows 0..255 of a stage are bank rows,
  // 256..511 query rows.
  const int prow = tid >> 2;
  const int ppart = tid & 3;
  const uint16_t* qsrc = queries + (q_base + prow) * q_stride + ppart * 8;
  unsigned q_ok = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) q_ok |= (q_base + prow + 64 * i < m) ? (1u << i) : 0u;
  const int64_t q_step = 64 * q_stride;
  const int64_t b_step = 64 * bank_stride;

  u32x4 pre[kLoadsPerThread];
  auto load_stage = [&](int64_t tile, int kb) {
    const int64_t r0 = tile * kTile + prow;
    const uint16_t* bsrc = bank + r0 * bank_stride + ppart * 8 + kb * kBK;
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < 4; ++i)
      pre[i] = (r0 + 64 * i < n) ? *reinterpret_cast<const u32x4*>(bsrc + i * b_step) : z;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      pre[4 + i] = ((q_ok >> i) & 1u) ? *reinterpret_cast<const u32x4*>(qsrc + i * q_step + kb * kBK) : z;
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kLoadsPerThread; ++i) tiles[buf][slot(prow + 64 * i, ppart)] = pre[i];
  };

#pragma unroll
  for (int i = 0; i < KCAP; ++i) lists[i * 256 + tid] = 0;
  float thr = -INFINITY;  // score of list[KCAP-1] (-inf while the list is not full)
  float run_m = -INFINITY;
  float run_s = 0.f;
  const int64_t my_q = q_base + wave * 64 + lane;
  const int64_t self_row = self_base >= 0 ? self_base + my_q : -1;

  const int frag_row = lane & 31;
  const int frag_part = lane >> 5;
  f32x16 acc[8][2];
  auto mfma_stage = [&](int buf) {
    const u32x4* st = tiles[buf];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      bf16x8 bq[2];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
        bq[qb] = as_bf16x8(st[slot(kTile + wave * 64 + qb * 32 + frag_row, ks * 2 + frag_part)]);
#pragma unroll
      for (int blk = 0; blk < 8; ++blk) {
        const bf16x8 a = as_bf16x8(st[slot(blk * 32 + frag_row, ks * 2 + frag_part)]);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
          acc[blk][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bq[qb], acc[blk][qb], 0, 0, 0);
      }
    }
  };

  int buf = 0;
  if (t0 < t1) {
    load_stage(t0, 0);
    store_stage(0);
  }
  __syncthreads();

  for (int64_t tile = t0; tile < t1; ++tile) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
    }
    for (int kb = 0; kb + 1 < nk; ++kb) {
      load_stage(tile, kb + 1);
      mfma_stage(buf);
      store_stage(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }
    const bool has_next = tile + 1 < t1;
    if (has_next) load_stage(tile + 1, 0);
    mfma_stage(buf);

    // ---------------- epilogue for bank tile `tile`
    const int64_t row_base = tile * kTile;
    const bool tail = row_base + kTile > n;
    const bool diag = self_row >= row_base && self_row < row_base + kTile;
    const bool lo = lane < 32;
    auto load_half = [&](int hb, float (&v)[16]) {
      extract_half(acc, hb, lo, v);
      if (tail || diag) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int64_t row = row_base + hb * 16 + j;
          if (row >= n || row == self_row) v[j] = -INFINITY;
        }
      }
    };
    // pass 1: softmax normaliser over the tile, and which half blocks hold
    // scores above the current threshold
    unsigned cand = 0;
#pragma unroll
    for (int hb = 0; hb < 16; ++hb) {
      float v[16];
      load_half(hb, v);
      float hm = v[0];
#pragma unroll
      for (int j = 1; j < 16; ++j) hm = fmaxf(hm, v[j]);
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
      cand |= (hm > thr) ? (1u << hb) : 0u;
    }
    // pass 2 (rare once the threshold has risen): stash the half blocks'
    // survivors and insert them into the LDS list
    if (__ballot(cand != 0) != 0) {
      for (int hb = 0; hb < 16; ++hb) {
        if (__ballot((cand >> hb) & 1u) == 0) continue;
        float v[16];
        switch (hb) {
#define MEMATTN_HALF(H) \
  case H:               \
    load_half(H, v);    \
    break;
          MEMATTN_HALF(0) MEMATTN_HALF(1) MEMATTN_HALF(2) MEMATTN_HALF(3) MEMATTN_HALF(4) MEMATTN_HALF(5)
          MEMATTN_HALF(6) MEMATTN_HALF(7) MEMATTN_HALF(8) MEMATTN_HALF(9) MEMATTN_HALF(10) MEMATTN_HALF(11)
          MEMATTN_HALF(12) MEMATTN_HALF(13) MEMATTN_HALF(14) MEMATTN_HALF(15)
#undef MEMATTN_HALF
        }
        int cnt = 0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          if (v[j] > thr) {
            stash[cnt * 256 + tid] = make_key(v[j], static_cast<uint32_t>(row_base + hb * 16 + j));
            ++cnt;
          }
        }
        if (__ballot(cnt != 0) == 0) continue;
        uint64_t list[KCAP];
#pragma unroll
        for (int i = 0; i < KCAP; ++i) list[i] = lists[i * 256 + tid];
        for (int r = 0; __ballot(r < cnt) != 0; ++r) {
          if (r < cnt) list_insert<KCAP>(list, stash[r * 256 + tid]);
        }
#pragma unroll
        for (int i = 0; i < KCAP; ++i) lists[i * 256 + tid] = list[i];
        thr = list[KCAP - 1] == 0 ? -INFINITY : key_score(list[KCAP - 1]);
      }
    }

    if (has_next) store_stage(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }

  if (my_q < m) {
    const int64_t out_slot = my_q * n_splits + split;
#pragma unroll
    for (int i = 0; i < KCAP; ++i) part_keys[out_slot * KCAP + i] = lists[i * 256 + tid];
    part_ms[out_slot] = make_float2(run_m, run_s);
  }
}

}  // namespace

hipError_t launch_topk_mfma(const Plan& p, const uint16_t* bank, int64_t bank_stride, int64_t n,
                            const uint16_t* queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                            int64_t self_base, void* ws, hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* keys = reinterpret_cast<uint64_t*>(w + p.ws_part_keys);
  auto* ms = reinterpret_cast<float2*>(w + p.ws_part_ms);
  const dim3 grid(static_cast<unsigned>(p.q_tiles * p.n_splits));
  switch (p.kcap) {
    case 8:
      topk_mfma_kernel<8><<<grid, 256, 0, stream>>>(bank, bank_stride, n, queries, q_stride, m, d, c2, self_base,
                                                    p.q_tiles, p.n_splits, p.tiles_per_split, keys, ms);
      break;
    case 16:
      topk_mfma_kernel<16><<<grid, 256, 0, stream>>>(bank, bank_stride, n, queries, q_stride, m, d, c2, self_base,
                                                     p.q_tiles, p.n_splits, p.tiles_per_split, keys, ms);
      break;
    case 32:
      topk_mfma_kernel<32><<<grid, 256, 0, stream>>>(bank, bank_stride, n, queries, q_stride, m, d, c2, self_base,
                                                     p.q_tiles, p.n_splits, p.tiles_per_split, keys, ms);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace memattn
