// VALU selection path: any dtype, any d <= 8192, k <= 64, optional full
// probability output.  Serves the latency-bound tiny workloads (fp32
// embeddings) and shapes the matrix-core kernel does not take.
//
// One workgroup (256 threads) scores one query against one bank split, 256
// rows per step: thread t computes s = <q, b_j> for row j = base + t in fp32,
// folds it into its running softmax state, and offers its key to the
// block's sorted candidate list in LDS (block_list_insert: only the step's
// keys above the list's last entry are ranked into it).  Dense-only
// relevance of the paper's Section 5.5 applied to LLMSelect of Algorithm 1.
#include <atomic>

#include "device_common.h"
#include "launch.h"

namespace memattn {

namespace {

// Insert the block's new keys (one per thread, 0 = none; keys are unique)
// into the descending list buf[0, kcap) (kcap <= 256; zeros past its last
// key).  The keys above the list's last entry are compacted to buf[256 + i]
// by ballots; each of them takes its rank in the union (binary search in the
// list plus a count over the other candidates), each list key its new
// position, and every key of rank < kcap is written there.  The ranks are
// distinct and the union has at least as many keys as before, so every slot
// up to the new key count is written once and the rest stay 0.  Three
// barriers (none when no key qualifies), against 45 for a bitonic sort of
// the 512 entries.  wcount: 4 ints of LDS.  Every thread of the (4-wave)
// block must call it.
__device__ __forceinline__ void block_list_insert(uint64_t* buf, uint64_t key, int kcap, int* wcount) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const bool mine = key > buf[kcap - 1];
  const uint64_t bal = __ballot(mine);
  if (lane == 0) wcount[wave] = __popcll(bal);
  __syncthreads();  // counts visible; every read of the list's last entry done
  int base = 0, total = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int c = wcount[w];
    base += w < wave ? c : 0;
    total += c;
  }
  if (total == 0) return;  // (uniform)
  uint64_t* cand = buf + 256;
  if (mine) cand[base + __popcll(bal & ((uint64_t{1} << lane) - 1))] = key;
  __syncthreads();  // candidates visible
  int r_new = kcap;
  if (mine) {
    int lo = 0, hi = kcap;  // list keys above the key
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (buf[mid] > key) lo = mid + 1; else hi = mid;
    }
    r_new = lo;
    for (int i = 0; i < total; ++i) r_new += cand[i] > key ? 1 : 0;
  }
  uint64_t y = 0;
  int r_old = kcap;
  if (tid < kcap) {
    y = buf[tid];
    if (y != 0) {
      r_old = tid;
      for (int i = 0; i < total; ++i) r_old += cand[i] > y ? 1 : 0;
    }
  }
  __syncthreads();  // every read of the old list and the candidates done
  if (r_new < kcap) buf[r_new] = key;
  if (r_old < kcap) buf[r_old] = y;
  __syncthreads();
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, int64_t i) {
  return p[i];
}
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, int64_t i) {
  return bf16_to_f32(p[i]);
}

template <typename T>
__global__ __launch_bounds__(256) void topk_valu_kernel(const T* __restrict__ bank, int64_t bank_stride, int64_t n,
                                                        const T* __restrict__ queries, int64_t q_stride, int32_t d,
                                                        float c2, int64_t self_base, int64_t rows_per_split,
                                                        int n_splits, int kcap, uint64_t* __restrict__ part_keys,
                                                        float2* __restrict__ part_ms,
                                                        float* __restrict__ full_scores,
                                                        const int32_t* __restrict__ row_ns,
                                                        const int32_t* __restrict__ key_ns) {
  __shared__ float qv[kMaxD];
  __shared__ uint64_t buf[2 * kGenericRows];
  __shared__ float red_m[4];
  __shared__ double red_s[4];
  __shared__ int wcount[4];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t q = blockIdx.x / n_splits;
  const int split = static_cast<int>(blockIdx.x % n_splits);
  const int64_t self_row = self_base >= 0 ? self_base + q : -1;
  // scoped selection: candidates are the live rows (row_ns >= 0) of the
  // query's namespace
  const int32_t my_ns = row_ns ? key_ns[q] : 0;

  for (int t = tid; t < d; t += 256) qv[t] = load_elem<T>(queries, q * q_stride + t);
  buf[tid] = 0;
  __syncthreads();

  const int64_t row0 = static_cast<int64_t>(split) * rows_per_split;
  const int64_t row1 = min(n, row0 + rows_per_split);
  float m_run = -INFINITY;
  double s_run = 0.0;

  for (int64_t base = row0; base < row1; base += kGenericRows) {
    const int64_t j = base + tid;
    uint64_t key = 0;
    if (j < row1) {
      const T* row = bank + j * bank_stride;
      float acc = 0.f;
      for (int t = 0; t < d; ++t) acc = fmaf(qv[t], load_elem<T>(row, t), acc);
      const bool cand = j != self_row && (!row_ns || (my_ns >= 0 && row_ns[j] == my_ns));
      // a row outside the candidates gets probability 0 in the full output
      if (full_scores) full_scores[q * n + j] = cand ? acc : -INFINITY;
      if (cand) {
        const float x = acc * c2;
        if (x > m_run) {
          s_run = s_run * static_cast<double>(fast_exp2(m_run - x));
          m_run = x;
        }
        s_run += static_cast<double>(fast_exp2(x - m_run));
        key = make_key(acc, static_cast<uint32_t>(j));
      }
    }
    block_list_insert(buf, key, kcap, wcount);
  }

  // softmax partial: the threads' (m, sum) pairs, within each wave and then
  // across the four waves
  float m_w = m_run;
  for (int off = 32; off > 0; off >>= 1) m_w = fmaxf(m_w, __shfl_xor(m_w, off));
  if (lane == 0) red_m[wave] = m_w;
  __syncthreads();
  const float m_all = fmaxf(fmaxf(red_m[0], red_m[1]), fmaxf(red_m[2], red_m[3]));
  double s_w = (m_run == -INFINITY) ? 0.0 : s_run * static_cast<double>(fast_exp2(m_run - m_all));
  for (int off = 32; off > 0; off >>= 1) s_w += __shfl_xor(s_w, off);
  if (lane == 0) red_s[wave] = s_w;
  __syncthreads();
  const int64_t slot = q * n_splits + split;
  if (tid < kcap) part_keys[slot * kcap + tid] = buf[tid];
  if (tid == 0) part_ms[slot] = make_float2(m_all, static_cast<float>((red_s[0] + red_s[1]) + (red_s[2] + red_s[3])));
}

// One workgroup per query: merge n_splits partial lists of kcap keys
// (consecutive lists list_stride keys apart).
__global__ __launch_bounds__(256) void topk_merge_kernel(const uint64_t* __restrict__ part_keys,
                                                         const float2* __restrict__ part_ms, int n_splits, int kcap,
                                                         int list_stride,
                                                         int k, float c2, int32_t* __restrict__ idx,
                                                         float* __restrict__ score, float* __restrict__ prob,
                                                         float* __restrict__ lse, float* __restrict__ lse2_out) {
  __shared__ uint64_t buf[512];
  __shared__ float red_m[256];
  __shared__ double red_s[256];
  __shared__ int wcount[4];
  const int tid = threadIdx.x;
  const int64_t q = blockIdx.x;
  const float2* ms = part_ms + q * n_splits;

  float m_loc = -INFINITY;
  for (int s = tid; s < n_splits; s += 256) m_loc = fmaxf(m_loc, ms[s].x);
  red_m[tid] = m_loc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red_m[tid] = fmaxf(red_m[tid], red_m[tid + s]);
    __syncthreads();
  }
  const float m_all = red_m[0];
  double s_loc = 0.0;
  for (int s = tid; s < n_splits; s += 256) {
    const float2 v = ms[s];
    if (v.x != -INFINITY) s_loc += static_cast<double>(v.y) * static_cast<double>(fast_exp2(v.x - m_all));
  }
  red_s[tid] = s_loc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (tid < s) red_s[tid] += red_s[tid + s];
    __syncthreads();
  }
  const float lse2 = m_all + static_cast<float>(log2(red_s[0]));

  const uint64_t* keys = part_keys + q * static_cast<int64_t>(n_splits) * list_stride;
  const int64_t total = static_cast<int64_t>(n_splits) * kcap;
  buf[tid] = 0;
  __syncthreads();  // the empty list is in place before its last entry is read
  for (int64_t base = 0; base < total; base += 256) {
    const int64_t i = base + tid;
    const uint64_t key = i < total ? keys[(i / kcap) * list_stride + i % kcap] : 0;
    block_list_insert(buf, key, k, wcount);
  }
  __syncthreads();
  if (tid < k) write_selected(buf[tid], c2, lse2, q * k + tid, idx, score, prob);
  if (tid == 0) {
    if (lse) lse[q] = lse2 * kLn2;
    lse2_out[q] = lse2;
  }
}

// Softmax partials of one query, combined by one wave: lse2 = log2 of the
// normaliser in the scaled log2 domain (max, then the rescaled sum in fp64).
// Up to 64 * kLseRegs partials are read once into registers (one round
// trip); longer rows are read twice.
constexpr int kLseRegs = 8;
__device__ __forceinline__ float wave_lse2(const float2* __restrict__ ms, int n_parts, int lane) {
  float m_loc = -INFINITY;
  double s_loc = 0.0;
  if (n_parts <= 64 * kLseRegs) {
    float2 v[kLseRegs];
#pragma unroll
    for (int j = 0; j < kLseRegs; ++j) {
      const int s = lane + 64 * j;
      v[j] = s < n_parts ? ms[s] : make_float2(-INFINITY, 0.f);
    }
#pragma unroll
    for (int j = 0; j < kLseRegs; ++j) m_loc = fmaxf(m_loc, v[j].x);
    for (int off = 32; off > 0; off >>= 1) m_loc = fmaxf(m_loc, __shfl_xor(m_loc, off));
#pragma unroll
    for (int j = 0; j < kLseRegs; ++j)
      if (v[j].x != -INFINITY) s_loc += static_cast<double>(v[j].y) * static_cast<double>(fast_exp2(v[j].x - m_loc));
  } else {
    for (int s = lane; s < n_parts; s += 64) m_loc = fmaxf(m_loc, ms[s].x);
    for (int off = 32; off > 0; off >>= 1) m_loc = fmaxf(m_loc, __shfl_xor(m_loc, off));
    for (int s = lane; s < n_parts; s += 64) {
      const float2 v = ms[s];
      if (v.x != -INFINITY) s_loc += static_cast<double>(v.y) * static_cast<double>(fast_exp2(v.x - m_loc));
    }
  }
  for (int off = 32; off > 0; off >>= 1) s_loc += __shfl_xor(s_loc, off);
  return m_loc + static_cast<float>(log2(s_loc));
}

// Copy the first k keys of lists [l0, l0 + nl) (list l at keys + l * kcap)
// into dst[(l - l0) * k + j] with one wave, 16 loads in flight per lane.
__device__ __forceinline__ void stage_list_heads(uint64_t* dst, const uint64_t* __restrict__ keys, int l0, int nl,
                                                 int k, int kcap, int lane) {
  constexpr int kU = 16;
  const int total = nl * k;
  for (int base = 0; base < total; base += 64 * kU) {
    uint64_t v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = base + u * 64 + lane;
      v[u] = i < total ? keys[static_cast<int64_t>(l0 + i / k) * kcap + i % k] : 0;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = base + u * 64 + lane;
      if (i < total) dst[i] = v[u];
    }
  }
}

// One wave per key, four keys per workgroup, for few partial lists
// (S * k <= kRankMaxKeys): the first k keys of every list are staged in LDS
// and each staged key finds its rank in the union by a binary search in
// every (descending) list; keys are unique (except empty slots, which rank
// below every real key), so the keys of rank < k are exactly the top-k and
// each lands in its own output slot.
// LDS is sized per launch (rank_lds_bytes): four waves' staged keys and
// chosen keys, so that short rows leave room for more workgroups per CU.
// With `full` set (a bank of at most kRankFullMax rows) the wave also turns
// its query's row of raw scores there into probabilities, saving the
// separate launch of full_prob_kernel (same arithmetic).
constexpr int kRankMaxKeys = 1024;
constexpr int64_t kRankFullMax = 4096;
size_t rank_lds_bytes(int n_parts, int k) {
  return 4 * (static_cast<size_t>(n_parts) * k + kMaxK) * sizeof(uint64_t);
}

__global__ __launch_bounds__(256) void topk_merge_rank_kernel(const uint64_t* __restrict__ part_keys,
                                                              const float2* __restrict__ part_ms, int64_t m,
                                                              int n_parts, int kcap, int k, float c2,
                                                              int32_t* __restrict__ idx, float* __restrict__ score,
                                                              float* __restrict__ prob, float* __restrict__ lse,
                                                              float* __restrict__ lse2_out, float* __restrict__ full,
                                                              int64_t n_full, int64_t self_base) {
  extern __shared__ uint64_t rank_smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * 4 + wave;
  if (q >= m) return;  // whole waves only; no workgroup barrier below
  const int total = n_parts * k;
  uint64_t* st = rank_smem + static_cast<int64_t>(wave) * (total + kMaxK);
  uint64_t* chosen = st + total;
  const uint64_t* keys = part_keys + q * static_cast<int64_t>(n_parts) * kcap;
  // ranks that no key takes (fewer than k candidates) stay empty
  if (lane < k) chosen[lane] = 0;
  const float lse2 = wave_lse2(part_ms + q * n_parts, n_parts, lane);
  stage_list_heads(st, keys, 0, n_parts, k, kcap, lane);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  for (int i = lane; i < total; i += 64) {
    const uint64_t x = st[i];
    if (x == 0) continue;
    int rank = 0;
    for (int s = 0; s < n_parts; ++s) {
      // number of keys > x in list s: first position holding a key <= x
      const uint64_t* l = st + s * k;
      int lo = 0, hi = k;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (l[mid] > x) lo = mid + 1; else hi = mid;
      }
      rank += lo;
    }
    if (rank < k) chosen[rank] = x;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (lane < k) write_selected(chosen[lane], c2, lse2, q * k + lane, idx, score, prob);
  if (lane == 0) {
    if (lse) lse[q] = lse2 * kLn2;
    lse2_out[q] = lse2;
  }
  if (full != nullptr) {
    // 16 values per lane in flight at a time (n_full <= kRankFullMax)
    float* row = full + q * n_full;
    constexpr int kU = 16;
    for (int64_t base = 0; base < n_full; base += 64 * kU) {
      float v[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t j = base + u * 64 + lane;
        v[u] = j < n_full ? row[j] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int64_t j = base + u * 64 + lane;
        if (j < n_full)
          row[j] = ((self_base >= 0 && j == self_base + q) || lse2 == -INFINITY) ? 0.f : fast_exp2(v[u] * c2 - lse2);
      }
    }
  }
}

constexpr size_t kHeadLdsBytes = 160 * 1024;  // dynamic LDS per workgroup (gfx950)

// One workgroup of W waves per key for many partial lists: wave w stages the
// first k keys of lists [w*Lw, (w+1)*Lw) in LDS and reads their top-k off by
// a k-step tournament over the list heads (each lane tracks the best head
// among its lists, the wave takes the maximum, the winning lane advances
// that list); wave 0 then ranks the W sorted results against each other by
// binary search, as in topk_merge_rank_kernel.  LDS is sized per launch.
__global__ __launch_bounds__(512) void topk_merge_multi_kernel(const uint64_t* __restrict__ part_keys,
                                                               const float2* __restrict__ part_ms, int n_parts,
                                                               int lists_per_wave, int kcap, int k, float c2,
                                                               int32_t* __restrict__ idx, float* __restrict__ score,
                                                               float* __restrict__ prob, float* __restrict__ lse,
                                                               float* __restrict__ lse2_out) {
  extern __shared__ uint64_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int W = blockDim.x >> 6;
  const int Lw = lists_per_wave;
  const int64_t q = blockIdx.x;
  uint64_t* heads = smem + static_cast<int64_t>(wave) * Lw * k;      // [Lw][k] of this wave
  uint64_t* tops = smem + static_cast<int64_t>(W) * Lw * k;          // [W][k]
  uint64_t* chosen = tops + W * k;                                   // [k]
  uint16_t* pos = reinterpret_cast<uint16_t*>(chosen + kMaxK) + wave * Lw;
  const int l0 = wave * Lw;
  const int nl = max(0, min(Lw, n_parts - l0));

  const uint64_t* keys = part_keys + q * static_cast<int64_t>(n_parts) * kcap;
  stage_list_heads(heads, keys, l0, nl, k, kcap, lane);
  for (int s = lane; s < nl; s += 64) pos[s] = 0;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  auto local_best = [&](int& best_list) -> uint64_t {
    uint64_t b = 0;
    best_list = -1;
    for (int s = lane; s < nl; s += 64) {
      const int p = pos[s];
      const uint64_t v = p < k ? heads[s * k + p] : 0;
      if (v > b) {
        b = v;
        best_list = s;
      }
    }
    return b;
  };
  int my_list;
  uint64_t my_best = local_best(my_list);
  for (int r = 0; r < k; ++r) {
    const uint64_t w = wave_max_u64(my_best);
    if (lane == 0) tops[wave * k + r] = w;
    if (w != 0 && my_best == w) {  // keys are unique, so exactly one lane wins
      pos[my_list] = static_cast<uint16_t>(pos[my_list] + 1);
      my_best = local_best(my_list);
    }
  }
  // ranks that no key takes (fewer than k candidates) stay empty
  if (wave == 0 && lane < k) chosen[lane] = 0;
  __syncthreads();
  if (wave != 0) return;  // no workgroup barrier below
  const float lse2 = wave_lse2(part_ms + q * n_parts, n_parts, lane);
  for (int i = lane; i < W * k; i += 64) {
    const uint64_t x = tops[i];
    if (x == 0) continue;
    int rank = 0;
    for (int s = 0; s < W; ++s) {
      const uint64_t* l = tops + s * k;
      int lo = 0, hi = k;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (l[mid] > x) lo = mid + 1; else hi = mid;
      }
      rank += lo;
    }
    if (rank < k) chosen[rank] = x;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (lane < k) write_selected(chosen[lane], c2, lse2, q * k + lane, idx, score, prob);
  if (lane == 0) {
    if (lse) lse[q] = lse2 * kLn2;
    lse2_out[q] = lse2;
  }
}

// One wave per key, up to four keys per workgroup (fewer when the lists
// are long), when every key's lists fit in LDS: every split's list is
// sorted, so the top-k of their union is read off by a k-step tournament
// over the list heads -- each lane tracks the best head among its lists, the
// wave takes the maximum, and the winning lane advances that list.  Only the
// first k entries of each list can contribute.  LDS is sized per launch.

__global__ __launch_bounds__(256) void topk_merge_heads_kernel(const uint64_t* __restrict__ part_keys,
                                                               const float2* __restrict__ part_ms, int64_t m,
                                                               int n_splits, int kcap, int k, float c2,
                                                               int32_t* __restrict__ idx, float* __restrict__ score,
                                                               float* __restrict__ prob, float* __restrict__ lse,
                                                               float* __restrict__ lse2_out) {
  extern __shared__ uint64_t smem[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wpb = blockDim.x >> 6;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * wpb + wave;
  const int total = n_splits * k;
  uint64_t* heads = smem + wave * (total + kMaxK);
  uint64_t* chosen = heads + total;
  uint16_t* pos = reinterpret_cast<uint16_t*>(smem + wpb * (total + kMaxK)) + wave * n_splits;
  if (q >= m) return;  // whole waves only; no workgroup barrier below
  const float lse2 = wave_lse2(part_ms + q * n_splits, n_splits, lane);

  // the first k keys of every list; lane l owns lists l, l+64, ...
  const uint64_t* keys = part_keys + q * static_cast<int64_t>(n_splits) * kcap;
  stage_list_heads(heads, keys, 0, n_splits, k, kcap, lane);
  for (int s = lane; s < n_splits; s += 64) pos[s] = 0;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  auto local_best = [&](int& best_list) -> uint64_t {
    uint64_t b = 0;
    best_list = -1;
    for (int s = lane; s < n_splits; s += 64) {
      const int p = pos[s];
      const uint64_t v = p < k ? heads[s * k + p] : 0;
      if (v > b) {
        b = v;
        best_list = s;
      }
    }
    return b;
  };
  int my_list;
  uint64_t my_best = local_best(my_list);
  for (int r = 0; r < k; ++r) {
    const uint64_t w = wave_max_u64(my_best);
    if (lane == 0) chosen[r] = w;
    if (w != 0 && my_best == w) {  // keys are unique, so exactly one lane wins
      pos[my_list] = static_cast<uint16_t>(pos[my_list] + 1);
      my_best = local_best(my_list);
    }
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  if (lane < k) write_selected(chosen[lane], c2, lse2, q * k + lane, idx, score, prob);
  if (lane == 0) {
    if (lse) lse[q] = lse2 * kLn2;
    lse2_out[q] = lse2;
  }
}

__global__ __launch_bounds__(256) void full_prob_kernel(float* __restrict__ full, int64_t n, float c2,
                                                        int64_t self_base, const float* __restrict__ lse2) {
  const int64_t q = blockIdx.y;
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= n) return;
  const float l = lse2[q];
  float* p = full + q * n + j;
  // rows outside the candidates hold -inf scores; with no candidate at all
  // (an empty namespace) lse is -inf and every probability is 0
  *p = ((self_base >= 0 && j == self_base + q) || l == -INFINITY) ? 0.f : fast_exp2(*p * c2 - l);
}

}  // namespace

hipError_t launch_topk_generic(const Plan& p, const void* bank, int64_t bank_stride, int64_t n, const void* queries,
                               int64_t q_stride, int64_t m, int32_t d, int32_t dtype, float c2, int64_t self_base,
                               const Scope& scope, void* ws, float* full_scores, hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  auto* keys = reinterpret_cast<uint64_t*>(w + p.ws_part_keys);
  auto* ms = reinterpret_cast<float2*>(w + p.ws_part_ms);
  const dim3 grid(static_cast<unsigned>(m * p.n_splits));
  if (dtype == 0) {
    topk_valu_kernel<float><<<grid, 256, 0, stream>>>(
        static_cast<const float*>(bank), bank_stride, n, static_cast<const float*>(queries), q_stride, d, c2,
        self_base, p.rows_per_split, p.n_splits, p.kcap, keys, ms, full_scores, scope.row_ns, scope.key_ns);
  } else {
    topk_valu_kernel<uint16_t><<<grid, 256, 0, stream>>>(
        static_cast<const uint16_t*>(bank), bank_stride, n, static_cast<const uint16_t*>(queries), q_stride, d, c2,
        self_base, p.rows_per_split, p.n_splits, p.kcap, keys, ms, full_scores, scope.row_ns, scope.key_ns);
  }
  return hipGetLastError();
}

// Dynamic LDS above the default 64 KiB needs a per-kernel opt-in; it is
// requested once per process and kernel (later calls skip it).
static hipError_t allow_large_lds(const void* fn, int which) {
  static std::atomic<bool> done[2];
  if (done[which].load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e =
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kHeadLdsBytes));
  if (e == hipSuccess) done[which].store(true, std::memory_order_release);
  return e;
}

hipError_t launch_topk_merge(const Plan& p, int64_t m, int32_t k, float c2, int32_t* idx, float* score, float* prob,
                             float* lse, void* ws, hipStream_t stream, const FullProb& fp) {
  // every merge but the fused rank merge leaves the full rows to full_prob_kernel
  auto finish = [&](hipError_t e) -> hipError_t {
    if (e != hipSuccess || fp.full == nullptr) return e;
    return launch_full_prob(p, m, fp.n, c2, fp.self_base, fp.full, ws, stream);
  };
  char* w = static_cast<char*>(ws);
  const auto* keys = reinterpret_cast<const uint64_t*>(w + p.ws_part_keys);
  const auto* ms = reinterpret_cast<const float2*>(w + p.ws_part_ms);
  auto* lse2 = reinterpret_cast<float*>(w + p.ws_lse2);
  const int64_t S = p.n_parts;
  // consecutive lists of a key start kcap_eff keys apart (every part_stride-th slot)
  const int kcap_eff = p.kcap * p.part_stride;
  if (S * k <= kRankMaxKeys && S <= 4) {
    const bool fused = fp.full != nullptr && fp.n <= kRankFullMax;
    topk_merge_rank_kernel<<<dim3(static_cast<unsigned>((m + 3) / 4)), 256, rank_lds_bytes(p.n_parts, k), stream>>>(
        keys, ms, m, p.n_parts, kcap_eff, k, c2, idx, score, prob, lse, lse2, fused ? fp.full : nullptr, fp.n,
        fp.self_base);
    return fused ? hipGetLastError() : finish(hipGetLastError());
  }
  if (S > 64) {
    // W waves per key, each over Lw <= 64 lists (one or a few per lane)
    const int W = static_cast<int>(S >= 512 ? 8 : (S + 63) / 64);
    const int Lw = static_cast<int>((S + W - 1) / W);
    const size_t bytes = (static_cast<size_t>(W) * Lw * k + static_cast<size_t>(W) * k + kMaxK) * sizeof(uint64_t) +
                         static_cast<size_t>(W) * Lw * sizeof(uint16_t);
    if (bytes <= kHeadLdsBytes) {
      if (bytes > 64 * 1024) {
        const hipError_t e = allow_large_lds(reinterpret_cast<const void*>(&topk_merge_multi_kernel), 0);
        if (e != hipSuccess) return e;
      }
      topk_merge_multi_kernel<<<dim3(static_cast<unsigned>(m)), 64 * W, bytes, stream>>>(
          keys, ms, p.n_parts, Lw, kcap_eff, k, c2, idx, score, prob, lse, lse2);
      return finish(hipGetLastError());
    }
  }
  // one wave's heads + chosen keys + list positions
  const size_t per_wave = static_cast<size_t>(S * k + kMaxK) * sizeof(uint64_t) + static_cast<size_t>(S) * sizeof(uint16_t);
  if (per_wave <= kHeadLdsBytes) {
    int wpb = 4;
    while (wpb > 1 && wpb * per_wave > kHeadLdsBytes) wpb /= 2;
    if (wpb * per_wave > 64 * 1024) {
      const hipError_t e = allow_large_lds(reinterpret_cast<const void*>(&topk_merge_heads_kernel), 1);
      if (e != hipSuccess) return e;
    }
    topk_merge_heads_kernel<<<dim3(static_cast<unsigned>((m + wpb - 1) / wpb)), 64 * wpb, wpb * per_wave, stream>>>(
        keys, ms, m, p.n_parts, kcap_eff, k, c2, idx, score, prob, lse, lse2);
    return finish(hipGetLastError());
  }
  topk_merge_kernel<<<dim3(static_cast<unsigned>(m)), 256, 0, stream>>>(keys, ms, p.n_parts, p.kcap, kcap_eff, k, c2, idx,
                                                                         score, prob, lse, lse2);
  return finish(hipGetLastError());
}

hipError_t launch_full_prob(const Plan& p, int64_t m, int64_t n, float c2, int64_t self_base, float* full, void* ws,
                            hipStream_t stream) {
  char* w = static_cast<char*>(ws);
  const dim3 grid(static_cast<unsigned>((n + 255) / 256), static_cast<unsigned>(m));
  full_prob_kernel<<<grid, 256, 0, stream>>>(full, n, c2, self_base, reinterpret_cast<const float*>(w + p.ws_lse2));
  return hipGetLastError();
}

}  // namespace memattn
