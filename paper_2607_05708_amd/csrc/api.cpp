// C ABI of libmemattn.so (declared in include/memattn.h): host-side argument
// validation, the split plan and kernel launches.  Nothing is enqueued
// before all arguments have been checked.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "memattn.h"
#include "launch.h"

namespace memattn {

namespace {

thread_local std::string g_last_error;

mem_status fail(mem_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
mem_status fail(mem_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

mem_status device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return MEM_OK;
  return fail(MEM_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Sample keys per query: at most 32,768 and at most 128 MiB of 16-bit keys.
int64_t sample_cap(int64_t m) {
  const int64_t by_bytes = ((int64_t{64} << 20) / (m > 0 ? m : 1)) / kMfmaTile * kMfmaTile;
  return by_bytes < 32768 ? by_bytes : 32768;
}

int pow2_at_least(int x) {
  int p = 8;
  while (p < x) p <<= 1;
  return p;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

mem_status check_bank(const mem_bank* bank) {
  if (!bank) return fail(MEM_ERR_INVALID_ARG, "bank is NULL");
  if (!bank->emb) return fail(MEM_ERR_INVALID_ARG, "bank->emb is NULL");
  if (bank->dtype != MEM_F32 && bank->dtype != MEM_BF16)
    return fail(MEM_ERR_INVALID_ARG, "bank->dtype %d is neither MEM_F32 nor MEM_BF16", bank->dtype);
  if (bank->d < 1 || bank->d > kMaxD) return fail(MEM_ERR_INVALID_ARG, "d = %d outside [1, %d]", bank->d, kMaxD);
  if (bank->n < 1 || bank->n > INT32_MAX - 1)
    return fail(MEM_ERR_INVALID_ARG, "bank->n = %lld outside [1, 2^31 - 2]", static_cast<long long>(bank->n));
  if (bank->row_stride < bank->d)
    return fail(MEM_ERR_INVALID_ARG, "row_stride %lld < d %d", static_cast<long long>(bank->row_stride), bank->d);
  return MEM_OK;
}

// Scratch memory of the allocation-free retrieval: a file-scope device
// array, one copy per GPU the library runs on, held until the process ends.
// Host code never uses the array's name except to look up its device
// address (hipGetSymbolAddress, once per device, with that device current);
// everything else uses that address.
constexpr size_t kScratchBytes = size_t{128} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array.
mem_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(MEM_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(MEM_ERR_UNSUPPORTED, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(MEM_ERR_DEVICE, "scratch address on device %d: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return MEM_OK;
}

// Shared body of retrieval and relation building.  With use_scratch the
// workspace is the current device's scratch array (ws and ws_bytes are
// ignored); its address is resolved only once every argument has been
// checked.
mem_status select_topk(const mem_bank* bank, const void* queries, int64_t m, int64_t q_stride, int32_t k, float scale,
                       int64_t self_base, const Scope& scope, const mem_topk_out& out, float* full_prob, void* ws,
                       size_t ws_bytes, void* stream, bool use_scratch = false) {
  const int64_t cand = bank->n - (self_base >= 0 ? 1 : 0);
  if (k < 1 || k > kMaxK) return fail(MEM_ERR_INVALID_ARG, "k = %d outside [1, %d]", k, kMaxK);
  // (a scoped selection pads rows with fewer than k candidates instead)
  if (!scope.row_ns && k > cand)
    return fail(MEM_ERR_INVALID_ARG, "k = %d exceeds the %lld candidates per row", k, static_cast<long long>(cand));
  if (!(std::isfinite(scale) && scale > 0.f)) return fail(MEM_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (m < 0) return fail(MEM_ERR_INVALID_ARG, "m < 0");
  if (m == 0) return MEM_OK;
  if (!queries) return fail(MEM_ERR_INVALID_ARG, "queries is NULL");
  if (q_stride < bank->d) return fail(MEM_ERR_INVALID_ARG, "q_stride < d");
  if (!out.idx) return fail(MEM_ERR_INVALID_ARG, "out.idx is NULL");
  if (scope.row_ns && !scope.key_ns) return fail(MEM_ERR_INVALID_ARG, "query namespaces are NULL");

  const bool mfma_ok = bank->dtype == MEM_BF16 && bank->d % 32 == 0 && k <= kMfmaMaxK && full_prob == nullptr &&
                       bank->row_stride % 8 == 0 && q_stride % 8 == 0 && bank->row_stride <= 65536 &&
                       q_stride <= 65536 && aligned16(bank->emb) && aligned16(queries);
  const bool relation = queries == bank->emb && q_stride == bank->row_stride && m == bank->n;
  // (a scoped relation build keeps the bank order, so its sample as well)
  const Plan p = make_plan(m, bank->n, bank->d, k, bank->dtype, mfma_ok, relation && scope.row_ns == nullptr);
  if (static_cast<int64_t>(p.n_splits) * (p.mfma ? p.q_tiles : m) > INT32_MAX)
    return fail(MEM_ERR_UNSUPPORTED, "problem too large for one launch");
  if (m > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "m too large");
  if (use_scratch) {
    if (p.ws_bytes > kScratchBytes)
      return fail(MEM_ERR_WORKSPACE, "this call needs %zu bytes of scratch; the allocation-free call holds %zu",
                  p.ws_bytes, kScratchBytes);
    if (mem_status st = scratch_address(&ws); st != MEM_OK) return st;
    ws_bytes = kScratchBytes;
  }
  if (!ws) return fail(MEM_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < p.ws_bytes)
    return fail(MEM_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, p.ws_bytes);

  hipStream_t s = static_cast<hipStream_t>(stream);
  const float c2 = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
  hipError_t e;
  if (p.mfma) {
    e = launch_topk_mfma(p, static_cast<const uint16_t*>(bank->emb), bank->row_stride, bank->n,
                         static_cast<const uint16_t*>(queries), q_stride, m, bank->d, c2, self_base, k, scope,
                         relation, ws, s);
  } else {
    e = launch_topk_generic(p, bank->emb, bank->row_stride, bank->n, queries, q_stride, m, bank->d, bank->dtype, c2,
                            self_base, scope, ws, full_prob, s);
  }
  if (e != hipSuccess) return device_status(e, "partial selection launch");
  FullProb fp;
  fp.full = full_prob;
  fp.n = bank->n;
  fp.self_base = self_base;
  e = launch_topk_merge(p, m, k, c2, out.idx, out.score, out.prob, out.lse, ws, s, fp);
  if (e != hipSuccess) return device_status(e, "merge launch");
  return MEM_OK;
}

}  // namespace

Plan make_grouped_plan(int64_t m, int32_t n_ns, int64_t n_entries, int32_t k) {
  Plan p{};
  p.mfma = true;
  p.qw = 1;
  p.tile_rows = 512;
  p.tile_queries = 64;
  p.kcap = k <= 8 ? 8 : (k <= 16 ? 16 : 32);
  // Work items are (namespace, 64-query tile, split).  Each active
  // namespace has at least one query tile, so about min(n_ns, m) tiles; aim
  // for about one item per CU (256): a launch just over a multiple of the
  // CU count leaves most CUs idle through its last round.  No more splits
  // than a mean-sized table has 512-row tiles; 1 to 32 splits.
  const int64_t mean = n_entries / (n_ns > 0 ? n_ns : 1);
  const int64_t qt_est = n_ns < m ? (n_ns > 0 ? n_ns : 1) : (m > 0 ? m : 1);
  int64_t S = 256 / qt_est;
  const int64_t mean_tiles = ceil_div(mean, 512);
  S = S > mean_tiles ? mean_tiles : S;
  S = S < 1 ? 1 : (S > 32 ? 32 : S);
  p.n_splits = static_cast<int>(S);
  p.n_parts = p.n_splits;
  p.part_stride = p.tile_rows / 128;
  const size_t mm = static_cast<size_t>(m > 0 ? m : 0);
  const size_t slots = static_cast<size_t>(p.n_splits) * p.part_stride;
  p.ws_part_keys = 0;
  p.ws_part_ms = align256(mm * slots * p.kcap * sizeof(uint64_t));
  p.ws_lse2 = p.ws_part_ms + align256(mm * p.n_splits * 2 * sizeof(float));
  // Threshold sample: the first tile of every table.  It pays where a
  // split's first tile would otherwise merge many stash overflows into a
  // long list (k > 8): always for lists of 32, for lists of 16 only when
  // the mean table spans at least four tiles (else the sample re-reads a
  // large share of each table).  Lists of 8 merge cheaply: no sample.
  p.ns = (p.kcap == 32 || (p.kcap == 16 && mean >= 4 * p.tile_rows)) ? 1 : 0;
  p.samp_stride = 1;
  p.n_samp = p.tile_rows;
  p.ws_samp = p.ws_lse2 + align256(mm * sizeof(float));
  p.ws_t0 = p.ws_samp + align256(mm * static_cast<size_t>(p.n_samp) * sizeof(uint16_t));
  p.ws_thr = p.ws_t0 + align256(mm * sizeof(float));
  p.ph_split = 0;
  p.ws_lane_ms = p.ws_thr + align256(mm * sizeof(uint32_t));
  p.ws_bytes = p.ws_lane_ms;
  return p;
}

Plan make_plan(int64_t m, int64_t n, int32_t d, int32_t k, int32_t dtype, bool mfma_ok, bool relation) {
  Plan p{};
  // The workspace is sized for the most splits any bank of at most n rows
  // can get (min(tiles, split target)), so that the size never decreases
  // with n: a workspace sized for a bank also serves every smaller one.
  int64_t splits_cap = 1;
  const bool mfma = mfma_ok && dtype == MEM_BF16 && d % 32 == 0 && k <= kMfmaMaxK;
  // Whether the workspace holds the clustered query order (m and d only).
  const bool room =
      mfma && m >= kOrderMinQueries && static_cast<size_t>(m) * static_cast<size_t>(d) * 2 <= kOrderMaxQueryBytes;
  if (mfma) {
    p.mfma = true;
    p.qw = m <= 64 ? 1 : (m <= 128 ? 2 : 4);
    p.tile_rows = p.qw == 1 ? 512 : 256;
    p.tile_queries = 64 * p.qw;
    p.kcap = k <= 8 ? 8 : (k <= 16 ? 16 : 32);
    p.q_tiles = static_cast<int>(ceil_div(m, p.tile_queries));
    const int64_t nt = ceil_div(n, p.tile_rows);
    // One workgroup fills a CU, so the grid runs in rounds of 256.  Of the
    // split counts up to s_max, take the fewest that minimise rounds x tiles
    // per split: ceil(256 / q_tiles) splits of a tile count that does not
    // divide 256 overshoot into a second, nearly empty round (48 query tiles
    // x 6 splits = 288 workgroups; 5 splits take one round).  With more
    // than 64 query tiles s_max allows up to four rounds: one split of 157
    // query tiles leaves 99 CUs idle, three take two full rounds.  s_max
    // sizes the workspace (it depends on m, and on n only through nt).
    int64_t s_max = ceil_div(p.q_tiles > 64 ? 1024 : 256, p.q_tiles);
    s_max = s_max < 1 ? 1 : (s_max > nt ? nt : s_max);
    splits_cap = s_max;
    int64_t s = s_max, best = INT64_MAX;
    for (int64_t c = 1; c <= s_max; ++c) {
      const int64_t cost = ceil_div(p.q_tiles * c, 256) * ceil_div(nt, c);
      if (cost < best) {
        best = cost;
        s = c;
      }
    }
    const int64_t tps = ceil_div(nt, s);
    p.tiles_per_split = static_cast<int>(tps);
    p.n_splits = static_cast<int>(ceil_div(nt, tps));
    p.rows_per_split = tps * p.tile_rows;
    // Threshold sample: about n/32 rows per query (4096 to 32768, and never
    // more than sample_cap(m), which sizes the workspace), taken as whole
    // tiles at the start of every samp_stride-th split, ns tiles each.  The
    // sample's k-th best is a lower bound on the query's k-th best.  Skipped
    // when it would cost more than 1/16 of the bank (small banks: each
    // partial's own list then tightens its threshold about as fast), or
    // more than 1/32 with lists of 8, whose merges are cheap.  A relation
    // build in clustered order takes n/32 rows down to 1,024: its keys'
    // neighbours bound them as well, and the coarser sample groups them
    // into fewer, larger clusters (1.8 instead of 2.5 labels per wave on
    // the 32,768-chunk build, 0.09 ms less).  With lists of 16 or 32 such a
    // build takes its sample up to a quarter of the bank: the order then
    // reaches builds of 4,096 to 32,767 keys, which it makes 1.4 to 1.8
    // times faster (lists of 8 gain nothing from it).
    {
      const int64_t floor_rows = (relation && room) ? kOrderSampleFloor : 4096;
      int64_t target = n / 32;
      target = target < floor_rows ? floor_rows : (target > 32768 ? 32768 : target);
      const int64_t cap_tiles = sample_cap(m) / p.tile_rows;
      int64_t want = ceil_div(target, p.tile_rows);
      want = want > cap_tiles ? cap_tiles : want;
      // the sample costs at most 1/max_share of the bank
      const int64_t max_share = (relation && room && p.kcap > 8) ? 4 : (p.kcap == 8 ? 32 : 16);
      if (want >= 1 && want * max_share <= nt) {
        int64_t stride = 1, ns = 1;
        if (want <= p.n_splits) {
          stride = p.n_splits / want;
        } else {
          ns = want / p.n_splits;
          ns = ns > tps ? tps : ns;
        }
        const int64_t sampled = ceil_div(p.n_splits, stride);
        if (sampled * ns <= cap_tiles) {
          p.ns = static_cast<int>(ns);
          p.samp_stride = static_cast<int>(stride);
          p.n_samp_splits = static_cast<int>(sampled);
          p.n_samp = sampled * ns * p.tile_rows;
        }
      }
    }
  } else {
    p.mfma = false;
    p.kcap = pow2_at_least(k);
    const int64_t nt = ceil_div(n, kGenericRows);
    int64_t s = ceil_div(1024, m > 0 ? m : 1);
    s = s < 1 ? 1 : (s > nt ? nt : s);
    splits_cap = s;
    p.rows_per_split = ceil_div(nt, s) * kGenericRows;
    p.n_splits = static_cast<int>(ceil_div(n, p.rows_per_split));
    p.q_tiles = 0;
    p.tiles_per_split = 0;
  }
  // The matrix-core kernel keeps one partial per bank part while it runs and
  // leaves one per split (in part 0's slot); the merge reads every
  // part_stride-th slot.
  p.n_parts = p.n_splits;
  p.part_stride = p.mfma ? p.tile_rows / 128 : 1;
  const size_t slots = static_cast<size_t>(splits_cap > p.n_splits ? splits_cap : p.n_splits) * p.part_stride;
  const size_t mm = static_cast<size_t>(m > 0 ? m : 0);
  p.ws_part_keys = 0;
  p.ws_part_ms = align256(mm * slots * p.kcap * sizeof(uint64_t));
  p.ws_lse2 = p.ws_part_ms + align256(mm * slots * 2 * sizeof(float));
  p.ws_samp = p.ws_lse2 + align256(mm * sizeof(float));
  p.ws_t0 = p.ws_samp + (p.mfma ? align256(mm * static_cast<size_t>(sample_cap(m)) * sizeof(uint16_t)) : 0);
  p.ws_thr = p.ws_t0 + align256(mm * sizeof(float));
  // Two launches per split where a threshold sample is taken and a split
  // spans at least 32 tiles: its first quarter, then the rest, bounded by
  // each query's k-th best over the first quarters of all splits (about a
  // quarter of the bank, against the sample's 1/32).  On the 1M-chunk
  // retrieval the two launches take 0.60 + 1.60 ms against 2.37 ms for one;
  // with shorter splits the extra launch and bound search cost more than
  // the tighter bound saves.
  p.ph_split = (p.mfma && p.ns > 0 && p.tiles_per_split >= 32) ? p.tiles_per_split / 4 : 0;
  p.ws_lane_ms = p.ws_thr + align256(mm * sizeof(uint32_t));
  size_t o = p.ws_lane_ms + (p.mfma ? align256(mm * slots * sizeof(float) * 2) : 0);
  // Clustered query order (a relation build whose queries are many): each
  // query's best sampled position, the order, and the queries copied in it.
  // The room depends on m and d only, so the size still never decreases
  // with n; it is used where a sample is taken.  On the 32,768-chunk
  // relation build the full pass takes 12 % less time in that order.
  p.order = (room && p.ns > 0 && p.n_samp <= kOrderMaxSample) ? 1 : 0;
  if (room) {
    p.ws_near = o;
    o += align256(mm * sizeof(int32_t));
    p.ws_perm = o;
    o += align256(mm * sizeof(int32_t));
    p.ws_olab = o;
    o += align256(static_cast<size_t>(kOrderMaxSample) * sizeof(int32_t));
    p.ws_ocnt = o;
    o += align256(static_cast<size_t>(kOrderMaxSample) * sizeof(int32_t));
    p.ws_orank = o;
    o += align256(mm * sizeof(int32_t));
    p.ws_stop = o;
    o += align256(mm * 64 * sizeof(uint32_t));
    p.ws_qbuf = o;
    o += align256(mm * static_cast<size_t>(d) * 2);
  }
  p.ws_bytes = o;
  return p;
}

}  // namespace memattn

using namespace memattn;

extern "C" {

size_t mem_workspace_bytes(int64_t m, int64_t n, int32_t d, int32_t k, int32_t dtype) {
  if (m < 0 || n < 1 || d < 1 || d > kMaxD || k < 1 || k > kMaxK || (dtype != MEM_F32 && dtype != MEM_BF16))
    return 0;
  const size_t a = make_plan(m, n, d, k, dtype, true).ws_bytes;
  const size_t b = make_plan(m, n, d, k, dtype, false).ws_bytes;
  return a > b ? a : b;
}

mem_status mem_retrieve_topk(const mem_bank* bank, const void* queries, int64_t m, int64_t q_stride, int32_t k,
                             float scale, mem_topk_out out, float* full_prob, void* workspace, size_t ws_bytes,
                             void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  return select_topk(bank, queries, m, q_stride, k, scale, -1, Scope{}, out, full_prob, workspace, ws_bytes, stream);
}

size_t mem_scratch_bytes(void) { return kScratchBytes; }

mem_status mem_retrieve_topk_noalloc(const mem_bank* bank, const void* queries, int64_t m, int64_t q_stride,
                                     int32_t k, float scale, mem_topk_out out, float* full_prob, void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  return select_topk(bank, queries, m, q_stride, k, scale, -1, Scope{}, out, full_prob, nullptr, 0, stream, true);
}

mem_status mem_build_relations(const mem_bank* bank, int32_t k, float scale, int32_t exclude_self,
                               mem_topk_out out, void* workspace, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  return select_topk(bank, bank->emb, bank->n, bank->row_stride, k, scale, exclude_self ? 0 : -1, Scope{}, out,
                     nullptr, workspace, ws_bytes, stream);
}

mem_status mem_retrieve_topk_scoped(const mem_bank* bank, const int32_t* row_ns, const void* queries,
                                    const int32_t* query_ns, int64_t m, int64_t q_stride, int32_t k, float scale,
                                    mem_topk_out out, float* full_prob, void* workspace, size_t ws_bytes,
                                    void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  if (!row_ns) return fail(MEM_ERR_INVALID_ARG, "row_ns is NULL");
  if (m > 0 && !query_ns) return fail(MEM_ERR_INVALID_ARG, "query_ns is NULL");
  if ((reinterpret_cast<uintptr_t>(row_ns) | reinterpret_cast<uintptr_t>(query_ns)) & 3u)
    return fail(MEM_ERR_INVALID_ARG, "row_ns and query_ns must be 4-byte aligned");
  return select_topk(bank, queries, m, q_stride, k, scale, -1, Scope{row_ns, query_ns}, out, full_prob, workspace,
                     ws_bytes, stream);
}

mem_status mem_build_relations_scoped(const mem_bank* bank, const int32_t* row_ns, int32_t k, float scale,
                                      int32_t exclude_self, mem_topk_out out, void* workspace, size_t ws_bytes,
                                      void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  if (!row_ns) return fail(MEM_ERR_INVALID_ARG, "row_ns is NULL");
  if (reinterpret_cast<uintptr_t>(row_ns) & 3u) return fail(MEM_ERR_INVALID_ARG, "row_ns must be 4-byte aligned");
  // every row is a key in its own namespace (a tombstoned key has none)
  return select_topk(bank, bank->emb, bank->n, bank->row_stride, k, scale, exclude_self ? 0 : -1,
                     Scope{row_ns, row_ns}, out, nullptr, workspace, ws_bytes, stream);
}

size_t mem_workspace_bytes_grouped(int64_t m, int32_t n_ns, int64_t n_entries, int32_t d, int32_t k) {
  if (m < 0 || n_ns < 0 || n_entries < 0 || d < 1 || d > kMaxD || k < 1 || k > kMfmaMaxK) return 0;
  const Plan p = make_grouped_plan(m, n_ns, n_entries, k);
  return group_layout(m, n_ns, d, p.ws_bytes).bytes;
}

mem_status mem_retrieve_topk_grouped(const mem_bank* bank, const mem_chunk_tables* tables, const void* queries,
                                     const int32_t* query_ns, int64_t m, int64_t q_stride, int32_t k, float scale,
                                     mem_topk_out out, void* workspace, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (mem_status st = check_bank(bank); st != MEM_OK) return st;
  if (!tables) return fail(MEM_ERR_INVALID_ARG, "tables is NULL");
  const int32_t n_ns = tables->n_ns;
  const int64_t n_entries = tables->n_entries;
  if (n_ns < 0 || n_entries < 0 || n_entries > INT32_MAX)
    return fail(MEM_ERR_INVALID_ARG, "bad namespace or entry count");
  if (n_ns > 0 && !tables->offsets) return fail(MEM_ERR_INVALID_ARG, "tables->offsets is NULL");
  if (n_entries > 0 && (n_ns < 1 || !tables->chunks))
    return fail(MEM_ERR_INVALID_ARG, "chunk tables need chunks and at least one namespace");
  if (k < 1 || k > kMfmaMaxK) return fail(MEM_ERR_INVALID_ARG, "k = %d outside [1, %d]", k, kMfmaMaxK);
  if (!(std::isfinite(scale) && scale > 0.f)) return fail(MEM_ERR_INVALID_ARG, "scale must be finite and > 0");
  if (m < 0) return fail(MEM_ERR_INVALID_ARG, "m < 0");
  if (m == 0) return MEM_OK;
  if (!queries || !query_ns) return fail(MEM_ERR_INVALID_ARG, "queries or query_ns is NULL");
  if (q_stride < bank->d) return fail(MEM_ERR_INVALID_ARG, "q_stride < d");
  if (!out.idx) return fail(MEM_ERR_INVALID_ARG, "out.idx is NULL");
  if (reinterpret_cast<uintptr_t>(query_ns) & 3u) return fail(MEM_ERR_INVALID_ARG, "query_ns must be 4-byte aligned");
  if (bank->dtype != MEM_BF16 || bank->d % 32 != 0 || bank->d < 96 || bank->row_stride % 8 != 0 ||
      q_stride % 8 != 0 || bank->row_stride > 65536 || !aligned16(bank->emb) || !aligned16(queries))
    return fail(MEM_ERR_UNSUPPORTED,
                "grouped retrieval needs bf16 rows with d a multiple of 32 and >= 96, strides a multiple of 8 "
                "(at most 65536) and 16-byte aligned data; mem_retrieve_topk_scoped serves other shapes");
  if (bank->n * bank->row_stride * 2 > (int64_t{1} << 32) - 4096)
    return fail(MEM_ERR_UNSUPPORTED, "grouped retrieval addresses at most 4 GiB of bank rows");
  const Plan p = make_grouped_plan(m, n_ns, n_entries, k);
  const GroupLayout G = group_layout(m, n_ns, bank->d, p.ws_bytes);
  const int64_t bound = (ceil_div(m, 64) + (m < n_ns ? m : n_ns)) * p.n_splits;
  if (bound > INT32_MAX || m > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "problem too large for one launch");
  if (!workspace) return fail(MEM_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < G.bytes) return fail(MEM_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, G.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const float c2 = static_cast<float>(static_cast<double>(scale) * 1.4426950408889634);
  // (with no namespace at all every query is padded: no work item runs and
  // the merge sees empty partials)
  hipError_t e = launch_topk_grouped(p, G, static_cast<const uint16_t*>(bank->emb), bank->row_stride, bank->n,
                                     static_cast<const uint16_t*>(queries), q_stride, m, bank->d, c2, k,
                                     tables->offsets, tables->chunks, n_ns, n_entries, query_ns, workspace, s);
  if (e != hipSuccess) return device_status(e, "grouped selection launch");
  e = launch_topk_merge(p, m, k, c2, out.idx, out.score, out.prob, out.lse, workspace, s);
  if (e != hipSuccess) return device_status(e, "merge launch");
  return MEM_OK;
}

mem_status mem_gather_chunks(const mem_pages* pages, const int32_t* ids, int64_t count, int32_t order, int32_t group,
                             void* out, void* stream) {
  g_last_error.clear();
  if (!pages) return fail(MEM_ERR_INVALID_ARG, "pages is NULL");
  if (count < 0) return fail(MEM_ERR_INVALID_ARG, "count < 0");
  if (order != MEM_ORDER_RANK && order != MEM_ORDER_TIME) return fail(MEM_ERR_INVALID_ARG, "unknown order %d", order);
  if (order == MEM_ORDER_TIME && (group < 1 || group > 1024))
    return fail(MEM_ERR_INVALID_ARG, "group = %d outside [1, 1024]", group);
  if (pages->page_bytes <= 0 || pages->page_bytes % 16 != 0)
    return fail(MEM_ERR_INVALID_ARG, "page_bytes must be a positive multiple of 16");
  if (pages->pages_per_chunk < 1 || pages->pages_per_chunk > 64)
    return fail(MEM_ERR_INVALID_ARG, "pages_per_chunk outside [1, 64]");
  if (pages->n_pages < 0 || pages->n_chunks < 0) return fail(MEM_ERR_INVALID_ARG, "negative pool or table size");
  if (count == 0) return MEM_OK;
  if (!pages->pool || !pages->table || !ids || !out) return fail(MEM_ERR_INVALID_ARG, "NULL pool, table, ids or out");
  if (!aligned16(pages->pool) || !aligned16(out)) return fail(MEM_ERR_INVALID_ARG, "pool and out must be 16-byte aligned");
  if (count * pages->pages_per_chunk > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "count too large for one launch");
  const uintptr_t o0 = reinterpret_cast<uintptr_t>(out);
  const uintptr_t o1 = o0 + static_cast<uintptr_t>(count * pages->pages_per_chunk * pages->page_bytes);
  const uintptr_t p0 = reinterpret_cast<uintptr_t>(pages->pool);
  const uintptr_t p1 = p0 + static_cast<uintptr_t>(pages->n_pages * pages->page_bytes);
  if (o0 < p1 && p0 < o1) return fail(MEM_ERR_INVALID_ARG, "out overlaps the page pool");
  return device_status(launch_gather(pages->pool, pages->n_pages, pages->page_bytes, pages->table, pages->n_chunks,
                                     pages->pages_per_chunk, ids, count, order, order == MEM_ORDER_TIME ? group : 1,
                                     out, static_cast<hipStream_t>(stream)),
                       "gather launch");
}

mem_status mem_gather_budget(const mem_pages* pages, const int32_t* tok_len, int32_t row_bytes, const int32_t* ids,
                             int64_t m, int32_t k, int32_t budget_tokens, void* out, int32_t* out_tokens,
                             int32_t* out_ids, void* stream) {
  g_last_error.clear();
  if (!pages) return fail(MEM_ERR_INVALID_ARG, "pages is NULL");
  if (pages->page_bytes <= 0 || pages->page_bytes % 16 != 0)
    return fail(MEM_ERR_INVALID_ARG, "page_bytes must be a positive multiple of 16");
  if (pages->pages_per_chunk < 1 || pages->pages_per_chunk > 64)
    return fail(MEM_ERR_INVALID_ARG, "pages_per_chunk outside [1, 64]");
  if (pages->n_pages < 0 || pages->n_chunks < 0) return fail(MEM_ERR_INVALID_ARG, "negative pool or table size");
  if (row_bytes <= 0 || row_bytes % 16 != 0 || pages->page_bytes % row_bytes != 0)
    return fail(MEM_ERR_INVALID_ARG, "row_bytes must be a positive multiple of 16 that divides page_bytes");
  if (pages->page_bytes / row_bytes * pages->pages_per_chunk > (INT32_MAX / 64))
    return fail(MEM_ERR_UNSUPPORTED, "too many token rows per chunk");
  if (k < 1 || k > 64) return fail(MEM_ERR_INVALID_ARG, "k = %d outside [1, 64]", k);
  if (m < 0) return fail(MEM_ERR_INVALID_ARG, "m < 0");
  if (budget_tokens < 0) return fail(MEM_ERR_INVALID_ARG, "budget_tokens < 0");
  if (m == 0) return MEM_OK;
  if (!pages->pool || !pages->table || !tok_len || !ids || !out_tokens)
    return fail(MEM_ERR_INVALID_ARG, "NULL pool, table, tok_len, ids or out_tokens");
  if (budget_tokens > 0 && !out) return fail(MEM_ERR_INVALID_ARG, "out is NULL");
  if (!aligned16(pages->pool) || (out && !aligned16(out)))
    return fail(MEM_ERR_INVALID_ARG, "pool and out must be 16-byte aligned");
  const int64_t blocks = m * ((static_cast<int64_t>(budget_tokens) + 511) / 512 + 1);
  if (blocks > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "m * budget too large for one launch");
  if (out) {
    const uintptr_t o0 = reinterpret_cast<uintptr_t>(out);
    const uintptr_t o1 = o0 + static_cast<uintptr_t>(m * budget_tokens * static_cast<int64_t>(row_bytes));
    const uintptr_t p0 = reinterpret_cast<uintptr_t>(pages->pool);
    const uintptr_t p1 = p0 + static_cast<uintptr_t>(pages->n_pages * pages->page_bytes);
    if (o0 < p1 && p0 < o1) return fail(MEM_ERR_INVALID_ARG, "out overlaps the page pool");
  }
  return device_status(launch_gather_budget(pages->pool, pages->n_pages, pages->page_bytes, pages->table,
                                            pages->n_chunks, pages->pages_per_chunk, tok_len, row_bytes, ids, m, k,
                                            budget_tokens, out, out_tokens, out_ids,
                                            static_cast<hipStream_t>(stream)),
                       "budget gather launch");
}

size_t mem_compact_workspace_bytes(int64_t next_free_page, int32_t pages_per_block, int64_t n_entries,
                                   int32_t pages_per_chunk, int32_t n_ns) {
  if (next_free_page < 0 || pages_per_block < 1 || n_entries < 0 || pages_per_chunk < 1 || pages_per_chunk > 64 ||
      n_ns < 0)
    return 0;
  return compact_layout(next_free_page, pages_per_block, n_entries, pages_per_chunk, n_ns).bytes;
}

mem_status mem_compact_blocks(void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table, int64_t n_chunks,
                              int32_t pages_per_chunk, const mem_chunk_tables* tables, int32_t pages_per_block,
                              float theta, int64_t next_free_page, float* phi, uint8_t* released,
                              mem_compact_result* result, void* workspace, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!result) return fail(MEM_ERR_INVALID_ARG, "result is NULL");
  if (!tables) return fail(MEM_ERR_INVALID_ARG, "tables is NULL");
  if (!pool || !aligned16(pool)) return fail(MEM_ERR_INVALID_ARG, "pool is NULL or not 16-byte aligned");
  if (page_bytes <= 0 || page_bytes % 16 != 0)
    return fail(MEM_ERR_INVALID_ARG, "page_bytes must be a positive multiple of 16");
  if (pages_per_chunk < 1 || pages_per_chunk > 64) return fail(MEM_ERR_INVALID_ARG, "pages_per_chunk outside [1, 64]");
  if (n_chunks < 0 || (n_chunks > 0 && !table)) return fail(MEM_ERR_INVALID_ARG, "bad table");
  if (n_pages < 0 || n_pages > INT32_MAX) return fail(MEM_ERR_INVALID_ARG, "n_pages outside [0, 2^31 - 1]");
  if (next_free_page < 0 || next_free_page > n_pages)
    return fail(MEM_ERR_INVALID_ARG, "next_free_page outside [0, n_pages]");
  if (pages_per_block < 1) return fail(MEM_ERR_INVALID_ARG, "pages_per_block < 1");
  if (!std::isfinite(theta)) return fail(MEM_ERR_INVALID_ARG, "theta must be finite");
  const int32_t n_ns = tables->n_ns;
  const int64_t n_entries = tables->n_entries;
  if (n_ns < 0 || n_entries < 0) return fail(MEM_ERR_INVALID_ARG, "negative namespace or entry count");
  if (n_entries > 0 && (n_ns < 1 || !tables->offsets || !tables->chunks))
    return fail(MEM_ERR_INVALID_ARG, "chunk tables need offsets, chunks and at least one namespace");
  if (n_entries * pages_per_chunk > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "too many chunk-table entries");
  const CompactLayout L = compact_layout(next_free_page, pages_per_block, n_entries, pages_per_chunk, n_ns);
  if (!workspace) return fail(MEM_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < L.bytes) return fail(MEM_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, L.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // moving pages, fresh pages, compacted blocks and malformed-table flag (int32s, low halves)
  int64_t totals[4] = {0, 0, 0, 0};
  mem_status st = device_status(launch_compact_plan(L, table, n_chunks, pages_per_chunk, tables->offsets,
                                                    tables->chunks, n_ns, n_entries, pages_per_block,
                                                    next_free_page, static_cast<double>(theta), phi, released,
                                                    workspace, totals, s),
                                "compaction plan");
  if (st != MEM_OK) return st;
  if (totals[3] != 0)
    return fail(MEM_ERR_INVALID_ARG,
                "chunk tables malformed (offsets must run from 0 to n_entries without falling; ids must be valid and "
                "ascending within a namespace)");
  const int64_t moved = totals[0];
  const int64_t first_new = L.n_blocks * pages_per_block;
  const int64_t end = first_new + totals[1];
  if (moved > 0 && end > n_pages)
    return fail(MEM_ERR_INVALID_ARG, "compaction needs pages up to %lld but the pool has %lld",
                static_cast<long long>(end), static_cast<long long>(n_pages));
  st = device_status(launch_compact_move(L, pool, page_bytes, table, n_chunks, pages_per_chunk, tables->offsets,
                                         tables->chunks, n_ns, n_entries, pages_per_block, next_free_page, first_new,
                                         moved, workspace, s),
                     "compaction move");
  if (st != MEM_OK) return st;
  result->moved_pages = moved;
  result->released_blocks = static_cast<int32_t>(totals[2]);
  result->next_free_page = moved > 0 ? end : next_free_page;
  return MEM_OK;
}

size_t mem_colocate_workspace_bytes(int64_t m, int32_t k, int64_t n_chunks) {
  if (m < 0 || k < 1 || k > 64 || n_chunks < 0) return 0;
  return coloc_layout(m, k, n_chunks).bytes;
}

mem_status mem_colocate(void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table, int64_t n_chunks,
                        int32_t pages_per_chunk, const int32_t* ids, const float* scores, int64_t m, int32_t k,
                        float tau, int32_t min_group, int64_t next_free_page, mem_colocate_result* result,
                        void* workspace, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!result) return fail(MEM_ERR_INVALID_ARG, "result is NULL");
  if (!pool || !aligned16(pool)) return fail(MEM_ERR_INVALID_ARG, "pool is NULL or not 16-byte aligned");
  if (page_bytes <= 0 || page_bytes % 16 != 0)
    return fail(MEM_ERR_INVALID_ARG, "page_bytes must be a positive multiple of 16");
  if (pages_per_chunk < 1 || pages_per_chunk > 64) return fail(MEM_ERR_INVALID_ARG, "pages_per_chunk outside [1, 64]");
  if (n_chunks < 0 || (n_chunks > 0 && !table)) return fail(MEM_ERR_INVALID_ARG, "bad table");
  if (n_pages < 0 || n_pages > INT32_MAX) return fail(MEM_ERR_INVALID_ARG, "n_pages outside [0, 2^31 - 1]");
  if (next_free_page < 0 || next_free_page > n_pages)
    return fail(MEM_ERR_INVALID_ARG, "next_free_page outside [0, n_pages]");
  if (k < 1 || k > 64) return fail(MEM_ERR_INVALID_ARG, "k = %d outside [1, 64]", k);
  if (m < 0) return fail(MEM_ERR_INVALID_ARG, "m < 0");
  if (min_group < 1) return fail(MEM_ERR_INVALID_ARG, "min_group < 1");
  if (!std::isfinite(tau)) return fail(MEM_ERR_INVALID_ARG, "tau must be finite");
  if (m > 0 && (!ids || !scores)) return fail(MEM_ERR_INVALID_ARG, "ids or scores is NULL");
  if (m * k * pages_per_chunk > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "too many selections for one call");
  const ColocLayout L = coloc_layout(m, k, n_chunks);
  if (!workspace) return fail(MEM_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < L.bytes) return fail(MEM_ERR_WORKSPACE, "workspace of %zu bytes < %zu needed", ws_bytes, L.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int64_t totals[2] = {0, 0};  // moved chunks, groups (int32, low half)
  mem_status st = device_status(launch_coloc_plan(L, ids, scores, m, k, static_cast<double>(tau), min_group, n_chunks,
                                                  workspace, totals, s),
                                "relocation plan");
  if (st != MEM_OK) return st;
  const int64_t moved = totals[0];
  const int64_t end = next_free_page + moved * pages_per_chunk;
  if (end > n_pages)
    return fail(MEM_ERR_INVALID_ARG, "relocation needs pages up to %lld but the pool has %lld",
                static_cast<long long>(end), static_cast<long long>(n_pages));
  st = device_status(launch_coloc_move(L, pool, n_pages, page_bytes, table, pages_per_chunk, m, k, next_free_page, moved,
                                       workspace, s),
                     "relocation move");
  if (st != MEM_OK) return st;
  result->moved_chunks = moved;
  result->groups = static_cast<int32_t>(totals[1]);
  result->next_free_page = end;
  return MEM_OK;
}

mem_status mem_append_chunks(mem_bank* bank, int64_t capacity_rows, const void* new_emb, int64_t m,
                             int64_t new_stride, int32_t* table, int32_t pages_per_chunk, int64_t* next_free_page,
                             int64_t n_pages_cap, void* stream) {
  g_last_error.clear();
  if (!bank || !bank->emb) return fail(MEM_ERR_INVALID_ARG, "bank or bank->emb is NULL");
  if (bank->dtype != MEM_F32 && bank->dtype != MEM_BF16) return fail(MEM_ERR_INVALID_ARG, "bad bank dtype");
  if (bank->d < 1 || bank->d > kMaxD || bank->row_stride < bank->d || bank->n < 0)
    return fail(MEM_ERR_INVALID_ARG, "bad bank shape");
  if (m < 0) return fail(MEM_ERR_INVALID_ARG, "m < 0");
  if (!table || !next_free_page) return fail(MEM_ERR_INVALID_ARG, "table or next_free_page is NULL");
  if (pages_per_chunk < 1 || pages_per_chunk > 64) return fail(MEM_ERR_INVALID_ARG, "pages_per_chunk outside [1, 64]");
  if (*next_free_page < 0) return fail(MEM_ERR_INVALID_ARG, "*next_free_page < 0");
  if (bank->n + m > capacity_rows) return fail(MEM_ERR_INVALID_ARG, "bank capacity exceeded");
  if (bank->n + m > INT32_MAX - 1) return fail(MEM_ERR_UNSUPPORTED, "more than 2^31 - 2 chunks");
  const int64_t pages_needed = m * pages_per_chunk;
  if (*next_free_page + pages_needed > n_pages_cap) return fail(MEM_ERR_INVALID_ARG, "page pool exhausted");
  if (*next_free_page + pages_needed > INT32_MAX) return fail(MEM_ERR_UNSUPPORTED, "page ids exceed int32");
  if (m == 0) return MEM_OK;
  if (!new_emb) return fail(MEM_ERR_INVALID_ARG, "new_emb is NULL");
  if (new_stride < bank->d) return fail(MEM_ERR_INVALID_ARG, "new_stride < d");
  const int elem = bank->dtype == MEM_BF16 ? 2 : 4;
  const mem_status st = device_status(
      launch_append(const_cast<void*>(bank->emb), bank->row_stride, bank->n, new_emb, new_stride, m, bank->d, elem,
                    table, pages_per_chunk, *next_free_page, static_cast<hipStream_t>(stream)),
      "append launch");
  if (st != MEM_OK) return st;
  bank->n += m;
  *next_free_page += pages_needed;
  return MEM_OK;
}

const char* mem_status_string(mem_status s) {
  switch (s) {
    case MEM_OK:
      return "ok";
    case MEM_ERR_INVALID_ARG:
      return "invalid argument";
    case MEM_ERR_UNSUPPORTED:
      return "unsupported request";
    case MEM_ERR_WORKSPACE:
      return "workspace missing or too small";
    case MEM_ERR_DEVICE:
      return "device error";
  }
  return "unknown status";
}

const char* mem_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
