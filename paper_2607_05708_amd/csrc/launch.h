// Host-side launchers for the libmemattn kernels and the selection plan.
// Internal to the library: the public interface is include/memattn.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace memattn {

// How one retrieval/relation call is split over the GPU.
struct Plan {
  bool mfma;              // bf16 matrix-core path (else the VALU path)
  int qw;                 // matrix-core workgroup shape: 64 * qw queries (1, 2 or 4)
  int tile_rows;          // bank rows per matrix-core tile (512 for qw = 1, else 256)
  int tile_queries;       // queries per matrix-core workgroup
  int kcap;               // partial list length per split (power of two >= k)
  int n_splits;           // bank splits per query row
  int n_parts;            // partial (list, max, sum) entries per query row seen by the merge
  int part_stride;        // ... at every part_stride-th workspace slot
  int64_t rows_per_split; // bank rows per split (multiple of the row tile)
  int q_tiles;            // query tiles (MFMA path)
  int tiles_per_split;    // bank tiles per split (MFMA path)
  size_t ws_part_keys;    // byte offsets into the workspace
  size_t ws_part_ms;
  size_t ws_lse2;
  int ns;                 // sampled tiles per sampled split (0 = no threshold sample)
  int samp_stride;        // every samp_stride-th split is sampled
  int n_samp_splits;      // sampled splits
  int64_t n_samp;         // sample scores per query (n_samp_splits * ns * tile)
  size_t ws_samp;         // 16-bit sample order keys [m, n_samp]
  size_t ws_t0;           // sampled k-th-best lower bound per query [m]
  size_t ws_thr;          // per-query score bound shared by its partials [m] (order keys)
  int ph_split;           // matrix-core full pass in two launches split at this tile of each split (0: one)
  size_t ws_lane_ms;      // per-slot softmax state between the two launches [m, slots] (float2)
  int order;              // room for the clustered query order (used by relation builds with a sample)
  size_t ws_near;         // best sampled position, then order label, per query [m] (int32)
  size_t ws_perm;         // clustered position -> query [m] (int32)
  size_t ws_olab;         // label of each sampled position [kOrderMaxSample] (int32)
  size_t ws_ocnt;         // queries per label, then each label's first position [kOrderMaxSample] (int32)
  size_t ws_orank;        // each query's rank among its label's queries [m] (int32)
  size_t ws_stop;         // each query's sampled keys at or above its k-th, with positions [m, 64] (uint32)
  size_t ws_qbuf;         // the queries in clustered order [m, d] (bf16)
  size_t ws_bytes;        // total workspace bytes
};

constexpr int kMfmaTile = 256;   // bank rows and query rows per workgroup tile
constexpr int kMfmaMaxK = 32;    // largest k served by the matrix-core path
// Clustered query order: from this many queries on (a wave's 64 lanes can
// then share a region of the bank), while the reordered copy of the queries
// stays within 1 GiB, and for samples of at most 32,768 positions (the order
// kernel's labels live in LDS).
constexpr int64_t kOrderMinQueries = 4096;
constexpr size_t kOrderMaxQueryBytes = size_t{1} << 30;
constexpr int64_t kOrderMaxSample = 32768;
constexpr int64_t kOrderSampleFloor = 1024;  // fewest sampled rows of a relation build in that order
// Matrix-core workgroup shapes by query count: 64 x 512-row tiles (<= 64
// queries), 128 x 256 (<= 128), else 256 x 256; every wave owns 128 rows of
// a tile, so a split keeps tile_rows / 128 partials while the kernel runs.
constexpr int kGenericRows = 256; // bank rows per VALU-path step
constexpr int kMaxK = 64;
constexpr int kMaxD = 8192;

// Namespace scope of a selection (both NULL = the whole bank): row j is a
// candidate of query i only if row_ns[j] >= 0 and row_ns[j] == key_ns[i].
struct Scope {
  const int32_t* row_ns;  // device [n]; negative = tombstoned row
  const int32_t* key_ns;  // device [m]; negative = no candidates
};

// mfma_ok: caller allows the matrix-core path (bf16, d % 32 == 0, k <= 32,
// no full probability output).  relation: the queries are the bank's own
// rows (only the sample size depends on it, never the workspace size).
Plan make_plan(int64_t m, int64_t n, int32_t d, int32_t k, int32_t dtype, bool mfma_ok, bool relation = false);
// Grouped selection over per-namespace chunk tables: the narrow matrix-core
// shape, S splits per namespace (S from the mean table size), no sample.
Plan make_grouped_plan(int64_t m, int32_t n_ns, int64_t n_entries, int32_t k);

// Partial selection over bank splits.  `self_base` >= 0 removes bank row
// self_base + i from query i's candidates.  All launches go to `stream`.
hipError_t launch_topk_generic(const Plan& p, const void* bank, int64_t bank_stride, int64_t n, const void* queries,
                               int64_t q_stride, int64_t m, int32_t d, int32_t dtype, float c2, int64_t self_base,
                               const Scope& scope, void* ws, float* full_scores, hipStream_t stream);
// With p.ns > 0 a sample pass over the first ns tiles of every split first
// bounds each query's k-th best score from below; the full pass starts its
// thresholds there.
// `relation`: query i is bank row i (a relation build); the full pass may
// then take the queries in clustered order (p.order).
hipError_t launch_topk_mfma(const Plan& p, const uint16_t* bank, int64_t bank_stride, int64_t n,
                            const uint16_t* queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                            int64_t self_base, int32_t k, const Scope& scope, bool relation, void* ws,
                            hipStream_t stream);
// Grouped selection over per-namespace chunk tables: workspace regions after
// the plan's (from byte `base` on) and the launch (preparation + matrix-core
// pass; the merge follows with launch_topk_merge).  The plan must be the
// narrow matrix-core shape with n_splits = S splits per namespace.
struct GroupLayout {
  size_t q_cnt, fill, q_off, item_off, bsum, perm, qbuf, bytes;
};
GroupLayout group_layout(int64_t m, int32_t n_ns, int32_t d, size_t base);
hipError_t launch_topk_grouped(const Plan& p, const GroupLayout& G, const uint16_t* bank, int64_t bank_stride,
                               int64_t n, const uint16_t* queries, int64_t q_stride, int64_t m, int32_t d, float c2,
                               int32_t k, const int32_t* ns_off, const int32_t* rows, int32_t n_ns,
                               int64_t n_entries, const int32_t* key_ns, void* ws, hipStream_t stream);
// Optional full probability output: full[i, j] holds the raw score s_ij on
// entry and p_ij on exit (0 for the excluded row self_base + i).
struct FullProb {
  float* full = nullptr;   // device [m, n] or NULL
  int64_t n = 0;
  int64_t self_base = -1;
};
// Merge split partials into the final top-k, probabilities and lse, and
// finish the full probability rows if requested (in the merge's own launch
// for a rank merge over a small bank, else with launch_full_prob after it).
hipError_t launch_topk_merge(const Plan& p, int64_t m, int32_t k, float c2, int32_t* idx, float* score, float* prob,
                             float* lse, void* ws, hipStream_t stream, const FullProb& fp = FullProb{});
// full[i, j] <- exp2(full[i, j] * c2 - lse2[i]) (0 for the excluded row).
hipError_t launch_full_prob(const Plan& p, int64_t m, int64_t n, float c2, int64_t self_base, float* full, void* ws,
                            hipStream_t stream);

hipError_t launch_gather(const void* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                         int64_t n_chunks, int32_t ppc, const int32_t* ids, int64_t count, int32_t order,
                         int32_t group, void* out, hipStream_t stream);

// Budget-aware, time-ordered materialisation of rank-ordered ids [m, k]
// into [m, budget, row_bytes] token rows.
hipError_t launch_gather_budget(const void* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                                int64_t n_chunks, int32_t ppc, const int32_t* tok_len, int32_t row_bytes,
                                const int32_t* ids, int64_t m, int32_t k, int32_t budget, void* out,
                                int32_t* out_tokens, int32_t* out_ids, hipStream_t stream);

// Background block compaction: workspace layout (byte offsets) and the two
// launch phases.  The plan phase leaves {moving pages, fresh pages,
// compacted blocks, malformed-table flag} in totals_host[0..3] and
// synchronises `stream`; the move phase copies the pages and updates the
// directory.
struct CompactLayout {
  int64_t n_blocks;
  size_t live, cand, pos, bsum, ns_base, moves, counter, flags, totals, bytes;
};
CompactLayout compact_layout(int64_t next_free, int32_t P, int64_t n_entries, int32_t ppc, int32_t n_ns);
hipError_t launch_compact_plan(const CompactLayout& L, const int32_t* table, int64_t n_chunks, int32_t ppc,
                               const int32_t* offsets, const int32_t* chunks, int32_t n_ns, int64_t n_entries,
                               int32_t P, int64_t next_free, double theta, float* phi_out, uint8_t* released,
                               void* ws, int64_t* totals_host, hipStream_t stream);
hipError_t launch_compact_move(const CompactLayout& L, void* pool, int64_t page_bytes, int32_t* table,
                               int64_t n_chunks, int32_t ppc, const int32_t* offsets, const int32_t* chunks,
                               int32_t n_ns, int64_t n_entries, int32_t P, int64_t next_free, int64_t first_new,
                               int64_t moved, void* ws, hipStream_t stream);

// Association-aware relocation: workspace layout and the two launch
// phases (the plan leaves {moved chunks, groups} in totals_host and
// synchronises `stream`).
struct ColocLayout {
  size_t owner, klist, cnt, kbase, bsum, counter, totals, bytes;
};
ColocLayout coloc_layout(int64_t m, int32_t k, int64_t n_chunks);
hipError_t launch_coloc_plan(const ColocLayout& L, const int32_t* ids, const float* scores, int64_t m, int32_t k,
                             double tau, int32_t min_group, int64_t n_chunks, void* ws, int64_t* totals_host,
                             hipStream_t stream);
hipError_t launch_coloc_move(const ColocLayout& L, void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table,
                             int32_t ppc, int64_t m, int32_t k, int64_t next_free, int64_t moved, void* ws,
                             hipStream_t stream);

hipError_t launch_append(void* bank, int64_t bank_stride, int64_t n0, const void* new_emb, int64_t new_stride,
                         int64_t m, int32_t d, int32_t elem_bytes, int32_t* table, int32_t ppc, int64_t first_page,
                         hipStream_t stream);

}  // namespace memattn
