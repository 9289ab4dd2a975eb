/*
 * memattn.h -- C ABI of libmemattn.so: dense MemAttention retrieval and
 * chunk materialisation on one AMD Instinct MI355X (gfx950).
 *
 * The calls follow the paper's statement of MemAttention (Algorithm 1) and
 * of the Memory Manager's block directory (Section 4.2):
 *
 *   mem_retrieve_topk    LLMSelect(K_q, M, p) of query-aware retrieval, in the
 *                        Dense-only form of the Section 5.5 ablation:
 *                        s_ij = <q_i, b_j>, softmax over the bank, top-k by s.
 *   mem_build_relations  LLMSelect(K_m, M, p) of cross-chunk reconciliation,
 *                        applied to every chunk of the bank against all others.
 *   mem_gather_chunks    FetchByID + SortByTime: materialise the selected
 *                        chunks' token blocks through the page table.
 *   mem_append_chunks    Insert: append chunk records (embedding row + pages
 *                        from an append-only bump allocator).
 *   mem_retrieve_topk_scoped, mem_build_relations_scoped
 *                        the selections restricted to each key's (user,
 *                        session) namespace T[u][s] and to live rows.
 *   mem_retrieve_topk_grouped
 *                        the scoped retrieval over per-namespace chunk
 *                        tables, scoring each query against its own table only.
 *   mem_gather_budget    FetchByID + SortByTime + Concat within a memory
 *                        token budget (Section 4.3), as packed token rows.
 *   mem_compact_blocks   background block compaction: invalid ratio of
 *                        Eq. 2, live pages repacked per namespace in time
 *                        order (Algorithm 2).
 *   mem_colocate         association-aware relocation: each key's strongly
 *                        related retrieved chunks rewritten together, in time
 *                        order, into fresh pages (Algorithm 2, online stage).
 *
 * Conventions shared by every call
 *   - Pointers are DEVICE pointers unless marked HOST.  The caller owns every
 *     buffer, including the workspace; the library allocates no device
 *     memory and keeps no state between calls except a thread-local
 *     last-error message.
 *   - `stream` is a hipStream_t passed as void* (NULL = default stream).  All
 *     device work is enqueued on it; calls return before it completes
 *     (mem_compact_blocks and mem_colocate wait once for their plans, as
 *     documented).
 *   - Arguments are validated on the host before anything is enqueued; a
 *     negative mem_status is returned and nothing is launched.  A failed
 *     launch returns MEM_ERR_DEVICE.  Faults inside kernels surface at the
 *     caller's next synchronisation.
 *   - Embeddings are row-major, `row_stride` elements apart, in fp32 or bf16
 *     (raw bf16 bit patterns).  Scores accumulate in fp32.
 *   - Ids are int32 bank row numbers; a chunk's id is its append order, so
 *     ascending id is chronological order.
 */
#ifndef MEMATTN_H
#define MEMATTN_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define MEMATTN_API __attribute__((visibility("default")))
#else
#define MEMATTN_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MEM_OK = 0,
  MEM_ERR_INVALID_ARG = -1, /* null pointer, size or value out of range */
  MEM_ERR_UNSUPPORTED = -2, /* valid request the library does not implement */
  MEM_ERR_WORKSPACE = -3,   /* workspace missing or smaller than mem_workspace_bytes() */
  MEM_ERR_DEVICE = -4       /* a HIP call or kernel launch failed */
} mem_status;

typedef enum { MEM_F32 = 0, MEM_BF16 = 1 } mem_dtype;

typedef enum {
  MEM_ORDER_RANK = 0, /* ids as given (rank order from mem_retrieve_topk) */
  MEM_ORDER_TIME = 1  /* ascending id within each group: SortByTime of Algorithm 1 */
} mem_order;

/* The resident memory bank: one embedding row per chunk (the chunk table of
 * Algorithm 1 with keyword metadata replaced by embeddings). */
typedef struct {
  const void* emb;    /* device [n rows, row_stride elements], dtype below */
  int64_t n;          /* rows in the bank, >= 1 */
  int32_t d;          /* embedding dimension, 1..8192 */
  int32_t dtype;      /* mem_dtype */
  int64_t row_stride; /* elements between consecutive rows, >= d */
} mem_bank;

/* Per-row selection results; rows in rank order (score descending, then id
 * ascending). */
typedef struct {
  int32_t* idx; /* device [m, k] selected chunk ids; required */
  float* score; /* device [m, k] raw scores s_ij (fp32); may be NULL */
  float* prob;  /* device [m, k] p_ij = exp(scale*s_ij - lse_i); may be NULL */
  float* lse;   /* device [m] lse_i = log sum_{j in J_i} exp(scale*s_ij); may be NULL */
} mem_topk_out;

/* Block directory (Section 4.2): logical chunk -> physical pages. */
typedef struct {
  const void* pool;        /* device, n_pages * page_bytes bytes */
  int64_t n_pages;         /* pages in the pool */
  int64_t page_bytes;      /* bytes per page; a positive multiple of 16 */
  const int32_t* table;    /* device [n_chunks, pages_per_chunk] physical page ids */
  int64_t n_chunks;        /* rows of `table` */
  int32_t pages_per_chunk; /* 1..64 */
} mem_pages;

/*
 * Device workspace needed by mem_retrieve_topk (m queries) or
 * mem_build_relations (m = n) for these sizes.  Depends only on the
 * arguments and never decreases with n, so a workspace sized for a bank's
 * capacity serves it as it grows; 0 on invalid sizes.  The workspace holds per-split partial
 * top-k lists and softmax partial sums (and, for m >= 4,096 bf16 queries, a
 * reordered copy of the queries: a relation build scores them grouped by
 * region of the bank) and is fully rewritten by each call;
 * calls that share a workspace must not overlap (enqueue them on one stream).
 */
MEMATTN_API size_t mem_workspace_bytes(int64_t m, int64_t n, int32_t d, int32_t k, int32_t dtype);

/*
 * Query-aware retrieval (Algorithm 1, query side; Dense-only relevance of
 * Section 5.5).  For each query row i of `queries` ([m, q_stride] elements,
 * same dtype and d as the bank):
 *   s_ij  = sum_t q_it * b_jt  over all bank rows j (candidate set J_i = bank)
 *   lse_i = log sum_j exp(scale * s_ij)
 *   top-k = the k rows with the largest s_ij, ties to the lower id.
 * Selection uses s, not p; `scale` is the softmax inverse temperature (> 0,
 * finite) and does not change which ids are selected.
 * 1 <= k <= 64 and k <= n.  `full_prob` (nullable, device [m, n] fp32)
 * receives p_ij for every bank row; requesting it selects the VALU path.
 * The workspace must be at least mem_workspace_bytes(m, n, d, k, dtype).
 */
MEMATTN_API mem_status mem_retrieve_topk(const mem_bank* bank, const void* queries, int64_t m, int64_t q_stride, int32_t k,
                             float scale, mem_topk_out out, float* full_prob, void* workspace, size_t ws_bytes,
                             void* stream);

/*
 * mem_retrieve_topk without a workspace argument and without any device
 * allocation, for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, kernels, results and errors as mem_retrieve_topk; the
 * workspace is instead a fixed scratch array of mem_scratch_bytes() bytes
 * (128 MiB) that the library holds in every GPU it runs on until the
 * process ends.  Calls whose workspace (mem_workspace_bytes) exceeds it
 * fail with MEM_ERR_WORKSPACE before anything is enqueued (up to 1,024
 * queries fit at any bank size and k).  The first call on a device
 * looks up the array's address there (make that first call outside graph
 * capture); later calls only enqueue kernels.  Every call on one GPU shares
 * that GPU's array, which keeps the last call's contents (the kernels
 * initialise what they read): calls that overlap on one GPU (different
 * streams, or different host threads) race and must not be issued.
 */
MEMATTN_API mem_status mem_retrieve_topk_noalloc(const mem_bank* bank, const void* queries, int64_t m,
                                                 int64_t q_stride, int32_t k, float scale, mem_topk_out out,
                                                 float* full_prob, void* stream);

/* Size in bytes of the scratch array behind mem_retrieve_topk_noalloc. */
MEMATTN_API size_t mem_scratch_bytes(void);

/*
 * Cross-chunk relation building (Algorithm 1, compaction side): every bank
 * row is a key against the whole bank.  Outputs are [n, k] and [n].  With
 * exclude_self != 0 row i is removed from its own candidates (J_i = bank
 * minus {i}), in the softmax as well as the top-k; then k <= n - 1.
 * Same rules as mem_retrieve_topk otherwise.
 */
MEMATTN_API mem_status mem_build_relations(const mem_bank* bank, int32_t k, float scale, int32_t exclude_self,
                               mem_topk_out out, void* workspace, size_t ws_bytes, void* stream);

/*
 * Namespace-scoped retrieval.  Algorithm 1 selects from the chunk table of
 * the request's own (user, session) namespace, T[u][s] (Section 4.1), and
 * out-of-place updates leave the old copy of a chunk behind as an invalid
 * (tombstoned) entry (Section 4.2).  With one bank shared by all namespaces:
 *   row_ns   device int32 [bank->n]: namespace id of each bank row; a
 *            negative value marks a tombstoned row (never a candidate).
 *   query_ns device int32 [m]: namespace id of each query; a negative value
 *            gives the query no candidates.
 * J_i = { j : row_ns[j] >= 0 and row_ns[j] == query_ns[i] }; scores, lse_i,
 * p_ij and the top-k are those of mem_retrieve_topk restricted to J_i.  A row
 * with fewer than k candidates is padded with id -1, score -inf and p 0
 * (k may then exceed |J_i|, even n); an empty J_i gives lse_i = -inf.
 * `full_prob` rows hold 0 outside J_i.  Both arrays are 4-byte aligned and
 * only read.  Same workspace size and other rules as mem_retrieve_topk.
 */
MEMATTN_API mem_status mem_retrieve_topk_scoped(const mem_bank* bank, const int32_t* row_ns, const void* queries,
                                    const int32_t* query_ns, int64_t m, int64_t q_stride, int32_t k, float scale,
                                    mem_topk_out out, float* full_prob, void* workspace, size_t ws_bytes,
                                    void* stream);

/*
 * Namespace-scoped relation building: mem_build_relations where row i's
 * candidates are the live rows of its own namespace, J_i = { j :
 * row_ns[j] >= 0 and row_ns[j] == row_ns[i] } (minus i itself with
 * exclude_self != 0).  A tombstoned row (row_ns[i] < 0) has no candidates:
 * its output row is all padding and its lse is -inf.  Padding as in
 * mem_retrieve_topk_scoped; k <= 64 with no bound from n.
 */
MEMATTN_API mem_status mem_build_relations_scoped(const mem_bank* bank, const int32_t* row_ns, int32_t k, float scale,
                                      int32_t exclude_self, mem_topk_out out, void* workspace, size_t ws_bytes,
                                      void* stream);

/* Per-namespace chunk tables T[u][s] (Section 4.1) as one CSR structure:
 * namespace u's live chunks are chunks[offsets[u] .. offsets[u + 1]). */
typedef struct {
  const int32_t* offsets; /* device int32 [n_ns + 1], non-decreasing, offsets[0] = 0 */
  const int32_t* chunks;  /* device int32 [n_entries]: chunk ids, ascending within a namespace,
                             each live chunk listed once */
  int32_t n_ns;
  int64_t n_entries;      /* = offsets[n_ns] */
} mem_chunk_tables;

/* Workspace for mem_retrieve_topk_grouped (0 on invalid sizes). */
MEMATTN_API size_t mem_workspace_bytes_grouped(int64_t m, int32_t n_ns, int64_t n_entries, int32_t d, int32_t k);

/*
 * Grouped retrieval over the per-namespace chunk tables T[u][s] (Section
 * 4.1; Algorithm 1 selects from the request's own table): query i scores
 * only the bank rows listed in namespace query_ns[i]'s table,
 *   J_i = { tables->chunks[e] : offsets[u] <= e < offsets[u + 1] }, u = query_ns[i],
 * with the same scores, lse, probabilities, top-k and padding as
 * mem_retrieve_topk_scoped given row_ns[j] = u for the rows listed in u and
 * -1 for the rest (deleted chunks are simply not listed).  A query whose
 * namespace is negative or >= n_ns has no candidates.  Each table must list
 * distinct bank rows in ascending order (time order); entries outside
 * [0, bank->n) are ignored, and offsets are clamped to [0, n_entries].  Work is proportional to the queries times the
 * size of their own table, not to the bank.  Needs bf16 rows with d a
 * multiple of 32 and at least 96, k <= 32, strides multiples of 8 (at most
 * 65536), 16-byte aligned bank and queries and a bank of at most 4 GiB;
 * other shapes return MEM_ERR_UNSUPPORTED (mem_retrieve_topk_scoped serves
 * them).  The workspace must be at least mem_workspace_bytes_grouped(m,
 * n_ns, n_entries, d, k).
 */
MEMATTN_API mem_status mem_retrieve_topk_grouped(const mem_bank* bank, const mem_chunk_tables* tables,
                                     const void* queries, const int32_t* query_ns, int64_t m, int64_t q_stride,
                                     int32_t k, float scale, mem_topk_out out, void* workspace, size_t ws_bytes,
                                     void* stream);

/*
 * Chunk materialisation (FetchByID then SortByTime of Algorithm 1, through
 * the directory of Section 4.2).  For output slot i in [0, count) and page p:
 *   out[(i*ppc + p)*page_bytes ...] = pool[table[id'_i * ppc + p]*page_bytes ...]
 * where id' = ids for MEM_ORDER_RANK, or ids sorted ascending within each
 * consecutive group of `group` entries for MEM_ORDER_TIME (1 <= group <= 1024;
 * a trailing partial group is sorted on its own).  An id of -1 yields a zero
 * block, and so does any id outside [0, n_chunks) or a table entry outside
 * [0, n_pages) (the kernel never reads out of bounds).  `out` is device
 * memory of count * ppc * page_bytes bytes and must not overlap the pool.
 */
MEMATTN_API mem_status mem_gather_chunks(const mem_pages* pages, const int32_t* ids, int64_t count, int32_t order, int32_t group,
                             void* out, void* stream);

/*
 * Budget-aware materialisation of the prompt prefix (Section 4.3: the
 * selected chunks are fetched, put back in chronological order and
 * prepended within the request's memory_budget_tokens; Algorithm 1's
 * FetchByID, SortByTime and Concat).  Chunk c holds tok_len[c] token rows
 * of row_bytes bytes (device int32 [n_chunks]); with tpp = page_bytes /
 * row_bytes rows per page, token t of chunk c is row t % tpp of page
 * table[c, t / tpp].  For key i with ids[i, 0..k) in rank order (device
 * int32 [m, k], as written by mem_retrieve_topk; -1 = none):
 *   1. chunks are admitted in rank order while the running token total
 *      stays <= budget_tokens; the first chunk that does not fit, or the
 *      first id that is -1 or outside [0, n_chunks), ends admission;
 *   2. the admitted chunks are ordered by ascending id (time order);
 *   3. out[i] (device, [m, budget_tokens, row_bytes] bytes) receives their
 *      token rows back to back, then zero rows; out_tokens[i] (device int32
 *      [m]) = rows written; out_ids (device int32 [m, k], nullable) = the
 *      admitted ids in time order, then -1.
 * Token counts are clamped to [0, ppc * tpp]; table entries outside
 * [0, n_pages) give zero rows.  row_bytes is a positive multiple of 16 that
 * divides page_bytes; 1 <= k <= 64; budget_tokens >= 0.  `out` must be
 * 16-byte aligned and must not overlap the pool.
 */
MEMATTN_API mem_status mem_gather_budget(const mem_pages* pages, const int32_t* tok_len, int32_t row_bytes,
                             const int32_t* ids, int64_t m, int32_t k, int32_t budget_tokens, void* out,
                             int32_t* out_tokens, int32_t* out_ids, void* stream);


typedef struct {
  int64_t moved_pages;     /* live pages rewritten into fresh blocks */
  int64_t released_blocks; /* blocks compacted (their pages are free once the copies complete) */
  int64_t next_free_page;  /* the allocator frontier after the fresh blocks */
} mem_compact_result;

/* Workspace for mem_compact_blocks with these sizes (0 on invalid sizes). */
MEMATTN_API size_t mem_compact_workspace_bytes(int64_t next_free_page, int32_t pages_per_block, int64_t n_entries,
                                   int32_t pages_per_chunk, int32_t n_ns);

/*
 * Background block compaction (Section 4.2, Eq. 2, and the background stage
 * of Algorithm 2).  The pool's pages form blocks of pages_per_block
 * consecutive pages; pages below next_free_page (the append allocator's
 * frontier) have been written.  A written page that no live chunk's
 * directory entry (`table`, device int32 [n_chunks, pages_per_chunk],
 * updated in place) points to holds an invalid copy:
 *     phi(B) = (written pages of B - live pages of B) / pages_per_block.
 * Every block wholly below the frontier with phi >= theta is compacted
 * (Eq. 2 uses 0.75; Section 5.5 names 0.3 as the default: theta is the
 * caller's).  For each namespace u in order, the pages of u's live chunks
 * that lie in compacted blocks, in (chunk id, page) order, are copied to
 * consecutive fresh pages starting at a block boundary (so no fresh block
 * mixes namespaces; fresh pages begin at the first block boundary at or
 * after the frontier), and their directory entries are pointed there.  phi
 * (device float [n_blocks], nullable) and released (device uint8 [n_blocks],
 * 1 = compacted, nullable) are written for the n_blocks = ceil(next_free /
 * pages_per_block) blocks.  *result (HOST) receives the counts and the new
 * frontier.  The call synchronises `stream` once, after planning, to learn
 * how many fresh pages are needed; if they would pass n_pages it returns
 * MEM_ERR_INVALID_ARG with pool and table unchanged (phi and released are
 * still written).  The copies are then enqueued on `stream`.  The plan
 * also checks the chunk tables on the device (offsets from 0 to n_entries,
 * never falling; chunk ids inside [0, n_chunks) and strictly ascending
 * within a namespace) and returns MEM_ERR_INVALID_ARG, moving nothing, if
 * they are malformed.  Directory entries outside [0, next_free) are
 * ignored.  Requires an injective directory over live pages.
 */
MEMATTN_API mem_status mem_compact_blocks(void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table,
                              int64_t n_chunks, int32_t pages_per_chunk, const mem_chunk_tables* tables,
                              int32_t pages_per_block, float theta, int64_t next_free_page, float* phi,
                              uint8_t* released, mem_compact_result* result, void* workspace, size_t ws_bytes,
                              void* stream);

typedef struct {
  int64_t moved_chunks;   /* chunks rewritten into fresh pages */
  int64_t groups;         /* keys that moved at least one chunk */
  int64_t next_free_page; /* the allocator frontier after the fresh pages */
} mem_colocate_result;

/* Workspace for mem_colocate with these sizes (0 on invalid sizes). */
MEMATTN_API size_t mem_colocate_workspace_bytes(int64_t m, int32_t k, int64_t n_chunks);

/*
 * Association-aware relocation (Section 4.2; the online stage of Algorithm
 * 2: LLMCoLocate, PackIntoNewBlocks(SortByTime(G)), MarkInvalid, UpdateDir),
 * with the model's co-location choice replaced by the dense relation score.
 * For key i with selection ids[i, 0..k) and scores scores[i, 0..k) (device
 * int32 / float [m, k], e.g. the output of mem_build_relations or
 * mem_retrieve_topk; -1 = no chunk):
 *     G_i = { ids[i, r] : scores[i, r] >= tau }   (tau_assoc, 0.7 by default
 *                                                   in Section 5.5)
 * and G_i is relocated when it has at least min_group entries (ids outside
 * [0, n_chunks) are ignored, a repeated id counts for the size but moves
 * once).  A chunk in several qualifying groups goes with the lowest key
 * index (as if keys were served in order).  Key by key, each group's
 * chunks in ascending id order (time order) get consecutive fresh pages
 * from next_free_page on, pages_per_chunk each; the pages are copied there
 * and the directory entries (`table`, device int32 [n_chunks,
 * pages_per_chunk], updated in place) point to them, which leaves the old
 * copies invalid for mem_compact_blocks to reclaim (a relocated chunk's
 * entry outside [0, n_pages) is not read: its fresh page is written as
 * zeros).  *result (HOST) gets the counts and the new frontier.  The call
 * synchronises `stream` once, after
 * planning; if the fresh pages would pass n_pages it returns
 * MEM_ERR_INVALID_ARG with pool and table unchanged.  1 <= k <= 64,
 * min_group >= 1, tau finite.
 */
MEMATTN_API mem_status mem_colocate(void* pool, int64_t n_pages, int64_t page_bytes, int32_t* table, int64_t n_chunks,
                        int32_t pages_per_chunk, const int32_t* ids, const float* scores, int64_t m, int32_t k,
                        float tau, int32_t min_group, int64_t next_free_page, mem_colocate_result* result,
                        void* workspace, size_t ws_bytes, void* stream);

/*
 * Insert (Algorithm 1) with append-only placement (Section 4.2).  Copies the
 * m rows of `new_emb` ([m, new_stride] elements, the bank's dtype) into bank
 * rows [n, n + m) (bank->emb must be writable device memory of
 * capacity_rows rows), and writes table rows [n, n + m) (device int32
 * [capacity_rows, pages_per_chunk]) with the pages *next_free_page + r*ppc + p.
 * On success the HOST-side counters advance synchronously: bank->n += m and
 * *next_free_page += m * pages_per_chunk; the device copies are enqueued on
 * `stream`.  Fails without side effects if the bank or the page pool
 * (n_pages_cap pages) would overflow.
 */
MEMATTN_API mem_status mem_append_chunks(mem_bank* bank, int64_t capacity_rows, const void* new_emb, int64_t m,
                             int64_t new_stride, int32_t* table, int32_t pages_per_chunk,
                             int64_t* next_free_page /* HOST */, int64_t n_pages_cap, void* stream);

/* Static description of a status code. */
MEMATTN_API const char* mem_status_string(mem_status s);

/* Message describing the last failed call on this thread ("" if none). */
MEMATTN_API const char* mem_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MEMATTN_H */
