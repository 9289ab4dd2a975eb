/*
 * fp64 CPU oracle for dense MemAttention retrieval and chunk materialisation.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the GPU library; both consume the same input
 * bytes produced by the seeded generators.
 *
 * What it computes (the paper gives the steps, not formulas; the readings
 * are listed with each function):
 *
 *   Relevance selection.  Algorithm 1 selects, for a key (a new chunk during
 *   cross-chunk reconciliation, or the current query during retrieval), the
 *   top-p related chunks of the namespace's chunk table (Section 4.1, p = 5
 *   by default).  The paper's "Dense-only" ablation (Section 5.5) replaces
 *   the model-driven matcher by embedding similarity; that is the relevance
 *   function computed here:
 *       s_ij   = sum_t q_it * b_jt                   (dot product of stored unit vectors)
 *       J_i    = {0..n-1} minus {self_i} when a self index is given
 *       lse_i  = M_i + ln sum_{j in J_i} exp(scale*s_ij - M_i),  M_i = max_j scale*s_ij
 *       p_ij   = exp(scale*s_ij - lse_i)
 *       top-k  = first k of J_i sorted by (s_ij descending, j ascending)
 *   Selection uses s, never p.  oracle_retrieve_scoped restricts J_i to the
 *   live rows of the key's namespace (Section 4.1's T[u][s]; tombstones of
 *   Section 4.2's out-of-place updates).
 *
 *   Materialisation.  FetchByID then SortByTime (Algorithm 1) read the
 *   selected chunks through the block directory that separates a chunk's
 *   logical identity from its physical placement (Section 4.2):
 *       out[i, page p] = pool[table[id'_i, p]]
 *   where id' is ids reordered ascending within each group when time order is
 *   requested (chunk ids are assigned in append order), and id -1 yields a
 *   zero block.  oracle_gather_budget admits chunks in rank order within a
 *   token budget, restores time order and packs their token rows (the
 *   prompt prefix of Section 4.3).
 *
 *   Compaction.  oracle_compact computes the invalid ratio of Eq. 2 per
 *   block and repacks the live pages of blocks at or above the threshold,
 *   per namespace and in time order, into fresh blocks (Algorithm 2's
 *   background stage).
 *
 *   Relocation.  oracle_colocate rewrites each key's strongly related
 *   retrieved chunks (relation score >= tau_assoc) in time order into fresh
 *   pages and updates the directory (Algorithm 2's online stage).
 *
 *   Insertion.  Insert (Algorithm 1) appends a chunk record; out-of-place,
 *   append-only writes (Section 4.2) give chunk n+r the physical pages
 *   next_free + r*ppc + p.
 *
 * Every element is decoded exactly to fp64 (bf16 = upper 16 bits of an
 * fp32); dot products are summed sequentially in fp64.  Plain loops, no BLAS.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#define NTHREADS(t) ((t) > 0 ? (t) : omp_get_max_threads())
#else
#define NTHREADS(t) 1
#endif

enum { OR_F32 = 0, OR_BF16 = 1 };
enum { OR_ORDER_RANK = 0, OR_ORDER_TIME = 1 };

static double decode(const void* base, int32_t dtype, int64_t i) {
  if (dtype == OR_F32) return (double)((const float*)base)[i];
  uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* s_ij = sum_t q_it b_jt, sequential fp64 sum. */
static double dot(const void* q, int64_t qrow, const void* b, int64_t brow, int32_t d, int32_t dtype) {
  double acc = 0.0;
  for (int32_t t = 0; t < d; ++t) acc += decode(q, dtype, qrow + t) * decode(b, dtype, brow + t);
  return acc;
}

void oracle_scores(const void* q, int64_t q_stride, const void* b, int64_t b_stride, int64_t m, int64_t n,
                   int32_t d, int32_t dtype, double* out, int32_t threads) {
#pragma omp parallel for schedule(dynamic) num_threads(NTHREADS(threads))
  for (int64_t i = 0; i < m; ++i)
    for (int64_t j = 0; j < n; ++j) out[i * n + j] = dot(q, i * q_stride, b, j * b_stride, d, dtype);
}

typedef struct {
  double s;
  int64_t j;
} cand;

/* (score descending, index ascending): a total order on candidates. */
static int by_score_then_index(const void* pa, const void* pb) {
  const cand* a = (const cand*)pa;
  const cand* b = (const cand*)pb;
  if (a->s > b->s) return -1;
  if (a->s < b->s) return 1;
  return (a->j < b->j) ? -1 : (a->j > b->j);
}

/* lse = M + ln sum_t exp(scale*s_t - M), M = max_t scale*s_t, over nc > 0 candidates. */
static double softmax_lse(const cand* c, int64_t nc, double scale) {
  double mx = -INFINITY;
  for (int64_t t = 0; t < nc; ++t) mx = fmax(mx, scale * c[t].s);
  double sum = 0.0;
  for (int64_t t = 0; t < nc; ++t) sum += exp(scale * c[t].s - mx);
  return mx + log(sum);
}

/*
 * Dense relevance selection for m keys against an n-row bank.
 * self_idx (nullable): per key, a bank row excluded from its candidates
 * (relation building over the bank itself), or -1.
 * Outputs: idx/score/prob [m, k]; lse [m]; full_prob (nullable) [m, n] with 0
 * for an excluded row.  Returns 0, or -1 if some key has fewer than k candidates.
 */
int oracle_retrieve(const void* q, int64_t q_stride, const void* b, int64_t b_stride, int64_t m, int64_t n,
                    int32_t d, int32_t dtype, int32_t k, double scale, const int64_t* self_idx,
                    int32_t* idx_out, double* score_out, double* prob_out, double* lse_out, double* full_prob,
                    int32_t threads) {
  int bad = 0;
#pragma omp parallel for schedule(dynamic) num_threads(NTHREADS(threads)) reduction(| : bad)
  for (int64_t i = 0; i < m; ++i) {
    const int64_t self = self_idx ? self_idx[i] : -1;
    cand* c = (cand*)malloc((size_t)n * sizeof(cand));
    int64_t nc = 0;
    for (int64_t j = 0; j < n; ++j) {
      if (j == self) continue;
      c[nc].s = dot(q, i * q_stride, b, j * b_stride, d, dtype);
      c[nc].j = j;
      ++nc;
    }
    if (nc < k || nc == 0) {
      bad |= 1;
      free(c);
      continue;
    }
    /* softmax normaliser over all candidates */
    const double lse = softmax_lse(c, nc, scale);
    if (lse_out) lse_out[i] = lse;
    if (full_prob) {
      for (int64_t j = 0; j < n; ++j) full_prob[i * n + j] = 0.0;
      for (int64_t t = 0; t < nc; ++t) full_prob[i * n + c[t].j] = exp(scale * c[t].s - lse);
    }
    /* top-k: sort all candidates by (s desc, j asc), keep the first k */
    qsort(c, (size_t)nc, sizeof(cand), by_score_then_index);
    for (int32_t r = 0; r < k; ++r) {
      if (idx_out) idx_out[i * k + r] = (int32_t)c[r].j;
      if (score_out) score_out[i * k + r] = c[r].s;
      if (prob_out) prob_out[i * k + r] = exp(scale * c[r].s - lse);
    }
    free(c);
  }
  return bad ? -1 : 0;
}

/*
 * Namespace-scoped, tombstone-aware selection.  Algorithm 1 draws the
 * candidates of a key from T[u][s], the chunk table of the key's own
 * (user, session) namespace (Section 4.1), and out-of-place updates leave
 * invalidated copies behind as tombstones (Section 4.2).  Here every bank row
 * carries a namespace id and a live flag, and every key a namespace id:
 *     J_i = {j : row_live[j] != 0 and row_ns[j] == key_ns[i]} minus {self_i}
 * Softmax and top-k are then computed over J_i exactly as in
 * oracle_retrieve.  When |J_i| < k the remaining output slots hold id -1,
 * score -inf and p 0; with J_i empty, lse is -inf.
 */
int oracle_retrieve_scoped(const void* q, int64_t q_stride, const void* b, int64_t b_stride, int64_t m, int64_t n,
                           int32_t d, int32_t dtype, int32_t k, double scale, const int64_t* self_idx,
                           const int32_t* row_ns, const uint8_t* row_live, const int32_t* key_ns,
                           int32_t* idx_out, double* score_out, double* prob_out, double* lse_out,
                           double* full_prob, int32_t threads) {
#pragma omp parallel for schedule(dynamic) num_threads(NTHREADS(threads))
  for (int64_t i = 0; i < m; ++i) {
    const int64_t self = self_idx ? self_idx[i] : -1;
    cand* c = (cand*)malloc((size_t)(n > 0 ? n : 1) * sizeof(cand));
    int64_t nc = 0;
    for (int64_t j = 0; j < n; ++j) {
      if (j == self || !row_live[j] || row_ns[j] != key_ns[i]) continue;
      c[nc].s = dot(q, i * q_stride, b, j * b_stride, d, dtype);
      c[nc].j = j;
      ++nc;
    }
    const double lse = nc > 0 ? softmax_lse(c, nc, scale) : -INFINITY;
    if (lse_out) lse_out[i] = lse;
    if (full_prob) {
      for (int64_t j = 0; j < n; ++j) full_prob[i * n + j] = 0.0;
      for (int64_t t = 0; t < nc; ++t) full_prob[i * n + c[t].j] = exp(scale * c[t].s - lse);
    }
    qsort(c, (size_t)nc, sizeof(cand), by_score_then_index);
    for (int32_t r = 0; r < k; ++r) {
      const int have = r < nc;
      if (idx_out) idx_out[i * k + r] = have ? (int32_t)c[r].j : -1;
      if (score_out) score_out[i * k + r] = have ? c[r].s : -INFINITY;
      if (prob_out) prob_out[i * k + r] = have ? exp(scale * c[r].s - lse) : 0.0;
    }
    free(c);
  }
  return 0;
}

/* SortByTime: ascending chunk id (= append order) within each group of `group`. */
void oracle_time_order(const int32_t* ids, int64_t count, int32_t group, int32_t* out) {
  memcpy(out, ids, (size_t)count * sizeof(int32_t));
  for (int64_t g0 = 0; g0 < count; g0 += group) {
    int64_t g1 = g0 + group < count ? g0 + group : count;
    for (int64_t a = g0 + 1; a < g1; ++a) { /* insertion sort: stable, obviously correct */
      int32_t v = out[a];
      int64_t p = a;
      while (p > g0 && out[p - 1] > v) {
        out[p] = out[p - 1];
        --p;
      }
      out[p] = v;
    }
  }
}

/* FetchByID through the directory: out[i, p] = pool[table[id'_i, p]], id -1 -> zeros. */
int oracle_gather(const uint8_t* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table, int64_t n_chunks,
                  int32_t ppc, const int32_t* ids, int64_t count, int32_t order, int32_t group, uint8_t* out) {
  int32_t* ord = (int32_t*)malloc((size_t)(count > 0 ? count : 1) * sizeof(int32_t));
  if (order == OR_ORDER_TIME)
    oracle_time_order(ids, count, group, ord);
  else
    memcpy(ord, ids, (size_t)count * sizeof(int32_t));
  int bad = 0;
  for (int64_t i = 0; i < count; ++i) {
    for (int32_t p = 0; p < ppc; ++p) {
      uint8_t* dst = out + (i * ppc + p) * page_bytes;
      int32_t c = ord[i];
      if (c == -1) {
        memset(dst, 0, (size_t)page_bytes);
        continue;
      }
      if (c < 0 || c >= n_chunks) {
        bad = 1;
        memset(dst, 0, (size_t)page_bytes);
        continue;
      }
      int64_t page = table[(int64_t)c * ppc + p];
      if (page < 0 || page >= n_pages) {
        bad = 1;
        memset(dst, 0, (size_t)page_bytes);
        continue;
      }
      memcpy(dst, pool + page * page_bytes, (size_t)page_bytes);
    }
  }
  free(ord);
  return bad ? -1 : 0;
}

/*
 * Budget-aware materialisation.  After selection the system fetches the
 * chosen chunks, restores their chronological order and prepends them to
 * the prompt within the request's memory token budget (Section 4.3,
 * memory_budget_tokens; B_mem of Section 5.5).  Chunk c holds tok_len[c]
 * token rows of row_bytes bytes; with tpp = page_bytes / row_bytes rows per
 * page, token t of chunk c sits in page table[c, t / tpp] at byte
 * (t % tpp) * row_bytes.  For key i, with ids[i, 0..k) in rank order
 * (-1 = no chunk):
 *   1. admit chunks in rank order while the running token total stays
 *      within `budget`; the first chunk that does not fit, or the first -1,
 *      ends admission, so the kept chunks are a prefix of the rank order;
 *   2. SortByTime: order the kept chunks by ascending id;
 *   3. out[i] = their token rows back to back ([budget, row_bytes] bytes),
 *      zero rows after them; out_tokens[i] = rows written; out_ids[i] = the
 *      kept ids in time order, then -1.
 * Returns -1 (and writes nothing for that key) on an id, length or page out
 * of range.
 */
int oracle_gather_budget(const uint8_t* pool, int64_t n_pages, int64_t page_bytes, const int32_t* table,
                         int64_t n_chunks, int32_t ppc, const int32_t* tok_len, int32_t row_bytes,
                         const int32_t* ids, int64_t m, int32_t k, int32_t budget, uint8_t* out,
                         int32_t* out_tokens, int32_t* out_ids) {
  const int64_t tpp = page_bytes / row_bytes;
  const int64_t cap = tpp * ppc;
  int bad = 0;
  int32_t* ranked = (int32_t*)malloc((size_t)(k > 0 ? k : 1) * sizeof(int32_t));
  int32_t* kept = (int32_t*)malloc((size_t)(k > 0 ? k : 1) * sizeof(int32_t));
  for (int64_t i = 0; i < m; ++i) {
    /* 1. admission in rank order */
    int32_t nk = 0;
    int64_t total = 0;
    int ok = 1;
    for (int32_t r = 0; r < k; ++r) {
      const int32_t c = ids[i * k + r];
      if (c == -1) break;
      if (c < 0 || c >= n_chunks || tok_len[c] < 0 || tok_len[c] > cap) {
        ok = 0;
        break;
      }
      if (total + tok_len[c] > budget) break;
      total += tok_len[c];
      ranked[nk++] = c;
    }
    if (!ok) {
      bad = 1;
      continue;
    }
    /* 2. SortByTime */
    oracle_time_order(ranked, nk, nk > 0 ? nk : 1, kept);
    /* 3. concatenate token rows, then zeros */
    uint8_t* dst = out + i * (int64_t)budget * row_bytes;
    int64_t row = 0;
    for (int32_t a = 0; a < nk && ok; ++a) {
      const int32_t c = kept[a];
      for (int32_t t = 0; t < tok_len[c]; ++t, ++row) {
        const int64_t page = table[(int64_t)c * ppc + t / tpp];
        if (page < 0 || page >= n_pages) {
          ok = 0;
          break;
        }
        memcpy(dst + row * row_bytes, pool + page * page_bytes + (t % tpp) * row_bytes, (size_t)row_bytes);
      }
    }
    if (!ok) {
      bad = 1;
      continue;
    }
    memset(dst + row * row_bytes, 0, (size_t)((budget - row) * row_bytes));
    out_tokens[i] = (int32_t)row;
    for (int32_t a = 0; a < k; ++a) out_ids[i * k + a] = a < nk ? kept[a] : -1;
  }
  free(ranked);
  free(kept);
  return bad ? -1 : 0;
}

/*
 * SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): output number `i`
 * (0-based) of the stream seeded with `key` is mix(key + (i+1) * golden).
 * The oracle's own implementation of the generator that defines page
 * contents, used to know what a page holds without reading the pool.
 */
static uint64_t splitmix64_at(uint64_t key, uint64_t i) {
  uint64_t z = key + (i + 1u) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Words of logical page `page` of chunk `chunk`. */
void oracle_payload_page(uint64_t key, int64_t chunk, int32_t page, int32_t ppc, int64_t page_bytes,
                         uint64_t* out) {
  const int64_t wpp = page_bytes / 8;
  const uint64_t base = (uint64_t)((chunk * ppc + page) * wpp);
  for (int64_t w = 0; w < wpp; ++w) out[w] = splitmix64_at(key, base + (uint64_t)w);
}

/*
 * Expected gathered blocks when the pool holds payload(c, p) at page
 * table[c, p]: slot i receives the payload of chunk id'_i (zeros for -1).
 * `slots` selects which output slots to produce (nullable = all `count`).
 */
void oracle_expected_blocks(uint64_t key, const int32_t* ids, int64_t count, int32_t order, int32_t group,
                            int32_t ppc, int64_t page_bytes, const int64_t* slots, int64_t n_slots,
                            uint64_t* out, int32_t threads) {
  int32_t* ord = (int32_t*)malloc((size_t)(count > 0 ? count : 1) * sizeof(int32_t));
  if (order == OR_ORDER_TIME)
    oracle_time_order(ids, count, group, ord);
  else
    memcpy(ord, ids, (size_t)count * sizeof(int32_t));
  const int64_t ns = slots ? n_slots : count;
  const int64_t wpp = page_bytes / 8;
#pragma omp parallel for schedule(static) num_threads(NTHREADS(threads))
  for (int64_t s = 0; s < ns; ++s) {
    const int64_t i = slots ? slots[s] : s;
    for (int32_t p = 0; p < ppc; ++p) {
      uint64_t* dst = out + (s * ppc + p) * wpp;
      if (ord[i] == -1)
        memset(dst, 0, (size_t)page_bytes);
      else
        oracle_payload_page(key, ord[i], p, ppc, page_bytes, dst);
    }
  }
  free(ord);
}

/* Insert: table rows of the m appended chunks (bump allocation in id order). */
void oracle_append_table(int64_t m, int32_t ppc, int64_t next_free, int32_t* rows_out) {
  for (int64_t r = 0; r < m; ++r)
    for (int32_t p = 0; p < ppc; ++p) rows_out[r * ppc + p] = (int32_t)(next_free + r * ppc + p);
}

/*
 * Background block compaction (Section 4.2, Eq. 2; the background stage of
 * Algorithm 2).  The pool's pages form blocks of P consecutive pages, and
 * pages below the allocator frontier `next_free` have been written.  The live
 * chunks are the ones listed in the per-namespace chunk tables T[u][s]
 * (CSR: chunks[offsets[u] .. offsets[u+1]) are namespace u's live chunk ids,
 * ascending); a written page that no live chunk's directory entry points to
 * holds an invalid copy, so
 *     phi(B) = N_invalid(B) / N_total(B) = (written(B) - live(B)) / P.
 * Every block wholly below the frontier with phi >= theta is compacted:
 * LiveChunks, PartitionByUserSession and, per partition, PackIntoNewBlocks
 * of the pages in time order.  For each namespace u in ascending order, the
 * pages of u's live chunks that lie in compacted blocks, in (chunk id, page)
 * order, go to consecutive fresh pages; each namespace starts a fresh block,
 * so no new block mixes namespaces.  Fresh pages start at the first block
 * boundary at or after the frontier.  UpdateDir points the moved directory
 * entries at their new pages, Release frees the compacted blocks, and the
 * frontier moves past the last fresh block used (it stays put when nothing
 * moves).  (Grouping by model-inferred affinity inside a partition needs the
 * model; every partition is one group here.)
 * Returns -1, changing nothing, when the fresh blocks would not fit in the
 * pool's n_pages or a namespace's chunk ids are not ascending.
 */
/* PackIntoNewBlocks for every namespace in turn: returns the position after
 * the last fresh block used; with apply != 0 also copies the pages and
 * updates the directory. */
static int64_t pack_namespaces(uint8_t* pool, int64_t page_bytes, int32_t* table, int32_t ppc,
                               const int32_t* offsets, const int32_t* chunks, int32_t n_ns, int32_t P,
                               int64_t next_free, const uint8_t* cand, int64_t first_new, int apply,
                               int64_t* moved) {
  int64_t pos = first_new;
  *moved = 0;
  for (int32_t u = 0; u < n_ns; ++u) {
    const int64_t start = pos;
    for (int32_t e = offsets[u]; e < offsets[u + 1]; ++e) {
      for (int32_t pp = 0; pp < ppc; ++pp) {
        int32_t* entry = &table[(int64_t)chunks[e] * ppc + pp];
        const int64_t pg = *entry;
        if (pg < 0 || pg >= next_free || !cand[pg / P]) continue;
        if (apply) {
          memcpy(pool + pos * page_bytes, pool + pg * page_bytes, (size_t)page_bytes);
          *entry = (int32_t)pos;
        }
        ++pos;
        ++*moved;
      }
    }
    if (pos > start) pos = start + ((pos - start + P - 1) / P) * P;
  }
  return pos;
}

int oracle_compact(uint8_t* pool, int64_t n_pages, int64_t page_bytes, int32_t* table, int64_t n_chunks, int32_t ppc,
                   const int32_t* offsets, const int32_t* chunks, int32_t n_ns, int32_t P, double theta,
                   int64_t next_free, double* phi_out, uint8_t* released_out, int64_t* new_next_free_out,
                   int64_t* n_moved_out) {
  const int64_t n_blocks = (next_free + P - 1) / P;
  int64_t* live = (int64_t*)calloc((size_t)(n_blocks > 0 ? n_blocks : 1), sizeof(int64_t));
  uint8_t* cand = (uint8_t*)calloc((size_t)(n_blocks > 0 ? n_blocks : 1), 1);
  /* live pages per block */
  for (int32_t u = 0; u < n_ns; ++u) {
    for (int32_t e = offsets[u]; e < offsets[u + 1]; ++e) {
      const int32_t c = chunks[e];
      if (c < 0 || c >= n_chunks || (e > offsets[u] && chunks[e - 1] >= c)) {
        free(live);
        free(cand);
        return -1;
      }
      for (int32_t p = 0; p < ppc; ++p) {
        const int64_t pg = table[(int64_t)c * ppc + p];
        if (pg >= 0 && pg < next_free) live[pg / P] += 1;
      }
    }
  }
  /* invalid ratio and candidates */
  for (int64_t b = 0; b < n_blocks; ++b) {
    const int64_t written = (next_free - b * P) < P ? (next_free - b * P) : P;
    const double phi = (double)(written - live[b]) / (double)P;
    if (phi_out) phi_out[b] = phi;
    cand[b] = ((b + 1) * P <= next_free) && phi >= theta;
  }
  /* plan (fresh pages per namespace, in time order), check space, apply */
  const int64_t first_new = n_blocks * P;
  int64_t moved = 0;
  const int64_t end = pack_namespaces(pool, page_bytes, table, ppc, offsets, chunks, n_ns, P, next_free, cand,
                                      first_new, 0, &moved);
  if (end > n_pages) {
    free(live);
    free(cand);
    return -1;
  }
  pack_namespaces(pool, page_bytes, table, ppc, offsets, chunks, n_ns, P, next_free, cand, first_new, 1, &moved);
  for (int64_t b = 0; b < n_blocks; ++b)
    if (released_out) released_out[b] = cand[b];
  *new_next_free_out = moved > 0 ? end : next_free;
  *n_moved_out = moved;
  free(live);
  free(cand);
  return 0;
}

/*
 * Association-aware relocation (Section 4.2; the online stage of
 * Algorithm 2: LLMCoLocate, PackIntoNewBlocks(SortByTime(G)), MarkInvalid,
 * UpdateDir), with the model's co-location choice replaced by the dense
 * relation score: for key i, whose selection is ids[i, 0..k) with scores
 * scores[i, 0..k) (-1 = no chunk),
 *     G_i = { ids[i, r] : scores[i, r] >= tau }      (tau_assoc, Section 5.5)
 * and the group is relocated only if |G_i| >= min_group.  Keys are taken in
 * order; a chunk already relocated by an earlier key of the same call stays
 * where that key put it (and an id repeated within a key counts once).  Key i's remaining chunks, in ascending id order
 * (SortByTime), get consecutive fresh pages at the frontier, ppc pages per
 * chunk in page order; their pages are copied there and their directory
 * entries updated, which leaves the old copies invalid (no entry points at
 * them); an entry outside [0, n_pages) is not read and its fresh page holds
 * zeros.  The frontier advances by the pages written.
 * Returns -1, changing nothing, if an id is outside [0, n_chunks) or the
 * fresh pages would pass n_pages.
 */
int oracle_colocate(uint8_t* pool, int64_t n_pages, int64_t page_bytes, int32_t* table, int64_t n_chunks,
                    int32_t ppc, const int32_t* ids, const float* scores, int64_t m, int32_t k, float tau,
                    int32_t min_group, int64_t next_free, int64_t* new_next_free_out, int64_t* moved_out,
                    int64_t* groups_out) {
  uint8_t* done = (uint8_t*)calloc((size_t)(n_chunks > 0 ? n_chunks : 1), 1);
  int32_t* grp = (int32_t*)malloc((size_t)(k > 0 ? k : 1) * sizeof(int32_t));
  int32_t* ord = (int32_t*)malloc((size_t)(k > 0 ? k : 1) * sizeof(int32_t));
  int64_t pos = next_free, moved = 0, groups = 0;
  for (int pass = 0; pass < 2; ++pass) { /* pass 0 checks, pass 1 applies */
    memset(done, 0, (size_t)(n_chunks > 0 ? n_chunks : 1));
    pos = next_free;
    moved = groups = 0;
    for (int64_t i = 0; i < m; ++i) {
      int32_t g = 0;
      for (int32_t r = 0; r < k; ++r) {
        const int32_t c = ids[i * k + r];
        if (c == -1) continue;
        if (c < 0 || c >= n_chunks) {
          free(done), free(grp), free(ord);
          return -1;
        }
        if ((double)scores[i * k + r] >= (double)tau) grp[g++] = c;
      }
      if (g < min_group) continue;
      /* drop chunks relocated by an earlier key (and repeats of an id) */
      int32_t nk = 0;
      for (int32_t a = 0; a < g; ++a)
        if (!done[grp[a]]) {
          done[grp[a]] = 1;
          grp[nk++] = grp[a];
        }
      if (nk == 0) continue;
      oracle_time_order(grp, nk, nk, ord);
      ++groups;
      for (int32_t a = 0; a < nk; ++a) {
        const int32_t c = ord[a];
        ++moved;
        for (int32_t p = 0; p < ppc; ++p, ++pos) {
          if (!pass) continue;
          int32_t* entry = &table[(int64_t)c * ppc + p];
          if (*entry >= 0 && *entry < n_pages)
            memcpy(pool + pos * page_bytes, pool + (int64_t)(*entry) * page_bytes, (size_t)page_bytes);
          else /* an entry outside the pool is not read: the fresh page holds zeros */
            memset(pool + pos * page_bytes, 0, (size_t)page_bytes);
          *entry = (int32_t)pos; /* UpdateDir; the old copy is now invalid */
        }
      }
    }
    if (!pass && pos > n_pages) {
      free(done), free(grp), free(ord);
      return -1;
    }
  }
  *new_next_free_out = pos;
  *moved_out = moved;
  *groups_out = groups;
  free(done), free(grp), free(ord);
  return 0;
}
