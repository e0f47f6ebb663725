/*
 * Oracle for the draft-stage hot path of FastCoder (arXiv 2502.17139).
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, deliberately slow CPU
 * implementation of what the method computes, written from the paper's
 * definitions.  Only the test suite, the smoke check and the benchmark's CPU
 * baseline call it; the GPU library never does, and the two share no code,
 * header, table or helper.
 *
 * Every function follows one passage:
 *   - suffix order and the suffix array: Section III-A (exact suffix match over
 *     a suffix array, after Manber and Myers);
 *   - datastore organisation (every position of a file splits it into a
 *     context and a continuation): Section IV-A, eq. (1)-(2);
 *   - retrieval (longest context suffix, n from n_max down, all matches):
 *     Section III-A; two sources searched side by side: Section IV-C;
 *   - weighted trie (node weight alpha*t_r + beta*t_c): Section IV-D, eq. (3);
 *   - top-weighted draft selection (at most 64 draft tokens): Section IV-D and
 *     Section V-D;
 *   - tree attention mask and position ids: Section IV-D, eq. (4);
 *   - acceptance (all correct tokens from the start, nothing after the first
 *     error): Section IV-D.
 * Points the paper leaves open are fixed by the readings listed with each
 * function (separator handling, source budget, which matches are kept when
 * there are more than k, tie-breaks, emission order, the mask diagonal).
 *
 * Pins: tests/test_oracle_*.py check every function against brute force on
 * tiny inputs, closed forms, trie invariants and hand-worked examples.
 */
#define _GNU_SOURCE
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------- */
/* Suffix order (Section III-A).  Suffix i of T[0..N) is T[i..N).  Suffixes   */
/* compare token by token by numeric id; when one ends first (it is a proper  */
/* prefix of the other) it is the smaller.                                    */
/* ------------------------------------------------------------------------- */
int oracle_suffix_cmp(const uint16_t* T, uint64_t N, uint64_t i, uint64_t j) {
  if (i == j) return 0;
  while (i < N && j < N) {
    if (T[i] != T[j]) return T[i] < T[j] ? -1 : 1;
    ++i;
    ++j;
  }
  return (i == N) ? -1 : 1; /* the one that ran out first is shorter */
}

typedef struct {
  const uint16_t* T;
  uint64_t N;
} text_ref;

static int cmp_sa_entries(const void* a, const void* b, void* ctx) {
  const text_ref* t = (const text_ref*)ctx;
  return oracle_suffix_cmp(t->T, t->N, *(const uint32_t*)a, *(const uint32_t*)b);
}

/* Suffix array: the start positions 0..N-1 sorted by suffix order, by a plain
 * comparison sort with the direct suffix comparison above. */
void oracle_suffix_array(const uint16_t* T, uint64_t N, uint32_t* sa) {
  for (uint64_t i = 0; i < N; ++i) sa[i] = (uint32_t)i;
  text_ref t = {T, N};
  qsort_r(sa, N, sizeof(uint32_t), cmp_sa_entries, &t);
}

/*
 * Linear-time suffix-array check (Burkhardt and Kaerkkaeinen, CPM 2003):
 * `sa` is the suffix array of T iff it is a permutation of 0..N-1 and, for
 * every pair a = sa[r], b = sa[r+1], (T[a], rank[a+1]) < (T[b], rank[b+1]),
 * where rank is the inverse permutation and the empty suffix ranks below all.
 * Returns 0 when valid, 1 when not a permutation, 2 on an order violation;
 * *where receives the offending SA index.  rank_ws holds N uint32.
 */
int oracle_check_sa(const uint16_t* T, uint64_t N, const uint32_t* sa, uint32_t* rank_ws, uint64_t* where) {
  const uint32_t UNSET = 0xFFFFFFFFu;
  for (uint64_t i = 0; i < N; ++i) rank_ws[i] = UNSET;
  for (uint64_t r = 0; r < N; ++r) {
    uint64_t p = sa[r];
    if (p >= N || rank_ws[p] != UNSET) {
      if (where) *where = r;
      return 1;
    }
    rank_ws[p] = (uint32_t)r;
  }
  for (uint64_t r = 0; r + 1 < N; ++r) {
    uint64_t a = sa[r], b = sa[r + 1];
    int ok;
    if (T[a] != T[b]) {
      ok = T[a] < T[b];
    } else {
      int64_t ra = (a + 1 < N) ? (int64_t)rank_ws[a + 1] : -1;
      int64_t rb = (b + 1 < N) ? (int64_t)rank_ws[b + 1] : -1;
      ok = ra < rb;
    }
    if (!ok) {
      if (where) *where = r;
      return 2;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------- */
/* Retrieval (Section III-A, Section IV-A, Section IV-C).                      */
/* ------------------------------------------------------------------------- */

/*
 * Longest usable suffix length of a context row (reading: a context lives
 * inside one file, so the query suffix never reaches back past a separator 0
 * and no match can straddle two files): min(n_max, L, number of trailing
 * non-zero tokens).
 */
static int query_limit(const uint16_t* row, int L, int n_max) {
  int d = 0;
  while (d < L && row[L - 1 - d] != 0) ++d;
  int h = n_max;
  if (L < h) h = L;
  if (d < h) h = d;
  return h;
}

/*
 * Largest l <= n_hi such that the last l tokens of the context occur in T.
 * An occurrence of the length-n suffix q_n at start j ends at e = j + n, and
 * it exists iff T and the context agree on the n tokens before e; one pass
 * over every end position e measures that agreement backwards, capped at
 * n_hi, which answers "does q_n occur" for every n at once.
 */
static int longest_occurring_suffix(const uint16_t* T, uint64_t N, const uint16_t* ctx_end, int n_hi) {
  int best = 0;
  for (uint64_t e = 1; e <= N && best < n_hi; ++e) {
    int l = 0;
    while (l < n_hi && (uint64_t)l < e && T[e - 1 - l] == ctx_end[-1 - l]) ++l;
    if (l > best) best = l;
  }
  return best;
}

/* Compare suffix i with pattern q[0..n): -1 below, 0 starts with q, +1 above. */
static int cmp_suffix_pattern(const uint16_t* T, uint64_t N, uint64_t i, const uint16_t* q, int n) {
  for (int x = 0; x < n; ++x) {
    if (i + x == N) return -1; /* the suffix ends first: shorter is smaller */
    if (T[i + x] != q[x]) return T[i + x] < q[x] ? -1 : 1;
  }
  return 0;
}

typedef struct {
  int32_t match_n;
  uint32_t range_lo, range_cnt;
  uint32_t* occ; /* start positions of q_{match_n}, in suffix order */
} source_match;

/*
 * Suffix match in one store.  For n = n_hi down to n_min the suffix q_n =
 * ctx[L-n..L) is looked up; the first n with at least one occurrence wins
 * (n = 1 is never tried when n_min >= 2).  The occurrences are returned in
 * suffix order; range_lo is the suffix-array index of the smallest of them,
 * i.e. the number of suffixes that compare below q_n; range_lo is 0 when
 * there is no match.
 */
static void match_one_source(const uint16_t* T, uint64_t N, const uint16_t* row, int L, int n_max, int n_min,
                             source_match* out) {
  out->match_n = 0;
  out->range_lo = 0;
  out->range_cnt = 0;
  out->occ = NULL;
  int n_hi = query_limit(row, L, n_max);
  if (n_hi < n_min || N == 0) return;
  int n = longest_occurring_suffix(T, N, row + L, n_hi);
  if (n < n_min) return;
  const uint16_t* q = row + L - n;
  uint64_t cnt = 0, cap = 16;
  uint32_t* occ = (uint32_t*)malloc(cap * sizeof(uint32_t));
  for (uint64_t j = 0; j + n <= N; ++j) {
    if (T[j] == q[0] && memcmp(T + j, q, (size_t)n * sizeof(uint16_t)) == 0) {
      if (cnt == cap) {
        cap *= 2;
        occ = (uint32_t*)realloc(occ, cap * sizeof(uint32_t));
      }
      occ[cnt++] = (uint32_t)j;
    }
  }
  text_ref t = {T, N};
  qsort_r(occ, cnt, sizeof(uint32_t), cmp_sa_entries, &t);
  uint64_t below = 0;
  for (uint64_t i = 0; i < N; ++i)
    if (cmp_suffix_pattern(T, N, i, q, n) < 0) ++below;
  out->match_n = n;
  out->range_lo = (uint32_t)below;
  out->range_cnt = (uint32_t)cnt;
  out->occ = occ;
}

/*
 * Batched retrieval over S stores given in priority order (the repository
 * store first, then the common store; Section IV-A).  Every store is searched
 * and reported (the two searches are independent, Section IV-C).
 *
 * Readings:
 *  - budget: store s may fill k minus the slots taken by stores before it;
 *    taken_s = min(budget_s, cnt_s);
 *  - when cnt_s exceeds the budget b, the kept occurrences are those at
 *    offsets floor(i*cnt/b), i = 0..b-1, in suffix order, so each continuation
 *    prefix keeps its frequency to within one; otherwise all are kept;
 *  - the continuation of an occurrence at j of a length-n suffix is
 *    T[j+n .. j+n+m), cut before the first 0 and at the end of T;
 *  - slot layout per query: store 0's slots in suffix order, then store 1's,
 *    ...; unused slots hold pos 0xFFFFFFFF, src 0xFF, len 0, tokens 0;
 *  - cont_pos is the text position where the continuation starts (j + n).
 *
 * Arrays: ctx [B][L]; match_n, range_lo, range_cnt, taken [B][S];
 * cont_pos, cont_src, cont_len [B][k]; cont_tok [B][k][m].
 */
void oracle_retrieve(int S, const uint16_t* const* texts, const uint64_t* lens, const uint16_t* ctx, int B, int L,
                     int n_max, int n_min, int k, int m, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                     int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len, uint16_t* cont_tok) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    const uint16_t* row = ctx + (size_t)b * L;
    uint32_t* pos = cont_pos + (size_t)b * k;
    uint8_t* src = cont_src + (size_t)b * k;
    uint8_t* len = cont_len + (size_t)b * k;
    uint16_t* tok = cont_tok + (size_t)b * k * m;
    for (int i = 0; i < k; ++i) {
      pos[i] = 0xFFFFFFFFu;
      src[i] = 0xFF;
      len[i] = 0;
    }
    memset(tok, 0, (size_t)k * m * sizeof(uint16_t));
    int64_t used = 0;
    for (int s = 0; s < S; ++s) {
      source_match sm;
      match_one_source(texts[s], lens[s], row, L, n_max, n_min, &sm);
      int64_t budget = k - used;
      int64_t t = (int64_t)sm.range_cnt < budget ? (int64_t)sm.range_cnt : budget;
      match_n[b * S + s] = sm.match_n;
      range_lo[b * S + s] = sm.range_lo;
      range_cnt[b * S + s] = sm.range_cnt;
      taken[b * S + s] = (int32_t)t;
      for (int64_t i = 0; i < t; ++i) {
        uint64_t off = ((int64_t)sm.range_cnt > budget) ? (uint64_t)i * sm.range_cnt / (uint64_t)budget : (uint64_t)i;
        uint64_t start = (uint64_t)sm.occ[off] + (uint64_t)sm.match_n;
        int64_t slot = used + i;
        int l = 0;
        while (l < m && start + l < lens[s] && texts[s][start + l] != 0) {
          tok[slot * m + l] = texts[s][start + l];
          ++l;
        }
        pos[slot] = (uint32_t)start;
        src[slot] = (uint8_t)s;
        len[slot] = (uint8_t)l;
      }
      used += t;
      free(sm.occ);
    }
  }
}

/*
 * The same retrieval as oracle_retrieve, computed with the text scans shared
 * by the whole batch: each store is read by one pass per question instead of
 * three passes per query, which makes batches of a thousand queries over a
 * billion-token store practical on the CPU.  Every query's answer is the one
 * oracle_retrieve defines, step for step:
 *   1. its longest occurring suffix: the agreement of the context with the
 *      text before every end position e, capped at n_hi; the queries are
 *      listed by their last token, so at e only the queries whose last token
 *      is T[e-1] are compared (for the others the agreement is 0);
 *   2. for the chosen q_n, at every start j: when T[j] equals q_n's first
 *      token, the suffix at j is compared with q_n (an occurrence, or below,
 *      or above); a suffix whose first token is smaller than q_n's is below,
 *      counted through the number of start positions per first token;
 *   3. the occurrences in suffix order by the direct suffix comparison;
 *   4. the budget fill, strided picks and continuation cut of
 *      oracle_retrieve.
 * Steps 1 and 2 split the text into chunks, one per thread, and add up
 * per-thread results; nothing else is reordered.
 */
typedef struct {
  uint32_t* v;
  uint64_t n, cap;
} u32_list;

static void u32_push(u32_list* l, uint32_t x) {
  if (l->n == l->cap) {
    l->cap = l->cap ? 2 * l->cap : 16;
    l->v = (uint32_t*)realloc(l->v, l->cap * sizeof(uint32_t));
  }
  l->v[l->n++] = x;
}

static int omp_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

static int omp_thread(void) {
#ifdef _OPENMP
  return omp_get_thread_num();
#else
  return 0;
#endif
}

/* match_n, range_lo, occurrences (suffix order) of every query in one store */
static void match_batch_one_source(const uint16_t* T, uint64_t N, const uint16_t* ctx, int B, int L, int n_max,
                                   int n_min, source_match* out) {
  const int nt = omp_threads();
  int* n_hi = (int*)malloc((size_t)(B ? B : 1) * sizeof(int));
  int* head = (int*)malloc(65536 * sizeof(int));
  int* next = (int*)malloc((size_t)(B ? B : 1) * sizeof(int));
  for (int b = 0; b < B; ++b) {
    out[b].match_n = 0;
    out[b].range_lo = 0;
    out[b].range_cnt = 0;
    out[b].occ = NULL;
    n_hi[b] = query_limit(ctx + (size_t)b * L, L, n_max);
  }
  if (N > 0) {
    /* step 1: longest agreement before every end position, per query */
    for (int t = 0; t < 65536; ++t) head[t] = -1;
    for (int b = B - 1; b >= 0; --b) {
      if (n_hi[b] < n_min || n_hi[b] < 1) continue;
      const uint16_t last = ctx[(size_t)b * L + L - 1];
      next[b] = head[last];
      head[last] = b;
    }
    int* best = (int*)calloc((size_t)nt * (B ? B : 1), sizeof(int));
#pragma omp parallel
    {
      int* mine = best + (size_t)omp_thread() * (B ? B : 1);
#pragma omp for schedule(static)
      for (uint64_t e = 1; e <= N; ++e) {
        for (int b = head[T[e - 1]]; b >= 0; b = next[b]) {
          const uint16_t* end = ctx + (size_t)b * L + L;
          int l = 0;
          while (l < n_hi[b] && (uint64_t)l < e && T[e - 1 - l] == end[-1 - l]) ++l;
          if (l > mine[b]) mine[b] = l;
        }
      }
    }
    for (int b = 0; b < B; ++b) {
      int l = 0;
      for (int t = 0; t < nt; ++t)
        if (best[(size_t)t * B + b] > l) l = best[(size_t)t * B + b];
      out[b].match_n = l >= n_min ? l : 0;
    }
    free(best);

    /* step 2: occurrences and the suffixes below q_n, per query */
    {
      uint64_t* first = (uint64_t*)calloc(65536, sizeof(uint64_t)); /* start positions per first token */
      for (int t = 0; t < 65536; ++t) head[t] = -1;
      for (int b = B - 1; b >= 0; --b) {
        const int n = out[b].match_n;
        if (n == 0) continue;
        const uint16_t q0 = ctx[(size_t)b * L + L - n];
        next[b] = head[q0];
        head[q0] = b;
      }
      uint64_t* below = (uint64_t*)calloc((size_t)nt * (B ? B : 1), sizeof(uint64_t));
      u32_list* occ = (u32_list*)calloc((size_t)nt * (B ? B : 1), sizeof(u32_list));
      uint64_t* first_t = (uint64_t*)calloc((size_t)nt * 65536, sizeof(uint64_t));
#pragma omp parallel
      {
        const int me = omp_thread();
        uint64_t* my_below = below + (size_t)me * (B ? B : 1);
        u32_list* my_occ = occ + (size_t)me * (B ? B : 1);
        uint64_t* my_first = first_t + (size_t)me * 65536;
#pragma omp for schedule(static)
        for (uint64_t j = 0; j < N; ++j) {
          my_first[T[j]]++;
          for (int b = head[T[j]]; b >= 0; b = next[b]) {
            const int n = out[b].match_n;
            const int c = cmp_suffix_pattern(T, N, j, ctx + (size_t)b * L + L - n, n);
            if (c < 0) my_below[b]++;
            else if (c == 0) u32_push(&my_occ[b], (uint32_t)j);
          }
        }
      }
      for (int t = 0; t < nt; ++t)
        for (int x = 0; x < 65536; ++x) first[x] += first_t[(size_t)t * 65536 + x];
#pragma omp parallel for schedule(dynamic, 1)
      for (int b = 0; b < B; ++b) {
        const int n = out[b].match_n;
        if (n == 0) continue;
        const uint16_t q0 = ctx[(size_t)b * L + L - n];
        uint64_t lo = 0, cnt = 0;
        for (int x = 0; x < q0; ++x) lo += first[x];
        for (int t = 0; t < nt; ++t) {
          lo += below[(size_t)t * B + b];
          cnt += occ[(size_t)t * B + b].n;
        }
        uint32_t* all = (uint32_t*)malloc((size_t)(cnt ? cnt : 1) * sizeof(uint32_t));
        uint64_t at = 0;
        for (int t = 0; t < nt; ++t) {
          u32_list* l = &occ[(size_t)t * B + b];
          if (l->n) memcpy(all + at, l->v, l->n * sizeof(uint32_t));
          at += l->n;
          free(l->v);
        }
        /* step 3 */
        text_ref tr = {T, N};
        qsort_r(all, cnt, sizeof(uint32_t), cmp_sa_entries, &tr);
        out[b].range_lo = (uint32_t)lo;
        out[b].range_cnt = (uint32_t)cnt;
        out[b].occ = all;
      }
      free(first_t);
      free(occ);
      free(below);
      free(first);
    }
  }
  free(next);
  free(head);
  free(n_hi);
}

void oracle_retrieve_batched(int S, const uint16_t* const* texts, const uint64_t* lens, const uint16_t* ctx, int B,
                             int L, int n_max, int n_min, int k, int m, int32_t* match_n, uint32_t* range_lo,
                             uint32_t* range_cnt, int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src,
                             uint8_t* cont_len, uint16_t* cont_tok) {
  source_match* sm = (source_match*)malloc((size_t)(B ? B : 1) * S * sizeof(source_match));
  for (int s = 0; s < S; ++s) match_batch_one_source(texts[s], lens[s], ctx, B, L, n_max, n_min, sm + (size_t)s * B);
  /* step 4: exactly the fill of oracle_retrieve */
#pragma omp parallel for schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    uint32_t* pos = cont_pos + (size_t)b * k;
    uint8_t* src = cont_src + (size_t)b * k;
    uint8_t* len = cont_len + (size_t)b * k;
    uint16_t* tok = cont_tok + (size_t)b * k * m;
    for (int i = 0; i < k; ++i) {
      pos[i] = 0xFFFFFFFFu;
      src[i] = 0xFF;
      len[i] = 0;
    }
    memset(tok, 0, (size_t)k * m * sizeof(uint16_t));
    int64_t used = 0;
    for (int s = 0; s < S; ++s) {
      const source_match* x = &sm[(size_t)s * B + b];
      int64_t budget = k - used;
      int64_t t = (int64_t)x->range_cnt < budget ? (int64_t)x->range_cnt : budget;
      match_n[b * S + s] = x->match_n;
      range_lo[b * S + s] = x->range_lo;
      range_cnt[b * S + s] = x->range_cnt;
      taken[b * S + s] = (int32_t)t;
      for (int64_t i = 0; i < t; ++i) {
        uint64_t off = ((int64_t)x->range_cnt > budget) ? (uint64_t)i * x->range_cnt / (uint64_t)budget : (uint64_t)i;
        uint64_t start = (uint64_t)x->occ[off] + (uint64_t)x->match_n;
        int64_t slot = used + i;
        int l = 0;
        while (l < m && start + l < lens[s] && texts[s][start + l] != 0) {
          tok[slot * m + l] = texts[s][start + l];
          ++l;
        }
        pos[slot] = (uint32_t)start;
        src[slot] = (uint8_t)s;
        len[slot] = (uint8_t)l;
      }
      used += t;
    }
  }
  for (size_t i = 0; i < (size_t)B * S; ++i) free(sm[i].occ);
  free(sm);
}

/* ------------------------------------------------------------------------- */
/* Weighted trie, top-c selection, tree emission (Section IV-D, eq. (3)-(4)).  */
/* ------------------------------------------------------------------------- */

typedef struct {
  uint16_t tok;
  int32_t depth;
  uint64_t weight;
  int32_t parent, first_child, next_sibling; /* children kept in token order */
  int32_t selected, out_index;
} tnode;

typedef struct {
  tnode* nodes;
  int32_t count;
} trie;

static int32_t trie_child(trie* t, int32_t u, uint16_t tok, int create) {
  int32_t prev = -1, v = t->nodes[u].first_child;
  while (v >= 0 && t->nodes[v].tok < tok) {
    prev = v;
    v = t->nodes[v].next_sibling;
  }
  if (v >= 0 && t->nodes[v].tok == tok) return v;
  if (!create) return -1;
  int32_t w = t->count++;
  tnode* n = &t->nodes[w];
  n->tok = tok;
  n->depth = t->nodes[u].depth + 1;
  n->weight = 0;
  n->parent = u;
  n->first_child = -1;
  n->next_sibling = v;
  n->selected = 0;
  n->out_index = -1;
  if (prev < 0) t->nodes[u].first_child = w; else t->nodes[prev].next_sibling = w;
  return w;
}

/* Tokens of the path root -> v into buf (length = depth). */
static int trie_path(const trie* t, int32_t v, uint16_t* buf) {
  int d = t->nodes[v].depth;
  for (int x = d - 1; x >= 0; --x) {
    buf[x] = t->nodes[v].tok;
    v = t->nodes[v].parent;
  }
  return d;
}

typedef struct {
  const trie* t;
  uint16_t *pa, *pb;
} rank_ctx;

/*
 * Selection order (reading; the paper names no tie-break): higher weight
 * first; equal weights by path, compared token by token, a prefix before its
 * extensions.  A parent never ranks below its child (its weight is at least
 * the child's and its path is a prefix), so any top-c set is closed under
 * taking ancestors.
 */
static int cmp_rank(const void* a, const void* b, void* vctx) {
  rank_ctx* c = (rank_ctx*)vctx;
  int32_t u = *(const int32_t*)a, v = *(const int32_t*)b;
  uint64_t wu = c->t->nodes[u].weight, wv = c->t->nodes[v].weight;
  if (wu != wv) return wu > wv ? -1 : 1;
  int du = trie_path(c->t, u, c->pa), dv = trie_path(c->t, v, c->pb);
  for (int x = 0; x < du && x < dv; ++x)
    if (c->pa[x] != c->pb[x]) return c->pa[x] < c->pb[x] ? -1 : 1;
  return (du < dv) ? -1 : (du > dv) ? 1 : 0;
}

/* Preorder walk (children in token order) that numbers the selected nodes. */
static void emit_preorder(trie* t, int32_t u, int32_t* next_index) {
  for (int32_t v = t->nodes[u].first_child; v >= 0; v = t->nodes[v].next_sibling) {
    if (t->nodes[v].selected) {
      t->nodes[v].out_index = (*next_index)++;
      emit_preorder(t, v, next_index);
    }
  }
}

/*
 * Draft tree per query.
 *
 * The slots of query b belong to store s when they fall in its taken range
 * (store 0's taken slots first, then store 1's, ...); later slots are unused.
 * Every non-empty continuation is inserted into a trie rooted at the last
 * context token; node weight = sum of alpha[s] over the continuations that
 * pass through it (eq. (3) with t_r, t_c the occurrence counts in R_r, R_c).
 * The c highest nodes in the selection order above are kept (at most c draft
 * tokens).  Output row 0 is the root (token ctx[L-1], parent -1, weight = sum
 * of alpha over non-empty continuations, depth 0), followed by the kept nodes
 * in preorder with children in token order.  pos_ids = depth (the caller adds
 * its own offset).  mask[i][j] = 1 iff j is i or an ancestor of i, the root
 * included (eq. (4) read with the diagonal set, since a token attends to
 * itself).  Rows past num_nodes are padding: token 0, parent -1, weight 0,
 * pos 0, mask row and column 0.
 *
 * Arrays: alpha [S]; taken [B][S]; cont_len [B][k]; cont_tok [B][k][m];
 * ctx [B][L]; num_nodes [B]; node_tok, parent, pos_ids [B][c+1];
 * weight [B][c+1]; mask [B][c+1][c+1].
 */
void oracle_build_tree(int B, int S, int k, int m, int c, const uint32_t* alpha, const int32_t* taken,
                       const uint8_t* cont_len, const uint16_t* cont_tok, const uint16_t* ctx, int L,
                       int32_t* num_nodes, int32_t* node_tok, int32_t* parent, uint32_t* weight, int32_t* pos_ids,
                       int32_t* mask) {
  const int R = c + 1;
#pragma omp parallel for schedule(dynamic, 1)
  for (int b = 0; b < B; ++b) {
    int64_t total_len = 0;
    for (int i = 0; i < k; ++i) total_len += cont_len[(size_t)b * k + i];
    trie t;
    t.nodes = (tnode*)malloc((size_t)(total_len + 1) * sizeof(tnode));
    t.count = 1;
    tnode* root = &t.nodes[0];
    root->tok = ctx[(size_t)b * L + L - 1];
    root->depth = 0;
    root->weight = 0;
    root->parent = -1;
    root->first_child = -1;
    root->next_sibling = -1;
    root->selected = 1;
    root->out_index = 0;

    int slot = 0;
    for (int s = 0; s < S; ++s) {
      for (int32_t i = 0; i < taken[b * S + s]; ++i, ++slot) {
        int l = cont_len[(size_t)b * k + slot];
        if (l == 0) continue;
        const uint16_t* str = cont_tok + ((size_t)b * k + slot) * m;
        int32_t u = 0;
        t.nodes[0].weight += alpha[s];
        for (int x = 0; x < l; ++x) {
          u = trie_child(&t, u, str[x], 1);
          t.nodes[u].weight += alpha[s];
        }
      }
    }

    int32_t n_cand = t.count - 1;
    int32_t* order = (int32_t*)malloc((size_t)(n_cand ? n_cand : 1) * sizeof(int32_t));
    for (int32_t i = 0; i < n_cand; ++i) order[i] = i + 1;
    uint16_t* pa = (uint16_t*)malloc((size_t)(m + 1) * sizeof(uint16_t));
    uint16_t* pb = (uint16_t*)malloc((size_t)(m + 1) * sizeof(uint16_t));
    rank_ctx rc = {&t, pa, pb};
    qsort_r(order, n_cand, sizeof(int32_t), cmp_rank, &rc);
    int32_t keep = n_cand < c ? n_cand : c;
    for (int32_t i = 0; i < keep; ++i) t.nodes[order[i]].selected = 1;
    int32_t next_index = 1;
    emit_preorder(&t, 0, &next_index);

    int32_t* tok_o = node_tok + (size_t)b * R;
    int32_t* par_o = parent + (size_t)b * R;
    uint32_t* w_o = weight + (size_t)b * R;
    int32_t* pos_o = pos_ids + (size_t)b * R;
    int32_t* mask_o = mask + (size_t)b * R * R;
    for (int i = 0; i < R; ++i) {
      tok_o[i] = 0;
      par_o[i] = -1;
      w_o[i] = 0;
      pos_o[i] = 0;
    }
    memset(mask_o, 0, (size_t)R * R * sizeof(int32_t));
    for (int32_t v = 0; v < t.count; ++v) {
      if (!t.nodes[v].selected) continue;
      int32_t o = t.nodes[v].out_index;
      tok_o[o] = t.nodes[v].tok;
      par_o[o] = (v == 0) ? -1 : t.nodes[t.nodes[v].parent].out_index;
      w_o[o] = (uint32_t)t.nodes[v].weight;
      pos_o[o] = t.nodes[v].depth;
    }
    num_nodes[b] = next_index;
    for (int32_t i = 0; i < next_index; ++i)
      for (int32_t j = i; j >= 0; j = par_o[j]) mask_o[(size_t)i * R + j] = 1;

    free(pa);
    free(pb);
    free(order);
    free(t.nodes);
  }
}

/* ------------------------------------------------------------------------- */
/* Acceptance (Section IV-D: every correct token from the start is accepted,   */
/* everything after the first error is rejected).                              */
/* ------------------------------------------------------------------------- */

/*
 * target[b][i] is the target model's next token after tree row i (-1 when
 * there is none).  From the root, step to the child whose token equals the
 * target at the current node while one exists (children carry distinct
 * tokens).  accept_len = depth(u) + 1 (the path plus the target's own token
 * at u), or depth(u) when target[u] is -1.  accept_tok lists the path tokens
 * then target[u]; unused entries are -1.  last_node = u.
 * Precondition: no row is deeper than m (every tree built from continuations
 * of at most m tokens meets it).  accept_tok holds m + 1 tokens, so for a
 * deeper tree the walk stops once m + 1 tokens are accepted (and the
 * target's own token is then not added); nothing is written past m + 1.
 * Arrays: num_nodes [B]; node_tok, parent, pos_ids, target [B][c+1];
 * accept_len, last_node [B]; accept_tok [B][m+1].
 */
void oracle_verify_accept(int B, int c, int m, const int32_t* num_nodes, const int32_t* node_tok,
                          const int32_t* parent, const int32_t* pos_ids, const int32_t* target, int32_t* accept_len,
                          int32_t* accept_tok, int32_t* last_node) {
  const int R = c + 1;
  for (int b = 0; b < B; ++b) {
    const int32_t* tok = node_tok + (size_t)b * R;
    const int32_t* par = parent + (size_t)b * R;
    const int32_t* tgt = target + (size_t)b * R;
    int32_t* out = accept_tok + (size_t)b * (m + 1);
    for (int i = 0; i <= m; ++i) out[i] = -1;
    int32_t u = 0, n = num_nodes[b];
    int len = 0;
    for (;;) {
      if (len == m + 1) break; /* accept_tok is full: only a tree deeper than m gets here */
      int32_t next = -1;
      if (tgt[u] >= 0)
        for (int32_t v = 1; v < n; ++v)
          if (par[v] == u && tok[v] == tgt[u]) {
            next = v;
            break;
          }
      if (next < 0) break;
      out[len++] = tok[next];
      u = next;
    }
    if (tgt[u] >= 0 && len < m + 1) out[len++] = tgt[u];
    (void)pos_ids;
    accept_len[b] = len;
    last_node[b] = u;
  }
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
