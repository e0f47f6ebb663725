/*
 * fastcoder.h - C ABI of the MI355X (gfx950) draft-stage library for
 * retrieval-based speculative decoding after FastCoder (arXiv 2502.17139).
 *
 * The library implements the data-parallel hot path of the draft stage:
 * suffix-array construction over token datastores, longest-suffix retrieval
 * over prioritised stores with continuation gather, the frequency-weighted
 * draft trie pruned to c nodes with its tree-attention mask and position ids,
 * and greedy acceptance of the longest matching root-to-leaf path.
 *
 * Conventions shared by every entry point:
 *  - Buffers named in a signature are DEVICE pointers (HBM) owned by the
 *    caller, unless marked "host".  The library never allocates or frees
 *    device memory; scratch space comes from a caller-provided workspace whose
 *    size the matching *_workspace_bytes function reports.
 *  - Calls enqueue work on `stream` and return without waiting, except
 *    fc_datastore_build, which synchronises `stream` between its rounds.
 *  - Arguments are validated on the host before anything is launched; a
 *    failed check returns its status and writes nothing.  FC_ERR_DEVICE
 *    reports a HIP launch or runtime error.  No exception crosses the ABI,
 *    nothing calls exit/abort, and there is no global mutable state: calls on
 *    different streams may run concurrently when their buffers do not overlap.
 *  - Arrays are row-major and densely packed; [B][k] means B rows of k.
 *  - Tokens are uint16.  Token 0 separates files: a context never reaches
 *    back past a 0, so no match straddles two files.
 */
#ifndef FASTCODER_H
#define FASTCODER_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum fc_status {
  FC_OK = 0,
  FC_ERR_INVALID = 1,     /* null pointer, size or parameter out of range */
  FC_ERR_WORKSPACE = 2,   /* workspace pointer null or smaller than required */
  FC_ERR_DEVICE = 3,      /* HIP launch/runtime error, or a device-side check failed */
  FC_ERR_UNSUPPORTED = 4  /* valid request outside what the library handles */
} fc_status;

#define FC_MAX_SOURCES 4     /* stores per retrieval */
#define FC_MAX_NMAX 16       /* longest context suffix searched (n_max) */
#define FC_MAX_TREE_ROWS 256 /* c + 1 (root + kept nodes) */
#define FC_BUCKETS 65537     /* entries of a store's first-token table */

/* ABI revision; bumped on any incompatible change. */
int32_t fc_abi_version(void);

/* Human-readable name of a status code (static storage, never NULL). */
const char* fc_status_string(fc_status s);

/* ------------------------------------------------------------------------ */
/* Datastore index                                                           */
/* ------------------------------------------------------------------------ */

/*
 * Suffix array of a token datastore (Section III-A: exact suffix matching
 * over a suffix array after Manber and Myers; Section IV-A: every position of
 * a file splits it into a context and a continuation).
 *
 * tokens [n]   : the datastore text, files joined by single 0 tokens.
 * sa_out [n]   : receives the start positions 0..n-1 sorted by suffix order:
 *                token by token by numeric id, a suffix that ends first
 *                (a proper prefix) sorting lower.  The order is total, so the
 *                result is unique.
 * ws, ws_bytes : workspace of at least fc_datastore_build_workspace_bytes(n)
 *                (about 28.6 bytes per token, 36.6 from 2^26 tokens on).
 * Built by prefix doubling: suffixes are sorted by their first 3 tokens, then
 * by (rank of the first h tokens, rank of the h tokens after them) with h
 * doubling, each round an LSD radix sort restricted to still-tied suffixes.
 * Synchronises `stream` once per round (it reads the number of tied
 * suffixes).  Requires n < 2^32 - 1.  n == 0 is a no-op.
 */
size_t fc_datastore_build_workspace_bytes(uint64_t n);
fc_status fc_datastore_build(const uint16_t* tokens, uint64_t n, uint32_t* sa_out, void* ws, size_t ws_bytes,
                             hipStream_t stream);

/*
 * fc_datastore_build that also reports how the doubling went (host struct,
 * filled when the call returns; stats may be NULL).  Round r sorted the
 * sorted[r] suffixes still tied after round r - 1 by their first
 * prefix_len[r] tokens, and left unresolved[r] of them tied.  The last
 * round leaves none tied, so the longest common prefix of two suffixes is
 * below prefix_len[rounds - 1] and, when rounds > 1, at least
 * prefix_len[rounds - 2].  sort_passes counts the radix passes run (a pass
 * per key byte that is not the same for every suffix).
 */
#define FC_MAX_BUILD_ROUNDS 40
typedef struct fc_build_stats {
  int32_t rounds;
  int32_t sort_passes;
  uint64_t prefix_len[FC_MAX_BUILD_ROUNDS];
  uint64_t sorted[FC_MAX_BUILD_ROUNDS];
  uint64_t unresolved[FC_MAX_BUILD_ROUNDS];
} fc_build_stats;
fc_status fc_datastore_build_stats(const uint16_t* tokens, uint64_t n, uint32_t* sa_out, void* ws, size_t ws_bytes,
                                   fc_build_stats* stats, hipStream_t stream);

/*
 * Batched construction of many small stores (per-repository stores, Section
 * IV-A: the repository store is built per repository, offline, Section
 * V-D).  tokens holds n_seg stores back to back, store r at
 * [seg_off[r], seg_off[r+1]) (seg_off on the host: seg_off[0] = 0,
 * non-decreasing, total n = seg_off[n_seg] < 2^32 - 1; empty stores
 * allowed).  On return sa_out[seg_off[r] .. seg_off[r+1]) is exactly the
 * suffix array fc_datastore_build gives for store r alone, with positions
 * local to that store.  One prefix-doubling build covers every store: the
 * store index leads each suffix's first key and a suffix ends at its own
 * store's end.  Workspace of fc_datastore_build_batched_workspace_bytes(n,
 * n_seg) bytes; synchronises `stream` once per doubling round, as
 * fc_datastore_build does.
 */
size_t fc_datastore_build_batched_workspace_bytes(uint64_t n, int32_t n_seg);
fc_status fc_datastore_build_batched(const uint16_t* tokens, const uint64_t* seg_off, int32_t n_seg,
                                     uint32_t* sa_out, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Extension of a store by new files without a full rebuild (a repository
 * store grows as its files are written, Section IV-A; the suffix array is
 * the Section III-A index).  The new files go in FRONT of the old store:
 * tokens[n] = new[n_new] . old[n - n_new], where new already ends with the
 * 0 token that joins it to the old store's first file.  Every suffix of the
 * old store is then a suffix of the new text, so its order is kept and
 * only the n_new new suffixes are sorted: each is first placed among the
 * old suffixes by doubling over the old array and its inverse, then the
 * new suffixes are ordered among themselves by prefix doubling, and the two
 * lists are merged.
 *
 * old_sa [n - n_new]  : suffix array of tokens[n_new .. n) alone (as
 *                       fc_datastore_build gives it; positions local to the
 *                       old store).  Read only.
 * old_isa [n - n_new] : optional (NULL: computed in the workspace, one
 *                       random-write pass over the old store): its inverse,
 *                       old_isa[old_sa[j]] = j.  A store that keeps its
 *                       inverse (isa_out of its last extension) skips that
 *                       pass.
 * sa_out [n]          : receives exactly what fc_datastore_build(tokens, n)
 *                       would.
 * isa_out [n]         : optional: receives the inverse of sa_out.
 * No output may overlap an input.  Workspace of
 * fc_datastore_extend_workspace_bytes(n, n_new, old_isa != NULL) bytes
 * (without old_isa it holds the inverse: 4 bytes per old token).
 * n_new == 0 copies old_sa (and inverts it into isa_out); n == n_new is a
 * plain build.  Requires n < 2^32 - 1 and n_new <= n.  Synchronises
 * `stream` once per doubling round.  If old_sa (or old_isa) is not the old
 * store's array the result is unspecified (no access leaves the buffers).
 */
size_t fc_datastore_extend_workspace_bytes(uint64_t n, uint64_t n_new, int32_t isa_given);
fc_status fc_datastore_extend(const uint16_t* tokens, uint64_t n, uint64_t n_new, const uint32_t* old_sa,
                              const uint32_t* old_isa, uint32_t* sa_out, uint32_t* isa_out, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/*
 * First-token table of a store: bucket_out[t] (t = 0..65536) = number of
 * suffixes whose first token is below t, i.e. the suffix-array index where
 * suffixes starting with token t begin (the bucket table Manber and Myers
 * use to shorten the search).  bucket_out has FC_BUCKETS entries.
 */
fc_status fc_store_prepare(const uint16_t* tokens, const uint32_t* sa, uint64_t n, uint32_t* bucket_out,
                           hipStream_t stream);

/*
 * Optional two-token prefix table of a store (the same bucket idea one token
 * deeper): for every pair (t0, u) with t0 < V and u in [0, V],
 * pair_out[t0*(V+1) + u] = number of suffixes whose first two tokens sort
 * below (t0, u), where u = 0 stands for "the suffix ends after t0" and
 * u = t1 + 1 for a second token t1; the last entry, index V*(V+1), is n.
 * A search for a pattern starting with (t0, t1) then starts from the range
 * [pair[t0*(V+1)+t1+1], pair[t0*(V+1)+t1+2]) instead of the whole first-token
 * bucket.  pair_out holds fc_pair_table_entries(V) entries (4.16 GB at
 * V = 32256).  V must exceed every token of the store: the call checks it,
 * which synchronises `stream`, and returns FC_ERR_INVALID otherwise (the
 * table is then unspecified).  1 <= V <= 65536.
 */
uint64_t fc_pair_table_entries(uint32_t V);
fc_status fc_store_prepare_pairs(const uint16_t* tokens, const uint32_t* sa, uint64_t n, uint32_t V,
                                 uint32_t* pair_out, hipStream_t stream);

/*
 * Optional inline-prefix records of a store.  Record i is FC_RECORD_BYTES =
 * 64 bytes: sa[i] as a uint32, then the FC_RECORD_TOKENS = 30 tokens
 * T[sa[i]+2 .. sa[i]+32) as uint16 (0 for positions at or past n).
 * - A suffix search of Section III-A reads one record per probe and decides
 *   the comparison from it alone (the two-token table fixes the first two
 *   tokens and n_max <= 16), so a probe costs one memory round trip and no
 *   second, dependent read of the text.  A 0 stored past the end compares
 *   exactly like the end itself: query tokens are never 0.
 * - The continuation gather of a match of length n >= 2 reads its m tokens
 *   from the same record when they lie inside it (n + m <= 30 or so,
 *   depending on alignment), so a kept slot costs one read of 64 contiguous
 *   bytes at its suffix-array position instead of a suffix-array read
 *   followed by a random read of the text.
 * rec_out is fc_record_bytes(n) bytes (64 GB at n = 1e9, affordable in a
 * 288 GB HBM part), 64-byte aligned, written on `stream`.
 */
#define FC_RECORD_BYTES 64
#define FC_RECORD_TOKENS 30
uint64_t fc_record_bytes(uint64_t n);
fc_status fc_store_prepare_records(const uint16_t* tokens, const uint32_t* sa, uint64_t n, void* rec_out,
                                   hipStream_t stream);

/*
 * Optional top-level sample of a store's records for the suffix search of
 * Section III-A: entry t is the first FC_TOP_BYTES = 32 bytes of record
 * t * FC_TOP_STRIDE (its suffix-array entry and tokens 2..15), for t = 0 ..
 * ceil(n / FC_TOP_STRIDE) - 1.  A search whose two-token range spans more
 * than two sample strides first narrows the range over the sample (a dense
 * array of n / 8 bytes: 125 MB at n = 1e9, small enough to stay in the
 * memory-side cache), then finishes inside one stride of the records, so
 * most of its dependent round trips avoid the 64-byte-per-suffix records.
 * Results are identical with or without it.
 * top_out is fc_store_top_bytes(n) bytes, 32-byte aligned, written on
 * `stream` from the store's records (rec, as from fc_store_prepare_records).
 */
#define FC_TOP_STRIDE 256
#define FC_TOP_BYTES 32
uint64_t fc_store_top_bytes(uint64_t n);
fc_status fc_store_prepare_top(const void* rec, uint64_t n, void* top_out, hipStream_t stream);

/* A read-only view of one store; all pointers are device pointers. */
typedef struct fc_store {
  const uint16_t* tokens; /* [n] text */
  const uint32_t* sa;     /* [n] suffix array of tokens */
  const uint32_t* bucket; /* [FC_BUCKETS] table from fc_store_prepare */
  uint64_t n;             /* tokens in the store, < 2^32 - 1 */
  const uint32_t* pair;   /* optional two-token table from fc_store_prepare_pairs, or NULL */
  uint32_t pair_vocab;    /* its V (ignored when pair is NULL) */
  const void* rec;        /* optional records from fc_store_prepare_records (needs pair), or NULL */
  const void* top;        /* optional sample from fc_store_prepare_top (needs rec), or NULL */
} fc_store;

/* ------------------------------------------------------------------------ */
/* Retrieval                                                                 */
/* ------------------------------------------------------------------------ */

typedef struct fc_retrieve_params {
  int32_t n_max; /* longest context suffix tried, 1..16 (paper: 16) */
  int32_t n_min; /* shortest suffix tried, 1..n_max */
  int32_t k;     /* continuation slots per query (retrieval cap), >= 1 */
  int32_t m;     /* tokens per continuation, 1..255 */
} fc_retrieve_params;

/*
 * Batched longest-suffix retrieval over S stores in priority order
 * (Section III-A; two stores, the repository store first and the common store
 * second, searched side by side: Section IV-A, Section IV-C).
 *
 * stores (host) [S] : store views, S in 1..FC_MAX_SOURCES.  A store with
 *                    records must also have a two-token table, and its
 *                    records must be 64-byte aligned (FC_ERR_INVALID).
 * ctx [B][L]        : the last L context tokens of each query.
 * For each query and store: n_hi = min(n_max, L, trailing non-zero tokens of
 * the context); for n = n_hi down to n_min the suffix q = ctx[L-n..L) is
 * searched and the first n with an occurrence wins.
 * match_n   [B][S] : that n, or 0 when no n in [n_min, n_hi] occurs.
 * range_lo  [B][S] : suffix-array index of the first suffix starting with q
 *                    (0 when there is no match).
 * range_cnt [B][S] : number of occurrences of q.
 * taken     [B][S] : slots store s fills: min(k - slots of stores before it,
 *                    range_cnt).  When range_cnt exceeds that budget b, the
 *                    occurrences at range offsets floor(i*range_cnt/b),
 *                    i = 0..b-1, are kept (a strided sample that keeps every
 *                    continuation prefix's share to within one); otherwise
 *                    all are kept, in suffix-array order.
 * Slot i of a query: store 0's kept occurrences first, then store 1's, ...;
 * slots at or past the query's total taken are not written (their contents
 * are whatever the buffers held), which saves writing k slots per query.
 * cont_pos [B][k]    : text position where the continuation starts (match
 *                      start + match_n).
 * cont_src [B][k]    : store index.
 * cont_len [B][k]    : continuation length 0..m: up to m tokens, cut before
 *                      the first 0 and at the end of the store.
 * cont_tok [B][k][m] : continuation tokens, 0 past cont_len.
 * Within one store's slots the continuations come out in lexicographic order
 * (suffix order), which fc_build_tree relies on.
 * rows [B], n_rows : optional row map.  When rows is not NULL, query b's
 *                per-store results and slots go to row rows[b] of every output
 *                array, which then has n_rows rows ([n_rows][S], [n_rows][k],
 *                [n_rows][k][m]) - e.g. straight into the slots of a
 *                retrieval cache.  Rows must be distinct; a query whose row
 *                is outside [0, n_rows) is skipped.  When rows is NULL, row b
 *                is query b and n_rows is ignored.
 * ws, ws_bytes : workspace of at least fc_retrieve_workspace_bytes(B, S, p)
 *                (4*(B+1) bytes: the batch's slot offsets); its contents on
 *                entry do not matter.
 * B * k must not exceed 2^31 - 1 (the batch's slots are numbered in 32
 * bits with room for the grid stride); FC_ERR_UNSUPPORTED otherwise.
 */
size_t fc_retrieve_workspace_bytes(int32_t B, int32_t S, fc_retrieve_params p);
fc_status fc_retrieve(const fc_store* stores, int32_t S, const uint16_t* ctx, int32_t B, int32_t L,
                      fc_retrieve_params p, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                      int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len, uint16_t* cont_tok,
                      const int32_t* rows, int32_t n_rows, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * fc_retrieve without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, outputs and checks as fc_retrieve;
 * the workspace is a static device array of FC_RETRIEVE_NOALLOC_BYTES that
 * the library holds on every GPU it runs on until the process ends.  The
 * call allocates nothing.  Limit: fc_retrieve_workspace_bytes(B, S, p) must
 * not exceed FC_RETRIEVE_NOALLOC_BYTES (FC_ERR_UNSUPPORTED otherwise, before
 * anything touches the device).  Every call on one GPU uses that GPU's one
 * array, so calls that overlap on the same GPU (different streams or host
 * threads) race and must be serialised by the caller.  The first call on a
 * device looks the array's address up (FC_ERR_DEVICE if that fails).
 */
#define FC_RETRIEVE_NOALLOC_BYTES (1u << 20)
size_t fc_retrieve_noalloc_max_bytes(void);
fc_status fc_retrieve_noalloc(const fc_store* stores, int32_t S, const uint16_t* ctx, int32_t B, int32_t L,
                              fc_retrieve_params p, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                              int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len,
                              uint16_t* cont_tok, const int32_t* rows, int32_t n_rows, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* CACHE (Section IV-B)                                                      */
/* ------------------------------------------------------------------------ */

#define FC_MAX_CACHE_TOKENS 16384 /* longest CACHE text (sequences joined by 0) */

/*
 * Retrieval from the context- and LLM preference-aware CACHE of Section
 * IV-B, which Alg. 1 searches before the datastores.  A CACHE's text is its
 * sequences joined by single 0 tokens; it is searched exactly like a store
 * (Section III-A), so the results equal those of fc_retrieve over one store
 * holding that text: the same match length, range_lo (the suffix-array index
 * of the first occurrence within the text), range_cnt, taken = min(k, cnt),
 * strided selection beyond k, and continuations in suffix order (cont_src =
 * 0).  No suffix array is needed: one workgroup per query holds the text in
 * LDS.
 *
 * texts [n_texts][stride] : CACHE texts, row r holding text_len[r] tokens
 *                           (clamped to [0, stride]); 1 <= stride <=
 *                           FC_MAX_CACHE_TOKENS.
 * text_row [B]            : the text query b searches (NULL: text b); a row
 *                           outside [0, n_texts) reads as an empty text.
 * ctx, B, L, p            : as fc_retrieve.
 * outputs                 : as fc_retrieve with S = 1 (match_n, range_lo,
 *                           range_cnt, taken [rows][1]; slots [rows][k]),
 *                           including the optional row map rows/n_rows.
 * The LDS needed is fc_cache_lds_bytes(stride) (96 KB at the maximum);
 * FC_ERR_UNSUPPORTED when the device has less.
 */
size_t fc_cache_lds_bytes(int64_t stride);
fc_status fc_cache_retrieve(const uint16_t* texts, int64_t stride, int32_t n_texts, const int32_t* text_len,
                            const int32_t* text_row, const uint16_t* ctx, int32_t B, int32_t L, fc_retrieve_params p,
                            int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt, int32_t* taken,
                            uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len, uint16_t* cont_tok,
                            const int32_t* rows, int32_t n_rows, hipStream_t stream);

/*
 * Batched CACHE update (Section IV-B: verified retrieved sequences and the
 * LLM's output are added after each step).  Segment i copies src_len[i]
 * tokens from src_tok + src_off[i] into text row dst_row[i] at offset
 * dst_off[i] and sets text_len[dst_row[i]] = new_len[i] (clamped to [0,
 * stride]); the caller lays out the appended sequences with their 0
 * separators.  Segments of one row must not overlap; a row outside [0,
 * n_texts) is skipped and tokens past the row's end are not written.  All
 * arrays are device memory.
 */
fc_status fc_cache_write(uint16_t* texts, int64_t stride, int32_t n_texts, int32_t* text_len, int32_t n_seg,
                         const int32_t* dst_row, const int32_t* dst_off, const int32_t* new_len,
                         const int64_t* src_off, const int32_t* src_len, const uint16_t* src_tok,
                         hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Draft tree                                                                */
/* ------------------------------------------------------------------------ */

typedef struct fc_tree_params {
  int32_t c;                       /* kept nodes (draft tokens), 1..255 (paper: 64) */
  uint32_t alpha[FC_MAX_SOURCES];  /* weight of one occurrence per store (paper: alpha = beta = 1) */
} fc_tree_params;

/*
 * Frequency-weighted draft trie pruned to c nodes (Section IV-D, eq. (3));
 * tree-attention mask and position ids (Section IV-D, eq. (4)).
 *
 * Inputs are fc_retrieve's outputs: taken [B][S], cont_len [B][k],
 * cont_tok [B][k][m], and ctx [B][L] for the root token ctx[L-1].
 * Precondition: within each store's slots the continuations are in
 * lexicographic order (a prefix first), as fc_retrieve produces them; a query
 * that violates it gets num_nodes = -1 and padding rows.
 * Every non-empty continuation enters a trie; node weight = sum of alpha[s]
 * over the continuations through the node.  The c highest nodes are kept,
 * ranked by weight, ties by path (token by token, a prefix first); this set
 * is closed under ancestors.  Rows: 0 is the root (token ctx[L-1], parent -1,
 * weight = sum of alpha over non-empty continuations, position 0), then the
 * kept nodes in preorder with children in token order.
 * num_nodes [B]           : 1 + kept nodes.
 * node_tok, parent [B][c+1], weight [B][c+1] (uint32), pos_ids [B][c+1]
 *                         : token, parent row, weight, depth of each row.
 * mask [B][c+1][c+1]      : 1 where column j is row i or an ancestor of i
 *                           (root included), else 0.
 * Rows past num_nodes: token 0, parent -1, weight 0, position 0, mask 0.
 * rows [B], n_rows       : optional row map: query b reads row rows[b] of
 *                           taken, cont_len and cont_tok (n_rows rows each);
 *                           its outputs stay at b.  A row outside
 *                           [0, n_rows) gives num_nodes = -1.  NULL: row b.
 * ws, ws_bytes           : workspace of at least fc_build_tree_workspace_bytes(B)
 *                           (the batch split into light and heavy queries).
 * Limits: S <= FC_MAX_SOURCES, k <= 65535, alpha[s]*k < 2^32, and the
 * per-query working set (about k*(2m+9) bytes) must fit one workgroup's LDS
 * (FC_ERR_UNSUPPORTED).
 */
size_t fc_build_tree_workspace_bytes(int32_t B);
fc_status fc_build_tree(const int32_t* taken, const uint8_t* cont_len, const uint16_t* cont_tok,
                        const uint16_t* ctx, int32_t B, int32_t L, int32_t S, int32_t k, int32_t m, fc_tree_params t,
                        int32_t* num_nodes, int32_t* node_tok, int32_t* parent, uint32_t* weight, int32_t* pos_ids,
                        int32_t* mask, const int32_t* rows, int32_t n_rows, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Acceptance                                                                */
/* ------------------------------------------------------------------------ */

/*
 * Greedy acceptance (Section IV-D: every correct draft token from the start
 * is accepted, everything after the first error rejected).
 * target [B][c+1]: the target model's next token after each tree row, -1
 * when there is none.  From the root, step to the child whose token equals
 * the current row's target while one exists.  With u the row reached:
 * accept_len [B]    : depth(u) + 1 (the path plus target[u]), or depth(u)
 *                     when target[u] is -1.
 * accept_tok [B][m+1]: the path tokens then target[u]; -1 past accept_len.
 * last_node [B]     : u.
 * The tree arrays are fc_build_tree's outputs; a query with num_nodes < 1 is
 * treated as a bare root.
 */
fc_status fc_verify_accept(const int32_t* num_nodes, const int32_t* node_tok, const int32_t* parent,
                           const int32_t* pos_ids, const int32_t* target, int32_t B, int32_t c, int32_t m,
                           int32_t* accept_len, int32_t* accept_tok, int32_t* last_node, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Tree attention (verification of the draft tree)                           */
/* ------------------------------------------------------------------------ */

#define FC_TREE_ATTN_HEAD_DIM 128 /* head dimension the library supports */

/*
 * The attention step of the target model's forward pass over a draft tree
 * (Section IV-D, eq. (4): one pass verifies every draft sequence, each row
 * attending to its ancestors through the tree mask, at the positions the
 * position ids give).  Row i of tree b sits at position prefix_len[b] +
 * pos_ids[b][i] (the root, depth 0, right after the cached prefix) and
 * attends to the prefix_len[b] cached tokens and to the tree rows j with
 * mask[b][i][j] = 1 (fc_build_tree's mask, pos_ids and num_nodes).  Queries
 * and the tree's keys are rotated by their positions (rotary embedding,
 * rotate-half form: the pair (d, d + D/2) turns by position *
 * rope_base^(-2d/D)); cached keys are stored already rotated.  Scores are
 * q.k / sqrt(D), softmax in fp32; out = softmax-weighted sum of values.
 * Rows at or past num_nodes[b] (and every row of a tree with num_nodes < 1)
 * are 0.  Query head h reads key/value head h / (H / Hkv).
 *
 * q [B][R][H][D], k_tree, v_tree [B][R][Hkv][D], k_cache, v_cache
 * [B][Pmax][Hkv][D]: bf16 bit patterns as uint16, 16-byte aligned;
 * prefix_len, num_nodes [B] and pos_ids [B][R], mask [B][R][R]: int32
 * (device lengths are clamped to [0, Pmax] and [0, R]); out [B][R][H][D]
 * fp32, 16-byte aligned.  D must be FC_TREE_ATTN_HEAD_DIM
 * (FC_ERR_UNSUPPORTED otherwise); 1 <= R <= FC_MAX_TREE_ROWS, H % Hkv == 0,
 * rope_base > 1.  The products run on bf16 matrix cores: rotated queries
 * and keys and the softmax weights are rounded to bf16, accumulations are
 * fp32.
 */
fc_status fc_tree_attention(const uint16_t* q, const uint16_t* k_tree, const uint16_t* v_tree,
                            const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* prefix_len,
                            const int32_t* num_nodes, const int32_t* mask, const int32_t* pos_ids, int32_t B,
                            int32_t R, int32_t H, int32_t Hkv, int32_t D, int32_t Pmax, float rope_base, float* out,
                            hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Decode-trace replay                                                       */
/* ------------------------------------------------------------------------ */

/*
 * Stand-in for the target model when replaying a known token stream (the
 * accepted length per forward step is the paper's average acceptance length
 * metric, Section V-C eq. (7)): after the path to tree row i the model would
 * produce the true token at position start[b] + pos_ids[b][i].
 * truth  : stream s starts at truth + s*truth_stride and has truth_len tokens.
 * seq [B] : stream of query b (NULL: stream b); start [B]: position of the
 *           token after query b's context in its stream.
 * target [B][c+1] : truth[seq[b]][start[b] + pos_ids[b][i]] for rows
 *                   i < num_nodes[b] whose position is below truth_len,
 *                   else -1.
 */
fc_status fc_targets_from_truth(const uint16_t* truth, int32_t truth_len, int64_t truth_stride, const int32_t* seq,
                                const int32_t* start, const int32_t* num_nodes, const int32_t* pos_ids, int32_t B,
                                int32_t c, int32_t* target, hipStream_t stream);

/*
 * Device-resident replay engine: the whole decode-trace replay above (the
 * average acceptance length of Section V-C, eq. (7)) with every per-step
 * decision on the GPU.  Each step, for every stream b with pos[b] <
 * truth_len: its context truth[b][pos[b]-ctx_len .. pos[b]) is looked up in
 * an LRU of `lru` recent retrievals keyed by the exact context (a hit
 * becomes most recent; a miss takes the next free slot, or the least
 * recently used one when all are taken, and is retrieved into it); the
 * draft tree is built from the slot (fc_build_tree), the true tokens are
 * its targets (as fc_targets_from_truth gives them), acceptance is greedy
 * (as fc_verify_accept; both in one pass here, into accept_len, accept_tok
 * and last_node) and pos[b] advances by the accepted length.  A step is a
 * fixed chain of launches on `stream` with no host round trip.
 *
 * All pointers are device memory owned by the caller:
 *   pos, lru_count, hits, lookups, rows_retrieve, rows_tree [n_streams];
 *   lru_key [n_streams][lru][ctx_len]; lru_used [n_streams][lru];
 *   ctx [n_streams][ctx_len]; live [2]: live[s & 1] counts the streams
 *   still live after step s; history [max_steps][n_streams]: the accepted length of each
 *   stream at each step, -1 once the stream is finished;
 *   retrieval outputs (fc_retrieve's, with n_streams * lru rows: row
 *   b * lru + slot is stream b's slot) and workspace for a batch of
 *   n_streams; tree outputs and acceptance outputs for n_streams (`target`
 *   is not used and may be NULL).
 * Limits: 1 <= ctx_len <= 64 (also fc_retrieve's n_max <= ctx_len is the
 * caller's choice), 1 <= lru <= 64, truth_stride >= truth_len.
 *
 * Optionally the CACHE of Section IV-B with Alg. 1's cache branch
 * (cache_l >= 0) and Alg. 1's retrieval-timing control (missing != 0:
 * contexts whose datastore retrieval found nothing are not retrieved again;
 * skip_tok >= 0: a context ending with skip_tok is retrieved only when the
 * step's draw skip_draws[step][b] is below skip_thr).  Per step, for a live
 * stream whose CACHE holds at least cache_l sequences the context is first
 * searched in the CACHE's text (fc_cache_retrieve, results in the c_*
 * arrays, row b); a non-empty result is "served": it is copied into the
 * stream's own retrieval row n_streams * lru + 1 + b as the first store's
 * slots (the other stores' counts 0), its tree is built from it alone and
 * the datastores are not touched.  A served tree's weights are therefore
 * tp.alpha[0] per slot instead of 1 (the same nodes and order; tp.alpha[0]
 * must not be 0 with the CACHE on).
 * Otherwise the missing table and then the skip gate may skip the context
 * (its tree is the bare root read from retrieval row n_streams * lru, which
 * fc_replay_init empties), else the LRU step above runs and, with the
 * missing table on, a context whose result is empty is added to it.  After
 * acceptance the CACHE gets the context plus the accepted draft tokens
 * (when the draft contributed any) and every completed chunk of
 * cache_every output tokens; a sequence longer than cache_cap keeps its
 * last cache_cap tokens, and the oldest sequences go when the text (the
 * sequences joined by 0 tokens) would outgrow cache_cap.
 * Extra device arrays (caller-owned): ctext [n_streams][cache_cap], clen,
 * seq_head, seq_count, chunks, served, rows_cache, state [n_streams],
 * seq_len [n_streams][max_seqs] (max_seqs >= (cache_cap + 1) / 2 + 1); CACHE
 * retrieval outputs (S = 1) for n_streams (c_num_nodes .. c_mask are not
 * used and may be NULL); miss_key [n_streams][miss_cap][ctx_len], miss_used
 * [n_streams][miss_cap] (miss_cap a power of two above max_steps), m_skips,
 * g_skips [n_streams]; skip_draws [max_steps][n_streams].  With the
 * control on, the retrieval outputs need n_streams * lru + 1 rows; with the
 * CACHE on, n_streams * lru + 1 + n_streams.
 *
 * fc_replay_init sets pos = ctx_len, empties every LRU, CACHE and missing
 * table and zeroes the counters.  fc_replay_run runs steps first_step ..
 * first_step + n_steps - 1 (their history rows), first_step + n_steps <=
 * max_steps; read live[(last step) & 1] between calls to stop once it is
 * 0.  Errors of the calls it makes are returned as they come.
 */
typedef struct fc_replay {
  const uint16_t* truth;
  int64_t truth_stride;
  int32_t truth_len;
  int32_t n_streams;
  int32_t ctx_len;
  int32_t lru;
  int32_t max_steps;
  fc_retrieve_params rp;
  fc_tree_params tp;
  int32_t* pos;
  uint16_t* lru_key;
  int32_t* lru_used;
  int32_t* lru_count;
  int32_t* hits;
  int32_t* lookups;
  uint16_t* ctx;
  int32_t* rows_retrieve;
  int32_t* rows_tree;
  int32_t* live;
  int32_t* history;
  int32_t* match_n;
  uint32_t* range_lo;
  uint32_t* range_cnt;
  int32_t* taken;
  uint32_t* cont_pos;
  uint8_t* cont_src;
  uint8_t* cont_len;
  uint16_t* cont_tok;
  void* retrieve_ws;
  size_t retrieve_ws_bytes;
  int32_t* num_nodes;
  int32_t* node_tok;
  int32_t* parent;
  uint32_t* weight;
  int32_t* pos_ids;
  int32_t* mask;
  void* tree_ws;
  size_t tree_ws_bytes;
  int32_t* target;
  int32_t* accept_len;
  int32_t* accept_tok;
  int32_t* last_node;
  /* CACHE (cache_l < 0: off) */
  int32_t cache_l;
  int32_t cache_every;
  int32_t cache_cap;
  int32_t max_seqs;
  uint16_t* ctext;
  int32_t* clen;
  int32_t* seq_len;
  int32_t* seq_head;
  int32_t* seq_count;
  int32_t* chunks;
  int32_t* served;
  int32_t* rows_cache;
  int32_t* state;
  int32_t* c_match_n;
  uint32_t* c_range_lo;
  uint32_t* c_range_cnt;
  int32_t* c_taken;
  uint32_t* c_cont_pos;
  uint8_t* c_cont_src;
  uint8_t* c_cont_len;
  uint16_t* c_cont_tok;
  int32_t* c_num_nodes; /* not used (may be NULL) */
  int32_t* c_node_tok;
  int32_t* c_parent;
  uint32_t* c_weight;
  int32_t* c_pos_ids;
  int32_t* c_mask;
  /* Alg. 1's retrieval-timing control */
  int32_t missing;
  int32_t miss_cap;
  uint16_t* miss_key;
  uint8_t* miss_used;
  int32_t* m_skips;
  int32_t skip_tok;
  uint32_t skip_thr;
  const int32_t* skip_draws;
  int32_t* g_skips;
} fc_replay;

fc_status fc_replay_init(fc_replay* r, hipStream_t stream);
fc_status fc_replay_run(const fc_store* stores, int32_t S, const fc_replay* r, int32_t first_step, int32_t n_steps,
                        hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FASTCODER_H */
