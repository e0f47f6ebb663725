// Longest-suffix retrieval with continuation gather on gfx950 (fc_retrieve).
//
// For every query and store the method looks for the longest suffix of the
// context, from n_max tokens down, that occurs in the datastore, and returns
// what follows each occurrence (Section III-A; the repository store and the
// common store are searched side by side, Section IV-A and Section IV-C).
//
// k_search: one workgroup per query.  Every (store, n, bound) search task -
// 2 stores x 15 lengths x {lower, upper} = 60 at the paper's n_max = 16,
// n_min = 2 - gets a group of G lanes (G = 4 in 256 threads), so every
// candidate length is searched at once.  Each search starts from the store's
// two-token table when it has one (one table read replaces the top ~25
// levels of the search on a 1B-token store) or else from its first-token
// bucket.  With the store's inline-prefix records the group reads the records
// at 2G - 1 evenly spaced pivots of its range per round trip (a 2G-ary
// search: log_2G of the range in dependent round trips), comparing only the
// tokens the table does not already fix; without them each lane runs a
// binary search over the suffix-array entries and the text.  The workgroup
// then keeps, per store, the longest n whose range is non-empty and fills
// the k slots in store priority order.
//
// k_gather: the kept slots of the whole batch are numbered consecutively and
// cut into one contiguous piece per workgroup of a grid that is resident at
// once; every workgroup numbers them itself (an exclusive scan of the
// queries' kept counts into LDS), or, past 4,095 queries, reads the numbering
// k_offsets wrote.  A slot maps to its store and range offset (strided
// floor(i*cnt/b) when the range exceeds the store's budget b), reads the
// record (or the suffix-array entry and then the text) and copies up to m
// continuation tokens, cut before a 0 and at the end of the store.  Strided
// samples of large ranges put every slot on a cache line of its own, so the
// gather runs at the rate of scattered line reads, not of HBM streaming.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kSearchThreads = 256;
constexpr int kSearchWide = 512;      // threads per query for batches of at most kSearchWideMaxB
constexpr int kSearchWideMaxB = 256;
constexpr int kSearchWidest = 1024;   // and for batches of at most kSearchWidestMaxB
constexpr int kSearchWidestMaxB = 128;
constexpr int kGatherThreads = 256;
constexpr int kScanThreads = 1024;
constexpr int kOffsetsInLds = 4096;
// gather grids that are resident at once: five workgroups per CU for rows of
// up to 10 tokens (90 VGPRs), four for up to 16 (108 VGPRs)
constexpr int kGatherBlocks10 = 1280;
constexpr int kGatherBlocks16 = 1024;

struct StoreArgs {
  const uint16_t* tok[FC_MAX_SOURCES];
  const uint32_t* sa[FC_MAX_SOURCES];
  const uint32_t* bucket[FC_MAX_SOURCES];
  const uint32_t* pair[FC_MAX_SOURCES];
  const uint4* rec[FC_MAX_SOURCES];
  const uint4* top[FC_MAX_SOURCES];  // sample of every FC_TOP_STRIDE-th record's first 32 bytes, or null
  uint32_t n[FC_MAX_SOURCES];
  uint32_t pair_vocab[FC_MAX_SOURCES];
};

// Suffix j against pattern q[0..n), knowing tokens before `from` match: -1 below
// (a suffix that ends first is below), 0 starts with q, +1 above.  Tokens are
// fetched in two batches of independent loads (1..8, then 9..15 only when the
// first eight all match), so a probe costs one memory round trip in the
// common case instead of a chain of dependent loads.
__device__ __forceinline__ int cmp_suffix(const uint16_t* __restrict__ T, uint32_t N, uint32_t j,
                                          const uint16_t* q, int n, int from) {
  constexpr int kBatch = 8;
  uint16_t t[kBatch];
  for (int x0 = from; x0 < n; x0 += kBatch) {
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint64_t p = (uint64_t)j + (uint64_t)(x0 + u);
      t[u] = (x0 + u < n && p < N) ? T[p] : (uint16_t)0;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int x = x0 + u;
      if (x >= n) return 0;
      if ((uint64_t)j + (uint64_t)x >= N) return -1;
      const uint16_t b = q[x];
      if (t[u] != b) return t[u] < b ? -1 : 1;
    }
  }
  return 0;
}

// A pattern's tokens at offsets 2..15 packed two per word like a record's
// token words (offset 2 + 2x in the low half of word x), each word rotated
// by 16 bits so that one unsigned compare orders two tokens
// lexicographically; positions at or past n are masked out on both sides.
constexpr int kSearchWords = (FC_MAX_NMAX - 1) / 2;  // token words of offsets 2..15
constexpr int kRecQuads = FC_RECORD_BYTES / 16;     // 16-byte pieces per record
static_assert(2 + 2 * kSearchWords <= FC_RECORD_TOKENS + 2 && kSearchWords == 7, "search words");

struct RecQuery {
  uint32_t rot[kSearchWords];
  uint32_t mask[kSearchWords];
};

__device__ __forceinline__ uint32_t rot16(uint32_t x) { return __builtin_amdgcn_alignbit(x, x, 16); }

__device__ __forceinline__ RecQuery rec_query(const uint16_t* q, int n) {
  RecQuery r;
#pragma unroll
  for (int x = 0; x < kSearchWords; ++x) {
    const int o = 2 + 2 * x;
    const uint32_t a = o < n ? q[o] : 0u;
    const uint32_t b = o + 1 < n ? q[o + 1] : 0u;
    r.rot[x] = rot16(a | (b << 16));
    r.mask[x] = (o < n ? 0xFFFFu : 0u) | (o + 1 < n ? 0xFFFF0000u : 0u);
  }
  return r;
}

// A record's first 32 bytes (offsets 2..15 of its suffix) against the
// pattern: -1 below, 0 starts with it, +1 above.  The first differing word decides.
__device__ __forceinline__ int rec_cmp(const uint4& h0, const uint4& h1, const RecQuery& r) {
  const uint32_t t[kSearchWords] = {h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
  int res = 0;
#pragma unroll
  for (int x = kSearchWords - 1; x >= 0; --x) {
    const uint32_t u = rot16(t[x] & r.mask[x]);
    res = u != r.rot[x] ? (u < r.rot[x] ? -1 : 1) : res;
  }
  return res;
}

// Search of query b by the whole workgroup: s_lo / s_hi[s][n_max - n] get
// the bounds of every tried (store, n) that can still matter; untried
// entries stay 0.  Only the longest n with an occurrence counts per store,
// so once both bounds of some n are known and enclose a non-empty range
// (s_best[s] = n), the tasks of that store's shorter lengths stop at their
// next round trip: those are the short suffixes whose two-token ranges are
// the largest, and the slowest searches.  Their entries are left partial;
// the keep step never looks below the longest non-empty n.
__device__ __forceinline__ void search_query(const StoreArgs& st, int S, const uint16_t* __restrict__ ctx, int b,
                                             int L, int n_max, int n_min, int G, int log2_2g, uint16_t* s_q,
                                             uint32_t (*s_lo)[FC_MAX_NMAX], uint32_t (*s_hi)[FC_MAX_NMAX],
                                             int* s_nhi, uint32_t (*s_done)[FC_MAX_NMAX], int* s_best) {
  const int tid = (int)threadIdx.x;
  const int lane = fc::lane_id();
  const int nq = L < FC_MAX_NMAX ? L : FC_MAX_NMAX;
  if (tid < nq) s_q[FC_MAX_NMAX - nq + tid] = ctx[(int64_t)b * L + (L - nq + tid)];
  if (tid < FC_MAX_SOURCES * FC_MAX_NMAX) {
    (&s_lo[0][0])[tid] = 0;
    (&s_hi[0][0])[tid] = 0;
    (&s_done[0][0])[tid] = 0;
  }
  if (tid < FC_MAX_SOURCES) s_best[tid] = 0;
  __syncthreads();
  if (tid == 0) {
    int tail = 0;
    while (tail < nq && s_q[FC_MAX_NMAX - 1 - tail] != 0) ++tail;
    const int h = n_max < L ? n_max : L;
    *s_nhi = tail < h ? tail : h;
  }
  __syncthreads();

  const int NN = n_max - n_min + 1;
  const int tasks = S * NN * 2;
  const int task = tid / G;
  const int gl = tid - task * G;
  const int n_hi = *s_nhi;
  int s = 0, ni = 0, upper = 0, n = 0;
  bool act = task < tasks;
  if (act) {
    s = task / (2 * NN);
    const int rem = task - s * 2 * NN;
    ni = rem >> 1;
    upper = rem & 1;
    n = n_max - ni;
    act = n <= n_hi && n >= n_min;
  }
  uint32_t lo = 0, hi = 0;
  int from = 1;
  const uint16_t* q = &s_q[FC_MAX_NMAX - (act ? n : 1)];
  if (act && st.n[s] > 0) {
    const uint32_t V = st.pair_vocab[s];
    if (n >= 2 && st.pair[s] != nullptr && q[0] < V && q[1] < V) {
      const uint64_t idx = (uint64_t)q[0] * (V + 1) + q[1] + 1;
      lo = st.pair[s][idx];
      hi = st.pair[s][idx + 1];
      from = 2;
    } else if (n >= 2 && st.pair[s] != nullptr) {
      hi = lo = 0;  // a token >= V cannot occur in the store
    } else {
      lo = st.bucket[s][q[0]];
      hi = st.bucket[s][q[0] + 1];
    }
  }
  const bool kary = act && from < n && lo < hi && from == 2 && st.rec[s] != nullptr;
  if (act && !kary) {
    if (from < n && lo < hi) {
      const uint16_t* T = st.tok[s];
      const uint32_t* SA = st.sa[s];
      const uint32_t N = st.n[s];
      uint32_t mid = lo + ((hi - lo) >> 1);
      uint32_t j = SA[mid];
      for (;;) {
        const uint32_t lmid = lo + ((mid - lo) >> 1);
        const uint32_t rmid = (mid + 1) + ((hi - mid - 1) >> 1);
        const uint32_t jl = lo < mid ? SA[lmid] : 0u;
        const uint32_t jr = mid + 1 < hi ? SA[rmid] : 0u;
        const int c = cmp_suffix(T, N, j, q, n, from);
        if (upper ? (c <= 0) : (c < 0)) {
          lo = mid + 1;
          mid = rmid;
          j = jr;
        } else {
          hi = mid;
          mid = lmid;
          j = jl;
        }
        if (lo >= hi) break;
      }
    } else if (upper) {
      lo = hi;  // range already final: its end is the upper bound
    }
  }
  // a task's final bound: recorded, and the second bound of a (store, n)
  // to arrive raises the store's best n when the range is non-empty
  auto finish = [&](uint32_t bound) {
    if (gl != 0) return;
    if (upper) s_hi[s][ni] = bound; else s_lo[s][ni] = bound;
    if (atomicAdd(&s_done[s][ni], 1u) == 1u) {
      const uint32_t a = *(volatile uint32_t*)&s_lo[s][ni];
      const uint32_t z = *(volatile uint32_t*)&s_hi[s][ni];
      if (z > a) atomicMax(&s_best[s], n);
    }
  };
  if (act && !kary) finish(lo);
  {
    const RecQuery rq = rec_query(q, act ? n : 2);
    const uint4* R = st.rec[s];
    const uint4* TP = st.top[s];
    const bool two = n > 8;  // tokens past offset 7 sit in the record's second quad
    const int gbase = lane - gl;
    const uint64_t gmask = G >= 64 ? ~0ull : ((1ull << G) - 1);
    const int P = 2 * G - 1;  // pivots per round trip
    bool searching = kary;
    // A range spanning two sample strides or more is first searched over the
    // sample: the positions t * FC_TOP_STRIDE in [lo, hi) are t in [ta, tb),
    // and the first t whose record is not below the bound brackets the bound
    // within one stride of records.
    uint32_t ta = 0, tb = 0;
    bool in_top = false;
    if (kary && TP != nullptr) {
      ta = (uint32_t)(((uint64_t)lo + FC_TOP_STRIDE - 1) / FC_TOP_STRIDE);
      tb = (uint32_t)(((uint64_t)hi + FC_TOP_STRIDE - 1) / FC_TOP_STRIDE);
      in_top = tb > ta + 1;
    }
    uint32_t clo = in_top ? ta : lo, chi = in_top ? tb : hi;  // the interval of the current phase
    while (fc::ballot(searching) != 0) {
      bool ca = false, cb = false;
      if (searching && n < *(volatile int*)&s_best[s]) searching = false;  // a longer n has occurrences
      if (searching) {
        const uint64_t span = chi - clo;
        const uint32_t pa = clo + (uint32_t)(((uint64_t)(2 * gl + 1) * span) >> log2_2g);
        const bool vb = 2 * gl + 2 <= P;
        const uint32_t pb = vb ? clo + (uint32_t)(((uint64_t)(2 * gl + 2) * span) >> log2_2g) : pa;
        const uint4* Qa = in_top ? TP + 2 * (uint64_t)pa : R + kRecQuads * (uint64_t)pa;
        const uint4* Qb = in_top ? TP + 2 * (uint64_t)pb : R + kRecQuads * (uint64_t)pb;
        const uint4 a0 = Qa[0];
        const uint4 b0 = Qb[0];
        uint4 a1 = make_uint4(0, 0, 0, 0), b1 = a1;
        if (two) {
          a1 = Qa[1];
          b1 = Qb[1];
        }
        const int c1 = rec_cmp(a0, a1, rq);
        const int c2 = rec_cmp(b0, b1, rq);
        ca = upper ? c1 <= 0 : c1 < 0;
        cb = vb && (upper ? c2 <= 0 : c2 < 0);
      }
      const uint64_t ba = fc::ballot(searching && ca);
      const uint64_t bb = fc::ballot(searching && cb);
      if (searching) {
        // the pivots before the bound form a prefix of the 2G - 1 pivots
        const int c = __popcll((ba >> gbase) & gmask) + __popcll((bb >> gbase) & gmask);
        const uint64_t span = chi - clo;
        const uint32_t plo = c > 0 ? clo + (uint32_t)(((uint64_t)c * span) >> log2_2g) + 1 : clo;
        const uint32_t phi = c < P ? clo + (uint32_t)(((uint64_t)(c + 1) * span) >> log2_2g) : chi;
        clo = plo;
        chi = phi;
        if (clo >= chi && in_top) {
          // sample t = clo is the first not below the bound (tb: none is):
          // the bound lies in ((t - 1) * stride, t * stride]
          const uint32_t t = clo;
          clo = t > ta ? (t - 1) * FC_TOP_STRIDE + 1 : lo;
          chi = t < tb ? t * FC_TOP_STRIDE : hi;
          in_top = false;
        }
        searching = clo < chi;
        if (!searching) finish(clo);
      }
    }
  }
  __syncthreads();
}

// One query per workgroup: the 2G-ary search of every (store, n, bound),
// then the kept ranges (the longest non-empty n per store, store priority
// order) written to the query's row.
template <int NT>
__global__ void __launch_bounds__(NT) k_search(StoreArgs st, int S, const uint16_t* __restrict__ ctx,
                                                           int L, int n_max, int n_min, int k, int G, int log2_2g,
                                                           const int32_t* __restrict__ rows, int n_rows,
                                                           int32_t* __restrict__ match_n,
                                                           uint32_t* __restrict__ range_lo,
                                                           uint32_t* __restrict__ range_cnt,
                                                           int32_t* __restrict__ taken) {
  __shared__ uint16_t s_q[FC_MAX_NMAX];
  __shared__ uint32_t s_lo[FC_MAX_SOURCES][FC_MAX_NMAX];
  __shared__ uint32_t s_hi[FC_MAX_SOURCES][FC_MAX_NMAX];
  __shared__ int s_nhi;
  __shared__ uint32_t s_done[FC_MAX_SOURCES][FC_MAX_NMAX];
  __shared__ int s_best[FC_MAX_SOURCES];
  const int b = (int)blockIdx.x;
  const int row = fc::map_row(rows, n_rows, b);
  if (row < 0) return;  // skipped query: the whole workgroup leaves
  const int tid = (int)threadIdx.x;
  const int lane = fc::lane_id();
  search_query(st, S, ctx, b, L, n_max, n_min, G, log2_2g, s_q, s_lo, s_hi, &s_nhi, s_done, s_best);
  if (tid < fc::kWave) {
    const int NN = n_max - n_min + 1;
    const int n_hi = s_nhi;
    bool ne = false;
    if (lane < S * NN) {
      const int u = lane / NN, x = lane - (lane / NN) * NN;
      const int nn = n_max - x;
      ne = nn <= n_hi && nn >= n_min && s_hi[u][x] > s_lo[u][x];
    }
    const uint64_t bal = fc::ballot(ne);
    if (lane < S) {
      // store `lane`: its longest non-empty n, then the budget left by the
      // stores before it
      int used = 0, mine = 0;
      int mn = 0;
      uint32_t rlo = 0, cnt = 0;
      for (int u = 0; u <= lane; ++u) {
        const uint32_t bits = (uint32_t)(bal >> (u * NN)) & ((1u << NN) - 1u);
        uint32_t c = 0;
        int x = 0;
        if (bits) {
          x = __builtin_ctz(bits);
          c = s_hi[u][x] - s_lo[u][x];
        }
        const int budget = k - used;
        const int tk = (int64_t)c < (int64_t)budget ? (int)c : budget;
        if (u == lane) {
          mine = tk;
          mn = bits ? n_max - x : 0;
          rlo = bits ? s_lo[u][x] : 0u;
          cnt = c;
        }
        used += tk;
      }
      const int64_t o = (int64_t)row * S + lane;
      match_n[o] = mn;
      range_lo[o] = rlo;
      range_cnt[o] = cnt;
      taken[o] = mine;
    }
  }
}

// Exclusive prefix of kept slots over the batch (one workgroup):
// offsets[b] = slots kept by queries before b; offsets[B] = total.
__global__ void __launch_bounds__(kScanThreads) k_offsets(const int32_t* __restrict__ taken, int B, int S,
                                                          const int32_t* __restrict__ rows, int n_rows,
                                                          uint32_t* __restrict__ offsets) {
  __shared__ uint32_t scratch[kScanThreads / fc::kWave + 1];
  const int per = (B + kScanThreads - 1) / kScanThreads;
  const int b0 = (int)threadIdx.x * per;
  const int b1 = b0 + per < B ? b0 + per : B;
  auto kept = [&](int b) -> uint32_t {
    const int r = fc::map_row(rows, n_rows, b);
    uint32_t t = 0;
    if (r >= 0)
      for (int s = 0; s < S; ++s) t += (uint32_t)taken[(int64_t)r * S + s];
    return t;
  };
  uint32_t sum = 0;
  for (int b = b0; b < b1; ++b) sum += kept(b);
  uint32_t total;
  uint32_t run = fc::block_excl_sum<uint32_t>(sum, scratch, &total);
  for (int b = b0; b < b1; ++b) {
    offsets[b] = run;
    run += kept(b);
  }
  if (threadIdx.x == 0) offsets[B] = total;
}

// floor(local * cnt / budget), the strided pick of a range larger than its
// budget: local < budget <= k < 2^31 and cnt < 2^32.  Below 2^53 the product
// is exact in a double and the double quotient lies within a small fraction
// of the true one, so its integer part is off by at most one, which one
// integer check corrects; larger products take the 64-bit division.
__device__ __forceinline__ uint64_t strided_pick(uint64_t local, uint64_t cnt, uint64_t budget) {
  const uint64_t prod = local * cnt;
  if (prod >= (1ull << 53)) return prod / budget;
  uint64_t q = (uint64_t)((double)prod / (double)budget);
  if (q * budget > prod) --q;
  else if ((q + 1) * budget <= prod) ++q;
  return q;
}

// MAXM tokens from MAXM/2 + 1 consecutive 32-bit words holding two tokens
// each (low half first), starting at the high half of the first word when
// `odd`; every load is issued before any is used.
template <int MAXM>
__device__ __forceinline__ void words_window(const uint32_t* __restrict__ W, int odd, uint16_t (&v)[MAXM]) {
  constexpr int kWords = MAXM / 2 + 1;
  uint32_t wd[kWords];
#pragma unroll
  for (int u = 0; u < kWords; ++u) wd[u] = W[u];
#pragma unroll
  for (int x = 0; x < MAXM; ++x) {
    const uint16_t even_v = (uint16_t)(wd[x >> 1] >> (16 * (x & 1)));
    const uint16_t odd_v = (uint16_t)(wd[(x + 1) >> 1] >> (16 * ((x + 1) & 1)));
    v[x] = odd ? odd_v : even_v;
  }
}

// Continuation tokens [start, start + MAXM) of one slot from the text: the
// words from the aligned word at or before start.  Tokens at or past N
// read as 0.
template <int MAXM>
__device__ __forceinline__ void load_window(const uint16_t* __restrict__ T, uint64_t N, uint64_t start,
                                           uint16_t (&v)[MAXM]) {
  constexpr int kWords = MAXM / 2 + 1;
  const uint64_t w0 = start >> 1;
  if (2 * (w0 + kWords) <= N) {
    words_window<MAXM>((const uint32_t*)T + w0, (int)(start & 1), v);
  } else {
#pragma unroll
    for (int x = 0; x < MAXM; ++x) v[x] = (start + x < N) ? T[start + x] : (uint16_t)0;
  }
}

// Kept slots of the whole batch as one flat range (slot g belongs to the
// query b with offsets[b] <= g < offsets[b+1]), cut into one contiguous piece
// per workgroup of a grid that fits on the GPU at once.  Every workgroup
// numbers the slots itself: the queries' kept counts are loaded all at once
// (one memory round trip) and scanned in LDS; past 4,095 queries it reads
// the numbering k_offsets wrote.  The piece's queries (a contiguous run,
// usually a handful) have their per-store fields copied into LDS once, so a
// slot costs an LDS lookup and then one record read.  Each thread takes
// kGatherUnroll slots at a time with all their reads issued before any is
// used; consecutive lanes take consecutive slots, so a kept range is read at
// consecutive records and the outputs are written contiguously.  The window
// is cut at the first 0 in registers and written two tokens per 32-bit store
// when rows are 4-byte aligned.
constexpr int kGatherUnroll = 4;
constexpr int kMetaQueries = 64;  // queries of a piece whose fields fit in LDS
constexpr int kMaxPerThread = kOffsetsInLds / kGatherThreads;

template <int MAXM>
__global__ void __launch_bounds__(kGatherThreads) k_gather(StoreArgs st, int S, int B, int k, int m,
                                                           const int32_t* __restrict__ match_n,
                                                           const uint32_t* __restrict__ range_lo,
                                                           const uint32_t* __restrict__ range_cnt,
                                                           const int32_t* __restrict__ taken,
                                                           const uint32_t* __restrict__ offsets, int words,
                                                           int out_words, const int32_t* __restrict__ rows,
                                                           int n_rows, uint32_t* __restrict__ cont_pos,
                                                           uint8_t* __restrict__ cont_src,
                                                           uint8_t* __restrict__ cont_len,
                                                           uint16_t* __restrict__ cont_tok) {
  __shared__ uint32_t s_off[kOffsetsInLds];
  __shared__ uint32_t s_scan[kGatherThreads / fc::kWave + 1];
  __shared__ int s_qab[2];  // the queries owning the piece's first and last slots
  __shared__ int32_t s_taken[kMetaQueries][FC_MAX_SOURCES];
  __shared__ uint32_t s_cnt[kMetaQueries][FC_MAX_SOURCES], s_lo[kMetaQueries][FC_MAX_SOURCES];
  __shared__ int32_t s_n[kMetaQueries][FC_MAX_SOURCES];
  __shared__ int s_row[kMetaQueries];
  const int tid = (int)threadIdx.x;
  const bool in_lds = B + 1 <= kOffsetsInLds;
  if (in_lds) {
    // kept slots of queries tid, tid + 256, ...: every load issued at once
    uint32_t t[kMaxPerThread];
#pragma unroll
    for (int i = 0; i < kMaxPerThread; ++i) {
      const int q = tid + i * kGatherThreads;
      t[i] = 0;
      if (q < B) {
        const int r = fc::map_row(rows, n_rows, q);
        if (r >= 0) {
#pragma unroll
          for (int u = 0; u < FC_MAX_SOURCES; ++u)
            if (u < S) t[i] += (uint32_t)taken[(int64_t)r * S + u];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kMaxPerThread; ++i) {
      const int q = tid + i * kGatherThreads;
      if (q < B) s_off[q] = t[i];
    }
    __syncthreads();
    // exclusive scan: each thread a run of consecutive queries
    const int per = (B + kGatherThreads - 1) / kGatherThreads;
    const int b0 = tid * per;
    const int b1 = b0 + per < B ? b0 + per : B;
    uint32_t sum = 0;
    for (int q = b0; q < b1; ++q) sum += s_off[q];
    uint32_t all;
    uint32_t run = fc::block_excl_sum<uint32_t>(sum, s_scan, &all);
    // this workgroup's piece, and the queries owning its first and last
    // slots, found while the offsets are written (no search afterwards)
    const uint32_t pa = (uint32_t)(((uint64_t)all * blockIdx.x) / gridDim.x);
    const uint32_t pe = (uint32_t)(((uint64_t)all * (blockIdx.x + 1)) / gridDim.x);
    for (int q = b0; q < b1; ++q) {
      const uint32_t x = s_off[q];
      s_off[q] = run;
      if (pa < pe && run <= pa && pa < run + x) s_qab[0] = q;
      if (pa < pe && run <= pe - 1 && pe - 1 < run + x) s_qab[1] = q;
      run += x;
    }
    if (tid == 0) s_off[B] = all;
  }
  __syncthreads();
  const uint32_t* off_tab = in_lds ? s_off : offsets;
  const uint32_t total = off_tab[B];
  const uint32_t a = (uint32_t)(((uint64_t)total * blockIdx.x) / gridDim.x);
  const uint32_t e = (uint32_t)(((uint64_t)total * (blockIdx.x + 1)) / gridDim.x);
  if (a >= e) return;
  // last query with offsets <= g, searched in [lo, hi)
  auto owner = [&](uint32_t g, int lo, int hi) {
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off_tab[mid] <= g) lo = mid; else hi = mid;
    }
    return lo;
  };
  const int qa = in_lds ? s_qab[0] : owner(a, 0, B);
  const int qb = in_lds ? s_qab[1] : owner(e - 1, qa, B);
  const int nq = qb - qa + 1;
  const bool meta_lds = nq <= kMetaQueries;
  if (meta_lds && tid < nq * FC_MAX_SOURCES) {
    const int x = tid / FC_MAX_SOURCES, u = tid - x * FC_MAX_SOURCES;
    const int r = fc::map_row(rows, n_rows, qa + x);  // >= 0 for a query that owns slots
    if (u == 0) s_row[x] = r;
    if (u < S && r >= 0) {
      const int64_t o = (int64_t)r * S + u;
      s_taken[x][u] = taken[o];
      s_cnt[x][u] = range_cnt[o];
      s_lo[x][u] = range_lo[o];
      s_n[x][u] = match_n[o];
    } else {
      s_taken[x][u] = 0;
      s_cnt[x][u] = 0;
      s_lo[x][u] = 0;
      s_n[x][u] = 0;
    }
  }
  __syncthreads();

  constexpr int kWords = MAXM / 2 + 1;
  for (uint32_t g0 = a + (uint32_t)tid; g0 < e; g0 += kGatherThreads * kGatherUnroll) {
    uint32_t wd[kGatherUnroll][kWords];
    uint32_t jv[kGatherUnroll];
    int sv[kGatherUnroll], nv[kGatherUnroll], rowv[kGatherUnroll], iv[kGatherUnroll];
    bool in_rec[kGatherUnroll];
#pragma unroll
    for (int v = 0; v < kGatherUnroll; ++v) {
      const uint32_t g = g0 + (uint32_t)(v * kGatherThreads);
      sv[v] = 0;
      nv[v] = 0;
      rowv[v] = 0;
      iv[v] = 0;
      jv[v] = 0;
      in_rec[v] = false;
      if (g < e) {
        const int q = owner(g, qa, qb + 1);
        const int i = (int)(g - off_tab[q]);
        int tk[FC_MAX_SOURCES], nn[FC_MAX_SOURCES];
        uint32_t ct[FC_MAX_SOURCES], lw[FC_MAX_SOURCES];
        int row;
        if (meta_lds) {
          const int x = q - qa;
          row = s_row[x];
#pragma unroll
          for (int u = 0; u < FC_MAX_SOURCES; ++u) {
            tk[u] = s_taken[x][u];
            ct[u] = s_cnt[x][u];
            lw[u] = s_lo[x][u];
            nn[u] = s_n[x][u];
          }
        } else {
          row = fc::map_row(rows, n_rows, q);
#pragma unroll
          for (int u = 0; u < FC_MAX_SOURCES; ++u) {
            const int64_t o = (int64_t)row * S + u;
            tk[u] = u < S ? taken[o] : 0;
            ct[u] = u < S ? range_cnt[o] : 0u;
            lw[u] = u < S ? range_lo[o] : 0u;
            nn[u] = u < S ? match_n[o] : 0;
          }
        }
        // the slot's store: stores before it fill the first slots
        int s = 0;
        int before = 0;
        uint64_t cnt = ct[0], rlo = lw[0];
        int n = nn[0];
#pragma unroll
        for (int u = 1; u < FC_MAX_SOURCES; ++u) {
          const int nb = before + tk[u - 1];
          if (u < S && s == u - 1 && i >= nb) {
            s = u;
            before = nb;
            cnt = ct[u];
            rlo = lw[u];
            n = nn[u];
          }
        }
        const uint64_t budget = (uint64_t)(k - before);
        const uint64_t local = (uint64_t)(i - before);
        const uint64_t idx = rlo + (cnt > budget ? strided_pick(local, cnt, budget) : local);
        sv[v] = s;
        nv[v] = n;
        rowv[v] = row;
        iv[v] = i;
        // the window's words (token n - 2 onward) inside the record: no text
        // read.  The record is read as 16-byte quads - quad 0 (sa entry and
        // tokens 2..7) and only the later quads the window reaches - so a
        // slot costs two to four vector loads instead of one per word.
        const int t0 = n - 2;
        if (st.rec[s] != nullptr && t0 >= 0 && (t0 >> 1) + MAXM / 2 <= FC_RECORD_TOKENS / 2 - 1) {
          const uint4* Q = st.rec[s] + kRecQuads * idx;
          const int wf = 1 + (t0 >> 1);  // first window word
          const int wl = wf + kWords - 1;  // last window word
          const uint4 q0 = Q[0];
          uint4 q1 = make_uint4(0, 0, 0, 0), q2 = q1, q3 = q1;
          if (wf <= 7) q1 = Q[1];
          if (wf <= 11 && wl >= 8) q2 = Q[2];
          if (wl >= 12) q3 = Q[3];
          in_rec[v] = true;
          jv[v] = q0.x;
          uint32_t w[16] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                            q2.x, q2.y, q2.z, q2.w, q3.x, q3.y, q3.z, q3.w};
          // words wf.. by a barrel shift of the 16 words (wf < 16)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const bool on = (wf >> b) & 1;
#pragma unroll
            for (int x = 0; x < 16; ++x) {
              const int y = x + (1 << b);
              w[x] = on ? (y < 16 ? w[y] : 0u) : w[x];
            }
          }
#pragma unroll
          for (int x = 0; x < kWords; ++x) wd[v][x] = w[x];
        } else {
          jv[v] = st.sa[s][idx];
        }
      }
    }
#pragma unroll
    for (int v = 0; v < kGatherUnroll; ++v) {
      const uint32_t g = g0 + (uint32_t)(v * kGatherThreads);
      if (g >= e) continue;
      const int s = sv[v];
      const int n = nv[v];
      const uint64_t start = (uint64_t)jv[v] + (uint64_t)n;
      // the window as MAXM / 2 words of two tokens (token 2y in the low
      // half of word y): from a record, each word is one funnel shift of
      // two record words (or the word itself when the window starts on a
      // word boundary)
      uint32_t ow[MAXM / 2];
      if (in_rec[v]) {
        const bool odd = ((n - 2) & 1) != 0;
#pragma unroll
        for (int y = 0; y < MAXM / 2; ++y)
          ow[y] = odd ? __builtin_amdgcn_alignbit(wd[v][y + 1], wd[v][y], 16) : wd[v][y];
      } else {
        uint16_t tok[MAXM];
        if (words) {
          load_window<MAXM>(st.tok[s], st.n[s], start, tok);
        } else {
          const uint64_t N = st.n[s];
#pragma unroll
          for (int x = 0; x < MAXM; ++x) tok[x] = (start + x < N) ? st.tok[s][start + x] : (uint16_t)0;
        }
#pragma unroll
        for (int y = 0; y < MAXM / 2; ++y) ow[y] = (uint32_t)tok[2 * y] | ((uint32_t)tok[2 * y + 1] << 16);
      }
      // cut before the first 0 (and at m): one bit per zero token
      uint32_t zm = 1u << m;
#pragma unroll
      for (int y = 0; y < MAXM / 2; ++y) {
        zm |= (ow[y] & 0xFFFFu) == 0u ? 1u << (2 * y) : 0u;
        zm |= (ow[y] >> 16) == 0u ? 2u << (2 * y) : 0u;
      }
      const int len = __builtin_ctz(zm);
#pragma unroll
      for (int y = 0; y < MAXM / 2; ++y)
        ow[y] &= (2 * y < len ? 0xFFFFu : 0u) | (2 * y + 1 < len ? 0xFFFF0000u : 0u);
      const int64_t slot = (int64_t)rowv[v] * k + iv[v];
      uint16_t* out = cont_tok + slot * m;
      if (out_words) {
        uint32_t* out32 = (uint32_t*)out;
        if (m == MAXM) {
          // a full row: dword-aligned 16-byte stores plus single words
#pragma unroll
          for (int x = 0; x + 4 <= MAXM / 2; x += 4) {
            fc::u32x4_a4 q4;
            q4.x = ow[x];
            q4.y = ow[x + 1];
            q4.z = ow[x + 2];
            q4.w = ow[x + 3];
            *(fc::u32x4_a4*)(out32 + x) = q4;
          }
#pragma unroll
          for (int x = MAXM / 2 / 4 * 4; x < MAXM / 2; ++x) out32[x] = ow[x];
        } else {
#pragma unroll
          for (int x = 0; x < MAXM / 2; ++x)
            if (2 * x < m) out32[x] = ow[x];
        }
      } else {
#pragma unroll
        for (int x = 0; x < MAXM; ++x)
          if (x < m) out[x] = (uint16_t)(ow[x >> 1] >> (16 * (x & 1)));
      }
      cont_pos[slot] = (uint32_t)start;
      cont_src[slot] = (uint8_t)s;
      cont_len[slot] = (uint8_t)len;
    }
  }
}

// Any m up to 255: the token copy loops over m with a cut flag.
__global__ void __launch_bounds__(kGatherThreads) k_gather_any(StoreArgs st, int S, int k, int m,
                                                               const int32_t* __restrict__ match_n,
                                                               const uint32_t* __restrict__ range_lo,
                                                               const uint32_t* __restrict__ range_cnt,
                                                               const int32_t* __restrict__ taken,
                                                               uint32_t* __restrict__ cont_pos,
                                                               uint8_t* __restrict__ cont_src,
                                                               uint8_t* __restrict__ cont_len,
                                                               uint16_t* __restrict__ cont_tok,
                                                               const int32_t* __restrict__ rows, int n_rows) {
  const int b = fc::map_row(rows, n_rows, (int)blockIdx.x);  // row of this query
  if (b < 0) return;
  int64_t total = 0;
  for (int s = 0; s < S; ++s) total += taken[(int64_t)b * S + s];
  for (int i = (int)threadIdx.x; i < total; i += kGatherThreads) {
    int64_t before = 0;
    int src = 0;
    for (int s = 0; s < S; ++s) {
      const int64_t t = taken[(int64_t)b * S + s];
      if (i < before + t) {
        src = s;
        break;
      }
      before += t;
    }
    const int64_t o = (int64_t)b * S + src;
    const uint64_t cnt = range_cnt[o];
    const uint64_t budget = (uint64_t)((int64_t)k - before);
    const uint64_t local = (uint64_t)(i - before);
    const uint64_t off = cnt > budget ? (local * cnt) / budget : local;
    const uint32_t jj = st.sa[src][(uint64_t)range_lo[o] + off];
    const uint64_t start = (uint64_t)jj + (uint64_t)match_n[o];
    const uint16_t* T = st.tok[src];
    const uint64_t N = st.n[src];
    const int64_t slot = (int64_t)b * k + i;
    uint16_t* out = cont_tok + slot * m;
    int len = 0;
    bool open = true;
    for (int x = 0; x < m; ++x) {
      uint16_t v = 0;
      if (open) {
        const uint64_t p = start + (uint64_t)x;
        if (p < N) v = T[p];
        if (v == 0) open = false; else ++len;
      }
      out[x] = open ? v : 0;
    }
    cont_pos[slot] = (uint32_t)start;
    cont_src[slot] = (uint8_t)src;
    cont_len[slot] = (uint8_t)len;
  }
}

}  // namespace

extern "C" size_t fc_retrieve_workspace_bytes(int32_t B, int32_t S, fc_retrieve_params p) {
  (void)S;
  (void)p;
  return B > 0 ? ((size_t)B + 1) * sizeof(uint32_t) : 0;
}

namespace {

// Host-side checks shared by fc_retrieve and fc_retrieve_noalloc; fills the
// kernels' store arguments.  Nothing touches the device.
fc_status retrieve_check(const fc_store* stores, int32_t S, const uint16_t* ctx, int32_t B, int32_t L,
                         const fc_retrieve_params& p, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                         int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len,
                         uint16_t* cont_tok, const int32_t* rows, int32_t n_rows, StoreArgs& st) {
  if (!stores || S < 1 || S > FC_MAX_SOURCES) return FC_ERR_INVALID;
  if (B < 0 || L < 1) return FC_ERR_INVALID;
  if (p.n_max < 1 || p.n_max > FC_MAX_NMAX || p.n_min < 1 || p.n_min > p.n_max) return FC_ERR_INVALID;
  if (p.k < 1 || p.m < 1 || p.m > 255) return FC_ERR_INVALID;
  if ((int64_t)S * (p.n_max - p.n_min + 1) * 2 > 4 * fc::kWave) return FC_ERR_INVALID;
  if ((uint64_t)B * (uint64_t)p.k > 0x7FFFFFFFull) return FC_ERR_UNSUPPORTED;  // slot numbers stay below 2^31
  st = StoreArgs{};
  for (int s = 0; s < S; ++s) {
    const fc_store& x = stores[s];
    if (x.n >= 0xFFFFFFFFull) return FC_ERR_INVALID;
    if (x.n > 0 && (!x.tokens || !x.sa || !x.bucket)) return FC_ERR_INVALID;
    st.tok[s] = x.tokens;
    st.sa[s] = x.sa;
    st.bucket[s] = x.bucket;
    st.n[s] = (uint32_t)x.n;
    st.pair[s] = x.pair;
    st.pair_vocab[s] = x.pair ? x.pair_vocab : 0u;
    if (x.pair && (x.pair_vocab < 1 || x.pair_vocab > 65536)) return FC_ERR_INVALID;
    if (x.rec && (!x.pair || ((uintptr_t)x.rec & (FC_RECORD_BYTES - 1)))) return FC_ERR_INVALID;
    st.rec[s] = x.n > 0 ? (const uint4*)x.rec : nullptr;
    if (x.top && (!x.rec || ((uintptr_t)x.top & (FC_TOP_BYTES - 1)))) return FC_ERR_INVALID;
    st.top[s] = x.n > 0 ? (const uint4*)x.top : nullptr;
  }
  if (B == 0) return FC_OK;
  if (!ctx || !match_n || !range_lo || !range_cnt || !taken || !cont_pos || !cont_src || !cont_len || !cont_tok)
    return FC_ERR_INVALID;
  if (rows && n_rows < 1) return FC_ERR_INVALID;
  return FC_OK;
}

// The launches of one retrieval (after retrieve_check and with a workspace
// of at least fc_retrieve_workspace_bytes bytes).
fc_status retrieve_launch(const StoreArgs& st, int32_t S, const uint16_t* ctx, int32_t B, int32_t L,
                          const fc_retrieve_params& p, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                          int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len,
                          uint16_t* cont_tok, const int32_t* rows, int32_t n_rows, void* ws, hipStream_t stream) {
  (void)hipGetLastError();
  // lanes per search task: the largest power of two <= 16 that fits; a
  // small batch leaves CUs idle, so its workgroups are two or four times as
  // wide
  const bool widest = B <= kSearchWidestMaxB, wide = B <= kSearchWideMaxB;
  const int nt = widest ? kSearchWidest : wide ? kSearchWide : kSearchThreads;
  const int tasks = S * (p.n_max - p.n_min + 1) * 2;
  int G = 16;
  while (G > 1 && G * tasks > nt) G >>= 1;
  int log2_2g = 1;
  while ((1 << log2_2g) < 2 * G) ++log2_2g;
  if (widest)
    hipLaunchKernelGGL(k_search<kSearchWidest>, dim3(B), dim3(kSearchWidest), 0, stream, st, S, ctx, L, p.n_max,
                       p.n_min, p.k, G, log2_2g, rows, n_rows, match_n, range_lo, range_cnt, taken);
  else if (wide)
    hipLaunchKernelGGL(k_search<kSearchWide>, dim3(B), dim3(kSearchWide), 0, stream, st, S, ctx, L, p.n_max, p.n_min,
                       p.k, G, log2_2g, rows, n_rows, match_n, range_lo, range_cnt, taken);
  else
    hipLaunchKernelGGL(k_search<kSearchThreads>, dim3(B), dim3(kSearchThreads), 0, stream, st, S, ctx, L, p.n_max,
                       p.n_min, p.k, G, log2_2g, rows, n_rows, match_n, range_lo, range_cnt, taken);
  FC_CHECK_LAUNCH();
  if (p.m <= 16) {
    uint32_t* offsets = (uint32_t*)ws;
    if (B + 1 > kOffsetsInLds) {  // else every gather workgroup numbers the slots itself
      hipLaunchKernelGGL(k_offsets, dim3(1), dim3(kScanThreads), 0, stream, taken, B, S, rows, n_rows, offsets);
      FC_CHECK_LAUNCH();
    }
    int words = 1;
    for (int s = 0; s < S; ++s) words &= (((uintptr_t)st.tok[s]) & 3) == 0;
    const int out_words = (p.m % 2 == 0) && (((uintptr_t)cont_tok) & 3) == 0;
    const uint64_t want = ((uint64_t)B * p.k + kGatherThreads - 1) / kGatherThreads;
    const uint64_t cap = p.m <= 10 ? kGatherBlocks10 : kGatherBlocks16;
    const uint32_t blocks = (uint32_t)(want < cap ? want : cap);
    if (p.m <= 10)
      hipLaunchKernelGGL(k_gather<10>, dim3(blocks), dim3(kGatherThreads), 0, stream, st, S, B, p.k, p.m, match_n,
                         range_lo, range_cnt, taken, offsets, words, out_words, rows, n_rows, cont_pos, cont_src, cont_len,
                         cont_tok);
    else
      hipLaunchKernelGGL(k_gather<16>, dim3(blocks), dim3(kGatherThreads), 0, stream, st, S, B, p.k, p.m, match_n,
                         range_lo, range_cnt, taken, offsets, words, out_words, rows, n_rows, cont_pos, cont_src, cont_len,
                         cont_tok);
  } else {
    hipLaunchKernelGGL(k_gather_any, dim3(B), dim3(kGatherThreads), 0, stream, st, S, p.k, p.m, match_n, range_lo,
                       range_cnt, taken, cont_pos, cont_src, cont_len, cont_tok, rows, n_rows);
  }
  FC_CHECK_LAUNCH();
  return FC_OK;
}

}  // namespace

extern "C" fc_status fc_retrieve(const fc_store* stores, int32_t S, const uint16_t* ctx, int32_t B, int32_t L,
                                 fc_retrieve_params p, int32_t* match_n, uint32_t* range_lo, uint32_t* range_cnt,
                                 int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src, uint8_t* cont_len,
                                 uint16_t* cont_tok, const int32_t* rows, int32_t n_rows, void* ws,
                                 size_t ws_bytes, hipStream_t stream) {
  StoreArgs st;
  const fc_status e = retrieve_check(stores, S, ctx, B, L, p, match_n, range_lo, range_cnt, taken, cont_pos,
                                     cont_src, cont_len, cont_tok, rows, n_rows, st);
  if (e != FC_OK || B == 0) return e;
  if (!ws || ws_bytes < fc_retrieve_workspace_bytes(B, S, p)) return FC_ERR_WORKSPACE;
  return retrieve_launch(st, S, ctx, B, L, p, match_n, range_lo, range_cnt, taken, cont_pos, cont_src, cont_len,
                         cont_tok, rows, n_rows, ws, stream);
}

// ---------------------------------------------------------------------------
// fc_retrieve_noalloc: fc_retrieve with its workspace in a static device
// array instead of a caller buffer, for callers that cannot allocate.  Each
// GPU holds its own copy of the array for the life of the process; its
// device address is looked up once per device (hipGetSymbolAddress, with
// that device current) and only that address is ever passed to kernels.
// Calls on one GPU share the array, so calls that overlap on one GPU race.
namespace {

constexpr size_t kNoAllocBytes = FC_RETRIEVE_NOALLOC_BYTES;
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// The device address of the current GPU's scratch array, or null on failure.
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" size_t fc_retrieve_noalloc_max_bytes(void) { return kNoAllocBytes; }

extern "C" fc_status fc_retrieve_noalloc(const fc_store* stores, int32_t S, const uint16_t* ctx, int32_t B,
                                         int32_t L, fc_retrieve_params p, int32_t* match_n, uint32_t* range_lo,
                                         uint32_t* range_cnt, int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src,
                                         uint8_t* cont_len, uint16_t* cont_tok, const int32_t* rows, int32_t n_rows,
                                         hipStream_t stream) {
  StoreArgs st;
  const fc_status e = retrieve_check(stores, S, ctx, B, L, p, match_n, range_lo, range_cnt, taken, cont_pos,
                                     cont_src, cont_len, cont_tok, rows, n_rows, st);
  if (e != FC_OK || B == 0) return e;
  if (fc_retrieve_workspace_bytes(B, S, p) > kNoAllocBytes) return FC_ERR_UNSUPPORTED;
  void* ws = device_scratch();
  if (!ws) return FC_ERR_DEVICE;
  return retrieve_launch(st, S, ctx, B, L, p, match_n, range_lo, range_cnt, taken, cont_pos, cont_src, cont_len,
                         cont_tok, rows, n_rows, ws, stream);
}
