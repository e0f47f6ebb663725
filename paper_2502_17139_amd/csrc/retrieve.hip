// Longest-suffix retrieval with continuation gather on gfx950 (fc_retrieve).
//
// For every query and store the method looks for the longest suffix of the
// context, from n_max tokens down, that occurs in the datastore, and returns
// what follows each occurrence (Section III-A; the repository store and the
// common store are searched side by side, Section IV-A and Section IV-C).
//
// k_search: one wave per query.  The wave's lanes take the (store, n, bound)
// triples - 2 stores x 15 lengths x {lower, upper} = 60 lanes at the paper's
// n_max = 16, n_min = 2 - so every candidate length is searched at once and
// the dependent probe chain is one binary search long instead of fifteen.
// Each search starts from the store's two-token table when it has one (one
// table read replaces the top ~25 levels of the search on a 1B-token store)
// or else from its first-token bucket, and compares only the tokens the
// table does not already fix.  With the store's inline-prefix records a
// probe is one 32-byte read of a record and two levels are resolved per round
// trip; without them each probe reads the suffix-array entry (prefetched a
// level ahead) and then the text.  The wave then keeps, per store, the longest n whose range
// is non-empty and fills the k slots in store priority order.
//
// k_offsets + k_gather: the kept slots of the whole batch are numbered
// consecutively and spread evenly over a persistent grid.  A slot maps to its
// store and range offset (strided floor(i*cnt/b) when the range exceeds the
// store's budget b), reads the suffix-array entry and copies up to m
// continuation tokens, cut before a 0 and at the end of the store.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kSearchThreads = 256;
constexpr int kQueriesPerBlock = kSearchThreads / fc::kWave;
constexpr int kGatherThreads = 256;
constexpr int kScanThreads = 1024;
constexpr int kOffsetsInLds = 4096;
constexpr int kGatherBlocks = 2048;

struct StoreArgs {
  const uint16_t* tok[FC_MAX_SOURCES];
  const uint32_t* sa[FC_MAX_SOURCES];
  const uint32_t* bucket[FC_MAX_SOURCES];
  const uint32_t* pair[FC_MAX_SOURCES];
  const uint4* rec[FC_MAX_SOURCES];
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

// Lower (upper = false) or upper bound of the pattern in suffix-array range
// [lo, hi) over the records: two levels of the binary search per memory
// round trip, by loading the midpoint's record together with the records
// of both possible next midpoints.
__device__ __forceinline__ uint32_t rec_search(const uint4* __restrict__ R, uint32_t lo, uint32_t hi,
                                               const RecQuery& rq, bool upper) {
  while (lo < hi) {
    const uint32_t mid = lo + ((hi - lo) >> 1);
    const uint32_t lmid = lo < mid ? lo + ((mid - lo) >> 1) : mid;
    const uint32_t rmid = mid + 1 < hi ? (mid + 1) + ((hi - mid - 1) >> 1) : mid;
    const uint4 m0 = R[kRecQuads * (uint64_t)mid], m1 = R[kRecQuads * (uint64_t)mid + 1];
    const uint4 l0 = R[kRecQuads * (uint64_t)lmid], l1 = R[kRecQuads * (uint64_t)lmid + 1];
    const uint4 r0 = R[kRecQuads * (uint64_t)rmid], r1 = R[kRecQuads * (uint64_t)rmid + 1];
    const int c = rec_cmp(m0, m1, rq);
    const bool right = upper ? c <= 0 : c < 0;
    if (right) lo = mid + 1; else hi = mid;
    if (lo < hi) {
      const uint32_t nm = right ? rmid : lmid;
      const uint4 a0 = right ? r0 : l0, a1 = right ? r1 : l1;
      const int c2 = rec_cmp(a0, a1, rq);
      if (upper ? c2 <= 0 : c2 < 0) lo = nm + 1; else hi = nm;
    }
  }
  return lo;
}

__global__ void __launch_bounds__(kSearchThreads) k_search(StoreArgs st, int S, const uint16_t* __restrict__ ctx,
                                                           int B, int L, int n_max, int n_min, int k,
                                                           const int32_t* __restrict__ rows, int n_rows,
                                                           int32_t* __restrict__ match_n,
                                                           uint32_t* __restrict__ range_lo,
                                                           uint32_t* __restrict__ range_cnt,
                                                           int32_t* __restrict__ taken) {
  __shared__ uint16_t s_q[kQueriesPerBlock][FC_MAX_NMAX];
  __shared__ uint32_t s_lo[kQueriesPerBlock][FC_MAX_SOURCES][FC_MAX_NMAX];
  __shared__ uint32_t s_hi[kQueriesPerBlock][FC_MAX_SOURCES][FC_MAX_NMAX];
  __shared__ int s_nhi[kQueriesPerBlock];

  const int w = threadIdx.x / fc::kWave;
  const int lane = fc::lane_id();
  const int b = blockIdx.x * kQueriesPerBlock + w;
  const bool active = b < B;
  const int nq = L < FC_MAX_NMAX ? L : FC_MAX_NMAX;  // tokens of the context kept

  if (active && lane < nq) s_q[w][FC_MAX_NMAX - nq + lane] = ctx[(int64_t)b * L + (L - nq + lane)];
  if (active && lane < FC_MAX_SOURCES * FC_MAX_NMAX) {
    (&s_lo[w][0][0])[lane] = 0;
    (&s_hi[w][0][0])[lane] = 0;
  }
  __syncthreads();
  if (active && lane == 0) {
    int tail = 0;
    while (tail < nq && s_q[w][FC_MAX_NMAX - 1 - tail] != 0) ++tail;
    int h = n_max < L ? n_max : L;
    s_nhi[w] = tail < h ? tail : h;
  }
  __syncthreads();

  const int NN = n_max - n_min + 1;
  const int tasks = S * NN * 2;
  if (active) {
    const int n_hi = s_nhi[w];
    for (int t = lane; t < tasks; t += fc::kWave) {
      const int s = t / (2 * NN);
      const int rem = t - s * 2 * NN;
      const int ni = rem >> 1;
      const int upper = rem & 1;
      const int n = n_max - ni;
      if (n > n_hi || n < n_min) continue;
      const uint16_t* q = &s_q[w][FC_MAX_NMAX - n];
      const uint16_t* T = st.tok[s];
      const uint32_t* SA = st.sa[s];
      const uint32_t N = st.n[s];
      uint32_t lo = 0, hi = 0;
      int from = 1;
      if (N > 0) {
        const uint32_t V = st.pair_vocab[s];
        if (n >= 2 && st.pair[s] != nullptr && q[0] < V && q[1] < V) {
          // two-token table: the range of suffixes starting with q[0] q[1]
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
      // Binary search, over the records when the store has them; else the
      // suffix-array entries of both possible next midpoints are fetched
      // together with the current probe's text, so each level costs one
      // dependent round trip.  When the table already covers the whole
      // pattern the range is final.
      if (from < n && lo < hi && from == 2 && st.rec[s] != nullptr) {
        lo = rec_search(st.rec[s], lo, hi, rec_query(q, n), upper);
      } else if (from < n && lo < hi) {
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
      if (upper) s_hi[w][s][ni] = lo; else s_lo[w][s][ni] = lo;
    }
  }
  __syncthreads();
  const int row = active ? fc::map_row(rows, n_rows, b) : -1;
  if (active && lane == 0 && row >= 0) {
    const int n_hi = s_nhi[w];
    int64_t used = 0;
    for (int s = 0; s < S; ++s) {
      int mn = 0;
      uint32_t lo = 0, cnt = 0;
      for (int n = n_hi; n >= n_min; --n) {
        const int ni = n_max - n;
        const uint32_t c = s_hi[w][s][ni] - s_lo[w][s][ni];
        if (c > 0) {
          mn = n;
          lo = s_lo[w][s][ni];
          cnt = c;
          break;
        }
      }
      const int64_t budget = (int64_t)k - used;
      const int64_t tk = (int64_t)cnt < budget ? (int64_t)cnt : budget;
      const int64_t o = (int64_t)row * S + s;
      match_n[o] = mn;
      range_lo[o] = lo;
      range_cnt[o] = cnt;
      taken[o] = (int32_t)tk;
      used += tk;
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

// The per-store fields of one query's row that its slots need.
struct RowMeta {
  int32_t taken[FC_MAX_SOURCES];
  uint32_t cnt[FC_MAX_SOURCES], lo[FC_MAX_SOURCES];
  int32_t n[FC_MAX_SOURCES];
};

__device__ __forceinline__ RowMeta load_meta(const int32_t* __restrict__ taken, const uint32_t* __restrict__ range_cnt,
                                             const uint32_t* __restrict__ range_lo,
                                             const int32_t* __restrict__ match_n, int64_t row, int S) {
  RowMeta r;
#pragma unroll
  for (int u = 0; u < FC_MAX_SOURCES; ++u) {
    const int64_t o = row * S + u;
    r.taken[u] = u < S ? taken[o] : 0;
    r.cnt[u] = u < S ? range_cnt[o] : 0u;
    r.lo[u] = u < S ? range_lo[o] : 0u;
    r.n[u] = u < S ? match_n[o] : 0;
  }
  return r;
}

// Kept slots of the whole batch as one flat range, split evenly over a
// persistent grid: slot g belongs to the query b with offsets[b] <= g <
// offsets[b+1] (binary search in an LDS copy of the offsets).  A wave whose
// slots all belong to one query (the common case) reads that query's
// per-store fields with scalar loads.  Each slot reads its inline-prefix
// record (or else its suffix-array entry and then the text) at consecutive
// positions when the whole range is kept, cuts the window at the first 0 in
// registers and writes the tokens two per 32-bit store when rows are
// 4-byte aligned.
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
  const bool in_lds = B + 1 <= kOffsetsInLds;
  if (in_lds)
    for (int i = (int)threadIdx.x; i <= B; i += kGatherThreads) s_off[i] = offsets[i];
  __syncthreads();
  const uint32_t* off_tab = in_lds ? s_off : offsets;
  const uint32_t total = off_tab[B];
  for (uint32_t g = blockIdx.x * kGatherThreads + threadIdx.x; g < total; g += gridDim.x * kGatherThreads) {
    int lo = 0, hi = B;  // last b with offsets[b] <= g
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (off_tab[mid] <= g) lo = mid; else hi = mid;
    }
    const int b = lo;
    const int row = fc::map_row(rows, n_rows, b);  // >= 0: a skipped query owns no slots
    const int i = (int)(g - off_tab[b]);
    const int rf = __builtin_amdgcn_readfirstlane(row);
    const RowMeta meta = fc::ballot(row != rf) == 0 ? load_meta(taken, range_cnt, range_lo, match_n, rf, S)
                                                    : load_meta(taken, range_cnt, range_lo, match_n, row, S);
    // the slot's store: stores before it fill the first slots
    int s = 0;
    int64_t before = 0;
    uint64_t cnt = meta.cnt[0], rlo = meta.lo[0];
    int n = meta.n[0];
#pragma unroll
    for (int u = 1; u < FC_MAX_SOURCES; ++u) {
      const int64_t nb = before + meta.taken[u - 1];
      if (u < S && s == u - 1 && i >= nb) {
        s = u;
        before = nb;
        cnt = meta.cnt[u];
        rlo = meta.lo[u];
        n = meta.n[u];
      }
    }
    const uint64_t budget = (uint64_t)((int64_t)k - before);
    const uint64_t local = (uint64_t)(i - before);
    const uint64_t off = cnt > budget ? (local * cnt) / budget : local;
    const uint64_t idx = rlo + off;
    const uint64_t N = st.n[s];
    uint16_t v[MAXM];
    uint32_t j;
    // the window's words (token n - 2 onward) inside the record: no text read
    const int t0 = n - 2;
    if (st.rec[s] != nullptr && t0 >= 0 && (t0 >> 1) + MAXM / 2 <= FC_RECORD_TOKENS / 2 - 1) {
      const uint32_t* W = (const uint32_t*)(st.rec[s] + kRecQuads * idx);
      j = W[0];
      words_window<MAXM>(W + 1 + (t0 >> 1), t0 & 1, v);
    } else {
      j = st.sa[s][idx];
      const uint64_t start = (uint64_t)j + (uint64_t)n;
      if (words) load_window<MAXM>(st.tok[s], N, start, v);
      else {
#pragma unroll
        for (int x = 0; x < MAXM; ++x) v[x] = (start + x < N) ? st.tok[s][start + x] : (uint16_t)0;
      }
    }
    const uint64_t start = (uint64_t)j + (uint64_t)n;
    int len = m;
#pragma unroll
    for (int x = MAXM - 1; x >= 0; --x)
      if (x < m && v[x] == 0) len = x;
    const int64_t slot = (int64_t)row * k + i;
    uint16_t* out = cont_tok + slot * m;
    if (out_words) {
      uint32_t* out32 = (uint32_t*)out;
#pragma unroll
      for (int x = 0; x < MAXM / 2; ++x) {
        const uint32_t a = 2 * x < len ? v[2 * x] : 0u;
        const uint32_t c2 = 2 * x + 1 < len ? v[2 * x + 1] : 0u;
        if (2 * x < m) out32[x] = a | (c2 << 16);
      }
    } else {
#pragma unroll
      for (int x = 0; x < MAXM; ++x)
        if (x < m) out[x] = x < len ? v[x] : (uint16_t)0;
    }
    cont_pos[slot] = (uint32_t)start;
    cont_src[slot] = (uint8_t)s;
    cont_len[slot] = (uint8_t)len;
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
  hipLaunchKernelGGL(k_search, dim3(fc::div_up(B, kQueriesPerBlock)), dim3(kSearchThreads), 0, stream, st, S, ctx,
                     B, L, p.n_max, p.n_min, p.k, rows, n_rows, match_n, range_lo, range_cnt, taken);
  FC_CHECK_LAUNCH();
  if (p.m <= 16) {
    uint32_t* offsets = (uint32_t*)ws;
    hipLaunchKernelGGL(k_offsets, dim3(1), dim3(kScanThreads), 0, stream, taken, B, S, rows, n_rows, offsets);
    FC_CHECK_LAUNCH();
    int words = 1;
    for (int s = 0; s < S; ++s) words &= (((uintptr_t)st.tok[s]) & 3) == 0;
    const int out_words = (p.m % 2 == 0) && (((uintptr_t)cont_tok) & 3) == 0;
    const uint64_t want = ((uint64_t)B * p.k + kGatherThreads - 1) / kGatherThreads;
    const uint32_t blocks = (uint32_t)(want < (uint64_t)kGatherBlocks ? want : (uint64_t)kGatherBlocks);
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
