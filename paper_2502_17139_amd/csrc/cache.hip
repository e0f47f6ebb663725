// The CACHE of Section IV-B on gfx950: retrieval from small per-stream texts
// (fc_cache_retrieve) and their batched update (fc_cache_write).
//
// A CACHE holds token sequences; searched as a store (Section III-A) its text
// is the sequences joined by single 0 tokens.  It is small (at most
// FC_MAX_CACHE_TOKENS tokens) and changes every decoding step, so it gets no
// suffix array: one workgroup per query loads the whole text into LDS and
// answers the query by brute force, with results identical to a suffix-array
// search of a one-store datastore holding that text:
//   1. agreement: for every end position e, how many tokens before e agree
//      with the end of the context (capped at n_hi); the longest agreement
//      is the match length n;
//   2. one comparison of every suffix with the n-token pattern gives
//      range_lo (the suffixes below it) and the occurrences (the suffixes
//      that start with it), numbered in text order by a block scan;
//   3. the occurrences in suffix order: ranks by counting pairwise
//      comparisons when there are at most 128 (beyond 32, each unordered
//      pair compared once), else a bitonic sort in LDS;
//   4. the kept ones (strided floor(i*cnt/k) beyond k) and their
//      continuations, cut before a 0 and at the end of the text.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kCacheThreads = 1024;
constexpr uint32_t kNone = 0xFFFFFFFFu;  // sorts after every occurrence

__host__ __device__ inline uint32_t pow2_at_least(uint32_t x) {
  uint32_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Tokens p .. p+15 of T[0..len) (T 4-byte aligned) as 8 words holding two
// tokens each, the earlier in the high half, so that one unsigned compare
// orders two tokens lexicographically; words at or past len read as 0 (the
// caller bounds the compare by the lengths).
__device__ __forceinline__ void token_pairs(const uint16_t* T, uint32_t len, uint32_t p, uint32_t (&w)[8]) {
  const uint32_t* W = (const uint32_t*)T;
  const uint32_t wi = p >> 1;
  uint32_t r[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) r[k] = 2 * (wi + k) < len ? W[wi + k] : 0u;
  if (p & 1) {
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = (r[k] & 0xFFFF0000u) | (r[k + 1] & 0xFFFFu);
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) w[k] = __builtin_amdgcn_alignbit(r[k], r[k], 16);
  }
}

// Suffix a below suffix b of T[0..len), knowing their first `from` tokens
// agree (a != b, so one is a proper prefix of the other or they differ).
// Sixteen tokens of each are read per LDS round trip, as word pairs: CACHE
// texts repeat, so suffixes that share q often agree far beyond it.
__device__ __forceinline__ bool suffix_less(const uint16_t* T, uint32_t len, uint32_t a, uint32_t b, int from) {
  if (a == kNone) return false;
  if (b == kNone) return true;
  for (uint32_t x0 = (uint32_t)from;; x0 += 16) {
    uint32_t wa[8], wb[8];
    token_pairs(T, len, a + x0, wa);
    token_pairs(T, len, b + x0, wb);
    const uint32_t ra = len - (a + x0), rb = len - (b + x0);  // tokens left (never both 0)
    int d = 16;  // first differing token of the window
#pragma unroll
    for (int k = 7; k >= 0; --k) {
      const uint32_t x = wa[k] ^ wb[k];
      if (x) d = 2 * k + ((x >> 16) ? 0 : 1);
    }
    const uint32_t lim = ra < rb ? (ra < 16u ? ra : 16u) : (rb < 16u ? rb : 16u);
    if ((uint32_t)d < lim) {
      const int k = d >> 1;
      const uint32_t ta = (d & 1) ? (wa[k] & 0xFFFFu) : (wa[k] >> 16);
      const uint32_t tb = (d & 1) ? (wb[k] & 0xFFFFu) : (wb[k] >> 16);
      return ta < tb;
    }
    if (lim < 16u) return ra < rb;  // the shorter ends first and is smaller (ra != rb as a != b)
  }
}

__global__ void __launch_bounds__(kCacheThreads) k_cache_retrieve(
    const uint16_t* __restrict__ texts, int64_t stride, int n_texts, const int32_t* __restrict__ text_len,
    const int32_t* __restrict__ text_row, const uint16_t* __restrict__ ctx, int L, int n_max, int n_min, int k, int m,
    const int32_t* __restrict__ rows, int n_rows, int32_t* __restrict__ match_n, uint32_t* __restrict__ range_lo,
    uint32_t* __restrict__ range_cnt, int32_t* __restrict__ taken, uint32_t* __restrict__ cont_pos,
    uint8_t* __restrict__ cont_src, uint8_t* __restrict__ cont_len, uint16_t* __restrict__ cont_tok) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ uint16_t s_q[FC_MAX_NMAX];
  __shared__ uint32_t s_red[kCacheThreads / fc::kWave + 1];
  __shared__ int s_nhi;
  const int b = (int)blockIdx.x;
  const int tid = (int)threadIdx.x;
  const int row = fc::map_row(rows, n_rows, b);
  if (row < 0) return;  // the whole workgroup: a skipped query
  const int tr = text_row ? text_row[b] : b;
  const bool have = tr >= 0 && tr < n_texts;  // a text outside the buffer reads as empty
  int len_i = have ? text_len[tr] : 0;
  len_i = len_i < 0 ? 0 : (len_i > stride ? (int)stride : len_i);
  const uint32_t len = (uint32_t)len_i;
  uint16_t* T = (uint16_t*)smem;
  uint32_t* occ = (uint32_t*)(smem + (((size_t)stride * 2 + 15) & ~(size_t)15));

  const uint16_t* src = texts + (int64_t)(have ? tr : 0) * stride;
  uint32_t head = 0;  // tokens loaded 16 bytes at a time
  if ((((uintptr_t)src) & 15) == 0) {
    head = len & ~7u;
    for (uint32_t v = tid; v < (head >> 3); v += kCacheThreads) ((uint4*)T)[v] = ((const uint4*)src)[v];
  }
  for (uint32_t i = head + tid; i < len; i += kCacheThreads) T[i] = src[i];
  const int nq = L < FC_MAX_NMAX ? L : FC_MAX_NMAX;
  if (tid < nq) s_q[FC_MAX_NMAX - nq + tid] = ctx[(int64_t)b * L + (L - nq + tid)];
  __syncthreads();
  if (tid == 0) {
    int tail = 0;
    while (tail < nq && s_q[FC_MAX_NMAX - 1 - tail] != 0) ++tail;
    const int h = n_max < L ? n_max : L;
    s_nhi = tail < h ? tail : h;
  }
  __syncthreads();
  const int n_hi = s_nhi;
  const uint16_t* qend = s_q + FC_MAX_NMAX;  // qend[-1] is the last context token

  // 1. longest agreement over every end position.  The token before e is
  //    checked first; only where it equals the context's last token are the
  //    tokens before it read, all at once.
  uint32_t best = 0;
  if (n_hi >= n_min) {
    uint16_t qr[FC_MAX_NMAX];  // qr[l] = the l-th token from the end of the context
#pragma unroll
    for (int l = 0; l < FC_MAX_NMAX; ++l) qr[l] = l < n_hi ? qend[-1 - l] : (uint16_t)0;
    for (uint32_t e = tid + 1; e <= len; e += kCacheThreads) {
      if (T[e - 1] != qr[0]) continue;
      uint16_t t[FC_MAX_NMAX];
#pragma unroll
      for (int l = 1; l < FC_MAX_NMAX; ++l) t[l] = (l < n_hi && (uint32_t)l < e) ? T[e - 1 - l] : (uint16_t)0;
      uint32_t a = 1;
      bool on = true;
#pragma unroll
      for (int l = 1; l < FC_MAX_NMAX; ++l) {
        on = on && l < n_hi && (uint32_t)l < e && t[l] == qr[l];
        a += on ? 1u : 0u;
      }
      best = a > best ? a : best;
    }
  }
  best = fc::block_max<uint32_t>(best, s_red);
  const int n = (n_hi >= n_min && (int)best >= n_min) ? (int)best : 0;
  const int64_t o = row;  // one source
  if (n == 0) {
    if (tid == 0) {
      match_n[o] = 0;
      range_lo[o] = 0;
      range_cnt[o] = 0;
      taken[o] = 0;
    }
    return;
  }

  // 2. one pass over the suffixes, in contiguous chunks: each is compared
  //    with the n-token pattern q (its first token alone, then, where that
  //    agrees, eight tokens per LDS round trip) and is
  //    below it, starts with it (an occurrence) or is above it.  A chunk has
  //    at most FC_MAX_CACHE_TOKENS / kCacheThreads = 16 suffixes, so its
  //    occurrences fit a bit mask; one block scan of (below << 16 | occurrences)
  //    numbers the occurrences in text order and totals both (each total is at
  //    most 16,384, so the halves never carry into each other).
  uint16_t qv[FC_MAX_NMAX];
#pragma unroll
  for (int x = 0; x < FC_MAX_NMAX; ++x) qv[x] = x < n ? qend[x - n] : (uint16_t)0;
  auto cmp_q = [&](uint32_t i) -> int {
#pragma unroll
    for (int x0 = 0; x0 < FC_MAX_NMAX; x0 += 8) {
      if (x0 >= n) return 0;
      uint16_t t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = (x0 + u < n && i + x0 + u < len) ? T[i + x0 + u] : (uint16_t)0;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int x = x0 + u;
        if (x >= n) return 0;
        if (i + x >= len) return -1;  // the suffix ends first: a proper prefix of q
        if (t[u] != qv[x]) return t[u] < qv[x] ? -1 : 1;
      }
    }
    return 0;
  };
  const uint32_t per = (len + kCacheThreads - 1) / kCacheThreads;
  const uint32_t i0 = tid * per < len ? tid * per : len;
  const uint32_t i1 = i0 + per < len ? i0 + per : len;
  uint32_t occ_bits = 0, packed = 0;
  for (uint32_t i = i0; i < i1; ++i) {
    // most suffixes differ from q at their first token: one LDS read decides
    const uint16_t t0 = T[i];
    const int c = t0 != qv[0] ? (t0 < qv[0] ? -1 : 1) : cmp_q(i);
    packed += c < 0 ? (1u << 16) : (c == 0 ? 1u : 0u);
    occ_bits |= c == 0 ? (1u << (i - i0)) : 0u;
  }
  uint32_t tot;
  uint32_t at = fc::block_excl_sum<uint32_t>(packed, s_red, &tot) & 0xFFFFu;
  const uint32_t cnt = tot & 0xFFFFu, below = tot >> 16;
  for (uint32_t bits = occ_bits; bits; bits &= bits - 1) occ[at++] = i0 + (uint32_t)__builtin_ctz(bits);
  const uint32_t Pc = pow2_at_least(cnt);
  for (uint32_t i = cnt + tid; i < Pc; i += kCacheThreads) occ[i] = kNone;
  __syncthreads();

  // 3. suffix order (every occurrence starts with q: compare from offset n).
  //    Up to 32 occurrences, thread (i, j) = (tid / 32, tid % 32) tells
  //    whether occurrence j's suffix is below occurrence i's and a ballot
  //    over i's 32 lanes gives i's rank; up to P = 64 or 128, i's G = 1024 / P
  //    lanes (i, j0) = (tid / G, tid % G) compare j = j0, j0 + G, ... and add
  //    their counts; more take a bitonic sort.
  if (cnt <= 32) {
    const uint32_t i = (uint32_t)tid >> 5, j = (uint32_t)tid & 31u;
    const bool lt = i < cnt && j < cnt && j != i && suffix_less(T, len, occ[j], occ[i], n);
    const uint64_t bl = fc::ballot(lt);
    const uint32_t rank = (uint32_t)__builtin_popcount((tid & 32) ? (uint32_t)(bl >> 32) : (uint32_t)bl);
    const uint32_t mine = (i < cnt && j == 0) ? occ[i] : 0u;
    __syncthreads();
    if (i < cnt && j == 0) occ[rank] = mine;
    __syncthreads();
  } else if (cnt <= 128 && Pc + 4 * cnt <= pow2_at_least((uint32_t)stride)) {
    // every unordered pair compared once, both answers kept in a bit matrix
    // past the occurrence list: bit j of row i (4 words a row) says that
    // occurrence j's suffix is below occurrence i's, and i's rank is its
    // row's population count
    uint32_t* lt = occ + Pc;
    for (uint32_t x = (uint32_t)tid; x < 4 * cnt; x += kCacheThreads) lt[x] = 0;
    __syncthreads();
    const uint32_t npairs = cnt * (cnt - 1) / 2;
    for (uint32_t q = (uint32_t)tid; q < npairs; q += kCacheThreads) {
      // pair q is (i, j), i < j, with j(j - 1) / 2 <= q < j(j + 1) / 2
      uint32_t j = (uint32_t)((sqrtf(8.0f * (float)q + 1.0f) + 1.0f) * 0.5f);
      while (j * (j - 1) / 2 > q) --j;
      while (j * (j + 1) / 2 <= q) ++j;
      const uint32_t i = q - j * (j - 1) / 2;
      if (suffix_less(T, len, occ[j], occ[i], n)) atomicOr(&lt[4 * i + (j >> 5)], 1u << (j & 31));
      else atomicOr(&lt[4 * j + (i >> 5)], 1u << (i & 31));
    }
    __syncthreads();
    const uint32_t i = (uint32_t)tid;
    uint32_t rank = 0, mine = 0;
    if (i < cnt) {
      rank = (uint32_t)(__builtin_popcount(lt[4 * i]) + __builtin_popcount(lt[4 * i + 1]) +
                        __builtin_popcount(lt[4 * i + 2]) + __builtin_popcount(lt[4 * i + 3]));
      mine = occ[i];
    }
    __syncthreads();
    if (i < cnt) occ[rank] = mine;
    __syncthreads();
  } else if (cnt <= 128) {
    const uint32_t G = cnt <= 64 ? 16u : 8u;  // lanes per occurrence i
    const uint32_t i = (uint32_t)tid / G, j0 = (uint32_t)tid % G;
    uint32_t rank = 0;
    if (i < cnt)
      for (uint32_t j = j0; j < cnt; j += G) rank += (j != i && suffix_less(T, len, occ[j], occ[i], n)) ? 1u : 0u;
    for (uint32_t off = G >> 1; off >= 1; off >>= 1) rank += (uint32_t)__shfl_xor((int)rank, (int)off, (int)G);
    const uint32_t mine = (i < cnt && j0 == 0) ? occ[i] : 0u;
    __syncthreads();
    if (i < cnt && j0 == 0) occ[rank] = mine;
    __syncthreads();
  } else {
    for (uint32_t k2 = 2; k2 <= Pc; k2 <<= 1) {
      for (uint32_t j2 = k2 >> 1; j2 > 0; j2 >>= 1) {
        for (uint32_t i = tid; i < Pc; i += kCacheThreads) {
          const uint32_t x = i ^ j2;
          if (x > i) {
            const uint32_t a = occ[i], c = occ[x];
            const bool up = (i & k2) == 0;
            const bool swap = up ? suffix_less(T, len, c, a, n) : suffix_less(T, len, a, c, n);
            if (swap) {
              occ[i] = c;
              occ[x] = a;
            }
          }
        }
        __syncthreads();
      }
    }
  }

  // 4. kept occurrences and their continuations
  const uint32_t tk = cnt < (uint32_t)k ? cnt : (uint32_t)k;
  if (tid == 0) {
    match_n[o] = n;
    range_lo[o] = below;
    range_cnt[o] = cnt;
    taken[o] = (int32_t)tk;
  }
  for (uint32_t i = tid; i < tk; i += kCacheThreads) {
    const uint64_t off = cnt > (uint32_t)k ? ((uint64_t)i * cnt) / (uint64_t)k : (uint64_t)i;
    const uint32_t start = occ[off] + (uint32_t)n;
    const int64_t slot = (int64_t)row * k + i;
    uint16_t* out = cont_tok + slot * m;
    int l = 0;
    bool open = true;
    for (int x = 0; x < m; ++x) {
      uint16_t v = 0;
      if (open) {
        if (start + x < len) v = T[start + x];
        if (v == 0) open = false; else ++l;
      }
      out[x] = open ? v : (uint16_t)0;
    }
    cont_pos[slot] = start;
    cont_src[slot] = 0;
    cont_len[slot] = (uint8_t)l;
  }
}

// Segment copy: segment i writes src_len[i] tokens from src_tok + src_off[i]
// to row dst_row[i] of the CACHE texts at dst_off[i], and sets that row's
// length to new_len[i].  One workgroup per segment; a segment naming a row
// outside [0, n_texts) is skipped and tokens that would land outside the row
// are not written.
__global__ void __launch_bounds__(256) k_cache_write(uint16_t* __restrict__ texts, int64_t stride, int n_texts,
                                                     int32_t* __restrict__ text_len, const int32_t* __restrict__ dst_row,
                                                     const int32_t* __restrict__ dst_off,
                                                     const int32_t* __restrict__ new_len,
                                                     const int64_t* __restrict__ src_off,
                                                     const int32_t* __restrict__ src_len,
                                                     const uint16_t* __restrict__ src_tok) {
  const int i = (int)blockIdx.x;
  const int r = dst_row[i], d = dst_off[i], n = src_len[i];
  if (r < 0 || r >= n_texts || d < 0) return;
  uint16_t* dst = texts + (int64_t)r * stride + d;
  const uint16_t* s = src_tok + src_off[i];
  for (int x = (int)threadIdx.x; x < n && d + x < stride; x += 256) dst[x] = s[x];
  if (threadIdx.x == 0) {
    const int nl = new_len[i];
    text_len[r] = nl < 0 ? 0 : (nl > stride ? (int)stride : nl);
  }
}

}  // namespace

extern "C" size_t fc_cache_lds_bytes(int64_t stride) {
  if (stride < 1 || stride > FC_MAX_CACHE_TOKENS) return 0;
  return (((size_t)stride * 2 + 15) & ~(size_t)15) + (size_t)pow2_at_least((uint32_t)stride) * 4;
}

extern "C" fc_status fc_cache_retrieve(const uint16_t* texts, int64_t stride, int32_t n_texts, const int32_t* text_len,
                                       const int32_t* text_row, const uint16_t* ctx, int32_t B, int32_t L,
                                       fc_retrieve_params p, int32_t* match_n, uint32_t* range_lo,
                                       uint32_t* range_cnt, int32_t* taken, uint32_t* cont_pos, uint8_t* cont_src,
                                       uint8_t* cont_len, uint16_t* cont_tok, const int32_t* rows, int32_t n_rows,
                                       hipStream_t stream) {
  if (B < 0 || L < 1 || n_texts < 1 || stride < 1 || stride > FC_MAX_CACHE_TOKENS) return FC_ERR_INVALID;
  if (p.n_max < 1 || p.n_max > FC_MAX_NMAX || p.n_min < 1 || p.n_min > p.n_max) return FC_ERR_INVALID;
  if (p.k < 1 || p.m < 1 || p.m > 255) return FC_ERR_INVALID;
  if (rows && n_rows < 1) return FC_ERR_INVALID;
  if (B == 0) return FC_OK;
  if (!texts || !text_len || !ctx || !match_n || !range_lo || !range_cnt || !taken || !cont_pos || !cont_src ||
      !cont_len || !cont_tok)
    return FC_ERR_INVALID;
  const size_t lds = fc_cache_lds_bytes(stride);
  int dev = 0, max_lds = 0;
  FC_CHECK_HIP(hipGetDevice(&dev));
  FC_CHECK_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
  if (lds + 1024 > (size_t)max_lds) return FC_ERR_UNSUPPORTED;
  if (lds > 64 * 1024)
    (void)hipFuncSetAttribute((const void*)k_cache_retrieve, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_cache_retrieve, dim3(B), dim3(kCacheThreads), lds, stream, texts, stride, n_texts, text_len,
                     text_row,
                     ctx, L, p.n_max, p.n_min, p.k, p.m, rows, n_rows, match_n, range_lo, range_cnt, taken, cont_pos,
                     cont_src, cont_len, cont_tok);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" fc_status fc_cache_write(uint16_t* texts, int64_t stride, int32_t n_texts, int32_t* text_len, int32_t n_seg,
                                    const int32_t* dst_row, const int32_t* dst_off, const int32_t* new_len,
                                    const int64_t* src_off, const int32_t* src_len, const uint16_t* src_tok,
                                    hipStream_t stream) {
  if (n_seg < 0 || n_texts < 1 || stride < 1 || stride > FC_MAX_CACHE_TOKENS) return FC_ERR_INVALID;
  if (n_seg == 0) return FC_OK;
  if (!texts || !text_len || !dst_row || !dst_off || !new_len || !src_off || !src_len || !src_tok)
    return FC_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_cache_write, dim3(n_seg), dim3(256), 0, stream, texts, stride, n_texts, text_len, dst_row,
                     dst_off,
                     new_len, src_off, src_len, src_tok);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
