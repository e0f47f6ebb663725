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
//      is the match length n, and the occurrences of the n-token suffix are
//      the positions where it reaches n;
//   2. range_lo: the number of suffixes of the text below the pattern;
//   3. the occurrences, sorted into suffix order by a bitonic sort in LDS;
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

// Suffix a below suffix b of T[0..len), knowing their first `from` tokens
// agree (a != b, so one is a proper prefix of the other or they differ).
__device__ __forceinline__ bool suffix_less(const uint16_t* T, uint32_t len, uint32_t a, uint32_t b, int from) {
  if (a == kNone) return false;
  if (b == kNone) return true;
  for (uint32_t x = (uint32_t)from;; ++x) {
    if (a + x == len) return true;   // a ends first: the shorter is smaller
    if (b + x == len) return false;
    const uint16_t ta = T[a + x], tb = T[b + x];
    if (ta != tb) return ta < tb;
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
  for (uint32_t i = tid; i < len; i += kCacheThreads) T[i] = src[i];
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

  // 1. longest agreement over every end position
  uint32_t best = 0;
  if (n_hi >= n_min)
    for (uint32_t e = tid + 1; e <= len; e += kCacheThreads) {
      uint32_t l = 0;
      while ((int)l < n_hi && l < e && T[e - 1 - l] == qend[-1 - (int)l]) ++l;
      best = l > best ? l : best;
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
  const uint16_t* q = qend - n;

  // occurrences of q (start j: T[j..j+n) == q), compacted in text order
  const uint32_t span = len >= (uint32_t)n ? len - (uint32_t)n + 1 : 0u;
  const uint32_t per = (span + kCacheThreads - 1) / kCacheThreads;
  const uint32_t j0 = tid * per < span ? tid * per : span;
  const uint32_t j1 = j0 + per < span ? j0 + per : span;
  auto is_occ = [&](uint32_t j) -> bool {
    for (int x = 0; x < n; ++x)
      if (T[j + x] != q[x]) return false;
    return true;
  };
  uint32_t mine = 0;
  for (uint32_t j = j0; j < j1; ++j) mine += is_occ(j) ? 1u : 0u;
  uint32_t cnt;
  uint32_t at = fc::block_excl_sum<uint32_t>(mine, s_red, &cnt);
  for (uint32_t j = j0; j < j1; ++j)
    if (is_occ(j)) occ[at++] = j;
  const uint32_t Pc = pow2_at_least(cnt);
  for (uint32_t i = cnt + tid; i < Pc; i += kCacheThreads) occ[i] = kNone;

  // 2. suffixes of the text below q
  uint32_t below = 0;
  for (uint32_t i = tid; i < len; i += kCacheThreads) {
    int c = 0;
    for (int x = 0; x < n; ++x) {
      if (i + x == len) {
        c = -1;
        break;
      }
      if (T[i + x] != q[x]) {
        c = T[i + x] < q[x] ? -1 : 1;
        break;
      }
    }
    below += c < 0 ? 1u : 0u;
  }
  below = fc::block_sum<uint32_t>(below, s_red);

  // 3. suffix order (every occurrence starts with q: compare from offset n)
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
