// Frequency-weighted draft trie, top-c pruning, tree mask and position ids on
// gfx950 (fc_build_tree).
//
// The retrieved continuations share prefixes; a trie over them verifies each
// shared prefix once, node weight = alpha * (occurrences in the repository
// store's results) + beta * (occurrences in the common store's results), and
// the top-weighted part of the trie is kept as the draft (Section IV-D,
// eq. (3); at most 64 draft tokens, Section V-D).  The kept nodes form the
// tree whose attention mask lets a token see only its own ancestors
// (Section IV-D, eq. (4)).
//
// One workgroup per query, everything in LDS, no hash table and no pointer
// chasing.  fc_retrieve hands each store's continuations over in suffix
// order, i.e. already sorted lexicographically, so:
//   1. the per-store sorted lists are merged into one sorted list (each
//      string finds its merged position by binary search in the other
//      stores' lists);
//   2. trie nodes are the distinct prefixes: string p owns the nodes of depth
//      d in (lcp(p-1, p), len(p)], and node (p, d)'s subtree is the run of
//      strings from p up to the next q with lcp(q-1, q) < d, so its weight is
//      a difference of alpha prefix sums - a per-depth "next head" scan gives
//      every run end;
//   3. the c-th largest weight is found by radix select (8-bit digits, LDS
//      histograms); ties are taken in (p, d) order, which is exactly
//      lexicographic path order with a prefix before its extensions, and
//      also preorder, so an ordered compaction emits the kept nodes already
//      in output order;
//   4. a node's parent is the nearest earlier kept node one level up; the
//      mask rows are ancestor bitsets expanded into int32.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kTreeThreads = 512;
constexpr int kMaskWords = FC_MAX_TREE_ROWS / 32;

struct Alpha {
  uint32_t a[FC_MAX_SOURCES];
};

struct TreeLayout {
  size_t str, A, perm, len, lcp, mlen, total;
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__host__ __device__ inline TreeLayout tree_layout(int k, int m) {
  TreeLayout t;
  size_t o = 0;
  t.str = o;  // k*m uint16 tokens (by slot); later run ends E[p][d-1]; later mask bitsets
  size_t str_bytes = (size_t)k * m * 2;
  const size_t mask_bytes = (size_t)FC_MAX_TREE_ROWS * kMaskWords * 4;
  if (str_bytes < mask_bytes) str_bytes = mask_bytes;
  o = align_up(o + str_bytes, 16);
  t.A = o;  // k+1 uint32 alpha prefix sums over merged order
  o = align_up(o + (size_t)(k + 1) * 4, 16);
  t.perm = o;  // k uint16: merged position -> slot
  o = align_up(o + (size_t)k * 2, 16);
  t.len = o;  // k uint8 by slot
  o = align_up(o + (size_t)k, 16);
  t.lcp = o;  // k uint8 by merged position
  o = align_up(o + (size_t)k, 16);
  t.mlen = o;  // k uint8 by merged position
  o = align_up(o + (size_t)k, 16);
  t.total = o;
  return t;
}

__device__ __forceinline__ int str_cmp(const uint16_t* a, int la, const uint16_t* b, int lb) {
  const int n = la < lb ? la : lb;
  for (int x = 0; x < n; ++x)
    if (a[x] != b[x]) return a[x] < b[x] ? -1 : 1;
  return la < lb ? -1 : (la > lb ? 1 : 0);
}

__device__ __forceinline__ int str_lcp(const uint16_t* a, int la, const uint16_t* b, int lb) {
  const int n = la < lb ? la : lb;
  int x = 0;
  while (x < n && a[x] == b[x]) ++x;
  return x;
}

__device__ __forceinline__ int src_of(const int* seg, int S, int i) {
  int s = 0;
  while (s + 1 < S && i >= seg[s + 1]) ++s;
  return s;
}

__global__ void __launch_bounds__(kTreeThreads) k_tree(const int32_t* __restrict__ taken,
                                                       const uint8_t* __restrict__ cont_len,
                                                       const uint16_t* __restrict__ cont_tok,
                                                       const uint16_t* __restrict__ ctx, int L, int S, int k, int m,
                                                       int c, Alpha alpha, int32_t* __restrict__ num_nodes,
                                                       int32_t* __restrict__ node_tok, int32_t* __restrict__ parent,
                                                       uint32_t* __restrict__ weight, int32_t* __restrict__ pos_ids,
                                                       int32_t* __restrict__ mask) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int s_seg[FC_MAX_SOURCES + 1];
  __shared__ int s_err;
  __shared__ uint32_t s_scratch[kTreeThreads / fc::kWave + 1];
  __shared__ uint32_t s_chunk[kTreeThreads];
  __shared__ uint32_t s_hist[256];
  __shared__ uint32_t s_sel_w[FC_MAX_TREE_ROWS];
  __shared__ uint16_t s_sel_p[FC_MAX_TREE_ROWS];
  __shared__ uint8_t s_sel_d[FC_MAX_TREE_ROWS];
  __shared__ int16_t s_par[FC_MAX_TREE_ROWS];
  __shared__ uint64_t s_sel[2];

  const TreeLayout lay = tree_layout(k, m);
  uint16_t* str = (uint16_t*)(smem + lay.str);
  uint16_t* E = str;  // reused once the tokens are no longer needed
  uint32_t* anc = (uint32_t*)(smem + lay.str);
  uint32_t* A = (uint32_t*)(smem + lay.A);
  uint16_t* perm = (uint16_t*)(smem + lay.perm);
  uint8_t* len = smem + lay.len;
  uint8_t* lcp = smem + lay.lcp;
  uint8_t* mlen = smem + lay.mlen;

  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int R = c + 1;
  const int64_t row0 = (int64_t)b * k;

  if (tid == 0) {
    int acc = 0, err = 0;
    for (int s = 0; s < S; ++s) {
      const int t = taken[(int64_t)b * S + s];
      if (t < 0) err = 1;
      s_seg[s] = acc;
      acc += t > 0 ? t : 0;
      if (acc > k) {
        err = 1;
        acc = k;
      }
    }
    s_seg[S] = acc;
    s_err = err;
  }
  __syncthreads();
  const int T = s_err ? 0 : s_seg[S];

  for (int i = tid; i < T; i += kTreeThreads) {
    const uint8_t l = cont_len[row0 + i];
    len[i] = l;
    if (l > m) s_err = 1;
  }
  for (int64_t e = tid; e < (int64_t)T * m; e += kTreeThreads) str[e] = cont_tok[row0 * m + e];
  __syncthreads();

  // Precondition: each store's slots are sorted.
  for (int i = tid; i < T; i += kTreeThreads) {
    const int s = src_of(s_seg, S, i);
    if (i > s_seg[s] && len[i - 1] <= m && len[i] <= m &&
        str_cmp(str + (int64_t)(i - 1) * m, len[i - 1], str + (int64_t)i * m, len[i]) > 0)
      s_err = 1;
  }
  __syncthreads();
  const bool err = s_err != 0;

  int nsel = 0;
  uint32_t root_w = 0;
  if (!err) {
    // 1. merged positions
    for (int i = tid; i < T; i += kTreeThreads) {
      const int s = src_of(s_seg, S, i);
      const uint16_t* x = str + (int64_t)i * m;
      const int lx = len[i];
      int mp = i - s_seg[s];
      for (int s2 = 0; s2 < S; ++s2) {
        if (s2 == s) continue;
        int lo = s_seg[s2], hi = s_seg[s2 + 1];
        const int base = lo;
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          const int cc = str_cmp(str + (int64_t)mid * m, len[mid], x, lx);
          if (s2 < s ? (cc <= 0) : (cc < 0)) lo = mid + 1; else hi = mid;
        }
        mp += lo - base;
      }
      perm[mp] = (uint16_t)i;
    }
    __syncthreads();

    // 2. merged lengths, adjacent LCPs, alpha prefix sums, root weight
    const int per = (T + kTreeThreads - 1) / kTreeThreads;
    const int p0 = tid * per < T ? tid * per : T;
    const int p1 = p0 + per < T ? p0 + per : T;
    uint32_t asum = 0, rw = 0;
    for (int p = p0; p < p1; ++p) {
      const int i = perm[p];
      const int li = len[i];
      mlen[p] = (uint8_t)li;
      lcp[p] = (uint8_t)(p == 0 ? 0 : str_lcp(str + (int64_t)perm[p - 1] * m, len[perm[p - 1]], str + (int64_t)i * m, li));
      const uint32_t a = alpha.a[src_of(s_seg, S, i)];
      asum += a;
      if (li > 0) rw += a;
    }
    uint32_t atot;
    uint32_t run = fc::block_excl_sum<uint32_t>(asum, s_scratch, &atot);
    for (int p = p0; p < p1; ++p) {
      A[p] = run;
      run += alpha.a[src_of(s_seg, S, perm[p])];
    }
    if (tid == 0) A[T] = atot;
    root_w = fc::block_sum<uint32_t>(rw, s_scratch);
    __syncthreads();

    // 3. run ends: E[p][d-1] = first q > p with lcp[q] < d (or T)
    for (int d = 1; d <= m; ++d) {
      uint32_t f = (uint32_t)T;
      for (int q = p0; q < p1; ++q)
        if (lcp[q] < d) {
          f = (uint32_t)q;
          break;
        }
      s_chunk[tid] = f;
      __syncthreads();
      const uint32_t rv = s_chunk[kTreeThreads - 1 - tid];
      __syncthreads();
      const uint32_t ex = fc::block_excl_min<uint32_t>(rv, (uint32_t)T, s_scratch);
      s_chunk[kTreeThreads - 1 - tid] = ex;
      __syncthreads();
      uint32_t nh = s_chunk[tid];  // first head in later chunks
      for (int q = p1 - 1; q >= p0; --q) {
        if (lcp[q] < d) {
          if (mlen[q] >= d) E[(int64_t)q * m + d - 1] = (uint16_t)nh;
          nh = (uint32_t)q;
        }
      }
      __syncthreads();
    }

    // 4. node count, largest weight
    uint32_t nodes = 0, wmax = 0;
    for (int p = p0; p < p1; ++p) {
      for (int d = lcp[p] + 1; d <= mlen[p]; ++d) {
        const uint32_t W = A[E[(int64_t)p * m + d - 1]] - A[p];
        wmax = W > wmax ? W : wmax;
        ++nodes;
      }
    }
    nodes = fc::block_sum<uint32_t>(nodes, s_scratch);
    wmax = fc::block_max<uint32_t>(wmax, s_scratch);
    const uint32_t need = nodes < (uint32_t)c ? nodes : (uint32_t)c;

    // 5. radix select: W* = need-th largest weight; take_eq nodes of weight W*
    uint64_t prefix = 0;
    uint32_t remaining = need;
    int bits = 0;
    for (uint32_t x = wmax; x; x >>= 1) ++bits;
    if (need > 0 && bits > 0) {
      for (int shift = ((bits - 1) / 8) * 8; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += kTreeThreads) s_hist[i] = 0;
        __syncthreads();
        for (int p = p0; p < p1; ++p) {
          for (int d = lcp[p] + 1; d <= mlen[p]; ++d) {
            const uint64_t W = A[E[(int64_t)p * m + d - 1]] - A[p];
            if ((W >> (shift + 8)) == (prefix >> (shift + 8))) atomicAdd(&s_hist[(W >> shift) & 0xFF], 1u);
          }
        }
        __syncthreads();
        if (tid == 0) {
          uint32_t acc = 0;
          int sel = 0;
          for (int bin = 255; bin >= 0; --bin) {
            if (acc + s_hist[bin] >= remaining) {
              sel = bin;
              break;
            }
            acc += s_hist[bin];
          }
          s_sel[0] = prefix | ((uint64_t)sel << shift);
          s_sel[1] = remaining - acc;
        }
        __syncthreads();
        prefix = s_sel[0];
        remaining = (uint32_t)s_sel[1];
        __syncthreads();
      }
    }
    const uint64_t wstar = prefix;
    const uint32_t take_eq = remaining;

    // 6. ordered selection in (p, d) order = preorder
    uint32_t eq = 0;
    for (int p = p0; p < p1; ++p)
      for (int d = lcp[p] + 1; d <= mlen[p]; ++d)
        if ((uint64_t)(A[E[(int64_t)p * m + d - 1]] - A[p]) == wstar) ++eq;
    uint32_t eq_rank = fc::block_excl_sum<uint32_t>(eq, s_scratch, nullptr);
    uint32_t cnt = 0;
    {
      uint32_t r = eq_rank;
      for (int p = p0; p < p1; ++p)
        for (int d = lcp[p] + 1; d <= mlen[p]; ++d) {
          const uint64_t W = A[E[(int64_t)p * m + d - 1]] - A[p];
          bool keep = false;
          if (W > wstar) keep = true;
          else if (W == wstar) keep = (r++ < take_eq);
          cnt += keep ? 1u : 0u;
        }
    }
    uint32_t total_sel;
    uint32_t o = 1 + fc::block_excl_sum<uint32_t>(cnt, s_scratch, &total_sel);
    if (need == 0) total_sel = 0;
    if (need > 0) {
      uint32_t r = eq_rank;
      for (int p = p0; p < p1; ++p)
        for (int d = lcp[p] + 1; d <= mlen[p]; ++d) {
          const uint64_t W = A[E[(int64_t)p * m + d - 1]] - A[p];
          bool keep = false;
          if (W > wstar) keep = true;
          else if (W == wstar) keep = (r++ < take_eq);
          if (keep && o < (uint32_t)FC_MAX_TREE_ROWS) {
            s_sel_p[o] = (uint16_t)p;
            s_sel_d[o] = (uint8_t)d;
            s_sel_w[o] = (uint32_t)W;
            ++o;
          }
        }
    }
    nsel = (int)(total_sel < (uint32_t)c ? total_sel : (uint32_t)c);
    if (tid == 0) s_sel_d[0] = 0;
    __syncthreads();
    // parents: nearest earlier kept node one level up
    for (int r = tid + 1; r <= nsel; r += kTreeThreads) {
      const int d = s_sel_d[r];
      int q = r - 1;
      while (q > 0 && s_sel_d[q] != d - 1) --q;
      s_par[r] = (int16_t)q;
    }
    if (tid == 0) s_par[0] = -1;
    __syncthreads();
  }

  // 7. emit rows
  const int num = err ? 0 : 1 + nsel;
  for (int r = tid; r < R; r += kTreeThreads) {
    const int64_t out = (int64_t)b * R + r;
    int32_t tk = 0, pr = -1, ps = 0;
    uint32_t wt = 0;
    if (r < num) {
      if (r == 0) {
        tk = ctx[(int64_t)b * L + L - 1];
        wt = root_w;
      } else {
        const int p = s_sel_p[r];
        const int d = s_sel_d[r];
        tk = cont_tok[(row0 + perm[p]) * m + d - 1];
        pr = s_par[r];
        wt = s_sel_w[r];
        ps = d;
      }
    }
    node_tok[out] = tk;
    parent[out] = pr;
    weight[out] = wt;
    pos_ids[out] = ps;
  }
  // mask: ancestor bitsets (the LDS token area is free by now)
  for (int i = tid; i < FC_MAX_TREE_ROWS * kMaskWords; i += kTreeThreads) anc[i] = 0;
  __syncthreads();
  for (int r = tid; r < num; r += kTreeThreads) {
    int j = r;
    while (j >= 0) {
      anc[r * kMaskWords + (j >> 5)] |= 1u << (j & 31);
      j = (j == 0) ? -1 : s_par[j];
    }
  }
  __syncthreads();
  const int64_t mbase = (int64_t)b * R * R;
  for (int e = tid; e < R * R; e += kTreeThreads) {
    const int i = e / R, j = e - (e / R) * R;
    mask[mbase + e] = (i < num) ? (int32_t)((anc[i * kMaskWords + (j >> 5)] >> (j & 31)) & 1u) : 0;
  }
  if (tid == 0) num_nodes[b] = err ? -1 : num;
}

}  // namespace

extern "C" fc_status fc_build_tree(const int32_t* taken, const uint8_t* cont_len, const uint16_t* cont_tok,
                                   const uint16_t* ctx, int32_t B, int32_t L, int32_t S, int32_t k, int32_t m,
                                   fc_tree_params t, int32_t* num_nodes, int32_t* node_tok, int32_t* parent,
                                   uint32_t* weight, int32_t* pos_ids, int32_t* mask, hipStream_t stream) {
  if (B < 0 || L < 1 || S < 1 || S > FC_MAX_SOURCES) return FC_ERR_INVALID;
  if (k < 1 || m < 1 || m > 255 || t.c < 1 || t.c + 1 > FC_MAX_TREE_ROWS) return FC_ERR_INVALID;
  if (k > 65535) return FC_ERR_UNSUPPORTED;
  for (int s = 0; s < S; ++s)
    if ((uint64_t)t.alpha[s] * (uint64_t)k > 0xFFFFFFFFull) return FC_ERR_UNSUPPORTED;
  if (B == 0) return FC_OK;
  if (!taken || !cont_len || !cont_tok || !ctx || !num_nodes || !node_tok || !parent || !weight || !pos_ids || !mask)
    return FC_ERR_INVALID;
  const TreeLayout lay = tree_layout(k, m);
  int dev = 0, max_lds = 0;
  FC_CHECK_HIP(hipGetDevice(&dev));
  FC_CHECK_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
  const size_t static_lds = 6 * 1024;
  if (lay.total + static_lds > (size_t)max_lds) return FC_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  if (lay.total > 64 * 1024)
    (void)hipFuncSetAttribute((const void*)k_tree, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lay.total);
  (void)hipGetLastError();
  Alpha a = {};
  for (int s = 0; s < S; ++s) a.a[s] = t.alpha[s];
  hipLaunchKernelGGL(k_tree, dim3(B), dim3(kTreeThreads), lay.total, stream, taken, cont_len, cont_tok, ctx, L, S, k,
                     m, t.c, a, num_nodes, node_tok, parent, weight, pos_ids, mask);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
