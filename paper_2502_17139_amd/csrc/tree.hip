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
// One workgroup per query, no hash table and no pointer chasing.
// fc_retrieve hands each store's continuations over in suffix order, i.e.
// already sorted lexicographically, so:
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
//   4. a node's parent is the nearest earlier kept node one level up; in
//      preorder a node's subtree is the run of rows from it to its subtree
//      end (the first later row no deeper than it), so mask row j is set
//      exactly at the ancestors of j: the rows i <= j whose subtree end lies
//      past j.
// Three kernels implement this: k_tree_flat (m <= 16: only the short stores'
// strings in LDS, the long store's read in place), k_tree_fast (every kept
// string in LDS, also for the short lists too long for the flat path) and
// k_tree_any (any m).  k_tree_plan orders the queries heaviest first when
// the batch is large enough for the order to matter.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kTreeThreads = 512;
constexpr int kMaskWords = FC_MAX_TREE_ROWS / 32;
constexpr int kSmallClass = 256;  // kept slots handled by the small-LDS launch (one per thread)

struct Alpha {
  uint32_t a[FC_MAX_SOURCES];
};

struct TreeLayout {
  size_t str, A, perm, len, lcp, mlen, E, total;
};

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// sep_e: the run ends E get a region of their own instead of reusing the
// strings' (the strings then stay readable until the rows are written).
__host__ __device__ inline TreeLayout tree_layout(int k, int m, bool sep_e = false) {
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
  t.E = t.str;
  if (sep_e) {
    t.E = o;  // k*m uint16 run ends / weights
    o = align_up(o + (size_t)k * m * 2, 16);
  }
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

// alpha[s] without indexing the argument struct at run time (which would
// place it in scratch memory).
__device__ __forceinline__ uint32_t alpha_of(const Alpha& a, int s) {
  return s == 0 ? a.a[0] : s == 1 ? a.a[1] : s == 2 ? a.a[2] : a.a[3];
}

__device__ __forceinline__ int src_of(const int* seg, int S, int i) {
  int s = 0;
  while (s + 1 < S && i >= seg[s + 1]) ++s;
  return s;
}

__global__ void __launch_bounds__(kTreeThreads) k_tree_any(const int32_t* __restrict__ taken,
                                                       const uint8_t* __restrict__ cont_len,
                                                       const uint16_t* __restrict__ cont_tok,
                                                       const uint16_t* __restrict__ ctx, int L, int S, int k, int m,
                                                       int c, Alpha alpha, const int32_t* __restrict__ rows,
                                                       int n_rows, int32_t* __restrict__ num_nodes,
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
  const int in_row = fc::map_row(rows, n_rows, b);
  const int64_t row0 = (int64_t)(in_row < 0 ? 0 : in_row) * k;

  if (tid == 0) {
    int acc = 0, err = in_row < 0;
    for (int s = 0; s < S; ++s) {
      const int t = in_row < 0 ? 0 : taken[(int64_t)in_row * S + s];
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


// ---------------------------------------------------------------------------
// Fast path (m <= 16).  One workgroup of NT threads per query; queries are
// split into two launches by their kept-slot count T, each with an LDS
// layout sized for its class, so light queries run several workgroups per CU.
// Every thread owns a contiguous chunk of merged positions; per-chunk
// summaries are combined with wave shuffles and one LDS exchange, which keeps
// the number of barriers per query small.
// ---------------------------------------------------------------------------

// Longest common prefix of two rows of `m` tokens (lengths la, lb), reading
// the rows as 32-bit words: all word loads are independent, so the result
// costs one LDS round trip instead of one per token.  Requires even m (rows
// 4-byte aligned); tokens past a row's length are ignored.
template <int MAXW>
__device__ __forceinline__ int row_lcp_w(const uint16_t* a, int la, const uint16_t* b, int lb) {
  const int n = la < lb ? la : lb;
  const uint32_t* wa = (const uint32_t*)a;
  const uint32_t* wb = (const uint32_t*)b;
  int first = 2 * MAXW;
#pragma unroll
  for (int j = MAXW - 1; j >= 0; --j) {
    if (2 * j < n) {
      const uint32_t d = wa[j] ^ wb[j];
      if (d) first = 2 * j + ((d & 0xFFFFu) == 0 ? 1 : 0);
    }
  }
  return first < n ? first : n;
}

// Lexicographic comparison of two rows (a prefix first), word-wise.
template <int MAXW>
__device__ __forceinline__ int row_cmp_w(const uint16_t* a, int la, const uint16_t* b, int lb) {
  const int x = row_lcp_w<MAXW>(a, la, b, lb);
  const int n = la < lb ? la : lb;
  if (x < n) return a[x] < b[x] ? -1 : 1;
  return la < lb ? -1 : (la > lb ? 1 : 0);
}

template <int NT>
struct Scan2 {
  // Exclusive prefix sums of (x, y) over the block plus their totals, and
  // optionally the block total of z; two barriers.
  __device__ __forceinline__ static void run(uint32_t x, uint32_t y, uint32_t* sx, uint32_t* sy, uint32_t* ex,
                                             uint32_t* ey,
                             uint32_t* tx, uint32_t* ty, uint32_t z = 0, uint32_t* sz = nullptr,
                             uint32_t* tz = nullptr) {
    constexpr int NW = NT / fc::kWave;
    const int w = (int)threadIdx.x / fc::kWave;
    const uint32_t ix = fc::wave_incl_sum_u32(x), iy = fc::wave_incl_sum_u32(y);
    const uint32_t iz = sz ? fc::wave_sum_u32(z) : 0u;
    if (fc::lane_id() == fc::kWave - 1) {
      sx[w] = ix;
      sy[w] = iy;
      if (sz) sz[w] = iz;
    }
    __syncthreads();
    uint32_t px = 0, py = 0, ax = 0, ay = 0, az = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const uint32_t vx = sx[i], vy = sy[i];
      if (i < w) {
        px += vx;
        py += vy;
      }
      ax += vx;
      ay += vy;
      if (sz) az += sz[i];
    }
    *ex = px + ix - x;
    *ey = py + iy - y;
    *tx = ax;
    *ty = ay;
    if (tz) *tz = az;
    __syncthreads();
  }
};

template <int NT, int K>
struct ScanK {
  // Exclusive prefix sums of v[0..K) over the block and their totals, plus
  // the block total of z; two barriers.  s holds (K + 1) x (NT/64) words.
  __device__ __forceinline__ static void run(const uint32_t (&v)[K], uint32_t z, uint32_t* s, uint32_t (&ex)[K],
                                             uint32_t (&tot)[K], uint32_t* tz) {
    constexpr int NW = NT / fc::kWave;
    const int w = (int)threadIdx.x / fc::kWave;
    uint32_t inc[K];
#pragma unroll
    for (int u = 0; u < K; ++u) inc[u] = fc::wave_incl_sum_u32(v[u]);
    const uint32_t iz = fc::wave_sum_u32(z);
    if (fc::lane_id() == fc::kWave - 1) {
#pragma unroll
      for (int u = 0; u < K; ++u) s[u * NW + w] = inc[u];
      s[K * NW + w] = iz;
    }
    __syncthreads();
    uint32_t az = 0;
#pragma unroll
    for (int u = 0; u < K; ++u) {
      uint32_t pre = 0, all = 0;
#pragma unroll
      for (int i = 0; i < NW; ++i) {
        const uint32_t x = s[u * NW + i];
        pre += i < w ? x : 0u;
        all += x;
      }
      ex[u] = pre + inc[u] - v[u];
      tot[u] = all;
    }
#pragma unroll
    for (int i = 0; i < NW; ++i) az += s[K * NW + i];
    *tz = az;
    __syncthreads();
  }
};

// NARROW: every store has the same alpha and alpha * k fits 16 bits, so the
// alpha prefix sums are linear and every node weight is stored as is; the
// hot loops are compiled without the general paths.
template <int NT, int MAXM, bool NARROW>
__global__ void __launch_bounds__(NT, 4) k_tree_fast(const int32_t* __restrict__ taken,
                                                  const uint8_t* __restrict__ cont_len,
                                                  const uint16_t* __restrict__ cont_tok,
                                                  const uint16_t* __restrict__ ctx, int L, int S, int k, int m, int c,
                                                  Alpha alpha, const int32_t* __restrict__ list,
                                                  const int32_t* __restrict__ list_count,
                                                  int32_t* __restrict__ heavy_list, int32_t* __restrict__ heavy_count,
                                                  int B, int t_hi, int words,
                                                  const int32_t* __restrict__ rows, int n_rows,
                                                  int32_t* __restrict__ num_nodes, int32_t* __restrict__ node_tok,
                                                  int32_t* __restrict__ parent, uint32_t* __restrict__ weight,
                                                  int32_t* __restrict__ pos_ids, int32_t* __restrict__ mask) {
  constexpr int NW = NT / fc::kWave;
  static_assert(NT >= FC_MAX_TREE_ROWS, "one thread per tree row");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int s_seg[FC_MAX_SOURCES + 1];
  __shared__ int s_err;
  __shared__ uint32_t s_x[NW + 1], s_y[NW + 1], s_z[NW + 1];
  __shared__ uint16_t s_wmin[NW][MAXM + 1];
  __shared__ uint16_t s_wsuf[NW][MAXM + 1];
  __shared__ uint32_t s_hist[256];
  __shared__ uint32_t s_sel_w[FC_MAX_TREE_ROWS];
  __shared__ uint16_t s_sel_p[FC_MAX_TREE_ROWS];
  __shared__ uint8_t s_sel_d[FC_MAX_TREE_ROWS];
  __shared__ uint16_t s_sel_t[FC_MAX_TREE_ROWS];  // token of a kept node (light launch)
  __shared__ int16_t s_par[FC_MAX_TREE_ROWS];
  __shared__ uint64_t s_dball[FC_MAX_TREE_ROWS / fc::kWave][MAXM];
  __shared__ uint64_t s_shallow[FC_MAX_TREE_ROWS / fc::kWave][MAXM + 1];
  __shared__ int16_t s_end[FC_MAX_TREE_ROWS];
  __shared__ uint32_t s_pick[3];

  const int tid = threadIdx.x;
  int b;
  if (list) {
    // This launch owns the queries in `list` (written by the light launch);
    // workgroups past the list's length leave at once, after every real
    // one has been dispatched.  (list has B entries: reading it before the
    // count check saves a round trip.)
    const int b_raw = list[blockIdx.x];
    if ((int)blockIdx.x >= *list_count) return;
    b = b_raw;
  } else {
    // The light launch: workgroup q takes query q when it has T <= t_hi
    // kept slots (malformed rows too) and leaves at once otherwise; one
    // extra workgroup (q = B) writes the list of the others, in query order,
    // for the heavy launch.
    auto heavy = [&](int q) {
      const int r = fc::map_row(rows, n_rows, q);
      if (r < 0) return false;
      int T = 0, bad = 0;
      for (int u = 0; u < S; ++u) {
        const int t = taken[(int64_t)r * S + u];
        bad |= t < 0;
        T += t > 0 ? t : 0;
      }
      return !bad && T <= k && T > t_hi;
    };
    if ((int)blockIdx.x == B) {
      const int per = (B + NT - 1) / NT;
      const int q0 = tid * per < B ? tid * per : B;
      const int q1 = q0 + per < B ? q0 + per : B;
      uint32_t nh = 0;
      for (int q = q0; q < q1; ++q) nh += heavy(q) ? 1u : 0u;
      uint32_t eh, dummy, th, dummy2;
      Scan2<NT>::run(nh, 0u, s_x, s_y, &eh, &dummy, &th, &dummy2);
      for (int q = q0; q < q1; ++q)
        if (heavy(q)) heavy_list[eh++] = q;
      if (tid == 0) *heavy_count = (int32_t)th;
      return;
    }
    b = (int)blockIdx.x;
    if (heavy(b)) return;
  }
  const int lane = fc::lane_id();
  const int w = tid / fc::kWave;
  const int R = c + 1;
  const int in_row = fc::map_row(rows, n_rows, b);
  const int64_t row0 = (int64_t)(in_row < 0 ? 0 : in_row) * k;

  // The light launch keeps the strings next to the run ends, so kept
  // nodes take their tokens from LDS.
  constexpr bool kSepE = NT < 1024;
  const uint16_t root_tok = ctx[(int64_t)b * L + L - 1];  // issued early, used at the end
  // Malformed rows (a row outside the map's range, a negative count or more
  // than k slots) count as T = 0 and are reported with num_nodes = -1.
  int T_raw = 0, bad = in_row < 0;
  int tk_s[FC_MAX_SOURCES] = {0, 0, 0, 0};
#pragma unroll
  for (int s = 0; s < FC_MAX_SOURCES; ++s) {
    if (s < S && in_row >= 0) {
      const int t = taken[(int64_t)in_row * S + s];
      tk_s[s] = t;
      bad |= t < 0;
      T_raw += t > 0 ? t : 0;
    }
  }
  bad |= T_raw > k;
  bad |= T_raw > t_hi;  // cannot happen: the light launch routes queries by T
  if (bad) T_raw = 0;

  const TreeLayout lay = tree_layout(t_hi, m, kSepE);
  uint16_t* str = (uint16_t*)(smem + lay.str);
  uint16_t* E = (uint16_t*)(smem + lay.E);
  uint32_t* A = (uint32_t*)(smem + lay.A);
  uint16_t* perm = (uint16_t*)(smem + lay.perm);
  uint8_t* len = smem + lay.len;
  uint8_t* lcp = smem + lay.lcp;
  uint8_t* mlen = smem + lay.mlen;

  if (tid == 0) {
    int acc = 0;
#pragma unroll
    for (int s = 0; s < FC_MAX_SOURCES; ++s) {
      if (s < S) {
        s_seg[s] = acc;
        acc += bad ? 0 : tk_s[s];
      }
    }
    s_seg[S] = acc;
    s_err = bad;
    s_pick[0] = 0;
    s_pick[1] = 0;
    s_pick[2] = 0;
  }
  for (int i = tid; i < 256; i += NT) s_hist[i] = 0;
  __syncthreads();
  const int T = T_raw;

  // At most one kept continuation: the tree is the chain of its first
  // min(len, c) tokens, every node of that store's weight alpha, so the
  // general passes are skipped (same rows, weights and mask).
  const int len0 = (!bad && T == 1) ? (int)cont_len[row0] : 0;
  if (!bad && T <= 1 && len0 <= m) {
    int s0 = 0;
#pragma unroll
    for (int s = FC_MAX_SOURCES - 1; s >= 0; --s)
      if (s < S && tk_s[s] > 0) s0 = s;
    const uint32_t a0 = alpha_of(alpha, s0);
    const int num = 1 + (len0 < c ? len0 : c);
    for (int r = tid; r < R; r += NT) {
      const int64_t o = (int64_t)b * R + r;
      node_tok[o] = r == 0 ? (int32_t)root_tok : (r < num ? (int32_t)cont_tok[row0 * m + r - 1] : 0);
      parent[o] = (r >= 1 && r < num) ? r - 1 : -1;
      weight[o] = r == 0 ? (len0 > 0 ? a0 : 0u) : (r < num ? a0 : 0u);
      pos_ids[o] = r < num ? r : 0;
    }
    const int64_t mb = (int64_t)b * R * R;
    int i = tid / R, j = tid - (tid / R) * R;
    const int di = NT / R, dj = NT - (NT / R) * R;
    for (int e = tid; e < R * R; e += NT) {
      mask[mb + e] = (i < num && j <= i) ? 1 : 0;
      i += di;
      j += dj;
      if (j >= R) {
        j -= R;
        ++i;
      }
    }
    if (tid == 0) num_nodes[b] = num;
    return;
  }
  // store boundaries in registers (no LDS round trip per lookup)
  const int seg1 = s_seg[1 < S ? 1 : S], seg2 = s_seg[2 < S ? 2 : S], seg3 = s_seg[3 < S ? 3 : S];
  auto store_of = [&](int i) -> int { return (S > 1 && i >= seg1) + (S > 2 && i >= seg2) + (S > 3 && i >= seg3); };
  // with one weight for every store the alpha prefix sum is linear
  const bool alpha_flat = NARROW || ((S < 2 || alpha.a[1] == alpha.a[0]) && (S < 3 || alpha.a[2] == alpha.a[0]) &&
                                     (S < 4 || alpha.a[3] == alpha.a[0]));
  const bool even_m = (m & 1) == 0;  // rows are 4-byte aligned in LDS
  auto rcmp = [&](int i, int j) -> int {
    return even_m ? row_cmp_w<MAXM / 2>(str + i * m, len[i], str + j * m, len[j])
                  : str_cmp(str + i * m, len[i], str + j * m, len[j]);
  };
  auto rlcp = [&](int i, int j) -> int {
    return even_m ? row_lcp_w<MAXM / 2>(str + i * m, len[i], str + j * m, len[j])
                  : str_lcp(str + i * m, len[i], str + j * m, len[j]);
  };

  // 1. load lengths and tokens (32-bit words when the rows are aligned)
  for (int i = tid; i < T; i += NT) {
    const uint8_t l = cont_len[row0 + i];
    len[i] = l;
    if (l > m) s_err = 1;
  }
  if (words == 2) {
    // 16-byte rows: 8 tokens per load, four loads in flight per thread
    const uint4* src = (const uint4*)(cont_tok + row0 * m);
    uint4* dst = (uint4*)str;
    const int nv = (T * m + 7) >> 3;
#pragma unroll 4
    for (int e = tid; e < nv; e += NT) dst[e] = src[e];
  } else if (words == 1) {
    const uint32_t* src = (const uint32_t*)(cont_tok + row0 * m);
    uint32_t* dst = (uint32_t*)str;
    const int nw = (T * m + 1) >> 1;
    for (int e = tid; e < nw; e += NT) dst[e] = src[e];
  } else {
    for (int e = tid; e < T * m; e += NT) str[e] = cont_tok[row0 * m + e];
  }
  __syncthreads();

  // 2. precondition (each store's slots sorted) and merged order
  for (int i = tid; i < T; i += NT) {
    const int s = store_of(i);
    const int first = s == 0 ? 0 : s == 1 ? seg1 : s == 2 ? seg2 : seg3;
    if (i > first && len[i - 1] <= m && len[i] <= m && rcmp(i - 1, i) > 0) s_err = 1;
  }
  const int per = (T + NT - 1) / NT;
  const int p0 = tid * per < T ? tid * per : T;
  const int p1 = p0 + per < T ? p0 + per : T;
  const int na = s_seg[1] - s_seg[0];
  if (S == 1) {
    for (int p = p0; p < p1; ++p) perm[p] = (uint16_t)p;
  } else if (S == 2 || s_seg[2] == T) {
    // merge path over two sorted lists (store 0 first on equal strings)
    const int nb = T - na;
    int lo = p0 - nb > 0 ? p0 - nb : 0;
    int hi = p0 < na ? p0 : na;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      const int jb = na + (p0 - mid - 1);
      if (rcmp(mid, jb) <= 0) lo = mid + 1; else hi = mid;
    }
    int ia = lo, ib = p0 - lo;
    for (int p = p0; p < p1; ++p) {
      bool take_a;
      if (ia >= na) take_a = false;
      else if (ib >= nb) take_a = true;
      else take_a = rcmp(ia, na + ib) <= 0;
      perm[p] = (uint16_t)(take_a ? ia++ : na + ib++);
    }
  } else {
    for (int i = tid; i < T; i += NT) {
      const int s = src_of(s_seg, S, i);
      const uint16_t* x = str + i * m;
      const int lx = len[i];
      int mp = i - s_seg[s];
      for (int s2 = 0; s2 < S; ++s2) {
        if (s2 == s) continue;
        int lo2 = s_seg[s2], hi2 = s_seg[s2 + 1];
        const int base = lo2;
        while (lo2 < hi2) {
          const int mid = (lo2 + hi2) >> 1;
          const int cc = even_m ? row_cmp_w<MAXM / 2>(str + mid * m, len[mid], x, lx)
                                : str_cmp(str + mid * m, len[mid], x, lx);
          if (s2 < s ? (cc <= 0) : (cc < 0)) lo2 = mid + 1; else hi2 = mid;
        }
        mp += lo2 - base;
      }
      perm[mp] = (uint16_t)i;
    }
  }
  __syncthreads();
  const bool err = s_err != 0;

  int nsel = 0;
  uint32_t root_w = 0;
  if (!err) {
    // 3. merged lengths, adjacent LCPs, alpha sums, node counts, and each
    //    chunk's first head per depth (first q with lcp[q] < d)
    uint32_t asum = 0, rw = 0, nodes = 0;
    uint16_t f[MAXM + 1];
#pragma unroll
    for (int d = 0; d <= MAXM; ++d) f[d] = (uint16_t)T;
    for (int p = p1 - 1; p >= p0; --p) {
      const int i = perm[p];
      const int li = len[i];
      const int l = p > 0 ? rlcp(perm[p - 1], i) : 0;
      mlen[p] = (uint8_t)li;
      lcp[p] = (uint8_t)l;
      const uint32_t a = alpha_of(alpha, store_of(i));
      asum += a;
      if (li > 0) rw += a;
      nodes += (uint32_t)(li - l);
#pragma unroll
      for (int d = 1; d <= MAXM; ++d)
        if (l < d) f[d] = (uint16_t)p;
    }
    uint32_t a_ex, dummy, a_tot, n_tot;
    Scan2<NT>::run(asum, nodes, s_x, s_y, &a_ex, &dummy, &a_tot, &n_tot, rw, s_z, &root_w);
    // first head after the chunk at every depth: minimum of f over later
    // chunks (DPP within the wave, then over the later waves)
    uint16_t nh[MAXM + 1];
#pragma unroll
    for (int d = 1; d <= MAXM; ++d) {
      uint32_t wave_min = (uint32_t)T;
      if (d <= m) nh[d] = (uint16_t)fc::wave_excl_suffix_min_u32(f[d], (uint32_t)T, &wave_min);
      if (lane == 0) s_wmin[w][d] = (uint16_t)wave_min;
    }
    __syncthreads();
    // one thread per (wave, depth): minimum over the later waves, every
    // load issued before any is used
    if (tid < NW * MAXM) {
      const int w0 = tid / MAXM, d0 = tid % MAXM + 1;
      uint32_t v = (uint32_t)T;
#pragma unroll
      for (int u = 0; u < NW; ++u) {
        const uint32_t x = s_wmin[u][d0];
        v = (u > w0 && x < v) ? x : v;
      }
      s_wsuf[w0][d0] = (uint16_t)v;
    }
    __syncthreads();
#pragma unroll
    for (int d = 1; d <= MAXM; ++d) {
      const uint32_t x = s_wsuf[w][d];
      if (d <= m && x < nh[d]) nh[d] = (uint16_t)x;
    }
    // alpha prefix sums (with one weight for every store they are
    // alpha * position and never stored)
    if (!alpha_flat) {
      uint32_t run = a_ex;
      for (int p = p0; p < p1; ++p) {
        A[p] = run;
        run += alpha_of(alpha, store_of(perm[p]));
      }
      if (tid == 0) A[T] = a_tot;
    }
    __syncthreads();  // in the heavy launch str is dead from here on: E reuses it
    // alpha weight of merged positions [p, e)
    auto wsum = [&](uint32_t e, uint32_t p) -> uint32_t {
      return alpha_flat ? alpha.a[0] * (e - p) : A[e] - A[p];
    };

    // 4. run ends, right to left through the chunk, with the weight
    //    histogram of the chunk's own nodes counted on the way.  The node
    //    weight is stored directly when every weight fits 16 bits (weights
    //    never exceed the root's); otherwise the run end is stored and the
    //    weight recomputed where needed.
    //    The histogram serves step 5: weights 1 and 2 (the bulk: unshared
    //    continuation tails) are counted in registers, other weights below
    //    256 with LDS atomics, heavier ones lumped.
    const bool wide = !NARROW && root_w > 0xFFFFu;
    {
      uint32_t r1 = 0, r2 = 0, rbig = 0;
      for (int q = p1 - 1; q >= p0; --q) {
        const int l = lcp[q], ml = mlen[q];
        const uint32_t aq = alpha_flat ? 0u : A[q];
#pragma unroll
        for (int d = 1; d <= MAXM; ++d) {
          if (d > l && d <= ml) {
            const uint32_t W = alpha_flat ? alpha.a[0] * ((uint32_t)nh[d] - (uint32_t)q) : A[nh[d]] - aq;
            E[q * m + d - 1] = wide ? nh[d] : (uint16_t)W;
            r1 += W == 1u ? 1u : 0u;
            r2 += W == 2u ? 1u : 0u;
            rbig += W >= 256u ? 1u : 0u;
            if (W != 1u && W != 2u && W < 256u) atomicAdd(&s_hist[W], 1u);
          }
          if (d > l) nh[d] = (uint16_t)q;
        }
      }
      const uint32_t x1 = fc::wave_sum_u32(r1), x2 = fc::wave_sum_u32(r2), xb = fc::wave_sum_u32(rbig);
      if (lane == 0 && x1) atomicAdd(&s_hist[1], x1);
      if (lane == 0 && x2) atomicAdd(&s_hist[2], x2);
      if (lane == 0 && xb) atomicAdd(&s_pick[2], xb);
    }
    __syncthreads();
    auto node_w = [&](int p, int d) -> uint32_t {
      const uint16_t e = E[p * m + d - 1];
      return wide ? wsum(e, (uint32_t)p) : (uint32_t)e;
    };
    // The weights of all depths of string p, fetched together (the depth
    // bound m is uniform, so every load issues before any is used); depths
    // that are not p's own nodes hold unused values.
    auto row_w = [&](int p, uint32_t (&wv)[MAXM + 1]) {
#pragma unroll
      for (int d = 1; d <= MAXM; ++d) wv[d] = d <= m ? (uint32_t)E[p * m + d - 1] : 0u;
      if (wide) {
#pragma unroll
        for (int d = 1; d <= MAXM; ++d) wv[d] = d <= m ? wsum(wv[d], (uint32_t)p) : 0u;
      }
    };

    // 5. the need-th largest weight W* and how many nodes of weight W* to
    //    take (in (p, d) order), from the histogram; only when W* itself is
    //    256 or more does a radix select over the (few) heavy nodes follow.
    const uint32_t need = n_tot < (uint32_t)c ? n_tot : (uint32_t)c;
    uint32_t prefix = 0, remaining = need;
    const uint32_t n_heavy = s_pick[2];
    if (need > 0 && n_heavy < need) {
      // W* < 256: wave 0 walks the histogram from the top
      if (tid < fc::kWave) {
        const uint32_t want = need - n_heavy;
        uint32_t cnt[4];
        uint32_t lsum = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          cnt[u] = s_hist[255 - (lane * 4 + u)];
          lsum += cnt[u];
        }
        const uint32_t incl = fc::wave_incl_sum_u32(lsum);
        const uint32_t before = incl - lsum;
        if (before < want && incl >= want) {
          uint32_t acc = before;
          int bin = 0;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (acc + cnt[u] >= want) {
              bin = 255 - (lane * 4 + u);
              break;
            }
            acc += cnt[u];
          }
          s_pick[0] = (uint32_t)bin;
          s_pick[1] = want - acc;
        }
      }
      __syncthreads();
      prefix = s_pick[0];
      remaining = s_pick[1];
    } else if (need > 0) {
      // W* >= 256: radix select over the heavy nodes only
      uint32_t wmax = 0;
      for (int p = p0; p < p1; ++p) {
        const int d = lcp[p] + 1;  // the shallowest own node is the heaviest
        if (d <= mlen[p]) {
          const uint32_t W = node_w(p, d);
          wmax = W > wmax ? W : wmax;
        }
      }
      wmax = fc::block_max<uint32_t>(wmax, s_z);
      int bits = 0;
      for (uint32_t x = wmax; x; x >>= 1) ++bits;
      for (int shift = ((bits - 1) / 8) * 8; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += NT) s_hist[i] = 0;
        __syncthreads();
        const uint64_t hi_mask = shift + 8 >= 32 ? 0ull : (uint64_t)prefix >> (shift + 8);
        for (int p = p0; p < p1; ++p) {
          for (int d = lcp[p] + 1; d <= mlen[p]; ++d) {
            const uint32_t W = node_w(p, d);
            if (W < 256) break;  // own nodes get lighter with depth
            if ((shift + 8 >= 32 ? 0ull : (uint64_t)(W >> (shift + 8))) == hi_mask)
              atomicAdd(&s_hist[(W >> shift) & 0xFF], 1u);
          }
        }
        __syncthreads();
        if (tid < fc::kWave) {
          uint32_t cnt[4];
          uint32_t lsum = 0;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            cnt[u] = s_hist[255 - (lane * 4 + u)];
            lsum += cnt[u];
          }
          const uint32_t incl = fc::wave_incl_sum_u32(lsum);
          const uint32_t before = incl - lsum;
          if (before < remaining && incl >= remaining) {
            uint32_t acc = before;
            int bin = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              if (acc + cnt[u] >= remaining) {
                bin = 255 - (lane * 4 + u);
                break;
              }
              acc += cnt[u];
            }
            s_pick[0] = prefix | ((uint32_t)bin << shift);
            s_pick[1] = remaining - acc;
          }
        }
        __syncthreads();
        prefix = s_pick[0];
        remaining = s_pick[1];
      }
    }
    const uint32_t wstar = prefix;
    const uint32_t take_eq = remaining;

    // 6. kept nodes in (p, d) order = preorder.  A string's own nodes get
    //    lighter with depth, so a string whose shallowest own node is below
    //    W* has none to keep and is passed over after one read.
    uint32_t gt = 0, eq = 0;
    if (need > 0) {
      for (int p = p0; p < p1; ++p) {
        const int l = lcp[p], ml = mlen[p];
        if (l >= ml || node_w(p, l + 1) < wstar) continue;
        uint32_t wv[MAXM + 1];
        row_w(p, wv);
#pragma unroll
        for (int d = 1; d <= MAXM; ++d) {
          const bool own = d > l && d <= ml;
          gt += (own && wv[d] > wstar) ? 1u : 0u;
          eq += (own && wv[d] == wstar) ? 1u : 0u;
        }
      }
    }
    uint32_t gt_ex, eq_ex, gt_tot, eq_tot;
    Scan2<NT>::run(gt, eq, s_x, s_y, &gt_ex, &eq_ex, &gt_tot, &eq_tot);
    if (need > 0 && (gt + eq) > 0) {
      uint32_t o = 1 + gt_ex + (eq_ex < take_eq ? eq_ex : take_eq);
      uint32_t r = eq_ex;
      for (int p = p0; p < p1; ++p) {
        const int l = lcp[p], ml = mlen[p];
        if (l >= ml || node_w(p, l + 1) < wstar) continue;
        uint32_t wv[MAXM + 1];
        row_w(p, wv);
#pragma unroll
        for (int d = 1; d <= MAXM; ++d) {
          if (d <= l || d > ml) continue;
          const uint32_t W = wv[d];
          bool keep = W > wstar;
          if (W == wstar) keep = r++ < take_eq;
          if (keep && o < (uint32_t)FC_MAX_TREE_ROWS) {
            s_sel_p[o] = (uint16_t)p;
            s_sel_d[o] = (uint8_t)d;
            s_sel_w[o] = W;
            if (kSepE) s_sel_t[o] = str[perm[p] * m + d - 1];
            ++o;
          }
        }
      }
    }
    const uint32_t total_sel = need > 0 ? gt_tot + (eq_tot < take_eq ? eq_tot : take_eq) : 0;
    nsel = (int)(total_sel < (uint32_t)c ? total_sel : (uint32_t)c);
    if (tid == 0) s_sel_d[0] = 0;
    __syncthreads();
    // Parent of row r: the last row before it one level shallower (rows are
    // in preorder and the kept set is ancestor-closed).  The first four
    // waves hold one row per lane and publish, per depth, a ballot of their
    // rows at that depth; row r then takes the highest such row below it,
    // in its own wave or else in the nearest earlier one.
    if (tid < FC_MAX_TREE_ROWS) {
      const int g = tid / fc::kWave;
      const int d = tid <= nsel ? (int)s_sel_d[tid] : -1;
#pragma unroll
      for (int D = 0; D < MAXM; ++D) {
        const uint64_t bl = fc::ballot(d == D);
        if (lane == 0) s_dball[g][D] = bl;
      }
    }
    __syncthreads();
    if (tid >= 1 && tid <= nsel) {
      const int g = tid / fc::kWave;
      const int D = (int)s_sel_d[tid] - 1;
      uint64_t bl = s_dball[g][D] & fc::lanemask_lt();
      int gg = g;
      while (bl == 0 && gg > 0) bl = s_dball[--gg][D];
      s_par[tid] = bl ? (int16_t)(gg * fc::kWave + 63 - __builtin_clzll(bl)) : (int16_t)0;
    }
    if (tid == 0) s_par[0] = -1;
    __syncthreads();
  }

  // 7. rows, then the mask.  Rows are in preorder and the kept set is
  //    ancestor-closed, so row j's subtree is the run of rows from j up to
  //    the next row at j's depth or shallower (end(j)), and A[i][j] = 1
  //    exactly when j <= i < end(j).
  const int num = err ? 0 : 1 + nsel;
  for (int r = tid; r < R; r += NT) {
    const int64_t out = (int64_t)b * R + r;
    int32_t tk = 0, pr = -1, ps = 0;
    uint32_t wt = 0;
    if (r < num) {
      if (r == 0) {
        tk = root_tok;
        wt = root_w;
      } else {
        const int p = s_sel_p[r];
        const int d = s_sel_d[r];
        tk = kSepE ? s_sel_t[r] : cont_tok[(row0 + perm[p]) * m + d - 1];
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
  // end(j) from one ballot per group of 64 rows and depth D of the rows at
  // depth <= D: the first such row after j, in j's group or a later one.
  for (int g = w; g * fc::kWave < num; g += NW) {
    const int r = g * fc::kWave + lane;
    const int d = r < num ? (int)s_sel_d[r] : MAXM + 1;
#pragma unroll
    for (int D = 0; D <= MAXM; ++D) {
      const uint64_t bl = fc::ballot(d <= D);
      if (lane == 0) s_shallow[g][D] = bl;
    }
  }
  __syncthreads();
  for (int r = tid; r < num; r += NT) {
    const int g = r / fc::kWave, d = s_sel_d[r];
    uint64_t bl = s_shallow[g][d] & ~((2ull << (r % fc::kWave)) - 1ull);  // rows after r in its group
    int gg = g;
    while (bl == 0 && (gg + 1) * fc::kWave < num) bl = s_shallow[++gg][d];
    s_end[r] = (int16_t)(bl ? gg * fc::kWave + __builtin_ctzll(bl) : num);
  }
  __syncthreads();
  // each thread owns one column j (NT >= R) and every (NT / R)-th row of it
  const int64_t mbase = (int64_t)b * R * R;
  const int col = tid % R, row_step = NT / R;
  if (tid / R < row_step) {
    const int end_j = col < num ? (int)s_end[col] : -1;
    for (int i = tid / R; i < R; i += row_step)
      mask[mbase + (int64_t)i * R + col] = (col <= i && i < end_j) ? 1 : 0;
  }
  if (tid == 0) num_nodes[b] = err ? -1 : num;
}

// ---------------------------------------------------------------------------
// Flat path (m <= 16, every query unless its short lists are too long).  One
// workgroup of kFlatThreads threads per query, and no continuation text in
// LDS except the strings of the query's short stores: every store but the
// one with the most kept slots (the long store), which in practice hold a
// handful of strings beside thousands.  The long store's strings stay in
// the retrieval output (L2-resident right after fc_retrieve) and are read
// once, coalesced:
//   1. each long string finds its place among the short strings by binary
//      search in LDS; its merged position is its own index plus that rank,
//      and its adjacent LCP comes from its neighbour in the long list (a
//      lane shuffle) or from the short string just before it;
//   2. the merged positions the long strings leave free are the short
//      strings', in their own merged order;
//   3. from the per-position LCP and length, the run ends, weights, top-c
//      selection and emission of the trie follow as in the fast path, with
//      every node weight recomputed from the per-depth next heads in each
//      pass instead of being stored (that array was k*m*2 bytes).
// LDS per query is then 3 bytes per kept slot plus the short strings, so two
// queries of the largest size share a CU.
// ---------------------------------------------------------------------------

constexpr int kFlatThreads = 512;
constexpr int kFlatWide = 1024;     // threads per query for batches of at most kFlatWideMaxB queries
constexpr int kFlatWideMaxB = 256;
// long-string rows in flight per lane: five for rows of up to 10 tokens (a
// 5,000-string list in two passes of a 512-thread workgroup), four for up to
// 16 (where a fifth would cost a wave per SIMD)
template <int MAXM>
constexpr int flat_rows() { return MAXM <= 10 ? 5 : 4; }
constexpr int kFlatShortCap = 256;  // short strings a query may keep in LDS
constexpr int kFlatList = 2048;     // shared trie nodes (two strings or more) listed in LDS

struct FlatLayout {
  size_t perm, lm, A, sstr, slen, sidx, sh_key, sh_w, total;
};

// Head bits (one 64-bit word per 64 merged positions and depth, positions
// 0..T) need every weight to be one store weight times a run length and one
// byte per position's (LCP, length); at most kHeadWords words per depth.
constexpr int kHeadWords = 192;
__host__ __device__ inline int head_words(int T) { return (T + 1 + 63) / 64; }
__host__ __device__ inline bool flat_masks(int k, int maxm, bool with_A) {
  return !with_A && maxm <= 15 && head_words(k) <= kHeadWords;
}

// maxm: the instantiation's row width (rows of maxm/2 32-bit words);
// cap: short strings held; with_A: alpha prefix sums (stores of different
// weights); S > 2: the short strings' merged order needs its own index.
__host__ __device__ inline FlatLayout flat_layout(int k, int maxm, int cap, int S, bool with_A) {
  FlatLayout t;
  size_t o = 0;
  t.perm = o;  // k uint16: merged position -> slot
  o = align_up(o + (size_t)k * 2, 16);
  t.lm = o;  // k packed (lcp, merged length)
  o = align_up(o + (size_t)k * (maxm <= 15 ? 1 : 2), 16);
  t.A = o;  // k+1 uint32 alpha prefix sums
  if (with_A) o = align_up(o + (size_t)(k + 1) * 4, 16);
  t.sstr = o;  // cap rows of maxm/2 words; later the head bits, then the kept tail nodes
  const size_t rows = (size_t)cap * maxm * 2, tails = (size_t)FC_MAX_TREE_ROWS * 4;
  const size_t heads = flat_masks(k, maxm, with_A) ? (size_t)maxm * head_words(k) * 8 : 0;
  size_t region = rows > tails ? rows : tails;
  region = region > heads ? region : heads;
  o = align_up(o + region, 16);
  t.slen = o;  // cap uint8
  o = align_up(o + (size_t)cap, 16);
  t.sidx = o;  // cap uint16: short merged order -> LDS row
  if (S > 2) o = align_up(o + (size_t)cap * 2, 16);
  t.sh_key = o;  // shared trie nodes in (position, depth) order: position << 5 | depth
  o = align_up(o + (size_t)kFlatList * 4, 16);
  t.sh_w = o;  // their weights (16 bits when no weight can exceed them)
  o = align_up(o + (size_t)kFlatList * (with_A ? 4 : 2), 16);
  t.total = o;
  return t;
}

// Per-store kept slots of query q, their total, the store with the most
// slots (the lowest index on ties) and whether the row is malformed (outside
// the row map's range, a negative count, or more than k slots in all;
// malformed rows count as empty and are reported with num_nodes = -1).
struct QueryShape {
  int tk[FC_MAX_SOURCES];
  int T, longest, n_long;  // n_long = tk[longest]
  bool bad;
};

__device__ __forceinline__ QueryShape query_shape(const int32_t* __restrict__ taken, int S, int k,
                                                  const int32_t* __restrict__ rows, int n_rows, int q) {
  QueryShape r;
  const int row = fc::map_row(rows, n_rows, q);
  r.bad = row < 0;
  r.T = 0;
#pragma unroll
  for (int s = 0; s < FC_MAX_SOURCES; ++s) {
    r.tk[s] = (s < S && row >= 0) ? taken[(int64_t)row * S + s] : 0;
    r.bad |= r.tk[s] < 0;
    r.T += r.tk[s] > 0 ? r.tk[s] : 0;
  }
  r.bad |= r.T > k;
  if (r.bad) {
#pragma unroll
    for (int s = 0; s < FC_MAX_SOURCES; ++s) r.tk[s] = 0;
    r.T = 0;
  }
  r.longest = 0;
  r.n_long = r.tk[0];
#pragma unroll
  for (int s = 1; s < FC_MAX_SOURCES; ++s)
    if (r.tk[s] > r.n_long) r.longest = s, r.n_long = r.tk[s];
  return r;
}

// Tokens [0, len) of a continuation row as MAXM/2 words (token 2x in the
// low half of word x), zero past len.
template <int MAXM>
__device__ __forceinline__ void load_row_words(const uint16_t* __restrict__ src, int m, int len, bool words,
                                               uint32_t (&v)[MAXM / 2]) {
  if (words) {
    const uint32_t* s32 = (const uint32_t*)src;
#pragma unroll
    for (int x = 0; x < MAXM / 2; ++x) v[x] = 2 * x < m ? s32[x] : 0u;
  } else {
#pragma unroll
    for (int x = 0; x < MAXM / 2; ++x) {
      const uint32_t a = 2 * x < m ? src[2 * x] : 0u;
      const uint32_t b = 2 * x + 1 < m ? src[2 * x + 1] : 0u;
      v[x] = a | (b << 16);
    }
  }
#pragma unroll
  for (int x = 0; x < MAXM / 2; ++x)
    v[x] &= (2 * x < len ? 0xFFFFu : 0u) | (2 * x + 1 < len ? 0xFFFF0000u : 0u);
}

// LCP and order of two word rows (zero past their lengths).
template <int W>
__device__ __forceinline__ int lcp_words(const uint32_t (&a)[W], int la, const uint32_t (&b)[W], int lb) {
  const int n = la < lb ? la : lb;
  int first = 2 * W;
#pragma unroll
  for (int j = W - 1; j >= 0; --j) {
    const uint32_t d = a[j] ^ b[j];
    if (d) first = 2 * j + ((d & 0xFFFFu) == 0 ? 1 : 0);
  }
  return first < n ? first : n;
}

template <int W>
__device__ __forceinline__ int cmp_words(const uint32_t (&a)[W], int la, const uint32_t (&b)[W], int lb) {
  const int x = lcp_words<W>(a, la, b, lb);
  const int n = la < lb ? la : lb;
  if (x < n) {
    uint32_t wa = 0, wb = 0;
#pragma unroll
    for (int j = 0; j < W; ++j)
      if (j == (x >> 1)) wa = a[j], wb = b[j];
    const uint32_t ta = (x & 1) ? wa >> 16 : wa & 0xFFFFu, tb = (x & 1) ? wb >> 16 : wb & 0xFFFFu;
    return ta < tb ? -1 : 1;
  }
  return la < lb ? -1 : (la > lb ? 1 : 0);
}

// A continuation row and its length straight from the retrieval output (the
// rare case of a short list too long for LDS).
template <int MAXM>
__device__ __forceinline__ int global_row(const uint16_t* __restrict__ cont_tok,
                                                    const uint8_t* __restrict__ cont_len, int64_t slot, int m,
                                                    int words, uint32_t (&v)[MAXM / 2]) {
  int len = cont_len[slot];
  len = len < m ? len : m;
  load_row_words<MAXM>(cont_tok + slot * m, m, len, words != 0, v);
  return len;
}

template <int W>
__device__ __forceinline__ void lds_row(const uint32_t* __restrict__ sstr, int ci, uint32_t (&v)[W]) {
#pragma unroll
  for (int x = 0; x < W; ++x) v[x] = sstr[ci * W + x];
}

// Strings of the LDS rows [lo, hi) that precede string (v, len) in merged
// order: those <= it when their store comes first on ties (upper), those
// < it otherwise.
template <int W, typename Row>
__device__ __forceinline__ int count_before(Row row, int lo, int hi, const uint32_t (&v)[W], int len, bool upper) {
  const int base = lo;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    uint32_t r[W];
    const int rl = row(mid, r);
    const int cc = cmp_words<W>(r, rl, v, len);
    if (upper ? cc <= 0 : cc < 0) lo = mid + 1; else hi = mid;
  }
  return lo - base;
}

// The flat kernel's workgroup order: queries of 2,048 kept slots or more
// first, then those above 256, then the rest, each class in query order, so
// that the first round of workgroups spreads the heaviest queries over the
// CUs instead of letting a few CUs draw several.  With three stores or more,
// the queries whose short lists exceed the flat layout (cap) come last and
// are also listed for the full-LDS kernel.
constexpr int kPlanThreads = 1024;

__global__ void __launch_bounds__(kPlanThreads) k_tree_plan(const int32_t* __restrict__ taken, int S, int k,
                                                           const int32_t* __restrict__ rows, int n_rows, int B,
                                                           int cap, int32_t* __restrict__ order,
                                                           int32_t* __restrict__ defer_list,
                                                           int32_t* __restrict__ defer_count) {
  constexpr int NT = kPlanThreads;
  constexpr int NW = NT / fc::kWave;
  __shared__ uint32_t s_x[NW + 1], s_y[NW + 1];
  const int tid = threadIdx.x;
  auto cls = [&](int q) -> int {
    const QueryShape qs = query_shape(taken, S, k, rows, n_rows, q);
    if (S > 2 && !qs.bad && qs.T - qs.n_long > cap) return 3;
    return qs.T >= 2048 ? 0 : qs.T > 256 ? 1 : 2;
  };
  const int per = (B + NT - 1) / NT;
  const int q0 = tid * per < B ? tid * per : B;
  const int q1 = q0 + per < B ? q0 + per : B;
  uint32_t n[4] = {0, 0, 0, 0};
  for (int q = q0; q < q1; ++q) {
    const int c = cls(q);
    n[0] += c == 0;
    n[1] += c == 1;
    n[2] += c == 2;
    n[3] += c == 3;
  }
  uint32_t e[4], t[4];
  Scan2<NT>::run(n[0], n[1], s_x, s_y, &e[0], &e[1], &t[0], &t[1]);
  Scan2<NT>::run(n[2], n[3], s_x, s_y, &e[2], &e[3], &t[2], &t[3]);
  uint32_t o[4] = {e[0], t[0] + e[1], t[0] + t[1] + e[2], t[0] + t[1] + t[2] + e[3]};
  uint32_t d = e[3];
  for (int q = q0; q < q1; ++q) {
    const int c = cls(q);
    const uint32_t at = c == 0 ? o[0]++ : c == 1 ? o[1]++ : c == 2 ? o[2]++ : o[3]++;
    order[at] = q;
    if (c == 3 && defer_list) defer_list[d++] = q;
  }
  if (tid == 0 && defer_count) *defer_count = (int32_t)t[3];
}

template <int MAXM, bool NARROW, int NT_ = kFlatThreads>
__global__ void __launch_bounds__(NT_, NT_ == kFlatThreads && MAXM <= 10 ? 6 : 4) k_tree_flat(const int32_t* __restrict__ taken,
                                                            const uint8_t* __restrict__ cont_len,
                                                            const uint16_t* __restrict__ cont_tok,
                                                            const uint16_t* __restrict__ ctx, int L, int S, int k,
                                                            int m, int c, Alpha alpha, int cap, int words,
                                                            const int32_t* __restrict__ order, int self_plan, int B,
                                                            const int32_t* __restrict__ rows, int n_rows,
                                                            int32_t* __restrict__ num_nodes,
                                                            int32_t* __restrict__ node_tok,
                                                            int32_t* __restrict__ parent, uint32_t* __restrict__ weight,
                                                            int32_t* __restrict__ pos_ids, int32_t* __restrict__ mask) {
  constexpr int NT = NT_;
  constexpr int NW = NT / fc::kWave;
  constexpr int W = MAXM / 2;
  using LMT = typename std::conditional<(MAXM <= 15), uint8_t, uint16_t>::type;
  using SWT = typename std::conditional<NARROW, uint16_t, uint32_t>::type;  // NARROW: every weight < 2^16
  constexpr int kSh = MAXM <= 15 ? 4 : 8;
  constexpr uint32_t kLo = (1u << kSh) - 1u;
  static_assert(NT >= FC_MAX_TREE_ROWS, "one thread per tree row");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int s_seg[FC_MAX_SOURCES + 1];
  __shared__ int s_cs[FC_MAX_SOURCES + 1];
  __shared__ int s_err;
  __shared__ uint32_t s_x[NW + 1], s_y[NW + 1], s_z[NW + 1];
  __shared__ uint16_t s_wmin[NW][MAXM + 1];
  __shared__ uint16_t s_wsuf[NW][MAXM + 1];
  __shared__ uint32_t s_hist[256];
  __shared__ uint32_t s_sel_w[FC_MAX_TREE_ROWS];
  __shared__ uint16_t s_sel_p[FC_MAX_TREE_ROWS];
  __shared__ uint8_t s_sel_d[FC_MAX_TREE_ROWS];
  __shared__ int16_t s_par[FC_MAX_TREE_ROWS];
  __shared__ uint64_t s_dball[FC_MAX_TREE_ROWS / fc::kWave][MAXM];
  __shared__ uint64_t s_shallow[FC_MAX_TREE_ROWS / fc::kWave][MAXM + 1];
  __shared__ int16_t s_end[FC_MAX_TREE_ROWS];
  __shared__ uint32_t s_pick[3];
  __shared__ uint32_t s_scan4[4 * NW];
  __shared__ uint64_t s_nzw[MAXM][kHeadWords / 64];  // per depth: which head words are non-empty
  __shared__ int16_t s_runj[kFlatShortCap];  // first short string of a run: long strings before it (else -1)
  __shared__ uint8_t s_plcp[kFlatShortCap];  // and its LCP with the long string just before it

  const int tid = threadIdx.x;
  const int lane = fc::lane_id();
  const int w = tid / fc::kWave;
  // with three stores or more, short lists past the LDS cap go to the
  // full-LDS kernel; with two, they are searched in place (slower, rare)
  auto deferred = [&](const QueryShape& qs) { return S > 2 && !qs.bad && qs.T - qs.n_long > cap; };
  // this workgroup's query: from the planning launch's order, from the same
  // order worked out here (self_plan: every workgroup classifies the batch,
  // scans the class counts and picks the query at its own position, which
  // saves the planning launch when nothing is deferred), or by index
  __shared__ int s_self_b;
  int b = (int)blockIdx.x;
  if (order) {
    b = order[blockIdx.x];
  } else if (self_plan) {
    // a thread's queries: the first kPlanRegs classes are kept in registers
    // (all loads issued at once), later ones are classified again
    constexpr int kPlanRegs = 4;
    const int per = (B + NT - 1) / NT;
    const int q0 = (int)threadIdx.x * per < B ? (int)threadIdx.x * per : B;
    const int q1 = q0 + per < B ? q0 + per : B;
    auto cls = [&](int q) {
      const int T2 = query_shape(taken, S, k, rows, n_rows, q).T;
      return T2 >= 2048 ? 0 : T2 > 256 ? 1 : 2;
    };
    int creg[kPlanRegs];
#pragma unroll
    for (int i = 0; i < kPlanRegs; ++i) creg[i] = q0 + i < q1 ? cls(q0 + i) : 3;
    uint32_t n0 = 0, n1 = 0;
#pragma unroll
    for (int i = 0; i < kPlanRegs; ++i) {
      n0 += creg[i] == 0;
      n1 += creg[i] == 1;
    }
    for (int q = q0 + kPlanRegs; q < q1; ++q) {
      const int cq = cls(q);
      n0 += cq == 0;
      n1 += cq == 1;
    }
    const uint32_t n2 = (uint32_t)(q1 - q0) - n0 - n1;
    if (threadIdx.x == 0) s_self_b = (int)blockIdx.x;  // overwritten below: every position has one query
    uint32_t e0, e1, t0, t1;
    Scan2<NT>::run(n0, n1, s_x, s_y, &e0, &e1, &t0, &t1);
    const uint32_t e2 = (uint32_t)q0 - e0 - e1;  // queries before q0 of class 2
    const uint32_t pos = blockIdx.x;
    const int want = pos < t0 ? 0 : (pos < t0 + t1 ? 1 : 2);
    const uint32_t r = want == 0 ? pos : (want == 1 ? pos - t0 : pos - t0 - t1);
    const uint32_t e = want == 0 ? e0 : (want == 1 ? e1 : e2);
    const uint32_t nn = want == 0 ? n0 : (want == 1 ? n1 : n2);
    if (r >= e && r < e + nn) {
      uint32_t seen = e;
      for (int q = q0; q < q1; ++q) {
        int cq = 0;
#pragma unroll
        for (int i = 0; i < kPlanRegs; ++i)
          if (q == q0 + i) cq = creg[i];
        if (q >= q0 + kPlanRegs) cq = cls(q);
        if (cq != want) continue;
        if (seen == r) {
          s_self_b = q;
          break;
        }
        ++seen;
      }
    }
    __syncthreads();
    b = s_self_b;
  }
  const QueryShape qs = query_shape(taken, S, k, rows, n_rows, b);
  if (deferred(qs)) return;
  const int R = c + 1;
  const int in_row = fc::map_row(rows, n_rows, b);
  const int64_t row0 = (int64_t)(in_row < 0 ? 0 : in_row) * k;
  const uint16_t root_tok = ctx[(int64_t)b * L + L - 1];  // issued early, used at the end
  const int T = qs.T;
  const int sL = qs.longest;
  const int nL = qs.n_long;
  const int n_short = T - nL;

  if (tid == 0) {
    int acc = 0, cacc = 0;
#pragma unroll
    for (int s = 0; s < FC_MAX_SOURCES; ++s) {
      if (s < S) {
        s_seg[s] = acc;
        s_cs[s] = cacc;
        acc += qs.tk[s];
        cacc += s == sL ? 0 : qs.tk[s];
      }
    }
    s_seg[S] = acc;
    s_cs[S] = cacc;
    s_err = qs.bad;
    s_pick[0] = 0;
    s_pick[1] = 0;
    s_pick[2] = 0;
  }
  for (int i = tid; i < 256; i += NT) s_hist[i] = 0;
  __syncthreads();

  // At most one kept continuation: the tree is the chain of its first
  // min(len, c) tokens, every node of that store's weight alpha.
  const int len0 = (!qs.bad && T == 1) ? (int)cont_len[row0] : 0;
  if (!qs.bad && T <= 1 && len0 <= m) {
    int s0 = 0;
#pragma unroll
    for (int s = FC_MAX_SOURCES - 1; s >= 0; --s)
      if (s < S && qs.tk[s] > 0) s0 = s;
    const uint32_t a0 = alpha_of(alpha, s0);
    const int num = 1 + (len0 < c ? len0 : c);
    for (int r = tid; r < R; r += NT) {
      const int64_t o = (int64_t)b * R + r;
      node_tok[o] = r == 0 ? (int32_t)root_tok : (r < num ? (int32_t)cont_tok[row0 * m + r - 1] : 0);
      parent[o] = (r >= 1 && r < num) ? r - 1 : -1;
      weight[o] = r == 0 ? (len0 > 0 ? a0 : 0u) : (r < num ? a0 : 0u);
      pos_ids[o] = r < num ? r : 0;
    }
    const int64_t mb = (int64_t)b * R * R;
    int i = tid / R, j = tid - (tid / R) * R;
    const int di = NT / R, dj = NT - (NT / R) * R;
    for (int e = tid; e < R * R; e += NT) {
      mask[mb + e] = (i < num && j <= i) ? 1 : 0;
      i += di;
      j += dj;
      if (j >= R) {
        j -= R;
        ++i;
      }
    }
    if (tid == 0) num_nodes[b] = num;
    return;
  }

  const FlatLayout lay = flat_layout(k, MAXM, cap, S, !NARROW);
  uint16_t* perm = (uint16_t*)(smem + lay.perm);
  LMT* lm = (LMT*)(smem + lay.lm);
  uint32_t* A = (uint32_t*)(smem + lay.A);
  uint32_t* sstr = (uint32_t*)(smem + lay.sstr);
  uint8_t* slen = smem + lay.slen;
  uint16_t* sidx = (uint16_t*)(smem + lay.sidx);
  const int seg1 = s_seg[1 < S ? 1 : S], seg2 = s_seg[2 < S ? 2 : S], seg3 = s_seg[3 < S ? 3 : S];
  auto store_of = [&](int slot) -> int {
    return (S > 1 && slot >= seg1) + (S > 2 && slot >= seg2) + (S > 3 && slot >= seg3);
  };
  // the short store of LDS row ci, and that row's slot
  auto short_store = [&](int ci) -> int {
    int s = 0;
#pragma unroll
    for (int u = 0; u < FC_MAX_SOURCES; ++u)
      if (u < S && u != sL && ci >= s_cs[u] && ci < s_cs[u] + qs.tk[u]) s = u;
    return s;
  };
  auto short_slot = [&](int ci) -> int {
    const int s = short_store(ci);
    return s_seg[s] + (ci - s_cs[s]);
  };
  const bool alpha_flat = NARROW || ((S < 2 || alpha.a[1] == alpha.a[0]) && (S < 3 || alpha.a[2] == alpha.a[0]) &&
                                     (S < 4 || alpha.a[3] == alpha.a[0]));
  // short string ci (its row as words and its length): from LDS, or, past
  // the cap (two stores only), from the retrieval output itself
  const bool in_lds = n_short <= cap;
  auto srow = [&](int ci, uint32_t (&v)[W]) -> int {
    if (in_lds) {
      lds_row<W>(sstr, ci, v);
      return slen[ci];
    }
    return global_row<MAXM>(cont_tok, cont_len, row0 + short_slot(ci), m, words, v);
  };

  // 1. the short strings into LDS, each store's order checked; with three
  //    or more stores, their merged order among themselves.  Free merged
  //    positions are marked only for the gap pass (short strings read in
  //    place, or no long strings); with no short string at all the pass is
  //    skipped, barriers included.
  if (n_short > 0 && !(in_lds && nL > 0))
    for (int p = tid; p < T; p += NT) perm[p] = 0xFFFF;
  for (int g = tid; g < n_short && g < kFlatShortCap; g += NT) s_runj[g] = -1;
  if (S > 2)
    for (int g = tid; g < n_short; g += NT) sidx[g] = 0;  // every entry valid even if unsorted input collides
  for (int ci = tid; ci < n_short; ci += NT) {
    const int slot = short_slot(ci);
    int len = cont_len[row0 + slot];
    if (len > m) s_err = 1;
    if (!in_lds) continue;
    len = len < m ? len : m;
    uint32_t v[W];
    load_row_words<MAXM>(cont_tok + (row0 + slot) * m, m, len, words != 0, v);
#pragma unroll
    for (int x = 0; x < W; ++x) sstr[ci * W + x] = v[x];
    slen[ci] = (uint8_t)len;
  }
  if (n_short > 0) __syncthreads();
  for (int ci = tid; ci < n_short; ci += NT) {
    const int s = short_store(ci);
    const int i = ci - s_cs[s];
    uint32_t v[W];
    const int len = srow(ci, v);
    if (i > 0) {
      uint32_t pv[W];
      const int plen = srow(ci - 1, pv);
      if (cmp_words<W>(pv, plen, v, len) > 0) s_err = 1;
    }
    if (S > 2) {
      int pos = i;
#pragma unroll
      for (int u = 0; u < FC_MAX_SOURCES; ++u)
        if (u < S && u != sL && u != s && qs.tk[u] > 0)
          pos += count_before<W>(srow, s_cs[u], s_cs[u] + qs.tk[u], v, len, u < s);
      sidx[pos] = (uint16_t)ci;
    }
  }
  if (n_short > 0) __syncthreads();

  // 2. long strings: rank among the short strings, merged position, LCP
  //    with the merged predecessor when that is long (its neighbour in the
  //    long list) or the short string just before.  Each wave takes 63
  //    consecutive long strings per pass and its lane 0 the string before
  //    them, so every predecessor comes from the lane below; kFlatRows
  //    passes have their loads in flight together.
  auto lds_srow = [&](int ci, uint32_t (&v)[W]) -> int {
    lds_row<W>(sstr, ci, v);
    return slen[ci];
  };
  const int lslot0 = s_seg[sL];
  constexpr int kPass = NW * (fc::kWave - 1);  // long strings per pass of the block
  // one pass over the long strings with the short strings read through
  // `row` (compiled twice, so the common LDS case carries no registers of
  // the in-place one)
  auto long_pass = [&](auto&& row) {
    auto rank_short = [&](const uint32_t (&v)[W], int len) -> int {
      int r = 0;
#pragma unroll
      for (int u = 0; u < FC_MAX_SOURCES; ++u)
        if (u < S && u != sL && qs.tk[u] > 0) r += count_before<W>(row, s_cs[u], s_cs[u] + qs.tk[u], v, len, u < sL);
      return r;
    };
    // with every short string in LDS the long pass also places them
    const bool place = in_lds && n_short > 0;
    constexpr int kFlatRows = flat_rows<MAXM>();
    for (int j0 = 0; j0 < nL; j0 += kPass * kFlatRows) {
      uint32_t v[kFlatRows][W];
      int len[kFlatRows];
#pragma unroll
      for (int u = 0; u < kFlatRows; ++u) {
        const int j = j0 + u * kPass + w * (fc::kWave - 1) + lane - 1;
        len[u] = 0;
        if (j >= 0 && j < nL) {
          len[u] = cont_len[row0 + lslot0 + j];
          const uint16_t* src = cont_tok + (row0 + lslot0 + j) * m;
          if (words && m == MAXM) {
            // a full row: 16-byte loads (dword-aligned) plus single words
            const uint32_t* s32 = (const uint32_t*)src;
#pragma unroll
            for (int x = 0; x + 4 <= W; x += 4) {
              const fc::u32x4_a4 q4 = *(const fc::u32x4_a4*)(s32 + x);
              v[u][x] = q4.x;
              v[u][x + 1] = q4.y;
              v[u][x + 2] = q4.z;
              v[u][x + 3] = q4.w;
            }
#pragma unroll
            for (int x = W / 4 * 4; x < W; ++x) v[u][x] = s32[x];
          } else if (words) {
            const uint32_t* s32 = (const uint32_t*)src;
#pragma unroll
            for (int x = 0; x < W; ++x) v[u][x] = 2 * x < m ? s32[x] : 0u;
          } else {
#pragma unroll
            for (int x = 0; x < W; ++x) {
              const uint32_t a0 = 2 * x < m ? src[2 * x] : 0u;
              const uint32_t a1 = 2 * x + 1 < m ? src[2 * x + 1] : 0u;
              v[u][x] = a0 | (a1 << 16);
            }
          }
        } else {
#pragma unroll
          for (int x = 0; x < W; ++x) v[u][x] = 0u;
        }
      }
#pragma unroll
      for (int u = 0; u < kFlatRows; ++u) {
        const int j = j0 + u * kPass + w * (fc::kWave - 1) + lane - 1;
        const bool have = j >= 0 && j < nL;
        if (have && len[u] > m) s_err = 1;
        const int ln = len[u] < m ? len[u] : m;
#pragma unroll
        for (int x = 0; x < W; ++x) v[u][x] &= (2 * x < ln ? 0xFFFFu : 0u) | (2 * x + 1 < ln ? 0xFFFF0000u : 0u);
        const int r = have && n_short > 0 ? rank_short(v[u], ln) : 0;
        uint32_t pv[W];
#pragma unroll
        for (int x = 0; x < W; ++x) pv[x] = fc::wave_shr1(v[u][x], 0u);
        const int plen = (int)fc::wave_shr1((uint32_t)ln, 0u);
        const int pr = (int)fc::wave_shr1((uint32_t)r, 0u);
        if (have && lane > 0) {
          if (j > 0 && cmp_words<W>(pv, plen, v[u], ln) > 0) s_err = 1;
          int l = 0;
          if (j > 0 && pr == r) {
            l = lcp_words<W>(pv, plen, v[u], ln);
          } else if (r > 0) {
            const int ci = S > 2 ? (int)sidx[r - 1] : r - 1;
            uint32_t sv[W];
            const int sl = row(ci, sv);
            l = lcp_words<W>(sv, sl, v[u], ln);
          }
          const int P = j + r;
          perm[P] = (uint16_t)(lslot0 + j);
          lm[P] = (LMT)((uint32_t)l | ((uint32_t)ln << kSh));
          // a run of short strings merged right after long j - 1 (in short
          // order [pr, r); [0, r) before the first long) or after the last
          // long ([r, n_short)): the run's first string records the number
          // of long strings before it and its LCP with the long string just
          // before it, whose row is in registers here
          if (place) {
            if (j == 0 ? r > 0 : pr < r) {
              const int g = j == 0 ? 0 : pr;
              s_runj[g] = (int16_t)j;
              if (j > 0) {
                const int ci = S > 2 ? (int)sidx[g] : g;
                uint32_t sv[W];
                const int sl = lds_srow(ci, sv);
                s_plcp[g] = (uint8_t)lcp_words<W>(pv, plen, sv, sl);
              }
            }
            if (j == nL - 1 && r < n_short) {
              const int ci = S > 2 ? (int)sidx[r] : r;
              uint32_t sv[W];
              const int sl = lds_srow(ci, sv);
              s_runj[r] = (int16_t)nL;
              s_plcp[r] = (uint8_t)lcp_words<W>(v[u], ln, sv, sl);
            }
          }
        }
      }
    }
  };
  if (in_lds) long_pass(lds_srow);
  else long_pass([&](int ci, uint32_t (&v)[W]) -> int {
    return global_row<MAXM>(cont_tok, cont_len, row0 + short_slot(ci), m, words, v);
  });
  __syncthreads();

  // 3. the free merged positions take the short strings in order: with the
  //    short strings in LDS and long ones present, short g goes to g plus
  //    the long strings before its run (recorded by the long pass), one
  //    thread per short string; otherwise the chunks count their free
  //    positions and fill them
  const int per = (T + NT - 1) / NT;
  const int p0 = tid * per < T ? tid * per : T;
  const int p1 = p0 + per < T ? p0 + per : T;
  if (n_short > 0 && in_lds && nL > 0) {
    for (int g = tid; g < n_short; g += NT) {
      int st = g;
      while (st > 0 && s_runj[st] < 0) --st;
      const int jb = s_runj[st] < 0 ? 0 : (int)s_runj[st];
      const int ci = S > 2 ? (int)sidx[g] : g;
      uint32_t v[W];
      const int len = lds_srow(ci, v);
      int l = 0;
      if (st == g && jb > 0) {
        l = s_plcp[g];  // right after a long string
      } else if (g > 0) {
        const int pci = S > 2 ? (int)sidx[g - 1] : g - 1;
        uint32_t pv[W];
        const int pl = lds_srow(pci, pv);
        l = lcp_words<W>(pv, pl, v, len);
      }
      perm[g + jb] = (uint16_t)short_slot(ci);
      lm[g + jb] = (LMT)((uint32_t)l | ((uint32_t)len << kSh));
    }
  } else if (n_short > 0) {
    uint32_t gaps = 0;
    for (int p = p0; p < p1; ++p) gaps += perm[p] == 0xFFFF ? 1u : 0u;
    // the predecessor of the chunk, read before anything is rewritten
    const uint16_t before = p0 > 0 && p0 < p1 ? perm[p0 - 1] : (uint16_t)0;
    const uint32_t before_lm = p0 > 0 && p0 < p1 ? (uint32_t)lm[p0 - 1] : 0u;
    uint32_t g0, dummy, gtot, dummy2;
    Scan2<NT>::run(gaps, 0u, s_x, s_y, &g0, &dummy, &gtot, &dummy2);
    bool prev_gap = before == 0xFFFF;
    uint16_t prev_slot = before;
    uint32_t prev_len = before_lm >> kSh;
    for (int p = p0; p < p1; ++p) {
      const uint16_t cur = perm[p];
      if (cur != 0xFFFF) {
        prev_gap = false;
        prev_slot = cur;
        prev_len = (uint32_t)lm[p] >> kSh;
        continue;
      }
      const int g = (int)g0++;
      if (g >= n_short) {
        s_err = 1;  // only unsorted input can leave more free positions than short strings
        break;
      }
      const int ci = S > 2 ? (int)sidx[g] : g;
      uint32_t v[W];
      const int len = srow(ci, v);
      int l = 0;
      if (p > 0 && prev_gap) {
        const int pci = S > 2 ? (int)sidx[g - 1] : g - 1;
        uint32_t pv[W];
        const int pl = srow(pci, pv);
        l = lcp_words<W>(pv, pl, v, len);
      } else if (p > 0) {
        uint32_t pv[W];
        load_row_words<MAXM>(cont_tok + (row0 + prev_slot) * m, m, (int)prev_len, words != 0, pv);
        l = lcp_words<W>(pv, (int)prev_len, v, len);
      }
      const uint16_t slot = (uint16_t)short_slot(ci);
      perm[p] = slot;
      lm[p] = (LMT)((uint32_t)l | ((uint32_t)len << kSh));
      prev_gap = true;
      prev_slot = slot;
      prev_len = (uint32_t)len;
    }
  }
  __syncthreads();
  const bool err = s_err != 0;

  int nsel = 0;
  uint32_t root_w = 0;
  uint16_t row_tok = 0;  // this thread's kept row's token (row tid)
  if (!err) {
    // 4. chunk sums: alpha, non-empty strings (root weight), nodes, the
    //    chunk's shared nodes (depths past its own LCP, up to the next
    //    string's: they fix where the chunk's part of the list of shared
    //    nodes starts) and tail nodes (depths past both LCPs)
    const uint32_t a0 = alpha.a[0];
    uint32_t asum = 0, rw = 0, nodes = 0, nsh = 0, ntail = 0;
    int l_after = p1 < T ? (int)((uint32_t)lm[p1] & kLo) : 0;
    for (int p = p1 - 1; p >= p0; --p) {
      const uint32_t x = lm[p];
      const int l = (int)(x & kLo), li = (int)(x >> kSh);
      const uint32_t a = alpha_flat ? a0 : alpha_of(alpha, store_of(perm[p]));
      asum += a;
      if (li > 0) rw += a;
      nodes += (uint32_t)(li - l);
      const int top = li < l_after ? li : l_after;
      nsh += top > l ? (uint32_t)(top - l) : 0u;
      const int lo_t = l > l_after ? l : l_after;
      ntail += li > lo_t ? (uint32_t)(li - lo_t) : 0u;
      l_after = l;
    }
    // With one store weight, shared node (q, d) weighs alpha times the
    // distance from q to the next head of depth d (the next position whose
    // LCP is below d, or T).  Per depth, one bit per position says whether
    // it is a head (positions T and past are), so a node's weight is a bit
    // search instead of the chunk walk below ("direct").  A head word is
    // built by one thread from 64 (LCP, length) bytes, four at a time: with
    // the LCP in a byte's low nibble, adding 16 - d sets the byte's bit 4
    // exactly when LCP >= d.
    const int nwd = head_words(T);
    const bool direct = alpha_flat && flat_masks(k, MAXM, !NARROW) && m <= MAXM;
    uint64_t* heads = (uint64_t*)(smem + lay.sstr);
    if (direct) {
      if (tid < MAXM * (kHeadWords / 64)) (&s_nzw[0][0])[tid] = 0ull;
      __syncthreads();
      for (int x = tid; x < m * nwd; x += NT) {
        // consecutive threads take the depths of one word: same LDS bytes
        const int wd = x / m, d = x - (x / m) * m + 1;
        const uint4* src = (const uint4*)(lm + wd * 64);
        const uint32_t add = (uint32_t)(16 - d) * 0x01010101u;
        uint64_t hb = 0;
#pragma unroll
        for (int c4 = 0; c4 < 4; ++c4) {
          const uint4 v = src[c4];
          const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const uint32_t ge = (((wv[u] & 0x0F0F0F0Fu) + add) >> 4) & 0x01010101u;  // bit 8i: LCP_i >= d
            const uint32_t nib = (ge | (ge >> 7) | (ge >> 14) | (ge >> 21)) & 0xFu;
            hb |= (uint64_t)(~nib & 0xFu) << (16 * c4 + 4 * u);
          }
        }
        const int past = T - wd * 64;  // positions at or past T are heads
        if (past < 64) hb |= past <= 0 ? ~0ull : (~0ull << past);
        heads[(d - 1) * nwd + wd] = hb;
        if (hb != 0ull) atomicOr((unsigned long long*)&s_nzw[d - 1][wd >> 6], 1ull << (wd & 63));
      }
    }
    uint32_t a_ex, a_tot, n_tot, sh_ex, sh_tot;
    {
      const uint32_t v3[3] = {asum, nodes, nsh};
      uint32_t ex3[3], tot3[3];
      ScanK<NT, 3>::run(v3, rw, s_scan4, ex3, tot3, &root_w);
      a_ex = ex3[0];
      sh_ex = ex3[2];
      a_tot = tot3[0];
      n_tot = tot3[1];
      sh_tot = tot3[2];
    }
    const bool listed = sh_tot <= (uint32_t)kFlatList;

    // The walk's set-up, done once and only when a walk is needed: the next
    // head per depth after each chunk, and the alpha prefix sums of stores
    // of different weights.
    uint16_t nh[MAXM + 1];
    bool walk_ready = false;
    auto prepare_walk = [&]() {
      if (walk_ready) return;
      walk_ready = true;
      // the chunk's first head per depth (first q with lcp[q] < d), from
      // the LCPs again (not kept from the sums, whose hot path needs none)
      uint16_t f[MAXM + 1];
#pragma unroll
      for (int d = 0; d <= MAXM; ++d) f[d] = (uint16_t)T;
      for (int p = p1 - 1; p >= p0; --p) {
        const int l = (int)((uint32_t)lm[p] & kLo);
#pragma unroll
        for (int d = 1; d <= MAXM; ++d)
          if (l < d) f[d] = (uint16_t)p;
      }
#pragma unroll
      for (int d = 1; d <= MAXM; ++d) {
        uint32_t wave_min = (uint32_t)T;
        nh[d] = (uint16_t)T;
        if (d <= m) nh[d] = (uint16_t)fc::wave_excl_suffix_min_u32(f[d], (uint32_t)T, &wave_min);
        if (lane == 0) s_wmin[w][d] = (uint16_t)wave_min;
      }
      __syncthreads();
      if (tid < NW * MAXM) {
        const int w0 = tid / MAXM, d0 = tid % MAXM + 1;
        uint32_t v = (uint32_t)T;
#pragma unroll
        for (int u = 0; u < NW; ++u) {
          const uint32_t x = s_wmin[u][d0];
          v = (u > w0 && x < v) ? x : v;
        }
        s_wsuf[w0][d0] = (uint16_t)v;
      }
      __syncthreads();
#pragma unroll
      for (int d = 1; d <= MAXM; ++d) {
        const uint32_t x = s_wsuf[w][d];
        if (d <= m && x < nh[d]) nh[d] = (uint16_t)x;
      }
      if (!alpha_flat) {
        uint32_t run = a_ex;
        for (int p = p0; p < p1; ++p) {
          A[p] = run;
          run += alpha_of(alpha, store_of(perm[p]));
        }
        if (tid == 0) A[T] = a_tot;
        __syncthreads();
      }
    };
    // The own nodes of the chunk, right to left and deepest first (the
    // reverse of (p, d) order), with their weights: node (q, d) covers the
    // run from q to the next head of depth d.  Below the next string's LCP
    // (shared nodes, weight of two strings or more) the weight is that
    // difference; past it (the string's own tail) the run is q alone and the
    // weight is q's alpha, so tails are handed over as one range (tail(q,
    // d_lo, d_hi, w): depths d_lo < d <= d_hi) and shared nodes one by one
    // (shared(q, d, w)), tail first.  prepare_walk() must have run.
    auto walk = [&](auto&& tail, auto&& shared) {
      uint32_t h[MAXM + 1];
#pragma unroll
      for (int d = 1; d <= MAXM; ++d) h[d] = nh[d];
      int l_next = p1 < T ? (int)((uint32_t)lm[p1] & kLo) : 0;
      uint32_t a_next = alpha_flat ? 0u : A[p1];
      for (int q = p1 - 1; q >= p0; --q) {
        const uint32_t x = lm[q];
        const int l = (int)(x & kLo), ml = (int)(x >> kSh);
        const uint32_t aq = alpha_flat ? 0u : A[q];
        const uint32_t wq = alpha_flat ? a0 : a_next - aq;
        const int lo_t = l > l_next ? l : l_next;
        if (ml > lo_t) tail(q, lo_t, ml, wq);
        const int hi_s = ml < l_next ? ml : l_next;
#pragma unroll
        for (int d = MAXM; d >= 1; --d) {
          if (d > l && d <= hi_s) {
            const uint32_t Wt = alpha_flat ? a0 * (h[d] - (uint32_t)q) : A[h[d]] - aq;
            shared(q, d, Wt);
          }
        }
#pragma unroll
        for (int d = 1; d <= MAXM; ++d)
          if (d > l) h[d] = (uint32_t)q;
        l_next = l;
        a_next = aq;
      }
    };
    uint32_t* sh_key = (uint32_t*)(smem + lay.sh_key);
    SWT* sh_w = (SWT*)(smem + lay.sh_w);

    // 5. weight histogram: 1 and 2 (the bulk) in registers, other weights
    //    below 256 by LDS atomics, heavier ones only counted.  The shared
    //    nodes are listed in (position, depth) order with no atomics: each
    //    chunk fills its part of the list, which starts at its exclusive
    //    count.  Direct: each chunk lists its shared nodes, then every
    //    thread takes list entries one by one and finds their weights by
    //    bit search.  Otherwise the walk, which meets a chunk's shared nodes
    //    in reverse order, fills the chunk's part from its end with their
    //    weights, and with the list the weights are counted from it
    //    afterwards (so the walk has no LDS atomics to wait on).
    {
      uint32_t r1 = 0, r2 = 0, rbig = 0;
      auto count = [&](uint32_t Wt, uint32_t n) {
        r1 += Wt == 1u ? n : 0u;
        r2 += Wt == 2u ? n : 0u;
        rbig += Wt >= 256u ? n : 0u;
        if (Wt != 1u && Wt != 2u && Wt < 256u) atomicAdd(&s_hist[Wt], n);
      };
      if (direct && listed) {
        uint32_t o = sh_ex;
        uint32_t x = p0 < p1 ? (uint32_t)lm[p0] : 0u;
        for (int q = p0; q < p1; ++q) {
          const uint32_t xn = q + 1 < T ? (uint32_t)lm[q + 1] : 0u;
          const int l = (int)(x & kLo), ml = (int)(x >> kSh), ln = (int)(xn & kLo);
          const int hi = ml < ln ? ml : ln;
          for (int d = l + 1; d <= hi; ++d) sh_key[o++] = ((uint32_t)q << 5) | (uint32_t)d;
          x = xn;
        }
        count(a0, ntail);
        __syncthreads();
        // (q, d) with d <= lcp(q + 1): the next head of depth d is past q + 1
        for (uint32_t e = (uint32_t)tid; e < sh_tot; e += NT) {
          const uint32_t key = sh_key[e];
          const int q = (int)(key >> 5), d = (int)(key & 31u);
          const uint64_t* hd = heads + (d - 1) * nwd;
          const int p = q + 2;  // <= T: a shared node's string is not the last
          const int j = p >> 6;
          const uint64_t bits = hd[j] & (~0ull << (p & 63));
          int nxt;
          if (bits != 0ull) {
            nxt = (j << 6) + __builtin_ctzll(bits);
          } else {
            // the first non-empty word after j (word nwd - 1 holds position T)
            int j2 = -1;
#pragma unroll
            for (int c = kHeadWords / 64 - 1; c >= 0; --c) {
              const int lo_bit = c * 64;
              uint64_t z = s_nzw[d - 1][c];
              if (j + 1 > lo_bit) z = (j + 1 - lo_bit) >= 64 ? 0ull : z & (~0ull << (j + 1 - lo_bit));
              if (z != 0ull) j2 = lo_bit + __builtin_ctzll(z);
            }
            nxt = (j2 << 6) + __builtin_ctzll(hd[j2]);
          }
          const uint32_t Wt = a0 * (uint32_t)(nxt - q);
          sh_w[e] = (SWT)Wt;
          count(Wt, 1u);
        }
      } else {
        prepare_walk();
        uint32_t at = sh_ex + nsh;
        walk([&](int, int lo, int hi, uint32_t Wt) { count(Wt, (uint32_t)(hi - lo)); },
             [&](int q, int d, uint32_t Wt) {
               if (listed) {
                 --at;
                 sh_key[at] = ((uint32_t)q << 5) | (uint32_t)d;
                 sh_w[at] = (SWT)Wt;
               } else {
                 count(Wt, 1u);
               }
             });
        if (listed) {
          __syncthreads();
          const uint32_t pl = (sh_tot + NT - 1) / NT;
          const uint32_t e0 = (uint32_t)tid * pl < sh_tot ? (uint32_t)tid * pl : sh_tot;
          const uint32_t e1 = e0 + pl < sh_tot ? e0 + pl : sh_tot;
          for (uint32_t i = e0; i < e1; ++i) count((uint32_t)sh_w[i], 1u);
        }
      }
      const uint32_t x1 = fc::wave_sum_u32(r1), x2 = fc::wave_sum_u32(r2), xb = fc::wave_sum_u32(rbig);
      if (lane == 0 && x1) atomicAdd(&s_hist[1], x1);
      if (lane == 0 && x2) atomicAdd(&s_hist[2], x2);
      if (lane == 0 && xb) atomicAdd(&s_pick[2], xb);
    }
    __syncthreads();

    // 6. the need-th largest weight W* and how many nodes of weight W* to
    //    take (in (p, d) order)
    const uint32_t need = n_tot < (uint32_t)c ? n_tot : (uint32_t)c;
    uint32_t prefix = 0, remaining = need;
    const uint32_t n_heavy = s_pick[2];
    auto pick_bin = [&](uint32_t want, uint32_t base_prefix, int shift) {
      // wave 0: the bin holding the want-th largest, from the top
      if (tid < fc::kWave) {
        uint32_t cnt4[4];
        uint32_t lsum = 0;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          cnt4[u] = s_hist[255 - (lane * 4 + u)];
          lsum += cnt4[u];
        }
        const uint32_t incl = fc::wave_incl_sum_u32(lsum);
        const uint32_t before = incl - lsum;
        if (before < want && incl >= want) {
          uint32_t acc = before;
          int bin = 0;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (acc + cnt4[u] >= want) {
              bin = 255 - (lane * 4 + u);
              break;
            }
            acc += cnt4[u];
          }
          s_pick[0] = base_prefix | ((uint32_t)bin << shift);
          s_pick[1] = want - acc;
        }
      }
      __syncthreads();
    };
    if (need > 0 && n_heavy < need) {
      pick_bin(need - n_heavy, 0u, 0);
      prefix = s_pick[0];
      remaining = s_pick[1];
    } else if (need > 0) {
      // W* >= 256: radix select over the heavy nodes only
      prepare_walk();
      uint32_t wmax = 0;
      auto top = [&](uint32_t Wt) { wmax = Wt > wmax ? Wt : wmax; };
      walk([&](int, int, int, uint32_t Wt) { top(Wt); }, [&](int, int, uint32_t Wt) { top(Wt); });
      wmax = fc::block_max<uint32_t>(wmax, s_z);
      int bits = 0;
      for (uint32_t x = wmax; x; x >>= 1) ++bits;
      for (int shift = ((bits - 1) / 8) * 8; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += NT) s_hist[i] = 0;
        __syncthreads();
        const uint64_t hi_mask = shift + 8 >= 32 ? 0ull : (uint64_t)prefix >> (shift + 8);
        auto digit = [&](uint32_t Wt, uint32_t n) {
          if (n && Wt >= 256u && (shift + 8 >= 32 ? 0ull : (uint64_t)(Wt >> (shift + 8))) == hi_mask)
            atomicAdd(&s_hist[(Wt >> shift) & 0xFF], n);
        };
        walk([&](int, int lo, int hi, uint32_t Wt) { digit(Wt, (uint32_t)(hi - lo)); },
             [&](int, int, uint32_t Wt) { digit(Wt, 1u); });
        __syncthreads();
        pick_bin(remaining, prefix, shift);
        prefix = s_pick[0];
        remaining = s_pick[1];
      }
    }
    const uint32_t wstar = prefix;
    const uint32_t take_eq = remaining;

    // 7. kept nodes in (p, d) order = preorder.  The list of shared nodes
    //    (weight of two strings or more) is already in that order.  When
    //    every tail is lighter than W* (the usual case) the kept nodes are
    //    the listed ones heavier than W* and the first take_eq of weight W*:
    //    each thread counts both over a contiguous piece of the list, and
    //    one scan gives every kept node its row.  With one store weight and
    //    W* equal to it, every shared node is kept (its weight is at least
    //    twice that) and so are the first take_eq tail nodes in (p, d)
    //    order; the two ordered lists are merged by binary search.
    //    Otherwise (a list that did not fit) the chunks count their kept
    //    nodes in a walk and emit them in order.
    uint32_t tail_max = a0;
#pragma unroll
    for (int u = 1; u < FC_MAX_SOURCES; ++u)
      if (u < S && alpha.a[u] > tail_max) tail_max = alpha.a[u];
    const bool tails_eq = alpha_flat && a0 > 0 && wstar == a0;
    bool fast_emit = listed && need > 0 && (wstar > tail_max || tails_eq);
    if (fast_emit && !tails_eq) {
      const uint32_t pl = (sh_tot + NT - 1) / NT;
      const uint32_t e0 = (uint32_t)tid * pl < sh_tot ? (uint32_t)tid * pl : sh_tot;
      const uint32_t e1 = e0 + pl < sh_tot ? e0 + pl : sh_tot;
      uint32_t g = 0, e = 0;
      for (uint32_t i = e0; i < e1; ++i) {
        const uint32_t Wt = sh_w[i];
        g += Wt > wstar ? 1u : 0u;
        e += Wt == wstar ? 1u : 0u;
      }
      uint32_t gb, eb, gtot, etot;
      Scan2<NT>::run(g, e, s_x, s_y, &gb, &eb, &gtot, &etot);
      for (uint32_t i = e0; i < e1 && (g > 0 || eb < take_eq); ++i) {
        const uint32_t Wt = sh_w[i];
        uint32_t row = 0;
        if (Wt > wstar) {
          row = 1 + gb + (eb < take_eq ? eb : take_eq);
          ++gb;
          --g;
        } else if (Wt == wstar && eb < take_eq) {
          row = 1 + gb + eb;
          ++eb;
        }
        if (row > 0 && row < (uint32_t)FC_MAX_TREE_ROWS) {
          const uint32_t key = sh_key[i];
          s_sel_p[row] = (uint16_t)(key >> 5);
          s_sel_d[row] = (uint8_t)(key & 31u);
          s_sel_w[row] = Wt;
        }
      }
      nsel = (int)(need < (uint32_t)c ? need : (uint32_t)c);
    } else if (fast_emit) {
      // the first take_eq tail nodes, in (p, d) order: tails of position q
      // are the depths past both its own LCP and the next string's
      uint32_t* tail_key = (uint32_t*)(smem + lay.sstr);
      auto tails_of = [&](int q, int& lo, int& hi) {
        const uint32_t x = lm[q];
        const int l = (int)(x & kLo), ml = (int)(x >> kSh);
        const int ln = q + 1 < T ? (int)((uint32_t)lm[q + 1] & kLo) : 0;
        lo = l > ln ? l : ln;
        hi = ml;
      };
      uint32_t t_ex, dmy, t_tot, dmy2;
      Scan2<NT>::run(ntail, 0u, s_x, s_y, &t_ex, &dmy, &t_tot, &dmy2);  // the chunk's tails, counted in pass 4
      for (int q = p0; q < p1 && t_ex < take_eq; ++q) {
        int lo, hi;
        tails_of(q, lo, hi);
        for (int d = lo + 1; d <= hi && t_ex < take_eq; ++d, ++t_ex) tail_key[t_ex] = ((uint32_t)q << 5) | (uint32_t)d;
      }
      __syncthreads();
      // a listed node's row: its list index plus the kept tails before it;
      // a kept tail's: its index plus the listed nodes before it
      for (uint32_t i = (uint32_t)tid; i < sh_tot + take_eq; i += NT) {
        const bool is_tail = i >= sh_tot;
        const uint32_t j = is_tail ? i - sh_tot : i;
        const uint32_t key = is_tail ? tail_key[j] : sh_key[j];
        const uint32_t* other = is_tail ? sh_key : tail_key;
        uint32_t lo = 0, hi = is_tail ? sh_tot : take_eq;
        while (lo < hi) {
          const uint32_t mid = (lo + hi) >> 1;
          if (other[mid] < key) lo = mid + 1; else hi = mid;
        }
        const uint32_t row = 1 + j + lo;
        if (row < (uint32_t)FC_MAX_TREE_ROWS) {
          s_sel_p[row] = (uint16_t)(key >> 5);
          s_sel_d[row] = (uint8_t)(key & 31u);
          s_sel_w[row] = is_tail ? a0 : (uint32_t)sh_w[j];
        }
      }
      nsel = (int)(need < (uint32_t)c ? need : (uint32_t)c);
    } else {
      uint32_t gt = 0, eq = 0;
      prepare_walk();
      if (need > 0)
        walk(
            [&](int, int lo, int hi, uint32_t Wt) {
              gt += Wt > wstar ? (uint32_t)(hi - lo) : 0u;
              eq += Wt == wstar ? (uint32_t)(hi - lo) : 0u;
            },
            [&](int, int, uint32_t Wt) {
              gt += Wt > wstar ? 1u : 0u;
              eq += Wt == wstar ? 1u : 0u;
            });
      uint32_t gt_ex, eq_ex, gt_tot, eq_tot;
      Scan2<NT>::run(gt, eq, s_x, s_y, &gt_ex, &eq_ex, &gt_tot, &eq_tot);
      if (need > 0 && (gt + eq) > 0) {
        const uint32_t keq = take_eq > eq_ex ? (take_eq - eq_ex < eq ? take_eq - eq_ex : eq) : 0u;
        uint32_t o = 1 + gt_ex + (eq_ex < take_eq ? eq_ex : take_eq) + gt + keq;
        uint32_t eq_left = eq;
        auto emit = [&](int q, int d, uint32_t Wt) {
          bool keep = Wt > wstar;
          if (Wt == wstar) keep = --eq_left < keq;
          if (keep) {
            --o;
            if (o < (uint32_t)FC_MAX_TREE_ROWS) {
              s_sel_p[o] = (uint16_t)q;
              s_sel_d[o] = (uint8_t)d;
              s_sel_w[o] = Wt;
            }
          }
        };
        walk(
            [&](int q, int lo, int hi, uint32_t Wt) {
              if (Wt >= wstar)
                for (int d = hi; d > lo; --d) emit(q, d, Wt);
            },
            emit);
      }
      const uint32_t total_sel = need > 0 ? gt_tot + (eq_tot < take_eq ? eq_tot : take_eq) : 0;
      nsel = (int)(total_sel < (uint32_t)c ? total_sel : (uint32_t)c);
    }
    if (tid == 0) s_sel_d[0] = 0;
    __syncthreads();
    // the kept rows' tokens are loaded now and used when the rows are
    // written, so the load overlaps the parent search
    if (tid >= 1 && tid <= nsel) row_tok = cont_tok[(row0 + perm[s_sel_p[tid]]) * m + s_sel_d[tid] - 1];
    // 8. parent of row r: the last row before it one level shallower (rows
    //    are in preorder and the kept set is ancestor-closed), from per-depth
    //    ballots of the first four waves' rows
    if (tid < FC_MAX_TREE_ROWS) {
      const int g = tid / fc::kWave;
      const int d = tid <= nsel ? (int)s_sel_d[tid] : -1;
#pragma unroll
      for (int D = 0; D < MAXM; ++D) {
        const uint64_t bl = fc::ballot(d == D);
        if (lane == 0) s_dball[g][D] = bl;
      }
    }
    __syncthreads();
    if (tid >= 1 && tid <= nsel) {
      const int g = tid / fc::kWave;
      const int D = (int)s_sel_d[tid] - 1;
      uint64_t bl = s_dball[g][D] & fc::lanemask_lt();
      int gg = g;
      while (bl == 0 && gg > 0) bl = s_dball[--gg][D];
      s_par[tid] = bl ? (int16_t)(gg * fc::kWave + 63 - __builtin_clzll(bl)) : (int16_t)0;
    }
    if (tid == 0) s_par[0] = -1;
    __syncthreads();
  }

  // 9. rows, then the mask: row j's subtree is the run of rows from j up to
  //    the next row at j's depth or shallower, so A[i][j] = [j <= i < end(j)]
  const int num = err ? 0 : 1 + nsel;
  for (int r = tid; r < R; r += NT) {
    const int64_t out = (int64_t)b * R + r;
    int32_t tk = 0, pr = -1, ps = 0;
    uint32_t wt = 0;
    if (r < num) {
      if (r == 0) {
        tk = root_tok;
        wt = root_w;
      } else {
        const int p = s_sel_p[r];
        const int d = s_sel_d[r];
        tk = r == tid ? row_tok : cont_tok[(row0 + perm[p]) * m + d - 1];
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
  for (int g = w; g * fc::kWave < num; g += NW) {
    const int r = g * fc::kWave + lane;
    const int d = r < num ? (int)s_sel_d[r] : MAXM + 1;
#pragma unroll
    for (int D = 0; D <= MAXM; ++D) {
      const uint64_t bl = fc::ballot(d <= D);
      if (lane == 0) s_shallow[g][D] = bl;
    }
  }
  __syncthreads();
  for (int r = tid; r < num; r += NT) {
    const int g = r / fc::kWave, d = s_sel_d[r];
    uint64_t bl = s_shallow[g][d] & ~((2ull << (r % fc::kWave)) - 1ull);
    int gg = g;
    while (bl == 0 && (gg + 1) * fc::kWave < num) bl = s_shallow[++gg][d];
    s_end[r] = (int16_t)(bl ? gg * fc::kWave + __builtin_ctzll(bl) : num);
  }
  __syncthreads();
  const int64_t mbase = (int64_t)b * R * R;
  const int col = tid % R, row_step = NT / R;
  if (tid / R < row_step) {
    const int end_j = col < num ? (int)s_end[col] : -1;
    for (int i = tid / R; i < R; i += row_step)
      mask[mbase + (int64_t)i * R + col] = (col <= i && i < end_j) ? 1 : 0;
  }
  if (tid == 0) num_nodes[b] = err ? -1 : num;
}

// Per-device facts the launches need, looked up once per device: the LDS a
// workgroup may use, and each kernel's own static LDS (the dynamic limit of
// every kernel is raised once to what the device allows).
struct TreeDevice {
  bool ready = false;
  int max_lds = 0;
  size_t flat_static[2][2] = {{0, 0}, {0, 0}};  // [MAXM 10/16][NARROW]
  size_t wide_static[2] = {0, 0};                // the kFlatWide-thread flat kernel (MAXM 10), [NARROW]
  size_t full_static[2][2] = {{0, 0}, {0, 0}};  // the full-LDS kernel, same indexes
  size_t any_static = 0;
};

std::mutex g_tree_mu;
TreeDevice g_tree_dev[64];

template <typename K>
size_t raise_lds(K kernel, int max_lds) {
  hipFuncAttributes at{};
  if (hipFuncGetAttributes(&at, (const void*)kernel) != hipSuccess) {
    (void)hipGetLastError();
    return (size_t)max_lds;
  }
  const int dyn = max_lds - (int)at.sharedSizeBytes;
  if (dyn > 0) (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, dyn);
  (void)hipGetLastError();
  return at.sharedSizeBytes;
}

const TreeDevice* tree_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_tree_mu);
  TreeDevice& d = g_tree_dev[dev];
  if (!d.ready) {
    if (hipDeviceGetAttribute(&d.max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    d.flat_static[0][1] = raise_lds(k_tree_flat<10, true>, d.max_lds);
    d.flat_static[0][0] = raise_lds(k_tree_flat<10, false>, d.max_lds);
    d.flat_static[1][1] = raise_lds(k_tree_flat<16, true>, d.max_lds);
    d.flat_static[1][0] = raise_lds(k_tree_flat<16, false>, d.max_lds);
    d.wide_static[1] = raise_lds(k_tree_flat<10, true, kFlatWide>, d.max_lds);
    d.wide_static[0] = raise_lds(k_tree_flat<10, false, kFlatWide>, d.max_lds);
    raise_lds(k_tree_fast<256, 10, true>, d.max_lds);
    raise_lds(k_tree_fast<256, 10, false>, d.max_lds);
    raise_lds(k_tree_fast<256, 16, true>, d.max_lds);
    raise_lds(k_tree_fast<256, 16, false>, d.max_lds);
    d.full_static[0][1] = raise_lds(k_tree_fast<1024, 10, true>, d.max_lds);
    d.full_static[0][0] = raise_lds(k_tree_fast<1024, 10, false>, d.max_lds);
    d.full_static[1][1] = raise_lds(k_tree_fast<1024, 16, true>, d.max_lds);
    d.full_static[1][0] = raise_lds(k_tree_fast<1024, 16, false>, d.max_lds);
    d.any_static = raise_lds(k_tree_any, d.max_lds);
    d.ready = true;
  }
  return &d;
}

// Row loads of the two-launch path: 16-byte vectors when every query's
// block of rows is 16-byte aligned, else 32-bit words when 4-byte aligned,
// else single tokens.
int block_words(const uint16_t* cont_tok, int32_t k, int32_t m) {
  if ((((uintptr_t)cont_tok) & 15) == 0 && ((size_t)k * m) % 8 == 0) return 2;
  if ((((uintptr_t)cont_tok) & 3) == 0 && ((size_t)k * m) % 2 == 0) return 1;
  return 0;
}

template <int MAXM, bool NARROW>
fc_status launch_fast(const int32_t* taken, const uint8_t* cont_len, const uint16_t* cont_tok, const uint16_t* ctx,
                      int32_t B, int32_t L, int32_t S, int32_t k, int32_t m, fc_tree_params t, Alpha a,
                      const TreeLayout& full, int32_t* num_nodes, int32_t* node_tok, int32_t* parent,
                      uint32_t* weight, int32_t* pos_ids, int32_t* mask, const int32_t* rows, int32_t n_rows, void* ws,
                      hipStream_t stream) {
  // light queries (T <= 256) in small-LDS workgroups, the rest in full-LDS
  // ones, each launch walking its own list of queries
  const int t_small = k < kSmallClass ? k : kSmallClass;
  int32_t* lists = (int32_t*)ws;
  int32_t* counts = lists + 2 * (size_t)B;
  const int words = block_words(cont_tok, k, m);
  const TreeLayout small = tree_layout(t_small, m, true);
  (void)hipGetLastError();
  hipLaunchKernelGGL((k_tree_fast<256, MAXM, NARROW>), dim3(B + 1), dim3(256), small.total, stream, taken, cont_len,
                     cont_tok, ctx, L, S, k, m, t.c, a, nullptr, nullptr, lists + B, counts + 1, B, t_small, words,
                     rows, n_rows, num_nodes, node_tok, parent, weight, pos_ids, mask);
  FC_CHECK_LAUNCH();
  if (k > t_small) {
    hipLaunchKernelGGL((k_tree_fast<1024, MAXM, NARROW>), dim3(B), dim3(1024), full.total, stream, taken, cont_len,
                       cont_tok, ctx, L, S, k, m, t.c, a, lists + B, counts + 1, nullptr, nullptr, B, k, words, rows,
                       n_rows, num_nodes, node_tok, parent, weight, pos_ids, mask);
    FC_CHECK_LAUNCH();
  }
  return FC_OK;
}

// The flat path when its layout fits (with as many short strings as a query
// can have, or else as many as fit, the rest of the queries going to the
// full-LDS kernel through a list); returns FC_ERR_UNSUPPORTED when it does
// not apply, before launching anything.
template <int MAXM, bool NARROW>
fc_status launch_flat(const int32_t* taken, const uint8_t* cont_len, const uint16_t* cont_tok, const uint16_t* ctx,
                      int32_t B, int32_t L, int32_t S, int32_t k, int32_t m, fc_tree_params t, Alpha a,
                      const TreeLayout& full, const TreeDevice& dv, int32_t* num_nodes, int32_t* node_tok,
                      int32_t* parent, uint32_t* weight, int32_t* pos_ids, int32_t* mask, const int32_t* rows,
                      int32_t n_rows, void* ws, hipStream_t stream) {
  const size_t stat = dv.flat_static[MAXM == 10 ? 0 : 1][NARROW ? 1 : 0];
  if (stat >= (size_t)dv.max_lds) return FC_ERR_UNSUPPORTED;
  const size_t budget = (size_t)dv.max_lds - stat;
  const int worst_short = k - (k + S - 1) / S;  // the long store holds at least ceil(T / S)
  // LDS for every possible short list would cost occupancy for nothing (in
  // typical batches a second store's list holds a few strings)
  int cap = worst_short < kFlatShortCap ? worst_short : kFlatShortCap;
  while (cap > 0 && flat_layout(k, MAXM, cap, S, !NARROW).total > budget) cap = cap * 7 / 8;
  const FlatLayout lay = flat_layout(k, MAXM, cap, S, !NARROW);
  if (lay.total > budget) return FC_ERR_UNSUPPORTED;
  // with two stores a query's short list past the cap is searched in place;
  // with more, such queries go to the full-LDS kernel
  const bool defer = S > 2 && cap < worst_short;
  if (defer && full.total + dv.full_static[MAXM == 10 ? 0 : 1][NARROW ? 1 : 0] > (size_t)dv.max_lds)
    return FC_ERR_UNSUPPORTED;
  int32_t* order = (int32_t*)ws;
  int32_t* defer_list = order + B;
  int32_t* counts = order + 2 * (size_t)B;
  const bool plan = defer;          // a planning launch (which also lists the deferred queries)
  const int self_plan = !defer && B > 256;  // else the flat workgroups order themselves
  const int words = ((((uintptr_t)cont_tok) & 3) == 0 && (m % 2) == 0) ? 1 : 0;
  (void)hipGetLastError();
  if (plan) {
    hipLaunchKernelGGL(k_tree_plan, dim3(1), dim3(kPlanThreads), 0, stream, taken, S, k, rows, n_rows, B, cap, order,
                       defer ? defer_list : nullptr, defer ? counts : nullptr);
    FC_CHECK_LAUNCH();
  }
  // a small batch leaves CUs idle: each query gets a workgroup twice as wide
  bool wide = false;
  if constexpr (MAXM == 10) {
    wide = !plan && B <= kFlatWideMaxB && lay.total + dv.wide_static[NARROW ? 1 : 0] <= (size_t)dv.max_lds;
    if (wide)
      hipLaunchKernelGGL((k_tree_flat<MAXM, NARROW, kFlatWide>), dim3(B), dim3(kFlatWide), lay.total, stream, taken,
                         cont_len, cont_tok, ctx, L, S, k, m, t.c, a, cap, words, nullptr, self_plan, B, rows, n_rows,
                         num_nodes, node_tok, parent, weight, pos_ids, mask);
  }
  if (!wide)
    hipLaunchKernelGGL((k_tree_flat<MAXM, NARROW>), dim3(B), dim3(kFlatThreads), lay.total, stream, taken, cont_len,
                       cont_tok, ctx, L, S, k, m, t.c, a, cap, words, plan ? order : nullptr, self_plan, B, rows,
                       n_rows, num_nodes, node_tok, parent, weight, pos_ids, mask);
  FC_CHECK_LAUNCH();
  if (defer) {
    hipLaunchKernelGGL((k_tree_fast<1024, MAXM, NARROW>), dim3(B), dim3(1024), full.total, stream, taken, cont_len,
                       cont_tok, ctx, L, S, k, m, t.c, a, defer_list, counts, nullptr, nullptr, B, k,
                       block_words(cont_tok, k, m), rows, n_rows, num_nodes, node_tok, parent, weight, pos_ids, mask);
    FC_CHECK_LAUNCH();
  }
  return FC_OK;
}

}  // namespace

extern "C" size_t fc_build_tree_workspace_bytes(int32_t B) {
  return B > 0 ? (2 * (size_t)B + 2) * sizeof(int32_t) : 0;
}

extern "C" fc_status fc_build_tree(const int32_t* taken, const uint8_t* cont_len, const uint16_t* cont_tok,
                                   const uint16_t* ctx, int32_t B, int32_t L, int32_t S, int32_t k, int32_t m,
                                   fc_tree_params t, int32_t* num_nodes, int32_t* node_tok, int32_t* parent,
                                   uint32_t* weight, int32_t* pos_ids, int32_t* mask, const int32_t* rows,
                                   int32_t n_rows, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (B < 0 || L < 1 || S < 1 || S > FC_MAX_SOURCES) return FC_ERR_INVALID;
  if (k < 1 || m < 1 || m > 255 || t.c < 1 || t.c + 1 > FC_MAX_TREE_ROWS) return FC_ERR_INVALID;
  if (k > 65535) return FC_ERR_UNSUPPORTED;
  for (int s = 0; s < S; ++s)
    if ((uint64_t)t.alpha[s] * (uint64_t)k > 0xFFFFFFFFull) return FC_ERR_UNSUPPORTED;
  if (B == 0) return FC_OK;
  if (!taken || !cont_len || !cont_tok || !ctx || !num_nodes || !node_tok || !parent || !weight || !pos_ids || !mask)
    return FC_ERR_INVALID;
  if (rows && n_rows < 1) return FC_ERR_INVALID;
  if (!ws || ws_bytes < fc_build_tree_workspace_bytes(B)) return FC_ERR_WORKSPACE;
  const TreeDevice* dv = tree_device();
  if (!dv) return FC_ERR_DEVICE;
  Alpha a = {};
  for (int s = 0; s < S; ++s) a.a[s] = t.alpha[s];
  const TreeLayout full = tree_layout(k, m);
  bool narrow = (uint64_t)t.alpha[0] * (uint64_t)k <= 0xFFFFull;
  for (int s = 1; s < S; ++s) narrow = narrow && t.alpha[s] == t.alpha[0];
  fc_status st = FC_ERR_UNSUPPORTED;
#define FC_FLAT(MM, NN)                                                                                              \
  st = launch_flat<MM, NN>(taken, cont_len, cont_tok, ctx, B, L, S, k, m, t, a, full, *dv, num_nodes, node_tok,      \
                           parent, weight, pos_ids, mask, rows, n_rows, ws, stream)
  if (m <= 10) {
    if (narrow) FC_FLAT(10, true);
    else FC_FLAT(10, false);
  } else if (m <= 16) {
    if (narrow) FC_FLAT(16, true);
    else FC_FLAT(16, false);
  }
#undef FC_FLAT
  if (st != FC_ERR_UNSUPPORTED) return st;
  const size_t static_lds = m <= 16 ? dv->full_static[m <= 10 ? 0 : 1][narrow ? 1 : 0] : dv->any_static;
  if (full.total + static_lds > (size_t)dv->max_lds) return FC_ERR_UNSUPPORTED;
#define FC_FAST(MM, NN)                                                                                              \
  return launch_fast<MM, NN>(taken, cont_len, cont_tok, ctx, B, L, S, k, m, t, a, full, num_nodes, node_tok, parent, \
                             weight, pos_ids, mask, rows, n_rows, ws, stream)
  if (m <= 10) {
    if (narrow) FC_FAST(10, true);
    FC_FAST(10, false);
  }
  if (m <= 16) {
    if (narrow) FC_FAST(16, true);
    FC_FAST(16, false);
  }
#undef FC_FAST
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_tree_any, dim3(B), dim3(kTreeThreads), full.total, stream, taken, cont_len, cont_tok, ctx, L,
                     S, k, m, t.c, a, rows, n_rows, num_nodes, node_tok, parent, weight, pos_ids, mask);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
