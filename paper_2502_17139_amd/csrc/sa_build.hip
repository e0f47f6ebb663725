// Suffix-array construction on gfx950 (fc_datastore_build, fc_store_prepare).
//
// The datastore is indexed for exact suffix matching with a suffix array
// (Section III-A, after Manber and Myers; datastore organisation in
// Section IV-A).  Construction is prefix doubling, which is what Manber and
// Myers' own construction does, with every round's sort done as an LSD radix
// sort so it runs at HBM bandwidth:
//
//   round 0  key(i) = the first 3 tokens of suffix i, each as token+1 in as
//            many bits as the largest token + 1 needs (at most 17), with 0
//            past the end, so a suffix that ends first sorts first; all n
//            suffixes are sorted.
//   round r  (h = 3 * 2^(r-1)) only suffixes still tied with another are
//            re-sorted, by key(i) = (rank[i], rank[i+h] + 1, or 0 past the
//            end), where rank[i] is the suffix-array index at which i's group
//            of equal h-token prefixes starts (Larsson and Sadakane's group
//            numbering).  Suffixes whose group becomes a singleton drop out.
//   a suffix whose group becomes a singleton has its final index, rank[i],
//   and sa[rank[i]] = i is written in that round (in sorted order, so at
//   nearly sequential addresses).
//
// Each radix sort is a global digit histogram followed by one "onesweep"
// pass per 8-bit digit (Adinets and Merrill 2022): a workgroup takes a tile
// of 4,096 keys (its tile id from an atomic ticket, so tiles start in order),
// ranks them stably inside the tile with wave ballots, publishes per-digit
// tile counts and resolves its global offsets by decoupled look-back over the
// earlier tiles, stages the tile in LDS in digit order, and writes it out in
// runs.  Digit passes in which every key has the same digit are skipped.
//
// After each sort, head flags of the new and old groups are turned into
// group starts with a three-phase scan (tile partials, one-workgroup scan of
// the partials, per-tile apply), which also compacts the still-tied suffixes.
// Both tile passes run wave-striped (a wave takes 1,024 consecutive sorted
// positions, 64 at a time), so every load and store of a wave is coalesced
// except the rank scatter itself, which is indexed by suffix.  Where the
// rank array outgrows the MALL (64M suffixes or more), a random 4-byte write
// costs a 32-byte memory write, so the round's (suffix, rank) pairs are
// written in sorted order instead, sorted by the suffix's top 24 bits
// (three keys-only passes), and then stored one small window of the rank
// array after another, each wave's stores falling on a few cache lines.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kSortThreads = 256;
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortThreads * kSortItems;  // 4,096 keys per tile
constexpr int kRadix = 256;
constexpr int kMaxDigits = 8;
constexpr int kSegThreads = 256;
constexpr int kSegItems = 16;
constexpr int kSegTile = kSegThreads * kSegItems;
constexpr int kScanThreads = 1024;
constexpr int kMaxPasses = 1024;  // ticket counters per build
constexpr int kMaxRounds = 40;
constexpr int kHistBlocks = 2048;
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kLookWindow = 2;  // earlier tiles examined per look-back step (with the counts
                                // published early, wider windows only add loads)

constexpr uint64_t kFlagAgg = 1ull << 46;
constexpr uint64_t kFlagInc = 2ull << 46;
constexpr uint64_t kFlagMask = 3ull << 46;
constexpr uint64_t kCountMask = (1ull << 46) - 1;

__device__ __forceinline__ uint64_t pack_status(uint32_t epoch, uint64_t flag, uint64_t count) {
  return ((uint64_t)epoch << 48) | flag | count;
}

// ---------------------------------------------------------------- keys ----

__global__ void __launch_bounds__(256) k_init_keys(const uint16_t* __restrict__ tok, uint32_t n, int tb,
                                                     uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint64_t a = (uint64_t)tok[i] + 1;
  uint64_t b = (i + 1 < n) ? (uint64_t)tok[i + 1] + 1 : 0;
  uint64_t c = (i + 2 < n) ? (uint64_t)tok[i + 2] + 1 : 0;
  keys[i] = (a << (2 * tb)) | (b << tb) | c;
  vals[i] = i;
}

// The high half of each key (the suffix's own rank) was written in place by
// the previous round's k_seg_apply, in this round's order, so only the rank
// h positions on is gathered.
__global__ void __launch_bounds__(256) k_pair_keys(const uint32_t* __restrict__ vals, uint32_t U,
                                                     const uint32_t* __restrict__ rank, uint32_t n, uint64_t h,
                                                     uint64_t* __restrict__ keys) {
  uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= U) return;
  uint32_t i = vals[r];
  uint64_t lo = ((uint64_t)i + h < n) ? (uint64_t)rank[i + h] + 1 : 0;
  keys[r] |= lo;
}

// Batched build: position i belongs to the segment r with off[r] <= i <
// off[r+1] (the last r with off[r] <= i, so empty segments are skipped).
__device__ __forceinline__ uint32_t segment_of(const uint64_t* __restrict__ off, uint32_t R, uint64_t i) {
  uint32_t lo = 0, hi = R - 1;
  while (lo < hi) {
    const uint32_t mid = (lo + hi + 1) >> 1;
    if (off[mid] <= i) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Round 0 of a batched build: key = (segment, first two tokens as token+1,
// 0 past the segment's end), so suffixes of different segments never share
// a group and every suffix ends at its own segment's end.
__global__ void __launch_bounds__(256) k_init_keys_seg(const uint16_t* __restrict__ tok, uint32_t n,
                                                         const uint64_t* __restrict__ off, uint32_t R,
                                                         uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                                         uint32_t* __restrict__ end_of) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t r = segment_of(off, R, i);
  const uint32_t end = (uint32_t)off[r + 1];
  const uint64_t a = (uint64_t)tok[i] + 1;
  const uint64_t b = (i + 1 < end) ? (uint64_t)tok[i + 1] + 1 : 0;
  keys[i] = ((uint64_t)r << 34) | (a << 17) | b;
  vals[i] = i;
  end_of[i] = end;
}

__global__ void __launch_bounds__(256) k_pair_keys_seg(const uint32_t* __restrict__ vals, uint32_t U,
                                                         const uint32_t* __restrict__ rank,
                                                         const uint32_t* __restrict__ end_of, uint64_t h,
                                                         uint32_t sb, uint64_t* __restrict__ keys) {
  const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= U) return;
  const uint32_t i = vals[r];
  const uint64_t hi = rank[i];
  const uint64_t lo = ((uint64_t)i + h < end_of[i]) ? (uint64_t)rank[i + h] + 1 : 0;
  keys[r] = (hi << sb) | lo;
}

// Segment-major suffix array -> positions local to each segment.
__global__ void __launch_bounds__(256) k_localize_sa(uint32_t* __restrict__ sa, uint32_t n,
                                                       const uint64_t* __restrict__ off, uint32_t R) {
  const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < n) sa[r] -= (uint32_t)off[segment_of(off, R, r)];
}

// ------------------------------------------------------------ extension --
//
// fc_datastore_extend: text = X . T, X the o new tokens in front of the old
// store T (n_old tokens) whose suffix array is known.  Suffixes of T are
// suffixes of the new text, so their order is kept.  For each new suffix p
// the build finds ins(p) = the number of old suffixes smaller than it, then
// orders the new suffixes among themselves, and merges.

// inverse of the old suffix array
__global__ void __launch_bounds__(256) k_isa(const uint32_t* __restrict__ sa, uint32_t n_old,
                                               uint32_t* __restrict__ isa) {
  const uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < n_old) {
    const uint32_t q = sa[j];
    if (q < n_old) isa[q] = j;  // a malformed array cannot write out of bounds
  }
}

// ins by doubling over h = 64, 128, ...: [lo, hi) is the suffix-array range
// of the old suffixes whose first h tokens equal those of new suffix p.
// Inside such a range the old suffixes are ordered by what follows their
// first h tokens, i.e. by isa[q + h] (0 for an empty rest, isa + 1 else),
// so the next range is found by two binary searches against p + h's range
// (or, once p + h lies in T, against the single old suffix there).  An
// empty range is final: its start is ins(p).

// First ranges, for h = kExtFirst tokens at once: a binary search of the
// new suffix's first kExtFirst tokens over the old array, comparing token by
// token from the common prefix both bounds share (Manber and Myers' search).
// Most new suffixes of real text are placed here; only those sharing more
// than kExtFirst tokens with an old suffix go on to the doubling rounds.
constexpr uint32_t kExtFirst = 64;

// sign of (new suffix p, at most kExtFirst tokens) - (old suffix q), from
// offset d on; *lcp receives the common length, capped at kExtFirst
__device__ __forceinline__ int ext_cmp(const uint16_t* __restrict__ tok, uint32_t o, uint64_t n, uint32_t n_old,
                                       uint32_t p, uint32_t q, uint32_t d, uint32_t* lcp) {
  for (; d < kExtFirst; ++d) {
    if ((uint64_t)q + d >= n_old) { *lcp = d; return 1; }   // the old suffix ended first
    if ((uint64_t)p + d >= n) { *lcp = d; return -1; }
    const uint32_t a = tok[p + d], b = tok[(uint64_t)o + q + d];
    if (a != b) { *lcp = d; return a > b ? 1 : -1; }
  }
  *lcp = kExtFirst;
  return 0;
}

__global__ void __launch_bounds__(256) k_ext_init(const uint16_t* __restrict__ tok, uint32_t o, uint64_t n,
                                                    const uint32_t* __restrict__ sa, uint32_t n_old,
                                                    uint32_t* __restrict__ lo0, uint32_t* __restrict__ hi0,
                                                    uint32_t* __restrict__ lo1, uint32_t* __restrict__ hi1,
                                                    uint32_t* __restrict__ active, uint32_t* __restrict__ count) {
  const uint32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= o) return;
  auto old_at = [&](uint32_t r) -> uint32_t {
    const uint32_t q = sa[r];
    return q < n_old ? q : n_old;  // a malformed array reads as an ended suffix
  };
  // lower end: first r whose suffix is >= the new suffix's first tokens
  uint32_t a = 0, b = n_old, la = 0, lb = 0;
  while (a < b) {
    const uint32_t mid = (a + b) >> 1;
    uint32_t l;
    const int c = ext_cmp(tok, o, n, n_old, p, old_at(mid), la < lb ? la : lb, &l);
    if (c > 0) { a = mid + 1; la = l; } else { b = mid; lb = l; }
  }
  // upper end: first r whose suffix is > them (the search resumes from a,
  // whose left neighbour shares la tokens)
  uint32_t e = a, f = n_old, le = la, lf = 0;
  while (e < f) {
    const uint32_t mid = (e + f) >> 1;
    uint32_t l;
    const int c = ext_cmp(tok, o, n, n_old, p, old_at(mid), le < lf ? le : lf, &l);
    if (c >= 0) { e = mid + 1; le = l; } else { f = mid; lf = l; }
  }
  lo0[p] = lo1[p] = a;
  hi0[p] = hi1[p] = e;
  if (a < e) active[atomicAdd(count, 1u)] = p;
}

__device__ __forceinline__ uint32_t ext_key(const uint32_t* __restrict__ sa, const uint32_t* __restrict__ isa,
                                            uint32_t n_old, uint64_t h, uint32_t r) {
  const uint64_t q = (uint64_t)sa[r] + h;
  return q < n_old ? isa[q] + 1 : 0u;
}

__global__ void __launch_bounds__(256) k_ext_round(uint32_t o, uint64_t n, uint32_t n_old,
                                                     const uint32_t* __restrict__ sa,
                                                     const uint32_t* __restrict__ isa, uint64_t h,
                                                     const uint32_t* __restrict__ clo,
                                                     const uint32_t* __restrict__ chi, uint32_t* __restrict__ nlo,
                                                     uint32_t* __restrict__ nhi, const uint32_t* __restrict__ act,
                                                     const uint32_t* __restrict__ n_act,
                                                     uint32_t* __restrict__ act_out,
                                                     uint32_t* __restrict__ done_out,
                                                     uint32_t* __restrict__ counts) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= *n_act) return;
  const uint32_t p = act[t];
  const uint32_t lo = clo[p], hi = chi[p];
  const uint64_t z = (uint64_t)p + h;
  uint32_t a, b;
  if (z < o) {
    a = clo[z] + 1;
    b = chi[z] + 1;
  } else if (z < n) {
    a = b = isa[z - o] + 1;
  } else {
    a = b = 0;
  }
  uint32_t x = lo, y = hi;
  while (x < y) {
    const uint32_t mid = (x + y) >> 1;
    if (ext_key(sa, isa, n_old, h, mid) < a) x = mid + 1; else y = mid;
  }
  const uint32_t nl = x;
  if (a != b) {
    y = hi;
    while (x < y) {
      const uint32_t mid = (x + y) >> 1;
      if (ext_key(sa, isa, n_old, h, mid) < b) x = mid + 1; else y = mid;
    }
  }
  nlo[p] = nl;
  nhi[p] = x;
  if (nl < x) act_out[atomicAdd(&counts[0], 1u)] = p;
  else done_out[atomicAdd(&counts[1], 1u)] = p;
}

// a range that became final this round is copied into the other buffer
// (no other work of the next round touches it)
__global__ void __launch_bounds__(256) k_ext_fix(const uint32_t* __restrict__ done,
                                                   const uint32_t* __restrict__ n_done,
                                                   const uint32_t* __restrict__ nlo, uint32_t* __restrict__ olo,
                                                   uint32_t* __restrict__ ohi) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= *n_done) return;
  const uint32_t p = done[t];
  olo[p] = ohi[p] = nlo[p];
}

// Ordering the new suffixes: prefix doubling as in the plain build, over the
// o new positions only, with ins(p) as the most significant field of round
// 0's key.  A new suffix's group label is ins(p) + rank[p] and an old
// suffix's is its final index isa + (new suffixes with ins <= isa): both are
// positions in the final array's order, so the rank of whatever follows the
// first h tokens can be either kind.
__global__ void __launch_bounds__(256) k_init_keys_ext(const uint16_t* __restrict__ tok, uint32_t o, uint64_t n,
                                                         const uint32_t* __restrict__ ins, int two,
                                                         uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
  const uint32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= o) return;
  const uint64_t a = (uint64_t)tok[p] + 1;
  const uint64_t b = ((uint64_t)p + 1 < n) ? (uint64_t)tok[p + 1] + 1 : 0;
  keys[p] = two ? (((uint64_t)ins[p] << 34) | (a << 17) | b) : (((uint64_t)ins[p] << 17) | a);
  vals[p] = p;
}

__global__ void __launch_bounds__(256) k_ins_sorted(const uint64_t* __restrict__ keys, uint32_t o, int shift,
                                                      uint32_t* __restrict__ out) {
  const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r < o) out[r] = (uint32_t)(keys[r] >> shift);
}

// number of s[0..len) that are <= j (s non-decreasing)
__device__ __forceinline__ uint32_t count_le(const uint32_t* __restrict__ s, uint32_t len, uint32_t j) {
  uint32_t a = 0, b = len;
  while (a < b) {
    const uint32_t mid = (a + b) >> 1;
    if (s[mid] <= j) a = mid + 1; else b = mid;
  }
  return a;
}

__global__ void __launch_bounds__(256) k_pair_keys_ext(const uint32_t* __restrict__ vals, uint32_t U,
                                                         const uint32_t* __restrict__ rank,
                                                         const uint32_t* __restrict__ ins,
                                                         const uint32_t* __restrict__ isa,
                                                         const uint32_t* __restrict__ ins_sorted, uint32_t o,
                                                         uint64_t n, uint64_t h, uint32_t sb,
                                                         uint64_t* __restrict__ keys) {
  const uint32_t r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= U) return;
  const uint32_t p = vals[r];
  const uint64_t z = (uint64_t)p + h;
  uint64_t lo;
  if (z < o) {
    lo = (uint64_t)rank[z] + ins[z] + 1;
  } else if (z < n) {
    const uint32_t j = isa[z - o];
    lo = (uint64_t)j + count_le(ins_sorted, o, j) + 1;
  } else {
    lo = 0;
  }
  keys[r] = ((uint64_t)rank[p] << sb) | lo;
}

// merge: new suffix p goes to ins(p) + rank[p], old suffix at index j to
// j + (new suffixes with ins <= j), at position sa[j] + o
__global__ void __launch_bounds__(256) k_ext_new_out(const uint32_t* __restrict__ rank,
                                                       const uint32_t* __restrict__ ins, uint32_t o,
                                                       uint32_t* __restrict__ out) {
  const uint32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < o) out[rank[p] + ins[p]] = p;
}

constexpr int kOldItems = 8;
constexpr int kCountShift = 11;  // one coarse count per 2048 old indexes (256 threads x kOldItems)
static_assert((256 * kOldItems) == (1 << kCountShift), "a merge workgroup covers one coarse block");

// coarse[b] = number of new suffixes with ins < b * 2048, b = 0 .. n_old/2048 + 1
__global__ void __launch_bounds__(256) k_ext_coarse(const uint32_t* __restrict__ ins_sorted, uint32_t o,
                                                      uint32_t nb, uint32_t* __restrict__ coarse) {
  const uint32_t b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= nb) return;
  const uint64_t v = (uint64_t)b << kCountShift;
  uint32_t x = 0, y = o;
  while (x < y) {
    const uint32_t mid = (x + y) >> 1;
    if (ins_sorted[mid] < v) x = mid + 1; else y = mid;
  }
  coarse[b] = x;
}

// number of new suffixes with ins <= j, from the coarse table
__device__ __forceinline__ uint32_t count_new_le(const uint32_t* __restrict__ ins_sorted,
                                                 const uint32_t* __restrict__ coarse, uint32_t j) {
  const uint32_t b = j >> kCountShift;
  uint32_t x = coarse[b], y = coarse[b + 1];
  while (x < y) {
    const uint32_t mid = (x + y) >> 1;
    if (ins_sorted[mid] <= j) x = mid + 1; else y = mid;
  }
  return x;
}

__global__ void __launch_bounds__(256) k_ext_old_out(const uint32_t* __restrict__ sa, uint32_t n_old,
                                                       const uint32_t* __restrict__ ins_sorted,
                                                       const uint32_t* __restrict__ coarse, uint32_t o,
                                                       uint32_t* __restrict__ out) {
  // workgroup b covers old indexes [2048 b, 2048 (b + 1)): one coarse block,
  // whose few inserted suffixes every thread searches; j = base + t + 256 i
  // keeps each step's reads and writes coalesced
  const uint32_t base = blockIdx.x << kCountShift;
  const uint32_t c0 = o ? coarse[blockIdx.x] : 0u, c1 = o ? coarse[blockIdx.x + 1] : 0u;
  for (int i = 0; i < kOldItems; ++i) {
    const uint32_t j = base + threadIdx.x + 256 * i;
    if (j >= n_old) break;
    uint32_t x = c0, y = c1;
    while (x < y) {
      const uint32_t mid = (x + y) >> 1;
      if (ins_sorted[mid] <= j) x = mid + 1; else y = mid;
    }
    out[j + x] = sa[j] + o;
  }
}

// inverse of the result: new position p at ins(p) + rank[p]; old position q
// (now q + o) at isa[q] + (new suffixes with ins <= isa[q])
__global__ void __launch_bounds__(256) k_ext_isa_new(const uint32_t* __restrict__ rank,
                                                       const uint32_t* __restrict__ ins, uint32_t o,
                                                       uint32_t* __restrict__ isa_out) {
  const uint32_t p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p < o) isa_out[p] = rank[p] + ins[p];
}

__global__ void __launch_bounds__(256) k_ext_isa_old(const uint32_t* __restrict__ isa, uint32_t n_old,
                                                       const uint32_t* __restrict__ ins_sorted,
                                                       const uint32_t* __restrict__ coarse, uint32_t o,
                                                       uint32_t* __restrict__ isa_out) {
  const uint32_t q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= n_old) return;
  uint32_t j = isa[q];
  j = j < n_old ? j : n_old - 1;  // a malformed inverse cannot read out of bounds
  isa_out[q + o] = j + (o ? count_new_le(ins_sorted, coarse, j) : 0u);
}

// ------------------------------------------------------------ histogram ---

__global__ void __launch_bounds__(256) k_hist(const uint64_t* __restrict__ keys, uint32_t U, int shift0,
                                                int digits, uint32_t* __restrict__ hist) {
  __shared__ uint32_t s[kMaxDigits][kRadix];
  for (int i = threadIdx.x; i < kMaxDigits * kRadix; i += blockDim.x) (&s[0][0])[i] = 0;
  __syncthreads();
  // 64-bit index: U can come within a grid stride of 2^32.  The keys are in
  // the previous round's sorted order, so a wave's 64 consecutive keys
  // mostly share their high digits, in runs: each run of equal digits in
  // consecutive lanes is counted with one LDS atomic by its first lane
  // (lanes colliding on one bin would serialise).  Each wave takes kHistRun
  // runs of 64 consecutive keys per step, their loads issued together.
  constexpr int kHistRun = 4;
  const uint64_t wave0 = (uint64_t)blockIdx.x * blockDim.x * kHistRun + (threadIdx.x & ~(uint32_t)(fc::kWave - 1)) * kHistRun;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x * kHistRun;
  for (uint64_t i0 = wave0; i0 < U; i0 += stride) {
    uint64_t kv[kHistRun];
#pragma unroll
    for (int u = 0; u < kHistRun; ++u) {
      const uint64_t i = i0 + (uint64_t)(u * fc::kWave + fc::lane_id());
      kv[u] = i < U ? keys[i] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < kHistRun; ++u) {
      const uint64_t i = i0 + (uint64_t)(u * fc::kWave + fc::lane_id());
      const bool valid = i < U;
      const uint64_t k = kv[u];
      const uint64_t act = fc::ballot(valid);
      if (act == 0) continue;
      const uint32_t cnt = (uint32_t)__popcll(act);  // the valid lanes are a prefix
      const uint32_t lane = (uint32_t)fc::lane_id();
      for (int d = 0; d < digits; ++d) {
        const uint32_t dig = (uint32_t)(k >> (shift0 + 8 * d)) & 0xFF;
        const bool head = valid && dig != fc::wave_shr1(dig, ~0u);
        const uint64_t after = fc::ballot(head) >> lane >> 1;  // heads above this lane
        const uint32_t next = after ? lane + 1u + (uint32_t)__builtin_ctzll(after) : cnt;
        if (head) atomicAdd(&s[d][dig], next - lane);
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < digits * kRadix; i += blockDim.x) {
    uint32_t v = (&s[0][0])[i];
    if (v) atomicAdd(&hist[i], v);
  }
}

// One workgroup of 256 threads: digit offsets (exclusive scan per digit) and
// the "trivial" flag of each digit (all keys share it).
__global__ void __launch_bounds__(256) k_hist_scan(const uint32_t* __restrict__ hist, uint32_t U, int digits,
                                                     uint32_t* __restrict__ offsets, uint32_t* __restrict__ trivial) {
  __shared__ uint32_t scratch[8];
  for (int d = 0; d < digits; ++d) {
    uint32_t v = hist[d * kRadix + threadIdx.x];
    uint32_t total;
    uint32_t ex = fc::block_excl_sum<uint32_t>(v, scratch, &total);
    offsets[d * kRadix + threadIdx.x] = ex;
    uint32_t any_full = fc::block_sum<uint32_t>(v == U ? 1u : 0u, scratch);
    if (threadIdx.x == 0) trivial[d] = any_full ? 1u : 0u;
  }
}

// ------------------------------------------------------------- onesweep ---

// kVals false: keys only (vin and vout unused), compiled for four waves per
// SIMD, so four tiles share a CU.
template <bool kVals>
__global__ void __launch_bounds__(kSortThreads, kVals ? 1 : 4) k_onesweep(const uint64_t* __restrict__ kin,
                                                           const uint32_t* __restrict__ vin,
                                                           uint64_t* __restrict__ kout, uint32_t* __restrict__ vout,
                                                           uint32_t U, uint32_t shift,
                                                           const uint32_t* __restrict__ digit_base,
                                                           uint64_t* status, uint32_t* ticket, uint32_t epoch,
                                                           uint32_t* err) {
  __shared__ uint32_t s_tile;
  // per-wave digit counts and then per-wave offsets (below kSortTile), 16
  // bits each: with these the LDS of a tile fits three tiles per CU, which
  // matters because a tile spends most of its time waiting
  __shared__ uint16_t s_wcnt[kSortThreads / fc::kWave][kRadix];
  __shared__ uint16_t s_dstart[kRadix];  // tile-local digit starts (below kSortTile)
  __shared__ uint32_t s_gbase[kRadix];
  __shared__ uint32_t s_scan[kSortThreads / fc::kWave + 1];
  __shared__ uint64_t s_keys[kSortTile];
  __shared__ uint32_t s_vals[kVals ? kSortTile : 1];

  const int tid = threadIdx.x;
  const int w = tid / fc::kWave;
  const int lane = fc::lane_id();
  for (int i = tid; i < (kSortThreads / fc::kWave) * kRadix; i += kSortThreads) (&s_wcnt[0][0])[i] = 0;
  if (tid == 0) s_tile = atomicAdd(ticket, 1u);
  __syncthreads();
  const uint32_t tile = s_tile;
  const uint64_t base = (uint64_t)tile * kSortTile;
  const uint32_t nvalid = (uint32_t)((U - base) < (uint64_t)kSortTile ? (U - base) : (uint64_t)kSortTile);

  uint64_t k[kSortItems];
  uint32_t v[kSortItems];
  uint32_t rk[kSortItems];
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const uint32_t idx = (uint32_t)(w * kSortItems * fc::kWave + j * fc::kWave + lane);
    const bool valid = idx < nvalid;
    k[j] = valid ? kin[base + idx] : ~0ull;
    v[j] = kVals && valid ? vin[base + idx] : 0u;
  }
  const uint64_t lt = fc::lanemask_lt();
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const uint32_t idx = (uint32_t)(w * kSortItems * fc::kWave + j * fc::kWave + lane);
    const bool valid = idx < nvalid;
    const uint32_t d = (uint32_t)(k[j] >> shift) & 0xFF;
    uint64_t peers = fc::ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t ones = fc::ballot(valid && bit);
      peers &= bit ? ones : ~ones;
    }
    const uint32_t below = (uint32_t)__popcll(peers & lt);
    const uint32_t old = s_wcnt[w][d];
    if (valid && below == 0) s_wcnt[w][d] = (uint16_t)(old + (uint32_t)__popcll(peers));
    rk[j] = old + below;
  }
  __syncthreads();

  // Per digit: offsets of each wave's elements, tile count, tile-local start.
  const uint32_t t = (uint32_t)tid;  // this thread's digit
  uint32_t total = 0;
#pragma unroll
  for (int ww = 0; ww < kSortThreads / fc::kWave; ++ww) {
    uint32_t c = s_wcnt[ww][t];
    s_wcnt[ww][t] = (uint16_t)total;
    total += c;
  }
  // publish this tile's digit count at once (tile 0: its inclusive prefix),
  // before the tile-local scan and staging, so later tiles' look-backs find it
  uint64_t* mine = status + (uint64_t)tile * kRadix + t;
  __hip_atomic_store(mine, pack_status(epoch, tile > 0 ? kFlagAgg : kFlagInc, total), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  uint32_t tile_sum;
  s_dstart[t] = (uint16_t)fc::block_excl_sum<uint32_t>(total, s_scan, &tile_sum);
  __syncthreads();

  // Stage in LDS in digit order (before the look-back, so the keys leave
  // the registers while the look-back runs).
#pragma unroll
  for (int j = 0; j < kSortItems; ++j) {
    const uint32_t idx = (uint32_t)(w * kSortItems * fc::kWave + j * fc::kWave + lane);
    if (idx < nvalid) {
      const uint32_t d = (uint32_t)(k[j] >> shift) & 0xFF;
      const uint32_t pos = s_dstart[d] + s_wcnt[w][d] + rk[j];
      s_keys[pos] = k[j];
      if (kVals) s_vals[pos] = v[j];
    }
  }

  // Decoupled look-back for this digit's global offset, kLookWindow earlier
  // tiles per step: their status words are loaded together (for the block,
  // a contiguous run per tile), then taken nearest first - aggregates are
  // added until an inclusive prefix ends the walk; a tile that has published
  // nothing yet makes the walk wait and reload from there.  One round trip
  // then covers as many tiles as the window instead of one.
  uint64_t excl = 0;
  if (tile > 0) {
    int64_t p = (int64_t)tile - 1;  // nearest tile not yet taken
    uint32_t spins = 0;
    bool done = false;
    while (!done) {
      uint64_t sw[kLookWindow];
#pragma unroll
      for (int i = 0; i < kLookWindow; ++i)
        sw[i] = p - i >= 0 ? __hip_atomic_load(status + (uint64_t)(p - i) * kRadix + t, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT)
                           : pack_status(epoch, kFlagInc, 0);  // before tile 0: an empty prefix
      int taken = 0;
      bool stalled = false;
#pragma unroll
      for (int i = 0; i < kLookWindow; ++i) {
        if (done || stalled) continue;
        const uint64_t s = sw[i];
        const uint64_t fl = s & kFlagMask;
        if ((uint32_t)(s >> 48) != epoch || fl == 0) {
          stalled = true;
          continue;
        }
        excl += s & kCountMask;
        ++taken;
        if (fl == kFlagInc) done = true;
      }
      p -= taken;
      if (stalled && !done) {
        if (++spins > kSpinLimit) {
          atomicOr(err, 1u);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  if (tile > 0)
    __hip_atomic_store(mine, pack_status(epoch, kFlagInc, excl + total), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  s_gbase[t] = digit_base[t] + (uint32_t)excl;
  __syncthreads();

  for (uint32_t i = (uint32_t)tid; i < nvalid; i += kSortThreads) {
    const uint64_t key = s_keys[i];
    const uint32_t d = (uint32_t)(key >> shift) & 0xFF;
    const uint32_t dst = s_gbase[d] + (i - s_dstart[d]);
    if (dst < U) {  // always true unless a look-back gave up (then err is set)
      kout[dst] = key;
      if (kVals) vout[dst] = s_vals[i];
    }
  }
}

// ------------------------------------------------------ group bookkeeping --

struct SegFlags {
  bool new_head, old_head, keep;
};

__device__ __forceinline__ SegFlags seg_flags(const uint64_t* __restrict__ keys, uint32_t U, uint32_t r,
                                              uint32_t sb, bool round0) {
  const uint64_t kr = keys[r];
  SegFlags f;
  if (r == 0) {
    f.new_head = true;
    f.old_head = true;
  } else {
    const uint64_t kp = keys[r - 1];
    f.new_head = kr != kp;
    f.old_head = round0 ? false : ((kr >> sb) != (kp >> sb));
  }
  const bool last_of_group = (r + 1 == U) || (keys[r + 1] != kr);
  f.keep = !(f.new_head && last_of_group);
  return f;
}

// Per tile: last new-group head, last old-group head, number kept.
__global__ void __launch_bounds__(kSegThreads) k_seg_partials(const uint64_t* __restrict__ keys, uint32_t U,
                                                                uint32_t sb, int round0, uint32_t* __restrict__ part_h,
                                                                uint32_t* __restrict__ part_g,
                                                                uint32_t* __restrict__ part_k) {
  __shared__ uint32_t scratch[kSegThreads / fc::kWave + 1];
  const uint32_t r0 = blockIdx.x * kSegTile + threadIdx.x;
  uint32_t mh = 0, mg = 0, kc = 0;
  for (int j = 0; j < kSegItems; ++j) {
    const uint32_t r = r0 + (uint32_t)j * kSegThreads;  // coalesced; max and sum ignore the order
    if (r >= U) break;
    const SegFlags f = seg_flags(keys, U, r, sb, round0 != 0);
    if (f.new_head) mh = r;
    if (f.old_head) mg = r;
    kc += f.keep ? 1u : 0u;
  }
  mh = fc::block_max<uint32_t>(mh, scratch);
  mg = fc::block_max<uint32_t>(mg, scratch);
  kc = fc::block_sum<uint32_t>(kc, scratch);
  if (threadIdx.x == 0) {
    part_h[blockIdx.x] = mh;
    part_g[blockIdx.x] = mg;
    part_k[blockIdx.x] = kc;
  }
}

// One workgroup: exclusive max / max / sum scans of the tile partials, in
// place; *u_next receives the number kept.  The partials are taken in chunks
// of kScanThreads * kScanRun, each thread a run of kScanRun consecutive ones
// (so a wave's loads and stores cover contiguous memory), with the chunk
// totals carried from chunk to chunk.
constexpr int kScanRun = 8;
__global__ void __launch_bounds__(kScanThreads) k_seg_scan(uint32_t* __restrict__ part_h,
                                                             uint32_t* __restrict__ part_g,
                                                             uint32_t* __restrict__ part_k, uint32_t ntiles,
                                                             uint32_t* __restrict__ u_next) {
  __shared__ uint32_t scratch[kScanThreads / fc::kWave + 1];
  __shared__ uint32_t s_last[3];
  uint32_t ch = 0, cg = 0, ck = 0;  // carries: maxima and sum over the earlier chunks
  for (uint32_t c0 = 0; c0 < ntiles; c0 += kScanThreads * kScanRun) {
    const uint32_t b0 = c0 + threadIdx.x * kScanRun;
    uint32_t h[kScanRun], g[kScanRun], k[kScanRun];
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) {
      const uint32_t i = b0 + (uint32_t)j;
      h[j] = i < ntiles ? part_h[i] : 0u;
      g[j] = i < ntiles ? part_g[i] : 0u;
      k[j] = i < ntiles ? part_k[i] : 0u;
    }
    uint32_t mh = 0, mg = 0, kc = 0;
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) {
      mh = h[j] > mh ? h[j] : mh;
      mg = g[j] > mg ? g[j] : mg;
      kc += k[j];
    }
    uint32_t total;
    uint32_t eh = fc::block_excl_max<uint32_t>(mh, 0u, scratch);
    uint32_t eg = fc::block_excl_max<uint32_t>(mg, 0u, scratch);
    uint32_t ek = fc::block_excl_sum<uint32_t>(kc, scratch, &total);
    eh = eh > ch ? eh : ch;
    eg = eg > cg ? eg : cg;
    ek += ck;
#pragma unroll
    for (int j = 0; j < kScanRun; ++j) {
      const uint32_t i = b0 + (uint32_t)j;
      if (i < ntiles) {
        part_h[i] = eh;
        part_g[i] = eg;
        part_k[i] = ek;
      }
      eh = h[j] > eh ? h[j] : eh;
      eg = g[j] > eg ? g[j] : eg;
      ek += k[j];
    }
    if (threadIdx.x == kScanThreads - 1) {
      s_last[0] = eh;
      s_last[1] = eg;
      s_last[2] = ek;
    }
    __syncthreads();
    ch = s_last[0];
    cg = s_last[1];
    ck = s_last[2];
    __syncthreads();
  }
  if (threadIdx.x == 0) *u_next = ck;
}

// Per element: new rank = old group start + (new head index - old head index)
// in the sorted list; tied suffixes are compacted into vals_next.  A suffix
// whose group is now a singleton has its final index, so its suffix array
// entry is written here (sa_out, unless null), in sorted order.  The ranks
// go to rank[] directly (a random 4-byte write each), or, with pairs, as
// (suffix << 32 | rank) at the element's own position, for k_rank_write
// after a sort by suffix.  Wave w of
// the tile takes positions [w * 1024, (w + 1) * 1024) of it, 64 consecutive
// ones per step: the running head indexes and the kept count are wave scans
// carried from step to step, started from the earlier waves' totals and the
// tile prefix.
__global__ void __launch_bounds__(kSegThreads) k_seg_apply(const uint64_t* __restrict__ keys,
                                                             const uint32_t* __restrict__ vals, uint32_t U,
                                                             uint32_t sb, int round0,
                                                             const uint32_t* __restrict__ pre_h,
                                                             const uint32_t* __restrict__ pre_g,
                                                             const uint32_t* __restrict__ pre_k,
                                                             uint32_t* __restrict__ rank,
                                                             uint64_t* __restrict__ pairs,
                                                             uint32_t* __restrict__ vals_next,
                                                             uint64_t* __restrict__ hi_next,
                                                             uint32_t* __restrict__ sa_out) {
  constexpr int kWaves = kSegThreads / fc::kWave;
  constexpr uint32_t kPerWave = kSegTile / kWaves;
  __shared__ uint32_t s_tot[3][kWaves];
  const int w = (int)threadIdx.x / fc::kWave;
  const uint32_t lane = (uint32_t)fc::lane_id();
  const uint32_t base = blockIdx.x * kSegTile + (uint32_t)w * kPerWave;
  const bool r0f = round0 != 0;
  // the wave's totals
  uint32_t mh = 0, mg = 0, kc = 0;
  for (int j = 0; j < kSegItems; ++j) {
    const uint32_t r = base + (uint32_t)j * fc::kWave + lane;
    if (r < U) {
      const SegFlags f = seg_flags(keys, U, r, sb, r0f);
      if (f.new_head) mh = r;
      if (f.old_head) mg = r;
      kc += f.keep ? 1u : 0u;
    }
  }
  mh = fc::wave_max<uint32_t>(mh);
  mg = fc::wave_max<uint32_t>(mg);
  kc = fc::wave_sum<uint32_t>(kc);
  if (lane == 0) {
    s_tot[0][w] = mh;
    s_tot[1][w] = mg;
    s_tot[2][w] = kc;
  }
  __syncthreads();
  uint32_t hh = pre_h[blockIdx.x], gg = pre_g[blockIdx.x], out = pre_k[blockIdx.x];
  for (int v = 0; v < w; ++v) {
    hh = s_tot[0][v] > hh ? s_tot[0][v] : hh;
    gg = s_tot[1][v] > gg ? s_tot[1][v] : gg;
    out += s_tot[2][v];
  }
  for (int j = 0; j < kSegItems; ++j) {
    const uint32_t r = base + (uint32_t)j * fc::kWave + lane;
    const bool valid = r < U;
    SegFlags f{false, false, false};
    if (valid) f = seg_flags(keys, U, r, sb, r0f);
    uint32_t hr = fc::wave_incl_max<uint32_t>(f.new_head ? r : 0u);
    uint32_t gr = fc::wave_incl_max<uint32_t>(f.old_head ? r : 0u);
    const uint32_t kr = fc::wave_incl_sum_u32(f.keep ? 1u : 0u);
    hr = hr > hh ? hr : hh;
    gr = gr > gg ? gr : gg;
    if (valid) {
      const uint32_t start = r0f ? 0u : (uint32_t)(keys[r] >> sb);
      const uint32_t i = vals[r];
      const uint32_t rk = start + (hr - gr);
      // in the first new group of its old group a suffix keeps its rank (the
      // old group start, already in rank[i]): only round 0 and the later
      // new groups write (a pair rewrites an unchanged rank with itself)
      if (pairs) pairs[r] = ((uint64_t)i << 32) | rk;
      else if (r0f || hr != gr) rank[i] = rk;
      if (f.keep) {
        vals_next[out + kr - 1u] = i;
        if (hi_next) hi_next[out + kr - 1u] = (uint64_t)rk << sb;  // the next round's key, high half
      }
      else if (sa_out) sa_out[rk] = i;  // a singleton group: rk is the suffix's final index
    }
    hh = __shfl(hr, fc::kWave - 1);
    gg = __shfl(gr, fc::kWave - 1);
    out += __shfl(kr, fc::kWave - 1);
  }
}

// rank[i] = rk for a round's (i << 32 | rk) pairs, sorted by the high bits
// of i so that each run of equal high bits covers one window of the rank
// array (256 bytes at 1G suffixes), and a wave's 64 stores fall on a few
// cache lines.  Workgroup w takes chunk (w % 8) * per_xcd + w / 8 of
// kRankChunk pairs: workgroups are dealt to the eight XCDs in turn, so each
// XCD writes one contiguous eighth of the sorted pairs, and a line is
// assembled in one L2 rather than written back in pieces from several.
constexpr int kRankChunk = 4096;
constexpr int kXcds = 8;
constexpr int kRankSortBits = 24;  // high bits of the suffix index sorted on
constexpr uint64_t kPairRanksMin = 1ull << 26;  // suffixes (4-byte ranks: 256 MB)
__global__ void __launch_bounds__(256) k_rank_write(const uint64_t* __restrict__ pairs, uint32_t U,
                                                    uint32_t per_xcd, uint32_t* __restrict__ rank) {
  const uint32_t c = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  const uint64_t b = (uint64_t)c * kRankChunk;
  if (b >= U) return;
#pragma unroll 4
  for (int j = 0; j < kRankChunk / 256; ++j) {
    const uint64_t r = b + (uint64_t)j * 256 + threadIdx.x;
    if (r < U) {
      const uint64_t p = pairs[r];
      rank[p >> 32] = (uint32_t)p;
    }
  }
}

// ------------------------------------------------------- first-token table --

__global__ void __launch_bounds__(256) k_bucket(const uint16_t* __restrict__ tok, const uint32_t* __restrict__ sa,
                                                  uint32_t n, uint32_t* __restrict__ bucket) {
  const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= FC_BUCKETS) return;
  // first SA index whose suffix starts with a token >= t
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = lo + (hi - lo) / 2;
    if ((uint32_t)tok[sa[mid]] < t) lo = mid + 1; else hi = mid;
  }
  bucket[t] = lo;
}

// Largest token of a store, for the pair-table precondition (out[0] starts
// at 0).
__global__ void __launch_bounds__(256) k_max_token(const uint16_t* __restrict__ tok, uint32_t n,
                                                   uint32_t* __restrict__ out) {
  uint32_t mx = 0;
  for (uint64_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    mx = tok[i] > mx ? tok[i] : mx;
  mx = fc::wave_max(mx);
  if (fc::lane_id() == 0 && mx) atomicMax(out, mx);
}

// Two-token table: suffix-array position r owns the table entries between
// the previous suffix's pair key (exclusive) and its own (inclusive); keys
// never decrease along the suffix array.  r = n owns the rest up to the
// final entry.  Each wave takes 64 consecutive positions and writes their
// ranges one after another with all 64 lanes, so long ranges are written
// in coalesced runs.
__global__ void __launch_bounds__(256) k_pairs(const uint16_t* __restrict__ tok, const uint32_t* __restrict__ sa,
                                               uint32_t n, uint32_t V, uint32_t* __restrict__ pair) {
  const uint64_t base = ((uint64_t)blockIdx.x * blockDim.x + threadIdx.x) & ~(uint64_t)(fc::kWave - 1);
  const int lane = fc::lane_id();
  if (base > n) return;  // whole wave
  const uint64_t end = (uint64_t)V * (V + 1);
  auto key = [&](uint64_t rr) -> uint64_t {
    if (rr >= n) return end;
    const uint32_t j = sa[rr];
    const uint64_t t0 = tok[j];
    const uint64_t u = (uint64_t)j + 1 < n ? (uint64_t)tok[j + 1] + 1 : 0;
    const uint64_t k = t0 * (V + 1) + u;
    return k < end ? k : end;  // tokens >= V were rejected before launch
  };
  const uint64_t r = base + lane;
  uint64_t hi = 0, lo = 1;  // empty unless r <= n
  if (r <= n) {
    hi = key(r);
    lo = r == 0 ? 0 : key(r - 1) + 1;
  }
  for (int jl = 0; jl < fc::kWave; ++jl) {
    const uint64_t l2 = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(lo >> 32), jl) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)lo, jl);
    const uint64_t h2 = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(hi >> 32), jl) << 32) |
                        (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)hi, jl);
    const uint32_t val = (uint32_t)(base + jl);
    for (uint64_t k = l2 + lane; k <= h2; k += fc::kWave) pair[k] = val;
  }
}

// Inline-prefix records: one thread per suffix-array position writes
// {sa[i], T[sa[i]+2 .. sa[i]+32)} as four 16-byte stores (0 past the end).
// The 60 text bytes come from five aligned 16-byte loads (the 80 bytes from
// the 16-byte boundary at or below the first token), re-aligned in
// registers; suffixes whose window would leave the text take token loads.
__global__ void __launch_bounds__(256) k_records(const uint16_t* __restrict__ tok, const uint32_t* __restrict__ sa,
                                                 uint32_t n, uint4* __restrict__ rec) {
  static_assert(FC_RECORD_BYTES == 64 && FC_RECORD_TOKENS == 30, "record layout");
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t j = sa[i];
  uint32_t w[16];
  w[0] = j;
  const uintptr_t base = (uintptr_t)tok;
  const uintptr_t first = base + 2 * ((uint64_t)j + 2);
  const uintptr_t lo = first & ~(uintptr_t)15;
  if (lo >= base && lo + 80 <= base + 2 * (uint64_t)n) {
    uint32_t d[20];
#pragma unroll
    for (int u = 0; u < 5; ++u) {
      const uint4 v = ((const uint4*)lo)[u];
      d[4 * u] = v.x;
      d[4 * u + 1] = v.y;
      d[4 * u + 2] = v.z;
      d[4 * u + 3] = v.w;
    }
    const uint32_t off = (uint32_t)(first - lo);  // 0, 2, .., 14 bytes
    const uint32_t q = off >> 2, half = off & 2;
#pragma unroll
    for (int x = 0; x < FC_RECORD_TOKENS / 2; ++x) {
      // the dword starting at byte off + 4x: dwords q + x and q + x + 1
      const uint32_t a0 = q == 0 ? d[x] : q == 1 ? d[x + 1] : q == 2 ? d[x + 2] : d[x + 3];
      const uint32_t a1 = q == 0 ? d[x + 1] : q == 1 ? d[x + 2] : q == 2 ? d[x + 3] : d[x + 4];
      w[1 + x] = half ? __builtin_amdgcn_alignbyte(a1, a0, 2) : a0;
    }
  } else {
#pragma unroll
    for (int x = 0; x < FC_RECORD_TOKENS / 2; ++x) {
      const uint64_t p = (uint64_t)j + 2 + 2 * x;
      const uint32_t a = p < n ? tok[p] : 0u;
      const uint32_t b = p + 1 < n ? tok[p + 1] : 0u;
      w[1 + x] = a | (b << 16);
    }
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) rec[4 * i + u] = make_uint4(w[4 * u], w[4 * u + 1], w[4 * u + 2], w[4 * u + 3]);
}

struct BuildWs {
  uint32_t* rank;
  uint64_t* keys[2];
  uint32_t* vals[2];
  uint64_t* status;
  uint32_t *part_h, *part_g, *part_k;
  uint32_t* hist;
  uint32_t* offsets;
  uint32_t* tickets;
  uint32_t* misc;  // [0] error flag, [1] next U, [2..9] trivial digit flags, [10] largest token
  uint64_t* pairs;    // plain build: a round's (suffix, rank) pairs
  uint32_t* end_of;   // batched build: end of each position's segment
  uint64_t* seg_off;  // batched build: segment offsets (device copy)
};

size_t carve_build(void* p, uint64_t n, BuildWs* w, uint32_t n_seg = 0) {
  fc::Carver c(p);
  const uint64_t tiles = (n + kSortTile - 1) / kSortTile;
  const uint64_t seg_tiles = (n + kSegTile - 1) / kSegTile;
  BuildWs tmp;
  tmp.rank = c.take<uint32_t>(n);
  tmp.keys[0] = c.take<uint64_t>(n);
  tmp.keys[1] = c.take<uint64_t>(n);
  tmp.vals[0] = c.take<uint32_t>(n);
  tmp.vals[1] = c.take<uint32_t>(n);
  tmp.status = c.take<uint64_t>(tiles * kRadix);
  tmp.part_h = c.take<uint32_t>(seg_tiles);
  tmp.part_g = c.take<uint32_t>(seg_tiles);
  tmp.part_k = c.take<uint32_t>(seg_tiles);
  tmp.hist = c.take<uint32_t>(kMaxDigits * kRadix);
  tmp.offsets = c.take<uint32_t>(kMaxDigits * kRadix);
  tmp.tickets = c.take<uint32_t>(kMaxPasses);
  tmp.misc = c.take<uint32_t>(16);
  tmp.end_of = n_seg ? c.take<uint32_t>(n) : nullptr;
  tmp.seg_off = n_seg ? c.take<uint64_t>((size_t)n_seg + 1) : nullptr;
  tmp.pairs = n_seg == 0 && n >= kPairRanksMin ? c.take<uint64_t>(n) : nullptr;
  if (w) *w = tmp;
  return c.used + 256;
}

int bit_length(uint64_t x) {
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

struct SortState {
  uint32_t epoch = 0;
  uint32_t ticket = 0;
};

// LSD radix sort over key bits [shift0, shift0 + key_bits) of kb[src], with
// vb[src] carried alongside unless vb is null, the passes alternating
// between the two buffers.  *result is the index (0 or 1) of the buffer
// that holds the result.
fc_status radix_sort(BuildWs& w, uint64_t* const kb[2], uint32_t* const vb[2], int src, uint32_t U, int shift0,
                     int key_bits, SortState& st, hipStream_t stream, int* result) {
  const int digits = (key_bits + 7) / 8;
  FC_CHECK_HIP(hipMemsetAsync(w.hist, 0, sizeof(uint32_t) * kMaxDigits * kRadix, stream));
  const uint32_t hist_blocks = fc::div_up(U, 256) < (uint32_t)kHistBlocks ? fc::div_up(U, 256) : kHistBlocks;
  hipLaunchKernelGGL(k_hist, dim3(hist_blocks), dim3(256), 0, stream, kb[src], U, shift0, digits, w.hist);
  FC_CHECK_LAUNCH();
  hipLaunchKernelGGL(k_hist_scan, dim3(1), dim3(256), 0, stream, w.hist, U, digits, w.offsets, w.misc + 2);
  FC_CHECK_LAUNCH();
  uint32_t trivial[kMaxDigits] = {0};
  FC_CHECK_HIP(hipMemcpyAsync(trivial, w.misc + 2, sizeof(uint32_t) * digits, hipMemcpyDeviceToHost, stream));
  FC_CHECK_HIP(hipStreamSynchronize(stream));
  int cur = src;
  const uint32_t tiles = fc::div_up(U, kSortTile);
  for (int d = 0; d < digits; ++d) {
    if (trivial[d]) continue;
    if (st.ticket >= (uint32_t)kMaxPasses) return FC_ERR_UNSUPPORTED;
    ++st.epoch;
    const uint32_t shift = (uint32_t)(shift0 + 8 * d);
    if (vb)
      hipLaunchKernelGGL(k_onesweep<true>, dim3(tiles), dim3(kSortThreads), 0, stream, kb[cur], vb[cur],
                         kb[cur ^ 1], vb[cur ^ 1], U, shift, w.offsets + d * kRadix, w.status, w.tickets + st.ticket,
                         st.epoch, w.misc);
    else
      hipLaunchKernelGGL(k_onesweep<false>, dim3(tiles), dim3(kSortThreads), 0, stream, kb[cur], nullptr,
                         kb[cur ^ 1], nullptr, U, shift, w.offsets + d * kRadix, w.status, w.tickets + st.ticket,
                         st.epoch, w.misc);
    FC_CHECK_LAUNCH();
    ++st.ticket;
    cur ^= 1;
  }
  *result = cur;
  return FC_OK;
}

// The new suffixes of an extension (see k_init_keys_ext).
struct ExtendArgs {
  const uint32_t* ins;  // per new position
  const uint32_t* isa;  // inverse of the old suffix array
  uint32_t* ins_sorted; // ins in the sorted order of the new suffixes
  uint64_t n;           // whole text
  int n_old_bits;
};

// Prefix doubling over all n suffixes (n_seg = 0), over the suffixes of
// n_seg segments at once, each ending at its segment's end (n_seg >= 1,
// offsets already in w.seg_off), or over the n new suffixes of an extension
// (ext; leaves their ranks in w.rank and writes no suffix array).
fc_status build_sa(const uint16_t* tokens, uint64_t n, uint32_t n_seg, BuildWs& w, uint32_t* sa_out,
                   hipStream_t stream, const ExtendArgs* ext = nullptr, fc_build_stats* stats = nullptr) {
  const uint32_t N = (uint32_t)n;
  const uint64_t tiles = (n + kSortTile - 1) / kSortTile;
  FC_CHECK_HIP(hipMemsetAsync(w.status, 0, sizeof(uint64_t) * tiles * kRadix, stream));
  FC_CHECK_HIP(hipMemsetAsync(w.tickets, 0, sizeof(uint32_t) * kMaxPasses, stream));
  FC_CHECK_HIP(hipMemsetAsync(w.misc, 0, sizeof(uint32_t) * 16, stream));

  // every rank + 1 <= n (an extension's labels: <= the whole text) fits in sb bits
  const uint32_t sb = (uint32_t)bit_length(ext ? ext->n : n);
  SortState st;
  uint64_t h;
  int key0_bits;
  int ext_shift = 0;
  if (ext) {
    const int two = ext->n_old_bits + 34 <= 64;
    ext_shift = two ? 34 : 17;
    hipLaunchKernelGGL(k_init_keys_ext, dim3(fc::div_up(N, 256)), dim3(256), 0, stream, tokens, N, ext->n,
                       ext->ins, two, w.keys[0], w.vals[0]);
    h = two ? 2 : 1;
    key0_bits = ext_shift + ext->n_old_bits;
  } else if (n_seg == 0) {
    // token + 1 in tb bits: the largest token decides tb (misc[10] is zero)
    const uint32_t blocks = fc::div_up(N, 256) < 4096u ? fc::div_up(N, 256) : 4096u;
    hipLaunchKernelGGL(k_max_token, dim3(blocks), dim3(256), 0, stream, tokens, N, w.misc + 10);
    FC_CHECK_LAUNCH();
    uint32_t mx = 0;
    FC_CHECK_HIP(hipMemcpyAsync(&mx, w.misc + 10, sizeof(uint32_t), hipMemcpyDeviceToHost, stream));
    FC_CHECK_HIP(hipStreamSynchronize(stream));
    const int tb = bit_length((uint64_t)mx + 1);
    hipLaunchKernelGGL(k_init_keys, dim3(fc::div_up(N, 256)), dim3(256), 0, stream, tokens, N, tb, w.keys[0],
                       w.vals[0]);
    h = 3;
    key0_bits = 3 * tb;
  } else {
    hipLaunchKernelGGL(k_init_keys_seg, dim3(fc::div_up(N, 256)), dim3(256), 0, stream, tokens, N, w.seg_off, n_seg,
                       w.keys[0], w.vals[0], w.end_of);
    h = 2;
    key0_bits = 34 + bit_length(n_seg - 1);
  }
  FC_CHECK_LAUNCH();
  uint32_t U = N;
  int vin = 0;  // buffer holding the suffixes to sort
  // ranks through k_rank_write when the rank array is at least the size of
  // the 256 MB MALL; a smaller one takes the random writes in the MALL
  const bool pair_ranks = !ext && n_seg == 0 && n >= kPairRanksMin;
  for (int round = 0;; ++round) {
    if (round >= kMaxRounds) return FC_ERR_DEVICE;
    if (round > 0) {
      if (ext)
        hipLaunchKernelGGL(k_pair_keys_ext, dim3(fc::div_up(U, 256)), dim3(256), 0, stream, w.vals[vin], U, w.rank,
                           ext->ins, ext->isa, ext->ins_sorted, N, ext->n, h, sb, w.keys[vin]);
      else if (n_seg == 0)
        hipLaunchKernelGGL(k_pair_keys, dim3(fc::div_up(U, 256)), dim3(256), 0, stream, w.vals[vin], U, w.rank, N,
                           h, w.keys[vin]);
      else
        hipLaunchKernelGGL(k_pair_keys_seg, dim3(fc::div_up(U, 256)), dim3(256), 0, stream, w.vals[vin], U, w.rank,
                           w.end_of, h, sb, w.keys[vin]);
      FC_CHECK_LAUNCH();
      h *= 2;
    }
    int res = vin;
    fc_status s = radix_sort(w, w.keys, w.vals, vin, U, 0, round == 0 ? key0_bits : (int)(2 * sb), st, stream,
                             &res);
    if (s != FC_OK) return s;
    if (ext && round == 0) {
      hipLaunchKernelGGL(k_ins_sorted, dim3(fc::div_up(N, 256)), dim3(256), 0, stream, w.keys[res], N, ext_shift,
                         ext->ins_sorted);
      FC_CHECK_LAUNCH();
    }
    const uint32_t seg_tiles = fc::div_up(U, kSegTile);
    hipLaunchKernelGGL(k_seg_partials, dim3(seg_tiles), dim3(kSegThreads), 0, stream, w.keys[res], U, sb,
                       round == 0 ? 1 : 0, w.part_h, w.part_g, w.part_k);
    FC_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_seg_scan, dim3(1), dim3(kScanThreads), 0, stream, w.part_h, w.part_g, w.part_k, seg_tiles,
                       w.misc + 1);
    FC_CHECK_LAUNCH();
    hipLaunchKernelGGL(k_seg_apply, dim3(seg_tiles), dim3(kSegThreads), 0, stream, w.keys[res], w.vals[res], U, sb,
                       round == 0 ? 1 : 0, w.part_h, w.part_g, w.part_k, w.rank, pair_ranks ? w.pairs : nullptr,
                       w.vals[res ^ 1], (ext || n_seg > 0) ? nullptr : w.keys[res ^ 1], ext ? nullptr : sa_out);
    FC_CHECK_LAUNCH();
    uint32_t host_misc[2] = {0, 0};
    FC_CHECK_HIP(hipMemcpyAsync(host_misc, w.misc, sizeof(uint32_t) * 2, hipMemcpyDeviceToHost, stream));
    FC_CHECK_HIP(hipStreamSynchronize(stream));
    if (host_misc[0]) return FC_ERR_DEVICE;
    if (stats && round < FC_MAX_BUILD_ROUNDS) {
      stats->prefix_len[round] = h;
      stats->sorted[round] = U;
      stats->unresolved[round] = host_misc[1];
      stats->rounds = round + 1;
      stats->sort_passes = (int32_t)st.ticket;
    }
    if (pair_ranks && host_misc[1] > 0) {
      // the round's ranks, for the next round's keys: the pairs sorted by the
      // suffix's top kRankSortBits bits (the other sort buffer is free now),
      // then written window by window
      uint64_t* const pb[2] = {w.pairs, w.keys[res]};
      const int hb = (int)sb < kRankSortBits ? (int)sb : kRankSortBits;
      int pres = 0;
      s = radix_sort(w, pb, nullptr, 0, U, 32 + (int)sb - hb, hb, st, stream, &pres);
      if (s != FC_OK) return s;
      const uint32_t per_xcd = fc::div_up(fc::div_up(U, kRankChunk), kXcds);
      hipLaunchKernelGGL(k_rank_write, dim3(per_xcd * kXcds), dim3(256), 0, stream, pb[pres], U, per_xcd, w.rank);
      FC_CHECK_LAUNCH();
    }
    U = host_misc[1];
    vin = res ^ 1;
    if (U == 0) break;
  }
  if (ext) return FC_OK;
  // every suffix array entry was written when its suffix's group became a
  // singleton (k_seg_apply)
  if (n_seg > 0) {
    hipLaunchKernelGGL(k_localize_sa, dim3(fc::div_up(N, 256)), dim3(256), 0, stream, sa_out, N, w.seg_off, n_seg);
    FC_CHECK_LAUNCH();
  }
  return FC_OK;
}

}  // namespace

extern "C" size_t fc_datastore_build_workspace_bytes(uint64_t n) { return carve_build(nullptr, n, nullptr); }

extern "C" fc_status fc_datastore_build_stats(const uint16_t* tokens, uint64_t n, uint32_t* sa_out, void* ws,
                                              size_t ws_bytes, fc_build_stats* stats, hipStream_t stream) {
  if (n >= 0xFFFFFFFFull) return FC_ERR_INVALID;
  if (stats) *stats = fc_build_stats{};
  if (n == 0) return FC_OK;
  if (!tokens || !sa_out) return FC_ERR_INVALID;
  if (!ws || ws_bytes < fc_datastore_build_workspace_bytes(n)) return FC_ERR_WORKSPACE;
  (void)hipGetLastError();
  BuildWs w;
  carve_build(ws, n, &w);
  return build_sa(tokens, n, 0, w, sa_out, stream, nullptr, stats);
}

extern "C" fc_status fc_datastore_build(const uint16_t* tokens, uint64_t n, uint32_t* sa_out, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  return fc_datastore_build_stats(tokens, n, sa_out, ws, ws_bytes, nullptr, stream);
}

extern "C" size_t fc_datastore_build_batched_workspace_bytes(uint64_t n, int32_t n_seg) {
  return n_seg >= 1 ? carve_build(nullptr, n, nullptr, (uint32_t)n_seg) : 0;
}

extern "C" fc_status fc_datastore_build_batched(const uint16_t* tokens, const uint64_t* seg_off, int32_t n_seg,
                                                uint32_t* sa_out, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (n_seg < 1 || !seg_off) return FC_ERR_INVALID;
  if (seg_off[0] != 0) return FC_ERR_INVALID;
  for (int32_t r = 0; r < n_seg; ++r)
    if (seg_off[r + 1] < seg_off[r]) return FC_ERR_INVALID;
  const uint64_t n = seg_off[n_seg];
  if (n >= 0xFFFFFFFFull || 34 + bit_length((uint64_t)n_seg - 1) > 64) return FC_ERR_INVALID;
  if (n == 0) return FC_OK;
  if (!tokens || !sa_out) return FC_ERR_INVALID;
  if (!ws || ws_bytes < fc_datastore_build_batched_workspace_bytes(n, n_seg)) return FC_ERR_WORKSPACE;
  (void)hipGetLastError();
  BuildWs w;
  carve_build(ws, n, &w, (uint32_t)n_seg);
  FC_CHECK_HIP(hipMemcpyAsync(w.seg_off, seg_off, sizeof(uint64_t) * ((size_t)n_seg + 1), hipMemcpyHostToDevice,
                              stream));
  return build_sa(tokens, n, (uint32_t)n_seg, w, sa_out, stream);
}

namespace {

struct ExtendWs {
  uint32_t* isa;  // inverse of the old array, unless the caller passes it
  uint32_t *lo[2], *hi[2];
  uint32_t *act[2], *done;
  uint32_t* counts;  // [0] still ranged, [1] final this round, [2] active now
  uint32_t* ins_sorted;
  uint32_t* coarse;
  BuildWs b;
};

uint32_t coarse_entries(uint64_t n_old) { return (uint32_t)((n_old + (1u << kCountShift) - 1) >> kCountShift) + 1; }

size_t carve_extend(void* p, uint64_t n, uint64_t o, bool isa_given, ExtendWs* w) {
  fc::Carver c(p);
  ExtendWs t;
  t.isa = c.take<uint32_t>(isa_given ? 0 : n - o);
  for (int i = 0; i < 2; ++i) {
    t.lo[i] = c.take<uint32_t>(o);
    t.hi[i] = c.take<uint32_t>(o);
    t.act[i] = c.take<uint32_t>(o);
  }
  t.done = c.take<uint32_t>(o);
  t.counts = c.take<uint32_t>(4);
  t.ins_sorted = c.take<uint32_t>(o);
  t.coarse = c.take<uint32_t>(coarse_entries(n - o));
  char* rest = p ? (char*)p + ((c.used + 255) & ~(size_t)255) : nullptr;
  const size_t head = (c.used + 255) & ~(size_t)255;
  const size_t tail = o ? carve_build(rest, o, &t.b) : 0;
  if (w) *w = t;
  return head + tail;
}

}  // namespace

extern "C" size_t fc_datastore_extend_workspace_bytes(uint64_t n, uint64_t n_new, int32_t isa_given) {
  return n_new <= n && n < 0xFFFFFFFFull ? carve_extend(nullptr, n, n_new, isa_given != 0, nullptr) : 0;
}

extern "C" fc_status fc_datastore_extend(const uint16_t* tokens, uint64_t n, uint64_t n_new, const uint32_t* old_sa,
                                         const uint32_t* old_isa, uint32_t* sa_out, uint32_t* isa_out, void* ws,
                                         size_t ws_bytes, hipStream_t stream) {
  if (n >= 0xFFFFFFFFull || n_new > n) return FC_ERR_INVALID;
  if (n == 0) return FC_OK;
  const uint32_t o = (uint32_t)n_new, n_old = (uint32_t)(n - n_new);
  if (!tokens || !sa_out || (n_old > 0 && !old_sa)) return FC_ERR_INVALID;
  const bool isa_given = old_isa != nullptr;
  if (!ws || ws_bytes < fc_datastore_extend_workspace_bytes(n, n_new, isa_given ? 1 : 0)) return FC_ERR_WORKSPACE;
  (void)hipGetLastError();
  ExtendWs w;
  carve_extend(ws, n, n_new, isa_given, &w);
  const uint32_t* isa = isa_given ? old_isa : w.isa;
  const bool need_isa = n_old > 0 && (o > 0 || isa_out);
  if (need_isa && !isa_given) {
    hipLaunchKernelGGL(k_isa, dim3(fc::div_up(n_old, 256)), dim3(256), 0, stream, old_sa, n_old, w.isa);
    FC_CHECK_LAUNCH();
  }
  if (o > 0) {
    FC_CHECK_HIP(hipMemsetAsync(w.counts, 0, sizeof(uint32_t) * 4, stream));
    hipLaunchKernelGGL(k_ext_init, dim3(fc::div_up(o, 256)), dim3(256), 0, stream, tokens, o, (uint64_t)n, old_sa,
                       n_old, w.lo[0], w.hi[0], w.lo[1], w.hi[1], w.act[0], w.counts + 2);
    FC_CHECK_LAUNCH();
    uint32_t n_act = 0;
    FC_CHECK_HIP(hipMemcpyAsync(&n_act, w.counts + 2, sizeof(uint32_t), hipMemcpyDeviceToHost, stream));
    FC_CHECK_HIP(hipStreamSynchronize(stream));
    int cur = 0;
    uint32_t* act_in = w.act[0];
    uint32_t* act_out = w.act[1];
    for (uint64_t h = kExtFirst; n_act > 0; h *= 2) {
      if (h > 2 * n) return FC_ERR_DEVICE;  // every new suffix is final once p + h reaches the old text
      FC_CHECK_HIP(hipMemsetAsync(w.counts, 0, sizeof(uint32_t) * 2, stream));
      hipLaunchKernelGGL(k_ext_round, dim3(fc::div_up(n_act, 256)), dim3(256), 0, stream, o, (uint64_t)n, n_old,
                         old_sa, isa, h, w.lo[cur], w.hi[cur], w.lo[cur ^ 1], w.hi[cur ^ 1], act_in,
                         w.counts + 2, act_out, w.done, w.counts);
      FC_CHECK_LAUNCH();
      hipLaunchKernelGGL(k_ext_fix, dim3(fc::div_up(n_act, 256)), dim3(256), 0, stream, w.done, w.counts + 1,
                         w.lo[cur ^ 1], w.lo[cur], w.hi[cur]);
      FC_CHECK_LAUNCH();
      FC_CHECK_HIP(hipMemcpyAsync(w.counts + 2, w.counts, sizeof(uint32_t), hipMemcpyDeviceToDevice, stream));
      FC_CHECK_HIP(hipMemcpyAsync(&n_act, w.counts, sizeof(uint32_t), hipMemcpyDeviceToHost, stream));
      FC_CHECK_HIP(hipStreamSynchronize(stream));
      uint32_t* t = act_in;
      act_in = act_out;
      act_out = t;
      cur ^= 1;
    }
    // every range is final and in both buffers: w.lo[0] holds ins
    ExtendArgs ea;
    ea.ins = w.lo[0];
    ea.isa = isa;
    ea.ins_sorted = w.ins_sorted;
    ea.n = n;
    ea.n_old_bits = bit_length(n_old);
    fc_status s = build_sa(tokens, o, 0, w.b, nullptr, stream, &ea);
    if (s != FC_OK) return s;
    hipLaunchKernelGGL(k_ext_new_out, dim3(fc::div_up(o, 256)), dim3(256), 0, stream, w.b.rank, w.lo[0], o, sa_out);
    FC_CHECK_LAUNCH();
    if (isa_out) {
      hipLaunchKernelGGL(k_ext_isa_new, dim3(fc::div_up(o, 256)), dim3(256), 0, stream, w.b.rank, w.lo[0], o,
                         isa_out);
      FC_CHECK_LAUNCH();
    }
  }
  if (n_old > 0) {
    const uint32_t nc = coarse_entries(n_old);
    if (o > 0) {
      hipLaunchKernelGGL(k_ext_coarse, dim3(fc::div_up(nc, 256)), dim3(256), 0, stream, w.ins_sorted, o, nc,
                         w.coarse);
      FC_CHECK_LAUNCH();
    }
    hipLaunchKernelGGL(k_ext_old_out, dim3(nc - 1), dim3(256), 0, stream, old_sa, n_old, w.ins_sorted, w.coarse, o,
                       sa_out);
    FC_CHECK_LAUNCH();
    if (isa_out) {
      hipLaunchKernelGGL(k_ext_isa_old, dim3(fc::div_up(n_old, 256)), dim3(256), 0, stream, isa, n_old, w.ins_sorted,
                         w.coarse, o, isa_out);
      FC_CHECK_LAUNCH();
    }
  }
  return FC_OK;
}

extern "C" fc_status fc_store_prepare(const uint16_t* tokens, const uint32_t* sa, uint64_t n, uint32_t* bucket_out,
                                      hipStream_t stream) {
  if (n >= 0xFFFFFFFFull || !bucket_out) return FC_ERR_INVALID;
  if (n > 0 && (!tokens || !sa)) return FC_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_bucket, dim3(fc::div_up(FC_BUCKETS, 256)), dim3(256), 0, stream, tokens, sa, (uint32_t)n,
                     bucket_out);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" uint64_t fc_pair_table_entries(uint32_t V) { return (uint64_t)V * ((uint64_t)V + 1) + 1; }

extern "C" fc_status fc_store_prepare_pairs(const uint16_t* tokens, const uint32_t* sa, uint64_t n, uint32_t V,
                                            uint32_t* pair_out, hipStream_t stream) {
  if (n >= 0xFFFFFFFFull || !pair_out || V < 1 || V > 65536) return FC_ERR_INVALID;
  if (n > 0 && (!tokens || !sa)) return FC_ERR_INVALID;
  (void)hipGetLastError();
  if (n > 0) {
    // precondition: every token < V (pair_out[0] serves as the reduction cell)
    FC_CHECK_HIP(hipMemsetAsync(pair_out, 0, sizeof(uint32_t), stream));
    const uint32_t blocks = fc::div_up(n, 256) < 4096u ? fc::div_up(n, 256) : 4096u;
    hipLaunchKernelGGL(k_max_token, dim3(blocks), dim3(256), 0, stream, tokens, (uint32_t)n, pair_out);
    FC_CHECK_LAUNCH();
    uint32_t mx = 0;
    FC_CHECK_HIP(hipMemcpyAsync(&mx, pair_out, sizeof(uint32_t), hipMemcpyDeviceToHost, stream));
    FC_CHECK_HIP(hipStreamSynchronize(stream));
    if (mx >= V) return FC_ERR_INVALID;
  }
  if (n == 0) {  // every entry is 0
    FC_CHECK_HIP(hipMemsetAsync(pair_out, 0, sizeof(uint32_t) * fc_pair_table_entries(V), stream));
    return FC_OK;
  }
  const uint64_t threads = n + 1;
  hipLaunchKernelGGL(k_pairs, dim3((uint32_t)((threads + 255) / 256)), dim3(256), 0, stream, tokens, sa,
                     (uint32_t)n, V, pair_out);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" uint64_t fc_record_bytes(uint64_t n) { return (uint64_t)FC_RECORD_BYTES * n; }

namespace {

// entry t of the top-level sample: the first two 16-byte quads of record
// t * FC_TOP_STRIDE
__global__ void __launch_bounds__(256) k_top(const uint4* __restrict__ rec, uint64_t n_top,
                                               uint4* __restrict__ top) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;  // one quad per thread
  if (i >= 2 * n_top) return;
  const uint64_t t = i >> 1, q = i & 1;
  top[i] = rec[(t * FC_TOP_STRIDE) * (FC_RECORD_BYTES / 16) + q];
}

}  // namespace

extern "C" uint64_t fc_store_top_bytes(uint64_t n) {
  return ((n + FC_TOP_STRIDE - 1) / FC_TOP_STRIDE) * (uint64_t)FC_TOP_BYTES;
}

extern "C" fc_status fc_store_prepare_top(const void* rec, uint64_t n, void* top_out, hipStream_t stream) {
  if (n >= 0xFFFFFFFFull) return FC_ERR_INVALID;
  if (n == 0) return FC_OK;
  if (!rec || !top_out || ((uintptr_t)rec & (FC_RECORD_BYTES - 1)) || ((uintptr_t)top_out & (FC_TOP_BYTES - 1)))
    return FC_ERR_INVALID;
  const uint64_t n_top = (n + FC_TOP_STRIDE - 1) / FC_TOP_STRIDE;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_top, dim3(fc::div_up(2 * n_top, 256)), dim3(256), 0, stream, (const uint4*)rec, n_top,
                     (uint4*)top_out);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" fc_status fc_store_prepare_records(const uint16_t* tokens, const uint32_t* sa, uint64_t n, void* rec_out,
                                              hipStream_t stream) {
  if (n >= 0xFFFFFFFFull) return FC_ERR_INVALID;
  if (n == 0) return FC_OK;
  if (!tokens || !sa || !rec_out || ((uintptr_t)rec_out & (FC_RECORD_BYTES - 1))) return FC_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_records, dim3(fc::div_up(n, 256)), dim3(256), 0, stream, tokens, sa, (uint32_t)n,
                     (uint4*)rec_out);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
