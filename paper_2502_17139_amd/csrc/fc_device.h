// Device-side helpers shared by the library's kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fc {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Lanes below this one, as a 64-bit mask.
__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }

// Four 32-bit words at a 4-byte aligned address: one 16-byte load (the
// hardware takes multi-dword loads at dword alignment).
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

// ---- DPP wave primitives (32-bit).  Within each row of 16 lanes values move
// with DPP row shifts (plain VALU ops); rows are combined with readlane.
// Lanes whose DPP source falls outside the row take the identity explicitly,
// so the result does not depend on how out-of-row reads are filled.  Call
// with the whole wave active.

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

constexpr int kRowShr1 = 0x111, kRowShr2 = 0x112, kRowShr4 = 0x114, kRowShr8 = 0x118;
constexpr int kRowShl1 = 0x101, kRowShl2 = 0x102, kRowShl4 = 0x104, kRowShl8 = 0x108;

// The value of the lane below (lane 0 gets `fill`): one DPP wave shift
// (wave_shr:1 crosses the rows of 16 lanes).
__device__ __forceinline__ uint32_t wave_shr1(uint32_t x, uint32_t fill) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)fill, (int)x, 0x138, 0xF, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes.
__device__ __forceinline__ uint32_t wave_incl_sum_u32(uint32_t v) {
  const int r = lane_id() & 15;
  uint32_t x = v, y;
  y = dpp_mov<kRowShr1>(x); x += r >= 1 ? y : 0u;
  y = dpp_mov<kRowShr2>(x); x += r >= 2 ? y : 0u;
  y = dpp_mov<kRowShr4>(x); x += r >= 4 ? y : 0u;
  y = dpp_mov<kRowShr8>(x); x += r >= 8 ? y : 0u;
  const uint32_t t0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t t1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t t2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = lane_id() >> 4;
  return x + (row == 0 ? 0u : row == 1 ? t0 : row == 2 ? t0 + t1 : t0 + t1 + t2);
}

// Sum over the 64 lanes (every lane gets it).
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
  const int r = lane_id() & 15;
  uint32_t x = v, y;
  y = dpp_mov<kRowShr1>(x); x += r >= 1 ? y : 0u;
  y = dpp_mov<kRowShr2>(x); x += r >= 2 ? y : 0u;
  y = dpp_mov<kRowShr4>(x); x += r >= 4 ? y : 0u;
  y = dpp_mov<kRowShr8>(x); x += r >= 8 ? y : 0u;
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 15) + (uint32_t)__builtin_amdgcn_readlane((int)x, 31) +
         (uint32_t)__builtin_amdgcn_readlane((int)x, 47) + (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Minimum over the lanes above this one (ident for lane 63); *total gets
// the minimum over the whole wave.
__device__ __forceinline__ uint32_t wave_excl_suffix_min_u32(uint32_t v, uint32_t ident, uint32_t* total) {
  const int r = lane_id() & 15;
  uint32_t x = v, y;
  y = dpp_mov<kRowShl1>(x); x = (r <= 14 && y < x) ? y : x;
  y = dpp_mov<kRowShl2>(x); x = (r <= 13 && y < x) ? y : x;
  y = dpp_mov<kRowShl4>(x); x = (r <= 11 && y < x) ? y : x;
  y = dpp_mov<kRowShl8>(x); x = (r <= 7 && y < x) ? y : x;
  // x = minimum over lanes r..15 of this row
  y = dpp_mov<kRowShl1>(x);
  uint32_t ex = r <= 14 ? y : ident;  // lanes r+1..15 of this row
  const uint32_t m1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 16);
  const uint32_t m2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 32);
  const uint32_t m3 = (uint32_t)__builtin_amdgcn_readlane((int)x, 48);
  const uint32_t m0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 0);
  const uint32_t t3 = m3, t2 = m2 < t3 ? m2 : t3, t1 = m1 < t2 ? m1 : t2;
  const int row = lane_id() >> 4;
  const uint32_t tail = row == 0 ? t1 : row == 1 ? t2 : row == 2 ? t3 : ident;
  ex = tail < ex ? tail : ex;
  *total = m0 < t1 ? m0 : t1;
  return ex;
}

template <typename T>
__device__ __forceinline__ T wave_incl_sum(T v) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T n = __shfl_up(v, off, kWave);
    if (l >= off) v += n;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_incl_max(T v) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T n = __shfl_up(v, off, kWave);
    if (l >= off && n > v) v = n;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_max(T v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    T n = __shfl_xor(v, off, kWave);
    v = n > v ? n : v;
  }
  return v;
}

template <typename T>
__device__ __forceinline__ T wave_min(T v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) {
    T n = __shfl_xor(v, off, kWave);
    v = n < v ? n : v;
  }
  return v;
}

// Exclusive prefix sum over the block (blockDim.x a multiple of 64, at most
// 1024).  scratch holds at least blockDim.x/64 + 1 entries.  Every thread of
// the block must call it; it contains barriers.  *total receives the sum.
template <typename T>
__device__ __forceinline__ T wave_incl_sum_any(T v) {
  if constexpr (sizeof(T) == 4) return (T)wave_incl_sum_u32((uint32_t)v);
  else return wave_incl_sum(v);
}

template <typename T>
__device__ __forceinline__ T block_excl_sum(T v, T* scratch, T* total) {
  const int nw = (int)(blockDim.x / kWave), w = (int)(threadIdx.x / kWave);
  T inc = wave_incl_sum_any(v);
  if (lane_id() == kWave - 1) scratch[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = 0;
    for (int i = 0; i < nw; ++i) {
      T x = scratch[i];
      scratch[i] = run;
      run += x;
    }
    scratch[nw] = run;
  }
  __syncthreads();
  T res = scratch[w] + inc - v;
  if (total) *total = scratch[nw];
  __syncthreads();
  return res;
}

// Exclusive prefix maximum over the block (identity `ident`); same contract
// as block_excl_sum.
template <typename T>
__device__ __forceinline__ T block_excl_max(T v, T ident, T* scratch) {
  const int nw = (int)(blockDim.x / kWave), w = (int)(threadIdx.x / kWave);
  T inc = wave_incl_max(v);
  T exc = __shfl_up(inc, 1, kWave);
  if (lane_id() == 0) exc = ident;
  if (lane_id() == kWave - 1) scratch[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = ident;
    for (int i = 0; i < nw; ++i) {
      T x = scratch[i];
      scratch[i] = run;
      run = x > run ? x : run;
    }
  }
  __syncthreads();
  T pre = scratch[w];
  T res = exc > pre ? exc : pre;
  __syncthreads();
  return res;
}

// Exclusive prefix minimum over the block (identity `ident`); same contract
// as block_excl_sum.
template <typename T>
__device__ __forceinline__ T block_excl_min(T v, T ident, T* scratch) {
  const int nw = (int)(blockDim.x / kWave), w = (int)(threadIdx.x / kWave);
  const int l = lane_id();
  T inc = v;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T n = __shfl_up(inc, off, kWave);
    if (l >= off && n < inc) inc = n;
  }
  T exc = __shfl_up(inc, 1, kWave);
  if (l == 0) exc = ident;
  if (l == kWave - 1) scratch[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = ident;
    for (int i = 0; i < nw; ++i) {
      T x = scratch[i];
      scratch[i] = run;
      run = x < run ? x : run;
    }
  }
  __syncthreads();
  T pre = scratch[w];
  T res = exc < pre ? exc : pre;
  __syncthreads();
  return res;
}

// Block-wide sum (all threads get it).
template <typename T>
__device__ __forceinline__ T block_sum(T v, T* scratch) {
  T total;
  (void)block_excl_sum(v, scratch, &total);
  return total;
}

// Block-wide maximum (all threads get it).
template <typename T>
__device__ __forceinline__ T block_max(T v, T* scratch) {
  const int nw = (int)(blockDim.x / kWave), w = (int)(threadIdx.x / kWave);
  T m = wave_max(v);
  if (lane_id() == 0) scratch[w] = m;
  __syncthreads();
  T r = scratch[0];
  for (int i = 1; i < nw; ++i) r = scratch[i] > r ? scratch[i] : r;
  __syncthreads();
  return r;
}

__host__ __device__ __forceinline__ uint32_t div_up(uint64_t a, uint64_t b) { return (uint32_t)((a + b - 1) / b); }

// Row of query b under an optional row map: rows[b] when it lies in
// [0, n_rows), -1 when it does not, b when there is no map.
__device__ __forceinline__ int map_row(const int32_t* rows, int n_rows, int b) {
  if (!rows) return b;
  const int r = rows[b];
  return (r >= 0 && r < n_rows) ? r : -1;
}

typedef int int32x4 __attribute__((ext_vector_type(4)));

// Buffer resource over `bytes` bytes at p (raw, no stride): loads at or past
// `bytes` return zeros.
__device__ __forceinline__ int32x4 buffer_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)p;
  int32x4 r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));
  r.z = __builtin_amdgcn_readfirstlane((int)bytes);
  r.w = 0x00020000;
  return r;
}

// One wave loads 64 x 16 bytes from the buffer at byte offsets voff (one per
// lane) into LDS bytes [lds, lds + 1024), lane L at lds + 16 L.  The load is
// counted by vmcnt like any vector load; the compiler does not track it.
__device__ __forceinline__ void lds_load16(uint32_t lds, uint32_t voff, int32x4 rsrc) {
  asm volatile("s_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds"
               :
               : "v"(voff), "s"(__builtin_amdgcn_readfirstlane((int)lds)), "s"(rsrc)
               : "memory");
}


// Greedy acceptance walk of one draft tree by one wave (Section IV-D):
// from the root, step to the child whose token equals target(u) while one
// exists; the target at the stopping row is accepted too.  Rows 1..n-1 of
// the tree (n clamped to [1, R]) are held four per lane, with the targets of
// rows 0..n-1 loaded beside them before the walk, so that each step is one
// ballot per 64 rows and one lane shuffle instead of a dependent load.  The
// row loads do not wait for n: every row v < R is read (target(v) is called
// for each and must be safe for each) and rows at n or past it are masked.
// Writes the accepted tokens (m + 1 slots, -1 past the end) and returns the
// accepted length and the last row in len and u.
template <int MAXROWS, typename Target>
__device__ __forceinline__ void accept_walk(int n, const int32_t* __restrict__ node_tok,
                                            const int32_t* __restrict__ parent, int R, int m, Target target,
                                            int32_t* __restrict__ out, int& len, int& u) {
  constexpr int kChunks = MAXROWS / kWave;
  const int lane = lane_id();
  n = n < 1 ? 1 : (n > R ? R : n);
  int32_t par[kChunks], tok[kChunks], tgt[kChunks];
#pragma unroll
  for (int h = 0; h < kChunks; ++h) {
    const int v = lane + h * kWave;
    par[h] = v < R ? parent[v] : -2;
    tok[h] = v < R ? node_tok[v] : -1;
    tgt[h] = v < R ? target(v) : -1;
  }
#pragma unroll
  for (int h = 0; h < kChunks; ++h) {
    const int v = lane + h * kWave;
    if (v < 1 || v >= n) par[h] = -2, tok[h] = -1;
    if (v >= n) tgt[h] = -1;
  }
  // target of row x < n (x wave-uniform): its chunk, then its lane.
  const auto target_of = [&](int x) -> int32_t {
    int32_t t = tgt[0];
#pragma unroll
    for (int h = 1; h < kChunks; ++h)
      if (x / kWave == h) t = tgt[h];
    return __shfl(t, x % kWave, kWave);
  };
  u = 0;
  len = 0;
  for (;;) {
    const int32_t want = target_of(u);
    if (want < 0 || len >= m + 1) break;
    int next = -1;
#pragma unroll
    for (int h = 0; h < kChunks; ++h) {
      const uint64_t hit = ballot(par[h] == u && tok[h] == want);
      if (next < 0 && hit) next = h * kWave + (int)__builtin_ctzll(hit);
    }
    if (next < 0) break;
    if (lane == 0) out[len] = want;
    ++len;
    u = next;
  }
  const int32_t bonus = target_of(u);
  if (bonus >= 0 && len < m + 1) {
    if (lane == 0) out[len] = bonus;
    ++len;
  }
  for (int x = len + lane; x < m + 1; x += kWave) out[x] = -1;
}

// accept_walk for targets that depend only on a row's depth (a replay's
// ground truth: the target of a row at depth d is the truth token d places
// after the stream's position).  A path row at depth d is reached after d
// accepted tokens, so the walk takes its target from lane `len` of win
// (lane d holds the target at depth d, or -1); requires m + 1 <= 64.
template <int MAXROWS>
__device__ __forceinline__ void accept_walk_depth(int n, const int32_t* __restrict__ node_tok,
                                                  const int32_t* __restrict__ parent, int R, int m, int32_t win,
                                                  int32_t* __restrict__ out, int& len, int& u) {
  constexpr int kChunks = MAXROWS / kWave;
  const int lane = lane_id();
  n = n < 1 ? 1 : (n > R ? R : n);
  int32_t par[kChunks], tok[kChunks];
#pragma unroll
  for (int h = 0; h < kChunks; ++h) {
    const int v = lane + h * kWave;
    par[h] = v < R ? parent[v] : -2;
    tok[h] = v < R ? node_tok[v] : -1;
  }
#pragma unroll
  for (int h = 0; h < kChunks; ++h) {
    const int v = lane + h * kWave;
    if (v < 1 || v >= n) par[h] = -2, tok[h] = -1;
  }
  u = 0;
  len = 0;
  for (;;) {
    const int32_t want = len <= m ? __shfl(win, len, kWave) : -1;
    if (want < 0) break;
    int next = -1;
#pragma unroll
    for (int h = 0; h < kChunks; ++h) {
      const uint64_t hit = ballot(par[h] == u && tok[h] == want);
      if (next < 0 && hit) next = h * kWave + (int)__builtin_ctzll(hit);
    }
    if (next < 0) break;
    if (lane == 0) out[len] = want;
    ++len;
    u = next;
  }
  const int32_t bonus = len <= m ? __shfl(win, len, kWave) : -1;
  if (bonus >= 0) {
    if (lane == 0) out[len] = bonus;
    ++len;
  }
  for (int x = len + lane; x < m + 1; x += kWave) out[x] = -1;
}

}  // namespace fc
