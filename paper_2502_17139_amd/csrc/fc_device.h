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
__device__ __forceinline__ T block_excl_sum(T v, T* scratch, T* total) {
  const int nw = (int)(blockDim.x / kWave), w = (int)(threadIdx.x / kWave);
  T inc = wave_incl_sum(v);
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

}  // namespace fc
