// Tree attention of draft trees on gfx950 matrix cores (fc_tree_attention).
//
// The draft tree is verified in one forward pass of the target model
// (Section IV-D, eq. (4)): row i of tree b sits at position prefix_len[b] +
// pos_ids[b][i] and attends to every cached prefix token and to the tree
// rows j with mask[b][i][j] = 1.  This is the layer's attention step for
// those rows, with the rotary embedding of the queries and the tree's keys
// applied by their positions (cached keys are stored rotated).
//
// One workgroup per (tree, query head); one wave per 16 tree rows.  Keys
// and values stream through LDS in blocks of 32 (the cached prefix first,
// then the tree), shared by the workgroup's waves.  Per block a wave
// computes the transposed scores S^T = K Q^T with 16x16x32 bf16 MFMAs (two
// 16-key tiles), applies the mask, updates a running softmax (fp32) and
// accumulates O^T += V^T P^T with eight more MFMAs over the 128 output
// dims.  Working on the transposes keeps every operand in the lane layout
// the MFMA wants: a lane's eight scores are exactly its eight probabilities
// of the value product, so nothing is shuffled between the two products.
//
// The cached prefix moves straight from HBM into LDS with buffer loads that
// write LDS (16 bytes a lane, no registers), through a ring of four blocks,
// so three blocks are in flight while one is used; the loads of rows past
// the prefix fall outside the buffer's range and read as zeros.  Rows sit in
// LDS as written (key-major), each 16-byte chunk XOR-swizzled by the row, so
// the score product reads K rows without bank conflicts and the value
// product takes V^T with the transposing LDS read (ds_read_b64_tr_b16),
// which hands each lane four keys of one output dim.  The tree's own keys
// are rotated on the way in, through registers.  Workgroups are numbered so
// that the query heads sharing a key head run on the same XCD and its L2
// serves their shared key/value reads.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kD = FC_TREE_ATTN_HEAD_DIM;   // 128
constexpr int kBlock = 32;                  // keys per block
constexpr int kRowBytes = kD * 2;           // 256: one key row
constexpr int kPart = kBlock * kRowBytes;   // 8 KB: a block's keys (or values)
constexpr int kStage = 2 * kPart;           // keys then values
constexpr int kStages = 4;                  // ring depth
constexpr int kDTiles = kD / 16;            // output tiles of 16 dims
constexpr int kDSteps = kD / 32;            // 32-dim steps of the score product
constexpr int kDmaWaves = 4;                // waves issuing a block's 16 loads, 4 each
constexpr int kXcds = 8;

__device__ __forceinline__ __bf16 f2bf(float x) { return (__bf16)x; }

// byte offset inside a block part of 16-byte chunk c of row r (swizzled)
__device__ __forceinline__ uint32_t chunk_at(int r, int c) { return (uint32_t)(r * kRowBytes + ((c ^ (r & 15)) << 4)); }

// sin and cos of the rotary angle position * base^(-2d/D) of the pair (d,
// d + D/2).  The angle is taken in revolutions and reduced to [0, 1) in
// double precision, so large positions keep full accuracy; the hardware
// sine and cosine then take revolutions directly.
__device__ __forceinline__ void rope_sincos(int pos, int d, double log2_base, float& s, float& c) {
  constexpr double kInv2Pi = 0.15915494309189533577;
  const double rev = (double)pos * exp2(-2.0 * (double)d / (double)kD * log2_base) * kInv2Pi;
  const float f = (float)(rev - floor(rev));
  s = __builtin_amdgcn_sinf(f);
  c = __builtin_amdgcn_cosf(f);
}

// 8 bf16 (16 bytes) at p as floats.
__device__ __forceinline__ void load8(const uint16_t* __restrict__ p, float (&v)[8]) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[2 * e] = __uint_as_float(w[e] << 16);
    v[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
  }
}

template <int MAXT>
__global__ void __launch_bounds__(MAXT) k_tree_attn(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_tree, const uint16_t* __restrict__ v_tree,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ prefix_len, const int32_t* __restrict__ num_nodes, const int32_t* __restrict__ mask,
    const int32_t* __restrict__ pos_ids, int B, int R, int H, int Hkv, int Pmax, double log2_base,
    float* __restrict__ out) {
  __shared__ __align__(16) uint8_t s_ring[kStages * kStage];

  // workgroup -> (tree, head): consecutive ids on one XCD when the count
  // divides evenly, so the heads of one key head share an L2
  const int total = B * H;
  const int x = (int)blockIdx.x;
  const int lin = (total % kXcds == 0) ? (x % kXcds) * (total / kXcds) + x / kXcds : x;
  const int b = lin / H, h = lin - (lin / H) * H;
  const int g_kv = h / (H / Hkv);
  const int tid = (int)threadIdx.x, nt = (int)blockDim.x;
  const int lane = fc::lane_id(), w = tid / fc::kWave;
  const int lg = lane >> 4, lc = lane & 15;  // lane group (0..3), lane column (0..15)
  // lengths from the device are clamped to the buffers (a malformed tree,
  // num_nodes = -1, has no rows)
  const int P = prefix_len[b] < 0 ? 0 : (prefix_len[b] > Pmax ? Pmax : prefix_len[b]);
  const int n = num_nodes[b] < 0 ? 0 : (num_nodes[b] > R ? R : num_nodes[b]);
  const uint32_t ring = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)s_ring;

  // Prefix block loads: load u (0..15) of a block covers rows 4(u%8) ..
  // 4(u%8)+3 of the keys (u < 8) or values; lane L takes row 4(u%8) + L/16
  // and fills physical chunk L%16, i.e. logical chunk (L%16) ^ (row%16).
  // Waves 0..3 issue loads w, w+4, w+8, w+12 of every block.
  const int64_t row_stride = (int64_t)Hkv * kD * 2;  // bytes between consecutive keys
  const uint32_t pre_bytes = P > 0 ? (uint32_t)((int64_t)(P - 1) * row_stride + kRowBytes) : 0u;
  const fc::int32x4 rk = fc::buffer_rsrc(k_cache + ((int64_t)b * Pmax * Hkv + g_kv) * kD, pre_bytes);
  const fc::int32x4 rv = fc::buffer_rsrc(v_cache + ((int64_t)b * Pmax * Hkv + g_kv) * kD, pre_bytes);
  const bool dma_wave = w < kDmaWaves;
  auto issue_block = [&](int blk) {  // rows past P (also whole blocks past the prefix) read as zeros
    if (!dma_wave) return;
    const uint32_t slot = ring + (uint32_t)((blk % kStages) * kStage);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int u = w + kDmaWaves * i;
      const int r = 4 * (u & 7) + (lane >> 4);
      const int c = (lane & 15) ^ (r & 15);
      const int64_t key = (int64_t)blk * kBlock + r;
      const uint32_t voff = key < P ? (uint32_t)(key * row_stride + 16 * c) : pre_bytes;
      fc::lds_load16(slot + (u < 8 ? 0u : (uint32_t)kPart) + (uint32_t)(u & 7) * 1024u, voff, u < 8 ? rk : rv);
    }
  };

  // this lane's query row and its rotated dims as the B operand of S^T
  const int qr = w * 16 + lc;
  const bool q_in = qr < R;
  bf16x8 qf[kDSteps];
  {
    float v[kDSteps][8];
#pragma unroll
    for (int kc = 0; kc < kDSteps; ++kc) {
      if (q_in) load8(q + (((int64_t)b * R + qr) * H + h) * kD + 32 * kc + 8 * lg, v[kc]);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) v[kc][e] = 0.0f;
    }
    const int pos = P + (q_in ? pos_ids[(int64_t)b * R + qr] : 0);
#pragma unroll
    for (int kc = 0; kc < kDSteps / 2; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // dims d and d + D/2 sit in steps kc and kc + 2 of the same lane
        float s, c;
        rope_sincos(pos, 32 * kc + 8 * lg + e, log2_base, s, c);
        const float x0 = v[kc][e], x1 = v[kc + 2][e];
        v[kc][e] = x0 * c - x1 * s;
        v[kc + 2][e] = x1 * c + x0 * s;
      }
#pragma unroll
    for (int kc = 0; kc < kDSteps; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[kc][e] = f2bf(v[kc][e]);
  }

  floatx4 o[kDTiles];
#pragma unroll
  for (int t = 0; t < kDTiles; ++t) o[t] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_run = -INFINITY, l_run = 0.0f;
  const float scale = 1.0f / sqrtf((float)kD);

  // One block of the two products from the K and V parts at slot_off (a byte
  // offset in s_ring); `tree` blocks take the mask, prefix blocks only the
  // prefix bound.
  auto consume = [&](uint32_t slot_off, int base, int lim, bool tree) {
    const uint8_t* sk = s_ring + slot_off;
    floatx4 st0 = {0.0f, 0.0f, 0.0f, 0.0f}, st1 = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kc = 0; kc < kDSteps; ++kc) {
      const bf16x8 a0 = *(const bf16x8*)(sk + chunk_at(lc, 4 * kc + lg));
      const bf16x8 a1 = *(const bf16x8*)(sk + chunk_at(16 + lc, 4 * kc + lg));
      st0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, qf[kc], st0, 0, 0, 0);
      st1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, qf[kc], st1, 0, 0, 0);
    }
    // this lane holds keys 4*lg + i and 16 + 4*lg + i for query row qr
    float sv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int kk = e < 4 ? 4 * lg + e : 16 + 4 * lg + (e - 4);
      const int j = base + kk;
      bool ok = j < lim && q_in;
      if (ok && tree) ok = qr < n && mask[((int64_t)b * R + qr) * R + j] == 1;
      const float raw = e < 4 ? st0[e] : st1[e - 4];
      sv[e] = ok ? raw * scale : -INFINITY;
    }
    float mb = sv[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mb = fmaxf(mb, sv[e]);
    mb = fmaxf(mb, __shfl_xor(mb, 16));
    mb = fmaxf(mb, __shfl_xor(mb, 32));
    const float m_new = fmaxf(m_run, mb);
    const bool none = m_new == -INFINITY;  // no allowed key for this row yet
    const float alpha = none ? 1.0f : __expf(m_run - m_new);
    bf16x8 pb;
    float ps = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pe = none ? 0.0f : __expf(sv[e] - m_new);
      ps += pe;
      pb[e] = f2bf(pe);
    }
    m_run = m_new;
    l_run = l_run * alpha + ps;
    // V^T for output tile t: a transposing read gives lane (lg, lc) dims
    // 16t + lc of keys 4lg + e (first read) and 16 + 4lg + e (second); the
    // addressing lane (lg, 4e + i) points at dims 16t + 4i of that key
    const uint32_t vbase = ring + slot_off + (uint32_t)kPart;
    const int vr0 = 4 * lg + (lc >> 2), vr1 = 16 + 4 * lg + (lc >> 2), vq = lc & 3;
#pragma unroll
    for (int t = 0; t < kDTiles; ++t) {
      o[t] *= alpha;
      const int cc = 2 * t + (vq >> 1);
      const uint32_t half = (uint32_t)(vq & 1) * 8u;
      const bf16x4 lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (lds_bf16x4*)(uintptr_t)(vbase + chunk_at(vr0, cc) + half));
      const bf16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (lds_bf16x4*)(uintptr_t)(vbase + chunk_at(vr1, cc) + half));
      const bf16x8 a = {lo4[0], lo4[1], lo4[2], lo4[3], hi4[0], hi4[1], hi4[2], hi4[3]};
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb, o[t], 0, 0, 0);
    }
  };

  // the cached prefix: a ring of kStages blocks, kStages - 1 in flight
  const int n_pre = (P + kBlock - 1) / kBlock, n_tree = (n + kBlock - 1) / kBlock;
#pragma unroll
  for (int blk = 0; blk < kStages - 1; ++blk) issue_block(blk);
  for (int blk = 0; blk < n_pre; ++blk) {
    // this wave's loads of block blk are done once at most the loads of the
    // kStages - 2 later blocks (4 each) are outstanding; the barrier makes every
    // wave's visible, and frees the slot the next issue overwrites
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(4 * (kStages - 2)) : "memory");
    __syncthreads();
    issue_block(blk + kStages - 1);
    consume((uint32_t)((blk % kStages) * kStage), blk * kBlock, P, false);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // the tree's rows: keys rotated by their positions, values as they are,
  // staged through registers into slot 0
  for (int tb = 0; tb < n_tree; ++tb) {
    const int base = tb * kBlock;
    uint8_t* sk = s_ring;
    for (int it = tid; it < kBlock * (kD / 16); it += nt) {
      const int kk = it / (kD / 16), c = it - kk * (kD / 16);  // key, chunks c and c + D/16
      const int j = base + kk;
      float a[8], bb[8];
      if (j < n) {
        const uint16_t* src = k_tree + (((int64_t)b * R + j) * Hkv + g_kv) * kD;
        load8(src + 8 * c, a);
        load8(src + kD / 2 + 8 * c, bb);
        const int pos = P + pos_ids[(int64_t)b * R + j];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          float sn, cs;
          rope_sincos(pos, 8 * c + e, log2_base, sn, cs);
          const float x0 = a[e], x1 = bb[e];
          a[e] = x0 * cs - x1 * sn;
          bb[e] = x1 * cs + x0 * sn;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] = bb[e] = 0.0f;
      }
      bf16x8 pa, pbb;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pa[e] = f2bf(a[e]);
        pbb[e] = f2bf(bb[e]);
      }
      *(bf16x8*)(sk + chunk_at(kk, c)) = pa;
      *(bf16x8*)(sk + chunk_at(kk, c + kD / 16)) = pbb;
    }
    for (int it = tid; it < kBlock * (kD / 8); it += nt) {
      const int kk = it / (kD / 8), c = it - kk * (kD / 8);
      const int j = base + kk;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (j < n) v = *(const uint4*)(v_tree + (((int64_t)b * R + j) * Hkv + g_kv) * kD + 8 * c);
      *(uint4*)(sk + kPart + chunk_at(kk, c)) = v;
    }
    __syncthreads();
    consume(0u, base, n, true);
    __syncthreads();
  }

  // normalise by the row's total weight (summed over the four lane groups)
  float lt = l_run + __shfl_xor(l_run, 16);
  lt = lt + __shfl_xor(lt, 32);
  if (q_in) {
    const bool live = qr < n && lt > 0.0f;
    const float inv = live ? 1.0f / lt : 0.0f;
    float* dst = out + (((int64_t)b * R + qr) * H + h) * kD;
#pragma unroll
    for (int t = 0; t < kDTiles; ++t) {
      floatx4 r = o[t] * inv;
      *(floatx4*)(dst + 16 * t + 4 * lg) = r;
    }
  }
}

}  // namespace

extern "C" fc_status fc_tree_attention(const uint16_t* q, const uint16_t* k_tree, const uint16_t* v_tree,
                                       const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* prefix_len,
                                       const int32_t* num_nodes, const int32_t* mask, const int32_t* pos_ids,
                                       int32_t B, int32_t R, int32_t H, int32_t Hkv, int32_t D, int32_t Pmax,
                                       float rope_base, float* out, hipStream_t stream) {
  if (B < 0 || R < 1 || R > FC_MAX_TREE_ROWS || H < 1 || Hkv < 1 || H % Hkv != 0 || Pmax < 0) return FC_ERR_INVALID;
  if (!(rope_base > 1.0f)) return FC_ERR_INVALID;
  if (D != FC_TREE_ATTN_HEAD_DIM) return FC_ERR_UNSUPPORTED;
  if (B == 0) return FC_OK;
  if (!q || !k_tree || !v_tree || !prefix_len || !num_nodes || !mask || !pos_ids || !out) return FC_ERR_INVALID;
  if (Pmax > 0 && (!k_cache || !v_cache)) return FC_ERR_INVALID;
  const uintptr_t al = (uintptr_t)q | (uintptr_t)k_tree | (uintptr_t)v_tree | (uintptr_t)out |
                       (Pmax > 0 ? ((uintptr_t)k_cache | (uintptr_t)v_cache) : 0);
  if (al & 15) return FC_ERR_INVALID;
  // the prefix of one (tree, key head) is read with 32-bit byte offsets
  if ((int64_t)Pmax * Hkv * D * 2 >= (int64_t)1 << 32) return FC_ERR_UNSUPPORTED;
  const int rows_waves = (R + 15) / 16;
  const int waves = rows_waves < 4 ? 4 : rows_waves;  // at least 256 threads stage a block
  const dim3 grid((uint32_t)B * (uint32_t)H), block(waves * fc::kWave);
  (void)hipGetLastError();
  // trees of up to 128 rows (c <= 127) in workgroups of at most 8 waves,
  // which leaves each lane the registers the accumulators need
  if (waves <= 8)
    hipLaunchKernelGGL(k_tree_attn<512>, grid, block, 0, stream, q, k_tree, v_tree, k_cache, v_cache, prefix_len,
                       num_nodes, mask, pos_ids, B, R, H, Hkv, Pmax, log2((double)rope_base), out);
  else
    hipLaunchKernelGGL(k_tree_attn<1024>, grid, block, 0, stream, q, k_tree, v_tree, k_cache, v_cache, prefix_len,
                       num_nodes, mask, pos_ids, B, R, H, Hkv, Pmax, log2((double)rope_base), out);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
