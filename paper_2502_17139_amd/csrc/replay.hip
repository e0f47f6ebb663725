// Device-resident decode-trace replay (fc_replay_init, fc_replay_run).
//
// The draft stage driven over known token streams as a stand-in for a
// decoding loop, the way the average acceptance length is measured
// (Section V-C, eq. (7)): every step each live stream looks its 16-token
// context up in an LRU of its recent retrievals, retrieves on a miss
// (Section III-A over the stores in priority order), builds its draft tree
// (Section IV-D), takes the true next tokens as the target model's outputs,
// accepts greedily and advances by the accepted length.
//
// Everything a step decides lives on the GPU, so a step is a fixed chain of
// launches on one stream with no host round trip:
//   k_replay_prepare   one wave per stream: the context from the stream, the
//                      LRU probe (keys compared by the lanes, least recent
//                      slot by a wave minimum), the row maps;
//   fc_retrieve        every stream, misses into their LRU slot (hits and
//                      finished streams have no row and are skipped);
//   fc_build_tree      every live stream from its slot;
//   fc_targets_from_truth, fc_verify_accept;
//   k_replay_advance   one thread per stream: position += accepted length,
//                      the step's history row and the live count.
// The LRU keeps the exact semantics of an ordered map: slots fill in order,
// a hit becomes most recent, a miss in a full table replaces the least
// recently used slot (last-use steps are distinct per stream).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kPrepThreads = 256;
constexpr int kStreamsPerBlock = kPrepThreads / fc::kWave;

__global__ void __launch_bounds__(256) k_replay_init(int32_t n, int32_t L, int32_t* __restrict__ pos,
                                                     int32_t* __restrict__ lru_count, int32_t* __restrict__ hits,
                                                     int32_t* __restrict__ lookups, int32_t* __restrict__ live,
                                                     int32_t truth_len) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b == 0) *live = L < truth_len ? n : 0;
  if (b >= n) return;
  pos[b] = L;
  lru_count[b] = 0;
  hits[b] = 0;
  lookups[b] = 0;
}

__global__ void __launch_bounds__(kPrepThreads) k_replay_prepare(fc_replay r, int32_t step) {
  const int lane = fc::lane_id();
  const int b = blockIdx.x * kStreamsPerBlock + (int)threadIdx.x / fc::kWave;
  if (blockIdx.x == 0 && threadIdx.x == 0) *r.live = 0;
  if (b >= r.n_streams) return;
  const int L = r.ctx_len, lru = r.lru;
  const int p = r.pos[b];
  if (p >= r.truth_len) {  // finished: no retrieval, no tree row
    if (lane == 0) {
      r.rows_retrieve[b] = -1;
      r.rows_tree[b] = -1;
    }
    return;
  }
  // the context: the L tokens before the position
  const uint16_t* src = r.truth + (int64_t)b * r.truth_stride + (p - L);
  uint16_t* ctx = r.ctx + (int64_t)b * L;
  const uint16_t tok = lane < L ? src[lane] : (uint16_t)0;
  if (lane < L) ctx[lane] = tok;
  // probe: lane e compares slot e's key with the context
  const int count = r.lru_count[b];
  const uint16_t* keys = r.lru_key + (int64_t)b * lru * L;
  int32_t* used = r.lru_used + (int64_t)b * lru;
  bool match = false;
  if (lane < count) {
    match = true;
    const uint16_t* key = keys + (int64_t)lane * L;
    for (int t = 0; t < L; ++t) match &= key[t] == src[t];
  }
  const uint64_t hit_mask = fc::ballot(match);
  int slot;
  if (hit_mask) {
    slot = __builtin_ctzll(hit_mask);
  } else if (count < lru) {
    slot = count;
  } else {
    // least recently used: the smallest last-use step (distinct per stream)
    int best = lane < lru ? used[lane] : 0x7FFFFFFF;
    int arg = lane;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      const int ob = __shfl_xor(best, off), oa = __shfl_xor(arg, off);
      if (ob < best || (ob == best && oa < arg)) {
        best = ob;
        arg = oa;
      }
    }
    slot = arg;
  }
  if (!hit_mask && lane < L) r.lru_key[((int64_t)b * lru + slot) * L + lane] = tok;
  if (lane == 0) {
    used[slot] = step;
    if (!hit_mask && count < lru) r.lru_count[b] = count + 1;
    r.lookups[b] += 1;
    r.hits[b] += hit_mask ? 1 : 0;
    const int row = b * lru + slot;
    r.rows_retrieve[b] = hit_mask ? -1 : row;
    r.rows_tree[b] = row;
  }
}

__global__ void __launch_bounds__(256) k_replay_advance(fc_replay r, int32_t step) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= r.n_streams) return;
  int32_t* hist = r.history + (int64_t)step * r.n_streams;
  const int p = r.pos[b];
  if (p >= r.truth_len) {
    hist[b] = -1;
    return;
  }
  const int a = r.accept_len[b];
  hist[b] = a;
  r.pos[b] = p + a;
  if (p + a < r.truth_len) atomicAdd(r.live, 1);
}

}  // namespace

extern "C" fc_status fc_replay_init(fc_replay* r, hipStream_t stream) {
  if (!r || r->n_streams < 1 || r->ctx_len < 1 || r->ctx_len > fc::kWave || r->lru < 1 || r->lru > fc::kWave)
    return FC_ERR_INVALID;
  if (!r->pos || !r->lru_count || !r->hits || !r->lookups || !r->live) return FC_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_replay_init, dim3(fc::div_up(r->n_streams, 256)), dim3(256), 0, stream, r->n_streams,
                     r->ctx_len, r->pos, r->lru_count, r->hits, r->lookups, r->live, r->truth_len);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" fc_status fc_replay_run(const fc_store* stores, int32_t S, const fc_replay* r, int32_t first_step,
                                   int32_t n_steps, hipStream_t stream) {
  if (!r || !stores || S < 1 || S > FC_MAX_SOURCES) return FC_ERR_INVALID;
  if (r->n_streams < 1 || r->ctx_len < 1 || r->ctx_len > fc::kWave || r->lru < 1 || r->lru > fc::kWave)
    return FC_ERR_INVALID;
  if (r->truth_len < 0 || r->truth_stride < r->truth_len || !r->truth) return FC_ERR_INVALID;
  if (first_step < 0 || n_steps < 0 || (int64_t)first_step + n_steps > r->max_steps) return FC_ERR_INVALID;
  if ((int64_t)r->n_streams * r->lru > 0x7FFFFFFF) return FC_ERR_INVALID;
  if (!r->pos || !r->lru_key || !r->lru_used || !r->lru_count || !r->hits || !r->lookups || !r->ctx ||
      !r->rows_retrieve || !r->rows_tree || !r->live || !r->history)
    return FC_ERR_INVALID;
  const int32_t B = r->n_streams, n_rows = r->n_streams * r->lru;
  for (int32_t i = 0; i < n_steps; ++i) {
    const int32_t step = first_step + i;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_replay_prepare, dim3(fc::div_up(B, kStreamsPerBlock)), dim3(kPrepThreads), 0, stream, *r,
                       step);
    FC_CHECK_LAUNCH();
    fc_status s = fc_retrieve(stores, S, r->ctx, B, r->ctx_len, r->rp, r->match_n, r->range_lo, r->range_cnt,
                              r->taken, r->cont_pos, r->cont_src, r->cont_len, r->cont_tok, r->rows_retrieve, n_rows,
                              r->retrieve_ws, r->retrieve_ws_bytes, stream);
    if (s != FC_OK) return s;
    s = fc_build_tree(r->taken, r->cont_len, r->cont_tok, r->ctx, B, r->ctx_len, S, r->rp.k, r->rp.m, r->tp,
                      r->num_nodes, r->node_tok, r->parent, r->weight, r->pos_ids, r->mask, r->rows_tree, n_rows,
                      r->tree_ws, r->tree_ws_bytes, stream);
    if (s != FC_OK) return s;
    s = fc_targets_from_truth(r->truth, r->truth_len, r->truth_stride, nullptr, r->pos, r->num_nodes, r->pos_ids, B,
                              r->tp.c, r->target, stream);
    if (s != FC_OK) return s;
    s = fc_verify_accept(r->num_nodes, r->node_tok, r->parent, r->pos_ids, r->target, B, r->tp.c, r->rp.m,
                         r->accept_len, r->accept_tok, r->last_node, stream);
    if (s != FC_OK) return s;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_replay_advance, dim3(fc::div_up(B, 256)), dim3(256), 0, stream, *r, step);
    FC_CHECK_LAUNCH();
  }
  return FC_OK;
}
