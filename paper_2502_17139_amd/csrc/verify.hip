// Greedy acceptance of a draft tree on gfx950 (fc_verify_accept).
//
// The target model checks every draft in one forward pass; the accepted
// draft is the longest root path whose tokens all agree with the model, and
// everything after the first disagreement is discarded (Section IV-D).  From
// the root, at row u the walk moves to the child whose token equals the
// model's token after u, and stops when there is none; the model's own token
// at the stopping row is accepted as well.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fastcoder.h"
#include "fc_device.h"
#include "fc_host.h"

namespace {

constexpr int kVerifyThreads = 256;
constexpr int kQueriesPerBlock = kVerifyThreads / fc::kWave;

// One wave per query (the walk in fc_device.h: lane l holds rows l, l+64,
// l+128, l+192; a path of depth d costs d ballots per 64 rows).
__global__ void __launch_bounds__(kVerifyThreads) k_verify(const int32_t* __restrict__ num_nodes,
                                                           const int32_t* __restrict__ node_tok,
                                                           const int32_t* __restrict__ parent,
                                                           const int32_t* __restrict__ target, int B, int c, int m,
                                                           int32_t* __restrict__ accept_len,
                                                           int32_t* __restrict__ accept_tok,
                                                           int32_t* __restrict__ last_node) {
  const int b = blockIdx.x * kQueriesPerBlock + (int)(threadIdx.x / fc::kWave);
  const int lane = fc::lane_id();
  if (b >= B) return;  // whole wave leaves together
  const int R = c + 1;
  const int64_t row = (int64_t)b * R;
  const int32_t* tgt = target + row;
  int len, u;
  fc::accept_walk<FC_MAX_TREE_ROWS>(num_nodes[b], node_tok + row, parent + row, R, m,
                                     [&](int v) { return tgt[v]; }, accept_tok + (int64_t)b * (m + 1), len, u);
  if (lane == 0) {
    accept_len[b] = len;
    last_node[b] = u;
  }
}

// target[b][i] = truth[b][start[b] + pos_ids[b][i]] for live rows inside
// the stream, else -1; one thread per (query, row).
__global__ void __launch_bounds__(256) k_targets(const uint16_t* __restrict__ truth, int truth_len,
                                                 int64_t stride, const int32_t* __restrict__ seq,
                                                 const int32_t* __restrict__ start,
                                                 const int32_t* __restrict__ num_nodes,
                                                 const int32_t* __restrict__ pos_ids, int B, int R,
                                                 int32_t* __restrict__ target) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (int64_t)B * R) return;
  const int b = (int)(e / R), i = (int)(e - (int64_t)b * R);
  int32_t v = -1;
  if (i < num_nodes[b]) {
    const int64_t pos = (int64_t)start[b] + pos_ids[e];
    const int64_t sq = seq ? seq[b] : b;
    if (pos >= 0 && pos < truth_len) v = truth[sq * stride + pos];
  }
  target[e] = v;
}

}  // namespace

extern "C" fc_status fc_verify_accept(const int32_t* num_nodes, const int32_t* node_tok, const int32_t* parent,
                                      const int32_t* pos_ids, const int32_t* target, int32_t B, int32_t c, int32_t m,
                                      int32_t* accept_len, int32_t* accept_tok, int32_t* last_node,
                                      hipStream_t stream) {
  (void)pos_ids;
  if (B < 0 || c < 0 || c + 1 > FC_MAX_TREE_ROWS || m < 0 || m > 255) return FC_ERR_INVALID;
  if (B == 0) return FC_OK;
  if (!num_nodes || !node_tok || !parent || !target || !accept_len || !accept_tok || !last_node)
    return FC_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_verify, dim3(fc::div_up(B, kQueriesPerBlock)), dim3(kVerifyThreads), 0, stream, num_nodes,
                     node_tok, parent, target, B, c, m, accept_len, accept_tok, last_node);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" fc_status fc_targets_from_truth(const uint16_t* truth, int32_t truth_len, int64_t truth_stride,
                                           const int32_t* seq, const int32_t* start, const int32_t* num_nodes,
                                           const int32_t* pos_ids, int32_t B, int32_t c, int32_t* target,
                                           hipStream_t stream) {
  if (B < 0 || c < 0 || c + 1 > FC_MAX_TREE_ROWS || truth_len < 0 || truth_stride < truth_len) return FC_ERR_INVALID;
  if (B == 0) return FC_OK;
  if (!truth || !start || !num_nodes || !pos_ids || !target) return FC_ERR_INVALID;
  (void)hipGetLastError();
  const int64_t n = (int64_t)B * (c + 1);
  hipLaunchKernelGGL(k_targets, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, stream, truth, truth_len,
                     truth_stride, seq, start, num_nodes, pos_ids, B, c + 1, target);
  FC_CHECK_LAUNCH();
  return FC_OK;
}
