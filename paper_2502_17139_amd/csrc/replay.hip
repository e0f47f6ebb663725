// Device-resident decode-trace replay (fc_replay_init, fc_replay_run).
//
// The draft stage driven over known token streams as a stand-in for a
// decoding loop, the way the average acceptance length is measured
// (Section V-C, eq. (7)): every step each live stream looks its 16-token
// context up in an LRU of its recent retrievals, retrieves on a miss
// (Section III-A over the stores in priority order), builds its draft tree
// (Section IV-D), takes the true next tokens as the target model's outputs,
// accepts greedily and advances by the accepted length.  Optionally the
// CACHE of Section IV-B comes first (Alg. 1's cache branch) and Alg. 1's
// retrieval-timing control (missing table, skip gate) may skip a retrieval.
//
// Everything a step decides lives on the GPU, so a step is a fixed chain of
// launches on one stream with no host round trip:
//   k_replay_context   (CACHE on, first step of a call) the context and the
//                      CACHE row map;
//   fc_cache_retrieve  (CACHE on) streams whose CACHE is old enough;
//   k_replay_decide    one wave per stream: served by the CACHE (its result
//                      is copied into the stream's own row after the LRU
//                      rows, so one tree call serves both kinds of
//                      stream), else the missing table and the skip gate,
//                      else the LRU probe (keys compared by the lanes, the
//                      least recent slot by a wave minimum); the row maps;
//   fc_retrieve        misses into their LRU slot (everything else skipped);
//   k_replay_missing   (table on) empty results enter the missing table;
//   fc_build_tree      from the mapped rows;
//   k_replay_finish    one wave per stream: the acceptance walk with the
//                      true tokens as targets (fc_targets_from_truth and
//                      fc_verify_accept in one pass), position += accepted
//                      length, the step's history row, the live count and
//                      (CACHE on) the CACHE additions; then, within a call,
//                      the next step's context and CACHE row map (CACHE on)
//                      or the next step's decision (CACHE off), so those
//                      launches run only on a call's first step.
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

enum StreamState : int32_t { kNeed = 0, kServed = 1, kSkipped = 2, kDone = -1 };

__device__ __forceinline__ bool cache_on(const fc_replay& r) { return r.cache_l >= 0; }
__device__ __forceinline__ bool control_on(const fc_replay& r) { return r.missing || r.skip_tok >= 0; }

__global__ void __launch_bounds__(256) k_replay_init(fc_replay r) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b == 0) r.live[0] = r.live[1] = 0;
  if (b >= r.n_streams) return;
  r.pos[b] = r.ctx_len;
  r.lru_count[b] = 0;
  r.hits[b] = 0;
  r.lookups[b] = 0;
  if (cache_on(r)) {
    r.clen[b] = 0;
    r.seq_head[b] = 0;
    r.seq_count[b] = 0;
    r.chunks[b] = 0;
    r.served[b] = 0;
  }
  if (control_on(r)) {
    r.m_skips[b] = 0;
    r.g_skips[b] = 0;
  }
}

// empties the missing tables and the skipped contexts' retrieval row
__global__ void __launch_bounds__(256) k_replay_init_tables(fc_replay r, int32_t S) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < S) r.taken[(int64_t)r.n_streams * r.lru * S + i] = 0;
  if (r.missing && i < (int64_t)r.n_streams * r.miss_cap) r.miss_used[i] = 0;
}

// The context (the L tokens before the position) of every live stream, and
// (CACHE on) which streams search their CACHE this step.
__global__ void __launch_bounds__(256) k_replay_context(fc_replay r) {
  const int b = blockIdx.x;
  const int L = r.ctx_len;
  const int p = r.pos[b];
  const bool live = p < r.truth_len;
  if (threadIdx.x == 0) r.rows_cache[b] = (live && r.seq_count[b] >= r.cache_l) ? b : -1;
  if (live && (int)threadIdx.x < L)
    r.ctx[(int64_t)b * L + threadIdx.x] = r.truth[(int64_t)b * r.truth_stride + (p - L) + threadIdx.x];
}

__device__ __forceinline__ uint32_t ctx_hash(const uint16_t* c, int L) {
  uint32_t h = 2166136261u;  // FNV-1a over the tokens
  for (int t = 0; t < L; ++t) {
    h = (h ^ (uint32_t)(c[t] & 0xFF)) * 16777619u;
    h = (h ^ (uint32_t)(c[t] >> 8)) * 16777619u;
  }
  return h;
}

// Missing table of stream b: open addressing over miss_cap slots, probed 64
// at a time by the wave.  Returns the slot holding ctx, or -1 - (first free
// slot) when it is absent.  The table never fills (miss_cap > max_steps >=
// insertions), so the probe ends.
__device__ int miss_find(const fc_replay& r, int b, const uint16_t* ctx) {
  const int L = r.ctx_len, lane = fc::lane_id();
  const uint32_t mask = (uint32_t)r.miss_cap - 1u;
  const uint32_t h = ctx_hash(ctx, L);
  const uint16_t* keys = r.miss_key + (int64_t)b * r.miss_cap * L;
  const uint8_t* used = r.miss_used + (int64_t)b * r.miss_cap;
  for (uint32_t base = 0; base < (uint32_t)r.miss_cap; base += fc::kWave) {
    const uint32_t slot = (h + base + (uint32_t)lane) & mask;
    const bool u = used[slot] != 0;
    bool eq = u;
    if (u) {
      const uint16_t* key = keys + (int64_t)slot * L;
      for (int t = 0; t < L; ++t) eq &= key[t] == ctx[t];
    }
    const uint64_t hit = fc::ballot(eq), empty = fc::ballot(!u);
    // the first slot in probe order that matches or is empty decides
    const uint64_t any = hit | empty;
    if (any) {
      const int first = __builtin_ctzll(any);
      const int s = __shfl((int)slot, first);
      return ((hit >> first) & 1ull) ? s : -1 - s;
    }
  }
  return -1 - (int)(h & mask);  // not reached
}

// One wave: stream b's decision for `step` at position p, and its row maps.
// Row of stream b's CACHE result in the retrieval outputs (CACHE on): after
// the n_streams * lru LRU rows and the empty row.
__device__ __forceinline__ int cache_row(const fc_replay& r, int b) { return r.n_streams * r.lru + 1 + b; }

__device__ void decide_stream(const fc_replay& r, int S, int b, int32_t step, int p) {
  const int lane = fc::lane_id();
  const int L = r.ctx_len, lru = r.lru;
  if (p >= r.truth_len) {  // finished: no retrieval, no tree row
    if (lane == 0) {
      r.rows_retrieve[b] = -1;
      r.rows_tree[b] = -1;
      if (cache_on(r)) r.rows_cache[b] = -1;
      r.state[b] = kDone;
    }
    return;
  }
  const uint16_t* src = r.truth + (int64_t)b * r.truth_stride + (p - L);
  uint16_t* ctx = r.ctx + (int64_t)b * L;
  const uint16_t tok = lane < L ? src[lane] : (uint16_t)0;
  if (lane < L) ctx[lane] = tok;
  // Alg. 1: the CACHE first
  if (cache_on(r)) {
    const bool served = r.rows_cache[b] >= 0 && r.c_taken[b] > 0;
    if (served) {
      // the CACHE result as a retrieval row: all its slots from the first
      // store (the CACHE is searched as one store), none from the others
      const int row = cache_row(r, b);
      const int T = r.c_taken[b];
      const int k = r.rp.k, m = r.rp.m;
      if (lane < S) r.taken[(int64_t)row * S + lane] = lane == 0 ? T : 0;
      const uint8_t* sl = r.c_cont_len + (int64_t)b * k;
      uint8_t* dl = r.cont_len + (int64_t)row * k;
      for (int i = lane; i < T; i += fc::kWave) dl[i] = sl[i];
      const uint16_t* stk = r.c_cont_tok + (int64_t)b * k * m;
      uint16_t* dtk = r.cont_tok + (int64_t)row * k * m;
      for (int64_t e = lane; e < (int64_t)T * m; e += fc::kWave) dtk[e] = stk[e];
      if (lane == 0) {
        r.rows_retrieve[b] = -1;
        r.rows_tree[b] = row;
        r.state[b] = kServed;
      }
      return;
    }
    if (lane == 0) r.rows_cache[b] = -1;
  }
  // the timing control: the missing table, then the skip gate
  bool skip = false;
  if (r.missing && miss_find(r, b, src) >= 0) {
    skip = true;
    if (lane == 0) r.m_skips[b] += 1;
  } else if (r.skip_tok >= 0 && (int)src[L - 1] == r.skip_tok &&
             !((uint32_t)r.skip_draws[(int64_t)step * r.n_streams + b] < r.skip_thr)) {
    skip = true;
    if (lane == 0) r.g_skips[b] += 1;
  }
  if (skip) {
    if (lane == 0) {
      r.rows_retrieve[b] = -1;
      r.rows_tree[b] = r.n_streams * lru;  // the empty row: a bare root
      r.state[b] = kSkipped;
    }
    return;
  }
  // the LRU probe: lane e compares slot e's key with the context
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
    r.state[b] = kNeed;
  }
}

__global__ void __launch_bounds__(kPrepThreads) k_replay_decide(fc_replay r, int S, int32_t step) {
  const int b = blockIdx.x * kStreamsPerBlock + (int)threadIdx.x / fc::kWave;
  if (b < r.n_streams) decide_stream(r, S, b, step, r.pos[b]);
}

// One wave per stream: a looked-up context whose result is empty enters the
// missing table.
__global__ void __launch_bounds__(kPrepThreads) k_replay_missing(fc_replay r, int32_t S) {
  const int lane = fc::lane_id();
  const int b = blockIdx.x * kStreamsPerBlock + (int)threadIdx.x / fc::kWave;
  if (b >= r.n_streams || r.state[b] != kNeed) return;
  const int row = r.rows_tree[b];
  int tot = 0;
  for (int s = 0; s < S; ++s) tot += r.taken[(int64_t)row * S + s];
  if (tot != 0) return;
  const int L = r.ctx_len;
  const uint16_t* ctx = r.ctx + (int64_t)b * L;
  const int f = miss_find(r, b, ctx);
  if (f >= 0) return;
  const int slot = -1 - f;
  if (lane < L) r.miss_key[((int64_t)b * r.miss_cap + slot) * L + lane] = ctx[lane];
  if (lane == 0) r.miss_used[(int64_t)b * r.miss_cap + slot] = 1;
}

// One workgroup per stream: a served stream's tree comes from the CACHE's.
// A stream's CACHE bookkeeping, held in registers (the same in every lane)
// while one wave adds its sequences.
struct CacheState {
  int len, head, cnt;
};

// Adds seq[0 .. len) to stream b's CACHE (one wave): the sequence keeps its
// last cache_cap tokens; the oldest sequences go while the text, the
// sequences joined by 0, would be longer than cache_cap.  Lane 0 keeps the
// ring of sequence lengths; a workgroup fence at the end makes this
// addition's writes visible to every lane before the next one reads them.
__device__ void cache_add(const fc_replay& r, int b, CacheState& st, const uint16_t* seq, int len) {
  const int lane = fc::lane_id();
  const int cap = r.cache_cap;
  if (len > cap) {
    seq += len - cap;
    len = cap;
  }
  if (len <= 0) return;
  uint16_t* text = r.ctext + (int64_t)b * cap;
  int* lens = r.seq_len + (int64_t)b * r.max_seqs;
  const int old = st.len;
  const int total = old + (st.cnt > 0 ? 1 : 0) + len;
  int cut = 0;
  while (total - cut > cap) {  // only old sequences go: the new one fits alone
    cut += lens[st.head] + 1;
    st.head = st.head + 1 == r.max_seqs ? 0 : st.head + 1;
    --st.cnt;
  }
  const int keep = old - cut;  // -1 when every old sequence went (with the separator)
  if (cut > 0 && keep > 0) {
    // move the kept text to the front, 64 tokens a pass in increasing order
    // (a pass's loads complete before its stores, and later passes read
    // above what earlier ones wrote)
    for (int i = 0; i < keep; i += fc::kWave) {
      const int j = i + lane;
      const uint16_t v = j < keep ? text[cut + j] : (uint16_t)0;
      if (j < keep) text[j] = v;
    }
  }
  const int start = keep > 0 ? keep + 1 : 0;
  if (keep > 0 && lane == 0) text[keep] = 0;
  for (int i = lane; i < len; i += fc::kWave) text[start + i] = seq[i];
  if (lane == 0) lens[(st.head + st.cnt) % r.max_seqs] = len;
  st.cnt += 1;
  st.len = start + len;
  __threadfence_block();
}

// One wave per stream: acceptance (the target after row i is the true token
// at pos + pos_ids[i], -1 past the stream or for rows past num_nodes), the
// history row, the new position, the live count and (CACHE on) the CACHE
// additions of this step.
// Then, within a call, the same wave prepares its stream's next step:
// `next` = 1 takes the next step's decision (CACHE off), `next` = 2 writes
// the next step's context and CACHE row map (CACHE on: the CACHE search
// comes between them and the decision).  live[step & 1] counts the streams
// live after the step; this launch clears the other counter for the next
// step.
__global__ void __launch_bounds__(kPrepThreads) k_replay_finish(fc_replay r, int S, int32_t step, int next) {
  const int lane = fc::lane_id();
  const int b = blockIdx.x * kStreamsPerBlock + (int)threadIdx.x / fc::kWave;
  if (blockIdx.x == 0 && threadIdx.x == 0) r.live[(step + 1) & 1] = 0;
  if (b >= r.n_streams) return;
  int32_t* hist = r.history + (int64_t)step * r.n_streams;
  const int p = r.pos[b];
  const int tlen = r.truth_len, L = r.ctx_len;
  if (p >= tlen) {
    if (lane == 0) hist[b] = -1;
    if (next == 1) decide_stream(r, S, b, step + 1, p);
    if (next == 2 && lane == 0) r.rows_cache[b] = -1;
    return;
  }
  const int R = r.tp.c + 1;
  const int64_t row = (int64_t)b * R;
  const int nn = r.num_nodes[b];
  const uint16_t* srow = r.truth + (int64_t)b * r.truth_stride;
  const int32_t* pid = r.pos_ids + row;
  int a, last;
  if (r.rp.m + 1 <= fc::kWave) {
    // a row's target is the truth token its depth places after p: the
    // window p .. p + m, one token per lane, loaded with the tree rows
    const int32_t win = (lane <= r.rp.m && p + lane < tlen) ? (int32_t)srow[p + lane] : -1;
    fc::accept_walk_depth<FC_MAX_TREE_ROWS>(nn, r.node_tok + row, r.parent + row, R, r.rp.m, win,
                                            r.accept_tok + (int64_t)b * (r.rp.m + 1), a, last);
  } else {
    fc::accept_walk<FC_MAX_TREE_ROWS>(
        nn, r.node_tok + row, r.parent + row, R, r.rp.m,
        [&](int v) -> int32_t {
          if (v >= nn) return -1;
          const int64_t q = (int64_t)p + pid[v];
          return (q >= 0 && q < tlen) ? (int32_t)srow[q] : -1;
        },
        r.accept_tok + (int64_t)b * (r.rp.m + 1), a, last);
  }
  if (lane == 0) {
    r.accept_len[b] = a;
    r.last_node[b] = last;
  }
  const int np = p + a;
  if (cache_on(r)) {
    const uint16_t* row = srow;
    if (lane == 0 && r.state[b] == kServed) r.served[b] += 1;
    const int depth = (last >= 0 && last < R) ? pid[last] : 0;
    CacheState st = {r.clen[b], r.seq_head[b], r.seq_count[b]};
    if (depth >= 1) {  // a verified draft: the context and its accepted tokens
      const int end = p + depth < tlen ? p + depth : tlen;
      cache_add(r, b, st, row + (p - L), end - (p - L));
    }
    int ch = r.chunks[b];
    const int lim = np < tlen ? np : tlen;
    while (L + r.cache_every * (ch + 1) <= lim) {  // every completed output chunk
      cache_add(r, b, st, row + L + r.cache_every * ch, r.cache_every);
      ++ch;
    }
    if (lane == 0) {
      r.chunks[b] = ch;
      r.clen[b] = st.len;
      r.seq_head[b] = st.head;
      r.seq_count[b] = st.cnt;
    }
    if (next == 2) {  // the next step's context and CACHE row map
      const bool live = np < tlen;
      if (lane == 0) r.rows_cache[b] = (live && st.cnt >= r.cache_l) ? b : -1;
      if (live && lane < L) r.ctx[(int64_t)b * L + lane] = srow[(np - L) + lane];
    }
  }
  if (lane == 0) {
    hist[b] = a;
    r.pos[b] = np;
    if (np < tlen) atomicAdd(&r.live[step & 1], 1);
  }
  if (next == 1) decide_stream(r, S, b, step + 1, np);
}

fc_status check_replay(const fc_replay* r) {
  if (!r || r->n_streams < 1 || r->ctx_len < 1 || r->ctx_len > fc::kWave || r->lru < 1 || r->lru > fc::kWave)
    return FC_ERR_INVALID;
  if (r->truth_len < 0 || r->truth_stride < r->truth_len || !r->truth || r->max_steps < 0) return FC_ERR_INVALID;
  if ((int64_t)r->n_streams * (r->lru + 1) + 1 > 0x7FFFFFFF) return FC_ERR_INVALID;
  if (!r->pos || !r->lru_key || !r->lru_used || !r->lru_count || !r->hits || !r->lookups || !r->ctx ||
      !r->rows_retrieve || !r->rows_tree || !r->live || !r->history || !r->taken || !r->state || !r->accept_len ||
      !r->accept_tok || !r->last_node)
    return FC_ERR_INVALID;
  if (r->cache_l >= 0) {
    if (r->cache_every < 1 || r->cache_cap < 1 || r->cache_cap > FC_MAX_CACHE_TOKENS ||
        r->max_seqs < (r->cache_cap + 1) / 2 + 1)
      return FC_ERR_INVALID;
    if (!r->ctext || !r->clen || !r->seq_len || !r->seq_head || !r->seq_count || !r->chunks || !r->served ||
        !r->rows_cache || !r->c_match_n || !r->c_range_lo || !r->c_range_cnt || !r->c_taken || !r->c_cont_pos ||
        !r->c_cont_src || !r->c_cont_len || !r->c_cont_tok)
      return FC_ERR_INVALID;
    if (r->tp.alpha[0] == 0) return FC_ERR_INVALID;  // a served tree is weighted by the first store's alpha
  }
  if (r->missing) {
    if (r->miss_cap < 1 || (r->miss_cap & (r->miss_cap - 1)) || r->miss_cap <= r->max_steps || !r->miss_key ||
        !r->miss_used)
      return FC_ERR_INVALID;
  }
  if ((r->missing || r->skip_tok >= 0) && (!r->m_skips || !r->g_skips)) return FC_ERR_INVALID;
  if (r->skip_tok >= 0 && !r->skip_draws) return FC_ERR_INVALID;
  return FC_OK;
}

}  // namespace

extern "C" fc_status fc_replay_init(fc_replay* r, hipStream_t stream) {
  fc_status s = check_replay(r);
  if (s != FC_OK) return s;
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_replay_init, dim3(fc::div_up(r->n_streams, 256)), dim3(256), 0, stream, *r);
  FC_CHECK_LAUNCH();
  return FC_OK;
}

extern "C" fc_status fc_replay_run(const fc_store* stores, int32_t S, const fc_replay* r, int32_t first_step,
                                   int32_t n_steps, hipStream_t stream) {
  if (!stores || S < 1 || S > FC_MAX_SOURCES) return FC_ERR_INVALID;
  fc_status s = check_replay(r);
  if (s != FC_OK) return s;
  if (first_step < 0 || n_steps < 0 || (int64_t)first_step + n_steps > r->max_steps) return FC_ERR_INVALID;
  const int32_t B = r->n_streams, n_rows = r->n_streams * r->lru + 1;
  const bool cache = r->cache_l >= 0, control = r->missing || r->skip_tok >= 0;
  if (first_step == 0 && control) {  // a replay's first call: the empty row and the missing tables
    const int64_t tab = r->missing ? (int64_t)B * r->miss_cap : 0;
    const int64_t work = tab > S ? tab : (int64_t)S;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_replay_init_tables, dim3((uint32_t)((work + 255) / 256)), dim3(256), 0, stream, *r, S);
    FC_CHECK_LAUNCH();
  }
  const int32_t tree_rows = n_rows + (cache ? B : 0);  // (CACHE on) one CACHE row per stream
  for (int32_t i = 0; i < n_steps; ++i) {
    const int32_t step = first_step + i;
    (void)hipGetLastError();
    if (cache) {
      if (i == 0) {  // otherwise the previous step's finish wrote the context
        hipLaunchKernelGGL(k_replay_context, dim3(B), dim3(fc::kWave), 0, stream, *r);
        FC_CHECK_LAUNCH();
      }
      s = fc_cache_retrieve(r->ctext, r->cache_cap, B, r->clen, nullptr, r->ctx, B, r->ctx_len, r->rp, r->c_match_n,
                            r->c_range_lo, r->c_range_cnt, r->c_taken, r->c_cont_pos, r->c_cont_src, r->c_cont_len,
                            r->c_cont_tok, r->rows_cache, B, stream);
      if (s != FC_OK) return s;
    }
    if (cache || i == 0) {  // otherwise the previous step's finish took this step's decision
      hipLaunchKernelGGL(k_replay_decide, dim3(fc::div_up(B, kStreamsPerBlock)), dim3(kPrepThreads), 0, stream, *r,
                         S, step);
      FC_CHECK_LAUNCH();
    }
    s = fc_retrieve(stores, S, r->ctx, B, r->ctx_len, r->rp, r->match_n, r->range_lo, r->range_cnt, r->taken,
                    r->cont_pos, r->cont_src, r->cont_len, r->cont_tok, r->rows_retrieve, n_rows, r->retrieve_ws,
                    r->retrieve_ws_bytes, stream);
    if (s != FC_OK) return s;
    if (r->missing) {
      hipLaunchKernelGGL(k_replay_missing, dim3(fc::div_up(B, kStreamsPerBlock)), dim3(kPrepThreads), 0, stream,
                         *r, S);
      FC_CHECK_LAUNCH();
    }
    s = fc_build_tree(r->taken, r->cont_len, r->cont_tok, r->ctx, B, r->ctx_len, S, r->rp.k, r->rp.m, r->tp,
                      r->num_nodes, r->node_tok, r->parent, r->weight, r->pos_ids, r->mask, r->rows_tree, tree_rows,
                      r->tree_ws, r->tree_ws_bytes, stream);
    if (s != FC_OK) return s;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_replay_finish, dim3(fc::div_up(B, kStreamsPerBlock)), dim3(kPrepThreads), 0, stream, *r, S,
                       step, i + 1 < n_steps ? (cache ? 2 : 1) : 0);
    FC_CHECK_LAUNCH();
  }
  return FC_OK;
}
