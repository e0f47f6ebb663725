/*
 * Seeded synthetic token data: template pools, Zipf-drawn files, queries and
 * ground-truth streams that stand in for the paper's code corpora (its common
 * store is drawn from The Stack, its repository store from each project's own
 * files; Section IV-A and Section V-D).  Both the oracle's tests and the GPU
 * path's tests and benchmark read their inputs from here.  This file holds no
 * part of the retrieval method itself.
 *
 * Random numbers: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used as a counter-based
 * generator: draw i of stream key K is mix(K + (i + 1) * GOLDEN).  Every
 * template, file and query owns its own stream, so files generate in parallel
 * and the result does not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* Stream key for (seed, role, index). */
uint64_t synth_stream_key(uint64_t seed, uint64_t role, uint64_t index) {
  return mix64(mix64(mix64(seed + GOLDEN) ^ (role * GOLDEN + 1)) ^ (index + 0x632BE59BD9B4E019ULL));
}

static uint64_t draw(uint64_t key, uint64_t i) { return mix64(key + (i + 1) * GOLDEN); }

/* Uniform integer in [lo, hi] from the high 32 bits (multiply-shift). */
static uint32_t uni(uint64_t r, uint32_t lo, uint32_t hi) {
  uint64_t span = (uint64_t)hi - lo + 1;
  return lo + (uint32_t)(((r >> 32) * span) >> 32);
}

/* Uniform double in [0, 1) with 53 random bits. */
static double unit(uint64_t r) { return (double)(r >> 11) * (1.0 / 9007199254740992.0); }

/* Roles of the random streams. */
enum { ROLE_POOL = 1, ROLE_FILE = 2, ROLE_NOISE = 3 };

/* Lengths of the n_templates templates of a pool; returns the total. */
uint64_t synth_pool_lengths(uint64_t seed, uint64_t n_templates, uint32_t min_len, uint32_t max_len,
                            uint64_t* offsets /* n_templates + 1 */) {
  uint64_t total = 0;
  for (uint64_t t = 0; t < n_templates; ++t) {
    offsets[t] = total;
    total += uni(draw(synth_stream_key(seed, ROLE_POOL, t), 0), min_len, max_len);
  }
  offsets[n_templates] = total;
  return total;
}

/* Template tokens, uniform over [1, vocab - 1]. */
void synth_pool_tokens(uint64_t seed, uint64_t n_templates, uint32_t vocab, const uint64_t* offsets,
                       uint16_t* tokens) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < (int64_t)n_templates; ++t) {
    uint64_t key = synth_stream_key(seed, ROLE_POOL, (uint64_t)t);
    uint64_t len = offsets[t + 1] - offsets[t];
    for (uint64_t x = 0; x < len; ++x) tokens[offsets[t] + x] = (uint16_t)uni(draw(key, x + 1), 1, vocab - 1);
  }
}

/* Unnormalised Zipf cumulative table: cum[t] = sum_{u <= t} (u + 1)^(-s). */
void synth_zipf_table(uint64_t n_templates, double s, double* cum) {
  double acc = 0.0;
  for (uint64_t t = 0; t < n_templates; ++t) {
    acc += pow((double)(t + 1), -s);
    cum[t] = acc;
  }
}

static uint64_t zipf_pick(const double* cum, uint64_t n, double u) {
  double target = u * cum[n - 1];
  uint64_t lo = 0, hi = n - 1; /* smallest t with cum[t] > target */
  while (lo < hi) {
    uint64_t mid = lo + (hi - lo) / 2;
    if (cum[mid] > target) hi = mid; else lo = mid + 1;
  }
  return lo;
}

/*
 * Writes n_files files of file_len tokens each.  File f is drawn from the
 * stream (file_seed, ROLE_FILE, first_index + f): templates are appended in
 * Zipf order until file_len tokens, the last one cut.  Then every token is,
 * with probability noise, replaced by a uniform token from [1, vocab - 1]
 * (stream ROLE_NOISE).  With sep != 0 a single 0 token separates consecutive
 * files (none after the last), so out holds n_files*file_len + n_files - 1
 * tokens; otherwise n_files*file_len.
 */
void synth_files(const uint64_t* offsets, const uint16_t* pool, uint64_t n_templates, const double* cum,
                 double noise, uint32_t vocab, uint64_t file_seed, uint64_t first_index, uint64_t n_files,
                 uint32_t file_len, int sep, uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t f = 0; f < (int64_t)n_files; ++f) {
    uint16_t* dst = out + (uint64_t)f * (file_len + (sep ? 1 : 0));
    uint64_t fkey = synth_stream_key(file_seed, ROLE_FILE, first_index + (uint64_t)f);
    uint64_t nkey = synth_stream_key(file_seed, ROLE_NOISE, first_index + (uint64_t)f);
    uint64_t fill = 0, ctr = 0;
    while (fill < file_len) {
      uint64_t t = zipf_pick(cum, n_templates, unit(draw(fkey, ctr++)));
      uint64_t len = offsets[t + 1] - offsets[t];
      for (uint64_t x = 0; x < len && fill < file_len; ++x) dst[fill++] = pool[offsets[t] + x];
    }
    for (uint64_t x = 0; x < file_len; ++x) {
      if (unit(draw(nkey, 2 * x)) < noise) dst[x] = (uint16_t)uni(draw(nkey, 2 * x + 1), 1, vocab - 1);
    }
    if (sep && (uint64_t)f + 1 < n_files) dst[file_len] = 0;
  }
}

/* n uniform integers in [lo, hi] from stream (seed, role, index). */
void synth_uniform(uint64_t seed, uint64_t role, uint64_t index, uint64_t n, uint32_t lo, uint32_t hi,
                   uint32_t* out) {
  uint64_t key = synth_stream_key(seed, role, index);
  for (uint64_t i = 0; i < n; ++i) out[i] = uni(draw(key, i), lo, hi);
}
