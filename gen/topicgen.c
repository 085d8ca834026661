/*
 * Seeded synthetic inputs for cluster-level sparse prefill: the topic-structured Q/K/V workload.
 *
 * This file holds NO arithmetic of the method (no block means, no scoring, no attention). It only
 * draws numbers. Both the HIP path and the oracle consume what it writes, so any element can be
 * reproduced from (seed, layer, tensor, index) alone, in any thread order.
 *
 * Random source: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014), used as a counter-based generator: output n of stream `key` is the
 * SplitMix64 finaliser applied to key + (n + 1) * 0x9E3779B97F4A7C15.
 * Uniforms take the top 53 bits. Normals come in pairs by Box-Muller (Box and Muller, 1958):
 * pair j of a stream uses outputs 2j and 2j+1, element 2j is r*cos(2*pi*u2) and element 2j+1 is
 * r*sin(2*pi*u2), with r = sqrt(-2 ln u1) and u1 = 1 - uniform (so u1 is in (0, 1]).
 *
 * Workload (per layer; d = head_dim):
 *   topic vectors   T[i][c] = N(0,1) / sqrt(d),   i < n_topics, shared by every head
 *   query topics    a run-length process over sub-chunks: draw a topic uniformly, draw a run
 *                   length uniformly in [run_lo, run_hi], give that topic to the next run-length
 *                   sub-chunks (truncated at the last one), repeat; run r also draws a topic
 *                   strength s_r uniformly in [s_lo, s_hi] from a stream of its own (s_lo = s_hi
 *                   gives every run that strength exactly)
 *   KV block topics each block of B tokens draws its topic uniformly and independently
 *   Q[p][h][c]  = s(p / L) T[qtopic(p / L)][c] + N(0,1)   (s = the strength of the sub-chunk's run)
 *   K[t][g][c]  = 2 T[kvtopic(t / B)][c] + N(0,1)
 *   V[t][g][c]  = N(0,1)
 * Every value is rounded to fp32 (round-to-nearest-even) and then to bf16 (RNE); bf16 values are
 * returned as raw uint16 bit patterns. K and V are written in the paged layout
 * [block][kv_head][B][d] with page b holding logical block b.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

enum { T_TOPICS = 1, T_QTOPIC = 2, T_KVTOPIC = 3, T_QNOISE = 4, T_KNOISE = 5, T_V = 6, T_QSCALE = 7 };

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t key, uint64_t n) { return mix64(key + (n + 1) * GOLDEN); }

/* Key of one stream: chained draws over (seed, layer, tensor). */
uint64_t tg_stream_key(uint64_t seed, uint64_t layer, uint64_t tensor) {
  uint64_t k = draw(0x5CA1E5CA1E5CA1EULL, seed);
  k = draw(k, layer);
  return draw(k, tensor);
}

static inline double uniform53(uint64_t x) { return (double)(x >> 11) * (1.0 / 9007199254740992.0); }

/* Element `i` of the standard-normal sequence of stream `key`. */
static inline double normal_at(uint64_t key, uint64_t i) {
  uint64_t j = i >> 1;
  double u1 = 1.0 - uniform53(draw(key, 2 * j));
  double u2 = uniform53(draw(key, 2 * j + 1));
  double r = sqrt(-2.0 * log(u1));
  double a = 6.283185307179586476925286766559 * u2;
  return (i & 1) ? r * sin(a) : r * cos(a);
}

/* Fill out[0..count) with normals i0 .. i0+count of stream `key` (pairs computed once). */
static void normals(uint64_t key, uint64_t i0, int64_t count, double* out) {
  int64_t n = 0;
  uint64_t i = i0;
  if ((i & 1) && n < count) { out[n++] = normal_at(key, i++); }
  for (; n + 1 < count; n += 2, i += 2) {
    uint64_t j = i >> 1;
    double u1 = 1.0 - uniform53(draw(key, 2 * j));
    double u2 = uniform53(draw(key, 2 * j + 1));
    double r = sqrt(-2.0 * log(u1));
    double a = 6.283185307179586476925286766559 * u2;
    out[n] = r * cos(a);
    out[n + 1] = r * sin(a);
  }
  if (n < count) out[n] = normal_at(key, i);
}

static inline uint16_t to_bf16(double x) {
  float f = (float)x;          /* fp64 -> fp32, round to nearest even */
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFF) ? 0x40 : 0));
  u += 0x7FFFu + ((u >> 16) & 1u);   /* fp32 -> bf16, round to nearest even */
  return (uint16_t)(u >> 16);
}

static inline int64_t uniform_int(uint64_t x, int64_t n) {
  int64_t v = (int64_t)(uniform53(x) * (double)n);
  return v < n ? v : n - 1;
}

/* topics[n_topics][d] in fp64. */
void tg_topics(uint64_t seed, int layer, int n_topics, int d, double* topics) {
  uint64_t key = tg_stream_key(seed, (uint64_t)layer, T_TOPICS);
  double s = 1.0 / sqrt((double)d);
  normals(key, 0, (int64_t)n_topics * d, topics);
  for (int64_t i = 0; i < (int64_t)n_topics * d; ++i) topics[i] *= s;
}

/* qtopic[M], qscale[M]: topic and topic strength of each sub-chunk from the run-length process. */
void tg_query_topics(uint64_t seed, int layer, int n_topics, int run_lo, int run_hi, int M,
                     double scale_lo, double scale_hi, int32_t* qtopic, double* qscale) {
  uint64_t key = tg_stream_key(seed, (uint64_t)layer, T_QTOPIC);
  uint64_t skey = tg_stream_key(seed, (uint64_t)layer, T_QSCALE);
  uint64_t n = 0, run_index = 0;
  int m = 0;
  while (m < M) {
    int32_t topic = (int32_t)uniform_int(draw(key, n++), n_topics);
    int run = run_lo + (int)uniform_int(draw(key, n++), (int64_t)(run_hi - run_lo + 1));
    double s = scale_lo == scale_hi ? scale_lo
                                    : scale_lo + (scale_hi - scale_lo) * uniform53(draw(skey, run_index));
    ++run_index;
    for (int r = 0; r < run && m < M; ++r) {
      qtopic[m] = topic;
      qscale[m] = s;
      ++m;
    }
  }
}

/* kvtopic[n_blocks]: topic of each KV block. */
void tg_kv_topics(uint64_t seed, int layer, int n_topics, int n_blocks, int32_t* kvtopic) {
  uint64_t key = tg_stream_key(seed, (uint64_t)layer, T_KVTOPIC);
  for (int b = 0; b < n_blocks; ++b) kvtopic[b] = (int32_t)uniform_int(draw(key, (uint64_t)b), n_topics);
}

/* Q rows [row0, row0 + n_rows) as bf16 bits, row-major [row][Hq][d]. */
void tg_fill_q(uint64_t seed, int layer, const double* topics, const int32_t* qtopic,
               const double* qscale, int L, int Hq, int d, int64_t row0, int64_t n_rows, uint16_t* q) {
  uint64_t key = tg_stream_key(seed, (uint64_t)layer, T_QNOISE);
  int64_t row_elems = (int64_t)Hq * d;
#pragma omp parallel
  {
    double buf[8 * 256];
#pragma omp for schedule(static)
    for (int64_t r = 0; r < n_rows; ++r) {
      int64_t p = row0 + r;
      const double* t = topics + (int64_t)qtopic[p / L] * d;
      const double s = qscale[p / L];
      for (int64_t off = 0; off < row_elems; off += 2048) {
        int64_t cnt = row_elems - off < 2048 ? row_elems - off : 2048;
        normals(key, (uint64_t)(p * row_elems + off), cnt, buf);
        for (int64_t e = 0; e < cnt; ++e) {
          int c = (int)((off + e) % d);
          q[r * row_elems + off + e] = to_bf16(s * t[c] + buf[e]);
        }
      }
    }
  }
}

/* K and V for blocks [blk0, blk0 + n_blk) in the paged layout [block][Hkv][B][d] (bf16 bits).
 * k or v may be NULL to skip it. */
void tg_fill_kv(uint64_t seed, int layer, const double* topics, const int32_t* kvtopic, int B,
                int Hkv, int d, int64_t blk0, int64_t n_blk, uint16_t* k, uint16_t* v) {
  uint64_t kkey = tg_stream_key(seed, (uint64_t)layer, T_KNOISE);
  uint64_t vkey = tg_stream_key(seed, (uint64_t)layer, T_V);
#pragma omp parallel
  {
    double buf[256];
#pragma omp for schedule(static) collapse(2)
    for (int64_t bi = 0; bi < n_blk; ++bi) {
      for (int64_t tt = 0; tt < B; ++tt) {
        int64_t b = blk0 + bi;
        int64_t t = b * B + tt;
        const double* tv = topics + (int64_t)kvtopic[b] * d;
        for (int g = 0; g < Hkv; ++g) {
          int64_t src = (t * Hkv + g) * d;          /* token-major element index */
          int64_t dst = ((bi * Hkv + g) * B + tt) * d; /* paged layout */
          if (k) {
            normals(kkey, (uint64_t)src, d, buf);
            for (int c = 0; c < d; ++c) k[dst + c] = to_bf16(2.0 * tv[c] + buf[c]);
          }
          if (v) {
            normals(vkey, (uint64_t)src, d, buf);
            for (int c = 0; c < d; ++c) v[dst + c] = to_bf16(buf[c]);
          }
        }
      }
    }
  }
}

/* Raw access for tests of the generator itself. */
uint64_t tg_draw(uint64_t key, uint64_t n) { return draw(key, n); }
double tg_normal(uint64_t key, uint64_t i) { return normal_at(key, i); }
uint16_t tg_bf16(double x) { return to_bf16(x); }
