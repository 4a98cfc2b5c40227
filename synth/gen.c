/* Seeded synthetic byte-stream sources: input infrastructure shared by the
 * oracle tests, the GPU tests and the benchmark.  Nothing here computes any
 * part of the estimator; it only draws bytes and reports each source's own
 * code length (sum of -log2 p_source(x)) as context for the model's bits/byte.
 *
 * Generators: splitmix64 (Vigna) for seeding, xoshiro256** (Blackman & Vigna)
 * for draws, Marsaglia & Tsang (2000) for Gamma variates (with the U^(1/a)
 * boost for a < 1), Dirichlet rows as normalised Gamma draws, inverse-CDF
 * sampling by binary search.  Built with gcc -O2 -fopenmp; no fast-math. */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline uint64_t sm64(uint64_t *s) {
  uint64_t z = (*s += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

uint64_t synth_splitmix64(uint64_t x) {
  uint64_t s = x;
  return sm64(&s);
}

typedef struct { uint64_t s[4]; } xo256;

static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static void xo_seed(xo256 *r, uint64_t seed) {
  uint64_t t = seed;
  for (int i = 0; i < 4; ++i) r->s[i] = sm64(&t);
}

static inline uint64_t xo_next(xo256 *r) {
  uint64_t *s = r->s;
  const uint64_t out = rotl(s[1] * 5, 7) * 9;
  const uint64_t t = s[1] << 17;
  s[2] ^= s[0];
  s[3] ^= s[1];
  s[1] ^= s[2];
  s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return out;
}

static inline double u01(xo256 *r) { return (double)(xo_next(r) >> 11) * 0x1.0p-53; }          /* [0,1) */
static inline double u01o(xo256 *r) { return ((double)(xo_next(r) >> 11) + 0.5) * 0x1.0p-53; } /* (0,1) */

static double normal(xo256 *r) {
  double a = u01o(r), b = u01o(r);
  return sqrt(-2.0 * log(a)) * cos(6.283185307179586 * b);
}

static double gamma_mt(xo256 *r, double a) {
  if (a < 1.0) {
    double g = gamma_mt(r, a + 1.0);
    return g * pow(u01o(r), 1.0 / a);
  }
  const double d = a - 1.0 / 3.0, c = 1.0 / sqrt(9.0 * d);
  for (;;) {
    double x, v;
    do {
      x = normal(r);
      v = 1.0 + c * x;
    } while (v <= 0.0);
    v = v * v * v;
    double u = u01o(r);
    if (log(u) < 0.5 * x * x + d - d * v + d * log(v)) return d * v;
  }
}

/* Cumulative table (float) of one 256-way distribution given as doubles. */
static void to_cdf(const double *p, float *cdf) {
  double s = 0.0, acc = 0.0;
  for (int v = 0; v < 256; ++v) s += p[v];
  if (!(s > 0.0)) {
    for (int v = 0; v < 256; ++v) cdf[v] = (float)((v + 1) / 256.0);
    return;
  }
  for (int v = 0; v < 256; ++v) {
    acc += p[v] / s;
    cdf[v] = (float)acc;
  }
}

/* Rows of an order-k Markov source: 256^k rows for k <= 2, else 65536 hashed
 * rows.  Row r is Dirichlet(alpha) drawn from its own generator, seeded with
 * splitmix64(seed ^ r), so it does not depend on any visit order. */
int64_t synth_markov_rows(int order) { return order <= 1 ? 256 : 65536; }

int synth_markov_table(int order, double alpha, uint64_t seed, float *cdf) {
  if (order < 1 || order > 4 || !(alpha > 0.0) || !cdf) return -1;
  const int64_t n = synth_markov_rows(order);
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < n; ++r) {
    xo256 g;
    xo_seed(&g, synth_splitmix64(seed ^ (uint64_t)r));
    double p[256];
    for (int v = 0; v < 256; ++v) p[v] = gamma_mt(&g, alpha);
    to_cdf(p, cdf + r * 256);
  }
  return 0;
}

/* Zipf(s) over ranks 1..256, rank r emitted as symbol perm[r-1] for a seeded
 * Fisher-Yates permutation. */
int synth_zipf_table(double s, uint64_t seed, float *cdf) {
  if (!cdf) return -1;
  xo256 g;
  xo_seed(&g, seed);
  int perm[256];
  for (int i = 0; i < 256; ++i) perm[i] = i;
  for (int i = 255; i > 0; --i) {
    int j = (int)(xo_next(&g) % (uint64_t)(i + 1));
    int t = perm[i];
    perm[i] = perm[j];
    perm[j] = t;
  }
  double q[256];
  for (int r = 1; r <= 256; ++r) q[perm[r - 1]] = pow((double)r, -s);
  to_cdf(q, cdf);
  return 0;
}

enum { SRC_MARKOV = 0, SRC_ZIPF = 1, SRC_UNIFORM = 2, SRC_RUNS = 3 };

typedef struct {
  int32_t type;
  int32_t order; /* markov only */
  const float *cdf;
} synth_source;

static inline int draw(xo256 *g, const float *cdf, double *bits) {
  const float tot = cdf[255];
  const double tgt = u01(g) * (double)tot;
  int lo = 0, hi = 255;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((double)cdf[mid] > tgt) hi = mid;
    else lo = mid + 1;
  }
  const double pv = ((double)cdf[lo] - (lo ? (double)cdf[lo - 1] : 0.0)) / (double)tot;
  *bits += -log2(pv);
  return lo;
}

static inline int64_t markov_row(uint32_t ctx, int order) {
  if (order <= 2) return (int64_t)ctx;
  return (int64_t)(((uint64_t)ctx * 0x9E3779B97F4A7C15ULL) >> 48);
}

/* Streams b = 0..B-1 of length L.  Segment s = [s*seg_len, (s+1)*seg_len) of
 * stream b is drawn from srcs[src_of[b*n_seg + s]]; the byte context carries
 * across segments.  stream_seed[b] seeds stream b's generator.  codelen[b]
 * receives the source's own code length of the stream in bits (first bytes
 * without a full context at 8 bits each). */
int synth_streams(uint8_t *out, int64_t B, int64_t L, const int32_t *src_of, int32_t n_seg,
                  int64_t seg_len, const synth_source *srcs, int32_t n_src,
                  const uint64_t *stream_seed, double *codelen) {
  if (!out || !src_of || !srcs || !stream_seed || B < 0 || L < 0 || n_seg < 1 || seg_len < 1) return -1;
  for (int64_t i = 0; i < B * (int64_t)n_seg; ++i)
    if (src_of[i] < 0 || src_of[i] >= n_src) return -1;
  const double p_end = 1.0 / 64.0;
  const double ln_keep = log(1.0 - p_end);
  const double bits_same = -log2((1.0 - p_end) + p_end / 256.0);
  const double bits_new = -log2(p_end / 256.0);
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t b = 0; b < B; ++b) {
    xo256 g;
    xo_seed(&g, stream_seed[b]);
    uint8_t *o = out + b * L;
    uint32_t ctx = 0;
    double bits = 0.0;
    int run_byte = -1;
    int64_t run_left = 0;
    for (int64_t i = 0; i < L; ++i) {
      int64_t seg = i / seg_len;
      if (seg >= n_seg) seg = n_seg - 1;
      const synth_source *S = &srcs[src_of[b * n_seg + seg]];
      int x;
      switch (S->type) {
        case SRC_MARKOV:
          if (i < S->order) {
            x = (int)(xo_next(&g) >> 56);
            bits += 8.0;
          } else {
            uint32_t c = S->order >= 4 ? ctx : (ctx & ((1u << (8 * S->order)) - 1u));
            x = draw(&g, S->cdf + markov_row(c, S->order) * 256, &bits);
          }
          break;
        case SRC_ZIPF:
          x = draw(&g, S->cdf, &bits);
          break;
        case SRC_UNIFORM:
          x = (int)(xo_next(&g) >> 56);
          bits += 8.0;
          break;
        default: /* SRC_RUNS: uniform byte repeated Geometric(1/64) times */
          if (run_left == 0) {
            int nb = (int)(xo_next(&g) >> 56);
            run_left = 1 + (int64_t)floor(log(u01o(&g)) / ln_keep);
            bits += (i == 0) ? 8.0 : (nb == run_byte ? bits_same : bits_new);
            run_byte = nb;
          } else {
            bits += bits_same;
          }
          --run_left;
          x = run_byte;
          break;
      }
      if (S->type != SRC_RUNS) run_left = 0, run_byte = x;
      o[i] = (uint8_t)x;
      ctx = (ctx << 8) | (uint32_t)x;
    }
    if (codelen) codelen[b] = bits;
  }
  return 0;
}
