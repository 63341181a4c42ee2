/*
 * Seeded synthetic inputs for the K-VEC eviction step.
 *
 * This module generates the Q window rows, the K cache and the V cache that
 * both the CPU oracle and the GPU library consume.  It holds none of the
 * eviction method's arithmetic: it only draws Gaussian tensors, applies the
 * rotary position embedding to Q and K, and plants "heavy-hitter" keys.
 *
 * Every value is a pure function of (seed, tensor tag, layer, sequence, head,
 * position, dimension), so any slice can be regenerated independently:
 *
 *   hash     : the SplitMix64 output function (Steele, Lea and Flood, OOPSLA
 *              2014), used as a counter-based generator.  The n-th draw of a
 *              stream with key s is mix64(s + (n + 1) * 0x9e3779b97f4a7c15).
 *   stream key: key = mix64(seed + tag*GAMMA); then key = mix64(key + a) for
 *              each of (layer, sequence, head) in that order.
 *   Gaussians: Box-Muller in double precision; one 64-bit draw gives a pair
 *              (its high and low 32-bit halves are the two uniforms), and the
 *              pair fills the two consecutive dimensions 2m and 2m+1.
 *   RoPE     : rotate-half pairing (i, i + d/2), frequency theta^(-2i/d),
 *              position = absolute token index, applied in double.
 *   heavy hitters: for t in the head's position set, k_t += s * sqrt(d) * u,
 *              u = a normalised Gaussian direction of the (layer, seq, head);
 *              added after RoPE.  Sinks (t < sink_count) add a second
 *              direction scaled by sink_scale.
 *   rounding : double -> fp32 (round to nearest even) -> bf16 (round to
 *              nearest even) for bf16 tensors; double -> fp32 for fp32 ones.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GAMMA 0x9e3779b97f4a7c15ULL

enum { TAG_Q = 1, TAG_K = 2, TAG_V = 3, TAG_DIR = 4, TAG_SINKDIR = 5,
       TAG_POS = 6, TAG_POS_CORE = 7, TAG_PERM = 8 };

typedef struct synth_cfg {
  uint64_t seed;
  int32_t n_layers, batch, n_kv_heads, n_q_heads, head_dim;
  int32_t seq_len;      /* T */
  int32_t window;       /* O: positions [T-O, T) are the observation window */
  int32_t window_ext;   /* O': number of query rows generated (clamped to T) */
  int32_t dtype;        /* 0 = bf16 (uint16 storage), 1 = fp32 */
  int32_t rope;         /* 1 = apply RoPE to Q and K */
  double rope_theta;
  int32_t hh_count;     /* heavy-hitter positions per (layer, seq, head) */
  int32_t hh_shared;    /* of which this many are shared by every head */
  double hh_scale;
  int32_t sink_count;   /* positions [0, sink_count) get the sink direction */
  double sink_scale;
  int32_t zipf_clusters;/* > 0: positions drawn from a Zipf law over clusters */
  double zipf_s;
} synth_cfg;

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t key, uint64_t n) { return mix64(key + (n + 1) * GAMMA); }

static uint64_t stream_key(uint64_t seed, int tag, int64_t a, int64_t b, int64_t c) {
  uint64_t k = mix64(seed + (uint64_t)tag * GAMMA);
  k = mix64(k + (uint64_t)a);
  k = mix64(k + (uint64_t)b);
  k = mix64(k + (uint64_t)c);
  return k;
}

/* Two independent N(0,1) values from one 64-bit draw (Box-Muller). */
static inline void gauss_pair(uint64_t h, double* z0, double* z1) {
  const double u1 = ((double)(h >> 32) + 0.5) * (1.0 / 4294967296.0);
  const double u2 = ((double)(h & 0xffffffffULL) + 0.5) * (1.0 / 4294967296.0);
  const double r = sqrt(-2.0 * log(u1));
  const double a = 6.283185307179586476925286766559 * u2;
  *z0 = r * cos(a);
  *z1 = r * sin(a);
}

/* Uniform integer in [0, n) from a draw (multiply-shift on the high half). */
static inline int64_t uniform_below(uint64_t h, int64_t n) {
  return (int64_t)(((h >> 32) * (uint64_t)n) >> 32);
}

static inline uint16_t f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40); /* NaN */
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static inline void store(const synth_cfg* c, void* out, int64_t i, double v) {
  const float f = (float)v;
  if (c->dtype == 0) ((uint16_t*)out)[i] = f32_to_bf16(f);
  else ((float*)out)[i] = f;
}

static int candidates(const synth_cfg* c) {
  int tc = c->seq_len - c->window;
  return tc < 0 ? 0 : tc;
}

static int window_rows(const synth_cfg* c) {
  return c->window_ext < c->seq_len ? c->window_ext : c->seq_len;
}

/* Unit direction of length d for (tag, layer, seq, head). */
static void direction(const synth_cfg* c, int tag, int layer, int b, int h, double* u) {
  const int d = c->head_dim;
  const uint64_t key = stream_key(c->seed, tag, layer, b, h);
  double nrm = 0.0;
  for (int m = 0; m < d / 2; ++m) {
    double z0, z1;
    gauss_pair(draw(key, (uint64_t)m), &z0, &z1);
    u[2 * m] = z0;
    u[2 * m + 1] = z1;
  }
  for (int i = 0; i < d; ++i) nrm += u[i] * u[i];
  nrm = sqrt(nrm);
  for (int i = 0; i < d; ++i) u[i] /= nrm;
}

/* Draw `want` distinct positions in [0, tc) into `mark` (byte map), rejecting
 * positions already marked.  Returns how many were added. */
static int draw_uniform_set(uint64_t key, int want, int tc, unsigned char* mark, int already) {
  int added = 0;
  uint64_t n = 0;
  if (want > tc - already) want = tc - already;
  while (added < want) {
    const int64_t p = uniform_below(draw(key, n++), tc);
    if (!mark[p]) { mark[p] = 1; ++added; }
  }
  return added;
}

/* Zipf-over-clusters draw: clusters of size ceil(T/C) ranked by a seeded
 * permutation of the (layer, seq); P(rank r) proportional to r^-s; uniform
 * within the cluster; positions >= tc or already marked are rejected. */
static int draw_zipf_set(const synth_cfg* c, int layer, int b, int h, int want, int tc,
                         unsigned char* mark) {
  const int C = c->zipf_clusters;
  const int csize = (c->seq_len + C - 1) / C;
  int* perm = (int*)malloc(sizeof(int) * (size_t)C);
  double* cdf = (double*)malloc(sizeof(double) * (size_t)C);
  const uint64_t pkey = stream_key(c->seed, TAG_PERM, layer, b, 0);
  for (int i = 0; i < C; ++i) perm[i] = i;
  for (int i = C - 1; i > 0; --i) { /* Fisher-Yates */
    const int j = (int)uniform_below(draw(pkey, (uint64_t)i), i + 1);
    const int t = perm[i]; perm[i] = perm[j]; perm[j] = t;
  }
  double acc = 0.0;
  for (int r = 0; r < C; ++r) { acc += pow((double)(r + 1), -c->zipf_s); cdf[r] = acc; }
  const uint64_t key = stream_key(c->seed, TAG_POS, layer, b, h);
  int added = 0;
  uint64_t n = 0;
  int64_t budget = 1000LL * (want + 1);
  while (added < want && budget-- > 0) {
    const uint64_t h1 = draw(key, n++);
    const double u = ((double)(h1 >> 11) + 0.5) * (1.0 / 9007199254740992.0) * acc;
    int lo = 0, hi = C - 1;
    while (lo < hi) { const int mid = (lo + hi) / 2; if (cdf[mid] < u) lo = mid + 1; else hi = mid; }
    const int64_t p = (int64_t)perm[lo] * csize + uniform_below(draw(key, n++), csize);
    if (p >= tc || mark[p]) continue;
    mark[p] = 1;
    ++added;
  }
  free(perm);
  free(cdf);
  return added;
}

/* Heavy-hitter position set of (layer, seq, head) as a byte map over [0, tc). */
static void hh_mark(const synth_cfg* c, int layer, int b, int h, unsigned char* mark) {
  const int tc = candidates(c);
  memset(mark, 0, (size_t)tc);
  if (tc == 0 || c->hh_count <= 0) return;
  int want = c->hh_count;
  if (c->zipf_clusters > 0) { draw_zipf_set(c, layer, b, h, want, tc, mark); return; }
  int have = 0;
  if (c->hh_shared > 0) {
    have = draw_uniform_set(stream_key(c->seed, TAG_POS_CORE, layer, b, 0),
                            c->hh_shared < want ? c->hh_shared : want, tc, mark, 0);
  }
  draw_uniform_set(stream_key(c->seed, TAG_POS, layer, b, h), want - have, tc, mark, have);
}

/* Sorted heavy-hitter positions of (layer, seq, head); returns the count. */
int synth_hh_positions(const synth_cfg* c, int layer, int b, int h, int32_t* out, int cap) {
  const int tc = candidates(c);
  unsigned char* mark = (unsigned char*)malloc((size_t)(tc > 0 ? tc : 1));
  hh_mark(c, layer, b, h, mark);
  int n = 0;
  for (int t = 0; t < tc; ++t)
    if (mark[t]) { if (n < cap) out[n] = t; ++n; }
  free(mark);
  return n;
}

/* cos/sin table for positions [p0, p0 + np), pairs i < d/2. */
static void rope_table(const synth_cfg* c, int64_t p0, int64_t np, double* cs, double* sn) {
  const int half = c->head_dim / 2;
  double* inv = (double*)malloc(sizeof(double) * (size_t)half);
  for (int i = 0; i < half; ++i) inv[i] = pow(c->rope_theta, -2.0 * i / c->head_dim);
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < np; ++p) {
    for (int i = 0; i < half; ++i) {
      const double a = (double)(p0 + p) * inv[i];
      cs[p * half + i] = cos(a);
      sn[p * half + i] = sin(a);
    }
  }
  free(inv);
}

/* Gaussian row x[0..d) of stream `key` at row index `row`. */
static inline void gauss_row(uint64_t key, int64_t row, int d, double* x) {
  for (int m = 0; m < d / 2; ++m) {
    double z0, z1;
    gauss_pair(draw(key, (uint64_t)(row * (d / 2) + m)), &z0, &z1);
    x[2 * m] = z0;
    x[2 * m + 1] = z1;
  }
}

static inline void rope_apply(int d, const double* cs, const double* sn, double* x) {
  const int half = d / 2;
  for (int i = 0; i < half; ++i) {
    const double a = x[i], b = x[i + half];
    x[i] = a * cs[i] - b * sn[i];
    x[i + half] = b * cs[i] + a * sn[i];
  }
}

/* K rows of heads [h0,h1) and positions [t0,t1) of (layer, seq b).
 * Output layout: [h1-h0][t1-t0][d]. */
void synth_keys(const synth_cfg* c, int layer, int b, int h0, int h1, int t0, int t1, void* out) {
  const int d = c->head_dim, half = d / 2, tc = candidates(c);
  const int64_t nt = t1 - t0;
  double *cs = NULL, *sn = NULL;
  if (c->rope) {
    cs = (double*)malloc(sizeof(double) * (size_t)(nt * half + 1));
    sn = (double*)malloc(sizeof(double) * (size_t)(nt * half + 1));
    rope_table(c, t0, nt, cs, sn);
  }
  for (int h = h0; h < h1; ++h) {
    unsigned char* mark = (unsigned char*)malloc((size_t)(tc > 0 ? tc : 1));
    hh_mark(c, layer, b, h, mark);
    double u[512], us[512];
    direction(c, TAG_DIR, layer, b, h, u);
    direction(c, TAG_SINKDIR, layer, b, h, us);
    const uint64_t key = stream_key(c->seed, TAG_K, layer, b, h);
    const double hs = c->hh_scale * sqrt((double)d), ss = c->sink_scale * sqrt((double)d);
#pragma omp parallel for schedule(static)
    for (int64_t tt = 0; tt < nt; ++tt) {
      const int64_t t = t0 + tt;
      double x[512];
      gauss_row(key, t, d, x);
      if (c->rope) rope_apply(d, cs + tt * half, sn + tt * half, x);
      if (t < tc && mark[t]) for (int i = 0; i < d; ++i) x[i] += hs * u[i];
      if (t < c->sink_count) for (int i = 0; i < d; ++i) x[i] += ss * us[i];
      const int64_t base = ((int64_t)(h - h0) * nt + tt) * d;
      for (int i = 0; i < d; ++i) store(c, out, base + i, x[i]);
    }
    free(mark);
  }
  free(cs);
  free(sn);
}

/* V rows of heads [h0,h1) and positions [t0,t1): plain N(0,1). */
void synth_values(const synth_cfg* c, int layer, int b, int h0, int h1, int t0, int t1, void* out) {
  const int d = c->head_dim;
  const int64_t nt = t1 - t0;
  for (int h = h0; h < h1; ++h) {
    const uint64_t key = stream_key(c->seed, TAG_V, layer, b, h);
#pragma omp parallel for schedule(static)
    for (int64_t tt = 0; tt < nt; ++tt) {
      double x[512];
      gauss_row(key, t0 + tt, d, x);
      const int64_t base = ((int64_t)(h - h0) * nt + tt) * d;
      for (int i = 0; i < d; ++i) store(c, out, base + i, x[i]);
    }
  }
}

/* Q window rows of query heads [j0,j1) of (layer, seq b): the last O' positions
 * T-O'..T-1 (O' clamped to T).  Output layout: [j1-j0][O'][d]. */
void synth_queries(const synth_cfg* c, int layer, int b, int j0, int j1, void* out) {
  const int d = c->head_dim, half = d / 2, wn = window_rows(c);
  const int64_t p0 = (int64_t)c->seq_len - wn;
  double *cs = NULL, *sn = NULL;
  if (c->rope) {
    cs = (double*)malloc(sizeof(double) * (size_t)(wn * half + 1));
    sn = (double*)malloc(sizeof(double) * (size_t)(wn * half + 1));
    rope_table(c, p0, wn, cs, sn);
  }
  for (int j = j0; j < j1; ++j) {
    const uint64_t key = stream_key(c->seed, TAG_Q, layer, b, j);
    for (int r = 0; r < wn; ++r) {
      double x[512];
      gauss_row(key, p0 + r, d, x);
      if (c->rope) rope_apply(d, cs + (int64_t)r * half, sn + (int64_t)r * half, x);
      const int64_t base = ((int64_t)(j - j0) * wn + r) * d;
      for (int i = 0; i < d; ++i) store(c, out, base + i, x[i]);
    }
  }
  free(cs);
  free(sn);
}
