/*
 * Seeded synthetic inputs for the mini-batch GNN path: graphs, feature
 * tables.  This module is shared by the CPU oracle and the GPU path as the
 * *input* source only; it holds none of the method's arithmetic (no
 * sampling, relabelling, aggregation or linear layers).
 *
 * Randomness: a counter-based SplitMix64 finaliser (Steele, Lea & Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014).  Every
 * value is a pure function of (seed, stream tag, index), so the outputs do
 * not depend on the number of threads.
 *
 * Graph generators:
 *   - directed G(n, p) by geometric skipping (Batagelj & Brandes, "Efficient
 *     generation of large random networks", Phys. Rev. E 71, 2005), stored as
 *     an in-neighbour CSR (row v lists the sources u of edges u -> v);
 *   - R-MAT (Chakrabarti, Zhan & Faloutsos, SDM 2004) with a seeded vertex
 *     permutation, rejection of permuted ids >= N, self-loop removal,
 *     symmetrisation and de-duplication;
 *   - hub injection: extra distinct in-sources for chosen vertices, then the
 *     graph is symmetrised and de-duplicated again.
 * Every CSR produced here has rows sorted ascending, unique, and without
 * self-loops.
 *
 * Features: N(0,1) by Box-Muller in double, rounded to fp32 (and, for the
 * bf16 tables, fp32 -> bf16 round-to-nearest-even).
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* Key of an independent stream: derived from the user seed and a tag. */
static inline uint64_t dg_key(uint64_t seed, uint64_t tag) {
  return mix64(mix64(seed + GOLDEN) ^ (tag * 0xD1B54A32D192ED03ULL));
}

/* i-th 64-bit word of stream `key`. */
static inline uint64_t dg_word(uint64_t key, uint64_t i) {
  return mix64(key + (i + 1) * GOLDEN);
}

/* Uniform double in [0, 1). */
static inline double dg_unif(uint64_t key, uint64_t i) {
  return (double)(dg_word(key, i) >> 11) * (1.0 / 9007199254740992.0);
}

/* ------------------------------------------------------------------ */
/* tiny thread pool helper: run fn(arg, tid, nthreads) on nthreads     */

typedef void (*dg_fn)(void* arg, int tid, int nth);
typedef struct { dg_fn fn; void* arg; int tid, nth; } dg_job;

static void* dg_tramp(void* p) {
  dg_job* j = (dg_job*)p;
  j->fn(j->arg, j->tid, j->nth);
  return NULL;
}

static int g_threads = 0;

void dg_set_threads(int n) { g_threads = n; }

static int dg_nthreads(void) {
  if (g_threads > 0) return g_threads;
  long n = sysconf(_SC_NPROCESSORS_ONLN);
  if (n < 1) n = 1;
  if (n > 16) n = 16;
  return (int)n;
}

static void dg_parallel(dg_fn fn, void* arg) {
  int nth = dg_nthreads();
  pthread_t th[64];
  dg_job jobs[64];
  if (nth > 64) nth = 64;
  for (int t = 0; t < nth; ++t) {
    jobs[t].fn = fn; jobs[t].arg = arg; jobs[t].tid = t; jobs[t].nth = nth;
    if (t > 0) pthread_create(&th[t], NULL, dg_tramp, &jobs[t]);
  }
  dg_tramp(&jobs[0]);
  for (int t = 1; t < nth; ++t) pthread_join(th[t], NULL);
}

static inline void dg_range(int64_t n, int tid, int nth, int64_t* b, int64_t* e) {
  int64_t chunk = (n + nth - 1) / nth;
  *b = chunk * tid;
  *e = *b + chunk;
  if (*b > n) *b = n;
  if (*e > n) *e = n;
}

/* ------------------------------------------------------------------ */
/* directed G(n, p), in-neighbour CSR                                  */

typedef struct {
  int64_t n; double p; uint64_t key;
  int64_t* indptr;   /* [n+1]; pass 1 writes counts at indptr[v+1] */
  int32_t* indices;  /* NULL in pass 1 */
} er_arg;

static void er_row(const er_arg* a, int64_t v, int32_t* out, int64_t* count) {
  const int64_t cand = a->n - 1;          /* every u != v */
  const double lp = log1p(-a->p);
  const uint64_t rkey = dg_key(a->key, (uint64_t)v);
  int64_t w = -1, c = 0;
  uint64_t i = 0;
  for (;;) {
    double r = dg_unif(rkey, i++);
    w += 1 + (int64_t)floor(log1p(-r) / lp);
    if (w >= cand) break;
    if (out) out[c] = (int32_t)(w < v ? w : w + 1);
    ++c;
  }
  *count = c;
}

static void er_pass(void* p, int tid, int nth) {
  er_arg* a = (er_arg*)p;
  int64_t b, e;
  dg_range(a->n, tid, nth, &b, &e);
  for (int64_t v = b; v < e; ++v) {
    int64_t c;
    if (a->indices == NULL) {
      er_row(a, v, NULL, &c);
      a->indptr[v + 1] = c;
    } else {
      er_row(a, v, a->indices + a->indptr[v], &c);
    }
  }
}

/* Pass 1: returns the edge count and fills indptr[n+1]. */
int64_t dg_er_count(int64_t n, double p, uint64_t seed, int64_t* indptr) {
  er_arg a = {n, p, dg_key(seed, 1), indptr, NULL};
  indptr[0] = 0;
  dg_parallel(er_pass, &a);
  for (int64_t v = 0; v < n; ++v) indptr[v + 1] += indptr[v];
  return indptr[n];
}

/* Pass 2: fills indices (size from pass 1). */
void dg_er_fill(int64_t n, double p, uint64_t seed, const int64_t* indptr, int32_t* indices) {
  er_arg a = {n, p, dg_key(seed, 1), (int64_t*)indptr, indices};
  dg_parallel(er_pass, &a);
}

/* ------------------------------------------------------------------ */
/* edge list -> sorted, de-duplicated CSR (rows = destination)         */

typedef struct {
  int64_t n, m;
  const int32_t* src; const int32_t* dst;   /* m directed edges src -> dst */
  int64_t* cnt;        /* [n+1] */
  int64_t* cursor;     /* [n] */
  int32_t* tmp;        /* [m] */
  int64_t* newdeg;     /* [n+1] */
  int32_t* out;        /* final indices */
  int phase;
} csr_arg;

static int cmp_i32(const void* x, const void* y) {
  int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
  return (a > b) - (a < b);
}

static void csr_pass(void* p, int tid, int nth) {
  csr_arg* a = (csr_arg*)p;
  int64_t b, e;
  if (a->phase == 0) {            /* count */
    dg_range(a->m, tid, nth, &b, &e);
    for (int64_t i = b; i < e; ++i)
      __atomic_fetch_add(&a->cnt[a->dst[i] + 1], 1, __ATOMIC_RELAXED);
  } else if (a->phase == 1) {     /* scatter */
    dg_range(a->m, tid, nth, &b, &e);
    for (int64_t i = b; i < e; ++i) {
      int64_t pos = __atomic_fetch_add(&a->cursor[a->dst[i]], 1, __ATOMIC_RELAXED);
      a->tmp[pos] = a->src[i];
    }
  } else if (a->phase == 2) {     /* sort + unique each row */
    dg_range(a->n, tid, nth, &b, &e);
    for (int64_t v = b; v < e; ++v) {
      int32_t* row = a->tmp + a->cnt[v];
      int64_t len = a->cnt[v + 1] - a->cnt[v];
      qsort(row, (size_t)len, sizeof(int32_t), cmp_i32);
      int64_t k = 0;
      for (int64_t i = 0; i < len; ++i)
        if (row[i] != v && (k == 0 || row[i] != row[k - 1])) row[k++] = row[i];
      a->newdeg[v + 1] = k;
    }
  } else {                        /* compact */
    dg_range(a->n, tid, nth, &b, &e);
    for (int64_t v = b; v < e; ++v) {
      int64_t len = a->newdeg[v + 1] - a->newdeg[v];
      memcpy(a->out + a->newdeg[v], a->tmp + a->cnt[v], (size_t)len * sizeof(int32_t));
    }
  }
}

/* Builds the CSR of the given directed edges (duplicates and self-loops are
 * dropped).  *indices_out is malloc'ed; indptr must hold n+1 entries.
 * Returns nnz, or -1 on allocation failure. */
static int64_t build_csr(int64_t n, int64_t m, const int32_t* src, const int32_t* dst,
                         int64_t* indptr, int32_t** indices_out) {
  csr_arg a;
  memset(&a, 0, sizeof a);
  a.n = n; a.m = m; a.src = src; a.dst = dst;
  a.cnt = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
  a.cursor = (int64_t*)malloc((size_t)n * sizeof(int64_t));
  a.tmp = (int32_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(int32_t));
  a.newdeg = indptr;
  if (!a.cnt || !a.cursor || !a.tmp) { free(a.cnt); free(a.cursor); free(a.tmp); return -1; }
  a.phase = 0; dg_parallel(csr_pass, &a);
  for (int64_t v = 0; v < n; ++v) a.cnt[v + 1] += a.cnt[v];
  memcpy(a.cursor, a.cnt, (size_t)n * sizeof(int64_t));
  a.phase = 1; dg_parallel(csr_pass, &a);
  indptr[0] = 0;
  a.phase = 2; dg_parallel(csr_pass, &a);
  for (int64_t v = 0; v < n; ++v) indptr[v + 1] += indptr[v];
  a.out = (int32_t*)malloc((size_t)(indptr[n] > 0 ? indptr[n] : 1) * sizeof(int32_t));
  if (!a.out) { free(a.cnt); free(a.cursor); free(a.tmp); return -1; }
  a.phase = 3; dg_parallel(csr_pass, &a);
  free(a.cnt); free(a.cursor); free(a.tmp);
  *indices_out = a.out;
  return indptr[n];
}

void dg_free(void* p) { free(p); }

/* ------------------------------------------------------------------ */
/* R-MAT                                                               */

typedef struct {
  int scale; int64_t n; int64_t draws; uint64_t key;
  uint32_t ta, tab, tabc;    /* cumulative 32-bit thresholds of a, a+b, a+b+c */
  const int32_t* perm;       /* [2^scale] */
  int32_t* src; int32_t* dst;  /* [2*draws]; rejected draws are marked -1 */
} rmat_arg;

static void rmat_pass(void* p, int tid, int nth) {
  rmat_arg* a = (rmat_arg*)p;
  int64_t b, e;
  dg_range(a->draws, tid, nth, &b, &e);
  const int words = (a->scale + 1) / 2;
  for (int64_t i = b; i < e; ++i) {
    uint64_t u = 0, v = 0;
    int level = 0;
    for (int w = 0; w < words; ++w) {
      uint64_t r = dg_word(a->key, (uint64_t)i * (uint64_t)words + (uint64_t)w);
      for (int h = 0; h < 2 && level < a->scale; ++h, ++level) {
        uint32_t q = (uint32_t)(r >> (32 * h));
        uint64_t bu = 0, bv = 0;
        if (q < a->ta) { bu = 0; bv = 0; }
        else if (q < a->tab) { bu = 0; bv = 1; }
        else if (q < a->tabc) { bu = 1; bv = 0; }
        else { bu = 1; bv = 1; }
        u = (u << 1) | bu;
        v = (v << 1) | bv;
      }
    }
    int32_t pu = a->perm[u], pv = a->perm[v];
    int ok = pu < a->n && pv < a->n && pu != pv;
    a->src[2 * i] = ok ? pu : -1;     a->dst[2 * i] = ok ? pv : -1;
    a->src[2 * i + 1] = ok ? pv : -1; a->dst[2 * i + 1] = ok ? pu : -1;
  }
}

static void seeded_perm(int32_t* perm, int64_t n, uint64_t key) {
  for (int64_t i = 0; i < n; ++i) perm[i] = (int32_t)i;
  for (int64_t i = n - 1; i > 0; --i) {
    /* j uniform in [0, i] (multiply-shift; bias < 2^-30, irrelevant for inputs) */
    uint64_t r = dg_word(key, (uint64_t)i) >> 32;
    int64_t j = (int64_t)((r * (uint64_t)(i + 1)) >> 32);
    int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
  }
}

/* Symmetrised R-MAT CSR.  Returns nnz (>= 0) and sets *indices_out
 * (malloc'ed; free with dg_free), or -1 on failure. */
int64_t dg_rmat(int scale, int64_t n, int64_t draws, double a, double b, double c,
                uint64_t seed, int64_t* indptr, int32_t** indices_out) {
  int64_t full = (int64_t)1 << scale;
  if (n > full || n <= 0) return -1;
  int32_t* perm = (int32_t*)malloc((size_t)full * sizeof(int32_t));
  int32_t* src = (int32_t*)malloc((size_t)(2 * draws) * sizeof(int32_t));
  int32_t* dst = (int32_t*)malloc((size_t)(2 * draws) * sizeof(int32_t));
  if (!perm || !src || !dst) { free(perm); free(src); free(dst); return -1; }
  seeded_perm(perm, full, dg_key(seed, 2));
  rmat_arg ra;
  ra.scale = scale; ra.n = n; ra.draws = draws; ra.key = dg_key(seed, 3);
  ra.ta = (uint32_t)llround(a * 4294967296.0);
  ra.tab = (uint32_t)llround((a + b) * 4294967296.0);
  ra.tabc = (uint32_t)llround((a + b + c) * 4294967296.0);
  ra.perm = perm; ra.src = src; ra.dst = dst;
  dg_parallel(rmat_pass, &ra);
  free(perm);
  /* squeeze out rejected draws */
  int64_t m = 0;
  for (int64_t i = 0; i < 2 * draws; ++i)
    if (src[i] >= 0) { src[m] = src[i]; dst[m] = dst[i]; ++m; }
  int64_t nnz = build_csr(n, m, src, dst, indptr, indices_out);
  free(src); free(dst);
  return nnz;
}

/* Adds `num_hubs` hub vertices to a CSR: hub h (a distinct seeded vertex)
 * receives `hub_deg` distinct seeded sources; all added edges are
 * symmetrised and the result de-duplicated.  Hub ids are written to
 * hubs_out[num_hubs].  Returns the new nnz and sets *indices_out. */
int64_t dg_inject_hubs(int64_t n, const int64_t* indptr_in, const int32_t* indices_in,
                       int64_t num_hubs, int64_t hub_deg, uint64_t seed,
                       int64_t* hubs_out, int64_t* indptr_out, int32_t** indices_out) {
  if (hub_deg >= n || num_hubs > n) return -1;
  int64_t nnz0 = indptr_in[n];
  int64_t extra = 2 * num_hubs * hub_deg;
  int64_t m = nnz0 + extra;
  int32_t* src = (int32_t*)malloc((size_t)m * sizeof(int32_t));
  int32_t* dst = (int32_t*)malloc((size_t)m * sizeof(int32_t));
  int32_t* perm = (int32_t*)malloc((size_t)n * sizeof(int32_t));
  if (!src || !dst || !perm) { free(src); free(dst); free(perm); return -1; }
  for (int64_t v = 0; v < n; ++v)
    for (int64_t e = indptr_in[v]; e < indptr_in[v + 1]; ++e) { src[e] = indices_in[e]; dst[e] = (int32_t)v; }
  /* hubs: first num_hubs entries of a seeded permutation */
  seeded_perm(perm, n, dg_key(seed, 4));
  int64_t pos = nnz0;
  for (int64_t h = 0; h < num_hubs; ++h) {
    int32_t hub = perm[h];
    hubs_out[h] = hub;
    /* hub_deg distinct sources by a partial Fisher-Yates over a private permutation */
    int32_t* cand = (int32_t*)malloc((size_t)n * sizeof(int32_t));
    if (!cand) { free(src); free(dst); free(perm); return -1; }
    for (int64_t i = 0; i < n; ++i) cand[i] = (int32_t)i;
    uint64_t hk = dg_key(seed, 1000 + (uint64_t)h);
    int64_t taken = 0, i = 0;
    while (taken < hub_deg) {
      uint64_t r = dg_word(hk, (uint64_t)i) >> 32;
      int64_t j = i + (int64_t)((r * (uint64_t)(n - i)) >> 32);
      int32_t t = cand[i]; cand[i] = cand[j]; cand[j] = t;
      if (cand[i] != hub) {
        src[pos] = cand[i]; dst[pos] = hub; ++pos;
        src[pos] = hub; dst[pos] = cand[i]; ++pos;
        ++taken;
      }
      ++i;
    }
    free(cand);
  }
  free(perm);
  int64_t nnz = build_csr(n, pos, src, dst, indptr_out, indices_out);
  free(src); free(dst);
  return nnz;
}

/* ------------------------------------------------------------------ */
/* features                                                            */

typedef struct {
  int64_t rows; int64_t dim; uint64_t key; int bf16;
  float* f32; uint16_t* b16;
} feat_arg;

static inline uint16_t f32_to_bf16_rne(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static void feat_pass(void* p, int tid, int nth) {
  feat_arg* a = (feat_arg*)p;
  int64_t b, e;
  dg_range(a->rows, tid, nth, &b, &e);
  const double two_pi = 6.283185307179586476925286766559;
  for (int64_t r = b; r < e; ++r) {
    for (int64_t c = 0; c < a->dim; ++c) {
      uint64_t idx = (uint64_t)(r * a->dim + c);
      double u1 = 1.0 - dg_unif(a->key, 2 * idx);     /* (0, 1] */
      double u2 = dg_unif(a->key, 2 * idx + 1);
      double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
      float f = (float)z;
      if (a->bf16) a->b16[idx] = f32_to_bf16_rne(f);
      else a->f32[idx] = f;
    }
  }
}

void dg_features_f32(int64_t rows, int64_t dim, uint64_t seed, float* out) {
  feat_arg a = {rows, dim, dg_key(seed, 5), 0, out, NULL};
  dg_parallel(feat_pass, &a);
}

void dg_features_bf16(int64_t rows, int64_t dim, uint64_t seed, uint16_t* out) {
  feat_arg a = {rows, dim, dg_key(seed, 5), 1, NULL, out};
  dg_parallel(feat_pass, &a);
}
