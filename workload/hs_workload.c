/*
 * Seeded synthetic inputs for the HiSparse decode hot path: KV records, decode queries
 * and per-step top-k selection streams.
 *
 * This module holds none of the method's arithmetic (no residency, no replacement, no
 * attention). It only draws inputs, so both the GPU path's tests/benchmark and the CPU
 * oracle can consume the same bytes. Every value is a pure function of (seed, coordinates):
 * any record, query or step can be regenerated independently.
 *
 * Random numbers: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014), used both as a counter hash (hs_key) and as a sequential
 * generator seeded per (stream, step).
 *
 * Normal values: a 65536-entry inverse-CDF table of N(0,1) at the midpoints (i + 0.5)/65536,
 * each rounded to bf16 (round-to-nearest-even); a 16-bit slice of a hash indexes it. This is
 * an exact 16-bit quantile sampler of N(0,1) (tails truncated at about 4.2 sigma), finer
 * than bf16's own 8-bit significand.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { DOM_KV = 1, DOM_Q = 2, DOM_SEL = 3, DOM_PERM = 4, DOM_BASE = 5 };

static inline uint64_t sm64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

uint64_t hs_splitmix64(uint64_t x) { return sm64(x); }

uint64_t hs_key(uint64_t seed, uint64_t a, uint64_t b, uint64_t c, uint64_t d) {
  uint64_t h = sm64(seed);
  h = sm64(h ^ a);
  h = sm64(h ^ b);
  h = sm64(h ^ c);
  return sm64(h ^ d);
}

/* sequential SplitMix64 */
typedef struct { uint64_t s; } rng_t;
static inline uint64_t rng_next(rng_t* r) {
  r->s += 0x9E3779B97F4A7C15ull;
  uint64_t z = r->s;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static inline double rng_unif(rng_t* r) { return (double)(rng_next(r) >> 11) * 0x1.0p-53; }
static inline uint64_t rng_below(rng_t* r, uint64_t n) {
  return (uint64_t)(((unsigned __int128)rng_next(r) * n) >> 64);
}

/* ---------------- N(0,1) quantile table in bf16 ---------------- */
static uint16_t g_norm[65536];
static pthread_once_t g_norm_once = PTHREAD_ONCE_INIT;

static uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)(u >> 16); /* inf/nan: not produced */
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

static void build_norm_table(void) {
  for (int i = 0; i < 65536; ++i) {
    double p = (i + 0.5) / 65536.0, lo = -12.0, hi = 12.0;
    for (int it = 0; it < 90; ++it) { /* bisection on Phi(x) = erfc(-x/sqrt2)/2 */
      double mid = 0.5 * (lo + hi);
      if (0.5 * erfc(-mid / sqrt(2.0)) < p) lo = mid; else hi = mid;
    }
    g_norm[i] = f32_to_bf16_rne((float)(0.5 * (lo + hi)));
  }
}

const uint16_t* hs_normal_table(void) {
  pthread_once(&g_norm_once, build_norm_table);
  return g_norm;
}

/* ---------------- KV records ---------------- */
/* Element e of record r of (layer, unit) is g_norm[16-bit lane (e & 3) of sm64(h_rec ^ (e >> 2))],
 * with h_rec = hs_key(seed, DOM_KV, layer, unit, r). */
static void kv_record(uint16_t* dst, int32_t elems, uint64_t seed, int32_t layer, int64_t unit,
                      int64_t rec) {
  uint64_t h = hs_key(seed, DOM_KV, (uint64_t)layer, (uint64_t)unit, (uint64_t)rec);
  int32_t g = 0;
  for (; 4 * g + 3 < elems; ++g) {
    uint64_t w = sm64(h ^ (uint64_t)g);
    dst[4 * g + 0] = g_norm[w & 0xFFFF];
    dst[4 * g + 1] = g_norm[(w >> 16) & 0xFFFF];
    dst[4 * g + 2] = g_norm[(w >> 32) & 0xFFFF];
    dst[4 * g + 3] = g_norm[(w >> 48) & 0xFFFF];
  }
  if (4 * g < elems) {
    uint64_t w = sm64(h ^ (uint64_t)g);
    for (int32_t e = 4 * g; e < elems; ++e, w >>= 16) dst[e] = g_norm[w & 0xFFFF];
  }
}

typedef struct {
  uint16_t* dst;
  uint64_t seed;
  int32_t layer, elems;
  int64_t unit0, n_units, rec0, n_rec, begin, end; /* [begin, end) over n_units * n_rec */
} kv_job_t;

static void* kv_worker(void* arg) {
  kv_job_t* j = (kv_job_t*)arg;
  for (int64_t i = j->begin; i < j->end; ++i) {
    int64_t u = i / j->n_rec, r = i % j->n_rec;
    kv_record(j->dst + i * (int64_t)j->elems, j->elems, j->seed, j->layer, j->unit0 + u,
              j->rec0 + r);
  }
  return NULL;
}

/* Fill dst[n_units][n_rec][elems] (bf16 bits) with records (unit0+u, rec0+r) of `layer`. */
int hs_fill_kv(void* dst, uint64_t seed, int32_t layer, int64_t unit0, int64_t n_units,
               int64_t rec0, int64_t n_rec, int32_t elems, int32_t nthreads) {
  if (!dst || elems <= 0 || n_units < 0 || n_rec < 0) return -1;
  hs_normal_table();
  int64_t total = n_units * n_rec;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (total < 4096) nthreads = 1;
  kv_job_t jobs[256];
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = (kv_job_t){(uint16_t*)dst, seed, layer, elems, unit0, n_units, rec0, n_rec,
                         total * t / nthreads, total * (t + 1) / nthreads};
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, kv_worker, &jobs[t]);
  kv_worker(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
  return 0;
}

/* ---------------- decode queries ---------------- */
/* q[u][h][d] for (step, layer, unit0+u, head h): lane (d & 3) of sm64(hs_key(seed, DOM_Q, step,
 * layer, (unit*heads + h)) ^ (d >> 2)). */
int hs_fill_q(void* dst, uint64_t seed, int32_t step, int32_t layer, int64_t unit0,
              int64_t n_units, int32_t heads, int32_t dim) {
  if (!dst || heads <= 0 || dim <= 0) return -1;
  hs_normal_table();
  uint16_t* q = (uint16_t*)dst;
  for (int64_t u = 0; u < n_units; ++u)
    for (int32_t h = 0; h < heads; ++h) {
      uint64_t key = hs_key(seed, DOM_Q, (uint64_t)step, (uint64_t)layer,
                            (uint64_t)((unit0 + u) * heads + h));
      uint16_t* row = q + (u * heads + h) * (int64_t)dim;
      for (int32_t d = 0; d < dim; d += 4) {
        uint64_t w = sm64(key ^ (uint64_t)(d >> 2));
        for (int32_t e = d; e < d + 4 && e < dim; ++e, w >>= 16) row[e] = g_norm[w & 0xFFFF];
      }
    }
  return 0;
}

/* ---------------- selection streams ---------------- */
typedef struct {
  int64_t L;        /* records per unit (positions 0..L-1) */
  int32_t k;        /* selections per step */
  int32_t window;   /* W: records L-W..L-1 are selected every step */
  int32_t carry;    /* records kept from the previous step's non-window part */
  int32_t steps;
  int32_t kind;     /* 0: Zipf ranks through a drifting permutation; 1: Gumbel top-n */
  double zipf_s;    /* Zipf exponent over ranks (0 = uniform) */
  double drift;     /* rank offset added per step */
  uint64_t seed;
} hs_stream_params_t;

typedef struct {
  const hs_stream_params_t* p;
  const double* cdf; /* Zipf CDF over ranks, NULL for uniform / Gumbel */
  int32_t* out;
  int64_t stream0, n_streams, s_begin, s_end;
  int rc;
} sel_job_t;

static inline int bit_get(const uint64_t* b, int64_t i) { return (int)((b[i >> 6] >> (i & 63)) & 1); }
static inline void bit_set(uint64_t* b, int64_t i) { b[i >> 6] |= 1ull << (i & 63); }
static inline void bit_clr(uint64_t* b, int64_t i) { b[i >> 6] &= ~(1ull << (i & 63)); }

static int64_t zipf_rank(const double* cdf, int64_t n, double u) {
  int64_t lo = 0, hi = n - 1; /* first r with cdf[r] > u */
  while (lo < hi) {
    int64_t mid = (lo + hi) >> 1;
    if (cdf[mid] > u) hi = mid; else lo = mid + 1;
  }
  return lo;
}

static int gen_one_stream(const hs_stream_params_t* p, const double* cdf, int64_t sid,
                          int32_t* out, int64_t out_stride_step) {
  const int64_t L = p->L, H = L - p->window;
  const int32_t k = p->k, W = p->window, nsel = k - W;
  const int reject_prev = p->carry > 0;
  int64_t words = (L + 63) / 64;
  uint64_t* cur = calloc((size_t)words, 8);
  uint64_t* prev = calloc((size_t)words, 8);
  int32_t* prev_list = malloc(sizeof(int32_t) * (size_t)(nsel > 0 ? nsel : 1));
  int32_t* cur_list = malloc(sizeof(int32_t) * (size_t)(nsel > 0 ? nsel : 1));
  int32_t* set = malloc(sizeof(int32_t) * (size_t)k);
  int32_t* perm = NULL;
  float* base = NULL;
  double* score = NULL;
  int rc = 0;
  if (!cur || !prev || !prev_list || !cur_list || !set) { rc = -2; goto done; }
  if (p->kind == 0) {
    perm = malloc(sizeof(int32_t) * (size_t)H);
    if (!perm) { rc = -2; goto done; }
    for (int64_t i = 0; i < H; ++i) perm[i] = (int32_t)i;
    rng_t r = {hs_key(p->seed, DOM_PERM, (uint64_t)sid, 0, 0)};
    for (int64_t i = H - 1; i > 0; --i) { /* Fisher-Yates */
      int64_t j = (int64_t)rng_below(&r, (uint64_t)(i + 1));
      int32_t t = perm[i]; perm[i] = perm[j]; perm[j] = t;
    }
  } else {
    base = malloc(sizeof(float) * (size_t)H);
    score = malloc(sizeof(double) * (size_t)H);
    if (!base || !score) { rc = -2; goto done; }
    uint64_t h = hs_key(p->seed, DOM_BASE, (uint64_t)sid, 0, 0);
    for (int64_t j = 0; j < H; ++j) {
      uint16_t b = g_norm[sm64(h ^ (uint64_t)j) & 0xFFFF];
      uint32_t u = (uint32_t)b << 16;
      memcpy(&base[j], &u, 4);
    }
  }
  int32_t n_prev = 0;
  for (int32_t t = 0; t < p->steps; ++t) {
    rng_t r = {hs_key(p->seed, DOM_SEL, (uint64_t)sid, (uint64_t)t, 0)};
    int32_t n_cur = 0;
    /* carried subset of the previous step (uniform, partial Fisher-Yates) */
    int32_t c = (t == 0) ? 0 : p->carry;
    for (int32_t i = 0; i < c; ++i) {
      int32_t j = i + (int32_t)rng_below(&r, (uint64_t)(n_prev - i));
      int32_t tmp = prev_list[i]; prev_list[i] = prev_list[j]; prev_list[j] = tmp;
      cur_list[n_cur++] = prev_list[i];
      bit_set(cur, prev_list[i]);
    }
    int32_t fresh = nsel - c;
    if (p->kind == 0) {
      int64_t off = (int64_t)floor(p->drift * t);
      int64_t tries = 0, max_tries = 1000000 + 1000LL * fresh;
      while (fresh > 0) {
        int64_t rank = cdf ? zipf_rank(cdf, H, rng_unif(&r)) : (int64_t)rng_below(&r, (uint64_t)H);
        int64_t pos = perm[(rank + off) % H];
        if (++tries > max_tries) { rc = -3; goto done; }
        if (bit_get(cur, pos) || (reject_prev && t > 0 && bit_get(prev, pos))) continue;
        bit_set(cur, pos);
        cur_list[n_cur++] = (int32_t)pos;
        --fresh;
      }
    } else {
      /* Gumbel top-n: score_j = base_j + G_{t,j}; take the `fresh` best eligible blocks */
      uint64_t hg = hs_key(p->seed, DOM_SEL, (uint64_t)sid, (uint64_t)t, 1);
      for (int64_t j = 0; j < H; ++j) {
        double u = ((double)(sm64(hg ^ (uint64_t)j) >> 11) + 0.5) * 0x1.0p-53;
        score[j] = (double)base[j] - log(-log(u));
      }
      for (int32_t n = 0; n < fresh; ++n) {
        int64_t best = -1;
        for (int64_t j = 0; j < H; ++j) {
          if (bit_get(cur, j) || (reject_prev && t > 0 && bit_get(prev, j))) continue;
          if (best < 0 || score[j] > score[best]) best = j;
        }
        if (best < 0) { rc = -3; goto done; }
        bit_set(cur, best);
        cur_list[n_cur++] = (int32_t)best;
      }
    }
    /* emit window + non-window members in a seeded shuffled order */
    int32_t n = 0;
    for (int32_t w = 0; w < W; ++w) set[n++] = (int32_t)(H + w);
    for (int32_t i = 0; i < n_cur; ++i) set[n++] = cur_list[i];
    for (int32_t i = k - 1; i > 0; --i) {
      int32_t j = (int32_t)rng_below(&r, (uint64_t)(i + 1));
      int32_t tmp = set[i]; set[i] = set[j]; set[j] = tmp;
    }
    memcpy(out + (int64_t)t * out_stride_step, set, sizeof(int32_t) * (size_t)k);
    /* roll: prev <- cur */
    for (int32_t i = 0; i < n_prev; ++i) bit_clr(prev, prev_list[i]);
    for (int32_t i = 0; i < n_cur; ++i) { bit_clr(cur, cur_list[i]); bit_set(prev, cur_list[i]); }
    memcpy(prev_list, cur_list, sizeof(int32_t) * (size_t)n_cur);
    n_prev = n_cur;
  }
done:
  free(cur); free(prev); free(prev_list); free(cur_list); free(set);
  free(perm); free(base); free(score);
  return rc;
}

static void* sel_worker(void* arg) {
  sel_job_t* j = (sel_job_t*)arg;
  const int32_t k = j->p->k;
  for (int64_t s = j->s_begin; s < j->s_end && j->rc == 0; ++s)
    j->rc = gen_one_stream(j->p, j->cdf, j->stream0 + s, j->out + s * k, j->n_streams * k);
  return NULL;
}

/* out[step][stream][k] for streams stream0 .. stream0+n_streams-1. Returns 0, or <0 on error. */
int hs_gen_streams(const hs_stream_params_t* p, int64_t stream0, int64_t n_streams,
                   int32_t* out, int32_t nthreads) {
  if (!p || !out || p->L <= 0 || p->k <= 0 || p->window < 0 || p->window > p->k ||
      p->L - p->window < p->k - p->window || p->carry < 0 || p->carry > p->k - p->window ||
      p->steps <= 0 || p->L > 0x7FFFFFFFLL)
    return -1;
  hs_normal_table();
  const int64_t H = p->L - p->window;
  double* cdf = NULL;
  if (p->kind == 0 && p->zipf_s != 0.0) {
    cdf = malloc(sizeof(double) * (size_t)H);
    if (!cdf) return -2;
    double acc = 0.0;
    for (int64_t r = 0; r < H; ++r) { acc += pow((double)(r + 1), -p->zipf_s); cdf[r] = acc; }
    for (int64_t r = 0; r < H; ++r) cdf[r] /= acc;
    cdf[H - 1] = 2.0; /* guard: u < 1 always finds a rank */
  }
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (nthreads > n_streams) nthreads = (int32_t)(n_streams > 0 ? n_streams : 1);
  sel_job_t jobs[256];
  pthread_t th[256];
  for (int t = 0; t < nthreads; ++t)
    jobs[t] = (sel_job_t){p, cdf, out, stream0, n_streams, n_streams * t / nthreads,
                          n_streams * (t + 1) / nthreads, 0};
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, sel_worker, &jobs[t]);
  sel_worker(&jobs[0]);
  int rc = jobs[0].rc;
  for (int t = 1; t < nthreads; ++t) {
    pthread_join(th[t], NULL);
    if (jobs[t].rc) rc = jobs[t].rc;
  }
  free(cdf);
  return rc;
}
