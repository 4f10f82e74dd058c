/*
 * tracegen.c - seeded synthetic multi-model request-event traces.
 *
 * This module only produces INPUTS: it holds none of the token-service-share
 * arithmetic and none of the rebalancing rules. Both the CPU oracle and the
 * GPU library consume the columns written here.
 *
 * Model of a trace (open loop: the trace does not react to any replay
 * decision):
 *   - per model, requests arrive by one of four processes (Poisson, a
 *     two-state Markov-modulated Poisson process, a diurnal sinusoid driving
 *     a gamma renewal process in rescaled time, Poisson with synchronized
 *     flash crowds);
 *   - prompt and output lengths are rounded, clipped lognormals;
 *   - each model is an FCFS queue with `slots` concurrent serving slots, each
 *     slot serving `slot_rate` prefill-weighted tokens per second;
 *   - every request emits ARRIVE, one PREFILL per prompt chunk (the first
 *     one carries the ADMIT bit and is emitted at service start), one DECODE
 *     per decode chunk (at chunk completion) and FINISH at the last decode.
 *
 * Event columns (structure of arrays):
 *   ts      int64   milliseconds from trace start, [0, duration_ms)
 *   model   uint8   model index
 *   req     uint32  request id, unique within a trace
 *   type    uint8   bits 0-1 kind (0 ARRIVE, 1 PREFILL, 2 DECODE, 3 FINISH),
 *                   bit 7 ADMIT (only on the first PREFILL of a request)
 *   tokens  uint16  ARRIVE: prompt length; PREFILL/DECODE: tokens in the
 *                   chunk; FINISH: 0
 * Within a trace events are sorted by ts; equal timestamps keep generation
 * order (model, request, lifecycle order), so a request's own events always
 * appear in lifecycle order.
 *
 * Randomness: xoshiro256** streams seeded through splitmix64 from
 * (seed, trace, model, stream id), so a trace's events do not depend on the
 * batch it was generated in or on the number of threads.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define TG_POISSON 0
#define TG_MMPP2 1
#define TG_DIURNAL_GAMMA 2
#define TG_FLASH 3

#define K_ARRIVE 0u
#define K_PREFILL 1u
#define K_DECODE 2u
#define K_FINISH 3u
#define F_ADMIT 0x80u

typedef struct {
  int32_t n_models;
  int32_t process;
  int64_t duration_ms;
  uint64_t seed;
  const double* rate;       /* [n_models] base arrival rate, requests/s   */
  const double* slot_rate;  /* [n_models] prefill-weighted tokens/s/slot  */
  const int32_t* slots;     /* [n_models] concurrent FCFS serving slots    */
  const double* prompt_mu;  /* [n_models] lognormal parameters            */
  const double* prompt_sigma;
  const double* out_mu;
  const double* out_sigma;
  int32_t prompt_min, prompt_max, out_min, out_max;
  double prefill_weight;    /* service cost of one prompt token vs decode */
  int32_t prefill_chunk, decode_chunk;
  double mmpp_mult, mmpp_dwell_s;
  double diurnal_amp, diurnal_period_s, gamma_shape;
  double flash_mult, flash_len_s, flash_first_s, flash_every_s;
  int32_t flash_models;
} tg_config;

/* ------------------------------------------------------------------ RNG */
typedef struct { uint64_t s[4]; int has_spare; double spare; } rng_t;

static uint64_t splitmix64(uint64_t* x) {
  uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static void rng_seed(rng_t* r, uint64_t seed, uint64_t a, uint64_t b, uint64_t c) {
  uint64_t x = seed ^ (a * 0xD1B54A32D192ED03ull) ^ (b * 0xABC98388FB8FAC03ull) ^
               (c * 0x8CB92BA72F3D8DD7ull);
  for (int i = 0; i < 4; ++i) r->s[i] = splitmix64(&x);
  r->has_spare = 0;
}
static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }
static inline uint64_t rng_next(rng_t* r) {
  uint64_t* s = r->s;
  uint64_t res = rotl(s[1] * 5, 7) * 9, t = s[1] << 17;
  s[2] ^= s[0]; s[3] ^= s[1]; s[1] ^= s[2]; s[0] ^= s[3]; s[2] ^= t; s[3] = rotl(s[3], 45);
  return res;
}
/* uniform in (0, 1), never 0 or 1 */
static inline double rng_u01(rng_t* r) {
  return ((double)(rng_next(r) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}
static inline double rng_exp(rng_t* r, double rate) { return -log(rng_u01(r)) / rate; }
static double rng_normal(rng_t* r) {
  if (r->has_spare) { r->has_spare = 0; return r->spare; }
  double u1 = rng_u01(r), u2 = rng_u01(r);
  double rad = sqrt(-2.0 * log(u1)), th = 6.283185307179586 * u2;
  r->spare = rad * sin(th); r->has_spare = 1;
  return rad * cos(th);
}
/* Marsaglia-Tsang gamma(shape, 1); shape < 1 by the u^(1/shape) boost */
static double rng_gamma(rng_t* r, double shape) {
  if (shape < 1.0) return rng_gamma(r, shape + 1.0) * pow(rng_u01(r), 1.0 / shape);
  double d = shape - 1.0 / 3.0, c = 1.0 / sqrt(9.0 * d);
  for (;;) {
    double x = rng_normal(r), v = 1.0 + c * x;
    if (v <= 0.0) continue;
    v = v * v * v;
    double u = rng_u01(r);
    if (log(u) < 0.5 * x * x + d - d * v + d * log(v)) return d * v;
  }
}

/* --------------------------------------------------------------- buffers */
typedef struct { double* v; size_t n, cap; } dvec;
static int dvec_push(dvec* a, double x) {
  if (a->n == a->cap) {
    size_t nc = a->cap ? a->cap * 2 : 1024;
    double* p = (double*)realloc(a->v, nc * sizeof(double));
    if (!p) return -1;
    a->v = p; a->cap = nc;
  }
  a->v[a->n++] = x;
  return 0;
}

typedef struct {
  uint32_t ts;
  uint32_t req;
  uint16_t tokens;
  uint8_t model;
  uint8_t type;
} rec_t;
typedef struct { rec_t* v; size_t n, cap; } rvec;
static int rvec_push(rvec* a, uint32_t ts, uint32_t req, uint32_t tokens, uint32_t model,
                     uint32_t type) {
  if (a->n == a->cap) {
    size_t nc = a->cap ? a->cap * 2 : 4096;
    rec_t* p = (rec_t*)realloc(a->v, nc * sizeof(rec_t));
    if (!p) return -1;
    a->v = p; a->cap = nc;
  }
  rec_t* e = &a->v[a->n++];
  e->ts = ts; e->req = req; e->tokens = (uint16_t)tokens; e->model = (uint8_t)model;
  e->type = (uint8_t)type;
  return 0;
}

/* ------------------------------------------------------ arrival processes */
static int arrivals_poisson_piecewise(rng_t* r, double T, double base, const double* bnd,
                                      const double* mult, int nseg, dvec* out) {
  /* piecewise-constant rate: segment i is [bnd[i], bnd[i+1]) with rate
     base*mult[i]; the exponential clock restarts at every boundary, which is
     exact for a Poisson process */
  for (int i = 0; i < nseg; ++i) {
    double lo = bnd[i], hi = bnd[i + 1] < T ? bnd[i + 1] : T, rate = base * mult[i];
    if (lo >= T) break;
    if (rate <= 0.0) continue;
    double t = lo;
    for (;;) {
      t += rng_exp(r, rate);
      if (t >= hi) break;
      if (dvec_push(out, t)) return -1;
    }
  }
  return 0;
}

static int arrivals_mmpp2(rng_t* r, double T, double base, double hi_mult, double dwell,
                          dvec* out) {
  double t = 0.0, end = rng_exp(r, 1.0 / dwell);
  int state = 0;
  while (t < T) {
    double rate = state ? base * hi_mult : base;
    double gap = rng_exp(r, rate);
    if (t + gap < end) {
      t += gap;
      if (t < T && dvec_push(out, t)) return -1;
    } else {
      t = end;
      state ^= 1;
      end = t + rng_exp(r, 1.0 / dwell);
    }
  }
  return 0;
}

/* integrated intensity of lambda(t) = lb*(1 + a*sin(2*pi*t/P + phi)) */
static double diurnal_Lambda(double t, double lb, double a, double P, double phi) {
  const double w = 6.283185307179586 / P;
  return lb * (t - (a / w) * (cos(w * t + phi) - cos(phi)));
}

static int arrivals_diurnal_gamma(rng_t* r, double T, double lb, double a, double P,
                                  double shape, double phi, dvec* out) {
  /* unit-rate gamma renewal process in operational time tau, mapped back
     through the inverse of the integrated intensity */
  const double w = 6.283185307179586 / P;
  double tau = 0.0, t = 0.0;
  for (;;) {
    double g = rng_gamma(r, shape) / shape; /* mean 1, CV^2 = 1/shape */
    tau += g;
    /* bracket: Lambda grows at least lb*(1-a) and at most lb*(1+a) per second */
    double lo = t, hi = t + g / (lb * (1.0 - a)) + 1e-9;
    double x = t + g / lb;
    if (x < lo || x > hi) x = 0.5 * (lo + hi);
    for (int it = 0; it < 100; ++it) {
      double f = diurnal_Lambda(x, lb, a, P, phi) - tau;
      if (f > 0) hi = x; else lo = x;
      double d = lb * (1.0 + a * sin(w * x + phi));
      double xn = x - f / d;
      if (!(xn > lo && xn < hi)) xn = 0.5 * (lo + hi);
      if (fabs(xn - x) < 1e-10) { x = xn; break; }
      x = xn;
    }
    t = x;
    if (t >= T) break;
    if (dvec_push(out, t)) return -1;
  }
  return 0;
}

/* ---------------------------------------------------------- FCFS service */
static void heap_sift_down(double* h, int n, int i) {
  for (;;) {
    int l = 2 * i + 1, m = i;
    if (l < n && h[l] < h[m]) m = l;
    if (l + 1 < n && h[l + 1] < h[m]) m = l + 1;
    if (m == i) return;
    double t = h[i]; h[i] = h[m]; h[m] = t; i = m;
  }
}

static inline int64_t to_ms(double t_s) { return (int64_t)floor(t_s * 1000.0); }

static int clip_len(double x, int lo, int hi) {
  double v = floor(x + 0.5);
  if (v < lo) return lo;
  if (v > hi) return hi;
  return (int)v;
}

static int serve_model(const tg_config* c, int m, uint64_t trace, const dvec* arr, rvec* out) {
  const int64_t dur = c->duration_ms;
  const double rate = c->slot_rate[m];
  const int S = c->slots[m] > 0 ? c->slots[m] : 1;
  double* heap = (double*)calloc((size_t)S, sizeof(double));
  if (!heap) return -1;
  rng_t lr;
  rng_seed(&lr, c->seed, trace + 1, (uint64_t)m + 1, 2);
  const uint32_t M = (uint32_t)c->n_models;
  int rc = 0;
  for (size_t i = 0; i < arr->n && rc == 0; ++i) {
    double a = arr->v[i];
    int prompt = clip_len(exp(c->prompt_mu[m] + c->prompt_sigma[m] * rng_normal(&lr)),
                          c->prompt_min, c->prompt_max);
    int output = clip_len(exp(c->out_mu[m] + c->out_sigma[m] * rng_normal(&lr)),
                          c->out_min, c->out_max);
    uint32_t req = (uint32_t)(i * M + (uint32_t)m);
    int64_t ta = to_ms(a);
    if (ta >= dur) continue;
    rc |= rvec_push(out, (uint32_t)ta, req, (uint32_t)prompt, (uint32_t)m, K_ARRIVE);
    double start = a > heap[0] ? a : heap[0];
    double t = start;
    int left = prompt, first = 1;
    while (left > 0) {
      int ch = left < c->prefill_chunk ? left : c->prefill_chunk;
      int64_t ms = to_ms(t);
      if (ms < dur)
        rc |= rvec_push(out, (uint32_t)ms, req, (uint32_t)ch, (uint32_t)m,
                        K_PREFILL | (first ? F_ADMIT : 0u));
      first = 0;
      t += c->prefill_weight * (double)ch / rate;
      left -= ch;
    }
    left = output;
    int64_t last_ms = to_ms(t);
    while (left > 0) {
      int ch = left < c->decode_chunk ? left : c->decode_chunk;
      t += (double)ch / rate;
      last_ms = to_ms(t);
      if (last_ms < dur) rc |= rvec_push(out, (uint32_t)last_ms, req, (uint32_t)ch, (uint32_t)m, K_DECODE);
      left -= ch;
    }
    if (last_ms < dur) rc |= rvec_push(out, (uint32_t)last_ms, req, 0u, (uint32_t)m, K_FINISH);
    heap[0] = t;
    heap_sift_down(heap, S, 0);
  }
  free(heap);
  return rc;
}

/* stable LSD radix sort of records by ts (8-bit digits); tmp has room for n */
static void sort_by_ts(rvec* v, rec_t* tmp) {
  size_t n = v->n;
  if (n < 2) return;
  uint32_t mx = 0;
  for (size_t i = 0; i < n; ++i) if (v->v[i].ts > mx) mx = v->v[i].ts;
  rec_t *src = v->v, *dst = tmp;
  size_t cnt[256];
  for (int shift = 0; shift < 32 && (mx >> shift) != 0; shift += 8) {
    memset(cnt, 0, sizeof cnt);
    for (size_t i = 0; i < n; ++i) cnt[(src[i].ts >> shift) & 255u]++;
    size_t sum = 0;
    for (int d = 0; d < 256; ++d) { size_t k = cnt[d]; cnt[d] = sum; sum += k; }
    for (size_t i = 0; i < n; ++i) dst[cnt[(src[i].ts >> shift) & 255u]++] = src[i];
    rec_t* t = src; src = dst; dst = t;
  }
  if (src != v->v) memcpy(v->v, src, n * sizeof(rec_t));
}

/* request table of one model instead of its served events: the same length
   draws as serve_model, in the same order, without the FCFS service */
typedef struct {
  uint32_t ts, req;
  uint16_t prompt, output;
  uint8_t model;
} qrec_t;
typedef struct { qrec_t* v; size_t n, cap; } qvec;

static int list_requests(const tg_config* c, int m, uint64_t trace, const dvec* arr, qvec* out) {
  const int64_t dur = c->duration_ms;
  rng_t lr;
  rng_seed(&lr, c->seed, trace + 1, (uint64_t)m + 1, 2);
  const uint32_t M = (uint32_t)c->n_models;
  for (size_t i = 0; i < arr->n; ++i) {
    int prompt = clip_len(exp(c->prompt_mu[m] + c->prompt_sigma[m] * rng_normal(&lr)),
                          c->prompt_min, c->prompt_max);
    int output = clip_len(exp(c->out_mu[m] + c->out_sigma[m] * rng_normal(&lr)),
                          c->out_min, c->out_max);
    int64_t ta = to_ms(arr->v[i]);
    if (ta >= dur) continue;
    if (out->n == out->cap) {
      size_t nc = out->cap ? out->cap * 2 : 4096;
      qrec_t* p = (qrec_t*)realloc(out->v, nc * sizeof(qrec_t));
      if (!p) return -1;
      out->v = p; out->cap = nc;
    }
    qrec_t* q = &out->v[out->n++];
    q->ts = (uint32_t)ta; q->req = (uint32_t)(i * M + (uint32_t)m);
    q->prompt = (uint16_t)prompt; q->output = (uint16_t)output; q->model = (uint8_t)m;
  }
  return 0;
}

static int gen_trace_into(const tg_config* c, uint64_t trace, rvec* out, qvec* reqs);

static int gen_trace(const tg_config* c, uint64_t trace, rvec* out) { return gen_trace_into(c, trace, out, 0); }

/* events of one trace (reqs == NULL), or its request table (out unused) */
static int gen_trace_into(const tg_config* c, uint64_t trace, rvec* out, qvec* reqs) {
  const double T = (double)c->duration_ms / 1000.0;
  const int M = c->n_models;
  dvec arr = {0, 0, 0};
  int rc = 0;
  /* flash crowds: which models of this trace spike (partial Fisher-Yates) */
  int spiked[256];
  memset(spiked, 0, sizeof spiked);
  if (c->process == TG_FLASH) {
    rng_t fr;
    rng_seed(&fr, c->seed, trace + 1, 0, 3);
    int idx[256];
    for (int i = 0; i < M; ++i) idx[i] = i;
    int k = c->flash_models < M ? c->flash_models : M;
    for (int i = 0; i < k; ++i) {
      int j = i + (int)(rng_u01(&fr) * (double)(M - i));
      if (j >= M) j = M - 1;
      int t = idx[i]; idx[i] = idx[j]; idx[j] = t;
      spiked[idx[i]] = 1;
    }
  }
  for (int m = 0; m < M && rc == 0; ++m) {
    rng_t ar;
    rng_seed(&ar, c->seed, trace + 1, (uint64_t)m + 1, 1);
    arr.n = 0;
    if (!(c->rate[m] > 0.0)) continue; /* a model with no traffic */
    switch (c->process) {
      case TG_POISSON: {
        double b[2] = {0.0, T}, mu[1] = {1.0};
        rc = arrivals_poisson_piecewise(&ar, T, c->rate[m], b, mu, 1, &arr);
        break;
      }
      case TG_MMPP2:
        rc = arrivals_mmpp2(&ar, T, c->rate[m], c->mmpp_mult, c->mmpp_dwell_s, &arr);
        break;
      case TG_DIURNAL_GAMMA: {
        double phi = 6.283185307179586 * rng_u01(&ar);
        rc = arrivals_diurnal_gamma(&ar, T, c->rate[m], c->diurnal_amp, c->diurnal_period_s,
                                    c->gamma_shape, phi, &arr);
        break;
      }
      case TG_FLASH: {
        /* segment boundaries: spike k covers [first + k*every, +len) */
        int nmax = 2 + 2 * (int)(T / (c->flash_every_s > 0 ? c->flash_every_s : T) + 2);
        double* b = (double*)malloc(sizeof(double) * (size_t)(nmax + 1));
        double* mu = (double*)malloc(sizeof(double) * (size_t)nmax);
        if (!b || !mu) { free(b); free(mu); rc = -1; break; }
        int ns = 0;
        double t = 0.0;
        if (spiked[m] && c->flash_every_s > 0) {
          for (double s = c->flash_first_s; s < T && ns + 2 < nmax; s += c->flash_every_s) {
            b[ns] = t; mu[ns] = 1.0; ++ns;
            b[ns] = s; mu[ns] = c->flash_mult; ++ns;
            t = s + c->flash_len_s;
          }
        }
        b[ns] = t; mu[ns] = 1.0; ++ns;
        b[ns] = T > t ? T : t;
        rc = arrivals_poisson_piecewise(&ar, T, c->rate[m], b, mu, ns, &arr);
        free(b); free(mu);
        break;
      }
      default: rc = -2;
    }
    if (rc == 0) rc = reqs ? list_requests(c, m, trace, &arr, reqs) : serve_model(c, m, trace, &arr, out);
  }
  free(arr.v);
  return rc;
}

/* ------------------------------------------------------------ batch API */
typedef struct {
  const tg_config* cfg;
  uint64_t t0, t1;
  int64_t* counts;            /* pass 1 output, or NULL */
  const int64_t* off;         /* pass 2: element offset of each trace */
  int64_t* ts; uint8_t* model; uint32_t* req; uint8_t* type; uint16_t* tokens;
  int err;
  uint64_t next;
  pthread_mutex_t mu;
} job_t;

static void* worker(void* p) {
  job_t* j = (job_t*)p;
  rvec buf = {0, 0, 0};
  rec_t* tmp = 0;
  size_t tmp_cap = 0;
  for (;;) {
    pthread_mutex_lock(&j->mu);
    uint64_t t = j->next++;
    pthread_mutex_unlock(&j->mu);
    if (t >= j->t1 - j->t0) break;
    buf.n = 0;
    int rc = gen_trace(j->cfg, j->t0 + t, &buf);
    if (rc == 0 && j->counts) j->counts[t] = (int64_t)buf.n;
    if (rc == 0 && j->off) {
      if (j->counts == 0 && (int64_t)buf.n != j->off[t + 1] - j->off[t]) rc = -3;
      if (rc == 0 && tmp_cap < buf.n) {
        free(tmp);
        tmp_cap = buf.cap;
        tmp = (rec_t*)malloc(tmp_cap * sizeof(rec_t));
        if (!tmp) { tmp_cap = 0; rc = -1; }
      }
      if (rc == 0) {
        sort_by_ts(&buf, tmp);
        int64_t o = j->off[t];
        for (size_t i = 0; i < buf.n; ++i) {
          const rec_t* x = &buf.v[i];
          if (j->ts) j->ts[o + (int64_t)i] = (int64_t)x->ts;
          if (j->model) j->model[o + (int64_t)i] = x->model;
          if (j->req) j->req[o + (int64_t)i] = x->req;
          if (j->type) j->type[o + (int64_t)i] = x->type;
          if (j->tokens) j->tokens[o + (int64_t)i] = x->tokens;
        }
      }
    }
    if (rc) {
      pthread_mutex_lock(&j->mu);
      j->err = rc;
      pthread_mutex_unlock(&j->mu);
    }
  }
  free(buf.v);
  free(tmp);
  return 0;
}

static int run_job(job_t* j, int n_threads) {
  if (n_threads < 1) n_threads = 1;
  if (n_threads > 256) n_threads = 256;
  if ((uint64_t)n_threads > j->t1 - j->t0) n_threads = (int)(j->t1 - j->t0 ? j->t1 - j->t0 : 1);
  pthread_mutex_init(&j->mu, 0);
  pthread_t th[256];
  for (int i = 0; i < n_threads; ++i) pthread_create(&th[i], 0, worker, j);
  for (int i = 0; i < n_threads; ++i) pthread_join(th[i], 0);
  pthread_mutex_destroy(&j->mu);
  return j->err;
}

/* Pass 1: number of events of each trace in [t0, t1). Returns 0 on success. */
int tg_count(const tg_config* cfg, uint64_t t0, uint64_t t1, int n_threads, int64_t* counts) {
  if (!cfg || !counts || t1 < t0 || cfg->n_models < 1 || cfg->n_models > 256) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.cfg = cfg; j.t0 = t0; j.t1 = t1; j.counts = counts;
  return run_job(&j, n_threads);
}

/* Pass 2: write trace t0+i at element offset off[i] of every non-NULL column;
   off has t1-t0+1 entries and must come from tg_count's counts (a mismatch
   returns -3). */
int tg_fill(const tg_config* cfg, uint64_t t0, uint64_t t1, int n_threads, const int64_t* off,
            int64_t* ts, uint8_t* model, uint32_t* req, uint8_t* type, uint16_t* tokens) {
  if (!cfg || !off || t1 < t0 || cfg->n_models < 1 || cfg->n_models > 256) return -1;
  job_t j;
  memset(&j, 0, sizeof j);
  j.cfg = cfg; j.t0 = t0; j.t1 = t1; j.off = off;
  j.ts = ts; j.model = model; j.req = req; j.type = type; j.tokens = tokens;
  return run_job(&j, n_threads);
}

/* Request table of one trace: per request its arrival (ms), model, id,
   prompt and output lengths, model by model, arrivals in order within a
   model (the draws of tg_fill, without the fixed-capacity service). With
   cap too small, returns -5 and sets *n to the count needed. */
int tg_requests(const tg_config* cfg, uint64_t trace, int64_t cap, int64_t* n, int64_t* arrival_ms,
                uint8_t* model, uint32_t* req, uint16_t* prompt, uint16_t* output) {
  if (!cfg || !n || cfg->n_models < 1 || cfg->n_models > 256) return -1;
  qvec q = {0, 0, 0};
  int rc = gen_trace_into(cfg, trace, 0, &q);
  if (rc == 0) {
    *n = (int64_t)q.n;
    if ((int64_t)q.n > cap) {
      rc = -5;
    } else {
      for (size_t i = 0; i < q.n; ++i) {
        arrival_ms[i] = q.v[i].ts; model[i] = q.v[i].model; req[i] = q.v[i].req;
        prompt[i] = q.v[i].prompt; output[i] = q.v[i].output;
      }
    }
  }
  free(q.v);
  return rc;
}
