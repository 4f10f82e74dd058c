/*
 * tre_oracle_calib.c - CPU oracle for the calibration sweep: per-request
 * latencies joined from the event stream by request id, per-window SLO
 * attainment, and the fit of each model's healthy boundary theta from the
 * smoothed TSS.
 *
 * TEST INFRASTRUCTURE ONLY, like tre_oracle.c: linked by the tests, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product
 * path, and sharing no code with the GPU library.
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE).
 *   - Section on SLOs and token-level demand: a request's SLO is stated on
 *     TTFT, TPOT and E2E latency, enforced as tail percentiles (P95 TTFT
 *     within a bound, and so on);
 *   - Section "Smoothing, Normalization, and Calibration": the profile is
 *     derived offline across the healthy-to-degraded transition, and
 *     theta_m is the smallest smoothed TSS that still achieves the target
 *     SLO reliability;
 *   - RQ1: TSS should follow the SLO-health ordering; the counts of healthy
 *     windows above and below the fitted boundary are reported for that
 *     check.
 *
 * Readings (listed in the design notes):
 *   - a request's record is joined from the events carrying its id: the
 *     first ARRIVE (arrival time, model), the first DECODE (the first output
 *     tokens are observed when that chunk completes), the first FINISH, and
 *     the sum of its DECODE tokens; events of other kinds are not used;
 *   - a request is judged only when all three events lie in the trace;
 *     requests cut off by the end of the trace are censored;
 *   - TTFT = t(first DECODE) - t(ARRIVE); E2E = t(FINISH) - t(ARRIVE);
 *     TPOT = (t(FINISH) - t(first DECODE)) / (DECODE tokens after the first
 *     DECODE event), defined only when that count is positive;
 *   - a judged request meets its model's SLO when TTFT <= ttft, E2E <= e2e
 *     and (TPOT undefined or TPOT <= tpot), compared in fp64 (a bound of
 *     +inf disables it);
 *   - a request counts in the window of its arrival (requests bucketed by
 *     arrival time, the retrospective view);
 *   - a window with at least one judged request is healthy when
 *     ok >= q * judged in fp64 (q = 0.95 means its P95 latency is within
 *     the bound);
 *   - candidate windows: at least one judged request, TSS initialised and
 *     the window not idle. theta = the smallest S_w over candidates such
 *     that, over the candidates with S >= S_w, healthy >= rho * count in
 *     fp64; +inf when no candidate qualifies;
 *   - events whose request id is >= req_cap are ignored and counted.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OC_ARRIVE 0u
#define OC_DECODE 2u
#define OC_FINISH 3u
#define OC_IDLE 1
#define OC_INIT 2
#define OC_NONE 0xFFFFFFFFu

typedef struct {
  double ttft_ms, tpot_ms, e2e_ms;  /* latency bounds (+inf: no bound) */
  double attain_q;                  /* window healthy when ok >= q * judged */
  double reliability;               /* target fraction of healthy windows above theta */
} oc_slo;

typedef struct {
  double theta;                     /* fitted boundary, +inf when none */
  uint32_t n_cand, n_healthy;       /* candidate windows, healthy among them */
  uint32_t n_above, healthy_above;  /* candidates with S >= theta, healthy among them */
  uint32_t concordant, discordant;  /* pairs of different S: the larger S healthy / unhealthy */
} oc_fit;

typedef struct {
  int64_t ttft_ms, e2e_ms;          /* valid when complete */
  double tpot_ms;                   /* valid when has_tpot */
  int32_t model;                    /* -1 when no ARRIVE */
  uint8_t complete, has_tpot, ok, pad;
} oc_req;

/*
 * Per-request join, latencies and per-window SLO attainment of one trace.
 * Events [n] sorted by ts; slo [M]; judged, ok: [M][n_windows] (zeroed
 * here); reqs [req_cap] (may be NULL). Returns the number of events whose
 * request id is >= req_cap, or -1 on bad arguments.
 */
int64_t oracle_calib_requests(int64_t window_ms, int64_t duration_ms, int32_t M, int64_t n,
                              const int64_t* ts, const uint8_t* model, const uint32_t* req,
                              const uint8_t* type, const uint16_t* tokens, const oc_slo* slo,
                              uint32_t req_cap, uint32_t* judged, uint32_t* ok, oc_req* reqs) {
  if (window_ms <= 0 || duration_ms % window_ms || M < 1 || n < 0) return -1;
  const int64_t nW = duration_ms / window_ms;
  memset(judged, 0, sizeof(uint32_t) * (size_t)(M * nW));
  memset(ok, 0, sizeof(uint32_t) * (size_t)(M * nW));
  /* first ARRIVE / DECODE / FINISH row of each request, DECODE token sum */
  uint32_t* a = malloc(sizeof(uint32_t) * (size_t)(req_cap ? req_cap : 1));
  uint32_t* f = malloc(sizeof(uint32_t) * (size_t)(req_cap ? req_cap : 1));
  uint32_t* e = malloc(sizeof(uint32_t) * (size_t)(req_cap ? req_cap : 1));
  uint64_t* d = calloc(req_cap ? req_cap : 1, sizeof(uint64_t));
  if (!a || !f || !e || !d) {
    free(a); free(f); free(e); free(d);
    return -1;
  }
  for (uint32_t r = 0; r < req_cap; ++r) a[r] = f[r] = e[r] = OC_NONE;
  int64_t bad = 0;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t r = req[i];
    if (r >= req_cap) {
      ++bad;
      continue;
    }
    const uint32_t kind = type[i] & 3u;
    if (kind == OC_ARRIVE && a[r] == OC_NONE) a[r] = (uint32_t)i;
    if (kind == OC_DECODE) {
      if (f[r] == OC_NONE) f[r] = (uint32_t)i;
      d[r] += tokens[i];
    }
    if (kind == OC_FINISH && e[r] == OC_NONE) e[r] = (uint32_t)i;
  }
  for (uint32_t r = 0; r < req_cap; ++r) {
    oc_req q = {0, 0, 0.0, -1, 0, 0, 0, 0};
    if (a[r] != OC_NONE) q.model = model[a[r]];
    if (a[r] != OC_NONE && f[r] != OC_NONE && e[r] != OC_NONE && q.model < M) {
      const int m = q.model;
      q.complete = 1;
      q.ttft_ms = ts[f[r]] - ts[a[r]];
      q.e2e_ms = ts[e[r]] - ts[a[r]];
      const uint64_t after_first = d[r] - tokens[f[r]];
      int good = (double)q.ttft_ms <= slo[m].ttft_ms && (double)q.e2e_ms <= slo[m].e2e_ms;
      if (after_first > 0) {
        q.has_tpot = 1;
        q.tpot_ms = (double)(ts[e[r]] - ts[f[r]]) / (double)after_first;
        good = good && q.tpot_ms <= slo[m].tpot_ms;
      }
      q.ok = (uint8_t)good;
      const int64_t w = ts[a[r]] / window_ms;  /* window of arrival */
      if (w >= 0 && w < nW) {
        judged[m * nW + w] += 1;
        ok[m * nW + w] += (uint32_t)good;
      }
    }
    if (reqs) reqs[r] = q;
  }
  free(a); free(f); free(e); free(d);
  return bad;
}

typedef struct {
  double s;
  int healthy;
} oc_cand;

static int by_s_descending(const void* x, const void* y) {
  const double a = ((const oc_cand*)x)->s, b = ((const oc_cand*)y)->s;
  return a > b ? -1 : (a < b ? 1 : 0);
}

/*
 * Fit of theta for each model of one trace from the smoothed TSS S and the
 * flags ([n_windows][M]) and the per-window counts ([M][n_windows]).
 * Returns 0, or -1 on bad arguments.
 */
int oracle_calib_fit(int64_t n_windows, int32_t M, const double* S, const uint8_t* flags,
                     const uint32_t* judged, const uint32_t* ok, const oc_slo* slo, oc_fit* fit) {
  if (n_windows < 0 || M < 1) return -1;
  oc_cand* c = malloc(sizeof(oc_cand) * (size_t)(n_windows ? n_windows : 1));
  if (!c) return -1;
  for (int m = 0; m < M; ++m) {
    int64_t k = 0;
    uint32_t n_healthy = 0;
    for (int64_t w = 0; w < n_windows; ++w) {
      const uint8_t fl = flags[w * M + m];
      const uint32_t j = judged[m * n_windows + w];
      if (j == 0 || !(fl & OC_INIT) || (fl & OC_IDLE)) continue;
      c[k].s = S[w * M + m];
      c[k].healthy = (double)ok[m * n_windows + w] >= slo[m].attain_q * (double)j;
      n_healthy += (uint32_t)c[k].healthy;
      ++k;
    }
    qsort(c, (size_t)k, sizeof(oc_cand), by_s_descending);
    /* walk from the largest S down; a threshold s covers every candidate
       with S >= s, so it is evaluated after the last of a run of equal S.
       The ordering check (RQ1: TSS should follow the SLO-health ordering):
       every window already passed has a larger S than the run, so each
       unhealthy window of the run pairs concordantly with the healthy ones
       passed, and each healthy window discordantly with the unhealthy ones
       passed; windows of equal S do not pair. */
    oc_fit best = {INFINITY, (uint32_t)k, n_healthy, 0, 0, 0, 0};
    uint32_t N = 0, H = 0;
    for (int64_t i = 0; i < k;) {
      int64_t j = i;
      uint32_t run_h = 0, run_n = 0;
      while (j < k && c[j].s == c[i].s) {
        run_n += 1;
        run_h += (uint32_t)c[j].healthy;
        ++j;
      }
      best.concordant += (run_n - run_h) * H;
      best.discordant += run_h * (N - H);
      N += run_n;
      H += run_h;
      if ((double)H >= slo[m].reliability * (double)N) {
        best.theta = c[i].s;  /* smaller than any earlier qualifying value */
        best.n_above = N;
        best.healthy_above = H;
      }
      i = j;
    }
    fit[m] = best;
  }
  free(c);
  return 0;
}
