/*
 * tre_oracle.c - CPU oracle for Token Service Share (TSS) evaluation and
 * TSS-guided receiver/donor rebalancing.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, single-threaded
 * statement of what the replay computes; it is linked only by the tests, by
 * the smoke check and by the benchmark's CPU-baseline leg. The product path
 * never calls it. It shares no code, header or constant with the GPU library.
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE).
 *   Eq. (1)  raw TSS = (w_p * r_prefill + r_decode) / (A + w_q * W)
 *            (Section "Token Service Share", "Design Rationale and Definition")
 *   smoothing with alpha, Eq. (2) Z = TSS / theta, regions tau_crit < 1 <
 *            tau_surplus (Section "Smoothing, Normalization, and Calibration")
 *   rescue / rebalancing, Eq. (3) receiver = argmin Z, donor preference
 *            (Section "Dual-Speed Control")
 *   bounded transfer: receiver below its healthy boundary, donor above its
 *            replica floor, fixed budget (Section "Bounded Pairwise Transfer")
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   - A_m and W_m are the time averages of the active / waiting request
 *     counts over the window (the paper motivates TSS with an "average"
 *     waiting queue); rates are tokens per second;
 *   - the denominator has a floor of one request (the paper's "signal
 *     floor" under which a raw inverse reads 1.0);
 *   - an idle window (no tokens, nothing active or waiting) holds the
 *     smoothed value and reads Z = +inf; the first non-idle window
 *     initialises the smoothed value to the raw ratio;
 *   - the smoothed value is S = alpha * raw + (1 - alpha) * S_prev;
 *   - ties in argmin / argmax go to the lowest model index;
 *   - up to K (scenario "max moves") greedy transfers per tick, each model in
 *     at most one transfer per tick; idle budget is used before any donor.
 *
 * Floating point: IEEE binary64, round to nearest even, no contraction
 * (build with -ffp-contract=off), in exactly the operation order written
 * below. Integer tallies are exact.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* event type byte: bits 0-1 kind, bit 7 admit */
#define OR_ARRIVE 0
#define OR_PREFILL 1
#define OR_DECODE 2
#define OR_FINISH 3
#define OR_ADMIT 0x80

#define OR_RESCUE 1
#define OR_REBALANCE 2
#define OR_POOL 0xFF

#define OR_IDLE 1
#define OR_INIT 2

#define OR_MAX_MODELS 256

/* Per-model control profile: the paper's six scalars per model-SLO pair
   (w_p, w_q, alpha, theta, tau_crit, tau_surplus) plus the minimum routable
   replica floor and the initial routable replica count. 56 bytes. */
typedef struct {
  double w_p, w_q, alpha, theta, tau_crit, tau_surplus;
  int32_t r_min, r_init;
} or_profile;

/* One what-if scenario over one trace. 24 bytes. */
typedef struct {
  uint32_t trace;
  uint32_t max_moves;          /* K: transfers allowed per tick            */
  double theta_scale;          /* healthy boundary used = theta * scale    */
  double tau_crit_override;    /* >= 0 replaces every profile's tau_crit   */
} or_scenario;

/* One capacity transition. 8 bytes. */
typedef struct {
  uint32_t window;             /* window at whose end the tick fired        */
  uint8_t path;                /* OR_RESCUE or OR_REBALANCE                 */
  uint8_t receiver;
  uint8_t donor;               /* OR_POOL: idle budget                      */
  uint8_t pad;
} or_move;

/* ----------------------------------------------------------------------
 * Eq. (1) for one model and one window, from the window's observations:
 *   P, D   prefill / decode tokens served in the window;
 *   A_int  integral of the active-request count over the window (req * ms);
 *   W_int  integral of the waiting-request count over the window (req * ms).
 * With Delta_s = window_ms / 1000, r = tokens / Delta_s,
 * A = A_int / window_ms, W = W_int / window_ms and a floor of one request:
 *   raw = (w_p*P/Delta_s + D/Delta_s) / max(A + w_q*W, 1)
 *       = 1000 * (w_p*P + D) / max(A_int + w_q*W_int, window_ms).
 * The second (algebraically equal) form is the one evaluated.
 * -------------------------------------------------------------------- */
double oracle_raw_tss(double w_p, double w_q, int64_t P, int64_t D, int64_t A_int,
                      int64_t W_int, int64_t window_ms) {
  double num = w_p * (double)P;
  num = num + (double)D;
  num = num * 1000.0;
  double q = w_q * (double)W_int;
  double den = (double)A_int + q;
  if (den < (double)window_ms) den = (double)window_ms;
  return num / den;
}

/* Exponential smoothing: the new smoothed value combines the window's raw
   ratio (weight alpha) with the previous smoothed value (weight 1 - alpha). */
double oracle_smooth(double alpha, double raw, double s_prev) {
  double t1 = alpha * raw;
  double t2 = (1.0 - alpha) * s_prev;
  return t1 + t2;
}

/* add the integral of a constant count over [from, to) to per-window sums,
   splitting at window boundaries */
static void integrate(int64_t* integ, int32_t M, int32_t m, int64_t window_ms, int64_t count,
                      int64_t from, int64_t to) {
  const int64_t n_w = (to + window_ms - 1) / window_ms;  /* to <= duration: rows [0, n_w) exist */
  while (from < to) {
    int64_t w = from / window_ms;
    int64_t seg_end = (w + 1) * window_ms;
    if (seg_end > to) seg_end = to;
    if (w < 0 || w >= n_w || seg_end <= from) break; /* never for valid input; keeps writes inside the rows */
    integ[w * M + m] += count * (seg_end - from);
    from = seg_end;
  }
}

/* ----------------------------------------------------------------------
 * Window observations and smoothed TSS for one trace.
 * Events must be sorted by ts within the trace, 0 <= ts < duration_ms.
 * Outputs are [n_windows][n_models], n_windows = duration_ms / window_ms.
 * Returns 0, or a negative code for invalid input:
 *   -2  timestamp unsorted or outside [0, duration_ms)
 *   -3  model index >= M or undefined type bits
 *   -5  A_m(t) or W_m(t) negative at some instant t.
 * The last code follows from the definition of Eq. (1) (Section "Design
 * Rationale and Definition"): A_m(t) and W_m(t) are the numbers of active and
 * of waiting requests of model m at time t, so neither can be negative. They
 * are the right-continuous step functions of the transitions, so the value
 * at t counts every event with ts <= t: the order of the rows that share one
 * timestamp does not matter, only the counts after the last of them.
 * The first two kinds are checked over the whole trace before the third.
 * -------------------------------------------------------------------- */
int oracle_tss_trace(const int64_t* ts, const uint8_t* model, const uint8_t* type,
                     const uint16_t* tokens, int64_t n_events, int64_t window_ms,
                     int64_t duration_ms, int32_t M, const or_profile* prof, int64_t* P,
                     int64_t* D, int64_t* A_int, int64_t* W_int, double* S, uint8_t* flags) {
  if (window_ms <= 0 || duration_ms <= 0 || duration_ms % window_ms || M < 1 ||
      M > OR_MAX_MODELS)
    return -1;
  const int64_t nW = duration_ms / window_ms;
  memset(P, 0, sizeof(int64_t) * (size_t)(nW * M));
  memset(D, 0, sizeof(int64_t) * (size_t)(nW * M));
  memset(A_int, 0, sizeof(int64_t) * (size_t)(nW * M));
  memset(W_int, 0, sizeof(int64_t) * (size_t)(nW * M));

  /* order and schema of every row first */
  for (int64_t i = 0; i < n_events; ++i) {
    if (ts[i] < 0 || ts[i] >= duration_ms || (i > 0 && ts[i] < ts[i - 1])) return -2;
    const int admit = (type[i] & OR_ADMIT) != 0;
    if (model[i] >= M || (type[i] & 0x7C) || (admit && (type[i] & 3) != OR_PREFILL)) return -3;
  }

  /* A_m(t), W_m(t): right-continuous step functions starting at 0 */
  int64_t A[OR_MAX_MODELS], W[OR_MAX_MODELS], t_last[OR_MAX_MODELS];
  for (int m = 0; m < M; ++m) { A[m] = 0; W[m] = 0; t_last[m] = 0; }

  for (int64_t i = 0; i < n_events; ++i) {
    const int64_t t = ts[i];
    const int m = model[i];
    const int kind = type[i] & 3;
    const int admit = (type[i] & OR_ADMIT) != 0;
    /* the counts held on [t_last, t) */
    integrate(A_int, M, m, window_ms, A[m], t_last[m], t);
    integrate(W_int, M, m, window_ms, W[m], t_last[m], t);
    t_last[m] = t;
    const int64_t w = t / window_ms;
    switch (kind) {
      case OR_ARRIVE: W[m] += 1; break;               /* joins the front-door queue */
      case OR_PREFILL:
        P[w * M + m] += tokens[i];
        if (admit) { W[m] -= 1; A[m] += 1; }          /* admitted: waiting -> active */
        break;
      case OR_DECODE: D[w * M + m] += tokens[i]; break;
      case OR_FINISH: A[m] -= 1; break;               /* leaves the active set */
    }
    /* after the last row at this instant every count is the value of its
       step function there */
    if (i == n_events - 1 || ts[i + 1] != t)
      for (int k = 0; k < M; ++k)
        if (A[k] < 0 || W[k] < 0) return -5;
  }
  for (int m = 0; m < M; ++m) {
    integrate(A_int, M, m, window_ms, A[m], t_last[m], duration_ms);
    integrate(W_int, M, m, window_ms, W[m], t_last[m], duration_ms);
  }

  for (int m = 0; m < M; ++m) {
    double s = 0.0;
    int init = 0;
    for (int64_t w = 0; w < nW; ++w) {
      const int64_t c = w * M + m;
      const int idle = P[c] == 0 && D[c] == 0 && A_int[c] == 0 && W_int[c] == 0;
      if (!idle) {
        double raw = oracle_raw_tss(prof[m].w_p, prof[m].w_q, P[c], D[c], A_int[c], W_int[c],
                                    window_ms);
        if (init) s = oracle_smooth(prof[m].alpha, raw, s);
        else { s = raw; init = 1; }
      }
      S[c] = s;
      flags[c] = (uint8_t)((idle ? OR_IDLE : 0) | (init ? OR_INIT : 0));
    }
  }
  return 0;
}

/* ----------------------------------------------------------------------
 * Control replay of one scenario over its trace's smoothed TSS.
 * S, flags: [n_windows][M] of the scenario's trace; prof: [M] of that trace.
 * Writes up to move_cap moves (in selection order), the total number of
 * moves, the final routable replicas and, per model, the sum over windows
 * of the replicas in force during each window.
 * -------------------------------------------------------------------- */
int oracle_control(int64_t window_ms, int64_t duration_ms, int64_t fast_ms, int64_t slow_ms,
                   int32_t M, int32_t budget, const or_profile* prof, const double* S,
                   const uint8_t* flags, const or_scenario* sc, or_move* moves,
                   uint32_t move_cap, uint32_t* n_moves, int32_t* r_final,
                   int64_t* r_windows) {
  if (window_ms <= 0 || duration_ms % window_ms || fast_ms <= 0 || slow_ms <= 0 || M < 1 ||
      M > OR_MAX_MODELS)
    return -1;
  const int64_t nW = duration_ms / window_ms;
  int32_t R[OR_MAX_MODELS];
  double theta_eff[OR_MAX_MODELS], tau_c[OR_MAX_MODELS], Z[OR_MAX_MODELS];
  int crit[OR_MAX_MODELS], surplus[OR_MAX_MODELS], ok[OR_MAX_MODELS], used[OR_MAX_MODELS];
  int64_t pool = budget;
  for (int m = 0; m < M; ++m) {
    R[m] = prof[m].r_init;
    pool -= R[m];
    r_windows[m] = 0;
    theta_eff[m] = prof[m].theta * sc->theta_scale;
    tau_c[m] = sc->tau_crit_override >= 0.0 ? sc->tau_crit_override : prof[m].tau_crit;
  }
  if (pool < 0) return -4;
  uint32_t nm = 0;

  for (int64_t w = 0; w < nW; ++w) {
    for (int m = 0; m < M; ++m) r_windows[m] += R[m];   /* replicas serving window w */
    const int64_t t_end = (w + 1) * window_ms;
    const int fast = t_end % fast_ms == 0;
    const int slow = t_end % slow_ms == 0;
    if (!fast && !slow) continue;

    /* Eq. (2) and the three regions */
    int any_crit = 0;
    for (int m = 0; m < M; ++m) {
      const uint8_t f = flags[w * M + m];
      Z[m] = ((f & OR_IDLE) || !(f & OR_INIT)) ? INFINITY : S[w * M + m] / theta_eff[m];
      crit[m] = Z[m] < tau_c[m];
      surplus[m] = Z[m] > prof[m].tau_surplus;
      any_crit |= crit[m];
    }

    /* dual-speed control: a critical model makes this a rescue tick (fast
       cadence only) and defers all rebalancing; otherwise the slow cadence
       rebalances toward models below their healthy boundary */
    int path;
    if (any_crit) {
      if (!fast) continue;
      path = OR_RESCUE;
      for (int m = 0; m < M; ++m) ok[m] = crit[m];
    } else if (slow) {
      path = OR_REBALANCE;
      for (int m = 0; m < M; ++m) ok[m] = Z[m] < 1.0;
    } else {
      continue;
    }

    for (int m = 0; m < M; ++m) used[m] = 0;
    for (uint32_t k = 0; k < sc->max_moves; ++k) {
      /* Eq. (3): receiver = argmin Z among eligible models */
      int r = -1;
      for (int m = 0; m < M; ++m)
        if (ok[m] && !used[m] && (r < 0 || Z[m] < Z[r])) r = m;
      if (r < 0) break;
      int d = OR_POOL;
      if (pool > 0) {
        pool -= 1;                                         /* idle capacity first */
      } else {
        /* donor: surplus first, nominal only when no surplus donor exists;
           above its floor and strictly healthier than the receiver */
        int best = -1;
        for (int pass = 0; pass < 2 && best < 0; ++pass) {
          for (int m = 0; m < M; ++m) {
            const int nominal = !crit[m] && !surplus[m];
            const int in_class = pass == 0 ? surplus[m] : nominal;
            if (!in_class || used[m] || m == r || R[m] <= prof[m].r_min || !(Z[m] > Z[r]))
              continue;
            if (best < 0 || Z[m] > Z[best]) best = m;
          }
        }
        if (best < 0) break;
        d = best;
        R[d] -= 1;
        used[d] = 1;
      }
      R[r] += 1;
      used[r] = 1;
      if (nm < move_cap) {
        moves[nm].window = (uint32_t)w;
        moves[nm].path = (uint8_t)path;
        moves[nm].receiver = (uint8_t)r;
        moves[nm].donor = (uint8_t)d;
        moves[nm].pad = 0;
      }
      nm += 1;
    }
  }
  for (int m = 0; m < M; ++m) r_final[m] = R[m];
  *n_moves = nm;
  return 0;
}

static int cmp_u32(const void* a, const void* b) {
  const uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* ----------------------------------------------------------------------
 * Request identity check for one trace: a request is admitted once, on its
 * first prefill chunk (the ADMIT bit moves it from the waiting to the active
 * set of Eq. (1), Section "Design Rationale and Definition"). Returns 0, or
 * -6 when some request id carries the ADMIT bit on more than one row, with
 * the smallest such id in *dup_id. ids_scratch holds n_events ids.
 * -------------------------------------------------------------------- */
int oracle_check_admits(const uint32_t* req, const uint8_t* type, int64_t n_events,
                        uint32_t* ids_scratch, uint32_t* dup_id) {
  int64_t n = 0;
  for (int64_t i = 0; i < n_events; ++i)
    if (type[i] == (OR_PREFILL | OR_ADMIT)) ids_scratch[n++] = req[i];
  qsort(ids_scratch, (size_t)n, sizeof(uint32_t), cmp_u32);
  for (int64_t i = 1; i < n; ++i)
    if (ids_scratch[i] == ids_scratch[i - 1]) {
      *dup_id = ids_scratch[i];
      return -6;
    }
  return 0;
}

static int cmp_u64(const void* a, const void* b) {
  const uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

/* ----------------------------------------------------------------------
 * Request lifecycle check for one trace. A request enters the waiting set
 * once (its ARRIVE), leaves the active set once (its FINISH), and no longer
 * arrives or produces output afterwards (the request counts of Eq. (1),
 * Section "Design Rationale and Definition"): per request id at most one
 * ARRIVE row and one FINISH row, and no ARRIVE or DECODE row with a later
 * timestamp than the FINISH (rows of one instant may come in any order).
 * Returns 0, or -7 with the smallest offending id in *bad_id. keys_scratch
 * holds n_events uint64 words.
 * -------------------------------------------------------------------- */
int oracle_check_lifecycle(const uint32_t* req, const uint8_t* type, const int64_t* ts, int64_t n_events,
                           uint64_t* keys_scratch, uint32_t* bad_id) {
  int64_t n = 0;
  for (int64_t i = 0; i < n_events; ++i) {
    const uint32_t kind = type[i] & 3u;
    if (kind == OR_ARRIVE || kind == OR_DECODE || kind == OR_FINISH)
      keys_scratch[n++] = ((uint64_t)req[i] << 32) | (uint64_t)i;
  }
  qsort(keys_scratch, (size_t)n, sizeof(uint64_t), cmp_u64);
  for (int64_t g = 0; g < n;) {  /* the rows of one id */
    const uint32_t id = (uint32_t)(keys_scratch[g] >> 32);
    int64_t h = g;
    int arrivals = 0, finishes = 0;
    int64_t fin_ts = 0, last_ad_ts = INT64_MIN;
    for (; h < n && (uint32_t)(keys_scratch[h] >> 32) == id; ++h) {
      const int64_t row = (int64_t)(uint32_t)keys_scratch[h];
      const uint32_t kind = type[row] & 3u;
      if (kind == OR_FINISH) {
        ++finishes;
        fin_ts = ts[row];
      } else {
        if (kind == OR_ARRIVE) ++arrivals;
        if (ts[row] > last_ad_ts) last_ad_ts = ts[row];
      }
    }
    if (arrivals > 1 || finishes > 1 || (finishes == 1 && last_ad_ts > fin_ts)) {
      *bad_id = id;
      return -7;
    }
    g = h;
  }
  return 0;
}
