/*
 * tre_oracle_act.c - CPU oracle for the control replay with an actuation
 * model: replica wake / sleep delays, GPU footprints under the fixed budget,
 * transfers in progress that are not pre-empted, and donor-release vetoes.
 *
 * TEST INFRASTRUCTURE ONLY, like tre_oracle.c: linked by the tests, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product
 * path, and sharing no code with the GPU library. It is a separate
 * statement of the control rules (not a call into the base oracle), so the
 * tests can check that it reduces to the base rules when actuation is
 * instantaneous.
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE).
 *   - Section "Dual-Speed Control": rescue at the fast cadence when a model
 *     is critical, acquiring idle capacity before any donor release;
 *     rebalancing at the slow cadence otherwise; a transfer in progress is
 *     not pre-empted by a new request (hard guardrails are not modelled);
 *   - Section "Bounded Pairwise Transfer": one budget-feasible transition
 *     per receiver-donor pair per tick, counted in GPU footprints (not a
 *     one-to-one replica exchange); the donor-side release guard hides the
 *     replica, lets it drain, and commits the release by sleeping it, or
 *     defers the release when a local guardrail is violated;
 *   - Section "System Boundary and Replica State": only runtime-ready and
 *     gateway-visible replicas are routable; a reactivating replica becomes
 *     routable once ready;
 *   - Section on deployment overhead: sleep and wake take seconds (the
 *     paper measures 1.87 s and 1.31 s on its testbed).
 *
 * Readings (listed in the design notes):
 *   - the budget B is in GPUs and a replica of model m holds g_m >= 1 GPUs;
 *     idle GPUs F = B - sum_m g_m * (routable + waking + draining);
 *   - delays are whole windows; a transition completing at the end of window
 *     u takes effect from window u + 1, and for decisions from the first
 *     tick after window u;
 *   - pool path: if F >= g_r, the receiver wakes a replica on g_r idle GPUs
 *     and it is routable after wake_w windows;
 *   - donor path: the donor's replica stops being routable at once (hidden
 *     while it drains and sleeps, sleep_w windows); its g_d GPUs go to the
 *     receiver when the sleep completes, and the receiver's wake starts
 *     then; the shortfall max(0, g_r - g_d) is taken from the idle GPUs at
 *     the move (a donor is eligible only if F >= g_r - g_d), the excess
 *     max(0, g_d - g_r) returns to them when the sleep completes;
 *   - a model with a transition in flight is neither receiver nor donor;
 *   - veto[t] bit m: the release guard refuses model m as donor at tick t;
 *   - every other rule is the base rule (regions, cadence, argmin / argmax
 *     with the lowest index on ties, up to K moves per tick).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define OA_RESCUE 1
#define OA_REBALANCE 2
#define OA_POOL 0xFF
#define OA_IDLE 1
#define OA_INIT 2
#define OA_MAX_MODELS 256

#define OA_NONE 0
#define OA_WAKE 1
#define OA_SLEEP 2

/* the profile, scenario and move records of the base oracle (same layout) */
typedef struct {
  double w_p, w_q, alpha, theta, tau_crit, tau_surplus;
  int32_t r_min, r_init;
} oa_profile;

typedef struct {
  uint32_t trace, max_moves;
  double theta_scale, tau_crit_override;
} oa_scenario;

typedef struct {
  uint32_t window;
  uint8_t path, receiver, donor, pad;
} oa_move;

/*
 * Control replay of one scenario over one trace's smoothed TSS S and flags
 * ([n_windows][M]). footprint: [M] GPUs per replica (NULL: 1); veto:
 * [n_ticks] masks (NULL: none). Outputs as the base replay; idle_final
 * (may be NULL) receives the idle GPUs after the last window and held_final
 * ([M], may be NULL) the GPUs a transition still in flight holds (g for a
 * wake, the excess still to return for a sleep), so that
 * idle + sum g * r_final + sum held = budget.
 * Returns 0, -1 on bad arguments, -4 if the initial replicas exceed the
 * budget.
 */
int oracle_control_act(int64_t window_ms, int64_t duration_ms, int64_t fast_ms, int64_t slow_ms,
                       int32_t M, int32_t budget, const oa_profile* prof, const double* S,
                       const uint8_t* flags, const oa_scenario* sc, int64_t wake_w,
                       int64_t sleep_w, const int32_t* footprint, const uint64_t* veto,
                       oa_move* moves, uint32_t move_cap, uint32_t* n_moves, int32_t* r_final,
                       int64_t* r_windows, int64_t* idle_final, int32_t* held_final) {
  if (window_ms <= 0 || duration_ms % window_ms || fast_ms <= 0 || slow_ms <= 0 || M < 1 ||
      M > OA_MAX_MODELS || wake_w < 0 || sleep_w < 0)
    return -1;
  const int64_t nW = duration_ms / window_ms;
  int32_t R[OA_MAX_MODELS], g[OA_MAX_MODELS], kind[OA_MAX_MODELS];
  int64_t until[OA_MAX_MODELS], ret[OA_MAX_MODELS];
  double theta_eff[OA_MAX_MODELS], tau_c[OA_MAX_MODELS], Z[OA_MAX_MODELS];
  int crit[OA_MAX_MODELS], surplus[OA_MAX_MODELS], ok[OA_MAX_MODELS];
  int64_t idle = budget;
  for (int m = 0; m < M; ++m) {
    g[m] = footprint ? footprint[m] : 1;
    if (g[m] < 1) return -1;
    R[m] = prof[m].r_init;
    idle -= (int64_t)g[m] * R[m];
    kind[m] = OA_NONE;
    until[m] = -1;
    ret[m] = 0;
    r_windows[m] = 0;
    theta_eff[m] = prof[m].theta * sc->theta_scale;
    tau_c[m] = sc->tau_crit_override >= 0.0 ? sc->tau_crit_override : prof[m].tau_crit;
  }
  if (idle < 0) return -4;
  uint32_t nm = 0;
  int64_t tick = 0;

  for (int64_t w = 0; w < nW; ++w) {
    /* transitions that completed at the end of an earlier window */
    for (int m = 0; m < M; ++m) {
      if (kind[m] != OA_NONE && until[m] < w) {
        if (kind[m] == OA_WAKE) R[m] += 1;   /* routable from now on */
        else idle += ret[m];                 /* released GPUs are idle */
        kind[m] = OA_NONE;
        ret[m] = 0;
      }
    }
    for (int m = 0; m < M; ++m) r_windows[m] += R[m];  /* routable replicas in window w */
    const int64_t t_end = (w + 1) * window_ms;
    const int fast = t_end % fast_ms == 0;
    const int slow = t_end % slow_ms == 0;
    if (!fast && !slow) continue;
    const uint64_t vetoed = veto ? veto[tick] : 0u;
    tick += 1;

    int any_crit = 0;
    for (int m = 0; m < M; ++m) {
      const uint8_t f = flags[w * M + m];
      Z[m] = ((f & OA_IDLE) || !(f & OA_INIT)) ? INFINITY : S[w * M + m] / theta_eff[m];
      crit[m] = Z[m] < tau_c[m];
      surplus[m] = Z[m] > prof[m].tau_surplus;
      any_crit |= crit[m];
    }
    int path;
    if (any_crit) {
      if (!fast) continue;
      path = OA_RESCUE;
      for (int m = 0; m < M; ++m) ok[m] = crit[m];
    } else if (slow) {
      path = OA_REBALANCE;
      for (int m = 0; m < M; ++m) ok[m] = Z[m] < 1.0;
    } else {
      continue;
    }

    for (uint32_t k = 0; k < sc->max_moves; ++k) {
      /* Eq. (3) over models with no transition in flight */
      int r = -1;
      for (int m = 0; m < M; ++m)
        if (ok[m] && kind[m] == OA_NONE && (r < 0 || Z[m] < Z[r])) r = m;
      if (r < 0) break;
      int d = OA_POOL;
      if (idle >= g[r]) {
        idle -= g[r];
        kind[r] = OA_WAKE;
        until[r] = w + wake_w;
      } else {
        int best = -1;
        for (int pass = 0; pass < 2 && best < 0; ++pass) {
          for (int m = 0; m < M; ++m) {
            const int nominal = !crit[m] && !surplus[m];
            const int in_class = pass == 0 ? surplus[m] : nominal;
            if (!in_class || kind[m] != OA_NONE || m == r || R[m] <= prof[m].r_min ||
                !(Z[m] > Z[r]) || ((vetoed >> m) & 1u) || idle < (int64_t)g[r] - g[m])
              continue;
            if (best < 0 || Z[m] > Z[best]) best = m;
          }
        }
        if (best < 0) break;
        d = best;
        const int64_t short_by = (int64_t)g[r] - g[d];
        if (short_by > 0) idle -= short_by;
        R[d] -= 1;  /* hidden from routing at once */
        kind[d] = OA_SLEEP;
        until[d] = w + sleep_w;
        ret[d] = short_by < 0 ? -short_by : 0;
        kind[r] = OA_WAKE;
        until[r] = w + sleep_w + wake_w;
      }
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
  /* transitions completing at the end of the last window count as done */
  for (int m = 0; m < M; ++m) {
    if (kind[m] != OA_NONE && until[m] < nW) {
      if (kind[m] == OA_WAKE) R[m] += 1;
      else idle += ret[m];
      kind[m] = OA_NONE;
    }
  }
  for (int m = 0; m < M; ++m) {
    r_final[m] = R[m];
    if (held_final) held_final[m] = kind[m] == OA_WAKE ? g[m] : (kind[m] == OA_SLEEP ? (int32_t)ret[m] : 0);
  }
  if (idle_final) *idle_final = idle;
  *n_moves = nm;
  return 0;
}
