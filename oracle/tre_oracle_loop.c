/*
 * tre_oracle_loop.c - CPU oracle for the closed-loop replay: the requests of
 * a trace are served by each model's routable replicas, the controller's
 * moves change those replicas, and the TSS the controller reads comes from
 * the events that this service produces.
 *
 * TEST INFRASTRUCTURE ONLY, like tre_oracle.c: linked by the tests, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product
 * path, and sharing no code with the GPU library. The TSS at each tick is
 * the base oracle's (oracle_tss_trace over the events final by then).
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE).
 *   - Sections "Dual-Speed Control" and "Bounded Pairwise Transfer": the
 *     rules applied at each tick (as the base replay);
 *   - Section "System Boundary and Replica State": only routable replicas
 *     serve new requests; a hidden replica drains its in-flight requests;
 *   - Section "Bounded Pairwise Transfer": after each transition the
 *     controller observes the resulting service and re-evaluates at the
 *     next tick (here: the moves change the service that produces the
 *     next TSS).
 *
 * Readings (listed in the design notes):
 *   - each routable replica of model m has spr slots; a request holds one
 *     slot from its start to its last decode; requests of a model start in
 *     arrival order (FCFS) on the slot that frees first (lowest index on
 *     ties), at max(arrival, that slot's free time);
 *   - service times are whole milliseconds: a prompt chunk of c tokens
 *     takes ceil(c * prefill_us / 1000) ms, an output chunk of c tokens
 *     ceil(c * decode_us / 1000) ms; events as in the traces: ARRIVE at the
 *     arrival, one PREFILL per prompt chunk at its start (the first with
 *     ADMIT), one DECODE per output chunk at its completion, FINISH at the
 *     last decode; events at or after the end of the trace are dropped;
 *   - a move at the end of window w acts from (w+1)*window_ms: the
 *     receiver gains spr slots free from then; the donor's replica stops
 *     taking requests: its spr slots that free first are removed (requests
 *     running on them finish normally);
 *   - a receiver must have fewer than r_cap replicas; every other rule is
 *     the base rule (idle budget first, surplus then nominal donors, up to
 *     K moves per tick, each model in at most one move per tick);
 *   - latency outcomes as in the calibration sweep: a request whose FINISH
 *     is in the trace is judged (TTFT, E2E, TPOT against its model's SLO);
 *   - with the actuation model (oracle_loop_act), the actuation replay's
 *     rules (tre_oracle_act.c): the budget in GPUs with g_m GPUs per
 *     replica, a woken replica routable wake_w windows after its wake
 *     starts (its slots free from the start of the window after its wake
 *     completes), a donor's replica hidden at once (its earliest-free slots
 *     leave at the move) with its GPUs reaching the receiver after sleep_w
 *     windows, when the receiver's wake starts, a model with a transition
 *     in flight neither receiver nor donor, vetoed models not released; with
 *     no delays, unit footprints and no vetoes it is the plain closed loop.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OL_ARRIVE 0u
#define OL_PREFILL 1u
#define OL_DECODE 2u
#define OL_FINISH 3u
#define OL_ADMIT 0x80u
#define OL_RESCUE 1
#define OL_REBALANCE 2
#define OL_POOL 0xFF
#define OL_IDLE 1
#define OL_INIT 2
#define OL_MAX_MODELS 256
#define OL_NONE 0
#define OL_WAKE 1
#define OL_SLEEP 2

typedef struct {
  double w_p, w_q, alpha, theta, tau_crit, tau_surplus;
  int32_t r_min, r_init;
} ol_profile;

typedef struct {
  uint32_t trace, max_moves;
  double theta_scale, tau_crit_override;
} ol_scenario;

typedef struct {
  uint32_t window;
  uint8_t path, receiver, donor, pad;
} ol_move;

typedef struct {
  double ttft_ms, tpot_ms, e2e_ms, attain_q, reliability;
} ol_slo;

typedef struct {
  uint32_t prefill_us, decode_us;  /* per token on one slot */
} ol_svc;

typedef struct {
  uint32_t n_arrived, n_started, n_done, n_ok;
  int64_t e2e_sum, e2e_max;
} ol_stats;

/* the base oracle's TSS of one trace (tre_oracle.c) */
int oracle_tss_trace(const int64_t* ts, const uint8_t* model, const uint8_t* type, const uint16_t* tokens,
                     int64_t n, int64_t window_ms, int64_t duration_ms, int32_t M, const ol_profile* prof,
                     int64_t* P, int64_t* D, int64_t* A_int, int64_t* W_int, double* S, uint8_t* flags);

typedef struct {
  int64_t* ts;
  uint8_t* model;
  uint8_t* type;
  uint16_t* tokens;
  size_t n, cap;
} evbuf;

static int ev_push(evbuf* b, int64_t ts, int m, uint32_t type, uint32_t tokens) {
  if (b->n == b->cap) {
    size_t nc = b->cap ? 2 * b->cap : 4096;
    int64_t* t = realloc(b->ts, nc * sizeof(int64_t));
    if (!t) return -1;
    b->ts = t;
    uint8_t* mo = realloc(b->model, nc);
    if (!mo) return -1;
    b->model = mo;
    uint8_t* ty = realloc(b->type, nc);
    if (!ty) return -1;
    b->type = ty;
    uint16_t* to = realloc(b->tokens, nc * sizeof(uint16_t));
    if (!to) return -1;
    b->tokens = to;
    b->cap = nc;
  }
  b->ts[b->n] = ts;
  b->model[b->n] = (uint8_t)m;
  b->type[b->n] = (uint8_t)type;
  b->tokens[b->n] = (uint16_t)tokens;
  b->n += 1;
  return 0;
}

static void ev_free(evbuf* b) {
  free(b->ts);
  free(b->model);
  free(b->type);
  free(b->tokens);
}

static int64_t ceil_ms(int64_t tokens, uint32_t us) { return (tokens * (int64_t)us + 999) / 1000; }

typedef struct {
  int64_t ts;
  size_t i;
} ol_key;

static int by_ts_then_order(const void* x, const void* y) {
  const ol_key *a = (const ol_key*)x, *b = (const ol_key*)y;
  if (a->ts != b->ts) return a->ts < b->ts ? -1 : 1;
  return a->i < b->i ? -1 : (a->i > b->i ? 1 : 0);
}

/* move the pending events with ts < t_end to the final list in ts order
   (generation order on equal ts); they all lie at or after the final
   list's last event, since every event is generated at or after the start
   of the window in which it is generated */
static int settle(evbuf* fin, evbuf* pend, int64_t t_end) {
  ol_key* key = malloc(sizeof(ol_key) * (pend->n ? pend->n : 1));
  if (!key) return -1;
  size_t nsel = 0, k = 0;
  for (size_t i = 0; i < pend->n; ++i)
    if (pend->ts[i] < t_end) {
      key[nsel].ts = pend->ts[i];
      key[nsel].i = i;
      ++nsel;
    }
  qsort(key, nsel, sizeof(ol_key), by_ts_then_order);
  for (size_t a = 0; a < nsel; ++a) {
    const size_t i = key[a].i;
    if (ev_push(fin, pend->ts[i], pend->model[i], pend->type[i], pend->tokens[i])) {
      free(key);
      return -1;
    }
  }
  for (size_t i = 0; i < pend->n; ++i) {
    if (pend->ts[i] < t_end) continue;
    pend->ts[k] = pend->ts[i];
    pend->model[k] = pend->model[i];
    pend->type[k] = pend->type[i];
    pend->tokens[k] = pend->tokens[i];
    ++k;
  }
  pend->n = k;
  free(key);
  return 0;
}

/*
 * Closed-loop replay of one scenario over one trace's requests, with the
 * actuation model. req_off [M+1]: requests of model m are
 * [req_off[m], req_off[m+1]) of arrival_ms / prompt / output, in arrival
 * order. wake_w, sleep_w: delays in whole windows; footprint [M] GPUs per
 * replica (NULL: 1), the budget then in GPUs; veto [n_ticks] donor-release
 * masks (NULL: none). Outputs as the base replay (moves, n_moves, r_final
 * counting transitions completed by the end of the last window,
 * r_windows), per-model stats [M], optionally the idle GPUs at the end and
 * the GPUs transitions still in flight hold ([M]), the whole trace's
 * smoothed TSS and flags [n_windows][M], its event count and its events
 * (when they fit ev_cap). Returns 0, -1 on bad arguments, -2 out of
 * memory, -4 if the initial replicas exceed the budget.
 */
int oracle_loop_act(int64_t window_ms, int64_t duration_ms, int64_t fast_ms, int64_t slow_ms, int32_t M,
                    int32_t budget, const ol_profile* prof, const ol_scenario* sc, const ol_slo* slo,
                    const ol_svc* svc, int32_t spr, int32_t r_cap, int32_t prefill_chunk, int32_t decode_chunk,
                    const int64_t* req_off, const int64_t* arrival_ms, const uint16_t* prompt,
                    const uint16_t* output, int64_t wake_w, int64_t sleep_w, const int32_t* footprint,
                    const uint64_t* veto, ol_move* moves, uint32_t move_cap, uint32_t* n_moves, int32_t* r_final,
                    int64_t* r_windows, ol_stats* stats, int64_t* idle_final, int32_t* held_final, double* S_out,
                    uint8_t* flags_out, int64_t* n_events_out, int64_t ev_cap, int64_t* ev_ts, uint8_t* ev_model,
                    uint8_t* ev_type, uint16_t* ev_tokens) {
  if (window_ms <= 0 || duration_ms % window_ms || fast_ms <= 0 || slow_ms <= 0 || M < 1 ||
      M > OL_MAX_MODELS || spr < 1 || r_cap < 1 || prefill_chunk < 1 || decode_chunk < 1 || wake_w < 0 ||
      sleep_w < 0)
    return -1;
  const int64_t nW = duration_ms / window_ms;
  int32_t R[OL_MAX_MODELS], g[OL_MAX_MODELS], kind[OL_MAX_MODELS];
  int64_t until[OL_MAX_MODELS], ret[OL_MAX_MODELS];
  int64_t idle = budget;  /* idle GPUs */
  for (int m = 0; m < M; ++m) {
    R[m] = prof[m].r_init;
    g[m] = footprint ? footprint[m] : 1;
    if (R[m] < 0 || R[m] > r_cap || g[m] < 1) return -1;
    idle -= (int64_t)g[m] * R[m];
    kind[m] = OL_NONE;
    until[m] = -1;
    ret[m] = 0;
    r_windows[m] = 0;
    memset(&stats[m], 0, sizeof(ol_stats));
  }
  if (idle < 0) return -4;
  int rc = 0;
  /* slot free times per model: R[m] * spr active slots */
  int64_t** slot = calloc((size_t)M, sizeof(int64_t*));
  int64_t* next_arr = calloc((size_t)M, sizeof(int64_t));   /* next request to arrive */
  int64_t* next_start = calloc((size_t)M, sizeof(int64_t)); /* next request to start */
  double* S = malloc(sizeof(double) * (size_t)(nW * M));
  uint8_t* fl = malloc((size_t)(nW * M));
  int64_t* Pt = malloc(sizeof(int64_t) * (size_t)(nW * M));
  int64_t* Dt = malloc(sizeof(int64_t) * (size_t)(nW * M));
  int64_t* At = malloc(sizeof(int64_t) * (size_t)(nW * M));
  int64_t* Wt = malloc(sizeof(int64_t) * (size_t)(nW * M));
  evbuf fin = {0}, pend = {0};
  if (!slot || !next_arr || !next_start || !S || !fl || !Pt || !Dt || !At || !Wt) {
    rc = -2;
    goto done;
  }
  for (int m = 0; m < M; ++m) {
    /* a model never holds more than the budget's replicas */
    slot[m] = malloc(sizeof(int64_t) * (size_t)(r_cap > budget ? r_cap : budget) * (size_t)spr);
    if (!slot[m]) {
      rc = -2;
      goto done;
    }
    for (int64_t i = 0; i < (int64_t)R[m] * spr; ++i) slot[m][i] = 0;
    next_arr[m] = req_off[m];
    next_start[m] = req_off[m];
  }
  uint32_t nm = 0;
  int64_t tick = 0;
  for (int64_t w = 0; w < nW; ++w) {
    const int64_t w_end = (w + 1) * window_ms;
    /* transitions that completed at the end of an earlier window: a woken
       replica's slots are free from the start of this window */
    for (int m = 0; m < M; ++m) {
      if (kind[m] != OL_NONE && until[m] < w) {
        if (kind[m] == OL_WAKE) {
          for (int q = 0; q < spr; ++q) slot[m][(int64_t)R[m] * spr + q] = w * window_ms;
          R[m] += 1;
        } else {
          idle += ret[m];
        }
        kind[m] = OL_NONE;
        ret[m] = 0;
      }
    }
    for (int m = 0; m < M; ++m) {
      /* arrivals in this window */
      while (next_arr[m] < req_off[m + 1] && arrival_ms[next_arr[m]] < w_end) {
        if (ev_push(&pend, arrival_ms[next_arr[m]], m, OL_ARRIVE, prompt[next_arr[m]])) { rc = -2; goto done; }
        stats[m].n_arrived += 1;
        next_arr[m] += 1;
      }
      /* starts in this window, FCFS on the slot that frees first */
      const int64_t ns = (int64_t)R[m] * spr;
      while (next_start[m] < next_arr[m] && ns > 0) {
        int64_t best = 0;
        for (int64_t k = 1; k < ns; ++k)
          if (slot[m][k] < slot[m][best]) best = k;
        const int64_t i = next_start[m];
        const int64_t s = arrival_ms[i] > slot[m][best] ? arrival_ms[i] : slot[m][best];
        if (s >= w_end) break;  /* waits for the next window (capacity may change at its start) */
        int64_t t = s;
        int64_t left = prompt[i];
        int first = 1;
        while (left > 0) {
          const int64_t ch = left < prefill_chunk ? left : prefill_chunk;
          if (t < duration_ms && ev_push(&pend, t, m, OL_PREFILL | (first ? OL_ADMIT : 0u), (uint32_t)ch)) {
            rc = -2;
            goto done;
          }
          first = 0;
          t += ceil_ms(ch, svc[m].prefill_us);
          left -= ch;
        }
        left = output[i];
        int64_t t_first = -1, first_ch = 0;
        while (left > 0) {
          const int64_t ch = left < decode_chunk ? left : decode_chunk;
          t += ceil_ms(ch, svc[m].decode_us);
          if (t_first < 0) {
            t_first = t;
            first_ch = ch;
          }
          if (t < duration_ms && ev_push(&pend, t, m, OL_DECODE, (uint32_t)ch)) { rc = -2; goto done; }
          left -= ch;
        }
        if (t < duration_ms && ev_push(&pend, t, m, OL_FINISH, 0)) { rc = -2; goto done; }
        slot[m][best] = t;
        stats[m].n_started += 1;
        if (t < duration_ms && t_first >= 0) {  /* judged */
          const int64_t ttft = t_first - arrival_ms[i], e2e = t - arrival_ms[i];
          const int64_t after = (int64_t)output[i] - first_ch;
          int good = (double)ttft <= slo[m].ttft_ms && (double)e2e <= slo[m].e2e_ms;
          if (after > 0) good = good && (double)(t - t_first) / (double)after <= slo[m].tpot_ms;
          stats[m].n_done += 1;
          stats[m].n_ok += (uint32_t)good;
          stats[m].e2e_sum += e2e;
          if (e2e > stats[m].e2e_max) stats[m].e2e_max = e2e;
        }
        next_start[m] += 1;
      }
    }
    for (int m = 0; m < M; ++m) r_windows[m] += R[m];
    const int fast = w_end % fast_ms == 0, slow = w_end % slow_ms == 0;
    if (!fast && !slow) continue;
    const uint64_t vetoed = veto ? veto[tick] : 0u;
    tick += 1;
    /* the TSS of window w from the events final by its end */
    if (settle(&fin, &pend, w_end)) { rc = -2; goto done; }
    if (oracle_tss_trace(fin.ts, fin.model, fin.type, fin.tokens, (int64_t)fin.n, window_ms, duration_ms, M,
                         prof, Pt, Dt, At, Wt, S, fl)) {
      rc = -1;
      goto done;
    }
    double Z[OL_MAX_MODELS];
    int crit[OL_MAX_MODELS], surplus[OL_MAX_MODELS], ok[OL_MAX_MODELS];
    int any_crit = 0;
    for (int m = 0; m < M; ++m) {
      const uint8_t f = fl[w * M + m];
      const double tau_c = sc->tau_crit_override >= 0.0 ? sc->tau_crit_override : prof[m].tau_crit;
      Z[m] = ((f & OL_IDLE) || !(f & OL_INIT)) ? INFINITY : S[w * M + m] / (prof[m].theta * sc->theta_scale);
      crit[m] = Z[m] < tau_c;
      surplus[m] = Z[m] > prof[m].tau_surplus;
      any_crit |= crit[m];
    }
    int path;
    if (any_crit) {
      if (!fast) continue;
      path = OL_RESCUE;
      for (int m = 0; m < M; ++m) ok[m] = crit[m];
    } else if (slow) {
      path = OL_REBALANCE;
      for (int m = 0; m < M; ++m) ok[m] = Z[m] < 1.0;
    } else {
      continue;
    }
    /* a model in a move this tick, or with a transition in flight, has
       kind != OL_NONE: neither receiver nor donor */
    for (uint32_t k = 0; k < sc->max_moves; ++k) {
      int r = -1;
      for (int m = 0; m < M; ++m)
        if (ok[m] && kind[m] == OL_NONE && R[m] < r_cap && (r < 0 || Z[m] < Z[r])) r = m;
      if (r < 0) break;
      int d = OL_POOL;
      if (idle >= g[r]) {
        idle -= g[r];
        kind[r] = OL_WAKE;
        until[r] = w + wake_w;
      } else {
        int best = -1;
        for (int pass = 0; pass < 2 && best < 0; ++pass) {
          for (int m = 0; m < M; ++m) {
            const int in_class = pass == 0 ? surplus[m] : (!crit[m] && !surplus[m]);
            if (!in_class || kind[m] != OL_NONE || m == r || R[m] <= prof[m].r_min || !(Z[m] > Z[r]) ||
                ((vetoed >> m) & 1u) || idle < (int64_t)g[r] - g[m])
              continue;
            if (best < 0 || Z[m] > Z[best]) best = m;
          }
        }
        if (best < 0) break;
        d = best;
        const int64_t short_by = (int64_t)g[r] - g[d];
        if (short_by > 0) idle -= short_by;
        /* the donor's replica: its spr slots that free first leave */
        for (int q = 0; q < spr; ++q) {
          int64_t ns = (int64_t)R[d] * spr - q, lo = 0;
          if (ns <= 0) break;
          for (int64_t x = 1; x < ns; ++x)
            if (slot[d][x] < slot[d][lo]) lo = x;
          for (int64_t x = lo; x + 1 < ns; ++x) slot[d][x] = slot[d][x + 1];
        }
        if (R[d] > 0) R[d] -= 1;  /* always: a donor is above its floor */
        kind[d] = OL_SLEEP;
        until[d] = w + sleep_w;
        ret[d] = short_by < 0 ? -short_by : 0;
        kind[r] = OL_WAKE;
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
  *n_moves = nm;
  /* transitions completing at the end of the last window count as done */
  for (int m = 0; m < M; ++m) {
    if (kind[m] != OL_NONE && until[m] < nW) {
      if (kind[m] == OL_WAKE) R[m] += 1;
      else idle += ret[m];
      kind[m] = OL_NONE;
      ret[m] = 0;
    }
  }
  for (int m = 0; m < M; ++m) {
    r_final[m] = R[m];
    if (held_final) held_final[m] = kind[m] == OL_WAKE ? g[m] : (kind[m] == OL_SLEEP ? (int32_t)ret[m] : 0);
  }
  if (idle_final) *idle_final = idle;
  if (settle(&fin, &pend, duration_ms)) { rc = -2; goto done; }
  if (n_events_out) *n_events_out = (int64_t)fin.n;
  if (ev_ts && (int64_t)fin.n <= ev_cap) {
    memcpy(ev_ts, fin.ts, sizeof(int64_t) * fin.n);
    memcpy(ev_model, fin.model, fin.n);
    memcpy(ev_type, fin.type, fin.n);
    memcpy(ev_tokens, fin.tokens, sizeof(uint16_t) * fin.n);
  }
  if (S_out || flags_out) {
    if (oracle_tss_trace(fin.ts, fin.model, fin.type, fin.tokens, (int64_t)fin.n, window_ms, duration_ms, M, prof,
                         Pt, Dt, At, Wt, S, fl)) {
      rc = -1;
      goto done;
    }
    if (S_out) memcpy(S_out, S, sizeof(double) * (size_t)(nW * M));
    if (flags_out) memcpy(flags_out, fl, (size_t)(nW * M));
  }
done:
  if (slot)
    for (int m = 0; m < M; ++m) free(slot[m]);
  free(slot);
  free(next_arr);
  free(next_start);
  free(S);
  free(fl);
  free(Pt);
  free(Dt);
  free(At);
  free(Wt);
  ev_free(&fin);
  ev_free(&pend);
  return rc;
}

/* the closed loop with instantaneous actuation, unit footprints, no vetoes */
int oracle_loop(int64_t window_ms, int64_t duration_ms, int64_t fast_ms, int64_t slow_ms, int32_t M,
                int32_t budget, const ol_profile* prof, const ol_scenario* sc, const ol_slo* slo,
                const ol_svc* svc, int32_t spr, int32_t r_cap, int32_t prefill_chunk, int32_t decode_chunk,
                const int64_t* req_off, const int64_t* arrival_ms, const uint16_t* prompt,
                const uint16_t* output, ol_move* moves, uint32_t move_cap, uint32_t* n_moves,
                int32_t* r_final, int64_t* r_windows, ol_stats* stats, double* S_out, uint8_t* flags_out,
                int64_t* n_events_out, int64_t ev_cap, int64_t* ev_ts, uint8_t* ev_model, uint8_t* ev_type,
                uint16_t* ev_tokens) {
  return oracle_loop_act(window_ms, duration_ms, fast_ms, slow_ms, M, budget, prof, sc, slo, svc, spr, r_cap,
                         prefill_chunk, decode_chunk, req_off, arrival_ms, prompt, output, 0, 0, NULL, NULL, moves,
                         move_cap, n_moves, r_final, r_windows, stats, NULL, NULL, S_out, flags_out, n_events_out,
                         ev_cap, ev_ts, ev_model, ev_type, ev_tokens);
}
