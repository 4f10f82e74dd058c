/*
 * tre.h - C ABI of the MI355X (gfx950) replay library for Token Service
 * Share (TSS) evaluation and TSS-guided receiver/donor rebalancing.
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE).
 *   - TSS, Eq. (1): effective token service per active-or-waiting request,
 *     Section "Design Rationale and Definition";
 *   - smoothing, Eq. (2) normalisation Z = TSS/theta and the three regions
 *     tau_crit < 1 < tau_surplus, Section "Smoothing, Normalization, and
 *     Calibration";
 *   - rescue / rebalancing cadences and Eq. (3) receiver = argmin Z, donor
 *     preference, Section "Dual-Speed Control";
 *   - one bounded transition per pair and tick, receiver below its boundary,
 *     donor above its floor, fixed budget, Section "Bounded Pairwise Transfer".
 *
 * Conventions
 *   - Every call returns a status (TRE_OK = 0); nothing throws or exits.
 *     tre_last_error() gives a message for the calling thread's last error.
 *   - "device" pointers are HIP device memory owned by the caller; "host"
 *     pointers are ordinary host memory, read during the call only.
 *   - Hot calls (tre_eval_tss, tre_rebalance, tre_sweep) only check their
 *     arguments on the host and enqueue work on `stream` (a hipStream_t, or
 *     NULL for the default stream); they return before the work completes.
 *     Parameter tables are checked by tre_check_params (synchronous); the
 *     hot calls trust them. Invalid tables cannot make a kernel read or write
 *     out of bounds, but their results are unspecified.
 *   - Per-cell arrays are laid out [trace][window][model], row-major.
 *   - Handles are immutable after tre_load_events; concurrent calls on one
 *     handle with distinct outputs and workspaces are safe.
 *   - Floating point: IEEE binary64, round to nearest even, no contraction,
 *     in the operation order documented at tre_eval_tss; results are
 *     bit-identical across launches and grid shapes.
 */
#ifndef TRE_H
#define TRE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------- status */
#define TRE_OK 0
#define TRE_EINVAL 1  /* bad argument, configuration or parameter table       */
#define TRE_EORDER 2  /* timestamps unsorted within a trace or out of range    */
#define TRE_ESCHEMA 3 /* model index >= n_models or undefined type bits        */
#define TRE_ERANGE 4  /* a trace exceeds the library's counting limits         */
#define TRE_ENOMEM 5  /* workspace too small                                   */
#define TRE_EHIP 6    /* HIP runtime error                                     */
#define TRE_ESTATE 7  /* a request count of Eq. (1) below zero, or a request
                         id off its lifecycle (see tre_load_events)          */

/* Maximum models per trace (one wavefront lane per model). */
#define TRE_MAX_MODELS 64
/* Maximum events that may fall in one window of one trace; the limit is
   also at most (2^31 - 1) / window_ms, which keeps every per-window sum
   inside its packed 32-bit field. */
#define TRE_MAX_EVENTS_PER_WINDOW 65535

/* ------------------------------------------------------------- events
 * One event per row, structure of arrays, sorted by ts within each trace:
 *   ts      int64   ms from trace start, 0 <= ts < duration_ms
 *   model   uint8   model index < n_models
 *   req     uint32  request id (read only by the load-time admission check
 *                   and the calibration sweep; may be NULL otherwise)
 *   type    uint8   bits 0-1 kind: 0 ARRIVE (joins the model's waiting
 *                   queue), 1 PREFILL (prompt tokens served), 2 DECODE
 *                   (output tokens served), 3 FINISH (leaves the active set);
 *                   bit 7 ADMIT, only on a PREFILL (waiting -> active);
 *                   other bits 0
 *   tokens  uint16  tokens served by a PREFILL / DECODE; ignored otherwise
 * The active count A_m(t) and waiting count W_m(t) of Eq. (1) are the
 * running sums of these transitions, starting at 0. */
#define TRE_ARRIVE 0
#define TRE_PREFILL 1
#define TRE_DECODE 2
#define TRE_FINISH 3
#define TRE_ADMIT 0x80

/* Shared shape of every trace in a handle. window_ms must divide
   duration_ms and both periods. The fast period is the rescue cadence, the
   slow period the rebalancing cadence (Section "Dual-Speed Control"). */
typedef struct {
  int64_t window_ms;
  int64_t duration_ms;
  int64_t fast_period_ms;
  int64_t slow_period_ms;
  int32_t n_models;  /* 1 .. TRE_MAX_MODELS */
  int32_t budget;    /* fixed replica budget (unit footprint) */
} tre_trace_cfg;

/* Per-(trace, model) control profile: the paper's six scalars per
   model-SLO pair (Section "Smoothing, Normalization, and Calibration") plus
   the minimum routable-replica floor and the initial routable replicas.
   Requirements (tre_check_params): w_p >= 0, w_q >= 0, 0 < alpha <= 1,
   theta > 0, 0 <= tau_crit < tau_surplus, r_min >= 0, r_init >= 0. */
typedef struct {
  double w_p, w_q, alpha, theta, tau_crit, tau_surplus;
  int32_t r_min, r_init;
} tre_profile; /* 56 bytes */

/* One what-if scenario: a trace, the moves allowed per tick (K), a scale
   applied to every healthy boundary theta, and a rescue threshold that
   replaces every profile's tau_crit when >= 0. */
typedef struct {
  uint32_t trace;
  uint32_t max_moves;
  double theta_scale;
  double tau_crit_override;
} tre_scenario; /* 24 bytes */

#define TRE_PATH_RESCUE 1
#define TRE_PATH_REBALANCE 2
#define TRE_DONOR_POOL 0xFF

/* One capacity transition decided at the end of window `window`; donor
   TRE_DONOR_POOL means idle budget. */
typedef struct {
  uint32_t window;
  uint8_t path, receiver, donor, pad;
} tre_move; /* 8 bytes */

typedef struct tre_events tre_events; /* opaque */

typedef struct {
  uint32_t n_traces;
  uint32_t n_models;
  int64_t n_events;   /* trace_off[n_traces] - trace_off[0] */
  int64_t n_windows;  /* duration_ms / window_ms */
  int64_t n_ticks;    /* windows that end on a fast or slow period */
} tre_info;

/* Optional per-cell outputs of tre_eval_tss, each [n_traces][n_windows]
   [n_models] in device memory, any may be NULL:
     prefill, decode  tokens served in the window;
     a_int, w_int     integral of A_m(t), W_m(t) over the window (request*ms);
     tss64            smoothed TSS (fp64);
     tss32            smoothed TSS rounded to fp32;
     flags            bit 0: idle window (no tokens, nothing active or
                      waiting), bit 1: smoothed value initialised. */
typedef struct {
  uint32_t* prefill;
  uint32_t* decode;
  int64_t* a_int;
  int64_t* w_int;
  double* tss64;
  float* tss32;
  uint8_t* flags;
} tre_tss_out;

#define TRE_FLAG_IDLE 1
#define TRE_FLAG_INIT 2

/* Outputs of the control replay, device memory:
     moves      [n_scenarios][move_cap]: moves in selection order; only the
                first min(n_moves[s], move_cap) entries of a scenario are
                written;
     n_moves    [n_scenarios]: moves decided (may exceed move_cap);
     r_final    [n_scenarios][n_models]: routable replicas after the last
                window;
     r_windows  [n_scenarios][n_models]: sum over windows of the replicas in
                force during the window. */
typedef struct {
  tre_move* moves;
  uint32_t move_cap;
  uint32_t* n_moves;
  int32_t* r_final;
  int64_t* r_windows;
} tre_ctl_out;

/* Message for the calling thread's last non-OK status ("" if none). */
const char* tre_last_error(void);

/* Register event columns (device, borrowed: the caller keeps them alive
   and unchanged while the handle is used) and CSR trace offsets (host,
   copied: trace i is rows [trace_off[i], trace_off[i+1]) of every column,
   non-decreasing, trace_off[0] >= 0). `cfg` (host) is copied. Column
   pointers need 16-byte alignment (ts, tokens) or 8-byte (model, type),
   and every column must stay readable for 16 bytes past its last row
   (row trace_off[n_traces] - 1): tile loads are rounded up to 16 bytes.
   duration_ms must be below 2^32 and a trace below 2^27 events.
   With flags & TRE_VALIDATE the events are checked on the device and the
   call waits for the result:
     TRE_EORDER   a timestamp unsorted within its trace or outside
                  [0, duration_ms);
     TRE_ESCHEMA  a model index >= n_models or undefined type bits;
     TRE_ERANGE   more events in one window of one trace than the limit;
     TRE_ESTATE   the active or the waiting count of a model (A_m(t),
                  W_m(t) of Eq. (1), Section "Design Rationale and
                  Definition": numbers of requests) below zero at some
                  instant t, i.e. after the last row with that timestamp
                  (rows of one instant may come in any order); or, when
                  `req` is given, a request id off its lifecycle within a
                  trace: the ADMIT bit on more than one row (a request is
                  admitted once), more than one ARRIVE or more than one
                  FINISH row, or an ARRIVE or DECODE row with a later
                  timestamp than the id's FINISH (a finished request
                  neither arrives nor produces output again; rows of its
                  FINISH instant may come in any order).
   The first three are checked together and the message names the lowest
   failing row and its kind; TRE_ESTATE is checked only when they pass
   (the lowest failing row, or the smallest trace and id in error).
   The id checks allocate temporary device memory: one bit per id up to the
   largest admitted id of each trace, then 4 bytes and one bit per id up to
   the largest ARRIVE or FINISH id (at most 256 MiB at a time, or one
   trace's tables if larger), freed before the call returns. Without
   TRE_VALIDATE, events that break these rules give unspecified results,
   never an access outside the columns, outputs or workspace. The
   handle owns small device tables (offsets, tick list); free it with
   tre_free_events. */
#define TRE_VALIDATE 1u
int tre_load_events(const int64_t* ts, const uint8_t* model, const uint32_t* req,
                    const uint8_t* type, const uint16_t* tokens, const int64_t* trace_off,
                    uint32_t n_traces, const tre_trace_cfg* cfg, uint32_t flags, void* stream,
                    tre_events** out);

/* Release a handle (NULL is a no-op). Does not touch the event columns. */
void tre_free_events(tre_events* ev);

int tre_events_info(const tre_events* ev, tre_info* info);

/* Check a profile table ([n_traces][n_models], device) and a scenario table
   ([n_scenarios], device, may be NULL when n_scenarios is 0) against the
   requirements above and the budget (sum of r_init <= budget per trace).
   Synchronous. */
int tre_check_params(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                     uint32_t n_scenarios);

/* Workspace bytes for tre_sweep with n_scenarios scenarios (0 for the other
   calls). */
int tre_workspace_size(const tre_events* ev, uint32_t n_scenarios, size_t* bytes);

/* Steps a1-a4: per (trace, model, window) tallies, active / waiting
   integrals and smoothed TSS. For each model the raw ratio of Eq. (1) with
   rates in tokens/s, A and W the window time averages and a floor of one
   request is evaluated as
     num = w_p*P; num = num + D; num = num*1000;
     q = w_q*W_int; den = A_int + q; if (den < window_ms) den = window_ms;
     raw = num/den
   (all fp64), then S = alpha*raw + (1-alpha)*S_prev as t1 = alpha*raw,
   t2 = (1-alpha)*S_prev, S = t1 + t2; an idle window holds S; the first
   non-idle window sets S = raw. prof: device [n_traces][n_models]. */
int tre_eval_tss(const tre_events* ev, const tre_profile* prof, const tre_tss_out* out,
                 void* stream);

/* Steps a5-a8 for n_scenarios scenarios over per-cell smoothed TSS and
   flags produced by tre_eval_tss (device, [n_traces][n_windows][n_models]).
   At each tick window: Z = S/(theta*theta_scale) (+inf when idle or not
   initialised); critical Z < tau_crit, surplus Z > tau_surplus. If a model
   is critical: at a fast tick rescue (receivers = critical models),
   otherwise no action. Else at a slow tick rebalance (receivers = Z < 1).
   Up to max_moves greedy moves: receiver = argmin Z over unused eligible
   models; source = idle budget if any, else argmax Z over unused surplus
   models, else over unused nominal models, with R > r_min and Z above the
   receiver's; no source ends the tick; ties go to the lowest model index.
   sc: device [n_scenarios]. */
int tre_rebalance(const tre_events* ev, const tre_profile* prof, const double* tss64,
                  const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                  const tre_ctl_out* out, void* stream);

/* Steps a1-a8 in one call: the smoothed TSS is kept only at tick windows
   (in the workspace) and fed to the control replay. Outputs as
   tre_rebalance; tss32 (device [n_traces][n_windows][n_models]) may be
   NULL. ws: device workspace of at least tre_workspace_size bytes. */
int tre_sweep(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
              uint32_t n_scenarios, const tre_ctl_out* out, float* tss32, void* ws,
              size_t ws_bytes, void* stream);

/* tre_sweep for callers that cannot allocate device memory (code under
   HIP graph capture, tight serving loops, harnesses that forbid
   hipMalloc): the same results as tre_sweep, with the sweep's scratch in a
   static device array of TRE_NOALLOC_SCRATCH_BYTES that each GPU holds
   from the first call on it until the process ends. The call allocates
   nothing (no hipMalloc or hipFree, no event objects: tre_set_timing does
   not record it). Returns TRE_ENOMEM, launching nothing, when the sweep
   needs more scratch than that (tre_workspace_size bytes: 8 per trace,
   tick and model). Every call on one GPU shares its array: calls that
   overlap on one GPU (other streams, other threads) race and give
   unspecified results; calls in order on one stream are safe. */
#define TRE_NOALLOC_SCRATCH_BYTES (64u << 20)
int tre_sweep_noalloc(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                      uint32_t n_scenarios, const tre_ctl_out* out, float* tss32, void* stream);

/* ------------------------------------------------------- actuation model
 * Optional model of how a decided transition is carried out (Sections
 * "Dual-Speed Control", "Bounded Pairwise Transfer", "System Boundary and
 * Replica State"; the paper measures seconds for sleep and wake):
 *   - cfg.budget counts GPUs and a replica of model m holds footprint[m]
 *     GPUs (NULL: 1 each); idle GPUs = budget - GPUs of routable, waking and
 *     draining replicas;
 *   - idle capacity: if at least g_r GPUs are idle the receiver wakes a
 *     replica on them; it is routable wake_ms later;
 *   - donor release: the donor's replica stops being routable at once
 *     (hidden while it drains and sleeps, sleep_ms); its GPUs reach the
 *     receiver when the sleep completes and the receiver's wake starts then;
 *     a shortfall g_r - g_d is taken from the idle GPUs at the move (a donor
 *     qualifies only if enough are idle), an excess returns to them after the
 *     sleep;
 *   - a model with a transition in flight is neither receiver nor donor (a
 *     transfer in progress is not pre-empted);
 *   - veto (NULL: none): [n_traces][n_ticks] masks, bit m set when the
 *     donor-side release guard refuses model m at that tick;
 *   - delays are rounded up to whole windows; a transition completing at the
 *     end of window u counts from window u + 1 (routable replicas, idle GPUs
 *     for the next tick); r_final counts transitions completing by the end of
 *     the last window.
 * With zero delays, unit footprints and no vetoes the results equal those of
 * the calls without the model. footprint and veto are device memory. */
typedef struct {
  int64_t wake_ms;
  int64_t sleep_ms;
  const int32_t* footprint;  /* device [n_traces][n_models], >= 1, or NULL */
  const uint64_t* veto;      /* device [n_traces][n_ticks], or NULL        */
} tre_actuation;

/* Check an actuation model against a profile table (device): footprints in
   1 .. budget and the initial replicas' GPUs within the budget per trace.
   Synchronous. */
int tre_check_actuation(const tre_events* ev, const tre_profile* prof, const tre_actuation* act);

/* tre_rebalance and tre_sweep with the actuation model (act: host, read
   during the call). */
int tre_rebalance_act(const tre_events* ev, const tre_profile* prof, const double* tss64,
                      const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                      const tre_actuation* act, const tre_ctl_out* out, void* stream);
int tre_sweep_act(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                  uint32_t n_scenarios, const tre_actuation* act, const tre_ctl_out* out,
                  float* tss32, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------ calibration sweep
 * Per-request latencies, per-window SLO attainment and the fit of each
 * model's healthy boundary theta (Section "Smoothing, Normalization, and
 * Calibration": theta_m is the smallest smoothed TSS that still achieves the
 * target SLO reliability; SLOs are stated on TTFT, TPOT and E2E latency as
 * tail percentiles):
 *   - a request's record is joined from the events with its id (the
 *     handle's req column, ids below req_cap): its first ARRIVE (time,
 *     model), first DECODE and first FINISH events and the sum of its
 *     DECODE tokens (below 2^32); ids >= req_cap are ignored and counted;
 *   - a request is judged when all three events are in its trace (requests
 *     cut off by the end are censored): TTFT = t(first DECODE) - t(ARRIVE),
 *     E2E = t(FINISH) - t(ARRIVE), TPOT = (t(FINISH) - t(first DECODE)) /
 *     (DECODE tokens after the first DECODE event) when that count is
 *     positive; it meets the SLO when TTFT <= ttft_ms, E2E <= e2e_ms and
 *     (no TPOT or TPOT <= tpot_ms), compared in fp64;
 *   - it counts in the window of its arrival; a window with judged >= 1 is
 *     healthy when ok >= attain_q * judged (fp64);
 *   - candidates of (trace, model): windows with judged >= 1 whose TSS is
 *     initialised and not idle. theta = the smallest candidate S such that,
 *     over the candidates with S >= theta, healthy >= reliability * count
 *     (fp64); +inf when none qualifies;
 *   - the ordering check (RQ1 asks that TSS follow the SLO-health ordering):
 *     over the pairs of candidates of one (trace, model) with different S,
 *     one healthy and one not, `concordant` counts those whose larger S is
 *     the healthy window's and `discordant` the others; pairs of equal S are
 *     in neither (healthy * unhealthy - concordant - discordant of them). */
typedef struct {
  double ttft_ms, tpot_ms, e2e_ms;  /* bounds; +inf disables one            */
  double attain_q;                  /* window healthy when ok >= q * judged */
  double reliability;               /* target healthy fraction above theta  */
} tre_slo;                          /* 40 bytes */

typedef struct {
  double theta;                     /* +inf when no candidate qualifies     */
  uint32_t n_cand, n_healthy;       /* candidate windows, healthy ones      */
  uint32_t n_above, healthy_above;  /* candidates with S >= theta, healthy  */
  uint32_t concordant;  /* candidate pairs whose higher S is the healthy one
                           (tre_calib_order; 0 from tre_calibrate)        */
  uint32_t discordant;  /* ... whose higher S is the unhealthy one        */
} tre_fit;                          /* 32 bytes */

#define TRE_REQ_ARRIVED 1   /* an ARRIVE event was seen                  */
#define TRE_REQ_COMPLETE 2  /* judged: ARRIVE, DECODE and FINISH present */
#define TRE_REQ_TPOT 4      /* tpot_ms defined                           */
#define TRE_REQ_OK 8        /* met its model's SLO                       */
typedef struct {
  uint32_t ttft_ms, e2e_ms;         /* valid with TRE_REQ_COMPLETE          */
  double tpot_ms;                   /* valid with TRE_REQ_TPOT              */
  uint8_t model;                    /* 0xFF without an ARRIVE               */
  uint8_t flags;
  uint8_t pad[6];
} tre_req_latency;                  /* 24 bytes */

/* Workspace bytes of tre_calibrate: 256, two lists of 4 + 4 * n_traces
   bytes each rounded up to 256, and 16 per request slot and trace. */
int tre_calib_workspace_size(const tre_events* ev, uint32_t req_cap, size_t* bytes);

/* The calibration sweep over the handle's traces (device pointers):
     slo     [n_traces][n_models] (any values; comparisons follow IEEE);
     tss64, flags  [n_traces][n_windows][n_models] from tre_eval_tss;
     counts  [n_traces][n_models][n_windows] (16-byte aligned) receives
             judged << 16 | ok per window of arrival;
     fit     [n_traces][n_models];
     reqs    [n_traces][req_cap] per-request latencies, or NULL;
     n_bad_ids  one uint64: events whose id is >= req_cap, or NULL.
   The handle needs its req column; at most 16384 windows (TRE_ERANGE);
   req_cap at most 2^31 (TRE_ERANGE).
   Request lifecycle (checked by tre_load_events with TRE_VALIDATE and a req
   column, TRE_ESTATE): per trace, a request id has at most one ARRIVE row
   and at most one FINISH row, and no ARRIVE or DECODE row with a later
   timestamp than its FINISH (rows of one instant may come in any order).
   Events that break it give unspecified results, never an access out of
   bounds.
   Each trace is streamed once by one workgroup that keeps its requests in
   flight in LDS. A trace with more requests in flight than that table
   holds (or more than 256 FINISH rows at one instant) is redone with a
   table twice as large, and a trace that overflows that one by request-id
   records in the workspace; after the call completes, the uint32 at byte
   256 of ws counts the traces redone with the larger table and the uint32
   at byte 256 + (4 + 4 * n_traces rounded up to 256) those redone by
   records (diagnostics; the results do not depend on the path).
   ws: 16-byte aligned device workspace of tre_calib_workspace_size bytes.
   Enqueued on `stream`. */
int tre_calibrate(const tre_events* ev, const tre_slo* slo, const double* tss64,
                  const uint8_t* flags, uint32_t req_cap, uint32_t* counts, tre_fit* fit,
                  tre_req_latency* reqs, uint64_t* n_bad_ids, void* ws, size_t ws_bytes,
                  void* stream);

/* The fits of tre_calibrate again, with the ordering check: concordant and
   discordant filled (tre_calibrate leaves them 0). counts are the per-window
   counts tre_calibrate wrote for the same handle, SLOs and TSS (the window
   health comes from them); the other arguments as tre_calibrate. Costs a full
   sort of each (trace, model)'s candidate windows where the buckets of the
   fit's histogram that hold both healthy and unhealthy windows have more than
   1024 of them. Enqueued on `stream`. */
int tre_calib_order(const tre_events* ev, const tre_slo* slo, const double* tss64, const uint8_t* flags,
                    const uint32_t* counts, tre_fit* fit, void* stream);

/* ---------------------------------------------------- closed-loop replay
 * The requests of each trace are served by each model's routable replicas,
 * the rules above move replicas at tick windows, and the TSS the controller
 * reads comes from the events this service produces (Sections "Dual-Speed
 * Control", "Bounded Pairwise Transfer": after each transition the
 * controller observes the result at the next tick; Section "System
 * Boundary and Replica State": only routable replicas take new requests, a
 * hidden replica drains):
 *   - a routable replica of model m has slots_per_replica slots; requests of
 *     a model start in arrival order on the slot that frees first (lowest
 *     index on ties) at max(arrival, its free time);
 *   - a prompt chunk of c tokens takes ceil(c * prefill_us / 1000) ms on its
 *     slot, an output chunk ceil(c * decode_us / 1000) ms; the events are
 *     those of the traces (ARRIVE, one PREFILL per prompt chunk at its start
 *     with ADMIT on the first, one DECODE per output chunk at its end, FINISH
 *     at the last), dropped at or after the end of the trace;
 *   - TSS per window, Eq. (1) and the smoothing as in tre_eval_tss;
 *   - at each tick the rules of tre_rebalance, with receivers below r_cap
 *     replicas; a move acts from the end of its window: the receiver gains
 *     slots free from then, the donor's replica stops taking requests and its
 *     slots that free first are removed (requests on them finish);
 *   - a request whose FINISH lies in the trace is judged against its
 *     model's SLO as in tre_calibrate. */
typedef struct {
  uint32_t prefill_us;  /* per prompt token on one slot */
  uint32_t decode_us;   /* per output token on one slot */
} tre_service;

typedef struct {
  const int64_t* arrival_ms;   /* device [n_requests], ms from trace start      */
  const uint16_t* prompt;      /* device [n_requests], prompt tokens            */
  const uint16_t* output;      /* device [n_requests], output tokens (>= 1)      */
  const int64_t* req_off;      /* device [n_traces * n_models + 1]: requests of
                                  (trace t, model m) are [req_off[t*M+m],
                                  req_off[t*M+m+1]), arrivals non-decreasing    */
  const tre_service* service;  /* device [n_traces][n_models]                   */
  const tre_slo* slo;          /* device [n_traces][n_models]                   */
  int32_t slots_per_replica;
  int32_t r_cap;               /* receivers must hold fewer replicas            */
  int32_t prefill_chunk;       /* prompt tokens per PREFILL event               */
  int32_t decode_chunk;        /* output tokens per DECODE event                */
  uint32_t max_prompt, max_output;         /* bounds over the table (host)      */
  uint32_t max_prefill_us, max_decode_us;  /* bounds over service (host)        */
  uint32_t max_replicas;       /* most replicas holding slots at once in one
                                  scenario, a bound the caller declares (0:
                                  none); it sizes the slot pool below       */
} tre_loop_requests;

typedef struct {
  uint32_t n_arrived, n_started, n_done, n_ok;  /* n_done: judged requests */
  int64_t e2e_sum, e2e_max;                     /* over judged requests, ms */
} tre_loop_stats;                               /* 32 bytes */

/* Workspace bytes of tre_loop: 256, plus per scenario and model a ring of
   16-byte tallies of future windows, its length the power of two that
   covers the longest service the declared bounds allow (in windows, + 2),
   plus per scenario the words of its slot-heap pool (below) as scratch.
   The pool holds min(budget, n_models * min(r_cap, budget), max_replicas
   when nonzero) * slots_per_replica + 4 x n_models words (6 x n_models when
   slots_per_replica is not a multiple of 4), rounded up to 4; TRE_EINVAL when 4
   bytes x (that pool + 44 x n_models) exceed the 160 KiB of LDS one
   scenario's workgroup may use; TRE_ERANGE when duration_ms plus that
   longest service reaches 2^31 ms. */
int tre_loop_workspace_size(const tre_trace_cfg* cfg, const tre_loop_requests* rq, uint32_t n_scenarios,
                            size_t* bytes);

/* Closed-loop replay of n_scenarios scenarios (device sc, as tre_rebalance)
   over the request tables (rq: host struct of device pointers) with the
   profiles prof (device [n_traces][n_models]) and cfg (host; budget in
   replicas). Outputs as tre_rebalance, plus stats (device
   [n_scenarios][n_models]) and optionally the per-window smoothed TSS
   (device [n_scenarios][n_windows][n_models], or NULL). r_init must lie in
   [0, min(r_cap, budget)] with the sum within the budget, and req_off must
   index the request arrays; other inputs give unspecified results (never an
   access outside them). Requests beyond the declared bounds, or more
   replicas at once than max_replicas, give unspecified results too; the
   workspace's first 8 bytes then count the events dropped plus the
   replicas' slots the pool could not hold (0 otherwise). Enqueued on
   `stream`. */
int tre_loop(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq, const tre_profile* prof,
             const tre_scenario* sc, uint32_t n_scenarios, const tre_ctl_out* out, tre_loop_stats* stats,
             double* tss64, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------- stage-aware shares */
/* Flags of tre_stage_tss, one byte per cell. */
#define TRE_STAGE_P_IDLE 1 /* no prompt tokens and nothing waiting in the window */
#define TRE_STAGE_P_INIT 2 /* prefill share initialised                        */
#define TRE_STAGE_D_IDLE 4 /* no output tokens and nothing active in the window */
#define TRE_STAGE_D_INIT 8 /* decode share initialised                          */

/* Stage-aware service shares (paper, Sections "Discussion" and "Future
   Work": for disaggregated prefill / decode serving the scalar score becomes
   a per-stage vector; the paper gives no formula, and these are the two
   parts of Eq. (1), each with its one-request floor):
     prefill  raw_p = 1000 * w_p * P / max(w_q * W_int, window_ms)
     decode   raw_d = 1000 * D / max(A_int, window_ms)
   evaluated in that operation order in binary64, then smoothed per stage as
   the scalar share (Section "Smoothing, Normalization, and Calibration"): a
   stage idle in a window (its tokens and its demand integral both zero)
   holds its value, its first busy window sets it to the raw ratio, later
   ones give alpha * raw + (1 - alpha) * S_prev. Where neither floor binds,
   Eq. (1)'s raw ratio is the mediant of raw_p and raw_d.
   tallies: the prefill, decode, a_int and w_int outputs of tre_eval_tss for
   the same handle and profiles (device, [n_traces][n_windows][n_models]; the
   other fields are ignored). Outputs, each optional but not all NULL:
   stage64 (device [n_traces][n_windows][n_models][2] binary64, prefill then
   decode; 16-byte aligned), stage32 (the same rounded to binary32; 8-byte
   aligned), flags (device [n_traces][n_windows][n_models], TRE_STAGE_*).
   Enqueued on `stream`. */
int tre_stage_tss(const tre_events* ev, const tre_profile* prof, const tre_tss_out* tallies, double* stage64,
                  float* stage32, uint8_t* flags, void* stream);

/* The same shares computed straight from the events (the tallies never
   leave the chip): tre_eval_tss's pass over each trace with the two stage
   ratios staged beside Eq. (1)'s and smoothed in the same chain. Outputs as
   tre_stage_tss (each optional but not all NULL, same layout, alignment
   and values bit for bit). Enqueued on `stream`. */
int tre_eval_stage(const tre_events* ev, const tre_profile* prof, double* stage64, float* stage32,
                   uint8_t* flags, void* stream);

/* tre_loop with the actuation model (paper, Sections "System Boundary and
   Replica State" and "Bounded Pairwise Transfer": transitions hide, drain,
   sleep and wake replicas, budget-feasible in GPU footprints; act: host,
   read during the call; its footprint and veto tables device
   [n_traces][n_models] and [n_traces][n_ticks], either NULL). The budget
   then counts GPUs, a replica of model
   m holding footprint[m] (1 to budget); delays are whole windows rounded up
   from wake_ms / sleep_ms, as tre_rebalance_act. A woken replica's slots
   are free from the start of the window after its wake completes; a
   donor's replica stops taking requests at the move (its slots that free
   first leave) and its GPUs reach the receiver when its sleep completes,
   when the receiver's wake starts; a model with a transition in flight is
   neither receiver nor donor; veto bit m at a tick keeps model m from
   releasing. r_final counts wakes completing by the end of the last
   window. With zero delays, unit footprints and no vetoes the outputs
   equal tre_loop's. Footprints outside 1 .. budget or initial replicas'
   GPUs beyond the budget give unspecified results (never an access outside
   the buffers). Same workspace as tre_loop; TRE_EINVAL also for a NULL act
   or a negative delay. */
int tre_loop_act(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq, const tre_profile* prof,
                 const tre_scenario* sc, uint32_t n_scenarios, const tre_actuation* act, const tre_ctl_out* out,
                 tre_loop_stats* stats, double* tss64, void* ws, size_t ws_bytes, void* stream);

/* Kernel timing (HIP events recorded around each launch on its stream).
   tre_set_timing(1) starts recording; tre_kernel_time waits for the
   recorded launches of `kernel` ("tss_stream", "rebalance", "validate",
   "calib_fill", "calib_stream", "calib_fallback" (the second stream tier
   and the chunked path together), "calib_fit", "calib_order",
   "loop_replay", "stage_tss")
   and returns their total milliseconds and count, then forgets them. */
int tre_set_timing(int enable);
int tre_kernel_time(const char* kernel, double* total_ms, uint64_t* launches);

#ifdef __cplusplus
}
#endif
#endif /* TRE_H */
