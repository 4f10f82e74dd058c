// loop.hip - the closed-loop replay on MI355X (gfx950): each model's
// requests are served on the slots of its routable replicas, the controller's
// moves change those replicas at tick windows, and the TSS it reads comes
// from the events that this service produces.
//
// Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE). The rules
// at each tick are those of Sections "Dual-Speed Control" and "Bounded
// Pairwise Transfer" (Eq. (2) regions, cadence, Eq. (3) receiver, idle
// capacity before surplus before nominal donors); only routable replicas
// serve new requests and a hidden replica drains (Section "System Boundary
// and Replica State"); after each transition the controller observes the
// resulting service at the next tick. TSS per window is Eq. (1) with the
// smoothing of Section "Smoothing, Normalization, and Calibration".
//
// Kernel
//   loop_replay  one wave per scenario, lane = model, windows in order. A
//                lane keeps its model's slot free times and a ring of the
//                future windows' tallies (prompt and output tokens, finishes
//                of requests already started) in the workspace; per window
//                it takes its arrivals, starts requests FCFS on the slot that
//                frees first while the start falls in the window, writes each
//                started request's events into the ring, reads the window's
//                tallies and evaluates Eq. (1) and the smoothing in fp64; at
//                a tick the wave decides the moves (ballots over lanes) and
//                the receiver and donor lanes change their slots.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "tre.h"
#include "tre_internal.h"

#pragma clang fp contract(off)

using tre_internal::fail;
using tre_internal::LaunchTimer;

namespace {

constexpr int kLoopWaves = 4;  // scenarios per workgroup

struct RingCell {         // tallies of one future window of one model
  uint32_t p, d;          // prompt / output tokens of its PREFILL / DECODE events
  uint32_t n_fin, pad;    // FINISH events in it
  uint64_t e_fin;         // sum over them of (window end - finish time)
};

struct LoopParams {
  const int64_t* arrival;
  const uint16_t* prompt;
  const uint16_t* output;
  const int64_t* req_off;
  const tre_service* svc;
  const tre_slo* slo;
  const tre_profile* prof;
  const tre_scenario* sc;
  tre_move* moves;
  uint32_t* n_moves;
  int32_t* r_final;
  int64_t* r_windows;
  tre_loop_stats* stats;
  double* tss64;                // [scenario][window][model] or NULL
  int64_t* slots;               // [scenario][model][slot_cap]
  RingCell* ring;               // [scenario][model][ring_len]
  unsigned long long* overflow; // events beyond the ring (declared bounds exceeded)
  uint32_t move_cap;
  uint32_t n_sc;
  uint32_t n_traces;
  int32_t M;
  int32_t budget;
  int32_t spr;
  int32_t r_cap;
  int32_t pchunk;
  int32_t dchunk;
  int32_t slot_cap;
  uint32_t ring_len;            // power of two
  int64_t window_ms;
  int64_t duration_ms;
  int64_t n_windows;
  int64_t fast_w, slow_w;       // periods in windows
};

__device__ __forceinline__ int64_t ceil_ms(int64_t tokens, uint32_t us) {
  return (tokens * (int64_t)us + 999) / 1000;
}

__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }

// lowest lane with the smallest (kMax false) or largest Z among `cand`;
// -1 if none. Z >= 0 or +inf, never NaN, so bit patterns order like values.
template <bool kMax>
__device__ __forceinline__ int pick_lane(unsigned long long cand, double Z, int lane) {
  if (!cand) return -1;
  const bool c = (cand >> lane) & 1ull;
  uint64_t key = c ? dbits(Z) : (kMax ? 0ull : ~0ull);
  int idx = c ? lane : 64;
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t ok = ((uint64_t)(uint32_t)__shfl_xor((int)(key >> 32), o) << 32) |
                        (uint32_t)__shfl_xor((int)(uint32_t)key, o);
    const int oi = __shfl_xor(idx, o);
    const bool better = kMax ? (ok > key || (ok == key && oi < idx)) : (ok < key || (ok == key && oi < idx));
    if (better) {
      key = ok;
      idx = oi;
    }
  }
  return idx < 64 ? idx : -1;
}

__device__ __forceinline__ double lane_f64(double x, int l) {
  const uint64_t b = dbits(x);
  const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)b, l), hi = (uint32_t)__shfl((int)(uint32_t)(b >> 32), l);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__global__ void zero_u64(unsigned long long* x) { *x = 0ull; }

__global__ __launch_bounds__(64 * kLoopWaves) void loop_replay(LoopParams p) {
  const int lane = threadIdx.x & 63;
  const uint32_t s = blockIdx.x * kLoopWaves + (threadIdx.x >> 6);
  if (s >= p.n_sc) return;  // whole wave
  const int M = p.M;
  const bool act = lane < M;
  const int mc = act ? lane : 0;
  const tre_scenario sc = p.sc[s];
  const uint32_t t = sc.trace < p.n_traces ? sc.trace : 0;
  const uint64_t tm = (uint64_t)t * M + mc;
  const tre_profile pr = p.prof[tm];
  const tre_slo sl = p.slo[tm];
  const tre_service sv = p.svc[tm];
  const double theta_eff = pr.theta * sc.theta_scale;
  const double tau_c = sc.tau_crit_override >= 0.0 ? sc.tau_crit_override : pr.tau_crit;
  const int64_t W = p.window_ms, dur = p.duration_ms;
  const uint32_t L = p.ring_len;
  // initial replicas within the slot array (min(r_cap, budget) replicas)
  const int r_hi = p.slot_cap / p.spr;
  int R = act ? (pr.r_init < 0 ? 0 : (pr.r_init > r_hi ? r_hi : pr.r_init)) : 0;
  int rsum = R;
  for (int o = 32; o > 0; o >>= 1) rsum += __shfl_xor(rsum, o);
  int pool = p.budget - rsum;
  int64_t* slot = p.slots + ((uint64_t)s * M + mc) * p.slot_cap;
  RingCell* ring = p.ring + ((uint64_t)s * M + mc) * L;
  if (act) {
    for (uint32_t i = 0; i < L; ++i) ring[i] = RingCell{0u, 0u, 0u, 0u, 0ull};
    for (int i = 0; i < R * p.spr; ++i) slot[i] = 0;
  }
  const int64_t q1 = act ? p.req_off[tm + 1] : 0;
  int64_t next_arr = act ? p.req_off[tm] : 0, next_start = next_arr;
  int64_t cA = 0, cW = 0;  // active / waiting requests at the current window's start
  double S = 0.0;
  bool init = false;
  uint32_t n_arr = 0, n_start = 0, n_done = 0, n_ok = 0;
  int64_t e2e_sum = 0, e2e_max = 0, rw = 0;
  unsigned overflow = 0;
  uint32_t nm = 0;
  const unsigned long long live = __ballot(act);

  for (int64_t w = 0; w < p.n_windows; ++w) {
    const int64_t w_end = (w + 1) * W;
    uint32_t P = 0, D = 0;
    int64_t eA = 0, eW = 0, dA = 0, dW = 0;
    bool idle = true;
    if (act) {
      RingCell* rc = ring + (w & (L - 1));
      P = rc->p;
      D = rc->d;
      dA -= rc->n_fin;
      eA -= (int64_t)rc->e_fin;
      *rc = RingCell{0u, 0u, 0u, 0u, 0ull};
      // arrivals: a request waits from its arrival
      while (next_arr < q1 && p.arrival[next_arr] < w_end) {
        eW += w_end - p.arrival[next_arr];
        dW += 1;
        ++n_arr;
        ++next_arr;
      }
      // starts, in arrival order, on the slot that frees first
      const int ns = R * p.spr;
      while (next_start < next_arr && ns > 0) {
        int best = 0;
        int64_t bf = slot[0];
        for (int k = 1; k < ns; ++k) {
          const int64_t f = slot[k];
          if (f < bf) {
            bf = f;
            best = k;
          }
        }
        const int64_t a = p.arrival[next_start];
        const int64_t st = a > bf ? a : bf;
        if (st >= w_end) break;  // capacity may change at the window's end
        // admission: waiting -> active
        eW -= w_end - st;
        dW -= 1;
        eA += w_end - st;
        dA += 1;
        int64_t tt = st;
        int64_t left = p.prompt[next_start];
        while (left > 0) {
          const int64_t ch = left < p.pchunk ? left : p.pchunk;
          if (tt < dur) {
            const int64_t wf = tt / W;
            if (wf == w) P += (uint32_t)ch;
            else if (wf - w < (int64_t)L) ring[wf & (L - 1)].p += (uint32_t)ch;
            else ++overflow;
          }
          tt += ceil_ms(ch, sv.prefill_us);
          left -= ch;
        }
        const int64_t out_tok = p.output[next_start];
        left = out_tok;
        int64_t t_first = -1, first_ch = 0;
        while (left > 0) {
          const int64_t ch = left < p.dchunk ? left : p.dchunk;
          tt += ceil_ms(ch, sv.decode_us);
          if (t_first < 0) {
            t_first = tt;
            first_ch = ch;
          }
          if (tt < dur) {
            const int64_t wf = tt / W;
            if (wf == w) D += (uint32_t)ch;
            else if (wf - w < (int64_t)L) ring[wf & (L - 1)].d += (uint32_t)ch;
            else ++overflow;
          }
          left -= ch;
        }
        if (tt < dur) {  // FINISH: active -> gone
          const int64_t wf = tt / W;
          if (wf == w) {
            eA -= w_end - tt;
            dA -= 1;
          } else if (wf - w < (int64_t)L) {
            RingCell& c = ring[wf & (L - 1)];
            c.n_fin += 1;
            c.e_fin += (uint64_t)((wf + 1) * W - tt);
          } else {
            ++overflow;
          }
          if (t_first >= 0) {  // judged as in the calibration sweep
            const int64_t ttft = t_first - a, e2e = tt - a, after = out_tok - first_ch;
            bool good = (double)ttft <= sl.ttft_ms && (double)e2e <= sl.e2e_ms;
            if (after > 0) good = good && (double)(tt - t_first) / (double)after <= sl.tpot_ms;
            ++n_done;
            n_ok += good ? 1u : 0u;
            e2e_sum += e2e;
            e2e_max = e2e > e2e_max ? e2e : e2e_max;
          }
        }
        slot[best] = tt;
        ++n_start;
        ++next_start;
      }
      // the window's tallies, Eq. (1) and the smoothing
      const int64_t A_int = W * cA + eA, W_int = W * cW + eW;
      cA += dA;
      cW += dW;
      idle = P == 0 && D == 0 && A_int == 0 && W_int == 0;
      if (!idle) {
        double num = pr.w_p * (double)P;
        num = num + (double)D;
        num = num * 1000.0;
        const double q = pr.w_q * (double)W_int;
        double den = (double)A_int + q;
        if (den < (double)W) den = (double)W;
        const double raw = num / den;
        if (init) {
          const double t1 = pr.alpha * raw;
          const double t2 = (1.0 - pr.alpha) * S;
          S = t1 + t2;
        } else {
          S = raw;
          init = true;
        }
      }
      if (p.tss64) p.tss64[((uint64_t)s * p.n_windows + w) * M + lane] = S;
      rw += R;
    }
    // ---- tick: the controller's rules on this window's TSS
    const bool fast = (w + 1) % p.fast_w == 0, slow = (w + 1) % p.slow_w == 0;
    if (!fast && !slow) continue;
    const double Z = (act && !idle && init) ? S / theta_eff : INFINITY;  // Eq. (2)
    const unsigned long long crit = __ballot(act && Z < tau_c);
    unsigned long long ok;
    int path;
    if (crit) {
      if (!fast) continue;  // rescue pending: rebalancing defers
      path = TRE_PATH_RESCUE;
      ok = crit;
    } else if (slow) {
      path = TRE_PATH_REBALANCE;
      ok = __ballot(act && Z < 1.0);
    } else {
      continue;
    }
    const unsigned long long sur = __ballot(act && Z > pr.tau_surplus);
    unsigned long long used = 0ull;
    for (uint32_t k = 0; k < sc.max_moves; ++k) {
      const int r = pick_lane<false>(ok & ~used & __ballot(act && R < p.r_cap), Z, lane);  // Eq. (3)
      if (r < 0) break;
      int d;
      if (pool > 0) {
        pool -= 1;
        d = TRE_DONOR_POOL;
      } else {
        const double Zr = lane_f64(Z, r);
        const unsigned long long cd = __ballot(act && R > pr.r_min && Z > Zr) & ~crit & ~used & ~(1ull << r) & live;
        d = pick_lane<true>(cd & sur, Z, lane);
        if (d < 0) d = pick_lane<true>(cd & ~sur, Z, lane);
        if (d < 0) break;
        used |= 1ull << d;
        if (lane == d) {  // the replica's slots that free first leave
          for (int q = 0; q < p.spr; ++q) {
            const int ns = R * p.spr - q;
            if (ns <= 0) break;
            int lo = 0;
            for (int x = 1; x < ns; ++x)
              if (slot[x] < slot[lo]) lo = x;
            for (int x = lo; x + 1 < ns; ++x) slot[x] = slot[x + 1];
          }
          if (R > 0) R -= 1;
        }
      }
      used |= 1ull << r;
      if (lane == r) {  // the new replica's slots are free from the window's end
        for (int q = 0; q < p.spr; ++q) slot[R * p.spr + q] = w_end;
        R += 1;
      }
      if (lane == 0 && nm < p.move_cap) {
        tre_move mv;
        mv.window = (uint32_t)w;
        mv.path = (uint8_t)path;
        mv.receiver = (uint8_t)r;
        mv.donor = (uint8_t)d;
        mv.pad = 0;
        p.moves[(uint64_t)s * p.move_cap + nm] = mv;
      }
      ++nm;
    }
  }
  if (act) {
    p.r_final[(uint64_t)s * M + lane] = R;
    p.r_windows[(uint64_t)s * M + lane] = rw;
    tre_loop_stats st;
    st.n_arrived = n_arr;
    st.n_started = n_start;
    st.n_done = n_done;
    st.n_ok = n_ok;
    st.e2e_sum = e2e_sum;
    st.e2e_max = e2e_max;
    p.stats[(uint64_t)s * M + lane] = st;
  }
  if (lane == 0) p.n_moves[s] = nm;
  for (int o = 32; o > 0; o >>= 1) overflow += __shfl_xor(overflow, o);
  if (lane == 0 && overflow) atomicAdd(p.overflow, (unsigned long long)overflow);
}

// longest service of any request allowed by the declared bounds (ms)
int64_t max_service_ms(const tre_loop_requests* rq) {
  const int64_t np = (rq->max_prompt + rq->prefill_chunk - 1) / rq->prefill_chunk;
  const int64_t nd = (rq->max_output + rq->decode_chunk - 1) / rq->decode_chunk;
  return np * (((int64_t)rq->prefill_chunk * rq->max_prefill_us + 999) / 1000) +
         nd * (((int64_t)rq->decode_chunk * rq->max_decode_us + 999) / 1000);
}

uint32_t ring_len(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  const int64_t span = max_service_ms(rq) / cfg->window_ms + 2;
  uint32_t L = 2;
  while ((int64_t)L < span) L <<= 1;
  return L;
}

int slot_cap(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  return (rq->r_cap < cfg->budget ? rq->r_cap : cfg->budget) * rq->slots_per_replica;
}

int check_loop_args(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  if (!cfg || !rq) return fail(TRE_EINVAL, "tre_loop: NULL cfg or request table");
  if (cfg->window_ms < 1 || cfg->duration_ms <= 0 || cfg->duration_ms % cfg->window_ms ||
      cfg->fast_period_ms <= 0 || cfg->slow_period_ms <= 0 || cfg->fast_period_ms % cfg->window_ms ||
      cfg->slow_period_ms % cfg->window_ms || cfg->duration_ms >= (1ll << 40))
    return fail(TRE_EINVAL, "tre_loop: bad window, duration or periods");
  if (cfg->n_models < 1 || cfg->n_models > TRE_MAX_MODELS || cfg->budget < 0)
    return fail(TRE_EINVAL, "tre_loop: n_models outside [1, %d] or negative budget", TRE_MAX_MODELS);
  if (rq->slots_per_replica < 1 || rq->r_cap < 1 || rq->prefill_chunk < 1 || rq->decode_chunk < 1)
    return fail(TRE_EINVAL, "tre_loop: slots_per_replica, r_cap and chunks must be positive");
  if (max_service_ms(rq) / cfg->window_ms > (1 << 24))
    return fail(TRE_ERANGE, "tre_loop: a request may span more than 2^24 windows");
  return TRE_OK;
}

}  // namespace

// --------------------------------------------------------------- host ABI
extern "C" int tre_loop_workspace_size(const tre_trace_cfg* cfg, const tre_loop_requests* rq,
                                       uint32_t n_scenarios, size_t* bytes) {
  if (!bytes) return fail(TRE_EINVAL, "tre_loop_workspace_size: NULL bytes");
  const int rc = check_loop_args(cfg, rq);
  if (rc) return rc;
  const uint64_t per = (uint64_t)slot_cap(cfg, rq) * 8 + (uint64_t)ring_len(cfg, rq) * sizeof(RingCell);
  *bytes = (size_t)(256 + (uint64_t)n_scenarios * cfg->n_models * per);
  return TRE_OK;
}

extern "C" int tre_loop(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq,
                        const tre_profile* prof, const tre_scenario* sc, uint32_t n_scenarios,
                        const tre_ctl_out* out, tre_loop_stats* stats, double* tss64, void* ws, size_t ws_bytes,
                        void* stream) {
  int rc = check_loop_args(cfg, rq);
  if (rc) return rc;
  if (!prof || !out || !stats || !ws || !rq->arrival_ms || !rq->prompt || !rq->output || !rq->req_off ||
      !rq->service || !rq->slo || (n_scenarios && (!sc || !out->moves || !out->n_moves || !out->r_final ||
                                                   !out->r_windows)))
    return fail(TRE_EINVAL, "tre_loop: NULL argument");
  if (n_traces == 0) return fail(TRE_EINVAL, "tre_loop: no traces");
  if ((uintptr_t)ws & 15) return fail(TRE_EINVAL, "tre_loop: workspace needs 16-byte alignment");
  size_t need = 0;
  tre_loop_workspace_size(cfg, rq, n_scenarios, &need);
  if (ws_bytes < need) return fail(TRE_ENOMEM, "tre_loop: workspace %zu < %zu bytes", ws_bytes, need);
  if (n_scenarios == 0) return TRE_OK;
  hipStream_t st = (hipStream_t)stream;
  const int M = cfg->n_models;
  const uint32_t L = ring_len(cfg, rq);
  const int scap = slot_cap(cfg, rq);
  char* base = (char*)ws;
  unsigned long long* overflow = (unsigned long long*)base;
  int64_t* slots = (int64_t*)(base + 256);
  RingCell* ring = (RingCell*)(base + 256 + (uint64_t)n_scenarios * M * scap * 8);
  hipLaunchKernelGGL(zero_u64, dim3(1), dim3(1), 0, st, overflow);
  LoopParams lp{};
  lp.arrival = rq->arrival_ms;
  lp.prompt = rq->prompt;
  lp.output = rq->output;
  lp.req_off = rq->req_off;
  lp.svc = rq->service;
  lp.slo = rq->slo;
  lp.prof = prof;
  lp.sc = sc;
  lp.moves = out->moves;
  lp.n_moves = out->n_moves;
  lp.r_final = out->r_final;
  lp.r_windows = out->r_windows;
  lp.stats = stats;
  lp.tss64 = tss64;
  lp.slots = slots;
  lp.ring = ring;
  lp.overflow = overflow;
  lp.move_cap = out->move_cap;
  lp.n_sc = n_scenarios;
  lp.n_traces = n_traces;
  lp.M = M;
  lp.budget = cfg->budget;
  lp.spr = rq->slots_per_replica;
  lp.r_cap = rq->r_cap;
  lp.pchunk = rq->prefill_chunk;
  lp.dchunk = rq->decode_chunk;
  lp.slot_cap = scap;
  lp.ring_len = L;
  lp.window_ms = cfg->window_ms;
  lp.duration_ms = cfg->duration_ms;
  lp.n_windows = cfg->duration_ms / cfg->window_ms;
  lp.fast_w = cfg->fast_period_ms / cfg->window_ms;
  lp.slow_w = cfg->slow_period_ms / cfg->window_ms;
  LaunchTimer lt("loop_replay", st);
  hipLaunchKernelGGL(loop_replay, dim3((n_scenarios + kLoopWaves - 1) / kLoopWaves), dim3(64 * kLoopWaves), 0, st,
                     lp);
  lt.done();
  HIP_TRY(hipGetLastError());
  return TRE_OK;
}
