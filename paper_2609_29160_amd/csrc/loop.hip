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
//   loop_replay  one wave per scenario (one workgroup), lane = model,
//                windows in order. Its LDS holds the models' slot heaps
//                (packed in a pool; a tick that moves replicas repacks them
//                into a second pool), a ring of the next kNear windows'
//                tallies (prompt and output tokens, finishes of requests
//                already started), staged requests and the starts recorded
//                for the event pass; tallies further ahead go to a ring in
//                HBM with fire-and-forget atomics and are moved into LDS one
//                window before they can be needed. Per window a lane takes
//                its arrivals and starts requests FCFS on the slot that
//                frees first while the start falls in the window (finish,
//                judging and slot in closed form); the whole wave then adds
//                the recorded starts' PREFILL / DECODE events to the rings,
//                their chunks spread over the lanes; each lane reads its
//                window's tallies and evaluates Eq. (1) and the smoothing in
//                fp64; at a tick the wave decides the moves (ballots over
//                lanes). Which of several equally early slots a request
//                takes, and where a removed slot's place goes, changes no
//                output: only the multiset of free times matters.
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

constexpr int kNear = 4;  // windows ahead whose tallies sit in LDS (power of two)
constexpr int kStage = 4;  // requests per lane staged in LDS for the starts
constexpr int kEnt = 2;    // starts a lane records per pass of the wave's event generation
constexpr uint32_t kNone = 0xffffffffu;
constexpr int64_t kNever = INT64_MAX;
constexpr int32_t kArrNever = INT32_MAX;
constexpr int kLdsMax = 160 * 1024;

// Tallies of one window of one model beyond the LDS ring, in three rings of
// [scenario][ring cell][model]: the output tokens of DECODE events (one add
// per output chunk) and the prompt tokens of PREFILL events in 4-byte cells,
// so that one window's cells of 32 models share one cache line and the few
// dozen windows a scenario is adding into stay in L2; its FINISH events in
// 8-byte cells, count << 32 plus the sum of (window end - finish time) (below
// 2^32, as the LDS ring's 32-bit cell), one add per finishing request.

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
  uint32_t* far_p;              // [scenario][ring_len][model]: prompt tokens
  uint32_t* far_d;              // [scenario][ring_len][model]: output tokens
  unsigned long long* far_f;    // [scenario][ring_len][model]: FINISH count << 32 | sum of time to window end
  uint32_t* scratch;            // [scenario][pool_words]: heaps in transit at a repack
  // the actuation model (the kAct instantiation)
  const int32_t* footprint;     // [trace][M] GPUs per replica, or NULL (1); the budget is then in GPUs
  const uint64_t* veto;         // [trace][n_ticks] donor releases refused, or NULL
  int32_t wake_w, sleep_w;      // whole windows
  int32_t n_ticks;
  unsigned long long* overflow; // declared bounds exceeded: events beyond the ring, replica slots beyond the pool
  uint32_t move_cap;
  uint32_t n_sc;
  uint32_t n_traces;
  int32_t M;
  int32_t budget;
  int32_t spr;
  int32_t r_cap;
  int32_t pchunk;
  int32_t dchunk;
  int32_t pool_words;           // the heap pool: pool_reps * spr + 4 or 6 words per model, multiple of 4
  int32_t pool_reps;            // replicas the pool holds: min(budget, M * r_hi, the declared bound)
  uint32_t wmagic;              // x / window_ms == umulhi(x, wmagic) >> wshift for x < 2^31 (wshift < 0: x)
  int32_t wshift;
  uint32_t pmagic, dmagic;      // x / chunk == umulhi(x, magic) for x < 2^16 (magic 0: chunk 1, x)
  int32_t svc32;                // every remainder chunk's tokens * us + 999 below 2^32 (declared bounds)
  int32_t r_hi;                 // min(r_cap, budget): replicas one model may hold
  uint32_t ring_len;            // power of two above the longest span of a request in windows
  int32_t window_ms;
  int32_t duration_ms;          // duration + longest service < 2^31
  int32_t n_windows;
  int32_t fast_w, slow_w;       // periods in windows
};

__device__ __forceinline__ int64_t ceil_ms(int64_t tokens, uint32_t us) {
  return (tokens * (int64_t)us + 999) / 1000;
}
// the same when tokens * us + 999 < 2^32: y / 1000 == umulhi(y, ceil(2^38 / 1000)) >> 6
// for every 32-bit y (the multiplier's excess, 0.056 / 2^38 per unit of y,
// stays below the 1/1000 gap to the next integer)
__device__ __forceinline__ uint32_t ceil_ms32(uint32_t tokens, uint32_t us) {
  return __umulhi(tokens * us + 999u, 0x10624DD3u) >> 6;
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

// A lane's slot free times in LDS as a 4-ary min-heap: node i at h[i + 3],
// h 16-byte aligned, so that the children 4i + 1 .. 4i + 4 of node i fill
// the aligned group h[4i + 4 .. 4i + 7] and one LDS read fetches them all
// (half the depth of a binary heap on the chain each start waits for). A heap
// of n > 0 nodes owns words h[0 .. (n + 6) & ~3): the nodes from n to the end
// hold kNone, which no free time reaches (free times stay below 2^31), so the
// sift-down needs no bounds on a group. Only the multiset of free times
// matters, so the heap order is free.
struct Heap {
  uint32_t* h;

  __device__ uint32_t& at(int i) const { return h[i + 3]; }

  // words a heap of n nodes owns
  __host__ __device__ static int words(int n) { return n > 0 ? (n + 6) & ~3 : 0; }

  // the root (the smallest) replaced by v, n > 0 nodes; returns the new root
  __device__ uint32_t replace_top(int n, uint32_t v) const {
    int i = 0;
    uint32_t top = v;
    for (;;) {
      const int c = 4 * i + 1;
      if (c >= n) break;
      const uint4 q = *(const uint4*)(h + 4 * i + 4);
      const bool b1 = q.y < q.x, b2 = q.w < q.z;
      const uint32_t m01 = b1 ? q.y : q.x, m23 = b2 ? q.w : q.z;
      const bool b3 = m23 < m01;
      const uint32_t m = b3 ? m23 : m01;
      if (m >= v) break;
      at(i) = m;
      top = i == 0 ? m : top;
      i = c + (b3 ? (b2 ? 3 : 2) : (b1 ? 1 : 0));
    }
    at(i) = v;
    return top;
  }

  // v added to n nodes (node n inside the words the heap owns)
  __device__ void push(int n, uint32_t v) const {
    int i = n;
    while (i > 0) {
      const int par = (i - 1) >> 2;
      const uint32_t pv = at(par);
      if (pv <= v) break;
      at(i) = pv;
      i = par;
    }
    at(i) = v;
  }

  // the root removed from n > 0 nodes (its last node marked free)
  __device__ void pop(int n) const {
    const uint32_t last = at(n - 1);
    at(n - 1) = kNone;
    if (n > 1) replace_top(n - 1, last);
  }
};

__device__ __forceinline__ void lds_add(uint32_t* a, uint32_t v) {
  __hip_atomic_fetch_add(a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
// a scenario's far ring is read and written by its own workgroup only, so
// workgroup scope suffices (with agent scope the drain's loads and stores
// carry the device-coherence bit, and the kernel writes a third more bytes
// to HBM)
__device__ __forceinline__ void far_add(uint32_t* a, uint32_t v) {
  __hip_atomic_fetch_add(a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ uint32_t far_load(uint32_t* a) {
  return __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void far_store(uint32_t* a, uint32_t v) {
  __hip_atomic_store(a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void far_add(unsigned long long* a, unsigned long long v) {
  __hip_atomic_fetch_add(a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ unsigned long long far_load(unsigned long long* a) {
  return __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void far_store(unsigned long long* a, unsigned long long v) {
  __hip_atomic_store(a, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__global__ void zero_u64(unsigned long long* x) { *x = 0ull; }

// kAct: the actuation model. A woken replica is routable wake_w windows
// after its wake starts (its slots free from the start of the window after
// the wake completes); a donor's replica stops being routable at once (its
// earliest-free slots leave at the move) and its GPUs reach the receiver
// after sleep_w windows, when the receiver's wake starts (a shortfall comes
// from the idle GPUs at the move, an excess returns when the sleep ends); a
// model with a transition in flight is neither receiver nor donor; vetoed
// models do not release; the budget counts GPUs (footprint g per replica).
template <bool kAct>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4, 8))) void loop_replay(LoopParams p) {
  extern __shared__ __align__(16) uint32_t lds[];
  const int lane = threadIdx.x;
  const uint32_t s = blockIdx.x;
  const int M = p.M;
  const bool act = lane < M;
  const int mc = act ? lane : 0;
  const tre_scenario sc = p.sc[s];
  const uint32_t t = sc.trace < p.n_traces ? sc.trace : 0;
  const uint64_t tm = (uint64_t)t * M + mc;
  // the profile's smoothing terms stay in registers; the thresholds are
  // read again at ticks, the SLO bounds sit in LDS
  const double w_p = p.prof[tm].w_p, w_q = p.prof[tm].w_q, alpha = p.prof[tm].alpha;
  const int r_init = p.prof[tm].r_init;
  const tre_service sv = p.svc[tm];
  const int32_t W = p.window_ms, dur = p.duration_ms;
  const uint32_t L = p.ring_len;
  const int spr = p.spr;
  const int64_t p_full = ceil_ms(p.pchunk, sv.prefill_us), d_full = ceil_ms(p.dchunk, sv.decode_us);
  // the slot heaps: the models' heaps packed one after another, each in the
  // words it owns (a multiple of 4 words, so that a root's neighbour roots lie
  // an odd number of 16-byte groups away when the heaps are alike: different
  // banks); a tick that moves replicas repacks them through the scenario's
  // scratch in HBM
  uint32_t* const hpool = lds;
  uint32_t* const rest = lds + p.pool_words;
  double* const slo_t = (double*)rest + mc;  // ttft, tpot, e2e bounds at slo_t[i * M]
  uint32_t* near = rest + 6 * M + mc;  // field f of ring cell c at near[(f * kNear + c) * M]
  // requests sbase .. sbase + kStage - 1: arrival (ms, at most the duration)
  // at stg[2 * e * M], prompt | output << 16 at stg[(2 * e + 1) * M]
  int32_t* stg = (int32_t*)(rest + (6 + 4 * kNear) * M + mc);
  // starts recorded for the wave's event pass: field f (start, prompt | output
  // << 16, end of the prompt, first chunk's number) of entry k at
  // ent[(f * kEnt + k) * M]; each lane's first chunk number and entry count;
  // each lane's chunk times and rates (prompt chunk, output chunk, prefill_us,
  // decode_us) at cst[i * M]
  uint32_t* ent = rest + (6 + 4 * kNear + 2 * kStage) * M + mc;
  uint32_t* lane_off = rest + (6 + 4 * kNear + 2 * kStage + 4 * kEnt) * M;
  uint32_t* lane_cnt = lane_off + M;
  uint32_t* cst = lane_cnt + M + mc;
  // the far rings' cell c of this lane at index fo + c * M (one offset for
  // the three rings keeps one register pair)
  const uint64_t fo = (uint64_t)s * L * M + mc;
  // initial replicas: at most r_hi per model and pool_reps in all (initial
  // replicas within the budget and the declared bound are never cut; cut
  // ones are counted as bounds exceeded)
  const int r_hi = p.r_hi;
  int R = act ? (r_init < 0 ? 0 : (r_init > r_hi ? r_hi : r_init)) : 0;
  unsigned slots_over = 0;  // replicas / slots the pool could not hold
  {
    int incl = R;
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (lane >= o) incl += v;
    }
    const int room = p.pool_reps - (incl - R);
    const int R0 = R;
    R = R < room ? R : (room > 0 ? room : 0);
    slots_over += (unsigned)(R0 - R);
  }
  // GPUs per replica (1 without the actuation model); idle GPUs (replicas)
  // (at least 1, so that the replicas never outnumber the budget's GPUs and
  // the heaps' pool always holds their slots)
  const int g_in = (kAct && p.footprint && act) ? p.footprint[tm] : 1;
  const int g = g_in < 1 ? 1 : g_in;
  int rsum = R * g;
  for (int o = 32; o > 0; o >>= 1) rsum += __shfl_xor(rsum, o);
  int pool = p.budget - rsum;
  // the lane's transition in flight (0 none, 1 wake, 2 sleep), the window at
  // whose end it completes, and the GPUs a sleep returns to the idle pool
  int tkind = 0, tuntil = 0, tret = 0;
  int hs = R * spr;  // heap size (R <= r_hi)
  // each lane's heap of n nodes placed after the lower lanes' (the first
  // word of its own, a multiple of 4), its unused nodes marked free; called
  // by the whole wave
  auto place = [&](int n) {
    const int own = act ? Heap::words(n) : 0;
    int incl = own;
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o);
      if (lane >= o) incl += v;
    }
    return incl - own;
  };
  auto mark_free = [&](const Heap& hp, int from, int n) {
    for (int i = from; i < Heap::words(n) - 3; ++i) hp.at(i) = kNone;
  };
  int base = place(hs);  // the current heap's first word in the pool
  auto heap = [&]() { return Heap{hpool + base}; };
  if (act) {
    const tre_slo sl = p.slo[tm];
    slo_t[0] = sl.ttft_ms;
    slo_t[M] = sl.tpot_ms;
    slo_t[2 * M] = sl.e2e_ms;
    cst[0] = (uint32_t)p_full;
    cst[M] = (uint32_t)d_full;
    cst[2 * M] = sv.prefill_us;
    cst[3 * M] = sv.decode_us;
    for (int i = 0; i < 4 * kNear; ++i) near[i * M] = 0u;
    const Heap h0 = heap();
    for (int i = 0; i < hs; ++i) h0.at(i) = 0u;  // equal keys form a heap
    mark_free(h0, hs, hs);
    for (uint32_t c = 0; c < L; ++c) {
      far_store(&p.far_p[fo + (uint64_t)c * M], 0u);
      far_store(&p.far_d[fo + (uint64_t)c * M], 0u);
      far_store(&p.far_f[fo + (uint64_t)c * M], 0ull);
    }
  }
  uint32_t bf = act && hs > 0 ? 0u : kNone;  // earliest slot free time (the heap's root)
  // the donors' earliest-free slots leave their heaps; every heap is packed
  // again (through the scratch: each lane copies its own heap out, then,
  // after every lane's reads, back in at its new place); the receivers'
  // slots, free from `from`, join there. Called by the whole wave.
  auto repack = [&](int pops, int pushes, uint32_t from) {
    const Heap old = heap();
    for (int q = 0; q < pops && hs > 0; ++q) old.pop(hs--);
    // the pool holds pool_reps * spr slots: pushes beyond it (a declared
    // replica bound exceeded) are dropped, in lane order (in fours when spr is
    // a multiple of 4, so that every heap size stays one: the pool's words
    // then count 4, not 6, beyond each heap's nodes)
    {
      int tot = hs, pin = pushes;
      for (int o = 1; o < 64; o <<= 1) {
        const int v = __shfl_up(pin, o);
        if (lane >= o) pin += v;
      }
      for (int o = 32; o > 0; o >>= 1) tot += __shfl_xor(tot, o);
      int allowed = p.pool_reps * spr - tot - (pin - pushes);
      allowed = allowed < 0 ? 0 : (allowed > pushes ? pushes : allowed);
      if (spr % 4 == 0) allowed &= ~3;
      slots_over += (unsigned)(pushes - allowed);
      pushes = allowed;
    }
    const int want = act ? hs + pushes : 0;
    const int nbase = place(want);
    uint32_t* tmp = p.scratch + (uint64_t)s * p.pool_words + nbase;
    if (act)
      for (int i = 0; i < hs; ++i) tmp[i] = old.at(i);
    const Heap fresh{hpool + nbase};
    if (act) {
      for (int i = 0; i < hs; ++i) fresh.at(i) = tmp[i];
      mark_free(fresh, hs, want);
    }
    for (int q = 0; q < pushes; ++q) fresh.push(hs + q, from);
    hs += pushes;
    base = nbase;
    bf = act && hs > 0 ? fresh.at(0) : kNone;
  };
  const uint32_t wmagic = p.wmagic, pmagic = p.pmagic, dmagic = p.dmagic;
  const int wshift = p.wshift;
  // x / W for x < 2^31; x / prefill_chunk and x / decode_chunk for x < 2^16
  auto win = [&](uint32_t x) { return (int32_t)(wshift < 0 ? x : __umulhi(x, wmagic) >> wshift); };
  auto div_p = [&](uint32_t x) { return pmagic ? __umulhi(x, pmagic) : x; };
  auto div_d = [&](uint32_t x) { return dmagic ? __umulhi(x, dmagic) : x; };
  // a remainder chunk's time (ms): 32-bit when the declared bounds allow
  const bool svc32 = p.svc32 != 0;
  auto rem_ms = [&](uint32_t tok, uint32_t us) { return svc32 ? ceil_ms32(tok, us) : (uint32_t)ceil_ms(tok, us); };
  const uint32_t udur = (uint32_t)dur;
  // the model's requests: rq0 + [0, nq); indices below relative to rq0
  const int64_t rq0 = act ? p.req_off[tm] : 0;
  const int64_t rq1 = act ? p.req_off[tm + 1] : 0;
  const uint32_t nq = rq1 > rq0 ? (uint32_t)(rq1 - rq0) : 0u;
  const int64_t* const arrival = p.arrival + rq0;
  uint32_t next_arr = 0, next_start = 0;
  // arrival of request i, kArrNever when past the table or at or after the
  // end of the replay (such a request never arrives)
  auto arr = [&](uint32_t i) -> int32_t {
    if (i >= nq) return kArrNever;
    const int64_t v = arrival[i];
    return v >= (int64_t)dur ? kArrNever : (v > (int64_t)INT32_MIN ? (int32_t)v : INT32_MIN);
  };
  // arrival times of requests next_arr .. next_arr + 3
  int32_t a0 = arr(0), a1 = arr(1), a2 = arr(2), a3 = arr(3);
  // the next kStage requests to start, fetched together (one wait per kStage starts)
  uint32_t sbase = next_start;
  auto stage = [&](uint32_t from) {
    int64_t av[kStage] = {};
    uint32_t pv[kStage] = {};
    if (nq) {  // every load issued before any is used (one wait); past the table, the last request's
#pragma unroll
      for (int e = 0; e < kStage; ++e) {
        const uint32_t i = from + e < nq ? from + e : nq - 1;
        av[e] = arrival[i];
        pv[e] = (uint32_t)p.prompt[rq0 + i] | (uint32_t)p.output[rq0 + i] << 16;
      }
    }
#pragma unroll
    for (int e = 0; e < kStage; ++e) {
      const bool in = from + e < nq;
      av[e] = in ? av[e] : kNever;
      pv[e] = in ? pv[e] : 0u;
    }
#pragma unroll
    for (int e = 0; e < kStage; ++e) {
      stg[2 * e * M] = (int32_t)(av[e] < (int64_t)dur ? (av[e] > INT32_MIN ? av[e] : INT32_MIN) : dur);
      stg[(2 * e + 1) * M] = (int32_t)pv[e];
    }
    sbase = from;
  };
  if (act) stage(next_start);
  uint32_t fp = 0, fd = 0, fn = 0, fe = 0;  // far cell of window w - 1 + kNear, loaded at window w - 1
  int32_t cA = 0, cW = 0;  // active / waiting requests at the current window's start
  double S = 0.0;
  bool init = false;
  uint32_t n_arr = 0, n_start = 0, n_done = 0, n_ok = 0;
  int64_t e2e_sum = 0, rw = 0;
  int32_t e2e_max = 0;
  unsigned overflow = 0;
  uint32_t nm = 0;
  int tick = 0;  // ticks so far (wave-uniform)
  const unsigned long long live = __ballot(act);

  for (int32_t w = 0; w < p.n_windows; ++w) {
    const int32_t w_end = (w + 1) * W;
    if constexpr (kAct) {  // transitions that completed at the end of an earlier window
      const bool done = tkind != 0 && tuntil < w;
      int push = 0;
      if (done && tkind == 1) {
        push = R < r_hi ? spr : 0;
        R += 1;
      }
      unsigned long long back = __ballot(done && tkind == 2 && tret > 0);
      while (back) {
        const int l = __ffsll((long long)back) - 1;
        pool += __builtin_amdgcn_readlane(tret, l);
        back &= back - 1ull;
      }
      if (done) {
        tkind = 0;
        tret = 0;
      }
      if (__ballot(push > 0)) repack(0, push, (uint32_t)(w * W));
    }
    uint32_t P = 0, D = 0;
    int64_t eA = 0, eW = 0;
    int32_t dA = 0, dW = 0;
    bool idle = true;
    if (act) {
      // arrivals: a request waits from its arrival
      while (a0 < w_end) {
        eW += w_end - a0;
        dW += 1;
        ++n_arr;
        ++next_arr;
        a0 = a1;
        a1 = a2;
        a2 = a3;
        a3 = arr(next_arr + 3);
      }
    }
    // ---- starts, in arrival order, on the slot that frees first. A lane
    // starts up to kEnt requests per pass (their finish, judging and slot
    // in closed form) and records them; the whole wave then adds their
    // PREFILL / DECODE events to the rings, chunks spread over the lanes.
    bool more = act;
    for (;;) {
      int cnt = 0;
      uint32_t ntot = 0;
      if (more) {
        const int ns = hs;
        const Heap slot = heap();
        more = false;
        while (next_start < next_arr && ns > 0) {
          if (next_start - sbase >= kStage) stage(next_start);
          const int e = (int)(next_start - sbase);
          const int64_t a = stg[2 * e * M];
          const uint32_t po = (uint32_t)stg[(2 * e + 1) * M];
          const int64_t st = a > (int64_t)bf ? a : (int64_t)bf;
          if (st >= w_end) break;  // capacity may change at the window's end
          // admission: waiting -> active
          eW -= w_end - st;
          dW -= 1;
          eA += w_end - st;
          dA += 1;
          // chunks: PREFILL events at the start of each prompt chunk, DECODE
          // events at the end of each output chunk, FINISH at the last
          const uint32_t pt = po & 0xffffu, out_tok = po >> 16;
          const uint32_t npf = div_p(pt), prem = pt - npf * (uint32_t)p.pchunk;
          const uint32_t ndf = div_d(out_tok), drem = out_tok - ndf * (uint32_t)p.dchunk;
          const uint32_t t_prem = prem ? rem_ms(prem, cst[2 * M]) : 0u;
          const uint32_t t_drem = drem ? rem_ms(drem, cst[3 * M]) : 0u;
          const uint32_t td = (uint32_t)st + npf * (uint32_t)p_full + t_prem;  // end of the prompt
          const uint32_t tt = td + ndf * (uint32_t)d_full + t_drem;            // the last output chunk
          if (tt < udur) {  // FINISH: active -> gone
            const int32_t xw = win(tt);
            const uint32_t ahead = (uint32_t)(xw - w), ef = (uint32_t)(xw + 1) * (uint32_t)W - tt;
            if (ahead == 0u) {
              eA -= w_end - (int64_t)tt;
              dA -= 1;
            } else if (ahead < (uint32_t)kNear) {
              uint32_t* nc = near + (xw & (kNear - 1)) * M;
              lds_add(nc + 2 * kNear * M, 1u);
              lds_add(nc + 3 * kNear * M, ef);
            } else if (ahead < L) {
              far_add(&p.far_f[fo + (uint64_t)(xw & (L - 1)) * M], (1ull << 32) | ef);
            } else {
              ++overflow;
            }
            if (out_tok) {  // judged as in the calibration sweep
              // 32-bit differences: every time here is in [0, 2^31) (arrivals
              // non-negative, the duration plus the longest service below 2^31)
              const uint32_t t_first = td + (ndf ? (uint32_t)d_full : t_drem);
              const uint32_t first_ch = ndf ? (uint32_t)p.dchunk : drem;
              const int32_t ttft = (int32_t)(t_first - (uint32_t)a), e2e = (int32_t)(tt - (uint32_t)a);
              const int32_t after = (int32_t)(out_tok - first_ch);
              bool good = (double)ttft <= slo_t[0] && (double)e2e <= slo_t[2 * M];
              if (after > 0) good = good && (double)(int32_t)(tt - t_first) / (double)after <= slo_t[M];
              ++n_done;
              n_ok += good ? 1u : 0u;
              e2e_sum += e2e;
              e2e_max = e2e > e2e_max ? e2e : e2e_max;
            }
          }
          bf = slot.replace_top(ns, tt);  // tt >= st >= the root
          ent[(0 * kEnt + cnt) * M] = (uint32_t)st;
          ent[(1 * kEnt + cnt) * M] = po;
          ent[(2 * kEnt + cnt) * M] = td;
          ent[(3 * kEnt + cnt) * M] = ntot;
          ntot += npf + (prem ? 1u : 0u) + ndf + (drem ? 1u : 0u);
          ++cnt;
          ++n_start;
          ++next_start;
          if (cnt == kEnt) {
            more = true;
            break;
          }
        }
      }
      if (!__ballot(cnt > 0)) break;
      // the recorded chunks of every lane, numbered by an exclusive scan
      uint32_t incl = ntot;
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t v = (uint32_t)__shfl_up((int)incl, o);
        if (lane >= o) incl += v;
      }
      const uint32_t C = (uint32_t)__shfl((int)incl, 63);
      if (lane < M) {
        lane_off[lane] = incl - ntot;
        lane_cnt[lane] = (uint32_t)cnt;
      }
      __syncthreads();
      for (uint32_t c = (uint32_t)lane; c < C; c += 64) {
        int l = 0;  // the owner: the last lane whose first chunk is at or before c
        for (int step = 32; step > 0; step >>= 1)
          if (l + step < M && lane_off[l + step] <= c) l += step;
        const uint32_t r = c - lane_off[l];
        int k = 0;
        const int cn = (int)lane_cnt[l];
        while (k + 1 < cn && ent[(3 * kEnt + k + 1) * M + (l - mc)] <= r) ++k;
        const uint32_t* en = ent + k * M + (l - mc);
        const uint32_t j = r - en[3 * kEnt * M];
        const uint32_t st = en[0], po = en[kEnt * M], td = en[2 * kEnt * M];
        const uint32_t* cl = cst + (l - mc);  // owner's chunk times and rates
        const uint32_t pt = po & 0xffffu, out_tok = po >> 16;
        const uint32_t npf = div_p(pt), prem = pt - npf * (uint32_t)p.pchunk;
        const uint32_t np = npf + (prem ? 1u : 0u);
        uint32_t t, tok;
        int f;
        if (j < np) {
          t = st + j * cl[0];
          tok = j < npf ? (uint32_t)p.pchunk : prem;
          f = 0;
        } else {
          const uint32_t q = j - np, ndf = div_d(out_tok);
          if (q < ndf) {
            t = td + (q + 1u) * cl[M];
            tok = (uint32_t)p.dchunk;
          } else {
            const uint32_t drem = out_tok - ndf * (uint32_t)p.dchunk;
            t = td + ndf * cl[M] + rem_ms(drem, cl[3 * M]);
            tok = drem;
          }
          f = 1;
        }
        if (t < udur) {
          const int32_t x = win(t);
          const uint32_t ahead = (uint32_t)(x - w);
          if (ahead < (uint32_t)kNear) {
            lds_add(near + (l - mc) + (f * kNear + (x & (kNear - 1))) * M, tok);
          } else if (ahead < L) {
            const uint64_t fcell = (uint64_t)(x & (L - 1)) * M + (l - mc);
            far_add(f ? &p.far_d[fo + fcell] : &p.far_p[fo + fcell], tok);
          } else {
            ++overflow;
          }
        }
      }
      __syncthreads();
      if (!__ballot(more)) break;
    }
    if (act) {
      {  // the window's tallies, now complete: requests started before it and in it
        uint32_t* nc = near + (w & (kNear - 1)) * M;
        P = nc[0];
        D = nc[kNear * M];
        const uint32_t nf = nc[2 * kNear * M], ef = nc[3 * kNear * M];
        nc[0] = 0u;
        nc[kNear * M] = 0u;
        nc[2 * kNear * M] = 0u;
        nc[3 * kNear * M] = 0u;
        dA -= nf;
        eA -= ef;
      }
      {  // far tallies: those of window w - 1 + kNear into LDS, then fetch those of w + kNear
        if (fp | fd | fn | fe) {
          uint32_t* nc = near + ((w - 1) & (kNear - 1)) * M;
          if (fp) lds_add(nc, fp);
          if (fd) lds_add(nc + kNear * M, fd);
          if (fn) lds_add(nc + 2 * kNear * M, fn);
          if (fe) lds_add(nc + 3 * kNear * M, fe);
          const uint64_t c0 = (uint64_t)((uint32_t)(w - 1 + kNear) & (L - 1)) * M;
          far_store(&p.far_p[fo + c0], 0u);
          far_store(&p.far_d[fo + c0], 0u);
          far_store(&p.far_f[fo + c0], 0ull);
        }
        const uint64_t c1 = (uint64_t)((uint32_t)(w + kNear) & (L - 1)) * M;
        fp = far_load(&p.far_p[fo + c1]);
        fd = far_load(&p.far_d[fo + c1]);
        const unsigned long long ff = far_load(&p.far_f[fo + c1]);
        fn = (uint32_t)(ff >> 32);
        fe = (uint32_t)ff;
      }
      // the window's tallies, Eq. (1) and the smoothing
      const int64_t A_int = (int64_t)W * cA + eA, W_int = (int64_t)W * cW + eW;  // counts below 2^31
      cA += dA;
      cW += dW;
      idle = P == 0 && D == 0 && A_int == 0 && W_int == 0;
      if (!idle) {
        double num = w_p * (double)P;
        num = num + (double)D;
        num = num * 1000.0;
        const double q = w_q * (double)W_int;
        double den = (double)A_int + q;
        if (den < (double)W) den = (double)W;
        const double raw = num / den;
        if (init) {
          const double t1 = alpha * raw;
          const double t2 = (1.0 - alpha) * S;
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
    const int tk = tick++;
    const tre_profile prt = p.prof[tm];  // the thresholds, read at ticks only
    const double theta_eff = prt.theta * sc.theta_scale;
    const double tau_c = sc.tau_crit_override >= 0.0 ? sc.tau_crit_override : prt.tau_crit;
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
    const unsigned long long sur = __ballot(act && Z > prt.tau_surplus);
    // models already in a move: earlier in this tick, or (kAct) in flight
    unsigned long long used = kAct ? __ballot(tkind != 0) : 0ull;
    const unsigned long long veto_mask = (kAct && p.veto) ? p.veto[(uint64_t)t * p.n_ticks + tk] : 0ull;
    int pops = 0, pushes = 0;  // this tick's slot changes of this lane (a model moves at most once per tick)
    for (uint32_t k = 0; k < sc.max_moves; ++k) {
      const int r = pick_lane<false>(ok & ~used & __ballot(act && R < p.r_cap), Z, lane);  // Eq. (3)
      if (r < 0) break;
      const int g_r = kAct ? __builtin_amdgcn_readlane(g, r) : 1;
      int d;
      if (pool >= g_r) {
        pool -= g_r;
        d = TRE_DONOR_POOL;
        if (kAct && lane == r) {
          tkind = 1;
          tuntil = w + p.wake_w;
        }
      } else {
        const double Zr = lane_f64(Z, r);
        const unsigned long long cd = __ballot(act && R > prt.r_min && Z > Zr && (!kAct || pool >= g_r - g)) &
                                      ~crit & ~used & ~(1ull << r) & live & ~veto_mask;
        d = pick_lane<true>(cd & sur, Z, lane);
        if (d < 0) d = pick_lane<true>(cd & ~sur, Z, lane);
        if (d < 0) break;
        used |= 1ull << d;
        const int short_by = kAct ? g_r - __builtin_amdgcn_readlane(g, d) : 0;
        if (short_by > 0) pool -= short_by;
        if (lane == d && R > 0) {  // the replica's slots that free first leave
          pops = spr;
          R -= 1;
        }
        if (kAct && lane == d) {
          tkind = 2;
          tuntil = w + p.sleep_w;
          tret = short_by < 0 ? -short_by : 0;
        }
        if (kAct && lane == r) {
          tkind = 1;
          tuntil = w + p.sleep_w + p.wake_w;
        }
      }
      used |= 1ull << r;
      if (!kAct && lane == r) {  // the new replica's slots, free from the window's end
        pushes = R < r_hi ? spr : 0;
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
    if (__ballot(pops > 0 || pushes > 0)) repack(pops, pushes, (uint32_t)w_end);
  }
  if constexpr (kAct) {  // wakes completing at the end of the last window count
    if (tkind == 1 && tuntil < p.n_windows) R += 1;
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
    st.e2e_max = (int64_t)e2e_max;
    p.stats[(uint64_t)s * M + lane] = st;
  }
  if (lane == 0) p.n_moves[s] = nm;
  overflow += slots_over;
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

int r_hi(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  return rq->r_cap < cfg->budget ? rq->r_cap : cfg->budget;
}

// replicas the heap pool holds, and its words: the heaps' nodes, plus up to
// 6 words per model that the heaps own beyond their nodes (4 when every heap
// size is a multiple of 4), a multiple of 4
int pool_reps(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  const int64_t all = (int64_t)cfg->n_models * r_hi(cfg, rq);
  int64_t v = cfg->budget < all ? cfg->budget : all;
  if (rq->max_replicas > 0 && (int64_t)rq->max_replicas < v) v = rq->max_replicas;
  return (int)v;
}
int pool_words(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  const int64_t pad = rq->slots_per_replica % 4 == 0 ? 4 : 6;
  return (int)(((int64_t)pool_reps(cfg, rq) * rq->slots_per_replica + pad * cfg->n_models + 3) & ~3ll);
}

// LDS bytes of one scenario: the slot heaps' pool, then per model its SLO
// bounds, the four planes of the near ring, the staged requests (arrival,
// prompt and output), the recorded starts, the model's chunk offset and
// count, its chunk times and rates
size_t lds_bytes(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  return ((size_t)pool_words(cfg, rq) + (size_t)(6 + 4 * kNear + 2 * kStage + 4 * kEnt + 2 + 4) * cfg->n_models) * 4;
}

// x / d == umulhi(x, m) >> sh for x < 2^31 and 1 <= d < 2^31: with 2^(l-1) < d
// <= 2^l, m = ceil(2^(31 + l) / d) < 2^32 and sh = l - 1 (the multiplier's
// excess adds less than x / 2^(31 + l) < 1 / d, below the gap to the next
// integer); d = 1 gives sh = -1 (x itself)
void magic31(int64_t d, uint32_t* m, int32_t* sh) {
  int l = 0;
  while ((1ll << l) < d) ++l;
  *sh = l - 1;
  *m = l == 0 ? 0u : (uint32_t)(((1ull << (31 + l)) + (uint64_t)d - 1) / (uint64_t)d);
}

// x / d == umulhi(x, m) for x < 2^16 and d >= 2: m = floor(2^32 / d) + 1 (the
// excess adds at most x / 2^32 < 1 / d while x * d < 2^32; m = 1 for d >=
// 2^16, where every such x / d is 0); m = 0 for d = 1 (x itself)
uint32_t magic16(int64_t d) {
  if (d == 1) return 0u;
  if (d >= 65536) return 1u;
  return (uint32_t)((1ull << 32) / (uint64_t)d) + 1u;
}

int check_loop_args(const tre_trace_cfg* cfg, const tre_loop_requests* rq) {
  if (!cfg || !rq) return fail(TRE_EINVAL, "tre_loop: NULL cfg or request table");
  if (cfg->window_ms < 1 || cfg->duration_ms <= 0 || cfg->duration_ms % cfg->window_ms ||
      cfg->fast_period_ms <= 0 || cfg->slow_period_ms <= 0 || cfg->fast_period_ms % cfg->window_ms ||
      cfg->slow_period_ms % cfg->window_ms || cfg->duration_ms >= (1ll << 40))
    return fail(TRE_EINVAL, "tre_loop: bad window, duration or periods");
  if (cfg->n_models < 1 || cfg->n_models > TRE_MAX_MODELS || cfg->budget < 0)
    return fail(TRE_EINVAL, "tre_loop: n_models outside [1, %d] or negative budget", TRE_MAX_MODELS);
  if (rq->slots_per_replica < 1 || rq->r_cap < 1 || rq->prefill_chunk < 1 || rq->decode_chunk < 1 ||
      rq->slots_per_replica > 4096 || rq->r_cap > 4096)
    return fail(TRE_EINVAL, "tre_loop: slots_per_replica, r_cap and chunks must be positive (and at most 4096)");
  if (max_service_ms(rq) / cfg->window_ms > (1 << 24))
    return fail(TRE_ERANGE, "tre_loop: a request may span more than 2^24 windows");
  if (cfg->duration_ms + max_service_ms(rq) + 2 * cfg->window_ms >= (1ll << 31))
    return fail(TRE_ERANGE, "tre_loop: duration plus the longest service must stay below 2^31 ms");
  if (lds_bytes(cfg, rq) > (size_t)kLdsMax)
    return fail(TRE_EINVAL, "tre_loop: %d models x %d slots need %zu bytes of LDS (at most %d)", cfg->n_models,
                r_hi(cfg, rq) * rq->slots_per_replica, lds_bytes(cfg, rq), kLdsMax);
  return TRE_OK;
}

}  // namespace

// --------------------------------------------------------------- host ABI
extern "C" int tre_loop_workspace_size(const tre_trace_cfg* cfg, const tre_loop_requests* rq,
                                       uint32_t n_scenarios, size_t* bytes) {
  if (!bytes) return fail(TRE_EINVAL, "tre_loop_workspace_size: NULL bytes");
  const int rc = check_loop_args(cfg, rq);
  if (rc) return rc;
  *bytes = (size_t)(256 + (uint64_t)n_scenarios * cfg->n_models * ring_len(cfg, rq) * 16 +
                    (uint64_t)n_scenarios * pool_words(cfg, rq) * 4);
  return TRE_OK;
}

static int loop_impl(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq,
                     const tre_profile* prof, const tre_scenario* sc, uint32_t n_scenarios, const tre_actuation* act,
                     const tre_ctl_out* out, tre_loop_stats* stats, double* tss64, void* ws, size_t ws_bytes,
                     void* stream, const char* who) {
  int rc = check_loop_args(cfg, rq);
  if (rc) return rc;
  if (!prof || !out || !stats || !ws || !rq->arrival_ms || !rq->prompt || !rq->output || !rq->req_off ||
      !rq->service || !rq->slo || (n_scenarios && (!sc || !out->moves || !out->n_moves || !out->r_final ||
                                                   !out->r_windows)))
    return fail(TRE_EINVAL, "%s: NULL argument", who);
  if (n_traces == 0) return fail(TRE_EINVAL, "%s: no traces", who);
  if ((uintptr_t)ws & 15) return fail(TRE_EINVAL, "%s: workspace needs 16-byte alignment", who);
  const int64_t nW = cfg->duration_ms / cfg->window_ms;
  int32_t wake_w = 0, sleep_w = 0;
  if (act) {
    if (act->wake_ms < 0 || act->sleep_ms < 0) return fail(TRE_EINVAL, "%s: actuation delays must be >= 0", who);
    // whole windows, rounded up; a transition completing after the last
    // window never counts, so the delays are capped just past the trace
    const int64_t win = cfg->window_ms, cap = nW + 1;
    auto to_windows = [&](int64_t ms) { return ms > cap * win ? cap : (ms + win - 1) / win; };
    wake_w = (int32_t)to_windows(act->wake_ms);
    sleep_w = (int32_t)to_windows(act->sleep_ms);
  }
  size_t need = 0;
  tre_loop_workspace_size(cfg, rq, n_scenarios, &need);
  if (ws_bytes < need) return fail(TRE_ENOMEM, "%s: workspace %zu < %zu bytes", who, ws_bytes, need);
  if (n_scenarios == 0) return TRE_OK;
  hipStream_t st = (hipStream_t)stream;
  const int M = cfg->n_models;
  const uint32_t L = ring_len(cfg, rq);
  char* base = (char*)ws;
  unsigned long long* overflow = (unsigned long long*)base;
  const uint64_t cells = (uint64_t)n_scenarios * M * L;  // the rings: 4 + 4 + 8 bytes per cell
  uint32_t* far_p = (uint32_t*)(base + 256);
  uint32_t* far_d = (uint32_t*)(base + 256 + cells * 4);
  unsigned long long* far_f = (unsigned long long*)(base + 256 + cells * 8);
  uint32_t* scratch = (uint32_t*)(base + 256 + cells * 16);
  const size_t lds = lds_bytes(cfg, rq);
  const void* kern = act ? (const void*)loop_replay<true> : (const void*)loop_replay<false>;
  HIP_TRY(hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
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
  lp.far_p = far_p;
  lp.far_d = far_d;
  lp.far_f = far_f;
  lp.scratch = scratch;
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
  lp.pool_words = pool_words(cfg, rq);
  lp.pool_reps = pool_reps(cfg, rq);
  lp.r_hi = r_hi(cfg, rq);
  magic31(cfg->window_ms, &lp.wmagic, &lp.wshift);
  lp.pmagic = magic16(rq->prefill_chunk);
  lp.dmagic = magic16(rq->decode_chunk);
  lp.svc32 = (int64_t)rq->prefill_chunk * rq->max_prefill_us + 999 < (1ll << 32) &&
             (int64_t)rq->decode_chunk * rq->max_decode_us + 999 < (1ll << 32);
  lp.ring_len = L;
  lp.window_ms = (int32_t)cfg->window_ms;
  lp.duration_ms = (int32_t)cfg->duration_ms;
  lp.n_windows = (int32_t)nW;
  // a period longer than the replay never ticks
  lp.fast_w = (int32_t)std::min<int64_t>(cfg->fast_period_ms / cfg->window_ms, lp.n_windows + 1);
  lp.slow_w = (int32_t)std::min<int64_t>(cfg->slow_period_ms / cfg->window_ms, lp.n_windows + 1);
  if (act) {
    lp.footprint = act->footprint;
    lp.veto = act->veto;
    lp.wake_w = wake_w;
    lp.sleep_w = sleep_w;
    int32_t nt = 0;
    for (int64_t w = 0; w < nW; ++w)
      if ((w + 1) % lp.fast_w == 0 || (w + 1) % lp.slow_w == 0) ++nt;
    lp.n_ticks = nt;
  }
  LaunchTimer lt("loop_replay", st);
  if (act)
    hipLaunchKernelGGL(loop_replay<true>, dim3(n_scenarios), dim3(64), lds, st, lp);
  else
    hipLaunchKernelGGL(loop_replay<false>, dim3(n_scenarios), dim3(64), lds, st, lp);
  lt.done();
  HIP_TRY(hipGetLastError());
  return TRE_OK;
}

extern "C" int tre_loop(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq,
                        const tre_profile* prof, const tre_scenario* sc, uint32_t n_scenarios,
                        const tre_ctl_out* out, tre_loop_stats* stats, double* tss64, void* ws, size_t ws_bytes,
                        void* stream) {
  return loop_impl(cfg, n_traces, rq, prof, sc, n_scenarios, nullptr, out, stats, tss64, ws, ws_bytes, stream,
                   "tre_loop");
}

extern "C" int tre_loop_act(const tre_trace_cfg* cfg, uint32_t n_traces, const tre_loop_requests* rq,
                            const tre_profile* prof, const tre_scenario* sc, uint32_t n_scenarios,
                            const tre_actuation* act, const tre_ctl_out* out, tre_loop_stats* stats, double* tss64,
                            void* ws, size_t ws_bytes, void* stream) {
  if (!act) return fail(TRE_EINVAL, "tre_loop_act: NULL actuation model");
  return loop_impl(cfg, n_traces, rq, prof, sc, n_scenarios, act, out, stats, tss64, ws, ws_bytes, stream,
                   "tre_loop_act");
}
