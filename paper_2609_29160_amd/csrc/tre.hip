// tre.hip - MI355X (gfx950) replay of Token Service Share (TSS) evaluation and
// TSS-guided receiver/donor rebalancing, behind the C ABI of include/tre.h.
//
// Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE): Eq. (1) TSS,
// smoothing, Eq. (2) normalisation and the three regions (Section "Smoothing,
// Normalization, and Calibration"), dual-speed control and Eq. (3) (Section
// "Dual-Speed Control"), bounded pairwise transfer (Section "Bounded Pairwise
// Transfer").
//
// Kernels
//   tss_stream  one workgroup (4 waves) per trace, one barrier per tile of
//               rows. Every thread loads (per-trace buffer resources, the
//               next tile in flight while the current one is tallied) and
//               tallies its rows into an LDS ring of (window, model) cells
//               with one packed 64-bit LDS atomic per row (two for an
//               ADMIT row); completed
//               windows are then evaluated one cell per thread (carry scan,
//               in-window integrals, Eq. (1) in fp64) and one wave per step
//               runs the smoothing chain over the previous chunk.
//   rebalance   one wave per scenario, lane = model: Eq. (2), regions,
//               cadence and the greedy receiver/donor moves, with ballots
//               as candidate sets and DPP wave folds for argmin / argmax
//               (lowest index on ties), so every decision is a scalar.
//   validate    checks the event columns once, at load time.
#include <hip/hip_runtime.h>

#include <limits.h>
#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "tre.h"
#include "tre_internal.h"

#pragma clang fp contract(off)

using tre_internal::check_device;
using tre_internal::fail;
using tre_internal::LaunchTimer;

// ------------------------------------------------------------------ errors
static thread_local std::string g_err;

int tre_internal::fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

extern "C" const char* tre_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------ handle

// ------------------------------------------------------------ constants
constexpr int kStreamWaves = 4;            // tss_stream workgroup (waves) with many traces
constexpr int kEvalThreads = 256;          // threads that evaluate a step's cells (one cell each)
constexpr int kStreamEPT = 4;              // rows per lane per tile
constexpr int kRingBytes = 17 * 1024;      // LDS budget of the tally ring
constexpr uint32_t kNoDefer = 0xFFFFFFFFu;

typedef long long v2i64 __attribute__((ext_vector_type(2)));
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
typedef unsigned int v2u32 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------- tss_stream
struct StreamParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint8_t* type;
  const uint16_t* tokens;
  const int64_t* off;
  int64_t n_rows;
  const tre_profile* prof;
  int64_t window_ms;
  uint32_t magic;   // floor(2^32 / window_ms), 2^32-1 for a 1 ms window
  int32_t n_windows;
  int32_t M;
  uint32_t wcap;    // ring windows, power of two
  double inv2_window;  // 1 / (2 window_ms), rounded to nearest
  int32_t chunk;    // windows evaluated per step (cells <= threads)
  int32_t fast_w;   // fast period in windows
  int32_t slow_w;   // slow period in windows
  uint32_t magic_fast;  // floor(2^32 / fast_w), 2^32 - 1 for 1
  uint32_t magic_slow;
  int32_t n_ticks;
  uint32_t* prefill;
  uint32_t* decode;
  int64_t* a_int;
  int64_t* w_int;
  double* tss64;
  float* tss32;
  uint8_t* flags;
  double* snap;     // [trace][tick][M]: S, or +inf when idle / not initialised
  // the kStage instantiation: stage-aware shares per cell (tre_eval_stage)
  double* stage64;  // [trace][w][M][2]: prefill, decode
  float* stage32;
  uint8_t* sflags;  // TRE_STAGE_*
  // the control replay streamed with its trace (tre_sweep without the
  // actuation model, for traces that carry exactly one scenario)
  const tre_scenario* sc;
  const uint32_t* sc_count;  // [trace] scenarios on the trace, or NULL
  const uint32_t* sc_first;  // [trace] the scenario when the count is 1
  int32_t budget;
  tre_move* moves;
  uint32_t move_cap;
  uint32_t* n_moves;
  int32_t* r_final;
  int64_t* r_windows;
};

// quotient and remainder of rel / window_ms for any 32-bit rel: the
// multiply-high by floor(2^32/window) undershoots by at most one
__device__ __forceinline__ void div_window(uint32_t rel, uint32_t magic, uint32_t win, uint32_t& q,
                                           uint32_t& r) {
  q = __umulhi(rel, magic);
  r = rel - q * win;
  if (r >= win) {
    q += 1;
    r -= win;
  }
}

// One producer lane's share of a tile: kEPT consecutive rows.
template <int kEPT>
struct Slice {
  long long ts[kEPT];
  uint32_t mw[kEPT / 4];  // model bytes, 4 per word
  uint32_t tw[kEPT / 4];  // type bytes
  uint32_t kw[kEPT / 2];  // tokens, 2 per word
};

// Buffer resources over one trace's rows of each column, from its first
// kEPT-aligned row; a load past the range reads zeros (no fault), so tile
// loads need no bounds branches and never touch another trace's rows
// beyond the 16-byte rounding of the range.
struct TraceRsrc {
  __amdgpu_buffer_rsrc_t ts, model, type, tokens;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, long long bytes) {
  const long long n = (bytes + 15) & ~15ll;  // columns are readable 16 bytes past the last row
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

template <int kEPT>
__device__ __forceinline__ void load_slice(Slice<kEPT>& s, const TraceRsrc& rs, int r0) {
  // r0: first row of the lane's slice, relative to the resources' base row
#pragma unroll
  for (int j = 0; j < kEPT / 2; ++j) {
    const v4u32 v = __builtin_bit_cast(
        v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.ts, r0 * 8 + 16 * j, 0, 0));
    s.ts[2 * j] = (long long)(((unsigned long long)v.y << 32) | v.x);
    s.ts[2 * j + 1] = (long long)(((unsigned long long)v.w << 32) | v.z);
  }
  if constexpr (kEPT == 4) {
    s.mw[0] = __builtin_amdgcn_raw_buffer_load_b32(rs.model, r0, 0, 0);
    s.tw[0] = __builtin_amdgcn_raw_buffer_load_b32(rs.type, r0, 0, 0);
    const v2u32 k = __builtin_bit_cast(v2u32, __builtin_amdgcn_raw_buffer_load_b64(rs.tokens, r0 * 2, 0, 0));
    s.kw[0] = k.x; s.kw[1] = k.y;
  } else if constexpr (kEPT == 8) {
    const v2u32 m = __builtin_bit_cast(v2u32, __builtin_amdgcn_raw_buffer_load_b64(rs.model, r0, 0, 0));
    const v2u32 t = __builtin_bit_cast(v2u32, __builtin_amdgcn_raw_buffer_load_b64(rs.type, r0, 0, 0));
    const v4u32 k = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.tokens, r0 * 2, 0, 0));
    s.mw[0] = m.x; s.mw[1] = m.y;
    s.tw[0] = t.x; s.tw[1] = t.y;
    s.kw[0] = k.x; s.kw[1] = k.y; s.kw[2] = k.z; s.kw[3] = k.w;
  } else {
    static_assert(kEPT % 16 == 0, "kEPT is 4, 8 or a multiple of 16");
#pragma unroll
    for (int j = 0; j < kEPT / 16; ++j) {
      const v4u32 m = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.model, r0 + 16 * j, 0, 0));
      const v4u32 t = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.type, r0 + 16 * j, 0, 0));
      s.mw[4 * j] = m.x; s.mw[4 * j + 1] = m.y; s.mw[4 * j + 2] = m.z; s.mw[4 * j + 3] = m.w;
      s.tw[4 * j] = t.x; s.tw[4 * j + 1] = t.y; s.tw[4 * j + 2] = t.z; s.tw[4 * j + 3] = t.w;
    }
#pragma unroll
    for (int j = 0; j < kEPT / 8; ++j) {
      const v4u32 k = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.tokens, r0 * 2 + 16 * j, 0, 0));
      s.kw[4 * j] = k.x; s.kw[4 * j + 1] = k.y; s.kw[4 * j + 2] = k.z; s.kw[4 * j + 3] = k.w;
    }
  }
}

// Ring layout: window slot s, model m owns the four 64-bit words at
// s * (4M + 1) + 4m (the odd slot stride puts one model's cells of
// neighbouring windows on different LDS banks):
//   +0 tokens    P (low 32 bits) | D (high 32 bits)
//   +1 arrivals  (count << 32) + sum of te over the window's ARRIVE rows
//   +2 admits    (count << 32) + sum of te over its PREFILL|ADMIT rows
//   +3 finishes  (count << 32) + sum of te over its FINISH rows
// with te = t_end - ts in [1, window_ms]. The te sums stay below 2^31
// (events per window * window_ms < 2^31), so no low half carries into its
// count. From them, per window: dA = admits - finishes, dW = arrivals -
// admits, and the in-window integral terms sum(dA * te) and sum(dW * te)
// are the same differences of the te sums.
//
// A row adds one 64-bit word: PREFILL and DECODE rows their tokens to P or
// D, ARRIVE / ADMIT / FINISH rows (1 << 32) + te to their kind's word; an
// ADMIT row also adds its prompt tokens to P. The word and the kind come
// from a table indexed by code = kind | ADMIT >> 5 (4 bits per code:
// word index, bit 2 "high half", bit 3 "lifecycle word"):
//   0 ARRIVE -> word 1, lifecycle; 1 PREFILL -> P; 2 DECODE -> D;
//   3 FINISH -> word 3, lifecycle; 5 PREFILL|ADMIT -> word 2, lifecycle
//   (+ P); 4, 6, 7 (undefined bits, unvalidated input only) -> P.
constexpr uint32_t kRowTable = 0x00A0B409u;

// cb: byte offset of the row's cell (its word 0) in the ring
__device__ __forceinline__ void tally_row(unsigned long long* ring, uint32_t cb, uint32_t ty,
                                          uint32_t tok, uint32_t te) {
  const uint32_t code = (ty & 3u) | ((ty >> 5) & 4u);
  const uint32_t nib = __builtin_amdgcn_ubfe(kRowTable, code << 2, 4);
  // token rows (word 0): the tokens shifted into their half by 32 * "high
  // half" (nib * 8 is that for them); lifecycle rows: (1 << 32) + te
  const unsigned long long tv = (unsigned long long)tok << ((nib << 3) & 63u);
  const bool life = nib >= 8u;
  const uint32_t lo = life ? te : (uint32_t)tv, hi = life ? 1u : (uint32_t)(tv >> 32);
  unsigned char* const cell = (unsigned char*)ring + cb;
  atomicAdd((unsigned long long*)(cell + ((nib & 3u) << 3)), ((unsigned long long)hi << 32) | lo);
  if (code == 5u) atomicAdd((uint32_t*)cell, tok);  // the admitted request's first prompt chunk
}

// General tally of the lane's rows in [e0, e_end) whose window fits the
// ring [cbase, cbase + wcap), with per-row checks (first and last tiles of a
// trace, and tiles that reach past the ring). The first row that does not
// fit stops the lane and is published in *defer (relative to a0) with its
// window in *wdef; the lane holding row t_last (the tile's last) stores
// that row's window in *wlast. Offsets are 32-bit: timestamps are below
// 2^32 ms; a row whose high timestamp word is set (unvalidated input only)
// is skipped.
template <int kEPT>
__device__ __forceinline__ void tally_slice(const Slice<kEPT>& s, int c0, int a0, int e0, int e_end,
                                            int t_last, int cbase, uint32_t base_lo, uint32_t cap,
                                            uint32_t magic, uint32_t win32, uint32_t wmask,
                                            uint32_t sstride, uint32_t mlast,
                                            unsigned long long* ring, unsigned* defer, int* wdef,
                                            int* wlast) {
  const int lo0 = e0 - c0, hi0 = e_end - c0;
  const int lo = lo0 < 0 ? 0 : (lo0 > kEPT ? kEPT : lo0);
  const int hi = hi0 < 0 ? 0 : (hi0 > kEPT ? kEPT : hi0);
  int jdef = kEPT, wdf = INT_MAX;
  bool go = true;  // rows are sorted: the lane stops at its first row past the ring
#pragma unroll
  for (int j = 0; j < kEPT; ++j) {
    const long long ts = s.ts[j];
    if (go && j >= lo && j < hi && ((unsigned long long)ts >> 32) == 0) {
      const uint32_t d = (uint32_t)ts - base_lo;
      uint32_t q, r;
      div_window(d, magic, win32, q, r);
      const int w = cbase + (int)q;
      if (d >= cap) {
        jdef = j;
        wdf = w;
        go = false;
      } else {
        if (c0 + j == t_last) *wlast = w;
        uint32_t mdl = (s.mw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
        mdl = mdl < mlast ? mdl : mlast;
        const uint32_t ty = (s.tw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
        const uint32_t tok = (s.kw[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        tally_row(ring, (((uint32_t)w & wmask) * sstride + 4u * mdl) << 3, ty, tok, win32 - r);
      }
    }
  }
  if (__ballot(jdef < kEPT)) {  // some row of this wave waits for a later tile
    if (jdef < kEPT) {
      atomicMin(defer, (unsigned)(c0 + jdef - a0));
      atomicMin(wdef, wdf);
    }
  }
}

// Tally of a lane whose rows all lie in the trace with the last one inside
// the ring (rows are sorted, so every row fits): no per-row checks. Here
// d = ts - base < 2^31 and the quotient q = floor(d / window) < 2^8 is
// trunc((2d + 1) * fl(1 / (2 window))) in fp64: (2d + 1) / (2 window) lies
// at least 1/(2 window) >= 2^-24 away from every integer, far above the
// product's rounding error (below 2^-43). te = (q + 1) * window - d.
// Model bytes are clamped to M - 1, so unvalidated input cannot leave the
// ring.
template <int kEPT>
__device__ __forceinline__ void tally_fast(const Slice<kEPT>& s, uint32_t base_lo, double inv2_win,
                                           uint32_t win32, uint32_t cbm, uint32_t wmask,
                                           uint32_t sstride, uint32_t mlast, bool last, int cbase,
                                           unsigned long long* ring, int* wlast) {
  // (ts << 1) + odd = 2d + 1 (one shift-add: the compiler is not shown how
  // odd derives from base_lo); q * window + wb - ts = te
  uint32_t odd = 1u - 2u * base_lo;
  __asm__("" : "+s"(odd));
  const uint32_t wb = win32 + base_lo;
  const uint32_t sstride8 = sstride << 3;  // ring bytes per window slot
  uint32_t ql = 0;
#pragma unroll
  for (int j = 0; j < kEPT; ++j) {
    const uint32_t t = (uint32_t)s.ts[j];
    const uint32_t q = (uint32_t)((double)((t << 1) + odd) * inv2_win);
    const uint32_t te = __umul24(q, win32) + wb - t;
    ql = q;
    uint32_t mdl = (s.mw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
    mdl = mdl < mlast ? mdl : mlast;
    const uint32_t ty = (s.tw[j >> 2] >> (8 * (j & 3))) & 0xFFu;
    const uint32_t tok = (s.kw[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    tally_row(ring, __umul24((q + cbm) & wmask, sstride8) + (mdl << 5), ty, tok, te);
  }
  if (last) *wlast = cbase + (int)ql;
}

// x mod d for x < 2^32, with magic = floor(2^32 / d) (2^32 - 1 for d = 1):
// the multiply-high undershoots the quotient by at most one
__device__ __forceinline__ uint32_t mod_magic(uint32_t x, uint32_t d, uint32_t magic) {
  const uint32_t r = x - __umulhi(x, magic) * d;
  return r >= d ? r - d : r;
}

// ------------------------------------------------------- control rules
__device__ __forceinline__ unsigned long long dbits(double x) {
  return (unsigned long long)__double_as_longlong(x);
}

// Wave-wide min / max of a 32-bit value, broadcast as a scalar: butterfly
// within quads and rows (DPP quad_perm, half-row and row mirrors), then
// rows folded through row broadcasts; lane 63 ends with the result.
template <bool kMax>
__device__ __forceinline__ uint32_t wave_fold(uint32_t x) {
  // lanes a step does not reach read the identity, so each step is one
  // DPP-sourced min / max
  constexpr int id = kMax ? 0 : -1;
  auto op = [](uint32_t a, uint32_t b) { return kMax ? (a > b ? a : b) : (a < b ? a : b); };
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x140, 0xF, 0xF, false));  // row_mirror
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x142, 0xA, 0xF, false));  // row_bcast:15
  x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x143, 0xC, 0xF, false));  // row_bcast:31
  return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Lowest lane among the candidates (bit per lane in cand) holding the
// minimum (kMax: maximum) of Z, or -1. Z >= 0 and never NaN, so its bit
// pattern orders like its value: the high words decide, and the low words
// only where several candidates share the highest / lowest high word
// (for +inf the low word is zero).
template <bool kMax>
__device__ __forceinline__ int wave_arg(unsigned long long cand, double Z, int lane) {
  if (cand == 0ull) return -1;
  const bool c = (cand >> lane) & 1ull;
  const unsigned long long key = dbits(Z);
  const uint32_t hi = (uint32_t)(key >> 32), lo = (uint32_t)key;
  const uint32_t h = wave_fold<kMax>(c ? hi : (kMax ? 0u : 0xFFFFFFFFu));
  unsigned long long tie = __ballot(c && hi == h);
  if (__popcll(tie) > 1 && h != 0x7FF00000u) {
    const bool c2 = (tie >> lane) & 1ull;
    const uint32_t l = wave_fold<kMax>(c2 ? lo : (kMax ? 0u : 0xFFFFFFFFu));
    tie = __ballot(c2 && lo == l);
  }
  return __ffsll((long long)tie) - 1;
}

__device__ __forceinline__ double read_lane_f64(double x, int l) {
  const unsigned long long b = dbits(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

constexpr int kTickBlock = 8;  // ticks loaded and normalised per block

// Replica state of one scenario in the control replay, lane m = model m;
// pool and nm hold the same value in every lane.
struct CtlState {
  int R;          // routable replicas of the lane's model
  long long rw;   // replica-window sum over the windows before `since`
  int since;
  int pool;       // idle replicas (GPUs under the actuation model)
  uint32_t nm;    // moves decided so far
  int g;          // GPUs per replica (1 without the actuation model)
  // actuation: transition in flight (0 none, 1 wake, 2 sleep), the window at
  // whose end it completes, GPUs a sleep returns to the idle pool
  int tkind, tuntil, tret;
};

// Per-scenario constants of the replay, lane m = model m.
struct CtlConst {
  double tau_c, tau_s;
  int r_min;
  uint32_t K;                    // moves allowed per tick
  bool act;                      // the lane holds a model
  unsigned long long live_lanes;
  int32_t wake_w, sleep_w;       // actuation delays in windows
  tre_move* moves;               // the scenario's move log
  uint32_t move_cap;
};

// Transitions that completed before window w (actuation model only): a
// finished wake closes the lane's replica-window sum and raises R; finished
// sleeps return GPUs to the idle pool.
template <bool kAct>
__device__ __forceinline__ void ctl_complete(CtlState& st, int w) {
  if constexpr (kAct) {
    const bool done = st.tkind != 0 && st.tuntil < w;
    if (done && st.tkind == 1) {
      st.rw += (long long)st.R * (st.tuntil + 1 - st.since);
      st.since = st.tuntil + 1;
      st.R += 1;
    }
    unsigned long long back = __ballot(done && st.tkind == 2 && st.tret > 0);
    while (back) {
      const int l = __ffsll((long long)back) - 1;
      st.pool += __builtin_amdgcn_readlane(st.tret, l);
      back &= back - 1ull;
    }
    if (done) st.tkind = 0;
  }
}

// One tick of the control rules at the end of window w (tws: w in bits
// 0-29, kind in bits 30-31: bit 0 fast, bit 1 slow; wave-uniform), with the
// lane's normalised state Z (Eq. (2); +inf when idle or not initialised):
// the regions, the cadence rule, then up to K greedy moves with Eq. (3) for
// the receiver and the donor order of the bounded transfer. Every decision
// is wave-uniform (ballots are the candidate sets, receiver and donor are
// scalars). kAct adds the actuation model: the budget counts GPUs
// (footprint g per replica); a woken replica becomes routable wake_w
// windows after its wake starts; a donor's replica stops being routable at
// once and its GPUs reach the receiver after sleep_w windows, when the
// receiver's wake starts (any shortfall g_r - g_d comes from the idle GPUs
// at the move, any excess returns to them after the sleep); a model with a
// transition in flight is neither receiver nor donor; vetoed models do not
// release. A transition completing at the end of window u counts from
// window u + 1.
template <bool kAct>
__device__ __forceinline__ void ctl_tick(CtlState& st, const CtlConst& c, int lane, uint32_t tws, double Z,
                                         unsigned long long vetoed) {
  const int w = (int)(tws & 0x3FFFFFFFu);
  const uint32_t kind = tws >> 30;
  ctl_complete<kAct>(st, w);
  const unsigned long long crit = __ballot(c.act && Z < c.tau_c);
  unsigned long long ok;
  int path;
  if (crit) {
    if (!(kind & 1u)) return;  // rescue pending: rebalancing defers
    path = TRE_PATH_RESCUE;
    ok = crit;
  } else if (kind & 2u) {
    path = TRE_PATH_REBALANCE;
    ok = __ballot(c.act && Z < 1.0);
  } else {
    return;
  }
  const unsigned long long sur = __ballot(c.act && Z > c.tau_s);
  // models already in a transition: earlier in this tick, or in flight
  unsigned long long used = kAct ? __ballot(st.tkind != 0) : 0ull;
  // both halves widened as unsigned (a set bit 31 must not sign-extend)
  const unsigned long long veto_mask =
      kAct ? ((unsigned long long)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)vetoed) |
              ((unsigned long long)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(vetoed >> 32)) << 32))
           : 0ull;
  for (uint32_t k = 0; k < c.K; ++k) {
    const int r = wave_arg<false>(ok & ~used, Z, lane);  // Eq. (3)
    if (r < 0) break;
    const int g_r = kAct ? __builtin_amdgcn_readlane(st.g, r) : 1;
    int d;
    if (st.pool >= g_r) {
      st.pool -= g_r;
      d = TRE_DONOR_POOL;
      if (kAct && lane == r) {
        st.tkind = 1;
        st.tuntil = w + c.wake_w;
      }
    } else {
      const double Zr = read_lane_f64(Z, r);
      const unsigned long long cd =
          __ballot(c.act && st.R > c.r_min && Z > Zr && (!kAct || st.pool >= g_r - st.g)) & ~crit & ~used &
          ~(1ull << r) & c.live_lanes & ~veto_mask;
      d = wave_arg<true>(cd & sur, Z, lane);
      if (d < 0) d = wave_arg<true>(cd & ~sur, Z, lane);
      if (d < 0) break;
      used |= 1ull << d;
      if constexpr (kAct) {
        const int short_by = g_r - __builtin_amdgcn_readlane(st.g, d);
        if (short_by > 0) st.pool -= short_by;
        if (lane == d) {
          st.tkind = 2;
          st.tuntil = w + c.sleep_w;
          st.tret = short_by < 0 ? -short_by : 0;
        }
        if (lane == r) {
          st.tkind = 1;
          st.tuntil = w + c.sleep_w + c.wake_w;
        }
      }
    }
    used |= 1ull << r;
    // routable changes: the donor's at once (from w+1), the receiver's here
    // only without the actuation model (else when its wake completes)
    if (lane == d || (!kAct && lane == r)) {
      st.rw += (long long)st.R * (w + 1 - st.since);
      st.since = w + 1;
      st.R += lane == d ? -1 : 1;
    }
    if (lane == 0 && st.nm < c.move_cap) {
      tre_move mv;
      mv.window = (uint32_t)w;
      mv.path = (uint8_t)path;
      mv.receiver = (uint8_t)r;
      mv.donor = (uint8_t)d;
      mv.pad = 0;
      c.moves[st.nm] = mv;
    }
    ++st.nm;
  }
}

// One model's replay constants and state in LDS, for a replay that moves
// between waves from step to step.
struct CtlModel {
  double theta;     // theta * theta_scale
  double tau_c, tau_s;
  long long rw;
  int R, since, r_min, pad;
};

// Initial replica state of a scenario (lane m = model m): R = r_init, idle
// = budget - sum of g * r_init over the models.
__device__ __forceinline__ void ctl_init(CtlState& st, int r_init, int g, bool act, int budget) {
  st.R = act ? r_init : 0;
  st.g = g;
  int rsum = st.R * g;
  rsum += __shfl_xor(rsum, 1);
  rsum += __shfl_xor(rsum, 2);
  rsum += __shfl_xor(rsum, 4);
  rsum += __shfl_xor(rsum, 8);
  rsum += __shfl_xor(rsum, 16);
  rsum += __shfl_xor(rsum, 32);
  st.pool = budget - __builtin_amdgcn_readfirstlane(rsum);
  st.rw = 0;
  st.since = 0;
  st.nm = 0;
  st.tkind = 0;
  st.tuntil = 0;
  st.tret = 0;
}

// One workgroup per trace; every thread tallies and evaluates, one barrier
// per step. Step k, with [cA, cB) the chunk evaluated in step k-1 and
// [cB, cC), cC = min(wl, cB + C), the windows completed by earlier tiles
// (wl: the window of the last row tallied so far, or of the first row
// deferred):
//   - wave k % kWaves runs the smoothing chain over [cA, cB) from the
//     staging buffer of step k-1 (state in LDS, so the chain can move
//     between waves), its tick windows from one ballot; first, so that its
//     LDS reads find the queue the barrier just drained;
//   - read and clear the ring cells of [cB, cC): complete windows;
//   - issue the loads of tile k+1 and tally tile k into the ring: rows
//     whose window reaches cB + wcap wait for a later tile. Rows of tile k
//     come after every row of a complete window, so they land in windows
//     >= cC, on slots disjoint from the chunk's;
//   - evaluate [cB, cC), one (window, model) cell per thread: carry prefix
//     over the chunk, window integrals, Eq. (1) -> raw ratio, staged in LDS
//     (two staging buffers, by step parity);
//   -- barrier -- the tile's rows are in; windows < wl are complete.
template <int kWaves, int kEPT, bool kCells, bool kStage>
__device__ __forceinline__ void stream_body(const StreamParams& p) {
  constexpr int kThreads = kWaves * 64;
  constexpr long long kTile = (long long)kThreads * kEPT;
  extern __shared__ unsigned long long ring[];
  __shared__ int s_carry[2][2][TRE_MAX_MODELS];  // [parity][active, waiting][model], |count| < 2^27
  __shared__ double s_S[TRE_MAX_MODELS];               // smoothed TSS per model
  __shared__ double s_alpha[TRE_MAX_MODELS];
  __shared__ uint8_t s_init[TRE_MAX_MODELS];
  __shared__ int s_tick[3];                            // fast / slow counters, tick ordinal
  __shared__ unsigned s_defer[3];
  __shared__ int s_wdef[3];
  __shared__ int s_wlast[3];  // window of the tile's last row

  const int trace = blockIdx.x;
  const int tid = threadIdx.x;
  const int M = p.M;
  const uint32_t wcap = p.wcap;
  const int C = p.chunk;
  const uint32_t sstride = 4u * (uint32_t)M + 1u;  // ring words per window slot
  const int nring = (int)(wcap * sstride);
  // [nbuf][C][M] staged raw ratios (>= 0), -1 marks an idle window. Step k's
  // evaluation writes buffer k % nbuf and the smoothing chain of step k + 1
  // reads it; with the control replay in the stream the chain writes the
  // smoothed values of its tick windows back into it, and the replay reads
  // them in step k + 2 (hence three buffers)
  constexpr int nbuf = kStage ? 2 : 3;
  double* st_raw = (double*)(ring + nring);
  // kStage (no scalar TSS is written): the staged prefill ratios in the
  // scalar ratios' place and the decode ratios after them ([2][C][M] each,
  // -1 idle), then each model's smoothed shares and init flags
  double* const st_p = st_raw;
  double* const st_d = st_raw + 2 * C * M;
  double* const s_Sp = st_d + 2 * C * M;
  double* const s_Sd = s_Sp + M;
  uint8_t* const s_ip = (uint8_t*)(s_Sd + M);
  uint8_t* const s_id = s_ip + M;
  // the control replay (not kStage): one record per model, then idle
  // replicas, moves, and per staging buffer the fast- and slow-tick masks of
  // its chunk and the chunk's first window
  CtlModel* const s_cm = (CtlModel*)(st_raw + 3 * C * M);
  uint32_t* const s_cmeta = (uint32_t*)(s_cm + M);  // [0] idle, [1] moves, [2+b] fast, [5+b] slow, [8+b] window
  const long long e_begin = p.off[trace];
  const long long e_end = p.off[trace + 1];
  const long long win = p.window_ms;
  const uint32_t win32 = (uint32_t)win;
  const double dwin = (double)win;
  const int nW = p.n_windows;
  constexpr bool cells = kCells;

  for (int i = tid; i < nring; i += kThreads) ring[i] = 0ull;
  for (int i = tid; i < 2 * 2 * TRE_MAX_MODELS; i += kThreads) (&s_carry[0][0][0])[i] = 0;
  if (tid < 3) {
    s_defer[tid] = kNoDefer;
    s_wdef[tid] = INT_MAX;
    s_wlast[tid] = -1;
  }

  // the cell this thread evaluates: model rm, window offset rj in the chunk
  // (C is a power of two and C * M <= kEvalThreads <= threads; the rest have no cell)
  const int rm = tid / C, rj = tid & (C - 1);
  const bool r_thread = rm < M;
  // bit sh set where the lane 2^sh below lies in the same group of C lanes
  // (rj >= 2^sh, so never for 2^sh >= C); opaque to the compiler so that it
  // stays one per-lane register, not four lane masks held in SGPRs
  uint32_t r_take = 0;
#pragma unroll
  for (int sh = 0; sh < 4; ++sh) r_take |= rj >= (1 << sh) ? 1u << sh : 0u;
  __asm__("" : "+v"(r_take));
  double w_p = 0.0, w_q = 0.0;
  if (r_thread) {
    const tre_profile pr = p.prof[(int64_t)trace * M + rm];
    w_p = pr.w_p;
    w_q = pr.w_q;
  }
  // smoothing chain: one wave per step (rotating), lane m owns model m; its
  // state lives in LDS between steps
  if (tid < M) {
    s_alpha[tid] = p.prof[(int64_t)trace * M + tid].alpha;
    s_S[tid] = 0.0;
    s_init[tid] = 0;
    if constexpr (kStage) {
      s_Sp[tid] = 0.0;
      s_Sd[tid] = 0.0;
      s_ip[tid] = 0;
      s_id[tid] = 0;
    }
  }
  if (tid < 3) s_tick[tid] = 0;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;

  // the trace's one scenario, replayed here (else -1: the tick snapshot is
  // written for a separate replay)
  int ctl_s = -1;
  uint32_t ctl_K = 0;
  if constexpr (!kStage) {
    if (p.sc_count && p.sc_count[trace] == 1u) ctl_s = (int)p.sc_first[trace];
  }
  ctl_s = __builtin_amdgcn_readfirstlane(ctl_s);
  if (ctl_s >= 0) {
    const tre_scenario sc = p.sc[ctl_s];
    ctl_K = sc.max_moves;
    if (wave == 0) {
      const bool act = lane < M;
      const tre_profile pr = p.prof[(int64_t)trace * M + (act ? lane : 0)];
      CtlState st;
      ctl_init(st, pr.r_init, 1, act, p.budget);
      if (act) {
        CtlModel cm;
        cm.theta = pr.theta * sc.theta_scale;
        cm.tau_c = sc.tau_crit_override >= 0.0 ? sc.tau_crit_override : pr.tau_crit;
        cm.tau_s = pr.tau_surplus;
        cm.rw = 0;
        cm.R = st.R;
        cm.since = 0;
        cm.r_min = pr.r_min;
        cm.pad = 0;
        s_cm[lane] = cm;
      }
      if (lane < 11) s_cmeta[lane] = lane == 0 ? (uint32_t)st.pool : 0u;
    }
  }
  // the replay of the ticks the chain recorded in staging buffer b: state
  // from LDS, ctl_tick per tick in window order, state back to LDS; the
  // buffer's ticks are then consumed
  auto ctl_run = [&](int b) {
    const uint32_t tmf = (uint32_t)__builtin_amdgcn_readfirstlane((int)s_cmeta[2 + b]);
    const uint32_t tms = (uint32_t)__builtin_amdgcn_readfirstlane((int)s_cmeta[5 + b]);
    uint32_t tm = tmf | tms;
    if (!tm) return;
    const int w0 = __builtin_amdgcn_readfirstlane((int)s_cmeta[8 + b]);
    const bool act = lane < M;
    const int m = act ? lane : 0;
    CtlModel* const cm = s_cm + m;
    CtlState st;
    st.R = cm->R;
    st.rw = cm->rw;
    st.since = cm->since;
    st.pool = __builtin_amdgcn_readfirstlane((int)s_cmeta[0]);
    st.nm = (uint32_t)__builtin_amdgcn_readfirstlane((int)s_cmeta[1]);
    st.g = 1;
    st.tkind = 0;
    st.tuntil = 0;
    st.tret = 0;
    CtlConst c;
    c.tau_c = cm->tau_c;
    c.tau_s = cm->tau_s;
    c.r_min = cm->r_min;
    c.K = ctl_K;
    c.act = act;
    c.live_lanes = __ballot(act);
    c.wake_w = 0;
    c.sleep_w = 0;
    c.moves = p.moves + (int64_t)ctl_s * p.move_cap;
    c.move_cap = p.move_cap;
    const double th = cm->theta;
    const double* sb = st_raw + b * C * M + m;
    while (tm) {
      const int u = __ffs(tm) - 1;
      tm &= tm - 1u;
      const double Z = act ? sb[u * M] / th : INFINITY;  // Eq. (2); the buffer holds +inf when idle / not initialised
      const uint32_t kind = ((tmf >> u) & 1u) | (((tms >> u) & 1u) << 1);
      ctl_tick<false>(st, c, lane, (uint32_t)(w0 + u) | (kind << 30), Z, 0ull);
    }
    if (act) {
      cm->R = st.R;
      cm->rw = st.rw;
      cm->since = st.since;
    }
    if (lane == 0) {
      s_cmeta[0] = (uint32_t)st.pool;
      s_cmeta[1] = st.nm;
      s_cmeta[2 + b] = 0u;
      s_cmeta[5 + b] = 0u;
    }
  };

  // rows are counted from the trace's first kEPT-aligned row (below 2^27)
  const long long brow = e_begin & ~(long long)(kEPT - 1);
  const int rend = (int)(e_end - brow);  // one past the trace's last row
  int e0 = (int)(e_begin - brow);        // first row not yet tallied
  int cA = 0, cB = 0, wl = 0;
  TraceRsrc rs;
  rs.ts = rsrc(p.ts + brow, (long long)rend * 8);
  rs.model = rsrc(p.model + brow, rend);
  rs.type = rsrc(p.type + brow, rend);
  rs.tokens = rsrc(p.tokens + brow, (long long)rend * 2);
  Slice<kEPT> buf0, buf1;
  int held = 0;  // tile base held by the current buffer
  load_slice<kEPT>(buf0, rs, tid * kEPT);
  __syncthreads();

  // one step; returns true when every window has been smoothed
  auto step = [&](Slice<kEPT>& cur, Slice<kEPT>& nxt, int k) -> bool {
    if (cA >= nW) return true;
    const int b3 = k % 3;
    // ---- issue the loads of tile k+1 first (and of tile k again when the
    // prefetch missed it): with both buffers live from here on, nothing
    // below reuses a register a load is still filling
    const int a0 = e0 & ~(kEPT - 1);
    if (held != a0) load_slice<kEPT>(cur, rs, a0 + tid * kEPT);  // prefetch missed
    const int pref = a0 + (int)kTile;
    load_slice<kEPT>(nxt, rs, pref + tid * kEPT);  // zeros past the trace
    // ---- smooth [cA, cB) (staged last step); wave k mod kWaves, lanes < M
    if (wave == k % kWaves && cB > cA) {
      // the whole workgroup waits for this wave at the step's barrier: let its
      // dependent chain issue ahead of the other waves on its SIMD
      __builtin_amdgcn_s_setprio(3);
      const bool own = lane < M;
      const int m = own ? lane : 0;
      const int bc = (k + nbuf - 1) % nbuf;  // staged in step k - 1
      double* const pr = st_raw + bc * C * M + m;
      const double alpha = s_alpha[m];
      const double oma = 1.0 - alpha;
      double S = s_S[m];
      bool init = s_init[m] != 0;
      double Sp = 0.0, Sd = 0.0;
      bool ip = false, id = false;
      if constexpr (kStage) {
        Sp = s_Sp[m];
        Sd = s_Sd[m];
        ip = s_ip[m] != 0;
        id = s_id[m] != 0;
      }
      // windows since the last fast / slow tick before cA, ticks so far
      const uint32_t fctr = (uint32_t)__builtin_amdgcn_readfirstlane(s_tick[0]);
      const uint32_t sctr = (uint32_t)__builtin_amdgcn_readfirstlane(s_tick[1]);
      int tick = __builtin_amdgcn_readfirstlane(s_tick[2]);
      const int nw = cB - cA;
      // tick windows of the chunk: bit u for window cA + u (u < nw), fast
      // and slow cadences apart (scalar loops over the period ends)
      uint32_t tmf = 0u, tms = 0u;
      for (uint32_t u = (uint32_t)p.fast_w - 1u - fctr; u < (uint32_t)nw; u += (uint32_t)p.fast_w) tmf |= 1u << u;
      for (uint32_t u = (uint32_t)p.slow_w - 1u - sctr; u < (uint32_t)nw; u += (uint32_t)p.slow_w) tms |= 1u << u;
      const uint32_t tm = tmf | tms;
      for (int u0 = 0; u0 < nw; u0 += 4) {
        double rv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) rv[u] = pr[((u0 + u) & (C - 1)) * M];  // past nw: unused
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          if (u0 + u < nw) {
            const int w = cA + u0 + u;
            const double raw = rv[u];
            const bool idle = raw < 0.0;
            if constexpr (!kStage) {
              const double t1 = alpha * raw;
              const double t2 = oma * S;
              const double Sn = t1 + t2;
              S = idle ? S : (init ? Sn : raw);
              init = init || !idle;
            }
            if (cells && own) {
              const int64_t c = ((int64_t)trace * nW + w) * M + m;
              if (p.tss64) p.tss64[c] = S;
              if (p.tss32) p.tss32[c] = (float)S;
              if (p.flags) p.flags[c] = (uint8_t)((idle ? TRE_FLAG_IDLE : 0) | (init ? TRE_FLAG_INIT : 0));
            }
            if constexpr (kStage) {  // the stage shares: the same smoothing per stage
              const int j = ((u0 + u) & (C - 1)) * M + bc * C * M + m;
              const double rp = raw, rd = st_d[j];  // st_p is st_raw
              const bool pi = rp < 0.0, di = rd < 0.0;
              const double p1 = alpha * rp;
              const double p2 = oma * Sp;
              const double pn = p1 + p2;
              Sp = pi ? Sp : (ip ? pn : rp);
              ip = ip || !pi;
              const double d1 = alpha * rd;
              const double d2 = oma * Sd;
              const double dn = d1 + d2;
              Sd = di ? Sd : (id ? dn : rd);
              id = id || !di;
              if (own) {
                const int64_t c = ((int64_t)trace * nW + w) * M + m;
                if (p.stage64) *(double2*)(p.stage64 + 2 * c) = make_double2(Sp, Sd);
                if (p.stage32) *(float2*)(p.stage32 + 2 * c) = make_float2((float)Sp, (float)Sd);
                if (p.sflags)
                  p.sflags[c] = (uint8_t)((pi ? TRE_STAGE_P_IDLE : 0) | (ip ? TRE_STAGE_P_INIT : 0) |
                                          (di ? TRE_STAGE_D_IDLE : 0) | (id ? TRE_STAGE_D_INIT : 0));
              }
            }
            if ((tm >> (u0 + u)) & 1u) {
              const double zs = (idle || !init) ? INFINITY : S;
              if (ctl_s >= 0) {  // for the replay two steps on (the raw ratio is read already)
                if (own) pr[((u0 + u) & (C - 1)) * M] = zs;
              } else if (own && p.snap && tick < p.n_ticks) {
                p.snap[((int64_t)trace * p.n_ticks + tick) * M + m] = zs;
              }
              ++tick;
            }
          }
        }
      }
      if (own) {
        s_S[m] = S;
        s_init[m] = init ? 1 : 0;
        if constexpr (kStage) {
          s_Sp[m] = Sp;
          s_Sd[m] = Sd;
          s_ip[m] = ip ? 1 : 0;
          s_id[m] = id ? 1 : 0;
        }
      }
      if (lane == 0) {
        s_tick[0] = (int)mod_magic(fctr + (uint32_t)nw, (uint32_t)p.fast_w, p.magic_fast);
        s_tick[1] = (int)mod_magic(sctr + (uint32_t)nw, (uint32_t)p.slow_w, p.magic_slow);
        s_tick[2] = tick;
        if (ctl_s >= 0) {
          s_cmeta[2 + bc] = tmf;
          s_cmeta[5 + bc] = tms;
          s_cmeta[8 + bc] = (uint32_t)cA;
        }
      }
      __builtin_amdgcn_s_setprio(0);
    }
    // ---- read and clear the cells of [cB, cC), one cell per thread (groups
    // of C lanes per model): complete windows that no row of this tile
    // reaches. LDS operations of a wave retire in order, so these reads go
    // ahead of the tally's atomics.
    const int cC = wl < cB + C ? wl : cB + C;
    const int n = cC - cB;
    const bool valid = r_thread && rj < n;
    unsigned long long pd = 0, w_arr = 0, w_adm = 0, w_fin = 0;
    if (valid) {
      const uint32_t c = ((uint32_t)(cB + rj) & (wcap - 1)) * sstride + 4u * (uint32_t)rm;
      pd = ring[c];
      w_arr = ring[c + 1];
      w_adm = ring[c + 2];
      w_fin = ring[c + 3];
      ring[c] = 0ull;
      ring[c + 1] = 0ull;
      ring[c + 2] = 0ull;
      ring[c + 3] = 0ull;
    }
    // ---- tally tile k (tile k+1 loading meanwhile), capacity [cB, cB + wcap)
    const int t_last = (pref < rend ? pref : rend) - 1;
    {
      const int c0 = a0 + tid * kEPT;
      const uint32_t base_lo = (uint32_t)((long long)cB * win);
      const uint32_t cap = wcap * win32;
      const bool lane_fast = c0 >= e0 && c0 + kEPT <= rend && (uint32_t)cur.ts[kEPT - 1] - base_lo < cap;
      if (__ballot(!lane_fast) == 0ull)  // wave-uniform
        tally_fast<kEPT>(cur, base_lo, p.inv2_window, win32, (uint32_t)cB & (wcap - 1), wcap - 1, sstride,
                         (uint32_t)M - 1u, c0 + kEPT - 1 == t_last, cB, ring, &s_wlast[b3]);
      else
        tally_slice<kEPT>(cur, c0, a0, e0, rend, t_last, cB, base_lo, cap, p.magic, win32, wcap - 1,
                          sstride, (uint32_t)M - 1u, ring, &s_defer[b3], &s_wdef[b3], &s_wlast[b3]);
    }
    // ---- evaluate [cB, cC): carry prefix, window integrals, Eq. (1)
    const int* cin = s_carry[k & 1][0];
    int* cout = s_carry[(k + 1) & 1][0];
    double* sr = st_raw + (k % nbuf) * C * M;
    if (r_thread) {  // uniform over each group of C lanes
      // net active / waiting changes and their in-window integral terms
      const int ca = (int)((uint32_t)(w_adm >> 32) - (uint32_t)(w_fin >> 32));
      const int cw = (int)((uint32_t)(w_arr >> 32) - (uint32_t)(w_adm >> 32));
      const int la32 = (int)((uint32_t)w_adm - (uint32_t)w_fin);
      const int lw32 = (int)((uint32_t)w_arr - (uint32_t)w_adm);
      int ia = ca, iw = cw;  // inclusive prefix over the chunk's windows
      if (C <= 16) {
        uint32_t rt = r_take;  // re-read each step: the masks are not kept live across steps
        __asm__ volatile("" : "+v"(rt));
        // row shifts by 1, 2, 4, 8 lanes (groups are aligned inside a row),
        // each taken where the neighbour lies in the lane's own group; the
        // masks are per-lane integers, so no lane mask stays live in SGPRs
#define TRE_ROW_SHR_STAGE(sh)                                                   \
  {                                                                             \
    const int ya = __builtin_amdgcn_mov_dpp(ia, 0x110 | (1 << (sh)), 0xF, 0xF, true); \
    const int yw = __builtin_amdgcn_mov_dpp(iw, 0x110 | (1 << (sh)), 0xF, 0xF, true); \
    const int mk = __builtin_amdgcn_sbfe((int)rt, (sh), 1); /* -1 or 0 */       \
    ia += ya & mk;                                                              \
    iw += yw & mk;                                                              \
  }
        TRE_ROW_SHR_STAGE(0)
        TRE_ROW_SHR_STAGE(1)
        TRE_ROW_SHR_STAGE(2)
        TRE_ROW_SHR_STAGE(3)
#undef TRE_ROW_SHR_STAGE
      } else {
        for (int dd = 1; dd < C; dd <<= 1) {
          const int ya = __shfl_up(ia, dd, C);
          const int yw = __shfl_up(iw, dd, C);
          if (rj >= dd) {
            ia += ya;
            iw += yw;
          }
        }
      }
      if (valid) {
        const int w = cB + rj;
        const int A0 = cin[rm] + (ia - ca), W0 = cin[TRE_MAX_MODELS + rm] + (iw - cw);
        // the window integrals in fp64, exactly: a trace has fewer than 2^27
        // rows, so |A0|, |W0| < 2^27, A0 * window < 2^50 and the sum with the
        // in-window term (below 2^31) stays below 2^53
        const double A_f = __builtin_fma((double)A0, dwin, (double)la32);
        const double W_f = __builtin_fma((double)W0, dwin, (double)lw32);
        const uint32_t P = (uint32_t)pd, Dt = (uint32_t)(pd >> 32);
        const bool idle = pd == 0ull && A_f == 0.0 && W_f == 0.0;
        double raw = 0.0;
        if (!kStage && !idle) {
          // Eq. (1), evaluated in the documented order
          double num = w_p * (double)P;
          num = num + (double)Dt;
          num = num * 1000.0;
          const double q = w_q * W_f;
          double den = A_f + q;
          if (den < dwin) den = dwin;
          raw = num / den;
        }
        if constexpr (!kStage) sr[rj * M + rm] = idle ? -1.0 : raw;
        if constexpr (kStage) {
          // the two parts of Eq. (1), each with its one-request floor; a
          // stage is idle when its tokens and its demand integral are zero
          double rp = -1.0, rd = -1.0;
          if (P != 0u || W_f != 0.0) {
            double num = w_p * (double)P;
            num = num * 1000.0;
            double den = w_q * W_f;
            if (den < dwin) den = dwin;
            rp = num / den;
          }
          if (Dt != 0u || A_f != 0.0) {
            const double num = (double)Dt * 1000.0;
            double den = A_f;
            if (den < dwin) den = dwin;
            rd = num / den;
          }
          st_p[(k % nbuf) * C * M + rj * M + rm] = rp;
          st_d[(k % nbuf) * C * M + rj * M + rm] = rd;
        }
        if (cells) {
          const int64_t o = ((int64_t)trace * nW + w) * M + rm;
          if (p.prefill) p.prefill[o] = P;
          if (p.decode) p.decode[o] = Dt;
          if (p.a_int) p.a_int[o] = (long long)A0 * win + la32;
          if (p.w_int) p.w_int[o] = (long long)W0 * win + lw32;
        }
        if (rj == n - 1) {
          cout[rm] = cin[rm] + ia;
          cout[TRE_MAX_MODELS + rm] = cin[TRE_MAX_MODELS + rm] + iw;
        }
      }
    }
    if (n == 0 && tid < M) {
      cout[tid] = cin[tid];
      cout[TRE_MAX_MODELS + tid] = cin[TRE_MAX_MODELS + tid];
    }
    // ---- the control replay of the ticks the chain smoothed in step k - 1,
    // on another wave than this step's chain, after its tally (the tile it
    // tallied no longer holds registers)
    if (ctl_s >= 0 && wave == (k + kWaves / 2) % kWaves) {
      __builtin_amdgcn_s_setprio(3);
      ctl_run((k + 1) % 3);
      __builtin_amdgcn_s_setprio(0);
    }
    // entries rotate over three steps: step k writes entry k % 3, every wave
    // reads it right after the barrier that ends step k, and it is reset
    // here in step k + 2 (a barrier after those reads, a barrier before its
    // next use in step k + 3)
    if (tid == 0) {
      const int r = (k + 1) % 3;
      s_defer[r] = kNoDefer;
      s_wdef[r] = INT_MAX;
      s_wlast[r] = -1;
    }
    __syncthreads();
    // ---- the next tile and the completeness bound (same on every thread;
    // shared scalars are read into scalar registers)
    const unsigned dfr = (unsigned)__builtin_amdgcn_readfirstlane((int)s_defer[b3]);
    int en = a0 + (int)kTile;
    if (en > rend) en = rend;
    if (en < e0) en = e0;
    int wn;
    if (dfr != kNoDefer) {
      en = a0 + dfr;
      wn = __builtin_amdgcn_readfirstlane(s_wdef[b3]);
    } else if (en >= rend) {
      wn = nW;
    } else {
      wn = __builtin_amdgcn_readfirstlane(s_wlast[b3]);
    }
    wn = wn > nW ? nW : wn;
    e0 = en;
    wl = wn < wl ? wl : wn;
    held = pref;
    cA = cB;
    cB = cC;
    return false;
  };
  int k_end = 0;
  for (int k = 0;; k += 2) {
    if (step(buf0, buf1, k)) {
      k_end = k;
      break;
    }
    if (step(buf1, buf0, k + 1)) {
      k_end = k + 1;
      break;
    }
  }
  // the ticks of the last chunk, then the replay's outputs (the last step's
  // barrier made the chain's values visible)
  if (ctl_s >= 0 && wave == 0) {
    ctl_run((k_end + 1) % 3);
    if (lane < M) {
      const CtlModel cm = s_cm[lane];
      p.r_final[(int64_t)ctl_s * M + lane] = cm.R;
      p.r_windows[(int64_t)ctl_s * M + lane] = cm.rw + (long long)cm.R * (nW - cm.since);
    }
    if (lane == 0) p.n_moves[ctl_s] = s_cmeta[1];
  }
}

template <int kWaves, int kEPT, bool kCells>
__global__ __launch_bounds__(kWaves * 64) void tss_stream(StreamParams p) {
  stream_body<kWaves, kEPT, kCells, false>(p);
}

// the stage-share instantiation, held to 80 VGPRs so that six workgroups
// fit on a CU (its LDS allows six)
template <int kWaves, int kEPT>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(6))) void tss_stream_stage(
    StreamParams p) {
  stream_body<kWaves, kEPT, false, true>(p);
}

// --------------------------------------------------------------- rebalance
struct CtlParams {
  const tre_profile* prof;
  const tre_scenario* sc;
  uint32_t n_sc;
  const double* vals;     // snapshot [trace][tick][M] (flags NULL) or S [trace][w][M]
  const uint8_t* flags;   // per-cell flags, or NULL
  const uint32_t* tick_window;
  const uint8_t* tick_kind;  // bit 0 fast, bit 1 slow
  int32_t n_ticks;
  int32_t n_windows;
  int32_t M;
  int32_t budget;
  uint32_t n_traces;
  tre_move* moves;
  uint32_t move_cap;
  uint32_t* n_moves;
  int32_t* r_final;
  int64_t* r_windows;
  // actuation model (the kAct instantiation)
  int32_t wake_w;            // windows from a wake's start until routable
  int32_t sleep_w;           // windows a released replica hides, drains and sleeps
  const int32_t* footprint;  // [trace][M] GPUs per replica, or NULL (1)
  const uint64_t* veto;      // [trace][tick] donor releases refused, or NULL
  const uint32_t* sc_count;  // [trace] scenarios per trace of a sweep, or NULL
};

// One wave per scenario, lane m = model m: per tick Z = S / (theta * scale)
// (Eq. (2)), then ctl_tick. Scenarios whose trace streamed its own replay
// (sc_count[trace] == 1 in a sweep) are skipped.
template <bool kAct>
__global__ __launch_bounds__(256) void rebalance(CtlParams p) {
  const int lane = threadIdx.x & 63;
  const uint32_t s = (uint32_t)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
  if (s >= p.n_sc) return;  // whole wave
  const int M = p.M;
  const bool act = lane < M;
  const int mc = act ? lane : 0;
  const tre_scenario sc = p.sc[s];
  const uint32_t trace = sc.trace < p.n_traces ? sc.trace : 0;
  if (p.sc_count && p.sc_count[trace] == 1u) return;  // replayed in the stream
  const tre_profile pr = p.prof[(int64_t)trace * M + mc];
  const double theta_eff = pr.theta * sc.theta_scale;
  CtlConst c;
  c.tau_c = sc.tau_crit_override >= 0.0 ? sc.tau_crit_override : pr.tau_crit;
  c.tau_s = pr.tau_surplus;
  c.r_min = pr.r_min;
  c.K = sc.max_moves;
  c.act = act;
  c.live_lanes = __ballot(act);
  c.wake_w = p.wake_w;
  c.sleep_w = p.sleep_w;
  c.moves = p.moves + (int64_t)s * p.move_cap;
  c.move_cap = p.move_cap;
  int g = 1;
  if (kAct && p.footprint && act) g = p.footprint[(int64_t)trace * M + lane];
  CtlState st;
  ctl_init(st, pr.r_init, g, act, p.budget);

  const int nt = p.n_ticks;
  const int64_t tbase = (int64_t)trace * (p.flags ? p.n_windows : nt);
  // normalised values of ticks [t0, t0 + kTickBlock): unconditional loads
  // from clamped indices, then the divisions, independent of each other
  // (the tick's window, kind and vetoes ride along: loads that other
  // threads' stores might alias stay vector loads, so they are issued a
  // block ahead)
  auto load_block = [&](int t0, double (&v)[kTickBlock], uint32_t (&f)[kTickBlock],
                        uint32_t (&tw)[kTickBlock], unsigned long long (&vt)[kTickBlock]) {
#pragma unroll
    for (int u = 0; u < kTickBlock; ++u) {
      const int t = t0 + u < nt ? t0 + u : nt - 1;
      tw[u] = p.tick_window[t] | ((uint32_t)p.tick_kind[t] << 30);
      vt[u] = (kAct && p.veto) ? p.veto[(int64_t)trace * nt + t] : 0ull;
      if (p.flags) {
        const int64_t cc = (tbase + p.tick_window[t]) * M + mc;
        v[u] = p.vals[cc];
        f[u] = p.flags[cc];
      } else {
        v[u] = p.vals[(tbase + t) * M + mc];
        f[u] = TRE_FLAG_INIT;
      }
    }
  };
  auto normalise = [&](double (&v)[kTickBlock], const uint32_t (&f)[kTickBlock]) {
#pragma unroll
    for (int u = 0; u < kTickBlock; ++u) {
      const bool live = act && !(f[u] & TRE_FLAG_IDLE) && (f[u] & TRE_FLAG_INIT);
      v[u] = live ? v[u] / theta_eff : INFINITY;  // Eq. (2); +inf when idle or not initialised
    }
  };
  auto decide = [&](uint32_t twk, double Z, unsigned long long vetoed) {
    ctl_tick<kAct>(st, c, lane, (uint32_t)__builtin_amdgcn_readfirstlane((int)twk), Z, vetoed);
  };
  if (nt > 0) {
    double va[kTickBlock], vb[kTickBlock];
    uint32_t fa[kTickBlock], fb[kTickBlock], wa[kTickBlock], wb[kTickBlock];
    unsigned long long xa[kTickBlock], xb[kTickBlock];
    load_block(0, va, fa, wa, xa);
    for (int t0 = 0; t0 < nt; t0 += 2 * kTickBlock) {
      load_block(t0 + kTickBlock, vb, fb, wb, xb);
      normalise(va, fa);
#pragma unroll
      for (int u = 0; u < kTickBlock; ++u)
        if (t0 + u < nt) decide(wa[u], va[u], xa[u]);
      load_block(t0 + 2 * kTickBlock, va, fa, wa, xa);
      normalise(vb, fb);
#pragma unroll
      for (int u = 0; u < kTickBlock; ++u)
        if (t0 + kTickBlock + u < nt) decide(wb[u], vb[u], xb[u]);
    }
  }
  ctl_complete<kAct>(st, p.n_windows);  // transitions completing at the end of the last window count as done
  st.rw += (long long)st.R * (p.n_windows - st.since);
  if (act) {
    p.r_final[(int64_t)s * M + lane] = st.R;
    p.r_windows[(int64_t)s * M + lane] = st.rw;
  }
  if (lane == 0) p.n_moves[s] = st.nm;
}

// ---------------------------------------------------------------- validate
// Error kinds of the load-time checks, one bit and one lowest-row slot each.
enum { kValOrder = 0, kValSchema = 1, kValRange = 2, kValState = 3, kValKinds = 4 };

struct ValParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint8_t* type;
  const int64_t* off;
  uint32_t n_traces;
  int64_t duration_ms;
  int64_t window_ms;
  int32_t M;
  int64_t max_per_window;
  unsigned* err;             // bit k: an error of kind k
  unsigned long long* first; // [kValKinds] lowest failing row of each kind
};

constexpr int kValChunk = 16384;

__global__ __launch_bounds__(256) void validate(ValParams p) {
  for (uint32_t t = blockIdx.y; t < p.n_traces; t += gridDim.y) {
    const int64_t b = p.off[t], e = p.off[t + 1];
    const int64_t c0 = b + (int64_t)blockIdx.x * kValChunk;
    if (c0 >= e) continue;
    const int64_t c1 = c0 + kValChunk < e ? c0 + kValChunk : e;
    for (int64_t i = c0 + threadIdx.x; i < c1; i += 256) {
      const int64_t t_i = p.ts[i];
      const uint32_t ty = p.type[i];
      unsigned bad = 0;
      if (t_i < 0 || t_i >= p.duration_ms || (i > b && t_i < p.ts[i - 1])) bad |= 1u << kValOrder;
      if (p.model[i] >= p.M || (ty & 0x7Cu) || ((ty & TRE_ADMIT) && (ty & 3u) != TRE_PREFILL))
        bad |= 1u << kValSchema;
      const int64_t j = i + p.max_per_window;
      if (!(bad & 1u) && j < e && p.ts[j] / p.window_ms == t_i / p.window_ms) bad |= 1u << kValRange;
      if (bad) {
        atomicOr(p.err, bad);
        for (int k = 0; k < kValState; ++k)
          if (bad & (1u << k)) atomicMin(&p.first[k], (unsigned long long)i);
      }
    }
  }
}

// A_m(t) and W_m(t) of Eq. (1) count active and waiting requests, so a
// stream whose transitions take either below zero at some instant is
// invalid. They are right-continuous step functions: the value at t counts
// every row with ts <= t, so only the counts after the last row of an
// instant are checked (rows of one instant may come in any order). For
// model m that is the count after its last row with that timestamp.
//
// One wave per trace (the trace's rows are already known sorted, with valid
// models and types), 64 rows per step, one per lane. Rows of the same model
// are found with ballots over the model's bits; a lane's count is its
// model's carry plus the signed transitions of the same-model lanes up to
// it. A row whose next same-model row in the step has a later timestamp is
// the last of its instant and is checked at once; the model's last row of a
// step is checked when the model's next row (in a later step) has a later
// timestamp, or at the end of the trace. Per-model state (carries, the
// timestamp and row of the last row seen) lives in the wave's LDS slice.
struct StateParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint8_t* type;
  const int64_t* off;
  uint32_t n_traces;
  int32_t M;
  unsigned* err;
  unsigned long long* first;
};

__global__ __launch_bounds__(256) void validate_state(StateParams p) {
  __shared__ int s_a[4][TRE_MAX_MODELS], s_w[4][TRE_MAX_MODELS];  // counts after the rows seen
  __shared__ long long s_t[4][TRE_MAX_MODELS];                     // timestamp of the model's last row, -1 none
  __shared__ long long s_r[4][TRE_MAX_MODELS];                     // that row
  const int wv = (int)(threadIdx.x >> 6), lane = (int)(threadIdx.x & 63);
  const uint32_t t = blockIdx.x * 4u + (uint32_t)wv;
  if (t >= p.n_traces) return;  // whole wave; the waves share no barrier
  int* ca = s_a[wv];
  int* cw = s_w[wv];
  long long* lt = s_t[wv];
  long long* lr = s_r[wv];
  ca[lane] = 0;
  cw[lane] = 0;
  lt[lane] = -1;
  lr[lane] = 0;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int nbits = p.M > 1 ? 32 - __clz(p.M - 1) : 0;
  const unsigned long long le = (2ull << lane) - 1ull;  // lanes <= this one
  const int64_t b = p.off[t], e = p.off[t + 1];
  long long bad = LLONG_MAX;
  // rows of the next step are loaded before the current one is processed
  auto load = [&](int64_t i, long long& ts, uint32_t& m, uint32_t& ty) {
    const bool v = i < e;
    ts = v ? (long long)p.ts[i] : 0;
    m = v ? (uint32_t)p.model[i] & 63u : 0u;
    ty = v ? (uint32_t)p.type[i] : 0xFFu;
  };
  long long tsn;
  uint32_t mn, tyn;
  load(b + lane, tsn, mn, tyn);
  for (int64_t r0 = b; r0 < e; r0 += 64) {
    const int64_t i = r0 + lane;
    const bool v = i < e;
    const long long ts = tsn;
    const uint32_t m = mn, ty = tyn;
    load(i + 64, tsn, mn, tyn);
    const int dA = (ty == (TRE_PREFILL | TRE_ADMIT) ? 1 : 0) - (ty == TRE_FINISH ? 1 : 0);
    const int dW = (ty == TRE_ARRIVE ? 1 : 0) - (ty == (TRE_PREFILL | TRE_ADMIT) ? 1 : 0);
    unsigned long long same = __ballot(v);
    for (int k = 0; k < nbits; ++k) {
      const unsigned long long bk = __ballot((m >> k) & 1u);
      same &= ((m >> k) & 1u) ? bk : ~bk;
    }
    const unsigned long long pa = __ballot(dA > 0), na = __ballot(dA < 0);
    const unsigned long long pw = __ballot(dW > 0), nw = __ballot(dW < 0);
    const unsigned long long upto = same & le;
    const int va = ca[m] + __popcll(pa & upto) - __popcll(na & upto);
    const int vw = cw[m] + __popcll(pw & upto) - __popcll(nw & upto);
    const unsigned long long after = same & ~le;
    const int nl = after ? __ffsll((long long)after) - 1 : lane;
    const long long tnext = __shfl(ts, nl);
    // the last row of its instant inside this step
    if (v && after && tnext != ts && (va < 0 || vw < 0)) bad = bad < i ? bad : i;
    // the model's first row in this step settles its last row of an earlier step
    if (v && (upto & ~(1ull << lane)) == 0ull) {
      const long long tp = lt[m];
      if (tp >= 0 && tp != ts && (ca[m] < 0 || cw[m] < 0)) bad = bad < lr[m] ? bad : lr[m];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (v && !after) {  // the model's last row in this step
      ca[m] = va;
      cw[m] = vw;
      lt[m] = ts;
      lr[m] = i;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // each model's last row is the last of its instant
  if (lane < p.M && lt[lane] >= 0 && (ca[lane] < 0 || cw[lane] < 0)) bad = bad < lr[lane] ? bad : lr[lane];
  if (bad != LLONG_MAX) {
    atomicOr(p.err, 1u << kValState);
    atomicMin(p.first, (unsigned long long)bad);
  }
}

// A request is admitted once (its first prefill chunk carries the ADMIT
// bit). With request ids given, pass 1 finds the largest admitted id of
// each trace; pass 2 sets one bit per admitted id in a per-trace bitmap
// and records the smallest (trace, id) whose bit was already set.
struct AdmitParams {
  const uint32_t* req;
  const uint8_t* type;
  const int64_t* off;
  uint32_t t0, n_traces;        // traces [t0, t0 + n_traces) of this launch
  uint32_t* maxid;              // pass 1: [all traces] largest admitted id
  const uint64_t* word_off;     // pass 2: [all traces] first bitmap word of each trace
  uint64_t word_base;           // word_off of trace t0
  uint32_t* bits;               // pass 2: bitmaps of this launch's traces
  unsigned long long* dup;      // pass 2: smallest (trace << 32 | id) admitted twice
};

template <bool kMark>
__global__ __launch_bounds__(256) void admit_scan(AdmitParams p) {
  for (uint32_t tt = blockIdx.y; tt < p.n_traces; tt += gridDim.y) {
    const uint32_t t = p.t0 + tt;
    const int64_t b = p.off[t], e = p.off[t + 1];
    const int64_t c0 = b + (int64_t)blockIdx.x * kValChunk;
    if (c0 >= e) continue;  // uniform over the block
    const int64_t c1 = c0 + kValChunk < e ? c0 + kValChunk : e;
    uint32_t mx = 0;
    for (int64_t i = c0 + threadIdx.x; i < c1; i += 256) {
      if (p.type[i] != (TRE_PREFILL | TRE_ADMIT)) continue;
      const uint32_t id = p.req[i];
      if constexpr (!kMark) {
        mx = id > mx ? id : mx;
      } else {
        if ((uint64_t)(id >> 5) >= p.word_off[t + 1] - p.word_off[t]) continue;  // above pass 1's largest id
        const uint32_t bit = 1u << (id & 31u);
        const uint32_t old = atomicOr(&p.bits[p.word_off[t] - p.word_base + (id >> 5)], bit);
        if (old & bit) atomicMin(p.dup, ((unsigned long long)t << 32) | id);
      }
    }
    if constexpr (!kMark) {
      for (int d = 32; d >= 1; d >>= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)mx, d);
        mx = o > mx ? o : mx;
      }
      if ((threadIdx.x & 63) == 0 && mx) atomicMax(&p.maxid[t], mx);
    }
  }
}

// A request arrives once, finishes once, and neither arrives nor decodes
// after it finished (rows of its FINISH instant in any order): the request
// counts of Eq. (1) follow one lifecycle per id. Pass 0 finds the largest
// id of an ARRIVE or FINISH row per trace; pass 1 marks each id's ARRIVE in
// a bitmap and stores its FINISH timestamp (a second one of either is an
// error); pass 2 checks every ARRIVE and DECODE row against the FINISH
// timestamp of its id. The smallest (trace, id) in error is kept.
struct LifeParams {
  const int64_t* ts;
  const uint32_t* req;
  const uint8_t* type;
  const int64_t* off;
  uint32_t t0, n_traces;        // traces [t0, t0 + n_traces) of this launch
  uint32_t* maxid;              // pass 0: [all traces] largest id of an ARRIVE or FINISH row
  const uint64_t* slot_off;     // passes 1, 2: [all traces] first slot of each trace's ids
  uint64_t slot_base;           // slot_off of trace t0
  uint32_t* fin;                // FINISH timestamp per slot, 0xFFFFFFFF when none
  uint32_t* arr;                // ARRIVE bit per slot
  unsigned long long* bad;      // smallest (trace << 32 | id) in error
};

template <int kPass>
__global__ __launch_bounds__(256) void life_scan(LifeParams p) {
  for (uint32_t tt = blockIdx.y; tt < p.n_traces; tt += gridDim.y) {
    const uint32_t t = p.t0 + tt;
    const int64_t b = p.off[t], e = p.off[t + 1];
    const int64_t c0 = b + (int64_t)blockIdx.x * kValChunk;
    if (c0 >= e) continue;  // uniform over the block
    const int64_t c1 = c0 + kValChunk < e ? c0 + kValChunk : e;
    uint32_t mx = 0;
    for (int64_t i = c0 + threadIdx.x; i < c1; i += 256) {
      const uint32_t ty = p.type[i], kind = ty & 3u, id = p.req[i];
      if constexpr (kPass == 0) {
        if ((kind == TRE_ARRIVE || kind == TRE_FINISH) && id > mx) mx = id;
      } else {
        if ((uint64_t)id >= p.slot_off[t + 1] - p.slot_off[t]) continue;  // no ARRIVE or FINISH of this id
        const uint64_t sl = p.slot_off[t] - p.slot_base + id;
        const uint32_t ts = (uint32_t)p.ts[i];  // timestamps lie in [0, duration) below 2^32
        bool err = false;
        if constexpr (kPass == 1) {
          if (kind == TRE_ARRIVE) {
            const uint32_t bit = 1u << (sl & 31u);
            err = (atomicOr(&p.arr[sl >> 5], bit) & bit) != 0;
          } else if (kind == TRE_FINISH) {
            err = atomicCAS(&p.fin[sl], 0xFFFFFFFFu, ts) != 0xFFFFFFFFu;
          }
        } else {
          if (kind == TRE_ARRIVE || kind == TRE_DECODE) {
            const uint32_t f = p.fin[sl];
            err = f != 0xFFFFFFFFu && ts > f;
          }
        }
        if (err) atomicMin(p.bad, ((unsigned long long)t << 32) | id);
      }
    }
    if constexpr (kPass == 0) {
      for (int d = 32; d >= 1; d >>= 1) {
        const uint32_t o = (uint32_t)__shfl_xor((int)mx, d);
        mx = o > mx ? o : mx;
      }
      if ((threadIdx.x & 63) == 0 && mx) atomicMax(&p.maxid[t], mx);
    }
  }
}

// ------------------------------------------------------------------ timing
namespace {
struct Pending {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_tmu;
bool g_timing = false;
std::vector<Pending> g_pending;

}  // namespace

static thread_local int g_no_timing = 0;

tre_internal::NoTimingScope::NoTimingScope() { ++g_no_timing; }
tre_internal::NoTimingScope::~NoTimingScope() { --g_no_timing; }

tre_internal::LaunchTimer::LaunchTimer(const char* name, hipStream_t s) : st_(s) {
  if (g_no_timing) return;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!g_timing) return;
  name_ = name;
  if (hipEventCreate(&start_) != hipSuccess) return;
  if (hipEventCreate(&stop_) != hipSuccess) {
    (void)hipEventDestroy(start_);
    return;
  }
  on_ = hipEventRecord(start_, st_) == hipSuccess;
}

void tre_internal::LaunchTimer::done() {
  if (!on_) return;
  (void)hipEventRecord(stop_, st_);
  std::lock_guard<std::mutex> lk(g_tmu);
  g_pending.push_back(Pending{name_, start_, stop_});
  on_ = false;
}


extern "C" int tre_set_timing(int enable) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing = enable != 0;
  return TRE_OK;
}

extern "C" int tre_kernel_time(const char* kernel, double* total_ms, uint64_t* launches) {
  if (!kernel || !total_ms || !launches) return fail(TRE_EINVAL, "tre_kernel_time: NULL argument");
  std::vector<Pending> mine;
  {
    std::lock_guard<std::mutex> lk(g_tmu);
    std::vector<Pending> rest;
    for (auto& pe : g_pending) (strcmp(pe.name, kernel) == 0 ? mine : rest).push_back(pe);
    g_pending.swap(rest);
  }
  double tot = 0.0;
  int rc = TRE_OK;
  for (auto& pe : mine) {
    float ms = 0.f;
    if (hipEventSynchronize(pe.stop) != hipSuccess ||
        hipEventElapsedTime(&ms, pe.start, pe.stop) != hipSuccess)
      rc = fail(TRE_EHIP, "tre_kernel_time: event query failed");
    tot += ms;
    (void)hipEventDestroy(pe.start);
    (void)hipEventDestroy(pe.stop);
  }
  *total_ms = tot;
  *launches = mine.size();
  return rc;
}

// --------------------------------------------------------------- host ABI
int tre_internal::check_device(const tre_events* ev) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ev->device)
    return fail(TRE_EINVAL, "handle belongs to device %d, current device is %d", ev->device, dev);
  return TRE_OK;
}

// events one window of one trace may hold: the packed per-window sums stay
// inside their 32-bit halves
static int64_t max_events_per_window(int64_t window_ms) {
  const int64_t by_integral = 2147483647ll / window_ms;
  return by_integral < TRE_MAX_EVENTS_PER_WINDOW ? by_integral : TRE_MAX_EVENTS_PER_WINDOW;
}

static uint32_t ring_windows(int M) {
  uint32_t w = 256;
  while (w > 2 && (size_t)w * (4 * (size_t)M + 1) * 8 > (size_t)kRingBytes) w >>= 1;
  return w;
}

// windows evaluated per step: a power of two, one cell per thread of the
// first kEvalThreads, at most half the ring (the same for every workgroup
// size, so the LDS layout does not depend on it)
static int chunk_windows(int M, uint32_t wcap) {
  int c = 32;
  while (c > 1 && (c * M > kEvalThreads || c > (int)wcap / 2)) c >>= 1;
  return c;
}

// Waves per tss_stream workgroup. One workgroup streams one trace; with 4
// waves (about 75 VGPRs) six fit on a CU, so 1536 traces fill the chip.
// With fewer traces the resident workgroups alone cannot keep enough loads
// in flight, so each trace gets a larger workgroup: 16 waves (one per CU,
// four per SIMD) up to 384 traces, 8 waves up to 768.
static int stream_waves(uint32_t n_traces) {
  return n_traces <= 384 ? 16 : (n_traces <= 768 ? 8 : kStreamWaves);
}

static size_t stream_lds(const tre_events* ev, bool stage = false) {
  const size_t M = (size_t)ev->cfg.n_models, C = (size_t)chunk_windows(ev->cfg.n_models, ev->wcap);
  const size_t ring = ev->wcap * (4 * M + 1) * 8;
  // stage: two staging buffers of prefill ratios (in the scalar ratios'
  // place) and two of decode ratios, two shares and two flags per model
  if (stage) return ring + 4 * C * M * 8 + 2 * M * 8 + ((2 * M + 7) & ~(size_t)7);
  // three staging buffers, then the control replay's per-model records and
  // 11 words
  return ring + 3 * C * M * 8 + M * sizeof(CtlModel) + ((11 * 4 + 7) & ~(size_t)7);
}

// The load-time checks (synchronous): order, schema and per-window range
// of every row; then, on valid rows, counts never negative; then, with
// request ids, no id admitted twice. The error reported is the kind of the
// lowest failing row among the first three kinds (order before schema
// before range on one row), else a negative count (its lowest row), else a
// duplicate admission (the smallest trace, then id).
static int validate_events(const tre_events* ev, hipStream_t st) {
  const uint32_t n_traces = ev->n_traces;
  const tre_trace_cfg& c = ev->cfg;
  int64_t maxlen = 0;
  for (uint32_t i = 0; i < n_traces; ++i) maxlen = std::max<int64_t>(maxlen, ev->h_off[i + 1] - ev->h_off[i]);
  if (maxlen == 0) return TRE_OK;
  // err (8 bytes), first rows [kValKinds], duplicate key
  struct Slots {
    unsigned err, pad;
    unsigned long long first[kValKinds];
    unsigned long long dup, life;
  } h;
  void* slots = nullptr;
  if (hipMalloc(&slots, sizeof(Slots)) != hipSuccess) return fail(TRE_EHIP, "hipMalloc failed");
  Slots* d = (Slots*)slots;
  memset(&h, 0xFF, sizeof h);
  h.err = 0;
  h.pad = 0;
  const dim3 grid((unsigned)((maxlen + kValChunk - 1) / kValChunk), std::min<uint32_t>(n_traces, 65535u));
  auto readback = [&]() {
    return hipMemcpyAsync(&h, d, sizeof h, hipMemcpyDeviceToHost, st) == hipSuccess &&
           hipStreamSynchronize(st) == hipSuccess;
  };
  bool ok = hipMemcpyAsync(d, &h, sizeof h, hipMemcpyHostToDevice, st) == hipSuccess;
  if (ok) {
    ValParams vp{ev->ts, ev->model, ev->type, ev->d_off, n_traces, c.duration_ms, c.window_ms, c.n_models,
                 max_events_per_window(c.window_ms), &d->err, d->first};
    LaunchTimer lt("validate", st);
    hipLaunchKernelGGL(validate, grid, dim3(256), 0, st, vp);
    ok = hipGetLastError() == hipSuccess;
    lt.done();
  }
  ok = ok && readback();
  int rc = TRE_OK;
  if (ok && h.err) {
    int kind = -1;
    for (int k = 0; k < kValState; ++k)
      if ((h.err >> k & 1u) && (kind < 0 || h.first[k] < h.first[kind])) kind = k;
    const unsigned long long row = h.first[kind];
    if (kind == kValOrder) rc = fail(TRE_EORDER, "row %llu: timestamp unsorted or outside [0, duration)", row);
    else if (kind == kValSchema) rc = fail(TRE_ESCHEMA, "row %llu: model index or type byte invalid", row);
    else
      rc = fail(TRE_ERANGE, "row %llu: more than %lld events in one window", row,
                (long long)max_events_per_window(c.window_ms));
  }
  if (ok && rc == TRE_OK) {
    StateParams sp{ev->ts, ev->model, ev->type, ev->d_off, n_traces, c.n_models, &d->err, &d->first[kValState]};
    hipLaunchKernelGGL(validate_state, dim3((n_traces + 3) / 4), dim3(256), 0, st, sp);
    ok = hipGetLastError() == hipSuccess && readback();
    if (ok && (h.err >> kValState & 1u))
      rc = fail(TRE_ESTATE, "row %llu: an active or waiting count below zero after this instant",
                h.first[kValState]);
  }
  if (ok && rc == TRE_OK && ev->req) {
    // pass 1: largest admitted id per trace; then bitmaps of at most 2^26
    // words (256 MiB) at a time, or one trace's if larger
    uint32_t* d_max = nullptr;
    uint64_t* d_woff = nullptr;
    uint32_t* d_bits = nullptr;
    std::vector<uint32_t> hmax(n_traces);
    std::vector<uint64_t> woff(n_traces + 1);
    ok = hipMalloc(&d_max, sizeof(uint32_t) * n_traces) == hipSuccess &&
         hipMemsetAsync(d_max, 0, sizeof(uint32_t) * n_traces, st) == hipSuccess;
    AdmitParams ap{};
    ap.req = ev->req;
    ap.type = ev->type;
    ap.off = ev->d_off;
    ap.maxid = d_max;
    ap.dup = &d->dup;
    for (uint32_t t0 = 0; ok && t0 < n_traces; t0 += 65535u) {
      ap.t0 = t0;
      ap.n_traces = std::min<uint32_t>(n_traces - t0, 65535u);
      hipLaunchKernelGGL(admit_scan<false>, dim3(grid.x, ap.n_traces), dim3(256), 0, st, ap);
      ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipMemcpyAsync(hmax.data(), d_max, sizeof(uint32_t) * n_traces, hipMemcpyDeviceToHost, st) ==
                   hipSuccess &&
         hipStreamSynchronize(st) == hipSuccess;
    woff[0] = 0;
    uint64_t most = 0;
    for (uint32_t t = 0; t < n_traces; ++t) {
      const uint64_t w = (uint64_t)(hmax[t] >> 5) + 1u;
      woff[t + 1] = woff[t] + w;
      most = std::max(most, w);
    }
    const uint64_t cap = std::max<uint64_t>(most, std::min<uint64_t>(woff[n_traces], 1ull << 26));
    ok = ok && hipMalloc(&d_woff, sizeof(uint64_t) * (n_traces + 1)) == hipSuccess &&
         hipMalloc(&d_bits, sizeof(uint32_t) * cap) == hipSuccess &&
         hipMemcpyAsync(d_woff, woff.data(), sizeof(uint64_t) * (n_traces + 1), hipMemcpyHostToDevice, st) ==
             hipSuccess;
    ap.word_off = d_woff;
    ap.bits = d_bits;
    for (uint32_t t0 = 0; ok && t0 < n_traces;) {
      uint32_t t1 = t0 + 1;
      while (t1 < n_traces && t1 - t0 < 65535u && woff[t1 + 1] - woff[t0] <= cap) ++t1;
      int64_t len = 0;
      for (uint32_t t = t0; t < t1; ++t) len = std::max<int64_t>(len, ev->h_off[t + 1] - ev->h_off[t]);
      ap.t0 = t0;
      ap.n_traces = t1 - t0;
      ap.word_base = woff[t0];
      ok = hipMemsetAsync(d_bits, 0, sizeof(uint32_t) * (woff[t1] - woff[t0]), st) == hipSuccess;
      if (ok && len > 0) {
        hipLaunchKernelGGL(admit_scan<true>, dim3((unsigned)((len + kValChunk - 1) / kValChunk), t1 - t0),
                           dim3(256), 0, st, ap);
        ok = hipGetLastError() == hipSuccess;
      }
      t0 = t1;
    }
    ok = ok && readback();
    if (d_max) (void)hipFree(d_max);
    if (d_woff) (void)hipFree(d_woff);
    if (d_bits) (void)hipFree(d_bits);
    if (ok && h.dup != ~0ull)
      rc = fail(TRE_ESTATE, "trace %u: request id %u admitted more than once", (unsigned)(h.dup >> 32),
                (unsigned)h.dup);
  }
  if (ok && rc == TRE_OK && ev->req) {
    // the lifecycle of each id: pass 0 sizes per-trace tables (ids up to the
    // largest ARRIVE or FINISH id), passes 1 and 2 run over batches of at
    // most 2^26 slots (256 MiB of FINISH timestamps), or one trace if larger
    uint32_t* d_max = nullptr;
    uint64_t* d_soff = nullptr;
    uint32_t* d_fin = nullptr;
    uint32_t* d_arr = nullptr;
    std::vector<uint32_t> hmax(n_traces);
    std::vector<uint64_t> soff(n_traces + 1);
    ok = hipMalloc(&d_max, sizeof(uint32_t) * n_traces) == hipSuccess &&
         hipMemsetAsync(d_max, 0, sizeof(uint32_t) * n_traces, st) == hipSuccess;
    LifeParams lp{};
    lp.ts = ev->ts;
    lp.req = ev->req;
    lp.type = ev->type;
    lp.off = ev->d_off;
    lp.maxid = d_max;
    lp.bad = &d->life;
    for (uint32_t t0 = 0; ok && t0 < n_traces; t0 += 65535u) {
      lp.t0 = t0;
      lp.n_traces = std::min<uint32_t>(n_traces - t0, 65535u);
      hipLaunchKernelGGL(life_scan<0>, dim3(grid.x, lp.n_traces), dim3(256), 0, st, lp);
      ok = hipGetLastError() == hipSuccess;
    }
    ok = ok && hipMemcpyAsync(hmax.data(), d_max, sizeof(uint32_t) * n_traces, hipMemcpyDeviceToHost, st) ==
                   hipSuccess &&
         hipStreamSynchronize(st) == hipSuccess;
    soff[0] = 0;
    uint64_t most = 0;
    for (uint32_t t = 0; t < n_traces; ++t) {
      const uint64_t n = (uint64_t)hmax[t] + 1u;
      soff[t + 1] = soff[t] + n;
      most = std::max(most, n);
    }
    const uint64_t cap = std::max<uint64_t>(most, std::min<uint64_t>(soff[n_traces], 1ull << 26));
    ok = ok && hipMalloc(&d_soff, sizeof(uint64_t) * (n_traces + 1)) == hipSuccess &&
         hipMalloc(&d_fin, sizeof(uint32_t) * cap) == hipSuccess &&
         hipMalloc(&d_arr, sizeof(uint32_t) * (cap / 32 + 1)) == hipSuccess &&
         hipMemcpyAsync(d_soff, soff.data(), sizeof(uint64_t) * (n_traces + 1), hipMemcpyHostToDevice, st) ==
             hipSuccess;
    lp.slot_off = d_soff;
    lp.fin = d_fin;
    lp.arr = d_arr;
    for (uint32_t t0 = 0; ok && t0 < n_traces;) {
      uint32_t t1 = t0 + 1;
      while (t1 < n_traces && t1 - t0 < 65535u && soff[t1 + 1] - soff[t0] <= cap) ++t1;
      int64_t len = 0;
      for (uint32_t t = t0; t < t1; ++t) len = std::max<int64_t>(len, ev->h_off[t + 1] - ev->h_off[t]);
      const uint64_t slots = soff[t1] - soff[t0];
      lp.t0 = t0;
      lp.n_traces = t1 - t0;
      lp.slot_base = soff[t0];
      ok = hipMemsetAsync(d_fin, 0xFF, sizeof(uint32_t) * slots, st) == hipSuccess &&
           hipMemsetAsync(d_arr, 0, sizeof(uint32_t) * (slots / 32 + 1), st) == hipSuccess;
      if (ok && len > 0) {
        const dim3 g((unsigned)((len + kValChunk - 1) / kValChunk), t1 - t0);
        hipLaunchKernelGGL(life_scan<1>, g, dim3(256), 0, st, lp);
        hipLaunchKernelGGL(life_scan<2>, g, dim3(256), 0, st, lp);
        ok = hipGetLastError() == hipSuccess;
      }
      t0 = t1;
    }
    ok = ok && readback();
    if (d_max) (void)hipFree(d_max);
    if (d_soff) (void)hipFree(d_soff);
    if (d_fin) (void)hipFree(d_fin);
    if (d_arr) (void)hipFree(d_arr);
    if (ok && h.life != ~0ull)
      rc = fail(TRE_ESTATE, "trace %u: request id %u arrives or finishes twice, or arrives or decodes after its FINISH",
                (unsigned)(h.life >> 32), (unsigned)h.life);
  }
  (void)hipFree(slots);
  if (!ok) return fail(TRE_EHIP, "validation launch failed");
  return rc;
}

extern "C" int tre_load_events(const int64_t* ts, const uint8_t* model, const uint32_t* req,
                               const uint8_t* type, const uint16_t* tokens,
                               const int64_t* trace_off, uint32_t n_traces,
                               const tre_trace_cfg* cfg, uint32_t flags, void* stream,
                               tre_events** out) {
  if (!out) return fail(TRE_EINVAL, "tre_load_events: out is NULL");
  *out = nullptr;
  if (!ts || !model || !type || !tokens || !trace_off || !cfg)
    return fail(TRE_EINVAL, "tre_load_events: NULL column, offsets or cfg");
  if (n_traces == 0) return fail(TRE_EINVAL, "tre_load_events: no traces");
  if (((uintptr_t)ts & 15) || ((uintptr_t)tokens & 15) || ((uintptr_t)model & 7) ||
      ((uintptr_t)type & 7))
    return fail(TRE_EINVAL, "tre_load_events: misaligned column (ts/tokens need 16, model/type 8)");
  const tre_trace_cfg c = *cfg;
  if (c.window_ms < 1 || c.window_ms > (1 << 23))
    return fail(TRE_EINVAL, "window_ms %lld outside [1, 2^23]", (long long)c.window_ms);
  if (c.duration_ms <= 0 || c.duration_ms % c.window_ms)
    return fail(TRE_EINVAL, "duration_ms must be a positive multiple of window_ms");
  if (c.duration_ms >= (1ll << 32)) return fail(TRE_EINVAL, "duration_ms must be below 2^32");
  if (c.duration_ms / c.window_ms > (1ll << 30)) return fail(TRE_EINVAL, "too many windows");
  if (c.fast_period_ms <= 0 || c.slow_period_ms <= 0 || c.fast_period_ms % c.window_ms ||
      c.slow_period_ms % c.window_ms)
    return fail(TRE_EINVAL, "periods must be positive multiples of window_ms");
  if (c.n_models < 1 || c.n_models > TRE_MAX_MODELS)
    return fail(TRE_EINVAL, "n_models %d outside [1, %d]", c.n_models, TRE_MAX_MODELS);
  if (c.budget < 0) return fail(TRE_EINVAL, "negative budget");
  if (trace_off[0] < 0) return fail(TRE_EINVAL, "trace_off[0] < 0");
  for (uint32_t i = 0; i < n_traces; ++i) {
    if (trace_off[i + 1] < trace_off[i]) return fail(TRE_EINVAL, "trace_off decreases at %u", i);
    if (trace_off[i + 1] - trace_off[i] >= (1ll << 27))
      return fail(TRE_ERANGE, "trace %u has 2^27 or more events", i);
  }
  tre_events* ev = new (std::nothrow) tre_events();
  if (!ev) return fail(TRE_EINVAL, "out of host memory");
  ev->ts = ts;
  ev->model = model;
  ev->req = req;
  ev->type = type;
  ev->tokens = tokens;
  ev->n_traces = n_traces;
  ev->cfg = c;
  ev->n_windows = c.duration_ms / c.window_ms;
  ev->h_off.assign(trace_off, trace_off + n_traces + 1);
  ev->n_events = trace_off[n_traces] - trace_off[0];
  ev->n_rows = trace_off[n_traces];
  ev->wcap = ring_windows(c.n_models);
  const int64_t fw = c.fast_period_ms / c.window_ms, sw = c.slow_period_ms / c.window_ms;
  std::vector<uint32_t> tw;
  std::vector<uint8_t> tk;
  for (int64_t w = 0; w < ev->n_windows; ++w) {
    const uint8_t k = (uint8_t)(((w + 1) % fw == 0 ? 1 : 0) | ((w + 1) % sw == 0 ? 2 : 0));
    if (k) {
      tw.push_back((uint32_t)w);
      tk.push_back(k);
    }
  }
  ev->n_ticks = (int64_t)tw.size();
  hipStream_t st = (hipStream_t)stream;
  int rc = TRE_OK;
  auto cleanup = [&](int code) {
    tre_free_events(ev);
    return code;
  };
  if (hipGetDevice(&ev->device) != hipSuccess) return cleanup(fail(TRE_EHIP, "hipGetDevice failed"));
  if (hipMalloc(&ev->d_off, sizeof(int64_t) * (n_traces + 1)) != hipSuccess ||
      hipMalloc(&ev->d_tick_window, sizeof(uint32_t) * (tw.size() + 1)) != hipSuccess ||
      hipMalloc(&ev->d_tick_kind, tw.size() + 1) != hipSuccess)
    return cleanup(fail(TRE_EHIP, "hipMalloc of handle tables failed"));
  if (hipMemcpyAsync(ev->d_off, trace_off, sizeof(int64_t) * (n_traces + 1), hipMemcpyHostToDevice,
                     st) != hipSuccess ||
      (!tw.empty() && hipMemcpyAsync(ev->d_tick_window, tw.data(), sizeof(uint32_t) * tw.size(),
                                     hipMemcpyHostToDevice, st) != hipSuccess) ||
      (!tk.empty() &&
       hipMemcpyAsync(ev->d_tick_kind, tk.data(), tk.size(), hipMemcpyHostToDevice, st) != hipSuccess) ||
      hipStreamSynchronize(st) != hipSuccess)
    return cleanup(fail(TRE_EHIP, "copy of handle tables failed"));

  if (flags & TRE_VALIDATE) {
    rc = validate_events(ev, st);
    if (rc != TRE_OK) return cleanup(rc);
  }
  *out = ev;
  return TRE_OK;
}

extern "C" void tre_free_events(tre_events* ev) {
  if (!ev) return;
  if (ev->d_off) (void)hipFree(ev->d_off);
  if (ev->d_tick_window) (void)hipFree(ev->d_tick_window);
  if (ev->d_tick_kind) (void)hipFree(ev->d_tick_kind);
  delete ev;
}

extern "C" int tre_events_info(const tre_events* ev, tre_info* info) {
  if (!ev || !info) return fail(TRE_EINVAL, "tre_events_info: NULL argument");
  info->n_traces = ev->n_traces;
  info->n_models = (uint32_t)ev->cfg.n_models;
  info->n_events = ev->n_events;
  info->n_windows = ev->n_windows;
  info->n_ticks = ev->n_ticks;
  return TRE_OK;
}

// tre_sweep's workspace: the per-tick smoothed TSS of every trace (read by
// the separate replay of traces with several scenarios), then per trace
// its scenario count and one of its scenarios
static size_t snapshot_bytes(const tre_events* ev) {
  return ((size_t)ev->n_traces * (size_t)ev->n_ticks * (size_t)ev->cfg.n_models * sizeof(double) + 255) &
         ~(size_t)255;
}

extern "C" int tre_workspace_size(const tre_events* ev, uint32_t n_scenarios, size_t* bytes) {
  if (!ev || !bytes) return fail(TRE_EINVAL, "tre_workspace_size: NULL argument");
  (void)n_scenarios;
  *bytes = snapshot_bytes(ev) + 2 * sizeof(uint32_t) * (size_t)ev->n_traces;
  return TRE_OK;
}

extern "C" int tre_check_params(const tre_events* ev, const tre_profile* prof,
                                const tre_scenario* sc, uint32_t n_scenarios) {
  if (!ev || !prof) return fail(TRE_EINVAL, "tre_check_params: NULL handle or profiles");
  if (n_scenarios && !sc) return fail(TRE_EINVAL, "tre_check_params: NULL scenarios");
  int rc = check_device(ev);
  if (rc) return rc;
  const size_t M = (size_t)ev->cfg.n_models;
  std::vector<tre_profile> hp((size_t)ev->n_traces * M);
  std::vector<tre_scenario> hs(n_scenarios);
  HIP_TRY(hipMemcpy(hp.data(), prof, hp.size() * sizeof(tre_profile), hipMemcpyDeviceToHost));
  if (n_scenarios)
    HIP_TRY(hipMemcpy(hs.data(), sc, hs.size() * sizeof(tre_scenario), hipMemcpyDeviceToHost));
  for (uint32_t t = 0; t < ev->n_traces; ++t) {
    long long rsum = 0;
    for (size_t m = 0; m < M; ++m) {
      const tre_profile& q = hp[t * M + m];
      if (!(q.w_p >= 0.0 && q.w_q >= 0.0 && q.alpha > 0.0 && q.alpha <= 1.0 && q.theta > 0.0 &&
            isfinite(q.w_p) && isfinite(q.w_q) && isfinite(q.theta) && q.tau_crit >= 0.0 &&
            q.tau_crit < q.tau_surplus && q.r_min >= 0 && q.r_init >= 0))
        return fail(TRE_EINVAL, "profile of trace %u model %zu out of range", t, m);
      rsum += q.r_init;
    }
    if (rsum > ev->cfg.budget)
      return fail(TRE_EINVAL, "trace %u: initial replicas %lld exceed the budget %d", t, rsum,
                  ev->cfg.budget);
  }
  for (uint32_t s = 0; s < n_scenarios; ++s) {
    const tre_scenario& q = hs[s];
    if (q.trace >= ev->n_traces) return fail(TRE_EINVAL, "scenario %u: trace out of range", s);
    if (!(q.theta_scale > 0.0 && isfinite(q.theta_scale)))
      return fail(TRE_EINVAL, "scenario %u: theta_scale must be positive", s);
    if (q.tau_crit_override >= 0.0) {
      for (size_t m = 0; m < M; ++m)
        if (!(q.tau_crit_override < hp[q.trace * M + m].tau_surplus))
          return fail(TRE_EINVAL, "scenario %u: tau_crit_override >= tau_surplus", s);
    }
  }
  return TRE_OK;
}

static StreamParams stream_params(const tre_events* ev, const tre_profile* prof) {
  StreamParams p{};
  p.ts = ev->ts;
  p.model = ev->model;
  p.type = ev->type;
  p.tokens = ev->tokens;
  p.off = ev->d_off;
  p.n_rows = ev->n_rows;
  p.prof = prof;
  p.window_ms = ev->cfg.window_ms;
  p.magic = ev->cfg.window_ms == 1 ? 0xFFFFFFFFu
                                   : (uint32_t)((1ull << 32) / (uint64_t)ev->cfg.window_ms);
  p.inv2_window = 0.5 / (double)ev->cfg.window_ms;
  p.n_windows = (int32_t)ev->n_windows;
  p.M = ev->cfg.n_models;
  p.wcap = ev->wcap;
  p.chunk = chunk_windows(ev->cfg.n_models, ev->wcap);
  p.fast_w = (int32_t)(ev->cfg.fast_period_ms / ev->cfg.window_ms);
  p.slow_w = (int32_t)(ev->cfg.slow_period_ms / ev->cfg.window_ms);
  p.magic_fast = p.fast_w == 1 ? 0xFFFFFFFFu : (uint32_t)((1ull << 32) / (uint64_t)p.fast_w);
  p.magic_slow = p.slow_w == 1 ? 0xFFFFFFFFu : (uint32_t)((1ull << 32) / (uint64_t)p.slow_w);
  p.n_ticks = (int32_t)ev->n_ticks;
  return p;
}

// Scenarios per trace of a sweep: count[t] and, for a trace with exactly
// one, that scenario in first[t] (count is zeroed first)
__global__ __launch_bounds__(256) void zero_u32(uint32_t* q, uint32_t n) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) q[i] = 0u;
}

__global__ __launch_bounds__(256) void sweep_map(const tre_scenario* sc, uint32_t n_sc, uint32_t n_traces,
                                                 uint32_t* count, uint32_t* first) {
  const uint32_t s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_sc) return;
  const uint32_t t = sc[s].trace;
  if (t >= n_traces) return;
  if (atomicAdd(&count[t], 1u) == 0u) first[t] = s;
}

static int launch_stream(const tre_events* ev, const StreamParams& p, hipStream_t st) {
  const bool stage = p.stage64 || p.stage32 || p.sflags;
  const size_t lds = stream_lds(ev, stage);
  LaunchTimer lt("tss_stream", st);
  const bool cells = p.prefill || p.decode || p.a_int || p.w_int || p.tss64 || p.tss32 || p.flags;
  const int waves = stream_waves(ev->n_traces);
  if (stage)
    hipLaunchKernelGGL((tss_stream_stage<kStreamWaves, kStreamEPT>), dim3(ev->n_traces),
                       dim3(kStreamWaves * 64), lds, st, p);
  else if (waves == 16 && cells)
    hipLaunchKernelGGL((tss_stream<16, kStreamEPT, true>), dim3(ev->n_traces), dim3(16 * 64), lds, st, p);
  else if (waves == 16)
    hipLaunchKernelGGL((tss_stream<16, kStreamEPT, false>), dim3(ev->n_traces), dim3(16 * 64), lds, st, p);
  else if (waves == 8 && cells)
    hipLaunchKernelGGL((tss_stream<8, kStreamEPT, true>), dim3(ev->n_traces), dim3(8 * 64), lds, st, p);
  else if (waves == 8)
    hipLaunchKernelGGL((tss_stream<8, kStreamEPT, false>), dim3(ev->n_traces), dim3(8 * 64), lds, st, p);
  else if (cells)
    hipLaunchKernelGGL((tss_stream<kStreamWaves, kStreamEPT, true>), dim3(ev->n_traces),
                       dim3(kStreamWaves * 64), lds, st, p);
  else
    hipLaunchKernelGGL((tss_stream<kStreamWaves, kStreamEPT, false>), dim3(ev->n_traces),
                       dim3(kStreamWaves * 64), lds, st, p);
  const hipError_t e = hipGetLastError();
  lt.done();
  if (e != hipSuccess) return fail(TRE_EHIP, "tss_stream launch: %s", hipGetErrorString(e));
  return TRE_OK;
}

// the actuation model in whole windows (delays rounded up)
struct ActWindows {
  int32_t wake_w, sleep_w;
  const int32_t* footprint;
  const uint64_t* veto;
};

static int act_windows(const tre_events* ev, const tre_actuation* act, ActWindows* aw) {
  if (!act) return fail(TRE_EINVAL, "NULL actuation model");
  if (act->wake_ms < 0 || act->sleep_ms < 0)
    return fail(TRE_EINVAL, "actuation delays must be >= 0");
  const int64_t win = ev->cfg.window_ms;
  // whole windows, rounded up; a transition completing after the last window
  // never counts, so the delays are capped just past the trace
  const int64_t cap = ev->n_windows + 1;
  auto to_windows = [&](int64_t ms) { return ms > cap * win ? cap : (ms + win - 1) / win; };
  aw->wake_w = (int32_t)to_windows(act->wake_ms);
  aw->sleep_w = (int32_t)to_windows(act->sleep_ms);
  aw->footprint = act->footprint;
  aw->veto = act->veto;
  return TRE_OK;
}

static int launch_rebalance(const tre_events* ev, const tre_profile* prof, const double* vals,
                            const uint8_t* flags, const tre_scenario* sc, uint32_t n_sc,
                            const tre_ctl_out* out, const ActWindows* aw, hipStream_t st,
                            const uint32_t* sc_count = nullptr) {
  CtlParams c{};
  c.sc_count = sc_count;
  c.prof = prof;
  c.sc = sc;
  c.n_sc = n_sc;
  c.vals = vals;
  c.flags = flags;
  c.tick_window = ev->d_tick_window;
  c.tick_kind = ev->d_tick_kind;
  c.n_ticks = (int32_t)ev->n_ticks;
  c.n_windows = (int32_t)ev->n_windows;
  c.M = ev->cfg.n_models;
  c.budget = ev->cfg.budget;
  c.n_traces = ev->n_traces;
  c.moves = out->moves;
  c.move_cap = out->move_cap;
  c.n_moves = out->n_moves;
  c.r_final = out->r_final;
  c.r_windows = out->r_windows;
  if (aw) {
    c.wake_w = aw->wake_w;
    c.sleep_w = aw->sleep_w;
    c.footprint = aw->footprint;
    c.veto = aw->veto;
  }
  // one wave per scenario, four per workgroup
  const dim3 grid((unsigned)(((uint64_t)n_sc + 3) / 4)), block(256);
  LaunchTimer lt("rebalance", st);
  if (aw)
    hipLaunchKernelGGL(rebalance<true>, grid, block, 0, st, c);
  else
    hipLaunchKernelGGL(rebalance<false>, grid, block, 0, st, c);
  const hipError_t e = hipGetLastError();
  lt.done();
  if (e != hipSuccess) return fail(TRE_EHIP, "rebalance launch: %s", hipGetErrorString(e));
  return TRE_OK;
}

static int check_ctl_out(const tre_ctl_out* out, uint32_t n_sc) {
  if (!out) return fail(TRE_EINVAL, "NULL control outputs");
  if (n_sc && (!out->n_moves || !out->r_final || !out->r_windows || (out->move_cap && !out->moves)))
    return fail(TRE_EINVAL, "NULL control output array");
  return TRE_OK;
}

extern "C" int tre_eval_tss(const tre_events* ev, const tre_profile* prof, const tre_tss_out* out,
                            void* stream) {
  if (!ev || !prof || !out) return fail(TRE_EINVAL, "tre_eval_tss: NULL argument");
  int rc = check_device(ev);
  if (rc) return rc;
  StreamParams p = stream_params(ev, prof);
  p.prefill = out->prefill;
  p.decode = out->decode;
  p.a_int = out->a_int;
  p.w_int = out->w_int;
  p.tss64 = out->tss64;
  p.tss32 = out->tss32;
  p.flags = out->flags;
  return launch_stream(ev, p, (hipStream_t)stream);
}

extern "C" int tre_eval_stage(const tre_events* ev, const tre_profile* prof, double* stage64, float* stage32,
                              uint8_t* flags, void* stream) {
  if (!ev || !prof) return fail(TRE_EINVAL, "tre_eval_stage: NULL handle or profiles");
  if (!stage64 && !stage32 && !flags) return fail(TRE_EINVAL, "tre_eval_stage: no output");
  if (((uintptr_t)stage64 & 15) || ((uintptr_t)stage32 & 7))
    return fail(TRE_EINVAL, "tre_eval_stage: stage64 needs 16-byte, stage32 8-byte alignment");
  int rc = check_device(ev);
  if (rc) return rc;
  StreamParams p = stream_params(ev, prof);
  p.stage64 = stage64;
  p.stage32 = stage32;
  p.sflags = flags;
  return launch_stream(ev, p, (hipStream_t)stream);
}

static int rebalance_impl(const tre_events* ev, const tre_profile* prof, const double* tss64,
                          const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                          const tre_actuation* act, const tre_ctl_out* out, void* stream,
                          const char* who) {
  if (!ev || !prof || !tss64 || !flags) return fail(TRE_EINVAL, "%s: NULL argument", who);
  if (n_scenarios && !sc) return fail(TRE_EINVAL, "%s: NULL scenarios", who);
  int rc = check_ctl_out(out, n_scenarios);
  if (rc) return rc;
  rc = check_device(ev);
  if (rc) return rc;
  ActWindows aw;
  if (act && (rc = act_windows(ev, act, &aw))) return rc;
  if (n_scenarios == 0) return TRE_OK;
  return launch_rebalance(ev, prof, tss64, flags, sc, n_scenarios, out, act ? &aw : nullptr,
                          (hipStream_t)stream);
}

static int sweep_impl(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                      uint32_t n_scenarios, const tre_actuation* act, const tre_ctl_out* out,
                      float* tss32, void* ws, size_t ws_bytes, void* stream, const char* who) {
  if (!ev || !prof) return fail(TRE_EINVAL, "%s: NULL argument", who);
  if (n_scenarios && !sc) return fail(TRE_EINVAL, "%s: NULL scenarios", who);
  int rc = check_ctl_out(out, n_scenarios);
  if (rc) return rc;
  rc = check_device(ev);
  if (rc) return rc;
  ActWindows aw;
  if (act && (rc = act_windows(ev, act, &aw))) return rc;
  size_t need = 0;
  tre_workspace_size(ev, n_scenarios, &need);
  if (!ws || ws_bytes < need)
    return fail(TRE_ENOMEM, "workspace of %zu bytes is smaller than the %zu needed", ws_bytes, need);
  if ((uintptr_t)ws & 7) return fail(TRE_EINVAL, "workspace must be 8-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  StreamParams p = stream_params(ev, prof);
  p.tss32 = tss32;
  p.snap = (double*)ws;
  // without the actuation model, a trace with exactly one scenario replays
  // it in the stream (rebalance skips it)
  uint32_t* count = nullptr;
  if (n_scenarios && !act) {
    count = (uint32_t*)((char*)ws + snapshot_bytes(ev));
    uint32_t* first = count + ev->n_traces;
    hipLaunchKernelGGL(zero_u32, dim3((ev->n_traces + 255) / 256), dim3(256), 0, st, count, ev->n_traces);
    hipLaunchKernelGGL(sweep_map, dim3((n_scenarios + 255) / 256), dim3(256), 0, st, sc, n_scenarios,
                       ev->n_traces, count, (uint32_t*)first);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(TRE_EHIP, "sweep_map launch: %s", hipGetErrorString(e));
    p.sc = sc;
    p.sc_count = count;
    p.sc_first = first;
    p.budget = ev->cfg.budget;
    p.moves = out->moves;
    p.move_cap = out->move_cap;
    p.n_moves = out->n_moves;
    p.r_final = out->r_final;
    p.r_windows = out->r_windows;
  }
  rc = launch_stream(ev, p, st);
  if (rc || n_scenarios == 0) return rc;
  return launch_rebalance(ev, prof, (const double*)ws, nullptr, sc, n_scenarios, out,
                          act ? &aw : nullptr, st, count);
}

extern "C" int tre_rebalance(const tre_events* ev, const tre_profile* prof, const double* tss64,
                             const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                             const tre_ctl_out* out, void* stream) {
  return rebalance_impl(ev, prof, tss64, flags, sc, n_scenarios, nullptr, out, stream, "tre_rebalance");
}

extern "C" int tre_sweep(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                         uint32_t n_scenarios, const tre_ctl_out* out, float* tss32, void* ws,
                         size_t ws_bytes, void* stream) {
  return sweep_impl(ev, prof, sc, n_scenarios, nullptr, out, tss32, ws, ws_bytes, stream, "tre_sweep");
}

// ------------------------------------------------ sweep without allocation
// The sweep's scratch (the per-tick smoothed TSS snapshot) in a static
// device array for callers that cannot allocate. Each GPU the library runs
// on holds its own copy until the process ends; its device address is
// looked up once per device, with that device current, at the entry
// point's first call there, and only that address is used afterwards.
static __device__ __align__(256) unsigned char scratch[TRE_NOALLOC_SCRATCH_BYTES];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[256];  // per device ordinal, NULL until looked up
}  // namespace

static int scratch_for(int dev, void** out) {
  if (dev < 0 || dev >= 256) return fail(TRE_EINVAL, "device ordinal %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(TRE_EHIP, "hipGetSymbolAddress of the static scratch: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return TRE_OK;
}

extern "C" int tre_sweep_noalloc(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                                 uint32_t n_scenarios, const tre_ctl_out* out, float* tss32, void* stream) {
  if (!ev) return fail(TRE_EINVAL, "tre_sweep_noalloc: NULL handle");
  int rc = check_device(ev);  // the handle's device is the current one
  if (rc) return rc;
  size_t need = 0;
  tre_workspace_size(ev, n_scenarios, &need);
  if (need > (size_t)TRE_NOALLOC_SCRATCH_BYTES)
    return fail(TRE_ENOMEM, "tre_sweep_noalloc: the sweep needs %zu bytes of scratch, above the static %zu",
                need, (size_t)TRE_NOALLOC_SCRATCH_BYTES);
  void* ws = nullptr;
  if ((rc = scratch_for(ev->device, &ws))) return rc;
  tre_internal::NoTimingScope quiet;  // no event objects are created for this call
  return sweep_impl(ev, prof, sc, n_scenarios, nullptr, out, tss32, ws, (size_t)TRE_NOALLOC_SCRATCH_BYTES, stream,
                    "tre_sweep_noalloc");
}

extern "C" int tre_rebalance_act(const tre_events* ev, const tre_profile* prof, const double* tss64,
                                 const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                                 const tre_actuation* act, const tre_ctl_out* out, void* stream) {
  if (!act) return fail(TRE_EINVAL, "tre_rebalance_act: NULL actuation model");
  return rebalance_impl(ev, prof, tss64, flags, sc, n_scenarios, act, out, stream, "tre_rebalance_act");
}

extern "C" int tre_sweep_act(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                             uint32_t n_scenarios, const tre_actuation* act, const tre_ctl_out* out,
                             float* tss32, void* ws, size_t ws_bytes, void* stream) {
  if (!act) return fail(TRE_EINVAL, "tre_sweep_act: NULL actuation model");
  return sweep_impl(ev, prof, sc, n_scenarios, act, out, tss32, ws, ws_bytes, stream, "tre_sweep_act");
}

extern "C" int tre_check_actuation(const tre_events* ev, const tre_profile* prof,
                                   const tre_actuation* act) {
  if (!ev || !prof || !act) return fail(TRE_EINVAL, "tre_check_actuation: NULL argument");
  int rc = check_device(ev);
  if (rc) return rc;
  ActWindows aw;
  if ((rc = act_windows(ev, act, &aw))) return rc;
  const size_t M = (size_t)ev->cfg.n_models;
  std::vector<tre_profile> hp((size_t)ev->n_traces * M);
  HIP_TRY(hipMemcpy(hp.data(), prof, hp.size() * sizeof(tre_profile), hipMemcpyDeviceToHost));
  std::vector<int32_t> g(hp.size(), 1);
  if (act->footprint)
    HIP_TRY(hipMemcpy(g.data(), act->footprint, g.size() * sizeof(int32_t), hipMemcpyDeviceToHost));
  for (uint32_t t = 0; t < ev->n_traces; ++t) {
    long long gsum = 0;
    for (size_t m = 0; m < M; ++m) {
      const int32_t gm = g[t * M + m];
      if (gm < 1 || gm > ev->cfg.budget)
        return fail(TRE_EINVAL, "trace %u model %zu: footprint %d outside 1 .. budget", t, m, gm);
      gsum += (long long)gm * hp[t * M + m].r_init;
    }
    if (gsum > ev->cfg.budget)
      return fail(TRE_EINVAL, "trace %u: initial replicas hold %lld GPUs, above the budget %d", t,
                  gsum, ev->cfg.budget);
  }
  return TRE_OK;
}
