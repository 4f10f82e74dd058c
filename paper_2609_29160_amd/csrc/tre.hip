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
//   tss_stream  one workgroup per trace. Producer waves stream the SoA event
//               columns (nontemporal 16/8-byte vector loads, 8 events per
//               lane) and tally each event into an LDS ring of per-(window,
//               model) cells with 64-bit LDS atomics (three packed words per
//               cell). One consumer wave, lanes = models, walks the completed
//               windows in order: carry scan of the active / waiting counts,
//               in-window integrals, Eq. (1) in fp64, smoothing, outputs.
//   rebalance   one lane group of G = next_pow2(n_models) lanes per scenario
//               (64/G scenarios per wave64): Eq. (2), regions, cadence, and
//               the greedy receiver/donor moves with wave ballots and
//               shuffles for argmin / argmax (lowest index on ties).
//   validate    checks the event columns once, at load time.
#include <hip/hip_runtime.h>

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

#pragma clang fp contract(off)

// ------------------------------------------------------------------ errors
static thread_local std::string g_err;

static int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(TRE_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

extern "C" const char* tre_last_error(void) { return g_err.c_str(); }

// ------------------------------------------------------------------ handle
struct tre_events {
  const int64_t* ts;
  const uint8_t* model;
  const uint32_t* req;
  const uint8_t* type;
  const uint16_t* tokens;
  uint32_t n_traces;
  tre_trace_cfg cfg;
  int64_t n_windows;
  int64_t n_ticks;
  int64_t n_events;
  int64_t n_rows;  // rows [0, n_rows) of every column are readable
  int64_t* d_off;
  uint32_t* d_tick_window;
  uint8_t* d_tick_kind;
  std::vector<int64_t> h_off;
  uint32_t wcap;
  int device;
};

// ------------------------------------------------------------ constants
constexpr int kBlock = 512;                // tss_stream workgroup
constexpr int kEPT = 8;                    // events per producer lane per tile
constexpr int kProducers = kBlock - 64;    // wave 0 is the consumer
constexpr int kTile = kProducers * kEPT;   // events per tile
constexpr int kRingBytes = 48 * 1024;      // LDS budget of the tally ring
constexpr uint64_t kOne40 = 1ull << 40;    // packed (count << 40) + integral
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
  int32_t fast_w;   // fast period in windows
  int32_t slow_w;   // slow period in windows
  int32_t n_ticks;
  uint32_t* prefill;
  uint32_t* decode;
  int64_t* a_int;
  int64_t* w_int;
  double* tss64;
  float* tss32;
  uint8_t* flags;
  double* snap;     // [trace][tick][M]: S, or +inf when idle / not initialised
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

// sign-extended low 40 bits and the count above them
__device__ __forceinline__ void unpack40(unsigned long long v, long long& count, long long& integ) {
  long long s = (long long)v;
  integ = (long long)(v << 24) >> 24;
  count = (s - integ) >> 40;
}

__global__ __launch_bounds__(kBlock) void tss_stream(StreamParams p) {
  extern __shared__ unsigned long long ring[];
  __shared__ long long s_e;
  __shared__ int s_wdone;
  __shared__ int s_wnext;
  __shared__ unsigned s_defer;

  const int trace = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const bool consumer = tid < 64;
  const int M = p.M;
  const uint32_t wcap = p.wcap;
  const int ncell = (int)wcap * M;
  unsigned long long* r_pd = ring;              // P (low 32) | D (high 32)
  unsigned long long* r_a = ring + ncell;       // (dA << 40) + dA*(t_end - ts)
  unsigned long long* r_w = ring + 2 * ncell;   // (dW << 40) + dW*(t_end - ts)
  const int64_t e_begin = p.off[trace];
  const int64_t e_end = p.off[trace + 1];
  const int64_t win = p.window_ms;
  const uint32_t win32 = (uint32_t)win;
  const int nW = p.n_windows;

  for (int i = tid; i < 3 * ncell; i += kBlock) ring[i] = 0ull;
  if (tid == 0) {
    s_e = e_begin;
    s_wdone = 0;
    s_defer = kNoDefer;
  }

  // consumer state: lane m owns model m
  const bool own = consumer && lane < M;
  long long a_start = 0, w_start = 0;
  double S = 0.0;
  bool init = false;
  double w_p = 0.0, w_q = 0.0, alpha = 0.0, oma = 0.0;
  if (own) {
    const tre_profile pr = p.prof[(int64_t)trace * M + lane];
    w_p = pr.w_p;
    w_q = pr.w_q;
    alpha = pr.alpha;
    oma = 1.0 - alpha;
  }
  int fctr = 0, sctr = 0, tick = 0;
  const double dwin = (double)win;
  const bool cells = p.prefill || p.decode || p.a_int || p.w_int || p.tss64 || p.tss32 || p.flags;

  __syncthreads();
  for (;;) {
    const long long e0 = s_e;
    const int wd = s_wdone;
    if (wd >= nW) break;
    if (consumer) {
      // windows before the first unprocessed event are complete
      long long wl64 = nW;
      if (e0 < e_end) wl64 = p.ts[e0] / win;
      // never backwards, never past the last window (only matters for
      // unvalidated, unsorted input)
      const int wl = (int)(wl64 < wd ? wd : (wl64 > nW ? nW : wl64));
      for (int w = wd; w < wl; ++w) {
        unsigned long long pd = 0, ap = 0, wp = 0;
        if (own && w < wd + (int)wcap) {
          const int c = (int)((uint32_t)w & (wcap - 1)) * M + lane;
          pd = r_pd[c];
          ap = r_a[c];
          wp = r_w[c];
          r_pd[c] = 0ull;
          r_a[c] = 0ull;
          r_w[c] = 0ull;
        }
        long long na, la, nw, lw;
        unpack40(ap, na, la);
        unpack40(wp, nw, lw);
        const long long A_int = a_start * win + la;
        const long long W_int = w_start * win + lw;
        a_start += na;
        w_start += nw;
        const uint32_t P = (uint32_t)pd;
        const uint32_t Dt = (uint32_t)(pd >> 32);
        const bool idle = pd == 0ull && A_int == 0 && W_int == 0;
        if (!idle) {
          // Eq. (1), evaluated in the documented order
          double num = w_p * (double)P;
          num = num + (double)Dt;
          num = num * 1000.0;
          const double q = w_q * (double)W_int;
          double den = (double)A_int + q;
          if (den < dwin) den = dwin;
          const double raw = num / den;
          if (init) {
            const double t1 = alpha * raw;
            const double t2 = oma * S;
            S = t1 + t2;
          } else {
            S = raw;
            init = true;
          }
        }
        if (own && cells) {
          const int64_t c = ((int64_t)trace * nW + w) * M + lane;
          if (p.prefill) p.prefill[c] = P;
          if (p.decode) p.decode[c] = Dt;
          if (p.a_int) p.a_int[c] = A_int;
          if (p.w_int) p.w_int[c] = W_int;
          if (p.tss64) p.tss64[c] = S;
          if (p.tss32) p.tss32[c] = (float)S;
          if (p.flags) p.flags[c] = (uint8_t)((idle ? TRE_FLAG_IDLE : 0) | (init ? TRE_FLAG_INIT : 0));
        }
        ++fctr;
        ++sctr;
        const bool fast = fctr == p.fast_w;
        const bool slow = sctr == p.slow_w;
        if (fast) fctr = 0;
        if (slow) sctr = 0;
        if (fast || slow) {
          if (own && p.snap && tick < p.n_ticks)
            p.snap[((int64_t)trace * p.n_ticks + tick) * M + lane] = (idle || !init) ? INFINITY : S;
          ++tick;
        }
      }
      if (lane == 0) s_wnext = wl;
    } else {
      // producers: events [max(e0, a0), min(a0 + tile, e_end)) whose window
      // fits the ring; the first that does not is where the next tile starts
      const int pt = tid - 64;
      const long long a0 = e0 & ~(long long)(kEPT - 1);
      const long long c0 = a0 + (long long)pt * kEPT;
      if (c0 + kEPT > e0 && c0 < e_end) {
        long long tsv[kEPT];
        uint32_t mw[2], tw[2], kw[4];
        if (c0 + kEPT <= p.n_rows) {
          const v2i64* tp = (const v2i64*)(p.ts + c0);
#pragma unroll
          for (int j = 0; j < kEPT / 2; ++j) {
            v2i64 v = __builtin_nontemporal_load(tp + j);
            tsv[2 * j] = v.x;
            tsv[2 * j + 1] = v.y;
          }
          v2u32 mv = __builtin_nontemporal_load((const v2u32*)(p.model + c0));
          v2u32 tv = __builtin_nontemporal_load((const v2u32*)(p.type + c0));
          v4u32 kv = __builtin_nontemporal_load((const v4u32*)(p.tokens + c0));
          mw[0] = mv.x; mw[1] = mv.y;
          tw[0] = tv.x; tw[1] = tv.y;
          kw[0] = kv.x; kw[1] = kv.y; kw[2] = kv.z; kw[3] = kv.w;
        } else {
          // ragged end of the columns: element loads inside [0, n_rows)
          mw[0] = mw[1] = tw[0] = tw[1] = 0;
          kw[0] = kw[1] = kw[2] = kw[3] = 0;
#pragma unroll
          for (int j = 0; j < kEPT; ++j) {
            const long long i = c0 + j;
            tsv[j] = 0;
            if (i < p.n_rows) {
              tsv[j] = p.ts[i];
              mw[j >> 2] |= (uint32_t)p.model[i] << (8 * (j & 3));
              tw[j >> 2] |= (uint32_t)p.type[i] << (8 * (j & 3));
              kw[j >> 1] |= (uint32_t)p.tokens[i] << (16 * (j & 1));
            }
          }
        }
        const long long base_ms = (long long)wd * win;
        const long long cap_ms = (long long)wcap * win;
#pragma unroll
        for (int j = 0; j < kEPT; ++j) {
          const long long i = c0 + j;
          if (i < e0 || i >= e_end) continue;
          const int mdl = (mw[j >> 2] >> (8 * (j & 3))) & 0xFF;
          const uint32_t ty = (tw[j >> 2] >> (8 * (j & 3))) & 0xFF;
          const uint32_t tok = (kw[j >> 1] >> (16 * (j & 1))) & 0xFFFF;
          const long long d = tsv[j] - base_ms;
          if (d >= cap_ms) {
            atomicMin(&s_defer, (unsigned)(i - a0));
            break;  // later events of this lane are not earlier
          }
          if (d < 0 || mdl >= M) continue;  // only reachable with unvalidated input
          uint32_t q, r;
          div_window((uint32_t)d, p.magic, win32, q, r);
          const int c = (int)(((uint32_t)wd + q) & (wcap - 1)) * M + mdl;
          const unsigned long long one = kOne40 + (unsigned long long)(win32 - r);
          switch (ty & 3u) {
            case TRE_ARRIVE:
              atomicAdd(&r_w[c], one);
              break;
            case TRE_PREFILL:
              atomicAdd(&r_pd[c], (unsigned long long)tok);
              if (ty & TRE_ADMIT) {
                atomicAdd(&r_w[c], 0ull - one);
                atomicAdd(&r_a[c], one);
              }
              break;
            case TRE_DECODE:
              atomicAdd(&r_pd[c], (unsigned long long)tok << 32);
              break;
            default:
              atomicAdd(&r_a[c], 0ull - one);
              break;
          }
        }
      }
    }
    __syncthreads();
    if (tid == 0) {
      const long long a0 = e0 & ~(long long)(kEPT - 1);
      long long en = a0 + kTile;
      if (en > e_end) en = e_end;
      if (en < e0) en = e0;
      const unsigned dfr = s_defer;
      if (dfr != kNoDefer) en = a0 + dfr;
      s_e = en;
      s_wdone = s_wnext;
      s_defer = kNoDefer;
    }
    __syncthreads();
  }
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
  int32_t g_log2;
  int32_t budget;
  uint32_t n_traces;
  tre_move* moves;
  uint32_t move_cap;
  uint32_t* n_moves;
  int32_t* r_final;
  int64_t* r_windows;
};

__device__ __forceinline__ unsigned long long dbits(double x) {
  return (unsigned long long)__double_as_longlong(x);
}

// lowest lane of the group holding the minimum (or maximum) Z among
// candidates; Z >= 0 so its bit pattern orders like its value; -1 if none
template <bool kMax>
__device__ __forceinline__ int group_arg(bool cand, double Z, int G, int gbase,
                                         unsigned long long gmask) {
  const unsigned long long any = __ballot(cand) & gmask;
  if (any == 0ull) return -1;
  unsigned long long key = cand ? dbits(Z) : (kMax ? 0ull : ~0ull);
  for (int off = G >> 1; off > 0; off >>= 1) {
    const unsigned long long o = __shfl_xor(key, off, G);
    key = kMax ? (o > key ? o : key) : (o < key ? o : key);
  }
  const unsigned long long win = __ballot(cand && dbits(Z) == key) & gmask;
  return __ffsll((long long)win) - 1 - gbase;
}

__global__ __launch_bounds__(256) void rebalance(CtlParams p) {
  const int lane = threadIdx.x & 63;
  const int G = 1 << p.g_log2;
  const uint32_t wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const uint32_t s = wave * (uint32_t)(64 >> p.g_log2) + (uint32_t)(lane >> p.g_log2);
  const int m = lane & (G - 1);
  const int gbase = lane & ~(G - 1);
  const unsigned long long gmask = G == 64 ? ~0ull : (((1ull << G) - 1ull) << gbase);
  const bool sc_ok = s < p.n_sc;
  const int M = p.M;

  uint32_t trace = 0, K = 0;
  double theta_scale = 1.0, ovr = -1.0;
  if (sc_ok) {
    const tre_scenario sc = p.sc[s];
    trace = sc.trace < p.n_traces ? sc.trace : 0;
    K = sc.max_moves;
    theta_scale = sc.theta_scale;
    ovr = sc.tau_crit_override;
  }
  const bool act = sc_ok && m < M;
  double theta_eff = 1.0, tau_c = 0.0, tau_s = INFINITY;
  int R = 0, r_min = 0;
  if (act) {
    const tre_profile pr = p.prof[(int64_t)trace * M + m];
    theta_eff = pr.theta * theta_scale;
    tau_c = ovr >= 0.0 ? ovr : pr.tau_crit;
    tau_s = pr.tau_surplus;
    R = pr.r_init;
    r_min = pr.r_min;
  }
  int rsum = R;
  for (int off = G >> 1; off > 0; off >>= 1) rsum += __shfl_xor(rsum, off, G);
  int pool = p.budget - rsum;
  long long rw = 0;
  int wprev = -1;
  uint32_t nm = 0;

  for (int t = 0; t < p.n_ticks; ++t) {
    const int w = (int)p.tick_window[t];
    const uint32_t kind = p.tick_kind[t];
    double Z = INFINITY;
    if (act) {
      double v;
      if (p.flags) {
        const int64_t c = ((int64_t)trace * p.n_windows + w) * M + m;
        const uint8_t f = p.flags[c];
        v = ((f & TRE_FLAG_IDLE) || !(f & TRE_FLAG_INIT)) ? INFINITY : p.vals[c];
      } else {
        v = p.vals[((int64_t)trace * p.n_ticks + t) * M + m];
      }
      Z = v / theta_eff;  // Eq. (2)
    }
    rw += (long long)R * (w - wprev);
    wprev = w;
    const bool crit = act && Z < tau_c;
    const bool sur = act && Z > tau_s;
    const bool any_crit = (__ballot(crit) & gmask) != 0ull;
    int path;
    bool ok;
    if (any_crit) {
      if (!(kind & 1u)) continue;  // rescue pending: rebalancing defers
      path = TRE_PATH_RESCUE;
      ok = crit;
    } else if (kind & 2u) {
      path = TRE_PATH_REBALANCE;
      ok = act && Z < 1.0;
    } else {
      continue;
    }
    bool used = false;
    for (uint32_t k = 0; k < K; ++k) {
      const int r = group_arg<false>(ok && !used, Z, G, gbase, gmask);  // Eq. (3)
      if (r < 0) break;
      const double Zr = __shfl(Z, r, G);
      int d;
      if (pool > 0) {
        pool -= 1;
        d = TRE_DONOR_POOL;
      } else {
        const bool cd = act && !used && m != r && R > r_min && Z > Zr && !crit;
        d = group_arg<true>(cd && sur, Z, G, gbase, gmask);
        if (d < 0) d = group_arg<true>(cd && !sur, Z, G, gbase, gmask);
        if (d < 0) break;
        if (m == d) {
          R -= 1;
          used = true;
        }
      }
      if (m == r) {
        R += 1;
        used = true;
      }
      if (m == 0 && nm < p.move_cap) {
        tre_move mv;
        mv.window = (uint32_t)w;
        mv.path = (uint8_t)path;
        mv.receiver = (uint8_t)r;
        mv.donor = (uint8_t)d;
        mv.pad = 0;
        p.moves[(int64_t)s * p.move_cap + nm] = mv;
      }
      ++nm;
    }
  }
  rw += (long long)R * (p.n_windows - 1 - wprev);
  if (act) {
    p.r_final[(int64_t)s * M + m] = R;
    p.r_windows[(int64_t)s * M + m] = rw;
  }
  if (sc_ok && m == 0) p.n_moves[s] = nm;
}

// ---------------------------------------------------------------- validate
struct ValParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint8_t* type;
  const int64_t* off;
  uint32_t n_traces;
  int64_t duration_ms;
  int64_t window_ms;
  int32_t M;
  unsigned* err;             // bit 0 order, bit 1 schema, bit 2 range
  unsigned long long* first; // lowest failing row
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
      if (t_i < 0 || t_i >= p.duration_ms || (i > b && t_i < p.ts[i - 1])) bad |= 1u;
      if (p.model[i] >= p.M || (ty & 0x7Cu) || ((ty & TRE_ADMIT) && (ty & 3u) != TRE_PREFILL)) bad |= 2u;
      const int64_t j = i + TRE_MAX_EVENTS_PER_WINDOW;
      if (!(bad & 1u) && j < e && p.ts[j] / p.window_ms == t_i / p.window_ms) bad |= 4u;
      if (bad) {
        atomicOr(p.err, bad);
        atomicMin(p.first, (unsigned long long)i);
      }
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

struct LaunchTimer {
  Pending pe{};
  bool on = false;
  hipStream_t st;
  LaunchTimer(const char* name, hipStream_t s) : st(s) {
    std::lock_guard<std::mutex> lk(g_tmu);
    if (!g_timing) return;
    pe.name = name;
    if (hipEventCreate(&pe.start) != hipSuccess) return;
    if (hipEventCreate(&pe.stop) != hipSuccess) {
      (void)hipEventDestroy(pe.start);
      return;
    }
    on = hipEventRecord(pe.start, st) == hipSuccess;
  }
  void done() {
    if (!on) return;
    (void)hipEventRecord(pe.stop, st);
    std::lock_guard<std::mutex> lk(g_tmu);
    g_pending.push_back(pe);
    on = false;
  }
};
}  // namespace

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
static int check_device(const tre_events* ev) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != ev->device)
    return fail(TRE_EINVAL, "handle belongs to device %d, current device is %d", ev->device, dev);
  return TRE_OK;
}

static uint32_t ring_windows(int M) {
  uint32_t w = 256;
  while (w > 2 && (size_t)3 * w * (size_t)M * 8 > (size_t)kRingBytes) w >>= 1;
  return w;
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
    if (trace_off[i + 1] - trace_off[i] >= (1ll << 31))
      return fail(TRE_ERANGE, "trace %u has 2^31 or more events", i);
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
    int64_t maxlen = 0;
    for (uint32_t i = 0; i < n_traces; ++i)
      maxlen = std::max<int64_t>(maxlen, trace_off[i + 1] - trace_off[i]);
    void* scratch = nullptr;
    if (hipMalloc(&scratch, 16) != hipSuccess) return cleanup(fail(TRE_EHIP, "hipMalloc failed"));
    unsigned* d_err = (unsigned*)scratch;
    unsigned long long* d_first = (unsigned long long*)((char*)scratch + 8);
    unsigned h_init[4] = {0u, 0u, 0xFFFFFFFFu, 0xFFFFFFFFu};
    unsigned long long h_first = ~0ull;
    unsigned h_err = 0;
    bool ok = hipMemcpyAsync(scratch, h_init, 16, hipMemcpyHostToDevice, st) == hipSuccess;
    if (ok && maxlen > 0) {
      ValParams vp{ts, model, type, ev->d_off, n_traces, c.duration_ms, c.window_ms, c.n_models, d_err, d_first};
      dim3 grid((unsigned)((maxlen + kValChunk - 1) / kValChunk), std::min<uint32_t>(n_traces, 65535u));
      LaunchTimer lt("validate", st);
      hipLaunchKernelGGL(validate, grid, dim3(256), 0, st, vp);
      ok = hipGetLastError() == hipSuccess;
      lt.done();
    }
    ok = ok && hipMemcpyAsync(&h_err, d_err, 4, hipMemcpyDeviceToHost, st) == hipSuccess &&
         hipMemcpyAsync(&h_first, d_first, 8, hipMemcpyDeviceToHost, st) == hipSuccess &&
         hipStreamSynchronize(st) == hipSuccess;
    (void)hipFree(scratch);
    if (!ok) return cleanup(fail(TRE_EHIP, "validation launch failed"));
    if (h_err & 1u) rc = fail(TRE_EORDER, "row %llu: timestamp unsorted or outside [0, duration)", h_first);
    else if (h_err & 2u) rc = fail(TRE_ESCHEMA, "row %llu: model index or type byte invalid", h_first);
    else if (h_err & 4u)
      rc = fail(TRE_ERANGE, "row %llu: more than %d events in one window", h_first,
                TRE_MAX_EVENTS_PER_WINDOW);
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

extern "C" int tre_workspace_size(const tre_events* ev, uint32_t n_scenarios, size_t* bytes) {
  if (!ev || !bytes) return fail(TRE_EINVAL, "tre_workspace_size: NULL argument");
  (void)n_scenarios;
  *bytes = (size_t)ev->n_traces * (size_t)ev->n_ticks * (size_t)ev->cfg.n_models * sizeof(double);
  if (*bytes == 0) *bytes = 256;
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
  p.n_windows = (int32_t)ev->n_windows;
  p.M = ev->cfg.n_models;
  p.wcap = ev->wcap;
  p.fast_w = (int32_t)(ev->cfg.fast_period_ms / ev->cfg.window_ms);
  p.slow_w = (int32_t)(ev->cfg.slow_period_ms / ev->cfg.window_ms);
  p.n_ticks = (int32_t)ev->n_ticks;
  return p;
}

static int launch_stream(const tre_events* ev, const StreamParams& p, hipStream_t st) {
  const size_t lds = (size_t)3 * ev->wcap * (size_t)ev->cfg.n_models * sizeof(unsigned long long);
  LaunchTimer lt("tss_stream", st);
  hipLaunchKernelGGL(tss_stream, dim3(ev->n_traces), dim3(kBlock), lds, st, p);
  const hipError_t e = hipGetLastError();
  lt.done();
  if (e != hipSuccess) return fail(TRE_EHIP, "tss_stream launch: %s", hipGetErrorString(e));
  return TRE_OK;
}

static int g_log2_for(int M) {
  int g = 0;
  while ((1 << g) < M) ++g;
  return g;
}

static int launch_rebalance(const tre_events* ev, const tre_profile* prof, const double* vals,
                            const uint8_t* flags, const tre_scenario* sc, uint32_t n_sc,
                            const tre_ctl_out* out, hipStream_t st) {
  CtlParams c{};
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
  c.g_log2 = g_log2_for(ev->cfg.n_models);
  c.budget = ev->cfg.budget;
  c.n_traces = ev->n_traces;
  c.moves = out->moves;
  c.move_cap = out->move_cap;
  c.n_moves = out->n_moves;
  c.r_final = out->r_final;
  c.r_windows = out->r_windows;
  const uint32_t spw = 64u >> c.g_log2;
  const uint64_t waves = ((uint64_t)n_sc + spw - 1) / spw;
  const uint64_t blocks = (waves + 3) / 4;
  LaunchTimer lt("rebalance", st);
  hipLaunchKernelGGL(rebalance, dim3((unsigned)blocks), dim3(256), 0, st, c);
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

extern "C" int tre_rebalance(const tre_events* ev, const tre_profile* prof, const double* tss64,
                             const uint8_t* flags, const tre_scenario* sc, uint32_t n_scenarios,
                             const tre_ctl_out* out, void* stream) {
  if (!ev || !prof || !tss64 || !flags) return fail(TRE_EINVAL, "tre_rebalance: NULL argument");
  if (n_scenarios && !sc) return fail(TRE_EINVAL, "tre_rebalance: NULL scenarios");
  int rc = check_ctl_out(out, n_scenarios);
  if (rc) return rc;
  rc = check_device(ev);
  if (rc) return rc;
  if (n_scenarios == 0) return TRE_OK;
  return launch_rebalance(ev, prof, tss64, flags, sc, n_scenarios, out, (hipStream_t)stream);
}

extern "C" int tre_sweep(const tre_events* ev, const tre_profile* prof, const tre_scenario* sc,
                         uint32_t n_scenarios, const tre_ctl_out* out, float* tss32, void* ws,
                         size_t ws_bytes, void* stream) {
  if (!ev || !prof) return fail(TRE_EINVAL, "tre_sweep: NULL argument");
  if (n_scenarios && !sc) return fail(TRE_EINVAL, "tre_sweep: NULL scenarios");
  int rc = check_ctl_out(out, n_scenarios);
  if (rc) return rc;
  rc = check_device(ev);
  if (rc) return rc;
  size_t need = 0;
  tre_workspace_size(ev, n_scenarios, &need);
  if (!ws || ws_bytes < need)
    return fail(TRE_ENOMEM, "workspace of %zu bytes is smaller than the %zu needed", ws_bytes, need);
  if ((uintptr_t)ws & 7) return fail(TRE_EINVAL, "workspace must be 8-byte aligned");
  hipStream_t st = (hipStream_t)stream;
  StreamParams p = stream_params(ev, prof);
  p.tss32 = tss32;
  p.snap = (double*)ws;
  rc = launch_stream(ev, p, st);
  if (rc || n_scenarios == 0) return rc;
  return launch_rebalance(ev, prof, (const double*)ws, nullptr, sc, n_scenarios, out, st);
}
