// calib.hip - the calibration sweep on MI355X (gfx950): per-request latencies
// joined from the event stream by request id, per-window SLO attainment, and
// the fit of each model's healthy boundary theta from the smoothed TSS.
//
// Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE). SLOs are
// stated on TTFT, TPOT and E2E latency as tail percentiles (background
// section on SLOs); theta_m is the smallest smoothed TSS that still achieves
// the target SLO reliability, derived offline across the healthy-to-degraded
// transition (Section "Smoothing, Normalization, and Calibration"); RQ1 asks
// that TSS follow the SLO-health ordering, reported here as the healthy
// counts above the fitted boundary.
//
// Kernels (all on the caller's stream)
//   fill_u32     sets the request table to all ones and the counts to zero.
//   calib_join   one workgroup per chunk of a trace: streams (req, type,
//                tokens), combines each request's events in an LDS hash table
//                (minimum ARRIVE / DECODE / FINISH rows, DECODE token sum),
//                judges the requests whose events all lie in the chunk
//                (latencies, SLO test, one atomic add into the arrival
//                window's packed (judged, ok) counter) and merges the others
//                into their 16-byte global records with atomics.
//   calib_judge  one thread per request slot: the requests that spanned
//                chunks or never finished, judged the same way from their
//                records (ts, model and tokens gathered at the rows).
//   calib_fit    one 1024-thread workgroup per (trace, model): candidate keys
//                (S bit pattern, health bit) in registers, an LSD radix sort
//                in LDS (8-bit digits, constant digits skipped, stable ranks
//                from wave ballots), then one scan for the smallest
//                qualifying threshold.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "tre.h"
#include "tre_internal.h"

#pragma clang fp contract(off)

using tre_internal::check_device;
using tre_internal::fail;
using tre_internal::LaunchTimer;

namespace {

constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr int kJoinChunk = 8192;    // events per calib_join workgroup
constexpr int kFitThreads = 1024;   // calib_fit workgroup
constexpr int kFitWaves = kFitThreads / 64;
constexpr int kFitMaxKPT = 16;      // keys per thread: windows up to 16384

__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }

// ------------------------------------------------------------------- fill
__global__ __launch_bounds__(256) void fill_u32(uint32_t* p, uint64_t n, uint32_t v) {
  const uint64_t n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint4* q = (uint4*)p;
  const uint4 vv = make_uint4(v, v, v, v);
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) q[i] = vv;
  for (uint64_t i = 4 * n4 + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// ------------------------------------------------------------------- join
struct JoinParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint32_t* req;
  const uint8_t* type;
  const uint16_t* tokens;
  const int64_t* off;
  const tre_slo* slo;           // [n_traces][M]
  uint32_t* counts;             // [n_traces][M][n_windows]: judged << 16 | ok
  tre_req_latency* reqs;        // [n_traces][req_cap] or NULL
  uint32_t* tab;                // [n_traces][req_cap][4]: a, f, e, ~dsum
  unsigned long long* n_bad;    // events whose id is >= req_cap
  uint32_t n_traces;
  uint32_t req_cap;
  uint32_t n_chunks;            // chunks of the longest trace
  int32_t M;
  int64_t window_ms;
  int64_t n_windows;
};

constexpr int kHashSlots = 2048;           // LDS records per chunk (load factor about 0.4)
constexpr int kProbes = 16;                // linear probes before the global fallback
constexpr int kJoinBatch = 8;              // events per thread loaded together
constexpr uint32_t kDone = 0xFFFFFFFEu;    // record judged inside the join

// latencies and the SLO test of one judged request from its event times
__device__ __forceinline__ tre_req_latency judge_one(int64_t ta, int64_t tf, int64_t te, uint32_t after_first,
                                                     uint32_t m, const tre_slo& s) {
  tre_req_latency out;
  out.model = (uint8_t)m;
  out.flags = TRE_REQ_ARRIVED | TRE_REQ_COMPLETE;
  for (int i = 0; i < 6; ++i) out.pad[i] = 0;
  const int64_t ttft = tf - ta, e2e = te - ta;
  bool good = (double)ttft <= s.ttft_ms && (double)e2e <= s.e2e_ms;
  out.tpot_ms = 0.0;
  if (after_first > 0) {
    const double tpot = (double)(te - tf) / (double)after_first;
    good = good && tpot <= s.tpot_ms;
    out.tpot_ms = tpot;
    out.flags |= TRE_REQ_TPOT;
  }
  if (good) out.flags |= TRE_REQ_OK;
  out.ttft_ms = (uint32_t)ttft;
  out.e2e_ms = (uint32_t)e2e;
  return out;
}

__device__ __forceinline__ tre_req_latency not_judged(uint32_t m) {
  tre_req_latency out;
  out.ttft_ms = out.e2e_ms = 0;
  out.tpot_ms = 0.0;
  out.model = (uint8_t)m;
  out.flags = TRE_REQ_ARRIVED;
  for (int i = 0; i < 6; ++i) out.pad[i] = 0;
  return out;
}

// One workgroup per chunk of kJoinChunk rows of one trace. The chunk's
// events are first combined per request in an LDS hash table (minimum rows
// of ARRIVE / DECODE / FINISH, DECODE token sum). A request whose ARRIVE,
// DECODE and FINISH all fall in the chunk has every event in it (a
// request's events lie between its ARRIVE and FINISH), so it is judged
// right here and never touches the global table; the others merge into
// their global records with atomics, for calib_judge. Chunks of one trace
// are numbered onto one XCD.
__global__ __launch_bounds__(256) void calib_join(JoinParams p) {
  __shared__ uint32_t h_id[kHashSlots], h_a[kHashSlots], h_f[kHashSlots], h_e[kHashSlots], h_d[kHashSlots];
  const uint32_t xcd = blockIdx.x & 7u, kk = blockIdx.x >> 3;
  const uint32_t t = (kk / p.n_chunks) * 8u + xcd, chunk = kk % p.n_chunks;
  if (t >= p.n_traces) return;  // whole block
  const int64_t b = p.off[t], e = p.off[t + 1];
  const int64_t c0 = b + (int64_t)chunk * kJoinChunk;
  if (c0 >= e) return;  // whole block
  const int64_t c1 = c0 + kJoinChunk < e ? c0 + kJoinChunk : e;
  uint32_t* tt = p.tab + (uint64_t)t * p.req_cap * 4;
  for (int i = threadIdx.x; i < kHashSlots; i += 256) {
    h_id[i] = kNone;
    h_a[i] = kNone;
    h_f[i] = kNone;
    h_e[i] = kNone;
    h_d[i] = 0;
  }
  __syncthreads();
  unsigned bad = 0;
  for (int64_t i0 = c0 + threadIdx.x; i0 < c1; i0 += 256 * kJoinBatch) {
    uint32_t rr[kJoinBatch], kt[kJoinBatch], tk[kJoinBatch];
#pragma unroll
    for (int u = 0; u < kJoinBatch; ++u) {
      const int64_t i = i0 + 256 * u;
      const bool in = i < c1;
      rr[u] = in ? p.req[i] : kNone;
      kt[u] = in ? p.type[i] : TRE_PREFILL;
      tk[u] = in ? p.tokens[i] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kJoinBatch; ++u) {
      const int64_t i = i0 + 256 * u;
      if (i >= c1) continue;
      const uint32_t r = rr[u];
      if (r >= p.req_cap) {
        ++bad;
        continue;
      }
      const uint32_t k = kt[u] & 3u;
      if (k == TRE_PREFILL) continue;
      const uint32_t row = (uint32_t)(i - b);
      uint32_t h = (r * 0x9E3779B1u) >> (32 - 11);
      int slot = -1;
      for (int q = 0; q < kProbes; ++q) {
        const uint32_t old = atomicCAS(&h_id[h], kNone, r);
        if (old == kNone || old == r) {
          slot = (int)h;
          break;
        }
        h = (h + 1) & (kHashSlots - 1);
      }
      if (slot >= 0) {
        if (k == TRE_ARRIVE) {
          atomicMin(&h_a[slot], row);
        } else if (k == TRE_DECODE) {
          atomicMin(&h_f[slot], row);
          atomicAdd(&h_d[slot], tk[u]);
        } else {
          atomicMin(&h_e[slot], row);
        }
      } else {  // table crowded: straight to the global record
        uint32_t* rec = tt + (uint64_t)r * 4;
        if (k == TRE_ARRIVE) {
          atomicMin(rec, row);
        } else if (k == TRE_DECODE) {
          atomicMin(rec + 1, row);
          atomicSub(rec + 3, tk[u]);
        } else {
          atomicMin(rec + 2, row);
        }
      }
    }
  }
  __syncthreads();
  for (int s = threadIdx.x; s < kHashSlots; s += 256) {
    const uint32_t r = h_id[s];
    if (r == kNone) continue;
    uint32_t* rec = tt + (uint64_t)r * 4;
    const uint32_t a = h_a[s], f = h_f[s], fin = h_e[s], d = h_d[s];
    if (a != kNone && f != kNone && fin != kNone) {
      const uint32_t m = p.model[b + a];
      tre_req_latency out;
      if (m < (uint32_t)p.M) {
        const int64_t ta = p.ts[b + a];
        out = judge_one(ta, p.ts[b + f], p.ts[b + fin], d - (uint32_t)p.tokens[b + f], m,
                        p.slo[(uint64_t)t * p.M + m]);
        const int64_t w = ta / p.window_ms;  // window of arrival
        if (w >= 0 && w < p.n_windows)
          atomicAdd(p.counts + ((uint64_t)t * p.M + m) * p.n_windows + w,
                    (1u << 16) | ((out.flags & TRE_REQ_OK) ? 1u : 0u));
      } else {
        out = not_judged(m);
      }
      if (p.reqs) {
        p.reqs[(uint64_t)t * p.req_cap + r] = out;
        rec[0] = kDone;  // calib_judge leaves this slot alone
      }
      continue;
    }
    if (a != kNone) atomicMin(rec, a);
    if (f != kNone) {
      atomicMin(rec + 1, f);
      atomicSub(rec + 3, d);
    }
    if (fin != kNone) atomicMin(rec + 2, fin);
  }
  // one atomic per wave for the ids out of range
  for (int o = 32; o > 0; o >>= 1) bad += __shfl_xor(bad, o);
  if ((threadIdx.x & 63) == 0 && bad) atomicAdd(p.n_bad, (unsigned long long)bad);
}

// ------------------------------------------------------------------ judge
struct JudgeParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint16_t* tokens;
  const int64_t* off;
  const uint32_t* tab;
  const tre_slo* slo;           // [n_traces][M]
  uint32_t* counts;             // [n_traces][M][n_windows]: judged << 16 | ok
  tre_req_latency* reqs;        // [n_traces][req_cap] or NULL
  uint32_t n_traces;
  uint32_t req_cap;
  int32_t M;
  int64_t window_ms;
  int64_t n_windows;
};

// The requests the join could not finish: one thread per request slot.
__global__ __launch_bounds__(256) void calib_judge(JudgeParams p) {
  const uint32_t r = blockIdx.x * 256 + threadIdx.x;
  if (r >= p.req_cap) return;
  for (uint32_t t = blockIdx.y; t < p.n_traces; t += gridDim.y) {
    const uint64_t slot = (uint64_t)t * p.req_cap + r;
    const uint4 rec = ((const uint4*)p.tab)[slot];
    if (rec.x == kDone) continue;  // judged inside the join
    const int64_t b = p.off[t];
    tre_req_latency out = not_judged(0xFF);
    out.flags = 0;
    if (rec.x != kNone) {
      const uint32_t m = p.model[b + rec.x];
      out = not_judged(m);
      if (rec.y != kNone && rec.z != kNone && m < (uint32_t)p.M) {
        const int64_t ta = p.ts[b + rec.x];
        out = judge_one(ta, p.ts[b + rec.y], p.ts[b + rec.z], ~rec.w - (uint32_t)p.tokens[b + rec.y], m,
                        p.slo[(uint64_t)t * p.M + m]);
        const int64_t w = ta / p.window_ms;  // window of arrival
        if (w >= 0 && w < p.n_windows)
          atomicAdd(p.counts + ((uint64_t)t * p.M + m) * p.n_windows + w,
                    (1u << 16) | ((out.flags & TRE_REQ_OK) ? 1u : 0u));
      }
    }
    if (p.reqs) p.reqs[slot] = out;
  }
}

// -------------------------------------------------------------------- fit
struct FitParams {
  const double* tss64;          // [n_traces][n_windows][M]
  const uint8_t* flags;         // [n_traces][n_windows][M]
  const uint32_t* counts;       // [n_traces][M][n_windows]
  const tre_slo* slo;           // [n_traces][M]
  tre_fit* fit;                 // [n_traces][M]
  int32_t order;                // also the ordering counts (tre_calib_order)
  uint32_t n_traces;
  int32_t M;
  int64_t n_windows;
};

// exclusive prefix sum over the workgroup of one value per thread; `tot`
// receives the total. Uses sc[kFitWaves + 1].
__device__ __forceinline__ uint32_t block_exclusive_sum(uint32_t v, uint32_t* sc, uint32_t& tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) sc[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < kFitWaves; ++w) {
      const uint32_t c = sc[w];
      sc[w] = run;
      run += c;
    }
    sc[kFitWaves] = run;
  }
  __syncthreads();
  const uint32_t r = sc[wave] + x - v;
  tot = sc[kFitWaves];
  __syncthreads();
  return r;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int o) {
  return ((uint64_t)(uint32_t)__shfl_xor((int)(x >> 32), o) << 32) | (uint32_t)__shfl_xor((int)(uint32_t)x, o);
}

// workgroup reductions of 64-bit values: 0 OR, 1 AND, 2 MIN, 3 MAX
template <int kOp>
__device__ __forceinline__ uint64_t block_reduce_u64(uint64_t v, uint64_t* sc) {
  auto op = [](uint64_t a, uint64_t b) {
    return kOp == 0 ? (a | b) : kOp == 1 ? (a & b) : kOp == 2 ? (a < b ? a : b) : (a > b ? a : b);
  };
  for (int o = 32; o > 0; o >>= 1) v = op(v, shfl_xor_u64(v, o));
  if ((threadIdx.x & 63) == 0) sc[threadIdx.x >> 6] = v;
  __syncthreads();
  uint64_t r = sc[0];
  for (int w = 1; w < kFitWaves; ++w) r = op(r, sc[w]);
  __syncthreads();
  return r;
}

__device__ __forceinline__ uint32_t block_min_u32(uint32_t v, uint32_t* sc) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t y = (uint32_t)__shfl_xor((int)v, o);
    v = y < v ? y : v;
  }
  if ((threadIdx.x & 63) == 0) sc[threadIdx.x >> 6] = v;
  __syncthreads();
  uint32_t r = sc[0];
  for (int w = 1; w < kFitWaves; ++w) r = sc[w] < r ? sc[w] : r;
  __syncthreads();
  return r;
}

constexpr int kBuckets = 2048;      // histogram of the fit (2^11)
constexpr int kResolveCap = 1024;   // keys sorted exactly before the radix fallback

// One 1024-thread workgroup per (trace, model). Candidate keys
// (S bit pattern << 1 | healthy) go to LDS; they order like S, and equal S
// differ only in bit 0. A threshold at a run of equal S covers the run and
// every larger S; in ascending order the run starts at position g, with
// N = n - g candidates and H = Ht - (healthy below g) healthy ones at or
// above it, and qualifies when H >= rho * N (fp64). theta is the smallest
// qualifying S, i.e. the lowest qualifying g.
//   1. Histogram of the keys into 2048 buckets on the 11 highest bits above
//      bit 0 where keys differ (equal S share a bucket); an exclusive scan
//      gives each bucket's first position G_b and healthy count below P_b,
//      so each bucket's first position is tested exactly.
//   2. A position inside bucket b (c keys, u of them unhealthy) can only
//      qualify if the test can move from failing to passing within the
//      bucket: at most rho * u is gained, so for 0 <= rho <= 1 the bucket is
//      skipped when rho * (N - u) >= H + 1 (the margin of one absorbs the
//      rounding of the products); otherwise H < rho * (N - c + 1) is used.
//   3. Let b* be the lowest bucket whose first position qualifies. The keys
//      of the remaining buckets below b* are gathered, sorted (bitonic in
//      LDS) and tested at each run start; the lowest qualifying one, else
//      b*'s first position, is the answer.
//   4. If those keys exceed kResolveCap, every key is sorted instead (LSD
//      radix, 8-bit digits, constant digits skipped, stable ranks from wave
//      ballots) and every run start tested.
template <int KPT>
__global__ __launch_bounds__(kFitThreads) void calib_fit(FitParams p) {
  __shared__ uint64_t keys_lds[kFitThreads * KPT];
  __shared__ uint32_t hist[2 * kBuckets];  // buckets: counts then (G, P), compact offsets; radix: [digit][wave]
  __shared__ uint64_t cmp[kResolveCap];
  __shared__ uint64_t sc64[kFitWaves];
  __shared__ uint32_t sc32[kFitWaves + 1];
  __shared__ uint32_t n_gathered;
  __shared__ uint32_t hpre_s[kFitThreads];  // healthy keys before each gathered position
  static_assert(256 * kFitWaves == 2 * kBuckets, "radix histogram and bucket tables share LDS");

  // XCD-aware block order: consecutive blocks go to different XCDs, so the
  // models of one trace are numbered to land on one XCD and share its L2
  // for the strided per-cell reads
  const uint32_t b = blockIdx.x;
  const uint32_t xcd = b & 7u, k = b >> 3;
  const uint32_t t = (k / (uint32_t)p.M) * 8u + xcd;
  const uint32_t m = k % (uint32_t)p.M;
  if (t >= p.n_traces) return;  // whole block
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tid = threadIdx.x;
  const int64_t nW = p.n_windows;
  const tre_slo s = p.slo[(uint64_t)t * p.M + m];
  const double rho = s.reliability;
  const uint32_t* cnt = p.counts + ((uint64_t)t * p.M + m) * nW;
  tre_fit* dst = p.fit + (uint64_t)t * p.M + m;

  // candidate keys to LDS in element order; non-candidates marked ~0 (no key
  // of a finite S reaches it)
  uint64_t kmax = 0, kor = 0, kand = ~0ull;
  uint32_t n_real = 0, h_real = 0;
#pragma unroll 2
  for (int j = 0; j < KPT; ++j) {
    const int64_t w = (int64_t)wave * KPT * 64 + j * 64 + lane;
    uint64_t kk = ~0ull;
    if (w < nW) {
      const uint32_t c = cnt[w];
      const uint32_t judged = c >> 16, ok = c & 0xFFFFu;
      const uint64_t cell = ((uint64_t)t * nW + w) * p.M + m;
      const uint8_t fl = p.flags[cell];
      if (judged > 0 && (fl & TRE_FLAG_INIT) && !(fl & TRE_FLAG_IDLE)) {
        const bool healthy = (double)ok >= s.attain_q * (double)judged;
        kk = (dbits(p.tss64[cell]) << 1) | (healthy ? 1ull : 0ull);
        kmax = kk > kmax ? kk : kmax;
        kor |= kk;
        kand &= kk;
        ++n_real;
        h_real += healthy ? 1u : 0u;
      }
    }
    keys_lds[wave * KPT * 64 + j * 64 + lane] = kk;
  }
  uint32_t n_cand, Ht;
  (void)block_exclusive_sum(n_real, sc32, n_cand);
  (void)block_exclusive_sum(h_real, sc32, Ht);
  tre_fit out;
  out.theta = INFINITY;
  out.n_cand = n_cand;
  out.n_healthy = Ht;
  out.n_above = 0;
  out.healthy_above = 0;
  out.concordant = 0;  // no pair of candidates with different S: none either way
  out.discordant = 0;
  if (n_cand == 0) {
    if (tid == 0) *dst = out;
    return;
  }
  kmax = block_reduce_u64<3>(kmax, sc64);
  const uint64_t vary = block_reduce_u64<0>(kor, sc64) ^ block_reduce_u64<1>(kand, sc64);
  const uint64_t vary_s = vary & ~1ull;
  if (vary_s == 0) {  // one value of S: a single run covering every candidate
    if (tid == 0) {
      if ((double)Ht >= rho * (double)n_cand) {
        out.theta = __longlong_as_double((long long)(kmax >> 1));
        out.n_above = n_cand;
        out.healthy_above = Ht;
      }
      *dst = out;
    }
    return;
  }

  // ---- 1. histogram over buckets, packed (healthy << 16) | count
  const int hb = 63 - __clzll((long long)vary_s);
  const int lo = hb >= 11 ? hb - 10 : 1;
  auto bucket = [&](uint64_t key) { return (uint32_t)(key >> lo) & (uint32_t)(kBuckets - 1); };
  for (int i = tid; i < kBuckets; i += kFitThreads) hist[i] = 0;
  __syncthreads();
#pragma unroll 4
  for (int j = 0; j < KPT; ++j) {
    const uint64_t kk = keys_lds[wave * KPT * 64 + j * 64 + lane];
    if (kk != ~0ull) atomicAdd(&hist[bucket(kk)], ((uint32_t)(kk & 1ull) << 16) | 1u);
  }
  __syncthreads();
  // two buckets per thread; counts and healthy counts stay below 2^16
  const uint32_t v0 = hist[2 * tid], v1 = hist[2 * tid + 1];
  uint32_t tot;
  const uint32_t ex = block_exclusive_sum(v0 + v1, sc32, tot);
  const uint32_t offs[2] = {ex, ex + v0}, cnts[2] = {v0, v1};
  // ---- 2. bucket status; the ordering counts across buckets: every key of
  // a lower bucket has a smaller S, so bucket b pairs its u unhealthy keys
  // with the P healthy keys below it (discordant) and its healthy keys with
  // the G - P unhealthy keys below it (concordant). Pairs inside a bucket
  // need its keys in order; only buckets holding both kinds have any.
  uint32_t qual_b = kNone;
  bool maybe[2];
  uint32_t d_cross = 0, c_cross = 0, hu_mixed = 0, mixed[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const uint32_t c = cnts[q] & 0xFFFFu, h = cnts[q] >> 16, u = c - h;
    const uint32_t G = offs[q] & 0xFFFFu, P = offs[q] >> 16;
    const uint32_t N = n_cand - G, H = Ht - P;
    d_cross += u * P;
    c_cross += h * (G - P);
    mixed[q] = (h != 0u && u != 0u) ? c : 0u;
    hu_mixed += h * u;
    maybe[q] = false;
    if (c == 0) continue;
    if ((double)H >= rho * (double)N) {
      if (qual_b == kNone) qual_b = 2u * tid + q;
    } else if (c >= 2) {
      const bool skip = (rho >= 0.0 && rho <= 1.0) ? rho * (double)(N - u) >= (double)H + 1.0
                                                   : (double)H < rho * (double)(N - c + 1);
      maybe[q] = !skip;
    }
  }
  const uint32_t bstar = block_min_u32(qual_b, sc32);
  uint32_t D_cross = 0, C_cross = 0, HU_mixed = 0, mx_tot = 0, mx_ex = 0;
  if (p.order) {  // uniform
    (void)block_exclusive_sum(d_cross, sc32, D_cross);
    (void)block_exclusive_sum(c_cross, sc32, C_cross);
    (void)block_exclusive_sum(hu_mixed, sc32, HU_mixed);
    mx_ex = block_exclusive_sum(mixed[0] + mixed[1], sc32, mx_tot);
  }
  // ---- 3. keys of the undecided buckets below b*
  uint32_t mc[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) mc[q] = (maybe[q] && 2u * tid + q < bstar) ? (cnts[q] & 0xFFFFu) : 0u;
  uint32_t mtot;
  const uint32_t mex = block_exclusive_sum(mc[0] + mc[1], sc32, mtot);
  __shared__ tre_fit s_out;
  // the keys of the listed buckets (bit 31 of their hist[kBuckets + b] entry),
  // gathered into cmp at their compact offsets and sorted (bitonic); returns
  // with every thread holding cmp[tid] (or ~0) in `ck`
  auto gather_sort = [&](uint32_t n_keys, uint64_t& ck) {
    if (tid == 0) n_gathered = 0;
    __syncthreads();
#pragma unroll 4
    for (int j = 0; j < KPT; ++j) {
      const uint64_t kk = keys_lds[wave * KPT * 64 + j * 64 + lane];
      if (kk == ~0ull) continue;
      if (hist[kBuckets + bucket(kk)] & 0x80000000u) cmp[atomicAdd(&n_gathered, 1u)] = kk;
    }
    uint32_t p2 = 2;
    while (p2 < n_keys) p2 <<= 1;
    for (uint32_t i = n_keys + tid; i < p2; i += kFitThreads) cmp[i] = ~0ull;
    __syncthreads();
    for (uint32_t kk2 = 2; kk2 <= p2; kk2 <<= 1) {
      for (uint32_t jj = kk2 >> 1; jj > 0; jj >>= 1) {
        const uint32_t i = tid, ixj = tid ^ jj;
        if (i < p2 && ixj > i) {
          const uint64_t x = cmp[i], y = cmp[ixj];
          if ((x > y) == ((i & kk2) == 0)) {
            cmp[i] = y;
            cmp[ixj] = x;
          }
        }
        __syncthreads();
      }
    }
    ck = tid < (int)n_keys ? cmp[tid] : ~0ull;
  };
  if (mtot <= (uint32_t)kResolveCap && (!p.order || mx_tot <= (uint32_t)kResolveCap)) {
    // per bucket: (G, P) and the compact offset with bit 31 marking a gathered bucket
    hist[2 * tid] = offs[0];
    hist[2 * tid + 1] = offs[1];
    hist[kBuckets + 2 * tid] = mex | (mc[0] ? 0x80000000u : 0u);
    hist[kBuckets + 2 * tid + 1] = (mex + mc[0]) | (mc[1] ? 0x80000000u : 0u);
    uint64_t kstar = ~0ull;  // smallest key of bucket b*
#pragma unroll 4
    for (int j = 0; j < KPT; ++j) {
      const uint64_t kk = keys_lds[wave * KPT * 64 + j * 64 + lane];
      if (kk != ~0ull && bucket(kk) == bstar) kstar = kk < kstar ? kk : kstar;
    }
    kstar = block_reduce_u64<2>(kstar, sc64);
    uint64_t ck;
    gather_sort(mtot, ck);
    // healthy keys before each gathered position; the gathered keys of one
    // bucket are contiguous, from its compact offset
    uint32_t unused;
    const uint32_t hpre = block_exclusive_sum(tid < (int)mtot ? (uint32_t)(ck & 1ull) : 0u, sc32, unused);
    uint32_t* const hpre_l = hpre_s;
    hpre_l[tid] = hpre;
    __syncthreads();
    uint32_t cand_g = kNone, cand_h = 0;
    if (tid < (int)mtot) {
      const uint32_t bk = bucket(ck);
      const uint32_t cf = hist[kBuckets + bk] & 0x7FFFFFFFu, GP = hist[bk];
      const uint32_t i = (uint32_t)tid - cf, g = (GP & 0xFFFFu) + i;
      if (i == 0 || (cmp[tid - 1] >> 1) != (ck >> 1)) {
        const uint32_t H = Ht - ((GP >> 16) + hpre - hpre_l[cf]), N = n_cand - g;
        if ((double)H >= rho * (double)N) {
          cand_g = g;
          cand_h = H;
        }
      }
    }
    const uint32_t gmin = block_min_u32(cand_g, sc32);
    if (gmin != kNone) {
      if (cand_g == gmin) {
        s_out.theta = __longlong_as_double((long long)(ck >> 1));
        s_out.n_above = n_cand - gmin;
        s_out.healthy_above = cand_h;
      }
    } else if (tid == 0) {
      s_out.theta = INFINITY;
      s_out.n_above = 0;
      s_out.healthy_above = 0;
      if (bstar != kNone) {
        const uint32_t GP = hist[bstar];
        s_out.theta = __longlong_as_double((long long)(kstar >> 1));
        s_out.n_above = n_cand - (GP & 0xFFFFu);
        s_out.healthy_above = Ht - (GP >> 16);
      }
    }
    if (!p.order) {
      if (tid == 0) {
        out.theta = s_out.theta;
        out.n_above = s_out.n_above;
        out.healthy_above = s_out.healthy_above;
        *dst = out;
      }
      return;
    }
    // ---- the ordering counts inside the buckets that hold both kinds:
    // their keys gathered and sorted; in a run of equal S the unhealthy keys
    // (bit 0 clear) come first, so the healthy keys before an unhealthy one
    // inside its bucket all have a smaller S (discordant pairs); the mixed
    // pairs of equal S are counted per run, the rest are concordant
    hist[kBuckets + 2 * tid] = mx_ex | (mixed[0] ? 0x80000000u : 0u);
    hist[kBuckets + 2 * tid + 1] = (mx_ex + mixed[0]) | (mixed[1] ? 0x80000000u : 0u);
    uint64_t mk;
    gather_sort(mx_tot, mk);
    const bool in = tid < (int)mx_tot;
    const uint32_t mh = block_exclusive_sum(in ? (uint32_t)(mk & 1ull) : 0u, sc32, unused);
    hpre_l[tid] = mh;
    __syncthreads();
    uint32_t d_in = 0, tie = 0;
    if (in) {
      const uint32_t cf = hist[kBuckets + bucket(mk)] & 0x7FFFFFFFu;
      if (!(mk & 1ull)) d_in = mh - hpre_l[cf];
      if (tid == (int)cf || (cmp[tid - 1] >> 1) != (mk >> 1)) {  // a run start: walk the run
        uint32_t ru = 0, rh = 0;
        for (uint32_t i = (uint32_t)tid; i < mx_tot && (cmp[i] >> 1) == (mk >> 1); ++i) {
          if (cmp[i] & 1ull) ++rh;
          else ++ru;
        }
        tie = ru * rh;
      }
    }
    uint32_t D_in, T_in;
    (void)block_exclusive_sum(d_in, sc32, D_in);
    (void)block_exclusive_sum(tie, sc32, T_in);
    if (tid == 0) {
      out.theta = s_out.theta;
      out.n_above = s_out.n_above;
      out.healthy_above = s_out.healthy_above;
      out.discordant = D_cross + D_in;
      out.concordant = C_cross + (HU_mixed - D_in - T_in);
      *dst = out;
    }
    return;
  }

  // ---- 4. fallback: sort every key. Non-candidates become copies of the
  // largest key, so they sort after every candidate; only positions below
  // n_cand are counted. Element e lives in wave e / (KPT*64), slot
  // (e / 64) % KPT, lane e % 64: ranks that follow (wave, slot, lane) order
  // keep every pass stable.
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    uint64_t* q = keys_lds + wave * KPT * 64 + j * 64 + lane;
    if (*q == ~0ull) *q = kmax;
  }
  __syncthreads();
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = pass * 8;
    if (((vary >> shift) & 0xFFull) == 0) continue;  // digit equal in every key
    for (int i = tid; i < 256 * kFitWaves; i += kFitThreads) hist[i] = 0;
    __syncthreads();
    uint32_t pos[(KPT + 1) / 2];  // ranks within the wave's digit bucket, two 16-bit halves each
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint32_t d = (uint32_t)(keys_lds[wave * KPT * 64 + j * 64 + lane] >> shift) & 0xFFu;
      uint64_t peers = ~0ull;
#pragma unroll
      for (int bit = 0; bit < 8; ++bit) {
        const uint64_t bl = __ballot((d >> bit) & 1u);
        peers &= ((d >> bit) & 1u) ? bl : ~bl;
      }
      const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
      uint32_t* h = hist + d * kFitWaves + wave;
      const uint32_t base = *h;
      if (j & 1) pos[j >> 1] |= (base + below) << 16;
      else pos[j >> 1] = base + below;
      // the lowest lane of each digit group advances the wave's count; the
      // loads above complete first (a wave's LDS operations stay in order)
      __builtin_amdgcn_wave_barrier();
      if (below == 0) *h = base + (uint32_t)__popcll(peers);
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    // exclusive offsets in (digit, wave) order: 4 entries per thread
    {
      uint32_t* h4 = hist + tid * 4;
      const uint32_t a0 = h4[0], a1 = h4[1], a2 = h4[2], a3 = h4[3];
      uint32_t tot4;
      const uint32_t base = block_exclusive_sum(a0 + a1 + a2 + a3, sc32, tot4);
      h4[0] = base;
      h4[1] = base + a0;
      h4[2] = base + a0 + a1;
      h4[3] = base + a0 + a1 + a2;
    }
    // every key is read before any is written back
    uint64_t key[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) key[j] = keys_lds[wave * KPT * 64 + j * 64 + lane];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const uint32_t d = (uint32_t)(key[j] >> shift) & 0xFFu;
      keys_lds[hist[d * kFitWaves + wave] + ((pos[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu)] = key[j];
    }
    __syncthreads();
  }
  // keys_lds holds the keys in ascending order; healthy count per wave (a
  // wave's elements are one contiguous block)
  uint32_t hsum = 0, hbits = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const uint32_t e = (uint32_t)(wave * KPT * 64 + j * 64 + lane);
    const uint32_t hbit = (e < n_cand) ? (uint32_t)(keys_lds[e] & 1ull) : 0u;
    hbits |= hbit << j;
    hsum += hbit;
  }
  __syncthreads();
  for (int o = 32; o > 0; o >>= 1) hsum += __shfl_xor(hsum, o);
  if (lane == 0) sc32[wave] = hsum;
  __syncthreads();
  uint32_t wbase = 0;
  for (int w = 0; w < kFitWaves; ++w) wbase += w < wave ? sc32[w] : 0u;
  __syncthreads();
  uint32_t best = kNone, best_h = 0;
  uint32_t run = wbase;  // healthy candidates before the current slot
  // the ordering counts: an unhealthy key pairs with every healthy key
  // before it (all of a smaller S, since in a run of equal S the unhealthy
  // keys come first); the mixed pairs of equal S are counted per run
  uint32_t d_all = 0, tie = 0;
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const uint32_t e = (uint32_t)(wave * KPT * 64 + j * 64 + lane);
    const uint64_t hbal = __ballot((hbits >> j) & 1u);
    const uint32_t before = run + (uint32_t)__popcll(hbal & lt_mask);
    run += (uint32_t)__popcll(hbal);
    if (e < n_cand && !((hbits >> j) & 1u)) d_all += before;
    if (e < n_cand && (e == 0 || (keys_lds[e - 1] >> 1) != (keys_lds[e] >> 1))) {
      const uint32_t N = n_cand - e, H = Ht - before;
      if ((double)H >= rho * (double)N && e < best) {
        best = e;
        best_h = H;
      }
      uint32_t ru = 0, rh = 0;
      for (uint32_t i = e; i < n_cand && (keys_lds[i] >> 1) == (keys_lds[e] >> 1); ++i) {
        if (keys_lds[i] & 1ull) ++rh;
        else ++ru;
      }
      tie += ru * rh;
    }
  }
  const uint32_t g = block_min_u32(best, sc32);
  uint32_t D_all, T_all;
  (void)block_exclusive_sum(d_all, sc32, D_all);
  (void)block_exclusive_sum(tie, sc32, T_all);
  if (g != kNone && best == g) {
    s_out.theta = __longlong_as_double((long long)(keys_lds[g] >> 1));
    s_out.n_above = n_cand - g;
    s_out.healthy_above = best_h;
  }
  __syncthreads();
  if (tid == 0) {
    if (g != kNone) {
      out.theta = s_out.theta;
      out.n_above = s_out.n_above;
      out.healthy_above = s_out.healthy_above;
    }
    if (p.order) {
      out.discordant = D_all;
      out.concordant = Ht * (n_cand - Ht) - D_all - T_all;
    }
    *dst = out;
  }
}

}  // namespace

// --------------------------------------------------------------- host ABI
static uint64_t calib_table_bytes(const tre_events* ev, uint32_t req_cap) {
  return (uint64_t)ev->n_traces * req_cap * 16ull;
}

extern "C" int tre_calib_workspace_size(const tre_events* ev, uint32_t req_cap, size_t* bytes) {
  if (!ev || !bytes) return fail(TRE_EINVAL, "tre_calib_workspace_size: NULL argument");
  *bytes = (size_t)(256 + calib_table_bytes(ev, req_cap));
  return TRE_OK;
}

// the fit of every (trace, model), with the ordering counts when `order`
static int launch_fit(const tre_events* ev, const tre_slo* slo, const double* tss64, const uint8_t* flags,
                      const uint32_t* counts, tre_fit* fit, int order, hipStream_t st) {
  const int M = ev->cfg.n_models;
  const int64_t nW = ev->n_windows;
  FitParams fp{tss64, flags, counts, slo, fit, order, ev->n_traces, M, nW};
  const uint32_t blocks = ((ev->n_traces + 7) / 8) * 8 * (uint32_t)M;
  const int kpt = nW <= 1024 ? 1 : nW <= 2048 ? 2 : nW <= 4096 ? 4 : nW <= 8192 ? 8 : 16;
  LaunchTimer lt(order ? "calib_order" : "calib_fit", st);
  switch (kpt) {
    case 1: hipLaunchKernelGGL(calib_fit<1>, dim3(blocks), dim3(kFitThreads), 0, st, fp); break;
    case 2: hipLaunchKernelGGL(calib_fit<2>, dim3(blocks), dim3(kFitThreads), 0, st, fp); break;
    case 4: hipLaunchKernelGGL(calib_fit<4>, dim3(blocks), dim3(kFitThreads), 0, st, fp); break;
    case 8: hipLaunchKernelGGL(calib_fit<8>, dim3(blocks), dim3(kFitThreads), 0, st, fp); break;
    default: hipLaunchKernelGGL(calib_fit<16>, dim3(blocks), dim3(kFitThreads), 0, st, fp); break;
  }
  lt.done();
  HIP_TRY(hipGetLastError());
  return TRE_OK;
}

extern "C" int tre_calibrate(const tre_events* ev, const tre_slo* slo, const double* tss64,
                             const uint8_t* flags, uint32_t req_cap, uint32_t* counts, tre_fit* fit,
                             tre_req_latency* reqs, uint64_t* n_bad_ids, void* ws, size_t ws_bytes,
                             void* stream) {
  if (!ev || !slo || !tss64 || !flags || !counts || !fit || !ws)
    return fail(TRE_EINVAL, "tre_calibrate: NULL argument");
  if (!ev->req) return fail(TRE_EINVAL, "tre_calibrate: the handle has no request-id column");
  if (req_cap == 0) return fail(TRE_EINVAL, "tre_calibrate: req_cap is 0");
  if (ev->n_windows > (int64_t)kFitThreads * kFitMaxKPT)
    return fail(TRE_ERANGE, "tre_calibrate: %lld windows, at most %d", (long long)ev->n_windows,
                kFitThreads * kFitMaxKPT);
  if (((uintptr_t)counts & 15) || ((uintptr_t)ws & 15))
    return fail(TRE_EINVAL, "tre_calibrate: counts and workspace need 16-byte alignment");
  size_t need = 0;
  tre_calib_workspace_size(ev, req_cap, &need);
  if (ws_bytes < need) return fail(TRE_ENOMEM, "tre_calibrate: workspace %zu < %zu bytes", ws_bytes, need);
  int rc = check_device(ev);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  const int M = ev->cfg.n_models;
  const int64_t nW = ev->n_windows;
  unsigned long long* bad = n_bad_ids ? (unsigned long long*)n_bad_ids : (unsigned long long*)ws;
  uint32_t* tab = (uint32_t*)((char*)ws + 256);
  const uint64_t tab_words = calib_table_bytes(ev, req_cap) / 4;
  const uint64_t cnt_words = (uint64_t)ev->n_traces * M * nW;
  int64_t maxlen = 0;
  for (uint32_t i = 0; i < ev->n_traces; ++i) maxlen = std::max<int64_t>(maxlen, ev->h_off[i + 1] - ev->h_off[i]);
  {
    LaunchTimer lt("calib_fill", st);
    hipLaunchKernelGGL(fill_u32, dim3(4096), dim3(256), 0, st, tab, tab_words, kNone);
    hipLaunchKernelGGL(fill_u32, dim3(4096), dim3(256), 0, st, counts, cnt_words, 0u);
    hipLaunchKernelGGL(fill_u32, dim3(1), dim3(256), 0, st, (uint32_t*)bad, (uint64_t)2, 0u);
    lt.done();
  }
  HIP_TRY(hipGetLastError());
  if (maxlen > 0) {
    const uint32_t C = (uint32_t)((maxlen + kJoinChunk - 1) / kJoinChunk);
    JoinParams jp{ev->ts, ev->model, ev->req, ev->type, ev->tokens, ev->d_off, slo, counts, reqs, tab, bad,
                  ev->n_traces, req_cap, C, M, ev->cfg.window_ms, nW};
    dim3 grid(8u * C * ((ev->n_traces + 7) / 8));
    LaunchTimer lt("calib_join", st);
    hipLaunchKernelGGL(calib_join, grid, dim3(256), 0, st, jp);
    lt.done();
    HIP_TRY(hipGetLastError());
  }
  {
    JudgeParams pp{ev->ts, ev->model, ev->tokens, ev->d_off, tab, slo, counts, reqs,
                   ev->n_traces, req_cap, M, ev->cfg.window_ms, nW};
    dim3 grid((req_cap + 255) / 256, std::min<uint32_t>(ev->n_traces, 65535u));
    LaunchTimer lt("calib_judge", st);
    hipLaunchKernelGGL(calib_judge, grid, dim3(256), 0, st, pp);
    lt.done();
    HIP_TRY(hipGetLastError());
  }
  return launch_fit(ev, slo, tss64, flags, counts, fit, 0, st);
}

extern "C" int tre_calib_order(const tre_events* ev, const tre_slo* slo, const double* tss64, const uint8_t* flags,
                               const uint32_t* counts, tre_fit* fit, void* stream) {
  if (!ev || !slo || !tss64 || !flags || !counts || !fit) return fail(TRE_EINVAL, "tre_calib_order: NULL argument");
  if (ev->n_windows > (int64_t)kFitThreads * kFitMaxKPT)
    return fail(TRE_ERANGE, "tre_calib_order: %lld windows, at most %d", (long long)ev->n_windows,
                kFitThreads * kFitMaxKPT);
  const int rc = check_device(ev);
  if (rc) return rc;
  return launch_fit(ev, slo, tss64, flags, counts, fit, 1, (hipStream_t)stream);
}
