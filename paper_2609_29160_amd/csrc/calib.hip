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
//   fill_u32, fill_unseen  the diagnostic counts and tier lists to zero, the
//                optional per-request records to the unseen pattern.
//   calib_stream one workgroup per trace (first tier: 768 threads of two rows
//                and a 3548-slot table; second tier: 1024 threads of four rows
//                and twice the table, for the traces the first one lists):
//                zeroes the trace's counters, streams its rows in tiles, keeps
//                the requests in flight in an LDS hash table keyed by id
//                (ARRIVE timestamp and model, first DECODE, DECODE tokens
//                after the first), judges each request at its FINISH
//                (latencies, SLO test, one atomic add into the arrival
//                window's packed (judged, ok) counter) and retires its slot;
//                a trace that overflows the table is listed for the next tier.
//   fb_reset, calib_join, calib_judge  the chunked path for the traces the
//                second tier lists: per-chunk LDS combining merged into
//                16-byte id-indexed records with atomics, then one thread per
//                record judges it. It assumes nothing about row order.
//   calib_fit    one 1024-thread workgroup per pair of models of a trace
//                (one load request for both models' TSS and flags of a
//                window), or per (trace, model): candidate keys (S bit
//                pattern, health bit) in LDS, a 2048-bucket histogram
//                that decides most thresholds from bucket counts, a sort of
//                the few undecided keys (bitonic in LDS; an LSD radix sort of
//                all keys beyond 1024), and the ordering counts in its own
//                instantiation.
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
constexpr int kJoinChunk = 8192;    // events per calib_join work item
constexpr int kFitThreads = 1024;   // calib_fit workgroup
constexpr int kFitWaves = kFitThreads / 64;
constexpr int kFitMaxKPT = 16;      // keys per thread: windows up to 16384


template <typename T>
__device__ __forceinline__ T lds_load(const T& x) {
  return __hip_atomic_load(&x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// ------------------------------------------------------------------- fill
__global__ __launch_bounds__(256) void fill_u32(uint32_t* p, uint64_t n, uint32_t v) {
  const uint64_t n4 = n / 4;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint4* q = (uint4*)p;
  const uint4 vv = make_uint4(v, v, v, v);
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) q[i] = vv;
  for (uint64_t i = 4 * n4 + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// request slots that no ARRIVE reaches: model 0xFF, no flags, zero latencies
__global__ __launch_bounds__(256) void fill_unseen(tre_req_latency* r, uint64_t n) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    unsigned long long* w = (unsigned long long*)(r + i);
    w[0] = 0ull;
    w[1] = 0ull;
    w[2] = 0xFFull;
  }
}

// latencies and the SLO test of one judged request from its event times
__device__ __forceinline__ tre_req_latency judge_one(int64_t ta, int64_t tf, int64_t te, uint32_t after_first,
                                                     uint32_t m, double ttft_ms, double tpot_ms, double e2e_ms) {
  tre_req_latency out;
  out.model = (uint8_t)m;
  out.flags = TRE_REQ_ARRIVED | TRE_REQ_COMPLETE;
  for (int i = 0; i < 6; ++i) out.pad[i] = 0;
  const int64_t ttft = tf - ta, e2e = te - ta;
  bool good = (double)ttft <= ttft_ms && (double)e2e <= e2e_ms;
  out.tpot_ms = 0.0;
  if (after_first > 0) {
    const double tpot = (double)(te - tf) / (double)after_first;
    good = good && tpot <= tpot_ms;
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

// ----------------------------------------------------------------- stream
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
typedef unsigned int v2u32 __attribute__((ext_vector_type(2)));

constexpr int kMaxBuckets = 32;        // buckets of one probe run
constexpr int kDeferCap = 256;         // FINISH rows at the last instant of one tile
constexpr uint32_t kTomb = 0xFFFFFFFEu;  // record of a judged request
constexpr unsigned long long kNone64 = ~0ull;
// the two table sizes, in buckets of four records (a prime count, so that
// every probe step reaches every bucket): 887 buckets (two workgroups per
// CU) for every trace, 1789 (one per CU) for the traces that overflow the
// first
constexpr int kBuckets1 = 887, kThreads1 = 768, kRows1 = 2;
constexpr int kBuckets2 = 1789, kThreads2 = 1024, kRows2 = 4;

// murmur3's 32-bit finalizer: request ids are often arithmetic sequences,
// which a multiplicative hash alone maps to correlated buckets
__device__ __forceinline__ uint32_t mix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

struct StreamParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint32_t* req;
  const uint8_t* type;
  const uint16_t* tokens;
  const int64_t* off;
  const tre_slo* slo;            // [n_traces][M]
  uint32_t* counts;              // [n_traces][M][n_windows]: judged << 16 | ok
  tre_req_latency* reqs;         // [n_traces][req_cap] or NULL
  unsigned long long* n_bad;     // events whose id is >= req_cap
  const uint32_t* list_in;       // NULL: workgroup i takes trace i; else [0]: count, [1 + i]: trace
  uint32_t* list_out;            // [0]: traces that overflowed, [1 + i]: their indices
  uint32_t req_cap;
  int32_t M;
  int64_t window_ms;
  int64_t n_windows;             // at most 16384 (checked by tre_calibrate)
  uint32_t magic_w;              // floor(2^32 / window_ms), 2^32 - 1 for a 1 ms window
};

// floor(2^32 / window_ms), clamped to 32 bits
static uint32_t window_magic(int64_t window_ms) {
  const unsigned long long m = (1ull << 32) / (unsigned long long)window_ms;
  return m > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)m;
}

struct StreamRsrc {
  __amdgpu_buffer_rsrc_t ts, model, req, type, tokens;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t col_rsrc(const void* base, long long bytes) {
  const long long n = (bytes + 15) & ~15ll;  // columns stay readable 16 bytes past the last row
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// one thread's kR (2 or 4) consecutive rows of a tile
template <int kR>
struct StreamRows {
  uint32_t req[kR];
  uint32_t ts[kR];  // low words: timestamps lie in [0, duration) below 2^32
  uint32_t ty, mdl;          // one byte per row
  uint32_t tok[kR / 2];      // two 16-bit token counts per word
};

template <int kR>
__device__ __forceinline__ void load_rows(StreamRows<kR>& s, const StreamRsrc& rs, int r0) {
  static_assert(kR == 2 || kR == 4, "two or four rows per thread");
  const v4u32 t0 = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.ts, r0 * 8, 0, 0));
  s.ts[0] = t0.x;
  s.ts[1] = t0.z;
  if constexpr (kR == 4) {
    const v4u32 t1 = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.ts, r0 * 8 + 16, 0, 0));
    const v4u32 q = __builtin_bit_cast(v4u32, __builtin_amdgcn_raw_buffer_load_b128(rs.req, r0 * 4, 0, 0));
    const v2u32 k = __builtin_bit_cast(v2u32, __builtin_amdgcn_raw_buffer_load_b64(rs.tokens, r0 * 2, 0, 0));
    s.ty = __builtin_amdgcn_raw_buffer_load_b32(rs.type, r0, 0, 0);
    s.mdl = __builtin_amdgcn_raw_buffer_load_b32(rs.model, r0, 0, 0);
    s.ts[2] = t1.x;
    s.ts[3] = t1.z;
    s.req[0] = q.x;
    s.req[1] = q.y;
    s.req[2] = q.z;
    s.req[3] = q.w;
    s.tok[0] = k.x;
    s.tok[1] = k.y;
  } else {
    const v2u32 q = __builtin_bit_cast(v2u32, __builtin_amdgcn_raw_buffer_load_b64(rs.req, r0 * 4, 0, 0));
    s.tok[0] = __builtin_amdgcn_raw_buffer_load_b32(rs.tokens, r0 * 2, 0, 0);
    s.ty = __builtin_amdgcn_raw_buffer_load_b16(rs.type, r0, 0, 0);
    s.mdl = __builtin_amdgcn_raw_buffer_load_b16(rs.model, r0, 0, 0);
    s.req[0] = q.x;
    s.req[1] = q.y;
  }
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// One workgroup streams one whole trace in tiles of 4 rows per thread,
// keeping the records of the requests in flight in an LDS hash table keyed
// by request id: kBuckets buckets of four ids, probed by double hashing from
// the id's mixed hash (one 16-byte read per bucket). A record holds the
// ARRIVE's timestamp and model, the first DECODE as a (row << 32 |
// timestamp) minimum, and the DECODE tokens after the first one. Callers
// guarantee that a request has at most one ARRIVE and one FINISH, and no
// ARRIVE or DECODE row at a later timestamp than its FINISH; rows of one
// instant may come in any order, so a FINISH at the last instant of a tile
// is judged after the next tile. Per tile:
//   phase 1  every ARRIVE / DECODE / FINISH row finds or inserts its
//            record, in rounds that each read one bucket and issue one
//            claim (CAS on the bucket's first empty slot) per pending row,
//            then folds its row in: the ARRIVE stores its timestamp and
//            model, a DECODE adds its tokens and offers its key to the
//            first-DECODE minimum;
//   phase 2  the first DECODE takes its own tokens back out of the sum;
//            FINISH rows are queued (or deferred to the next tile);
//   phase 3  the queue is judged, one FINISH per thread (one atomic add on
//            the arrival window's counter), and the slots retired; rows the
//            queue had no room for are judged by their own threads. This
//            overlaps phase 1 of the next tile, which touches other records.
// Retired slots stay occupied until a rebuild re-inserts the live records
// (when more than half the slots are in use). A trace whose table
// overflows (a probe run past kMaxBuckets, more than three quarters of the
// slots live after a rebuild, more than kDeferCap FINISH rows at a tile's
// last instant, an instant longer than a tile) stops and is listed for the
// next tier, which redoes it from scratch.
template <int kBuckets, int kStreamThreads, int kStreamRows>
__global__ __launch_bounds__(kStreamThreads) void calib_stream(StreamParams p) {
  constexpr int kSlots = 4 * kBuckets;
  constexpr int kStreamTile = kStreamThreads * kStreamRows;
  constexpr int kSlotsPerThread = (kSlots + kStreamThreads - 1) / kStreamThreads;
  constexpr uint32_t kRebuildAt = kSlots / 2;      // slots in use (live or retired) that trigger a rebuild
  constexpr uint32_t kMaxLive = 3 * kSlots / 4;    // live records a rebuild may leave
  constexpr uint32_t kQueue = kStreamTile * 3 / 16;  // FINISH rows judged per tile
  // ids; 64 words past the table are per-lane targets for the claims of
  // rows that claim nothing (never the empty marker, so their CAS fails)
  __shared__ __align__(16) uint32_t h_id[kSlots + 64];
  __shared__ unsigned long long h_f[kSlots];  // first DECODE: row << 32 | timestamp
  __shared__ uint32_t h_ta[kSlots];           // ARRIVE timestamp, kNone before it
  __shared__ uint32_t h_d[kSlots];            // DECODE tokens after the first DECODE
  __shared__ uint8_t h_m[kSlots];             // model of the ARRIVE
  // FINISH rows of tile k: queued (slot, timestamp) in s_q, counted in
  // s_nq[k % 2]; those at its last instant deferred (ids) to s_def[k % 3].
  // Each count is reset in the phase 2 before the one that fills it, after
  // the phase 3 that last read it.
  __shared__ uint2 s_q[kQueue];
  __shared__ uint32_t s_def[3][kDeferCap];
  __shared__ uint32_t s_ndef[3], s_nq[2];
  __shared__ uint32_t s_occ, s_over, s_tl;
  const int tid = threadIdx.x, lane = tid & 63;
  if (p.list_in && blockIdx.x >= p.list_in[0]) return;  // whole block
  const uint32_t t = p.list_in ? p.list_in[1 + blockIdx.x] : blockIdx.x;
  const int64_t b = p.off[t], e = p.off[t + 1];
  auto clear_slot = [&](int s) {
    h_id[s] = kNone;
    h_f[s] = kNone64;
    h_ta[s] = kNone;
    h_d[s] = 0u;
    h_m[s] = 0;
  };
  for (int s = tid; s < kSlots; s += kStreamThreads) clear_slot(s);
  if (tid < 64) h_id[kSlots + tid] = 0u;
  if (tid == 0) {
    s_ndef[0] = s_ndef[1] = s_ndef[2] = 0u;
    s_nq[0] = s_nq[1] = 0u;
    s_occ = 0u;
    s_over = 0u;
  }
  if (!p.list_in) {
    // the first tier zeroes its trace's counters (M * n_windows contiguous
    // words; the base is 16-byte aligned, a trace's block need not be),
    // overlapping the other workgroups' streams; a trace handed to a later
    // tier has them zeroed again by that tier's reset. The barrier below
    // orders these stores before every judge's atomic add.
    uint32_t* const c = p.counts + (uint64_t)t * p.M * p.n_windows;
    const uint64_t n = (uint64_t)p.M * (uint64_t)p.n_windows;
    uint64_t head = ((16u - ((uintptr_t)c & 15u)) & 15u) / 4u;
    head = head < n ? head : n;
    const uint64_t n4 = (n - head) / 4u;
    for (uint64_t i = tid; i < head; i += kStreamThreads) c[i] = 0u;
    uint4* const c4 = (uint4*)(c + head);
    for (uint64_t i = tid; i < n4; i += kStreamThreads) c4[i] = make_uint4(0u, 0u, 0u, 0u);
    for (uint64_t i = head + 4u * n4 + tid; i < n; i += kStreamThreads) c[i] = 0u;
  }
  __syncthreads();
  // rows are counted from the trace's first 4-aligned row (below 2^27)
  const long long brow = b & ~3ll;
  const int rend = (int)(e - brow), rfirst = (int)(b - brow);
  StreamRsrc rs;
  rs.ts = col_rsrc(p.ts + brow, (long long)rend * 8);
  rs.model = col_rsrc(p.model + brow, rend);
  rs.req = col_rsrc(p.req + brow, (long long)rend * 4);
  rs.type = col_rsrc(p.type + brow, rend);
  rs.tokens = col_rsrc(p.tokens + brow, (long long)rend * 2);
  uint32_t* cnt = p.counts + (uint64_t)t * p.M * p.n_windows;
  const tre_slo* slo = p.slo + (uint64_t)t * p.M;
  tre_req_latency* rq = p.reqs ? p.reqs + (uint64_t)t * p.req_cap : nullptr;
  const uint32_t M = (uint32_t)p.M;

  // first bucket and probe step (1 .. kBuckets - 1) of an id's mixed hash
  auto home = [](uint32_t h) { return (uint32_t)(((unsigned long long)h * kBuckets) >> 32); };
  auto stride = [](uint32_t h) { return 1u + (((h & 0xFFFFu) * (uint32_t)(kBuckets - 1)) >> 16); };
  auto next = [](uint32_t bk, uint32_t st) { return bk + st >= (uint32_t)kBuckets ? bk + st - kBuckets : bk + st; };
  // a bucket's four ids in one LDS read; a value may be stale by the time
  // it is used, which the claim protocol tolerates: a slot seen empty is
  // claimed by CAS, a slot once taken stays taken (until a rebuild), so an
  // id present lies before every empty slot of its probe order
  auto bucket_ids = [&](uint32_t bk) { return *(const v4u32*)&h_id[4 * bk]; };
  // the lowest of a bucket's four slots holding x, or -1 (the lowest empty
  // one is the one every inserter of an id claims, so that two lanes adding
  // the same id from the same read claim the same slot)
  auto first_of = [](v4u32 v, uint32_t x) {
    return v.x == x ? 0 : v.y == x ? 1 : v.z == x ? 2 : v.w == x ? 3 : -1;
  };
  // the records of up to kN ids (`want` bit u: ids[u] wanted), found or
  // inserted in rounds; slot[u] = -1 when a probe run ends first. Each
  // round reads one bucket and issues one CAS per id, all of them without
  // branches (ids not wanted read and claim harmlessly) so that the reads,
  // and then the CAS, are in flight together.
  auto find_or_insert = [&](auto& ids, auto& slot, uint32_t want, uint32_t& inserted) {
    constexpr int kN = sizeof(slot) / sizeof(slot[0]);
    uint32_t bkt[kN], st[kN], probes[kN];
#pragma unroll
    for (int u = 0; u < kN; ++u) {
      slot[u] = -1;
      const uint32_t h = mix32(ids[u]);
      bkt[u] = home(h);
      st[u] = stride(h);
      probes[u] = 0;
    }
    const uint32_t dummy = (uint32_t)(kSlots + lane);
    while (want) {
      v4u32 v[kN];
      uint32_t claim[kN], old[kN];
#pragma unroll
      for (int u = 0; u < kN; ++u) v[u] = bucket_ids(bkt[u]);
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        const bool w = (want >> u & 1u) != 0;
        const int ie = first_of(v[u], ids[u]), ix = first_of(v[u], kNone);
        const bool found = w && ie >= 0, full = w && ie < 0 && ix < 0;
        claim[u] = (w && ie < 0 && ix >= 0) ? 4 * bkt[u] + (uint32_t)ix : dummy;
        if (found) slot[u] = (int)(4 * bkt[u]) + ie;
        probes[u] += full ? 1u : 0u;
        const bool ended = full && probes[u] >= (uint32_t)kMaxBuckets;  // slot stays -1
        bkt[u] = full ? next(bkt[u], st[u]) : bkt[u];
        want &= (found || ended) ? ~(1u << u) : ~0u;
      }
#pragma unroll
      for (int u = 0; u < kN; ++u) old[u] = atomicCAS(&h_id[claim[u]], kNone, ids[u]);
#pragma unroll
      for (int u = 0; u < kN; ++u) {
        // a lost claim reads its bucket again next round
        const bool won = claim[u] != dummy && (old[u] == kNone || old[u] == ids[u]);
        if (won) slot[u] = (int)claim[u];
        want &= won ? ~(1u << u) : ~0u;
        inserted += (claim[u] != dummy && old[u] == kNone) ? 1u : 0u;
      }
    }
  };
  auto find = [&](uint32_t r) -> int {
    const uint32_t h = mix32(r), st = stride(h);
    uint32_t bk = home(h);
#pragma unroll 1  // kept a loop: unrolled, its exit masks took every SGPR and spilled across the kernel
    for (int q = 0; q < kMaxBuckets; ++q) {
      const v4u32 v = bucket_ids(bk);
      const int ie = first_of(v, r);
      if (ie >= 0) return (int)(4 * bk) + ie;
      if (first_of(v, kNone) >= 0) return -1;
      bk = next(bk, st);
    }
    return -1;
  };
  // judge the request of slot s, finished at te, and retire the slot
  auto judge = [&](int s, uint32_t te) {
    const uint32_t r = h_id[s], ta = h_ta[s];
    if (ta != kNone) {
      const uint32_t m = h_m[s];
      const unsigned long long f = h_f[s];
      tre_req_latency out;
      if (f != kNone64 && m < M) {
        const tre_slo& q = slo[m];
        out = judge_one((int64_t)ta, (int64_t)(uint32_t)f, (int64_t)te, h_d[s], m, q.ttft_ms, q.tpot_ms, q.e2e_ms);
        // window of arrival, ta / window_ms: the multiply-high by magic_w
        // undershoots by at most one (ta < 2^32, window_ms <= 2^23)
        const uint32_t win = (uint32_t)p.window_ms, nw = (uint32_t)p.n_windows;
        uint32_t w = __umulhi(ta, p.magic_w);
        w += ta - w * win >= win ? 1u : 0u;
        if (w < nw) atomicAdd(cnt + m * nw + w, (1u << 16) | ((out.flags & TRE_REQ_OK) ? 1u : 0u));
      } else {
        out = not_judged(m);
      }
      if (rq) rq[r] = out;
    }
    __hip_atomic_store(&h_id[s], kTomb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  auto set_over = [&]() { __hip_atomic_store(&s_over, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP); };

  unsigned bad = 0;
  bool over = false;
  uint32_t tl_prev = 0;
  StreamRows<kStreamRows> cur, nxt;
  if (rend > 0) load_rows(cur, rs, tid * kStreamRows);
  int k = 0;
  for (int tb = 0; tb < rend; tb += kStreamTile, ++k) {
    const bool last = tb + kStreamTile >= rend;
    // the next tile's loads, always issued (rows past the trace read zeros)
    // so that the waits for this tile's rows can count them
    load_rows(nxt, rs, tb + kStreamTile + tid * kStreamRows);
    const int r0 = tb + tid * kStreamRows;
    // the tile's last instant, from the thread holding its last row (read
    // after the next barrier)
    {
      const int lrow = (last ? rend : tb + kStreamTile) - 1;
#pragma unroll
      for (int u = 0; u < kStreamRows; ++u)
        if (r0 + u == lrow) s_tl = cur.ts[u];
    }
    // ---- phase 1
    int slot[kStreamRows];
    uint32_t want = 0, inserted = 0;
#pragma unroll
    for (int u = 0; u < kStreamRows; ++u) {
      const int row = r0 + u;
      const uint32_t kind = (cur.ty >> (8 * u)) & 3u;
      const bool in = row >= rfirst && row < rend;
      if (in && cur.req[u] >= p.req_cap) ++bad;
      if (in && cur.req[u] < p.req_cap && kind != TRE_PREFILL) want |= 1u << u;
    }
    const uint32_t wanted = want;
    find_or_insert(cur.req, slot, want, inserted);
#pragma unroll
    for (int u = 0; u < kStreamRows; ++u) {
      const int s = slot[u];
      if (s < 0) {
        if (wanted >> u & 1u) set_over();
        continue;
      }
      const uint32_t kind = (cur.ty >> (8 * u)) & 3u;
      if (kind == TRE_ARRIVE) {
        h_ta[s] = cur.ts[u];
        h_m[s] = (uint8_t)(cur.mdl >> (8 * u));
      } else if (kind == TRE_DECODE) {
        atomicAdd(&h_d[s], (cur.tok[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
        atomicMin(&h_f[s], ((unsigned long long)(uint32_t)(r0 + u) << 32) | cur.ts[u]);
      }
    }
    if (inserted) atomicAdd(&s_occ, inserted);  // no return: nothing waits on it
    __syncthreads();
    // ---- phase 2 (the flags are settled: nothing writes them before the
    // next barrier)
    const uint32_t occ = lds_load(s_occ), tl = lds_load(s_tl);
    if (lds_load(s_over)) {
      over = true;
      break;
    }
    const int kd = k % 3;
    uint32_t own = 0;  // FINISH rows the queue had no room for
    if (tid == 0) {
      s_ndef[(k + 1) % 3] = 0u;
      s_nq[(k + 1) & 1] = 0u;
    }
    uint32_t fin = 0, dfr = 0;  // FINISH rows to queue, to defer
    unsigned long long hf[kStreamRows];
#pragma unroll
    for (int u = 0; u < kStreamRows; ++u) hf[u] = slot[u] >= 0 ? h_f[slot[u]] : 0ull;
#pragma unroll
    for (int u = 0; u < kStreamRows; ++u) {
      const int s = slot[u];
      const uint32_t kind = (cur.ty >> (8 * u)) & 3u;
      if (s >= 0 && kind == TRE_DECODE && (uint32_t)(hf[u] >> 32) == (uint32_t)(r0 + u))
        atomicSub(&h_d[s], (cur.tok[u >> 1] >> (16 * (u & 1))) & 0xFFFFu);
      const bool f = s >= 0 && kind == TRE_FINISH;
      const bool d = f && !last && cur.ts[u] == tl;
      fin |= (f && !d) ? 1u << u : 0u;
      dfr |= d ? 1u << u : 0u;
    }
    if (dfr) {
#pragma unroll
      for (int u = 0; u < kStreamRows; ++u) {
        if (!(dfr >> u & 1u)) continue;
        const uint32_t i = atomicAdd(&s_ndef[kd], 1u);
        if (i < (uint32_t)kDeferCap) s_def[kd][i] = cur.req[u];
        else set_over();
      }
    }
    // queue the others: one LDS atomic per wave for its four row positions
    {
      unsigned long long mq[kStreamRows];
      uint32_t wtot = 0;
#pragma unroll
      for (int u = 0; u < kStreamRows; ++u) {
        mq[u] = __ballot((fin >> u & 1u) != 0);
        wtot += (uint32_t)__popcll(mq[u]);
      }
      if (wtot) {
        uint32_t base = 0;
        if (lane == 0) base = atomicAdd(&s_nq[k & 1], wtot);
        base = __builtin_amdgcn_readfirstlane(base);
        const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
        for (int u = 0; u < kStreamRows; ++u) {
          if (fin >> u & 1u) {
            const uint32_t i = base + (uint32_t)__popcll(mq[u] & below);
            if (i < kQueue) s_q[i] = make_uint2((uint32_t)slot[u], cur.ts[u]);
            else own |= 1u << u;
          }
          base += (uint32_t)__popcll(mq[u]);
        }
      }
    }
    __syncthreads();
    // ---- phase 3: the queue, then the previous tile's deferred FINISH rows
    // once their instant has ended (this tile reaches a later one, or the
    // trace ends)
    {
      const uint32_t n = lds_load(s_nq[k & 1]), nq = n < kQueue ? n : kQueue;
      for (uint32_t i = tid; i < nq; i += kStreamThreads) {
        const uint2 q = s_q[i];
        judge((int)q.x, q.y);
      }
      if (own) {
#pragma unroll
        for (int u = 0; u < kStreamRows; ++u)
          if (own >> u & 1u) judge(slot[u], cur.ts[u]);
      }
    }
    if (k > 0) {
      const int kp = (k + 2) % 3;  // tile k - 1
      const uint32_t nd = s_ndef[kp];
      if (nd > 0u) {
        if (tl > tl_prev || last) {
          for (uint32_t i = tid; i < nd; i += kStreamThreads) {
            const int s = find(s_def[kp][i]);
            if (s >= 0) judge(s, tl_prev);
          }
        } else if (tid == 0) {
          s_over = 1u;  // one instant longer than a tile
        }
      }
    }
    if (occ > kRebuildAt) {
      // ---- rebuild: re-insert the live records into a cleared table
      __syncthreads();
      uint32_t rid[kSlotsPerThread], rta[kSlotsPerThread], rd[kSlotsPerThread];
      unsigned long long rf[kSlotsPerThread];
      uint8_t rm[kSlotsPerThread];
      uint32_t live = 0;
#pragma unroll
      for (int j = 0; j < kSlotsPerThread; ++j) {
        const int s = tid + j * kStreamThreads;
        rid[j] = kTomb;
        if (s >= kSlots) continue;
        rid[j] = h_id[s];
        rta[j] = h_ta[s];
        rf[j] = h_f[s];
        rd[j] = h_d[s];
        rm[j] = h_m[s];
        if (rid[j] < kTomb) live |= 1u << j;
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < kSlotsPerThread; ++j)
        if (tid + j * kStreamThreads < kSlots) clear_slot(tid + j * kStreamThreads);
      if (tid == 0) s_occ = 0u;
      __syncthreads();
      uint32_t again = 0;
#pragma unroll
      for (int j = 0; j < kSlotsPerThread; ++j) {
        // one record at a time keeps the registers of the saved ones few
        uint32_t id1[1] = {rid[j]};
        int s1[1];
        find_or_insert(id1, s1, live >> j & 1u, again);
        if (!(live >> j & 1u)) continue;
        const int s = s1[0];
        if (s < 0) {
          set_over();
          continue;
        }
        h_ta[s] = rta[j];
        h_f[s] = rf[j];
        h_d[s] = rd[j];
        h_m[s] = rm[j];
      }
      if (again) atomicAdd(&s_occ, again);
      __syncthreads();
      if (tid == 0 && lds_load(s_occ) > kMaxLive) s_over = 1u;
    }
    tl_prev = tl;
    cur = nxt;
  }
  if (over) {
    // the next tier redoes the whole trace (its counters, request slots and
    // ids out of range included)
    if (tid == 0) {
      const uint32_t i = atomicAdd(p.list_out, 1u);
      p.list_out[1 + i] = t;
    }
    return;
  }
  __syncthreads();
  // requests still in flight at the end: arrived, not judged
  if (rq) {
    for (int s = tid; s < kSlots; s += kStreamThreads) {
      const uint32_t r = h_id[s];
      if (r < kTomb && h_ta[s] != kNone) rq[r] = not_judged(h_m[s]);
    }
  }
  bad = wave_sum(bad);
  if (lane == 0 && bad) atomicAdd(p.n_bad, (unsigned long long)bad);
}

// --------------------------------------------------------------- fallback
// The traces both stream tiers handed over, redone by request-id records in
// the workspace: fb_reset clears their counters, request slots and (for the
// chunked path) records;
// calib_join combines each chunk's events per request in LDS and merges them
// into the 16-byte records with atomics (minimum ARRIVE / DECODE / FINISH
// rows, complemented DECODE token sum); calib_judge judges every record.
// This path takes the definition literally and assumes nothing about where
// a request's rows lie.
struct FallbackParams {
  const int64_t* ts;
  const uint8_t* model;
  const uint32_t* req;
  const uint8_t* type;
  const uint16_t* tokens;
  const int64_t* off;
  const tre_slo* slo;           // [n_traces][M]
  uint32_t* counts;             // [n_traces][M][n_windows]: judged << 16 | ok
  tre_req_latency* reqs;        // [n_traces][req_cap] or NULL
  uint32_t* tab;                // [n_traces][req_cap][4]: a, f, e, ~dsum, or NULL (fb_reset only)
  unsigned long long* n_bad;    // events whose id is >= req_cap
  const uint32_t* fb;           // [0]: listed traces, [1 + i]: their indices
  uint32_t req_cap;
  uint32_t n_chunks;            // chunks of the longest trace
  int32_t M;
  int64_t window_ms;
  int64_t n_windows;
};

__global__ __launch_bounds__(256) void fb_reset(FallbackParams p) {
  const uint32_t n_list = p.fb[0];
  const uint64_t cw = (uint64_t)p.M * p.n_windows, tw = (uint64_t)p.req_cap * 4;
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint32_t pos = blockIdx.y; pos < n_list; pos += gridDim.y) {
    const uint32_t t = p.fb[1 + pos];
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < cw; i += stride)
      p.counts[(uint64_t)t * cw + i] = 0u;
    if (p.tab)
      for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < tw; i += stride)
        p.tab[(uint64_t)t * tw + i] = kNone;
    if (p.reqs) {
      for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < p.req_cap; i += stride) {
        unsigned long long* w = (unsigned long long*)(p.reqs + (uint64_t)t * p.req_cap + i);
        w[0] = 0ull;
        w[1] = 0ull;
        w[2] = 0xFFull;
      }
    }
  }
}

constexpr int kHashSlots = 2048;           // LDS records per chunk (load factor about 0.4)
constexpr int kProbes = 16;                // linear probes before the global fallback
constexpr int kJoinBatch = 8;              // events per thread loaded together

// Work items (listed trace, chunk of kJoinChunk rows), one per workgroup at
// a time.
__global__ __launch_bounds__(256) void calib_join(FallbackParams p) {
  __shared__ uint32_t h_id[kHashSlots], h_a[kHashSlots], h_f[kHashSlots], h_e[kHashSlots], h_d[kHashSlots];
  const uint64_t items = (uint64_t)p.fb[0] * p.n_chunks;
  unsigned bad = 0;
  for (uint64_t it = blockIdx.x; it < items; it += gridDim.x) {
    const uint32_t t = p.fb[1 + it / p.n_chunks], chunk = (uint32_t)(it % p.n_chunks);
    const int64_t b = p.off[t], e = p.off[t + 1];
    const int64_t c0 = b + (int64_t)chunk * kJoinChunk;
    if (c0 >= e) continue;  // whole block
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
      if (h_a[s] != kNone) atomicMin(rec, h_a[s]);
      if (h_f[s] != kNone) {
        atomicMin(rec + 1, h_f[s]);
        atomicSub(rec + 3, h_d[s]);
      }
      if (h_e[s] != kNone) atomicMin(rec + 2, h_e[s]);
    }
    __syncthreads();
  }
  // one atomic per wave for the ids out of range
  bad = wave_sum(bad);
  if ((threadIdx.x & 63) == 0 && bad) atomicAdd(p.n_bad, (unsigned long long)bad);
}

// One thread per (listed trace, request slot).
__global__ __launch_bounds__(256) void calib_judge(FallbackParams p) {
  const uint64_t items = (uint64_t)p.fb[0] * p.req_cap;
  for (uint64_t it = (uint64_t)blockIdx.x * 256 + threadIdx.x; it < items; it += (uint64_t)gridDim.x * 256) {
    const uint32_t t = p.fb[1 + it / p.req_cap], r = (uint32_t)(it % p.req_cap);
    const uint64_t slot = (uint64_t)t * p.req_cap + r;
    const uint4 rec = ((const uint4*)p.tab)[slot];
    if (rec.x == kNone) continue;  // no ARRIVE: the reset left the slot unseen
    const int64_t b = p.off[t];
    const uint32_t m = p.model[b + rec.x];
    tre_req_latency out = not_judged(m);
    if (rec.y != kNone && rec.z != kNone && m < (uint32_t)p.M) {
      const tre_slo& q = p.slo[(uint64_t)t * p.M + m];
      const int64_t ta = p.ts[b + rec.x];
      out = judge_one(ta, p.ts[b + rec.y], p.ts[b + rec.z], ~rec.w - (uint32_t)p.tokens[b + rec.y], m, q.ttft_ms,
                      q.tpot_ms, q.e2e_ms);
      const int64_t w = ta / p.window_ms;  // window of arrival
      if (w >= 0 && w < p.n_windows)
        atomicAdd(p.counts + ((uint64_t)t * p.M + m) * p.n_windows + w,
                  (1u << 16) | ((out.flags & TRE_REQ_OK) ? 1u : 0u));
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
  int32_t order;                // also the ordering counts (tre_calib_order): calib_fit<KPT, true>
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

// One 1024-thread workgroup per (trace, model), or (kPair) per two models
// fitted one after the other. Candidate keys
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
// kOrder: also the ordering counts (tre_calib_order); the instantiation
// without them carries none of their registers.
template <int KPT, bool kOrder, bool kPair>
__global__ __launch_bounds__(kFitThreads) void calib_fit(FitParams p) {
  static_assert(!(kPair && kOrder), "the ordering counts take one model per workgroup");
  __shared__ uint64_t keys_lds[kFitThreads * KPT];
  __shared__ uint32_t hist[2 * kBuckets];  // buckets: counts then (G, P), compact offsets; radix: [digit][wave]
  __shared__ uint64_t cmp[kResolveCap];
  __shared__ uint64_t sc64[kFitWaves];
  __shared__ uint32_t sc32[kFitWaves + 1];
  __shared__ uint32_t n_gathered;
  __shared__ uint32_t hpre_s[kFitThreads];  // healthy keys before each gathered position
  __shared__ uint32_t red_n[2][kFitWaves];  // per model of the pair
  __shared__ uint64_t red_k[2][2][kFitWaves];  // max, min
  __shared__ uint32_t red_o[kFitWaves];     // waves whose pair of key runs met
  __shared__ uint64_t s_kmin;               // smallest key of bucket b* when nothing is gathered
  __shared__ tre_fit s_out;
  static_assert(256 * kFitWaves == 2 * kBuckets, "radix histogram and bucket tables share LDS");

  // XCD-aware block order: consecutive blocks go to different XCDs, so the
  // models of one trace are numbered to land on one XCD and share its L2
  // for the strided per-cell reads. kPair: models m, m + 1 (M even), whose
  // TSS and flags lie side by side, so one load request serves both
  const uint32_t b = blockIdx.x;
  const uint32_t xcd = b & 7u, k = b >> 3;
  const uint32_t per = kPair ? (uint32_t)p.M / 2u : (uint32_t)p.M;
  const uint32_t t = (k / per) * 8u + xcd;
  const uint32_t m = (k % per) * (kPair ? 2u : 1u);
  if (t >= p.n_traces) return;  // whole block
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tid = threadIdx.x;
  const int64_t nW = p.n_windows;

  // candidate keys to LDS, each wave's packed from the front of its KPT * 64
  // slots in element order (kPair: the second model's from the back). Three
  // rounds of loads, each issued for a batch of the thread's windows before
  // any is waited on: the packed counts, the flags of the windows that judged
  // a request, the TSS of the candidates. A load a lane skips gets an offset
  // past its buffer, which reads zero and costs no cache-line request: the
  // flags and TSS of one model lie M and 8M bytes apart, one line per window,
  // and the per-CU line-request rate, not HBM, bounds this phase (a round that
  // skips no lane is slower than the extra round trip).
  constexpr uint32_t kSkip = 0x80000000u;  // past every buffer below (nW * M * 8 < 2^31)
  constexpr int kCap = KPT * 64;           // key slots per wave
  const uint32_t Mu = (uint32_t)p.M;
  const uint64_t tbase = (uint64_t)t * nW * Mu;
  const __amdgpu_buffer_rsrc_t r_fl =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.flags + tbase), (short)0, (int)(nW * Mu), 0x00020000);
  const __amdgpu_buffer_rsrc_t r_s =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<double*>(p.tss64 + tbase), (short)0, (int)(nW * Mu * 8), 0x00020000);
  auto cnt_rsrc = [&](uint32_t mm) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(p.counts + ((uint64_t)t * p.M + mm) * nW), (short)0,
                                             (int)(nW * 4), 0x00020000);
  };
  // a window's code: 0 (no candidate) or 2 | healthy
  auto code_of = [&](uint32_t c, uint32_t fl, const tre_slo& sl) {
    const uint32_t judged = c >> 16, ok = c & 0xFFFFu;
    const bool cand = judged > 0 && (fl & TRE_FLAG_INIT) && !(fl & TRE_FLAG_IDLE);
    const bool healthy = (double)ok >= sl.attain_q * (double)judged;
    return cand ? (2u | (healthy ? 1u : 0u)) : 0u;
  };
  const uint64_t lt = (1ull << lane) - 1ull;
  uint64_t* const R = keys_lds + wave * kCap;  // this wave's slots
  struct Sum {  // a lane's keys: count, healthy count, min, max
    uint32_t n = 0, h = 0;
    uint64_t kmin = ~0ull, kmax = 0;
    __device__ void add(uint64_t kk) {
      kmin = kk < kmin ? kk : kmin;
      kmax = kk > kmax ? kk : kmax;
      ++n;
      h += (uint32_t)(kk & 1ull);
    }
  };
  constexpr int kLB = KPT < 8 ? KPT : 8;  // windows per batch of the three rounds
  // one model's keys from the front of the wave's slots; returns their count
  auto load_one = [&](uint32_t mm, Sum& su) {
    // the lane index made opaque, so that the second model's reload derives
    // its offsets afresh instead of keeping the pair loads' ones live (in
    // scratch) across the first model's fit
    int ln = lane;
    __asm__ volatile("" : "+v"(ln));
    const uint64_t lt1 = (1ull << ln) - 1ull;
    const tre_slo sl = p.slo[(uint64_t)t * p.M + mm];
    const __amdgpu_buffer_rsrc_t r_cnt = cnt_rsrc(mm);
    int f = 0;
#pragma unroll
    for (int j0 = 0; j0 < KPT; j0 += kLB) {
      uint32_t code[kLB], fl[kLB];
#pragma unroll
      for (int j = 0; j < kLB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + ln);
        code[j] = __builtin_amdgcn_raw_buffer_load_b32(r_cnt, (int64_t)w < nW ? w * 4u : kSkip, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kLB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + ln);
        fl[j] = __builtin_amdgcn_raw_buffer_load_b8(r_fl, (code[j] >> 16) ? w * Mu + mm : kSkip, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kLB; ++j) code[j] = code_of(code[j], fl[j], sl);
      uint64_t sb[kLB];
#pragma unroll
      for (int j = 0; j < kLB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + ln);
        sb[j] = __builtin_bit_cast(uint64_t,
                                   __builtin_amdgcn_raw_buffer_load_b64(r_s, code[j] ? (w * Mu + mm) * 8u : kSkip, 0, 0));
      }
#pragma unroll
      for (int j = 0; j < kLB; ++j) {
        const uint64_t bal = __ballot(code[j] != 0u);
        if (code[j]) {
          const uint64_t kk = (sb[j] << 1) | (code[j] & 1u);
          R[f + __popcll(bal & lt1)] = kk;
          su.add(kk);
        }
        f += __popcll(bal);
      }
    }
    return f;
  };
  // hist is first used after the reduction's barrier below
  for (int i = tid; i < kBuckets; i += kFitThreads) hist[i] = 0;
  if (tid == 0) s_kmin = ~0ull;
  Sum su0, su1;
  int n0 = 0, n1 = 0;  // the wave's key counts (the second model's at the back)
  if constexpr (!kPair) {
    n0 = load_one(m, su0);
  } else {
    // both models: counts from two rows, flags as 2 bytes, TSS as 16 bytes;
    // the second model's keys go to the back of the wave's slots while they
    // stay above the first model's (a wave where the two runs meet reloads
    // the second model after the first one's fit)
    const tre_slo sl0 = p.slo[(uint64_t)t * p.M + m], sl1 = p.slo[(uint64_t)t * p.M + m + 1];
    const __amdgpu_buffer_rsrc_t r_c0 = cnt_rsrc(m), r_c1 = cnt_rsrc(m + 1);
    constexpr int kPB = KPT < 8 ? KPT : 8;  // windows per batch
#pragma unroll
    for (int j0 = 0; j0 < KPT; j0 += kPB) {
      uint32_t c0[kPB], c1[kPB], fl[kPB];
#pragma unroll
      for (int j = 0; j < kPB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + lane);
        const uint32_t off = (int64_t)w < nW ? w * 4u : kSkip;
        c0[j] = __builtin_amdgcn_raw_buffer_load_b32(r_c0, off, 0, 0);
        c1[j] = __builtin_amdgcn_raw_buffer_load_b32(r_c1, off, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kPB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + lane);
        fl[j] = __builtin_amdgcn_raw_buffer_load_b16(r_fl, ((c0[j] | c1[j]) >> 16) ? w * Mu + m : kSkip, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kPB; ++j)  // the two codes, 2 bits each
        c0[j] = code_of(c0[j], fl[j] & 0xFFu, sl0) | (code_of(c1[j], fl[j] >> 8, sl1) << 2);
      __attribute__((ext_vector_type(4))) uint32_t v[kPB];
#pragma unroll
      for (int j = 0; j < kPB; ++j) {
        const uint32_t w = (uint32_t)(wave * kCap + (j0 + j) * 64 + lane);
        v[j] = __builtin_amdgcn_raw_buffer_load_b128(r_s, c0[j] ? (w * Mu + m) * 8u : kSkip, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < kPB; ++j) {
        const uint32_t q0 = c0[j] & 3u, q1 = c0[j] >> 2;
        const uint64_t bal0 = __ballot(q0 != 0u), bal1 = __ballot(q1 != 0u);
        if (q0) {
          const uint64_t kk = ((((uint64_t)v[j][1] << 32) | v[j][0]) << 1) | (q0 & 1u);
          R[n0 + __popcll(bal0 & lt)] = kk;
          su0.add(kk);
        }
        n0 += __popcll(bal0);
        if (q1) {
          const uint64_t kk = ((((uint64_t)v[j][3] << 32) | v[j][2]) << 1) | (q1 & 1u);
          const int q = kCap - 1 - (n1 + __popcll(bal1 & lt));
          if (q >= n0) R[q] = kk;
          su1.add(kk);
        }
        n1 += __popcll(bal1);
      }
    }
  }
  // one workgroup reduction of each model's candidate and healthy counts
  // (packed n << 16 | h, both at most 16384) and its smallest and largest key
  auto reduce = [&](Sum& su, int q) {
    uint32_t nh = (su.n << 16) | su.h;
    for (int o = 32; o > 0; o >>= 1) {
      nh += (uint32_t)__shfl_xor((int)nh, o);
      const uint64_t a = shfl_xor_u64(su.kmax, o);
      su.kmax = a > su.kmax ? a : su.kmax;
      const uint64_t b = shfl_xor_u64(su.kmin, o);
      su.kmin = b < su.kmin ? b : su.kmin;
    }
    if (lane == 0) {
      red_n[q][wave] = nh;
      red_k[q][0][wave] = su.kmax;
      red_k[q][1][wave] = su.kmin;
    }
  };
  auto gather = [&](Sum& su, int q) {
    uint32_t nh = 0;
    su.kmax = 0;
    su.kmin = ~0ull;
    for (int v = 0; v < kFitWaves; ++v) {
      nh += red_n[q][v];
      su.kmax = red_k[q][0][v] > su.kmax ? red_k[q][0][v] : su.kmax;
      su.kmin = red_k[q][1][v] < su.kmin ? red_k[q][1][v] : su.kmin;
    }
    su.n = nh >> 16;
    su.h = nh & 0xFFFFu;
  };
  reduce(su0, 0);
  if constexpr (kPair) {
    reduce(su1, 1);
    if (lane == 0) red_o[wave] = n0 + n1 > kCap ? 1u : 0u;
  }
  __syncthreads();
  gather(su0, 0);
  // the fit of one model from this wave's keys R[roff .. roff + nk) and the
  // workgroup's summary su, written to dst; true when it sorted every slot
  // (the radix fallback), which overwrites the other model's keys
  auto fit_one = [&](const int roff, const int nk, const Sum& su, const tre_slo& s, tre_fit* const dst) -> bool {
    const double rho = s.reliability;
    const uint32_t n_cand = su.n, Ht = su.h;
    const uint64_t kmax = su.kmax;
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
      return false;
    }
    // the highest bit above bit 0 where keys differ: where the smallest and
    // the largest differ (every key shares their common prefix)
    const uint64_t vary_s = (kmax ^ su.kmin) & ~1ull;
    if (vary_s == 0) {  // one value of S: a single run covering every candidate
      if (tid == 0) {
        if ((double)Ht >= rho * (double)n_cand) {
          out.theta = __longlong_as_double((long long)(kmax >> 1));
          out.n_above = n_cand;
          out.healthy_above = Ht;
        }
        *dst = out;
      }
      return false;
    }

    // ---- 1. histogram over buckets, packed (healthy << 16) | count
    const int hb = 63 - __clzll((long long)vary_s);
    const int lo = hb >= 11 ? hb - 10 : 1;
    auto bucket = [&](uint64_t key) { return (uint32_t)(key >> lo) & (uint32_t)(kBuckets - 1); };
    for (int e = lane; e < nk; e += 64) {
      const uint64_t kk = R[roff + e];
      atomicAdd(&hist[bucket(kk)], ((uint32_t)(kk & 1ull) << 16) | 1u);
    }
    __syncthreads();
    // two buckets per thread; counts and healthy counts stay below 2^16
    const uint32_t v0 = hist[2 * tid], v1 = hist[2 * tid + 1];
    uint32_t tot;
    const uint32_t ex = block_exclusive_sum(v0 + v1, sc32, tot);
    const uint32_t offs[2] = {ex, ex + v0}, cnts[2] = {v0, v1};
    // each bucket's (G, P) replaces its count (read above by this thread
    // only): read back from LDS where needed, so that no register holds it
    // across the scans below
    hist[2 * tid] = offs[0];
    hist[2 * tid + 1] = offs[1];
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
    if constexpr (kOrder) {
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
    if (mtot == 0 && !kOrder) {  // uniform: no bucket below b* can hold the answer
      if (bstar != kNone) {        // b*'s first position: its smallest key
        uint64_t kb = ~0ull;
        for (int e = lane; e < nk; e += 64) {
          const uint64_t kk = R[roff + e];
          if (bucket(kk) == bstar) kb = kk < kb ? kk : kb;
        }
        for (int o = 32; o > 0; o >>= 1) {
          const uint64_t a = shfl_xor_u64(kb, o);
          kb = a < kb ? a : kb;
        }
        if (lane == 0 && kb != ~0ull) atomicMin(&s_kmin, (unsigned long long)kb);
        __syncthreads();
        if (tid == 0) {
          const uint32_t GP = hist[bstar];
          out.theta = __longlong_as_double((long long)(s_kmin >> 1));
          out.n_above = n_cand - (GP & 0xFFFFu);
          out.healthy_above = Ht - (GP >> 16);
          *dst = out;
        }
      } else if (tid == 0) {
        *dst = out;
      }
      return false;
    }
    // the keys of the listed buckets (bit 31 of their hist[kBuckets + b] entry),
    // gathered into cmp at their compact offsets and sorted (bitonic); returns
    // with every thread holding cmp[tid] (or ~0) in `ck`
    auto gather_sort = [&](uint32_t n_keys, uint64_t& ck) {
      if (tid == 0) n_gathered = 0;
      __syncthreads();
      for (int e = lane; e < nk; e += 64) {
        const uint64_t kk = R[roff + e];
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
    if (mtot <= (uint32_t)kResolveCap && (!kOrder || mx_tot <= (uint32_t)kResolveCap)) {
      // per bucket: (G, P) (written above) and the compact offset with bit 31
      // marking a gathered bucket
      hist[kBuckets + 2 * tid] = mex | (mc[0] ? 0x80000000u : 0u);
      hist[kBuckets + 2 * tid + 1] = (mex + mc[0]) | (mc[1] ? 0x80000000u : 0u);
      uint64_t kstar = ~0ull;  // smallest key of bucket b*
      for (int e = lane; e < nk; e += 64) {
        const uint64_t kk = R[roff + e];
        if (bucket(kk) == bstar) kstar = kk < kstar ? kk : kstar;
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
      __syncthreads();  // s_out written by one thread, read by thread 0
      if constexpr (!kOrder) {
        if (tid == 0) {
          out.theta = s_out.theta;
          out.n_above = s_out.n_above;
          out.healthy_above = s_out.healthy_above;
          *dst = out;
        }
        return false;
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
      return false;
    }

    // ---- 4. fallback: sort every slot. The slots that hold no key of this
    // model become copies of the largest key, so they sort after every
    // candidate; only positions below n_cand are counted. Element e lives in
    // wave e / (KPT*64), slot (e / 64) % KPT, lane e % 64: ranks that follow
    // (wave, slot, lane) order keep every pass stable. Digits equal in every
    // key are skipped.
    uint64_t k_or = 0, k_and = ~0ull;
    for (int e = lane; e < nk; e += 64) {
      const uint64_t kk = R[roff + e];
      k_or |= kk;
      k_and &= kk;
    }
    const uint64_t vary = block_reduce_u64<0>(k_or, sc64) ^ block_reduce_u64<1>(k_and, sc64);
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
      const int e = j * 64 + lane;
      if (e < roff || e >= roff + nk) R[e] = kmax;
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
      if constexpr (kOrder) {
        out.discordant = D_all;
        out.concordant = Ht * (n_cand - Ht) - D_all - T_all;
      }
      *dst = out;
    }
    return true;
  };
  const bool sorted_all = fit_one(0, n0, su0, p.slo[(uint64_t)t * p.M + m], p.fit + (uint64_t)t * p.M + m);
  if constexpr (kPair) {
    // the second model: its keys where the runs never met and the first fit
    // left every slot in place; else loaded again on its own
    bool met = sorted_all;
    for (int v = 0; v < kFitWaves; ++v) met = met || red_o[v] != 0u;
    int roff = kCap - n1;
    __syncthreads();  // the first fit's last reads of the keys and tables
    for (int i = tid; i < kBuckets; i += kFitThreads) hist[i] = 0;
    if (tid == 0) s_kmin = ~0ull;
    if (met) {
      Sum su;
      n1 = load_one(m + 1, su);
      roff = 0;
      reduce(su, 1);
    }
    __syncthreads();
    Sum su1w;
    gather(su1w, 1);
    (void)fit_one(roff, n1, su1w, p.slo[(uint64_t)t * p.M + m + 1], p.fit + (uint64_t)t * p.M + m + 1);
  } else {
    (void)sorted_all;
  }
}

}  // namespace

// --------------------------------------------------------------- host ABI
// workspace: the id-out-of-range count (8 bytes, when the caller passes no
// counter) in a 256-byte header, the fallback list (count, then trace
// indices) rounded up to 256 bytes, then the fallback's request records
static uint64_t calib_list_bytes(const tre_events* ev) { return ((4ull + 4ull * ev->n_traces) + 255) & ~255ull; }
// two lists: the traces the first stream tier hands to the second, and those
// the second hands to the chunked path

static uint64_t calib_table_bytes(const tre_events* ev, uint32_t req_cap) {
  return (uint64_t)ev->n_traces * req_cap * 16ull;
}

extern "C" int tre_calib_workspace_size(const tre_events* ev, uint32_t req_cap, size_t* bytes) {
  if (!ev || !bytes) return fail(TRE_EINVAL, "tre_calib_workspace_size: NULL argument");
  *bytes = (size_t)(256 + 2 * calib_list_bytes(ev) + calib_table_bytes(ev, req_cap));
  return TRE_OK;
}

// the fit of every (trace, model), with the ordering counts when `order`
static int launch_fit(const tre_events* ev, const tre_slo* slo, const double* tss64, const uint8_t* flags,
                      const uint32_t* counts, tre_fit* fit, int order, hipStream_t st) {
  const int M = ev->cfg.n_models;
  const int64_t nW = ev->n_windows;
  FitParams fp{tss64, flags, counts, slo, fit, order, ev->n_traces, M, nW};
  // models in pairs (one load request for both models' TSS and flags) when
  // their pairs' TSS are 16-byte aligned and their flags 2-byte aligned
  const bool pair = !order && M % 2 == 0 && ((uintptr_t)tss64 & 15) == 0 && ((uintptr_t)flags & 1) == 0;
  const uint32_t blocks = ((ev->n_traces + 7) / 8) * 8 * (uint32_t)(pair ? M / 2 : M);
  const int kpt = nW <= 1024 ? 1 : nW <= 2048 ? 2 : nW <= 4096 ? 4 : nW <= 8192 ? 8 : 16;
  LaunchTimer lt(order ? "calib_order" : "calib_fit", st);
  auto go = [&](auto kernel) { hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kFitThreads), 0, st, fp); };
  switch (kpt * 4 + (order ? 1 : 0) + (pair ? 2 : 0)) {
    case 4: go(calib_fit<1, false, false>); break;
    case 5: go(calib_fit<1, true, false>); break;
    case 6: go(calib_fit<1, false, true>); break;
    case 8: go(calib_fit<2, false, false>); break;
    case 9: go(calib_fit<2, true, false>); break;
    case 10: go(calib_fit<2, false, true>); break;
    case 16: go(calib_fit<4, false, false>); break;
    case 17: go(calib_fit<4, true, false>); break;
    case 18: go(calib_fit<4, false, true>); break;
    case 32: go(calib_fit<8, false, false>); break;
    case 33: go(calib_fit<8, true, false>); break;
    case 34: go(calib_fit<8, false, true>); break;
    case 64: go(calib_fit<16, false, false>); break;
    case 65: go(calib_fit<16, true, false>); break;
    default: go(calib_fit<16, false, true>); break;
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
  if (req_cap > (1u << 31)) return fail(TRE_ERANGE, "tre_calibrate: req_cap %u is above 2^31", req_cap);
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
  uint32_t* l1 = (uint32_t*)((char*)ws + 256);
  uint32_t* l2 = (uint32_t*)((char*)ws + 256 + calib_list_bytes(ev));
  uint32_t* tab = (uint32_t*)((char*)ws + 256 + 2 * calib_list_bytes(ev));
  int64_t maxlen = 0;
  for (uint32_t i = 0; i < ev->n_traces; ++i) maxlen = std::max<int64_t>(maxlen, ev->h_off[i + 1] - ev->h_off[i]);
  {
    LaunchTimer lt("calib_fill", st);
    hipLaunchKernelGGL(fill_u32, dim3(1), dim3(256), 0, st, (uint32_t*)bad, (uint64_t)2, 0u);
    hipLaunchKernelGGL(fill_u32, dim3(1), dim3(256), 0, st, l1, (uint64_t)1, 0u);
    hipLaunchKernelGGL(fill_u32, dim3(1), dim3(256), 0, st, l2, (uint64_t)1, 0u);
    if (reqs)
      hipLaunchKernelGGL(fill_unseen, dim3(4096), dim3(256), 0, st, reqs, (uint64_t)ev->n_traces * req_cap);
    lt.done();
  }
  HIP_TRY(hipGetLastError());
  if (ev->n_traces > 0) {
    StreamParams sp{ev->ts, ev->model, ev->req, ev->type, ev->tokens, ev->d_off, slo, counts, reqs, bad,
                    nullptr, l1, req_cap, M, ev->cfg.window_ms, nW, window_magic(ev->cfg.window_ms)};
    LaunchTimer lt("calib_stream", st);
    hipLaunchKernelGGL((calib_stream<kBuckets1, kThreads1, kRows1>), dim3(ev->n_traces), dim3(kThreads1), 0, st, sp);
    lt.done();
    HIP_TRY(hipGetLastError());
  }
  if (maxlen > 0) {
    // the traces the first tier listed, then those the second listed (none
    // on most inputs: the launches then end at once)
    const uint32_t C = (uint32_t)((maxlen + kJoinChunk - 1) / kJoinChunk);
    FallbackParams f1{ev->ts, ev->model, ev->req, ev->type, ev->tokens, ev->d_off, slo, counts, reqs, nullptr, bad,
                      l1, req_cap, C, M, ev->cfg.window_ms, nW};
    FallbackParams f2 = f1;
    f2.tab = tab;
    f2.fb = l2;
    StreamParams sp{ev->ts, ev->model, ev->req, ev->type, ev->tokens, ev->d_off, slo, counts, reqs, bad,
                    l1, l2, req_cap, M, ev->cfg.window_ms, nW, window_magic(ev->cfg.window_ms)};
    LaunchTimer lt("calib_fallback", st);
    hipLaunchKernelGGL(fb_reset, dim3(64, 16), dim3(256), 0, st, f1);
    hipLaunchKernelGGL((calib_stream<kBuckets2, kThreads2, kRows2>), dim3(ev->n_traces), dim3(kThreads2), 0, st, sp);
    hipLaunchKernelGGL(fb_reset, dim3(64, 16), dim3(256), 0, st, f2);
    hipLaunchKernelGGL(calib_join, dim3(1024), dim3(256), 0, st, f2);
    hipLaunchKernelGGL(calib_judge, dim3(1024), dim3(256), 0, st, f2);
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
