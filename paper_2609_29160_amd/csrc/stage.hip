// stage.hip - stage-aware service shares on MI355X (gfx950): per model and
// window, one smoothed share for the prefill stage and one for the decode
// stage, from the window tallies that tre_eval_tss writes.
//
// Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE), Sections
// "Discussion" and "Future Work": for disaggregated prefill / decode pools
// the scalar score becomes a vector estimating each stage's service deficit
// separately. No formula is given; the shares here are Eq. (1)'s two parts,
// each with the one-request floor:
//   prefill  raw_p = 1000 * w_p * P / max(w_q * W_int, window_ms)
//   decode   raw_d = 1000 * D / max(A_int, window_ms)
// (where neither floor binds, Eq. (1)'s ratio is their mediant). A stage is
// idle when its tokens and its demand integral are both zero: its smoothed
// value holds; the first busy window initialises it; later ones smooth with
// the model's alpha (Section "Smoothing, Normalization, and Calibration").
//
// Kernel
//   stage_tss  one thread per (trace, model), windows in order (the
//              smoothing is a sequential recurrence with a fixed rounding
//              order); threads of consecutive models read consecutive
//              tallies of a window, so each load and store is coalesced
//              across a trace's models; four windows' tallies are loaded
//              ahead. HBM-bound: 24 bytes read and up to 17 written per cell.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "tre.h"
#include "tre_internal.h"

#pragma clang fp contract(off)

using tre_internal::check_device;
using tre_internal::fail;
using tre_internal::LaunchTimer;

namespace {

constexpr int kAhead = 4;  // windows of tallies loaded ahead

struct StageParams {
  const tre_profile* prof;
  const uint32_t* prefill;
  const uint32_t* decode;
  const int64_t* a_int;
  const int64_t* w_int;
  double* stage64;
  float* stage32;
  uint8_t* flags;
  uint64_t n_series;  // n_traces * n_models
  int64_t n_windows;
  int32_t M;
  double window;
};

__global__ __launch_bounds__(256) void stage_tss(StageParams p) {
  const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= p.n_series) return;
  const uint64_t trace = i / (uint64_t)p.M;
  const int m = (int)(i - trace * (uint64_t)p.M);
  const tre_profile pr = p.prof[i];
  const double oma = 1.0 - pr.alpha;
  const int64_t nW = p.n_windows;
  const uint64_t c0 = trace * (uint64_t)nW * p.M + m;  // cell of window 0
  double sp = 0.0, sd = 0.0;
  bool ip = false, id = false;
  for (int64_t w0 = 0; w0 < nW; w0 += kAhead) {
    uint32_t P[kAhead], D[kAhead];
    int64_t Ai[kAhead], Wi[kAhead];
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      const bool in = w0 + u < nW;
      const uint64_t c = c0 + (uint64_t)(in ? w0 + u : 0) * p.M;
      P[u] = in ? p.prefill[c] : 0u;
      D[u] = in ? p.decode[c] : 0u;
      Ai[u] = in ? p.a_int[c] : 0;
      Wi[u] = in ? p.w_int[c] : 0;
    }
#pragma unroll
    for (int u = 0; u < kAhead; ++u) {
      if (w0 + u >= nW) break;
      const uint64_t c = c0 + (uint64_t)(w0 + u) * p.M;
      const bool p_idle = P[u] == 0u && Wi[u] == 0;
      const bool d_idle = D[u] == 0u && Ai[u] == 0;
      if (!p_idle) {
        double num = pr.w_p * (double)P[u];
        num = num * 1000.0;
        double den = pr.w_q * (double)Wi[u];
        if (den < p.window) den = p.window;
        const double raw = num / den;
        if (ip) {
          const double t1 = pr.alpha * raw;
          const double t2 = oma * sp;
          sp = t1 + t2;
        } else {
          sp = raw;
          ip = true;
        }
      }
      if (!d_idle) {
        double num = (double)D[u] * 1000.0;
        double den = (double)Ai[u];
        if (den < p.window) den = p.window;
        const double raw = num / den;
        if (id) {
          const double t1 = pr.alpha * raw;
          const double t2 = oma * sd;
          sd = t1 + t2;
        } else {
          sd = raw;
          id = true;
        }
      }
      if (p.stage64) *(double2*)(p.stage64 + 2 * c) = make_double2(sp, sd);
      if (p.stage32) *(float2*)(p.stage32 + 2 * c) = make_float2((float)sp, (float)sd);
      if (p.flags)
        p.flags[c] = (uint8_t)((p_idle ? TRE_STAGE_P_IDLE : 0) | (ip ? TRE_STAGE_P_INIT : 0) |
                               (d_idle ? TRE_STAGE_D_IDLE : 0) | (id ? TRE_STAGE_D_INIT : 0));
    }
  }
}

}  // namespace

extern "C" int tre_stage_tss(const tre_events* ev, const tre_profile* prof, const tre_tss_out* tallies,
                             double* stage64, float* stage32, uint8_t* flags, void* stream) {
  if (!ev || !prof || !tallies) return fail(TRE_EINVAL, "tre_stage_tss: NULL handle, profiles or tallies");
  if (!tallies->prefill || !tallies->decode || !tallies->a_int || !tallies->w_int)
    return fail(TRE_EINVAL, "tre_stage_tss: the prefill, decode, a_int and w_int tallies are all needed");
  if (!stage64 && !stage32 && !flags) return fail(TRE_EINVAL, "tre_stage_tss: no output");
  if (((uintptr_t)stage64 & 15) || ((uintptr_t)stage32 & 7))
    return fail(TRE_EINVAL, "tre_stage_tss: stage64 needs 16-byte, stage32 8-byte alignment");
  int rc = check_device(ev);
  if (rc) return rc;
  const uint64_t n = (uint64_t)ev->n_traces * ev->cfg.n_models;
  if (n == 0 || ev->n_windows == 0) return TRE_OK;
  StageParams p{};
  p.prof = prof;
  p.prefill = tallies->prefill;
  p.decode = tallies->decode;
  p.a_int = tallies->a_int;
  p.w_int = tallies->w_int;
  p.stage64 = stage64;
  p.stage32 = stage32;
  p.flags = flags;
  p.n_series = n;
  p.n_windows = ev->n_windows;
  p.M = ev->cfg.n_models;
  p.window = (double)ev->cfg.window_ms;
  hipStream_t st = (hipStream_t)stream;
  LaunchTimer lt("stage_tss", st);
  hipLaunchKernelGGL(stage_tss, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p);
  lt.done();
  HIP_TRY(hipGetLastError());
  return TRE_OK;
}
