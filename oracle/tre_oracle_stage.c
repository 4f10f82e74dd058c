/*
 * tre_oracle_stage.c - CPU oracle for the stage-aware service shares: one
 * smoothed share for the prefill stage and one for the decode stage per
 * model and window, from the window tallies of the base oracle.
 *
 * TEST INFRASTRUCTURE ONLY, like tre_oracle.c: linked by the tests, the
 * smoke check and the benchmark's CPU-baseline leg, never by the product
 * path, and sharing no code with the GPU library.
 *
 * Paper: "Cross-Model Autoscaling for Shared LLM Serving" (TRE), Section
 * "Discussion" and "Future Work": for disaggregated prefill / decode pools
 * the scalar score becomes a stage-specific vector estimating prefill and
 * decode service deficits separately. The paper gives no formula; the
 * reading used here (listed in the design notes) splits Eq. (1) into its
 * two stages:
 *   prefill: weighted prefill token rate over the weighted waiting demand,
 *            raw_p = 1000 * w_p * P / max(w_q * W_int, window_ms);
 *   decode:  decode token rate over the active demand,
 *            raw_d = 1000 * D / max(A_int, window_ms);
 * each with the one-request floor of Eq. (1). Wherever neither floor
 * binds, Eq. (1)'s raw ratio is the mediant of the two:
 *   raw = (num_p + num_d) / (den_p + den_d).
 * A stage is idle in a window when its tokens and its demand integral are
 * both zero; idle holds the smoothed value, the first non-idle window
 * initialises it to the raw ratio, later ones smooth with the model's alpha
 * (Section "Smoothing, Normalization, and Calibration").
 *
 * Floating point: IEEE binary64, round to nearest even, no contraction, in
 * the operation order written below.
 */
#include <stdint.h>

#define OS_MAX_MODELS 256
#define OS_P_IDLE 1
#define OS_P_INIT 2
#define OS_D_IDLE 4
#define OS_D_INIT 8

typedef struct {
  double w_p, w_q, alpha, theta, tau_crit, tau_surplus;
  int32_t r_min, r_init;
} os_profile;

/* raw prefill-stage share of one window */
double oracle_stage_raw_prefill(double w_p, double w_q, int64_t P, int64_t W_int, int64_t window_ms) {
  double num = w_p * (double)P;
  num = num * 1000.0;
  double den = w_q * (double)W_int;
  if (den < (double)window_ms) den = (double)window_ms;
  return num / den;
}

/* raw decode-stage share of one window */
double oracle_stage_raw_decode(int64_t D, int64_t A_int, int64_t window_ms) {
  double num = (double)D * 1000.0;
  double den = (double)A_int;
  if (den < (double)window_ms) den = (double)window_ms;
  return num / den;
}

/*
 * Per-window tallies [n_windows][M] (prefill tokens P, decode tokens D,
 * integrals A_int, W_int in request*ms) -> smoothed shares S [n_windows][M][2]
 * (prefill, decode) and flags [n_windows][M] (OS_* bits). Returns 0, or -1
 * for bad shapes.
 */
int oracle_stage_tss(int64_t n_windows, int32_t M, int64_t window_ms, const os_profile* prof, const int64_t* P,
                     const int64_t* D, const int64_t* A_int, const int64_t* W_int, double* S, uint8_t* flags) {
  if (n_windows < 0 || M < 1 || M > OS_MAX_MODELS || window_ms <= 0) return -1;
  for (int m = 0; m < M; ++m) {
    double sp = 0.0, sd = 0.0;
    int ip = 0, id = 0;
    for (int64_t w = 0; w < n_windows; ++w) {
      const int64_t c = w * M + m;
      const int p_idle = P[c] == 0 && W_int[c] == 0;
      const int d_idle = D[c] == 0 && A_int[c] == 0;
      if (!p_idle) {
        const double raw = oracle_stage_raw_prefill(prof[m].w_p, prof[m].w_q, P[c], W_int[c], window_ms);
        if (ip) {
          const double t1 = prof[m].alpha * raw;
          const double t2 = (1.0 - prof[m].alpha) * sp;
          sp = t1 + t2;
        } else {
          sp = raw;
          ip = 1;
        }
      }
      if (!d_idle) {
        const double raw = oracle_stage_raw_decode(D[c], A_int[c], window_ms);
        if (id) {
          const double t1 = prof[m].alpha * raw;
          const double t2 = (1.0 - prof[m].alpha) * sd;
          sd = t1 + t2;
        } else {
          sd = raw;
          id = 1;
        }
      }
      S[2 * c] = sp;
      S[2 * c + 1] = sd;
      flags[c] = (uint8_t)((p_idle ? OS_P_IDLE : 0) | (ip ? OS_P_INIT : 0) | (d_idle ? OS_D_IDLE : 0) |
                           (id ? OS_D_INIT : 0));
    }
  }
  return 0;
}
