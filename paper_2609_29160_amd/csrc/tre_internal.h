// tre_internal.h - definitions shared by the library's source files (the
// events handle, error reporting, launch timing). Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <stdint.h>

#include <vector>

#include "tre.h"

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

namespace tre_internal {

// records the message for tre_last_error and returns `code`
int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// TRE_OK when the handle belongs to the current device
int check_device(const tre_events* ev);

// HIP events recorded around one launch on its stream while timing is on
// (tre_set_timing); tre_kernel_time collects them by kernel name
class LaunchTimer {
 public:
  LaunchTimer(const char* name, hipStream_t s);
  void done();

 private:
  const char* name_ = nullptr;
  hipEvent_t start_ = nullptr, stop_ = nullptr;
  hipStream_t st_;
  bool on_ = false;
};

// while one exists on this thread, LaunchTimer records nothing (calls that
// must not create runtime objects)
struct NoTimingScope {
  NoTimingScope();
  ~NoTimingScope();
};

}  // namespace tre_internal

#define HIP_TRY(expr)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess)                                                                      \
      return tre_internal::fail(TRE_EHIP, "%s: %s", #expr, hipGetErrorString(e_));             \
  } while (0)
