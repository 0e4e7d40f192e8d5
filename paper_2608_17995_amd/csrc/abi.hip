// Error state, version and launch timing of the C ABI.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "common.h"

namespace avits {

static thread_local char g_last_error[512] = "";

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

// Status of the launches just enqueued by this thread.
int launch_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return set_error(AVITS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return AVITS_OK;
}

// ---------------------------------------------------------------------------
// Launch timing: when enabled, every internal launch is bracketed by a pair of
// HIP events on its stream; avits_timing_read() waits for them and adds the
// elapsed times to per-family totals.  Single-threaded use only.
static const char* const kFamilies[] = {"score_spatial", "score_combine", "score_finalize", "select",
                                        "gather_upsample", "scatter", "ln_mod", "gemm_qkv", "gemm_o",
                                        "gemm_mlp_in", "gemm_mlp_out", "gemm_single_in", "gemm_single_out",
                                        "splitk_reduce", "qk_rope", "attention", "joint_lse",
                                        "gather_mixed", "scatter_mixed", "linear", "final_linear", "euler", "noise"};
constexpr int kNumFamilies = sizeof(kFamilies) / sizeof(kFamilies[0]);

struct Pending {
  hipEvent_t start, stop;
  int family;
};
static bool g_timing = false;
static std::vector<Pending> g_pending;
static std::vector<hipEvent_t> g_free_events;
static double g_ms[kNumFamilies];
static int64_t g_launches[kNumFamilies];

static int family_index(const char* name) {
  for (int i = 0; i < kNumFamilies; ++i)
    if (strcmp(kFamilies[i], name) == 0) return i;
  return -1;
}

static hipEvent_t take_event() {
  if (!g_free_events.empty()) {
    hipEvent_t e = g_free_events.back();
    g_free_events.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

TimedLaunch::TimedLaunch(const char* family, hipStream_t stream) : family_(-1), stream_(stream) {
  if (!g_timing) return;
  family_ = family_index(family);
  if (family_ < 0) return;
  start_ = take_event();
  if (start_ && hipEventRecord(start_, stream_) != hipSuccess) family_ = -1;
}

TimedLaunch::~TimedLaunch() {
  if (family_ < 0 || !start_) return;
  hipEvent_t stop = take_event();
  if (!stop || hipEventRecord(stop, stream_) != hipSuccess) return;
  g_pending.push_back({start_, stop, family_});
}

static void drain() {
  for (const Pending& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.stop) == hipSuccess && hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
      g_ms[p.family] += ms;
      g_launches[p.family] += 1;
    }
    g_free_events.push_back(p.start);
    g_free_events.push_back(p.stop);
  }
  g_pending.clear();
}

}  // namespace avits

extern "C" int avits_timing_enable(int on) {
  avits::g_timing = on != 0;
  return AVITS_OK;
}

extern "C" void avits_timing_reset(void) {
  avits::drain();
  for (int i = 0; i < avits::kNumFamilies; ++i) {
    avits::g_ms[i] = 0.0;
    avits::g_launches[i] = 0;
  }
}

extern "C" int avits_timing_read(const char* family, double* total_ms, int64_t* launches) {
  // "gemm" sums every GEMM family.
  const bool all_gemm = family && strcmp(family, "gemm") == 0;
  const int f = family && !all_gemm ? avits::family_index(family) : -1;
  if (f < 0 && !all_gemm)
    return avits::set_error(AVITS_ERR_INVALID_ARG, "timing_read: unknown launch family '%s'",
                            family ? family : "(null)");
  avits::drain();
  double ms = 0.0;
  int64_t n = 0;
  for (int i = 0; i < avits::kNumFamilies; ++i) {
    if (all_gemm ? strncmp(avits::kFamilies[i], "gemm_", 5) == 0 : i == f) {
      ms += avits::g_ms[i];
      n += avits::g_launches[i];
    }
  }
  if (total_ms) *total_ms = ms;
  if (launches) *launches = n;
  return AVITS_OK;
}

extern "C" const char* avits_version(void) { return "0.1.0"; }

extern "C" const char* avits_last_error(void) { return avits::g_last_error; }
