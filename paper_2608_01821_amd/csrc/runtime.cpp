// Library runtime: thread-local error strings, version, and the optional
// per-kernel-class event timing used by the measurement harness.

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "common.h"

namespace davet {

static thread_local std::string g_last_error;

int set_error(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

static const char* kClassNames[KC_COUNT] = {
    "views",      "view_maps", "assemble_norm", "rmsnorm",    "gemm_qkv",
    "rope",       "attention", "gemm_o",        "gemm_gateup", "gemm_down",
    "head_prep",  "head_gemm", "head_merge",    "unmask",     "gemm_f32",
    "attention_f32", "misc", "realizer_keys", "realizer_maps"};

const char* kernel_class_name(int c) {
  return (c >= 0 && c < KC_COUNT) ? kClassNames[c] : "";
}

// Profiling state: a fixed pool of event pairs created by davet_prof_enable.
// Single-threaded use; launches past the pool size are not timed.
struct Prof {
  bool on = false;
  int used = 0;
  int only = -1;        // record only this class (-1: every class)
  std::vector<hipEvent_t> start, stop;
  std::vector<int> cls;
};
static Prof g_prof;

ProfScope::ProfScope(int c, hipStream_t s) : slot(-1), stream(s) {
  if (!g_prof.on || g_prof.used >= (int)g_prof.start.size()) return;
  if (g_prof.only >= 0 && c != g_prof.only) return;
  slot = g_prof.used++;
  g_prof.cls[slot] = c;
  if (hipEventRecord(g_prof.start[slot], s) != hipSuccess) slot = -1;
}

ProfScope::~ProfScope() {
  if (slot >= 0) (void)hipEventRecord(g_prof.stop[slot], stream);
}

static void prof_release() {
  for (auto e : g_prof.start) (void)hipEventDestroy(e);
  for (auto e : g_prof.stop) (void)hipEventDestroy(e);
  g_prof.start.clear();
  g_prof.stop.clear();
  g_prof.cls.clear();
  g_prof.used = 0;
  g_prof.on = false;
}

}  // namespace davet

extern "C" const char* davet_last_error(void) {
  return davet::g_last_error.c_str();
}

extern "C" const char* davet_version(void) { return "davet-mi355x 0.1 (gfx950)"; }

extern "C" int davet_prof_enable(int32_t max_launches) {
  using namespace davet;
  prof_release();
  if (max_launches <= 0) return DAVET_OK;
  g_prof.start.resize(max_launches);
  g_prof.stop.resize(max_launches);
  g_prof.cls.assign(max_launches, -1);
  for (int i = 0; i < max_launches; ++i) {
    if (hipEventCreate(&g_prof.start[i]) != hipSuccess ||
        hipEventCreate(&g_prof.stop[i]) != hipSuccess) {
      g_prof.start.resize(i);
      g_prof.stop.resize(i);
      prof_release();
      return set_error(DAVET_EHIP, "davet_prof_enable: hipEventCreate failed");
    }
  }
  g_prof.on = true;
  return DAVET_OK;
}

extern "C" int davet_prof_reset(void) {
  davet::g_prof.used = 0;
  return DAVET_OK;
}

extern "C" int davet_prof_only(int32_t cls) {
  using namespace davet;
  DAVET_CHECK_ARG(cls >= -1 && cls < KC_COUNT, DAVET_EINVAL,
                  "davet_prof_only: class out of range");
  g_prof.only = cls;
  return DAVET_OK;
}

extern "C" int davet_prof_read(int32_t n_classes, int64_t* counts,
                               double* total_ms) {
  using namespace davet;
  DAVET_CHECK_ARG(counts && total_ms && n_classes >= 0, DAVET_EINVAL,
                  "davet_prof_read: null output");
  const int n = n_classes < KC_COUNT ? n_classes : KC_COUNT;
  for (int c = 0; c < n; ++c) { counts[c] = 0; total_ms[c] = 0.0; }
  for (int i = 0; i < g_prof.used; ++i) {
    DAVET_HIP(hipEventSynchronize(g_prof.stop[i]));
    float ms = 0.f;
    DAVET_HIP(hipEventElapsedTime(&ms, g_prof.start[i], g_prof.stop[i]));
    const int c = g_prof.cls[i];
    if (c >= 0 && c < n) { counts[c] += 1; total_ms[c] += ms; }
  }
  return KC_COUNT;
}

extern "C" const char* davet_prof_class_name(int32_t cls) {
  return davet::kernel_class_name(cls);
}
