// Per-launch timing of the orchestration's kernels: when enabled, ggnn_forward
// and ggnn_backward bracket each kernel launch they enqueue with a pair of HIP
// events on the launch's stream, so a caller can read the device time of
// every launch of a real pass (not of a relaunch in isolation).
#include <hip/hip_runtime.h>

#include <vector>

#include "common.h"
#include "profile.h"

namespace ggnn {
namespace {

struct Record {
  hipEvent_t start = nullptr, stop = nullptr;
  int id = -1;
};

// Process-wide state, driven by one host thread (see ggnn.h).
struct State {
  std::vector<Record> recs;
  int used = 0;
  bool on = false;
  int open = -1;   // record whose start event was placed, awaiting its stop
} g_prof;

const char* const kNames[PROF_COUNT] = {
    "step_fwd",        "step_fwd_gru",  "gru_fwd",        "transform_fwd", "banded_fwd",
    "gru_rev",         "step_rev",      "step_rev_gru",   "banded_rev",    "transform_rev_dx",
    "wgrad_gru",       "wgrad_transform", "reduce",      "super_record",  "super"};

void release() {
  for (Record& r : g_prof.recs) {
    if (r.start) (void)hipEventDestroy(r.start);
    if (r.stop) (void)hipEventDestroy(r.stop);
  }
  g_prof.recs.clear();
  g_prof.used = 0;
  g_prof.open = -1;
  g_prof.on = false;
}

}  // namespace

void prof_begin(hipStream_t s) {
  g_prof.open = -1;
  if (!g_prof.on || g_prof.used >= (int)g_prof.recs.size()) return;
  // Events recorded while the stream is being captured into a HIP graph would
  // become graph nodes: such launches are not timed.
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
  Record& r = g_prof.recs[g_prof.used];
  if (hipEventRecord(r.start, s) != hipSuccess) return;
  g_prof.open = g_prof.used;
}

void prof_end(hipStream_t s, int id) {
  if (g_prof.open < 0) return;
  Record& r = g_prof.recs[g_prof.open];
  g_prof.open = -1;
  if (hipEventRecord(r.stop, s) != hipSuccess) return;
  r.id = id;
  ++g_prof.used;
}

}  // namespace ggnn

using namespace ggnn;

extern "C" {

ggnn_status ggnn_profile_start(int32_t capacity) {
  clear_error();
  GGNN_CHECK_ARG(capacity >= 0 && capacity <= (1 << 20), "capacity=%d must be in [0, 2^20]", capacity);
  release();
  if (capacity == 0) return GGNN_OK;
  g_prof.recs.resize(capacity);
  for (Record& r : g_prof.recs) {
    if (hipEventCreate(&r.start) != hipSuccess || hipEventCreate(&r.stop) != hipSuccess) {
      release();
      return fail(GGNN_ERR_DEVICE, "profile_start: hipEventCreate failed");
    }
  }
  g_prof.on = true;
  return GGNN_OK;
}

ggnn_status ggnn_profile_stop(void) {
  clear_error();
  g_prof.on = false;
  g_prof.open = -1;
  return GGNN_OK;
}

int32_t ggnn_profile_count(void) { return g_prof.used; }

ggnn_status ggnn_profile_read(int32_t i, int32_t* id, float* ms) {
  clear_error();
  GGNN_CHECK_ARG(i >= 0 && i < g_prof.used, "record %d out of range [0, %d)", i, g_prof.used);
  GGNN_CHECK_ARG(id != nullptr && ms != nullptr, "id and ms must not be NULL");
  const Record& r = g_prof.recs[i];
  hipError_t e = hipEventSynchronize(r.stop);
  if (e == hipSuccess) e = hipEventElapsedTime(ms, r.start, r.stop);
  if (e != hipSuccess) return fail(GGNN_ERR_DEVICE, "profile_read: %s", hipGetErrorString(e));
  *id = r.id;
  return GGNN_OK;
}

const char* ggnn_profile_name(int32_t id) { return id >= 0 && id < PROF_COUNT ? kNames[id] : ""; }

}  // extern "C"
