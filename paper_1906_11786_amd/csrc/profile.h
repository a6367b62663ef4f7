// Internal side of the launch profiler (ggnn_profile_* in ggnn.h): the
// orchestration brackets each kernel launch with prof_begin / prof_end.
#pragma once

#include <hip/hip_runtime.h>

namespace ggnn {

// Launch kinds, in the order of ggnn_profile_name().
enum ProfId {
  PROF_STEP_FWD = 0,      // band step forward, propagation only (1-bit band)
  PROF_STEP_FWD_GRU,      // band step forward with the GRU fused (1-bit band)
  PROF_GRU_FWD,           // GRU update kernel
  PROF_TRANSFORM_FWD,     // message transform (dense band)
  PROF_BANDED_FWD,        // banded product (dense band)
  PROF_GRU_REV,           // GRU node reverse kernel
  PROF_STEP_REV,          // band step reverse, propagation and dX only (1-bit band)
  PROF_STEP_REV_GRU,      // band step reverse with the previous step's GRU reverse fused (1-bit band)
  PROF_BANDED_REV,        // banded reverse product (dense band)
  PROF_TRANSFORM_REV_DX,  // dX of the message transform (dense band)
  PROF_WGRAD_GRU,         // GRU weight-gradient contraction
  PROF_WGRAD_TRANSFORM,   // message-transform weight-gradient contraction
  PROF_REDUCE,            // fixed-order reduction of weight-gradient partials
  PROF_SUPER_RECORD,      // supernode rows' record of a fused supernode step (gather, or long contraction + sum)
  PROF_SUPER,             // stand-alone supernode slice kernels (forward or reverse share of one step)
  PROF_COUNT
};

// Place the start event of the next record on s (no-op unless profiling is
// on, records are left and s is not capturing).
void prof_begin(hipStream_t s);
// Close the record opened by the last prof_begin with its stop event.
void prof_end(hipStream_t s, int id);

}  // namespace ggnn
