// Host-side helpers shared by the device entry points: shape validation and
// HIP launch-status mapping.  Nothing here runs on the GPU.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "dasc.h"

namespace dasc {

inline bool valid_shape(const dasc_shape* s) {
  if (!s) return false;
  if (s->arch != DASC_ARCH_KDA && s->arch != DASC_ARCH_GDN) return false;
  if (s->n_layers <= 0 || s->n_heads <= 0 || s->n_qk_heads <= 0 || s->dk <= 0 || s->dv <= 0)
    return false;
  if (s->n_heads % s->n_qk_heads != 0) return false;
  const int64_t rows = int64_t(s->n_layers) * s->n_heads * s->dk;
  return rows < (int64_t(1) << 31);
}

inline int64_t rows_per_state(const dasc_shape* s) {
  return int64_t(s->n_layers) * s->n_heads * s->dk;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Map the launch status of the kernel just enqueued to a DASC status code.
inline int launch_status() {
  return hipGetLastError() == hipSuccess ? DASC_OK : DASC_E_HIP;
}

}  // namespace dasc
