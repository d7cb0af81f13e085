// Host-side argument checks shared by the entry points of the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "resbm.h"

namespace resbm_host {

inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Byte extent of a rows x cols matrix with row stride ld (elements of es bytes).
inline size_t extent(int64_t rows, int64_t cols, int64_t ld, size_t es) {
  return rows > 0 ? (size_t)(((rows - 1) * ld + cols) * (int64_t)es) : 0;
}

// Whether [a, a + na) and [b, b + nb) intersect (NULL or empty ranges never do).
inline bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + nb && pb < pa + na;
}

// A leading dimension of a matrix with n used columns: ld >= n, ld % 8 == 0.
inline bool ld_ok(int64_t ld, int n) { return ld >= n && ld % 8 == 0; }

// RESBM_E_HIP if a launch since the last call failed.
inline int32_t launch_status() { return hipGetLastError() == hipSuccess ? RESBM_OK : RESBM_E_HIP; }

}  // namespace resbm_host
