// Calls between the library's own source files (not part of the C ABI).
#pragma once

#include <cstdint>

#include "trackfit.h"

// The encoder's front end alone ((x, y, z) embedding or the Fourier front end)
// for a handle with no layers: row (hit row - offsets[0]) of x0 [rows][d]
// receives the hit's d values in the 16-bit operand type of the handle's
// mode (fp32 for TF_FP32).  Asynchronous; rows of rejected tracks are not
// written.
tf_status tf_internal_front_end(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                const tf_weights *w, void *x0, long long rows, hipStream_t stream);
