// Launchers of the HIP kernels, called by the executor.
#pragma once

#include <hip/hip_runtime.h>

#include "plan.h"

namespace ce {

// Generic strided pairwise step (any kind in K_GENERIC_*).
hipError_t launch_generic(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s);

// Specialised kernels (every other kind).
hipError_t launch_fast(const Launch& ln, const void* a, const void* b, void* c, void* d,
                       hipStream_t s);

// General contraction (K_TC main launch: a = A, b = B, c = C, d = partials;
// K_TC_REDUCE: d = partials, c = C).
hipError_t launch_tc(const Launch& ln, const void* a, const void* b, void* c, void* d, hipStream_t s);

// Fused CP chain forward: ops = {X, Us, Kh, Kw, Ut}.
hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s);

// Fused CP chain backward: ops = {X, dY, dX (may be NULL), Us, Kh, Kw, Ut,
// Pus, Put, Pkh, Pkw}.
hipError_t launch_cp_bwd(const Launch& ln, const void* const* ops, hipStream_t s);

}  // namespace ce
