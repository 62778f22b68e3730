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

// Up to four ordered partial sums (K_REDUCE_MULTI, MultiReduceDesc): parts[j]
// the fp32 partials, outs[j] the fp32 output (null: skipped).
hipError_t launch_reduce_multi(const Launch& ln, const void* const* parts, void* const* outs, hipStream_t s);

// Small-output contraction over a long reduction (K_THINW / K_THINW_REDUCE,
// ThinwDesc): p, q = the operands, part = fp32 partials, c = the output.
hipError_t launch_thinw(const Launch& ln, const void* p, const void* q, void* part, void* c, hipStream_t s);

// Plane convolution contracted over one index (K_CRED / K_CREDW, CredDesc):
// z = the stacked planes, o = the filter (K_CRED) or the output gradient
// (K_CREDW), y = the output plane (K_CRED) or the fp32 partials (K_CREDW).
// Convolution contracted over one channel index (K_CCONV, CconvDesc): z = the
// input planes, f = the filter, y = the output planes (bf16 or fp32).
hipError_t launch_cconv(const Launch& ln, const void* z, const void* f, void* y, hipStream_t s);
hipError_t launch_cred(const Launch& ln, const void* z, const void* o, void* y, hipStream_t s);
// Its filter gradient on fp32 MFMA tiles (K_WGCONV): z = the stacked planes,
// o = the output gradient, part = the fp32 partials (summed by K_CREDW_REDUCE).
hipError_t launch_wgconv(const Launch& ln, const void* z, const void* o, void* part, hipStream_t s);

// Both gradients of a channel-mixing step (K_GPAIR, GpairDesc): a = the
// step's activation input A, f = its factor F, g = the output gradient, da =
// dA (NULL: not wanted), part = the per-block partials of dF.
hipError_t launch_gpair(const Launch& ln, const void* a, const void* f, const void* g, void* da, void* part,
                        hipStream_t s);

// Thin channel mixing (K_THIN, GemmDesc): a = factor, b = activations, c = out.
hipError_t launch_thin(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s);

// General contraction (K_TC main launch: a = A, b = B, c = C, d = partials;
// K_TC_REDUCE: d = partials, c = C).
hipError_t launch_tc(const Launch& ln, const void* a, const void* b, void* c, void* d, hipStream_t s);

// Fused tensor-train contraction + convolution forward (K_TT_FWD) and its
// prepared convolution operands (K_TT_PREP): ops = {X, F1, F2, A2}, y = Y.
hipError_t launch_tt_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s);

// Fused CP chain forward: ops = {X, Us, Kh, Kw, Ut}.
hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s);

// Fused reshaped-CP chain forward: ops = {X, W1, W2, W3, W0}, y = Y.
hipError_t launch_rcp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s);

// Fused reshaped-CP chain backward: ops = {X, dY, W1, W2, W3, W0, DXP, P0, P1, P2, P3, TB},
// and its factor table: ops = {W1, W2, W3, W0, TB}.
hipError_t launch_rcp_bwd(const Launch& ln, const void* const* ops, hipStream_t s);
hipError_t launch_rcp_prep(const Launch& ln, const void* const* ops, hipStream_t s);

// Fused CP chain backward: ops = {X, dY, dX (may be NULL), Us, Kh, Kw, Ut,
// Pus, Put, Pkh, Pkw}.
hipError_t launch_cp_bwd(const Launch& ln, const void* const* ops, hipStream_t s);

}  // namespace ce
