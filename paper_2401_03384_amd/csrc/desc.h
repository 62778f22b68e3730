// Plain-old-data kernel descriptors, filled by the host planner and passed
// by value to the HIP kernels.  No HIP types here: this header is included
// by host-only sources as well.
#pragma once

#include <cstdint>

namespace ce {

enum DType : int32_t { DT_F32 = 0, DT_BF16 = 1 };

constexpr int kMaxDims = 8;   // loop dimensions of a generic pairwise step
constexpr int kMaxConv = 4;   // convolved labels of one step

// A pairwise step in its most general form:
//
//   C[o] = sum_r  L[offL(o, r)] * R[offR(o, r)]
//
// o runs over the output dims (the layout of C), r over the reduction dims.
// A plain dim contributes index * stride to each operand.  A convolved label
// owns one output dim (index p) and one reduction dim (index j) whose plain
// strides are zero; it contributes pos * stride to an operand, where
// pos = a * p + b * j + g must lie in [0, lim) or the term is skipped.  This
// covers the forward step (feature read at p + j - c, filter at j), the
// gradient of the feature side (dC read at p - j + c) and the gradient of the
// filter side (feature read at j + p - c, dC at j).
struct GenericDesc {
    int32_t nout, nred, nconv;
    int32_t has_r;                     // 0: R is absent (treated as 1)
    int64_t total_out, total_red;
    int64_t out_size[kMaxDims], out_sL[kMaxDims], out_sR[kMaxDims], out_sC[kMaxDims];
    int64_t red_size[kMaxDims], red_sL[kMaxDims], red_sR[kMaxDims];
    int32_t cv_out[kMaxConv], cv_red[kMaxConv];    // dim indices
    int32_t cv_aL[kMaxConv], cv_bL[kMaxConv], cv_aR[kMaxConv], cv_bR[kMaxConv];
    int64_t cv_gL[kMaxConv], cv_limL[kMaxConv], cv_sL[kMaxConv];
    int64_t cv_gR[kMaxConv], cv_limR[kMaxConv], cv_sR[kMaxConv];
};

enum KernelKind : int32_t {
    K_GENERIC_THREAD = 1,   // one thread per output element
    K_GENERIC_WAVE = 2,     // one 64-lane wavefront per output element
    K_GENERIC_BLOCK = 3,    // one 256-thread block per output element
};

}  // namespace ce
