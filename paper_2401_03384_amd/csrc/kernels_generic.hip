// Generic strided pairwise-step kernel.
//
// Evaluates any pairwise step of the forward or backward pass described by a
// GenericDesc: contraction, batch and outer-product labels by strides, each
// convolved label by its affine position map with zero outside the operand
// (same padding), or taken modulo N for a circular label.  It is the reference HIP implementation every specialised
// kernel is checked against, and the fallback for steps no specialised kernel
// takes.  Accumulation is float32; long reductions are split over the lanes
// of a wavefront or a block and summed by a fixed butterfly / tree, so results
// are deterministic.
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

struct OutPos {
    int64_t offL, offR, offC;
    int64_t conv_p[kMaxConv];
};

__device__ __forceinline__ OutPos decode_out(const GenericDesc& d, int64_t o) {
    OutPos r;
    r.offL = r.offR = r.offC = 0;
    int64_t idx[kMaxDims];
#pragma unroll
    for (int i = kMaxDims - 1; i >= 0; --i) {
        if (i < d.nout) {
            int64_t sz = d.out_size[i];
            int64_t q = o / sz;
            int64_t x = o - q * sz;
            o = q;
            idx[i] = x;
            r.offL += x * d.out_sL[i];
            r.offR += x * d.out_sR[i];
            r.offC += x * d.out_sC[i];
        } else {
            idx[i] = 0;
        }
    }
#pragma unroll
    for (int k = 0; k < kMaxConv; k++) {
        int64_t v = 0;
#pragma unroll
        for (int i = 0; i < kMaxDims; i++)
            if (k < d.nconv && i == d.cv_out[k]) v = idx[i];
        r.conv_p[k] = v;
    }
    return r;
}

template <typename TL, typename TR>
__device__ __forceinline__ float term(const GenericDesc& d, const TL* __restrict__ L,
                                      const TR* __restrict__ R, const OutPos& op, int64_t r) {
    int64_t offL = op.offL, offR = op.offR;
    int64_t idx[kMaxDims];
#pragma unroll
    for (int i = kMaxDims - 1; i >= 0; --i) {
        if (i < d.nred) {
            int64_t sz = d.red_size[i];
            int64_t q = r / sz;
            int64_t x = r - q * sz;
            r = q;
            idx[i] = x;
            offL += x * d.red_sL[i];
            offR += x * d.red_sR[i];
        } else {
            idx[i] = 0;
        }
    }
#pragma unroll
    for (int k = 0; k < kMaxConv; k++) {
        if (k < d.nconv) {
            int64_t j = 0;
#pragma unroll
            for (int i = 0; i < kMaxDims; i++)
                if (i == d.cv_red[k]) j = idx[i];
            int64_t p = op.conv_p[k];
            int64_t pl = d.cv_aL[k] * p + d.cv_bL[k] * j + d.cv_gL[k];
            int64_t pr = d.cv_aR[k] * p + d.cv_bR[k] * j + d.cv_gR[k];
            if (d.cv_modL[k]) pl = ((pl % d.cv_modL[k]) + d.cv_modL[k]) % d.cv_modL[k];
            if (d.cv_modR[k]) pr = ((pr % d.cv_modR[k]) + d.cv_modR[k]) % d.cv_modR[k];
            if (pl < 0 || pl >= d.cv_limL[k] || pr < 0 || pr >= d.cv_limR[k]) return 0.f;
            offL += pl * d.cv_sL[k];
            offR += pr * d.cv_sR[k];
        }
    }
    float a = load(L, offL);
    return d.has_r ? a * load(R, offR) : a;
}

template <typename TL, typename TR, typename TC>
__global__ void __launch_bounds__(256) generic_thread(GenericDesc d, const TL* __restrict__ L,
                                                      const TR* __restrict__ R, TC* __restrict__ C) {
    int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (o >= d.total_out) return;
    OutPos op = decode_out(d, o);
    float acc = 0.f;
    for (int64_t r = 0; r < d.total_red; r++) acc += term(d, L, R, op, r);
    store(C, op.offC, acc);
}

template <typename TL, typename TR, typename TC>
__global__ void __launch_bounds__(256) generic_wave(GenericDesc d, const TL* __restrict__ L,
                                                    const TR* __restrict__ R, TC* __restrict__ C) {
    int64_t o = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    int lane = threadIdx.x & 63;
    if (o >= d.total_out) return;   // uniform per wavefront
    OutPos op = decode_out(d, o);
    float acc = 0.f;
    for (int64_t r = lane; r < d.total_red; r += 64) acc += term(d, L, R, op, r);
    acc = wave_sum(acc);
    if (lane == 0) store(C, op.offC, acc);
}

template <typename TL, typename TR, typename TC>
__global__ void __launch_bounds__(256) generic_block(GenericDesc d, const TL* __restrict__ L,
                                                     const TR* __restrict__ R, TC* __restrict__ C) {
    __shared__ float part[4];
    int64_t o = blockIdx.x;
    OutPos op = decode_out(d, o);
    float acc = 0.f;
    for (int64_t r = threadIdx.x; r < d.total_red; r += 256) acc += term(d, L, R, op, r);
    acc = wave_sum(acc);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) store(C, op.offC, (part[0] + part[1]) + (part[2] + part[3]));
}

template <typename TL, typename TR, typename TC>
hipError_t launch_t(int variant, const Launch& ln, const void* a, const void* b, void* c,
                    hipStream_t s) {
    GenericDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    dim3 g(ln.grid[0], ln.grid[1], ln.grid[2]), bl(ln.block[0], ln.block[1], ln.block[2]);
    const TL* L = (const TL*)a;
    const TR* R = (const TR*)(d.has_r ? b : a);
    TC* C = (TC*)c;
    if (variant == K_GENERIC_THREAD)
        hipLaunchKernelGGL((generic_thread<TL, TR, TC>), g, bl, 0, s, d, L, R, C);
    else if (variant == K_GENERIC_WAVE)
        hipLaunchKernelGGL((generic_wave<TL, TR, TC>), g, bl, 0, s, d, L, R, C);
    else
        hipLaunchKernelGGL((generic_block<TL, TR, TC>), g, bl, 0, s, d, L, R, C);
    return hipGetLastError();
}

template <typename TL, typename TR>
hipError_t launch_c(int variant, int tC, const Launch& ln, const void* a, const void* b, void* c,
                    hipStream_t s) {
    return tC ? launch_t<TL, TR, bf16_t>(variant, ln, a, b, c, s)
              : launch_t<TL, TR, float>(variant, ln, a, b, c, s);
}

template <typename TL>
hipError_t launch_r(int variant, int tR, int tC, const Launch& ln, const void* a, const void* b,
                    void* c, hipStream_t s) {
    return tR ? launch_c<TL, bf16_t>(variant, tC, ln, a, b, c, s)
              : launch_c<TL, float>(variant, tC, ln, a, b, c, s);
}

}  // namespace

hipError_t launch_generic(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s) {
    int variant = ln.kind & 0xff;
    int tL = (ln.kind >> 8) & 1, tR = (ln.kind >> 9) & 1, tC = (ln.kind >> 10) & 1;
    return tL ? launch_r<bf16_t>(variant, tR, tC, ln, a, b, c, s)
              : launch_r<float>(variant, tR, tC, ln, a, b, c, s);
}

}  // namespace ce
