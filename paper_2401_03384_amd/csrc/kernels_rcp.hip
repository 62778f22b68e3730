// Fused reshaped-CP chain forward for gfx950 (RcpDesc; the phases are in
// rcp_body.h).
//
// The three mode products and the rank-summed 2-D convolution of a reshaped
// CP layer (Section 2.3; Appendix A.3 RCP string) run in one launch: each
// workgroup keeps its sample's X values in registers, builds Z2 and Z3 of one
// rank at a time in LDS and accumulates Y over the ranks in registers, so none
// of the three rank-expanded intermediates (64x the input at rank 64) touches
// HBM.  bf16 pairs feed v_dot2_f32_bf16 throughout: pairs along s1, s2 and s3
// for the mode products, pairs of ranks for the convolution.  The work is
// plain vector ALU (the contractions have 4 or 8 terms), so the roofline is
// the fp32 vector rate (two bf16 products per dot2 lane-op).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>

#include "desc_rcp.h"
#include "hip_util.h"
#include "kernels.h"

#define RCP_FN __device__ __forceinline__
#define RCP_HD __host__ __device__ inline
#include "rcp_body.h"
#define RCPB_FN __device__ __forceinline__
#define RCPB_HD __host__ __device__ inline
#include "rcpb_body.h"

namespace ce {
namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct DevMem {
    uint32_t* lds;
    __device__ __forceinline__ uint16_t ld16(const uint16_t* p, int64_t i) const { return p[i]; }
    __device__ __forceinline__ uint32_t ldw(const uint16_t* p, int64_t i) const {
        return *reinterpret_cast<const uint32_t*>(p + i);
    }
    __device__ __forceinline__ void st16(uint16_t* p, int64_t i, uint16_t v) const { p[i] = v; }
    __device__ __forceinline__ uint32_t lr(int i) const { return lds[i]; }
    __device__ __forceinline__ uint16_t lr16(int i, int half) const {
        return reinterpret_cast<const uint16_t*>(lds)[2 * i + half];
    }
    __device__ __forceinline__ void lr4(int i, uint32_t* o) const {
        const uint4 v = *reinterpret_cast<const uint4*>(lds + i);
        o[0] = v.x;
        o[1] = v.y;
        o[2] = v.z;
        o[3] = v.w;
    }
    __device__ __forceinline__ void lw(int i, uint32_t v) const { lds[i] = v; }
    __device__ __forceinline__ void lw16(int i, int half, uint16_t v) const {
        reinterpret_cast<uint16_t*>(lds)[2 * i + half] = v;
    }
    __device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) const {
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                              __builtin_bit_cast(bf16x2_t, b), c, false);
    }
    __device__ __forceinline__ uint32_t pk(float lo, float hi) const { return pk_bf16(lo, hi); }
    __device__ __forceinline__ uint16_t bf(float f) const { return f32_to_bf16(f); }
    __device__ __forceinline__ float f(uint16_t h) const { return to_f32(h); }
    __device__ __forceinline__ uint32_t fbits(float v) const { return __float_as_uint(v); }
    __device__ __forceinline__ float fof(uint32_t u) const { return __uint_as_float(u); }
    __device__ __forceinline__ void stf(float* p, int64_t i, float v) const { p[i] = v; }
    __device__ __forceinline__ uint32_t ldt(const uint32_t* p, int64_t i) const { return p[i]; }
    // sum of x over the 16 lanes of this lane's row (DPP row shifts); the
    // row's last lane writes it to LDS word `word`
    __device__ __forceinline__ void rowsum(float x, int lane, int word) const {
        x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x111, 0xf, 0xf, true));
        x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x112, 0xf, 0xf, true));
        x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x114, 0xf, 0xf, true));
        x += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), 0x118, 0xf, 0xf, true));
        if ((lane & 15) == 15) lds[word] = __float_as_uint(x);
    }
    // acc += A B on one 32x32x16 bf16 MFMA tile (wave-wide)
    __device__ __forceinline__ void mfma(const uint32_t* a, const uint32_t* b, float* acc) const {
        const uint4 av = {a[0], a[1], a[2], a[3]}, bv = {b[0], b[1], b[2], b[3]};
        f32x16_t c;
#pragma unroll
        for (int i = 0; i < 16; i++) c[i] = acc[i];
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                    __builtin_bit_cast(bf16x8_t, bv), c, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 16; i++) acc[i] = c[i];
    }
};

template <class C>
__global__ void __launch_bounds__(C::NT) rcp_fwd(RcpDesc d, const uint16_t* __restrict__ X,
                                                const uint16_t* __restrict__ W1,
                                                const uint16_t* __restrict__ W2,
                                                const uint16_t* __restrict__ W3,
                                                const uint16_t* __restrict__ W0,
                                                uint16_t* __restrict__ Y) {
    extern __shared__ uint32_t lds_words[];
    DevMem m{lds_words};
    const int tid = threadIdx.x;
    int b, t1, tile, chunk;
    rcp::block_coords(d, blockIdx.x, b, t1, tile, chunk);
    const rcp::Tile t = rcp::tile_rows(d, tile);
    rcp::State<C> st;
    rcp::init<C>(m, d, tid, b, t, X, st);
    rcp::phase_a<C>(m, d, t, 0, t1, chunk, 0, W1, W2, st);
    __syncthreads();
    const int np = d.R / 2;
    for (int rp = 0; rp < np; rp++) {
        const int r0 = 2 * rp;
        rcp::phase_b<C>(m, d, t, r0, 0, W3, st);
        rcp::phase_a<C>(m, d, t, r0 + 1, t1, chunk, 1, W1, W2, st);
        __syncthreads();
        rcp::phase_b<C>(m, d, t, r0 + 1, 1, W3, st);
        __syncthreads();
        rcp::phase_c<C>(m, d, r0, W0, st);
        if (rp + 1 < np) rcp::phase_a<C>(m, d, t, r0 + 2, t1, chunk, 0, W1, W2, st);
        __syncthreads();
    }
    rcp::store<C>(m, d, tid, b, t1, t, chunk, Y, st);
}

template <int I>
using CfgOf = rcp::Cfg<kRcpCfgs[I].S1, kRcpCfgs[I].S2, kRcpCfgs[I].S3, kRcpCfgs[I].T2, kRcpCfgs[I].T3,
                       kRcpCfgs[I].K, kRcpCfgs[I].T2C, kRcpCfgs[I].NT, kRcpCfgs[I].UA, kRcpCfgs[I].UB,
                       kRcpCfgs[I].UC>;
static_assert(kNumRcpCfgs == 2, "one launch branch per instantiation");

// The descriptor matches instantiation C and every tile's units fit its
// per-thread bounds.
template <class C>
bool fits(const RcpDesc& d) {
    if (!rcp::layout_ok(d) || d.S1 != C::S1 || d.S2 != C::S2 || d.S3 != C::S3 || d.T2 != C::T2 ||
        d.T3 != C::T3 || d.K != C::K || d.T2C != C::T2C || d.NT != C::NT)
        return false;
    for (int i = 0; i < d.ntiles; i++) {
        const rcp::Tile t = rcp::tile_rows(d, i);
        if (rcp::units_a(d, t) > C::UA * C::NT || rcp::units_b(d, t) > C::UB * C::NT ||
            rcp::units_c(d, t) > C::UC * C::NT)
            return false;
    }
    return true;
}

template <class C>
hipError_t launch_rcp_c(const RcpDesc& d, const void* const* o, void* y, hipStream_t s) {
    auto k = rcp_fwd<C>;
    static std::atomic<uint64_t> allowed{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || d.lds_bytes > 160 * 1024) return hipErrorInvalidValue;
    if (d.lds_bytes > 64 * 1024 && !(allowed.load() & (1ull << dev))) {
        e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        allowed.fetch_or(1ull << dev);
    }
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(C::NT), d.lds_bytes, s, d,
                       (const uint16_t*)o[0], (const uint16_t*)o[1], (const uint16_t*)o[2],
                       (const uint16_t*)o[3], (const uint16_t*)o[4], (uint16_t*)y);
    return hipGetLastError();
}

template <class C>
__global__ void __launch_bounds__(C::NT, C::MW) rcp_bwd(RcpBwdDesc d, const uint16_t* __restrict__ X,
                                                const uint16_t* __restrict__ dY,
                                                const uint16_t* __restrict__ W1,
                                                const uint16_t* __restrict__ W2,
                                                const uint16_t* __restrict__ W3,
                                                const uint16_t* __restrict__ W0, float* __restrict__ DXP,
                                                float* __restrict__ P0, float* __restrict__ P1,
                                                float* __restrict__ P2, float* __restrict__ P3,
                                                const uint32_t* __restrict__ TB) {
    extern __shared__ uint32_t lds_words[];
    DevMem m{lds_words};
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int64_t blk;
    int b, t1, tile, chunk, h0, h1;
    rcpb::block_coords_b(d, blockIdx.x, blk, b, t1, tile, chunk);
    rcpb::tile_of(d, tile, h0, h1);
    const int P = (h1 - h0) * d.W;
    rcpb::State<C> st;
    rcpb::init<C>(m, d, tid, b, t1, h0, h1, chunk, X, dY, st);
    __syncthreads();
    for (int r = 0; r < d.R; r++) {
        rcpb::phase_a<C>(m, d, r, t1, chunk, W1, W2, st);
        if (r > 0) rcpb::phase_f<C>(m, d, tid, blk, r - 1, t1, chunk, P0, P1, P2, P3);
        __syncthreads();
        rcpb::phase_b<C>(m, d, r, P, W3, st);
        __syncthreads();
        rcpb::phase_c<C>(m, d, lane, wave, r, P, TB, st);
        __syncthreads();
        rcpb::phase_d<C>(m, d, r, TB, st);
        {
            float acc[16] = {};
            rcpb::mfma_part<C>(m, lane, wave, d.o_g3, d.o_z2, d.L2, C::T2C * d.PP / 16, C::T3, C::S3, acc);
            rcpb::mfma_store<C>(m, lane, d.o_m3 + wave * C::T3 * C::S3, C::T3, C::S3, acc);
        }
        __syncthreads();
        rcpb::phase_e<C>(m, d, lane, wave, r, t1, chunk, TB, st);
        {
            float acc[16] = {};
            rcpb::mfma_part<C>(m, lane, wave, d.o_g2, d.o_z1, d.L13, C::S3 * d.PP / 16, C::T2C, C::S2, acc);
            rcpb::mfma_store<C>(m, lane, d.o_m2 + wave * C::T2C * C::S2, C::T2C, C::S2, acc);
        }
        __syncthreads();
    }
    rcpb::phase_f<C>(m, d, tid, blk, d.R - 1, t1, chunk, P0, P1, P2, P3);
    rcpb::store_dx<C>(m, d, b, t1, h0, chunk, DXP, st);
}

// The prepared factor table of the backward (rcpb::table_word), one word a thread.
__global__ void __launch_bounds__(256) rcp_prep(RcpBwdDesc d, const uint16_t* __restrict__ W1,
                                                const uint16_t* __restrict__ W2,
                                                const uint16_t* __restrict__ W3,
                                                const uint16_t* __restrict__ W0, uint32_t* __restrict__ TB) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)d.R * d.tbs) return;
    DevMem m{nullptr};
    TB[i] = rcpb::table_word(m, d, i, W1, W2, W3, W0);
}

template <int I>
using BCfgOf = rcpb::Cfg<kRcpBwdCfgs[I].S1, kRcpBwdCfgs[I].S2, kRcpBwdCfgs[I].S3, kRcpBwdCfgs[I].T2,
                         kRcpBwdCfgs[I].T3, kRcpBwdCfgs[I].K, kRcpBwdCfgs[I].T2C, kRcpBwdCfgs[I].NT,
                         kRcpBwdCfgs[I].UA, kRcpBwdCfgs[I].UB, kRcpBwdCfgs[I].UC, kRcpBwdCfgs[I].MW>;
static_assert(kNumRcpBwdCfgs == 2, "one launch branch per instantiation");

template <class C>
bool fits_b(const RcpBwdDesc& d) {
    if (!rcpb::layout_ok_b(d) || d.S1 != C::S1 || d.S2 != C::S2 || d.S3 != C::S3 || d.T2 != C::T2 ||
        d.T3 != C::T3 || d.K != C::K || d.T2C != C::T2C || d.NT != C::NT)
        return false;
    const int P = d.TH * d.W;   // the largest tile
    return P * C::S3 <= C::UA * C::NT && P * C::T2C <= C::UB * C::NT &&
           C::T2C * C::T3 * d.TH * d.QW <= C::UC * C::NT;
}

template <class C>
hipError_t launch_rcpb_c(const RcpBwdDesc& d, const void* const* o, hipStream_t s) {
    auto k = rcp_bwd<C>;
    static std::atomic<uint64_t> allowed{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || d.lds_bytes > 160 * 1024) return hipErrorInvalidValue;
    if (d.lds_bytes > 64 * 1024 && !(allowed.load() & (1ull << dev))) {
        e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        allowed.fetch_or(1ull << dev);
    }
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(C::NT), d.lds_bytes, s, d, (const uint16_t*)o[0],
                       (const uint16_t*)o[1], (const uint16_t*)o[2], (const uint16_t*)o[3],
                       (const uint16_t*)o[4], (const uint16_t*)o[5], (float*)o[6], (float*)o[7],
                       (float*)o[8], (float*)o[9], (float*)o[10], (const uint32_t*)o[11]);
    return hipGetLastError();
}

}  // namespace

// ops = {X, W1, W2, W3, W0}; y = Y.  The mode factors are read as 32-bit
// words (bf16 pairs), so their base addresses must be 4-byte aligned.
hipError_t launch_rcp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    RcpDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    for (int i = 1; i <= 3; i++)
        if (((uintptr_t)ops[i]) & 3) return hipErrorInvalidValue;
    const int64_t want = (int64_t)d.B * d.T1 * d.ntiles * d.nc;
    if (d.blocks != want || d.R % 2 || d.R < 2 || ln.lds != d.lds_bytes) return hipErrorInvalidValue;
    if (fits<CfgOf<0>>(d)) return launch_rcp_c<CfgOf<0>>(d, ops, y, s);
    if (fits<CfgOf<1>>(d)) return launch_rcp_c<CfgOf<1>>(d, ops, y, s);
    return hipErrorInvalidValue;
}

// ops = {X, dY, W1, W2, W3, W0, DXP, P0, P1, P2, P3, TB}; the mode factors are
// read as 32-bit words (4-byte aligned base addresses).
hipError_t launch_rcp_bwd(const Launch& ln, const void* const* ops, hipStream_t s) {
    RcpBwdDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    for (int i = 2; i <= 4; i++)
        if (((uintptr_t)ops[i]) & 3) return hipErrorInvalidValue;
    for (int i = 0; i < 12; i++)
        if (!ops[i]) return hipErrorInvalidValue;
    const int64_t want = (int64_t)d.B * d.T1 * d.ntiles * d.nc;
    if (d.blocks != want || ln.lds != d.lds_bytes) return hipErrorInvalidValue;
    if (fits_b<BCfgOf<0>>(d)) return launch_rcpb_c<BCfgOf<0>>(d, ops, s);
    if (fits_b<BCfgOf<1>>(d)) return launch_rcpb_c<BCfgOf<1>>(d, ops, s);
    return hipErrorInvalidValue;
}

// ops = {W1, W2, W3, W0, TB}.
hipError_t launch_rcp_prep(const Launch& ln, const void* const* ops, hipStream_t s) {
    RcpBwdDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int64_t n = (int64_t)d.R * d.tbs;
    if (n <= 0 || (int64_t)ln.grid[0] * 256 < n || !ops[4]) return hipErrorInvalidValue;
    hipLaunchKernelGGL(rcp_prep, dim3(ln.grid[0]), dim3(256), 0, s, d, (const uint16_t*)ops[0],
                       (const uint16_t*)ops[1], (const uint16_t*)ops[2], (const uint16_t*)ops[3], (uint32_t*)ops[4]);
    return hipGetLastError();
}

}  // namespace ce
