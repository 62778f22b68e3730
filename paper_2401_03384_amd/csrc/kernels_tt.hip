// Fused tensor-train chain forward (TtDesc, desc.h): the step that contracts
// the input's first channel modes with the merged leading cores and the step
// that convolves the result with the merged trailing core (the reshaped
// tensor-train layer of Appendix A.3 (3b); Section 3.3 on intermediates as
// the memory cost), in one launch.  The intermediate Z never reaches HBM:
//
//   Z[b][g][u][r][p] = sum_k X[b][k][u][p] * F1[g][k][r]
//   Y[b][g][t][p]    = sum_{u, r, kh, kw} Z[b][g][u][r][p + (kh - 1, kw - 1)] * F2[t][u][r][kh][kw]
//
// A block owns one (b, g) and four output rows.  For each u it
//   1. forms the 16 channels r of Z on the six rows the 3x3 taps reach
//      (fp32 MFMA 16x16x4: M = r, N = 16 pixels, K = k), written to an LDS
//      plane per r with a zero column on each side (zero rows outside the
//      image come from loads that read 0), then
//   2. accumulates Y on fp32 MFMA 16x16x4 tiles whose 16 rows are (t, one of
//      two output rows) and whose K runs over (r, four tap rows covering both
//      output rows, three tap columns): the A operand is F2 placed at the tap
//      row of each output row (zero elsewhere), so eight output channels fill
//      the tile at 9/12 of its multiply-adds.  A small launch (tt_prep) lays
//      these A operands out beforehand in the order the lanes load them.
// Operand layouts of the 16x16x4 f32 MFMA: lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16] and holds D[4 (l / 16) + i][l % 16], i < 4.
#include <cstdint>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// a byte offset past every operand (extents < 2^31 bytes): the load reads 0
constexpr int kOut = (int)0x80000000u;

// Wait states after an MFMA chain whose results VALU code reads next, on every
// path before any branch (the compiler's own padding has been seen to fall
// short on a branch path that jumps straight to such a read).
__device__ __forceinline__ void mfma_drain() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ float ldf(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}

// Phase-2 A operand of step u, k step s (tap row khp = (s / 4) / 3, tap column
// kw = (s / 4) % 3, r = 4 (s % 4) + lane / 16) for lane `lane` (row m = lane %
// 16: channel t = m % 8 at output row m / 8): F2 at tap row khp - m / 8, zero
// outside the filter or past T.
__device__ __forceinline__ float tt_a2(const TtDesc& d, const float* __restrict__ F2, int u, int s, int lane) {
    const int q = lane >> 4, c16 = lane & 15, t3 = c16 & 7, dy = c16 >> 3;
    const int rh = s & 3, kw = (s >> 2) % 3, khp = (s >> 2) / 3, kh = khp - dy;
    if (t3 >= d.T || kh < 0 || kh >= 3) return 0.f;
    return F2[(int64_t)t3 * d.f2_st + (int64_t)u * d.f2_su + (int64_t)(4 * rh + q) * d.f2_sr +
              (int64_t)kh * d.f2_sh + (int64_t)kw * d.f2_sw];
}

// The phase-2 A operands of every u, in the order the main kernel loads them:
// A2[u][s / 4][lane][s % 4] (one 16-byte load a lane per four k steps).
__global__ void __launch_bounds__(256) tt_prep(TtDesc d, const float* __restrict__ F2, float* __restrict__ A2) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)d.U * 48 * 64) return;
    const int j = (int)(i & 3), lane = (int)((i >> 2) & 63);
    const int64_t us4 = i >> 8;
    const int s4 = (int)(us4 % 12), u = (int)(us4 / 12);
    A2[i] = tt_a2(d, F2, u, 4 * s4 + j, lane);
}

template <int XT>
struct TtLds {
    static constexpr int PW = 16 * XT + 2;                                 // words of a Z row
    static constexpr int plane = ((6 * PW - 16 + 63) / 64) * 64 + 16;      // words of one r (= 16 mod 64)
};

// NS1: phase-1 k steps (4 values of k each); XT: 16-column tiles of a row
template <int NS1, int XT>
__global__ void __launch_bounds__(256) tt_fwd(TtDesc d, const float* __restrict__ X,
                                              const float* __restrict__ F1,
                                              const float4* __restrict__ A2, float* __restrict__ Y) {
    constexpr int PW = TtLds<XT>::PW, PL = TtLds<XT>::plane;
    constexpr int NS2 = 4 * 3 * 4;              // (tap row 0..3, tap column 0..2, r / 4)
    constexpr int MAXC = (2 * XT + 3) / 4;      // output tiles of a wave
    extern __shared__ __attribute__((aligned(16))) float zc[];   // [16][PL]
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), q = lane >> 4, c16 = lane & 15;
    int64_t bid = blockIdx.x;
    if (d.xcd_remap) {
        // consecutive block ids go to different XCDs: give each XCD a
        // contiguous run of work so the blocks of one sample share its L2
        const int64_t per = d.blocks >> 3;
        bid = (bid & 7) * per + (bid >> 3);
    }
    const int band = (int)(bid % d.nbands);
    bid /= d.nbands;
    const int g = (int)(bid % d.G);
    const int64_t b = bid / d.G;
    const int y0 = band * 4;
    for (int i = threadIdx.x; i < 16 * PL; i += 256) zc[i] = 0.f;

    const __amdgpu_buffer_rsrc_t rX =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(X), (short)0, (int)(4 * d.x_numel), 0x00020000);
    const __amdgpu_buffer_rsrc_t rF1 =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(F1), (short)0, (int)(4 * d.f1_numel), 0x00020000);

    // phase-1 A operand: F1[g][k][r] with r = c16, k = 4 s + q (zero past K1)
    float a1[NS1];
#pragma unroll
    for (int s = 0; s < NS1; s++) {
        const int k = 4 * s + q;
        const int64_t o = (int64_t)g * d.f1_sg + (int64_t)k * d.f1_sk + (int64_t)c16 * d.f1_sr;
        a1[s] = ldf(rF1, k < d.K1 ? (int)(4 * o) : kOut, 0);
    }
    f32x4 acc[MAXC];
#pragma unroll
    for (int j = 0; j < MAXC; j++) acc[j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    const int npx = 6 * d.W, ntile = (npx + 15) >> 4;
    // phase-1 B operands (X) of this wave's tiles ti = wave + 4 j of step u:
    // those of step u + 1 load while step u's phase 2 runs
    constexpr int MAXT1 = (6 * XT + 3) / 4;
    float bv[MAXT1][NS1];
    auto load_x = [&](int u) {
#pragma unroll
        for (int j = 0; j < MAXT1; j++) {
            const int ti = wave + 4 * j;
            const int e = (ti << 4) + c16;
            const int rr = e / d.W, cc = e - rr * d.W;
            const int y = y0 - 1 + rr;
            const bool ok = ti < ntile && e < npx && y >= 0 && y < d.H;
            const int64_t o = b * d.x_sb + (int64_t)q * d.x_sk + (int64_t)u * d.x_su + (int64_t)y * d.W + cc;
            const int voff = ok ? (int)(4 * o) : kOut;
#pragma unroll
            for (int s = 0; s < NS1; s++) bv[j][s] = ldf(rX, voff, (int)(16 * s * d.x_sk));
        }
    };
    load_x(0);
    __syncthreads();

    for (int u = 0; u < d.U; u++) {
        // this u's phase-2 A operand, loaded before phase 1 so the loads are in flight meanwhile
        float a2[NS2];
        {
            const float4* src = A2 + (int64_t)u * (NS2 / 4) * 64 + lane;
#pragma unroll
            for (int s4 = 0; s4 < NS2 / 4; s4++) {
                const float4 v = src[s4 * 64];
                a2[4 * s4] = v.x;
                a2[4 * s4 + 1] = v.y;
                a2[4 * s4 + 2] = v.z;
                a2[4 * s4 + 3] = v.w;
            }
        }
        // phase 1: Z of this u on rows y0 - 1 .. y0 + 4 into LDS (operands
        // loaded during the previous step)
        f32x4 z[MAXT1];
#pragma unroll
        for (int j = 0; j < MAXT1; j++) {
            z[j] = (f32x4){0.f, 0.f, 0.f, 0.f};
            if (wave + 4 * j < ntile) {
#pragma unroll
                for (int s = 0; s < NS1; s++)
                    z[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[s], bv[j][s], z[j], 0, 0, 0);
            }
        }
        // the next step's operands, in flight during this step's phase 2
        if (u + 1 < d.U) load_x(u + 1);
        mfma_drain();
#pragma unroll
        for (int j = 0; j < MAXT1; j++) {
            const int ti = wave + 4 * j;
            const int e = (ti << 4) + c16;
            if (ti < ntile && e < npx) {
                const int rr = e / d.W, cc = e - rr * d.W;
                float* dst = zc + (4 * q) * PL + rr * PW + cc + 1;
#pragma unroll
                for (int i = 0; i < 4; i++) dst[i * PL] = z[j][i];
            }
        }
        __syncthreads();
        // phase 2: output tiles (row pair, 16 columns) of this wave
#pragma unroll
        for (int j = 0; j < MAXC; j++) {
            const int cmb = wave + 4 * j;
            if (cmb < d.ncombo) {
                const int pr = cmb / XT, xt = cmb - pr * XT;
                const float* src = zc + q * PL + (2 * pr) * PW + xt * 16 + c16;
#pragma unroll
                for (int s = 0; s < NS2; s++) {
                    const int rh = s & 3, kw = (s >> 2) % 3, khp = (s >> 2) / 3;
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a2[s], src[4 * rh * PL + khp * PW + kw], acc[j], 0, 0, 0);
                }
            }
        }
        __syncthreads();
    }
    mfma_drain();
    // D row 4q + i of a tile: channel t = (4q + i) % 8, output row 2 pr + (4q + i) / 8
#pragma unroll
    for (int j = 0; j < MAXC; j++) {
        const int cmb = wave + 4 * j;
        if (cmb < d.ncombo) {
            const int pr = cmb / XT, xt = cmb - pr * XT;
            const int x = xt * 16 + c16;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int m = 4 * q + i, t = m & 7, y = y0 + 2 * pr + (m >> 3);
                if (t < d.T && y < d.H && x < d.W)
                    Y[b * d.y_sb + (int64_t)g * d.y_sg + (int64_t)t * d.y_st + (int64_t)y * d.W + x] = acc[j][i];
            }
        }
    }
}

template <int NS1, int XT>
hipError_t tt_go(const TtDesc& d, const void* const* ops, void* y, hipStream_t s) {
    hipLaunchKernelGGL((tt_fwd<NS1, XT>), dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d,
                       (const float*)ops[0], (const float*)ops[1], (const float4*)ops[3], (float*)y);
    return hipGetLastError();
}

template <int NS1>
hipError_t tt_xt(const TtDesc& d, const void* const* ops, void* y, hipStream_t s) {
    switch (d.XT) {
        case 1: return tt_go<NS1, 1>(d, ops, y, s);
        case 2: return tt_go<NS1, 2>(d, ops, y, s);
        case 4: return tt_go<NS1, 4>(d, ops, y, s);
    }
    return hipErrorInvalidValue;
}

int tt_ns1(int K1) {
    const int n = (K1 + 3) / 4;
    return n <= 1 ? 1 : n <= 2 ? 2 : n <= 4 ? 4 : n <= 8 ? 8 : n <= 16 ? 16 : 0;
}

int tt_plane(int XT) {
    switch (XT) {
        case 1: return TtLds<1>::plane;
        case 2: return TtLds<2>::plane;
        case 4: return TtLds<4>::plane;
    }
    return 0;
}

}  // namespace

// ops = {X, F1, F2, A2}: K_TT_PREP writes A2 from F2, K_TT_FWD reads X, F1, A2
hipError_t launch_tt_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    TtDesc d;
    if (ln.desc.size() != sizeof(d)) return hipErrorInvalidValue;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (!ops[3]) return hipErrorInvalidValue;
    if ((ln.kind & 0xff) == K_TT_PREP) {
        if (d.U < 1 || d.T < 1 || d.T > 8 || d.R != 16 || !ops[2]) return hipErrorInvalidValue;
        const int64_t n = (int64_t)d.U * 48 * 64;
        hipLaunchKernelGGL(tt_prep, dim3((uint32_t)((n + 255) / 256)), dim3(256), 0, s, d, (const float*)ops[2],
                           (float*)ops[3]);
        return hipGetLastError();
    }
    // the descriptor must be the one the kernel indexes: every LDS access
    // stays inside 16 planes, every global offset inside 2^31 bytes
    const int ns1 = tt_ns1(d.K1);
    if (ns1 == 0 || d.R != 16 || d.T < 1 || d.T > 8 || d.TH != 4 || d.U < 1 || d.G < 1 || d.B < 1 ||
        d.H < 1 || d.W < 1 || !(d.XT == 1 || d.XT == 2 || d.XT == 4) || d.W > 16 * d.XT ||
        d.PW != 16 * d.XT + 2 || d.plane != tt_plane(d.XT) || d.plane < 6 * d.PW ||
        d.lds_bytes != (uint32_t)(16 * d.plane * 4) || d.ncombo != 2 * d.XT ||
        (int64_t)d.nbands * 4 < d.H || d.blocks != (int64_t)d.B * d.G * d.nbands ||
        (int64_t)ln.grid[0] != d.blocks || d.blocks > 0x7fffffff || (d.xcd_remap && (d.blocks & 7)) ||
        d.x_numel <= 0 || d.x_numel >= (1ll << 29) || d.f1_numel <= 0 || d.f1_numel >= (1ll << 29) ||
        d.f2_numel <= 0 || d.f2_numel >= (1ll << 29))
        return hipErrorInvalidValue;
    switch (ns1) {
        case 1: return tt_xt<1>(d, ops, y, s);
        case 2: return tt_xt<2>(d, ops, y, s);
        case 4: return tt_xt<4>(d, ops, y, s);
        case 8: return tt_xt<8>(d, ops, y, s);
        case 16: return tt_xt<16>(d, ops, y, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace ce
