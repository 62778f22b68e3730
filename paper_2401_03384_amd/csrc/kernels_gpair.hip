// Both gradients of a channel-mixing step, from one read of its output
// gradient (GpairDesc).  The step C[g][k][n] = sum_m A[g][m][n] F[k][m]
// (Section 3.1: a contraction of an activation A with a factor F; Appendix B:
// its two gradients g1, g2) has
//   dA[g][m][n] = sum_k F[k][m] G[g][k][n]            (g1)
//   dF[k][m]    = sum_{g, n} A[g][m][n] G[g][k][n]     (g2)
// with G = dC the large operand (K rows per g, e.g. the rank-expanded
// activation of a tensor-train layer).  Computed apart, each reads G from HBM;
// here a block stages each 64 x 64 chunk of G in LDS once and feeds both
// products from it on fp32 16x16x4 MFMA tiles.
//
// A block: eight wavefronts, gper consecutive g, every n in tiles of 64, k in
// NKC chunks of 64.  Wavefront w = (mt, q): mt = w / 4 the m tile (16 rows of
// m; M <= 32), q = w % 4.  Per chunk it
//   dA:  the tile (m tile mt, n columns 16q..16q+15): A operand F[k][m] (LDS,
//        k = the chunk's 64 in steps of 4), B operand G[k][n] (LDS);
//   dF:  the tile (k rows 16q.. of the chunk, m tile mt): A operand G[k][n]
//        (LDS, transposed read), B operand A[m][n] (LDS), reduced over the
//        tile's 64 n in steps of 4; one accumulator tile per chunk, kept for
//        the whole block and written as the block's partial at the end.
// F is staged once per block ([k][m], pitch 33); the next chunk of G (and, at
// a new n tile, the next A tile) load into registers while the current chunk
// computes; G and A tiles are double-buffered in LDS, one barrier a chunk.
#include <algorithm>
#include <atomic>
#include <cstdint>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));

constexpr int kGpLF = 33;   // pitch of F [k][m] in LDS
constexpr int kGpLG = 65;   // pitch of the G chunk [k][n] and the A tile [m][n]

__device__ __forceinline__ void gp_offs(const GpairDesc& d, int64_t g, int64_t& oa, int64_t& og, int64_t& od) {
    oa = og = od = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        const int64_t x = g % d.g_size[i];
        g /= d.g_size[i];
        oa += x * d.g_sA[i];
        og += x * d.g_sG[i];
        od += x * d.g_sD[i];
    }
}

template <int NKC, bool VEC>
__global__ void __launch_bounds__(512, 1) gpair(GpairDesc d, const float* __restrict__ A,
                                                const float* __restrict__ F, const float* __restrict__ G,
                                                float* __restrict__ dA, float* __restrict__ P) {
    extern __shared__ float4 lds4[];
    float* Fs = reinterpret_cast<float*>(lds4);               // [NKC * 64][kGpLF]
    float* Gs = Fs + NKC * 64 * kGpLF;                        // [2][64][kGpLG]
    float* As = Gs + 2 * 64 * kGpLG;                          // [2][32][kGpLG]
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int mt = wave >> 2, q = wave & 3, i16 = lane & 15, kq = lane >> 4;
    const int M = d.M, K = d.K, N = d.N;
    const int64_t g0 = (int64_t)blockIdx.x * d.gper, g1 = min(d.G, g0 + d.gper);
    const bool want_da = dA != nullptr;

    // ---- F, once per block: Fs[k][m] (zero past K and M) ----
    for (int e = tid; e < NKC * 64 * 32; e += 512) {
        const int k = e >> 5, m = e & 31;
        float v = 0.f;
        if (k < K && m < M) {
            const int k1 = k / d.K2, k2 = k - k1 * d.K2;
            v = F[k1 * d.sF1 + k2 * d.sF2 + m * d.sFm];
        }
        Fs[k * kGpLF + m] = v;
    }

    // ---- staging: the G chunk (two float4 of a row a thread) and the A tile
    // (one float4 a thread); rows / columns past the ends are zero ----
    auto g_load = [&](int64_t og, int kc, int n0, float4 (&v)[2]) {
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int f = tid + 512 * i, r = f >> 4, c = 4 * (f & 15);
            const int k = 64 * kc + r, n = n0 + c;
            v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (k < K) {
                const int k1 = k / d.K2, k2 = k - k1 * d.K2;
                const float* src = G + og + k1 * d.sG1 + k2 * d.sG2 + n;
                if constexpr (VEC) {
                    if (n < N) v[i] = *reinterpret_cast<const float4*>(src);
                } else {
                    float t[4];
#pragma unroll
                    for (int j = 0; j < 4; j++) t[j] = n + j < N ? src[j] : 0.f;
                    v[i] = make_float4(t[0], t[1], t[2], t[3]);
                }
            }
        }
    };
    auto g_store = [&](int buf, const float4 (&v)[2]) {
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int f = tid + 512 * i, r = f >> 4, c = 4 * (f & 15);
            float* dst = Gs + (buf * 64 + r) * kGpLG + c;
            dst[0] = v[i].x;
            dst[1] = v[i].y;
            dst[2] = v[i].z;
            dst[3] = v[i].w;
        }
    };
    auto a_load = [&](int64_t oa, int n0, float4& v) {
        const int m = tid >> 4, c = 4 * (tid & 15), n = n0 + c;
        v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (m < M) {
            const float* src = A + oa + m * d.sAm + n;
            if constexpr (VEC) {
                if (n < N) v = *reinterpret_cast<const float4*>(src);
            } else {
                float t[4];
#pragma unroll
                for (int j = 0; j < 4; j++) t[j] = n + j < N ? src[j] : 0.f;
                v = make_float4(t[0], t[1], t[2], t[3]);
            }
        }
    };
    auto a_store = [&](int buf, const float4& v) {
        const int m = tid >> 4, c = 4 * (tid & 15);
        float* dst = As + (buf * 32 + m) * kGpLG + c;
        dst[0] = v.x;
        dst[1] = v.y;
        dst[2] = v.z;
        dst[3] = v.w;
    };

    f32x4 accF[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; kc++) accF[kc] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // first chunk
    if (g0 < g1) {
        int64_t oa, og, od;
        gp_offs(d, g0, oa, og, od);
        float4 gv[2], av;
        g_load(og, 0, 0, gv);
        a_load(oa, 0, av);
        g_store(0, gv);
        a_store(0, av);
    }
    __syncthreads();

    int gbuf = 0, abuf = 0;
    for (int64_t g = g0; g < g1; g++) {
        int64_t oa, og, od;
        gp_offs(d, g, oa, og, od);
        for (int nt = 0; nt < d.ntiles; nt++) {
            const int n0 = 64 * nt;
            // the (g, n tile) after this one: its first chunk and its A tile
            const bool last_nt = nt + 1 == d.ntiles;
            const bool more = !last_nt || g + 1 < g1;
            int64_t noa = oa, nog = og;
            int nn0 = n0 + 64;
            if (last_nt && more) {
                int64_t nod;
                gp_offs(d, g + 1, noa, nog, nod);
                nn0 = 0;
            }
            f32x4 accA = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kc = 0; kc < NKC; kc++) {
                // next chunk into registers
                float4 gv[2], av;
                const bool next_tile = kc + 1 == NKC;
                if (!next_tile) g_load(og, kc + 1, n0, gv);
                else if (more) {
                    g_load(nog, 0, nn0, gv);
                    a_load(noa, nn0, av);
                }
                const float* gs = Gs + gbuf * 64 * kGpLG;
                const float* as = As + abuf * 32 * kGpLG;
                // dA tile (m tile mt, columns 16q..): sum over the chunk's k
                if (want_da) {
#pragma unroll
                    for (int s = 0; s < 16; s++) {
                        const int kk = 4 * s + kq;
                        const float a = Fs[(64 * kc + kk) * kGpLF + 16 * mt + i16];
                        const float b = gs[kk * kGpLG + 16 * q + i16];
                        accA = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, accA, 0, 0, 0);
                    }
                }
                // dF tile (k rows 16q.. of the chunk, m tile mt): sum over the tile's n
#pragma unroll
                for (int s = 0; s < 16; s++) {
                    const int nn = 4 * s + kq;
                    const float a = gs[(16 * q + i16) * kGpLG + nn];
                    const float b = as[(16 * mt + i16) * kGpLG + nn];
                    accF[kc] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, accF[kc], 0, 0, 0);
                }
                if (next_tile && want_da) {
                    // dA[g][m][n]: accumulator r = row 4 kq + r, column i16
#pragma unroll
                    for (int r = 0; r < 4; r++) {
                        const int m = 16 * mt + 4 * kq + r, n = n0 + 16 * q + i16;
                        if (m < M && n < N) dA[od + (int64_t)m * d.sDm + n] = accA[r];
                    }
                }
                // registers into the other buffers (their previous readers
                // passed the barrier at the end of the last chunk)
                if (!next_tile) {
                    g_store(1 - gbuf, gv);
                } else if (more) {
                    g_store(1 - gbuf, gv);
                    a_store(1 - abuf, av);
                }
                __syncthreads();
                gbuf = 1 - gbuf;
                if (next_tile) abuf = 1 - abuf;
            }
        }
    }

    // the block's partial of dF, in F's layout: accumulator r = k row 4 kq + r
    // of tile q of chunk kc, column i16 = m
    float* pb = P + (int64_t)blockIdx.x * d.fnumel;
#pragma unroll
    for (int kc = 0; kc < NKC; kc++)
#pragma unroll
        for (int r = 0; r < 4; r++) {
            const int k = 64 * kc + 16 * q + 4 * kq + r, m = 16 * mt + i16;
            if (k < K && m < M) {
                const int k1 = k / d.K2, k2 = k - k1 * d.K2;
                pb[k1 * d.sF1 + k2 * d.sF2 + m * d.sFm] = accF[kc][r];
            }
        }
}

template <int NKC>
hipError_t gpair_go(const GpairDesc& d, bool vec, const float* a, const float* f, const float* g, float* da,
                    float* part, hipStream_t s) {
    static std::atomic<uint64_t> ok{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidValue;
    if (!(ok.load() & (1ull << dev))) {
        e = hipFuncSetAttribute((const void*)gpair<NKC, true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                160 * 1024);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void*)gpair<NKC, false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                    160 * 1024);
        if (e != hipSuccess) return e;
        ok.fetch_or(1ull << dev);
    }
    auto k = vec ? gpair<NKC, true> : gpair<NKC, false>;
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(512), d.lds_bytes, s, d, a, f, g, da, part);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gpair(const Launch& ln, const void* a, const void* f, const void* g, void* da, void* part,
                        hipStream_t s) {
    GpairDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int nkc = d.nkc;
    const uint32_t lds = (uint32_t)(4 * (nkc * 64 * kGpLF + 2 * 64 * kGpLG + 2 * 32 * kGpLG));
    // the shapes the kernel assumes (the lowering guarantees them)
    if (((ln.kind >> kBitIn) & 1) || d.M < 1 || d.M > 32 || d.K < 1 || d.K2 < 1 || d.K1 * d.K2 != d.K ||
        (nkc != 1 && nkc != 2 && nkc != 4 && nkc != 8) || d.K > 64 * nkc || d.N < 1 ||
        d.ntiles != (d.N + 63) / 64 || d.gper < 1 || d.blocks != (d.G + d.gper - 1) / d.gper ||
        d.lds_bytes != lds || ln.grid[0] != (uint32_t)d.blocks || ln.block[0] != 512 || !a || !f || !g || !part)
        return hipErrorInvalidValue;
    // 16-byte rows of A, G and dA: n runs start at multiples of four floats
    bool vec = d.N % 4 == 0 && d.sAm % 4 == 0 && d.sG1 % 4 == 0 && d.sG2 % 4 == 0 && (uintptr_t)a % 16 == 0 &&
               (uintptr_t)g % 16 == 0;
    for (int i = 0; i < d.ng; i++) vec = vec && d.g_sA[i] % 4 == 0 && d.g_sG[i] % 4 == 0;
    const float* A = (const float*)a;
    const float* F = (const float*)f;
    const float* Gp = (const float*)g;
    float* dA = (float*)da;
    float* Pp = (float*)part;
    switch (nkc) {
        case 1: return gpair_go<1>(d, vec, A, F, Gp, dA, Pp, s);
        case 2: return gpair_go<2>(d, vec, A, F, Gp, dA, Pp, s);
        case 4: return gpair_go<4>(d, vec, A, F, Gp, dA, Pp, s);
        default: return gpair_go<8>(d, vec, A, F, Gp, dA, Pp, s);
    }
}

}  // namespace ce
