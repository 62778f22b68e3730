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
// A block: sixteen wavefronts (four a SIMD), gper consecutive g, every n in
// tiles of 64, k in NKC chunks of 64.  Wavefronts 0-7 compute dA, 8-15 dF;
// within each half w = (mt, q): mt = w / 4 the m tile (16 rows of m; M <= 32),
// q = w % 4.  Per chunk a wavefront computes
//   dA:  the tile (m tile mt, n columns 16q..16q+15): A operand F[k][m], B
//        operand G[k][n], k = 4s + kq at k step s (lane kq = lane / 16);
//   dF:  the tile (k rows 16q.. of the chunk, m tile mt): A operand G[k][n],
//        B operand A[m][n], reduced over the tile's 64 n with n = 16 kq + s at
//        step s (a lane's sixteen n are contiguous: four 16-byte LDS reads);
//        one accumulator tile per chunk, kept for the whole block and written
//        as the block's partial at the end.
// F is staged once per block; chunk c + 2 of G (and, at a new n tile, its A
// tile) loads into registers while chunk c computes; G and A tiles are
// double-buffered in LDS, one barrier a chunk.
//
// LDS layouts (bank = word mod 32; 4-byte reads are served a half-wavefront,
// lanes (i16, kq < 2) or (i16, kq >= 2), at a time, 16-byte reads eight
// lanes at a time): the G chunk is read along k by the dA tile (row 4s + kq,
// column 16q + i16, 4 bytes) and along n by the dF tile (row 16q + i16,
// columns 16 kq .. + 15, 16 bytes); row r starts at 96 r + 16 (r & 1) +
// 4 ((r >> 1) & 3), so that both cover the banks without conflicts.  F is
// stored as each lane reads it, [m][kc][kq][s] = F[64 kc + 4s + kq][m] (m pitch
// 64 NKC + 4), the A tile [m][n] with pitch 68 (read once a tile).
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

constexpr int kGpLG = 96;   // row pitch of the G chunk (row r at 96 r + skew(r))
constexpr int kGpLA = 68;   // pitch of the A tile [m][n]

__device__ __forceinline__ int gp_skew(int r) { return 16 * (r & 1) + 4 * ((r >> 1) & 3); }
__host__ __device__ constexpr int gp_lf(int nkc) { return 64 * nkc + 4; }   // m pitch of F in LDS

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
__global__ void __launch_bounds__(1024, 1) gpair(GpairDesc d, const float* __restrict__ A,
                                                const float* __restrict__ F, const float* __restrict__ G,
                                                float* __restrict__ dA, float* __restrict__ P) {
    extern __shared__ float4 lds4[];
    constexpr int LF = gp_lf(NKC);
    float* Fs = reinterpret_cast<float*>(lds4);               // [32][LF]
    float* Gs = Fs + 32 * LF;                                 // [2][64 kGpLG]
    float* As = Gs + 2 * 64 * kGpLG;                          // [2][32][kGpLA]
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool is_df = wave >= 8;   // wave-uniform role
    const int mt = (wave & 7) >> 2, q = wave & 3, i16 = lane & 15, kq = lane >> 4;
    const int M = d.M, K = d.K, N = d.N;
    const int64_t g0 = (int64_t)blockIdx.x * d.gper, g1 = min(d.G, g0 + d.gper);
    const bool want_da = dA != nullptr;

    // ---- F, once per block: Fs[k][m] (zero past K and M) ----
    for (int e = tid; e < NKC * 64 * 32; e += 1024) {
        // e = (m, kc, kq, s): k = 64 kc + 4s + kq
        const int m = e / (64 * NKC), rest = e - m * (64 * NKC), kc = rest >> 6, kq4 = (rest >> 4) & 3, st = rest & 15;
        const int k = 64 * kc + 4 * st + kq4;
        float v = 0.f;
        if (k < K && m < M) {
            const int k1 = k / d.K2, k2 = k - k1 * d.K2;
            v = F[k1 * d.sF1 + k2 * d.sF2 + m * d.sFm];
        }
        Fs[m * LF + rest] = v;
    }

    // ---- staging: the G chunk (one float4 of a row a thread) and the A tile
    // (one float4 a thread of the first 512); rows / columns past the ends are zero ----
    // branch-free loads (raw buffer loads over one g's slice: an offset past
    // it reads 0), so that the compiler counts the loads in flight exactly and
    // waits only for the chunk it stores
    constexpr int kOut = (int)0x80000000u;
    auto ld4 = [&](__amdgpu_buffer_rsrc_t r, int e, bool ok, int nleft) {
        if constexpr (VEC) {
            return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, ok ? 4 * e : kOut, 0, 0));
        } else {
            float t[4];
#pragma unroll
            for (int j = 0; j < 4; j++)
                t[j] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, ok && j < nleft ? 4 * (e + j) : kOut, 0, 0));
            return make_float4(t[0], t[1], t[2], t[3]);
        }
    };
    const int gr = tid >> 4, gc = 4 * (tid & 15);   // this thread's row and columns of a G chunk
    auto g_load = [&](int64_t og, int kc, int n0, float4& v) {
        const __amdgpu_buffer_rsrc_t rG =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(G + og), (short)0, (int)(4 * d.gext), 0x00020000);
        const int k = 64 * kc + gr, n = n0 + gc;
        const int k1 = k / d.K2, k2 = k - k1 * d.K2;
        v = ld4(rG, (int)(k1 * d.sG1 + k2 * d.sG2) + n, k < K && n < N, N - n);
    };
    auto g_store = [&](int buf, const float4& v) {
        *reinterpret_cast<float4*>(Gs + buf * 64 * kGpLG + gr * kGpLG + gp_skew(gr) + gc) = v;
    };
    auto a_load = [&](int64_t oa, int n0, float4& v) {
        const __amdgpu_buffer_rsrc_t rA =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(A + oa), (short)0, (int)(4 * d.aext), 0x00020000);
        const int m = tid >> 4, c = 4 * (tid & 15), n = n0 + c;
        v = ld4(rA, (int)(m * d.sAm) + n, m < M && n < N, N - n);
    };
    auto a_store = [&](int buf, const float4& v) {
        const int m = tid >> 4, c = 4 * (tid & 15);
        if (wave < 8) *reinterpret_cast<float4*>(As + (buf * 32 + m) * kGpLA + c) = v;   // rows m < 32
    };

    f32x4 accF[NKC];
#pragma unroll
    for (int kc = 0; kc < NKC; kc++) accF[kc] = (f32x4){0.f, 0.f, 0.f, 0.f};

    // The block's work is a sequence of tiles t = (g - g0) ntiles + nt, each of
    // NKC chunks; chunk c = t NKC + kc.  Chunk c + 2 loads into register set
    // c & 1 while chunk c computes (two chunks of cover for the loads), chunk
    // c + 1 goes from register set (c + 1) & 1 into G buffer (c + 1) & 1 at the
    // end of chunk c; the A tile of tile t + 1 loads with its first chunk and
    // goes to A buffer (t + 1) & 1.  Tiles run in pairs when NKC is odd, so
    // that the register set of every chunk is known at compile time.
    constexpr int TU = (NKC & 1) ? 2 : 1;
    const int64_t ntl = (g1 - g0) * d.ntiles;
    auto tile_src = [&](int64_t t, int64_t& oa, int64_t& og, int64_t& od, int& n0) {
        const int64_t gg = t / d.ntiles;
        n0 = 64 * (int)(t - gg * d.ntiles);
        gp_offs(d, g0 + gg, oa, og, od);
    };
    float4 gv[2], av[2];
    // chunks 0 and 1: chunk 0 into the LDS buffers, chunk 1 into register set 1
    if (ntl > 0) {
        int64_t oa, og, od;
        int n0;
        tile_src(0, oa, og, od, n0);
        g_load(og, 0, n0, gv[0]);
        a_load(oa, n0, av[0]);
        g_store(0, gv[0]);
        a_store(0, av[0]);
        const int64_t t1 = NKC > 1 ? 0 : 1;
        if (t1 < ntl) {
            if (t1 != 0) tile_src(t1, oa, og, od, n0);
            g_load(og, NKC > 1 ? 1 : 0, n0, gv[1]);
            if (NKC == 1) a_load(oa, n0, av[1]);
        }
    }
    __syncthreads();

    // lane-constant parts of the LDS reads (the k step s adds a constant):
    //   dA, F:  [16 mt + i16][kc][kq][s]
    //   dA, G:  row 4s + kq, column 16q + i16: 96 (4s + kq) + skew(4s + kq) + 16q + i16
    //           = [96 kq + 16 (kq & 1) + 4 (kq >> 1) + 16q + i16] + [384 s + 8 (s & 1)]
    //   dF, G:  row 16q + i16, columns 16 kq + s: 96 (16q + i16) + skew(i16) + 16 kq + s
    //   dF, A:  row 16 mt + i16, columns 16 kq + s
    const int fA = (16 * mt + i16) * LF + 16 * kq;
    const int gA = kq * kGpLG + 16 * (kq & 1) + 4 * (kq >> 1) + 16 * q + i16;
    const int gF = (16 * q + i16) * kGpLG + gp_skew(i16) + 16 * kq;
    const int aF = (16 * mt + i16) * kGpLA + 16 * kq;
    for (int64_t tb = 0; tb < ntl; tb += TU) {
#pragma unroll
        for (int u = 0; u < TU; u++) {
            const int64_t t = tb + u;
            if (t >= ntl) break;
            int64_t oa, og, od;
            int n0;
            tile_src(t, oa, og, od, n0);
            // the sources of tiles t + 1 and (NKC = 1) t + 2, for the prefetches
            int64_t oa1 = 0, og1 = 0, oa2 = 0, og2 = 0, odx;
            int n01 = 0, n02 = 0;
            if (t + 1 < ntl) tile_src(t + 1, oa1, og1, odx, n01);
            if (NKC == 1 && t + 2 < ntl) tile_src(t + 2, oa2, og2, odx, n02);
            f32x4 accA = (f32x4){0.f, 0.f, 0.f, 0.f};
            float av16[16];   // this tile's dF B operand (the A tile), read at its first chunk
#pragma unroll
            for (int kc = 0; kc < NKC; kc++) {
                const int par = (u * NKC + kc) & 1;   // parity of chunk c (TU NKC is even)
                // chunk c + 2 into register set par
                {
                    const int ahead = (kc + 2) / NKC, kc2 = (kc + 2) % NKC;   // tiles ahead: 0, 1 or 2
                    if (t + ahead < ntl) {
                        const int64_t ogx = ahead == 0 ? og : ahead == 1 ? og1 : og2;
                        const int64_t oax = ahead == 0 ? oa : ahead == 1 ? oa1 : oa2;
                        const int n0x = ahead == 0 ? n0 : ahead == 1 ? n01 : n02;
                        g_load(ogx, kc2, n0x, gv[par]);
                        if (kc2 == 0) a_load(oax, n0x, av[par]);
                    }
                }
                const float* gs = Gs + par * 64 * kGpLG;
                if (is_df) {
                    if (kc == 0) {
                        const float4* as4 = reinterpret_cast<const float4*>(As + (int)(t & 1) * 32 * kGpLA + aF);
#pragma unroll
                        for (int j = 0; j < 4; j++) {
                            const float4 v = as4[j];
                            av16[4 * j] = v.x;
                            av16[4 * j + 1] = v.y;
                            av16[4 * j + 2] = v.z;
                            av16[4 * j + 3] = v.w;
                        }
                    }
                    // dF tile (k rows 16q.. of the chunk, m tile mt): sum over the
                    // tile's n; the G rows as 16-byte reads
                    float gf[16];
                    const float4* g4 = reinterpret_cast<const float4*>(gs + gF);
#pragma unroll
                    for (int j = 0; j < 4; j++) {
                        const float4 v = g4[j];
                        gf[4 * j] = v.x;
                        gf[4 * j + 1] = v.y;
                        gf[4 * j + 2] = v.z;
                        gf[4 * j + 3] = v.w;
                    }
#pragma unroll
                    for (int st = 0; st < 16; st++)
                        accF[kc] = __builtin_amdgcn_mfma_f32_16x16x4f32(gf[st], av16[st], accF[kc], 0, 0, 0);
                } else if (want_da) {
                    // dA tile (m tile mt, columns 16q..): sum over the chunk's k
                    float fa[16], ga[16];
                    const float4* f4 = reinterpret_cast<const float4*>(Fs + fA + 64 * kc);
#pragma unroll
                    for (int j = 0; j < 4; j++) {
                        const float4 w = f4[j];
                        fa[4 * j] = w.x;
                        fa[4 * j + 1] = w.y;
                        fa[4 * j + 2] = w.z;
                        fa[4 * j + 3] = w.w;
                    }
#pragma unroll
                    for (int st = 0; st < 16; st++) ga[st] = gs[gA + 384 * st + 8 * (st & 1)];
#pragma unroll
                    for (int st = 0; st < 16; st++)
                        accA = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[st], ga[st], accA, 0, 0, 0);
                }
                const bool last = kc + 1 == NKC;
                if (last && want_da && !is_df) {
                    // dA[g][m][n]: accumulator r = row 4 kq + r, column i16
#pragma unroll
                    for (int r = 0; r < 4; r++) {
                        const int m = 16 * mt + 4 * kq + r, n = n0 + 16 * q + i16;
                        if (m < M && n < N) dA[od + (int64_t)m * d.sDm + n] = accA[r];
                    }
                }
                // chunk c + 1 (register set 1 - par) into the other buffers
                // (their previous readers passed the barrier of chunk c - 1)
                if (!last || t + 1 < ntl) {
                    g_store(1 - par, gv[1 - par]);
                    if (last) a_store((int)((t + 1) & 1), av[1 - par]);
                }
                __syncthreads();
            }
        }
    }

    // the block's partial of dF, in F's layout: accumulator r = k row 4 kq + r
    // of tile q of chunk kc, column i16 = m
    float* pb = P + (int64_t)blockIdx.x * d.fnumel;
    if (is_df)
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
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(1024), d.lds_bytes, s, d, a, f, g, da, part);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gpair(const Launch& ln, const void* a, const void* f, const void* g, void* da, void* part,
                        hipStream_t s) {
    GpairDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int nkc = d.nkc;
    const uint32_t lds = (uint32_t)(4 * (32 * gp_lf(nkc) + 2 * 64 * kGpLG + 2 * 32 * kGpLA));
    // the shapes the kernel assumes (the lowering guarantees them)
    if (((ln.kind >> kBitIn) & 1) || d.M < 1 || d.M > 32 || d.K < 1 || d.K2 < 1 || d.K1 * d.K2 != d.K ||
        (nkc != 1 && nkc != 2 && nkc != 4 && nkc != 8) || d.K > 64 * nkc || d.N < 1 ||
        d.ntiles != (d.N + 63) / 64 || d.gper < 1 || d.blocks != (d.G + d.gper - 1) / d.gper ||
        d.lds_bytes != lds || ln.grid[0] != (uint32_t)d.blocks || ln.block[0] != 1024 || !a || !f || !g || !part ||
        d.gext != (int64_t)(d.K1 - 1) * d.sG1 + (int64_t)(d.K2 - 1) * d.sG2 + d.N || d.gext * 4 >= (1ll << 31) ||
        d.aext != (int64_t)(d.M - 1) * d.sAm + d.N || d.aext * 4 >= (1ll << 31) || d.sG1 < 0 || d.sG2 < 0 ||
        d.sAm < 0)
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
