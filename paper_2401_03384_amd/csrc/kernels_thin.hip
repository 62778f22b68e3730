// Thin channel mixing: C[g][m][n] = sum_k A[g][m][k] B[g][k][n] with at most
// 16 rows, 16 reduced channels and 64 products per column (the mode products
// of reshaped CP layers, Section 2.3: one factor per reshaped mode with a
// handful of channels).  There is no tile to fill, so the kernel streams B
// and C: a thread owns one column (consecutive lanes, consecutive columns of
// the flattened batch x column index, so every load and store is
// coalesced); the block first stages the factor slices of the few batch
// indices its 256 columns span in LDS, padded to MM x KK, and every thread
// reads its slice from there as float4 broadcasts.
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

constexpr int kMinN = 16;                       // columns per batch index, at least
constexpr int kSlices = 256 / kMinN + 2;        // batch indices one block can span

template <typename T, typename TC, int MM, int KK>
__global__ void __launch_bounds__(256) thin_gemm(GemmDesc d, uint32_t total, const T* __restrict__ A,
                                                 const T* __restrict__ B, TC* __restrict__ C) {
    constexpr int SL = MM * KK;
    __shared__ float4 sa4[kSlices * SL / 4];
    float* sa = reinterpret_cast<float*>(sa4);
    const uint32_t N = (uint32_t)d.N;
    const uint32_t f0 = blockIdx.x * 256u, flast = min(total - 1u, f0 + 255u);
    const uint32_t g0 = f0 / N, ns = flast / N - g0 + 1;
    // batch offsets of a flat batch index
    auto offs = [&](uint32_t g, int64_t& oA, int64_t& oB, int64_t& oC) {
        oA = oB = oC = 0;
        for (int i = d.ng - 1; i >= 0; --i) {
            const uint32_t sz = (uint32_t)d.g_size[i], x = g % sz;
            g /= sz;
            oA += x * d.g_sA[i];
            oB += x * d.g_sB[i];
            oC += x * d.g_sC[i];
        }
    };
    for (uint32_t e = threadIdx.x; e < ns * SL; e += 256) {
        const uint32_t sl = e / SL, q = e - sl * SL, m = q / KK, k = q - m * KK;
        float v = 0.f;
        if (m < (uint32_t)d.M && k < (uint32_t)d.K) {
            int64_t oA, oB, oC;
            offs(g0 + sl, oA, oB, oC);
            v = load(A, oA + (int64_t)m * d.sAm + (int64_t)k * d.sAk);
        }
        sa[e] = v;
    }
    __syncthreads();
    const uint32_t f = f0 + threadIdx.x;
    if (f >= total) return;
    const uint32_t g = f / N, n = f - g * N;
    int64_t oA, oB, oC;
    offs(g, oA, oB, oC);
    float b[KK];
#pragma unroll
    for (int k = 0; k < KK; k++) b[k] = k < d.K ? load(B, oB + (int64_t)k * d.sBk + n) : 0.f;
    const float4* a4 = sa4 + (g - g0) * (SL / 4);
#pragma unroll
    for (int m = 0; m < MM; m++) {
        if (m >= d.M) break;
        float acc = 0.f;
#pragma unroll
        for (int k4 = 0; k4 < KK / 4; k4++) {
            const float4 a = a4[m * (KK / 4) + k4];
            acc += a.x * b[4 * k4] + a.y * b[4 * k4 + 1] + a.z * b[4 * k4 + 2] + a.w * b[4 * k4 + 3];
        }
        store(C, oC + (int64_t)m * d.sCm + n, acc);
    }
}

template <typename T, typename TC>
hipError_t thin_t(const GemmDesc& d, dim3 grid, const void* a, const void* b, void* c, hipStream_t s) {
    int64_t G = 1;
    for (int i = 0; i < d.ng; i++) G *= d.g_size[i];
    if (d.N < kMinN || G * d.N >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    const uint32_t total = (uint32_t)(G * d.N);
    const int MM = d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16, KK = d.K <= 4 ? 4 : d.K <= 8 ? 8 : 16;
    const T* A = (const T*)a;
    const T* B = (const T*)b;
    TC* C = (TC*)c;
    dim3 bl(256);
#define THIN(m, k) \
    if (MM == m && KK == k) { hipLaunchKernelGGL((thin_gemm<T, TC, m, k>), grid, bl, 0, s, d, total, A, B, C); return hipGetLastError(); }
    THIN(4, 4) THIN(4, 8) THIN(4, 16) THIN(8, 4) THIN(8, 8) THIN(16, 4)
#undef THIN
    return hipErrorInvalidValue;
}

// ---- small-output contraction over a long reduction ------------------------
// C[g][m][n] = sum_k P[g][m][k] Q[g][n][k] (ThinwDesc).  Consecutive lanes
// take consecutive elements of the contiguous inner run (coalesced loads of
// MM rows of P and NN rows of Q each); every thread keeps the MM x NN
// products in registers; the block's outer-index offsets come from an LDS
// table; at the end a wave-shuffle and a fixed-order LDS sum give one
// partial per block.
constexpr int kOrowsMax = 512;   // outer indices per block (LDS offset table)

template <typename T, int MM, int NN>
__global__ void __launch_bounds__(256) thinw(ThinwDesc d, const T* __restrict__ P, const T* __restrict__ Q,
                                             float* __restrict__ part) {
    __shared__ int64_t offP[kOrowsMax], offQ[kOrowsMax];
    __shared__ float wsum[4][MM * NN];
    const int tid = threadIdx.x;
    const int64_t g = blockIdx.x / d.kchunks, kc = blockIdx.x - g * d.kchunks;
    const int64_t oa = kc * d.orows, ob = min(d.Kout, oa + d.orows);
    const int rows = (int)(ob - oa);
    for (int q = tid; q < rows; q += 256) {
        int64_t o = oa + q, sp = 0, sq = 0;
        for (int i = d.no - 1; i >= 0; --i) {
            const int64_t x = o % d.o_size[i];
            o /= d.o_size[i];
            sp += x * d.o_sP[i];
            sq += x * d.o_sQ[i];
        }
        offP[q] = sp;
        offQ[q] = sq;
    }
    int64_t gP = 0, gQ = 0;
    {
        int64_t x = g;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t y = x % d.g_size[i];
            x /= d.g_size[i];
            gP += y * d.g_sP[i];
            gQ += y * d.g_sQ[i];
        }
    }
    __syncthreads();
    float acc[MM][NN];
#pragma unroll
    for (int m = 0; m < MM; m++)
#pragma unroll
        for (int n = 0; n < NN; n++) acc[m][n] = 0.f;
    const uint32_t Kin = (uint32_t)d.Kin, total = (uint32_t)rows * Kin;
    const uint32_t so = 256u / Kin, si = 256u % Kin;
    uint32_t o = (uint32_t)tid / Kin, i = (uint32_t)tid % Kin;
    for (uint32_t e = tid; e < total; e += 256) {
        const T* p = P + gP + offP[o] + i;
        const T* q = Q + gQ + offQ[o] + i;
        float a[MM], b[NN];
#pragma unroll
        for (int m = 0; m < MM; m++) a[m] = m < d.M ? load(p, m * d.sPm) : 0.f;
#pragma unroll
        for (int n = 0; n < NN; n++) b[n] = n < d.N ? load(q, n * d.sQn) : 0.f;
#pragma unroll
        for (int m = 0; m < MM; m++)
#pragma unroll
            for (int n = 0; n < NN; n++) acc[m][n] += a[m] * b[n];
        i += si;
        o += so;
        if (i >= Kin) {
            i -= Kin;
            o++;
        }
    }
    // wave sums, then the four waves in order
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
#pragma unroll
    for (int m = 0; m < MM; m++)
#pragma unroll
        for (int n = 0; n < NN; n++) {
            float v = acc[m][n];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
            if (lane == 0) wsum[wave][m * NN + n] = v;
        }
    __syncthreads();
    if (tid < MM * NN) {
        const float v = (wsum[0][tid] + wsum[1][tid]) + (wsum[2][tid] + wsum[3][tid]);
        part[blockIdx.x * (int64_t)(MM * NN) + tid] = v;
    }
}

// C[g][m][n] = sum over the chunks of the partials, in chunk order
template <typename TC, int MM, int NN>
__global__ void __launch_bounds__(256) thinw_reduce(ThinwDesc d, const float* __restrict__ part,
                                                    TC* __restrict__ C) {
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= d.G * d.M * d.N) return;
    const int64_t g = t / (d.M * d.N), r = t - g * d.M * d.N, m = r / d.N, n = r - m * d.N;
    float s = 0.f;
    for (int64_t kc = 0; kc < d.kchunks; kc++) s += part[(g * d.kchunks + kc) * (MM * NN) + m * NN + n];
    int64_t off = m * d.sCm + n * d.sCn, x = g;
    for (int i = d.ng - 1; i >= 0; --i) {
        off += (x % d.g_size[i]) * d.g_sC[i];
        x /= d.g_size[i];
    }
    store(C, off, s);
}

template <typename T, typename TC>
hipError_t thinw_t(const Launch& ln, const ThinwDesc& d, const void* p, const void* q, void* part, void* c,
                   hipStream_t s) {
    const bool red = (ln.kind & 0xff) == K_THINW_REDUCE;
    const int MM = d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16, NN = d.N <= 4 ? 4 : d.N <= 8 ? 8 : 16;
    if (d.orows > kOrowsMax || d.orows * d.Kin >= ((int64_t)1 << 31) || d.Kin < 1) return hipErrorInvalidValue;
    dim3 g(ln.grid[0]), bl(256);
#define THINW(m, n) \
    if (MM == m && NN == n) { \
        if (red) hipLaunchKernelGGL((thinw_reduce<TC, m, n>), g, bl, 0, s, d, (const float*)part, (TC*)c); \
        else hipLaunchKernelGGL((thinw<T, m, n>), g, bl, 0, s, d, (const T*)p, (const T*)q, (float*)part); \
        return hipGetLastError(); }
    THINW(4, 4) THINW(4, 8) THINW(4, 16) THINW(8, 4) THINW(8, 8) THINW(16, 4)
#undef THINW
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_thin(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s) {
    GemmDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    dim3 g(ln.grid[0]);
    if (tIn) return tC ? thin_t<bf16_t, bf16_t>(d, g, a, b, c, s) : thin_t<bf16_t, float>(d, g, a, b, c, s);
    return tC ? thin_t<float, bf16_t>(d, g, a, b, c, s) : thin_t<float, float>(d, g, a, b, c, s);
}

hipError_t launch_thinw(const Launch& ln, const void* p, const void* q, void* part, void* c, hipStream_t s) {
    ThinwDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    if (tIn) return tC ? thinw_t<bf16_t, bf16_t>(ln, d, p, q, part, c, s) : thinw_t<bf16_t, float>(ln, d, p, q, part, c, s);
    return tC ? thinw_t<float, bf16_t>(ln, d, p, q, part, c, s) : thinw_t<float, float>(ln, d, p, q, part, c, s);
}

}  // namespace ce
