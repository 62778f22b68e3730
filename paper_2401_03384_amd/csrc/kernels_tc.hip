// General contraction on MFMA tiles (see TcDesc): the pairwise steps that no
// specialised kernel matches -- convolutions that also contract channels
// (Section 3.1: contraction and convolution in one step), their feature- and
// filter-side gradients, and channel products whose labels interleave in
// memory.
//
// A block computes a 32*MT x 128 tile of C for one batch index g.  The index
// maps of the tile's rows (m), columns (n) and of each 32-wide slice of the
// reduction (k) are decoded once into LDS offset tables; the A and B slices
// are then gathered through those tables (coalesced along n when n is
// unit-stride in B) and multiplied on 32x32 MFMA tiles (fp32: 32x32x2, bf16:
// 32x32x16).  Positions of convolved labels outside [0, lim) read zero.
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

__device__ __forceinline__ int row32(int i, int lane) { return 8 * (i >> 2) + 4 * ((lane >> 5) & 1) + (i & 3); }

__device__ __forceinline__ bf16x8 ld8(const bf16_t* p) {
    bf16x8 v;
    __builtin_memcpy(&v, p, 16);
    return v;
}

template <typename T, typename TC, int MT>
__global__ void __launch_bounds__(256) tc_gemm(TcDesc d, const T* __restrict__ A, const T* __restrict__ B,
                                               TC* __restrict__ C, float* __restrict__ P) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int TM = 32 * MT, TN = 128, TK = 32;
    constexpr int LA = BF ? TK + 8 : TK + 1;      // A tile row pitch
    constexpr int LB = BF ? TK + 8 : TN + 4;      // B tile pitch ([n][k] for bf16, [k][n] for fp32)
    __shared__ __attribute__((aligned(16))) T As[TM * LA];
    __shared__ __attribute__((aligned(16))) T Bs[BF ? TN * LB : TK * LB];
    __shared__ int64_t mA[TM], mC[TM], nB[TN], nC[TN], kA[TK], kB[TK];
    __shared__ int32_t np[2][TN], kj[2][TK];
    __shared__ unsigned char mok[TM], nok[TN], kok[TK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, cl = lane & 31, hf = lane >> 5;
    int64_t bid = blockIdx.x;
    const int nt = (int)(bid % d.ntiles);
    bid /= d.ntiles;
    const int mt = (int)(bid % d.mtiles);
    bid /= d.mtiles;
    const int ks = (int)(bid % d.ksplit);
    const int64_t g = bid / d.ksplit;
    const int64_t m0 = (int64_t)mt * TM, n0 = (int64_t)nt * TN;

    int64_t gA = 0, gB = 0, gC = 0;
    {
        int64_t x = g;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t c = x % d.g_size[i];
            x /= d.g_size[i];
            gA += c * d.g_sA[i];
            gB += c * d.g_sB[i];
            gC += c * d.g_sC[i];
        }
    }
    if (tid < TM) {
        const int64_t m = m0 + tid;
        int64_t x = m, oa = 0, oc = 0;
        for (int i = d.nm - 1; i >= 0; --i) {
            const int64_t c = x % d.m_size[i];
            x /= d.m_size[i];
            oa += c * d.m_sA[i];
            oc += c * d.m_sC[i];
        }
        mA[tid] = oa;
        mC[tid] = oc;
        mok[tid] = m < d.M;
    } else if (tid >= 128 && tid < 128 + TN) {
        const int t = tid - 128;
        const int64_t n = n0 + t;
        int64_t x = n, ob = 0, oc = 0;
        np[0][t] = np[1][t] = 0;
        for (int i = d.nn - 1; i >= 0; --i) {
            const int64_t c = x % d.n_size[i];
            x /= d.n_size[i];
            ob += c * d.n_sB[i];
            oc += c * d.n_sC[i];
            if (d.n_cv[i] >= 0) np[d.n_cv[i]][t] = (int32_t)c;
        }
        nB[t] = ob;
        nC[t] = oc;
        nok[t] = n < d.N;
    }

    f32x16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.f;

    const int64_t kb = (int64_t)ks * d.kchunk;
    const int64_t ke = min(d.K, kb + d.kchunk);
    for (int64_t k0 = kb; k0 < ke; k0 += TK) {
        __syncthreads();   // previous slice consumed; m / n tables written
        if (tid < TK) {
            const int64_t k = k0 + tid;
            int64_t x = k, oa = 0, ob = 0;
            kj[0][tid] = kj[1][tid] = 0;
            for (int i = d.nk - 1; i >= 0; --i) {
                const int64_t c = x % d.k_size[i];
                x /= d.k_size[i];
                oa += c * d.k_sA[i];
                ob += c * d.k_sB[i];
                if (d.k_cv[i] >= 0) kj[d.k_cv[i]][tid] = (int32_t)c;
            }
            kA[tid] = oa;
            kB[tid] = ob;
            kok[tid] = k < ke;
        }
        __syncthreads();
        for (int e = tid; e < TM * TK; e += 256) {
            const int mm = e / TK, kk = e - mm * TK;
            As[mm * LA + kk] = (mok[mm] && kok[kk]) ? A[gA + mA[mm] + kA[kk]] : (T)0;
        }
#pragma unroll 4
        for (int e = tid; e < TK * TN; e += 256) {
            const int kk = e / TN, nn = e - kk * TN;
            bool ok = kok[kk] && nok[nn];
            int64_t off = gB + kB[kk] + nB[nn];
            for (int c = 0; c < d.ncv; c++) {
                const int64_t pos = (int64_t)d.cv_a[c] * np[c][nn] + (int64_t)d.cv_b[c] * kj[c][kk] + d.cv_g[c];
                ok = ok && pos >= 0 && pos < d.cv_lim[c];
                off += pos * d.cv_s[c];
            }
            const T v = ok ? B[off] : (T)0;
            if constexpr (BF) Bs[nn * LB + kk] = v;
            else Bs[kk * LB + nn] = v;
        }
        __syncthreads();
        if constexpr (BF) {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 16) {
                const bf16x8 b = ld8(&Bs[(wave * 32 + cl) * LB + kk + 8 * hf]);
#pragma unroll
                for (int i = 0; i < MT; i++)
                    acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(&As[(i * 32 + cl) * LA + kk + 8 * hf]), b,
                                                                     acc[i], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 2) {
                const float b = Bs[(kk + hf) * LB + wave * 32 + cl];
#pragma unroll
                for (int i = 0; i < MT; i++)
                    acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(As[(i * 32 + cl) * LA + kk + hf], b, acc[i], 0, 0, 0);
            }
        }
    }
    // results (the MFMA results are read after the loop's barrier-free tail;
    // pad so every path has the wait states before the first read)
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    const int tn = wave * 32 + cl;
    if (!nok[tn]) return;
    const int64_t n = n0 + tn;
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const int mm = i * 32 + row32(r, lane);
            if (!mok[mm]) continue;
            if (d.ksplit == 1) store(C, gC + mC[mm] + nC[tn], acc[i][r]);
            else P[((g * d.ksplit + ks) * d.M + (m0 + mm)) * d.N + n] = acc[i][r];
        }
}

// C[g][m][n] = sum over chunks (in order) of P[g][chunk][m][n], in double.
template <typename TC>
__global__ void __launch_bounds__(256) tc_reduce(TcDesc d, const float* __restrict__ P, TC* __restrict__ C) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t MN = d.M * d.N;
    if (e >= d.G * MN) return;
    const int64_t g = e / MN, mn = e - g * MN, m = mn / d.N, n = mn - m * d.N;
    int64_t off = 0, x = g;
    for (int i = d.ng - 1; i >= 0; --i) {
        off += (x % d.g_size[i]) * d.g_sC[i];
        x /= d.g_size[i];
    }
    x = m;
    for (int i = d.nm - 1; i >= 0; --i) {
        off += (x % d.m_size[i]) * d.m_sC[i];
        x /= d.m_size[i];
    }
    x = n;
    for (int i = d.nn - 1; i >= 0; --i) {
        off += (x % d.n_size[i]) * d.n_sC[i];
        x /= d.n_size[i];
    }
    double s = 0.0;
    const float* p = P + g * d.ksplit * MN + mn;
    for (int c = 0; c < d.ksplit; c++) s += (double)p[c * MN];
    store(C, off, (float)s);
}

template <typename T, typename TC>
hipError_t tc_launch_t(const TcDesc& d, const Launch& ln, const void* a, const void* b, void* c, void* p,
                       hipStream_t s) {
    const int MT = d.M > 32 ? 2 : 1;
    dim3 g(ln.grid[0]), bl(256);
    if (MT == 2)
        hipLaunchKernelGGL((tc_gemm<T, TC, 2>), g, bl, 0, s, d, (const T*)a, (const T*)b, (TC*)c, (float*)p);
    else
        hipLaunchKernelGGL((tc_gemm<T, TC, 1>), g, bl, 0, s, d, (const T*)a, (const T*)b, (TC*)c, (float*)p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_tc(const Launch& ln, const void* a, const void* b, void* c, void* d, hipStream_t s) {
    TcDesc t;
    std::memcpy(&t, ln.desc.data(), sizeof(t));
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    if ((ln.kind & 0xff) == K_TC_REDUCE) {
        dim3 g(ln.grid[0]), bl(256);
        if (tC) hipLaunchKernelGGL((tc_reduce<bf16_t>), g, bl, 0, s, t, (const float*)d, (bf16_t*)c);
        else hipLaunchKernelGGL((tc_reduce<float>), g, bl, 0, s, t, (const float*)d, (float*)c);
        return hipGetLastError();
    }
    if (tIn) return tC ? tc_launch_t<bf16_t, bf16_t>(t, ln, a, b, c, d, s) : tc_launch_t<bf16_t, float>(t, ln, a, b, c, d, s);
    return tC ? tc_launch_t<float, bf16_t>(t, ln, a, b, c, d, s) : tc_launch_t<float, float>(t, ln, a, b, c, d, s);
}

}  // namespace ce
