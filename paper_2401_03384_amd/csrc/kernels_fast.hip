// Specialised kernels for the pairwise steps of tensorial convolution layers
// on gfx950 (wave64, MFMA, 160 KB LDS per CU).
//
//  gemm_f32 / gemm_bf16   channel mixing C[g][m][n] = sum_k A[m][k] B[g][k][n]:
//                         the factor A is staged in LDS, the activation B
//                         streams through LDS in coalesced 16-byte rows, the
//                         product runs on 32x32 MFMA tiles (fp32: 32x32x2,
//                         bf16: 32x32x16), results go straight from the
//                         accumulators to HBM with unit-stride rows.
//  wgrad                  factor gradients sum_{kb,k} A[kb][m][k] B[kb][n][k]:
//                         each block reduces one chunk of the long unit-stride
//                         reduction into a 64x64 partial tile.
//  reduce_partials        ordered (deterministic) sum of the partial tiles.
//  dw_conv                depthwise convolution along one axis (forward, or
//                         transposed for the feature gradient): whole lines
//                         of the axis are staged in LDS, taps in registers.
//  dw_tapgrad / reduce    filter-tap gradients: per-block partial sums, then
//                         an ordered reduction over the blocks of each row.
#include <atomic>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

__device__ __forceinline__ bf16x8 lds_bf16x8(const bf16_t* p) {
    bf16x8 v;
    __builtin_memcpy(&v, p, 16);
    return v;
}

// Row of the 32x32 MFMA result held by accumulator r of a lane.
__device__ __forceinline__ int mfma32_row(int r, int lane) {
    return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

// ---------------------------------------------------------------------------
// channel-mixing GEMM
// ---------------------------------------------------------------------------
__device__ __forceinline__ void gemm_offsets(const GemmDesc& d, int64_t g, int64_t& oA,
                                             int64_t& oB, int64_t& oC) {
    oA = oB = oC = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        int64_t x = g % d.g_size[i];
        g /= d.g_size[i];
        oA += x * d.g_sA[i];
        oB += x * d.g_sB[i];
        oC += x * d.g_sC[i];
    }
}

template <typename TC, int MT, bool VEC>
__global__ void __launch_bounds__(256) gemm_f32(GemmDesc d, const float* __restrict__ A,
                                                const float* __restrict__ B,
                                                TC* __restrict__ C) {
    constexpr int TM = 32 * MT, TN = 128, TK = 32;
    __shared__ float As[TM][TK + 1];
    __shared__ __attribute__((aligned(16))) float Bs[TK][TN + 4];
    int64_t bid = blockIdx.x;
    const int nt = (int)(bid % d.ntiles);
    bid /= d.ntiles;
    const int mt = (int)(bid % d.mtiles);
    bid /= d.mtiles;
    int64_t oA, oB, oC;
    gemm_offsets(d, bid, oA, oB, oC);
    const int m0 = mt * TM, n0 = nt * TN;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    f32x16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.f;

    for (int k0 = 0; k0 < d.K; k0 += TK) {
        for (int e = tid; e < TM * TK; e += 256) {
            int mm = e / TK, kk = e % TK, m = m0 + mm, k = k0 + kk;
            As[mm][kk] = (m < d.M && k < d.K) ? A[oA + (int64_t)m * d.sAm + (int64_t)k * d.sAk] : 0.f;
        }
#pragma unroll
        for (int it = 0; it < TK * TN / 4 / 256; it++) {
            int e = tid + it * 256;
            int kk = e / (TN / 4), nn = (e % (TN / 4)) * 4, k = k0 + kk, n = n0 + nn;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (k < d.K) {
                const float* p = B + oB + (int64_t)k * d.sBk + n;
                if (VEC && n + 3 < d.N) {
                    v = *(const f32x4*)p;
                } else {
#pragma unroll
                    for (int j = 0; j < 4; j++)
                        if (n + j < d.N) v[j] = p[j];
                }
            }
            *(f32x4*)&Bs[kk][nn] = v;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; kk += 2) {
            float b = Bs[kk + (lane >> 5)][wave * 32 + (lane & 31)];
#pragma unroll
            for (int i = 0; i < MT; i++) {
                float a = As[i * 32 + (lane & 31)][kk + (lane >> 5)];
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[i], 0, 0, 0);
            }
        }
        __syncthreads();
    }
    const int n = n0 + wave * 32 + (lane & 31);
    if (n >= d.N) return;
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
            int m = m0 + i * 32 + mfma32_row(r, lane);
            if (m < d.M) store(C, oC + (int64_t)m * d.sCm + n, acc[i][r]);
        }
}

template <typename TC, int MT, bool VEC>
__global__ void __launch_bounds__(256) gemm_bf16(GemmDesc d, const bf16_t* __restrict__ A,
                                                 const bf16_t* __restrict__ B,
                                                 TC* __restrict__ C) {
    constexpr int TM = 32 * MT, TN = 128, TK = 32, LDK = TK + 8;
    __shared__ __attribute__((aligned(16))) bf16_t As[TM][LDK];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[TN][LDK];   // transposed: [n][k]
    int64_t bid = blockIdx.x;
    const int nt = (int)(bid % d.ntiles);
    bid /= d.ntiles;
    const int mt = (int)(bid % d.mtiles);
    bid /= d.mtiles;
    int64_t oA, oB, oC;
    gemm_offsets(d, bid, oA, oB, oC);
    const int m0 = mt * TM, n0 = nt * TN;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    f32x16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.f;

    const int nn = (tid & 31) * 4, kq = (tid >> 5) * 4;
    for (int k0 = 0; k0 < d.K; k0 += TK) {
        for (int e = tid; e < TM * TK; e += 256) {
            int mm = e / TK, kk = e % TK, m = m0 + mm, k = k0 + kk;
            As[mm][kk] = (m < d.M && k < d.K) ? A[oA + (int64_t)m * d.sAm + (int64_t)k * d.sAk]
                                              : (bf16_t)0;
        }
        // 4 k-rows x 4 n-columns per thread, written transposed as 4-element k-runs
        bf16_t v[4][4];
        const int n = n0 + nn;
#pragma unroll
        for (int r = 0; r < 4; r++) {
            int k = k0 + kq + r;
#pragma unroll
            for (int j = 0; j < 4; j++) v[r][j] = 0;
            if (k < d.K) {
                const bf16_t* p = B + oB + (int64_t)k * d.sBk + n;
                if (VEC && n + 3 < d.N) {
                    uint2 raw = *(const uint2*)p;
                    v[r][0] = (bf16_t)(raw.x & 0xffff);
                    v[r][1] = (bf16_t)(raw.x >> 16);
                    v[r][2] = (bf16_t)(raw.y & 0xffff);
                    v[r][3] = (bf16_t)(raw.y >> 16);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; j++)
                        if (n + j < d.N) v[r][j] = p[j];
                }
            }
        }
#pragma unroll
        for (int j = 0; j < 4; j++) {
            uint2 w;
            w.x = (uint32_t)v[0][j] | ((uint32_t)v[1][j] << 16);
            w.y = (uint32_t)v[2][j] | ((uint32_t)v[3][j] << 16);
            *(uint2*)&Bs[nn + j][kq] = w;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; kk += 16) {
            bf16x8 b = lds_bf16x8(&Bs[wave * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
#pragma unroll
            for (int i = 0; i < MT; i++) {
                bf16x8 a = lds_bf16x8(&As[i * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
            }
        }
        __syncthreads();
    }
    const int n = n0 + wave * 32 + (lane & 31);
    if (n >= d.N) return;
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
            int m = m0 + i * 32 + mfma32_row(r, lane);
            if (m < d.M) store(C, oC + (int64_t)m * d.sCm + n, acc[i][r]);
        }
}

// The same channel mix in bf16 over flattened columns f = g * N + n (N a
// multiple of 4, rows of B and C 8-byte aligned), so that small planes fill
// whole 128-column tiles: a block takes TM rows x 128 columns, a wavefront one
// 32-column MFMA tile.  K goes in chunks of TK (64, or 256 when K <= 256, so
// that a block makes one memory round trip); the next chunk's elements load
// into registers while the current chunk's MFMAs run (one LDS copy, two
// barriers a chunk).  Thread mapping: B, four consecutive columns 4(tid / 8)
// (one 8-byte row piece) x k rows 4(tid % 8) + 32 h + {0..3}, transposed into
// LDS rows [n][k] by byte permutes; A, TM x TK / 256 consecutive k of one row.
template <typename TC, int MT, int TK>
__global__ void __launch_bounds__(256) gemm_bf16f(GemmDesc d, const bf16_t* __restrict__ A,
                                                  const bf16_t* __restrict__ B, TC* __restrict__ C) {
    constexpr int TM = 32 * MT, TN = 128, LDK = TK + 8, KH = TK / 32;
    constexpr int AE = TM * TK / 256;   // A elements a thread
    extern __shared__ __attribute__((aligned(16))) bf16_t lds_g[];
    bf16_t(*As)[LDK] = reinterpret_cast<bf16_t(*)[LDK]>(lds_g);
    bf16_t(*Bs)[LDK] = reinterpret_cast<bf16_t(*)[LDK]>(lds_g + TM * LDK);   // transposed: [n][k]
    const int nt = (int)(blockIdx.x % d.ntiles), mt = (int)(blockIdx.x / d.ntiles);
    const int m0 = mt * TM;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int64_t G = 1;
    for (int i = 0; i < d.ng; i++) G *= d.g_size[i];
    const int64_t NF = G * d.N;
    // this thread's four B columns (one g, since N % 4 == 0) and k rows: eight
    // consecutive lanes take eight k groups of one column quad, so that the
    // transposed 8-byte LDS writes of sixteen lanes cover 32 distinct words
    const int nq = tid >> 3, kq = 4 * (tid & 7);
    const int64_t fb = (int64_t)nt * TN + 4 * nq;
    const bool colok = fb < NF;
    int64_t ob = 0;
    {
        const int64_t g = colok ? fb / d.N : 0;
        int64_t oA, oC;
        gemm_offsets(d, g, oA, ob, oC);
        ob += colok ? fb - g * d.N : 0;   // columns past the end read column 0 (masked)
    }
    // this thread's A elements e: tile index tid + 256 e, rows fastest when
    // A's rows are unit-stride (so that a load instruction reads consecutive
    // elements), else k fastest; either way element e sits at a fixed stride
    // from element 0 (256 / TM k-steps or 256 / TK rows)
    const bool mfast = d.sAm == 1 && d.sAk != 1;
    auto a_at = [&](int e, int& m, int& k) {
        const int i = tid + 256 * e;
        if (mfast) {
            m = i % TM;
            k = i / TM;
        } else {
            m = i / TK;
            k = i % TK;
        }
    };
    int am0, ak0;
    a_at(0, am0, ak0);
    const int64_t a_step = (int64_t)(256 / TM) * d.sAk;   // rows-fastest layout
    const bf16_t* pa = A + (int64_t)min(m0 + am0, d.M - 1) * d.sAm + (int64_t)ak0 * d.sAk;
    // B rows of this thread: kq + 32 h + r, r = 0..3 (columns past the end read column 0)
    const bf16_t* pb = B + ob + (int64_t)kq * d.sBk;
    const int64_t sb = d.sBk;
    uint2 vb[KH][4];
    bf16_t va[AE];
    // Full chunks load without guards; the last, partial chunk clamps each
    // address and masks the value (a guard around a load would become a branch
    // and a wait per load).
    auto load = [&](int k0) {
        const bf16_t* p = pb + (int64_t)k0 * sb;
        const uint32_t ckeep = colok ? 0xffffffffu : 0u;
        if (k0 + TK <= d.K) {
#pragma unroll
            for (int h = 0; h < KH; h++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const uint2 v = *(const uint2*)(p + (32 * h + r) * sb);
                    vb[h][r] = make_uint2(v.x & ckeep, v.y & ckeep);
                }
            if (mfast) {
                // one row (clamped) for every element, k steps of 256 / TM
                const bf16_t* q = pa + (int64_t)k0 * d.sAk;
                const bool rowok = m0 + am0 < d.M;
#pragma unroll
                for (int e = 0; e < AE; e++) {
                    const bf16_t v = q[e * a_step];
                    va[e] = rowok ? v : (bf16_t)0;
                }
            } else {
                // one k for every element, rows 256 / TK apart (each clamped)
                const int64_t ko = (int64_t)(k0 + ak0) * d.sAk;
#pragma unroll
                for (int e = 0; e < AE; e++) {
                    const int mr = m0 + am0 + e * (256 / TK), mc = mr < d.M ? mr : d.M - 1;
                    const bf16_t v = A[(int64_t)mc * d.sAm + ko];
                    va[e] = mr < d.M ? v : (bf16_t)0;
                }
            }
        } else {
#pragma unroll
            for (int h = 0; h < KH; h++)
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const int k = k0 + kq + 32 * h + r, kc = k < d.K ? k : d.K - 1;
                    const uint2 v = *(const uint2*)(B + ob + (int64_t)kc * sb);
                    const uint32_t keep = k < d.K ? ckeep : 0u;
                    vb[h][r] = make_uint2(v.x & keep, v.y & keep);
                }
#pragma unroll
            for (int e = 0; e < AE; e++) {
                int m, k;
                a_at(e, m, k);
                m += m0;
                k += k0;
                const int mc = m < d.M ? m : d.M - 1, kc = k < d.K ? k : d.K - 1;
                const bf16_t v = A[(int64_t)mc * d.sAm + (int64_t)kc * d.sAk];
                va[e] = (m < d.M && k < d.K) ? v : (bf16_t)0;
            }
        }
    };
    f32x16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.f;
    load(0);
    for (int k0 = 0; k0 < d.K; k0 += TK) {
        __syncthreads();   // the previous chunk's LDS reads are done
#pragma unroll
        for (int e = 0; e < AE; e++) {
            int m, k;
            a_at(e, m, k);
            As[m][k] = va[e];
        }
#pragma unroll
        for (int h = 0; h < KH; h++)
#pragma unroll
            for (int j = 0; j < 4; j++) {
                // column 4 nq + j, k rows kq + 32 h + 0..3: one 8-byte LDS write;
                // each word pairs column j of two k rows (one byte permute:
                // selector 0x05040100 takes the low halves, 0x07060302 the high)
                const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
                auto col = [&](int r) { return (j < 2) ? vb[h][r].x : vb[h][r].y; };
                uint2 w;
                w.x = __builtin_amdgcn_perm(col(1), col(0), sel);
                w.y = __builtin_amdgcn_perm(col(3), col(2), sel);
                *(uint2*)&Bs[4 * nq + j][kq + 32 * h] = w;
            }
        __syncthreads();
        if (k0 + TK < d.K) load(k0 + TK);
        const int kend = min(TK, d.K - k0);
#pragma unroll
        for (int kk = 0; kk < TK; kk += 16) {
            if (kk >= kend) break;
            const bf16x8 b = lds_bf16x8(&Bs[wave * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
#pragma unroll
            for (int i = 0; i < MT; i++) {
                const bf16x8 a = lds_bf16x8(&As[i * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
                acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[i], 0, 0, 0);
            }
        }
    }
    const int64_t f = (int64_t)nt * TN + wave * 32 + (lane & 31);
    if (f >= NF) return;
    const int64_t g = f / d.N, n = f - g * d.N;
    int64_t oA, oB, oC;
    gemm_offsets(d, g, oA, oB, oC);
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const int m = m0 + i * 32 + mfma32_row(r, lane);
            if (m < d.M) store(C, oC + (int64_t)m * d.sCm + n, acc[i][r]);
        }
}

template <typename TC, int MT, int TK>
hipError_t gemm_bf16f_launch(const GemmDesc& d, dim3 g, const bf16_t* A, const bf16_t* B, TC* C, hipStream_t s) {
    constexpr uint32_t lds = (32 * MT + 128) * (TK + 8) * 2;
    if constexpr (lds > 64 * 1024) {
        static std::atomic<uint64_t> ok{0};
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        if (dev < 0 || dev >= 64) return hipErrorInvalidValue;
        if (!(ok.load() & (1ull << dev))) {
            e = hipFuncSetAttribute((const void*)gemm_bf16f<TC, MT, TK>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                    (int)lds);
            if (e != hipSuccess) return e;
            ok.fetch_or(1ull << dev);
        }
    }
    hipLaunchKernelGGL((gemm_bf16f<TC, MT, TK>), g, dim3(256), lds, s, d, A, B, C);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// factor gradients: partial NT GEMM over a chunk of the reduction
// ---------------------------------------------------------------------------
template <typename T, bool VEC>
__global__ void __launch_bounds__(256) wgrad(WgradDesc d, const T* __restrict__ A,
                                             const T* __restrict__ B, float* __restrict__ part) {
    constexpr int TM = 64, TN = 64, TK = 32;
    constexpr bool BF = sizeof(T) == 2;
    constexpr int LDK = BF ? TK + 8 : TK + 1;
    __shared__ __attribute__((aligned(16))) T As[TM][LDK];
    __shared__ __attribute__((aligned(16))) T Bs[TN][LDK];
    int64_t bid = blockIdx.x;
    const int nt = (int)(bid % d.ntiles);
    bid /= d.ntiles;
    const int mt = (int)(bid % d.mtiles);
    bid /= d.mtiles;
    const int64_t s = bid;                       // partial index
    int64_t kbi = s / d.ksplit;
    const int kc = (int)(s % d.ksplit);
    int64_t oA = 0, oB = 0;
    for (int i = d.nkb - 1; i >= 0; --i) {
        int64_t x = kbi % d.kb_size[i];
        kbi /= d.kb_size[i];
        oA += x * d.kb_sA[i];
        oB += x * d.kb_sB[i];
    }
    const int64_t kbeg = (int64_t)kc * d.kchunk;
    const int64_t kend = min(d.K, kbeg + d.kchunk);
    const int m0 = mt * TM, n0 = nt * TN;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; r++) acc[r] = 0.f;

    for (int64_t k0 = kbeg; k0 < kend; k0 += TK) {
        // 64 rows x 32 k per operand: 4-element runs along k, 2 per thread per operand
#pragma unroll
        for (int it = 0; it < 2; it++) {
            int e = tid + it * 256;
            int row = e >> 3, kk = (e & 7) * 4;
            int64_t k = k0 + kk;
#pragma unroll
            for (int op = 0; op < 2; op++) {
                const T* src = op ? B : A;
                int base_row = op ? n0 : m0;
                int lim = op ? d.N : d.M;
                int64_t o = op ? oB : oA;
                int64_t sr = op ? d.sBn : d.sAm;
                T (*dst)[LDK] = op ? Bs : As;
                T v[4] = {0, 0, 0, 0};
                int rr = base_row + row;
                if (rr < lim) {
                    const T* p = src + o + (int64_t)rr * sr + k;
                    if (VEC && k + 3 < kend) {
                        if constexpr (BF) {
                            uint2 raw = *(const uint2*)p;
                            v[0] = (T)(raw.x & 0xffff);
                            v[1] = (T)(raw.x >> 16);
                            v[2] = (T)(raw.y & 0xffff);
                            v[3] = (T)(raw.y >> 16);
                        } else {
                            f32x4 raw = *(const f32x4*)p;
                            __builtin_memcpy(v, &raw, 16);
                        }
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; j++)
                            if (k + j < kend) v[j] = p[j];
                    }
                }
                if constexpr (BF) {
                    uint2 w;
                    w.x = (uint32_t)(uint16_t)v[0] | ((uint32_t)(uint16_t)v[1] << 16);
                    w.y = (uint32_t)(uint16_t)v[2] | ((uint32_t)(uint16_t)v[3] << 16);
                    *(uint2*)&dst[row][kk] = w;
                } else {
#pragma unroll
                    for (int j = 0; j < 4; j++) dst[row][kk + j] = v[j];
                }
            }
        }
        __syncthreads();
        if constexpr (BF) {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 16) {
                bf16x8 a = lds_bf16x8((const bf16_t*)&As[wm * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
                bf16x8 b = lds_bf16x8((const bf16_t*)&Bs[wn * 32 + (lane & 31)][kk + 8 * (lane >> 5)]);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 2) {
                float a = (float)As[wm * 32 + (lane & 31)][kk + (lane >> 5)];
                float b = (float)Bs[wn * 32 + (lane & 31)][kk + (lane >> 5)];
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
            }
        }
        __syncthreads();
    }
    const int n = n0 + wn * 32 + (lane & 31);
    if (n >= d.N) return;
    float* out = part + s * (int64_t)d.M * d.N;
#pragma unroll
    for (int r = 0; r < 16; r++) {
        int m = m0 + wm * 32 + mfma32_row(r, lane);
        if (m < d.M) out[(int64_t)m * d.N + n] = acc[r];
    }
}

// C[e] = sum_s part[s][e]: 64 outputs a block; the NW waves of the block sum consecutive runs of the
// partials (16 loads in flight a lane), then wave 0 adds the NW run sums in
// wave order: a fixed order for a given NW, which the launcher derives from
// nsplit alone (1 wave up to 8 partials, 4 up to 64, else 16).
template <int NW, typename TC>
__device__ __forceinline__ void reduce_block(const ReduceDesc& d, const float* __restrict__ part,
                                             TC* __restrict__ C, int64_t blk, double (*q)[64]) {
    const int lane = threadIdx.x & 63, wave = NW == 1 ? 0 : __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t mn = (int64_t)d.M * d.N;
    const int64_t e = blk * 64 + lane;
    const int64_t per = (d.nsplit + NW - 1) / NW;
    const int64_t s0 = wave * per, s1 = min(d.nsplit, s0 + per);
    double acc = 0.0;
    if (e < mn) {
        int64_t s = s0;
        for (; s + 16 <= s1; s += 16) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; u++) v[u] = part[(s + u) * mn + e];
#pragma unroll
            for (int u = 0; u < 16; u++) acc += v[u];
        }
        for (; s < s1; s++) acc += part[s * mn + e];
    }
    if constexpr (NW > 1) {
        q[wave][lane] = acc;
        __syncthreads();
        if (wave != 0) return;
        acc = q[0][lane];
#pragma unroll
        for (int w = 1; w < NW; w++) acc += q[w][lane];
    }
    if (e < mn) {
        int64_t m = e / d.N, n = e - m * d.N;
        store(C, m * d.sCm + n * d.sCn, (float)acc);
    }
}

template <int NW, typename TC>
__global__ void __launch_bounds__(64 * NW) reduce_partials(ReduceDesc d, const float* __restrict__ part,
                                                           TC* __restrict__ C) {
    __shared__ double q[NW][64];
    reduce_block<NW>(d, part, C, blockIdx.x, q);
}

struct MultiPtrs {
    const float* part[4];
    float* out[4];
};

template <int NW>
__global__ void __launch_bounds__(64 * NW) reduce_multi(MultiReduceDesc d, MultiPtrs p) {
    __shared__ double q[NW][64];
    int j = 0;
    while (j + 1 < d.n && blockIdx.x >= d.block0[j + 1]) j++;
    if (!p.out[j]) return;   // uniform over the block
    reduce_block<NW>(d.part[j], p.part[j], p.out[j], blockIdx.x - d.block0[j], q);
}

// ---------------------------------------------------------------------------
// depthwise convolution along one axis
// ---------------------------------------------------------------------------
constexpr int kDwLds = 4096;   // elements of a block's region staged in LDS
constexpr int kDwMaxSlabs = 256;

template <typename T, typename TF, typename TC, int KT>
__global__ void __launch_bounds__(256) dw_conv(DwDesc d, const T* __restrict__ in,
                                               const TF* __restrict__ f, TC* __restrict__ out) {
    __shared__ float buf[kDwLds];
    __shared__ float taps[kDwMaxSlabs][KT];
    const int64_t slab0 = (int64_t)blockIdx.x * d.spb;
    const int nsl = (int)min((int64_t)d.spb, d.nslab - slab0);
    const int slabsz = d.A * d.inner;
    const int total = nsl * slabsz;
    const int64_t base = slab0 * slabsz;
    const int tid = threadIdx.x;
    for (int e = tid; e < total; e += 256) buf[e] = load(in, base + e);
    for (int e = tid; e < nsl * KT; e += 256) {
        int sl = e / KT, j = e - sl * KT;
        int64_t o = slab0 + sl;
        int64_t frow = ((o / d.r_div) % d.r_size) * d.r_stride;
        taps[sl][j] = load(f, frow + (int64_t)j * d.f_sj);
    }
    __syncthreads();
    for (int e = tid; e < total; e += 256) {
        int sl = e / slabsz, rem = e - sl * slabsz, p = rem / d.inner, q = rem - p * d.inner;
        const float* row = buf + sl * slabsz + q;
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < KT; j++) {
            int pp = p + d.sign * j + d.off;
            if (pp >= 0 && pp < d.A) acc += row[pp * d.inner] * taps[sl][j];
        }
        store(out, base + e, acc);
    }
}

// part[block][j] = sum over the block's region of in[p + j + off] * g[p]
template <typename T, int KT>
__global__ void __launch_bounds__(256) dw_tapgrad(DwDesc d, const T* __restrict__ in,
                                                  const T* __restrict__ g, float* __restrict__ part) {
    __shared__ float buf[kDwLds];
    __shared__ float red[4][KT];
    const int64_t slab0 = (int64_t)blockIdx.x * d.spb;
    const int nsl = (int)min((int64_t)d.spb, d.nslab - slab0);
    const int slabsz = d.A * d.inner;
    const int total = nsl * slabsz;
    const int64_t base = slab0 * slabsz;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    for (int e = tid; e < total; e += 256) buf[e] = load(in, base + e);
    __syncthreads();
    float acc[KT];
#pragma unroll
    for (int j = 0; j < KT; j++) acc[j] = 0.f;
    for (int e = tid; e < total; e += 256) {
        int sl = e / slabsz, rem = e - sl * slabsz, p = rem / d.inner, q = rem - p * d.inner;
        const float* row = buf + sl * slabsz + q;
        float gv = load(g, base + e);
#pragma unroll
        for (int j = 0; j < KT; j++) {
            int pp = p + j + d.off;
            if (pp >= 0 && pp < d.A) acc[j] += row[pp * d.inner] * gv;
        }
    }
#pragma unroll
    for (int j = 0; j < KT; j++) {
        float v = wave_sum(acc[j]);
        if (lane == 0) red[wave][j] = v;
    }
    __syncthreads();
    if (tid < KT) part[blockIdx.x * (int64_t)KT + tid] = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
}

// out[r][j] = sum over the blocks whose slabs use filter row r: one block per
// r, threads stride over that row's partials, then a fixed-order block sum.
template <typename TC, int KT>
__global__ void __launch_bounds__(256) dw_tapreduce(DwDesc d, const float* __restrict__ part,
                                                    TC* __restrict__ out) {
    __shared__ double red[4][KT];
    const int64_t r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t run = d.r_div / d.spb;              // consecutive blocks of one row
    const int64_t period = run * d.r_size;
    const int64_t cnt = (d.nblocks / period) * run;   // partials of row r
    double acc[KT];
#pragma unroll
    for (int j = 0; j < KT; j++) acc[j] = 0.0;
    for (int64_t i = tid; i < cnt; i += 256) {
        int64_t a = i / run, c = i - a * run;
        const float* p = part + (a * period + r * run + c) * KT;
#pragma unroll
        for (int j = 0; j < KT; j++) acc[j] += p[j];
    }
#pragma unroll
    for (int j = 0; j < KT; j++) {
        double v = acc[j];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
        if (lane == 0) red[wave][j] = v;
    }
    __syncthreads();
    if (tid < KT)
        store(out, r * d.o_sr + tid * d.o_sj, (float)((red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid])));
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
template <typename D>
D desc_of(const Launch& ln) {
    D d;
    std::memcpy(&d, ln.desc.data(), sizeof(D));
    return d;
}

hipError_t launch_gemm(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s) {
    GemmDesc d = desc_of<GemmDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    int opt = ln.kind >> kShiftOpt;
    int MT = (opt & 1) ? 2 : 1;
    // vector loads need 16 B (fp32) / 8 B (bf16) aligned rows of B
    bool vec = (opt & 2) && ((uintptr_t)b % (tIn ? 8 : 16) == 0);
    dim3 g(ln.grid[0]), bl(256);
    if (tIn && (opt & 4)) {
        // flattened columns: 8-byte rows of B (N, sBk and the batch strides
        // multiples of 4 were checked by the lowering; here the base)
        if ((uintptr_t)b % 8 != 0 || d.N % 4 != 0) return hipErrorInvalidValue;
        const bf16_t* A = (const bf16_t*)a;
        const bf16_t* B = (const bf16_t*)b;
        const bool one = false;   // 256-wide chunks (one block a CU) measured slower
        if (tC) {
            bf16_t* C = (bf16_t*)c;
            if (MT == 2) return one ? gemm_bf16f_launch<bf16_t, 2, 256>(d, g, A, B, C, s)
                                    : gemm_bf16f_launch<bf16_t, 2, 64>(d, g, A, B, C, s);
            return one ? gemm_bf16f_launch<bf16_t, 1, 256>(d, g, A, B, C, s)
                       : gemm_bf16f_launch<bf16_t, 1, 64>(d, g, A, B, C, s);
        }
        float* C = (float*)c;
        if (MT == 2) return one ? gemm_bf16f_launch<float, 2, 256>(d, g, A, B, C, s)
                                : gemm_bf16f_launch<float, 2, 64>(d, g, A, B, C, s);
        return one ? gemm_bf16f_launch<float, 1, 256>(d, g, A, B, C, s)
                   : gemm_bf16f_launch<float, 1, 64>(d, g, A, B, C, s);
    }
    if (tIn) {
        const bf16_t* A = (const bf16_t*)a;
        const bf16_t* B = (const bf16_t*)b;
        if (tC) {
            if (MT == 2) { if (vec) hipLaunchKernelGGL((gemm_bf16<bf16_t, 2, true>), g, bl, 0, s, d, A, B, (bf16_t*)c);
                           else hipLaunchKernelGGL((gemm_bf16<bf16_t, 2, false>), g, bl, 0, s, d, A, B, (bf16_t*)c); }
            else { if (vec) hipLaunchKernelGGL((gemm_bf16<bf16_t, 1, true>), g, bl, 0, s, d, A, B, (bf16_t*)c);
                   else hipLaunchKernelGGL((gemm_bf16<bf16_t, 1, false>), g, bl, 0, s, d, A, B, (bf16_t*)c); }
        } else {
            if (MT == 2) { if (vec) hipLaunchKernelGGL((gemm_bf16<float, 2, true>), g, bl, 0, s, d, A, B, (float*)c);
                           else hipLaunchKernelGGL((gemm_bf16<float, 2, false>), g, bl, 0, s, d, A, B, (float*)c); }
            else { if (vec) hipLaunchKernelGGL((gemm_bf16<float, 1, true>), g, bl, 0, s, d, A, B, (float*)c);
                   else hipLaunchKernelGGL((gemm_bf16<float, 1, false>), g, bl, 0, s, d, A, B, (float*)c); }
        }
    } else {
        const float* A = (const float*)a;
        const float* B = (const float*)b;
        if (tC) {
            if (MT == 2) { if (vec) hipLaunchKernelGGL((gemm_f32<bf16_t, 2, true>), g, bl, 0, s, d, A, B, (bf16_t*)c);
                           else hipLaunchKernelGGL((gemm_f32<bf16_t, 2, false>), g, bl, 0, s, d, A, B, (bf16_t*)c); }
            else { if (vec) hipLaunchKernelGGL((gemm_f32<bf16_t, 1, true>), g, bl, 0, s, d, A, B, (bf16_t*)c);
                   else hipLaunchKernelGGL((gemm_f32<bf16_t, 1, false>), g, bl, 0, s, d, A, B, (bf16_t*)c); }
        } else {
            if (MT == 2) { if (vec) hipLaunchKernelGGL((gemm_f32<float, 2, true>), g, bl, 0, s, d, A, B, (float*)c);
                           else hipLaunchKernelGGL((gemm_f32<float, 2, false>), g, bl, 0, s, d, A, B, (float*)c); }
            else { if (vec) hipLaunchKernelGGL((gemm_f32<float, 1, true>), g, bl, 0, s, d, A, B, (float*)c);
                   else hipLaunchKernelGGL((gemm_f32<float, 1, false>), g, bl, 0, s, d, A, B, (float*)c); }
        }
    }
    return hipGetLastError();
}

hipError_t launch_wgrad(const Launch& ln, const void* a, const void* b, void* part, hipStream_t s) {
    WgradDesc d = desc_of<WgradDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1;
    int opt = ln.kind >> kShiftOpt;
    bool vec = (opt & 2) && ((uintptr_t)a % (tIn ? 8 : 16) == 0) && ((uintptr_t)b % (tIn ? 8 : 16) == 0);
    dim3 g(ln.grid[0]), bl(256);
    if (tIn) {
        if (vec) hipLaunchKernelGGL((wgrad<bf16_t, true>), g, bl, 0, s, d, (const bf16_t*)a, (const bf16_t*)b, (float*)part);
        else hipLaunchKernelGGL((wgrad<bf16_t, false>), g, bl, 0, s, d, (const bf16_t*)a, (const bf16_t*)b, (float*)part);
    } else {
        if (vec) hipLaunchKernelGGL((wgrad<float, true>), g, bl, 0, s, d, (const float*)a, (const float*)b, (float*)part);
        else hipLaunchKernelGGL((wgrad<float, false>), g, bl, 0, s, d, (const float*)a, (const float*)b, (float*)part);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_reduce_multi(const Launch& ln, const void* const* parts, void* const* outs, hipStream_t s) {
    MultiReduceDesc d = desc_of<MultiReduceDesc>(ln);
    if (d.n < 1 || d.n > 4 || (int64_t)ln.grid[0] != d.block0[d.n]) return hipErrorInvalidValue;
    MultiPtrs p;
    for (int j = 0; j < 4; j++) {
        p.part[j] = j < d.n ? (const float*)parts[j] : nullptr;
        p.out[j] = j < d.n ? (float*)outs[j] : nullptr;
    }
    // every part of one launch takes the wave count of the largest partial count
    int64_t ns = 0;
    for (int j = 0; j < d.n; j++) ns = d.part[j].nsplit > ns ? d.part[j].nsplit : ns;
    switch (reduce_waves(ns)) {
        case 1: hipLaunchKernelGGL(reduce_multi<1>, dim3(ln.grid[0]), dim3(64), 0, s, d, p); break;
        case 4: hipLaunchKernelGGL(reduce_multi<4>, dim3(ln.grid[0]), dim3(256), 0, s, d, p); break;
        default: hipLaunchKernelGGL(reduce_multi<16>, dim3(ln.grid[0]), dim3(1024), 0, s, d, p); break;
    }
    return hipGetLastError();
}

namespace {

hipError_t launch_reduce(const Launch& ln, const void* part, void* c, hipStream_t s) {
    ReduceDesc d = desc_of<ReduceDesc>(ln);
    int tC = (ln.kind >> kBitOut) & 1;
    if ((int64_t)ln.grid[0] * 64 < (int64_t)d.M * d.N) return hipErrorInvalidValue;
    dim3 g(ln.grid[0]);
#define RP_LAUNCH(nw) \
    do { \
        if (tC) hipLaunchKernelGGL((reduce_partials<nw, bf16_t>), g, dim3(64 * nw), 0, s, d, (const float*)part, (bf16_t*)c); \
        else hipLaunchKernelGGL((reduce_partials<nw, float>), g, dim3(64 * nw), 0, s, d, (const float*)part, (float*)c); \
    } while (0)
    switch (reduce_waves(d.nsplit)) {
        case 1: RP_LAUNCH(1); break;
        case 4: RP_LAUNCH(4); break;
        default: RP_LAUNCH(16); break;
    }
#undef RP_LAUNCH
    return hipGetLastError();
}

template <typename T, typename TF, typename TC>
hipError_t dw_conv_k(int K, const DwDesc& d, dim3 g, const void* a, const void* b, void* c, hipStream_t s) {
    const T* in = (const T*)a;
    const TF* f = (const TF*)b;
    TC* out = (TC*)c;
    dim3 bl(256);
    switch (K) {
        case 1: hipLaunchKernelGGL((dw_conv<T, TF, TC, 1>), g, bl, 0, s, d, in, f, out); break;
        case 2: hipLaunchKernelGGL((dw_conv<T, TF, TC, 2>), g, bl, 0, s, d, in, f, out); break;
        case 3: hipLaunchKernelGGL((dw_conv<T, TF, TC, 3>), g, bl, 0, s, d, in, f, out); break;
        case 4: hipLaunchKernelGGL((dw_conv<T, TF, TC, 4>), g, bl, 0, s, d, in, f, out); break;
        case 5: hipLaunchKernelGGL((dw_conv<T, TF, TC, 5>), g, bl, 0, s, d, in, f, out); break;
        case 6: hipLaunchKernelGGL((dw_conv<T, TF, TC, 6>), g, bl, 0, s, d, in, f, out); break;
        case 7: hipLaunchKernelGGL((dw_conv<T, TF, TC, 7>), g, bl, 0, s, d, in, f, out); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_dw(const Launch& ln, const void* a, const void* b, void* c, hipStream_t s) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1, tF = (ln.kind >> kBitAux) & 1, tC = (ln.kind >> kBitOut) & 1;
    dim3 g(ln.grid[0]);
    if (tIn) {
        if (tF) return tC ? dw_conv_k<bf16_t, bf16_t, bf16_t>(d.K, d, g, a, b, c, s)
                          : dw_conv_k<bf16_t, bf16_t, float>(d.K, d, g, a, b, c, s);
        return tC ? dw_conv_k<bf16_t, float, bf16_t>(d.K, d, g, a, b, c, s)
                  : dw_conv_k<bf16_t, float, float>(d.K, d, g, a, b, c, s);
    }
    if (tF) return tC ? dw_conv_k<float, bf16_t, bf16_t>(d.K, d, g, a, b, c, s)
                      : dw_conv_k<float, bf16_t, float>(d.K, d, g, a, b, c, s);
    return tC ? dw_conv_k<float, float, bf16_t>(d.K, d, g, a, b, c, s)
              : dw_conv_k<float, float, float>(d.K, d, g, a, b, c, s);
}

template <typename T>
hipError_t dw_tapgrad_k(int K, const DwDesc& d, dim3 g, const void* a, const void* b, void* part,
                        hipStream_t s) {
    const T* in = (const T*)a;
    const T* gr = (const T*)b;
    float* p = (float*)part;
    dim3 bl(256);
    switch (K) {
        case 1: hipLaunchKernelGGL((dw_tapgrad<T, 1>), g, bl, 0, s, d, in, gr, p); break;
        case 2: hipLaunchKernelGGL((dw_tapgrad<T, 2>), g, bl, 0, s, d, in, gr, p); break;
        case 3: hipLaunchKernelGGL((dw_tapgrad<T, 3>), g, bl, 0, s, d, in, gr, p); break;
        case 4: hipLaunchKernelGGL((dw_tapgrad<T, 4>), g, bl, 0, s, d, in, gr, p); break;
        case 5: hipLaunchKernelGGL((dw_tapgrad<T, 5>), g, bl, 0, s, d, in, gr, p); break;
        case 6: hipLaunchKernelGGL((dw_tapgrad<T, 6>), g, bl, 0, s, d, in, gr, p); break;
        case 7: hipLaunchKernelGGL((dw_tapgrad<T, 7>), g, bl, 0, s, d, in, gr, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_dw_tapgrad(const Launch& ln, const void* a, const void* b, void* part, hipStream_t s) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1;
    dim3 g(ln.grid[0]);
    return tIn ? dw_tapgrad_k<bf16_t>(d.K, d, g, a, b, part, s)
               : dw_tapgrad_k<float>(d.K, d, g, a, b, part, s);
}

template <typename TC>
hipError_t dw_tapreduce_k(int K, const DwDesc& d, dim3 g, const void* part, void* c, hipStream_t s) {
    const float* p = (const float*)part;
    TC* out = (TC*)c;
    dim3 bl(256);
    switch (K) {
        case 1: hipLaunchKernelGGL((dw_tapreduce<TC, 1>), g, bl, 0, s, d, p, out); break;
        case 2: hipLaunchKernelGGL((dw_tapreduce<TC, 2>), g, bl, 0, s, d, p, out); break;
        case 3: hipLaunchKernelGGL((dw_tapreduce<TC, 3>), g, bl, 0, s, d, p, out); break;
        case 4: hipLaunchKernelGGL((dw_tapreduce<TC, 4>), g, bl, 0, s, d, p, out); break;
        case 5: hipLaunchKernelGGL((dw_tapreduce<TC, 5>), g, bl, 0, s, d, p, out); break;
        case 6: hipLaunchKernelGGL((dw_tapreduce<TC, 6>), g, bl, 0, s, d, p, out); break;
        case 7: hipLaunchKernelGGL((dw_tapreduce<TC, 7>), g, bl, 0, s, d, p, out); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_dw_tapreduce(const Launch& ln, const void* part, void* c, hipStream_t s) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tC = (ln.kind >> kBitOut) & 1;
    dim3 g(ln.grid[0]);
    return tC ? dw_tapreduce_k<bf16_t>(d.K, d, g, part, c, s)
              : dw_tapreduce_k<float>(d.K, d, g, part, c, s);
}

}  // namespace

hipError_t launch_fast(const Launch& ln, const void* a, const void* b, void* c, void* d,
                       hipStream_t s) {
    switch (ln.kind & 0xff) {
        case K_GEMM: return launch_gemm(ln, a, b, c, s);
        case K_WGRAD: return launch_wgrad(ln, a, b, d, s);
        case K_REDUCE: return launch_reduce(ln, d, c, s);
        case K_DW: return launch_dw(ln, a, b, c, s);
        case K_DW_TAPGRAD: return launch_dw_tapgrad(ln, a, b, d, s);
        case K_DW_TAPREDUCE: return launch_dw_tapreduce(ln, d, c, s);
        case K_TC:
        case K_TC_REDUCE: return launch_tc(ln, a, b, c, d, s);
        case K_THIN: return launch_thin(ln, a, b, c, s);
        case K_CRED: return launch_cred(ln, b, a, c, s);
        case K_CCONV: return launch_cconv(ln, a, b, c, s);
        case K_CREDW: return launch_cred(ln, a, b, d, s);
        case K_WGCONV: return launch_wgconv(ln, a, b, d, s);
        case K_CREDW_REDUCE: return launch_cred(ln, nullptr, d, c, s);
        case K_THINW:
        case K_THINW_REDUCE: return launch_thinw(ln, a, b, d, c, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace ce
