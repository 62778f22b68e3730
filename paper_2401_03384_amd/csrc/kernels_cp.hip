// Fused CP chain for gfx950: the four forward steps of a CP-factorised 2-D
// convolution layer (Section 2.3, CP convolutional layer; the pairwise steps
// the sequencer picks for it: contract s, convolve h, convolve w, contract r)
// in one kernel, with the rank-32 intermediates held in registers.
//
// One wavefront owns a strip of 32 image columns of one sample (strips
// overlap by the conv_w halo) and walks seg_rows rows down it:
//   GEMM1   Z1 for the row entering the ring (32x32 MFMA, X read straight from
//           HBM in the B-operand layout: lanes 0-31 one channel row, 32-63 the
//           next).  The accumulator layout holds Z1[r][col] with col = lane%32
//           and r = 8*(i/4) + 4*(lane/32) + i%4 for accumulator i.
//   conv_h  a ring of KH such accumulator sets: per-element FMAs.
//   conv_w  neighbouring columns are neighbouring lanes of the same half:
//           lane permutes; the strip's edge lanes are discarded.
//   GEMM2   consumes Z3 straight from the accumulator layout: instruction i
//           pairs k-slot 0 (lanes 0-31) with r = row(i, 0) and k-slot 1 (lanes
//           32-63) with r = row(i, 32); the A operand (Ut) is permuted to the
//           same pairing in LDS, so no data movement is needed.
// Rows and columns outside the image read X as zero, which is the same
// padding of both convolutions.
#include <atomic>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));

__device__ __forceinline__ bf16x8 lds8(const bf16_t* p) {
    bf16x8 v;
    __builtin_memcpy(&v, p, 16);
    return v;
}

__device__ __forceinline__ bf16x8 pack8(const bf16_t* v) {
    bf16x8 r;
    __builtin_memcpy(&r, v, 16);
    return r;
}

// r held by accumulator i of a lane in a 32x32 MFMA result
__device__ __forceinline__ int row32(int i, int lane) {
    return 8 * (i >> 2) + 4 * ((lane >> 5) & 1) + (i & 3);
}

// Two blocks per CU (256 VGPRs a lane) except for the bf16 5x5 variant, whose
// larger ring and bf16 operand packing do not fit that without spilling.
template <typename T, int KH, int KW, int MB2>
__global__ void __launch_bounds__(256, (sizeof(T) == 2 && KH == 5) ? 1 : 2) cp_fwd(CpDesc d, const T* __restrict__ X,
                                              const T* __restrict__ Us, const T* __restrict__ Kh,
                                              const T* __restrict__ Kw, const T* __restrict__ Ut,
                                              T* __restrict__ Y) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int TT = 32 * MB2;
    constexpr int CH = (KH - 1) / 2, HWW = (KW - 1) / 2;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int S = d.S, H = d.H, W = d.W;
    const int LDA = d.lda;
    T* UsL = (T*)smem;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, half = lane >> 5;

    // ---- tables ----
    {
    T* UtP = (T*)(smem + d.o_ut);
    float* KhP = (float*)(smem + d.o_kh);
    float* KwP = (float*)(smem + d.o_kw);
    for (int e = tid; e < 32 * S; e += 256) {
        int r = e / S, s = e - r * S;
        UsL[r * LDA + s] = Us[r * d.us_sr + s * d.us_ss];
    }
    if constexpr (BF) {
        // UtP[q][hf][t][j] = Ut[row32(8q+j, 32*hf)][t]
        for (int e = tid; e < 2 * 2 * TT * 8; e += 256) {
            int j = e & 7, t = (e >> 3) % TT, hf = (e / (8 * TT)) & 1, q = e / (16 * TT);
            UtP[e] = Ut[row32(8 * q + j, 32 * hf) * d.ut_sr + t * d.ut_st];
        }
    } else {
        // UtP[i][hf][t] = Ut[row32(i, 32*hf)][t]
        for (int e = tid; e < 16 * 2 * TT; e += 256) {
            int t = e % TT, hf = (e / TT) & 1, i = e / (2 * TT);
            UtP[e] = Ut[row32(i, 32 * hf) * d.ut_sr + t * d.ut_st];
        }
    }
    for (int e = tid; e < 16 * 2 * KH; e += 256) {
        int j = e % KH, hf = (e / KH) & 1, i = e / (2 * KH);
        KhP[e] = load(Kh, row32(i, 32 * hf) * d.kh_sr + j * d.kh_sj);
    }
    for (int e = tid; e < 16 * 2 * KW; e += 256) {
        int j = e % KW, hf = (e / KW) & 1, i = e / (2 * KW);
        KwP[e] = load(Kw, row32(i, 32 * hf) * d.kw_sr + j * d.kw_sj);
    }
    }
    __syncthreads();

    // ---- this wavefront's strip ----
    const int64_t gw = (int64_t)blockIdx.x * 4 + wave;
    if (gw >= d.waves) return;
    const int seg = (int)(gw % d.segs);
    const int64_t rest = gw / d.segs;
    const int cb = (int)(rest % d.ncb);
    const int b = (int)(rest / d.ncb);
    const int col = cb * d.colstride - HWW + (lane & 31);
    const bool colok = col >= 0 && col < W;
    const int h0 = seg * d.seg_rows, h1 = min(H, h0 + d.seg_rows);
    const T* Xc = X + (int64_t)b * d.x_sb + (colok ? col : 0);
    T* Yc = Y + (int64_t)b * d.y_sb + (colok ? col : 0);
    const bool store_lane = colok && (lane & 31) >= HWW && (lane & 31) < 32 - HWW;

    auto gemm1 = [&](int row) {
        f32x16 acc;
#pragma unroll
        for (int i = 0; i < 16; i++) acc[i] = 0.f;
        if (row < 0 || row >= H) return acc;   // uniform over the wave
        const T* xr = Xc + (int64_t)row * W;
        if constexpr (BF) {
            for (int k = 0; k < S; k += 16) {
                bf16_t xv[8];
#pragma unroll
                for (int j = 0; j < 8; j++)
                    xv[j] = colok ? xr[(int64_t)(k + 8 * half + j) * d.x_ss] : (bf16_t)0;
                bf16x8 av = lds8(UsL + (lane & 31) * LDA + k + 8 * half);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pack8(xv), acc, 0, 0, 0);
            }
        } else {
            for (int k = 0; k < S; k += 16) {
                float xv[8];
#pragma unroll
                for (int u = 0; u < 8; u++)
                    xv[u] = colok ? xr[(int64_t)(k + 2 * u + half) * d.x_ss] : 0.f;
#pragma unroll
                for (int u = 0; u < 8; u++) {
                    float av = UsL[(lane & 31) * LDA + k + 2 * u + half];
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, xv[u], acc, 0, 0, 0);
                }
            }
        }
        return acc;
    };

    f32x16 ring[KH];
#pragma unroll
    for (int j = 0; j < KH - 1; j++) ring[j] = gemm1(h0 - CH + j);
    for (int h = h0; h < h1; h++) {
        // The tap and Ut tables are re-read from LDS every row: the offsets
        // pass through an empty asm so the loads are not hoisted out of the
        // loop, where they would hold 16*(KH+KW+MB2) registers for its life.
        uint32_t o_ut = d.o_ut, o_kh = d.o_kh, o_kw = d.o_kw;
        asm volatile("" : "+s"(o_ut), "+s"(o_kh), "+s"(o_kw));
        const T* UtP = (const T*)(smem + o_ut);
        const float* KhP = (const float*)(smem + o_kh);
        const float* KwP = (const float*)(smem + o_kw);
        ring[KH - 1] = gemm1(h + KH - 1 - CH);
        // conv along h
        f32x16 z2;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < KH; j++) a += KhP[(i * 2 + half) * KH + j] * ring[j][i];
            z2[i] = a;
        }
#pragma unroll
        for (int j = 0; j < KH - 1; j++) ring[j] = ring[j + 1];
        // conv along w: neighbouring columns are neighbouring lanes of the half
        f32x16 z3;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int jw = 0; jw < KW; jw++) {
                int dd = jw - HWW;
                float v;
                if (dd == 0) {
                    v = z2[i];
                } else {
                    int src = (lane & 31) + dd;
                    src = src < 0 ? 0 : (src > 31 ? 31 : src);
                    v = __shfl(z2[i], (lane & 32) | src, 64);
                }
                a += KwP[(i * 2 + half) * KW + jw] * v;
            }
            z3[i] = a;
        }
        // GEMM2: Y[t][col] = sum_r Ut[r][t] Z3[r][col]
        f32x16 acc2[MB2];
#pragma unroll
        for (int mb = 0; mb < MB2; mb++)
#pragma unroll
            for (int i = 0; i < 16; i++) acc2[mb][i] = 0.f;
        if constexpr (BF) {
#pragma unroll
            for (int q = 0; q < 2; q++) {
                bf16_t zb[8];
#pragma unroll
                for (int j = 0; j < 8; j++) zb[j] = f32_to_bf16(z3[8 * q + j]);
                bf16x8 bv = pack8(zb);
#pragma unroll
                for (int mb = 0; mb < MB2; mb++) {
                    bf16x8 av = lds8(UtP + (((q * 2 + half) * TT) + mb * 32 + (lane & 31)) * 8);
                    acc2[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc2[mb], 0, 0, 0);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < 16; i++) {
#pragma unroll
                for (int mb = 0; mb < MB2; mb++) {
                    float av = UtP[(i * 2 + half) * TT + mb * 32 + (lane & 31)];
                    acc2[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, z3[i], acc2[mb], 0, 0, 0);
                }
            }
        }
        if (store_lane) {
            T* yr = Yc + (int64_t)h * W;
#pragma unroll
            for (int mb = 0; mb < MB2; mb++)
#pragma unroll
                for (int i = 0; i < 16; i++)
                    store(yr, (int64_t)(mb * 32 + row32(i, lane)) * d.y_st, acc2[mb][i]);
        }
    }
}

template <typename T, int K, int MB2>
hipError_t launch_cp_t(const CpDesc& d, const void* const* ops, void* y, hipStream_t s) {
    auto k = cp_fwd<T, K, K, MB2>;
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d, (const T*)ops[0],
                       (const T*)ops[1], (const T*)ops[2], (const T*)ops[3], (const T*)ops[4], (T*)y);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_cp_ty(const CpDesc& d, const void* const* ops, void* y, hipStream_t s) {
    if (d.KH == 3 && d.KW == 3)
        return d.T == 32 ? launch_cp_t<T, 3, 1>(d, ops, y, s) : launch_cp_t<T, 3, 2>(d, ops, y, s);
    if (d.KH == 5 && d.KW == 5)
        return d.T == 32 ? launch_cp_t<T, 5, 1>(d, ops, y, s) : launch_cp_t<T, 5, 2>(d, ops, y, s);
    return hipErrorInvalidValue;
}


// ---------------------------------------------------------------------------
// Backward of the chain (Section 3.2: every pairwise step's two gradients, in
// reverse order, with the intermediates recomputed), fused the same way.  One
// wavefront walks its strip over rows h = h0-CH .. h1+CH-1 and at row h
//   recomputes  Z1[h+CH] (ring of KH rows), Z2[h], Z3[h]
//   dZ3[h] = Ut^T dY[h]                  row GEMM over t
//   dUt   += Z3[h] dY[h]^T               MFMA over the strip's columns
//   dKw   += sum_w Z2[h][w+j-c] dZ3[h][w]
//   dZ2[h] = transposed conv along w of dZ3[h] (lane permutes)
//   dKh   += sum_w Z1[h+j-c][w] dZ2[h][w]
//   dZ1[h-CH] from the ring of the last KH dZ2 rows
//   dX[h-CH] = Us^T dZ1[h-CH]            (accumulator-layout product)
//   dUs   += dZ1[h-CH] X[h-CH]^T         MFMA over the strip's columns
// Every weight-gradient term is counted once: rows in [h0, h1) and the
// strip's own columns only.  The column reductions of dUt / dUs need the
// columns on the MFMA k axis: Z3 / dZ1 go through a wave-private LDS tile
// ([col][r]) and dY / X are read channel-major straight from memory.  The tap
// products are summed over the 32 lanes of each half by recursive halving.

template <int K>
__device__ __forceinline__ float swz_xor(float v) {
    // ds_swizzle bit-mask mode: lane i of each 32-lane group reads lane i ^ K
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1f | (K << 10)));
}

template <int K>
__device__ __forceinline__ void halve(float (&v)[32], bool up) {
#pragma unroll
    for (int q = 0; q < K; q++) {
        float send = up ? v[q] : v[q + K];
        float keep = up ? v[q + K] : v[q];
        v[q] = keep + swz_xor<K>(send);
    }
}

// Sum of v[0..31] over the 32 lanes of each half-wavefront; lane cl gets the
// total of entry cl.  Each step keeps the half of the list picked by one bit
// of the lane index and adds the partner's copy of that half.
__device__ __forceinline__ float half_reduce32(float (&v)[32], int cl) {
    halve<16>(v, cl & 16);
    halve<8>(v, cl & 8);
    halve<4>(v, cl & 4);
    halve<2>(v, cl & 2);
    halve<1>(v, cl & 1);
    return v[0];
}

// One 256-thread block per CU (the whole register file for one wavefront per
// SIMD): the strip state and the factor-gradient accumulators do not fit half
// of it.
template <typename T, int KH, int KW, int MT, int MS>
__global__ void __launch_bounds__(256, 1)
    cp_bwd(CpBwdDesc d, const T* __restrict__ X, const T* __restrict__ dY,
           const T* __restrict__ Us, const T* __restrict__ Kh, const T* __restrict__ Kw,
           const T* __restrict__ Ut, T* __restrict__ dX, float* __restrict__ Pus,
           float* __restrict__ Put, float* __restrict__ Pkh, float* __restrict__ Pkw) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int NT = 32 * MT, NS = 32 * MS;
    constexpr int CH = (KH - 1) / 2, CW = (KW - 1) / 2;
    constexpr int NG = (KH + KW) / 2;   // groups of two taps (32 products)
    constexpr int LZ = 33;              // transpose tile row pitch (floats)
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int H = d.H, W = d.W;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, hf = lane >> 5, cl = lane & 31;
    float* Zt = (float*)(smem + d.o_zt) + wave * (32 * LZ);
    // per-lane running sums of the tap-gradient products, wave-private:
    // float4 slot q of lane l at Tap[(q * 64 + l) * 4], q < 4 * (KW + KH)
    // (taps 0..KW-1 along w, then KH along h; 16 values per tap)
    float* Tap = (float*)(smem + d.o_tap) + wave * (64 * 16 * (KH + KW));

    // ---- tables ----
    {
        T* usa = (T*)smem;
        T* uta = (T*)(smem + d.o_uta);
        T* UsP = (T*)(smem + d.o_usp);
        float* KhP = (float*)(smem + d.o_kh);
        float* KwP = (float*)(smem + d.o_kw);
        for (int e = tid; e < 32 * NS; e += 256) {
            int r = e / NS, s = e - r * NS;
            usa[r * d.lda_s + s] = Us[r * d.us_sr + s * d.us_ss];
        }
        for (int e = tid; e < 32 * NT; e += 256) {
            int r = e / NT, t = e - r * NT;
            uta[r * d.lda_t + t] = Ut[r * d.ut_sr + t * d.ut_st];
        }
        if constexpr (BF) {
            // UsP[q][hf][s][j] = Us[row32(8q+j, 32*hf)][s]
            for (int e = tid; e < 2 * 2 * NS * 8; e += 256) {
                int j = e & 7, s = (e >> 3) % NS, h2 = (e / (8 * NS)) & 1, q = e / (16 * NS);
                UsP[e] = Us[row32(8 * q + j, 32 * h2) * d.us_sr + s * d.us_ss];
            }
        } else {
            // UsP[i][hf][s] = Us[row32(i, 32*hf)][s]
            for (int e = tid; e < 16 * 2 * NS; e += 256) {
                int s = e % NS, h2 = (e / NS) & 1, i = e / (2 * NS);
                UsP[e] = Us[row32(i, 32 * h2) * d.us_sr + s * d.us_ss];
            }
        }
        for (int e = tid; e < 16 * 2 * KH; e += 256) {
            int j = e % KH, h2 = (e / KH) & 1, i = e / (2 * KH);
            KhP[e] = load(Kh, row32(i, 32 * h2) * d.kh_sr + j * d.kh_sj);
        }
        for (int e = tid; e < 16 * 2 * KW; e += 256) {
            int j = e % KW, h2 = (e / KW) & 1, i = e / (2 * KW);
            KwP[e] = load(Kw, row32(i, 32 * h2) * d.kw_sr + j * d.kw_sj);
        }
    }
    __syncthreads();

    // ---- this wavefront's strip (waves past the end run no rows) ----
    const int64_t gw = (int64_t)blockIdx.x * 4 + wave;
    const bool wok = gw < d.waves;
    int seg = 0, cb = 0, b = 0;
    if (wok) {
        seg = (int)(gw % d.segs);
        const int64_t rest = gw / d.segs;
        cb = (int)(rest % d.ncb);
        b = (int)(rest / d.ncb);
    }
    const int h0 = seg * d.seg_rows, h1 = wok ? min(H, h0 + d.seg_rows) : h0;
    const int col0 = cb * d.colstride - CW;
    const int col = col0 + cl;
    const bool colok = col >= 0 && col < W;
    const bool own = colok && cl >= CW && cl < 32 - CW;
    const T* Xb = X + (int64_t)b * d.x_sb;
    const T* dYb = dY + (int64_t)b * d.y_sb;

    // Row GEMM: acc[r][col] = sum_k tab[r][k] src[k][row][col] (src channel
    // stride cs), the B operand read in its MFMA layout (coalesced columns).
    auto rowgemm = [&](const T* src, int64_t cs, const T* tab, int lda, int K, int row) {
        f32x16 acc;
#pragma unroll
        for (int i = 0; i < 16; i++) acc[i] = 0.f;
        if (row < 0 || row >= H) return acc;   // uniform over the wave
        const T* sr = src + (int64_t)row * W + (colok ? col : 0);
        if constexpr (BF) {
#pragma unroll 1
            for (int k = 0; k < K; k += 16) {
                bf16_t xv[8];
#pragma unroll
                for (int j = 0; j < 8; j++)
                    xv[j] = colok ? sr[(int64_t)(k + 8 * hf + j) * cs] : (bf16_t)0;
                bf16x8 av = lds8(tab + cl * lda + k + 8 * hf);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pack8(xv), acc, 0, 0, 0);
            }
        } else {
#pragma unroll 1
            for (int k = 0; k < K; k += 16) {
                float xv[8];
#pragma unroll
                for (int u = 0; u < 8; u++) xv[u] = colok ? sr[(int64_t)(k + 2 * u + hf) * cs] : 0.f;
#pragma unroll
                for (int u = 0; u < 8; u++)
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(tab[cl * lda + k + 2 * u + hf], xv[u],
                                                               acc, 0, 0, 0);
            }
        }
        return acc;
    };

    // acc[n][r][ch] += sum over the strip's columns of Zt[col][r] * src[32n+ch][row][col]
    // (Zt holds zeros outside the strip's own columns).
    auto colgemm = [&](f32x16* acc, int NN, const T* src, int64_t cs, int row) {
        const T* sr = src + (int64_t)row * W;
        if constexpr (BF) {
#pragma unroll 1
            for (int q = 0; q < 2; q++) {
                bf16_t za[8];
#pragma unroll
                for (int j = 0; j < 8; j++) za[j] = f32_to_bf16(Zt[(16 * q + 8 * hf + j) * LZ + cl]);
                const bf16x8 av = pack8(za);
                for (int n = 0; n < NN; n++) {
                    const T* sc = sr + (int64_t)(32 * n + cl) * cs;
                    bf16_t bv[8];
#pragma unroll
                    for (int j = 0; j < 8; j++) {
                        const int c = col0 + 16 * q + 8 * hf + j;
                        bv[j] = (c >= 0 && c < W) ? sc[c] : (bf16_t)0;
                    }
                    acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pack8(bv), acc[n], 0, 0, 0);
                }
            }
        } else {
            for (int n = 0; n < NN; n++) {
                const T* sc = sr + (int64_t)(32 * n + cl) * cs;
#pragma unroll 1
                for (int u0 = 0; u0 < 16; u0 += 8) {
                    float bv[8];
#pragma unroll
                    for (int u = 0; u < 8; u++) {
                        const int c = col0 + 2 * (u0 + u) + hf;
                        bv[u] = (c >= 0 && c < W) ? sc[c] : 0.f;
                    }
#pragma unroll
                    for (int u = 0; u < 8; u++)
                        acc[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                            Zt[(2 * (u0 + u) + hf) * LZ + cl], bv[u], acc[n], 0, 0, 0);
                }
            }
        }
    };

    // accumulator layout -> transpose tile, own columns only
    auto to_tile = [&](const f32x16& v) {
#pragma unroll
        for (int i = 0; i < 16; i++) Zt[cl * LZ + row32(i, lane)] = own ? v[i] : 0.f;
    };

    f32x16 ring[KH], dr[KH], accUt[MT], accUs[MS];
#pragma unroll
    for (int i = 0; i < 16; i++) {
#pragma unroll
        for (int j = 0; j < KH; j++) ring[j][i] = dr[j][i] = 0.f;
#pragma unroll
        for (int n = 0; n < MT; n++) accUt[n][i] = 0.f;
#pragma unroll
        for (int n = 0; n < MS; n++) accUs[n][i] = 0.f;
    }
    for (int q = 0; q < 4 * (KH + KW); q++)
        *(float4*)(Tap + (q * 64 + lane) * 4) = make_float4(0.f, 0.f, 0.f, 0.f);
    // Tap[jj][i] += p[i] for this lane (16 values, four float4 slots)
    auto tap_add = [&](int jj, const float* p) {
#pragma unroll
        for (int c = 0; c < 4; c++) {
            float4* q = (float4*)(Tap + ((jj * 4 + c) * 64 + lane) * 4);
            float4 v = *q;
            v.x += p[4 * c];
            v.y += p[4 * c + 1];
            v.z += p[4 * c + 2];
            v.w += p[4 * c + 3];
            *q = v;
        }
    };

    const int hs = h0 - CH, he = wok ? h1 + CH : hs;
    if (wok) {
#pragma unroll
        for (int j = 0; j < KH - 1; j++)
            ring[j] = rowgemm(Xb, d.x_ss, (const T*)smem, d.lda_s, NS, hs - CH + j);
    }
    for (int h = hs; h < he; h++) {
        // Tables re-read from LDS every row: the offsets pass through an empty
        // asm so that the loop-invariant loads are not hoisted into registers.
        uint32_t o_usa = 0, o_uta = d.o_uta, o_usp = d.o_usp, o_kh = d.o_kh, o_kw = d.o_kw;
        asm volatile("" : "+s"(o_usa), "+s"(o_uta), "+s"(o_usp), "+s"(o_kh), "+s"(o_kw));
        const T* UsA = (const T*)(smem + o_usa);
        const T* UtA = (const T*)(smem + o_uta);
        const T* UsP = (const T*)(smem + o_usp);
        const float* KhP = (const float*)(smem + o_kh);
        const float* KwP = (const float*)(smem + o_kw);

        ring[KH - 1] = rowgemm(Xb, d.x_ss, UsA, d.lda_s, NS, h + CH);
        const bool rin = h >= h0 && h < h1;
        const f32x16 dz3 = rowgemm(dYb, d.y_st, UtA, d.lda_t, NT, h);
        f32x16 z2;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < KH; j++) a += KhP[(i * 2 + hf) * KH + j] * ring[j][i];
            z2[i] = a;
        }
        // conv along w (Z3) and the dKw products
        f32x16 z3;
#pragma unroll
        for (int i = 0; i < 16; i++) z3[i] = 0.f;
#pragma unroll
        for (int jw = 0; jw < KW; jw++) {
            const int dd = jw - CW;
            float pr[16];
#pragma unroll
            for (int i = 0; i < 16; i++) {
                float v;
                if (dd == 0) {
                    v = z2[i];
                } else {
                    int src = cl + dd;
                    src = src < 0 ? 0 : (src > 31 ? 31 : src);
                    v = __shfl(z2[i], (lane & 32) | src, 64);
                }
                z3[i] += KwP[(i * 2 + hf) * KW + jw] * v;
                pr[i] = v * dz3[i];
            }
            if (rin && own) tap_add(jw, pr);
        }
        if (rin) {
            to_tile(z3);
            colgemm(accUt, MT, dYb, d.y_st, h);
        }
        // dZ2: transposed conv along w
        f32x16 dz2;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int jw = 0; jw < KW; jw++) {
                const int dd = jw - CW;
                float v;
                if (dd == 0) {
                    v = dz3[i];
                } else {
                    int src = cl - dd;
                    src = src < 0 ? 0 : (src > 31 ? 31 : src);
                    v = __shfl(dz3[i], (lane & 32) | src, 64);
                }
                a += KwP[(i * 2 + hf) * KW + jw] * v;
            }
            dz2[i] = a;
        }
        dr[KH - 1] = dz2;
        // dKh products
        if (rin && own) {
#pragma unroll
            for (int j = 0; j < KH; j++) {
                float pr[16];
#pragma unroll
                for (int i = 0; i < 16; i++) pr[i] = ring[j][i] * dz2[i];
                tap_add(KW + j, pr);
            }
        }
        // dZ1 for row h - CH
        f32x16 dz1;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < KH; j++) a += KhP[(i * 2 + hf) * KH + j] * dr[KH - 1 - j][i];
            dz1[i] = a;
        }
#pragma unroll
        for (int j = 0; j < KH - 1; j++) {
            ring[j] = ring[j + 1];
            dr[j] = dr[j + 1];
        }
        const int hx = h - CH;
        if (hx >= h0 && hx < h1) {
            if (dX) {
                f32x16 accX[MS];
#pragma unroll
                for (int n = 0; n < MS; n++)
#pragma unroll
                    for (int i = 0; i < 16; i++) accX[n][i] = 0.f;
                if constexpr (BF) {
#pragma unroll
                    for (int q = 0; q < 2; q++) {
                        bf16_t zb[8];
#pragma unroll
                        for (int j = 0; j < 8; j++) zb[j] = f32_to_bf16(dz1[8 * q + j]);
                        const bf16x8 bv = pack8(zb);
#pragma unroll
                        for (int n = 0; n < MS; n++) {
                            bf16x8 av = lds8(UsP + (((q * 2 + hf) * NS) + n * 32 + cl) * 8);
                            accX[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, accX[n], 0, 0, 0);
                        }
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 16; i++)
#pragma unroll
                        for (int n = 0; n < MS; n++)
                            accX[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(
                                UsP[(i * 2 + hf) * NS + n * 32 + cl], dz1[i], accX[n], 0, 0, 0);
                }
                if (own) {
                    T* xr = dX + (int64_t)b * d.x_sb + (int64_t)hx * W + col;
#pragma unroll
                    for (int n = 0; n < MS; n++)
#pragma unroll
                        for (int i = 0; i < 16; i++)
                            store(xr, (int64_t)(n * 32 + row32(i, lane)) * d.x_ss, accX[n][i]);
                }
            }
            to_tile(dz1);
            colgemm(accUs, MS, Xb, d.x_ss, hx);
        }
    }

    // ---- tap products summed over the lanes of each half (wave-private area,
    // read before any block-wide reuse of LDS) ----
    constexpr int NJ = KH + KW;
    // products of tap jj = 0..KW-1 (w) then KW..NJ-1 (h), 16 per tap; groups of
    // two taps; lane cl of a half ends with tap 2g + cl/16, accumulator cl%16
    float tsum[NG];
#pragma unroll
    for (int g = 0; g < NG; g++) {
        float v[32];
#pragma unroll
        for (int c = 0; c < 8; c++) {
            const float4 t4 = *(const float4*)(Tap + ((8 * g + c) * 64 + lane) * 4);
            v[4 * c] = t4.x;
            v[4 * c + 1] = t4.y;
            v[4 * c + 2] = t4.z;
            v[4 * c + 3] = t4.w;
        }
        tsum[g] = half_reduce32(v, cl);
    }

    // ---- block sums of the wavefront partials, in a fixed order ----
    __syncthreads();
    float* red = (float*)smem;
    const int64_t blk = blockIdx.x;
#pragma unroll
    for (int n = 0; n < MT; n++)
#pragma unroll
        for (int i = 0; i < 16; i++) red[wave * 32 * NT + row32(i, lane) * NT + 32 * n + cl] = accUt[n][i];
    __syncthreads();
    for (int e = tid; e < 32 * NT; e += 256)
        Put[blk * 32 * NT + e] = ((red[e] + red[32 * NT + e]) + red[64 * NT + e]) + red[96 * NT + e];
    __syncthreads();
#pragma unroll
    for (int n = 0; n < MS; n++)
#pragma unroll
        for (int i = 0; i < 16; i++) red[wave * 32 * NS + row32(i, lane) * NS + 32 * n + cl] = accUs[n][i];
    __syncthreads();
    for (int e = tid; e < 32 * NS; e += 256)
        Pus[blk * 32 * NS + e] = ((red[e] + red[32 * NS + e]) + red[64 * NS + e]) + red[96 * NS + e];
    __syncthreads();
#pragma unroll
    for (int g = 0; g < NG; g++) {
        const int jj = 2 * g + (cl >> 4), i = cl & 15;
        red[wave * 32 * NJ + row32(i, lane) * NJ + jj] = tsum[g];
    }
    __syncthreads();
    for (int e = tid; e < 32 * NJ; e += 256) {
        const int r = e / NJ, jj = e - r * NJ;
        const float v = ((red[e] + red[32 * NJ + e]) + red[64 * NJ + e]) + red[96 * NJ + e];
        if (jj < KW) Pkw[blk * 32 * KW + r * KW + jj] = v;
        else Pkh[blk * 32 * KH + r * KH + (jj - KW)] = v;
    }
}

constexpr uint32_t kMaxLds = 160 * 1024;   // LDS of one gfx950 CU

template <typename T, int K, int M>
hipError_t launch_cpb_t(const CpBwdDesc& d, const void* const* o, hipStream_t s) {
    auto k = cp_bwd<T, K, K, M, M>;
    // dynamic LDS above 64 KB has to be allowed per kernel, once per device
    static std::atomic<uint64_t> allowed{0};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || d.lds_bytes > kMaxLds) return hipErrorInvalidValue;
    if (!(allowed.load() & (1ull << dev))) {
        e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
        if (e != hipSuccess) return e;
        allowed.fetch_or(1ull << dev);
    }
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d, (const T*)o[0],
                       (const T*)o[1], (const T*)o[3], (const T*)o[4], (const T*)o[5], (const T*)o[6],
                       (T*)o[2], (float*)o[7], (float*)o[8], (float*)o[9], (float*)o[10]);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_cpb_ty(const CpBwdDesc& d, const void* const* o, hipStream_t s) {
    const int m = d.T / 32;
    if (d.KH == 3) return m == 1 ? launch_cpb_t<T, 3, 1>(d, o, s) : launch_cpb_t<T, 3, 2>(d, o, s);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    CpDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (d.R != 32 || !(d.T == 32 || d.T == 64)) return hipErrorInvalidValue;
    int bf = (ln.kind >> kBitIn) & 1;
    return bf ? launch_cp_ty<bf16_t>(d, ops, y, s) : launch_cp_ty<float>(d, ops, y, s);
}

// ops = {X, dY, dX (may be NULL), Us, Kh, Kw, Ut, Pus, Put, Pkh, Pkw}
hipError_t launch_cp_bwd(const Launch& ln, const void* const* ops, hipStream_t s) {
    CpBwdDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (d.R != 32 || d.S != d.T || !(d.T == 32 || d.T == 64) || d.KH != d.KW) return hipErrorInvalidValue;
    int bf = (ln.kind >> kBitIn) & 1;
    return bf ? launch_cpb_ty<bf16_t>(d, ops, s) : launch_cpb_ty<float>(d, ops, s);
}

}  // namespace ce
