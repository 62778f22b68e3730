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

}  // namespace

hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    CpDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (d.R != 32 || !(d.T == 32 || d.T == 64)) return hipErrorInvalidValue;
    int bf = (ln.kind >> kBitIn) & 1;
    return bf ? launch_cp_ty<bf16_t>(d, ops, y, s) : launch_cp_ty<float>(d, ops, y, s);
}

}  // namespace ce
