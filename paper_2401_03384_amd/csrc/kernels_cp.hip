// Fused CP chain for gfx950: the four forward steps of a CP-factorised 2-D
// convolution layer (Section 2.3, CP convolutional layer; the pairwise steps
// the sequencer picks for it: contract s, convolve h, convolve w, contract r)
// in one kernel, so the rank-R intermediates never leave the CU.
//
// A block owns seg_rows image rows of one sample and walks them in chunks of
// TH rows.  Per chunk:
//   GEMM1  Z1 rows entering the ring:  Z1[r][p] = sum_s Us[r][s] X[s][p]
//          (X staged through LDS in 32-channel slices; bf16 staged transposed
//          so each lane reads one 16-byte k-run per MFMA)
//   conv_h Z2[row][r][w] from the ring of KH-1 + TH rows of Z1
//   conv_w Z3 (MFMA-ready layout, zero padding at the row ends)
//   GEMM2  Y[t][p] = sum_r Ut[r][t] Z3[r][p], stored from the accumulators.
// Rows outside the image are zero in the ring (same padding of conv_h).
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

__device__ __forceinline__ int row32(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// CBW column blocks of 32 pixels per wave at most; M blocks (R/32, T/32) at most 2.
template <typename T, int NW, int CBW>
__global__ void __launch_bounds__(NW * 64) cp_fwd(CpDesc d, const T* __restrict__ X,
                                                  const T* __restrict__ Us, const T* __restrict__ Kh,
                                                  const T* __restrict__ Kw, const T* __restrict__ Ut,
                                                  T* __restrict__ Y) {
    constexpr bool BF = sizeof(T) == 2;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    T* UsL = (T*)(smem + d.o_us);
    T* UtL = (T*)(smem + d.o_ut);
    float* KhL = (float*)(smem + d.o_kh);
    float* KwL = (float*)(smem + d.o_kw);
    float* ring = (float*)(smem + d.o_ring);
    float* Z2 = (float*)(smem + d.o_z2);
    unsigned char* XZ = smem + d.o_xz;
    const int R = d.R, S = d.S, TT = d.T, W = d.W, H = d.H, KH = d.KH, KW = d.KW, TH = d.TH;
    const int NR = d.nr, PXP = d.pxp, LDA = d.lda, LDU = d.ldu;
    const int ch = (KH - 1) / 2, cw = (KW - 1) / 2;
    const int nmb = R / 32, nmb2 = TT / 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = (int)(blockIdx.x / d.segs), seg = (int)(blockIdx.x % d.segs);
    const int h_begin = seg * d.seg_rows;
    const int h_end = min(H, h_begin + d.seg_rows);
    if (h_begin >= h_end) return;   // whole block

    for (int e = tid; e < R * S; e += NW * 64) {
        int r = e / S, s = e - r * S;
        UsL[r * LDA + s] = Us[r * d.us_sr + s * d.us_ss];
    }
    for (int e = tid; e < TT * R; e += NW * 64) {
        int t = e / R, r = e - t * R;
        UtL[t * LDU + r] = Ut[r * d.ut_sr + t * d.ut_st];
    }
    for (int e = tid; e < R * KH; e += NW * 64) {
        int r = e / KH, j = e - r * KH;
        KhL[e] = load(Kh, r * d.kh_sr + j * d.kh_sj);
    }
    for (int e = tid; e < R * KW; e += NW * 64) {
        int r = e / KW, j = e - r * KW;
        KwL[e] = load(Kw, r * d.kw_sr + j * d.kw_sj);
    }
    __syncthreads();

    const T* Xb = X + (int64_t)b * d.x_sb;
    T* Yb = Y + (int64_t)b * d.y_sb;
    const int base_row = h_begin - ch;
    auto slot = [&](int hh) { return (hh - base_row) % NR; };

    // Z1 for image rows [r0, r0 + nr), nr <= TH, into the ring
    auto gemm1 = [&](int r0, int nr) {
        const int np = nr * W, ncb = (np + 31) / 32;
        f32x16 acc[CBW][2];
#pragma unroll
        for (int c = 0; c < CBW; c++)
#pragma unroll
            for (int mb = 0; mb < 2; mb++)
#pragma unroll
                for (int i = 0; i < 16; i++) acc[c][mb][i] = 0.f;
        for (int s0 = 0; s0 < S; s0 += 32) {
            for (int e = tid; e < 32 * PXP; e += NW * 64) {
                int ss = e / PXP, px = e - ss * PXP;
                int row = r0 + px / W;
                T v = (T)0;
                if (px < np && row >= 0 && row < H)
                    v = Xb[(int64_t)(s0 + ss) * d.x_ss + (int64_t)r0 * W + px];
                if constexpr (BF)
                    ((bf16_t*)XZ)[px * 40 + ss] = v;
                else
                    ((float*)XZ)[ss * PXP + px] = v;
            }
            __syncthreads();
#pragma unroll
            for (int c = 0; c < CBW; c++) {
                int cb = wave + c * NW;
                if (cb < ncb) {
                    if constexpr (BF) {
#pragma unroll
                        for (int kk = 0; kk < 32; kk += 16) {
                            bf16x8 bv = lds8((const bf16_t*)XZ + (cb * 32 + (lane & 31)) * 40 + kk + 8 * (lane >> 5));
#pragma unroll
                            for (int mb = 0; mb < 2; mb++)
                                if (mb < nmb) {
                                    bf16x8 av = lds8((const bf16_t*)UsL + (mb * 32 + (lane & 31)) * LDA + s0 + kk + 8 * (lane >> 5));
                                    acc[c][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[c][mb], 0, 0, 0);
                                }
                        }
                    } else {
#pragma unroll 4
                        for (int kk = 0; kk < 32; kk += 2) {
                            float bv = ((const float*)XZ)[(kk + (lane >> 5)) * PXP + cb * 32 + (lane & 31)];
#pragma unroll
                            for (int mb = 0; mb < 2; mb++)
                                if (mb < nmb) {
                                    float av = ((const float*)UsL)[(mb * 32 + (lane & 31)) * LDA + s0 + kk + (lane >> 5)];
                                    acc[c][mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[c][mb], 0, 0, 0);
                                }
                        }
                    }
                }
            }
            __syncthreads();
        }
#pragma unroll
        for (int c = 0; c < CBW; c++) {
            int cb = wave + c * NW;
            int px = cb * 32 + (lane & 31);
            if (cb < ncb && px < np) {
                int row = r0 + px / W, w = px - (px / W) * W;
                float* dst = ring + (size_t)slot(row) * R * W + w;
#pragma unroll
                for (int mb = 0; mb < 2; mb++)
                    if (mb < nmb)
#pragma unroll
                        for (int i = 0; i < 16; i++) dst[(mb * 32 + row32(i, lane)) * W] = acc[c][mb][i];
            }
        }
    };

    // fill the ring with the KH-1 rows above the first chunk's lookahead
    {
        int pre = KH - 1;
        for (int r0 = base_row; r0 < base_row + pre; r0 += TH) gemm1(r0, min(TH, base_row + pre - r0));
    }
    for (int h = h_begin; h < h_end; h += TH) {
        const int nr = min(TH, h_end - h);
        // rows entering the ring: [h + KH-1-ch, h + nr + KH-1-ch)
        gemm1(h + (KH - 1 - ch), nr);
        __syncthreads();
        // conv along h
        for (int e = tid; e < nr * R * W; e += NW * 64) {
            int row = e / (R * W), rem = e - row * R * W, r = rem / W, w = rem - r * W;
            float a = 0.f;
            for (int j = 0; j < KH; j++)
                a += ring[((size_t)slot(h + row + j - ch) * R + r) * W + w] * KhL[r * KH + j];
            Z2[e] = a;
        }
        __syncthreads();
        // conv along w into the MFMA layout of Z3
        const int np = nr * W;
        for (int e = tid; e < R * PXP; e += NW * 64) {
            int r = e / PXP, px = e - r * PXP;
            float a = 0.f;
            if (px < np) {
                int row = px / W, w = px - row * W;
                const float* z = Z2 + ((size_t)row * R + r) * W;
                for (int j = 0; j < KW; j++) {
                    int ww = w + j - cw;
                    if (ww >= 0 && ww < W) a += z[ww] * KwL[r * KW + j];
                }
            }
            if constexpr (BF)
                ((bf16_t*)XZ)[px * LDU + r] = f32_to_bf16(a);
            else
                ((float*)XZ)[r * PXP + px] = a;
        }
        __syncthreads();
        // GEMM2 and store
        const int ncb = (np + 31) / 32;
#pragma unroll
        for (int c = 0; c < CBW; c++) {
            int cb = wave + c * NW;
            if (cb >= ncb) continue;
            f32x16 acc[2];
#pragma unroll
            for (int mb = 0; mb < 2; mb++)
#pragma unroll
                for (int i = 0; i < 16; i++) acc[mb][i] = 0.f;
            if constexpr (BF) {
                for (int kk = 0; kk < R; kk += 16) {
                    bf16x8 bv = lds8((const bf16_t*)XZ + (cb * 32 + (lane & 31)) * LDU + kk + 8 * (lane >> 5));
#pragma unroll
                    for (int mb = 0; mb < 2; mb++)
                        if (mb < nmb2) {
                            bf16x8 av = lds8((const bf16_t*)UtL + (mb * 32 + (lane & 31)) * LDU + kk + 8 * (lane >> 5));
                            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[mb], 0, 0, 0);
                        }
                }
            } else {
#pragma unroll 4
                for (int kk = 0; kk < R; kk += 2) {
                    float bv = ((const float*)XZ)[(kk + (lane >> 5)) * PXP + cb * 32 + (lane & 31)];
#pragma unroll
                    for (int mb = 0; mb < 2; mb++)
                        if (mb < nmb2) {
                            float av = ((const float*)UtL)[(mb * 32 + (lane & 31)) * LDU + kk + (lane >> 5)];
                            acc[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[mb], 0, 0, 0);
                        }
                }
            }
            int px = cb * 32 + (lane & 31);
            if (px < np) {
                T* dst = Yb + (int64_t)h * W + px;
#pragma unroll
                for (int mb = 0; mb < 2; mb++)
                    if (mb < nmb2)
#pragma unroll
                        for (int i = 0; i < 16; i++) store(dst, (int64_t)(mb * 32 + row32(i, lane)) * d.y_st, acc[mb][i]);
            }
        }
        __syncthreads();
    }
}

}  // namespace



hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    CpDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    int bf = (ln.kind >> kBitIn) & 1;
    dim3 g((uint32_t)d.blocks), bl(d.nthreads);
    size_t lds = d.lds_bytes;
    if (d.nthreads != 256) return hipErrorInvalidValue;
    if (bf) {
        auto k = cp_fwd<bf16_t, 4, 2>;
        hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k, g, bl, lds, s, d, (const bf16_t*)ops[0], (const bf16_t*)ops[1],
                           (const bf16_t*)ops[2], (const bf16_t*)ops[3], (const bf16_t*)ops[4], (bf16_t*)y);
    } else {
        auto k = cp_fwd<float, 4, 2>;
        hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL(k, g, bl, lds, s, d, (const float*)ops[0], (const float*)ops[1],
                           (const float*)ops[2], (const float*)ops[3], (const float*)ops[4], (float*)y);
    }
    return hipGetLastError();
}

}  // namespace ce
