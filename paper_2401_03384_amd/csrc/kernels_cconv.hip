// Convolution contracted over one channel index on bf16 MFMA tiles (CconvDesc):
//   Y[g][q][h][w] = sum_p sum_taps Z[g][p][h + dh][w + dw] * F[p][q][fh][fw]
// the pairwise step of a Tucker layer that convolves the core with the
// projected input (Section 2.3, Tucker convolutional layer; the implicit-GEMM
// lowering of a step with both a contraction and convolved labels), and the
// input gradient of such a step (the same form with the taps reversed).
//
// Per output tile it is a GEMM with M = 32 values of q, N = 32 pixels and
// K = taps x channels.  A block stages its filter slice and its input rows
// (with the zero halo) in LDS, channels innermost as bf16 pairs, so that one
// 16-byte LDS read gives a lane its eight consecutive k values of a
// 32x32x16 MFMA operand (lane l: A row / B column l % 32, k half l / 32).
// Each wavefront computes two pixel tiles against the same filter operand.
#include <atomic>
#include <cstdint>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) {
    bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// CB = Ppad / 16 channel blocks of one tap (compile time: the k loop of a tap unrolls)
// T = bf16_t: 32x32x16 bf16 MFMA, channels as bf16 pairs (Ppad = 16 CB);
// T = float: 32x32x2 fp32 MFMA, one channel a word (Ppad = 8 CB), odd pitches
template <int CB, typename T, typename TC>
__global__ void __launch_bounds__(256) cconv(CconvDesc d, const T* __restrict__ Z,
                                             const T* __restrict__ F, TC* __restrict__ Y) {
    constexpr bool BF = sizeof(T) == 2;
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    uint32_t* tab = lds;                        // [32][pw_tab]: word t * tp + pp of row q
    uint32_t* img = lds + 32 * d.pw_tab;        // [HP * WP][pw_img]: word pp of a pixel
    constexpr int PW2 = 8 * CB;                 // words of one tap's channels
    int64_t bid = blockIdx.x;
    const int qt = (int)(bid % d.nq);
    bid /= d.nq;
    const int tile = (int)(bid % d.ntiles);
    int64_t g = bid / d.ntiles;
    int64_t oz = 0, oy = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        const int64_t x = g % d.g_size[i];
        g /= d.g_size[i];
        oz += x * d.g_sZ[i];
        oy += x * d.g_sY[i];
    }
    const int h0 = tile * d.TH, th = min(d.TH, d.H - h0);
    const int q0 = qt * 32, KT = d.KH * d.KW;
    const int dhmin = min(d.zh0, d.zh0 + d.zhs * (d.KH - 1));
    const int dwmin = min(d.zw0, d.zw0 + d.zws * (d.KW - 1));
    // Staging: a thread takes one (q, tap) of the filter slice, then one pixel
    // of the input rows, and loads all its channel pairs (2pp, 2pp + 1) before
    // writing them to LDS four words at a time.  Raw buffer loads: the lane's
    // byte offset in a register, the channel step a wave-uniform offset;
    // offsets past the range (q past Q, pixels outside the plane) read 0.
    constexpr uint32_t kOut = 0x80000000u;
    constexpr uint32_t E = sizeof(T);
    const __amdgpu_buffer_rsrc_t rF = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(F), (short)0, (int)(E * d.f_numel), 0x00020000);
    const __amdgpu_buffer_rsrc_t rZ =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(Z + oz), (short)0, (int)(E * (d.z_numel - oz)), 0x00020000);
    // fp32: one channel a word, written one word at a time (odd pitches)
    auto chans = [&](__amdgpu_buffer_rsrc_t r, uint32_t voff, int64_t sp, uint32_t* dst) {
        uint32_t w[PW2];
#pragma unroll
        for (int p = 0; p < PW2; p++) {
            const bool ok = p < d.P;
            const uint32_t v = __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, ok ? (int)(4 * p * sp) : 0, 0);
            w[p] = ok ? v : 0u;
        }
#pragma unroll
        for (int p = 0; p < PW2; p++) dst[p] = w[p];
    };
    auto pairs = [&](__amdgpu_buffer_rsrc_t r, uint32_t voff, int64_t sp, uint32_t* dst) {
        uint32_t w[PW2];
#pragma unroll
        for (int pp = 0; pp < PW2; pp++) {
            // no branches around the loads (a branch makes the wave wait for
            // each pair in turn): channels past P load channel 0 and are masked
            const int p = 2 * pp;
            const bool ok0 = p < d.P, ok1 = p + 1 < d.P;
            const uint32_t lo = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, ok0 ? (int)(2 * p * sp) : 0, 0);
            const uint32_t hi = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, ok1 ? (int)(2 * (p + 1) * sp) : 0, 0);
            w[pp] = (ok0 ? lo : 0u) | ((ok1 ? hi : 0u) << 16);
        }
#pragma unroll
        for (int u = 0; u < PW2; u += 4)
            *reinterpret_cast<uint4*>(dst + u) = make_uint4(w[u], w[u + 1], w[u + 2], w[u + 3]);
    };
    for (int ct = threadIdx.x; ct < 32 * KT; ct += 256) {
        const int q = ct / KT, t = ct - q * KT, tr = t / d.KW, tc = t - tr * d.KW;
        const int64_t o = (int64_t)(q0 + q) * d.f_sq + (int64_t)(d.fh0 + d.fhs * tr) * d.f_sh +
                          (int64_t)(d.fw0 + d.fws * tc) * d.f_sw;
        const uint32_t voff = q0 + q < d.Q ? (uint32_t)(E * o) : kOut;
        if constexpr (BF) pairs(rF, voff, d.f_sp, tab + q * d.pw_tab + t * d.tp);
        else chans(rF, voff, d.f_sp, tab + q * d.pw_tab + t * d.tp);
    }
    // input rows h0 + dhmin .. (HP rows), columns dwmin .. (WP)
    for (int px = threadIdx.x; px < d.HP * d.WP; px += 256) {
        const int rr = px / d.WP, cc = px - rr * d.WP;
        const int hh = h0 + dhmin + rr, ww = dwmin + cc;
        const bool in = hh >= 0 && hh < d.H && ww >= 0 && ww < d.W;
        const uint32_t voff = in ? (uint32_t)(E * (hh * d.W + ww)) : kOut;
        if constexpr (BF) pairs(rZ, voff, d.z_sp, img + px * d.pw_img);
        else chans(rZ, voff, d.z_sp, img + px * d.pw_img);
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), hf = lane >> 5, cl = lane & 31;
    const int npx = th * d.W, ptiles = (npx + 31) / 32;
    const uint32_t* arow = tab + cl * d.pw_tab + (BF ? 4 * hf : hf);
    for (int pt = 2 * wave; pt < ptiles; pt += 8) {
        const int n0 = pt * 32 + cl, n1 = n0 + 32;
        const bool v0 = n0 < npx, v1 = n1 < npx;
        // pixels past the tile read pixel 0 (in the LDS tile) and store nothing
        const int r0 = v0 ? n0 / d.W : 0, c0 = v0 ? n0 - r0 * d.W : 0;
        const int r1 = v1 ? n1 / d.W : 0, c1 = v1 ? n1 - r1 * d.W : 0;
        f32x16 acc0, acc1;
#pragma unroll
        for (int i = 0; i < 16; i++) acc0[i] = acc1[i] = 0.f;
        for (int t = 0; t < KT; t++) {
            const int tr = t / d.KW, tc = t - tr * d.KW;
            const int dr = d.zh0 + d.zhs * tr - dhmin, dc = d.zw0 + d.zws * tc - dwmin;
            const uint32_t* b0 = img + ((r0 + dr) * d.WP + c0 + dc) * d.pw_img + (BF ? 4 * hf : hf);
            const uint32_t* b1 = img + ((r1 + dr) * d.WP + c1 + dc) * d.pw_img + (BF ? 4 * hf : hf);
            const uint32_t* a = arow + t * d.tp;
            if constexpr (!BF) {
                // k step of two channels: lane half hf supplies channel 2i + hf
                float af[4 * CB], bf0[4 * CB], bf1[4 * CB];
#pragma unroll
                for (int i = 0; i < 4 * CB; i++) {
                    af[i] = __uint_as_float(a[2 * i]);
                    bf0[i] = __uint_as_float(b0[2 * i]);
                    bf1[i] = __uint_as_float(b1[2 * i]);
                }
#pragma unroll
                for (int i = 0; i < 4 * CB; i++) {
                    acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf0[i], acc0, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i], bf1[i], acc1, 0, 0, 0);
                }
                continue;
            }
            uint4 av[CB], bv0[CB], bv1[CB];
#pragma unroll
            for (int cb = 0; cb < CB; cb++) {
                av[cb] = *reinterpret_cast<const uint4*>(a + 8 * cb);
                bv0[cb] = *reinterpret_cast<const uint4*>(b0 + 8 * cb);
                bv1[cb] = *reinterpret_cast<const uint4*>(b1 + 8 * cb);
            }
#pragma unroll
            for (int cb = 0; cb < CB; cb++) {
                acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(av[cb]), as_bf16x8(bv0[cb]), acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(av[cb]), as_bf16x8(bv1[cb]), acc1, 0, 0, 0);
            }
        }
        // accumulator i of a lane: q = q0 + 8(i/4) + 4hf + i%4, pixel = the lane's
#pragma unroll
        for (int i = 0; i < 16; i++) {
            const int q = q0 + 8 * (i >> 2) + 4 * hf + (i & 3);
            if (q < d.Q) {
                const int64_t oq = oy + q * d.y_sq;
                if (v0) store(Y, oq + (int64_t)(h0 + r0) * d.W + c0, acc0[i]);
                if (v1) store(Y, oq + (int64_t)(h0 + r1) * d.W + c1, acc1[i]);
            }
        }
    }
}

// fp32, at most eight channels and KT taps (rega; KT = KH KW, compile time): a block takes one g and
// one row tile for every q tile, LDS holds its input rows only.  The block's
// work items (q tile, pair of pixel tiles) are split into four contiguous
// runs, one a wavefront; a wavefront keeps its q tile's filter operands in
// registers (tap t, k step i: channel 2i + hf of row q0 + cl, zero past P and
// Q) and loads the next tap's pixel operands while the current tap's MFMAs
// run.  The stores are range-checked buffer stores over the g's span of Y:
// pixels past the tile and q past Q carry an offset past the range and are
// dropped.
// s_waitcnt vmcnt(0), the other counters at their maximum (expcnt 7, lgkmcnt 15)
constexpr int kVmcnt0 = 0x0F70;

template <int KT>
__global__ void __launch_bounds__(256) cconv_r(CconvDesc d, const float* __restrict__ Z,
                                               const float* __restrict__ F, float* __restrict__ Y) {
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    const float* img = reinterpret_cast<const float*>(lds);   // [HP * WP][pw_img]
    int64_t bid = blockIdx.x;
    const int tile = (int)(bid % d.ntiles);
    int64_t g = bid / d.ntiles;
    int64_t oz = 0, oy = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        const int64_t x = g % d.g_size[i];
        g /= d.g_size[i];
        oz += x * d.g_sZ[i];
        oy += x * d.g_sY[i];
    }
    const int h0 = tile * d.TH, th = min(d.TH, d.H - h0);
    const int dhmin = min(d.zh0, d.zh0 + d.zhs * (d.KH - 1));
    const int dwmin = min(d.zw0, d.zw0 + d.zws * (d.KW - 1));
    constexpr uint32_t kOut = 0x80000000u;
    const __amdgpu_buffer_rsrc_t rZ =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(Z + oz), (short)0, (int)(4 * (d.z_numel - oz)), 0x00020000);
    // input rows h0 + dhmin .. (HP rows), columns dwmin .. (WP): a thread loads
    // the eight channels of four pixels (px, px + 256, ...) before writing any,
    // so that a block's staging waits for one round of loads, not four
    const int npix = d.HP * d.WP;
    for (int px0 = 0; px0 < npix; px0 += 1024) {
        uint32_t w[4][8];
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int px = px0 + 256 * j + (int)threadIdx.x;
            const int rr = px / d.WP, cc = px - rr * d.WP;
            const int hh = h0 + dhmin + rr, ww = dwmin + cc;
            const bool in = px < npix && hh >= 0 && hh < d.H && ww >= 0 && ww < d.W;
            const uint32_t voff = in ? (uint32_t)(4 * (hh * d.W + ww)) : kOut;
#pragma unroll
            for (int p = 0; p < 8; p++) {
                const bool ok = p < d.P;
                const uint32_t v = __builtin_amdgcn_raw_buffer_load_b32(rZ, (int)voff, ok ? (int)(4 * p * d.z_sp) : 0, 0);
                w[j][p] = ok ? v : 0u;
            }
        }
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int px = px0 + 256 * j + (int)threadIdx.x;
            if (px < npix) {
                uint32_t* dst = lds + px * d.pw_img;
#pragma unroll
                for (int p = 0; p < 8; p++) dst[p] = w[j][p];
            }
        }
    }
    __syncthreads();
    // the wavefront index is uniform: the item range, q tile and pair below are scalars
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int hf = lane >> 5, cl = lane & 31;
    const int npx = __builtin_amdgcn_readfirstlane(th * d.W), ptiles = (npx + 31) / 32, npairs = (ptiles + 1) / 2;
    const int items = d.nq * npairs, per = (items + 3) / 4;
    const int it0 = __builtin_amdgcn_readfirstlane(wave * per), it1 = __builtin_amdgcn_readfirstlane(min(items, it0 + per));
    // LDS word offset of tap t from a pixel's own word (wave-uniform)
    int toff[KT];
#pragma unroll
    for (int t = 0; t < KT; t++) {
        const int tr = t / d.KW, tc = t - tr * d.KW;
        toff[t] = ((d.zh0 + d.zhs * tr - dhmin) * d.WP + (d.zw0 + d.zws * tc - dwmin)) * d.pw_img;
    }
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(Y + oy, (short)0, (int)(4 * d.y_ext), 0x00020000);
    float a[KT][4];
    int cur = -1;
    for (int it = it0; it < it1; it++) {
        const int qt = __builtin_amdgcn_readfirstlane(it / npairs), pr = it - qt * npairs, q0 = 32 * qt;
        if (qt != cur) {
            cur = qt;
            const int q = q0 + cl;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int tr = t / d.KW, tc = t - tr * d.KW;
                const int64_t o = (int64_t)q * d.f_sq + (int64_t)(d.fh0 + d.fhs * tr) * d.f_sh +
                                  (int64_t)(d.fw0 + d.fws * tc) * d.f_sw;
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int p = 2 * i + hf;
                    a[t][i] = (q < d.Q && p < d.P) ? F[o + p * d.f_sp] : 0.f;
                }
            }
            // complete these loads here: the vector-memory counter also counts
            // the previous item's stores, and a wait at the first MFMA (where
            // the compiler cannot tell whether this block ran) would drain them
            __builtin_amdgcn_s_waitcnt(kVmcnt0);
        }
        const int n0 = 64 * pr + cl, n1 = n0 + 32;
        const bool v0 = n0 < npx, v1 = n1 < npx;
        // pixels past the tile read pixel 0 (in the LDS tile) and store nothing
        const int r0 = v0 ? n0 / d.W : 0, c0 = v0 ? n0 - r0 * d.W : 0;
        const int r1 = v1 ? n1 / d.W : 0, c1 = v1 ? n1 - r1 * d.W : 0;
        const float* b0 = img + (r0 * d.WP + c0) * d.pw_img + hf;
        const float* b1 = img + (r1 * d.WP + c1) * d.pw_img + hf;
        f32x16 acc0, acc1;
#pragma unroll
        for (int i = 0; i < 16; i++) acc0[i] = acc1[i] = 0.f;
        // a pair whose second tile is past the plane computes it from pixel 0
        // and stores nothing (every lane's n1 is past npx)
        float x0[2][4], x1[2][4];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            x0[0][i] = b0[toff[0] + 2 * i];
            x1[0][i] = b1[toff[0] + 2 * i];
        }
#pragma unroll
        for (int t = 0; t < KT; t++) {
            const int cb = t & 1, nb = cb ^ 1;
            if (t + 1 < KT) {
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    x0[nb][i] = b0[toff[t + 1 < KT ? t + 1 : t] + 2 * i];
                    x1[nb][i] = b1[toff[t + 1 < KT ? t + 1 : t] + 2 * i];
                }
            }
#pragma unroll
            for (int i = 0; i < 4; i++) {
                acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t][i], x0[cb][i], acc0, 0, 0, 0);
                acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t][i], x1[cb][i], acc1, 0, 0, 0);
            }
        }
        // accumulator i of a lane: q = q0 + 8(i/4) + 4hf + i%4, pixel = the lane's
        const int64_t ob0 = (int64_t)(q0 + 4 * hf) * d.y_sq + (int64_t)h0 * d.W;
        const uint32_t p0 = (uint32_t)(4 * (ob0 + r0 * d.W + c0)), p1 = (uint32_t)(4 * (ob0 + r1 * d.W + c1));
        const bool fullq = q0 + 32 <= d.Q;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            const int dq = 8 * (i >> 2) + (i & 3);
            const bool qok = fullq || q0 + 4 * hf + dq < d.Q;
            // wave-uniform; zero where no lane has a q below Q (no overflow)
            const int so = dq < d.Q - q0 ? (int)(4 * dq * d.y_sq) : 0;
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc0[i]), rY, (v0 && qok) ? (int)p0 : (int)kOut, so, 0);
            __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc1[i]), rY, (v1 && qok) ? (int)p1 : (int)kOut, so, 0);
        }
    }
}

template <int KT>
hipError_t cconv_r_go(const CconvDesc& d, dim3 g, const void* z, const void* f, void* y, hipStream_t s) {
    auto k = cconv_r<KT>;
    static std::atomic<uint64_t> allowed{0};
    if (d.lds_bytes > 64 * 1024) {
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        if (dev < 0 || dev >= 64) return hipErrorInvalidValue;
        if (!(allowed.load() & (1ull << dev))) {
            e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e != hipSuccess) return e;
            allowed.fetch_or(1ull << dev);
        }
    }
    hipLaunchKernelGGL(k, g, dim3(256), d.lds_bytes, s, d, (const float*)z, (const float*)f, (float*)y);
    return hipGetLastError();
}

template <int CB, typename T, typename TC>
hipError_t cconv_go(const CconvDesc& d, dim3 g, const void* z, const void* f, void* y, hipStream_t s) {
    auto k = cconv<CB, T, TC>;
    // dynamic LDS above 64 KB has to be allowed per kernel, once per device
    static std::atomic<uint64_t> allowed{0};
    if (d.lds_bytes > 64 * 1024) {
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        if (dev < 0 || dev >= 64) return hipErrorInvalidValue;
        if (!(allowed.load() & (1ull << dev))) {
            e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e != hipSuccess) return e;
            allowed.fetch_or(1ull << dev);
        }
    }
    hipLaunchKernelGGL(k, g, dim3(256), d.lds_bytes, s, d, (const T*)z, (const T*)f, (TC*)y);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_cconv(const Launch& ln, const void* z, const void* f, void* y, hipStream_t s) {
    CconvDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    const int CB = d.Ppad / (tIn ? 16 : 8);
    if (d.rega) {
        // fp32, P <= 8, at most nine taps, the input rows alone in LDS, every
        // q tile in one block, the g's span of Y within 32-bit byte offsets
        if (tIn || tC || d.Ppad != 8 || d.P < 1 || d.P > 8 || d.pw_img != 9 || d.KH < 1 || d.KW < 1 ||
            d.KH * d.KW > 9 || d.TH < 1 || d.HP != d.TH + d.KH - 1 || d.WP != d.W + d.KW - 1 || d.nq * 32 < d.Q ||
            d.nq < 1 || d.Q < 1 || d.z_numel <= 0 || d.z_numel >= (1ll << 30) || d.f_numel <= 0 ||
            d.f_numel >= (1ll << 30) || (int64_t)d.ntiles * d.TH < d.H || d.y_sq < 1 ||
            d.y_ext != (int64_t)(d.Q - 1) * d.y_sq + (int64_t)d.H * d.W || d.y_ext * 4 >= (1ll << 31) ||
            d.lds_bytes != 4u * (uint32_t)(d.HP * d.WP * d.pw_img) || d.lds_bytes > 160 * 1024 ||
            (int64_t)ln.grid[0] != d.G * d.ntiles || d.blocks != (int64_t)ln.grid[0])
            return hipErrorInvalidValue;
        const dim3 g(ln.grid[0]);
        switch (d.KH * d.KW) {
            case 1: return cconv_r_go<1>(d, g, z, f, y, s);
            case 2: return cconv_r_go<2>(d, g, z, f, y, s);
            case 3: return cconv_r_go<3>(d, g, z, f, y, s);
            case 4: return cconv_r_go<4>(d, g, z, f, y, s);
            case 5: return cconv_r_go<5>(d, g, z, f, y, s);
            case 6: return cconv_r_go<6>(d, g, z, f, y, s);
            case 7: return cconv_r_go<7>(d, g, z, f, y, s);
            case 8: return cconv_r_go<8>(d, g, z, f, y, s);
            default: return cconv_r_go<9>(d, g, z, f, y, s);
        }
    }
    // the descriptor's LDS layout is the one the kernel indexes
    const bool lay = tIn ? (d.Ppad == 16 * CB && d.pw_img == 8 * CB + 4 && d.tp == 8 * CB + 4 && !(d.pw_tab & 3))
                         : (d.Ppad == 8 * CB && d.pw_img == 8 * CB + 1 && d.tp == 8 * CB && (d.pw_tab & 1));
    if (!(CB == 1 || CB == 2 || CB == 4 || CB == 8) || !lay || (!tIn && tC) || d.TH < 1 || d.HP != d.TH + d.KH - 1 ||
        d.WP != d.W + d.KW - 1 || d.pw_tab < d.KH * d.KW * d.tp ||
        d.P > d.Ppad || d.nq * 32 < d.Q || d.z_numel <= 0 || d.z_numel >= (1ll << 30) || d.f_numel <= 0 ||
        d.f_numel >= (1ll << 30) || (int64_t)d.ntiles * d.TH < d.H ||
        d.lds_bytes != 4u * (uint32_t)(32 * d.pw_tab + d.HP * d.WP * d.pw_img) || d.lds_bytes > 160 * 1024 ||
        (int64_t)ln.grid[0] != d.G * d.ntiles * d.nq || d.blocks != (int64_t)ln.grid[0])
        return hipErrorInvalidValue;
    const dim3 g(ln.grid[0]);
#define CC_CASE(cb)                                                                          \
    case cb:                                                                                 \
        if (!tIn) return cconv_go<cb, float, float>(d, g, z, f, y, s);                      \
        if (tC) return cconv_go<cb, bf16_t, bf16_t>(d, g, z, f, y, s);                      \
        return cconv_go<cb, bf16_t, float>(d, g, z, f, y, s);
    switch (CB) {
        CC_CASE(1)
        CC_CASE(2)
        CC_CASE(4)
        CC_CASE(8)
    }
#undef CC_CASE
    return hipErrorInvalidValue;
}

}  // namespace ce
