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
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hf = lane >> 5, cl = lane & 31;
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
