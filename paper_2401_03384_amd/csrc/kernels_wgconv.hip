// Filter gradient of a plane convolution contracted over one shared index, on
// fp32 16x16x4 MFMA tiles (CredDesc; the same partial sums as K_CREDW):
//
//   P[chunk][u][m][tap] = sum_{g in chunk} sum_j Z[g][u][j + tap - c] * O[g][m][j]
//                       = sum_{g in chunk} sum_p Z[g][u][p] * O[g][m][p - tap + c]
//
// (Appendix B: g2 of a convolution step, the output gradient correlated with
// the step's input over every pixel and batch index).  Moving the shift from
// Z onto O, the second form reads every Z value once, unshifted: Z is the
// large operand (one plane per rank index u and batch index g), O the other
// one.  As a matrix product: rows u, columns n = (m, tap), reduction over
// (g, p).  Planes are fp32 or bf16 (converted to fp32 as they load; the
// products and sums are fp32).
//
// A block is four wavefronts with RT row tiles of 16 each (64 RT rows of u)
// and NT column tiles of 16 (a column block: the block stages only the planes
// of O its columns need).  The pixels of one plane go in groups of 16: lane
// (i, kq) (i = lane % 16, kq = lane / 16) loads Z[u0 + i][q0 + 4kq .. +3] with
// one 16-byte (fp32) or 8-byte (bf16) load per row tile; element t of it is
// the lane's K value of the group's MFMA t (pixel q0 + 4kq + t).  The column
// operand of MFMA t is O at the lane's column (m, tap) and the pixel
// q0 + 4kq + t shifted by the tap, read from LDS, where the planes of the
// current g sit with a zero halo (tap offsets are constant per lane).  The
// planes of g + 1 load into registers while g's groups run (double-buffered
// LDS); the row loads run kWgSlots groups ahead, each into the register
// slot it is computed from.
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

constexpr int kWgStage = 8;   // float4 of the next planes a thread holds while it computes
constexpr int kWgSlots = 3;   // register slots of row loads (items loaded ahead of the one computed)

__device__ __forceinline__ int64_t wg_zoff(const CredDesc& d, int64_t g) {
    int64_t oz = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        oz += (g % d.g_size[i]) * d.g_sZ[i];
        g /= d.g_size[i];
    }
    return oz;
}
__device__ __forceinline__ int64_t wg_ooff(const CredDesc& d, int64_t g) {
    int64_t oy = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        oy += (g % d.g_size[i]) * d.g_sY[i];
        g /= d.g_size[i];
    }
    return oy;
}

// Raw buffer loads (a wave-uniform resource: base and byte range; per-lane
// byte offsets): offsets past the range read zero, so a load needs no guard.
constexpr int kWgOut = (int)0x80000000u;
__device__ __forceinline__ float4 bld4(__amdgpu_buffer_rsrc_t r, int voff, float*) {
    typedef float f4 __attribute__((ext_vector_type(4)));
    const f4 v = __builtin_bit_cast(f4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 bld4(__amdgpu_buffer_rsrc_t r, int voff, bf16_t*) {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    const u2 u = __builtin_bit_cast(u2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, 0, 0));
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ float bld1(__amdgpu_buffer_rsrc_t r, int voff, float*) {
    return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, 0, 0));
}
__device__ __forceinline__ float bld1(__amdgpu_buffer_rsrc_t r, int voff, bf16_t*) {
    return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, voff, 0, 0) << 16);
}

// four consecutive elements from p (fp32: one 16-byte load; bf16: one 8-byte load)
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld4(const bf16_t* p) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
}

template <typename T, int RT, int NT, bool VEC>
__global__ void __launch_bounds__(256, 2) wgconv(CredDesc d, const T* __restrict__ Z, const T* __restrict__ O,
                                                 float* __restrict__ P) {
    extern __shared__ float4 lds4[];
    float* pl = reinterpret_cast<float*>(lds4);
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int W = d.W, HW = d.H * d.W, WP = d.PWp, PLN = d.PH * d.PWp;
    const int KK = d.KH * d.KW, N = d.M * KK, BUF = d.mb * PLN;
    const int top = d.KH - 1 - d.ch, left = d.KW - 1 - d.cw;   // halo before the interior
    const int64_t ub = blockIdx.x % d.nrb, rest = blockIdx.x / d.nrb;
    const int cb = (int)(rest % d.ncb);
    const int64_t ck = rest / d.ncb;
    const int64_t g0 = ck * d.gchunk, g1 = min(d.G, g0 + d.gchunk);
    const int i16 = lane & 15, kq = lane >> 4;
    // this block's columns and the planes of O they read
    const int n0 = cb * 16 * NT, mlo = n0 / KK;
    const int mhi = min(d.M, (n0 + 16 * NT - 1) / KK + 1), MB = mhi - mlo;
    // rows of this wavefront's row tiles
    const int64_t urow = ub * 64 * RT + wave * 16 * RT + i16;
    bool rok[RT];
    int64_t zr[RT];
#pragma unroll
    for (int mt = 0; mt < RT; mt++) {
        rok[mt] = urow + 16 * mt < d.R;
        zr[mt] = (rok[mt] ? urow + 16 * mt : 0) * d.z_sr;
    }

    // LDS offset of this lane's column (m, tap) in every column tile
    int toff[NT];
#pragma unroll
    for (int j = 0; j < NT; j++) {
        const int n = n0 + 16 * j + i16;
        toff[j] = 0;
        if (n < N) {
            const int m = n / KK, t = n - m * KK, jh = t / d.KW, jw = t - jh * d.KW;
            toff[j] = (m - mlo) * PLN + (d.KH - 1 - jh) * WP + (d.KW - 1 - jw);
        }
    }

    // planes mlo..mhi-1 of O[g] into buffer `buf`: interior only (the halo
    // stays zero).  The prefetched path holds kWgStage float4 a thread across
    // the groups of the current g; a float4 is four pixels of one row
    // (W % 4 == 0), and its offsets are recomputed where they are used from an
    // opaque copy of the thread index (hoisted out of the loop they would hold
    // 3 kWgStage registers for its life).
    const int n4 = (MB * HW + 3) / 4;   // float4 of one g's planes
    const bool pref = VEC && W % 4 == 0 && n4 <= 256 * kWgStage;
    auto stage_load = [&](int64_t g, float4 (&sv)[kWgStage]) {
        const T* src = O + wg_ooff(d, g) + (int64_t)mlo * d.o_sm;
        int t0 = tid;
        asm volatile("" : "+v"(t0));
#pragma unroll
        for (int k = 0; k < kWgStage; k++) {
            const int e4 = t0 + 256 * k;
            if (e4 < n4) {
                const int e = 4 * e4, m = e / HW, p = e - m * HW;
                sv[k] = ld4(src + m * d.o_sm + p);
            }
        }
    };
    auto stage_store = [&](int buf, const float4 (&sv)[kWgStage]) {
        int t0 = tid;
        asm volatile("" : "+v"(t0));
#pragma unroll
        for (int k = 0; k < kWgStage; k++) {
            const int e4 = t0 + 256 * k;
            if (e4 < n4) {
                const int e = 4 * e4, m = e / HW, p = e - m * HW, h = p / W, w = p - h * W;
                float* dst = pl + buf * BUF + m * PLN + (h + top) * WP + (w + left);
                dst[0] = sv[k].x;
                dst[1] = sv[k].y;
                dst[2] = sv[k].z;
                dst[3] = sv[k].w;
            }
        }
    };
    auto stage_direct = [&](int64_t g, int buf) {   // without the register prefetch
        const T* src = O + wg_ooff(d, g) + (int64_t)mlo * d.o_sm;
        for (int e = tid; e < MB * HW; e += 256) {
            const int m = e / HW, p = e - m * HW, h = p / W, w = p - h * W;
            pl[buf * BUF + m * PLN + (h + top) * WP + (w + left)] = load(src, m * d.o_sm + p);
        }
    };

    for (int e = tid; e < 2 * BUF; e += 256) pl[e] = 0.f;
    __syncthreads();
    if (g0 < g1) {
        if (pref) {
            float4 sv[kWgStage];
            stage_load(g0, sv);
            stage_store(0, sv);
        } else {
            stage_direct(g0, 0);
        }
    }
    __syncthreads();

    // row loads: items (g, group) in order, each loaded kWgSlots items before
    // it is computed into a fixed register slot (the item loop is unrolled by
    // kWgSlots, so no register moves wait on loads in flight).  The load
    // cursor's batch offset changes once a g (a uniform branch).
    const int NG = (HW + 15) / 16;
    auto zoff = [&](int64_t g) { return g < g1 ? wg_zoff(d, g) : (int64_t)0; };
    int64_t lg = g0;
    int lgrp = 0;
    int64_t loz = zoff(g0);
    // Z through a range-checked buffer (its extent < 2^31 bytes, checked by the
    // lowering): rows past R, pixels past the plane and items past the chunk
    // take an offset past the range and read zero, so no load is guarded
    const __amdgpu_buffer_rsrc_t rZ =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(Z), (short)0, (int)(d.zext * (int64_t)sizeof(T)), 0x00020000);
    auto next_load = [&](float4 (&dst)[RT]) {
        const int q = 16 * lgrp + 4 * kq;
        const bool ok = lg < g1;
#pragma unroll
        for (int mt = 0; mt < RT; mt++) {
            const int64_t e = loz + zr[mt] + q;
            if constexpr (VEC) {
                const int voff = (ok && rok[mt] && q < HW) ? (int)(e * (int64_t)sizeof(T)) : kWgOut;
                dst[mt] = bld4(rZ, voff, (T*)nullptr);
            } else {
                float a[4];
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int voff = (ok && rok[mt] && q + t < HW) ? (int)((e + t) * (int64_t)sizeof(T)) : kWgOut;
                    a[t] = bld1(rZ, voff, (T*)nullptr);
                }
                dst[mt] = make_float4(a[0], a[1], a[2], a[3]);
            }
        }
        if (++lgrp == NG) {
            lgrp = 0;
            ++lg;
            loz = zoff(lg);
        }
    };

    f32x4 acc[RT][NT];
#pragma unroll
    for (int mt = 0; mt < RT; mt++)
#pragma unroll
        for (int j = 0; j < NT; j++) acc[mt][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

    float4 ra[kWgSlots][RT];
#pragma unroll
    for (int sl = 0; sl < kWgSlots; sl++) next_load(ra[sl]);
    // (h, w) of this lane's first pixel of a group, and the step to the next group
    const int h00 = (4 * kq) / W, w00 = 4 * kq - h00 * W, dh = 16 / W, dw = 16 - dh * W;
    int h0 = h00, w0 = w00, grp = 0, cur = 0;
    int64_t g = g0;
    bool more = g0 + 1 < g1;
    float4 sv[kWgStage];
    if (more && pref) stage_load(g0 + 1, sv);
    const int64_t total = (g1 - g0) * NG;
    for (int64_t it = 0; it < total; it += kWgSlots) {
#pragma unroll
        for (int sl = 0; sl < kWgSlots; sl++) {
            if (it + sl < total) {
                const float* pb = pl + cur * BUF;
                const int q = 16 * grp + 4 * kq;
                int bt[4];
                {
                    int h = h0, w = w0;
#pragma unroll
                    for (int t = 0; t < 4; t++) {
                        bt[t] = (q + t < HW) ? h * WP + w : 0;
                        if (++w == W) {
                            w = 0;
                            ++h;
                        }
                    }
                }
                float bv[NT][4];
#pragma unroll
                for (int t = 0; t < 4; t++)
#pragma unroll
                    for (int j = 0; j < NT; j++) bv[j][t] = pb[bt[t] + toff[j]];
#pragma unroll
                for (int t = 0; t < 4; t++)
#pragma unroll
                    for (int mt = 0; mt < RT; mt++) {
                        const float4 v = ra[sl][mt];
                        const float a = t == 0 ? v.x : t == 1 ? v.y : t == 2 ? v.z : v.w;
#pragma unroll
                        for (int j = 0; j < NT; j++)
                            acc[mt][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bv[j][t], acc[mt][j], 0, 0, 0);
                    }
                // the item kWgSlots ahead into this slot
                next_load(ra[sl]);
                w0 += dw;
                h0 += dh;
                if (w0 >= W) {
                    w0 -= W;
                    ++h0;
                }
                if (++grp == NG) {
                    // end of this g: the next g's planes into the other buffer
                    if (more) {
                        if (pref) stage_store(1 - cur, sv);
                        else stage_direct(g + 1, 1 - cur);
                    }
                    __syncthreads();
                    cur ^= 1;
                    ++g;
                    grp = 0;
                    h0 = h00;
                    w0 = w00;
                    more = g + 1 < g1;
                    if (more && pref) stage_load(g + 1, sv);
                }
            }
        }
    }

    // accumulator r of a lane: row 4 kq + r of the tile, column i16
#pragma unroll
    for (int mt = 0; mt < RT; mt++)
#pragma unroll
        for (int j = 0; j < NT; j++)
#pragma unroll
            for (int r = 0; r < 4; r++) {
                const int64_t u = ub * 64 * RT + wave * 16 * RT + 16 * mt + 4 * kq + r;
                const int n = n0 + 16 * j + i16;
                if (u < d.R && n < N) P[(ck * d.R + u) * N + n] = acc[mt][j][r];
            }
}

template <typename T, int RT, int NT>
hipError_t wgconv_go(const CredDesc& d, bool vec, const void* z, const void* o, float* part, hipStream_t s) {
    auto k = vec ? wgconv<T, RT, NT, true> : wgconv<T, RT, NT, false>;
    static std::atomic<uint64_t> ok{0};
    // dynamic LDS above 64 KB has to be allowed per kernel, once per device
    if (d.lds_bytes > 64 * 1024) {
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return e;
        if (dev < 0 || dev >= 64 || d.lds_bytes > 160 * 1024) return hipErrorInvalidValue;
        if (!(ok.load() & (1ull << dev))) {
            e = hipFuncSetAttribute((const void*)wgconv<T, RT, NT, true>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e == hipSuccess)
                e = hipFuncSetAttribute((const void*)wgconv<T, RT, NT, false>,
                                        hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
            if (e != hipSuccess) return e;
            ok.fetch_or(1ull << dev);
        }
    }
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d, (const T*)z, (const T*)o, part);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_wgconv(const Launch& ln, const void* z, const void* o, void* part, hipStream_t s) {
    CredDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int bf = (ln.kind >> kBitIn) & 1;
    const int KK = d.KH * d.KW, N = d.M * KK;
    // the shapes the kernel assumes (the lowering guarantees them)
    const bool nct_ok = bf ? (d.nct == 6 || (d.nct == 3 && N <= 48)) : (d.nct >= 1 && d.nct <= 6);
    if (d.M < 1 || KK < 1 || !nct_ok || (d.rt != 1 && d.rt != 2) || (!bf && d.rt != 2) ||
        d.ncb != (N + 16 * d.nct - 1) / (16 * d.nct) || d.mb < 1 || d.mb > d.M || d.H < 1 || d.W < 1 ||
        d.PH != d.H + d.KH - 1 || d.PWp < d.W + d.KW - 1 || d.ch < 0 || d.ch >= d.KH || d.cw < 0 ||
        d.cw >= d.KW || d.nrb != (d.R + 64 * d.rt - 1) / (64 * d.rt) || d.gchunk < 1 ||
        d.nchunks != (d.G + d.gchunk - 1) / d.gchunk || d.blocks != (int64_t)d.nrb * d.ncb * d.nchunks ||
        d.lds_bytes != (uint32_t)(2 * d.mb * d.PH * d.PWp * 4) || d.lds_bytes > 160 * 1024 ||
        (int64_t)d.H * d.W * d.M >= (1ll << 30) || ln.grid[0] != (uint32_t)d.blocks || ln.block[0] != 256 ||
        d.zext < 1 || d.zext * (bf ? 2 : 4) >= (1ll << 31))
        return hipErrorInvalidValue;
    // every column block's planes fit the mb staged
    for (int cb = 0; cb < d.ncb; cb++) {
        const int n0 = cb * 16 * d.nct, mlo = n0 / KK, mhi = std::min(d.M, (n0 + 16 * d.nct - 1) / KK + 1);
        if (mhi - mlo > d.mb) return hipErrorInvalidValue;
    }
    // wide loads: rows of Z and of O start at multiples of four elements
    const int64_t HW = (int64_t)d.H * d.W;
    const uintptr_t al = bf ? 8 : 16;
    bool vec = HW % 4 == 0 && d.z_sr % 4 == 0 && (d.M == 1 || d.o_sm % 4 == 0) && (uintptr_t)z % al == 0 &&
               (uintptr_t)o % al == 0;
    for (int i = 0; i < d.ng; i++) vec = vec && d.g_sZ[i] % 4 == 0 && d.g_sY[i] % 4 == 0;
    float* Pp = (float*)part;
    if (bf) {
        if (d.rt == 1) return d.nct == 6 ? wgconv_go<bf16_t, 1, 6>(d, vec, z, o, Pp, s)
                                         : wgconv_go<bf16_t, 1, 3>(d, vec, z, o, Pp, s);
        return d.nct == 6 ? wgconv_go<bf16_t, 2, 6>(d, vec, z, o, Pp, s) : wgconv_go<bf16_t, 2, 3>(d, vec, z, o, Pp, s);
    }
    switch (d.nct) {
        case 1: return wgconv_go<float, 2, 1>(d, vec, z, o, Pp, s);
        case 2: return wgconv_go<float, 2, 2>(d, vec, z, o, Pp, s);
        case 3: return wgconv_go<float, 2, 3>(d, vec, z, o, Pp, s);
        case 4: return wgconv_go<float, 2, 4>(d, vec, z, o, Pp, s);
        case 5: return wgconv_go<float, 2, 5>(d, vec, z, o, Pp, s);
        default: return wgconv_go<float, 2, 6>(d, vec, z, o, Pp, s);
    }
}

}  // namespace ce
