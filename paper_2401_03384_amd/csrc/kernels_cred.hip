// Convolution of a stack of planes contracted over one shared index
// (CredDesc): the last step of reshaped-CP layers (Section 2.3: the spatial
// factor convolved with every rank slice and contracted over the rank) and
// its filter gradient.  The result has a single channel (forward) or a few
// taps per rank (gradient), so no matrix-core tile shape fits; both are
// plain FMA work on planes staged in LDS with their zero halo.
//
//   cred   forward: a thread owns four consecutive pixels of one output row
//          of one batch index, for every channel m, and runs over the ranks; each rank's planes
//          are staged (double-buffered) by the threads that own the pixels,
//          and every staged row segment serves all KW taps of a filter row.
//   credw  filter gradient: a thread owns four pixels of one rank's plane
//          and runs over a chunk of batch indices, accumulating all KH x KW
//          taps of every channel m; the block then sums its threads' taps in
//          a fixed order into one partial per (chunk, rank, m, tap), which
//          credw_reduce sums over the chunks in order.
#include <atomic>
#include <cstdint>
#include <cstring>

#include "desc.h"
#include "hip_util.h"
#include "kernels.h"

namespace ce {
namespace {

constexpr int kPx = 4;         // pixels per thread (along a row)
constexpr int kMaxTapsW = 25;  // taps a gradient thread keeps in registers
constexpr int kMaxAccW = 72;   // channels (at most 8) x taps a gradient thread keeps in registers

// four consecutive elements z[0..3] of a row, zero past column `left`
template <typename T, bool VEC>
__device__ __forceinline__ void load4(const T* z, int left, float v[kPx]) {
    if constexpr (VEC) {
        if constexpr (sizeof(T) == 2) {
            const uint2 u = *reinterpret_cast<const uint2*>(z);
            v[0] = __uint_as_float(u.x << 16);
            v[1] = __uint_as_float(u.x & 0xffff0000u);
            v[2] = __uint_as_float(u.y << 16);
            v[3] = __uint_as_float(u.y & 0xffff0000u);
        } else {
            const float4 u = *reinterpret_cast<const float4*>(z);
            v[0] = u.x;
            v[1] = u.y;
            v[2] = u.z;
            v[3] = u.w;
        }
    } else {
#pragma unroll
        for (int p = 0; p < kPx; p++) v[p] = p < left ? load(z, p) : 0.f;
    }
}

__device__ __forceinline__ void batch_offsets(const CredDesc& d, int64_t g, int64_t& oz, int64_t& oy) {
    oz = oy = 0;
    for (int i = d.ng - 1; i >= 0; --i) {
        const int64_t x = g % d.g_size[i];
        g /= d.g_size[i];
        oz += x * d.g_sZ[i];
        oy += x * d.g_sY[i];
    }
}

// the row segment (kPx + KW - 1 values, rounded up to float4s) that a
// thread's pixels meet in one filter row
template <int KW>
struct Seg {
    static constexpr int n4 = (kPx + KW - 1 + 3) / 4;
    float v[4 * n4];
    __device__ __forceinline__ void read(const float* src) {
#pragma unroll
        for (int q = 0; q < n4; q++) {
            const float4 t = reinterpret_cast<const float4*>(src)[q];
            v[4 * q] = t.x;
            v[4 * q + 1] = t.y;
            v[4 * q + 2] = t.z;
            v[4 * q + 3] = t.w;
        }
    }
};

// channels m of O a thread serves: MO covers the M of the descriptor; the
// ones past M read channel M - 1 and are never stored
__device__ __forceinline__ int mclamp(int mo, int M) { return mo < M ? mo : M - 1; }

template <typename T, int KH, int KW, int MO, bool VEC>
__global__ void __launch_bounds__(1024) cred(CredDesc d, const T* __restrict__ Z, const T* __restrict__ F,
                                             T* __restrict__ Y) {
    extern __shared__ float4 lds4[];
    float* pl = reinterpret_cast<float*>(lds4);
    const int W = d.W, PWp = d.PWp, plane = d.PH * PWp;
    const int tid = threadIdx.x, nt = blockDim.x;
    const int gl = tid / d.items, it = tid - gl * d.items;
    const int oh = it / d.wchunks, ow0 = (it - oh * d.wchunks) * kPx;
    const int64_t g = (int64_t)blockIdx.x * d.per + gl;
    const bool active = gl < d.per && g < d.G;
    const int left = W - ow0;
    for (int e = tid; e < 2 * d.per * plane; e += nt) pl[e] = 0.f;
    int64_t oz = 0, oy = 0;
    if (active) batch_offsets(d, g, oz, oy);
    const T* zp = Z + oz + (int64_t)oh * W + ow0;
    float* wr = pl + (size_t)gl * plane + (oh + d.ch) * PWp + ow0 + d.cw;   // this thread's pixels
    const float* rd = pl + (size_t)gl * plane + oh * PWp + ow0;            // its window origin
    const int bufstride = d.per * plane;
    float v[kPx];
    if (active) load4<T, VEC>(zp, left, v);
    __syncthreads();   // zeroed
    if (active)
#pragma unroll
        for (int p = 0; p < kPx; p++)
            if (p < left) wr[p] = v[p];
    float acc[MO][kPx];
#pragma unroll
    for (int mo = 0; mo < MO; mo++)
#pragma unroll
        for (int p = 0; p < kPx; p++) acc[mo][p] = 0.f;
    for (int64_t r = 0; r < d.R; r++) {
        const int cur = (int)(r & 1);
        const bool more = r + 1 < d.R;
        if (active && more) load4<T, VEC>(zp + (r + 1) * d.z_sr, left, v);
        __syncthreads();   // plane r staged by all; plane r - 1 no longer read
        if (active) {
            const float* src = rd + cur * bufstride;
            const T* f = F + r * d.f_sr;
#pragma unroll
            for (int jh = 0; jh < KH; jh++) {
                Seg<KW> s;
                s.read(src + jh * PWp);
#pragma unroll
                for (int jw = 0; jw < KW; jw++)
#pragma unroll
                    for (int mo = 0; mo < MO; mo++) {
                        const float fv = load(f, mclamp(mo, d.M) * d.o_sm + jh * d.f_sh + jw * d.f_sw);
#pragma unroll
                        for (int p = 0; p < kPx; p++) acc[mo][p] += s.v[p + jw] * fv;
                    }
            }
            if (more)
#pragma unroll
                for (int p = 0; p < kPx; p++)
                    if (p < left) wr[(1 - cur) * bufstride + p] = v[p];
        }
    }
    if (!active) return;
    T* y = Y + oy + (int64_t)oh * W + ow0;
#pragma unroll
    for (int mo = 0; mo < MO; mo++) {
        if (mo >= d.M) break;
#pragma unroll
        for (int p = 0; p < kPx; p++)
            if (p < left) store(y, mo * d.y_sm + p, acc[mo][p]);
    }
}

template <typename T, int KH, int KW, int MO, bool VEC>
__global__ void __launch_bounds__(MO >= 4 ? 512 : 1024) credw(CredDesc d, const T* __restrict__ Z,
                                                              const T* __restrict__ D, float* __restrict__ P) {
    constexpr int KK = KH * KW;
    extern __shared__ float4 lds4[];
    float* pl = reinterpret_cast<float*>(lds4);
    const int W = d.W, PWp = d.PWp, plane = d.PH * PWp;
    const int tid = threadIdx.x, nt = blockDim.x;
    const int64_t rgi = blockIdx.x % d.nrb, gci = blockIdx.x / d.nrb;
    const int rl = tid / d.items, it = tid - rl * d.items;
    const int oh = it / d.wchunks, ow0 = (it - oh * d.wchunks) * kPx;
    const int64_t r = rgi * d.per + rl;
    const bool active = rl < d.per && r < d.R;
    const int left = W - ow0;
    const int64_t g0 = gci * d.gchunk, g1 = min(d.G, g0 + d.gchunk);
    for (int e = tid; e < 2 * d.per * plane; e += nt) pl[e] = 0.f;
    const int64_t pix = (int64_t)oh * W + ow0;
    float* wr = pl + (size_t)rl * plane + (oh + d.ch) * PWp + ow0 + d.cw;
    const float* rd = pl + (size_t)rl * plane + oh * PWp + ow0;
    const int bufstride = d.per * plane;
    float v[kPx], dy[MO][kPx], ndy[MO][kPx];
    auto fetch = [&](int64_t g, float* zv, float (*yv)[kPx]) {
        int64_t oz, oy;
        batch_offsets(d, g, oz, oy);
        load4<T, VEC>(Z + oz + r * d.z_sr + pix, left, zv);
#pragma unroll
        for (int mo = 0; mo < MO; mo++) load4<T, VEC>(D + oy + mclamp(mo, d.M) * d.o_sm + pix, left, yv[mo]);
    };
    if (active) fetch(g0, v, dy);
    __syncthreads();   // zeroed
    if (active)
#pragma unroll
        for (int p = 0; p < kPx; p++)
            if (p < left) wr[p] = v[p];
    float acc[MO][KK];
#pragma unroll
    for (int mo = 0; mo < MO; mo++)
#pragma unroll
        for (int k = 0; k < KK; k++) acc[mo][k] = 0.f;
    for (int64_t g = g0; g < g1; g++) {
        const int cur = (int)((g - g0) & 1);
        const bool more = g + 1 < g1;
        if (active && more) fetch(g + 1, v, ndy);
        __syncthreads();
        if (active) {
            const float* src = rd + cur * bufstride;
#pragma unroll
            for (int jh = 0; jh < KH; jh++) {
                Seg<KW> s;
                s.read(src + jh * PWp);
#pragma unroll
                for (int jw = 0; jw < KW; jw++)
#pragma unroll
                    for (int mo = 0; mo < MO; mo++)
#pragma unroll
                        for (int p = 0; p < kPx; p++) acc[mo][jh * KW + jw] += s.v[p + jw] * dy[mo][p];
            }
            if (more) {
#pragma unroll
                for (int p = 0; p < kPx; p++)
                    if (p < left) wr[(1 - cur) * bufstride + p] = v[p];
#pragma unroll
                for (int mo = 0; mo < MO; mo++)
#pragma unroll
                    for (int p = 0; p < kPx; p++) dy[mo][p] = ndy[mo][p];
            }
        }
    }
    // sum the threads of each rank in a fixed order, one channel m at a time
    float* red = pl;
#pragma unroll
    for (int mo = 0; mo < MO; mo++) {
        if (mo >= d.M) break;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < KK; k++) red[(size_t)tid * KK + k] = active ? acc[mo][k] : 0.f;
        __syncthreads();
        for (int q = tid; q < d.per * KK; q += nt) {
            const int ql = q / KK, k = q - ql * KK;
            const int64_t rq = rgi * d.per + ql;
            if (rq >= d.R) continue;
            float sum = 0.f;
            for (int i = 0; i < d.items; i++) sum += red[(size_t)(ql * d.items + i) * KK + k];
            P[((gci * d.R + rq) * d.M + mo) * KK + k] = sum;
        }
    }
}

// C[m][u][tap] (output strides c_*) = sum over the chunks of the partials:
// a block takes 64 consecutive outputs (one per lane); its four wavefronts sum
// contiguous quarters of the chunks with eight loads in flight, in double,
// and the quarters are added in a fixed order.
template <typename TC>
__global__ void __launch_bounds__(256) credw_reduce(CredDesc d, const float* __restrict__ P, TC* __restrict__ C) {
    __shared__ double q4[4][64];
    const int KK = d.KH * d.KW;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t per_chunk = d.R * d.M * KK;
    const int64_t t = (int64_t)blockIdx.x * 64 + lane;
    const int64_t quarter = (d.nchunks + 3) / 4;
    const int64_t c0 = wave * quarter, c1 = min(d.nchunks, c0 + quarter);
    double acc = 0.0;
    if (t < per_chunk) {
        int64_t c = c0;
        for (; c + 8 <= c1; c += 8) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; u++) v[u] = P[(c + u) * per_chunk + t];
#pragma unroll
            for (int u = 0; u < 8; u++) acc += v[u];
        }
        for (; c < c1; c++) acc += P[c * per_chunk + t];
    }
    q4[wave][lane] = acc;
    __syncthreads();
    if (wave != 0 || t >= per_chunk) return;
    const double sum = (q4[0][lane] + q4[1][lane]) + (q4[2][lane] + q4[3][lane]);
    const int64_t r = t / (d.M * KK), q = t - r * d.M * KK;
    const int m = (int)(q / KK), k = (int)(q - (int64_t)m * KK), jh = k / d.KW, jw = k - jh * d.KW;
    store(C, m * d.c_sm + r * d.c_sr + jh * d.c_sh + jw * d.c_sw, (float)sum);
}

// dynamic LDS above 64 KB has to be allowed per kernel, once per device
hipError_t allow_lds(const void* k, std::atomic<uint64_t>& allowed, uint32_t bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || bytes > 160 * 1024) return hipErrorInvalidValue;
    if (!(allowed.load() & (1ull << dev))) {
        e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
        if (e != hipSuccess) return e;
        allowed.fetch_or(1ull << dev);
    }
    return hipSuccess;
}

template <typename T, bool VEC>
hipError_t cred_t(const CredDesc& d, bool wgrad, const void* z, const void* o, void* y, hipStream_t s) {
    dim3 g((uint32_t)d.blocks), bl(d.threads);
    const int MO = d.M == 1 ? 1 : d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16;
#define CRED_MO(kh, kw, mo) \
    if (MO == mo) { \
        if (wgrad) { \
            if constexpr (kh * kw > kMaxTapsW || mo * kh * kw > kMaxAccW || mo > 8) return hipErrorInvalidValue; \
            else { \
                static std::atomic<uint64_t> ok{0}; \
                auto k = credw<T, kh, kw, mo, VEC>; \
                hipError_t e = allow_lds((const void*)k, ok, d.lds_bytes); \
                if (e != hipSuccess) return e; \
                hipLaunchKernelGGL(k, g, bl, d.lds_bytes, s, d, (const T*)z, (const T*)o, (float*)y); \
            } \
        } else { \
            static std::atomic<uint64_t> ok{0}; \
            auto k = cred<T, kh, kw, mo, VEC>; \
            hipError_t e = allow_lds((const void*)k, ok, d.lds_bytes); \
            if (e != hipSuccess) return e; \
            hipLaunchKernelGGL(k, g, bl, d.lds_bytes, s, d, (const T*)z, (const T*)o, (T*)y); \
        } \
        return hipGetLastError(); }
#define CRED(kh, kw) \
    if (d.KH == kh && d.KW == kw) { \
        CRED_MO(kh, kw, 1) CRED_MO(kh, kw, 4) CRED_MO(kh, kw, 8) CRED_MO(kh, kw, 16) \
        return hipErrorInvalidValue; }
    CRED(3, 3) CRED(5, 5) CRED(7, 7) CRED(1, 3) CRED(3, 1)
#undef CRED
#undef CRED_MO
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_cred(const Launch& ln, const void* z, const void* o, void* y, hipStream_t s) {
    CredDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    const int kind = ln.kind & 0xff;
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    if (d.M < 1) return hipErrorInvalidValue;
    if (kind == K_CREDW_REDUCE) {
        // here o = the partials, y = the output
        dim3 g((uint32_t)((d.R * d.M * d.KH * d.KW + 63) / 64)), bl(256);
        if (tC) hipLaunchKernelGGL(credw_reduce<bf16_t>, g, bl, 0, s, d, (const float*)o, (bf16_t*)y);
        else hipLaunchKernelGGL(credw_reduce<float>, g, bl, 0, s, d, (const float*)o, (float*)y);
        return hipGetLastError();
    }
    if (d.M > 16) return hipErrorInvalidValue;   // the partial-sum kernels: M <= 16
    const bool wgrad = kind == K_CREDW;
    if (!wgrad && tIn != tC) return hipErrorInvalidValue;   // forward keeps the input type
    // four-wide loads: every row start of Z (and of the plane operand of the
    // gradient) a multiple of four elements, and the buffers aligned to them
    const uintptr_t al = tIn ? 8 : 16;
    bool vec = d.W % 4 == 0 && d.z_sr % 4 == 0 && (uintptr_t)z % al == 0;
    for (int i = 0; i < d.ng; i++) vec = vec && d.g_sZ[i] % 4 == 0 && (!wgrad || d.g_sY[i] % 4 == 0);
    if (wgrad) vec = vec && (uintptr_t)o % al == 0 && (d.M == 1 || d.o_sm % 4 == 0);
    if (tIn) return vec ? cred_t<bf16_t, true>(d, wgrad, z, o, y, s) : cred_t<bf16_t, false>(d, wgrad, z, o, y, s);
    return vec ? cred_t<float, true>(d, wgrad, z, o, y, s) : cred_t<float, false>(d, wgrad, z, o, y, s);
}

}  // namespace ce
