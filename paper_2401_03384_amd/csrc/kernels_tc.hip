// General contraction on MFMA tiles (see TcDesc): the pairwise steps that no
// specialised kernel matches -- convolutions that also contract channels
// (Section 3.1: contraction and convolution in one step), their feature- and
// filter-side gradients, and channel products whose labels interleave in
// memory.
//
// A block computes a 32*MT x 128 tile of C for one batch index g, walking
// the reduction in slices of 32 (fp32) or 64 (bf16).  Each thread owns one
// row of the A tile and one column of the B tile for the whole block (their
// offsets and convolution bases stay in registers); the k offsets of a slice
// come from a small LDS table built one slice ahead.  Slices are double
// buffered: the next slice's elements are loaded into registers (coalesced
// along n when n is unit-stride in B) while the MFMAs run on the current one
// (fp32: 32x32x2, bf16: 32x32x16), then written to the other LDS buffer, one
// barrier a slice.  Positions of convolved labels outside [0, lim) read zero;
// with 31-bit offsets the loads are range-checked buffer loads (an
// out-of-range offset reads zero), else predicated 64-bit loads.
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

constexpr uint32_t kOff = 0x80000000u;   // a byte offset past every buffer range: reads 0

// One element of an operand: a range-checked buffer load (off32) or a
// predicated load.
template <typename T, typename IT>
__device__ __forceinline__ T gload(const T* base, __amdgpu_buffer_rsrc_t r, IT off, bool ok) {
    if constexpr (sizeof(IT) == 4) {
        const uint32_t b = ok ? (uint32_t)off * (uint32_t)sizeof(T) : kOff;
        if constexpr (sizeof(T) == 2) return (T)__builtin_amdgcn_raw_buffer_load_b16(r, (int)b, 0, 0);
        else return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)b, 0, 0));
    } else {
        return ok ? base[off] : (T)0;
    }
}

template <typename T, typename TC, int MT, typename IT, int TK, int NB, bool KM>
__global__ void __launch_bounds__(256) tc_gemm(TcDesc d, const T* __restrict__ A, const T* __restrict__ B,
                                               TC* __restrict__ C, float* __restrict__ P) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int TM = 32 * MT, TN = 128;
    static_assert(TK == 32 || (BF && TK == 64), "reduction slice");
    constexpr int LA = BF ? TK + 8 : TK + 1;       // A tile: [m][k]
    constexpr int LB = BF ? TK + 8 : (KM ? TN + 1 : TN + 4);   // B tile: [n][k] (bf16), [k][n] (fp32)
    constexpr int ASZ = TM * LA, BSZ = BF ? TN * LB : TK * LB;
    constexpr int EA = TM * TK / 256, EB = TN * TK / 256;   // tile elements a thread loads
    constexpr int LC = TN + 4;                               // output tile pitch (fp32)
    // NB = 1: every block's reduction is one slice (no second buffer)
    constexpr int TILES = NB * (ASZ + BSZ) * (int)sizeof(T), CT = 32 * LC * 4;
    // the operand slices, and after the reduction the output tile, in one area
    __shared__ __attribute__((aligned(16))) unsigned char sm[TILES > CT ? TILES : CT];
    T (*As)[ASZ] = reinterpret_cast<T (*)[ASZ]>(sm);
    T (*Bs)[BSZ] = reinterpret_cast<T (*)[BSZ]>(sm + NB * ASZ * sizeof(T));
    __shared__ IT kA[2][TK], kB[2][TK];
    __shared__ int32_t kj[2][2][TK];
    __shared__ unsigned char kok[2][TK];
    __shared__ IT mC[TM], nC[TN];
    __shared__ unsigned char mok[TM], nok[TN];
    // k-major loads: the rows' / columns' offsets (and convolution bases) by table
    __shared__ IT mAt[KM ? TM : 1], nBt[KM ? TN : 1];
    __shared__ IT npa[KM ? 2 : 1][KM ? TN : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), cl = lane & 31, hf = lane >> 5;
    int64_t bid = blockIdx.x;
    const int nt = (int)(bid % d.ntiles);
    bid /= d.ntiles;
    const int mt = (int)(bid % d.mtiles);
    bid /= d.mtiles;
    const int ks = (int)(bid % d.ksplit);
    const int64_t g = bid / d.ksplit;
    const int64_t m0 = (int64_t)mt * TM, n0 = (int64_t)nt * TN;

    IT gA = 0, gB = 0, gC = 0;
    {
        int64_t x = g;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t c = x % d.g_size[i];
            x /= d.g_size[i];
            gA += (IT)(c * d.g_sA[i]);
            gB += (IT)(c * d.g_sB[i]);
            gC += (IT)(c * d.g_sC[i]);
        }
    }
    const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(A), (short)0,
                                                                         (int)(sizeof(IT) == 4 ? d.extA : 0), 0x00020000);
    const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(B), (short)0,
                                                                         (int)(sizeof(IT) == 4 ? d.extB : 0), 0x00020000);

    // this thread's A row (fixed for the block) and its k positions in a slice
    const int am = tid % TM;
    IT aoff;
    bool aok;
    {
        const int64_t m = m0 + am;
        int64_t x = m;
        IT oa = 0, oc = 0;
        for (int i = d.nm - 1; i >= 0; --i) {
            const int64_t c = x % d.m_size[i];
            x /= d.m_size[i];
            oa += (IT)(c * d.m_sA[i]);
            oc += (IT)(c * d.m_sC[i]);
        }
        aoff = gA + oa;
        aok = m < d.M;
        if (tid < TM) {
            mC[tid] = oc;
            mok[tid] = aok;
            if constexpr (KM) mAt[tid] = aoff;
        }
    }
    auto akk = [&](int j) { return BF ? (tid / TM) * EA + j : tid / TM + (256 / TM) * j; };
    // this thread's B column (fixed) and its k positions
    const int bn = tid % TN, bkr = tid / TN;
    IT boff, bpa[2] = {0, 0};
    bool bok;
    uint32_t tmask = 0;
    {
        const int64_t n = n0 + bn;
        int64_t x = n;
        IT ob = 0, oc = 0;
        int32_t np[2] = {0, 0};
        for (int i = d.nn - 1; i >= 0; --i) {
            const int64_t c = x % d.n_size[i];
            x /= d.n_size[i];
            ob += (IT)(c * d.n_sB[i]);
            oc += (IT)(c * d.n_sC[i]);
            if (d.n_cv[i] >= 0) np[d.n_cv[i]] = (int32_t)c;
        }
        boff = gB + ob;
        bok = n < d.N;
        for (int c = 0; c < d.ncv; c++) bpa[c] = (IT)((int64_t)d.cv_a[c] * np[c] + d.cv_g[c]);
        if (d.tapmask) {
            // valid taps of this output position; their offsets come from the k table
            for (int c = 0; c < d.ncv; c++) boff += bpa[c] * (IT)d.cv_s[c];
            const int J1 = d.tapJ1;
            int Jc[2] = {1, 1};
            for (int i = 0; i < d.nk; i++)
                if (d.k_cv[i] >= 0) Jc[d.k_cv[i]] = (int)d.k_size[i];
            uint32_t mask = 0;
            for (int j0 = 0; j0 < Jc[0]; j0++) {
                const IT p0 = bpa[0] + (IT)d.cv_b[0] * j0;
                if (p0 < 0 || p0 >= (IT)d.cv_lim[0]) continue;
                for (int j1 = 0; j1 < J1; j1++) {
                    if (d.ncv > 1) {
                        const IT p1 = bpa[1] + (IT)d.cv_b[1] * j1;
                        if (p1 < 0 || p1 >= (IT)d.cv_lim[1]) continue;
                    }
                    mask |= 1u << (j0 * J1 + j1);
                }
            }
            tmask = mask;
        }
        if (tid < TN) {
            nC[tid] = oc;
            nok[tid] = bok;
            if constexpr (KM) {
                nBt[tid] = boff;
                npa[0][tid] = bpa[0];
                if (d.ncv > 1) npa[1][tid] = bpa[1];
            }
        }
    }
    auto bkk = [&](int j) { return BF ? bkr * EB + j : bkr + 2 * j; };

    const int64_t kb = (int64_t)ks * d.kchunk;
    const int64_t ke = min(d.K, kb + d.kchunk);
    const int ns = (int)((ke - kb + TK - 1) / TK);

    // k table of the slice at k0 into buffer t
    auto ktab = [&](int t, int64_t k0) {
        if (tid < TK) {
            const int64_t k = k0 + tid;
            int64_t x = k;
            IT oa = 0, ob = 0;
            kj[t][0][tid] = kj[t][1][tid] = 0;
            for (int i = d.nk - 1; i >= 0; --i) {
                const int64_t c = x % d.k_size[i];
                x /= d.k_size[i];
                oa += (IT)(c * d.k_sA[i]);
                ob += (IT)(c * d.k_sB[i]);
                if (d.k_cv[i] >= 0) kj[t][d.k_cv[i]][tid] = (int32_t)c;
            }
            if (d.tapmask) {
                // the taps' offsets, and the tap index in kj[t][0]
                for (int c = 0; c < d.ncv; c++) ob += (IT)d.cv_b[c] * (IT)kj[t][c][tid] * (IT)d.cv_s[c];
                kj[t][0][tid] = kj[t][0][tid] * d.tapJ1 + (d.ncv > 1 ? kj[t][1][tid] : 0);
            }
            kA[t][tid] = oa;
            kB[t][tid] = ob;
            kok[t][tid] = k < ke;
        }
    };
    T ra[EA], rb[EB];
    // loads of slice k0 (table t); k positions past the chunk end are skipped
    // (a branch uniform over the wavefront where the thread's k positions are)
    auto load = [&](int t, int64_t k0) {
        const int kv = (int)min((int64_t)TK, ke - k0);   // valid k positions of the slice
        if constexpr (KM) {
            // lanes walk k (unit-stride in A and B): this thread's k position
            const int kk = tid % TK;
            const bool kin = kk < kv;
            const IT ka = kA[t][kk], kbo = kB[t][kk];
            int32_t kjv[2] = {kj[t][0][kk], kj[t][1][kk]};
#pragma unroll
            for (int j = 0; j < EA; j++) {
                const int mm = tid / TK + (256 / TK) * j;
                ra[j] = gload<T, IT>(A, rA, mAt[mm] + ka, kin && mok[mm]);
            }
#pragma unroll
            for (int j = 0; j < EB; j++) {
                const int nn = tid / TK + (256 / TK) * j;
                bool ok = kin && nok[nn];
                IT off = nBt[nn] + kbo;
                for (int c = 0; c < d.ncv; c++) {
                    const IT pos = npa[c][nn] + (IT)d.cv_b[c] * (IT)kjv[c];
                    ok = ok && pos >= 0 && pos < (IT)d.cv_lim[c];
                    off += pos * (IT)d.cv_s[c];
                }
                rb[j] = gload<T, IT>(B, rB, off, ok);
            }
            return;
        }
        // k positions past the slice's valid ones load nothing through the
        // ok flag rather than a branch (every table entry below TK is
        // written): a branch around each load made the wave wait for its
        // table read before the next one
#pragma unroll
        for (int j = 0; j < EA; j++) {
            const int kk = akk(j);
            ra[j] = gload<T, IT>(A, rA, aoff + kA[t][kk], aok && kk < kv);
        }
        if (d.tapmask) {
#pragma unroll
            for (int j = 0; j < EB; j++) {
                const int kk = bkk(j);
                const bool ok = bok && kk < kv && ((tmask >> kj[t][0][kk]) & 1u);
                rb[j] = gload<T, IT>(B, rB, boff + kB[t][kk], ok);
            }
        } else {
#pragma unroll
            for (int j = 0; j < EB; j++) {
                const int kk = bkk(j);
                bool ok = bok && kk < kv;
                IT off = boff + kB[t][kk];
                for (int c = 0; c < d.ncv; c++) {
                    const IT pos = bpa[c] + (IT)d.cv_b[c] * (IT)kj[t][c][kk];
                    ok = ok && pos >= 0 && pos < (IT)d.cv_lim[c];
                    off += pos * (IT)d.cv_s[c];
                }
                rb[j] = gload<T, IT>(B, rB, off, ok);
            }
        }
    };
    auto put = [&](int t) {
        if constexpr (KM) {
            const int kk = tid % TK;
#pragma unroll
            for (int j = 0; j < EA; j++) As[t][(tid / TK + (256 / TK) * j) * LA + kk] = ra[j];
#pragma unroll
            for (int j = 0; j < EB; j++) {
                const int nn = tid / TK + (256 / TK) * j;
                if constexpr (BF) Bs[t][nn * LB + kk] = rb[j];
                else Bs[t][kk * LB + nn] = rb[j];
            }
            return;
        }
        if constexpr (BF) {
            // contiguous k runs: 16-byte LDS stores
            T* pa = &As[t][am * LA + (tid / TM) * EA];
#pragma unroll
            for (int j = 0; j < EA; j += 8) __builtin_memcpy(pa + j, ra + j, 16);
            T* pb = &Bs[t][bn * LB + bkr * EB];
#pragma unroll
            for (int j = 0; j < EB; j += 8) __builtin_memcpy(pb + j, rb + j, 16);
        } else {
#pragma unroll
            for (int j = 0; j < EA; j++) As[t][am * LA + akk(j)] = ra[j];
#pragma unroll
            for (int j = 0; j < EB; j++) Bs[t][bkk(j) * LB + bn] = rb[j];
        }
    };

    f32x16 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[i][r] = 0.f;

    ktab(0, kb);
    __syncthreads();
    load(0, kb);
    put(0);
    if (NB == 2 && ns > 1) ktab(1, kb + TK);
    __syncthreads();
    for (int s = 0; s < (NB == 2 ? ns : 1); s++) {
        const int cur = NB == 2 ? s & 1 : 0;
        if (NB == 2 && s + 1 < ns) load(cur ^ 1, kb + (int64_t)(s + 1) * TK);   // next slice in flight during this one's MFMAs
        const T* as = As[cur];
        const T* bs = Bs[cur];
        if constexpr (BF) {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 16) {
                const bf16x8 b = ld8(&bs[(wave * 32 + cl) * LB + kk + 8 * hf]);
#pragma unroll
                for (int i = 0; i < MT; i++)
                    acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld8(&as[(i * 32 + cl) * LA + kk + 8 * hf]), b,
                                                                     acc[i], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int kk = 0; kk < TK; kk += 2) {
                const float b = bs[(kk + hf) * LB + wave * 32 + cl];
#pragma unroll
                for (int i = 0; i < MT; i++)
                    acc[i] = __builtin_amdgcn_mfma_f32_32x32x2f32(as[(i * 32 + cl) * LA + kk + hf], b, acc[i], 0, 0, 0);
            }
        }
        if (NB == 2 && s + 1 < ns) put(cur ^ 1);
        if (NB == 2 && s + 2 < ns) ktab(cur, kb + (int64_t)(s + 2) * TK);
        __syncthreads();
    }
    // results (pad so every path has the wait states before the first read),
    // through the output tile in LDS (the loop's last barrier freed it): each
    // thread then writes runs of 8 consecutive n, 16 bytes at a time where C
    // (or the partial) is contiguous there and the address 16-byte aligned
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    float* Ct = reinterpret_cast<float*>(sm);
#pragma unroll
    for (int i = 0; i < MT; i++) {   // 32 rows of the tile a pass
        if (i > 0) __syncthreads();   // the previous pass's rows are written out
#pragma unroll
        for (int r = 0; r < 16; r++) Ct[row32(r, lane) * LC + wave * 32 + cl] = acc[i][r];
        __syncthreads();
        for (int q = tid; q < 32 * (TN / 8); q += 256) {
            const int mr = q / (TN / 8), nn = (q - mr * (TN / 8)) * 8, mm = i * 32 + mr;
            if (!mok[mm] || !nok[nn]) continue;
            float v[8];
            const float4 v0 = *reinterpret_cast<const float4*>(&Ct[mr * LC + nn]);
            const float4 v1 = *reinterpret_cast<const float4*>(&Ct[mr * LC + nn + 4]);
            v[0] = v0.x; v[1] = v0.y; v[2] = v0.z; v[3] = v0.w;
            v[4] = v1.x; v[5] = v1.y; v[6] = v1.z; v[7] = v1.w;
            if (d.ksplit > 1) {
                const int64_t base = ((g * d.ksplit + ks) * d.M + (m0 + mm)) * d.N + n0 + nn;
                if (nok[nn + 7] && ((uintptr_t)(P + base) & 15) == 0) {
                    *reinterpret_cast<float4*>(P + base) = v0;
                    *reinterpret_cast<float4*>(P + base + 4) = v1;
                } else {
                    for (int e = 0; e < 8; e++)
                        if (nok[nn + e]) P[base + e] = v[e];
                }
                continue;
            }
            const IT base = gC + mC[mm] + nC[nn];
            const bool run = nok[nn + 7] && nC[nn + 7] == nC[nn] + 7;
            if constexpr (sizeof(TC) == 2) {
                if (run && ((uintptr_t)(C + base) & 15) == 0) {
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; e++) w[e] = pk_bf16(v[2 * e], v[2 * e + 1]);
                    *reinterpret_cast<uint4*>(C + base) = make_uint4(w[0], w[1], w[2], w[3]);
                    continue;
                }
            } else {
                if (run && ((uintptr_t)(C + base) & 15) == 0) {
                    *reinterpret_cast<float4*>(C + base) = v0;
                    *reinterpret_cast<float4*>(C + base + 4) = v1;
                    continue;
                }
            }
            for (int e = 0; e < 8; e++)
                if (nok[nn + e]) store(C, (int64_t)(gC + mC[mm] + nC[nn + e]), v[e]);
        }
    }
}

// C[g][m][n] = sum over chunks (in order) of P[g][chunk][m][n], in double: a
// block takes 64 consecutive outputs (one per lane) of one g; its four
// wavefronts sum contiguous quarters of the chunks with eight loads in flight,
// then the quarters are added in a fixed order.
__device__ __forceinline__ int64_t tc_out_offset(const TcDesc& d, int64_t g, int64_t m, int64_t n) {
    if (d.off32) {
        // every index and offset fits 31 bits: 32-bit divisions (64-bit ones
        // are long software sequences)
        uint32_t off = 0, x = (uint32_t)g;
        for (int i = d.ng - 1; i >= 0; --i) {
            const uint32_t sz = (uint32_t)d.g_size[i];
            off += (x % sz) * (uint32_t)d.g_sC[i];
            x /= sz;
        }
        x = (uint32_t)m;
        for (int i = d.nm - 1; i >= 0; --i) {
            const uint32_t sz = (uint32_t)d.m_size[i];
            off += (x % sz) * (uint32_t)d.m_sC[i];
            x /= sz;
        }
        x = (uint32_t)n;
        for (int i = d.nn - 1; i >= 0; --i) {
            const uint32_t sz = (uint32_t)d.n_size[i];
            off += (x % sz) * (uint32_t)d.n_sC[i];
            x /= sz;
        }
        return off;
    }
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
    return off;
}

// Few chunks (ksplit <= 8): one output a thread, its partials summed in
// chunk order (in double); 256 outputs of one g a block.
template <typename TC>
__global__ void __launch_bounds__(256) tc_reduce_few(TcDesc d, const float* __restrict__ P, TC* __restrict__ C) {
    const int64_t MN = d.M * d.N, per_g = (MN + 255) / 256;
    const int64_t g = blockIdx.x / per_g, mn = (blockIdx.x - g * per_g) * 256 + threadIdx.x;
    if (g >= d.G || mn >= MN) return;
    const float* p = P + g * d.ksplit * MN + mn;
    float v[8];
#pragma unroll
    for (int c = 0; c < 8; c++) v[c] = c < d.ksplit ? p[c * MN] : 0.f;
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < 8; c++) acc += v[c];
    int64_t m, n;
    if (d.off32) {
        m = (uint32_t)mn / (uint32_t)d.N;
        n = (uint32_t)mn - (uint32_t)m * (uint32_t)d.N;
    } else {
        m = mn / d.N;
        n = mn - m * d.N;
    }
    store(C, tc_out_offset(d, g, m, n), (float)acc);
}

// More chunks: 64 outputs of one g a block; its NW waves sum consecutive runs
// of the chunks (16 loads in flight a lane), wave 0 adds the run sums in wave
// order (NW from ksplit alone: 4 up to 64 chunks, else 16).
template <int NW, typename TC>
__global__ void __launch_bounds__(64 * NW) tc_reduce(TcDesc d, const float* __restrict__ P, TC* __restrict__ C) {
    __shared__ double q[NW][64];
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t MN = d.M * d.N, per_g = (MN + 63) / 64;
    const int64_t g = blockIdx.x / per_g, mn = (blockIdx.x - g * per_g) * 64 + lane;
    const int64_t run = (d.ksplit + NW - 1) / NW;
    const int64_t c0 = wave * run, c1 = min((int64_t)d.ksplit, c0 + run);
    double acc = 0.0;
    if (g < d.G && mn < MN) {
        const float* p = P + g * d.ksplit * MN + mn;
        int64_t c = c0;
        for (; c + 16 <= c1; c += 16) {
            float v[16];
#pragma unroll
            for (int u = 0; u < 16; u++) v[u] = p[(c + u) * MN];
#pragma unroll
            for (int u = 0; u < 16; u++) acc += v[u];
        }
        for (; c < c1; c++) acc += p[c * MN];
    }
    q[wave][lane] = acc;
    __syncthreads();
    if (wave != 0 || g >= d.G || mn >= MN) return;
    double sum = q[0][lane];
#pragma unroll
    for (int w = 1; w < NW; w++) sum += q[w][lane];
    const int64_t m = mn / d.N, n = mn - m * d.N;
    store(C, tc_out_offset(d, g, m, n), (float)sum);
}

template <typename T, typename TC>
hipError_t tc_launch_t(const TcDesc& d, const Launch& ln, const void* a, const void* b, void* c, void* p,
                       hipStream_t s) {
    const int MT = d.M > 32 ? 2 : 1;
    dim3 g(ln.grid[0]), bl(256);
    if (d.off32 && (d.extA >= ((int64_t)1 << 31) || d.extB >= ((int64_t)1 << 31))) return hipErrorInvalidValue;
    // bf16 reductions of 64 and more take slices of 64
    constexpr int TKW = sizeof(T) == 2 ? 64 : 32;
    const bool wide = sizeof(T) == 2 && d.K >= 64;
    // one slice a block (every chunk within one slice): single-buffered
    const bool one = d.kchunk <= (wide ? TKW : 32);
#define TC_LAUNCH(mt, IT, tk, nb) \
    do { \
        if (d.kmajor) hipLaunchKernelGGL((tc_gemm<T, TC, mt, IT, tk, nb, true>), g, bl, 0, s, d, (const T*)a, (const T*)b, (TC*)c, (float*)p); \
        else hipLaunchKernelGGL((tc_gemm<T, TC, mt, IT, tk, nb, false>), g, bl, 0, s, d, (const T*)a, (const T*)b, (TC*)c, (float*)p); \
    } while (0)
#define TC_TK(mt, IT) \
    do { \
        if (wide) { if (one) TC_LAUNCH(mt, IT, TKW, 1); else TC_LAUNCH(mt, IT, TKW, 2); } \
        else { if (one) TC_LAUNCH(mt, IT, 32, 1); else TC_LAUNCH(mt, IT, 32, 2); } \
    } while (0)
    if (d.off32) {
        if (MT == 2) TC_TK(2, int32_t);
        else TC_TK(1, int32_t);
    } else {
        if (MT == 2) TC_TK(2, int64_t);
        else TC_TK(1, int64_t);
    }
#undef TC_TK
#undef TC_LAUNCH
    return hipGetLastError();
}

}  // namespace

hipError_t launch_tc(const Launch& ln, const void* a, const void* b, void* c, void* d, hipStream_t s) {
    TcDesc t;
    std::memcpy(&t, ln.desc.data(), sizeof(t));
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    if ((ln.kind & 0xff) == K_TC_REDUCE) {
        dim3 g(ln.grid[0]), bl(256);
        const int64_t per = t.ksplit <= 8 ? 256 : 64;   // outputs of one g a block
        if ((int64_t)ln.grid[0] != t.G * ((t.M * t.N + per - 1) / per)) return hipErrorInvalidValue;
        if (t.ksplit <= 8) {
            if (tC) hipLaunchKernelGGL((tc_reduce_few<bf16_t>), g, bl, 0, s, t, (const float*)d, (bf16_t*)c);
            else hipLaunchKernelGGL((tc_reduce_few<float>), g, bl, 0, s, t, (const float*)d, (float*)c);
        } else if (t.ksplit <= 64) {
            if (tC) hipLaunchKernelGGL((tc_reduce<4, bf16_t>), g, dim3(256), 0, s, t, (const float*)d, (bf16_t*)c);
            else hipLaunchKernelGGL((tc_reduce<4, float>), g, dim3(256), 0, s, t, (const float*)d, (float*)c);
        } else {
            if (tC) hipLaunchKernelGGL((tc_reduce<16, bf16_t>), g, dim3(1024), 0, s, t, (const float*)d, (bf16_t*)c);
            else hipLaunchKernelGGL((tc_reduce<16, float>), g, dim3(1024), 0, s, t, (const float*)d, (float*)c);
        }
        return hipGetLastError();
    }
    if (tIn) return tC ? tc_launch_t<bf16_t, bf16_t>(t, ln, a, b, c, d, s) : tc_launch_t<bf16_t, float>(t, ln, a, b, c, d, s);
    return tC ? tc_launch_t<float, bf16_t>(t, ln, a, b, c, d, s) : tc_launch_t<float, float>(t, ln, a, b, c, d, s);
}

}  // namespace ce
