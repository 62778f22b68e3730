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
#include <type_traits>

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

// v where m is all ones, zero where it is zero
__device__ __forceinline__ bf16x8 mask8(bf16x8 v, uint32_t m) {
    uint32_t w[4];
    __builtin_memcpy(w, &v, 16);
#pragma unroll
    for (int i = 0; i < 4; i++) w[i] &= m;
    __builtin_memcpy(&v, w, 16);
    return v;
}

// eight float32 -> bf16x8 by four paired conversions
__device__ __forceinline__ bf16x8 cvt8(const float* v) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; i++) w[i] = pk_bf16(v[2 * i], v[2 * i + 1]);
    bf16x8 r;
    __builtin_memcpy(&r, w, 16);
    return r;
}

// Twenty wait states after an MFMA chain whose result VALU code reads next.
// The compiler's hazard padding has been seen to miss the read of a 16-pass
// MFMA result on a branch path that skips straight to it; this pads on every
// path, before any branch (about 1% of a row's MFMA time).
__device__ __forceinline__ void mfma_drain() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Logical tile of a block: the dispatcher deals consecutive blocks round-robin
// to the 8 XCDs (each with its own L2), so XCD x gets a contiguous range of
// logical tiles; neighbouring strips and segments, which share halo rows and
// cache lines, then meet in one L2.
__device__ __forceinline__ int64_t xcd_tile(int64_t bid, int64_t nb) {
    const int64_t q = nb / 8, r = nb % 8, x = bid % 8, i = bid / 8;
    return x * q + (x < r ? x : r) + i;
}

// the value of lane l - 1 (lane_prev) or l + 1 (lane_next) of the wavefront;
// zero past its ends (DPP whole-wave shifts)
__device__ __forceinline__ float lane_prev(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x138, 0xf, 0xf, true));
}
__device__ __forceinline__ float lane_next(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x130, 0xf, 0xf, true));
}

// r held by accumulator i of a lane in a 32x32 MFMA result
__device__ __forceinline__ int row32(int i, int lane) {
    return 8 * (i >> 2) + 4 * ((lane >> 5) & 1) + (i & 3);
}

// A-operand slots are stored one per 32-bit word (a bf16 value zero-extended).
// bf16 pairs are packed only where the MFMA consumes them, behind an empty asm
// that pins the loaded word: packing right after the load would make the wave
// wait for it there and undo the prefetch.
template <typename T> struct Slots { static constexpr int per_word = 1; };

// bf16x8 from eight zero-extended 16-bit words, packed at the point of use
__device__ __forceinline__ bf16x8 pack_words(const uint32_t* w) {
    uint32_t p[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        uint32_t lo = w[2 * i], hi = w[2 * i + 1];
        asm volatile("" : "+v"(lo), "+v"(hi));
        p[i] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);   // low halves of lo, hi
    }
    bf16x8 v;
    __builtin_memcpy(&v, p, 16);
    return v;
}


// Operands of one chunk of an MFMA chain, read from LDS ahead of use.
template <int N> struct Opnd { float v[N]; };

// No side work (see piped).
struct NoSide {
    __device__ void operator()(int) const {}
};

// Runs the MFMA chunks mm(c, buf[c]) for c = 0..NC-1 with the LDS operands of
// chunk c + D requested (ld) before chunk c's MFMAs issue; the scheduling
// fences keep that order, so each chunk's LDS latency hides behind D chunks of
// MFMA work instead of stalling the chain at every step.  side(c) is further
// memory work (LDS writes, global loads and stores) issued with chunk c: such
// instructions issue while a 32x32x2 fp32 MFMA executes (VALU instructions do
// not), so spread over the chain they cost no time of their own.
template <int NC, int D, int N, typename Ld, typename Mm, typename Sd = NoSide>
__device__ __forceinline__ void piped(Ld ld, Mm mm, Sd side = {}) {
    Opnd<N> buf[NC];
#pragma unroll
    for (int c = 0; c < (D < NC ? D : NC); c++) buf[c] = ld(c);
#pragma unroll
    for (int c = 0; c < NC; c++) {
        if (c + D < NC) buf[c + D] = ld(c + D);
        __builtin_amdgcn_sched_barrier(0);
        mm(c, buf[c]);
        side(c);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Channel of A-operand slot u of a lane in half hf (K channels per row GEMM):
// fp32 32x32x2 steps take channels 2u + hf; bf16 32x32x16 steps take
// 16*(u/8) + 8*hf + u%8.
template <bool BF>
__device__ __forceinline__ int achan(int u, int hf) {
    return BF ? 16 * (u >> 3) + 8 * hf + (u & 7) : 2 * u + hf;
}

// Z^T[col][r] = sum_k a[k][col] tab[r][k]: a = one activation row in A-operand
// slots (K/2 values a lane), tab = [32][lda] factor table in LDS.  side(c),
// c = 0..K/4-1, is memory work issued along the chain (see piped).
template <typename T, int K, bool DRAIN = true, typename Sd = NoSide>
__device__ __forceinline__ f32x16 tgemm(const uint32_t (&a)[K / 2 / Slots<T>::per_word], const T* tab, int lda,
                                        int cl, int hf, Sd side = {}) {
    f32x16 acc;
#pragma unroll
    for (int i = 0; i < 16; i++) acc[i] = 0.f;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int q = 0; q < K / 16; q++) {
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pack_words(a + 8 * q), lds8(tab + cl * lda + 16 * q + 8 * hf),
                                                          acc, 0, 0, 0);
#pragma unroll
            for (int c = 4 * q; c < 4 * q + 4; c++) side(c);
        }
    } else {
        // MFMA u takes k = 2u + hf; chunks of two MFMAs, operands four chunks ahead
        const float* tb = tab + cl * lda + hf;
        piped<K / 4, 4, 2>(
            [&](int c) {
                Opnd<2> o;
                o.v[0] = tb[4 * c];
                o.v[1] = tb[4 * c + 2];
                return o;
            },
            [&](int c, const Opnd<2>& o) {
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[2 * c]), o.v[0], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[2 * c + 1]), o.v[1], acc, 0, 0, 0);
            },
            side);
    }
    if constexpr (DRAIN) mfma_drain();
    return acc;
}

// Raw buffer access (gfx9 family): a wave-uniform resource (base, byte range)
// and a per-lane byte offset.  The range check covers the per-lane offset:
// loads past the range return 0 and stores past it are dropped.
constexpr int kBufCfg = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t brsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kBufCfg);
}
template <typename T>
__device__ __forceinline__ T bload(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    if constexpr (sizeof(T) == 2) return (T)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)soff, 0);
    else return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
}
__device__ __forceinline__ void bstore(float v, __amdgpu_buffer_rsrc_t r, uint32_t voff) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)voff, 0, 0);
}
__device__ __forceinline__ void bstore(float v, bf16_t*, __amdgpu_buffer_rsrc_t r, uint32_t voff) {
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(v), r, (int)voff, 0, 0);
}
__device__ __forceinline__ void bstore(float v, float*, __amdgpu_buffer_rsrc_t r, uint32_t voff) {
    bstore(v, r, voff);
}
// the same with a wave-uniform offset soff added (scalar register operand)
__device__ __forceinline__ void bstore(float v, bf16_t*, __amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(v), r, (int)voff, (int)soff, 0);
}
__device__ __forceinline__ void bstore(float v, float*, __amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)voff, (int)soff, 0);
}

// One activation row in A-operand slots: a[u] = src[achan(u, hf)][row][col].
// voff = byte offset of (channel hf, row, the lane's column), or an offset
// past the range for lanes outside the image (which then read zeros); cs =
// channel stride in bytes.  The channel step goes in the uniform offset.
template <typename T, int K>
__device__ __forceinline__ void arow(uint32_t (&a)[K / 2], __amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t cs) {
#pragma unroll
    for (int u = 0; u < K / 2; u++) {
        if constexpr (sizeof(T) == 2)
            a[u] = __builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)((16 * (u >> 3) + (u & 7)) * cs), 0);
        else
            a[u] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)(2 * u * cs), 0);
    }
}

// A-operand slot u of an activation row (one element of arow).
template <typename T>
__device__ __forceinline__ uint32_t aslot(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t cs, int u) {
    if constexpr (sizeof(T) == 2)
        return __builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)((16 * (u >> 3) + (u & 7)) * cs), 0);
    else
        return __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)(2 * u * cs), 0);
}

// Two blocks per CU (256 VGPRs a lane) except for the bf16 5x5 variant, whose
// larger ring and bf16 operand packing do not fit that without spilling.
// PT: T is not a whole number of 32-channel blocks (bf16 stores then go
// through the range-checked Y buffer, which drops the padded channels)
template <typename T, int KH, int KW, int MB2, int MS, bool PT = false>
__global__ void __launch_bounds__(256, (sizeof(T) == 2 && KH == 5) ? 1 : 2) cp_fwd(CpDesc d, const T* __restrict__ X,
                                              const T* __restrict__ Us, const T* __restrict__ Kh,
                                              const T* __restrict__ Kw, const T* __restrict__ Ut,
                                              T* __restrict__ Y) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int TT = 32 * MB2, NS = 32 * MS;
    constexpr int CH = (KH - 1) / 2, HWW = (KW - 1) / 2;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int H = d.H, W = d.W;
    const int LDA = d.lda;
    T* UsL = (T*)smem;
    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // ---- this wavefront's strip ----
    // strips fastest: the waves of a block share halo rows and cache lines
    // (set up before the tables, so that its first X rows are in flight
    // while they load; waves past the end load nothing and leave after the
    // barrier)
    const int64_t gw = xcd_tile(blockIdx.x, gridDim.x) * 4 + wave;
    const bool wok = gw < d.waves;
    int cb = 0, seg = 0, b = 0;
    if (wok) {
        cb = (int)(gw % d.ncb);
        const int64_t rest = gw / d.ncb;
        seg = (int)(rest % d.segs);
        b = (int)(rest / d.segs);
    }
    const int col = cb * d.colstride - HWW + (lane & 31);
    const bool colok = col >= 0 && col < W;
    // Rows in walk order: for bf16, odd segments walk upwards (walk row r is
    // image row H - 1 - r, and the vertical taps are taken reversed), so that
    // the two segments at every boundary read its halo rows at the same time,
    // both at their starts or both at their ends, and the second read finds
    // them in L2 (C2 bf16: forward + backward 86.0 -> 84.5 us; for fp32 the
    // step measured 1.5% slower, with a forward no faster).  h0, h1 bound the
    // segment in walk rows.
    const bool up = BF && (seg & 1) != 0;
    const int p0 = seg * d.seg_rows, p1 = min(H, p0 + d.seg_rows);
    const int h0 = up ? H - p1 : p0, h1 = up ? H - p0 : p1;
    auto prow = [&](int r) { return up ? H - 1 - r : r; };
    const bool store_lane = colok && (lane & 31) >= HWW && (lane & 31) < 32 - HWW;
    const int cl = lane & 31;

    // X rows as B-operand slots (the same slot layout as arow), loaded PD rows
    // ahead through a raw buffer: rows and lanes outside the image read zeros,
    // and so do the rows past the segment's last (X row h1 - 1 + CH), which
    // the last rows' prefetches would otherwise fetch for nothing
    constexpr uint32_t E = sizeof(T);
    constexpr int PD = BF ? 1 : 2;
    const __amdgpu_buffer_rsrc_t rX = brsrc(X + (int64_t)b * d.x_sb, (uint32_t)(d.S * d.x_ss * E));
    const uint32_t xcs = (uint32_t)(d.x_ss * E);
    const uint32_t kOut = 0x80000000u;   // past the range: reads 0
    const uint32_t xa0 = colok ? (uint32_t)(col * E) + (BF ? 8u : 1u) * half * xcs : kOut;
    const int xlast = min(H - 1, h1 - 1 + CH);
    auto xoff = [&](int row) { return (row >= 0 && row <= xlast) ? xa0 + (uint32_t)(prow(row) * W) * E : kOut; };
    // fp32: two row buffers, the rows of the walk alternating between them
    uint32_t xa[NS / 2], xb[NS / 2];
    // Z1[r][col] = sum_s Us[r][s] X[s][row][col] for the row held in a; side(c),
    // c = 0..NS/4-1, is memory work issued along the chain (see piped)
    auto gemm1 = [&](const uint32_t (&a)[NS / 2], auto side) {
        f32x16 acc;
#pragma unroll
        for (int i = 0; i < 16; i++) acc[i] = 0.f;
        if constexpr (BF) {
#pragma unroll
            for (int q = 0; q < NS / 16; q++) {
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(UsL + cl * LDA + 16 * q + 8 * half),
                                                              pack_words(a + 8 * q), acc, 0, 0, 0);
#pragma unroll
                for (int c = 4 * q; c < 4 * q + 4; c++) side(c);
            }
        } else {
            // MFMA u takes channel 2u + half; chunks of two MFMAs, operands four chunks ahead
            const T* ub = UsL + cl * LDA + half;
            piped<NS / 4, 4, 2>(
                [&](int c) {
                    Opnd<2> o;
                    o.v[0] = ub[4 * c];
                    o.v[1] = ub[4 * c + 2];
                    return o;
                },
                [&](int c, const Opnd<2>& o) {
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(o.v[0], __uint_as_float(a[2 * c]), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(o.v[1], __uint_as_float(a[2 * c + 1]), acc, 0, 0, 0);
                },
                side);
        }
        mfma_drain();
        return acc;
    };

    // The first row of the walk is requested before the tables load, each
    // further row of the ring fill just before the row ahead of it is
    // computed (NP row buffers): at the start every wavefront asks at once,
    // and its first row then waits behind fewer requests.
    constexpr int NP = KH < 3 ? KH : 3;
    uint32_t xp[NP][NS / 2];
    if (wok) {
#pragma unroll
        for (int p = 0; p < 1; p++) arow<T, NS>(xp[p], rX, xoff(h0 - CH + p), xcs);
    }
    // ---- tables ----
    // Each thread issues all of its table loads before any LDS store, so that
    // their memory latencies overlap.
    {
    T* UtP = (T*)(smem + d.o_ut);
    float* KhP = (float*)(smem + d.o_kh);
    float* KwP = (float*)(smem + d.o_kw);
    constexpr int QS = NS / 8, QT = TT / 8;     // elements a thread (256 threads)
    constexpr int NKH = 32 * KH, NKW = 32 * KW;  // tap tables, at most one element a thread
    static_assert(NKH <= 256 && NKW <= 256, "tap tables fit one pass");
    T vs[QS], vt[QT];
    float vkh = 0.f, vkw = 0.f;
    // UtP[q][hf][t][j] = Ut[row32(8q+j, 32*hf)][t] (bf16), UtP[i][hf][t] = Ut[row32(i, 32*hf)][t] (fp32).
    // A rank of R < 32 leaves ranks R..31 of every table zero: their Z1, Z2
    // and Z3 rows are zero and add nothing to Y.
    auto ut_rank = [&](int e) {
        if constexpr (BF) return row32(8 * (e / (16 * TT)) + (e & 7), 32 * ((e / (8 * TT)) & 1));
        else return row32(e / (2 * TT), 32 * ((e / TT) & 1));
    };
    auto ut_col = [&](int e) { return BF ? (e >> 3) % TT : e % TT; };
#pragma unroll
    for (int q = 0; q < QS; q++) {
        const int e = tid + 256 * q, r = e / NS, s = e - r * NS;
        vs[q] = Us[min(r, d.R - 1) * d.us_sr + min(s, d.S - 1) * d.us_ss];
    }
#pragma unroll
    for (int q = 0; q < QT; q++) {
        const int e = tid + 256 * q;
        vt[q] = Ut[min(ut_rank(e), d.R - 1) * d.ut_sr + min(ut_col(e), d.T - 1) * d.ut_st];
    }
    // (every load unconditional, at a clamped index: a load under a condition
    // makes the compiler wait for all outstanding loads, the first X row's
    // included, before the next memory use; the padding is zeroed at the stores)
    if (tid < NKH) {
        const int j = tid % KH, hf = (tid / KH) & 1, r = row32(tid / (2 * KH), 32 * hf);
        vkh = load(Kh, min(r, d.R - 1) * d.kh_sr + j * d.kh_sj);
    }
    if (tid < NKW) {
        const int j = tid % KW, hf = (tid / KW) & 1, r = row32(tid / (2 * KW), 32 * hf);
        vkw = load(Kw, min(r, d.R - 1) * d.kw_sr + j * d.kw_sj);
    }
#pragma unroll
    for (int q = 0; q < QS; q++) {
        const int e = tid + 256 * q, r = e / NS, s = e - r * NS;
        UsL[r * LDA + s] = r < d.R && s < d.S ? vs[q] : (T)0;
    }
#pragma unroll
    for (int q = 0; q < QT; q++) {
        const int e = tid + 256 * q;
        UtP[e] = ut_rank(e) < d.R && ut_col(e) < d.T ? vt[q] : (T)0;
    }
    if (tid < NKH) {
        // and the same taps reversed at o_khr, for the upward walk
        const int j = tid % KH, hf = (tid / KH) & 1, r = row32(tid / (2 * KH), 32 * hf);
        const float v = r < d.R ? vkh : 0.f;
        KhP[tid] = v;
        ((float*)(smem + d.o_khr))[tid + KH - 1 - 2 * j] = v;
    }
    if (tid < NKW) {
        const int hf = (tid / KW) & 1, r = row32(tid / (2 * KW), 32 * hf);
        KwP[tid] = r < d.R ? vkw : 0.f;
    }
    }
    __syncthreads();
    if (!wok) return;

    f32x16 ring[KH];
#pragma unroll
    for (int j = 0; j < KH - 1; j++) {
        if (j + 1 < NP) arow<T, NS>(xp[j + 1], rX, xoff(h0 - CH + j + 1), xcs);
        ring[j] = gemm1(xp[j % NP], NoSide{});
        if (j + NP < KH) arow<T, NS>(xp[j % NP], rX, xoff(h0 - CH + j + NP), xcs);
    }
#pragma unroll
    for (int u = 0; u < NS / 2; u++) xa[u] = xp[(KH - 1) % NP][u];
    if constexpr (PD == 2) arow<T, NS>(xb, rX, xoff(h0 + CH + 1), xcs);
    // Y rows through a raw buffer (one sample; stores past the range are
    // dropped): the lane's column and channel 4*half in the lane offset, the
    // rest of the channel in the uniform offset (Y's channel stride is X's)
    const __amdgpu_buffer_rsrc_t rYo = brsrc(Y + (int64_t)b * d.y_sb, (uint32_t)(d.T * d.x_ss * E));
    const uint32_t yv0 = store_lane ? (uint32_t)(col * E) + 4u * half * xcs : kOut;
    // Y row h - 1, stored along the next row's first chain
    f32x16 accYp[MB2];
#pragma unroll
    for (int mb = 0; mb < MB2; mb++)
#pragma unroll
        for (int i = 0; i < 16; i++) accYp[mb][i] = 0.f;
    auto store_y = [&](int item, uint32_t v0) {   // item = 16 mb + i
        const int mb = item >> 4, i = item & 15, ch = 32 * mb + row32(i, 0);   // + 4 half, in yv0
        bstore(accYp[mb][i], (T*)nullptr, rYo, (ch & 1) ? v0 + xcs : v0, (uint32_t)(2 * (ch >> 1)) * xcs);
    };
    // row h: Z1 of X row h + CH from cur, which then takes X row h + CH + PD
    auto fwd_row = [&](int h, auto PST, uint32_t (&cur)[NS / 2]) {
        // The tap and Ut tables are re-read from LDS every row: the offsets
        // pass through an empty asm so the loads are not hoisted out of the
        // loop, where they would hold 16*(KH+KW+MB2) registers for its life.
        uint32_t o_ut = d.o_ut, o_kh = up ? d.o_khr : d.o_kh, o_kw = d.o_kw;
        asm volatile("" : "+s"(o_ut), "+s"(o_kh), "+s"(o_kw));
        const T* UtP = (const T*)(smem + o_ut);
        const float* KhP = (const float*)(smem + o_kh);
        const float* KwP = (const float*)(smem + o_kw);
        // fp32: memory work along the chains (their MFMAs leave the issue free
        // for it): the stores of Y row h - 1 along Z1 (pst), the loads of the
        // X row two rows ahead along GEMM2 (a whole row of latency cover: under
        // the load of the full chip a half row was not enough).  bf16 (short
        // chains): the loads of the next row right after Z1, the stores at the
        // end of the row.
        const uint32_t pv0 = yv0 + (uint32_t)(prow(h - 1) * W) * E;
        auto side_a = [&](int c) {   // c = 0..NS/4-1
            if constexpr (!BF && decltype(PST)::value) {
                constexpr int NC = NS / 4, PS = (16 * MB2 + NC - 1) / NC;
#pragma unroll
                for (int j = 0; j < PS; j++)
                    if (c * PS + j < 16 * MB2) store_y(c * PS + j, pv0);
            }
        };
        ring[KH - 1] = gemm1(cur, side_a);
        const uint32_t xo = xoff(h + CH + PD);   // used PD rows later
        if constexpr (BF) arow<T, NS>(cur, rX, xo, xcs);
        auto side_b = [&](int c) {   // c = 0..15
            if constexpr (BF) return;
            constexpr int PX = (NS / 2 + 15) / 16;
#pragma unroll
            for (int j = 0; j < PX; j++)
                if (c * PX + j < NS / 2) cur[c * PX + j] = aslot<T>(rX, xo, xcs, c * PX + j);
        };
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
        // conv along w: neighbouring columns are neighbouring lanes of the half;
        // whole-wave lane shifts (DPP) bring lane l - 1 and l + 1; what crosses
        // the half boundary lands in a halo column, which is never stored
        f32x16 z3;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float sh[KW];
            sh[HWW] = z2[i];
#pragma unroll
            for (int k = 1; k <= HWW; k++) {
                sh[HWW - k] = lane_prev(sh[HWW - k + 1]);
                sh[HWW + k] = lane_next(sh[HWW + k - 1]);
            }
            float a = 0.f;
#pragma unroll
            for (int jw = 0; jw < KW; jw++) a += KwP[(i * 2 + half) * KW + jw] * sh[jw];
            z3[i] = a;
        }
        // GEMM2: Y[t][col] = sum_r Ut[r][t] Z3[r][col] (fp32: into accYp, stored
        // along the next row's first chain)
        auto gemm2 = [&](f32x16 (&acc2)[MB2]) {
#pragma unroll
        for (int mb = 0; mb < MB2; mb++)
#pragma unroll
            for (int i = 0; i < 16; i++) acc2[mb][i] = 0.f;
        if constexpr (BF) {
#pragma unroll
            for (int q = 0; q < 2; q++) {
                float zf[8];
#pragma unroll
                for (int j = 0; j < 8; j++) zf[j] = z3[8 * q + j];
                bf16x8 bv = cvt8(zf);
#pragma unroll
                for (int mb = 0; mb < MB2; mb++) {
                    bf16x8 av = lds8(UtP + (((q * 2 + half) * TT) + mb * 32 + (lane & 31)) * 8);
                    acc2[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc2[mb], 0, 0, 0);
                }
            }
        } else {
            // chunk i: rank row32(i, half) of each channel block, three chunks ahead
            const T* ut = UtP + half * TT + (lane & 31);
            piped<16, 3, MB2>(
                [&](int i) {
                    Opnd<MB2> o;
#pragma unroll
                    for (int mb = 0; mb < MB2; mb++) o.v[mb] = ut[2 * i * TT + mb * 32];
                    return o;
                },
                [&](int i, const Opnd<MB2>& o) {
#pragma unroll
                    for (int mb = 0; mb < MB2; mb++)
                        acc2[mb] = __builtin_amdgcn_mfma_f32_32x32x2f32(o.v[mb], z3[i], acc2[mb], 0, 0, 0);
                },
                side_b);
        }
        mfma_drain();   // acc2 is read by the stores
        };
        if constexpr (BF) {
            f32x16 acc2[MB2];
            gemm2(acc2);
            if constexpr (PT) {
                // through the Y buffer (as the fp32 stores): lanes outside the
                // strip's own columns and padded channels fall outside its range
                const uint32_t pv = yv0 + (uint32_t)(prow(h) * W) * E;
#pragma unroll
                for (int mb = 0; mb < MB2; mb++)
#pragma unroll
                    for (int i = 0; i < 16; i++) {
                        const int ch = 32 * mb + row32(i, 0);   // + 4 half, in yv0
                        bstore(acc2[mb][i], (T*)nullptr, rYo, (ch & 1) ? pv + xcs : pv,
                               (uint32_t)(2 * (ch >> 1)) * xcs);
                    }
            } else if (store_lane) {
                T* yr = Y + (int64_t)b * d.y_sb + col + (int64_t)prow(h) * W;
#pragma unroll
                for (int mb = 0; mb < MB2; mb++)
#pragma unroll
                    for (int i = 0; i < 16; i++)
                        store(yr, (int64_t)(mb * 32 + row32(i, lane)) * d.y_st, acc2[mb][i]);
            }
        } else {
            gemm2(accYp);
        }
    };
    // The first rows run outside the loop: the loop is then entered, like its
    // back edge, with a Y row pending and the same memory operations
    // outstanding, so the wait counts the compiler derives for the prefetched
    // X rows at the loop head are those of the steady state.  fp32: the loop
    // takes two rows (buffers xa, xb), a last odd row follows it.
    const std::true_type yes;
    const std::false_type no;
    fwd_row(h0, no, xa);
    if constexpr (PD == 1) {
        for (int h = h0 + 1; h < h1; h++) fwd_row(h, yes, xa);
    } else if (h0 + 1 < h1) {
        fwd_row(h0 + 1, yes, xb);
        int h = h0 + 2;
        for (; h + 1 < h1; h += 2) {
            fwd_row(h, yes, xa);
            fwd_row(h + 1, yes, xb);
        }
        if (h < h1) fwd_row(h, yes, xa);
    }
    if constexpr (!BF) {
        const uint32_t lv0 = yv0 + (uint32_t)(prow(h1 - 1) * W) * E;
#pragma unroll
        for (int item = 0; item < 16 * MB2; item++) store_y(item, lv0);
    }
}

template <typename T, int K, int MB2>
hipError_t launch_cp_t(const CpDesc& d, const void* const* ops, void* y, hipStream_t s) {
    if (d.S < 1 || d.S > 64) return hipErrorInvalidValue;
    // bf16 with a padded T stores through the Y buffer (fp32 always does)
    const bool pt = sizeof(T) == 2 && d.T != 32 * MB2;
    auto k = d.S <= 32 ? (pt ? cp_fwd<T, K, K, MB2, 1, true> : cp_fwd<T, K, K, MB2, 1>)
                       : (pt ? cp_fwd<T, K, K, MB2, 2, true> : cp_fwd<T, K, K, MB2, 2>);
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d, (const T*)ops[0],
                       (const T*)ops[1], (const T*)ops[2], (const T*)ops[3], (const T*)ops[4], (T*)y);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_cp_ty(const CpDesc& d, const void* const* ops, void* y, hipStream_t s) {
    if (d.KH == 3 && d.KW == 3)
        return d.T <= 32 ? launch_cp_t<T, 3, 1>(d, ops, y, s) : launch_cp_t<T, 3, 2>(d, ops, y, s);
    if (d.KH == 5 && d.KW == 5)
        return d.T <= 32 ? launch_cp_t<T, 5, 1>(d, ops, y, s) : launch_cp_t<T, 5, 2>(d, ops, y, s);
    return hipErrorInvalidValue;
}


// ---------------------------------------------------------------------------
// Backward of the chain (Section 3.2: every pairwise step's two gradients, in
// reverse order, with the intermediates recomputed), fused the same way.  One
// wavefront walks its 32-column strip over rows h = h0-CH .. h1+CH-1 and at row h
//   recomputes  Z1[h+CH] (ring of KH rows), Z2[h], Z3[h]
//   dZ3[h] = Ut^T dY[h]
//   dUt   += Z3[h] dY[h]^T               (reduction over the strip's columns)
//   dKw   += sum_w Z2[h][w+j-c] dZ3[h][w]
//   dZ2[h] = transposed conv along w of dZ3[h]
//   dKh   += sum_w Z1[h+j-c][w] dZ2[h][w]
//   dZ1[h-CH] from the ring of the last KH dZ2 rows
//   dX[h-CH] = Us^T dZ1[h-CH]
//   dUs   += dZ1[h-CH] X[h-CH]^T
// Each weight-gradient term is counted once: rows in [h0, h1) and the strip's
// own columns only.
//
// The rank intermediates are held transposed: the MFMA computes Z^T[col][r]
// (A operand = the activation row, one column per lane; B operand = the factor
// table in LDS), so a lane holds one rank r (lane % 32) and the 16 columns
// tcol(i, half) of its accumulators.  Then
//   * conv along h is per element, conv along w a shift of the register index
//     (four cross-half exchanges per shift);
//   * the column reductions of dUt / dUs take Z^T straight from the
//     accumulators as the MFMA A operand (k slot = column);
//   * the tap-gradient products reduce over columns inside the lane;
//   * dX goes through one LDS transpose of dZ1 (and is stored coalesced).
// dY reaches the dUt product through a wave-private LDS tile; the X row of the
// dUs product is read channel-major from memory (it was read two rows earlier
// by the same wavefront).  The operands of the next row are loaded while the
// current row is computed.

// column held by accumulator i of a lane in half hf of a transposed tile
__device__ __forceinline__ int tcol(int i, int hf) { return 8 * (i >> 2) + 4 * hf + (i & 3); }

// a where the mask m is all ones, b where it is zero (one v_bfi_b32).  m is
// opaque to the compiler, which would otherwise turn a lane-dependent choice
// between two fixed elements of a register array into a dynamic index (a
// fifteen-step compare/select chain per use).
__device__ __forceinline__ float blend(uint32_t m, float a, float b) {
    return __uint_as_float((__float_as_uint(a) & m) | (__float_as_uint(b) & ~m));
}
__device__ __forceinline__ uint32_t half_mask(int hf) {
    uint32_t m = hf ? 0xffffffffu : 0u;
    asm volatile("" : "+v"(m));
    return m;
}

// w[i] = v at column tcol(i, hf) + DD of the same rank (DD = +-1); values
// that would come from outside the 32 columns are unspecified.  hm =
// half_mask(hf).  Columns that cross between the lane halves come from lane
// l ^ 32: one v_permlane32_swap exchanges a pair of registers between the
// halves (p's upper half with q's lower half), then each half keeps its part.
template <int DD>
__device__ __forceinline__ f32x16 tshift(const f32x16& v, uint32_t hm) {
    float rcv[4];
#pragma unroll
    for (int a = 0; a < 4; a++) {
        // p: wanted by the lower half from the upper; q: by the upper from the lower
        float p, q;
        if constexpr (DD == 1) {
            p = v[4 * a];
            q = v[a < 3 ? 4 * a + 4 : 0];
        } else {
            p = v[a > 0 ? 4 * a - 1 : 0];
            q = v[4 * a + 3];
        }
        // r[0] = (p lanes 0-31, q lanes 0-31), r[1] = (p lanes 32-63, q lanes 32-63)
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(p), __float_as_uint(q), false, false);
        rcv[a] = blend(hm, __uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    f32x16 w;
#pragma unroll
    for (int i = 0; i < 16; i++) {
        const int b = i & 3;
        if constexpr (DD == 1) w[i] = b < 3 ? v[i + 1] : rcv[i >> 2];
        else w[i] = b > 0 ? v[i - 1] : rcv[i >> 2];
    }
    return w;
}

// LDS pitches (elements) of the backward kernel's tiles, fixed per type:
// factor tables [32][C + pad], bf16 transposed Us [C][40], dY tile [C][LY],
// X ring [3][C][LX] (8-byte bf16 / 16-byte fp32 column runs stay aligned).
template <typename T, int C> constexpr int cp_bwd_pitch_s() { return sizeof(T) == 2 ? C + 8 : C + 1; }
template <typename T> constexpr int cp_bwd_pitch_u() { return 40; }
template <typename T> constexpr int cp_bwd_pitch_y() { return sizeof(T) == 2 ? 40 : 33; }
template <typename T> constexpr int cp_bwd_pitch_x() { return sizeof(T) == 2 ? 40 : 36; }

// GEN: a rank below 32 or channel counts off the 32-channel blocks (clamped
// table loads, zeroed padding, compacted partials); the whole-block shapes
// compile without any of that (it moved the scheduling of the row loop and
// cost about 1.6 % of the kernel's time at R = 32, S = T = 64).
template <typename T, int KH, int KW, int MT, int MS, bool GEN>
__global__ void __launch_bounds__(256, 1)
    cp_bwd(CpBwdDesc d, const T* __restrict__ X, const T* __restrict__ dY,
           const T* __restrict__ Us, const T* __restrict__ Kh, const T* __restrict__ Kw,
           const T* __restrict__ Ut, T* __restrict__ dX, float* __restrict__ Pus,
           float* __restrict__ Put, float* __restrict__ Pkh, float* __restrict__ Pkw) {
    constexpr bool BF = sizeof(T) == 2;
    constexpr int NT = 32 * MT, NS = 32 * MS;
    constexpr int CH = (KH - 1) / 2, CW = (KW - 1) / 2;
    constexpr int LZ = 33;   // dZ1 transpose tile pitch (floats)
    // LDS pitches (elements) of the factor tables, the dY tile and the X ring;
    // the launcher checks that the descriptor's layout uses the same
    constexpr int LDA_S = cp_bwd_pitch_s<T, NS>(), LDA_T = cp_bwd_pitch_s<T, NT>();
    constexpr int LDU = cp_bwd_pitch_u<T>(), LY = cp_bwd_pitch_y<T>(), LX = cp_bwd_pitch_x<T>();
    static_assert(KW == 3, "column shifts of one");
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int H = d.H, W = d.W;
    const int tid = threadIdx.x, lane = tid & 63, hf = lane >> 5, cl = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    float* Tz = (float*)(smem + d.o_tz + (size_t)wave * d.tz_stride);
    T* Yt = (T*)(smem + d.o_yt + (size_t)wave * d.yt_bytes);
    T* Xl = (T*)(smem + d.o_xl + (size_t)wave * d.xl_bytes);   // ring of 3 X rows [slot][s][col]

    // ---- this wavefront's strip (waves past the end run no rows) ----
    const int64_t gw = xcd_tile(blockIdx.x, gridDim.x) * 4 + wave;
    const bool wok = gw < d.waves;
    int seg = 0, cb = 0, b = 0;
    if (wok) {   // strips fastest (see the forward kernel)
        cb = (int)(gw % d.ncb);
        const int64_t rest = gw / d.ncb;
        seg = (int)(rest % d.segs);
        b = (int)(rest / d.segs);
    }
    const int h0 = seg * d.seg_rows, h1 = wok ? min(H, h0 + d.seg_rows) : h0;
    const int col0 = cb * d.colstride - CW;
    const int col = col0 + cl;                       // the lane's column (A operands, dX)
    const bool colok = col >= 0 && col < W;
    const bool ownlane = colok && cl >= CW && cl < 32 - CW;
    const uint32_t hm = half_mask(hf);
    // v with the strip-overlap columns zeroed: column 0 is accumulator 0 of the
    // lower lane half, column 31 accumulator 15 of the upper (one column of
    // overlap on each side: KW == 3)
    auto own_cols = [hm](const f32x16& v) {
        f32x16 w = v;
        w[0] = blend(hm, v[0], 0.f);
        w[15] = blend(~hm, v[15], 0.f);
        return w;
    };
    constexpr uint32_t E = sizeof(T);
    // one sample of X / dY / dX (fits a 32-bit byte range; checked by the planner)
    const __amdgpu_buffer_rsrc_t rX = brsrc(X + (int64_t)b * d.x_sb, (uint32_t)(d.S * d.x_ss * E));
    const __amdgpu_buffer_rsrc_t rY = brsrc(dY + (int64_t)b * d.y_sb, (uint32_t)(d.T * d.y_st * E));
    const uint32_t xcs = (uint32_t)(d.x_ss * E), ycs = (uint32_t)(d.y_st * E);
    const uint32_t kOut = 0x80000000u;   // past every range: reads 0
    // A-operand lane offsets (channel hf, row 0, the lane's column)
    const uint32_t xa0 = colok ? (uint32_t)(col * E) + (BF ? 8u : 1u) * hf * xcs : kOut;
    const uint32_t ya0 = colok ? (uint32_t)(col * E) + (BF ? 8u : 1u) * hf * ycs : kOut;
    float kh[KH], kw[KW];                            // this lane's rank: r = cl
#pragma unroll
    // (a lane past the rank R reads rank R - 1's taps: its Z1 and dZ3 rows are
    // zero, so they multiply zeros, and its tap gradients are not written)
    for (int j = 0; j < KH; j++) kh[j] = load(Kh, (GEN ? min(cl, d.R - 1) : cl) * d.kh_sr + j * d.kh_sj);
#pragma unroll
    for (int j = 0; j < KW; j++) kw[j] = load(Kw, (GEN ? min(cl, d.R - 1) : cl) * d.kw_sr + j * d.kw_sj);

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
    float tk[KH], tw[KW];                            // tap-gradient sums of rank cl
#pragma unroll
    for (int j = 0; j < KH; j++) tk[j] = 0.f;
#pragma unroll
    for (int j = 0; j < KW; j++) tw[j] = 0.f;

    const T* UsA = (const T*)smem;
    const T* UtA = (const T*)(smem + d.o_uta);
    const T* UsT = (const T*)(smem + d.o_ust);
    const int hs = h0 - CH;
    // A-operand row offsets: rows outside the image (and lanes outside it) read zeros
    // (X rows past h1 are not read: the last row's prefetch would fetch one for nothing)
    const int xlast = min(H - 1, h1);
    auto xoff = [&](int row) { return (row >= 0 && row <= xlast) ? xa0 + (uint32_t)(row * W) * E : kOut; };
    auto yoff = [&](int row) { return (row >= 0 && row < H) ? ya0 + (uint32_t)(row * W) * E : kOut; };
    // dX: a zero range drops every store when the gradient is not wanted
    const __amdgpu_buffer_rsrc_t rD =
        brsrc(dX ? (const T*)dX + (int64_t)b * d.x_sb : X, dX ? (uint32_t)(d.S * d.x_ss * E) : 0u);
    const uint32_t dx0 = ownlane ? (uint32_t)(col * (int)E) + 4u * hf * xcs : kOut;
    constexpr int PW = Slots<T>::per_word;
    uint32_t xa[NS / 2 / PW], ya[NT / 2 / PW];
    // the X row held in xa into ring slot `slot` (channel-major), for the dUs
    // product CH rows later; X row r sits in slot (r - (hs - CH)) % 3
    auto xl_put = [&](int slot, const uint32_t (&src)[NS / 2 / PW]) {
        T* dst = Xl + slot * NS * LX + cl;
#pragma unroll
        for (int u = 0; u < NS / 2; u++) {
            if constexpr (BF) dst[achan<BF>(u, hf) * LX] = (T)src[u];
            else dst[achan<BF>(u, hf) * LX] = __uint_as_float(src[u]);
        }
    };
    auto xl_one = [&](int slot, int u, uint32_t v) {
        T* dst = Xl + slot * NS * LX + achan<BF>(u, hf) * LX + cl;
        if constexpr (BF) *dst = (T)v;
        else *dst = __uint_as_float(v);
    };
    f32x16 accXp[MS];   // the dX row of the previous row, stored along the next row's first chain
#pragma unroll
    for (int n = 0; n < MS; n++)
#pragma unroll
        for (int i = 0; i < 16; i++) accXp[n][i] = 0.f;
    // The first ring row is requested before the factor tables load, each
    // further operand row just before the ring row ahead of it is computed
    // (at the start every wavefront asks at once; its first row then waits
    // behind fewer requests).
    uint32_t xp[KH - 1][NS / 2 / PW];
    if (wok) {
        arow<T, NS>(xp[0], rX, xoff(hs - CH), xcs);
    }
    // ---- tables: UsA [32][lda_s], UtA [32][lda_t] (and UsT [NS][ldu] for bf16) ----
    // Each thread issues all of its table loads before any LDS store, so that
    // their memory latencies overlap.
    {
        constexpr int QS = NS / 8, QT = NT / 8;   // elements a thread (256 threads)
        T vs[QS], vt[QT], vu[QS];
#pragma unroll
        for (int q = 0; q < QS; q++) {
            const int e = tid + 256 * q, r = e / NS, s = e - r * NS;
            vs[q] = GEN ? Us[min(r, d.R - 1) * d.us_sr + min(s, d.S - 1) * d.us_ss] : Us[r * d.us_sr + s * d.us_ss];
            if constexpr (BF) {
                const int s2 = e / 32, r2 = e - s2 * 32;
                vu[q] = GEN ? Us[min(r2, d.R - 1) * d.us_sr + min(s2, d.S - 1) * d.us_ss]
                            : Us[r2 * d.us_sr + s2 * d.us_ss];
            }
        }
#pragma unroll
        for (int q = 0; q < QT; q++) {
            const int e = tid + 256 * q, r = e / NT, t = e - r * NT;
            vt[q] = GEN ? Ut[min(r, d.R - 1) * d.ut_sr + min(t, d.T - 1) * d.ut_st] : Ut[r * d.ut_sr + t * d.ut_st];
        }
        T* usa = (T*)smem;
        T* uta = (T*)(smem + d.o_uta);
#pragma unroll
        for (int q = 0; q < QS; q++) {
            const int e = tid + 256 * q, r = e / NS, s = e - r * NS;
            // (loads at clamped indices; ranks past R and padded channels zeroed here)
            usa[r * LDA_S + s] = !GEN || (r < d.R && s < d.S) ? vs[q] : (T)0;
            if constexpr (BF) {
                const int s2 = e / 32, r2 = e - s2 * 32;
                ((T*)(smem + d.o_ust))[s2 * LDU + r2] = !GEN || (r2 < d.R && s2 < d.S) ? vu[q] : (T)0;
            }
        }
#pragma unroll
        for (int q = 0; q < QT; q++) {
            const int e = tid + 256 * q, r = e / NT, t = e - r * NT;
            uta[r * LDA_T + t] = !GEN || (r < d.R && t < d.T) ? vt[q] : (T)0;
        }
    }
    __syncthreads();
    if (wok) {
#pragma unroll
        for (int j = 0; j < KH - 1; j++) {
            if (j + 1 < KH - 1) arow<T, NS>(xp[j + 1], rX, xoff(hs - CH + j + 1), xcs);
            if (j + 1 == KH - 1) {
                arow<T, NS>(xa, rX, xoff(hs + CH), xcs);
                arow<T, NT>(ya, rY, yoff(hs), ycs);
            }
            ring[j] = tgemm<T, NS>(xp[j], UsA, LDA_S, cl, hf);
            xl_put(j, xp[j]);
        }
    }

    // One row of the walk.  Ownership of the weight-gradient terms: loads
    // outside the image read zeros, so every product there vanishes by
    // itself (dY = 0 makes dZ3 = 0, X = 0 makes Z1 = 0); what remains is the
    // strip overlap (columns 0 and 31, zeroed by own_cols) and the segment
    // halo rows: row h counts for dUt, dKw and dKh only inside the segment
    // (rin), row h - CH for dX and dUs (xin).  The halo rows run as separate
    // instances of the row code (compile-time flags) without those products,
    // and the last row also without Z1[h + CH], which only they would read;
    // the loop body itself stays free of branches.
    auto row_step = [&](int h, auto RIN, auto XIN, auto Z1N, auto PST) {
        constexpr bool rin = decltype(RIN)::value, xin = decltype(XIN)::value;
        constexpr bool z1 = decltype(Z1N)::value, pst = decltype(PST)::value;
        const int hx = h - CH;
        const int k = h - hs;   // ring slots: X row h + CH goes to (k + 2) % 3, row hx is read from k % 3
        // Memory work rides on the MFMA chains (see piped):
        //   along Z1[h+CH]: the stores of the dX row of the previous row (pst)
        //   along dUt:      X row h + CH into its ring slot and the loads of X
        //                   row h + 1 + CH (rows followed by another: z1)
        //   along dUs:      the loads of dY[h + 1] (z1)
        // Rows without one of those products issue its share on their own.
        // Loaded rows are first used about half a row later or more: under
        // the full load of the chip a load takes several microseconds.
        const uint32_t pv0 = dx0 + (uint32_t)((hx - 1) * W) * E, pv1 = pv0 + xcs;
        const uint32_t xo = xoff(h + 1 + CH), yo = yoff(h + 1);   // the next rows' operands
        auto side_a = [&](int c) {
#pragma unroll
            for (int j = 0; j < 2; j++) {
                const int u = 2 * c + j;   // 0 .. NS/2 - 1 (= NT/2 - 1)
                if constexpr (pst) {
                    const int n = u >> 4, i = u & 15, ch = 32 * n + row32(i, 0);   // + 4hf, in dx0
                    bstore(accXp[n][i], (T*)nullptr, rD, (ch & 1) ? pv1 : pv0, (uint32_t)(2 * (ch >> 1)) * xcs);
                }
            }
        };
        f32x16 z1n;
        if constexpr (z1) {
            z1n = tgemm<T, NS>(xa, UsA, LDA_S, cl, hf, side_a);
        } else {
#pragma unroll
            for (int i = 0; i < 16; i++) z1n[i] = 0.f;
#pragma unroll
            for (int c = 0; c < NS / 4; c++) side_a(c);
        }
        const f32x16 dz3 = tgemm<T, NT, false>(ya, UtA, LDA_T, cl, hf);
        if constexpr (rin) {   // dY[h] into the LDS tile of the dUt product
#pragma unroll
            for (int u = 0; u < NT / 2; u++) {
                if constexpr (BF) Yt[achan<BF>(u, hf) * LY + cl] = (T)ya[u];
                else Yt[achan<BF>(u, hf) * LY + cl] = __uint_as_float(ya[u]);
            }
        }
        ring[KH - 1] = z1n;
        // Z2[h] (conv along h), Z3[h] (conv along w: tap j reads column + j - 1)
        f32x16 z2, z3, zm, zp;
        if constexpr (rin) {
#pragma unroll
            for (int i = 0; i < 16; i++) {
                float a = 0.f;
#pragma unroll
                for (int j = 0; j < KH; j++) a += kh[j] * ring[j][i];
                z2[i] = a;
            }
            zm = tshift<-1>(z2, hm);
            zp = tshift<1>(z2, hm);
#pragma unroll
            for (int i = 0; i < 16; i++) z3[i] = kw[0] * zm[i] + kw[1] * z2[i] + kw[2] * zp[i];
        }
        auto side_c = [&](int c) {   // c = 0..7
            if constexpr (z1) {
                constexpr int PX = NS / 16;
#pragma unroll
                for (int j = 0; j < PX; j++) {
                    const int u = c * PX + j;
                    xl_one((k + 2) % 3, u, xa[u]);
                    xa[u] = aslot<T>(rX, xo, xcs, u);
                }
            }
        };
        auto side_d = [&](int c) {   // c = 0..11
            if constexpr (z1) {
                constexpr int PY = NT / 8;
#pragma unroll
                for (int j = 0; j < PY; j++) {
                    const int u = c * PY + j;
                    if (c < 4) ya[u] = aslot<T>(rY, yo, ycs, u);
                }
            }
        };
        mfma_drain();   // dz3 is read below
        if constexpr (rin) {
            // dKw products
            const f32x16 g = own_cols(dz3);
            float t0 = 0.f, t1 = 0.f, t2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; i++) {
                t0 += zm[i] * g[i];
                t1 += z2[i] * g[i];
                t2 += zp[i] * g[i];
            }
            tw[0] += t0;
            tw[1] += t1;
            tw[2] += t2;
            const f32x16 z3o = own_cols(z3);
            // dUt += Z3[h] dY[h]^T
            if constexpr (BF) {
#pragma unroll
                for (int q = 0; q < 2; q++) {
                    float zf[8];
#pragma unroll
                    for (int j = 0; j < 8; j++) zf[j] = z3o[8 * q + j];
                    const bf16x8 av = cvt8(zf);
#pragma unroll
                    for (int n = 0; n < MT; n++) {
                        // columns tcol(8q + j, hf): 16q + 4hf + {0..3} and 16q + 8 + 4hf + {0..3}
                        const bf16_t* yr = Yt + (32 * n + cl) * LY + 16 * q + 4 * hf;
                        bf16_t bv[8];
                        __builtin_memcpy(bv, yr, 8);
                        __builtin_memcpy(bv + 4, yr + 8, 8);
                        accUt[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pack8(bv), accUt[n], 0, 0, 0);
                    }
#pragma unroll
                    for (int c = 4 * q; c < 4 * q + 4; c++) side_c(c);
                }
            } else {
                // chunk c: columns tcol(2c, hf) and tcol(2c + 1, hf) (adjacent) of each
                // channel block, three chunks ahead
                const float* yb = Yt + cl * LY + 4 * hf;
                piped<8, 3, 2 * MT>(
                    [&](int c) {
                        Opnd<2 * MT> o;
                        const int cc = 8 * (c >> 1) + 2 * (c & 1);   // tcol(2c, hf) - 4hf
#pragma unroll
                        for (int n = 0; n < MT; n++) {
                            o.v[2 * n] = yb[32 * n * LY + cc];
                            o.v[2 * n + 1] = yb[32 * n * LY + cc + 1];
                        }
                        return o;
                    },
                    [&](int c, const Opnd<2 * MT>& o) {
#pragma unroll
                        for (int j = 0; j < 2; j++) {
                            const float av = z3o[2 * c + j];
#pragma unroll
                            for (int n = 0; n < MT; n++)
                                accUt[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, o.v[2 * n + j], accUt[n], 0, 0, 0);
                        }
                    },
                    side_c);
            }
        } else {
#pragma unroll
            for (int c = 0; c < 8; c++) side_c(c);
        }
        // dZ2[h]: transposed conv along w (tap j reads column - j + 1)
        f32x16 dz2;
        {
            const f32x16 gp = tshift<1>(dz3, hm);
            const f32x16 gm = tshift<-1>(dz3, hm);
#pragma unroll
            for (int i = 0; i < 16; i++) dz2[i] = kw[0] * gp[i] + kw[1] * dz3[i] + kw[2] * gm[i];
        }
        dr[KH - 1] = dz2;
        if constexpr (rin) {   // dKh products
            const f32x16 g = own_cols(dz2);
            float t[KH];
#pragma unroll
            for (int j = 0; j < KH; j++) t[j] = 0.f;
#pragma unroll
            for (int i = 0; i < 16; i++)
#pragma unroll
                for (int j = 0; j < KH; j++) t[j] += ring[j][i] * g[i];
#pragma unroll
            for (int j = 0; j < KH; j++) tk[j] += t[j];
        }
        // dZ1 for row h - CH
        f32x16 dz1;
#pragma unroll
        for (int i = 0; i < 16; i++) {
            float a = 0.f;
#pragma unroll
            for (int j = 0; j < KH; j++) a += kh[j] * dr[KH - 1 - j][i];
            dz1[i] = a;
        }
#pragma unroll
        for (int j = 0; j < KH - 1; j++) {
            ring[j] = ring[j + 1];
            dr[j] = dr[j + 1];
        }
        if constexpr (xin) {
            // dX[hx] = Us^T dZ1[hx]: dZ1 through the LDS tile Tz[col][r], which
            // may share the dY tile: every read of that precedes these writes
            asm volatile("" ::: "memory");
#pragma unroll
            for (int i = 0; i < 16; i++) Tz[tcol(i, hf) * LZ + cl] = dz1[i];
            f32x16 (&accX)[MS] = accXp;   // stored along the next row's first chain
#pragma unroll
            for (int n = 0; n < MS; n++)
#pragma unroll
                for (int i = 0; i < 16; i++) accX[n][i] = 0.f;
            // dUs += dZ1[hx] X[hx]^T, X row hx from its ring slot (channel 32n + cl)
            const f32x16 dz1o = own_cols(dz1);
            const T* xrow = Xl + (k % 3) * NS * LX + cl * LX;
            if constexpr (BF) {
#pragma unroll
                for (int q = 0; q < 2; q++) {
                    float zf[8];
#pragma unroll
                    for (int j = 0; j < 8; j++) zf[j] = Tz[cl * LZ + 16 * q + 8 * hf + j];
                    const bf16x8 bv = cvt8(zf);
#pragma unroll
                    for (int n = 0; n < MS; n++)
                        accX[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds8(UsT + (32 * n + cl) * LDU + 16 * q + 8 * hf),
                                                                          bv, accX[n], 0, 0, 0);
                }
#pragma unroll
                for (int q = 0; q < 2; q++) {
                    float zf[8];
#pragma unroll
                    for (int j = 0; j < 8; j++) zf[j] = dz1o[8 * q + j];
                    const bf16x8 av = cvt8(zf);
#pragma unroll
                    for (int n = 0; n < MS; n++) {
                        // columns tcol(8q + j, hf): 16q + 4hf + {0..3} and 16q + 8 + 4hf + {0..3}
                        const bf16_t* xr = xrow + (32 * n) * LX + 16 * q + 4 * hf;
                        bf16_t bv[8];
                        __builtin_memcpy(bv, xr, 8);
                        __builtin_memcpy(bv + 4, xr + 8, 8);
                        accUs[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pack8(bv), accUs[n], 0, 0, 0);
                    }
                }
            } else {
                // One pipeline: chunks 0-3 the dUs product (columns tcol(i, hf) =
                // 8(i/4) + 4hf + i%4: one aligned run of four a chunk and channel
                // block), chunks 4-11 the dX product (ranks 2u + hf, two u a chunk),
                // whose reads of the dZ1 tile are in flight while dUs runs.
                constexpr int NO = 4 * MS > 2 * MS + 2 ? 4 * MS : 2 * MS + 2;
                const float* tzr = Tz + cl * LZ + hf;
                const float* usr = UsA + hf * LDA_S + cl;
                piped<12, 3, NO>(
                    [&](int c) {
                        Opnd<NO> o;
                        if (c < 4) {
#pragma unroll
                            for (int n = 0; n < MS; n++) {
                                const float4 t = *reinterpret_cast<const float4*>(xrow + (32 * n) * LX + 8 * c + 4 * hf);
                                o.v[4 * n] = t.x;
                                o.v[4 * n + 1] = t.y;
                                o.v[4 * n + 2] = t.z;
                                o.v[4 * n + 3] = t.w;
                            }
                        } else {
                            const int u = 2 * (c - 4);
#pragma unroll
                            for (int j = 0; j < 2; j++) {
#pragma unroll
                                for (int n = 0; n < MS; n++) o.v[j * MS + n] = usr[2 * (u + j) * LDA_S + 32 * n];
                                o.v[2 * MS + j] = tzr[2 * (u + j)];
                            }
                        }
                        return o;
                    },
                    [&](int c, const Opnd<NO>& o) {
                        if (c < 4) {
#pragma unroll
                            for (int j = 0; j < 4; j++) {
                                const float av = dz1o[4 * c + j];
#pragma unroll
                                for (int n = 0; n < MS; n++)
                                    accUs[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, o.v[4 * n + j], accUs[n], 0, 0, 0);
                            }
                        } else {
#pragma unroll
                            for (int j = 0; j < 2; j++)
#pragma unroll
                                for (int n = 0; n < MS; n++)
                                    accX[n] = __builtin_amdgcn_mfma_f32_32x32x2f32(o.v[j * MS + n], o.v[2 * MS + j],
                                                                                   accX[n], 0, 0, 0);
                        }
                    },
                    side_d);
            }
            if constexpr (BF) {
#pragma unroll
                for (int c = 0; c < 12; c++) side_d(c);
            }
            mfma_drain();   // accX is read by the stores
        } else {
#pragma unroll
            for (int c = 0; c < 12; c++) side_d(c);
        }
    };
    // Rows hs = h0 - 1 (halo), h0 (no dX row yet), h0 + 1 .. h1 - 1 and h1
    // (halo).  The first full row runs outside the loop: the loop is then
    // entered, like its back edge, with a dX row pending and the same memory
    // operations outstanding, so the wait counts the compiler derives for the
    // prefetched operands at the loop head are those of the steady state.
    static_assert(CH == 1, "one halo row on each side");
    const std::true_type yes;
    const std::false_type no;
    if (wok) {
        row_step(hs, no, no, yes, no);
        row_step(h0, yes, no, yes, no);
        if (h0 + 1 < h1) {
            row_step(h0 + 1, yes, yes, yes, no);
            for (int h = h0 + 2; h < h1; h++) row_step(h, yes, yes, yes, yes);
            row_step(h1, no, yes, no, yes);
        } else {
            row_step(h1, no, yes, no, no);
        }
        // the dX row of the last row
        const uint32_t v0 = dx0 + (uint32_t)((h1 - CH) * W) * E, v1 = v0 + xcs;
#pragma unroll
        for (int n = 0; n < MS; n++)
#pragma unroll
            for (int i = 0; i < 16; i++) {
                const int ch = 32 * n + row32(i, 0);
                bstore(accXp[n][i], (T*)nullptr, rD, (ch & 1) ? v1 : v0, (uint32_t)(2 * (ch >> 1)) * xcs);
            }
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
    // partials [R][T] and [R][S] a block: ranks past R and padded channels
    // are zero and not written
    // (whole-block shapes: R = 32, T = NT, S = NS, the same layout with no checks)
    const int RR = GEN ? d.R : 32, TR = GEN ? d.T : NT, SR = GEN ? d.S : NS;
    for (int e = tid; e < RR * NT; e += 256) {
        const int r = e / NT, t = e - r * NT;
        if (!GEN || t < TR)
            Put[blk * RR * TR + r * TR + t] = ((red[e] + red[32 * NT + e]) + red[64 * NT + e]) + red[96 * NT + e];
    }
    __syncthreads();
#pragma unroll
    for (int n = 0; n < MS; n++)
#pragma unroll
        for (int i = 0; i < 16; i++) red[wave * 32 * NS + row32(i, lane) * NS + 32 * n + cl] = accUs[n][i];
    __syncthreads();
    for (int e = tid; e < RR * NS; e += 256) {
        const int r = e / NS, s = e - r * NS;
        if (!GEN || s < SR)
            Pus[blk * RR * SR + r * SR + s] = ((red[e] + red[32 * NS + e]) + red[64 * NS + e]) + red[96 * NS + e];
    }
    __syncthreads();
    // taps: red[wave][half][r][KH + KW], summed over waves and halves in order
    constexpr int NJ = KH + KW;
#pragma unroll
    for (int j = 0; j < KW; j++) red[((wave * 2 + hf) * 32 + cl) * NJ + j] = tw[j];
#pragma unroll
    for (int j = 0; j < KH; j++) red[((wave * 2 + hf) * 32 + cl) * NJ + KW + j] = tk[j];
    __syncthreads();
    for (int e = tid; e < 32 * NJ; e += 256) {
        const int r = e / NJ, jj = e - r * NJ;
        float v = 0.f;
#pragma unroll
        for (int q = 0; q < 8; q++) v += red[q * 32 * NJ + e];
        if (GEN && r >= RR) continue;
        if (jj < KW) Pkw[blk * RR * KW + r * KW + jj] = v;
        else Pkh[blk * RR * KH + r * KH + (jj - KW)] = v;
    }
}

constexpr uint32_t kMaxLds = 160 * 1024;   // LDS of one gfx950 CU

template <typename T, int K, int M>
hipError_t launch_cpb_t(const CpBwdDesc& d, const void* const* o, hipStream_t s) {
    const bool gen = !(d.R == 32 && d.S == 32 * M && d.T == 32 * M);
    auto k = gen ? cp_bwd<T, K, K, M, M, true> : cp_bwd<T, K, K, M, M, false>;
    // the kernel's compile-time LDS pitches must be the descriptor's
    if (d.lda_s != cp_bwd_pitch_s<T, 32 * M>() || d.lda_t != cp_bwd_pitch_s<T, 32 * M>() || d.ly != cp_bwd_pitch_y<T>() ||
        d.lx != cp_bwd_pitch_x<T>() || (sizeof(T) == 2 && d.ldu != cp_bwd_pitch_u<T>()))
        return hipErrorInvalidValue;
    // dynamic LDS above 64 KB has to be allowed per kernel, once per device
    static std::atomic<uint64_t> allowed[2];   // per kernel (gen), a bit per device
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64 || d.lds_bytes > kMaxLds) return hipErrorInvalidValue;
    if (!(allowed[gen].load() & (1ull << dev))) {
        e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kMaxLds);
        if (e != hipSuccess) return e;
        allowed[gen].fetch_or(1ull << dev);
    }
    hipLaunchKernelGGL(k, dim3((uint32_t)d.blocks), dim3(256), d.lds_bytes, s, d, (const T*)o[0],
                       (const T*)o[1], (const T*)o[3], (const T*)o[4], (const T*)o[5], (const T*)o[6],
                       (T*)o[2], (float*)o[7], (float*)o[8], (float*)o[9], (float*)o[10]);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_cpb_ty(const CpBwdDesc& d, const void* const* o, hipStream_t s) {
    const int m = (d.T + 31) / 32;
    if (d.KH == 3) return m == 1 ? launch_cpb_t<T, 3, 1>(d, o, s) : launch_cpb_t<T, 3, 2>(d, o, s);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_cp_fwd(const Launch& ln, const void* const* ops, void* y, hipStream_t s) {
    CpDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (d.R < 1 || d.R > 32 || d.T < 1 || d.T > 64) return hipErrorInvalidValue;
    int bf = (ln.kind >> kBitIn) & 1;
    return bf ? launch_cp_ty<bf16_t>(d, ops, y, s) : launch_cp_ty<float>(d, ops, y, s);
}

// ops = {X, dY, dX (may be NULL), Us, Kh, Kw, Ut, Pus, Put, Pkh, Pkw}
hipError_t launch_cp_bwd(const Launch& ln, const void* const* ops, hipStream_t s) {
    CpBwdDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    if (d.R < 1 || d.R > 32 || d.S < 1 || d.T < 1 || d.T > 64 || (d.S + 31) / 32 != (d.T + 31) / 32 ||
        d.KH != d.KW)
        return hipErrorInvalidValue;
    int bf = (ln.kind >> kBitIn) & 1;
    return bf ? launch_cpb_ty<bf16_t>(d, ops, s) : launch_cpb_ty<float>(d, ops, s);
}

}  // namespace ce
