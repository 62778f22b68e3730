// Per-thread phases of the fused reshaped-CP chain forward (RcpDesc).
//
// Shared by the gfx950 kernel (kernels_rcp.hip) and the host-side checker
// that runs the same index arithmetic with every LDS and global access
// bounds-checked.  The includer defines RCP_FN (qualifiers of the phases)
// and RCP_HD (of the size helpers, also called by host code) and supplies
// the memory/arithmetic policy M:
//   ld16(p, i), ldw(p, i) (two bf16 at even i as one word), st16(p, i, v);
//   lr(i), lr4(i, out[4]) (i % 4 == 0), lw(i, v), lw16(i, half, v) on LDS words;
//   dot2(a, b, c) = a.lo*b.lo + a.hi*b.hi + c on bf16 pairs (fp32 result);
//   pk(lo, hi) two floats -> a bf16 pair (round to nearest even); bf(f).
//
// Arithmetic: bf16 operands, fp32 accumulation; every intermediate of the
// chain (Z1, Z2, Z3) is rounded to bf16 before its next contraction, as the
// unfused steps store them.
//
// Work of one workgroup (sample b, mode index t1, row tile, t2 chunk), per
// rank r:
//   phase A: Z2[t2][s3][p] for its t2 chunk on the tile's computed rows, from
//            the X values the thread keeps in registers (contract s1 then s2,
//            per pixel);
//   phase B: Z3[t2][t3][p] (contract s3) into the rank's half of the Zc words;
//   phase C: once per rank pair, Y[t2][t3][p] += sum over the two ranks and the
//            K x K taps of W0 * Z3 at the shifted positions (zero border).
#pragma once

#include <cstdint>

#include "desc_rcp.h"

namespace ce {
namespace rcp {

template <int S1_, int S2_, int S3_, int T2_, int T3_, int K_, int T2C_, int NT_, int UA_, int UB_, int UC_>
struct Cfg {
    static constexpr int S1 = S1_, S2 = S2_, S3 = S3_, T2 = T2_, T3 = T3_, K = K_, T2C = T2C_;
    static constexpr int NT = NT_;    // threads per workgroup
    static constexpr int UA = UA_;    // phase-A units per thread (pixel, s3 pair)
    static constexpr int UB = UB_;    // phase-B units per thread (pixel, t2)
    static constexpr int UC = UC_;    // phase-C units per thread (plane, row, 4 columns)
    static constexpr int S1P = S1 / 2, S2P = S2 / 2, S3P = S3 / 2;
    static constexpr int KK = K * K, C0 = (K - 1) / 2;
    static_assert(S1 % 2 == 0 && S2 % 2 == 0 && S3 % 2 == 0, "contracted modes come in pairs");
    static_assert(T2 % T2C == 0 && K % 2 == 1 && K <= 5, "shape");
};

// Rows of one tile: output rows [h0, h1), computed rows [ha, hb) (the output
// rows and up to (K-1)/2 halo rows on each side, clipped to the image).
struct Tile {
    int h0, h1, ha, hb;
};
RCP_HD Tile tile_rows(const RcpDesc& d, int tile) {
    Tile t;
    const int c0 = (d.K - 1) / 2;
    t.h0 = tile * d.TH;
    t.h1 = t.h0 + d.TH < d.H ? t.h0 + d.TH : d.H;
    t.ha = t.h0 - c0 > 0 ? t.h0 - c0 : 0;
    t.hb = t.h1 + c0 < d.H ? t.h1 + c0 : d.H;
    return t;
}

// Unit counts of one tile.
RCP_HD int units_a(const RcpDesc& d, const Tile& t) { return (t.hb - t.ha) * d.W * (d.S3 / 2); }
RCP_HD int units_b(const RcpDesc& d, const Tile& t) { return (t.hb - t.ha) * d.W * d.T2C; }
RCP_HD int units_c(const RcpDesc& d, const Tile& t) { return d.T2C * d.T3 * (t.h1 - t.h0) * d.QW; }

// The LDS layout invariants every access of the phases relies on: a Zb
// buffer holds T2C * S3/2 words per computed pixel of any tile, a Zc plane
// has rows 0 .. TH+K-2 and columns up to 4*QW + 3 (the last window of phase
// C), both regions 16-byte aligned; the tiles cover the image.
RCP_HD bool layout_ok(const RcpDesc& d) {
    if (d.H <= 0 || d.W <= 0 || d.K % 2 != 1 || d.TH <= 0 || d.ntiles != (d.H + d.TH - 1) / d.TH)
        return false;
    int rows = 0;   // most computed rows of a tile
    for (int i = 0; i < d.ntiles; i++) {
        const Tile t = tile_rows(d, i);
        rows = t.hb - t.ha > rows ? t.hb - t.ha : rows;
    }
    return d.QW == (d.W + 3) / 4 && d.WP % 4 == 0 && d.WP >= 4 * d.QW + 4 && d.HP >= d.TH + d.K - 1 &&
           d.plane_dw == d.HP * d.WP && d.zb_dw % 4 == 0 && d.zb_dw >= d.T2C * (d.S3 / 2) * rows * d.W &&
           d.zc_dw == d.T2C * d.T3 * d.plane_dw && d.T2C > 0 && d.T2 == d.nc * d.T2C &&
           (int64_t)d.lds_bytes >= 4 * ((int64_t)2 * d.zb_dw + d.zc_dw) && d.R >= 2 && d.R % 2 == 0;
}

// Block -> (b, t1, row tile, t2 chunk).  With a multiple of 8 blocks, the
// blocks of one sample (consecutive logical ids) land on one XCD: hardware
// block i runs on XCD i % 8.
RCP_HD void block_coords(const RcpDesc& d, int64_t bid, int& b, int& t1, int& tile, int& chunk) {
    int64_t l = bid;
    if (d.blocks % 8 == 0) l = (bid % 8) * (d.blocks / 8) + bid / 8;
    chunk = (int)(l % d.nc);
    l /= d.nc;
    tile = (int)(l % d.ntiles);
    l /= d.ntiles;
    t1 = (int)(l % d.T1);
    b = (int)(l / d.T1);
}

template <class C>
struct State {
    uint32_t xp[C::UA][C::S1P][C::S2][2];   // X pairs along s1 at s3 = 2*s3p + e
    float acc[C::UC][4];                    // Y of the phase-C units
    int a_zb[C::UA];                        // Zb word of (t2 = 0, s3p, pixel), -1: no unit
    int b_zb[C::UB], b_zc[C::UB];           // Zb word of (t2, 0, pixel); Zc word of (t2, t3 = 0, pixel); -1: none
    int c_row[C::UC];                       // Zc word of the unit's first window row, -1: none
};

// Unit coordinates, X values, zero accumulators and the zero Zc planes.
// Computed pixel n of the tile is (ha + n / W, n % W); Zc row of image row h
// is h - h0 + (K-1)/2.
template <class C, class M>
RCP_FN void init(M& m, const RcpDesc& d, int tid, int b, const Tile& t, const uint16_t* X, State<C>& st) {
    const int HW = d.H * d.W, W = d.W, NP = (t.hb - t.ha) * W;
    const int nA = units_a(d, t), nB = units_b(d, t), nC = units_c(d, t);
    const int zc0 = 2 * d.zb_dw;
    const int64_t xb = (int64_t)b * (C::S1 * C::S2 * C::S3) * HW + (int64_t)t.ha * W;
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        const int u = tid + k * C::NT;
        st.a_zb[k] = -1;
        if (u < nA) {
            const int n = u % NP, s3p = u / NP;
            st.a_zb[k] = s3p * NP + n;
#pragma unroll
            for (int j = 0; j < C::S1P; j++)
#pragma unroll
                for (int s2 = 0; s2 < C::S2; s2++)
#pragma unroll
                    for (int e = 0; e < 2; e++) {
                        const int s3 = 2 * s3p + e;
                        const int64_t o0 = xb + ((int64_t)((2 * j) * C::S2 + s2) * C::S3 + s3) * HW + n;
                        const int64_t o1 = o0 + (int64_t)C::S2 * C::S3 * HW;
                        st.xp[k][j][s2][e] = (uint32_t)m.ld16(X, o0) | ((uint32_t)m.ld16(X, o1) << 16);
                    }
        } else {
#pragma unroll
            for (int j = 0; j < C::S1P; j++)
#pragma unroll
                for (int s2 = 0; s2 < C::S2; s2++) st.xp[k][j][s2][0] = st.xp[k][j][s2][1] = 0;
        }
    }
#pragma unroll
    for (int k = 0; k < C::UB; k++) {
        const int v = tid + k * C::NT;
        st.b_zb[k] = st.b_zc[k] = -1;
        if (v < nB) {
            const int n = v % NP, t2 = v / NP;
            const int h = t.ha + n / W, w = n % W;
            st.b_zb[k] = t2 * C::S3P * NP + n;
            st.b_zc[k] = zc0 + t2 * C::T3 * d.plane_dw + (h - t.h0 + C::C0) * d.WP + w + C::C0;
        }
    }
    const int TR = t.h1 - t.h0;
#pragma unroll
    for (int k = 0; k < C::UC; k++) {
        const int c = tid + k * C::NT;
        st.c_row[k] = -1;
        if (c < nC) {
            const int q = c % d.QW, hl = (c / d.QW) % TR, plane = c / (d.QW * TR);
            st.c_row[k] = zc0 + plane * d.plane_dw + hl * d.WP + 4 * q;
        }
#pragma unroll
        for (int o = 0; o < 4; o++) st.acc[k][o] = 0.f;
    }
    for (int i = tid; i < d.zc_dw; i += C::NT) m.lw(zc0 + i, 0u);
}

// Phase A of rank r into Zb buffer `buf`: per unit (pixel p, s3 pair) and
// e = 0, 1: Z1[s2] = sum_s1 W1[r][t1][s1] X[s1][s2][2 s3p + e][p] (bf16),
// Z2[t2] = sum_s2 W2[r][t2][s2] Z1[s2]; the two s3 values of each t2 form one word.
template <class C, class M>
RCP_FN void phase_a(M& m, const RcpDesc& d, const Tile& t, int r, int t1, int chunk, int buf,
                    const uint16_t* W1, const uint16_t* W2, const State<C>& st) {
    uint32_t w1[C::S1P], w2[C::T2C][C::S2P];
    const int64_t o1 = ((int64_t)r * d.T1 + t1) * C::S1;
#pragma unroll
    for (int j = 0; j < C::S1P; j++) w1[j] = m.ldw(W1, o1 + 2 * j);
#pragma unroll
    for (int t = 0; t < C::T2C; t++) {
        const int64_t o2 = ((int64_t)r * C::T2 + chunk * C::T2C + t) * C::S2;
#pragma unroll
        for (int i = 0; i < C::S2P; i++) w2[t][i] = m.ldw(W2, o2 + 2 * i);
    }
    const int NP = (t.hb - t.ha) * d.W, zb = buf * d.zb_dw;
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        if (st.a_zb[k] < 0) continue;
        float z2[2][C::T2C];
#pragma unroll
        for (int e = 0; e < 2; e++) {
            uint32_t z1p[C::S2P];
#pragma unroll
            for (int i = 0; i < C::S2P; i++) {
                float a0 = 0.f, a1 = 0.f;
#pragma unroll
                for (int j = 0; j < C::S1P; j++) {
                    a0 = m.dot2(w1[j], st.xp[k][j][2 * i][e], a0);
                    a1 = m.dot2(w1[j], st.xp[k][j][2 * i + 1][e], a1);
                }
                z1p[i] = m.pk(a0, a1);
            }
#pragma unroll
            for (int t = 0; t < C::T2C; t++) {
                float a = 0.f;
#pragma unroll
                for (int i = 0; i < C::S2P; i++) a = m.dot2(w2[t][i], z1p[i], a);
                z2[e][t] = a;
            }
        }
#pragma unroll
        for (int t = 0; t < C::T2C; t++) m.lw(zb + t * C::S3P * NP + st.a_zb[k], m.pk(z2[0][t], z2[1][t]));
    }
}

// Phase B of rank r from Zb buffer `buf`: Z3[t2][t3][p] = sum_s3 W3[r][t3][s3] Z2[t2][s3][p],
// stored (bf16) in half r & 1 of the Zc word of (t2, t3) at the padded position of p.
template <class C, class M>
RCP_FN void phase_b(M& m, const RcpDesc& d, const Tile& tl, int r, int buf, const uint16_t* W3,
                    const State<C>& st) {
    uint32_t w3[C::T3][C::S3P];
#pragma unroll
    for (int t = 0; t < C::T3; t++)
#pragma unroll
        for (int i = 0; i < C::S3P; i++) w3[t][i] = m.ldw(W3, ((int64_t)r * C::T3 + t) * C::S3 + 2 * i);
    const int NP = (tl.hb - tl.ha) * d.W, zb = buf * d.zb_dw, half = r & 1;
#pragma unroll
    for (int k = 0; k < C::UB; k++) {
        if (st.b_zb[k] < 0) continue;
        uint32_t z[C::S3P];
#pragma unroll
        for (int i = 0; i < C::S3P; i++) z[i] = m.lr(zb + st.b_zb[k] + i * NP);
#pragma unroll
        for (int t = 0; t < C::T3; t++) {
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < C::S3P; i++) a = m.dot2(w3[t][i], z[i], a);
            m.lw16(st.b_zc[k] + t * d.plane_dw, half, m.bf(a));
        }
    }
}

// Phase C of the rank pair (r0, r0 + 1): Y[plane][h][4q + o] +=
// sum_{i,j} (W0[r0][i][j], W0[r0+1][i][j]) . Zc[plane][h + i][4q + o + j].
template <class C, class M>
RCP_FN void phase_c(M& m, const RcpDesc& d, int r0, const uint16_t* W0, State<C>& st) {
    uint32_t w0[C::KK];
#pragma unroll
    for (int t = 0; t < C::KK; t++)
        w0[t] = (uint32_t)m.ld16(W0, (int64_t)r0 * C::KK + t) |
                ((uint32_t)m.ld16(W0, (int64_t)(r0 + 1) * C::KK + t) << 16);
#pragma unroll
    for (int k = 0; k < C::UC; k++) {
        if (st.c_row[k] < 0) continue;
#pragma unroll
        for (int i = 0; i < C::K; i++) {
            uint32_t win[8];
            const int row = st.c_row[k] + i * d.WP;
            m.lr4(row, win);
            m.lr4(row + 4, win + 4);
#pragma unroll
            for (int o = 0; o < 4; o++)
#pragma unroll
                for (int j = 0; j < C::K; j++) st.acc[k][o] = m.dot2(w0[i * C::K + j], win[o + j], st.acc[k][o]);
        }
    }
}

// Y (bf16) of the phase-C units; columns past W are not stored.
template <class C, class M>
RCP_FN void store(M& m, const RcpDesc& d, int tid, int b, int t1, const Tile& t, int chunk, uint16_t* Y,
                  const State<C>& st) {
    const int HW = d.H * d.W, nC = units_c(d, t), TR = t.h1 - t.h0;
#pragma unroll
    for (int k = 0; k < C::UC; k++) {
        const int c = tid + k * C::NT;
        if (c >= nC) continue;
        const int q = c % d.QW, h = t.h0 + (c / d.QW) % TR, plane = c / (d.QW * TR);
        const int t2 = chunk * C::T2C + plane / C::T3, t3 = plane % C::T3;
        const int64_t base = ((((int64_t)b * d.T1 + t1) * C::T2 + t2) * C::T3 + t3) * HW + (int64_t)h * d.W;
#pragma unroll
        for (int o = 0; o < 4; o++)
            if (4 * q + o < d.W) m.st16(Y, base + 4 * q + o, m.bf(st.acc[k][o]));
    }
}

}  // namespace rcp
}  // namespace ce
