// Per-thread phases of the fused reshaped-CP chain backward (RcpBwdDesc).
//
// The gradient of each pairwise step of the RCP chain (Appendix B: g1 of a
// step is the output gradient contracted with the other operand, g2 the
// output gradient contracted with the step's input), for one rank r at a time:
//   G3[t][p] = sum_{ij} W0[r][i][j] dY[t][p - (i,j) + c]       (step 3, g1: transposed conv)
//   dW0[r][i][j] = sum_{b,t,p} Z3[t][p] dY[t][p - (i,j) + c]   (step 3, g2)
//   G2[t1 t2 s3] = sum_t3 W3[r][t3][s3] G3[t1 t2 t3]            (step 2, g1)
//   dW3[r][t3][s3] = sum G3[t1 t2 t3][p] Z2[t1 t2 s3][p]        (step 2, g2)
//   G1[t1 s2 s3] = sum_t2 W2[r][t2][s2] G2[t1 t2 s3]            (step 1, g1)
//   dW2[r][t2][s2] = sum G2[t1 t2 s3][p] Z1[t1 s2 s3][p]        (step 1, g2)
//   dX[s1 s2 s3] += sum_t1 W1[r][t1][s1] G1[t1 s2 s3]           (step 0, g1)
//   dW1[r][t1][s1] = sum G1[t1 s2 s3][p] X[s1 s2 s3][p]         (step 0, g2)
// with Z1, Z2, Z3 recomputed from X (checkpointing).  Every intermediate and
// intermediate gradient is rounded to bf16 before it is used, as the unfused
// steps store them; sums are fp32.
//
// One workgroup owns sample b, mode index t1, a tile of TH rows and a chunk
// of T2C values of t2, and loops over the rank.  Its dX is a partial sum
// (over its t1 and t2 chunk) and its factor gradients are partial sums over
// its pixels; both go to fp32 partial buffers that ordered reductions sum.
//
// Phases of rank r (barriers in between):
//   A  unit (pixel n, s3): Z1[s2] (-> Z1k), Z2[t2] (-> Z2k) from the thread's X
//   B  unit (n, t2): Z3[t3] (-> Z3k)
//   C  unit (plane (t2,t3), row, 4 columns): G3 (-> G3k) and the dW0 partial
//      from a window of the dY plane (kept in LDS with a zero border)
//   D  unit (n, t2): G2[s3] (-> G2k); per wave, dW3 on MFMA from G3k and Z2k
//   E  unit (n, s3): G1[s2], dX accumulation, the dW1 partial; per wave, dW2
//      on MFMA from G2k and Z1k
//   F  (with A of the next rank): ordered sums of the per-row and per-wave
//      partials, written to the workgroup's partial slots
// Z1k, Z2k, G3k, G2k are k-contiguous bf16 rows (the MFMA operands) over a
// pixel range padded to PP (multiple of 16) with zeros.
#pragma once

#include <cstdint>

#include "desc_rcp.h"

namespace ce {
namespace rcpb {

template <int S1_, int S2_, int S3_, int T2_, int T3_, int K_, int T2C_, int NT_, int UA_, int UB_, int UC_, int MW_>
struct Cfg {
    static constexpr int MW = MW_;   // waves per SIMD of the launch bound
    static constexpr int S1 = S1_, S2 = S2_, S3 = S3_, T2 = T2_, T3 = T3_, K = K_, T2C = T2C_;
    static constexpr int NT = NT_, NW = NT_ / 64;
    static constexpr int UA = UA_;   // units (n, s3) per thread: phases A, E
    static constexpr int UB = UB_;   // units (n, t2) per thread: phases B, D
    static constexpr int UC = UC_;   // units (plane, row, 4 columns) per thread: phase C
    static constexpr int S1P = S1 / 2, S2P = S2 / 2, S3P = S3 / 2, T3P = T3 / 2;
    static constexpr int KK = K * K, C0 = (K - 1) / 2;
    static constexpr int NV = KK + S1;   // per-thread partial values (dW0 taps, dW1)
    static_assert(S1 % 2 == 0 && S2 % 2 == 0 && S3 % 2 == 0 && T3 % 2 == 0, "pairs");
    static_assert(NT % 64 == 0 && T3 <= 32 && S3 <= 32 && T2C <= 32 && S2 <= 32, "shape");
};

// Rows of tile i: [h0, h1).
RCPB_HD void tile_of(const RcpBwdDesc& d, int i, int& h0, int& h1) {
    h0 = i * d.TH;
    h1 = h0 + d.TH < d.H ? h0 + d.TH : d.H;
}

// The LDS layout invariants every access relies on.
RCPB_HD bool layout_ok_b(const RcpBwdDesc& d) {
    const int P = d.TH * d.W, S3 = d.S3, T3 = d.T3, T2C = d.T2C;
    const int64_t e_z1 = (int64_t)d.S2 * d.L13, e_z2 = (int64_t)S3 * d.L2, e_z3 = (int64_t)T2C * T3 * P,
                  e_g3 = (int64_t)T3 * d.L2, e_g2 = (int64_t)T2C * d.L13;
    const int64_t w_dy = (int64_t)T2C * T3 * d.HPb * d.WP;
    const int nv = d.K * d.K + d.S1, nw = d.NT / 64;
    return d.H > 0 && d.W > 0 && d.K % 2 == 1 && d.TH > 0 && d.ntiles == (d.H + d.TH - 1) / d.TH &&
           d.QW == (d.W + 3) / 4 && d.WP % 4 == 0 && d.WP >= 4 * d.QW + 4 && d.HPb == d.TH + d.K - 1 &&
           d.PP % 16 == 0 && d.PP >= P && d.T2 == d.nc * T2C && d.R >= 1 && d.NT % 64 == 0 &&
           d.L13 == S3 * d.PP + 8 && d.L2 == T2C * d.PP + 8 &&
           d.tbs == d.K * d.K + S3 * (T3 / 2) + d.T1 * d.S1 + d.S2 * (d.T2 / 2) &&
           d.o_dy == 0 && d.o_z1 >= d.o_dy + w_dy && d.o_z1 % 4 == 0 && d.o_z2 >= d.o_z1 + e_z1 / 2 &&
           d.o_z2 % 4 == 0 && d.o_z3 >= d.o_z2 + e_z2 / 2 && d.o_z3 % 4 == 0 &&
           d.o_g3 >= d.o_z3 + (e_z3 + 1) / 2 && d.o_g3 % 4 == 0 && d.o_g2 >= d.o_g3 + e_g3 / 2 && d.o_g2 % 4 == 0 &&
           d.o_q >= d.o_g2 + e_g2 / 2 && d.o_m3 >= d.o_q + (int64_t)nv * 4 * nw &&
           d.o_m2 >= d.o_m3 + (int64_t)nw * T3 * S3 &&
           (int64_t)d.lds_bytes >= 4 * ((int64_t)d.o_m2 + (int64_t)nw * T2C * d.S2);}

// Block -> (b, t1, tile, chunk), the forward's order (and XCD grouping).
RCPB_HD void block_coords_b(const RcpBwdDesc& d, int64_t bid, int64_t& l, int& b, int& t1, int& tile, int& chunk) {
    l = bid;
    if (d.blocks % 8 == 0) l = (bid % 8) * (d.blocks / 8) + bid / 8;
    int64_t x = l;
    chunk = (int)(x % d.nc);
    x /= d.nc;
    tile = (int)(x % d.ntiles);
    x /= d.ntiles;
    t1 = (int)(x % d.T1);
    b = (int)(x / d.T1);
}

template <class C>
struct State {
    uint32_t xp[C::UA][C::S1P][C::S2];   // X pairs along s1 at the unit's (s3, n)
    float dxa[C::UA][C::S1][C::S2];      // dX of the unit (this workgroup's t1, t2 chunk)
    int a_n[C::UA], a_s3[C::UA];         // unit (n, s3); a_n = -1: no unit
    int b_n[C::UB], b_t2[C::UB];         // unit (n, t2l); b_n = -1: none
    int c_pl[C::UC], c_hl[C::UC], c_q[C::UC];   // unit (plane, row, quad); c_pl = -1: none
};

// bf16 element e of an LDS region that starts at word o.
template <class M>
RCPB_FN uint16_t lds_e(M& m, int o, int e) {
    return m.lr16(o + (e >> 1), e & 1);
}
template <class M>
RCPB_FN void lds_se(M& m, int o, int e, uint16_t v) {
    m.lw16(o + (e >> 1), e & 1, v);
}

// Element index of the k-contiguous rows: Z1k row s2 and G2k row t2l hold
// k = s3 * PP + n (pitch L13), Z2k row s3 and G3k row t3 hold k = t2l * PP + n
// (pitch L2); each pitch is 8 elements past the row so that consecutive
// rows start 16 bytes apart in the LDS banks.
RCPB_FN int iz1(const RcpBwdDesc& d, int s2, int s3, int n) { return s2 * d.L13 + s3 * d.PP + n; }
RCPB_FN int ig2(const RcpBwdDesc& d, int t2l, int s3, int n) { return t2l * d.L13 + s3 * d.PP + n; }
RCPB_FN int iz2(const RcpBwdDesc& d, int s3, int t2l, int n) { return s3 * d.L2 + t2l * d.PP + n; }
RCPB_FN int ig3(const RcpBwdDesc& d, int t3, int t2l, int n) { return t3 * d.L2 + t2l * d.PP + n; }

// Unit coordinates, X, zero dX, the dY planes (zero outside the image) and
// zero padding columns of the k-contiguous rows.
template <class C, class M>
RCPB_FN void init(M& m, const RcpBwdDesc& d, int tid, int b, int t1, int h0, int h1, int chunk,
                  const uint16_t* X, const uint16_t* dY, State<C>& st) {
    const int W = d.W, HW = d.H * d.W, P = (h1 - h0) * W, TR = h1 - h0;
    const int64_t xb = (int64_t)b * (C::S1 * C::S2 * C::S3) * HW + (int64_t)h0 * W;
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        const int u = tid + k * C::NT;
        st.a_n[k] = st.a_s3[k] = -1;
        if (u < P * C::S3) {
            const int n = u % P, s3 = u / P;
            st.a_n[k] = n;
            st.a_s3[k] = s3;
#pragma unroll
            for (int j = 0; j < C::S1P; j++)
#pragma unroll
                for (int s2 = 0; s2 < C::S2; s2++) {
                    const int64_t o0 = xb + ((int64_t)((2 * j) * C::S2 + s2) * C::S3 + s3) * HW + n;
                    const int64_t o1 = o0 + (int64_t)C::S2 * C::S3 * HW;
                    st.xp[k][j][s2] = (uint32_t)m.ld16(X, o0) | ((uint32_t)m.ld16(X, o1) << 16);
                }
        } else {
#pragma unroll
            for (int j = 0; j < C::S1P; j++)
#pragma unroll
                for (int s2 = 0; s2 < C::S2; s2++) st.xp[k][j][s2] = 0;
        }
#pragma unroll
        for (int s1 = 0; s1 < C::S1; s1++)
#pragma unroll
            for (int s2 = 0; s2 < C::S2; s2++) st.dxa[k][s1][s2] = 0.f;
    }
#pragma unroll
    for (int k = 0; k < C::UB; k++) {
        const int v = tid + k * C::NT;
        st.b_n[k] = st.b_t2[k] = -1;
        if (v < P * C::T2C) {
            st.b_n[k] = v % P;
            st.b_t2[k] = v / P;
        }
    }
#pragma unroll
    for (int k = 0; k < C::UC; k++) {
        const int c = tid + k * C::NT;
        st.c_pl[k] = st.c_hl[k] = st.c_q[k] = -1;
        if (c < C::T2C * C::T3 * TR * d.QW) {
            st.c_q[k] = c % d.QW;
            st.c_hl[k] = (c / d.QW) % TR;
            st.c_pl[k] = c / (d.QW * TR);
        }
    }
    // dY planes [t2l * T3 + t3][rho][kappa]: image row h0 - c0 + rho, column kappa - c0
    const int nplane = d.HPb * d.WP, ndy = C::T2C * C::T3 * nplane;
    for (int i = tid; i < ndy; i += C::NT) {
        const int pl = i / nplane, rho = (i / d.WP) % d.HPb, kap = i % d.WP;
        const int h = h0 - C::C0 + rho, w = kap - C::C0;
        float v = 0.f;
        if (h >= 0 && h < d.H && w >= 0 && w < W) {
            const int t2 = chunk * C::T2C + pl / C::T3, t3 = pl % C::T3;
            v = m.f(m.ld16(dY, ((((int64_t)b * d.T1 + t1) * C::T2 + t2) * C::T3 + t3) * HW + (int64_t)h * W + w));
        }
        m.lw(d.o_dy + i, m.fbits(v));
    }
    // zero padding of the k-contiguous rows (pixels P .. PP-1), never written later
    const int pad = d.PP - P;
    const int g1 = C::S2 * C::S3, g2 = C::S3 * C::T2C, g3 = C::T3 * C::T2C, g4 = C::T2C * C::S3;
    for (int i = tid; i < (g1 + g2 + g3 + g4) * pad; i += C::NT) {
        int row = i / pad;
        const int e = P + i % pad;
        if (row < g1) {
            lds_se(m, d.o_z1, iz1(d, row / C::S3, row % C::S3, e), 0);
        } else if ((row -= g1) < g2) {
            lds_se(m, d.o_z2, iz2(d, row / C::T2C, row % C::T2C, e), 0);
        } else if ((row -= g2) < g3) {
            lds_se(m, d.o_g3, ig3(d, row / C::T2C, row % C::T2C, e), 0);
        } else {
            row -= g3;
            lds_se(m, d.o_g2, ig2(d, row / C::S3, row % C::S3, e), 0);
        }
    }
}

// A: Z1[s2] at (n, s3) for t1 -> Z1k; Z2[t2l] -> Z2k.
template <class C, class M>
RCPB_FN void phase_a(M& m, const RcpBwdDesc& d, int r, int t1, int chunk, const uint16_t* W1,
                     const uint16_t* W2, const State<C>& st) {
    uint32_t w1[C::S1P], w2[C::T2C][C::S2P];
    const int64_t o1 = ((int64_t)r * d.T1 + t1) * C::S1;
#pragma unroll
    for (int j = 0; j < C::S1P; j++) w1[j] = m.ldw(W1, o1 + 2 * j);
#pragma unroll
    for (int t = 0; t < C::T2C; t++)
#pragma unroll
        for (int i = 0; i < C::S2P; i++)
            w2[t][i] = m.ldw(W2, ((int64_t)r * C::T2 + chunk * C::T2C + t) * C::S2 + 2 * i);
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        if (st.a_n[k] < 0) continue;
        const int n = st.a_n[k], s3 = st.a_s3[k];
        uint32_t z1p[C::S2P];
#pragma unroll
        for (int i = 0; i < C::S2P; i++) {
            float a0 = 0.f, a1 = 0.f;
#pragma unroll
            for (int j = 0; j < C::S1P; j++) {
                a0 = m.dot2(w1[j], st.xp[k][j][2 * i], a0);
                a1 = m.dot2(w1[j], st.xp[k][j][2 * i + 1], a1);
            }
            z1p[i] = m.pk(a0, a1);
            lds_se(m, d.o_z1, iz1(d, 2 * i, s3, n), (uint16_t)(z1p[i] & 0xffff));
            lds_se(m, d.o_z1, iz1(d, 2 * i + 1, s3, n), (uint16_t)(z1p[i] >> 16));
        }
#pragma unroll
        for (int t = 0; t < C::T2C; t++) {
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < C::S2P; i++) a = m.dot2(w2[t][i], z1p[i], a);
            lds_se(m, d.o_z2, iz2(d, s3, t, n), m.bf(a));
        }
    }
}

// B: Z3[t3] at (n, t2l) -> Z3k[(t2l T3 + t3) P + n].
template <class C, class M>
RCPB_FN void phase_b(M& m, const RcpBwdDesc& d, int r, int P, const uint16_t* W3, const State<C>& st) {
    uint32_t w3[C::T3][C::S3P];
#pragma unroll
    for (int t = 0; t < C::T3; t++)
#pragma unroll
        for (int i = 0; i < C::S3P; i++) w3[t][i] = m.ldw(W3, ((int64_t)r * C::T3 + t) * C::S3 + 2 * i);
#pragma unroll
    for (int k = 0; k < C::UB; k++) {
        if (st.b_n[k] < 0) continue;
        const int n = st.b_n[k], t2l = st.b_t2[k];
        uint32_t z[C::S3P];
#pragma unroll
        for (int i = 0; i < C::S3P; i++)
            z[i] = (uint32_t)lds_e(m, d.o_z2, iz2(d, 2 * i, t2l, n)) |
                   ((uint32_t)lds_e(m, d.o_z2, iz2(d, 2 * i + 1, t2l, n)) << 16);
#pragma unroll
        for (int t = 0; t < C::T3; t++) {
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < C::S3P; i++) a = m.dot2(w3[t][i], z[i], a);
            lds_se(m, d.o_z3, (t2l * C::T3 + t) * P + n, m.bf(a));
        }
    }
}

// C: per unit (plane, row hl, columns 4q..4q+3) the window of dY rows
// hl - i + 2c0 and columns 4q .. 4q+7 gives G3 (transposed conv) and the
// unit's dW0 terms; the thread's dW0 partials are summed over each 16-lane
// row of the wave into Q.
template <class C, class M>
RCPB_FN void phase_c(M& m, const RcpBwdDesc& d, int lane, int wave, int r, int P, const uint32_t* TB,
                     const State<C>& st) {
    float w0[C::KK], dw[C::KK];
#pragma unroll
    for (int t = 0; t < C::KK; t++) {
        w0[t] = m.fof(m.ldt(TB, (int64_t)r * d.tbs + t));
        dw[t] = 0.f;
    }
#pragma unroll
    for (int k = 0; k < C::UC; k++) {
        if (st.c_pl[k] < 0) continue;
        const int pl = st.c_pl[k], hl = st.c_hl[k], q = st.c_q[k];
        const int t2l = pl / C::T3, t3 = pl % C::T3;
        float z3[4], g[4];
#pragma unroll
        for (int o = 0; o < 4; o++) {
            z3[o] = 4 * q + o < d.W ? m.f(lds_e(m, d.o_z3, pl * P + hl * d.W + 4 * q + o)) : 0.f;
            g[o] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < C::K; i++) {
            uint32_t wr[8];
            const int row = d.o_dy + (pl * d.HPb + hl - i + 2 * C::C0) * d.WP + 4 * q;
            m.lr4(row, wr);
            m.lr4(row + 4, wr + 4);
            float win[8];
#pragma unroll
            for (int x = 0; x < 8; x++) win[x] = m.fof(wr[x]);
#pragma unroll
            for (int j = 0; j < C::K; j++)
#pragma unroll
                for (int o = 0; o < 4; o++) {
                    g[o] += w0[i * C::K + j] * win[o - j + 2 * C::C0];
                    dw[i * C::K + j] += z3[o] * win[o - j + 2 * C::C0];
                }
        }
#pragma unroll
        for (int o = 0; o < 4; o++)
            if (4 * q + o < d.W) lds_se(m, d.o_g3, ig3(d, t3, t2l, hl * d.W + 4 * q + o), m.bf(g[o]));
    }
    // sums over each 16-lane row of the wave: Q[tap][4 wave + row]
#pragma unroll
    for (int t = 0; t < C::KK; t++) m.rowsum(dw[t], lane, d.o_q + t * 4 * C::NW + 4 * wave + (lane >> 4));
}

// D: G2[s3] at (n, t2l) -> G2k.
template <class C, class M>
RCPB_FN void phase_d(M& m, const RcpBwdDesc& d, int r, const uint32_t* TB, const State<C>& st) {
    uint32_t w3t[C::S3][C::T3P];   // (W3[2i][s3], W3[2i+1][s3])
#pragma unroll
    for (int s = 0; s < C::S3; s++)
#pragma unroll
        for (int i = 0; i < C::T3P; i++) w3t[s][i] = m.ldt(TB, (int64_t)r * d.tbs + C::KK + s * C::T3P + i);
#pragma unroll
    for (int k = 0; k < C::UB; k++) {
        if (st.b_n[k] < 0) continue;
        const int n = st.b_n[k], t2l = st.b_t2[k];
        uint32_t g[C::T3P];
#pragma unroll
        for (int i = 0; i < C::T3P; i++)
            g[i] = (uint32_t)lds_e(m, d.o_g3, ig3(d, 2 * i, t2l, n)) |
                   ((uint32_t)lds_e(m, d.o_g3, ig3(d, 2 * i + 1, t2l, n)) << 16);
#pragma unroll
        for (int s = 0; s < C::S3; s++) {
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < C::T3P; i++) a = m.dot2(w3t[s][i], g[i], a);
            lds_se(m, d.o_g2, ig2(d, t2l, s, n), m.bf(a));
        }
    }
}

// One wave's share of a small reduction on 32x32x16 MFMA tiles:
// acc[m][n] += sum_k A[m][k] B[k][n] with A rows and B columns k-contiguous
// bf16 rows in LDS (row stride `ld` elements, K = nk * 16), m < Mv, n < Nv;
// the wave takes k-steps wave, wave + NW, ...  Lane l supplies
// A[l % 32][8 (l / 32) .. + 7] and B[same k][l % 32].
template <class C, class M>
RCPB_FN void mfma_part(M& m, int lane, int wave, int oA, int oB, int ld, int nk, int Mv, int Nv, float* acc) {
    const int mm = lane & 31, kh = 8 * (lane >> 5);
    for (int j = wave; j < nk; j += C::NW) {
        uint32_t a[4] = {0, 0, 0, 0}, b[4] = {0, 0, 0, 0};
        const int k0 = 16 * j + kh;
        if (mm < Mv) m.lr4(oA + ((mm * ld + k0) >> 1), a);
        if (mm < Nv) m.lr4(oB + ((mm * ld + k0) >> 1), b);
        m.mfma(a, b, acc);
    }
}

// Lane l's accumulator value i is D[8 (i/4) + 4 (l/32) + i%4][l % 32]; the
// valid ones go to out[m * Nv + n] (the wave's slot).
template <class C, class M>
RCPB_FN void mfma_store(M& m, int lane, int o, int Mv, int Nv, const float* acc) {
    const int n = lane & 31;
    if (n >= Nv) return;
#pragma unroll
    for (int i = 0; i < 16; i++) {
        const int mm = 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
        if (mm < Mv) m.lw(o + mm * Nv + n, m.fbits(acc[i]));
    }
}

// E: G1[s2] = sum_t2l W2[t2][s2] G2[t2l][s3][n] (bf16), dX[s1][s2] += W1[t1][s1] G1[s2],
// dW1[s1] partial += G1[s2] X[s1][s2]; row sums of the dW1 partials -> Q.
template <class C, class M>
RCPB_FN void phase_e(M& m, const RcpBwdDesc& d, int lane, int wave, int r, int t1, int chunk,
                     const uint32_t* TB, State<C>& st) {
    static_assert(C::T2C % 2 == 0, "t2 chunks come in pairs");
    constexpr int T2P = C::T2C / 2;
    float w1[C::S1], dw1[C::S1];
    uint32_t w2p[C::S2][T2P];   // (W2[2i][s2], W2[2i+1][s2]) of the chunk
    const int64_t o1 = (int64_t)r * d.tbs + C::KK + C::S3 * C::T3P, o2 = o1 + (int64_t)d.T1 * C::S1;
#pragma unroll
    for (int s = 0; s < C::S1; s++) {
        w1[s] = m.fof(m.ldt(TB, o1 + t1 * C::S1 + s));
        dw1[s] = 0.f;
    }
#pragma unroll
    for (int s = 0; s < C::S2; s++)
#pragma unroll
        for (int i = 0; i < T2P; i++) w2p[s][i] = m.ldt(TB, o2 + s * (C::T2 / 2) + chunk * T2P + i);
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        if (st.a_n[k] < 0) continue;
        const int n = st.a_n[k], s3 = st.a_s3[k];
        uint32_t g2[T2P];
#pragma unroll
        for (int i = 0; i < T2P; i++)
            g2[i] = (uint32_t)lds_e(m, d.o_g2, ig2(d, 2 * i, s3, n)) |
                    ((uint32_t)lds_e(m, d.o_g2, ig2(d, 2 * i + 1, s3, n)) << 16);
#pragma unroll
        for (int s2 = 0; s2 < C::S2; s2++) {
            float g1 = 0.f;
#pragma unroll
            for (int i = 0; i < T2P; i++) g1 = m.dot2(w2p[s2][i], g2[i], g1);
            g1 = m.f(m.bf(g1));
#pragma unroll
            for (int j = 0; j < C::S1P; j++) {
                const uint32_t xw = st.xp[k][j][s2];
                st.dxa[k][2 * j][s2] += w1[2 * j] * g1;
                st.dxa[k][2 * j + 1][s2] += w1[2 * j + 1] * g1;
                dw1[2 * j] += g1 * m.f((uint16_t)(xw & 0xffff));
                dw1[2 * j + 1] += g1 * m.f((uint16_t)(xw >> 16));
            }
        }
    }
#pragma unroll
    for (int s = 0; s < C::S1; s++)
        m.rowsum(dw1[s], lane, d.o_q + (C::KK + s) * 4 * C::NW + 4 * wave + (lane >> 4));
}

// F: the workgroup's partials of rank r: dW0 taps and dW1 from the row sums
// in Q, dW3 and dW2 from the wave slots (each summed in slot order); zeros for the t1 rows and
// t2 chunks other workgroups own.  Slot layouts: P0[blk][r][KK],
// P1[blk][r][T1*S1], P2[blk][r][T2*S2], P3[blk][r][T3*S3].
template <class C, class M>
RCPB_FN void phase_f(M& m, const RcpBwdDesc& d, int tid, int64_t blk, int r, int t1, int chunk,
                      float* P0, float* P1, float* P2, float* P3) {
    const int n0 = C::KK, n1 = d.T1 * C::S1, n2 = C::T2 * C::S2, n3 = C::T3 * C::S3;
    for (int i = tid; i < n0 + n1 + n2 + n3; i += C::NT) {
        if (i < n0) {
            float s = 0.f;
            for (int g = 0; g < 4 * C::NW; g++) s += m.fof(m.lr(d.o_q + i * 4 * C::NW + g));
            m.stf(P0, (blk * d.R + r) * n0 + i, s);
        } else if (i < n0 + n1) {
            const int e = i - n0, tt = e / C::S1, s1 = e % C::S1;
            float s = 0.f;
            if (tt == t1)
                for (int g = 0; g < 4 * C::NW; g++) s += m.fof(m.lr(d.o_q + (C::KK + s1) * 4 * C::NW + g));
            m.stf(P1, (blk * d.R + r) * n1 + e, s);
        } else if (i < n0 + n1 + n2) {
            const int e = i - n0 - n1, t2 = e / C::S2, s2 = e % C::S2;
            float s = 0.f;
            if (t2 / C::T2C == chunk)
                for (int w = 0; w < C::NW; w++)
                    s += m.fof(m.lr(d.o_m2 + w * C::T2C * C::S2 + (t2 % C::T2C) * C::S2 + s2));
            m.stf(P2, (blk * d.R + r) * n2 + e, s);
        } else {
            const int e = i - n0 - n1 - n2;
            float s = 0.f;
            for (int w = 0; w < C::NW; w++) s += m.fof(m.lr(d.o_m3 + w * C::T3 * C::S3 + e));
            m.stf(P3, (blk * d.R + r) * n3 + e, s);
        }
    }
}

// Word i of the prepared factor table (row r = i / tbs):
//   [0, KK)                W0[r][tap] as fp32
//   [KK, + S3*T3/2)        (W3[r][2j][s3], W3[r][2j+1][s3]) at s3 * T3/2 + j
//   [.., + T1*S1)          W1[r][t1][s1] as fp32 at t1 * S1 + s1
//   [.., + S2*T2/2)        (W2[r][2j][s2], W2[r][2j+1][s2]) at s2 * T2/2 + j
template <class M>
RCPB_FN uint32_t table_word(M& m, const RcpBwdDesc& d, int64_t i, const uint16_t* W1, const uint16_t* W2,
                            const uint16_t* W3, const uint16_t* W0) {
    const int64_t r = i / d.tbs;
    int64_t e = i % d.tbs;
    const int KK = d.K * d.K, T3P = d.T3 / 2, T2P = d.T2 / 2;
    if (e < KK) return m.fbits(m.f(m.ld16(W0, r * KK + e)));
    e -= KK;
    if (e < (int64_t)d.S3 * T3P) {
        const int s3 = (int)(e / T3P), j = (int)(e % T3P);
        return (uint32_t)m.ld16(W3, (r * d.T3 + 2 * j) * d.S3 + s3) |
               ((uint32_t)m.ld16(W3, (r * d.T3 + 2 * j + 1) * d.S3 + s3) << 16);
    }
    e -= (int64_t)d.S3 * T3P;
    if (e < (int64_t)d.T1 * d.S1) return m.fbits(m.f(m.ld16(W1, r * d.T1 * d.S1 + e)));
    e -= (int64_t)d.T1 * d.S1;
    const int s2 = (int)(e / T2P), j = (int)(e % T2P);
    return (uint32_t)m.ld16(W2, (r * d.T2 + 2 * j) * d.S2 + s2) |
           ((uint32_t)m.ld16(W2, (r * d.T2 + 2 * j + 1) * d.S2 + s2) << 16);
}

// dX partial of the workgroup: DXP[t1 * nc + chunk][b][s1][s2][s3][h0 W + n].
template <class C, class M>
RCPB_FN void store_dx(M& m, const RcpBwdDesc& d, int b, int t1, int h0, int chunk, float* DXP, const State<C>& st) {
    const int64_t HW = (int64_t)d.H * d.W, S = C::S1 * C::S2 * C::S3;
    const int64_t base = (((int64_t)t1 * d.nc + chunk) * d.B + b) * S * HW + (int64_t)h0 * d.W;
#pragma unroll
    for (int k = 0; k < C::UA; k++) {
        if (st.a_n[k] < 0) continue;
        const int n = st.a_n[k], s3 = st.a_s3[k];
#pragma unroll
        for (int s1 = 0; s1 < C::S1; s1++)
#pragma unroll
            for (int s2 = 0; s2 < C::S2; s2++)
                m.stf(DXP, base + ((int64_t)(s1 * C::S2 + s2) * C::S3 + s3) * HW + n, st.dxa[k][s1][s2]);
    }
}

}  // namespace rcpb
}  // namespace ce
