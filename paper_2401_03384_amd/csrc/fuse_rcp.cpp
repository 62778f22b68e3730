// Fusion of the reshaped-CP chain (Section 2.3, reshaped CP layer; the RCP
// string of Appendix A.3 with three modes) into one forward launch.
//
// Matched at the level of the plan: the expression must read
//   X[b][s1][s2][s3][h][w], W1[r][t1][s1], W2[r][t2][s2], W3[r][t3][s3], W0[r][h][w]
//   -> Y[b][t1][t2][t3][h][w],  h and w convolved (X the feature side),
// every tensor dense in that label order, and the planned tree must apply the
// factors one at a time in the order W1, W2, W3, W0 (the canonical optimum of
// the tnn-cost sequencer for these layers).  The fused kernel then computes
// exactly the planned steps (mode product by mode product, then the
// convolution summed over the rank) without storing their intermediates.
#include <algorithm>
#include <cstring>

#include "desc_rcp.h"
#include "plan.h"

namespace ce {

namespace {

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

}  // namespace

bool fuse_rcp_forward(const ce_plan& p, Launch& out) {
    const ce_expr& E = p.e;
    if (p.dtype != CE_BF16 || E.n != 5 || p.steps.size() != 4) return false;
    const int X = E.feature_operand;
    if (X != 0) return false;
    // the chain: ((((X, F1), F2), F3), F0)
    int f[4];
    for (int s = 0; s < 4; s++) {
        const Step& st = p.steps[s];
        if (st.a != (s == 0 ? X : p.steps[s - 1].c) || st.b >= E.n || st.b == X) return false;
        f[s] = st.b;
    }
    const std::vector<int>& xl = E.ops[X];
    if (xl.size() != 6 || E.out.size() != 6) return false;
    const int lb = xl[0], lh = xl[4], lw = xl[5];
    if (!E.is_conv(lh) || !E.is_conv(lw) || E.is_conv(lb) || E.feature_of(lh) != X || E.feature_of(lw) != X)
        return false;
    // mode factors [r][t_i][s_i] with s_i the (i+1)-th label of X, in step order
    int lr = -1, lt[3];
    int64_t S[3], T[3];
    for (int i = 0; i < 3; i++) {
        const std::vector<int>& l = E.ops[f[i]];
        if (l.size() != 3 || l[2] != xl[1 + i] || E.is_conv(l[0]) || E.is_conv(l[1])) return false;
        if (i == 0) lr = l[0];
        if (l[0] != lr || E.in_out(lr) || !E.in_out(l[1])) return false;
        lt[i] = l[1];
        S[i] = E.dims[X][1 + i];
        T[i] = E.dims[f[i]][1];
        if (E.dims[f[i]][2] != S[i]) return false;
    }
    for (int l : xl)
        if (l == lr) return false;
    // spatial factor [r][h][w]
    const std::vector<int>& l0 = E.ops[f[3]];
    if (l0.size() != 3 || l0[0] != lr || l0[1] != lh || l0[2] != lw) return false;
    const int64_t K = E.dims[f[3]][1];
    if (E.dims[f[3]][2] != K || K % 2 == 0) return false;
    // output [b][t1][t2][t3][h][w]
    const std::vector<int>& ol = E.out;
    if (ol[0] != lb || ol[1] != lt[0] || ol[2] != lt[1] || ol[3] != lt[2] || ol[4] != lh || ol[5] != lw)
        return false;
    // labels of X must not appear elsewhere except as described (b only in X and Y)
    for (int i = 0; i < 5; i++)
        if (i != X)
            for (int l : E.ops[i])
                if (l == lb) return false;
    const int64_t B = E.dims[X][0], H = E.dims[X][4], W = E.dims[X][5];
    const int64_t R = E.dims[f[0]][0];
    if (B < 1 || H < K || W < K || R < 2 || R % 2) return false;
    if (B * S[0] * S[1] * S[2] * H * W >= (1ll << 31) || B * T[0] * T[1] * T[2] * H * W >= (1ll << 31))
        return false;
    for (int c = 0; c < kNumRcpCfgs; c++) {
        const RcpCfgInfo& g = kRcpCfgs[c];
        if (S[0] != g.S1 || S[1] != g.S2 || S[2] != g.S3 || T[1] != g.T2 || T[2] != g.T3 || K != g.K) continue;
        RcpDesc d;
        std::memset(&d, 0, sizeof(d));
        d.S1 = g.S1; d.S2 = g.S2; d.S3 = g.S3; d.T2 = g.T2; d.T3 = g.T3; d.K = g.K;
        d.T2C = g.T2C; d.NT = g.NT;
        d.B = (int32_t)B; d.T1 = (int32_t)T[0]; d.R = (int32_t)R; d.H = (int32_t)H; d.W = (int32_t)W;
        d.nc = g.T2 / g.T2C;
        d.QW = (int32_t)((W + 3) / 4);
        d.WP = (int32_t)round_up(4 * d.QW + K - 1, 4);
        // fewest row tiles whose units fit the instantiation and whose LDS fits
        const int64_t c0 = (K - 1) / 2;
        bool found = false;
        for (int64_t nt = 1; nt <= H && !found; nt++) {
            const int64_t TH = (H + nt - 1) / nt, ntiles = (H + TH - 1) / TH;
            int64_t rows = 0;
            for (int64_t i = 0; i < ntiles; i++) {
                const int64_t h0 = i * TH, h1 = std::min(H, h0 + TH);
                rows = std::max(rows, std::min(H, h1 + c0) - std::max<int64_t>(0, h0 - c0));
            }
            const int64_t zb = round_up((int64_t)g.T2C * (g.S3 / 2) * rows * W, 4);
            const int64_t plane = (TH + K - 1) * d.WP, zc = (int64_t)g.T2C * g.T3 * plane;
            const int64_t lds = 4 * (2 * zb + zc);
            if (rows * W * (g.S3 / 2) > (int64_t)g.UA * g.NT || rows * W * g.T2C > (int64_t)g.UB * g.NT ||
                (int64_t)g.T2C * g.T3 * TH * d.QW > (int64_t)g.UC * g.NT || lds > 160 * 1024)
                continue;
            d.TH = (int32_t)TH;
            d.ntiles = (int32_t)ntiles;
            d.HP = (int32_t)(TH + K - 1);
            d.zb_dw = (int32_t)zb;
            d.plane_dw = (int32_t)plane;
            d.zc_dw = (int32_t)zc;
            d.lds_bytes = (uint32_t)lds;
            found = true;
        }
        if (!found) continue;
        d.blocks = B * T[0] * d.ntiles * d.nc;
        if (d.blocks > 0x7fffffff) continue;
        const int64_t HW = H * W;
        out = Launch();
        out.kind = K_RCP_FWD | (1 << kBitIn) | (1 << kBitAux) | (1 << kBitOut);
        BufRef bx, bw[4];
        bx.kind = BUF_IN;
        bx.index = X;
        for (int i = 0; i < 4; i++) {
            bw[i].kind = BUF_IN;
            bw[i].index = f[i];
        }
        out.a = bx;
        out.b = bw[0];
        out.extra = {bw[1], bw[2], bw[3]};
        out.c.kind = BUF_OUT;
        out.grid[0] = (uint32_t)d.blocks;
        out.block[0] = (uint32_t)g.NT;
        out.lds = d.lds_bytes;
        out.desc.resize(sizeof(d));
        std::memcpy(out.desc.data(), &d, sizeof(d));
        out.need = 0x1f;
        out.what = "fused RCP chain: steps 0-3 (mode products s1, s2, s3; rank-summed conv hw)";
        // the kernel's template name as profilers print it
        out.kname = "rcp_fwd<ce::rcp::Cfg<";
        const int tp[11] = {g.S1, g.S2, g.S3, g.T2, g.T3, g.K, g.T2C, g.NT, g.UA, g.UB, g.UC};
        for (int i = 0; i < 11; i++) out.kname += std::to_string(tp[i]) + (i < 10 ? ", " : "> >");
        double macs = 0;
        for (const Step& st : p.steps) macs += (double)st.macs;
        out.alg_flops = 2.0 * macs;
        const double Sx = (double)(S[0] * S[1] * S[2]), Ty = (double)(T[0] * T[1] * T[2]);
        out.alg_bytes = 2.0 * ((double)B * HW * (Sx + Ty) +
                               (double)R * (T[0] * S[0] + T[1] * S[1] + T[2] * S[2] + K * K));
        return true;
    }
    return false;
}

}  // namespace ce

namespace ce {

namespace {

int64_t al4(int64_t x) { return (x + 3) & ~int64_t(3); }

}  // namespace

bool fuse_rcp_backward(const Launch& f, const ce_plan& p, ScratchAlloc& scratch, std::vector<Launch>& out) {
    if ((f.kind & 0xff) != K_RCP_FWD || f.extra.size() != 3) return false;
    RcpDesc fd;
    std::memcpy(&fd, f.desc.data(), sizeof(fd));
    const int64_t B = fd.B, T1 = fd.T1, R = fd.R, H = fd.H, W = fd.W, K = fd.K;
    const int64_t S1 = fd.S1, S2 = fd.S2, S3 = fd.S3, T2 = fd.T2, T3 = fd.T3;
    const int64_t HW = H * W, S = S1 * S2 * S3, KK = K * K;
    if (R % 2) return false;   // factor buffers of an even element count (word loads)
    for (int c = 0; c < kNumRcpBwdCfgs; c++) {
        const RcpCfgInfo& g = kRcpBwdCfgs[c];
        if (S1 != g.S1 || S2 != g.S2 || S3 != g.S3 || T2 != g.T2 || T3 != g.T3 || K != g.K) continue;
        RcpBwdDesc d;
        std::memset(&d, 0, sizeof(d));
        d.S1 = g.S1; d.S2 = g.S2; d.S3 = g.S3; d.T2 = g.T2; d.T3 = g.T3; d.K = g.K;
        d.T2C = g.T2C; d.NT = g.NT;
        d.B = (int32_t)B; d.T1 = (int32_t)T1; d.R = (int32_t)R; d.H = (int32_t)H; d.W = (int32_t)W;
        d.nc = g.T2 / g.T2C;
        d.QW = (int32_t)((W + 3) / 4);
        d.WP = (int32_t)(((4 * d.QW + K - 1) + 3) / 4 * 4);
        const int64_t NW = g.NT / 64, NV = KK + S1;
        // the tallest tile whose units fit the instantiation and whose LDS fits
        bool found = false;
        for (int64_t TH = H; TH >= 1 && !found; TH--) {
            const int64_t P = TH * W, PP = (P + 15) / 16 * 16, HPb = TH + K - 1;
            const int64_t L13 = g.S3 * PP + 8, L2 = g.T2C * PP + 8;
            if (P * g.S3 > (int64_t)g.UA * g.NT || P * g.T2C > (int64_t)g.UB * g.NT ||
                (int64_t)g.T2C * g.T3 * TH * d.QW > (int64_t)g.UC * g.NT)
                continue;
            int64_t o = al4((int64_t)g.T2C * g.T3 * HPb * d.WP);
            const int64_t o_z1 = o;
            o = al4(o + g.S2 * L13 / 2);
            const int64_t o_z2 = o;
            o = al4(o + g.S3 * L2 / 2);
            const int64_t o_z3 = o;
            o = al4(o + (g.T2C * g.T3 * P + 1) / 2);
            const int64_t o_g3 = o;
            o = al4(o + g.T3 * L2 / 2);
            const int64_t o_g2 = o;
            o = al4(o + g.T2C * L13 / 2);
            const int64_t o_q = o;
            o += NV * 4 * NW;
            const int64_t o_m3 = o;
            o += NW * g.T3 * g.S3;
            const int64_t o_m2 = o;
            o += NW * g.T2C * g.S2;
            if (4 * o > 160 * 1024) continue;
            d.TH = (int32_t)TH;
            d.ntiles = (int32_t)((H + TH - 1) / TH);
            d.HPb = (int32_t)HPb;
            d.PP = (int32_t)PP;
            d.L13 = (int32_t)L13;
            d.L2 = (int32_t)L2;
            d.o_dy = 0; d.o_z1 = (int32_t)o_z1; d.o_z2 = (int32_t)o_z2; d.o_z3 = (int32_t)o_z3;
            d.o_g3 = (int32_t)o_g3; d.o_g2 = (int32_t)o_g2; d.o_q = (int32_t)o_q;
            d.o_m3 = (int32_t)o_m3; d.o_m2 = (int32_t)o_m2;
            d.lds_bytes = (uint32_t)(4 * o);
            found = true;
        }
        if (!found) continue;
        d.blocks = B * T1 * d.ntiles * d.nc;
        if (d.blocks > 0x7fffffff) continue;
        d.tbs = (int32_t)(KK + S3 * (T3 / 2) + T1 * S1 + S2 * (T2 / 2));
        const int64_t nblk = d.blocks, nslot = T1 * d.nc;
        const int64_t n0 = KK, n1 = T1 * S1, n2 = T2 * S2, n3 = T3 * S3;
        const BufRef DXP = scratch.alloc((size_t)(nslot * B * S * HW) * 4);
        const BufRef P0 = scratch.alloc((size_t)(nblk * R * n0) * 4);
        const BufRef P1 = scratch.alloc((size_t)(nblk * R * n1) * 4);
        const BufRef P2 = scratch.alloc((size_t)(nblk * R * n2) * 4);
        const BufRef P3 = scratch.alloc((size_t)(nblk * R * n3) * 4);
        const BufRef TB = scratch.alloc((size_t)(R * d.tbs) * 4);
        const BufRef X = f.a, W1 = f.b, W2 = f.extra[0], W3 = f.extra[1], W0 = f.extra[2];
        // the factor table: fp32 taps and rows, pairs along the contracted mode
        Launch lp;
        lp.kind = K_RCP_PREP;
        lp.extra = {W1, W2, W3, W0, TB};
        lp.grid[0] = (uint32_t)((R * d.tbs + 255) / 256);
        lp.block[0] = 256;
        lp.desc.resize(sizeof(d));
        std::memcpy(lp.desc.data(), &d, sizeof(d));
        lp.need = 0x1f;
        lp.what = "factor table of the fused RCP backward";
        lp.kname = "rcp_prep";
        lp.alg_bytes = 2.0 * R * (KK + T1 * S1 + T2 * S2 + T3 * S3) + 4.0 * R * d.tbs;
        out.push_back(lp);
        auto din = [](const BufRef& in) {
            BufRef r;
            r.kind = BUF_DIN;
            r.index = in.index;
            return r;
        };
        Launch m;
        m.kind = K_RCP_BWD | (1 << kBitIn) | (1 << kBitAux) | (1 << kBitOut);
        m.a = X;
        m.b.kind = BUF_DOUT;
        m.extra = {W1, W2, W3, W0, DXP, P0, P1, P2, P3, TB};
        m.grid[0] = (uint32_t)d.blocks;
        m.block[0] = (uint32_t)g.NT;
        m.lds = d.lds_bytes;
        m.desc.resize(sizeof(d));
        std::memcpy(m.desc.data(), &d, sizeof(d));
        m.need = 0x1f;
        m.what = "fused RCP chain backward: steps 3-0 (recompute, g1 and g2 of every step)";
        m.kname = "rcp_bwd<ce::rcpb::Cfg<";
        const int tp[12] = {g.S1, g.S2, g.S3, g.T2, g.T3, g.K, g.T2C, g.NT, g.UA, g.UB, g.UC, g.MW};
        for (int i = 0; i < 12; i++) m.kname += std::to_string(tp[i]) + (i < 11 ? ", " : "> >");
        // algorithmic bytes: X and dY read, dX partials and factor partials written
        const double act = (double)B * HW;
        m.alg_bytes = 2.0 * act * (double)(S + T1 * T2 * T3) + 4.0 * (double)nslot * act * S +
                      4.0 * (double)nblk * R * (n0 + n1 + n2 + n3) + 2.0 * R * (n0 + n1 + n2 + n3);
        m.alg_flops = 2.0 * f.alg_flops;   // backward multiplications are twice the forward's
        out.push_back(m);
        // the four factor gradients: ordered sums over the workgroups
        MultiReduceDesc md;
        std::memset(&md, 0, sizeof(md));
        md.n = 4;
        const BufRef parts[4] = {P1, P2, P3, P0}, outs[4] = {din(W1), din(W2), din(W3), din(W0)};
        const int64_t ns[4] = {n1, n2, n3, n0};
        for (int j = 0; j < 4; j++) {
            ReduceDesc& rd = md.part[j];
            rd.M = (int32_t)R;
            rd.N = (int32_t)ns[j];
            rd.nsplit = nblk;
            rd.sCm = ns[j];
            rd.sCn = 1;
            md.block0[j + 1] = md.block0[j] + (R * ns[j] + 63) / 64;
        }
        Launch lr;
        lr.kind = K_REDUCE_MULTI;
        lr.extra = {parts[0], outs[0], parts[1], outs[1], parts[2], outs[2], parts[3], outs[3]};
        lr.grid[0] = (uint32_t)md.block0[4];
        lr.block[0] = (uint32_t)(64 * reduce_waves(nblk));
        lr.desc.resize(sizeof(md));
        std::memcpy(lr.desc.data(), &md, sizeof(md));
        lr.need = (1u << W1.index) | (1u << W2.index) | (1u << W3.index) | (1u << W0.index);
        lr.what = "dW1, dW2, dW3, dW0: sums of workgroup partials";
        lr.kname = "reduce_multi<" + std::to_string(reduce_waves(nblk)) + ">";
        lr.alg_bytes = 4.0 * (double)nblk * R * (n0 + n1 + n2 + n3) + 4.0 * R * (n0 + n1 + n2 + n3);
        out.push_back(lr);
        // dX: ordered sum of the per-(t1, t2 chunk) partials, rounded to bf16
        ReduceDesc rd;
        std::memset(&rd, 0, sizeof(rd));
        rd.M = (int32_t)B;
        rd.N = (int32_t)(S * HW);
        rd.nsplit = nslot;
        rd.sCm = S * HW;
        rd.sCn = 1;
        Launch lx;
        lx.kind = K_REDUCE | (0 << kBitIn) | (0 << kBitAux) | (1 << kBitOut);
        lx.d = DXP;
        lx.c = din(X);
        lx.grid[0] = (uint32_t)((B * S * HW + 63) / 64);
        lx.block[0] = (uint32_t)(64 * reduce_waves(nslot));
        lx.desc.resize(sizeof(rd));
        std::memcpy(lx.desc.data(), &rd, sizeof(rd));
        lx.need = 1u << X.index;
        lx.what = "dX: sum of the per-(t1, t2 chunk) partials";
        lx.kname = "reduce_partials<" + std::to_string(reduce_waves(rd.nsplit)) + ", unsigned short>";
        lx.alg_bytes = 4.0 * (double)nslot * act * S + 2.0 * act * S;
        out.push_back(lx);
        return true;
    }
    return false;
}

}  // namespace ce
