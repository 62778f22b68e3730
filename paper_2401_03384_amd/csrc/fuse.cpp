// Launch-level fusion of pairwise steps into fused kernels.
//
// CP chain (Section 2.3, CP convolutional layer): the planned forward steps
//   GEMM  Z1[b][r][hw] = sum_s Us[r][s] X[b][s][hw]
//   DW    Z2 = Z1 convolved along h with Kh[r]
//   DW    Z3 = Z2 convolved along w with Kw[r]
//   GEMM  Y[b][t][hw]  = sum_r Ut[r][t] Z3[b][r][hw]
// chained through workspace intermediates become one launch of the fused
// kernel, which keeps Z1..Z3 on chip.
#include <algorithm>
#include <cstring>

#include "plan.h"

namespace ce {

namespace {

size_t al16(size_t x) { return (x + 15) & ~size_t(15); }

// LDS operand tables of the fused CP kernel: Us as [32][S+pad] (the GEMM1 A
// operand rows; bf16 rows padded to keep 16-byte k-runs aligned), Ut permuted
// to the accumulator-layout pairing of GEMM2 (fp32 [16][2][T], bf16
// [2][2][T][8]) and the taps permuted the same way ([16][2][K]).
// Channel counts below 32 or between 32 and 64 run padded to 32 or 64 (the
// kernels' channel blocks): the tables hold zeros there.
int pad32(int n) { return 32 * ((n + 31) / 32); }

void cp_tables(CpDesc& d, bool bf) {
    const int SP = pad32(d.S), TP = pad32(d.T);
    d.lda = bf ? SP + 8 : SP + 1;
    size_t o = al16((size_t)32 * d.lda * (bf ? 2 : 4));
    d.o_ut = (uint32_t)o;
    o = al16(o + (bf ? (size_t)2 * 2 * TP * 8 * 2 : (size_t)16 * 2 * TP * 4));
    d.o_kh = (uint32_t)o;
    o += (size_t)16 * 2 * d.KH * 4;
    d.o_kw = (uint32_t)o;
    o += (size_t)16 * 2 * d.KW * 4;
    d.o_khr = (uint32_t)o;
    o += (size_t)16 * 2 * d.KH * 4;
    d.lds_bytes = (uint32_t)al16(o);
}

template <typename D>
D desc(const Launch& ln) {
    D d;
    std::memcpy(&d, ln.desc.data(), sizeof(D));
    return d;
}

bool same(const BufRef& a, const BufRef& b) {
    return a.kind == b.kind && a.index == b.index && a.offset == b.offset;
}

int dtin(const Launch& l) { return (l.kind >> kBitIn) & 1; }
int dtaux(const Launch& l) { return (l.kind >> kBitAux) & 1; }
int dtout(const Launch& l) { return (l.kind >> kBitOut) & 1; }

bool match_cp_fwd(const std::vector<Launch>& v, size_t i, Launch& fused) {
    if (i + 4 > v.size()) return false;
    const Launch &g1 = v[i], &d1 = v[i + 1], &d2 = v[i + 2], &g2 = v[i + 3];
    if ((g1.kind & 0xff) != K_GEMM || (d1.kind & 0xff) != K_DW || (d2.kind & 0xff) != K_DW ||
        (g2.kind & 0xff) != K_GEMM)
        return false;
    if (g1.c.kind != BUF_WS || !same(g1.c, d1.a) || !same(d1.c, d2.a) || !same(d2.c, g2.b) ||
        d1.c.kind != BUF_WS || d2.c.kind != BUF_WS)
        return false;
    int dt = dtin(g1);
    for (const Launch* l : {&g1, &d1, &d2, &g2})
        if (dtin(*l) != dt || dtout(*l) != dt) return false;
    if (dtaux(d1) != dt || dtaux(d2) != dt || dtaux(g1) != dt || dtaux(g2) != dt) return false;
    GemmDesc a = desc<GemmDesc>(g1), c = desc<GemmDesc>(g2);
    DwDesc h = desc<DwDesc>(d1), w = desc<DwDesc>(d2);
    const int64_t R = a.M, S = a.K, T = c.M, H = h.A, W = h.inner;
    if (a.ng != 1 || c.ng != 1 || a.g_sA[0] != 0 || c.g_sA[0] != 0) return false;
    const int64_t B = a.g_size[0];
    if (c.g_size[0] != B || a.N != H * W || c.N != H * W || c.K != R) return false;
    if (a.g_sC[0] != R * H * W || a.sCm != H * W || c.sBk != H * W || c.g_sB[0] != R * H * W)
        return false;
    if (h.nslab != B * R || h.r_div != 1 || h.r_size != R || h.sign != 1 ||
        h.off != -((h.K - 1) / 2))
        return false;
    if (w.nslab != B * R * H || w.A != W || w.inner != 1 || w.r_div != H || w.r_size != R ||
        w.sign != 1 || w.off != -((w.K - 1) / 2))
        return false;
    // register-resident strips: rank at most 32 (ranks past R as zero rows),
    // S and T at most 64 (padded to 32 or 64), 3x3 or 5x5 filters
    if (R < 1 || R > 32 || T < 1 || T > 64 || S < 1 || S > 64 || h.K != w.K || !(h.K == 3 || h.K == 5))
        return false;
    // one sample of X and of Y within a 32-bit byte range (raw buffer loads and
    // stores), both with channel stride H*W
    if (S * a.sBk * (dt ? 2 : 4) >= (1ll << 31) || a.sBk != H * W) return false;
    if (T * c.sCm * (dt ? 2 : 4) >= (1ll << 31) || c.sCm != H * W) return false;
    CpDesc d;
    std::memset(&d, 0, sizeof(d));
    d.B = (int32_t)B;
    d.S = (int32_t)S;
    d.R = (int32_t)R;
    d.T = (int32_t)T;
    d.H = (int32_t)H;
    d.W = (int32_t)W;
    d.KH = h.K;
    d.KW = w.K;
    d.x_sb = a.g_sB[0];
    d.x_ss = a.sBk;
    d.y_sb = c.g_sC[0];
    d.y_st = c.sCm;
    d.us_sr = a.sAm;
    d.us_ss = a.sAk;
    d.ut_st = c.sAm;
    d.ut_sr = c.sAk;
    d.kh_sr = h.r_stride;
    d.kh_sj = h.f_sj;
    d.kw_sr = w.r_stride;
    d.kw_sj = w.f_sj;
    d.colstride = 32 - (w.K - 1);
    d.ncb = (int32_t)((W + d.colstride - 1) / d.colstride);
    // wavefronts: about two per SIMD of the 1024 SIMDs; each strip segment
    // recomputes KH-1 rows of Z1 (bf16 forward, C2: 4096 waves with 4-row
    // segments 40 us, 2048 with 7-row segments 35 us; fp32 unchanged)
    const int64_t want = 2048;
    int64_t segs = std::max<int64_t>(1, std::min<int64_t>(H, want / std::max<int64_t>(1, B * d.ncb)));
    d.seg_rows = (int32_t)((H + segs - 1) / segs);
    d.segs = (int32_t)((H + d.seg_rows - 1) / d.seg_rows);
    d.waves = B * d.ncb * d.segs;
    d.blocks = (d.waves + 3) / 4;
    if (d.blocks > 0x7fffffff) return false;
    cp_tables(d, dt == 1);
    fused = Launch();
    fused.kind = K_CP_FWD | (dt << kBitIn) | (dt << kBitAux) | (dt << kBitOut);
    fused.a = g1.b;                       // X
    fused.b = g1.a;                       // Us
    fused.c = g2.c;                       // Y
    fused.extra = {d1.b, d2.b, g2.a};     // Kh, Kw, Ut
    fused.grid[0] = (uint32_t)d.blocks;
    fused.block[0] = 256;
    fused.lds = d.lds_bytes;
    fused.desc.resize(sizeof(d));
    std::memcpy(fused.desc.data(), &d, sizeof(d));
    fused.need = g1.need | d1.need | d2.need | g2.need;
    fused.what = "fused CP chain: " + g1.what + " | " + d1.what + " | " + d2.what + " | " + g2.what;
    fused.kname = std::string("cp_fwd<") + (dt ? "unsigned short" : "float") + ", " +
                  std::to_string(h.K) + ", " + std::to_string(w.K) + ", " + std::to_string(pad32((int)T) / 32) + ", " +
                  std::to_string(pad32((int)S) / 32) + ((dt == 1 && T != pad32((int)T)) ? ", true>" : ", false>");
    fused.alg_bytes = g1.alg_bytes + d1.alg_bytes + d2.alg_bytes + g2.alg_bytes;
    fused.alg_flops = g1.alg_flops + d1.alg_flops + d2.alg_flops + g2.alg_flops;
    // algorithmic bytes of the fused launch: X, factors and Y only
    double e = dt ? 2 : 4;
    fused.alg_bytes = e * (double)(B * S * H * W + B * T * H * W + R * S + R * T + R * (h.K + w.K));
    return true;
}


// LDS of the fused backward (see CpBwdDesc).
void cp_bwd_tables(CpBwdDesc& d, bool bf) {
    const size_t e = bf ? 2 : 4;
    const int SP = pad32(d.S), TP = pad32(d.T);
    d.lda_s = bf ? SP + 8 : SP + 1;
    d.lda_t = bf ? TP + 8 : TP + 1;
    d.ldu = bf ? 32 + 8 : 0;
    d.ly = bf ? 40 : 33;
    d.lx = bf ? 40 : 36;   // 8-byte (bf16) / 16-byte (fp32) column runs stay aligned
    size_t o = al16((size_t)32 * d.lda_s * e);
    d.o_uta = (uint32_t)o;
    o = al16(o + (size_t)32 * d.lda_t * e);
    d.o_ust = (uint32_t)o;
    if (bf) o = al16(o + (size_t)SP * d.ldu * 2);
    const size_t tz = (size_t)32 * 33 * 4, yt = al16((size_t)TP * d.ly * e);
    const size_t xl = al16((size_t)3 * SP * d.lx * e);
    // the dZ1 transpose tile gets its own space when everything fits, else it
    // shares the wave's dY tile (used earlier in each row)
    const bool share = o + 4 * (tz + yt + xl) > (size_t)160 * 1024;
    d.o_tz = (uint32_t)o;
    d.tz_stride = (uint32_t)(share ? std::max(tz, yt) : tz);
    if (!share) o += 4 * tz;
    d.o_yt = (uint32_t)o;
    d.yt_bytes = (uint32_t)(share ? d.tz_stride : yt);
    o += (size_t)4 * d.yt_bytes;
    d.o_xl = (uint32_t)o;
    d.xl_bytes = (uint32_t)xl;
    o += 4 * xl;
    d.red_bytes = (uint32_t)(4 * std::max<size_t>({(size_t)4 * 32 * SP, (size_t)4 * 32 * TP,
                                                   (size_t)8 * 32 * (d.KH + d.KW)}));
    d.lds_bytes = (uint32_t)std::max<size_t>(al16(o), d.red_bytes);
}


}  // namespace

bool fuse_cp_backward(const Launch& f, int feature_operand, ScratchAlloc& scratch,
                      std::vector<Launch>& out) {
    if ((f.kind & 0xff) != K_CP_FWD || f.extra.size() != 3) return false;
    if (f.a.kind != BUF_IN || f.b.kind != BUF_IN || f.c.kind != BUF_OUT) return false;
    for (const BufRef& x : f.extra)
        if (x.kind != BUF_IN) return false;
    if (f.a.index != feature_operand) return false;   // dX is in the input type
    const CpDesc c = desc<CpDesc>(f);
    // 3x3 filters, S and T padded to the same channel block count (32 or 64:
    // the kernel's register budget), rank at most 32 (one rank a lane; ranks
    // past R run as zero rows)
    if (c.KH != 3 || c.KW != 3 || c.S < 1 || c.S > 64 || c.T < 1 || c.T > 64 || pad32(c.S) != pad32(c.T) ||
        c.R < 1 || c.R > 32)
        return false;
    const int dt = dtin(f);
    // one sample of X, dY and dX is addressed with 31-bit byte offsets
    const int64_t e_in = dt ? 2 : 4;
    if ((int64_t)c.S * c.x_ss * e_in >= (1ll << 31) || (int64_t)c.T * c.y_st * e_in >= (1ll << 31) ||
        c.x_ss != (int64_t)c.H * c.W || c.y_st != (int64_t)c.H * c.W)
        return false;
    CpBwdDesc d;
    std::memset(&d, 0, sizeof(d));
    d.B = c.B; d.S = c.S; d.R = c.R; d.T = c.T; d.H = c.H; d.W = c.W; d.KH = c.KH; d.KW = c.KW;
    d.ncb = c.ncb;
    d.colstride = c.colstride;
    d.x_sb = c.x_sb; d.x_ss = c.x_ss; d.y_sb = c.y_sb; d.y_st = c.y_st;
    d.us_sr = c.us_sr; d.us_ss = c.us_ss; d.ut_sr = c.ut_sr; d.ut_st = c.ut_st;
    d.kh_sr = c.kh_sr; d.kh_sj = c.kh_sj; d.kw_sr = c.kw_sr; d.kw_sj = c.kw_sj;
    // one wavefront per SIMD (1024 on the chip); each segment recomputes
    // 2*CH rows of the chain above and below it
    const int64_t want = 1024;
    const int64_t strips = (int64_t)d.B * d.ncb;
    const int64_t segs = std::max<int64_t>(1, std::min<int64_t>(d.H, want / std::max<int64_t>(1, strips)));
    d.seg_rows = (int32_t)((d.H + segs - 1) / segs);
    d.segs = (int32_t)((d.H + d.seg_rows - 1) / d.seg_rows);
    d.waves = strips * d.segs;
    d.blocks = (d.waves + 3) / 4;
    if (d.blocks > 0x7fffffff) return false;
    cp_bwd_tables(d, dt == 1);
    if (d.lds_bytes > 160 * 1024) return false;

    const int64_t R = d.R, nb = d.blocks;
    const BufRef Pus = scratch.alloc((size_t)(nb * R * d.S) * 4);
    const BufRef Put = scratch.alloc((size_t)(nb * R * d.T) * 4);
    const BufRef Pkh = scratch.alloc((size_t)(nb * R * d.KH) * 4);
    const BufRef Pkw = scratch.alloc((size_t)(nb * R * d.KW) * 4);
    const BufRef us = f.b, kh = f.extra[0], kw = f.extra[1], ut = f.extra[2];
    auto din = [](const BufRef& in) {
        BufRef g;
        g.kind = BUF_DIN;
        g.index = in.index;
        return g;
    };
    Launch m;
    m.kind = K_CP_BWD | (dt << kBitIn) | (dt << kBitAux) | (dt << kBitOut);
    m.a = f.a;                      // X
    m.b.kind = BUF_DOUT;            // dY
    m.c = din(f.a);                 // dX (NULL when not wanted)
    m.extra = {us, kh, kw, ut, Pus, Put, Pkh, Pkw};
    m.grid[0] = (uint32_t)d.blocks;
    m.block[0] = 256;
    m.lds = d.lds_bytes;
    m.desc.resize(sizeof(d));
    std::memcpy(m.desc.data(), &d, sizeof(d));
    m.need = (1u << f.a.index) | (1u << us.index) | (1u << kh.index) | (1u << kw.index) | (1u << ut.index);
    m.what = "fused CP chain backward";
    m.kname = std::string("cp_bwd<") + (dt ? "unsigned short" : "float") + ", 3, 3, " +
              std::to_string(pad32(d.T) / 32) + ", " + std::to_string(pad32(d.S) / 32) +
              ((d.R == 32 && d.S == pad32(d.S) && d.T == pad32(d.T)) ? ", false>" : ", true>");
    // algorithmic bytes: X and dY read, dX written, factors read, partials written
    const double e = dt ? 2 : 4;
    const double act = (double)d.B * d.S * d.H * d.W;   // S = T
    m.alg_bytes = e * 3 * act + e * (double)R * (d.S + d.T + d.KH + d.KW) +
                  4.0 * (double)nb * R * (d.S + d.T + d.KH + d.KW);
    m.alg_flops = 2.0 * f.alg_flops;   // backward MACs are twice the forward's
    out.push_back(m);
    // the four factor gradients: ordered sums of the block partials, one launch
    MultiReduceDesc md;
    std::memset(&md, 0, sizeof(md));
    md.n = 4;
    const int64_t dims[4][4] = {{d.S, c.us_sr, c.us_ss, 0}, {d.T, c.ut_sr, c.ut_st, 0},
                                {d.KH, c.kh_sr, c.kh_sj, 0}, {d.KW, c.kw_sr, c.kw_sj, 0}};
    for (int j = 0; j < 4; j++) {
        ReduceDesc& rd = md.part[j];
        rd.M = (int32_t)R;
        rd.N = (int32_t)dims[j][0];
        rd.nsplit = nb;
        rd.sCm = dims[j][1];
        rd.sCn = dims[j][2];
        md.block0[j + 1] = md.block0[j] + (R * dims[j][0] + 63) / 64;
    }
    Launch lr;
    lr.kind = K_REDUCE_MULTI;
    lr.extra = {Pus, din(us), Put, din(ut), Pkh, din(kh), Pkw, din(kw)};
    lr.grid[0] = (uint32_t)md.block0[4];
    lr.block[0] = (uint32_t)(64 * reduce_waves(nb));
    lr.desc.resize(sizeof(md));
    std::memcpy(lr.desc.data(), &md, sizeof(md));
    lr.need = (1u << us.index) | (1u << ut.index) | (1u << kh.index) | (1u << kw.index);
    lr.what = "dUs, dUt, dKh, dKw: sums of block partials";
    lr.kname = "reduce_multi<" + std::to_string(reduce_waves(nb)) + ">";
    lr.alg_bytes = 4.0 * (double)nb * R * (d.S + d.T + d.KH + d.KW) + 4.0 * R * (d.S + d.T + d.KH + d.KW);
    out.push_back(lr);
    return true;
}

namespace {
}  // namespace

int fuse_launches(std::vector<Launch>& v, bool backward) {
    int n = 0;
    if (backward) return 0;
    for (size_t i = 0; i < v.size(); i++) {
        Launch f;
        if (match_cp_fwd(v, i, f)) {
            v.erase(v.begin() + i, v.begin() + i + 4);
            v.insert(v.begin() + i, f);
            n++;
        }
    }
    return n;
}

}  // namespace ce
