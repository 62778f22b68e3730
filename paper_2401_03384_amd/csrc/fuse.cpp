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
void cp_tables(CpDesc& d, bool bf) {
    d.lda = bf ? d.S + 8 : d.S + 1;
    size_t o = al16((size_t)32 * d.lda * (bf ? 2 : 4));
    d.o_ut = (uint32_t)o;
    o = al16(o + (bf ? (size_t)2 * 2 * d.T * 8 * 2 : (size_t)16 * 2 * d.T * 4));
    d.o_kh = (uint32_t)o;
    o += (size_t)16 * 2 * d.KH * 4;
    d.o_kw = (uint32_t)o;
    o += (size_t)16 * 2 * d.KW * 4;
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
    // register-resident strips: rank 32, T in {32, 64}, 3x3 or 5x5 filters
    if (R != 32 || !(T == 32 || T == 64) || S % 32 || h.K != w.K || !(h.K == 3 || h.K == 5))
        return false;
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
    // wavefronts: about two (fp32) or four (bf16) per SIMD of the 1024 SIMDs;
    // each strip segment recomputes KH-1 rows of Z1
    int64_t want = dt ? 4096 : 2048;
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
                  std::to_string(h.K) + ", " + std::to_string(w.K) + ", " + std::to_string(T / 32) + ">";
    fused.alg_bytes = g1.alg_bytes + d1.alg_bytes + d2.alg_bytes + g2.alg_bytes;
    fused.alg_flops = g1.alg_flops + d1.alg_flops + d2.alg_flops + g2.alg_flops;
    // algorithmic bytes of the fused launch: X, factors and Y only
    double e = dt ? 2 : 4;
    fused.alg_bytes = e * (double)(B * S * H * W + B * T * H * W + R * S + R * T + R * (h.K + w.K));
    return true;
}

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
