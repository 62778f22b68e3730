// Fusion of a contraction step with the convolution step that consumes its
// result, the pattern of the reshaped tensor-train layer (Appendix A.3 (3b)):
//   Z = X x F1   (contracts X's leading channel modes k with the merged
//                 leading cores, keeps X's remaining channel modes u, adds the
//                 cores' rank r and output modes g)
//   Y = Z (*) F2 (contracts u and r with the merged trailing core, convolves
//                 the two spatial labels, adds the output modes t)
// into one launch (K_TT_FWD, TtDesc), so Z is never written (Section 3.3:
// intermediates are the memory cost of the pairwise evaluation).
//
// The match works on the lowered pairwise ops, not on the string: every label
// of the two steps must fall in one of the classes below, each class a single
// linear index in every tensor that holds it.
#include <algorithm>
#include <cstring>
#include <string>
#include <vector>

#include "plan.h"

namespace ce {

namespace {

// One index class: its labels in a reference order, its size, and its
// element stride in a tensor (0 when the tensor lacks it); -1 when its labels'
// strides do not chain in that tensor.
struct LinIdx {
    std::vector<int> labels;
    int64_t size = 1;
};

int64_t lin_stride(const TensorRef& t, const LinIdx& c) {
    if (c.labels.empty()) return 0;
    // labels in the class's order must chain: stride(l_i) = stride(l_{i+1}) * dim(l_{i+1})
    for (size_t i = 0; i + 1 < c.labels.size(); i++) {
        const int a = c.labels[i], b = c.labels[i + 1];
        if (!t.has(a) || !t.has(b) || t.stride_of(a) != t.stride_of(b) * t.dim_of(b)) return -1;
    }
    if (!t.has(c.labels.back())) return -1;
    return t.stride_of(c.labels.back());
}

int64_t extent(const TensorRef& t) {
    int64_t e = 1;
    for (size_t i = 0; i < t.dims.size(); i++) e += (t.dims[i] - 1) * t.strides[i];
    return e;
}

bool same_buf(const BufRef& a, const BufRef& b) {
    return a.kind == b.kind && a.index == b.index && a.shift == b.shift;
}

}  // namespace

bool fuse_tt_forward(const PairOp& prod, const PairOp& cons, Launch& out) {
    if (!prod.has_r || !cons.has_r || !prod.convs.empty() || cons.convs.size() != 2) return false;
    if (prod.C.buf.kind != BUF_WS) return false;
    const TensorRef& Z = prod.C;
    int zside;
    if (same_buf(cons.L.buf, Z.buf)) zside = 0;
    else if (same_buf(cons.R.buf, Z.buf)) zside = 1;
    else return false;
    const TensorRef& F2 = zside == 0 ? cons.R : cons.L;
    const TensorRef& Y = cons.C;
    // convolved labels: Z the feature side, stride 1, zero 'same', 3 taps
    int lh = -1, lw = -1;
    for (const ConvMap& m : cons.convs) {
        const int aZ = zside == 0 ? m.aL : m.aR, bZ = zside == 0 ? m.bL : m.bR;
        const int aF = zside == 0 ? m.aR : m.aL, bF = zside == 0 ? m.bR : m.bL;
        const int64_t gZ = zside == 0 ? m.gL : m.gR, gF = zside == 0 ? m.gR : m.gL;
        const int64_t limZ = zside == 0 ? m.limL : m.limR, limF = zside == 0 ? m.limR : m.limL;
        if (m.modL || m.modR || aZ != 1 || bZ != 1 || gZ != -1 || aF != 0 || bF != 1 || gF != 0 ||
            m.J != 3 || limF != 3 || m.O != limZ)
            return false;
        if (Y.stride_of(m.label) == 1) lw = m.label;
        else lh = m.label;
    }
    if (lh < 0 || lw < 0) return false;
    // X: the operand of the first step holding the convolved labels
    int xside = -1;
    if (prod.L.has(lh) && prod.L.has(lw)) xside = 0;
    if (prod.R.has(lh) && prod.R.has(lw)) xside = xside < 0 ? 1 : -2;
    if (xside < 0) return false;
    const TensorRef& X = xside == 0 ? prod.L : prod.R;
    const TensorRef& F1 = xside == 0 ? prod.R : prod.L;
    if (F1.has(lh) || F1.has(lw)) return false;
    for (const TensorRef* t : {&X, &F1, &F2, &Y})
        if (t->dtype != DT_F32) return false;
    // planes dense in X and Y: w unit-stride, h of stride W
    const int64_t H = X.dim_of(lh), W = X.dim_of(lw);
    if (Z.dim_of(lh) != H || Z.dim_of(lw) != W || Y.dim_of(lh) != H || Y.dim_of(lw) != W) return false;
    if (X.stride_of(lw) != 1 || X.stride_of(lh) != W || Y.stride_of(lw) != 1 || Y.stride_of(lh) != W) return false;
    if (F2.dim_of(lh) != 3 || F2.dim_of(lw) != 3) return false;
    // classify the other labels by the tensors holding them
    LinIdx cb, ck, cu, cr, cg, ct;
    std::vector<int> all;
    for (const TensorRef* t : {&X, &F1, &Z, &F2, &Y})
        for (int l : t->labels)
            if (l != lh && l != lw && std::find(all.begin(), all.end(), l) == all.end()) all.push_back(l);
    for (int l : all) {
        const int m = (X.has(l) ? 1 : 0) | (F1.has(l) ? 2 : 0) | (Z.has(l) ? 4 : 0) | (F2.has(l) ? 8 : 0) |
                      (Y.has(l) ? 16 : 0);
        LinIdx* c = m == (1 | 4 | 16) ? &cb : m == (1 | 2) ? &ck : m == (1 | 4 | 8) ? &cu
                  : m == (2 | 4 | 8) ? &cr : m == (2 | 4 | 16) ? &cg : m == (8 | 16) ? &ct : nullptr;
        if (!c) return false;
        // sizes agree wherever the label is held
        int64_t dsz = -1;
        for (const TensorRef* t : {&X, &F1, &Z, &F2, &Y})
            if (t->has(l)) {
                if (dsz >= 0 && t->dim_of(l) != dsz) return false;
                dsz = t->dim_of(l);
            }
        c->labels.push_back(l);
        c->size *= dsz;
    }
    // reference order of each class: the order of its labels in the first
    // tensor that holds it (chaining is then checked in every holder)
    auto order_by = [](LinIdx& c, const TensorRef& t) {
        std::vector<int> o;
        for (int l : t.labels)
            if (std::find(c.labels.begin(), c.labels.end(), l) != c.labels.end()) o.push_back(l);
        c.labels = o;
    };
    order_by(cb, X);
    order_by(ck, X);
    order_by(cu, X);
    order_by(cr, F1);
    order_by(cg, F1);
    order_by(ct, F2);
    TtDesc d;
    std::memset(&d, 0, sizeof(d));
    const int64_t sx_b = lin_stride(X, cb), sy_b = lin_stride(Y, cb);
    const int64_t sx_k = lin_stride(X, ck), s1_k = lin_stride(F1, ck);
    const int64_t sx_u = lin_stride(X, cu), s2_u = lin_stride(F2, cu);
    const int64_t s1_r = lin_stride(F1, cr), s2_r = lin_stride(F2, cr);
    const int64_t s1_g = lin_stride(F1, cg), sy_g = lin_stride(Y, cg);
    const int64_t s2_t = lin_stride(F2, ct), sy_t = lin_stride(Y, ct);
    for (int64_t v : {sx_b, sy_b, sx_k, s1_k, sx_u, s2_u, s1_r, s2_r, s1_g, sy_g, s2_t, sy_t})
        if (v < 0) return false;
    if (cr.size != 16 || ct.size < 1 || ct.size > 8 || ck.size < 1 || ck.size > 64 || cu.size < 1 ||
        W > 64 || H < 1)
        return false;
    const int XT = W <= 16 ? 1 : W <= 32 ? 2 : 4;
    const int PW = 16 * XT + 2;
    const int plane = ((6 * PW - 16 + 63) / 64) * 64 + 16;
    d.B = (int32_t)cb.size;
    d.G = (int32_t)cg.size;
    d.K1 = (int32_t)ck.size;
    d.U = (int32_t)cu.size;
    d.R = 16;
    d.T = (int32_t)ct.size;
    d.H = (int32_t)H;
    d.W = (int32_t)W;
    d.TH = 4;
    d.nbands = (int32_t)((H + 3) / 4);
    d.XT = XT;
    d.PW = PW;
    d.plane = plane;
    d.ncombo = 2 * XT;
    d.x_sb = sx_b;
    d.x_sk = sx_k;
    d.x_su = sx_u;
    d.y_sb = sy_b;
    d.y_sg = sy_g;
    d.y_st = sy_t;
    d.f1_sg = s1_g;
    d.f1_sk = s1_k;
    d.f1_sr = s1_r;
    d.f2_st = s2_t;
    d.f2_su = s2_u;
    d.f2_sr = s2_r;
    d.f2_sh = F2.stride_of(lh);
    d.f2_sw = F2.stride_of(lw);
    d.x_numel = extent(X);
    d.f1_numel = extent(F1);
    d.f2_numel = extent(F2);
    if (d.x_numel >= (1ll << 29) || d.f1_numel >= (1ll << 29) || d.f2_numel >= (1ll << 29)) return false;
    d.blocks = (int64_t)d.B * d.G * d.nbands;
    if (d.blocks > 0x7fffffff || d.blocks < 1) return false;
    d.xcd_remap = (d.blocks % 8 == 0) ? 1u : 0u;
    d.lds_bytes = (uint32_t)(16 * plane * 4);
    out = Launch();
    out.kind = K_TT_FWD;
    out.a = X.buf;
    out.b = F1.buf;
    out.extra = {F2.buf};
    out.c = Y.buf;
    out.grid[0] = (uint32_t)d.blocks;
    out.block[0] = 256;
    out.lds = d.lds_bytes;
    out.desc.resize(sizeof(d));
    std::memcpy(out.desc.data(), &d, sizeof(d));
    const int n1 = (d.K1 + 3) / 4;
    const int ns1 = n1 <= 1 ? 1 : n1 <= 2 ? 2 : n1 <= 4 ? 4 : n1 <= 8 ? 8 : 16;
    out.kname = "tt_fwd<" + std::to_string(ns1) + ", " + std::to_string(XT) + ">";
    auto bytes = [](const TensorRef& t) { return (double)t.numel() * (t.dtype == DT_BF16 ? 2 : 4); };
    out.alg_bytes = bytes(X) + bytes(F1) + bytes(F2) + bytes(Y);
    out.alg_flops = 2.0 * ((double)prod.macs + (double)cons.macs);
    out.need = prod.need | cons.need;
    return true;
}

}  // namespace ce
