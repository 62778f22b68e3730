// Lowering of pairwise ops to specialised kernels.
//
// A pairwise op (Section 3.1: contraction, batch and outer-product labels,
// plus convolved labels) is matched against the label structures the fast
// kernels implement; anything else runs on the generic strided kernel.
//
//   channel-mixing GEMM   C[g][m][n] = sum_k F[g?][m][k] D[g][k][n], with the
//                         output's innermost labels (n) unit-stride in the large
//                         operand D and in C, absent from the small operand F
//   factor gradient       C[m][n] = sum_{kb,k} L[kb][m][k] R[kb][n][k], with the
//                         reduced labels k unit-stride in both operands
//   depthwise conv        one convolved label, a large operand with the layout
//                         of C, and a filter indexed by the conv label and by a
//                         run of C's labels ahead of the convolved axis
//   filter-tap gradient   the same structure with the filter as the result
//   general contraction   everything else with two operands, no self-contracted
//                         labels and at most two convolved labels: batch, row,
//                         column and reduction dims of any layout, convolved
//                         labels read with shifted, bounds-checked positions
#include <algorithm>
#include <cstring>

#include "plan.h"

namespace ce {
namespace {

double tensor_bytes(const TensorRef& t) {
    return (double)t.numel() * (t.dtype == DT_BF16 ? 2 : 4);
}

bool has(const std::vector<int>& v, int l) { return std::find(v.begin(), v.end(), l) != v.end(); }

// Labels `labs` (outer to inner) form one dimension of tensor t: strides chain.
// Returns size and innermost stride (size 1, stride 0 for an empty group).
bool merged(const TensorRef& t, const std::vector<int>& labs, int64_t& size, int64_t& stride) {
    size = 1;
    stride = 0;
    if (labs.empty()) return true;
    int64_t expect = -1;
    for (int k = (int)labs.size() - 1; k >= 0; --k) {
        int p = t.pos(labs[k]);
        if (p < 0) return false;
        if (k == (int)labs.size() - 1) {
            stride = t.strides[p];
            expect = stride * t.dims[p];
        } else {
            if (t.strides[p] != expect) return false;
            expect *= t.dims[p];
        }
        size *= t.dims[p];
    }
    return true;
}

struct BDim {
    int64_t size, s0, s1, s2;
};

// Merge neighbouring batch dims whose strides chain in all three tensors.
std::vector<BDim> merge_dims(std::vector<BDim> v) {
    for (size_t i = 0; i + 1 < v.size();) {
        BDim& a = v[i];
        BDim& b = v[i + 1];
        if (a.s0 == b.s0 * b.size && a.s1 == b.s1 * b.size && a.s2 == b.s2 * b.size) {
            a.size *= b.size;
            a.s0 = b.s0;
            a.s1 = b.s1;
            a.s2 = b.s2;
            v.erase(v.begin() + i + 1);
        } else {
            i++;
        }
    }
    return v;
}

int32_t dt_bits(DType in, DType aux, DType out) {
    return ((int32_t)in << kBitIn) | ((int32_t)aux << kBitAux) | ((int32_t)out << kBitOut);
}

template <typename D>
void set_desc(Launch& ln, const D& d) {
    ln.desc.resize(sizeof(D));
    std::memcpy(ln.desc.data(), &d, sizeof(D));
}

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Element type as it appears in the kernel's template arguments.
const char* tname(DType t) { return t == DT_BF16 ? "unsigned short" : "float"; }

// ---- channel-mixing GEMM -------------------------------------------------
bool try_gemm(const PairOp& op, std::vector<Launch>& out) {
    if (!op.convs.empty() || !op.has_r) return false;
    const TensorRef& C = op.C;
    for (int dside = 0; dside < 2; dside++) {
        const TensorRef& D = dside == 0 ? op.L : op.R;
        const TensorRef& F = dside == 0 ? op.R : op.L;
        const BufRef& dbuf = dside == 0 ? op.L.buf : op.R.buf;
        const BufRef& fbuf = dside == 0 ? op.R.buf : op.L.buf;
        if (D.dtype != F.dtype) continue;
        // n: innermost labels of C, unit-stride in C and D, not in F
        std::vector<int> ng;
        int64_t expect = 1;
        for (int k = (int)C.labels.size() - 1; k >= 0; --k) {
            int l = C.labels[k];
            if (!D.has(l) || F.has(l)) break;
            if (C.strides[k] != expect || D.stride_of(l) != expect) break;
            ng.insert(ng.begin(), l);
            expect *= C.dims[k];
        }
        if (ng.empty()) continue;
        int64_t N = expect;
        std::vector<int> mg, kg, gg;
        for (int l : C.labels)
            if (F.has(l) && !D.has(l)) mg.push_back(l);
        for (int l : D.labels)
            if (F.has(l) && !C.has(l)) kg.push_back(l);
        bool ok = true;
        for (int l : D.labels)
            if (!C.has(l) && !F.has(l)) ok = false;     // self-contracted in D
        for (int l : F.labels)
            if (!C.has(l) && !D.has(l)) ok = false;     // self-contracted in F
        std::vector<BDim> bd;
        for (int l : C.labels) {
            if (has(ng, l) || has(mg, l)) continue;
            if (!D.has(l)) { ok = false; break; }
            gg.push_back(l);
            bd.push_back({C.dim_of(l), F.stride_of(l), D.stride_of(l), C.stride_of(l)});
        }
        if (!ok) continue;
        int64_t M, sFm, sCm_unused, K, sFk, sDk, Mc;
        if (!merged(F, mg, M, sFm) || !merged(C, mg, Mc, sCm_unused)) continue;
        if (!merged(F, kg, K, sFk) || !merged(D, kg, K, sDk)) continue;
        int64_t sCm = 0, tmp;
        merged(C, mg, tmp, sCm);
        bd = merge_dims(bd);
        if (bd.size() > 3) continue;
        if (M > (1 << 20) || N > (int64_t)1 << 31 || K > (1 << 20)) continue;
        GemmDesc d;
        std::memset(&d, 0, sizeof(d));
        d.M = (int32_t)M;
        d.N = (int32_t)N;
        d.K = (int32_t)K;
        d.ng = (int32_t)bd.size();
        int64_t G = 1;
        for (size_t i = 0; i < bd.size(); i++) {
            d.g_size[i] = bd[i].size;
            d.g_sA[i] = bd[i].s0;
            d.g_sB[i] = bd[i].s1;
            d.g_sC[i] = bd[i].s2;
            G *= bd[i].size;
        }
        d.sAm = sFm;
        d.sAk = sFk;
        d.sBk = sDk;
        d.sCm = sCm;
        // few rows and few reduced channels: a column-streaming kernel, no tiles
        const int thinM = M <= 4 ? 4 : M <= 8 ? 8 : 16, thinK = K <= 4 ? 4 : K <= 8 ? 8 : 16;
        if (M <= 16 && K <= 16 && thinM * thinK <= 64 && N >= 16 && G * N < ((int64_t)1 << 31)) {
            d.mtiles = d.ntiles = 1;
            d.blocks = cdiv(G * N, 256);   // one column per thread
            Launch ln;
            ln.kind = K_THIN | dt_bits(D.dtype, F.dtype, C.dtype);
            ln.a = fbuf;
            ln.b = dbuf;
            ln.c = C.buf;
            ln.grid[0] = (uint32_t)d.blocks;
            ln.block[0] = 256;
            set_desc(ln, d);
            ln.kname = std::string("thin_gemm<") + tname(D.dtype) + ", " + tname(C.dtype) + ", " +
                       std::to_string(thinM) + ", " + std::to_string(thinK) + ">";
            out.push_back(ln);
            return true;
        }
        int MT = M > 32 ? 2 : 1;
        d.mtiles = (int32_t)cdiv(M, 32 * MT);
        d.ntiles = (int32_t)cdiv(N, 128);
        d.blocks = (int64_t)d.mtiles * d.ntiles * G;
        if (d.blocks > 0x7fffffff) continue;
        bool vec = (d.sBk % 4 == 0);
        for (int i = 0; i < d.ng; i++) vec = vec && (d.g_sB[i] % 4 == 0);
        // bf16 with 8-byte rows: tiles of 32 rows over the flattened (batch,
        // column) index
        const bool flat = D.dtype == DT_BF16 && vec && N % 4 == 0 && G * N < ((int64_t)1 << 31);
        if (flat) {
            const int64_t nt = cdiv(G * N, 128);
            MT = 1;
            d.mtiles = (int32_t)cdiv(M, 32 * MT);
            d.ntiles = (int32_t)nt;
            d.blocks = (int64_t)d.mtiles * d.ntiles;
        }
        Launch ln;
        ln.kind = K_GEMM | dt_bits(D.dtype, F.dtype, C.dtype) |
                  (((MT == 2 ? 1 : 0) | (vec ? 2 : 0) | (flat ? 4 : 0)) << kShiftOpt);
        ln.a = fbuf;
        ln.b = dbuf;
        ln.c = C.buf;
        ln.grid[0] = (uint32_t)d.blocks;
        ln.block[0] = 256;
        set_desc(ln, d);
        ln.kname = flat ? std::string("gemm_bf16f<") + tname(C.dtype) + (MT == 2 ? ", 2>" : ", 1>")
                        : std::string(D.dtype == DT_BF16 ? "gemm_bf16<" : "gemm_f32<") + tname(C.dtype) +
                              (MT == 2 ? ", 2, " : ", 1, ") + (vec ? "true>" : "false>");
        out.push_back(ln);
        return true;
    }
    return false;
}

// ---- factor gradient: split NT GEMM + ordered reduction ---------------------
bool try_wgrad(const PairOp& op, ScratchAlloc& scratch, std::vector<Launch>& out) {
    if (!op.convs.empty() || !op.has_r) return false;
    const TensorRef &L = op.L, &R = op.R, &C = op.C;
    if (L.dtype != R.dtype) return false;
    // k: innermost labels of L, unit-stride in L and R, reduced (not in C)
    std::vector<int> kg;
    int64_t expect = 1;
    for (int k = (int)L.labels.size() - 1; k >= 0; --k) {
        int l = L.labels[k];
        if (!R.has(l) || C.has(l)) break;
        if (L.strides[k] != expect || R.stride_of(l) != expect) break;
        kg.insert(kg.begin(), l);
        expect *= L.dims[k];
    }
    if (kg.empty()) return false;
    int64_t K = expect;
    std::vector<int> mg, ng;
    std::vector<BDim> kb;
    for (int l : C.labels) {
        bool inL = L.has(l), inR = R.has(l);
        if (inL && inR) return false;          // batch labels: not this kernel
        if (inL) mg.push_back(l);
        else if (inR) ng.push_back(l);
        else return false;
    }
    for (int l : L.labels) {
        if (C.has(l) || has(kg, l)) continue;
        if (!R.has(l)) return false;           // self-contracted
        kb.push_back({L.dim_of(l), L.stride_of(l), R.stride_of(l), 0});
    }
    for (int l : R.labels)
        if (!C.has(l) && !L.has(l)) return false;
    int64_t M, sAm, N, sBn, tmp, sCm, sCn;
    if (!merged(L, mg, M, sAm) || !merged(C, mg, tmp, sCm)) return false;
    if (!merged(R, ng, N, sBn) || !merged(C, ng, tmp, sCn)) return false;
    kb = merge_dims(kb);
    if (kb.size() > 3) return false;
    if (K < 64 || M > 4096 || N > 4096) return false;
    WgradDesc d;
    std::memset(&d, 0, sizeof(d));
    d.M = (int32_t)M;
    d.N = (int32_t)N;
    d.K = K;
    d.nkb = (int32_t)kb.size();
    int64_t KB = 1;
    for (size_t i = 0; i < kb.size(); i++) {
        d.kb_size[i] = kb[i].size;
        d.kb_sA[i] = kb[i].s0;
        d.kb_sB[i] = kb[i].s1;
        KB *= kb[i].size;
    }
    d.sAm = sAm;
    d.sBn = sBn;
    d.mtiles = (int32_t)cdiv(M, 64);
    d.ntiles = (int32_t)cdiv(N, 64);
    int64_t tiles = (int64_t)d.mtiles * d.ntiles;
    // aim at ~512 blocks (two per CU): few partials to reduce, long chunks;
    // chunks are multiples of the 32-element tile
    int64_t want = std::max<int64_t>(1, cdiv(512, KB * tiles));
    int64_t kchunk = std::max<int64_t>(32, cdiv(cdiv(K, want), 32) * 32);
    d.kchunk = (int32_t)std::min<int64_t>(kchunk, (int64_t)1 << 30);
    d.ksplit = (int32_t)cdiv(K, d.kchunk);
    d.nsplit = KB * d.ksplit;
    d.blocks = d.nsplit * tiles;
    if (d.blocks > 0x7fffffff || d.nsplit * M * N > ((int64_t)1 << 31)) return false;
    bool vec = (d.sAm % 4 == 0) && (d.sBn % 4 == 0) && (d.kchunk % 4 == 0);
    for (int i = 0; i < d.nkb; i++) vec = vec && (d.kb_sA[i] % 4 == 0) && (d.kb_sB[i] % 4 == 0);
    BufRef part = scratch.alloc((size_t)(d.nsplit * M * N * 4));
    Launch ln;
    ln.kind = K_WGRAD | dt_bits(L.dtype, R.dtype, DT_F32) | ((vec ? 2 : 0) << kShiftOpt);
    ln.a = L.buf;
    ln.b = R.buf;
    ln.d = part;
    ln.grid[0] = (uint32_t)d.blocks;
    ln.block[0] = 256;
    set_desc(ln, d);
    ln.kname = std::string("wgrad<") + tname(L.dtype) + (vec ? ", true>" : ", false>");
    out.push_back(ln);
    ReduceDesc rd;
    std::memset(&rd, 0, sizeof(rd));
    rd.M = (int32_t)M;
    rd.N = (int32_t)N;
    rd.nsplit = d.nsplit;
    rd.sCm = sCm;
    rd.sCn = sCn;
    Launch lr;
    lr.kind = K_REDUCE | dt_bits(DT_F32, DT_F32, C.dtype);
    lr.d = part;
    lr.c = C.buf;
    lr.grid[0] = (uint32_t)cdiv(M * N, 64);
    lr.block[0] = (uint32_t)(64 * reduce_waves(rd.nsplit));
    set_desc(lr, rd);
    lr.kname = "reduce_partials<" + std::to_string(reduce_waves(rd.nsplit)) + ", " + tname(C.dtype) + ">";
    out.push_back(lr);
    return true;
}

// ---- depthwise convolution along one axis --------------------------------
// View of a dense tensor t around its label `axis`: [slabs][A][inner].
struct AxisView {
    int pos;
    int64_t nslab, A, inner;
};

bool axis_view(const TensorRef& t, int axis, AxisView& v) {
    v.pos = t.pos(axis);
    if (v.pos < 0) return false;
    v.nslab = 1;
    v.inner = 1;
    for (int k = 0; k < v.pos; k++) v.nslab *= t.dims[k];
    for (int k = v.pos + 1; k < (int)t.dims.size(); k++) v.inner *= t.dims[k];
    v.A = t.dims[v.pos];
    // dense row-major
    int64_t s = 1;
    for (int k = (int)t.dims.size() - 1; k >= 0; --k) {
        if (t.strides[k] != s) return false;
        s *= t.dims[k];
    }
    return true;
}

bool same_layout(const TensorRef& a, const TensorRef& b) {
    return a.labels == b.labels && a.dims == b.dims && a.strides == b.strides;
}

// Filter-row labels: the labels of `filt` other than the axis must be a run of
// `big`'s labels ahead of the axis, mergeable in `filt`.
bool filter_rows(const TensorRef& big, const TensorRef& filt, int axis, const AxisView& v,
                 int64_t& r_div, int64_t& r_size, int64_t& r_stride) {
    std::vector<int> run;
    for (int l : filt.labels)
        if (l != axis) run.push_back(l);
    r_size = 1;
    r_div = 1;
    r_stride = 0;
    if (run.empty()) {
        r_div = 1;
        return true;
    }
    // order the run by its positions in `big` (must be consecutive, before the axis)
    std::vector<int> pos;
    for (int l : run) {
        int p = big.pos(l);
        if (p < 0 || p >= v.pos) return false;
        pos.push_back(p);
    }
    std::sort(pos.begin(), pos.end());
    for (size_t i = 1; i < pos.size(); i++)
        if (pos[i] != pos[i - 1] + 1) return false;
    std::vector<int> ordered;
    for (int p : pos) ordered.push_back(big.labels[p]);
    int64_t sz, st;
    if (!merged(filt, ordered, sz, st)) return false;
    r_size = sz;
    r_stride = st;
    r_div = 1;
    for (int k = pos.back() + 1; k < v.pos; k++) r_div *= big.dims[k];
    return true;
}

int64_t choose_spb(int64_t r_div, int64_t slabsz) {
    int64_t best = 1;
    for (int64_t d = 1; d <= std::min<int64_t>(r_div, 256); d++)
        if (r_div % d == 0 && d * slabsz <= 4096) best = d;
    return best;
}

bool try_dw(const PairOp& op, ScratchAlloc& scratch, std::vector<Launch>& out) {
    if (op.convs.size() != 1 || !op.has_r) return false;
    const ConvMap& cm = op.convs[0];
    const int axis = cm.label;
    // (a) forward / transposed: the large operand has C's layout
    for (int side = 0; side < 2; side++) {
        const TensorRef& X = side == 0 ? op.L : op.R;
        const TensorRef& Fl = side == 0 ? op.R : op.L;
        int aX = side == 0 ? cm.aL : cm.aR, bX = side == 0 ? cm.bL : cm.bR;
        int64_t gX = side == 0 ? cm.gL : cm.gR;
        int aF = side == 0 ? cm.aR : cm.aL, bF = side == 0 ? cm.bR : cm.bL;
        int64_t gF = side == 0 ? cm.gR : cm.gL;
        if (!same_layout(X, op.C)) continue;
        if (!(aX == 1 && (bX == 1 || bX == -1) && aF == 0 && bF == 1 && gF == 0)) continue;
        AxisView v;
        if (!axis_view(X, axis, v)) continue;
        if (cm.O != v.A || cm.J > 7 || cm.J < 1) continue;
        if (Fl.dim_of(axis) != cm.J) continue;
        int64_t r_div, r_size, r_stride;
        if (!filter_rows(X, Fl, axis, v, r_div, r_size, r_stride)) continue;
        int64_t slabsz = v.A * v.inner;
        if (slabsz > 4096) continue;
        DwDesc d;
        std::memset(&d, 0, sizeof(d));
        d.nslab = v.nslab;
        d.A = (int32_t)v.A;
        d.inner = (int32_t)v.inner;
        d.K = (int32_t)cm.J;
        d.sign = bX;
        d.off = (int32_t)gX;
        d.spb = (int32_t)choose_spb(r_div, slabsz);
        d.r_div = r_div;
        d.r_size = r_size;
        d.r_stride = r_stride;
        d.f_sj = Fl.stride_of(axis);
        d.nblocks = cdiv(d.nslab, d.spb);
        if (d.nblocks > 0x7fffffff) continue;
        Launch ln;
        ln.kind = K_DW | dt_bits(X.dtype, Fl.dtype, op.C.dtype);
        ln.a = X.buf;
        ln.b = Fl.buf;
        ln.c = op.C.buf;
        ln.grid[0] = (uint32_t)d.nblocks;
        ln.block[0] = 256;
        set_desc(ln, d);
        ln.kname = std::string("dw_conv<") + tname(X.dtype) + ", " + tname(Fl.dtype) + ", " +
                   tname(op.C.dtype) + ", " + std::to_string(d.K) + ">";
        out.push_back(ln);
        return true;
    }
    // (b) filter-tap gradient: C is the filter; feature and gradient share a layout
    for (int side = 0; side < 2; side++) {
        const TensorRef& Xf = side == 0 ? op.L : op.R;   // feature (read at p + j + off)
        const TensorRef& Xg = side == 0 ? op.R : op.L;   // output gradient (read at p)
        int aF = side == 0 ? cm.aL : cm.aR, bF = side == 0 ? cm.bL : cm.bR;
        int64_t gF = side == 0 ? cm.gL : cm.gR;
        int aG = side == 0 ? cm.aR : cm.aL, bG = side == 0 ? cm.bR : cm.bL;
        int64_t gG = side == 0 ? cm.gR : cm.gL;
        if (!same_layout(Xf, Xg) || Xf.dtype != Xg.dtype) continue;
        if (!(aF == 1 && bF == 1 && aG == 0 && bG == 1 && gG == 0)) continue;
        AxisView v;
        if (!axis_view(Xf, axis, v)) continue;
        if (cm.J != v.A || cm.O > 7 || cm.O < 1 || op.C.dim_of(axis) != cm.O) continue;
        int64_t r_div, r_size, r_stride;
        if (!filter_rows(Xf, op.C, axis, v, r_div, r_size, r_stride)) continue;
        int64_t slabsz = v.A * v.inner;
        if (slabsz > 4096) continue;
        DwDesc d;
        std::memset(&d, 0, sizeof(d));
        d.nslab = v.nslab;
        d.A = (int32_t)v.A;
        d.inner = (int32_t)v.inner;
        d.K = (int32_t)cm.O;
        d.sign = 1;
        d.off = (int32_t)gF;
        d.spb = (int32_t)choose_spb(r_div, slabsz);
        d.r_div = r_div;
        d.r_size = r_size;
        d.r_stride = r_stride;
        d.nblocks = cdiv(d.nslab, d.spb);
        d.o_sr = r_stride;
        d.o_sj = op.C.stride_of(axis);
        if (d.nblocks > 0x7fffffff || d.nslab % d.spb) continue;
        BufRef part = scratch.alloc((size_t)(d.nblocks * d.K * 4));
        Launch ln;
        ln.kind = K_DW_TAPGRAD | dt_bits(Xf.dtype, Xg.dtype, DT_F32);
        ln.a = Xf.buf;
        ln.b = Xg.buf;
        ln.d = part;
        ln.grid[0] = (uint32_t)d.nblocks;
        ln.block[0] = 256;
        set_desc(ln, d);
        ln.kname = std::string("dw_tapgrad<") + tname(Xf.dtype) + ", " + std::to_string(d.K) + ">";
        out.push_back(ln);
        Launch lr;
        lr.kind = K_DW_TAPREDUCE | dt_bits(DT_F32, DT_F32, op.C.dtype);
        lr.d = part;
        lr.c = op.C.buf;
        lr.grid[0] = (uint32_t)d.r_size;
        lr.block[0] = 256;
        set_desc(lr, d);
        lr.kname = std::string("dw_tapreduce<") + tname(op.C.dtype) + ", " + std::to_string(d.K) + ">";
        out.push_back(lr);
        return true;
    }
    return false;
}


// ---- small output per batch index, long reduction ---------------------------
//   C[g][m][n] = sum_k P[g][m][k] Q[g][n][k], M, N <= 16, k with an inner run
// contiguous in both operands: a streaming kernel plus an ordered chunk sum.
bool try_thinw(const PairOp& op, ScratchAlloc& scratch, std::vector<Launch>& out) {
    if (!op.has_r || !op.convs.empty() || op.L.dtype != op.R.dtype) return false;
    const TensorRef &P = op.L, &Q = op.R, &C = op.C;
    struct Dm {
        int64_t size, sP, sQ, sC;
    };
    std::vector<Dm> G, Ko;
    std::vector<int> ponly, qonly;   // C's labels held by one operand, in C's order
    for (size_t k = 0; k < C.labels.size(); k++) {
        const int l = C.labels[k];
        const bool inP = P.has(l), inQ = Q.has(l);
        if (inP && inQ) G.push_back({C.dims[k], P.stride_of(l), Q.stride_of(l), C.strides[k]});
        else if (inP) ponly.push_back(l);
        else if (inQ) qonly.push_back(l);
        else return false;
    }
    // the innermost one-sided label of at most 16 becomes m (n); the rest are batch dims
    auto pick = [&](std::vector<int>& only, const TensorRef& T, bool isP, int64_t& size, int64_t& sT,
                    int64_t& sC) {
        size = 1;
        sT = sC = 0;
        int sel = -1;
        for (int i = (int)only.size() - 1; i >= 0; --i)
            if (T.dim_of(only[i]) <= 16) {
                sel = i;
                break;
            }
        if (!only.empty() && sel < 0) return false;
        for (int i = 0; i < (int)only.size(); i++) {
            const int l = only[i];
            if (i == sel) {
                size = T.dim_of(l);
                sT = T.stride_of(l);
                sC = C.stride_of(l);
            } else {
                G.push_back({T.dim_of(l), isP ? T.stride_of(l) : 0, isP ? 0 : T.stride_of(l), C.stride_of(l)});
            }
        }
        return true;
    };
    int64_t M, N, sPm, sQn, sCm, sCn;
    if (!pick(ponly, P, true, M, sPm, sCm) || !pick(qonly, Q, false, N, sQn, sCn)) return false;
    const int MM = M <= 4 ? 4 : M <= 8 ? 8 : 16, NN = N <= 4 ? 4 : N <= 8 ? 8 : 16;
    if (MM * NN > 64) return false;
    for (size_t k = 0; k < P.labels.size(); k++) {   // reduced labels in P's order
        const int l = P.labels[k];
        if (C.has(l)) continue;
        if (!Q.has(l)) return false;
        Ko.push_back({P.dims[k], P.strides[k], Q.stride_of(l), 0});
    }
    for (int l : Q.labels)
        if (!C.has(l) && !P.has(l)) return false;
    auto merge = [](std::vector<Dm>& v) {
        for (size_t i = 0; i + 1 < v.size();) {
            Dm& a = v[i];
            const Dm& b = v[i + 1];
            if (a.sP == b.sP * b.size && a.sQ == b.sQ * b.size && a.sC == b.sC * b.size) {
                a.size *= b.size;
                a.sP = b.sP;
                a.sQ = b.sQ;
                a.sC = b.sC;
                v.erase(v.begin() + i + 1);
            } else {
                i++;
            }
        }
    };
    merge(G);
    merge(Ko);
    if (Ko.empty() || Ko.back().sP != 1 || Ko.back().sQ != 1) return false;
    const int64_t Kin = Ko.back().size;
    Ko.pop_back();
    if (Kin < 16 || G.size() > 3 || Ko.size() > 3) return false;
    ThinwDesc d;
    std::memset(&d, 0, sizeof(d));
    d.ng = (int32_t)G.size();
    d.no = (int32_t)Ko.size();
    d.M = (int32_t)M;
    d.N = (int32_t)N;
    d.G = 1;
    for (size_t i = 0; i < G.size(); i++) {
        d.g_size[i] = G[i].size;
        d.g_sP[i] = G[i].sP;
        d.g_sQ[i] = G[i].sQ;
        d.g_sC[i] = G[i].sC;
        d.G *= G[i].size;
    }
    d.Kout = 1;
    for (size_t i = 0; i < Ko.size(); i++) {
        d.o_size[i] = Ko[i].size;
        d.o_sP[i] = Ko[i].sP;
        d.o_sQ[i] = Ko[i].sQ;
        d.Kout *= Ko[i].size;
    }
    d.Kin = Kin;
    d.sPm = sPm;
    d.sQn = sQn;
    d.sCm = sCm;
    d.sCn = sCn;
    // enough reduction per g to be worth a stream, at least 32 elements per thread
    if (d.Kout * Kin < 16384) return false;
    const int64_t maxrows = std::min<int64_t>(512, ((int64_t)1 << 30) / Kin);
    int64_t chunks = std::max<int64_t>(1, cdiv(2048, d.G));
    chunks = std::min(chunks, std::max<int64_t>(1, d.Kout * Kin / (256 * 32)));
    d.orows = std::min(cdiv(d.Kout, chunks), maxrows);
    if (d.orows < 1) return false;
    d.kchunks = cdiv(d.Kout, d.orows);
    d.blocks = d.G * d.kchunks;
    if (d.blocks > 0x7fffffff) return false;
    const std::string shape = std::to_string(MM) + ", " + std::to_string(NN) + ">";
    const BufRef part = scratch.alloc((size_t)(d.blocks * MM * NN * 4));
    Launch ln;
    ln.kind = K_THINW | dt_bits(P.dtype, P.dtype, DT_F32);
    ln.a = P.buf;
    ln.b = Q.buf;
    ln.d = part;
    ln.grid[0] = (uint32_t)d.blocks;
    ln.block[0] = 256;
    set_desc(ln, d);
    ln.kname = std::string("thinw<") + tname(P.dtype) + ", " + shape;
    out.push_back(ln);
    Launch lr;
    lr.kind = K_THINW_REDUCE | dt_bits(DT_F32, DT_F32, C.dtype);
    lr.d = part;
    lr.c = C.buf;
    lr.grid[0] = (uint32_t)cdiv(d.G * M * N, 256);
    lr.block[0] = 256;
    set_desc(lr, d);
    lr.kname = std::string("thinw_reduce<") + tname(C.dtype) + ", " + shape;
    out.push_back(lr);
    return true;
}

// ---- plane convolution contracted over one index ---------------------------
//   C[u][m][p] = sum_s sum_j Z[u][s][p + j - c] * O[m][s][j],  M <= 16
// Forward (p = output pixels, j = taps) runs as K_CRED; the filter gradient
// (p = taps, j = pixels) as K_CREDW plus an ordered chunk sum.
bool try_cred(const PairOp& op, ScratchAlloc& scratch, std::vector<Launch>& out) {
    if (!op.has_r || op.convs.size() != 2 || op.L.dtype != op.R.dtype) return false;
    const int zside = op.convs[0].aL != 0 ? 0 : 1;
    const TensorRef& Z = zside == 0 ? op.L : op.R;
    const TensorRef& O = zside == 0 ? op.R : op.L;
    const TensorRef& C = op.C;
    struct Cv {
        int label;
        int64_t O, J, g, limZ, limO;
    } cv[2];
    for (int k = 0; k < 2; k++) {
        const ConvMap& cm = op.convs[k];
        const int aZ = zside == 0 ? cm.aL : cm.aR, bZ = zside == 0 ? cm.bL : cm.bR;
        const int aO = zside == 0 ? cm.aR : cm.aL, bO = zside == 0 ? cm.bR : cm.bL;
        const int64_t gO = zside == 0 ? cm.gR : cm.gL;
        if (aZ != 1 || bZ != 1 || aO != 0 || bO != 1 || gO != 0) return false;
        cv[k] = {cm.label, cm.O, cm.J, zside == 0 ? cm.gL : cm.gR, zside == 0 ? cm.limL : cm.limR,
                 zside == 0 ? cm.limR : cm.limL};
        if (cv[k].limO < cm.J || !Z.has(cm.label) || !O.has(cm.label) || !C.has(cm.label)) return false;
    }
    // w: the convolved label with unit stride in Z
    if (Z.stride_of(cv[0].label) == 1) std::swap(cv[0], cv[1]);
    const Cv& ch = cv[0];
    const Cv& cw = cv[1];
    if (Z.stride_of(cw.label) != 1 || Z.stride_of(ch.label) != cw.limZ) return false;
    const bool wgrad = ch.O < ch.J;   // p over taps, j over the plane
    const int64_t H = ch.limZ, W = cw.limZ;
    const int64_t KH = wgrad ? ch.O : ch.J, KW = wgrad ? cw.O : cw.J;
    if ((wgrad ? ch.J : ch.O) != H || (wgrad ? cw.J : cw.O) != W) return false;
    const int64_t pch = -ch.g, pcw = -cw.g;
    if (pch < 0 || pch >= KH || pcw < 0 || pcw >= KW) return false;
    const bool kok = (KH == KW && (KH == 3 || KH == 5 || KH == 7)) || (KH == 1 && KW == 3) ||
                     (KH == 3 && KW == 1);
    if (!kok || (wgrad && KH * KW > 25)) return false;   // gradient taps live in registers
    // the plane of the output (forward) or of O (gradient) is dense as well
    const TensorRef& P = wgrad ? O : C;
    if (P.stride_of(cw.label) != 1 || P.stride_of(ch.label) != W) return false;
    if (wgrad && (ch.limO != H || cw.limO != W)) return false;
    auto is_conv = [&](int l) { return l == ch.label || l == cw.label; };
    struct Dm {
        int64_t size, s1, s2;
    };
    auto merge = [](std::vector<Dm>& v) {
        for (size_t i = 0; i + 1 < v.size();) {
            if (v[i].s1 == v[i + 1].s1 * v[i + 1].size && v[i].s2 == v[i + 1].s2 * v[i + 1].size) {
                v[i].size *= v[i + 1].size;
                v[i].s1 = v[i + 1].s1;
                v[i].s2 = v[i + 1].s2;
                v.erase(v.begin() + i + 1);
            } else {
                i++;
            }
        }
    };
    // u: C's labels in Z only; m: C's labels in O only (strides in O, C);
    // s: the reduced ones (in Z and O)
    std::vector<Dm> U, S, Mv;
    for (size_t k = 0; k < C.labels.size(); k++) {
        const int l = C.labels[k];
        if (is_conv(l)) continue;
        const bool inZ = Z.has(l), inO = O.has(l);
        if (inZ && !inO) U.push_back({C.dims[k], Z.stride_of(l), C.strides[k]});
        else if (inO && !inZ) Mv.push_back({C.dims[k], O.stride_of(l), C.strides[k]});
        else return false;
    }
    for (size_t k = 0; k < Z.labels.size(); k++) {
        const int l = Z.labels[k];
        if (is_conv(l) || C.has(l)) continue;
        if (!O.has(l)) return false;
        S.push_back({Z.dims[k], Z.strides[k], O.stride_of(l)});
    }
    for (int l : O.labels)
        if (!is_conv(l) && !C.has(l) && !Z.has(l)) return false;
    merge(U);
    merge(S);
    merge(Mv);
    // the batch dims (forward: u, gradient: s) and the single rank dim
    std::vector<Dm>& Bd = wgrad ? S : U;
    std::vector<Dm>& Rd = wgrad ? U : S;
    if (Bd.size() > 2 || Rd.size() > 1 || Mv.size() > 1) return false;
    const int64_t M = Mv.empty() ? 1 : Mv[0].size;
    if (wgrad && Z.dtype == O.dtype) {
        // filter gradient on fp32 MFMA tiles: rows u in blocks of 64 rt, the
        // columns (m, tap) in blocks of 16 nct (each block stages the planes
        // of O its columns read), the batch split into about two blocks a CU
        const bool bf = Z.dtype == DT_BF16;
        const int64_t N = M * KH * KW, KK = KH * KW;
        CredDesc d;
        std::memset(&d, 0, sizeof(d));
        d.H = (int32_t)H;
        d.W = (int32_t)W;
        d.KH = (int32_t)KH;
        d.KW = (int32_t)KW;
        d.ch = (int32_t)pch;
        d.cw = (int32_t)pcw;
        d.M = (int32_t)M;
        d.o_sm = Mv.empty() ? 0 : Mv[0].s1;
        d.c_sm = Mv.empty() ? 0 : Mv[0].s2;
        d.PH = (int32_t)(H + KH - 1);
        d.PWp = (int32_t)(W + KW - 1);
        d.ng = (int32_t)Bd.size();
        d.G = 1;
        for (size_t i = 0; i < Bd.size(); i++) {
            d.g_size[i] = Bd[i].size;
            d.g_sZ[i] = Bd[i].s1;
            d.g_sY[i] = Bd[i].s2;
            d.G *= Bd[i].size;
        }
        d.R = Rd.empty() ? 1 : Rd[0].size;
        d.z_sr = Rd.empty() ? 0 : Rd[0].s1;
        d.c_sr = Rd.empty() ? 0 : Rd[0].s2;
        d.c_sh = C.stride_of(ch.label);
        d.c_sw = C.stride_of(cw.label);
        d.rt = (bf && d.R <= 64) ? 1 : 2;
        d.nct = bf ? (N <= 48 ? 3 : 6) : (int32_t)std::min<int64_t>(6, cdiv(N, 16));
        d.ncb = (int32_t)cdiv(N, 16 * d.nct);
        d.mb = 1;
        for (int64_t cb = 0; cb < d.ncb; cb++) {
            const int64_t n0 = cb * 16 * d.nct, mlo = n0 / KK, mhi = std::min<int64_t>(M, (n0 + 16 * d.nct - 1) / KK + 1);
            d.mb = (int32_t)std::max<int64_t>(d.mb, mhi - mlo);
        }
        d.nrb = cdiv(d.R, 64 * d.rt);
        const int64_t chunks = std::max<int64_t>(1, std::min<int64_t>(d.G, cdiv(512, d.nrb * d.ncb)));
        d.gchunk = cdiv(d.G, chunks);
        d.nchunks = cdiv(d.G, d.gchunk);
        d.blocks = d.nrb * d.ncb * d.nchunks;
        d.threads = 256;
        const int64_t lds = 2 * (int64_t)d.mb * d.PH * d.PWp * 4;
        int64_t zext = 1;
        for (size_t i = 0; i < Z.dims.size(); i++) zext += (Z.dims[i] - 1) * Z.strides[i];
        d.zext = zext;
        const bool zfits = zext * (bf ? 2 : 4) < ((int64_t)1 << 31);   // 32-bit buffer offsets
        if (zfits && lds <= 160 * 1024 && d.blocks <= 0x7fffffff && H * W * M < ((int64_t)1 << 30)) {
            d.lds_bytes = (uint32_t)lds;
            const BufRef part = scratch.alloc((size_t)(d.nchunks * d.R * N * 4));
            Launch ln;
            ln.kind = K_WGCONV | dt_bits(Z.dtype, Z.dtype, DT_F32);
            ln.a = Z.buf;
            ln.b = O.buf;
            ln.d = part;
            ln.grid[0] = (uint32_t)d.blocks;
            ln.block[0] = 256;
            ln.lds = d.lds_bytes;
            set_desc(ln, d);
            ln.kname = std::string("wgconv<") + tname(Z.dtype) + ", " + std::to_string(d.rt) + ", " +
                       std::to_string(d.nct) + ">";
            out.push_back(ln);
            Launch lr;
            lr.kind = K_CREDW_REDUCE | dt_bits(DT_F32, DT_F32, C.dtype);
            lr.d = part;
            lr.c = C.buf;
            lr.grid[0] = (uint32_t)cdiv(d.R * N, 64);   // 64 outputs per block
            lr.block[0] = 256;
            set_desc(lr, d);
            lr.kname = std::string("credw_reduce<") + tname(C.dtype) + ">";
            out.push_back(lr);
            return true;
        }
    }
    const int MO = M == 1 ? 1 : M <= 4 ? 4 : M <= 8 ? 8 : 16;
    if (M > 16 || (wgrad && (MO > 8 || MO * KH * KW > 72))) return false;
    CredDesc d;
    std::memset(&d, 0, sizeof(d));
    d.H = (int32_t)H;
    d.W = (int32_t)W;
    d.KH = (int32_t)KH;
    d.KW = (int32_t)KW;
    d.ch = (int32_t)pch;
    d.cw = (int32_t)pcw;
    d.M = (int32_t)M;
    d.o_sm = Mv.empty() ? 0 : Mv[0].s1;
    d.wchunks = (int32_t)cdiv(W, 4);
    d.items = (int32_t)(H * d.wchunks);
    const int maxthreads = wgrad && MO >= 4 ? 512 : 1024;
    if (d.items > maxthreads) return false;
    const int n4 = (int)cdiv(4 + KW - 1, 4);
    d.PH = (int32_t)(H + KH - 1);
    d.PWp = (int32_t)(cdiv(std::max<int64_t>(W + KW - 1, 4 * (d.wchunks - 1) + 4 * n4), 4) * 4);
    d.ng = (int32_t)Bd.size();
    d.G = 1;
    for (size_t i = 0; i < Bd.size(); i++) {
        d.g_size[i] = Bd[i].size;
        d.g_sZ[i] = Bd[i].s1;
        d.g_sY[i] = Bd[i].s2;
        d.G *= Bd[i].size;
    }
    d.R = Rd.empty() ? 1 : Rd[0].size;
    d.z_sr = Rd.empty() ? 0 : Rd[0].s1;
    const int64_t plane = (int64_t)d.PH * d.PWp;
    const int maxper = maxthreads / d.items;
    if (!wgrad) {
        if (C.dtype != Z.dtype) return false;
        d.f_sr = Rd.empty() ? 0 : Rd[0].s2;
        d.f_sh = O.stride_of(ch.label);
        d.f_sw = O.stride_of(cw.label);
        d.y_sm = Mv.empty() ? 0 : Mv[0].s2;
        // batch indices per block: enough blocks to fill the chip first
        d.per = (int32_t)std::max<int64_t>(1, std::min<int64_t>(maxper, d.G / 1024));
        while (d.per > 1 && 2 * d.per * plane * 4 > 64 * 1024) d.per--;
        d.blocks = cdiv(d.G, d.per);
    } else {
        d.c_sm = Mv.empty() ? 0 : Mv[0].s2;
        d.c_sr = Rd.empty() ? 0 : Rd[0].s2;
        d.c_sh = C.stride_of(ch.label);
        d.c_sw = C.stride_of(cw.label);
        // ranks per block: the largest divisor of R that fits the block
        int64_t per = std::min<int64_t>(maxper, d.R);
        while (per > 1 && d.R % per) per--;
        while (per > 1 && 2 * per * plane * 4 > 96 * 1024) per--;
        d.per = (int32_t)per;
        d.nrb = cdiv(d.R, per);
        const int64_t chunks = std::max<int64_t>(1, std::min<int64_t>(d.G, cdiv(1024, d.nrb)));
        d.gchunk = cdiv(d.G, chunks);
        d.nchunks = cdiv(d.G, d.gchunk);
        d.blocks = d.nrb * d.nchunks;
    }
    if (d.blocks > 0x7fffffff) return false;
    d.threads = (uint32_t)(cdiv((int64_t)d.per * d.items, 64) * 64);
    int64_t lds = 2 * (int64_t)d.per * plane * 4;
    if (wgrad) lds = std::max<int64_t>(lds, (int64_t)d.threads * KH * KW * 4);
    if (lds > 160 * 1024) return false;
    d.lds_bytes = (uint32_t)lds;
    const std::string shape = std::to_string(KH) + ", " + std::to_string(KW) + ", " + std::to_string(MO) + ">";
    Launch ln;
    ln.grid[0] = (uint32_t)d.blocks;
    ln.block[0] = d.threads;
    ln.lds = d.lds_bytes;
    if (!wgrad) {
        ln.kind = K_CRED | dt_bits(Z.dtype, Z.dtype, C.dtype);
        ln.a = O.buf;
        ln.b = Z.buf;
        ln.c = C.buf;
        set_desc(ln, d);
        ln.kname = std::string("cred<") + tname(Z.dtype) + ", " + shape;
        out.push_back(ln);
        return true;
    }
    const BufRef part = scratch.alloc((size_t)(d.nchunks * d.R * M * KH * KW * 4));
    ln.kind = K_CREDW | dt_bits(Z.dtype, Z.dtype, DT_F32);
    ln.a = Z.buf;
    ln.b = O.buf;
    ln.d = part;
    set_desc(ln, d);
    ln.kname = std::string("credw<") + tname(Z.dtype) + ", " + shape;
    out.push_back(ln);
    Launch lr;
    lr.kind = K_CREDW_REDUCE | dt_bits(DT_F32, DT_F32, C.dtype);
    lr.d = part;
    lr.c = C.buf;
    lr.grid[0] = (uint32_t)cdiv(d.R * M * KH * KW, 64);   // 64 outputs per block
    lr.block[0] = 256;
    set_desc(lr, d);
    lr.kname = std::string("credw_reduce<") + tname(C.dtype) + ">";
    out.push_back(lr);
    return true;
}

// ---- convolution contracted over one channel index, on MFMA tiles ----------
//   C[u][q][h][w] = sum_p sum_taps Z[u][p][h + dh][w + dw] * O[p][q][fh][fw]
// in bf16 (CconvDesc): the forward of a Tucker-core step and its input
// gradient (taps reversed).  Few output channels stay with try_cred, the
// filter gradient (taps as outputs) with try_tc.
bool try_cconv(const PairOp& op, std::vector<Launch>& out) {
    if (!op.has_r || op.convs.size() != 2 || op.L.dtype != op.R.dtype) return false;
    const bool bf = op.L.dtype == DT_BF16;
    if (!bf && op.C.dtype != DT_F32) return false;
    const int zside = op.convs[0].aL != 0 ? 0 : 1;
    const TensorRef& Z = zside == 0 ? op.L : op.R;
    const TensorRef& O = zside == 0 ? op.R : op.L;
    const TensorRef& C = op.C;
    struct Cv {
        int label;
        int64_t J, H;
        int bZ, bO;
        int64_t gZ, gO;
    } cv[2];
    for (int k = 0; k < 2; k++) {
        const ConvMap& cm = op.convs[k];
        const int aZ = zside == 0 ? cm.aL : cm.aR, bZ = zside == 0 ? cm.bL : cm.bR;
        const int aO = zside == 0 ? cm.aR : cm.aL, bO = zside == 0 ? cm.bR : cm.bL;
        const int64_t gZ = zside == 0 ? cm.gL : cm.gR, gO = zside == 0 ? cm.gR : cm.gL;
        const int64_t limZ = zside == 0 ? cm.limL : cm.limR, limO = zside == 0 ? cm.limR : cm.limL;
        if (aZ != 1 || (bZ != 1 && bZ != -1) || aO != 0 || (bO != 1 && bO != -1)) return false;
        // same-size planes, taps within the filter, offsets of at most a filter width
        if (cm.O != limZ || cm.J < 1 || cm.J > 7) return false;
        const int64_t f0 = gO, f1 = gO + bO * (cm.J - 1);
        if (f0 < 0 || f0 >= limO || f1 < 0 || f1 >= limO) return false;
        if (gZ < -cm.J || gZ > cm.J) return false;
        if (!Z.has(cm.label) || !O.has(cm.label) || !C.has(cm.label)) return false;
        cv[k] = {cm.label, cm.J, limZ, bZ, bO, gZ, gO};
    }
    if (Z.stride_of(cv[0].label) == 1) std::swap(cv[0], cv[1]);
    const Cv& ch = cv[0];
    const Cv& cw = cv[1];
    const int64_t H = ch.H, W = cw.H;
    if (Z.stride_of(cw.label) != 1 || Z.stride_of(ch.label) != W || C.stride_of(cw.label) != 1 ||
        C.stride_of(ch.label) != W || C.dim_of(ch.label) != H || C.dim_of(cw.label) != W)
        return false;
    auto is_conv = [&](int l) { return l == ch.label || l == cw.label; };
    struct Dm {
        int64_t size, s1, s2;
    };
    auto merge = [](std::vector<Dm>& v) {
        for (size_t i = 0; i + 1 < v.size();) {
            if (v[i].s1 == v[i + 1].s1 * v[i + 1].size && v[i].s2 == v[i + 1].s2 * v[i + 1].size) {
                v[i].size *= v[i + 1].size;
                v[i].s1 = v[i + 1].s1;
                v[i].s2 = v[i + 1].s2;
                v.erase(v.begin() + i + 1);
            } else {
                i++;
            }
        }
    };
    // u: C's labels in Z only (strides in Z, C); q: C's labels in O only (O, C);
    // p: the contracted ones (Z, O)
    std::vector<Dm> U, Pd, Qd;
    for (size_t k = 0; k < C.labels.size(); k++) {
        const int l = C.labels[k];
        if (is_conv(l)) continue;
        const bool inZ = Z.has(l), inO = O.has(l);
        if (inZ && !inO) U.push_back({C.dims[k], Z.stride_of(l), C.strides[k]});
        else if (inO && !inZ) Qd.push_back({C.dims[k], O.stride_of(l), C.strides[k]});
        else return false;
    }
    for (size_t k = 0; k < Z.labels.size(); k++) {
        const int l = Z.labels[k];
        if (is_conv(l) || C.has(l)) continue;
        if (!O.has(l)) return false;
        Pd.push_back({Z.dims[k], Z.strides[k], O.stride_of(l)});
    }
    for (int l : O.labels)
        if (!is_conv(l) && !C.has(l) && !Z.has(l)) return false;
    merge(U);
    merge(Pd);
    merge(Qd);
    if (U.size() > 2 || Pd.size() != 1 || Qd.size() != 1) return false;
    const int64_t P = Pd[0].size, Q = Qd[0].size;
    // fp32: at most 8 contracted channels.  With more, the general contraction
    // is faster (64 channels, 3x3: a 64 x 64 dense step 517 against 1631 us, a
    // Tucker core over 14 x 14 planes 50 + 15 against 390 us)
    if (P > (bf ? 128 : 8) || Q <= 16) return false;
    CconvDesc d;
    std::memset(&d, 0, sizeof(d));
    d.H = (int32_t)H;
    d.W = (int32_t)W;
    d.KH = (int32_t)ch.J;
    d.KW = (int32_t)cw.J;
    d.zh0 = (int32_t)ch.gZ;
    d.zhs = ch.bZ;
    d.zw0 = (int32_t)cw.gZ;
    d.zws = cw.bZ;
    d.fh0 = (int32_t)ch.gO;
    d.fhs = ch.bO;
    d.fw0 = (int32_t)cw.gO;
    d.fws = cw.bO;
    d.P = (int32_t)P;
    d.Q = (int32_t)Q;
    // bf16: pairs of channels a word, 16 CB channels, 16-byte runs padded by 4
    // words; fp32: a channel a word, 8 CB channels, odd pitches
    const int unit = bf ? 16 : 8;
    const int CB = P <= unit ? 1 : P <= 2 * unit ? 2 : P <= 4 * unit ? 4 : 8;
    d.Ppad = unit * CB;
    d.pw_img = bf ? 8 * CB + 4 : 8 * CB + 1;
    // tap runs padded by 4 words (lanes writing consecutive taps hit different
    // banks), q rows to an odd multiple of 4 words (the MFMA reads of 32 rows)
    d.tp = bf ? 8 * CB + 4 : 8 * CB;
    d.pw_tab = d.KH * d.KW * d.tp;
    if (bf && (d.pw_tab / 4) % 2 == 0) d.pw_tab += 4;
    if (!bf) d.pw_tab += 1;
    d.WP = (int32_t)(W + d.KW - 1);
    d.y_sq = Qd[0].s2;
    // fp32 with at most eight channels and nine taps: the filter operands of a
    // q tile fit a wavefront's registers, LDS holds the input rows only
    const int64_t y_ext = (Q - 1) * d.y_sq + H * W;
    d.rega = !bf && CB == 1 && d.KH * d.KW <= 9 && d.y_sq >= 1 && y_ext * 4 < ((int64_t)1 << 31);
    // output rows a block: the whole plane when two blocks' LDS fit a CU (four
    // for rega, whose LDS is the input rows only)
    auto lds_of = [&](int64_t th) {
        return 4 * ((d.rega ? 0 : 32 * (int64_t)d.pw_tab) + (th + d.KH - 1) * d.WP * d.pw_img);
    };
    const int64_t lds_cap = d.rega ? 40 * 1024 : 80 * 1024;
    int64_t TH = H;
    while (TH > 1 && lds_of(TH) > lds_cap) TH = (TH + 1) / 2;
    if (lds_of(TH) > 160 * 1024) return false;
    d.TH = (int32_t)TH;
    d.HP = (int32_t)(TH + d.KH - 1);
    d.ntiles = (int32_t)cdiv(H, TH);
    d.nq = (int32_t)cdiv(Q, 32);
    d.lds_bytes = (uint32_t)lds_of(TH);
    d.y_ext = d.rega ? y_ext : 0;
    d.ng = (int32_t)U.size();
    d.G = 1;
    for (size_t i = 0; i < U.size(); i++) {
        d.g_size[i] = U[i].size;
        d.g_sZ[i] = U[i].s1;
        d.g_sY[i] = U[i].s2;
        d.G *= U[i].size;
    }
    d.z_sp = Pd[0].s1;
    d.f_sp = Pd[0].s2;
    d.f_sq = Qd[0].s1;
    d.f_sh = O.stride_of(ch.label);
    d.f_sw = O.stride_of(cw.label);
    d.z_numel = Z.numel();
    d.f_numel = O.numel();
    if (d.z_numel >= (int64_t(1) << 30) || d.f_numel >= (int64_t(1) << 30)) return false;
    d.blocks = d.G * d.ntiles * (d.rega ? 1 : d.nq);
    if (d.blocks > 0x7fffffff) return false;
    Launch ln;
    ln.kind = K_CCONV | dt_bits(op.L.dtype, op.L.dtype, C.dtype);
    ln.a = Z.buf;
    ln.b = O.buf;
    ln.c = C.buf;
    ln.grid[0] = (uint32_t)d.blocks;
    ln.block[0] = 256;
    ln.lds = d.lds_bytes;
    set_desc(ln, d);
    ln.kname = d.rega ? "cconv_r<" + std::to_string(d.KH * d.KW) + ">"
                      : "cconv<" + std::to_string(CB) + ", " + tname(op.L.dtype) + ", " + tname(C.dtype) + ">";
    out.push_back(ln);
    return true;
}

// ---- general contraction on MFMA tiles --------------------------------------
bool try_tc(const PairOp& op, ScratchAlloc& scratch, std::vector<Launch>& out, bool wide) {
    if (!op.has_r || op.convs.size() > 2 || op.L.dtype != op.R.dtype) return false;
    // B is the operand whose positions mix an output and a reduction index
    int bside = -1;   // 0: L is B, 1: R is B
    for (const ConvMap& cm : op.convs) {
        const bool lmix = cm.aL != 0, rmix = cm.aR != 0;
        const int sd = (lmix && !rmix) ? 0 : (!lmix && rmix) ? 1 : -2;
        if (sd == -2) return false;
        if (bside == -1) bside = sd;
        else if (bside != sd) return false;
    }
    const TensorRef& C = op.C;
    if (bside == -1) {
        // plain contraction: B holds the output's innermost label (unit-stride columns)
        const int last = C.labels.empty() ? -1 : C.labels.back();
        const bool inL = last >= 0 && op.L.has(last), inR = last >= 0 && op.R.has(last);
        if (inR && !inL) bside = 1;
        else if (inL && !inR) bside = 0;
        else bside = op.R.numel() >= op.L.numel() ? 1 : 0;
    }
    const TensorRef& Bt = bside == 0 ? op.L : op.R;
    const TensorRef& At = bside == 0 ? op.R : op.L;
    const BufRef& bbuf = Bt.buf;
    const BufRef& abuf = At.buf;
    auto conv_of = [&](int l) -> int {
        for (size_t k = 0; k < op.convs.size(); k++)
            if (op.convs[k].label == l) return (int)k;
        return -1;
    };
    // the A side reads a convolved label as its plain reduction index
    for (const ConvMap& cm : op.convs) {
        const int a = bside == 0 ? cm.aR : cm.aL, b = bside == 0 ? cm.bR : cm.bL;
        const int64_t g = bside == 0 ? cm.gR : cm.gL, lim = bside == 0 ? cm.limR : cm.limL;
        if (a != 0 || b != 1 || g != 0 || lim < cm.J || !At.has(cm.label)) return false;
    }
    struct Dm {
        int64_t size, sA, sB, sC;
        int cv;
    };
    std::vector<Dm> G, M, N, K;
    for (size_t k = 0; k < C.labels.size(); k++) {
        const int l = C.labels[k];
        const int ci = conv_of(l);
        if (ci >= 0) {
            N.push_back({op.convs[ci].O, 0, 0, C.strides[k], ci});
            continue;
        }
        const bool inA = At.has(l), inB = Bt.has(l);
        if (inA && inB) G.push_back({C.dims[k], At.stride_of(l), Bt.stride_of(l), C.strides[k], -1});
        else if (inA) M.push_back({C.dims[k], At.stride_of(l), 0, C.strides[k], -1});
        else if (inB) N.push_back({C.dims[k], 0, Bt.stride_of(l), C.strides[k], -1});
        else return false;   // output label broadcast from neither operand
    }
    for (size_t k = 0; k < At.labels.size(); k++) {   // reduction dims in A's order
        const int l = At.labels[k];
        const int ci = conv_of(l);   // a convolved label: its reduction index, even though C has it
        if (ci >= 0) {
            K.push_back({op.convs[ci].J, At.strides[k], 0, 0, ci});
            continue;
        }
        if (C.has(l)) continue;
        if (!Bt.has(l)) return false;   // self-contracted in A
        K.push_back({At.dims[k], At.strides[k], Bt.stride_of(l), 0, -1});
    }
    for (int l : Bt.labels)
        if (!C.has(l) && !At.has(l) && conv_of(l) < 0) return false;   // self-contracted in B
    auto merge = [](std::vector<Dm>& v) {
        for (size_t i = 0; i + 1 < v.size();) {
            Dm& a = v[i];
            const Dm& b = v[i + 1];
            if (a.cv < 0 && b.cv < 0 && a.sA == b.sA * b.size && a.sB == b.sB * b.size &&
                a.sC == b.sC * b.size) {
                a.size *= b.size;
                a.sA = b.sA;
                a.sB = b.sB;
                a.sC = b.sC;
                v.erase(v.begin() + i + 1);
            } else {
                i++;
            }
        }
    };
    merge(G);
    merge(M);
    merge(N);
    merge(K);
    if (G.size() > 4 || M.size() > 4 || N.size() > 4 || K.size() > 4) return false;
    auto total = [](const std::vector<Dm>& v) {
        int64_t t = 1;
        for (const Dm& x : v) t *= x.size;
        return t;
    };
    const int64_t Mt = total(M), Nt = total(N), Kt = total(K), Gt = total(G);
    if (Mt >= (1ll << 31) || Nt >= (1ll << 31) || Kt >= (1ll << 31) || Mt * Nt == 0 || Kt == 0) return false;
    TcDesc d;
    std::memset(&d, 0, sizeof(d));
    d.ng = (int32_t)G.size();
    d.nm = (int32_t)M.size();
    d.nn = (int32_t)N.size();
    d.nk = (int32_t)K.size();
    d.ncv = (int32_t)op.convs.size();
    d.M = Mt;
    d.N = Nt;
    d.K = Kt;
    d.G = Gt;
    for (size_t i = 0; i < G.size(); i++) {
        d.g_size[i] = G[i].size;
        d.g_sA[i] = G[i].sA;
        d.g_sB[i] = G[i].sB;
        d.g_sC[i] = G[i].sC;
    }
    for (size_t i = 0; i < M.size(); i++) {
        d.m_size[i] = M[i].size;
        d.m_sA[i] = M[i].sA;
        d.m_sC[i] = M[i].sC;
    }
    for (size_t i = 0; i < 4; i++) d.n_cv[i] = d.k_cv[i] = -1;
    for (size_t i = 0; i < N.size(); i++) {
        d.n_size[i] = N[i].size;
        d.n_sB[i] = N[i].sB;
        d.n_sC[i] = N[i].sC;
        d.n_cv[i] = N[i].cv;
    }
    for (size_t i = 0; i < K.size(); i++) {
        d.k_size[i] = K[i].size;
        d.k_sA[i] = K[i].sA;
        d.k_sB[i] = K[i].sB;
        d.k_cv[i] = K[i].cv;
    }
    for (size_t c = 0; c < op.convs.size(); c++) {
        const ConvMap& cm = op.convs[c];
        d.cv_a[c] = bside == 0 ? cm.aL : cm.aR;
        d.cv_b[c] = bside == 0 ? cm.bL : cm.bR;
        d.cv_g[c] = bside == 0 ? cm.gL : cm.gR;
        d.cv_lim[c] = bside == 0 ? cm.limL : cm.limR;
        d.cv_s[c] = Bt.stride_of(cm.label);
    }
    const int MT = Mt > 32 ? 2 : 1;
    d.mtiles = (int32_t)cdiv(Mt, 32 * MT);
    d.ntiles = (int32_t)cdiv(Nt, 128);
    const int64_t tiles = Gt * d.mtiles * d.ntiles;
    // split the reduction when the output alone gives too few blocks
    int64_t ksplit = 1;
    if (tiles < 1024 && Kt > 512) ksplit = std::min<int64_t>(cdiv(2048, tiles), cdiv(Kt, 256));
    while (ksplit > 1 && (double)Gt * ksplit * Mt * Nt * 4.0 > 512.0 * (1 << 20)) ksplit /= 2;
    const int64_t kq = At.dtype == DT_BF16 && Kt >= 64 ? 64 : 32;   // the kernel's reduction slice
    d.kchunk = cdiv(cdiv(Kt, ksplit), kq) * kq;
    d.ksplit = (int32_t)cdiv(Kt, d.kchunk);
    d.blocks = tiles * d.ksplit;
    if (d.blocks > 0x7fffffff || Gt * Mt * Nt > ((int64_t)1 << 40)) return false;
    // 31-bit offsets when every element offset of A, B and C (and the byte
    // extents of A and B) fit
    auto extent = [](const TensorRef& t) {
        int64_t e = 1;
        for (size_t i = 0; i < t.dims.size(); i++) e += (t.dims[i] - 1) * t.strides[i];
        return e;
    };
    const int64_t esz = At.dtype == DT_BF16 ? 2 : 4, lim31 = (int64_t)1 << 31;
    const int64_t eA = extent(At), eB = extent(Bt), eC = extent(C);
    d.off32 = !wide && eA * esz < lim31 && eB * esz < lim31 && eC < lim31 ? 1 : 0;
    d.extA = eA * esz;
    d.extB = eB * esz;
    // k-major tile loads: the innermost reduction dim is unit-stride in A and
    // B while the innermost column dim is not unit-stride in B
    if (!K.empty() && K.back().cv < 0 && K.back().sA == 1 && K.back().sB == 1 &&
        (N.empty() || N.back().cv >= 0 || N.back().sB != 1))
        d.kmajor = 1;
    // at most 32 combinations of the convolved reduction indices: tap bitmasks
    if (!d.kmajor && !op.convs.empty()) {
        const int64_t J0 = op.convs[0].J, J1 = op.convs.size() > 1 ? op.convs[1].J : 1;
        if (J0 * J1 <= 32) {
            d.tapmask = 1;
            d.tapJ1 = (int32_t)J1;
        }
    }
    const char* tin = tname(At.dtype);
    Launch ln;
    ln.kind = K_TC | dt_bits(At.dtype, At.dtype, C.dtype);
    ln.a = abuf;
    ln.b = bbuf;
    ln.grid[0] = (uint32_t)d.blocks;
    ln.block[0] = 256;
    ln.kname = std::string("tc_gemm<") + tin + ", " + tname(d.ksplit > 1 ? C.dtype : C.dtype) + ", " +
               (MT == 2 ? "2>" : "1>");
    if (d.ksplit == 1) {
        ln.c = C.buf;
        set_desc(ln, d);
        out.push_back(ln);
        return true;
    }
    const BufRef part = scratch.alloc((size_t)(Gt * d.ksplit * Mt * Nt) * 4);
    ln.d = part;
    set_desc(ln, d);
    out.push_back(ln);
    Launch lr;
    lr.kind = K_TC_REDUCE | dt_bits(DT_F32, DT_F32, C.dtype);
    lr.d = part;
    lr.c = C.buf;
    // outputs of one g a block: 256 (one a thread) for at most 8 chunks, else 64
    lr.grid[0] = (uint32_t)(Gt * cdiv(Mt * Nt, d.ksplit <= 8 ? 256 : 64));
    lr.block[0] = d.ksplit <= 64 ? 256 : 1024;
    set_desc(lr, d);
    lr.kname = d.ksplit <= 8 ? std::string("tc_reduce_few<") + tname(C.dtype) + ">"
                             : std::string("tc_reduce<") + (d.ksplit <= 64 ? "4, " : "16, ") + tname(C.dtype) + ">";
    out.push_back(lr);
    return true;
}

// ---- both gradients of a channel-mixing step in one launch -----------------
// The step C[g][k][n] = sum_m A[g][m][n] F[k][m] (fp32); gl = its "grad lhs"
// op (dC x rhs -> d lhs), gr = its "grad rhs" op (lhs x dC -> d rhs).
bool try_gpair_ops(const PairOp& gl, const PairOp& gr, ScratchAlloc& scratch, std::vector<Launch>& out,
                   int& fside) {
    if (!gl.has_r || !gr.has_r || !gl.convs.empty() || !gr.convs.empty()) return false;
    const TensorRef& Gt = gl.L;   // the output gradient
    for (int side = 0; side < 2; side++) {
        // side 0: lhs = A (activation), rhs = F; side 1: lhs = F, rhs = A
        const TensorRef& At = side == 0 ? gr.L : gl.R;
        const TensorRef& Ft = side == 0 ? gl.R : gr.L;
        const TensorRef& dAt = side == 0 ? gl.C : gr.C;
        const TensorRef& dFt = side == 0 ? gr.C : gl.C;
        if (At.dtype != DT_F32 || Ft.dtype != DT_F32 || Gt.dtype != DT_F32 || dAt.dtype != DT_F32 ||
            dFt.dtype != DT_F32)
            continue;
        // dA and dF have the layouts of A and F
        bool same = dAt.labels == At.labels && dFt.labels == Ft.labels && dFt.strides == Ft.strides;
        if (!same) continue;
        // label classes
        std::vector<int> ml, kl, gl_, nl;
        bool ok = true;
        for (int l : At.labels) {
            const bool inF = Ft.has(l), inG = Gt.has(l);
            if (inF && inG) ok = false;
            else if (inF) ml.push_back(l);
            else if (!inG) ok = false;
        }
        for (int l : Ft.labels)
            if (!At.has(l)) {
                if (Gt.has(l)) kl.push_back(l);
                else ok = false;
            }
        for (int l : Gt.labels)
            if (!At.has(l) && !Ft.has(l)) ok = false;
        if (!ok || ml.empty() || kl.empty()) continue;
        // n: the innermost labels of G, unit-stride runs in A, G and dA
        int64_t expect = 1;
        for (int k = (int)Gt.labels.size() - 1; k >= 0; --k) {
            const int l = Gt.labels[k];
            if (!At.has(l) || Ft.has(l)) break;
            if (Gt.strides[k] != expect || At.stride_of(l) != expect || dAt.stride_of(l) != expect) break;
            nl.insert(nl.begin(), l);
            expect *= Gt.dims[k];
        }
        if (nl.empty()) continue;
        const int64_t N = expect;
        for (int l : Gt.labels)
            if (At.has(l) && std::find(nl.begin(), nl.end(), l) == nl.end()) gl_.push_back(l);
        // m: one merged dim in A, dA and F
        int64_t M, sAm, sDm, sFm, t1, t2;
        if (!merged(At, ml, M, sAm) || !merged(dAt, ml, t1, sDm) || !merged(Ft, ml, t2, sFm)) {
            // try m in F's order
            std::vector<int> mf;
            for (int l : Ft.labels)
                if (std::find(ml.begin(), ml.end(), l) != ml.end()) mf.push_back(l);
            if (!merged(At, mf, M, sAm) || !merged(dAt, mf, t1, sDm) || !merged(Ft, mf, t2, sFm)) continue;
        }
        // k: G's order, split into at most two runs that chain in G and F
        std::vector<int> kg;
        for (int l : Gt.labels)
            if (std::find(kl.begin(), kl.end(), l) != kl.end()) kg.push_back(l);
        std::vector<std::vector<int>> runs;
        for (int l : kg) {
            if (!runs.empty()) {
                std::vector<int> t = runs.back();
                t.push_back(l);
                int64_t a, b, c, e;
                if (merged(Gt, t, a, b) && merged(Ft, t, c, e)) {
                    runs.back() = t;
                    continue;
                }
            }
            runs.push_back({l});
        }
        if (runs.size() > 2) continue;
        int64_t K1 = 1, sG1 = 0, sF1 = 0, K2, sG2, sF2, tk;
        if (!merged(Gt, runs.back(), K2, sG2) || !merged(Ft, runs.back(), tk, sF2)) continue;
        if (runs.size() == 2 && (!merged(Gt, runs[0], K1, sG1) || !merged(Ft, runs[0], tk, sF1))) continue;
        const int64_t K = K1 * K2;
        // g: merged runs in A, G and dA (at most two)
        std::vector<BDim> bd;
        for (int l : gl_) bd.push_back({At.dim_of(l), At.stride_of(l), Gt.stride_of(l), dAt.stride_of(l)});
        bd = merge_dims(bd);
        if (bd.size() > 2 || M > 32 || K > 512) continue;
        int64_t G = 1;
        for (const BDim& b : bd) G *= b.size;
        int64_t fnumel = 1;
        for (int64_t dm : Ft.dims) fnumel *= dm;
        // F dense (the partials take its layout)
        {
            int64_t ext = 1;
            for (size_t i = 0; i < Ft.dims.size(); i++) ext += (Ft.dims[i] - 1) * Ft.strides[i];
            if (ext != fnumel) continue;
        }
        GpairDesc d;
        std::memset(&d, 0, sizeof(d));
        d.M = (int32_t)M;
        d.K = (int32_t)K;
        d.K1 = (int32_t)K1;
        d.K2 = (int32_t)K2;
        d.N = (int32_t)N;
        d.ng = (int32_t)bd.size();
        d.nkc = K <= 64 ? 1 : K <= 128 ? 2 : K <= 256 ? 4 : 8;
        d.ntiles = (int32_t)cdiv(N, 64);
        for (size_t i = 0; i < bd.size(); i++) {
            d.g_size[i] = bd[i].size;
            d.g_sA[i] = bd[i].s0;
            d.g_sG[i] = bd[i].s1;
            d.g_sD[i] = bd[i].s2;
        }
        d.sAm = sAm;
        d.sDm = sDm;
        d.sFm = sFm;
        d.sG1 = sG1;
        d.sG2 = sG2;
        d.sF1 = sF1;
        d.sF2 = sF2;
        d.G = G;
        d.gper = cdiv(G, 1024);
        d.blocks = cdiv(G, d.gper);
        d.fnumel = fnumel;
        d.lds_bytes = (uint32_t)(4 * (32 * (64 * d.nkc + 4) + 2 * 64 * 96 + 2 * 32 * 68));
        d.gext = (K1 - 1) * sG1 + (K2 - 1) * sG2 + N;
        d.aext = (M - 1) * sAm + N;
        if (N >= ((int64_t)1 << 31) || fnumel >= ((int64_t)1 << 31) || d.blocks * fnumel > ((int64_t)1 << 28) ||
            d.gext * 4 >= ((int64_t)1 << 31) || d.aext * 4 >= ((int64_t)1 << 31) || sG1 < 0 || sG2 < 0 || sAm < 0)
            continue;
        const BufRef part = scratch.alloc((size_t)(d.blocks * fnumel * 4));
        Launch ln;
        ln.kind = K_GPAIR | dt_bits(DT_F32, DT_F32, DT_F32);
        ln.a = At.buf;
        ln.b = Ft.buf;
        ln.c = Gt.buf;
        ln.d = part;
        ln.extra = {dAt.buf};
        ln.grid[0] = (uint32_t)d.blocks;
        ln.block[0] = 1024;
        ln.lds = d.lds_bytes;
        set_desc(ln, d);
        ln.kname = "gpair<" + std::to_string(d.nkc) + ">";
        out.push_back(ln);
        ReduceDesc rd;
        rd.M = 1;
        rd.N = (int32_t)fnumel;
        rd.nsplit = d.blocks;
        rd.sCm = 0;
        rd.sCn = 1;
        Launch lr;
        lr.kind = K_REDUCE | dt_bits(DT_F32, DT_F32, DT_F32);
        lr.d = part;
        lr.c = dFt.buf;
        lr.grid[0] = (uint32_t)cdiv(fnumel, 64);
        lr.block[0] = (uint32_t)(64 * reduce_waves(rd.nsplit));
        set_desc(lr, rd);
        lr.kname = "reduce_partials<" + std::to_string(reduce_waves(rd.nsplit)) + ", float>";
        out.push_back(lr);
        fside = side;
        return true;
    }
    return false;
}

}  // namespace

// Both gradient ops of one step in a single fused launch (plus its ordered
// partial sum) when they match try_gpair_ops; empty otherwise.
std::vector<Launch> lower_grad_pair(const PairOp& gl, const PairOp& gr, unsigned flags, ScratchAlloc& scratch) {
    std::vector<Launch> out;
    if ((flags & (CE_FLAG_GENERIC_ONLY | CE_FLAG_NO_FUSION)) || gl.generic_only || gr.generic_only) return out;
    int fside = 0;
    if (!try_gpair_ops(gl, gr, scratch, out, fside)) {
        out.clear();
        return out;
    }
    const double bytes = tensor_bytes(gl.L) + tensor_bytes(gl.R) + tensor_bytes(gr.L) + tensor_bytes(gl.C) +
                         tensor_bytes(gr.C);
    out[0].need = gl.need | gr.need;
    out[0].what = gl.what + " + " + gr.what.substr(gr.what.find("grad"));
    out[0].alg_bytes = bytes;
    out[0].alg_flops = 4.0 * (double)gl.macs;
    // the partial sum runs when the factor's gradient is wanted (side 0: the
    // factor is the step's rhs, its gradient the grad rhs op's)
    out[1].need = fside == 0 ? gr.need : gl.need;
    out[1].what = out[0].what;
    return out;
}

std::vector<Launch> lower_op(const ce_expr& e, const PairOp& op, unsigned flags,
                             ScratchAlloc& scratch) {
    (void)e;
    std::vector<Launch> out;
    bool circular = false;   // circular maps run on the generic kernel only
    for (const ConvMap& cm : op.convs)
        if (cm.modL || cm.modR) circular = true;
    bool fast = !(flags & CE_FLAG_GENERIC_ONLY) && !op.generic_only && !circular &&
                (try_gemm(op, out) || try_wgrad(op, scratch, out) || try_dw(op, scratch, out) ||
                 try_cred(op, scratch, out) || try_cconv(op, out) || try_thinw(op, scratch, out) ||
                 try_tc(op, scratch, out, (flags & CE_FLAG_WIDE_OFFSETS) != 0));
    if (!fast) {
        out.clear();
        Launch ln = lower_generic(op);
        int v = ln.kind & 0xff;
        ln.kname = std::string(v == K_GENERIC_THREAD ? "generic_thread<" : v == K_GENERIC_WAVE
                                                                              ? "generic_wave<"
                                                                              : "generic_block<") +
                   tname(op.L.dtype) + ", " + tname(op.has_r ? op.R.dtype : DT_F32) + ", " +
                   tname(op.C.dtype) + ">";
        out.push_back(ln);
    }
    double bytes = tensor_bytes(op.L) + (op.has_r ? tensor_bytes(op.R) : 0) + tensor_bytes(op.C);
    for (auto& ln : out) {
        ln.need = op.need;
        ln.what = op.what;
        ln.alg_bytes = bytes / out.size();
        ln.alg_flops = 2.0 * (double)op.macs / out.size();
    }
    // the main launch of a split op carries the op's bytes and flops
    if (out.size() == 2) {
        out[0].alg_bytes = bytes;
        out[0].alg_flops = 2.0 * (double)op.macs;
        out[1].alg_bytes = 0;
        out[1].alg_flops = 0;
    }
    return out;
}

}  // namespace ce
