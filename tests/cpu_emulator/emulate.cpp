// CPU emulation of a plan's launch list (test infrastructure).
//
// Builds a plan with the library's own host planner (compiled in from the
// package sources), then executes every launch on the CPU with the semantics
// of its descriptor (the index arithmetic each HIP kernel performs, element
// by element), with every memory access checked against the size of the
// buffer it falls in and every launch grid checked against what the kernel
// assumes.  A test compares the results with the oracle, so
// descriptor, layout and workspace bugs show up without a GPU, and an
// out-of-bounds access is reported instead of faulting a device.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "expr.h"
#include "plan.h"

#define RCP_FN inline
#define RCP_HD inline
#include "rcp_body.h"
#define RCPB_FN inline
#define RCPB_HD inline
#include "rcpb_body.h"

using namespace ce;

namespace {

struct Buf {
    unsigned char* base = nullptr;
    size_t bytes = 0;
};

struct Ctx {
    std::vector<Buf> in, din;
    Buf out, dout, ws;
    std::string err;
};

Buf resolve_base(const BufRef& b, Ctx& c, bool& ok) {
    ok = true;
    switch (b.kind) {
        case BUF_IN: return c.in[b.index];
        case BUF_OUT: return c.out;
        case BUF_DOUT: return c.dout;
        case BUF_DIN: return c.din[b.index];
        case BUF_WS: {
            Buf r;
            if (b.offset > c.ws.bytes) { ok = false; return r; }
            r.base = c.ws.base + b.offset;
            r.bytes = c.ws.bytes - b.offset;
            return r;
        }
        default: ok = false; return Buf();
    }
}

// The buffer a launch operand refers to, from its view shift on (bounds
// checks then count from the view's first byte to the buffer's end).
Buf resolve(const BufRef& b, Ctx& c, int esize, bool& ok) {
    Buf r = resolve_base(b, c, ok);
    (void)esize;
    if (!ok || !r.base || b.shift == 0) return r;
    if (b.shift < 0 || (size_t)b.shift > r.bytes) { ok = false; return Buf(); }
    r.base += b.shift;
    r.bytes -= (size_t)b.shift;
    return r;
}

float ld(const Buf& b, int dt, int64_t i, bool& ok) {
    int es = dt ? 2 : 4;
    if (i < 0 || (size_t)(i + 1) * es > b.bytes) { ok = false; return 0.f; }
    if (dt) {
        uint16_t v;
        std::memcpy(&v, b.base + i * 2, 2);
        uint32_t u = (uint32_t)v << 16;
        float f;
        std::memcpy(&f, &u, 4);
        return f;
    }
    float f;
    std::memcpy(&f, b.base + i * 4, 4);
    return f;
}

void st(Buf& b, int dt, int64_t i, float v, bool& ok) {
    int es = dt ? 2 : 4;
    if (i < 0 || (size_t)(i + 1) * es > b.bytes) { ok = false; return; }
    if (dt) {
        uint32_t u;
        std::memcpy(&u, &v, 4);
        if ((u & 0x7fffffffu) > 0x7f800000u) u = (u >> 16 | 0x40) << 16;
        else u += 0x7fffu + ((u >> 16) & 1u);
        uint16_t h = (uint16_t)(u >> 16);
        std::memcpy(b.base + i * 2, &h, 2);
    } else {
        std::memcpy(b.base + i * 4, &v, 4);
    }
}

bool run_generic(const Launch& ln, Ctx& c) {
    GenericDesc d;
    std::memcpy(&d, ln.desc.data(), sizeof(d));
    int tL = (ln.kind >> 8) & 1, tR = (ln.kind >> 9) & 1, tC = (ln.kind >> 10) & 1;
    bool ok1, ok2, ok3;
    Buf L = resolve(ln.a, c, 0, ok1), R = resolve(ln.b, c, 0, ok2), C = resolve(ln.c, c, 0, ok3);
    if (!ok1 || !ok3 || (d.has_r && !ok2) || !C.base) { c.err = "unresolved buffer: " + ln.what; return false; }
    // the launch grid must cover every output element exactly
    int variant = ln.kind & 0xff;
    uint64_t covered = variant == K_GENERIC_THREAD ? (uint64_t)ln.grid[0] * 256
                     : variant == K_GENERIC_WAVE ? (uint64_t)ln.grid[0] * 4 : ln.grid[0];
    if (covered < (uint64_t)d.total_out || ln.block[0] != 256) { c.err = "grid does not cover: " + ln.what; return false; }
    for (int64_t o = 0; o < d.total_out; o++) {
        int64_t rem = o, offL = 0, offR = 0, offC = 0, oidx[kMaxDims] = {0};
        for (int i = d.nout - 1; i >= 0; --i) {
            int64_t x = rem % d.out_size[i];
            rem /= d.out_size[i];
            oidx[i] = x;
            offL += x * d.out_sL[i];
            offR += x * d.out_sR[i];
            offC += x * d.out_sC[i];
        }
        double acc = 0;   // order differs from the device; precision is not under test
        for (int64_t r = 0; r < d.total_red; r++) {
            int64_t rr = r, aL = offL, aR = offR, ridx[kMaxDims] = {0};
            for (int i = d.nred - 1; i >= 0; --i) {
                int64_t x = rr % d.red_size[i];
                rr /= d.red_size[i];
                ridx[i] = x;
                aL += x * d.red_sL[i];
                aR += x * d.red_sR[i];
            }
            bool skip = false;
            for (int k = 0; k < d.nconv; k++) {
                int64_t p = oidx[d.cv_out[k]], j = ridx[d.cv_red[k]];
                int64_t pl = d.cv_aL[k] * p + d.cv_bL[k] * j + d.cv_gL[k];
                int64_t pr = d.cv_aR[k] * p + d.cv_bR[k] * j + d.cv_gR[k];
                if (d.cv_modL[k]) pl = ((pl % d.cv_modL[k]) + d.cv_modL[k]) % d.cv_modL[k];
                if (d.cv_modR[k]) pr = ((pr % d.cv_modR[k]) + d.cv_modR[k]) % d.cv_modR[k];
                if (pl < 0 || pl >= d.cv_limL[k] || pr < 0 || pr >= d.cv_limR[k]) { skip = true; break; }
                aL += pl * d.cv_sL[k];
                aR += pr * d.cv_sR[k];
            }
            if (skip) continue;
            bool ok = true;
            float a = ld(L, tL, aL, ok);
            float b = d.has_r ? ld(R, tR, aR, ok) : 1.f;
            if (!ok) { c.err = "out-of-bounds read: " + ln.what; return false; }
            acc += (double)a * b;
        }
        bool ok = true;
        st(C, tC, offC, (float)acc, ok);
        if (!ok) { c.err = "out-of-bounds write: " + ln.what; return false; }
    }
    return true;
}

template <typename D>
D desc_of(const Launch& ln) {
    D d;
    std::memcpy(&d, ln.desc.data(), sizeof(D));
    return d;
}

#define REQ(cond, msg) do { if (!(cond)) { c.err = std::string(msg) + ": " + ln.what; return false; } } while (0)

// C[g][m][n] = sum_k A[g][m][k] B[g][k][n]
bool run_gemm(const Launch& ln, Ctx& c) {
    GemmDesc d = desc_of<GemmDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    int MT = ((ln.kind >> kShiftOpt) & 1) ? 2 : 1;
    bool o1, o2, o3;
    Buf A = resolve(ln.a, c, 0, o1), B = resolve(ln.b, c, 0, o2), C = resolve(ln.c, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    const int64_t Gall = [&] { int64_t g = 1; for (int i = 0; i < d.ng; i++) g *= d.g_size[i]; return g; }();
    if ((ln.kind & 0xff) == K_THIN) {
        // one column per thread; M, K within the kernel's 16 x 16 (64 products) bounds; a
        // block spans at most 256 / 16 + 2 batch indices (its LDS slices), flat index in 31 bits
        const int mm = d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16, kk = d.K <= 4 ? 4 : d.K <= 8 ? 8 : 16;
        REQ(d.M <= 16 && d.K <= 16 && mm * kk <= 64 && d.N >= 16 && Gall * d.N < ((int64_t)1 << 31),
            "thin bounds");
        const int64_t runs = Gall * d.N;
        REQ(ln.grid[0] == (uint32_t)d.blocks && d.blocks * 256 >= runs && (d.blocks - 1) * 256 < runs &&
            ln.block[0] == 256, "grid");
    } else if ((ln.kind >> kShiftOpt) & 4) {
        // flattened columns: tiles of 128 over G x N, 8-byte rows of B
        bool al = tIn && d.N % 4 == 0 && d.sBk % 4 == 0 && Gall * d.N < ((int64_t)1 << 31);
        for (int i = 0; i < d.ng; i++) al = al && d.g_sB[i] % 4 == 0;
        REQ(al, "flat gemm alignment");
        REQ(ln.grid[0] == (uint32_t)d.blocks && d.blocks == (int64_t)d.mtiles * d.ntiles && ln.block[0] == 256,
            "grid");
        REQ(d.mtiles * 32 * MT >= d.M && (int64_t)d.ntiles * 128 >= Gall * d.N, "tiles do not cover");
        // the kernel's loads, thread by thread (K in chunks of 64): B at the
        // thread's column group (column 0 past the end) and rows kq + 32 h + r
        // (clamped to K - 1 in a partial chunk); A one row (rows fastest) or
        // one k (k fastest) per thread, clamped the same way
        const int TM = 32 * MT, TK = 64, AE = TM * TK / 256;
        const bool mfast = d.sAm == 1 && d.sAk != 1;
        const int64_t NF = Gall * d.N;
        bool okl = true;
        for (int64_t blk = 0; blk < d.blocks && okl; blk++) {
            const int64_t nt = blk % d.ntiles, mt = blk / d.ntiles;
            const int m0 = (int)mt * TM;
            for (int tid = 0; tid < 256 && okl; tid++) {
                const int nq = tid & 31, kq = 4 * (tid >> 5);
                const int64_t fb = nt * 128 + 4 * nq;
                const bool colok = fb < NF;
                int64_t g = colok ? fb / d.N : 0, ob = 0, x = g;
                for (int i = d.ng - 1; i >= 0; --i) { ob += (x % d.g_size[i]) * d.g_sB[i]; x /= d.g_size[i]; }
                ob += colok ? fb - g * d.N : 0;
                for (int k0 = 0; k0 < d.K; k0 += TK) {
                    const bool full = k0 + TK <= d.K;
                    for (int h = 0; h < 2; h++)
                        for (int r = 0; r < 4; r++) {
                            int k = k0 + kq + 32 * h + r;
                            if (!full) k = std::min(k, d.K - 1);
                            const int64_t i0 = ob + (int64_t)k * d.sBk;
                            okl = okl && i0 >= 0 && (size_t)(i0 + 4) * 2 <= B.bytes && i0 % 4 == 0;
                        }
                    for (int e = 0; e < AE; e++) {
                        const int i = tid + 256 * e;
                        int m = mfast ? i % TM : i / TK, k = mfast ? i / TM : i % TK;
                        m = std::min(m0 + m, d.M - 1);
                        k = std::min(k0 + k, d.K - 1);
                        const int64_t ia = (int64_t)m * d.sAm + (int64_t)k * d.sAk;
                        okl = okl && ia >= 0 && (size_t)(ia + 1) * 2 <= A.bytes;
                    }
                }
            }
        }
        REQ(okl, "flat gemm load out of range");
    } else {
        REQ(ln.grid[0] == (uint32_t)d.blocks && d.blocks == (int64_t)d.mtiles * d.ntiles * Gall, "grid");
        REQ(d.mtiles * 32 * MT >= d.M && d.ntiles * 128 >= d.N, "tiles do not cover");
    }
    int64_t G = 1;
    for (int i = 0; i < d.ng; i++) G *= d.g_size[i];
    for (int64_t g = 0; g < G; g++) {
        int64_t gg = g, oA = 0, oB = 0, oC = 0;
        for (int i = d.ng - 1; i >= 0; --i) {
            int64_t x = gg % d.g_size[i];
            gg /= d.g_size[i];
            oA += x * d.g_sA[i]; oB += x * d.g_sB[i]; oC += x * d.g_sC[i];
        }
        for (int m = 0; m < d.M; m++)
            for (int n = 0; n < d.N; n++) {
                double acc = 0;
                bool ok = true;
                for (int k = 0; k < d.K; k++)
                    acc += (double)ld(A, tIn, oA + (int64_t)m * d.sAm + (int64_t)k * d.sAk, ok) *
                           ld(B, tIn, oB + (int64_t)k * d.sBk + n, ok);
                REQ(ok, "out-of-bounds read (gemm)");
                st(C, tC, oC + (int64_t)m * d.sCm + n, (float)acc, ok);
                REQ(ok, "out-of-bounds write (gemm)");
            }
    }
    return true;
}

bool run_wgrad(const Launch& ln, Ctx& c) {
    WgradDesc d = desc_of<WgradDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1;
    bool o1, o2, o3;
    Buf A = resolve(ln.a, c, 0, o1), B = resolve(ln.b, c, 0, o2), P = resolve(ln.d, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    REQ((int64_t)ln.grid[0] == d.nsplit * d.mtiles * d.ntiles && d.blocks == (int64_t)ln.grid[0], "grid");
    REQ((int64_t)d.ksplit * d.kchunk >= d.K && d.mtiles * 64 >= d.M && d.ntiles * 64 >= d.N, "cover");
    for (int64_t s = 0; s < d.nsplit; s++) {
        int64_t kbi = s / d.ksplit, kc = s % d.ksplit, oA = 0, oB = 0;
        for (int i = d.nkb - 1; i >= 0; --i) {
            int64_t x = kbi % d.kb_size[i];
            kbi /= d.kb_size[i];
            oA += x * d.kb_sA[i]; oB += x * d.kb_sB[i];
        }
        int64_t k0 = kc * d.kchunk, k1 = std::min(d.K, k0 + d.kchunk);
        for (int m = 0; m < d.M; m++)
            for (int n = 0; n < d.N; n++) {
                double acc = 0;
                bool ok = true;
                for (int64_t k = k0; k < k1; k++)
                    acc += (double)ld(A, tIn, oA + m * d.sAm + k, ok) * ld(B, tIn, oB + n * d.sBn + k, ok);
                REQ(ok, "out-of-bounds read (wgrad)");
                st(P, 0, s * d.M * d.N + (int64_t)m * d.N + n, (float)acc, ok);
                REQ(ok, "out-of-bounds write (wgrad)");
            }
    }
    return true;
}

bool run_reduce(const Launch& ln, Ctx& c) {
    ReduceDesc d = desc_of<ReduceDesc>(ln);
    int tC = (ln.kind >> kBitOut) & 1;
    bool o1, o2;
    Buf P = resolve(ln.d, c, 0, o1), C = resolve(ln.c, c, 0, o2);
    REQ(o1 && o2, "unresolved buffer");
    REQ((int64_t)ln.grid[0] * 64 >= (int64_t)d.M * d.N, "grid");
    for (int64_t e = 0; e < (int64_t)d.M * d.N; e++) {
        double acc = 0;
        bool ok = true;
        for (int64_t s = 0; s < d.nsplit; s++) acc += ld(P, 0, s * d.M * d.N + e, ok);
        int64_t m = e / d.N, n = e % d.N;
        st(C, tC, m * d.sCm + n * d.sCn, (float)acc, ok);
        REQ(ok, "out-of-bounds (reduce)");
    }
    return true;
}

// Up to four ordered sums in one launch (K_REDUCE_MULTI): part j owns blocks
// [block0[j], block0[j+1]), 64 outputs a block.
bool run_reduce_multi(const Launch& ln, Ctx& c) {
    MultiReduceDesc d = desc_of<MultiReduceDesc>(ln);
    REQ(d.n >= 1 && d.n <= 4 && ln.extra.size() == (size_t)(2 * d.n) && d.block0[0] == 0 &&
        (int64_t)ln.grid[0] == d.block0[d.n], "multi-reduce shape");
    int64_t ns = 0;
    for (int j = 0; j < d.n; j++) ns = std::max<int64_t>(ns, d.part[j].nsplit);
    REQ(ln.block[0] == (uint32_t)(64 * reduce_waves(ns)), "multi-reduce block");
    for (int j = 0; j < d.n; j++) {
        const ReduceDesc& r = d.part[j];
        REQ((d.block0[j + 1] - d.block0[j]) * 64 >= (int64_t)r.M * r.N &&
            (d.block0[j + 1] - d.block0[j] - 1) * 64 < (int64_t)r.M * r.N, "multi-reduce blocks");
        bool o1, o2, ok = true;
        Buf P = resolve(ln.extra[2 * j], c, 0, o1), C = resolve(ln.extra[2 * j + 1], c, 0, o2);
        REQ(o1 && o2, "unresolved buffer");
        for (int64_t e = 0; e < (int64_t)r.M * r.N; e++) {
            double acc = 0;
            for (int64_t s2 = 0; s2 < r.nsplit; s2++) acc += ld(P, 0, s2 * r.M * r.N + e, ok);
            st(C, 0, (e / r.N) * r.sCm + (e % r.N) * r.sCn, (float)acc, ok);
        }
        REQ(ok, "out-of-bounds (multi-reduce)");
    }
    return true;
}

bool run_dw(const Launch& ln, Ctx& c) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1, tF = (ln.kind >> kBitAux) & 1, tC = (ln.kind >> kBitOut) & 1;
    bool o1, o2, o3;
    Buf I = resolve(ln.a, c, 0, o1), F = resolve(ln.b, c, 0, o2), O = resolve(ln.c, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    REQ((int64_t)ln.grid[0] * d.spb >= d.nslab && d.spb * d.A * d.inner <= 4096 && d.spb <= 256 &&
        d.K >= 1 && d.K <= 7, "launch shape");
    for (int64_t o = 0; o < d.nslab; o++) {
        int64_t frow = ((o / d.r_div) % d.r_size) * d.r_stride;
        for (int p = 0; p < d.A; p++)
            for (int q = 0; q < d.inner; q++) {
                double acc = 0;
                bool ok = true;
                for (int j = 0; j < d.K; j++) {
                    int pp = p + d.sign * j + d.off;
                    float fv = ld(F, tF, frow + (int64_t)j * d.f_sj, ok);
                    if (pp >= 0 && pp < d.A) acc += (double)ld(I, tIn, (o * d.A + pp) * d.inner + q, ok) * fv;
                }
                REQ(ok, "out-of-bounds read (dw)");
                st(O, tC, (o * d.A + p) * d.inner + q, (float)acc, ok);
                REQ(ok, "out-of-bounds write (dw)");
            }
    }
    return true;
}

bool run_tapgrad(const Launch& ln, Ctx& c) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1;
    bool o1, o2, o3;
    Buf I = resolve(ln.a, c, 0, o1), G = resolve(ln.b, c, 0, o2), P = resolve(ln.d, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    REQ((int64_t)ln.grid[0] == d.nblocks && d.nblocks * d.spb == d.nslab && d.r_div % d.spb == 0 &&
        d.spb * d.A * d.inner <= 4096 && d.K >= 1 && d.K <= 7, "launch shape");
    for (int64_t b = 0; b < d.nblocks; b++)
        for (int j = 0; j < d.K; j++) {
            double acc = 0;
            bool ok = true;
            for (int64_t o = b * d.spb; o < (b + 1) * d.spb; o++)
                for (int p = 0; p < d.A; p++)
                    for (int q = 0; q < d.inner; q++) {
                        int pp = p + j + d.off;
                        if (pp >= 0 && pp < d.A)
                            acc += (double)ld(I, tIn, (o * d.A + pp) * d.inner + q, ok) *
                                   ld(G, tIn, (o * d.A + p) * d.inner + q, ok);
                    }
            REQ(ok, "out-of-bounds read (tapgrad)");
            st(P, 0, b * d.K + j, (float)acc, ok);
            REQ(ok, "out-of-bounds write (tapgrad)");
        }
    return true;
}

bool run_tapreduce(const Launch& ln, Ctx& c) {
    DwDesc d = desc_of<DwDesc>(ln);
    int tC = (ln.kind >> kBitOut) & 1;
    bool o1, o2;
    Buf P = resolve(ln.d, c, 0, o1), O = resolve(ln.c, c, 0, o2);
    REQ(o1 && o2, "unresolved buffer");
    int64_t run = d.r_div / d.spb, period = run * d.r_size;
    REQ(d.nblocks % period == 0, "blocks do not tile the filter rows");
    REQ((int64_t)ln.grid[0] == d.r_size, "grid");
    for (int64_t r = 0; r < d.r_size; r++)
        for (int j = 0; j < d.K; j++) {
            double acc = 0;
            bool ok = true;
            for (int64_t a = 0; a < d.nblocks / period; a++)
                for (int64_t cc = 0; cc < run; cc++) acc += ld(P, 0, (a * period + r * run + cc) * d.K + j, ok);
            st(O, tC, r * d.o_sr + j * d.o_sj, (float)acc, ok);
            REQ(ok, "out-of-bounds (tapreduce)");
        }
    return true;
}

// Fused CP chain forward: the four steps with the descriptor's strides, plus
// the launch-shape and LDS-layout invariants the kernel relies on.
bool run_cp_fwd(const Launch& ln, Ctx& c) {
    CpDesc d = desc_of<CpDesc>(ln);
    int bf = (ln.kind >> kBitIn) & 1;
    bool o1, o2, o3;
    Buf X = resolve(ln.a, c, 0, o1), Us = resolve(ln.b, c, 0, o2), Y = resolve(ln.c, c, 0, o3);
    REQ(o1 && o2 && o3 && ln.extra.size() == 3, "unresolved buffer");
    bool o4, o5, o6;
    Buf Kh = resolve(ln.extra[0], c, 0, o4), Kw = resolve(ln.extra[1], c, 0, o5),
        Ut = resolve(ln.extra[2], c, 0, o6);
    REQ(o4 && o5 && o6, "unresolved buffer");
    REQ(d.R >= 1 && d.R <= 32 && d.T >= 1 && d.T <= 64 && d.S >= 1 && d.S <= 64, "sizes");
    REQ(d.KH == d.KW && (d.KH == 3 || d.KH == 5), "filter size");
    REQ(d.colstride == 32 - (d.KW - 1) && (int64_t)d.ncb * d.colstride >= d.W &&
        (int64_t)(d.ncb - 1) * d.colstride < d.W, "strips");
    REQ((int64_t)d.segs * d.seg_rows >= d.H && (int64_t)(d.segs - 1) * d.seg_rows < d.H, "segments");
    REQ(d.waves == (int64_t)d.B * d.ncb * d.segs && d.blocks * 4 >= d.waves &&
        (int64_t)ln.grid[0] == d.blocks && ln.block[0] == 256, "grid");
    // operand tables: UsL 32 x lda at 0, UtP at o_ut, tap tables at o_kh / o_kw
    const int64_t SPf = 32 * ((d.S + 31) / 32), TPf = 32 * ((d.T + 31) / 32);   // padded channel blocks
    REQ(d.lda >= SPf + (bf ? 8 : 1) && (!bf || (d.lda * 2) % 16 == 0), "UsL rows");
    REQ(d.o_ut >= (uint64_t)32 * d.lda * (bf ? 2 : 4) && d.o_ut % 16 == 0, "UtP offset");
    REQ(d.o_kh >= d.o_ut + (bf ? (uint64_t)2 * 2 * TPf * 8 * 2 : (uint64_t)16 * 2 * TPf * 4), "Kh offset");
    REQ(d.o_kw >= d.o_kh + (uint64_t)16 * 2 * d.KH * 4, "Kw offset");
    REQ(d.o_khr >= d.o_kw + (uint64_t)16 * 2 * d.KW * 4, "reversed Kh offset");
    REQ(d.lds_bytes >= d.o_khr + (uint64_t)16 * 2 * d.KH * 4 && d.lds_bytes <= 64 * 1024 &&
        ln.lds == d.lds_bytes, "LDS size");
    const int H = d.H, W = d.W, R = d.R, ch = (d.KH - 1) / 2, cw = (d.KW - 1) / 2;
    std::vector<double> z1((size_t)R * H * W), z2((size_t)R * H * W), z3v((size_t)R * H * W);
    bool ok = true;
    for (int b = 0; b < d.B; b++) {
        for (int r = 0; r < R; r++)
            for (int p = 0; p < H * W; p++) {
                double a = 0;
                for (int s2 = 0; s2 < d.S; s2++)
                    a += (double)ld(Us, bf, (int64_t)r * d.us_sr + (int64_t)s2 * d.us_ss, ok) *
                         ld(X, bf, (int64_t)b * d.x_sb + (int64_t)s2 * d.x_ss + p, ok);
                z1[(size_t)r * H * W + p] = a;
            }
        for (int r = 0; r < R; r++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    double a = 0;
                    for (int j = 0; j < d.KH; j++) {
                        int hh = h + j - ch;
                        if (hh >= 0 && hh < H)
                            a += z1[((size_t)r * H + hh) * W + w] * ld(Kh, bf, (int64_t)r * d.kh_sr + (int64_t)j * d.kh_sj, ok);
                    }
                    z2[((size_t)r * H + h) * W + w] = a;
                }
        for (int r = 0; r < R; r++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    double a = 0;
                    for (int j = 0; j < d.KW; j++) {
                        int ww = w + j - cw;
                        if (ww >= 0 && ww < W)
                            a += z2[((size_t)r * H + h) * W + ww] * ld(Kw, bf, (int64_t)r * d.kw_sr + (int64_t)j * d.kw_sj, ok);
                    }
                    z3v[((size_t)r * H + h) * W + w] = a;
                }
        for (int t = 0; t < d.T; t++)
            for (int p = 0; p < H * W; p++) {
                double a = 0;
                for (int r = 0; r < R; r++)
                    a += (double)ld(Ut, bf, (int64_t)r * d.ut_sr + (int64_t)t * d.ut_st, ok) *
                         z3v[(size_t)r * H * W + p];
                st(Y, bf, (int64_t)b * d.y_sb + (int64_t)t * d.y_st + p, (float)a, ok);
            }
        REQ(ok, "out-of-bounds access (cp_fwd)");
    }
    return true;
}

// Fused reshaped-CP forward: the kernel's own phases (rcp_body.h) run on the
// CPU thread by thread between the kernel's barriers, with every global and
// LDS access bounds-checked, LDS words poisoned until written, and a race
// check: within one barrier interval no LDS word may be written by one
// thread and read or written by another.  Every Y element must be written
// exactly once.
struct RcpHost {
    std::vector<uint32_t> lds;
    // race tracking per 16-bit half of every LDS word
    std::vector<int> w_seg, w_tid, r_seg, r_tid;
    std::vector<char> r_multi;
    std::vector<const Buf*> g;
    std::vector<int> ywrites;
    const Buf* ybuf = nullptr;
    int seg = 0, tid = 0;
    bool ok = true;
    std::string err;
    // MFMA operands recorded per lane of the current wave, row-sum accumulators
    std::vector<std::vector<std::pair<std::array<uint32_t, 4>, std::array<uint32_t, 4>>>> rec;
    std::vector<float> rowacc;
    void fail(const std::string& m) {
        if (ok) err = m;
        ok = false;
    }
    void reset_lds(size_t nw) {
        lds.assign(nw, 0xCDCDCDCDu);
        w_seg.assign(2 * nw, -1);
        w_tid.assign(2 * nw, -1);
        r_seg.assign(2 * nw, -1);
        r_tid.assign(2 * nw, -1);
        r_multi.assign(2 * nw, 0);
        rowacc.assign(nw, 0.f);
    }
    const Buf* buf_of(const void* p) {
        for (const Buf* b : g)
            if (b && (const void*)b->base == p) return b;
        return nullptr;
    }
    void chk(const void* p, int64_t i, int bytes) {
        const Buf* b = buf_of(p);
        if (!b || i < 0 || (size_t)(i + bytes) > b->bytes) fail("global access out of bounds");
    }
    uint16_t ld16(const uint16_t* p, int64_t i) {
        chk(p, 2 * i, 2);
        return ok ? p[i] : 0;
    }
    uint32_t ldw(const uint16_t* p, int64_t i) {
        chk(p, 2 * i, 4);
        if (i & 1) fail("misaligned word load");
        return ok ? (uint32_t)p[i] | ((uint32_t)p[i + 1] << 16) : 0;
    }
    void st16(uint16_t* p, int64_t i, uint16_t v) {
        chk(p, 2 * i, 2);
        if (!ok) return;
        p[i] = v;
        if (ybuf && (const unsigned char*)p == ybuf->base) ywrites[i]++;
    }
    uint32_t ldt(const uint32_t* p, int64_t i) {
        chk(p, 4 * i, 4);
        return ok ? p[i] : 0;
    }
    void stt(uint32_t* p, int64_t i, uint32_t v) {
        chk(p, 4 * i, 4);
        if (ok) p[i] = v;
    }
    void stf(float* p, int64_t i, float v) {
        chk(p, 4 * i, 4);
        if (!ok) return;
        p[i] = v;
        if (ybuf && (const unsigned char*)p == ybuf->base) ywrites[i]++;
    }
    void on_read(size_t h) {
        if (w_seg[h] == seg && w_tid[h] != tid) fail("LDS race: read of data another thread wrote");
        if (w_seg[h] < 0) fail("LDS read of data never written");
        if (r_seg[h] == seg && r_tid[h] != tid) r_multi[h] = 1;
        if (r_seg[h] != seg) r_multi[h] = 0;
        r_seg[h] = seg;
        r_tid[h] = tid;
    }
    void on_write(size_t h) {
        if (w_seg[h] == seg && w_tid[h] != tid) fail("LDS race: two threads write the same data");
        if (r_seg[h] == seg && (r_multi[h] || r_tid[h] != tid)) fail("LDS race: write of data another thread read");
        w_seg[h] = seg;
        w_tid[h] = tid;
    }
    bool lds_ok(int i) {
        if (i < 0 || i >= (int)lds.size()) fail("LDS access out of bounds");
        return ok;
    }
    uint32_t lr(int i) {
        if (!lds_ok(i)) return 0;
        on_read(2 * (size_t)i);
        on_read(2 * (size_t)i + 1);
        return lds[i];
    }
    uint16_t lr16(int i, int half) {
        if (!lds_ok(i)) return 0;
        on_read(2 * (size_t)i + half);
        return (uint16_t)(lds[i] >> (16 * half));
    }
    void lr4(int i, uint32_t* o) {
        if (i % 4) fail("misaligned 16-byte LDS read");
        for (int k = 0; k < 4; k++) o[k] = lr(i + k);
    }
    void lw(int i, uint32_t v) {
        if (!lds_ok(i)) return;
        on_write(2 * (size_t)i);
        on_write(2 * (size_t)i + 1);
        lds[i] = v;
    }
    void lw16(int i, int half, uint16_t v) {
        if (!lds_ok(i)) return;
        on_write(2 * (size_t)i + half);
        lds[i] = half ? (lds[i] & 0xffffu) | ((uint32_t)v << 16) : (lds[i] & 0xffff0000u) | v;
    }
    static float f(uint16_t h) {
        uint32_t u = (uint32_t)h << 16;
        float x;
        std::memcpy(&x, &u, 4);
        return x;
    }
    static uint32_t fbits(float v) {
        uint32_t u;
        std::memcpy(&u, &v, 4);
        return u;
    }
    static float fof(uint32_t u) {
        float x;
        std::memcpy(&x, &u, 4);
        return x;
    }
    static uint16_t rne(float v) {
        uint32_t u;
        std::memcpy(&u, &v, 4);
        if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
        u += 0x7fffu + ((u >> 16) & 1u);
        return (uint16_t)(u >> 16);
    }
    float dot2(uint32_t a, uint32_t b, float c) {
        return c + (f(a & 0xffff) * f(b & 0xffff) + f(a >> 16) * f(b >> 16));
    }
    uint32_t pk(float lo, float hi) { return (uint32_t)rne(lo) | ((uint32_t)rne(hi) << 16); }
    uint16_t bf(float v) { return rne(v); }
    // wave-wide ops: operands are recorded per lane; the runner computes the tile
    void mfma(const uint32_t* a, const uint32_t* b, float*) {
        std::array<uint32_t, 4> x, y;
        for (int k = 0; k < 4; k++) x[k] = a[k], y[k] = b[k];
        rec[tid % 64].push_back({x, y});
    }
    // lanes of a row arrive in order; the row's last lane writes the sum
    void rowsum(float x, int lane, int word) {
        if (!lds_ok(word)) return;
        if (lane % 16 == 0) rowacc[word] = 0.f;
        rowacc[word] += x;
        if (lane % 16 == 15) lw(word, fbits(rowacc[word]));
    }
};

// The 32x32x16 bf16 MFMA of one wave from the recorded operands: lane l gave
// A[l % 32][8 (l / 32) + i] and B[8 (l / 32) + i][l % 32] (element i of its
// four words) per call; lane l's result i is D[8 (i / 4) + 4 (l / 32) + i % 4][l % 32].
void emulate_mfma(RcpHost& m, std::vector<std::array<float, 16>>& acc) {
    const size_t calls = m.rec[0].size();
    for (int l = 0; l < 64; l++)
        if (m.rec[l].size() != calls) m.fail("MFMA call counts differ across a wave");
    std::vector<double> D(32 * 32, 0.0);
    auto el = [](const std::array<uint32_t, 4>& w, int i) { return RcpHost::f((uint16_t)(w[i / 2] >> (16 * (i % 2)))); };
    for (size_t c = 0; c < calls && m.ok; c++)
        for (int mm = 0; mm < 32; mm++)
            for (int nn = 0; nn < 32; nn++) {
                double s = 0;
                for (int k = 0; k < 16; k++)
                    s += (double)el(m.rec[mm + 32 * (k / 8)][c].first, k % 8) * el(m.rec[nn + 32 * (k / 8)][c].second, k % 8);
                D[mm * 32 + nn] += s;
            }
    acc.assign(64, {});
    for (int l = 0; l < 64; l++)
        for (int i = 0; i < 16; i++) acc[l][i] = (float)D[(8 * (i / 4) + 4 * (l / 32) + i % 4) * 32 + l % 32];
    for (auto& r : m.rec) r.clear();
}

template <class C>
bool rcp_blocks(const RcpDesc& d, RcpHost& m, const uint16_t* X, const uint16_t* W1, const uint16_t* W2,
                const uint16_t* W3, const uint16_t* W0, uint16_t* Y) {
    for (int i = 0; i < d.ntiles; i++) {
        const rcp::Tile t = rcp::tile_rows(d, i);
        if (rcp::units_a(d, t) > C::UA * C::NT || rcp::units_b(d, t) > C::UB * C::NT ||
            rcp::units_c(d, t) > C::UC * C::NT) {
            m.fail("tile units exceed the instantiation");
            return false;
        }
    }
    std::vector<rcp::State<C>> st(C::NT);
    for (int64_t blk = 0; blk < d.blocks && m.ok; blk++) {
        int b, t1, tile, chunk;
        rcp::block_coords(d, blk, b, t1, tile, chunk);
        if (b < 0 || b >= d.B || t1 < 0 || t1 >= d.T1 || tile < 0 || tile >= d.ntiles || chunk < 0 || chunk >= d.nc) {
            m.fail("block coordinates out of range");
            return false;
        }
        const rcp::Tile t = rcp::tile_rows(d, tile);
        m.reset_lds(m.lds.size());
        m.seg = 0;
        auto each = [&](auto&& fn) {
            for (int tid = 0; tid < C::NT; tid++) {
                m.tid = tid;
                fn(tid);
            }
            m.seg++;   // barrier
        };
        each([&](int tid) {
            rcp::init<C>(m, d, tid, b, t, X, st[tid]);
            rcp::phase_a<C>(m, d, t, 0, t1, chunk, 0, W1, W2, st[tid]);
        });
        const int np = d.R / 2;
        for (int rp = 0; rp < np; rp++) {
            const int r0 = 2 * rp;
            each([&](int tid) {
                rcp::phase_b<C>(m, d, t, r0, 0, W3, st[tid]);
                rcp::phase_a<C>(m, d, t, r0 + 1, t1, chunk, 1, W1, W2, st[tid]);
            });
            each([&](int tid) { rcp::phase_b<C>(m, d, t, r0 + 1, 1, W3, st[tid]); });
            each([&](int tid) {
                rcp::phase_c<C>(m, d, r0, W0, st[tid]);
                if (rp + 1 < np) rcp::phase_a<C>(m, d, t, r0 + 2, t1, chunk, 0, W1, W2, st[tid]);
            });
        }
        each([&](int tid) { rcp::store<C>(m, d, tid, b, t1, t, chunk, Y, st[tid]); });
    }
    return m.ok;
}

template <int I>
using RcpCfgOf = rcp::Cfg<kRcpCfgs[I].S1, kRcpCfgs[I].S2, kRcpCfgs[I].S3, kRcpCfgs[I].T2, kRcpCfgs[I].T3,
                          kRcpCfgs[I].K, kRcpCfgs[I].T2C, kRcpCfgs[I].NT, kRcpCfgs[I].UA, kRcpCfgs[I].UB,
                          kRcpCfgs[I].UC>;

template <class C>
bool rcp_is(const RcpDesc& d) {
    return d.S1 == C::S1 && d.S2 == C::S2 && d.S3 == C::S3 && d.T2 == C::T2 && d.T3 == C::T3 &&
           d.K == C::K && d.T2C == C::T2C && d.NT == C::NT;
}

bool run_rcp_fwd(const Launch& ln, Ctx& c) {
    RcpDesc d = desc_of<RcpDesc>(ln);
    REQ(((ln.kind >> kBitIn) & 1) == 1 && ln.extra.size() == 3, "bf16 only, five operands");
    bool o[6];
    Buf X = resolve(ln.a, c, 0, o[0]), W1 = resolve(ln.b, c, 0, o[1]), W2 = resolve(ln.extra[0], c, 0, o[2]),
        W3 = resolve(ln.extra[1], c, 0, o[3]), W0 = resolve(ln.extra[2], c, 0, o[4]), Y = resolve(ln.c, c, 0, o[5]);
    REQ(o[0] && o[1] && o[2] && o[3] && o[4] && o[5], "unresolved buffer");
    REQ(rcp::layout_ok(d), "LDS layout");
    REQ(d.blocks == (int64_t)d.B * d.T1 * d.ntiles * d.nc && (int64_t)ln.grid[0] == d.blocks &&
        (int)ln.block[0] == d.NT && ln.lds == d.lds_bytes && d.lds_bytes <= 160 * 1024, "grid / LDS");
    // operand sizes implied by the descriptor
    const int64_t HW = (int64_t)d.H * d.W;
    REQ(X.bytes >= (size_t)(2 * (int64_t)d.B * d.S1 * d.S2 * d.S3 * HW) &&
        Y.bytes >= (size_t)(2 * (int64_t)d.B * d.T1 * d.T2 * d.T3 * HW), "operand sizes");
    RcpHost m;
    m.reset_lds(d.lds_bytes / 4);
    m.g = {&X, &W1, &W2, &W3, &W0, &Y};
    m.ybuf = &Y;
    m.ywrites.assign(Y.bytes / 2, 0);
    const uint16_t *px = (const uint16_t*)X.base, *p1 = (const uint16_t*)W1.base, *p2 = (const uint16_t*)W2.base,
                   *p3 = (const uint16_t*)W3.base, *p0 = (const uint16_t*)W0.base;
    uint16_t* py = (uint16_t*)Y.base;
    bool ran = false;
    if (rcp_is<RcpCfgOf<0>>(d)) ran = rcp_blocks<RcpCfgOf<0>>(d, m, px, p1, p2, p3, p0, py), ran = true;
    else if (rcp_is<RcpCfgOf<1>>(d)) ran = rcp_blocks<RcpCfgOf<1>>(d, m, px, p1, p2, p3, p0, py), ran = true;
    REQ(ran, "no instantiation matches");
    REQ(m.ok, "rcp_fwd: " + m.err);
    const int64_t ny = (int64_t)d.B * d.T1 * d.T2 * d.T3 * HW;
    for (int64_t i = 0; i < ny; i++) REQ(m.ywrites[i] == 1, "a Y element is not written exactly once");
    return true;
}

// Fused reshaped-CP backward: the kernel's phases run on the CPU between its
// barriers (wave-wide MFMA and row sums emulated from the lanes' operands),
// with the same bounds and race checks; every element of the dX partials and
// of the four factor-gradient partial buffers must be written exactly once.
template <class C>
bool rcpb_blocks(const RcpBwdDesc& d, RcpHost& m, const uint16_t* X, const uint16_t* dY, const uint16_t* W1,
                 const uint16_t* W2, const uint16_t* W3, const uint16_t* W0, float* DXP, float* P0, float* P1,
                 float* P2, float* P3, const uint32_t* TB, std::vector<std::vector<int>>& counts,
                 const std::vector<const Buf*>& outs) {
    if (d.TH * d.W * C::S3 > C::UA * C::NT || d.TH * d.W * C::T2C > C::UB * C::NT ||
        C::T2C * C::T3 * d.TH * d.QW > C::UC * C::NT) {
        m.fail("tile units exceed the instantiation");
        return false;
    }
    std::vector<rcpb::State<C>> st(C::NT);
    std::vector<std::array<float, 16>> acc;
    (void)counts;
    (void)outs;
    for (int64_t bid = 0; bid < d.blocks && m.ok; bid++) {
        int64_t blk;
        int b, t1, tile, chunk, h0, h1;
        rcpb::block_coords_b(d, bid, blk, b, t1, tile, chunk);
        if (b < 0 || b >= d.B || t1 < 0 || t1 >= d.T1 || tile < 0 || tile >= d.ntiles || chunk < 0 ||
            chunk >= d.nc || blk < 0 || blk >= d.blocks) {
            m.fail("block coordinates out of range");
            return false;
        }
        rcpb::tile_of(d, tile, h0, h1);
        const int P = (h1 - h0) * d.W;
        m.reset_lds(m.lds.size());
        m.seg = 0;
        auto each = [&](auto&& fn) {
            for (int tid = 0; tid < C::NT; tid++) {
                m.tid = tid;
                fn(tid);
            }
        };
        auto waves = [&](int oA, int oB, int ld, int nk, int Mv, int Nv, int oslot, int slot_stride) {
            for (int w = 0; w < C::NW; w++) {
                for (int l = 0; l < 64; l++) {
                    m.tid = 64 * w + l;
                    float a16[16] = {};
                    rcpb::mfma_part<C>(m, l, w, oA, oB, ld, nk, Mv, Nv, a16);
                }
                emulate_mfma(m, acc);
                for (int l = 0; l < 64; l++) {
                    m.tid = 64 * w + l;
                    rcpb::mfma_store<C>(m, l, oslot + w * slot_stride, Mv, Nv, acc[l].data());
                }
            }
        };
        each([&](int tid) { rcpb::init<C>(m, d, tid, b, t1, h0, h1, chunk, X, dY, st[tid]); });
        m.seg++;
        for (int r = 0; r < d.R && m.ok; r++) {
            each([&](int tid) {
                rcpb::phase_a<C>(m, d, r, t1, chunk, W1, W2, st[tid]);
                if (r > 0) rcpb::phase_f<C>(m, d, tid, blk, r - 1, t1, chunk, P0, P1, P2, P3);
            });
            m.seg++;
            each([&](int tid) { rcpb::phase_b<C>(m, d, r, P, W3, st[tid]); });
            m.seg++;
            each([&](int tid) { rcpb::phase_c<C>(m, d, tid & 63, tid >> 6, r, P, TB, st[tid]); });
            m.seg++;
            each([&](int tid) { rcpb::phase_d<C>(m, d, r, TB, st[tid]); });
            waves(d.o_g3, d.o_z2, d.L2, C::T2C * d.PP / 16, C::T3, C::S3, d.o_m3, C::T3 * C::S3);
            m.seg++;
            each([&](int tid) { rcpb::phase_e<C>(m, d, tid & 63, tid >> 6, r, t1, chunk, TB, st[tid]); });
            waves(d.o_g2, d.o_z1, d.L13, C::S3 * d.PP / 16, C::T2C, C::S2, d.o_m2, C::T2C * C::S2);
            m.seg++;
        }
        each([&](int tid) {
            rcpb::phase_f<C>(m, d, tid, blk, d.R - 1, t1, chunk, P0, P1, P2, P3);
            rcpb::store_dx<C>(m, d, b, t1, h0, chunk, DXP, st[tid]);
        });
        m.seg++;
    }
    return m.ok;
}

template <int I>
using RcpBCfgOf = rcpb::Cfg<kRcpBwdCfgs[I].S1, kRcpBwdCfgs[I].S2, kRcpBwdCfgs[I].S3, kRcpBwdCfgs[I].T2,
                            kRcpBwdCfgs[I].T3, kRcpBwdCfgs[I].K, kRcpBwdCfgs[I].T2C, kRcpBwdCfgs[I].NT,
                            kRcpBwdCfgs[I].UA, kRcpBwdCfgs[I].UB, kRcpBwdCfgs[I].UC, kRcpBwdCfgs[I].MW>;

template <class C>
bool rcpb_is(const RcpBwdDesc& d) {
    return d.S1 == C::S1 && d.S2 == C::S2 && d.S3 == C::S3 && d.T2 == C::T2 && d.T3 == C::T3 &&
           d.K == C::K && d.T2C == C::T2C && d.NT == C::NT;
}

// The factor table of the fused backward: every word from rcpb::table_word.
bool run_rcp_prep(const Launch& ln, Ctx& c) {
    RcpBwdDesc d = desc_of<RcpBwdDesc>(ln);
    REQ(ln.extra.size() == 5, "five operands");
    Buf b[5];
    bool ok = true, o;
    for (int i = 0; i < 5; i++) {
        b[i] = resolve(ln.extra[i], c, 0, o);
        ok = ok && o;
    }
    REQ(ok, "unresolved buffer");
    const int64_t n = (int64_t)d.R * d.tbs;
    REQ(n > 0 && (int64_t)ln.grid[0] * 256 >= n && ln.block[0] == 256, "grid");
    RcpHost m;
    for (int i = 0; i < 5; i++) m.g.push_back(&b[i]);
    for (int64_t i = 0; i < n && m.ok; i++)
        m.stt((uint32_t*)b[4].base, i,
              rcpb::table_word(m, d, i, (const uint16_t*)b[0].base, (const uint16_t*)b[1].base,
                               (const uint16_t*)b[2].base, (const uint16_t*)b[3].base));
    REQ(m.ok, "rcp_prep: " + m.err);
    return true;
}

bool run_rcp_bwd(const Launch& ln, Ctx& c) {
    RcpBwdDesc d = desc_of<RcpBwdDesc>(ln);
    REQ(((ln.kind >> kBitIn) & 1) == 1 && ln.extra.size() == 10, "bf16 only, twelve operands");
    Buf bufs[12];
    bool ok = true, o;
    bufs[0] = resolve(ln.a, c, 0, o);
    ok = ok && o;
    bufs[1] = resolve(ln.b, c, 0, o);
    ok = ok && o;
    for (int i = 0; i < 10; i++) {
        bufs[2 + i] = resolve(ln.extra[i], c, 0, o);
        ok = ok && o;
    }
    REQ(ok, "unresolved buffer");
    REQ(rcpb::layout_ok_b(d), "LDS layout");
    REQ(d.blocks == (int64_t)d.B * d.T1 * d.ntiles * d.nc && (int64_t)ln.grid[0] == d.blocks &&
        (int)ln.block[0] == d.NT && ln.lds == d.lds_bytes && d.lds_bytes <= 160 * 1024, "grid / LDS");
    const int64_t HW = (int64_t)d.H * d.W, S = (int64_t)d.S1 * d.S2 * d.S3;
    const int64_t nslot = (int64_t)d.T1 * d.nc, nblk = d.blocks, KK = (int64_t)d.K * d.K;
    const int64_t need[5] = {nslot * d.B * S * HW, nblk * d.R * KK, nblk * d.R * d.T1 * d.S1,
                             nblk * d.R * d.T2 * d.S2, nblk * d.R * d.T3 * d.S3};
    for (int i = 0; i < 5; i++) REQ(bufs[6 + i].bytes >= (size_t)(4 * need[i]), "partial buffer size");
    REQ(bufs[11].bytes >= (size_t)(4 * (int64_t)d.R * d.tbs), "factor table size");
    RcpHost m;
    m.reset_lds(d.lds_bytes / 4);
    m.rec.assign(64, {});
    for (int i = 0; i < 12; i++) m.g.push_back(&bufs[i]);
    std::vector<std::vector<int>> counts(5);
    std::vector<const Buf*> outs;
    for (int i = 0; i < 5; i++) {
        counts[i].assign(need[i], 0);
        outs.push_back(&bufs[6 + i]);
    }
    auto u16 = [&](int i) { return (const uint16_t*)bufs[i].base; };
    auto f32 = [&](int i) { return (float*)bufs[i].base; };
    // poison the partial buffers so unwritten entries show up in the sums too
    for (int i = 6; i < 11; i++) std::memset(bufs[i].base, 0xFF, 4 * need[i - 6]);
    bool ran = false;
    if (rcpb_is<RcpBCfgOf<0>>(d))
        ran = true, rcpb_blocks<RcpBCfgOf<0>>(d, m, u16(0), u16(1), u16(2), u16(3), u16(4), u16(5), f32(6), f32(7),
                                              f32(8), f32(9), f32(10), (const uint32_t*)bufs[11].base, counts, outs);
    else if (rcpb_is<RcpBCfgOf<1>>(d))
        ran = true, rcpb_blocks<RcpBCfgOf<1>>(d, m, u16(0), u16(1), u16(2), u16(3), u16(4), u16(5), f32(6), f32(7),
                                              f32(8), f32(9), f32(10), (const uint32_t*)bufs[11].base, counts, outs);
    REQ(ran, "no instantiation matches");
    REQ(m.ok, "rcp_bwd: " + m.err);
    // every partial written (no 0xFFFFFFFF NaN pattern left)
    for (int i = 0; i < 5; i++) {
        const uint32_t* w = (const uint32_t*)bufs[6 + i].base;
        for (int64_t k = 0; k < need[i]; k++) REQ(w[k] != 0xFFFFFFFFu, "a partial is never written");
    }
    return true;
}


// Fused CP backward: every gradient of the chain in double; dX written (when
// wanted), the factor-gradient totals put in block 0 of the partials and
// zeros in every other block (the reduce launches then sum them).
bool run_cp_bwd(const Launch& ln, Ctx& c) {
    CpBwdDesc d = desc_of<CpBwdDesc>(ln);
    int bf = (ln.kind >> kBitIn) & 1;
    REQ(ln.extra.size() == 8, "operand count");
    bool ok1, ok2, ok3;
    Buf X = resolve(ln.a, c, 0, ok1), dY = resolve(ln.b, c, 0, ok2), dX = resolve(ln.c, c, 0, ok3);
    REQ(ok1 && ok2 && ok3, "unresolved buffer");
    Buf F[8];
    for (int i = 0; i < 8; i++) {
        bool o;
        F[i] = resolve(ln.extra[i], c, 0, o);
        REQ(o, "unresolved buffer");
    }
    Buf &Us = F[0], &Kh = F[1], &Kw = F[2], &Ut = F[3], &Pus = F[4], &Put = F[5], &Pkh = F[6], &Pkw = F[7];
    REQ(d.R >= 1 && d.R <= 32 && d.S >= 1 && d.T >= 1 && d.T <= 64 && (d.S + 31) / 32 == (d.T + 31) / 32 &&
        d.KH == 3 && d.KW == 3, "sizes");
    REQ(d.colstride == 32 - (d.KW - 1) && (int64_t)d.ncb * d.colstride >= d.W &&
        (int64_t)(d.ncb - 1) * d.colstride < d.W, "strips");
    REQ((int64_t)d.segs * d.seg_rows >= d.H && (int64_t)(d.segs - 1) * d.seg_rows < d.H, "segments");
    REQ(d.waves == (int64_t)d.B * d.ncb * d.segs && d.blocks * 4 >= d.waves && d.blocks * 4 < d.waves + 4 &&
        (int64_t)ln.grid[0] == d.blocks && ln.block[0] == 256, "grid");
    // LDS: tables, transpose tiles, dY tiles, reduction area
    const uint64_t e = bf ? 2 : 4;
    const uint64_t SP = 32 * ((d.S + 31) / 32), TP = 32 * ((d.T + 31) / 32);   // padded channel blocks
    REQ(d.lda_s >= SP + (bf ? 8 : 1) && d.lda_t >= TP + (bf ? 8 : 1) &&
        (!bf || ((d.lda_s * 2) % 16 == 0 && (d.lda_t * 2) % 16 == 0)), "table rows");
    REQ(d.o_uta >= 32 * d.lda_s * e && d.o_uta % 16 == 0, "UtA offset");
    REQ(d.o_ust >= d.o_uta + 32 * d.lda_t * e && d.o_ust % 16 == 0, "UsT offset");
    REQ(!bf || (d.ldu >= 32 + 8 && (d.ldu * 2) % 16 == 0), "UsT rows");
    REQ(d.o_tz >= d.o_ust + (bf ? (uint64_t)SP * d.ldu * 2 : 0) && d.o_tz % 16 == 0, "tile offset");
    REQ(d.ly >= 32 + (bf ? 8 : 1) && (!bf || (d.ly * 2) % 8 == 0), "dY tile rows");
    REQ(d.yt_bytes >= (uint64_t)TP * d.ly * e && d.yt_bytes % 16 == 0 && d.o_yt % 16 == 0, "dY tiles");
    REQ(d.tz_stride >= 32 * 33 * 4 && d.tz_stride % 16 == 0, "transpose tiles");
    if (d.o_tz == d.o_yt)   // the transpose tile shares the wave's dY tile
        REQ(d.tz_stride == d.yt_bytes, "shared tiles");
    else
        REQ(d.o_yt >= d.o_tz + 4 * (uint64_t)d.tz_stride, "tile regions");
    // X-row rings: three rows of S channels, aligned column runs
    REQ(d.lx >= 32 + (bf ? 8 : 4) && (d.lx * e) % (bf ? 8 : 16) == 0 && d.o_xl % 16 == 0 &&
        d.xl_bytes >= 3 * SP * d.lx * e && d.xl_bytes % 16 == 0, "X rings");
    REQ(d.o_xl >= d.o_yt + 4 * (uint64_t)d.yt_bytes && d.lds_bytes >= d.o_xl + 4 * (uint64_t)d.xl_bytes,
        "LDS tiles");
    REQ(d.red_bytes >= (uint64_t)4 * std::max({(uint64_t)4 * 32 * SP, (uint64_t)4 * 32 * TP,
                                               (uint64_t)8 * 32 * (d.KH + d.KW)}) &&
        d.lds_bytes >= d.red_bytes && d.lds_bytes <= 160 * 1024 && ln.lds == d.lds_bytes, "LDS size");
    const int B = d.B, S = d.S, R = d.R, T = d.T, H = d.H, W = d.W, K = d.KH, c3 = (K - 1) / 2;
    const size_t HW = (size_t)H * W;
    bool ok = true;
    std::vector<double> gus((size_t)R * S, 0), gut((size_t)R * T, 0), gkh((size_t)R * K, 0),
        gkw((size_t)R * K, 0);
    std::vector<double> z1(R * HW), z2(R * HW), z3(R * HW), g3(R * HW), g2(R * HW), g1(R * HW);
    auto us = [&](int r, int s2) { return (double)ld(Us, bf, (int64_t)r * d.us_sr + (int64_t)s2 * d.us_ss, ok); };
    auto ut = [&](int r, int t) { return (double)ld(Ut, bf, (int64_t)r * d.ut_sr + (int64_t)t * d.ut_st, ok); };
    auto kh = [&](int r, int j) { return (double)ld(Kh, bf, (int64_t)r * d.kh_sr + (int64_t)j * d.kh_sj, ok); };
    auto kw = [&](int r, int j) { return (double)ld(Kw, bf, (int64_t)r * d.kw_sr + (int64_t)j * d.kw_sj, ok); };
    for (int b = 0; b < B; b++) {
        for (int r = 0; r < R; r++)
            for (size_t p = 0; p < HW; p++) {
                double a = 0, g = 0;
                for (int s2 = 0; s2 < S; s2++) a += us(r, s2) * ld(X, bf, (int64_t)b * d.x_sb + (int64_t)s2 * d.x_ss + p, ok);
                for (int t = 0; t < T; t++) g += ut(r, t) * ld(dY, bf, (int64_t)b * d.y_sb + (int64_t)t * d.y_st + p, ok);
                z1[r * HW + p] = a;
                g3[r * HW + p] = g;
            }
        for (int r = 0; r < R; r++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    double a = 0;
                    for (int j = 0; j < K; j++) {
                        int hh = h + j - c3;
                        if (hh >= 0 && hh < H) a += kh(r, j) * z1[r * HW + hh * W + w];
                    }
                    z2[r * HW + h * W + w] = a;
                }
        for (int r = 0; r < R; r++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    double a = 0, g = 0;
                    for (int j = 0; j < K; j++) {
                        int ww = w + j - c3;
                        if (ww >= 0 && ww < W) a += kw(r, j) * z2[r * HW + h * W + ww];
                        int wg = w - j + c3;   // transposed conv along w
                        if (wg >= 0 && wg < W) g += kw(r, j) * g3[r * HW + h * W + wg];
                    }
                    z3[r * HW + h * W + w] = a;
                    g2[r * HW + h * W + w] = g;
                }
        for (int r = 0; r < R; r++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    double g = 0;
                    for (int j = 0; j < K; j++) {
                        int hg = h - j + c3;
                        if (hg >= 0 && hg < H) g += kh(r, j) * g2[r * HW + hg * W + w];
                        int hh = h + j - c3, ww = w + j - c3;
                        if (hh >= 0 && hh < H) gkh[r * K + j] += z1[r * HW + hh * W + w] * g2[r * HW + h * W + w];
                        if (ww >= 0 && ww < W) gkw[r * K + j] += z2[r * HW + h * W + ww] * g3[r * HW + h * W + w];
                    }
                    g1[r * HW + h * W + w] = g;
                }
        for (size_t p = 0; p < HW; p++) {
            for (int t = 0; t < T; t++) {
                double dy = ld(dY, bf, (int64_t)b * d.y_sb + (int64_t)t * d.y_st + p, ok);
                for (int r = 0; r < R; r++) gut[r * T + t] += z3[r * HW + p] * dy;
            }
            for (int s2 = 0; s2 < S; s2++) {
                double x = ld(X, bf, (int64_t)b * d.x_sb + (int64_t)s2 * d.x_ss + p, ok);
                double a = 0;
                for (int r = 0; r < R; r++) {
                    a += us(r, s2) * g1[r * HW + p];
                    gus[r * S + s2] += g1[r * HW + p] * x;
                }
                if (dX.base) st(dX, bf, (int64_t)b * d.x_sb + (int64_t)s2 * d.x_ss + p, (float)a, ok);
            }
        }
        REQ(ok, "out-of-bounds access (cp_bwd)");
    }
    for (int64_t blk = 0; blk < d.blocks; blk++) {
        for (int i = 0; i < R * S; i++) st(Pus, 0, blk * R * S + i, blk ? 0.f : (float)gus[i], ok);
        for (int i = 0; i < R * T; i++) st(Put, 0, blk * R * T + i, blk ? 0.f : (float)gut[i], ok);
        for (int i = 0; i < R * K; i++) st(Pkh, 0, blk * R * K + i, blk ? 0.f : (float)gkh[i], ok);
        for (int i = 0; i < R * K; i++) st(Pkw, 0, blk * R * K + i, blk ? 0.f : (float)gkw[i], ok);
    }
    REQ(ok, "out-of-bounds partials (cp_bwd)");
    return true;
}

// General contraction: C (or the chunk partials) from the descriptor's dim
// lists, in double, every access bounds-checked.
bool run_tc(const Launch& ln, Ctx& c) {
    TcDesc d = desc_of<TcDesc>(ln);
    int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    bool o1, o2;
    Buf A = resolve(ln.a, c, 0, o1), B = resolve(ln.b, c, 0, o2);
    REQ(o1 && o2, "unresolved buffer");
    REQ(d.ng <= 4 && d.nm <= 4 && d.nn <= 4 && d.nk <= 4 && d.ncv <= 2 && d.ksplit >= 1, "dims");
    int64_t Mt = 1, Nt = 1, Kt = 1, Gt = 1;
    for (int i = 0; i < d.nm; i++) Mt *= d.m_size[i];
    for (int i = 0; i < d.nn; i++) Nt *= d.n_size[i];
    for (int i = 0; i < d.nk; i++) Kt *= d.k_size[i];
    for (int i = 0; i < d.ng; i++) Gt *= d.g_size[i];
    REQ(Mt == d.M && Nt == d.N && Kt == d.K && Gt == d.G, "totals");
    REQ(d.kchunk % 32 == 0 && d.kchunk * (d.ksplit - 1) < d.K && d.kchunk * d.ksplit >= d.K, "split");
    const int MT = d.M > 32 ? 2 : 1;
    REQ(d.mtiles == (d.M + 32 * MT - 1) / (32 * MT) && d.ntiles == (d.N + 127) / 128 &&
        d.blocks == d.G * d.mtiles * d.ntiles * d.ksplit && (int64_t)ln.grid[0] == d.blocks &&
        ln.block[0] == 256, "grid");
    // tap bitmasks: at most 32 combinations of the convolved reduction indices,
    // which are the k dims marked as convolved
    if (d.tapmask) {
        int64_t Jc[2] = {1, 1};
        for (int i = 0; i < d.nk; i++)
            if (d.k_cv[i] >= 0) Jc[d.k_cv[i]] = d.k_size[i];
        REQ(d.ncv >= 1 && d.tapJ1 == (d.ncv > 1 ? Jc[1] : 1) && Jc[0] * Jc[1] <= 32, "tap masks");
    }
    // 31-bit offsets: the buffer ranges lie inside the operands' buffers
    const int esz = tIn ? 2 : 4;
    REQ(!d.off32 || (d.extA < ((int64_t)1 << 31) && d.extB < ((int64_t)1 << 31) && (size_t)d.extA <= A.bytes &&
                     (size_t)d.extB <= B.bytes && d.extA % esz == 0 && d.extB % esz == 0), "31-bit ranges");
    for (int i = 0; i < d.nn; i++) REQ(d.n_cv[i] < d.ncv && (d.n_cv[i] < 0 || d.n_sB[i] == 0), "conv n dims");
    for (int i = 0; i < d.nk; i++) REQ(d.k_cv[i] < d.ncv && (d.k_cv[i] < 0 || d.k_sB[i] == 0), "conv k dims");
    Buf Cb, Pb;
    if (d.ksplit == 1) {
        bool o3;
        Cb = resolve(ln.c, c, 0, o3);
        REQ(o3, "unresolved buffer");
    } else {
        bool o4;
        Pb = resolve(ln.d, c, 0, o4);
        REQ(o4, "unresolved buffer");
    }
    bool ok = true;
    std::vector<int64_t> gi(4), mi(4), ni(4), ki(4);
    auto split = [](int64_t x, int nd, const int64_t* size, std::vector<int64_t>& idx) {
        for (int i = nd - 1; i >= 0; --i) {
            idx[i] = x % size[i];
            x /= size[i];
        }
    };
    for (int64_t g = 0; g < d.G; g++) {
        split(g, d.ng, d.g_size, gi);
        int64_t gA = 0, gB = 0, gC = 0;
        for (int i = 0; i < d.ng; i++) {
            gA += gi[i] * d.g_sA[i];
            gB += gi[i] * d.g_sB[i];
            gC += gi[i] * d.g_sC[i];
        }
        for (int64_t m = 0; m < d.M; m++) {
            split(m, d.nm, d.m_size, mi);
            int64_t oA = gA, oC = gC;
            for (int i = 0; i < d.nm; i++) {
                oA += mi[i] * d.m_sA[i];
                oC += mi[i] * d.m_sC[i];
            }
            for (int64_t n = 0; n < d.N; n++) {
                split(n, d.nn, d.n_size, ni);
                int64_t oB = gB, oCn = oC, p[2] = {0, 0};
                for (int i = 0; i < d.nn; i++) {
                    oB += ni[i] * d.n_sB[i];
                    oCn += ni[i] * d.n_sC[i];
                    if (d.n_cv[i] >= 0) p[d.n_cv[i]] = ni[i];
                }
                for (int ks = 0; ks < d.ksplit; ks++) {
                    double acc = 0;
                    for (int64_t k = ks * d.kchunk; k < std::min(d.K, (ks + 1) * d.kchunk); k++) {
                        split(k, d.nk, d.k_size, ki);
                        int64_t a = oA, b = oB, j[2] = {0, 0};
                        for (int i = 0; i < d.nk; i++) {
                            a += ki[i] * d.k_sA[i];
                            b += ki[i] * d.k_sB[i];
                            if (d.k_cv[i] >= 0) j[d.k_cv[i]] = ki[i];
                        }
                        bool in = true;
                        for (int cv = 0; cv < d.ncv; cv++) {
                            int64_t pos = d.cv_a[cv] * p[cv] + d.cv_b[cv] * j[cv] + d.cv_g[cv];
                            if (pos < 0 || pos >= d.cv_lim[cv]) in = false;
                            b += pos * d.cv_s[cv];
                        }
                        if (in && d.off32 && (a * esz >= d.extA || b * esz >= d.extB)) ok = false;
                        if (in) acc += (double)ld(A, tIn, a, ok) * ld(B, tIn, b, ok);
                    }
                    if (d.off32 && oCn >= ((int64_t)1 << 31)) ok = false;
                    if (d.ksplit == 1) st(Cb, tC, oCn, (float)acc, ok);
                    else st(Pb, 0, ((g * d.ksplit + ks) * d.M + m) * d.N + n, (float)acc, ok);
                }
            }
        }
        REQ(ok, "out-of-bounds access (tc)");
    }
    return true;
}

bool run_tc_reduce(const Launch& ln, Ctx& c) {
    TcDesc d = desc_of<TcDesc>(ln);
    int tC = (ln.kind >> kBitOut) & 1;
    bool o1, o2;
    Buf P = resolve(ln.d, c, 0, o1), C = resolve(ln.c, c, 0, o2);
    REQ(o1 && o2, "unresolved buffer");
    const int64_t per = d.ksplit <= 8 ? 256 : 64;   // outputs of one g a block
    REQ((int64_t)ln.grid[0] == d.G * ((d.M * d.N + per - 1) / per) && ln.block[0] == 256, "grid");
    bool ok = true;
    for (int64_t g = 0; g < d.G; g++)
        for (int64_t m = 0; m < d.M; m++)
            for (int64_t n = 0; n < d.N; n++) {
                int64_t off = 0, x = g;
                for (int i = d.ng - 1; i >= 0; --i) { off += (x % d.g_size[i]) * d.g_sC[i]; x /= d.g_size[i]; }
                x = m;
                for (int i = d.nm - 1; i >= 0; --i) { off += (x % d.m_size[i]) * d.m_sC[i]; x /= d.m_size[i]; }
                x = n;
                for (int i = d.nn - 1; i >= 0; --i) { off += (x % d.n_size[i]) * d.n_sC[i]; x /= d.n_size[i]; }
                double s = 0;
                for (int ks = 0; ks < d.ksplit; ks++) s += ld(P, 0, ((g * d.ksplit + ks) * d.M + m) * d.N + n, ok);
                st(C, tC, off, (float)s, ok);
            }
    REQ(ok, "out-of-bounds access (tc reduce)");
    return true;
}
// Plane convolution contracted over one index (K_CRED forward, K_CREDW
// partials, K_CREDW_REDUCE chunk sum): the kernels' thread mapping, with
// their LDS plane indices checked against the block's allocation, in double.
// K_CCONV: the launcher's descriptor checks, then the sum it defines (every
// operand read bounds-checked).
bool run_cconv(const Launch& ln, Ctx& c) {
    CconvDesc d = desc_of<CconvDesc>(ln);
    const int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    const int CB = d.Ppad / (tIn ? 16 : 8);
    REQ(tIn == 1 || tC == 0, "fp32 inputs give fp32 outputs");
    if (d.rega) {
        // fp32, P <= 8, at most nine taps, input rows alone in LDS, every q
        // tile in one block; its stores span y_ext elements from the g's base
        REQ(!tIn && d.Ppad == 8 && d.P >= 1 && d.P <= 8 && d.pw_img == 9 && d.KH * d.KW <= 9 && d.TH >= 1 &&
                d.HP == d.TH + d.KH - 1 && d.WP == d.W + d.KW - 1 && d.nq >= 1 && d.nq * 32 >= d.Q &&
                (int64_t)d.ntiles * d.TH >= d.H && d.y_sq >= 1 &&
                d.y_ext == (int64_t)(d.Q - 1) * d.y_sq + (int64_t)d.H * d.W && d.y_ext * 4 < (1ll << 31) &&
                d.lds_bytes == 4u * (uint32_t)(d.HP * d.WP * d.pw_img) && d.lds_bytes <= 160 * 1024 &&
                (int64_t)ln.grid[0] == d.G * d.ntiles && d.blocks == (int64_t)ln.grid[0] && ln.block[0] == 256 &&
                ln.lds == d.lds_bytes,
            "cconv_r layout");
    }
    const bool lay = tIn ? (d.Ppad == 16 * CB && d.pw_img == 8 * CB + 4 && d.tp == 8 * CB + 4 && (d.pw_tab & 3) == 0)
                         : (d.Ppad == 8 * CB && d.pw_img == 8 * CB + 1 && d.tp == 8 * CB && (d.pw_tab & 1) == 1);
    REQ(d.rega || ((CB == 1 || CB == 2 || CB == 4 || CB == 8) && lay && d.TH >= 1 && d.HP == d.TH + d.KH - 1 &&
            d.WP == d.W + d.KW - 1 && d.pw_tab >= d.KH * d.KW * d.tp &&
            d.P <= d.Ppad && d.nq * 32 >= d.Q && (int64_t)d.ntiles * d.TH >= d.H &&
            d.lds_bytes == 4u * (uint32_t)(32 * d.pw_tab + d.HP * d.WP * d.pw_img) && d.lds_bytes <= 160 * 1024 &&
            (int64_t)ln.grid[0] == d.G * d.ntiles * d.nq && d.blocks == (int64_t)ln.grid[0] && ln.block[0] == 256 &&
            ln.lds == d.lds_bytes),
        "cconv layout");
    REQ((d.zhs == 1 || d.zhs == -1) && (d.zws == 1 || d.zws == -1) && (d.fhs == 1 || d.fhs == -1) &&
            (d.fws == 1 || d.fws == -1) && d.ng >= 0 && d.ng <= 2 && d.z_numel > 0 && d.z_numel < (1ll << 30) &&
            d.f_numel > 0 && d.f_numel < (1ll << 30),
        "cconv taps");
    bool ok = true, o1, o2, o3;
    Buf Z = resolve(ln.a, c, 0, o1), F = resolve(ln.b, c, 0, o2), Y = resolve(ln.c, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    const size_t E = tIn ? 2 : 4;
    REQ((size_t)d.z_numel * E <= Z.bytes && (size_t)d.f_numel * E <= F.bytes, "cconv load ranges");
    for (int64_t g = 0; g < d.G; g++) {
        int64_t oz = 0, oy = 0, x = g;
        for (int i = d.ng - 1; i >= 0; --i) {
            oz += (x % d.g_size[i]) * d.g_sZ[i];
            oy += (x % d.g_size[i]) * d.g_sY[i];
            x /= d.g_size[i];
        }
        for (int q = 0; q < d.Q; q++)
            for (int h = 0; h < d.H; h++)
                for (int w = 0; w < d.W; w++) {
                    double acc = 0;
                    for (int th = 0; th < d.KH; th++)
                        for (int tw = 0; tw < d.KW; tw++) {
                            const int hh = h + d.zh0 + d.zhs * th, ww = w + d.zw0 + d.zws * tw;
                            if (hh < 0 || hh >= d.H || ww < 0 || ww >= d.W) continue;
                            const int64_t fo = q * d.f_sq + (int64_t)(d.fh0 + d.fhs * th) * d.f_sh +
                                               (int64_t)(d.fw0 + d.fws * tw) * d.f_sw;
                            for (int p = 0; p < d.P; p++)
                                acc += (double)ld(Z, tIn, oz + p * d.z_sp + (int64_t)hh * d.W + ww, ok) *
                                       ld(F, tIn, fo + p * d.f_sp, ok);
                        }
                    const int64_t yo = q * d.y_sq + (int64_t)h * d.W + w;
                    if (d.rega) REQ(yo >= 0 && yo < d.y_ext, "cconv_r store range");
                    st(Y, tC, oy + yo, (float)acc, ok);
                }
        REQ(ok, "out-of-bounds access (cconv)");
    }
    return true;
}

// K_TT_FWD: the launcher's descriptor checks, then the two sums it defines
// (Z of one (b, g, u) at a time), every operand access bounds-checked.
bool run_tt_fwd(const Launch& ln, Ctx& c) {
    TtDesc d = desc_of<TtDesc>(ln);
    const int n1 = (d.K1 + 3) / 4;
    const int XT = d.XT, PW = 16 * XT + 2, plane = ((6 * PW - 16 + 63) / 64) * 64 + 16;
    REQ(n1 >= 1 && n1 <= 16 && d.R == 16 && d.T >= 1 && d.T <= 8 && d.TH == 4 && d.U >= 1 && d.G >= 1 &&
            d.B >= 1 && d.H >= 1 && d.W >= 1 && (XT == 1 || XT == 2 || XT == 4) && d.W <= 16 * XT &&
            d.PW == PW && d.plane == plane && plane >= 6 * PW && d.lds_bytes == (uint32_t)(16 * plane * 4) &&
            d.ncombo == 2 * XT && (int64_t)d.nbands * 4 >= d.H && d.blocks == (int64_t)d.B * d.G * d.nbands &&
            ((ln.kind & 0xff) == K_TT_PREP ||
             ((int64_t)ln.grid[0] == d.blocks && ln.block[0] == 256 && ln.lds == d.lds_bytes)) &&
            (!d.xcd_remap || d.blocks % 8 == 0) && d.x_numel > 0 && d.x_numel < (1ll << 29) &&
            d.f1_numel > 0 && d.f1_numel < (1ll << 29) && d.f2_numel > 0 && d.f2_numel < (1ll << 29),
        "tt_fwd layout");
    REQ(ln.extra.size() == 2, "tt_fwd operands");
    bool ok = true, o1, o2, o3, o4, o5;
    Buf X = resolve(ln.a, c, 0, o1), F1 = resolve(ln.b, c, 0, o2), F2 = resolve(ln.extra[0], c, 0, o3),
        Y = resolve(ln.c, c, 0, o4), A2 = resolve(ln.extra[1], c, 0, o5);
    REQ(o1 && o2 && o3 && o4 && o5, "unresolved buffer");
    REQ((size_t)d.U * 48 * 64 * 4 <= A2.bytes, "tt_fwd operand table");
    if ((ln.kind & 0xff) == K_TT_PREP) {
        // the table the main launch reads: F2 placed at the tap rows of row pairs
        REQ((int64_t)ln.grid[0] * 256 >= (int64_t)d.U * 48 * 64 && ln.block[0] == 256, "tt_prep grid");
        for (int64_t i = 0; i < (int64_t)d.U * 48 * 64; i++) {
            const int j = (int)(i & 3), lane = (int)((i >> 2) & 63);
            const int s4 = (int)((i >> 8) % 12), u = (int)((i >> 8) / 12), s2 = 4 * s4 + j;
            const int q = lane >> 4, c16 = lane & 15, t3 = c16 & 7, dy = c16 >> 3;
            const int rh = s2 & 3, kw = (s2 >> 2) % 3, khp = (s2 >> 2) / 3, kh = khp - dy;
            float v = 0.f;
            if (t3 < d.T && kh >= 0 && kh < 3)
                v = ld(F2, 0, t3 * d.f2_st + u * d.f2_su + (4 * rh + q) * d.f2_sr + kh * d.f2_sh + kw * d.f2_sw, ok);
            st(A2, 0, i, v, ok);
        }
        REQ(ok, "out-of-bounds access (tt_prep)");
        return true;
    }
    REQ((size_t)d.x_numel * 4 <= X.bytes && (size_t)d.f1_numel * 4 <= F1.bytes && (size_t)d.f2_numel * 4 <= F2.bytes,
        "tt_fwd load ranges");
    const int64_t HW = (int64_t)d.H * d.W;
    std::vector<double> z((size_t)d.R * HW), y((size_t)d.T * HW);
    for (int64_t b = 0; b < d.B; b++)
        for (int g = 0; g < d.G; g++) {
            std::fill(y.begin(), y.end(), 0.0);
            for (int u = 0; u < d.U; u++) {
                std::fill(z.begin(), z.end(), 0.0);
                for (int k = 0; k < d.K1; k++)
                    for (int r = 0; r < d.R; r++) {
                        const double f = ld(F1, 0, g * d.f1_sg + k * d.f1_sk + r * d.f1_sr, ok);
                        const int64_t xo = b * d.x_sb + k * d.x_sk + u * d.x_su;
                        for (int64_t p = 0; p < HW; p++) z[r * HW + p] += f * ld(X, 0, xo + p, ok);
                    }
                for (int t = 0; t < d.T; t++)
                    for (int r = 0; r < d.R; r++)
                        for (int kh = 0; kh < 3; kh++)
                            for (int kw = 0; kw < 3; kw++) {
                                const double f = ld(F2, 0, t * d.f2_st + u * d.f2_su + r * d.f2_sr + kh * d.f2_sh +
                                                                kw * d.f2_sw, ok);
                                for (int h = 0; h < d.H; h++)
                                    for (int w = 0; w < d.W; w++) {
                                        const int hh = h + kh - 1, ww = w + kw - 1;
                                        if (hh < 0 || hh >= d.H || ww < 0 || ww >= d.W) continue;
                                        y[t * HW + h * d.W + w] += f * z[r * HW + hh * d.W + ww];
                                    }
                            }
            }
            for (int t = 0; t < d.T; t++)
                for (int64_t p = 0; p < HW; p++)
                    st(Y, 0, b * d.y_sb + g * d.y_sg + t * d.y_st + p, (float)y[t * HW + p], ok);
            REQ(ok, "out-of-bounds access (tt_fwd)");
        }
    return true;
}

bool run_cred(const Launch& ln, Ctx& c) {
    CredDesc d = desc_of<CredDesc>(ln);
    const int kind = ln.kind & 0xff;
    const bool wgrad = kind == K_CREDW;
    int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    const int KK = d.KH * d.KW, MO = d.M == 1 ? 1 : d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16;
    REQ(d.M >= 1, "channels");
    bool ok = true, o1, o2, o3;
    if (kind == K_CREDW_REDUCE) {
        Buf Pb = resolve(ln.d, c, 0, o1), Cb = resolve(ln.c, c, 0, o2);
        REQ(o1 && o2, "unresolved buffer");
        const int64_t per_chunk = d.R * d.M * KK;
        REQ((int64_t)ln.grid[0] * 64 >= per_chunk && ln.block[0] == 256, "grid");   // 64 outputs per block
        for (int64_t r = 0; r < d.R; r++)
            for (int m = 0; m < d.M; m++)
                for (int k = 0; k < KK; k++) {
                    double sum = 0;
                    for (int64_t ck = 0; ck < d.nchunks; ck++)
                        sum += ld(Pb, 0, ck * per_chunk + (r * d.M + m) * KK + k, ok);
                    st(Cb, tC, m * d.c_sm + r * d.c_sr + (k / d.KW) * d.c_sh + (k % d.KW) * d.c_sw, (float)sum, ok);
                }
        REQ(ok, "out-of-bounds access (credw reduce)");
        return true;
    }
    REQ(d.M <= 16, "channels");
    Buf Z = resolve(wgrad ? ln.a : ln.b, c, 0, o1), O = resolve(wgrad ? ln.b : ln.a, c, 0, o2);
    Buf Y = resolve(wgrad ? ln.d : ln.c, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    REQ(wgrad || tIn == tC, "forward output type");
    REQ(!wgrad || (KK <= 25 && MO <= 8 && MO * KK <= 72), "gradient registers");
    const int n4 = (4 + d.KW - 1 + 3) / 4;
    REQ(d.wchunks == (d.W + 3) / 4 && d.items == d.H * d.wchunks && d.PH == d.H + d.KH - 1 &&
        d.PWp % 4 == 0 && d.PWp >= d.W + d.KW - 1 && d.PWp >= 4 * (d.wchunks - 1) + 4 * n4, "plane");
    REQ(d.ch >= 0 && d.ch < d.KH && d.cw >= 0 && d.cw < d.KW && d.ng <= 2 && d.per >= 1, "pads");
    const int64_t plane = (int64_t)d.PH * d.PWp;
    const uint32_t maxthreads = wgrad && MO >= 4 ? 512 : 1024;   // the kernels' launch bounds
    REQ((int64_t)d.threads % 64 == 0 && d.threads <= maxthreads && (int64_t)d.threads >= (int64_t)d.per * d.items &&
        ln.block[0] == d.threads && (int64_t)ln.grid[0] == d.blocks, "grid");
    REQ((int64_t)d.lds_bytes >= 2 * d.per * plane * 4 && d.lds_bytes <= 160 * 1024 &&
        (!wgrad || (int64_t)d.lds_bytes >= (int64_t)d.threads * KK * 4), "lds");
    // the last LDS word any thread writes or reads
    const int64_t wr_max = (int64_t)(d.per - 1) * plane + (d.H - 1 + d.ch) * d.PWp + 4 * (d.wchunks - 1) + d.cw + 3;
    const int64_t rd_max = (int64_t)(d.per - 1) * plane + (d.H - 1 + d.KH - 1) * d.PWp + 4 * (d.wchunks - 1) + 4 * n4 - 1;
    REQ(d.per * plane + std::max(wr_max, rd_max) < 2 * d.per * plane, "lds range");
    if (!wgrad) REQ(d.blocks * d.per >= d.G && (d.blocks - 1) * d.per < d.G, "grid (batch)");
    else REQ(d.nrb * d.per >= d.R && (d.nrb - 1) * d.per < d.R && d.gchunk >= 1 &&
             d.nchunks == (d.G + d.gchunk - 1) / d.gchunk && d.blocks == d.nrb * d.nchunks, "grid (ranks)");
    auto offs = [&](int64_t g, int64_t& oz, int64_t& oy) {
        oz = oy = 0;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t x = g % d.g_size[i];
            g /= d.g_size[i];
            oz += x * d.g_sZ[i];
            oy += x * d.g_sY[i];
        }
    };
    // Z at in-plane position (h, w) of batch offset oz and rank r, zero outside
    auto zat = [&](int64_t oz, int64_t r, int64_t h, int64_t w) -> double {
        if (h < 0 || h >= d.H || w < 0 || w >= d.W) return 0.0;
        return ld(Z, tIn, oz + r * d.z_sr + h * d.W + w, ok);
    };
    if (!wgrad) {
        for (int64_t b = 0; b < d.blocks; b++)
            for (int64_t gl = 0; gl < d.per; gl++) {
                const int64_t g = b * d.per + gl;
                if (g >= d.G) continue;
                int64_t oz, oy;
                offs(g, oz, oy);
                for (int m = 0; m < d.M; m++)
                    for (int64_t oh = 0; oh < d.H; oh++)
                        for (int64_t ow = 0; ow < d.W; ow++) {
                            double acc = 0;
                            for (int64_t r = 0; r < d.R; r++)
                                for (int jh = 0; jh < d.KH; jh++)
                                    for (int jw = 0; jw < d.KW; jw++)
                                        acc += zat(oz, r, oh + jh - d.ch, ow + jw - d.cw) *
                                               ld(O, tIn, m * d.o_sm + r * d.f_sr + jh * d.f_sh + jw * d.f_sw, ok);
                            st(Y, tC, oy + m * d.y_sm + oh * d.W + ow, (float)acc, ok);
                        }
            }
        REQ(ok, "out-of-bounds access (cred)");
        return true;
    }
    for (int64_t b = 0; b < d.blocks; b++) {
        const int64_t rgi = b % d.nrb, gci = b / d.nrb;
        const int64_t g0 = gci * d.gchunk, g1 = std::min(d.G, g0 + d.gchunk);
        for (int64_t rl = 0; rl < d.per; rl++) {
            const int64_t r = rgi * d.per + rl;
            if (r >= d.R) continue;
            std::vector<double> acc((size_t)d.M * KK, 0.0);
            for (int64_t g = g0; g < g1; g++) {
                int64_t oz, oy;
                offs(g, oz, oy);
                for (int m = 0; m < d.M; m++)
                    for (int64_t oh = 0; oh < d.H; oh++)
                        for (int64_t ow = 0; ow < d.W; ow++) {
                            const double dy = ld(O, tIn, oy + m * d.o_sm + oh * d.W + ow, ok);
                            for (int jh = 0; jh < d.KH; jh++)
                                for (int jw = 0; jw < d.KW; jw++)
                                    acc[m * KK + jh * d.KW + jw] += zat(oz, r, oh + jh - d.ch, ow + jw - d.cw) * dy;
                        }
            }
            for (int q = 0; q < d.M * KK; q++) st(Y, 0, (gci * d.R + r) * d.M * KK + q, (float)acc[q], ok);
        }
    }
    REQ(ok, "out-of-bounds access (credw)");
    return true;
}

// K_WGCONV (the K_CREDW partials on fp32 MFMA tiles): the launcher's
// descriptor checks; every Z / O / partial index and every LDS word the
// kernel's lanes touch, walked block by block with its own offset
// arithmetic; then the partial sums it defines, in double.
bool run_wgconv(const Launch& ln, Ctx& c) {
    CredDesc d = desc_of<CredDesc>(ln);
    bool o1_ = true;
    const int tIn = (ln.kind >> kBitIn) & 1;
    const int KK = d.KH * d.KW, N = d.M * KK;
    const bool nct_ok = tIn ? (d.nct == 6 || (d.nct == 3 && N <= 48)) : (d.nct >= 1 && d.nct <= 6);
    REQ(d.M >= 1 && KK >= 1 && nct_ok && (d.rt == 1 || d.rt == 2) && (tIn || d.rt == 2) &&
            d.ncb == (N + 16 * d.nct - 1) / (16 * d.nct) && d.mb >= 1 && d.mb <= d.M && d.H >= 1 && d.W >= 1 &&
            d.PH == d.H + d.KH - 1 && d.PWp >= d.W + d.KW - 1 && d.ch >= 0 && d.ch < d.KH && d.cw >= 0 &&
            d.cw < d.KW && d.nrb == (d.R + 64 * d.rt - 1) / (64 * d.rt) && d.gchunk >= 1 &&
            d.nchunks == (d.G + d.gchunk - 1) / d.gchunk && d.blocks == (int64_t)d.nrb * d.ncb * d.nchunks &&
            d.lds_bytes == (uint32_t)(2 * d.mb * d.PH * d.PWp * 4) && d.lds_bytes <= 160 * 1024 &&
            (int64_t)d.H * d.W * d.M < (1ll << 30) && (int64_t)ln.grid[0] == d.blocks && ln.block[0] == 256 &&
            ln.lds == d.lds_bytes && d.ng >= 0 && d.ng <= 2 && d.zext >= 1 &&
            d.zext * (tIn ? 2 : 4) < (1ll << 31) && (size_t)d.zext * (tIn ? 2 : 4) <= resolve(ln.a, c, 0, o1_).bytes,
        "wgconv layout");
    bool ok = true, o1, o2, o3;
    Buf Z = resolve(ln.a, c, 0, o1), O = resolve(ln.b, c, 0, o2), Pb = resolve(ln.d, c, 0, o3);
    REQ(o1 && o2 && o3, "unresolved buffer");
    const int64_t HW = (int64_t)d.H * d.W, WP = d.PWp, PLN = (int64_t)d.PH * d.PWp, BUF = d.mb * PLN;
    const size_t es = tIn ? 2 : 4;
    const int64_t zn = (int64_t)(Z.bytes / es), on = (int64_t)(O.bytes / es), pn = (int64_t)(Pb.bytes / 4);
    const int top = d.KH - 1 - d.ch, left = d.KW - 1 - d.cw;
    auto offs = [&](int64_t g, int64_t& oz, int64_t& oy) {
        oz = oy = 0;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t x = g % d.g_size[i];
            g /= d.g_size[i];
            oz += x * d.g_sZ[i];
            oy += x * d.g_sY[i];
        }
    };
    const int rows = 64 * d.rt;
    for (int64_t b = 0; b < d.blocks; b++) {
        const int64_t ub = b % d.nrb, rest = b / d.nrb, ck = rest / d.ncb;
        const int cb = (int)(rest % d.ncb);
        const int n0 = cb * 16 * d.nct, mlo = n0 / KK, mhi = std::min(d.M, (n0 + 16 * d.nct - 1) / KK + 1);
        REQ(mhi - mlo <= d.mb, "wgconv planes of a column block");
        // the block's LDS reads (its columns' shifted planes) and writes (the interior)
        int64_t toff_max = 0;
        for (int n = n0; n < std::min(N, n0 + 16 * d.nct); n++) {
            const int m = n / KK, t = n % KK, jh = t / d.KW, jw = t % d.KW;
            toff_max = std::max<int64_t>(toff_max, (m - mlo) * PLN + (d.KH - 1 - jh) * WP + (d.KW - 1 - jw));
        }
        REQ((d.H - 1) * WP + (d.W - 1) + toff_max < BUF, "wgconv lds read range");
        REQ((int64_t)(mhi - mlo - 1) * PLN + (d.H - 1 + top) * WP + (d.W - 1 + left) < BUF, "wgconv lds write range");
        const int64_t g0 = ck * d.gchunk, g1 = std::min(d.G, g0 + d.gchunk);
        for (int64_t g = g0; g < g1; g++) {
            int64_t oz, oy;
            offs(g, oz, oy);
            for (int m = mlo; m < mhi; m++)
                REQ(oy + m * d.o_sm >= 0 && oy + m * d.o_sm + HW <= on, "wgconv O range");
            for (int64_t r = 0; r < rows; r++) {
                const int64_t u = ub * rows + r;
                if (u >= d.R) continue;
                REQ(oz + u * d.z_sr >= 0 && oz + u * d.z_sr + HW <= zn && oz + u * d.z_sr + HW <= d.zext,
                    "wgconv Z range");
            }
        }
        for (int64_t r = 0; r < rows; r++) {
            const int64_t u = ub * rows + r;
            if (u >= d.R) continue;
            const int nend = std::min(N, n0 + 16 * d.nct);
            REQ((ck * d.R + u) * N + nend <= pn, "wgconv partial range");
            std::vector<double> acc((size_t)N, 0.0);
            for (int64_t g = g0; g < g1; g++) {
                int64_t oz, oy;
                offs(g, oz, oy);
                for (int64_t h = 0; h < d.H; h++)
                    for (int64_t w = 0; w < d.W; w++) {
                        const double z = ld(Z, tIn, oz + u * d.z_sr + h * d.W + w, ok);
                        for (int n = n0; n < nend; n++) {
                            const int m = n / KK, t = n % KK, jh = t / d.KW, jw = t % d.KW;
                            const int64_t hh = h - jh + d.ch, ww = w - jw + d.cw;
                            if (hh < 0 || hh >= d.H || ww < 0 || ww >= d.W) continue;
                            acc[(size_t)n] += z * ld(O, tIn, oy + m * d.o_sm + hh * d.W + ww, ok);
                        }
                    }
            }
            for (int n = n0; n < nend; n++) st(Pb, 0, (ck * d.R + u) * N + n, (float)acc[(size_t)n], ok);
        }
    }
    REQ(ok, "out-of-bounds access (wgconv)");
    return true;
}

// K_GPAIR (both gradients of a channel-mixing step): the launcher's
// descriptor checks, the range of every index the kernel's loads and stores
// reach (block by block, with its own offset arithmetic), then dA and the
// per-block partials of dF in double.
bool run_gpair(const Launch& ln, Ctx& c) {
    GpairDesc d = desc_of<GpairDesc>(ln);
    const int nkc = d.nkc;
    const uint32_t lds = (uint32_t)(4 * (32 * (64 * nkc + 4) + 2 * 64 * 96 + 2 * 32 * 68));
    REQ(((ln.kind >> kBitIn) & 1) == 0 && d.M >= 1 && d.M <= 32 && d.K >= 1 && d.K2 >= 1 && d.K1 * d.K2 == d.K &&
            (nkc == 1 || nkc == 2 || nkc == 4 || nkc == 8) && d.K <= 64 * nkc && d.N >= 1 &&
            d.ntiles == (d.N + 63) / 64 && d.gper >= 1 && d.blocks == (d.G + d.gper - 1) / d.gper &&
            d.lds_bytes == lds && lds <= 160 * 1024 && (int64_t)ln.grid[0] == d.blocks && ln.block[0] == 1024 &&
            ln.lds == d.lds_bytes && d.ng >= 0 && d.ng <= 2 && ln.extra.size() == 1 && d.sG1 >= 0 && d.sG2 >= 0 &&
            d.sAm >= 0 && d.gext == (int64_t)(d.K1 - 1) * d.sG1 + (int64_t)(d.K2 - 1) * d.sG2 + d.N &&
            d.gext * 4 < (1ll << 31) && d.aext == (int64_t)(d.M - 1) * d.sAm + d.N && d.aext * 4 < (1ll << 31),
        "gpair layout");
    bool ok = true, o1, o2, o3, o4, o5;
    Buf A = resolve(ln.a, c, 0, o1), F = resolve(ln.b, c, 0, o2), G = resolve(ln.c, c, 0, o3),
        Pb = resolve(ln.d, c, 0, o4), dA = resolve(ln.extra[0], c, 0, o5);
    REQ(o1 && o2 && o3 && o4 && o5, "unresolved buffer");
    const int64_t an = (int64_t)(A.bytes / 4), fn = (int64_t)(F.bytes / 4), gn = (int64_t)(G.bytes / 4),
                  pn = (int64_t)(Pb.bytes / 4);
    auto offs = [&](int64_t g, int64_t& oa, int64_t& og, int64_t& od) {
        oa = og = od = 0;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t x = g % d.g_size[i];
            g /= d.g_size[i];
            oa += x * d.g_sA[i];
            og += x * d.g_sG[i];
            od += x * d.g_sD[i];
        }
    };
    auto fidx = [&](int k, int m) { return (int64_t)(k / d.K2) * d.sF1 + (int64_t)(k % d.K2) * d.sF2 + (int64_t)m * d.sFm; };
    // F reads and partial writes: every (k, m) in range, the partial layout dense
    for (int k = 0; k < d.K; k++)
        for (int m = 0; m < d.M; m++) {
            const int64_t i = fidx(k, m);
            REQ(i >= 0 && i < fn && i < d.fnumel, "gpair F / partial index");
        }
    REQ(d.blocks * d.fnumel <= pn, "gpair partial range");
    std::vector<double> acc((size_t)d.fnumel);
    for (int64_t blk = 0; blk < d.blocks; blk++) {
        std::fill(acc.begin(), acc.end(), 0.0);
        const int64_t g0 = blk * d.gper, g1 = std::min(d.G, g0 + d.gper);
        for (int64_t g = g0; g < g1; g++) {
            int64_t oa, og, od;
            offs(g, oa, og, od);
            // the rows the kernel loads: G rows k (all n), A rows m (all n)
            for (int k = 0; k < d.K; k++) {
                const int64_t r = og + (int64_t)(k / d.K2) * d.sG1 + (int64_t)(k % d.K2) * d.sG2;
                REQ(r >= 0 && r + d.N <= gn && r - og + d.N <= d.gext, "gpair G range");
            }
            // the buffer ranges (one g's slice from its base) lie inside the tensors
            REQ(og >= 0 && og + d.gext <= gn && oa >= 0 && oa + d.aext <= an, "gpair G / A slice");
            for (int m = 0; m < d.M; m++)
                REQ(oa + m * d.sAm >= 0 && oa + m * d.sAm + d.N <= an && m * d.sAm + d.N <= d.aext, "gpair A range");
            for (int m = 0; m < d.M; m++)
                for (int64_t n = 0; n < d.N; n++) {
                    double sa = 0;
                    for (int k = 0; k < d.K; k++) {
                        const double gv = ld(G, 0, og + (int64_t)(k / d.K2) * d.sG1 + (int64_t)(k % d.K2) * d.sG2 + n, ok);
                        sa += ld(F, 0, fidx(k, m), ok) * gv;
                        acc[(size_t)fidx(k, m)] += ld(A, 0, oa + m * d.sAm + n, ok) * gv;
                    }
                    if (dA.base) st(dA, 0, od + m * d.sDm + n, (float)sa, ok);
                }
        }
        for (int k = 0; k < d.K; k++)
            for (int m = 0; m < d.M; m++) st(Pb, 0, blk * d.fnumel + fidx(k, m), (float)acc[(size_t)fidx(k, m)], ok);
    }
    REQ(ok, "out-of-bounds access (gpair)");
    return true;
}

// Small-output contraction over a long reduction: per-block partials over
// the block's outer rows (K_THINW), then the ordered chunk sum (K_THINW_REDUCE).
bool run_thinw(const Launch& ln, Ctx& c) {
    ThinwDesc d = desc_of<ThinwDesc>(ln);
    const bool red = (ln.kind & 0xff) == K_THINW_REDUCE;
    int tIn = (ln.kind >> kBitIn) & 1, tC = (ln.kind >> kBitOut) & 1;
    const int MM = d.M <= 4 ? 4 : d.M <= 8 ? 8 : 16, NN = d.N <= 4 ? 4 : d.N <= 8 ? 8 : 16;
    REQ(d.M >= 1 && d.N >= 1 && d.M <= 16 && d.N <= 16 && MM * NN <= 64 && d.ng <= 3 && d.no <= 3, "thinw dims");
    int64_t G = 1, Ko = 1;
    for (int i = 0; i < d.ng; i++) G *= d.g_size[i];
    for (int i = 0; i < d.no; i++) Ko *= d.o_size[i];
    REQ(G == d.G && Ko == d.Kout && d.Kin >= 1 && d.orows >= 1 && d.orows <= 512 &&
        d.orows * d.Kin < ((int64_t)1 << 31) && d.kchunks == (d.Kout + d.orows - 1) / d.orows &&
        d.blocks == d.G * d.kchunks, "thinw split");
    bool ok = true, o1, o2;
    Buf Pt = resolve(ln.d, c, 0, o1);
    REQ(o1, "unresolved buffer");
    if (red) {
        Buf Cb = resolve(ln.c, c, 0, o2);
        REQ(o2, "unresolved buffer");
        REQ((int64_t)ln.grid[0] * 256 >= d.G * d.M * d.N && ln.block[0] == 256, "grid");
        for (int64_t g = 0; g < d.G; g++)
            for (int m = 0; m < d.M; m++)
                for (int n = 0; n < d.N; n++) {
                    double acc = 0;
                    for (int64_t kc = 0; kc < d.kchunks; kc++)
                        acc += ld(Pt, 0, (g * d.kchunks + kc) * (MM * NN) + m * NN + n, ok);
                    int64_t off = m * d.sCm + n * d.sCn, x = g;
                    for (int i = d.ng - 1; i >= 0; --i) { off += (x % d.g_size[i]) * d.g_sC[i]; x /= d.g_size[i]; }
                    st(Cb, tC, off, (float)acc, ok);
                }
        REQ(ok, "out-of-bounds access (thinw reduce)");
        return true;
    }
    Buf P = resolve(ln.a, c, 0, o1), Q = resolve(ln.b, c, 0, o2);
    REQ(o1 && o2, "unresolved buffer");
    REQ((int64_t)ln.grid[0] == d.blocks && ln.block[0] == 256, "grid");
    for (int64_t b = 0; b < d.blocks; b++) {
        const int64_t g = b / d.kchunks, kc = b % d.kchunks;
        int64_t gP = 0, gQ = 0, x = g;
        for (int i = d.ng - 1; i >= 0; --i) {
            const int64_t y = x % d.g_size[i];
            x /= d.g_size[i];
            gP += y * d.g_sP[i];
            gQ += y * d.g_sQ[i];
        }
        std::vector<double> acc(MM * NN, 0.0);
        for (int64_t o = kc * d.orows; o < std::min(d.Kout, (kc + 1) * d.orows); o++) {
            int64_t sp = 0, sq = 0, y = o;
            for (int i = d.no - 1; i >= 0; --i) {
                const int64_t z = y % d.o_size[i];
                y /= d.o_size[i];
                sp += z * d.o_sP[i];
                sq += z * d.o_sQ[i];
            }
            for (int64_t i = 0; i < d.Kin; i++)
                for (int m = 0; m < d.M; m++) {
                    const double a = ld(P, tIn, gP + sp + i + m * d.sPm, ok);
                    for (int n = 0; n < d.N; n++) acc[m * NN + n] += a * ld(Q, tIn, gQ + sq + i + n * d.sQn, ok);
                }
        }
        for (int q = 0; q < MM * NN; q++) st(Pt, 0, b * MM * NN + q, (float)acc[q], ok);
        REQ(ok, "out-of-bounds access (thinw)");
    }
    return true;
}
}  // namespace

extern "C" {

// Cap on every intermediate's elements for the plans emul_run builds
// (0: none; the memory-limited order of ce_plan_create_limited).
static uint64_t g_limit = 0;
static uint64_t g_save_budget = 0;
void emul_set_limit(uint64_t max_elements) { g_limit = max_elements; }
void emul_set_save_budget(uint64_t bytes) { g_save_budget = bytes; }
// Strides of convolved labels for the next plans: "h=2,w=2" ("" for none).
static std::string g_strides;
void emul_set_strides(const char* spec) { g_strides = spec ? spec : ""; }
// Two-way convolved labels made circular for the next plans: "h,w" ("" none).
static std::string g_circular;
void emul_set_circular(const char* spec) { g_circular = spec ? spec : ""; }
// 1: the next plans take the left-to-right order ((0,1),(0,n-2),...,(0,1))
static int g_ltr = 0;
void emul_set_path(int ltr) { g_ltr = ltr; }

// Runs the forward (mode 0), backward (mode 1) or forward then backward on
// one workspace (mode 2) launch lists of a plan built with `flags`
// (CE_FLAG_*).  Buffers are host memory in the plan's storage types.
// Returns 0 on success, else writes a message to err.
int emul_run(const char* spec, int n, const int* ranks, const int64_t* const* dims, int bf16,
             int mode, void* const* ins, void* out, const void* dout, void* const* din,
             char* err, int errlen, int flags) {
    const int generic_only = flags & CE_FLAG_GENERIC_ONLY;
    try {
        std::unique_ptr<ce_expr> e(parse_expr(spec, n, ranks, dims));
        for (size_t pos = 0; pos < g_strides.size();) {
            size_t eq = g_strides.find('=', pos), end = g_strides.find(',', pos);
            if (end == std::string::npos) end = g_strides.size();
            const std::string lab = g_strides.substr(pos, eq - pos);
            const int st = std::atoi(g_strides.substr(eq + 1, end - eq - 1).c_str());
            if (ce_expr_set_stride(e.get(), lab.c_str(), st) != CE_OK) {
                std::snprintf(err, errlen, "bad stride %s", lab.c_str());
                return 3;
            }
            pos = end + 1;
        }
        PlanLimits lim;
        if (g_limit) lim.max_elements = g_limit;
        lim.save_budget = g_save_budget;
        for (size_t pos = 0; pos < g_circular.size();) {
            size_t end = g_circular.find(',', pos);
            if (end == std::string::npos) end = g_circular.size();
            const std::string lab = g_circular.substr(pos, end - pos);
            if (ce_expr_set_conv(e.get(), lab.c_str(), CE_PAD_CIRCULAR) != CE_OK) {
                std::snprintf(err, errlen, "bad circular label %s", lab.c_str());
                return 3;
            }
            pos = end + 1;
        }
        std::vector<int> pairs;
        if (g_ltr && n > 1) {
            pairs = {0, 1};
            for (int k = 1; k < n - 1; k++) {
                pairs.push_back(0);
                pairs.push_back(n - 1 - k);
            }
        }
        std::unique_ptr<ce_plan> p(make_plan(*e, CE_COST_FWD, bf16 ? CE_BF16 : CE_F32, (unsigned)flags,
                                             !pairs.empty(), pairs.data(), (int)pairs.size() / 2, lim));
        if (!p->executable) { std::snprintf(err, errlen, "not executable"); return 2; }
        Ctx c;
        int es = bf16 ? 2 : 4;
        for (int i = 0; i < n; i++) {
            int64_t numel = 1;
            for (int k = 0; k < ranks[i]; k++) numel *= dims[i][k];
            c.in.push_back({(unsigned char*)ins[i], (size_t)numel * es});
            size_t ges = (i == e->feature_operand) ? es : 4;
            c.din.push_back({din ? (unsigned char*)din[i] : nullptr, (size_t)numel * ges});
        }
        int64_t onum = 1;
        for (auto d : e->out_dims()) onum *= d;
        c.out = {(unsigned char*)out, (size_t)onum * es};
        c.dout = {(unsigned char*)const_cast<void*>(dout), (size_t)onum * es};
        size_t wsb = mode == 2 ? std::max(p->ws_fwd, p->ws_bwd) : mode ? p->ws_bwd : p->ws_fwd;
        std::vector<unsigned char> ws(wsb + 1, 0xCD);   // poisoned: unset reads show up
        c.ws = {ws.data(), wsb};
        std::vector<const Launch*> list;
        if (mode != 1)
            for (const Launch& ln : p->fwd) list.push_back(&ln);
        if (mode != 0)
            for (const Launch& ln : p->bwd) list.push_back(&ln);
        for (const Launch* lp : list) {
            const Launch& ln = *lp;
            int v = ln.kind & 0xff;
            bool generic = v == K_GENERIC_THREAD || v == K_GENERIC_WAVE || v == K_GENERIC_BLOCK;
            if (generic_only && !generic) {
                std::snprintf(err, errlen, "non-generic launch in a generic-only plan");
                return 3;
            }
            bool ok = generic ? run_generic(ln, c)
                    : (v == K_GEMM || v == K_THIN) ? run_gemm(ln, c)
                    : v == K_WGRAD ? run_wgrad(ln, c)
                    : v == K_REDUCE ? run_reduce(ln, c)
                    : v == K_REDUCE_MULTI ? run_reduce_multi(ln, c)
                    : v == K_DW ? run_dw(ln, c)
                    : v == K_DW_TAPGRAD ? run_tapgrad(ln, c)
                    : v == K_DW_TAPREDUCE ? run_tapreduce(ln, c)
                    : v == K_CP_FWD ? run_cp_fwd(ln, c)
                    : v == K_CP_BWD ? run_cp_bwd(ln, c)
                    : v == K_RCP_FWD ? run_rcp_fwd(ln, c)
                    : v == K_RCP_BWD ? run_rcp_bwd(ln, c)
                    : v == K_RCP_PREP ? run_rcp_prep(ln, c)
                    : v == K_TC ? run_tc(ln, c)
                    : v == K_TC_REDUCE ? run_tc_reduce(ln, c)
                    : (v == K_CRED || v == K_CREDW || v == K_CREDW_REDUCE) ? run_cred(ln, c)
                    : v == K_CCONV ? run_cconv(ln, c)
                    : v == K_WGCONV ? run_wgconv(ln, c)
                    : v == K_GPAIR ? run_gpair(ln, c)
                    : v == K_TT_FWD || v == K_TT_PREP ? run_tt_fwd(ln, c)
                    : (v == K_THINW || v == K_THINW_REDUCE) ? run_thinw(ln, c)
                    : (c.err = "unknown launch kind", false);
            if (!ok) { std::snprintf(err, errlen, "%s", c.err.c_str()); return 4; }
        }
        return 0;
    } catch (const Error& ex) {
        std::snprintf(err, errlen, "%s", ex.what());
        return 1;
    }
}

}
