// Plain-old-data kernel descriptors, filled by the host planner and passed
// by value to the HIP kernels.  No HIP types here: this header is included
// by host-only sources as well.
#pragma once

#include <cstdint>

namespace ce {

enum DType : int32_t { DT_F32 = 0, DT_BF16 = 1 };

constexpr int kMaxDims = 8;   // loop dimensions of a generic pairwise step
constexpr int kMaxConv = 4;   // convolved labels of one step

// A pairwise step in its most general form:
//
//   C[o] = sum_r  L[offL(o, r)] * R[offR(o, r)]
//
// o runs over the output dims (the layout of C), r over the reduction dims.
// A plain dim contributes index * stride to each operand.  A convolved label
// owns one output dim (index p) and one reduction dim (index j) whose plain
// strides are zero; it contributes pos * stride to an operand, where
// pos = a * p + b * j + g must lie in [0, lim) or the term is skipped.  This
// covers the forward step (feature read at p + j - c, filter at j), the
// gradient of the feature side (dC read at p - j + c) and the gradient of the
// filter side (feature read at j + p - c, dC at j).  For a circular label the
// position is first taken modulo N (cv_modL / cv_modR): indices add modulo N.
struct GenericDesc {
    int32_t nout, nred, nconv;
    int32_t has_r;                     // 0: R is absent (treated as 1)
    int64_t total_out, total_red;
    int64_t out_size[kMaxDims], out_sL[kMaxDims], out_sR[kMaxDims], out_sC[kMaxDims];
    int64_t red_size[kMaxDims], red_sL[kMaxDims], red_sR[kMaxDims];
    int32_t cv_out[kMaxConv], cv_red[kMaxConv];    // dim indices
    int32_t cv_aL[kMaxConv], cv_bL[kMaxConv], cv_aR[kMaxConv], cv_bR[kMaxConv];
    int64_t cv_gL[kMaxConv], cv_limL[kMaxConv], cv_sL[kMaxConv];
    int64_t cv_gR[kMaxConv], cv_limR[kMaxConv], cv_sR[kMaxConv];
    // circular labels: a position is first reduced modulo cv_mod? (0: not)
    int64_t cv_modL[kMaxConv], cv_modR[kMaxConv];
};

enum KernelKind : int32_t {
    K_GENERIC_THREAD = 1,   // one thread per output element
    K_GENERIC_WAVE = 2,     // one 64-lane wavefront per output element
    K_GENERIC_BLOCK = 3,    // one 256-thread block per output element
    K_GEMM = 16,            // channel-mixing GEMM (GemmDesc)
    K_WGRAD = 17,           // split-reduction NT GEMM into partials (WgradDesc)
    K_REDUCE = 18,          // ordered sum of partials (ReduceDesc)
    K_DW = 19,              // depthwise convolution along one axis (DwDesc)
    K_DW_TAPGRAD = 20,      // per-block partial filter-tap gradients (DwDesc)
    K_DW_TAPREDUCE = 21,    // ordered sum of tap partials (DwDesc)
    K_CP_FWD = 22,          // fused CP chain forward (CpDesc)
    K_CP_BWD = 23,          // fused CP chain backward (CpBwdDesc)
    K_TC = 24,              // tiled MFMA contraction with convolved labels (TcDesc)
    K_TC_REDUCE = 25,       // ordered sum of its split-reduction partials (TcDesc)
    K_THIN = 26,            // channel mix with few rows and few reduced channels (GemmDesc)
    K_CRED = 27,            // 2-D convolution summed over channels into one plane (CredDesc)
    K_CREDW = 28,           // filter-tap partials of the same convolution (CredDesc)
    K_THINW = 29,           // small-output contraction over a long reduction (ThinwDesc)
    K_THINW_REDUCE = 30,    // ordered sum of its partials (ThinwDesc)
    K_CREDW_REDUCE = 31,    // ordered sum of the K_CREDW partials (CredDesc)
    K_REDUCE_MULTI = 32,    // up to four ordered partial sums in one launch (MultiReduceDesc)
    K_RCP_FWD = 33,         // fused reshaped-CP chain forward (RcpDesc, desc_rcp.h)
    K_RCP_BWD = 34,         // fused reshaped-CP chain backward (RcpBwdDesc, desc_rcp.h)
    K_RCP_PREP = 35,        // its prepared factor table (RcpBwdDesc)
    K_CCONV = 36,           // convolution contracted over one channel index, MFMA tiles (CconvDesc)
    K_TT_FWD = 37,          // fused contraction + convolution of a tensor-train chain (TtDesc)
    K_TT_PREP = 38,         // its convolution's A operands in load order (TtDesc)
    K_WGCONV = 39,          // K_CREDW's partials on fp32 MFMA tiles (CredDesc)
    K_GPAIR = 40,           // both gradients of a channel-mixing step from one read of dC (GpairDesc)
};

// Launch kind = variant | element-type bits (1 = bfloat16, 0 = float32).
constexpr int32_t kBitIn = 8;     // main inputs
constexpr int32_t kBitAux = 9;    // second input (filter / factor) when it may differ
constexpr int32_t kBitOut = 10;   // output
constexpr int32_t kShiftOpt = 12; // kernel-specific option bits

// C[g][m][n] = sum_k A[g][m][k] * B[g][k][n] with n unit-stride in B and C.
// A is the small operand (a factor), B and C the large ones (activations).
// Blocks: ntiles x mtiles x prod(g_size), flattened.
struct GemmDesc {
    int32_t M, N, K;
    int32_t ng;
    int64_t g_size[3], g_sA[3], g_sB[3], g_sC[3];
    int64_t sAm, sAk, sBk, sCm;
    int32_t mtiles, ntiles;
    int64_t blocks;
};

// partial[s][m][n] = sum over reduction chunk s of A[kb][m][k] * B[kb][n][k]
// with k unit-stride in A and B; s = (kb index) * ksplit + (k chunk).
struct WgradDesc {
    int32_t M, N;
    int64_t K;                 // unit-stride reduction length
    int32_t nkb;
    int64_t kb_size[3], kb_sA[3], kb_sB[3];
    int64_t sAm, sBn;
    int32_t ksplit, kchunk;    // chunks of k per kb index and their length
    int64_t nsplit;            // number of partials
    int32_t mtiles, ntiles;
    int64_t blocks;
};

// C[m * sCm + n * sCn] = sum_{s < nsplit} partial[s][m][n]
struct ReduceDesc {
    int32_t M, N;
    int64_t nsplit;
    int64_t sCm, sCn;
};

// Both gradients of a channel-mixing step C[g][k][n] = sum_m A[g][m][n] F[k][m]
// (fp32) from one read of the output gradient G = dC:
//   dA[g][m][n] = sum_k F[k][m] G[g][k][n]
//   P[blk][F's layout] = sum over the block's g and every n of A[g][m][n] G[g][k][n]
// n: unit-stride in A, G and dA; k = (k1, k2) with k2 fastest (K = K1 K2);
// g: up to two dims.  A block takes gper consecutive g, all n in tiles of 64
// and the reduction over k in nkc chunks of 64; M <= 32, K <= 64 nkc <= 512.
struct GpairDesc {
    int32_t M, K, K1, K2, N, ng;
    int32_t nkc, ntiles;
    int64_t G, gper, blocks;
    int64_t g_size[2], g_sA[2], g_sG[2], g_sD[2];
    int64_t sAm, sDm, sFm, sG1, sG2, sF1, sF2;
    int64_t fnumel;            // elements of F (dense): one partial's size
    int64_t gext, aext;        // elements one g's rows of G and of A span (buffer-load ranges, < 2^29)
    uint32_t lds_bytes, pad_;
};

// Waves a block of the ordered partial sums (64 outputs a block), from the
// number of partials alone, so that the summation order is fixed per shape.
inline int reduce_waves(int64_t nsplit) { return nsplit <= 8 ? 1 : nsplit <= 64 ? 4 : 16; }

// Up to four independent ordered sums (ReduceDesc each, fp32 outputs) in one
// launch: part j owns blocks [block0[j], block0[j+1]); a part whose output
// pointer is null (gradient not requested) is skipped.
struct MultiReduceDesc {
    int32_t n, pad_;
    ReduceDesc part[4];
    int64_t block0[5];
};

// Depthwise convolution along one axis of a dense tensor viewed as
// [nslab][A][inner]: out[o][p][q] = sum_j in[o][p + sign*j + off][q] * f[frow(o) + j*f_sj]
// with in zero outside [0, A) and frow(o) = ((o / r_div) % r_size) * r_stride.
// A block covers spb consecutive slabs.  For the tap gradient the same view
// gives part[block][j] = sum in[o][p + j + off][q] * g[o][p][q], reduced over the
// blocks sharing a filter row into out[r * o_sr + j * o_sj].
struct DwDesc {
    int64_t nslab;
    int32_t A, inner, K, sign, off, spb;
    int64_t r_div, r_size, r_stride, f_sj;
    int64_t nblocks;
    int64_t o_sr, o_sj;        // tap reduce: output strides
};

// Fused CP chain (the four forward steps of a CP-factorised 2-D conv layer):
//   Z1[r][p] = sum_s Us[r][s] X[b][s][p]          (channel contraction)
//   Z2 = Z1 (*)_h Kh[r],  Z3 = Z2 (*)_w Kw[r]     (depthwise, same padding)
//   Y[b][t][p] = sum_r Ut[r][t] Z3[r][p]          (channel expansion)
// p = h*W + w is unit-stride in X and Y.  One wavefront owns a strip of 32
// columns (overlapping its neighbours by the conv_w halo) over seg_rows rows
// of one sample.
struct CpDesc {
    int32_t B, S, R, T, H, W, KH, KW;
    int32_t ncb, colstride, segs, seg_rows;
    int64_t x_sb, x_ss, y_sb, y_st;
    int64_t us_sr, us_ss, ut_sr, ut_st;
    int64_t kh_sr, kh_sj, kw_sr, kw_sj;
    int64_t waves, blocks;
    // LDS operand tables, laid out by the planner: UsL [32][lda] at 0, the
    // permuted Ut operands at o_ut, the permuted taps at o_kh / o_kw, the
    // vertical taps reversed (for segments walked upwards) at o_khr
    uint32_t lds_bytes, o_ut, o_kh, o_kw;
    int32_t lda;
    uint32_t o_khr;
};

// General contraction on MFMA tiles:
//
//   C[g][m][n] = sum_k A[g][m][k] * B[g][k][n]
//
// g, m, n and k are each a list of up to four dims (outermost first) with a
// stride per operand (zero where the operand lacks the dim).  A convolved
// label (up to two) contributes one n dim (its output index p, n_cv = label
// slot) and one k dim (its reduction index j, k_cv = slot): B is read at
// position cv_a*p + cv_b*j + cv_g with stride cv_s, zero outside [0, cv_lim);
// A reads j as a plain k index.  This covers the forward convolution, the
// gradient of its feature side (transposed convolution) and of its filter
// side (p = filter tap, j = image position).  With ksplit > 1 the k range is
// cut in chunks of kchunk; block (g, chunk) writes P[g][chunk][m][n] (fp32)
// and the reduce launch sums the chunks in order into C.
struct TcDesc {
    int32_t ng, nm, nn, nk, ncv, ksplit;
    int64_t M, N, K, G;
    int64_t g_size[4], g_sA[4], g_sB[4], g_sC[4];
    int64_t m_size[4], m_sA[4], m_sC[4];
    int64_t n_size[4], n_sB[4], n_sC[4];
    int64_t k_size[4], k_sA[4], k_sB[4];
    int32_t n_cv[4], k_cv[4];
    int32_t cv_a[2], cv_b[2];
    int64_t cv_g[2], cv_lim[2], cv_s[2];
    int32_t mtiles, ntiles;
    int64_t kchunk, blocks;
    // off32: every offset of A, B and C fits 31 bits and A, B fit 2 GiB
    // (extA / extB bytes): 32-bit index arithmetic and range-checked buffer
    // loads; else 64-bit offsets and predicated loads
    int32_t off32, pad_;
    int64_t extA, extB;
    // tapmask: the convolved reduction indices take at most 32 combinations
    // (tap = j0 * tapJ1 + j1): a thread's valid taps form a bitmask, and the
    // taps' offsets go into the k table
    int32_t tapmask, tapJ1;
    // kmajor: k (not n) is unit-stride in B and in A: lanes walk k when
    // loading the tiles, the rows' / columns' offsets come from LDS tables
    int32_t kmajor, pad2_;
};

// Convolution of a stack of planes contracted over one shared index:
//   C[u][m][p] = sum_s sum_j Z[u][s][p + j - c] * O[m][s][j]
// over 2-D positions p (output) and j (reduction), Z zero outside its plane,
// m < M <= 16 a channel of O only.  Two instances, both with the plane held
// in LDS with its zero halo:
//   K_CRED  (forward): p runs over an H x W output plane, j over KH x KW
//           filter taps; u = batch (up to two dims), s = rank (one dim);
//           O = the filter F[m][s][jh][jw].
//   K_CREDW (filter gradient): p runs over KH x KW taps, j over the H x W
//           plane; u = rank (one dim), s = batch (up to two dims); O = the
//           output gradient; writes partials P[chunk][u][m][tap], summed in
//           chunk order by K_CREDW_REDUCE.
//   K_WGCONV (filter gradient on fp32 MFMA tiles, fp32 or bf16 planes): the
//           same partials as K_CREDW with u in blocks of 64 rt (nrb blocks)
//           and the columns (m, tap) in ncb blocks of 16 nct; a block's mb
//           planes of O sit in LDS with a zero halo (PH rows of pitch PWp,
//           fp32), double-buffered.
// Planes (Z, the output of K_CRED, O of K_CREDW) are dense: row stride W,
// unit columns.  ch, cw: zero padding before the first row / column.
struct CredDesc {
    int32_t H, W, KH, KW, ch, cw;
    int32_t PH, PWp, wchunks, items;   // LDS plane (rows, padded row pitch); 4-pixel items
    int32_t ng, per, M, pad_;          // batch dims; planes per block; channels m
    int64_t R, G;                      // rank count; batch count
    int64_t g_size[2], g_sZ[2], g_sY[2];
    int64_t z_sr, f_sr, f_sh, f_sw;    // K_CRED: F strides
    int64_t o_sm, y_sm;                // m strides: of O; of the output (K_CRED)
    int64_t c_sm, c_sr, c_sh, c_sw;    // K_CREDW_REDUCE: output strides
    int64_t gchunk, nrb, nchunks;      // K_CREDW: batch indices per block, rank groups, chunks
    int64_t blocks;
    uint32_t lds_bytes, threads;
    // K_WGCONV: column blocks of 16 * (column tiles) columns (m, tap), row
    // tiles of 16 a wavefront (rows a block: 64 * rt), channel planes a
    // block stages (mb)
    int32_t ncb, nct, rt, mb;
    int64_t zext;   // K_WGCONV: elements of Z from its base (its buffer loads are range-checked)
};

// Convolution contracted over one channel index, on bf16 MFMA tiles:
//   Y[g][q][h][w] = sum_p sum_{th, tw} Z[g][p][h + dh(th)][w + dw(tw)] * F[p][q][fh(th)][fw(tw)]
// with dh(t) = zh0 + zhs * t and fh(t) = fh0 + fhs * t (zhs, fhs = +-1; the
// same along w), Z read as zero outside its H x W plane.  This is the forward
// of a convolution step with a contraction (the Tucker core, Section 2.3) and,
// with reversed taps, its input gradient.  Z and Y planes are dense (row
// stride W); p, q and up to two batch dims have free strides.  A block takes
// one g, TH output rows and 32 values of q: the filter slice [32][taps][Ppad]
// and the zero-padded input rows [HP][WP][Ppad] (channels innermost) sit in
// LDS as bf16 pairs, rows padded to pw_tab / pw_img 32-bit words.
struct CconvDesc {
    int32_t H, W, KH, KW;
    int32_t zh0, zhs, zw0, zws;        // plane offset of tap t: z?0 + z?s * t
    int32_t fh0, fhs, fw0, fws;        // filter index of tap t: f?0 + f?s * t
    int32_t P, Q, Ppad, ng;            // contracted / output channels; P rounded up to 16; batch dims
    int32_t TH, ntiles, nq, HP;        // output rows a tile; tiles; q tiles of 32; LDS input rows
    int32_t WP, pw_img, pw_tab, tp;    // LDS input columns; word pitches of a pixel, of a q row, of a tap
    // rega (fp32, P <= 8, at most 9 taps): a block covers every q tile of its
    // rows, the filter operands stay in registers and LDS holds the input rows
    int32_t rega, pad_;
    int64_t G, g_size[2], g_sZ[2], g_sY[2];
    int64_t z_numel, f_numel;          // elements of Z and F (byte ranges of the raw buffer loads, < 2^30)
    int64_t z_sp, y_sq, f_sp, f_sq, f_sh, f_sw;
    int64_t y_ext;                     // rega: elements of Y one g spans (its stores are range-checked)
    int64_t blocks;
    uint32_t lds_bytes, pad2_;
};

// Contraction with a small output per batch index and a long reduction:
//   C[g][m][n] = sum_k P[g][m][k] * Q[g][n][k]
// (factor gradients of reshaped-CP layers), M, N <= 16.  k runs over an
// inner run of Kin elements contiguous in P and Q and up to three outer
// dims; g over up to three dims (a zero stride where an operand lacks one).
// A block takes one g and `orows` consecutive outer indices and writes one
// partial per (g, chunk, m, n); K_THINW_REDUCE sums the chunks in order.
struct ThinwDesc {
    int32_t ng, no, M, N;
    int64_t G, Kin, Kout;
    int64_t g_size[3], g_sP[3], g_sQ[3], g_sC[3];
    int64_t o_size[3], o_sP[3], o_sQ[3];
    int64_t sPm, sQn, sCm, sCn;
    int64_t orows, kchunks, blocks;
};

// Backward of the same chain.  Strips and segments as in CpDesc (dX has X's
// layout, dY has Y's).  Every block writes its partial factor gradients
// (summed over its four wavefronts in a fixed order) to row blockIdx of
// Pus[blocks][R][S], Put[blocks][R][T], Pkh[blocks][R][KH], Pkw[blocks][R][KW].
// LDS: UsA [32][lda_s] at 0, UtA [32][lda_t] at o_uta, for bf16 UsT [S][ldu]
// (Us transposed) at o_ust, four wave-private fp32 [32][33] tiles at o_tz and
// four wave-private [T][ly] tiles of yt_bytes each at o_yt; the end-of-block
// reduction reuses the first red_bytes.
struct CpBwdDesc {
    int32_t B, S, R, T, H, W, KH, KW;
    int32_t ncb, colstride, segs, seg_rows;
    int64_t x_sb, x_ss, y_sb, y_st;
    int64_t us_sr, us_ss, ut_sr, ut_st;
    int64_t kh_sr, kh_sj, kw_sr, kw_sj;
    int64_t waves, blocks;
    uint32_t lds_bytes, o_uta, o_ust, o_tz, o_yt, yt_bytes, red_bytes;
    int32_t lda_s, lda_t, ldu, ly;
    // per-wave ring of the last three X rows (channel-major, row pitch lx);
    // the dZ1 transpose tile of a wave sits at o_tz + wave * tz_stride (it may
    // share the wave's dY tile: o_tz == o_yt, tz_stride == yt_bytes)
    uint32_t o_xl, xl_bytes, tz_stride;
    int32_t lx;
};

// Two consecutive steps of a (reshaped) tensor-train layer fused so that the
// first step's result never leaves the chip:
//   Z[b][g][u][r][p] = sum_k X[b][k][u][p] * F1[g][k][r]                (step A)
//   Y[b][g][t][p]    = sum_{u, r, taps} Z[b][g][u][r][p + tap - c] * F2[t][u][r][tap]   (step B)
// p = (h, w) over an H x W plane (dense, w unit-stride, in X and Y), the
// taps KH x KW with zero 'same' padding.  Each index set (b, g, k, u, r, t)
// is one linear index per tensor (its labels' strides chain).  A block takes
// one (b, g) and TH output rows: per u it forms the R = 16 channels of Z on
// the TH + KH - 1 rows it needs (MFMA 16x16x4: M = r, N = 16 pixels,
// K = k) in LDS, then accumulates step B on MFMA 16x16x4 tiles whose M rows
// are (t, one of two output rows) and whose K runs over (r, KH + 1 tap rows,
// KW tap columns), so the T <= 8 output channels fill the tile.
struct TtDesc {
    int32_t B, G, K1, U, R, T, H, W;
    int32_t TH, nbands, XT, PW, plane, ncombo;
    int64_t x_sb, x_sk, x_su, y_sb, y_sg, y_st;
    int64_t f1_sg, f1_sk, f1_sr;
    int64_t f2_st, f2_su, f2_sr, f2_sh, f2_sw;
    int64_t x_numel, f1_numel, f2_numel;   // element extents of the operands (< 2^29)
    int64_t blocks;
    uint32_t lds_bytes, xcd_remap;          // xcd_remap: blocks % 8 == 0, runs of a sample on one XCD
};

}  // namespace ce
