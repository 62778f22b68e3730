// Descriptor of the fused reshaped-CP chain (host planner and HIP kernel).
//
// Reshaped CP layer (Section 2.3, reshaped tensor decompositions; the RCP
// string of Appendix A.3 with three modes):
//   Y[b][t1][t2][t3][h][w] = sum_r sum_{s1 s2 s3} W1[r][t1][s1] W2[r][t2][s2] W3[r][t3][s3]
//                            sum_{i j} W0[r][i][j] X[b][s1][s2][s3][h+i-c][w+j-c]
// planned as the chain  Z1 = X x1 W1 (contract s1), Z2 = Z1 x2 W2 (contract s2),
// Z3 = Z2 x3 W3 (contract s3), Y = sum_r Z3 (*) W0[r] (2-D convolution, same
// zero padding), all tensors dense in their string's label order.
#pragma once

#include <cstdint>

namespace ce {

// One workgroup owns sample b, output mode index t1, a chunk of T2C values of
// t2 and a tile of TH output rows; it computes Z2 and Z3 on the tile's rows
// plus (K-1)/2 halo rows on each side (clipped to the image) and loops over
// the rank in pairs.  LDS (32-bit words): two Zb buffers [T2C][S3/2][pixels]
// of bf16 pairs along s3 (the Z2 values of one rank), then the Zc planes
// [T2C*T3][HP][WP] holding Z3 of a rank pair as bf16 pairs (even rank in the
// low half) with zero rows and columns outside the image.
struct RcpDesc {
    int32_t S1, S2, S3, T2, T3, K, T2C, NT;   // the instantiation's compile-time sizes
    int32_t B, T1, R, H, W;
    int32_t nc;                // t2 chunks = T2 / T2C
    int32_t TH, ntiles;        // output rows per tile, tiles per image
    int32_t QW, WP, HP;        // output column quads per row; Zc plane pitch and rows
    int32_t zb_dw;             // one Zb buffer, 32-bit words (multiple of 4)
    int32_t plane_dw;          // one Zc plane = HP * WP words (multiple of 4)
    int32_t zc_dw;             // all Zc planes
    uint32_t lds_bytes;
    int64_t blocks;
};

// Fused backward of the same chain: one workgroup per (b, t1, tile of TH
// rows, t2 chunk), no halo recompute (the dY planes carry the halo).  LDS
// word offsets: o_dy dY planes [T2C*T3][HPb][WP] (fp32, zero outside the
// image), o_z1 Z1k [S2*S3][PP], o_z2 Z2k [S3*T2C][PP], o_z3 Z3k [T2C*T3][P],
// o_g3 G3k [T3*T2C][PP], o_g2 G2k [T2C*S3][PP] (bf16 rows), o_q the dW0 and
// dW1 partials summed over 16-lane rows [KK + S1][4 * NT/64], o_m3 / o_m2
// per-wave MFMA partials [NT/64][T3*S3] / [NT/64][T2C*S2] (fp32).
struct RcpBwdDesc {
    int32_t S1, S2, S3, T2, T3, K, T2C, NT;
    int32_t B, T1, R, H, W;
    int32_t nc, TH, ntiles;
    int32_t QW, WP, HPb, PP, L13, L2;   // bf16 row pitches: L13 = S3*PP + 8, L2 = T2C*PP + 8
    int32_t o_dy, o_z1, o_z2, o_z3, o_g3, o_g2, o_q, o_m3, o_m2;
    int32_t tbs;                        // words per rank of the prepared factor table
    uint32_t lds_bytes;
    int64_t blocks;
};

// The compiled instantiations: mode sizes S1, S2, S3, T2, T3 (T1 is free),
// filter size K, t2 chunk T2C, threads NT and the per-thread unit bounds of
// phases A, B, C (the planner picks the first that fits; the kernel file
// instantiates each).
struct RcpCfgInfo {
    int S1, S2, S3, T2, T3, K, T2C, NT, UA, UB, UC;
    int MW;   // backward: waves per SIMD the register budget is set for (launch bound)
};
constexpr RcpCfgInfo kRcpCfgs[] = {
    // 8x8x8 modes, 3x3 (tiles up to 9 x 7 with halo); a t2 chunk of 4 (C5a 97 us; 8: 109, 2: 137)
    {8, 8, 8, 8, 8, 3, 4, 256, 1, 2, 4, 0},
    // 4x4x8 modes, 5x5 (tiles up to 18 x 28 with halo); 512 threads (C5b 307 us; 448: 328;
    // 256 threads with twice the units a thread: 443; a t2 chunk of 1: 475)
    {4, 4, 8, 4, 8, 5, 2, 512, 4, 2, 4, 0},
};
constexpr int kNumRcpCfgs = 2;

// Backward instantiations (same fields; UA, UB, UC bound the units (pixel,
// s3), (pixel, t2) and (plane, row, 4 columns) of one tile per thread).
constexpr RcpCfgInfo kRcpBwdCfgs[] = {
    // 8x8x8 modes, 3x3 (tiles up to 64 pixels); one workgroup per CU (C5a: whole 7x7
    // planes, 449 us; 4-row tiles 689 us, 2-row 1242 us, a t2 chunk of 4 750 us)
    {8, 8, 8, 8, 8, 3, 8, 512, 1, 1, 2, 2},
    // 4x4x8 modes, 5x5 (tiles up to 64 pixels); 256 threads with registers capped at 128,
    // so that four workgroups share a CU and their barrier waits overlap (C5b: 2-row tiles,
    // 3584 workgroups, 1.96 ms; 448 threads and 4-row tiles 2.38 ms; 448 threads without
    // the cap 2.60 ms; a t2 chunk of 4 3.1-3.4 ms; 1-row tiles 2.9 ms)
    {4, 4, 8, 4, 8, 5, 2, 256, 2, 1, 1, 4},
};
constexpr int kNumRcpBwdCfgs = 2;

}  // namespace ce
