"""Seeded synthetic inputs for the tensorial-convolution layers.

This module is shared by the oracle (CPU, float64) and by the HIP path.  It
holds no arithmetic of the method itself: only layer strings, operand shapes,
the random draws and the rounding of those draws to the storage type.

Layer strings follow the conv_einsum notation of Section 2.2 and the layer
catalogue of Appendix A.3 (CP, Tucker-2, reshaped TT, reshaped CP); the shapes
are ResNet stage shapes standing in for the paper's ImageNet/CIFAR activations
(Section 5), which are not available here.

Recipe, per workload:
  * numpy Generator(PCG64) streams from SeedSequence(seed).spawn(n_in + 1); the
    last stream draws the output gradient dY;
  * the feature operand (operand 0) is N(0, 1); factors are N(0, sigma^2);
  * values are drawn in float64, rounded to float32, and for bf16 workloads
    rounded again to bfloat16 (round-to-nearest-even on the float32 bit
    pattern, from the format definition: 1 sign, 8 exponent, 7 mantissa bits).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = ["Workload", "WORKLOADS", "PARITY_WORKLOADS", "make_inputs", "cp_layer",
           "RESNET34_CONVS", "cp_rank", "resnet34_cp_layer",
           "tucker2_layer", "rtt_layer", "rcp_layer", "round_to_bf16", "bf16_bits", "f32_bits"]


@dataclass(frozen=True)
class Workload:
    name: str
    spec: str
    shapes: tuple            # one shape per input operand, label order of the string
    dtype: str               # "f32" or "bf16": storage type of inputs
    seed: int
    sigmas: tuple            # std of each input operand
    out_shape: tuple         # output shape, label order of the string
    backward: bool = True
    note: str = ""


def _kaiming_sigma(fan_in: int, ranks: int, n_factors: int) -> float:
    """Per-factor std so that the reconstructed dense kernel has variance
    2/fan_in: each dense entry is a sum of `ranks` products of `n_factors`
    independent factor entries."""
    return (2.0 / (fan_in * ranks)) ** (1.0 / (2 * n_factors))


def cp_layer(name, b, s, t, h, w, r, k, dtype, seed, backward=True, sig=None, note=""):
    spec = "bshw,rs,rt,rh,rw->bthw|hw"
    shapes = ((b, s, h, w), (r, s), (r, t), (r, k), (r, k))
    if sig is None:
        sg = _kaiming_sigma(s * k * k, r, 4)
        sig = (1.0, sg, sg, sg, sg)
    return Workload(name, spec, shapes, dtype, seed, tuple(sig), (b, t, h, w), backward, note)


def tucker2_layer(name, b, s, t, h, w, p, q, k, dtype, seed, note=""):
    spec = "bshw,sp,pqhw,qt->bthw|hw"
    shapes = ((b, s, h, w), (s, p), (p, q, k, k), (q, t))
    sg = _kaiming_sigma(s * k * k, p * q, 3)
    return Workload(name, spec, shapes, dtype, seed, (1.0, sg, sg, sg), (b, t, h, w), True, note)


def rtt_layer(name, b, s3s, t3s, h, w, r, k, dtype, seed, note=""):
    spec = ("b(s1)(s2)(s3)hw,(r1)(t1)(s1),(r1)(r2)(t2)(s2),(r2)(r3)(t3)(s3),(r3)hw"
            "->b(t1)(t2)(t3)hw|hw")
    s1, s2, s3 = s3s
    t1, t2, t3 = t3s
    shapes = ((b, s1, s2, s3, h, w), (r, t1, s1), (r, r, t2, s2), (r, r, t3, s3), (r, k, k))
    sg = _kaiming_sigma(s1 * s2 * s3 * k * k, r ** 3, 4)
    return Workload(name, spec, shapes, dtype, seed, (1.0, sg, sg, sg, sg),
                    (b, t1, t2, t3, h, w), True, note)


def rcp_layer(name, b, s3s, t3s, h, w, r, k, dtype, seed, note=""):
    spec = "b(s1)(s2)(s3)hw,r(t1)(s1),r(t2)(s2),r(t3)(s3),rhw->b(t1)(t2)(t3)hw|hw"
    s1, s2, s3 = s3s
    t1, t2, t3 = t3s
    shapes = ((b, s1, s2, s3, h, w), (r, t1, s1), (r, t2, s2), (r, t3, s3), (r, k, k))
    sg = _kaiming_sigma(s1 * s2 * s3 * k * k, r, 4)
    return Workload(name, spec, shapes, dtype, seed, (1.0, sg, sg, sg, sg),
                    (b, t1, t2, t3, h, w), True, note)


# Full-size layers.  C1 uses std 1/sqrt(fan), fan = the size summed when the
# factor is applied (U_s: s, U_t: r, K_h/K_w: taps).
WORKLOADS = {
    "C1": cp_layer("C1", 2, 16, 16, 8, 8, 8, 3, "f32", 1, backward=False,
              sig=(1.0, 1 / math.sqrt(16), 1 / math.sqrt(8), 1 / math.sqrt(3), 1 / math.sqrt(3)),
              note="CP 3x3, tiny, forward only"),
    "C2": cp_layer("C2", 128, 64, 64, 56, 56, 32, 3, "f32", 2,
              note="CP 3x3, ResNet stage-1 shape, rank 32"),
    "C2_bf16": cp_layer("C2_bf16", 128, 64, 64, 56, 56, 32, 3, "bf16", 2,
                   note="CP 3x3, ResNet stage-1 shape, rank 32, bf16 inputs"),
    "C3": tucker2_layer("C3", 128, 256, 256, 14, 14, 64, 64, 3, "bf16", 3,
                   note="Tucker-2 3x3, core 64x64"),
    "C4": rtt_layer("C4", 64, (4, 8, 8), (4, 8, 8), 28, 28, 16, 3, "f32", 4,
               note="reshaped tensor-train 3x3, channels 4x8x8, TT rank 16"),
    "C5a": rcp_layer("C5a", 32, (8, 8, 8), (8, 8, 8), 7, 7, 64, 3, "bf16", 5,
                note="reshaped CP 3x3, channels 8x8x8, rank 64, 7x7"),
    "C5b": rcp_layer("C5b", 32, (4, 4, 8), (4, 4, 8), 28, 28, 64, 5, "bf16", 6,
                note="reshaped CP 5x5, channels 4x4x8, rank 64, 28x28"),
}

# Reduced sizes (same strings, same ranks) that the float64 oracle finishes in
# seconds while still spanning several kernel tiles and a ragged tail.
PARITY_WORKLOADS = {
    "C1": WORKLOADS["C1"],
    "C2s": cp_layer("C2s", 2, 64, 64, 19, 19, 32, 3, "f32", 12),
    "C2s_bf16": cp_layer("C2s_bf16", 2, 64, 64, 19, 19, 32, 3, "bf16", 12),
    "C2r32": cp_layer("C2r32", 3, 32, 32, 13, 37, 32, 3, "f32", 17),
    "C2r32_bf16": cp_layer("C2r32_bf16", 3, 32, 32, 13, 37, 32, 3, "bf16", 17),
    "C2k5": cp_layer("C2k5", 2, 64, 32, 12, 29, 32, 5, "f32", 18),
    # enough strips that the fused backward walks segments of several rows,
    # with a one-row segment at the bottom (4-row and 2-row segments)
    "C2seg": cp_layer("C2seg", 128, 32, 32, 29, 16, 32, 3, "f32", 21),
    "C2seg_bf16": cp_layer("C2seg_bf16", 64, 64, 64, 23, 20, 32, 3, "bf16", 22),
    # enough samples that the fused forward walks segments of several rows:
    # 6-row segments (the two-row loop, no odd row; backward: one 12-row
    # segment), 4-row segments over 13 rows (a 1-row last segment; backward
    # 7-row segments), and bf16 5-row segments (odd ones walked upwards)
    "C2fseg6": cp_layer("C2fseg6", 1024, 32, 32, 12, 8, 32, 3, "f32", 23),
    "C2fseg4": cp_layer("C2fseg4", 512, 32, 32, 13, 8, 32, 3, "f32", 24),
    "C2fseg5_bf16": cp_layer("C2fseg5_bf16", 1024, 32, 32, 10, 8, 32, 3, "bf16", 25),
    # fused CP chains with ranks below 32 (ranks past R run as zero rows)
    "C2r16": cp_layer("C2r16", 3, 64, 64, 13, 37, 16, 3, "f32", 26),
    "C2r8_bf16": cp_layer("C2r8_bf16", 3, 32, 64, 11, 19, 8, 3, "bf16", 27),
    "C2r20k5": cp_layer("C2r20k5", 2, 64, 32, 12, 29, 20, 5, "f32", 28),
    # channel counts off the 32 / 64 blocks (padded with zero table entries)
    "C2c48": cp_layer("C2c48", 2, 48, 40, 13, 37, 24, 3, "f32", 29),
    "C2c16_bf16": cp_layer("C2c16_bf16", 3, 16, 16, 11, 19, 8, 3, "bf16", 30),
    "C2c20k5": cp_layer("C2c20k5", 2, 20, 56, 12, 29, 32, 5, "f32", 31),
    "C3s": tucker2_layer("C3s", 3, 256, 256, 11, 13, 64, 64, 3, "bf16", 13),
    "C3s_f32": tucker2_layer("C3s_f32", 3, 256, 256, 11, 13, 64, 64, 3, "f32", 13),
    "C4s": rtt_layer("C4s", 2, (4, 8, 8), (4, 8, 8), 13, 13, 16, 3, "f32", 14),
    "C5as": rcp_layer("C5as", 3, (8, 8, 8), (8, 8, 8), 7, 7, 64, 3, "bf16", 15),
    "C5as_f32": rcp_layer("C5as_f32", 3, (8, 8, 8), (8, 8, 8), 7, 7, 64, 3, "f32", 15),
    "C5bs": rcp_layer("C5bs", 2, (4, 4, 8), (4, 4, 8), 11, 11, 64, 5, "bf16", 16),
    # fused reshaped-CP forward on row tiles: two tiles (23 x 26) and three
    # (50 x 20, a middle tile with halo rows on both sides)
    "C5bt2": rcp_layer("C5bt2", 1, (4, 4, 8), (2, 4, 8), 23, 26, 4, 5, "bf16", 27),
    "C5bt3": rcp_layer("C5bt3", 1, (4, 4, 8), (3, 4, 8), 50, 20, 2, 5, "bf16", 28),
    # Tucker cores on MFMA tiles: ragged channel counts (padded to 16 / 32),
    # 5 x 5 taps, and an input too wide for one block's LDS (row tiles)
    "C3c": tucker2_layer("C3c", 2, 24, 40, 5, 11, 20, 40, 3, "bf16", 31),
    "C3c5": tucker2_layer("C3c5", 1, 16, 24, 6, 7, 36, 24, 5, "bf16", 32),
    "C3m": tucker2_layer("C3m", 2, 16, 24, 6, 20, 128, 40, 3, "bf16", 33),
    # channel mixes over flattened (batch, pixel) columns: 144-pixel planes
    # across 128-column tiles, reductions of 96 and 48 (a partial 64-chunk),
    # ragged row tiles (40, 72 rows); and 256 rows in 64-row tiles
    "C3f": tucker2_layer("C3f", 3, 96, 72, 12, 12, 40, 48, 3, "bf16", 41),
    "C3f2": tucker2_layer("C3f2", 32, 72, 256, 16, 16, 24, 40, 3, "bf16", 42),
    # the same kernel in fp32 (Tucker core; the tensor-train layer's transposed conv)
    "C3c_f32": tucker2_layer("C3c_f32", 2, 24, 40, 5, 11, 20, 40, 3, "f32", 31),
    # the fp32 conv-contraction kernel proper (6 contracted channels, 5 x 5
    # taps, a ragged 12 x 13 plane)
    "C3p5": tucker2_layer("C3p5", 2, 32, 24, 12, 13, 6, 40, 5, "f32", 47),
    "C4c": rtt_layer("C4c", 1, (2, 2, 4), (2, 2, 2), 6, 7, 16, 3, "f32", 34),
    # the full tensor-train chain at channel sizes of the 28x28 layer, small planes
    "C4w": rtt_layer("C4w", 2, (4, 8, 8), (4, 8, 8), 9, 11, 16, 3, "f32", 35),
    # the fused contraction + convolution with 17-32 and 33-64 columns, ragged
    # row bands, fewer than 8 output channels, and a contraction of 12 (not a
    # multiple of 4) or 8 terms
    "C4x2": rtt_layer("C4x2", 2, (4, 8, 4), (4, 4, 4), 21, 30, 16, 3, "f32", 36),
    "C4x4": rtt_layer("C4x4", 2, (3, 8, 4), (4, 4, 6), 9, 40, 16, 3, "f32", 37),
    "C4x1": rtt_layer("C4x1", 3, (4, 8, 4), (4, 8, 5), 6, 16, 16, 3, "f32", 38),
    # the transposed convolution with its filter operands in registers: a
    # partial q tile (48 columns) and 7 channels on a ragged plane, a 2 x 2
    # filter, a 40 x 36 plane in two row tiles
    "C4q": rtt_layer("C4q", 2, (4, 8, 3), (4, 8, 7), 9, 11, 16, 3, "f32", 43),
    "C4k2": rtt_layer("C4k2", 2, (4, 8, 3), (4, 8, 7), 9, 11, 16, 2, "f32", 44),
    "C4p": rtt_layer("C4p", 1, (4, 8, 3), (4, 8, 7), 40, 36, 16, 3, "f32", 45),
    # enough reduction per rank for the streaming factor-gradient kernel
    # (ragged 15 x 15 planes, and 16 x 16 with four-wide loads)
    "C5cs": rcp_layer("C5cs", 20, (2, 2, 4), (2, 2, 4), 15, 15, 8, 3, "bf16", 19),
    "C5cs_f32": rcp_layer("C5cs_f32", 16, (2, 2, 4), (2, 2, 4), 16, 16, 8, 5, "f32", 20),
}


# The convolutions of ResNet-34 on 224 x 224 inputs (stem, the four stages'
# first and repeated 3x3 convolutions, and the strided 1x1 shortcuts) as CP
# layers: (name, C_in, C_out, input size, kernel size, stride).  These are the
# layer shapes of the paper's per-layer FLOPs comparison (Section 5, Table 2:
# ResNet-34, CP layers, compression rate 100%).
RESNET34_CONVS = [
    ("conv1", 3, 64, 224, 7, 2),
    ("conv2_x", 64, 64, 56, 3, 1),
    ("conv3_1", 64, 128, 56, 3, 2),
    ("conv3_x", 128, 128, 28, 3, 1),
    ("conv3_sc", 64, 128, 56, 1, 2),
    ("conv4_1", 128, 256, 28, 3, 2),
    ("conv4_x", 256, 256, 14, 3, 1),
    ("conv4_sc", 128, 256, 28, 1, 2),
    ("conv5_1", 256, 512, 14, 3, 2),
    ("conv5_x", 512, 512, 7, 3, 1),
    ("conv5_sc", 256, 512, 14, 1, 2),
]


def cp_rank(s, t, k, cr=1.0):
    """CP rank whose factors hold cr times the parameters of the dense
    t x s x k x k kernel: R (s + t + 2k) = cr * t s k^2, rounded down (at
    least 1)."""
    return max(1, int(cr * t * s * k * k) // (s + t + 2 * k))


def resnet34_cp_layer(name, batch=128, cr=1.0, scale=1, dtype="f32", seed=50):
    """CP layer of a ResNet-34 convolution (RESNET34_CONVS) with strides on h
    and w; `scale` divides the channel counts and the input size (at least
    3 channels, 5 positions) for reduced-size cases.  Returns (Workload,
    strides)."""
    row = {r[0]: r for r in RESNET34_CONVS}[name]
    _, s, t, hw, k, st = row
    if scale > 1:
        s, t, hw = max(3, s // scale), max(3, t // scale), max(5, hw // scale)
    r = cp_rank(s, t, k, cr)
    out = -(-hw // st)
    sg = _kaiming_sigma(s * k * k, r, 4)
    w = Workload(f"{name}_b{batch}" + (f"_s{scale}" if scale > 1 else ""),
                 "bshw,rs,rt,rh,rw->bthw|hw",
                 ((batch, s, hw, hw), (r, s), (r, t), (r, k), (r, k)), dtype, seed,
                 (1.0, sg, sg, sg, sg), (batch, t, out, out), True,
                 note=f"ResNet-34 {name} as a CP layer, stride {st}")
    return w, ({"h": st, "w": st} if st > 1 else {})


def round_to_bf16(x) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns
    float32 arrays holding exactly representable bfloat16 values."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    out = u.astype(np.uint32).view(np.float32)
    nan = np.isnan(f)
    if nan.any():
        out = out.copy()
        out[nan] = np.float32("nan")
    return out


def bf16_bits(x) -> np.ndarray:
    """Raw bfloat16 bit patterns (uint16) of values already representable in
    bfloat16 (as produced by round_to_bf16)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def f32_bits(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float32))


def make_inputs(w: Workload, with_dy: bool = True):
    """Draw the operands (and dY) of workload `w`.

    Returns (inputs, dy): a list of float64 arrays and one float64 array (or
    None) whose values are exactly the stored values (float32, or bfloat16
    for bf16 workloads).
    """
    n = len(w.shapes)
    streams = np.random.SeedSequence(w.seed).spawn(n + 1)
    rnd = round_to_bf16 if w.dtype == "bf16" else (lambda a: np.asarray(a, np.float32))
    ins = []
    for i, shp in enumerate(w.shapes):
        g = np.random.Generator(np.random.PCG64(streams[i]))
        a = g.standard_normal(size=shp) * w.sigmas[i]
        ins.append(rnd(a.astype(np.float32)).astype(np.float64))
    dy = None
    if with_dy:
        g = np.random.Generator(np.random.PCG64(streams[n]))
        dy = rnd(g.standard_normal(size=tuple(w.out_shape)).astype(np.float32)).astype(np.float64)
    return ins, dy
