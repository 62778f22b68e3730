import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (HIP device)")
    config.addinivalue_line("markers", "slow: long-running CPU check")


def load_layer_strings():
    path = os.path.join(ROOT, "tests", "golden", "layer_strings.txt")
    out = {}
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, spec, cite = [x.strip() for x in line.split(" | ")]
            out[name] = (spec, cite)
    return out


# Small operand shapes for every executable layer string the paper prints
# (tests/golden/layer_strings.txt): convolved labels 9 (or 10, 11) on the
# feature side and 3 on the filter side, other labels 2 to 6.
PAPER_SHAPES = {
    "standard_conv": [(2, 3, 9, 9), (4, 3, 3, 3)],
    "cp_conv": [(2, 6, 9, 9), (3, 5), (3, 6), (3, 3), (3, 3)],
    "rcp_conv": [(2, 2, 3, 2, 9, 9), (4, 2, 2), (4, 3, 3), (4, 2, 2), (4, 3, 3)],
    "tucker_conv": [(2, 6, 9, 9), (3, 5), (2, 6), (3, 2, 3, 3)],
    "rtk_conv": [(2, 2, 3, 2, 9, 9), (2, 2, 2), (3, 3, 3), (2, 2, 2), (2, 3, 3), (2, 2, 3, 2)],
    "tt_conv": [(2, 6, 9, 9), (2, 5), (2, 3, 3), (3, 2, 3), (2, 6)],
    "rtt_conv": [(2, 2, 3, 2, 9, 9), (2, 2, 2), (2, 3, 3, 3), (3, 2, 2, 2), (2, 3, 3)],
    "tr_conv": [(2, 6, 9, 9), (2, 3, 5), (3, 2, 3), (2, 2, 3), (2, 2, 6)],
    "rtr_conv": [(2, 2, 3, 2, 9, 9), (2, 2, 2, 2), (2, 3, 3, 3), (3, 2, 2, 2), (2, 2, 3, 3)],
    "bt_conv": [(2, 2, 3, 2, 9, 9), (2, 2, 2, 2), (2, 2, 3, 3), (2, 2, 2, 2), (2, 2, 3, 3),
                (2, 2, 2, 2, 2)],
    "ht_conv": [(1, 2, 3, 2, 9, 9), (2, 2, 2), (2, 3, 3), (2, 2, 2), (2, 3, 3), (2, 2, 2),
                (2, 2, 2), (2, 2)],
    "separable_depthwise": [(2, 5, 9, 9), (5, 3), (5, 3)],
    "interleaved_group": [(2, 2, 3, 9, 9), (4, 2, 3, 3), (5, 3, 3, 3)],
    "sequencer_example": [(4, 7, 9), (10, 5), (5, 4, 2), (6, 8, 9, 2)],
    "conv1d": [(2, 3, 11), (4, 3, 3)],
    "group_conv1d": [(2, 3, 2, 3), (2, 2, 2, 10)],
    "three_way_contraction": [(2, 3, 4), (3, 5, 3), (4, 4, 5)],
    "interleaved_group_sec2": [(2, 2, 3, 9, 9), (2, 4, 3, 3), (3, 5, 3, 3)],
    "group_conv2d": [(2, 3, 2, 3, 3), (2, 2, 2, 9, 9)],
    "tensor_conv": [(5, 2, 3), (3, 2, 4)],
    "contraction": [(3, 2, 4), (3, 5, 2)],
    "outer": [(2, 3, 2), (2, 2, 3)],
    "batch": [(2, 3, 4), (2, 3, 5)],
}

# The method's degenerate and edge cases: (string, operand shapes, designated
# feature operand).  Section 3.1 case (5) pre-sums, a single operand, the
# feature side held by the second operand, equal feature / filter sizes
# resolved by the designated feature operand, even filter sizes.
EDGE_CASES = {
    "self_contraction": ("bsm,mt->bt", [(3, 4, 5), (5, 6)], 0),
    "self_contraction_conv": ("bsmh,mth->bth|h", [(2, 3, 4, 9), (4, 5, 3)], 0),
    "single_operand_sum": ("ijk->i", [(3, 4, 5)], 0),
    "single_operand_permute": ("ijk->kji", [(3, 4, 5)], 0),
    "feature_second": ("tsh,bsh->bth|h", [(4, 3, 3), (2, 3, 11)], 0),
    "feature_second_2d": ("tshw,bshw->bthw|hw", [(4, 3, 3, 2), (2, 3, 9, 8)], 0),
    "equal_sizes_feature0": ("bsh,tsh->bth|h", [(2, 3, 5), (4, 3, 5)], 0),
    "equal_sizes_feature1": ("bsh,tsh->bth|h", [(2, 3, 5), (4, 3, 5)], 1),
    "even_filter_conv": ("bshw,tshw->bthw|hw", [(2, 3, 9, 10), (4, 3, 4, 4)], 0),
    "even_filter_cp": ("bshw,rs,rt,rh,rw->bthw|hw", [(2, 6, 9, 9), (3, 6), (3, 5), (3, 4), (3, 2)], 0),
    # three and four convolved labels in one step (conv3d, conv4d; Section 3.1)
    "conv3d": ("bsdhw,tsdhw->btdhw|dhw", [(2, 3, 6, 7, 8), (4, 3, 3, 3, 3)], 0),
    "conv4d": ("bsdhwx,tsdhwx->btdhwx|dhwx", [(1, 2, 5, 6, 4, 5), (3, 2, 3, 3, 2, 3)], 0),
}

# Circular (commutative) convolutions, Appendix B: (string, shapes, two-way
# labels made circular).  Labels held by three or more operands are circular
# by default.
CIRCULAR_CASES = {
    "circ_3way_1d": ("bi,ci,di->bcdi|i", [(2, 9), (3, 3), (2, 4)], ()),
    "circ_2way": ("bsh,tsh->bth|h", [(2, 3, 8), (4, 3, 5)], ("h",)),
    "circ_2way_2d": ("bshw,tshw->bthw|hw", [(2, 3, 7, 6), (4, 3, 3, 4)], ("h", "w")),
    "circ_interleaved": ("bmshw,nmhw,tshw->bnthw|hw",
                         [(2, 3, 4, 9, 10), (5, 3, 3, 3), (4, 4, 5, 2)], ()),
    "circ_4way": ("ai,bi,ci,di->abcdi|i", [(2, 7), (2, 3), (1, 7), (2, 2)], ()),
}


# Strided convolutions (Appendix B varieties): name -> (string, shapes,
# strides as "label=stride,...").  3x3 and 7x7 with stride 2, a strided 1x1
# (taps reach only every other position), stride 3, CP and Tucker layers,
# the feature operand second.
STRIDED_CASES = {
    "conv3_s2": ("bshw,tshw->bthw|hw", [(2, 3, 9, 8), (5, 3, 3, 3)], "h=2,w=2"),
    "conv7_s2": ("bshw,tshw->bthw|hw", [(1, 3, 13, 12), (4, 3, 7, 7)], "h=2,w=2"),
    "conv1_s2": ("bshw,tshw->bthw|hw", [(2, 6, 7, 8), (5, 6, 1, 1)], "h=2,w=2"),
    "conv3_s3h": ("bshw,tshw->bthw|hw", [(2, 3, 10, 9), (4, 3, 3, 3)], "h=3"),
    "cp_s2": ("bshw,rs,rt,rh,rw->bthw|hw", [(2, 6, 9, 10), (4, 6), (4, 5), (4, 3), (4, 3)],
              "h=2,w=2"),
    "tucker_s2": ("bshw,sp,pqhw,qt->bthw|hw", [(2, 8, 9, 9), (8, 4), (4, 6, 3, 3), (6, 5)],
                  "h=2,w=2"),
    "feature_second_s2": ("tsh,bsh->bth|h", [(4, 3, 3), (2, 3, 11)], "h=2"),
}


def strides_of(text):
    return {kv.split("=")[0]: int(kv.split("=")[1]) for kv in text.split(",") if kv}
