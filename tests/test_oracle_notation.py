"""Pins for the oracle's string grammar and size binding (CPU)."""
import pytest

import oracle as O
from conftest import load_layer_strings

STRINGS = load_layer_strings()


@pytest.mark.parametrize("name", sorted(STRINGS))
def test_every_printed_layer_string_parses(name):
    spec, _ = STRINGS[name]
    e = O.parse(spec)
    # every output label comes from some operand; conv labels are kept
    present = {l for t in e.inputs for l in t}
    assert set(e.output) <= present
    assert set(e.conv) <= set(e.output)


def test_multichar_labels_and_roles():
    e = O.parse(STRINGS["rcp_conv"][0])
    assert e.inputs[0] == ["b", "s1", "s2", "s3", "h", "w"]
    assert e.inputs[1] == ["r", "t1", "s1"]
    assert e.inputs[4] == ["r", "h", "w"]
    assert e.output == ["b", "t1", "t2", "t3", "h", "w"]
    assert e.conv == ["h", "w"]
    ht = O.parse(STRINGS["ht_conv"][0])
    assert ht.n == 8 and ht.inputs[7] == ["r4", "r5"]


def test_conv_list_forms_agree():
    a = O.parse("gtshw,bgshw->bgthw|h,w")
    b = O.parse("gtshw,bgshw->bgthw|hw")
    c = O.parse(" g t s h w , b g s h w -> b g t h w | h w ")
    assert a.conv == b.conv == c.conv == ["h", "w"]
    assert a.inputs == b.inputs == c.inputs


@pytest.mark.parametrize("bad", [
    "bshw,tshw",                  # no '->'
    "bshw->bsh->b",               # two arrows
    "bssw,tshw->bthw|hw",         # repeated label in one operand
    "bshw,tshw->bthwx|hw",        # output label in no operand
    "bshw,tshw->bthw|hz",         # convolved label in no operand
    "bshw,tshw->bt|hw",           # convolved label dropped from the output
    "bshw,tshw->bbthw",           # repeated output label
    "bs(h,tshw->bthw",            # unclosed parenthesis
    "bs1,ts->bt",                 # digit outside parentheses
])
def test_malformed_strings_are_rejected(bad):
    with pytest.raises(ValueError):
        O.parse(bad)


def test_non_convolved_sizes_must_agree():
    e = O.parse("bshw,tshw->bthw|hw")
    with pytest.raises(ValueError):
        O.bind(e, [(2, 3, 8, 8), (4, 5, 3, 3)])       # s = 3 vs 5
    with pytest.raises(ValueError):
        O.bind(O.parse("bshw,tshw->bthw|hw"), [(2, 3, 8), (4, 3, 3, 3)])  # rank


def test_convolved_sizes_may_differ_and_feature_is_larger():
    e = O.bind(O.parse("bshw,tshw->bthw|hw"), [(2, 3, 8, 9), (4, 3, 3, 5)])
    assert e.feature == {"h": 0, "w": 0}
    assert e.out_sizes == {"b": 2, "t": 4, "h": 8, "w": 9}
    e = O.bind(O.parse("tshw,bshw->bthw|hw"), [(4, 3, 3, 5), (2, 3, 8, 9)])
    assert e.feature == {"h": 1, "w": 1}


def test_equal_sizes_go_to_designated_feature_operand():
    e = O.bind(O.parse("bsh,tsh->bth|h"), [(2, 3, 5), (4, 3, 5)])
    assert e.feature == {"h": 0}
    e = O.bind(O.parse("bsh,tsh->bth|h"), [(2, 3, 5), (4, 3, 5)], feature_operand=1)
    assert e.feature == {"h": 1}


def test_multiway_label_has_no_feature_side():
    e = O.bind(O.parse(STRINGS["sequencer_example"][0]), [(4, 7, 9), (10, 5), (5, 4, 2), (6, 8, 9, 2)])
    assert "j" not in e.feature
    assert e.out_sizes["j"] == 10
