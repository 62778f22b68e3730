"""The seeded input generator: bf16 rounding against PyTorch's float32 ->
bfloat16 conversion (round to nearest even), reproducibility and shapes."""
import numpy as np
import torch

import workloads as W


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    x = np.concatenate([g.standard_normal(100000).astype(np.float32) * 3,
                        np.float32([1.0, 1.00390625, 1.005859375, -2.5, 0.0, -0.0, 1e-40,
                                    3.3e38, 65504.0])])
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(W.round_to_bf16(x), ref)
    bits = W.bf16_bits(W.round_to_bf16(x))
    np.testing.assert_array_equal(bits, torch.tensor(ref).to(torch.bfloat16).view(torch.int16)
                                  .numpy().view(np.uint16))


def test_inputs_are_reproducible_and_shaped():
    for w in W.PARITY_WORKLOADS.values():
        a, dy = W.make_inputs(w)
        b, dy2 = W.make_inputs(w)
        assert [x.shape for x in a] == [tuple(s) for s in w.shapes]
        assert dy.shape == tuple(w.out_shape)
        for x, y in zip(a, b):
            np.testing.assert_array_equal(x, y)
        if w.dtype == "bf16":
            for x in a:
                np.testing.assert_array_equal(W.round_to_bf16(x.astype(np.float32)), x)
        else:
            for x in a:
                np.testing.assert_array_equal(x.astype(np.float32).astype(np.float64), x)
