"""The allocation-free backward entry point (ce_backward_noalloc) through the
C ABI: its gradients equal ce_backward's (bit for bit: the same kernels on
the same inputs) and the oracle's, over several calls in a row that share the
library's fixed device workspace, each later call on a smaller layer than
the one before (the array keeps the previous call's contents)."""
import sys

import numpy as np
import pytest

import oracle as O
import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# largest backward workspace first: fused reshaped CP (partials), Tucker-2
# (intermediates and split-reduction partials), fused CP, unfused CP
SEQUENCE = ["C5bs", "C3s", "C2s", "C1"]


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _dev(a, bf16):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return (t.to(torch.bfloat16) if bf16 else t).cuda()


def _host(t):
    return t.float().cpu().numpy().astype(np.float64)


def test_noalloc_backward_matches_backward():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    import paper_2401_03384_amd as P
    P.lib()
    prev_ws = None
    for name in SEQUENCE:
        w = W.PARITY_WORKLOADS[name]
        bf16 = w.dtype == "bf16"
        tol = 2e-2 if bf16 else 1e-5
        plan = P.Plan(w.spec, w.shapes, w.dtype)
        _say(f"case {name} shapes={w.shapes} workspace {plan.ws_bwd} B")
        assert 0 < plan.ws_bwd <= P.CE_NOALLOC_WORKSPACE_BYTES
        if prev_ws is not None:
            assert plan.ws_bwd < prev_ws
        prev_ws = plan.ws_bwd
        ins, dy = W.make_inputs(w)
        xs = [_dev(a, bf16) for a in ins]
        d = _dev(dy, bf16)
        ref = plan.backward(xs, d)
        got = [torch.full_like(g, float("nan")) for g in ref]
        stream = torch.cuda.current_stream().cuda_stream
        P.ce_backward_noalloc(plan.handle, [x.data_ptr() for x in xs], d.data_ptr(),
                              [g.data_ptr() for g in got], stream)
        torch.cuda.synchronize()
        e = O.bind(O.parse(w.spec), w.shapes)
        tree = O.optimal_tree(e)[0]
        g_ref = O.grads_pairwise(e, ins, tree, dy)
        for i, (a, b, r) in enumerate(zip(got, ref, g_ref)):
            assert torch.equal(a, b), (name, i)
            h = _host(a)
            rel = float(np.linalg.norm(h - r) / np.linalg.norm(r))
            worst = float(np.abs(h - r).max() / np.abs(r).max())
            _say(f"  d{i}: rel-L2 {rel:.3e}, worst element {worst:.3e}")
            assert rel <= tol and worst <= tol, (name, i, rel, worst)
