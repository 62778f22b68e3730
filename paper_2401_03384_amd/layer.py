"""PyTorch-facing layer over the C ABI.

PyTorch supplies device memory (tensors, the workspace) and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
"""
from __future__ import annotations

import math
import threading

import torch

from . import binding as B

_DT = {"f32": B.CE_F32, "bf16": B.CE_BF16}
_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}
_MODE = {"fwd": B.CE_COST_FWD, "train_paper": B.CE_COST_TRAIN_PAPER}


class Plan:
    """A planned conv_einsum layer: string, operand shapes, dtype.

    `path` (optional) is an opt_einsum-style list of pairs replacing the
    optimal order (e.g. the left-to-right baseline); `max_elements` (optional)
    caps the elements of every intermediate and `max_step_cost` the cost of
    every pairwise step (the cheapest order that fits); `save_budget`
    (bytes) lets the backward read that much of the forward's intermediates
    instead of recomputing them (the backward must then get the forward's
    workspace, see `forward(..., workspace=)`); `strides` maps convolved
    labels to their stride; `circular` lists two-way convolved labels to
    convolve circularly (labels of three or more operands always are)."""

    def __init__(self, spec: str, shapes, dtype: str = "f32", mode: str = "fwd", flags: int = 0,
                 path=None, feature_operand: int = 0, max_elements=None, max_step_cost=None,
                 save_budget=None, strides=None, circular=()):
        if dtype not in _DT:
            raise ValueError(f"dtype must be one of {list(_DT)}")
        self.spec = spec
        self.shapes = [tuple(int(d) for d in s) for s in shapes]
        self.dtype = dtype
        self.torch_dtype = _TORCH_DT[dtype]
        self.feature_operand = feature_operand
        self._expr = B.ce_expr_parse(spec, self.shapes)
        self._plan = None
        try:
            if feature_operand:
                B.ce_expr_set_feature(self._expr, feature_operand)
            self.strides = dict(strides or {})
            for label, st in self.strides.items():
                B.ce_expr_set_stride(self._expr, label, st)
            for label in circular:
                B.ce_expr_set_conv(self._expr, label, B.CE_PAD_CIRCULAR)
            self.out_shape = B.ce_expr_output_shape(self._expr)
            if path is None and (max_step_cost is not None or save_budget is not None):
                self._plan = B.ce_plan_create_ex(self._expr, _MODE[mode], _DT[dtype], flags,
                                                 int(max_step_cost or 0), int(max_elements or 0),
                                                 int(save_budget or 0))
            elif path is None and max_elements is not None:
                self._plan = B.ce_plan_create_limited(self._expr, _MODE[mode], _DT[dtype], flags,
                                                      int(max_elements))
            elif path is None:
                self._plan = B.ce_plan_create(self._expr, _MODE[mode], _DT[dtype], flags)
            else:
                self._plan = B.ce_plan_create_with_path(self._expr, path, _DT[dtype], flags)
        finally:
            B.ce_expr_destroy(self._expr)
            self._expr = None
        self.num_steps = B.ce_plan_num_steps(self._plan)
        self.steps = [B.ce_plan_step(self._plan, i) for i in range(self.num_steps)]
        self.total_cost, self.fwd_macs = B.ce_plan_cost(self._plan)
        self.ws_fwd = B.ce_plan_workspace_size(self._plan, 0)
        self.ws_bwd = B.ce_plan_workspace_size(self._plan, 1)
        self.saved_steps, self.saved_bytes, self.recompute_macs = B.ce_plan_checkpoint(self._plan)

    def __del__(self):
        if getattr(self, "_plan", None):
            B.ce_plan_destroy(self._plan)
            self._plan = None

    @property
    def handle(self):
        return self._plan

    def left_to_right_cost(self) -> int:
        return B.ce_plan_left_to_right_cost(self._plan)

    def describe(self) -> str:
        return B.ce_plan_describe(self._plan)

    def grad_dtype(self, i: int):
        return self.torch_dtype if i == self.feature_operand else torch.float32

    def _check_inputs(self, inputs):
        if len(inputs) != len(self.shapes):
            raise ValueError(f"expected {len(self.shapes)} operands")
        dev = inputs[0].device
        for i, (t, s) in enumerate(zip(inputs, self.shapes)):
            if tuple(t.shape) != s:
                raise ValueError(f"operand {i}: shape {tuple(t.shape)} != {s}")
            if t.dtype != self.torch_dtype:
                raise TypeError(f"operand {i}: dtype {t.dtype} != {self.torch_dtype}")
            if not t.is_cuda or t.device != dev:
                raise ValueError(f"operand {i} must be on {dev}")
            if not t.is_contiguous():
                raise ValueError(f"operand {i} must be contiguous")
        return dev

    @staticmethod
    def _stream(dev):
        return torch.cuda.current_stream(dev).cuda_stream

    def workspace(self, backward: bool, device) -> torch.Tensor:
        n = self.ws_bwd if backward else self.ws_fwd
        return torch.empty(max(n, 1), dtype=torch.uint8, device=device)

    def forward(self, inputs, out=None, workspace=None):
        dev = self._check_inputs(inputs)
        if out is None:
            out = torch.empty(self.out_shape, dtype=self.torch_dtype, device=dev)
        if workspace is None:
            workspace = self.workspace(False, dev)
        B.ce_forward(self._plan, [t.data_ptr() for t in inputs], out.data_ptr(),
                     workspace.data_ptr(), workspace.numel(), self._stream(dev))
        return out

    def backward(self, inputs, dout, needs=None, grads=None, workspace=None):
        dev = self._check_inputs(inputs)
        if tuple(dout.shape) != tuple(self.out_shape) or dout.dtype != self.torch_dtype or \
                not dout.is_contiguous():
            raise ValueError("dout must be contiguous, of the output shape and plan dtype")
        n = len(inputs)
        needs = [True] * n if needs is None else list(needs)
        if grads is None:
            grads = [torch.empty(self.shapes[i], dtype=self.grad_dtype(i), device=dev)
                     if needs[i] else None for i in range(n)]
        if workspace is None:
            workspace = self.workspace(True, dev)
        B.ce_backward(self._plan, [t.data_ptr() for t in inputs], dout.data_ptr(),
                      [g.data_ptr() if g is not None else 0 for g in grads],
                      workspace.data_ptr(), workspace.numel(), self._stream(dev))
        return grads


class GraphStep:
    """One forward + backward of a plan captured as a HIP graph on fixed
    buffers: replay() re-runs every launch without host work (planning and
    launch overhead gone; for launch-bound layers).  The inputs and dout given
    here are the graph's operands: refill them in place between replays.
    Outputs land in .out and .grads (allocated here), the workspace in .ws."""

    def __init__(self, plan: Plan, inputs, dout, warmup: int = 2):
        dev = plan._check_inputs(inputs)
        self.plan = plan
        self.inputs = list(inputs)
        self.dout = dout
        self.out = torch.empty(plan.out_shape, dtype=plan.torch_dtype, device=dev)
        self.grads = [torch.empty(s, dtype=plan.grad_dtype(i), device=dev)
                      for i, s in enumerate(plan.shapes)]
        self.ws = torch.empty(max(plan.ws_fwd, plan.ws_bwd, 1), dtype=torch.uint8, device=dev)
        side = torch.cuda.Stream(device=dev)   # default priority
        side.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(side):
            for _ in range(warmup):   # first launches set kernel attributes outside the capture
                self._run()
        torch.cuda.current_stream(dev).wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self._run()

    def _run(self):
        self.plan.forward(self.inputs, out=self.out, workspace=self.ws)
        self.plan.backward(self.inputs, self.dout, grads=self.grads, workspace=self.ws)

    def replay(self):
        self.graph.replay()


_cache = {}
_cache_lock = threading.Lock()


def plan(spec: str, shapes, dtype: str = "f32", mode: str = "fwd", flags: int = 0) -> Plan:
    """Cached Plan for (spec, shapes, dtype, mode, flags)."""
    key = (spec, tuple(tuple(s) for s in shapes), dtype, mode, flags)
    with _cache_lock:
        p = _cache.get(key)
        if p is None:
            p = Plan(spec, shapes, dtype, mode, flags)
            _cache[key] = p
        return p


class _ConvEinsumFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, spec, flags, *tensors):
        dtype = "bf16" if tensors[0].dtype == torch.bfloat16 else "f32"
        p = plan(spec, [t.shape for t in tensors], dtype, flags=flags)
        ctx.plan = p
        ctx.save_for_backward(*tensors)
        ctx.ws = None
        if flags & B.CE_FLAG_SAVE_INTERMEDIATES:
            # the backward reads the intermediates this forward leaves in its workspace
            ctx.ws = p.workspace(True, tensors[0].device)
            return p.forward(list(tensors), workspace=ctx.ws)
        return p.forward(list(tensors))

    @staticmethod
    def backward(ctx, dy):
        tensors = ctx.saved_tensors
        p = ctx.plan
        needs = list(ctx.needs_input_grad[2:])
        grads = p.backward(list(tensors), dy.contiguous().to(p.torch_dtype), needs=needs,
                           workspace=ctx.ws)
        grads = [g.to(t.dtype) if g is not None else None for g, t in zip(grads, tensors)]
        return (None, None, *grads)


def conv_einsum(spec: str, *tensors, flags: int = 0):
    """Evaluate a conv_einsum string on device tensors (differentiable)."""
    tensors = [t.contiguous() for t in tensors]
    return _ConvEinsumFn.apply(spec, flags, *tensors)


def contract_path(spec: str, *shapes, mode: str = "fwd", max_elements=None):
    """Planned order without executing: ([(lhs_mask, rhs_mask, macs)], info)."""
    p = Plan(spec, shapes, "f32", mode, max_elements=max_elements)
    info = {"total_cost": p.total_cost, "fwd_macs": p.fwd_macs,
            "left_to_right_cost": p.left_to_right_cost(), "text": p.describe()}
    return p.steps, info


def step_bytes(p: Plan) -> int:
    """Device bytes one forward + backward of plan `p` holds: operands,
    output and output gradient, operand gradients, and one workspace serving
    both passes."""
    e = 2 if p.dtype == "bf16" else 4
    ins = sum(math.prod(s) for s in p.shapes) * e
    out = 2 * math.prod(p.out_shape) * e
    grads = sum(math.prod(s) * (e if i == p.feature_operand else 4) for i, s in enumerate(p.shapes))
    return ins + out + grads + max(p.ws_fwd, p.ws_bwd)


def max_batch(spec: str, shapes, budget_bytes: int, dtype: str = "f32", order: str = "optimal",
              save: bool = False, fusion: bool = True, batch=((0, 0),), limit: int = 1 << 20) -> int:
    """Largest batch size whose training step (step_bytes) fits in
    budget_bytes: the one-layer analogue of the maximum-batch comparison of
    Section 5 (Table 3).  `batch` lists the (operand, axis) pairs that carry
    the batch size; order "optimal" is the planned order, "ltr" the
    left-to-right baseline; save=True keeps every intermediate for the
    backward (no checkpointing); fusion=False materialises every pairwise
    result (one launch per step, as an evaluation without fused chains does).
    0 when even a batch of one does not fit."""
    n = len(shapes)
    path = None
    if order == "ltr":
        path = [(0, 1)] + [(0, n - 1 - k) for k in range(1, n - 1)]
    elif order != "optimal":
        raise ValueError("order must be 'optimal' or 'ltr'")
    flags = (B.CE_FLAG_SAVE_INTERMEDIATES if save else 0) | (0 if fusion else B.CE_FLAG_NO_FUSION)

    def fits(bs):
        shp = [list(s) for s in shapes]
        for i, ax in batch:
            shp[i][ax] = bs
        try:
            return step_bytes(Plan(spec, shp, dtype, flags=flags, path=path)) <= budget_bytes
        except B.CeError:
            return False

    if not fits(1):
        return 0
    lo, hi = 1, 2
    while hi <= limit and fits(hi):
        lo, hi = hi, hi * 2
    hi = min(hi, limit + 1)
    while hi - lo > 1:     # fits(lo), not fits(hi)
        mid = (lo + hi) // 2
        if fits(mid):
            lo = mid
        else:
            hi = mid
    return lo
