"""Registers a PyTorch model's parameter gradients as GNMR units.

Each unit is the set of parameters that `unit_of(name)` maps to one key
(default: every parameter is its own unit; mapping a whole block's parameters
to one key gives the block-as-unit granularity of Sec. 3.4).  A unit's
segments are its parameters' `.grad` tensors, in registration order.  The
gradient pointers are passed to the library on every step, because
`zero_grad(set_to_none=True)` reallocates `.grad` buffers.

Argument marshalling only: the controller pass runs in libgnmr.
"""
from __future__ import annotations

from collections import OrderedDict

import numpy as np

from .binding import GNMR_BF16, GNMR_BUDGET_ACTIVE, GNMR_F32, Controller

LLAMA_LINEARS = ("q_proj", "k_proj", "v_proj", "o_proj", "gate_proj", "up_proj", "down_proj")


def _current(stream):
    """`stream`, or torch's current stream when it is None: the stream that
    backward wrote the gradients on and that K4 and K5 are launched on, so a
    controller call is ordered after them also under `torch.cuda.stream(s)`."""
    if stream is not None:
        return stream
    import torch

    return torch.cuda.current_stream()


def llama_linear_units(name: str):
    """Default unit map for LLaMA-style models: each attention / SwiGLU
    projection weight is one recoverable unit (Sec. 2 operator view); other
    parameters are not monitored."""
    parts = name.split(".")
    if len(parts) >= 2 and parts[-1] == "weight" and parts[-2] in LLAMA_LINEARS:
        return ".".join(parts[:-1])
    return None


class TorchUnits:
    def __init__(self, named_parameters, window: int = 5, max_o: int = 8, lock_len: int = 8,
                 eps: float = 1e-12, unit_of=lambda name: name, recoverable=None,
                 budget_mode: int = GNMR_BUDGET_ACTIVE, warmup_steps: int = 0, stream=None):
        import torch

        groups = OrderedDict()
        for name, p in named_parameters:
            key = unit_of(name)
            if key is None or not p.requires_grad:
                continue
            if p.dtype not in (torch.bfloat16, torch.float32):
                raise TypeError(f"{name}: only bf16 and fp32 gradients are supported")
            groups.setdefault(key, []).append((name, p))
        if not groups:
            raise ValueError("no parameter was mapped to a unit")
        self.unit_names = list(groups.keys())
        self.params = [p for ps in groups.values() for _, p in ps]
        self.param_names = [n for ps in groups.values() for n, _ in ps]
        off = np.zeros(len(groups) + 1, dtype=np.int64)
        off[1:] = np.cumsum([len(ps) for ps in groups.values()])
        numel = [p.numel() for p in self.params]
        dtype = [GNMR_BF16 if p.dtype == torch.bfloat16 else GNMR_F32 for p in self.params]
        rec = None
        if recoverable is not None:
            rec = np.array([1 if recoverable(u) else 0 for u in self.unit_names], np.uint8)
        self.ctl = Controller(len(groups), window, max_o, lock_len, eps, off, numel, dtype,
                              None, rec, _current(stream), budget_mode, warmup_steps)

    def grad_pointers(self):
        ptrs = []
        for name, p in zip(self.param_names, self.params):
            g = p.grad
            if g is None:
                raise RuntimeError(f"{name}.grad is None; run backward before the controller step")
            if not g.is_contiguous() or g.dtype != p.dtype or g.device != p.device:
                raise RuntimeError(f"{name}.grad must be a contiguous {p.dtype} tensor on {p.device}")
            ptrs.append(g.data_ptr())
        return ptrs

    def step(self, alpha_t: float, beta_t: float, stream=None) -> None:
        """One controller step over the current gradients (asynchronous)."""
        self.ctl.step(alpha_t, beta_t, seg_ptr=self.grad_pointers(), stream=_current(stream))

    def query(self, stream=None) -> dict:
        out = self.ctl.query(_current(stream))
        out["units"] = self.unit_names
        return out

    def recovery_set(self, stream=None) -> list:
        """Names of the units on the recovery path after the last step (A_t)."""
        m = self.ctl.query(_current(stream))["mask"]
        return [u for u, a in zip(self.unit_names, m) if a]

    def close(self):
        self.ctl.close()


_FUNCTION = None


def _fused_linear_function():
    """The autograd function of a linear layer whose weight gradient comes
    from gnmr_wgrad_sumsq (built on first use, so that importing this module
    does not import torch)."""
    global _FUNCTION
    if _FUNCTION is None:
        import torch

        class FusedWgradLinear(torch.autograd.Function):
            @staticmethod
            def forward(ctx, x, weight, bias, units, index):
                spec = units._save_spec[index]
                # the activation kept for the weight gradient: the input
                # itself, or its per-token quantised copy (QuantizedSavedInputs)
                ctx.save_for_backward(x if spec is None else _quantize_rows(x, spec), weight)
                ctx.units, ctx.index = units, index
                ctx.has_bias = bias is not None
                # the same product as nn.Linear (bias fused: one rounding)
                return torch.nn.functional.linear(x, weight, bias)

            @staticmethod
            def backward(ctx, dy):
                x, weight = ctx.saved_tensors
                dx = torch.matmul(dy, weight) if ctx.needs_input_grad[0] else None
                if ctx.needs_input_grad[1]:
                    # K5 writes (or accumulates into) weight.grad itself, so
                    # autograd receives no weight gradient to accumulate
                    ctx.units._weight_grad(ctx.index, weight, dy, x)
                db = None
                if ctx.has_bias and ctx.needs_input_grad[2]:
                    db = dy.reshape(-1, dy.shape[-1]).sum(0)
                return dx, None, db, None, None

        _FUNCTION = FusedWgradLinear
    return _FUNCTION


def _quantize_rows(x, spec):
    """The per-token fake quantisation of x (K4, gnmr_actuate_matrix) as a
    new [tokens][features] bf16 tensor; spec = (device mask, unit, fmt_low,
    fmt_recovery).  The mask entry is read when the kernel runs."""
    import torch

    from .binding import gnmr_actuate_matrix

    d_mask, unit, fmt_low, fmt_recovery = spec
    if x.dtype != torch.bfloat16 or not x.is_cuda:
        # the kernel reads bf16 rows: any other element type would be misread
        raise TypeError(f"per-token quantisation needs a bf16 tensor on a HIP device, got "
                        f"{x.dtype} on {x.device}")
    cols = x.shape[-1]
    x2 = _kernel_operand(x, cols)
    out = torch.empty_like(x2)
    gnmr_actuate_matrix(x2, out, x2.shape[0], cols, d_mask, unit, fmt_low, fmt_recovery,
                        torch.cuda.current_stream())
    return out


def _kernel_operand(t, features: int):
    """t as a contiguous, 16-byte-aligned [tokens][features] bf16 matrix
    (a copy only when the view is neither)."""
    t = t.reshape(-1, features)
    if not t.is_contiguous():
        t = t.contiguous()
    if t.data_ptr() % 16:
        t = t.clone()
    return t


class FusedWgradUnits:
    """Bias-free or biased bf16 `torch.nn.Linear` layers as GNMR units whose
    norms come from the weight-gradient GEMM itself (K5, the sum of squares
    in its epilogue).  Each layer's forward is routed through an autograd
    function whose backward computes dx with torch and dW = dy^T x with
    gnmr_wgrad_sumsq_batched straight into `weight.grad`: into a new tensor
    when `weight.grad` is None, otherwise accumulated into the existing one
    (gradient accumulation over micro-batches, as torch would accumulate),
    and writes the layer's tile partials of the stored gradient.  `step()`
    then runs the controller from those partials (gnmr_step_from_partials),
    so the gradients are never re-read for their norms.  The forward is
    nn.Linear's (bias fused into the product); only the weight is the unit,
    and a bias gradient is the sum of dy over the tokens.

    The weight gradient does not pass through autograd's accumulation, so
    hooks registered on the weights' gradient accumulation do not run.
    `step()` raises if a layer did not run since the last step or if
    `weight.grad` was replaced since its backward.
    """

    def __init__(self, named_linears, window: int = 5, max_o: int = 8, lock_len: int = 8,
                 eps: float = 1e-12, recoverable=None, budget_mode: int = GNMR_BUDGET_ACTIVE,
                 warmup_steps: int = 0, stream=None):
        import torch

        from .binding import gnmr_wgrad_num_tiles

        self.unit_names, self.modules, self.shapes = [], [], []
        for name, m in named_linears:
            w = m.weight
            if w.dtype != torch.bfloat16 or not w.is_cuda:
                raise TypeError(f"{name}: the weight must be a bf16 tensor on a HIP device")
            o, i = w.shape
            if o % 8 or i % 8 or o >= 1 << 24 or i >= 1 << 24:
                raise ValueError(f"{name}: features must be multiples of 8 below 2^24, got {o}x{i}")
            self.unit_names.append(name)
            self.modules.append(m)
            self.shapes.append((o, i))
        if not self.modules:
            raise ValueError("no linear layer given")
        U = len(self.modules)
        tiles = [gnmr_wgrad_num_tiles(o, i) for o, i in self.shapes]
        self.part_off = np.zeros(U + 1, dtype=np.int64)
        self.part_off[1:] = np.cumsum(tiles)
        self.partials = torch.zeros(int(self.part_off[-1]), dtype=torch.float32,
                                    device=self.modules[0].weight.device)
        rec = None
        if recoverable is not None:
            rec = np.array([1 if recoverable(u) else 0 for u in self.unit_names], np.uint8)
        self.ctl = Controller(U, window, max_o, lock_len, eps, np.zeros(U + 1, np.int64), [], [],
                              None, rec, _current(stream), budget_mode, warmup_steps)
        self.ctl.bind_partials(self.part_off)
        self._produced = [None] * U   # data pointer of each layer's weight.grad
        self._save_spec = [None] * U  # per-token quantisation of the saved input, or None
        self._saved_forward = []
        for b, m in enumerate(self.modules):
            self._saved_forward.append(m.__dict__.get("forward"))
            m.forward = self._routed_forward(m, b)

    def _routed_forward(self, m, b):
        fn = _fused_linear_function()

        def forward(x):
            return fn.apply(x, m.weight, m.bias, self, b)
        return forward

    def _weight_grad(self, b, weight, dy, x):
        import torch

        from .binding import gnmr_wgrad_sumsq_batched

        o, i = self.shapes[b]
        if dy.dtype != torch.bfloat16 or x.dtype != torch.bfloat16:
            raise TypeError(f"{self.unit_names[b]}: activations and gradients must be bf16")
        dy2, x2 = _kernel_operand(dy, o), _kernel_operand(x, i)
        g = weight.grad
        if g is None:
            g = torch.empty((o, i), dtype=torch.bfloat16, device=dy.device)
            accumulate = 0
        else:
            if g.dtype != torch.bfloat16 or not g.is_contiguous() or g.data_ptr() % 16:
                raise RuntimeError(f"{self.unit_names[b]}: an existing weight.grad must be a "
                                   "contiguous, 16-byte-aligned bf16 tensor")
            accumulate = 1
        lo, hi = int(self.part_off[b]), int(self.part_off[b + 1])
        gnmr_wgrad_sumsq_batched([(dy2, x2, g, dy2.shape[0], o, i, accumulate)],
                                 self.partials[lo:hi], torch.cuda.current_stream())
        if accumulate == 0:
            weight.grad = g
        self._produced[b] = g.data_ptr()

    def step(self, alpha_t: float, beta_t: float, stream=None) -> None:
        """One controller step from this backward's tile partials (asynchronous)."""
        for b, m in enumerate(self.modules):
            g = m.weight.grad
            if self._produced[b] is None or g is None or g.data_ptr() != self._produced[b]:
                raise RuntimeError(
                    f"{self.unit_names[b]}: weight.grad is not the gradient the fused backward "
                    "wrote since the last step (the layer did not run, or .grad was replaced)")
        self.ctl.step_from_partials(self.partials, alpha_t, beta_t, _current(stream))
        self._produced = [None] * len(self.modules)

    def query(self, stream=None) -> dict:
        out = self.ctl.query(_current(stream))
        out["units"] = self.unit_names
        return out

    def recovery_set(self, stream=None) -> list:
        m = self.ctl.query(_current(stream))["mask"]
        return [u for u, a in zip(self.unit_names, m) if a]

    def close(self):
        for m, f in zip(self.modules, self._saved_forward):
            if f is None:
                m.__dict__.pop("forward", None)
            else:
                m.forward = f
        self._saved_forward = [None] * len(self.modules)
        self.ctl.close()


_QUANT = None


def _fake_quant_function():
    """The autograd function of the actuator on a layer input: forward is the
    per-token fake quantisation (gnmr_actuate_matrix), backward passes the
    gradient straight through to the unquantised input."""
    global _QUANT
    if _QUANT is None:
        import torch

        from .binding import gnmr_actuate_matrix

        class FakeQuantInput(torch.autograd.Function):
            @staticmethod
            def forward(ctx, x, d_mask, unit, fmt_low, fmt_recovery):
                cols = x.shape[-1]
                x2 = _kernel_operand(x, cols)
                out = torch.empty_like(x2)
                gnmr_actuate_matrix(x2, out, x2.shape[0], cols, d_mask, unit, fmt_low,
                                    fmt_recovery, torch.cuda.current_stream())
                return out.view(x.shape)

            @staticmethod
            def backward(ctx, g):
                return g, None, None, None, None

        _QUANT = FakeQuantInput
    return _QUANT


class QuantizedInputs:
    """The recovery actuator inside a forward pass: each listed layer's input
    is fake-quantised per token (K4, gnmr_actuate_matrix) before the layer
    runs, in fmt_recovery when the layer's unit is in A_t and in fmt_low
    otherwise (Alg. 2; App. E.2 quantisation-simulated operators; Sec. 5.1
    token-wise low-bit activations), so the layer computes with, and saves for
    its backward, the quantised activation.  The gradient reaches the
    unquantised input unchanged (straight through).

    `units` is a TorchUnits or FusedWgradUnits; a module is actuated when
    its name (as given in `named_modules`) is one of units.unit_names, and
    follows that unit's entry of the controller's device mask.  The mask is
    read when each kernel runs, so the formats follow the latest controller
    step in stream order, with no host synchronisation (before the first step
    every unit is on the low-cost path).  Inputs must be bf16 with a last
    dimension that is a multiple of 8 in [8, 16384].
    """

    def __init__(self, units, named_modules, fmt_low: int, fmt_recovery: int):
        index = {n: b for b, n in enumerate(units.unit_names)}
        self.units = units
        self.d_mask = units.ctl.device_outputs()["mask"]
        self.fmt_low, self.fmt_recovery = int(fmt_low), int(fmt_recovery)
        self.handles, self.names = [], []
        for name, m in named_modules:
            if name not in index:
                continue
            self.handles.append(m.register_forward_pre_hook(self._hook(name, index[name])))
            self.names.append(name)
        if not self.handles:
            raise ValueError("no module name matches a unit of the controller")

    def _hook(self, name, unit):
        import torch

        fn = _fake_quant_function()

        def hook(module, args):
            x = args[0]
            if x.dtype != torch.bfloat16 or not x.is_cuda:
                raise TypeError(f"{name}: the input must be a bf16 tensor on a HIP device")
            return (fn.apply(x, self.d_mask, unit, self.fmt_low, self.fmt_recovery),) + args[1:]
        return hook

    def close(self):
        for h in self.handles:
            h.remove()
        self.handles = []


_SAVED = None


def _saved_quant_linear_function():
    """The autograd function of a linear layer whose saved input is the
    per-token quantised copy: the forward product uses the input itself, the
    weight gradient the quantised copy."""
    global _SAVED
    if _SAVED is None:
        import torch

        class QuantSavedLinear(torch.autograd.Function):
            @staticmethod
            def forward(ctx, x, weight, bias, spec):
                ctx.save_for_backward(_quantize_rows(x, spec), weight)
                ctx.has_bias = bias is not None
                # the same product as nn.Linear, on the unquantised input
                return torch.nn.functional.linear(x, weight, bias)

            @staticmethod
            def backward(ctx, dy):
                xq, weight = ctx.saved_tensors
                dy2 = dy.reshape(-1, dy.shape[-1])
                dx = torch.matmul(dy, weight) if ctx.needs_input_grad[0] else None
                # dW = dy^T x_q, as nn.Linear's backward forms dy^T x
                dw = dy2.t().mm(xq) if ctx.needs_input_grad[1] else None
                db = dy2.sum(0) if ctx.has_bias and ctx.needs_input_grad[2] else None
                return dx, dw, db, None

        _SAVED = QuantSavedLinear
    return _SAVED


class QuantizedSavedInputs:
    """The recovery actuator on saved activations only: the low-cost path of
    the activation-quantisation stress bench (Sec. 5.1; App. E.2, recoverable
    scope; App. E.4) quantises the activation a linear layer keeps for its
    backward, not the input of its forward product.  Each listed layer
    computes its output from its bf16 input unchanged; the copy it saves for
    the weight gradient is fake-quantised per token (K4,
    gnmr_actuate_matrix), in fmt_recovery when the layer's unit is in A_t and
    in fmt_low otherwise, so dW = dy^T x_q while dx = dy W is exact in the
    input.

    `units` is a TorchUnits or a FusedWgradUnits; a module is actuated when
    its name (as given in `named_modules`) is one of units.unit_names, and
    follows that unit's entry of the controller's device mask, read when each
    kernel runs (in stream order, no host synchronisation; before the first
    step every unit is on the low-cost path).  With a FusedWgradUnits the
    weight gradient and its tile sums come from K5 over the quantised copy;
    otherwise the module's forward is routed through an autograd function
    whose weight gradient is torch's product with the quantised copy.  The
    modules must be bf16 nn.Linear layers whose input's last dimension is a
    multiple of 8 in [8, 16384].  QuantizedInputs is the other reading: it
    quantises the forward input itself.
    """

    def __init__(self, units, named_modules, fmt_low: int, fmt_recovery: int):
        import torch

        index = {n: b for b, n in enumerate(units.unit_names)}
        self.units = units
        self.d_mask = units.ctl.device_outputs()["mask"]
        self.fmt_low, self.fmt_recovery = int(fmt_low), int(fmt_recovery)
        self.fused = isinstance(units, FusedWgradUnits)
        self.names, self._routed = [], []
        for name, m in named_modules:
            if name not in index:
                continue
            if m.weight.dtype != torch.bfloat16 or not m.weight.is_cuda:
                raise TypeError(f"{name}: the weight must be a bf16 tensor on a HIP device")
            spec = (self.d_mask, index[name], self.fmt_low, self.fmt_recovery)
            if self.fused:
                units._save_spec[index[name]] = spec
            else:
                self._routed.append((m, m.__dict__.get("forward")))
                m.forward = self._routed_forward(m, spec)
            self.names.append(name)
        if not self.names:
            raise ValueError("no module name matches a unit of the controller")

    @staticmethod
    def _routed_forward(m, spec):
        fn = _saved_quant_linear_function()

        def forward(x):
            return fn.apply(x, m.weight, m.bias, spec)
        return forward

    def close(self):
        if self.fused:
            for name in self.names:
                self.units._save_spec[self.units.unit_names.index(name)] = None
        for m, f in self._routed:
            if f is None:
                m.__dict__.pop("forward", None)
            else:
                m.forward = f
        self._routed, self.names = [], []


_QSIM = None


def _qsim_linear_function():
    """The autograd function of the quantisation-simulated linear operator."""
    global _QSIM
    if _QSIM is None:
        import torch

        class QuantSimLinear(torch.autograd.Function):
            @staticmethod
            def forward(ctx, x, weight, spec, capture):
                d_mask, unit, f_lo, b_lo, f_hi, b_hi = spec
                fwd = (d_mask, unit, f_lo, f_hi)
                x_q = _quantize_rows(x, fwd)                         # per token
                w_q = _quantize_rows(weight, fwd)                    # per output channel
                y = torch.nn.functional.linear(x_q, w_q)
                y_q = _quantize_rows(y, fwd)                         # per token
                ctx.save_for_backward(x_q, w_q)
                ctx.spec, ctx.capture, ctx.x_shape = spec, capture, x.shape
                if capture is not None:
                    capture.update(x_q=x_q, w_q=w_q, y=y, y_q=y_q)
                return y_q.view(*x.shape[:-1], weight.shape[0])

            @staticmethod
            def backward(ctx, dy):
                x_q, w_q = ctx.saved_tensors
                d_mask, unit, f_lo, b_lo, f_hi, b_hi = ctx.spec
                bwd = (d_mask, unit, b_lo, b_hi)
                dy_q = _quantize_rows(dy, bwd)                       # per token
                dx_q = dw_q = None
                if ctx.needs_input_grad[0]:
                    dx = torch.matmul(dy_q, w_q)
                    dx_q = _quantize_rows(dx, bwd).view(ctx.x_shape)
                if ctx.needs_input_grad[1]:
                    dw = dy_q.t().mm(x_q)
                    dw_q = _quantize_rows(dw, bwd)                   # per output channel
                if ctx.capture is not None:
                    ctx.capture.update(dy=dy.reshape(-1, dy.shape[-1]).clone(), dy_q=dy_q,
                                       dx_q=dx_q, dw_q=dw_q)
                return dx_q, dw_q, None, None

        _QSIM = QuantSimLinear
    return _QSIM


class QuantSimLinears:
    """The quantisation-simulated low-precision linear operator of App. E.2
    on bias-free bf16 `nn.Linear` layers, its formats switched per unit by
    the controller: forward, the input x and the weight w are fake-quantised
    before the product and the output y again; backward, the incoming
    gradient dy is quantised, and the computed dx and dw are quantised before
    they go on (dx to the previous layer, dw to the optimiser and the
    controller).  Every quantisation is K4's per-row recipe
    (gnmr_actuate_matrix): rows are tokens for x, y, dy and dx and output
    channels for w and dw.  The products are library GEMMs on the quantised
    bf16 tensors (fp32 accumulation).

    `low` and `recovery` are (forward format, backward format) pairs: a unit
    outside A_t uses `low` (the paper's 4-bit E2M1 or 6-bit E3M2), a unit in
    A_t `recovery` (the paper's hybrid FP8: E4M3 forward, E5M2 backward).  The
    controller's device mask is read when each kernel runs, so a training
    step's forward and backward use the decision of the last controller step
    in stream order.  `units` is a TorchUnits whose units include the listed
    modules' weights (their .grad is the quantised dw); modules are matched
    by name against units.unit_names.  With capture=True the tensors of each
    module's last forward and backward are kept in self.captured[name].
    """

    def __init__(self, units, named_modules, low=(1, 1), recovery=(3, 4), capture=False):
        import torch

        if isinstance(units, FusedWgradUnits):
            raise TypeError("the weight gradient is quantised after its product: use "
                            "TorchUnits, whose gradient pass reads the quantised .grad")
        index = {n: b for b, n in enumerate(units.unit_names)}
        self.units = units
        self.d_mask = units.ctl.device_outputs()["mask"]
        self.low, self.recovery = tuple(int(f) for f in low), tuple(int(f) for f in recovery)
        self.captured = {} if capture else None
        self.names, self._routed = [], []
        for name, m in named_modules:
            if name not in index:
                continue
            if m.weight.dtype != torch.bfloat16 or not m.weight.is_cuda:
                raise TypeError(f"{name}: the weight must be a bf16 tensor on a HIP device")
            if getattr(m, "bias", None) is not None:
                raise TypeError(f"{name}: the simulated operator is bias-free")
            spec = (self.d_mask, index[name], self.low[0], self.low[1], self.recovery[0],
                    self.recovery[1])
            cap = None
            if capture:
                cap = self.captured.setdefault(name, {})
            self._routed.append((m, m.__dict__.get("forward")))
            m.forward = self._routed_forward(m, spec, cap)
            self.names.append(name)
        if not self.names:
            raise ValueError("no module name matches a unit of the controller")

    @staticmethod
    def _routed_forward(m, spec, cap):
        fn = _qsim_linear_function()

        def forward(x):
            return fn.apply(x, m.weight, spec, cap)
        return forward

    def close(self):
        for m, f in self._routed:
            if f is None:
                m.__dict__.pop("forward", None)
            else:
                m.forward = f
        self._routed, self.names = [], []
