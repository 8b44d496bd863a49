"""Guarded dispatch of PyTorch operator calls to libkf355.

Kernel Forge exports its kernels as guarded packages: a generated kernel
replaces a PyTorch call only when it is available, compatible with the call,
numerically valid on the recorded inputs and faster than PyTorch eager for
that variant; otherwise the original eager path runs, and every variant is
labelled with the path it took (Section III-E, "Packaging, Guarded Dispatch,
and Audit Labels"; variants are concrete call patterns, not operator names,
Section III-A).  This module applies that policy to libkf355:

* `GuardedDispatcher.call` keys each call by its variant (operator, shapes,
  dtypes, strides, device, scalar arguments).  The first call of a variant
  runs both paths on the live input, compares them with the tolerance
  configured for the output dtype (Section III-C), times both with HIP events,
  and records a `Decision` with its audit label; later calls of the variant
  take the recorded path.
* `install()` / `uninstall()` (or the `installed()` context manager) route
  `torch.softmax`, `torch.Tensor.softmax`, `F.softmax`, `F.layer_norm`,
  `F.group_norm`, `F.adaptive_avg_pool2d` and `F.max_pool2d` through a
  dispatcher for CUDA
  tensors in inference (no autograd); anything else goes straight to the
  original function.
* `save()` / `load()` write and read the decisions as JSON, the package a
  deployment reuses without re-measuring.

The eager fallback here is the policy itself: it happens per variant, for a
recorded reason, and is visible in `report()`.  The library is still
required: `install()` raises if libkf355.so is missing.
"""
from __future__ import annotations

import contextlib
import dataclasses
import json
import threading

import torch
import torch.nn.functional as F

from . import kf355

# Output-dtype tolerances for the kf355-vs-eager validity check, as
# (rtol, scale_tol): an element agrees when |kf - eager| <= rtol * |eager| +
# scale_tol * max|eager|.  Both sides approximate the same definition, and the
# eager side is not always the closer one: eager GroupNorm in bf16 on ROCm
# forms its output from a bf16-rounded product and shift, so near zero it is
# off by about 2^-10 of the output's scale (hundreds of bf16 ulps of the
# element), while the library stays within half an ulp of the exact result.
# The scale term admits that error; a real fault (a wrong row, a missing
# term) is orders of magnitude larger.
TOLERANCES = {
    torch.float32: (1e-5, 1e-6),
    torch.bfloat16: (2 ** -6, 2 ** -7),
    torch.float16: (2 ** -9, 2 ** -10),
}
UNSUPPORTED = {2, 3, 4, 5}  # bad shape / dtype / argument / layout for the library


@dataclasses.dataclass
class Decision:
    op: str
    variant: str
    backend: str            # "kf355" or "eager"
    reason: str
    kf_us: float | None = None
    eager_us: float | None = None
    max_abs_diff: float | None = None
    kernel: str | None = None

    def label(self) -> str:
        return f"{self.backend} ({self.reason})"


def agree(y_kf, y_ref) -> tuple[bool, float]:
    """(every element within TOLERANCES of the eager result, max |difference|).
    NaN must sit at the same positions on both sides; infinities must match.
    Integer outputs (pooling indices) must be equal; tuples agree element by
    element."""
    if isinstance(y_ref, (tuple, list)):
        if not isinstance(y_kf, (tuple, list)) or len(y_kf) != len(y_ref):
            return False, float("inf")
        results = [agree(a, b) for a, b in zip(y_kf, y_ref)]
        return all(ok for ok, _ in results), max((d for _, d in results), default=0.0)
    if y_kf.shape != y_ref.shape or y_kf.dtype != y_ref.dtype:
        return False, float("inf")
    if y_ref.numel() == 0:
        return True, 0.0
    if not y_ref.dtype.is_floating_point:
        return bool(torch.equal(y_kf, y_ref)), float((y_kf.double() - y_ref.double()).abs().max().item())
    rtol, stol = TOLERANCES.get(y_ref.dtype, (1e-5, 1e-6))
    a, b = y_kf.double(), y_ref.double()
    nan_a, nan_b = torch.isnan(a), torch.isnan(b)
    if not torch.equal(nan_a, nan_b):
        return False, float("nan")
    fin = torch.isfinite(b)
    if not torch.equal(a[~fin & ~nan_b], b[~fin & ~nan_b]):
        return False, float("inf")
    a, b = a[fin], b[fin]
    if b.numel() == 0:
        return True, 0.0
    err = (a - b).abs()
    lim = rtol * b.abs() + stol * float(b.abs().max().item())
    return bool((err <= lim).all().item()), float(err.max().item())


def _describe(v) -> str:
    if isinstance(v, torch.Tensor):
        return f"T{tuple(v.shape)}:{str(v.dtype).replace('torch.', '')}:{tuple(v.stride())}:{v.device}"
    return repr(v)


def variant_key(op: str, args: tuple) -> str:
    return op + "(" + ", ".join(_describe(a) for a in args) + ")"


def _time_us(fn, reps: int) -> float:
    for _ in range(2):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


class GuardedDispatcher:
    """Per-variant choice between a libkf355 call and PyTorch eager."""

    def __init__(self, reps: int = 10, validate: bool = True, measure: bool = True, timer=None):
        self.reps = reps
        self.validate = validate
        self.measure = measure
        self.timer = timer or _time_us   # (fn, reps) -> microseconds per call
        self.decisions: dict[str, Decision] = {}
        self._lock = threading.RLock()

    def call(self, op: str, key_args: tuple, kf_fn, eager_fn):
        key = variant_key(op, key_args)
        d = self.decisions.get(key)
        if d is None:
            with self._lock:
                d = self.decisions.get(key)
                if d is None:
                    d, y = self._decide(op, key, kf_fn, eager_fn)
                    self.decisions[key] = d
                    return y
        return kf_fn() if d.backend == "kf355" else eager_fn()

    def _decide(self, op, key, kf_fn, eager_fn):
        """Returns the decision and the output of the chosen path for the
        call that triggered it (both paths were evaluated on its input)."""
        try:
            y_kf = kf_fn()
        except kf355.KfError as e:
            if e.status in UNSUPPORTED:
                return Decision(op, key, "eager", f"unsupported: {e}"), eager_fn()
            raise
        d, y_ref = self._judge(op, key, kf_fn, eager_fn, y_kf)
        return d, (y_kf if d.backend == "kf355" else y_ref)

    def _judge(self, op, key, kf_fn, eager_fn, y_kf):
        kernel = kf355.last_variant()
        y_ref = eager_fn()
        diff = None
        if self.validate:
            ok, diff = agree(y_kf, y_ref)
            if not ok:
                return Decision(op, key, "eager", f"invalid: max |kf355 - eager| = {diff:.3g}",
                                max_abs_diff=diff, kernel=kernel), y_ref
        if not self.measure:
            return Decision(op, key, "kf355", "valid (not timed)", max_abs_diff=diff, kernel=kernel), y_ref
        kf_us = self.timer(kf_fn, self.reps)
        eager_us = self.timer(eager_fn, self.reps)
        if kf_us < eager_us:
            return Decision(op, key, "kf355", f"faster: {kf_us:.1f} us vs eager {eager_us:.1f} us", kf_us,
                            eager_us, diff, kernel), y_ref
        return Decision(op, key, "eager", f"slower: {kf_us:.1f} us vs eager {eager_us:.1f} us", kf_us, eager_us,
                        diff, kernel), y_ref

    # -- audit and packaging ---------------------------------------------
    def report(self) -> list[dict]:
        return [dataclasses.asdict(d) | {"label": d.label()} for d in self.decisions.values()]

    def save(self, path: str):
        with open(path, "w") as f:
            json.dump([dataclasses.asdict(d) for d in self.decisions.values()], f, indent=1)

    def load(self, path: str):
        with open(path) as f:
            for d in json.load(f):
                self.decisions[d["variant"]] = Decision(**d)


# --------------------------------------------------------------------------
# Routing of the PyTorch entry points.

_ORIG: dict = {}
_ACTIVE: GuardedDispatcher | None = None


def _eligible(x) -> bool:
    return isinstance(x, torch.Tensor) and x.is_cuda and not (torch.is_grad_enabled() and x.requires_grad)


def _softmax(x, dim=None, dtype=None, orig=None):
    if dim is None or not _eligible(x) or (dtype is not None and dtype != torch.float32):
        return orig(x, dim, dtype=dtype) if dtype is not None else orig(x, dim)
    out_dtype = dtype or x.dtype
    return _ACTIVE.call("softmax", (x, dim, out_dtype),
                        lambda: kf355.kf_softmax_split(x, dim, out_dtype=out_dtype),
                        lambda: orig(x, dim, dtype=dtype) if dtype is not None else orig(x, dim))


def _torch_softmax(input, dim, dtype=None):
    return _softmax(input, dim, dtype, _ORIG["torch.softmax"])


def _tensor_softmax(self, dim, dtype=None):
    return _softmax(self, dim, dtype, _ORIG["Tensor.softmax"])


def _f_softmax(input, dim=None, _stacklevel=3, dtype=None):
    if dim is None:   # implicit-dim legacy form: the original picks dim and calls Tensor.softmax
        return _ORIG["F.softmax"](input, dim, _stacklevel, dtype)
    # The eager leg calls the C method directly: F.softmax itself goes through
    # Tensor.softmax, which is routed here too and would re-enter the dispatcher.
    return _softmax(input, dim, dtype, _ORIG["Tensor.softmax"])


def _f_layer_norm(input, normalized_shape, weight=None, bias=None, eps=1e-5):
    orig = _ORIG["F.layer_norm"]
    if not _eligible(input):
        return orig(input, normalized_shape, weight, bias, eps)
    ns = tuple(normalized_shape) if not isinstance(normalized_shape, int) else (normalized_shape,)
    return _ACTIVE.call("layer_norm", (input, ns, weight, bias, eps),
                        lambda: kf355.kf_layer_norm(input, ns, weight, bias, eps),
                        lambda: orig(input, normalized_shape, weight, bias, eps))


def _f_group_norm(input, num_groups, weight=None, bias=None, eps=1e-5):
    orig = _ORIG["F.group_norm"]
    if not _eligible(input):
        return orig(input, num_groups, weight, bias, eps)
    return _ACTIVE.call("group_norm", (input, num_groups, weight, bias, eps),
                        lambda: kf355.kf_group_norm(input, num_groups, weight, bias, eps),
                        lambda: orig(input, num_groups, weight, bias, eps))


def _f_adaptive_avg_pool2d(input, output_size):
    orig = _ORIG["F.adaptive_avg_pool2d"]
    if not _eligible(input) or input.dim() not in (3, 4):
        return orig(input, output_size)
    size = (output_size, output_size) if isinstance(output_size, int) else tuple(output_size)
    if any(s is None for s in size):
        return orig(input, output_size)
    return _ACTIVE.call("adaptive_avg_pool2d", (input, size),
                        lambda: kf355.kf_adaptive_avgpool2d(input, size),
                        lambda: orig(input, output_size))


def _f_max_pool2d(input, kernel_size, stride=None, padding=0, dilation=1, ceil_mode=False, return_indices=False):
    orig = _ORIG["F.max_pool2d"]
    args = (input, kernel_size, stride, padding, dilation)
    if not _eligible(input) or input.dim() not in (3, 4):
        return orig(*args, ceil_mode=ceil_mode, return_indices=return_indices)
    norm = lambda v: tuple(v) if isinstance(v, (tuple, list)) else v  # noqa: E731
    st = None if stride is None or (isinstance(stride, (tuple, list)) and len(stride) == 0) else norm(stride)
    return _ACTIVE.call("max_pool2d", (input, norm(kernel_size), st, norm(padding), norm(dilation), bool(ceil_mode),
                                       bool(return_indices)),
                        lambda: kf355.kf_max_pool2d(input, kernel_size, st, padding, dilation, ceil_mode,
                                                    return_indices),
                        lambda: orig(*args, ceil_mode=ceil_mode, return_indices=return_indices))


def install(dispatcher: GuardedDispatcher | None = None) -> GuardedDispatcher:
    """Route the supported PyTorch operators through `dispatcher` (a new one
    by default).  Raises if libkf355 is not built."""
    global _ACTIVE
    kf355.lib()
    if _ORIG:
        raise RuntimeError("libkf355 dispatch is already installed")
    _ACTIVE = dispatcher or GuardedDispatcher()
    _ORIG.update({"torch.softmax": torch.softmax, "Tensor.softmax": torch.Tensor.softmax,
                  "F.softmax": F.softmax, "F.layer_norm": F.layer_norm, "F.group_norm": F.group_norm,
                  "F.adaptive_avg_pool2d": F.adaptive_avg_pool2d, "F.max_pool2d": F.max_pool2d})
    torch.softmax = _torch_softmax
    torch.Tensor.softmax = _tensor_softmax
    F.softmax = _f_softmax
    F.layer_norm = _f_layer_norm
    F.group_norm = _f_group_norm
    F.adaptive_avg_pool2d = _f_adaptive_avg_pool2d
    F.max_pool2d = _f_max_pool2d
    return _ACTIVE


def uninstall():
    global _ACTIVE
    if not _ORIG:
        return
    torch.softmax = _ORIG["torch.softmax"]
    torch.Tensor.softmax = _ORIG["Tensor.softmax"]
    F.softmax = _ORIG["F.softmax"]
    F.layer_norm = _ORIG["F.layer_norm"]
    F.group_norm = _ORIG["F.group_norm"]
    F.adaptive_avg_pool2d = _ORIG["F.adaptive_avg_pool2d"]
    F.max_pool2d = _ORIG["F.max_pool2d"]
    _ORIG.clear()
    _ACTIVE = None


@contextlib.contextmanager
def installed(dispatcher: GuardedDispatcher | None = None):
    d = install(dispatcher)
    try:
        yield d
    finally:
        uninstall()
