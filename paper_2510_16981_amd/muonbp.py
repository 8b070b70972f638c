"""ctypes binding of ``libmuonbp.so`` (C ABI in ``include/muonbp.h``).

Argument marshalling only: every step of the optimizer runs in the HIP
library.  torch supplies device memory (``data_ptr``) and the current HIP
stream.  There is no fallback: if the library is missing, loading raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmuonbp.so")

F32, BF16 = 0, 1
KERNEL_KINDS = ("momentum", "scale", "pack", "gram", "poly", "apply", "update", "ns_span")
NS_KINDS = ("gram", "poly", "apply")

STATUS = {0: "MUONBP_OK", 1: "MUONBP_E_INVALID", 2: "MUONBP_E_SHAPE",
          3: "MUONBP_E_DTYPE", 4: "MUONBP_E_NOMEM", 5: "MUONBP_E_HIP",
          6: "MUONBP_E_STATE", 7: "MUONBP_E_NONFINITE", 8: "MUONBP_E_TOO_LARGE"}
STATIC_SCRATCH_BYTES = 128 << 20


class MuonBPError(RuntimeError):
    def __init__(self, status: int, detail: str = ""):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {detail}")


class Matrix(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("grid_rows", ctypes.c_int32), ("grid_cols", ctypes.c_int32)]


class Options(ctypes.Structure):
    _fields_ = [("ns_steps", ctypes.c_int32), ("a", ctypes.c_float),
                ("b", ctypes.c_float), ("c", ctypes.c_float),
                ("eps", ctypes.c_float), ("nesterov", ctypes.c_int32),
                ("scale_mode", ctypes.c_int32), ("rms_beta", ctypes.c_float),
                ("param_dtype", ctypes.c_int), ("state_dtype", ctypes.c_int),
                ("ns_dtype", ctypes.c_int), ("tile_policy", ctypes.c_int32),
                ("k_split", ctypes.c_int32), ("coeff_count", ctypes.c_int32),
                ("coeff_table", ctypes.c_float * (3 * 16)), ("stream_hint", ctypes.c_int32),
                ("apply_mode", ctypes.c_int32), ("check_finite", ctypes.c_int32),
                ("device_memory_limit", ctypes.c_int64), ("gram_iteration", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("n_problems", ctypes.c_int64), ("n_elements", ctypes.c_int64),
                ("gemm_tiles", ctypes.c_int64 * 3), ("gemm_tile_rows", ctypes.c_int32 * 3),
                ("gemm_tile_cols", ctypes.c_int32 * 3), ("gemm_launches", ctypes.c_int64),
                ("ns_flops", ctypes.c_double),
                ("ns_dense_flops", ctypes.c_double),
                ("elementwise_bytes", ctypes.c_double),
                ("workspace_bytes", ctypes.c_int64),
                ("gemm_split", ctypes.c_int32 * 3), ("apply_nn", ctypes.c_int32),
                ("static_scratch_bytes", ctypes.c_int64), ("device_bytes", ctypes.c_int64),
                ("gram_units", ctypes.c_int64), ("pack_elements", ctypes.c_int64)]


class AdamwOptions(ctypes.Structure):
    _fields_ = [("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("max_grad_norm", ctypes.c_float),
                ("param_dtype", ctypes.c_int), ("stream_hint", ctypes.c_int32),
                ("algorithm", ctypes.c_int32)]


class Profile(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 8), ("launches", ctypes.c_int64 * 8),
                ("ms_full_steps", ctypes.c_double * 8),
                ("launches_full_steps", ctypes.c_int64 * 8)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises when it has not been built).

    torch is imported first: its wheel ships its own HIP runtime under the
    same soname as the system one, and the library must bind to the runtime
    that owns torch's memory and streams (loaded the other way round, the
    process would end up with two runtimes)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2510_16981_amd.build`")
    import torch  # noqa: F401  (see above)
    lib = ctypes.CDLL(path)
    P, I32, I64, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    sig = {
        "muonbp_options_default": (None, [ctypes.POINTER(Options)]),
        "muonbp_create": (ctypes.c_int, [ctypes.POINTER(Matrix), I32, I64, F, F, F, F,
                                         ctypes.POINTER(Options), P, ctypes.POINTER(P)]),
        "muonbp_step": (ctypes.c_int, [P, ctypes.POINTER(P), ctypes.POINTER(P), I64]),
        "muonbp_set_lr": (ctypes.c_int, [P, F, F]),
        "muonbp_set_period": (ctypes.c_int, [P, I64]),
        "muonbp_set_stream": (ctypes.c_int, [P, P]),
        "muonbp_get_momentum": (ctypes.c_int, [P, I32, P]),
        "muonbp_set_momentum": (ctypes.c_int, [P, I32, P]),
        "muonbp_get_update": (ctypes.c_int, [P, I32, P]),
        "muonbp_synchronize": (ctypes.c_int, [P]),
        "muonbp_describe_plan": (ctypes.c_int, [ctypes.POINTER(Matrix), I32,
                                                ctypes.POINTER(Options), I32,
                                                ctypes.POINTER(PlanInfo)]),
        "muonbp_profile_enable": (ctypes.c_int, [P, I32]),
        "muonbp_profile_read": (ctypes.c_int, [P, ctypes.POINTER(Profile)]),
        "muonbp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "muonbp_last_error": (ctypes.c_char_p, [P]),
        "muonbp_destroy": (None, [P]),
        "muonbp_adamw_options_default": (None, [ctypes.POINTER(AdamwOptions)]),
        "muonbp_adamw_create": (ctypes.c_int, [ctypes.POINTER(I64), I32, ctypes.POINTER(AdamwOptions),
                                               P, ctypes.POINTER(P)]),
        "muonbp_adamw_step": (ctypes.c_int, [P, ctypes.POINTER(P), ctypes.POINTER(P), I64, F]),
        "muonbp_adamw_grad_norm": (ctypes.c_int, [P, ctypes.POINTER(F)]),
        "muonbp_adamw_get_state": (ctypes.c_int, [P, I32, P, P]),
        "muonbp_adamw_set_state": (ctypes.c_int, [P, I32, P, P]),
        "muonbp_adamw_set_stream": (ctypes.c_int, [P, P]),
        "muonbp_adamw_synchronize": (ctypes.c_int, [P]),
        "muonbp_adamw_last_error": (ctypes.c_char_p, [P]),
        "muonbp_adamw_destroy": (None, [P]),
        "muonbp_step_static": (ctypes.c_int, [ctypes.POINTER(Matrix), I32, ctypes.POINTER(P),
                                              ctypes.POINTER(P), P, I64, I64, F, F, F, F,
                                              ctypes.POINTER(Options), P]),
        "muonbp_lr_cosine": (ctypes.c_double, [I64, I64, ctypes.c_double, ctypes.c_double, I64]),
        "muonbp_lr_wsd": (ctypes.c_double, [I64, I64, ctypes.c_double, ctypes.c_double, I64, I64]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


MAX_COEFFS = 16


def options_default(**overrides) -> Options:
    """Library defaults with fields overridden by keyword; ``coeffs`` (a list
    of (a, b, c) triples, one per NS iteration, the last repeated) fills
    coeff_count and coeff_table."""
    o = Options()
    load_library().muonbp_options_default(ctypes.byref(o))
    table = overrides.pop("coeffs", None)
    for k, v in overrides.items():
        if not hasattr(o, k):
            raise AttributeError(k)
        setattr(o, k, v)
    if table is not None:
        if not 1 <= len(table) <= MAX_COEFFS:
            raise ValueError(f"1..{MAX_COEFFS} coefficient triples")
        o.coeff_count = len(table)
        for i, (a, b, c) in enumerate(table):
            o.coeff_table[3 * i:3 * i + 3] = (float(a), float(b), float(c))
    return o


def _mats(mats: Sequence[Tuple[int, int, int, int]]):
    arr = (Matrix * len(mats))()
    for i, (r, c, gr, gc) in enumerate(mats):
        arr[i] = Matrix(r, c, gr, gc)
    return arr


def describe_plan(mats, full: bool, options: Optional[Options] = None) -> PlanInfo:
    """Host-only description of the block (full=False) or full plan."""
    lib = load_library()
    info = PlanInfo()
    st = lib.muonbp_describe_plan(_mats(mats), len(mats),
                                  ctypes.byref(options) if options else None,
                                  int(bool(full)), ctypes.byref(info))
    if st:
        raise MuonBPError(st, "describe_plan")
    return info


def step_static(mats, params: List, grads: List, momentum, step: int, period: int,
                lr_block: float, lr_full: float, mu: float, weight_decay: float = 0.0,
                options: Optional[Options] = None, stream=None) -> None:
    """One allocation-free step (muonbp_step_static): the momentum is the
    caller's ``momentum`` tensor (all matrices back to back, state dtype),
    everything else lives in the library's static scratch array.  Returns
    after the step has completed on ``stream``."""
    import torch
    lib = load_library()
    mats = [tuple(int(v) for v in m) for m in mats]
    n = len(mats)
    if len(params) != n or len(grads) != n:
        raise ValueError("one param and one grad per matrix")
    opts = options if options is not None else options_default()
    total = sum(r * c for r, c, _, _ in mats)
    if not (momentum.is_cuda and momentum.is_contiguous() and momentum.numel() == total
            and momentum.dtype == _torch_dtype(opts.state_dtype)):
        raise ValueError(f"momentum: need a contiguous {_torch_dtype(opts.state_dtype)} CUDA "
                         f"tensor of {total} elements")
    for i, (r, c, _, _) in enumerate(mats):
        for t in (params[i], grads[i]):
            if not (t.is_cuda and t.is_contiguous() and t.dtype == _torch_dtype(opts.param_dtype)
                    and tuple(t.shape) == (r, c)):
                raise ValueError(f"matrix {i}: need contiguous {_torch_dtype(opts.param_dtype)} "
                                 f"CUDA tensors of shape {(r, c)}")
    if stream is None:
        stream = torch.cuda.current_stream()
    pp = (ctypes.c_void_p * n)(*[p.data_ptr() for p in params])
    gp = (ctypes.c_void_p * n)(*[g.data_ptr() for g in grads])
    st = lib.muonbp_step_static(_mats(mats), n, pp, gp, ctypes.c_void_p(momentum.data_ptr()),
                                int(step), int(period), float(lr_block), float(lr_full), float(mu),
                                float(weight_decay), ctypes.byref(opts),
                                ctypes.c_void_p(stream.cuda_stream))
    if st:
        raise MuonBPError(st, "muonbp_step_static")


def _torch_dtype(code: int):
    import torch
    return {F32: torch.float32, BF16: torch.bfloat16}[code]


class MuonBP:
    """One optimizer context over a fixed list of matrices (Algorithm 1)."""

    def __init__(self, mats: Sequence[Tuple[int, int, int, int]], period: int,
                 lr_block: float, lr_full: float, momentum: float,
                 weight_decay: float = 0.0, options: Optional[Options] = None,
                 stream=None):
        import torch
        self.lib = load_library()
        self.mats = [tuple(int(v) for v in m) for m in mats]
        self.options = options if options is not None else options_default()
        if stream is None:
            stream = torch.cuda.current_stream()
        self._stream = stream
        ctx = ctypes.c_void_p()
        st = self.lib.muonbp_create(_mats(self.mats), len(self.mats), int(period),
                                    float(lr_block), float(lr_full), float(momentum),
                                    float(weight_decay), ctypes.byref(self.options),
                                    ctypes.c_void_p(stream.cuda_stream), ctypes.byref(ctx))
        if st:
            raise MuonBPError(st, "muonbp_create")
        self.ctx = ctx
        self.period = int(period)
        self._ptrs = (ctypes.c_void_p * len(self.mats))()
        self._gptrs = (ctypes.c_void_p * len(self.mats))()

    # -- helpers
    def _check(self, st: int, what: str):
        if st:
            detail = self.lib.muonbp_last_error(self.ctx)
            raise MuonBPError(st, f"{what}: {detail.decode() if detail else ''}")

    def _check_tensor(self, t, i, dtype_code):
        import torch
        r, c = self.mats[i][:2]
        if not (t.is_cuda and t.is_contiguous() and t.dtype == _torch_dtype(dtype_code)
                and tuple(t.shape) == (r, c)):
            raise ValueError(f"matrix {i}: need a contiguous {_torch_dtype(dtype_code)} "
                             f"CUDA tensor of shape {(r, c)}, got {t.dtype} {tuple(t.shape)}")

    def is_full(self, t: int) -> bool:
        return self.period > 0 and t % self.period == 0

    # -- API
    def step(self, params: List, grads: List, t: int) -> None:
        n = len(self.mats)
        if len(params) != n or len(grads) != n:
            raise ValueError("one param and one grad per matrix")
        for i in range(n):
            self._check_tensor(params[i], i, self.options.param_dtype)
            self._check_tensor(grads[i], i, self.options.param_dtype)
            self._ptrs[i] = params[i].data_ptr()
            self._gptrs[i] = grads[i].data_ptr()
        self._check(self.lib.muonbp_step(self.ctx, self._ptrs, self._gptrs, int(t)), "step")

    def set_lr(self, lr_block: float, lr_full: float) -> None:
        self._check(self.lib.muonbp_set_lr(self.ctx, float(lr_block), float(lr_full)), "set_lr")

    def set_period(self, period: int) -> None:
        self._check(self.lib.muonbp_set_period(self.ctx, int(period)), "set_period")
        self.period = int(period)

    def set_stream(self, stream) -> None:
        self._check(self.lib.muonbp_set_stream(self.ctx, ctypes.c_void_p(stream.cuda_stream)),
                    "set_stream")
        self._stream = stream

    def get_momentum(self, i: int, out=None):
        import torch
        r, c = self.mats[i][:2]
        if out is None:
            out = torch.empty((r, c), dtype=_torch_dtype(self.options.state_dtype), device="cuda")
        self._check_tensor(out, i, self.options.state_dtype)
        self._check(self.lib.muonbp_get_momentum(self.ctx, i, ctypes.c_void_p(out.data_ptr())),
                    "get_momentum")
        return out

    def set_momentum(self, i: int, src) -> None:
        self._check_tensor(src, i, self.options.state_dtype)
        self._check(self.lib.muonbp_set_momentum(self.ctx, i, ctypes.c_void_p(src.data_ptr())),
                    "set_momentum")

    def get_update(self, i: int, out=None):
        import torch
        r, c = self.mats[i][:2]
        if out is None:
            out = torch.empty((r, c), dtype=_torch_dtype(self.options.ns_dtype), device="cuda")
        self._check_tensor(out, i, self.options.ns_dtype)
        self._check(self.lib.muonbp_get_update(self.ctx, i, ctypes.c_void_p(out.data_ptr())),
                    "get_update")
        return out

    def synchronize(self) -> None:
        self._check(self.lib.muonbp_synchronize(self.ctx), "synchronize")

    def profile_enable(self, on=True) -> None:
        """True / 1: events around every launch; 2: one span per step over
        the NS GEMM launches (kind "ns_span"); False / 0: off."""
        self._check(self.lib.muonbp_profile_enable(self.ctx, int(on)), "profile_enable")

    def profile_read(self, split: bool = False) -> dict:
        """{kind: (ms, launches)} summed over the launches recorded since the
        last read; with split=True, {"block": {...}, "full": {...}} by the
        kind of step that enqueued them."""
        p = Profile()
        self._check(self.lib.muonbp_profile_read(self.ctx, ctypes.byref(p)), "profile_read")
        if not split:
            return {k: (p.ms[i], p.launches[i]) for i, k in enumerate(KERNEL_KINDS)}
        return {"full": {k: (p.ms_full_steps[i], p.launches_full_steps[i])
                         for i, k in enumerate(KERNEL_KINDS)},
                "block": {k: (p.ms[i] - p.ms_full_steps[i], p.launches[i] - p.launches_full_steps[i])
                          for i, k in enumerate(KERNEL_KINDS)}}

    def close(self) -> None:
        if getattr(self, "ctx", None):
            self.lib.muonbp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- scalar optimizer

def adamw_options_default(**overrides) -> AdamwOptions:
    """Library defaults (beta1 0.9, beta2 0.95, eps 1e-8, weight decay 0.1,
    clipping at 1.0, bf16) with fields overridden by keyword."""
    o = AdamwOptions()
    load_library().muonbp_adamw_options_default(ctypes.byref(o))
    for k, v in overrides.items():
        if not hasattr(o, k):
            raise AttributeError(k)
        setattr(o, k, v)
    return o


class AdamW:
    """AdamW with global-norm clipping over a fixed list of tensors (the
    parameters MuonBP does not orthogonalize)."""

    def __init__(self, sizes: Sequence[int], options: Optional[AdamwOptions] = None, stream=None):
        import torch
        self.lib = load_library()
        self.sizes = [int(n) for n in sizes]
        self.options = options if options is not None else adamw_options_default()
        if stream is None:
            stream = torch.cuda.current_stream()
        arr = (ctypes.c_int64 * len(self.sizes))(*self.sizes)
        ctx = ctypes.c_void_p()
        st = self.lib.muonbp_adamw_create(arr, len(self.sizes), ctypes.byref(self.options),
                                          ctypes.c_void_p(stream.cuda_stream), ctypes.byref(ctx))
        if st:
            raise MuonBPError(st, "muonbp_adamw_create")
        self.ctx = ctx
        self._ptrs = (ctypes.c_void_p * len(self.sizes))()
        self._gptrs = (ctypes.c_void_p * len(self.sizes))()

    def _check(self, st: int, what: str):
        if st:
            detail = self.lib.muonbp_adamw_last_error(self.ctx)
            raise MuonBPError(st, f"{what}: {detail.decode() if detail else ''}")

    def _check_tensor(self, t, i, dtype):
        if not (t.is_cuda and t.is_contiguous() and t.dtype == dtype and t.numel() == self.sizes[i]):
            raise ValueError(f"tensor {i}: need a contiguous {dtype} CUDA tensor of "
                             f"{self.sizes[i]} elements, got {t.dtype} {tuple(t.shape)}")

    def step(self, params: List, grads: List, t: int, lr: float) -> None:
        import torch
        n = len(self.sizes)
        if len(params) != n or len(grads) != n:
            raise ValueError("one param and one grad per tensor")
        dt = _torch_dtype(self.options.param_dtype)
        for i in range(n):
            self._check_tensor(params[i], i, dt)
            self._check_tensor(grads[i], i, dt)
            self._ptrs[i] = params[i].data_ptr()
            self._gptrs[i] = grads[i].data_ptr()
        self._check(self.lib.muonbp_adamw_step(self.ctx, self._ptrs, self._gptrs, int(t), float(lr)),
                    "adamw_step")

    def grad_norm(self) -> float:
        out = ctypes.c_float()
        self._check(self.lib.muonbp_adamw_grad_norm(self.ctx, ctypes.byref(out)), "grad_norm")
        return float(out.value)

    def get_state(self, i: int):
        import torch
        m = torch.empty(self.sizes[i], dtype=torch.float32, device="cuda")
        v = torch.empty_like(m)
        self._check(self.lib.muonbp_adamw_get_state(self.ctx, i, ctypes.c_void_p(m.data_ptr()),
                                                    ctypes.c_void_p(v.data_ptr())), "get_state")
        return m, v

    def set_state(self, i: int, m, v) -> None:
        import torch
        for t in (m, v):
            self._check_tensor(t, i, torch.float32)
        self._check(self.lib.muonbp_adamw_set_state(self.ctx, i, ctypes.c_void_p(m.data_ptr()),
                                                    ctypes.c_void_p(v.data_ptr())), "set_state")

    def synchronize(self) -> None:
        self._check(self.lib.muonbp_adamw_synchronize(self.ctx), "synchronize")

    def close(self) -> None:
        if getattr(self, "ctx", None):
            self.lib.muonbp_adamw_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def lr_cosine(t: int, total: int, lr_max: float, lr_min: float = 0.0, warmup: int = 0) -> float:
    """Cosine schedule of the library (muonbp_lr_cosine)."""
    return load_library().muonbp_lr_cosine(int(t), int(total), float(lr_max), float(lr_min), int(warmup))


def lr_wsd(t: int, total: int, lr_max: float, lr_min: float = 0.0, warmup: int = 0,
           decay: int = 0) -> float:
    """Warmup-stable-decay schedule of the library (muonbp_lr_wsd)."""
    return load_library().muonbp_lr_wsd(int(t), int(total), float(lr_max), float(lr_min), int(warmup),
                                        int(decay))
