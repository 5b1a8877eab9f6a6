"""ctypes binding of libjorge.so: argument marshalling only.

Every step of the Jorge update runs in the HIP kernels behind the C ABI of
include/jorge.h. torch is used only to own device tensors and to name the
current HIP stream; there is no CPU fallback: if the library is missing or
fails to load, construction raises.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libjorge.so")

JORGE_OK = 0
BETA_MODES = {"fixed": 0, "dynamic": 1, "clamped": 2}
STATE_KINDS = {"L": 0, "R": 1, "mom": 2, "mom_sgd": 3}
FACTOR_FORMS = {"auto": 0, "explicit": 1, "factored": 2, "squared": 3}
DIAG_NAMES = ("nu_L", "nu_R", "beta_L", "beta_R", "norm_m", "norm_sgd", "g")


class JorgeError(RuntimeError):
    def __init__(self, status: int, detail: str = ""):
        self.status = status
        super().__init__(f"jorge status {status}: {detail}")


class Shape(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("cols", ctypes.c_int64)]


class HParams(ctypes.Structure):
    _fields_ = [("eps", ctypes.c_double), ("precond_interval", ctypes.c_int32),
                ("beta_mode", ctypes.c_int32), ("graft", ctypes.c_int32),
                ("symmetrize", ctypes.c_int32), ("factor_form", ctypes.c_int32),
                ("split_k", ctypes.c_int32), ("lds_chain_max", ctypes.c_int32),
                ("precond_lowrank", ctypes.c_int32), ("series_order", ctypes.c_int32)]


_LIB = None

# name -> (restype, argtypes); mirrors include/jorge.h
_P = ctypes.c_void_p
_SIGNATURES = {
    "jorge_hparams_default": (ctypes.c_int32, [ctypes.POINTER(HParams)]),
    "jorge_create": (ctypes.c_int32, [ctypes.POINTER(Shape), ctypes.c_int32, ctypes.POINTER(HParams), _P,
                                      ctypes.POINTER(_P)]),
    "jorge_plan": (ctypes.c_int32, [ctypes.POINTER(Shape), ctypes.c_int32, ctypes.POINTER(HParams),
                                    ctypes.POINTER(ctypes.c_int64)]),
    "jorge_plan_stages": (ctypes.c_int32, [ctypes.POINTER(Shape), ctypes.c_int32, ctypes.POINTER(HParams),
                                           ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64),
                                           ctypes.POINTER(ctypes.c_int64), ctypes.c_int32]),
    "jorge_step": (ctypes.c_int32, [_P, ctypes.POINTER(_P), ctypes.POINTER(_P), ctypes.c_double,
                                    ctypes.c_double, ctypes.c_double, ctypes.c_double]),
    "jorge_step_noalloc": (ctypes.c_int32, [ctypes.POINTER(Shape), ctypes.POINTER(HParams), ctypes.c_int64, _P, _P,
                                            _P, _P, _P, _P, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                            ctypes.c_double, _P]),
    "jorge_get_state": (ctypes.c_int32, [_P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64]),
    "jorge_set_state": (ctypes.c_int32, [_P, ctypes.c_int32, ctypes.c_int32, _P, ctypes.c_int64]),
    "jorge_state_ptr": (ctypes.c_int32, [_P, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_P),
                                         ctypes.POINTER(ctypes.c_int64)]),
    "jorge_get_step": (ctypes.c_int32, [_P, ctypes.POINTER(ctypes.c_int64)]),
    "jorge_set_step": (ctypes.c_int32, [_P, ctypes.c_int64]),
    "jorge_read_diag": (ctypes.c_int32, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)]),
    "jorge_nonfinite": (ctypes.c_int32, [_P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
    "jorge_set_stream": (ctypes.c_int32, [_P, _P]),
    "jorge_synchronize": (ctypes.c_int32, [_P]),
    "jorge_device_bytes": (ctypes.c_int32, [_P, ctypes.POINTER(ctypes.c_int64)]),
    "jorge_set_timing": (ctypes.c_int32, [_P, ctypes.c_int32]),
    "jorge_read_timing": (ctypes.c_int32, [_P, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_int64), ctypes.c_int32]),
    "jorge_reset_timing": (ctypes.c_int32, [_P]),
    "jorge_num_stages": (ctypes.c_int32, []),
    "jorge_stage_flops": (ctypes.c_int32, [_P, ctypes.POINTER(ctypes.c_double), ctypes.c_int32]),
    "jorge_factor_form": (ctypes.c_int32, [_P, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
    "jorge_stage_name": (ctypes.c_char_p, [ctypes.c_int32]),
    "jorge_destroy": (None, [_P]),
    "jorge_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "jorge_last_error": (ctypes.c_char_p, [_P]),
}


def load_library(path: str | None = None) -> ctypes.CDLL:
    """Loads libjorge.so (built by paper_2310_12298_amd.build); raises if absent.

    path: the library file, LIB_PATH by default (read at call time, so a test can
    point the binding at another build of the same sources).
    """
    global _LIB
    if _LIB is not None:
        return _LIB
    path = LIB_PATH if path is None else path
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is not built; run __graft_entry__.build() or "
                                f"python -m paper_2310_12298_amd.build")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def _check(lib, status, ctx=None):
    if status != JORGE_OK:
        detail = lib.jorge_status_string(status).decode()
        if ctx:
            extra = lib.jorge_last_error(ctx).decode()
            if extra:
                detail += f" ({extra})"
        raise JorgeError(status, detail)


def _current_stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


class Jorge:
    """A Jorge optimizer context over a fixed list of m x n layers.

    shapes: list of (rows, cols). State lives on the current HIP device.
    """

    def __init__(self, shapes, eps=1e-6, precond_interval=1, beta_mode="clamped", graft=True,
                 symmetrize=True, factor_form="auto", split_k=True, lds_chain_max=128, precond_lowrank=True,
                 series_order=2, stream=None):
        self.lib = load_library()
        self.shapes = [(int(m), int(n)) for m, n in shapes]
        hp = self.hparams(eps, precond_interval, beta_mode, graft, symmetrize, factor_form, split_k,
                          lds_chain_max, precond_lowrank, series_order)
        arr = (Shape * len(self.shapes))(*[Shape(m, n) for m, n in self.shapes])
        ctx = _P()
        s = _current_stream() if stream is None else int(stream)
        _check(self.lib, self.lib.jorge_create(arr, len(self.shapes), ctypes.byref(hp), _P(s),
                                               ctypes.byref(ctx)))
        self.ctx = ctx

    @staticmethod
    def hparams(eps=1e-6, precond_interval=1, beta_mode="clamped", graft=True, symmetrize=True,
                factor_form="auto", split_k=True, lds_chain_max=128, precond_lowrank=True, series_order=2):
        lib = load_library()
        hp = HParams()
        _check(lib, lib.jorge_hparams_default(ctypes.byref(hp)))
        hp.eps = float(eps)
        hp.precond_interval = int(precond_interval)
        hp.beta_mode = BETA_MODES[beta_mode] if isinstance(beta_mode, str) else int(beta_mode)
        hp.graft = int(bool(graft))
        hp.symmetrize = int(bool(symmetrize))
        hp.factor_form = FACTOR_FORMS[factor_form] if isinstance(factor_form, str) else int(factor_form)
        hp.split_k = int(split_k)
        hp.lds_chain_max = int(lds_chain_max)
        hp.precond_lowrank = int(bool(precond_lowrank))
        hp.series_order = int(series_order)
        return hp

    @staticmethod
    def plan(shapes, **hp):
        """Device bytes a context would hold; builds and checks its launch tables on the host (no GPU)."""
        lib = load_library()
        shapes = [(int(m), int(n)) for m, n in shapes]
        arr = (Shape * max(1, len(shapes)))(*[Shape(m, n) for m, n in shapes])
        h = Jorge.hparams(**hp)
        v = ctypes.c_int64()
        _check(lib, lib.jorge_plan(arr, len(shapes), ctypes.byref(h), ctypes.byref(v)))
        return v.value

    @staticmethod
    def plan_stages(shapes, **hp):
        """Per stage name: (work units, tiles split along K, small-mode blocks) of its grouped
        GEMM launches (no GPU)."""
        lib = load_library()
        shapes = [(int(m), int(n)) for m, n in shapes]
        arr = (Shape * max(1, len(shapes)))(*[Shape(m, n) for m, n in shapes])
        h = Jorge.hparams(**hp)
        n = lib.jorge_num_stages()
        units, split, small = (ctypes.c_int64 * n)(), (ctypes.c_int64 * n)(), (ctypes.c_int64 * n)()
        _check(lib, lib.jorge_plan_stages(arr, len(shapes), ctypes.byref(h), units, split, small, n))
        return {lib.jorge_stage_name(i).decode(): (units[i], split[i], small[i]) for i in range(n)}

    # -------------------------------------------------------------- stepping
    def _ptrs(self, tensors, what):
        import torch
        if len(tensors) != len(self.shapes):
            raise ValueError(f"{what}: expected {len(self.shapes)} tensors, got {len(tensors)}")
        for t, (m, n) in zip(tensors, self.shapes):
            if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.float32
                    and t.is_contiguous() and tuple(t.shape) == (m, n)):
                raise ValueError(f"{what}: need contiguous fp32 cuda tensors of shape {(m, n)}")
        return (_P * len(tensors))(*[t.data_ptr() for t in tensors])

    def step(self, params, grads, lr, beta2=0.9, beta1=0.9, weight_decay=0.0):
        """One Jorge step for all layers on the context's stream (params updated in place)."""
        p = self._ptrs(params, "params")
        g = self._ptrs(grads, "grads")
        _check(self.lib, self.lib.jorge_step(self.ctx, p, g, float(lr), float(beta2), float(beta1),
                                             float(weight_decay)), self.ctx)

    def step_ptrs(self, param_ptrs, grad_ptrs, lr, beta2=0.9, beta1=0.9, weight_decay=0.0):
        """Same as step, from prebuilt ctypes pointer arrays (no per-call checks)."""
        _check(self.lib, self.lib.jorge_step(self.ctx, param_ptrs, grad_ptrs, float(lr), float(beta2),
                                             float(beta1), float(weight_decay)), self.ctx)

    @staticmethod
    def step_noalloc(t, theta, grad, L, R, mom, mom_sgd, lr, beta2=0.9, beta1=0.9, weight_decay=0.0, stream=None,
                     **hp):
        """One step of one layer through jorge_step_noalloc: the caller's tensors hold the state
        (L, R, mom, mom_sgd updated in place with theta); temporaries live in the library's static
        device scratch. t: the number of this step (>= 1). Returns after the step has run."""
        import torch
        lib = load_library()
        m, n = theta.shape
        for x, shp in ((theta, (m, n)), (grad, (m, n)), (L, (m, m)), (R, (n, n)), (mom, (m, n)),
                       (mom_sgd, (m, n))):
            if not (isinstance(x, torch.Tensor) and x.is_cuda and x.dtype == torch.float32 and x.is_contiguous()
                    and tuple(x.shape) == shp):
                raise ValueError(f"need a contiguous fp32 cuda tensor of shape {shp}")
        shape = Shape(m, n)
        h = Jorge.hparams(**hp)
        s = _current_stream() if stream is None else int(stream)
        _check(lib, lib.jorge_step_noalloc(ctypes.byref(shape), ctypes.byref(h), int(t), _P(theta.data_ptr()),
                                           _P(grad.data_ptr()), _P(L.data_ptr()), _P(R.data_ptr()),
                                           _P(mom.data_ptr()), _P(mom_sgd.data_ptr()), float(lr), float(beta2),
                                           float(beta1), float(weight_decay), _P(s)))

    @staticmethod
    def pointer_array(tensors):
        return (_P * len(tensors))(*[t.data_ptr() for t in tensors])

    # -------------------------------------------------------------- state
    def _dims(self, layer, kind):
        m, n = self.shapes[layer]
        return {0: (m, m), 1: (n, n), 2: (m, n), 3: (m, n)}[kind]

    def get_state(self, layer, kind):
        """Copy of one state tensor as a new fp32 device tensor (stream-ordered)."""
        import torch
        kind = STATE_KINDS[kind] if isinstance(kind, str) else int(kind)
        r, c = self._dims(layer, kind)
        out = torch.empty((r, c), dtype=torch.float32, device="cuda")
        _check(self.lib, self.lib.jorge_get_state(self.ctx, layer, kind, _P(out.data_ptr()), c), self.ctx)
        return out

    def set_state(self, layer, kind, tensor):
        import torch
        kind = STATE_KINDS[kind] if isinstance(kind, str) else int(kind)
        r, c = self._dims(layer, kind)
        t = tensor.to(device="cuda", dtype=torch.float32).contiguous()
        if tuple(t.shape) != (r, c):
            raise ValueError(f"state shape {tuple(t.shape)} != {(r, c)}")
        _check(self.lib, self.lib.jorge_set_state(self.ctx, layer, kind, _P(t.data_ptr()), c), self.ctx)
        self.synchronize()            # t may be freed once this returns

    def state_ptr(self, layer, kind):
        kind = STATE_KINDS[kind] if isinstance(kind, str) else int(kind)
        p, ld = _P(), ctypes.c_int64()
        _check(self.lib, self.lib.jorge_state_ptr(self.ctx, layer, kind, ctypes.byref(p), ctypes.byref(ld)),
               self.ctx)
        return p.value, ld.value

    @property
    def t(self):
        v = ctypes.c_int64()
        _check(self.lib, self.lib.jorge_get_step(self.ctx, ctypes.byref(v)))
        return v.value

    @t.setter
    def t(self, value):
        _check(self.lib, self.lib.jorge_set_step(self.ctx, int(value)), self.ctx)

    def read_diag(self, layer):
        out = (ctypes.c_double * len(DIAG_NAMES))()
        _check(self.lib, self.lib.jorge_read_diag(self.ctx, layer, out), self.ctx)
        return dict(zip(DIAG_NAMES, list(out)))

    def nonfinite(self):
        """(count, first): layers whose gradient held a NaN or an infinity in any step since the
        last call (first = the lowest such layer, -1 if none); clears the flags. Synchronises."""
        n, f = ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib, self.lib.jorge_nonfinite(self.ctx, ctypes.byref(n), ctypes.byref(f)), self.ctx)
        return n.value, f.value

    def synchronize(self):
        _check(self.lib, self.lib.jorge_synchronize(self.ctx), self.ctx)

    def set_stream(self, stream):
        _check(self.lib, self.lib.jorge_set_stream(self.ctx, _P(int(stream))), self.ctx)

    def device_bytes(self):
        v = ctypes.c_int64()
        _check(self.lib, self.lib.jorge_device_bytes(self.ctx, ctypes.byref(v)))
        return v.value

    def factor_form(self, layer, side):
        """'explicit', 'factored' or 'squared': the evaluation order of L_hat (side 0) or R_hat (side 1)."""
        v = ctypes.c_int32()
        _check(self.lib, self.lib.jorge_factor_form(self.ctx, int(layer), int(side), ctypes.byref(v)), self.ctx)
        return {1: "explicit", 2: "factored", 3: "squared"}[v.value]

    # -------------------------------------------------------------- timing
    def set_timing(self, enable: bool):
        _check(self.lib, self.lib.jorge_set_timing(self.ctx, int(bool(enable))), self.ctx)

    def reset_timing(self):
        _check(self.lib, self.lib.jorge_reset_timing(self.ctx), self.ctx)

    def read_timing(self):
        """{stage name: (total ms, launches)} accumulated since the last reset (synchronises)."""
        n = self.lib.jorge_num_stages()
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check(self.lib, self.lib.jorge_read_timing(self.ctx, ms, cnt, n), self.ctx)
        return {self.lib.jorge_stage_name(i).decode(): (ms[i], cnt[i]) for i in range(n)}

    def stage_flops(self):
        """{stage name: algorithmic flops of that stage in one factor-updating step}."""
        n = self.lib.jorge_num_stages()
        fl = (ctypes.c_double * n)()
        _check(self.lib, self.lib.jorge_stage_flops(self.ctx, fl, n), self.ctx)
        return {self.lib.jorge_stage_name(i).decode(): fl[i] for i in range(n)}

    # -------------------------------------------------------------- lifetime
    def close(self):
        if getattr(self, "ctx", None):
            self.lib.jorge_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
