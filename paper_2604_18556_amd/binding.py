"""ctypes binding of include/gsq.h: argument marshalling only.

Every computation runs in ``libgsq.so``; this module passes device pointers
(``tensor.data_ptr()``) and the current HIP stream to it and turns status codes
into exceptions.  Loading fails loudly when the library has not been built.
"""
import ctypes
import os
from dataclasses import dataclass, field

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgsq.so")

GSQ_OK, GSQ_EINVAL, GSQ_ENOMEM, GSQ_EHIP, GSQ_ENONFINITE, GSQ_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
LAYOUT_GROUP, LAYOUT_SUPERBLOCK, LAYOUT_BASE3 = 0, 1, 2
RELAX_GRID, RELAX_SHIFT, RELAX_TERNARY = 0, 1, 2
MAX_LEVELS = 16             # GSQ_MAX_LEVELS
SHIFT_WINDOW = 5            # GSQ_SHIFT_WINDOW
PREC_FP32, PREC_BF16 = 0, 1
DT_FP32, DT_BF16 = 0, 1
OPT_ADAM, OPT_LION = 0, 1
MAX_SAMPLES = 16            # GSQ_MAX_SAMPLES
STATUS_NAMES = {0: "GSQ_OK", -1: "GSQ_EINVAL", -2: "GSQ_ENOMEM", -3: "GSQ_EHIP",
                -4: "GSQ_ENONFINITE", -5: "GSQ_EUNSUPPORTED"}

EXPORTS = ("gsq_layer_init", "gsq_step", "gsq_step_static", "gsq_harden", "gsq_packed_size",
           "gsq_pack", "gsq_get_state", "gsq_set_state", "gsq_get_intermediates", "gsq_gumbel", "gsq_check",
           "gsq_layer_destroy", "gsq_last_error", "gsq_timing", "gsq_timing_read")
KERNEL_NAMES = ("init", "forward", "contract", "reduce", "backward", "harden", "pack")


class GsqError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class CConfig(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("out_features", ctypes.c_int32),
                ("in_features", ctypes.c_int32), ("n_levels", ctypes.c_int32),
                ("levels", ctypes.c_float * MAX_LEVELS), ("group_size", ctypes.c_int32),
                ("layout", ctypes.c_int32), ("precision", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("alpha", ctypes.c_float), ("sigma_init", ctypes.c_float),
                ("init_noise", ctypes.c_int32), ("relaxation", ctypes.c_int32)]


class CStepParams(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_float), ("kappa", ctypes.c_float), ("lr_logits", ctypes.c_float),
                ("lr_scales", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("gumbel_noise", ctypes.c_int32),
                ("tau_next", ctypes.c_float), ("kappa_next", ctypes.c_float),
                ("optimizer", ctypes.c_int32), ("weight_decay", ctypes.c_float),
                ("samples", ctypes.c_int32)]


@dataclass
class LayerConfig:
    out_features: int
    in_features: int
    levels: tuple
    group_size: int = 128
    batch: int = 1
    layout: int = LAYOUT_GROUP
    precision: int = PREC_BF16
    seed: int = 0
    alpha: float = 6.0
    sigma_init: float = 1.0
    init_noise: bool = True
    relaxation: int = RELAX_GRID

    def to_c(self):
        c = CConfig()
        c.batch, c.out_features, c.in_features = self.batch, self.out_features, self.in_features
        c.n_levels = len(self.levels)
        for k, x in enumerate(self.levels):
            c.levels[k] = float(x)
        c.group_size, c.layout, c.precision = self.group_size, self.layout, self.precision
        c.seed, c.alpha, c.sigma_init = self.seed, self.alpha, self.sigma_init
        c.init_noise = 1 if self.init_noise else 0
        c.relaxation = self.relaxation
        return c

    @property
    def gs(self):
        return 16 if self.layout == LAYOUT_SUPERBLOCK else self.group_size

    @property
    def K(self):
        """Logits per coordinate."""
        return {RELAX_SHIFT: SHIFT_WINDOW, RELAX_TERNARY: 2}.get(self.relaxation, len(self.levels))


@dataclass
class StepParams:
    tau: float
    kappa: float = 1.0
    lr_logits: float = 1e-2
    lr_scales: float = 5e-5
    beta1: float = 0.9
    beta2: float = 0.95
    eps: float = 1e-8
    gumbel_noise: bool = True
    tau_next: float = 0.0
    kappa_next: float = 1.0
    optimizer: int = OPT_ADAM
    weight_decay: float = 0.0
    samples: int = 1

    def to_c(self):
        return CStepParams(self.tau, self.kappa, self.lr_logits, self.lr_scales, self.beta1,
                           self.beta2, self.eps, 1 if self.gumbel_noise else 0, self.tau_next,
                           self.kappa_next, self.optimizer, self.weight_decay, self.samples)


_lib = None


def load(path=None):
    """Load libgsq.so (raises if it is missing: there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or _LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(hipcc, gfx950); the GSQ step has no other implementation")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.gsq_layer_init.argtypes = [ctypes.POINTER(CConfig), vp, i32, vp, vp, vp, ctypes.POINTER(vp)]
    lib.gsq_step.argtypes = [vp, ctypes.POINTER(CStepParams), vp, vp]
    lib.gsq_step_static.argtypes = [vp, ctypes.POINTER(CStepParams), vp, vp]
    lib.gsq_harden.argtypes = [vp, vp, vp, vp, vp]
    lib.gsq_packed_size.argtypes = [ctypes.POINTER(CConfig)]
    lib.gsq_packed_size.restype = sz
    lib.gsq_pack.argtypes = [vp, vp, sz, vp]
    lib.gsq_get_state.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(i64), vp]
    lib.gsq_set_state.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, vp]
    lib.gsq_get_intermediates.argtypes = [vp, vp, vp, vp]
    lib.gsq_gumbel.argtypes = [ctypes.POINTER(CConfig), i64, i64, i64, vp, vp]
    lib.gsq_check.argtypes = [vp, vp]
    lib.gsq_layer_destroy.argtypes = [vp]
    lib.gsq_last_error.restype = ctypes.c_char_p
    lib.gsq_timing.argtypes = [vp, i32]
    lib.gsq_timing_read.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64), i32, vp]
    for name in ("gsq_layer_init", "gsq_step", "gsq_step_static", "gsq_harden", "gsq_pack",
                 "gsq_get_state", "gsq_set_state", "gsq_get_intermediates", "gsq_gumbel", "gsq_check",
                 "gsq_layer_destroy", "gsq_timing", "gsq_timing_read"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(status):
    if status != GSQ_OK:
        raise GsqError(status, load().gsq_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _arg(t, name, numel, dtypes):
    """Check a tensor argument before its pointer reaches the library, which reads or writes
    exactly ``numel`` elements through it: a dense device tensor of one of ``dtypes``."""
    if t is None:
        return
    if not (t.is_cuda and t.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements, got {t.numel()}")


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def packed_size(cfg):
    return int(load().gsq_packed_size(ctypes.byref(cfg.to_c())))


def gumbel(cfg, e0, count, t, out, stream=None):
    """Noise of coordinates [e0, e0 + count) at step t into ``out`` (cuda fp32, count x Z):
    Z = K Gumbel values, or for TERNARY the two pairs' logistic values."""
    import torch
    if count > 0:
        _arg(out, "out", count * cfg.K, (torch.float32,))
    _check(load().gsq_gumbel(ctypes.byref(cfg.to_c()), e0, count, t, _ptr(out), _stream(stream)))


class Layer:
    """One handle of the library (gsq_layer*)."""

    def __init__(self, cfg, W, H, scales_init=None, stream=None):
        import torch
        lib = load()
        self.cfg = cfg
        self._c = cfg.to_c()
        if W.dtype == torch.bfloat16:
            wdt = DT_BF16
        elif W.dtype == torch.float32:
            wdt = DT_FP32
        else:
            raise TypeError("W must be float32 or bfloat16")
        for name, t in (("W", W), ("H", H), ("scales_init", scales_init)):
            if t is not None and not (t.is_cuda and t.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous device tensor")
        if H.dtype != torch.float32:
            raise TypeError("H must be float32")
        B, O, I = cfg.batch, cfg.out_features, cfg.in_features
        _arg(W, "W", B * O * I, (torch.float32, torch.bfloat16))
        _arg(H, "H", B * I * I, (torch.float32,))
        _arg(scales_init, "scales_init", B * O * (I // cfg.gs), (torch.float32,))
        h = ctypes.c_void_p()
        _check(lib.gsq_layer_init(ctypes.byref(self._c), _ptr(W), wdt, _ptr(H), _ptr(scales_init),
                                  _stream(stream), ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("layer destroyed")
        return self._h

    # element counts of the caller-side tensors
    @property
    def _n(self):
        c = self.cfg
        return c.batch * c.out_features * c.in_features

    @property
    def _ng(self):
        c = self.cfg
        return c.batch * c.out_features * (c.in_features // c.gs)

    def step(self, params, loss_out=None, stream=None):
        import torch
        _arg(loss_out, "loss_out", self.cfg.batch, (torch.float32,))
        _check(load().gsq_step(self.handle, ctypes.byref(params.to_c()), _ptr(loss_out),
                               _stream(stream)))

    def step_static(self, params, loss_out=None, stream=None):
        """gsq_step_static: the same step with no allocation (static scratch of the library)."""
        import torch
        _arg(loss_out, "loss_out", self.cfg.batch, (torch.float32,))
        _check(load().gsq_step_static(self.handle, ctypes.byref(params.to_c()), _ptr(loss_out),
                                      _stream(stream)))

    def harden(self, codes=None, scales=None, hard_loss=None, stream=None):
        import torch
        _arg(codes, "codes", self._n, (torch.uint8,))
        _arg(scales, "scales", self._ng, (torch.float32,))
        _arg(hard_loss, "hard_loss", self.cfg.batch, (torch.float32,))
        _check(load().gsq_harden(self.handle, _ptr(codes), _ptr(scales), _ptr(hard_loss),
                                 _stream(stream)))

    def pack(self, out, stream=None):
        if not (out.is_cuda and out.is_contiguous()):
            raise ValueError("out must be a contiguous device tensor")
        _check(load().gsq_pack(self.handle, _ptr(out), out.numel() * out.element_size(),
                               _stream(stream)))

    def get_state(self, logits=None, m=None, v=None, scales=None, m_s=None, v_s=None, base=None,
                  stream=None):
        self._state_args(logits, m, v, scales, m_s, v_s, base)
        t = ctypes.c_int64()
        _check(load().gsq_get_state(self.handle, _ptr(logits), _ptr(m), _ptr(v), _ptr(scales),
                                    _ptr(m_s), _ptr(v_s), _ptr(base), ctypes.byref(t),
                                    _stream(stream)))
        return t.value

    def set_state(self, t, logits=None, m=None, v=None, scales=None, m_s=None, v_s=None, base=None,
                  stream=None):
        self._state_args(logits, m, v, scales, m_s, v_s, base)
        _check(load().gsq_set_state(self.handle, _ptr(logits), _ptr(m), _ptr(v), _ptr(scales),
                                    _ptr(m_s), _ptr(v_s), _ptr(base), int(t), _stream(stream)))

    def _state_args(self, logits, m, v, scales, m_s, v_s, base):
        import torch
        for name, x in (("logits", logits), ("m", m), ("v", v)):
            _arg(x, name, self._n * self.cfg.K, (torch.float32,))
        for name, x in (("scales", scales), ("m_s", m_s), ("v_s", v_s)):
            _arg(x, name, self._ng, (torch.float32,))
        _arg(base, "base", self._n, (torch.uint8,))

    def intermediates(self, residual=None, grad=None, stream=None):
        import torch
        _arg(residual, "residual", self._n,
             (torch.bfloat16,) if self.cfg.precision == PREC_BF16 else (torch.float32,))
        _arg(grad, "grad", self._n, (torch.float32,))
        _check(load().gsq_get_intermediates(self.handle, _ptr(residual), _ptr(grad), _stream(stream)))

    def timing(self, enable):
        _check(load().gsq_timing(self.handle, 1 if enable else 0))

    def timing_read(self, reset=True, stream=None):
        """{kernel: (total ms, launches)} since the last reset (synchronises the stream)."""
        n = len(KERNEL_NAMES)
        ms = (ctypes.c_double * n)()
        cnt = (ctypes.c_int64 * n)()
        _check(load().gsq_timing_read(self.handle, ms, cnt, 1 if reset else 0, _stream(stream)))
        return {KERNEL_NAMES[k]: (ms[k], cnt[k]) for k in range(n)}

    def check(self, stream=None):
        _check(load().gsq_check(self.handle, _stream(stream)))

    def destroy(self):
        if self._h is not None:
            load().gsq_layer_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass
