"""ctypes binding of librikfad.so (declared in include/rikfad.h).

Argument marshalling only: every step of the optimiser runs in the library's
HIP kernels.  The functions keep the C names; ``RIKFAD``, ``IKFAD`` and
``ADAFM`` (the Adafactor-m baseline) are small conveniences that collect device pointers from torch tensors and
allocate the optimiser state as zero-filled torch tensors.  There is no CPU
fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librikfad.so")

RIKFAD_OK, RIKFAD_EINVAL, RIKFAD_EALIGN, RIKFAD_EDTYPE = 0, -1, -2, -3
RIKFAD_ENOMEM, RIKFAD_EHIP, RIKFAD_ESTATE = -4, -5, -6
RIKFAD_FP32, RIKFAD_BF16 = 0, 1
RIKFAD_FLAG_TWO_PASS = 1


class RikfadError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {rikfad_status_string(status)} ({status}): "
                         f"{rikfad_last_error()}")


class rikfad_tensor(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("g", ctypes.c_void_p), ("p", ctypes.c_void_p),
                ("r", ctypes.c_void_p), ("c", ctypes.c_void_p),
                ("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class ikfad_tensor(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("g", ctypes.c_void_p), ("p", ctypes.c_void_p),
                ("xi", ctypes.c_void_p), ("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class rikfad_hparams(ctypes.Structure):
    _fields_ = [("h", ctypes.c_double), ("gamma", ctypes.c_double),
                ("alpha", ctypes.c_double), ("mu", ctypes.c_double),
                ("eps_stab", ctypes.c_double)]


class rikfad_info(ctypes.Structure):
    _fields_ = [(nm, ctypes.c_int64) for nm in (
        "tensors", "matrices", "vectors", "elements", "state_bytes", "ikfad_state_bytes",
        "workspace_bytes", "min_bytes_per_step", "stream_min_bytes", "stream_tiles",
        "finalize_items")] + [("pending", ctypes.c_int32), ("two_pass", ctypes.c_int32)]


class adafm_hparams(ctypes.Structure):
    _fields_ = [("h", ctypes.c_double), ("beta1", ctypes.c_double),
                ("decay_rate", ctypes.c_double), ("eps1", ctypes.c_double),
                ("eps2", ctypes.c_double), ("clip_threshold", ctypes.c_double),
                ("scale_parameter", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class rikfad_friction_stats(ctypes.Structure):
    _fields_ = [(nm, ctypes.c_double) for nm in (
        "xi_fro2", "err_fro2", "sum_r", "sigma1", "rel_err", "eckart_young_floor",
        "stable_rank")] + [("power_iters", ctypes.c_int32), ("reserved", ctypes.c_int32)]


_lib = None

# name -> (restype, argtypes)
_vp, _i64, _i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
_st = ctypes.c_int
_P = ctypes.POINTER
_SIGNATURES = {
    "rikfad_create": (_st, [_vp, _i64, _P(rikfad_hparams), ctypes.c_uint32, _P(_vp)]),
    "rikfad_step": (_st, [_vp, _vp]),
    "rikfad_step_grads": (_st, [_vp, _vp, _vp]),
    "rikfad_set_hparams": (_st, [_vp, _P(rikfad_hparams), _vp]),
    "rikfad_sync_momentum": (_st, [_vp, _vp]),
    "rikfad_state_changed": (_st, [_vp]),
    "rikfad_query": (_st, [_vp, _P(rikfad_info)]),
    "rikfad_state_bytes": (_st, [_vp, _i64, _P(_i64), _P(_i64)]),
    "rikfad_nonfinite": (_st, [_vp, _vp, _P(_i32)]),
    "rikfad_timing_enable": (_st, [_vp, _i32]),
    "rikfad_timing_read": (_st, [_vp, _P(ctypes.c_double), _P(ctypes.c_double),
                                 _P(ctypes.c_double), _P(_i64)]),
    "rikfad_destroy": (None, [_vp]),
    "rikfad_status_string": (ctypes.c_char_p, [_st]),
    "rikfad_last_error": (ctypes.c_char_p, []),
    "ikfad_create": (_st, [_vp, _i64, _P(rikfad_hparams), _P(_vp)]),
    "ikfad_step": (_st, [_vp, _vp]),
    "ikfad_set_hparams": (_st, [_vp, _P(rikfad_hparams)]),
    "ikfad_timing_enable": (_st, [_vp, _i32]),
    "ikfad_timing_read": (_st, [_vp, _P(ctypes.c_double), _P(_i64)]),
    "ikfad_nonfinite": (_st, [_vp, _vp, _P(_i32)]),
    "ikfad_destroy": (None, [_vp]),
    "rikfad_friction_report": (_st, [_vp, _i64, _i64, ctypes.c_double, _i32, _vp,
                                     _P(rikfad_friction_stats)]),
    "rikfad_friction_report_noalloc": (_st, [_vp, _i64, _i64, ctypes.c_double, _i32, _vp,
                                             _P(rikfad_friction_stats)]),
    "rikfad_friction_report_noalloc_max_bytes": (_i64, []),
    "rikfad_friction_report_workspace_bytes": (_i64, [_i64, _i64]),
    "adafm_create": (_st, [_vp, _i64, _P(adafm_hparams), _P(_vp)]),
    "adafm_step": (_st, [_vp, _vp]),
    "adafm_step_grads": (_st, [_vp, _vp, _vp]),
    "adafm_set_hparams": (_st, [_vp, _P(adafm_hparams)]),
    "adafm_set_step": (_st, [_vp, _i64]),
    "adafm_get_step": (_st, [_vp, _P(_i64)]),
    "adafm_min_bytes": (_st, [_vp, _P(_i64), _P(_i64), _P(_i64)]),
    "adafm_nonfinite": (_st, [_vp, _vp, _P(_i32)]),
    "adafm_timing_enable": (_st, [_vp, _i32]),
    "adafm_timing_read": (_st, [_vp, _P(ctypes.c_double), _P(_i64)]),
    "adafm_destroy": (None, [_vp]),
    "rikfad_probe_stream": (_st, [_vp, _vp, _vp, _vp, _vp, _i64, _vp]),
    "rikfad_probe_copy": (_st, [_vp, _vp, _i64, _vp]),
    "rikfad_probe_mix": (_st, [_vp, _vp, _vp, _i64, _i32, _i32, _vp]),
    "rikfad_probe_read": (_st, [_vp, _i64, _vp, _vp]),
    "rikfad_probe_write": (_st, [_vp, _i64, ctypes.c_uint32, _vp]),
}


def lib():
    """Load librikfad.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                               "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status, what):
    if status != RIKFAD_OK:
        raise RikfadError(status, what)


def rikfad_status_string(status):
    return lib().rikfad_status_string(int(status)).decode()


def rikfad_last_error():
    return lib().rikfad_last_error().decode()


def hparams(h, gamma=0.0, alpha=0.1, mu=1.0, eps_stab=1e-8):
    return rikfad_hparams(float(h), float(gamma), float(alpha), float(mu), float(eps_stab))


def _array(structs, cls):
    arr = (cls * max(1, len(structs)))()
    for i, s in enumerate(structs):
        arr[i] = s
    return arr


def rikfad_create(tensors, hp, flags=0):
    arr = _array(tensors, rikfad_tensor)
    ctx = ctypes.c_void_p()
    _check(lib().rikfad_create(ctypes.addressof(arr), len(tensors), ctypes.byref(hp),
                               int(flags), ctypes.byref(ctx)), "rikfad_create")
    return ctx


def rikfad_step(ctx, stream=None):
    _check(lib().rikfad_step(ctx, stream), "rikfad_step")


def rikfad_step_grads(ctx, grads, stream=None):
    arr = (ctypes.c_void_p * max(1, len(grads)))(*grads)
    _check(lib().rikfad_step_grads(ctx, ctypes.addressof(arr), stream), "rikfad_step_grads")


def rikfad_set_hparams(ctx, hp, stream=None):
    _check(lib().rikfad_set_hparams(ctx, ctypes.byref(hp), stream), "rikfad_set_hparams")


def rikfad_sync_momentum(ctx, stream=None):
    _check(lib().rikfad_sync_momentum(ctx, stream), "rikfad_sync_momentum")


def rikfad_state_changed(ctx):
    _check(lib().rikfad_state_changed(ctx), "rikfad_state_changed")


def rikfad_query(ctx):
    info = rikfad_info()
    _check(lib().rikfad_query(ctx, ctypes.byref(info)), "rikfad_query")
    return {nm: getattr(info, nm) for nm, _ in rikfad_info._fields_}


def rikfad_state_bytes(tensors):
    arr = _array(tensors, rikfad_tensor)
    a, b = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().rikfad_state_bytes(ctypes.addressof(arr), len(tensors), ctypes.byref(a),
                                    ctypes.byref(b)), "rikfad_state_bytes")
    return a.value, b.value


def rikfad_nonfinite(ctx, stream=None):
    v = ctypes.c_int32()
    _check(lib().rikfad_nonfinite(ctx, stream, ctypes.byref(v)), "rikfad_nonfinite")
    return bool(v.value)


def rikfad_timing_enable(ctx, enable=True):
    _check(lib().rikfad_timing_enable(ctx, int(bool(enable))), "rikfad_timing_enable")


def rikfad_timing_read(ctx):
    a, b, c = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().rikfad_timing_read(ctx, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c),
                                    ctypes.byref(n)), "rikfad_timing_read")
    return a.value, b.value, c.value, n.value


def rikfad_destroy(ctx):
    if ctx:
        lib().rikfad_destroy(ctx)


def ikfad_create(tensors, hp):
    arr = _array(tensors, ikfad_tensor)
    ctx = ctypes.c_void_p()
    _check(lib().ikfad_create(ctypes.addressof(arr), len(tensors), ctypes.byref(hp),
                              ctypes.byref(ctx)), "ikfad_create")
    return ctx


def ikfad_step(ctx, stream=None):
    _check(lib().ikfad_step(ctx, stream), "ikfad_step")


def ikfad_set_hparams(ctx, hp):
    _check(lib().ikfad_set_hparams(ctx, ctypes.byref(hp)), "ikfad_set_hparams")


def ikfad_timing_enable(ctx, enable=True):
    _check(lib().ikfad_timing_enable(ctx, int(bool(enable))), "ikfad_timing_enable")


def ikfad_timing_read(ctx):
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().ikfad_timing_read(ctx, ctypes.byref(ms), ctypes.byref(n)), "ikfad_timing_read")
    return ms.value, n.value


def ikfad_destroy(ctx):
    if ctx:
        lib().ikfad_destroy(ctx)


def rikfad_friction_report(xi, m, n, eps_stab=0.0, power_iters=60, stream=None):
    """Rank-1 friction statistics of an iKFAD friction tensor (device
    pointer, m x n fp32); blocking.  Returns a dict."""
    out = rikfad_friction_stats()
    _check(lib().rikfad_friction_report(xi, int(m), int(n), float(eps_stab), int(power_iters),
                                        stream, ctypes.byref(out)), "rikfad_friction_report")
    return {nm: getattr(out, nm) for nm, _ in rikfad_friction_stats._fields_}


def rikfad_friction_report_noalloc(xi, m, n, eps_stab=0.0, power_iters=60, stream=None):
    """rikfad_friction_report on the library's static device workspace (no
    device allocation); blocking.  Returns a dict."""
    out = rikfad_friction_stats()
    _check(lib().rikfad_friction_report_noalloc(xi, int(m), int(n), float(eps_stab),
                                                int(power_iters), stream, ctypes.byref(out)),
           "rikfad_friction_report_noalloc")
    return {nm: getattr(out, nm) for nm, _ in rikfad_friction_stats._fields_}


def rikfad_friction_report_noalloc_max_bytes():
    return int(lib().rikfad_friction_report_noalloc_max_bytes())


def rikfad_friction_report_workspace_bytes(m, n):
    return int(lib().rikfad_friction_report_workspace_bytes(int(m), int(n)))


def rikfad_probe_stream(a, b, c, d, e, nfloat, stream=None):
    _check(lib().rikfad_probe_stream(a, b, c, d, e, int(nfloat), stream), "rikfad_probe_stream")


def rikfad_probe_copy(src, dst, nbytes, stream=None):
    _check(lib().rikfad_probe_copy(src, dst, int(nbytes), stream), "rikfad_probe_copy")


def rikfad_probe_mix(x, g, p, nelem, dtype, shape, stream=None):
    _check(lib().rikfad_probe_mix(x, g, p, int(nelem), int(dtype), int(shape), stream),
           "rikfad_probe_mix")


def rikfad_probe_read(src, nbytes, out, stream=None):
    _check(lib().rikfad_probe_read(src, int(nbytes), out, stream), "rikfad_probe_read")


def rikfad_probe_write(dst, nbytes, value, stream=None):
    _check(lib().rikfad_probe_write(dst, int(nbytes), int(value) & 0xffffffff, stream),
           "rikfad_probe_write")


def adafm_params(h, beta1=0.9, decay_rate=-0.8, eps1=1e-30, eps2=1e-3, clip_threshold=1.0,
                 scale_parameter=False):
    return adafm_hparams(float(h), float(beta1), float(decay_rate), float(eps1), float(eps2),
                         float(clip_threshold), int(bool(scale_parameter)), 0)


def adafm_create(tensors, hp):
    arr = _array(tensors, rikfad_tensor)
    ctx = ctypes.c_void_p()
    _check(lib().adafm_create(ctypes.addressof(arr), len(tensors), ctypes.byref(hp),
                              ctypes.byref(ctx)), "adafm_create")
    return ctx


def adafm_step(ctx, stream=None):
    _check(lib().adafm_step(ctx, stream), "adafm_step")


def adafm_step_grads(ctx, grads, stream=None):
    arr = (ctypes.c_void_p * max(1, len(grads)))(*grads)
    _check(lib().adafm_step_grads(ctx, ctypes.addressof(arr), stream), "adafm_step_grads")


def adafm_set_hparams(ctx, hp):
    _check(lib().adafm_set_hparams(ctx, ctypes.byref(hp)), "adafm_set_hparams")


def adafm_set_step(ctx, steps_taken):
    _check(lib().adafm_set_step(ctx, int(steps_taken)), "adafm_set_step")


def adafm_get_step(ctx):
    v = ctypes.c_int64()
    _check(lib().adafm_get_step(ctx, ctypes.byref(v)), "adafm_get_step")
    return v.value


def adafm_min_bytes(ctx):
    """(bytes per step, bytes of the update pass, state bytes)."""
    a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(lib().adafm_min_bytes(ctx, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "adafm_min_bytes")
    return a.value, b.value, c.value


def adafm_nonfinite(ctx, stream=None):
    v = ctypes.c_int32()
    _check(lib().adafm_nonfinite(ctx, stream, ctypes.byref(v)), "adafm_nonfinite")
    return bool(v.value)


def adafm_timing_enable(ctx, enable=True):
    _check(lib().adafm_timing_enable(ctx, int(bool(enable))), "adafm_timing_enable")


def adafm_timing_read(ctx):
    """(ms of the statistics pass, finalisation, RMS pass, scale kernel,
    update pass) summed over the timed steps, and the step count."""
    ms = (ctypes.c_double * 5)()
    steps = ctypes.c_int64()
    _check(lib().adafm_timing_read(ctx, ms, ctypes.byref(steps)), "adafm_timing_read")
    return tuple(ms), steps.value


def adafm_destroy(ctx):
    if ctx:
        lib().adafm_destroy(ctx)


# ------------------------------------------------------------- torch glue

def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return RIKFAD_FP32
    if t.dtype == torch.bfloat16:
        return RIKFAD_BF16
    raise TypeError(f"unsupported parameter dtype {t.dtype}")


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _shape2(t):
    if t.dim() == 0:
        return 1, 1
    if t.dim() == 1:
        return 1, t.shape[0]
    return t.shape[0], t.numel() // t.shape[0]


def _check_pair(i, x, g):
    if not (x.is_cuda and g.is_cuda and x.is_contiguous() and g.is_contiguous()):
        raise ValueError(f"tensor {i}: parameters and gradients must be contiguous "
                         "device tensors")
    if g.dtype != x.dtype or g.numel() != x.numel() or g.device != x.device:
        raise ValueError(f"tensor {i}: gradient does not match its parameter")


def _check_state(i, x, tensors, sizes, names):
    """Caller-provided state: each a contiguous fp32 tensor on x's device with
    exactly the element count the kernels address (the C ABI sees only
    pointers, so a short or strided buffer would be read past its end)."""
    import torch
    for t, k, nm in zip(tensors, sizes, names):
        if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or t.device != x.device \
                or not t.is_contiguous() or t.numel() != k:
            raise ValueError(f"tensor {i}: state {nm} must be a contiguous fp32 tensor of {k} "
                             f"elements on {x.device}")


class RIKFAD:
    """R-iKFAD over a list of (parameter, gradient) torch tensors on one GPU.

    Parameters with more than two dimensions are viewed as (shape[0], rest),
    one-dimensional ones as 1 x n.  State p (m x n), r (m) and c (n) is
    allocated zero-filled in fp32; a vector keeps its friction in c (1 x n)
    or r (m x 1).  All work is enqueued on the given (or current) stream.
    """

    def __init__(self, params, grads, h, gamma=0.0, alpha=0.1, mu=1.0, eps_stab=1e-8,
                 two_pass=False, state=None):
        import torch
        self.params = list(params)
        self.grads = list(grads)
        self.state = []
        structs = []
        for i, (x, g) in enumerate(zip(self.params, self.grads)):
            _check_pair(i, x, g)
            m, n = _shape2(x)
            if state is not None:
                p, r, c = state[i]
                _check_state(i, x, (p, r, c), (m * n, m, n), ("p", "r", "c"))
            else:
                p = torch.zeros((m, n), device=x.device, dtype=torch.float32)
                r = torch.zeros(m, device=x.device, dtype=torch.float32)
                c = torch.zeros(n, device=x.device, dtype=torch.float32)
            self.state.append((p, r, c))
            structs.append(rikfad_tensor(x.data_ptr(), g.data_ptr(), p.data_ptr(),
                                         r.data_ptr(), c.data_ptr(), m, n, _dtype_code(x), 0))
        self.hp = hparams(h, gamma, alpha, mu, eps_stab)
        self.ctx = rikfad_create(structs, self.hp, RIKFAD_FLAG_TWO_PASS if two_pass else 0)

    def step(self, grads=None, stream=None):
        s = _stream_handle(stream)
        if grads is None:
            rikfad_step(self.ctx, s)
        else:
            self.grads = list(grads)
            rikfad_step_grads(self.ctx, [g.data_ptr() for g in self.grads], s)

    def sync_momentum(self, stream=None):
        rikfad_sync_momentum(self.ctx, _stream_handle(stream))

    def set_hparams(self, stream=None, **kw):
        cur = {nm: getattr(self.hp, nm) for nm, _ in rikfad_hparams._fields_}
        cur.update(kw)
        hp = hparams(**cur)
        rikfad_set_hparams(self.ctx, hp, _stream_handle(stream))
        self.hp = hp

    def state_changed(self):
        rikfad_state_changed(self.ctx)

    def query(self):
        return rikfad_query(self.ctx)

    def nonfinite(self, stream=None):
        return rikfad_nonfinite(self.ctx, _stream_handle(stream))

    def close(self):
        rikfad_destroy(self.ctx)
        self.ctx = None

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                self.close()
        except Exception:
            pass


class IKFAD:
    """Full-tensor iKFAD (comparison point) over (parameter, gradient) pairs."""

    def __init__(self, params, grads, h, gamma=0.0, alpha=0.1, mu=1.0):
        import torch
        self.params, self.grads, self.state = list(params), list(grads), []
        structs = []
        for i, (x, g) in enumerate(zip(self.params, self.grads)):
            _check_pair(i, x, g)
            m, n = _shape2(x)
            p = torch.zeros((m, n), device=x.device, dtype=torch.float32)
            xi = torch.zeros((m, n), device=x.device, dtype=torch.float32)
            self.state.append((p, xi))
            structs.append(ikfad_tensor(x.data_ptr(), g.data_ptr(), p.data_ptr(), xi.data_ptr(),
                                        m, n, _dtype_code(x), 0))
        self.ctx = ikfad_create(structs, hparams(h, gamma, alpha, mu, 0.0))

    def step(self, stream=None):
        ikfad_step(self.ctx, _stream_handle(stream))

    def nonfinite(self, stream=None):
        v = ctypes.c_int32()
        _check(lib().ikfad_nonfinite(self.ctx, _stream_handle(stream), ctypes.byref(v)),
               "ikfad_nonfinite")
        return bool(v.value)

    def close(self):
        ikfad_destroy(self.ctx)
        self.ctx = None

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                self.close()
        except Exception:
            pass


class ADAFM:
    """Adafactor-m (the paper's baseline) over (parameter, gradient) pairs.

    Same tensor conventions as ``RIKFAD``: state is the first moment
    (m x n fp32) and the second-moment factors r (m), c (n); a vector keeps
    its unfactored second moment in c (1 x n) or r (m x 1).
    """

    def __init__(self, params, grads, h, beta1=0.9, decay_rate=-0.8, eps1=1e-30, eps2=1e-3,
                 clip_threshold=1.0, scale_parameter=False, state=None):
        import torch
        self.params, self.grads, self.state = list(params), list(grads), []
        structs = []
        for i, (x, g) in enumerate(zip(self.params, self.grads)):
            _check_pair(i, x, g)
            m, n = _shape2(x)
            if state is not None:
                mom, r, c = state[i]
                _check_state(i, x, (mom, r, c), (m * n, m, n), ("first moment", "r", "c"))
            else:
                mom = torch.zeros((m, n), device=x.device, dtype=torch.float32)
                r = torch.zeros(m, device=x.device, dtype=torch.float32)
                c = torch.zeros(n, device=x.device, dtype=torch.float32)
            self.state.append((mom, r, c))
            structs.append(rikfad_tensor(x.data_ptr(), g.data_ptr(), mom.data_ptr(),
                                         r.data_ptr(), c.data_ptr(), m, n, _dtype_code(x), 0))
        self.hp = adafm_params(h, beta1, decay_rate, eps1, eps2, clip_threshold, scale_parameter)
        self.ctx = adafm_create(structs, self.hp)

    def step(self, grads=None, stream=None):
        s = _stream_handle(stream)
        if grads is None:
            adafm_step(self.ctx, s)
        else:
            self.grads = list(grads)
            adafm_step_grads(self.ctx, [g.data_ptr() for g in self.grads], s)

    @property
    def steps_taken(self):
        return adafm_get_step(self.ctx)

    def close(self):
        adafm_destroy(self.ctx)
        self.ctx = None

    def __del__(self):
        try:
            if getattr(self, "ctx", None):
                self.close()
        except Exception:
            pass
