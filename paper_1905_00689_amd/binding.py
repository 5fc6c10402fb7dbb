"""ctypes binding of libapprox_lstm.so, same names as the C ABI in
``include/approx_lstm.h``.  Argument marshalling only: every step of the
computation runs in the library (host factorisation in C++, the run in HIP
kernels).  Device arrays are torch tensors on a ROCm device; torch supplies
memory and streams and nothing else.  If the shared library is missing this
module raises at import time rather than falling back to anything.
"""

import ctypes
import os

import numpy as np
import torch  # noqa: F401  (loaded first so that its HIP runtime is the one in the process)

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libapprox_lstm.so")

OK = 0
ERR_INVALID_ARG = 1
ERR_OUT_OF_MEMORY = 2
ERR_DEVICE = 3
ERR_NOT_CONVERGED = 4
ERR_DEADLINE_INFEASIBLE = 5
ERR_UNSUPPORTED = 6
MAX_LEVELS = 16
FLAG_HOST_ONLY = 1 << 0
FLAG_KEEP_UNPRUNED = 1 << 1
FLAG_DEVICE_FACTORISE = 1 << 2
FLAG_NON_RESIDUAL = 1 << 3


class ApproxLstmError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"approx_lstm status {status}: {msg}")
        self.status = status


class PrepareParams(ctypes.Structure):
    _fields_ = [("input_size", ctypes.c_int32), ("hidden_size", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("nz", ctypes.c_int32),
                ("prune_ratio", ctypes.c_double), ("groups", ctypes.c_int32),
                ("factor_dtype", ctypes.c_int32), ("flags", ctypes.c_uint64)]


class Info(ctypes.Structure):
    _fields_ = [("input_size", ctypes.c_int32), ("hidden_size", ctypes.c_int32),
                ("aug_size", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("rows_per_group", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("nz", ctypes.c_int32), ("eff_rank", ctypes.c_int32 * 4),
                ("unconverged_steps", ctypes.c_int32), ("has_device_store", ctypes.c_int32),
                ("device_bytes", ctypes.c_uint64), ("factor_dtype", ctypes.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_1905_00689_amd.build`")
lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _f32p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_float)
_sigs = {
    "approx_lstm_prepare": [_vp, _vp, _vp, ctypes.POINTER(PrepareParams), _vp, ctypes.POINTER(_vp)],
    "approx_lstm_run": [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp],
    "approx_lstm_reserve": [_vp, _i32, _i32, _i32],
    "approx_lstm_run_stack": [_vp, _i32, _vp, _i32, _i32, _vp, _i32, _vp, _vp],
    "approx_lstm_run_deadline": [_vp, _vp, _i32, _i32, _vp, _vp, ctypes.c_double, _vp, _vp, _vp, _vp],
    "approx_lstm_run_anytime": [_vp, _vp, _i32, _i32, _vp, _vp, ctypes.c_double, _vp, _vp, _vp, _vp],
    "approx_lstm_run_schedule": [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp],
    "approx_lstm_run_noalloc": [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp],
    "approx_lstm_plan": [_vp, _i32, _i32, _vp, _i32, _i32, _i32, _vp],
    "approx_lstm_check": [_vp, _vp],
    "approx_lstm_set_launch": [_vp, _i32, _i32],
    "approx_lstm_set_batched_path": [_vp, _i32],
    "approx_lstm_set_recurrence": [_vp, _i32],
    "approx_lstm_model_info": [_vp, ctypes.POINTER(Info)],
    "approx_lstm_set_timing": [_vp, _i32],
    "approx_lstm_get_timing": [_vp, _vp, _vp, _i32],
    "approx_lstm_get_factors": [_vp, _i32, _vp, _vp, _vp, _vp],
    "approx_lstm_get_factors_f64": [_vp, _i32, _vp, _vp, _vp],
    "approx_lstm_exact_prepare": [_vp, _vp, _vp, _i32, _i32, _vp, ctypes.POINTER(_vp)],
    "approx_lstm_exact_run": [_vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _vp],
    "approx_lstm_exact_run_rows": [_vp, _vp, _i32, _i32, _vp, _vp, _i32, _vp, _vp, _vp],
    "approx_lstm_exact_check": [_vp, _vp],
    "approx_lstm_exact_set_launch": [_vp, _i32],
}
for _name, _args in _sigs.items():
    getattr(lib, _name).argtypes = _args
    getattr(lib, _name).restype = ctypes.c_int
lib.approx_lstm_destroy.argtypes = [_vp]
lib.approx_lstm_destroy.restype = None
lib.approx_lstm_exact_destroy.argtypes = [_vp]
lib.approx_lstm_exact_destroy.restype = None
lib.approx_lstm_last_error.argtypes = []
lib.approx_lstm_last_error.restype = ctypes.c_char_p


def _check(status, allow=()):
    if status != OK and status not in allow:
        raise ApproxLstmError(status, lib.approx_lstm_last_error().decode())
    return status


def _host(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def _dev(t, name, shape=None):
    """Device pointer of a float32 contiguous torch tensor (or None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a torch tensor on the GPU")
    if t.dtype != torch.float32 or not t.is_contiguous():
        raise TypeError(f"{name} must be contiguous float32")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return int(stream) if not hasattr(stream, "cuda_stream") else stream.cuda_stream


class Model:
    """Owning handle of an approx_lstm_model (destroyed with the object)."""

    def __init__(self, handle, status):
        self.handle = handle
        self.status = status
        self.hidden_size = approx_lstm_model_info(self)["hidden_size"]

    def __del__(self, _destroy=lib.approx_lstm_destroy):
        h, self.handle = getattr(self, "handle", None), None
        if h:
            _destroy(h)

    @property
    def info(self):
        return approx_lstm_model_info(self)


def approx_lstm_prepare(w_ih, w_hh, bias, input_size, hidden_size, rank, nz=0, prune_ratio=0.0,
                        groups=4, flags=0, factor_dtype=0, stream=0, allow_not_converged=True):
    """Host float32 arrays in; returns a Model.  stream: HIP stream handle (0 = default)."""
    H, D = hidden_size, input_size
    w_ih, p_ih = _host(w_ih, np.float32)
    w_hh, p_hh = _host(w_hh, np.float32)
    assert w_ih.shape == (4 * H, D) and w_hh.shape == (4 * H, H)
    p_b = None
    if bias is not None:
        bias, p_b = _host(bias, np.float32)
        assert bias.shape == (4 * H,)
    prm = PrepareParams(D, H, rank, nz, float(prune_ratio), groups, factor_dtype, flags)
    out = ctypes.c_void_p()
    st = lib.approx_lstm_prepare(p_ih, p_hh, p_b, ctypes.byref(prm), ctypes.c_void_p(stream or 0),
                                 ctypes.byref(out))
    _check(st, allow=(ERR_NOT_CONVERGED,) if allow_not_converged else ())
    return Model(out.value, st)


def approx_lstm_run(model, x, levels, h_out, h0=None, c0=None, c_out=None, stream=None):
    """x [T, B, D], h_out [L, T, B, H], c_out [L, B, H], h0/c0 [B, H]: GPU float32 tensors."""
    T, B, D = x.shape
    lv = (ctypes.c_int32 * len(levels))(*[int(k) for k in levels])
    H = model.hidden_size
    st = lib.approx_lstm_run(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)), _dev(c0, "c0", (B, H)),
                             lv, len(levels), _dev(h_out, "h_out", (len(levels), T, B, H)),
                             _dev(c_out, "c_out", (len(levels), B, H)), ctypes.c_void_p(_stream(stream)))
    return _check(st)


def approx_lstm_run_noalloc(model, x, levels, h_out, h0=None, c0=None, c_out=None, stream=None):
    """As approx_lstm_run, with the workspace in the library's static device
    scratch (no allocation in the call)."""
    T, B, D = x.shape
    lv = (ctypes.c_int32 * len(levels))(*[int(k) for k in levels])
    H = model.hidden_size
    st = lib.approx_lstm_run_noalloc(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)),
                                     _dev(c0, "c0", (B, H)), lv, len(levels),
                                     _dev(h_out, "h_out", (len(levels), T, B, H)),
                                     _dev(c_out, "c_out", (len(levels), B, H)), ctypes.c_void_p(_stream(stream)))
    return _check(st)


def approx_lstm_run_deadline(model, x, deadline_us, h_out, h0=None, c0=None, stream=None):
    """x [T, B, D], h_out [T, B, H] GPU float32.  Returns (k_achieved [T], step_us [T]) numpy arrays."""
    T, B, D = x.shape
    H = model.hidden_size
    k = np.zeros(T, np.int32)
    us = np.zeros(T, np.float32)
    st = lib.approx_lstm_run_deadline(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)), _dev(c0, "c0", (B, H)),
                                      float(deadline_us), _dev(h_out, "h_out", (T, B, H)), k.ctypes.data,
                                      us.ctypes.data, ctypes.c_void_p(_stream(stream)))
    _check(st)
    return k, us



def approx_lstm_run_anytime(model, x, deadline_us, h_out, h0=None, c0=None, stream=None):
    """Budget chosen per timestep on the device.  x [T, B, D], h_out [T, B, H]
    GPU float32.  Returns (k_achieved [T], step_us [T]) numpy arrays."""
    T, B, D = x.shape
    H = model.hidden_size
    k = np.zeros(T, np.int32)
    us = np.zeros(T, np.float32)
    st = lib.approx_lstm_run_anytime(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)), _dev(c0, "c0", (B, H)),
                                     float(deadline_us), _dev(h_out, "h_out", (T, B, H)), k.ctypes.data,
                                     us.ctypes.data, ctypes.c_void_p(_stream(stream)))
    _check(st)
    return k, us

def approx_lstm_run_schedule(model, x, k_sched, h_out, h0=None, c0=None, c_out=None, stream=None):
    """Budget K_t given per timestep (host ints, length T).  x [T, B, D],
    h_out [T, B, H], c_out [B, H] or None, GPU float32."""
    T, B, D = x.shape
    H = model.hidden_size
    ks, kp = _host(k_sched, np.int32)
    if ks.shape != (T,):
        raise ValueError(f"k_sched has shape {ks.shape}, expected ({T},)")
    st = lib.approx_lstm_run_schedule(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)),
                                      _dev(c0, "c0", (B, H)), kp, _dev(h_out, "h_out", (T, B, H)),
                                      _dev(c_out, "c_out", (B, H)), ctypes.c_void_p(_stream(stream)))
    return _check(st)


PLAN_FIELDS = ("blocks", "px_all", "allpairs", "hpl", "upt", "opt", "bulk_h", "lds_bytes", "pair_kernel",
               "ktile")


def approx_lstm_plan(model, T, B, levels=None, online=0, num_cu=0):
    """Launch plan of an fp32 run (no device work): dict of PLAN_FIELDS."""
    lv = levels if levels is not None else [0]
    arr, ap = _host(lv, np.int32)
    out = np.zeros(len(PLAN_FIELDS), np.int32)
    _check(lib.approx_lstm_plan(model.handle, T, B, ap, len(arr), int(online), int(num_cu), out.ctypes.data))
    return dict(zip(PLAN_FIELDS, (int(v) for v in out)))


def approx_lstm_run_stack(models, x, levels, h_out, stream=None):
    """models: list of Model; x [T, B, D0]; levels: [n_levels][n_layers] ints;
    h_out [n_levels, T, B, H_last] GPU float32 tensor."""
    T, B, D = x.shape
    nl, L = len(models), len(levels)
    arr = (ctypes.c_void_p * nl)(*[m.handle for m in models])
    flat = [int(k) for row in levels for k in row]
    assert len(flat) == nl * L
    lv = (ctypes.c_int32 * len(flat))(*flat)
    H = models[-1].hidden_size
    st = lib.approx_lstm_run_stack(arr, nl, _dev(x, "x"), T, B, lv, L, _dev(h_out, "h_out", (L, T, B, H)),
                                   ctypes.c_void_p(_stream(stream)))
    return _check(st)


def approx_lstm_reserve(model, T_max, B_max, L_max):
    return _check(lib.approx_lstm_reserve(model.handle, T_max, B_max, L_max))


def approx_lstm_check(model, stream=None):
    return _check(lib.approx_lstm_check(model.handle, ctypes.c_void_p(_stream(stream))))


def approx_lstm_set_launch(model, blocks, cooperative=0):
    return _check(lib.approx_lstm_set_launch(model.handle, int(blocks), int(cooperative)))


def approx_lstm_set_recurrence(model, kernel):
    return _check(lib.approx_lstm_set_recurrence(model.handle, int(kernel)))


def approx_lstm_set_batched_path(model, persistent):
    return _check(lib.approx_lstm_set_batched_path(model.handle, int(persistent)))


def approx_lstm_set_timing(model, enable):
    return _check(lib.approx_lstm_set_timing(model.handle, int(enable)))


def approx_lstm_get_timing(model, T, stream=None):
    """Stamps of the last timed run, microseconds: array [2 + 4T]."""
    out = np.zeros(2 + 4 * T)
    _check(lib.approx_lstm_get_timing(model.handle, ctypes.c_void_p(_stream(stream)), out.ctypes.data, out.size))
    return out


def approx_lstm_model_info(model):
    inf = Info()
    _check(lib.approx_lstm_model_info(model.handle, ctypes.byref(inf)))
    d = {name: getattr(inf, name) for name, _ in Info._fields_}
    d["eff_rank"] = list(inf.eff_rank)[: inf.groups]
    return d


def approx_lstm_get_factors(model, group):
    """Group `group`'s terms as stored (fp32): sigma [N], u [N, R_g], v_idx [N, NZ], v_val [N, NZ]."""
    inf = approx_lstm_model_info(model)
    N, Rg, nz = inf["rank"], inf["rows_per_group"], inf["nz"]
    sigma = np.empty(N, np.float32)
    u = np.empty((N, Rg), np.float32)
    vi = np.empty((N, nz), np.int32)
    vv = np.empty((N, nz), np.float32)
    _check(lib.approx_lstm_get_factors(model.handle, group, sigma.ctypes.data, u.ctypes.data,
                                       vi.ctypes.data, vv.ctypes.data))
    return dict(sigma=sigma, u=u, v_idx=vi, v_val=vv)


def approx_lstm_get_factors_f64(model, group):
    inf = approx_lstm_model_info(model)
    N, Rg, C = inf["rank"], inf["rows_per_group"], inf["aug_size"]
    sigma = np.empty(N)
    u = np.empty((N, Rg))
    v = np.empty((N, C))
    _check(lib.approx_lstm_get_factors_f64(model.handle, group, sigma.ctypes.data, u.ctypes.data,
                                           v.ctypes.data))
    return dict(sigma=sigma, u=u, v=v)


def approx_lstm_last_error():
    return lib.approx_lstm_last_error().decode()


class ExactModel:
    """Owning handle of an approx_lstm_exact (the dense baseline)."""

    def __init__(self, handle, hidden_size):
        self.handle = handle
        self.hidden_size = hidden_size

    def __del__(self, _destroy=lib.approx_lstm_exact_destroy):
        h, self.handle = getattr(self, "handle", None), None
        if h:
            _destroy(h)


def approx_lstm_exact_prepare(w_ih, w_hh, bias, input_size, hidden_size, stream=0):
    """Host float32 weights in (gate rows i, f, g, o); returns an ExactModel."""
    H, D = hidden_size, input_size
    w_ih, p_ih = _host(w_ih, np.float32)
    w_hh, p_hh = _host(w_hh, np.float32)
    assert w_ih.shape == (4 * H, D) and w_hh.shape == (4 * H, H)
    p_b = None
    if bias is not None:
        bias, p_b = _host(bias, np.float32)
        assert bias.shape == (4 * H,)
    out = ctypes.c_void_p()
    _check(lib.approx_lstm_exact_prepare(p_ih, p_hh, p_b, D, H, ctypes.c_void_p(stream or 0), ctypes.byref(out)))
    return ExactModel(out.value, H)


def approx_lstm_exact_run(model, x, h_out, h0=None, c0=None, c_out=None, stream=None):
    """x [T, B, D], h_out [T, B, H], c_out [B, H], h0/c0 [B, H]: GPU float32 tensors."""
    T, B, D = x.shape
    H = model.hidden_size
    st = lib.approx_lstm_exact_run(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)), _dev(c0, "c0", (B, H)),
                                   _dev(h_out, "h_out", (T, B, H)), _dev(c_out, "c_out", (B, H)),
                                   ctypes.c_void_p(_stream(stream)))
    return _check(st)


def approx_lstm_exact_run_rows(model, x, rows, h_out, h0=None, c0=None, c_out=None, stream=None):
    """The exact recurrence stopped after `rows` rows of every gate (the
    row-tile anytime baseline); tensors as for approx_lstm_exact_run."""
    T, B, D = x.shape
    H = model.hidden_size
    st = lib.approx_lstm_exact_run_rows(model.handle, _dev(x, "x"), T, B, _dev(h0, "h0", (B, H)),
                                        _dev(c0, "c0", (B, H)), int(rows), _dev(h_out, "h_out", (T, B, H)),
                                        _dev(c_out, "c_out", (B, H)), ctypes.c_void_p(_stream(stream)))
    return _check(st)


def approx_lstm_exact_check(model, stream=None):
    return _check(lib.approx_lstm_exact_check(model.handle, ctypes.c_void_p(_stream(stream))))


def approx_lstm_exact_set_launch(model, blocks):
    return _check(lib.approx_lstm_exact_set_launch(model.handle, int(blocks)))
