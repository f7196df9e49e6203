"""Python binding of libfpsketch.so (the C ABI in include/fpsketch.h).

Argument marshalling only: every step of the verifier runs in the library's HIP kernels and host
code.  There is no CPU fallback; if the shared library is missing, loading raises.  Device
matrices are passed as torch tensors (their data pointers and the current HIP stream) or as raw
integer device pointers.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfpsketch.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "include", "fpsketch.h")

OK, EINVAL, EDTYPE, ESHAPE, ENOMEM, EHIP, ECAPACITY, ENODEV = range(8)
F16, BF16, F32 = 0, 1, 2
DTYPE_CODE = {"fp16": F16, "bf16": BF16, "f32": F32}


class FpsketchError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class Params(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("rounds", ctypes.c_int32), ("r_star", ctypes.c_int32),
                ("r_max", ctypes.c_int32), ("s_budget", ctypes.c_int32),
                ("delta_rc", ctypes.c_int32), ("k_cap", ctypes.c_int32),
                ("b_layout", ctypes.c_int32), ("rho_min", ctypes.c_double),
                ("mu", ctypes.c_double), ("c_valid", ctypes.c_double),
                ("b_star", ctypes.c_double), ("c_coll", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("law_cf_bf16", ctypes.c_double),
                ("law_cf_fp16", ctypes.c_double), ("law_n2_exp", ctypes.c_double)]


class Fault(ctypes.Structure):
    _fields_ = [("i", ctypes.c_int64), ("j", ctypes.c_int64), ("delta", ctypes.c_double),
                ("absolute", ctypes.c_int32), ("round", ctypes.c_int32)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("m", ctypes.c_int32), ("m_loc", ctypes.c_int32), ("r", ctypes.c_int32),
                ("fallback", ctypes.c_int32), ("n_abs", ctypes.c_int32),
                ("n_rechecked", ctypes.c_int32), ("sigma_hat", ctypes.c_double),
                ("rms_hat", ctypes.c_double), ("B", ctypes.c_double), ("tau", ctypes.c_double)]


_P = ctypes.c_void_p
_I32, _I64, _U64, _D = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double
_SIGS = {
    "fpsketch_default_params": (None, [ctypes.POINTER(Params)]),
    "fpsketch_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "fpsketch_last_error": (ctypes.c_char_p, []),
    "fpsketch_create": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, ctypes.POINTER(Params),
                                       ctypes.POINTER(_P)]),
    "fpsketch_destroy": (None, [_P]),
    "fpsketch_probe": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, _P, _P]),
    "fpsketch_localize": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, _U64, _I32,
                                         ctypes.POINTER(Fault), _I32, ctypes.POINTER(_I32), _P]),
    "fpsketch_cache_b": (ctypes.c_int, [_P, _P, _P]),
    "fpsketch_probe_cached": (ctypes.c_int, [_P, _P, _P, ctypes.c_int, _P, _P]),
    "fpsketch_probe_deferred": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, _P, _P]),
    "fpsketch_probe_noalloc": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, _P, _P]),
    "fpsketch_probe_flush": (ctypes.c_int, [_P, _P]),
    "fpsketch_probe_cached_deferred": (ctypes.c_int, [_P, _P, _P, ctypes.c_int, _P, _P]),
    "fpsketch_apply": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, ctypes.POINTER(Fault), _I32,
                                      _U64, ctypes.POINTER(_I32), _P]),
    "fpsketch_calibrate_noise": (ctypes.c_int, [_P, _P, ctypes.c_int, _P, ctypes.POINTER(_I32),
                                                ctypes.POINTER(_D), ctypes.POINTER(_I32)]),
    "fpsketch_get_plan": (ctypes.c_int, [_P, ctypes.POINTER(PlanInfo)]),
    "fpsketch_get_m": (ctypes.c_int, [_P, ctypes.POINTER(_I32)]),
    "fpsketch_probe_stats": (ctypes.c_int, [_P, ctypes.POINTER(_D), _P]),
    "fpsketch_sketch": (ctypes.c_int, [_P, _P, _P, _P, ctypes.c_int, _U64, _I32, _I32, _I32,
                                       ctypes.POINTER(_D), ctypes.POINTER(_D),
                                       ctypes.POINTER(_D), ctypes.POINTER(_D), _P]),
    "fpsketch_recheck": (ctypes.c_int, [_P, _P, _P, ctypes.POINTER(_I64), _I32,
                                        ctypes.POINTER(_D), ctypes.POINTER(_D), _P]),
    "fpsketch_timing": (ctypes.c_int, [_P, _I32]),
    "fpsketch_timing_read": (ctypes.c_int, [_P, ctypes.POINTER(_D), ctypes.POINTER(_D),
                                            ctypes.POINTER(_I64)]),
    "fpsketch_stream_read": (ctypes.c_int, [_P, _I64, _P, _I32, _P]),
    "fpsketch_stream_copy": (ctypes.c_int, [_P, _P, _I64, _I32, _P]),
    "fpsketch_hash_table": (ctypes.c_int, [_U64, _I32, _I32, _I64, _I32,
                                           ctypes.POINTER(_I32), ctypes.POINTER(ctypes.c_int8)]),
    "fpsketch_m_start": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, ctypes.POINTER(Params),
                                        ctypes.POINTER(_I32)]),
    "fpsketch_plan_host": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, _I32, _D, _D,
                                          ctypes.POINTER(Params), ctypes.POINTER(_I32),
                                          ctypes.POINTER(_I32), ctypes.POINTER(_D),
                                          ctypes.POINTER(_I32)]),
    "fpsketch_recalibrate_host": (ctypes.c_int, [_I64, _I64, _I32, _D, _D,
                                                 ctypes.POINTER(Params), ctypes.POINTER(_I32),
                                                 ctypes.POINTER(_I32)]),
    "fpsketch_rms_hat_samples": (_D, [ctypes.POINTER(ctypes.c_float), _I64]),
}

_lib = None


def header_symbols() -> list[str]:
    """Names of the functions include/fpsketch.h declares."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:[\w\*]+\s+)+\**(fpsketch_\w+)\s*\(", text, re.M)))


def load():
    """Load libfpsketch.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FpsketchError(-1, "load", f"{LIB_PATH} is missing; build it with "
                                        "__graft_entry__.build()")
    # torch carries its own HIP runtime.  Loaded before torch, this library bound a second runtime
    # whose calls found no device once torch had initialized its own; importing torch first makes
    # the library resolve its HIP dependency to the runtime torch already holds.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != OK:
        lib = load()
        detail = lib.fpsketch_last_error().decode() or lib.fpsketch_status_str(status).decode()
        raise FpsketchError(status, where, detail)


def default_params(**overrides) -> Params:
    p = Params()
    load().fpsketch_default_params(ctypes.byref(p))
    for k, v in overrides.items():
        if not hasattr(p, k):
            raise KeyError(k)
        setattr(p, k, v)
    return p


# ---- pointer helpers ---------------------------------------------------------------------

def _ptr(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if not x.is_contiguous():
        raise ValueError("matrices must be contiguous row-major")
    return int(x.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


def _check_tensor(x, what: str, shapes, dtypes, device: Optional[int]):
    """Raises ValueError unless the torch tensor x has one of `shapes` (or is 1-D with as many
    elements), a dtype in `dtypes` (None: any), is contiguous and lives on GPU `device` (None:
    any GPU).  None and raw integer device pointers pass unchecked: those are the caller's
    responsibility.  Checked before any call into the library, so that a wrong-sized buffer is
    never read or written out of bounds and a half matrix of the other format is not decoded as
    if it were the context's."""
    if x is None or isinstance(x, int):
        return
    shape = tuple(x.shape)
    if shape not in [tuple(s) for s in shapes] and not (
            x.dim() == 1 and any(x.numel() == int(np.prod(s)) for s in shapes)):
        raise ValueError(f"{what}: shape {shape}, expected "
                         f"{' or '.join(str(tuple(s)) for s in shapes)}")
    if dtypes is not None and x.dtype not in dtypes:
        raise ValueError(f"{what}: dtype {x.dtype}, expected "
                         f"{' or '.join(str(d) for d in dtypes)}")
    if not x.is_contiguous():
        raise ValueError(f"{what}: not contiguous (row-major without padding is required)")
    if not x.is_cuda:
        raise ValueError(f"{what}: on {x.device}, expected a GPU tensor")
    if device is not None and x.device.index != device:
        raise ValueError(f"{what}: on {x.device}, the context is on cuda:{device}")


def half_dtype(fmt: str):
    import torch
    return {"bf16": torch.bfloat16, "fp16": torch.float16}[fmt]


def check_operands(n1: int, n2: int, n3: int, fmt: str, b_layout: int, device: Optional[int],
                   A=None, B=None, C=None, d_dirty=None, c_float: bool = True):
    """Validates the operands of one call against a context's shape and format: A (n1 x n2) and B
    (n2 x n3, or W = B^T n3 x n2 with b_layout 1) in the context's half format, C (n1 x n3, and
    FP32 when c_float; otherwise its type code is passed on and checked by the library before it
    reads C), d_dirty an int32 flag; all contiguous and on the context's GPU."""
    import torch
    h = [half_dtype(fmt)]
    _check_tensor(A, "A", [(n1, n2)], h, device)
    _check_tensor(B, "W = B^T" if b_layout else "B", [(n3, n2) if b_layout else (n2, n3)], h,
                  device)
    _check_tensor(C, "C", [(n1, n3)], [torch.float32] if c_float else None, device)
    if d_dirty is not None and not isinstance(d_dirty, int):
        if d_dirty.dtype != torch.int32 or d_dirty.numel() < 1:
            raise ValueError(f"d_dirty: {d_dirty.dtype} with {d_dirty.numel()} elements, "
                             "expected at least one int32")
        _check_tensor(d_dirty, "d_dirty", [tuple(d_dirty.shape)], None, device)


def _c_dtype(C, c_dtype: Optional[int]) -> int:
    if c_dtype is not None:
        return c_dtype
    import torch
    return {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16}.get(C.dtype, -1)


# ---- host-only helpers (no GPU needed) ---------------------------------------------------

def hash_table(seed: int, rnd: int, side: int, n: int, m: int):
    b = np.empty(n, dtype=np.int32)
    s = np.empty(n, dtype=np.int8)
    _check(load().fpsketch_hash_table(seed, rnd, side, n, m,
                                      b.ctypes.data_as(ctypes.POINTER(_I32)),
                                      s.ctypes.data_as(ctypes.POINTER(ctypes.c_int8))),
           "fpsketch_hash_table")
    return b, s


def m_start(n1: int, n2: int, n3: int, fmt: str, params: Optional[Params] = None) -> int:
    out = _I32()
    _check(load().fpsketch_m_start(n1, n2, n3, DTYPE_CODE[fmt],
                                   ctypes.byref(params) if params else None, ctypes.byref(out)),
           "fpsketch_m_start")
    return out.value


def plan_host(n1, n2, n3, fmt, m, sigma_hat, rms, params: Optional[Params] = None):
    ml, r, B, fb = _I32(), _I32(), _D(), _I32()
    _check(load().fpsketch_plan_host(n1, n2, n3, DTYPE_CODE[fmt], m, sigma_hat, rms,
                                     ctypes.byref(params) if params else None, ctypes.byref(ml),
                                     ctypes.byref(r), ctypes.byref(B), ctypes.byref(fb)),
           "fpsketch_plan_host")
    return ml.value, r.value, B.value, bool(fb.value)


def recalibrate_host(n1, n3, m, sigma_bar, rms, params: Optional[Params] = None):
    mn, rb = _I32(), _I32()
    _check(load().fpsketch_recalibrate_host(n1, n3, m, sigma_bar, rms,
                                            ctypes.byref(params) if params else None,
                                            ctypes.byref(mn), ctypes.byref(rb)),
           "fpsketch_recalibrate_host")
    return mn.value, bool(rb.value)


def rms_hat_samples(samples: np.ndarray) -> float:
    s = np.ascontiguousarray(samples, dtype=np.float32)
    return float(load().fpsketch_rms_hat_samples(
        s.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), s.size))


def stream_read(src, nbytes: int, d_out, grid: int = 2048, stream=None):
    _check(load().fpsketch_stream_read(_ptr(src), nbytes, _ptr(d_out), grid, _stream(stream)),
           "fpsketch_stream_read")


def stream_copy(src, dst, nbytes: int, grid: int = 2048, stream=None):
    _check(load().fpsketch_stream_copy(_ptr(src), _ptr(dst), nbytes, grid, _stream(stream)),
           "fpsketch_stream_copy")


# ---- context -----------------------------------------------------------------------------

class Verifier:
    """One verifier context for products A (n1 x n2) x B (n2 x n3) in `fmt` on the current
    HIP device.  With b_layout=1 every call takes W = B^T (n3 x n2, a linear layer's weight,
    C = A W^T) where it takes B."""

    def __init__(self, n1: int, n2: int, n3: int, fmt: str, params: Optional[Params] = None,
                 **overrides):
        self.lib = load()
        self.n1, self.n2, self.n3, self.fmt = n1, n2, n3, fmt
        self.params = params if params is not None else default_params(**overrides)
        h = _P()
        _check(self.lib.fpsketch_create(n1, n2, n3, DTYPE_CODE[fmt], ctypes.byref(self.params),
                                        ctypes.byref(h)), "fpsketch_create")
        self.handle = h
        import torch
        self.device = torch.cuda.current_device()

    def _ops(self, A=None, B=None, C=None, d_dirty=None, c_dtype=None):
        # C's type code goes to the library, which rejects anything but FP32 before it reads C;
        # only a code of FP32 stated for a tensor of another type would make it read past C
        check_operands(self.n1, self.n2, self.n3, self.fmt, self.params.b_layout, self.device,
                       A, B, C, d_dirty, c_float=c_dtype == F32)

    def close(self):
        if getattr(self, "handle", None):
            self.lib.fpsketch_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def m(self) -> int:
        out = _I32()
        _check(self.lib.fpsketch_get_m(self.handle, ctypes.byref(out)), "fpsketch_get_m")
        return out.value

    def probe_status(self, A, B, C, d_dirty=None, stream=None, c_dtype=None) -> int:
        """Raw status of fpsketch_probe (used to test error paths)."""
        self._ops(A, B, C, d_dirty, c_dtype)
        return self.lib.fpsketch_probe(self.handle, _ptr(A), _ptr(B), _ptr(C),
                                       _c_dtype(C, c_dtype), _ptr(d_dirty), _stream(stream))

    def probe(self, A, B, C, d_dirty=None, stream=None, c_dtype=None):
        _check(self.probe_status(A, B, C, d_dirty, stream, c_dtype), "fpsketch_probe")

    def probe_noalloc_status(self, A, B, C, d_dirty=None, stream=None, c_dtype=None) -> int:
        """Raw status of fpsketch_probe_noalloc (the probe with the library's static scratch)."""
        self._ops(A, B, C, d_dirty, c_dtype)
        return self.lib.fpsketch_probe_noalloc(self.handle, _ptr(A), _ptr(B), _ptr(C),
                                               _c_dtype(C, c_dtype), _ptr(d_dirty),
                                               _stream(stream))

    def probe_noalloc(self, A, B, C, d_dirty=None, stream=None, c_dtype=None):
        _check(self.probe_noalloc_status(A, B, C, d_dirty, stream, c_dtype),
               "fpsketch_probe_noalloc")

    def probe_deferred(self, A, B, C, d_dirty=None, stream=None, c_dtype=None):
        """fpsketch_probe_deferred: the verdict is final after two more deferred calls or
        probe_flush."""
        self._ops(A, B, C, d_dirty, c_dtype)
        _check(self.lib.fpsketch_probe_deferred(self.handle, _ptr(A), _ptr(B), _ptr(C),
                                                _c_dtype(C, c_dtype), _ptr(d_dirty),
                                                _stream(stream)), "fpsketch_probe_deferred")

    def probe_cached_deferred(self, A, C, d_dirty=None, stream=None, c_dtype=None):
        """fpsketch_probe_cached_deferred (A and C streamed, verdict after the flush)."""
        self._ops(A, None, C, d_dirty, c_dtype)
        _check(self.lib.fpsketch_probe_cached_deferred(self.handle, _ptr(A), _ptr(C),
                                                       _c_dtype(C, c_dtype), _ptr(d_dirty),
                                                       _stream(stream)),
               "fpsketch_probe_cached_deferred")

    def probe_flush(self, stream=None):
        _check(self.lib.fpsketch_probe_flush(self.handle, _stream(stream)), "fpsketch_probe_flush")

    def cache_b(self, B, stream=None):
        """Forms and keeps the probe's B side (B H2^T and max|B|) for the current m."""
        self._ops(B=B)
        _check(self.lib.fpsketch_cache_b(self.handle, _ptr(B), _stream(stream)), "fpsketch_cache_b")

    def probe_cached_status(self, A, C, d_dirty=None, stream=None, c_dtype=None) -> int:
        self._ops(A, None, C, d_dirty, c_dtype)
        return self.lib.fpsketch_probe_cached(self.handle, _ptr(A), _ptr(C), _c_dtype(C, c_dtype),
                                              _ptr(d_dirty), _stream(stream))

    def probe_cached(self, A, C, d_dirty=None, stream=None, c_dtype=None):
        """fpsketch_probe with the cached B side (A and C streamed)."""
        _check(self.probe_cached_status(A, C, d_dirty, stream, c_dtype), "fpsketch_probe_cached")

    def probe_stats(self, stream=None) -> dict:
        out = (_D * 8)()
        _check(self.lib.fpsketch_probe_stats(self.handle, out, _stream(stream)),
               "fpsketch_probe_stats")
        keys = ["sigma_hat", "thr", "tau", "max_abs", "finite", "dirty", "max_a", "max_b"]
        return dict(zip(keys, list(out)))

    def localize(self, A, B, C, seed: int, sigma_from_probe: bool = False, cap: int = 4096,
                 stream=None, c_dtype=None):
        self._ops(A, B, C, None, c_dtype)
        buf = (Fault * max(cap, 1))()
        n = _I32()
        st = self.lib.fpsketch_localize(self.handle, _ptr(A), _ptr(B), _ptr(C),
                                        _c_dtype(C, c_dtype), seed, int(sigma_from_probe), buf,
                                        cap, ctypes.byref(n), _stream(stream))
        if st not in (OK, ECAPACITY):
            _check(st, "fpsketch_localize")
        recs = [(buf[t].i, buf[t].j, buf[t].delta, bool(buf[t].absolute), buf[t].round)
                for t in range(min(n.value, cap))]
        return recs, n.value, st

    def apply_status(self, A, B, C, recs, seed: int, stream=None, c_dtype=None):
        """Raw status and still-dirty flag of fpsketch_apply (records as localize returns them:
        (i, j, delta, absolute, round) tuples)."""
        self._ops(A, B, C, None, c_dtype)
        n = len(recs)
        buf = (Fault * max(n, 1))()
        for t, (i, j, d, ab, rnd) in enumerate(recs):
            buf[t].i, buf[t].j, buf[t].delta = int(i), int(j), float(d)
            buf[t].absolute, buf[t].round = int(bool(ab)), int(rnd)
        dirty = _I32()
        st = self.lib.fpsketch_apply(self.handle, _ptr(A), _ptr(B), _ptr(C), _c_dtype(C, c_dtype),
                                     buf, n, seed, ctypes.byref(dirty), _stream(stream))
        return st, bool(dirty.value)

    def apply(self, A, B, C, recs, seed: int, stream=None, c_dtype=None) -> bool:
        """Writes the records into C and re-probes with hash round 0 of `seed`; True when the
        re-probe still fires (the caller then recomputes C)."""
        st, dirty = self.apply_status(A, B, C, recs, seed, stream, c_dtype)
        _check(st, "fpsketch_apply")
        return dirty

    def timing(self, enable: bool):
        _check(self.lib.fpsketch_timing(self.handle, int(enable)), "fpsketch_timing")

    def timing_read(self):
        a, b, n = _D(), _D(), _I64()
        _check(self.lib.fpsketch_timing_read(self.handle, ctypes.byref(a), ctypes.byref(b),
                                             ctypes.byref(n)), "fpsketch_timing_read")
        return a.value, b.value, n.value

    def plan(self) -> dict:
        pi = PlanInfo()
        _check(self.lib.fpsketch_get_plan(self.handle, ctypes.byref(pi)), "fpsketch_get_plan")
        return {k: getattr(pi, k) for k, _ in PlanInfo._fields_}

    def calibrate_noise(self, C, stream=None, c_dtype=None):
        self._ops(C=C, c_dtype=c_dtype)
        m, sb, rb = _I32(), _D(), _I32()
        _check(self.lib.fpsketch_calibrate_noise(self.handle, _ptr(C), _c_dtype(C, c_dtype),
                                                 _stream(stream), ctypes.byref(m),
                                                 ctypes.byref(sb), ctypes.byref(rb)),
               "fpsketch_calibrate_noise")
        return m.value, sb.value, bool(rb.value)

    def sketch(self, A, B, C, seed: int, rnd: int, m: int, moments: bool = True, stream=None):
        self._ops(A, B, C)
        S = np.empty(m * m, dtype=np.float64)
        R = np.empty(m * m, dtype=np.float64)
        T = np.empty(m * m, dtype=np.float64)
        mx = np.empty(2, dtype=np.float64)
        dp = ctypes.POINTER(_D)
        _check(self.lib.fpsketch_sketch(self.handle, _ptr(A), _ptr(B), _ptr(C),
                                        _c_dtype(C, None), seed, rnd, m, int(moments),
                                        S.ctypes.data_as(dp), R.ctypes.data_as(dp),
                                        T.ctypes.data_as(dp), mx.ctypes.data_as(dp),
                                        _stream(stream)), "fpsketch_sketch")
        shape = (m, m)
        return (S.reshape(shape), R.reshape(shape) if moments else None,
                T.reshape(shape) if moments else None, float(mx[0]), float(mx[1]))

    def recheck(self, A, B, coords, stream=None):
        self._ops(A, B)
        cs = np.ascontiguousarray(np.asarray(coords, dtype=np.int64).reshape(-1, 2))
        n = cs.shape[0]
        g = np.empty(max(n, 1), dtype=np.float64)
        a = np.empty(max(n, 1), dtype=np.float64)
        dp = ctypes.POINTER(_D)
        _check(self.lib.fpsketch_recheck(self.handle, _ptr(A), _ptr(B),
                                         cs.ctypes.data_as(ctypes.POINTER(_I64)), n,
                                         g.ctypes.data_as(dp), a.ctypes.data_as(dp),
                                         _stream(stream)), "fpsketch_recheck")
        return g[:n], a[:n]
