"""CPU oracle for the fused depthwise/pointwise convolution modules -- TEST INFRASTRUCTURE.

Plain, slow, obviously correct reference of what every module computes (arXiv
2404.19331, Sec. II-B for the DW/PW definitions, Sec. III for the modules and their
per-stage convolution-normalisation-activation). The arithmetic lives in
``fcm_oracle.c`` (nested loops, exact accumulation); this module only builds it with
gcc, marshals numpy arrays through ctypes and returns numpy arrays.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package. It shares no code with the HIP library.

Array conventions (storage formats):
  f32  -> numpy float32          bf16 -> numpy uint16 (raw bfloat16 bits)
  i8   -> numpy int8             f64  -> numpy float64 (oracle-only exact mode)
Biases: float32 for f32/bf16, float64 for f64, int32 for i8; ``None`` means zero.
Weights: depthwise [C, K, K], pointwise [C_out, C_in] (row-major, contiguous).
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fcm_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libfcm_oracle.so")

DTYPES = {"f32": 0, "bf16": 1, "i8": 2, "f64": 3}
LAYOUTS = {"nchw": 0, "nhwc": 1}
ACTS = {"none": 0, "relu": 1, "relu6": 2}
STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported", 3: "int32 accumulator overflow"}
_NP = {"f32": np.float32, "bf16": np.uint16, "i8": np.int8, "f64": np.float64}


class OracleError(RuntimeError):
    pass


class _Rq(ctypes.Structure):
    _fields_ = [("mult", ctypes.c_int32), ("shift", ctypes.c_int32),
                ("qmin", ctypes.c_int32), ("qmax", ctypes.c_int32), ("zero_point", ctypes.c_int32)]


class _Desc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_mid", ctypes.c_int32), ("c_out", ctypes.c_int32),
                ("k", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("act", ctypes.c_int32 * 3), ("rq", _Rq * 3),
                ("rqc", ctypes.POINTER(ctypes.c_int32) * 3), ("zp_in", ctypes.c_int32)]


def build(force=False):
    """Compile fcm_oracle.c with gcc (-O2, OpenMP, no BLAS, no intrinsics)."""
    if (not force and os.path.exists(_LIB_PATH)
            and os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC)):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall",
                    "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib_handle = None


def _lib():
    global _lib_handle
    if _lib_handle is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        vp = ctypes.c_void_p
        dp = ctypes.POINTER(_Desc)
        lib.orc_dw.argtypes = [dp, vp, vp, vp, vp]
        lib.orc_pw.argtypes = [dp, vp, vp, vp, vp]
        lib.orc_dw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp]
        lib.orc_pw_dw.argtypes = [dp, vp, vp, vp, vp, vp, vp]
        lib.orc_pw_dw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp]
        lib.orc_pw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp]
        for f in (lib.orc_dw, lib.orc_pw, lib.orc_dw_pw, lib.orc_pw_dw, lib.orc_pw_dw_pw, lib.orc_pw_pw):
            f.restype = ctypes.c_int
        lib.orc_requant.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32]
        lib.orc_requant.restype = ctypes.c_int64
        lib.orc_bf16_from_f32.argtypes = [ctypes.c_float]
        lib.orc_bf16_from_f32.restype = ctypes.c_uint16
        lib.orc_f32_from_bf16.argtypes = [ctypes.c_uint16]
        lib.orc_f32_from_bf16.restype = ctypes.c_float
        lib.orc_num_threads.restype = ctypes.c_int
        lib.orc_set_num_threads.argtypes = [ctypes.c_int]
        lib.orc_set_num_threads.restype = None
        _lib_handle = lib
    return _lib_handle


def _get(case, key, default=None):
    if isinstance(case, dict):
        return case.get(key, default)
    return getattr(case, key, default)


def _desc(case):
    d = _Desc()
    for f in ("n", "h", "w", "k", "stride", "pad"):
        setattr(d, f, int(_get(case, f, 1 if f in ("k", "stride") else 0)))
    d.c_in = int(_get(case, "c_in"))
    d.c_mid = int(_get(case, "c_mid", d.c_in) or d.c_in)
    d.c_out = int(_get(case, "c_out", d.c_mid) or d.c_mid)
    d.dtype = DTYPES[_get(case, "dtype")]
    d.layout = LAYOUTS[_get(case, "layout")]
    acts = list(_get(case, "act", ("none",) * 3))
    acts = (acts + ["none"] * 3)[:3]
    for i, a in enumerate(acts):
        d.act[i] = ACTS[a] if isinstance(a, str) else int(a)
    rqs = list(_get(case, "rq", ()) or ())
    rqs = (rqs + [(1, 0, -128, 127)] * 3)[:3]
    for i, r in enumerate(rqs):
        # (mult, shift, qmin, qmax[, zero point of the stage's output])
        r = tuple(r) + (0,) * (5 - len(r))
        d.rq[i].mult, d.rq[i].shift, d.rq[i].qmin, d.rq[i].qmax, d.rq[i].zero_point = (int(v) for v in r)
    d.zp_in = int(_get(case, "zp_in", 0) or 0)  # int8 zero point of the input
    # int8 per-channel requantisation: rq_channel[i] = (multipliers, shifts) of stage i's
    # output channels, or None for the per-tensor rq[i]
    d._keep = []
    for i, pc in enumerate(list(_get(case, "rq_channel", None) or [None] * 3)[:3]):
        if pc is None:
            continue
        a = np.ascontiguousarray(np.concatenate([np.asarray(pc[0]), np.asarray(pc[1])]).astype(np.int32))
        d._keep.append(a)
        d.rqc[i] = a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    return d


def out_hw(h, w, k, stride, pad):
    """Output spatial size of a KxK convolution with symmetric zero padding."""
    return (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1


def _shape(layout, n, c, h, w):
    return (n, c, h, w) if layout == "nchw" else (n, h, w, c)


def _arr(a, dtype_name):
    if a is None:
        return None
    want = _NP[dtype_name]
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError("expected %s array for dtype %s, got %s" % (want, dtype_name, a.dtype))
    return a


def _bias(b, dtype_name):
    if b is None:
        return None
    want = {"f32": np.float32, "bf16": np.float32, "i8": np.int32, "f64": np.float64}[dtype_name]
    b = np.ascontiguousarray(b)
    if b.dtype != want:
        raise TypeError("expected %s bias for dtype %s, got %s" % (want, dtype_name, b.dtype))
    return b


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(st):
    if st != 0:
        raise OracleError("oracle returned %d (%s)" % (st, STATUS.get(st, "?")))


def dw(case, x, w_dw, b_dw=None):
    """Single depthwise layer (stage 0 activation / requantisation)."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    ho, wo = out_hw(d.h, d.w, d.k, d.stride, d.pad)
    x, w_dw, b_dw = _arr(x, dt), _arr(w_dw, dt), _bias(b_dw, dt)
    y = np.empty(_shape(lay, d.n, d.c_in, ho, wo), dtype=_NP[dt])
    _check(_lib().orc_dw(ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(y)))
    return y


def pw(case, x, w_pw, b_pw=None):
    """Single pointwise layer c_in -> c_out (stage 0 activation / requantisation)."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    x, w_pw, b_pw = _arr(x, dt), _arr(w_pw, dt), _bias(b_pw, dt)
    y = np.empty(_shape(lay, d.n, d.c_out, d.h, d.w), dtype=_NP[dt])
    _check(_lib().orc_pw(ctypes.byref(d), _ptr(x), _ptr(w_pw), _ptr(b_pw), _ptr(y)))
    return y


def dw_pw(case, x, w_dw, b_dw, w_pw, b_pw):
    """Depthwise separable convolution DW -> PW."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    ho, wo = out_hw(d.h, d.w, d.k, d.stride, d.pad)
    x, w_dw, w_pw = _arr(x, dt), _arr(w_dw, dt), _arr(w_pw, dt)
    b_dw, b_pw = _bias(b_dw, dt), _bias(b_pw, dt)
    y = np.empty(_shape(lay, d.n, d.c_out, ho, wo), dtype=_NP[dt])
    _check(_lib().orc_dw_pw(ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(w_pw),
                            _ptr(b_pw), _ptr(y)))
    return y


def pw_dw(case, x, w_pw, b_pw, w_dw, b_dw):
    """PW -> DW (output has c_mid channels)."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    ho, wo = out_hw(d.h, d.w, d.k, d.stride, d.pad)
    x, w_pw, w_dw = _arr(x, dt), _arr(w_pw, dt), _arr(w_dw, dt)
    b_pw, b_dw = _bias(b_pw, dt), _bias(b_dw, dt)
    y = np.empty(_shape(lay, d.n, d.c_mid, ho, wo), dtype=_NP[dt])
    _check(_lib().orc_pw_dw(ctypes.byref(d), _ptr(x), _ptr(w_pw), _ptr(b_pw), _ptr(w_dw),
                            _ptr(b_dw), _ptr(y)))
    return y


def pw_dw_pw(case, x, w_pw1, b_pw1, w_dw, b_dw, w_pw2, b_pw2):
    """Inverted residual PW -> DW -> PW (no skip connection)."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    ho, wo = out_hw(d.h, d.w, d.k, d.stride, d.pad)
    x, w_pw1, w_dw, w_pw2 = (_arr(a, dt) for a in (x, w_pw1, w_dw, w_pw2))
    b_pw1, b_dw, b_pw2 = (_bias(b, dt) for b in (b_pw1, b_dw, b_pw2))
    y = np.empty(_shape(lay, d.n, d.c_out, ho, wo), dtype=_NP[dt])
    _check(_lib().orc_pw_dw_pw(ctypes.byref(d), _ptr(x), _ptr(w_pw1), _ptr(b_pw1), _ptr(w_dw),
                               _ptr(b_dw), _ptr(w_pw2), _ptr(b_pw2), _ptr(y)))
    return y


def pw_pw(case, x, w_pw1, b_pw1, w_pw2, b_pw2):
    """Two pointwise layers c_in -> c_mid -> c_out (spatial size unchanged)."""
    dt, lay = _get(case, "dtype"), _get(case, "layout")
    d = _desc(case)
    x, w_pw1, w_pw2 = (_arr(a, dt) for a in (x, w_pw1, w_pw2))
    b_pw1, b_pw2 = (_bias(b, dt) for b in (b_pw1, b_pw2))
    y = np.empty(_shape(lay, d.n, d.c_out, d.h, d.w), dtype=_NP[dt])
    _check(_lib().orc_pw_pw(ctypes.byref(d), _ptr(x), _ptr(w_pw1), _ptr(b_pw1), _ptr(w_pw2), _ptr(b_pw2),
                            _ptr(y)))
    return y


def run(op, case, inputs):
    """Dispatch by module name with the inputs dict produced by the seeded generators."""
    g = inputs.get
    if op == "dw_pw":
        return dw_pw(case, g("x"), g("w_dw"), g("b_dw"), g("w_pw"), g("b_pw"))
    if op == "pw_dw":
        return pw_dw(case, g("x"), g("w_pw"), g("b_pw"), g("w_dw"), g("b_dw"))
    if op == "pw_dw_pw":
        return pw_dw_pw(case, g("x"), g("w_pw1"), g("b_pw1"), g("w_dw"), g("b_dw"),
                        g("w_pw2"), g("b_pw2"))
    if op == "pw_pw":
        return pw_pw(case, g("x"), g("w_pw1"), g("b_pw1"), g("w_pw2"), g("b_pw2"))
    if op == "dw":
        return dw(case, g("x"), g("w_dw"), g("b_dw"))
    if op == "pw":
        return pw(case, g("x"), g("w_pw"), g("b_pw"))
    raise ValueError("unknown module %r" % (op,))


def requant(acc, mult, shift, qmin=-128, qmax=127):
    """Integer requantisation: round-half-to-even(acc*mult/2^shift), saturated."""
    return int(_lib().orc_requant(int(acc), int(mult), int(shift), int(qmin), int(qmax)))


def bf16_bits(f):
    """Round a float32 value to bfloat16 (nearest, ties to even); returns the bits."""
    return int(_lib().orc_bf16_from_f32(float(np.float32(f))))


def bf16_value(bits):
    return float(_lib().orc_f32_from_bf16(int(bits)))


def num_threads():
    """Threads the oracle's OpenMP loops use (OMP_NUM_THREADS or all cores)."""
    return int(_lib().orc_num_threads())


def set_num_threads(n):
    """Threads of the oracle's OpenMP loops from now on in this thread (timing only)."""
    _lib().orc_set_num_threads(int(n))
