"""ctypes binding of libfcm.so (argument marshalling only).

Every computation happens in the HIP kernels behind the C ABI (include/fcm.h). PyTorch
provides device memory and the current stream; this module checks tensors, fills the
descriptor, allocates the output tensor with torch when none is given, and calls the
library. There is no fallback: if libfcm.so is missing or cannot load, importing the
binding's functions raises.

Entry points mirror the C ABI: dw_pw, pw_dw, pw_pw, pw_dw_pw, dw, pw, plan, plan_evaluate,
chain_desc, chain_plan, chain_run, fold_batchnorm.
Tensors: x is [n, c, h, w] (layout="nchw") or [n, h, w, c] (layout="nhwc");
depthwise weights [c, k, k] (or [c, 1, k, k]); pointwise weights [c_out, c_in]
(or [c_out, c_in, 1, 1]); biases float32 (float paths) or int32 (int8) or None.
dtype follows x: float32, bfloat16, int8.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libfcm.so")

OP = {"dw_pw": 0, "pw_dw": 1, "pw_dw_pw": 2, "dw": 3, "pw": 4, "pw_pw": 5}
DTYPE = {"f32": 0, "bf16": 1, "i8": 2}
LAYOUT = {"nchw": 0, "nhwc": 1}
ACT = {"none": 0, "relu": 1, "relu6": 2}
STATUS = {0: "FCM_OK", 1: "FCM_EINVAL", 2: "FCM_EUNSUPPORTED", 3: "FCM_EDEVICE"}


class FcmError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS.get(status, status), msg))
        self.status = status


class Requant(ctypes.Structure):
    _fields_ = [("mult", ctypes.c_int32), ("shift", ctypes.c_int32),
                ("qmin", ctypes.c_int32), ("qmax", ctypes.c_int32), ("zero_point", ctypes.c_int32)]

    def set(self, r):
        """(mult, shift, qmin, qmax[, zero point of the stage's output])."""
        r = tuple(int(v) for v in r) + (0,) * (5 - len(r))
        self.mult, self.shift, self.qmin, self.qmax, self.zero_point = r


class Desc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c_in", ctypes.c_int32), ("c_mid", ctypes.c_int32), ("c_out", ctypes.c_int32),
                ("k", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32),
                ("act", ctypes.c_int32 * 3), ("rq", Requant * 3), ("rq_channel", ctypes.c_void_p * 3),
                ("zp_in", ctypes.c_int32)]


class HwDesc(ctypes.Structure):
    _fields_ = [("num_cus", ctypes.c_int32), ("num_xcds", ctypes.c_int32),
                ("wave_size", ctypes.c_int32), ("lds_per_wg", ctypes.c_int32),
                ("lds_per_cu", ctypes.c_int32), ("l2_per_xcd", ctypes.c_int64),
                ("mall_bytes", ctypes.c_int64), ("hbm_bytes_per_s", ctypes.c_double)]


class Plan(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("tile_h", ctypes.c_int32), ("tile_w", ctypes.c_int32),
                ("c_block", ctypes.c_int32), ("co_block", ctypes.c_int32),
                ("variant", ctypes.c_int32), ("waves", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("workgroups", ctypes.c_int32),
                ("fuse", ctypes.c_int32), ("depth", ctypes.c_int32), ("splits", ctypes.c_int32),
                ("bytes_ideal", ctypes.c_int64), ("bytes_tiled", ctypes.c_int64),
                ("bytes_paper", ctypes.c_int64), ("bytes_lbl_paper", ctypes.c_int64),
                ("bytes_lbl_ideal", ctypes.c_int64), ("redundancy", ctypes.c_double)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


CHAIN_MAX_LAYERS = 128
LAYER_KIND = {"dw": 0, "pw": 1}
OBJECTIVE = {"bytes": 0, "time": 1, "unfused": 2}


class Layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("c_out", ctypes.c_int32), ("k", ctypes.c_int32),
                ("stride", ctypes.c_int32), ("pad", ctypes.c_int32), ("act", ctypes.c_int32), ("rq", Requant)]


class ChainDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32), ("c", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("layout", ctypes.c_int32), ("zp_in", ctypes.c_int32),
                ("num_layers", ctypes.c_int32), ("layers", Layer * CHAIN_MAX_LAYERS)]


class ChainPlan(ctypes.Structure):
    _fields_ = [("objective", ctypes.c_int32), ("num_groups", ctypes.c_int32),
                ("first", ctypes.c_int32 * CHAIN_MAX_LAYERS), ("op", ctypes.c_int32 * CHAIN_MAX_LAYERS),
                ("plan", Plan * CHAIN_MAX_LAYERS), ("fused_layers", ctypes.c_int32),
                ("act_bytes_max", ctypes.c_int64), ("bytes_paper", ctypes.c_int64),
                ("bytes_lbl_paper", ctypes.c_int64), ("time_est", ctypes.c_double),
                ("time_lbl_est", ctypes.c_double)]

    def groups(self):
        """[(first layer, op name, Plan)] of the chain's kernels in order."""
        names = {v: k for k, v in OP.items()}
        return [(self.first[g], names[self.op[g]], self.plan[g]) for g in range(self.num_groups)]


_lib = None


def lib():
    """Load libfcm.so (raises if it has not been built).

    torch is imported first: its ROCm build carries its own HIP and HSA runtimes, and
    libfcm.so must bind to those already-loaded copies. Loaded the other way round, the
    process ends up with two HIP runtimes, and the one libfcm.so uses finds no device
    once torch's has opened it."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FcmError(-1, "libfcm.so not found at %s; build it with "
                               "`python -m paper_2404_19331_amd.build`" % LIB_PATH)
        import torch  # noqa: F401  (see above)
        L = ctypes.CDLL(LIB_PATH)
        vp, dp, pp = ctypes.c_void_p, ctypes.POINTER(Desc), ctypes.POINTER(Plan)
        hp = ctypes.POINTER(HwDesc)
        L.fcm_plan.argtypes = [ctypes.c_int32, dp, hp, pp]
        L.fcm_plan_evaluate.argtypes = [dp, hp, pp]
        L.fcm_dw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp, pp, vp]
        L.fcm_pw_dw.argtypes = [dp, vp, vp, vp, vp, vp, vp, pp, vp]
        L.fcm_pw_dw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, pp, vp]
        L.fcm_pw_pw.argtypes = [dp, vp, vp, vp, vp, vp, vp, pp, vp]
        L.fcm_dw.argtypes = [dp, vp, vp, vp, vp, pp, vp]
        L.fcm_pw.argtypes = [dp, vp, vp, vp, vp, pp, vp]
        i64 = ctypes.c_int64
        L.fcm_dw_pw_ws.argtypes = [dp, vp, vp, vp, vp, vp, vp, pp, vp, i64, vp]
        L.fcm_pw_ws.argtypes = [dp, vp, vp, vp, vp, pp, vp, i64, vp]
        L.fcm_dw_pw_ws.restype = L.fcm_pw_ws.restype = ctypes.c_int
        L.fcm_workspace_bytes.argtypes = [dp, pp]
        L.fcm_dw_pw_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, pp, vp]
        L.fcm_dw_pw_noalloc.restype = ctypes.c_int
        L.fcm_plan_limited.argtypes = [ctypes.c_int32, dp, hp, i64, pp]
        L.fcm_plan_limited.restype = ctypes.c_int
        L.fcm_plan_candidates.argtypes = [ctypes.c_int32, dp, hp, i64, pp, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]
        L.fcm_plan_candidates.restype = ctypes.c_int
        L.fcm_workspace_bytes.restype = i64
        for f in (L.fcm_plan, L.fcm_plan_evaluate, L.fcm_dw_pw, L.fcm_pw_dw, L.fcm_pw_dw_pw,
                  L.fcm_pw_pw, L.fcm_dw, L.fcm_pw):
            f.restype = ctypes.c_int
        L.fcm_status_string.argtypes = [ctypes.c_int]
        L.fcm_status_string.restype = ctypes.c_char_p
        L.fcm_last_error.restype = ctypes.c_char_p
        L.fcm_version.restype = ctypes.c_char_p
        L.fcm_variant_name.argtypes = [ctypes.c_int32]
        L.fcm_variant_name.restype = ctypes.c_char_p
        L.fcm_variant_count.restype = ctypes.c_int32
        cdp, cpp = ctypes.POINTER(ChainDesc), ctypes.POINTER(ChainPlan)
        L.fcm_chain_plan.argtypes = [cdp, ctypes.c_int32, hp, cpp]
        L.fcm_chain_plan.restype = ctypes.c_int
        L.fcm_chain_workspace_bytes.argtypes = [cpp]
        L.fcm_chain_workspace_bytes.restype = ctypes.c_int64
        L.fcm_chain_run.argtypes = [cdp, cpp, vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp, vp]
        L.fcm_chain_run.restype = ctypes.c_int
        fp = ctypes.POINTER(ctypes.c_float)
        L.fcm_fold_batchnorm.argtypes = [ctypes.c_int32, ctypes.c_int32, fp, fp, fp, fp, fp, fp, ctypes.c_float, fp, fp]
        L.fcm_fold_batchnorm.restype = ctypes.c_int
        L.fcm_plan_time_estimate.argtypes = [dp, hp, pp]
        L.fcm_plan_time_estimate.restype = ctypes.c_double
        _lib = L
    return _lib


def variant_name(v):
    n = lib().fcm_variant_name(int(v))
    return None if n is None else n.decode()


def last_error():
    return lib().fcm_last_error().decode()


def _check(st):
    if st != 0:
        raise FcmError(st, last_error())


def make_desc(n, h, w, c_in, c_mid, c_out, k=3, stride=1, pad=1, dtype="f32", layout="nchw",
              act=("none", "none", "none"), rq=None, rq_channel=None, zp_in=0):
    """rq: per stage (mult, shift, qmin, qmax[, output zero point]); zp_in: int8 zero point
    of the input (the code of real 0)."""
    d = Desc()
    d.n, d.h, d.w = n, h, w
    d.c_in, d.c_mid, d.c_out = c_in, c_mid, c_out
    d.k, d.stride, d.pad = k, stride, pad
    d.dtype = DTYPE[dtype] if isinstance(dtype, str) else int(dtype)
    d.layout = LAYOUT[layout] if isinstance(layout, str) else int(layout)
    acts = (list(act) + ["none"] * 3)[:3]
    for i, a in enumerate(acts):
        d.act[i] = ACT[a] if isinstance(a, str) else int(a)
    rqs = (list(rq or []) + [(1, 0, -128, 127)] * 3)[:3]
    for i, r in enumerate(rqs):
        d.rq[i].set(r)
    d.zp_in = int(zp_in)
    # int8 per-channel requantisation: device int32 tensors [2 * channels] per stage or None
    d._keep = []
    for i, t in enumerate(list(rq_channel or [])[:3]):
        if t is None:
            continue
        if not (t.is_cuda and t.dtype == _torch().int32 and t.is_contiguous()):
            raise ValueError("rq_channel entries must be contiguous int32 device tensors")
        d.rq_channel[i] = t.data_ptr()
        d._keep.append(t)
    return d


def desc_from_case(case):
    """Descriptor from a workloads.Case (or any object/dict with the same fields)."""
    g = (lambda k: case[k]) if isinstance(case, dict) else (lambda k: getattr(case, k))
    zp = case.get("zp_in", 0) if isinstance(case, dict) else getattr(case, "zp_in", 0)
    return make_desc(g("n"), g("h"), g("w"), g("c_in"), g("c_mid"), g("c_out"), g("k"), g("stride"),
                     g("pad"), g("dtype"), g("layout"), g("act"), g("rq"), zp_in=zp or 0)


def plan(op, desc, hw=None):
    """FusePlanner: the tiling fcm_plan chooses, as a dict."""
    p = Plan()
    _check(lib().fcm_plan(OP[op], ctypes.byref(desc), ctypes.byref(hw) if hw else None, ctypes.byref(p)))
    return p


_find_plan = plan  # (the entry points' `plan` argument shadows the function)


def plan_limited(op, desc, max_workspace_bytes, hw=None):
    """The planner's best plan among those needing at most `max_workspace_bytes` of
    caller workspace (0: none)."""
    p = Plan()
    _check(lib().fcm_plan_limited(OP[op], ctypes.byref(desc), ctypes.byref(hw) if hw else None,
                                  int(max_workspace_bytes), ctypes.byref(p)))
    return p


def plan_candidates(op, desc, max_count=12, max_workspace_bytes=0, hw=None):
    """The planner's candidate plans, its own choice first (fcm_plan_candidates)."""
    arr = (Plan * max_count)()
    n = ctypes.c_int32(0)
    _check(lib().fcm_plan_candidates(OP[op], ctypes.byref(desc), ctypes.byref(hw) if hw else None,
                                     int(max_workspace_bytes), arr, max_count, ctypes.byref(n)))
    return [arr[i] for i in range(n.value)]


def plan_time_estimate(desc, plan, hw=None):
    """Seconds the planner's time model gives the plan's launch (0.0 on error)."""
    return lib().fcm_plan_time_estimate(ctypes.byref(desc), ctypes.byref(hw) if hw else None, ctypes.byref(plan))


def plan_evaluate(op, desc, tile_h, tile_w, c_block, co_block, variant, hw=None, workgroups=0, depth=0, splits=0):
    """Evaluate a caller-chosen tiling. For the persistent kernels `workgroups` > 0 caps
    the number of workgroups launched, `depth` > 0 sets the LDS ring depth and
    `splits` > 1 splits each work tile's channel chunks over that many workgroups."""
    p = Plan()
    p.op, p.tile_h, p.tile_w, p.c_block, p.co_block, p.variant = OP[op], tile_h, tile_w, c_block, co_block, variant
    p.workgroups = workgroups
    p.depth = depth
    p.splits = splits
    _check(lib().fcm_plan_evaluate(ctypes.byref(desc), ctypes.byref(hw) if hw else None, ctypes.byref(p)))
    return p


# ------------------------------------------------------------------------------------
# torch-facing entry points
# ------------------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_name(t):
    torch = _torch()
    m = {torch.float32: "f32", torch.bfloat16: "bf16", torch.int8: "i8"}
    if t.dtype not in m:
        raise TypeError("unsupported dtype %s (float32, bfloat16, int8)" % t.dtype)
    return m[t.dtype]


def _dims(x, layout):
    if x.dim() != 4:
        raise ValueError("x must be 4-D")
    if layout == "nchw":
        n, c, h, w = x.shape
    else:
        n, h, w, c = x.shape
    return int(n), int(c), int(h), int(w)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _prep(x, tensors, biases, dt):
    torch = _torch()
    if not x.is_cuda:
        raise ValueError("tensors must be on a GPU device")
    for t in tensors:
        if t is None:
            raise ValueError("weights must not be None")
        if t.device != x.device or t.dtype != x.dtype:
            raise ValueError("weights must match x in device and dtype")
        if not t.is_contiguous():
            raise ValueError("weights must be contiguous")
    bdt = torch.int32 if dt == "i8" else torch.float32
    for b in biases:
        if b is not None and (b.device != x.device or b.dtype != bdt or not b.is_contiguous()):
            raise ValueError("bias must be a contiguous %s tensor on x's device" % bdt)
    if not x.is_contiguous():
        raise ValueError("x must be contiguous in its layout")


def _out(x, layout, n, c, h, w, out):
    torch = _torch()
    shape = (n, c, h, w) if layout == "nchw" else (n, h, w, c)
    if out is None:
        return torch.empty(shape, dtype=x.dtype, device=x.device)
    if tuple(out.shape) != shape or out.dtype != x.dtype or out.device != x.device or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of shape %s" % (x.dtype, shape))
    return out


def _stream(x, stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class Prepared:
    """A C-ABI launch whose arguments were marshalled once; calling it launches again
    (same tensors, same plan, same stream). Used for repeated timed launches. `keep`
    holds tensors the launch uses that the caller did not pass (a split plan's workspace)."""

    def __init__(self, fn, args, y, keep=None):
        self.fn, self.args, self.y, self.keep = fn, args, y, keep

    def __call__(self):
        st = self.fn(*self.args)
        if st != 0:
            raise FcmError(st, last_error())
        return self.y


def _call(fn, args, y, prepare, keep=None):
    if prepare:
        return Prepared(fn, args, y, keep)
    _check(fn(*args))
    return y


def workspace_bytes(desc, plan):
    """Device bytes of workspace `plan` needs (0 unless it splits channel chunks)."""
    n = lib().fcm_workspace_bytes(ctypes.byref(desc), ctypes.byref(plan))
    if n < 0:
        raise FcmError(1, last_error())
    return int(n)


def _with_workspace(op, d, x, plan, workspace):
    """The plan to launch (the planner's best when None) and the workspace it needs: the
    caller's tensor, or a fresh one from torch's allocator (the library allocates nothing)."""
    if plan is None:
        plan = _find_plan(op, d)
    need = workspace_bytes(d, plan)
    if need == 0:
        return plan, None
    torch = _torch()
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    elif workspace.numel() * workspace.element_size() < need or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous device tensor of at least %d bytes" % need)
    return plan, workspace


def _plan_arg(plan):
    return ctypes.byref(plan) if plan is not None else None


def out_hw(h, w, k, stride, pad):
    return (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1


def _kk(w_dw):
    return int(w_dw.shape[-1])


def dw_pw(x, w_dw, w_pw, b_dw=None, b_pw=None, *, stride=1, pad=None, act=("none", "none"), rq=None, rq_channel=None,
          layout="nchw", plan=None, out=None, stream=None, prepare=False, zp_in=0, workspace=None):
    """DW -> PW module in one kernel. Returns y [n, c_out, h_o, w_o] in `layout`.
    A plan that splits channel chunks (the planner's choice when `plan` is None) runs with
    `workspace`, or with a device tensor allocated here through torch."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    k = _kk(w_dw)
    pad = (k - 1) // 2 if pad is None else pad
    co = int(w_pw.shape[0])
    _prep(x, [w_dw, w_pw], [b_dw, b_pw], dt)
    d = make_desc(n, h, w, c, c, co, k, stride, pad, dt, layout, act, rq, rq_channel=rq_channel, zp_in=zp_in)
    ho, wo = out_hw(h, w, k, stride, pad)
    y = _out(x, layout, n, co, ho, wo, out)
    plan, ws = _with_workspace("dw_pw", d, x, plan, workspace)
    if ws is None:
        return _call(lib().fcm_dw_pw, (ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(w_pw), _ptr(b_pw),
                                       _ptr(y), _plan_arg(plan), _stream(x, stream)), y, prepare)
    return _call(lib().fcm_dw_pw_ws, (ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(w_pw), _ptr(b_pw),
                                      _ptr(y), _plan_arg(plan), _ptr(ws), ws.numel() * ws.element_size(),
                                      _stream(x, stream)), y, prepare, keep=ws)


NOALLOC_SCRATCH_BYTES = 16 << 20  # FCM_NOALLOC_SCRATCH_BYTES


def dw_pw_noalloc(x, w_dw, w_pw, b_dw=None, b_pw=None, *, stride=1, pad=None, act=("none", "none"), rq=None,
                  rq_channel=None, layout="nchw", plan=None, out=None, stream=None, zp_in=0):
    """DW -> PW module through fcm_dw_pw_noalloc: a split plan's partial sums go to the
    library's fixed per-GPU array instead of a workspace (pass `out` to allocate nothing
    here either). Calls overlapping on one GPU race on that array."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    k = _kk(w_dw)
    pad = (k - 1) // 2 if pad is None else pad
    co = int(w_pw.shape[0])
    _prep(x, [w_dw, w_pw], [b_dw, b_pw], dt)
    d = make_desc(n, h, w, c, c, co, k, stride, pad, dt, layout, act, rq, rq_channel=rq_channel, zp_in=zp_in)
    ho, wo = out_hw(h, w, k, stride, pad)
    y = _out(x, layout, n, co, ho, wo, out)
    return _call(lib().fcm_dw_pw_noalloc, (ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(w_pw), _ptr(b_pw),
                                           _ptr(y), _plan_arg(plan), _stream(x, stream)), y, False)


def pw_dw(x, w_pw, w_dw, b_pw=None, b_dw=None, *, stride=1, pad=None, act=("none", "none"), rq=None, rq_channel=None,
          layout="nchw", plan=None, out=None, stream=None, prepare=False, zp_in=0):
    """PW -> DW module in one kernel. Returns y [n, c_mid, h_o, w_o]."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    k = _kk(w_dw)
    pad = (k - 1) // 2 if pad is None else pad
    cm = int(w_pw.shape[0])
    _prep(x, [w_pw, w_dw], [b_pw, b_dw], dt)
    d = make_desc(n, h, w, c, cm, cm, k, stride, pad, dt, layout, act, rq, rq_channel=rq_channel, zp_in=zp_in)
    ho, wo = out_hw(h, w, k, stride, pad)
    y = _out(x, layout, n, cm, ho, wo, out)
    return _call(lib().fcm_pw_dw, (ctypes.byref(d), _ptr(x), _ptr(w_pw), _ptr(b_pw), _ptr(w_dw), _ptr(b_dw),
                                   _ptr(y), _plan_arg(plan), _stream(x, stream)), y, prepare)


def pw_dw_pw(x, w_pw1, w_dw, w_pw2, b_pw1=None, b_dw=None, b_pw2=None, *, stride=1, pad=None,
             act=("none", "none", "none"), rq=None, rq_channel=None, layout="nchw", plan=None, out=None, stream=None,
             prepare=False, zp_in=0):
    """PW -> DW -> PW inverted residual in one kernel. Returns y [n, c_out, h_o, w_o]."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    k = _kk(w_dw)
    pad = (k - 1) // 2 if pad is None else pad
    cm, co = int(w_pw1.shape[0]), int(w_pw2.shape[0])
    _prep(x, [w_pw1, w_dw, w_pw2], [b_pw1, b_dw, b_pw2], dt)
    d = make_desc(n, h, w, c, cm, co, k, stride, pad, dt, layout, act, rq, rq_channel=rq_channel, zp_in=zp_in)
    ho, wo = out_hw(h, w, k, stride, pad)
    y = _out(x, layout, n, co, ho, wo, out)
    return _call(lib().fcm_pw_dw_pw, (ctypes.byref(d), _ptr(x), _ptr(w_pw1), _ptr(b_pw1), _ptr(w_dw), _ptr(b_dw),
                                      _ptr(w_pw2), _ptr(b_pw2), _ptr(y), _plan_arg(plan), _stream(x, stream)),
                 y, prepare)


def pw_pw(x, w_pw1, w_pw2, b_pw1=None, b_pw2=None, *, act=("none", "none"), rq=None, rq_channel=None, layout="nchw", plan=None,
          out=None, stream=None, prepare=False, zp_in=0):
    """PW -> PW module in one kernel. Returns y [n, c_out, h, w]."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    cm, co = int(w_pw1.shape[0]), int(w_pw2.shape[0])
    _prep(x, [w_pw1, w_pw2], [b_pw1, b_pw2], dt)
    d = make_desc(n, h, w, c, cm, co, 1, 1, 0, dt, layout, act, rq, rq_channel=rq_channel, zp_in=zp_in)
    y = _out(x, layout, n, co, h, w, out)
    return _call(lib().fcm_pw_pw, (ctypes.byref(d), _ptr(x), _ptr(w_pw1), _ptr(b_pw1), _ptr(w_pw2), _ptr(b_pw2),
                                   _ptr(y), _plan_arg(plan), _stream(x, stream)), y, prepare)


def dw(x, w_dw, b_dw=None, *, stride=1, pad=None, act="none", rq=None, rq_channel=None, layout="nchw", plan=None, out=None,
       stream=None, prepare=False, zp_in=0):
    """Single depthwise layer (layer-by-layer kernel)."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    k = _kk(w_dw)
    pad = (k - 1) // 2 if pad is None else pad
    _prep(x, [w_dw], [b_dw], dt)
    d = make_desc(n, h, w, c, c, c, k, stride, pad, dt, layout, (act,), [rq] if rq else None, rq_channel=rq_channel, zp_in=zp_in)
    ho, wo = out_hw(h, w, k, stride, pad)
    y = _out(x, layout, n, c, ho, wo, out)
    return _call(lib().fcm_dw, (ctypes.byref(d), _ptr(x), _ptr(w_dw), _ptr(b_dw), _ptr(y), _plan_arg(plan),
                                _stream(x, stream)), y, prepare)


def pw(x, w_pw, b_pw=None, *, act="none", rq=None, rq_channel=None, layout="nchw", plan=None, out=None, stream=None,
       prepare=False, zp_in=0, workspace=None):
    """Single pointwise layer (layer-by-layer kernel); split plans as in dw_pw."""
    dt = _dtype_name(x)
    n, c, h, w = _dims(x, layout)
    co = int(w_pw.shape[0])
    _prep(x, [w_pw], [b_pw], dt)
    d = make_desc(n, h, w, c, c, co, 1, 1, 0, dt, layout, (act,), [rq] if rq else None, rq_channel=rq_channel, zp_in=zp_in)
    y = _out(x, layout, n, co, h, w, out)
    plan, ws = _with_workspace("pw", d, x, plan, workspace)
    if ws is None:
        return _call(lib().fcm_pw, (ctypes.byref(d), _ptr(x), _ptr(w_pw), _ptr(b_pw), _ptr(y), _plan_arg(plan),
                                    _stream(x, stream)), y, prepare)
    return _call(lib().fcm_pw_ws, (ctypes.byref(d), _ptr(x), _ptr(w_pw), _ptr(b_pw), _ptr(y), _plan_arg(plan),
                                   _ptr(ws), ws.numel() * ws.element_size(), _stream(x, stream)), y, prepare, keep=ws)


# ------------------------------------------------------------------------------------
# Layer-by-layer chains (the unfused comparison): each layer is its own kernel and every
# intermediate feature map goes through device memory.
# ------------------------------------------------------------------------------------

class _Chain:
    """Several prepared launches issued in order (a layer-by-layer chain)."""

    def __init__(self, calls):
        self.calls = calls
        self.y = calls[-1].y

    def __call__(self):
        for c in self.calls:
            c()
        return self.y


def _zp_out(r):
    """Output zero point of an int8 stage's (mult, shift, qmin, qmax[, zero point])."""
    return int(r[4]) if r is not None and len(r) > 4 else 0


def dw_then_pw(x, w_dw, w_pw, b_dw=None, b_pw=None, *, stride=1, pad=None, act=("none", "none"), rq=None,
               layout="nchw", mid=None, out=None, stream=None, prepare=False, zp_in=0, plans=(None, None),
               workspace=None):
    """DW then PW as two kernels (the intermediate through device memory); `plans` are
    the stages' plans (None: the planner's), `workspace` the PW stage's (split plans)."""
    rq = list(rq) if rq else [None, None]
    c1 = dw(x, w_dw, b_dw, stride=stride, pad=pad, act=act[0], rq=rq[0], layout=layout, out=mid, stream=stream,
            prepare=prepare, zp_in=zp_in, plan=plans[0])
    m = c1.y if prepare else c1
    c2 = pw(m, w_pw, b_pw, act=act[1], rq=rq[1], layout=layout, out=out, stream=stream, prepare=prepare,
            zp_in=_zp_out(rq[0]), plan=plans[1], workspace=workspace)
    return _Chain([c1, c2]) if prepare else c2


def pw_then_dw(x, w_pw, w_dw, b_pw=None, b_dw=None, *, stride=1, pad=None, act=("none", "none"), rq=None,
               layout="nchw", mid=None, out=None, stream=None, prepare=False, zp_in=0, plans=(None, None),
               workspace=None):
    rq = list(rq) if rq else [None, None]
    c1 = pw(x, w_pw, b_pw, act=act[0], rq=rq[0], layout=layout, out=mid, stream=stream, prepare=prepare,
            zp_in=zp_in, plan=plans[0], workspace=workspace)
    m = c1.y if prepare else c1
    c2 = dw(m, w_dw, b_dw, stride=stride, pad=pad, act=act[1], rq=rq[1], layout=layout, out=out, stream=stream,
            prepare=prepare, zp_in=_zp_out(rq[0]), plan=plans[1])
    return _Chain([c1, c2]) if prepare else c2


def pw_then_pw(x, w_pw1, w_pw2, b_pw1=None, b_pw2=None, *, act=("none", "none"), rq=None, layout="nchw",
               mid=None, out=None, stream=None, prepare=False, zp_in=0, plans=(None, None), workspace=None):
    rq = list(rq) if rq else [None, None]
    c1 = pw(x, w_pw1, b_pw1, act=act[0], rq=rq[0], layout=layout, out=mid, stream=stream, prepare=prepare,
            zp_in=zp_in, plan=plans[0], workspace=workspace)
    m = c1.y if prepare else c1
    c2 = pw(m, w_pw2, b_pw2, act=act[1], rq=rq[1], layout=layout, out=out, stream=stream, prepare=prepare,
            zp_in=_zp_out(rq[0]), plan=plans[1], workspace=workspace)
    return _Chain([c1, c2]) if prepare else c2


def pw_then_dw_then_pw(x, w_pw1, w_dw, w_pw2, b_pw1=None, b_dw=None, b_pw2=None, *, stride=1, pad=None,
                       act=("none", "none", "none"), rq=None, layout="nchw", mids=(None, None), out=None,
                       stream=None, prepare=False, zp_in=0, plans=(None, None, None), workspace=None):
    rq = list(rq) if rq else [None, None, None]
    c1 = pw(x, w_pw1, b_pw1, act=act[0], rq=rq[0], layout=layout, out=mids[0], stream=stream, prepare=prepare,
            zp_in=zp_in, plan=plans[0], workspace=workspace)
    m1 = c1.y if prepare else c1
    c2 = dw(m1, w_dw, b_dw, stride=stride, pad=pad, act=act[1], rq=rq[1], layout=layout, out=mids[1],
            stream=stream, prepare=prepare, zp_in=_zp_out(rq[0]), plan=plans[1])
    m2 = c2.y if prepare else c2
    c3 = pw(m2, w_pw2, b_pw2, act=act[2], rq=rq[2], layout=layout, out=out, stream=stream, prepare=prepare,
            zp_in=_zp_out(rq[1]), plan=plans[2], workspace=workspace)
    return _Chain([c1, c2, c3]) if prepare else c3


# ------------------------------------------------------------------------------------
# Chains of layers (FusePlanner over a network): plan once, run every group's kernel
# ------------------------------------------------------------------------------------

def chain_desc(n, h, w, c, layers, dtype="i8", layout="nhwc", zp_in=0):
    """Chain descriptor. layers: dicts with kind ("dw" | "pw"), c_out (PW), k, stride,
    pad (DW), act ("none" | "relu" | "relu6"), rq ((mult, shift, qmin, qmax[, output
    zero point]), int8). zp_in: int8 zero point of the chain input."""
    if not 1 <= len(layers) <= CHAIN_MAX_LAYERS:
        raise ValueError("a chain has 1 .. %d layers" % CHAIN_MAX_LAYERS)
    d = ChainDesc()
    d.n, d.h, d.w, d.c = n, h, w, c
    d.dtype = DTYPE[dtype] if isinstance(dtype, str) else int(dtype)
    d.layout = LAYOUT[layout] if isinstance(layout, str) else int(layout)
    d.zp_in = int(zp_in)
    d.num_layers = len(layers)
    for i, L in enumerate(layers):
        t = d.layers[i]
        t.kind = LAYER_KIND[L["kind"]]
        t.c_out = int(L.get("c_out", 0))
        t.k, t.stride, t.pad = int(L.get("k", 1)), int(L.get("stride", 1)), int(L.get("pad", 0))
        a = L.get("act", "none")
        t.act = ACT[a] if isinstance(a, str) else int(a)
        t.rq.set(L.get("rq") or (1, 0, -128, 127))
    return d


def chain_plan(desc, objective="bytes", hw=None):
    p = ChainPlan()
    _check(lib().fcm_chain_plan(ctypes.byref(desc), OBJECTIVE[objective], ctypes.byref(hw) if hw else None,
                                ctypes.byref(p)))
    return p


def chain_output_shape(desc):
    h, w, c = desc.h, desc.w, desc.c
    for i in range(desc.num_layers):
        L = desc.layers[i]
        if L.kind == LAYER_KIND["pw"]:
            c = L.c_out
        else:
            h, w = out_hw(h, w, L.k, L.stride, L.pad)
    return (desc.n, c, h, w) if desc.layout == LAYOUT["nchw"] else (desc.n, h, w, c)


class _ChainRun(Prepared):
    def __init__(self, fn, args, y, keep):
        super().__init__(fn, args, y)
        self.keep = keep  # the pointer arrays and workspace the arguments refer to


def chain_run(desc, plan, x, weights, biases=None, *, out=None, workspace=None, stream=None, prepare=False):
    """Run a planned chain: x the input tensor, weights/biases per layer (biases may be
    None or hold None). The inter-group workspace is a torch allocation unless given."""
    torch = _torch()
    if len(weights) != desc.num_layers:
        raise ValueError("one weight tensor per layer")
    biases = list(biases) if biases is not None else [None] * desc.num_layers
    _prep(x, weights, biases, _dtype_name(x))
    shape = chain_output_shape(desc)
    y = torch.empty(shape, dtype=x.dtype, device=x.device) if out is None else out
    if tuple(y.shape) != shape or y.dtype != x.dtype or not y.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of shape %s" % (x.dtype, shape))
    nbytes = lib().fcm_chain_workspace_bytes(ctypes.byref(plan))
    if workspace is None and nbytes > 0:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
    if workspace is not None and workspace.numel() * workspace.element_size() < nbytes:
        raise ValueError("workspace smaller than fcm_chain_workspace_bytes")
    W = (ctypes.c_void_p * desc.num_layers)(*[t.data_ptr() for t in weights])
    B = (ctypes.c_void_p * desc.num_layers)(*[(b.data_ptr() if b is not None else None) for b in biases])
    args = (ctypes.byref(desc), ctypes.byref(plan), _ptr(x), W, B, _ptr(workspace), _ptr(y), _stream(x, stream))
    r = _ChainRun(lib().fcm_chain_run, args, y, (W, B, workspace, desc, plan))
    return r if prepare else r()


def fold_batchnorm(w, b, gamma, beta, mean, var, eps=1e-5):
    """Fold an inference batch normalisation into the preceding convolution (host numpy
    float32 arrays; w is [c_out, ...]). Returns (w_folded, b_folded)."""
    import numpy as np
    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    w = f32(w)
    c_out = w.shape[0]
    row = int(w.size // c_out)
    g, bt, m, v = f32(gamma), f32(beta), f32(mean), f32(var)
    for a in (g, bt, m, v):
        if a.shape != (c_out,):
            raise ValueError("gamma, beta, mean, var must have c_out = %d entries" % c_out)
    bb = None if b is None else f32(b)
    wo, bo = np.empty_like(w), np.empty(c_out, dtype=np.float32)
    p = lambda a: None if a is None else a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    _check(lib().fcm_fold_batchnorm(c_out, row, p(w), p(bb), p(g), p(bt), p(m), p(v), float(eps), p(wo), p(bo)))
    return wo, bo
