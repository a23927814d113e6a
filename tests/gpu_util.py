"""Helpers for the GPU parity tests: move seeded numpy inputs to the device, run the HIP
path through the C ABI binding, compare against the CPU oracle at the stated tolerances."""
import numpy as np

import oracle
from paper_2404_19331_amd import fcm

# Tolerances (written once, used by every parity test):
#   f32:  |g - r| <= 1e-4 + 1e-5 |r|                       (elementwise)
#   bf16: |g - r| <= 2e-2 max(|r|, rms(r))                 (2e-2 relative, with a floor at
#         2e-2 of the reference's RMS so that outputs near zero are not held to a pure
#         relative bound that rounding of the bf16 intermediate cannot meet)
#   i8:   bit-exact
F32_ATOL, F32_RTOL = 1e-4, 1e-5
BF16_RTOL = 2e-2


def torch():
    import torch as t
    return t


def to_dev(a, dtype):
    t = torch()
    if a is None:
        return None
    if a.dtype == np.uint16:  # bf16 bits
        return t.from_numpy(a.view(np.int16).copy()).view(t.bfloat16).cuda()
    return t.from_numpy(np.ascontiguousarray(a)).cuda()


def to_np(x):
    t = torch()
    x = x.detach().cpu()
    if x.dtype == t.bfloat16:
        return x.view(t.int16).numpy().view(np.uint16)
    return x.numpy()


def bf16_to_f32(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


def values(a, dtype):
    """Storage array -> float64 values for comparisons."""
    if dtype == "bf16":
        return bf16_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def assert_close(got, ref, dtype, what=""):
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if dtype == "i8":
        bad = np.argwhere(got != ref)
        assert bad.size == 0, "%s: %d int8 mismatches, first at %s: got %d ref %d" % (
            what, len(bad), tuple(bad[0]), got[tuple(bad[0])], ref[tuple(bad[0])])
        return
    g, r = values(got, dtype), values(ref, dtype)
    assert np.all(np.isfinite(g)), "%s: non-finite output" % what
    if dtype == "f32":
        tol = F32_ATOL + F32_RTOL * np.abs(r)
    else:
        rms = np.sqrt(np.mean(r * r)) if r.size else 0.0
        tol = BF16_RTOL * np.maximum(np.abs(r), rms)
    err = np.abs(g - r)
    bad = err > tol
    if err.size:
        print("%s: max |err| / tolerance = %.3f" % (what, float(np.max(err / np.maximum(tol, 1e-300)))))
    if np.any(bad):
        i = tuple(np.argwhere(bad)[0])
        raise AssertionError("%s: %d/%d outside tolerance; first at %s got %r ref %r (max err %.3g)" % (
            what, int(bad.sum()), bad.size, i, g[i], r[i], float(err.max())))


def dev_inputs(inp, dtype):
    return {k: to_dev(v, dtype) for k, v in inp.items()}


def run_fused(case, d, plan=None, out=None, rq_channel=None):
    """Run the case's module on the GPU through the C ABI. d: dict of device tensors.
    rq_channel: int8 per-channel requantisation tensors per stage (or None)."""
    kw = dict(stride=case.stride, pad=case.pad, layout=case.layout, plan=plan, out=out)
    if rq_channel is not None:
        kw["rq_channel"] = rq_channel
    rq = list(case.rq) if case.dtype == "i8" else None
    if case.dtype == "i8":
        kw["zp_in"] = getattr(case, "zp_in", 0)
    if case.op == "dw_pw":
        return fcm.dw_pw(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=case.act[:2], rq=rq, **kw)
    if case.op == "pw_dw":
        return fcm.pw_dw(d["x"], d["w_pw"], d["w_dw"], d.get("b_pw"), d.get("b_dw"), act=case.act[:2], rq=rq, **kw)
    if case.op == "pw_dw_pw":
        return fcm.pw_dw_pw(d["x"], d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"),
                            d.get("b_pw2"), act=case.act, rq=rq, **kw)
    if case.op == "pw_pw":
        kw.pop("stride"), kw.pop("pad")
        return fcm.pw_pw(d["x"], d["w_pw1"], d["w_pw2"], d.get("b_pw1"), d.get("b_pw2"), act=case.act[:2], rq=rq,
                         **kw)
    if case.op == "dw":
        return fcm.dw(d["x"], d["w_dw"], d.get("b_dw"), act=case.act[0], rq=rq[0] if rq else None, **kw)
    if case.op == "pw":
        kw.pop("stride"), kw.pop("pad")
        return fcm.pw(d["x"], d["w_pw"], d.get("b_pw"), act=case.act[0], rq=rq[0] if rq else None, **kw)
    raise ValueError(case.op)


def run_unfused(case, d):
    kw = dict(stride=case.stride, pad=case.pad, layout=case.layout)
    rq = list(case.rq) if case.dtype == "i8" else None
    if case.dtype == "i8":
        kw["zp_in"] = getattr(case, "zp_in", 0)
    if case.op == "dw_pw":
        return fcm.dw_then_pw(d["x"], d["w_dw"], d["w_pw"], d.get("b_dw"), d.get("b_pw"), act=case.act[:2],
                              rq=rq, **kw)
    if case.op == "pw_dw":
        return fcm.pw_then_dw(d["x"], d["w_pw"], d["w_dw"], d.get("b_pw"), d.get("b_dw"), act=case.act[:2],
                              rq=rq, **kw)
    if case.op == "pw_dw_pw":
        return fcm.pw_then_dw_then_pw(d["x"], d["w_pw1"], d["w_dw"], d["w_pw2"], d.get("b_pw1"), d.get("b_dw"),
                                      d.get("b_pw2"), act=case.act, rq=rq, **kw)
    if case.op == "pw_pw":
        return fcm.pw_then_pw(d["x"], d["w_pw1"], d["w_pw2"], d.get("b_pw1"), d.get("b_pw2"), act=case.act[:2],
                              rq=rq, layout=case.layout, zp_in=kw.get("zp_in", 0))
    raise ValueError(case.op)


def oracle_ref(case, inp):
    return oracle.run(case.op, case, inp)


def batch_slice(inp, idx):
    out = dict(inp)
    out["x"] = np.ascontiguousarray(inp["x"][idx])
    return out


def oracle_chain(spec, x, ws, bs, upto=None):
    """The chain on the CPU oracle, one layer at a time (definition of the chain)."""
    h, w, c = spec.h, spec.w, spec.c
    zp = getattr(spec, "zp_in", 0)
    for i, L in enumerate(spec.layers[:upto]):
        k, s, p = (L["k"], L["stride"], L["pad"]) if L["kind"] == "dw" else (1, 1, 0)
        co = c if L["kind"] == "dw" else L["c_out"]
        rq = list(L.get("rq") or (1, 0, -128, 127))
        case = dict(n=spec.n, h=h, w=w, c_in=c, c_mid=c, c_out=co, k=k, stride=s, pad=p, dtype=spec.dtype,
                    layout=spec.layout, act=[L["act"], "none", "none"], rq=[rq] * 3, zp_in=zp)
        zp = rq[4] if len(rq) > 4 else 0
        if L["kind"] == "dw":
            x = oracle.dw(case, x, ws[i], bs[i])
            h, w = fcm.out_hw(h, w, k, s, p)
        else:
            x = oracle.pw(case, x, ws[i], bs[i])
            c = co
    return x


def run_chain(spec, objective, x, ws, bs, upto=None):
    """The chain through the C ABI (fcm_chain_plan + fcm_chain_run) on device tensors."""
    layers = spec.layers[:upto]
    d = fcm.chain_desc(spec.n, spec.h, spec.w, spec.c, layers, spec.dtype, spec.layout,
                       zp_in=getattr(spec, "zp_in", 0))
    p = fcm.chain_plan(d, objective)
    return fcm.chain_run(d, p, x, ws[:len(layers)], bs[:len(layers)]), p


def assert_close_dev(got, ref, dtype, what=""):
    """assert_close on the device: got is the HIP path's output tensor, ref the oracle's
    (numpy, storage format); the same tolerances."""
    t = torch()
    r = t.from_numpy(values(ref, dtype).astype(np.float32)).to(got.device)
    g = got.float()
    assert tuple(g.shape) == tuple(r.shape), (tuple(g.shape), tuple(r.shape))
    if dtype == "i8":
        bad = int((g != r).sum().item())
        assert bad == 0, "%s: %d int8 mismatches" % (what, bad)
        return
    assert bool(t.isfinite(g).all()), "%s: non-finite output" % what
    if dtype == "f32":
        tol = F32_ATOL + F32_RTOL * r.abs()
    else:
        rms = t.sqrt(t.mean(r.double() * r.double())).float() if r.numel() else t.zeros((), device=r.device)
        tol = BF16_RTOL * t.maximum(r.abs(), rms)
    ratio = float(((g - r).abs() / tol.clamp_min(1e-30)).max().item()) if r.numel() else 0.0
    print("%s: max |err| / tolerance = %.3f" % (what, ratio))
    assert ratio <= 1.0, "%s: outside tolerance (max err / tol = %.3f)" % (what, ratio)
