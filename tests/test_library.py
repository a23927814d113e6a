"""Host-side tests of the C-ABI library (no GPU needed): libfcm.so loads and exports every
function include/fcm.h declares, the FusePlanner (Sec. IV) returns consistent plans for
every layer of the five workloads, its byte model matches the closed forms of
"input + weights + output" and "plus twice each intermediate" (Sec. IV, Eq. 1-4 and the
layer-by-layer comparison of Sec. II-D), and invalid descriptors or plans are rejected
with the documented status codes. Nothing here launches a kernel."""
import ctypes
import os
import re
import subprocess
import sys

import pytest

import bench
from paper_2404_19331_amd import fcm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fcm.h")
ELT = {"f32": 4, "bf16": 2, "i8": 1}
EINVAL, EUNSUPPORTED = 1, 2


def _header():
    with open(HEADER) as f:
        return f.read()


def _declared_functions():
    src = re.sub(r"/\*.*?\*/", " ", _header(), flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(fcm_\w+)\s*\(", src, flags=re.M)))


def _workspace_limit():
    m = re.search(r"#define\s+FCM_SPLIT_WORKSPACE_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", _header())
    return int(m.group(1)) << int(m.group(2))


def _all_cases():
    out = []
    for wl in ("C1", "C2", "C3b1", "C3b32", "C4", "C5", "PWPW"):
        cases, _ = bench.workload_cases(wl)
        out += [(wl, c) for c in cases]
    return out


CASES = _all_cases()


def test_library_exports_every_declared_function():
    names = _declared_functions()
    assert len(names) >= 12, names
    L = fcm.lib()
    for n in names:
        assert hasattr(L, n), "libfcm.so does not export %s" % n


def test_status_strings_version_and_variant_table():
    L = fcm.lib()
    for st in range(4):
        assert L.fcm_status_string(st)
    assert fcm.lib().fcm_version().decode().startswith("fcm ")
    n = L.fcm_variant_count()
    names = [fcm.variant_name(v) for v in range(n)]
    assert n > 50 and all(names)
    persistent = [x for x in names if re.match(r"k_\w+3<", x)]  # these names carry the element type
    assert persistent and len(set(persistent)) == len(persistent)
    assert fcm.variant_name(n) is None and fcm.variant_name(-1) is None


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(fcm, "_lib", None)
    monkeypatch.setattr(fcm, "LIB_PATH", os.path.join(ROOT, "no_such_dir", "libfcm.so"))
    with pytest.raises(fcm.FcmError):
        fcm.lib()


@pytest.mark.parametrize("wl,case", CASES, ids=lambda v: v if isinstance(v, str) else v.name)
def test_plan_every_layer(wl, case):
    d = fcm.desc_from_case(case)
    p = fcm.plan(case.op, d)
    ho, wo = fcm.out_hw(case.h, case.w, case.k, case.stride, case.pad)
    name = fcm.variant_name(p.variant)
    fam = {"dw_pw": "k_dwpw", "pw_dw": "k_pwdw", "pw_dw_pw": "k_pwdwpw", "pw_pw": "k_pwpw", "dw": "k_dw",
           "pw": "k_pw"}[case.op]
    assert name.startswith(fam), name
    assert 1 <= p.tile_h and 1 <= p.tile_w and p.co_block >= 1 and p.c_block >= 1
    if name.startswith("k_pwpw4"):  # registers; LDS only for the partial sums of split waves
        assert p.tile_h == 1 and p.tile_w in (16, 32) and p.splits in (1, 2, 4)
        assert p.splits <= -(-case.c_mid * ELT[case.dtype] // 64)
        assert p.lds_bytes == (4 * (p.tile_w // 16) * -(-case.c_out // 16) * 1024 if p.splits > 1 else 0)
    else:
        assert 0 < p.lds_bytes <= 160 * 1024
    assert p.workgroups >= 1 and p.waves == (8 if name.startswith("k_dwpw7<") else 4)
    assert p.bytes_tiled >= p.bytes_ideal > 0
    if name.endswith(">") and re.match(r"k_\w+3<", name):  # persistent kernels
        assert p.depth in (2, 3)
        assert p.splits in (1, 2, 4, 8)
        if p.splits > 1:
            tiles = case.n * -(-ho // p.tile_h) * -(-wo // p.tile_w) * -(-case.c_out // p.co_block)
            assert p.splits * tiles * p.tile_h * p.tile_w * p.co_block * 4 <= _workspace_limit()
    # same answer every time (the plan cache and the search are deterministic)
    q = fcm.plan(case.op, d)
    assert p.as_dict() == q.as_dict()


@pytest.mark.parametrize("wl,case", [(w, c) for w, c in CASES if c.op == "dw_pw"],
                         ids=lambda v: v if isinstance(v, str) else v.name)
def test_dw_pw_byte_model_closed_forms(wl, case):
    p = fcm.plan(case.op, fcm.desc_from_case(case))
    ho, wo = fcm.out_hw(case.h, case.w, case.k, case.stride, case.pad)
    e = ELT[case.dtype]
    x = case.n * case.h * case.w * case.c_in
    mid = case.n * ho * wo * case.c_in
    y = case.n * ho * wo * case.c_out
    w = case.c_in * case.k * case.k + case.c_out * case.c_in
    assert p.bytes_ideal == (x + w + y) * e
    assert p.bytes_lbl_ideal == (x + w + y + 2 * mid) * e


def test_fusion_saves_half_the_traffic_when_widths_match():
    # Fig. 1's sanity check: with C_in = C_out and stride 1 the layer-by-layer chain
    # moves x, mid (twice) and y, all of one size, the fused module only x and y.
    d = fcm.make_desc(8, 112, 112, 64, 64, 64, k=3, stride=1, pad=1, dtype="bf16", layout="nhwc")
    p = fcm.plan("dw_pw", d)
    saved = 1 - p.bytes_ideal / p.bytes_lbl_ideal
    assert abs(saved - 0.5) < 0.005


def _evaluate(op, d, th, tw, variant_prefix, **kw):
    for v in range(fcm.lib().fcm_variant_count()):
        if fcm.variant_name(v).startswith(variant_prefix):
            ct = int(fcm.variant_name(v).split(",")[4])
            return fcm.plan_evaluate(op, d, th, tw, 64 // ELT["bf16"], 16 * ct, v, **kw)
    raise AssertionError(variant_prefix)


def test_plan_evaluate_checks_depth_and_splits():
    d = fcm.make_desc(1, 14, 14, 512, 512, 512, k=3, stride=1, pad=1, dtype="bf16", layout="nhwc")
    p = _evaluate("dw_pw", d, 2, 7, "k_dwpw3<bf16,3,1,4,4,p16>", depth=3, splits=4)
    assert (p.depth, p.splits) == (3, 4)
    assert _evaluate("dw_pw", d, 2, 7, "k_dwpw3<bf16,3,1,4,4,p16>").splits == 1  # 0 = no split
    for kw in (dict(depth=9), dict(depth=1), dict(splits=32)):  # 16 channel chunks: 32 splits leave some empty
        with pytest.raises(fcm.FcmError) as e:
            _evaluate("dw_pw", d, 2, 7, "k_dwpw3<bf16,3,1,4,4,p16>", **kw)
        assert e.value.status == EUNSUPPORTED
    dd = fcm.make_desc(1, 14, 14, 512, 512, 512, k=3, stride=1, pad=1, dtype="bf16", layout="nhwc")
    with pytest.raises(fcm.FcmError):  # a depthwise-only kernel has no contraction to split
        _evaluate("dw", dd, 2, 7, "k_dw3<bf16,3,1", splits=2)


def test_plan_evaluate_rejects_what_no_kernel_implements():
    d = fcm.make_desc(1, 56, 56, 64, 64, 64, k=3, stride=1, pad=1, dtype="bf16", layout="nhwc")
    with pytest.raises(fcm.FcmError):  # window wider than the kernel's LDS row pitch
        _evaluate("dw_pw", d, 2, 28, "k_dwpw3<bf16,3,1,4,4,p16>")
    with pytest.raises(fcm.FcmError):  # unknown variant
        fcm.plan_evaluate("dw_pw", d, 4, 4, 32, 64, 10 ** 6)


@pytest.mark.parametrize("kw,status", [
    (dict(n=0), EINVAL), (dict(h=0), EINVAL), (dict(c_in=0), EINVAL), (dict(c_out=0), EINVAL),
    (dict(c_mid=16), EINVAL), (dict(pad=3), EINVAL), (dict(stride=0), EINVAL), (dict(h=1, w=1, pad=0), EINVAL),
    (dict(k=4), EUNSUPPORTED), (dict(k=7), EUNSUPPORTED), (dict(stride=3), EUNSUPPORTED),
    (dict(dtype="i8", rq=[(1, 70, -128, 127)]), EINVAL), (dict(dtype="i8", rq=[(1, 8, 5, -5)]), EINVAL)])
def test_descriptor_validation(kw, status):
    a = dict(n=1, h=16, w=16, c_in=32, c_mid=32, c_out=32, k=3, stride=1, pad=1, dtype="f32", layout="nchw")
    a.update(kw)
    d = fcm.make_desc(**a)
    with pytest.raises(fcm.FcmError) as e:
        fcm.plan("dw_pw", d)
    assert e.value.status == status


def test_int8_relu6_plans_as_the_quantised_clamp():
    d = fcm.make_desc(1, 16, 16, 32, 32, 32, k=3, stride=1, pad=1, dtype="i8", layout="nhwc",
                      act=("relu6", "relu6", "none"), rq=[(1, 6, -127, 24)] * 3)
    assert fcm.plan("dw_pw", d).variant >= 0


def test_header_is_plain_c():
    src = _header()
    assert "extern \"C\"" in src and "#include <stdint.h>" in src
    assert "hip" not in re.sub(r"/\*.*?\*/", " ", src, flags=re.S).lower()
    L = fcm.lib()
    # the plan struct the Python binding marshals has the size the library fills in
    assert ctypes.sizeof(fcm.Plan) % 8 == 0
    assert L.fcm_variant_count() > 0


@pytest.mark.parametrize("wl,case", [(w, c) for w, c in CASES if c.op == "pw_pw"],
                         ids=lambda v: v if isinstance(v, str) else v.name)
def test_pw_pw_byte_model_closed_forms(wl, case):
    # two pointwise layers: the fused module moves x, both weight matrices and y; the
    # layer-by-layer pair also writes and reads the c_mid-wide intermediate
    p = fcm.plan(case.op, fcm.desc_from_case(case))
    px = case.n * case.h * case.w
    w = case.c_mid * case.c_in + case.c_out * case.c_mid
    assert p.bytes_ideal == px * (case.c_in + case.c_out) + w
    assert p.bytes_lbl_ideal == p.bytes_ideal + 2 * px * case.c_mid


def _v4_variant(dt, prefix):
    for v in range(fcm.lib().fcm_variant_count()):
        if fcm.variant_name(v).startswith("k_pwpw4<%s,%s" % (dt, prefix)):
            return v
    raise AssertionError(prefix)


def test_register_kernel_plan_checks():
    d = fcm.make_desc(2, 14, 14, 64, 384, 64, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
                      act=("relu", "none", "none"))
    v = _v4_variant("i8", "1,4,1")
    npg = -(-2 * 14 * 14 // 16)
    for s, wgs in ((1, -(-npg // 4)), (2, -(-npg // 2)), (4, npg)):
        p = fcm.plan_evaluate("pw_pw", d, 1, 16, 64, 64, v, splits=s)
        assert (p.splits, p.workgroups) == (s, wgs)
        assert p.lds_bytes == (4 * 4 * 1024 if s > 1 else 0)
    assert p.bytes_ideal == (2 * 14 * 14 * 128 + 2 * 64 * 384)
    assert p.bytes_paper == p.bytes_tiled == 2 * 14 * 14 * 128 + npg * 2 * 64 * 384
    bad = [dict(splits=3), dict(splits=8),       # one workgroup: 1, 2 or 4 waves per pixel group
           dict(tile_w=32), dict(co_block=128)]  # the variant's tiling is fixed
    for kw in bad:
        a = dict(tile_h=1, tile_w=16, c_block=64, co_block=64, splits=1)
        a.update(kw)
        with pytest.raises(fcm.FcmError) as e:
            fcm.plan_evaluate("pw_pw", d, a["tile_h"], a["tile_w"], a["c_block"], a["co_block"], v,
                              splits=a["splits"])
        assert e.value.status == EUNSUPPORTED
    # more splits than intermediate chunks (64 channels: one chunk)
    d1 = fcm.make_desc(2, 14, 14, 64, 64, 64, k=1, stride=1, pad=0, dtype="i8", layout="nhwc")
    with pytest.raises(fcm.FcmError):
        fcm.plan_evaluate("pw_pw", d1, 1, 16, 64, 64, v, splits=2)
    # too many input channels for one k-step, output channels not in fours, NCHW
    for kw in (dict(c_in=80), dict(c_out=62), dict(layout="nchw")):
        a = dict(n=2, h=14, w=14, c_in=64, c_mid=384, c_out=64, k=1, stride=1, pad=0, dtype="i8", layout="nhwc")
        a.update(kw)
        dd = fcm.make_desc(**a)
        with pytest.raises(fcm.FcmError) as e:
            fcm.plan_evaluate("pw_pw", dd, 1, 16, 64, -(-a["c_out"] // 16) * 16, v)
        assert e.value.status == EUNSUPPORTED
        # the planner still finds a kernel (the first-generation one where the register kernel cannot run)
        assert fcm.plan("pw_pw", dd).variant >= 0


def test_library_binds_to_the_hip_runtime_torch_loads():
    # torch's ROCm build ships its own HIP runtime; libfcm.so loaded before torch would
    # pull in a second one, which finds no device once torch's has opened it
    code = ("from paper_2404_19331_amd import fcm; fcm.lib(); import torch; "
            "m = open('/proc/self/maps').read().splitlines(); "
            "print(len({l.split()[-1] for l in m if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


# --------------------------------------------------------------------------------------
# Asymmetric int8 (zero points): planned on the first-generation kernels, the int8
# persistent kernels and the PW->PW register kernel
# --------------------------------------------------------------------------------------

def _first_gen(v):
    return re.search(r"\d<", fcm.variant_name(v)) is None


def _persistent(p):
    return re.match(r"k_(dwpw|dw|pw)3<i8,", fcm.variant_name(p.variant)) is not None


ZP_SHAPES = {"dw_pw": (64, 64, 64, 3), "pw_dw": (32, 96, 96, 3), "pw_dw_pw": (32, 96, 32, 3),
             "pw_pw": (64, 128, 64, 1), "dw": (64, 64, 64, 3), "pw": (64, 64, 96, 1)}


def _zp_desc(op, zp_in=0, zps=(0, 0, 0), dtype="i8"):
    ci, cm, co, k = ZP_SHAPES[op]
    rq = [(1, 6, -128, 127, z) for z in zps]
    return fcm.make_desc(4, 28, 28, ci, cm, co, k=k, stride=1, pad=k // 2, dtype=dtype, layout="nhwc",
                         act=("relu", "relu", "none"), rq=rq, zp_in=zp_in)


@pytest.mark.parametrize("op", list(ZP_SHAPES))
def test_zero_points_plan_capable_kernels(op):
    stages = {"pw_dw_pw": 3, "dw": 1, "pw": 1}.get(op, 2)
    sym = fcm.plan(op, _zp_desc(op))
    if op in ("dw_pw", "pw_pw", "dw", "pw"):
        assert not _first_gen(sym.variant)  # not vacuous: symmetric int8 runs on a newer kernel
    variants = [(5, (0, 0, 0))] + [(0, tuple(-7 if j == i else 0 for j in range(3))) for i in range(stages)]
    for zin, zps in variants:
        p = fcm.plan(op, _zp_desc(op, zin, zps))
        name = fcm.variant_name(p.variant)
        if op == "pw_pw":  # the register kernel carries zero points (up to 192 output channels)
            assert name.startswith("k_pwpw4<i8,"), (zin, zps, name)
        elif op in ("dw_pw", "dw", "pw"):  # the int8 persistent kernels
            assert _persistent(p), (zin, zps, name, p.splits)
        else:
            assert _first_gen(p.variant), (zin, zps, name)
    # a zero point of a stage the module does not have is ignored, as are float types
    if stages < 3:
        assert fcm.plan(op, _zp_desc(op, 0, (0, 0, 9) if stages == 2 else (0, 9, 9))).as_dict() == sym.as_dict()
    f = fcm.plan(op, _zp_desc(op, 5, (3, 3, 3), dtype="bf16"))
    assert f.as_dict() == fcm.plan(op, _zp_desc(op, dtype="bf16")).as_dict()


def _pc_desc(op, stages, zp_in=0):
    """A descriptor with per-channel requantisation on `stages`: for planning only (the
    planner never dereferences the pointers, so stand-in addresses serve)."""
    d = _zp_desc(op, zp_in)
    for i in stages:
        d.rq_channel[i] = 0x10000 * (i + 1)
    return d


@pytest.mark.parametrize("op", list(ZP_SHAPES))
def test_per_channel_plan_capable_kernels(op):
    """Per-channel requantisation plans on the int8 persistent kernels where they
    implement the module (DW->PW, DW, PW), else on the first-generation kernels; the ring
    slot grows by the three KiB of staged multipliers and shifts."""
    stages = {"pw_dw_pw": 3, "dw": 1, "pw": 1}.get(op, 2)
    sym = fcm.plan(op, _zp_desc(op))
    for sel in ([0], [stages - 1], list(range(stages))):
        for zin in (0, -5):
            p = fcm.plan(op, _pc_desc(op, sel, zin))
            name = fcm.variant_name(p.variant)
            if op in ("dw_pw", "dw", "pw"):
                assert _persistent(p), (sel, zin, name, p.splits)
            else:
                assert _first_gen(p.variant), (sel, zin, name)
    # a stage the module does not have is ignored
    if stages < 3:
        assert fcm.plan(op, _pc_desc(op, [2])).as_dict() == sym.as_dict()
    if op in ("dw_pw", "dw", "pw"):
        pc = _pc_desc(op, [0])
        a = fcm.plan_evaluate(op, _zp_desc(op), sym.tile_h, sym.tile_w, sym.c_block, sym.co_block, sym.variant,
                              depth=2)
        b = fcm.plan_evaluate(op, pc, sym.tile_h, sym.tile_w, sym.c_block, sym.co_block, sym.variant, depth=2)
        assert b.lds_bytes - a.lds_bytes == 2 * 3072 and b.splits == 1


def test_zero_points_on_the_register_kernel_up_to_192_output_channels():
    for co, reg in ((64, True), (128, True), (192, True), (208, False), (256, False)):
        d = fcm.make_desc(4, 28, 28, 64, 128, co, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
                          act=("relu", "none"), rq=[(1, 6, -128, 127, 3)] * 3, zp_in=-2)
        name = fcm.variant_name(fcm.plan("pw_pw", d).variant)
        assert name.startswith("k_pwpw4<i8,") == reg, (co, name)
        if not reg:
            assert _first_gen(fcm.plan("pw_pw", d).variant)
    # an explicit plan on a register-kernel instance with more output tiles is refused
    d = fcm.make_desc(4, 28, 28, 64, 128, 256, k=1, stride=1, pad=0, dtype="i8", layout="nhwc",
                      rq=[(1, 6, -128, 127, 3)] * 3)
    big = [v for v in range(fcm.lib().fcm_variant_count()) if fcm.variant_name(v) == "k_pwpw4<i8,4,16,1>"][0]
    with pytest.raises(fcm.FcmError) as e:
        fcm.plan_evaluate("pw_pw", d, 1, 16, 64, 256, big)
    assert e.value.status == EUNSUPPORTED and "zero points" in str(e.value)


def test_zero_points_validation_and_explicit_plans():
    for zin, zps in ((128, (0, 0, 0)), (-129, (0, 0, 0)), (0, (0, 200, 0)), (0, (-300, 0, 0))):
        with pytest.raises(fcm.FcmError) as e:
            fcm.plan("dw_pw", _zp_desc("dw_pw", zin, zps))
        assert e.value.status == EINVAL and "zero point" in str(e.value)
    # an explicit persistent plan is accepted for an asymmetric descriptor, unsplit and
    # split; one on a newer kernel without zero points (PW->DW streaming) is refused
    sym = fcm.plan("dw_pw", _zp_desc("dw_pw"))
    assert re.match(r"k_dwpw3<i8,", fcm.variant_name(sym.variant))
    un = fcm.plan_evaluate("dw_pw", _zp_desc("dw_pw", 3), sym.tile_h, sym.tile_w, sym.c_block, sym.co_block,
                           sym.variant)
    assert un.splits == 1
    wide = fcm.make_desc(4, 14, 14, 256, 256, 64, k=3, stride=1, pad=1, dtype="i8", layout="nhwc",
                         rq=[(1, 6, -128, 127, 4)] * 3, zp_in=3)
    sp = fcm.plan_evaluate("dw_pw", wide, 7, 7, 64, 64, sym.variant, splits=2)
    assert sp.splits == 2 and fcm.workspace_bytes(wide, sp) > 0
    pd = fcm.plan("pw_dw", _zp_desc("pw_dw"))
    if not _first_gen(pd.variant):
        with pytest.raises(fcm.FcmError) as e:
            fcm.plan_evaluate("pw_dw", _zp_desc("pw_dw", 3), pd.tile_h, pd.tile_w, pd.c_block, pd.co_block,
                              pd.variant)
        assert e.value.status == EUNSUPPORTED


def test_chain_zero_points_reach_the_groups_they_touch():
    """A zero point on one layer's output moves to the zero-point kernels (first generation,
    int8 persistent) exactly the groups that write that tensor or read it; the
    others keep the symmetric plan."""
    layers = [dict(kind="pw", c_out=96, act="relu", rq=(1, 6, -128, 127)),
              dict(kind="dw", k=3, stride=1, pad=1, act="relu", rq=(1, 4, -128, 127)),
              dict(kind="pw", c_out=64, act="none", rq=(1, 7, -128, 127)),
              dict(kind="pw", c_out=128, act="relu", rq=(1, 6, -128, 127)),
              dict(kind="dw", k=3, stride=1, pad=1, act="relu", rq=(1, 4, -128, 127)),
              dict(kind="pw", c_out=64, act="none", rq=(1, 7, -128, 127))]
    sym = fcm.chain_plan(fcm.chain_desc(4, 28, 28, 64, layers, "i8"), "unfused")
    for j in range(len(layers)):
        zl = [dict(L) for L in layers]
        zl[j]["rq"] = tuple(zl[j]["rq"]) + (-11,)
        p = fcm.chain_plan(fcm.chain_desc(4, 28, 28, 64, zl, "i8"), "unfused")
        for g, (first, op, plan) in enumerate(p.groups()):
            touched = first in (j, j + 1)  # unfused: one layer per group
            assert _first_gen(plan.variant) or _persistent(plan) or not touched, (j, first)
            if not touched:
                assert plan.as_dict() == sym.plan[g].as_dict()
    # the chain input's zero point reaches the first group only
    p = fcm.chain_plan(fcm.chain_desc(4, 28, 28, 64, layers, "i8", zp_in=-128), "unfused")
    assert (_first_gen(p.plan[0].variant) or _persistent(p.plan[0])) and \
        p.plan[1].as_dict() == sym.plan[1].as_dict()


def test_abi_struct_sizes_match_the_binding(tmp_path):
    """The ctypes mirrors of the descriptor structs have the C sizes and field offsets."""
    src = tmp_path / "sizes.c"
    src.write_text('#include <stdio.h>\n#include <stddef.h>\n#include "fcm.h"\nint main(void){\n'
                   'printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(fcm_requant), sizeof(fcm_desc),'
                   ' offsetof(fcm_desc, zp_in), sizeof(fcm_layer), sizeof(fcm_chain_desc),'
                   ' offsetof(fcm_chain_desc, layers), sizeof(fcm_chain_plan_t));\nreturn 0;}\n')
    exe = tmp_path / "sizes"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    assert got == [ctypes.sizeof(fcm.Requant), ctypes.sizeof(fcm.Desc), fcm.Desc.zp_in.offset,
                   ctypes.sizeof(fcm.Layer), ctypes.sizeof(fcm.ChainDesc), fcm.ChainDesc.layers.offset,
                   ctypes.sizeof(fcm.ChainPlan)]


def test_zero_point_time_models_are_their_own():
    """First-generation kernels under zero points are priced by their own fitted figures:
    the same plan of the same shapes gets another estimate than symmetric, while a float
    descriptor (zero points ignored) keeps the symmetric one."""
    for op in ("pw_dw", "pw_dw_pw"):
        sym = _zp_desc(op)
        asym = _zp_desc(op, -128, (5, 5, 5))
        p = fcm.plan(op, asym)
        assert _first_gen(p.variant)
        t_sym, t_zp = fcm.plan_time_estimate(sym, p), fcm.plan_time_estimate(asym, p)
        assert t_sym > 0 and t_zp > 0 and t_sym != t_zp, op
        f_sym, f_zp = _zp_desc(op, dtype="bf16"), _zp_desc(op, -128, (5, 5, 5), dtype="bf16")
        q = fcm.plan(op, f_sym)
        assert fcm.plan_time_estimate(f_sym, q) == fcm.plan_time_estimate(f_zp, q)


def test_split_plans_need_a_caller_workspace():
    """The library allocates nothing: a plan that splits channel chunks names the workspace
    it needs, the entry points without one refuse it, and a short workspace is refused;
    all before anything reaches the device (the pointers below are never dereferenced)."""
    d = fcm.make_desc(1, 14, 14, 512, 512, 512, k=3, stride=1, pad=1, dtype="bf16", layout="nhwc")
    p = _evaluate("dw_pw", d, 2, 7, "k_dwpw3<bf16,3,1,4,4,p16>", splits=4)
    need = fcm.workspace_bytes(d, p)
    tiles = 7 * 2 * (512 // 64)  # spatial tiles x output-channel blocks of 64
    assert need == 4 * tiles * 14 * 64 * 4  # [split][tile][pixel][channel] fp32 partial sums
    assert fcm.workspace_bytes(d, _evaluate("dw_pw", d, 2, 7, "k_dwpw3<bf16,3,1,4,4,p16>")) == 0
    L = fcm.lib()
    dev = ctypes.c_void_p(1 << 20)  # aligned stand-in: validation fails before any launch
    args = (ctypes.byref(d), dev, dev, None, dev, None, dev, ctypes.byref(p))
    assert L.fcm_dw_pw(*args, None) == EINVAL
    assert "workspace" in fcm.last_error()
    assert L.fcm_dw_pw_ws(*args, dev, need - 16, None) == EINVAL
    assert L.fcm_dw_pw_ws(*args, ctypes.c_void_p((1 << 20) + 8), need, None) == EINVAL  # misaligned
    assert L.fcm_dw_pw_ws(*args, dev, -1, None) == EINVAL
    dp = fcm.make_desc(1, 14, 14, 512, 512, 512, dtype="bf16", layout="nhwc")
    pp = _evaluate("pw", dp, 2, 7, "k_pw3<bf16,1,1,4,4,p16>", splits=2)
    assert fcm.workspace_bytes(dp, pp) > 0
    assert L.fcm_pw(ctypes.byref(dp), dev, dev, None, dev, ctypes.byref(pp), None) == EINVAL
    with pytest.raises(fcm.FcmError):
        bad = fcm.make_desc(0, 14, 14, 512, 512, 512, dtype="bf16", layout="nhwc")
        fcm.workspace_bytes(bad, p)


def test_library_sources_do_not_allocate_device_memory():
    """No allocation call anywhere in the library's host sources."""
    csrc = os.path.join(ROOT, "paper_2404_19331_amd", "csrc")
    for f in os.listdir(csrc):
        if f.endswith((".cpp", ".h", ".hip", ".inc")):
            src = open(os.path.join(csrc, f)).read()
            assert not re.search(r"\bhip(Malloc|MallocAsync|HostMalloc|ExtMallocWithFlags|Free)\w*\s*\(", src), f


def test_plan_limited_respects_the_workspace_budget():
    """Where the unrestricted planner splits, a zero budget yields a plan needing none."""
    found = False
    for wl in ("C3b1", "C4"):
        for case in bench.workload_cases(wl)[0]:
            d = fcm.desc_from_case(case)
            p = fcm.plan(case.op, d)
            q = fcm.plan_limited(case.op, d, 0)
            assert fcm.workspace_bytes(d, q) == 0
            if fcm.workspace_bytes(d, p) > 0:
                found = True
                r = fcm.plan_limited(case.op, d, fcm.workspace_bytes(d, p))
                assert (r.variant, r.tile_h, r.tile_w, r.splits) == (p.variant, p.tile_h, p.tile_w, p.splits)
    assert found, "no workload layer is planned with a split"


def _same(p, q):
    return (p.variant, p.tile_h, p.tile_w, p.c_block, p.co_block, p.depth, p.splits, p.workgroups) == (
        q.variant, q.tile_h, q.tile_w, q.c_block, q.co_block, q.depth, q.splits, q.workgroups)


@pytest.mark.parametrize("wl", ["C1", "C2", "C3b1", "C3b32", "C4", "C5", "PWPW"])
def test_plan_candidates_lead_with_the_planners_choice(wl):
    """fcm_plan_candidates: the workspace-limited planner's plan first, distinct plans,
    each within the workspace limit and reproduced by fcm_plan_evaluate."""
    for case in bench.workload_cases(wl)[0]:
        d = fcm.desc_from_case(case)
        for ws in (0, 64 << 20):
            cands = fcm.plan_candidates(case.op, d, 12, ws)
            assert 1 <= len(cands) <= 12
            assert _same(cands[0], fcm.plan_limited(case.op, d, ws))
            for i, p in enumerate(cands):
                assert fcm.workspace_bytes(d, p) <= ws
                assert not any(_same(p, q) for q in cands[:i])
                e = fcm.plan_evaluate(case.op, d, p.tile_h, p.tile_w, p.c_block, p.co_block, p.variant,
                                      workgroups=p.workgroups, depth=p.depth, splits=p.splits)
                assert (e.bytes_tiled, e.lds_bytes, e.workgroups) == (p.bytes_tiled, p.lds_bytes, p.workgroups)
        # each compiled variant that implements the layer appears before any variant repeats
        cands = fcm.plan_candidates(case.op, d, 64, 0)
        seen, repeated = set(), False
        for p in cands[1:]:
            if p.variant in seen:
                repeated = True
            else:
                assert not repeated, "a new variant after a repeated one"
                seen.add(p.variant)


def test_plan_candidates_rejects_bad_arguments():
    d = fcm.desc_from_case(bench.workload_cases("C1")[0][0])
    arr = (fcm.Plan * 4)()
    n = ctypes.c_int32(7)
    assert fcm.lib().fcm_plan_candidates(fcm.OP["dw_pw"], ctypes.byref(d), None, 0, arr, 0, ctypes.byref(n)) == 1
    assert n.value == 0
    assert fcm.lib().fcm_plan_candidates(fcm.OP["dw_pw"], ctypes.byref(d), None, -1, arr, 4, ctypes.byref(n)) == 1
    assert fcm.lib().fcm_plan_candidates(fcm.OP["dw_pw"], ctypes.byref(d), None, 0, None, 4, ctypes.byref(n)) == 1
