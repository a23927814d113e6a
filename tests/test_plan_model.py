"""Pins of the FusePlanner byte model (oracle/plan_model.py) and of the library planner's
byte figures against it (CPU only).

The model writes out arXiv 2404.19331 Sec. IV: Eq. 1 (tile overlap), Eq. 2 (PW), Eq. 3
(DW), Eq. 4 (PW->DW) and the module equations built the same way, plus a brute-force
count of what a tiled kernel moves. Here it is pinned to things other than itself: the
special cases and the geometric meaning of Eq. 1, the worked tiling example of the
paper's tiled-convolution figure (Sec. II-D), hand-worked values of Eq. 2-4 on a tiny
layer, and a second, independently written count of the staged windows. Then the
library's planner (fcm_plan / fcm_plan_evaluate: bytes_ideal, bytes_tiled, bytes_paper)
must equal the model on tiny shapes and on every workload layer.
"""
from math import ceil

import numpy as np
import pytest

import bench
from oracle import plan_model as M
from paper_2404_19331_amd import fcm
from paper_2404_19331_amd import workloads as W

ELT = {"f32": 4, "bf16": 2, "i8": 1}


# ---------------------------------------------------------------------------------
# Eq. 1
# ---------------------------------------------------------------------------------

def test_eq1_special_cases_and_hand_value():
    # one tile along both axes: nothing is read twice
    assert M.overlap(10, 8, 1, 1, 3, 3, 1) == 0
    # filter width equal to the stride: neighbouring windows do not overlap
    assert M.overlap(10, 8, 5, 4, 2, 2, 2) == 0
    # 10 wide, 8 high, 2 tiles across, 3 down, 3x3 filter, stride 1:
    # (2-1)*(3-1)*8 + (3-1)*(3-1)*10 = 16 + 40
    assert M.overlap(10, 8, 2, 3, 3, 3, 1) == 56
    # stride 2 with a 3x3 filter overlaps one column per boundary: (4-1)*1*6 + (2-1)*1*9
    assert M.overlap(9, 6, 4, 2, 3, 3, 2) == 27


@pytest.mark.parametrize("h,w,k,th,tw", [(7, 7, 2, 3, 3), (10, 12, 3, 4, 5), (9, 9, 3, 7, 7), (13, 8, 5, 3, 4),
                                         (6, 6, 3, 4, 4)])
def test_eq1_is_the_double_count_of_boundary_strips(h, w, k, th, tw):
    """Stride 1, no padding, tiles dividing the output: the windows of all tiles cover
    H*W positions plus Eq. 1's boundary strips plus the (K-1)^2 corner squares where four
    windows meet (enumerated by the brute force, not by a formula)."""
    ho, wo = h - k + 1, w - k + 1
    if ho % th or wo % tw:
        pytest.skip("tiles must divide the output")
    nty, ntx = ho // th, wo // tw
    staged = sum(M._staged_positions(ty, tx, th, tw, k, 1, 0, h, w) for ty in range(nty) for tx in range(ntx))
    corners = (nty - 1) * (ntx - 1) * (k - 1) ** 2
    assert staged - h * w == M.overlap(w, h, ntx, nty, k, k, 1) + corners


def test_tiled_convolution_figure_example():
    """Sec. II-D figure: 2x2 DW filters and a 3x3 OFM tile read a 4x4 IFM tile. On a 6x6
    output (7x7 input) cut into 2x2 such tiles, Eq. 1 counts one shared row and column of
    7 (twice 7 = 14) and the four windows share one corner position besides."""
    assert M._staged_positions(1, 1, 3, 3, 2, 1, 0, 100, 100) == 16
    assert M.overlap(7, 7, 2, 2, 2, 2, 1) == 14
    staged = sum(M._staged_positions(ty, tx, 3, 3, 2, 1, 0, 7, 7) for ty in range(2) for tx in range(2))
    assert staged == 4 * 16 == 7 * 7 + 14 + 1


# ---------------------------------------------------------------------------------
# Eq. 2, 3, 4 on a tiny layer, worked by hand
# ---------------------------------------------------------------------------------
# N=1, 4x4 input, C_in=2, C_mid=C_out=3, 3x3 DW, stride 1, pad 1 (4x4 output), 2x2 output
# tiles (4 spatial tiles), one channel block, sizes in elements (1 byte each).
#   IFMs 4*4*2 = 32; PW OFMs 4*4*3 = 48; PW weights 3*2 = 6; DW weights (2 ch) 2*9 = 18
#   Overlap (Eq. 1) per channel: (2-1)*(3-1)*4 + (2-1)*(3-1)*4 = 16


def test_eq2_hand_value():
    # 1 weight tile * 32 + 48 + 4 spatial tiles * 6
    assert M.pw_gma(6, 1, 32, 48, 4) == 104
    # printed form: ceil(6/6)*32 + 48 + ceil(48/12)*6 with 12-element OFM tiles (2x2x3)
    assert M.pw_gma_literal(6, 6, 32, 48, 12) == 104
    # with the filters split in 3 weight tiles the printed weight term counts 3x more
    # OFM tiles (2x2x1 each) than spatial tiles: 3*32 + 48 + 12*6 vs 3*32 + 48 + 4*6
    assert M.pw_gma_literal(6, 2, 32, 48, 4) == 216
    assert M.pw_gma(6, 3, 32, 48, 4) == 168


def test_eq3_hand_value():
    # 2 * 2 * 16 + 32 + 32 (DW OFMs 4*4*2) + 4 * 18
    assert M.dw_gma(2, 16, 32, 32, 4, 18) == 200


def test_eq4_hand_value():
    # PW 2->3 then DW 3x3 on 3 channels, one mid-channel block:
    # (2*2*16 + 32) * max(1, 1) + 4 * 6 + 4 * 27 + 48 (output, the term Eq. 4 omits)
    assert M.pwdw_gma(2, 16, 32, 1, 1, 4, 6, 4, 27, 48) == 276
    # three mid-channel blocks recompute the PW per block: the input term triples
    assert M.pwdw_gma(2, 16, 32, 3, 3, 4, 6, 4, 27, 48) == 96 * 3 + 24 + 108 + 48


def test_derived_module_equations_hand_values():
    # DW->PW, C=2 -> 3 outputs, 2 output-channel blocks: input with overlap per block,
    # PW weights per spatial tile, DW weights per tile and block, output once
    assert M.dwpw_gma(2, 16, 32, 2, 4, 6, 18, 48) == (64 + 32) * 2 + 4 * 6 + 4 * 2 * 18 + 48
    # PW->DW->PW 2 -> 3 -> 3, 2 output blocks: PW1 and DW per block, PW2 (9) per tile
    assert M.pwdwpw_gma(2, 16, 32, 2, 4, 6, 27, 9, 48) == 96 * 2 + 4 * 2 * 33 + 4 * 9 + 48
    # PW->PW: no overlap
    assert M.pwpw_gma(32, 2, 4, 6, 9, 48) == 64 + 48 + 36 + 48


# ---------------------------------------------------------------------------------
# Brute force, counted a second way
# ---------------------------------------------------------------------------------

def _clipped_counts(n, h, w, ho, wo, th, tw, k, s, p):
    """Staged input positions and valid outputs of every tile from clipped intervals
    (numpy, one row per tile) rather than position by position."""
    nty, ntx = ceil(ho / th), ceil(wo / tw)
    ty, tx = np.meshgrid(np.arange(nty), np.arange(ntx), indexing="ij")
    y0, x0 = ty * th * s - p, tx * tw * s - p
    y1, x1 = y0 + (th - 1) * s + k, x0 + (tw - 1) * s + k
    rows = np.clip(y1, 0, h) - np.clip(y0, 0, h)
    cols = np.clip(x1, 0, w) - np.clip(x0, 0, w)
    orow = np.minimum(ho, (ty + 1) * th) - ty * th
    ocol = np.minimum(wo, (tx + 1) * tw) - tx * tw
    return n * int((rows * cols).sum()), n * int((orow * ocol).sum()), n * nty * ntx


SHAPES = [dict(n=2, h=9, w=7, c_in=5, c_mid=6, c_out=7, k=3, stride=1, pad=1),
          dict(n=1, h=11, w=10, c_in=3, c_mid=8, c_out=5, k=5, stride=2, pad=2),
          dict(n=1, h=8, w=8, c_in=4, c_mid=4, c_out=9, k=3, stride=2, pad=0),
          dict(n=3, h=5, w=6, c_in=2, c_mid=3, c_out=2, k=3, stride=1, pad=0)]
TILINGS = [(2, 3, 2), (4, 4, 4), (3, 5, 3), (1, 7, 16)]


@pytest.mark.parametrize("g", SHAPES)
@pytest.mark.parametrize("op", ["dw_pw", "pw", "dw", "pw_dw", "pw_dw_pw", "pw_pw"])
def test_brute_force_against_clipped_intervals(g, op):
    k, s, p = (1, 1, 0) if op in ("pw", "pw_pw") else (g["k"], g["stride"], g["pad"])
    ho, wo = M.out_dim(g["h"], k, s, p), M.out_dim(g["w"], k, s, p)
    ci, cm, co, kk = g["c_in"], g["c_mid"], g["c_out"], k * k
    for th, tw, cob in TILINGS:
        staged, outs, T = _clipped_counts(g["n"], g["h"], g["w"], ho, wo, th, tw, k, s, p)
        last = cm if op in ("pw_dw", "dw") else co
        nb = ceil(last / cob)
        want = {"dw_pw": nb * staged * ci + T * co * ci + T * nb * ci * kk + outs * co,
                "pw": nb * staged * ci + T * co * ci + outs * co,
                "dw": staged * ci + T * ci * kk + outs * ci,
                "pw_dw": nb * staged * ci + T * (cm * ci + cm * kk) + outs * cm,
                "pw_dw_pw": nb * staged * ci + T * nb * (cm * ci + cm * kk) + T * co * cm + outs * co,
                "pw_pw": nb * staged * ci + T * nb * cm * ci + T * co * cm + outs * co}[op]
        assert M.brute_force_bytes(op, g, dict(tile_h=th, tile_w=tw, co_block=cob), 2) == 2 * want


def test_fusion_saves_half_when_widths_match():
    """Sec. I: fusing a DW and a PW of equal widths (weights aside) halves the off-chip
    traffic of the intermediate-free module against the two layers: x + y vs x + 2m + y
    with m = x = y."""
    g = dict(n=1, h=56, w=56, c_in=128, c_mid=128, c_out=128, k=3, stride=1, pad=1)
    fused = M.ideal_bytes("dw_pw", g, 1) - 128 * 9 - 128 * 128
    lbl = M.ideal_bytes("dw", g, 1) - 128 * 9 + M.ideal_bytes("pw", g, 1) - 128 * 128
    assert fused * 2 == lbl


# ---------------------------------------------------------------------------------
# The library planner against the model
# ---------------------------------------------------------------------------------

def _geom(case):
    return dict(n=case.n, h=case.h, w=case.w, c_in=case.c_in, c_mid=case.c_mid, c_out=case.c_out, k=case.k,
                stride=case.stride, pad=case.pad)


def _model_paper(op, g, th, tw, cob, e):
    n, h, w = g["n"], g["h"], g["w"]
    ci, cm, co = g["c_in"], g["c_mid"], g["c_out"]
    k, s, p = (1, 1, 0) if op in ("pw", "pw_pw") else (g["k"], g["stride"], g["pad"])
    ho, wo = M.out_dim(h, k, s, p), M.out_dim(w, k, s, p)
    nty, ntx = ceil(ho / th), ceil(wo / tw)
    T = n * nty * ntx
    ovl = n * M.overlap(w, h, ntx, nty, k, k, s)
    x = n * h * w * ci
    kk = k * k
    if op == "dw_pw":
        v = M.dwpw_gma(ci, ovl, x, ceil(co / cob), T, co * ci, ci * kk, n * ho * wo * co)
    elif op == "pw":
        v = M.pw_gma(co * ci, ceil(co / cob), x, n * h * w * co, T)
    elif op == "dw":
        v = M.dw_gma(ci, ovl, x, n * ho * wo * ci, T, ci * kk)
    elif op == "pw_dw":
        nb = ceil(cm / cob)
        v = M.pwdw_gma(ci, ovl, x, nb, nb, T, cm * ci, T, cm * kk, n * ho * wo * cm)
    elif op == "pw_dw_pw":
        v = M.pwdwpw_gma(ci, ovl, x, ceil(co / cob), T, cm * ci, cm * kk, co * cm, n * ho * wo * co)
    else:
        v = M.pwpw_gma(x, ceil(co / cob), T, cm * ci, co * cm, n * h * w * co)
    return v * e


def _check_plan(op, case, p):
    g, e = _geom(case), ELT[case.dtype]
    assert p.bytes_ideal == M.ideal_bytes(op, g, e)
    name = fcm.variant_name(p.variant)
    if name.startswith("k_pwpw4"):  # register kernel: pixel groups of tile_w pixels
        assert p.bytes_tiled == p.bytes_paper == M.register_pwpw_bytes(g, p.tile_w, e)
        return
    tiling = dict(tile_h=p.tile_h, tile_w=p.tile_w, co_block=p.co_block)
    assert p.bytes_tiled == M.brute_force_bytes(op, g, tiling, e), name
    assert p.bytes_paper == _model_paper(op, g, p.tile_h, p.tile_w, p.co_block, e), name


TINY = []
for i, g in enumerate(SHAPES):
    for dt, lay in (("f32", "nchw"), ("bf16", "nhwc"), ("i8", "nhwc")):
        for op in ("dw_pw", "pw", "dw", "pw_dw", "pw_dw_pw", "pw_pw"):
            gg = dict(g)
            if op in ("dw_pw", "dw"):
                gg["c_mid"] = gg["c_in"]
            if op in ("pw_dw", "dw"):
                gg["c_out"] = gg["c_mid"]
            if op in ("pw", "pw_pw"):
                gg.update(k=1, stride=1, pad=0)
            TINY.append(W.Case(op, **gg, dtype=dt, layout=lay, name="%s-%s-%d" % (op, dt, i)))


@pytest.mark.parametrize("case", TINY, ids=lambda c: c.name)
def test_planner_bytes_equal_the_model_on_tiny_shapes(case):
    d = fcm.desc_from_case(case)
    p = fcm.plan(case.op, d)
    _check_plan(case.op, case, p)
    # and on a few other tilings of the same kernel
    for th, tw in ((1, 4), (2, 8), (4, 4)):
        for cob in (16, 32):
            try:
                q = fcm.plan_evaluate(case.op, d, th, tw, p.c_block, cob, p.variant)
            except fcm.FcmError:
                continue
            _check_plan(case.op, case, q)


WORKLOAD_LAYERS = [c for wl in ("C1", "C2", "C3b1", "C3b32", "C4", "C5", "PWPW") for c in bench.workload_cases(wl)[0]]


@pytest.mark.parametrize("case", WORKLOAD_LAYERS, ids=lambda c: c.name.replace(" ", "_"))
def test_planner_bytes_equal_the_model_on_workload_layers(case):
    d = fcm.desc_from_case(case)
    _check_plan(case.op, case, fcm.plan(case.op, d))
    _check_plan(case.op, case, fcm.plan_limited(case.op, d, 0))
