"""FusePlanner cost model, written out from the paper -- TEST INFRASTRUCTURE.

Only tests/ use this module; the library's planner (csrc/fcm_plan.cpp) shares no code
with it and is checked against it.

arXiv 2404.19331, Sec. IV. Two families of numbers are modelled here:

1. The paper's closed-form global-memory-access estimates:
     Eq. 1  Overlap   (halo elements re-read per channel across tile boundaries)
     Eq. 2  PwGMA     (pointwise layer, layer-by-layer)
     Eq. 3  DwGMA     (depthwise layer, layer-by-layer)
     Eq. 4  PwDwGMA   (PW->DW module)
   and the module equations the paper says are "constructed similarly" (Sec. IV-B)
   but does not print: DwPwGMA and PwDwPwGMA, derived here the same way.

2. A brute-force count of what a tiled kernel moves between global memory and the
   compute unit: every workgroup's staged input region (halo included, clipped at the
   image border), every weight block it loads, and every output element written once.
   Loops visit each tile and each position; no closed form is used.

Readings where the paper is silent or ambiguous (listed in the design notes as well):
  * sizes are in bytes (element count x element size);
  * "ceil(ChannelW/TileW)" in Eq. 1 is the number of tiles along W, i.e.
    ceil(Wo/TW) for an output tile of width TW; batch multiplies the overlap;
  * Eq. 2's weight term uses the number of spatial tiles (ceil(OFMsHW/OFMsTileHW)),
    as Eq. 3 does; the literal variant is kept as ``pw_gma_literal``;
  * Eq. 4 gets the output-write term (+DwOFMsSz) the printed equation omits, and its
    PW-weight term ceil(DwOFMsSz/DwOFMsTileSz) is read, like Eq. 2's, as the number of
    spatial tiles: the workgroups of one spatial tile together read the PW weights once
    (the literal count of output tiles would charge them once per channel block);
  * biases are not counted (the paper's model has none).
"""
from math import ceil


# ----------------------------------------------------------------------------------
# Eq. 1 - 4
# ----------------------------------------------------------------------------------

def overlap(channel_w, channel_h, n_tiles_w, n_tiles_h, filter_w, filter_h, strides):
    """Eq. 1: (tiles_w - 1)*(FilterW - S)*ChannelH + (tiles_h - 1)*(FilterH - S)*ChannelW."""
    return ((n_tiles_w - 1) * (filter_w - strides) * channel_h
            + (n_tiles_h - 1) * (filter_h - strides) * channel_w)


def pw_gma(weights_sz, n_weight_tiles, ifms_sz, ofms_sz, n_spatial_tiles):
    """Eq. 2 with the spatial-tile reading of its weight term."""
    return n_weight_tiles * ifms_sz + ofms_sz + n_spatial_tiles * weights_sz


def pw_gma_literal(weights_sz, weights_tile_sz, ifms_sz, ofms_sz, ofms_tile_sz):
    """Eq. 2 exactly as printed."""
    return ceil(weights_sz / weights_tile_sz) * ifms_sz + ofms_sz + ceil(ofms_sz / ofms_tile_sz) * weights_sz


def dw_gma(ifms_d, ovl, ifms_sz, ofms_sz, n_spatial_tiles, weights_sz):
    """Eq. 3: 2*IFMsD*Overlap + IFMsSz + OFMsSz + ceil(OFMsHW/OFMsTileHW)*WeightsSz."""
    return 2 * ifms_d * ovl + ifms_sz + ofms_sz + n_spatial_tiles * weights_sz


def pwdw_gma(pw_ifms_d, dw_overlap, pw_ifms_sz, n_pw_weight_tiles, n_dw_weight_tiles,
             n_spatial_tiles_x_pw_weight_tiles, pw_weights_sz, n_spatial_tiles, dw_weights_sz,
             dw_ofms_sz):
    """Eq. 4 (+ the output write):
    (2*PwIFMsD*DwOverlap + PwIFMsSz) * max(ceil(PwW/PwWT), ceil(DwW/DwWT))
      + ceil(DwOFMsSz/DwOFMsTileSz) * PwWeightsSz
      + ceil(DwOFMsHW/DwOFMsTileHW) * DwWeightsSz + DwOFMsSz."""
    return ((2 * pw_ifms_d * dw_overlap + pw_ifms_sz) * max(n_pw_weight_tiles, n_dw_weight_tiles)
            + n_spatial_tiles_x_pw_weight_tiles * pw_weights_sz
            + n_spatial_tiles * dw_weights_sz + dw_ofms_sz)


def dwpw_gma(c, dw_overlap, dw_ifms_sz, n_co_blocks, n_spatial_tiles, pw_weights_sz,
             dw_weights_sz, pw_ofms_sz):
    """Derived DW->PW module estimate (Sec. IV-B "constructed similarly"): the DW input
    (with its overlap) is re-read once per output-channel block because the DW output
    is never written out; every spatial tile reads all PW weights once; each workgroup
    reads the DW weights; the output is written once."""
    return ((2 * c * dw_overlap + dw_ifms_sz) * n_co_blocks + n_spatial_tiles * pw_weights_sz
            + n_spatial_tiles * n_co_blocks * dw_weights_sz + pw_ofms_sz)


def pwdwpw_gma(ci, dw_overlap, pw1_ifms_sz, n_co_blocks, n_spatial_tiles, pw1_weights_sz, dw_weights_sz,
               pw2_weights_sz, ofms_sz):
    """Derived PW->DW->PW module estimate (built as Eq. 4): a workgroup owns a spatial tile
    and a block of the last layer's output channels and streams every intermediate
    channel through PW1 and DW itself, so the input (with its overlap), PW1's and DW's
    weights are read once per output-channel block; PW2's weights once per spatial tile
    (its rows are split over the blocks); the output is written once."""
    return ((2 * ci * dw_overlap + pw1_ifms_sz) * n_co_blocks
            + n_spatial_tiles * n_co_blocks * (pw1_weights_sz + dw_weights_sz)
            + n_spatial_tiles * pw2_weights_sz + ofms_sz)


def pwpw_gma(ifms_sz, n_co_blocks, n_spatial_tiles, pw1_weights_sz, pw2_weights_sz, ofms_sz):
    """Derived PW->PW module estimate (as PW->DW->PW without the depthwise layer and its
    overlap): the input and PW1's weights per output-channel block, PW2's weights per
    spatial tile, the output once."""
    return (ifms_sz * n_co_blocks + n_spatial_tiles * n_co_blocks * pw1_weights_sz
            + n_spatial_tiles * pw2_weights_sz + ofms_sz)


# ----------------------------------------------------------------------------------
# Brute-force per-workgroup counting
# ----------------------------------------------------------------------------------

def out_dim(x, k, s, p):
    return (x + 2 * p - k) // s + 1


def _staged_positions(ty, tx, th, tw, k, s, p, h, w):
    """Count input positions inside the image of a tile's haloed input window."""
    ih, iw = (th - 1) * s + k, (tw - 1) * s + k
    iy0, ix0 = ty * th * s - p, tx * tw * s - p
    cnt = 0
    for dy in range(ih):
        for dx in range(iw):
            y, x = iy0 + dy, ix0 + dx
            if 0 <= y < h and 0 <= x < w:
                cnt += 1
    return cnt


def _valid_outputs(ty, tx, th, tw, ho, wo):
    cnt = 0
    for dy in range(th):
        for dx in range(tw):
            if ty * th + dy < ho and tx * tw + dx < wo:
                cnt += 1
    return cnt


def brute_force_bytes(op, g, tiling, elt):
    """Global bytes moved by a tiled kernel, counted workgroup by workgroup.

    op: 'dw_pw' | 'pw' | 'dw' | 'pw_dw' | 'pw_dw_pw' | 'pw_pw'
    g:  dict(n, h, w, c_in, c_mid, c_out, k, stride, pad)
    tiling: dict(tile_h, tile_w, co_block) -- co_block is the output-channel block of the
            last convolution (dw_pw, pw, pw_dw_pw, pw_pw) or the intermediate-channel
            block (pw_dw, dw). A pw_dw_pw / pw_pw workgroup computes every intermediate
            channel of its spatial tile itself, block after block.
    """
    n, h, w = g["n"], g["h"], g["w"]
    ci, cm, co = g["c_in"], g["c_mid"], g["c_out"]
    k, s, p = g["k"], g["stride"], g["pad"]
    th, tw = tiling["tile_h"], tiling["tile_w"]
    if op in ("pw", "pw_pw"):
        k, s, p = 1, 1, 0
    ho, wo = out_dim(h, k, s, p), out_dim(w, k, s, p)
    nty, ntx = ceil(ho / th), ceil(wo / tw)
    total = 0
    for _b in range(n):
        for ty in range(nty):
            for tx in range(ntx):
                pos = _staged_positions(ty, tx, th, tw, k, s, p, h, w)
                outs = _valid_outputs(ty, tx, th, tw, ho, wo)
                if op in ("dw_pw", "pw"):
                    cob = tiling["co_block"]
                    for c0 in range(0, co, cob):
                        ce = min(cob, co - c0)
                        total += pos * ci                       # staged input, all channels
                        total += ce * ci                        # PW weight block
                        if op == "dw_pw":
                            total += ci * k * k                 # DW weights
                        total += outs * ce                      # output block
                elif op in ("dw", "pw_dw"):
                    mb = tiling["co_block"]
                    chans = cm if op == "pw_dw" else ci
                    for m0 in range(0, chans, mb):
                        me = min(mb, chans - m0)
                        if op == "pw_dw":
                            total += pos * ci + me * ci         # all input channels + PW block
                        else:
                            total += pos * me                   # this channel block only
                        total += me * k * k + outs * me
                elif op in ("pw_dw_pw", "pw_pw"):
                    cob = tiling["co_block"]
                    for c0 in range(0, co, cob):
                        ce = min(cob, co - c0)
                        total += pos * ci + cm * ci             # staged input, all of PW1
                        if op == "pw_dw_pw":
                            total += cm * k * k                 # all DW weights
                        total += ce * cm + outs * ce            # PW2 rows of the block, output
                else:
                    raise ValueError(op)
    return total * elt


def register_pwpw_bytes(g, pixels_per_group, elt):
    """PW->PW on pixel groups (the register-resident kernel: a group of pixels in one
    wave with every channel): input and output once, both weight matrices once per
    group, counted group by group."""
    npix = g["n"] * g["h"] * g["w"]
    ci, cm, co = g["c_in"], g["c_mid"], g["c_out"]
    total = 0
    for p0 in range(0, npix, pixels_per_group):
        px = min(pixels_per_group, npix - p0)
        total += px * (ci + co) + cm * ci + co * cm
    return total * elt


def ideal_bytes(op, g, elt):
    """What the module must move at least: input + all weights + output (bytes)."""
    n, h, w = g["n"], g["h"], g["w"]
    ci, cm, co = g["c_in"], g["c_mid"], g["c_out"]
    k, s, p = g["k"], g["stride"], g["pad"]
    if op == "pw":
        return (n * h * w * ci + co * ci + n * h * w * co) * elt
    if op == "pw_pw":
        return (n * h * w * ci + cm * ci + co * cm + n * h * w * co) * elt
    ho, wo = out_dim(h, k, s, p), out_dim(w, k, s, p)
    x = n * h * w * ci
    if op == "dw":
        return (x + ci * k * k + n * ho * wo * ci) * elt
    if op == "dw_pw":
        return (x + ci * k * k + co * ci + n * ho * wo * co) * elt
    if op == "pw_dw":
        return (x + cm * ci + cm * k * k + n * ho * wo * cm) * elt
    if op == "pw_dw_pw":
        return (x + cm * ci + cm * k * k + co * cm + n * ho * wo * co) * elt
    raise ValueError(op)
