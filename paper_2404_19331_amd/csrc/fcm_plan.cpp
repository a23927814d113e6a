// fcm_plan.cpp -- FusePlanner for CDNA4 (arXiv 2404.19331, Sec. IV).
//
// For a module and a tiling, three global-memory figures are computed:
//   * bytes_ideal: what the module must move at least (input + weights + output once);
//   * bytes_tiled: what the tiled kernel loads and stores, workgroup by workgroup: the
//     haloed input window of every workgroup clipped at the image border, the weight
//     blocks each workgroup stages, and each output once. This is exact for the kernels
//     in this library (sums of per-axis clipped extents);
//   * bytes_paper: the paper's closed-form estimate: Eq. 1 (overlap), Eq. 2 (PW),
//     Eq. 3 (DW), Eq. 4 (PW->DW) and the DW->PW / PW->DW->PW estimates built the same
//     way (Sec. IV-B says the other modules follow the same construction).
// The search enumerates the tilings the compiled kernels implement, keeps those whose
// LDS footprint fits a workgroup (the paper's "tiles fit in L1/shared memory"
// constraint), prefers tilings with at least one workgroup per CU (the paper's
// "#tiles >= #SMs"), and minimises bytes_tiled. The fuse verdict compares the module's
// estimate with the layer-by-layer chain's (Sec. IV-B: fuse when the fused estimate is
// lower).
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "fcm_host.h"

namespace fcm {

fcm_hw_desc default_hw() {
  fcm_hw_desc hw;
  hw.num_cus = 256;
  hw.num_xcds = 8;
  hw.wave_size = 64;
  hw.lds_per_wg = kMaxLdsPerWg;
  hw.lds_per_cu = kMaxLdsPerWg;
  hw.l2_per_xcd = 4ll << 20;
  hw.mall_bytes = 256ll << 20;
  hw.hbm_bytes_per_s = 8.0e12;
  return hw;
}

static int out_dim(int x, int k, int s, int p) { return (x + 2 * p - k) / s + 1; }

Geom geometry(int op, const fcm_desc* d) {
  Geom g = {};
  g.op = op;
  int8_features(op, d, &g.zp, &g.pc);
  g.n = d->n;
  g.h = d->h;
  g.w = d->w;
  g.dtype = d->dtype;
  g.elt = elt_size(d->dtype);
  g.layout = d->layout;
  g.k = d->k;
  g.s = d->stride;
  g.pad = d->pad;
  switch (op) {
    case FCM_OP_DW_PW: g.family = FAM_DWPW; g.ci = d->c_in; g.cm = d->c_in; g.co = d->c_out; break;
    case FCM_OP_PW_DW: g.family = FAM_PWDW; g.ci = d->c_in; g.cm = d->c_mid; g.co = d->c_mid; break;
    case FCM_OP_PW_DW_PW: g.family = FAM_PWDWPW; g.ci = d->c_in; g.cm = d->c_mid; g.co = d->c_out; break;
    case FCM_OP_DW: g.family = FAM_DW; g.ci = d->c_in; g.cm = d->c_in; g.co = d->c_in; break;
    case FCM_OP_PW_PW:
      g.family = FAM_PWPW; g.ci = d->c_in; g.cm = d->c_mid; g.co = d->c_out; g.k = 1; g.s = 1; g.pad = 0;
      break;
    default: g.family = FAM_PW; g.ci = d->c_in; g.cm = d->c_in; g.co = d->c_out; g.k = 1; g.s = 1; g.pad = 0; break;
  }
  g.ho = out_dim(g.h, g.k, g.s, g.pad);
  g.wo = out_dim(g.w, g.k, g.s, g.pad);
  return g;
}

// Sum over tiles t of |[t*T*S - P, t*T*S - P + (T-1)*S + K) intersected with [0, X)|:
// the input rows (or columns) staged by all tiles along one axis.
static int64_t staged_extent_sum(int X, int XO, int T, int K, int S, int P) {
  const int nt = ceil_div(XO, T);
  const int ext = (T - 1) * S + K;
  int64_t sum = 0;
  for (int t = 0; t < nt; ++t) {
    const int lo = std::max(0, t * T * S - P), hi = std::min(X, t * T * S - P + ext);
    if (hi > lo) sum += hi - lo;
  }
  return sum;
}

// Eq. 1 overlap, in elements per channel (and per image): (tiles_w - 1)(K - S) H +
// (tiles_h - 1)(K - S) W; number of tiles along an axis = tiles covering the output.
static int64_t eq1_overlap(int H, int W, int nty, int ntx, int K, int S) {
  return (int64_t)(ntx - 1) * (K - S) * H + (int64_t)(nty - 1) * (K - S) * W;
}

struct Bytes {
  int64_t ideal, tiled, paper;
  double redundancy;
};

static Bytes module_bytes(const Geom& g, int TH, int TW, int COB) {
  const int64_t e = g.elt, N = g.n;
  const int nty = ceil_div(g.ho, TH), ntx = ceil_div(g.wo, TW);
  const int64_t T = N * nty * ntx;  // spatial tiles
  const int64_t SR = staged_extent_sum(g.h, g.ho, TH, g.k, g.s, g.pad);
  const int64_t SC = staged_extent_sum(g.w, g.wo, TW, g.k, g.s, g.pad);
  const int64_t staged = N * SR * SC;  // staged input positions over all spatial tiles
  const int64_t x_el = N * g.h * g.w * (int64_t)g.ci;
  const int64_t kk = (int64_t)g.k * g.k;
  const int64_t ovl = N * eq1_overlap(g.h, g.w, nty, ntx, g.k, g.s);
  Bytes b = {};
  switch (g.family) {
    case FAM_DWPW: {
      const int64_t ncb = ceil_div(g.co, COB);
      const int64_t y_el = N * g.ho * (int64_t)g.wo * g.co;
      b.ideal = (x_el + g.ci * kk + (int64_t)g.co * g.ci + y_el) * e;
      b.tiled = (ncb * staged * g.ci + T * (int64_t)g.co * g.ci + T * ncb * g.ci * kk + y_el) * e;
      b.paper = ((2 * g.ci * ovl + x_el) * ncb + T * (int64_t)g.co * g.ci + T * ncb * g.ci * kk + y_el) * e;
      break;
    }
    case FAM_PW: {
      const int64_t ncb = ceil_div(g.co, COB);
      const int64_t y_el = N * g.h * (int64_t)g.w * g.co;
      b.ideal = (x_el + (int64_t)g.co * g.ci + y_el) * e;
      b.tiled = (ncb * staged * g.ci + T * (int64_t)g.co * g.ci + y_el) * e;
      // Eq. 2 (weight term counted per spatial tile)
      b.paper = (ncb * x_el + y_el + T * (int64_t)g.co * g.ci) * e;
      break;
    }
    case FAM_DW: {
      const int64_t y_el = N * g.ho * (int64_t)g.wo * g.ci;
      b.ideal = (x_el + g.ci * kk + y_el) * e;
      b.tiled = (staged * g.ci + T * g.ci * kk + y_el) * e;
      // Eq. 3
      b.paper = (2 * g.ci * ovl + x_el + y_el + T * g.ci * kk) * e;
      break;
    }
    case FAM_PWDW: {
      const int64_t nmb = ceil_div(g.cm, COB);
      const int64_t y_el = N * g.ho * (int64_t)g.wo * g.cm;
      b.ideal = (x_el + (int64_t)g.cm * g.ci + g.cm * kk + y_el) * e;
      b.tiled = (nmb * staged * g.ci + T * ((int64_t)g.cm * g.ci + g.cm * kk) + y_el) * e;
      // Eq. 4 (+ output write); both weight-tile counts are the mid-channel blocks
      b.paper = ((2 * g.ci * ovl + x_el) * nmb + T * (int64_t)g.cm * g.ci + T * g.cm * kk + y_el) * e;
      b.redundancy = (double)(SR * SC) / ((double)g.h * g.w) - 1.0;
      break;
    }
    case FAM_PWPW: {
      // as PW->DW->PW without the depthwise weights and halo: x per output-channel block,
      // the first layer's weights per tile and block, the second's per tile
      const int64_t ncb = ceil_div(g.co, COB);
      const int64_t y_el = N * g.h * (int64_t)g.w * g.co;
      b.ideal = (x_el + (int64_t)g.cm * g.ci + (int64_t)g.co * g.cm + y_el) * e;
      b.tiled = (ncb * staged * g.ci + T * ncb * (int64_t)g.cm * g.ci + T * (int64_t)g.co * g.cm + y_el) * e;
      b.paper = (ncb * x_el + T * ncb * (int64_t)g.cm * g.ci + T * (int64_t)g.co * g.cm + y_el) * e;
      break;
    }
    case FAM_PWDWPW: {
      const int64_t ncb = ceil_div(g.co, COB);
      const int64_t y_el = N * g.ho * (int64_t)g.wo * g.co;
      b.ideal = (x_el + (int64_t)g.cm * g.ci + g.cm * kk + (int64_t)g.co * g.cm + y_el) * e;
      b.tiled = (ncb * staged * g.ci + T * ncb * ((int64_t)g.cm * g.ci + g.cm * kk) + T * (int64_t)g.co * g.cm +
                 y_el) * e;
      b.paper = ((2 * g.ci * ovl + x_el) * ncb + T * ncb * ((int64_t)g.cm * g.ci + g.cm * kk) +
                 T * (int64_t)g.co * g.cm + y_el) * e;
      b.redundancy = (double)(SR * SC) / ((double)g.h * g.w) - 1.0;
      break;
    }
  }
  return b;
}

// Ring depth of a persistent kernel: the caller's `want` (2..8), else 3 buffers (two
// items in flight) where they fit, else 2. Every depth keeps the partial wait on the
// copies of the items in flight (per copy wave) within the 6-bit vector-memory counter.
// 0 if `want` is invalid.
static int ring_depth3(int want, int buf, int per_item, int lds_per_wg) {
  const int dmax = std::min(kMaxDepth3, 63 / per_item + 2);
  if (want > 0) return (want >= 2 && want <= dmax && want * buf <= lds_per_wg) ? want : 0;
  return (dmax >= 3 && 3 * buf <= lds_per_wg) ? 3 : 2;
}

// Workspace bytes of a split plan: fp32 / int32 partial sums [split][work tile][TH*TW][COB].
static int64_t split_workspace_bytes(int64_t tiles, int pixels, int cob, int splits) {
  return (int64_t)splits * tiles * pixels * cob * 4;
}

int64_t plan_workspace_bytes(const Geom& g, const fcm_plan_t& p) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  if (p.variant < 0 || p.variant >= nv || vs[p.variant].gen != 3 || p.splits <= 1) return 0;
  const int last = (g.family == FAM_PWDW || g.family == FAM_DW) ? g.cm : g.co;
  const int64_t tiles =
      (int64_t)g.n * ceil_div(g.ho, p.tile_h) * ceil_div(g.wo, p.tile_w) * ceil_div(last, p.co_block);
  return split_workspace_bytes(tiles, p.tile_h * p.tile_w, p.co_block, p.splits);
}

// LDS bytes of a tiling (0 if the variant cannot implement it). For the persistent
// kernels *depth is the requested ring depth on input (0 = choose) and the chosen one on
// output.
static int tiling_lds(const Variant& v, const Geom& g, int TH, int TW, int CB, int COB, int lds_per_wg,
                      int* depth) {
  const int kb = k_block(g.dtype);
  if (TH <= 0 || TW <= 0 || COB <= 0 || COB % 16) return 0;
  if (v.dw_r && TW % v.dw_r) return 0;
  if (v.gen != 6 && COB > v.max_cob) return 0;  // (gen 6: every channel, bounded by LDS)
  const int P = TH * TW;
  const int Q = ((TH - 1) * g.s + g.k) * ((TW - 1) * g.s + g.k);
  if (v.max_p && P > v.max_p) return 0;
  if (v.gen < 3 && v.max_q && Q > v.max_q) return 0;
  if (v.gen == 6) {
    // the compiled tile and every channel of the last convolution in one workgroup
    const int last = (g.family == FAM_PWDW || g.family == FAM_DW) ? g.cm : g.co;
    if (TH != v.tile_h || TW != v.tile_w || COB != round_up(last, 16)) return 0;
    // flat 16-byte weight copies: input and depthwise channels in fours
    if (g.ci % 4 || (g.family != FAM_DWPW && g.cm % 4)) return 0;
    const int mode = g.family == FAM_DWPW ? M6_DWPW : (g.family == FAM_PWDW ? M6_PWDW : M6_PWDWPW);
    const int64_t bytes = 4 * (int64_t)lds6(mode, g.k, g.s, TH, TW, g.ci, g.cm, g.co).floats;
    return bytes > lds_per_wg ? lds_per_wg + 1 : (int)bytes;
  }
  if (v.gen == 7) {
    // NHWC, input channels in whole 32-channel chunks, whole 16-byte output granules,
    // images and weights below 2^30 bytes (32-bit buffer offsets with room for an
    // out-of-range scalar part), the compiled tile and channel block
    if (g.layout != FCM_NHWC || g.family != FAM_DWPW) return 0;
    if (g.ci % (32 * v.kc) || (g.co * g.elt) % 16) return 0;
    if ((int64_t)g.h * g.w * g.ci * g.elt >= ((int64_t)1 << 30)) return 0;
    if ((int64_t)g.ho * g.wo * g.co * g.elt >= ((int64_t)1 << 30)) return 0;
    if ((int64_t)(g.co + COB) * g.ci * g.elt >= ((int64_t)1 << 30)) return 0;
    if (CB != 64 / g.elt || COB != v.max_cob || TH != v.tile_h || TW != v.tile_w) return 0;
    return lds7(g.s, TH, TW, v.max_cob / 64, g.ci, v.kc).total;
  }
  if (v.gen == 5) {
    // NHWC, 16-byte input channel rows, 32-bit buffer offsets, 64-byte chunk, run-time
    // tile of at most max_p pixels whose window fits the kernel's copy list
    if (g.layout != FCM_NHWC) return 0;
    const bool dw_only = g.family == FAM_DW;
    const int cin = dw_only ? g.cm : g.ci;
    if ((cin * g.elt) % 16) return 0;
    if (dw_only ? (g.cm * g.elt) % 16 : (g.co * g.elt) % 4) return 0;
    if ((int64_t)g.h * g.w * cin * g.elt >= ((int64_t)1 << 31)) return 0;
    if (!dw_only && (int64_t)(g.co + COB) * g.ci * g.elt >= ((int64_t)1 << 31)) return 0;
    if (CB != 64 / g.elt || COB != v.max_cob || TH != v.tile_h || TW != v.tile_w) return 0;
    const int mode = g.family == FAM_DWPW ? M3_DWPW : (g.family == FAM_PW ? M3_PW : M3_DW);
    const int KE = mode == M3_PW ? 1 : g.k, SE = mode == M3_PW ? 1 : g.s;
    const int IH = (TH - 1) * SE + KE, IW = (TW - 1) * SE + KE;
    if (round_up(IH * IW, 32) > 512) return 0;  // window copies: 8 per wave at most
    const bool share = mode == M3_DWPW && v.wc > 1;
    const int wp = 4 / v.wc, nbt = ((P + 15) / 16 + wp - 1) / wp * wp;  // pixel blocks, as the kernel
    return lds5(g.dtype, mode, KE, IH, IW, COB, v.ks, share ? 16 * nbt : 0).total;
  }
  if (v.gen == 3) {
    // NHWC, 16-byte input channel rows, 32-bit buffer offsets, 64-byte chunk, run-time
    // tile whose input window fits the kernel's LDS row pitch
    if (g.layout != FCM_NHWC) return 0;
    const bool dw_only = g.family == FAM_DW;
    const int cin = dw_only ? g.cm : g.ci;
    if ((cin * g.elt) % 16) return 0;
    if (dw_only ? (g.cm * g.elt) % 16 : (g.co * g.elt) % 4) return 0;
    if ((int64_t)g.h * g.w * cin * g.elt >= ((int64_t)1 << 31)) return 0;
    // weight rows up to the last block's padding are addressed with 32-bit offsets
    if (!dw_only && (int64_t)(g.co + COB) * g.ci * g.elt >= ((int64_t)1 << 31)) return 0;
    if (CB != 64 / g.elt || COB != v.max_cob) return 0;
    if (P > v.max_p) return 0;
    const int mode = g.family == FAM_DWPW ? M3_DWPW : (g.family == FAM_PW ? M3_PW : M3_DW);
    const int IW = mode == M3_PW ? TW : (TW - 1) * g.s + g.k;
    const int IH = mode == M3_PW ? TH : (TH - 1) * g.s + g.k;
    if (IW > v.pitch) return 0;
    const int KE = mode == M3_PW ? 1 : g.k;
    const int per_item = copies_per_wave3(mode, KE, IH, v.pitch, COB / 16, v.ks, g.pc);
    if (per_item > 63) return 0;
    const int buf = lds3p(g.dtype, KE, mode, IH, v.pitch, COB / 16, 2, v.ks, g.pc).buf_bytes;
    const int d = ring_depth3(*depth, buf, per_item, lds_per_wg);
    if (d == 0) return 0;
    *depth = d;
    return lds3p(g.dtype, KE, mode, IH, v.pitch, COB / 16, d, v.ks, g.pc).total;
  }
  switch (v.family) {
    case FAM_DWPW:
    case FAM_PW:
      if (CB <= 0 || CB % kb) return 0;
      return lds_layout_dwpw(g.dtype, g.k, g.s, v.family == FAM_DWPW, TH, TW, CB, COB).bytes;
    case FAM_PWDW:
      if (CB <= 0 || CB % kb) return 0;
      return lds_layout_pwdw(g.dtype, g.k, g.s, true, TH, TW, CB, COB).bytes;
    case FAM_DW:
      if (CB != COB) return 0;
      return lds_layout_pwdw(g.dtype, g.k, g.s, false, TH, TW, CB, COB).bytes;
    case FAM_PWDWPW:
    case FAM_PWPW:
      // CB = intermediate chunk: a multiple of both the MFMA M tile and its K step
      if (CB <= 0 || CB % 16 || CB % kb || CB > v.max_mb) return 0;
      return lds_layout_pwdwpw(g.dtype, g.k, g.s, TH, TW, g.ci, CB, COB).bytes;
  }
  return 0;
}

bool variant_needs_alignment(int variant) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  return variant >= 0 && variant < nv && vs[variant].gen >= 2;
}

// Generations 2 and up need the full set; with zero points (KSET_REG) also the int8
// persistent kernels and the register kernel's instances of at most kZpMaxTiles output
// tiles; with per-channel requantisation (KSET_PC) the int8 persistent kernels.
static bool in_set(const Variant& v, int kset) {
  if (v.gen < 2) return true;
  if (kset == KSET_PC) return v.gen == 3 && v.dtype == DT_I8;
  if (kset & KSET_DMA) return true;
  if (!(kset & KSET_REG)) return false;
  return (v.gen == 3 && v.dtype == DT_I8) || (v.gen == 4 && v.max_cob <= 16 * kZpMaxTiles);
}

bool variant_in_set(int variant, int kset) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  return variant >= 0 && variant < nv && in_set(vs[variant], kset);
}

static bool variant_matches(const Variant& v, const Geom& g) {
  if (v.family != g.family || v.dtype != g.dtype) return false;
  if (g.family == FAM_PW) return true;
  return v.k == g.k && v.stride == g.s;
}

// Pixel groups of the PW -> PW register kernel (gen 4): one wave each.
static int64_t pixel_groups4(const Variant& v, const Geom& g) {
  return ceil_div((int64_t)g.n * g.h * g.w, (int64_t)v.max_p);
}

// LDS bytes of the PW -> PW register kernel: with splits > 1 the four waves' partial
// sums, [wave][pixel block][output tile][64 lanes] of 16 bytes.
static int lds_bytes4(const Variant& v, const Geom& g, int splits) {
  return splits > 1 ? 4 * (v.max_p / 16) * ceil_div(g.co, 16) * 1024 : 0;
}

// Plan of the PW -> PW register kernel: its tiling is fixed by the variant (pixel groups of
// max_p pixels, 64-byte intermediate chunks, every output channel); only the number of
// waves sharing a pixel group's intermediate chunks (1, 2 or 4, in one workgroup) is chosen.
static fcm_status evaluate_plan4(const Variant& v, const Geom& g, const fcm_hw_desc& hw, fcm_plan_t* p) {
  const int e = g.elt;
  if (g.layout != FCM_NHWC) return fail(FCM_EUNSUPPORTED, "plan: the register kernel needs NHWC");
  if ((g.ci * e) % 4 || (g.cm * e) % 4 || g.co % 4)
    return fail(FCM_EUNSUPPORTED, "plan: the register kernel needs 4-byte channel rows and output channels in fours");
  if (g.ci * e > 64 * v.ks || g.co > v.max_cob)
    return fail(FCM_EUNSUPPORTED, "plan: channels exceed what the kernel variant holds in registers");
  if (p->tile_h != 1 || p->tile_w != v.max_p || p->c_block != 64 / e || p->co_block != round_up(g.co, 16))
    return fail(FCM_EUNSUPPORTED, "plan: tiling not implemented by the kernel variant");
  const int64_t npix = (int64_t)g.n * g.h * g.w;
  // buffer addressing: 32-bit byte offsets below 2^31 for x, y and both weight matrices
  const int64_t lim = (int64_t)1 << 31;
  if (npix * std::max(g.ci, g.co) * (int64_t)e >= lim || (int64_t)g.cm * g.ci * e >= lim ||
      (int64_t)g.co * g.cm * e >= lim || npix + v.max_p >= (1 << 30))
    return fail(FCM_EUNSUPPORTED, "plan: tensor too large for the register kernel");
  const int64_t npg = pixel_groups4(v, g);
  const int nch = ceil_div(g.cm * e, 64);
  const int splits = std::max(1, (int)p->splits);
  if (splits != 1 && splits != 2 && splits != 4)
    return fail(FCM_EUNSUPPORTED, "plan: the register kernel splits over 1, 2 or 4 waves");
  if (splits > nch) return fail(FCM_EUNSUPPORTED, "plan: more splits than intermediate channel chunks");
  const int lds = lds_bytes4(v, g, splits);
  if (lds > hw.lds_per_wg) return fail(FCM_EUNSUPPORTED, "plan: partial sums exceed the LDS per workgroup");
  const int64_t grid = ceil_div(npg, (int64_t)(4 / splits));
  if (grid > 0x7fffffff) return fail(FCM_EUNSUPPORTED, "plan: grid too large");
  // bytes: x and y once, both weight matrices once per pixel group (Eq. 1 style: every
  // output tile convolves with all filters)
  const int64_t w_el = (int64_t)g.cm * g.ci + (int64_t)g.co * g.cm;
  const int64_t xy_el = npix * (g.ci + g.co);
  p->bytes_ideal = (xy_el + w_el) * e;
  p->bytes_paper = (xy_el + npg * w_el) * e;
  p->bytes_tiled = p->bytes_paper;
  p->redundancy = 0.0;
  p->workgroups = (int32_t)grid;
  p->depth = 0;
  p->splits = splits;
  p->waves = 4;
  p->lds_bytes = lds;
  return FCM_OK;
}

fcm_status evaluate_plan(const Geom& g, const fcm_desc* d, const fcm_hw_desc& hw, fcm_plan_t* p) {
  (void)d;
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  if (p->variant < 0 || p->variant >= nv) return fail(FCM_EUNSUPPORTED, "plan: unknown kernel variant");
  const Variant& v = vs[p->variant];
  if (!variant_matches(v, g)) return fail(FCM_EUNSUPPORTED, "plan: kernel variant does not implement this module");
  if (v.gen == 4) return evaluate_plan4(v, g, hw, p);
  int depth = v.gen == 3 ? p->depth : 0;
  const int lds = tiling_lds(v, g, p->tile_h, p->tile_w, p->c_block, p->co_block, hw.lds_per_wg, &depth);
  if (lds <= 0) return fail(FCM_EUNSUPPORTED, "plan: tiling not implemented by the kernel variant");
  if (lds > hw.lds_per_wg) return fail(FCM_EUNSUPPORTED, "plan: tiling exceeds the LDS per workgroup");
  const int nty = ceil_div(g.ho, p->tile_h), ntx = ceil_div(g.wo, p->tile_w);
  const int last = (g.family == FAM_PWDW || g.family == FAM_DW) ? g.cm : g.co;
  const int64_t wgs = (int64_t)g.n * nty * ntx * ceil_div(last, p->co_block);
  if (wgs <= 0 || wgs > 0x7fffffff) return fail(FCM_EUNSUPPORTED, "plan: grid too large");
  const Bytes b = module_bytes(g, p->tile_h, p->tile_w, p->co_block);
  if (v.gen != 3 && p->splits > 1) return fail(FCM_EUNSUPPORTED, "plan: this kernel variant does not split");
  if (v.gen == 5 || v.gen == 7) {
    // persistent: the workgroups resident at once (LDS-limited estimate; the launcher
    // also applies the compiled kernel's register-limited occupancy), at most one per
    // work tile; a caller's cap is kept
    // (the deep kernels' eight waves hold every VGPR of a CU: one workgroup per CU)
    const int64_t per_cu =
        v.gen == 7 ? 1 : std::max<int64_t>(1, std::min<int64_t>(8, hw.lds_per_cu / lds));
    int64_t grid = std::min<int64_t>(wgs, per_cu * hw.num_cus);
    if (p->workgroups > 0 && p->workgroups < grid) grid = p->workgroups;
    if (v.gen == 7) {  // as launched: a multiple of the output-channel blocks
      const int64_t ncb = ceil_div(g.co, p->co_block);
      grid = std::max<int64_t>(ncb, grid - grid % ncb);
    }
    p->workgroups = (int32_t)grid;
    p->depth = v.ks;
    p->splits = 1;
    p->waves = v.gen == 7 ? 8 : 4;
    p->lds_bytes = lds;
    p->bytes_ideal = b.ideal;
    p->bytes_tiled = b.tiled;
    p->bytes_paper = b.paper;
    p->redundancy = b.redundancy;
    return FCM_OK;
  }
  if (v.gen == 3) {
    const int splits = p->splits > 1 ? p->splits : 1;
    if (splits > 1) {
      if (v.family == FAM_DW) return fail(FCM_EUNSUPPORTED, "plan: a depthwise-only kernel does not split");
      const int ipt = ceil_div(g.ci, v.ks * (64 / g.elt));
      if (!splits_valid3(ipt, splits)) return fail(FCM_EUNSUPPORTED, "plan: more splits than channel chunks");
      if (split_workspace_bytes(wgs, p->tile_h * p->tile_w, p->co_block, splits) > FCM_SPLIT_WORKSPACE_BYTES)
        return fail(FCM_EUNSUPPORTED, "plan: split workspace too large");
    }
    // persistent: the workgroups resident at once (LDS-limited estimate; the launcher
    // also applies the compiled kernel's register-limited occupancy), at most one per
    // work unit (work tile x split)
    const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(8, hw.lds_per_cu / lds));
    int64_t grid = std::min<int64_t>(wgs * splits, per_cu * hw.num_cus);
    if (p->workgroups > 0 && p->workgroups < grid) grid = p->workgroups;  // caller's cap
    p->workgroups = (int32_t)grid;
    p->depth = depth;
    p->splits = splits;
    p->waves = 4;
    p->lds_bytes = lds;
    p->bytes_ideal = b.ideal;
    p->bytes_tiled = b.tiled;
    p->bytes_paper = b.paper;
    p->redundancy = b.redundancy;
    return FCM_OK;
  }
  p->waves = 4;
  p->depth = 0;
  p->splits = 1;
  p->lds_bytes = lds;
  p->workgroups = (int32_t)wgs;
  p->bytes_ideal = b.ideal;
  p->bytes_tiled = b.tiled;
  p->bytes_paper = b.paper;
  p->redundancy = b.redundancy;
  return FCM_OK;
}

// ---------------------------------------------------------------------------------
// Search
// ---------------------------------------------------------------------------------

// Time model of a persistent (gen 3) kernel launch, in seconds. Each workgroup runs a
// pipeline of items (tile x ks channel chunks of 64 bytes): two copy waves issue the
// LDS copies of items i+1 .. i+depth-1 while four compute waves run item i, so an item
// costs the largest of: the busiest compute wave's depthwise dot instructions
// (workgroups sharing a CU share its SIMDs), the LDS bytes the compute waves read, the
// busier copy wave's copy instructions, and the item's copy bytes at the CU's copy rate,
// which is capped and limited by the bytes in flight (Little's law). Launch overhead is
// added and the launch is never faster than its HBM traffic. The constants were fitted
// (least squares on log time, then on the quality of the chosen plans) to timings of
// every plan of the MobileNetV1, ViT-projection and MBConv DW->PW layers on MI355X,
// unsplit and split (global search over the constants for the quality of the chosen
// plans). A split plan adds its partial sums' round trip and the second kernel.
static double persistent_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p,
                                       const fcm_hw_desc& hw) {
  constexpr double kItem0 = 332.0;        // cycles per item, fixed (busiest compute wave)
  constexpr double kPerDot = 11.2;        // cycles per depthwise dot instruction
  constexpr double kPerMfma = 29.4;       // cycles per MFMA instruction
  constexpr double kPerLdsKiB = 10.5;     // cycles per KiB read from LDS by the compute waves
  constexpr double kPerCopy = 115.2;      // cycles per 1 KiB copy instruction (one copy wave)
  constexpr double kCopy0 = 257.0;        // cycles per item, fixed (copy wave)
  constexpr double kShallow = 189.0;      // cycles per item lost with one item in flight
  constexpr double kLaunch = 16820.0;     // cycles of launch, prologue and drain
  constexpr double kHbm = 4.26e12;        // bytes/s
  constexpr double kCuRate = 13.2;        // copy bytes per cycle and CU, at most
  constexpr double kLatency = 578.0;      // cycles: copy bytes in flight / rate
  constexpr double kClock = 2.4e9;
  constexpr double kCombineLaunch = 8800.0;  // cycles: second kernel of a split plan
  const bool has_dw = v.family != FAM_PW, has_pw = v.family != FAM_DW;
  const int K = has_dw ? g.k : 1, S = has_dw ? g.s : 1;
  const int P = p.tile_h * p.tile_w;
  const int bpw = std::max(1, v.max_p / 64);
  const int nbt = ceil_div(P, 16);
  const int ct = has_pw ? p.co_block / 16 : 0;
  int nb_max = 0;  // pixel blocks of the busiest compute wave
  double lds_kib = 0;  // LDS KiB the compute waves read per chunk
  for (int w = 0; w < 4; ++w) {
    int n = 0;
    for (int b = 0; b < bpw; ++b) n += (b * 4 + w < nbt) ? 1 : 0;
    nb_max = std::max(nb_max, n);
    if (n > 0) lds_kib += (double)K * K * n + (has_dw ? K * K * (4 / g.elt) : 0) + ct;
  }
  const int cin = v.family == FAM_DW ? g.cm : g.ci;
  const int splits = std::max(1, p.splits);
  const int nchunks = v.family == FAM_DW ? 1 : items_per_split3(ceil_div(cin, v.ks * 64 / g.elt), splits);  // items per unit
  const int last = v.family == FAM_DW ? g.cm : g.co;
  const int64_t ntile = (int64_t)g.n * ceil_div(g.ho, p.tile_h) * ceil_div(g.wo, p.tile_w) * ceil_div(last, p.co_block);
  const int64_t nwork = ntile * splits;  // work units
  const int IH = has_dw ? (p.tile_h - 1) * S + K : p.tile_h;
  const int mode = v.family == FAM_DWPW ? M3_DWPW : (v.family == FAM_PW ? M3_PW : M3_DW);
  const double dots = has_dw ? (double)v.ks * nb_max * K * K * (16 / g.elt) : 0.0;
  const double mfmas = (double)v.ks * nb_max * ct * (g.elt == 4 ? 4 : 1);
  const double comp = kItem0 + kPerDot * dots + kPerMfma * mfmas;
  const double lds = kPerLdsKiB * v.ks * lds_kib;
  const double prod = kCopy0 + kPerCopy * copies_per_wave3(mode, K, IH, v.pitch, ct, v.ks, g.pc);
  const double item_bytes = 1024.0 * copies_per_item3(mode, K, IH, v.pitch, ct, v.ks, g.pc);
  const int64_t grid = std::max<int64_t>(1, p.workgroups);
  const double wpc = std::max(1.0, (double)grid / hw.num_cus);
  const int depth = std::max(2, p.depth);
  const double rate = std::min(kCuRate, wpc * (depth - 1) * item_bytes / kLatency);
  const double per = std::max(std::max(comp * wpc, lds * wpc), std::max(prod, item_bytes * wpc / rate)) +
                     (depth == 2 ? kShallow : 0.0);
  const double ipw = (double)ceil_div((int)std::min<int64_t>(nwork, 1 << 30), (int)grid) * nchunks;
  double t_pipe = (ipw * per + kLaunch) / kClock;
  double t_mem = (double)p.bytes_tiled / kHbm;
  if (splits > 1) {
    // partial sums out and back in, and the second kernel
    const double ws = (double)split_workspace_bytes(ntile, P, p.co_block, splits);
    t_pipe += kCombineLaunch / kClock + ws / kHbm;
    t_mem += 2.0 * ws / kHbm;
  }
  // (the pipeline term breaks ties between traffic-bound tilings)
  return std::max(t_pipe, t_mem) + 1e-3 * t_pipe;
}

// Time model of a streaming (gen 5) kernel launch, in seconds. A workgroup runs its items
// (work tile x 64-byte channel chunk) one after another with the next item's copies in
// flight, so a launch costs its items per workgroup times a per-item cost: fixed work,
// the busiest wave's depthwise dot instructions, its MFMAs, the copy instructions of the
// item, the epilogue's share per item and the exchange barrier of a channel-split tile,
// scaled by how many workgroups share a CU; never faster than the module's HBM bytes.
// Constants fitted (least squares on log time) to 329 timed plans of the MobileNetV1
// (batch 1 and 32) and ViT-projection DW->PW layers on MI355X: within about 0.89-1.11x
// of the timings for 80% of them.
static double streaming_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw) {
  constexpr double kLaunchUs = 4.0;
  constexpr double kItem = 773.7, kPerDot = 7.54, kPerMfma = 39.0, kPerCopy = 42.1, kPerEpi = 381.3;
  constexpr double kShareExp = 0.649;
  constexpr double kClockMHz = 2400.0, kHbm = 5.2e12, kLaunchFloorUs = 2.5;
  const bool has_dw = v.family != FAM_PW, has_pw = v.family != FAM_DW;
  const int K = has_dw ? g.k : 1, S = has_dw ? g.s : 1;
  const int TH = v.tile_h, TW = v.tile_w, P = TH * TW;
  const int wp = 4 / v.wc;
  const int NB = ceil_div(ceil_div(P, 16), wp), NBT = NB * wp;
  const bool share = has_dw && has_pw && v.wc > 1;
  const int nbd = share ? ceil_div(NBT, 4) : NB;
  const int ctw = has_pw ? v.max_cob / 16 / v.wc : 0;
  const int ogtiles = 4 / g.elt;  // MFMA tiles per 16-byte output granule
  const int cin = v.family == FAM_DW ? g.cm : g.ci, last = v.family == FAM_DW ? g.cm : g.co;
  const int nch = v.family == FAM_DW ? 1 : ceil_div(cin * g.elt, 64);
  const int64_t ntiles = (int64_t)g.n * ceil_div(g.ho, TH) * ceil_div(g.wo, TW) * ceil_div(last, p.co_block);
  const int ncb = ceil_div(last, p.co_block);
  int64_t G = std::min<int64_t>(std::max(1, p.workgroups), ntiles);
  G -= G % ncb;
  G = std::max<int64_t>(G, ncb);
  const double ipw = (double)ceil_div((int)std::min<int64_t>(ntiles, 1 << 30), (int)G) * nch;
  const double wpc = std::max(1.0, (double)G / hw.num_cus);
  const int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K;
  const int copies = round_up(IH * IW, 32) / 16 + (has_pw ? round_up(p.co_block, 32) / 16 : 0) + (has_dw ? 1 : 0);
  const double dots = has_dw ? (double)nbd * K * K * (16 / g.elt) : 0.0;
  const double mfmas = has_pw ? (double)NB * ctw * (g.elt == 4 ? 4 : 1) : 0.0;
  const double epi = has_pw ? (double)NB * std::max(1, ctw / ogtiles) / nch : (double)nbd;
  const double per = kItem + kPerDot * dots + kPerMfma * mfmas + kPerCopy * copies + kPerEpi * epi;
  const double t_us = kLaunchUs + ipw * per * std::pow(wpc, kShareExp) / kClockMHz;
  const double t_mem_us = (double)p.bytes_ideal / kHbm * 1e6 + kLaunchFloorUs;
  return std::max(t_us, t_mem_us) * 1e-6;
}

// Time model of the PW -> PW register kernel (gen 4), in seconds: each wave runs its
// chunks one after another, each chunk costing its operand loads (1 KiB per 16-byte-per-
// lane load, the CU's cache port shared by the resident waves), its MFMAs and a memory
// latency that the resident waves overlap; splitting a pixel group's chunks over waves
// adds the LDS exchange of the partial sums.
static double pwpw4_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw) {
  constexpr double kLat = 900.0;       // cycles of memory latency per chunk
  constexpr double kPerLoad = 16.0;    // cycles per 1 KiB operand load (cache port)
  constexpr double kPerMfma = 16.0;    // cycles per 16x16 MFMA step
  constexpr double kResident = 8.0;    // waves resident per CU
  constexpr double kLaunch = 7000.0;   // cycles of launch and drain
  constexpr double kReduce = 400.0;    // cycles: partial sums through LDS and the barrier
  constexpr double kClock = 2.4e9;
  const int e = g.elt;
  const int pb = v.max_p / 16;
  const int tpc = 4 / e;
  const int ks = ceil_div(g.ci * e, 64), ct = ceil_div(g.co, 16);
  const int nch = ceil_div(g.cm * e, 64);
  const int splits = std::max(1, (int)p.splits);
  const int cu = ceil_div(nch, splits);                                  // chunks of the busiest wave
  const double loads = tpc * ks + ct + (e == 1 ? 4 : 2);                 // + bias
  const double mfmas = (double)pb * (tpc * ks + ct) * (e == 4 ? 4 : 1);
  const double waves = 4.0 * std::max(1, (int)p.workgroups);
  const double per_cu = std::max(1.0, waves / hw.num_cus);               // waves per CU over the launch
  const double issue = kPerLoad * loads + kPerMfma * mfmas;              // one wave, one chunk
  const double lat_bound = std::ceil(per_cu / kResident) * cu * (kLat + issue);
  const double thr_bound = per_cu * cu * issue;
  double cyc = kLaunch + std::max(lat_bound, thr_bound);
  if (splits > 1) cyc += kReduce + kPerLoad * pb * ct;
  return cyc / kClock;
}

// Multiply-accumulate work of a module, counted as 2 flops each (the recomputed PW halo
// of PW->DW is not included).
static double module_flops(const Geom& g) {
  const double px = (double)g.n * g.h * g.w, po = (double)g.n * g.ho * g.wo;
  const double kk = (double)g.k * g.k;
  switch (g.family) {
    case FAM_DWPW: return 2.0 * po * g.ci * (kk + g.co);
    case FAM_PWDW: return 2.0 * (px * g.ci * g.cm + po * g.cm * kk);
    case FAM_PWDWPW: return 2.0 * (px * g.ci * g.cm + po * g.cm * (kk + g.co));
    case FAM_PWPW: return 2.0 * px * g.cm * (g.ci + g.co);
    case FAM_DW: return 2.0 * po * g.cm * kk;
    default: return 2.0 * px * g.ci * g.co;  // FAM_PW
  }
}

// Linear time models of the kernels without a structural one: microseconds =
// c0 + per_mb * bytes_tiled/1e6 + per_gflop * flops/1e9 + per_kwg * workgroups/1e3,
// fitted (non-negative least squares on relative error) to every candidate module of the
// MobileNetV2 layer chain, int8 and bf16, batch 1 and 32, timed on MI355X; the fitted
// figures are within about 0.5-1.5x of the timings. FP32 takes the bf16 figures.
// zp = 1: the first-generation kernels with int8 zero points (they add the weight-row sums
// and run layers the persistent kernels would otherwise take), fitted the same way to every
// candidate module of the MobileNetV2 int8 chain at batch 32 with a zero point on every
// tensor (0.34-1.41x of the timings).
struct LinModel {
  int family, gen, dtype, zp;
  double c0, per_mb, per_gflop, per_kwg;
};
static const LinModel kLinModels[] = {
    {FAM_PW, 1, DT_I8, 0, 6.56, 3.617, 0.0, 0.0},
    {FAM_PWDW, 1, DT_BF16, 0, 7.97, 0.0, 27.647, 12.939},
    {FAM_PWDW, 1, DT_I8, 0, 10.05, 0.0, 24.499, 15.288},
    {FAM_PWDWPW, 1, DT_BF16, 0, 21.16, 1.864, 0.0, 3.306},
    {FAM_PWDWPW, 1, DT_I8, 0, 33.52, 4.262, 0.0, 25.127},
    {FAM_PWPW, 1, DT_BF16, 0, 6.16, 0.649, 0.0, 0.0},
    {FAM_PWPW, 1, DT_I8, 0, 6.21, 0.822, 0.0, 0.0},
    {FAM_PWPW, 4, DT_BF16, 0, 3.97, 0.0, 27.116, 0.661},
    {FAM_PWPW, 4, DT_I8, 0, 7.01, 0.0, 14.325, 12.663},
    {FAM_DWPW, 1, DT_I8, 1, 0.00, 1.024, 92.594, 2.451},
    {FAM_DW, 1, DT_I8, 1, 3.96, 0.833, 18.913, 8.613},
    {FAM_PW, 1, DT_I8, 1, 4.04, 0.000, 27.904, 8.483},
    {FAM_PWDW, 1, DT_I8, 1, 11.61, 0.000, 26.027, 29.295},
    {FAM_PWDWPW, 1, DT_I8, 1, 0.00, 4.790, 38.501, 44.039},
    {FAM_PWPW, 1, DT_I8, 1, 0.00, 2.057, 0.000, 0.000},
};

static double linear_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p) {
  const int dt = g.dtype == DT_F32 ? DT_BF16 : g.dtype;
  const LinModel* m = nullptr;
  for (const LinModel& l : kLinModels)  // the zero-point figure if there is one
    if (l.family == v.family && l.gen == v.gen && l.dtype == dt && (l.zp == g.zp || (!m && l.zp == 0))) m = &l;
  // kernels never timed for the fit: a conservative generic figure
  static const LinModel kGeneric = {0, 0, 0, 0, 10.0, 2.0, 25.0, 10.0};
  if (!m) m = &kGeneric;
  const double us = m->c0 + m->per_mb * (double)p.bytes_tiled / 1e6 + m->per_gflop * module_flops(g) / 1e9 +
                    m->per_kwg * (double)p.workgroups / 1e3;
  return us * 1e-6;
}

// Time model of the whole-module fp32 kernels (gen 6), in seconds: the launch, then as
// many rounds of workgroups as the LDS lets the CUs hold; a workgroup costs a fixed part
// (its loads' latency and the stage barriers), the busiest wave's MFMA instructions and its
// share of the window elements it stages. Cycle figures fitted (non-negative least
// squares) to the eight C1 / C2 tilings timed on MI355X (within 0.8-1.15x).
static double small_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw) {
  constexpr double kLaunch = 1.6e-6, kFixed = 9254.0, kPerMfma = 112.3, kPerWindowElt = 329.7, kClock = 2.4e9;
  const int TH = v.tile_h, TW = v.tile_w;
  const int IW = (TW - 1) * g.s + g.k, IH = (TH - 1) * g.s + g.k;
  const int nqt = ceil_div(IH * IW, 16), npt = ceil_div(TH * TW, 16);
  const bool pw1 = g.family == FAM_PWDW || g.family == FAM_PWDWPW;
  const bool pw2 = g.family == FAM_DWPW || g.family == FAM_PWDWPW;
  const int cd = pw1 ? g.cm : g.ci;
  const int ci16 = ceil_div(g.ci, 16), cd16 = ceil_div(cd, 16);
  double mfma = 0;
  if (pw1) mfma += (double)ceil_div(ceil_div(g.cm, 16), 4) * nqt * ci16 * 4;
  if (pw2) {
    const int npair = ceil_div(ceil_div(g.co, 16), 2);
    const int nsplit = std::max(1, std::min(4 / npair, cd16));
    mfma += (double)ceil_div(npair * nsplit, 4) * 2 * npt * ceil_div(cd16, nsplit) * 4;
  }
  const double xpt = ceil_div(IH * IW * ci16 * 16, 256);
  const int per_cu = std::max(1, std::min(8, (int)(hw.lds_per_cu / std::max(1, (int)p.lds_bytes))));
  const double rounds = std::ceil((double)std::max(1, (int)p.workgroups) / ((double)per_cu * hw.num_cus));
  return kLaunch + rounds * (kFixed + kPerMfma * mfma + kPerWindowElt * xpt) / kClock;
}

// Time model of the deep DW->PW kernels (gen 7), in seconds: the launch with the first
// loads and the last stores, then each workgroup's items (tile x 32-channel chunk) one
// after another, an item costing a fixed part, the window copies of a depthwise wave and
// the MFMA wave's output tiles, and each work tile its epilogue, scaled by the workgroups
// sharing a CU; or the module's HBM bytes at the rate these kernels reach, if slower
// (cycles and rate fitted to MobileNetV1 layers 1-13 at batch 1 and 32 and the token
// grids at batch 64).
static double deep_time_estimate(const Variant& v, const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw) {
  constexpr double kLaunch = 3.5e-6, kItem = 800.0, kPerCopy = 250.0, kPerTile = 100.0, kPerWork = 1000.0,
                   kClock = 2.4e9, kRate = 3.0e12;
  const int ctw = v.max_cob / 64;
  const int iw = (v.tile_w - 1) * g.s + 3, ih = (v.tile_h - 1) * g.s + 3;
  const int copies = ceil_div(ih * iw, 64);
  const int nch = ceil_div(g.ci, 32);
  const int64_t nwork = (int64_t)g.n * ceil_div(g.ho, v.tile_h) * ceil_div(g.wo, v.tile_w) * ceil_div(g.co, v.max_cob);
  const int grid = std::max(1, (int)p.workgroups);
  const double tiles = (double)ceil_div(nwork, (int64_t)grid);
  const double share = std::max(1.0, (double)grid / hw.num_cus);
  // per 32-channel chunk; items of two chunks pay the per-item part (barrier, waits) once,
  // which measured faster only for long stride-1 chunk streams (7x7x1024: 21.5 against
  // 23.0 us) and slower with stride 2 or few chunks (the larger items' copies)
  const double item = kItem * (v.kc == 2 ? (g.s == 1 && g.ci >= 1024 ? 0.8 : 1.2) : 1.0);
  const double cyc = (tiles * nch * (item + kPerCopy * copies + kPerTile * ctw) + tiles * kPerWork) * share;
  return kLaunch + std::max(cyc / kClock, (double)p.bytes_ideal / kRate);
}

double plan_time_estimate(const Geom& g, const fcm_plan_t& p, const fcm_hw_desc& hw) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  if (p.variant < 0 || p.variant >= nv) return 0.0;
  const Variant& v = vs[p.variant];
  if (v.gen == 3) return persistent_time_estimate(v, g, p, hw);
  if (v.gen == 5) return streaming_time_estimate(v, g, p, hw);
  if (v.gen == 6) return small_time_estimate(v, g, p, hw);
  if (v.gen == 7) return deep_time_estimate(v, g, p, hw);
  // the register kernel's structural model ranks its own plans; for comparisons with other
  // kernels the fitted figure bounds it from below
  if (v.gen == 4) return std::max(pwpw4_time_estimate(v, g, p, hw), linear_time_estimate(v, g, p));
  return linear_time_estimate(v, g, p);
}

struct Cand {
  fcm_plan_t p;
  int64_t bytes;
  int wgs;
  int lds;
  int area;
  int cap;  // variant capacity (prefer the smallest that fits)
};

static std::vector<int> tile_ws(const Variant& v) {
  if (v.dw_r) return {4, 8, 16, 32};
  return {1, 2, 4, 7, 8, 14, 16, 28, 32, 56, 64};
}

static const int kTileH[] = {1, 2, 4, 7, 8, 14, 16, 28, 32};

// Tile shapes (TH, TW) searched for the persistent kernels: the shapes over which their
// time model was fitted (widths whose windows fill the copy rows reasonably).
static const int kTiles3[][2] = {{16, 14}, {8, 14}, {7, 14}, {4, 14}, {14, 14}, {28, 8}, {14, 7}, {8, 7}, {7, 7},
                                 {16, 7},  {9, 14}, {12, 14}, {7, 28}, {4, 28}, {8, 28}, {9, 28}, {16, 16}, {8, 16},
                                 {4, 16},  {2, 14}, {1, 14}, {3, 14}, {5, 14}, {6, 14}, {2, 7},  {4, 7},  {1, 7},
                                 {2, 4},   {4, 4},  {2, 2},  {3, 7},  {6, 7},  {12, 7}};

// Every plan the compiled kernels can run for the shape (within the workspace limit).
static void collect(const Geom& g, const fcm_desc* d, const fcm_hw_desc& hw, int kset, int64_t ws_max,
                    std::vector<Cand>& cands) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  const int kb = k_block(g.dtype);
  const int last = (g.family == FAM_PWDW || g.family == FAM_DW) ? g.cm : g.co;
  for (int vi = 0; vi < nv; ++vi) {
    const Variant& v = vs[vi];
    if (!variant_matches(v, g)) continue;
    if (!in_set(v, kset)) continue;
    if (v.gen == 5 || v.gen == 7) {
      // streaming and deep kernels: one compiled tile and output-channel block each
      Cand c;
      memset(&c.p, 0, sizeof(c.p));
      c.p.op = g.op;
      c.p.tile_h = v.tile_h;
      c.p.tile_w = v.tile_w;
      c.p.c_block = 64 / g.elt;
      c.p.co_block = v.max_cob;
      c.p.variant = vi;
      if (evaluate_plan(g, d, hw, &c.p) != FCM_OK) continue;
      c.bytes = c.p.bytes_tiled;
      c.wgs = c.p.workgroups;
      c.lds = c.p.lds_bytes;
      c.area = v.tile_h * v.tile_w;
      c.cap = v.max_cob * 1024 + v.max_p;
      cands.push_back(c);
      continue;
    }
    if (v.gen == 6) {
      // whole-module kernels: one compiled tile, every channel
      Cand c;
      memset(&c.p, 0, sizeof(c.p));
      c.p.op = g.op;
      c.p.tile_h = v.tile_h;
      c.p.tile_w = v.tile_w;
      c.p.c_block = 16;
      c.p.co_block = round_up(last, 16);
      c.p.variant = vi;
      if (evaluate_plan(g, d, hw, &c.p) != FCM_OK) continue;
      c.bytes = c.p.bytes_tiled;
      c.wgs = c.p.workgroups;
      c.lds = c.p.lds_bytes;
      c.area = v.tile_h * v.tile_w;
      c.cap = v.max_p;
      cands.push_back(c);
      continue;
    }
    if (v.gen == 4) {
      const int nch = ceil_div(g.cm * g.elt, 64);
      for (int sp = 1; sp <= std::min(4, nch); sp *= 2) {
        Cand c;
        memset(&c.p, 0, sizeof(c.p));
        c.p.op = g.op;
        c.p.tile_h = 1;
        c.p.tile_w = v.max_p;
        c.p.c_block = 64 / g.elt;
        c.p.co_block = round_up(g.co, 16);
        c.p.variant = vi;
        c.p.splits = sp;
        if (evaluate_plan(g, d, hw, &c.p) != FCM_OK) continue;
        c.bytes = c.p.bytes_tiled;
        c.wgs = c.p.workgroups;
        c.lds = 0;
        c.area = v.max_p;
        c.cap = v.max_cob * 1024 + v.ks;
        cands.push_back(c);
      }
      continue;
    }
    std::vector<int> cbs;
    if (v.family == FAM_DW) {
      cbs = {0};  // CB follows COB
    } else if (v.family == FAM_PWDWPW || v.family == FAM_PWPW) {
      const int step = std::max(16, kb);
      for (int c = step; c <= std::min(v.max_mb, round_up(g.cm, step)); c += step) cbs.push_back(c);
    } else {
      for (int c = kb; c <= std::min(round_up(g.ci, kb), 8 * kb); c *= 2) cbs.push_back(c);
      if (round_up(g.ci, kb) < 8 * kb && std::find(cbs.begin(), cbs.end(), round_up(g.ci, kb)) == cbs.end())
        cbs.push_back(round_up(g.ci, kb));
    }
    std::vector<int> tws = v.tile_w ? std::vector<int>{v.tile_w} : tile_ws(v);
    std::vector<int> ths = v.tile_h ? std::vector<int>{v.tile_h}
                                    : std::vector<int>(std::begin(kTileH), std::end(kTileH));
    std::vector<std::pair<int, int>> tiles;
    if (v.gen == 3) {
      for (const auto& t : kTiles3) tiles.push_back({t[0], t[1]});
    } else {
      for (int TW : tws)
        for (int TH : ths) tiles.push_back({TH, TW});
    }
    for (const auto& tile : tiles) {
      const int TH = tile.first, TW = tile.second;
      if (!v.tile_w && TW > round_up(g.wo, v.dw_r ? v.dw_r : 1) && TW > 4) continue;
      {
        if (!v.tile_h && TH > g.ho && TH > 1) continue;
        // persistent kernels have one compiled output-channel block (the last is masked)
        const int cob_lo = v.gen == 3 ? v.max_cob : 16;
        const int cob_hi = v.gen == 3 ? v.max_cob : std::min(v.max_cob, round_up(last, 16));
        for (int COB = cob_lo; COB <= cob_hi; COB += 16) {
          for (int cb0 : cbs) {
            const int CB = v.family == FAM_DW ? COB : cb0;
            // persistent kernels: one or two items in flight (deeper rings measured no faster)
            const int depths[2] = {2, 3};
            // persistent kernels with a PW stage: also split each work tile's channel chunks
            const int splitss[4] = {1, 2, 4, 8};
            const int nsplits = (v.gen == 3 && v.family != FAM_DW) ? 4 : 1;
            for (int si = 0; si < nsplits; ++si)
            for (int di = 0; di < (v.gen == 3 ? 2 : 1); ++di) {
              int depth = v.gen == 3 ? depths[di] : 0;
              const int lds = tiling_lds(v, g, TH, TW, CB, COB, hw.lds_per_wg, &depth);
              if (lds <= 0 || lds > hw.lds_per_wg) continue;
              Cand c;
              memset(&c.p, 0, sizeof(c.p));
              c.p.op = g.op;
              c.p.tile_h = TH;
              c.p.tile_w = TW;
              c.p.c_block = CB;
              c.p.co_block = COB;
              c.p.variant = vi;
              c.p.depth = depth;
              c.p.splits = splitss[si];
              if (evaluate_plan(g, d, hw, &c.p) != FCM_OK) continue;
              if (plan_workspace_bytes(g, c.p) > ws_max) continue;
              c.bytes = c.p.bytes_tiled;
              c.wgs = c.p.workgroups;
              c.lds = lds;
              c.area = TH * TW;
              c.cap = v.max_cob * 1024 + (v.max_p ? v.max_p : v.max_q);
              cands.push_back(c);
            }
          }
        }
      }
    }
  }
}

static fcm_status search(const Geom& g, const fcm_desc* d, const fcm_hw_desc& hw, fcm_plan_t* best_out,
                         int kset, int64_t ws_max) {
  int nv = 0;
  const Variant* vs = all_variants(&nv);
  std::vector<Cand> cands;
  collect(g, d, hw, kset, ws_max, cands);
  if (cands.empty()) return fail(FCM_EUNSUPPORTED, "plan: no compiled kernel implements this shape");
  // The PW -> PW register kernel (gen 4) is preferred wherever one implements the shape:
  // the plan with the least estimated time, ties to the smaller variant.
  {
    const Cand* best4 = nullptr;
    double best_t = 0;
    for (const Cand& c : cands) {
      if (vs[c.p.variant].gen != 4) continue;
      const double t = pwpw4_time_estimate(vs[c.p.variant], g, c.p, hw);
      if (!best4 || t < best_t || (t == best_t && c.cap < best4->cap)) {
        best4 = &c;
        best_t = t;
      }
    }
    if (best4) {
      *best_out = best4->p;
      return FCM_OK;
    }
  }
  // The persistent (gen 3), streaming (gen 5) and whole-module (gen 6) kernels are
  // preferred wherever one implements the shape; among them the plan with the least
  // estimated time under its kernel family's fitted model wins.
  {
    const Cand* best35 = nullptr;
    double best_t = 0;
    for (const Cand& c : cands) {
      const int gen = vs[c.p.variant].gen;
      if (gen != 3 && gen != 5 && gen != 6 && gen != 7) continue;
      const double t = plan_time_estimate(g, c.p, hw);
      if (!best35 || t < best_t || (t == best_t && c.p.variant < best35->p.variant)) {
        best35 = &c;
        best_t = t;
      }
    }
    if (best35) {
      *best_out = best35->p;
      return FCM_OK;
    }
  }
  bool any_full = false;
  for (const Cand& c : cands) any_full |= c.wgs >= hw.num_cus;
  const int target = 2 * hw.num_cus;
  auto better = [&](const Cand& a, const Cand& b) {
    // 1. the paper's occupancy constraint (#tiles >= #SMs) where reachable
    const bool fa = a.wgs >= hw.num_cus, fb = b.wgs >= hw.num_cus;
    if (any_full && fa != fb) return fa;
    if (!any_full && a.wgs != b.wgs) return a.wgs > b.wgs;
    // 2. fewest global bytes
    if (a.bytes != b.bytes) return a.bytes < b.bytes;
    // 3. two workgroups fit a CU's LDS
    const bool ha = 2 * a.lds <= hw.lds_per_cu, hb = 2 * b.lds <= hw.lds_per_cu;
    if (ha != hb) return ha;
    // 4. more workgroups, up to two per CU
    const int wa = std::min(a.wgs, target), wb = std::min(b.wgs, target);
    if (wa != wb) return wa > wb;
    // 5. larger tiles, larger channel chunks, smallest kernel capacity, lowest id
    if (a.area != b.area) return a.area > b.area;
    if (a.p.c_block != b.p.c_block) return a.p.c_block > b.p.c_block;
    if (a.cap != b.cap) return a.cap < b.cap;
    return a.p.variant < b.p.variant;
  };
  const Cand* best = &cands[0];
  for (const Cand& c : cands)
    if (better(c, *best)) best = &c;
  *best_out = best->p;
  return FCM_OK;
}

// Stage decomposition for the layer-by-layer estimate of a module.
static void lbl_stages(int op, const fcm_desc* d, std::vector<std::pair<int, fcm_desc>>* out) {
  fcm_desc s = *d;
  auto one = [&](int sop, int h, int w, int ci, int co, int stage) {
    fcm_desc t = *d;
    t.h = h;
    t.w = w;
    t.c_in = ci;
    t.c_mid = ci;
    t.c_out = co;
    t.act[0] = t.act[1] = t.act[2] = d->act[stage];
    t.rq[0] = t.rq[1] = t.rq[2] = d->rq[stage];
    t.rq_channel[0] = d->rq_channel[stage];
    t.rq_channel[1] = t.rq_channel[2] = nullptr;
    t.zp_in = stage == 0 ? d->zp_in : d->rq[stage - 1].zero_point;
    if (sop == FCM_OP_PW) {
      t.k = 1;
      t.stride = 1;
      t.pad = 0;
    }
    out->push_back({sop, t});
  };
  const int ho = out_dim(s.h, s.k, s.stride, s.pad), wo = out_dim(s.w, s.k, s.stride, s.pad);
  switch (op) {
    case FCM_OP_DW_PW:
      one(FCM_OP_DW, s.h, s.w, s.c_in, s.c_in, 0);
      one(FCM_OP_PW, ho, wo, s.c_in, s.c_out, 1);
      break;
    case FCM_OP_PW_DW:
      one(FCM_OP_PW, s.h, s.w, s.c_in, s.c_mid, 0);
      one(FCM_OP_DW, s.h, s.w, s.c_mid, s.c_mid, 1);
      break;
    case FCM_OP_PW_DW_PW:
      one(FCM_OP_PW, s.h, s.w, s.c_in, s.c_mid, 0);
      one(FCM_OP_DW, s.h, s.w, s.c_mid, s.c_mid, 1);
      one(FCM_OP_PW, ho, wo, s.c_mid, s.c_out, 2);
      break;
    case FCM_OP_PW_PW:
      one(FCM_OP_PW, s.h, s.w, s.c_in, s.c_mid, 0);
      one(FCM_OP_PW, s.h, s.w, s.c_mid, s.c_out, 1);
      break;
    default:
      break;
  }
}

static std::mutex g_cache_mu;
static std::map<std::vector<int64_t>, fcm_plan_t> g_cache;

static std::vector<int64_t> cache_key(int op, const fcm_desc* d, const fcm_hw_desc& hw) {
  std::vector<int64_t> k = {op, d->n, d->h, d->w, d->c_in, d->c_mid, d->c_out, d->k, d->stride, d->pad,
                            d->dtype, hw.num_cus, hw.lds_per_wg, hw.lds_per_cu};
  return k;
}

fcm_status find_plan(int op, const fcm_desc* d, const fcm_hw_desc* hw_in, fcm_plan_t* out, int kset,
                     int64_t ws_max) {
  const fcm_hw_desc hw = hw_in ? *hw_in : default_hw();
  if (hw.num_cus <= 0 || hw.lds_per_wg <= 0 || hw.lds_per_cu <= 0)
    return fail(FCM_EINVAL, "plan: hardware description has non-positive sizes");
  std::vector<int64_t> key = cache_key(op, d, hw);
  key.push_back(kset);
  key.push_back(d->layout);
  key.push_back(std::min<int64_t>(ws_max, FCM_SPLIT_WORKSPACE_BYTES));
  {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    auto it = g_cache.find(key);
    if (it != g_cache.end()) {
      *out = it->second;
      return FCM_OK;
    }
  }
  const Geom g = geometry(op, d);
  fcm_plan_t p;
  fcm_status st = search(g, d, hw, &p, kset, ws_max);
  if (st != FCM_OK) return st;
  // layer-by-layer chain: each stage planned on its own (first pass of Sec. IV)
  std::vector<std::pair<int, fcm_desc>> stages;
  lbl_stages(op, d, &stages);
  if (stages.empty()) {
    p.bytes_lbl_paper = p.bytes_paper;
    p.bytes_lbl_ideal = p.bytes_ideal;
    p.fuse = 0;
  } else {
    int64_t lp = 0, li = 0;
    for (auto& sd : stages) {
      fcm_plan_t sp;
      st = find_plan(sd.first, &sd.second, &hw, &sp, kset);
      if (st != FCM_OK) return st;
      lp += sp.bytes_paper;
      li += sp.bytes_ideal;
    }
    p.bytes_lbl_paper = lp;
    p.bytes_lbl_ideal = li;
    p.fuse = p.bytes_paper < lp ? 1 : 0;
  }
  {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    g_cache[key] = p;
  }
  *out = p;
  return FCM_OK;
}

static bool same_plan(const fcm_plan_t& a, const fcm_plan_t& b) {
  return a.variant == b.variant && a.tile_h == b.tile_h && a.tile_w == b.tile_w && a.c_block == b.c_block &&
         a.co_block == b.co_block && a.depth == b.depth && a.splits == b.splits && a.workgroups == b.workgroups;
}

fcm_status find_candidates(int op, const fcm_desc* d, const fcm_hw_desc* hw_in, int kset, int64_t ws_max,
                           fcm_plan_t* out, int max_count, int* count) {
  *count = 0;
  const fcm_hw_desc hw = hw_in ? *hw_in : default_hw();
  fcm_plan_t best;
  fcm_status st = find_plan(op, d, &hw, &best, kset, ws_max);
  if (st != FCM_OK) return st;
  const Geom g = geometry(op, d);
  std::vector<Cand> cands;
  collect(g, d, hw, kset, ws_max, cands);
  // each variant's fastest plan by the time models first (so that a mispredicted kernel
  // family still gets timed), then the remaining plans, fastest first
  std::vector<std::pair<double, int>> order;
  for (int i = 0; i < (int)cands.size(); ++i) order.push_back({plan_time_estimate(g, cands[i].p, hw), i});
  std::stable_sort(order.begin(), order.end());
  std::vector<int> firsts, rest;
  std::vector<char> seen_variant(1024, 0);
  for (const auto& o : order) {
    if (same_plan(cands[o.second].p, best)) continue;
    const int v = cands[o.second].p.variant;
    if (v >= 0 && v < 1024 && !seen_variant[v]) {
      seen_variant[v] = 1;
      firsts.push_back(o.second);
    } else {
      rest.push_back(o.second);
    }
  }
  firsts.insert(firsts.end(), rest.begin(), rest.end());
  int n = 0;
  if (max_count > 0) out[n++] = best;  // the planner's own choice leads
  for (int i : firsts) {
    if (n >= max_count) break;
    fcm_plan_t p = cands[i].p;
    p.bytes_lbl_paper = best.bytes_lbl_paper;
    p.bytes_lbl_ideal = best.bytes_lbl_ideal;
    p.fuse = (op == FCM_OP_DW || op == FCM_OP_PW) ? 0 : (p.bytes_paper < p.bytes_lbl_paper ? 1 : 0);
    out[n++] = p;
  }
  *count = n;
  return FCM_OK;
}

}  // namespace fcm
