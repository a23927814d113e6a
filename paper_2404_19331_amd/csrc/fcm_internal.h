// fcm_internal.h -- definitions shared by the host library (planner, C ABI) and the
// kernels: kernel argument blocks, the LDS layout of each kernel family, and the table
// of compiled kernel variants.
#pragma once

#include <stdint.h>
#include <type_traits>

#ifdef __HIPCC__
#define FCM_HD __host__ __device__
#else
#define FCM_HD
#endif

namespace fcm {

constexpr int kNumXcd = 8;
constexpr int kMaxLdsPerWg = 160 * 1024;

enum { LAYOUT_NCHW = 0, LAYOUT_NHWC = 1 };
enum { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2 };
enum { DT_F32 = 0, DT_BF16 = 1, DT_I8 = 2 };

// Kernel families. A "variant" is one compiled instance of a family.
enum Family {
  FAM_DWPW = 0,    // DW -> PW (fused)
  FAM_PW = 1,      // PW alone (family DWPW with the DW stage off)
  FAM_PWDW = 2,    // PW -> DW (fused, halo recomputed)
  FAM_DW = 3,      // DW alone (family PWDW with the PW stage off)
  FAM_PWDWPW = 4,  // PW -> DW -> PW (fused)
  FAM_PWPW = 5,    // PW -> PW (fused; family PWDWPW with the DW stage off)
};

// zp: the code of real 0 in the stage's output (asymmetric int8), added after rounding.
struct Requant {
  int32_t mult, shift, qmin, qmax, zp;
};

// int8 per-channel requantisation of one stage: p = device array [2][n] (the stage's n
// output channels' multipliers, then their shifts); p == nullptr: the per-tensor Requant.
struct ReqCh {
  const int32_t* p = nullptr;
  int n = 0;
};

// Zero points (int8) on the PW->PW register kernel: instances of at most this many
// output-channel tiles of 16.
constexpr int kZpMaxTiles = 12;

FCM_HD constexpr int elt_size(int dt) { return dt == DT_F32 ? 4 : (dt == DT_BF16 ? 2 : 1); }
// contraction elements per MFMA operand step (64 bytes of k per row)
FCM_HD inline int k_block(int dt) { return 64 / elt_size(dt); }
FCM_HD constexpr int round_up(int a, int b) { return (a + b - 1) / b * b; }
FCM_HD constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------------
// LDS layout: byte offsets of each buffer and row strides. Rows are padded by 16 bytes
// so that the 16 lanes reading one MFMA operand column hit distinct banks.
// ---------------------------------------------------------------------------------
struct LdsLayout {
  int off_in, ps_in;    // staged input window (pixel stride)
  int off_w, rs_w;      // first pointwise weight block
  int off_wd;           // depthwise weights [K*K][cb] + bias [cb] (4-byte values)
  int off_e, rs_e;      // intermediate (PW output over the halo window) [Q][mb]
  int off_d, rs_d;      // depthwise output [P][cb]
  int off_w2, rs_w2;    // second pointwise weight block
  int off_out, rs_out;  // output tile [P][cob]
  int bytes;
};

// DW->PW (has_dw) and PW alone. Tile TH x TW output pixels, contraction chunk CB,
// output-channel block COB.
FCM_HD inline LdsLayout lds_layout_dwpw(int dt, int K, int S, bool has_dw, int TH, int TW, int CB, int COB) {
  LdsLayout L = {};
  const int e = elt_size(dt);
  const int P = TH * TW, P16 = round_up(P, 16);
  const int IH = has_dw ? (TH - 1) * S + K : TH, IW = has_dw ? (TW - 1) * S + K : TW;
  int rows_in = IH * IW;
  if (!has_dw && rows_in < P16) rows_in = P16;
  L.ps_in = CB * e + 16;
  L.off_in = 0;
  int off = rows_in * L.ps_in;
  if (has_dw) {
    L.rs_d = CB * e + 16;
    L.off_d = off;
    off += P16 * L.rs_d;
  }
  L.rs_w = CB * e + 16;
  L.off_w = off;
  off += round_up(COB, 16) * L.rs_w;
  if (has_dw) {
    L.off_wd = off;
    off += (K * K + 1) * CB * 4;
  }
  L.rs_out = COB * e + 16;
  L.off_out = 0;
  const int out_bytes = P16 * L.rs_out;
  L.bytes = round_up(off > out_bytes ? off : out_bytes, 16);
  return L;
}

// PW->DW (has_pw) and DW alone. Tile TH x TW outputs; Q = haloed window positions;
// CB = input-channel chunk of the PW contraction; MB = intermediate-channel block.
FCM_HD inline LdsLayout lds_layout_pwdw(int dt, int K, int S, bool has_pw, int TH, int TW, int CB, int MB) {
  LdsLayout L = {};
  const int e = elt_size(dt);
  const int P16 = round_up(TH * TW, 16);
  const int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K;
  const int Q16 = round_up(IH * IW, 16);
  int off = 0;
  L.rs_e = MB * e + 16;
  L.off_e = 0;
  off = Q16 * L.rs_e;
  if (has_pw) {
    L.ps_in = CB * e + 16;
    L.off_in = off;
    off += Q16 * L.ps_in;
    L.rs_w = CB * e + 16;
    L.off_w = off;
    off += round_up(MB, 16) * L.rs_w;
  } else {
    L.ps_in = L.rs_e;
    L.off_in = L.off_e;
  }
  L.off_wd = off;
  off += (K * K + 1) * MB * 4;
  L.rs_out = MB * e + 16;
  L.off_out = off;
  off += P16 * L.rs_out;
  L.bytes = round_up(off, 16);
  return L;
}

// PW->DW->PW. Whole input channel range CIN staged once (padded to the MFMA step),
// intermediate chunk MB, output-channel block COB.
FCM_HD inline LdsLayout lds_layout_pwdwpw(int dt, int K, int S, int TH, int TW, int CIN, int MB, int COB) {
  LdsLayout L = {};
  const int e = elt_size(dt);
  const int P16 = round_up(TH * TW, 16);
  const int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K;
  const int Q16 = round_up(IH * IW, 16);
  const int CIP = round_up(CIN, k_block(dt));
  int off = 0;
  L.ps_in = CIP * e + 16;
  L.off_in = off;
  off += Q16 * L.ps_in;
  L.rs_w = CIP * e + 16;
  L.off_w = off;
  off += round_up(MB, 16) * L.rs_w;
  L.rs_e = MB * e + 16;
  L.off_e = off;
  off += Q16 * L.rs_e;
  L.off_wd = off;
  off += (K * K + 1) * MB * 4;
  L.rs_d = MB * e + 16;
  L.off_d = off;
  off += P16 * L.rs_d;
  L.rs_w2 = MB * e + 16;
  L.off_w2 = off;
  off += round_up(COB, 16) * L.rs_w2;
  L.rs_out = COB * e + 16;
  L.off_out = 0;
  const int out_bytes = P16 * L.rs_out;
  L.bytes = round_up(off > out_bytes ? off : out_bytes, 16);
  return L;
}

// LDS-DMA kernels: bytes of channels per pixel row per staged chunk (one MFMA k-step).
constexpr int kRowB = 64;

// Persistent NHWC kernels (k_fused3): module selector and LDS bytes of one buffer.
enum { M3_DWPW = 0, M3_PW = 1, M3_DW = 2 };

// Byte sizes and offsets of one LDS buffer of the persistent kernels (host and device):
// the input window of IH rows at a pitch of IWP pixels of 64 bytes; the pointwise weight
// block (16*CT rows of 64 bytes); the depthwise weights of one chunk as 32-bit
// dot-operand words [K*K][CB]; the raw depthwise weights as copied ([CB][K*K] elements,
// whole KiB); and two KiB of biases (depthwise, then pointwise). With per-channel int8
// requantisation (pc) three more KiB follow: the depthwise multipliers and shifts (half
// a KiB each), then the pointwise multipliers and shifts (a KiB each). `depth` buffers
// form the ring (the copy wave runs depth - 1 items ahead).
constexpr int kCopyWaves3 = 2;  // copy waves (each issues about half of an item's copies)
constexpr int kThreads3 = 64 * (kCopyWaves3 + 4);  // + four compute waves
constexpr int kMaxDepth3 = 8;   // ring buffers at most
struct Lds3 {
  int in_bytes, w_bytes, wd_off, raw_off, plane_bytes, bias_off, buf_bytes, total;
};
// One buffer holds `ks` planes (one per 64-byte channel chunk of the item: window, PW
// weights, DW dot-operand words, raw DW weights) and then the biases of the item.
FCM_HD inline Lds3 lds3p(int dt, int K, int mode, int IH, int IWP, int CT, int depth = 2, int ks = 1, int pc = 0) {
  Lds3 r;
  const int cb = kRowB / elt_size(dt);
  r.in_bytes = IH * IWP * kRowB;
  r.w_bytes = mode == M3_DW ? 0 : CT * 1024;
  int off = r.in_bytes + r.w_bytes;
  r.wd_off = off;
  if (mode != M3_PW) off += (K * K * cb * 4 + 15) / 16 * 16;
  r.raw_off = off;
  if (mode != M3_PW) off += (64 * K * K + 1023) / 1024 * 1024;
  r.plane_bytes = off;
  r.bias_off = ks * off;
  r.buf_bytes = r.bias_off + (pc ? 2048 + 3072 : 2048);
  r.total = depth * r.buf_bytes;
  return r;
}

// Split plans: items per split of a work tile with `ipt` items, and whether every split
// gets at least one item.
FCM_HD inline int items_per_split3(int ipt, int splits) { return (ipt + splits - 1) / splits; }
FCM_HD inline bool splits_valid3(int ipt, int splits) {
  return splits >= 1 && (splits - 1) * items_per_split3(ipt, splits) < ipt;
}

// Copy instructions of one item (ks channel chunks) of a persistent kernel (host and
// device), in issue order: raw DW weights of each chunk and the DW bias (and with pc
// the DW multipliers and shifts), window rows, PW weight rows of each chunk, PW bias
// (and with pc the PW multipliers, then shifts).
FCM_HD inline int ndw_copies3(int mode, int K, int ks, int pc) {
  return mode != M3_PW ? ks * ((64 * K * K + 1023) / 1024) + 1 + (pc ? 1 : 0) : 0;
}
FCM_HD inline int copies_per_item3(int mode, int K, int IH, int IWP, int CT, int ks = 1, int pc = 0) {
  int n = ks * IH * (IWP / 16);
  if (mode != M3_DW) n += ks * CT + 1 + (pc ? 2 : 0);  // PW weight rows, PW bias (, scales)
  return n + ndw_copies3(mode, K, ks, pc);
}
// Split of an item's copies between the two copy waves: wave 0 issues the DW weights
// and bias (it converts them) and window rows [0, r0) of every chunk, wave 1 rows
// [r0, IH), the PW weight rows and the PW bias; r0 balances the two counts.
FCM_HD inline int rows_wave0_3(int mode, int K, int IH, int IWP, int CT, int ks = 1, int pc = 0) {
  const int ipr = (IWP / 16) * ks;
  const int ndw = ndw_copies3(mode, K, ks, pc);
  const int t = copies_per_item3(mode, K, IH, IWP, CT, ks, pc);
  int r0 = (t - 2 * ndw + ipr) / (2 * ipr);
  r0 = r0 < 0 ? 0 : (r0 > IH ? IH : r0);
  return r0;
}
FCM_HD inline int copies_wave0_3(int mode, int K, int IH, int IWP, int CT, int ks = 1, int pc = 0) {
  return ndw_copies3(mode, K, ks, pc) + rows_wave0_3(mode, K, IH, IWP, CT, ks, pc) * (IWP / 16) * ks;
}
// The larger per-wave share: a partial wait on the vector-memory counter covers at most
// 63 outstanding copies of one wave.
FCM_HD inline int copies_per_wave3(int mode, int K, int IH, int IWP, int CT, int ks = 1, int pc = 0) {
  const int t = copies_per_item3(mode, K, IH, IWP, CT, ks, pc);
  const int w0 = copies_wave0_3(mode, K, IH, IWP, CT, ks, pc);
  return w0 > t - w0 ? w0 : t - w0;
}

// Streaming NHWC kernels (k_fused5, host and device): bytes of one LDS ring slot and of
// the whole allocation. Window and pointwise weights are stored as two planes, plane h
// holding the 16-byte slots 2h and 2h+1 of each 64-byte channel row at 32 bytes per
// pixel (or row): the 32 lanes of a half-wave that read one MFMA operand (16 pixels x
// two slots) then cover 512 distinct bytes, which ds_read_b128 serves without bank
// conflicts. One LDS-DMA instruction fills 32 pixels (rows) of one plane.
//   slot:  window [2][nqp][32 B] | PW weights [2][cobp][32 B] | DW words [K*K][CB] + bias [CB]
//   after the ring: PW bias [COB] (fp32 / int32, whole KiB) | DW output exchange [2][pp][32 B]
struct Lds5 {
  int nqp;         // window pixels rounded up to 32
  int win_bytes;   // 64 * nqp
  int cobp;        // pointwise rows rounded up to 32 (0 without a PW stage)
  int dw_off;      // depthwise words within a slot
  int slot_bytes;
  int pwb_off;     // PW bias block
  int dwo_off;     // depthwise output exchange (pp > 0 only)
  int total;
};
FCM_HD constexpr Lds5 lds5(int dt, int mode, int K, int IH, int IW, int COB, int ring, int pp) {
  Lds5 L{};
  const int cb = kRowB / elt_size(dt);
  const bool pw = mode != M3_DW, dw = mode != M3_PW;
  L.nqp = round_up(IH * IW, 32);
  L.win_bytes = 64 * L.nqp;
  L.cobp = pw ? round_up(COB, 32) : 0;
  L.dw_off = L.win_bytes + 64 * L.cobp;
  L.slot_bytes = L.dw_off + (dw ? round_up((K * K + 1) * cb * 4, 16) : 0);
  L.pwb_off = ring * L.slot_bytes;
  L.dwo_off = L.pwb_off + (pw ? round_up(COB * 4, 1024) : 0);
  L.total = L.dwo_off + 64 * pp;
  return L;
}

// Deep DW->PW kernels (k_deep7, bf16, 3x3): LDS bytes. Three ring slots of the haloed
// window and two depthwise output exchange buffers, both as 4 KC planes of 8 channels
// (KC 32-channel chunks per item; 16 bytes per position: a wave reading one plane at
// consecutive positions touches every bank once), the PW bias block of 64 * CTW channels (fp32), and all C input channels'
// depthwise weights ([C][3][3] bf16) and biases (fp32), each in whole KiB. Window
// positions are rounded up to 64 (one LDS-DMA copy fills 64 positions of one plane).
struct Lds7 {
  int nqp, win_plane, win_bytes, exch_off, exch_plane, exch_bytes, pwb_off, dww_off, dwb_off, total;
};
FCM_HD constexpr Lds7 lds7(int S, int TH, int TW, int CTW, int C, int KC = 1) {
  Lds7 L{};
  const int IH = (TH - 1) * S + 3, IW = (TW - 1) * S + 3;
  L.nqp = round_up(IH * IW, 64);
  L.win_plane = 16 * L.nqp;
  L.win_bytes = 4 * KC * L.win_plane;
  L.exch_off = 3 * L.win_bytes;
  L.exch_plane = (TH * TW + 15) / 16 * 16 * 16;
  L.exch_bytes = 4 * KC * L.exch_plane;
  L.pwb_off = L.exch_off + 2 * L.exch_bytes;
  L.dww_off = L.pwb_off + round_up(64 * CTW * 4, 1024);
  L.dwb_off = L.dww_off + round_up(C * 18, 1024);
  L.total = L.dwb_off + round_up(C * 4, 1024);
  return L;
}

// Whole-module fp32 kernels for small batches (k_small6): module selector and the LDS
// layout, in floats, for the run-time channel counts (host and device compute it alike).
enum { M6_DWPW = 0, M6_PWDW = 1, M6_PWDWPW = 2 };
struct Lds6 {
  int cip, px;        // input channels rounded up to 16; row pitch of the window
  int nqp;            // window positions rounded up to 16
  int cmp;            // first PW's output rows rounded up to 16 (0 without one)
  int cdp, pd;        // depthwise channels rounded up to 16; row pitch of D
  int np;             // tile pixels rounded up to 16
  int cop;            // last PW's output rows rounded up to 16 (0 without one)
  int xs, w1, b1, wd, bd, es, ds, w2, b2, red;  // offsets
  int floats;         // total
};
FCM_HD inline Lds6 lds6(int mode, int K, int S, int TH, int TW, int ci, int cm, int co) {
  Lds6 L{};
  const bool pw1 = mode != M6_DWPW, pw2 = mode != M6_PWDW;
  const int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K, nq = IH * IW, p = TH * TW;
  const int cd = pw1 ? cm : ci;
  L.cip = round_up(ci, 16);
  L.px = L.cip + 4;
  L.nqp = round_up(nq, 16);
  L.cmp = pw1 ? round_up(cm, 16) : 0;
  L.cdp = round_up(cd, 16);
  L.pd = L.cdp + 4;
  L.np = round_up(p, 16);
  L.cop = pw2 ? round_up(co, 16) : 0;
  int off = 0;
  auto take = [&](int n) {
    const int o = off;
    off += round_up(n, 4);
    return o;
  };
  L.xs = take(L.nqp * L.px);
  L.w1 = take(pw1 ? L.cmp * ci + 16 : 0);  // [cm][ci] as stored, rows up to cmp, 16 zeros after cm rows
  L.b1 = take(L.cmp);
  L.wd = take(cd * K * K);
  L.bd = take(cd);
  L.es = take(pw1 ? L.cmp * L.nqp : 0);  // [cmp][nqp]
  L.ds = take(pw2 ? L.np * L.pd : 0);
  L.w2 = take(pw2 ? L.cop * cd + 16 : 0);  // [co][cd] as stored, likewise
  L.b2 = take(L.cop);
  {
    // partial sums of the last PW: [split][pair][2][pixel tile][64 lanes x 4]
    const int npt = (p + 15) / 16, npair = (L.cop / 16 + 1) / 2, cdp16 = L.cdp / 16;
    int nsplit = npair > 0 ? 4 / npair : 1;
    nsplit = nsplit < 1 ? 1 : (nsplit > cdp16 ? cdp16 : nsplit);
    L.red = take(pw2 && nsplit > 1 ? nsplit * npair * 2 * npt * 256 : 0);
  }
  L.floats = off;
  return L;
}

// ---------------------------------------------------------------------------------
// Kernel argument block (one struct for all families; unused fields ignored).
// ---------------------------------------------------------------------------------
struct KArgs {
  const void* x;
  const void* w1;  // first conv weights  (dwpw/dw: depthwise; pw, pwdw, pwdwpw: pointwise)
  const void* b1;
  const void* w2;  // second conv weights (dwpw: pointwise; pwdw, pwdwpw: depthwise)
  const void* b2;
  const void* w3;  // third conv weights  (pwdwpw: pointwise)
  const void* b3;
  void* y;
  int N, H, W;        // input
  int Ci, Cm, Co;     // channels: input, intermediate, output
  int Ho, Wo, pad;
  int layout;
  int TH, TW, CB, COB;  // tile, contraction chunk, channel block (see fcm_plan_t)
  int tiles_y, tiles_x, n_cb;  // grid decomposition: N x tiles_y x tiles_x x n_cb
  int act[3];
  Requant rq[3];
  int vec_x, vec_w1, vec_w2, vec_w3, vec_y;
  LdsLayout L;
  int nwork;     // persistent kernels: work units (work tiles x splits)
  int depth;     // persistent kernels: LDS ring buffers (>= 2)
  int splits;    // persistent kernels: workgroups sharing one work tile's channel chunks
  void* ws;      // splits > 1: partial sums [split][work tile][TH*TW][COB] (fp32 / int32)
  int cus;       // compute units of the device
  int grid_cap;  // persistent kernels: at most this many workgroups (0 = no cap)
  const int32_t* rqc[3];  // int8 per-channel requantisation per stage ([2][channels]) or nullptr
  int zin[3];             // int8 zero point of each stage's input
};

// One compiled kernel instance and the tilings it implements.
typedef int (*LaunchFn)(const KArgs& a, int grid, void* stream);

struct Variant {
  int family;
  int dtype;
  int k, stride;    // depthwise geometry (1, 1 for the pointwise-only family)
  int max_p;        // output pixels per tile (TH*TW), 0 = bounded by LDS only
  int max_q;        // haloed input-window positions per tile, 0 = bounded by LDS only
  int max_cob;      // channel block of the last convolution (COB / depthwise channel block)
  int max_mb;       // intermediate-channel chunk (PW->DW->PW only), else 0
  int dw_r;         // output pixels per depthwise thread (TW must be a multiple), 0 = no DW
  LaunchFn launch;
  const char* name;
  int tile_h = 0;   // compile-time tile (0 = chosen at run time)
  int tile_w = 0;
  int gen = 1;      // 1: first generation (any layout and alignment, LDS staging)
                    // 3: NHWC persistent kernels, 16-byte channel rows, LDS-DMA staging,
                    //    run-time tile, max_p = 64 * blocks per wave
                    // 4: PW -> PW with the intermediate in registers, one pixel group per
                    //    wave (max_p = 16 * blocks), all output channels, no LDS
                    // 5: NHWC streaming kernels, compile-time tile of max_p pixels,
                    //    one compiled output-channel block
                    // 6: fp32 whole-module kernels for small batches: compile-time tile,
                    //    every channel of every stage in one workgroup
                    // 7: deep DW->PW kernels (bf16, 3x3): compile-time tile of at most 64
                    //    pixels, one compiled output-channel block
  int pitch = 0;    // gen 3: LDS window row pitch in pixels (window width must not exceed it)
  int ks = 1;       // gen 3: 64-byte channel chunks per item; gen 4: 64-byte k-steps of the
                    // first convolution held in registers (input channels <= 64 * ks bytes);
                    // gen 5: LDS ring slots
  int wc = 1;       // gen 5: waves across output channels (1, 2 or 4)
  int kc = 1;       // gen 7: 32-channel chunks per item (1 or 2)
};

// Compiled variants of each translation unit, and all of them in a fixed order
// (the index in that order is the plan's `variant`).
const Variant* variants_dwpw_f32(int* count);
const Variant* variants_dwpw_bf16(int* count);
const Variant* variants_dwpw_i8(int* count);
const Variant* variants_pwdw(int* count);
const Variant* variants_v5_dwpw_bf16_s1(int* count);
const Variant* variants_v5_dwpw_bf16_s2(int* count);
const Variant* variants_v5_pwdw_bf16(int* count);
const Variant* variants_v6_f32(int* count);
const Variant* variants_v7_bf16(int* count);
const Variant* variants_pwdwpw(int* count);
const Variant* variants_v3_dwpw_bf16_s1(int* count);
const Variant* variants_v3_dwpw_bf16_s2(int* count);
const Variant* variants_v3_dwpw_f32(int* count);
const Variant* variants_v3_dwpw_i8(int* count);
const Variant* variants_v3_pw(int* count);
const Variant* variants_v3_pw_f32(int* count);
const Variant* variants_v3_pw_i8(int* count);
const Variant* variants_v3_dw_bf16(int* count);
const Variant* variants_v3_dw_f32(int* count);
const Variant* variants_v3_dw_i8(int* count);
const Variant* variants_v4_pwpw_i8(int* count);
const Variant* variants_v4_pwpw_bf16(int* count);
const Variant* variants_v4_pwpw_f32(int* count);
const Variant* all_variants(int* count);

}  // namespace fcm
