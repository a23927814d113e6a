// fcm_kernels_v5.h -- streaming NHWC kernels for gfx950: the DW->PW module and the
// layer-by-layer PW and DW kernels built from the same pieces.
//
// k_fused5<DT, K, S, MODE, TH, TW, CTW, WC>
//   A workgroup (four waves) computes a sequence of work tiles: tile ids L, L + G, ...
//   (G workgroups), each an image, a TH x TW output tile (compile-time: the window
//   geometry and LDS layout are constants) and a block of
//   COB = 16 * CTW * WC output channels (DW: one 64-byte channel chunk). Several
//   workgroups are resident on each CU; their copies, arithmetic and stores interleave,
//   which keeps HBM busy (Sec. III-B: the module stages what the first convolution needs,
//   computes it into an on-chip buffer and writes only the second convolution's output).
//
//   The input channels are consumed in chunks of 64 bytes (one MFMA k-step); an item is
//   one chunk of one tile, and the workgroup's items form one stream. For each item, all
//   four waves issue the LDS-DMA copies (buffer_load ... lds, 16 bytes per lane;
//   out-of-range offsets read zero, which is the convolution's zero padding) of the
//   haloed input window, the chunk's pointwise weight rows and the depthwise bias, plus a
//   register load of the raw depthwise weights. Two LDS slots let the copies of item i+1
//   run while item i is computed. Waits are explicit (s_waitcnt plus a barrier). A
//   finished tile's stores are issued one item later, after the next item's copies, so
//   that by the next wait they have had a whole item's arithmetic to complete.
//
//   Waves form a WP x WC grid (WP = 4 / WC): wave (wp, wc) owns pixel blocks
//   b * WP + wp (b < NB, 16 pixels each) and output-channel tiles wc * CTW .. + CTW.
//   Lane l of a block holds pixel l % 16 and the 16-byte channel slot l / 16: exactly its
//   MFMA B operand. With WC == 1 each wave computes the depthwise stencil of its own
//   blocks straight into that operand (the DW output never leaves the registers); with
//   WC > 1 the waves split the depthwise work by blocks and exchange the result through
//   an LDS buffer, so each pixel's stencil is computed once per workgroup. The depthwise
//   multiply-adds use packed dot instructions with one half of the weight operand zero.
//   The pointwise contraction runs on MFMA with accumulators kept across chunks
//   (output-stationary). Weight rows are staged in an order that gives each accumulator
//   lane whole 16-byte granules of output channels, the four lane groups holding adjacent
//   granules, so each 16-byte store instruction writes 64 contiguous bytes of a pixel;
//   stores are non-temporal (the output is not read again by this kernel).
//
//   MODE M3_PW: no depthwise stage (window = output tile). M3_DW: no pointwise stage;
//   each lane stores its 16 bytes of depthwise output.
#pragma once

#include "fcm_kernels_v3.h"

namespace fcm {

constexpr int kThreads5 = 256;
constexpr int kWinPerWave5 = 8;  // window copy instructions per wave (window <= 512 pixels)
constexpr int kPwPerWave5 = 8;   // PW weight row copies per wave (output-channel block <= 1024)

// dma16 with a scalar part of the offset (added by the buffer unit; an out-of-range lane
// offset stays out of range since both parts are below 2^31).
__device__ __forceinline__ void dma16s(rsrc_t r, char* wave_base, uint32_t voff, uint32_t soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)wave_base, 16, voff, soff, 0,
                                           0);
}

__device__ __forceinline__ u32x4 buf_load16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ void store_nt16(void* p, const u32x4& v) { __builtin_nontemporal_store(v, (u32x4*)p); }
__device__ __forceinline__ void store_nt4(void* p, uint32_t v) { __builtin_nontemporal_store(v, (uint32_t*)p); }

template <class DT, int K, int S, int MODE, int TH, int TW, int CTW, int WC>
__global__ __launch_bounds__(kThreads5) void k_fused5(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  using D3 = Dw3<DT>;
  constexpr bool HAS_DW = MODE != M3_PW;
  constexpr bool HAS_PW = MODE != M3_DW;
  constexpr int KE = HAS_DW ? K : 1, SE = HAS_DW ? S : 1;
  constexpr int KK = KE * KE;
  constexpr int ELT = DT::ELT;
  constexpr int CB = kRowB / ELT;  // channels per chunk
  constexpr int CPL = D3::CPL;     // channels per 16-byte lane slot
  constexpr int WQ = D3::WQ;
  constexpr int WP = 4 / WC;
  constexpr int CT = CTW * WC;  // output-channel tiles of the work tile
  constexpr int COB = 16 * CT;
  constexpr int OGE = 16 / ELT;   // channels per 16-byte output granule
  constexpr int OTPG = OGE / 4;   // MFMA tiles per granule
  constexpr int NGW = HAS_PW ? CTW / OTPG : 1;  // output granules per lane
  constexpr bool SHARE = HAS_DW && HAS_PW && WC > 1;
  constexpr int P = TH * TW;
  constexpr int NB = ((P + 15) / 16 + WP - 1) / WP;  // pixel blocks per wave
  constexpr int NBT = NB * WP;                // pixel blocks of the work tile (some may be empty)
  constexpr int NBD = SHARE ? (NBT + 3) / 4 : NB;  // depthwise blocks per wave (the last may hold no pixels)
  constexpr int NRAW = HAS_DW ? (CB * KK * ELT + 1023) / 1024 : 0;  // raw DW weight loads (waves 0..)
  static_assert(WC == 1 || WC == 2 || WC == 4, "wave grid");
  static_assert(!HAS_PW || CTW % OTPG == 0, "whole output granules per lane");
  static_assert(MODE != M3_DW || WC == 1, "a depthwise-only tile has no channel split");
  static_assert(NRAW <= 4, "raw depthwise weights: one load per wave at most");
  static_assert(COB <= 1024, "PW bias block");

  constexpr int IH = HAS_DW ? (TH - 1) * SE + KE : TH;
  constexpr int IW = HAS_DW ? (TW - 1) * SE + KE : TW;
  constexpr int IWE = SE == 2 ? (IW + 1) / 2 : IW;  // stride 2: even columns first, then odd
  constexpr int NQ = IH * IW;
  constexpr Lds5 lay = lds5(dtype_id<DT>(), MODE, KE, IH, IW, COB, 2, SHARE ? 16 * NBT : 0);
  constexpr int NWI = lay.nqp / 16;                // window copies: 2 planes x nqp / 32
  constexpr int NPW = HAS_PW ? lay.cobp / 16 : 0;  // PW weight row copies
  constexpr int NTOT = NWI + NPW + (HAS_DW ? 1 : 0);  // + DW bias
  static_assert(NWI <= 4 * kWinPerWave5, "window copies per wave");
  static_assert(NPW <= 4 * kPwPerWave5, "weight row copies per wave");
  const int C = MODE == M3_DW ? a.Cm : a.Ci;
  const int nch = MODE == M3_DW ? 1 : ceil_div(C, CB);

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const int wp = wave % WP, wc = wave / WP;

  // ---- this workgroup's work tiles: logical ids L, L + G, L + 2G, ... (consecutive
  // logical ids share an XCD, so at each step an XCD works on a contiguous run of tiles:
  // the output-channel blocks of a tile and its neighbours read the same input through
  // one L2). The grid is a multiple of the number of channel blocks, so the block (and
  // with it the PW bias and weight rows) is fixed per workgroup. ----
  const int G = gridDim.x;
  const int L = xcd_remap(blockIdx.x, G);
  if (L >= a.nwork) return;
  const int ntw = (a.nwork - L + G - 1) / G;  // work tiles of this workgroup
  const int nit = ntw * nch;                  // items (tile x chunk)
  const int cb = L % a.n_cb;
  const int co0 = cb * COB;
  struct Tile {
    int n, oy0, ox0;
  };
  auto decode = [&](int id) {
    Tile r;
    int t = id / a.n_cb;
    const int tx = t % a.tiles_x;
    t /= a.tiles_x;
    const int ty = t % a.tiles_y;
    r.n = t / a.tiles_y;
    r.oy0 = ty * TH;
    r.ox0 = tx * TW;
    return r;
  };

  const T* x = (const T*)a.x;
  const size_t img = (size_t)a.H * a.W * C;
  const T* wpw = (const T*)(MODE == M3_PW ? a.w1 : a.w2);
  const T* wdw = (const T*)a.w1;
  const void* bd = a.b1;
  const void* bp = MODE == M3_PW ? a.b1 : a.b2;
  const rsrc_t rw = make_rsrc(wpw, HAS_PW ? (uint32_t)((size_t)a.Co * a.Ci * ELT) : 0u);
  const rsrc_t rwd = make_rsrc(wdw, HAS_DW ? (uint32_t)((size_t)C * KK * ELT) : 0u);
  const rsrc_t rbd = make_rsrc(bd ? bd : (const void*)wdw, (HAS_DW && bd) ? (uint32_t)(C * 4) : 0u);
  const rsrc_t rbp = make_rsrc(bp ? bp : (const void*)wpw, (HAS_PW && bp) ? (uint32_t)(a.Co * 4) : 0u);

  // This wave's copies of a chunk: instructions i = wave + 4k of the list
  // [window | PW weight rows | DW bias]; i & 1 is the plane (both parts have an even
  // count), so each lane always copies 16-byte slot `sl` of a channel row.
  const int sl = 2 * (wave & 1) + (lane & 1);
  // Window pixel this lane copies in its k-th window instruction, the same for every
  // tile: (wy << 16) | wx within the window, or -1 beyond it.
  int wyx[kWinPerWave5];
#pragma unroll
  for (int k = 0; k < kWinPerWave5; ++k) {
    const int i = wave + 4 * k;
    wyx[k] = -1;
    if (i >= NWI) break;  // wave-uniform
    const int q = 32 * (i >> 1) + (lane >> 1);  // stored window position
    if (q < NQ) {
      const int wy = q / IW, wxs = q - wy * IW;
      wyx[k] = (wy << 16) | (SE == 2 ? (wxs < IWE ? 2 * wxs : 2 * (wxs - IWE) + 1) : wxs);
    }
  }
  const uint32_t pixb = (uint32_t)(C * ELT), rowb = (uint32_t)a.W * pixb;
  // Per tile: the lane part of each window copy's byte offset (kOob outside the image)
  // and a scalar part: interior tiles put the tile origin in the scalar part and need no
  // bounds checks; border tiles check every position.
  uint32_t woff[kWinPerWave5];
  uint32_t wsoff = 0;
  auto window_offsets = [&](const Tile& t) {
    const int iy0 = HAS_DW ? t.oy0 * SE - a.pad : t.oy0;
    const int ix0 = HAS_DW ? t.ox0 * SE - a.pad : t.ox0;
    const bool interior = iy0 >= 0 && ix0 >= 0 && iy0 + IH <= a.H && ix0 + IW <= a.W;  // wave-uniform
    wsoff = interior ? (uint32_t)(iy0 * a.W + ix0) * pixb : 0u;
#pragma unroll
    for (int k = 0; k < kWinPerWave5; ++k) {
      if (wave + 4 * k >= NWI) break;
      const int v = wyx[k], wy = v >> 16, wx = v & 0xffff;
      if (interior) {
        woff[k] = v < 0 ? kOob : __umul24((uint32_t)wy, rowb) + __umul24((uint32_t)wx, pixb);
      } else {
        const int gy = iy0 + wy, gx = ix0 + wx;
        const bool ok = v >= 0 && (unsigned)gy < (unsigned)a.H && (unsigned)gx < (unsigned)a.W;
        woff[k] = ok ? (uint32_t)(gy * a.W + gx) * pixb : kOob;
      }
    }
  };
  // pointwise weight rows of this wave's copies (fixed: the channel block is): byte
  // offset of the row, or kOob for rows beyond the block or beyond c_out
  const int pw_first = wave + 4 * ((NWI - wave + 3) / 4);  // first instruction of the PW part
  uint32_t poff[kPwPerWave5];
#pragma unroll
  for (int k = 0; k < kPwPerWave5; ++k) {
    poff[k] = kOob;
    const int tt = pw_first + 4 * k - NWI;
    if (!HAS_PW || tt >= NPW) break;  // wave-uniform
    const int r = 32 * (tt >> 1) + (lane >> 1);  // staged row
    const int ti = r >> 4, m = r & 15;
    const int co = co0 + OGE * (4 * (ti / OTPG) + (m >> 2)) + 4 * (ti % OTPG) + (m & 3);
    if (r < COB && co < a.Co) poff[k] = (uint32_t)(co * a.Ci * ELT);
  }

  auto slotp = [&](int s) { return smem + s * lay.slot_bytes; };
  // Issue the copies of chunk c of a tile of image n into ring slot s (window offsets
  // already computed for the tile); `raw` receives this lane's 16 bytes of the chunk's
  // raw depthwise weights ([c][k][k] order).
  auto issue = [&](int n, int c, int s, u32x4& raw) {
    char* sb = slotp(s);
    const int c0 = MODE == M3_DW ? cb * CB : c * CB;
    if constexpr (HAS_DW) {
      if (wave < NRAW) raw = buf_load16(rwd, (uint32_t)(c0 * KK * ELT + wave * 1024 + lane * 16));
    }
    const rsrc_t rx = make_rsrc(x + (size_t)n * img, (uint32_t)(img * ELT));
    const int cs = c0 + sl * CPL;  // first channel of this lane's slot
    const bool cok = c0 + CB <= C || cs < C;  // (only a ragged last chunk has lanes beyond C)
    const uint32_t coff = (uint32_t)(sl * CPL * ELT);
    const uint32_t soff = wsoff + (uint32_t)(c0 * ELT);  // scalar
#pragma unroll
    for (int k = 0; k < kWinPerWave5; ++k) {
      const int i = wave + 4 * k;
      if (i >= NWI) break;
      dma16s(rx, sb + (i & 1) * (lay.nqp * 32) + (i >> 1) * 1024, cok ? woff[k] + coff : kOob, soff);
    }
    if constexpr (HAS_PW) {
#pragma unroll
      for (int k = 0; k < kPwPerWave5; ++k) {
        const int tt = pw_first + 4 * k - NWI;
        if (tt >= NPW) break;  // wave-uniform
        dma16s(rw, sb + lay.win_bytes + (tt & 1) * (lay.cobp * 32) + (tt >> 1) * 1024, cok ? poff[k] + coff : kOob,
               (uint32_t)(c0 * ELT));
      }
    }
    if constexpr (HAS_DW) {
      if (wave == (NTOT - 1) % 4 && lane < CB / 4)
        dma16(rbd, sb + lay.dw_off + KK * CB * 4, (uint32_t)(c0 * 4 + lane * 16));
    }
  };
  // Raw depthwise weights of a chunk (in registers) -> dot-operand words [tap][CB] in
  // the slot.
  auto convert = [&](int s, const u32x4& raw) {
    if constexpr (HAS_DW) {
      if (wave >= NRAW) return;
      constexpr int EPV = 16 / ELT;
      uint32_t* dst = (uint32_t*)(slotp(s) + lay.dw_off);
#pragma unroll
      for (int k = 0; k < EPV; ++k) {
        const int e = (wave * 64 + lane) * EPV + k;
        if (e < CB * KK) {
          const uint32_t word = raw[k * ELT / 4];
          uint32_t el;
          if constexpr (ELT == 4)
            el = word;
          else if constexpr (ELT == 2)
            el = (k & 1) ? word >> 16 : word & 0xffffu;
          else
            el = (word >> (8 * (k & 3))) & 0xffu;
          const int ci = e / KK, tap = e - (e / KK) * KK;
          dst[tap * CB + ci] = D3::weight_word(el, ci);
        }
      }
    }
  };

  // ---- per-lane compute state ----
  const Epi3 ep_dw = make_epi3(a.act[0], a.rq[0]);
  const Epi3 ep_pw = MODE == M3_PW ? ep_dw : make_epi3(a.act[1], a.rq[1]);
  AccV acc[NB][CTW];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < CTW; ++i) acc[b][i] = AccV{0, 0, 0, 0};
  u32x4 bop[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) bop[b] = u32x4{0u, 0u, 0u, 0u};
  // depthwise blocks of this wave: with WC == 1 its own MFMA blocks, else wave + 4j
  auto dw_block = [&](int j) { return SHARE ? wave + 4 * j : j * 4 + wave; };
  int nlive = 0;  // depthwise blocks of this wave that hold pixels (a prefix; wave-uniform)
#pragma unroll
  for (int j = 0; j < NBD; ++j)
    if (dw_block(j) * 16 < P) nlive = j + 1;
  const int plane_in = (g >> 1) * (lay.nqp * 32) + (g & 1) * 16;  // this lane's slot in a window pixel

  // ---- epilogue of a finished work tile, straight from registers to global memory:
  // +bias, activation, cast (PW); the depthwise output (DW only). Issued one item late,
  // after the next item's copies, so that the wait for those copies never has to wait
  // for fresh stores as well (stores and loads share the counter). ----
  const bool full16 = (a.Co * ELT) % 16 == 0;
  // Output pixel of each of this lane's pixel blocks within a tile, the same for every
  // tile: (py << 16) | px, or -1 past the tile; and its byte offset from the tile's first
  // output pixel (the lane's first channel included). A tile's base address is scalar.
  const int cl0 = co0 + OGE * (4 * wc * NGW + g);  // this lane's first output channel (PW)
  const int nbo = HAS_PW ? NB : NBD;              // blocks this lane stores
  int eyx[HAS_PW ? NB : NBD];
  uint32_t eoff[HAS_PW ? NB : NBD];
  const int ochan = HAS_PW ? a.Co : C;  // channels of an output pixel
#pragma unroll
  for (int b = 0; b < nbo; ++b) {
    const int p = (HAS_PW ? (b * WP + wp) : dw_block(b)) * 16 + r16;
    const int py = p / TW, px = p - py * TW;
    eyx[b] = p < P ? (py << 16) | px : -1;
    eoff[b] = (uint32_t)(((py * a.Wo + px) * ochan + (HAS_PW ? cl0 : cb * CB + g * CPL)) * ELT);
  }
  // lanes whose pixel lies in the image (tiles at the right and bottom edges are partial)
  auto out_ok = [&](const Tile& t, int b) {
    const int v = eyx[b];
    const bool full = t.oy0 + TH <= a.Ho && t.ox0 + TW <= a.Wo;  // wave-uniform
    return v >= 0 && (full || ((v >> 16) < a.Ho - t.oy0 && (v & 0xffff) < a.Wo - t.ox0));
  };
  auto epilogue = [&](const Tile& t) {
    char* tbase = (char*)a.y + (size_t)((t.n * a.Ho + t.oy0) * a.Wo + t.ox0) * ochan * ELT;
    if constexpr (HAS_PW) {
      const char* bl = smem + lay.pwb_off;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        if (!out_ok(t, b)) continue;
        // granule k of this lane: channels cl0 + 4 * OGE * k + [0, OGE); channel
        // cl0 + 4 * OGE * k + 4t + e is value e of local tile k * OTPG + t
        char* dpx = tbase + eoff[b];
#pragma unroll
        for (int k = 0; k < NGW; ++k) {
          if (cl0 + 4 * OGE * k >= a.Co) break;
          Acc bias[OGE];
#pragma unroll
          for (int q = 0; q < OGE / 4; ++q) {
            const u32x4 bv = *(const u32x4*)(bl + (OGE * (4 * (wc * NGW + k) + g) + 4 * q) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t u = bv[e];
              bias[4 * q + e] = __builtin_bit_cast(Acc, u);
            }
          }
          uint32_t wd4[4];
          if constexpr (ELT == 4) {
#pragma unroll
            for (int e = 0; e < 4; ++e) wd4[e] = __float_as_uint(epi_f(acc[b][k][e] + bias[e], ep_pw));
          } else if constexpr (ELT == 2) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const int tt = w >> 1, e = 2 * (w & 1);
              wd4[w] = pack_bf16x2(epi_f(acc[b][2 * k + tt][e] + bias[4 * tt + e], ep_pw),
                                   epi_f(acc[b][2 * k + tt][e + 1] + bias[4 * tt + e + 1], ep_pw));
            }
          } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              uint32_t wv = 0;
#pragma unroll
              for (int e = 0; e < 4; ++e)
                wv |= ((uint32_t)epi_i(acc[b][4 * k + w][e] + bias[4 * w + e], ep_pw) & 0xffu) << (8 * e);
              wd4[w] = wv;
            }
          }
          char* dst = dpx + 64 * k;  // 4 * OGE channels of ELT bytes
          if (full16) {
            store_nt16(dst, u32x4{wd4[0], wd4[1], wd4[2], wd4[3]});
          } else {
            // c_out * elt is a multiple of 4: whole 32-bit words are in or out of range
#pragma unroll
            for (int w = 0; w < 4; ++w)
              if (cl0 + 4 * OGE * k + w * (4 / ELT) < a.Co) store_nt4(dst + 4 * w, wd4[w]);
          }
        }
      }
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < CTW; ++i) acc[b][i] = AccV{0, 0, 0, 0};
    } else {
      // depthwise only: this lane's 16 bytes of channels of each of its pixels
      const bool chok = cb * CB + g * CPL < C;
#pragma unroll
      for (int j = 0; j < NBD; ++j)
        if (chok && out_ok(t, j)) store_nt16(tbase + eoff[j], bop[j]);
    }
  };

  // ---- prologue: PW bias block of the channel block, window offsets and copies of the
  // first item ----
  if constexpr (HAS_PW) {
    if (wave == 0) {
#pragma unroll
      for (int j = 0; j < (COB * 4 + 1023) / 1024; ++j)
        if (j * 1024 + lane * 16 < COB * 4)
          dma16(rbp, smem + lay.pwb_off + j * 1024, (uint32_t)(co0 * 4 + j * 1024 + lane * 16));
    }
  }
  u32x4 raw = {0u, 0u, 0u, 0u};
  int is_k = 0, is_c = 0;  // next item to issue: tile index, chunk
  Tile is_t = decode(L);
  window_offsets(is_t);
  issue(is_t.n, 0, 0, raw);
  if (++is_c == nch) {
    is_c = 0;
    ++is_k;
  }
  Tile pend_t = is_t;
  int cur_c = 0;  // chunk of the item being computed
  bool pending = false;

  for (int it = 0; it < nit; ++it) {
    const int s = it & 1;
    // this wave's copies of item it (and its stores of the tile before) are complete
    wait_vm_n<0>();
    convert(s, raw);
    wait_lgkm0();
    barrier3();  // every wave's copies and conversions of item it are visible; slot s ^ 1 is free
    if (it + 1 < nit) {
      if (is_c == 0) {
        is_t = decode(L + is_k * G);
        window_offsets(is_t);
      }
      issue(is_t.n, is_c, s ^ 1, raw);
      if (++is_c == nch) {
        is_c = 0;
        ++is_k;
      }
    }
    if (pending) {
      epilogue(pend_t);
      pending = false;
    }
    const char* sb = slotp(s);

    if constexpr (HAS_DW) {
      // The first NL depthwise blocks of this wave hold pixels; NL is a compile-time
      // constant of each instance of `dw`, so the unrolled tap loop carries no branches.
      auto dw = [&](auto nl_tag) {
        constexpr int NL = decltype(nl_tag)::value;
        const char* wl = sb + lay.dw_off;
        const char* xb[NL];
#pragma unroll
        for (int j = 0; j < NL; ++j) {
          const int p = min(dw_block(j) * 16 + r16, P - 1);
          const int py = p / TW, px = p - py * TW;
          xb[j] = sb + plane_in + ((py * SE) * IW + px) * 32;
        }
        Acc dacc[NL][CPL];
        {
          u32x4 bv[WQ];
#pragma unroll
          for (int q = 0; q < WQ; ++q) bv[q] = *(const u32x4*)(wl + (KK * CB + g * CPL + 4 * q) * 4);
#pragma unroll
          for (int j = 0; j < NL; ++j)
#pragma unroll
            for (int e = 0; e < CPL; ++e) {
              const uint32_t u = bv[e >> 2][e & 3];
              dacc[j][e] = __builtin_bit_cast(Acc, u);
            }
        }
#pragma unroll
        for (int ky = 0; ky < KE; ++ky) {
#pragma unroll
          for (int kx = 0; kx < KE; ++kx) {
            const int toff = (ky * IW + (SE == 2 ? ((kx & 1) ? IWE + (kx >> 1) : (kx >> 1)) : kx)) * 32;
            u32x4 wv[WQ];
#pragma unroll
            for (int q = 0; q < WQ; ++q) wv[q] = *(const u32x4*)(wl + ((ky * KE + kx) * CB + g * CPL + 4 * q) * 4);
#pragma unroll
            for (int j = 0; j < NL; ++j) D3::tap(dacc[j], *(const u32x4*)(xb[j] + toff), wv);
          }
        }
#pragma unroll
        for (int j = 0; j < NL; ++j) {
          const u32x4 out = D3::finish(dacc[j], ep_dw);
          if constexpr (SHARE)
            *(u32x4*)(smem + lay.dwo_off + (g >> 1) * (16 * NBT * 32) + (dw_block(j) * 16 + r16) * 32 + (g & 1) * 16) =
                out;
          else
            bop[j] = out;
        }
      };
      if (nlive == NBD) {
        dw(std::integral_constant<int, NBD>{});
      } else if constexpr (NBD > 1) {
        if (nlive == 1) dw(std::integral_constant<int, 1>{});
        else if (nlive == 2) dw(std::integral_constant<int, (NBD > 2 ? 2 : 1)>{});
        else if (nlive == 3) dw(std::integral_constant<int, (NBD > 3 ? 3 : 1)>{});
        else if (nlive >= 4) dw(std::integral_constant<int, (NBD > 4 ? 4 : 1)>{});
      }
    }
    if constexpr (HAS_PW) {
      if constexpr (SHARE) {
        wait_lgkm0();
        barrier3();  // depthwise output of the whole tile is in the exchange buffer
      }
      // B operands of this wave's blocks
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int pb = b * WP + wp;
        if constexpr (SHARE) {
          bop[b] = *(const u32x4*)(smem + lay.dwo_off + (g >> 1) * (16 * NBT * 32) + (pb * 16 + r16) * 32 + (g & 1) * 16);
        } else if constexpr (!HAS_DW) {
          const int p = min(pb * 16 + r16, P - 1);
          bop[b] = *(const u32x4*)(sb + plane_in + p * 32);
        }
      }
      const char* wl = sb + lay.win_bytes + (g >> 1) * (lay.cobp * 32) + (g & 1) * 16;
#pragma unroll
      for (int i = 0; i < CTW; ++i) {
        const u32x4 av = *(const u32x4*)(wl + ((wc * CTW + i) * 16 + r16) * 32);
#pragma unroll
        for (int b = 0; b < NB; ++b)
          if ((b * WP + wp) * 16 < P) mma16(DT{}, acc[b][i], av, bop[b]);
      }
    }
    if (++cur_c == nch) {  // the work tile of item it is complete
      pending = true;
      pend_t = decode(L + (it / nch) * G);
      cur_c = 0;
    }
  }
  if (pending) epilogue(pend_t);
}

template <class DT, int K, int S, int MODE, int TH, int TW, int CTW, int WC>
int launch_fused5(const KArgs& a, int grid, void* stream) {
  auto fn = k_fused5<DT, K, S, MODE, TH, TW, CTW, WC>;
  const int lds = a.L.bytes;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return (int)e;
  }
  // persistent grid: the workgroups resident at once (or the plan's cap), at most one per
  // work tile, a multiple of the channel-block count (each workgroup keeps one block)
  static thread_local int cached_lds = -1, cached_occ = 1;
  if (cached_lds != lds) {
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)fn, kThreads5, lds) != hipSuccess || occ < 1)
      occ = 1;
    cached_lds = lds;
    cached_occ = occ;
  }
  int g = a.cus * cached_occ;
  if (a.grid_cap > 0 && g > a.grid_cap) g = a.grid_cap;
  if (g > a.nwork) g = a.nwork;
  g -= g % a.n_cb;
  if (g < a.n_cb) g = a.n_cb;
  (void)grid;
  return launch_args((const void*)fn, g, kThreads5, lds, stream, a);
}

}  // namespace fcm
