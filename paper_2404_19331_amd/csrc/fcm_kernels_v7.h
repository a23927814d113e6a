// fcm_kernels_v7.h -- DW->PW for deep layers (bf16, 3x3, many channels, small images).
//
// k_deep7<S, TH, TW, CTW, KC>
//   Persistent, eight waves, one workgroup per CU. A workgroup owns a block of COB = 64 * CTW
//   output channels and computes a sequence of work tiles (image, TH x TW output tile, at
//   most 64 pixels), each over the input channels in chunks of 32 (one MFMA k-step); an
//   item is KC chunks of one tile (two halve the barriers and waits per channel). Such
//   layers are bound neither by HBM nor by the matrix cores but by the instruction
//   streams of the waves, the latency of their loads and the LDS traffic, so the work of
//   an item is split over two kinds of waves, one of each on every SIMD, so that one's
//   vector ALU work and LDS reads overlap the other's MFMAs:
//   * Depthwise waves (0..3, wave d = 8-channel slot d of each chunk, lane = output
//     pixel): copy their own channel plane of each chunk of the haloed window of item
//     i + 3 into a ring of three LDS slots (LDS-DMA; LDS planes of 8 channels, so that a wave's reads at consecutive
//     positions are free of bank conflicts), compute the stencil of item i + 1 and write it to an LDS
//     exchange buffer (two of them, planes of 8 channels: the MFMA B-operand layout). All
//     depthwise weights and biases are copied into LDS once; per item the 72 weights of a
//     wave's slot and its 8 biases are read into four VGPRs spread over lanes 0..8 and
//     9..10 of each 16-lane row and reach every lane through the DPP operand of the dot
//     instruction (row_newbcast). The dot instruction multiplies two bf16 pairs and the
//     weights stored [C][3][3] come in pairs of consecutive taps of one channel, so the
//     lane pairs consecutive taps of its inputs to match (one byte permute per pair): a
//     channel's nine taps take four paired dots and one single one (other half zero).
//   * MFMA waves (4..7, wave m = output-channel tiles m*CTW .. +CTW): load the pointwise
//     weights of item i + 2 straight into MFMA A-operand registers (rows in the order that
//     gives each accumulator lane whole 16-byte granules of output channels), contract
//     every pixel block of item i's exchange buffer, and after a tile's last chunk store
//     it (+bias, activation, bf16) straight from the accumulators, one non-temporal 16-byte
//     buffer store per granule (out-of-range offsets outside the image, so every wave
//     issues the same number of stores).
//   One barrier per item; each wave's waits are counted (its loads of one item complete
//   before the item's use, two items later). Accumulators stay in registers across the
//   chunks of a tile (output-stationary, Sec. III-A).
#pragma once

#include "fcm_kernels_v5.h"

namespace fcm {

constexpr int kThreads7 = 512;

// acc += dot(bf16 pair w of lane N of this lane's row, bf16 pair x): the weight register
// is broadcast within each 16-lane row by DPP (every row holds the same weights). A dot
// instruction's result needs three wait states before another kind of VALU instruction
// may read it (a following dot reading it as its accumulator needs none), and the
// compiler does not see through the asm: the last dot of a chain (LAST) adds them.
template <int N, bool LAST = false>
__device__ __forceinline__ void dot_bcast7(float& acc, uint32_t w, uint32_t x) {
  if constexpr (LAST)
    asm("v_dot2c_f32_bf16_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf\n\ts_nop 2"
        : "+v"(acc)
        : "v"(w), "v"(x), "n"(N));
  else
    asm("v_dot2c_f32_bf16_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf" : "+v"(acc) : "v"(w), "v"(x),
        "n"(N));
}
template <int N>
__device__ __forceinline__ float bcast7(uint32_t v) {
  return __uint_as_float((uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x150 + N, 0xf, 0xf, true));
}
template <int B, int E, class F>
__device__ __forceinline__ void static_for7(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for7<B + 1, E>(f);
  }
}

// Depthwise taps of channel J (0..7) of a wave's 8-channel slot: xv[t] holds the slot's
// inputs at tap t (word k = channels 2k, 2k + 1), the weights are elements 9J .. 9J + 8 of
// the slot's 36 words, lane l (0..8) of each row holding words 4l .. 4l + 3. Even J: taps (0,1)
// (2,3) (4,5) (6,7) in one word each, tap 8 in the low half of the next; odd J: tap 0 in
// the high half of a word, then (1,2) .. (7,8). The inputs are paired to match.
template <int Q, bool LAST = false>
__device__ __forceinline__ void dot_word7(float& acc, const u32x4& wv, uint32_t x) {
  static_assert(Q >= 0 && Q < 36, "an 8-channel slot has 36 weight words");
  dot_bcast7<Q / 4, LAST>(acc, wv[Q % 4], x);
}
template <int J>
__device__ __forceinline__ void dw_channel7(float& acc, const u32x4 (&xv)[9], const u32x4& wv) {
  constexpr int k = J >> 1;
  if constexpr ((J & 1) == 0) {
    constexpr int q = 9 * J / 2;
    dot_word7<q + 0>(acc, wv, __builtin_amdgcn_perm(xv[1][k], xv[0][k], 0x05040100u));
    dot_word7<q + 1>(acc, wv, __builtin_amdgcn_perm(xv[3][k], xv[2][k], 0x05040100u));
    dot_word7<q + 2>(acc, wv, __builtin_amdgcn_perm(xv[5][k], xv[4][k], 0x05040100u));
    dot_word7<q + 3>(acc, wv, __builtin_amdgcn_perm(xv[7][k], xv[6][k], 0x05040100u));
    dot_word7<q + 4, true>(acc, wv, xv[8][k] & 0xffffu);
  } else {
    constexpr int q = (9 * J - 1) / 2;
    dot_word7<q + 0>(acc, wv, xv[0][k] & 0xffff0000u);
    dot_word7<q + 1>(acc, wv, __builtin_amdgcn_perm(xv[2][k], xv[1][k], 0x07060302u));
    dot_word7<q + 2>(acc, wv, __builtin_amdgcn_perm(xv[4][k], xv[3][k], 0x07060302u));
    dot_word7<q + 3>(acc, wv, __builtin_amdgcn_perm(xv[6][k], xv[5][k], 0x07060302u));
    dot_word7<q + 4, true>(acc, wv, __builtin_amdgcn_perm(xv[8][k], xv[7][k], 0x07060302u));
  }
}

__device__ __forceinline__ u32x4 buf_load16s(rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
__device__ __forceinline__ void buf_store_nt16(const u32x4& v, rsrc_t r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 2);
}

template <int S, int TH, int TW, int CTW, int KC>
__global__ __launch_bounds__(kThreads7) void k_deep7(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  constexpr int K = 3, ELT = 2, CB = 32;
  constexpr int P = TH * TW;
  static_assert(P <= 64, "one output pixel per lane");
  constexpr int NB = (P + 15) / 16;  // 16-pixel blocks
  constexpr int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K;
  constexpr int IWE = S == 2 ? (IW + 1) / 2 : IW;  // stride 2: even columns first, then odd
  constexpr int NQ = IH * IW;
  constexpr Lds7 lay = lds7(S, TH, TW, CTW, 0, KC);  // (the C-dependent offsets below)
  constexpr int ND = 4;               // depthwise waves, one 8-channel plane of each chunk
  constexpr int NWW = lay.nqp / 64;   // window copies (1 KiB: 64 positions) per wave
  static_assert(NWW <= kWinPerWave5, "window copies per wave");
  constexpr int COB = 64 * CTW;
  constexpr int OGE = 8, OTPG = 2, NGW = CTW / OTPG;
  static_assert(CTW % OTPG == 0, "whole output granules per lane");
  constexpr int NST = NB * NGW;  // epilogue stores per MFMA wave
  const int C = a.Ci;  // a multiple of the item's KC chunks
  const int nch = C / (CB * KC);  // items per tile

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;

  // ---- work tiles L, L + G, ... (the grid is a multiple of the channel-block count, so
  // the block is fixed per workgroup) ----
  const int G = gridDim.x;
  const int L = xcd_remap(blockIdx.x, G);
  if (L >= a.nwork) return;
  const int ntw = (a.nwork - L + G - 1) / G;
  const int nit = ntw * nch;
  const int cb = L % a.n_cb;
  const int co0 = cb * COB;
  // spatial tile (column, row, image) of tile index L / n_cb, stepped by G / n_cb without
  // divisions (the step's own parts are below tiles_x and tiles_y)
  struct Tile {
    int tx, ty, n;
  };
  const int step = G / a.n_cb;
  const int sx = step % a.tiles_x, sy = (step / a.tiles_x) % a.tiles_y, sn = step / (a.tiles_x * a.tiles_y);
  Tile t0;
  {
    const int t = L / a.n_cb;
    t0.tx = t % a.tiles_x;
    t0.ty = (t / a.tiles_x) % a.tiles_y;
    t0.n = t / (a.tiles_x * a.tiles_y);
  }
  auto advance = [&](Tile& t) {
    t.tx += sx;
    const int c1 = t.tx >= a.tiles_x;
    t.tx -= c1 ? a.tiles_x : 0;
    t.ty += sy + c1;
    const int c2 = t.ty >= a.tiles_y;
    t.ty -= c2 ? a.tiles_y : 0;
    t.n += sn + c2;
  };
  // scalar offset of a load that must read zeros: with per-lane offsets below 2^31 and
  // buffers below 2^30 bytes, the sum is out of range and does not wrap
  constexpr uint32_t kOobS = 0x40000000u;
  // the items run in groups of three (the register sets of the loads rotate with them);
  // no path back to a loop head skips a body, so loads retire in the order the counted
  // waits assume
  auto run_items = [&](auto&& body) {
    int it = 0;
    for (; it + 3 <= nit; it += 3) {
      body(std::integral_constant<int, 0>{}, it);
      body(std::integral_constant<int, 1>{}, it + 1);
      body(std::integral_constant<int, 2>{}, it + 2);
    }
    if (it < nit) body(std::integral_constant<int, 0>{}, it);
    if (it + 1 < nit) body(std::integral_constant<int, 1>{}, it + 1);
  };

  if (wave < ND) {
    // ================= depthwise waves =================
    const int wd = wave;
    const uint16_t* x = (const uint16_t*)a.x;
    const size_t img = (size_t)a.H * a.W * C;
    // window copies: wave wd fills plane wd (channels 8wd .. 8wd + 7 of the chunk); its
    // copy k covers stored positions 64k .. 64k + 63, lane l position 64k + l
    int wyx[NWW];
#pragma unroll
    for (int k = 0; k < NWW; ++k) {
      const int q = 64 * k + lane;
      wyx[k] = -1;
      if (q < NQ) {
        const int wy = q / IW, wxs = q - wy * IW;
        wyx[k] = (wy << 16) | (S == 2 ? (wxs < IWE ? 2 * wxs : 2 * (wxs - IWE) + 1) : wxs);
      }
    }
    const uint32_t pixb = (uint32_t)(C * ELT), rowb = (uint32_t)a.W * pixb;
    const uint32_t coff = (uint32_t)(wd * 16);
    uint32_t woff[NWW];
    uint32_t wsoff = 0;
    rsrc_t rx = make_rsrc(x, 0u);
    int w_c = 0;   // chunk of the next window to load
    Tile wt = t0;  // its tile
    auto window_tile = [&]() {
      rx = make_rsrc(x + (size_t)wt.n * img, (uint32_t)(img * ELT));
      const int iy0 = wt.ty * TH * S - a.pad, ix0 = wt.tx * TW * S - a.pad;
      const bool interior = iy0 >= 0 && ix0 >= 0 && iy0 + IH <= a.H && ix0 + IW <= a.W;
      wsoff = interior ? (uint32_t)(iy0 * a.W + ix0) * pixb : 0u;
#pragma unroll
      for (int k2 = 0; k2 < NWW; ++k2) {
        const int v = wyx[k2], wy = v >> 16, wx = v & 0xffff;
        if (interior) {
          woff[k2] = v < 0 ? kOob : __umul24((uint32_t)wy, rowb) + __umul24((uint32_t)wx, pixb) + coff;
        } else {
          const int gy = iy0 + wy, gx = ix0 + wx;
          const bool ok = v >= 0 && (unsigned)gy < (unsigned)a.H && (unsigned)gx < (unsigned)a.W;
          woff[k2] = ok ? (uint32_t)(gy * a.W + gx) * pixb + coff : kOob;
        }
      }
    };
    // window of the next item into ring slot SLOT (plane wd of each of its KC chunks at
    // planes wd, wd + 4, ..); an item at or beyond nit loads zeros
    auto issue = [&](int slot, bool valid) {
      if (valid && w_c == 0) window_tile();
#pragma unroll
      for (int s = 0; s < KC; ++s) {
        const uint32_t soff = valid ? wsoff + (uint32_t)((w_c * KC + s) * CB * ELT) : kOobS;
#pragma unroll
        for (int k = 0; k < NWW; ++k)
          dma16s(rx, smem + slot * lay.win_bytes + (wd + ND * s) * lay.win_plane + k * 1024, woff[k], soff);
      }
      if (valid && ++w_c == nch) {
        w_c = 0;
        advance(wt);
      }
    };
    // the stencil of one item: lane = output pixel (clamped into the tile); reads window
    // slot SLOT, writes exchange buffer e
    const int pl = lane < P ? lane : P - 1;
    const int ppy = pl / TW, ppx = pl - ppy * TW;
    const int xoff = wd * lay.win_plane + ((ppy * S) * IW + ppx) * 16;
    const int woutoff = lay.exch_off + wd * lay.exch_plane + lane * 16;
    const Epi3 ep_dw = make_epi3(a.act[0], a.rq[0]);
    // all depthwise weights and biases stay in LDS; a wave reads its slot's 36 weight words
    // into lanes 0..8 of each row (four each) and its 8 biases into lanes 9..10
    const int dwb_off = lay.dww_off + round_up(C * 18, 1024);
    const int wboff = r16 < 9 ? lay.dww_off + 8 * wd * 18 + 16 * r16
                              : (r16 < 11 ? dwb_off + 8 * wd * 4 + 16 * (r16 - 9) : lay.dww_off);
    int d_c = 0;  // chunk of the next depthwise item
    auto depthwise = [&](int slot, int e) {
#pragma unroll
      for (int s = 0; s < KC; ++s) {
        const int dc = d_c * KC + s;  // chunk of the tile
        const u32x4 wv = *(const u32x4*)(smem + wboff + (r16 < 9 ? dc * CB * 18 : (r16 < 11 ? dc * CB * 4 : 0)));
        const u32x4& bv = wv;
        const char* xb = smem + slot * lay.win_bytes + xoff + s * ND * lay.win_plane;
        u32x4 xv[9];
#pragma unroll
        for (int ky = 0; ky < K; ++ky)
#pragma unroll
          for (int kx = 0; kx < K; ++kx) {
            const int toff = (ky * IW + (S == 2 ? ((kx & 1) ? IWE + (kx >> 1) : (kx >> 1)) : kx)) * 16;
            xv[ky * K + kx] = *(const u32x4*)(xb + toff);
          }
        float acc[8];
        acc[0] = bcast7<9>(bv[0]);
        acc[1] = bcast7<9>(bv[1]);
        acc[2] = bcast7<9>(bv[2]);
        acc[3] = bcast7<9>(bv[3]);
        acc[4] = bcast7<10>(bv[0]);
        acc[5] = bcast7<10>(bv[1]);
        acc[6] = bcast7<10>(bv[2]);
        acc[7] = bcast7<10>(bv[3]);
        static_for7<0, 8>([&](auto jc) {
          constexpr int J = decltype(jc)::value;
          dw_channel7<J>(acc[J], xv, wv);
        });
        u32x4 out;
#pragma unroll
        for (int j = 0; j < 4; ++j) out[j] = pack_bf16x2(epi_f(acc[2 * j], ep_dw), epi_f(acc[2 * j + 1], ep_dw));
        if (lane < NB * 16) *(u32x4*)(smem + woutoff + e * lay.exch_bytes + s * ND * lay.exch_plane) = out;
      }
      if (++d_c == nch) d_c = 0;
    };

    // the weights and biases of every channel (1 KiB copies over the four waves, first),
    // then the windows of items 0..2
    {
      const rsrc_t rdw = make_rsrc(a.w1, (uint32_t)(C * 9 * ELT));
      const rsrc_t rdb = make_rsrc(a.b1 ? a.b1 : a.w1, a.b1 ? (uint32_t)(C * 4) : 0u);
      const int nbw = ceil_div(C * 18, 1024), nbb = ceil_div(C * 4, 1024);
      for (int j = wd; j < nbw + nbb; j += ND) {
        if (j < nbw) dma16(rdw, smem + lay.dww_off + j * 1024, (uint32_t)(j * 1024 + lane * 16));
        else dma16(rdb, smem + dwb_off + (j - nbw) * 1024, (uint32_t)((j - nbw) * 1024 + lane * 16));
      }
    }
    constexpr int NIS = NWW * KC;  // loads per item
    issue(0, true);
    issue(1, 1 < nit);
    issue(2, 2 < nit);
    wait_vm_n<2 * NIS>();  // the weights and the window of item 0
    barrier3();
    depthwise(0, 0);
    wait_vm_n<NIS>();  // window of item 1
    wait_lgkm0();
    barrier3();
    run_items([&](auto setc, int it) {
      constexpr int SET = decltype(setc)::value;
      constexpr int S1 = (SET + 1) % 3;
      issue(SET, it + 3 < nit);
      depthwise(S1, (it + 1) & 1);
      wait_vm_n<NIS>();  // window of item it + 2
      wait_lgkm0();
      barrier3();
    });
  } else {
    // ================= MFMA waves =================
    const int wm = wave - ND;
    // pointwise A operands: this lane's weight row of each of the wave's output tiles (16
    // bytes of channels 8g .. 8g + 7 of a chunk), byte offsets, kOob beyond c_out
    const rsrc_t rw = make_rsrc(a.w2, (uint32_t)((size_t)a.Co * a.Ci * ELT));
    uint32_t aoff[CTW];
#pragma unroll
    for (int i = 0; i < CTW; ++i) {
      const int ti = wm * CTW + i;
      const int co = co0 + OGE * (4 * (ti / OTPG) + (r16 >> 2)) + 4 * (ti % OTPG) + (r16 & 3);
      aoff[i] = co < a.Co ? (uint32_t)(co * a.Ci * ELT + g * 16) : kOob;
    }
    int a_c = 0;  // item of the next A operands to load
    auto load_a = [&](u32x4 (&dst)[KC][CTW], bool valid) {
#pragma unroll
      for (int s = 0; s < KC; ++s) {
        const uint32_t k0 = valid ? (uint32_t)((a_c * KC + s) * CB * ELT) : kOobS;
#pragma unroll
        for (int i = 0; i < CTW; ++i) dst[s][i] = buf_load16s(rw, aoff[i], k0);
      }
      if (++a_c == nch) a_c = 0;
    };
    // epilogue of a finished tile, straight from the accumulators
    const Epi3 ep_pw = make_epi3(a.act[1], a.rq[1]);
    const int cl0 = co0 + OGE * (4 * wm * NGW + g);  // this lane's first output channel
    int eyx[NB];
    uint32_t eoff[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int p = b * 16 + r16;
      const int py = p / TW, px = p - py * TW;
      eyx[b] = p < P ? (py << 16) | px : -1;
      eoff[b] = (uint32_t)(((py * a.Wo + px) * a.Co + cl0) * ELT);
    }
    f32x4 acc[NB][CTW];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int i = 0; i < CTW; ++i) acc[b][i] = f32x4{0, 0, 0, 0};
    int m_c = 0;   // chunk of the item whose MFMAs run next
    Tile mt = t0;  // its tile
    auto epilogue = [&]() {
      const int oy0 = mt.ty * TH, ox0 = mt.tx * TW;
      const char* tbase = (const char*)a.y + (size_t)((mt.n * a.Ho + oy0) * a.Wo + ox0) * a.Co * ELT;
      const rsrc_t ry = make_rsrc(tbase, 0x7fffffffu);
      const int rows = a.Ho - oy0, cols = a.Wo - ox0;
      const char* bl = smem + lay.pwb_off;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int v = eyx[b];
        const bool pok = v >= 0 && (v >> 16) < rows && (v & 0xffff) < cols;
#pragma unroll
        for (int k = 0; k < NGW; ++k) {
          const bool ok = pok && cl0 + 4 * OGE * k < a.Co;
          float bias[OGE];
#pragma unroll
          for (int q = 0; q < OGE / 4; ++q) {
            const u32x4 bq = *(const u32x4*)(bl + (OGE * (4 * (wm * NGW + k) + g) + 4 * q) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) bias[4 * q + e] = __uint_as_float(bq[e]);
          }
          u32x4 wd;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int tt = w >> 1, e = 2 * (w & 1);
            wd[w] = pack_bf16x2(epi_f(acc[b][2 * k + tt][e] + bias[4 * tt + e], ep_pw),
                                epi_f(acc[b][2 * k + tt][e + 1] + bias[4 * tt + e + 1], ep_pw));
          }
          buf_store_nt16(wd, ry, ok ? eoff[b] + 64 * k : kOob);
        }
      }
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int i = 0; i < CTW; ++i) acc[b][i] = f32x4{0, 0, 0, 0};
    };

    if (wm == 0) {  // the PW bias block
      const rsrc_t rbp = make_rsrc(a.b2 ? a.b2 : a.w2, a.b2 ? (uint32_t)(a.Co * 4) : 0u);
#pragma unroll
      for (int j = 0; j < (COB * 4 + 1023) / 1024; ++j)
        if (j * 1024 + lane * 16 < COB * 4)
          dma16(rbp, smem + lay.pwb_off + j * 1024, (uint32_t)(co0 * 4 + j * 1024 + lane * 16));
    }
    constexpr int NA = KC * CTW;  // A loads per item
    u32x4 am[3][KC][CTW];
    load_a(am[0], true);
    load_a(am[1], 1 < nit);
    barrier3();
    wait_vm_n<NA>();  // A operands of item 0 (and the bias block)
    barrier3();
    run_items([&](auto setc, int it) {
      constexpr int SET = decltype(setc)::value;
      constexpr int S2 = (SET + 2) % 3;
      const char* ex = smem + lay.exch_off + (it & 1) * lay.exch_bytes + g * lay.exch_plane + r16 * 16;
      u32x4 bop[KC][NB];
#pragma unroll
      for (int s = 0; s < KC; ++s)
#pragma unroll
        for (int b = 0; b < NB; ++b) bop[s][b] = *(const u32x4*)(ex + s * ND * lay.exch_plane + b * 256);
      load_a(am[S2], it + 2 < nit);
#pragma unroll
      for (int s = 0; s < KC; ++s)
#pragma unroll
        for (int i = 0; i < CTW; ++i)
#pragma unroll
          for (int b = 0; b < NB; ++b) mma16(TBF16{}, acc[b][i], am[SET][s][i], bop[s][b]);
      bool stored = false;
      if (++m_c == nch) {
        epilogue();
        stored = true;
        m_c = 0;
        advance(mt);
      }
      // A operands of item it + 1 are in: everything but this body's loads and stores
      if (stored) wait_vm_n<NA + NST>();
      else wait_vm_n<NA>();
      wait_lgkm0();
      barrier3();
    });
  }
}

template <int S, int TH, int TW, int CTW, int KC>
int launch_deep7(const KArgs& a, int grid, void* stream) {
  auto fn = k_deep7<S, TH, TW, CTW, KC>;
  const int lds = a.L.bytes;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return (int)e;
  }
  static thread_local int cached_lds = -1, cached_occ = 1;
  if (cached_lds != lds) {
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)fn, kThreads7, lds) != hipSuccess || occ < 1)
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
  return launch_args((const void*)fn, g, kThreads7, lds, stream, a);
}

}  // namespace fcm
