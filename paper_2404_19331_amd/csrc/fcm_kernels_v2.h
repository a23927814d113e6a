// fcm_kernels_v2.h -- NHWC kernels with compile-time tiles, LDS-DMA double buffering and
// the depthwise result produced directly in the MFMA operand registers (gfx950).
//
// k_dwpw2<DT, K, S, TH, TW, CO_MAX, HAS_DW>
//   DW -> PW module (and, with HAS_DW = false, the layer-by-layer PW kernel).
//   Workgroup = (image, TH x TW output tile, block of up to CO_MAX output channels); 4
//   waves, each owning P/64 blocks of 16 output pixels.
//   The input channels stream through LDS in chunks of one MFMA k-step (64 bytes of
//   channels per pixel). Each chunk's haloed input window and pointwise-weight block are
//   copied global -> LDS with buffer_load ... lds (16 bytes per lane, out-of-range
//   offsets read as zero, which is the convolution's zero padding), double-buffered so
//   that the copy of chunk c+1 overlaps the arithmetic of chunk c.
//   Lane l computes the depthwise stencil for pixel (l % 16) of its block and the 16
//   bytes of channels (l / 16) of the chunk: exactly the MFMA B operand that lane
//   supplies, so the depthwise output goes from the VALU into the matrix cores without
//   an LDS round trip (the paper's communication buffer, Sec. III-B, lives in registers
//   here). Pointwise accumulators stay in registers across chunks; the final output is
//   written once through an LDS transpose with 16-byte stores.
//
// k_dw2<DT, K, S, TH, TW>
//   Layer-by-layer depthwise kernel with the same staging and per-lane stencil; each
//   lane writes its 16 bytes of output channels straight to HBM.
//
// LDS row layout: a pixel (or weight row) holds 64 bytes = four 16-byte slots; logical
// slot j of row r is stored at slot j ^ (r & 3), which keeps the 16 lanes that read one
// MFMA column (16 consecutive rows, same logical slot) on distinct banks.
#pragma once

#include "fcm_kernels.h"

namespace fcm {

typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr uint32_t kOob = 0x80000000u;  // buffer offset beyond any record: reads as zero
constexpr int kSwz = kRowB / 16 - 1;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from (rsrc + voff) to LDS (wave_base + 16 * lane).
__device__ __forceinline__ void dma16(rsrc_t r, char* wave_base, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)wave_base, 16, voff, 0, 0,
                                           0);
}

__device__ __forceinline__ int swz(int row, int slot) { return slot ^ (row & kSwz); }

template <int TH, int TW, int K, int S>
struct TileGeom {
  static constexpr int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K;
  static constexpr int NPIN = IH * IW;
  static constexpr int P = TH * TW;
  static constexpr int PIX_PER_KB = 1024 / kRowB;
  static constexpr int IN_INSTR = (NPIN + PIX_PER_KB - 1) / PIX_PER_KB;
  static constexpr int IN_BYTES = IN_INSTR * 1024;
};

// Issue the DMA of one chunk's haloed input window: pixel q of the window, logical slot
// j -> image pixel (iy0 + q / IW, ix0 + q % IW), channels c0 + j * CPL .. + CPL.
template <class DT, class G>
__device__ __forceinline__ void dma_input(rsrc_t rx, char* dst, int wave, int lane, int iy0, int ix0, int H, int W,
                                          int C, int c0) {
  constexpr int CPL = 16 / DT::ELT;
#pragma unroll
  for (int i = 0; i < (G::IN_INSTR + 3) / 4; ++i) {
    const int ins = i * 4 + wave;
    if (ins < G::IN_INSTR) {
      const int byte = ins * 1024 + lane * 16;
      const int q = byte / kRowB, slot = (byte % kRowB) / 16;
      const int j = swz(q, slot);
      const int qy = q / G::IW, qx = q % G::IW;
      const int gy = iy0 + qy, gx = ix0 + qx, c = c0 + j * CPL;
      const bool ok = q < G::NPIN && (unsigned)gy < (unsigned)H && (unsigned)gx < (unsigned)W && c < C;
      dma16(rx, dst + ins * 1024, ok ? (uint32_t)(((gy * W + gx) * C + c) * DT::ELT) : kOob);
    }
  }
}

// Issue the DMA of pointwise-weight rows co0 .. co0 + 16 * m_tiles, columns c0 .. c0+CB.
template <class DT, int CO_MAX>
__device__ __forceinline__ void dma_weights(rsrc_t rw, char* dst, int wave, int lane, int m_tiles, int Co, int C,
                                            int co0, int c0) {
  constexpr int CPL = 16 / DT::ELT;
#pragma unroll
  for (int i = 0; i < (CO_MAX / 16 + 3) / 4; ++i) {
    const int ins = i * 4 + wave;  // one 1 KB instruction = 16 rows = one MFMA m-tile
    if (ins < m_tiles) {
      const int byte = ins * 1024 + lane * 16;
      const int r = byte / kRowB, slot = (byte % kRowB) / 16;
      const int j = swz(r, slot);
      const int co = co0 + r, c = c0 + j * CPL;
      const bool ok = co < Co && c < C;
      dma16(rw, dst + ins * 1024, ok ? (uint32_t)((co * C + c) * DT::ELT) : kOob);
    }
  }
}

// Depthwise weights + bias of one chunk (CB channels) as accumulator-type values,
// [K*K taps][CB] then [CB] bias, fetched into registers first (NDW items per thread).
template <class DT, int K, int CB>
struct DwChunk {
  static constexpr int ITEMS = (K * K + 1) * CB;
  static constexpr int NDW = (ITEMS + kThreads - 1) / kThreads;
  typename DwWeights<DT, K>::V v[NDW];
  int d[NDW];
  __device__ __forceinline__ void load(const DwWeights<DT, K>& L) {
#pragma unroll
    for (int j = 0; j < NDW; ++j) {
      const int i = threadIdx.x + j * kThreads;
      d[j] = L.load(min(i, ITEMS - 1), v[j]);
      if (i >= ITEMS) d[j] = -1;
    }
  }
  __device__ __forceinline__ void store(const DwWeights<DT, K>& L, char* s) const {
#pragma unroll
    for (int j = 0; j < NDW; ++j)
      if (d[j] >= 0) L.store(s, d[j], v[j]);
  }
};

// Unpack lane element e (of CPL) of a 16-byte slot to the accumulator type.
template <class DT>
__device__ __forceinline__ typename DT::Acc unpack(const u32x4& v, int e) {
  if constexpr (DT::ELT == 4) {
    return __uint_as_float(v[e]);
  } else if constexpr (DT::ELT == 2) {
    const uint32_t w = v[e >> 1];
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  } else {
    return (int32_t)(int8_t)((v[e >> 2] >> ((e & 3) * 8)) & 0xffu);
  }
}

// Pack CPL finished values (storage bits) into one 16-byte operand slot.
template <class DT>
__device__ __forceinline__ u32x4 pack16(const uint32_t (&o)[16 / DT::ELT]) {
  u32x4 r;
  if constexpr (DT::ELT == 4) {
    r = u32x4{o[0], o[1], o[2], o[3]};
  } else if constexpr (DT::ELT == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = o[2 * i] | (o[2 * i + 1] << 16);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = o[4 * i] | (o[4 * i + 1] << 8) | (o[4 * i + 2] << 16) | (o[4 * i + 3] << 24);
  }
  return r;
}

// Depthwise stencil of BPW pixels (one per block) x CPL channels (logical slot g of the
// chunk) from the staged window; returns finished storage values packed per block.
template <class DT, int K, int S, int TW, int BPW, int CB>
__device__ __forceinline__ void dw_lane(const char* in, const typename DT::Acc* wd, const int (&py)[BPW],
                                        const int (&px)[BPW], int g, int act, const Requant& rq,
                                        u32x4 (&out)[BPW]) {
  using Acc = typename DT::Acc;
  constexpr int CPL = 16 / DT::ELT;
  constexpr int IW = (TW - 1) * S + K;
  Acc acc[BPW][CPL];
#pragma unroll
  for (int b = 0; b < BPW; ++b)
#pragma unroll
    for (int e = 0; e < CPL; ++e) acc[b][e] = Acc(0);
  // one kernel row per iteration (not unrolled) bounds the live registers
#pragma unroll 1
  for (int ky = 0; ky < K; ++ky) {
#pragma unroll
    for (int kx = 0; kx < K; ++kx) {
      const Acc* wt = wd + (ky * K + kx) * CB + g * CPL;
      Acc w[CPL];
#pragma unroll
      for (int e = 0; e < CPL; ++e) w[e] = wt[e];
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int q = (py[b] * S + ky) * IW + px[b] * S + kx;
        const u32x4 v = *(const u32x4*)(in + q * kRowB + swz(q, g) * 16);
#pragma unroll
        for (int e = 0; e < CPL; ++e) acc[b][e] += w[e] * unpack<DT>(v, e);
      }
    }
  }
  const Acc* bias = wd + K * K * CB + g * CPL;
#pragma unroll
  for (int b = 0; b < BPW; ++b) {
    uint32_t o[CPL];
#pragma unroll
    for (int e = 0; e < CPL; ++e) o[e] = Fin<DT>::apply(acc[b][e], bias[e], act, rq);
    out[b] = pack16<DT>(o);
  }
}

template <class DT, int K, int S, int TH, int TW, int CO_MAX, bool HAS_DW>
__global__ __launch_bounds__(kThreads) void k_dwpw2(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  constexpr int KE = HAS_DW ? K : 1, SE = HAS_DW ? S : 1;
  using G = TileGeom<TH, TW, KE, SE>;
  constexpr int CB = kRowB / DT::ELT;  // channels per chunk = one MFMA k-step
  constexpr int NB = G::P / 16, BPW = NB / 4;
  constexpr int CT = CO_MAX / 16;
  constexpr int W_BYTES = CO_MAX * kRowB;
  constexpr int WD_BYTES = HAS_DW ? ((KE * KE + 1) * CB * 4 + 15) / 16 * 16 : 0;
  constexpr int BUF = G::IN_BYTES + W_BYTES + WD_BYTES;
  static_assert(NB % 4 == 0, "tile must hold a multiple of 64 pixels");

  const int G_ = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  const int lid = xcd_remap(blockIdx.x, G_);
  const int cob = lid % a.n_cb;
  int t = lid / a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;
  const int oy0 = ty * TH, ox0 = tx * TW;
  const int iy0 = HAS_DW ? oy0 * S - a.pad : oy0, ix0 = HAS_DW ? ox0 * S - a.pad : ox0;
  const int co0 = cob * a.COB, cob_eff = min(a.COB, a.Co - co0);
  const int m_tiles = ceil_div(cob_eff, 16);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  int py[BPW], px[BPW];
#pragma unroll
  for (int b = 0; b < BPW; ++b) {
    const int p = (wave * BPW + b) * 16 + r16;
    py[b] = p / TW;
    px[b] = p % TW;
  }

  const T* x = (const T*)a.x;
  const size_t img = (size_t)a.H * a.W * a.Ci;
  const rsrc_t rx = make_rsrc(x + (size_t)n * img, (uint32_t)(img * DT::ELT));
  const T* wp = (const T*)(HAS_DW ? a.w2 : a.w1);
  const rsrc_t rw = make_rsrc(wp, (uint32_t)((size_t)a.Co * a.Ci * DT::ELT));
  const void* bp = HAS_DW ? a.b2 : a.b1;
  const int act_pw = HAS_DW ? a.act[1] : a.act[0];
  const Requant rq_pw = HAS_DW ? a.rq[1] : a.rq[0];
  const int nchunks = ceil_div(a.Ci, CB);

  AccV acc[BPW][CT];
#pragma unroll
  for (int b = 0; b < BPW; ++b)
#pragma unroll
    for (int i = 0; i < CT; ++i) acc[b][i] = AccV{0, 0, 0, 0};

  // prologue: chunk 0 -> buffer 0
  {
    char* buf = smem;
    dma_input<DT, G>(rx, buf, wave, lane, iy0, ix0, a.H, a.W, a.Ci, 0);
    dma_weights<DT, CO_MAX>(rw, buf + G::IN_BYTES, wave, lane, m_tiles, a.Co, a.Ci, co0, 0);
    if constexpr (HAS_DW) {
      const DwWeights<DT, KE> L{(const T*)a.w1, a.b1, a.Ci, 0, CB, G::IN_BYTES + W_BYTES};
      DwChunk<DT, KE, CB> dwc;
      dwc.load(L);
      dwc.store(L, buf);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  for (int ch = 0; ch < nchunks; ++ch) {
    const int cur = ch & 1;
    char* buf = smem + cur * BUF;
    char* nxt = smem + (cur ^ 1) * BUF;
    const bool more = ch + 1 < nchunks;
    [[maybe_unused]] DwChunk<DT, KE, CB> dwc;
    [[maybe_unused]] const DwWeights<DT, KE> Ln{(const T*)a.w1, a.b1, a.Ci, (ch + 1) * CB, CB, G::IN_BYTES + W_BYTES};
    if (more) {
      dma_input<DT, G>(rx, nxt, wave, lane, iy0, ix0, a.H, a.W, a.Ci, (ch + 1) * CB);
      dma_weights<DT, CO_MAX>(rw, nxt + G::IN_BYTES, wave, lane, m_tiles, a.Co, a.Ci, co0, (ch + 1) * CB);
      if constexpr (HAS_DW) dwc.load(Ln);
    }
    // B operand: depthwise output (or the input itself) for this lane's pixel and slot
    u32x4 bop[BPW];
    if constexpr (HAS_DW) {
      dw_lane<DT, K, S, TW, BPW, CB>(buf, (const Acc*)(buf + G::IN_BYTES + W_BYTES), py, px, g, a.act[0], a.rq[0],
                                     bop);
    } else {
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int q = py[b] * TW + px[b];
        bop[b] = *(const u32x4*)(buf + q * kRowB + swz(q, g) * 16);
      }
    }
    const char* wl = buf + G::IN_BYTES;
#pragma unroll
    for (int i = 0; i < CT; ++i) {
      if (i < m_tiles) {
        const int row = i * 16 + r16;
        const u32x4 av = *(const u32x4*)(wl + row * kRowB + swz(row, g) * 16);
#pragma unroll
        for (int b = 0; b < BPW; ++b) mma16(DT{}, acc[b][i], av, bop[b]);
      }
    }
    if constexpr (HAS_DW) {
      if (more) dwc.store(Ln, nxt);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // epilogue: accumulators -> LDS [P][COB] (pixel-major) -> 16-byte coalesced stores
  const int rs_out = a.COB * DT::ELT + 16;
#pragma unroll
  for (int i = 0; i < CT; ++i) {
    if (i < m_tiles) {
      const int m = i * 16 + 4 * g;
      Acc bias[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        bias[v] = load_bias<DT>(bp, co0 + min(m + v, cob_eff - 1));
        if (m + v >= cob_eff) bias[v] = Acc(0);
      }
#pragma unroll
      for (int b = 0; b < BPW; ++b) {
        const int p = (wave * BPW + b) * 16 + r16;
        uint32_t o[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = Fin<DT>::apply(acc[b][i][v], bias[v], act_pw, rq_pw);
        lds_store4<DT>(smem + p * rs_out + m * DT::ELT, o[0], o[1], o[2], o[3]);
      }
    }
  }
  __syncthreads();
  store_tile<DT>(smem, rs_out, (T*)a.y, LAYOUT_NHWC, n, a.Co, a.Ho, a.Wo, oy0, ox0, TH, TW, co0, cob_eff,
                 (cob_eff * DT::ELT) % 16 == 0);
}

// Layer-by-layer depthwise: workgroup = (image, tile, chunk of CB channels).
template <class DT, int K, int S, int TH, int TW>
__global__ __launch_bounds__(kThreads) void k_dw2(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using G = TileGeom<TH, TW, K, S>;
  constexpr int CB = kRowB / DT::ELT;
  constexpr int CPL = 16 / DT::ELT;
  constexpr int NB = G::P / 16, BPW = NB / 4;
  static_assert(NB % 4 == 0, "tile must hold a multiple of 64 pixels");

  const int G_ = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  const int lid = xcd_remap(blockIdx.x, G_);
  const int cb = lid % a.n_cb;
  int t = lid / a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;
  const int oy0 = ty * TH, ox0 = tx * TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const int c0 = cb * CB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;

  const T* x = (const T*)a.x;
  const size_t img = (size_t)a.H * a.W * a.Cm;
  const rsrc_t rx = make_rsrc(x + (size_t)n * img, (uint32_t)(img * DT::ELT));
  dma_input<DT, G>(rx, smem, wave, lane, iy0, ix0, a.H, a.W, a.Cm, c0);
  const DwWeights<DT, K> L{(const T*)a.w1, a.b1, a.Cm, c0, CB, G::IN_BYTES};
  DwChunk<DT, K, CB> dwc;
  dwc.load(L);
  dwc.store(L, smem);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  int py[BPW], px[BPW];
#pragma unroll
  for (int b = 0; b < BPW; ++b) {
    const int p = (wave * BPW + b) * 16 + r16;
    py[b] = p / TW;
    px[b] = p % TW;
  }
  u32x4 outv[BPW];
  dw_lane<DT, K, S, TW, BPW, CB>(smem, (const Acc*)(smem + G::IN_BYTES), py, px, g, a.act[0], a.rq[0], outv);
  const int c = c0 + g * CPL;
#pragma unroll
  for (int b = 0; b < BPW; ++b) {
    const int oy = oy0 + py[b], ox = ox0 + px[b];
    if (oy < a.Ho && ox < a.Wo && c < a.Cm)
      *(u32x4*)((T*)a.y + (((size_t)n * a.Ho + oy) * a.Wo + ox) * a.Cm + c) = outv[b];
  }
}

template <class DT, int K, int S, int TH, int TW, int CO_MAX, bool HAS_DW>
int launch_dwpw2(const KArgs& a, int grid, void* stream) {
  return launch_kernel(k_dwpw2<DT, K, S, TH, TW, CO_MAX, HAS_DW>, a, grid, stream);
}

template <class DT, int K, int S, int TH, int TW>
int launch_dw2(const KArgs& a, int grid, void* stream) {
  return launch_kernel(k_dw2<DT, K, S, TH, TW>, a, grid, stream);
}

}  // namespace fcm
