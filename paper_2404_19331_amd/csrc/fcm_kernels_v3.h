// fcm_kernels_v3.h -- persistent NHWC kernels for gfx950: DW->PW module, and the
// layer-by-layer PW and DW kernels built from the same pieces.
//
// k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS>
//   A persistent workgroup (two copy waves, four compute waves) owns a contiguous range
//   of work tiles; a work tile is (image, TH x TW output tile, block of 16*CT output
//   channels). Work tiles are cut into items of KS input-channel chunks of 64 bytes (one
//   MFMA k-step each); the items of the whole range form one stream, and the copies of
//   items i+1 .. i+depth-1 (global -> LDS with buffer_load ... lds, out-of-range offsets
//   read as zero, i.e. the zero padding of the convolution) overlap the arithmetic of
//   item i, across tile boundaries as well.
//
//   Lane l of compute wave w owns, in each of its BPW pixel blocks, output pixel (l % 16) of the
//   block and the 16 bytes of channels (l / 16) of the chunk: exactly the MFMA B operand
//   the lane supplies. The depthwise stencil is computed straight into that operand, so
//   the DW output never leaves the registers (the paper's on-chip communication buffer,
//   Sec. III-B). Its multiply-adds use the packed dot instructions with one half of the
//   weight operand zero (bf16: v_dot2c_f32_bf16, int8: v_dot4c_i32_i8), so no unpacking
//   of the packed input is needed.
//
//   The pointwise weights rows are staged in a permuted order such that accumulator lane
//   (l % 16, l / 16) holds whole 16-byte granules of output channels of its pixel, and the
//   four lane groups hold adjacent granules: the epilogue (+bias, activation, cast)
//   writes 64 contiguous bytes per pixel with each 16-byte store instruction, straight
//   from registers, and the output is written once (output-stationary, Sec. III-A OS-LWS).
//
//   MODE M3_PW: the DW stage is off (window = output tile); M3_DW: the PW stage is off,
//   each lane writes its 16 bytes of depthwise output directly.
//
//   QX (int8 only): 1 adds zero points, 2 zero points and per-channel requantisation
//   (multipliers and shifts staged with the biases). Each is a separate instance,
//   launched only for descriptors that have the feature, so that the symmetric kernel
//   keeps its registers. Split plans too: the pointwise zero-point term is linear, so
//   each split subtracts its own channel range's share before writing its partial sums,
//   and the second kernel requantises.
//
// LDS: a ring of a.depth buffers (the copy waves run a.depth - 1 items ahead of the
// compute waves; deeper rings keep more bytes in flight per CU). Per buffer: window [npin pixels][64 B] (pixel q at 64 q, no padding;
// stride-2 windows keep even and odd columns in separate halves so that the lanes of a
// block read consecutive pixels), PW weights [16*CT rows][64 B] (16-byte slots XOR-
// swizzled by row bit 3, conflict-free MFMA A reads), DW weights [K*K taps][CB] 32-bit
// values in dot-operand form + bias [CB].
#pragma once

#include "fcm_kernels.h"

namespace fcm {


constexpr int kNiwMax = 10;  // window copy instructions per wave (<= 640 window pixels)

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Branch-free epilogue of a convolution stage. Float paths: activation as a clamp to
// [lo, hi] (NONE: unbounded, RELU: [0, inf), RELU6: [0, 6]). Int8: requantisation
// (round half to even of acc * mult / 2^shift), plus the output zero point zp, and a clamp
// to [qlo, qhi]: the saturation range with ReLU at real 0 (code zp) folded in,
// max(clamp(q, a, b), zp) = clamp(q, max(a, zp), max(b, zp)).
struct Epi3 {
  float lo, hi;
  int32_t mult, shift, qlo, qhi, zp;
};
__device__ __forceinline__ Epi3 make_epi3(int act, const Requant& rq) {
  Epi3 e;
  e.lo = act == ACT_NONE ? -__builtin_huge_valf() : 0.0f;
  e.hi = act == ACT_RELU6 ? 6.0f : __builtin_huge_valf();
  e.mult = rq.mult;
  e.shift = rq.shift;
  e.zp = rq.zp;
  e.qlo = act != ACT_NONE ? max(rq.qmin, rq.zp) : rq.qmin;  // int8 ReLU6: its 6 is qmax
  e.qhi = act != ACT_NONE ? max(rq.qmax, rq.zp) : rq.qmax;
  return e;
}
__device__ __forceinline__ float epi_f(float v, const Epi3& e) { return __builtin_amdgcn_fmed3f(v, e.lo, e.hi); }
// (the multiplier and shift of the value's channel: the stage's, or per-channel ones)
__device__ __forceinline__ int32_t epi_q(int32_t acc, int32_t mult, int32_t shift, const Epi3& e) {
  const int64_t t = (int64_t)acc * mult;
  const int64_t half = ((int64_t)1 << shift) >> 1;
  const int64_t rnd = shift > 0 ? half - 1 + ((t >> shift) & 1) : 0;
  int64_t q = ((t + rnd) >> shift) + e.zp;
  q = q < e.qlo ? e.qlo : q;
  q = q > e.qhi ? e.qhi : q;
  return (int32_t)q;
}
__device__ __forceinline__ int32_t epi_i(int32_t acc, const Epi3& e) { return epi_q(acc, e.mult, e.shift, e); }
// A per-channel shift as the first-generation kernels take it: clamped to [0, 62].
__device__ __forceinline__ int32_t pc_shift(uint32_t s) { return min(max((int32_t)s, 0), 62); }
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Depthwise arithmetic on one 16-byte lane slot of channels.
template <class DT>
struct Dw3;

template <>
struct Dw3<TF32> {
  static constexpr int CPL = 4;  // channels per 16-byte slot
  static constexpr int WQ = 1;   // 16-byte weight reads per tap and lane
  __device__ static __forceinline__ uint32_t weight_word(uint32_t raw, int) { return raw; }
  __device__ static __forceinline__ void tap(float (&acc)[4], const u32x4& x, const u32x4 (&w)[1]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(__uint_as_float(x[e]), __uint_as_float(w[0][e]), acc[e]);
  }
  __device__ static __forceinline__ u32x4 finish(const float (&acc)[4], const Epi3& ep) {
    u32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = __float_as_uint(epi_f(acc[e], ep));
    return r;
  }
};

template <>
struct Dw3<TBF16> {
  static constexpr int CPL = 8;
  static constexpr int WQ = 2;
  // dot operand for channel c: the weight in the half that multiplies channel c's half of
  // the packed input pair, zero in the other half
  __device__ static __forceinline__ uint32_t weight_word(uint32_t raw, int c) {
    return (c & 1) ? (raw << 16) : (raw & 0xffffu);
  }
  __device__ static __forceinline__ void tap(float (&acc)[8], const u32x4& x, const u32x4 (&w)[2]) {
    // (vector elements are copied to scalars before __builtin_bit_cast: applied to a vector
    // element expression directly, the cast reads element 0)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t xs = x[e >> 1], ws = w[e >> 2][e & 3];
      acc[e] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, xs), __builtin_bit_cast(bf16x2_t, ws),
                                               acc[e], false);
    }
  }
  __device__ static __forceinline__ u32x4 finish(const float (&acc)[8], const Epi3& ep) {
    u32x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = pack_bf16x2(epi_f(acc[2 * j], ep), epi_f(acc[2 * j + 1], ep));
    return r;
  }
};

template <>
struct Dw3<TI8> {
  static constexpr int CPL = 16;
  static constexpr int WQ = 4;
  __device__ static __forceinline__ uint32_t weight_word(uint32_t raw, int c) { return (raw & 0xffu) << (8 * (c & 3)); }
  __device__ static __forceinline__ void tap(int32_t (&acc)[16], const u32x4& x, const u32x4 (&w)[4]) {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      acc[e] = __builtin_amdgcn_sdot4((int)x[e >> 2], (int)w[e >> 2][e & 3], acc[e], false);
  }
  __device__ static __forceinline__ u32x4 finish(const int32_t (&acc)[16], const Epi3& ep) {
    u32x4 r;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t wv = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) wv |= ((uint32_t)epi_i(acc[4 * j + b], ep) & 0xffu) << (8 * b);
      r[j] = wv;
    }
    return r;
  }
};

// s_waitcnt vmcnt(n) with the other counters left alone, for a run-time n in [0, 63]:
// gfx9 encoding vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14.
template <int N>
__device__ __forceinline__ void wait_vm_n() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}
// s_waitcnt lgkmcnt(0) only (LDS operations of this wave are complete).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14)); }
// Workgroup barrier without the memory fences of __syncthreads: a release fence would
// make a copy wave wait for all of its outstanding copies (they are LDS writes). The
// waits each side needs are explicit; the empty asm statements keep the compiler from
// moving memory accesses across the barrier.
__device__ __forceinline__ void barrier3() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_vm(int n) {
  switch (n) {
#define FCM_W4(b) \
  case b: wait_vm_n<b>(); break; \
  case b + 1: wait_vm_n<b + 1>(); break; \
  case b + 2: wait_vm_n<b + 2>(); break; \
  case b + 3: wait_vm_n<b + 3>(); break;
    FCM_W4(0) FCM_W4(4) FCM_W4(8) FCM_W4(12) FCM_W4(16) FCM_W4(20) FCM_W4(24) FCM_W4(28)
    FCM_W4(32) FCM_W4(36) FCM_W4(40) FCM_W4(44) FCM_W4(48) FCM_W4(52) FCM_W4(56) FCM_W4(60)
#undef FCM_W4
    default: wait_vm_n<0>(); break;
  }
}

template <class DT, int K, int S, int BPW, int CT, int MODE, int IWP, int KS, bool SPLIT, int QX>
__global__ __launch_bounds__(kThreads3) void k_fused3(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  using D3 = Dw3<DT>;
  constexpr bool HAS_DW = MODE != M3_PW;
  constexpr bool HAS_PW = MODE != M3_DW;
  constexpr int KE = HAS_DW ? K : 1, SE = HAS_DW ? S : 1;
  constexpr int KK = KE * KE;
  constexpr int CB = kRowB / DT::ELT;  // channels per chunk
  constexpr int CPL = D3::CPL;
  constexpr int WQ = D3::WQ;
  constexpr int IPR = IWP / 16;  // copy instructions per window row
  constexpr int NRAW = (64 * K * K + 1023) / 1024;
  static_assert(CPL * 4 == CB, "lane slot layout");
  static_assert(IWP % 16 == 0, "window pitch");
  static_assert(MODE != M3_DW || KS == 1, "a depthwise-only item is one chunk");
  static_assert(QX == 0 || std::is_same<DT, TI8>::value, "zero points / per-channel: int8");
  constexpr int PCQ = QX == 2 ? 1 : 0;  // per-channel multipliers and shifts staged
  // Output-channel order of the PW accumulators: lane (l % 16, g = l / 16) of tile i holds
  // values v = 0..3 of channel OGE * (4 * (i / OTPG) + g) + 4 * (i % OTPG) + v, so that the
  // OTPG tiles of each 16-byte output granule sit in one lane and the four lane groups
  // write 64 contiguous bytes of a pixel with each store instruction.
  constexpr int OGE = 16 / DT::ELT;  // channels per 16-byte granule
  constexpr int OTPG = OGE / 4;      // MFMA tiles per granule
  static_assert(MODE == M3_DW || CT % OTPG == 0, "whole output granules per lane");
  static_assert(MODE == M3_DW || CT <= 16, "the block's PW bias (16*CT fp32 / int32) is one 1 KiB copy");

  const int TH = a.TH, TW = a.TW, P = TH * TW;
  const int IW = HAS_DW ? (TW - 1) * SE + KE : TW;
  const int IH = HAS_DW ? (TH - 1) * SE + KE : TH;
  const Lds3 lay = lds3p(dtype_id<DT>(), KE, MODE, IH, IWP, CT, 2, KS, PCQ);
  if constexpr (PCQ) {
    if ((a.depth < 2 ? 2 : a.depth) * lay.buf_bytes > a.L.bytes) return;  // (a plan for another layout)
  }
  const int C = MODE == M3_DW ? a.Cm : a.Ci;
  const int nchunks = MODE == M3_DW ? 1 : ceil_div(C, CB * KS);  // items per work tile
  const int per_item = copies_per_item3(MODE, KE, IH, IWP, CT, KS, PCQ);
  // Work units: split u % SPL of work tile u / SPL runs items [u_lo(u), u_hi(u)).
  // (a separate instance: the partial-sum epilogue in the same loop costs the unsplit
  // kernel its schedule)
  const int SPL = SPLIT ? a.splits : 1;
  const int ips = items_per_split3(nchunks, SPL);
  auto u_lo = [&](int u) { return (u % SPL) * ips; };
  auto u_hi = [&](int u) { return min(nchunks, (u % SPL) * ips + ips); };

  // ---- work range of this workgroup (consecutive logical ids share an XCD) ----
  const int G = gridDim.x;
  const int L = xcd_remap(blockIdx.x, G);
  const int wt0 = (int)((int64_t)a.nwork * L / G), wt1 = (int)((int64_t)a.nwork * (L + 1) / G);
  if (wt1 <= wt0) return;
  int nitems = 0;
  for (int u = wt0; u < wt1; ++u) nitems += u_hi(u) - u_lo(u);

  // waves 0..kCopyWaves3-1 copy, the next four compute; the wave index is uniform:
  // keep it scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, g = lane >> 4;
  const bool producer = wave < kCopyWaves3;
  const int cw = wave - kCopyWaves3;  // compute-wave index

  const T* x = (const T*)a.x;
  const size_t img = (size_t)a.H * a.W * C;
  const T* wp = (const T*)(MODE == M3_PW ? a.w1 : a.w2);
  const T* wd = (const T*)a.w1;
  const void* bd = a.b1;
  const void* bp = MODE == M3_PW ? a.b1 : a.b2;
  const int CoB = 16 * CT;

  struct Tile {
    int n, oy0, ox0, cb;  // cb: output-channel block (DW: channel chunk)
  };
  auto decode = [&](int wt) {
    Tile r;
    int t = wt;
    r.cb = t % a.n_cb;
    t /= a.n_cb;
    const int tx = t % a.tiles_x;
    t /= a.tiles_x;
    const int ty = t % a.tiles_y;
    r.n = t / a.tiles_y;
    r.oy0 = ty * TH;
    r.ox0 = tx * TW;
    return r;
  };
  const int D = a.depth < 2 ? 2 : a.depth;  // ring buffers
  auto bufp = [&](int slot) { return smem + slot * lay.buf_bytes; };
  auto next_slot = [&](int slot) { return slot + 1 == D ? 0 : slot + 1; };


  if (producer) {
    // ===== copy waves: all copies, D - 1 items ahead of the compute waves. Wave 0 issues
    // the DW weights and bias (and converts them) and window rows [0, r0); wave 1 the
    // rows [r0, IH), the PW weight rows and the PW bias. =====
    const int r0 = rows_wave0_3(MODE, KE, IH, IWP, CT, KS, PCQ);
    const int wy0 = wave == 0 ? 0 : r0, wy1 = wave == 0 ? r0 : IH;
    const int w0n = copies_wave0_3(MODE, KE, IH, IWP, CT, KS, PCQ);
    const int mine = wave == 0 ? w0n : per_item - w0n;  // copies per item of this wave
    const rsrc_t rw = make_rsrc(wp, HAS_PW ? (uint32_t)((size_t)a.Co * a.Ci * DT::ELT) : 0u);
    const rsrc_t rwd = make_rsrc(wd, HAS_DW ? (uint32_t)((size_t)C * KK * DT::ELT) : 0u);
    const rsrc_t rbd = make_rsrc(bd ? bd : (const void*)wd, (HAS_DW && bd) ? (uint32_t)(C * 4) : 0u);
    const rsrc_t rbp = make_rsrc(bp ? bp : (const void*)wp, (HAS_PW && bp) ? (uint32_t)(a.Co * 4) : 0u);
    // per-channel requantisation of each stage: [multipliers | shifts] of its channels
    const int32_t* qd = PCQ && HAS_DW ? a.rqc[0] : nullptr;
    const int32_t* qp = PCQ && HAS_PW ? a.rqc[MODE == M3_PW ? 0 : 1] : nullptr;
    const rsrc_t rqd = make_rsrc(qd ? (const void*)qd : (const void*)wd, qd ? (uint32_t)(2 * C * 4) : 0u);
    const rsrc_t rqp = make_rsrc(qp ? (const void*)qp : (const void*)wp, qp ? (uint32_t)(2 * a.Co * 4) : 0u);
    int wxl[IPR];
#pragma unroll
    for (int j = 0; j < IPR; ++j) {
      const int col = j * 16 + (lane >> 2);
      int wx = col;
      if (SE == 2) wx = col < IWP / 2 ? 2 * col : 2 * (col - IWP / 2) + 1;
      wxl[j] = wx < IW ? wx : -1;
    }
    int iss_slot = 0, iss_wt = wt0, iss_ch = u_lo(wt0), iss_hi = u_hi(wt0);
    Tile iss_t = decode(wt0 / SPL);
    // Asymmetric int8 input (zero point zin): the window positions outside the image must
    // hold zin (real 0), not the zeros the copies write there, and each depthwise sum loses
    // zin x its channel's weight sum (folded into the bias). Once an item's copies have
    // landed, each copy wave rewrites the out-of-image positions of its own rows, and
    // wave 0 the item's depthwise biases; a second item iterator follows the issue one.
    // (Every byte of a ring slot is a copy target, so no item data can ride along in it.)
    const int zin = (QX && HAS_DW) ? a.zin[0] : 0;
    int fx_slot = 0, fx_wt = wt0, fx_ch = u_lo(wt0), fx_hi = u_hi(wt0);
    Tile fx_t = iss_t;
    auto fix_next = [&]() {
      if (!QX || zin == 0) return;
      char* buf = bufp(fx_slot);
      const int iy0 = fx_t.oy0 * SE - a.pad, ix0 = fx_t.ox0 * SE - a.pad;
      fx_slot = next_slot(fx_slot);
      if (++fx_ch == fx_hi && ++fx_wt < wt1) {
        fx_ch = u_lo(fx_wt);
        fx_hi = u_hi(fx_wt);
        fx_t = decode(fx_wt / SPL);
      }
      if (iy0 < 0 || ix0 < 0 || iy0 + IH > a.H || ix0 + IW > a.W) {
        const uint32_t fill = zp_fill<DT>(zin);
        for (int wy = wy0; wy < wy1; ++wy) {
          const bool rok = (unsigned)(iy0 + wy) < (unsigned)a.H;
#pragma unroll
          for (int j = 0; j < IPR; ++j) {
            const int gx = ix0 + wxl[j];
            if (rok && wxl[j] >= 0 && (unsigned)gx < (unsigned)a.W) continue;
#pragma unroll
            for (int s = 0; s < KS; ++s)
              *(u32x4*)(buf + s * lay.plane_bytes + (wy * IPR + j) * 1024 + lane * 16) = u32x4{fill, fill, fill, fill};
          }
        }
      }
      if (wave == 0) {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int8_t* rb = (const int8_t*)(buf + s * lay.plane_bytes + lay.raw_off) + lane * KK;
          int32_t wsum = 0;
#pragma unroll
          for (int t = 0; t < KK; ++t) wsum += rb[t];
          int32_t* bb = (int32_t*)(buf + lay.bias_off) + s * CB + lane;
          *bb -= zin * wsum;
        }
      }
    };
    auto issue_next = [&]() {
      char* buf = bufp(iss_slot);
      const int c0 = MODE == M3_DW ? iss_t.cb * CB : iss_ch * (CB * KS);
      const int co0 = iss_t.cb * CoB;
      const int iy0 = HAS_DW ? iss_t.oy0 * SE - a.pad : iss_t.oy0;
      const int ix0 = HAS_DW ? iss_t.ox0 * SE - a.pad : iss_t.ox0;
      const rsrc_t rx = make_rsrc(x + (size_t)iss_t.n * img, (uint32_t)(img * DT::ELT));
      // Byte offsets: a per-lane part (window column, channel slot), fixed for the item,
      // plus a uniform part per window row. Lanes outside the image or the channel range
      // carry kOob, which stays out of range after the row offset (< 2^31) is added.
      uint32_t coff[KS][IPR];
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const int c = c0 + s * CB + (lane & 3) * CPL;
#pragma unroll
        for (int j = 0; j < IPR; ++j) {
          const int gx = ix0 + wxl[j];
          const bool ok = wxl[j] >= 0 && (unsigned)gx < (unsigned)a.W && c < C;
          coff[s][j] = ok ? (uint32_t)((gx * C + c) * DT::ELT) : kOob;
        }
      }
      const uint32_t rstride = (uint32_t)(a.W * C * DT::ELT);
      if (HAS_DW && wave == 0) {
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int r = 0; r < NRAW; ++r) {
            const int b = r * 1024 + lane * 16;
            dma16(rwd, buf + s * lay.plane_bytes + lay.raw_off + r * 1024,
                  b < CB * KK * DT::ELT ? (uint32_t)((c0 + s * CB) * KK * DT::ELT + b) : kOob);
          }
        dma16(rbd, buf + lay.bias_off, lane * 16 < KS * CB * 4 ? (uint32_t)(c0 * 4 + lane * 16) : kOob);
        if constexpr (PCQ) {  // lanes 0-31: multipliers of the item's channels, 32-63: their shifts
          const int j = lane & 31, ch = c0 + 4 * j;
          const bool ok = j * 16 < KS * CB * 4 && ch < C;
          dma16(rqd, buf + lay.bias_off + 2048, ok ? (uint32_t)(((lane < 32 ? 0 : C) + ch) * 4) : kOob);
        }
      }
      for (int wy = wy0; wy < wy1; ++wy) {
        const int gy = iy0 + wy;
        const bool rok = (unsigned)gy < (unsigned)a.H;
        const uint32_t roff = rok ? (uint32_t)gy * rstride : 0u;
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int j = 0; j < IPR; ++j)
            dma16(rx, buf + s * lay.plane_bytes + (wy * IPR + j) * 1024, rok ? coff[s][j] + roff : kOob);
      }
      if (HAS_PW && wave == 1) {
        const int mrow = lane >> 2;
        const int j = (lane & 3) ^ (((mrow >> 3) & 1) << 1);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const int cw_ = c0 + s * CB + j * CPL;
          // rows beyond c_out fall outside the weight tensor and read as zero
          const uint32_t woff =
              cw_ < a.Ci ? (uint32_t)(((co0 + OGE * (mrow >> 2) + (mrow & 3)) * a.Ci + cw_) * DT::ELT) : kOob;
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
            dma16(rw, buf + s * lay.plane_bytes + lay.in_bytes + ct * 1024,
                  woff + (uint32_t)((4 * OGE * (ct / OTPG) + 4 * (ct % OTPG)) * a.Ci * DT::ELT));
        }
        dma16(rbp, buf + lay.bias_off + 1024, lane * 16 < CoB * 4 ? (uint32_t)(co0 * 4 + lane * 16) : kOob);
        if constexpr (PCQ) {  // multipliers, then shifts, of the block's output channels
          const int ch = co0 + 4 * lane;
          const bool ok = lane * 16 < CoB * 4 && ch < a.Co;
          dma16(rqp, buf + lay.bias_off + 3072, ok ? (uint32_t)(ch * 4) : kOob);
          dma16(rqp, buf + lay.bias_off + 4096, ok ? (uint32_t)((a.Co + ch) * 4) : kOob);
        }
      }
      iss_slot = next_slot(iss_slot);
      if (++iss_ch == iss_hi && ++iss_wt < wt1) {
        iss_ch = u_lo(iss_wt);
        iss_hi = u_hi(iss_wt);
        iss_t = decode(iss_wt / SPL);
      }
    };
    // Depthwise weights of the item in ring slot `slot` (wave 0): raw [c][tap] elements
    // -> [tap][c] dot-operand words. All reads are issued before the first write.
    auto convert = [&](int slot) {
      if constexpr (HAS_DW) {
        if (wave != 0) return;
        constexpr int NEL = CB * KK;                      // weights of the chunk
        constexpr int EPV = 16 / DT::ELT;                 // elements per 16-byte vector
        constexpr int NV = (NEL * DT::ELT + 1023) / 1024;  // vectors per lane
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          char* plane = bufp(slot) + s * lay.plane_bytes;
          const char* raw = plane + lay.raw_off;
          uint32_t* dst = (uint32_t*)(plane + lay.wd_off);
          u32x4 rv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) rv[v] = *(const u32x4*)(raw + (v * 64 + lane) * 16);  // within the NRAW KiB
#pragma unroll
          for (int v = 0; v < NV; ++v) {
#pragma unroll
            for (int k = 0; k < EPV; ++k) {
              const int e = (v * 64 + lane) * EPV + k;
              if (e < NEL) {
                const uint32_t word = rv[v][k * DT::ELT / 4];
                uint32_t el;
                if constexpr (DT::ELT == 4)
                  el = word;
                else if constexpr (DT::ELT == 2)
                  el = (k & 1) ? word >> 16 : word & 0xffffu;
                else
                  el = (word >> (8 * (k & 3))) & 0xffu;
                const int ci = e / KK, tap = e - (e / KK) * KK;
                dst[tap * CB + ci] = D3::weight_word(el, ci);
              }
            }
          }
        }
      }
    };
    // Copies complete in issue order, so "item j has landed" is a wait until at most the
    // copies of the items issued after j are outstanding (the host keeps that count
    // <= 63; a larger one would fall back to a full wait).
    const int ahead = min(nitems, D - 1);
    for (int i = 0; i < ahead; ++i) issue_next();
    wait_vm((ahead - 1) * mine);
    fix_next();
    convert(0);
    wait_lgkm0();
    barrier3();
    int cv_slot = next_slot(0);
    for (int it = 0; it < nitems; ++it) {
      // slot of item it + D - 1 is the one item it - 1 used: released by the last barrier
      if (it + D - 1 < nitems) issue_next();
      if (it + 1 < nitems) {
        wait_vm((min(nitems, it + D) - (it + 2)) * mine);
        fix_next();
        convert(cv_slot);
      }
      cv_slot = next_slot(cv_slot);
      wait_lgkm0();
      barrier3();
    }
    return;
  }

  // ========================== compute waves ==========================================
  int base[BPW], pyx[BPW];
#pragma unroll
  for (int b = 0; b < BPW; ++b) {
    int p = (b * 4 + cw) * 16 + r16;
    const bool ok = p < P;
    if (!ok) p = P - 1;
    const int py = p / TW, px = p - py * TW;
    pyx[b] = ok ? (py << 16) | px : -1;
    base[b] = (py * SE * IWP + px) * kRowB + g * 16;
  }
  int nblk = 0;  // blocks holding at least one pixel of the tile (wave-uniform)
#pragma unroll
  for (int b = 0; b < BPW; ++b)
    if ((b * 4 + cw) * 16 < P) nblk = b + 1;
  const int a_row = r16 * kRowB + ((g ^ (((r16 >> 3) & 1) << 1)) * 16);  // swizzled MFMA A slot
  const Epi3 ep_dw = make_epi3(a.act[0], a.rq[0]);
  const Epi3 ep_pw = MODE == M3_PW ? ep_dw : make_epi3(a.act[1], a.rq[1]);
  // Asymmetric int8 PW input (zero point z_pw): every output channel loses z_pw x its
  // weight-row sum, which each lane accumulates from its A operands (16 bytes of a row per
  // chunk) and completes at the epilogue.
  const int z_pw = (QX && HAS_PW) ? a.zin[MODE == M3_PW ? 0 : 1] : 0;
  const bool pc_dw = PCQ && HAS_DW && a.rqc[0] != nullptr;  // (uniform)
  const bool pc_pw = PCQ && HAS_PW && a.rqc[MODE == M3_PW ? 0 : 1] != nullptr;
  int32_t rsp[CT];
#pragma unroll
  for (int i = 0; i < CT; ++i) rsp[i] = 0;

  AccV acc[BPW][CT];
#pragma unroll
  for (int b = 0; b < BPW; ++b)
#pragma unroll
    for (int i = 0; i < CT; ++i) acc[b][i] = AccV{0, 0, 0, 0};
  u32x4 bop[BPW];

  barrier3();  // item 0 is ready
  int wt = wt0, ch = u_lo(wt0), ch_hi = u_hi(wt0), slot = 0;
  Tile cur_t = decode(wt0 / SPL);
  for (int it = 0; it < nitems; ++it) {
    const char* buf = bufp(slot);
    slot = next_slot(slot);
    // B operand of each block: depthwise output of this lane's pixel and channel slot
    // (or the staged input itself for the PW kernel), then the PW contraction. The
    // number of blocks holding pixels is a compile-time constant of each instance of
    // `step`, so the unrolled loops carry no branches and the LDS reads of all taps
    // can be scheduled ahead of the arithmetic.
    auto step = [&](auto nb_tag) {
      constexpr int NB = decltype(nb_tag)::value;
#pragma unroll
      for (int s = 0; s < KS; ++s) {  // the item's channel chunks, one plane each
        const char* plane = buf + s * lay.plane_bytes;
        if constexpr (HAS_DW) {
          Acc dacc[NB][CPL];
          const char* wl = plane + lay.wd_off;
          {
            u32x4 bv[WQ];
#pragma unroll
            for (int q = 0; q < WQ; ++q)
              bv[q] = *(const u32x4*)(buf + lay.bias_off + (s * CB + g * CPL + 4 * q) * 4);
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
              for (int e = 0; e < CPL; ++e) {
                const uint32_t u = bv[e >> 2][e & 3];
                dacc[b][e] = __builtin_bit_cast(Acc, u);
              }
          }
          const char* xb[NB];
#pragma unroll
          for (int b = 0; b < NB; ++b) xb[b] = plane + base[b];
#pragma unroll
          for (int ky = 0; ky < KE; ++ky) {
#pragma unroll
            for (int kx = 0; kx < KE; ++kx) {
              const int toff = (ky * IWP + (SE == 2 ? (kx & 1) * (IWP / 2) + (kx >> 1) : kx)) * kRowB;
              u32x4 wv[WQ];
#pragma unroll
              for (int q = 0; q < WQ; ++q)
                wv[q] = *(const u32x4*)(wl + ((ky * KE + kx) * CB + g * CPL + 4 * q) * 4);
#pragma unroll
              for (int b = 0; b < NB; ++b) D3::tap(dacc[b], *(const u32x4*)(xb[b] + toff), wv);
            }
          }
          if constexpr (PCQ) {
            if (pc_dw) {
              // this lane's CPL channels of chunk s: multipliers, then (512 bytes on) shifts
              const char* pm = buf + lay.bias_off + 2048 + (s * CB + g * CPL) * 4;
              // One value at a time: each value's input is released by the previous
              // result (a wave issues its vector instructions in order, so the chain costs
              // no issue slots), which keeps the 64-bit temporaries of one value live
              // instead of those of all NB x CPL.
              int32_t tok = 0;
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const u32x4 mv = *(const u32x4*)(pm + 16 * j), sv = *(const u32x4*)(pm + 512 + 16 * j);
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                  uint32_t wv = 0;
#pragma unroll
                  for (int e = 0; e < 4; ++e) {
                    int32_t v = dacc[b][4 * j + e];
                    asm volatile("" : "+v"(v) : "v"(tok));
                    tok = epi_q(v, (int32_t)mv[e], pc_shift(sv[e]), ep_dw);
                    wv |= ((uint32_t)tok & 0xffu) << (8 * e);
                  }
                  bop[b][j] = wv;
                }
              }
            } else {
#pragma unroll
              for (int b = 0; b < NB; ++b) bop[b] = D3::finish(dacc[b], ep_dw);
            }
          } else {
#pragma unroll
            for (int b = 0; b < NB; ++b) bop[b] = D3::finish(dacc[b], ep_dw);
          }
        } else {
#pragma unroll
          for (int b = 0; b < NB; ++b) bop[b] = *(const u32x4*)(plane + base[b]);
        }
        if constexpr (HAS_PW) {
          const char* wl = plane + lay.in_bytes;
          auto contract = [&](auto rs_tag) {
#pragma unroll
            for (int i = 0; i < CT; ++i) {
              const u32x4 av = *(const u32x4*)(wl + i * 1024 + a_row);
#pragma unroll
              for (int b = 0; b < NB; ++b) mma16(DT{}, acc[b][i], av, bop[b]);
              if constexpr (decltype(rs_tag)::value) {
#pragma unroll
                for (int q = 0; q < 4; ++q) rsp[i] = __builtin_amdgcn_sdot4((int)av[q], 0x01010101, rsp[i], false);
              }
            }
          };
          if constexpr (QX != 0) {
            if (z_pw != 0) contract(std::true_type{});  // (uniform)
            else contract(std::false_type{});
          } else {
            contract(std::false_type{});
          }
        }
      }
    };
    if (nblk >= BPW) {
      step(std::integral_constant<int, BPW>{});
    } else if constexpr (BPW > 1) {
      if (nblk == 1) step(std::integral_constant<int, 1>{});
      else if (BPW > 2 && nblk == 2) step(std::integral_constant<int, (BPW > 2 ? 2 : 1)>{});
      else if (BPW > 3 && nblk == 3) step(std::integral_constant<int, (BPW > 3 ? 3 : 1)>{});
    }

    if (ch + 1 == ch_hi) {
      // ---- epilogue of the work unit: straight from registers to global memory ----
      if constexpr (QX != 0 && HAS_PW) {
        if (z_pw != 0) {
          // (a split: the weight-row sums over its own channel chunks) row m of tile i:
          // the four lanes l % 16 == m hold its quarters; then each accumulator lane takes
          // rows 4g + v
#pragma unroll
          for (int i = 0; i < CT; ++i) {
            int32_t s = rsp[i];
            s += __shfl_xor(s, 16);
            s += __shfl_xor(s, 32);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int32_t r = __shfl(s, 4 * g + v);
#pragma unroll
              for (int b = 0; b < BPW; ++b) acc[b][i][v] -= z_pw * r;
            }
          }
        }
#pragma unroll
        for (int i = 0; i < CT; ++i) rsp[i] = 0;
      }
      if constexpr (MODE == M3_DW) {
        const int c = cur_t.cb * CB + g * CPL;
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const int v = pyx[b];
          const int oy = cur_t.oy0 + (v >> 16), ox = cur_t.ox0 + (v & 0xffff);
          if (v >= 0 && oy < a.Ho && ox < a.Wo && c < C)
            *(u32x4*)((T*)a.y + (((size_t)cur_t.n * a.Ho + oy) * a.Wo + ox) * C + c) = bop[b];
        }
      } else if constexpr (SPLIT) {
        // a split of the work tile: its partial sums (before bias and activation) go to
        // slice [split][work tile][pixel][channel] of the workspace, 16 bytes per MFMA tile
        Acc* wsp = (Acc*)a.ws + ((size_t)(wt % SPL) * (a.nwork / SPL) + wt / SPL) * P * CoB;
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const int v = pyx[b];
          if (b >= nblk || v < 0) continue;
          Acc* row = wsp + (size_t)((v >> 16) * TW + (v & 0xffff)) * CoB;
#pragma unroll
          for (int i = 0; i < CT; ++i)
            *(AccV*)(row + OGE * (4 * (i / OTPG) + g) + 4 * (i % OTPG)) = acc[b][i];
        }
#pragma unroll
        for (int b = 0; b < BPW; ++b)
#pragma unroll
          for (int i = 0; i < CT; ++i) acc[b][i] = AccV{0, 0, 0, 0};
      } else {
        // this lane's output granules k = 0 .. CT/OTPG - 1: channels co_blk + OGE * (4k + g) + [0, OGE)
        constexpr int NG = MODE == M3_DW ? 1 : CT / OTPG;
        const int co_blk = cur_t.cb * CoB;
        const bool full16 = (a.Co * DT::ELT) % 16 == 0;
        Acc bias[NG][OGE];
        {
          const char* bl = buf + lay.bias_off + 1024;  // bias block of this co-block
#pragma unroll
          for (int k = 0; k < NG; ++k)
#pragma unroll
            for (int q = 0; q < OGE / 4; ++q) {
              const u32x4 bv = *(const u32x4*)(bl + (OGE * (4 * k + g) + 4 * q) * 4);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const uint32_t u = bv[e];
                bias[k][4 * q + e] = __builtin_bit_cast(Acc, u);
              }
            }
        }
#pragma unroll
        for (int b = 0; b < BPW; ++b) {
          const int v = pyx[b];
          const int oy = cur_t.oy0 + (v >> 16), ox = cur_t.ox0 + (v & 0xffff);
          if (b >= nblk || v < 0 || oy >= a.Ho || ox >= a.Wo) continue;
          char* dpx = (char*)a.y + (((size_t)cur_t.n * a.Ho + oy) * a.Wo + ox) * a.Co * DT::ELT;
#pragma unroll
          for (int k = 0; k < NG; ++k) {
            const int c0k = co_blk + OGE * (4 * k + g);
            if (c0k >= a.Co) continue;
            // channel c0k + j, j = 4t + e, is value e of tile k * OTPG + t
            uint32_t wd4[4];
            if constexpr (DT::ELT == 4) {
#pragma unroll
              for (int e = 0; e < 4; ++e) wd4[e] = __float_as_uint(epi_f(acc[b][k][e] + bias[k][e], ep_pw));
            } else if constexpr (DT::ELT == 2) {
#pragma unroll
              for (int w = 0; w < 4; ++w) {
                const int t = w >> 1, e = 2 * (w & 1);
                wd4[w] = pack_bf16x2(epi_f(acc[b][2 * k + t][e] + bias[k][4 * t + e], ep_pw),
                                     epi_f(acc[b][2 * k + t][e + 1] + bias[k][4 * t + e + 1], ep_pw));
              }
            } else {
#pragma unroll
              for (int w = 0; w < 4; ++w) {
                uint32_t wv = 0;
                if (PCQ && pc_pw) {
                  // multipliers (then, a KiB on, shifts) of channels c0k + 4w + [0, 4)
                  const char* pm = buf + lay.bias_off + 3072 + (OGE * (4 * k + g) + 4 * w) * 4;
                  const u32x4 mv = *(const u32x4*)pm, sv = *(const u32x4*)(pm + 1024);
#pragma unroll
                  for (int e = 0; e < 4; ++e)
                    wv |= ((uint32_t)epi_q(acc[b][4 * k + w][e] + bias[k][4 * w + e], (int32_t)mv[e], pc_shift(sv[e]),
                                           ep_pw) & 0xffu) << (8 * e);
                } else {
#pragma unroll
                  for (int e = 0; e < 4; ++e)
                    wv |= ((uint32_t)epi_i(acc[b][4 * k + w][e] + bias[k][4 * w + e], ep_pw) & 0xffu) << (8 * e);
                }
                wd4[w] = wv;
              }
            }
            char* dst = dpx + (size_t)c0k * DT::ELT;
            if (full16) {
              *(u32x4*)dst = u32x4{wd4[0], wd4[1], wd4[2], wd4[3]};
            } else {
              // c_out * elt is a multiple of 4: whole 32-bit words are in or out of range
#pragma unroll
              for (int w = 0; w < 4; ++w)
                if (c0k + w * (4 / DT::ELT) < a.Co) *(uint32_t*)(dst + 4 * w) = wd4[w];
            }
          }
        }
#pragma unroll
        for (int b = 0; b < BPW; ++b)
#pragma unroll
          for (int i = 0; i < CT; ++i) acc[b][i] = AccV{0, 0, 0, 0};
      }
      if (++wt < wt1) {
        ch = u_lo(wt);
        ch_hi = u_hi(wt);
        cur_t = decode(wt / SPL);
      }
    } else {
      ++ch;
    }
    wait_lgkm0();
    barrier3();  // item it+1 is ready; this item's buffer may be refilled
  }
}

// Second kernel of a split plan: for every work tile, pixel and group of four output
// channels, the partial sums of the splits are added in split order, then bias,
// activation and cast as in the single-kernel epilogue (same rounding: the fp32 or int32
// total of the contraction, then +bias, then the stage's activation / requantisation).
template <class DT, int STAGE>
__global__ __launch_bounds__(256) void k_combine3(KArgs a) {
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  const int SPL = a.splits, ntile = a.nwork / SPL;
  const int TH = a.TH, TW = a.TW, P = TH * TW, CoB = a.COB, nq = CoB / 4;
  const int64_t total = (int64_t)ntile * P * nq;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int q = (int)(idx % nq);
  const int64_t r = idx / nq;
  const int p = (int)(r % P), wtile = (int)(r / P);
  int t = wtile;
  const int cb = t % a.n_cb;
  t /= a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;
  const int oy = ty * TH + p / TW, ox = tx * TW + p % TW;
  const int co = cb * CoB + 4 * q;
  if (oy >= a.Ho || ox >= a.Wo || co >= a.Co) return;
  const size_t slice = (size_t)ntile * P * CoB;
  const Acc* src = (const Acc*)a.ws + ((size_t)wtile * P + p) * CoB + 4 * q;
  // the slices are read eight at a time, all eight loads in flight together, and added in
  // split order
  Acc sum[4] = {0, 0, 0, 0};
  for (int s0 = 0; s0 < SPL; s0 += 8) {
    typename DT::AccV v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < SPL) v[j] = *(const typename DT::AccV*)(src + (s0 + j) * slice);
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (s0 + j < SPL) {
#pragma unroll
        for (int e = 0; e < 4; ++e) sum[e] += v[j][e];
      }
  }
  const Epi3 ep = make_epi3(a.act[STAGE], a.rq[STAGE]);  // STAGE: index of the PW convolution
  const void* bp = STAGE == 0 ? a.b1 : a.b2;
  const int32_t* pc = a.rqc[STAGE];  // int8 per-channel [multipliers | shifts] or nullptr
  const size_t yo = (((size_t)n * a.Ho + oy) * a.Wo + ox) * a.Co + co;  // element offset
  T* y = (T*)a.y + yo;
  const int ne = a.Co - co < 4 ? a.Co - co : 4;
  uint32_t out[4];  // the four results' bit patterns
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    out[e] = 0u;
    if (e >= ne) break;
    if constexpr (DT::ELT == 1) {
      const int32_t b = bp ? ((const int32_t*)bp)[co + e] : 0;
      out[e] = (uint32_t)(pc ? epi_q(sum[e] + b, pc[co + e], pc_shift((uint32_t)pc[a.Co + co + e]), ep)
                             : epi_i(sum[e] + b, ep)) & 0xffu;
    } else {
      const float b = bp ? ((const float*)bp)[co + e] : 0.0f;
      const float o = epi_f(sum[e] + b, ep);
      out[e] = DT::ELT == 4 ? __float_as_uint(o) : (pack_bf16x2(o, 0.0f) & 0xffffu);
    }
  }
  if (ne == 4 && (uintptr_t)y % (4 * DT::ELT) == 0) {  // one aligned store of the four results
    if constexpr (DT::ELT == 1)
      *(uint32_t*)y = out[0] | (out[1] << 8) | (out[2] << 16) | (out[3] << 24);
    else if constexpr (DT::ELT == 2)
      *(u32x2*)y = u32x2{out[0] | (out[1] << 16), out[2] | (out[3] << 16)};
    else
      *(u32x4*)y = u32x4{out[0], out[1], out[2], out[3]};
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (e >= ne) break;
      if constexpr (DT::ELT == 1)
        y[e] = (T)out[e];
      else if constexpr (DT::ELT == 2)
        *(uint16_t*)(y + e) = (uint16_t)out[e];
      else
        y[e] = __uint_as_float(out[e]);
    }
  }
}

template <class DT, int K, int S, int BPW, int CT, int MODE, int IWP, int KS>
int launch_fused3(const KArgs& a, int grid, void* stream) {
  const bool split = MODE != M3_DW && a.splits > 1;
  // the zero-point (and per-channel) instances (int8) only where the module has
  // the feature, so that symmetric int8 runs without their registers
  constexpr bool kI8 = std::is_same<DT, TI8>::value;
  const bool two = MODE == M3_DWPW;  // stages whose input zero point / requantisation count
  const bool zp = a.zin[0] != 0 || (two && a.zin[1] != 0);
  const bool pc = a.rqc[0] != nullptr || (two && a.rqc[1] != nullptr);
  const int qx = !kI8 ? 0 : (pc ? 2 : (zp ? 1 : 0));
  constexpr bool SP = MODE != M3_DW;  // (the depthwise-only kernel never splits)
  auto fn = split ? (qx == 2   ? k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, SP, (kI8 ? 2 : 0)>
                     : qx == 1 ? k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, SP, (kI8 ? 1 : 0)>
                               : k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, SP, 0>)
            : qx == 2 ? k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, false, (kI8 ? 2 : 0)>
            : qx == 1 ? k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, false, (kI8 ? 1 : 0)>
                      : k_fused3<DT, K, S, BPW, CT, MODE, IWP, KS, false, 0>;
  const int lds = a.L.bytes;
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return (int)e;
  }
  // persistent grid: as many workgroups as are resident at once, at most one per work unit
  static thread_local int cached_lds[6] = {-1, -1, -1, -1, -1, -1}, cached_occ[6] = {1, 1, 1, 1, 1, 1};
  const int ci = (split ? 3 : 0) + qx;
  if (cached_lds[ci] != lds) {
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, (const void*)fn, kThreads3, lds) != hipSuccess || occ < 1)
      occ = 1;
    cached_lds[ci] = lds;
    cached_occ[ci] = occ;
  }
  int g = a.cus * cached_occ[ci];
  if (a.grid_cap > 0 && g > a.grid_cap) g = a.grid_cap;
  if (g > a.nwork) g = a.nwork;
  if (g < 1) g = 1;
  (void)grid;
  const int e = launch_args((const void*)fn, g, kThreads3, lds, stream, a);
  if (e != 0) return e;
  if constexpr (MODE != M3_DW) {
    if (a.splits > 1) {
      KArgs c = a;
      c.COB = 16 * CT;
      const int64_t total = (int64_t)(a.nwork / a.splits) * a.TH * a.TW * (4 * CT);
      return launch_args((const void*)k_combine3<DT, MODE == M3_PW ? 0 : 1>, (int)((total + 255) / 256), 256, 0,
                         stream, c);
    }
  }
  return 0;
}

}  // namespace fcm
