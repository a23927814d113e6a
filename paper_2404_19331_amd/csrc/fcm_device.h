// fcm_device.h -- device building blocks shared by the fused-module kernels (gfx950).
//
// Every kernel is a composition of the same four steps (Sec. III-B of arXiv 2404.19331
// describes the module skeleton: stage what the first convolution needs, compute it into
// an on-chip communication buffer, synchronise, compute the second convolution from that
// buffer and write only its output):
//   stage_*      global -> LDS, 16-byte vector loads where alignment allows, zero fill
//                outside the image and beyond the channel count;
//   dw_compute   depthwise KxK stencil from an LDS tile [rows][cols][channels] into an LDS
//                tile [pixels][channels] (+bias, activation, cast);
//   mma_chunk    pointwise contraction on MFMA: acc[m][p] += A[m][k] * B[p][k] with both
//                operands rows of k-contiguous data in LDS (16x16 output tiles per MFMA);
//   store_tile   LDS tile [pixels][channels] -> global NCHW/NHWC, 16-byte stores.
// The layouts in LDS are the same for every module, so the layer-by-layer kernels are
// the fused ones with a stage switched off (the paper's LBL baselines share the fused
// kernels' dataflow, Sec. V-C).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "fcm_internal.h"

namespace fcm {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;  // 4 waves of 64 lanes per workgroup

// ------------------------------------------------------------------------------------
// Element-type traits.
//   KB:  contraction elements consumed per 16-byte-per-lane MFMA operand step
//        (4 lane groups x 16 bytes = 64 bytes of k per row)
//   CPT: channels per depthwise thread-vector
// ------------------------------------------------------------------------------------
struct TF32 {
  using T = float;
  using Acc = float;
  using AccV = f32x4;
  static constexpr int ELT = 4, KB = 16, CPT = 4;
};
struct TBF16 {
  using T = uint16_t;
  using Acc = float;
  using AccV = f32x4;
  static constexpr int ELT = 2, KB = 32, CPT = 8;
};
struct TI8 {
  using T = int8_t;
  using Acc = int32_t;
  using AccV = i32x4;
  static constexpr int ELT = 1, KB = 64, CPT = 8;
};

// ------------------------------------------------------------------------------------
// Scalar conversions / epilogue arithmetic
// ------------------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bfloat16, round to nearest, ties to even; NaN stays a quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float act_f(float v, int act) {
  if (act == ACT_RELU) return fmaxf(v, 0.0f);
  if (act == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
  return v;
}

// q = clamp(round_half_even(acc * mult / 2^shift) + zp, qmin, qmax), then ReLU if asked,
// which clamps below at zp, the code of real 0 (ReLU6 too: its upper end is qmax, 6.0 in
// the output's quantised units).
__device__ __forceinline__ int32_t requant(int32_t acc, const Requant& rq, int act) {
  int64_t t = (int64_t)acc * (int64_t)rq.mult;
  int64_t q = t;
  if (rq.shift > 0) {
    q = t >> rq.shift;
    int64_t r = t - (q << rq.shift);
    int64_t half = (int64_t)1 << (rq.shift - 1);
    q += (r > half || (r == half && (q & 1))) ? 1 : 0;
  }
  q += rq.zp;
  q = q < rq.qmin ? rq.qmin : q;
  q = q > rq.qmax ? rq.qmax : q;
  if (act != ACT_NONE && q < rq.zp) q = rq.zp;
  return (int32_t)q;
}

// The requantisation of channel c: its own multiplier and shift when the stage has
// per-channel ones (shift kept in [0, 62]), the stage's clamp range either way.
__device__ __forceinline__ Requant rq_at(const Requant& rq, const ReqCh& pc, int c) {
  if (!pc.p) return rq;
  Requant r = rq;
  r.mult = pc.p[c];
  r.shift = min(max(pc.p[pc.n + c], 0), 62);
  return r;
}

// Finish one accumulator (+bias, activation, cast) into storage bits.
template <class DT>
struct Fin;
template <>
struct Fin<TF32> {
  __device__ static __forceinline__ uint32_t apply(float acc, float bias, int act, const Requant&) {
    return __float_as_uint(act_f(acc + bias, act));
  }
};
template <>
struct Fin<TBF16> {
  __device__ static __forceinline__ uint32_t apply(float acc, float bias, int act, const Requant&) {
    return f32_to_bf16(act_f(acc + bias, act));
  }
};
template <>
struct Fin<TI8> {
  __device__ static __forceinline__ uint32_t apply(int32_t acc, int32_t bias, int act, const Requant& rq) {
    return (uint32_t)(requant(acc + bias, rq, act) & 0xff);
  }
};

// Bias element as the accumulator type (float for float paths, int32 for int8).
template <class DT>
__device__ __forceinline__ typename DT::Acc load_bias(const void* b, int i) {
  if (!b) return typename DT::Acc(0);
  if constexpr (std::is_same<DT, TI8>::value)
    return ((const int32_t*)b)[i];
  else
    return ((const float*)b)[i];
}

// Store 4 consecutive finished values (bits) at an LDS address.
template <class DT>
__device__ __forceinline__ void lds_store4(char* p, uint32_t v0, uint32_t v1, uint32_t v2, uint32_t v3) {
  if constexpr (DT::ELT == 4) {
    *(u32x4*)p = u32x4{v0, v1, v2, v3};
  } else if constexpr (DT::ELT == 2) {
    *(u32x2*)p = u32x2{v0 | (v1 << 16), v2 | (v3 << 16)};
  } else {
    *(uint32_t*)p = v0 | (v1 << 8) | (v2 << 16) | (v3 << 24);
  }
}

// ------------------------------------------------------------------------------------
// MFMA: one 16-byte-per-lane operand step into a 16x16 accumulator tile.
// Lane l supplies row (l % 16) of A and column (l % 16) of B, and the 16 bytes at
// k-offset (l / 16) * 16 bytes of the step. A and B use the same k assignment, so any
// order of k inside a step is a valid contraction. Output: lane l holds
// C[m = 4 * (l / 16) + v][n = l % 16], v = 0..3.
// ------------------------------------------------------------------------------------
__device__ __forceinline__ void mma16(TF32, f32x4& c, const u32x4& a, const u32x4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
}
__device__ __forceinline__ void mma16(TBF16, f32x4& c, const u32x4& a, const u32x4& b) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                               0, 0, 0);
}
__device__ __forceinline__ void mma16(TI8, i32x4& c, const u32x4& a, const u32x4& b) {
  c = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0, 0,
                                             0);
}

// acc[i][j] += A[m_base + 16i .. +16][0..K) * B[n_base + 16j .. +16][0..K)^T
// A, B: LDS, rows of K contiguous elements at byte strides as_, bs_ (multiples of 16).
template <class DT, int TMW, int TNW>
__device__ __forceinline__ void mma_chunk(typename DT::AccV (&acc)[TMW][TNW], const char* A, int as_,
                                          const char* B, int bs_, int K, int m_base, int n_base, int m_act,
                                          int n_act) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  const int nkb = K / DT::KB;
  const char* pa = A + (m_base + r) * as_ + g * 16;
  const char* pb = B + (n_base + r) * bs_ + g * 16;
#pragma unroll 1
  for (int kb = 0; kb < nkb; ++kb) {
    u32x4 a[TMW], b[TNW];
#pragma unroll
    for (int i = 0; i < TMW; ++i)
      if (i < m_act) a[i] = *(const u32x4*)(pa + i * 16 * as_ + kb * 64);
#pragma unroll
    for (int j = 0; j < TNW; ++j)
      if (j < n_act) b[j] = *(const u32x4*)(pb + j * 16 * bs_ + kb * 64);
#pragma unroll
    for (int i = 0; i < TMW; ++i)
#pragma unroll
      for (int j = 0; j < TNW; ++j)
        if (i < m_act && j < n_act) mma16(DT{}, acc[i][j], a[i], b[j]);
  }
}

// ------------------------------------------------------------------------------------
// Staging: global -> LDS
//
// A copy job is a "loader": load(i, v) fetches item i into registers and returns where
// it goes in LDS; store(s, d, v) writes it. staged_copy runs up to three jobs together:
// in each round every thread issues kBatch loads per job before writing any of them, so
// a thread keeps up to 3*kBatch global loads in flight.
// Loads are unconditional: an item outside the image or the channel range reads a valid
// clamped address and carries kZero in its destination, and the zero is substituted at
// store time. (A load under a branch makes the compiler wait for it inside the branch,
// which would serialise one memory latency per item.)
// ------------------------------------------------------------------------------------
constexpr int kBatch = 4;
constexpr int kZero = 1 << 30;  // destination flag: store zero instead of the loaded value
constexpr int kAux = 1 << 29;   // destination flag used by DwWeights: the item is a bias
constexpr int kOffMask = (1 << 29) - 1;

struct NullLoader {
  using V = uint32_t;
  __device__ __forceinline__ int load(int, V&) const { return -1; }
  __device__ __forceinline__ void store(char*, int, const V&) const {}
};

template <int B, class LA, class LB, class LC>
__device__ __forceinline__ void staged_copy(char* s, int ta, const LA& la, int tb, const LB& lb, int tc,
                                            const LC& lc) {
  const int tmax = max(ta, max(tb, tc));
#pragma unroll 1
  for (int base = threadIdx.x; base < tmax; base += kThreads * B) {
    typename LA::V va[B];
    typename LB::V vb[B];
    typename LC::V vc[B];
    int da[B], db[B], dc[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int i = base + j * kThreads;
      // Callers pass NullLoader for an empty job, so a real loader always has t > 0 and
      // its load needs no guard (a branch here would put the loads under control flow).
      da[j] = la.load(min(i, ta - 1), va[j]);
      db[j] = lb.load(min(i, tb - 1), vb[j]);
      dc[j] = lc.load(min(i, tc - 1), vc[j]);
      if (i >= ta) da[j] = -1;
      if (i >= tb) db[j] = -1;
      if (i >= tc) dc[j] = -1;
    }
#pragma unroll
    for (int j = 0; j < B; ++j) {
      if (da[j] >= 0) la.store(s, da[j], va[j]);
      if (db[j] >= 0) lb.store(s, db[j], vb[j]);
      if (dc[j] >= 0) lc.store(s, dc[j], vc[j]);
    }
  }
}

template <int B, class LA>
__device__ __forceinline__ void staged_copy(char* s, int ta, const LA& la) {
  staged_copy<B>(s, ta, la, 0, NullLoader{}, 0, NullLoader{});
}

// fill: the bits stored for a kZero item (four copies of an int8 zero point for a window
// a depthwise stage pads; 0 everywhere else).
__device__ __forceinline__ void store_vec(char* s, int d, const u32x4& v, uint32_t fill = 0u) {
  *(u32x4*)(s + (d & kOffMask)) = (d & kZero) ? u32x4{fill, fill, fill, fill} : v;
}

template <class T>
__device__ __forceinline__ void store_elem(char* s, int d, const T& v, uint32_t fill = 0u) {
  *(T*)(s + (d & kOffMask)) = (d & kZero) ? (T)fill : v;
}

// Bits of four int8 codes equal to zero point z (0 for the float types).
template <class DT>
__device__ __forceinline__ uint32_t zp_fill(int z) {
  if constexpr (std::is_same<DT, TI8>::value)
    return (uint32_t)(uint8_t)z * 0x01010101u;
  else
    return 0u;
}

// Haloed input window rows [iy0, iy0+IH) x cols [ix0, ix0+IW), channels [c0, c0+CB) into
// LDS at `off` as [IH*IW pixels][CB] with pixel stride ps bytes. `fill` outside the image
// and for channels >= C: zero, or the code of real 0 of an asymmetric int8 input.
template <class DT>
struct InputVec {  // NHWC, 16-byte vectors (C*ELT % 16 == 0, x 16-byte aligned)
  using V = u32x4;
  static constexpr int VE = 16 / DT::ELT;
  const typename DT::T* x;
  int n, C, H, W, iy0, ix0, IW, c0, nv, ps, off;
  uint32_t fill = 0u;
  __device__ __forceinline__ int load(int i, V& v) const {
    const int vv = i % nv, pix = i / nv;
    const int py = pix / IW, px = pix - py * IW;
    const int gy = iy0 + py, gx = ix0 + px, c = c0 + vv * VE;
    const bool ok = (unsigned)gy < (unsigned)H && (unsigned)gx < (unsigned)W && c < C;
    const size_t idx = ok ? (((size_t)n * H + gy) * W + gx) * C + c : 0;
    v = *(const u32x4*)(x + idx);
    return (off + pix * ps + vv * 16) | (ok ? 0 : kZero);
  }
  __device__ __forceinline__ void store(char* s, int d, const V& v) const { store_vec(s, d, v, fill); }
};

template <class DT>
struct InputElem {  // NHWC or NCHW, one element per item
  using V = typename DT::T;
  const typename DT::T* x;
  int layout, n, C, H, W, iy0, ix0, IH, IW, c0, CB, ps, off;
  uint32_t fill = 0u;
  __device__ __forceinline__ int load(int i, V& v) const {
    int ci, py, px;
    if (layout == LAYOUT_NHWC) {
      ci = i % CB;
      const int pix = i / CB;
      py = pix / IW;
      px = pix - py * IW;
    } else {
      px = i % IW;
      const int t = i / IW;
      py = t % IH;
      ci = t / IH;
    }
    const int gy = iy0 + py, gx = ix0 + px, c = c0 + ci;
    const bool ok = (unsigned)gy < (unsigned)H && (unsigned)gx < (unsigned)W && c < C;
    const size_t idx = !ok ? 0
                           : (layout == LAYOUT_NHWC ? (((size_t)n * H + gy) * W + gx) * C + c
                                                    : (((size_t)n * C + c) * H + gy) * W + gx);
    v = x[idx];
    return (off + (py * IW + px) * ps + ci * DT::ELT) | (ok ? 0 : kZero);
  }
  __device__ __forceinline__ void store(char* s, int d, const V& v) const { store_elem(s, d, v, fill); }
};

// Rows [r0, r0+rows) x cols [c0, c0+CB) of a row-major [R][Cc] matrix into LDS rows of
// stride rs bytes at `off`; zero beyond R or Cc.
template <class DT>
struct RowsVec {  // Cc*ELT % 16 == 0 and w 16-byte aligned
  using V = u32x4;
  static constexpr int VE = 16 / DT::ELT;
  const typename DT::T* w;
  int R, Cc, r0, c0, nv, rs, off;
  __device__ __forceinline__ int load(int i, V& v) const {
    const int vv = i % nv, r = i / nv;
    const int gr = r0 + r, c = c0 + vv * VE;
    const bool ok = gr < R && c < Cc;
    v = *(const u32x4*)(w + (ok ? (size_t)gr * Cc + c : 0));
    return (off + r * rs + vv * 16) | (ok ? 0 : kZero);
  }
  __device__ __forceinline__ void store(char* s, int d, const V& v) const { store_vec(s, d, v); }
};

template <class DT>
struct RowsElem {
  using V = typename DT::T;
  const typename DT::T* w;
  int R, Cc, r0, c0, CB, rs, off;
  __device__ __forceinline__ int load(int i, V& v) const {
    const int ci = i % CB, r = i / CB;
    const int gr = r0 + r, c = c0 + ci;
    const bool ok = gr < R && c < Cc;
    v = w[ok ? (size_t)gr * Cc + c : 0];
    return (off + r * rs + ci * DT::ELT) | (ok ? 0 : kZero);
  }
  __device__ __forceinline__ void store(char* s, int d, const V& v) const { store_elem(s, d, v); }
};

// Depthwise weights [C][K][K] (channels c0..c0+CB) as accumulator-type values laid out
// [K*K taps][CB] at `off`, followed by the bias [CB]. Zero for channels >= C and for a
// NULL bias. The raw element is converted at store time.
template <class DT, int K>
struct DwWeights {
  using V = u32x2;  // {raw weight element, raw bias bits}; both always loaded, no branch
  const typename DT::T* wd;
  const void* bd;
  int C, c0, CB, off;
  __device__ __forceinline__ int load(int i, V& v) const {
    const int ci = i % CB, tap = i / CB;
    const int c = c0 + ci;
    const bool is_bias = tap >= K * K;
    const bool ok = c < C && (!is_bias || bd != nullptr);
    const int cc = c < C ? c : 0;
    const size_t wi = (size_t)cc * K * K + (is_bias ? 0 : tap);
    const uint32_t* bp = bd ? (const uint32_t*)bd : (const uint32_t*)wd;  // valid address either way
    uint32_t w;
    if constexpr (DT::ELT == 4)
      w = ((const uint32_t*)wd)[wi];
    else if constexpr (DT::ELT == 2)
      w = ((const uint16_t*)wd)[wi];
    else
      w = (uint32_t)(uint8_t)((const int8_t*)wd)[wi];
    v = V{w, bp[bd ? cc : 0]};
    return (off + i * 4) | (ok ? 0 : kZero) | (is_bias ? kAux : 0);
  }
  __device__ __forceinline__ void store(char* s, int d, const V& v) const {
    uint32_t bits = v.x;
    if constexpr (DT::ELT == 2) bits = v.x << 16;                             // bf16 -> f32
    else if constexpr (DT::ELT == 1) bits = (uint32_t)(int32_t)(int8_t)v.x;   // i8 -> i32
    if (d & kAux) bits = v.y;                                                 // float / int32 bias
    *(uint32_t*)(s + (d & kOffMask)) = (d & kZero) ? 0u : bits;
  }
};

template <class DT>
__device__ __forceinline__ InputVec<DT> input_vec(const typename DT::T* x, int n, int C, int H, int W, int iy0,
                                                  int ix0, int IW, int c0, int CB, int ps, int off,
                                                  uint32_t fill = 0u) {
  return InputVec<DT>{x, n, C, H, W, iy0, ix0, IW, c0, CB / InputVec<DT>::VE, ps, off, fill};
}
template <class DT>
__device__ __forceinline__ InputElem<DT> input_elem(const typename DT::T* x, int layout, int n, int C, int H, int W,
                                                    int iy0, int ix0, int IH, int IW, int c0, int CB, int ps,
                                                    int off, uint32_t fill = 0u) {
  return InputElem<DT>{x, layout, n, C, H, W, iy0, ix0, IH, IW, c0, CB, ps, off, fill};
}
template <class DT>
__device__ __forceinline__ RowsVec<DT> rows_vec(const typename DT::T* w, int R, int Cc, int r0, int c0, int CB,
                                                int rs, int off) {
  return RowsVec<DT>{w, R, Cc, r0, c0, CB / RowsVec<DT>::VE, rs, off};
}
template <class DT>
__device__ __forceinline__ RowsElem<DT> rows_elem(const typename DT::T* w, int R, int Cc, int r0, int c0, int CB,
                                                  int rs, int off) {
  return RowsElem<DT>{w, R, Cc, r0, c0, CB, rs, off};
}

// Stage a chunk: haloed input window (IH x IW x CB at off_in, pixel stride ps, `fill`
// outside the image), `rows` rows of a [R][Cc] weight matrix (columns c0..c0+CB at off_w,
// stride rs) and, with K > 0, the depthwise weights + bias of channels cd0..cd0+CBD at
// off_wd.
template <class DT, int K>
__device__ __forceinline__ void stage_chunk(char* s, const typename DT::T* x, int layout, bool vec_x, int n, int C,
                                            int H, int W, int iy0, int ix0, int IH, int IW, int c0, int CB, int ps,
                                            int off_in, const typename DT::T* w, bool vec_w, int R, int Cc, int r0,
                                            int rows, int rs, int off_w, const typename DT::T* wd, const void* bd,
                                            int Cd, int cd0, int CBD, int off_wd, uint32_t fill = 0u) {
  constexpr int VE = 16 / DT::ELT;
  const int t_in = x ? IH * IW * CB : 0;
  const int t_w = w ? rows * CB : 0;
  const int t_d = K > 0 ? (K * K + 1) * CBD : 0;
  const bool fast_in = layout == LAYOUT_NHWC && vec_x;
  if (fast_in && (vec_w || t_w == 0)) {
    const InputVec<DT> li = input_vec<DT>(x, n, C, H, W, iy0, ix0, IW, c0, CB, ps, off_in, fill);
    if constexpr (K > 0) {
      const DwWeights<DT, K> ld{wd, bd, Cd, cd0, CBD, off_wd};
      if (t_w > 0)
        staged_copy<kBatch>(s, t_in / VE, li, t_w / VE, rows_vec<DT>(w, R, Cc, r0, c0, CB, rs, off_w), t_d, ld);
      else
        staged_copy<kBatch>(s, t_in / VE, li, 0, NullLoader{}, t_d, ld);
    } else {
      if (t_w > 0)
        staged_copy<kBatch>(s, t_in / VE, li, t_w / VE, rows_vec<DT>(w, R, Cc, r0, c0, CB, rs, off_w), 0,
                            NullLoader{});
      else
        staged_copy<kBatch>(s, t_in / VE, li);
    }
    return;
  }
  if (fast_in)
    staged_copy<kBatch>(s, t_in / VE, input_vec<DT>(x, n, C, H, W, iy0, ix0, IW, c0, CB, ps, off_in, fill));
  else
    staged_copy<kBatch>(s, t_in,
                        input_elem<DT>(x, layout, n, C, H, W, iy0, ix0, IH, IW, c0, CB, ps, off_in, fill));
  if (t_w > 0) {
    if (vec_w)
      staged_copy<kBatch>(s, t_w / VE, rows_vec<DT>(w, R, Cc, r0, c0, CB, rs, off_w));
    else
      staged_copy<kBatch>(s, t_w, rows_elem<DT>(w, R, Cc, r0, c0, CB, rs, off_w));
  }
  if constexpr (K > 0) staged_copy<kBatch>(s, t_d, DwWeights<DT, K>{wd, bd, Cd, cd0, CBD, off_wd});
}

// Weight rows only (vector or element path).
template <class DT>
__device__ __forceinline__ void stage_rows(char* s, const typename DT::T* w, bool vec, int R, int Cc, int r0,
                                           int rows, int c0, int CB, int rs, int off) {
  constexpr int VE = 16 / DT::ELT;
  if (vec)
    staged_copy<kBatch>(s, rows * CB / VE, rows_vec<DT>(w, R, Cc, r0, c0, CB, rs, off));
  else
    staged_copy<kBatch>(s, rows * CB, rows_elem<DT>(w, R, Cc, r0, c0, CB, rs, off));
}

// ------------------------------------------------------------------------------------
// Depthwise stencil: LDS input [rows][cols][CB] (pixel stride ips) -> LDS output
// [TH*TW pixels][CB] (pixel stride ops), act + cast per stage. Each thread computes CPT
// channels of R horizontally adjacent output pixels, reusing each loaded input row
// across the K horizontal taps and the R pixels. TW must be a multiple of R.
// ------------------------------------------------------------------------------------
template <class DT>
struct Vec;  // CPT channels of one pixel, unpacked to the accumulator type
template <>
struct Vec<TF32> {
  u32x4 raw;
  __device__ __forceinline__ void load(const char* p) { raw = *(const u32x4*)p; }
  __device__ __forceinline__ float get(int e) const { return __uint_as_float(raw[e]); }
};
template <>
struct Vec<TBF16> {
  u32x4 raw;
  __device__ __forceinline__ void load(const char* p) { raw = *(const u32x4*)p; }
  __device__ __forceinline__ float get(int e) const {
    const uint32_t w = raw[e >> 1];
    return (e & 1) ? __uint_as_float(w & 0xffff0000u) : __uint_as_float(w << 16);
  }
};
template <>
struct Vec<TI8> {
  u32x2 raw;
  __device__ __forceinline__ void load(const char* p) { raw = *(const u32x2*)p; }
  __device__ __forceinline__ int32_t get(int e) const {
    const uint32_t w = raw[e >> 2];
    return (int32_t)(int8_t)((w >> ((e & 3) * 8)) & 0xff);
  }
};

// pc / ch0: per-channel requantisation of the stage (int8) and the global channel of the
// block's first channel (ch_valid channels exist).
// zin: int8 zero point of the input. The window holds codes, padded with zin (real 0), so
// sum_taps w * (code - zin) = sum_taps w * code - zin * sum_taps w.
template <class DT, int K, int S, int R>
__device__ __forceinline__ void dw_compute(const char* sin, int ips, int IW, const typename DT::Acc* swd, int CB, int TH, int TW,
                           int act, const Requant& rq, char* sout, int ops, ReqCh pc = ReqCh{}, int ch0 = 0,
                           int ch_valid = 1, int zin = 0) {
  using Acc = typename DT::Acc;
  constexpr int CPT = DT::CPT;
  constexpr int NIN = (R - 1) * S + K;
  const int ng = CB / CPT;
  const int spr = TW / R;
  const int tasks = ng * TH * spr;
#pragma unroll 1
  for (int t = threadIdx.x; t < tasks; t += kThreads) {
    const int g = t % ng, seg = t / ng;
    const int ty = seg / spr, tx0 = (seg - ty * spr) * R;
    Acc acc[R][CPT];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int e = 0; e < CPT; ++e) acc[r][e] = Acc(0);
    const Acc* wg = swd + g * CPT;
    // One kernel row per iteration (not unrolled): bounds the live registers to one row of
    // inputs, K weight vectors and the R x CPT accumulators.
#pragma unroll 1
    for (int ky = 0; ky < K; ++ky) {
      const char* row = sin + ((ty * S + ky) * IW + tx0 * S) * ips + g * CPT * DT::ELT;
      Vec<DT> in[NIN];
#pragma unroll
      for (int j = 0; j < NIN; ++j) in[j].load(row + j * ips);
#pragma unroll
      for (int kx = 0; kx < K; ++kx) {
        const Acc* wt = wg + (ky * K + kx) * CB;
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          const Acc wv = wt[e];
#pragma unroll
          for (int r = 0; r < R; ++r) acc[r][e] += wv * in[r * S + kx].get(e);
        }
      }
    }
    if constexpr (std::is_same<DT, TI8>::value) {
      if (zin != 0) {  // uniform: one zero point per launch
#pragma unroll
        for (int e = 0; e < CPT; ++e) {
          Acc wsum = 0;
#pragma unroll
          for (int tap = 0; tap < K * K; ++tap) wsum += wg[tap * CB + e];
#pragma unroll
          for (int r = 0; r < R; ++r) acc[r][e] -= zin * wsum;
        }
      }
    }
    const Acc* bias = swd + K * K * CB + g * CPT;
    Requant rqe[CPT];
#pragma unroll
    for (int e = 0; e < CPT; ++e) rqe[e] = rq_at(rq, pc, min(ch0 + g * CPT + e, ch_valid - 1));
#pragma unroll
    for (int r = 0; r < R; ++r) {
      char* o = sout + (ty * TW + tx0 + r) * ops + g * CPT * DT::ELT;
#pragma unroll
      for (int e = 0; e < CPT; e += 4) {
        lds_store4<DT>(o + e * DT::ELT, Fin<DT>::apply(acc[r][e + 0], bias[e + 0], act, rqe[e + 0]),
                       Fin<DT>::apply(acc[r][e + 1], bias[e + 1], act, rqe[e + 1]),
                       Fin<DT>::apply(acc[r][e + 2], bias[e + 2], act, rqe[e + 2]),
                       Fin<DT>::apply(acc[r][e + 3], bias[e + 3], act, rqe[e + 3]));
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Accumulator tiles -> LDS tile [pixels][channels] (finished values).
// acc[i][j] holds rows m = m_base + 16i + 4*(lane/16) + v, columns n = n_base + 16j + lane%16
// of C[m = channel][n = pixel].
// m_wr >= m_act tiles are written; tiles the MFMA loop skipped hold zero accumulators
// and come out as act(0 + 0), real 0 (bias is masked beyond m_valid).
// mask_iw > 0: pixel n is a position of an IW-wide window starting at (iy0, ix0) and
// positions outside [0,H)x[0,W) are written as real zero (PW output feeding a zero-padded
// DW): 0, or the output zero point of an asymmetric int8 stage.
// zin != 0 (int8): the B operand held codes of zero point zin, so each row m loses
// zin * sum_c wz[bias_off + m][c] (wz: the [rows][wz_cc] weights of this contraction).
// ------------------------------------------------------------------------------------

// Row sums of int8 weights w [rows][cc]: out[v] = sum_c w[row0 + 4 * (lane / 16) + v][c]
// (0 for rows >= rows_valid), the rows of this lane's accumulators. Lane l adds a quarter
// of row row0 + l % 16 (every fourth 4-byte word from word l / 16 with a four-way dot
// product against ones when rows are whole aligned words, else every fourth byte); two
// butterfly steps complete each sum and every lane then reads its four. All 64 lanes of
// the wave must call it.
__device__ __forceinline__ void int8_row_sums(const int8_t* w, int cc, int row0, int rows_valid,
                                              int32_t (&out)[4]) {
  const int lane = threadIdx.x & 63;
  const int row = row0 + (lane & 15);
  int32_t s = 0;
  if (row < rows_valid) {
    const int8_t* p = w + (size_t)row * cc;
    if ((cc & 3) == 0 && ((uintptr_t)w & 3) == 0) {
      const int32_t* p4 = (const int32_t*)p;
      const int nw = cc >> 2;
#pragma unroll 4
      for (int c = lane >> 4; c < nw; c += 4) s = __builtin_amdgcn_sdot4(p4[c], 0x01010101, s, false);
    } else {
#pragma unroll 4
      for (int c = lane >> 4; c < cc; c += 4) s += p[c];
    }
  }
  s += __shfl_xor(s, 16);
  s += __shfl_xor(s, 32);
#pragma unroll
  for (int v = 0; v < 4; ++v) out[v] = __shfl(s, 4 * (lane >> 4) + v);
}

template <class DT, int TMW, int TNW>
__device__ __forceinline__ void acc_to_lds(const typename DT::AccV (&acc)[TMW][TNW], int m_base, int n_base,
                                           int m_wr, int n_act, const void* bias, int bias_off, int m_valid,
                                           int act, const Requant& rq, char* so, int rs, int mask_iw, int iy0,
                                           int ix0, int H, int W, ReqCh pc = ReqCh{}, int zin = 0,
                                           const void* wz = nullptr, int wz_cc = 0) {
  const int lane = threadIdx.x & 63;
  const int r = lane & 15, g = lane >> 4;
  constexpr bool kI8 = std::is_same<DT, TI8>::value;
  const uint32_t real0 = kI8 ? (uint32_t)(rq.zp & 0xff) : 0u;  // storage bits of real 0
#pragma unroll
  for (int i = 0; i < TMW; ++i) {
    if (i >= m_wr) continue;
    const int m = m_base + i * 16 + 4 * g;
    typename DT::Acc b[4];
    Requant rqv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {  // unconditional load at a clamped index, then select
      b[v] = load_bias<DT>(bias, bias_off + min(m + v, m_valid - 1));
      if (m + v >= m_valid) b[v] = 0;
      rqv[v] = rq_at(rq, pc, bias_off + min(m + v, m_valid - 1));
    }
    if constexpr (kI8) {
      if (zin != 0) {  // uniform: one zero point per launch
        int32_t rsum[4];
        int8_row_sums((const int8_t*)wz, wz_cc, bias_off + m_base + i * 16, bias_off + m_valid, rsum);
#pragma unroll
        for (int v = 0; v < 4; ++v) b[v] -= zin * rsum[v];
      }
    }
#pragma unroll
    for (int j = 0; j < TNW; ++j) {
      if (j >= n_act) continue;
      const int n = n_base + j * 16 + r;
      uint32_t o[4];
#pragma unroll
      for (int v = 0; v < 4; ++v) o[v] = Fin<DT>::apply(acc[i][j][v], b[v], act, rqv[v]);
      if (mask_iw > 0) {
        const int qy = n / mask_iw, qx = n - qy * mask_iw;
        const int gy = iy0 + qy, gx = ix0 + qx;
        if (!((unsigned)gy < (unsigned)H && (unsigned)gx < (unsigned)W)) o[0] = o[1] = o[2] = o[3] = real0;
      }
      lds_store4<DT>(so + n * rs + m * DT::ELT, o[0], o[1], o[2], o[3]);
    }
  }
}

// LDS tile [TH*TW pixels][cb] (stride rs) -> y at output pixel (oy0, ox0), channels
// [c0, c0+cb) of a tensor with Cy channels and Ho x Wo pixels. vec: Cy*ELT % 16 == 0,
// cb*ELT % 16 == 0 and y 16-byte aligned.
template <class DT>
__device__ __forceinline__ void store_tile(const char* so, int rs, typename DT::T* __restrict__ y, int layout, int n, int Cy,
                           int Ho, int Wo, int oy0, int ox0, int TH, int TW, int c0, int cb, bool vec) {
  using T = typename DT::T;
  constexpr int VE = 16 / DT::ELT;
  if (layout == LAYOUT_NHWC) {
    if (vec) {
      const int nv = cb / VE;
      const int total = TH * TW * nv;
#pragma unroll 1
  for (int i = threadIdx.x; i < total; i += kThreads) {
        const int v = i % nv, p = i / nv;
        const int ty = p / TW, tx = p - ty * TW;
        const int oy = oy0 + ty, ox = ox0 + tx;
        if (oy < Ho && ox < Wo)
          *(u32x4*)(y + (((size_t)n * Ho + oy) * Wo + ox) * Cy + c0 + v * VE) = *(const u32x4*)(so + p * rs + v * 16);
      }
    } else {
      const int total = TH * TW * cb;
#pragma unroll 1
  for (int i = threadIdx.x; i < total; i += kThreads) {
        const int c = i % cb, p = i / cb;
        const int ty = p / TW, tx = p - ty * TW;
        const int oy = oy0 + ty, ox = ox0 + tx;
        if (oy < Ho && ox < Wo) y[(((size_t)n * Ho + oy) * Wo + ox) * Cy + c0 + c] = *(const T*)(so + p * rs + c * DT::ELT);
      }
    }
  } else {
    const int total = cb * TH * TW;
#pragma unroll 1
  for (int i = threadIdx.x; i < total; i += kThreads) {
      const int tx = i % TW;
      const int t = i / TW;
      const int ty = t % TH, c = t / TH;
      const int oy = oy0 + ty, ox = ox0 + tx;
      if (oy < Ho && ox < Wo)
        y[(((size_t)n * Cy + c0 + c) * Ho + oy) * Wo + ox] = *(const T*)(so + (ty * TW + tx) * rs + c * DT::ELT);
    }
  }
}

// Workgroup id -> logical tile id such that consecutive logical ids land on the same XCD
// (workgroups are dispatched round-robin over the 8 XCDs, each with its own L2), so the
// output-channel blocks of one spatial tile and its neighbours share an L2.
__device__ __forceinline__ int xcd_remap(int b, int G) {
  const int q = G / kNumXcd, r = G % kNumXcd;
  const int x = b % kNumXcd;
  return x * q + (x < r ? x : r) + b / kNumXcd;
}


// ------------------------------------------------------------------------------------
// Buffer resources: 32-bit offsets into [base, base + bytes); an offset at or beyond the
// end reads zero (the kernels put kOob where the convolution's zero padding or a ragged
// edge is), and LDS-DMA copies of 16 bytes per lane.
// ------------------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr uint32_t kOob = 0x80000000u;  // buffer offset beyond any record: reads as zero

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from (rsrc + voff) to LDS (wave_base + 16 * lane).
__device__ __forceinline__ void dma16(rsrc_t r, char* wave_base, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)wave_base, 16, voff, 0, 0,
                                           0);
}

}  // namespace fcm
