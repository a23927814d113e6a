// fcm_kernels_v6.h -- whole-module fp32 kernels for small batches (gfx950).
//
// k_small6<MODE, K, S, TH, TW>
//   One workgroup (four waves) computes one TH x TW output tile of one image through
//   every stage of the module and every channel: the DW -> PW module (Sec. III "DWPW"),
//   the PW -> DW module with the halo recomputed (Sec. II-D, III "PWDW_R") and the
//   PW -> DW -> PW inverted residual. Batch-1 layers have a few hundred tiles at most, so
//   what bounds them is the number of dependent steps, not bandwidth: the kernel stages
//   the haloed input window and all weights and biases in LDS with one round of loads,
//   then runs the stages back to back on LDS-resident operands with a barrier between
//   stages, and writes only the module's output.
//
//   Pointwise stages run on fp32 MFMA (16x16x4, four k-steps per 16-channel chunk) with
//   the weights as the A operand ([out][in] rows, as given) and the activations as the B
//   operand ([position][channel] rows: the window is staged transposed, the depthwise
//   output is written transposed). The first PW of PW -> DW covers the whole haloed
//   window; window positions outside the image are set to zero after its epilogue, which
//   is the depthwise zero padding of the intermediate. The depthwise stencil runs on the
//   vector ALU, one (channel, pixel) output per thread and step. When the last PW has
//   fewer 16 x 16 output tiles than waves, the waves split its channel chunks and add
//   their partial sums through LDS in a fixed order.
//
//   Channel counts are run-time values bounded by the LDS the planner grants (lds6); the
//   input and depthwise channel counts are multiples of four and the weights 16-byte
//   aligned, so that weights move as flat 16-byte copies and pointwise rows are 16-byte
//   aligned in LDS. Accumulation is fp32 throughout.
#pragma once

#include "fcm_kernels.h"

namespace fcm {

constexpr int kThreads6 = 256;

// Division by a run-time divisor d in [1, 2^20) of a non-negative i < 2^24 through a float
// reciprocal, corrected to the exact quotient.
struct Div6 {
  int d;
  float inv;
  __device__ explicit Div6(int d_) : d(d_), inv(1.0f / (float)d_) {}
  __device__ __forceinline__ int div(int i) const {
    int q = (int)((float)i * inv);
    if (q * d > i) --q;
    if ((q + 1) * d <= i) ++q;
    return q;
  }
};

// Flat copy of an array of n floats into LDS, in two steps so that every array's loads
// are in flight together: the constructor issues this thread's first NV loads, commit()
// writes them, copies what is left beyond the first round and zeroes `tail` floats after
// the array (src NULL: zeros throughout). VEC: 16-byte loads (src 16-byte aligned, n a
// multiple of 4); else element loads.
template <int NV, bool VEC>
struct Flat6 {
  using V = typename std::conditional<VEC, f32x4, float>::type;
  static constexpr int W = VEC ? 4 : 1;
  V v[NV];
  float* dst;
  const V* src;
  int nv, n, tail;
  __device__ Flat6(float* dst_, const float* src_, int n_, int tail_)
      : dst(dst_), src((const V*)src_), nv(n_ / W), n(n_), tail(tail_) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int e = tid + j * kThreads6;
      v[j] = (src && e < nv) ? src[e] : V{};
    }
  }
  __device__ void commit() const {
    const int tid = threadIdx.x;
    V* d = (V*)dst;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int e = tid + j * kThreads6;
      if (e < nv) d[e] = v[j];
    }
    for (int e = tid + NV * kThreads6; e < nv; e += kThreads6) d[e] = src ? src[e] : V{};
    for (int e = tid; e < tail; e += kThreads6) dst[n + e] = 0.0f;
  }
};

// Activation as a clamp to [lo, hi] (none: [-inf, inf], ReLU: [0, inf], ReLU6: [0, 6]),
// two branch-free instructions per value.
struct Clamp6 {
  float lo, hi;
  __device__ explicit Clamp6(int act)
      : lo(act == ACT_NONE ? -INFINITY : 0.0f), hi(act == ACT_RELU6 ? 6.0f : INFINITY) {}
  __device__ __forceinline__ float operator()(float v) const { return fminf(fmaxf(v, lo), hi); }
};

template <int MODE, int K, int S, int TH, int TW>
__global__ __launch_bounds__(kThreads6) void k_small6(KArgs a) {
  extern __shared__ __align__(16) float sm6[];
  constexpr bool PW1 = MODE != M6_DWPW;  // a PW stage before the depthwise one
  constexpr bool PW2 = MODE != M6_PWDW;  // a PW stage after it
  constexpr int P = TH * TW, KK = K * K;
  constexpr int IH = (TH - 1) * S + K, IW = (TW - 1) * S + K, NQ = IH * IW;
  constexpr int NQT = (NQ + 15) / 16;   // 16-position tiles of the window
  constexpr int NQP = NQT * 16;         // row pitch of the first PW's output
  constexpr int NPT = (P + 15) / 16;    // 16-pixel tiles of the output tile
  constexpr int NVX = 8;                // first-round window loads per thread
  static_assert(NPT <= 4 && (!PW1 || NQT <= 8), "tile");
  const Lds6 L = lds6(MODE, K, S, TH, TW, a.Ci, a.Cm, a.Co);
  const int ci = a.Ci;
  const int cd = PW1 ? a.Cm : a.Ci;  // depthwise channels
  const int co = PW2 ? a.Co : a.Cm;  // output channels
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, g = lane >> 4;

  int t = blockIdx.x;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;
  const int oy0 = ty * TH, ox0 = tx * TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const bool nchw = a.layout == 0;

  float* xs = sm6 + L.xs;
  float* w1s = sm6 + L.w1;
  float* b1s = sm6 + L.b1;
  float* wds = sm6 + L.wd;
  float* bds = sm6 + L.bd;
  float* es = sm6 + L.es;
  float* ds = sm6 + L.ds;
  float* w2s = sm6 + L.w2;
  float* b2s = sm6 + L.b2;
  float* red = sm6 + L.red;

  const float* wpw1 = (const float*)a.w1;
  const float* bpw1 = (const float*)a.b1;
  const float* wdw = (const float*)(PW1 ? a.w2 : a.w1);
  const float* bdw = (const float*)(PW1 ? a.b2 : a.b1);
  const float* wpw2 = (const float*)(MODE == M6_DWPW ? a.w2 : a.w3);
  const float* bpw2 = (const float*)(MODE == M6_DWPW ? a.b2 : a.b3);
  const Clamp6 act1(a.act[0]);
  const Clamp6 actd(a.act[PW1 ? 1 : 0]);
  const Clamp6 act2(a.act[MODE == M6_DWPW ? 1 : 2]);

  // ---- loads: every thread issues its first-round loads of the window (transposed, zero
  // outside the image and beyond the channels) and of every weight and bias array before
  // it writes any of them to LDS ----
  {
    const float* xi = (const float*)a.x + (size_t)n * a.H * a.W * ci;
    const int cip = L.cip;
    const Div6 dcip(cip);
    const int nx = NQ * cip;
    auto x_at = [&](int e, int& dst) {
      int c, q;
      if (nchw) {
        c = e / NQ;
        q = e - c * NQ;
      } else {
        q = dcip.div(e);
        c = e - q * cip;
      }
      const int qy = q / IW, qx = q - qy * IW;
      const int gy = iy0 + qy, gx = ix0 + qx;
      dst = q * L.px + c;
      float v = 0.0f;
      if (e < nx && c < ci && (unsigned)gy < (unsigned)a.H && (unsigned)gx < (unsigned)a.W)
        v = nchw ? xi[((size_t)c * a.H + gy) * a.W + gx] : xi[((size_t)gy * a.W + gx) * ci + c];
      return v;
    };
    float xv[NVX];
    int xd[NVX];
#pragma unroll
    for (int j = 0; j < NVX; ++j) xv[j] = x_at(tid + j * kThreads6, xd[j]);
    // weights and biases as stored ([out][in] rows); the pointwise rows are read a whole
    // 16-channel chunk at a time, so each matrix is followed by 16 zeros (a row's reads
    // beyond its channels meet zeros of the other operand)
    const Flat6<4, true> s_w1(w1s, PW1 ? wpw1 : nullptr, PW1 ? cd * ci : 0, PW1 ? 16 : 0);
    const Flat6<1, false> s_b1(b1s, PW1 ? bpw1 : nullptr, PW1 ? cd : 0, 0);
    const Flat6<2, true> s_wd(wds, wdw, cd * KK, 0);
    const Flat6<1, false> s_bd(bds, bdw, cd, 0);
    const Flat6<4, true> s_w2(w2s, PW2 ? wpw2 : nullptr, PW2 ? co * cd : 0, PW2 ? 16 : 0);
    const Flat6<1, false> s_b2(b2s, PW2 ? bpw2 : nullptr, PW2 ? co : 0, 0);
#pragma unroll
    for (int j = 0; j < NVX; ++j)
      if (tid + j * kThreads6 < nx) xs[xd[j]] = xv[j];
    for (int e = tid + NVX * kThreads6; e < nx; e += kThreads6) {
      int dst;
      const float v = x_at(e, dst);
      xs[dst] = v;
    }
    if constexpr (PW1) {
      s_w1.commit();
      s_b1.commit();
    }
    s_wd.commit();
    s_bd.commit();
    if constexpr (PW2) {
      s_w2.commit();
      s_b2.commit();
      // depthwise output channels [cd, cdp) of every pixel: zero (the last PW reads whole
      // 16-channel chunks)
      const int padc = L.cdp - cd;
      if (padc > 0) {
        for (int e = tid; e < P * padc; e += kThreads6) {
          const int p = e / padc;
          ds[p * L.pd + cd + (e - p * padc)] = 0.0f;
        }
      }
    }
  }
  __syncthreads();

  // ---- first PW over the haloed window: E[m][q] = act(W1[m] . X[q] + b1[m]), zero at
  // window positions outside the image. A wave takes a 16-channel tile of every window
  // position at a time (independent accumulators). ----
  if constexpr (PW1) {
    const int m1t = L.cmp / 16;
    bool inside[NQT];  // this lane's window position of each 16-position tile lies in the image
#pragma unroll
    for (int j = 0; j < NQT; ++j) {
      const int q = j * 16 + r16, qy = q / IW, qx = q - qy * IW;
      inside[j] = q < NQ && (unsigned)(iy0 + qy) < (unsigned)a.H && (unsigned)(ix0 + qx) < (unsigned)a.W;
    }
    for (int mt = wave; mt < m1t; mt += 4) {
      f32x4 acc[1][NQT];
#pragma unroll
      for (int j = 0; j < NQT; ++j) acc[0][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      mma_chunk<TF32, 1, NQT>(acc, (const char*)(w1s + mt * 16 * ci), ci * 4, (const char*)xs, L.px * 4, L.cip, 0,
                              0, 1, NQT);
      const f32x4 bb = *(const f32x4*)(b1s + mt * 16 + 4 * g);
      float* er = es + (mt * 16 + 4 * g) * NQP + r16;
#pragma unroll
      for (int j = 0; j < NQT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) er[v * NQP + j * 16] = inside[j] ? act1(acc[0][j][v] + bb[v]) : 0.0f;
    }
    __syncthreads();
  }

  // ---- depthwise stencil: a thread computes one output row of one channel, the K input
  // rows it needs held in registers ----
  for (int e = tid; e < cd * TH; e += kThreads6) {
    const int c = e / TH, py = e - c * TH;
    float w[KK];
#pragma unroll
    for (int k = 0; k < KK; ++k) w[k] = wds[c * KK + k];
    float acc[TW];
#pragma unroll
    for (int x = 0; x < TW; ++x) acc[x] = bds[c];
#pragma unroll
    for (int ky = 0; ky < K; ++ky) {
      float in[IW];
      const int q0 = (py * S + ky) * IW;
#pragma unroll
      for (int x = 0; x < IW; ++x) in[x] = PW1 ? es[c * NQP + q0 + x] : xs[(q0 + x) * L.px + c];
#pragma unroll
      for (int x = 0; x < TW; ++x)
#pragma unroll
        for (int kx = 0; kx < K; ++kx) acc[x] = fmaf(w[ky * K + kx], in[x * S + kx], acc[x]);
    }
#pragma unroll
    for (int x = 0; x < TW; ++x) {
      const float d = actd(acc[x]);
      const int p = py * TW + x;
      if constexpr (PW2) {
        ds[p * L.pd + c] = d;
      } else {
        const int oy = oy0 + py, ox = ox0 + x;
        if (oy < a.Ho && ox < a.Wo) {
          float* y = (float*)a.y;
          if (nchw)
            y[(((size_t)n * co + c) * a.Ho + oy) * a.Wo + ox] = d;
          else
            y[(((size_t)n * a.Ho + oy) * a.Wo + ox) * co + c] = d;
        }
      }
    }
  }

  // ---- last PW: y[m][p] = act(W2[m] . D[p] + b2[m]). A work unit is a pair of
  // 16-channel output tiles over a range of channel chunks; with few pairs the waves
  // split the chunks and add their partial sums through LDS in a fixed order. ----
  if constexpr (PW2) {
    __syncthreads();
    const int m2t = L.cop / 16, kc = L.cdp / 16;
    const int npair = (m2t + 1) >> 1;
    int nsplit = 4 / npair;
    nsplit = nsplit < 1 ? 1 : (nsplit > kc ? kc : nsplit);
    float* y = (float*)a.y;
    const size_t plane = (size_t)a.Ho * a.Wo;
    // this lane's output pixel of each 16-pixel tile: offset within an output channel
    // plane (NCHW) or pixel row (NHWC), or -1 outside the image or the tile
    int poff[NPT];
#pragma unroll
    for (int j = 0; j < NPT; ++j) {
      const int p = j * 16 + r16, py = p / TW, px = p - py * TW;
      const int oy = oy0 + py, ox = ox0 + px;
      const bool ok = p < P && oy < a.Ho && ox < a.Wo;
      poff[j] = ok ? (nchw ? oy * a.Wo + ox : (oy * a.Wo + ox) * co) : -1;
    }
    float* yn = y + (size_t)n * co * plane;
    auto store4 = [&](int m0, int j, const f32x4& v4) {  // channels m0 .. m0 + 3 of tile j
      if (poff[j] < 0) return;
      const f32x4 bb = *(const f32x4*)(b2s + m0);
#pragma unroll
      for (int v = 0; v < 4; ++v)
        if (m0 + v < co) yn[nchw ? (size_t)(m0 + v) * plane + poff[j] : (size_t)poff[j] + m0 + v] = act2(v4[v] + bb[v]);
    };
    for (int u = wave; u < npair * nsplit; u += 4) {
      const int pr = u / nsplit, sp = u - pr * nsplit;
      const int k0 = sp * kc / nsplit, k1 = (sp + 1) * kc / nsplit;
      const int mact = m2t - 2 * pr < 2 ? 1 : 2;
      f32x4 acc[2][NPT];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NPT; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
      mma_chunk<TF32, 2, NPT>(acc, (const char*)(w2s + 2 * pr * 16 * cd + k0 * 16), cd * 4,
                              (const char*)(ds + k0 * 16), L.pd * 4, (k1 - k0) * 16, 0, 0, mact, NPT);
      if (nsplit == 1) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          if (i < mact)
#pragma unroll
            for (int j = 0; j < NPT; ++j) store4((2 * pr + i) * 16 + 4 * g, j, acc[i][j]);
      } else {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < NPT; ++j)
            *(f32x4*)(red + (((sp * npair + pr) * 2 + i) * NPT + j) * 256 + lane * 4) = acc[i][j];
      }
    }
    if (nsplit > 1) {
      __syncthreads();
      // one lane per (pair, tile i, pixel tile j, lane): the partial sums in split order
      for (int e = tid; e < npair * 2 * NPT * 64; e += kThreads6) {
        const int l = e & 63, r = e >> 6;
        const int j = r % NPT, i = (r / NPT) & 1, pr = r / (2 * NPT);
        if (2 * pr + i >= m2t) continue;
        f32x4 s4 = *(const f32x4*)(red + ((pr * 2 + i) * NPT + j) * 256 + l * 4);
        for (int sp = 1; sp < nsplit; ++sp) {
          const f32x4 o = *(const f32x4*)(red + (((sp * npair + pr) * 2 + i) * NPT + j) * 256 + l * 4);
#pragma unroll
          for (int v = 0; v < 4; ++v) s4[v] += o[v];
        }
        // lane l's rows and column within the tile
        const int m0 = (2 * pr + i) * 16 + 4 * (l >> 4);
        const int p = j * 16 + (l & 15), py = p / TW, px = p - py * TW;
        const int oy = oy0 + py, ox = ox0 + px;
        if (p < P && oy < a.Ho && ox < a.Wo) {
          const f32x4 bb = *(const f32x4*)(b2s + m0);
          const int po = nchw ? oy * a.Wo + ox : (oy * a.Wo + ox) * co;
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (m0 + v < co) yn[nchw ? (size_t)(m0 + v) * plane + po : (size_t)po + m0 + v] = act2(s4[v] + bb[v]);
        }
      }
    }
  }
}

template <int MODE, int K, int S, int TH, int TW>
int launch_small6(const KArgs& a, int grid, void* stream) {
  auto fn = k_small6<MODE, K, S, TH, TW>;
  if (a.L.bytes > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, a.L.bytes);
    if (e != hipSuccess) return (int)e;
  }
  (void)grid;
  return launch_args((const void*)fn, a.N * a.tiles_y * a.tiles_x, kThreads6, a.L.bytes, stream, a);
}

}  // namespace fcm
