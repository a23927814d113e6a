// fcm_kernels.h -- the three kernel families and their host launchers (gfx950).
//
//   k_dwpw    DW -> PW module (Sec. III "DWPW") and, with the DW stage off, the
//             layer-by-layer PW kernel. Workgroup = (image, spatial tile, output-channel
//             block). For each input-channel chunk: stage the haloed input window, run the
//             depthwise stencil into an LDS tile, contract it with the pointwise weights on
//             MFMA; the accumulators stay in registers across chunks (output-stationary,
//             Sec. III-A OS-LWS), and only the final output is written.
//   k_pwdw    PW -> DW module (Sec. III "PWDW"/"PWDW_R") and, with the PW stage off, the
//             layer-by-layer DW kernel. Workgroup = (image, spatial tile, intermediate-
//             channel block). The PW is evaluated on the whole haloed window, so halo
//             positions are recomputed by neighbouring tiles (Sec. II-D); positions outside
//             the image are real zero, being the DW's zero padding.
//   k_pwdwpw  PW -> DW -> PW inverted residual in one kernel. Workgroup = (image, spatial
//             tile, output-channel block). The input window is staged once; the
//             intermediate channels stream through LDS in chunks, each chunk being expanded
//             (MFMA), filtered (DW) and projected (MFMA) into output accumulators that stay
//             in registers.
#pragma once

#include "fcm_device.h"

namespace fcm {

template <class DT, int K, int S, bool HAS_DW, int PMAX, int MMAX, int WM, int R>
__global__ __launch_bounds__(kThreads) void k_dwpw(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  constexpr int WN = 4 / WM;
  constexpr int TMW = MMAX / 16 / WM;
  constexpr int TNW = PMAX / 16 / WN;
  static_assert(TMW * WM * 16 == MMAX && TNW * WN * 16 == PMAX, "wave tiling");
  const LdsLayout& L = a.L;

  const int G = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  const int lid = xcd_remap(blockIdx.x, G);
  const int cob = lid % a.n_cb;
  int t = lid / a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;

  const int oy0 = ty * a.TH, ox0 = tx * a.TW;
  const int iy0 = HAS_DW ? oy0 * S - a.pad : oy0;
  const int ix0 = HAS_DW ? ox0 * S - a.pad : ox0;
  const int IH = HAS_DW ? (a.TH - 1) * S + K : a.TH;
  const int IW = HAS_DW ? (a.TW - 1) * S + K : a.TW;
  const int co0 = cob * a.COB;
  const int cob_eff = min(a.COB, a.Co - co0);

  const int wave = threadIdx.x >> 6, wm = wave / WN, wn = wave % WN;
  const int m_tiles = ceil_div(cob_eff, 16), n_tiles = ceil_div(a.TH * a.TW, 16);
  const int m_act = max(0, min(TMW, m_tiles - wm * TMW));
  const int n_act = max(0, min(TNW, n_tiles - wn * TNW));

  const T* x = (const T*)a.x;
  const T* wd = (const T*)a.w1;
  const T* wp = (const T*)(HAS_DW ? a.w2 : a.w1);
  const void* bp = HAS_DW ? a.b2 : a.b1;
  const int act_pw = HAS_DW ? a.act[1] : a.act[0];
  const Requant rq_pw = HAS_DW ? a.rq[1] : a.rq[0];
  const bool vec_wp = HAS_DW ? a.vec_w2 : a.vec_w1;

  AccV acc[TMW][TNW];
#pragma unroll
  for (int i = 0; i < TMW; ++i)
#pragma unroll
    for (int j = 0; j < TNW; ++j) acc[i][j] = AccV{0, 0, 0, 0};

  for (int c0 = 0; c0 < a.Ci; c0 += a.CB) {
    stage_chunk<DT, HAS_DW ? K : 0>(smem, x, a.layout, a.vec_x, n, a.Ci, a.H, a.W, iy0, ix0, IH, IW, c0, a.CB,
                                    L.ps_in, L.off_in, wp, vec_wp, a.Co, a.Ci, co0, m_tiles * 16, L.rs_w, L.off_w,
                                    wd, a.b1, a.Ci, c0, a.CB, L.off_wd, HAS_DW ? zp_fill<DT>(a.zin[0]) : 0u);
    __syncthreads();
    const char* B = smem + L.off_in;
    int bs = L.ps_in;
    if constexpr (HAS_DW) {
      dw_compute<DT, K, S, R>(smem + L.off_in, L.ps_in, IW, (const Acc*)(smem + L.off_wd), a.CB, a.TH, a.TW,
                              a.act[0], a.rq[0], smem + L.off_d, L.rs_d, ReqCh{a.rqc[0], a.Ci}, c0, a.Ci,
                              a.zin[0]);
      __syncthreads();
      B = smem + L.off_d;
      bs = L.rs_d;
    }
    mma_chunk<DT, TMW, TNW>(acc, smem + L.off_w, L.rs_w, B, bs, a.CB, wm * TMW * 16, wn * TNW * 16, m_act, n_act);
    __syncthreads();
  }

  acc_to_lds<DT, TMW, TNW>(acc, wm * TMW * 16, wn * TNW * 16, m_act, n_act, bp, co0, cob_eff, act_pw, rq_pw,
                           smem + L.off_out, L.rs_out, 0, 0, 0, 0, 0, ReqCh{a.rqc[HAS_DW ? 1 : 0], a.Co},
                           a.zin[HAS_DW ? 1 : 0], wp, a.Ci);
  __syncthreads();
  store_tile<DT>(smem + L.off_out, L.rs_out, (T*)a.y, a.layout, n, a.Co, a.Ho, a.Wo, oy0, ox0, a.TH, a.TW, co0,
                 cob_eff, a.vec_y && ((cob_eff * DT::ELT) % 16 == 0));
}

template <class DT, int K, int S, bool HAS_PW, int QMAX, int MMAX, int WM, int R>
__global__ __launch_bounds__(kThreads) void k_pwdw(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  const LdsLayout& L = a.L;

  const int G = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  const int lid = xcd_remap(blockIdx.x, G);
  const int mb = lid % a.n_cb;
  int t = lid / a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;

  const int oy0 = ty * a.TH, ox0 = tx * a.TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const int IH = (a.TH - 1) * S + K, IW = (a.TW - 1) * S + K;
  const int MB = a.COB;
  const int m0 = mb * MB;
  const int mb_eff = min(MB, a.Cm - m0);
  const T* x = (const T*)a.x;

  if constexpr (HAS_PW) {
    constexpr int WN = 4 / WM;
    constexpr int TMW = MMAX / 16 / WM;
    constexpr int TNW = QMAX / 16 / WN;
    static_assert(TMW * WM * 16 == MMAX && TNW * WN * 16 == QMAX, "wave tiling");
    const int wave = threadIdx.x >> 6, wm = wave / WN, wn = wave % WN;
    const int m_tiles = ceil_div(mb_eff, 16), q_tiles = ceil_div(IH * IW, 16);
    const int m_act = max(0, min(TMW, m_tiles - wm * TMW));
    const int n_act = max(0, min(TNW, q_tiles - wn * TNW));
    AccV acc[TMW][TNW];
#pragma unroll
    for (int i = 0; i < TMW; ++i)
#pragma unroll
      for (int j = 0; j < TNW; ++j) acc[i][j] = AccV{0, 0, 0, 0};
    for (int c0 = 0; c0 < a.Ci; c0 += a.CB) {
      stage_chunk<DT, 0>(smem, x, a.layout, a.vec_x, n, a.Ci, a.H, a.W, iy0, ix0, IH, IW, c0, a.CB, L.ps_in,
                         L.off_in, (const T*)a.w1, a.vec_w1, a.Cm, a.Ci, m0, m_tiles * 16, L.rs_w, L.off_w, nullptr,
                         nullptr, 0, 0, 0, 0);
      __syncthreads();
      mma_chunk<DT, TMW, TNW>(acc, smem + L.off_w, L.rs_w, smem + L.off_in, L.ps_in, a.CB, wm * TMW * 16,
                              wn * TNW * 16, m_act, n_act);
      __syncthreads();
    }
    // PW output over the haloed window -> E [Q][MB]; zero outside the image.
    acc_to_lds<DT, TMW, TNW>(acc, wm * TMW * 16, wn * TNW * 16, m_act, n_act, a.b1, m0, mb_eff, a.act[0], a.rq[0],
                             smem + L.off_e, L.rs_e, IW, iy0, ix0, a.H, a.W, ReqCh{a.rqc[0], a.Cm}, a.zin[0], a.w1,
                             a.Ci);
    staged_copy<kBatch>(smem, (K * K + 1) * MB, DwWeights<DT, K>{(const T*)a.w2, a.b2, a.Cm, m0, MB, L.off_wd});
  } else {
    stage_chunk<DT, K>(smem, x, a.layout, a.vec_x, n, a.Cm, a.H, a.W, iy0, ix0, IH, IW, m0, MB, L.rs_e, L.off_e,
                       nullptr, false, 0, 0, 0, 0, 0, 0, (const T*)a.w1, a.b1, a.Cm, m0, MB, L.off_wd,
                       zp_fill<DT>(a.zin[0]));
  }
  __syncthreads();
  const int act_dw = HAS_PW ? a.act[1] : a.act[0];
  const Requant rq_dw = HAS_PW ? a.rq[1] : a.rq[0];
  dw_compute<DT, K, S, R>(smem + L.off_e, L.rs_e, IW, (const Acc*)(smem + L.off_wd), MB, a.TH, a.TW, act_dw, rq_dw,
                          smem + L.off_out, L.rs_out, ReqCh{a.rqc[HAS_PW ? 1 : 0], a.Cm}, m0, a.Cm,
                          a.zin[HAS_PW ? 1 : 0]);
  __syncthreads();
  store_tile<DT>(smem + L.off_out, L.rs_out, (T*)a.y, a.layout, n, a.Cm, a.Ho, a.Wo, oy0, ox0, a.TH, a.TW, m0, mb_eff,
                 a.vec_y && ((mb_eff * DT::ELT) % 16 == 0));
}

// MIDDW false: the PW -> PW module (K = S = 1, pad 0, window = tile): no depthwise stage,
// the second PW reads the first's output chunk straight from LDS; its weights, bias and
// epilogue are stage 1 (w2, b2, act[1], rq[1]) instead of stage 2.
template <class DT, int K, int S, int QMAX, int MBMAX, int WM1, int OMAX, int PMAX, int WM2, int R, bool MIDDW>
__global__ __launch_bounds__(kThreads) void k_pwdwpw(KArgs a) {
  extern __shared__ __align__(16) char smem[];
  using T = typename DT::T;
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  constexpr int WN1 = 4 / WM1, TMW1 = MBMAX / 16 / WM1, TNW1 = QMAX / 16 / WN1;
  constexpr int WN2 = 4 / WM2, TMW2 = OMAX / 16 / WM2, TNW2 = PMAX / 16 / WN2;
  static_assert(TMW1 * WM1 * 16 == MBMAX && TNW1 * WN1 * 16 == QMAX, "wave tiling 1");
  static_assert(TMW2 * WM2 * 16 == OMAX && TNW2 * WN2 * 16 == PMAX, "wave tiling 2");
  const LdsLayout& L = a.L;

  const int G = a.N * a.tiles_y * a.tiles_x * a.n_cb;
  const int lid = xcd_remap(blockIdx.x, G);
  const int cob = lid % a.n_cb;
  int t = lid / a.n_cb;
  const int tx = t % a.tiles_x;
  t /= a.tiles_x;
  const int ty = t % a.tiles_y, n = t / a.tiles_y;

  const int oy0 = ty * a.TH, ox0 = tx * a.TW;
  const int iy0 = oy0 * S - a.pad, ix0 = ox0 * S - a.pad;
  const int IH = (a.TH - 1) * S + K, IW = (a.TW - 1) * S + K;
  const int CIP = round_up(a.Ci, DT::KB);
  const int MB = a.CB;  // intermediate chunk
  const int co0 = cob * a.COB, cob_eff = min(a.COB, a.Co - co0);

  const int wave = threadIdx.x >> 6;
  const int wm1 = wave / WN1, wn1 = wave % WN1, wm2 = wave / WN2, wn2 = wave % WN2;
  const int q_tiles = ceil_div(IH * IW, 16), p_tiles = ceil_div(a.TH * a.TW, 16);
  const int o_tiles = ceil_div(cob_eff, 16);
  const int n_act1 = max(0, min(TNW1, q_tiles - wn1 * TNW1));
  const int m_act2 = max(0, min(TMW2, o_tiles - wm2 * TMW2));
  const int n_act2 = max(0, min(TNW2, p_tiles - wn2 * TNW2));

  const T* x = (const T*)a.x;
  static_assert(MIDDW || (K == 1 && S == 1), "PW -> PW has no depthwise geometry");
  const T* w_last = (const T*)(MIDDW ? a.w3 : a.w2);  // weights of the last PW
  stage_chunk<DT, 0>(smem, x, a.layout, a.vec_x, n, a.Ci, a.H, a.W, iy0, ix0, IH, IW, 0, CIP, L.ps_in, L.off_in,
                     nullptr, false, 0, 0, 0, 0, 0, 0, nullptr, nullptr, 0, 0, 0, 0);

  AccV acc2[TMW2][TNW2];
#pragma unroll
  for (int i = 0; i < TMW2; ++i)
#pragma unroll
    for (int j = 0; j < TNW2; ++j) acc2[i][j] = AccV{0, 0, 0, 0};

  for (int m0 = 0; m0 < a.Cm; m0 += MB) {
    const int mb_eff = min(MB, a.Cm - m0);
    const int m_tiles = ceil_div(mb_eff, 16);
    const int m_act1 = max(0, min(TMW1, m_tiles - wm1 * TMW1));
    if constexpr (!MIDDW) {
      constexpr int VE = 16 / DT::ELT;
      if (a.vec_w1 && a.vec_w3) {
        staged_copy<kBatch>(smem, m_tiles * 16 * CIP / VE,
                            rows_vec<DT>((const T*)a.w1, a.Cm, a.Ci, m0, 0, CIP, L.rs_w, L.off_w),
                            o_tiles * 16 * MB / VE, rows_vec<DT>(w_last, a.Co, a.Cm, co0, m0, MB, L.rs_w2, L.off_w2), 0,
                            NullLoader{});
      } else {
        stage_rows<DT>(smem, (const T*)a.w1, a.vec_w1, a.Cm, a.Ci, m0, m_tiles * 16, 0, CIP, L.rs_w, L.off_w);
        stage_rows<DT>(smem, w_last, a.vec_w3, a.Co, a.Cm, co0, o_tiles * 16, m0, MB, L.rs_w2, L.off_w2);
      }
    } else {
      constexpr int VE = 16 / DT::ELT;
      const DwWeights<DT, K> dww{(const T*)a.w2, a.b2, a.Cm, m0, MB, L.off_wd};
      if (a.vec_w1 && a.vec_w3) {
        staged_copy<kBatch>(smem, m_tiles * 16 * CIP / VE,
                            rows_vec<DT>((const T*)a.w1, a.Cm, a.Ci, m0, 0, CIP, L.rs_w, L.off_w),
                            (K * K + 1) * MB, dww, o_tiles * 16 * MB / VE,
                            rows_vec<DT>((const T*)a.w3, a.Co, a.Cm, co0, m0, MB, L.rs_w2, L.off_w2));
      } else {
        stage_rows<DT>(smem, (const T*)a.w1, a.vec_w1, a.Cm, a.Ci, m0, m_tiles * 16, 0, CIP, L.rs_w, L.off_w);
        staged_copy<kBatch>(smem, (K * K + 1) * MB, dww);
        stage_rows<DT>(smem, (const T*)a.w3, a.vec_w3, a.Co, a.Cm, co0, o_tiles * 16, m0, MB, L.rs_w2, L.off_w2);
      }
    }
    __syncthreads();
    {
      AccV acc1[TMW1][TNW1];
#pragma unroll
      for (int i = 0; i < TMW1; ++i)
#pragma unroll
        for (int j = 0; j < TNW1; ++j) acc1[i][j] = AccV{0, 0, 0, 0};
      mma_chunk<DT, TMW1, TNW1>(acc1, smem + L.off_w, L.rs_w, smem + L.off_in, L.ps_in, CIP, wm1 * TMW1 * 16,
                                wn1 * TNW1 * 16, m_act1, n_act1);
      // Every channel of the chunk is written (zeros beyond mb_eff), so the DW and the
      // projection below never read uninitialised LDS.
      const int m_wr1 = max(0, min(TMW1, MB / 16 - wm1 * TMW1));
      acc_to_lds<DT, TMW1, TNW1>(acc1, wm1 * TMW1 * 16, wn1 * TNW1 * 16, m_wr1, n_act1, a.b1, m0, mb_eff, a.act[0],
                                 a.rq[0], smem + L.off_e, L.rs_e, IW, iy0, ix0, a.H, a.W, ReqCh{a.rqc[0], a.Cm},
                                 a.zin[0], a.w1, a.Ci);
    }
    __syncthreads();
    if constexpr (MIDDW) {
      dw_compute<DT, K, S, R>(smem + L.off_e, L.rs_e, IW, (const Acc*)(smem + L.off_wd), MB, a.TH, a.TW, a.act[1],
                              a.rq[1], smem + L.off_d, L.rs_d, ReqCh{a.rqc[1], a.Cm}, m0, a.Cm, a.zin[1]);
      __syncthreads();
      mma_chunk<DT, TMW2, TNW2>(acc2, smem + L.off_w2, L.rs_w2, smem + L.off_d, L.rs_d, MB, wm2 * TMW2 * 16,
                                wn2 * TNW2 * 16, m_act2, n_act2);
    } else {
      // window = tile: the first PW's output positions are the output pixels
      mma_chunk<DT, TMW2, TNW2>(acc2, smem + L.off_w2, L.rs_w2, smem + L.off_e, L.rs_e, MB, wm2 * TMW2 * 16,
                                wn2 * TNW2 * 16, m_act2, n_act2);
    }
    __syncthreads();
  }

  constexpr int LAST = MIDDW ? 2 : 1;  // stage index of the last PW
  acc_to_lds<DT, TMW2, TNW2>(acc2, wm2 * TMW2 * 16, wn2 * TNW2 * 16, m_act2, n_act2, MIDDW ? a.b3 : a.b2, co0,
                             cob_eff, a.act[LAST], a.rq[LAST], smem + L.off_out, L.rs_out, 0, 0, 0, 0, 0,
                             ReqCh{a.rqc[LAST], a.Co}, a.zin[LAST], w_last, a.Cm);
  __syncthreads();
  store_tile<DT>(smem + L.off_out, L.rs_out, (T*)a.y, a.layout, n, a.Co, a.Ho, a.Wo, oy0, ox0, a.TH, a.TW, co0,
                 cob_eff, a.vec_y && ((cob_eff * DT::ELT) % 16 == 0));
}

// ------------------------------------------------------------------------------------
// Host launchers
// ------------------------------------------------------------------------------------
// Launch a kernel taking one KArgs by value; returns this launch's own status (not an
// error left behind by an earlier runtime call of the process).
inline int launch_args(const void* fn, int grid, int threads, int lds, void* stream, const KArgs& a) {
  KArgs copy = a;
  void* args[] = {(void*)&copy};
  return (int)hipLaunchKernel(fn, dim3(grid), dim3(threads), args, (size_t)lds, (hipStream_t)stream);
}

template <class Kern>
inline int launch_kernel(Kern fn, const KArgs& a, int grid, void* stream) {
  if (a.L.bytes > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, a.L.bytes);
    if (e != hipSuccess) return (int)e;
  }
  return launch_args((const void*)fn, grid, kThreads, a.L.bytes, stream, a);
}

template <class DT, int K, int S, bool HAS_DW, int PMAX, int MMAX, int WM, int R>
int launch_dwpw(const KArgs& a, int grid, void* stream) {
  return launch_kernel(k_dwpw<DT, K, S, HAS_DW, PMAX, MMAX, WM, R>, a, grid, stream);
}

template <class DT, int K, int S, bool HAS_PW, int QMAX, int MMAX, int WM, int R>
int launch_pwdw(const KArgs& a, int grid, void* stream) {
  return launch_kernel(k_pwdw<DT, K, S, HAS_PW, QMAX, MMAX, WM, R>, a, grid, stream);
}

template <class DT, int K, int S, int QMAX, int MBMAX, int WM1, int OMAX, int PMAX, int WM2, int R, bool MIDDW>
int launch_pwdwpw(const KArgs& a, int grid, void* stream) {
  return launch_kernel(k_pwdwpw<DT, K, S, QMAX, MBMAX, WM1, OMAX, PMAX, WM2, R, MIDDW>, a, grid, stream);
}

template <class DT>
constexpr int dtype_elt() {
  return DT::ELT;
}

template <class DT>
constexpr int dtype_id() {
  return std::is_same<DT, TF32>::value ? DT_F32 : (std::is_same<DT, TBF16>::value ? DT_BF16 : DT_I8);
}

}  // namespace fcm
