// fcm_kernels_v4.h -- PW -> PW module for gfx950 with the intermediate handed from the
// first pointwise convolution to the second in registers (NHWC).
//
// k_pwpw4<DT, KS, CT, PB, VEC>
//   A workgroup is four waves. A pixel group (PB blocks of 16 pixels) is computed against
//   every output channel (up to 16*CT) by S = 1, 2 or 4 of them (a.splits): the
//   intermediate is cut into chunks of 64 bytes (one MFMA k-step of the second
//   convolution) and wave j of the S takes chunks j, j+S, j+2S, ... A workgroup covers
//   4/S neighbouring pixel groups; with S = 1 its four waves are independent (no LDS, no
//   barrier) and their weight loads are the same addresses, served by the CU's cache.
//
//   For each chunk the wave loads, straight into MFMA operand registers, the first
//   convolution's weight rows of the chunk and the chunk's 64-byte column slice of the
//   second convolution's weights. The first convolution's weight rows are taken in a
//   permuted order: MFMA row i of M-tile t is intermediate channel
//   m0 + (16/elt)*(i/4) + 4t + i%4, so the accumulator lane (pixel l%16, group l/16), which
//   holds rows 4*(l/16)..+3 of every tile, ends up with the 16 contiguous bytes of channels
//   m0 + (16/elt)*(l/16) + [0, 16/elt) after +bias, activation and the cast (int8:
//   requantisation). Those 16 bytes are exactly the B operand the lane supplies to the
//   second convolution's MFMA for that chunk: the paper's communication buffer between
//   the two layers (Sec. III-B) never leaves the registers. Output-stationary over the
//   chunks (Sec. III-A, OS-LWS), output written once.
//
//   S > 1: the S waves of a pixel group put their partial sums (fp32 / int32, MFMA lane
//   order) in LDS, meet at one barrier, and wave j then finishes the output tiles t with
//   t % S == j, adding the S partial sums in wave order (int8 sums are exact, float sums
//   always in the same order, so results are reproducible).
//
//   ZP (int8 with zero points): the MFMAs take raw codes; each contraction then loses
//   (input zero point) x (weight-row sum). The row sums come from the weight operands
//   already in registers: a lane adds the 16 bytes it holds with a four-way dot product
//   against ones, two butterfly shuffles complete the row over the four lane groups, and
//   each accumulator lane reads the rows it holds. The first convolution's sums are taken
//   per chunk (its rows change with the chunk), the second's accumulate over the wave's
//   chunks and are subtracted before the partial sums are combined. Epilogues add the
//   stage's output zero point after rounding and clamp ReLU there.
#pragma once

#include "fcm_kernels_v3.h"

namespace fcm {

// 16 bytes at byte offset off of a row that starts at row_off in the buffer r and has
// nbytes valid bytes (0: no row); bytes beyond nbytes read as zero. Buffer loads return
// zero for an offset beyond the buffer (kOob), so no lane selects or waits: the loads of a
// whole operand set stay in flight together. vec: rows are 16-byte aligned multiples of 16
// bytes (one 16-byte load); otherwise rows are multiples of 4 bytes (four word loads).
template <bool VEC>
__device__ __forceinline__ u32x4 load_slot4(rsrc_t r, uint32_t row_off, int off, int nbytes) {
  if constexpr (VEC) return __builtin_amdgcn_raw_buffer_load_b128(r, off < nbytes ? row_off + off : kOob, 0, 0);
  u32x4 v;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    v[e] = __builtin_amdgcn_raw_buffer_load_b32(r, off + 4 * e < nbytes ? row_off + off + 4 * e : kOob, 0, 0);
  return v;
}

// int8 epilogue with an output zero point: round half to even, add zp, clamp to
// [qlo, qhi] (which hold ReLU's floor at zp, see zp_epi).
__device__ __forceinline__ int32_t epi_i_zp(int32_t acc, const Epi3& e, int32_t zp) {
  const int64_t t = (int64_t)acc * e.mult;
  const int64_t half = ((int64_t)1 << e.shift) >> 1;
  const int64_t rnd = e.shift > 0 ? half - 1 + ((t >> e.shift) & 1) : 0;
  int64_t q = ((t + rnd) >> e.shift) + zp;
  q = q < e.qlo ? e.qlo : q;
  q = q > e.qhi ? e.qhi : q;
  return (int32_t)q;
}
// The clamp range of a stage whose output has zero point zp: ReLU / ReLU6 floor at zp.
__device__ __forceinline__ Epi3 zp_epi(int act, const Requant& rq) {
  Epi3 e = make_epi3(act, rq);
  e.qlo = act != ACT_NONE ? max(rq.qmin, rq.zp) : rq.qmin;
  e.qhi = act != ACT_NONE ? max(rq.qmax, rq.zp) : rq.qmax;
  return e;
}
// Sum of the 16 int8 codes of a 16-byte operand slot, added to acc.
__device__ __forceinline__ int32_t sum_i8x16(const u32x4& v, int32_t acc) {
#pragma unroll
  for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_sdot4((int)v[q], 0x01010101, acc, false);
  return acc;
}
// Row sums held by lanes (row l % 16, a quarter of it per lane group l / 16) completed
// over the four lane groups; out[v] = the sum of row 4 * (l / 16) + v, the accumulator
// rows of lane l. All 64 lanes of the wave take part.
__device__ __forceinline__ void rows_to_acc_lanes(int32_t part, int32_t (&out)[4]) {
  part += __shfl_xor(part, 16);
  part += __shfl_xor(part, 32);
  const int g = (threadIdx.x & 63) >> 4;
#pragma unroll
  for (int v = 0; v < 4; ++v) out[v] = __shfl(part, 4 * g + v);
}

// Stage-one epilogue of M-tile t into the lane's 16-byte operand slot: elements
// 4t .. 4t+3 of the slot (channels m0 + (16/elt)*group + 4t + v).
template <class DT>
struct Mid4;
template <>
struct Mid4<TI8> {
  __device__ static __forceinline__ void put(u32x4& slot, int t, const i32x4& acc, const int32_t (&b)[4],
                                             const Epi3& e) {
    uint32_t w = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int32_t s = acc[v];
      w |= ((uint32_t)epi_i(s + b[v], e) & 0xffu) << (8 * v);
    }
    slot[t] = w;
  }
  __device__ static __forceinline__ void put_zp(u32x4& slot, int t, const i32x4& acc, const int32_t (&b)[4],
                                                const Epi3& e, int32_t zp) {
    uint32_t w = 0;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int32_t s = acc[v];
      w |= ((uint32_t)epi_i_zp(s + b[v], e, zp) & 0xffu) << (8 * v);
    }
    slot[t] = w;
  }
};
template <>
struct Mid4<TBF16> {
  __device__ static __forceinline__ void put(u32x4& slot, int t, const f32x4& acc, const float (&b)[4],
                                             const Epi3& e) {
    const float a0 = acc[0], a1 = acc[1], a2 = acc[2], a3 = acc[3];
    slot[2 * t] = pack_bf16x2(epi_f(a0 + b[0], e), epi_f(a1 + b[1], e));
    slot[2 * t + 1] = pack_bf16x2(epi_f(a2 + b[2], e), epi_f(a3 + b[3], e));
  }
};
template <>
struct Mid4<TF32> {
  __device__ static __forceinline__ void put(u32x4& slot, int, const f32x4& acc, const float (&b)[4],
                                             const Epi3& e) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const float s = acc[v];
      slot[v] = __float_as_uint(epi_f(s + b[v], e));
    }
  }
};

// Final epilogue of four consecutive output channels: +bias, activation, cast, one store
// of 4 elements.
template <class DT>
__device__ __forceinline__ void store4_out(char* p, const typename DT::AccV& acc, const typename DT::Acc (&b)[4],
                                           const Epi3& e) {
  const typename DT::Acc s0 = acc[0], s1 = acc[1], s2 = acc[2], s3 = acc[3];
  if constexpr (std::is_same<DT, TI8>::value) {
    *(uint32_t*)p = ((uint32_t)epi_i(s0 + b[0], e) & 0xffu) | (((uint32_t)epi_i(s1 + b[1], e) & 0xffu) << 8) |
                    (((uint32_t)epi_i(s2 + b[2], e) & 0xffu) << 16) | ((uint32_t)epi_i(s3 + b[3], e) << 24);
  } else if constexpr (std::is_same<DT, TBF16>::value) {
    *(u32x2*)p = u32x2{pack_bf16x2(epi_f(s0 + b[0], e), epi_f(s1 + b[1], e)),
                       pack_bf16x2(epi_f(s2 + b[2], e), epi_f(s3 + b[3], e))};
  } else {
    *(u32x4*)p = u32x4{__float_as_uint(epi_f(s0 + b[0], e)), __float_as_uint(epi_f(s1 + b[1], e)),
                       __float_as_uint(epi_f(s2 + b[2], e)), __float_as_uint(epi_f(s3 + b[3], e))};
  }
}

// int8 output of four consecutive channels with an output zero point.
__device__ __forceinline__ void store4_out_zp(char* p, const i32x4& acc, const int32_t (&b)[4], const Epi3& e,
                                              int32_t zp) {
  const int32_t s0 = acc[0], s1 = acc[1], s2 = acc[2], s3 = acc[3];
  *(uint32_t*)p = ((uint32_t)epi_i_zp(s0 + b[0], e, zp) & 0xffu) |
                  (((uint32_t)epi_i_zp(s1 + b[1], e, zp) & 0xffu) << 8) |
                  (((uint32_t)epi_i_zp(s2 + b[2], e, zp) & 0xffu) << 16) |
                  ((uint32_t)epi_i_zp(s3 + b[3], e, zp) << 24);
}

// VEC: every operand row is a 16-byte aligned multiple of 16 bytes (x, both weight
// matrices, the first bias); otherwise operands are read as 4-byte words.
// ZP: int8 with zero points (a.zin: the inputs' of both convolutions, a.rq[].zp: their
// outputs').
template <class DT, int KS, int CT, int PB, bool VEC, bool ZP>
__global__ __launch_bounds__(256) void k_pwpw4(KArgs a) {
  static_assert(!ZP || std::is_same<DT, TI8>::value, "zero points are int8 only");
  using Acc = typename DT::Acc;
  using AccV = typename DT::AccV;
  constexpr int E = DT::ELT;
  constexpr int TPC = 4 / E;   // first-convolution M-tiles per 64-byte chunk
  constexpr int CPG = 16 / E;  // channels per 16-byte lane slot
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;

  const int S = a.splits;                  // waves per pixel group: 1, 2 or 4
  const int L = xcd_remap(blockIdx.x, gridDim.x);
  const int gi = wave / S, j = wave % S;   // pixel group in the workgroup, split
  const int pg = (4 / S) * L + gi;         // pixel group
  const bool active = pg < a.nwork;
  if (S == 1 && !active) return;           // (S > 1: every wave reaches the barrier)
  const int npix = a.N * a.H * a.W;
  const int ci_b = a.Ci * E, cm_b = a.Cm * E;
  const int ct = ceil_div(a.Co, 16);
  const int nch = ceil_div(cm_b, 64);
  // buffer resources (sizes below 2^31 bytes, checked by the planner)
  const rsrc_t rx = make_rsrc(a.x, (uint32_t)npix * ci_b);
  const rsrc_t rw1 = make_rsrc(a.w1, (uint32_t)a.Cm * ci_b);
  const rsrc_t rw2 = make_rsrc(a.w2, (uint32_t)a.Co * cm_b);
  const rsrc_t rb1 = make_rsrc(a.b1, a.b1 ? (uint32_t)a.Cm * 4 : 0u);

  // B operands of the first convolution: the group's pixels, all input channels
  u32x4 xb[PB][KS];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb) {
    const int p = (pg * PB + pb) * 16 + r16;
    const int nb = p < npix ? ci_b : 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) xb[pb][s] = load_slot4<VEC>(rx, (uint32_t)p * ci_b, 64 * s + 16 * g, nb);
  }

  AccV acc2[PB][CT];
#pragma unroll
  for (int pb = 0; pb < PB; ++pb)
#pragma unroll
    for (int u = 0; u < CT; ++u) acc2[pb][u] = AccV{0, 0, 0, 0};

  const Epi3 e1 = ZP ? zp_epi(a.act[0], a.rq[0]) : make_epi3(a.act[0], a.rq[0]);
  [[maybe_unused]] int32_t rs2[CT];  // ZP: partial row sums of the second weights (this wave's chunks)
  if constexpr (ZP) {
#pragma unroll
    for (int u = 0; u < CT; ++u) rs2[u] = 0;
  }
  // operands of one intermediate chunk: the first convolution's weight rows (permuted,
  // see above), the chunk's slice of the second convolution's weights, the first bias
  struct Ops {
    u32x4 a1[TPC][KS];
    u32x4 a2[CT];
    Acc b1[TPC][4];
  };
  // Every load and MFMA is issued whatever the shape (k-steps beyond the input channels
  // and tiles beyond the output channels read zeros and add zeros): with a fixed count of
  // loads per chunk the compiler's memory-counter waits let the next chunk's loads stay
  // in flight during this chunk's MFMAs.
  auto load_ops = [&](Ops& o, int c) {
    const int m0 = c * (64 / E);
#pragma unroll
    for (int t = 0; t < TPC; ++t) {
      const int ch = m0 + CPG * (r16 >> 2) + 4 * t + (r16 & 3);
      const int nb = ch < a.Cm ? ci_b : 0;
#pragma unroll
      for (int s = 0; s < KS; ++s) o.a1[t][s] = load_slot4<VEC>(rw1, (uint32_t)ch * ci_b, 64 * s + 16 * g, nb);
    }
#pragma unroll
    for (int u = 0; u < CT; ++u) {
      const int co = 16 * u + r16;
      const int nb = (u < ct && co < a.Co) ? cm_b : 0;
      o.a2[u] = load_slot4<VEC>(rw2, (uint32_t)co * cm_b, 64 * c + 16 * g, nb);
    }
    // bias of channels m0 + CPG*g + 4t + [0, 4): 16 contiguous bytes per t (Cm % 4 == 0)
#pragma unroll
    for (int t = 0; t < TPC; ++t) {
      const int ch = m0 + CPG * g + 4 * t;
      const u32x4 bv = load_slot4<VEC>(rb1, 0u, ch * 4, a.b1 ? a.Cm * 4 : 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t w = bv[q];
        o.b1[t][q] = __builtin_bit_cast(Acc, w);
      }
    }
    // keep the whole set issued here: a load the scheduler sank past the next chunk's
    // loads would make this chunk's arithmetic wait for those as well
    __builtin_amdgcn_sched_barrier(0);
  };
  auto compute = [&](const Ops& o) {
    [[maybe_unused]] int32_t b1z[TPC][4];  // ZP: first bias minus zin x row sums
    if constexpr (ZP) {
#pragma unroll
      for (int t = 0; t < TPC; ++t) {
        int32_t part = 0;
#pragma unroll
        for (int s = 0; s < KS; ++s) part = sum_i8x16(o.a1[t][s], part);
        int32_t rs[4];
        rows_to_acc_lanes(part, rs);
#pragma unroll
        for (int v = 0; v < 4; ++v) b1z[t][v] = o.b1[t][v] - a.zin[0] * rs[v];
      }
#pragma unroll
      for (int u = 0; u < CT; ++u) rs2[u] = sum_i8x16(o.a2[u], rs2[u]);
    }
#pragma unroll
    for (int pb = 0; pb < PB; ++pb) {
      u32x4 mid = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int t = 0; t < TPC; ++t) {
        AccV acc1 = AccV{0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < KS; ++s) mma16(DT(), acc1, o.a1[t][s], xb[pb][s]);
        if constexpr (ZP)
          Mid4<DT>::put_zp(mid, t, acc1, b1z[t], e1, a.rq[0].zp);
        else
          Mid4<DT>::put(mid, t, acc1, o.b1[t], e1);
      }
#pragma unroll
      for (int u = 0; u < CT; ++u) mma16(DT(), acc2[pb][u], o.a2[u], mid);
    }
  };
  // software pipeline over the wave's chunks j, j+S, ...: the next chunk's operand loads
  // are in flight while the current chunk's MFMAs run (two operand sets, alternating).
  // The loads of the chunk after the last are issued too (every offset out of range,
  // zeros, no memory traffic), so every path has the same loads outstanding.
  if (active && j < nch) {
    Ops o0, o1;
    int c = j;
    load_ops(o0, c);
#pragma unroll 1
    while (true) {
      load_ops(o1, c + S);
      compute(o0);
      c += S;
      if (c >= nch) break;
      load_ops(o0, c + S);
      compute(o1);
      c += S;
      if (c >= nch) break;
    }
  }

  if constexpr (ZP) {
    // the second convolution read codes of zero point zin[1]: subtract it times this
    // wave's share of each weight-row sum (the shares add up over the split waves)
    if (active && j < nch) {  // wave-uniform
#pragma unroll
      for (int u = 0; u < CT; ++u) {
        int32_t rs[4];
        rows_to_acc_lanes(rs2[u], rs);
#pragma unroll
        for (int pb = 0; pb < PB; ++pb)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc2[pb][u][v] -= a.zin[1] * rs[v];
      }
    }
  }
  const Epi3 e2 = ZP ? zp_epi(a.act[1], a.rq[1]) : make_epi3(a.act[1], a.rq[1]);
  char* y = (char*)a.y;
  // final epilogue of output tile u of pixel block pb: lane (pixel r16, group g) holds
  // output channels 16u + 4g + [0, 4)
  auto finish = [&](const AccV& v, int pb, int u) {
    const int p = (pg * PB + pb) * 16 + r16;
    const int co = 16 * u + 4 * g;
    if (p >= npix || co >= a.Co) return;
    Acc b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = load_bias<DT>(a.b2, co + q);
    if constexpr (ZP)
      store4_out_zp(y + ((size_t)p * a.Co + co) * E, v, b, e2, a.rq[1].zp);
    else
      store4_out<DT>(y + ((size_t)p * a.Co + co) * E, v, b, e2);
  };

  if (S > 1) {
    // partial sums through LDS: [wave][pixel block][output tile][lane], 16 bytes each
    extern __shared__ __align__(16) char smem[];
    AccV* red = (AccV*)smem;
    const int nt = PB * ct;
#pragma unroll
    for (int pb = 0; pb < PB; ++pb)
#pragma unroll
      for (int u = 0; u < CT; ++u)
        if (u < ct) red[(wave * nt + pb * ct + u) * 64 + lane] = acc2[pb][u];
    __syncthreads();
    if (!active) return;
    for (int t = j; t < nt; t += S) {
      AccV v = red[((gi * S) * nt + t) * 64 + lane];
      for (int jj = 1; jj < S; ++jj) v += red[((gi * S + jj) * nt + t) * 64 + lane];
      finish(v, t / ct, t % ct);
    }
    return;
  }
#pragma unroll
  for (int pb = 0; pb < PB; ++pb)
#pragma unroll
    for (int u = 0; u < CT; ++u)
      if (u < ct) finish(acc2[pb][u], pb, u);
}

template <class DT, int KS, int CT, int PB>
int launch_pwpw4(const KArgs& a, int grid, void* stream) {
  const bool vec = a.vec_x && a.vec_w1 && a.vec_w2 && ((uintptr_t)a.b1 & 15) == 0;
  const void* fn = vec ? (const void*)k_pwpw4<DT, KS, CT, PB, true, false>
                       : (const void*)k_pwpw4<DT, KS, CT, PB, false, false>;
  if ((a.zin[0] | a.zin[1] | a.rq[0].zp | a.rq[1].zp) != 0) {
    // zero points: int8 instances of at most kZpMaxTiles output tiles (the row sums of
    // the second weights need CT more registers; larger instances exceed the budget)
    if constexpr (std::is_same<DT, TI8>::value && CT <= kZpMaxTiles)
      fn = vec ? (const void*)k_pwpw4<DT, KS, CT, PB, true, true> : (const void*)k_pwpw4<DT, KS, CT, PB, false, true>;
    else
      return (int)hipErrorInvalidValue;  // the planner never selects such a plan
  }
  const int lds = a.splits > 1 ? 4 * PB * ceil_div(a.Co, 16) * 1024 : 0;
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return (int)e;
  }
  return launch_args(fn, grid, 256, lds, stream, a);
}

}  // namespace fcm
