// Family 4, IGEMM_F32: convolution as an implicit GEMM on the fp32 matrix
// cores (v_mfma_f32_32x32x2_f32 / v_mfma_f32_16x16x4_f32), NCHW x,
// K x C x R x S w, NCHW y.
//
// GEMM view: rows = output channels (K), columns = output pixels
// (N*OH*OW, flattened), reduction = C*R*S in the filter's memory order, so
// the A operand (filter) is a plain row-major matrix and the B operand is the
// im2col gather of x, formed on the fly and never stored in HBM.
//
// A block owns a BM x BN tile (BM = WM*TM*MF channels, BN = WN*TN*MF pixels)
// and WS reduction groups of WM x WN waves. Each reduction chunk of KC is
// staged in LDS (A as [BM][KC+1], B as [KC][BN]); reduction group g does the
// g-th share of the chunk's MFMA k-steps, and the groups' partial tiles are
// added in group order through LDS at the end. STAGES = 2 double-buffers the
// LDS tile and keeps the next chunk's global loads in flight during the
// MFMAs. SPLIT > 1 spreads contiguous chunk ranges over grid.z and adds the
// partial outputs in split order in a second kernel.
//
// All global loads are bounds-checked (zero fill), so any tile overhang and
// any ragged reduction tail are safe.
#pragma once
#include <hip/hip_runtime.h>

#include "ct_internal.h"

namespace ct {

struct IgF32Args {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw;
  int OH, OW, OHW;
  int npix, kred;
  int wm, wn, wsp, kc;
  int bm, bn, threads;
  int cps, chunks;
  int a_loads, b_loads, rows_a, rows_b;
  int64_t ny;
};

__host__ __device__ constexpr int ig_spec_r(int spec) { return spec == 1 || spec == 2 ? 1 : (spec == 3 || spec == 4 ? 3 : 0); }
__host__ __device__ constexpr int ig_spec_stride(int spec) { return spec == 1 || spec == 3 ? 1 : (spec == 2 || spec == 4 ? 2 : 0); }
// Threads per block that leave room for the accumulator tile in registers.
__host__ __device__ constexpr int mfma_max_threads(int acc_regs) { return acc_regs <= 32 ? 1024 : (acc_regs <= 64 ? 512 : 256); }

template <int MF>
struct MfmaF32;
template <>
struct MfmaF32<32> {
  static constexpr int ACC = 16, KSTEP = 2;
  typedef float V __attribute__((ext_vector_type(16)));
  __device__ static V op(float a, float b, V c) { return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0); }
  // row of accumulator element e held by `lane` (column = lane % 32)
  __device__ static int row(int e, int lane) { return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3); }
};
template <>
struct MfmaF32<16> {
  static constexpr int ACC = 4, KSTEP = 4;
  typedef float V __attribute__((ext_vector_type(4)));
  __device__ static V op(float a, float b, V c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }
  __device__ static int row(int e, int lane) { return 4 * (lane >> 4) + e; }
};

template <int MF, int TM, int TN, int STAGES, int SPEC>
__global__ void __launch_bounds__(mfma_max_threads(TM * TN * MfmaF32<MF>::ACC))
igemm_f32_kernel(const float* __restrict__ x, const float* __restrict__ w, float* __restrict__ out,
                 IgF32Args a) {
  using M = MfmaF32<MF>;
  using V = typename M::V;
  constexpr int ACC = M::ACC, KSTEP = M::KSTEP;
  constexpr int RC = ig_spec_r(SPEC), STC = ig_spec_stride(SPEC);
  const int R = RC ? RC : a.R, S = RC ? RC : a.S;
  const int sh = STC ? STC : a.sh, sw = STC ? STC : a.sw;
  const int dh = SPEC ? 1 : a.dh, dw = SPEC ? 1 : a.dw;
  const int ph = SPEC ? RC / 2 : a.ph, pw = SPEC ? RC / 2 : a.pw;
  const int RS = R * S;

  extern __shared__ float smem[];
  const int kc = a.kc, bm = a.bm, bn = a.bn;
  const int a_pitch = kc + 1;
  const int stage_floats = bm * a_pitch + kc * bn;

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wpg = a.wm * a.wn;
  const int wg = wave / wpg, wi = wave - wg * wpg;
  const int wmi = wi / a.wn, wni = wi - wmi * a.wn;
  const int m_off = wmi * TM * MF, n_off = wni * TN * MF;
  const int p0 = blockIdx.x * bn, k0 = blockIdx.y * bm, sp = blockIdx.z;

  // loader coordinates: A = filter rows of this block, B = im2col columns
  const int kr_a = t % kc, row_a0 = t / kc;
  const int pp = t % bn, krow_b0 = t / bn;
  const int p = p0 + pp;
  const bool pvalid = p < a.npix;
  int ih0 = 0, iw0 = 0, nimg = 0;
  if (pvalid) {
    nimg = p / a.OHW;
    const int rem = p - nimg * a.OHW;
    const int oh = rem / a.OW, ow = rem - oh * a.OW;
    ih0 = oh * sh - ph;
    iw0 = ow * sw - pw;
  }
  const float* xn = x + (int64_t)nimg * a.C * a.H * a.W;

  const int ch_begin = sp * a.cps;
  const int ch_end = min(a.chunks, ch_begin + a.cps);
  const int kr_end = min(a.kred, ch_end * kc);

  float ra[kMaxLoadsPerThread], rb[kMaxLoadsPerThread];
  auto load_chunk = [&](int ch) {
    const int kr0 = ch * kc;
#pragma unroll
    for (int i = 0; i < kMaxLoadsPerThread; ++i) {
      if (i < a.a_loads) {
        const int row = row_a0 + i * a.rows_a;
        const int kr = kr0 + kr_a;
        float v = 0.f;
        if (row < bm && k0 + row < a.K && kr < kr_end) v = w[(int64_t)(k0 + row) * a.kred + kr];
        ra[i] = v;
      }
    }
#pragma unroll
    for (int i = 0; i < kMaxLoadsPerThread; ++i) {
      if (i < a.b_loads) {
        const int krow = krow_b0 + i * a.rows_b;
        const int kr = kr0 + krow;
        float v = 0.f;
        if (pvalid && krow < kc && kr < kr_end) {
          const int c = kr / RS;
          const int rs = kr - c * RS;
          const int r = rs / S, s = rs - r * S;
          const int ih = ih0 + r * dh, iw = iw0 + s * dw;
          if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) v = xn[((int64_t)c * a.H + ih) * a.W + iw];
        }
        rb[i] = v;
      }
    }
  };
  auto store_chunk = [&](int stage) {
    float* As = smem + stage * stage_floats;
    float* Bs = As + bm * a_pitch;
#pragma unroll
    for (int i = 0; i < kMaxLoadsPerThread; ++i) {
      const int row = row_a0 + i * a.rows_a;
      if (i < a.a_loads && row < bm) As[row * a_pitch + kr_a] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < kMaxLoadsPerThread; ++i) {
      const int krow = krow_b0 + i * a.rows_b;
      if (i < a.b_loads && krow < kc) Bs[krow * bn + pp] = rb[i];
    }
  };

  V acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < ACC; ++e) acc[i][j][e] = 0.f;

  const int spg = (kc / KSTEP) / a.wsp;  // k-steps per reduction group
  const int lrow = lane % MF, kl_lane = lane / MF;
  auto compute = [&](int stage) {
    const float* As = smem + stage * stage_floats;
    const float* Bs = As + bm * a_pitch;
    const float* ap = As + (m_off + lrow) * a_pitch + kl_lane;
    const float* bp = Bs + kl_lane * bn + n_off + lrow;
    for (int st = wg * spg; st < (wg + 1) * spg; ++st) {
      const int kb = st * KSTEP;
      float fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = ap[i * MF * a_pitch + kb];
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[j] = bp[kb * bn + j * MF];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[i], fb[j], acc[i][j]);
    }
  };

  if constexpr (STAGES == 1) {
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      load_chunk(ch);
      __syncthreads();
      store_chunk(0);
      __syncthreads();
      compute(0);
    }
  } else {
    if (ch_begin < ch_end) {
      load_chunk(ch_begin);
      store_chunk(0);
      __syncthreads();
    }
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      const int cur = (ch - ch_begin) & 1;
      const bool more = ch + 1 < ch_end;
      if (more) load_chunk(ch + 1);
      compute(cur);
      if (more) store_chunk(cur ^ 1);
      __syncthreads();
    }
  }

  if (a.wsp > 1) {
    // add the reduction groups' partial tiles in group order
    __syncthreads();
    float* red = smem;
    if (wg > 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < ACC; ++e)
            red[((((wg - 1) * wpg + wi) * TM * TN + i * TN + j) * ACC + e) * 64 + lane] = acc[i][j][e];
    }
    __syncthreads();
    if (wg > 0) return;
    for (int g = 1; g < a.wsp; ++g) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < ACC; ++e)
            acc[i][j][e] += red[((((g - 1) * wpg + wi) * TM * TN + i * TN + j) * ACC + e) * 64 + lane];
    }
  }

  float* o = out + (int64_t)sp * a.ny;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int pq = p0 + n_off + j * MF + lrow;
    if (pq >= a.npix) continue;
    const int ni = pq / a.OHW;
    const int rem = pq - ni * a.OHW;
    float* op = o + (int64_t)ni * a.K * a.OHW + rem;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int e = 0; e < ACC; ++e) {
        const int k = k0 + m_off + i * MF + M::row(e, lane);
        if (k < a.K) op[(int64_t)k * a.OHW] = acc[i][j][e];
      }
    }
  }
}

using IgF32Fn = void (*)(const float*, const float*, float*, IgF32Args);

template <int MF, int TM, int TN, int STAGES>
IgF32Fn igf32_pick_spec(int spec) {
  switch (spec) {
    case SPEC_1X1_S1: return igemm_f32_kernel<MF, TM, TN, STAGES, 1>;
    case SPEC_1X1_S2: return igemm_f32_kernel<MF, TM, TN, STAGES, 2>;
    case SPEC_3X3_S1: return igemm_f32_kernel<MF, TM, TN, STAGES, 3>;
    case SPEC_3X3_S2: return igemm_f32_kernel<MF, TM, TN, STAGES, 4>;
    default: return igemm_f32_kernel<MF, TM, TN, STAGES, 0>;
  }
}
template <int MF, int TM, int TN>
IgF32Fn igf32_pick_stages(int stages, int spec) {
  return stages == 2 ? igf32_pick_spec<MF, TM, TN, 2>(spec) : igf32_pick_spec<MF, TM, TN, 1>(spec);
}
template <int MF, int TM>
IgF32Fn igf32_pick_tn(int tn, int stages, int spec) {
  switch (tn) {
    case 1: return igf32_pick_stages<MF, TM, 1>(stages, spec);
    case 2: return igf32_pick_stages<MF, TM, 2>(stages, spec);
    default: return igf32_pick_stages<MF, TM, 4>(stages, spec);
  }
}

}  // namespace ct
