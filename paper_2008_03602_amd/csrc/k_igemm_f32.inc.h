// Family 4, IGEMM_F32: convolution as an implicit GEMM on the fp32 matrix
// cores (v_mfma_f32_32x32x2_f32 / v_mfma_f32_16x16x4_f32), NCHW x,
// K x C x R x S w, NCHW y.
//
// GEMM view: rows = output channels, columns = output pixels, reduction =
// (filter tap, input channel). A block owns a BM x BN tile: BM = WM*TM*MF
// output channels by BN = WN*TN*MF output pixels, the pixels forming a
// TPH x TPW rectangle of one image (TPW = the TPW knob, TPH = BN / TPW).
//
// Staging. The reduction advances one chunk of CPC input channels at a time
// (padded to CPCP, a whole number of MFMA k-groups per reduction group). A
// chunk stages in LDS
//   * the input halo of the pixel rectangle, Xs[CPCP][HT][WT], loaded once:
//     every filter tap reads its operand from this tile, so a 3x3 filter
//     costs one global load per input element instead of nine;
//   * the filter slice As[BM][R*S][CPCP] (row pitch LDA), tap-major so that
//     consecutive MFMA k-steps are consecutive channels of one tap.
// Global reads are raw buffer loads: the descriptor base advances one chunk
// per iteration (scalar work); per-lane byte offsets are fixed for the whole
// kernel, and an element that is padding, overhang or a padded channel gets
// an offset beyond the buffer, which reads as 0. The staging plan is built
// with carry counters (no per-element divisions).
//
// MFMA k mapping. k lane-group g (= lane / MF) takes channels i*KSTEP + g,
// so for a fixed tap a step advances every operand address by a constant:
// A by KSTEP, B by KSTEP channel planes of the halo. WS reduction groups
// split the k-steps of each tap; their partial tiles are added in group order
// through LDS. STAGES = 2 double-buffers the LDS chunk and keeps the next
// chunk's loads in flight during the MFMAs. SPLIT > 1 spreads contiguous chunk
// ranges over grid.z; a second kernel adds the partials in split order.
#pragma once
#include <hip/hip_runtime.h>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

constexpr int kF32Slots = 16;  // staged elements per thread per chunk: halo + filter (max)

struct IgF32Args {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw;
  int OH, OW, kred;
  int wm, wn, wsp, cpc, cpcp;
  int tpw, tph, tiles_w, tiles_h;
  int ht, wt, lda;
  int bm, bn, threads;
  int cps, chunks;
  int n_halo, n_filt;  // staged halo / filter elements per thread per chunk
  // host-precomputed: exact reciprocals for small quotients, and the block
  // size decomposed over the halo (c, hh, ww) and filter (m, c, tap) indices
  float inv_plane, inv_wt, inv_perm, inv_rs, inv_tpw;
  int h_dc, h_dhh, h_dww, f_dm, f_dc, f_dtap;
  int64_t ny;
};

// floor(n / d) for 0 <= n < 2^22 given inv = 1/d in fp32: (n + 1/2)/d lies at
// least 1/(2d) from an integer and the fp32 product errs by less than that.
__device__ __forceinline__ int qdiv(int n, float inv) { return (int)(((float)n + 0.5f) * inv); }

__host__ __device__ constexpr int ig_spec_r(int spec) { return spec == 1 || spec == 2 ? 1 : (spec == 3 || spec == 4 ? 3 : 0); }
__host__ __device__ constexpr int ig_spec_stride(int spec) { return spec == 1 || spec == 3 ? 1 : (spec == 2 || spec == 4 ? 2 : 0); }
// Threads per block that leave room for the accumulator tile in registers.
__host__ __device__ constexpr int mfma_max_threads(int acc_regs) { return acc_regs <= 64 ? 512 : 256; }

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

constexpr int kOob = 0x7FFFFFF0;  // byte offset beyond every buffer: reads as 0

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float bload(__amdgpu_buffer_rsrc_t r, int off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

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
  const int HW = a.H * a.W;

  extern __shared__ float smem[];
  const int cpcp = a.cpcp, bm = a.bm, ht = a.ht, wt = a.wt, lda = a.lda;
  const int plane = ht * wt;
  const int xs_floats = cpcp * plane;
  const int stage_floats = xs_floats + bm * lda;

  const int t = threadIdx.x, lane = t & 63, wave = wave_id();
  const int wpg = a.wm * a.wn;
  const int wg = wave / wpg, wi = wave - wg * wpg;
  const int wmi = wi / a.wn, wni = wi - wmi * a.wn;
  const int m_off = wmi * TM * MF, n_off = wni * TN * MF;

  // block -> (image, pixel rectangle), output-channel tile, split
  const int tiles_hw = a.tiles_h * a.tiles_w;
  const int nimg = blockIdx.x / tiles_hw;
  const int trem = blockIdx.x - nimg * tiles_hw;
  const int th = trem / a.tiles_w, tw = trem - th * a.tiles_w;
  const int oh0 = th * a.tph, ow0 = tw * a.tpw;
  const int ih0 = oh0 * sh - ph, iw0 = ow0 * sw - pw;
  const int k0 = blockIdx.y * bm, sp = blockIdx.z;

  // ---- staging plan, fixed for the whole reduction (carry counters) ----
  // Each thread stages kF32Slots elements per chunk: slots [0, n_halo) are
  // halo elements, the next n_filt are filter elements, the rest are unused.
  // Every slot issues its load (an unused or padding slot reads out of range,
  // i.e. 0) and stores to LDS (an unused slot into a per-lane dummy word), so
  // the staging code has no branches and all loads are in flight at once.
  const int dummy = STAGES * stage_floats + lane;
  // channels of x per chunk: CPC divides C, or one chunk holds all C (< CPC)
  const int cl = min(a.cpc, a.C);
  int s_off[kF32Slots], s_lds[kF32Slots];
  {
    // halo element e = t + i*threads of Xs[cpcp][ht][wt] -> (c, hh, ww)
    const int T = a.threads;
    int c = qdiv(t, a.inv_plane), rem = t - c * plane;
    int hh = qdiv(rem, a.inv_wt), ww = rem - hh * wt;
    const int dc = a.h_dc, dhh = a.h_dhh, dww = a.h_dww;
#pragma unroll
    for (int i = 0; i < kF32Slots; ++i) {
      if (i < a.n_halo) {
        const int gh = ih0 + hh, gw = iw0 + ww;
        const int e = t + i * T;
        const bool ok = c < cl && gh >= 0 && gh < a.H && gw >= 0 && gw < a.W;
        s_off[i] = ok ? ((nimg * a.C + c) * HW + gh * a.W + gw) * 4 : kOob;
        s_lds[i] = e < xs_floats ? e : -1;
        ww += dww;
        if (ww >= wt) { ww -= wt; ++hh; }
        hh += dhh;
        if (hh >= ht) { hh -= ht; ++c; }
        c += dc;
      }
    }
  }
  {
    // filter element e = t + j*threads of the chunk's BM x CPCP x RS slice, in
    // global order (m, c, tap); LDS position m*lda + tap*cpcp + c
    const int per_m = cpcp * RS;
    int m = qdiv(t, a.inv_perm), rem = t - m * per_m;
    int c = qdiv(rem, a.inv_rs), tap = rem - c * RS;
    const int dm = a.f_dm, dcc = a.f_dc, dtap = a.f_dtap;
#pragma unroll
    for (int i = 0; i < kF32Slots; ++i) {
      const int j = i - a.n_halo;
      if (j >= 0 && j < a.n_filt) {
        const bool in_tile = m < bm;
        const bool ok = in_tile && k0 + m < a.K && c < cl;
        s_off[i] = ok ? ((k0 + m) * a.kred + c * RS + tap) * 4 : kOob;
        s_lds[i] = in_tile ? xs_floats + m * lda + tap * cpcp + c : -1;
        tap += dtap;
        if (tap >= RS) { tap -= RS; ++c; }
        c += dcc;
        if (c >= cpcp) { c -= cpcp; ++m; }
        m += dm;
      } else if (j >= a.n_filt) {
        s_off[i] = kOob;
        s_lds[i] = -1;
      }
    }
  }
  const int ch_begin = sp * a.cps;
  const int ch_end = min(a.chunks, ch_begin + a.cps);
  const int64_t xbytes = (int64_t)a.N * a.C * HW * 4, wbytes = (int64_t)a.K * a.kred * 4;

  float rv[kF32Slots];
  auto load_chunk = [&](int ch) {
    const int c0 = ch * a.cpc;
    // descriptors start at the chunk's first channel
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + (int64_t)c0 * HW, xbytes - (int64_t)c0 * HW * 4);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(w + (int64_t)c0 * RS, wbytes - (int64_t)c0 * RS * 4);
#pragma unroll
    for (int i = 0; i < kF32Slots; ++i) rv[i] = bload(i < a.n_halo ? rx : rw, s_off[i]);
  };
  auto store_chunk = [&](int stage) {
    const int base = stage * stage_floats;
#pragma unroll
    for (int i = 0; i < kF32Slots; ++i) smem[s_lds[i] >= 0 ? base + s_lds[i] : dummy] = rv[i];
  };

  V acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < ACC; ++e) acc[i][j][e] = 0.f;

  // this lane's operand bases: A row (output channel), B pixel in the halo
  const int lrow = lane % MF, kg = lane / MF;
  int a_base[TM], b_base[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) a_base[i] = (m_off + i * MF + lrow) * lda + kg;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int q = n_off + j * MF + lrow;
    const int pr = qdiv(q, a.inv_tpw), pc = q - pr * a.tpw;
    b_base[j] = kg * plane + (pr * sh) * wt + pc * sw;
  }
  const int n_i = cpcp / KSTEP / a.wsp;  // k-steps per tap for this reduction group
  const int i_begin = wg * n_i;
  // For each tap, the reduction group's channel steps run in groups of 4:
  // all fragment reads of a group are issued before its MFMAs.
  auto compute = [&](int stage) {
    const float* Xs = smem + stage * stage_floats;
    const float* As = Xs + xs_floats;
    for (int r = 0; r < R; ++r) {
      for (int s = 0; s < S; ++s) {
        const float* ap = As + (r * S + s) * cpcp + i_begin * KSTEP;
        const float* bp = Xs + (r * dh) * wt + s * dw + i_begin * KSTEP * plane;
        int ii = 0;
        for (; ii + 4 <= n_i; ii += 4) {
          float fa[4][TM], fb[4][TN];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[u][i] = ap[a_base[i] + (ii + u) * KSTEP];
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[u][j] = bp[b_base[j] + (ii + u) * KSTEP * plane];
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[u][i], fb[u][j], acc[i][j]);
        }
        for (; ii < n_i; ++ii) {
          float fa[TM], fb[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) fa[i] = ap[a_base[i] + ii * KSTEP];
#pragma unroll
          for (int j = 0; j < TN; ++j) fb[j] = bp[b_base[j] + ii * KSTEP * plane];
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[i], fb[j], acc[i][j]);
        }
      }
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
  const int ohw = a.OH * a.OW;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int q = n_off + j * MF + lrow;
    const int pr = qdiv(q, a.inv_tpw), pc = q - pr * a.tpw;
    const int oh = oh0 + pr, ow = ow0 + pc;
    if (oh >= a.OH || ow >= a.OW) continue;
    const int base = (nimg * a.K + k0 + m_off) * ohw + oh * a.OW + ow;  // y offset of channel k0+m_off
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int e = 0; e < ACC; ++e) {
        const int kr = i * MF + M::row(e, lane);
        if (k0 + m_off + kr < a.K) o[base + kr * ohw] = acc[i][j][e];
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
