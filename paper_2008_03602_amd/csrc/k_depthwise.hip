// Family 2, DEPTHWISE_F32: depthwise convolution (groups = C = K, one filter
// per channel) on the vector ALU, NCHW fp32. The operator does one
// multiply-add per filter tap and output, so it is bound by memory traffic:
// the knobs trade parallelism against halo re-reads.
//
// A block computes TOH x TOW outputs for TC channels of NB images. A thread
// owns VEC output columns (TOW/VEC apart) in each of RPT output rows
// (TOH/RPT apart), so the lanes of a wave sweep consecutive columns.
// LDS = 1 stages the input halo tile of the block once; LDS = 0 reads taps
// straight from global memory (L1/L2 absorb the overlap). ORDER picks the
// block numbering: tiles fastest (0) or channel groups fastest (1).
// Every global access is bounds-checked.
#include <hip/hip_runtime.h>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

struct DwArgs {
  int N, C, H, W, R, S, sh, sw, ph, pw, dh, dw;
  int OH, OW;
  int tc, toh, tow, nb, order;
  int tiles_h, tiles_w, tiles_c, tiles_n;
  int ih_t, iw_t;
  int threads, rows, cols;
};

__host__ __device__ constexpr int dw_spec_r(int spec) { return spec == 3 || spec == 4 ? 3 : 0; }
__host__ __device__ constexpr int dw_spec_stride(int spec) { return spec == 3 ? 1 : (spec == 4 ? 2 : 0); }

template <int VEC, int RPT, bool LDS, int SPEC>
__global__ void __launch_bounds__(1024)
depthwise_f32_kernel(const float* __restrict__ x, const float* __restrict__ w, float* __restrict__ y,
                     DwArgs a) {
  constexpr int RC = dw_spec_r(SPEC), STC = dw_spec_stride(SPEC);
  const int R = RC ? RC : a.R, S = RC ? RC : a.S;
  const int sh = STC ? STC : a.sh, sw = STC ? STC : a.sw;
  const int dh = RC ? 1 : a.dh, dw = RC ? 1 : a.dw;
  const int ph = RC ? 1 : a.ph, pw = RC ? 1 : a.pw;
  const int H = a.H, W = a.W, C = a.C;

  // block -> (image group, channel group, tile row, tile column)
  int b = blockIdx.x, tw, th, cg, ng;
  if (a.order == 0) {
    tw = b % a.tiles_w; b /= a.tiles_w;
    th = b % a.tiles_h; b /= a.tiles_h;
    cg = b % a.tiles_c; ng = b / a.tiles_c;
  } else {
    cg = b % a.tiles_c; b /= a.tiles_c;
    tw = b % a.tiles_w; b /= a.tiles_w;
    th = b % a.tiles_h; ng = b / a.tiles_h;
  }
  const int oh0 = th * a.toh, ow0 = tw * a.tow, c0 = cg * a.tc, n0 = ng * a.nb;

  // thread -> (image, channel, row group, column group), columns fastest
  int t = threadIdx.x;
  const int colg = t % a.cols; t /= a.cols;
  const int rowg = t % a.rows; t /= a.rows;
  const int ci = t % a.tc;
  const int ni = t / a.tc;
  const int c = c0 + ci, n = n0 + ni;
  const bool live = c < C && n < a.N;

  float wv[RC ? RC * RC : 1];
  if constexpr (RC != 0) {
#pragma unroll
    for (int i = 0; i < RC * RC; ++i) wv[i] = load_or_zero(w, (int64_t)c * RC * RC + i, live);
  }
  float acc[RPT][VEC];
#pragma unroll
  for (int u = 0; u < RPT; ++u)
#pragma unroll
    for (int v = 0; v < VEC; ++v) acc[u][v] = 0.f;

  const int ih_org = oh0 * sh - ph, iw_org = ow0 * sw - pw;
  if constexpr (LDS) {
    extern __shared__ float smem[];
    const int plane = a.ih_t * a.iw_t;
    const int total = a.nb * a.tc * plane;
    // four branch-free loads per thread, then four LDS stores
    for (int e0 = threadIdx.x; e0 < total; e0 += 4 * a.threads) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int e = e0 + u * a.threads;
        const int p = e / plane;  // (image, channel) pair within the block
        const int rem = e - p * plane;
        const int hh = rem / a.iw_t, ww = rem - hh * a.iw_t;
        const int pn = n0 + p / a.tc, pc = c0 + p % a.tc;
        const int gh = ih_org + hh, gw = iw_org + ww;
        const bool ok = e < total && pn < a.N && pc < C && gh >= 0 && gh < H && gw >= 0 && gw < W;
        v[u] = load_or_zero(x, (((int64_t)pn * C + pc) * H + gh) * W + gw, ok);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (e0 + u * a.threads < total) smem[e0 + u * a.threads] = v[u];
    }
    __syncthreads();
    const float* xs = smem + (ni * a.tc + ci) * plane;
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int lrow = (rowg + u * a.rows) * sh;
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const float wt = RC ? wv[r * RC + s] : (live ? w[((int64_t)c * R + r) * S + s] : 0.f);
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            const int lcol = (colg + v * a.cols) * sw;
            acc[u][v] = fmaf(wt, xs[(lrow + r * dh) * a.iw_t + lcol + s * dw], acc[u][v]);
          }
        }
      }
    }
  } else {
    const float* xc = x + ((int64_t)(live ? n : 0) * C + (live ? c : 0)) * H * W;
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int oh = oh0 + rowg + u * a.rows;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int gh = oh * sh - ph + r * dh;
        const bool hok = live && gh >= 0 && gh < H;
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const float wt = RC ? wv[r * RC + s] : (live ? w[((int64_t)c * R + r) * S + s] : 0.f);
#pragma unroll
          for (int v = 0; v < VEC; ++v) {
            const int gw = (ow0 + colg + v * a.cols) * sw - pw + s * dw;
            const float xv = load_or_zero(xc, (int64_t)gh * W + gw, hok && gw >= 0 && gw < W);
            acc[u][v] = fmaf(wt, xv, acc[u][v]);
          }
        }
      }
    }
  }

  if (!live) return;
  float* yc = y + ((int64_t)n * C + c) * a.OH * a.OW;
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    const int oh = oh0 + rowg + u * a.rows;
    if (oh >= a.OH) continue;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
      const int ow = ow0 + colg + v * a.cols;
      if (ow < a.OW) yc[(int64_t)oh * a.OW + ow] = acc[u][v];
    }
  }
}

using DwFn = void (*)(const float*, const float*, float*, DwArgs);

template <int VEC, int RPT, bool LDS>
static DwFn dw_pick_spec(int spec) {
  switch (spec) {
    case SPEC_3X3_S1: return depthwise_f32_kernel<VEC, RPT, LDS, 3>;
    case SPEC_3X3_S2: return depthwise_f32_kernel<VEC, RPT, LDS, 4>;
    default: return depthwise_f32_kernel<VEC, RPT, LDS, 0>;
  }
}
template <int VEC, int RPT>
static DwFn dw_pick_lds(int lds, int spec) {
  return lds ? dw_pick_spec<VEC, RPT, true>(spec) : dw_pick_spec<VEC, RPT, false>(spec);
}
template <int VEC>
static DwFn dw_pick_rpt(int rpt, int lds, int spec) {
  switch (rpt) {
    case 1: return dw_pick_lds<VEC, 1>(lds, spec);
    case 2: return dw_pick_lds<VEC, 2>(lds, spec);
    default: return dw_pick_lds<VEC, 4>(lds, spec);
  }
}
static DwFn dw_pick(int vec, int rpt, int lds, int spec) {
  switch (vec) {
    case 1: return dw_pick_rpt<1>(rpt, lds, spec);
    case 2: return dw_pick_rpt<2>(rpt, lds, spec);
    default: return dw_pick_rpt<4>(rpt, lds, spec);
  }
}

int launch_depthwise_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                         const void* w, void* y, float* /*ws*/, void* stream) {
  using namespace dw_knob;
  const ct_op& o = x.op;
  DwArgs a;
  a.N = o.n; a.C = o.c; a.H = o.h; a.W = o.w; a.R = o.r; a.S = o.s;
  a.sh = o.stride_h; a.sw = o.stride_w; a.ph = o.pad_h; a.pw = o.pad_w; a.dh = o.dil_h; a.dw = o.dil_w;
  a.OH = (int)x.oh; a.OW = (int)x.ow;
  a.tc = s.knob[TC]; a.toh = s.knob[TOH]; a.tow = s.knob[TOW]; a.nb = s.knob[NB]; a.order = s.knob[ORDER];
  a.tiles_h = (int)g.tiles_h; a.tiles_w = (int)g.tiles_w; a.tiles_c = (int)g.tiles_c; a.tiles_n = (int)g.tiles_n;
  a.ih_t = g.ih_t; a.iw_t = g.iw_t;
  a.threads = g.threads;
  a.rows = a.toh / s.knob[RPT];
  a.cols = a.tow / s.knob[VEC];
  // the 3x3 specialisation needs pad 1 and dilation 1, which op_spec checks
  DwFn fn = dw_pick(s.knob[VEC], s.knob[RPT], s.knob[LDS], g.spec);
  hipLaunchKernelGGL(fn, dim3((unsigned)g.blocks), dim3(g.threads), g.lds_bytes, (hipStream_t)stream,
                     (const float*)xin, (const float*)w, (float*)y, a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace ct
