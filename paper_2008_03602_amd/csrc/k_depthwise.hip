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
// Q4 = 1 (3x3 filters with pad 1 only) switches to depthwise_q4_kernel: a
// thread owns 4 consecutive output columns of RPT consecutive rows, reads
// each input row it needs once with 16-byte loads (plus the edge words) and
// keeps the taps in registers, so a wave reads and writes whole 16-byte
// words and an output costs well under one load instruction instead of nine.
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
  int vec_ld, vec_st;  // depthwise_q4_kernel: 16-byte input loads / output stores allowed
};

// Threads per block of the strided kernel that leave registers for its
// outputs per thread (16 outputs need 256 VGPRs: at most 512 threads).
__host__ __device__ constexpr int dw_max_threads(int outs) { return outs >= 16 ? 512 : 1024; }
__host__ __device__ constexpr int dw_spec_r(int spec) { return spec == 3 || spec == 4 ? 3 : 0; }
__host__ __device__ constexpr int dw_spec_stride(int spec) { return spec == 3 ? 1 : (spec == 4 ? 2 : 0); }

template <int VEC, int RPT, bool LDS, int SPEC>
__global__ void __launch_bounds__(dw_max_threads(VEC * RPT))
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

typedef float dwf4 __attribute__((ext_vector_type(4)));

// 3x3, pad 1, stride STRIDE: a thread computes 4 consecutive output columns of
// RPT consecutive output rows of one (image, channel) plane. It reads the
// (RPT - 1) * STRIDE + 3 input rows those outputs need, each as the
// 3 * STRIDE + 3 columns from ow * STRIDE - 1 on: with vec_ld, the interior
// 4 (stride 1) or 8 (stride 2) columns as 16-byte loads and the edge columns
// as words (which the neighbouring lanes' 16-byte loads have brought into
// L1). vec_ld holds when W is a multiple of 4, W = STRIDE * OW, OW is a
// multiple of 4 and x is 16-byte aligned: every 16-byte load then lies inside
// its row. Columns and rows outside the image read as zero.
template <int STRIDE, int RPT>
__global__ void __launch_bounds__(1024)
depthwise_q4_kernel(const float* __restrict__ x, const float* __restrict__ w, float* __restrict__ y, DwArgs a) {
  constexpr int NIN = (RPT - 1) * STRIDE + 3;  // input rows read
  constexpr int NCOL = 3 * STRIDE + 3;         // input columns per row
  const int H = a.H, W = a.W, C = a.C, OH = a.OH, OW = a.OW;

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
  int t = threadIdx.x;
  const int colq = t % a.cols; t /= a.cols;
  const int rowg = t % a.rows; t /= a.rows;
  const int ci = t % a.tc;
  const int ni = t / a.tc;
  const int c = cg * a.tc + ci, n = ng * a.nb + ni;
  const int ow = tw * a.tow + 4 * colq, oh = th * a.toh + rowg * RPT;
  if (c >= C || n >= a.N || ow >= OW || oh >= OH) return;  // no barriers in this kernel

  float wv[9];
#pragma unroll
  for (int i = 0; i < 9; ++i) wv[i] = w[(int64_t)c * 9 + i];
  const float* xp = x + ((int64_t)n * C + c) * H * W;
  const int ih0 = oh * STRIDE - 1, iw0 = ow * STRIDE - 1;

  float acc[RPT][4];
#pragma unroll
  for (int u = 0; u < RPT; ++u)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[u][j] = 0.f;

#pragma unroll
  for (int i = 0; i < NIN; ++i) {
    const int ih = ih0 + i;
    float v[NCOL];
#pragma unroll
    for (int k = 0; k < NCOL; ++k) v[k] = 0.f;
    if ((unsigned)ih < (unsigned)H) {
      const float* row = xp + (int64_t)ih * W;
      if (a.vec_ld) {
        v[0] = iw0 >= 0 ? row[iw0] : 0.f;
        const dwf4 q0 = *(const dwf4*)(row + iw0 + 1);
        v[1] = q0.x; v[2] = q0.y; v[3] = q0.z; v[4] = q0.w;
        if constexpr (STRIDE == 1) {
          v[5] = iw0 + 5 < W ? row[iw0 + 5] : 0.f;
        } else {
          const dwf4 q1 = *(const dwf4*)(row + iw0 + 5);
          v[5] = q1.x; v[6] = q1.y; v[7] = q1.z; v[8] = q1.w;
        }
      } else {
#pragma unroll
        for (int k = 0; k < NCOL; ++k) v[k] = load_or_zero(row, iw0 + k, (unsigned)(iw0 + k) < (unsigned)W);
      }
    }
    // input row i feeds output row u through filter row r = i - u * STRIDE
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int r = i - u * STRIDE;
      if (r < 0 || r > 2) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int s = 0; s < 3; ++s) acc[u][j] = fmaf(wv[r * 3 + s], v[j * STRIDE + s], acc[u][j]);
    }
  }

  float* yp = y + ((int64_t)n * C + c) * OH * OW;
#pragma unroll
  for (int u = 0; u < RPT; ++u) {
    if (oh + u >= OH) break;
    float* o = yp + (int64_t)(oh + u) * OW + ow;
    if (a.vec_st) {
      dwf4 q;
      q.x = acc[u][0]; q.y = acc[u][1]; q.z = acc[u][2]; q.w = acc[u][3];
      *(dwf4*)o = q;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (ow + j < OW) o[j] = acc[u][j];
    }
  }
}

using DwFn = void (*)(const float*, const float*, float*, DwArgs);

template <int STRIDE>
static DwFn dw_q4_pick(int rpt) {
  switch (rpt) {
    case 1: return depthwise_q4_kernel<STRIDE, 1>;
    case 2: return depthwise_q4_kernel<STRIDE, 2>;
    default: return depthwise_q4_kernel<STRIDE, 4>;
  }
}

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
  DwFn fn;
  if (s.knob[Q4]) {  // the validator admits it for 3x3 pad-1 ops (spec 3 or 4) with VEC = 4, LDS = 0
    const int st = g.spec == SPEC_3X3_S2 ? 2 : 1;
    a.cols = a.tow / 4;
    a.vec_ld = a.W % 4 == 0 && a.W == st * a.OW && a.OW % 4 == 0 && ((uintptr_t)xin % 16) == 0;
    a.vec_st = a.OW % 4 == 0 && ((uintptr_t)y % 16) == 0;
    fn = st == 2 ? dw_q4_pick<2>(s.knob[RPT]) : dw_q4_pick<1>(s.knob[RPT]);
  } else {
    a.vec_ld = a.vec_st = 0;
    fn = dw_pick(s.knob[VEC], s.knob[RPT], s.knob[LDS], g.spec);
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)g.blocks), dim3(g.threads), g.lds_bytes, (hipStream_t)stream,
                     (const float*)xin, (const float*)w, (float*)y, a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace ct
