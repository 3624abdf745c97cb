// Family 4, IGEMM_F32: launcher. The kernel and its description are in
// k_igemm_f32.inc.h; the instantiations live in one unit per MFMA shape.
#include "k_igemm_f32.inc.h"

namespace ct {

IgF32Fn igf32_pick_mf16_tm1(int tn, int stages, int spec);
IgF32Fn igf32_pick_mf16_tm2(int tn, int stages, int spec);
IgF32Fn igf32_pick_mf16_tm4(int tn, int stages, int spec);
IgF32Fn igf32_pick_mf32_tm1(int tn, int stages, int spec);
IgF32Fn igf32_pick_mf32_tm2(int tn, int stages, int spec);
IgF32Fn igf32_pick_mf32_tm4(int tn, int stages, int spec);

static IgF32Fn igf32_pick(int mf, int tm, int tn, int stages, int spec) {
  if (mf == 32) {
    if (tm == 1) return igf32_pick_mf32_tm1(tn, stages, spec);
    if (tm == 2) return igf32_pick_mf32_tm2(tn, stages, spec);
    return igf32_pick_mf32_tm4(tn, stages, spec);
  }
  if (tm == 1) return igf32_pick_mf16_tm1(tn, stages, spec);
  if (tm == 2) return igf32_pick_mf16_tm2(tn, stages, spec);
  return igf32_pick_mf16_tm4(tn, stages, spec);
}

int launch_igemm_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                     const void* w, void* y, float* ws, void* stream) {
  using namespace f32g_knob;
  const ct_op& o = x.op;
  IgF32Args a;
  a.N = o.n; a.C = o.c; a.H = o.h; a.W = o.w; a.K = o.k; a.R = o.r; a.S = o.s;
  a.sh = o.stride_h; a.sw = o.stride_w; a.ph = o.pad_h; a.pw = o.pad_w; a.dh = o.dil_h; a.dw = o.dil_w;
  a.OH = (int)x.oh; a.OW = (int)x.ow; a.kred = (int)x.kred;
  a.wm = s.knob[WM]; a.wn = s.knob[WN]; a.wsp = s.knob[WS]; a.cpc = s.knob[CPC]; a.cpcp = g.cpcp;
  a.tpw = g.tpw; a.tph = g.tph; a.tiles_w = (int)g.tiles_w; a.tiles_h = (int)g.tiles_h;
  a.ht = g.ih_t; a.wt = g.iw_t; a.lda = g.lda;
  a.bm = g.bm; a.bn = g.bn; a.threads = g.threads;
  a.cps = g.chunks_per_split; a.chunks = g.chunks;
  a.n_halo = g.a_loads; a.n_filt_units = g.bm * g.f_nseg;
  a.xs_pad = g.xs_pad; a.f_nseg = g.f_nseg;
  // 16-byte copies need 16-byte-aligned tensors (torch allocations are)
  if ((g.vec_h && ((uintptr_t)xin & 15)) || (g.vec_f && ((uintptr_t)w & 15))) {
    set_error("igemm_f32: this schedule copies 16 bytes per lane and needs 16-byte-aligned x and w");
    return -2;
  }
  // the copy plan's strides count the waves that copy: all of them, or the
  // four loader waves of STAGES 3 (which follow the MFMA waves)
  a.nmw = a.wm * a.wn * a.wsp;
  const int nw = s.knob[STAGES] == 3 ? 4 : a.threads / 64;
  const int T = 64 * nw;
  a.pp = g.hpp; a.rw = g.hrw; a.hshift = g.hshift; a.vec_h = g.vec_h; a.vec_f = g.vec_f;
  const int vh = g.vec_h ? 4 : 1;
  const int pu = a.pp / vh, ru = a.rw / vh;
  a.inv_pu = 1.0f / (float)pu;
  a.inv_ru = 1.0f / (float)ru;
  a.inv_tpw = 1.0f / (float)a.tpw;
  a.h_dc = T / pu;
  a.h_drem = T % pu;
  a.inv_tiles_hw = 1.0f / (float)(g.tiles_h * g.tiles_w);
  a.inv_tiles_w = 1.0f / (float)g.tiles_w;
  a.inv_nseg = 1.0f / (float)g.f_nseg;
  a.f_dm = nw / g.f_nseg;
  a.f_dseg = nw % g.f_nseg;
  a.lg_wpg = __builtin_ctz(a.wm * a.wn);
  a.lg_wn = __builtin_ctz(a.wn);
  a.lg_nw = __builtin_ctz(nw);
  a.ny = x.ny;
  dim3 grid((unsigned)(o.n * g.tiles_h * g.tiles_w), (unsigned)g.tiles_k, (unsigned)g.split);
  a.inv_gx = 1.0f / (float)grid.x;
  a.inv_gxy = 1.0f / (float)(grid.x * grid.y);
  IgF32Fn fn = igf32_pick(s.knob[MF], s.knob[TM], s.knob[TN], s.knob[STAGES], g.spec);
  if (!fn) {
    set_error("igemm_f32: no kernel instance for this accumulator tile");
    return -2;
  }
  float* out = g.split > 1 ? ws : (float*)y;
  hipLaunchKernelGGL(fn, grid, dim3(g.threads), g.lds_bytes, (hipStream_t)stream, (const float*)xin,
                     (const float*)w, out, a);
  if (hipGetLastError() != hipSuccess) return -1;
  if (g.split > 1) return launch_split_reduce(ws, (float*)y, x.ny, g.split, stream);
  return 0;
}

}  // namespace ct
