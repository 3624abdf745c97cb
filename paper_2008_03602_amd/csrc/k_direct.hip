// Family 1, DIRECT_F32: launcher. The kernel and its description are in
// k_direct.inc.h; the instantiations live in one unit per MK value.
#include "k_direct.inc.h"

namespace ct {

DirectFn pick_direct_mk1(int mw, int lds, int spec, int unr);
DirectFn pick_direct_mk2(int mw, int lds, int spec, int unr);
DirectFn pick_direct_mk4(int mw, int lds, int spec, int unr);
DirectFn pick_direct_mk8(int mw, int lds, int spec, int unr);

static DirectFn pick_direct(int mk, int mw, int lds, int spec, int unr) {
  switch (mk) {
    case 1: return pick_direct_mk1(mw, lds, spec, unr);
    case 2: return pick_direct_mk2(mw, lds, spec, unr);
    case 4: return pick_direct_mk4(mw, lds, spec, unr);
    default: return pick_direct_mk8(mw, lds, spec, unr);
  }
}

int launch_direct_f32(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                      const void* w, void* y, float* ws, void* stream) {
  using namespace direct_knob;
  const ct_op& o = x.op;
  DirectArgs a;
  a.N = o.n; a.C = o.c; a.H = o.h; a.W = o.w; a.K = o.k; a.R = o.r; a.S = o.s;
  a.sh = o.stride_h; a.sw = o.stride_w; a.ph = o.pad_h; a.pw = o.pad_w; a.dh = o.dil_h; a.dw = o.dil_w;
  a.OH = (int)x.oh; a.OW = (int)x.ow;
  a.toh = s.knob[TOH]; a.tow = s.knob[TOW]; a.tk = s.knob[TK]; a.ct = s.knob[CT];
  a.tiles_w = (int)g.tiles_w;
  a.split = g.split; a.cps = g.chunks_per_split;
  a.ih_t = g.ih_t; a.iw_t = g.iw_t;
  a.threads = g.threads;
  a.cols = a.tow / s.knob[MW];
  a.tp = a.toh * a.cols;
  const int rs = o.r * o.s;
  a.inv_plane = 1.0f / (float)(a.ih_t * a.iw_t);
  a.inv_iwt = 1.0f / (float)a.iw_t;
  a.inv_crs = 1.0f / (float)(a.ct * rs);
  a.inv_rs = 1.0f / (float)rs;
  a.ny = x.ny;
  DirectFn fn = pick_direct(s.knob[MK], s.knob[MW], s.knob[LDS], g.spec, s.knob[UNR]);
  dim3 grid((unsigned)(g.tiles_h * g.tiles_w), (unsigned)g.tiles_k, (unsigned)g.tiles_n);
  float* out = g.split > 1 ? ws : (float*)y;
  hipLaunchKernelGGL(fn, grid, dim3(g.threads), g.lds_bytes, (hipStream_t)stream, (const float*)xin,
                     (const float*)w, out, a);
  if (hipGetLastError() != hipSuccess) return -1;
  if (g.split > 1) return launch_split_reduce(ws, (float*)y, x.ny, g.split, stream);
  return 0;
}

}  // namespace ct
