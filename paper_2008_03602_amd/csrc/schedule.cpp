// Host rules of the tuning loop: knob grids, the validator and launch
// geometry of every kernel family, seeded candidate sampling, winner
// selection and CU-mask construction. No HIP calls in this file.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "ct_internal.h"

namespace ct {

// ---------------------------------------------------------------- knob tables
// Knob kinds follow the paper's list of what a tuner chooses for an operator
// (section 2.1): loop tiles and ordering, caching (here: LDS staging),
// unrolling, threading (waves, per-thread micro-tiles) and matrix units.
static const FamilyDef kFamilies[CT_NUM_FAMILIES] = {
    {CT_FAM_DIRECT_F32, "direct_f32", direct_knob::COUNT,
     {{"toh", 6, {1, 2, 4, 7, 8, 14}},
      {"tow", 8, {4, 7, 8, 14, 16, 28, 32, 56}},
      {"tk", 5, {4, 8, 16, 32, 64}},
      {"mk", 4, {1, 2, 4, 8}},
      {"mw", 3, {1, 2, 4}},
      {"lds", 2, {0, 1}},
      {"ct", 6, {1, 2, 4, 8, 16, 32}},
      {"split", 3, {1, 2, 4}},
      {"unroll", 2, {1, 2}}}},
    {CT_FAM_DEPTHWISE_F32, "depthwise_f32", dw_knob::COUNT,
     {{"tc", 5, {1, 2, 4, 8, 16}},
      {"toh", 8, {1, 2, 4, 7, 8, 14, 16, 28}},
      {"tow", 9, {4, 7, 8, 14, 16, 28, 32, 56, 64}},
      {"vec", 3, {1, 2, 4}},
      {"rpt", 3, {1, 2, 4}},
      {"lds", 2, {0, 1}},
      {"nb", 3, {1, 2, 4}},
      {"order", 2, {0, 1}},
      {"q4", 2, {0, 1}}}},
    {CT_FAM_IGEMM_BF16, "igemm_mfma_bf16", bf16_knob::COUNT,
     {{"mfma", 2, {16, 32}},
      {"tm", 3, {1, 2, 4}},
      {"tn", 3, {1, 2, 4}},
      {"wm", 3, {1, 2, 4}},
      {"wn", 3, {1, 2, 4}},
      {"kc", 3, {32, 64, 128}},
      {"lds", 2, {0, 1}},
      {"split", 3, {1, 2, 4}},
      {"swizzle", 2, {0, 1}}}},
    // tn 7 and the tile widths 7..56 give pixel tiles of whole rows of the
    // 7*2^k-wide maps of these networks (two 56-pixel rows = 7 MFMA tiles)
    {CT_FAM_IGEMM_F32, "igemm_mfma_f32", f32g_knob::COUNT,
     {{"mfma", 2, {16, 32}},
      {"tm", 3, {1, 2, 4}},
      {"tn", 4, {1, 2, 4, 7}},
      {"wm", 3, {1, 2, 4}},
      {"wn", 3, {1, 2, 4}},
      {"ws", 3, {1, 2, 4}},
      {"tpw", 8, {7, 8, 14, 16, 28, 32, 56, 64}},
      {"cpc", 7, {1, 2, 4, 8, 16, 32, 64}},
      {"stages", 3, {1, 2, 3}},  // 3: two stages, copies issued by four loader waves
      {"split", 4, {1, 2, 4, 8}}}},
};

const FamilyDef* family_def(int family) {
  if (family < 1 || family > CT_NUM_FAMILIES) return nullptr;
  return &kFamilies[family - 1];
}

int64_t family_grid_size(const FamilyDef& f) {
  int64_t n = 1;
  for (int i = 0; i < f.nknobs; ++i) n *= f.knobs[i].nvals;
  return n;
}

// ------------------------------------------------------------------ op facts
static int64_t out_extent(int64_t in, int64_t pad, int64_t dil, int64_t ker, int64_t stride) {
  int64_t span = in + 2 * pad - dil * (ker - 1) - 1;
  return span < 0 ? 0 : span / stride + 1;
}

bool derive_op(const ct_op& op, OpX* x, std::string* why) {
  auto bad = [&](const char* m) { if (why) *why = m; return false; };
  if (op.n <= 0 || op.c <= 0 || op.h <= 0 || op.w <= 0 || op.k <= 0 || op.r <= 0 || op.s <= 0)
    return bad("op: sizes must be positive");
  if (op.stride_h <= 0 || op.stride_w <= 0 || op.dil_h <= 0 || op.dil_w <= 0)
    return bad("op: stride and dilation must be positive");
  if (op.pad_h < 0 || op.pad_w < 0) return bad("op: padding must be >= 0");
  if (op.groups <= 0 || op.c % op.groups || op.k % op.groups)
    return bad("op: groups must divide C and K");
  if (op.dtype != CT_DT_F32 && op.dtype != CT_DT_BF16) return bad("op: unknown dtype");
  if (op.layout != CT_LAYOUT_NCHW && op.layout != CT_LAYOUT_NHWC) return bad("op: unknown layout");
  x->op = op;
  x->oh = out_extent(op.h, op.pad_h, op.dil_h, op.r, op.stride_h);
  x->ow = out_extent(op.w, op.pad_w, op.dil_w, op.s, op.stride_w);
  if (x->oh <= 0 || x->ow <= 0) return bad("op: empty output");
  x->cg = op.c / op.groups;
  x->kg = op.k / op.groups;
  x->kred = x->cg * op.r * op.s;
  x->npix = (int64_t)op.n * x->oh * x->ow;
  x->nx = (int64_t)op.n * op.c * op.h * op.w;
  x->nw = (int64_t)op.k * x->cg * op.r * op.s;
  x->ny = (int64_t)op.n * op.k * x->oh * x->ow;
  x->elem_bytes = op.dtype == CT_DT_BF16 ? 2 : 4;
  const int64_t lim = (int64_t)1 << 31;
  if (x->nx >= lim || x->nw >= lim || x->ny >= lim) return bad("op: tensor exceeds 2^31 elements");
  return true;
}

bool family_applies(int family, const OpX& x) {
  const ct_op& o = x.op;
  switch (family) {
    case CT_FAM_DIRECT_F32:
    case CT_FAM_IGEMM_F32:
      return o.dtype == CT_DT_F32 && o.layout == CT_LAYOUT_NCHW && o.groups == 1;
    case CT_FAM_DEPTHWISE_F32:
      return o.dtype == CT_DT_F32 && o.layout == CT_LAYOUT_NCHW && o.groups == o.c && o.k == o.c;
    case CT_FAM_IGEMM_BF16:
      return o.dtype == CT_DT_BF16 && o.layout == CT_LAYOUT_NHWC && o.groups == 1 && o.r == 1 &&
             o.s == 1 && o.pad_h == 0 && o.pad_w == 0 && o.c % 8 == 0;
    default:
      return false;
  }
}

Spec op_spec(const OpX& x) {
  const ct_op& o = x.op;
  if (o.dil_h != 1 || o.dil_w != 1 || o.stride_h != o.stride_w) return SPEC_GENERIC;
  if (o.r == 1 && o.s == 1 && o.pad_h == 0 && o.pad_w == 0) {
    if (o.stride_h == 1) return SPEC_1X1_S1;
    if (o.stride_h == 2) return SPEC_1X1_S2;
  }
  if (o.r == 3 && o.s == 3 && o.pad_h == 1 && o.pad_w == 1) {
    if (o.stride_h == 1) return SPEC_3X3_S1;
    if (o.stride_h == 2) return SPEC_3X3_S2;
  }
  return SPEC_GENERIC;
}

// ------------------------------------------------------------------ geometry
static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Smallest value of the knob list that is >= extent (the largest if none is):
// tiles may overhang the tensor by less than one grid step, never more.
static int32_t fit(const KnobDef& k, int64_t extent) {
  for (int i = 0; i < k.nvals; ++i)
    if (k.vals[i] >= extent) return k.vals[i];
  return k.vals[k.nvals - 1];
}
static int32_t fit_pow2(int64_t extent, int32_t lo, int32_t hi) {
  int32_t v = lo;
  while (v < extent && v < hi) v *= 2;
  return v;
}

// Block size that leaves room for an MFMA accumulator tile of acc_regs
// registers per lane (the kernels declare the same bound).
static int mfma_thread_limit(int acc_regs) { return acc_regs <= 64 ? 512 : 256; }

static bool knobs_in_table(const FamilyDef& f, const ct_schedule& s) {
  for (int i = 0; i < f.nknobs; ++i) {
    bool ok = false;
    for (int j = 0; j < f.knobs[i].nvals; ++j) ok |= (s.knob[i] == f.knobs[i].vals[j]);
    if (!ok) return false;
  }
  return true;
}

// Splits `chunks` reduction chunks into `split` contiguous ranges; every range
// must be non-empty.
static bool split_ok(int64_t chunks, int split, int64_t* cps) {
  if (split < 1 || split > chunks) return false;
  *cps = cdiv(chunks, split);
  return (split - 1) * (*cps) < chunks;
}

#define REJECT(msg)              \
  do {                           \
    if (why) *why = (msg);       \
    return CT_S_INVALID;         \
  } while (0)

static int geom_direct(const OpX& x, const ct_schedule& s, Geom* g, std::string* why) {
  using namespace direct_knob;
  const FamilyDef& f = *family_def(CT_FAM_DIRECT_F32);
  const ct_op& o = x.op;
  const int toh = s.knob[TOH], tow = s.knob[TOW], tk = s.knob[TK], mk = s.knob[MK], mw = s.knob[MW];
  const int lds = s.knob[LDS], ctile = s.knob[CT], split = s.knob[SPLIT];
  if (tk % mk) REJECT("tk not a multiple of mk");
  if (tow % mw) REJECT("tow not a multiple of mw");
  if (toh > fit(f.knobs[TOH], x.oh)) REJECT("toh exceeds the output height");
  if (tow > fit(f.knobs[TOW], x.ow)) REJECT("tow exceeds the output width");
  if (tk > fit(f.knobs[TK], o.k)) REJECT("tk exceeds K");
  if (ctile > fit(f.knobs[CT], x.cg)) REJECT("ct exceeds C");
  if (4 * x.nx >= ((int64_t)1 << 31) || 4 * x.nw >= ((int64_t)1 << 31))
    REJECT("tensor too large for 32-bit buffer offsets");
  const int64_t threads = (int64_t)(tk / mk) * (toh * tow / mw);
  // fewer threads than half a wave only where the tile already spans the whole
  // op (an op smaller than a wave): the block's other lanes stay masked off
  const bool spans = toh >= x.oh && tow >= x.ow && tk >= o.k;
  if ((threads < kMinThreads && !spans) || threads > kMaxThreads) REJECT("threads per block out of range");
  // the register budget of the kernel's launch bounds: an accumulator tile of
  // 16 or more outputs per thread allows at most 512 threads
  if (mk * mw >= 16 && threads > 512) REJECT("too many threads for the accumulator tile");
  const int64_t chunks = cdiv(x.cg, ctile);
  int64_t cps = 0;
  if (!split_ok(chunks, split, &cps)) REJECT("split leaves an empty channel range");
  g->ih_t = (int)((toh - 1) * o.stride_h + (o.r - 1) * o.dil_h + 1);
  g->iw_t = (int)((tow - 1) * o.stride_w + (o.s - 1) * o.dil_w + 1);
  int64_t lbytes = 0;
  if (lds) lbytes = 4 * ((int64_t)ctile * g->ih_t * g->iw_t + (int64_t)tk * ctile * o.r * o.s);
  if (lbytes > kMaxLdsBytes) REJECT("LDS tile too large");
  g->tiles_h = cdiv(x.oh, toh);
  g->tiles_w = cdiv(x.ow, tow);
  g->tiles_k = cdiv(o.k, tk);
  g->tiles_n = (int64_t)o.n * split;
  if (g->tiles_k > 65535 || g->tiles_n > 65535) REJECT("grid too large");
  g->threads = (int)threads;
  g->lds_bytes = (int)lbytes;
  g->blocks = g->tiles_h * g->tiles_w * g->tiles_k * g->tiles_n;
  g->split = split;
  g->chunks = (int)chunks;
  g->chunks_per_split = (int)cps;
  return CT_OK;
}

static int geom_depthwise(const OpX& x, const ct_schedule& s, Geom* g, std::string* why) {
  using namespace dw_knob;
  const FamilyDef& f = *family_def(CT_FAM_DEPTHWISE_F32);
  const ct_op& o = x.op;
  const int tc = s.knob[TC], toh = s.knob[TOH], tow = s.knob[TOW], vec = s.knob[VEC];
  const int rpt = s.knob[RPT], lds = s.knob[LDS], nb = s.knob[NB];
  if (s.knob[Q4]) {
    // 4 consecutive output columns per thread, registers only, 3x3 pad 1
    if (g->spec != SPEC_3X3_S1 && g->spec != SPEC_3X3_S2) REJECT("q4 needs a 3x3 filter with pad 1");
    if (vec != 4) REJECT("q4 takes 4 output columns per thread (vec 4)");
    if (lds) REJECT("q4 reads rows into registers (lds 0)");
  }
  if (tow % vec) REJECT("tow not a multiple of vec");
  if (toh % rpt) REJECT("toh not a multiple of rpt");
  if (toh > fit(f.knobs[TOH], x.oh)) REJECT("toh exceeds the output height");
  if (tow > fit(f.knobs[TOW], x.ow)) REJECT("tow exceeds the output width");
  if (tc > fit(f.knobs[TC], o.c)) REJECT("tc exceeds C");
  if (nb > fit(f.knobs[NB], o.n)) REJECT("nb exceeds N");
  const int64_t threads = (int64_t)tc * nb * (toh / rpt) * (tow / vec);
  const bool spans = tc >= o.c && nb >= o.n && toh >= x.oh && tow >= x.ow;  // as for the direct family
  if ((threads < kMinThreads && !spans) || threads > kMaxThreads) REJECT("threads per block out of range");
  // the strided kernel's 16 outputs per thread need 256 registers: 512 threads at most
  if (!s.knob[Q4] && vec * rpt >= 16 && threads > 512) REJECT("too many threads for 16 outputs per thread");
  g->ih_t = (int)((toh - 1) * o.stride_h + (o.r - 1) * o.dil_h + 1);
  g->iw_t = (int)((tow - 1) * o.stride_w + (o.s - 1) * o.dil_w + 1);
  int64_t lbytes = lds ? 4 * (int64_t)tc * nb * g->ih_t * g->iw_t : 0;
  if (lbytes > kMaxLdsBytes) REJECT("LDS tile too large");
  g->tiles_h = cdiv(x.oh, toh);
  g->tiles_w = cdiv(x.ow, tow);
  g->tiles_c = cdiv(o.c, tc);
  g->tiles_n = cdiv(o.n, nb);
  g->threads = (int)threads;
  g->lds_bytes = (int)lbytes;
  g->blocks = g->tiles_h * g->tiles_w * g->tiles_c * g->tiles_n;
  if (g->blocks >= ((int64_t)1 << 31)) REJECT("grid too large");
  g->split = 1;
  return CT_OK;
}

static int geom_igemm_bf16(const OpX& x, const ct_schedule& s, Geom* g, std::string* why) {
  using namespace bf16_knob;
  const FamilyDef& f = *family_def(CT_FAM_IGEMM_BF16);
  const ct_op& o = x.op;
  const int mf = s.knob[MF], tm = s.knob[TM], tn = s.knob[TN], wm = s.knob[WM], wn = s.knob[WN];
  const int kc = s.knob[KC], lds = s.knob[LDS], split = s.knob[SPLIT];
  const int bm = wm * tm * mf, bn = wn * tn * mf;
  if (bm > fit_pow2(x.npix, 16, 1024)) REJECT("block rows exceed the pixel count");
  if (bn > fit_pow2(o.k, 16, 512)) REJECT("block columns exceed K");
  if (kc > fit(f.knobs[KC], o.c)) REJECT("kc exceeds C");
  const int acc_regs = tm * tn * (mf == 32 ? 16 : 4);
  if (acc_regs > 128) REJECT("accumulator tile too large");
  const int threads = 64 * wm * wn;
  if (threads > mfma_thread_limit(acc_regs)) REJECT("too many threads for the accumulator tile");
  if (!lds) {
    const int steps = kc / (mf == 32 ? 16 : 32);
    if (steps > 4 || steps * (tm + tn) > 16) REJECT("too many fragments held in registers");
  }
  // the epilogue's buffer stores address a wave tile of y in 32-bit bytes
  if (4 * x.ny >= ((int64_t)1 << 31)) REJECT("output too large for 32-bit buffer offsets");
  const int64_t chunks = cdiv(o.c, kc);
  int64_t cps = 0;
  if (!split_ok(chunks, split, &cps)) REJECT("split leaves an empty channel range");
  int64_t lbytes = 0;
  if (lds) {
    lbytes = 2 * (int64_t)(bm + bn) * (kc + 8);
    const int64_t vecs_a = (int64_t)bm * (kc / 8), vecs_b = (int64_t)bn * (kc / 8);
    g->a_loads = (int)cdiv(vecs_a, threads);
    g->b_loads = (int)cdiv(vecs_b, threads);
    if (g->a_loads > kMaxLoadsPerThread || g->b_loads > kMaxLoadsPerThread)
      REJECT("too many staged loads per thread");
  } else {
    g->a_loads = g->b_loads = 0;
  }
  if (lbytes > kMaxLdsBytes) REJECT("LDS tile too large");
  g->bm = bm;
  g->bn = bn;
  g->tiles_h = cdiv(x.npix, bm);  // row tiles
  g->tiles_k = cdiv(o.k, bn);     // column tiles
  g->tiles_n = split;
  if (g->tiles_k > 65535) REJECT("grid too large");
  g->threads = threads;
  g->lds_bytes = (int)lbytes;
  g->blocks = g->tiles_h * g->tiles_k * split;
  g->split = split;
  g->chunks = (int)chunks;
  g->chunks_per_split = (int)cps;
  return CT_OK;
}

static int geom_igemm_f32(const OpX& x, const ct_schedule& s, Geom* g, std::string* why) {
  using namespace f32g_knob;
  const FamilyDef& f = *family_def(CT_FAM_IGEMM_F32);
  const ct_op& o = x.op;
  const int mf = s.knob[MF], tm = s.knob[TM], tn = s.knob[TN], wm = s.knob[WM], wn = s.knob[WN];
  const int wsplit = s.knob[WS], tpw = s.knob[TPW], cpc = s.knob[CPC], stages = s.knob[STAGES];
  const int split = s.knob[SPLIT];
  const int bm = wm * tm * mf;  // output channels per block
  const int bn = wn * tn * mf;  // output pixels per block: a tph x tpw rectangle
  if (bm > fit_pow2(o.k, 16, 512)) REJECT("block rows exceed K");
  if (bn % tpw) REJECT("pixel tile is not a whole number of rows");
  const int tph = bn / tpw;
  if (tpw > fit_pow2(x.ow, 8, 64)) REJECT("pixel tile wider than the output");
  if (tph > fit_pow2(x.oh, 1, 1024)) REJECT("pixel tile taller than the output");
  if (cpc > fit(f.knobs[CPC], x.cg)) REJECT("channels per chunk exceed C");
  // every chunk holds the same channels: no partial last chunk to mask
  if (cpc < x.cg && x.cg % cpc) REJECT("channels per chunk do not divide C");
  const int acc_regs = tm * tn * (mf == 32 ? 16 : 4);
  if (acc_regs > 128) REJECT("accumulator tile too large");
  // stages 3: the MFMA waves only compute, and four more waves build the copy
  // plan and issue every copy into the two stages
  const bool loaders = stages == 3;
  const int lds_stages = std::min(stages, 2);
  const int mfma_threads = 64 * wm * wn * wsplit;
  if (mfma_threads > (loaders ? 256 : mfma_thread_limit(acc_regs)))
    REJECT("too many threads for the accumulator tile");
  if (loaders && acc_regs > kLoaderMaxAcc) REJECT("accumulator tile too large beside loader waves");
  const int threads = mfma_threads + (loaders ? 256 : 0);
  // channels per chunk padded to whole k-steps for every reduction group
  const int kstep = mf == 32 ? 2 : 4;
  const int cpcp = (int)cdiv(cpc, kstep * wsplit) * kstep * wsplit;
  if (cpcp > 2 * cpc && cpc < x.cg) REJECT("chunk padding exceeds the chunk");
  const int rs = o.r * o.s;
  const int ht = (tph - 1) * o.stride_h + (o.r - 1) * o.dil_h + 1;
  const int wt = (tpw - 1) * o.stride_w + (o.s - 1) * o.dil_w + 1;
  // Copies move 64 units per wave instruction (a unit is 1 word, or 4 words
  // with 16-byte copies): the halo as a flat array padded to whole copies of
  // every wave, the filter row by row in 64-unit segments.
  // Halo: 16-byte copies need every unit wholly inside or outside the image,
  // so W and the tile's first column are multiples of 4 (rows then start
  // HSHIFT columns before the tile's first input column).
  // Filter: 16-byte copies need 16-byte-aligned rows in global memory and LDS.
  // Bank padding (32 banks, half a wave per LDS pass): with 16x16x4 MFMAs a
  // pass reads 16 filter rows at two k offsets R*S apart and 16 pixels at two
  // channels, so the channel pitch is 16 (mod 32) and the row pitch 2 (mod 32)
  // (4 (mod 8) for 16-byte rows: a 2-way conflict); with 32x32x2 a pass reads
  // 32 rows at one k, so the row pitch is odd. With 8-pixel rows (stride 1)
  // the 16 pixels span two halo rows: a pass reads 2 channels x 2 rows x 8
  // columns, which fall in distinct banks when the channel and row pitches
  // are 8 and 16 (mod 32), so a row pitch of 16 takes a channel pitch of 8.
  const int nw = loaders ? 4 : threads / 64;  // waves that copy
  const int cl = std::min<int>(cpc, (int)x.cg);
  const bool vec_h = o.w % 4 == 0 && (tpw * o.stride_w) % 4 == 0;
  const int hshift = vec_h ? (4 - o.pad_w % 4) % 4 : 0;
  const int rw = vec_h ? (int)cdiv(hshift + wt, 4) * 4 : wt;
  const int rows = ht * rw;
  const bool two_rows = mf == 16 && tpw == 8 && o.stride_h == 1 && o.stride_w == 1 && o.dil_w == 1 && rw % 32 == 16;
  const int pp = mf == 16 ? rows + (((two_rows ? 8 : 16) - rows) & 31) : (vec_h ? (int)cdiv(rows, 4) * 4 : rows);
  const int vh = vec_h ? 4 : 1;
  const int jw = rs * cpcp;
  const bool vec_f = mf == 16 && jw % 4 == 0 && x.kred % 4 == 0 && (cl * rs) % 4 == 0 &&
                     (cpc >= x.cg || (cpc * rs) % 4 == 0);
  const int vf = vec_f ? 4 : 1;
  const int nseg = (int)cdiv(jw, 64 * vf);
  int lda;
  if (vec_f) {
    const int l4 = (int)cdiv(jw, 4) * 4;
    lda = (l4 / 4) % 2 ? l4 : l4 + 4;
  } else {
    const int lrow = std::max(jw, 64);
    lda = mf == 16 ? lrow + ((2 - lrow) & 31) : (lrow | 1);
  }
  const int64_t units = (int64_t)cpcp * (pp / vh);
  g->a_loads = (int)cdiv(units, 64 * nw);            // halo copies per copying wave per chunk
  g->b_loads = (int)cdiv((int64_t)bm * nseg, nw);    // filter copies per copying wave per chunk
  if (g->a_loads > 16) REJECT("too many halo copies per wave");
  if (g->b_loads > 16) REJECT("too many filter copies per wave");
  const int64_t xs_pad = (int64_t)g->a_loads * 64 * nw * vh;
  if (4 * x.nx >= ((int64_t)1 << 31) || 4 * x.nw >= ((int64_t)1 << 31))
    REJECT("tensor too large for 32-bit buffer offsets");
  if (4 * x.ny >= ((int64_t)1 << 31)) REJECT("output too large for 32-bit buffer offsets");
  const int64_t chunks = cdiv(x.cg, cpc);
  int64_t cps = 0;
  if (!split_ok(chunks, split, &cps)) REJECT("split leaves an empty reduction range");
  const int64_t stage_bytes = 4 * (xs_pad + (int64_t)bm * lda);
  const int64_t red_bytes = wsplit > 1 ? 4 * (int64_t)(wsplit - 1) * bm * bn : 0;
  const int64_t lbytes = std::max(lds_stages * stage_bytes, red_bytes);
  if (lbytes > kMaxLdsBytes) REJECT("LDS tile too large");
  g->xs_pad = (int)xs_pad;
  g->f_nseg = nseg;
  g->hpp = pp;
  g->hrw = rw;
  g->hshift = hshift;
  g->vec_h = vec_h;
  g->vec_f = vec_f;
  g->bm = bm;
  g->bn = bn;
  g->cpcp = cpcp;
  g->lda = lda;
  g->tph = tph;
  g->tpw = tpw;
  g->ih_t = ht;
  g->iw_t = wt;
  g->tiles_h = cdiv(x.oh, tph);
  g->tiles_w = cdiv(x.ow, tpw);
  g->tiles_k = cdiv(o.k, bm);
  g->tiles_n = split;
  if (g->tiles_k > 65535) REJECT("grid too large");
  // the kernel splits blockIdx.x with an fp32 reciprocal, exact below 2^22
  if ((int64_t)o.n * g->tiles_h * g->tiles_w >= ((int64_t)1 << 22)) REJECT("grid too large");
  g->threads = threads;
  g->lds_bytes = (int)lbytes;
  g->blocks = (int64_t)o.n * g->tiles_h * g->tiles_w * g->tiles_k * split;
  // the XCD-band renumbering splits the linear block index the same way
  if (g->blocks >= ((int64_t)1 << 22)) REJECT("grid too large");
  g->split = split;
  g->chunks = (int)chunks;
  g->chunks_per_split = (int)cps;
  return CT_OK;
}

int compute_geom(const OpX& x, const ct_schedule& s, Geom* g, std::string* why) {
  const FamilyDef* f = family_def(s.family);
  if (!f) REJECT("unknown family");
  if (!family_applies(s.family, x)) REJECT("family does not fit the op's layout/dtype/groups");
  if (!knobs_in_table(*f, s)) REJECT("knob value outside the family's table");
  std::memset(g, 0, sizeof(*g));
  g->family = s.family;
  g->spec = op_spec(x);
  g->split = 1;
  int rc = CT_S_INVALID;
  switch (s.family) {
    case CT_FAM_DIRECT_F32: rc = geom_direct(x, s, g, why); break;
    case CT_FAM_DEPTHWISE_F32: rc = geom_depthwise(x, s, g, why); break;
    case CT_FAM_IGEMM_BF16: rc = geom_igemm_bf16(x, s, g, why); break;
    case CT_FAM_IGEMM_F32: rc = geom_igemm_f32(x, s, g, why); break;
  }
  if (rc != CT_OK) return rc;
  if (g->blocks <= 0) REJECT("empty grid");
  g->kernels = g->split > 1 ? 2 : 1;
  g->ws_floats = g->split > 1 ? (int64_t)g->split * x.ny : 0;
  return CT_OK;
}

uint64_t splitmix64_next(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

}  // namespace ct

// ================================================================= C ABI part
using namespace ct;

extern "C" {

int ct_build_cu_mask(int num_cus, double fraction, int slot, uint32_t* mask, int words) {
  if (!mask || num_cus <= 0 || slot < 0 || !(fraction > 0.0) || fraction > 1.0) {
    set_error("ct_build_cu_mask: bad argument");
    return CT_E_ARG;
  }
  if ((int64_t)words * 32 < num_cus) {
    set_error("ct_build_cu_mask: mask has fewer bits than the device has CUs");
    return CT_E_ARG;
  }
  const int64_t m = std::llround((double)num_cus * fraction);
  if (m <= 0 || (int64_t)(slot + 1) * m > num_cus) {
    set_error("ct_build_cu_mask: slot does not fit on the device");
    return CT_E_ARG;
  }
  std::memset(mask, 0, sizeof(uint32_t) * words);
  for (int64_t b = (int64_t)slot * m; b < (int64_t)(slot + 1) * m; ++b) mask[b / 32] |= 1u << (b % 32);
  return CT_OK;
}

int ct_grid_info(int family, int32_t* num_knobs, int64_t* grid_size) {
  const FamilyDef* f = family_def(family);
  if (!f) { set_error("ct_grid_info: unknown family"); return CT_E_ARG; }
  if (num_knobs) *num_knobs = f->nknobs;
  if (grid_size) *grid_size = family_grid_size(*f);
  return CT_OK;
}

int ct_knob_values(int family, int knob, int32_t* values, int32_t cap, int32_t* count) {
  const FamilyDef* f = family_def(family);
  if (!f || knob < 0 || knob >= f->nknobs) { set_error("ct_knob_values: bad family or knob"); return CT_E_ARG; }
  const KnobDef& k = f->knobs[knob];
  if (count) *count = k.nvals;
  for (int i = 0; i < k.nvals && i < cap && values; ++i) values[i] = k.vals[i];
  return CT_OK;
}

int ct_grid_decode(int family, int64_t index, ct_schedule* out) {
  const FamilyDef* f = family_def(family);
  if (!f || !out || index < 0 || index >= family_grid_size(*f)) {
    set_error("ct_grid_decode: bad family or index");
    return CT_E_ARG;
  }
  std::memset(out, 0, sizeof(*out));
  out->family = family;
  for (int i = f->nknobs - 1; i >= 0; --i) {  // last knob = least significant digit
    const int r = f->knobs[i].nvals;
    out->knob[i] = f->knobs[i].vals[index % r];
    index /= r;
  }
  return CT_OK;
}

int ct_grid_encode(const ct_schedule* s, int64_t* index) {
  const FamilyDef* f = s ? family_def(s->family) : nullptr;
  if (!f || !index) { set_error("ct_grid_encode: bad schedule"); return CT_E_ARG; }
  int64_t idx = 0;
  for (int i = 0; i < f->nknobs; ++i) {
    int d = -1;
    for (int j = 0; j < f->knobs[i].nvals; ++j)
      if (f->knobs[i].vals[j] == s->knob[i]) d = j;
    if (d < 0) { set_error("ct_grid_encode: knob value outside the table"); return CT_E_ARG; }
    idx = idx * f->knobs[i].nvals + d;
  }
  *index = idx;
  return CT_OK;
}

int ct_validate(const ct_op* op, const ct_schedule* s) {
  if (!op || !s) { set_error("ct_validate: null argument"); return CT_E_ARG; }
  OpX x;
  std::string why;
  if (!derive_op(*op, &x, &why)) { set_error(why); return CT_E_ARG; }
  Geom g;
  int rc = compute_geom(x, *s, &g, &why);
  if (rc != CT_OK) set_error("invalid schedule: " + why);
  return rc;
}

int ct_launch_shape(const ct_op* op, const ct_schedule* s, int32_t* lds_bytes, int32_t* threads,
                    int64_t* blocks, int32_t* kernels) {
  if (!op || !s) { set_error("ct_launch_shape: null argument"); return CT_E_ARG; }
  OpX x;
  std::string why;
  if (!derive_op(*op, &x, &why)) { set_error(why); return CT_E_ARG; }
  Geom g;
  if (compute_geom(x, *s, &g, &why) != CT_OK) { set_error("invalid schedule: " + why); return CT_E_ARG; }
  if (lds_bytes) *lds_bytes = g.lds_bytes;
  if (threads) *threads = g.threads;
  if (blocks) *blocks = g.blocks;
  if (kernels) *kernels = g.kernels;
  return CT_OK;
}

int ct_kernel_name(const ct_op* op, const ct_schedule* s, char* buf, int cap) {
  if (!op || !s || !buf || cap <= 0) { set_error("ct_kernel_name: bad argument"); return CT_E_ARG; }
  OpX x;
  std::string why;
  if (!derive_op(*op, &x, &why)) { set_error(why); return CT_E_ARG; }
  Geom g;
  if (compute_geom(x, *s, &g, &why) != CT_OK) { set_error("invalid schedule: " + why); return CT_E_ARG; }
  const int* k = s->knob;
  auto tf = [](int v) { return v ? "true" : "false"; };
  char tmp[128];
  switch (s->family) {
    case CT_FAM_DIRECT_F32:
      std::snprintf(tmp, sizeof tmp, "direct_f32_kernel<%d, %d, %s, %d, %d>", k[direct_knob::MK],
                    k[direct_knob::MW], tf(k[direct_knob::LDS]), (int)g.spec, k[direct_knob::UNR]);
      break;
    case CT_FAM_DEPTHWISE_F32: {
      const int spec = g.spec == SPEC_3X3_S1 ? 3 : (g.spec == SPEC_3X3_S2 ? 4 : 0);
      if (k[dw_knob::Q4])
        std::snprintf(tmp, sizeof tmp, "depthwise_q4_kernel<%d, %d>", spec == SPEC_3X3_S2 ? 2 : 1, k[dw_knob::RPT]);
      else
        std::snprintf(tmp, sizeof tmp, "depthwise_f32_kernel<%d, %d, %s, %d>", k[dw_knob::VEC], k[dw_knob::RPT],
                      tf(k[dw_knob::LDS]), spec);
      break;
    }
    case CT_FAM_IGEMM_BF16:
      std::snprintf(tmp, sizeof tmp, "igemm_bf16_kernel<%d, %d, %d, %s>", k[bf16_knob::MF], k[bf16_knob::TM],
                    k[bf16_knob::TN], tf(k[bf16_knob::LDS]));
      break;
    default:
      std::snprintf(tmp, sizeof tmp, "igemm_f32_kernel<%d, %d, %d, %d, %d>", k[f32g_knob::MF], k[f32g_knob::TM],
                    k[f32g_knob::TN], k[f32g_knob::STAGES], (int)g.spec);
  }
  std::snprintf(buf, (size_t)cap, "%s", tmp);
  return CT_OK;
}

static int valid_space(const ct_op* op, std::vector<ct_schedule>* out) {
  OpX x;
  std::string why;
  if (!derive_op(*op, &x, &why)) { set_error(why); return CT_E_ARG; }
  for (int fam = 1; fam <= CT_NUM_FAMILIES; ++fam) {
    if (!family_applies(fam, x)) continue;
    const FamilyDef& f = *family_def(fam);
    const int64_t n = family_grid_size(f);
    ct_schedule s;
    Geom g;
    for (int64_t i = 0; i < n; ++i) {
      ct_grid_decode(fam, i, &s);
      if (compute_geom(x, s, &g, nullptr) == CT_OK) out->push_back(s);
    }
  }
  return CT_OK;
}

int ct_grid_size(const ct_op* op, int family, int64_t* n) {
  if (!op || !n) { set_error("ct_grid_size: null argument"); return CT_E_ARG; }
  const FamilyDef* f = family_def(family);
  if (!f) { set_error("ct_grid_size: unknown family"); return CT_E_ARG; }
  OpX x;
  std::string why;
  if (!derive_op(*op, &x, &why)) { set_error(why); return CT_E_ARG; }
  *n = 0;
  if (!family_applies(family, x)) return CT_OK;
  const int64_t size = family_grid_size(*f);
  ct_schedule s;
  Geom g;
  for (int64_t i = 0; i < size; ++i) {
    ct_grid_decode(family, i, &s);
    if (compute_geom(x, s, &g, nullptr) == CT_OK) ++*n;
  }
  return CT_OK;
}

int ct_valid_space(const ct_op* op, ct_schedule* out, int64_t cap, int64_t* count) {
  if (!op || !count) { set_error("ct_valid_space: null argument"); return CT_E_ARG; }
  std::vector<ct_schedule> v;
  int rc = valid_space(op, &v);
  if (rc) return rc;
  *count = (int64_t)v.size();
  if (out) std::memcpy(out, v.data(), sizeof(ct_schedule) * (size_t)std::min<int64_t>(cap, v.size()));
  return CT_OK;
}

int ct_sample(const ct_op* op, uint64_t seed, int32_t config_id, int32_t layer_id, int32_t n,
              ct_schedule* out, int32_t* n_out) {
  if (!op || !out || !n_out || n < 0) { set_error("ct_sample: bad argument"); return CT_E_ARG; }
  std::vector<ct_schedule> v;
  int rc = valid_space(op, &v);
  if (rc) return rc;
  // the space is family by family: [begin, end) of each family present
  std::vector<size_t> fb, fe;
  for (size_t i = 0; i < v.size(); ++i) {
    if (i == 0 || v[i].family != v[i - 1].family) {
      if (i) fe.push_back(i);
      fb.push_back(i);
    }
  }
  if (!v.empty()) fe.push_back(v.size());
  const size_t nf = fb.size();
  // quotas: equal shares, the remainder to the first families, a family's
  // unused share handed on until n is reached or every family is exhausted
  std::vector<uint64_t> q(nf, 0);
  uint64_t rem = std::min<uint64_t>((uint64_t)n, v.size());
  while (rem > 0) {
    std::vector<size_t> act;
    for (size_t f = 0; f < nf; ++f)
      if (q[f] < fe[f] - fb[f]) act.push_back(f);
    const uint64_t base = rem / act.size(), extra = rem % act.size();
    for (size_t i = 0; i < act.size(); ++i) {
      const size_t f = act[i];
      const uint64_t add = std::min<uint64_t>(base + (i < extra ? 1 : 0), (fe[f] - fb[f]) - q[f]);
      q[f] += add;
      rem -= add;
    }
  }
  // per family: partial Fisher-Yates of its part of the space
  const uint64_t state0 = seed ^ (0x9E3779B97F4A7C15ull * (uint64_t)(1 + (int64_t)config_id)) ^
                          (0xC0FFEEull << 32) ^ (uint64_t)(uint32_t)layer_id;
  std::vector<std::vector<ct_schedule>> picks(nf);
  for (size_t f = 0; f < nf; ++f) {
    uint64_t state = state0 ^ (0xD1B54A32D192ED03ull * (uint64_t)v[fb[f]].family);
    splitmix64_next(&state);  // the first output is discarded
    const uint64_t size = fe[f] - fb[f];
    ct_schedule* part = v.data() + fb[f];
    for (uint64_t i = 0; i < q[f]; ++i) {
      const uint64_t j = i + splitmix64_next(&state) % (size - i);
      std::swap(part[i], part[j]);
      picks[f].push_back(part[i]);
    }
  }
  // interleaved: the k-th pick of every family in family order, then k + 1
  int32_t m = 0;
  for (uint64_t k = 0; m < (int32_t)std::min<uint64_t>((uint64_t)n, v.size()); ++k)
    for (size_t f = 0; f < nf; ++f)
      if (k < q[f]) out[m++] = picks[f][k];
  *n_out = m;
  return CT_OK;
}

int ct_sample_uniform(const ct_op* op, uint64_t seed, int32_t config_id, int32_t layer_id, int32_t n,
                      ct_schedule* out, int32_t* n_out) {
  if (!op || !out || !n_out || n < 0) { set_error("ct_sample_uniform: bad argument"); return CT_E_ARG; }
  std::vector<ct_schedule> v;
  int rc = valid_space(op, &v);
  if (rc) return rc;
  uint64_t state = seed ^ (0x9E3779B97F4A7C15ull * (uint64_t)(1 + (int64_t)config_id)) ^ (0xC0FFEEull << 32) ^
                   (uint64_t)(uint32_t)layer_id;
  splitmix64_next(&state);  // the first output is discarded
  const uint64_t size = v.size(), take = std::min<uint64_t>((uint64_t)n, size);
  for (uint64_t i = 0; i < take; ++i) {
    const uint64_t j = i + splitmix64_next(&state) % (size - i);
    std::swap(v[i], v[j]);
    out[i] = v[i];
  }
  *n_out = (int32_t)take;
  return CT_OK;
}

int ct_top_t(const float* lat_us, const int32_t* status, int n, int t, int32_t* top, int32_t* n_top) {
  if (!lat_us || !status || !top || !n_top || n < 0 || t < 0) { set_error("ct_top_t: bad argument"); return CT_E_ARG; }
  std::vector<int32_t> ok;
  for (int i = 0; i < n; ++i)
    if (status[i] == CT_S_OK && std::isfinite(lat_us[i])) ok.push_back(i);
  std::sort(ok.begin(), ok.end(), [&](int32_t a, int32_t b) {
    return lat_us[a] < lat_us[b] || (lat_us[a] == lat_us[b] && a < b);
  });
  const int m = std::min<int>(t, (int)ok.size());
  for (int i = 0; i < m; ++i) top[i] = ok[i];
  *n_top = m;
  return CT_OK;
}

int ct_select_winner(const float* lat_us, const int32_t* pos, int n, float eps, int32_t* winner) {
  if (!lat_us || !pos || !winner || n < 0 || !(eps >= 0.0f)) { set_error("ct_select_winner: bad argument"); return CT_E_ARG; }
  double best = INFINITY;
  for (int i = 0; i < n; ++i)
    if (std::isfinite(lat_us[i]) && (double)lat_us[i] < best) best = lat_us[i];
  *winner = -1;
  if (!std::isfinite(best)) return CT_OK;
  const double limit = best * (1.0 + (double)eps);
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(lat_us[i]) || (double)lat_us[i] > limit) continue;
    if (*winner < 0 || pos[i] < pos[*winner]) *winner = i;
  }
  return CT_OK;
}

}  // extern "C"
