// Family 3, IGEMM_BF16: pointwise (1x1) convolution as a GEMM on the bf16
// matrix cores (v_mfma_f32_16x16x32_bf16 / v_mfma_f32_32x32x16_bf16), NHWC
// bf16 x, K x C bf16 w, NHWC fp32 y (fp32 accumulation).
//
// GEMM view: rows = output pixels (N*OH*OW), columns = output channels K,
// reduction = C. With NHWC x and K x C w both operands are row-major along
// the reduction, so every MFMA fragment is one 16-byte load of 8 bf16.
//
// A block owns a BM x BN tile (BM = WM*TM*MF pixels, BN = WN*TN*MF
// channels), one wave per WM x WN sub-tile. LDS = 0 loads each wave's
// fragments straight from global memory, a whole reduction chunk (KC) at a
// time, the next chunk's loads in flight during the current chunk's MFMAs
// (two register sets, for TM + TN <= 4); LDS = 1 stages the chunk's A and B tiles
// in LDS with coalesced 16-byte loads shared by the block. SPLIT > 1 spreads
// contiguous chunk ranges over grid.y (partials added in split order by a
// second kernel). SWZ = 1 renumbers blocks so that the tiles each XCD
// receives (blocks are dealt to the 8 XCDs in turn) are contiguous, which
// keeps a row band of x in one XCD's L2.
// All global loads are bounds-checked (C is a multiple of 8, so a 16-byte
// group is either wholly inside the tensor or wholly outside).
#include <hip/hip_runtime.h>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

struct IgBf16Args {
  int N, H, W, C, K, OH, OW, sh, sw;
  int npix;
  int wm, wn, kc;
  int bm, bn, threads;
  int cps, chunks;
  int a_loads, b_loads;
  int tiles_m, tiles_n, swz;
  int64_t ny;
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int MF>
struct MfmaBf16;
template <>
struct MfmaBf16<16> {
  static constexpr int ACC = 4, KSTEP = 32;
  typedef float V __attribute__((ext_vector_type(4)));
  __device__ static V op(bf16x8 a, bf16x8 b, V c) { return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0); }
  __device__ static int row(int e, int lane) { return 4 * (lane >> 4) + e; }
};
template <>
struct MfmaBf16<32> {
  static constexpr int ACC = 16, KSTEP = 16;
  typedef float V __attribute__((ext_vector_type(16)));
  __device__ static V op(bf16x8 a, bf16x8 b, V c) { return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0); }
  __device__ static int row(int e, int lane) { return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3); }
};

__host__ __device__ constexpr int bf16_max_threads(int acc_regs) { return acc_regs <= 64 ? 512 : 256; }
constexpr int kBf16MaxSteps = 4;  // k-steps of fragments held in registers (LDS = 0)

__device__ inline int pixel_offset(int m, const IgBf16Args& a) {
  if (a.sh == 1 && a.sw == 1) return m * a.C;  // OH = H, OW = W
  const int ohw = a.OH * a.OW;
  const int n = m / ohw;
  const int rem = m - n * ohw;
  const int oh = rem / a.OW, ow = rem - oh * a.OW;
  return ((n * a.H + oh * a.sh) * a.W + ow * a.sw) * a.C;
}

// 16-byte fragment load, branch-free: an invalid fragment reads the tensor's
// first 16 bytes and is replaced by zeros.
__device__ inline bf16x8 load8(const unsigned short* base, int64_t off, bool ok) {
  const u32x4 v = *(const u32x4*)(base + (ok ? off : 0));
  const u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, ok ? v : z);
}

template <int MF, int TM, int TN, bool LDS>
__global__ void __launch_bounds__(bf16_max_threads(TM * TN * MfmaBf16<MF>::ACC))
igemm_bf16_kernel(const unsigned short* __restrict__ x, const unsigned short* __restrict__ w,
                  float* __restrict__ out, IgBf16Args a) {
  using M = MfmaBf16<MF>;
  using V = typename M::V;
  constexpr int ACC = M::ACC, KSTEP = M::KSTEP;

  // block -> tile (optionally renumbered so each XCD gets a contiguous range)
  const int T = a.tiles_m * a.tiles_n;
  int b = blockIdx.x;
  if (a.swz) b = xcd_band_tile(b, T);
  const int tmi = b / a.tiles_n, tni = b - tmi * a.tiles_n;
  const int m0 = tmi * a.bm, n0 = tni * a.bn, sp = blockIdx.y;

  const int t = threadIdx.x, lane = t & 63, wave = wave_id();
  const int wmi = wave / a.wn, wni = wave - wmi * a.wn;
  const int m_off = wmi * TM * MF, n_off = wni * TN * MF;
  const int lrow = lane % MF, kq = (lane / MF) * 8;  // fragment row and k offset of this lane

  const int ch_begin = sp * a.cps;
  const int ch_end = min(a.chunks, ch_begin + a.cps);
  const int kr_end = min(a.C, ch_end * a.kc);

  V acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < ACC; ++e) acc[i][j][e] = 0.f;

  if constexpr (!LDS) {
    int aoff[TM], boff[TN];
    bool aok[TM], bok[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + m_off + i * MF + lrow;
      aok[i] = m < a.npix;
      aoff[i] = aok[i] ? pixel_offset(m, a) : 0;
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + n_off + j * MF + lrow;
      bok[j] = n < a.K;
      boff[j] = bok[j] ? n * a.C : 0;
    }
    const int steps = a.kc / KSTEP;
    // The fragments of chunk ch+1 are loaded into a second register set
    // while the MFMAs of chunk ch run (two sets, used alternately).
    using FragA = bf16x8[kBf16MaxSteps][TM];
    using FragB = bf16x8[kBf16MaxSteps][TN];
    auto load_chunk = [&](int ch, FragA& fa, FragB& fb) {
      const int kr0 = ch * a.kc;
#pragma unroll
      for (int st = 0; st < kBf16MaxSteps; ++st) {
        const int k = kr0 + st * KSTEP + kq;
        const bool kok = st < steps && k < kr_end;
#pragma unroll
        for (int i = 0; i < TM; ++i) fa[st][i] = load8(x, (int64_t)aoff[i] + k, kok && aok[i]);
#pragma unroll
        for (int j = 0; j < TN; ++j) fb[st][j] = load8(w, (int64_t)boff[j] + k, kok && bok[j]);
      }
    };
    auto mma_chunk = [&](const FragA& fa, const FragB& fb) {
#pragma unroll
      for (int st = 0; st < kBf16MaxSteps; ++st) {
        if (st < steps) {
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[st][i], fb[st][j], acc[i][j]);
        }
      }
    };
    if constexpr (TM + TN <= 4) {
      FragA fa0, fa1;
      FragB fb0, fb1;
      if (ch_begin < ch_end) load_chunk(ch_begin, fa0, fb0);
      for (int ch = ch_begin; ch < ch_end; ch += 2) {
        if (ch + 1 < ch_end) load_chunk(ch + 1, fa1, fb1);
        mma_chunk(fa0, fb0);
        if (ch + 1 >= ch_end) break;
        if (ch + 2 < ch_end) load_chunk(ch + 2, fa0, fb0);
        mma_chunk(fa1, fb1);
      }
    } else {
      // larger fragment sets: one set (two would spill registers)
      FragA fa0;
      FragB fb0;
      for (int ch = ch_begin; ch < ch_end; ++ch) {
        load_chunk(ch, fa0, fb0);
        mma_chunk(fa0, fb0);
      }
    }
  } else {
    extern __shared__ unsigned short lds16[];
    const int pitch = a.kc + 8;  // bf16 elements per LDS row (16-byte pad)
    unsigned short* As = lds16;
    unsigned short* Bs = lds16 + a.bm * pitch;
    const int vpr = a.kc / 8;  // 16-byte vectors per row
    const int vcol = t % vpr, row0 = t / vpr, rstep = a.threads / vpr;
    int aoff[kMaxLoadsPerThread];
    bool aok[kMaxLoadsPerThread];
#pragma unroll
    for (int i = 0; i < kMaxLoadsPerThread; ++i) {
      const int m = m0 + row0 + i * rstep;
      aok[i] = i < a.a_loads && row0 + i * rstep < a.bm && m < a.npix;
      aoff[i] = aok[i] ? pixel_offset(m, a) : 0;
    }
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      const int k = ch * a.kc + vcol * 8;
      const bool kok = k < kr_end;
      // loads are issued unconditionally (invalid ones read offset 0) and the
      // zero-select happens at the LDS store, so all loads are in flight at once
      u32x4 ra[kMaxLoadsPerThread], rb[kMaxLoadsPerThread];
      unsigned oka = 0, okb = 0;
#pragma unroll
      for (int i = 0; i < kMaxLoadsPerThread; ++i) {
        if (i < a.a_loads) {
          const bool ok = kok && aok[i];
          ra[i] = *(const u32x4*)(x + (ok ? (int64_t)aoff[i] + k : 0));
          oka |= (unsigned)ok << i;
        }
      }
#pragma unroll
      for (int i = 0; i < kMaxLoadsPerThread; ++i) {
        if (i < a.b_loads) {
          const int rr = row0 + i * rstep;
          const int n = n0 + rr;
          const bool ok = rr < a.bn && n < a.K && kok;
          rb[i] = *(const u32x4*)(w + (ok ? (int64_t)n * a.C + k : 0));
          okb |= (unsigned)ok << i;
        }
      }
      __syncthreads();
      const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < kMaxLoadsPerThread; ++i) {
        const int rr = row0 + i * rstep;
        if (i < a.a_loads && rr < a.bm) *(u32x4*)(As + rr * pitch + vcol * 8) = (oka >> i & 1u) ? ra[i] : z;
        if (i < a.b_loads && rr < a.bn) *(u32x4*)(Bs + rr * pitch + vcol * 8) = (okb >> i & 1u) ? rb[i] : z;
      }
      __syncthreads();
      const int steps = a.kc / KSTEP;
      for (int st = 0; st < steps; ++st) {
        const int kk = st * KSTEP + kq;
        bf16x8 fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = __builtin_bit_cast(bf16x8, *(const u32x4*)(As + (m_off + i * MF + lrow) * pitch + kk));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          fb[j] = __builtin_bit_cast(bf16x8, *(const u32x4*)(Bs + (n_off + j * MF + lrow) * pitch + kk));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[i], fb[j], acc[i][j]);
      }
    }
  }

  // Store. An accumulator's pixel row is a wave-uniform part (tile i,
  // element e) plus a lane part, so where every pixel row of the wave tile
  // exists each store is a buffer store whose scalar offset carries the
  // uniform row and whose one 32-bit lane offset (row group and channel) is
  // computed once per channel column; a ragged pixel tail checks every
  // element.
  const int mw = m0 + m_off;  // first pixel row of this wave's tile
  float* ob = out + (int64_t)sp * a.ny + (int64_t)mw * a.K;
  if (mw + TM * MF <= a.npix) {
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(ob, (int64_t)TM * MF * a.K * 4);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + n_off + j * MF + lrow;
      if (n >= a.K) continue;
      const int lo = (M::row(0, lane) * a.K + n) * 4;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < ACC; ++e) {
          // through a scalar: a bit cast of a vector element read element 0
          const float v = acc[i][j][e];
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro, lo, (i * MF + M::row(e, 0)) * a.K * 4, 0);
        }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + n_off + j * MF + lrow;
      if (n >= a.K) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < ACC; ++e) {
          const int mr = i * MF + M::row(e, lane);
          if (mw + mr < a.npix) ob[(int64_t)mr * a.K + n] = acc[i][j][e];
        }
    }
  }
}

using IgBf16Fn = void (*)(const unsigned short*, const unsigned short*, float*, IgBf16Args);

template <int MF, int TM, int TN>
static IgBf16Fn bf_pick_lds(int lds) {
  if constexpr (TM * TN * MfmaBf16<MF>::ACC > 128)
    return nullptr;  // accumulator tiles the validator rejects: not instantiated
  else
    return lds ? igemm_bf16_kernel<MF, TM, TN, true> : igemm_bf16_kernel<MF, TM, TN, false>;
}
template <int MF, int TM>
static IgBf16Fn bf_pick_tn(int tn, int lds) {
  switch (tn) {
    case 1: return bf_pick_lds<MF, TM, 1>(lds);
    case 2: return bf_pick_lds<MF, TM, 2>(lds);
    default: return bf_pick_lds<MF, TM, 4>(lds);
  }
}
template <int MF>
static IgBf16Fn bf_pick_tm(int tm, int tn, int lds) {
  switch (tm) {
    case 1: return bf_pick_tn<MF, 1>(tn, lds);
    case 2: return bf_pick_tn<MF, 2>(tn, lds);
    default: return bf_pick_tn<MF, 4>(tn, lds);
  }
}

int launch_igemm_bf16(const OpX& x, const ct_schedule& s, const Geom& g, const void* xin,
                      const void* w, void* y, float* ws, void* stream) {
  using namespace bf16_knob;
  const ct_op& o = x.op;
  IgBf16Args a;
  a.N = o.n; a.H = o.h; a.W = o.w; a.C = o.c; a.K = o.k; a.OH = (int)x.oh; a.OW = (int)x.ow;
  a.sh = o.stride_h; a.sw = o.stride_w;
  a.npix = (int)x.npix;
  a.wm = s.knob[WM]; a.wn = s.knob[WN]; a.kc = s.knob[KC];
  a.bm = g.bm; a.bn = g.bn; a.threads = g.threads;
  a.cps = g.chunks_per_split; a.chunks = g.chunks;
  a.a_loads = g.a_loads; a.b_loads = g.b_loads;
  a.tiles_m = (int)g.tiles_h; a.tiles_n = (int)g.tiles_k; a.swz = s.knob[SWZ];
  a.ny = x.ny;
  IgBf16Fn fn = s.knob[MF] == 32 ? bf_pick_tm<32>(s.knob[TM], s.knob[TN], s.knob[LDS])
                                 : bf_pick_tm<16>(s.knob[TM], s.knob[TN], s.knob[LDS]);
  if (!fn) {
    set_error("igemm_bf16: no kernel instance for this accumulator tile");
    return -2;
  }
  dim3 grid((unsigned)(g.tiles_h * g.tiles_k), (unsigned)g.split);
  float* out = g.split > 1 ? ws : (float*)y;
  hipLaunchKernelGGL(fn, grid, dim3(g.threads), g.lds_bytes, (hipStream_t)stream,
                     (const unsigned short*)xin, (const unsigned short*)w, out, a);
  if (hipGetLastError() != hipSuccess) return -1;
  if (g.split > 1) return launch_split_reduce(ws, (float*)y, x.ny, g.split, stream);
  return 0;
}

}  // namespace ct
