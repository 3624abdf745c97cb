// Family 4, IGEMM_F32: convolution as an implicit GEMM on the fp32 matrix
// cores (v_mfma_f32_32x32x2_f32 / v_mfma_f32_16x16x4_f32), NCHW x,
// K x C x R x S w, NCHW y.
//
// GEMM view: rows = output channels, columns = output pixels, reduction =
// (input channel, filter tap). A block owns a BM x BN tile: BM = WM*TM*MF
// output channels by BN = WN*TN*MF output pixels, the pixels forming a
// TPH x TPW rectangle of one image (TPW = the TPW knob, TPH = BN / TPW).
//
// Staging. The reduction advances one chunk of CPC input channels at a time
// (CPC divides C, or a single chunk holds all of C), padded to CPCP channels
// so that every reduction group gets whole MFMA k-steps. A chunk stages in LDS
//   * the input halo of the pixel rectangle, Xs[CPCP][HT][WT], each channel
//     padded to PP words: every filter tap reads its operand from this tile,
//     so a 3x3 filter costs one global read per input element instead of nine;
//   * the filter slice As[BM][CPCP*R*S] in global order, rows padded to a
//     pitch LDA.
// The pitches keep MFMA operand reads free of bank conflicts (32 banks, half
// a wave per pass): for 16x16x4 one pass reads 16 rows of A at two k offsets
// R*S apart (odd) and 16 pixels of B at two channels, so LDA = 2 (mod 32) and
// PP = 16 (mod 32), or PP = 8 (mod 32) where the 16 pixels span two halo rows
// 16 (mod 32) apart; for 32x32x2 one pass reads 32 rows of A at one k, so LDA
// is odd. The host sets both pitches.
// Both are copied by buffer loads that write LDS directly, without a round
// trip through registers: one wave instruction fills 64 consecutive LDS
// words, lane i the i-th. The halo is copied as a flat array; the lanes'
// offsets into x are fixed for the whole kernel (built once, with carry
// counters) and a padding element, a padded channel or a channel past the
// chunk gets an offset that the buffer's range check turns into 0. The
// filter is copied 64 words of a row at a time.
//
// MFMA k mapping. Lane group g (= lane / MF) takes channels i*KSTEP + g, so
// for a fixed tap a k-step advances the A address by KSTEP*R*S words and the
// B address by KSTEP channel planes. WS reduction groups split the k-steps of
// each tap; their partial tiles are added in group order through LDS.
// STAGES = 2 double-buffers the chunk: the copy of chunk c+1 is in flight
// while the MFMAs of chunk c run. STAGES = 3 double-buffers the same way
// with four more waves in the block (after the MFMA waves) that build the
// copy plan and issue every copy, so the MFMA waves only compute. SPLIT > 1
// spreads contiguous chunk ranges over grid.z; a second kernel adds the
// partials in split order.
#pragma once
#include <hip/hip_runtime.h>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

constexpr int kHaloSlots = 16;  // halo loads per wave per chunk (max)
constexpr int kFiltSlots = 16;  // filter loads per wave per chunk (max)
constexpr int kRegCopies = 4;   // register-staged 16-byte copies of each kind per wave (max)
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct IgF32Args {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw;
  int OH, OW, kred;
  int wm, wn, wsp, cpc, cpcp;
  int tpw, tph, tiles_w, tiles_h;
  int ht, wt, lda;
  int bm, bn, threads;
  int cps, chunks;
  int xs_pad;          // halo words per stage: whole wave copies
  int n_halo;          // halo copies per wave per chunk
  int n_filt_units;    // filter copies per chunk (all waves): rows x segments
  int f_nseg;          // segments per filter row
  int pp;              // LDS words per halo channel (the rows plus bank padding)
  int rw;              // LDS words per halo row
  int hshift;          // LDS column of input column iw0 (rows start that much earlier)
  int vec_h, vec_f;    // 1: the halo / filter is copied 16 bytes per lane
  // host-precomputed, in copy units (1 or 4 words): exact reciprocals of the
  // units per channel and per row, and the block size over (channel, unit)
  float inv_pu, inv_ru, inv_tpw;
  int h_dc, h_drem;
  float inv_tiles_hw, inv_tiles_w, inv_nseg;
  int f_dm, f_dseg;            // the wave count over (filter row, segment)
  int lg_wpg, lg_wn, lg_nw;    // log2 of WM*WN, WN and the count of copying waves
  int nmw;                     // MFMA waves (WM*WN*WS); STAGES 3 adds 4 loader waves after them
  float inv_gx, inv_gxy;       // 1 / grid x, 1 / (grid x * grid y)
  int64_t ny;
};

__host__ __device__ constexpr int ig_spec_r(int spec) { return spec == 1 || spec == 2 ? 1 : (spec == 3 || spec == 4 ? 3 : 0); }
__host__ __device__ constexpr int ig_spec_stride(int spec) { return spec == 1 || spec == 3 ? 1 : (spec == 2 || spec == 4 ? 2 : 0); }
// Threads per block that leave room for the accumulator tile in registers
// (with STAGES 3, 256 MFMA threads and the 256 of the loader waves: two
// waves per SIMD).
__host__ __device__ constexpr int mfma_max_threads(int acc_regs) { return acc_regs <= 64 ? 512 : 256; }

template <int MF>
struct MfmaF32;
template <>
struct MfmaF32<32> {
  static constexpr int ACC = 16, KSTEP = 2;
  typedef float V __attribute__((ext_vector_type(16)));
  __device__ static V op(float a, float b, V c) { return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0); }
  // row of accumulator element e held by `lane` (column = lane % 32); for both
  // shapes it splits as row(e, 0) + row(0, lane)
  __device__ static int row(int e, int lane) { return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3); }
};
template <>
struct MfmaF32<16> {
  static constexpr int ACC = 4, KSTEP = 4;
  typedef float V __attribute__((ext_vector_type(4)));
  __device__ static V op(float a, float b, V c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }
  __device__ static int row(int e, int lane) { return 4 * (lane >> 4) + e; }
};

// 16 bytes at byte offset off of r (0 past the buffer's range)
__device__ __forceinline__ f32x4 bload16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}


template <int MF, int TM, int TN, int STAGES, int SPEC>
__global__ void __launch_bounds__(STAGES == 3 ? 512 : mfma_max_threads(TM * TN * MfmaF32<MF>::ACC))
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
  const int cpcp = a.cpcp, bm = a.bm, ht = a.ht, lda = a.lda;
  const int pp = a.pp, rw = a.rw;
  const int jw = cpcp * RS;  // filter words per output channel in a chunk
  const int stage_floats = a.xs_pad + bm * lda;

  const int t = threadIdx.x, lane = t & 63, wave = wave_id();
  // The waves that copy: all of them, or with STAGES 3 the four loader waves
  // after the MFMA waves (nw of them; this wave is number cwv among them and
  // this thread number ct).
  constexpr bool LOADERS = STAGES == 3;
  const bool loader = LOADERS && wave >= a.nmw;
  const int nw = LOADERS ? 4 : a.threads >> 6;
  const int cwv = LOADERS ? wave - a.nmw : wave;
  const int ct = LOADERS ? t - 64 * a.nmw : t;
  // WM, WN, WS and the wave count are powers of two: shifts, not divisions
  const int wpg = a.wm * a.wn;
  const int wg = wave >> a.lg_wpg, wi = wave & (wpg - 1);
  const int wmi = wi >> a.lg_wn, wni = wi & ((1 << a.lg_wn) - 1);
  const int m_off = wmi * TM * MF, n_off = wni * TN * MF;

  // block -> (image, pixel rectangle), output-channel tile, split. The
  // blocks are renumbered so that each XCD takes one contiguous band of the
  // grid in (pixel tile, channel tile, split) order: the tiles of a band
  // share their filter slice and the halo rows between vertically adjacent
  // tiles in that XCD's L2, instead of every XCD fetching them again.
  int bx, by, bz;
  {
    const int gx = gridDim.x, gxy = gx * gridDim.y;
    const int tb = xcd_band_tile(blockIdx.x + gx * blockIdx.y + gxy * blockIdx.z, gxy * gridDim.z);
    bz = qdiv(tb, a.inv_gxy);
    const int r = tb - bz * gxy;
    by = qdiv(r, a.inv_gx);
    bx = r - by * gx;
  }
  const int tiles_hw = a.tiles_h * a.tiles_w;
  const int nimg = qdiv(bx, a.inv_tiles_hw);
  const int trem = bx - nimg * tiles_hw;
  const int th = qdiv(trem, a.inv_tiles_w), tw = trem - th * a.tiles_w;
  const int oh0 = th * a.tph, ow0 = tw * a.tpw;
  const int ih0 = oh0 * sh - ph, iw0 = ow0 * sw - pw;
  const int k0 = by * bm, sp = bz;
  const int cl = min(a.cpc, a.C);  // channels of x in a chunk

  // ---- halo plan. Xs[CPCP][PP]: row hh of channel c at c*PP + hh*RW, LDS
  // column j holding input column iw0 - HSHIFT + j. Copy unit: 1 word, or 4
  // (16-byte copies: a unit is then wholly inside or wholly outside the
  // image). Slot i of copying wave cwv copies units (i*nw + cwv)*64 + lane of the
  // flat array; a unit past the rows of its channel is bank padding. ----
  const int vh = a.vec_h ? 4 : 1;
  const int ru = rw / vh;
  int h_off[kHaloSlots];
  if (!LOADERS || loader) {
    const int pu = pp / vh, rows_u = ht * ru;
    int c = qdiv(ct, a.inv_pu), rem = ct - c * pu;
#pragma unroll
    for (int i = 0; i < kHaloSlots; ++i) {
      if (i < a.n_halo) {
        const int hh = qdiv(rem, a.inv_ru), col = (rem - hh * ru) * vh;
        const int gh = ih0 + hh, gw = iw0 - a.hshift + col;
        const bool ok = c < cl && rem < rows_u && (unsigned)gh < (unsigned)a.H && (unsigned)gw < (unsigned)a.W;
        h_off[i] = ok ? (c * HW + gh * a.W + gw) * 4 : kOob;
        // advance by T units: (c, rem) += (h_dc, h_drem) with a carry
        rem += a.h_drem;
        const int cr = rem >= pu;
        rem -= cr ? pu : 0;
        c += a.h_dc + cr;
      }
    }
  }
  // ---- filter plan: slot j of this wave copies one segment (64 units) of row
  // m, starting at word f_dst - m*lda; unit u = j*nw + cwv enumerates
  // (m, segment) row-major. A row shorter than a segment copies only the
  // lanes it needs (a 1-word copy lands in padding of rows of at least 64
  // words); a longer row's last segment is aligned to the row end,
  // overlapping the one before it with the same data. ----
  const int vf = a.vec_f ? 4 : 1, seg_len = 64 * vf;
  const int nseg = a.f_nseg;
  const int n_filt_w = a.n_filt_units > cwv ? (a.n_filt_units - cwv + nw - 1) >> a.lg_nw : 0;
  // 1-word copies land in rows of at least 64 words; 16-byte copies of a row
  // shorter than a segment use only the lanes the row needs
  const bool f_lane = vf == 1 || lane * 4 < jw;
  int f_off[kFiltSlots], f_dst[kFiltSlots];
  if (!LOADERS || loader) {
    const int dm = a.f_dm, dseg = a.f_dseg;  // nw = dm*nseg + dseg
    int m = qdiv(cwv, a.inv_nseg), seg = cwv - m * nseg;
#pragma unroll
    for (int j = 0; j < kFiltSlots; ++j) {
      if (j < n_filt_w) {
        const int s0 = jw >= seg_len ? min(seg * seg_len, jw - seg_len) : 0;
        const int jj = s0 + lane * vf;
        f_off[j] = jj < cl * RS ? (m * a.kred + jj) * 4 : kOob;
        f_dst[j] = m * lda + s0;
        seg += dseg;
        m += dm;
        if (seg >= nseg) { seg -= nseg; ++m; }
      }
    }
  }

  const int ch_begin = sp * a.cps;
  const int ch_end = min(a.chunks, ch_begin + a.cps);

  // start the copies of chunk ch into LDS stage `stage`
  // x: this image's channels [c0, c0 + cl); w: rows [k0, K) from column c0*RS
  auto rsrc_x = [&](int c0) { return make_rsrc(x + ((int64_t)nimg * a.C + c0) * HW, (int64_t)cl * HW * 4); };
  auto rsrc_w = [&](int c0) {
    return make_rsrc(w + (int64_t)k0 * a.kred + (int64_t)c0 * RS,
                     ((int64_t)(a.K - k0) * a.kred - (int64_t)c0 * RS) * 4);
  };
  auto issue = [&](int ch, int stage) {
    const int c0 = ch * a.cpc;
    float* xs = smem + stage * stage_floats;
    float* as = xs + a.xs_pad;
    const __amdgpu_buffer_rsrc_t rx = rsrc_x(c0), rw = rsrc_w(c0);
    if (a.vec_h) {
#pragma unroll
      for (int i = 0; i < kHaloSlots; ++i)
        if (i < a.n_halo) copy16_to_lds(rx, xs + (i * nw + cwv) * 256, h_off[i]);
    } else {
#pragma unroll
      for (int i = 0; i < kHaloSlots; ++i)
        if (i < a.n_halo) copy_to_lds(rx, xs + (i * nw + cwv) * 64, h_off[i]);
    }
    if (f_lane) {
      if (a.vec_f) {
#pragma unroll
        for (int j = 0; j < kFiltSlots; ++j)
          if (j < n_filt_w) copy16_to_lds(rw, as + f_dst[j], f_off[j]);
      } else {
#pragma unroll
        for (int j = 0; j < kFiltSlots; ++j)
          if (j < n_filt_w) copy_to_lds(rw, as + f_dst[j], f_off[j]);
      }
    }
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
  for (int i = 0; i < TM; ++i) a_base[i] = (m_off + i * MF + lrow) * lda + kg * RS;
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int q = n_off + j * MF + lrow;
    const int pr = qdiv(q, a.inv_tpw), pc = q - pr * a.tpw;
    b_base[j] = kg * pp + (pr * sh) * rw + pc * sw + a.hshift;
  }
  const int n_i = cpcp / KSTEP / a.wsp;  // k-steps per tap for this reduction group
  const int i_begin = wg * n_i;
  const int astep = KSTEP * RS, bstep = KSTEP * pp;
  // One k-step (KSTEP channels) at a time, all filter taps unrolled inside it
  // when R and S are compile-time: tap offsets become immediate LDS offsets
  // and each step exposes R*S*TM*TN independent-enough MFMAs to the
  // scheduler. The pixel rows of the taps are per-lane bases set up once.
  int b_row[TN][RC ? RC : 1];
  if constexpr (RC != 0) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < RC; ++r) b_row[j][r] = b_base[j] + r * rw;
  }
  auto compute = [&](int stage) {
    const float* Xs = smem + stage * stage_floats;
    const float* As = Xs + a.xs_pad;
    if constexpr (RC != 0) {
      constexpr int kUnrollSteps = RC == 1 ? 4 : 1;  // a 1x1 filter has one tap per step
#pragma unroll kUnrollSteps
      for (int ii = 0; ii < n_i; ++ii) {
        const float* ap = As + (i_begin + ii) * astep;
        const float* bp = Xs + (i_begin + ii) * bstep;
#pragma unroll
        for (int r = 0; r < RC; ++r) {
#pragma unroll
          for (int s = 0; s < RC; ++s) {
            float fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[i] = ap[a_base[i] + r * RC + s];
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[j] = bp[b_row[j][r] + s];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[i], fb[j], acc[i][j]);
          }
        }
      }
    } else {
      for (int r = 0; r < R; ++r) {
        for (int s = 0; s < S; ++s) {
          const float* ap = As + (r * S + s) + i_begin * astep;
          const float* bp = Xs + (r * dh) * rw + s * dw + i_begin * bstep;
          for (int ii = 0; ii < n_i; ++ii) {
            float fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[i] = ap[a_base[i] + ii * astep];
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[j] = bp[b_base[j] + ii * bstep];
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
              for (int j = 0; j < TN; ++j) acc[i][j] = M::op(fa[i], fb[j], acc[i][j]);
          }
        }
      }
    }
  };

  // STAGES = 2 with 16-byte copies and at most kRegCopies of each kind per
  // wave: the next chunk goes through registers instead (16-byte loads that
  // stay in flight during the MFMAs, stored to LDS after them). A copy
  // straight to LDS holds its wave about one L2 round trip on this device,
  // so several of them in a row stall the wave that should be issuing MFMAs.
  // (Measured: staging the single-stage chunks, or the first chunk, the same
  // way is a few percent slower than copying them straight to LDS.)
  const bool via_regs = STAGES == 2 && a.vec_h && a.vec_f && a.n_halo <= kRegCopies &&
                        ((a.n_filt_units + nw - 1) >> a.lg_nw) <= kRegCopies;
  f32x4 rh[kRegCopies], rf[kRegCopies];
  auto load_regs = [&](int ch) {
    const int c0 = ch * a.cpc;
    const __amdgpu_buffer_rsrc_t rx = rsrc_x(c0), rw = rsrc_w(c0);
#pragma unroll
    for (int i = 0; i < kRegCopies; ++i)
      if (i < a.n_halo) rh[i] = bload16(rx, h_off[i]);
#pragma unroll
    for (int j = 0; j < kRegCopies; ++j)
      if (j < n_filt_w && f_lane) rf[j] = bload16(rw, f_off[j]);
  };
  auto store_regs = [&](int stage) {
    float* xs = smem + stage * stage_floats;
    float* as = xs + a.xs_pad;
#pragma unroll
    for (int i = 0; i < kRegCopies; ++i)
      if (i < a.n_halo) *(f32x4*)(xs + (i * nw + cwv) * 256 + lane * 4) = rh[i];
#pragma unroll
    for (int j = 0; j < kRegCopies; ++j)
      if (j < n_filt_w && f_lane) *(f32x4*)(as + f_dst[j] + lane * 4) = rf[j];
  };

  if constexpr (STAGES == 1) {
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      issue(ch, 0);
      wait_copies();
      __syncthreads();
      compute(0);
      __syncthreads();  // the next chunk's copies overwrite this stage
    }
  } else if constexpr (LOADERS) {
    // the loader waves copy, the MFMA waves compute; every wave passes every
    // barrier
    if (loader && ch_begin < ch_end) issue(ch_begin, 0);
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      const int cur = (ch - ch_begin) & 1;
      if (loader) wait_copies();
      __syncthreads();  // chunk ch has landed; the MFMA waves are done with chunk ch-1
      if (loader) {
        if (ch + 1 < ch_end) issue(ch + 1, cur ^ 1);
      } else {
        compute(cur);
      }
    }
  } else if (via_regs) {
    if (ch_begin < ch_end) {
      issue(ch_begin, 0);
      wait_copies();
    }
    __syncthreads();
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      const int cur = (ch - ch_begin) & 1;
      const bool more = ch + 1 < ch_end;
      if (more) load_regs(ch + 1);
      compute(cur);
      if (more) store_regs(cur ^ 1);  // the stage chunk ch-1 used, free since the last barrier
      __syncthreads();
    }
  } else {
    if (ch_begin < ch_end) issue(ch_begin, 0);
    for (int ch = ch_begin; ch < ch_end; ++ch) {
      const int cur = (ch - ch_begin) & 1;
      wait_copies();
      __syncthreads();  // chunk ch has landed; every wave is done with chunk ch-1
      if (ch + 1 < ch_end) issue(ch + 1, cur ^ 1);
      compute(cur);
    }
  }

  if (a.wsp > 1) {
    // add the reduction groups' partial tiles in group order; a lane's
    // accumulators of one MFMA tile sit side by side in LDS, so they move
    // 16 bytes per access (the 64 lanes of a wave cover 64 consecutive
    // 16-byte slots: no bank conflicts)
    __syncthreads();
    typedef float f4 __attribute__((ext_vector_type(4)));
    f4* red = (f4*)smem;
    constexpr int Q = ACC / 4;  // 16-byte quads per accumulator tile
    if (wg > 0 && !loader) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int qd = 0; qd < Q; ++qd) {
            f4 v;
            v.x = acc[i][j][4 * qd];
            v.y = acc[i][j][4 * qd + 1];
            v.z = acc[i][j][4 * qd + 2];
            v.w = acc[i][j][4 * qd + 3];
            red[((((wg - 1) * wpg + wi) * TM * TN + i * TN + j) * Q + qd) * 64 + lane] = v;
          }
    }
    __syncthreads();
    if (wg > 0) return;  // the other reduction groups and the loader waves are done
    for (int g = 1; g < a.wsp; ++g) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int qd = 0; qd < Q; ++qd) {
            const f4 v = red[((((g - 1) * wpg + wi) * TM * TN + i * TN + j) * Q + qd) * 64 + lane];
            acc[i][j][4 * qd] += v.x;
            acc[i][j][4 * qd + 1] += v.y;
            acc[i][j][4 * qd + 2] += v.z;
            acc[i][j][4 * qd + 3] += v.w;
          }
    }
  }

  if (loader) return;

  // Store. An accumulator's output channel splits into a wave-uniform part
  // (tile i, element e) and a lane part, so where the wave's whole channel
  // tile exists each store is a buffer store whose scalar offset carries the
  // uniform channel row and whose one 32-bit lane offset (channel-group row
  // and pixel) is computed once per pixel column: no per-store address
  // arithmetic on the vector ALU. A ragged channel tail checks every element.
  const int ohw = a.OH * a.OW;
  const int kw = k0 + m_off;  // first output channel of this wave's tile
  float* ob = out + (int64_t)sp * a.ny + (int64_t)(nimg * a.K + kw) * ohw;
  if (kw + TM * MF <= a.K) {
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(ob, (int64_t)TM * MF * ohw * 4);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int q = n_off + j * MF + lrow;
      const int pr = qdiv(q, a.inv_tpw), pc = q - pr * a.tpw;
      const int oh = oh0 + pr, ow = ow0 + pc;
      if (oh >= a.OH || ow >= a.OW) continue;
      const int lo = (M::row(0, lane) * ohw + oh * a.OW + ow) * 4;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < ACC; ++e) {
          // the element goes through a scalar first: a bit cast applied to a
          // vector element directly has compiled to a read of element 0
          const float v = acc[i][j][e];
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro, lo, (i * MF + M::row(e, 0)) * ohw * 4, 0);
        }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int q = n_off + j * MF + lrow;
      const int pr = qdiv(q, a.inv_tpw), pc = q - pr * a.tpw;
      const int oh = oh0 + pr, ow = ow0 + pc;
      if (oh >= a.OH || ow >= a.OW) continue;
      const int lo = oh * a.OW + ow;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int e = 0; e < ACC; ++e) {
          const int kr = i * MF + M::row(e, lane);
          if (kw + kr < a.K) ob[(int64_t)kr * ohw + lo] = acc[i][j][e];
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
  constexpr int acc = TM * TN * MfmaF32<MF>::ACC;
  if constexpr (acc > 128) {
    return nullptr;  // accumulator tiles the validator rejects: not instantiated
  } else {
    if (stages == 3) {
      if constexpr (acc > kLoaderMaxAcc)
        return nullptr;  // rejected beside loader waves: not instantiated
      else
        return igf32_pick_spec<MF, TM, TN, 3>(spec);
    }
    return stages == 2 ? igf32_pick_spec<MF, TM, TN, 2>(spec) : igf32_pick_spec<MF, TM, TN, 1>(spec);
  }
}
template <int MF, int TM>
IgF32Fn igf32_pick_tn(int tn, int stages, int spec) {
  switch (tn) {
    case 1: return igf32_pick_stages<MF, TM, 1>(stages, spec);
    case 2: return igf32_pick_stages<MF, TM, 2>(stages, spec);
    case 4: return igf32_pick_stages<MF, TM, 4>(stages, spec);
    default: return igf32_pick_stages<MF, TM, 7>(stages, spec);
  }
}

}  // namespace ct
