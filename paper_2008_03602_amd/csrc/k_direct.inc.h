#pragma once
// Kernel template of family 1, DIRECT_F32, included by the per-MK units.
// Family 1, DIRECT_F32: direct convolution on the vector ALU, NCHW x,
// K x C x R x S w, NCHW y, fp32 throughout.
//
// A block computes a TK x TOH x TOW output tile of one image. Each thread
// owns MK consecutive output channels and MW output columns of one row; the
// MW columns are TOW/MW apart, so a wave's lanes touch consecutive columns
// (coalesced global stores, conflict-free LDS reads). The reduction runs over
// input-channel chunks of CT; with LDS staging the input halo tile and the
// filter chunk are copied to LDS once per chunk and shared by the block.
// SPLIT > 1 gives each split a contiguous channel range and writes partial
// sums to a workspace that a second kernel adds in split order.
//
// Compile-time: MK, MW, LDS, UNR and the filter/stride specialisation
// (generic, 1x1 s1/s2, 3x3 pad 1 s1/s2). Runtime: tiles, CT, SPLIT.
// Global reads are raw buffer loads with 32-bit offsets: an element outside
// the tensor (padding, a tile past the edge) gets an offset past the buffer,
// which the hardware reads as 0. A load then needs one offset register and no
// branch, so a thread keeps many in flight: with few threads per CU (small
// grids) this, not the arithmetic, sets the time. An LDS chunk too deep for
// the register prefetch is copied straight into LDS by buffer loads, every
// element of the chunk in flight at once.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "ct_internal.h"
#include "k_util.h"

namespace ct {

struct DirectArgs {
  int N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw;
  int OH, OW;
  int toh, tow, tk, ct;
  int tiles_w;
  int split, cps;
  int ih_t, iw_t;
  int threads, tp, cols;
  // host-precomputed reciprocals of the staging divisors (see qdiv)
  float inv_plane, inv_iwt, inv_crs, inv_rs;
  int64_t ny;
};

// Threads per block that leave registers for an MK x MW accumulator tile
// and its operands without spilling.
__host__ __device__ constexpr int direct_max_threads(int tile) { return tile >= 16 ? 512 : 1024; }

__host__ __device__ constexpr int spec_r(int spec) { return spec == 1 || spec == 2 ? 1 : (spec == 3 || spec == 4 ? 3 : 0); }
__host__ __device__ constexpr int spec_stride(int spec) { return spec == 1 || spec == 3 ? 1 : (spec == 2 || spec == 4 ? 2 : 0); }

template <int MK, int MW, bool LDS, int SPEC, int UNR>
__global__ void __launch_bounds__(direct_max_threads(MK * MW))
direct_f32_kernel(const float* __restrict__ x, const float* __restrict__ w, float* __restrict__ out,
                  DirectArgs a) {
  constexpr int RC = spec_r(SPEC), STC = spec_stride(SPEC);
  const int R = RC ? RC : a.R, S = RC ? RC : a.S;
  const int sh = STC ? STC : a.sh, sw = STC ? STC : a.sw;
  const int dh = SPEC ? 1 : a.dh, dw = SPEC ? 1 : a.dw;
  const int ph = SPEC ? RC / 2 : a.ph, pw = SPEC ? RC / 2 : a.pw;
  const int RS = R * S;
  const int C = a.C, H = a.H, W = a.W, K = a.K;

  extern __shared__ float smem[];
  const int t = threadIdx.x;
  const int th = blockIdx.x / a.tiles_w, tw = blockIdx.x - th * a.tiles_w;
  const int k0 = blockIdx.y * a.tk;
  const int n = blockIdx.z / a.split, sp = blockIdx.z - n * a.split;
  const int oh0 = th * a.toh, ow0 = tw * a.tow;
  const int tki = t / a.tp, tpi = t - tki * a.tp;
  const int lr = tpi / a.cols, lc = tpi - lr * a.cols;
  const int oh = oh0 + lr;
  const int kbase = k0 + tki * MK;

  float acc[MK][MW];
#pragma unroll
  for (int i = 0; i < MK; ++i)
#pragma unroll
    for (int j = 0; j < MW; ++j) acc[i][j] = 0.f;

  const int c_begin = sp * a.cps * a.ct;
  const int c_end = min(C, c_begin + a.cps * a.ct);
  const int ih_org = oh0 * sh - ph, iw_org = ow0 * sw - pw;
  const float* xn = x + (int64_t)n * C * H * W;
  const int HW = H * W;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(xn, (int64_t)C * HW * 4);
  const __amdgpu_buffer_rsrc_t rwt = make_rsrc(w, (int64_t)K * C * RS * 4);

  // LDS path: the block's MACs over nc staged channels
  auto compute_lds = [&](const int nc) __attribute__((always_inline)) {
    const float* xs = smem;
    const float* wsm = smem + a.ct * a.ih_t * a.iw_t;
    const int plane = a.ih_t * a.iw_t;
#pragma unroll UNR
    for (int c = 0; c < nc; ++c) {
      const float* xr = xs + c * plane + (lr * sh) * a.iw_t + lc * sw;
      const float* wr = wsm + (tki * MK * a.ct + c) * RS;
#pragma unroll
      for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          float xv[MW], wv[MK];
#pragma unroll
          for (int j = 0; j < MW; ++j) xv[j] = xr[(r * dh) * a.iw_t + j * a.cols * sw + s * dw];
#pragma unroll
          for (int i = 0; i < MK; ++i) wv[i] = wr[i * a.ct * RS + r * S + s];
#pragma unroll
          for (int i = 0; i < MK; ++i)
#pragma unroll
            for (int j = 0; j < MW; ++j) acc[i][j] = fmaf(wv[i], xv[j], acc[i][j]);
        }
      }
    }
  };
  // byte offsets of staging element e of the chunk starting at channel cc
  // (nc channels): halo element, then filter element; kOob outside
  const int plane = a.ih_t * a.iw_t;
  const int xt = a.ct * plane;
  const int crs = a.ct * RS;
  const int wt = a.tk * crs;
  auto x_off = [&](const int e, const int cc, const int nc) {
    const int c = qdiv(e, a.inv_plane);
    const int rem = e - c * plane;
    const int hh = qdiv(rem, a.inv_iwt), ww = rem - hh * a.iw_t;
    const int gh = ih_org + hh, gw = iw_org + ww;
    const bool ok = e < xt && c < nc && (unsigned)gh < (unsigned)H && (unsigned)gw < (unsigned)W;
    return ok ? ((cc + c) * HW + gh * W + gw) * 4 : kOob;
  };
  auto w_off = [&](const int e, const int cc, const int nc) {
    const int kk = qdiv(e, a.inv_crs);
    const int rem = e - kk * crs;
    const int c = qdiv(rem, a.inv_rs), rs = rem - c * RS;
    const bool ok = e < wt && k0 + kk < K && c < nc;
    return ok ? (((k0 + kk) * C + cc + c) * RS + rs) * 4 : kOob;
  };
  // Chunks of at most NS staging elements per thread (halo and filter
  // each) go through registers: the next chunk's loads are in flight during
  // this chunk's MACs, so a block pays one memory round trip per chunk only
  // once. An element's offset depends on the chunk only through its first
  // channel cc, which moves the buffer's base instead: the offsets are
  // computed once, and a chunk's loads take no address arithmetic.
  // Channels of a last, partial chunk past nc stage values that the MACs
  // never read.
  const int nsx = (xt + a.threads - 1) / a.threads, nsw = (wt + a.threads - 1) / a.threads;
  auto prefetched = [&](auto ns) __attribute__((always_inline)) {
    constexpr int NS = decltype(ns)::value;
    int xo[NS], wo[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      xo[u] = kOob;
      wo[u] = kOob;
      const int e = t + u * a.threads;
      if (u < nsx) {
        const int c = qdiv(e, a.inv_plane);
        const int rem = e - c * plane;
        const int hh = qdiv(rem, a.inv_iwt), ww = rem - hh * a.iw_t;
        const int gh = ih_org + hh, gw = iw_org + ww;
        if (e < xt && (unsigned)gh < (unsigned)H && (unsigned)gw < (unsigned)W) xo[u] = (c * HW + gh * W + gw) * 4;
      }
      if (u < nsw) {
        const int kk = qdiv(e, a.inv_crs);
        const int rem = e - kk * crs;
        const int c = qdiv(rem, a.inv_rs), rs = rem - c * RS;
        if (e < wt && k0 + kk < K) wo[u] = ((k0 + kk) * C * RS + c * RS + rs) * 4;
      }
    }
    float px[NS], pw[NS];
    auto fetch = [&](const int cc) {
      const __amdgpu_buffer_rsrc_t rxc = make_rsrc(xn + (int64_t)cc * HW, (int64_t)(C - cc) * HW * 4);
      const __amdgpu_buffer_rsrc_t rwc = make_rsrc(w + (int64_t)cc * RS, ((int64_t)K * C - cc) * RS * 4);
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        if (u < nsx) px[u] = bload1(rxc, xo[u]);
        if (u < nsw) pw[u] = bload1(rwc, wo[u]);
      }
    };
    float* xs = smem;
    float* wsm = smem + xt;
    if (c_begin < c_end) fetch(c_begin);
    for (int cc = c_begin; cc < c_end; cc += a.ct) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        const int e = t + u * a.threads;
        if (u < nsx && e < xt) xs[e] = px[u];
        if (u < nsw && e < wt) wsm[e] = pw[u];
      }
      __syncthreads();
      if (cc + a.ct < c_end) fetch(cc + a.ct);
      compute_lds(min(a.ct, c_end - cc));
      __syncthreads();  // the next chunk's stores overwrite the tiles
    }
  };
  bool done = false;
  if constexpr (LDS) {
    // the deepest prefetch that leaves the MACs their registers: 16 elements
    // per thread where the launch bound gives 256 VGPRs (8 beside 32
    // accumulators), else 8, or beside two unrolled channels 4 (4
    // accumulators) or none (8)
    constexpr int kMaxNs = direct_max_threads(MK * MW) <= 512 ? (MK * MW >= 32 ? 8 : 16)
                           : UNR == 2 && MK * MW >= 8 ? 0
                           : UNR == 2 && MK * MW >= 4 ? 4 : 8;
    const int n_stage = max(nsx, nsw);
    done = kMaxNs > 0 && n_stage <= kMaxNs;
    if constexpr (kMaxNs > 0) {
      if (n_stage <= 2) {
        prefetched(std::integral_constant<int, 2>{});
      } else if (n_stage <= 4) {
        prefetched(std::integral_constant<int, 4>{});
      } else if constexpr (kMaxNs >= 8) {
        if (n_stage <= 8) {
          prefetched(std::integral_constant<int, 8>{});
        } else if constexpr (kMaxNs >= 16) {
          if (n_stage <= 16) prefetched(std::integral_constant<int, 16>{});
        }
      }
    }
  }

  for (int cc = c_begin; cc < c_end && !done; cc += a.ct) {
    const int nc = min(a.ct, c_end - cc);
    if constexpr (LDS) {
      float* xs = smem;
      float* wsm = smem + xt;
      // Stage the halo tile and the filter chunk straight into LDS: one
      // buffer load per element, thread t of copy j filling element
      // j * threads + t (so a block of fewer than 64 threads works too), every
      // copy of the chunk in flight at once, then one wait. A copy writes lane
      // i of its wave at its LDS base + i, so each wave's base is offset by 64
      // elements per wave before it. An element outside the tensor reads 0
      // through the buffer's range check; lanes past the tile copy nothing.
      const int wbase = wave_id() * 64;
      auto stage = [&](const int total, const __amdgpu_buffer_rsrc_t r, auto byte_off, float* dst) {
        for (int e0 = 0; e0 < total; e0 += a.threads) {
          const int e = e0 + t;
          if (e < total) copy_to_lds(r, dst + e0 + wbase, byte_off(e));
        }
      };
      stage(xt, rx, [&](const int e) { return x_off(e, cc, nc); }, xs);
      stage(wt, rwt, [&](const int e) { return w_off(e, cc, nc); }, wsm);
      wait_copies();
      __syncthreads();
      compute_lds(nc);
      __syncthreads();
    } else {
      // kb: first output channel of this thread. When every wave lies inside
      // one channel group (TP a multiple of 64), kb is the same on all lanes
      // and the filter reads are scalar loads, off the vector memory path.
      auto direct = [&](const int kb) __attribute__((always_inline)) {
        // filter rows of this thread's channels; a channel past K reads row
        // K-1 (its sums are never stored)
        const float* wrow[MK];
#pragma unroll
        for (int i = 0; i < MK; ++i) wrow[i] = w + min(kb + i, K - 1) * C * RS;
        if constexpr (RC != 0) {
          // fixed filter: this thread's input offset at every tap and column
          // is the same in every channel plane (kOob in the padding), so it
          // is computed once and a channel moves the buffer's base
          int xo[RC][RC][MW];
#pragma unroll
          for (int r = 0; r < RC; ++r) {
            const int gh = oh * sh - ph + r;
            const bool hok = (unsigned)gh < (unsigned)H && oh < a.OH;
#pragma unroll
            for (int s = 0; s < RC; ++s)
#pragma unroll
              for (int j = 0; j < MW; ++j) {
                const int gw = (ow0 + lc + j * a.cols) * sw - pw + s;
                xo[r][s][j] = hok && (unsigned)gw < (unsigned)W ? (gh * W + gw) * 4 : kOob;
              }
          }
          // STEP channels per step: every input and filter value of the step
          // is loaded first and the scheduling barrier keeps the MACs after
          // them, so a step costs one memory round trip (left to itself the
          // scheduler sinks each load next to its first use and waits for
          // them one at a time). The channels of a step past the chunk's
          // last one load nothing and add nothing. Each output still adds its
          // terms channel by channel, taps in order.
          // Two channels per step (UNR 2) only where their staged values, the
          // input offsets and the accumulators fit the launch bound's
          // registers (128 for 1024 threads, 256 for 512) with room to spare.
          constexpr int T = RC * RC;
          constexpr int kRegs = direct_max_threads(MK * MW) >= 1024 ? 128 : 256;
          constexpr int STEP = UNR == 2 && 2 * T * (MW + MK) + T * MW + MK * MW + 24 <= kRegs ? 2 : 1;
          for (int c = 0; c < nc; c += STEP) {
            float xv[STEP][T][MW], wv[STEP][MK][T];
#pragma unroll
            for (int u = 0; u < STEP; ++u) {
              if (u == 0 || c + u < nc) {
                const __amdgpu_buffer_rsrc_t rxc = make_rsrc(xn + (int64_t)(cc + c + u) * HW, (int64_t)HW * 4);
                const int co = (cc + c + u) * RS;
#pragma unroll
                for (int q = 0; q < T; ++q)
#pragma unroll
                  for (int j = 0; j < MW; ++j) xv[u][q][j] = bload1(rxc, xo[q / RC][q % RC][j]);
#pragma unroll
                for (int i = 0; i < MK; ++i)
#pragma unroll
                  for (int q = 0; q < T; ++q) wv[u][i][q] = wrow[i][co + q];
              }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int u = 0; u < STEP; ++u) {
              if (u > 0 && c + u >= nc) break;
#pragma unroll
              for (int q = 0; q < T; ++q)
#pragma unroll
                for (int i = 0; i < MK; ++i)
#pragma unroll
                  for (int j = 0; j < MW; ++j) acc[i][j] = fmaf(wv[u][i][q], xv[u][q][j], acc[i][j]);
            }
          }
          return;
        }
#pragma unroll UNR
        for (int c = 0; c < nc; ++c) {
          const int xo = (cc + c) * HW;
          const int co = (cc + c) * RS;
          for (int r = 0; r < R; ++r) {
            const int gh = oh * sh - ph + r * dh;
            const bool hok = (unsigned)gh < (unsigned)H && oh < a.OH;
            // the taps of a filter row go in groups of G, all of a group's
            // loads before its MACs (one memory round trip per group, not per
            // tap); taps past the row's end load and add nothing. G = 2 where
            // the launch bound leaves 128 registers and a tap loads 6 or more
            // values.
            constexpr int G = direct_max_threads(MK * MW) >= 1024 && MK + MW >= 6 ? 2 : 4;
            for (int s0 = 0; s0 < S; s0 += G) {
              float xv[G][MW], wv[G][MK];
#pragma unroll
              for (int u = 0; u < G; ++u) {
                if (u == 0 || s0 + u < S) {
                  const int s = s0 + u;
#pragma unroll
                  for (int j = 0; j < MW; ++j) {
                    const int ow = ow0 + lc + j * a.cols;
                    const int gw = ow * sw - pw + s * dw;
                    xv[u][j] = bload1(rx, hok && (unsigned)gw < (unsigned)W ? (xo + gh * W + gw) * 4 : kOob);
                  }
#pragma unroll
                  for (int i = 0; i < MK; ++i) wv[u][i] = wrow[i][co + r * S + s];
                }
              }
              __builtin_amdgcn_sched_barrier(0);
#pragma unroll
              for (int u = 0; u < G; ++u) {
                if (u > 0 && s0 + u >= S) break;
#pragma unroll
                for (int i = 0; i < MK; ++i)
#pragma unroll
                  for (int j = 0; j < MW; ++j) acc[i][j] = fmaf(wv[u][i], xv[u][j], acc[i][j]);
              }
            }
          }
        }
      };
      if ((a.tp & 63) == 0)
        direct(__builtin_amdgcn_readfirstlane(kbase));
      else
        direct(kbase);
    }
  }

  if (oh >= a.OH) return;
  float* o = out + (int64_t)sp * a.ny;
#pragma unroll
  for (int i = 0; i < MK; ++i) {
    const int k = kbase + i;
    if (k >= K) break;
#pragma unroll
    for (int j = 0; j < MW; ++j) {
      const int ow = ow0 + lc + j * a.cols;
      if (ow < a.OW) o[(((int64_t)n * K + k) * a.OH + oh) * a.OW + ow] = acc[i][j];
    }
  }
}

using DirectFn = void (*)(const float*, const float*, float*, DirectArgs);


template <int MK, int MW, bool LDS, int SPEC>
static DirectFn pick_unr(int unr) {
  return unr == 2 ? (DirectFn)direct_f32_kernel<MK, MW, LDS, SPEC, 2>
                  : (DirectFn)direct_f32_kernel<MK, MW, LDS, SPEC, 1>;
}
template <int MK, int MW, bool LDS>
static DirectFn pick_spec(int spec, int unr) {
  switch (spec) {
    case SPEC_1X1_S1: return pick_unr<MK, MW, LDS, 1>(unr);
    case SPEC_1X1_S2: return pick_unr<MK, MW, LDS, 2>(unr);
    case SPEC_3X3_S1: return pick_unr<MK, MW, LDS, 3>(unr);
    case SPEC_3X3_S2: return pick_unr<MK, MW, LDS, 4>(unr);
    default: return pick_unr<MK, MW, LDS, 0>(unr);
  }
}
template <int MK, int MW>
static DirectFn pick_lds(int lds, int spec, int unr) {
  return lds ? pick_spec<MK, MW, true>(spec, unr) : pick_spec<MK, MW, false>(spec, unr);
}
template <int MK>
DirectFn pick_mw(int mw, int lds, int spec, int unr) {
  switch (mw) {
    case 1: return pick_lds<MK, 1>(lds, spec, unr);
    case 2: return pick_lds<MK, 2>(lds, spec, unr);
    default: return pick_lds<MK, 4>(lds, spec, unr);
  }
}
}  // namespace ct
