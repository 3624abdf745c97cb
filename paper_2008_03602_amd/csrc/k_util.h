// Device helpers shared by the kernel families.
#pragma once
#include <hip/hip_runtime.h>

namespace ct {

// Bounds-checked load without a branch: the address is clamped to element 0
// when `ok` is false and the value is replaced by zero. Keeping loads out of
// divergent branches lets the compiler issue a whole batch of them before the
// first wait, instead of waiting for each one in turn.
template <typename T>
__device__ __forceinline__ T load_or_zero(const T* __restrict__ p, int64_t idx, bool ok) {
  const T v = p[ok ? idx : 0];
  return ok ? v : T{};
}

// Raw buffer resource over `bytes` bytes at base: loads at byte offsets at or
// past `bytes` return 0 (the hardware range check), so an out-of-range
// element needs no branch and no clamped address.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
constexpr int kOob = 0x7FFFFFF0;  // byte offset beyond every buffer: reads as 0

// One word at byte offset off of r (0 past the buffer's range).
__device__ __forceinline__ float bload1(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

typedef __attribute__((address_space(3))) void lds_void_t;
// One wave instruction: lane i copies the word at byte offset off of r to
// lds[i] (an inactive lane copies nothing), without a trip through registers.
__device__ __forceinline__ void copy_to_lds(__amdgpu_buffer_rsrc_t r, float* lds, int off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds, 4, off, 0, 0, 0);
}
// The same with 16 bytes per lane: lane i fills lds[4i .. 4i+3] (lds and the
// lane's source 16-byte aligned).
__device__ __forceinline__ void copy16_to_lds(__amdgpu_buffer_rsrc_t r, float* lds, int off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds, 16, off, 0, 0, 0);
}
// Waits for this wave's copies to land in LDS.
__device__ __forceinline__ void wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// floor(n / d) for 0 <= n < 2^22 given inv = 1/d in fp32: (n + 1/2)/d lies at
// least 1/(2d) from an integer and the fp32 product errs by less than that.
__device__ __forceinline__ int qdiv(int n, float inv) { return (int)(((float)n + 0.5f) * inv); }

// Block renumbering for XCD locality: the device deals consecutive blocks to
// its 8 XCDs in turn, so block b runs on XCD b mod 8. Tile of block b when
// each XCD takes one contiguous band of the T tiles (the first T mod 8 XCDs
// take one tile more), so neighbouring tiles share that XCD's L2.
__host__ __device__ inline int xcd_band_tile(int b, int T) {
  const int q = T / 8, r = T % 8, xcd = b % 8, idx = b / 8;
  return xcd < r ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// The wave index as a scalar value, so loops bounded by per-wave values stay
// uniform (scalar branches, unrollable) instead of exec-masked.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

}  // namespace ct
