// Kernels shared by every family: the fixed-order split reduction, the
// on-device verification of a candidate's output, and the probes behind CU
// masks and rooflines (CU identity, empty-kernel dispatch floor, copy
// bandwidth).
#include <hip/hip_runtime.h>

#include "ct_internal.h"

namespace ct {

// y[i] = ws[i] + ws[n + i] + ... in split order: the same sum for every run
// (the 16-byte variant below adds the same terms in the same order).
__global__ void split_reduce_kernel(const float* __restrict__ ws, float* __restrict__ y, int64_t n,
                                    int split) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    float s = ws[i];
    for (int j = 1; j < split; ++j) s += ws[(int64_t)j * n + i];
    y[i] = s;
  }
}

// The same sum 16 bytes per lane: n4 = n / 4 float4 per partial, partial j
// starting at ws + j * n (n a multiple of 4, ws and y 16-byte aligned).
typedef float f4v __attribute__((ext_vector_type(4)));
__global__ void split_reduce4_kernel(const f4v* __restrict__ ws, f4v* __restrict__ y, int64_t n4, int split) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    f4v s = ws[i];
    for (int j = 1; j < split; ++j) s += ws[(int64_t)j * n4 + i];
    y[i] = s;
  }
}

int launch_split_reduce(const float* ws, float* y, int64_t n, int split, void* stream) {
  const int threads = 256;
  if (n % 4 == 0 && ((uintptr_t)ws % 16) == 0 && ((uintptr_t)y % 16) == 0) {
    const int64_t n4 = n / 4;
    int64_t blocks = (n4 + threads - 1) / threads;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(split_reduce4_kernel, dim3((unsigned)blocks), dim3(threads), 0, (hipStream_t)stream,
                       (const f4v*)ws, (f4v*)y, n4, split);
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }
  int64_t blocks = (n + threads - 1) / threads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)blocks), dim3(threads), 0,
                     (hipStream_t)stream, ws, y, n, split);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Order-independent maxima of |y - ref| and |ref| (non-negative floats compare
// like their bit patterns, so integer atomicMax gives the exact maximum).
// A NaN in y counts as an infinite error.
__global__ void max_error_kernel(const float* __restrict__ y, const float* __restrict__ ref,
                                 int64_t n, unsigned* __restrict__ out) {
  float e = 0.f, m = 0.f;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float d = fabsf(y[i] - ref[i]);
    e = (d != d) ? INFINITY : fmaxf(e, d);
    m = fmaxf(m, fabsf(ref[i]));
  }
  for (int off = 32; off > 0; off >>= 1) {
    e = fmaxf(e, __shfl_xor(e, off));
    m = fmaxf(m, __shfl_xor(m, off));
  }
  if ((threadIdx.x & 63) == 0) {
    atomicMax(&out[0], __float_as_uint(e));
    atomicMax(&out[1], __float_as_uint(m));
  }
}

__global__ void fill_u32_kernel(unsigned* p, int n, unsigned v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

int launch_max_error(const float* y, const float* ref, int64_t n, unsigned* out2, hipStream_t st) {
  hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, st, out2, 2, 0u);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(max_error_kernel, dim3((unsigned)blocks), dim3(256), 0, st, y, ref, n, out2);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ---- probes ----
// Each one-wave block records where it ran: XCC_ID and HW_ID (SE, SH, CU).
__global__ void cu_probe_kernel(int* __restrict__ out, int nblocks) {
  // simm16 = (size - 1) << 11 | offset << 6 | register id; HW_ID is id 4,
  // XCC_ID is id 20 on this architecture.
  const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);
  const unsigned xcc = __builtin_amdgcn_s_getreg((15 << 11) | 20);
  // spin briefly so that blocks spread over the allowed CUs
  long t0 = clock64();
  while (clock64() - t0 < 20000) {
  }
  if (threadIdx.x == 0 && (int)blockIdx.x < nblocks) {
    const int cu = (hw >> 8) & 0xF, sh = (hw >> 12) & 0x1, se = (hw >> 13) & 0x7;
    out[blockIdx.x] = (int)((xcc & 0xF) << 12 | se << 8 | sh << 4 | cu);
  }
}

int launch_cu_probe(int* out, int nblocks, hipStream_t st) {
  hipLaunchKernelGGL(cu_probe_kernel, dim3(nblocks), dim3(64), 0, st, out, nblocks);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

__global__ void empty_kernel() {}

int launch_empty(int nblocks, hipStream_t st) {
  hipLaunchKernelGGL(empty_kernel, dim3(nblocks), dim3(64), 0, st);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// 16-byte vector copy; the tail is copied bytewise.
__global__ void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t nvec,
                            const unsigned char* __restrict__ src_b, unsigned char* __restrict__ dst_b,
                            int64_t tail_begin, int64_t tail_end) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t; i < nvec; i += stride) dst[i] = src[i];
  for (int64_t i = tail_begin + t; i < tail_end; i += stride) dst_b[i] = src_b[i];
}

int launch_copy(const void* src, void* dst, int64_t bytes, int nblocks, hipStream_t st) {
  const int64_t nvec = bytes / 16;
  hipLaunchKernelGGL(copy_kernel, dim3(nblocks), dim3(256), 0, st, (const uint4*)src, (uint4*)dst,
                     nvec, (const unsigned char*)src, (unsigned char*)dst, nvec * 16, bytes);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace ct
