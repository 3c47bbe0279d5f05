// Measurement probes: what the device sustains on the two resources the
// attention step is bound by, so that a kernel's rate can be stated as a
// fraction of a measured peak beside the datasheet one.
//
//   mpa_probe_stream_read  HBM read bandwidth: every byte of a buffer is read
//                          once with 16-byte non-temporal vector loads,
//                          contiguous 4 KB runs per workgroup (plain loads
//                          sustain about a tenth less on gfx950).
//   mpa_probe_mfma_bf16    dense bf16 matrix-core rate: independent chains of
//                          v_mfma_f32_32x32x16_bf16 with operands in registers.
//
// Neither is part of the attention path; both launch on the caller's stream
// and allocate nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mpa.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 4;       // 16-byte loads in flight per lane per iteration
constexpr int kReadGroups = 256 * 8; // workgroups: 8 per CU
constexpr int kMfmaThreads = 256;
constexpr int kMfmaGroups = 256 * 4; // 4 waves per SIMD
constexpr int kMfmaChains = 4;       // independent accumulators per wave

// Iteration `it` of workgroup g covers the kReadUnroll * 256 vectors from
// (it * grid + g) * kReadUnroll * 256; lane t reads vectors t, t + 256, ...
// of that run, so each wave instruction reads 1 KB contiguously.
__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const u32x4* __restrict__ src, size_t n16,
                                                                 uint32_t* sink) {
  const size_t run = (size_t)kReadThreads * kReadUnroll;
  uint32_t acc = 0;
  for (size_t base = (size_t)blockIdx.x * run; base < n16; base += (size_t)gridDim.x * run) {
    u32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) {
      const size_t i = base + (size_t)u * kReadThreads + threadIdx.x;
      v[u] = i < n16 ? __builtin_nontemporal_load(src + i) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  // The loads feed a value the kernel may store, so they cannot be removed.
  if (acc == 0x9e3779b9u) sink[0] = acc;
}

__global__ __launch_bounds__(kMfmaThreads) void mfma_bf16_kernel(int iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (__bf16)(0.001f * (float)((lane + e) & 7));
    b[e] = (__bf16)(0.001f * (float)((lane * 3 + e) & 7));
  }
  f32x16 c[kMfmaChains];
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) c[k][e] = 0.f;
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < kMfmaChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < kMfmaChains; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[k][e];
  if (s == -1.f) sink[0] = s;  // the products are >= 0: never taken, but keeps the MFMAs
}

}  // namespace

extern "C" {

int mpa_probe_stream_read(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
  if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || ((uintptr_t)buf & 15) != 0) return MPA_ERR_INVALID;
  (void)hipGetLastError();
  const size_t n16 = bytes / 16;
  const size_t runs = (n16 + (size_t)kReadThreads * kReadUnroll - 1) / ((size_t)kReadThreads * kReadUnroll);
  const unsigned grid = (unsigned)(runs < (size_t)kReadGroups ? runs : (size_t)kReadGroups);
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(kReadThreads), 0, (hipStream_t)stream,
                     (const u32x4*)buf, n16, sink);
  return hipGetLastError() == hipSuccess ? MPA_OK : MPA_ERR_HIP;
}

int mpa_probe_mfma_bf16(int32_t iters, float* sink, double* flops, void* stream) {
  if (iters <= 0 || !sink) return MPA_ERR_INVALID;
  (void)hipGetLastError();
  hipLaunchKernelGGL(mfma_bf16_kernel, dim3(kMfmaGroups), dim3(kMfmaThreads), 0, (hipStream_t)stream, iters, sink);
  if (flops)  // 32 x 32 x 16 multiply-adds per instruction per wave
    *flops = 2.0 * 32 * 32 * 16 * kMfmaChains * (double)iters * kMfmaGroups * (kMfmaThreads / 64);
  return hipGetLastError() == hipSuccess ? MPA_OK : MPA_ERR_HIP;
}

}  // extern "C"
