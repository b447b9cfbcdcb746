// Measurement helpers for the benchmark (libsplash_calib.so): the chip's
// achievable streaming-read bandwidth, its bf16 MFMA rate on random operands,
// and a clean cache flush (a read of a large buffer, which leaves no dirty
// lines to write back during the next timed kernel).  Nothing here is part of
// the attention path.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "splash_calib.h"

namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Grid-stride read of n16 16-byte words, four in flight per lane, with
// non-temporal loads; one word per thread is written so the reads stay.
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4* __restrict__ src, size_t n16,
                                                          uint32_t* sink) {
  u32x4 acc = {0, 0, 0, 0};
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(src + i), b = __builtin_nontemporal_load(src + i + stride);
    const u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride), d = __builtin_nontemporal_load(src + i + 3 * stride);
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n16; i += stride) acc ^= src[i];
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

// Four independent accumulation chains of v_mfma_f32_32x32x16_bf16 per wave,
// operands (8 fragments per lane) read once from memory.
__global__ __launch_bounds__(256) void mfma_loop_kernel(const bf16x8* ops, int iters, float* sink) {
  const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
  bf16x8 a[4], b[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    a[k] = ops[t * 8 + k];
    b[k] = ops[t * 8 + 4 + k];
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[k], b[k], c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(k + 1) & 3], b[k], c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(k + 2) & 3], b[k], c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(k + 3) & 3], b[k], c3, 0, 0, 0);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  sink[t] = s;
}

}  // namespace

extern "C" {

int splash_calib_stream_read(const void* buf, size_t bytes, void* sink, int32_t blocks, void* stream) {
  if (!buf || !sink || blocks < 1 || (reinterpret_cast<uintptr_t>(buf) & 15u)) return -1;
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const u32x4*>(buf), bytes / 16, static_cast<uint32_t*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

size_t splash_calib_mfma_ops_bytes(int32_t blocks) { return blocks < 1 ? 0 : (size_t)blocks * 256 * 8 * 16; }

int splash_calib_mfma_loop(const void* ops, int32_t iters, void* sink, int32_t blocks, void* stream) {
  if (!ops || !sink || blocks < 1 || iters < 1 || (reinterpret_cast<uintptr_t>(ops) & 15u)) return -1;
  hipLaunchKernelGGL(mfma_loop_kernel, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const bf16x8*>(ops), iters, static_cast<float*>(sink));
  return hipGetLastError() == hipSuccess ? 0 : -5;
}

double splash_calib_mfma_flops(int32_t blocks, int32_t iters) {
  // 4 waves x 16 MFMAs of 32 x 32 x 16 (2 * 16384 flops) per iteration
  return (double)blocks * 4.0 * 16.0 * 32768.0 * (double)iters;
}

}  // extern "C"
