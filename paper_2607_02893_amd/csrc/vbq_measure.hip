// Measurement aid of the roofline harness (not part of the method): the rate
// at which the device streams a large buffer from HBM with plain reads, the
// ceiling the fused GEMV kernels are measured against.
//
// Each lane reads 16-byte chunks with non-temporal loads, four in flight per
// iteration, in a grid-stride loop, and folds them with XOR; each workgroup
// writes one word, so no load can be dropped by the compiler.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/vbq.h"

vbq_status vbq_detail_hip_status(hipError_t e);

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kReadThreads = 256;

__global__ __launch_bounds__(kReadThreads) void vbq_read_kernel(const u32x4* __restrict__ src, uint64_t n16,
                                                                 uint32_t* __restrict__ sink) {
  const uint64_t stride = (uint64_t)gridDim.x * kReadThreads;
  uint64_t i = (uint64_t)blockIdx.x * kReadThreads + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(src + i);
    const u32x4 b = __builtin_nontemporal_load(src + i + stride);
    const u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride);
    const u32x4 d = __builtin_nontemporal_load(src + i + 3 * stride);
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n16; i += stride) acc ^= __builtin_nontemporal_load(src + i);
  uint32_t v = acc.x ^ acc.y ^ acc.z ^ acc.w;
  // a fixed butterfly over the wave, then one word per wave (the waves of a
  // block write adjacent words of the block's slot)
  for (int off = 32; off >= 1; off >>= 1) v ^= (uint32_t)__shfl_xor((int)v, off);
  if ((threadIdx.x & 63) == 0) sink[(size_t)blockIdx.x * (kReadThreads / 64) + (threadIdx.x >> 6)] = v;
}

}  // namespace

extern "C" {

vbq_status vbq_read_ceiling(const void* src_dev, size_t bytes, uint32_t blocks, uint32_t* sink_dev, void* stream) {
  if (bytes == 0) return VBQ_OK;
  if (!src_dev || !sink_dev) return VBQ_ERR_NULL;
  if (bytes % 16 || (uintptr_t)src_dev % 16 || (uintptr_t)sink_dev % 4) return VBQ_ERR_BUFFER;
  if (blocks == 0) blocks = 8192;
  if (blocks > (1u << 20)) return VBQ_ERR_UNSUPPORTED;
  uint64_t n16 = bytes / 16;
  void* args[] = {(void*)&src_dev, (void*)&n16, (void*)&sink_dev};
  return vbq_detail_hip_status(
      hipLaunchKernel((const void*)vbq_read_kernel, dim3(blocks), dim3(kReadThreads), args, 0, (hipStream_t)stream));
}

}  // extern "C"
