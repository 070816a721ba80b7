// Streaming-read probe of HBM (a measurement utility beside the codec): what
// plain reads of device memory reach on this device.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "hufflm.h"

namespace hl {

// Streaming read of n16 16-byte words (a measurement probe: what plain reads
// of HBM reach): every thread XORs its words, four 16-byte loads in flight,
// and one word per block is written so that the reads are not removed.
__global__ void __launch_bounds__(1024) read_probe_kernel(const uint4* src, uint64_t n16, uint32_t* out) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint4 acc = make_uint4(0, 0, 0, 0);
  for (; k + 3 * stride < n16; k += 4 * stride) {
    const uint4 a = src[k], b = src[k + stride], c = src[k + 2 * stride], d = src[k + 3 * stride];
    acc.x ^= a.x ^ b.x ^ c.x ^ d.x;
    acc.y ^= a.y ^ b.y ^ c.y ^ d.y;
    acc.z ^= a.z ^ b.z ^ c.z ^ d.z;
    acc.w ^= a.w ^ b.w ^ c.w ^ d.w;
  }
  for (; k < n16; k += stride) {
    const uint4 a = src[k];
    acc.x ^= a.x;
    acc.y ^= a.y;
    acc.z ^= a.z;
    acc.w ^= a.w;
  }
  uint32_t v = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v ^= (uint32_t)__shfl_xor((int)v, d, 64);
  __shared__ uint32_t s_red[16];
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (uint32_t w = 0; w < (blockDim.x >> 6); ++w) t ^= s_red[w];
    out[blockIdx.x] = t;
  }
}

static uint32_t probe_blocks() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus <= 0)
    cus = 256;
  return (uint32_t)cus * 4;
}

}  // namespace hl

extern "C" uint32_t hl_read_probe_blocks(void) { return hl::probe_blocks(); }

extern "C" hl_status hl_read_probe(const void* src_dev, size_t bytes, uint32_t* out_dev, void* stream) {
  if (!src_dev || !out_dev || bytes < 16 || bytes % 16 || reinterpret_cast<uintptr_t>(src_dev) % 16)
    return HL_EINVAL;
  hipLaunchKernelGGL(hl::read_probe_kernel, dim3(hl::probe_blocks()), dim3(1024), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint4*>(src_dev), (uint64_t)(bytes / 16), out_dev);
  return hipGetLastError() == hipSuccess ? HL_OK : HL_EHIP;
}
