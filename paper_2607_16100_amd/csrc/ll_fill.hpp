// Fill kernels used by the host entry points (region and output set-up).
#pragma once

#include "ll_device.hpp"

namespace llc {

// Set `bytes` bytes at `dst` (16-byte aligned) to 0xFF: the sentinel of
// every element type.
__global__ __launch_bounds__(256) void k_fill_ones(char *dst, uint64_t bytes) {
  const uint64_t full = bytes / 16;
  const u32x4 ones = {0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu, 0xFFFFFFFFu};
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (uint64_t i = t; i < full; i += (uint64_t)gridDim.x * blockDim.x) *(u32x4 *)(dst + i * 16) = ones;
  if (t < bytes % 16) dst[full * 16 + t] = (char)0xFF;
}

// Fill bytes [lo, hi) of every slice with the dword `value`.
__global__ __launch_bounds__(256) void k_fill_areas(char *sym, uint64_t stride, int nranks, uint64_t lo, uint64_t hi,
                                                  uint32_t value) {
  const uint64_t per = (hi - lo) / 16;
  const uint64_t total = per * (uint64_t)nranks;
  const u32x4 z = {value, value, value, value};
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (uint64_t)gridDim.x * blockDim.x) {
    const uint64_t rk = i / per;
    const uint64_t k = i % per;
    *(u32x4 *)(sym + rk * stride + lo + k * 16) = z;
  }
}

}  // namespace llc
