// Iterations of an AllReduce call, shared by the host plan and the kernels.
//
// A call of `total` elements per rank runs in iterations of `iter_n`
// elements (one iteration unless its scratch is bounded, Sec. IV
// "Bidirectional Communication & Double Buffering").  Iteration `it` covers
// elements [e0, e0 + n) of every rank; its two-shot chunk is ceil(n / P)
// rounded up to 16 bytes, so chunk c covers [c*chunk, min((c+1)*chunk, n))
// of the iteration and the last chunks may be short or empty.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace llc {

struct IterSpan {
  int64_t e0;     // first element of the iteration
  int64_t n;      // elements in the iteration
  int64_t chunk;  // two-shot chunk length of the iteration, in elements
};

__host__ __device__ inline IterSpan iter_span(int64_t total, int64_t iter_n, uint32_t it, int P, int esize) {
  IterSpan s;
  s.e0 = (int64_t)it * iter_n;
  const int64_t left = total - s.e0;
  s.n = left < 0 ? 0 : (left < iter_n ? left : iter_n);
  const int64_t g = 16 / esize;
  s.chunk = ((s.n + P - 1) / P + g - 1) / g * g;
  return s;
}

// Elements of chunk c within an iteration of n elements cut into chunks of C.
__host__ __device__ inline int64_t chunk_len(int64_t n, int64_t C, int c) {
  const int64_t left = n - (int64_t)c * C;
  return left < 0 ? 0 : (left < C ? left : C);
}

}  // namespace llc
