// Slice layout arithmetic (host side).
//
// A region is P slices of `stride` bytes.  Each slice is
//   [0, cap)                   input area (the rank's input at offset 0)
//   [cap, cap + A8)            8-byte packet area
//   [cap + A8, cap + A8 + A128) 128-byte line area
//   [.., .. + AA)              atomic accumulator and tile counters
//   [.., .. + AS)              sentinel area (payload only, reset after use)
// An area is present only if the region holds that packet format: the
// region's format set is (stride / 256) mod 16, a bit per format (kFmt8,
// kFmtLine, kFmtSent, kFmtAtomic), where 0 stands for all four -- so any
// stride that is a multiple of 4 KiB holds every format, and ll_slice_bytes
// adds the bits of a one-algorithm region to a multiple of 4 KiB.  cap is the
// largest multiple of 256 for which the present areas, each sized for the most
// demanding algorithm of its format at an input of cap bytes, fit in the
// slice.  The layout therefore depends only on (stride, P): a byte that
// holds input in one call is never read as a flag in another, and two packet
// formats never share bytes, so a stale payload word can never pose as a
// flag.  The sentinel area holds nothing but payload and sentinels.
//
// Within an area a call places its slots from the area's start:
//   one-shot / AllGather   P-1 slots, each holding a full input
//   ReduceScatter          P-1 slots, each holding one chunk
//   two-shot               P-1 ReduceScatter slots, then P-1 AllGather slots,
//                          each holding one chunk
// In the 8-byte area every packet is 8-byte aligned, so flags always sit at
// the odd dwords; in the line area every line is 128-byte aligned, so flags
// always sit at dwords 15 and 31 of a line.
#pragma once

#include <stdint.h>

#include <algorithm>

namespace llc {
namespace layout {

constexpr uint64_t kAlign = 256;
constexpr uint64_t kMaxInputBytes = 256ull << 20;  // keeps every call's P-1 slots within 4 GiB
constexpr uint64_t kMaxBufferedBytes = 16ull << 30;  // per-rank message of a bounded-scratch call

inline uint64_t roundup(uint64_t x, uint64_t m) { return (x + m - 1) / m * m; }
inline uint64_t ceil_div(uint64_t x, uint64_t m) { return (x + m - 1) / m; }

// Slot bytes for a payload of `bytes`.
inline uint64_t slot8(uint64_t bytes) { return roundup(ceil_div(bytes, 4) * 8, kAlign); }
// Line packets travel in 1 KiB units (a wave of 8 lines) carrying 240 payload words.
inline uint64_t slot128(uint64_t bytes) { return roundup(ceil_div(ceil_div(bytes, 4), 240) * 1024, kAlign); }

// Two-shot chunk length in elements: ceil(n / P) rounded up to 16 bytes.
inline uint64_t twoshot_chunk(uint64_t n, int P, int esize) {
  const uint64_t g = 16 / (uint64_t)esize;
  return roundup(ceil_div(n, (uint64_t)P), g);
}

// Upper bound of a two-shot chunk's bytes for an input of M bytes, for either
// element size (ceil(n/P)*esize <= M/P + 4).
inline uint64_t chunk_bound(uint64_t M, int P) { return roundup(ceil_div(M, (uint64_t)P) + 4, 16); }

inline uint64_t area8(uint64_t M, int P) {
  const uint64_t p1 = (uint64_t)(P - 1);
  return std::max(p1 * slot8(M), 2 * p1 * slot8(chunk_bound(M, P)));
}

inline uint64_t area128(uint64_t M, int P) {
  const uint64_t p1 = (uint64_t)(P - 1);
  return std::max(p1 * slot128(M), 2 * p1 * slot128(chunk_bound(M, P)));
}

// Sentinel slots carry payload only: a 16-byte unit holds 4 payload words.
inline uint64_t slotS(uint64_t bytes) { return roundup(ceil_div(bytes, 16) * 16, kAlign); }

inline uint64_t areaS(uint64_t M, int P) {
  const uint64_t p1 = (uint64_t)(P - 1);
  return std::max(p1 * slotS(M), 2 * p1 * slotS(chunk_bound(M, P)));
}

// Atomic-accumulation two-shot: a binary32 accumulator covering the rank's
// chunk in whole tiles of 1 KiB of input (4 KiB of accumulator for binary32
// tiles, 8 KiB for bfloat16), and one u32 counter per tile.
inline uint64_t atomic_acc_bytes(uint64_t chunk_bytes, int esize) {
  return roundup(ceil_div(chunk_bytes, 1024) * 4096 / (uint64_t)esize, kAlign);
}
inline uint64_t areaA(uint64_t M, int P) {
  const uint64_t cb = chunk_bound(M, P);
  return atomic_acc_bytes(cb, 2) + roundup(4 * ceil_div(cb, 1024), kAlign);
}

// Packet formats a region holds (bits of the format set).
constexpr unsigned kFmt8 = 1, kFmtLine = 2, kFmtSent = 4, kFmtAtomic = 8, kFmtAll = 15;
constexpr uint64_t kFmtUnit = 4096;  // strides with no format bits are multiples of this

// The format set of a region with this stride.
inline unsigned formats_of(uint64_t stride) {
  const unsigned m = (unsigned)((stride / kAlign) % 16);
  return m == 0 ? kFmtAll : m;
}

// Area sizes of a slice with input capacity cap and format set fmt.
struct Areas {
  uint64_t a8, a128, aa, as;
};
inline Areas areas(uint64_t cap, int P, unsigned fmt) {
  Areas a;
  a.a8 = (fmt & kFmt8) ? area8(cap, P) : 0;
  a.a128 = (fmt & kFmtLine) ? area128(cap, P) : 0;
  a.aa = (fmt & kFmtAtomic) ? areaA(cap, P) : 0;
  a.as = (fmt & kFmtSent) ? areaS(cap, P) : 0;
  return a;
}

inline uint64_t slice_for(uint64_t cap, int P, unsigned fmt = kFmtAll) {
  const Areas a = areas(cap, P, fmt);
  return cap + a.a8 + a.a128 + a.aa + a.as;
}

// The smallest stride with format set fmt whose slices hold an input of cap
// bytes: a multiple of 4 KiB plus the format bits.
inline uint64_t stride_for(uint64_t cap, int P, unsigned fmt) {
  const uint64_t need = slice_for(cap, P, fmt);
  const uint64_t bits = fmt == kFmtAll ? 0 : (uint64_t)fmt * kAlign;
  uint64_t s = need / kFmtUnit * kFmtUnit + bits;
  if (s < need) s += kFmtUnit;
  return s;
}

// Largest cap (multiple of 256, at most kMaxInputBytes) with
// slice_for(cap, P, formats_of(stride)) <= stride.
inline uint64_t capacity(uint64_t stride, int P) {
  const unsigned fmt = formats_of(stride);
  uint64_t lo = 0, hi = std::min(stride, kMaxInputBytes) / kAlign;
  while (lo < hi) {
    const uint64_t mid = (lo + hi + 1) / 2;
    if (slice_for(mid * kAlign, P, fmt) <= stride) {
      lo = mid;
    } else {
      hi = mid - 1;
    }
  }
  return lo * kAlign;
}

// Bounded scratch (multi-iteration calls with an input outside the region).
// A scratch slice holds, per packet format, two sub-buffers, each sized like
// that format's area for an input of D bytes; a call of M bytes per rank runs
// in ceil(M / D) iterations alternating between the sub-buffers:
//   [0, 2*A8(D))                 8-byte packet sub-buffers 0 and 1
//   [2*A8(D), .. + 2*A128(D))    line sub-buffers 0 and 1
//   [.., .. + 2*AS(D))           sentinel sub-buffers 0 and 1
inline uint64_t scratch_for(uint64_t D, int P) { return 2 * (area8(D, P) + area128(D, P) + areaS(D, P)); }

// Largest iteration size D (multiple of 256, at most kMaxInputBytes) whose
// scratch fits in `stride` bytes; 0 if none does.
inline uint64_t iter_capacity(uint64_t stride, int P) {
  uint64_t lo = 0, hi = std::min(stride, kMaxInputBytes) / kAlign;
  while (lo < hi) {
    const uint64_t mid = (lo + hi + 1) / 2;
    if (scratch_for(mid * kAlign, P) <= stride) {
      lo = mid;
    } else {
      hi = mid - 1;
    }
  }
  return lo * kAlign;
}

}  // namespace layout
}  // namespace llc
