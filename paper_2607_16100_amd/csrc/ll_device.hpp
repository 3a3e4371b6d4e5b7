// Device primitives for the low-latency collectives (gfx950 / CDNA4).
//
// Packets (the paper's LL protocol, Sec. IV; send/recv of Sec. V):
//   * 8-byte packet  = {payload u32, flag u32}.  A lane moves two packets in
//     one 16-byte store, so a wave writes 1 KiB contiguous per instruction.
//   * 128-byte line  = 8 lanes x 16 bytes.  The last dword of each 64-byte
//     half is the flag, the other 30 dwords are payload (120 of 128 bytes).
// The flag is the call's epoch.  A receiver accepts a packet once every flag
// covering it equals the epoch; zeroed scratch (flag 0) never matches.
//
// Cross-XCD visibility without fences: every packet store and every poll
// load carries the sc1 cache-policy bit (agent scope), which is how the
// compiler itself implements relaxed agent-scope atomic loads and stores on
// this chip.  Such a store is written through to the device coherence point
// and such a load does not hit a stale line in the reader's own L2, so no
// release/acquire fence (which would write back or invalidate a whole L2)
// is needed on the per-call path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace llc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// gfx950 cache-policy immediates for buffer instructions.
constexpr int kSC1 = 16;  // agent-scope coherent access
constexpr int kNT = 2;    // streaming (non-temporal) hint

// Third dword of a raw buffer resource on gfx9-family chips (32-bit data
// format so that range checking is in bytes).
constexpr int kRsrcWord3 = 0x00020000;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcWord3);
}

// Coherent 16-byte packet store / load.  Offsets past the resource's size are
// discarded (store) or read as zero (load), so a wrong offset can never touch
// memory outside the slot; a zero flag is never accepted.
__device__ __forceinline__ void st_pkt(rsrc_t rs, uint32_t off, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, rs, (int)off, 0, kSC1);
}
__device__ __forceinline__ u32x4 ld_pkt(rsrc_t rs, uint32_t off, uint32_t soff = 0) {
  return __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, (int)soff, kSC1);
}

// A value every lane of the wave holds; tells the compiler it lives in a
// scalar register (so buffer offsets never need a per-lane loop).
__device__ __forceinline__ uint32_t uniform_u32(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

// Keeps the compiler from treating a polled location as loop-invariant.
__device__ __forceinline__ void compiler_fence() { __asm__ __volatile__("" ::: "memory"); }

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// ---------------------------------------------------------------------------
// Element types.  A payload word holds one binary32 or two bfloat16 values
// (element 2k in the low half).
template <int DT> struct Elem;

template <> struct Elem<0> {  // binary32
  static constexpr int kBytes = 4;
  static constexpr int kPerWord = 1;
  __device__ static __forceinline__ void widen(uint32_t w, float *f) { f[0] = __uint_as_float(w); }
  __device__ static __forceinline__ uint32_t narrow(const float *f) { return __float_as_uint(f[0]); }
};

template <> struct Elem<1> {  // bfloat16
  static constexpr int kBytes = 2;
  static constexpr int kPerWord = 2;
  __device__ static __forceinline__ void widen(uint32_t w, float *f) {
    f[0] = __uint_as_float(w << 16);            // exact
    f[1] = __uint_as_float(w & 0xffff0000u);    // exact
  }
  // binary32 -> bfloat16 with round to nearest even (the hardware conversion).
  __device__ static __forceinline__ uint32_t narrow(const float *f) {
    __bf16 lo = (__bf16)f[0];
    __bf16 hi = (__bf16)f[1];
    uint16_t l = __builtin_bit_cast(uint16_t, lo);
    uint16_t h = __builtin_bit_cast(uint16_t, hi);
    return (uint32_t)l | ((uint32_t)h << 16);
  }
};

// ---------------------------------------------------------------------------
// Loading / storing a lane's payload words from / to element streams.
//
// A stream is `nelem` elements starting at byte address `base`.  Word k of a
// stream covers elements [k*kPerWord, (k+1)*kPerWord).  `al4` says the base is
// 4-byte aligned; otherwise (bfloat16 streams that start on an odd element)
// elements are moved one at a time.
template <int DT>
__device__ __forceinline__ u32x4 load_words(const char *base, int64_t w0, int cnt, int64_t nelem, bool al4) {
  constexpr int K = Elem<DT>::kPerWord;
  u32x4 v = {0u, 0u, 0u, 0u};
  const int64_t e0 = w0 * K;
  if (al4 && e0 + (int64_t)cnt * K <= nelem) {
    const char *p = base + w0 * 4;
    if (cnt == 4) {
      __builtin_memcpy(&v, p, 16);
    } else if (cnt == 3) {
      uint32_t t[3];
      __builtin_memcpy(t, p, 12);
      v.x = t[0]; v.y = t[1]; v.z = t[2];
    } else if (cnt == 2) {
      u32x2 t;
      __builtin_memcpy(&t, p, 8);
      v.x = t.x; v.y = t.y;
    } else {
      uint32_t t;
      __builtin_memcpy(&t, p, 4);
      v.x = t;
    }
    return v;
  }
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  for (int i = 0; i < cnt * K; ++i) {
    int64_t e = e0 + i;
    if (e < nelem) {
      uint32_t x;
      if (DT == 0) {
        x = *(const uint32_t *)(base + e * 4);
      } else {
        x = *(const uint16_t *)(base + e * 2);
      }
      w[i / K] |= x << (16 * (i % K));
    }
  }
  v.x = w[0]; v.y = w[1]; v.z = w[2]; v.w = w[3];
  return v;
}

template <int DT>
__device__ __forceinline__ void store_words(char *base, int64_t w0, int cnt, int64_t nelem, bool al4, u32x4 v) {
  constexpr int K = Elem<DT>::kPerWord;
  const int64_t e0 = w0 * K;
  if (al4 && e0 + (int64_t)cnt * K <= nelem) {
    char *p = base + w0 * 4;
    if (cnt == 4) {
      __builtin_memcpy(p, &v, 16);
    } else if (cnt == 3) {
      uint32_t t[3] = {v.x, v.y, v.z};
      __builtin_memcpy(p, t, 12);
    } else if (cnt == 2) {
      u32x2 t = {v.x, v.y};
      __builtin_memcpy(p, &t, 8);
    } else {
      const uint32_t t = v.x;
      __builtin_memcpy(p, &t, 4);
    }
    return;
  }
  uint32_t w[4] = {v.x, v.y, v.z, v.w};
  for (int i = 0; i < cnt * K; ++i) {
    int64_t e = e0 + i;
    if (e < nelem) {
      uint32_t x = w[i / K] >> (16 * (i % K));
      if (DT == 0) {
        *(uint32_t *)(base + e * 4) = x;
      } else {
        *(uint16_t *)(base + e * 2) = (uint16_t)x;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Packet formats.  `sub` is the lane's position inside a unit (0 for 8-byte
// packets, 0..7 for a line); a unit is what one group of lanes moves with one
// 16-byte store each.
struct ProtoLL {
  static constexpr int kLanes = 1;        // lanes per unit
  static constexpr int kUnitBytes = 16;   // bytes per unit in a slot
  static constexpr int kUnitWords = 2;    // payload words per unit
  static constexpr int kMaxWords = 2;     // payload words per lane
  __device__ static __forceinline__ int64_t word0(int64_t u, int /*sub*/) { return 2 * u; }
  __device__ static __forceinline__ int count(int /*sub*/) { return 2; }
  __device__ static __forceinline__ u32x4 pack(u32x4 w, uint32_t epoch, int /*sub*/) {
    u32x4 p = {w.x, epoch, w.y, epoch};
    return p;
  }
  __device__ static __forceinline__ bool ready(u32x4 p, uint32_t epoch) { return p.y == epoch && p.w == epoch; }
  __device__ static __forceinline__ u32x4 unpack(u32x4 p, int /*sub*/) {
    u32x4 w = {p.x, p.z, 0u, 0u};
    return w;
  }
  static constexpr __host__ __device__ int64_t units(int64_t words) { return (words + 1) / 2; }
};

struct ProtoLine {
  static constexpr int kLanes = 8;
  static constexpr int kUnitBytes = 128;
  static constexpr int kUnitWords = 30;
  static constexpr int kMaxWords = 4;
  __device__ static __forceinline__ int64_t word0(int64_t u, int sub) {
    return 30 * u + 15 * (sub >> 2) + 4 * (sub & 3);
  }
  __device__ static __forceinline__ int count(int sub) { return (sub & 3) == 3 ? 3 : 4; }
  __device__ static __forceinline__ u32x4 pack(u32x4 w, uint32_t epoch, int sub) {
    if ((sub & 3) == 3) w.w = epoch;
    return w;
  }
  // The flag of a 64-byte half sits in lane 3 of its quad; broadcast it to the
  // quad with DPP.  All four lanes of a quad are always active together.
  __device__ static __forceinline__ bool ready(u32x4 p, uint32_t epoch) {
    uint32_t f = (uint32_t)__builtin_amdgcn_mov_dpp((int)p.w, 0xFF /* quad_perm:[3,3,3,3] */, 0xF, 0xF, false);
    return f == epoch;
  }
  __device__ static __forceinline__ u32x4 unpack(u32x4 p, int sub) {
    if ((sub & 3) == 3) p.w = 0u;
    return p;
  }
  static constexpr __host__ __device__ int64_t units(int64_t words) { return (words + 29) / 30; }
};

// ---------------------------------------------------------------------------
// Status word shared by all kernels of the library: [0] = error code (0 = ok),
// [1] = rank, [2] = mask of peers not heard from, [3] = epoch.
extern __device__ uint32_t g_ll_status[4];

constexpr uint32_t kStatusTimeout = 1;

__device__ __forceinline__ void report_timeout(int rank, uint32_t pending, uint32_t epoch) {
  uint32_t expected = 0;
  if (__hip_atomic_compare_exchange_strong(&g_ll_status[0], &expected, kStatusTimeout, __ATOMIC_RELAXED,
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
    __hip_atomic_store(&g_ll_status[1], (uint32_t)rank, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&g_ll_status[2], pending, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&g_ll_status[3], epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

}  // namespace llc
