// Device primitives for the low-latency collectives (gfx950 / CDNA4).
//
// Packets (the paper's LL protocol, Sec. IV; send/recv of Sec. V):
//   * 8-byte packet  = {payload u32, flag u32}.  A lane moves two packets in
//     one 16-byte store, so a wave writes 1 KiB contiguous per instruction.
//   * 128-byte line  = 8 lanes x 16 bytes.  The last dword of each 64-byte
//     half is the flag, the other 30 dwords are payload (120 of 128 bytes);
//     which payload word goes where is chosen so that every access to the
//     input and output is 16-byte aligned (ProtoLine below).
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
__device__ __forceinline__ void st_pkt_at(rsrc_t rs, uint32_t off, uint32_t soff, u32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, rs, (int)off, (int)soff, kSC1);
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

// Budget of a call's flag waits, in ticks of the 100 MHz constant clock, and
// where an expired wait is reported.  The clock is read for the first time at
// a wait's first timeout check, not at kernel entry: a clock read is a scalar
// memory round trip, and at entry it would stand between the kernel's start
// and its first loads and stores.  The budget therefore starts when a wait
// first runs long, which is all a bound on waiting needs.
//
// Status word (4 dwords, owned by the stream the call runs on): [0] = error
// code (0 = ok), [1] = rank, [2] = mask of peers not heard from, [3] = epoch.
// The first wait to expire records itself; later ones leave it alone.
constexpr uint32_t kStatusTimeout = 1;

struct WaitBudget {
  uint64_t budget = 0;
  uint64_t deadline = 0;
  uint32_t *status = nullptr;
  __device__ WaitBudget() {}
  __device__ WaitBudget(uint64_t ticks, uint32_t *st) : budget(ticks), status(st) {}
  __device__ __forceinline__ bool expired() {
    const uint64_t t = now_ticks();
    if (deadline == 0) {
      deadline = t + budget;
      return false;
    }
    return t > deadline;
  }
  __device__ __forceinline__ void report(int rank, uint32_t pending, uint32_t epoch) const {
    uint32_t expected = 0;
    if (__hip_atomic_compare_exchange_strong(&status[0], &expected, kStatusTimeout, __ATOMIC_RELAXED,
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
      __hip_atomic_store(&status[1], (uint32_t)rank, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&status[2], pending, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&status[3], epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
};

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
// Inputs are read once and outputs written once per call: load and store them
// with the streaming (non-temporal) hint so they do not displace the packets,
// which are read back soon after they are written.  A kernel whose waves all
// read the same input words (the one-wave-per-peer one-shot) loads them
// through the cache instead (NT = false), so that the waves share one memory
// read.
#ifndef LLCOLL_NT_IN
#define LLCOLL_NT_IN 1
#endif
#ifndef LLCOLL_NT_OUT
#define LLCOLL_NT_OUT 1
#endif

template <int DT, bool NT = true>
__device__ __forceinline__ u32x4 load_words(const char *base, int64_t w0, int cnt, int64_t nelem, bool al4) {
  constexpr int K = Elem<DT>::kPerWord;
  constexpr bool kNT = LLCOLL_NT_IN && NT;
  u32x4 v = {0u, 0u, 0u, 0u};
  const int64_t e0 = w0 * K;
  if (al4 && e0 + (int64_t)cnt * K <= nelem) {
    const char *p = base + w0 * 4;
    if (kNT && cnt == 4 && ((uintptr_t)p & 15) == 0) {
      v = __builtin_nontemporal_load((const u32x4 *)p);
    } else if (kNT && cnt == 2 && ((uintptr_t)p & 7) == 0) {
      const u32x2 t = __builtin_nontemporal_load((const u32x2 *)p);
      v.x = t.x;
      v.y = t.y;
    } else if (cnt == 4) {
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
    if (LLCOLL_NT_OUT && cnt == 4 && ((uintptr_t)p & 15) == 0) {
      __builtin_nontemporal_store(v, (u32x4 *)p);
    } else if (LLCOLL_NT_OUT && cnt == 2 && ((uintptr_t)p & 7) == 0) {
      const u32x2 t = {v.x, v.y};
      __builtin_nontemporal_store(t, (u32x2 *)p);
    } else if (cnt == 4) {
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

// Loading / storing a one-lane unit's payload words through a buffer resource
// (kernels whose streams start 4-byte aligned).  The resource covers the
// stream's bytes rounded up to whole words, so the hardware range check
// returns zeros for words past the end and drops stores to them: no branch
// is needed around the access.  For bfloat16 a last word that holds only one
// element (an odd count) carries, in its other half, two bytes that lie past
// the stream but inside the input area; that element is never stored, and
// clear_tail zeroes it where it matters (sentinel units, where it could
// complete a sentinel dword).  The clearing is a separate step so that a
// caller can put independent work between the load and it.
template <int NW>
__device__ __forceinline__ u32x4 load_words_rs(rsrc_t rs, uint32_t w0) {
  u32x4 v = {0u, 0u, 0u, 0u};
  if constexpr (NW == 2) {
    const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(rs, (int)(w0 * 4), 0, 0);
    v.x = t.x;
    v.y = t.y;
  } else {
    v = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(w0 * 4), 0, 0);
  }
  return v;
}

template <int DT, int NW>
__device__ __forceinline__ u32x4 clear_tail(u32x4 v, uint32_t w0, uint32_t nelem) {
  if constexpr (DT == 1) {
    // word w holds elements 2w and 2w+1
    if (2 * w0 + 1 >= nelem) v.x &= 0xFFFFu;
    if (2 * w0 + 3 >= nelem) v.y &= 0xFFFFu;
    if constexpr (NW == 4) {
      if (2 * w0 + 5 >= nelem) v.z &= 0xFFFFu;
      if (2 * w0 + 7 >= nelem) v.w &= 0xFFFFu;
    }
  }
  return v;
}

// The matching store of NW words at word w0, for a stream whose byte length
// is a multiple of 4 (so that no word is partly past the end); with the
// streaming hint unless NT is false.  Tiny outputs of several ranks share
// cache lines (the P outputs lie back to back), and there streaming stores
// from several XCDs into one line cost up to 0.8 us a call (8 bytes per rank
// at 8 ranks); plain stores do not.
template <int NW, bool NT = true>
__device__ __forceinline__ void store_words_rs(rsrc_t rs, uint32_t w0, u32x4 v) {
  constexpr int kPolicy = NT ? kNT : 0;
  if constexpr (NW == 2) {
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{v.x, v.y}, rs, (int)(w0 * 4), 0, kPolicy);
  } else {
    __builtin_amdgcn_raw_buffer_store_b128(v, rs, (int)(w0 * 4), 0, kPolicy);
  }
}

// A word index whose byte offset lies past every buffer resource: a load
// from it returns zeros without touching memory.
constexpr uint32_t kNoWord = 0x3FFFFFFCu;

// ---------------------------------------------------------------------------
// Packet formats.  A unit is what one group of lanes moves with one 16-byte
// packet store each; `sub` is the lane's position in its group.  Each format
// says which payload words of a stream a lane carries (load/store), how they
// sit in its 16 bytes of packet (pack/unpack) and when they have arrived
// (ready).
struct ProtoLL {
  // 8-byte packets {payload, flag}: a lane carries payload words 2u, 2u+1.
  static constexpr int kLanes = 1;        // lanes per unit
  static constexpr int kUnitBytes = 16;   // packet bytes per unit in a slot
  static constexpr int kUnitWords = 2;    // payload words per unit
  static constexpr int kMaxWords = 2;     // payload words per lane
  template <int DT, bool NT = true>
  __device__ static __forceinline__ u32x4 load(const char *base, int64_t u, int /*sub*/, int64_t nelem, bool al4) {
    return load_words<DT, NT>(base, 2 * u, 2, nelem, al4);
  }
  template <int DT>
  __device__ static __forceinline__ void store(char *base, int64_t u, int /*sub*/, int64_t nelem, bool al4, u32x4 w) {
    store_words<DT>(base, 2 * u, 2, nelem, al4, w);
  }
  // The first payload word of unit u that the lane loads (kNoWord: none),
  // and the step after the load (none here); see ProtoLine.
  __device__ static __forceinline__ uint32_t first_word(uint32_t u, int /*sub*/) { return 2 * u; }
  __device__ static __forceinline__ u32x4 finish_load(u32x4 v, int /*sub*/) { return v; }
  __device__ static __forceinline__ u32x4 start_store(u32x4 w, int /*sub*/) { return w; }
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

// 128-byte line packets: 8 lanes x 16 bytes a line, the last dword of each
// 64-byte quarter-wave group ("quad", 4 lanes) is the flag, so a line carries
// 30 payload dwords and two flags.  A wave's 64 lanes (8 lines, 1 KiB) form
// one unit carrying 240 payload words:
//   * data lanes 0..59 carry the 16-byte-aligned words 4*sub .. 4*sub+3 of the
//     unit, except that the flag lane of each quad (sub % 4 == 3) leaves its
//     last word out -- the flag takes its place;
//   * the extra lanes 60..63 carry those 15 displaced words: lane 60+i holds
//     words 64i+16c+15, c = 0..3, of quads 4i+c (lane 63's last dword is the
//     quad's flag).
// Every load and store of payload is thus one 16-byte aligned access per data
// lane; the displaced words move between lanes through the LDS crossbar
// (ds_bpermute), not through memory.  This is the displacement of the
// paper's LL128 design (Sec. IV), with the extra lanes in the role of its
// extra threads.
struct ProtoLine {
  static constexpr int kLanes = 64;
  static constexpr int kUnitBytes = 1024;
  static constexpr int kUnitWords = 240;
  static constexpr int kMaxWords = 4;
  // Lane `src`'s value of v, for every lane (all 64 lanes must be active).
  __device__ static __forceinline__ uint32_t from_lane(int src, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_ds_bpermute(src * 4, (int)v);
  }
  // The load in two halves, so that a caller can put independent work
  // between the memory load and the lane permutes that wait for it: load_raw
  // loads the data lanes' words, finish_load (whole wave active) moves the
  // displaced words into the extra lanes.
  template <int DT, bool NT = true>
  __device__ static __forceinline__ u32x4 load_raw(const char *base, int64_t u, int sub, int64_t nelem, bool al4) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (sub < 60) v = load_words<DT, NT>(base, 240 * u + 4 * sub, 4, nelem, al4);
    return v;
  }
  __device__ static __forceinline__ u32x4 finish_load(u32x4 v, int sub) {
    // extra lane 60+i collects the last word of the flag lanes of quads 4i..4i+3
    const int i = (sub - 60) & 3;
    const uint32_t d0 = from_lane(16 * i + 3, v.w);
    const uint32_t d1 = from_lane(16 * i + 7, v.w);
    const uint32_t d2 = from_lane(16 * i + 11, v.w);
    const uint32_t d3 = from_lane((16 * i + 15) & 63, v.w);
    if (sub >= 60) {
      v.x = d0;
      v.y = d1;
      v.z = d2;
      v.w = i < 3 ? d3 : 0u;
    }
    return v;
  }
  // Called with the whole wave active (a unit is one wave).
  template <int DT, bool NT = true>
  __device__ static __forceinline__ u32x4 load(const char *base, int64_t u, int sub, int64_t nelem, bool al4) {
    return finish_load(load_raw<DT, NT>(base, u, sub, nelem, al4), sub);
  }
  // The first of the 4 payload words of unit u that a data lane loads; the
  // extra lanes load none.
  __device__ static __forceinline__ uint32_t first_word(uint32_t u, int sub) {
    return sub < 60 ? 240 * u + 4 * (uint32_t)sub : kNoWord;
  }
  // Payload word `wd` (0..239) of a unit: the lane and word slot that carry
  // it in packet order.
  __device__ static __forceinline__ void slot_of_word(int wd, int *lane, int *slot) {
    const int l = wd >> 2;
    if ((l & 3) == 3 && (wd & 3) == 3) {
      *lane = 60 + (l >> 4);
      *slot = (l >> 2) & 3;
    } else {
      *lane = l;
      *slot = wd & 3;
    }
  }
  // A data lane's 4 payload words in stream order, from w in packet order:
  // the flag lane of quad j takes its last word back from extra lane
  // 60 + j/4.  Called with the whole wave active.
  __device__ static __forceinline__ u32x4 start_store(u32x4 w, int sub) {
    const int j = (sub >> 2) & 15;
    const int src = 60 + (j >> 2);
    const uint32_t c0 = from_lane(src, w.x);
    const uint32_t c1 = from_lane(src, w.y);
    const uint32_t c2 = from_lane(src, w.z);
    const uint32_t c3 = from_lane(src, w.w);
    if ((sub & 3) == 3) {
      const int c = j & 3;
      w.w = c == 0 ? c0 : (c == 1 ? c1 : (c == 2 ? c2 : c3));
    }
    return w;
  }
  // Called with the whole wave active; w is in packet order.
  template <int DT>
  __device__ static __forceinline__ void store(char *base, int64_t u, int sub, int64_t nelem, bool al4, u32x4 w) {
    w = start_store(w, sub);
    if (sub < 60) store_words<DT>(base, 240 * u + 4 * sub, 4, nelem, al4, w);
  }
  __device__ static __forceinline__ u32x4 pack(u32x4 w, uint32_t epoch, int sub) {
    if ((sub & 3) == 3) w.w = epoch;
    return w;
  }
  // The flag of a quad sits in its lane 3; broadcast it to the quad with DPP.
  // All four lanes of a quad are always active together.
  __device__ static __forceinline__ bool ready(u32x4 p, uint32_t epoch) {
    uint32_t f = (uint32_t)__builtin_amdgcn_mov_dpp((int)p.w, 0xFF /* quad_perm:[3,3,3,3] */, 0xF, 0xF, false);
    return f == epoch;
  }
  __device__ static __forceinline__ u32x4 unpack(u32x4 p, int sub) {
    if ((sub & 3) == 3) p.w = 0u;
    return p;
  }
  static constexpr __host__ __device__ int64_t units(int64_t words) { return (words + 239) / 240; }
};

// Sentinel mode (Sec. IV, "Sentinel"): no flag at all.  A receive slot holds
// the sentinel 0xFFFFFFFF in every dword (a negative NaN as binary32, a pair
// of negative NaNs as bfloat16) until the sender's payload overwrites it; a
// lane moves 4 payload words per 16-byte store, so the full store bandwidth
// carries data.  The receiver resets every slot it has read back to the
// sentinel.  A payload dword that equals the sentinel can never be detected:
// such data is not supported (the wait times out).
struct ProtoSent {
  static constexpr int kLanes = 1;
  static constexpr int kUnitBytes = 16;
  static constexpr int kUnitWords = 4;
  static constexpr int kMaxWords = 4;
  static constexpr bool kReset = true;
  static constexpr uint32_t kSentinel = 0xFFFFFFFFu;
  template <int DT, bool NT = true>
  __device__ static __forceinline__ u32x4 load(const char *base, int64_t u, int /*sub*/, int64_t nelem, bool al4) {
    return load_words<DT, NT>(base, 4 * u, 4, nelem, al4);
  }
  template <int DT>
  __device__ static __forceinline__ void store(char *base, int64_t u, int /*sub*/, int64_t nelem, bool al4, u32x4 w) {
    store_words<DT>(base, 4 * u, 4, nelem, al4, w);
  }
  __device__ static __forceinline__ uint32_t first_word(uint32_t u, int /*sub*/) { return 4 * u; }
  __device__ static __forceinline__ u32x4 finish_load(u32x4 v, int /*sub*/) { return v; }
  __device__ static __forceinline__ u32x4 start_store(u32x4 w, int /*sub*/) { return w; }
  __device__ static __forceinline__ u32x4 pack(u32x4 w, uint32_t /*epoch*/, int /*sub*/) { return w; }
  __device__ static __forceinline__ bool ready(u32x4 p, uint32_t /*epoch*/) {
    return p.x != kSentinel && p.y != kSentinel && p.z != kSentinel && p.w != kSentinel;
  }
  __device__ static __forceinline__ u32x4 unpack(u32x4 p, int /*sub*/) { return p; }
  static constexpr __host__ __device__ int64_t units(int64_t words) { return (words + 3) / 4; }
};

// Whether a packet format resets the slots it has read.
template <class Pr> struct ResetsSlots { static constexpr bool value = false; };
template <> struct ResetsSlots<ProtoSent> { static constexpr bool value = true; };

}  // namespace llc
