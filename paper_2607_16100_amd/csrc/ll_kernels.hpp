// Collective kernels: one-shot and two-shot AllReduce, ReduceScatter and
// AllGather over P virtual ranks on one GPU.
//
// Grid = P * W workgroups.  Workgroup b serves rank r = b % P as its part
// w = b / P.  Workgroups are dispatched round-robin over the chip's XCDs, so
// with P = 8 every rank lives on its own XCD and every rank-to-rank hop
// crosses the fabric, the single-chip stand-in for a GPU-to-GPU link.
//
// Every rank moves its data to another rank only by storing flagged packets
// into a slot of that rank's slice ("push mode", Sec. III-A); it never reads
// another rank's input.  A slot (d <- s) is the region of rank d's slice that
// receives rank s's packets; slot number of s in d's list is s - (s > d).
//
// Work division: the lanes of all W workgroups of a rank cover the packet
// units of a stream in a grid-stride loop; lane g of part w handles the same
// unit indices on every rank, so a waiting lane only ever waits for the lanes
// of the same part on other ranks, which are resident (the host keeps the
// grid within what the chip holds at once).  Every wait is bounded.
#pragma once

#include "ll_device.hpp"
#include "ll_iter.hpp"

namespace llc {

struct KArgs {
  char *sym;          // symmetric region base
  uint64_t stride;    // bytes per rank slice
  char *out;          // dense per-rank outputs
  int64_t n;          // AllReduce: count; ReduceScatter: recvcount; AllGather: sendcount
  int64_t chunk;      // two-shot chunk length in elements
  uint64_t area;      // offset of the packet area used by this call, in every slice
  uint64_t slot;      // bytes per slot
  uint64_t timeout;   // flag-wait budget, 100 MHz ticks
  uint64_t *stamps;   // optional per-workgroup start/end times
  uint64_t *phases;   // optional per-workgroup phase times (diagnostics)
  uint32_t epoch;     // flag value of this call
  int32_t mute;       // rank that publishes nothing (test hook), or -1
  uint32_t al4;       // every element stream of this call starts 4-byte aligned
  uint16_t first_wait;  // idle time before the first poll, in units of 64 shader cycles
  uint16_t poll_gap;    // idle time between polls, in units of 64 shader cycles
  uint32_t lag;         // two-shot pipeline distance between publish, reduce and gather (>= 0)
  uint32_t in_al4;      // every rank's input starts 4-byte aligned
  uint32_t clear;       // flagged formats: the reader stores zeros back into every slot it has read
  const char *in;       // rank r's input at in + r * in_stride
  uint64_t in_stride;
  // Multi-iteration calls (bounded scratch, Sec. IV "Bidirectional
  // Communication & Double Buffering"): iteration i covers elements
  // [i * iter_n, (i+1) * iter_n) of every rank, uses sub-buffer i % 2 of the
  // area (sub_bytes apart) and the flag epoch + i.  One iteration: iters = 1,
  // iter_n = n.
  int64_t iter_n;
  uint64_t sub_bytes;
  uint32_t iters;
  int32_t root;         // Broadcast / Reduce root rank
  uint32_t grid;        // workgroups in the launch (gridDim.x, without its memory load)
  uint32_t block;       // threads per workgroup (blockDim.x, likewise)
  int64_t units;        // packet units of the call's stream (one-shot wave kernel)
  uint32_t *status;     // status word of the stream the call runs on (where a timed-out wait reports)
};

// Kernel arguments live in memory and reach a wave through scalar loads.  Left
// alone, the compiler loads the fields used inside a loop only after the loop
// test, a second round trip on the way to the first packet.  pin_args loads
// every field up front, in one batch.
template <class T>
__device__ __forceinline__ T in_sgpr(T v) {
  asm volatile("" : "+s"(v));
  return v;
}

__device__ __forceinline__ KArgs pin_args(const KArgs &k) {
  KArgs a;
  a.sym = in_sgpr(k.sym);
  a.stride = in_sgpr(k.stride);
  a.out = in_sgpr(k.out);
  a.n = in_sgpr(k.n);
  a.chunk = in_sgpr(k.chunk);
  a.area = in_sgpr(k.area);
  a.slot = in_sgpr(k.slot);
  a.timeout = in_sgpr(k.timeout);
  a.stamps = in_sgpr(k.stamps);
  a.phases = in_sgpr(k.phases);
  a.epoch = in_sgpr(k.epoch);
  a.mute = in_sgpr(k.mute);
  a.al4 = in_sgpr(k.al4);
  a.first_wait = (uint16_t)in_sgpr((uint32_t)k.first_wait);
  a.poll_gap = (uint16_t)in_sgpr((uint32_t)k.poll_gap);
  a.lag = in_sgpr(k.lag);
  a.in_al4 = in_sgpr(k.in_al4);
  a.clear = in_sgpr(k.clear);
  a.in = in_sgpr(k.in);
  a.in_stride = in_sgpr(k.in_stride);
  a.iter_n = in_sgpr(k.iter_n);
  a.sub_bytes = in_sgpr(k.sub_bytes);
  a.iters = in_sgpr(k.iters);
  a.root = in_sgpr(k.root);
  a.grid = in_sgpr(k.grid);
  a.block = in_sgpr(k.block);
  a.units = in_sgpr(k.units);
  a.status = in_sgpr(k.status);
  return a;
}

// Wait until every store this wave has issued is acknowledged.  Used between
// iterations in sentinel mode: a slot reset must be complete before the
// next iteration's packets, which let a peer refill that slot, go out.
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0f70); }  // vmcnt(0)

__device__ __forceinline__ int slot_of(int src, int dst) { return src - (src > dst ? 1 : 0); }

struct Part {
  int r, w, W;
};

template <int P>
__device__ __forceinline__ Part part_of_block(const KArgs &a) {
  Part p;
  p.r = (int)(blockIdx.x % P);
  p.w = (int)(blockIdx.x / P);
  p.W = (int)(a.grid / P);
  return p;
}

// Per-workgroup start and end times (diagnostics).  The start time is kept in
// a register and stored together with the end time: a store at kernel entry
// would delay the first load, since one memory counter covers both.
__device__ __forceinline__ uint64_t stamp_start(const KArgs &a) { return a.stamps != nullptr ? now_ticks() : 0; }

__device__ __forceinline__ void stamp_end(const KArgs &a, uint64_t t_start) {
  if (a.stamps != nullptr) {
    __syncthreads();
    if (threadIdx.x == 0) {
      a.stamps[blockIdx.x] = t_start;
      a.stamps[a.grid + blockIdx.x] = now_ticks();
    }
  }
}

// Poll the P-1 slots (r <- q) at byte offset `off` of every slot until every
// flag equals the epoch.  All pending loads of an iteration are issued before
// any is checked (parallel polling across ranks, Sec. VII Obs. 1); a lane
// re-loads only the peers it has not yet heard from.
__device__ __forceinline__ void idle64(int units) {
  for (int i = 0; i < units; ++i) __builtin_amdgcn_s_sleep(1);
}

template <class Pr, int P>
__device__ __forceinline__ int poll_all(char *area_r, uint64_t slot, uint32_t off, int r, uint32_t epoch,
                                         WaitBudget &budget, u32x4 *got, int first_wait = 0, int poll_gap = 0,
                                         uint32_t peers = 0xFFFFFFFFu) {
  // One resource covers the P-1 slots; the slot is selected by the scalar offset.
  const rsrc_t rs = make_rsrc(area_r, (uint32_t)((uint64_t)(P - 1) * slot));
  const uint32_t want = ((1u << P) - 1u) & ~(1u << r) & peers;
  uint32_t pend = want;
#pragma unroll
  for (int q = 0; q < P; ++q) got[q] = u32x4{0u, 0u, 0u, 0u};
  int spins = 1;
  idle64(first_wait);
  while (true) {
    compiler_fence();
#pragma unroll
    for (int q = 0; q < P; ++q) {
      if (q == r) continue;
      if (pend & (1u << q)) got[q] = ld_pkt(rs, off, uniform_u32((uint32_t)((uint64_t)slot_of(q, r) * slot)));
    }
#pragma unroll
    for (int q = 0; q < P; ++q) {
      if (q == r) continue;
      const bool rdy = Pr::ready(got[q], epoch);
      if ((pend & (1u << q)) && rdy) pend &= ~(1u << q);
    }
    if (pend == 0) break;
    idle64(poll_gap);
    if ((spins++ & 15) == 0 && budget.expired()) {
      budget.report(r, pend, epoch);
      break;
    }
  }
  if (ResetsSlots<Pr>::value) {
    // sentinel mode: give every slot read back to its next sender
    const u32x4 sent = {ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel};
#pragma unroll
    for (int q = 0; q < P; ++q) {
      if (!(want & (1u << q))) continue;
      st_pkt_at(rs, off, uniform_u32((uint32_t)((uint64_t)slot_of(q, r) * slot)), sent);
    }
  }
  return spins;
}

// Store one packet to slot (q <- r) of every peer q, starting with r+1 so
// that the ranks do not all write to the same peer at once.  Every address
// is computed from wave-uniform values.
template <int P>
__device__ __forceinline__ void bcast(const KArgs &a, uint64_t area, int r, uint32_t off, u32x4 pk) {
#pragma unroll
  for (int k = 1; k < P; ++k) {
    const int q = (r + k) % P;
    char *dst = a.sym + (uint64_t)q * a.stride + area + (uint64_t)slot_of(r, q) * a.slot;
    st_pkt(make_rsrc(dst, (uint32_t)a.slot), off, pk);
  }
}

// Reduce one lane's words: x_0 + x_1 + ... + x_{P-1} in ascending rank order,
// binary32 accumulation starting from x_0, own contribution at position r,
// one rounding to the element type (Sec. IV error analysis; recvReduce,
// Sec. V).  `got[q]` are unpacked payload words for q != r.
template <class Pr, int DT, int P>
__device__ __forceinline__ u32x4 reduce_ordered(const u32x4 *got, u32x4 own, int r) {
  constexpr int K = Elem<DT>::kPerWord;
  constexpr int NW = Pr::kMaxWords;
  float acc[NW * K];
#pragma unroll
  for (int q = 0; q < P; ++q) {
    const u32x4 x = (q == r) ? own : got[q];
    const uint32_t wv[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float f[K];
      Elem<DT>::widen(wv[j], f);
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (q == 0) {
          acc[j * K + k] = f[k];
        } else {
          acc[j * K + k] = acc[j * K + k] + f[k];
        }
      }
    }
  }
  uint32_t res[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int j = 0; j < NW; ++j) res[j] = Elem<DT>::narrow(&acc[j * K]);
  u32x4 v = {res[0], res[1], res[2], res[3]};
  return v;
}

// ---------------------------------------------------------------------------
// One-shot AllReduce (Sec. III-A; the per-thread load -> bcast -> recvReduce
// -> store sequence of Sec. V).  Slot (d <- s) holds all of s's input.
// Phase stamps of the one-lane one-shot are compiled in only on request
// (-DLLCOLL_ONESHOT_PHASES=1), like those of the wave kernel.
#ifndef LLCOLL_ONESHOT_PHASES
#define LLCOLL_ONESHOT_PHASES 0
#endif

template <class Pr, int DT, int P>
__global__ __launch_bounds__(1024) void k_oneshot(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;  // past every slot: the buffer resource discards the store
  const uint32_t r = blockIdx.x % P, w = blockIdx.x / P;
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const bool in_al4 = a.in_al4 != 0;
  // unit indices fit 32 bits: a call's P-1 slots span less than 4 GiB
  const uint32_t g = w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const uint32_t ustep = (a.grid / P) * a.block / Pr::kLanes;
  // A muted rank (test hook) stores at an offset past the slots, which the
  // buffer resource discards: no store is branched around, so the compiler
  // never has to wait for the stores' acknowledgements before the polls.
  const bool publish = (int)r != a.mute;
  WaitBudget budget(a.timeout, a.status);
  char *const slice_r = a.sym + (uint64_t)r * a.stride;
  char *const out_r = a.out + (uint64_t)r * (uint64_t)a.n * E;

  for (uint32_t it = 0; it < a.iters; ++it) {
    const IterSpan sp = iter_span(a.n, a.iter_n, it, P, E);
    const int64_t e0 = sp.e0, n = sp.n;
    const uint32_t units = (uint32_t)Pr::units((n * E + 3) / 4);
    const uint64_t area = a.area + (uint64_t)(it & 1u) * a.sub_bytes;
    const uint32_t epoch = a.epoch + it;
    char *const area_r = slice_r + area;
    const char *const in_i = in_r + e0 * E;
    char *const out_i = out_r + e0 * E;
    for (uint32_t u = g / Pr::kLanes; u < units; u += ustep) {
      const uint32_t off = u * Pr::kUnitBytes + sub * 16;
      const u32x4 own = Pr::template load<DT>(in_i, u, sub, n, in_al4);
      uint64_t t_loaded = 0, t_acked = 0;
      if (LLCOLL_ONESHOT_PHASES && a.phases != nullptr) t_loaded = now_ticks() + (own.x & 0u);
      bcast<P>(a, area, (int)r, publish ? off : kNowhere, Pr::pack(own, epoch, sub));
      if (LLCOLL_ONESHOT_PHASES && a.phases != nullptr) {
        __asm__ __volatile__("s_waitcnt vmcnt(0)" ::: "memory");
        t_acked = now_ticks();
      }
      u32x4 got[P];
      const int spins = poll_all<Pr, P>(area_r, a.slot, off, (int)r, epoch, budget, got, a.first_wait, a.poll_gap);
      if (LLCOLL_ONESHOT_PHASES && a.phases != nullptr && threadIdx.x == 0) {
        const uint64_t t_polled = now_ticks() + (got[(r + 1) % P].x & 0u);
        a.phases[4 * blockIdx.x + 0] = t_loaded;
        a.phases[4 * blockIdx.x + 1] = t_acked;
        a.phases[4 * blockIdx.x + 2] = t_polled;
        a.phases[4 * blockIdx.x + 3] = (uint64_t)spins;
      }
#pragma unroll
      for (int q = 0; q < P; ++q) got[q] = Pr::unpack(got[q], sub);
      const u32x4 res = reduce_ordered<Pr, DT, P>(got, own, (int)r);
      Pr::template store<DT>(out_i, u, sub, n, a.al4 != 0, res);
    }
    if (ResetsSlots<Pr>::value && it + 1 < a.iters) wait_vm_all();
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// One-shot AllReduce, one wave per peer, with LDS staging (8-byte packets,
// sentinel units or 128-byte lines).
//
// A workgroup has P waves and handles tiles of 64*U packet units (lane l owns
// units l, l+64, ..., l+64(U-1) of the tile, so every memory instruction of a
// wave covers 64 units; with lines a tile is U line units, each a whole
// wave).  For a tile, wave q != r sends the rank's units to
// peer q only and then polls only the units peer q sent to this rank; wave r
// keeps the rank's own values.  Each wave stages its rank's values, widened
// to binary32, in LDS row q; after a workgroup barrier the rows are summed in
// ascending rank order and rounded once.  Compared with one lane talking to
// all P-1 peers, a wave's poll never waits for more than its own U stores
// (the memory counter covers stores and loads alike on this chip) and a poll
// is U loads, not U*(P-1).
// Workgroup barrier that makes LDS writes visible but does not wait for the
// wave's outstanding global stores (packet stores need not be acknowledged
// before the workgroup goes on).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0); vmcnt and expcnt left alone
  __builtin_amdgcn_s_barrier();
}

// Unit addressing of the wave-per-peer kernels.  A tile is 64*U units of a
// one-lane format (lane l owns units l, l+64, ...) or U units of the 64-lane
// line format (the whole wave owns each unit; lane l is its part `sub`).
// Either way a lane holds kMaxWords payload words per unit slot k.
template <class Pr, int U>
struct WaveUnits {
  static constexpr bool kWave = Pr::kLanes == 64;
  static constexpr int64_t kPerTile = kWave ? U : 64 * U;
  __device__ static __forceinline__ int64_t unit(int64_t tile, int k, int lane) {
    return kWave ? tile * U + k : tile * 64 * U + k * 64 + lane;
  }
  __device__ static __forceinline__ int sub(int lane) { return kWave ? lane : 0; }
  __device__ static __forceinline__ uint32_t off(int64_t u, int lane) {
    return (uint32_t)(u * Pr::kUnitBytes + sub(lane) * 16);
  }
};

// Phase stamps of the wave-per-peer one-shot are compiled in only on request
// (-DLLCOLL_WAVE_PHASES=1): every instruction on the way from kernel entry to
// the output store adds to the call's latency.
#ifndef LLCOLL_WAVE_PHASES
#define LLCOLL_WAVE_PHASES 0
#endif

template <class Pr, int DT, int P, int U>
__global__ __launch_bounds__(512) void k_oneshot_waves(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  using WU = WaveUnits<Pr, U>;
  constexpr int WPU = Pr::kMaxWords;  // payload words per lane and unit slot
  constexpr int EPU = WPU * K;        // elements per lane and unit slot
  constexpr int TW = 64 * U * WPU;    // payload words per tile
  constexpr uint32_t kTileShift = WU::kPerTile == 1 ? 0 : (WU::kPerTile == 2 ? 1 : (WU::kPerTile == 4 ? 2 :
                                  (WU::kPerTile == 64 ? 6 : (WU::kPerTile == 128 ? 7 : 8))));
  static_assert((1 << kTileShift) == WU::kPerTile, "tiles hold a power-of-two number of units");
  __shared__ float stage[P][TW * K];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const int wv = (int)uniform_u32(threadIdx.x >> 6);  // the same in every lane of a wave
  const int lane = (int)(threadIdx.x & 63);
  const int sub = WU::sub(lane);
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const int64_t n = a.n;
  // unit and tile indices fit 32 bits: a call's P-1 slots span less than 4 GiB
  const uint32_t units = (uint32_t)a.units;
  const bool in_al4 = a.in_al4 != 0;

  // The input of a tile, loaded by every wave of the workgroup.  The first
  // tile's load is issued before the rest of the set-up below, which would
  // otherwise stand between kernel entry and the first packet store (a wave
  // issues at most one instruction every few cycles, and a workgroup's waves
  // share the scalar unit).  The host launches no more workgroups per rank
  // than there are tiles; a workgroup past the last tile (a forced launch
  // shape) loads and stores nothing, since every access is guarded by the
  // unit count.
  // For lines the load comes in two halves (memory, then lane permutes that
  // wait for it); the store set-up below goes between them, while the load
  // is in flight.
  auto load_tile = [&](uint32_t tile, u32x4 *own) {
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
      if constexpr (WU::kWave) {
        own[k] = u < units ? Pr::template load_raw<DT, false>(in_r, u, sub, n, in_al4) : u32x4{0u, 0u, 0u, 0u};
      } else {
        own[k] = u < units ? Pr::template load<DT, false>(in_r, u, sub, n, in_al4) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto finish_tile = [&](u32x4 *own) {
    if constexpr (WU::kWave) {
#pragma unroll
      for (int k = 0; k < U; ++k) own[k] = Pr::finish_load(own[k], sub);
    }
  };
  uint32_t tile = w;
  u32x4 own[U];
  load_tile(tile, own);

  // Then the tile's packet stores, again ahead of the set-up the polls and
  // the reduction need.  Every wave stores (the own-rank wave and, for a muted
  // rank, every wave, at an offset past the slot, which the buffer resource
  // discards), and no store is branched around: a branch would leave the
  // input load pending on one path, and the compiler would then wait for
  // every outstanding memory operation, this store's acknowledgement
  // included, before the first poll.
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;
  const uint32_t q = (uint32_t)wv;  // the peer this wave talks to (q == r: the own values)
  const uint32_t slot = (uint32_t)a.slot;
  const bool publish = (int)r != a.mute && q != r;
  const rsrc_t rd = make_rsrc(a.sym + a.area + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot, slot);
  auto store_tile = [&](uint32_t tile, const u32x4 *own) {
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
      st_pkt(rd, u < units && publish ? WU::off(u, lane) : kNowhere, Pr::pack(own[k], a.epoch, sub));
    }
  };
  finish_tile(own);
  store_tile(tile, own);

  const uint32_t W = a.grid / P;
  const uint32_t tiles = (units + (uint32_t)WU::kPerTile - 1u) >> kTileShift;

  WaitBudget budget(a.timeout, a.status);
  char *const out_r = a.out + (uint64_t)r * (uint64_t)n * E;
  const rsrc_t rs = make_rsrc(a.sym + a.area + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot, slot);

  // Stage a wave's U units (payload words) in its LDS row, widened to binary32.
  auto stage_row = [&](const u32x4 *v) {
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint32_t wv4[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
      for (int j = 0; j < WPU; ++j) {
        float f[K];
        Elem<DT>::widen(wv4[j], f);
#pragma unroll
        for (int e = 0; e < K; ++e) stage[q][(k * 64 + lane) * EPU + j * K + e] = f[e];
      }
    }
  };
// Diagnostics: the time of phase k of the first tile, for lane 0 of each wave.
#define LL_WAVE_PHASE(k, expr)                                              \
  do {                                                                      \
    if (LLCOLL_WAVE_PHASES && a.phases != nullptr && lane == 0 && tile == w) \
      a.phases[4 * (blockIdx.x * P + wv) + (k)] = (expr);                   \
  } while (0)

  // Poll the tile's units in slot (r <- q) until the wave has them all; the
  // loop runs while any lane of the wave still waits (a wave vote ends it),
  // and every round re-loads all U units: the few extra loads of lanes
  // already done cost less than per-lane branching, which would add
  // instructions to every round.  Sentinel units are given back once read.
  auto poll_tile = [&](uint32_t tile, u32x4 *v) {
    uint32_t pend = 0;
#pragma unroll
    for (int k = 0; k < U; ++k) {
      v[k] = u32x4{0u, 0u, 0u, 0u};
      pend |= ((uint32_t)WU::unit(tile, k, lane) < units ? 1u : 0u) << k;
    }
    const uint32_t want = pend;
    idle64(a.first_wait);
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      u32x4 pk[U];
#pragma unroll
      for (int k = 0; k < U; ++k) pk[k] = ld_pkt(rs, WU::off(WU::unit(tile, k, lane), lane));
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if ((pend & (1u << k)) && Pr::ready(pk[k], a.epoch)) {
          v[k] = Pr::unpack(pk[k], sub);
          pend &= ~(1u << k);
        }
      }
      if (__builtin_amdgcn_ballot_w64(pend != 0) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend != 0) budget.report((int)r, 1u << q, a.epoch);
        break;
      }
      idle64(a.poll_gap);
    }
    if (ResetsSlots<Pr>::value || a.clear != 0) {
      const uint32_t fill = ResetsSlots<Pr>::value ? ProtoSent::kSentinel : 0u;
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if (want & (1u << k)) st_pkt(rs, WU::off(WU::unit(tile, k, lane), lane), u32x4{fill, fill, fill, fill});
      }
    }
  };

  while (true) {
    LL_WAVE_PHASE(0, now_ticks() + (own[0].x & 0u));
    if (q == r) {
      stage_row(own);
      LL_WAVE_PHASE(1, now_ticks());
    } else {
      u32x4 v[U];
      poll_tile(tile, v);
      LL_WAVE_PHASE(1, now_ticks() + (v[0].x & 0u));
      stage_row(v);
    }
    lds_barrier();
    LL_WAVE_PHASE(2, now_ticks());
    if constexpr (WU::kWave && 64 * P >= 240 * U) {
      // line units are staged in packet order; with a thread per payload
      // word of the tile (U units of 240 words), thread t forms word t from
      // the lane and slot that carry it and stores it
      const int t = (int)threadIdx.x;
      if (t < 240 * U) {
        const int k = t / 240;
        const int wd = t - 240 * k;
        int sl, sj;
        Pr::slot_of_word(wd, &sl, &sj);
        const int at = (k * 64 + sl) * EPU + sj * K;
        float acc[K];
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = stage[0][at + e];
#pragma unroll
        for (int p = 1; p < P; ++p) {
#pragma unroll
          for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][at + e];
        }
        const u32x4 res = {Elem<DT>::narrow(acc), 0u, 0u, 0u};
        store_words<DT>(out_r, (int64_t)WU::unit(tile, k, 0) * 240 + wd, 1, n, a.al4 != 0, res);
      }
    } else if constexpr (WU::kWave) {
      // fewer threads than words: the own-rank wave sums its lanes' words in
      // packet order and stores whole units (the store puts displaced words
      // back)
      if (q == r) {
#pragma unroll
        for (int k = 0; k < U; ++k) {
          uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int j = 0; j < WPU; ++j) {
            float acc[K];
#pragma unroll
            for (int e = 0; e < K; ++e) acc[e] = stage[0][(k * 64 + lane) * EPU + j * K + e];
#pragma unroll
            for (int p = 1; p < P; ++p) {
#pragma unroll
              for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][(k * 64 + lane) * EPU + j * K + e];
            }
            o[j] = Elem<DT>::narrow(acc);
          }
          Pr::template store<DT>(out_r, WU::unit(tile, k, lane), sub, n, a.al4 != 0, u32x4{o[0], o[1], o[2], o[3]});
        }
      }
    } else {
      for (int j = (int)threadIdx.x; j < TW; j += (int)a.block) {
        float acc[K];
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = stage[0][j * K + e];
#pragma unroll
        for (int p = 1; p < P; ++p) {
#pragma unroll
          for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][j * K + e];
        }
        const u32x4 res = {Elem<DT>::narrow(acc), 0u, 0u, 0u};
        store_words<DT>(out_r, (int64_t)tile * TW + j, 1, n, a.al4 != 0, res);
      }
    }
    tile += W;
    if (tile >= tiles) break;
    lds_barrier();  // the next tile overwrites the staging rows
    load_tile(tile, own);
    finish_tile(own);
    store_tile(tile, own);
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// One-shot AllReduce for the latency-bound sizes: one wave per peer, one tile
// per workgroup, one-lane packet formats (8-byte packets or sentinel units),
// every stream 4-byte aligned.  The same exchange as k_oneshot_waves with
// U = 1, written as one short straight path: on this chip the code a kernel
// runs between its start and its last store is paid for in latency (every
// call starts with cold instruction caches), so this kernel carries no
// multi-tile loop and no element-wise fallback for unaligned streams.
//
// Wave q of the workgroup serving rank r and tile w: lane l owns unit
// u = 64w + l.  It loads the unit's input words through a buffer resource
// (words past the input read as zero), stores them as one packet to slot
// (q <- r) of peer q (the own-rank wave and a muted rank store at an offset
// past the slot, which the resource discards: no branch around the store),
// polls slot (r <- q) until the peer's packet carries the epoch, and stages
// the payload, widened to binary32, in LDS row q.  After one barrier wave 0
// forms the ordered sum of the P rows for its 64 lanes, rounds once and
// stores the tile's output, 4*kMaxWords bytes per lane.
template <class Pr, int DT, int P>
__global__ __launch_bounds__(512) void k_oneshot_tile(KArgs ka) {
  static_assert(Pr::kLanes == 1, "one-lane packet formats only");
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  constexpr int NW = Pr::kMaxWords;  // payload words per lane
  constexpr int EPL = NW * K;        // elements per lane
  __shared__ float stage[P][64 * EPL];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t u = w * 64 + lane;
  const uint32_t nb = (uint32_t)(a.n * E);  // input bytes per rank (< 256 MiB)
  const rsrc_t in_rs = make_rsrc(a.in + (uint64_t)r * a.in_stride, (nb + 3u) & ~3u);
  u32x4 x = load_words_rs<NW>(in_rs, u * NW);
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;
  const uint32_t slot = (uint32_t)a.slot;
  const bool publish = q != r && u < (uint32_t)a.units && (int)r != a.mute;
  const rsrc_t rd = make_rsrc(a.sym + a.area + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot, slot);
  if (ResetsSlots<Pr>::value) x = clear_tail<DT, NW>(x, u * NW, (uint32_t)a.n);
  st_pkt(rd, publish ? u * 16 : kNowhere, Pr::pack(x, a.epoch, 0));
  // diagnostics (-DLLCOLL_WAVE_PHASES=1): as in k_oneshot_waves
  const int wv = (int)q;
  const uint32_t tile = w;
  LL_WAVE_PHASE(0, now_ticks() + (x.x & 0u));
  WaitBudget budget(a.timeout, a.status);
  u32x4 v = x;
  if (q != r) {
    const rsrc_t rs = make_rsrc(a.sym + a.area + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot, slot);
    bool pend = u < (uint32_t)a.units;
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      const u32x4 pk = ld_pkt(rs, u * 16);
      if (pend && Pr::ready(pk, a.epoch)) {
        v = Pr::unpack(pk, 0);
        pend = false;
      }
      if (__builtin_amdgcn_ballot_w64(pend) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend) budget.report((int)r, 1u << q, a.epoch);
        break;
      }
    }
    if (ResetsSlots<Pr>::value) {
      const u32x4 sent = {ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel};
      if (u < (uint32_t)a.units) st_pkt(rs, u * 16, sent);
    } else if (a.clear != 0) {
      if (u < (uint32_t)a.units) st_pkt(rs, u * 16, u32x4{0u, 0u, 0u, 0u});
    }
  }
  LL_WAVE_PHASE(1, now_ticks() + (v.x & 0u));
  {
    const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float f[K];
      Elem<DT>::widen(vw[j], f);
#pragma unroll
      for (int e = 0; e < K; ++e) stage[q][lane * EPL + j * K + e] = f[e];
    }
  }
  lds_barrier();
  LL_WAVE_PHASE(2, now_ticks());
  if (q == 0) {
    uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      float acc[K];
#pragma unroll
      for (int e = 0; e < K; ++e) acc[e] = stage[0][lane * EPL + j * K + e];
#pragma unroll
      for (int p = 1; p < P; ++p) {
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][lane * EPL + j * K + e];
      }
      o[j] = Elem<DT>::narrow(acc);
    }
    // al4: nb is a whole number of words, so no stored word is partly past the end;
    // plain stores (the outputs of tiny calls share cache lines across ranks)
    store_words_rs<NW, false>(make_rsrc(a.out + (uint64_t)r * nb, nb), u * NW, u32x4{o[0], o[1], o[2], o[3]});
  }
  stamp_end(a, t_start);
}

// One-shot AllReduce with 128-byte line packets, one wave per peer and one
// line unit per workgroup, every stream 4-byte aligned: the straight-line
// counterpart of k_oneshot_waves<ProtoLine, DT, P, 1> for calls whose units
// are all resident at once, with no multi-tile loop and no element-wise
// fallback for unaligned streams (as for k_oneshot_tile, the instructions a
// call runs are paid for in latency).
//
// Workgroup (r, w) serves rank r and line unit w (payload words 240w ..
// 240w + 239 of every input).  Wave q loads the unit (the data lanes 4
// words each, the extra lanes the displaced words after the load), stores it
// as one unit of line packets to slot (q <- r) of peer q (the own-rank wave
// and a muted rank at an offset the resource discards), polls slot (r <- q)
// until both flags of every 128-byte line carry the epoch, and stages the
// payload in packet order, widened to binary32, in LDS row q.  After one
// barrier the ordered sum over the P rows is formed and rounded once: from 4
// ranks up, thread t < 240 takes payload word t from the lane and slot that
// carry it and stores it (4 bytes); with fewer threads than words the
// own-rank wave sums its lanes' words, moves the displaced words back (each
// flag lane takes its last word from an extra lane) and stores 16 bytes per
// data lane.
template <int DT, int P>
__global__ __launch_bounds__(512) void k_oneshot_line_tile(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  constexpr int EPL = 4 * K;  // elements per lane
  __shared__ float stage[P][64 * EPL];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);
  const int lane = (int)(threadIdx.x & 63);
  const uint32_t nb = (uint32_t)(a.n * E);  // input bytes per rank (< 256 MiB)
  const uint32_t w0 = ProtoLine::first_word(w, lane);
  const rsrc_t in_rs = make_rsrc(a.in + (uint64_t)r * a.in_stride, nb);
  u32x4 x = load_words_rs<4>(in_rs, w0);
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;
  const uint32_t slot = (uint32_t)a.slot;
  const uint32_t off = w * 1024u + (uint32_t)lane * 16u;
  const bool publish = q != r && w < (uint32_t)a.units && (int)r != a.mute;
  const rsrc_t rd = make_rsrc(a.sym + a.area + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot, slot);
  x = ProtoLine::finish_load(x, lane);
  st_pkt(rd, publish ? off : kNowhere, ProtoLine::pack(x, a.epoch, lane));
  const int wv = (int)q;  // diagnostics, as in k_oneshot_waves
  const uint32_t tile = w;
  LL_WAVE_PHASE(0, now_ticks() + (x.x & 0u));
  WaitBudget budget(a.timeout, a.status);
  u32x4 v = x;
  if (q != r) {
    const rsrc_t rs = make_rsrc(a.sym + a.area + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot, slot);
    bool pend = w < (uint32_t)a.units;
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      const u32x4 pk = ld_pkt(rs, off);
      // every lane of the wave runs the readiness check: it reads its quad's
      // flag lane
      const bool ready = ProtoLine::ready(pk, a.epoch);
      if (pend && ready) {
        v = ProtoLine::unpack(pk, lane);
        pend = false;
      }
      if (__builtin_amdgcn_ballot_w64(pend) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend) budget.report((int)r, 1u << q, a.epoch);
        break;
      }
    }
    if (a.clear != 0 && w < (uint32_t)a.units) st_pkt(rs, off, u32x4{0u, 0u, 0u, 0u});
  }
  LL_WAVE_PHASE(1, now_ticks() + (v.x & 0u));
  {
    const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float f[K];
      Elem<DT>::widen(vw[j], f);
#pragma unroll
      for (int e = 0; e < K; ++e) stage[q][lane * EPL + j * K + e] = f[e];
    }
  }
  lds_barrier();
  LL_WAVE_PHASE(2, now_ticks());
  if constexpr (64 * P >= 240) {
    const int t = (int)threadIdx.x;
    if (t < 240) {
      int sl, sj;
      ProtoLine::slot_of_word(t, &sl, &sj);
      const int at = sl * EPL + sj * K;
      float acc[K];
#pragma unroll
      for (int e = 0; e < K; ++e) acc[e] = stage[0][at + e];
#pragma unroll
      for (int p = 1; p < P; ++p) {
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][at + e];
      }
      // plain stores, as in k_oneshot_tile; a word past the end is discarded
      __builtin_amdgcn_raw_buffer_store_b32(Elem<DT>::narrow(acc), make_rsrc(a.out + (uint64_t)r * nb, nb),
                                            (int)((240u * w + (uint32_t)t) * 4u), 0, 0);
    }
  } else if (q == r) {
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float acc[K];
#pragma unroll
      for (int e = 0; e < K; ++e) acc[e] = stage[0][lane * EPL + j * K + e];
#pragma unroll
      for (int p = 1; p < P; ++p) {
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][lane * EPL + j * K + e];
      }
      o[j] = Elem<DT>::narrow(acc);
    }
    // plain stores, as in k_oneshot_tile; the extra lanes store nothing
    const u32x4 ow = ProtoLine::start_store(u32x4{o[0], o[1], o[2], o[3]}, lane);
    store_words_rs<4, false>(make_rsrc(a.out + (uint64_t)r * nb, nb), w0, ow);
  }
  stamp_end(a, t_start);
}
#undef LL_WAVE_PHASE

// ---------------------------------------------------------------------------
// Two-shot AllReduce (Sec. III-A): ReduceScatter then AllGather, fused in one
// kernel.  The input is cut into P chunks of `chunk` elements (the last ones
// may be short or empty); rank c owns chunk c.  For a packet unit u (the same
// offset in every chunk) a lane runs three steps:
//   publish  send unit u of chunk c to slot (c <- r) of its owner, c != r
//   reduce   reduce unit u of the own chunk r from the P-1 received copies
//            and the own input, store it, and send it to slot (q <- r) of
//            every peer's AllGather area
//   gather   receive unit u of every other reduced chunk and store it
// The steps of successive units are software-pipelined: at step s a lane
// publishes unit s, reduces unit s - lag and gathers unit s - 2*lag, so a
// packet is read back soon after it was written (while it is still in the
// memory-side cache) and the wait for peers overlaps the next unit's work.
// Every wait is for an earlier step of the same lane on another rank, so the
// pipeline cannot deadlock.  RS slots occupy the first P-1 slots of the
// area, AG slots the next P-1.
//
// Direct (sentinel mode only): the AllGather skips scratch.  The owner of
// chunk c stores its reduced units straight into block c of every peer's
// output, which the caller has filled with the sentinel beforehand, and each
// rank polls its own output until the peers' blocks no longer hold it
// (Sec. IV: sentinel-initialised output; Table I: scratch D instead of 2D).
// Every unit of a chunk is a full 16 bytes (the caller guarantees
// n * esize % 16 == 0), so units past a short last chunk are simply skipped.
template <int P>
__device__ __forceinline__ void poll_out(char *out_r, uint32_t out_bytes, uint32_t chunk_bytes, uint32_t off,
                                         uint32_t pend, int r, uint32_t epoch, WaitBudget &budget) {
  const rsrc_t rs = make_rsrc(out_r, out_bytes);
  int spins = 1;
  while (pend != 0) {
    compiler_fence();
    u32x4 got[P];
#pragma unroll
    for (int q = 0; q < P; ++q) {
      got[q] = u32x4{0u, 0u, 0u, 0u};
      if (pend & (1u << q)) got[q] = ld_pkt(rs, off, uniform_u32((uint32_t)q * chunk_bytes));
    }
#pragma unroll
    for (int q = 0; q < P; ++q) {
      if ((pend & (1u << q)) && ProtoSent::ready(got[q], epoch)) pend &= ~(1u << q);
    }
    if (pend == 0) break;
    if ((spins++ & 15) == 0 && budget.expired()) {
      budget.report(r, pend, epoch);
      break;
    }
  }
}

template <class Pr, int DT, int P, bool Direct = false>
struct TwoShot {
  static constexpr int E = Elem<DT>::kBytes;
  const KArgs &a;
  int r;
  char *slice_r;
  // the current iteration: its input and output (rank r), its elements, its
  // chunk length, its RS and AG slot offsets and its flag
  const char *in_r;
  char *out_r;
  uint64_t out_off;  // byte offset of the iteration within every rank's output
  int64_t n, C;
  uint64_t rs_area, ag_area;
  uint32_t epoch;
  mutable WaitBudget budget;
  bool publish, al4, in_al4;

  __device__ __forceinline__ int64_t chunk_len(int c) const {
    const int64_t left = n - (int64_t)c * C;
    return left < 0 ? 0 : (left < C ? left : C);
  }

  __device__ __forceinline__ void step_publish(int64_t u, int sub) const {
    const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
    u32x4 v[P];
#pragma unroll
    for (int k = 1; k < P; ++k) {
      const int c = (r + k) % P;
      v[k] = Pr::template load<DT>(in_r + c * C * E, u, sub, chunk_len(c), in_al4);
    }
#pragma unroll
    for (int k = 1; k < P; ++k) {
      const int c = (r + k) % P;
      char *dst = a.sym + (uint64_t)c * a.stride + rs_area + (uint64_t)slot_of(r, c) * a.slot;
      st_pkt(make_rsrc(dst, (uint32_t)a.slot), off, Pr::pack(v[k], epoch, sub));
    }
  }

  __device__ __forceinline__ void step_reduce(int64_t u, int sub) const {
    const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
    const int64_t nr = chunk_len(r);
    const u32x4 own = Pr::template load<DT>(in_r + r * C * E, u, sub, nr, in_al4);
    u32x4 got[P];
    poll_all<Pr, P>(slice_r + rs_area, a.slot, off, r, epoch, budget, got);
#pragma unroll
    for (int q = 0; q < P; ++q) got[q] = Pr::unpack(got[q], sub);
    const u32x4 res = reduce_ordered<Pr, DT, P>(got, own, r);
    Pr::template store<DT>(out_r + r * C * E, u, sub, nr, al4, res);
    if (!publish) return;
    if constexpr (Direct) {
      if ((int64_t)off >= nr * E) return;  // past a short last chunk
      const uint32_t at = uniform_u32((uint32_t)(r * C * E));
#pragma unroll
      for (int k = 1; k < P; ++k) {
        const int q = (r + k) % P;
        char *out_q = a.out + (uint64_t)q * (uint64_t)a.n * E + out_off;
        st_pkt_at(make_rsrc(out_q, (uint32_t)(n * E)), off, at, res);
      }
    } else {
      bcast<P>(a, ag_area, r, off, Pr::pack(res, epoch, sub));
    }
  }

  __device__ __forceinline__ void step_gather(int64_t u, int sub) const {
    const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
    if constexpr (Direct) {
      uint32_t pend = 0;
#pragma unroll
      for (int q = 0; q < P; ++q)
        if (q != r && (int64_t)off < chunk_len(q) * E) pend |= 1u << q;
      poll_out<P>(out_r, (uint32_t)(n * E), (uint32_t)(C * E), off, pend, r, epoch, budget);
      return;
    }
    u32x4 got[P];
    poll_all<Pr, P>(slice_r + ag_area, a.slot, off, r, epoch, budget, got);
#pragma unroll
    for (int q = 0; q < P; ++q) {
      if (q == r) continue;
      Pr::template store<DT>(out_r + q * C * E, u, sub, chunk_len(q), al4, Pr::unpack(got[q], sub));
    }
  }
};

#ifndef LLCOLL_TWOSHOT_WAVES_PER_EU
#define LLCOLL_TWOSHOT_WAVES_PER_EU 1
#endif

template <class Pr, int DT, int P, bool Direct = false>
__global__ __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(LLCOLL_TWOSHOT_WAVES_PER_EU))) void k_twoshot(
    KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  const Part pt = part_of_block<P>(a);
  TwoShot<Pr, DT, P, Direct> t{a};
  t.r = pt.r;
  constexpr int E = Elem<DT>::kBytes;
  t.budget = WaitBudget(a.timeout, a.status);
  t.slice_r = a.sym + (uint64_t)t.r * a.stride;
  t.publish = (t.r != a.mute);
  t.al4 = a.al4 != 0;
  t.in_al4 = a.in_al4 != 0;
  const char *const in_r = a.in + (uint64_t)t.r * a.in_stride;
  char *const out_r = a.out + (uint64_t)t.r * (uint64_t)a.n * E;
  const int64_t g = (int64_t)pt.w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const int64_t u0 = g / Pr::kLanes;
  const int64_t ustep = (int64_t)pt.W * a.block / Pr::kLanes;
  const int64_t lag = a.lag;
  for (uint32_t it = 0; it < a.iters; ++it) {
    const IterSpan sp = iter_span(a.n, a.iter_n, it, P, E);
    const int64_t e0 = sp.e0;
    t.n = sp.n;
    t.C = a.iters == 1 ? a.chunk : sp.chunk;
    t.in_r = in_r + e0 * E;
    t.out_off = (uint64_t)e0 * E;
    t.out_r = out_r + t.out_off;
    t.rs_area = a.area + (uint64_t)(it & 1u) * a.sub_bytes;
    t.ag_area = t.rs_area + (uint64_t)(P - 1) * a.slot;
    t.epoch = a.epoch + it;
    const int64_t units = Pr::units((t.C * E + 3) / 4);
    const int64_t steps = u0 < units ? (units - u0 + ustep - 1) / ustep : 0;
    for (int64_t s = 0; s < steps + 2 * lag; ++s) {
      if (s < steps && t.publish) t.step_publish(u0 + s * ustep, sub);
      if (s >= lag && s - lag < steps) t.step_reduce(u0 + (s - lag) * ustep, sub);
      if (s >= 2 * lag && s - 2 * lag < steps) t.step_gather(u0 + (s - 2 * lag) * ustep, sub);
    }
    if (ResetsSlots<Pr>::value && it + 1 < a.iters) wait_vm_all();
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// Two-shot AllReduce, one wave per peer, with LDS staging of the partial sums
// (8-byte packets, sentinel units or 128-byte lines); its two halves serve as
// the stand-alone ReduceScatter (Mode 1) and AllGather (Mode 2).
//
// A workgroup has P waves and handles one tile at the same offset in every
// chunk: 64*U units of a one-lane format (lane l owns units l, l+64, ...) or
// U line units (each a whole wave), as in WaveUnits.
// ReduceScatter: wave q != r sends the tile of chunk q to its owner q (one
// store per unit) and polls the tile of chunk r that peer q sent to this
// rank; wave r loads its own chunk r.  Each wave stages the raw payload
// words in LDS row q.  After a workgroup barrier the workgroup's threads
// share the ordered sum: each reduces some payload words of the tile over the
// P rows, widened to binary32 in ascending rank order, rounds once and
// writes the result to a reduced row; after a second barrier every wave reads
// its lanes' reduced words.  AllGather: wave q != r sends the reduced tile (for
// Mode 2: the own input) to peer q and polls the tile of chunk q that peer q
// sends back, and stores it; wave r stores the own chunk.  As in the one-shot
// wave kernel, a wave's polls wait for no stores but its own: those of this
// tile and, when the workgroup has another tile in the iteration, that
// tile's ReduceScatter packets, which go out ahead.  Readers clear the slots
// they have read when the call asks for it (KArgs::clear).
//
// Chunks: Mode 0 cuts the n-element input into chunks of a.chunk elements
// (the last ones may be short); Mode 1 takes P chunks of a.n elements;
// Mode 2 has one a.n-element input per rank.  Outputs: Mode 0, rank r's n
// elements; Mode 1, rank r's chunk; Mode 2, the P blocks of rank r.
template <class Pr, int DT, int P, int U, int Mode = 0>
__global__ __launch_bounds__(512) void k_twoshot_waves(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  using WU = WaveUnits<Pr, U>;
  constexpr int WPU = Pr::kMaxWords;  // payload words per lane and unit slot
  constexpr bool kRS = Mode != 2, kAG = Mode != 1;
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;  // past every slot: the buffer resource discards the store
  // ReduceScatter staging: the raw payload words of each rank's tile (row q:
  // rank q's values, in lane order), and the reduced tile.
  __shared__ u32x4 stage[kRS ? P : 1][64 * U];
  __shared__ u32x4 red[kRS ? 64 * U : 1];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);  // this wave's peer (q == r: the own values)
  const int lane = (int)(threadIdx.x & 63);
  const int sub = WU::sub(lane);
  const bool in_al4 = a.in_al4 != 0;
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const uint32_t slot = (uint32_t)a.slot;
  // The current iteration (Mode 0 calls may run several, each through
  // sub-buffer it % 2 with the flag epoch + it): its elements, chunk length,
  // input, output offset, packet area and flag.
  // Iteration 0 of a Mode 0 call holds min(n, iter_n) elements; its chunk
  // length a.chunk comes from the host (iter_span of iteration 0).
  int64_t n_all = Mode == 0 ? (a.n < a.iter_n ? a.n : a.iter_n) : (int64_t)P * a.n;
  int64_t C = Mode == 0 ? a.chunk : a.n;
  const char *in_it = in_r;
  uint64_t area = a.area;
  uint32_t epoch = a.epoch;
  auto in_chunk = [&](uint32_t c) -> const char * { return Mode == 2 ? in_it : in_it + (uint64_t)c * C * E; };
  auto chunk_len = [&](uint32_t c) -> int64_t {
    const int64_t left = n_all - (int64_t)c * C;
    return left < 0 ? 0 : (left < C ? left : C);
  };
  // unit and tile indices fit 32 bits: a call's slots span less than 4 GiB.
  // The first step uses the host's unit count and 32-bit chunk arithmetic
  // (element counts and chunk offsets fit 32 bits, an input being at most
  // 256 MiB), which keeps the set-up before the first packet store short.
  uint32_t units = (uint32_t)a.units;
  // Every packet store is issued, at an offset past the slot when there is
  // nothing to send (the own rank, a unit past the end, a muted rank), and no
  // store is branched around: a branch would leave the input load pending on
  // one path, and the compiler would then wait for every outstanding memory
  // operation, the store's acknowledgement included, before the next poll.
  const bool publish = (int)r != a.mute && q != r;
  auto store_units = [&](char *dst, uint32_t tile, const u32x4 *v) {
    const rsrc_t rd = make_rsrc(dst, slot);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
      st_pkt(rd, u < units && publish ? WU::off(u, lane) : kNowhere, Pr::pack(v[k], epoch, sub));
    }
  };
  // slot (q <- r) in peer q's slice and slot (r <- q) in this rank's slice
  char *const slot_out = a.sym + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot;
  char *const slot_in = a.sym + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot;
  const uint64_t ag_off = Mode == 2 ? 0 : (uint64_t)(P - 1) * slot;  // AllGather slots follow the RS slots

  // The first step of the first tile goes out before the rest of the set-up:
  // each wave loads the tile of chunk q (Mode 2: of its own input) and sends
  // it to peer q, the ReduceScatter packets (Mode 2: the AllGather packets).
  // The host launches no more workgroups per rank than there are tiles; a
  // workgroup past the last tile (a forced launch shape) loads and stores
  // nothing, since every access is guarded by the unit count.
  // With 4-byte aligned inputs the loads go through a buffer resource that
  // covers the chunk: no branch separates them, so the U loads of a lane are
  // all in flight before the first result is used (line units move their
  // displaced words only then).
  auto load_units = [&](const char *src, int64_t len, uint32_t tile, u32x4 *v) {
    if (in_al4) {
      const rsrc_t rs = make_rsrc(src, ((uint32_t)len * (uint32_t)E + 3u) & ~3u);
      uint32_t w0[U];
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
        w0[k] = u < units ? Pr::first_word(u, sub) : kNoWord;
        v[k] = load_words_rs<WPU>(rs, w0[k]);
      }
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if (ResetsSlots<Pr>::value) v[k] = clear_tail<DT, WPU>(v[k], w0[k], (uint32_t)len);
        v[k] = Pr::finish_load(v[k], sub);
      }
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
        v[k] = u < units ? Pr::template load<DT>(src, u, sub, len, in_al4) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  u32x4 first[U];
  {
    const uint32_t c0 = Mode == 2 ? r : q;
    const int32_t left = (int32_t)n_all - (int32_t)(c0 * (uint32_t)C);
    const int64_t len0 = left < 0 ? 0 : (left < (int32_t)C ? left : (int32_t)C);
    load_units(Mode == 2 ? in_it : in_it + (uint64_t)(c0 * (uint32_t)(C * E)), len0, w, first);
  }
  store_units(slot_out + area + (Mode == 2 ? ag_off : 0), w, first);
  units = (uint32_t)Pr::units((C * E + 3) / 4);  // the same count, for the loop below

  const bool al4 = a.al4 != 0;
  WaitBudget budget(a.timeout, a.status);
  // rank r's output: Mode 0 all n elements, Mode 1 its chunk, Mode 2 its P blocks
  char *const out_rank = a.out + (uint64_t)r * (uint64_t)(Mode == 2 ? (int64_t)P * a.n : a.n) * E;
  uint64_t out_off = 0;
  // where this rank's result for chunk c goes
  auto out_chunk = [&](uint32_t c) -> char * {
    if (Mode == 1) return out_rank;
    return out_rank + out_off + (uint64_t)c * C * E;
  };
  // Store U units (packet order) of a result stream of len elements.  With a
  // 4-byte aligned output and whole words the stores go through a buffer
  // resource that covers the stream (no branch, the range check drops what
  // lies past the end); otherwise element-wise at the edges.
  auto store_out = [&](char *dst, int64_t len, uint32_t tile, const u32x4 *v) {
    const uint32_t nb = (uint32_t)len * (uint32_t)E;
    if (al4 && (nb & 3u) == 0) {
      const rsrc_t rs = make_rsrc(dst, nb);
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
        const u32x4 w = Pr::start_store(v[k], sub);
        store_words_rs<WPU>(rs, u < units ? Pr::first_word(u, sub) : kNoWord, w);
      }
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) Pr::template store<DT>(dst, WU::unit(tile, k, lane), sub, len, al4, v[k]);
    }
  };

  auto stage_row = [&](const u32x4 *v) {
#pragma unroll
    for (int k = 0; k < U; ++k) stage[kRS ? q : 0][k * 64 + lane] = v[k];
  };

  // Poll U units of slot `src` (this rank's slice) from peer q; sentinel
  // units are given back to the sentinel once read, flagged units set to zero
  // when the call clears slots.  The loop runs while any
  // lane of the wave still waits (a wave vote ends it) and re-loads every
  // unit each round.
  auto poll_peer = [&](char *src, uint32_t tile, u32x4 *v) {
    const rsrc_t rs = make_rsrc(src, slot);
    uint32_t pend = 0;
#pragma unroll
    for (int k = 0; k < U; ++k) {
      v[k] = u32x4{0u, 0u, 0u, 0u};
      pend |= ((uint32_t)WU::unit(tile, k, lane) < units ? 1u : 0u) << k;
    }
    idle64(a.first_wait);
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      u32x4 pk[U];
#pragma unroll
      for (int k = 0; k < U; ++k) pk[k] = ld_pkt(rs, WU::off(WU::unit(tile, k, lane), lane));
#pragma unroll
      for (int k = 0; k < U; ++k) {
        if ((pend & (1u << k)) && Pr::ready(pk[k], epoch)) {
          v[k] = Pr::unpack(pk[k], sub);
          pend &= ~(1u << k);
        }
      }
      if (__builtin_amdgcn_ballot_w64(pend != 0) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend != 0) budget.report((int)r, 1u << q, epoch);
        break;
      }
      idle64(a.poll_gap);
    }
    if (ResetsSlots<Pr>::value || a.clear != 0) {
      const uint32_t fill = ResetsSlots<Pr>::value ? ProtoSent::kSentinel : 0u;
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const uint32_t u = (uint32_t)WU::unit(tile, k, lane);
        if (u < units) st_pkt(rs, WU::off(u, lane), u32x4{fill, fill, fill, fill});
      }
    }
  };

  const uint32_t iters = Mode == 0 ? a.iters : 1u;
  const uint32_t W = a.grid / P;
  bool pre_sent = true;  // the first tile's first step went out above
// Diagnostics (-DLLCOLL_WAVE_PHASES=1): for lane 0 of each wave and the first
// tile, the times its ReduceScatter packets went out (k = 0), its peer's
// ReduceScatter packets were seen (1), it left the barrier (2) and its peer's
// AllGather packets were seen (3).
#define LL_TW_PHASE(k, expr)                                                          \
  do {                                                                                \
    if (LLCOLL_WAVE_PHASES && a.phases != nullptr && lane == 0 && tile == w && it == 0) \
      a.phases[4 * (blockIdx.x * P + q) + (k)] = (expr);                              \
  } while (0)
  for (uint32_t it = 0; it < iters; ++it) {
    if (Mode == 0 && it > 0) {
      const IterSpan sp = iter_span(a.n, a.iter_n, it, P, E);
      const int64_t e0 = sp.e0;
      n_all = sp.n;
      C = sp.chunk;
      in_it = in_r + e0 * E;
      out_off = (uint64_t)e0 * E;
      area = a.area + (uint64_t)(it & 1u) * a.sub_bytes;
      epoch = a.epoch + it;
      units = (uint32_t)Pr::units((C * E + 3) / 4);
    }
    const uint32_t tiles = (uint32_t)((units + WU::kPerTile - 1) / WU::kPerTile);
    for (uint32_t tile = w; tile < tiles; tile += W) {
      const bool sent_already = pre_sent;  // this tile's first step went out earlier
      pre_sent = false;
      u32x4 res[U];
      if constexpr (kRS) {
        // ---- ReduceScatter of this tile: wave q sends chunk q's tile to
        // peer q (earlier, for the first tile and for one sent ahead), then
        // sends the workgroup's next tile of the iteration ahead, so that its
        // packets travel while this tile is reduced and gathered, and polls
        // what peer q sent for this tile
        u32x4 mine[U];
        if (sent_already) {
#pragma unroll
          for (int k = 0; k < U; ++k) mine[k] = first[k];
        } else {
          load_units(in_chunk(q), chunk_len(q), tile, mine);
          store_units(slot_out + area, tile, mine);
        }
        if (tile + W < tiles) {
          load_units(in_chunk(q), chunk_len(q), tile + W, first);
          store_units(slot_out + area, tile + W, first);
          pre_sent = true;
        }
        LL_TW_PHASE(0, now_ticks() + (mine[0].x & 0u));
        if (q == r) {
          stage_row(mine);
        } else {
          u32x4 v[U];
          poll_peer(slot_in + area, tile, v);
          LL_TW_PHASE(1, now_ticks() + (v[0].x & 0u));
          stage_row(v);
        }
        lds_barrier();
        LL_TW_PHASE(2, now_ticks());
        // ---- the ordered sum of the tile, split over the workgroup: thread
        // t reduces payload words t, t + 64 P, ... of the tile over the P
        // rows in ascending rank order, in binary32, and rounds once; then
        // every wave takes the reduced words of its lanes
        {
          constexpr int kWords = 64 * U * WPU;
          const uint32_t *const rows = reinterpret_cast<const uint32_t *>(&stage[0][0]);
          uint32_t *const red_w = reinterpret_cast<uint32_t *>(&red[0]);
          for (int i = (int)threadIdx.x; i < kWords; i += 64 * P) {
            const int at = (i / WPU) * 4 + i % WPU;  // word j of a lane's unit slot sits at 4 * slot + j
            float acc[K];
            Elem<DT>::widen(rows[at], acc);
#pragma unroll
            for (int p = 1; p < P; ++p) {
              float f[K];
              Elem<DT>::widen(rows[p * 64 * U * 4 + at], f);
#pragma unroll
              for (int e = 0; e < K; ++e) acc[e] = acc[e] + f[e];
            }
            red_w[at] = Elem<DT>::narrow(acc);
          }
        }
        lds_barrier();
#pragma unroll
        for (int k = 0; k < U; ++k) res[k] = red[k * 64 + lane];
      } else {
        if (sent_already) {
#pragma unroll
          for (int k = 0; k < U; ++k) res[k] = first[k];
        } else {
          load_units(in_chunk(r), C, tile, res);
        }
      }
      // ---- AllGather of this tile: wave q sends the reduced tile to peer q
      // (Mode 2: above, for the first tile) and stores what peer q sent; the
      // own-rank wave stores the rank's own result
      if constexpr (kAG) {
        if (!(Mode == 2 && sent_already)) store_units(slot_out + area + ag_off, tile, res);
        // one output store site for both kinds of wave (chunk q; q == r:
        // the own result): the kernel is shorter, and measured faster at
        // every size, than with an inlined store_out in each branch
        u32x4 v[U];
        if (q == r) {
#pragma unroll
          for (int k = 0; k < U; ++k) v[k] = res[k];
        } else {
          poll_peer(slot_in + area + ag_off, tile, v);
          LL_TW_PHASE(3, now_ticks() + (v[0].x & 0u));
        }
        store_out(out_chunk(q), chunk_len(q), tile, v);
      } else {
        if (q == r) store_out(out_chunk(r), chunk_len(r), tile, res);
      }
      if constexpr (kRS) lds_barrier();  // the next tile overwrites the staging rows
    }
    // slot resets are stores: acknowledged before the next iteration's packets
    // go out, so that none can land after a peer's refill of its sub-buffer
    if ((ResetsSlots<Pr>::value || a.clear != 0) && it + 1 < iters) wait_vm_all();
  }
  stamp_end(a, t_start);
}
#undef LL_TW_PHASE

// Two-shot AllReduce (Mode 0), stand-alone ReduceScatter (Mode 1) or
// AllGather (Mode 2), one wave per peer, one tile of U units per lane per
// workgroup (U line units, or 64 U one-lane units), one iteration, every
// stream 4-byte aligned: the straight-line counterpart of k_twoshot_waves<Pr,
// DT, P, U, Mode> for calls whose tiles are all resident at once.  It carries
// no tile loop, no tile sent ahead, no iteration and no element-wise
// fallback for unaligned streams, which shortens what every workgroup runs
// (the instructions of a latency-bound call are paid for in its latency, see
// k_oneshot_tile).
//
// Workgroup (r, w) serves rank r and tile w of every chunk.  ReduceScatter:
// wave q loads tile w of chunk q of rank r's input and sends it to peer q
// (the own-rank wave keeps its own chunk's tile); every other wave polls
// what peer q sent for chunk r, and each stages its row in LDS.  After a
// barrier the workgroup forms the ordered sum word by word (binary32 in
// ascending rank order, one rounding) into a reduced row (Mode 1: the own
// wave stores it).  AllGather: wave q sends the reduced tile (Mode 2: the
// tile of the rank's input) to peer q and polls the tile of chunk q that
// peer q sends back; every wave stores its chunk's (block's) tile of the
// output.
template <class Pr, int DT, int P, int U, int Mode = 0>
__global__ __launch_bounds__(512) void k_twoshot_tile(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  using WU = WaveUnits<Pr, U>;
  constexpr int WPU = Pr::kMaxWords;          // payload words per lane and unit slot
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;  // past every slot: the buffer resource discards the access
  constexpr bool kRS = Mode != 2, kAG = Mode != 1;
  __shared__ u32x4 stage[kRS ? P : 1][kRS ? 64 * U : 1];
  __shared__ u32x4 red[kRS ? 64 * U : 1];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);  // this wave's peer (q == r: the own values)
  const int lane = (int)(threadIdx.x & 63);
  const int sub = WU::sub(lane);
  // Mode 0: chunks of C elements (a multiple of 16 bytes), the last ones
  // short or empty; Mode 1: P chunks of n elements; Mode 2: one input of n
  // elements.  Every chunk's byte length is a multiple of 4.
  const uint32_t n = (uint32_t)a.n;
  const uint32_t C = Mode == 0 ? (uint32_t)a.chunk : n;
  auto chunk_bytes = [&](uint32_t c) -> uint32_t {
    if (Mode != 0) return n * (uint32_t)E;
    const uint32_t c0 = c * C;
    return c0 >= n ? 0u : ((n - c0 < C ? n - c0 : C) * (uint32_t)E);
  };
  // the lane's unit slots: first payload word and packet offset (past the
  // end for a unit beyond the chunk)
  uint32_t fw[U], off[U];
  uint32_t have = 0;
#pragma unroll
  for (int k = 0; k < U; ++k) {
    const uint32_t u = (uint32_t)WU::unit(w, k, lane);
    const bool h = u < (uint32_t)a.units;
    have |= (h ? 1u : 0u) << k;
    fw[k] = h ? Pr::first_word(u, sub) : kNoWord;
    off[k] = h ? WU::off(u, lane) : kNowhere;
  }
  u32x4 x[U];
  {
    const rsrc_t in_rs =
        make_rsrc(a.in + (uint64_t)r * a.in_stride + (Mode == 2 ? 0 : (uint64_t)q * C * E), chunk_bytes(q));
#pragma unroll
    for (int k = 0; k < U; ++k) x[k] = load_words_rs<WPU>(in_rs, fw[k]);
  }
  const uint32_t slot = (uint32_t)a.slot;
  const bool publish = (int)r != a.mute && q != r;
  // slot (q <- r) in peer q's slice and slot (r <- q) in this rank's slice;
  // the AllGather slots follow the P - 1 ReduceScatter slots (Mode 2 has
  // AllGather slots only).  The first store is the ReduceScatter (Mode 2:
  // the AllGather) of the tile.
  char *const slot_out = a.sym + a.area + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot;
  char *const slot_in = a.sym + a.area + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot;
  const uint64_t ag_off = Mode == 2 ? 0 : (uint64_t)(P - 1) * slot;
  {
    const rsrc_t rd = make_rsrc(slot_out, slot);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      x[k] = Pr::finish_load(x[k], sub);
      st_pkt(rd, publish ? off[k] : kNowhere, Pr::pack(x[k], a.epoch, sub));
    }
  }
#define LL_TT_PHASE(k, expr)                                            \
  do {                                                                  \
    if (LLCOLL_WAVE_PHASES && a.phases != nullptr && lane == 0)         \
      a.phases[4 * (blockIdx.x * P + q) + (k)] = (expr);                \
  } while (0)
  LL_TT_PHASE(0, now_ticks() + (x[0].x & 0u));
  WaitBudget budget(a.timeout, a.status);
  // Poll the U units from peer q in `src` (this rank's slice), then give the
  // slots back to the sentinel (sentinel units) or to zero (flagged units,
  // when the call clears slots).  Every lane runs the readiness check (a
  // line's flag sits in the last lane of each quad).
  auto poll = [&](char *src, u32x4 *v) {
    const rsrc_t rs = make_rsrc(src, slot);
    uint32_t pend = have;
#pragma unroll
    for (int k = 0; k < U; ++k) v[k] = u32x4{0u, 0u, 0u, 0u};
    idle64(a.first_wait);
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      u32x4 pk[U];
#pragma unroll
      for (int k = 0; k < U; ++k) pk[k] = ld_pkt(rs, off[k]);
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const bool ok = Pr::ready(pk[k], a.epoch);
        if ((pend & (1u << k)) && ok) {
          v[k] = Pr::unpack(pk[k], sub);
          pend &= ~(1u << k);
        }
      }
      if (__builtin_amdgcn_ballot_w64(pend != 0) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend != 0) budget.report((int)r, 1u << q, a.epoch);
        break;
      }
      idle64(a.poll_gap);
    }
    if (ResetsSlots<Pr>::value || a.clear != 0) {
      const uint32_t fill = ResetsSlots<Pr>::value ? ProtoSent::kSentinel : 0u;
#pragma unroll
      for (int k = 0; k < U; ++k) st_pkt(rs, off[k], u32x4{fill, fill, fill, fill});
    }
  };
  u32x4 res[U];
  if constexpr (kRS) {
    {
      u32x4 v[U];
      if (q != r) {
        poll(slot_in, v);
        LL_TT_PHASE(1, now_ticks() + (v[0].x & 0u));
      } else {
#pragma unroll
        for (int k = 0; k < U; ++k) v[k] = x[k];
      }
#pragma unroll
      for (int k = 0; k < U; ++k) stage[q][k * 64 + lane] = v[k];
    }
    lds_barrier();
    LL_TT_PHASE(2, now_ticks());
    // thread t reduces payload words t, t + 64 P, ... of the tile over the
    // P rows (word j of unit slot s sits at 4 * s + j)
    constexpr int kWords = 64 * U * WPU;
    const uint32_t *const rows = reinterpret_cast<const uint32_t *>(&stage[0][0]);
    uint32_t *const red_w = reinterpret_cast<uint32_t *>(&red[0]);
    for (int i = (int)threadIdx.x; i < kWords; i += 64 * P) {
      const int at = (i / WPU) * 4 + i % WPU;
      float acc[K];
      Elem<DT>::widen(rows[at], acc);
#pragma unroll
      for (int p = 1; p < P; ++p) {
        float f[K];
        Elem<DT>::widen(rows[p * 64 * U * 4 + at], f);
#pragma unroll
        for (int e = 0; e < K; ++e) acc[e] = acc[e] + f[e];
      }
      red_w[at] = Elem<DT>::narrow(acc);
    }
    lds_barrier();
#pragma unroll
    for (int k = 0; k < U; ++k) res[k] = red[k * 64 + lane];
  } else {
#pragma unroll
    for (int k = 0; k < U; ++k) res[k] = x[k];
  }
  if constexpr (kAG) {
    if constexpr (Mode == 0) {
      const rsrc_t rd = make_rsrc(slot_out + ag_off, slot);
#pragma unroll
      for (int k = 0; k < U; ++k) st_pkt(rd, publish ? off[k] : kNowhere, Pr::pack(res[k], a.epoch, sub));
    }
    u32x4 o[U];
    if (q != r) {
      poll(slot_in + ag_off, o);
      LL_TT_PHASE(3, now_ticks() + (o[0].x & 0u));
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) o[k] = res[k];
    }
    // Mode 0: the tile of chunk q of rank r's output; Mode 2: the tile of
    // block q of rank r's P blocks
    const uint64_t o0 = Mode == 0 ? (uint64_t)r * n + (uint64_t)q * C : ((uint64_t)r * P + q) * n;
    const rsrc_t out_rs = make_rsrc(a.out + o0 * E, chunk_bytes(q));
#pragma unroll
    for (int k = 0; k < U; ++k) store_words_rs<WPU>(out_rs, fw[k], Pr::start_store(o[k], sub));
  } else {
    // Mode 1: the own chunk's tile of rank r's output
    if (q == r) {
      const rsrc_t out_rs = make_rsrc(a.out + (uint64_t)r * n * E, n * (uint32_t)E);
#pragma unroll
      for (int k = 0; k < U; ++k) store_words_rs<WPU>(out_rs, fw[k], Pr::start_store(res[k], sub));
    }
  }
#undef LL_TT_PHASE
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// Two-shot AllReduce with atomic accumulation: the gfx950 analogue of the
// paper's two-shot LL128 atomic algorithm (Sec. IV, "LL128 Atomic AllReduce";
// Fig. 5).
//
// ReduceScatter.  Every rank adds its chunk c, widened to binary32, into an
// accumulator in rank c's slice with device-scope float atomic adds (its own
// chunk included).  The hardware gives no 128-byte line atomicity, so the
// flag cannot ride inside the data: after the adds of a tile (one wave's 64
// lanes x 16 input bytes) a wave bumps that tile's counter with a
// release-ordered atomic add.  Owner c waits (acquire) until the counter
// reaches P, then reads the accumulated tile, rounds once to the element type
// and resets accumulator and counter to zero for the next call.
// AllGather.  The owner stores the result into its own output and straight
// into every peer's output, which the caller has filled with the sentinel
// (as in the paper's Fig. 5); each rank polls its own output until the peers'
// blocks no longer hold it.
// Like the paper's algorithm it is not deterministic: the order of the
// atomic adds, and with it the binary32 rounding, varies from call to call
// (the result obeys the gamma_{P-1} bound of the end of Sec. IV, checked by
// the tests).  Every rank still receives the same bits, because each element
// is rounded once, by its owner.
// Slice layout of the area: accumulator (a.slot bytes: binary32 for every
// element of the chunk's whole tiles), then one u32 counter per tile.  The
// caller guarantees 16-byte aligned rows (count * esize % 16 == 0), so every
// lane's 16 input bytes are wholly inside or wholly outside a chunk.
template <int DT, int P>
__global__ __launch_bounds__(1024) void k_twoshot_atomic(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int EL = 16 / E;  // elements per lane: 16 input bytes
  constexpr int TE = 64 * EL; // elements per tile (one wave)
  const Part pt = part_of_block<P>(a);
  const int r = pt.r;
  const int lane = (int)(threadIdx.x & 63);
  const int64_t gw = ((int64_t)pt.w * a.block + threadIdx.x) >> 6;
  const int64_t GW = ((int64_t)pt.W * a.block) >> 6;
  const int64_t n = a.n, C = a.chunk;
  const int64_t tiles = (C + TE - 1) / TE;
  WaitBudget budget(a.timeout, a.status);
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  char *const out_r = a.out + (uint64_t)r * (uint64_t)n * E;
  const bool publish = (r != a.mute);
  auto chunk_len = [&](int c) -> int64_t {
    const int64_t left = n - (int64_t)c * C;
    return left < 0 ? 0 : (left < C ? left : C);
  };
  auto acc_of = [&](int c) -> float * { return (float *)(a.sym + (uint64_t)c * a.stride + a.area); };
  auto cnt_of = [&](int c) -> uint32_t * { return (uint32_t *)(a.sym + (uint64_t)c * a.stride + a.area + a.slot); };

  auto step_add = [&](int64_t t) {
    const int64_t e0 = t * TE + (int64_t)lane * EL;
    // Branch-free: all P loads first (a lane's 16 bytes lie wholly inside or
    // wholly outside a chunk), then all adds back to back.  The memory
    // counter covers loads and atomics alike, so any wait between the adds
    // would serialise them.  Lanes past a chunk's end add zeros into the
    // accumulator's tile padding, which is never read.
    u32x4 w[P];
#pragma unroll
    for (int k = 1; k <= P; ++k) {
      const int c = (r + k) % P;  // own chunk last
      const bool ok = e0 < chunk_len(c);
      const char *src = ok ? in_r + ((uint64_t)c * C + e0) * E : in_r;
      const u32x4 v = __builtin_nontemporal_load((const u32x4 *)src);
      w[k - 1] = ok ? v : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int k = 1; k <= P; ++k) {
      const int c = (r + k) % P;
      const uint32_t wv[4] = {w[k - 1].x, w[k - 1].y, w[k - 1].z, w[k - 1].w};
      float *acc = acc_of(c) + e0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float f[Elem<DT>::kPerWord];
        Elem<DT>::widen(wv[j], f);
#pragma unroll
        for (int h = 0; h < Elem<DT>::kPerWord; ++h)
          __hip_atomic_fetch_add(acc + j * Elem<DT>::kPerWord + h, f[h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    // the wave's adds of this tile are performed before its counters move
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    if (lane == 0) {
#pragma unroll
      for (int k = 1; k <= P; ++k) {
        const int c = (r + k) % P;
        if (t * TE < chunk_len(c))
          __hip_atomic_fetch_add(cnt_of(c) + t, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  };

  auto step_reduce = [&](int64_t t) {
    const int64_t len = chunk_len(r);
    if (t * TE >= len) return;
    uint32_t *cnt = cnt_of(r) + t;
    int spins = 1;
    while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != (uint32_t)P) {
      if ((spins++ & 15) == 0 && budget.expired()) {
        budget.report(r, ((1u << P) - 1u) & ~(1u << r), a.epoch);
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int64_t e0 = t * TE + (int64_t)lane * EL;
    if (e0 < len) {
      float *acc = acc_of(r) + e0;
      float f[EL];
#pragma unroll
      for (int j = 0; j < EL; ++j) f[j] = __hip_atomic_load(acc + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      uint32_t res[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) res[j] = Elem<DT>::narrow(&f[j * Elem<DT>::kPerWord]);
      const u32x4 v = {res[0], res[1], res[2], res[3]};
      store_words<DT>(out_r + (uint64_t)r * C * E, e0 / Elem<DT>::kPerWord, 4, len, true, v);
      if (publish) {
        const uint32_t at = uniform_u32((uint32_t)(r * C * E));
#pragma unroll
        for (int k = 1; k < P; ++k) {
          const int q = (r + k) % P;
          st_pkt_at(make_rsrc(a.out + (uint64_t)q * (uint64_t)n * E, (uint32_t)(n * E)), (uint32_t)(e0 * E), at, v);
        }
      }
      // back to zero for the next call (ordered by the kernel boundary)
#pragma unroll
      for (int j = 0; j < EL; ++j) __hip_atomic_store(acc + j, 0.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (lane == 0) __hip_atomic_store(cnt, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  };

  auto step_gather = [&](int64_t t) {
    const int64_t e0 = t * TE + (int64_t)lane * EL;
    uint32_t pend = 0;
#pragma unroll
    for (int q = 0; q < P; ++q)
      if (q != r && e0 < chunk_len(q)) pend |= 1u << q;
    poll_out<P>(out_r, (uint32_t)(n * E), (uint32_t)(C * E), (uint32_t)(e0 * E), pend, r, a.epoch, budget);
  };

  const int64_t steps = gw < tiles ? (tiles - gw + GW - 1) / GW : 0;
  const int64_t lag = a.lag;
  for (int64_t s = 0; s < steps + 2 * lag; ++s) {
    if (s < steps && publish) step_add(gw + s * GW);
    if (s >= lag && s - lag < steps) step_reduce(gw + (s - lag) * GW);
    if (s >= 2 * lag && s - 2 * lag < steps) step_gather(gw + (s - 2 * lag) * GW);
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// Broadcast and Reduce (the artifact's further collectives, Sec. V), one
// exchange each, from the same packet primitives.
//
// Broadcast: the root stores its input units into slot (q <- root) of every
// peer q and copies them to its own output; every other rank polls that one
// slot and stores what arrives.  Output: every rank's copy, back to back.
template <class Pr, int DT, int P>
__global__ __launch_bounds__(1024) void k_broadcast(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  const uint32_t r = blockIdx.x % P, w = blockIdx.x / P;
  const uint32_t root = (uint32_t)a.root;
  const int64_t n = a.n;
  // unit indices fit 32 bits: a call's P-1 slots span less than 4 GiB
  const uint32_t units = (uint32_t)a.units;
  const uint32_t g = w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const uint32_t ustep = (a.grid / P) * a.block / Pr::kLanes;
  if (r == root) {
    // The root's first unit is loaded and sent before the rest of its
    // set-up; a lane past the end stores at an offset past the slot, which
    // the buffer resource discards, so no store is branched around.
    constexpr uint32_t kNowhere = 0xFFFFFFF0u;
    const char *const in_r = a.in + (uint64_t)r * a.in_stride;
    const bool publish = (int)r != a.mute;
    for (uint32_t u = g / Pr::kLanes; u < units; u += ustep) {
      const uint32_t off = u * Pr::kUnitBytes + sub * 16;
      const u32x4 own = Pr::template load<DT>(in_r, u, sub, n, a.in_al4 != 0);
      bcast<P>(a, a.area, (int)r, publish ? off : kNowhere, Pr::pack(own, a.epoch, sub));
      Pr::template store<DT>(a.out + (uint64_t)r * (uint64_t)n * E, u, sub, n, a.al4 != 0, own);
    }
  } else {
    char *const area_r = a.sym + (uint64_t)r * a.stride + a.area;
    char *const out_r = a.out + (uint64_t)r * (uint64_t)n * E;
    WaitBudget budget(a.timeout, a.status);
    for (uint32_t u = g / Pr::kLanes; u < units; u += ustep) {
      const uint32_t off = u * Pr::kUnitBytes + sub * 16;
      u32x4 got[P];
      poll_all<Pr, P>(area_r, a.slot, off, (int)r, a.epoch, budget, got, 0, 0, 1u << root);
      Pr::template store<DT>(out_r, u, sub, n, a.al4 != 0, Pr::unpack(got[root], sub));
    }
  }
  stamp_end(a, t_start);
}

// Reduce: every rank but the root stores its input units into slot
// (root <- q) of the root; the root polls its P-1 slots and sums all P
// contributions in ascending rank order, rounding once (as AllReduce).
// Output: the root's result only, `n` elements at `out`.
template <class Pr, int DT, int P>
__global__ __launch_bounds__(1024) void k_reduce(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  const uint32_t r = blockIdx.x % P, w = blockIdx.x / P;
  const uint32_t root = (uint32_t)a.root;
  const int64_t n = a.n;
  const uint32_t units = (uint32_t)a.units;
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const uint32_t g = w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const uint32_t ustep = (a.grid / P) * a.block / Pr::kLanes;
  if (r != root) {
    // a sender: load and store, nothing else; a muted rank stores at an
    // offset past the slot, which the buffer resource discards
    constexpr uint32_t kNowhere = 0xFFFFFFF0u;
    const bool publish = (int)r != a.mute;
    const uint32_t slot = (uint32_t)a.slot;
    const rsrc_t rs = make_rsrc(a.sym + (uint64_t)root * a.stride + a.area + (r - (r > root ? 1u : 0u)) * slot, slot);
    for (uint32_t u = g / Pr::kLanes; u < units; u += ustep) {
      const uint32_t off = u * Pr::kUnitBytes + sub * 16;
      st_pkt(rs, publish ? off : kNowhere, Pr::pack(Pr::template load<DT>(in_r, u, sub, n, a.in_al4 != 0), a.epoch, sub));
    }
  } else {
    char *const area_r = a.sym + (uint64_t)r * a.stride + a.area;
    WaitBudget budget(a.timeout, a.status);
    for (uint32_t u = g / Pr::kLanes; u < units; u += ustep) {
      const uint32_t off = u * Pr::kUnitBytes + sub * 16;
      const u32x4 own = Pr::template load<DT>(in_r, u, sub, n, a.in_al4 != 0);
      u32x4 got[P];
      poll_all<Pr, P>(area_r, a.slot, off, (int)r, a.epoch, budget, got);
#pragma unroll
      for (int q = 0; q < P; ++q) got[q] = Pr::unpack(got[q], sub);
      Pr::template store<DT>(a.out, u, sub, n, a.al4 != 0, reduce_ordered<Pr, DT, P>(got, own, (int)r));
    }
  }
  stamp_end(a, t_start);
}

// Broadcast and Reduce with one wave per peer and one tile of 64 one-lane
// units per workgroup (8-byte packets or sentinel units), every stream 4-byte
// aligned, all tiles resident at once: the straight-line counterparts of
// k_broadcast and k_reduce, in the form of k_oneshot_tile.  Lane l of
// workgroup (r, w) owns unit u = 64 w + l.
//   Broadcast (Kind 0): on the root, wave q loads the unit of the root's
//     input and stores it as a packet to slot (q <- root) of peer q (the
//     root's own wave stores it to the root's output instead); on any other
//     rank, wave 0 polls slot (r <- root) and stores the payload to the
//     rank's output, and the other waves have nothing to do.
//   Reduce (Kind 1): on every other rank, wave 0 loads the unit and stores
//     it to slot (root <- r) of the root; on the root, wave q polls slot
//     (root <- q) (its own wave loads its input), stages the values widened
//     to binary32 in LDS row q, and after one barrier wave 0 sums the P rows
//     in ascending rank order, rounds once and stores the root's output.
// Readers clear (flagged) or reset (sentinel) the slots they have read.
template <class Pr, int DT, int P, int Kind>
__global__ __launch_bounds__(512) void k_rooted_tile(KArgs ka) {
  static_assert(Pr::kLanes == 1, "one-lane packet formats only");
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  constexpr int E = Elem<DT>::kBytes;
  constexpr int K = Elem<DT>::kPerWord;
  constexpr int NW = Pr::kMaxWords;  // payload words per lane
  constexpr int EPL = NW * K;        // elements per lane
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;
  __shared__ float stage[Kind == 1 ? P : 1][Kind == 1 ? 64 * EPL : 1];
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t u = w * 64 + lane;
  const uint32_t root = (uint32_t)a.root;
  const uint32_t nb = (uint32_t)(a.n * E);  // bytes per rank (< 256 MiB)
  const uint32_t slot = (uint32_t)a.slot;
  const bool have = u < (uint32_t)a.units;
  const uint32_t off = have ? u * 16 : kNowhere;
  const bool publish = (int)r != a.mute;
  // Poll the unit in slot `src` of this rank's slice, then clear or reset it.
  auto poll = [&](char *src) -> u32x4 {
    const rsrc_t rs = make_rsrc(src, slot);
    WaitBudget budget(a.timeout, a.status);
    u32x4 v = {0u, 0u, 0u, 0u};
    bool pend = have;
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      const u32x4 pk = ld_pkt(rs, off);
      if (pend && Pr::ready(pk, a.epoch)) {
        v = Pr::unpack(pk, 0);
        pend = false;
      }
      if (__builtin_amdgcn_ballot_w64(pend) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend) budget.report((int)r, 1u << (Kind == 0 ? root : q), a.epoch);
        break;
      }
    }
    if (ResetsSlots<Pr>::value) {
      st_pkt(rs, off, u32x4{ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel, ProtoSent::kSentinel});
    } else if (a.clear != 0) {
      st_pkt(rs, off, u32x4{0u, 0u, 0u, 0u});
    }
    return v;
  };
  auto load_own = [&]() -> u32x4 {
    u32x4 x = load_words_rs<NW>(make_rsrc(a.in + (uint64_t)r * a.in_stride, (nb + 3u) & ~3u), u * NW);
    if (ResetsSlots<Pr>::value) x = clear_tail<DT, NW>(x, u * NW, (uint32_t)a.n);
    return x;
  };
  if constexpr (Kind == 0) {
    if (r == root) {
      const u32x4 x = load_own();
      if (q != r) {
        char *const dst = a.sym + a.area + (uint64_t)q * a.stride + (uint64_t)slot_of((int)r, (int)q) * slot;
        st_pkt(make_rsrc(dst, slot), publish ? off : kNowhere, Pr::pack(x, a.epoch, 0));
      } else {
        store_words_rs<NW, false>(make_rsrc(a.out + (uint64_t)r * nb, nb), u * NW, x);
      }
    } else if (q == 0) {
      const u32x4 v = poll(a.sym + a.area + (uint64_t)r * a.stride + (uint64_t)slot_of((int)root, (int)r) * slot);
      store_words_rs<NW, false>(make_rsrc(a.out + (uint64_t)r * nb, nb), u * NW, v);
    }
  } else {
    if (r != root) {
      if (q == 0) {
        const u32x4 x = load_own();
        char *const dst = a.sym + a.area + (uint64_t)root * a.stride + (uint64_t)slot_of((int)r, (int)root) * slot;
        st_pkt(make_rsrc(dst, slot), publish ? off : kNowhere, Pr::pack(x, a.epoch, 0));
      }
    } else {
      u32x4 v;
      if (q == r) {
        v = load_own();
      } else {
        v = poll(a.sym + a.area + (uint64_t)r * a.stride + (uint64_t)slot_of((int)q, (int)r) * slot);
      }
      const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int j = 0; j < NW; ++j) {
        float f[K];
        Elem<DT>::widen(vw[j], f);
#pragma unroll
        for (int e = 0; e < K; ++e) stage[q][lane * EPL + j * K + e] = f[e];
      }
      lds_barrier();
      if (q == 0) {
        uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < NW; ++j) {
          float acc[K];
#pragma unroll
          for (int e = 0; e < K; ++e) acc[e] = stage[0][lane * EPL + j * K + e];
#pragma unroll
          for (int p = 1; p < P; ++p) {
#pragma unroll
            for (int e = 0; e < K; ++e) acc[e] = acc[e] + stage[p][lane * EPL + j * K + e];
          }
          o[j] = Elem<DT>::narrow(acc);
        }
        store_words_rs<NW, false>(make_rsrc(a.out, nb), u * NW, u32x4{o[0], o[1], o[2], o[3]});
      }
    }
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// Stand-alone ReduceScatter: rank r's input is P chunks of m = a.n elements;
// chunk c goes to slot (c <- r); rank r reduces chunk r.  The same two steps
// as the first two of the two-shot kernel, with chunks of exactly m
// elements, software-pipelined the same way (publish unit s, reduce unit
// s - lag).
template <class Pr, int DT, int P>
__global__ __launch_bounds__(1024) void k_reduce_scatter(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  const Part pt = part_of_block<P>(a);
  const int r = pt.r;
  constexpr int E = Elem<DT>::kBytes;
  WaitBudget budget(a.timeout, a.status);
  char *const slice_r = a.sym + (uint64_t)r * a.stride;
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const bool in_al4 = a.in_al4 != 0;
  char *const out_r = a.out + (uint64_t)r * (uint64_t)a.n * E;
  const int64_t m = a.n;
  const int64_t units = Pr::units((m * E + 3) / 4);
  const bool al4 = a.al4 != 0;
  const bool publish = (r != a.mute);
  const int64_t g = (int64_t)pt.w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const int64_t u0 = g / Pr::kLanes;
  const int64_t ustep = (int64_t)pt.W * a.block / Pr::kLanes;
  const int64_t steps = u0 < units ? (units - u0 + ustep - 1) / ustep : 0;
  const int64_t lag = a.lag;

  for (int64_t s = 0; s < steps + lag; ++s) {
    if (s < steps && publish) {
      const int64_t u = u0 + s * ustep;
      const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
      u32x4 v[P];
#pragma unroll
      for (int k = 1; k < P; ++k) {
        const int c = (r + k) % P;
        v[k] = Pr::template load<DT>(in_r + c * m * E, u, sub, m, in_al4);
      }
#pragma unroll
      for (int k = 1; k < P; ++k) {
        const int c = (r + k) % P;
        char *dst = a.sym + (uint64_t)c * a.stride + a.area + (uint64_t)slot_of(r, c) * a.slot;
        st_pkt(make_rsrc(dst, (uint32_t)a.slot), off, Pr::pack(v[k], a.epoch, sub));
      }
    }
    if (s >= lag && s - lag < steps) {
      const int64_t u = u0 + (s - lag) * ustep;
      const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
      const u32x4 own = Pr::template load<DT>(in_r + r * m * E, u, sub, m, in_al4);
      u32x4 got[P];
      poll_all<Pr, P>(slice_r + a.area, a.slot, off, r, a.epoch, budget, got);
#pragma unroll
      for (int q = 0; q < P; ++q) got[q] = Pr::unpack(got[q], sub);
      const u32x4 res = reduce_ordered<Pr, DT, P>(got, own, r);
      Pr::template store<DT>(out_r, u, sub, m, al4, res);
    }
  }
  stamp_end(a, t_start);
}

// ---------------------------------------------------------------------------
// Stand-alone AllGather: rank r sends its s = a.n input elements to slot
// (q <- r) of every peer, copies them to its own output, and stores what it
// receives from peer q at block q of its output.  Pipelined like the others:
// publish unit s, gather unit s - lag.
template <class Pr, int DT, int P>
__global__ __launch_bounds__(1024) void k_allgather(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  const Part pt = part_of_block<P>(a);
  const int r = pt.r;
  constexpr int E = Elem<DT>::kBytes;
  WaitBudget budget(a.timeout, a.status);
  char *const slice_r = a.sym + (uint64_t)r * a.stride;
  const char *const in_r = a.in + (uint64_t)r * a.in_stride;
  const int64_t n = a.n;
  const int64_t units = Pr::units((n * E + 3) / 4);
  const bool al4 = a.al4 != 0;
  char *const out_r = a.out + (uint64_t)r * (uint64_t)P * n * E;
  const bool publish = (r != a.mute);
  const int64_t g = (int64_t)pt.w * a.block + threadIdx.x;
  const int sub = (int)(g % Pr::kLanes);
  const int64_t u0 = g / Pr::kLanes;
  const int64_t ustep = (int64_t)pt.W * a.block / Pr::kLanes;
  const int64_t steps = u0 < units ? (units - u0 + ustep - 1) / ustep : 0;
  const int64_t lag = a.lag;

  for (int64_t s = 0; s < steps + lag; ++s) {
    if (s < steps) {
      const int64_t u = u0 + s * ustep;
      const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
      const u32x4 own = Pr::template load<DT>(in_r, u, sub, n, a.in_al4 != 0);
      if (publish) bcast<P>(a, a.area, r, off, Pr::pack(own, a.epoch, sub));
      Pr::template store<DT>(out_r + r * n * E, u, sub, n, al4, own);
    }
    if (s >= lag && s - lag < steps) {
      const int64_t u = u0 + (s - lag) * ustep;
      const uint32_t off = (uint32_t)(u * Pr::kUnitBytes + sub * 16);
      u32x4 got[P];
      poll_all<Pr, P>(slice_r + a.area, a.slot, off, r, a.epoch, budget, got);
#pragma unroll
      for (int q = 0; q < P; ++q) {
        if (q == r) continue;
        Pr::template store<DT>(out_r + q * n * E, u, sub, n, al4, Pr::unpack(got[q], sub));
      }
    }
  }
  stamp_end(a, t_start);
}

}  // namespace llc
