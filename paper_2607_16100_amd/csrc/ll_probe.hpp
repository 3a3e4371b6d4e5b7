// Measurement kernels: the single-GPU latency floor and the chip facts the
// packet protocols rely on.
//
// * Empty kernel and floor kernel: the floor of a small collective on one GPU
//   is a kernel launch plus one dependent HBM round trip (a load whose value
//   is stored).  Both are launched with the collective's grid so that
//   dispatch cost is the same.
// * Pointer chase: average latency of dependent loads that miss every cache.
// * Fence latency, L2-hit round trip and cross-XCD ping-pong: the pieces of
//   the paper's speed-of-light model (Sec. VI): L_SoL = 2 L_L2_RTT +
//   L_remote_store, with L_remote_store = (L_ping_pong - 2 L_L2_RTT) / 2.
// * XCD map: which XCD each workgroup of a grid runs on.
// * Litmus: whether 8-byte packets and 64-byte line halves written by one
//   workgroup are ever observed torn by a reader on another XCD.
// * Streaming: the HBM bandwidth that a plain kernel of 16-byte streaming
//   loads and stores reaches (copy, read only, write only), the practical
//   ceiling for the bandwidth-bound collectives.
// * Minimal exchange: the data movement of the one-wave-per-peer one-shot
//   with nothing else, the bound that kernel is measured against.
#pragma once

#include "ll_device.hpp"
#include "ll_kernels.hpp"

namespace llc {

// Start times are kept in a register and stored with the end times, as in the
// collectives, so that no store precedes the first load.
__global__ void k_probe_empty(uint64_t *stamps) {
  if (stamps != nullptr) {
    const uint64_t t0 = now_ticks();
    __syncthreads();
    if (threadIdx.x == 0) {
      stamps[blockIdx.x] = t0;
      stamps[gridDim.x + blockIdx.x] = now_ticks();
    }
  }
}

// One dependent HBM round trip: lane 0 of workgroup 0 loads chase[start]
// (a line nobody has touched recently) and stores the value.
__global__ void k_probe_floor(const uint64_t *chase, uint64_t start, uint64_t *sink, uint64_t *stamps) {
  const uint64_t t0 = stamps != nullptr ? now_ticks() : 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const uint64_t v = __builtin_nontemporal_load(chase + start);
    sink[0] = v;
  }
  if (stamps != nullptr) {
    __syncthreads();
    if (threadIdx.x == 0) {
      stamps[blockIdx.x] = t0;
      stamps[gridDim.x + blockIdx.x] = now_ticks();
    }
  }
}

// Dependent loads: idx = chase[idx], `steps` times, timed with the 100 MHz
// clock and the shader clock.  out = {realtime ticks, shader cycles, last idx}.
__global__ void k_probe_chase(const uint64_t *chase, uint64_t len, uint64_t start, int steps, uint64_t *out) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  uint64_t idx = start;
  const uint64_t t0 = now_ticks();
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  for (int i = 0; i < steps; ++i) {
    idx = __builtin_nontemporal_load(chase + idx);
    idx = idx < len ? idx : 0;  // a bad table can never send a load out of bounds
  }
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  const uint64_t t1 = now_ticks();
  out[0] = t1 - t0;
  out[1] = c1 - c0;
  out[2] = idx;
}

// Latencies in one lane, averaged over `iters` (out in 100 MHz ticks and
// shader cycles):
//   out[0..1]  a store followed by an agent-scope fence (__threadfence), the
//              paper's proxy for an L2 round trip (Sec. VI)
//   out[2..3]  a chain of dependent coherent (sc1) loads of one resident line,
//              the load the packet polls use
//   out[4..5]  a chain of dependent sc0 loads of one resident line
//   out[6]     sink
__global__ void k_probe_fence_l2(uint32_t *buf, int iters, uint64_t *out) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  uint64_t t0 = now_ticks();
  uint64_t c0 = __builtin_amdgcn_s_memtime();
  for (int i = 0; i < iters; ++i) {
    buf[0] = (uint32_t)i;
    __threadfence();
  }
  uint64_t c1 = __builtin_amdgcn_s_memtime();
  uint64_t t1 = now_ticks();
  out[0] = t1 - t0;
  out[1] = c1 - c0;
  const rsrc_t rs = make_rsrc(buf, 4096);
  uint32_t v = 0;
  for (int pass = 0; pass < 2; ++pass) {
    uint32_t idx = 16;
    t0 = now_ticks();
    c0 = __builtin_amdgcn_s_memtime();
    for (int i = 0; i < iters; ++i) {
      compiler_fence();
      v = pass == 0 ? __builtin_amdgcn_raw_buffer_load_b32(rs, (int)(idx * 4), 0, kSC1)
                    : __builtin_amdgcn_raw_buffer_load_b32(rs, (int)(idx * 4), 0, 1);
      idx = 16 + (v & 0x10000u);  // buf[16] holds 0, so idx stays 16 but depends on v
    }
    c1 = __builtin_amdgcn_s_memtime();
    t1 = now_ticks();
    out[2 + 2 * pass] = t1 - t0;
    out[3 + 2 * pass] = c1 - c0;
  }
  out[6] = v;
}

// Ping-pong between workgroup 0 and workgroup `peer` (placed on another XCD
// by the round-robin dispatch) through coherent stores and polls of two
// words 4 KiB apart.  Bounded: gives up after `limit` ticks per exchange.
// out = {total ticks, exchanges completed, shader cycles}.
__global__ void k_probe_pingpong(uint32_t *flags, int rounds, int peer, uint64_t limit, uint64_t *out) {
  if (threadIdx.x != 0) return;
  const int b = (int)blockIdx.x;
  if (b != 0 && b != peer) return;
  const rsrc_t rs = make_rsrc(flags, 8192);
  const uint32_t mine = (b == 0) ? 0u : 4096u;
  const uint32_t theirs = (b == 0) ? 4096u : 0u;
  const uint64_t t0 = now_ticks();
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  int done = 0;
  for (int i = 1; i <= rounds; ++i) {
    if (b == 0) {
      __builtin_amdgcn_raw_buffer_store_b32((uint32_t)i, rs, (int)theirs, 0, kSC1);
      const uint64_t end = now_ticks() + limit;
      uint32_t v;
      do {
        compiler_fence();
        v = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)mine, 0, kSC1);
      } while (v != (uint32_t)i && now_ticks() < end);
      if (v != (uint32_t)i) break;
    } else {
      const uint64_t end = now_ticks() + limit;
      uint32_t v;
      do {
        compiler_fence();
        v = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)mine, 0, kSC1);
      } while (v != (uint32_t)i && now_ticks() < end);
      if (v != (uint32_t)i) break;
      __builtin_amdgcn_raw_buffer_store_b32((uint32_t)i, rs, (int)theirs, 0, kSC1);
    }
    done = i;
  }
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  const uint64_t t1 = now_ticks();
  if (b == 0) {
    out[0] = t1 - t0;
    out[1] = (uint64_t)done;
    out[2] = c1 - c0;
  }
}

// One lane waits until `ticks` of the constant clock have passed since it
// started (at most 1 s), so that the host can queue launches behind it and
// they then run back to back without waiting for the host.
__global__ void k_probe_spin(uint64_t ticks) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  const uint64_t t0 = now_ticks();
  const uint64_t limit = ticks < 100000000ull ? ticks : 100000000ull;
  while (now_ticks() - t0 < limit) {
    __builtin_amdgcn_s_sleep(8);
  }
}

// XCD id (bits 3:0 of the XCC_ID hardware register) of every workgroup.
__global__ void k_probe_xcd(uint32_t *ids) {
  if (threadIdx.x == 0) ids[blockIdx.x] = __builtin_amdgcn_s_getreg(0xf814) & 0xfu;
}

// Litmus for packet atomicity across XCDs.  Workgroups [0, G/2) write,
// workgroups [G/2, G) read; reader b reads the lines written by writer
// (b - G/2 + 1) mod G/2, which the round-robin dispatch puts on another XCD.
// Each writer owns `lines` 128-byte lines and rewrites them `iters` times; in
// round e every payload dword k of line l holds mix(e, l, k), and the flags
// hold e.  layout 0: 8-byte packets {payload, flag} (a lane stores two);
// layout 1: 128-byte lines with a flag closing each 64-byte half.  A reader
// keeps loading and checks every unit whose flag is non-zero:
//   counts[0] units seen with a non-zero flag
//   counts[1] torn units: a payload dword that does not match its flag
//   counts[2] (layout 0) 16-byte lane loads whose two flags differ
//   counts[3] (layout 1) lines whose two halves carry different flags
__device__ __forceinline__ uint32_t litmus_mix(uint32_t e, uint32_t l, uint32_t k) {
  uint32_t x = e * 0x9E3779B1u ^ (l * 0x85EBCA77u + k * 0xC2B2AE3Du);
  x ^= x >> 15;
  x *= 0x2C1B3C6Du;
  x ^= x >> 12;
  return x;
}

__global__ __launch_bounds__(256) void k_probe_litmus(uint32_t *buf, int lines, int iters, int reads, int layout,
                                                    unsigned long long *counts) {
  const int G = (int)gridDim.x;
  const int half = G / 2;
  const int b = (int)blockIdx.x;
  const bool writer = b < half;
  const int owner = writer ? b : (b - half + 1) % half;
  uint32_t *base = buf + (size_t)owner * lines * 32;
  const rsrc_t rs = make_rsrc(base, (uint32_t)(lines * 128));
  const int lane = (int)threadIdx.x;
  const int sub = lane & 7;          // lane within a line
  const int l0 = lane >> 3;          // first line of this lane
  const int lstep = (int)blockDim.x >> 3;
  if (writer) {
    for (int e = 1; e <= iters; ++e) {
      for (int l = l0; l < lines; l += lstep) {
        u32x4 v;
        const uint32_t k0 = (uint32_t)sub * 4;
        if (layout == 0) {
          v.x = litmus_mix((uint32_t)e, (uint32_t)l, k0);
          v.y = (uint32_t)e;
          v.z = litmus_mix((uint32_t)e, (uint32_t)l, k0 + 2);
          v.w = (uint32_t)e;
        } else {
          v.x = litmus_mix((uint32_t)e, (uint32_t)l, k0);
          v.y = litmus_mix((uint32_t)e, (uint32_t)l, k0 + 1);
          v.z = litmus_mix((uint32_t)e, (uint32_t)l, k0 + 2);
          v.w = ((sub & 3) == 3) ? (uint32_t)e : litmus_mix((uint32_t)e, (uint32_t)l, k0 + 3);
        }
        st_pkt(rs, (uint32_t)(l * 128 + sub * 16), v);
      }
    }
    return;
  }
  unsigned long long seen = 0, torn = 0, split16 = 0, splitline = 0;
  for (int it = 0; it < reads; ++it) {
    for (int l = l0; l < lines; l += lstep) {
      compiler_fence();
      const u32x4 v = ld_pkt(rs, (uint32_t)(l * 128 + sub * 16));
      const uint32_t k0 = (uint32_t)sub * 4;
      if (layout == 0) {
        if (v.y != 0) {
          ++seen;
          if (v.x != litmus_mix(v.y, (uint32_t)l, k0)) ++torn;
        }
        if (v.w != 0) {
          ++seen;
          if (v.z != litmus_mix(v.w, (uint32_t)l, k0 + 2)) ++torn;
        }
        if (v.y != v.w) ++split16;
      } else {
        const uint32_t f = (uint32_t)__builtin_amdgcn_mov_dpp((int)v.w, 0xFF, 0xF, 0xF, false);
        // the other half's flag: lane 7 of the line for the first half, lane 3 for the second
        const uint32_t fo = (uint32_t)__builtin_amdgcn_ds_swizzle((int)f, 0x101F);  // xor lane id with 4
        if (f != 0) {
          bool bad = v.x != litmus_mix(f, (uint32_t)l, k0) || v.y != litmus_mix(f, (uint32_t)l, k0 + 1) ||
                     v.z != litmus_mix(f, (uint32_t)l, k0 + 2);
          if ((sub & 3) != 3) bad = bad || v.w != litmus_mix(f, (uint32_t)l, k0 + 3);
          if ((sub & 3) == 0) ++seen;
          if (bad) ++torn;
        }
        if (sub == 0 && f != fo) ++splitline;
      }
    }
  }
  atomicAdd(&counts[0], seen);
  atomicAdd(&counts[1], torn);
  atomicAdd(&counts[2], split16);
  atomicAdd(&counts[3], splitline);
}

// Streaming kernel over n16 16-byte words, grid-stride, one word per lane
// and step, non-temporal loads and stores.  mode 0: dst = src; mode 1: read
// src only (the xor of all words decides a store that never happens for
// these inputs, so the loads stay); mode 2: write dst only.
__global__ __launch_bounds__(1024) void k_probe_stream(const u32x4 *src, u32x4 *dst, uint64_t n16, int mode) {
  const uint64_t nth = (uint64_t)gridDim.x * blockDim.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += nth) {
    if (mode == 2) {
      __builtin_nontemporal_store(u32x4{(uint32_t)i, 1u, 2u, 3u}, &dst[i]);
      continue;
    }
    const u32x4 v = __builtin_nontemporal_load(&src[i]);
    if (mode == 0) {
      __builtin_nontemporal_store(v, &dst[i]);
    } else {
      acc ^= v;
    }
  }
  if (mode == 1 && acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u) dst[0] = acc;
}

// Minimal exchange with the grid and packet volume of the one-shot with one
// wave per peer and 8-byte packets (k_oneshot_waves): workgroup b serves rank
// r = b % P and tile w = b / P of 64 packet units (8 input bytes each); wave
// q of the workgroup loads the tile's input (each lane 8 bytes), stores it as
// one 16-byte packet store per lane into slot (q <- r) of peer q, polls the
// same units of slot (r <- q) in its own slice until both flags of every lane
// equal the epoch (a wave vote ends the loop), clears the slot it read when
// the call asks for it (as the one-shot collective does at every size), and
// stores the 8 payload bytes it received to the rank's output tile.  The
// own-rank wave stores its own input there without an exchange.  No LDS, no barrier, no sum: every wave of
// a workgroup writes the same output tile, so each output element ends up as
// one rank's input element (which one is unspecified).  The same instruction
// order as the collective: input load first, then the packet store with no
// branch around it.  Waits are bounded and report like the collectives'.
template <int P>
__global__ __launch_bounds__(512) void k_probe_exchange(KArgs ka) {
  const KArgs a = pin_args(ka);
  const uint64_t t_start = stamp_start(a);
  const uint32_t r = blockIdx.x % P;
  const uint32_t w = blockIdx.x / P;
  const uint32_t q = (uint32_t)uniform_u32(threadIdx.x >> 6);
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t units = (uint32_t)a.units;
  const uint32_t u = w * 64 + lane;
  const uint32_t in_bytes = (uint32_t)a.n;  // a.n: input bytes per rank
  const rsrc_t in_rs = make_rsrc(a.sym + (uint64_t)r * a.stride, in_bytes);
  const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(in_rs, (int)(u * 8), 0, 0);
  constexpr uint32_t kNowhere = 0xFFFFFFF0u;
  const uint32_t slot = (uint32_t)a.slot;
  const bool publish = q != r && u < units;
  const rsrc_t rd = make_rsrc(a.sym + a.area + (uint64_t)q * a.stride + (r - (r > q ? 1u : 0u)) * slot, slot);
  st_pkt(rd, publish ? u * 16 : kNowhere, u32x4{x.x, a.epoch, x.y, a.epoch});
  WaitBudget budget(a.timeout, a.status);
  u32x2 v = x;
  if (q != r) {
    const rsrc_t rs = make_rsrc(a.sym + a.area + (uint64_t)r * a.stride + (q - (q > r ? 1u : 0u)) * slot, slot);
    bool pend = u < units;
    uint32_t spins = 0;
    while (true) {
      compiler_fence();
      const u32x4 pk = ld_pkt(rs, u * 16);
      if (pend && pk.y == a.epoch && pk.w == a.epoch) {
        v = u32x2{pk.x, pk.z};
        pend = false;
      }
      if (__builtin_amdgcn_ballot_w64(pend) == 0) break;
      if ((++spins & 15) == 0 && budget.expired()) {
        if (pend) budget.report((int)r, 1u << q, a.epoch);
        break;
      }
    }
    if (a.clear != 0 && u < units) st_pkt(rs, u * 16, u32x4{0u, 0u, 0u, 0u});
  }
  const rsrc_t out_rs = make_rsrc(a.out + (uint64_t)r * in_bytes, in_bytes);
  __builtin_amdgcn_raw_buffer_store_b64(v, out_rs, (int)(u * 8), 0, kNT);
  stamp_end(a, t_start);
}

}  // namespace llc
