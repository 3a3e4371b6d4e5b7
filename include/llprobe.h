/*
 * llcoll measurement probes -- C ABI (same library as llcoll.h).
 *
 * These kernels measure what the collectives are judged against:
 *
 *  - The single-GPU latency floor: an empty kernel and a "floor" kernel (one
 *    dependent HBM round trip) launched with the collective's grid.  A small
 *    AllReduce on one GPU cannot finish faster than launching a kernel and
 *    waiting for one memory round trip.
 *  - The pieces of the paper's speed-of-light model (Sec. VI): the latency of
 *    a fence (the paper's L2 round-trip proxy), of a coherent load, and of a
 *    ping-pong between two workgroups on different XCDs (the single-chip
 *    stand-in for the GPU-to-GPU ping-pong), from which
 *    L_remote_store = (L_ping_pong - 2 L_L2_RTT) / 2 and
 *    L_SoL = 2 L_L2_RTT + L_remote_store.
 *  - Chip facts the packet formats rely on: the workgroup-to-XCD map and a
 *    litmus test for torn packets across XCDs.
 *
 * All pointers are device pointers; `stream` is a hipStream_t (NULL = null
 * stream).  Every wait inside a probe is bounded.  Return codes are those of
 * llcoll.h.  Times are in ticks of the 100 MHz constant clock ("ticks") or
 * shader-clock cycles ("cycles").
 */
#ifndef LLPROBE_H
#define LLPROBE_H

#include <stddef.h>
#include <stdint.h>

#include "llcoll.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Empty kernel.  If stamps != NULL, workgroup b writes its start time to
 * stamps[b] and its end time to stamps[grid + b]. */
int ll_probe_empty(int grid, int threads, uint64_t *stamps, void *stream);

/* Floor kernel: lane 0 of workgroup 0 loads chase[start] and stores it to
 * sink[0]; every other workgroup exits at once.  stamps as above. */
int ll_probe_floor(const uint64_t *chase, uint64_t chase_len, uint64_t start, uint64_t *sink, int grid,
                   int threads, uint64_t *stamps, void *stream);

/* One lane follows idx = chase[idx] `steps` times from `start`.
 * out3 = {ticks, cycles, final idx}. */
int ll_probe_chase(const uint64_t *chase, uint64_t chase_len, uint64_t start, int steps, uint64_t *out3,
                   void *stream);

/* One lane, `iters` times each: store + agent-scope fence; dependent coherent
 * (sc1) load of one line; dependent sc0 load of one line.  buf4k: 4 KiB of
 * device memory whose dword 16 is zero.  out7 = {fence ticks, fence cycles,
 * sc1 ticks, sc1 cycles, sc0 ticks, sc0 cycles, sink}. */
int ll_probe_fence_l2(uint32_t *buf4k, int iters, uint64_t *out7, void *stream);

/* Ping-pong between workgroup 0 and workgroup `peer` of a `grid`-workgroup
 * launch, `rounds` exchanges; each wait gives up after limit_ticks.
 * flags8k: 8 KiB of zeroed device memory.  out3 = {ticks, exchanges
 * completed, cycles}. */
int ll_probe_pingpong(uint32_t *flags8k, int rounds, int grid, int peer, uint64_t limit_ticks, uint64_t *out3,
                      void *stream);

/* A single lane that waits `ticks` (1 .. 1e8, i.e. at most 1 s) and exits.
 * Launched first, it holds the stream while the host queues the launches to
 * be timed, which then run back to back at the GPU's own pace. */
int ll_probe_spin(uint64_t ticks, void *stream);

/* Back-to-back launch loops run from C (so the host is never the bottleneck).
 *
 * ll_bench_allreduce: `calls` AllReduces (ll_allreduce_ex with op = sum) with
 * epochs first_epoch .. first_epoch+calls-1 and options `opt` (may be NULL).
 * If stamps != NULL, call i writes its per-workgroup start/end times at
 * stamps + i*stamp_stride (see ll_tuning.stamps; stamp_stride >= 2*grid).
 * ll_bench_reduce_scatter / ll_bench_allgather: the same for the stand-alone
 * collectives (proto as ll_proto).
 * ll_bench_floor: `calls` floor kernels; call i loads line
 * (first_line + i*line_step) mod (chase_len/16) of `chase` (16 words a line).
 * ll_bench_empty: `calls` empty kernels. */
int ll_bench_allreduce(void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int nranks,
                       uint32_t first_epoch, int calls, int algo, const ll_options *opt, uint64_t *stamps,
                       int stamp_stride, void *stream);
int ll_bench_reduce_scatter(void *sym_base, size_t rank_stride, void *out, size_t recvcount, int dt, int nranks,
                            uint32_t first_epoch, int calls, int proto, const ll_options *opt, uint64_t *stamps,
                            int stamp_stride, void *stream);
int ll_bench_allgather(void *sym_base, size_t rank_stride, void *out, size_t sendcount, int dt, int nranks,
                       uint32_t first_epoch, int calls, int proto, const ll_options *opt, uint64_t *stamps,
                       int stamp_stride, void *stream);
/* ll_bench_rooted: `calls` Broadcasts (kind 0) or Reduces (kind 1). */
int ll_bench_rooted(int kind, void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int root,
                    int nranks, uint32_t first_epoch, int calls, int proto, const ll_options *opt,
                    uint64_t *stamps, int stamp_stride, void *stream);
int ll_bench_floor(const uint64_t *chase, uint64_t chase_len, uint64_t first_line, uint64_t line_step,
                   uint64_t *sink, int grid, int threads, int calls, uint64_t *stamps, int stamp_stride,
                   void *stream);
int ll_bench_empty(int grid, int threads, int calls, uint64_t *stamps, int stamp_stride, void *stream);

/* Minimal-exchange probe: `calls` launches, epochs first_epoch ..
 * first_epoch+calls-1, of a kernel with the grid and packet volume of the
 * one-shot AllReduce with one wave per peer and 8-byte packets (LL_ALGO_
 * ONESHOT_WAVES, one unit per lane) on `count` elements of `dt` per rank:
 * per wave one input load, one coherent 16-byte packet store per lane to one
 * peer, a poll of that peer's packets, one output store; no LDS, barrier or
 * sum.  It moves the data the one-shot must move and nothing else, so its
 * call-to-call interval bounds the one-shot's from below (see the probe
 * kernel).  The region is an AllReduce region of at least `count`
 * elements (its 8-byte packet slots are used); count*esize must be a
 * positive multiple of 8 and fit one tile per workgroup with every
 * workgroup resident.  out receives nranks*count elements: each element of
 * rank r's output equals that element of some rank's input.  stamps as for
 * ll_bench_allreduce; grid_out (NULL or host memory) receives the grid. */
int ll_bench_exchange(void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int nranks,
                      uint32_t first_epoch, int calls, uint64_t *stamps, int stamp_stride, int *grid_out,
                      void *stream);

/* ids[b] = XCD index of workgroup b. */
int ll_probe_xcd(uint32_t *ids, int grid, int threads, void *stream);

/* Streaming bandwidth: a grid-stride kernel over bytes/16 16-byte words with
 * non-temporal loads and stores.  mode 0 copies src to dst, mode 1 only reads
 * src (dst must hold at least 16 bytes and is normally left untouched), mode 2
 * only writes dst (src unused, may be NULL).  bytes > 0 and a multiple of 16;
 * src and dst 16-byte aligned and bytes long; grid 1..65536, threads a
 * multiple of 64 up to 1024.  Sweeping grid gives the HBM bandwidth that a
 * simple streaming kernel reaches, the practical ceiling under the published
 * peak. */
int ll_probe_stream(const void *src, void *dst, size_t bytes, int mode, int grid, int threads, void *stream);

/* Torn-packet litmus across XCDs.  grid/2 writer workgroups each rewrite
 * `lines` 128-byte lines `iters` times; grid/2 reader workgroups read another
 * writer's lines `reads` times.  layout 0 = 8-byte packets, 1 = 128-byte lines
 * with a flag per 64-byte half.  buf: zeroed, >= grid/2 * lines * 128 bytes.
 * counts4 (zeroed) = {units seen, torn units, 16-byte loads with two different
 * flags, lines with two different half flags}. */
int ll_probe_litmus(uint32_t *buf, size_t buf_bytes, int grid, int lines, int iters, int reads, int layout,
                    unsigned long long *counts4, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LLPROBE_H */
