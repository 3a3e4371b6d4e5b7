/*
 * llcoll benchmark and test hooks -- C ABI (same library as llcoll.h).
 *
 * Nothing here is needed to use the collectives.  ll_tuning holds the
 * launch-shape and test hooks a benchmark or a test passes to one call,
 * through ll_options.tuning; the library keeps none of it between calls.
 * The other functions expose the library's host-side planning for the tests
 * that check it on the CPU.
 */
#ifndef LLTUNE_H
#define LLTUNE_H

#include <stddef.h>
#include <stdint.h>

#include "llcoll.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Launch-shape and test hooks of one call (ll_options.tuning).  Results never
 * depend on the launch-shape fields; the test hooks change only what they
 * name.  Fill with ll_tuning_init (every field off / automatic), then set
 * fields. */
struct ll_tuning {
  uint32_t size;            /* sizeof(ll_tuning), set by ll_tuning_init */
  int workgroups_per_rank;  /* 0 = automatic; never more than can be resident */
  int threads;              /* threads per workgroup of the one-lane kernels, a
                               multiple of 64 in [64, 1024]; 0 = automatic.
                               Either field set: the one-tile one-shot kernel
                               is not used. */
  int wave_units;           /* packet units per lane of the wave-per-peer
                               kernels: 1, 2 or 4; 0 = automatic */
  int wave_kernels;         /* stand-alone ReduceScatter / AllGather: 0 = by
                               size, 1 = one lane per unit, 2 = one wave per peer */
  int pipeline_lag;         /* two-shot distance between publish, reduce and
                               gather, in [0, 64]; -1 = the default (1) */
  int first_wait;           /* idle time before a lane's first poll, in units of
                               64 shader cycles, [0, 1000] */
  int poll_gap;             /* idle time between polls, same units */
  int mute_rank;            /* test hook: this rank publishes nothing, so its
                               peers' waits expire; -1 = off */
  int clear_slots;          /* whether the reader of a flagged packet slot
                               stores zeros back into it: 0 = by kernel and
                               size (the default), 1 = always (wave-per-peer
                               kernels), 2 = never */
  uint64_t *stamps;         /* device memory or NULL: each workgroup b writes its
                               start and end time (100 MHz ticks) to stamps[b]
                               and stamps[grid + b] */
  uint64_t *phases;         /* device memory or NULL: phase times of the wave
                               kernels, in a library built with
                               -DLLCOLL_WAVE_PHASES=1 (4*grid*nranks words: for
                               lane 0 of wave w of workgroup b, at
                               [4(b*nranks+w)]: one-shot: packet store issued,
                               [+1] peer's packets all seen, [+2] past the
                               workgroup barrier; two-shot AllReduce, the
                               workgroup's first tile: ReduceScatter packets
                               issued, [+1] peer's ReduceScatter packets seen,
                               [+2] past the barrier, [+3] peer's AllGather
                               packets seen); ignored otherwise */
  int *grid_out;            /* host memory or NULL: receives the launch's total
                               workgroups */
  int *threads_out;         /* host memory or NULL: receives its threads per
                               workgroup */
};

int ll_tuning_init(ll_tuning *t);

/* The iterations a bounded-scratch AllReduce (ll_allreduce_buffered) of
 * `count` elements of `dt` per rank runs through a scratch region of
 * `scratch_stride` bytes per slice: *iters iterations of *iter_count
 * elements (the last one may be shorter).  Host only.  Errors as
 * ll_allreduce_buffered's argument checks. */
int ll_buffered_plan(size_t count, ll_dtype dt, int nranks, size_t scratch_stride, uint32_t *iters,
                     size_t *iter_count);

/* Iteration `it` of a call of `count` elements per rank in iterations of
 * `iter_count` elements, as every kernel computes it: out3 = {first element,
 * elements in the iteration, two-shot chunk length in elements}.  Host only. */
int ll_iteration_span(size_t count, size_t iter_count, uint32_t it, int nranks, ll_dtype dt, int64_t *out3);

#ifdef __cplusplus
}
#endif

#endif /* LLTUNE_H */
