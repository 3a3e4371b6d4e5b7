/*
 * llcoll benchmark and test hooks -- C ABI (same library as llcoll.h).
 *
 * Nothing here is needed to use the collectives.  These calls expose the
 * library's host-side planning for the tests that check it on the CPU.
 */
#ifndef LLTUNE_H
#define LLTUNE_H

#include <stddef.h>
#include <stdint.h>

#include "llcoll.h"

#ifdef __cplusplus
extern "C" {
#endif

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
