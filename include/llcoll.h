/*
 * llcoll -- barrier-free low-latency collectives for one MI355X (gfx950).
 *
 * C ABI.  Every entry point takes plain pointers and sizes; device pointers
 * are HIP device addresses, `stream` is a hipStream_t passed as void* (NULL =
 * the null stream).  No call allocates, frees or synchronises, except
 * ll_check (which synchronises the stream it is given).  Every call checks its
 * arguments before it touches the HIP runtime, so argument errors are
 * reported the same way with or without a GPU.
 *
 * The method (the paper's Secs. III-V): an AllReduce in which every rank
 * pushes its data into peers' scratch ("push mode", Sec. III-A), and
 * receivers detect arrival from a flag packed into the same store as the data
 * (the LL protocol, Sec. IV), so no memory barrier is needed between ranks.
 * One-shot: every rank sends its whole input to every peer and reduces all P
 * contributions itself.  Two-shot: ReduceScatter (each rank reduces one
 * chunk) followed by AllGather of the reduced chunks (Sec. III-A).
 *
 * Virtual ranks.  The P ranks live on one GPU: rank r owns the slice
 * [sym_base + r*rank_stride, sym_base + (r+1)*rank_stride) of a single
 * symmetric allocation, and is served by its own workgroups.  Rank r's data
 * reaches another rank only through flagged packets written into that rank's
 * slice; no rank reads another rank's input.
 *
 * Slice layout (a pure function of rank_stride and nranks, identical for
 * every call on a region, so a byte's role never changes between calls):
 *   [0, cap)                      input area: the rank's input, at offset 0
 *   [cap, cap + A8)               8-byte packet area {payload u32, flag u32}
 *   [cap + A8, cap + A8 + A128)   128-byte line area
 *   [.., .. + AA)                 binary32 accumulators and tile counters (atomic two-shot)
 *   [.., .. + AS)                 sentinel area (payload only)
 * A region holds the areas of a set of packet formats, encoded in its
 * stride: (rank_stride / 256) mod 16 has one bit per format (LL_FMT_*), and
 * 0 means all of them, so every stride that is a multiple of 4 KiB holds all
 * formats.  ll_slice_bytes returns such a stride for LL_ALGO_AUTO and, for a
 * named algorithm, the smaller stride of a region that holds that
 * algorithm's format only.  cap (the input capacity, a multiple of 256
 * bytes) is the largest input for which the present areas fit every
 * algorithm of their format; ll_input_capacity reports it.  A call whose
 * packet format the region does not hold returns LL_ERR_SCRATCH.
 *
 * Element types: binary32 and bfloat16.  The reduction is the sum of the P
 * inputs in ascending rank order, accumulated in binary32, rounded once to the
 * element type (round to nearest even).  Results are therefore identical on
 * every rank and for every algorithm and launch shape.
 *
 * Epochs.  The flag carried by every packet is the caller's `epoch`, which
 * must be >= 1 and must strictly increase over all calls on one region (any
 * entry point); 0 marks zeroed scratch (ll_init).  Sentinel-mode calls check
 * the epoch like the others but do not use it.  After epoch 0xFFFFFFFF,
 * call ll_init again and restart at 1.  (The paper's buffer object keeps this
 * counter internally and advances it itself, Sec. V; here the caller owns it.)
 * A call captured into a HIP graph keeps the epoch it was captured with, so
 * every replay repeats it: reset the region (ll_init, or ll_scratch_init for
 * a bounded-scratch region) on the replay stream before each replay after
 * the first.  ll_allreduce_static takes its epochs when it is called, so a
 * captured static call may be replayed once.
 *
 * Outputs.  `out` is a separate device buffer (it must not overlap the
 * symmetric region) holding the P per-rank outputs back to back:
 *   AllReduce      rank r's result at out + r*count*esize
 *   ReduceScatter  rank r's chunk  at out + r*recvcount*esize
 *   AllGather      rank r's result at out + r*nranks*sendcount*esize
 *
 * Ownership.  The caller allocates and frees the symmetric region and `out`,
 * and keeps them alive until the stream has run the call.  The library keeps
 * no per-region state and no settings: what a call does depends on its
 * arguments only (and on its ll_options, for the entry points that take
 * them).  Its only global state is a lazily built, thread-safe table of
 * kernels and device properties and, per device, the status words of the
 * streams that ran calls.  Two calls on one region must not run concurrently
 * (use one stream per region).
 *
 * Failure.  Every wait on a flag is bounded (ll_options.poll_timeout,
 * default 2 s).  A wait that expires records LL_ERR_TIMEOUT in the status
 * word of the stream the call runs on and lets the kernel finish; ll_check
 * on that stream reports it.  The outputs of such a call are undefined.
 */
#ifndef LLCOLL_H
#define LLCOLL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { LL_F32 = 0, LL_BF16 = 1 } ll_dtype;
typedef enum { LL_SUM = 0 } ll_op;

/* AllReduce algorithm.  *_LINE variants carry 120 payload bytes per 128-byte
 * line instead of 4 per 8-byte packet. */
typedef enum {
  LL_ALGO_AUTO = 0,          /* chosen by message size */
  LL_ALGO_ONESHOT = 1,       /* one-shot, 8-byte packets (Sec. III-A, Sec. IV "LL") */
  LL_ALGO_TWOSHOT = 2,       /* two-shot (ReduceScatter + AllGather), 8-byte packets */
  LL_ALGO_TWOSHOT_LINE = 3,  /* two-shot, 128-byte line packets */
  LL_ALGO_ONESHOT_LINE = 4,  /* one-shot, 128-byte line packets */
  LL_ALGO_ONESHOT_WAVES = 5,  /* one-shot, 8-byte packets, one wave per peer, LDS staging */
  LL_ALGO_ONESHOT_SENTINEL = 6, /* one-shot, sentinel synchronisation (Sec. IV, "Sentinel") */
  LL_ALGO_TWOSHOT_SENTINEL = 7, /* two-shot, sentinel synchronisation */
  LL_ALGO_TWOSHOT_SENTINEL_OUT = 8, /* two-shot, sentinel; AllGather straight into the
                                       peers' sentinel-filled outputs (see ll_fill_sentinel) */
  LL_ALGO_TWOSHOT_ATOMIC = 9,       /* two-shot with atomic accumulation (Sec. IV, "LL128
                                       Atomic"): NOT deterministic, see below */
  LL_ALGO_TWOSHOT_WAVES = 10,       /* two-shot, 8-byte packets, one wave per peer, partial
                                       sums staged in LDS */
  LL_ALGO_TWOSHOT_SENTINEL_WAVES = 11, /* the same with sentinel units */
  LL_ALGO_ONESHOT_SENTINEL_WAVES = 12, /* one-shot, sentinel units, one wave per peer (single
                                          iteration only) */
  LL_ALGO_ONESHOT_LINE_WAVES = 13,     /* one-shot, 128-byte lines, one wave per peer */
  LL_ALGO_TWOSHOT_LINE_WAVES = 14      /* two-shot, 128-byte lines, one wave per peer */
} ll_algo;

/* LL_ALGO_TWOSHOT_ATOMIC, the analogue of the paper's two-shot LL128 atomic
 * AllReduce.  Every rank adds its chunk c, widened to binary32, into an
 * accumulator in rank c's slice with device-scope float atomic adds.  The
 * chip does not add a 128-byte line atomically, so the paper's in-line flag
 * becomes a per-tile counter (one per 1 KiB of chunk input) that each rank
 * bumps after its adds, with release ordering.  The owner waits until the
 * counter reaches nranks, rounds once and stores the result into every
 * rank's output.  Scratch per slice is about 2*count*esize/nranks.
 * Preconditions and errors are those of LL_ALGO_TWOSHOT_SENTINEL_OUT:
 * sentinel-filled outputs and count*esize % 16 == 0.  The summation order
 * depends on timing, so results differ from the ordered sum by up to
 * gamma_{P-1} * sum |x_i| (binary32, end of Sec. IV), plus one rounding to
 * bfloat16.  Every rank receives the same bits.  Not available through
 * ll_allreduce_buffered, and never chosen by AUTO. */

/* Packet format for the stand-alone ReduceScatter / AllGather. */
typedef enum { LL_PROTO_AUTO = 0, LL_PROTO_PACKET8 = 1, LL_PROTO_LINE128 = 2, LL_PROTO_SENTINEL = 3 } ll_proto;

/* Sentinel mode (LL_ALGO_*_SENTINEL, LL_PROTO_SENTINEL).  Receive slots hold
 * the dword 0xFFFFFFFF until payload overwrites them; the receiver polls until
 * every dword differs from it and then writes the sentinel back.  Payload
 * travels without flags (4 bytes of payload per 4 bytes stored).  Input data
 * must not contain the dword 0xFFFFFFFF (binary32: that negative NaN;
 * bfloat16: two adjacent 0xFFFF negative NaNs starting at an even index);
 * such a call times out (LL_ERR_TIMEOUT) instead of completing.  After a
 * timed-out call, ll_init restores the sentinels.
 *
 * LL_ALGO_TWOSHOT_SENTINEL_OUT keeps only the ReduceScatter slots in scratch
 * (Table I: scratch D rather than 2D): the owner of each chunk stores the
 * reduced chunk directly into every peer's output, and each rank polls its
 * own output until those blocks no longer hold the sentinel (Sec. IV, the
 * sentinel-initialised output of the two-shot variants).  Preconditions:
 * every element of the nranks*count outputs holds the sentinel
 * (ll_fill_sentinel on the same stream, once before every call), and
 * count*esize is a multiple of 16 (else LL_ERR_UNSUPPORTED).  A call on an
 * output that was not refilled may return the previous call's blocks. */

/* Status codes. */
#define LL_OK 0
#define LL_ERR_INVALID -1     /* null pointer, nranks outside [2,8], misaligned pointer or
                                 stride, epoch 0, out overlapping the region, bad enum value */
#define LL_ERR_UNSUPPORTED -2 /* dtype or op not supported */
#define LL_ERR_SCRATCH -3     /* input larger than the region's input capacity */
#define LL_ERR_HIP -4         /* the HIP runtime reported an error (see ll_strerror) */
#define LL_ERR_TIMEOUT -5     /* a flag wait expired (reported by ll_check) */

#define LL_MAX_RANKS 8
#define LL_ALIGN 256

/* Packet formats a region holds: bits of (rank_stride / 256) mod 16, where 0
 * means all formats. */
#define LL_FMT_PACKET8 1u   /* 8-byte packets */
#define LL_FMT_LINE128 2u   /* 128-byte lines */
#define LL_FMT_SENTINEL 4u  /* sentinel units */
#define LL_FMT_ATOMIC 8u    /* binary32 accumulators of LL_ALGO_TWOSHOT_ATOMIC */

/* Per-call options of the *_ex entry points (and ll_broadcast, ll_reduce,
 * ll_allreduce_buffered).  NULL means the defaults, which are also what the
 * entry points without options use.  Fill with ll_options_init, then set
 * fields. */
typedef struct ll_tuning ll_tuning; /* benchmark and test hooks: include/lltune.h */
typedef struct {
  uint32_t size;            /* sizeof(ll_options), set by ll_options_init */
  uint32_t flags;           /* LL_OPT_* bits; default 0 */
  uint64_t poll_timeout;    /* bound of every flag wait, in ticks of the 100 MHz
                               constant clock; 0 = the default, 2e8 (2 s) */
  const ll_tuning *tuning;  /* launch-shape and test hooks; NULL = none */
} ll_options;

/* The automatic choices (LL_ALGO_AUTO, LL_PROTO_AUTO) may use sentinel mode:
 * for callers whose data never holds the sentinel dword (see below).  Never
 * selects LL_ALGO_TWOSHOT_SENTINEL_OUT. */
#define LL_OPT_AUTO_SENTINEL 0x1u
/* The automatic choices never use 128-byte line packets, whose correctness
 * rests on a measured, not a guaranteed, property of the chip (a 64-byte
 * half of a line is never seen torn across XCDs): they take the 8-byte-packet
 * algorithm of the same shape instead.  Named line algorithms still run. */
#define LL_OPT_NO_LINES 0x2u

int ll_options_init(ll_options *opt);

/* Minimum rank_stride (bytes, multiple of 256) of a region whose input
 * capacity holds `count` elements of `dt` for nranks ranks and `algo`.
 * `count` is the per-rank input length of the largest call the region will
 * serve: count for AllReduce, nranks*recvcount for ReduceScatter, sendcount
 * for AllGather.  algo = LL_ALGO_AUTO sizes a region for every algorithm and
 * packet format (a multiple of 4 KiB); a named algorithm sizes it for that
 * algorithm's packet format only (the region then serves every call in that
 * format: ReduceScatter, AllGather, Broadcast and Reduce in it too, and AUTO
 * chooses within it).  This is the host-side sizing helper of Sec. V
 * ("Host-side Functions"). */
int ll_slice_bytes(size_t count, ll_dtype dt, int nranks, ll_algo algo, size_t *min_rank_stride);

/* Input capacity in bytes of a region with this rank_stride and rank count. */
int ll_input_capacity(size_t rank_stride, int nranks, size_t *capacity_bytes);

/* Byte offsets, within every slice, of the areas of the slice layout:
 * offsets6 = {input area (0), 8-byte packet area, line area, atomic
 * accumulator area, sentinel area, end of the sentinel area}; an area the
 * region does not hold is empty.  Host-only; errors as ll_input_capacity. */
int ll_slice_layout(size_t rank_stride, int nranks, size_t *offsets6);

/* Zero both flagged packet areas and the accumulator area of every slice
 * (flag 0 = nothing received) and fill the sentinel area with the sentinel,
 * on `stream`.  Call once after allocating a region, and again before reusing it
 * after epoch 0xFFFFFFFF or after a timed-out call.  Sec. V: the LL reset
 * value is zero. */
int ll_init(void *sym_base, size_t rank_stride, int nranks, void *stream);

/* Set the nranks*count elements of `out` (16-byte aligned device memory) to
 * the sentinel of `dt` (every byte 0xFF), on `stream`: the precondition of
 * LL_ALGO_TWOSHOT_SENTINEL_OUT (Sec. V, sentinel initialisation). */
int ll_fill_sentinel(void *out, size_t count, ll_dtype dt, int nranks, void *stream);

/* AllReduce (sum) of `count` elements per rank, algorithm chosen by size.
 * Input of rank r: sym_base + r*rank_stride, count elements.  One kernel
 * launch on `stream`; returns after enqueueing. */
int ll_allreduce(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt,
                 ll_op op, int nranks, uint32_t epoch, void *stream);

/* Same, with the algorithm named. */
int ll_allreduce_algo(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt,
                      ll_op op, int nranks, uint32_t epoch, void *stream, ll_algo algo);

/* Same, with per-call options (opt may be NULL). */
int ll_allreduce_ex(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op,
                    int nranks, uint32_t epoch, void *stream, ll_algo algo, const ll_options *opt);

/* The algorithm that LL_ALGO_AUTO runs for a single-call AllReduce of
 * `count` elements of `dt` per rank over `nranks` ranks on a region whose
 * stride is `rank_stride` (0: a region of every packet format), with options
 * `opt` (may be NULL), written to *algo.  The choice follows measured
 * crossovers on the MI355X: one-shot with one wave per peer for small
 * messages, the two-shot wave kernels for medium ones, the line two-shot for
 * large ones; within the region's packet formats and the options.  Host
 * only, no HIP call.  LL_ERR_INVALID: algo NULL or nranks outside [2, 8];
 * LL_ERR_UNSUPPORTED: unknown dtype; LL_ERR_SCRATCH: the region holds no
 * format AUTO may use. */
int ll_auto_algo(size_t count, ll_dtype dt, int nranks, size_t rank_stride, const ll_options *opt, ll_algo *algo);

/* ReduceScatter (sum): rank r's input is nranks*recvcount elements; rank r
 * receives elements [r*recvcount, (r+1)*recvcount) of the sum (Sec. III-A). */
int ll_reduce_scatter(void *sym_base, size_t rank_stride, void *out, size_t recvcount,
                      ll_dtype dt, ll_op op, int nranks, uint32_t epoch, void *stream);
/* Same, with the packet format named and per-call options (opt may be NULL). */
int ll_reduce_scatter_ex(void *sym_base, size_t rank_stride, void *out, size_t recvcount, ll_dtype dt,
                         ll_op op, int nranks, uint32_t epoch, void *stream, ll_proto proto,
                         const ll_options *opt);

/* AllGather: rank r's input is sendcount elements; every rank receives the
 * concatenation of all inputs in rank order (Sec. III-A). */
int ll_allgather(void *sym_base, size_t rank_stride, void *out, size_t sendcount, ll_dtype dt,
                 int nranks, uint32_t epoch, void *stream);
/* Same, with the packet format named and per-call options (opt may be NULL). */
int ll_allgather_ex(void *sym_base, size_t rank_stride, void *out, size_t sendcount, ll_dtype dt,
                    int nranks, uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt);

/* ---- bounded scratch: multi-iteration AllReduce with double buffering ----
 *
 * Sec. IV ("Bidirectional Communication & Double Buffering") and Sec. V
 * (round-robin sub-buffers).  The inputs live outside the scratch region:
 * rank r's input is `count` elements at in + r*count*esize, its output at
 * out + r*count*esize (in == out is an in-place AllReduce).  The scratch
 * region is nranks slices of scratch_stride bytes; each slice holds, per
 * packet format, two sub-buffers for an iteration of D bytes per rank
 * (ll_scratch_iter_bytes).  A call of M = count*esize bytes per rank runs in
 * k = ceil(M / D) iterations inside one kernel: iteration i moves elements
 * [i*D/esize, (i+1)*D/esize) of every rank through sub-buffer i % 2 with the
 * flag epoch + i.  No barrier separates iterations: a lane writes a peer's
 * sub-buffer again only after it has received that peer's packets of the
 * previous iteration, which the peer sends only after it has read the
 * sub-buffer (each receive is the credit for the next send).  In sentinel
 * mode every lane also waits for its slot resets to be acknowledged before
 * the next iteration.
 *
 * Epochs: such a call uses the k epochs epoch .. epoch+k-1 (*epochs_used =
 * k, 0 when count is 0); the next call on the same scratch region must use an
 * epoch above epoch+k-1.  Packet areas are never shared with a region of the
 * other kind: scratch regions have their own init (ll_scratch_init). */

/* Minimum scratch_stride (bytes, multiple of 256) for iterations of
 * `iter_bytes` bytes per rank (1 .. 256 MiB). */
int ll_scratch_bytes(size_t iter_bytes, int nranks, size_t *min_scratch_stride);

/* Iteration size D (bytes per rank, a multiple of 256) of a scratch region;
 * LL_ERR_SCRATCH if the stride holds no iteration at all. */
int ll_scratch_iter_bytes(size_t scratch_stride, int nranks, size_t *iter_bytes);

/* Zero the flagged sub-buffers and fill the sentinel sub-buffers of every
 * scratch slice, on `stream`.  Call after allocating, after epoch
 * 0xFFFFFFFF, and after a timed-out call. */
int ll_scratch_init(void *scratch_base, size_t scratch_stride, int nranks, void *stream);

/* AllReduce (sum) through a bounded scratch region.  in, out: 16-byte
 * aligned device memory, equal (in place) or disjoint, neither overlapping
 * the scratch region; scratch_base 256-byte aligned.  algo as for
 * ll_allreduce_algo (the one-shot wave-per-peer algorithms only for one
 * iteration; LL_ALGO_TWOSHOT_SENTINEL_OUT not in place; not
 * LL_ALGO_TWOSHOT_ATOMIC).  count*esize at most 16 GiB.
 * epochs_used may be NULL.  One kernel launch on `stream`. */
int ll_allreduce_buffered(const void *in, void *out, size_t count, ll_dtype dt, ll_op op, int nranks,
                          void *scratch_base, size_t scratch_stride, uint32_t epoch, void *stream, ll_algo algo,
                          const ll_options *opt, uint32_t *epochs_used);

/* ---- no allocation: AllReduce through a scratch the library holds ----
 *
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).
 * ll_allreduce_static is ll_allreduce_buffered with the scratch region held
 * by the library: a file-scope device array of LL_STATIC_SCRATCH_BYTES per
 * GPU, laid out for LL_MAX_RANKS slices, allocated when the library's code is
 * loaded on a GPU and held until the process ends.  The call itself
 * allocates nothing (no hipMalloc, hipFree or allocating library routine) and
 * takes no epoch: the library keeps one epoch counter per GPU for that GPU's
 * array.  The first call on a GPU, and the first call after ll_check has
 * reported a timeout on that GPU, first clears the array's flag areas with a
 * fill kernel on `stream`.
 *
 * in, out, count, dt, op, nranks, epochs_used: as ll_allreduce_buffered; in
 * and out are 16-byte aligned device memory, equal (in place) or disjoint.
 * algo: LL_ALGO_AUTO (flagged protocols only) or a flagged algorithm
 * (8-byte packets or 128-byte lines); sentinel and atomic algorithms return
 * LL_ERR_UNSUPPORTED (a timed-out sentinel call leaves slots only an
 * ll_init-style reset restores).  Messages of any size up to 16 GiB per
 * rank run in iterations of the array's iteration size; larger ones return
 * LL_ERR_UNSUPPORTED.
 *
 * Every call on a GPU shares that GPU's array, which keeps the last call's
 * packets: calls that overlap in time on one GPU (two streams, two threads)
 * race and their results are undefined.  Serialise them. */
#define LL_STATIC_SCRATCH_BYTES (64u << 20)

int ll_allreduce_static(const void *in, void *out, size_t count, ll_dtype dt, ll_op op, int nranks, void *stream,
                        ll_algo algo, uint32_t *epochs_used);

/* Broadcast: every rank receives the root's `count` input elements; rank r's
 * copy at out + r*count*esize (the root's own copy included).  One exchange:
 * the root stores packets into one slot of every peer (the paper lists
 * Broadcast among the collectives built from the same primitives, Sec. V).
 * root in [0, nranks).  proto as for ReduceScatter (AUTO: 8-byte packets up
 * to 64 KiB, then lines, or sentinel when allowed); opt may be NULL. */
int ll_broadcast(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, int root, int nranks,
                 uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt);

/* Reduce (sum): the root receives the AllReduce result, `count` elements at
 * `out` (only the root's result is written).  Every other rank stores its
 * input as packets into its slot of the root, which sums in ascending rank
 * order and rounds once, as ll_allreduce. */
int ll_reduce(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op, int root,
              int nranks, uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt);

/* Synchronise `stream`, then report and clear the status word of that stream
 * (the word its calls' timed-out waits report into): LL_OK, LL_ERR_TIMEOUT,
 * or LL_ERR_HIP.  Calls on other streams are not seen.  A stream keeps its
 * status word for the life of the process; beyond 256 streams per device,
 * later streams share words. */
int ll_check(void *stream);

/* Details of the last timeout ll_check reported in the calling thread: rank,
 * the bit mask of peers not heard from, and the epoch waited for.  Any
 * pointer may be NULL. */
int ll_last_timeout(int *rank, uint32_t *missing_peers, uint32_t *epoch);

/* Human-readable text for a status code. */
const char *ll_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* LLCOLL_H */
