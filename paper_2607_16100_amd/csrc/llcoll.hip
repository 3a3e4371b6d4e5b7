// C-ABI entry points of the llcoll library (declared in include/llcoll.h and
// include/llprobe.h): argument checking, slice layout, launch shape, kernel
// dispatch.  Argument checking happens before any HIP call.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <type_traits>

#include "../../include/llcoll.h"
#include "../../include/llprobe.h"
#include "../../include/lltune.h"
#include "ll_device.hpp"
#include "ll_fill.hpp"
#include "ll_iter.hpp"
#include "ll_layout.hpp"
#include "ll_probe.hpp"
#include "ll_table.hpp"

namespace llc {
// Status words, one per stream that has run a call (see status_of); each
// device holds its own copy of the array.
constexpr int kStatusSlots = 256;
__device__ uint32_t g_status[kStatusSlots][4];
}  // namespace llc

using namespace llc;
namespace L = llc::layout;

namespace {

// ---------------------------------------------------------------- per-call options
constexpr uint64_t kDefaultTimeout = 200000000ull;  // 2 s of the 100 MHz clock

// What one call runs with: its ll_options (and their ll_tuning) resolved
// against the defaults.  Nothing of it outlives the call.
struct CallOpts {
  uint32_t flags = 0;
  uint64_t timeout = kDefaultTimeout;
  int wg_per_rank = 0, threads = 0, wave_units = 0, wave_kernels = 0, lag = 1, first_wait = 0, poll_gap = 0;
  int clear_slots = 0;  // 0 = by kernel and size, 1 = always, 2 = never
  int mute = -1;
  uint64_t *stamps = nullptr, *phases = nullptr;
  int *grid_out = nullptr, *threads_out = nullptr;
  bool sentinel_ok() const { return (flags & LL_OPT_AUTO_SENTINEL) != 0; }
  bool lines_ok() const { return (flags & LL_OPT_NO_LINES) == 0; }
  bool forced_shape() const { return wg_per_rank != 0 || threads != 0; }
};

// Checks and resolves `o` (NULL = defaults); no HIP call.
int resolve_opts(const ll_options *o, CallOpts *c) {
  *c = CallOpts();
  if (o == nullptr) return LL_OK;
  if (o->size != sizeof(ll_options)) return LL_ERR_INVALID;
  if ((o->flags & ~(uint32_t)(LL_OPT_AUTO_SENTINEL | LL_OPT_NO_LINES)) != 0) return LL_ERR_INVALID;
  c->flags = o->flags;
  if (o->poll_timeout != 0) c->timeout = o->poll_timeout;
  const ll_tuning *t = o->tuning;
  if (t == nullptr) return LL_OK;
  if (t->size != sizeof(ll_tuning)) return LL_ERR_INVALID;
  if (t->workgroups_per_rank < 0 || t->workgroups_per_rank > 4096) return LL_ERR_INVALID;
  if (t->threads != 0 && (t->threads < 64 || t->threads > 1024 || t->threads % 64 != 0)) return LL_ERR_INVALID;
  if (t->wave_units != 0 && t->wave_units != 1 && t->wave_units != 2 && t->wave_units != 4) return LL_ERR_INVALID;
  if (t->wave_kernels < 0 || t->wave_kernels > 2) return LL_ERR_INVALID;
  if (t->pipeline_lag < -1 || t->pipeline_lag > 64) return LL_ERR_INVALID;
  if (t->first_wait < 0 || t->first_wait > 1000 || t->poll_gap < 0 || t->poll_gap > 1000) return LL_ERR_INVALID;
  if (t->mute_rank < -1 || t->mute_rank >= LL_MAX_RANKS) return LL_ERR_INVALID;
  if (t->clear_slots < 0 || t->clear_slots > 2) return LL_ERR_INVALID;
  c->wg_per_rank = t->workgroups_per_rank;
  c->threads = t->threads;
  c->wave_units = t->wave_units;
  c->wave_kernels = t->wave_kernels;
  c->lag = t->pipeline_lag < 0 ? 1 : t->pipeline_lag;
  c->first_wait = t->first_wait;
  c->poll_gap = t->poll_gap;
  c->mute = t->mute_rank;
  c->clear_slots = t->clear_slots;
  c->stamps = t->stamps;
  c->phases = t->phases;
  c->grid_out = t->grid_out;
  c->threads_out = t->threads_out;
  return LL_OK;
}

thread_local int t_last_hip = 0;
thread_local char t_msg[256];
struct TimeoutInfo {
  int rank = -1;
  uint32_t missing = 0, epoch = 0;
};
thread_local TimeoutInfo t_last_timeout;  // the last timeout this thread's ll_check saw
std::mutex g_mu;
std::mutex g_static_mu;  // the static scratch table (ll_allreduce_static)

// ---------------------------------------------------------------- kernels
constexpr int kWaveUnits[3] = {1, 2, 4};  // units per lane of the wave-per-peer kernels

const Table &table() {
  static const Table t = [] {
    Table x;
    memset(&x, 0, sizeof x);
    fill_table_p2(&x);
    fill_table_p3(&x);
    fill_table_p4(&x);
    fill_table_p5(&x);
    fill_table_p6(&x);
    fill_table_p7(&x);
    fill_table_p8(&x);
    return x;
  }();
  return t;
}

// Per-device facts, queried on first use: compute units, and the device
// address of that device's copy of the status array.
struct DevInfo {
  bool ok = false;
  int cus = 0;
  uint32_t *status = nullptr;
};
DevInfo g_dev[64];

int device_info(DevInfo *out, int *dev_out = nullptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  if (dev < 0 || dev >= 64) return LL_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_dev[dev].ok) {
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) {
      t_last_hip = (int)e;
      return LL_ERR_HIP;
    }
    void *st = nullptr;
    e = hipGetSymbolAddress(&st, HIP_SYMBOL(llc::g_status));
    if (e != hipSuccess) {
      t_last_hip = (int)e;
      return LL_ERR_HIP;
    }
    g_dev[dev].cus = cus;
    g_dev[dev].status = (uint32_t *)st;
    g_dev[dev].ok = true;
  }
  *out = g_dev[dev];
  if (dev_out) *dev_out = dev;
  return LL_OK;
}

// Status slots.  Every stream that runs a call owns one of the device's
// kStatusSlots status words: a kernel that times out reports into the word of
// its own stream, and ll_check(stream) reads and clears only that word, so
// calls on different streams (and different regions) report independently.
// A stream keeps its slot for the life of the process; if more than
// kStatusSlots streams of one device run calls, the later ones share slots
// (their timeouts may then be reported on either stream).
void *g_slot_owner[64][kStatusSlots];  // guarded by g_mu
bool g_slot_used[64][kStatusSlots];

int slot_index(int dev, void *stream, bool assign) {
  const uintptr_t h = ((uintptr_t)stream >> 4) * 0x9E3779B97F4A7C15ull;
  const int start = (int)((h >> 32) % kStatusSlots);
  std::lock_guard<std::mutex> lk(g_mu);
  for (int k = 0; k < kStatusSlots; ++k) {
    const int i = (start + k) % kStatusSlots;
    if (g_slot_used[dev][i] && g_slot_owner[dev][i] == stream) return i;
    if (!g_slot_used[dev][i]) {
      if (!assign) return -1;
      g_slot_used[dev][i] = true;
      g_slot_owner[dev][i] = stream;
      return i;
    }
  }
  return assign ? start : -1;  // every slot taken: share
}

// Device address of the status word of `stream` on the current device.
int status_of(void *stream, uint32_t **out) {
  DevInfo d;
  int dev = 0;
  const int st = device_info(&d, &dev);
  if (st != LL_OK) return st;
  *out = d.status + 4 * slot_index(dev, stream, true);
  return LL_OK;
}

// Workgroups of `fn` resident per CU with `threads` per workgroup, by device;
// filled on first use (one occupancy query per kernel shape and device).
std::map<std::tuple<int, const void *, int>, int> g_per_cu;  // guarded by g_mu

// Largest grid of `fn` that is resident at once with `threads` per workgroup.
int resident_grid(kernel_fn fn, int threads, int *grid_out) {
  DevInfo d;
  int st = device_info(&d);
  if (st != LL_OK) return st;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  const auto key = std::make_tuple(dev, reinterpret_cast<const void *>(fn), threads);
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_per_cu.find(key);
  if (it == g_per_cu.end()) {
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(fn), threads, 0);
    if (e != hipSuccess) {
      t_last_hip = (int)e;
      return LL_ERR_HIP;
    }
    it = g_per_cu.emplace(key, per_cu < 1 ? 1 : per_cu).first;
  }
  *grid_out = it->second * d.cus;
  return LL_OK;
}

inline int esize_of(ll_dtype dt) { return dt == LL_BF16 ? 2 : 4; }

int check_common(const void *sym_base, size_t rank_stride, const void *out, int nranks, uint32_t epoch) {
  if (sym_base == nullptr || out == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (((uintptr_t)sym_base % LL_ALIGN) != 0 || (rank_stride % LL_ALIGN) != 0 || rank_stride == 0) return LL_ERR_INVALID;
  if (((uintptr_t)out % 16) != 0) return LL_ERR_INVALID;
  if (epoch == 0) return LL_ERR_INVALID;
  return LL_OK;
}

int check_dtype_op(int dt, int op) {
  if (dt != LL_F32 && dt != LL_BF16) return LL_ERR_UNSUPPORTED;
  if (op != LL_SUM) return LL_ERR_UNSUPPORTED;
  return LL_OK;
}

bool overlaps(const void *a, uint64_t alen, const void *b, uint64_t blen) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + blen && b0 < a0 + alen;
}

struct Plan {
  Kind kind;
  Proto proto;
  int dt, P;
  KArgs a;
  int64_t units;  // packet units per stream
  CallOpts o;     // the call's options
  bool rooted_tile = false;  // Broadcast / Reduce on the one-tile kernel
};

// Launch shape of the two-shot AllReduce with one wave per peer, measured on
// MI355X (bfloat16, P = 2, 4, 6, 8, 128 KiB - 8 MiB per rank, p50 of
// back-to-back calls).  A workgroup has P waves, so a grid of G workgroups
// puts G P / CUs waves on a CU, of the 32 a CU holds.
//  1. The one-tile kernel (k_twoshot_tile: one unit per lane, one tile per
//     workgroup) is the fastest while its waves per CU stay at most 24 for
//     lines, 20 for sentinel units and 16 for 8-byte packets (and it needs
//     one iteration, 4-byte aligned streams, no forced launch shape, and
//     every tile resident at once).
//  2. Where the one-tile kernel could run but has too many waves, two units
//     per lane, in one round of at most 16 waves per CU (two workgroups of 8
//     waves), beats one unit per lane in more waves.
//  3. Otherwise the size rules of wave_units_log2.
// Whenever two units per lane result, lines take the one-tile kernel with
// two units per lane if its tiles are all resident (8 ranks, 1.5 MiB:
// 15.19 -> 14.48 us; 4 ranks, 3 MiB: 15.34 -> 13.04 us; 2 ranks, 4 MiB: 8.28
// -> 7.54 us); 8-byte packets and sentinel units keep the multi-tile kernel,
// which was as fast or faster for them at 4-8 ranks.  Against the best
// shape measured (one and two units per lane, one-tile and multi-tile
// kernels) the rule loses at most 0.3 us at 4-8 ranks; at 2 ranks and
// 4-8 MiB, where two units per lane in one tile would have been faster for
// 8-byte packets and sentinel units too, up to 0.8 us.
bool twoshot_tile_eligible(const Plan &pl) {
  const bool two = pl.kind == K_TWOSHOT_WAVES || pl.kind == K_RS_WAVES || pl.kind == K_AG_WAVES;
  return two && !pl.o.forced_shape() && pl.o.wave_units <= 2 && pl.a.al4 != 0 &&
         (pl.a.in == nullptr || pl.a.in_al4 != 0) && pl.a.iters <= 1;
}

// The one-tile kernel with 2^lu units per lane, if it can run this call:
// every tile resident, and (unless the units per lane are forced) within the
// waves-per-CU limit of rule 1 for one unit per lane.
bool twoshot_tile_ok(const Plan &pl, int wpr, int lu, kernel_fn *tf, int64_t *tiles) {
  if (!twoshot_tile_eligible(pl) || lu > 1) return false;
  const int mode = pl.kind == K_TWOSHOT_WAVES ? 0 : (pl.kind == K_RS_WAVES ? 1 : 2);
  kernel_fn f = table().ttile[mode][lu][wpr][pl.dt][pl.P];
  int cap = 0;
  DevInfo d;
  if (f == nullptr || resident_grid(f, 64 * pl.P, &cap) != LL_OK || device_info(&d) != LL_OK) return false;
  const int64_t blocks = pl.proto == PR_LINE ? pl.units : (pl.units + 63) / 64;
  const int64_t t = (blocks + (1 << lu) - 1) >> lu;
  if (t > cap / pl.P) return false;
  if (pl.o.wave_units == 0 && lu == 0) {
    const int64_t max_waves_per_cu = pl.proto == PR_LINE ? 24 : (pl.proto == PR_SENT ? 20 : 16);
    if (t * pl.P * pl.P > max_waves_per_cu * d.cus) return false;
  }
  *tf = f;
  *tiles = t;
  return true;
}

// Units per lane (U) of the wave-per-peer kernels, measured at 16 KiB ..
// 64 MiB per rank and 2 .. 8 ranks.  The two-shot AllReduce takes rules 1
// and 2 above first.  Otherwise one unit per lane, except in the two-shot
// AllReduce once its tiles would need a second round of workgroups, which
// costs a whole extra exchange:
//  - lines (a line unit is a whole wave): two units per lane once the P
//    tiles of a step hold more than 1200 line units, four once they hold
//    more than 8192 (from about 8 MiB per rank, where the kernel is bound by
//    bandwidth and fewer, longer waves move the bytes faster);
//  - 8-byte packets and sentinel units: two once a chunk has more tiles of
//    64 units than resident workgroups per rank.
// Elsewhere two units per lane are never more than about 3 % faster and up
// to 25 % slower.
int wave_units_log2(const Plan &pl, int wpr) {
  const int forced = pl.o.wave_units;
  if (forced == 1) return 0;
  if (forced == 2) return 1;
  if (forced == 4) return 2;
  if (pl.kind == K_RS_WAVES || pl.kind == K_AG_WAVES) {
    // stand-alone ReduceScatter / AllGather (measured at 4 and 8 ranks, C5
    // shapes, b = 1 .. 256): one unit per lane below 256 KiB of data per
    // rank; above, ReduceScatter two (8 ranks, lines, b = 64: 6.67 -> 5.55
    // us; b = 256: 17.51 -> 15.6 us), except at 2-4 ranks from 2 MiB, where
    // one stays faster (4 ranks, b = 256: 7.85 against 8.70 us); AllGather
    // four from 512 KiB if its workgroups then hold at most 16 waves per CU
    // (8 ranks, b = 128: 11.41 -> 10.09 us; 4 ranks, b = 256: 9.85 -> 9.28
    // us), otherwise two (8 ranks, b = 256: 23.3 us in the one-lane kernel,
    // 17.9 us).
    const uint64_t data = (uint64_t)pl.a.n * (pl.dt == LL_BF16 ? 2u : 4u) * (uint64_t)pl.P;
    const uint64_t KiB = 1024;
    if (data < 256 * KiB) return 0;
    if (pl.kind == K_RS_WAVES) return pl.P <= 4 && data >= 2048 * KiB ? 0 : 1;
    DevInfo d;
    const int64_t blocks = pl.proto == PR_LINE ? pl.units : (pl.units + 63) / 64;
    if (data >= 512 * KiB && device_info(&d) == LL_OK && (blocks + 3) / 4 * pl.P * pl.P <= 16 * (int64_t)d.cus)
      return 2;
    return 1;
  }
  if (pl.kind != K_TWOSHOT_WAVES) return 0;
  kernel_fn tf = nullptr;
  int64_t tiles = 0;
  if (twoshot_tile_ok(pl, wpr, 0, &tf, &tiles)) return 0;
  if (twoshot_tile_eligible(pl)) {
    DevInfo d;
    const int64_t blocks = pl.proto == PR_LINE ? pl.units : (pl.units + 63) / 64;
    if (device_info(&d) == LL_OK && (blocks + 1) / 2 * pl.P * pl.P <= 16 * (int64_t)d.cus) return 1;
  }
  if (pl.proto == PR_LINE) return pl.units * pl.P <= 1200 ? 0 : (pl.units * pl.P <= 8192 ? 1 : 2);
  int cap = 0;
  if (resident_grid(table().twaves[0][0][wpr][pl.dt][pl.P], 64 * pl.P, &cap) != LL_OK) return 1;
  return (pl.units + 63) / 64 <= cap / pl.P ? 0 : 1;
}

// Whether the reader of a flagged packet slot stores zeros back into it
// after reading it (KArgs::clear; sentinel slots are always reset).  A zero
// flag is never accepted, so the protocol is unchanged; what changes is
// timing.  Measured on MI355X, a slot that its reader has written back takes
// the next call's packets sooner: 0.26-0.34 us off the 16 KiB one-shot at 8
// ranks, 0.5-0.9 us off the 512 KiB-1 MiB line two-shot; but the stores cost
// bandwidth once a call is bound by it (the 8 MiB line two-shot at 8 ranks
// went from 59 to 70 us).  The crossover lies where the packet bytes of a
// call pass about 16 MiB, counted as (data per rank and iteration, the
// larger of input and output) x (P - 1) x (exchanges: 2 for the two-shot
// AllReduce, 1 for a stand-alone ReduceScatter or AllGather): measured at
// 2, 4 and 8 ranks for the AllReduce (1 / 2 / 8 MiB) and at 4 and 8 ranks
// for RS / AG (C5 shapes up to b = 512).  A call of several iterations
// must also wait at every iteration boundary for its clearing stores to be
// acknowledged, which costs more than clearing saves (32 MiB in 1 MiB
// iterations at 8 ranks: 339 -> 433 us).  So: on for the one-shot wave
// kernels, and for single-iteration two-shot and stand-alone RS / AG wave
// calls below that crossover.  The one-lane kernels never clear.
constexpr uint64_t kClearMaxBytes = 16ull << 20;

uint32_t clear_slots(const Plan &pl) {
  const bool waves = pl.kind == K_ONESHOT_WAVES || pl.kind == K_TWOSHOT_WAVES || pl.kind == K_RS_WAVES ||
                     pl.kind == K_AG_WAVES || pl.rooted_tile;
  if (!waves || pl.proto == PR_SENT || pl.o.clear_slots == 2) return 0;
  if (pl.o.clear_slots == 1 || pl.kind == K_ONESHOT_WAVES || pl.rooted_tile) return 1;
  if (pl.a.iters > 1) return 0;
  const uint64_t es = pl.dt == LL_BF16 ? 2 : 4;
  const uint64_t n = (uint64_t)(pl.a.iters > 1 ? pl.a.iter_n : pl.a.n);
  // AllReduce: n elements in and out; ReduceScatter: P*n in; AllGather: P*n out
  const uint64_t bytes = (pl.kind == K_TWOSHOT_WAVES ? 1 : (uint64_t)pl.P) * n * es;
  const uint64_t exchanges = pl.kind == K_TWOSHOT_WAVES ? 2 : 1;
  return bytes * (uint64_t)(pl.P - 1) * exchanges <= kClearMaxBytes ? 1u : 0u;
}

int launch_kernel(kernel_fn fn, const Plan &pl, int W, int threads, void *stream);

int launch(const Plan &pl, void *stream) {
  const bool two_waves = pl.kind == K_TWOSHOT_WAVES || pl.kind == K_RS_WAVES || pl.kind == K_AG_WAVES;
  const bool wave_kernel = pl.kind == K_ONESHOT_WAVES || two_waves;
  const int wpr = pl.proto == PR_SENT ? 1 : (pl.proto == PR_LINE ? 2 : 0);
  const int wlog = wave_kernel ? wave_units_log2(pl, wpr) : 0;
  kernel_fn fn = nullptr;
  if (pl.kind == K_ONESHOT_WAVES) {
    fn = table().waves[wlog][wpr][pl.dt][pl.P];
  } else if (two_waves) {
    const int mode = pl.kind == K_TWOSHOT_WAVES ? 0 : (pl.kind == K_RS_WAVES ? 1 : 2);
    fn = table().twaves[mode][wlog][wpr][pl.dt][pl.P];
  } else {
    fn = table().k[pl.proto][pl.dt][pl.P][pl.kind];
  }
  if (fn == nullptr) return LL_ERR_UNSUPPORTED;
  // The latency-bound one-shot: one tile per workgroup (64 one-lane units,
  // or one line unit), every stream 4-byte aligned, all tiles resident at
  // once, no forced launch shape -> the straight-line one-tile kernels.
  if (pl.kind == K_ONESHOT_WAVES && wlog == 0 && !pl.o.forced_shape() && pl.a.al4 != 0 &&
      (pl.a.in == nullptr || pl.a.in_al4 != 0) && pl.a.iters <= 1) {
    kernel_fn tf = table().tile[pl.proto == PR_SENT ? 1 : (pl.proto == PR_LINE ? 2 : 0)][pl.dt][pl.P];
    int cap = 0;
    const int rc = resident_grid(tf, 64 * pl.P, &cap);
    if (rc != LL_OK) return rc;
    const int64_t tiles = pl.proto == PR_LINE ? pl.units : (pl.units + 63) / 64;
    if (tf != nullptr && tiles <= cap / pl.P) return launch_kernel(tf, pl, (int)tiles, 64 * pl.P, stream);
  }
  // Broadcast / Reduce with a one-lane format under the same conditions:
  // the straight-line rooted kernel (one tile of 64 units per workgroup).
  if ((pl.kind == K_BCAST || pl.kind == K_REDUCE) && pl.proto != PR_LINE && !pl.o.forced_shape() &&
      pl.a.al4 != 0 && (pl.a.in == nullptr || pl.a.in_al4 != 0)) {
    kernel_fn tf = table().rtile[pl.proto == PR_SENT ? 1 : 0][pl.kind == K_BCAST ? 0 : 1][pl.dt][pl.P];
    int cap = 0;
    const int rc = resident_grid(tf, 64 * pl.P, &cap);
    if (rc != LL_OK) return rc;
    const int64_t tiles = (pl.units + 63) / 64;
    if (tf != nullptr && tiles <= cap / pl.P) {
      Plan tp = pl;
      tp.rooted_tile = true;
      return launch_kernel(tf, tp, (int)tiles, 64 * pl.P, stream);
    }
  }
  // The same for the two-shot AllReduce and the stand-alone ReduceScatter /
  // AllGather with one unit per lane (the AllReduce with lines also two)
  // and one iteration: the straight-line two-shot kernel.
  if (two_waves) {
    kernel_fn tf = nullptr;
    int64_t tiles = 0;
    if (twoshot_tile_ok(pl, wpr, wlog, &tf, &tiles)) return launch_kernel(tf, pl, (int)tiles, 64 * pl.P, stream);
  }
  int threads = pl.o.threads;
  if (threads == 0) threads = 256;
  int lanes_per_unit = pl.proto == PR_LINE ? ProtoLine::kLanes : 1;
  int64_t work_units = pl.units;
  if (wave_kernel) {  // one wave per rank; 64*U one-lane units (U line units) per workgroup and step
    threads = 64 * pl.P;
    const int64_t tile = (pl.proto == PR_LINE ? 1 : 64) * kWaveUnits[wlog];
    work_units = (pl.units + tile - 1) / tile;
    lanes_per_unit = threads;
  }
  int cap_grid = 0;
  int st = resident_grid(fn, threads, &cap_grid);
  if (st != LL_OK) return st;
  int wmax = cap_grid / pl.P;
  if (wmax < 1) return LL_ERR_UNSUPPORTED;
  int W = pl.o.wg_per_rank;
  if (W == 0) {
    const int64_t lanes = work_units * lanes_per_unit;
    int64_t want = (lanes + threads - 1) / threads;
    if (want < 1) want = 1;
    W = (int)(want < wmax ? want : wmax);
  } else if (W > wmax) {
    W = wmax;  // never launch more than can be resident: waits depend on co-residency
  }
  return launch_kernel(fn, pl, W, threads, stream);
}

// Launch `fn` with W workgroups per rank and `threads` per workgroup.
int launch_kernel(kernel_fn fn, const Plan &pl, int W, int threads, void *stream) {
  const int grid = W * pl.P;
  KArgs a = pl.a;
  if (a.in == nullptr) {  // input inside the region, at offset 0 of every slice
    a.in = a.sym;
    a.in_stride = a.stride;
    a.in_al4 = 1;
  }
  if (a.iters == 0) {
    a.iters = 1;
    a.iter_n = a.n;
  }
  a.timeout = pl.o.timeout;
  a.mute = pl.o.mute;
  a.first_wait = (uint16_t)pl.o.first_wait;
  a.poll_gap = (uint16_t)pl.o.poll_gap;
  a.lag = (uint32_t)pl.o.lag;
  a.clear = clear_slots(pl);
  a.grid = (uint32_t)grid;
  a.block = (uint32_t)threads;
  a.units = pl.units;
  const int st = status_of(stream, &a.status);
  if (st != LL_OK) return st;
  a.stamps = pl.o.stamps;
  a.phases = pl.o.phases;
  hipLaunchKernelGGL(fn, dim3(grid), dim3(threads), 0, (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (pl.o.grid_out) *pl.o.grid_out = grid;
  if (pl.o.threads_out) *pl.o.threads_out = threads;
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  return LL_OK;
}

// Region geometry of one call; fails with LL_ERR_SCRATCH when the input does
// not fit the region's input capacity.  fmt: the packet formats the region
// holds (L::kFmt* bits).
struct Region {
  uint64_t cap, a8, a128, aa, as;
  unsigned fmt;
  uint64_t area_of(int proto) const {
    return proto == PR_LINE ? cap + a8 : (proto == PR_SENT ? cap + a8 + a128 + aa : cap);
  }
  uint64_t atomic_area() const { return cap + a8 + a128; }
};

// Slot bytes and packet units for a payload of `bytes` in format `proto`.
uint64_t slot_bytes(int proto, uint64_t bytes) {
  return proto == PR_LINE ? L::slot128(bytes) : (proto == PR_SENT ? L::slotS(bytes) : L::slot8(bytes));
}
int64_t units_of(int proto, uint64_t bytes) {
  const int64_t words = (int64_t)L::ceil_div(bytes, 4);
  return proto == PR_LINE ? ProtoLine::units(words) : (proto == PR_SENT ? ProtoSent::units(words) : ProtoLL::units(words));
}

int region_of(size_t rank_stride, int P, uint64_t in_bytes, Region *rg) {
  const unsigned fmt = L::formats_of(rank_stride);
  const uint64_t cap = L::capacity(rank_stride, P);
  if (L::slice_for(cap, P, fmt) > rank_stride) return LL_ERR_SCRATCH;
  if (in_bytes > L::kMaxInputBytes) return LL_ERR_UNSUPPORTED;
  if (in_bytes > cap) return LL_ERR_SCRATCH;
  const L::Areas ar = L::areas(cap, P, fmt);
  rg->cap = cap;
  rg->a8 = ar.a8;
  rg->a128 = ar.a128;
  rg->aa = ar.aa;
  rg->as = ar.as;
  rg->fmt = fmt;
  return LL_OK;
}

KArgs base_args(void *sym_base, size_t rank_stride, void *out, uint32_t epoch) {
  KArgs a;
  memset(&a, 0, sizeof a);
  a.sym = (char *)sym_base;
  a.stride = rank_stride;
  a.out = (char *)out;
  a.epoch = epoch;
  a.mute = -1;
  return a;
}

// Size thresholds measured on MI355X (p50 of back-to-back calls of every
// algorithm at 2 KiB .. 16 MiB per rank, P = 2 .. 8, bfloat16; binary32
// crosses over at the same byte sizes); M = input bytes per rank.  Flags only
// unless the caller allows sentinel mode, which wins from the smallest sizes
// up to 1-8 MiB (by rank count), as the paper observes for larger messages
// and rank counts.
ll_algo auto_algo(uint64_t in_bytes, int P, bool sentinel_ok) {
  const uint64_t KiB = 1024, MiB = 1024 * 1024;
  // the line two-shot with one wave per peer at every size up to the
  // maximum, except above 16 MiB at 5-6 ranks, where the one-lane line
  // two-shot is faster (measured at 8-64 MiB, binary32)
  const uint64_t line_waves_max = (P == 5 || P == 6) ? 16 * MiB : L::kMaxInputBytes;
  auto large = [&]() { return in_bytes <= line_waves_max ? LL_ALGO_TWOSHOT_LINE_WAVES : LL_ALGO_TWOSHOT_LINE; };
  // With sentinel mode allowed, messages of at most 8 KiB at 3 or more ranks
  // still take the 8-byte one-shot (whose slots are cleared after reading),
  // which is as fast or faster there: flags win for the smallest messages.
  if (sentinel_ok && (P == 2 || in_bytes > 8 * KiB)) {
    uint64_t one_max, two_max;  // one-shot, then two-shot, sentinel units with one wave per peer
    if (P <= 3) {
      one_max = (P == 2 ? 2048 : 512) * KiB;
      two_max = (P == 2 ? 8 : 4) * MiB;
    } else if (P <= 5) {
      one_max = (P == 4 ? 256 : 128) * KiB;
      two_max = 2 * MiB;
    } else if (P <= 7) {
      one_max = (P == 6 ? 128 : 64) * KiB;
      two_max = (P == 6 ? 2 : 1) * MiB;
    } else {
      one_max = 64 * KiB;
      two_max = 1 * MiB;
    }
    if (in_bytes <= one_max) return LL_ALGO_ONESHOT_SENTINEL_WAVES;
    // at 2 ranks the line two-shot beats the sentinel two-shot from 2 to
    // 4 MiB (3 MiB: 6.41 against 7.25 us), the sentinel two-shot it above
    if (P == 2 && in_bytes <= 4 * MiB) return large();
    if (in_bytes <= two_max) return LL_ALGO_TWOSHOT_SENTINEL_WAVES;
    return large();
  }
  if (P == 2) {
    if (in_bytes <= 512 * KiB) return LL_ALGO_ONESHOT_WAVES;
    if (in_bytes <= 2 * MiB) return LL_ALGO_ONESHOT_LINE_WAVES;
    return large();
  }
  // one-shot with 8-byte packets, then with lines, then the line two-shot
  // (whose one-tile kernel takes the two-shot below the one-shot from
  // 32-512 KiB, by rank count)
  uint64_t one8_max, line_max;
  if (P == 3) {
    one8_max = 64 * KiB;
    line_max = 512 * KiB;
  } else if (P == 4) {
    one8_max = 32 * KiB;
    line_max = 128 * KiB;
  } else {
    one8_max = 16 * KiB;
    line_max = P == 8 ? 32 * KiB : (P == 5 ? 128 * KiB : 64 * KiB);
  }
  if (in_bytes <= one8_max) return LL_ALGO_ONESHOT_WAVES;
  if (in_bytes <= line_max) return LL_ALGO_ONESHOT_LINE_WAVES;
  return large();
}

// ReduceScatter / AllGather, by the bytes of data per rank (input for
// ReduceScatter, output for AllGather), measured the same way at 4 KiB ..
// 8 MiB at 4 and 8 ranks: ReduceScatter with 8-byte packets up to 128 KiB
// and lines above (4 ranks, b = 16, 224 KiB: 3.20 us with 8-byte packets,
// 3.08 us with lines); AllGather with lines at every size (8 ranks, b = 1,
// 14 KiB: 3.28 us with 8-byte packets, 3.08 us with lines); with sentinel
// mode allowed, sentinel units up to 2 MiB (4 MiB at 2-4 ranks).
ll_proto auto_proto(uint64_t bytes, int P, bool sentinel_ok, bool allgather) {
  const uint64_t KiB = 1024, MiB = 1024 * 1024;
  if (sentinel_ok) return bytes <= (P >= 5 ? 2 : 4) * MiB ? LL_PROTO_SENTINEL : LL_PROTO_LINE128;
  return !allgather && bytes <= 128 * KiB ? LL_PROTO_PACKET8 : LL_PROTO_LINE128;
}

// Broadcast / Reduce (8 ranks, bf16): up to 64 KiB per rank the one-tile
// kernel with 8-byte packets, or with sentinel units when allowed (16 KiB:
// Broadcast 3.24 and 2.93 us, Reduce 3.20 and 3.12 us); lines above (1 MiB:
// Broadcast 12.50 us against 12.74 with sentinel units, Reduce 12.44
// against 16.00).
ll_proto auto_proto_rooted(uint64_t bytes, bool sentinel_ok) {
  if (bytes <= (64u << 10)) return sentinel_ok ? LL_PROTO_SENTINEL : LL_PROTO_PACKET8;
  return LL_PROTO_LINE128;
}

// Stand-alone ReduceScatter / AllGather: the wave-per-peer kernels serve
// each format up to the size where the one-lane-per-unit kernels catch up
// (measured at 4 and 8 ranks): 8-byte packets and sentinel units up to
// 2 MiB of data per rank; lines up to 8 MiB at 2-4 ranks and 4 MiB at 5-8
// ranks (8 ranks, b = 256, 3.5 MiB: AllGather 23.3 us with one lane per
// unit, 17.9 us with one wave per peer at two units per lane).
// ll_tuning.wave_kernels forces either family.
bool use_wave_kernel(ll_proto proto, uint64_t bytes, int P, bool allgather, const CallOpts &o) {
  (void)allgather;
  const int m = o.wave_kernels;
  if (m != 0) return m == 2;
  const uint64_t MiB = 1024 * 1024;
  if (proto == LL_PROTO_LINE128) return bytes <= (P >= 5 ? 4 : 8) * MiB;
  return bytes <= 2 * MiB;
}

// The wave-per-peer one-shot kernels run a single iteration only.
bool is_wave_algo(ll_algo a) {
  return a == LL_ALGO_ONESHOT_WAVES || a == LL_ALGO_ONESHOT_SENTINEL_WAVES || a == LL_ALGO_ONESHOT_LINE_WAVES;
}

// Algorithms whose AllGather stores into the peers' sentinel-filled outputs.
bool fills_output(ll_algo algo) { return algo == LL_ALGO_TWOSHOT_SENTINEL_OUT || algo == LL_ALGO_TWOSHOT_ATOMIC; }

// The region format an AllReduce algorithm needs.
unsigned algo_fmt(ll_algo a) {
  switch (a) {
    case LL_ALGO_TWOSHOT_LINE: case LL_ALGO_ONESHOT_LINE: case LL_ALGO_ONESHOT_LINE_WAVES:
    case LL_ALGO_TWOSHOT_LINE_WAVES:
      return L::kFmtLine;
    case LL_ALGO_ONESHOT_SENTINEL: case LL_ALGO_TWOSHOT_SENTINEL: case LL_ALGO_TWOSHOT_SENTINEL_OUT:
    case LL_ALGO_TWOSHOT_SENTINEL_WAVES: case LL_ALGO_ONESHOT_SENTINEL_WAVES:
      return L::kFmtSent;
    case LL_ALGO_TWOSHOT_ATOMIC:
      return L::kFmtAtomic;
    case LL_ALGO_AUTO:
      return L::kFmtAll;
    default:
      return L::kFmt8;
  }
}
unsigned proto_fmt(ll_proto p) {
  return p == LL_PROTO_LINE128 ? L::kFmtLine : (p == LL_PROTO_SENTINEL ? L::kFmtSent : L::kFmt8);
}

// The algorithm of the same shape (one-shot or two-shot, one lane per unit
// or one wave per peer) in packet format f (kFmt8, kFmtLine or kFmtSent).
ll_algo in_format(ll_algo a, unsigned f) {
  int shape;  // 0 one-shot waves, 1 one-shot, 2 two-shot waves, 3 two-shot
  switch (a) {
    case LL_ALGO_ONESHOT_WAVES: case LL_ALGO_ONESHOT_LINE_WAVES: case LL_ALGO_ONESHOT_SENTINEL_WAVES: shape = 0; break;
    case LL_ALGO_ONESHOT: case LL_ALGO_ONESHOT_LINE: case LL_ALGO_ONESHOT_SENTINEL: shape = 1; break;
    case LL_ALGO_TWOSHOT_WAVES: case LL_ALGO_TWOSHOT_LINE_WAVES: case LL_ALGO_TWOSHOT_SENTINEL_WAVES: shape = 2; break;
    default: shape = 3; break;
  }
  static const ll_algo by[4][3] = {
      {LL_ALGO_ONESHOT_WAVES, LL_ALGO_ONESHOT_LINE_WAVES, LL_ALGO_ONESHOT_SENTINEL_WAVES},
      {LL_ALGO_ONESHOT, LL_ALGO_ONESHOT_LINE, LL_ALGO_ONESHOT_SENTINEL},
      {LL_ALGO_TWOSHOT_WAVES, LL_ALGO_TWOSHOT_LINE_WAVES, LL_ALGO_TWOSHOT_SENTINEL_WAVES},
      {LL_ALGO_TWOSHOT, LL_ALGO_TWOSHOT_LINE, LL_ALGO_TWOSHOT_SENTINEL}};
  return by[shape][f == L::kFmt8 ? 0 : (f == L::kFmtLine ? 1 : 2)];
}

// The formats AUTO may use on a region holding `region_fmt`: the flagged
// formats the region holds (not lines with LL_OPT_NO_LINES); sentinel units
// when the options allow them, or when the region holds no flagged format
// (it was sized for a sentinel algorithm).
unsigned auto_formats(unsigned region_fmt, const CallOpts &o) {
  unsigned f = region_fmt & (L::kFmt8 | (o.lines_ok() ? L::kFmtLine : 0u));
  if ((region_fmt & L::kFmtSent) && (o.sentinel_ok() || f == 0)) f |= L::kFmtSent;
  return f;
}

// The first of the formats in `order` that `allowed` holds; 0 if none.
unsigned first_allowed(const unsigned *order, int n, unsigned allowed) {
  for (int i = 0; i < n; ++i)
    if (allowed & order[i]) return order[i];
  return 0;
}

// AUTO for an AllReduce of in_bytes per rank: the measured choice among the
// allowed formats, moved to another allowed format of the same shape when
// its own is not (8-byte packets first, then lines, then sentinel units; a
// line choice goes to 8-byte packets first).  LL_ALGO_AUTO if no format is
// allowed.
ll_algo auto_choice(uint64_t in_bytes, int P, unsigned allowed) {
  if (allowed == 0) return LL_ALGO_AUTO;
  const ll_algo a = auto_algo(in_bytes, P, (allowed & L::kFmtSent) != 0);
  const unsigned f = algo_fmt(a);
  if (allowed & f) return a;
  static const unsigned order[3] = {L::kFmt8, L::kFmtLine, L::kFmtSent};
  return in_format(a, first_allowed(order, 3, allowed));
}

// AUTO for the stand-alone and rooted collectives, likewise; LL_PROTO_AUTO
// if no format is allowed.
ll_proto proto_choice(ll_proto p, unsigned allowed) {
  if (allowed == 0) return LL_PROTO_AUTO;
  if (allowed & proto_fmt(p)) return p;
  static const unsigned order[3] = {L::kFmt8, L::kFmtLine, L::kFmtSent};
  const unsigned f = first_allowed(order, 3, allowed);
  return f == L::kFmt8 ? LL_PROTO_PACKET8 : (f == L::kFmtLine ? LL_PROTO_LINE128 : LL_PROTO_SENTINEL);
}

// Kernel, packet format, slot size and unit count of an AllReduce of `count`
// elements per rank whose iterations hold `iter_count` elements.
// area_of(proto) gives the offset of that packet format's area in a slice.
template <class AreaOf>
void plan_allreduce(Plan *pl, ll_algo algo, uint64_t count, int es, int nranks, uint64_t iter_count,
                    AreaOf area_of) {
  const uint64_t it_bytes = iter_count * (uint64_t)es;
  const bool line = (algo == LL_ALGO_TWOSHOT_LINE || algo == LL_ALGO_ONESHOT_LINE ||
                     algo == LL_ALGO_ONESHOT_LINE_WAVES || algo == LL_ALGO_TWOSHOT_LINE_WAVES);
  const bool sent = (algo == LL_ALGO_ONESHOT_SENTINEL || algo == LL_ALGO_TWOSHOT_SENTINEL ||
                     algo == LL_ALGO_TWOSHOT_SENTINEL_OUT || algo == LL_ALGO_TWOSHOT_SENTINEL_WAVES ||
                     algo == LL_ALGO_ONESHOT_SENTINEL_WAVES);
  const bool waves = (algo == LL_ALGO_ONESHOT_WAVES || algo == LL_ALGO_ONESHOT_SENTINEL_WAVES ||
                      algo == LL_ALGO_ONESHOT_LINE_WAVES);
  pl->proto = line ? PR_LINE : (sent ? PR_SENT : PR_LL);
  pl->a.area = area_of(pl->proto);
  if (algo == LL_ALGO_ONESHOT || algo == LL_ALGO_ONESHOT_LINE || algo == LL_ALGO_ONESHOT_SENTINEL || waves) {
    pl->kind = waves ? K_ONESHOT_WAVES : K_ONESHOT;
    pl->a.slot = slot_bytes(pl->proto, it_bytes);
    pl->units = units_of(pl->proto, it_bytes);
  } else {
    pl->kind = algo == LL_ALGO_TWOSHOT_SENTINEL_OUT ? K_TWOSHOT_OUT : K_TWOSHOT;
    if (algo == LL_ALGO_TWOSHOT_WAVES || algo == LL_ALGO_TWOSHOT_SENTINEL_WAVES || algo == LL_ALGO_TWOSHOT_LINE_WAVES)
      pl->kind = K_TWOSHOT_WAVES;
    const uint64_t C = (uint64_t)iter_span((int64_t)count, (int64_t)iter_count, 0, nranks, es).chunk;
    pl->a.chunk = (int64_t)C;
    pl->a.slot = slot_bytes(pl->proto, C * es);
    pl->units = units_of(pl->proto, C * es);
  }
}

}  // namespace

// =================================================================== C ABI
extern "C" {

int ll_options_init(ll_options *opt) {
  if (opt == nullptr) return LL_ERR_INVALID;
  memset(opt, 0, sizeof *opt);
  opt->size = sizeof(ll_options);
  return LL_OK;
}

int ll_tuning_init(ll_tuning *t) {
  if (t == nullptr) return LL_ERR_INVALID;
  memset(t, 0, sizeof *t);
  t->size = sizeof(ll_tuning);
  t->pipeline_lag = -1;
  t->mute_rank = -1;
  return LL_OK;
}

int ll_slice_bytes(size_t count, ll_dtype dt, int nranks, ll_algo algo, size_t *min_rank_stride) {
  if (min_rank_stride == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (dt != LL_F32 && dt != LL_BF16) return LL_ERR_UNSUPPORTED;
  if ((int)algo < LL_ALGO_AUTO || (int)algo > LL_ALGO_TWOSHOT_LINE_WAVES) return LL_ERR_INVALID;
  const uint64_t es = (uint64_t)esize_of(dt);
  if (count > L::kMaxInputBytes / es) return LL_ERR_UNSUPPORTED;
  const uint64_t cap = L::roundup((uint64_t)count * es, L::kAlign);
  *min_rank_stride = (size_t)L::stride_for(cap, nranks, algo_fmt(algo));
  return LL_OK;
}

int ll_input_capacity(size_t rank_stride, int nranks, size_t *capacity_bytes) {
  if (capacity_bytes == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (rank_stride % LL_ALIGN != 0) return LL_ERR_INVALID;
  const uint64_t cap = L::capacity(rank_stride, nranks);
  if (L::slice_for(cap, nranks, L::formats_of(rank_stride)) > rank_stride) return LL_ERR_SCRATCH;
  *capacity_bytes = (size_t)cap;
  return LL_OK;
}

int ll_slice_layout(size_t rank_stride, int nranks, size_t *offsets6) {
  if (offsets6 == nullptr) return LL_ERR_INVALID;
  size_t cap = 0;
  const int st = ll_input_capacity(rank_stride, nranks, &cap);
  if (st != LL_OK) return st;
  const L::Areas ar = L::areas(cap, nranks, L::formats_of(rank_stride));
  offsets6[0] = 0;
  offsets6[1] = cap;
  offsets6[2] = cap + ar.a8;
  offsets6[3] = cap + ar.a8 + ar.a128;
  offsets6[4] = cap + ar.a8 + ar.a128 + ar.aa;
  offsets6[5] = cap + ar.a8 + ar.a128 + ar.aa + ar.as;
  return LL_OK;
}

int ll_init(void *sym_base, size_t rank_stride, int nranks, void *stream) {
  if (sym_base == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (((uintptr_t)sym_base % LL_ALIGN) != 0 || rank_stride % LL_ALIGN != 0 || rank_stride == 0) return LL_ERR_INVALID;
  Region rg;
  int st = region_of(rank_stride, nranks, 0, &rg);
  if (st != LL_OK) return st;
  DevInfo d;
  st = device_info(&d);
  if (st != LL_OK) return st;
  // flags start at 0 (never a valid epoch); sentinel slots start at the sentinel
  const uint64_t lo = rg.cap, mid = rg.cap + rg.a8 + rg.a128 + rg.aa, hi = mid + rg.as;
  if (mid > lo)
    hipLaunchKernelGGL(k_fill_areas, dim3(d.cus * 4), dim3(256), 0, (hipStream_t)stream, (char *)sym_base,
                       (uint64_t)rank_stride, nranks, lo, mid, 0u);
  if (hi > mid)
    hipLaunchKernelGGL(k_fill_areas, dim3(d.cus * 4), dim3(256), 0, (hipStream_t)stream, (char *)sym_base,
                       (uint64_t)rank_stride, nranks, mid, hi, ProtoSent::kSentinel);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  return LL_OK;
}

int ll_fill_sentinel(void *out, size_t count, ll_dtype dt, int nranks, void *stream) {
  if (out == nullptr || ((uintptr_t)out % 16) != 0) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (dt != LL_F32 && dt != LL_BF16) return LL_ERR_UNSUPPORTED;
  const uint64_t es = (uint64_t)esize_of(dt);
  if (count > L::kMaxInputBytes / es) return LL_ERR_UNSUPPORTED;
  const uint64_t bytes = (uint64_t)count * es * (uint64_t)nranks;
  if (bytes == 0) return LL_OK;
  DevInfo d;
  const int st = device_info(&d);
  if (st != LL_OK) return st;
  const uint64_t want = L::ceil_div(L::ceil_div(bytes, 16), 256);
  const int grid = (int)std::max<uint64_t>(1, std::min<uint64_t>(want, (uint64_t)d.cus * 8));
  hipLaunchKernelGGL(k_fill_ones, dim3(grid), dim3(256), 0, (hipStream_t)stream, (char *)out, bytes);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  return LL_OK;
}

int ll_allreduce_ex(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op, int nranks,
                    uint32_t epoch, void *stream, ll_algo algo, const ll_options *opt) {
  int st = check_common(sym_base, rank_stride, out, nranks, epoch);
  if (st != LL_OK) return st;
  st = check_dtype_op((int)dt, (int)op);
  if (st != LL_OK) return st;
  if ((int)algo < LL_ALGO_AUTO || (int)algo > LL_ALGO_TWOSHOT_LINE_WAVES) return LL_ERR_INVALID;
  CallOpts o;
  st = resolve_opts(opt, &o);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  const uint64_t in_bytes = (uint64_t)count * es;
  if (fills_output(algo) && in_bytes % 16 != 0) return LL_ERR_UNSUPPORTED;
  if (count > L::kMaxInputBytes) return LL_ERR_UNSUPPORTED;
  if (overlaps(out, in_bytes * nranks, sym_base, (uint64_t)rank_stride * nranks)) return LL_ERR_INVALID;
  Region rg;
  st = region_of(rank_stride, nranks, in_bytes, &rg);
  if (st != LL_OK) return st;
  if (algo == LL_ALGO_AUTO) {
    algo = auto_choice(in_bytes, nranks, auto_formats(rg.fmt, o));
    if (algo == LL_ALGO_AUTO) return LL_ERR_SCRATCH;  // no format AUTO may use
  }
  if ((rg.fmt & algo_fmt(algo)) == 0) return LL_ERR_SCRATCH;  // the region holds no area for this format
  if (count == 0) return LL_OK;

  Plan pl;
  pl.dt = (int)dt;
  pl.P = nranks;
  pl.o = o;
  pl.a = base_args(sym_base, rank_stride, out, epoch);
  pl.a.n = (int64_t)count;
  pl.a.al4 = (in_bytes % 4 == 0) ? 1u : 0u;
  if (algo == LL_ALGO_TWOSHOT_ATOMIC) {
    pl.kind = K_TWOSHOT_ATOMIC;
    pl.proto = PR_SENT;
    const uint64_t C = L::twoshot_chunk(count, nranks, es);
    pl.a.chunk = (int64_t)C;
    pl.a.area = rg.atomic_area();
    pl.a.slot = L::atomic_acc_bytes(C * es, es);  // binary32 accumulator in whole tiles
    pl.units = (int64_t)L::ceil_div(C * es, 1024) * 64;  // one lane per 16 input bytes
    return launch(pl, stream);
  }
  plan_allreduce(&pl, algo, count, es, nranks, count, [&](int proto) { return rg.area_of(proto); });
  return launch(pl, stream);
}

int ll_allreduce_algo(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op,
                      int nranks, uint32_t epoch, void *stream, ll_algo algo) {
  return ll_allreduce_ex(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, algo, nullptr);
}

int ll_auto_algo(size_t count, ll_dtype dt, int nranks, size_t rank_stride, const ll_options *opt, ll_algo *algo) {
  if (algo == nullptr || nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if ((int)dt != LL_F32 && (int)dt != LL_BF16) return LL_ERR_UNSUPPORTED;
  CallOpts o;
  const int st = resolve_opts(opt, &o);
  if (st != LL_OK) return st;
  const unsigned fmt = rank_stride == 0 ? L::kFmtAll : L::formats_of(rank_stride);
  const ll_algo a = auto_choice((uint64_t)count * esize_of(dt), nranks, auto_formats(fmt, o));
  if (a == LL_ALGO_AUTO) return LL_ERR_SCRATCH;
  *algo = a;
  return LL_OK;
}

int ll_allreduce(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op, int nranks,
                 uint32_t epoch, void *stream) {
  return ll_allreduce_ex(sym_base, rank_stride, out, count, dt, op, nranks, epoch, stream, LL_ALGO_AUTO, nullptr);
}

// ---------------------------------------------------------------- bounded scratch
int ll_scratch_bytes(size_t iter_bytes, int nranks, size_t *min_scratch_stride) {
  if (min_scratch_stride == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (iter_bytes == 0 || iter_bytes > L::kMaxInputBytes) return LL_ERR_INVALID;
  *min_scratch_stride = (size_t)L::scratch_for(L::roundup(iter_bytes, L::kAlign), nranks);
  return LL_OK;
}

int ll_scratch_iter_bytes(size_t scratch_stride, int nranks, size_t *iter_bytes) {
  if (iter_bytes == nullptr) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (scratch_stride == 0 || scratch_stride % LL_ALIGN != 0) return LL_ERR_INVALID;
  const uint64_t D = L::iter_capacity(scratch_stride, nranks);
  if (D == 0) return LL_ERR_SCRATCH;
  *iter_bytes = (size_t)D;
  return LL_OK;
}

int ll_scratch_init(void *scratch_base, size_t scratch_stride, int nranks, void *stream) {
  if (scratch_base == nullptr || ((uintptr_t)scratch_base % LL_ALIGN) != 0) return LL_ERR_INVALID;
  size_t D = 0;
  int st = ll_scratch_iter_bytes(scratch_stride, nranks, &D);
  if (st != LL_OK) return st;
  DevInfo d;
  st = device_info(&d);
  if (st != LL_OK) return st;
  const uint64_t mid = 2 * (L::area8(D, nranks) + L::area128(D, nranks));
  const uint64_t hi = mid + 2 * L::areaS(D, nranks);
  hipLaunchKernelGGL(k_fill_areas, dim3(d.cus * 4), dim3(256), 0, (hipStream_t)stream, (char *)scratch_base,
                     (uint64_t)scratch_stride, nranks, (uint64_t)0, mid, 0u);
  hipLaunchKernelGGL(k_fill_areas, dim3(d.cus * 4), dim3(256), 0, (hipStream_t)stream, (char *)scratch_base,
                     (uint64_t)scratch_stride, nranks, mid, hi, ProtoSent::kSentinel);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  return LL_OK;
}

static void buffered_iterations(uint64_t count, int es, uint64_t D, uint64_t *iter_count, uint64_t *iters) {
  *iter_count = std::min<uint64_t>(count, D / (uint64_t)es);
  *iters = *iter_count ? (count + *iter_count - 1) / *iter_count : 0;
}

int ll_buffered_plan(size_t count, ll_dtype dt, int nranks, size_t scratch_stride, uint32_t *iters,
                     size_t *iter_count) {
  if (iters == nullptr || iter_count == nullptr) return LL_ERR_INVALID;
  int st = check_dtype_op((int)dt, LL_SUM);
  if (st != LL_OK) return st;
  size_t D = 0;
  st = ll_scratch_iter_bytes(scratch_stride, nranks, &D);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  if (count > (L::kMaxBufferedBytes / (uint64_t)es)) return LL_ERR_UNSUPPORTED;
  uint64_t ic = 0, k = 0;
  buffered_iterations(count, es, D, &ic, &k);
  if (k > 0xFFFFFFFFull) return LL_ERR_UNSUPPORTED;
  *iters = (uint32_t)k;
  *iter_count = (size_t)ic;
  return LL_OK;
}

int ll_iteration_span(size_t count, size_t iter_count, uint32_t it, int nranks, ll_dtype dt, int64_t *out3) {
  if (out3 == nullptr || iter_count == 0 || nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  const int st = check_dtype_op((int)dt, LL_SUM);
  if (st != LL_OK) return st;
  const IterSpan sp = iter_span((int64_t)count, (int64_t)iter_count, it, nranks, esize_of(dt));
  out3[0] = sp.e0;
  out3[1] = sp.n;
  out3[2] = sp.chunk;
  return LL_OK;
}

// A bounded-scratch AllReduce through the scratch region at scratch_base,
// laid out for `layout_P` ranks (nranks <= layout_P: a call uses the first
// nranks slices and the first nranks-1 slots of every area, whose offsets
// depend on layout_P only).  With flags_only, sentinel algorithms are
// refused and AUTO picks among the flagged ones.
static int buffered_call(const void *in, void *out, size_t count, ll_dtype dt, ll_op op, int nranks,
                         void *scratch_base, size_t scratch_stride, int layout_P, bool flags_only, uint32_t epoch,
                         void *stream, ll_algo algo, const ll_options *opt, uint32_t *epochs_used) {
  if (epochs_used != nullptr) *epochs_used = 0;
  CallOpts o;
  const int so = resolve_opts(opt, &o);
  if (so != LL_OK) return so;
  if (flags_only) o.flags &= ~(uint32_t)LL_OPT_AUTO_SENTINEL;
  if (in == nullptr || out == nullptr || scratch_base == nullptr) return LL_ERR_INVALID;
  if (((uintptr_t)in % 16) != 0 || ((uintptr_t)out % 16) != 0) return LL_ERR_INVALID;
  if (((uintptr_t)scratch_base % LL_ALIGN) != 0) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  if (epoch == 0) return LL_ERR_INVALID;
  int st = check_dtype_op((int)dt, (int)op);
  if (st != LL_OK) return st;
  if ((int)algo < LL_ALGO_AUTO || (int)algo > LL_ALGO_TWOSHOT_LINE_WAVES) return LL_ERR_INVALID;
  if (algo == LL_ALGO_TWOSHOT_ATOMIC) return LL_ERR_UNSUPPORTED;  // single-iteration regions only
  if (flags_only && (algo == LL_ALGO_ONESHOT_SENTINEL || algo == LL_ALGO_TWOSHOT_SENTINEL ||
                     algo == LL_ALGO_TWOSHOT_SENTINEL_OUT || algo == LL_ALGO_TWOSHOT_SENTINEL_WAVES ||
                     algo == LL_ALGO_ONESHOT_SENTINEL_WAVES))
    return LL_ERR_UNSUPPORTED;
  if (nranks > layout_P) return LL_ERR_INVALID;
  size_t D = 0;
  st = ll_scratch_iter_bytes(scratch_stride, layout_P, &D);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  if (count > (L::kMaxBufferedBytes / (uint64_t)es)) return LL_ERR_UNSUPPORTED;
  const uint64_t in_bytes = (uint64_t)count * es;
  if (algo == LL_ALGO_TWOSHOT_SENTINEL_OUT && in_bytes % 16 != 0) return LL_ERR_UNSUPPORTED;
  if (algo == LL_ALGO_TWOSHOT_SENTINEL_OUT && in == out) return LL_ERR_INVALID;  // its output starts as sentinels
  const uint64_t all = in_bytes * (uint64_t)nranks, sbytes = (uint64_t)scratch_stride * nranks;
  if (in != out && overlaps(in, all, out, all)) return LL_ERR_INVALID;  // in place, or apart
  if (overlaps(in, all, scratch_base, sbytes) || overlaps(out, all, scratch_base, sbytes)) return LL_ERR_INVALID;
  if (count == 0) return LL_OK;
  uint64_t iter_count = 0, iters = 0;
  buffered_iterations(count, es, D, &iter_count, &iters);
  if ((uint64_t)epoch + iters - 1 > 0xFFFFFFFFull) return LL_ERR_INVALID;
  if (algo == LL_ALGO_AUTO) {
    // by the iteration size; the one-shot wave kernels run one iteration
    // only, and the two-shot wave kernels take their place (measured on the
    // paper's scratch study shape, 32 MiB at 8 ranks in 256 KiB .. 32 MiB
    // iterations)
    // (every scratch region holds all three formats)
    algo = auto_choice(iter_count * es, nranks, auto_formats(L::kFmt8 | L::kFmtLine | L::kFmtSent, o));
    if (iters > 1 && algo == LL_ALGO_ONESHOT_WAVES) algo = LL_ALGO_TWOSHOT_WAVES;
    if (iters > 1 && algo == LL_ALGO_ONESHOT_SENTINEL_WAVES) algo = LL_ALGO_TWOSHOT_SENTINEL_WAVES;
    if (iters > 1 && algo == LL_ALGO_ONESHOT_LINE_WAVES) algo = LL_ALGO_TWOSHOT_LINE_WAVES;
  }
  if (iters > 1 && is_wave_algo(algo))
    return LL_ERR_UNSUPPORTED;

  Plan pl;
  pl.dt = (int)dt;
  pl.P = nranks;
  pl.o = o;
  pl.a = base_args(scratch_base, scratch_stride, out, epoch);
  pl.a.in = (const char *)in;
  pl.a.in_stride = in_bytes;
  pl.a.in_al4 = (in_bytes % 4 == 0) ? 1u : 0u;
  pl.a.n = (int64_t)count;
  pl.a.al4 = (in_bytes % 4 == 0) ? 1u : 0u;
  pl.a.iters = (uint32_t)iters;
  pl.a.iter_n = (int64_t)iter_count;
  const uint64_t a8 = L::area8(D, layout_P), a128 = L::area128(D, layout_P), as = L::areaS(D, layout_P);
  plan_allreduce(&pl, algo, count, es, nranks, iter_count, [&](int proto) {
    return proto == PR_LINE ? 2 * a8 : (proto == PR_SENT ? 2 * (a8 + a128) : (uint64_t)0);
  });
  pl.a.sub_bytes = pl.proto == PR_LINE ? a128 : (pl.proto == PR_SENT ? as : a8);
  st = launch(pl, stream);
  if (st == LL_OK && epochs_used != nullptr) *epochs_used = (uint32_t)iters;
  return st;
}

int ll_allreduce_buffered(const void *in, void *out, size_t count, ll_dtype dt, ll_op op, int nranks,
                          void *scratch_base, size_t scratch_stride, uint32_t epoch, void *stream, ll_algo algo,
                          const ll_options *opt, uint32_t *epochs_used) {
  if (nranks < 2 || nranks > LL_MAX_RANKS) {
    if (epochs_used != nullptr) *epochs_used = 0;
    return LL_ERR_INVALID;
  }
  return buffered_call(in, out, count, dt, op, nranks, scratch_base, scratch_stride, nranks, false, epoch, stream,
                       algo, opt, epochs_used);
}

// ---------------------------------------------------------------- no allocation
// The scratch of ll_allreduce_static: a bounded-scratch region of
// LL_STATIC_SCRATCH_BYTES laid out for LL_MAX_RANKS slices, one copy per
// device, held until the process ends.  In host code the name stands for
// no device address: host code uses only the address that
// hipGetSymbolAddress reports for the current device (static_scratch_of).
static __device__ __align__(256) unsigned char scratch[LL_STATIC_SCRATCH_BYTES];

namespace {
struct StaticScratch {
  void *ptr = nullptr;      // device address of `scratch` on this device
  bool init_needed = true;  // flags not yet cleared, or a timeout seen since
  uint64_t next_epoch = 1;  // epochs of this device's static scratch, shared by all its callers
};
StaticScratch g_static[64];  // guarded by g_static_mu

constexpr size_t kStaticStride = LL_STATIC_SCRATCH_BYTES / LL_MAX_RANKS;
}  // namespace

// Device address of the current device's static scratch (looked up once per
// device), and the first of `iters` epochs for a call; clears the flag areas
// on `stream` first when they need it (first use on the device, a timeout
// reported by ll_check since, or the epochs running out).
static int static_scratch_of(uint64_t iters, void *stream, void **ptr, uint32_t *epoch) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  if (dev < 0 || dev >= 64) return LL_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_static_mu);
  StaticScratch &ss = g_static[dev];
  if (ss.ptr == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr) {
      t_last_hip = (int)e;
      return LL_ERR_HIP;
    }
    ss.ptr = p;
  }
  if (ss.next_epoch + iters - 1 > 0xFFFFFFFFull) ss.init_needed = true;
  if (ss.init_needed) {
    const int st = ll_scratch_init(ss.ptr, kStaticStride, LL_MAX_RANKS, stream);
    if (st != LL_OK) return st;
    ss.init_needed = false;
    ss.next_epoch = 1;
  }
  *ptr = ss.ptr;
  *epoch = (uint32_t)ss.next_epoch;
  ss.next_epoch += iters;
  return LL_OK;
}

int ll_allreduce_static(const void *in, void *out, size_t count, ll_dtype dt, ll_op op, int nranks, void *stream,
                        ll_algo algo, uint32_t *epochs_used) {
  if (epochs_used != nullptr) *epochs_used = 0;
  if (in == nullptr || out == nullptr) return LL_ERR_INVALID;
  if (((uintptr_t)in % 16) != 0 || ((uintptr_t)out % 16) != 0) return LL_ERR_INVALID;
  if (nranks < 2 || nranks > LL_MAX_RANKS) return LL_ERR_INVALID;
  int st = check_dtype_op((int)dt, (int)op);
  if (st != LL_OK) return st;
  if ((int)algo < LL_ALGO_AUTO || (int)algo > LL_ALGO_TWOSHOT_LINE_WAVES) return LL_ERR_INVALID;
  switch (algo) {
    case LL_ALGO_ONESHOT_SENTINEL: case LL_ALGO_TWOSHOT_SENTINEL: case LL_ALGO_TWOSHOT_SENTINEL_OUT:
    case LL_ALGO_TWOSHOT_ATOMIC: case LL_ALGO_TWOSHOT_SENTINEL_WAVES: case LL_ALGO_ONESHOT_SENTINEL_WAVES:
      return LL_ERR_UNSUPPORTED;  // flagged protocols only
    default:
      break;
  }
  const int es = esize_of(dt);
  if (count > L::kMaxBufferedBytes / (uint64_t)es) return LL_ERR_UNSUPPORTED;  // beyond the largest message
  if (count == 0) return LL_OK;
  // the same iteration plan as buffered_call's, to reserve the epochs
  const uint64_t D = L::iter_capacity(kStaticStride, LL_MAX_RANKS);
  uint64_t iter_count = 0, iters = 0;
  buffered_iterations(count, es, D, &iter_count, &iters);
  if (iters > 0xFFFFFFFFull - 1) return LL_ERR_UNSUPPORTED;
  void *base = nullptr;
  uint32_t epoch = 0;
  st = static_scratch_of(iters, stream, &base, &epoch);
  if (st != LL_OK) return st;
  return buffered_call(in, out, count, dt, op, nranks, base, kStaticStride, LL_MAX_RANKS, true, epoch, stream, algo,
                       nullptr, epochs_used);
}

int ll_reduce_scatter_ex(void *sym_base, size_t rank_stride, void *out, size_t recvcount, ll_dtype dt, ll_op op,
                         int nranks, uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt) {
  int st = check_common(sym_base, rank_stride, out, nranks, epoch);
  if (st != LL_OK) return st;
  st = check_dtype_op((int)dt, (int)op);
  if (st != LL_OK) return st;
  if ((int)proto < LL_PROTO_AUTO || (int)proto > LL_PROTO_SENTINEL) return LL_ERR_INVALID;
  CallOpts o;
  st = resolve_opts(opt, &o);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  if (recvcount > L::kMaxInputBytes) return LL_ERR_UNSUPPORTED;
  const uint64_t chunk_bytes = (uint64_t)recvcount * es;
  const uint64_t in_bytes = chunk_bytes * nranks;
  if (overlaps(out, chunk_bytes * nranks, sym_base, (uint64_t)rank_stride * nranks)) return LL_ERR_INVALID;
  Region rg;
  st = region_of(rank_stride, nranks, in_bytes, &rg);
  if (st != LL_OK) return st;
  if (proto == LL_PROTO_AUTO) {
    proto = proto_choice(auto_proto(in_bytes, nranks, o.sentinel_ok(), false), auto_formats(rg.fmt, o));
    if (proto == LL_PROTO_AUTO) return LL_ERR_SCRATCH;
  }
  if ((rg.fmt & proto_fmt(proto)) == 0) return LL_ERR_SCRATCH;
  if (recvcount == 0) return LL_OK;
  Plan pl;
  pl.kind = use_wave_kernel(proto, in_bytes, nranks, false, o) ? K_RS_WAVES : K_RS;
  pl.dt = (int)dt;
  pl.P = nranks;
  pl.o = o;
  pl.proto = proto == LL_PROTO_LINE128 ? PR_LINE : (proto == LL_PROTO_SENTINEL ? PR_SENT : PR_LL);
  pl.a = base_args(sym_base, rank_stride, out, epoch);
  pl.a.n = (int64_t)recvcount;
  pl.a.al4 = (chunk_bytes % 4 == 0) ? 1u : 0u;
  pl.a.area = rg.area_of(pl.proto);
  pl.a.slot = slot_bytes(pl.proto, chunk_bytes);
  pl.units = units_of(pl.proto, chunk_bytes);
  return launch(pl, stream);
}

int ll_reduce_scatter(void *sym_base, size_t rank_stride, void *out, size_t recvcount, ll_dtype dt, ll_op op,
                      int nranks, uint32_t epoch, void *stream) {
  return ll_reduce_scatter_ex(sym_base, rank_stride, out, recvcount, dt, op, nranks, epoch, stream, LL_PROTO_AUTO,
                              nullptr);
}

int ll_allgather_ex(void *sym_base, size_t rank_stride, void *out, size_t sendcount, ll_dtype dt, int nranks,
                    uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt) {
  int st = check_common(sym_base, rank_stride, out, nranks, epoch);
  if (st != LL_OK) return st;
  st = check_dtype_op((int)dt, LL_SUM);
  if (st != LL_OK) return st;
  if ((int)proto < LL_PROTO_AUTO || (int)proto > LL_PROTO_SENTINEL) return LL_ERR_INVALID;
  CallOpts o;
  st = resolve_opts(opt, &o);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  if (sendcount > L::kMaxInputBytes) return LL_ERR_UNSUPPORTED;
  const uint64_t in_bytes = (uint64_t)sendcount * es;
  if (overlaps(out, in_bytes * nranks * nranks, sym_base, (uint64_t)rank_stride * nranks)) return LL_ERR_INVALID;
  Region rg;
  st = region_of(rank_stride, nranks, in_bytes, &rg);
  if (st != LL_OK) return st;
  if (proto == LL_PROTO_AUTO) {
    proto = proto_choice(auto_proto(in_bytes * nranks, nranks, o.sentinel_ok(), true), auto_formats(rg.fmt, o));
    if (proto == LL_PROTO_AUTO) return LL_ERR_SCRATCH;
  }
  if ((rg.fmt & proto_fmt(proto)) == 0) return LL_ERR_SCRATCH;
  if (sendcount == 0) return LL_OK;
  Plan pl;
  pl.kind = use_wave_kernel(proto, in_bytes * nranks, nranks, true, o) ? K_AG_WAVES : K_AG;
  pl.dt = (int)dt;
  pl.P = nranks;
  pl.o = o;
  pl.proto = proto == LL_PROTO_LINE128 ? PR_LINE : (proto == LL_PROTO_SENTINEL ? PR_SENT : PR_LL);
  pl.a = base_args(sym_base, rank_stride, out, epoch);
  pl.a.n = (int64_t)sendcount;
  pl.a.al4 = (in_bytes % 4 == 0) ? 1u : 0u;
  pl.a.area = rg.area_of(pl.proto);
  pl.a.slot = slot_bytes(pl.proto, in_bytes);
  pl.units = units_of(pl.proto, in_bytes);
  return launch(pl, stream);
}

int ll_allgather(void *sym_base, size_t rank_stride, void *out, size_t sendcount, ll_dtype dt, int nranks,
                 uint32_t epoch, void *stream) {
  return ll_allgather_ex(sym_base, rank_stride, out, sendcount, dt, nranks, epoch, stream, LL_PROTO_AUTO, nullptr);
}

// Broadcast / Reduce: one exchange in the one-shot slots of the chosen format.
static int rooted_call(Kind kind, void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, int root,
                       int nranks, uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt) {
  int st = check_common(sym_base, rank_stride, out, nranks, epoch);
  if (st != LL_OK) return st;
  if (root < 0 || root >= nranks) return LL_ERR_INVALID;
  if ((int)proto < LL_PROTO_AUTO || (int)proto > LL_PROTO_SENTINEL) return LL_ERR_INVALID;
  CallOpts o;
  st = resolve_opts(opt, &o);
  if (st != LL_OK) return st;
  const int es = esize_of(dt);
  if (count > L::kMaxInputBytes) return LL_ERR_UNSUPPORTED;
  const uint64_t in_bytes = (uint64_t)count * es;
  const uint64_t out_bytes = kind == K_BCAST ? in_bytes * nranks : in_bytes;
  if (overlaps(out, out_bytes, sym_base, (uint64_t)rank_stride * nranks)) return LL_ERR_INVALID;
  Region rg;
  st = region_of(rank_stride, nranks, in_bytes, &rg);
  if (st != LL_OK) return st;
  if (proto == LL_PROTO_AUTO) {
    proto = proto_choice(auto_proto_rooted(in_bytes, o.sentinel_ok()), auto_formats(rg.fmt, o));
    if (proto == LL_PROTO_AUTO) return LL_ERR_SCRATCH;
  }
  if ((rg.fmt & proto_fmt(proto)) == 0) return LL_ERR_SCRATCH;
  if (count == 0) return LL_OK;
  Plan pl;
  pl.kind = kind;
  pl.dt = (int)dt;
  pl.P = nranks;
  pl.o = o;
  pl.proto = proto == LL_PROTO_LINE128 ? PR_LINE : (proto == LL_PROTO_SENTINEL ? PR_SENT : PR_LL);
  pl.a = base_args(sym_base, rank_stride, out, epoch);
  pl.a.n = (int64_t)count;
  pl.a.al4 = (in_bytes % 4 == 0) ? 1u : 0u;
  pl.a.root = root;
  pl.a.area = rg.area_of(pl.proto);
  pl.a.slot = slot_bytes(pl.proto, in_bytes);
  pl.units = units_of(pl.proto, in_bytes);
  return launch(pl, stream);
}

int ll_broadcast(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, int root, int nranks,
                 uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt) {
  const int st = check_dtype_op((int)dt, LL_SUM);
  if (st != LL_OK) return st;
  return rooted_call(K_BCAST, sym_base, rank_stride, out, count, dt, root, nranks, epoch, stream, proto, opt);
}

int ll_reduce(void *sym_base, size_t rank_stride, void *out, size_t count, ll_dtype dt, ll_op op, int root,
              int nranks, uint32_t epoch, void *stream, ll_proto proto, const ll_options *opt) {
  const int st = check_dtype_op((int)dt, (int)op);
  if (st != LL_OK) return st;
  return rooted_call(K_REDUCE, sym_base, rank_stride, out, count, dt, root, nranks, epoch, stream, proto, opt);
}

int ll_check(void *stream) {
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  DevInfo d;
  int dev = 0;
  int rc = device_info(&d, &dev);
  if (rc != LL_OK) return rc;
  const int slot = slot_index(dev, stream, false);
  if (slot < 0) return LL_OK;  // no call has run on this stream
  uint32_t *word = d.status + 4 * slot;
  uint32_t st[4] = {0, 0, 0, 0};
  e = hipMemcpyAsync(st, word, sizeof st, hipMemcpyDeviceToHost, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  if (st[0] == 0) return LL_OK;
  const uint32_t zero[4] = {0, 0, 0, 0};
  e = hipMemcpyAsync(word, zero, sizeof zero, hipMemcpyHostToDevice, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  {
    // a timed-out call may have left packets that a later call on the
    // device's static scratch could take for its own: clear it first
    std::lock_guard<std::mutex> lk(g_static_mu);
    g_static[dev].init_needed = true;
  }
  t_last_timeout.rank = (int)st[1];
  t_last_timeout.missing = st[2];
  t_last_timeout.epoch = st[3];
  return st[0] == kStatusTimeout ? LL_ERR_TIMEOUT : LL_ERR_HIP;
}

int ll_last_timeout(int *rank, uint32_t *missing_peers, uint32_t *epoch) {
  if (rank) *rank = t_last_timeout.rank;
  if (missing_peers) *missing_peers = t_last_timeout.missing;
  if (epoch) *epoch = t_last_timeout.epoch;
  return LL_OK;
}

const char *ll_strerror(int status) {
  switch (status) {
    case LL_OK:
      return "success";
    case LL_ERR_INVALID:
      return "invalid argument";
    case LL_ERR_UNSUPPORTED:
      return "unsupported data type, operation or size";
    case LL_ERR_SCRATCH:
      return "the region cannot serve this call: input larger than its input capacity, or no area for the "
             "call's packet format (rank_stride too small, or sized for another algorithm)";
    case LL_ERR_HIP:
      snprintf(t_msg, sizeof t_msg, "HIP runtime error: %s", hipGetErrorString((hipError_t)t_last_hip));
      return t_msg;
    case LL_ERR_TIMEOUT:
      return "a flag wait timed out (a peer never published, or the epoch was reused)";
    default:
      return "unknown status";
  }
}

// ------------------------------------------------------------------ probes
static int probe_launch_check(int grid, int threads) {
  if (grid < 1 || grid > 65536) return LL_ERR_INVALID;
  if (threads < 64 || threads > 1024 || threads % 64 != 0) return LL_ERR_INVALID;
  return LL_OK;
}

static int hip_status() {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    t_last_hip = (int)e;
    return LL_ERR_HIP;
  }
  return LL_OK;
}

int ll_probe_empty(int grid, int threads, uint64_t *stamps, void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  hipLaunchKernelGGL(k_probe_empty, dim3(grid), dim3(threads), 0, (hipStream_t)stream, stamps);
  return hip_status();
}

int ll_probe_floor(const uint64_t *chase, uint64_t chase_len, uint64_t start, uint64_t *sink, int grid, int threads,
                   uint64_t *stamps, void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  if (chase == nullptr || sink == nullptr || start >= chase_len) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_floor, dim3(grid), dim3(threads), 0, (hipStream_t)stream, chase, start, sink, stamps);
  return hip_status();
}

int ll_probe_chase(const uint64_t *chase, uint64_t chase_len, uint64_t start, int steps, uint64_t *out3,
                   void *stream) {
  if (chase == nullptr || out3 == nullptr || start >= chase_len || steps < 1) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_chase, dim3(1), dim3(64), 0, (hipStream_t)stream, chase, chase_len, start, steps, out3);
  return hip_status();
}

int ll_probe_fence_l2(uint32_t *buf4k, int iters, uint64_t *out7, void *stream) {
  if (buf4k == nullptr || out7 == nullptr || iters < 1) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_fence_l2, dim3(1), dim3(64), 0, (hipStream_t)stream, buf4k, iters, out7);
  return hip_status();
}

int ll_probe_pingpong(uint32_t *flags8k, int rounds, int grid, int peer, uint64_t limit_ticks, uint64_t *out3,
                      void *stream) {
  if (flags8k == nullptr || out3 == nullptr || rounds < 1 || grid < 2 || grid > 1024 || peer < 1 || peer >= grid ||
      limit_ticks == 0)
    return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_pingpong, dim3(grid), dim3(64), 0, (hipStream_t)stream, flags8k, rounds, peer,
                     limit_ticks, out3);
  return hip_status();
}

int ll_probe_spin(uint64_t ticks, void *stream) {
  if (ticks == 0 || ticks > 100000000ull) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_spin, dim3(1), dim3(64), 0, (hipStream_t)stream, ticks);
  return hip_status();
}

// Per-call options of a benchmark loop: a copy of `opt` (NULL = defaults)
// whose tuning points at the stamps of call i.
struct BenchOpts {
  ll_options o;
  ll_tuning t;
  uint64_t *stamps;
  int stride;
  BenchOpts(const ll_options *opt, uint64_t *st, int sd) : stamps(st), stride(sd) {
    ll_options_init(&o);
    ll_tuning_init(&t);
    if (opt != nullptr) {
      o = *opt;
      if (opt->tuning != nullptr) t = *opt->tuning;
    }
    o.tuning = &t;
  }
  const ll_options *at(int i) {
    t.stamps = stamps ? stamps + (size_t)i * (size_t)stride : nullptr;
    return &o;
  }
};

static int bench_args(uint32_t first_epoch, int calls, const uint64_t *stamps, int stamp_stride,
                      const ll_options *opt) {
  if (calls < 1 || first_epoch == 0 || (uint64_t)first_epoch + (uint64_t)calls - 1 > 0xFFFFFFFFull)
    return LL_ERR_INVALID;
  if (stamps != nullptr && stamp_stride < 1) return LL_ERR_INVALID;
  if (opt != nullptr && (opt->size != sizeof(ll_options) ||
                         (opt->tuning != nullptr && opt->tuning->size != sizeof(ll_tuning))))
    return LL_ERR_INVALID;
  return LL_OK;
}

int ll_bench_allreduce(void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int nranks,
                       uint32_t first_epoch, int calls, int algo, const ll_options *opt, uint64_t *stamps,
                       int stamp_stride, void *stream) {
  int st = bench_args(first_epoch, calls, stamps, stamp_stride, opt);
  if (st != LL_OK) return st;
  BenchOpts bo(opt, stamps, stamp_stride);
  for (int i = 0; i < calls; ++i) {
    if (fills_output((ll_algo)algo)) {  // its precondition, timed with it
      st = ll_fill_sentinel(out, count, (ll_dtype)dt, nranks, stream);
      if (st != LL_OK) return st;
    }
    st = ll_allreduce_ex(sym_base, rank_stride, out, count, (ll_dtype)dt, LL_SUM, nranks, first_epoch + (uint32_t)i,
                         stream, (ll_algo)algo, bo.at(i));
    if (st != LL_OK) return st;
  }
  return LL_OK;
}

int ll_bench_rooted(int kind, void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int root,
                    int nranks, uint32_t first_epoch, int calls, int proto, const ll_options *opt,
                    uint64_t *stamps, int stamp_stride, void *stream) {
  if (kind != 0 && kind != 1) return LL_ERR_INVALID;
  int st = bench_args(first_epoch, calls, stamps, stamp_stride, opt);
  if (st != LL_OK) return st;
  BenchOpts bo(opt, stamps, stamp_stride);
  for (int i = 0; i < calls; ++i) {
    const uint32_t e = first_epoch + (uint32_t)i;
    st = kind == 0 ? ll_broadcast(sym_base, rank_stride, out, count, (ll_dtype)dt, root, nranks, e, stream,
                                  (ll_proto)proto, bo.at(i))
                   : ll_reduce(sym_base, rank_stride, out, count, (ll_dtype)dt, LL_SUM, root, nranks, e, stream,
                               (ll_proto)proto, bo.at(i));
    if (st != LL_OK) return st;
  }
  return LL_OK;
}

int ll_bench_reduce_scatter(void *sym_base, size_t rank_stride, void *out, size_t recvcount, int dt, int nranks,
                            uint32_t first_epoch, int calls, int proto, const ll_options *opt, uint64_t *stamps,
                            int stamp_stride, void *stream) {
  int st = bench_args(first_epoch, calls, stamps, stamp_stride, opt);
  if (st != LL_OK) return st;
  BenchOpts bo(opt, stamps, stamp_stride);
  for (int i = 0; i < calls; ++i) {
    st = ll_reduce_scatter_ex(sym_base, rank_stride, out, recvcount, (ll_dtype)dt, LL_SUM, nranks,
                              first_epoch + (uint32_t)i, stream, (ll_proto)proto, bo.at(i));
    if (st != LL_OK) return st;
  }
  return LL_OK;
}

int ll_bench_allgather(void *sym_base, size_t rank_stride, void *out, size_t sendcount, int dt, int nranks,
                       uint32_t first_epoch, int calls, int proto, const ll_options *opt, uint64_t *stamps,
                       int stamp_stride, void *stream) {
  int st = bench_args(first_epoch, calls, stamps, stamp_stride, opt);
  if (st != LL_OK) return st;
  BenchOpts bo(opt, stamps, stamp_stride);
  for (int i = 0; i < calls; ++i) {
    st = ll_allgather_ex(sym_base, rank_stride, out, sendcount, (ll_dtype)dt, nranks, first_epoch + (uint32_t)i,
                         stream, (ll_proto)proto, bo.at(i));
    if (st != LL_OK) return st;
  }
  return LL_OK;
}

int ll_bench_floor(const uint64_t *chase, uint64_t chase_len, uint64_t first_line, uint64_t line_step,
                   uint64_t *sink, int grid, int threads, int calls, uint64_t *stamps, int stamp_stride,
                   void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  if (chase == nullptr || sink == nullptr || calls < 1 || chase_len < 16) return LL_ERR_INVALID;
  if (stamps != nullptr && stamp_stride < 2 * grid) return LL_ERR_INVALID;
  const uint64_t lines = chase_len / 16;
  for (int i = 0; i < calls; ++i) {
    const uint64_t start = ((first_line + (uint64_t)i * line_step) % lines) * 16;
    hipLaunchKernelGGL(k_probe_floor, dim3(grid), dim3(threads), 0, (hipStream_t)stream, chase, start, sink,
                       stamps ? stamps + (size_t)i * (size_t)stamp_stride : nullptr);
  }
  return hip_status();
}

int ll_bench_empty(int grid, int threads, int calls, uint64_t *stamps, int stamp_stride, void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  if (calls < 1) return LL_ERR_INVALID;
  if (stamps != nullptr && stamp_stride < 2 * grid) return LL_ERR_INVALID;
  for (int i = 0; i < calls; ++i) {
    hipLaunchKernelGGL(k_probe_empty, dim3(grid), dim3(threads), 0, (hipStream_t)stream,
                       stamps ? stamps + (size_t)i * (size_t)stamp_stride : nullptr);
  }
  return hip_status();
}

int ll_bench_exchange(void *sym_base, size_t rank_stride, void *out, size_t count, int dt, int nranks,
                      uint32_t first_epoch, int calls, uint64_t *stamps, int stamp_stride, int *grid_out,
                      void *stream) {
  int st = check_common(sym_base, rank_stride, out, nranks, first_epoch);
  if (st != LL_OK) return st;
  st = check_dtype_op(dt, LL_SUM);
  if (st != LL_OK) return st;
  if (calls < 1 || (uint64_t)first_epoch + (uint64_t)calls - 1 > 0xFFFFFFFFull) return LL_ERR_INVALID;
  const uint64_t bytes = (uint64_t)count * (uint64_t)esize_of((ll_dtype)dt);
  if (bytes == 0 || bytes % 8 != 0) return LL_ERR_UNSUPPORTED;
  if (overlaps(out, bytes * nranks, sym_base, (uint64_t)rank_stride * nranks)) return LL_ERR_INVALID;
  Region rg;
  st = region_of(rank_stride, nranks, bytes, &rg);
  if (st != LL_OK) return st;
  if ((rg.fmt & L::kFmt8) == 0) return LL_ERR_SCRATCH;
  static kernel_fn const fns[LL_MAX_RANKS + 1] = {nullptr,
                                                  nullptr,
                                                  k_probe_exchange<2>,
                                                  k_probe_exchange<3>,
                                                  k_probe_exchange<4>,
                                                  k_probe_exchange<5>,
                                                  k_probe_exchange<6>,
                                                  k_probe_exchange<7>,
                                                  k_probe_exchange<8>};
  const kernel_fn fn = fns[nranks];
  const int threads = 64 * nranks;
  int cap_grid = 0;
  st = resident_grid(fn, threads, &cap_grid);
  if (st != LL_OK) return st;
  const uint64_t units = bytes / 8;
  const uint64_t W = (units + 63) / 64;
  if (W > (uint64_t)(cap_grid / nranks)) return LL_ERR_UNSUPPORTED;  // one tile per workgroup, all resident
  const int grid = (int)W * nranks;
  if (stamps != nullptr && stamp_stride < 2 * grid) return LL_ERR_INVALID;
  KArgs a = base_args(sym_base, rank_stride, out, first_epoch);
  a.n = (int64_t)bytes;
  a.area = rg.area_of(PR_LL);
  a.slot = slot_bytes(PR_LL, bytes);
  a.units = (int64_t)units;
  a.timeout = kDefaultTimeout;
  a.grid = (uint32_t)grid;
  a.block = (uint32_t)threads;
  a.clear = 1;  // as the one-shot wave kernels
  st = status_of(stream, &a.status);
  if (st != LL_OK) return st;
  for (int i = 0; i < calls; ++i) {
    a.epoch = first_epoch + (uint32_t)i;
    a.stamps = stamps ? stamps + (size_t)i * (size_t)stamp_stride : nullptr;
    hipLaunchKernelGGL(fn, dim3(grid), dim3(threads), 0, (hipStream_t)stream, a);
  }
  if (grid_out != nullptr) *grid_out = grid;
  return hip_status();
}

int ll_probe_xcd(uint32_t *ids, int grid, int threads, void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  if (ids == nullptr) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_xcd, dim3(grid), dim3(threads), 0, (hipStream_t)stream, ids);
  return hip_status();
}

int ll_probe_stream(const void *src, void *dst, size_t bytes, int mode, int grid, int threads, void *stream) {
  int st = probe_launch_check(grid, threads);
  if (st != LL_OK) return st;
  if (mode < 0 || mode > 2 || dst == nullptr || (mode != 2 && src == nullptr)) return LL_ERR_INVALID;
  if (bytes == 0 || bytes % 16 != 0 || ((uintptr_t)src | (uintptr_t)dst) % 16 != 0) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_stream, dim3(grid), dim3(threads), 0, (hipStream_t)stream, (const u32x4 *)src,
                     (u32x4 *)dst, (uint64_t)(bytes / 16), mode);
  return hip_status();
}

int ll_probe_litmus(uint32_t *buf, size_t buf_bytes, int grid, int lines, int iters, int reads, int layout,
                    unsigned long long *counts4, void *stream) {
  if (buf == nullptr || counts4 == nullptr) return LL_ERR_INVALID;
  if (grid < 2 || grid % 2 != 0 || grid > 512 || lines < 1 || iters < 1 || reads < 1) return LL_ERR_INVALID;
  if (layout != 0 && layout != 1) return LL_ERR_INVALID;
  if ((uint64_t)(grid / 2) * (uint64_t)lines * 128u > buf_bytes) return LL_ERR_INVALID;
  if ((uint64_t)lines * 128u > 0xFFFFFFFFull) return LL_ERR_INVALID;
  hipLaunchKernelGGL(k_probe_litmus, dim3(grid), dim3(256), 0, (hipStream_t)stream, buf, lines, iters, reads, layout,
                     counts4);
  return hip_status();
}

}  // extern "C"
