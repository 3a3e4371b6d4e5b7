// The table of kernel instantiations the host dispatches to.
//
// Every kernel is a template over the packet format, the element type and the
// rank count P (and, for the wave-per-peer kernels, the units per lane and the
// mode).  The instantiations for one P are compiled in a unit of their own
// (ll_inst.hip, built once per P), so the seven units build in parallel; the
// host unit (llcoll.hip) only holds their addresses.
#pragma once

#include "ll_kernels.hpp"

namespace llc {

enum Kind {
  K_ONESHOT = 0,
  K_TWOSHOT = 1,
  K_RS = 2,
  K_AG = 3,
  K_ONESHOT_WAVES = 4,
  K_TWOSHOT_OUT = 5,
  K_TWOSHOT_ATOMIC = 6,
  K_BCAST = 7,
  K_REDUCE = 8,
  K_TWOSHOT_WAVES = 9,
  K_RS_WAVES = 10,
  K_AG_WAVES = 11,
  K_KINDS = 12
};
enum Proto { PR_LL = 0, PR_LINE = 1, PR_SENT = 2, PR_COUNT = 3 };
constexpr int kMaxRanks = 8;

typedef void (*kernel_fn)(KArgs);

struct Table {
  kernel_fn k[PR_COUNT][2][kMaxRanks + 1][K_KINDS];
  // one-shot, one wave per peer: [log2 U][8-byte packets, sentinel, lines][dtype][P]
  kernel_fn waves[3][3][2][kMaxRanks + 1];
  // two-shot, one wave per peer: [AllReduce, ReduceScatter, AllGather][log2 U][8-byte, sentinel, lines][dtype][P]
  kernel_fn twaves[3][3][3][2][kMaxRanks + 1];
  // one-shot, one tile per workgroup: [8-byte packets, sentinel, lines][dtype][P]
  kernel_fn tile[3][2][kMaxRanks + 1];
  // two-shot, one tile per workgroup: [AllReduce, ReduceScatter, AllGather][log2 U][8-byte packets, sentinel,
  // lines][dtype][P]
  kernel_fn ttile[3][2][3][2][kMaxRanks + 1];
  // Broadcast / Reduce, one tile per workgroup: [8-byte packets, sentinel][Broadcast, Reduce][dtype][P]
  kernel_fn rtile[2][2][2][kMaxRanks + 1];
};

// Defined in the unit built for that rank count.
void fill_table_p2(Table *t);
void fill_table_p3(Table *t);
void fill_table_p4(Table *t);
void fill_table_p5(Table *t);
void fill_table_p6(Table *t);
void fill_table_p7(Table *t);
void fill_table_p8(Table *t);

}  // namespace llc
