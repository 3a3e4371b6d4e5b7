// Kernel instantiations for one rank count, LL_INST_P (set by the build: this
// unit is compiled once per P in 2..8).
#include <type_traits>

#include "ll_table.hpp"

#ifndef LL_INST_P
#error "LL_INST_P (the rank count of this unit) must be defined"
#endif

namespace llc {
namespace {

template <class Pr, int DT, int P>
void fill_row(kernel_fn *row) {
  row[K_ONESHOT] = k_oneshot<Pr, DT, P>;
  row[K_TWOSHOT] = k_twoshot<Pr, DT, P>;
  row[K_RS] = k_reduce_scatter<Pr, DT, P>;
  row[K_AG] = k_allgather<Pr, DT, P>;
  row[K_ONESHOT_WAVES] = nullptr;
  row[K_BCAST] = k_broadcast<Pr, DT, P>;
  row[K_REDUCE] = k_reduce<Pr, DT, P>;
  row[K_TWOSHOT_OUT] = nullptr;
  row[K_TWOSHOT_ATOMIC] = nullptr;
  row[K_TWOSHOT_WAVES] = nullptr;
  row[K_RS_WAVES] = nullptr;
  row[K_AG_WAVES] = nullptr;
  if constexpr (std::is_same<Pr, ProtoSent>::value) {
    row[K_TWOSHOT_OUT] = k_twoshot<ProtoSent, DT, P, true>;
    row[K_TWOSHOT_ATOMIC] = k_twoshot_atomic<DT, P>;
  }
}

template <int M, int P>
void fill_twaves(Table *t) {
  t->twaves[M][0][0][0][P] = k_twoshot_waves<ProtoLL, 0, P, 1, M>;
  t->twaves[M][0][0][1][P] = k_twoshot_waves<ProtoLL, 1, P, 1, M>;
  t->twaves[M][1][0][0][P] = k_twoshot_waves<ProtoLL, 0, P, 2, M>;
  t->twaves[M][1][0][1][P] = k_twoshot_waves<ProtoLL, 1, P, 2, M>;
  t->twaves[M][2][0][0][P] = k_twoshot_waves<ProtoLL, 0, P, 4, M>;
  t->twaves[M][2][0][1][P] = k_twoshot_waves<ProtoLL, 1, P, 4, M>;
  t->twaves[M][0][1][0][P] = k_twoshot_waves<ProtoSent, 0, P, 1, M>;
  t->twaves[M][0][1][1][P] = k_twoshot_waves<ProtoSent, 1, P, 1, M>;
  t->twaves[M][1][1][0][P] = k_twoshot_waves<ProtoSent, 0, P, 2, M>;
  t->twaves[M][1][1][1][P] = k_twoshot_waves<ProtoSent, 1, P, 2, M>;
  t->twaves[M][2][1][0][P] = k_twoshot_waves<ProtoSent, 0, P, 4, M>;
  t->twaves[M][2][1][1][P] = k_twoshot_waves<ProtoSent, 1, P, 4, M>;
  t->twaves[M][0][2][0][P] = k_twoshot_waves<ProtoLine, 0, P, 1, M>;
  t->twaves[M][0][2][1][P] = k_twoshot_waves<ProtoLine, 1, P, 1, M>;
  t->twaves[M][1][2][0][P] = k_twoshot_waves<ProtoLine, 0, P, 2, M>;
  t->twaves[M][1][2][1][P] = k_twoshot_waves<ProtoLine, 1, P, 2, M>;
  t->twaves[M][2][2][0][P] = k_twoshot_waves<ProtoLine, 0, P, 4, M>;
  t->twaves[M][2][2][1][P] = k_twoshot_waves<ProtoLine, 1, P, 4, M>;
}

// One unit per lane for every packet format and mode; two for the AllReduce
// with lines only (with 8-byte packets and sentinel units the multi-tile
// kernel at two units per lane measured as fast or faster).
template <int M, int P>
void fill_ttile_u1(Table *t) {
  t->ttile[M][0][0][0][P] = k_twoshot_tile<ProtoLL, 0, P, 1, M>;
  t->ttile[M][0][0][1][P] = k_twoshot_tile<ProtoLL, 1, P, 1, M>;
  t->ttile[M][0][1][0][P] = k_twoshot_tile<ProtoSent, 0, P, 1, M>;
  t->ttile[M][0][1][1][P] = k_twoshot_tile<ProtoSent, 1, P, 1, M>;
  t->ttile[M][0][2][0][P] = k_twoshot_tile<ProtoLine, 0, P, 1, M>;
  t->ttile[M][0][2][1][P] = k_twoshot_tile<ProtoLine, 1, P, 1, M>;
}

template <int P>
void fill_ttile(Table *t) {
  fill_ttile_u1<0, P>(t);
  fill_ttile_u1<1, P>(t);
  fill_ttile_u1<2, P>(t);
  t->ttile[0][1][2][0][P] = k_twoshot_tile<ProtoLine, 0, P, 2, 0>;
  t->ttile[0][1][2][1][P] = k_twoshot_tile<ProtoLine, 1, P, 2, 0>;
}

template <int P>
void fill_rtile(Table *t) {
  t->rtile[0][0][0][P] = k_rooted_tile<ProtoLL, 0, P, 0>;
  t->rtile[0][0][1][P] = k_rooted_tile<ProtoLL, 1, P, 0>;
  t->rtile[0][1][0][P] = k_rooted_tile<ProtoLL, 0, P, 1>;
  t->rtile[0][1][1][P] = k_rooted_tile<ProtoLL, 1, P, 1>;
  t->rtile[1][0][0][P] = k_rooted_tile<ProtoSent, 0, P, 0>;
  t->rtile[1][0][1][P] = k_rooted_tile<ProtoSent, 1, P, 0>;
  t->rtile[1][1][0][P] = k_rooted_tile<ProtoSent, 0, P, 1>;
  t->rtile[1][1][1][P] = k_rooted_tile<ProtoSent, 1, P, 1>;
}

template <int P>
void fill(Table *t) {
  fill_row<ProtoLL, 0, P>(t->k[PR_LL][0][P]);
  fill_row<ProtoLL, 1, P>(t->k[PR_LL][1][P]);
  fill_row<ProtoLine, 0, P>(t->k[PR_LINE][0][P]);
  fill_row<ProtoLine, 1, P>(t->k[PR_LINE][1][P]);
  fill_row<ProtoSent, 0, P>(t->k[PR_SENT][0][P]);
  fill_row<ProtoSent, 1, P>(t->k[PR_SENT][1][P]);
  t->waves[0][0][0][P] = k_oneshot_waves<ProtoLL, 0, P, 1>;
  t->waves[0][0][1][P] = k_oneshot_waves<ProtoLL, 1, P, 1>;
  t->waves[1][0][0][P] = k_oneshot_waves<ProtoLL, 0, P, 2>;
  t->waves[1][0][1][P] = k_oneshot_waves<ProtoLL, 1, P, 2>;
  t->waves[2][0][0][P] = k_oneshot_waves<ProtoLL, 0, P, 4>;
  t->waves[2][0][1][P] = k_oneshot_waves<ProtoLL, 1, P, 4>;
  t->waves[0][1][0][P] = k_oneshot_waves<ProtoSent, 0, P, 1>;
  t->waves[0][1][1][P] = k_oneshot_waves<ProtoSent, 1, P, 1>;
  t->waves[1][1][0][P] = k_oneshot_waves<ProtoSent, 0, P, 2>;
  t->waves[1][1][1][P] = k_oneshot_waves<ProtoSent, 1, P, 2>;
  t->waves[2][1][0][P] = k_oneshot_waves<ProtoSent, 0, P, 4>;
  t->waves[2][1][1][P] = k_oneshot_waves<ProtoSent, 1, P, 4>;
  t->waves[0][2][0][P] = k_oneshot_waves<ProtoLine, 0, P, 1>;
  t->waves[0][2][1][P] = k_oneshot_waves<ProtoLine, 1, P, 1>;
  t->waves[1][2][0][P] = k_oneshot_waves<ProtoLine, 0, P, 2>;
  t->waves[1][2][1][P] = k_oneshot_waves<ProtoLine, 1, P, 2>;
  t->waves[2][2][0][P] = k_oneshot_waves<ProtoLine, 0, P, 4>;
  t->waves[2][2][1][P] = k_oneshot_waves<ProtoLine, 1, P, 4>;
  t->tile[0][0][P] = k_oneshot_tile<ProtoLL, 0, P>;
  t->tile[0][1][P] = k_oneshot_tile<ProtoLL, 1, P>;
  t->tile[1][0][P] = k_oneshot_tile<ProtoSent, 0, P>;
  t->tile[1][1][P] = k_oneshot_tile<ProtoSent, 1, P>;
  t->tile[2][0][P] = k_oneshot_line_tile<0, P>;
  t->tile[2][1][P] = k_oneshot_line_tile<1, P>;
  fill_ttile<P>(t);
  fill_rtile<P>(t);
  fill_twaves<0, P>(t);
  fill_twaves<1, P>(t);
  fill_twaves<2, P>(t);
}

}  // namespace

#define LL_FILL_NAME2(p) fill_table_p##p
#define LL_FILL_NAME(p) LL_FILL_NAME2(p)
void LL_FILL_NAME(LL_INST_P)(Table *t) { fill<LL_INST_P>(t); }

}  // namespace llc
