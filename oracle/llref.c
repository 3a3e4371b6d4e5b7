/*
 * CPU oracle for the low-latency collectives -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load this library.  The product path (the HIP library and its Python
 * binding) never calls it and shares no code with it.
 *
 * What it computes is the plain definition of the collectives in the paper,
 * written out as slow, obviously correct loops:
 *
 *   AllReduce (Sec. III, opening; one-shot in Sec. III-A: every rank ends
 *   with the element-wise sum of all N rank buffers).  The summation is
 *   sequential in ascending rank order, accumulated in binary32, and the
 *   result is rounded once to the element type.  This follows the
 *   forward-error analysis of fl(sum x_i) at the end of Sec. IV, the
 *   conversion to an accumulator type done by recvReduce (Sec. V), and the
 *   requirement that every rank observe the same result (Sec. IV, "Algorithm
 *   Comparison").
 *
 *   ReduceScatter (Sec. III-A, two-shot): rank r keeps chunk r of the
 *   AllReduce result.
 *
 *   AllGather (Sec. III-A, two-shot): rank r ends with the concatenation of
 *   every rank's input, in rank order.
 *
 *   Broadcast and Reduce (Sec. V, the artifact's further low-latency
 *   collectives; their meaning is the usual one): Broadcast gives every rank
 *   a copy of the root's input; Reduce gives the root alone the reduced
 *   value, the same ascending-rank binary32 sum as AllReduce.
 *
 * Element types: dtype 0 = IEEE binary32, dtype 1 = bfloat16.  Values are
 * passed as raw bit patterns so nothing on the Python side reinterprets them.
 * bfloat16 -> binary32 is exact (shift left by 16); binary32 -> bfloat16 is
 * IEEE round-to-nearest-even, NaN kept NaN (quieted).
 *
 * Floating-point environment: every entry point forces the SSE control word
 * to round-to-nearest-even with flush-to-zero and denormals-are-zero off, so
 * subnormals take part in the arithmetic exactly as IEEE 754 says, and
 * restores the caller's control word on return.  Built with gcc
 * -O2 -fno-fast-math -ffp-contract=off; x86-64 uses SSE2 scalar arithmetic
 * (no x87 extended precision).
 *
 * Layouts (all dense, row-major by rank):
 *   ref_allreduce      in [P][count]          out [P][count]
 *   ref_reduce_scatter in [P][P*recvcount]    out [P][recvcount]
 *   ref_allgather      in [P][sendcount]      out [P][P*sendcount]
 *   ref_broadcast      in [P][count]          out [P][count]
 *   ref_reduce         in [P][count]          out [count]       (the root's result)
 *
 * Return value: 0 on success, -1 on a bad argument.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#if defined(__x86_64__)
#include <xmmintrin.h>
#endif

#define REF_F32 0
#define REF_BF16 1

/* ---- floating-point environment ------------------------------------------------ */

static unsigned int fpenv_enter(void) {
#if defined(__x86_64__)
  unsigned int saved = _mm_getcsr();
  unsigned int csr = saved;
  csr &= ~(1u << 15);        /* FTZ off */
  csr &= ~(1u << 6);         /* DAZ off */
  csr &= ~(3u << 13);        /* rounding control: nearest-even */
  _mm_setcsr(csr);
  return saved;
#else
  return 0;
#endif
}

static void fpenv_leave(unsigned int saved) {
#if defined(__x86_64__)
  _mm_setcsr(saved);
#else
  (void)saved;
#endif
}

/* ---- element conversions ------------------------------------------------------- */

static float bits_to_f32(uint32_t u) {
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static uint32_t f32_to_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  return u;
}

/* bfloat16 is the upper half of a binary32: widening is exact. */
static float bf16_widen(uint16_t h) { return bits_to_f32((uint32_t)h << 16); }

/* binary32 -> bfloat16, round to nearest, ties to even. */
static uint16_t bf16_narrow_rne(float f) {
  uint32_t u = f32_to_bits(f);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0) {
    /* NaN: keep sign and the top payload bits, force the quiet bit. */
    return (uint16_t)((u >> 16) | 0x0040u);
  }
  /* Add half an ulp of the target format, plus one more unit when the kept
     part is odd, so exact halves go to the even neighbour.  A carry out of
     the mantissa correctly bumps the exponent (and reaches Inf on overflow). */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

static float load_elem(const void *base, size_t idx, int dtype) {
  if (dtype == REF_F32) {
    return bits_to_f32(((const uint32_t *)base)[idx]);
  }
  return bf16_widen(((const uint16_t *)base)[idx]);
}

static void store_elem(void *base, size_t idx, int dtype, float v) {
  if (dtype == REF_F32) {
    ((uint32_t *)base)[idx] = f32_to_bits(v);
  } else {
    ((uint16_t *)base)[idx] = bf16_narrow_rne(v);
  }
}

static size_t elem_size(int dtype) { return dtype == REF_F32 ? 4u : 2u; }

static int bad_args(const void *in, const void *out, int dtype, int nranks) {
  if (in == NULL || out == NULL) return 1;
  if (dtype != REF_F32 && dtype != REF_BF16) return 1;
  if (nranks < 1) return 1;
  return 0;
}

/* The reduced value of element i: x_0 + x_1 + ... + x_{P-1}, left to right,
   each addition rounded to binary32.  The first operand is x_0 itself (not
   +0.0 + x_0), so a sum of negative zeros stays -0.0. */
static float reduce_elem(const void *in, size_t row_elems, size_t i, int dtype, int nranks) {
  const unsigned char *base = (const unsigned char *)in;
  size_t row_bytes = row_elems * elem_size(dtype);
  volatile float acc = load_elem(base, i, dtype);
  for (int q = 1; q < nranks; ++q) {
    float x = load_elem(base + (size_t)q * row_bytes, i, dtype);
    acc = acc + x;
  }
  return acc;
}

/* ---- collectives ---------------------------------------------------------------- */

int ref_allreduce(const void *in, void *out, size_t count, int dtype, int nranks) {
  if (bad_args(in, out, dtype, nranks)) return -1;
  unsigned int env = fpenv_enter();
  size_t es = elem_size(dtype);
  unsigned char *obase = (unsigned char *)out;
  for (size_t i = 0; i < count; ++i) {
    float y = reduce_elem(in, count, i, dtype, nranks);
    for (int r = 0; r < nranks; ++r) {
      store_elem(obase + (size_t)r * count * es, i, dtype, y);
    }
  }
  fpenv_leave(env);
  return 0;
}

int ref_reduce_scatter(const void *in, void *out, size_t recvcount, int dtype, int nranks) {
  if (bad_args(in, out, dtype, nranks)) return -1;
  unsigned int env = fpenv_enter();
  size_t es = elem_size(dtype);
  size_t row = (size_t)nranks * recvcount;
  unsigned char *obase = (unsigned char *)out;
  for (int r = 0; r < nranks; ++r) {
    for (size_t j = 0; j < recvcount; ++j) {
      float y = reduce_elem(in, row, (size_t)r * recvcount + j, dtype, nranks);
      store_elem(obase + (size_t)r * recvcount * es, j, dtype, y);
    }
  }
  fpenv_leave(env);
  return 0;
}

int ref_allgather(const void *in, void *out, size_t sendcount, int dtype, int nranks) {
  if (bad_args(in, out, dtype, nranks)) return -1;
  size_t es = elem_size(dtype);
  const unsigned char *ibase = (const unsigned char *)in;
  unsigned char *obase = (unsigned char *)out;
  size_t block = sendcount * es;
  for (int r = 0; r < nranks; ++r) {
    for (int q = 0; q < nranks; ++q) {
      memcpy(obase + ((size_t)r * nranks + q) * block, ibase + (size_t)q * block, block);
    }
  }
  return 0;
}

int ref_broadcast(const void *in, void *out, size_t count, int dtype, int nranks, int root) {
  if (bad_args(in, out, dtype, nranks) || root < 0 || root >= nranks) return -1;
  size_t block = count * elem_size(dtype);
  const unsigned char *src = (const unsigned char *)in + (size_t)root * block;
  unsigned char *obase = (unsigned char *)out;
  for (int r = 0; r < nranks; ++r) memcpy(obase + (size_t)r * block, src, block);
  return 0;
}

int ref_reduce(const void *in, void *out, size_t count, int dtype, int nranks, int root) {
  if (bad_args(in, out, dtype, nranks) || root < 0 || root >= nranks) return -1;
  unsigned int env = fpenv_enter();
  for (size_t i = 0; i < count; ++i) store_elem(out, i, dtype, reduce_elem(in, count, i, dtype, nranks));
  fpenv_leave(env);
  return 0;
}

/* Single conversions, exported so the tests can pin them on their own. */
uint16_t ref_bf16_from_f32_bits(uint32_t u) {
  unsigned int env = fpenv_enter();
  uint16_t h = bf16_narrow_rne(bits_to_f32(u));
  fpenv_leave(env);
  return h;
}

uint32_t ref_f32_bits_from_bf16(uint16_t h) { return f32_to_bits(bf16_widen(h)); }
