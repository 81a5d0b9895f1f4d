/*
 * Division of a 32-bit unsigned numerator by a runtime-constant divisor with
 * one multiply-high, one add and one shift (Granlund & Montgomery, "Division
 * by invariant integers using multiplication", PLDI 1994, Sec. 4).
 *
 * For a divisor d in [1, 2^31): l = ceil(log2 d),
 * magic = floor(2^32 * (2^l - d) / d) + 1, and for every n < 2^31
 *   n / d == (umulhi(n, magic) + n) >> l.
 * (n < 2^31 keeps the 32-bit add from overflowing.)
 *
 * Shared by host code (which computes magic/shift once per call) and device
 * code (which divides a vector index by the row length in vectors).
 */
#ifndef IABN_DIVMAGIC_H
#define IABN_DIVMAGIC_H

#include <stdint.h>

#if defined(__HIPCC__)
#define IABN_HD __host__ __device__
#else
#define IABN_HD
#endif

typedef struct {
    uint32_t magic;
    uint32_t shift;
} iabn_divmagic_t;

static inline IABN_HD iabn_divmagic_t iabn_divmagic_make(uint32_t d) {
    iabn_divmagic_t r;
    uint32_t l = 0;
    while (l < 32 && (1ull << l) < (uint64_t)d) ++l;
    r.magic = (uint32_t)((((1ull << l) - (uint64_t)d) << 32) / (uint64_t)d + 1ull);
    r.shift = l;
    return r;
}

static inline IABN_HD uint32_t iabn_divmagic_div(uint32_t n, iabn_divmagic_t m) {
    const uint32_t hi = (uint32_t)(((uint64_t)n * (uint64_t)m.magic) >> 32);
    return (hi + n) >> m.shift;
}

#endif /* IABN_DIVMAGIC_H */
