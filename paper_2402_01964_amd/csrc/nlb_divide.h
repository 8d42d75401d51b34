// nlb_divide.h -- exact division and remainder of 32-bit unsigned numbers by
// a divisor fixed for a launch, by multiplication.  Private to libnlb.so.
//
// The kernels split flat output indices into (row, column) and slot-row
// indices into (query, slot), so every 32-bit numerator that a launch can
// form must give the exact quotient.  Both helpers below are plain integer
// arithmetic, identical in host and device code, so a host build checks
// the same source that the kernels compile.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define NLB_HD __host__ __device__ __forceinline__
#else
#define NLB_HD inline
#endif

// High 64 bits of M * f for a 32-bit f: with M = Mh 2^32 + Ml,
// M f / 2^64 = (Mh f + Ml f / 2^32) / 2^32, and dropping the fraction of
// Ml f / 2^32 cannot move the floor.  Mh f + (Ml f >> 32) < 2^64.
NLB_HD uint64_t nlb_mulhi_64x32(uint64_t M, uint32_t f) {
    const uint64_t lo = (uint64_t)(uint32_t)M * f;
    const uint64_t hi = (M >> 32) * (uint64_t)f;
    return (hi + (lo >> 32)) >> 32;
}

// floor(f / d) for every 32-bit f and 1 <= d < 2^32, given
// M = nlb_div_magic(d) (Granlund and Montgomery, PLDI 1994; the form of
// Lemire, Kaser and Kurz, 2019).  For d >= 2, M = floor((2^64 - 1) / d) + 1
// lies in [2^64 / d, 2^64 / d + 1), so M f / 2^64 lies in
// [f / d, f / d + f / 2^64); the fraction of f / d is at most (d - 1) / d and
// f / 2^64 < 1 / d because f d < 2^64, so the floor is exact.  d = 1 would
// need M = 2^64, which does not fit: it is encoded as M = 0 and the quotient
// is f itself.
NLB_HD uint64_t nlb_div_magic(uint32_t d) { return d <= 1u ? 0ull : ~0ull / d + 1ull; }

NLB_HD uint32_t nlb_div(uint32_t f, uint64_t M) {
    return M ? (uint32_t)nlb_mulhi_64x32(M, f) : f;
}

// f mod d for every 32-bit f and 1 <= d < 2^32, with M = nlb_div_magic(d)
// (Lemire, Kaser and Kurz, "Faster remainder by direct computation", 2019):
// the low 64 bits of M f hold the fraction of f / d, and multiplying that
// fraction by d gives the remainder in the high word.  d = 1 (M = 0) gives 0.
NLB_HD uint32_t nlb_mod(uint32_t f, uint64_t M, uint32_t d) {
    const uint64_t frac = M * f;
    return (uint32_t)nlb_mulhi_64x32(frac, d);
}
