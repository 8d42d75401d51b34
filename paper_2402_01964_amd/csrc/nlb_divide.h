// nlb_divide.h -- exact division and remainder of 32-bit unsigned numbers by
// a divisor fixed for a launch, by multiplication.  Private to libnlb.so.
//
// The kernels split flat output indices into (row, column) and slot-row
// indices into (query, slot), so every 32-bit numerator that a launch can
// form must give the exact quotient.  The helpers below are plain integer
// arithmetic, identical in host and device code (the constants are
// computed on the host), so a host build checks the same source that the
// kernels compile.  Neither helper branches on the divisor: a branch on a
// launch constant splits the kernel's straight-line code and keeps the
// compiler from grouping the loads around it.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define NLB_HD __host__ __device__ __forceinline__
#else
#define NLB_HD inline
#endif

// floor(M f / 2^64) for a 32-bit f (the bits of the 96-bit product above
// bit 63, which fit in 32 bits): with M = Mh 2^32 + Ml,
// M f / 2^64 = (Mh f + Ml f / 2^32) / 2^32, and dropping the fraction of
// Ml f / 2^32 cannot move the floor.  Mh f + (Ml f >> 32) < 2^64.
NLB_HD uint64_t nlb_mulhi_64x32(uint64_t M, uint32_t f) {
    const uint64_t lo = (uint64_t)(uint32_t)M * f;
    const uint64_t hi = (M >> 32) * (uint64_t)f;
    return (hi + (lo >> 32)) >> 32;
}

// floor(f / d) for every 32-bit f and 1 <= d < 2^32 (Granlund and
// Montgomery, PLDI 1994, Theorem 4.2 and their round-up method).  With
// l = ceil(log2 d) and m = floor(2^(32 + l) / d) + 1, m d lies in
// (2^(32 + l), 2^(32 + l) + d] and d <= 2^l, so floor(f / d) =
// floor(m f / 2^(32 + l)) for every f < 2^32.  m lies in (2^32, 2^33), so
// it is kept as m' = m - 2^32 in [1, 2^32): floor(m f / 2^32) =
// f + floor(m' f / 2^32), a 33-bit sum, shifted right by l.  d = 1 gives
// m' = 1 and l = 0 and needs no special case, so the kernels never branch on
// the divisor.  The constant packs m' in its low word and l in its high
// word; it is computed on the host.
inline uint64_t nlb_div_magic(uint32_t d) {
    uint32_t l = 0;
    while (l < 32u && (1ull << l) < d) l++;
    // floor(2^64 / d) for l = 32: d is not a power of two there, so it
    // equals floor((2^64 - 1) / d).
    const uint64_t q = l < 32u ? (1ull << (32u + l)) / d : ~0ull / d;
    return (q + 1ull - (1ull << 32)) | ((uint64_t)l << 32);
}

NLB_HD uint32_t nlb_div(uint32_t f, uint64_t magic) {
    const uint64_t t = ((uint64_t)(uint32_t)magic * f) >> 32;
    return (uint32_t)((t + f) >> (uint32_t)(magic >> 32));
}

// floor(f / d) for f < 2^12 and 1 <= d <= 2^12 (a slot row of a sample tile
// divided by s) with one 24-bit multiply: for N = 12 and l = ceil(log2 d),
// m = floor(2^(12 + l) / d) + 1 meets the same condition as above, so
// floor(f / d) = floor(m f / 2^(12 + l)); m < 2^13, so m f < 2^25 and both
// factors fit the 24-bit multiplier.  d = 1 gives m = 4097, l = 0.  The
// constant packs m in its low word and 12 + l in its high word.
inline uint64_t nlb_div12_magic(uint32_t d) {
    uint32_t l = 0;
    while (l < 12u && (1u << l) < d) l++;
    const uint64_t m = (1ull << (12u + l)) / d + 1ull;
    return m | ((uint64_t)(12u + l) << 32);
}

NLB_HD uint32_t nlb_div12(uint32_t f, uint64_t magic) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __umul24(f, (uint32_t)magic) >> (uint32_t)(magic >> 32);
#else
    return ((f & 0xFFFFFFu) * ((uint32_t)magic & 0xFFFFFFu)) >> (uint32_t)(magic >> 32);
#endif
}

// f mod d for every 32-bit f and 1 <= d < 2^32, with M = nlb_mod_magic(d)
// = floor((2^64 - 1) / d) + 1 (Lemire, Kaser and Kurz, "Faster remainder by
// direct computation", 2019): the low 64 bits of M f hold the fraction of
// f / d, and multiplying that fraction by d gives the remainder in the high
// word.  d = 1 is encoded as M = 0, which gives 0 with no special case.
inline uint64_t nlb_mod_magic(uint32_t d) { return d <= 1u ? 0ull : ~0ull / d + 1ull; }

NLB_HD uint32_t nlb_mod(uint32_t f, uint64_t M, uint32_t d) {
    const uint64_t frac = M * f;
    return (uint32_t)nlb_mulhi_64x32(frac, d);
}
