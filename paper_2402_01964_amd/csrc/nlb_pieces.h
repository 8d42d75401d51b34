// nlb_pieces.h -- gathered feature rows read in fixed-form pieces, shared by
// the aggregation and status-update kernels.
//
// A piece is one lane's eight consecutive elements c .. c+7 of a row, in one
// of three forms fixed per row matrix:
//   kBf16Vec  bf16 rows, size and base 16-byte aligned: one 16-byte load;
//   kBf16Word bf16 rows, size and base 4-byte aligned: four 4-byte loads;
//   kF32Vec   fp32 rows, size and base 16-byte aligned: two 16-byte loads.
// Each load then lies wholly inside or wholly past the row (the width is a
// multiple of 8, 2 or 4 elements respectively); a load past it reads the
// row's start instead (in bounds) and is zeroed when used.  Loading and use
// are separate steps so that a caller can put many loads in flight before it
// waits for the first.
#pragma once

#include "nlb_internal.h"

namespace {

constexpr int kBf16Vec = 0, kBf16Word = 1, kF32Vec = 2;

// The form of a row matrix, or -1 when none applies.
inline int piece_kind(uint32_t row_bytes, const void *base, bool bf16) {
    const uintptr_t a = (uintptr_t)base;
    if (row_bytes % 16 == 0 && a % 16 == 0) return bf16 ? kBf16Vec : kF32Vec;
    if (bf16 && row_bytes % 4 == 0 && a % 4 == 0) return kBf16Word;
    return -1;
}

template <int KIND>
struct Piece8 {
    u32x4 w[KIND == kF32Vec ? 2 : 1];
};

template <int KIND>
__device__ __forceinline__ void load_piece(const uint8_t *row, uint32_t dim, uint32_t c, Piece8<KIND> &r) {
    if constexpr (KIND == kBf16Vec) {
        r.w[0] = *(const u32x4 *)(row + (c + 8u <= dim ? 2u * c : 0u));
    } else if constexpr (KIND == kBf16Word) {
#pragma unroll
        for (int j = 0; j < 4; j++)
            r.w[0][j] = *(const uint32_t *)(row + (c + 2u * j + 2u <= dim ? 2u * (c + 2u * j) : 0u));
    } else {
        r.w[0] = *(const u32x4 *)(row + (c + 4u <= dim ? 4u * c : 0u));
        r.w[1] = *(const u32x4 *)(row + (c + 8u <= dim ? 4u * c + 16u : 0u));
    }
}

// bf16 forms: the piece's packed bf16 pairs, zero where `ok` is false or
// past the row.
template <int KIND>
__device__ __forceinline__ u32x4 piece_bf16_bits(const Piece8<KIND> &r, uint32_t dim, uint32_t c, bool ok) {
    static_assert(KIND != kF32Vec, "bf16 forms only");
    u32x4 w;
#pragma unroll
    for (int j = 0; j < 4; j++) {
        const bool in = ok && (KIND == kBf16Vec ? c + 8u <= dim : c + 2u * j + 2u <= dim);
        w[j] = in ? r.w[0][j] : 0u;
    }
    return w;
}

// Any form: the piece's values as fp32, zero where `ok` is false or past the
// row.
template <int KIND>
__device__ __forceinline__ void piece_floats(const Piece8<KIND> &r, uint32_t dim, uint32_t c, bool ok,
                                             float v[8]) {
    if constexpr (KIND == kF32Vec) {
        const bool in0 = ok && c + 4u <= dim, in1 = ok && c + 8u <= dim;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            v[i] = in0 ? __uint_as_float(r.w[0][i]) : 0.0f;
            v[4 + i] = in1 ? __uint_as_float(r.w[1][i]) : 0.0f;
        }
    } else {
        const u32x4 w = piece_bf16_bits<KIND>(r, dim, c, ok);
#pragma unroll
        for (int j = 0; j < 4; j++) {
            v[2 * j] = __uint_as_float(w[j] << 16);
            v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
        }
    }
}

}  // namespace
