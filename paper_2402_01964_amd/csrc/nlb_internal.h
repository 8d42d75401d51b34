// nlb_internal.h -- definitions shared by the library's HIP sources: the
// table handle, the key-word format, and device helpers.  Private to
// libnlb.so; the public interface is include/nlb.h.
//
// Table layout in HBM.  Node n owns one block of `block_bytes` bytes at
// blocks + n * block_bytes: s 64-bit keys, then s 32-bit neighbour ids.
// block_bytes is the smallest of 16, 32, 64, 128, 256, 384, ... that holds
// 12*s bytes, so a block of s <= 10 sits in one 128-byte cache line and a
// query reads its whole table with one line fetch.
//
// Key word (0 = empty slot):
//   bits 63..62  class: 3 = offer whose coin passed, 1 = offer whose coin failed
//   bits 61..30  arrival index e (class 3) or its complement ~e (class 1)
//   bits 29..0   timestamp t (< 2^30)
// Batch insertion must equal sequential insertion.  Sequentially, a slot
// ends the batch holding the latest offer whose coin passed; if none passed,
// it keeps its old entry, or, when it was empty, the first offer of the
// batch (an empty slot always accepts).  With the encoding above this is a
// plain unsigned maximum over the old word and all offer words: any passed
// offer beats every class-1 word and older passed entries (larger e wins);
// a failed offer can only win against an empty word, and among failed
// offers the smallest e wins (largest ~e).  A stored class-1 word keeps
// losing to later class-1 offers (smaller ~e), so stored words never need
// rewriting.  Pass 1 (resolve) applies 64-bit atomicMax per offer; pass 2
// (commit) lets the offer whose word survived write the neighbour id.
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/nlb.h"
#include "nlb_divide.h"

namespace {

constexpr uint64_t kClassPass = 3ull << 62;
constexpr uint64_t kClassFail = 1ull << 62;
constexpr uint32_t kTimeBits = 30;
constexpr uint32_t kTimeMask = (1u << kTimeBits) - 1u;
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;  // SplitMix64 state increment

// Device status words, kept after the slot blocks (32-bit words):
//   [0]     error flags (kStatusRange | kStatusOrder)
//   [1]     timestamp of the last link inserted so far
//   [4..5]  first arrival index of the batch in flight (64-bit; written by
//           insert_resolve, read by insert_commit)
//   [6..7]  links inserted so far (64-bit): the next batch's first arrival
//           index (read by insert_resolve, advanced by insert_commit)
// No kernel writes a word its own workgroups read, so the two insert kernels
// keep the stream position on the device without atomics or a last-finisher
// test, and an insert replayed from a captured HIP graph continues the stream.
constexpr uint32_t kStatusRange = 1u;   // node id out of range, or the arrival index would pass 2^32 - 2
constexpr uint32_t kStatusOrder = 2u;   // timestamp >= 2^30 or decreasing
constexpr uint32_t kWordLastT = 1, kWordBatch = 4, kWordLinks = 6;
constexpr size_t kStatusBytes = 256;

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------- cosine
// Arguments beyond the fast path's range: the device libm's double cos,
// which reduces exactly.  Kept out of line so that its registers do not
// weigh on the kernels (time encodings never reach it in practice).
__device__ __attribute__((noinline)) float cos_fp32_wide(float x) {
    return (float)cos((double)x);
}

// cos of an fp32 argument.  The argument is converted to revolutions in
// double, y = x / (2 pi), and reduced to f = y - rint(y) in [-1/2, 1/2]; for
// |x| < 2^33 the double product leaves f within 2.7e-7 revolutions of exact
// (half an ulp of y plus the constant's error), within 3.3e-8 for |x| < 1e9.
// The hardware cosine (v_cos_f32, cos(2 pi f)) then evaluates the reduced
// fraction; measured on gfx950 over a dense grid of [-1/2, 1/2] its error is
// below 1.3e-7.  Against a double-precision cosine the whole function stays
// below 3e-7 absolute for |x| < 1e9 and below 2e-6 for |x| < 2^33.
constexpr float kCosFastLimit = 8589934592.0f;   // 2^33

// The fast path alone, for a caller that has checked |x| < kCosFastLimit.
__device__ __forceinline__ float cos_fp32_small(float x) {
    const double y = (double)x * 0.15915494309189533577;
    const float f = (float)(y - __builtin_rint(y));
    return __builtin_amdgcn_cosf(f);
}

// Bits 1 .. 192 of the binary fraction of 1 / (2 pi) = 0.159154943...,
// most significant first (derived from Machin's formula for pi in exact
// integer arithmetic by inv2pi_bits.py).
__device__ const uint32_t kInv2PiBits[6] = {0x28be60dbu, 0x9391054au, 0x7f09d5f4u,
                                            0x7d4d3770u, 0x36d8a566u, 0x4f10e410u};

// cos of an fp32 argument with |x| >= kCosFastLimit, or not finite (NaN),
// inline and in integer arithmetic (the reduction of Payne and Hanek,
// 1983): x = m 2^e with a 24-bit integer m and e >= 10, so x / (2 pi) mod 1
// = m * 0.c_{e+1} c_{e+2} ... mod 1 for the bits c_i of 1 / (2 pi); the 64
// bits c_{e+1} .. c_{e+64} times m, modulo 2^64, give that fraction within
// m 2^-64 < 2^-40 of a revolution.  Its top 32 bits, read as a signed
// fraction in [-1/2, 1/2), go to the hardware cosine (as in the fast path).
__device__ __forceinline__ float cos_fp32_exact_wide(float x) {
    const uint32_t u = __float_as_uint(x), ex = (u >> 23) & 0xFFu;
    if (ex == 0xFFu) return __uint_as_float(0x7FC00000u);
    if (ex < 160u) return cos_fp32_small(x);   // |x| < 2^33: not a wide argument
    const uint64_t m = (u & 0x7FFFFFu) | 0x800000u;
    const uint32_t e = ex - 150u, w0 = e >> 5, sh = e & 31u;
    const uint64_t top = ((uint64_t)kInv2PiBits[w0] << 32) | kInv2PiBits[w0 + 1];
    const uint64_t w = (top << sh) | ((uint64_t)kInv2PiBits[w0 + 2] >> (32u - sh));
    const uint64_t q = m * w;
    return __builtin_amdgcn_cosf((float)(int32_t)(uint32_t)(q >> 32) * 0x1p-32f);
}

__device__ __forceinline__ float cos_fp32(float x) {
    if (fabsf(x) < kCosFastLimit) return cos_fp32_small(x);
    return cos_fp32_wide(x);
}

// One staged slot: x (-1 when the slot is not valid for its query), arrival
// index, timestamp and the fp32 gap tq - t'.
struct SlotLds {
    int32_t x;
    uint32_t e;
    uint32_t t;
    float dt;
};

// A slot as a query at time tq sees it, from its two stored words (the
// class-encoded key and x): eq. (1) keeps only entries stored strictly
// before tq.
__device__ __forceinline__ SlotLds decode_slot(uint64_t key, int32_t xv, uint32_t tq) {
    SlotLds sl = {-1, 0xFFFFFFFFu, 0xFFFFFFFFu, 0.0f};
    const uint32_t t = (uint32_t)key & kTimeMask;
    if (key != 0 && t < tq) {
        const uint32_t ef = (uint32_t)(key >> kTimeBits);
        sl.x = xv;
        sl.e = ((key >> 62) == 3u) ? ef : ~ef;
        sl.t = t;
        sl.dt = (float)(tq - t);
    }
    return sl;
}

// Slot a of node `node`'s block, seen by a query at time tq.
__device__ __forceinline__ SlotLds read_slot(const uint8_t *blocks, uint32_t block_bytes, uint32_t s,
                                             int32_t node, uint32_t a, uint32_t tq) {
    const uint8_t *blk = blocks + (size_t)node * block_bytes;
    return decode_slot(((const uint64_t *)blk)[a], ((const int32_t *)(blk + 8u * s))[a], tq);
}

// ---------------------------------------------------------------- LDS max-merge
// Open-addressing LDS table that merges 64-bit maxima per global address
// (byte offset `off`): merge_max records max(word) for off, so one global
// atomicMax per distinct address can replace many.  kMergeEntries entries
// hold up to half as many distinct addresses.
constexpr int kResolveLinks = 1024;               // links merged per workgroup (two addresses each)
constexpr int kMergeThreads = 1024;               // threads of a merging workgroup (one link each)
constexpr int kMergeBits = 12;                    // 2 * kResolveLinks addresses: load <= 1/2
constexpr int kMergeEntries = 1 << kMergeBits;
constexpr uint32_t kMergeMinBatch = 65536;        // batches from this size merge in LDS
static_assert(kMergeEntries >= 4 * kResolveLinks, "merge table size");

__device__ __forceinline__ void merge_max(unsigned long long *merge_off, unsigned long long *merge_word,
                                          uint64_t off, uint64_t word) {
    const unsigned long long tag = off + 1;  // 0 marks a free entry
    uint32_t h = (uint32_t)(((off >> 3) * kGolden) >> (64 - kMergeBits));
    for (;;) {
        const unsigned long long prev = atomicCAS(&merge_off[h], 0ull, tag);
        if (prev == 0ull || prev == tag) {
            atomicMax(&merge_word[h], (unsigned long long)word);
            return;
        }
        h = (h + 1) & (kMergeEntries - 1);
    }
}

// ---------------------------------------------------------------- feature rows, bf16 pairs
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits) {
    return __uint_as_float(bits << 16);
}

// Eight consecutive elements c0..c0+7 of a feature row (fp32 or bf16);
// elements at or beyond `dim` read as zero.
__device__ __forceinline__ void load8(const uint8_t *row, uint32_t dim, uint32_t is_bf16,
                                      uint32_t vec_ok, uint32_t c0, float v[8]) {
    if (vec_ok && c0 + 8 <= dim) {
        if (is_bf16) {
            const u32x4 q = *(const u32x4 *)(row + 2 * c0);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                v[2 * i] = bf16_bits_to_float(q[i] & 0xFFFFu);
                v[2 * i + 1] = bf16_bits_to_float(q[i] >> 16);
            }
        } else {
            const f32x4 a = *(const f32x4 *)(row + 4 * c0);
            const f32x4 b = *(const f32x4 *)(row + 4 * c0 + 16);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                v[i] = a[i];
                v[4 + i] = b[i];
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const uint32_t c = c0 + i;
        v[i] = 0.0f;
        if (c < dim)
            v[i] = is_bf16 ? bf16_bits_to_float(((const uint16_t *)row)[c]) : ((const float *)row)[c];
    }
}

// Store v as its bf16 pair (hi + lo) at hi[0..7] and lo[0..7] (16 bytes each).
__device__ __forceinline__ void store_split8(const float v[8], __bf16 *hi, __bf16 *lo) {
    bf16x8 h, l;
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const __bf16 t = (__bf16)v[i];
        h[i] = t;
        l[i] = (__bf16)(v[i] - (float)t);
    }
    *(bf16x8 *)hi = h;
    *(bf16x8 *)lo = l;
}

__device__ __forceinline__ void store_split1(float v, __bf16 *hi, __bf16 *lo) {
    const __bf16 t = (__bf16)v;
    *hi = t;
    *lo = (__bf16)(v - (float)t);
}

inline uint32_t pad16(uint32_t x) { return (x + 15u) & ~15u; }
inline uint32_t pad32(uint32_t x) { return (x + 31u) & ~31u; }
inline uint32_t align16(uint32_t x) { return (x + 15u) & ~15u; }

class DeviceGuard {
  public:
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev_) != hipSuccess) prev_ = -1;
        ok_ = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (prev_ >= 0) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }

  private:
    int prev_ = -1;
    bool ok_ = false;
};

// Widest copy unit (16, 8 or 4 bytes) that divides the row and keeps every
// source and destination address aligned.
inline uint32_t copy_width(uint32_t row_bytes, const void *src, const void *dst_or_null) {
    const uintptr_t a = (uintptr_t)src | (uintptr_t)dst_or_null;
    for (uint32_t w = 16; w >= 8; w /= 2)
        if (row_bytes % w == 0 && a % w == 0) return w;
    return 4;
}

}  // namespace

struct nlb_table {
    int device;
    int64_t num_nodes;
    uint32_t s;
    int32_t key_mode;
    double alpha;
    uint64_t thr;
    uint64_t seed;
    uint64_t q1, q2;
    uint32_t d_time;
    const float *w;
    const float *b;
    const uint8_t *efeat;
    int64_t edge_rows;
    uint32_t erb;
    const uint8_t *nfeat;
    uint32_t nrb;
    uint8_t *blocks;
    size_t table_bytes;
    uint32_t block_bytes;
    uint32_t *status;
    uint64_t interactions;            // links enqueued by eager calls (refreshed by nlb_status)
    // Node-status update (rnn.hip), allocated on first use.
    unsigned long long *rnn_winner;   // [N] latest pair-row code per node, zero between calls
    int32_t rnn_form;                 // GRU pass of the last update (NLB_RNN_FORM_*)
    uint8_t *rnn_cand;                // candidate status rows by pair row
    size_t rnn_cand_bytes;
    uint32_t *rnn_list;               // winner count, then the winners' pair rows
    uint64_t rnn_cand_rows;
};

