// aggregate.hip -- the attention aggregation of eq. (4) (Luo & Li, arXiv
// 2402.01964, Sec. 4.4) fused with retrieval:
//   Z_u = MLP_out(r_u, sum_i alpha_i MLP_in(r_v, e, t')),
//   {alpha_i} = softmax({w^T MLP_in(r_v, e, t')}) over the valid slots of S_u^t,
// MLP(x) = W_b ReLU(W_a x + b_a) + b_b.  The retrieved rows and the time
// encoding never leave the chip.  Two kernels: aggregate_rows (below), one
// wavefront per query at a time with every intermediate in registers, for
// the input shapes it is instantiated for; and aggregate_fused, a tiled
// kernel for any other shape, whose workgroup reads its tile's table slots,
// builds the inputs in LDS and runs the four layers on bf16 matrix cores.
//
// Numerics.  Every activation is fp32 and enters a matrix product as a pair
// of bf16 terms, hi = bf16(v) and lo = bf16(v - hi), which represent v to
// 2^-18 relative; both terms multiply the same bf16 weights and accumulate
// in fp32 (v_mfma_f32_16x16x32_bf16).  Inputs that are bf16 already (bf16
// feature rows) have lo = 0, and their lo products are skipped.
//
// MFMA operand layout (v_mfma_f32_16x16x32_bf16, checked on gfx950): lane l
// holds A[l % 16][8 (l / 16) + i], B[8 (l / 16) + i][l % 16] for i < 8, and
// D[4 (l / 16) + i][l % 16] for i < 4.  A is a 16-row block of activations
// in LDS (rows padded so 16-byte lane reads fall on distinct banks); B is a
// 32 x 16 block of a weight matrix read straight from global memory, whose
// rows (one per output column) are K-contiguous, so each lane reads 16
// consecutive bytes.  Each of the four wavefronts owns 16 of the 64 output
// columns and all row blocks of the tile.
#include <cstring>

#include "nlb_internal.h"
#include "nlb_pieces.h"

namespace {

constexpr int kAggThreads = 256;
constexpr int kH = NLB_AGG_HIDDEN;      // hidden and output width
constexpr int kHs = kH + 8;             // bf16 row stride of 64-wide activations in LDS
constexpr int kHf = kH + 4;             // fp32 row stride of the messages in LDS
constexpr int kMaxBlocks = 4;           // row blocks of 16: at most 64 slot rows per tile
constexpr uint32_t kAggLdsBudget = 40 * 1024;    // four workgroups per CU
constexpr uint32_t kAggLdsMax = 160 * 1024;      // gfx950: LDS of one workgroup at most
constexpr int kFillUnroll = 4;                   // input units whose loads are in flight together
constexpr uint32_t kAggTargetTiles = 2048;
static_assert(kH == 64, "the kernel maps four wavefronts onto 64 output columns");

struct AggParams {
    const uint8_t *blocks;
    uint32_t block_bytes;
    uint32_t s;
    int64_t num_nodes;
    const int32_t *node;
    const uint32_t *tq;
    uint32_t nq;
    uint32_t tile_q;      // queries per tile
    uint32_t rows;        // slot rows per tile, padded to 16
    uint32_t qrows;       // query rows per tile, padded to 16
    uint64_t s_m;         // nlb_div_magic(s)
    uint32_t d_time;
    const float *w;
    const float *b;
    const uint8_t *efeat;
    int64_t edge_rows;
    uint32_t e_dim, e_bf16, erb, e_vec;
    const uint8_t *nfeat;
    uint32_t n_dim, n_bf16, nrb, n_vec;
    uint32_t k1, off_e, off_t, k3;   // padded widths of w1 / w3 and segment offsets in w1
    uint32_t xs, ys;                 // LDS row strides (bf16 elements) of X and Y
    uint64_t g1_m, gq_m;             // nlb_div_magic(k1 / 8), nlb_div_magic(pad32(n_dim) / 8)
    uint32_t region_off, off_h, off_y, off_a3;
    const __bf16 *w1, *w2, *w3, *w4;
    const float *b1, *b2, *b3, *b4, *att;
    float *z;
    uint32_t *status;
    uint32_t heads;                  // attention heads, each over H / heads of the messages
};

// acc[rb] += A_rb (16 x K, from the LDS pair Ah/Al with row stride `as`)
//          * W^T (K x 16 columns col0.., W row-major [64][ld]) for rb < nrb.
// lo products are skipped on K ranges whose lo terms are all zero.
template <typename NeedLo>
__device__ __forceinline__ void mfma_rows(f32x4 (&acc)[kMaxBlocks], uint32_t nrb, const __bf16 *Ah,
                                          const __bf16 *Al, uint32_t as, const __bf16 *W,
                                          uint32_t ld, uint32_t K, uint32_t col0, uint32_t lane,
                                          NeedLo need_lo) {
    const uint32_t lr = lane & 15, lk = (lane >> 4) * 8;
    const __bf16 *wrow = W + (size_t)(col0 + lr) * ld + lk;
    for (uint32_t k0 = 0; k0 < K; k0 += 32) {
        const bf16x8 bv = *(const bf16x8 *)(wrow + k0);
        const bool lo = need_lo(k0);
#pragma unroll
        for (int rb = 0; rb < kMaxBlocks; rb++) {
            if ((uint32_t)rb < nrb) {
                const uint32_t off = (16u * rb + lr) * as + k0 + lk;
                acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8 *)(Ah + off), bv,
                                                                  acc[rb], 0, 0, 0);
                if (lo)
                    acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8 *)(Al + off),
                                                                      bv, acc[rb], 0, 0, 0);
            }
        }
    }
}

__device__ __forceinline__ void zero_acc(f32x4 (&acc)[kMaxBlocks]) {
#pragma unroll
    for (int rb = 0; rb < kMaxBlocks; rb++) acc[rb] = f32x4(0.0f);
}

__global__ __launch_bounds__(kAggThreads) void aggregate_fused(AggParams p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    SlotLds *slots = (SlotLds *)smem;
    int32_t *tnodes = (int32_t *)(smem + 16u * p.rows);
    uint8_t *region = smem + p.region_off;
    __bf16 *Xh = (__bf16 *)region;
    __bf16 *Xl = Xh + (size_t)p.rows * p.xs;
    __bf16 *A1h = (__bf16 *)region;                 // after layer 1 (X consumed)
    __bf16 *A1l = A1h + (size_t)p.rows * kHs;
    float *Hf = (float *)(region + p.off_h);
    float *logit = Hf + (size_t)p.rows * kHf;
    __bf16 *Yh = (__bf16 *)(region + p.off_y);
    __bf16 *Yl = Yh + (size_t)p.qrows * p.ys;
    __bf16 *A3h = (__bf16 *)(region + p.off_a3);
    __bf16 *A3l = A3h + (size_t)p.qrows * kHs;

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63, wave = tid >> 6;
    const uint64_t q0 = (uint64_t)blockIdx.x * p.tile_q;
    const uint32_t nqt = (uint32_t)min((uint64_t)p.tile_q, (uint64_t)p.nq - q0);
    const uint32_t s = p.s;
    const uint32_t ns = nqt * s;
    const uint32_t col = 16u * wave + (lane & 15);   // output column of this lane

    // Phase 1: table slots of the tile (eq. (1) strict mask).
    for (uint32_t j = tid; j < p.rows; j += kAggThreads) {
        SlotLds sl = {-1, 0xFFFFFFFFu, 0xFFFFFFFFu, 0.0f};
        if (j < ns) {
            const uint32_t ql = nlb_div(j, p.s_m);
            const uint32_t a = j - ql * s;
            const int32_t node = p.node[q0 + ql];
            const bool in_range = node >= 0 && (int64_t)node < p.num_nodes;
            if (in_range)
                sl = read_slot(p.blocks, p.block_bytes, s, node, a, p.tq[q0 + ql]);
            else if (a == 0)
                atomicOr(p.status, kStatusRange);
            if (a == 0) tnodes[ql] = in_range ? node : -1;
        }
        slots[j] = sl;
    }
    __syncthreads();

    // Phase 2: MLP_in inputs x = [r_v | e | T-enc(tq - t')], hi/lo pairs;
    // the row loads of kFillUnroll units are issued before their stores.
    const uint32_t g1 = p.k1 / 8;
    const uint32_t units = p.rows * g1;
    for (uint32_t base = tid; base < units; base += kAggThreads * kFillUnroll) {
        float v[kFillUnroll][8];
#pragma unroll
        for (int r = 0; r < kFillUnroll; r++) {
            const uint32_t u = base + r * kAggThreads;
#pragma unroll
            for (int i = 0; i < 8; i++) v[r][i] = 0.0f;
            if (u >= units) continue;
            const uint32_t j = nlb_div(u, p.g1_m);
            const uint32_t c0 = (u - j * g1) * 8;
            const SlotLds sl = slots[j];
            if (sl.x < 0) continue;
            if (c0 < p.off_e) {
                load8(p.nfeat + (size_t)sl.x * p.nrb, p.n_dim, p.n_bf16, p.n_vec, c0, v[r]);
            } else if (c0 < p.off_t) {
                if ((int64_t)sl.e < p.edge_rows)
                    load8(p.efeat + (size_t)sl.e * p.erb, p.e_dim, p.e_bf16, p.e_vec, c0 - p.off_e,
                          v[r]);
            } else {
                const uint32_t k = c0 - p.off_t;
#pragma unroll
                for (int i = 0; i < 8; i++)
                    if (k + i < p.d_time)
                        v[r][i] = cos_fp32(__builtin_fmaf(p.w[k + i], sl.dt, p.b[k + i]));
            }
        }
#pragma unroll
        for (int r = 0; r < kFillUnroll; r++) {
            const uint32_t u = base + r * kAggThreads;
            if (u >= units) continue;
            const uint32_t j = nlb_div(u, p.g1_m);
            const uint32_t c0 = (u - j * g1) * 8;
            store_split8(v[r], Xh + (size_t)j * p.xs + c0, Xl + (size_t)j * p.xs + c0);
        }
    }
    __syncthreads();

    const uint32_t nrb = p.rows / 16;
    const uint32_t nqb = p.qrows / 16;
    f32x4 acc[kMaxBlocks];

    // Layer 1: a1 = ReLU(W1 x + b1).
    zero_acc(acc);
    {
        const uint32_t off_e = p.off_e, off_t = p.off_t, nb = p.n_bf16, eb = p.e_bf16;
        mfma_rows(acc, nrb, Xh, Xl, p.xs, p.w1, p.k1, p.k1, 16u * wave, lane,
                  [=](uint32_t k0) { return k0 < off_e ? !nb : (k0 < off_t ? !eb : true); });
    }
    __syncthreads();   // X is consumed; A1 reuses its space
    {
        const float bias = p.b1[col];
#pragma unroll
        for (int rb = 0; rb < kMaxBlocks; rb++)
            if ((uint32_t)rb < nrb)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                    store_split1(fmaxf(acc[rb][i] + bias, 0.0f), A1h + row * kHs + col,
                                 A1l + row * kHs + col);
                }
    }
    __syncthreads();

    // Layer 2: messages h = W2 a1 + b2 (fp32 in LDS).
    zero_acc(acc);
    mfma_rows(acc, nrb, A1h, A1l, kHs, p.w2, kH, kH, 16u * wave, lane,
              [](uint32_t) { return true; });
    {
        const float bias = p.b2[col];
#pragma unroll
        for (int rb = 0; rb < kMaxBlocks; rb++)
            if ((uint32_t)rb < nrb)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                    Hf[row * kHf + col] = acc[rb][i] + bias;
                }
    }
    __syncthreads();

    // Attention logits of the valid slots, one per head over its slice of
    // the messages: logit[j * heads + a] = w[slice a] . h_j[slice a].
    const uint32_t heads = p.heads, hw = kH / heads;
    for (uint32_t u = tid; u < p.rows * heads; u += kAggThreads) {
        const uint32_t j = u / heads, a = u - j * heads;
        float l = 0.0f;
        if (slots[j].x >= 0) {
            const float *h = Hf + j * kHf;
            for (uint32_t n = a * hw; n < (a + 1) * hw; n++) l = __builtin_fmaf(p.att[n], h[n], l);
        }
        logit[u] = l;
    }
    __syncthreads();

    // MLP_out inputs y = [r_u | softmax-weighted sum of the messages].
    const uint32_t kn = p.k3 - kH;   // pad32(node_dim)
    for (uint32_t t = tid; t < p.qrows * kH; t += kAggThreads) {
        const uint32_t q = t / kH, n = t % kH, hd = n / hw;   // unit n belongs to head hd
        float value = 0.0f;
        if (q < nqt) {
            const uint32_t base = q * s;
            float m = -INFINITY;
            for (uint32_t a = 0; a < s; a++)
                if (slots[base + a].x >= 0) m = fmaxf(m, logit[(base + a) * heads + hd]);
            if (m > -INFINITY) {
                float den = 0.0f, num = 0.0f;
                for (uint32_t a = 0; a < s; a++) {
                    if (slots[base + a].x < 0) continue;
                    const float ex = expf(logit[(base + a) * heads + hd] - m);
                    den += ex;
                    num = __builtin_fmaf(ex, Hf[(base + a) * kHf + n], num);
                }
                value = num / den;
            }
        }
        store_split1(value, Yh + q * p.ys + kn + n, Yl + q * p.ys + kn + n);
    }
    if (kn) {
        const uint32_t gq = kn / 8;
        for (uint32_t u = tid; u < p.qrows * gq; u += kAggThreads) {
            const uint32_t q = nlb_div(u, p.gq_m);
            const uint32_t c0 = (u - q * gq) * 8;
            float v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if (q < nqt && tnodes[q] >= 0)
                load8(p.nfeat + (size_t)tnodes[q] * p.nrb, p.n_dim, p.n_bf16, p.n_vec, c0, v);
            store_split8(v, Yh + q * p.ys + c0, Yl + q * p.ys + c0);
        }
    }
    __syncthreads();

    // Layer 3: a3 = ReLU(W3 y + b3).
    zero_acc(acc);
    {
        const uint32_t nb = p.n_bf16;
        mfma_rows(acc, nqb, Yh, Yl, p.ys, p.w3, p.k3, p.k3, 16u * wave, lane,
                  [=](uint32_t k0) { return k0 < kn ? !nb : true; });
        const float bias = p.b3[col];
#pragma unroll
        for (int rb = 0; rb < kMaxBlocks; rb++)
            if ((uint32_t)rb < nqb)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                    store_split1(fmaxf(acc[rb][i] + bias, 0.0f), A3h + row * kHs + col,
                                 A3l + row * kHs + col);
                }
    }
    __syncthreads();

    // Layer 4: Z = W4 a3 + b4.
    zero_acc(acc);
    mfma_rows(acc, nqb, A3h, A3l, kHs, p.w4, kH, kH, 16u * wave, lane,
              [](uint32_t) { return true; });
    {
        const float bias = p.b4[col];
#pragma unroll
        for (int rb = 0; rb < kMaxBlocks; rb++)
            if ((uint32_t)rb < nqb)
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                    if (row < nqt) p.z[(q0 + row) * kH + col] = acc[rb][i] + bias;
                }
    }
}

// ---------------------------------------------------------------- wavefront-per-query kernel
// A second formulation of the same computation that keeps every
// intermediate in registers.  The matrix cores take the weights as the A
// operand (16 output units x 32 inputs) and the activations as the B operand
// (32 inputs x 16 rows): then lane l holds output units 4 (l / 16) + i of
// row l % 16 (i < 4), and two such blocks (units 32 ks + 4 (l / 16) + i and
// 32 ks + 16 + 4 (l / 16) + i) are exactly the eight inputs lane l supplies
// for k-step ks of the next layer -- with the next layer's weight columns
// permuted to that order when they are staged.  So ReLU, the bf16 split and
// the next product follow without an LDS round trip.
//
// Each wavefront takes one query at a time, one 16-row block of its slots
// at a time (s <= 16: one block), as a software pipeline: a block's slot
// words are read two blocks ahead of its computation and its row gathers
// one block ahead.  Per block: layer 1, the attention logits and an online
// softmax that sums the softmax-weighted layer-1 outputs (reductions over
// the 16 rows of a block, combined across blocks with a running maximum).
// MLP_in's second layer is affine, so it is applied once per query to that
// sum (the logits use v = W2^T att, the common shift att . b2 cancelling in
// the softmax).  A group of up to 16 queries then runs MLP_out as one
// 16-row block.  The weights of all four layers are staged in LDS once per
// persistent workgroup; the other LDS is each wavefront's time-encoding tile
// for blocks with few valid rows.  Wavefronts never wait for each other
// after the staging.
constexpr int kRowThreads = 512;    // 8 wavefronts per workgroup
constexpr uint32_t kMaxGroupQ = 16;  // queries per MLP_out block at most
constexpr int kRuSteps = 4;         // k-steps of r_u held in registers: node rows up to 128 wide
constexpr uint32_t kRowsMinQueries = 1;
constexpr float kLog2eAgg = 1.44269504088896340736f;
// Blocks with at least this many valid rows compute the time encoding of
// every row in registers; sparser blocks compute their valid rows only.
constexpr uint32_t kDenseRows = 12;

struct RowParams {
    const uint8_t *blocks;
    uint32_t block_bytes;
    uint32_t s;
    int64_t num_nodes;
    const int32_t *node;
    const uint32_t *tq;
    uint32_t nq;
    uint32_t gq;                     // queries per group (1..16)
    uint32_t nbq;                    // 16-row blocks per query
    uint32_t d_time;
    uint32_t nch;                    // 4-column chunks of the time encoding
    uint64_t nch_m;                  // ceil(2^32 / nch): i / nch = (i nch_m) >> 32 for i < 2^16
    const float *w;
    const float *b;
    const uint8_t *efeat;
    int64_t edge_rows;
    uint32_t e_dim, erb;
    const uint8_t *nfeat;
    uint32_t n_dim, nrb;
    const __bf16 *w1, *w2, *w3, *w4;
    const float *b1, *b2, *b3, *b4, *att;
    float *z;
    uint32_t *status;
};

// LDS row stride of the permuted w2 / w4: unpadded, as they are read once
// per query group only.
constexpr uint32_t kPs = kH;

// Chained layers take their weights' columns permuted: slot (ks, g, i) of a
// k-step's B operand (LDS column c = 32 ks + 8 g + i) holds input unit
// 32 ks + 4 g + i for i < 4 and 32 ks + 16 + 4 g + (i - 4) otherwise.
// chain_pos is the inverse, the LDS column of input unit gc; units gc0 ..
// gc0 + 3 (gc0 % 4 == 0) land on four consecutive LDS columns.
__device__ __forceinline__ uint32_t chain_pos(uint32_t gc) {
    const uint32_t b = gc & 31u;
    return (gc & ~31u) + 8u * ((b & 15u) >> 2) + (b & 3u) + (b >= 16u ? 4u : 0u);
}

// v = hi + lo (bf16 each, hi rounded to nearest).  Pairs are converted
// together and the fp32 value of each hi is taken from the packed bits.
__device__ __forceinline__ void split8(const float v[8], bf16x8 &hi, bf16x8 &lo) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    u32x4 hw, lw;
#pragma unroll
    for (int j = 0; j < 4; j++) {
        const uint32_t hb =
            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v[2 * j], v[2 * j + 1]}, bf16x2));
        const float h0 = __uint_as_float(hb << 16), h1 = __uint_as_float(hb & 0xFFFF0000u);
        hw[j] = hb;
        lw[j] = __builtin_bit_cast(uint32_t,
                                   __builtin_convertvector((f32x2){v[2 * j] - h0, v[2 * j + 1] - h1}, bf16x2));
    }
    hi = __builtin_bit_cast(bf16x8, hw);
    lo = __builtin_bit_cast(bf16x8, lw);
}

// The same split for four values, as packed bf16 pairs.
__device__ __forceinline__ void split4(const float v[4], u32x2 &hw, u32x2 &lw) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
#pragma unroll
    for (int j = 0; j < 2; j++) {
        const uint32_t hb =
            __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){v[2 * j], v[2 * j + 1]}, bf16x2));
        const float h0 = __uint_as_float(hb << 16), h1 = __uint_as_float(hb & 0xFFFF0000u);
        hw[j] = hb;
        lw[j] = __builtin_bit_cast(uint32_t,
                                   __builtin_convertvector((f32x2){v[2 * j] - h0, v[2 * j + 1] - h1}, bf16x2));
    }
}

// acc[ub] += W[16 ub .. 16 ub + 15][k-step] x (hi + lo) for the four unit blocks.
// The four hi products are issued before the four lo products, so that no
// product waits for the one just before it (the lo product of a unit block
// accumulates onto its hi product's result).
// Only the unit blocks UB0 <= ub < UB1 are computed.
template <int UB0 = 0, int UB1 = 4>
__device__ __forceinline__ void mfma4(f32x4 (&acc)[4], const __bf16 *W, uint32_t ls, uint32_t k0,
                                      uint32_t r16, uint32_t g, const bf16x8 &hi, const bf16x8 &lo,
                                      bool use_lo) {
    bf16x8 a[4];
#pragma unroll
    for (int ub = UB0; ub < UB1; ub++) a[ub] = *(const bf16x8 *)(W + (16u * ub + r16) * ls + k0 + 8u * g);
#pragma unroll
    for (int ub = UB0; ub < UB1; ub++)
        acc[ub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ub], hi, acc[ub], 0, 0, 0);
    if (use_lo) {
#pragma unroll
        for (int ub = UB0; ub < UB1; ub++)
            acc[ub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[ub], lo, acc[ub], 0, 0, 0);
    }
}

// The same product with the activations as the A operand and the weights as
// B (both operands hold the same registers as in mfma4): D = X W^T, the
// layer's output transposed -- lane l holds rows 4 (l / 16) + i of unit
// 16 ub + l % 16.
__device__ __forceinline__ void mfma4t(f32x4 (&acc)[4], const __bf16 *W, uint32_t ls, uint32_t k0,
                                       uint32_t r16, uint32_t g, const bf16x8 &hi, const bf16x8 &lo,
                                       bool use_lo) {
    bf16x8 a[4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) a[ub] = *(const bf16x8 *)(W + (16u * ub + r16) * ls + k0 + 8u * g);
#pragma unroll
    for (int ub = 0; ub < 4; ub++) acc[ub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, a[ub], acc[ub], 0, 0, 0);
    if (use_lo) {
#pragma unroll
        for (int ub = 0; ub < 4; ub++) acc[ub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, a[ub], acc[ub], 0, 0, 0);
    }
}

// act (a layer's output in the D layout, 64 units) -> next layer through
// weights whose 64 columns from k0 on are in chained order (row stride ls):
// out[ub] += Wp x act, for the output unit blocks UB0 <= ub < UB1.
template <int UB0 = 0, int UB1 = 4>
__device__ __forceinline__ void chain64(f32x4 (&out)[4], const f32x4 (&act)[4], const __bf16 *Wp,
                                        uint32_t ls, uint32_t k0, uint32_t r16, uint32_t g) {
#pragma unroll
    for (int ks = 0; ks < 2; ks++) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            v[i] = act[2 * ks][i];
            v[4 + i] = act[2 * ks + 1][i];
        }
        bf16x8 hi, lo;
        split8(v, hi, lo);
        mfma4<UB0, UB1>(out, Wp, ls, k0 + 32u * ks, r16, g, hi, lo, true);
    }
}

// cos of an fp32 argument with |x| < kCosFastLimit, as cos_fp32_small but
// with the revolutions reduced by v_fract_f64 (y - floor(y), exact in
// double) instead of a rounding and a subtraction: one instruction fewer.
// The fraction lies in [0, 1); its rounding to fp32 adds at most 2^-25 of a
// revolution.
__device__ __forceinline__ float cos_fast(float x) {
    const double y = (double)x * 0.15915494309189533577;
    return __builtin_amdgcn_cosf((float)__builtin_amdgcn_fract(y));
}

// Reductions over the 16 lanes of a DPP row (the 16 rows of a block), with
// the result in every lane: pair lanes by quad permutations (swap
// neighbours, then pairs), then mirror within each half-row and the row.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppSwap1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppSwap2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror
constexpr int kDppMirror = 0x140;      // row_mirror

__device__ __forceinline__ float xor16_sum(float v) {
    v += dpp<kDppSwap1>(v);
    v += dpp<kDppSwap2>(v);
    v += dpp<kDppHalfMirror>(v);
    v += dpp<kDppMirror>(v);
    return v;
}

// max(a, b) and max(x, 0) as medians with +inf: one instruction each for
// non-NaN operands.  fmaxf on a value the compiler cannot prove canonical (a
// lane permutation, a matrix-core result) first quiets a possible signalling
// NaN, which costs a second instruction per value.  The +inf bound passes
// through an empty asm statement: with a literal bound the compiler folds the
// median back into fmaxf.
__device__ __forceinline__ float opaque_inf() {
    uint32_t u = 0x7F800000u;
    asm("" : "+s"(u));
    return __uint_as_float(u);
}
__device__ __forceinline__ float max2(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, opaque_inf()); }
__device__ __forceinline__ float relu(float x) { return __builtin_amdgcn_fmed3f(x, 0.0f, opaque_inf()); }

// A lane permutation with no prior value: every lane of these four patterns
// has a source lane, so none keeps its old contents.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float xor16_max(float v) {
    v = max2(v, dpp_mov<kDppSwap1>(v));
    v = max2(v, dpp_mov<kDppSwap2>(v));
    v = max2(v, dpp_mov<kDppHalfMirror>(v));
    v = max2(v, dpp_mov<kDppMirror>(v));
    return v;
}

// Sum and maximum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (one lane of
// each lane group), in every lane, with gfx950's row-swap instructions:
// v_permlane16_swap on two copies of v leaves rows (0, 0, 2, 2) in one and
// (1, 1, 3, 3) in the other, v_permlane32_swap halves (lo, lo) and (hi, hi);
// combining each pair pairs lane l with l ^ 16, then with l ^ 32.
__device__ __forceinline__ float groups_sum(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float groups_max(float v) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = max2(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return max2(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// LDS layout of aggregate_rows for K1S / K3S k-steps of layers 1 and 3 and
// TKS k-steps of time encoding.
template <int K1S, int K3S, int TKS>
struct RowsLayout {
    static constexpr uint32_t ls1 = 32u * K1S + 8u, ls3 = 32u * K3S + 8u;
    static constexpr uint32_t o_w1 = 0;
    static constexpr uint32_t o_w2 = o_w1 + kH * ls1 * 2u;
    static constexpr uint32_t o_w3 = o_w2 + kH * kPs * 2u;
    static constexpr uint32_t o_w4 = o_w3 + kH * ls3 * 2u;
    static constexpr uint32_t o_vec = o_w4 + kH * kPs * 2u;
    static constexpr uint32_t o_tenc = o_vec + 6u * kH * 4u;   // w | b, 32 TKS each, zero-padded
    // Per wavefront: the time encodings of a block's 16 rows, bf16 hi | lo
    // (32 TKS each) plus 8 elements of padding per row, and the list of the
    // block's valid rows (row, dt).
    static constexpr uint32_t ts = 64u * TKS + 8u;
    static constexpr uint32_t o_t = o_tenc + 2u * 32u * TKS * 4u;
    static constexpr uint32_t o_rl = o_t + (kRowThreads / 64) * 16u * ts * 2u;
    static constexpr uint32_t bytes = o_rl + (kRowThreads / 64) * 16u * 8u;
};

// A piece as a matrix-core B operand, hi + lo (lo is not formed for bf16
// rows, whose values are exact in bf16), zero where `ok` is false or past
// the row.
template <int KIND>
__device__ __forceinline__ void piece_operand(const Piece8<KIND> &r, uint32_t dim, uint32_t c, bool ok,
                                              bf16x8 &hi, bf16x8 &lo) {
    if constexpr (KIND != kF32Vec) {
        hi = __builtin_bit_cast(bf16x8, piece_bf16_bits<KIND>(r, dim, c, ok));
        lo = hi;
    } else {
        float v[8];
        piece_floats<KIND>(r, dim, c, ok, v);
        split8(v, hi, lo);
    }
}

// MLP_out for a group of up to 16 queries: row r16 = query qb + r16, input
// [r_u | aggregate], the aggregate w2 aggd + b2 (zero for a query without
// valid rows, ne = 0); aggd[a] holds head a's finished aggregates
// sum_s alpha_{s,a} a1_s in the D layout (query r16's units 16 ub + 4 g + i
// in the lanes with that r16), of which head a's slice of w2's outputs is
// taken.  Writes z for the lanes with vq.
template <int NKS, int NK, uint32_t LS3, uint32_t PS, int HEADS>
__device__ __forceinline__ void mlp_out_group(const RowParams &p, const Piece8<NK> (&ru)[NKS > 0 ? NKS : 1],
                                              int32_t nr, bool vq, const f32x4 (&aggd)[HEADS][4], float ne,
                                              const __bf16 *W2, const __bf16 *W3, const __bf16 *W4,
                                              const float *b2, const float *b3, const float *b4, uint32_t r16,
                                              uint32_t g, uint64_t qb) {
    if (vq && g == 0 && nr < 0) atomicOr(p.status, kStatusRange);   // an out-of-range query
    f32x4 acc3[4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) acc3[ub] = f32x4(0.0f);
#pragma unroll
    for (int ks = 0; ks < NKS; ks++) {
        bf16x8 hi, lo;
        piece_operand<NK>(ru[ks], p.n_dim, 32u * ks + 8u * g, nr >= 0, hi, lo);
        mfma4(acc3, W3, LS3, 32u * ks, r16, g, hi, lo, NK == kF32Vec);
    }
    static_assert(HEADS == 1 || HEADS == 2, "one or two heads");
    f32x4 hq[4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) hq[ub] = f32x4(0.0f);
    if constexpr (HEADS == 1) {
        chain64(hq, aggd[0], W2, PS, 0, r16, g);
    } else {
        chain64<0, 2>(hq, aggd[0], W2, PS, 0, r16, g);
        chain64<2, 4>(hq, aggd[1], W2, PS, 0, r16, g);
    }
#pragma unroll
    for (int ub = 0; ub < 4; ub++)
#pragma unroll
        for (int i = 0; i < 4; i++) hq[ub][i] = ne * (hq[ub][i] + b2[16 * ub + 4 * g + i]);
    chain64(acc3, hq, W3, LS3, 32u * NKS, r16, g);
#pragma unroll
    for (int ub = 0; ub < 4; ub++)
#pragma unroll
        for (int i = 0; i < 4; i++) acc3[ub][i] = fmaxf(acc3[ub][i] + b3[16 * ub + 4 * g + i], 0.0f);
    f32x4 zo[4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) zo[ub] = f32x4(0.0f);
    chain64(zo, acc3, W4, PS, 0, r16, g);
    if (vq) {
#pragma unroll
        for (int ub = 0; ub < 4; ub++) {
#pragma unroll
            for (int i = 0; i < 4; i++) zo[ub][i] += b4[16 * ub + 4 * g + i];
            *(f32x4 *)(p.z + (qb + r16) * kH + 16 * ub + 4 * g) = zo[ub];
        }
    }
}

// Specialised per input shape: NKS, EKS and TKS k-steps of layer 1 hold r_v,
// e and the time encoding, NK / EK are the piece forms of the node / link
// rows; layer 3 has NKS + 2 k-steps (r_u, then the aggregate).  With the
// shape fixed at compile time every LDS address is a base plus an immediate
// offset, all k-loops unroll and each segment's loads have one fixed form.
// Queries are taken in groups of p.gq <= 16 (one MLP_out block each).
template <int NKS, int EKS, int TKS, int NK, int EK, int HEADS>
__global__ __launch_bounds__(kRowThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void aggregate_rows(RowParams p) {
    constexpr int GS = NKS + EKS, K1S = GS + TKS, K3S = NKS + 2;
    using L = RowsLayout<K1S, K3S, TKS>;
    static_assert(NKS <= kRuSteps, "shape");
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    __bf16 *W1 = (__bf16 *)(smem + L::o_w1);
    __bf16 *W2 = (__bf16 *)(smem + L::o_w2);
    __bf16 *W3 = (__bf16 *)(smem + L::o_w3);
    __bf16 *W4 = (__bf16 *)(smem + L::o_w4);
    float *vec = (float *)(smem + L::o_vec);   // b1 | b2 | b3 | b4 | v per head, 64 each

    // Stage the weights: w2, w4 and the aggregate columns of w3 in chained
    // order.  (Each loop is unrolled so that several iterations' loads are in
    // flight before their LDS stores: the staging is latency-bound otherwise.)
    const uint32_t tid = threadIdx.x;
    // The time-encoding columns past d_time are staged as zeros: the rows'
    // time encodings are then used unmasked (finite values, zero weight).
#pragma unroll 4
    for (uint32_t u = tid; u < kH * (K1S * 4u); u += kRowThreads) {
        const uint32_t r = u / (K1S * 4u), c = (u % (K1S * 4u)) * 8;
        bf16x8 v = *(const bf16x8 *)(p.w1 + (size_t)r * (32u * K1S) + c);
#pragma unroll
        for (int i = 0; i < 8; i++)
            if (c + i >= 32u * GS + p.d_time) v[i] = (__bf16)0.0f;
        *(bf16x8 *)(W1 + r * L::ls1 + c) = v;
    }
    if constexpr (NKS > 0) {
#pragma unroll 4
        for (uint32_t u = tid; u < kH * (NKS * 4u); u += kRowThreads) {
            const uint32_t r = u / (NKS * 4u), c = (u % (NKS * 4u)) * 8;
            *(bf16x8 *)(W3 + r * L::ls3 + c) = *(const bf16x8 *)(p.w3 + (size_t)r * (32u * K3S) + c);
        }
    }
    // A 16-byte piece of 8 columns gc0 + e lands as two 8-byte halves, at the
    // LDS columns of gc0 and gc0 + 4.
#pragma unroll 4
    for (uint32_t u = tid; u < kH * (kH / 8u); u += kRowThreads) {
        const uint32_t r = u / (kH / 8u), gc0 = (u % (kH / 8u)) * 8u;
        const u32x4 v2 = *(const u32x4 *)(p.w2 + r * kH + gc0), v4 = *(const u32x4 *)(p.w4 + r * kH + gc0),
                    v3 = *(const u32x4 *)(p.w3 + (size_t)r * (32u * K3S) + 32u * NKS + gc0);
        const uint32_t c0 = chain_pos(gc0), c1 = chain_pos(gc0 + 4u);
        *(u32x2 *)(W2 + r * kPs + c0) = u32x2{v2[0], v2[1]};
        *(u32x2 *)(W2 + r * kPs + c1) = u32x2{v2[2], v2[3]};
        *(u32x2 *)(W4 + r * kPs + c0) = u32x2{v4[0], v4[1]};
        *(u32x2 *)(W4 + r * kPs + c1) = u32x2{v4[2], v4[3]};
        *(u32x2 *)(W3 + r * L::ls3 + 32u * NKS + c0) = u32x2{v3[0], v3[1]};
        *(u32x2 *)(W3 + r * L::ls3 + 32u * NKS + c1) = u32x2{v3[2], v3[3]};
    }
    // Layer 2 is affine, so the logit att . (w2 a1 + b2) of a row is
    // v . a1 up to a shift common to all rows (which the softmax cancels),
    // with v = w2^T att; and the aggregate sum_s alpha_s (w2 a1_s + b2) is
    // w2 (sum_s alpha_s a1_s) + b2.  So layer 2 runs once per query.  With
    // heads, head a's logit vector is v_a = w2[slice a]^T att[slice a].
    for (uint32_t u = tid; u < (4u + HEADS) * kH; u += kRowThreads) {
        const uint32_t k = u / kH, c = u % kH;
        float val;
        if (k < 4) {
            val = (k == 0 ? p.b1 : k == 1 ? p.b2 : k == 2 ? p.b3 : p.b4)[c];
        } else {
            val = 0.0f;
            const uint32_t r0 = (k - 4u) * (kH / HEADS);
#pragma unroll
            for (uint32_t r = 0; r < kH / HEADS; r++)
                val = __builtin_fmaf(p.att[r0 + r], (float)p.w2[(r0 + r) * kH + c], val);
        }
        vec[u] = val;
    }
    float *tw = (float *)(smem + L::o_tenc), *tb = tw + 32 * TKS;
    for (uint32_t u = tid; u < 32u * TKS; u += kRowThreads) {
        tw[u] = u < p.d_time ? p.w[u] : 0.0f;
        tb[u] = u < p.d_time ? p.b[u] : 0.0f;
    }
    // The time-encoding tiles start as zeros: rows and columns a block does
    // not write keep finite values.
    for (uint32_t u = tid; u < (L::o_rl - L::o_t) / 16u; u += kRowThreads)
        *(u32x4 *)(smem + L::o_t + 16u * u) = u32x4(0u);
    __syncthreads();
    // max |w| and max |b| of the time encoding, for the per-unit test that
    // every argument w dt + b is inside the fast cosine's range.
    float wmax = 0.0f, bmax = 0.0f;
    for (uint32_t u = tid & 63; u < 32u * TKS; u += 64) {
        wmax = fmaxf(wmax, fabsf(tw[u]));
        bmax = fmaxf(bmax, fabsf(tb[u]));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        wmax = fmaxf(wmax, __shfl_xor(wmax, o));
        bmax = fmaxf(bmax, __shfl_xor(bmax, o));
    }
    wmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(wmax)));
    bmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(bmax)));

    // The wavefront index as a uniform value, so that all the cursor state
    // below lives in scalar registers and its branches are scalar.
    const uint32_t lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t r16 = lane & 15, g = lane >> 4;
    __bf16 *Tt = (__bf16 *)(smem + L::o_t) + (size_t)wave * 16u * L::ts;
    u32x2 *rl = (u32x2 *)(smem + L::o_rl) + wave * 16u;
    const float *b1 = vec, *b2 = vec + kH, *b3 = vec + 2 * kH, *b4 = vec + 3 * kH, *va = vec + 4 * kH;
    // This lane's unit column of layer 1 (16 ub + r16): its bias and its
    // weight in each head's logits.
    float b1v[4], vav[HEADS][4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) {
        b1v[ub] = b1[16 * ub + r16];
#pragma unroll
        for (int a = 0; a < HEADS; a++) vav[a][ub] = va[a * kH + 16 * ub + r16];
    }
    const uint32_t gq = p.gq;
    const uint64_t groups = ((uint64_t)p.nq + gq - 1) / gq;
    const uint64_t gstep = (uint64_t)gridDim.x * (kRowThreads / 64);
    // Consecutive groups go to different workgroups first, so a launch with
    // few groups spreads over the CUs.
    const uint64_t g0 = (uint64_t)wave * gridDim.x + blockIdx.x;
    if (g0 >= groups) return;   // no workgroup barrier follows

    auto group_size = [&](uint64_t grp) -> uint32_t {
        return (uint32_t)min((uint64_t)gq, (uint64_t)p.nq - grp * gq);
    };
    // Query ids of a group: query i of it in the lanes with r16 == i.  Lanes
    // past the last query read the last (in bounds; never used), so the loads
    // are unconditional and land in their final registers.
    auto load_ids = [&](uint64_t grp, int32_t &nd, uint32_t &t) {
        const uint64_t q = min(grp * gq + r16, (uint64_t)p.nq - 1);
        nd = p.node[q];
        t = p.tq[q];
    };

    // The wavefront's units, (group, query, 16-row block) in order over its
    // groups, run as a software pipeline: a unit's two slot words are read
    // two units ahead of its computation, its rows are gathered one unit
    // ahead, and the query ids of the group after next are read when a
    // group starts.  Only the computation waits, for loads issued a whole
    // unit earlier.
    struct SlotRaw {
        uint64_t key;
        int32_t x;
        uint32_t tq;
        bool ok;   // node in range and slot inside the table
    };
    uint64_t ig = g0;   // issue cursor (slot words)
    uint32_t iq = 0, ib = 0, inq = group_size(g0);
    int32_t id_nd, pre_nd;
    uint32_t id_t, pre_t;
    load_ids(g0, id_nd, id_t);
    load_ids(g0 + gstep, pre_nd, pre_t);
    // A unit's two slot words, read unconditionally (a unit past the end, an
    // out-of-range node or a slot past s reads slot 0 of node 0 and is
    // marked not ok).
    auto issue_slot = [&]() {
        SlotRaw r;
        const bool live = ig < groups;
        const int32_t nd = __builtin_amdgcn_readlane(id_nd, (int)iq);
        r.tq = (uint32_t)__builtin_amdgcn_readlane((int)id_t, (int)iq);
        const uint32_t a = 16u * ib + r16;
        r.ok = live && nd >= 0 && (int64_t)nd < p.num_nodes && a < p.s;
        const uint8_t *bp = p.blocks + (size_t)(r.ok ? nd : 0) * p.block_bytes;
        const uint32_t aa = r.ok ? a : 0u;
        r.key = ((const uint64_t *)bp)[aa];
        r.x = ((const int32_t *)(bp + 8u * p.s))[aa];
        if (live) {
            if (++ib == p.nbq) {
                ib = 0;
                if (++iq == inq) {
                    iq = 0;
                    ig += gstep;
                    id_nd = pre_nd;
                    id_t = pre_t;
                    if (ig < groups) inq = group_size(ig);
                    load_ids(ig + gstep, pre_nd, pre_t);
                }
            }
        }
        return r;
    };
    // Gathered inputs (r_v and e) of this lane's row of a unit; invalid rows
    // read row 0 and are zeroed when used.
    struct Rows {
        Piece8<NK> n[NKS > 0 ? NKS : 1];
        Piece8<EK> e[EKS > 0 ? EKS : 1];
    };
    auto issue_rows = [&](const SlotLds &sl, Rows &r) {
        const bool valid = sl.x >= 0;
        if constexpr (NKS > 0) {
            const uint8_t *nrow = p.nfeat + (size_t)(valid ? sl.x : 0) * p.nrb;
#pragma unroll
            for (int ks = 0; ks < NKS; ks++) load_piece<NK>(nrow, p.n_dim, 32u * ks + 8u * g, r.n[ks]);
        }
        if constexpr (EKS > 0) {
            const bool ev = valid && (int64_t)sl.e < p.edge_rows;
            const uint8_t *erow = p.efeat + (size_t)(ev ? sl.e : 0u) * p.erb;
#pragma unroll
            for (int ks = 0; ks < EKS; ks++) load_piece<EK>(erow, p.e_dim, 32u * ks + 8u * g, r.e[ks]);
        }
    };

    SlotRaw raw_n = issue_slot();
    SlotLds sl_c = decode_slot(raw_n.ok ? raw_n.key : 0ull, raw_n.x, raw_n.tq);
    Rows rows_c;
    issue_rows(sl_c, rows_c);
    raw_n = issue_slot();
    uint64_t cg = g0;   // compute cursor
    uint32_t cq = 0, cb = 0, cnq = group_size(g0);
    // Query ids of the compute group for MLP_out (lanes r16 >= cnq unused).
    int32_t mo_nd = p.node[min(g0 * gq + r16, (uint64_t)p.nq - 1)];
    // Layer 1 runs transposed (mfma4t): lane l holds rows 4 g + i of unit
    // 16 ub + r16.  The online softmax of the current query is kept per lane
    // group g, over its rows 4 g .. 4 g + 3 of each block: running maximum m,
    // sum of exponentials den, and agg, the exponential-weighted sums of this
    // lane's unit column.  At the query's end the four groups are combined
    // into aggd, the group's finished aggregates sum_s alpha_s a1_s: query
    // q's in the lanes with r16 == q, in the D layout (units 16 ub + 4 g + i),
    // with ne = 1 where the query had a valid row (else its aggregate is zero).
    // Each head keeps its own softmax state and aggregates.
    float m[HEADS], den[HEADS], ne = 0.0f;
    float agg[HEADS][4];
    f32x4 aggd[HEADS][4];
#pragma unroll
    for (int a = 0; a < HEADS; a++) {
        m[a] = -INFINITY;
        den[a] = 0.0f;
#pragma unroll
        for (int ub = 0; ub < 4; ub++) {
            agg[a][ub] = 0.0f;
            aggd[a][ub] = f32x4(0.0f);
        }
    }
    while (cg < groups) {
        // Keeps the LDS-resident biases from being hoisted into long-lived
        // registers.
        asm volatile("" ::: "memory");
        const bool last_blk = cb + 1 == p.nbq;
        const bool group_end = last_blk && cq + 1 == cnq;
        // The next unit's rows, the slot words of the one after, and at a
        // group's last unit its MLP_out rows r_u.
        const SlotLds sl_n = decode_slot(raw_n.ok ? raw_n.key : 0ull, raw_n.x, raw_n.tq);
        Rows rows_n;
        issue_rows(sl_n, rows_n);
        raw_n = issue_slot();
        const bool vq = r16 < cnq;
        const int32_t nr = (vq && mo_nd >= 0 && (int64_t)mo_nd < p.num_nodes) ? mo_nd : -1;
        Piece8<NK> ru[NKS > 0 ? NKS : 1];
        if constexpr (NKS > 0) {
            if (group_end) {
                const uint8_t *urow = p.nfeat + (size_t)(nr >= 0 ? nr : 0) * p.nrb;
#pragma unroll
                for (int ks = 0; ks < NKS; ks++) load_piece<NK>(urow, p.n_dim, 32u * ks + 8u * g, ru[ks]);
            }
        }
        // Keep the scheduler from sinking the loads to their uses.
        __builtin_amdgcn_sched_barrier(0);

        const SlotLds sl = sl_c;
        const bool valid = sl.x >= 0;
        const bool ev = valid && (int64_t)sl.e < p.edge_rows;
        // A block without a valid row changes nothing (wave-uniform test).
        if (__builtin_amdgcn_ballot_w64(valid) != 0) {
        // Layer 1: a1 = ReLU(W1 x + b1).
        f32x4 acc[4];
#pragma unroll
        for (int ub = 0; ub < 4; ub++) acc[ub] = f32x4(b1v[ub]);   // + b1
#pragma unroll
        for (int ks = 0; ks < NKS; ks++) {
            bf16x8 hi, lo;
            piece_operand<NK>(rows_c.n[ks], p.n_dim, 32u * ks + 8u * g, valid, hi, lo);
            mfma4t(acc, W1, L::ls1, 32u * ks, r16, g, hi, lo, NK == kF32Vec);
        }
#pragma unroll
        for (int ks = 0; ks < EKS; ks++) {
            bf16x8 hi, lo;
            piece_operand<EK>(rows_c.e[ks], p.e_dim, 32u * ks + 8u * g, ev, hi, lo);
            mfma4t(acc, W1, L::ls1, 32u * (NKS + ks), r16, g, hi, lo, EK == kF32Vec);
        }
        // Time encodings.  A block with few valid rows computes only those:
        // its (valid row, 4-column chunk) items are spread over the 64 lanes,
        // their bf16 hi / lo pairs go to the wavefront's LDS tile, and the
        // tile's rows are read back as matrix-core operands (rows the block
        // does not write hold earlier finite values and are excluded by the
        // softmax).  A block with many valid rows, or with an argument
        // outside the fast cosine's range, computes every row in registers
        // (an invalid row has dt = 0).  Columns past d_time have zero weight.
        // The fast cosine serves the whole block when max |w| max dt + max |b|
        // (with margin for the rounding of the bound) is inside its range.
        {
            const uint32_t vm = (uint32_t)__builtin_amdgcn_ballot_w64(valid) & 0xFFFFu;
            const uint32_t nv = (uint32_t)__builtin_popcount(vm);
            const float dtmax =
                __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(xor16_max(sl.dt))));
            const bool fast = wmax * dtmax + bmax < 0.5f * kCosFastLimit;
            if (fast && nv < kDenseRows) {
                if (g == 0 && valid) rl[__builtin_popcount(vm & ((1u << r16) - 1u))] = u32x2{r16, __float_as_uint(sl.dt)};
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                const uint32_t items = nv * p.nch;
                for (uint32_t base = 0; base < items; base += 64) {
                    const uint32_t it = base + lane;
                    if (it < items) {
                        const uint32_t j = (uint32_t)(((uint64_t)it * p.nch_m) >> 32), c = it - j * p.nch;
                        const u32x2 e = rl[j];
                        const float dt = __uint_as_float(e[1]);
                        const f32x4 wv = *(const f32x4 *)(tw + 4u * c), bv = *(const f32x4 *)(tb + 4u * c);
                        float t[4];
#pragma unroll
                        for (int i = 0; i < 4; i++) t[i] = cos_fast(__builtin_fmaf(wv[i], dt, bv[i]));
                        u32x2 hw, lw;
                        split4(t, hw, lw);
                        *(u32x2 *)(Tt + e[0] * L::ts + 4u * c) = hw;
                        *(u32x2 *)(Tt + e[0] * L::ts + 32u * TKS + 4u * c) = lw;
                    }
                }
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
                for (int ks = 0; ks < TKS; ks++) {
                    const bf16x8 hi = *(const bf16x8 *)(Tt + r16 * L::ts + 32u * ks + 8u * g);
                    const bf16x8 lo = *(const bf16x8 *)(Tt + r16 * L::ts + 32u * TKS + 32u * ks + 8u * g);
                    mfma4t(acc, W1, L::ls1, 32u * (GS + ks), r16, g, hi, lo, true);
                }
            } else if (fast) {
#pragma unroll 1
                for (int ks = 0; ks < TKS; ks++) {
                    const uint32_t k = 32u * ks + 8u * g;
                    const f32x4 w0 = *(const f32x4 *)(tw + k), w1 = *(const f32x4 *)(tw + k + 4);
                    const f32x4 c0 = *(const f32x4 *)(tb + k), c1 = *(const f32x4 *)(tb + k + 4);
                    float t[8];
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        t[i] = cos_fast(__builtin_fmaf(w0[i], sl.dt, c0[i]));
                        t[4 + i] = cos_fast(__builtin_fmaf(w1[i], sl.dt, c1[i]));
                    }
                    bf16x8 hi, lo;
                    split8(t, hi, lo);
                    mfma4t(acc, W1, L::ls1, 32u * (GS + ks), r16, g, hi, lo, true);
                }
            } else {
#pragma unroll 1
                for (int ks = 0; ks < TKS; ks++) {
                    const uint32_t k = 32u * ks + 8u * g;
                    float t[8];
#pragma unroll
                    for (int i = 0; i < 8; i++) t[i] = cos_fp32(__builtin_fmaf(tw[k + i], sl.dt, tb[k + i]));
                    bf16x8 hi, lo;
                    split8(t, hi, lo);
                    mfma4t(acc, W1, L::ls1, 32u * (GS + ks), r16, g, hi, lo, true);
                }
            }
        }
#pragma unroll
        for (int ub = 0; ub < 4; ub++)
#pragma unroll
            for (int i = 0; i < 4; i++) acc[ub][i] = relu(acc[ub][i]);
        const uint32_t nib = ((uint32_t)__builtin_amdgcn_ballot_w64(valid) >> (4u * g)) & 0xFu;
#pragma unroll
        for (int a = 0; a < HEADS; a++) {
        // Head a's logits v_a . a1 of rows 4 g + i (up to the common shift
        // att . b2): this lane's unit column's share, summed over the 16 lanes
        // of its group.
        float lg[4];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            float t = vav[a][0] * acc[0][i];
#pragma unroll
            for (int ub = 1; ub < 4; ub++) t = __builtin_fmaf(vav[a][ub], acc[ub][i], t);
            lg[i] = xor16_sum(t);
        }
        // Online softmax over the group's valid rows: an invalid row's logit
        // is -inf (weight 0), and a group without a valid row so far keeps
        // m = -inf, den = 0.  exp(x - mn) is the hardware 2^(x log2 e -
        // mn log2 e), one fused multiply-add: its rounding adds a relative
        // error of about |mn| 2^-24.
#pragma unroll
        for (int i = 0; i < 4; i++) lg[i] = ((nib >> i) & 1u) ? lg[i] : -INFINITY;
        const float mn = max2(m[a], max2(max2(lg[0], lg[1]), max2(lg[2], lg[3])));
        const float shift = (mn == -INFINITY) ? 0.0f : mn * kLog2eAgg;
        const float sc = __builtin_amdgcn_exp2f(__builtin_fmaf(m[a], kLog2eAgg, -shift));
        float e[4];
#pragma unroll
        for (int i = 0; i < 4; i++) e[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(lg[i], kLog2eAgg, -shift));
        den[a] = __builtin_fmaf(den[a], sc, (e[0] + e[1]) + (e[2] + e[3]));
#pragma unroll
        for (int ub = 0; ub < 4; ub++) {
            float t = agg[a][ub] * sc;
#pragma unroll
            for (int i = 0; i < 4; i++) t = __builtin_fmaf(e[i], acc[ub][i], t);
            agg[a][ub] = t;
        }
        m[a] = mn;
        }
        }
        if (last_blk) {
            // The query's four lane groups combined: with M the largest group
            // maximum, group g's share is r_g = exp(m_g - M) / sum_g' den_g'
            // exp(m_g' - M), and aggd[ub] += A B with A[unit][k = g] = agg of
            // lane (g, unit) and B[k = g][n] = r_g for n == cq, else 0.  In
            // v_mfma_f32_16x16x4f32 lane l holds A[l % 16][l / 16], B[l / 16]
            // [l % 16] and D[4 (l / 16) + i][l % 16]: the product sums the
            // groups, normalises, and leaves query cq's aggregate in column cq
            // of the D layout.
#pragma unroll
            for (int a = 0; a < HEADS; a++) {
                const float M = groups_max(m[a]);
                const float shift = (M == -INFINITY) ? 0.0f : M * kLog2eAgg;
                const float r = __builtin_amdgcn_exp2f(__builtin_fmaf(m[a], kLog2eAgg, -shift));
                float ds = den[a] * r;
                ds = groups_sum(ds);
                const float f = ds > 0.0f ? r * __builtin_amdgcn_rcpf(ds) : 0.0f;
                const float bq = r16 == cq ? f : 0.0f;
#pragma unroll
                for (int ub = 0; ub < 4; ub++)
                    aggd[a][ub] = __builtin_amdgcn_mfma_f32_16x16x4f32(agg[a][ub], bq, aggd[a][ub], 0, 0, 0);
                if (a == 0 && r16 == cq) ne = ds > 0.0f ? 1.0f : 0.0f;
                m[a] = -INFINITY;
                den[a] = 0.0f;
#pragma unroll
                for (int ub = 0; ub < 4; ub++) agg[a][ub] = 0.0f;
            }
        }
        if (group_end) {
            mlp_out_group<NKS, NK, L::ls3, kPs, HEADS>(p, ru, nr, vq, aggd, ne, W2, W3, W4, b2, b3, b4, r16, g,
                                                       cg * gq);
#pragma unroll
            for (int a = 0; a < HEADS; a++)
#pragma unroll
                for (int ub = 0; ub < 4; ub++) aggd[a][ub] = f32x4(0.0f);
            ne = 0.0f;
            cg += gstep;
            cq = 0;
            cb = 0;
            if (cg < groups) {
                cnq = group_size(cg);
                mo_nd = p.node[min(cg * gq + r16, (uint64_t)p.nq - 1)];
            }
        } else if (last_blk) {
            cq++;
            cb = 0;
        } else {
            cb++;
        }
        sl_c = sl_n;
        rows_c = rows_n;
    }
}

// ---------------------------------------------------------------- packed rows
// aggregate_packed: the computation of aggregate_rows with the valid rows of
// a query group packed into full 16-row blocks, for tables of at most 16
// slots.  In aggregate_rows every query takes a whole 16-row block, so with
// s = 10 and two thirds of the slots valid, three fifths of the rows that
// the matrix cores and the softmax process are empty.
//
// Per group of up to 16 queries a wavefront first reads all of the group's
// slot words (lane (q = l % 16, g = l / 16) slots g, g + 4, g + 8, g + 12 of
// query q, issued one group ahead), applies eq. (1) and writes the valid
// slots to a list in LDS, query by query, with each entry's query in a byte
// array beside it.  The list is then processed in 16-row blocks, whose rows
// may belong to several queries.  After the transposed layer 1, lane group g
// holds rows 4 g + i; each lane keeps the running maximum M_q and sum of
// exponentials of its column q = l % 16, and the block's rows are added to
// their queries' columns of the running aggregates by fp32 matrix products:
// for each i, A holds the rows 4 g + i of layer 1 (unit x lane group) and B
// the rows' weights exp(logit - M_q) in their queries' columns, so the
// product sums each row into its own query (the columns are rescaled first
// when a query's maximum grows).  At the group's end every column is divided
// by its sum of exponentials and MLP_out runs as in aggregate_rows.  Results
// differ from aggregate_rows by summation order only.  With two heads every
// row has one logit per head (v_a . a1 over all 64 units of layer 1), and
// each head keeps its own M_q, sum of exponentials and running aggregates;
// MLP_out takes head a's slice of w2's outputs from head a's aggregates.
constexpr uint32_t kPackMaxS = 16;                    // slots per node at most
constexpr uint32_t kPackMinGroup = 8;                 // queries per group at least
constexpr uint32_t kScanJ = kPackMaxS / 4;           // slots per lane in the group scan
constexpr uint32_t kPackList = kMaxGroupQ * kPackMaxS;   // list entries per group at most

// One list entry: a valid slot of query q of the group (x < 0: past the list).
struct PackEntry {
    int32_t x;
    uint32_t e;
    uint32_t q;
    float dt;
};

// A lane's row of a block, and the queries of its lane group's four rows
// (one byte each, 255 past the list).
struct PackRow {
    PackEntry en;
    uint32_t q4;
};

// LDS layout: weights and time-encoding vectors as RowsLayout (biases and
// the HEADS logit vectors in vec), then each wavefront's list.
template <int K1S, int K3S, int TKS, int HEADS>
struct PackedLayout {
    // w2 / w4 rows padded like the others, so that the 16-byte operand reads
    // of 16 consecutive rows fall on distinct banks.
    static constexpr uint32_t ls1 = 32u * K1S + 8u, ls3 = 32u * K3S + 8u, ps = kH + 8u;
    static constexpr uint32_t o_w1 = 0;
    static constexpr uint32_t o_w2 = o_w1 + kH * ls1 * 2u;
    static constexpr uint32_t o_w3 = o_w2 + kH * ps * 2u;
    static constexpr uint32_t o_w4 = o_w3 + kH * ls3 * 2u;
    static constexpr uint32_t o_vec = o_w4 + kH * ps * 2u;
    static constexpr uint32_t o_tenc = o_vec + (4u + HEADS) * kH * 4u;
    static constexpr uint32_t o_list = o_tenc + 2u * 32u * TKS * 4u;
    static constexpr uint32_t o_qs = o_list + (kRowThreads / 64) * kPackList * (uint32_t)sizeof(PackEntry);
    static constexpr uint32_t bytes = o_qs + (kRowThreads / 64) * kPackList;
};

// Time-encoding columns in lane-group order: k-step ks, lane group g and
// element i of a lane's 8-element operand piece hold column 4 (8 ks + i) + g,
// so with d_time columns every lane group needs elements j = 8 ks + i <
// ceil(d_time / 4) only -- a bound common to all lanes.
__device__ __forceinline__ uint32_t tenc_column(uint32_t kk) {
    const uint32_t ks = kk >> 5, g = (kk >> 3) & 3u, i = kk & 7u;
    return 4u * (8u * ks + i) + g;
}

template <int NKS, int EKS, int TKS, int NK, int EK, int HEADS>
__global__ __launch_bounds__(kRowThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void aggregate_packed(RowParams p) {
    constexpr int GS = NKS + EKS, K1S = GS + TKS, K3S = NKS + 2;
    using L = PackedLayout<K1S, K3S, TKS, HEADS>;
    static_assert(HEADS == 1 || HEADS == 2, "one or two heads");
    static_assert(NKS <= kRuSteps, "shape");
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    __bf16 *W1 = (__bf16 *)(smem + L::o_w1);
    __bf16 *W2 = (__bf16 *)(smem + L::o_w2);
    __bf16 *W3 = (__bf16 *)(smem + L::o_w3);
    __bf16 *W4 = (__bf16 *)(smem + L::o_w4);
    float *vec = (float *)(smem + L::o_vec);   // b1 | b2 | b3 | b4 | v_0 (| v_1), 64 each

    // Stage the weights as aggregate_rows does, except that the time-encoding
    // columns of w1 (and w, b) go in lane-group order (tenc_column).
    // (Each loop unrolled so that several iterations' loads are in flight
    // before their LDS stores: the staging is latency-bound otherwise.)
    const uint32_t tid = threadIdx.x;
#pragma unroll 8
    for (uint32_t u = tid; u < kH * (GS * 4u); u += kRowThreads) {
        const uint32_t r = u / (GS * 4u), c = (u % (GS * 4u)) * 8;
        *(bf16x8 *)(W1 + r * L::ls1 + c) = *(const bf16x8 *)(p.w1 + (size_t)r * (32u * K1S) + c);
    }
    // Time-encoding columns: 16-byte pieces of 8 columns c0 + e (c0 = 32 ks +
    // 8 j), element e to position kk = 32 ks + 8 (e % 4) + 2 j + e / 4, so
    // elements e and e + 4 form one 4-byte word (columns past d_time zero).
#pragma unroll 4
    for (uint32_t u = tid; u < kH * (4u * TKS); u += kRowThreads) {
        const uint32_t r = u / (4u * TKS), c0 = (u % (4u * TKS)) * 8u;
        const u32x4 v = *(const u32x4 *)(p.w1 + (size_t)r * (32u * K1S) + 32u * GS + c0);
        uint32_t el[8];
#pragma unroll
        for (int e = 0; e < 8; e++)
            el[e] = c0 + e < p.d_time ? (v[e >> 1] >> (16 * (e & 1))) & 0xFFFFu : 0u;
        const uint32_t kb = 32u * (c0 >> 5) + 2u * ((c0 & 31u) >> 3);
#pragma unroll
        for (int g = 0; g < 4; g++)
            *(uint32_t *)(W1 + r * L::ls1 + 32u * GS + kb + 8u * g) = el[g] | (el[g + 4] << 16);
    }
    if constexpr (NKS > 0) {
#pragma unroll 8
        for (uint32_t u = tid; u < kH * (NKS * 4u); u += kRowThreads) {
            const uint32_t r = u / (NKS * 4u), c = (u % (NKS * 4u)) * 8;
            *(bf16x8 *)(W3 + r * L::ls3 + c) = *(const bf16x8 *)(p.w3 + (size_t)r * (32u * K3S) + c);
        }
    }
    // Chain-ordered columns: a 16-byte piece of 8 columns gc0 + e lands as two
    // 8-byte halves, at the LDS columns of gc0 and gc0 + 4.
#pragma unroll 4
    for (uint32_t u = tid; u < kH * (kH / 8u); u += kRowThreads) {
        const uint32_t r = u / (kH / 8u), gc0 = (u % (kH / 8u)) * 8u;
        const u32x4 v2 = *(const u32x4 *)(p.w2 + r * kH + gc0), v4 = *(const u32x4 *)(p.w4 + r * kH + gc0),
                    v3 = *(const u32x4 *)(p.w3 + (size_t)r * (32u * K3S) + 32u * NKS + gc0);
        const uint32_t c0 = chain_pos(gc0), c1 = chain_pos(gc0 + 4u);
        *(u32x2 *)(W2 + r * L::ps + c0) = u32x2{v2[0], v2[1]};
        *(u32x2 *)(W2 + r * L::ps + c1) = u32x2{v2[2], v2[3]};
        *(u32x2 *)(W4 + r * L::ps + c0) = u32x2{v4[0], v4[1]};
        *(u32x2 *)(W4 + r * L::ps + c1) = u32x2{v4[2], v4[3]};
        *(u32x2 *)(W3 + r * L::ls3 + 32u * NKS + c0) = u32x2{v3[0], v3[1]};
        *(u32x2 *)(W3 + r * L::ls3 + 32u * NKS + c1) = u32x2{v3[2], v3[3]};
    }
    for (uint32_t u = tid; u < (4u + HEADS) * kH; u += kRowThreads) {
        const uint32_t k = u / kH, c = u % kH;
        float val;
        if (k < 4) {
            val = (k == 0 ? p.b1 : k == 1 ? p.b2 : k == 2 ? p.b3 : p.b4)[c];
        } else {
            val = 0.0f;
            const uint32_t r0 = (k - 4u) * (kH / HEADS);
#pragma unroll
            for (uint32_t r = 0; r < kH / HEADS; r++)
                val = __builtin_fmaf(p.att[r0 + r], (float)p.w2[(r0 + r) * kH + c], val);
        }
        vec[u] = val;
    }
    float *tw = (float *)(smem + L::o_tenc), *tb = tw + 32 * TKS;
    for (uint32_t kk = tid; kk < 32u * TKS; kk += kRowThreads) {
        const uint32_t c = tenc_column(kk);
        tw[kk] = c < p.d_time ? p.w[c] : 0.0f;
        tb[kk] = c < p.d_time ? p.b[c] : 0.0f;
    }
    __syncthreads();
    float wmax = 0.0f, bmax = 0.0f;
    for (uint32_t u = tid & 63; u < 32u * TKS; u += 64) {
        wmax = fmaxf(wmax, fabsf(tw[u]));
        bmax = fmaxf(bmax, fabsf(tb[u]));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        wmax = fmaxf(wmax, __shfl_xor(wmax, o));
        bmax = fmaxf(bmax, __shfl_xor(bmax, o));
    }
    wmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(wmax)));
    bmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(bmax)));
    // Elements of the last time-encoding k-step that a lane group computes.
    const uint32_t t_last = TKS > 0 ? (p.d_time + 3u) / 4u - 8u * (uint32_t)(TKS - 1) : 0u;

    const uint32_t lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t r16 = lane & 15, g = lane >> 4;
    PackEntry *lst = (PackEntry *)(smem + L::o_list) + (size_t)wave * kPackList;
    uint8_t *qs = smem + L::o_qs + (size_t)wave * kPackList;
    const float *b1 = vec, *b2 = vec + kH, *b3 = vec + 2 * kH, *b4 = vec + 3 * kH, *va = vec + 4 * kH;
    float b1v[4], vav1[4];
#pragma unroll
    for (int ub = 0; ub < 4; ub++) {
        b1v[ub] = b1[16 * ub + r16];
        vav1[ub] = va[16 * ub + r16];
    }
    const uint32_t gq = p.gq;
    const uint64_t groups = ((uint64_t)p.nq + gq - 1) / gq;
    const uint64_t gstep = (uint64_t)gridDim.x * (kRowThreads / 64);
    const uint64_t g0 = (uint64_t)wave * gridDim.x + blockIdx.x;
    if (g0 >= groups) return;   // no workgroup barrier follows

    auto group_size = [&](uint64_t grp) -> uint32_t {
        return grp < groups ? (uint32_t)min((uint64_t)gq, (uint64_t)p.nq - grp * gq) : 0u;
    };
    // Query ids of a group: query r16 of it in the lanes with that r16 (lanes
    // past the group's last query read the launch's last query, unused).
    auto load_ids = [&](uint64_t grp, int32_t &nd, uint32_t &t) {
        const uint64_t q = min(grp * gq + r16, (uint64_t)p.nq - 1);
        nd = p.node[q];
        t = p.tq[q];
    };
    // The group scan's slot words, read unconditionally (a slot past s, a
    // query past the group or an out-of-range node reads slot 0 of node 0
    // and is marked not ok).
    struct ScanRaw {
        uint64_t key[kScanJ];
        int32_t x[kScanJ];
        uint32_t tq, okm;
    };
    auto issue_scan = [&](uint64_t grp, int32_t nd, uint32_t t, ScanRaw &sr) {
        const bool in = r16 < group_size(grp) && nd >= 0 && (int64_t)nd < p.num_nodes;
        const uint8_t *bp = p.blocks + (size_t)(in ? nd : 0) * p.block_bytes;
        sr.tq = t;
        sr.okm = 0;
#pragma unroll
        for (uint32_t j = 0; j < kScanJ; j++) {
            const uint32_t a = g + 4u * j;
            const bool ok = in && a < p.s;
            const uint32_t aa = ok ? a : 0u;
            sr.key[j] = ((const uint64_t *)bp)[aa];
            sr.x[j] = ((const int32_t *)(bp + 8u * p.s))[aa];
            sr.okm |= (ok ? 1u : 0u) << j;
        }
    };
    // eq. (1) on the scanned words, then the list: query q's valid slots at
    // base_q .. base_q + v_q - 1 (lane groups in order), and the entries'
    // queries in qs, with 255 up to the end of the last block.  Returns the
    // list length.
    auto build_list = [&](const ScanRaw &sr) -> uint32_t {
        SlotLds sl[kScanJ];
        uint32_t c = 0;
#pragma unroll
        for (uint32_t j = 0; j < kScanJ; j++) {
            sl[j] = decode_slot(((sr.okm >> j) & 1u) ? sr.key[j] : 0ull, sr.x[j], sr.tq);
            c += sl[j].x >= 0 ? 1u : 0u;
        }
        // Inclusive prefix over the query's four lane groups, and its total.
        uint32_t inc = c;
        const uint32_t u16 = (uint32_t)__shfl_up((int)inc, 16);
        if (g >= 1) inc += u16;
        const uint32_t u32 = (uint32_t)__shfl_up((int)inc, 32);
        if (g >= 2) inc += u32;
        const uint32_t vq = (uint32_t)__shfl((int)inc, (int)(48u + r16));
        // Exclusive prefix of the runs over the 16 queries.
        uint32_t run = vq;
#pragma unroll
        for (uint32_t d = 1; d < 16; d <<= 1) {
            const uint32_t t = (uint32_t)__shfl_up((int)run, d, 16);
            if (r16 >= d) run += t;
        }
        const uint32_t base = run - vq;
        const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)run, 15);
        uint32_t pos = base + (inc - c);
#pragma unroll
        for (uint32_t j = 0; j < kScanJ; j++) {
            if (sl[j].x >= 0) {
                lst[pos] = PackEntry{sl[j].x, sl[j].e, r16, sl[j].dt};
                qs[pos] = (uint8_t)r16;
                pos++;
            }
        }
        if (lane < 16 && total + lane < ((total + 15u) & ~15u)) qs[total + lane] = 0xFFu;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        return total;
    };
    // Row r16 of block b of a list of n entries (past the end: empty), and
    // the queries of rows 4 g .. 4 g + 3.
    auto read_entry = [&](uint32_t n, uint32_t b) -> PackRow {
        const uint32_t idx = 16u * b + r16;
        PackRow pr;
        pr.en = lst[min(idx, n - 1u)];
        pr.q4 = *(const uint32_t *)(qs + 16u * b + 4u * g);
        if (idx >= n) {
            pr.en.x = -1;
            pr.en.dt = 0.0f;
        }
        return pr;
    };
    struct Rows {
        Piece8<NK> n[NKS > 0 ? NKS : 1];
        Piece8<EK> e[EKS > 0 ? EKS : 1];
    };
    auto issue_rows = [&](const PackEntry &en, Rows &r) {
        const bool valid = en.x >= 0;
        if constexpr (NKS > 0) {
            const uint8_t *nrow = p.nfeat + (size_t)(valid ? en.x : 0) * p.nrb;
#pragma unroll
            for (int ks = 0; ks < NKS; ks++) load_piece<NK>(nrow, p.n_dim, 32u * ks + 8u * g, r.n[ks]);
        }
        if constexpr (EKS > 0) {
            const bool ev = valid && (int64_t)en.e < p.edge_rows;
            const uint8_t *erow = p.efeat + (size_t)(ev ? en.e : 0u) * p.erb;
#pragma unroll
            for (int ks = 0; ks < EKS; ks++) load_piece<EK>(erow, p.e_dim, 32u * ks + 8u * g, r.e[ks]);
        }
    };

    // Running state of the group, per head a: aggd[a] holds, in the D
    // layout, each query's sum over its merged partials of exp(m - M) times
    // the partial's exponential-weighted sums, and the lanes with r16 == q
    // hold M_q (mrun[a]) and the matching sum of exponentials (drun[a]).
    f32x4 aggd[HEADS][4];
    float mrun[HEADS], drun[HEADS];
#pragma unroll
    for (int a = 0; a < HEADS; a++) {
#pragma unroll
        for (int ub = 0; ub < 4; ub++) aggd[a][ub] = f32x4(0.0f);
        mrun[a] = -INFINITY;
        drun[a] = 0.0f;
    }

    auto compute_block = [&](const PackRow &pr, const Rows &rc) {
        const PackEntry &en = pr.en;
        const bool valid = en.x >= 0;
        const bool ev = valid && (int64_t)en.e < p.edge_rows;
        f32x4 acc[4];
#pragma unroll
        for (int ub = 0; ub < 4; ub++) acc[ub] = f32x4(b1v[ub]);   // + b1
#pragma unroll
        for (int ks = 0; ks < NKS; ks++) {
            bf16x8 hi, lo;
            piece_operand<NK>(rc.n[ks], p.n_dim, 32u * ks + 8u * g, valid, hi, lo);
            mfma4t(acc, W1, L::ls1, 32u * ks, r16, g, hi, lo, NK == kF32Vec);
        }
#pragma unroll
        for (int ks = 0; ks < EKS; ks++) {
            bf16x8 hi, lo;
            piece_operand<EK>(rc.e[ks], p.e_dim, 32u * ks + 8u * g, ev, hi, lo);
            mfma4t(acc, W1, L::ls1, 32u * (NKS + ks), r16, g, hi, lo, EK == kF32Vec);
        }
        // Time encodings of the block's rows (an empty row has dt = 0; its
        // finite values get zero weight in the softmax).
        const float dtmax =
            __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(xor16_max(en.dt))));
        if (wmax * dtmax + bmax < 0.5f * kCosFastLimit) {
            // Every k-step but the last computes all of its elements; the
            // last computes the first t_last (the others have zero weight).
#pragma unroll 1
            for (int ks = 0; ks < TKS - 1; ks++) {
                const uint32_t k = 32u * ks + 8u * g;
                const f32x4 w0 = *(const f32x4 *)(tw + k), w1 = *(const f32x4 *)(tw + k + 4);
                const f32x4 c0 = *(const f32x4 *)(tb + k), c1 = *(const f32x4 *)(tb + k + 4);
                float t[8];
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    t[i] = cos_fast(__builtin_fmaf(w0[i], en.dt, c0[i]));
                    t[4 + i] = cos_fast(__builtin_fmaf(w1[i], en.dt, c1[i]));
                }
                bf16x8 hi, lo;
                split8(t, hi, lo);
                mfma4t(acc, W1, L::ls1, 32u * (GS + ks), r16, g, hi, lo, true);
            }
            if constexpr (TKS > 0) {
                const uint32_t k = 32u * (TKS - 1) + 8u * g;
                float t[8];
#pragma unroll
                for (int i = 0; i < 8; i++) {
                    t[i] = 0.0f;
                    if ((uint32_t)i < t_last) t[i] = cos_fast(__builtin_fmaf(tw[k + i], en.dt, tb[k + i]));
                }
                bf16x8 hi, lo;
                split8(t, hi, lo);
                mfma4t(acc, W1, L::ls1, 32u * (GS + TKS - 1), r16, g, hi, lo, true);
            }
        } else {
#pragma unroll 1
            for (int ks = 0; ks < TKS; ks++) {
                const uint32_t k = 32u * ks + 8u * g;
                float t[8];
#pragma unroll
                for (int i = 0; i < 8; i++) t[i] = cos_fp32(__builtin_fmaf(tw[k + i], en.dt, tb[k + i]));
                bf16x8 hi, lo;
                split8(t, hi, lo);
                mfma4t(acc, W1, L::ls1, 32u * (GS + ks), r16, g, hi, lo, true);
            }
        }
#pragma unroll
        for (int ub = 0; ub < 4; ub++)
#pragma unroll
            for (int i = 0; i < 4; i++) acc[ub][i] = relu(acc[ub][i]);
        const uint32_t nib = ((uint32_t)__builtin_amdgcn_ballot_w64(valid) >> (4u * g)) & 0xFu;
        // The block's rows into their queries' columns: the lane's column is
        // query r16.
        bool mine[4];
#pragma unroll
        for (int i = 0; i < 4; i++) mine[i] = ((pr.q4 >> (8 * i)) & 0xFFu) == r16;
#pragma unroll
        for (int a = 0; a < HEADS; a++) {
            // Head a's logits of rows 4 g + i (the lane group's rows; -inf
            // where empty); bm is the largest of its rows in the block.
            // (one head: the logit vector kept in registers; two: read from
            // LDS per block, the registers being taken by the aggregates)
            float vav[4];
#pragma unroll
            for (int ub = 0; ub < 4; ub++) vav[ub] = HEADS == 1 ? vav1[ub] : va[a * kH + 16 * ub + r16];
            float lg[4];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                float t = vav[0] * acc[0][i];
#pragma unroll
                for (int ub = 1; ub < 4; ub++) t = __builtin_fmaf(vav[ub], acc[ub][i], t);
                lg[i] = xor16_sum(t);
            }
#pragma unroll
            for (int i = 0; i < 4; i++) lg[i] = ((nib >> i) & 1u) ? lg[i] : -INFINITY;
            float bm = -INFINITY;
#pragma unroll
            for (int i = 0; i < 4; i++) bm = max2(bm, mine[i] ? lg[i] : -INFINITY);
            bm = groups_max(bm);
            const float mnew = max2(mrun[a], bm);
            const float scl =
                (mrun[a] == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f((mrun[a] - mnew) * kLog2eAgg);
            const float sh = (mnew == -INFINITY) ? 0.0f : mnew * kLog2eAgg;
            float wr[4];
#pragma unroll
            for (int i = 0; i < 4; i++)
                wr[i] = mine[i] ? __builtin_amdgcn_exp2f(__builtin_fmaf(lg[i], kLog2eAgg, -sh)) : 0.0f;
            const float dc = groups_sum((wr[0] + wr[1]) + (wr[2] + wr[3]));
            drun[a] = __builtin_fmaf(drun[a], scl, dc);
            mrun[a] = mnew;
#pragma unroll
            for (int ub = 0; ub < 4; ub++)
#pragma unroll
                for (int j = 0; j < 4; j++) aggd[a][ub][j] *= scl;
            // aggd[a][ub] += A_i B_i over the rows 4 g + i: A_i[unit][k = g]
            // is layer 1 of row 4 g + i (this lane's acc[ub][i]), B_i[k = g][n]
            // the row's weight in column n (this lane's wr[i] for n = r16).
#pragma unroll
            for (int i = 0; i < 4; i++)
#pragma unroll
                for (int ub = 0; ub < 4; ub++)
                    aggd[a][ub] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[ub][i], wr[i], aggd[a][ub], 0, 0, 0);
        }
    };

    // Prologue: the first group's list and the next group's scan in flight.
    // This lane's query node of the current group (mo_nd, for MLP_out) and
    // of the next (nx_nd); id_nd / id_t: the ids of the group whose scan is
    // issued next.
    int32_t mo_nd, nx_nd, id_nd;
    uint32_t id_t;
    load_ids(g0, mo_nd, id_t);
    ScanRaw sr;
    issue_scan(g0, mo_nd, id_t, sr);
    load_ids(g0 + gstep, nx_nd, id_t);
    uint32_t n_cur = build_list(sr);
    issue_scan(g0 + gstep, nx_nd, id_t, sr);
    load_ids(g0 + 2 * gstep, id_nd, id_t);
    PackRow en_c = n_cur ? read_entry(n_cur, 0) : PackRow{PackEntry{-1, 0u, 0u, 0.0f}, ~0u};
    Rows rows_c;
    issue_rows(en_c.en, rows_c);

    for (uint64_t cg = g0; cg < groups; cg += gstep) {
        asm volatile("" ::: "memory");
        const uint32_t cnq = group_size(cg);
        const bool vq = r16 < cnq;
        const int32_t nr = (vq && mo_nd >= 0 && (int64_t)mo_nd < p.num_nodes) ? mo_nd : -1;
        const uint32_t nb = (n_cur + 15u) / 16u;
        Piece8<NK> ru[NKS > 0 ? NKS : 1];
        uint32_t n_next = 0;
        // The step to the next group, taken at the current group's last block
        // (or at once for a group without blocks): this group's MLP_out rows
        // r_u, the next group's list (its scan was issued a group ago) and
        // the next group's first block of rows.  The scan of the group after
        // is issued once the blocks are done.
        auto advance = [&](PackRow &en_n, Rows &rows_n) {
            if constexpr (NKS > 0) {
                const uint8_t *urow = p.nfeat + (size_t)(nr >= 0 ? nr : 0) * p.nrb;
#pragma unroll
                for (int ks = 0; ks < NKS; ks++) load_piece<NK>(urow, p.n_dim, 32u * ks + 8u * g, ru[ks]);
            }
            n_next = build_list(sr);
            en_n = n_next ? read_entry(n_next, 0) : PackRow{PackEntry{-1, 0u, 0u, 0.0f}, ~0u};
            issue_rows(en_n.en, rows_n);
        };
        if (nb == 0) {
            PackRow en_n;
            Rows rows_n;
            advance(en_n, rows_n);
            en_c = en_n;
            rows_c = rows_n;
        }
        for (uint32_t b = 0; b < nb; b++) {
            // Keeps the LDS-resident weights from being hoisted out of the
            // loop into long-lived registers.
            asm volatile("" ::: "memory");
            PackRow en_n;
            Rows rows_n;
            if (b + 1 < nb) {
                en_n = read_entry(n_cur, b + 1);
                issue_rows(en_n.en, rows_n);
            } else {
                advance(en_n, rows_n);
            }
            // Keep the scheduler from sinking the loads to their uses.
            __builtin_amdgcn_sched_barrier(0);
            compute_block(en_c, rows_c);
            en_c = en_n;
            rows_c = rows_n;
        }
        issue_scan(cg + 2 * gstep, id_nd, id_t, sr);
        mo_nd = nx_nd;
        nx_nd = id_nd;
        load_ids(cg + 3 * gstep, id_nd, id_t);
        // The group's aggregates, normalised, then MLP_out.
        // (every head has the same valid rows: drun[0] > 0 iff the query
        // has one)
        const float ne = drun[0] > 0.0f ? 1.0f : 0.0f;
#pragma unroll
        for (int a = 0; a < HEADS; a++) {
            const float inv = drun[a] > 0.0f ? __builtin_amdgcn_rcpf(drun[a]) : 0.0f;
#pragma unroll
            for (int ub = 0; ub < 4; ub++)
#pragma unroll
                for (int i = 0; i < 4; i++) aggd[a][ub][i] *= inv;
        }
        mlp_out_group<NKS, NK, L::ls3, L::ps, HEADS>(p, ru, nr, vq, aggd, ne, W2, W3, W4, b2, b3, b4, r16, g,
                                                     cg * gq);
#pragma unroll
        for (int a = 0; a < HEADS; a++) {
#pragma unroll
            for (int ub = 0; ub < 4; ub++) aggd[a][ub] = f32x4(0.0f);
            mrun[a] = -INFINITY;
            drun[a] = 0.0f;
        }
        n_cur = n_next;
    }
}

// LDS layout of a tile with `rows` slot rows and `qrows` query rows.
uint32_t agg_layout(AggParams &p, uint32_t rows, uint32_t qrows) {
    p.rows = rows;
    p.qrows = qrows;
    p.region_off = align16(16u * rows + 4u * qrows);
    const uint32_t x_bytes = 2u * rows * p.xs * 2u;
    p.off_h = rows * kHs * 2u * 2u;
    p.off_y = align16(p.off_h + rows * kHf * 4u + rows * 4u * p.heads);
    p.off_a3 = align16(p.off_y + 2u * qrows * p.ys * 2u);
    const uint32_t late = p.off_a3 + 2u * qrows * kHs * 2u;
    return p.region_off + (x_bytes > late ? x_bytes : late);
}

}  // namespace

extern "C" int nlb_aggregate(nlb_table *h, const int32_t *node, const uint32_t *tq, uint32_t nq,
                             const nlb_agg_weights *wts, float *z, void *stream) {
    if (!h || !wts) return NLB_EINVAL;
    if (nq == 0) return NLB_OK;
    if (!node || !tq || !z) return NLB_EINVAL;
    if (wts->hidden != kH) return NLB_EINVAL;
    const uint32_t heads = wts->heads <= 1 ? 1u : (uint32_t)wts->heads;
    if (heads != 1 && heads != 2 && heads != 4 && heads != 8) return NLB_EINVAL;
    if (!wts->w1 || !wts->w2 || !wts->w3 || !wts->w4 || !wts->b1 || !wts->b2 || !wts->b3 ||
        !wts->b4 || !wts->att)
        return NLB_EINVAL;
    if (((uintptr_t)wts->w1 | (uintptr_t)wts->w2 | (uintptr_t)wts->w3 | (uintptr_t)wts->w4) % 16)
        return NLB_EINVAL;
    if ((uintptr_t)z % 4) return NLB_EINVAL;
    const int32_t nd = wts->node_dtype, ed = wts->edge_dtype;
    if ((nd != NLB_DTYPE_F32 && nd != NLB_DTYPE_BF16) || (ed != NLB_DTYPE_F32 && ed != NLB_DTYPE_BF16))
        return NLB_EINVAL;
    const uint32_t n_es = nd == NLB_DTYPE_BF16 ? 2 : 4, e_es = ed == NLB_DTYPE_BF16 ? 2 : 4;
    if (h->nrb % n_es || h->erb % e_es) return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;

    AggParams p;
    std::memset(&p, 0, sizeof(p));
    p.blocks = h->blocks;
    p.block_bytes = h->block_bytes;
    p.s = h->s;
    p.num_nodes = h->num_nodes;
    p.node = node;
    p.tq = tq;
    p.nq = nq;
    p.s_m = nlb_div_magic(h->s);
    p.d_time = h->d_time;
    p.w = h->w;
    p.b = h->b;
    p.efeat = h->efeat;
    p.edge_rows = h->edge_rows;
    p.e_dim = h->erb / e_es;
    p.e_bf16 = ed == NLB_DTYPE_BF16;
    p.erb = h->erb;
    p.e_vec = h->erb % 16 == 0 && (uintptr_t)h->efeat % 16 == 0;
    p.nfeat = h->nfeat;
    p.n_dim = h->nrb / n_es;
    p.n_bf16 = nd == NLB_DTYPE_BF16;
    p.nrb = h->nrb;
    p.n_vec = h->nrb % 16 == 0 && (uintptr_t)h->nfeat % 16 == 0;
    p.off_e = pad32(p.n_dim);
    p.off_t = p.off_e + pad32(p.e_dim);
    p.k1 = p.off_t + pad32(h->d_time);
    p.k3 = pad32(p.n_dim) + kH;
    if (p.k1 == 0) return NLB_EINVAL;   // no inputs at all
    p.xs = p.k1 + 8;
    p.ys = p.k3 + 8;
    p.g1_m = nlb_div_magic(p.k1 / 8);
    p.gq_m = nlb_div_magic(pad32(p.n_dim) / 8 ? pad32(p.n_dim) / 8 : 1);
    p.w1 = (const __bf16 *)wts->w1;
    p.w2 = (const __bf16 *)wts->w2;
    p.w3 = (const __bf16 *)wts->w3;
    p.w4 = (const __bf16 *)wts->w4;
    p.b1 = wts->b1;
    p.b2 = wts->b2;
    p.b3 = wts->b3;
    p.b4 = wts->b4;
    p.att = wts->att;
    p.z = z;
    p.status = h->status;
    p.heads = heads;

    // The wavefront-per-query kernel, for the input shapes it is instantiated
    // for (those of the synthetic workloads) when its weights fit one
    // workgroup's LDS; other shapes take the tiled kernel.
    const uint32_t nks = p.off_e / 32, eks = (p.off_t - p.off_e) / 32, tks = (p.k1 - p.off_t) / 32;
    const int nkind = nks ? piece_kind(p.nrb, p.nfeat, p.n_bf16) : 0;
    const int ekind = eks ? piece_kind(p.erb, p.efeat, p.e_bf16) : 0;
    if (nq >= kRowsMinQueries && nkind >= 0 && ekind >= 0) {
        RowParams r;
        std::memset(&r, 0, sizeof(r));
        r.blocks = p.blocks;
        r.block_bytes = p.block_bytes;
        r.s = p.s;
        r.num_nodes = p.num_nodes;
        r.node = node;
        r.tq = tq;
        r.nq = nq;
        r.nbq = (h->s + 15u) / 16u;
        r.d_time = p.d_time;
        r.nch = (p.d_time + 3u) / 4u;
        r.nch_m = r.nch ? ((1ull << 32) + r.nch - 1) / r.nch : 0u;
        r.w = p.w;
        r.b = p.b;
        r.efeat = p.efeat;
        r.edge_rows = p.edge_rows;
        r.e_dim = p.e_dim;
        r.erb = p.erb;
        r.nfeat = p.nfeat;
        r.n_dim = p.n_dim;
        r.nrb = p.nrb;
        r.w1 = p.w1;
        r.w2 = p.w2;
        r.w3 = p.w3;
        r.w4 = p.w4;
        r.b1 = p.b1;
        r.b2 = p.b2;
        r.b3 = p.b3;
        r.b4 = p.b4;
        r.att = p.att;
        r.z = z;
        r.status = h->status;
        const void *kern = nullptr;
        uint32_t bytes = 0;
        void (*launch)(dim3, uint32_t, hipStream_t, const RowParams &) = nullptr;
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess || cus < 1)
            return NLB_EDEVICE;
        // One persistent workgroup per CU; groups of up to 16 queries, fewer
        // when that leaves wavefronts without one.
        const uint64_t waves = (uint64_t)cus * (kRowThreads / 64);
        r.gq = (uint32_t)std::min<uint64_t>(kMaxGroupQ, std::max<uint64_t>(1, (nq + waves - 1) / waves));
        // Tables of at most 16 slots take the packed form when the groups
        // are large enough for packing to fill blocks (small launches are
        // bound by their per-group steps).
        const bool packed = h->s <= kPackMaxS && r.gq >= kPackMinGroup && heads <= 2;
        // One or two heads: the packed or the per-query kernel; more heads take
        // the tiled kernel.
        const bool rows_ok = heads <= 2;
#define NLB_ROWS_SHAPE(A, B, C, NK, EK)                                                              \
    if (!kern && rows_ok && nks == A && eks == B && tks == C && (A == 0 || nkind == NK) &&          \
        (B == 0 || ekind == EK)) {                                                                    \
        if (packed && heads == 1) {                                                                   \
            kern = (const void *)aggregate_packed<A, B, C, NK, EK, 1>;                                \
            bytes = PackedLayout<A + B + C, A + 2, C, 1>::bytes;                                      \
            launch = [](dim3 gr, uint32_t l, hipStream_t st, const RowParams &rp) {                   \
                hipLaunchKernelGGL((aggregate_packed<A, B, C, NK, EK, 1>), gr, dim3(kRowThreads), l, st, rp); \
            };                                                                                        \
        } else if (packed) {                                                                          \
            kern = (const void *)aggregate_packed<A, B, C, NK, EK, 2>;                                \
            bytes = PackedLayout<A + B + C, A + 2, C, 2>::bytes;                                      \
            launch = [](dim3 gr, uint32_t l, hipStream_t st, const RowParams &rp) {                   \
                hipLaunchKernelGGL((aggregate_packed<A, B, C, NK, EK, 2>), gr, dim3(kRowThreads), l, st, rp); \
            };                                                                                        \
        } else {                                                                                      \
            bytes = RowsLayout<A + B + C, A + 2, C>::bytes;                                           \
            if (heads == 1) {                                                                         \
                kern = (const void *)aggregate_rows<A, B, C, NK, EK, 1>;                              \
                launch = [](dim3 gr, uint32_t l, hipStream_t st, const RowParams &rp) {               \
                    hipLaunchKernelGGL((aggregate_rows<A, B, C, NK, EK, 1>), gr, dim3(kRowThreads), l, st, rp); \
                };                                                                                    \
            } else {                                                                                  \
                kern = (const void *)aggregate_rows<A, B, C, NK, EK, 2>;                              \
                launch = [](dim3 gr, uint32_t l, hipStream_t st, const RowParams &rp) {               \
                    hipLaunchKernelGGL((aggregate_rows<A, B, C, NK, EK, 2>), gr, dim3(kRowThreads), l, st, rp); \
                };                                                                                    \
            }                                                                                         \
        }                                                                                             \
    }
        // 100 time dims with: bf16 node rows 128 wide and bf16 link rows 128
        // wide or none; no node rows and fp32 link rows 100 or 172 wide, or
        // bf16 link rows 186 wide (4-byte aligned).
        NLB_ROWS_SHAPE(4, 0, 4, kBf16Vec, kBf16Vec)
        NLB_ROWS_SHAPE(4, 4, 4, kBf16Vec, kBf16Vec)
        NLB_ROWS_SHAPE(0, 6, 4, kBf16Vec, kF32Vec)
        NLB_ROWS_SHAPE(0, 4, 4, kBf16Vec, kF32Vec)
        NLB_ROWS_SHAPE(0, 6, 4, kBf16Vec, kBf16Word)
#undef NLB_ROWS_SHAPE
        if (kern && bytes <= kAggLdsMax) {
            if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kAggLdsMax) !=
                hipSuccess)
                return NLB_EDEVICE;
            const uint64_t groups = ((uint64_t)nq + r.gq - 1) / r.gq;
            launch(dim3((unsigned)std::min<uint64_t>(groups, (uint64_t)cus)), bytes, (hipStream_t)stream, r);
            if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
            return NLB_OK;
        }
    }

    // The tiled kernel holds at most 64 slot rows of one query.
    if (h->s > 16u * kMaxBlocks) return NLB_EINVAL;
    // Tile: as many queries as fit the LDS budget (at most 128 slot rows),
    // fewer when that leaves too few workgroups to fill the GPU.
    // A tile larger than one query must fit the budget that keeps four
    // workgroups per CU (the kernel is latency-bound: concurrency beats tile
    // size); a single query may use a workgroup's whole LDS.
    uint32_t tile_q = 0, lds = 0;
    const uint32_t want = (uint32_t)(((uint64_t)nq + kAggTargetTiles - 1) / kAggTargetTiles);
    for (uint32_t rows = 16u * kMaxBlocks; rows >= 16 && tile_q == 0; rows -= 16) {
        const uint32_t tq_cap = rows / h->s;
        if (tq_cap == 0) continue;
        const uint32_t t = tq_cap < (want ? want : 1) ? tq_cap : (want ? want : 1);
        AggParams trial = p;
        const uint32_t bytes = agg_layout(trial, pad16(t * h->s), pad16(t));
        if (bytes <= (t == 1 ? kAggLdsMax : kAggLdsBudget)) {
            tile_q = t;
            lds = bytes;
        }
    }
    if (tile_q == 0) return NLB_EINVAL;   // one query does not fit the LDS budget
    p.tile_q = tile_q;
    agg_layout(p, pad16(tile_q * h->s), pad16(tile_q));
    // Dynamic LDS beyond 64 KB has to be allowed per kernel before launch.
    if (lds > 64u * 1024u &&
        hipFuncSetAttribute((const void *)aggregate_fused, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kAggLdsMax) != hipSuccess)
        return NLB_EDEVICE;
    const dim3 grid((unsigned)(((uint64_t)nq + tile_q - 1) / tile_q));
    hipLaunchKernelGGL(aggregate_fused, grid, dim3(kAggThreads), lds, (hipStream_t)stream, p);
    if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
    return NLB_OK;
}
