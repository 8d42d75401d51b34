// rnn.hip -- the node-status update of Sec. 4.4 (Luo & Li, arXiv 2402.01964):
// after a link (u, v, t) with features e, each endpoint's status is updated
// by an RNN over [r_u, r_v, t, e].  The cell is a GRU with input
// x = [r_other ; T-enc(t) ; e] and hidden state h = r_self:
//   r = sigmoid(W_ir x + W_hr h + b_ir + b_hr)
//   z = sigmoid(W_iz x + W_hz h + b_iz + b_hz)
//   n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
//   h' = (1 - z) n + z h
// A batch is applied at once: every update reads the statuses from before
// the batch, and a node that several links of the batch touch takes the
// update of its latest one (larger arrival index; on a self-loop the second
// endpoint's).
//
// Four launches per batch:
//   resolve  each endpoint offers the code 2i + k + 1 of its pair row (link
//            i, endpoint k) to winner[node] with a 64-bit atomic maximum (the
//            array is all zero between calls: the scatter clears the words it
//            has used).  Large batches merge their offers per node in LDS
//            first (merge_max), as the table insertion does.
//   select   each pair row checks whether it won; the winners are appended
//            to a dense list (one atomic per wavefront).  The list order
//            varies from run to run; the results do not, because every row
//            of a matrix product depends on its own inputs only.
//   gru      where its registers suffice, the weight-stationary form
//            (rnn_gru_ws: one workgroup per CU keeps the weights in
//            registers and loops over 32-row tiles of listed rows);
//            otherwise a workgroup takes a tile of 16, 32 or 64 listed rows
//            and reads the weights from L2 (rnn_gru).  Both build the inputs
//            in LDS and run both GRU products on bf16 matrix cores; the
//            gates, the blend with h and the rounding to the status type
//            happen in registers, and the new status goes to a candidate
//            buffer indexed by pair row.
//   scatter  copies each listed winner's candidate row over its node's
//            status and clears the node's winner word.  Every node a valid
//            link touches has exactly one winner, so this restores the all-
//            zero array; no call number is needed, and a call captured in a
//            HIP graph can be replayed.
// The candidate buffer is what lets the gru pass read only pre-batch
// statuses: no status is written until every workgroup has read its inputs.
//
// Numerics.  fp32 activations (fp32 statuses, the time encoding, fp32 link
// rows) enter the products as bf16 pairs hi + lo (2^-18 relative), bf16 ones
// as a single term; the weights are bf16 and the products accumulate in fp32.
//
// Matrix-core mapping (v_mfma_f32_16x16x32_bf16; lane layout as in
// aggregate.hip).  Wavefront w computes the output units 16 ub .. 16 ub + 15
// for ub = w, w + 4, ...; for each it keeps four accumulators per 16-row
// block -- r and z (input and hidden products summed), the input part of n
// and the hidden part of n -- so a unit's three gates meet in one lane and
// the cell finishes without another LDS round trip.  The weight fragments
// (read from global memory, where the whole weight set stays L2-resident)
// go through a three-slot register ring, so each k-step's loads are issued
// two steps before their products.
#include <algorithm>
#include <cstring>
#include <mutex>

#include "nlb_internal.h"
#include "nlb_pieces.h"

namespace {

constexpr int kRnnThreads = 256;
constexpr uint32_t kGruMetaRows = 1024;           // LDS bytes of the tile's row list (4 words per row)
constexpr uint32_t kGruLdsBudget = 80 * 1024;     // two workgroups per CU
constexpr uint32_t kGruLdsMax = 160 * 1024;       // gfx950: LDS of one workgroup at most
constexpr uint32_t kGruTargetTiles = 1024;      // tiles wanted per launch (counted on 2n rows)

struct ResolveParams {
    const int32_t *src;
    const int32_t *dst;
    uint32_t n;
    int64_t num_nodes;
    unsigned long long *winner;
    uint32_t *status;
    uint32_t *count;      // winners listed by select; zeroed here
};

__device__ __forceinline__ bool endpoints_ok(int32_t u, int32_t v, int64_t num_nodes) {
    return u >= 0 && v >= 0 && (int64_t)u < num_nodes && (int64_t)v < num_nodes;
}

__global__ __launch_bounds__(kRnnThreads) void rnn_resolve(ResolveParams p) {
    const uint32_t i = blockIdx.x * kRnnThreads + threadIdx.x;
    if (i == 0) *p.count = 0;
    if (i >= p.n) return;
    const int32_t u = p.src[i], v = p.dst[i];
    if (!endpoints_ok(u, v, p.num_nodes)) {
        atomicOr(p.status, kStatusRange);
        return;
    }
    atomicMax(&p.winner[u], (unsigned long long)(2ull * i + 1));
    atomicMax(&p.winner[v], (unsigned long long)(2ull * i + 2));
}

__global__ __launch_bounds__(kMergeThreads) void rnn_resolve_merged(ResolveParams p) {
    __shared__ unsigned long long merge_off[kMergeEntries];
    __shared__ unsigned long long merge_word[kMergeEntries];
    for (int k = threadIdx.x; k < kMergeEntries; k += kMergeThreads) {
        merge_off[k] = 0ull;
        merge_word[k] = 0ull;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) *p.count = 0;
    __syncthreads();
    // All of a thread's links are loaded (a link past the batch re-reads
    // the last one, unused) before any is merged.
    constexpr int RR = kResolveLinks / kMergeThreads;
    const uint32_t first = blockIdx.x * kResolveLinks;
    int32_t uu[RR], vv[RR];
#pragma unroll
    for (int r = 0; r < RR; r++) {
        const uint32_t i = min(first + r * kMergeThreads + threadIdx.x, p.n - 1u);
        uu[r] = p.src[i];
        vv[r] = p.dst[i];
    }
#pragma unroll
    for (int r = 0; r < RR; r++) {
        const uint32_t i = first + r * kMergeThreads + threadIdx.x;
        if (i >= p.n) break;
        const int32_t u = uu[r], v = vv[r];
        if (!endpoints_ok(u, v, p.num_nodes)) {
            atomicOr(p.status, kStatusRange);
            continue;
        }
        merge_max(merge_off, merge_word, 8ull * (uint32_t)u, 2ull * i + 1);
        merge_max(merge_off, merge_word, 8ull * (uint32_t)v, 2ull * i + 2);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kMergeEntries; k += kMergeThreads) {
        const unsigned long long tag = merge_off[k];
        if (tag) atomicMax(&p.winner[(tag - 1) >> 3], merge_word[k]);
    }
}

struct SelectParams {
    const int32_t *src;
    const int32_t *dst;
    uint32_t n;
    int64_t num_nodes;
    const unsigned long long *winner;
    u32x4 *list;          // winners, dense: {pair row, self, other, 0}
    uint32_t *count;
};

// A workgroup checks kSelectRows consecutive pair rows, collects its
// winners in LDS (one LDS atomic per wavefront and pass) and appends them to
// the list with a single global atomic.
constexpr uint32_t kSelectRows = 1024;

__global__ __launch_bounds__(kRnnThreads) void rnn_select(SelectParams p) {
    __shared__ u32x4 rows[kSelectRows];
    __shared__ uint32_t n_local, base;
    const uint32_t lane = threadIdx.x & 63;
    if (threadIdx.x == 0) n_local = 0;
    __syncthreads();
    // A thread's pair rows: their links' endpoints, then the winner words
    // of their nodes, are read in two rounds of unconditional loads (rows
    // past the batch re-read the last link; invalid endpoints read
    // winner[0]) before any is used.
    constexpr int RS = kSelectRows / kRnnThreads;
    const uint64_t r0 = (uint64_t)blockIdx.x * kSelectRows;
    int32_t su[RS], sv[RS];
#pragma unroll
    for (int q = 0; q < RS; q++) {
        const uint64_t r = min(r0 + q * kRnnThreads + threadIdx.x, 2ull * p.n - 1ull);
        su[q] = p.src[(uint32_t)(r >> 1)];
        sv[q] = p.dst[(uint32_t)(r >> 1)];
    }
    unsigned long long wv[RS];
#pragma unroll
    for (int q = 0; q < RS; q++) {
        const uint64_t r = min(r0 + q * kRnnThreads + threadIdx.x, 2ull * p.n - 1ull);
        const int32_t self = (r & 1) ? sv[q] : su[q];
        wv[q] = p.winner[endpoints_ok(su[q], sv[q], p.num_nodes) ? self : 0];
    }
#pragma unroll
    for (int q = 0; q < RS; q++) {
        const uint32_t k = q * kRnnThreads + threadIdx.x;
        const uint64_t r = r0 + k;
        bool win = false;
        int32_t self = -1, other = -1;
        if (r < 2ull * p.n) {
            const int32_t u = su[q], v = sv[q];
            if (endpoints_ok(u, v, p.num_nodes)) {
                self = (r & 1) ? v : u;
                other = (r & 1) ? u : v;
                win = wv[q] == r + 1;
            }
        }
        const uint64_t mask = __ballot(win);
        if (mask == 0) continue;
        const uint32_t leader = (uint32_t)__ffsll((long long)mask) - 1u;
        uint32_t off = 0;
        if (lane == leader) off = atomicAdd(&n_local, (uint32_t)__popcll(mask));
        off = __shfl(off, (int)leader);
        if (win)
            rows[off + (uint32_t)__popcll(mask & ((1ull << lane) - 1ull))] =
                u32x4{(uint32_t)r, (uint32_t)self, (uint32_t)other, 0u};
    }
    __syncthreads();
    if (threadIdx.x == 0) base = n_local ? atomicAdd(p.count, n_local) : 0;
    __syncthreads();
    for (uint32_t k = threadIdx.x; k < n_local; k += kRnnThreads) p.list[base + k] = rows[k];
}

struct GruParams {
    const int32_t *src;
    const int32_t *dst;
    const uint32_t *t;
    uint32_t n;
    int64_t num_nodes;
    const u32x4 *list;                  // winners {pair row, self, other, 0} (select)
    const uint32_t *count;
    uint64_t first_eid;                 // arrival index (link-row index) of link 0, or NLB_EID_LAST_BATCH
    const uint32_t *table_status;       // the table's device status words (its link count)
    uint32_t d, d_time;
    const float *tw, *tb;               // time encoding
    uint32_t t_vec;                     // tw, tb 16-byte aligned
    const uint8_t *efeat;
    int64_t edge_rows;
    uint32_t e_dim, e_bf16, erb, e_vec;
    const uint8_t *st;                  // statuses [N][d]
    uint32_t s_bf16, srb, s_vec;
    uint8_t *cand;                      // [2n][srb] candidate rows by pair row
    uint32_t kd, off_e, kx;             // X = [r_other | T-enc | e]: columns [0,kd) [kd,off_e) [off_e,kx)
    uint32_t lo_begin, lo_end;          // X columns with a stored lo plane
    uint32_t h_lo;                      // fp32 statuses: H has a lo plane
    uint32_t xs, ls, hs;                // LDS row strides (bf16 elements)
    uint32_t rows;                      // listed rows per tile (16, 32 or 64)
    uint32_t off_xl, off_h, off_hl;     // LDS byte offsets
    uint64_t gx_m, gh_m;                // nlb_div_magic(kx / 8), nlb_div_magic(kd / 8)
    uint64_t gt_m, ge_m;                // nlb_div_magic((off_e - kd) / 8), nlb_div_magic((kx - off_e) / 8)
    int32_t s_kind, e_kind;             // piece forms of status / link rows (-1: none applies)
    uint32_t meta;                      // LDS bytes before X: row list, then T-enc w | b (pad32(d_time) each)
    uint32_t ws_lomask;                 // weight-stationary form: bit s set if X k-step s has a lo plane
    uint64_t ws_cpr_m;                  // nlb_div_magic(srb / 16)
    const __bf16 *w_ih, *w_hh;
    const float *b_ih, *b_hh;
};

// Arrival index of link 0 of the batch: given, or (NLB_EID_LAST_BATCH) the
// table's device link count minus n -- the batch inserted last -- read when
// the kernel runs, so that a captured update follows the inserts replayed
// before it.
__device__ __forceinline__ uint64_t first_eid_of(const GruParams &p) {
    if (p.first_eid != NLB_EID_LAST_BATCH) return p.first_eid;
    return *(const uint64_t *)(p.table_status + kWordLinks) - p.n;
}

__device__ __forceinline__ void store_hi8(const float v[8], __bf16 *hi) {
    bf16x8 h;
#pragma unroll
    for (int i = 0; i < 8; i++) h[i] = (__bf16)v[i];
    *(bf16x8 *)hi = h;
}

// Gates from the hardware base-2 exponential and reciprocal (each within a
// few ulp): sigmoid(a) = 1 / (1 + 2^(-a log2 e)), tanh(a) = 1 - 2 / (1 +
// 2^(2 a log2 e)).  Both saturate correctly when the exponential overflows
// to infinity or underflows to zero; tanh near 0 is accurate to ~1e-7
// absolute.
constexpr float kLog2e = 1.44269504088896340736f;

__device__ __forceinline__ float sigmoid_f32(float a) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-a * kLog2e));
}

__device__ __forceinline__ float tanh_f32(float a) {
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(2.0f * kLog2e * a));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// acc[g'][rb] += A_rb (16 x 32 blocks of the LDS pair Ah/Al, row stride
// `as`; the lo plane starts at column lo_b with its own stride `ls`)
//              * W_g^T for the three gate row blocks W_g = w0 + g * gstep,
// over the k-steps kb, kb + 32, .. < ke; g' = g for the r and z gates and
// g' = NIDX for the n gate.  LO adds the lo-plane products.
template <int NB, bool LO, int NIDX>
__device__ __forceinline__ void gate_seg(f32x4 (&acc)[4][NB], const __bf16 *Ah, const __bf16 *Al,
                                         uint32_t as, uint32_t ls, uint32_t lo_b, const __bf16 *w0,
                                         size_t gstep, uint32_t kb, uint32_t ke, uint32_t lr,
                                         uint32_t lk) {
    if (kb >= ke) return;
    const uint32_t last = ke - 32;
    bf16x8 r0[3], r1[3], r2[3];
    auto load = [&](bf16x8 (&b)[3], uint32_t k) {
#pragma unroll
        for (int g = 0; g < 3; g++) b[g] = *(const bf16x8 *)(w0 + g * gstep + k);
    };
    auto step = [&](const bf16x8 (&b)[3], uint32_t k0) {
        bf16x8 a[NB], al[NB];
#pragma unroll
        for (int rb = 0; rb < NB; rb++) a[rb] = *(const bf16x8 *)(Ah + (16u * rb + lr) * as + k0 + lk);
        if (LO) {
#pragma unroll
            for (int rb = 0; rb < NB; rb++)
                al[rb] = *(const bf16x8 *)(Al + (16u * rb + lr) * ls + (k0 - lo_b) + lk);
        }
#pragma unroll
        for (int rb = 0; rb < NB; rb++)
#pragma unroll
            for (int g = 0; g < 3; g++) {
                const int gi = g == 2 ? NIDX : g;
                acc[gi][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], b[g], acc[gi][rb], 0, 0, 0);
            }
        if (LO) {
#pragma unroll
            for (int rb = 0; rb < NB; rb++)
#pragma unroll
                for (int g = 0; g < 3; g++) {
                    const int gi = g == 2 ? NIDX : g;
                    acc[gi][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[rb], b[g], acc[gi][rb], 0, 0, 0);
                }
        }
        // All LDS reads of the step first, then its products.
        __builtin_amdgcn_sched_group_barrier(0x0100, LO ? 2 * NB : NB, 0);
        __builtin_amdgcn_sched_group_barrier(0x0008, LO ? 6 * NB : 3 * NB, 0);
    };
    // Three-slot ring: the loads of step k + 64 are issued before the
    // products of step k (the scheduling barriers keep them there).
    // Prefetches past the segment re-read its last step (in bounds, unused).
    load(r0, kb);
    load(r1, kb + 32 < ke ? kb + 32 : last);
    uint32_t k0 = kb;
    for (; k0 + 64 < ke; k0 += 96) {
        load(r2, k0 + 64);
        __builtin_amdgcn_sched_barrier(0);
        step(r0, k0);
        load(r0, k0 + 96 < ke ? k0 + 96 : last);
        __builtin_amdgcn_sched_barrier(0);
        step(r1, k0 + 32);
        load(r1, k0 + 128 < ke ? k0 + 128 : last);
        __builtin_amdgcn_sched_barrier(0);
        step(r2, k0 + 64);
    }
    if (k0 < ke) step(r0, k0);
    if (k0 + 32 < ke) step(r1, k0 + 32);
}

// One input segment of a tile: `units` pieces of 8 columns, piece u of tile
// row j = u / g at column c0 = 8 (u - j g), from the row row_of(j) (a valid
// address for every j < R); store(j, c0, piece) writes it to LDS.  F pieces
// per thread (of NT) are loaded before any is stored.
template <int KIND, int F, uint32_t NT = kRnnThreads, typename RowOf, typename Store>
__device__ __forceinline__ void fill_seg(uint32_t units, uint32_t g, uint64_t g_m, uint32_t dim, RowOf row_of,
                                         Store store) {
    for (uint32_t base = threadIdx.x; base < units; base += NT * F) {
        Piece8<KIND> pc[F];
#pragma unroll
        for (int f = 0; f < F; f++) {
            const uint32_t u = min(base + f * NT, units - 1u);
            const uint32_t j = nlb_div(u, g_m), c0 = (u - j * g) * 8u;
            load_piece<KIND>(row_of(j), dim, c0, pc[f]);
        }
#pragma unroll
        for (int f = 0; f < F; f++) {
            const uint32_t u = base + f * NT;
            if (u < units) {
                const uint32_t j = nlb_div(u, g_m), c0 = (u - j * g) * 8u;
                store(j, c0, pc[f]);
            }
        }
    }
}

// A tile's inputs X = [r_other | T-enc(t) | e] and H = r_self for tile rows
// j < m (rows m .. 16 NB - 1 are written as zeros), as bf16 hi planes at Xh
// and Hh and lo planes at Xl (columns [lo_begin, lo_end)) and Hl (fp32
// statuses), with row strides xs, ls, hs -- in LDS or in global memory.
// m_row .. m_t are the tile rows' list entries and link times, s_tw / s_tb
// the zero-padded time-encoding parameters (LDS).  The caller synchronises.
template <int NB>
__device__ __forceinline__ void gru_fill(const GruParams &p, uint32_t m, const uint32_t *m_row,
                                         const int32_t *m_self, const int32_t *m_other, const float *m_t,
                                         const float *s_tw, const float *s_tb, __bf16 *Xh, __bf16 *Xl,
                                         __bf16 *Hh, __bf16 *Hl, uint32_t xs, uint32_t ls, uint32_t hs) {
    const uint64_t first_eid = first_eid_of(p);
    constexpr uint32_t R = 16 * NB;
    // Input units (8 columns each) whose loads a thread keeps in flight
    // together (generic path): about all of its units for the common widths.
    constexpr int kFill = NB == 4 ? 12 : (NB == 2 ? 8 : 4);
    const uint32_t tid = threadIdx.x;
    if (p.s_kind >= 0 && (p.e_kind >= 0 || p.kx == p.off_e)) {
        // Inputs segment by segment, each with its rows' fixed piece form:
        // statuses (H = r_self, then X's r_other), the time encoding, link
        // rows.  Rows m .. R-1 of the tile read row 0 of the list and are
        // stored as zeros.
        const uint32_t d = p.d, gh = p.kd / 8, us = R * gh;
        auto status_fill = [&](auto kind) {
            constexpr int K = decltype(kind)::value;
            // Pieces u < us: H rows (self); us <= u < 2 us: X rows (other),
            // by tile row j = u / gh over 2R rows.
            fill_seg<K, 8>(
                2u * us, gh, p.gh_m, d,
                [&](uint32_t jj) {
                    const uint32_t j = jj < R ? jj : jj - R;
                    const int32_t node = (jj < R ? m_self : m_other)[j < m ? j : 0];
                    return p.st + (size_t)node * p.srb;
                },
                [&](uint32_t jj, uint32_t c0, const Piece8<K> &pc) {
                    const uint32_t j = jj < R ? jj : jj - R;
                    const bool ok = j < m;
                    if constexpr (K == kF32Vec) {
                        float v[8];
                        piece_floats<K>(pc, d, c0, ok, v);
                        if (jj < R)
                            store_split8(v, Hh + (size_t)j * hs + c0, Hl + (size_t)j * hs + c0);
                        else
                            store_split8(v, Xh + (size_t)j * xs + c0,
                                         Xl + (size_t)j * ls + (c0 - p.lo_begin));
                    } else {
                        const u32x4 w = piece_bf16_bits<K>(pc, d, c0, ok);
                        *(u32x4 *)(jj < R ? Hh + (size_t)j * hs + c0 : Xh + (size_t)j * xs + c0) = w;
                    }
                });
        };
        if (p.s_kind == kF32Vec)
            status_fill(std::integral_constant<int, kF32Vec>{});
        else if (p.s_kind == kBf16Word)
            status_fill(std::integral_constant<int, kBf16Word>{});
        else
            status_fill(std::integral_constant<int, kBf16Vec>{});

        // Time encoding cos(w_k t + b_k) of each row's link time.
        const uint32_t gt = (p.off_e - p.kd) / 8;
        for (uint32_t u = tid; u < R * gt; u += kRnnThreads) {
            const uint32_t j = nlb_div(u, p.gt_m), k = (u - j * gt) * 8u;
            const float tf = m_t[j < m ? j : 0];
            const f32x4 w0 = *(const f32x4 *)(s_tw + k), w1 = *(const f32x4 *)(s_tw + k + 4);
            const f32x4 b0 = *(const f32x4 *)(s_tb + k), b1 = *(const f32x4 *)(s_tb + k + 4);
            float v[8];
#pragma unroll
            for (int i = 0; i < 4; i++) {
                v[i] = cos_fp32(__builtin_fmaf(w0[i], tf, b0[i]));
                v[4 + i] = cos_fp32(__builtin_fmaf(w1[i], tf, b1[i]));
            }
#pragma unroll
            for (int i = 0; i < 8; i++) v[i] = (j < m && k + i < p.d_time) ? v[i] : 0.0f;
            store_split8(v, Xh + (size_t)j * xs + p.kd + k, Xl + (size_t)j * ls + (p.kd + k - p.lo_begin));
        }

        // Link rows (rows at or past edge_rows are zeros).
        if (p.kx > p.off_e) {
            const uint32_t ge = (p.kx - p.off_e) / 8;
            auto edge_fill = [&](auto kind) {
                constexpr int K = decltype(kind)::value;
                auto eid_of = [&](uint32_t j) { return first_eid + (m_row[j < m ? j : 0] >> 1); };
                fill_seg<K, 8>(
                    R * ge, ge, p.ge_m, p.e_dim,
                    [&](uint32_t j) {
                        const uint64_t e = eid_of(j);
                        return p.efeat + (size_t)(e < (uint64_t)p.edge_rows ? e : 0u) * p.erb;
                    },
                    [&](uint32_t j, uint32_t c0, const Piece8<K> &pc) {
                        const bool ok = j < m && eid_of(j) < (uint64_t)p.edge_rows;
                        if constexpr (K == kF32Vec) {
                            float v[8];
                            piece_floats<K>(pc, p.e_dim, c0, ok, v);
                            store_split8(v, Xh + (size_t)j * xs + p.off_e + c0,
                                         Xl + (size_t)j * ls + (p.off_e + c0 - p.lo_begin));
                        } else {
                            *(u32x4 *)(Xh + (size_t)j * xs + p.off_e + c0) =
                                piece_bf16_bits<K>(pc, p.e_dim, c0, ok);
                        }
                    });
            };
            if (p.e_kind == kF32Vec)
                edge_fill(std::integral_constant<int, kF32Vec>{});
            else if (p.e_kind == kBf16Word)
                edge_fill(std::integral_constant<int, kBf16Word>{});
            else
                edge_fill(std::integral_constant<int, kBf16Vec>{});
        }
    } else {

    // Inputs: X = [r_other | T-enc(t) | e] and H = r_self; rows m .. R-1
    // are zero.  Units of 8 columns: X's R * kx / 8 first, then H's; the
    // loads of kFill units per thread are in flight together.
    const uint32_t gx = p.kx / 8, gh = p.kd / 8;
    const uint32_t ux = R * gx;
    const uint32_t ut = ux + R * gh;
    for (uint32_t base = tid; base < ut; base += kRnnThreads * kFill) {
        float v[kFill][8];
#pragma unroll
        for (int f = 0; f < kFill; f++) {
            const uint32_t u = base + f * kRnnThreads;
#pragma unroll
            for (int i = 0; i < 8; i++) v[f][i] = 0.0f;
            if (u >= ut) continue;
            if (u >= ux) {
                const uint32_t j = nlb_div(u - ux, p.gh_m);
                const uint32_t c0 = (u - ux - j * gh) * 8;
                if (j < m) load8(p.st + (size_t)m_self[j] * p.srb, p.d, p.s_bf16, p.s_vec, c0, v[f]);
                continue;
            }
            const uint32_t j = nlb_div(u, p.gx_m);
            const uint32_t c0 = (u - j * gx) * 8;
            if (j >= m) continue;
            const uint32_t link = m_row[j] >> 1;
            if (c0 < p.kd) {
                load8(p.st + (size_t)m_other[j] * p.srb, p.d, p.s_bf16, p.s_vec, c0, v[f]);
            } else if (c0 < p.off_e) {
                const uint32_t k = c0 - p.kd;
                const float tf = (float)p.t[link];
                float wk[8], bk[8];
                if (p.t_vec && k + 8 <= p.d_time) {
                    const f32x4 w0 = *(const f32x4 *)(p.tw + k), w1 = *(const f32x4 *)(p.tw + k + 4);
                    const f32x4 b0 = *(const f32x4 *)(p.tb + k), b1 = *(const f32x4 *)(p.tb + k + 4);
#pragma unroll
                    for (int i = 0; i < 4; i++) {
                        wk[i] = w0[i];
                        wk[4 + i] = w1[i];
                        bk[i] = b0[i];
                        bk[4 + i] = b1[i];
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 8; i++) {
                        wk[i] = k + i < p.d_time ? p.tw[k + i] : 0.0f;
                        bk[i] = k + i < p.d_time ? p.tb[k + i] : 0.0f;
                    }
                }
#pragma unroll
                for (int i = 0; i < 8; i++)
                    if (k + i < p.d_time) v[f][i] = cos_fp32(__builtin_fmaf(wk[i], tf, bk[i]));
            } else {
                const uint64_t e = first_eid + link;
                if (e < (uint64_t)p.edge_rows)
                    load8(p.efeat + (size_t)e * p.erb, p.e_dim, p.e_bf16, p.e_vec, c0 - p.off_e, v[f]);
            }
        }
#pragma unroll
        for (int f = 0; f < kFill; f++) {
            const uint32_t u = base + f * kRnnThreads;
            if (u >= ut) continue;
            if (u >= ux) {
                const uint32_t j = nlb_div(u - ux, p.gh_m);
                const uint32_t c0 = (u - ux - j * gh) * 8;
                if (p.h_lo)
                    store_split8(v[f], Hh + (size_t)j * hs + c0, Hl + (size_t)j * hs + c0);
                else
                    store_hi8(v[f], Hh + (size_t)j * hs + c0);
                continue;
            }
            const uint32_t j = nlb_div(u, p.gx_m);
            const uint32_t c0 = (u - j * gx) * 8;
            if (c0 >= p.lo_begin && c0 < p.lo_end)
                store_split8(v[f], Xh + (size_t)j * xs + c0, Xl + (size_t)j * ls + (c0 - p.lo_begin));
            else
                store_hi8(v[f], Xh + (size_t)j * xs + c0);
        }
    }
    }

}

template <int NB>
__global__ __launch_bounds__(kRnnThreads) void rnn_gru(GruParams p) {
    constexpr uint32_t R = 16 * NB;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    uint32_t *m_row = (uint32_t *)smem;          // pair row of tile row j
    int32_t *m_self = (int32_t *)(m_row + 64);
    int32_t *m_other = m_self + 64;
    float *m_t = (float *)(m_other + 64);        // its link's time, as fp32
    float *s_tw = (float *)(smem + kGruMetaRows), *s_tb = s_tw + ((p.d_time + 31u) & ~31u);
    __bf16 *Xh = (__bf16 *)(smem + p.meta);
    __bf16 *Xl = (__bf16 *)(smem + p.off_xl);
    __bf16 *Hh = (__bf16 *)(smem + p.off_h);
    __bf16 *Hl = (__bf16 *)(smem + p.off_hl);

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63, wave = tid >> 6;
    const uint32_t count = *p.count;
    const uint64_t j0 = (uint64_t)blockIdx.x * R;
    if (j0 >= count) return;
    const uint32_t m = (uint32_t)min((uint64_t)R, (uint64_t)count - j0);
    if (tid < m) {
        const u32x4 e = p.list[j0 + tid];
        m_row[tid] = e[0];
        m_self[tid] = (int32_t)e[1];
        m_other[tid] = (int32_t)e[2];
        m_t[tid] = (float)p.t[e[0] >> 1];
    }
    for (uint32_t u = tid; u < ((p.d_time + 31u) & ~31u); u += kRnnThreads) {
        s_tw[u] = u < p.d_time ? p.tw[u] : 0.0f;
        s_tb[u] = u < p.d_time ? p.tb[u] : 0.0f;
    }
    __syncthreads();

    gru_fill<NB>(p, m, m_row, m_self, m_other, m_t, s_tw, s_tb, Xh, Xl, Hh, Hl, p.xs, p.ls, p.hs);
    __syncthreads();

    const uint32_t d = p.d;
    const uint32_t units = (d + 15) / 16;
    const uint32_t lr = lane & 15, lk = (lane >> 4) * 8;
    for (uint32_t ub = wave; ub < units; ub += kRnnThreads / 64) {
        const uint32_t j = 16 * ub + lr;
        const uint32_t jr = j < d ? j : d - 1;   // rows past d are read, never used
        // The epilogue's h values, loaded before the products so that
        // their latency overlaps them.
        float hv[NB][4];
#pragma unroll
        for (int rb = 0; rb < NB; rb++)
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                const uint8_t *srow = p.st + (size_t)m_self[row < m ? row : 0] * p.srb;
                hv[rb][i] = p.s_bf16 ? bf16_bits_to_float(((const uint16_t *)srow)[jr])
                                     : ((const float *)srow)[jr];
            }
        f32x4 acc[4][NB];   // r, z, input part of n, hidden part of n
#pragma unroll
        for (int g = 0; g < 4; g++)
#pragma unroll
            for (int rb = 0; rb < NB; rb++) acc[g][rb] = f32x4(0.0f);
        const __bf16 *wx = p.w_ih + (size_t)jr * p.kx + lk;
        const size_t gx_step = (size_t)d * p.kx;
        gate_seg<NB, false, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, gx_step, 0, p.lo_begin, lr, lk);
        gate_seg<NB, true, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, gx_step, p.lo_begin, p.lo_end, lr,
                              lk);
        gate_seg<NB, false, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, gx_step, p.lo_end, p.kx, lr, lk);
        const __bf16 *wh = p.w_hh + (size_t)jr * p.kd + lk;
        const size_t gh_step = (size_t)d * p.kd;
        if (p.h_lo)
            gate_seg<NB, true, 3>(acc, Hh, Hl, p.hs, p.hs, 0, wh, gh_step, 0, p.kd, lr, lk);
        else
            gate_seg<NB, false, 3>(acc, Hh, Hl, p.hs, p.hs, 0, wh, gh_step, 0, p.kd, lr, lk);
        if (j >= d) continue;
        const float br = p.b_ih[j] + p.b_hh[j];
        const float bz = p.b_ih[d + j] + p.b_hh[d + j];
        const float bin = p.b_ih[2 * d + j];
        const float bhn = p.b_hh[2 * d + j];
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const uint32_t row = 16u * rb + 4u * (lane >> 4) + i;
                if (row >= m) continue;
                const float rg = sigmoid_f32(acc[0][rb][i] + br);
                const float zg = sigmoid_f32(acc[1][rb][i] + bz);
                const float ng = tanh_f32(acc[2][rb][i] + bin + rg * (acc[3][rb][i] + bhn));
                const float out = (1.0f - zg) * ng + zg * hv[rb][i];
                uint8_t *crow = p.cand + (size_t)m_row[row] * p.srb;
                if (p.s_bf16)
                    ((uint16_t *)crow)[j] = f32_to_bf16_rne(out);
                else
                    ((float *)crow)[j] = out;
            }
        }
    }
}

// Weight-stationary form of the GRU pass, for status rows with a 16-byte
// piece form, kd <= 128, kx + kd <= 32 kWsSteps and a time encoding.  One
// workgroup per CU with kd / 16 wavefronts: wavefront w holds the weight
// fragments of output units 16 w .. 16 w + 15 (all three gates, every
// k-step: 12 registers per k-step) for the whole launch, and the workgroup
// loops over the 32-row tiles blockIdx.x, blockIdx.x + gridDim.x, ...
//
// A tile sits in LDS in matrix-operand order: the A operand of k-step s and
// row block rb is 1 KB, lane l's eight values at 16 l, so that every operand
// read is one contiguous 16-byte read per lane at a fixed offset.  Each
// tile buffer is two LDS arrays (so that the compiler can tell a write of
// one from a read or write of the other): S holds what the status rows
// fill (H hi, X hi of the r_other steps), T the rest (X hi of the
// time-encoding and link-row steps, X lo by step, H lo for fp32 statuses;
// lo planes only at steps inside [lo_begin, lo_end)).  Tiles alternate
// between two buffers: the status rows of the next tile are requested
// before the products of the current one and land in its S array meanwhile
// -- bf16 rows whose width is a multiple of 32 by direct global-to-LDS
// loads (one operand fragment per wavefront and load), other rows through
// registers, written after the products (fp32 ones as hi + lo).
//
// The two wavefronts that share a SIMD (w and w + KH) work in opposite
// order, so that one's vector work overlaps the other's products: the
// second half computes the next tile's time encoding before its products
// (from link times it read one tile ahead), the first half goes straight to
// its products; both then apply the gates.  The new statuses of a tile go
// to an LDS staging area and, after the tile's barrier, to the candidate
// rows in whole 16-byte pieces, so that their stores complete under the
// next tile's products.  List entries are read two tiles ahead into one of
// eight row-list slots.  Rows of a tile past the list's end repeat its last
// entry and are never written out.
constexpr int kWsSteps = 12;
constexpr uint32_t kWsRows = 32;
constexpr int kWsBf16Dma = 0, kWsBf16 = 1, kWsF32 = 2;   // how status rows reach the LDS

template <int KH>
struct WsLayout {
    static constexpr uint32_t NB = kWsRows / 16, KXM = kWsSteps - KH;
    static constexpr uint32_t frag = 1024;   // bytes of one 16 x 32 operand
    // S: X hi steps [0, KH), H hi
    static constexpr uint32_t sx = 0, sh = KH * NB * frag, s_bytes = 2 * KH * NB * frag;
    // T: X hi steps [KH, KXM), X lo steps [0, KXM), H lo
    static constexpr uint32_t tx = 0, tl = (KXM - KH) * NB * frag, th = tl + KXM * NB * frag,
                              t_bytes = th + KH * NB * frag;
    // output rows of a tile, row-major with a stride of the row plus 16
    // bytes against bank conflicts (at most fp32, kd = 32 KH)
    static constexpr uint32_t ostage = kWsRows * (32 * KH * 4 + 16);
    static constexpr uint32_t slots = 8;
    static constexpr uint32_t fixed = 2 * (s_bytes + t_bytes) + 2 * ostage + slots * 1024 + 4 * 32 * KH * 4;
};

// Byte offset of the eight values at row j, columns c .. c + 7 (c % 8 == 0)
// of a tile plane in operand order.
__device__ __forceinline__ uint32_t frag_off(uint32_t j, uint32_t c) {
    return (((c >> 5) * (kWsRows / 16) + (j >> 4)) * 64u + (j & 15u) + 16u * ((c >> 3) & 3u)) * 16u;
}

// A uniform value that the compiler re-reads where it is used (keeps loop
// invariant flags out of long-lived registers).
__device__ __forceinline__ uint32_t opaque_u32(uint32_t x) {
    x = __builtin_amdgcn_readfirstlane(x);
    asm volatile("" : "+s"(x));
    return x;
}

typedef __attribute__((address_space(3))) void *lds_ptr;

// One direct global-to-LDS load of 16 bytes per lane: lane l's bytes from g
// land at LDS byte address lds + 16 l (lds uniform, passed in M0, which the
// compiler sets; the nop is the wait state a load through M0 needs after
// M0 is written).  Written as assembly so that the compiler does not make
// later LDS accesses wait for it (it cannot tell which LDS array such a load
// writes); the caller waits for it (vmcnt) before the workgroup barrier that
// publishes the data.
__device__ __forceinline__ void lds_load16(const void *g, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :: "v"(g), "{m0}"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)(lds_ptr)p; }

template <int KH, int MODE>
__global__ __launch_bounds__(128 * KH) void rnn_gru_ws(GruParams p) {
    using L = WsLayout<KH>;
    constexpr uint32_t NB = L::NB, R = kWsRows, T = 128 * KH, GH = 4 * KH, FB = L::frag;
    constexpr int KXM = (int)L::KXM, KS = KXM + KH;
    constexpr int SK = MODE == kWsF32 ? kF32Vec : kBf16Vec;
    static_assert(R * GH == T, "one status piece of each input half per thread");
    static_assert(2 * KH == KH * NB, "one operand fragment of each input half per wavefront");
    __shared__ __attribute__((aligned(16))) uint8_t bs0[L::s_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bs1[L::s_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bt0[L::t_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bt1[L::t_bytes];
    constexpr uint32_t OSTR = 32 * KH * (MODE == kWsF32 ? 4 : 2) + 16;   // staging row stride
    __shared__ __attribute__((aligned(16))) uint8_t ost0[R * OSTR];
    __shared__ __attribute__((aligned(16))) uint8_t ost1[R * OSTR];
    // Row lists {pair row, self, other, 0} of 1 KB slots (R entries and room
    // for the duplicates a direct load of R entries writes); tile i in slot i % 8.
    constexpr uint32_t MS = 64;
    __shared__ __attribute__((aligned(16))) u32x4 meta[L::slots * MS];
    extern __shared__ __attribute__((aligned(16))) float s_tw[];   // T-enc w | b, pad32(d_time) each
    float *s_tb = s_tw + ((p.d_time + 31u) & ~31u);

    const uint32_t tid = threadIdx.x, lane = tid & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint64_t first_eid = first_eid_of(p);
    const bool second = wave >= (uint32_t)KH;   // shares its SIMD with wavefront wave - KH
    const uint32_t lr = lane & 15, lk = (lane >> 4) * 8;
    const uint32_t count = *p.count;
    const uint32_t tiles = (uint32_t)(((uint64_t)count + R - 1) / R);
    if (blockIdx.x >= tiles) return;
    const uint32_t d = p.d, kx_steps = p.kx / 32;
    const bool mma = wave < (d + 15) / 16;
    const uint32_t j = 16 * wave + lr, jr = j < d ? j : d - 1;
    const uint32_t gt = (p.off_e - p.kd) / 8, tu = R * gt;

    // This wavefront's weight fragments (loaded in the prologue, after the
    // first tile's requests) and the gate biases by output unit (LDS, read
    // per tile).
    bf16x8 bx[KXM][3], bh[KH][3];
    __shared__ float sbias[4][32 * KH];

    auto list_at = [&](uint32_t tl, uint32_t row) __attribute__((always_inline)) {
        return min((uint64_t)tl * R + row, (uint64_t)count - 1);
    };

    // Register path: a thread's status pieces, f = 0 of H (self) and f = 1
    // of X's r_other, both at tile row pj, columns pc0 .. pc0 + 7.  Direct
    // path: wavefront w's operand fragment w of H and of X's r_other, lane l
    // at tile row dj, column dc.
    const uint32_t pj = tid / GH, pc0 = 8 * (tid % GH);
    const uint32_t dj = 16 * (wave % NB) + lr, dc = 32 * (wave / NB) + lk;
    Piece8<SK> pc[2];
    auto request_tile = [&](uint8_t *nbS, uint32_t slot) __attribute__((always_inline)) {
        if constexpr (MODE == kWsBf16Dma) {
            const u32x4 e = meta[slot * MS + dj];
            lds_load16(p.st + (size_t)e[1] * p.srb + 2u * dc, lds_addr(nbS + L::sh + wave * FB));
            lds_load16(p.st + (size_t)e[2] * p.srb + 2u * dc, lds_addr(nbS + L::sx + wave * FB));
        } else {
            const u32x4 e = meta[slot * MS + pj];
            load_piece<SK>(p.st + (size_t)e[1] * p.srb, d, pc0, pc[0]);
            load_piece<SK>(p.st + (size_t)e[2] * p.srb, d, pc0, pc[1]);
        }
    };

    // Time-encoding unit u of a tile: row u / gt, encoding columns k .. k + 7
    // (X columns kd + k ..), from the row's link time tf.
    // Time-encoding unit u of a tile: lane l = u % 64 of operand fragment
    // f = u / 64 of the encoding's steps (step f / NB, row block f % NB), i.e.
    // tile row 16 (f % NB) + l % 16 and encoding columns 32 (f / NB) +
    // 8 (l / 16) .. + 7, so that its eight values sit at byte 16 u of their
    // plane (a wavefront's writes are contiguous).  Arguments beyond the fast
    // cosine's range are rare: their units are redone, exactly, only where a
    // wavefront meets one.
    auto unit_row = [](uint32_t u) { return 16u * ((u >> 6) % NB) + (u & 15u); };
    auto unit_col = [](uint32_t u) { return 32u * ((u >> 6) / NB) + 8u * ((u >> 4) & 3u); };
    auto tenc_unit = [&](uint8_t *nbT, uint32_t u, float tf) __attribute__((always_inline)) {
        const uint32_t k = unit_col(u);
        // two halves of four values (fewer registers live at once)
#pragma unroll
        for (int h = 0; h < 2; h++) {
            const f32x4 w = *(const f32x4 *)(s_tw + k + 4 * h), b = *(const f32x4 *)(s_tb + k + 4 * h);
            float x[4], v[4];
            bool wide = false;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                x[e] = __builtin_fmaf(w[e], tf, b[e]);
                v[e] = cos_fp32_small(x[e]);
                wide |= !(__builtin_fabsf(x[e]) < kCosFastLimit);
            }
            if (__builtin_expect(__ballot(wide) != 0, 0)) {
#pragma unroll
                for (int e = 0; e < 4; e++)
                    if (!(__builtin_fabsf(x[e]) < kCosFastLimit)) v[e] = cos_fp32_exact_wide(x[e]);
            }
            u32x2 hi, lo;
#pragma unroll
            for (int e = 0; e < 4; e += 2) {
                float a0 = k + 4 * h + e < p.d_time ? v[e] : 0.0f, a1 = k + 4 * h + e + 1 < p.d_time ? v[e + 1] : 0.0f;
                const __bf16 h0 = (__bf16)a0, h1 = (__bf16)a1;
                const __bf16 l0 = (__bf16)(a0 - (float)h0), l1 = (__bf16)(a1 - (float)h1);
                hi[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
                lo[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
            }
            *(u32x2 *)(nbT + L::tx + 16u * u + 8u * h) = hi;
            *(u32x2 *)(nbT + L::tl + KH * NB * FB + 16u * u + 8u * h) = lo;
        }
    };
    // A thread's time-encoding unit u = tid of every tile (if u < tu), with
    // the link time of its row for the tile whose encoding it computes next.
    uint32_t tB = 0;
    auto t_row = [&](uint32_t tl, uint32_t u) __attribute__((always_inline)) {
        return ((const uint32_t *)p.list)[4 * list_at(tl, unit_row(min(u, tu - 1u)))];
    };

    // What is written after the products: status pieces on the register
    // path, time-encoding units the second half does not cover (u >= T) and
    // link rows.
    auto write_tile = [&](uint8_t *nbS, uint8_t *nbT, uint32_t slot) __attribute__((always_inline)) {
        const uint32_t po = frag_off(pj, pc0);
        if constexpr (MODE == kWsF32) {
            float v[8];
            piece_floats<SK>(pc[0], d, pc0, true, v);
            store_split8(v, (__bf16 *)(nbS + L::sh + po), (__bf16 *)(nbT + L::th + po));
            piece_floats<SK>(pc[1], d, pc0, true, v);
            store_split8(v, (__bf16 *)(nbS + L::sx + po), (__bf16 *)(nbT + L::tl + po));   // lo_begin == 0
        } else if constexpr (MODE == kWsBf16) {
            *(u32x4 *)(nbS + L::sh + po) = piece_bf16_bits<SK>(pc[0], d, pc0, true);
            *(u32x4 *)(nbS + L::sx + po) = piece_bf16_bits<SK>(pc[1], d, pc0, true);
        }
        for (uint32_t u = tid + T; u < tu; u += T)
            tenc_unit(nbT, u, (float)p.t[meta[slot * MS + unit_row(u)][0] >> 1]);
        if (p.kx > p.off_e) {
            const uint32_t ge = (p.kx - p.off_e) / 8;
            auto edge_fill = [&](auto kind) __attribute__((always_inline)) {
                constexpr int K = decltype(kind)::value;
                auto eid_of = [&](uint32_t jj) __attribute__((always_inline)) {
                    return first_eid + (meta[slot * MS + jj][0] >> 1);
                };
                fill_seg<K, 4, T>(
                    R * ge, ge, p.ge_m, p.e_dim,
                    [&](uint32_t jj) __attribute__((always_inline)) {
                        const uint64_t e = eid_of(jj);
                        return p.efeat + (size_t)(e < (uint64_t)p.edge_rows ? e : 0u) * p.erb;
                    },
                    [&](uint32_t jj, uint32_t c0, const Piece8<K> &q) __attribute__((always_inline)) {
                        const bool ok = eid_of(jj) < (uint64_t)p.edge_rows;
                        const uint32_t c = p.off_e + c0;
                        __bf16 *hi = (__bf16 *)(nbT + L::tx + frag_off(jj, c - p.kd));
                        if constexpr (K == kF32Vec) {
                            float v[8];
                            piece_floats<K>(q, p.e_dim, c0, ok, v);
                            store_split8(v, hi, (__bf16 *)(nbT + L::tl + frag_off(jj, c)));
                        } else {
                            *(u32x4 *)hi = piece_bf16_bits<K>(q, p.e_dim, c0, ok);
                        }
                    });
            };
            if (p.e_kind == kF32Vec)
                edge_fill(std::integral_constant<int, kF32Vec>{});
            else if (p.e_kind == kBf16Word)
                edge_fill(std::integral_constant<int, kBf16Word>{});
            else
                edge_fill(std::integral_constant<int, kBf16Vec>{});
        }
    };
    // Direct loads into LDS count as outstanding vector-memory operations:
    // all of this wavefront's must have landed before the workgroup barrier
    // (the compiler does not know of them).
    auto tile_barrier = [&]() __attribute__((always_inline)) {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0), seen by the compiler's own wait tracking
        __syncthreads();
    };

    // Prologue, ordered so that the weights' transfer (about 300 KB per CU,
    // from L2) overlaps the first tile's dependent loads: time-encoding
    // parameters, row lists of the first two tiles and the list rows of the
    // second tile's encoding units; then the first tile's status rows and
    // the link times of both tiles' encoding units; then the weights and
    // biases; then the first tile's encoding and barrier.
    for (uint32_t u = tid; u < ((p.d_time + 31u) & ~31u); u += T) {
        s_tw[u] = u < p.d_time ? p.tw[u] : 0.0f;
        s_tb[u] = u < p.d_time ? p.tb[u] : 0.0f;
    }
    const uint32_t stride = gridDim.x;
    uint32_t tl = blockIdx.x;
    {
        const uint32_t t1 = tl + stride < tiles ? tl + stride : tl;
        const u32x4 e0 = p.list[list_at(tl, tid & (R - 1))], e1 = p.list[list_at(t1, tid & (R - 1))];
        const uint32_t r1 = t_row(t1, tid);
        if (tid < R) {
            meta[tid] = e0;
            meta[MS + tid] = e1;
        }
        tB = r1;
    }
    __syncthreads();
    request_tile(bs0, 0);
    const uint32_t t_first = p.t[meta[unit_row(min(tid, tu - 1u))][0] >> 1];
    tB = p.t[tB >> 1];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s < KXM; s++)
#pragma unroll
        for (int g = 0; g < 3; g++)
            bx[s][g] = *(const bf16x8 *)(p.w_ih + ((size_t)g * d + jr) * p.kx +
                                         32u * min((uint32_t)s, kx_steps - 1u) + lk);
#pragma unroll
    for (int s = 0; s < KH; s++)
#pragma unroll
        for (int g = 0; g < 3; g++)
            bh[s][g] = *(const bf16x8 *)(p.w_hh + ((size_t)g * d + jr) * p.kd + 32 * s + lk);
    if (lane < 16 && mma) {
        // r and z biases pre-scaled for the base-2 exponential, then the
        // input and hidden biases of n
        sbias[0][j] = -kLog2e * (p.b_ih[jr] + p.b_hh[jr]);
        sbias[1][j] = -kLog2e * (p.b_ih[d + jr] + p.b_hh[d + jr]);
        sbias[2][j] = p.b_ih[2 * d + jr];
        sbias[3][j] = p.b_hh[2 * d + jr];
    }
    write_tile(bs0, bt0, 0);
    if (tid < tu) tenc_unit(bt0, tid, (float)t_first);
    tile_barrier();

    // Candidate rows of tile tlp (row-list slot `slot`) from its staging
    // area, 16 bytes per thread and step.
    auto copy_out = [&](const uint8_t *ob, uint32_t slot, uint32_t tlp) __attribute__((always_inline)) {
        constexpr uint32_t CO = MODE == kWsF32 ? 2 : 1;   // >= R * (kd * element size / 16) / T
        const uint32_t cpr = p.srb / 16, units = min(R, count - tlp * R) * cpr;
#pragma unroll
        for (uint32_t k = 0; k < CO; k++) {
            const uint32_t u = tid + k * T;
            if (u < units) {
                const uint32_t row = nlb_div(u, p.ws_cpr_m), c = 16u * (u - row * cpr);
                const u32x4 v = *(const u32x4 *)(ob + row * OSTR + c);
                *(u32x4 *)(p.cand + (size_t)meta[slot * MS + row][0] * p.srb + c) = v;
            }
        }
    };

    // One tile: products from (cbS, cbT) (row-list slot i % 8) while the
    // next tile arrives in (nbS, nbT); new statuses to ob, those of the
    // previous tile out of obp; false after the workgroup's last tile.
    auto tile = [&](uint8_t *cbS, uint8_t *cbT, uint8_t *nbS, uint8_t *nbT, uint8_t *ob, const uint8_t *obp,
                    uint32_t i) __attribute__((always_inline)) {
        const uint32_t ms = i & 7, ns = (i + 1) & 7;
        const bool has_next = tl + stride < tiles, has_nn = tl + 2 * stride < tiles;
        const uint32_t tnn = has_nn ? tl + 2 * stride : tl;
        // Row list of the tile two strides on (straight into its slot; the
        // list rows of the threads' encoding units too) and status rows of the
        // next tile (re-reads of the current tile's when there is none: in
        // bounds, unused).
        if (has_nn && wave == 0)
            lds_load16(p.list + list_at(tnn, lane & (R - 1)), lds_addr(meta + ((i + 2) & 7) * MS));
        const uint32_t rB = t_row(tnn, tid);
        if (MODE != kWsBf16Dma || has_next) request_tile(nbS, has_next ? ns : ms);
        if (i > 0) copy_out(obp, (i - 1) & 7, tl - stride);
        // The second half encodes its units of the next tile now, the first
        // half after its products.
        const float tf = (float)tB;
        if (second && has_next && tid < tu) tenc_unit(nbT, tid, tf);
        f32x4 acc[4][NB];   // r, z, input part of n, hidden part of n
        if (mma) {
            const uint32_t lm = opaque_u32(p.ws_lomask), ks = opaque_u32(kx_steps);
            const uint8_t *bS = cbS + 16u * lane, *bT = cbT + 16u * lane;
#pragma unroll
            for (int g = 0; g < 4; g++)
#pragma unroll
                for (int rb = 0; rb < NB; rb++) acc[g][rb] = f32x4(0.0f);
            auto mfma3 = [&](const bf16x8 (&a)[NB], const bf16x8 (&w)[3], int nidx) __attribute__((always_inline)) {
#pragma unroll
                for (int rb = 0; rb < NB; rb++)
#pragma unroll
                    for (int g = 0; g < 3; g++) {
                        const int gi = g == 2 ? nidx : g;
                        acc[gi][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[rb], w[g], acc[gi][rb], 0, 0, 0);
                    }
            };
            // Operands of step s (X steps, then H steps): the hi plane
            // always, the lo plane where the step has one; those of step
            // s + 1 are read before the products of step s.
            auto load_step = [&](int s, bf16x8 (&a)[NB], bf16x8 (&al)[NB]) __attribute__((always_inline)) {
                const uint8_t *hi = s < KH ? bS + L::sx + s * NB * FB
                                  : s < KXM ? bT + L::tx + (s - KH) * NB * FB : bS + L::sh + (s - KXM) * NB * FB;
                const uint8_t *lo = s < KXM ? bT + L::tl + s * NB * FB : bT + L::th + (s - KXM) * NB * FB;
#pragma unroll
                for (int rb = 0; rb < NB; rb++) a[rb] = *(const bf16x8 *)(hi + rb * FB);
                if (s < KXM ? ((lm >> s) & 1u) != 0 : MODE == kWsF32) {
#pragma unroll
                    for (int rb = 0; rb < NB; rb++) al[rb] = *(const bf16x8 *)(lo + rb * FB);
                }
            };
            bf16x8 a[2][NB], al[NB];
            load_step(0, a[0], al);
#pragma unroll
            for (int s = 0; s < KS; s++) {
                bf16x8 nal[NB];
                if (s + 1 < KS) load_step(s + 1, a[(s + 1) & 1], nal);
                if (s < KXM) {
                    if ((uint32_t)s < ks) mfma3(a[s & 1], bx[s], 2);
                    if ((lm >> s) & 1u) mfma3(al, bx[s], 2);
                } else {
                    mfma3(a[s & 1], bh[s - KXM], 3);
                    if constexpr (MODE == kWsF32) mfma3(al, bh[s - KXM], 3);
                }
#pragma unroll
                for (int rb = 0; rb < NB; rb++) al[rb] = nal[rb];
            }
        }
        // Link times of the second half's next units, read while the gates
        // are applied (kept after the products: their addresses come from
        // loads issued with the direct ones, which a wait here would cover).
        __builtin_amdgcn_sched_barrier(0);
        tB = p.t[rB >> 1];
        if (mma) {
            float hv[NB][4];
#pragma unroll
            for (int rb = 0; rb < NB; rb++)
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const uint32_t row = 16u * rb + 4u * (lane >> 4) + q;
                    if constexpr (MODE == kWsF32)
                        hv[rb][q] = ((const float *)(p.st + (size_t)meta[ms * MS + row][1] * p.srb))[jr];
                    else
                        hv[rb][q] = (float)*(const __bf16 *)(cbS + L::sh + frag_off(row, jr & ~7u) + 2u * (jr & 7u));
                }
            if (j < d) {
                const float nbr = sbias[0][j], nbz = sbias[1][j], bin = sbias[2][j], bhn = sbias[3][j];
#pragma unroll
                for (int rb = 0; rb < NB; rb++)
#pragma unroll
                    for (int q = 0; q < 4; q++) {
                        const uint32_t row = 16u * rb + 4u * (lane >> 4) + q;
                        const float rg = __builtin_amdgcn_rcpf(
                            1.0f + __builtin_amdgcn_exp2f(__builtin_fmaf(acc[0][rb][q], -kLog2e, nbr)));
                        const float zg = __builtin_amdgcn_rcpf(
                            1.0f + __builtin_amdgcn_exp2f(__builtin_fmaf(acc[1][rb][q], -kLog2e, nbz)));
                        const float ng = tanh_f32(__builtin_fmaf(rg, acc[3][rb][q] + bhn, acc[2][rb][q] + bin));
                        const float out = __builtin_fmaf(zg, hv[rb][q] - ng, ng);   // (1 - z) n + z h
                        if constexpr (MODE == kWsF32)
                            ((float *)(ob + row * OSTR))[j] = out;
                        else
                            ((__bf16 *)(ob + row * OSTR))[j] = (__bf16)out;   // round to nearest even
                    }
            }
        }
        if (!second && has_next && tid < tu) tenc_unit(nbT, tid, tf);
        if (has_next) write_tile(nbS, nbT, ns);
        tile_barrier();
        tl += stride;
        return has_next;
    };
    for (uint32_t i = 0;; i += 2) {
        if (!tile(bs0, bt0, bs1, bt1, ost0, ost1, i)) {
            copy_out(ost0, i & 7, tl - stride);
            break;
        }
        if (!tile(bs1, bt1, bs0, bt0, ost1, ost0, i + 1)) {
            copy_out(ost1, (i + 1) & 7, tl - stride);
            break;
        }
    }
}

// Status rows of the winners: for each listed winner {pair row r, node},
// candidate row r -> status row node, in units of `w` bytes (upr units per
// row), and winner[node] = 0.  A wavefront pass copies 64 >> lg rows
// (lg = ceil(log2 upr) <= 6), or one row in passes of 64 units; wavefronts
// stride over the list.
__global__ __launch_bounds__(kRnnThreads) void rnn_scatter(const uint8_t *cand, const u32x4 *list,
                                                          const uint32_t *count, uint8_t *st, uint32_t srb,
                                                          uint32_t w, uint32_t upr, uint32_t lg,
                                                          unsigned long long *winner) {
    const uint32_t n = *count, lane = threadIdx.x & 63;
    const uint64_t gw = ((uint64_t)blockIdx.x * kRnnThreads + threadIdx.x) >> 6;
    const uint64_t nw = ((uint64_t)gridDim.x * kRnnThreads) >> 6;
    auto copy = [&](uint64_t k, uint32_t c) {
        const u32x4 e = list[k];
        const uint8_t *from = cand + (size_t)e[0] * srb + c * w;
        uint8_t *to = st + (size_t)e[1] * srb + c * w;
        if (w == 16)
            *(u32x4 *)to = *(const u32x4 *)from;
        else if (w == 8)
            *(u32x2 *)to = *(const u32x2 *)from;
        else if (w == 4)
            *(uint32_t *)to = *(const uint32_t *)from;
        else
            *(uint16_t *)to = *(const uint16_t *)from;
        if (c == 0) winner[e[1]] = 0ull;
    };
    if (lg <= 6) {
        const uint32_t per = 64u >> lg, c = lane & ((1u << lg) - 1u);
        for (uint64_t k = gw * per + (lane >> lg); k < n; k += nw * per)
            if (c < upr) copy(k, c);
    } else {
        for (uint64_t k = gw; k < n; k += nw)
            for (uint32_t c = lane; c < upr; c += 64) copy(k, c);
    }
}

// Zero fill of a winner array (the static one of the allocation-free call).
__global__ __launch_bounds__(kRnnThreads) void rnn_clear(unsigned long long *a, uint64_t n) {
    for (uint64_t i = (uint64_t)blockIdx.x * kRnnThreads + threadIdx.x; i < n;
         i += (uint64_t)gridDim.x * kRnnThreads)
        a[i] = 0ull;
}

// LDS layout of a tile of `rows` pair rows; returns its size in bytes.
uint32_t gru_layout(GruParams &p, uint32_t rows) {
    p.rows = rows;
    p.off_xl = align16(p.meta + rows * p.xs * 2u);
    p.off_h = align16(p.off_xl + (p.lo_end > p.lo_begin ? rows * p.ls * 2u : 0u));
    p.off_hl = align16(p.off_h + rows * p.hs * 2u);
    return p.off_hl + (p.h_lo ? rows * p.hs * 2u : 0u);
}

// Per-table working memory of the update, grown on demand.
int rnn_reserve(nlb_table *h, uint64_t pair_rows, uint32_t srb) {
    if (!h->rnn_winner) {
        const size_t bytes = (size_t)h->num_nodes * 8u;
        if (hipMalloc((void **)&h->rnn_winner, bytes) != hipSuccess) {
            (void)hipGetLastError();
            h->rnn_winner = nullptr;
            return NLB_ENOMEM;
        }
        if (hipMemset(h->rnn_winner, 0, bytes) != hipSuccess) return NLB_EDEVICE;
    }
    const size_t cbytes = (size_t)pair_rows * srb;
    if (cbytes > h->rnn_cand_bytes || pair_rows > h->rnn_cand_rows) {
        // Earlier updates may still read the old buffers.
        if (hipDeviceSynchronize() != hipSuccess) return NLB_EDEVICE;
        (void)hipFree(h->rnn_cand);
        (void)hipFree(h->rnn_list);
        h->rnn_cand = nullptr;
        h->rnn_list = nullptr;
        h->rnn_cand_bytes = 0;
        h->rnn_cand_rows = 0;
        // list: the winner count in word 0, the winners (4 words each) from word 64 on
        if (hipMalloc((void **)&h->rnn_cand, cbytes) != hipSuccess ||
            hipMalloc((void **)&h->rnn_list, ((size_t)pair_rows * 4u + 64u) * 4u) != hipSuccess) {
            (void)hipGetLastError();
            (void)hipFree(h->rnn_cand);
            h->rnn_cand = nullptr;
            h->rnn_list = nullptr;
            return NLB_ENOMEM;
        }
        h->rnn_cand_bytes = cbytes;
        h->rnn_cand_rows = pair_rows;
    }
    return NLB_OK;
}

// Working memory of one update: the winner word of every node (all zero
// between calls), the winner count and list, and the candidate rows.
struct RnnWork {
    unsigned long long *winner;
    bool clear_winner;    // zero winner[0 .. N) first (memory shared with other calls)
    uint8_t *cand;
    uint32_t *list;       // word 0: winner count; from word 64: the winners, 4 words each
};

// Working memory of the table, grown on demand (nlb_rnn_update).
int table_work(nlb_table *h, uint64_t pairs, uint32_t srb, RnnWork *wk) {
    const int rc = rnn_reserve(h, pairs, srb);
    if (rc != NLB_OK) return rc;
    *wk = {h->rnn_winner, false, h->rnn_cand, h->rnn_list};
    return NLB_OK;
}

// ---------------------------------------------------------------- static working memory
// nlb_rnn_update_noalloc works in this array instead of memory of the
// table's: every call on a device shares that device's copy (it keeps the
// last call's contents, and calls that overlap on one device race).  Each
// device holds its own copy at its own address, which hipGetSymbolAddress
// returns with that device current; host code uses only those addresses
// (the array's name on the host is not a device address).
constexpr size_t kScratchBytes = NLB_NOALLOC_SCRATCH;
__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kScratchDevices = 64;
std::mutex g_scratch_mutex;
uint8_t *g_scratch_addr[kScratchDevices];

// Device address of `scratch` on `dev` (the current device), looked up on
// the first call for that device.
int scratch_address(int dev, uint8_t **out) {
    if (dev < 0 || dev >= kScratchDevices) return NLB_EDEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_addr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            (void)hipGetLastError();
            return NLB_EDEVICE;
        }
        g_scratch_addr[dev] = (uint8_t *)ptr;
    }
    *out = g_scratch_addr[dev];
    return NLB_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// The update's working memory carved from `scratch`: winner words of all N
// nodes, the list, the candidate rows.  The winner words are cleared by a
// fill kernel at the start of every call.
int scratch_work(nlb_table *h, uint64_t pairs, uint32_t srb, RnnWork *wk) {
    const size_t winner_bytes = align256((size_t)h->num_nodes * 8u);
    const size_t list_bytes = align256(((size_t)pairs * 4u + 64u) * 4u);
    const size_t cand_bytes = (size_t)pairs * srb;
    if (winner_bytes + list_bytes + cand_bytes > kScratchBytes) return NLB_ESCRATCH;
    uint8_t *base = nullptr;
    const int rc = scratch_address(h->device, &base);
    if (rc != NLB_OK) return rc;
    *wk = {(unsigned long long *)base, true, base + winner_bytes + list_bytes, (uint32_t *)(base + winner_bytes)};
    return NLB_OK;
}

}  // namespace

// Both entry points: argument checks, the GRU form and tile shape, the
// working memory (the table's own, grown on demand, or the static array),
// then the four launches.
static int rnn_update(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t, uint32_t n,
                      uint64_t first_eid, const nlb_gru_weights *wts, void *status, void *stream,
                      bool use_scratch) {
    if (!h || !wts) return NLB_EINVAL;
    if (n == 0) return NLB_OK;
    if (!src || !dst || !t || !status) return NLB_EINVAL;
    if (n >= (1u << 31)) return NLB_EINVAL;
    const int32_t sd = wts->status_dtype, ed = wts->edge_dtype;
    if ((sd != NLB_DTYPE_F32 && sd != NLB_DTYPE_BF16) || (ed != NLB_DTYPE_F32 && ed != NLB_DTYPE_BF16))
        return NLB_EINVAL;
    if (wts->status_dim < 1 || wts->status_dim > NLB_RNN_MAX_DIM) return NLB_EINVAL;
    if (!wts->w_ih || !wts->w_hh || !wts->b_ih || !wts->b_hh) return NLB_EINVAL;
    if (((uintptr_t)wts->w_ih | (uintptr_t)wts->w_hh) % 16 || ((uintptr_t)wts->b_ih | (uintptr_t)wts->b_hh) % 4)
        return NLB_EINVAL;
    const uint32_t s_es = sd == NLB_DTYPE_BF16 ? 2 : 4, e_es = ed == NLB_DTYPE_BF16 ? 2 : 4;
    if ((uintptr_t)status % s_es || h->erb % e_es) return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;

    GruParams p;
    std::memset(&p, 0, sizeof(p));
    p.src = src;
    p.dst = dst;
    p.t = t;
    p.n = n;
    p.num_nodes = h->num_nodes;
    p.first_eid = first_eid;
    p.table_status = h->status;
    p.d = (uint32_t)wts->status_dim;
    p.d_time = h->d_time;
    p.tw = h->w;
    p.tb = h->b;
    p.t_vec = ((uintptr_t)h->w | (uintptr_t)h->b) % 16 == 0;
    p.efeat = h->efeat;
    p.edge_rows = h->edge_rows;
    p.e_dim = h->erb / e_es;
    p.e_bf16 = ed == NLB_DTYPE_BF16;
    p.erb = h->erb;
    p.e_vec = h->erb % 16 == 0 && (uintptr_t)h->efeat % 16 == 0;
    p.st = (const uint8_t *)status;
    p.s_bf16 = sd == NLB_DTYPE_BF16;
    p.srb = p.d * s_es;
    p.s_vec = p.srb % 16 == 0 && (uintptr_t)status % 16 == 0;
    p.kd = pad32(p.d);
    p.off_e = p.kd + pad32(p.d_time);
    p.kx = p.off_e + pad32(p.e_dim);
    // Columns whose values are not bf16 already: fp32 statuses, the time
    // encoding, fp32 link rows.  They form one range because the time
    // encoding sits between the other two segments.
    const bool lo_s = !p.s_bf16, lo_t = p.d_time > 0, lo_e = p.e_dim > 0 && !p.e_bf16;
    p.lo_begin = lo_s ? 0 : (lo_t ? p.kd : (lo_e ? p.off_e : 0));
    p.lo_end = lo_e ? p.kx : (lo_t ? p.off_e : (lo_s ? p.kd : 0));
    p.h_lo = lo_s;
    p.xs = p.kx + 8;
    p.ls = (p.lo_end - p.lo_begin) + 8;
    p.hs = p.kd + 8;
    p.gx_m = nlb_div_magic(p.kx / 8);
    p.gh_m = nlb_div_magic(p.kd / 8);
    p.gt_m = p.off_e > p.kd ? nlb_div_magic((p.off_e - p.kd) / 8) : 0;
    p.ge_m = p.kx > p.off_e ? nlb_div_magic((p.kx - p.off_e) / 8) : 0;
    p.s_kind = piece_kind(p.srb, status, p.s_bf16);
    p.e_kind = h->efeat ? piece_kind(h->erb, h->efeat, p.e_bf16) : -1;
    p.meta = align16(kGruMetaRows + 8u * pad32(p.d_time));
    p.w_ih = (const __bf16 *)wts->w_ih;
    p.w_hh = (const __bf16 *)wts->w_hh;
    p.b_ih = wts->b_ih;
    p.b_hh = wts->b_hh;

    // Weight-stationary form when its weight fragments fit the registers and
    // its two tile buffers the LDS; else tiles of 16 * nb listed rows: as
    // large as the LDS budget of two workgroups per CU allows, smaller when
    // the batch would give fewer than kGruTargetTiles tiles (counting all 2n
    // pair rows; the winners are fewer); a 16-row tile may use a workgroup's
    // whole LDS.
    const uint64_t pairs = 2ull * n;
    const uint32_t kh = p.kd / 32;
    // Forms whose registers fit without spills: bf16 rows of a width that is
    // a multiple of 32 (direct loads into LDS) up to kd = 128, other 16-byte
    // rows up to kd = 64.
    const int ws_mode = p.s_kind == kF32Vec ? kWsF32 : (p.d % 32 == 0 ? kWsBf16Dma : kWsBf16);
    bool ws = (p.s_kind == kBf16Vec || p.s_kind == kF32Vec) && kh <= (ws_mode == kWsBf16Dma ? 4u : 2u) &&
              p.kx / 32 + kh <= (uint32_t)kWsSteps && p.d_time > 0 && (p.kx == p.off_e || p.e_kind >= 0);
    uint32_t lds = 0, nb = 4;
    int cus = 0;
    if (ws) {
        // static LDS: tile buffers, staging areas, row-list slots; dynamic: T-enc w | b
        const uint32_t fixed = kh == 1 ? WsLayout<1>::fixed : kh == 2 ? WsLayout<2>::fixed
                             : kh == 3 ? WsLayout<3>::fixed : WsLayout<4>::fixed;
        lds = 8u * pad32(p.d_time);
        p.ws_cpr_m = nlb_div_magic(p.srb / 16);
        ws = fixed + lds <= kGruLdsMax &&
             hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device) == hipSuccess && cus > 0;
        for (uint32_t st = p.lo_begin / 32; st < p.lo_end / 32; st++) p.ws_lomask |= 1u << st;
    }
    if (!ws) {
        while (nb > 1 && pairs < (uint64_t)kGruTargetTiles * 16u * nb) nb /= 2;
        for (;; nb /= 2) {
            GruParams trial = p;
            lds = gru_layout(trial, 16u * nb);
            if (lds <= (nb == 1 ? kGruLdsMax : kGruLdsBudget)) break;
            if (nb == 1) return NLB_EINVAL;   // one 16-row tile does not fit the LDS
        }
        gru_layout(p, 16u * nb);
    }

    RnnWork wk;
    const int rc = use_scratch ? scratch_work(h, pairs, p.srb, &wk)
                               : table_work(h, pairs, p.srb, &wk);
    if (rc != NLB_OK) return rc;
    if (wk.clear_winner) {
        const uint64_t blocks = std::min<uint64_t>(4096, ((uint64_t)h->num_nodes + kRnnThreads - 1) / kRnnThreads);
        hipLaunchKernelGGL(rnn_clear, dim3((unsigned)blocks), dim3(kRnnThreads), 0, (hipStream_t)stream,
                           wk.winner, (uint64_t)h->num_nodes);
    }
    uint32_t *count = wk.list;
    u32x4 *list = (u32x4 *)(wk.list + 64);
    p.list = list;
    p.count = count;
    p.cand = wk.cand;

    ResolveParams rp = {src, dst, n, h->num_nodes, wk.winner, h->status, count};
    if (n >= kMergeMinBatch)
        hipLaunchKernelGGL(rnn_resolve_merged, dim3((n + kResolveLinks - 1) / kResolveLinks),
                           dim3(kMergeThreads), 0, (hipStream_t)stream, rp);
    else
        hipLaunchKernelGGL(rnn_resolve, dim3((n + kRnnThreads - 1) / kRnnThreads), dim3(kRnnThreads), 0,
                           (hipStream_t)stream, rp);
    SelectParams sp = {src, dst, n, h->num_nodes, wk.winner, list, count};
    hipLaunchKernelGGL(rnn_select, dim3((unsigned)((pairs + kSelectRows - 1) / kSelectRows)),
                       dim3(kRnnThreads), 0, (hipStream_t)stream, sp);
    if (ws) {
        const void *kern = nullptr;
        switch (kh * 4 + ws_mode) {
#define NLB_WS_CASE(KH, MODE) \
        case KH * 4 + MODE: kern = (const void *)rnn_gru_ws<KH, MODE>; break;
        NLB_WS_CASE(1, kWsBf16Dma) NLB_WS_CASE(1, kWsBf16) NLB_WS_CASE(1, kWsF32)
        NLB_WS_CASE(2, kWsBf16Dma) NLB_WS_CASE(2, kWsBf16) NLB_WS_CASE(2, kWsF32)
        NLB_WS_CASE(3, kWsBf16Dma) NLB_WS_CASE(4, kWsBf16Dma)
#undef NLB_WS_CASE
        default: return NLB_EINVAL;
        }
        const uint64_t tiles = (pairs + 31) / 32;
        const dim3 grid((unsigned)std::min<uint64_t>(tiles, (uint64_t)cus));
        void *args[] = {&p};
        if (hipLaunchKernel(kern, grid, dim3(128u * kh), args, lds, (hipStream_t)stream) != hipSuccess)
            return NLB_EDEVICE;
    } else {
        const void *kern = nb == 4 ? (const void *)rnn_gru<4>
                         : nb == 2 ? (const void *)rnn_gru<2> : (const void *)rnn_gru<1>;
        if (lds > 64u * 1024u &&
            hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGruLdsMax) != hipSuccess)
            return NLB_EDEVICE;
        const dim3 grid((unsigned)((pairs + 16u * nb - 1) / (16u * nb)));
        if (nb == 4)
            hipLaunchKernelGGL(rnn_gru<4>, grid, dim3(kRnnThreads), lds, (hipStream_t)stream, p);
        else if (nb == 2)
            hipLaunchKernelGGL(rnn_gru<2>, grid, dim3(kRnnThreads), lds, (hipStream_t)stream, p);
        else
            hipLaunchKernelGGL(rnn_gru<1>, grid, dim3(kRnnThreads), lds, (hipStream_t)stream, p);
    }
    h->rnn_form = ws ? NLB_RNN_FORM_WEIGHT_STATIONARY : NLB_RNN_FORM_TILED;
    uint32_t w = 2;
    for (uint32_t c = 16; c >= 4; c /= 2)
        if (p.srb % c == 0 && (uintptr_t)status % c == 0 && (uintptr_t)wk.cand % c == 0) {
            w = c;
            break;
        }
    const uint32_t upr = p.srb / w;
    uint32_t lg = 0;
    while ((1u << lg) < upr) lg++;
    const uint64_t per = lg <= 6 ? 64u >> lg : 1u;                       // rows per wavefront pass
    const uint64_t blocks = ((pairs + per - 1) / per * 64u + kRnnThreads - 1) / kRnnThreads;
    hipLaunchKernelGGL(rnn_scatter, dim3((unsigned)(blocks < 65536 ? blocks : 65536)),
                       dim3(kRnnThreads), 0, (hipStream_t)stream, (const uint8_t *)wk.cand,
                       (const u32x4 *)list, (const uint32_t *)count, (uint8_t *)status, p.srb, w, upr, lg,
                       wk.winner);
    if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
    return NLB_OK;
}

extern "C" int nlb_rnn_update(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t,
                              uint32_t n, uint64_t first_eid, const nlb_gru_weights *wts, void *status,
                              void *stream) {
    return rnn_update(h, src, dst, t, n, first_eid, wts, status, stream, false);
}

extern "C" int nlb_rnn_update_noalloc(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t,
                                      uint32_t n, uint64_t first_eid, const nlb_gru_weights *wts, void *status,
                                      void *stream) {
    return rnn_update(h, src, dst, t, n, first_eid, wts, status, stream, true);
}
