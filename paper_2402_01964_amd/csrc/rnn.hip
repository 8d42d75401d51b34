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
//            of a matrix product depends on its own inputs only.  The same
//            launch repacks the weights into matrix-operand fragments, so
//            that the gru pass reads each with one contiguous 1 KB load.
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
// (packed, read from global memory, where the whole weight set stays
// L2-resident) go through a three-slot register ring, so each k-step's
// loads are issued two steps before their products.
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
    // The GRU weights, repacked here in operand-fragment order for the GRU
    // pass: fragment (unit block b < kd / 16, k-step s < ks, gate g) is 64
    // lanes x 16 bytes at ((b * ks + s) * 3 + g) * 64, lane l holding unit
    // 16 b + l % 16 (clamped to d - 1), columns 32 s' + 8 (l / 16) .. + 7 of
    // W_i (steps s < kxm = kx / 32, s' = s) or of W_h (s' = s - kxm).
    const __bf16 *w_ih, *w_hh;
    u32x4 *wpack;
    uint32_t d, kx, kd, kxm, ks, pieces;
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
    // The weight pack: each 16-byte piece read once (row reads of 64 bytes)
    // and written once, contiguous in the order the GRU pass loads them.
    if (p.wpack) {
        for (uint32_t q = blockIdx.x * kRnnThreads + threadIdx.x; q < p.pieces; q += gridDim.x * kRnnThreads) {
            const uint32_t l = q & 63u, f = q >> 6, g = f % 3u, s = (f / 3u) % p.ks, b = f / (3u * p.ks);
            const uint32_t jr = min(16u * b + (l & 15u), p.d - 1u), lk = (l >> 4) * 8u;
            const __bf16 *src = s < p.kxm ? p.w_ih + ((size_t)g * p.d + jr) * p.kx + 32u * s + lk
                                          : p.w_hh + ((size_t)g * p.d + jr) * p.kd + 32u * (s - p.kxm) + lk;
            p.wpack[q] = *(const u32x4 *)src;
        }
    }
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
    const __bf16 *w_ih, *w_hh;
    const float *b_ih, *b_hh;
    const u32x4 *wpack;                 // the weights in operand-fragment order (rnn_select)
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

// cos of an fp32 argument with |x| < kCosFastLimit: the revolutions y =
// x / (2 pi) in double, reduced to [0, 1) by v_fract_f64 (exact), then the
// hardware cosine; as cos_fp32_small with one instruction fewer, the
// fraction's rounding to fp32 adding at most 2^-25 of a revolution.
__device__ __forceinline__ float cos_fract(float x) {
    const double y = (double)x * 0.15915494309189533577;
    return __builtin_amdgcn_cosf((float)__builtin_amdgcn_fract(y));
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    const uint32_t u = __float_as_uint(f);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// acc[g'][rb] += A_rb (16 x 32 blocks of the LDS pair Ah/Al, row stride
// `as`; the lo plane starts at column lo_b with its own stride `ls`)
//              * W_g^T for the three gates, over the k-steps kb, kb + 32, ..
// < ke; g' = g for the r and z gates and g' = NIDX for the n gate.  LO adds
// the lo-plane products.  The weights come packed (rnn_select): wp points at
// this lane's word of the fragment (k-step 0, gate 0) of the matrix and unit
// block; fragment (k-step s, gate g) is 192 s + 64 g words on.
template <int NB, bool LO, int NIDX>
__device__ __forceinline__ void gate_seg(f32x4 (&acc)[4][NB], const __bf16 *Ah, const __bf16 *Al,
                                         uint32_t as, uint32_t ls, uint32_t lo_b, const u32x4 *wp,
                                         uint32_t kb, uint32_t ke, uint32_t lr, uint32_t lk) {
    if (kb >= ke) return;
    const uint32_t last = ke - 32;
    bf16x8 r0[3], r1[3], r2[3];
    auto load = [&](bf16x8 (&b)[3], uint32_t k) {
#pragma unroll
        for (int g = 0; g < 3; g++) b[g] = __builtin_bit_cast(bf16x8, wp[(k >> 5) * 192u + g * 64u]);
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
        const u32x4 *wx = p.wpack + (size_t)ub * ((p.kx + p.kd) / 32u) * 192u + lane;
        gate_seg<NB, false, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, 0, p.lo_begin, lr, lk);
        gate_seg<NB, true, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, p.lo_begin, p.lo_end, lr, lk);
        gate_seg<NB, false, 2>(acc, Xh, Xl, p.xs, p.ls, p.lo_begin, wx, p.lo_end, p.kx, lr, lk);
        const u32x4 *wh = wx + (p.kx / 32u) * 192u;
        if (p.h_lo)
            gate_seg<NB, true, 3>(acc, Hh, Hl, p.hs, p.hs, 0, wh, 0, p.kd, lr, lk);
        else
            gate_seg<NB, false, 3>(acc, Hh, Hl, p.hs, p.hs, 0, wh, 0, p.kd, lr, lk);
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
// A tile sits in LDS in matrix-operand order: the operand of k-step s and
// row block rb is 1 KB, lane l's eight values at 16 l, so that every operand
// read is one contiguous 16-byte read per lane at a fixed offset.  Each
// tile buffer is two LDS arrays (so that the compiler can tell a write of
// one from a read or write of the other): S holds what the status rows
// fill (H hi, X hi of the r_other steps), T the rest (X hi of the
// time-encoding and link-row steps, X lo by step, H lo for fp32 statuses;
// lo planes only at steps inside [lo_begin, lo_end)).  Tiles alternate
// between two buffers: the status rows of the next tile are requested at
// the start of the current one and land in its S array meanwhile -- bf16
// rows whose width is a multiple of 32 by direct global-to-LDS loads (one
// operand fragment per load), other rows through registers, written before
// the tile's barrier (fp32 ones as hi + lo).
//
// The products are taken as W X^T (the weight fragment is the first
// operand), so that a lane's four accumulator values are four consecutive
// output units of one tile row: the accumulators start from the gate
// biases, the gates read the units' h values with one 8-byte LDS read (a
// 16-byte global read for fp32 statuses), and the new statuses go straight
// from registers to the candidate rows, 8 or 16 bytes per lane, with no
// exchange between wavefronts.
//
// The two wavefronts that share a SIMD (w and w + KH) alternate between
// matrix and vector work, which the SIMD runs side by side.  After a tile's
// barrier the first half starts on that tile's products at once, while the
// second half issues the loads of the tiles ahead, applies the gates of the
// previous tile (its accumulators and h values kept in registers across the
// barrier) and encodes its share of the next tile's time columns; then the
// second half takes its products while the first half applies its gates and
// encodes its share.  Row
// lists are read three tiles ahead into one of eight row-list slots, the
// link times of a tile's rows two tiles ahead into one of four LDS rows.
// Rows of a tile past the list's end repeat its last entry and are never
// written out.
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
    static constexpr uint32_t slots = 8, tslots = 4;
    // tile buffers, row-list slots, link-time rows, gate biases
    static constexpr uint32_t fixed = 2 * (s_bytes + t_bytes) + slots * 1024 + tslots * 256 + 4 * 32 * KH * 4;
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

// The same with 4 bytes per lane (lane l's word at lds + 4 l).
__device__ __forceinline__ void lds_load4(const void *g, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dword %0, off"
                 :: "v"(g), "{m0}"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)(lds_ptr)p; }

// Candidate-row stores, written as assembly: the compiler would otherwise
// make the next write of their source registers wait until the stores have
// completed (vmcnt), which stalls the loop for a memory round trip; the
// hardware has read the sources one wait state after issue (the nop).
__device__ __forceinline__ void store_b64_async(void *g, u32x2 v) {
    asm volatile("global_store_dwordx2 %0, %1, off\n\ts_nop 1" :: "v"(g), "v"(v) : "memory");
}
__device__ __forceinline__ void store_b128_async(void *g, u32x4 v) {
    asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 1" :: "v"(g), "v"(v) : "memory");
}

// Workgroup barriers of the tile loop.  The first half has no direct loads
// in flight and nothing in global memory that another wavefront reads, so it
// waits for its LDS accesses only (its candidate-row stores complete in the
// background); the second half also waits for its direct loads (vmcnt), which
// the compiler does not count.
__device__ __forceinline__ void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void barrier_loads() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// FULL: every X step is in use and exactly the steps KH .. KXM - 1 have a lo
// plane (kx = 32 KXM; the time encoding, and fp32 link rows if any, fill the
// steps after the status): the products then run without branches.
template <int KH>
constexpr uint32_t ws_full_lomask() { return ((1u << (kWsSteps - KH)) - 1u) & ~((1u << KH) - 1u); }

template <int KH, int MODE, bool FULL>
__global__ __launch_bounds__(128 * KH) void rnn_gru_ws(GruParams p) {
    using L = WsLayout<KH>;
    constexpr uint32_t NB = L::NB, R = kWsRows, T = 128 * KH, TH = T / 2, GH = 4 * KH, FB = L::frag;
    constexpr int KXM = (int)L::KXM, KS = KXM + KH;
    constexpr int SK = MODE == kWsF32 ? kF32Vec : kBf16Vec;
    static_assert(R * GH == T, "one status piece of each input half per thread");
    static_assert(2 * KH == KH * NB, "one operand fragment of each input half per wavefront");
    __shared__ __attribute__((aligned(16))) uint8_t bs0[L::s_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bs1[L::s_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bt0[L::t_bytes];
    __shared__ __attribute__((aligned(16))) uint8_t bt1[L::t_bytes];
    // Row lists {pair row, self, other, 0} of 1 KB slots (R entries and room
    // for the duplicates a direct load of R entries writes); tile i in slot
    // i % 8.  Link times of the rows of tile i in row i % 4 of tt (words
    // R .. 63 of a row: room for the duplicates a direct load writes).
    constexpr uint32_t MS = 64;
    __shared__ __attribute__((aligned(16))) u32x4 meta[L::slots * MS];
    __shared__ __attribute__((aligned(16))) uint32_t tt[L::tslots][64];
    // gate biases by output unit: b_ir + b_hr, b_iz + b_hz, b_in, b_hn
    __shared__ __attribute__((aligned(16))) float sbias[4][32 * KH];
    __shared__ float s_wb[2];   // largest |w| and |b| of the time encoding
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
    // Accumulator value q of row block rb of this lane: output unit u0 + q,
    // tile row 16 rb + lr.
    const uint32_t u0 = 16 * wave + 4 * (lane >> 4);
    const uint32_t gt = (p.off_e - p.kd) / 8, tu = R * gt;

    // This wavefront's weight fragments (loaded in the prologue, after the
    // first tile's requests): lane l holds unit 16 w + l % 16, columns
    // 32 s + 8 (l / 16) .. + 7 of step s.
    bf16x8 bx[KXM][3], bh[KH][3];

    auto list_at = [&](uint32_t tl, uint32_t row) __attribute__((always_inline)) {
        return min((uint64_t)tl * R + row, (uint64_t)count - 1);
    };

    // Direct path: operand fragment f (< 2 KH) of H and of X's r_other for
    // the tile in row-list slot `slot`, lane l from tile row 16 (f % NB) +
    // l % 16, columns 32 (f / NB) + 8 (l / 16) .. + 7.  Register path: a
    // thread's status pieces, f = 0 of H (self) and f = 1 of X's r_other,
    // both at tile row pj, columns pc0 .. pc0 + 7, written to LDS later.
    auto request_frag = [&](uint8_t *nbS, uint32_t slot, uint32_t f) __attribute__((always_inline)) {
        const uint32_t dj = 16 * (f % NB) + lr, dc = 32 * (f / NB) + lk;
        const u32x4 e = meta[slot * MS + dj];
        lds_load16(p.st + (size_t)e[1] * p.srb + 2u * dc, lds_addr(nbS + L::sh + f * FB));
        lds_load16(p.st + (size_t)e[2] * p.srb + 2u * dc, lds_addr(nbS + L::sx + f * FB));
    };
    const uint32_t pj = tid / GH, pc0 = 8 * (tid % GH);
    Piece8<SK> pc[2];
    auto request_pieces = [&](uint32_t slot) __attribute__((always_inline)) {
        const u32x4 e = meta[slot * MS + pj];
        load_piece<SK>(p.st + (size_t)e[1] * p.srb, d, pc0, pc[0]);
        load_piece<SK>(p.st + (size_t)e[2] * p.srb, d, pc0, pc[1]);
    };
    auto write_pieces = [&](uint8_t *nbS, uint8_t *nbT) __attribute__((always_inline)) {
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
    };

    // Time-encoding unit u of a tile: lane l = u % 64 of operand fragment
    // f = u / 64 of the encoding's steps (step f / NB, row block f % NB), i.e.
    // tile row 16 (f % NB) + l % 16 and encoding columns 32 (f / NB) +
    // 8 (l / 16) .. + 7, so that its eight values sit at byte 16 u of their
    // plane (a wavefront's writes are contiguous).  Arguments beyond the fast
    // cosine's range are rare: their units are redone, exactly, only where a
    // wavefront meets one.
    auto unit_row = [](uint32_t u) { return 16u * ((u >> 6) % NB) + (u & 15u); };
    auto unit_col = [](uint32_t u) { return 32u * ((u >> 6) / NB) + 8u * ((u >> 4) & 3u); };
    // Columns past d_time have w = b = 0 here, so their (finite) values meet
    // the weights' zero padding.  Where no argument of the wavefront's units
    // can reach the fast cosine's limit (|w| t + |b| below half of it for the
    // largest |w| and |b| of the encoding, wmax and bmax) the values take the
    // fast path with no per-value test.
    float wmax = 0.0f, bmax = 0.0f;   // set after the prologue
    auto tenc_unit = [&](uint8_t *nbT, uint32_t u, float tf) __attribute__((always_inline)) {
        const uint32_t k = unit_col(u);
        const bool fast = __ballot(!(__builtin_fmaf(wmax, tf, bmax) < 0.5f * kCosFastLimit)) == 0;
        // two halves of four values (fewer registers live at once)
#pragma unroll
        for (int h = 0; h < 2; h++) {
            const f32x4 w = *(const f32x4 *)(s_tw + k + 4 * h), b = *(const f32x4 *)(s_tb + k + 4 * h);
            float v[4];
            if (__builtin_expect(fast, 1)) {
#pragma unroll
                for (int e = 0; e < 4; e++) v[e] = cos_fract(__builtin_fmaf(w[e], tf, b[e]));
            } else {
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const float x = __builtin_fmaf(w[e], tf, b[e]);
                    v[e] = __builtin_fabsf(x) < kCosFastLimit ? cos_fp32_small(x) : cos_fp32_exact_wide(x);
                }
            }
            u32x2 hi, lo;
#pragma unroll
            for (int e = 0; e < 4; e += 2) {
                const float a0 = v[e], a1 = v[e + 1];
                const __bf16 h0 = (__bf16)a0, h1 = (__bf16)a1;
                const __bf16 l0 = (__bf16)(a0 - (float)h0), l1 = (__bf16)(a1 - (float)h1);
                hi[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
                lo[e / 2] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
            }
            *(u32x2 *)(nbT + L::tx + 16u * u + 8u * h) = hi;
            *(u32x2 *)(nbT + L::tl + KH * NB * FB + 16u * u + 8u * h) = lo;
        }
    };

    // The link rows of a tile (first half only).
    auto write_edges = [&](uint8_t *nbT, uint32_t slot) __attribute__((always_inline)) {
        if (!second && p.kx > p.off_e) {
            const uint32_t ge = (p.kx - p.off_e) / 8;
            auto edge_fill = [&](auto kind) __attribute__((always_inline)) {
                constexpr int K = decltype(kind)::value;
                auto eid_of = [&](uint32_t jj) __attribute__((always_inline)) {
                    return first_eid + (meta[slot * MS + jj][0] >> 1);
                };
                fill_seg<K, 4, TH>(
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
            // The fill's last loads may go unused; waiting for them here keeps
            // the compiler from waiting for them (and for every store issued
            // since) at the next write of their registers.
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
        }
    };

    // Prologue, ordered so that the weights' transfer (about 300 KB per CU,
    // from L2) overlaps the first tile's dependent loads and its time
    // encoding: the row lists of the first three tiles, the time-encoding
    // parameters and the biases, all issued before any is used; then the
    // link times of the first two tiles' rows (direct loads into tt), the
    // weights and the first tile's status rows; then, once the link times
    // are in, the first tile's time encoding, and one wait for everything
    // before the barrier.
    const uint32_t stride = gridDim.x;
    uint32_t tl = blockIdx.x;
    {
        constexpr uint32_t TW = (32u * (kWsSteps - 2 * KH) + T - 1) / T;   // pad32(d_time) <= 32 (KXM - KH)
        const uint32_t padt = (p.d_time + 31u) & ~31u;
        u32x4 le = {};
        if (tid < 3 * R) {
            const uint32_t k = tid / R, tk = tl + k * stride < tiles ? tl + k * stride : tl;
            le = p.list[list_at(tk, tid % R)];
        }
        float twv[TW], tbv[TW], bv[6];
#pragma unroll
        for (uint32_t k = 0; k < TW; k++) {
            const uint32_t u = tid + k * T;
            twv[k] = u < p.d_time ? p.tw[u] : 0.0f;
            tbv[k] = u < p.d_time ? p.tb[u] : 0.0f;
        }
        if (lane < 16 && mma) {
#pragma unroll
            for (int g = 0; g < 3; g++) {
                bv[2 * g] = p.b_ih[g * d + jr];
                bv[2 * g + 1] = p.b_hh[g * d + jr];
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (tid < 3 * R) meta[(tid / R) * MS + tid % R] = le;
#pragma unroll
        for (uint32_t k = 0; k < TW; k++) {
            const uint32_t u = tid + k * T;
            if (u < padt) {
                s_tw[u] = twv[k];
                s_tb[u] = tbv[k];
            }
        }
        if (lane < 16 && mma) {
            sbias[0][j] = bv[0] + bv[1];
            sbias[1][j] = bv[2] + bv[3];
            sbias[2][j] = bv[4];
            sbias[3][j] = bv[5];
        }
    }
    __syncthreads();
    if (wave == 0) {
        float mw = 0.0f, mb = 0.0f;
        for (uint32_t u = lane; u < ((p.d_time + 31u) & ~31u); u += 64) {
            mw = fmaxf(mw, __builtin_fabsf(s_tw[u]));
            mb = fmaxf(mb, __builtin_fabsf(s_tb[u]));
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            mw = fmaxf(mw, __shfl_xor(mw, o));
            mb = fmaxf(mb, __shfl_xor(mb, o));
        }
        if (lane == 0) {
            s_wb[0] = mw;
            s_wb[1] = mb;
        }
    }
    {   // link times of the first two tiles' rows, straight into tt rows 0 and 1 (every
        // wavefront loads the same words, so each needs to wait for its own loads only,
        // and no branch makes the compiler wait for them at its join)
        lds_load4(p.t + (meta[lane & (R - 1)][0] >> 1), lds_addr(tt[0]));
        lds_load4(p.t + (meta[MS + (lane & (R - 1))][0] >> 1), lds_addr(tt[1]));
    }
    __builtin_amdgcn_sched_barrier(0);
    {   // this wavefront's fragments, 1 KB each, contiguous (packed by rnn_select;
        // X steps past kx_steps re-read the last one, unused)
        const u32x4 *wf = p.wpack + (size_t)wave * (kx_steps + KH) * 192u + lane;
#pragma unroll
        for (int s = 0; s < KXM; s++)
#pragma unroll
            for (int g = 0; g < 3; g++)
                bx[s][g] = __builtin_bit_cast(bf16x8, wf[(min((uint32_t)s, kx_steps - 1u) * 3u + g) * 64u]);
#pragma unroll
        for (int s = 0; s < KH; s++)
#pragma unroll
            for (int g = 0; g < 3; g++) bh[s][g] = __builtin_bit_cast(bf16x8, wf[((kx_steps + s) * 3u + g) * 64u]);
    }
    if constexpr (MODE == kWsBf16Dma)
        request_frag(bs0, 0, wave);
    else
        request_pieces(0);
    __builtin_amdgcn_sched_barrier(0);
    // Wait for the two link-time loads only: at least the 36 weight loads
    // were issued after them, and loads complete in order.
    static_assert(3 * (KXM + KH) == 36, "weight loads per lane");
    asm volatile("s_waitcnt vmcnt(36)" ::: "memory");
    __syncthreads();
    wmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(s_wb[0])));
    bmax = __uint_as_float(__builtin_amdgcn_readfirstlane(__float_as_uint(s_wb[1])));
    for (uint32_t u = tid; u < tu; u += T) tenc_unit(bt0, u, (float)tt[0][unit_row(u)]);
    if constexpr (MODE != kWsBf16Dma) write_pieces(bs0, bt0);
    write_edges(bt0, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0), seen by the compiler's own wait tracking
    __syncthreads();

    // The products of a tile (buffers cbS, cbT) into acc, from the biases.
    f32x4 acc[4][NB];   // r, z, input part of n, hidden part of n
    auto products = [&](const uint8_t *cbS, const uint8_t *cbT) __attribute__((always_inline)) {
        {
            const f32x4 b0 = *(const f32x4 *)&sbias[0][u0], b1 = *(const f32x4 *)&sbias[1][u0],
                        b2 = *(const f32x4 *)&sbias[2][u0], b3 = *(const f32x4 *)&sbias[3][u0];
#pragma unroll
            for (int rb = 0; rb < NB; rb++) {
                acc[0][rb] = b0;
                acc[1][rb] = b1;
                acc[2][rb] = b2;
                acc[3][rb] = b3;
            }
        }
        const uint32_t lm = FULL ? ws_full_lomask<KH>() : opaque_u32(p.ws_lomask),
                       ks = FULL ? (uint32_t)KXM : opaque_u32(kx_steps);
        const uint8_t *bS = cbS + 16u * lane, *bT = cbT + 16u * lane;
        auto mfma3 = [&](const bf16x8 (&a)[NB], const bf16x8 (&w)[3], int nidx) __attribute__((always_inline)) {
#pragma unroll
            for (int rb = 0; rb < NB; rb++)
#pragma unroll
                for (int g = 0; g < 3; g++) {
                    const int gi = g == 2 ? nidx : g;
                    acc[gi][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[g], a[rb], acc[gi][rb], 0, 0, 0);
                }
        };
        // Operands of step s (X steps, then H steps): the hi plane always,
        // the lo plane where the step has one.  Hi operands are read AH steps
        // before their products (two where the registers allow), lo operands
        // one step before.
        constexpr int AH = 1;
        auto load_hi = [&](int s, bf16x8 (&a)[NB]) __attribute__((always_inline)) {
            const uint8_t *hi = s < KH ? bS + L::sx + s * NB * FB
                              : s < KXM ? bT + L::tx + (s - KH) * NB * FB : bS + L::sh + (s - KXM) * NB * FB;
#pragma unroll
            for (int rb = 0; rb < NB; rb++) a[rb] = *(const bf16x8 *)(hi + rb * FB);
        };
        auto load_lo = [&](int s, bf16x8 (&al)[NB]) __attribute__((always_inline)) {
            const uint8_t *lo = s < KXM ? bT + L::tl + s * NB * FB : bT + L::th + (s - KXM) * NB * FB;
            if (s < KXM ? ((lm >> s) & 1u) != 0 : MODE == kWsF32) {
#pragma unroll
                for (int rb = 0; rb < NB; rb++) al[rb] = *(const bf16x8 *)(lo + rb * FB);
            }
        };
        bf16x8 a[AH + 1][NB], al[NB];
#pragma unroll
        for (int s = 0; s < AH; s++) load_hi(s, a[s]);
        load_lo(0, al);
#pragma unroll
        for (int s = 0; s < KS; s++) {
            bf16x8 nal[NB];
            if (s + AH < KS) load_hi(s + AH, a[(s + AH) % (AH + 1)]);
            if (s + 1 < KS) load_lo(s + 1, nal);
            // (the loads stay ahead of this step's products: without branches
            // between the steps the scheduler would otherwise sink each read
            // to its first use and wait for it there)
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8 (&as)[NB] = a[s % (AH + 1)];
            if (s < KXM) {
                if ((uint32_t)s < ks) mfma3(as, bx[s], 2);
                if ((lm >> s) & 1u) mfma3(al, bx[s], 2);
            } else {
                mfma3(as, bh[s - KXM], 3);
                if constexpr (MODE == kWsF32) mfma3(al, bh[s - KXM], 3);
            }
#pragma unroll
            for (int rb = 0; rb < NB; rb++) al[rb] = nal[rb];
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // h values of this lane's units u0 .. u0 + 3 in the tile's rows: from the
    // tile's H plane (bf16 statuses, packed pairs) or the status rows (fp32).
    using HvT = std::conditional_t<MODE == kWsF32, f32x4, u32x2>;
    HvT hv[NB];
    uint32_t prow[NB];   // second half: pair rows of the tile whose gates are pending
    auto read_hv = [&](const uint8_t *cbS, uint32_t ms) __attribute__((always_inline)) {
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const uint32_t row = 16u * rb + lr;
            if constexpr (MODE == kWsF32)
                hv[rb] = u0 < d ? *(const f32x4 *)(p.st + (size_t)meta[ms * MS + row][1] * p.srb + 4u * u0) : f32x4(0.0f);
            else
                hv[rb] = *(const u32x2 *)(cbS + L::sh + frag_off(row, u0 & ~7u) + 2u * (u0 & 7u));
        }
    };
    auto h_at = [&](int rb, int q) __attribute__((always_inline)) {
        if constexpr (MODE == kWsF32)
            return hv[rb][q];
        else
            return __uint_as_float(q & 1 ? hv[rb][q >> 1] & 0xFFFF0000u : hv[rb][q >> 1] << 16);
    };
    // The gates of tile tlg of the launch from acc and hv; new statuses of
    // its listed rows to their candidate rows (pair rows pr of the lane's
    // tile rows 16 rb + lr, read from the tile's row-list slot).
    auto pair_rows = [&](uint32_t ms, uint32_t (&pr)[NB]) __attribute__((always_inline)) {
#pragma unroll
        for (int rb = 0; rb < NB; rb++) pr[rb] = meta[ms * MS + 16u * rb + lr][0];
    };
    auto gates = [&](const uint32_t (&pr)[NB], uint32_t tlg) __attribute__((always_inline)) {
        const uint32_t nrows = min(R, count - tlg * R);
#pragma unroll
        for (int rb = 0; rb < NB; rb++) {
            const uint32_t row = 16u * rb + lr;
            float out[4];
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const float rg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(acc[0][rb][q] * -kLog2e));
                const float zg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(acc[1][rb][q] * -kLog2e));
                const float ng = tanh_f32(__builtin_fmaf(rg, acc[3][rb][q], acc[2][rb][q]));
                out[q] = __builtin_fmaf(zg, h_at(rb, q) - ng, ng);   // (1 - z) n + z h
            }
            if (u0 < d && row < nrows) {
                uint8_t *dst = p.cand + (size_t)pr[rb] * p.srb;
                if constexpr (MODE == kWsF32) {
                    store_b128_async(dst + 4u * u0, u32x4{__float_as_uint(out[0]), __float_as_uint(out[1]),
                                                          __float_as_uint(out[2]), __float_as_uint(out[3])});
                } else {
                    u32x2 o;
#pragma unroll
                    for (int q = 0; q < 4; q += 2)   // round to nearest even
                        o[q / 2] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)out[q]) |
                                   ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)out[q + 1]) << 16);
                    store_b64_async(dst + 2u * u0, o);
                }
            }
        }
    };

    // Tile i of the workgroup (launch tile tl, buffers i % 2, row-list slot
    // i % 8) in the first half: products, gates, then its share of the next
    // tile's time encoding (units tid, tid + T, ..., as in the second half)
    // and the link rows; false after the workgroup's last tile.  (No loads here
    // on the direct path: a wait for one would also wait for the last tile's
    // candidate-row stores.)
    auto tile_first = [&](uint8_t *cbS, uint8_t *cbT, uint8_t *nbS, uint8_t *nbT, uint32_t i)
                          __attribute__((always_inline)) {
        const uint32_t ms = i & 7;
        const bool has_next = tl + stride < tiles;
        if (MODE != kWsBf16Dma && has_next) request_pieces((i + 1) & 7);
        if (mma) {
            products(cbS, cbT);
            read_hv(cbS, ms);
            uint32_t pr[NB];
            pair_rows(ms, pr);
            gates(pr, tl);
        }
        if (has_next) {
            for (uint32_t u = tid; u < tu; u += T) tenc_unit(nbT, u, (float)tt[(i + 1) & 3][unit_row(u)]);
            if (MODE != kWsBf16Dma) write_pieces(nbS, nbT);
            write_edges(nbT, (i + 1) & 7);
        }
        barrier_lds();
        tl += stride;
        return has_next;
    };
    // The same tile in the second half: the loads of the tiles ahead, the
    // gates of the previous tile, its share of the next tile's time encoding,
    // then the products and h values, kept for the next tile.  Wavefront KH reads
    // the row lists and link times.
    auto tile_second = [&](uint8_t *cbS, uint8_t *cbT, uint8_t *nbS, uint8_t *nbT, uint32_t i)
                           __attribute__((always_inline)) {
        const uint32_t ms = i & 7, ns = (i + 1) & 7;
        const bool has_next = tl + stride < tiles, has_nn = tl + 2 * stride < tiles,
                   has_n3 = tl + 3 * stride < tiles;
        if (wave == (uint32_t)KH && has_n3)   // row list of the tile three on, straight into its slot
            lds_load16(p.list + list_at(tl + 3 * stride, lane & (R - 1)), lds_addr(meta + ((i + 3) & 7) * MS));
        // link times of the rows of the tile two on (its row list arrived with
        // the last barrier), straight into their row of tt
        if (wave == (uint32_t)KH && has_nn)
            lds_load4(p.t + (meta[((i + 2) & 7) * MS + (lane & (R - 1))][0] >> 1), lds_addr(tt[(i + 2) & 3]));
        if (has_next) {
            if constexpr (MODE == kWsBf16Dma) {
                request_frag(nbS, ns, wave - KH);
                request_frag(nbS, ns, wave);
            } else {
                request_pieces(ns);
            }
        }
        if (i > 0 && mma) gates(prow, tl - stride);
        if (has_next) {
            for (uint32_t u = tid; u < tu; u += T) tenc_unit(nbT, u, (float)tt[(i + 1) & 3][unit_row(u)]);
            if (MODE != kWsBf16Dma) write_pieces(nbS, nbT);
        }
        if (mma) {
            products(cbS, cbT);
            read_hv(cbS, ms);
            pair_rows(ms, prow);
        }
        barrier_loads();
        tl += stride;
        return has_next;
    };
    if (!second) {
        for (uint32_t i = 0;; i += 2) {
            if (!tile_first(bs0, bt0, bs1, bt1, i)) break;
            if (!tile_first(bs1, bt1, bs0, bt0, i + 1)) break;
        }
    } else {
        uint32_t i = 0;
        for (;; i += 2) {
            if (!tile_second(bs0, bt0, bs1, bt1, i)) break;
            if (!tile_second(bs1, bt1, bs0, bt0, i + 1)) {
                i++;
                break;
            }
        }
        if (mma) gates(prow, tl - stride);   // the workgroup's last tile
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

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Per-table working memory of the update, grown on demand: the winner
// words, the list, and one buffer for the candidate rows followed (at a
// 256-byte boundary) by the packed GRU weights.
int rnn_reserve(nlb_table *h, uint64_t pair_rows, uint32_t srb, size_t wpack_bytes) {
    if (!h->rnn_winner) {
        const size_t bytes = (size_t)h->num_nodes * 8u;
        if (hipMalloc((void **)&h->rnn_winner, bytes) != hipSuccess) {
            (void)hipGetLastError();
            h->rnn_winner = nullptr;
            return NLB_ENOMEM;
        }
        if (hipMemset(h->rnn_winner, 0, bytes) != hipSuccess) return NLB_EDEVICE;
    }
    const size_t cbytes = align256((size_t)pair_rows * srb) + wpack_bytes;
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
    uint8_t *wpack;       // the weights in operand-fragment order
};

// Working memory of the table, grown on demand (nlb_rnn_update).
int table_work(nlb_table *h, uint64_t pairs, uint32_t srb, size_t wpack_bytes, RnnWork *wk) {
    const int rc = rnn_reserve(h, pairs, srb, wpack_bytes);
    if (rc != NLB_OK) return rc;
    *wk = {h->rnn_winner, false, h->rnn_cand, h->rnn_list,
           wpack_bytes ? h->rnn_cand + align256((size_t)pairs * srb) : nullptr};
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

// The update's working memory carved from `scratch`: winner words of all N
// nodes, the list, the packed weights, the candidate rows.  The winner words are cleared by a fill kernel at the
// start of every call.
int scratch_work(nlb_table *h, uint64_t pairs, uint32_t srb, size_t wpack_bytes, RnnWork *wk) {
    const size_t winner_bytes = align256((size_t)h->num_nodes * 8u);
    const size_t list_bytes = align256(((size_t)pairs * 4u + 64u) * 4u);
    const size_t pack_bytes = align256(wpack_bytes);
    const size_t cand_bytes = (size_t)pairs * srb;
    if (winner_bytes + list_bytes + pack_bytes + cand_bytes > kScratchBytes) return NLB_ESCRATCH;
    uint8_t *base = nullptr;
    const int rc = scratch_address(h->device, &base);
    if (rc != NLB_OK) return rc;
    *wk = {(unsigned long long *)base, true, base + winner_bytes + list_bytes + pack_bytes,
           (uint32_t *)(base + winner_bytes), wpack_bytes ? base + winner_bytes + list_bytes : nullptr};
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
        // static LDS: tile buffers, row-list slots, link times, biases; dynamic: T-enc w | b
        const uint32_t fixed = kh == 1 ? WsLayout<1>::fixed : kh == 2 ? WsLayout<2>::fixed
                             : kh == 3 ? WsLayout<3>::fixed : WsLayout<4>::fixed;
        lds = 8u * pad32(p.d_time);
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

    // packed weight fragments: kd / 16 unit blocks x (kx + kd) / 32 k-steps x 3 gates, 1 KB each
    const size_t wpack_bytes = (size_t)(p.kd / 16) * ((p.kx + p.kd) / 32) * 3 * 1024;
    RnnWork wk;
    const int rc = use_scratch ? scratch_work(h, pairs, p.srb, wpack_bytes, &wk)
                               : table_work(h, pairs, p.srb, wpack_bytes, &wk);
    if (rc != NLB_OK) return rc;
    p.wpack = (const u32x4 *)wk.wpack;
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
    SelectParams sp = {src, dst, n, h->num_nodes, wk.winner, list, count,
                       p.w_ih, p.w_hh, (u32x4 *)wk.wpack, p.d, p.kx, p.kd, p.kx / 32, (p.kx + p.kd) / 32,
                       (uint32_t)(wpack_bytes / 16)};
    // (at least enough workgroups for the weight pack at 8 pieces per thread:
    // workgroups past the pair rows select nothing)
    const uint64_t sel_blocks = std::max<uint64_t>((pairs + kSelectRows - 1) / kSelectRows,
                                                   (sp.pieces + 8u * kRnnThreads - 1) / (8u * kRnnThreads));
    hipLaunchKernelGGL(rnn_select, dim3((unsigned)sel_blocks), dim3(kRnnThreads), 0, (hipStream_t)stream, sp);
    if (ws) {
        const void *kern = nullptr;
        const bool full = ws_mode == kWsBf16Dma && kh == 4 && p.kx == 32u * (kWsSteps - 4) &&
                          p.ws_lomask == ws_full_lomask<4>();
        switch (kh * 4 + ws_mode) {
#define NLB_WS_CASE(KH, MODE) \
        case KH * 4 + MODE: kern = (const void *)rnn_gru_ws<KH, MODE, false>; break;
        NLB_WS_CASE(1, kWsBf16Dma) NLB_WS_CASE(1, kWsBf16) NLB_WS_CASE(1, kWsF32)
        NLB_WS_CASE(2, kWsBf16Dma) NLB_WS_CASE(2, kWsBf16) NLB_WS_CASE(2, kWsF32)
        NLB_WS_CASE(3, kWsBf16Dma) NLB_WS_CASE(4, kWsBf16Dma)
#undef NLB_WS_CASE
        default: return NLB_EINVAL;
        }
        if (full) kern = (const void *)rnn_gru_ws<4, kWsBf16Dma, true>;
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
