// nlb.hip -- gfx950 kernels and the C ABI (include/nlb.h) of NLB forward
// recent sampling (Luo & Li, arXiv 2402.01964, Sec. 4.2 and Sec. 4.4): table
// creation, batch insertion, first- and second-hop sampling, export.  The
// table layout and key-word format are described in nlb_internal.h.
#include <climits>
#include <cstring>
#include <new>

#include "nlb_internal.h"

namespace {

constexpr int kInsertThreads = 256;

// ---------------------------------------------------------------- integer helpers
// Output number n (n >= 1) of SplitMix64 started at `state0`; its mixing
// function is the one published by Steele, Lea & Flood (OOPSLA 2014).
__device__ __forceinline__ uint64_t splitmix64_nth(uint64_t state0, uint64_t n) {
    uint64_t z = state0 + n * kGolden;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// ---------------------------------------------------------------- insert
struct InsertParams {
    const int32_t *src;
    const int32_t *dst;
    const uint32_t *t;
    uint32_t n;
    uint8_t *blocks;
    uint32_t block_bytes;
    uint32_t s;
    int64_t num_nodes;
    uint64_t seed;
    uint64_t thr;         // replace when coin < thr
    uint64_t mod_m;       // nlb_mod_magic(s)
    uint32_t q1r, q2r;    // q1 mod s, q2 mod s
    uint32_t key_mode;
    uint32_t *status;     // device status words (nlb_internal.h)
};

// The batch's place in the stream, read from the device status words at
// the start of each insert kernel (the link count by insert_resolve, its copy
// for the batch in flight by insert_commit): e0 = arrival index of link 0,
// and whether the batch fits the 32-bit arrival indices (a batch that does
// not is skipped and flagged).
struct BatchPos {
    uint32_t e0;
    bool ok;
};

__device__ __forceinline__ BatchPos batch_pos(const InsertParams &p, uint32_t word) {
    const uint64_t links = *(const uint64_t *)(p.status + word);
    BatchPos b;
    b.e0 = (uint32_t)links;
    b.ok = links + p.n <= 0xFFFFFFFFull;
    return b;
}

// insert_resolve's record of the batch in flight, for insert_commit.
__device__ __forceinline__ void record_batch(const InsertParams &p, const BatchPos &bp) {
    if (blockIdx.x == 0 && threadIdx.x == 0) *(uint64_t *)(p.status + kWordBatch) = bp.e0;
}

// Slot of neighbour x at time t: eq. (2) (q1*x + q2*t) mod s, or eq. (3)
// q1*x mod s, evaluated on residues (exact: both products are < s^2).
__device__ __forceinline__ uint32_t slot_of(const InsertParams &p, uint32_t x, uint32_t t) {
    const uint32_t xr = nlb_mod(x, p.mod_m, p.s);
    uint32_t h = p.q1r * xr;
    if (p.key_mode == NLB_KEY_EDGE) h += p.q2r * nlb_mod(t, p.mod_m, p.s);
    return nlb_mod(h, p.mod_m, p.s);
}

__device__ __forceinline__ uint64_t offer_word(const InsertParams &p, uint32_t e, uint32_t k,
                                               uint32_t t) {
    const uint32_t coin = (uint32_t)(splitmix64_nth(p.seed, 2ull * e + k + 1) >> 32);
    return ((uint64_t)coin < p.thr)
               ? (kClassPass | ((uint64_t)e << kTimeBits) | t)
               : (kClassFail | ((uint64_t)(~e) << kTimeBits) | t);
}

__device__ __forceinline__ bool link_ok(const InsertParams &p, int32_t u, int32_t v, uint32_t t) {
    return u >= 0 && v >= 0 && (int64_t)u < p.num_nodes && (int64_t)v < p.num_nodes &&
           t <= kTimeMask;
}

// Pass 1.  Each link validates itself and turns into two offer words that
// go to their slots with a 64-bit atomic maximum.  For large batches a
// workgroup takes kResolveLinks consecutive links and first merges their
// offers per slot in an LDS hash table (open addressing on the key word's
// byte offset, 64-bit LDS atomics), so a slot that many of its offers hit --
// the slots of a popular node -- costs one global atomic per workgroup
// instead of one per offer; the maximum is associative, so the result is the
// same.  Small batches skip the merge: they have few workgroups and little
// same-slot traffic, and the plain atomics finish sooner.  The merge table
// is merge_max of nlb_internal.h.

// Validation of link i (ranges; timestamps non-decreasing inside the batch
// and against the last timestamp of the previous batch) and its two offers.
// Returns false when the link is skipped.
// link_offers_of takes the link's already-loaded u, v, t and the previous
// link's timestamp.
__device__ __forceinline__ bool link_offers_of(const InsertParams &p, const BatchPos &bp, uint32_t i, int32_t u,
                                               int32_t v, uint32_t t, uint32_t prev_t, uint64_t &ou,
                                               uint64_t &wu, uint64_t &ov, uint64_t &wv) {
    uint32_t flags = 0;
    if (u < 0 || v < 0 || (int64_t)u >= p.num_nodes || (int64_t)v >= p.num_nodes)
        flags |= kStatusRange;
    if (t > kTimeMask) flags |= kStatusOrder;
    if (t < prev_t) flags |= kStatusOrder;
    if (flags) atomicOr(p.status, flags);
    if (!link_ok(p, u, v, t)) return false;
    const uint32_t e = bp.e0 + i;
    // Sec. 4.2: S_u receives (v, t, e); S_v receives (u, t, e).
    ou = (uint64_t)u * p.block_bytes + 8u * slot_of(p, (uint32_t)v, t);
    ov = (uint64_t)v * p.block_bytes + 8u * slot_of(p, (uint32_t)u, t);
    wu = offer_word(p, e, 0, t);
    wv = offer_word(p, e, 1, t);
    return true;
}

// The previous link's timestamp (for link 0, the last of the previous batch,
// which insert_commit records).
__device__ __forceinline__ uint32_t prev_time(const InsertParams &p, uint32_t i) {
    return (i > 0) ? p.t[i - 1] : p.status[kWordLastT];
}

__device__ __forceinline__ bool link_offers(const InsertParams &p, const BatchPos &bp, uint32_t i,
                                            uint64_t &ou, uint64_t &wu, uint64_t &ov, uint64_t &wv) {
    return link_offers_of(p, bp, i, p.src[i], p.dst[i], p.t[i], prev_time(p, i), ou, wu, ov, wv);
}

__global__ __launch_bounds__(kInsertThreads) void insert_resolve(InsertParams p) {
    const uint32_t i = blockIdx.x * kInsertThreads + threadIdx.x;
    const BatchPos bp = batch_pos(p, kWordLinks);
    record_batch(p, bp);
    if (!bp.ok) {
        if (i == 0) atomicOr(p.status, kStatusRange);
        return;
    }
    if (i >= p.n) return;
    uint64_t ou, wu, ov, wv;
    if (!link_offers(p, bp, i, ou, wu, ov, wv)) return;
    atomicMax((unsigned long long *)(p.blocks + ou), (unsigned long long)wu);
    atomicMax((unsigned long long *)(p.blocks + ov), (unsigned long long)wv);
}

__global__ __launch_bounds__(kMergeThreads) void insert_resolve_merged(InsertParams p) {
    __shared__ unsigned long long merge_off[kMergeEntries];
    __shared__ unsigned long long merge_word[kMergeEntries];
    for (int k = threadIdx.x; k < kMergeEntries; k += kMergeThreads) {
        merge_off[k] = 0ull;
        merge_word[k] = 0ull;
    }
    __syncthreads();
    const BatchPos bp = batch_pos(p, kWordLinks);
    record_batch(p, bp);
    if (!bp.ok) {
        if (blockIdx.x == 0 && threadIdx.x == 0) atomicOr(p.status, kStatusRange);
        return;   // uniform over the grid: no workgroup waits at a later barrier
    }
    // All of a thread's links are loaded (a link past the batch re-reads
    // the last one, unused) before any is merged.
    constexpr int RR = kResolveLinks / kMergeThreads;
    const uint32_t first = blockIdx.x * kResolveLinks;
    int32_t uu[RR], vv[RR];
    uint32_t tt[RR], pt[RR];
#pragma unroll
    for (int r = 0; r < RR; r++) {
        const uint32_t i = min(first + r * kMergeThreads + threadIdx.x, p.n - 1u);
        uu[r] = p.src[i];
        vv[r] = p.dst[i];
        tt[r] = p.t[i];
        pt[r] = prev_time(p, i);
    }
#pragma unroll
    for (int r = 0; r < RR; r++) {
        const uint32_t i = first + r * kMergeThreads + threadIdx.x;
        if (i >= p.n) break;
        uint64_t ou, wu, ov, wv;
        if (link_offers_of(p, bp, i, uu[r], vv[r], tt[r], pt[r], ou, wu, ov, wv)) {
            merge_max(merge_off, merge_word, ou, wu);
            merge_max(merge_off, merge_word, ov, wv);
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < kMergeEntries; k += kMergeThreads) {
        const unsigned long long tag = merge_off[k];
        if (tag) atomicMax((unsigned long long *)(p.blocks + (tag - 1)), merge_word[k]);
    }
}

// Pass 2, also the batch's end: it reads the batch position insert_resolve
// recorded and advances the link count and the last timestamp for the next
// batch (words no workgroup of this kernel reads).
__global__ __launch_bounds__(kInsertThreads) void insert_commit(InsertParams p) {
    const uint32_t i = blockIdx.x * kInsertThreads + threadIdx.x;
    const BatchPos bp = batch_pos(p, kWordBatch);
    if (bp.ok && i == 0) *(uint64_t *)(p.status + kWordLinks) = (uint64_t)bp.e0 + p.n;
    if (bp.ok && i == p.n - 1) p.status[kWordLastT] = p.t[i];
    if (bp.ok && i < p.n) {
        const int32_t u = p.src[i];
        const int32_t v = p.dst[i];
        const uint32_t t = p.t[i];
        if (link_ok(p, u, v, t)) {
            const uint32_t e = bp.e0 + i;
            const uint32_t au = slot_of(p, (uint32_t)v, t);
            const uint32_t av = slot_of(p, (uint32_t)u, t);
            uint8_t *bu = p.blocks + (size_t)u * p.block_bytes;
            uint8_t *bv = p.blocks + (size_t)v * p.block_bytes;
            const uint64_t wu = ((const uint64_t *)bu)[au];
            const uint64_t wv = ((const uint64_t *)bv)[av];
            // Exactly one offer owns each surviving word (a self-loop's two
            // offers may share one; they write the same id).
            if (wu == offer_word(p, e, 0, t)) ((int32_t *)(bu + 8u * p.s))[au] = v;
            if (wv == offer_word(p, e, 1, t)) ((int32_t *)(bv + 8u * p.s))[av] = u;
        }
    }
}

// ---------------------------------------------------------------- sample
// A 256-thread workgroup answers a tile of consecutive queries.  Its outputs
// are contiguous ranges of every output array, so all stores are streamed
// full lines.  Phase 1 reads the tile's table slots (one thread per slot
// row), writes the id outputs and stages each slot's (neighbour, arrival
// index, timestamp, gap) in LDS.  The later phases walk the flattened output
// ranges (time encoding, link rows, neighbour rows, self rows) with every
// thread taking consecutive 16-, 12-, 8- or 4-byte units; they look up their slot
// in LDS and keep several row loads in flight before storing.
constexpr int kTileThreads = 256;
constexpr int kTileSlots = 1024;   // slot rows staged per tile (16 B each in LDS)

struct SampleParams {
    const uint8_t *blocks;
    uint32_t block_bytes;
    uint32_t s;
    int64_t num_nodes;
    const int32_t *node;
    const uint32_t *tq;
    uint32_t nq;
    uint32_t tile_q;      // queries per tile; tile_q * s <= kTileSlots
    uint64_t s_m;         // nlb_div12_magic(s): slot rows of a tile (< 2^12) by s (<= 2^12)
    uint32_t d_time;
    const float *w;
    const float *b;
    const uint8_t *efeat;
    int64_t edge_rows;
    uint32_t erb;         // bytes per edge row
    const uint8_t *nfeat;
    uint32_t nrb;         // bytes per node row
    int32_t *o_nbr;
    uint32_t *o_eid;
    uint32_t *o_ts;
    float *o_tenc;
    uint8_t *o_efeat;
    uint8_t *o_nfeat;
    uint8_t *o_self;
    uint32_t *status;
    // copy geometry: units per row and nlb_div_magic(units)
    uint32_t tenc_units, tenc_vec;  // tenc_vec = 4 (float4 stores) or 1
    uint64_t tenc_m;
    uint32_t e_units, e_width;
    uint64_t e_m;
    uint32_t n_units, n_width;
    uint64_t n_m;
};

template <int W> struct VecOf;
template <> struct VecOf<16> { typedef u32x4 T; };
template <> struct VecOf<8> { typedef u32x2 T; };
template <> struct VecOf<4> { typedef uint32_t T; };
// Three dwords, moved as three 4-byte accesses (which the compiler may join
// into one 12-byte access): a three-element vector type would be widened to
// 16 bytes and touch the next row's first word.
struct U32x3 {
    uint32_t x, y, z;
};
template <> struct VecOf<12> { typedef U32x3 T; };

template <typename V> __device__ __forceinline__ V unit_zero() { return V(0); }
template <> __device__ __forceinline__ U32x3 unit_zero<U32x3>() { return U32x3{0u, 0u, 0u}; }
template <typename V> __device__ __forceinline__ V unit_load(const uint8_t *p) { return *(const V *)p; }
template <> __device__ __forceinline__ U32x3 unit_load<U32x3>(const uint8_t *p) {
    const uint32_t *q = (const uint32_t *)p;
    return U32x3{q[0], q[1], q[2]};
}
template <typename V> __device__ __forceinline__ void unit_store(V v, uint8_t *p) {
    __builtin_nontemporal_store(v, (V *)p);
}
template <> __device__ __forceinline__ void unit_store<U32x3>(U32x3 v, uint8_t *p) {
    uint32_t *q = (uint32_t *)p;
    __builtin_nontemporal_store(v.x, q);
    __builtin_nontemporal_store(v.y, q + 1);
    __builtin_nontemporal_store(v.z, q + 2);
}

// Row source of output row j: the neighbour's node row (kind 0), the
// link's row (kind 1) or the query node's row (kind 2).
enum RowKind { kRowNeighbour = 0, kRowLink = 1, kRowSelf = 2 };

// A thread's (row, column) in a tile's flattened range, advanced by
// kTileThreads units per step without a division: with
// kTileThreads = dq units + dr (dr < units), a step adds dq rows and dr
// columns and carries at most one row.
struct RowCursor {
    uint32_t j, c;
    __device__ __forceinline__ RowCursor(uint32_t f, uint32_t units, uint64_t m) {
        j = nlb_div(f, m);
        c = f - j * units;
    }
    __device__ __forceinline__ void step(uint32_t units, uint32_t dq, uint32_t dr) {
        c += dr;
        j += dq;
        const bool carry = c >= units;
        c = carry ? c - units : c;
        j += carry ? 1u : 0u;
    }
};

// Copy `rows` output rows of `row_bytes` each, laid out contiguously at
// `out`, from their source rows; unit f of the flattened range is
// (row f / units, column f % units).  R loads per thread are issued before
// their stores.  Rows without a valid source are written as zeros.
template <int W, int KIND>
__device__ __forceinline__ void gather_tile(const uint8_t *__restrict__ src, uint32_t row_bytes,
                                            uint32_t units, uint64_t m, uint32_t rows,
                                            int64_t src_rows, const SlotLds *slots,
                                            const int32_t *tile_nodes, uint8_t *__restrict__ out,
                                            uint32_t tid) {
    typedef typename VecOf<W>::T V;
    constexpr int R = (W == 16) ? 4 : (W == 4 ? 8 : 6);
    const uint32_t total = rows * units;
    const uint32_t dq = nlb_div(kTileThreads, m), dr = kTileThreads - dq * units;
    RowCursor cur(tid, units, m);
    for (uint32_t base = 0; base < total; base += kTileThreads * R) {
        V val[R];
#pragma unroll
        for (int r = 0; r < R; r++) {
            const uint32_t f = base + r * kTileThreads + tid;
            const uint32_t j = cur.j, c = cur.c;
            cur.step(units, dq, dr);
            val[r] = unit_zero<V>();
            if (f < total) {
                int64_t row;
                if (KIND == kRowSelf) {
                    row = tile_nodes[j];
                } else {
                    const SlotLds sl = slots[j];
                    row = (sl.x < 0) ? -1 : (KIND == kRowNeighbour ? (int64_t)sl.x : (int64_t)sl.e);
                }
                if (row >= 0 && row < src_rows)
                    val[r] = unit_load<V>(src + (size_t)row * row_bytes + (size_t)c * W);
            }
        }
#pragma unroll
        for (int r = 0; r < R; r++) {
            const uint32_t f = base + r * kTileThreads + tid;
            if (f < total) unit_store<V>(val[r], out + (size_t)f * W);
        }
    }
}

template <int KIND>
__device__ __forceinline__ void gather_tile_w(uint32_t width, const uint8_t *src, uint32_t row_bytes,
                                              uint32_t units, uint64_t m, uint32_t rows,
                                              int64_t src_rows, const SlotLds *slots,
                                              const int32_t *tile_nodes, uint8_t *out,
                                              uint32_t tid) {
    if (width == 16)
        gather_tile<16, KIND>(src, row_bytes, units, m, rows, src_rows, slots, tile_nodes, out, tid);
    else if (width == 12)
        gather_tile<12, KIND>(src, row_bytes, units, m, rows, src_rows, slots, tile_nodes, out, tid);
    else if (width == 8)
        gather_tile<8, KIND>(src, row_bytes, units, m, rows, src_rows, slots, tile_nodes, out, tid);
    else
        gather_tile<4, KIND>(src, row_bytes, units, m, rows, src_rows, slots, tile_nodes, out, tid);
}

// HOP2: query i is (node[i], tq[i / s]) and a negative node is an empty
// answer (second-hop retrieval over first-hop outputs).
template <bool HOP2>
__global__ __launch_bounds__(kTileThreads) void sample_gather(SampleParams p) {
    __shared__ SlotLds slots[kTileSlots];
    __shared__ int32_t tile_nodes[kTileSlots];
    const uint32_t tid = threadIdx.x;
    const uint64_t q0 = (uint64_t)blockIdx.x * p.tile_q;
    const uint32_t nqt = (uint32_t)min((uint64_t)p.tile_q, (uint64_t)p.nq - q0);
    const uint32_t s = p.s;
    const uint32_t ns = nqt * s;                 // slot rows of this tile
    const size_t row0 = (size_t)q0 * s;          // first output slot row

    // Phase 1: table read, strict mask (eq. (1)), id outputs, LDS staging.
    // A thread's slot rows (at most kTileSlots / kTileThreads) are read in
    // two rounds of unconditional loads -- the query ids and times, then
    // the slot words (an out-of-range node or a row past the tile reads
    // slot 0 of node 0, which exists) -- before any is used.
    constexpr int P1 = kTileSlots / kTileThreads;
    static_assert(kTileSlots <= 4096 && NLB_MAX_SLOTS <= 4096, "slot rows of a tile split by nlb_div12");
    // Query and slot of each of the thread's rows (rows past the tile take
    // the tile's last row).
    uint32_t qlv[P1], av[P1];
#pragma unroll
    for (int r = 0; r < P1; r++) {
        const uint32_t j = min(tid + r * kTileThreads, ns - 1u);
        qlv[r] = nlb_div12(j, p.s_m);
        av[r] = j - qlv[r] * s;
    }
    int32_t nd[P1];
    uint32_t tqv[P1];
#pragma unroll
    for (int r = 0; r < P1; r++) {
        const uint64_t qg = q0 + qlv[r];
        nd[r] = p.node[qg];
        tqv[r] = p.tq[HOP2 ? (uint32_t)qg / s : qg];
    }
    uint64_t key[P1];
    int32_t xv[P1];
#pragma unroll
    for (int r = 0; r < P1; r++) {
        const uint32_t a = av[r];
        const bool in_range = nd[r] >= 0 && (int64_t)nd[r] < p.num_nodes;
        const uint8_t *bp = p.blocks + (size_t)(in_range ? nd[r] : 0) * p.block_bytes;
        const uint32_t aa = in_range ? a : 0u;
        key[r] = ((const uint64_t *)bp)[aa];
        xv[r] = ((const int32_t *)(bp + 8u * s))[aa];
    }
#pragma unroll
    for (int r = 0; r < P1; r++) {
        const uint32_t j = tid + r * kTileThreads;
        if (j >= ns) break;
        const uint32_t ql = qlv[r], a = av[r];
        const int32_t node = nd[r];
        const bool in_range = node >= 0 && (int64_t)node < p.num_nodes;
        const bool quiet = HOP2 && node < 0;   // empty first-hop slot
        const SlotLds sl = decode_slot(in_range ? key[r] : 0ull, xv[r], tqv[r]);
        if (!in_range && a == 0 && !quiet) atomicOr(p.status, kStatusRange);
        if (a == 0) tile_nodes[ql] = in_range ? node : -1;
        slots[j] = sl;
        if (p.o_nbr) p.o_nbr[row0 + j] = sl.x;
        if (p.o_eid) p.o_eid[row0 + j] = sl.e;
        if (p.o_ts) p.o_ts[row0 + j] = sl.t;
    }
    __syncthreads();

    // Phase 2: T-encoding (App. C): cos(w_k * dt + b_k), the argument formed
    // by one fp32 fused multiply-add; zeros on invalid slots.
    if (p.o_tenc) {
        const uint32_t units = p.tenc_units;
        const uint32_t total = ns * units;
        float *out = p.o_tenc + row0 * p.d_time;
        const uint32_t dq = nlb_div(kTileThreads, p.tenc_m), dr = kTileThreads - dq * units;
        RowCursor cur(tid, units, p.tenc_m);
        for (uint32_t f = tid; f < total; f += kTileThreads) {
            const uint32_t j = cur.j, c = cur.c;
            cur.step(units, dq, dr);
            const SlotLds sl = slots[j];
            if (p.tenc_vec == 4) {
                f32x4 r = f32x4(0.0f);
                if (sl.x >= 0) {
                    const f32x4 w4 = *(const f32x4 *)(p.w + 4 * c);
                    const f32x4 b4 = *(const f32x4 *)(p.b + 4 * c);
                    r.x = cos_fp32(__builtin_fmaf(w4.x, sl.dt, b4.x));
                    r.y = cos_fp32(__builtin_fmaf(w4.y, sl.dt, b4.y));
                    r.z = cos_fp32(__builtin_fmaf(w4.z, sl.dt, b4.z));
                    r.w = cos_fp32(__builtin_fmaf(w4.w, sl.dt, b4.w));
                }
                __builtin_nontemporal_store(r, (f32x4 *)(out + (size_t)f * 4));
            } else {
                float r = 0.0f;
                if (sl.x >= 0) r = cos_fp32(__builtin_fmaf(p.w[c], sl.dt, p.b[c]));
                __builtin_nontemporal_store(r, out + f);
            }
        }
    }
    // Phase 3-5: row gathers (Sec. 4.4: link features, neighbour status, self).
    if (p.o_efeat)
        gather_tile_w<kRowLink>(p.e_width, p.efeat, p.erb, p.e_units, p.e_m, ns, p.edge_rows, slots,
                                tile_nodes, p.o_efeat + row0 * p.erb, tid);
    if (p.o_nfeat)
        gather_tile_w<kRowNeighbour>(p.n_width, p.nfeat, p.nrb, p.n_units, p.n_m, ns, p.num_nodes,
                                     slots, tile_nodes, p.o_nfeat + row0 * p.nrb, tid);
    if (p.o_self)
        gather_tile_w<kRowSelf>(p.n_width, p.nfeat, p.nrb, p.n_units, p.n_m, nqt, p.num_nodes, slots,
                                tile_nodes, p.o_self + q0 * p.nrb, tid);
}

// Time encoding as its own stream, computed from an answer's timestamp output
// (the large first-hop launches of nlb_sample, and nlb_time_encode).  A
// tile-looping kernel's write streams reach about 5 TB/s on gfx950, short
// workgroups with one 16-byte store per thread the fill rate (~6.9 TB/s);
// here each thread of a 128-thread workgroup computes two outputs of V
// floats (kTencPerThread) whose timestamp and query-time reads are issued
// together, so one read latency covers two stores.  Slot row j = f / units
// belongs to query j / s; ts[j] = 0xFFFFFFFF marks an invalid slot (zeros).
// Both divisions are nlb_div (exact for every 32-bit numerator and divisor,
// 1 included).  V = 4 needs d_time % 4 == 0 and 16-byte aligned w, b and
// output; V = 1 takes any width and 4-byte alignment.
constexpr uint32_t kTencThreads = 128, kTencPerThread = 2;

template <uint32_t V>
__global__ __launch_bounds__(kTencThreads) void tenc_stream(const uint32_t *ts, const uint32_t *tq, uint64_t s_M,
                                                            uint32_t units, uint64_t u_M, uint32_t total,
                                                            const float *w, const float *b, float *out) {
    uint32_t t[kTencPerThread], q[kTencPerThread], cc[kTencPerThread], ff[kTencPerThread];
#pragma unroll
    for (uint32_t k = 0; k < kTencPerThread; k++) {
        ff[k] = (blockIdx.x * kTencPerThread + k) * kTencThreads + threadIdx.x;
        const uint32_t f = min(ff[k], total - 1u);   // past the end: re-read the last (unused)
        const uint32_t j = nlb_div(f, u_M);
        cc[k] = f - j * units;
        t[k] = ts[j];
        q[k] = tq[nlb_div(j, s_M)];
    }
#pragma unroll
    for (uint32_t k = 0; k < kTencPerThread; k++) {
        if constexpr (V == 4) {
            f32x4 r = f32x4(0.0f);
            if (t[k] != 0xFFFFFFFFu) {
                const float dt = (float)(q[k] - t[k]);
                const f32x4 w4 = *(const f32x4 *)(w + 4 * cc[k]);
                const f32x4 b4 = *(const f32x4 *)(b + 4 * cc[k]);
                r.x = cos_fp32(__builtin_fmaf(w4.x, dt, b4.x));
                r.y = cos_fp32(__builtin_fmaf(w4.y, dt, b4.y));
                r.z = cos_fp32(__builtin_fmaf(w4.z, dt, b4.z));
                r.w = cos_fp32(__builtin_fmaf(w4.w, dt, b4.w));
            }
            if (ff[k] < total) __builtin_nontemporal_store(r, (f32x4 *)(out + (size_t)ff[k] * 4));
        } else {
            float r = 0.0f;
            if (t[k] != 0xFFFFFFFFu) r = cos_fp32(__builtin_fmaf(w[cc[k]], (float)(q[k] - t[k]), b[cc[k]]));
            if (ff[k] < total) __builtin_nontemporal_store(r, out + ff[k]);
        }
    }
}

// ---------------------------------------------------------------- export
__global__ __launch_bounds__(256) void export_table(const uint8_t *blocks, uint32_t block_bytes,
                                                    uint32_t s, int64_t num_nodes, int32_t *nbr,
                                                    uint32_t *ts, uint32_t *eid) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (n >= num_nodes) return;
    const uint8_t *blk = blocks + (size_t)n * block_bytes;
    const uint64_t *keys = (const uint64_t *)blk;
    const int32_t *nb = (const int32_t *)(blk + 8u * s);
    for (uint32_t a = 0; a < s; a++) {
        const uint64_t key = keys[a];
        const size_t o = (size_t)n * s + a;
        if (key == 0) {
            nbr[o] = -1;
            ts[o] = 0xFFFFFFFFu;
            eid[o] = 0xFFFFFFFFu;
        } else {
            const uint32_t ef = (uint32_t)(key >> kTimeBits);
            nbr[o] = nb[a];
            ts[o] = (uint32_t)key & kTimeMask;
            eid[o] = ((key >> 62) == 3u) ? ef : ~ef;
        }
    }
}

// ---------------------------------------------------------------- host side
uint32_t block_bytes_for(uint32_t s) {
    const uint32_t need = 12u * s;
    if (need <= 128) {
        uint32_t b = 16;
        while (b < need) b *= 2;
        return b;
    }
    return (need + 127u) / 128u * 128u;
}

// Copy unit of the sample's row gathers: copy_width's 16 or 8 bytes, else 12
// for rows of a multiple of 12 bytes (e.g. 186 bf16 values), else 4.
uint32_t row_copy_width(uint32_t row_bytes, const void *src, const void *dst_or_null) {
    const uint32_t w = copy_width(row_bytes, src, dst_or_null);
    return w == 4 && row_bytes % 12 == 0 ? 12u : w;
}

// Queries per sample tile.  Large launches use as many queries as fit
// kTileSlots slot rows; smaller ones shrink the tile until the launch has
// about kTargetTiles workgroups, so that every CU gets work.  Tiles of 32
// queries or more are a multiple of 16, so they start on whole cache lines
// of every output array.
constexpr uint32_t kTargetTiles = 4096;
constexpr uint64_t kTencStreamMin = 1u << 20;   // float4 outputs from which tenc_stream is used

uint32_t tile_queries(uint32_t s, uint32_t nq) {
    uint32_t cap = kTileSlots / s;
    if (cap >= 32) cap = cap / 16 * 16;
    if (cap < 1) cap = 1;
    uint32_t want = (uint32_t)(((uint64_t)nq + kTargetTiles - 1) / kTargetTiles);
    if (want >= 32) want = (want + 15) / 16 * 16;
    if (want < 1) want = 1;
    return want < cap ? want : cap;
}

// The time encoding of nq answered queries from their timestamp output
// [nq][s] into tenc [nq][s][d_time], in launches of fewer than 2^31 output
// units (whole queries each; s * d_time < 2^31 by the limits of nlb_create).
bool launch_tenc(const nlb_table *h, const uint32_t *ts, const uint32_t *tq, uint32_t nq, float *tenc,
                 bool vec4, hipStream_t st) {
    const uint32_t units = vec4 ? h->d_time / 4 : h->d_time;
    const uint64_t per_q = (uint64_t)h->s * units;
    const uint64_t chunk = ((1ull << 31) - 1) / per_q;
    const uint64_t sM = nlb_div_magic(h->s), uM = nlb_div_magic(units);
    constexpr uint32_t kPerBlock = kTencThreads * kTencPerThread;
    for (uint64_t q0 = 0; q0 < nq; q0 += chunk) {
        const uint64_t n = nq - q0 < chunk ? nq - q0 : chunk;
        const uint32_t total = (uint32_t)(n * per_q);
        const dim3 grid((total + kPerBlock - 1) / kPerBlock);
        const uint32_t *t = ts + q0 * h->s;
        float *o = tenc + q0 * h->s * h->d_time;
        if (vec4)
            hipLaunchKernelGGL(tenc_stream<4>, grid, dim3(kTencThreads), 0, st, t, tq + q0, sM, units, uM,
                               total, h->w, h->b, o);
        else
            hipLaunchKernelGGL(tenc_stream<1>, grid, dim3(kTencThreads), 0, st, t, tq + q0, sM, units, uM,
                               total, h->w, h->b, o);
    }
    return hipGetLastError() == hipSuccess;
}

}  // namespace

extern "C" {

const char *nlb_strerror(int code) {
    switch (code) {
        case NLB_OK: return "success";
        case NLB_EINVAL: return "invalid argument";
        case NLB_ENOMEM: return "out of device memory";
        case NLB_EDEVICE: return "no usable GPU or HIP failure";
        case NLB_EORDER: return "timestamp out of order or >= 2^30";
        case NLB_ERANGE: return "node id or arrival index out of range";
        case NLB_ESCRATCH: return "working memory beyond the static array of the allocation-free call";
        default: return "unknown error";
    }
}

int nlb_create(const nlb_config *cfg, nlb_table **out) {
    if (!cfg || !out) return NLB_EINVAL;
    if (cfg->num_nodes < 1 || cfg->num_nodes > INT32_MAX) return NLB_EINVAL;
    if (cfg->s < 1 || cfg->s > NLB_MAX_SLOTS) return NLB_EINVAL;
    if (cfg->key_mode != NLB_KEY_EDGE && cfg->key_mode != NLB_KEY_NODE) return NLB_EINVAL;
    if (!(cfg->alpha > 0.0 && cfg->alpha <= 1.0)) return NLB_EINVAL;
    const uint64_t q1 = cfg->q1 ? cfg->q1 : 1000000007ull;
    const uint64_t q2 = cfg->q2 ? cfg->q2 : 998244353ull;
    if (q1 >= (1ull << 31) || q2 >= (1ull << 31)) return NLB_EINVAL;
    if (cfg->d_time < 0 || cfg->d_time > 65535) return NLB_EINVAL;
    if (cfg->d_time > 0 && (!cfg->time_w || !cfg->time_b)) return NLB_EINVAL;
    const bool has_e = cfg->edge_feat != nullptr;
    const bool has_n = cfg->node_feat != nullptr;
    if (has_e != (cfg->edge_row_bytes > 0) || has_n != (cfg->node_row_bytes > 0)) return NLB_EINVAL;
    if (cfg->edge_row_bytes < 0 || cfg->node_row_bytes < 0) return NLB_EINVAL;
    if (cfg->edge_row_bytes % 4 || cfg->node_row_bytes % 4) return NLB_EINVAL;
    if (cfg->edge_row_bytes > (1 << 18) || cfg->node_row_bytes > (1 << 18)) return NLB_EINVAL;
    if (has_e && cfg->edge_rows < 1) return NLB_EINVAL;
    if ((uintptr_t)cfg->edge_feat % 4 || (uintptr_t)cfg->node_feat % 4) return NLB_EINVAL;

    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return NLB_EDEVICE;
    int dev = cfg->device;
    if (dev < 0 && hipGetDevice(&dev) != hipSuccess) return NLB_EDEVICE;
    if (dev >= ndev) return NLB_EINVAL;
    DeviceGuard guard(dev);
    if (!guard.ok()) return NLB_EDEVICE;

    nlb_table *h = new (std::nothrow) nlb_table();
    if (!h) return NLB_ENOMEM;
    h->device = dev;
    h->num_nodes = cfg->num_nodes;
    h->s = (uint32_t)cfg->s;
    h->key_mode = cfg->key_mode;
    h->alpha = cfg->alpha;
    h->thr = (cfg->alpha >= 1.0) ? (1ull << 32) : (uint64_t)std::floor(cfg->alpha * 4294967296.0);
    h->seed = cfg->seed;
    h->q1 = q1;
    h->q2 = q2;
    h->d_time = (uint32_t)cfg->d_time;
    h->w = cfg->time_w;
    h->b = cfg->time_b;
    h->efeat = (const uint8_t *)cfg->edge_feat;
    h->edge_rows = has_e ? cfg->edge_rows : 0;
    h->erb = (uint32_t)cfg->edge_row_bytes;
    h->nfeat = (const uint8_t *)cfg->node_feat;
    h->nrb = (uint32_t)cfg->node_row_bytes;
    h->block_bytes = block_bytes_for(h->s);
    const size_t blocks_bytes = (size_t)h->num_nodes * h->block_bytes;
    h->table_bytes = blocks_bytes + kStatusBytes;
    if (hipMalloc((void **)&h->blocks, h->table_bytes) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return NLB_ENOMEM;
    }
    if (hipMemset(h->blocks, 0, h->table_bytes) != hipSuccess) {
        (void)hipFree(h->blocks);
        delete h;
        return NLB_EDEVICE;
    }
    h->status = (uint32_t *)(h->blocks + blocks_bytes);
    *out = h;
    return NLB_OK;
}

int nlb_destroy(nlb_table *h) {
    if (!h) return NLB_OK;
    int rc = NLB_OK;
    {
        DeviceGuard guard(h->device);
        if (hipDeviceSynchronize() != hipSuccess) rc = NLB_EDEVICE;
        if (hipFree(h->blocks) != hipSuccess) rc = NLB_EDEVICE;
        if (h->rnn_winner && hipFree(h->rnn_winner) != hipSuccess) rc = NLB_EDEVICE;
        if (h->rnn_cand && hipFree(h->rnn_cand) != hipSuccess) rc = NLB_EDEVICE;
        if (h->rnn_list && hipFree(h->rnn_list) != hipSuccess) rc = NLB_EDEVICE;
    }
    delete h;
    return rc;
}

int nlb_get_info(const nlb_table *h, nlb_info *info) {
    if (!h || !info) return NLB_EINVAL;
    info->num_nodes = h->num_nodes;
    info->s = (int32_t)h->s;
    info->key_mode = h->key_mode;
    info->threshold = h->thr;
    info->q1 = h->q1;
    info->q2 = h->q2;
    info->interactions = h->interactions;
    info->table_bytes = (int64_t)h->table_bytes;
    info->block_bytes = (int32_t)h->block_bytes;
    info->device = h->device;
    info->rnn_form = h->rnn_form;
    return NLB_OK;
}

int nlb_insert_batch(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t,
                     uint32_t n, void *stream) {
    if (!h) return NLB_EINVAL;
    if (n == 0) return NLB_OK;
    if (!src || !dst || !t) return NLB_EINVAL;
    // link and thread indices of the kernels are 32-bit
    if (n >= (1u << 31)) return NLB_EINVAL;
    // (the kernels make the same test on the device count, for replays)
    if (h->interactions + n > 0xFFFFFFFFull) return NLB_ERANGE;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;
    InsertParams p;
    p.src = src;
    p.dst = dst;
    p.t = t;
    p.n = n;
    p.blocks = h->blocks;
    p.block_bytes = h->block_bytes;
    p.s = h->s;
    p.num_nodes = h->num_nodes;
    p.seed = h->seed;
    p.thr = h->thr;
    p.mod_m = nlb_mod_magic(h->s);
    p.q1r = (uint32_t)(h->q1 % h->s);
    p.q2r = (uint32_t)(h->q2 % h->s);
    p.key_mode = (uint32_t)h->key_mode;
    p.status = h->status;
    const hipStream_t st = (hipStream_t)stream;
    if (n >= kMergeMinBatch)
        hipLaunchKernelGGL(insert_resolve_merged, dim3((n + kResolveLinks - 1) / kResolveLinks),
                           dim3(kMergeThreads), 0, st, p);
    else
        hipLaunchKernelGGL(insert_resolve, dim3((n + kInsertThreads - 1) / kInsertThreads),
                           dim3(kInsertThreads), 0, st, p);
    hipLaunchKernelGGL(insert_commit, dim3((n + kInsertThreads - 1) / kInsertThreads),
                       dim3(kInsertThreads), 0, st, p);
    if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
    h->interactions += n;
    return NLB_OK;
}

static int launch_sample(nlb_table *h, const int32_t *node, const uint32_t *tq, uint32_t nq,
                         uint32_t hop2, const nlb_sample_out *out, void *stream) {
    if (out->tenc && h->d_time == 0) return NLB_EINVAL;
    if (out->efeat && !h->efeat) return NLB_EINVAL;
    if ((out->nfeat || out->self) && !h->nfeat) return NLB_EINVAL;
    if ((uintptr_t)out->nbr % 4 || (uintptr_t)out->eid % 4 || (uintptr_t)out->ts % 4 ||
        (uintptr_t)out->tenc % 4 || (uintptr_t)out->efeat % 4 || (uintptr_t)out->nfeat % 4 ||
        (uintptr_t)out->self % 4)
        return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;
    SampleParams p;
    p.blocks = h->blocks;
    p.block_bytes = h->block_bytes;
    p.s = h->s;
    p.num_nodes = h->num_nodes;
    p.node = node;
    p.tq = tq;
    p.nq = nq;
    p.d_time = h->d_time;
    p.w = h->w;
    p.b = h->b;
    p.efeat = h->efeat;
    p.edge_rows = h->edge_rows;
    p.erb = h->erb;
    p.nfeat = h->nfeat;
    p.nrb = h->nrb;
    p.o_nbr = out->nbr;
    p.o_eid = out->eid;
    p.o_ts = out->ts;
    p.o_tenc = out->tenc;
    p.o_efeat = (uint8_t *)out->efeat;
    p.o_nfeat = (uint8_t *)out->nfeat;
    p.o_self = (uint8_t *)out->self;
    p.status = h->status;
    const bool vec4 = h->d_time % 4 == 0 && (uintptr_t)out->tenc % 16 == 0 &&
                      (uintptr_t)h->w % 16 == 0 && (uintptr_t)h->b % 16 == 0;
    p.tenc_vec = vec4 ? 4 : 1;
    p.tenc_units = h->d_time ? (vec4 ? h->d_time / 4 : h->d_time) : 1;
    p.tenc_m = nlb_div_magic(p.tenc_units);
    p.e_width = h->erb ? row_copy_width(h->erb, h->efeat, out->efeat) : 4;
    p.e_units = h->erb ? h->erb / p.e_width : 1;
    p.e_m = nlb_div_magic(p.e_units);
    // the same width serves the neighbour rows and the self row
    const uintptr_t nalign = (uintptr_t)out->nfeat | (uintptr_t)out->self;
    p.n_width = h->nrb ? row_copy_width(h->nrb, h->nfeat, (const void *)nalign) : 4;
    p.n_units = h->nrb ? h->nrb / p.n_width : 1;
    p.n_m = nlb_div_magic(p.n_units);
    p.tile_q = tile_queries(h->s, nq);
    p.s_m = nlb_div12_magic(h->s);
    const hipStream_t st = (hipStream_t)stream;
    const dim3 grid((unsigned)(((uint64_t)nq + p.tile_q - 1) / p.tile_q));
    // Large first-hop launches that also write timestamps take the time
    // encoding out of sample_gather into tenc_stream.
    const uint64_t tenc_total = (uint64_t)nq * h->s * p.tenc_units;
    const bool split = !hop2 && out->tenc && out->ts && vec4 && tenc_total >= kTencStreamMin;
    if (split) p.o_tenc = nullptr;
    if (hop2)
        hipLaunchKernelGGL(sample_gather<true>, grid, dim3(kTileThreads), 0, st, p);
    else
        hipLaunchKernelGGL(sample_gather<false>, grid, dim3(kTileThreads), 0, st, p);
    if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
    if (split && !launch_tenc(h, out->ts, tq, nq, out->tenc, true, st)) return NLB_EDEVICE;
    return NLB_OK;
}

int nlb_sample(nlb_table *h, const int32_t *node, const uint32_t *tq, uint32_t nq,
               const nlb_sample_out *out, void *stream) {
    if (!h || !out) return NLB_EINVAL;
    if (nq == 0) return NLB_OK;
    if (!node || !tq) return NLB_EINVAL;
    return launch_sample(h, node, tq, nq, 0, out, stream);
}

int nlb_time_encode(nlb_table *h, const uint32_t *ts, const uint32_t *tq, uint32_t nq, float *tenc,
                    void *stream) {
    if (!h) return NLB_EINVAL;
    if (nq == 0) return NLB_OK;
    if (!ts || !tq || !tenc || h->d_time == 0) return NLB_EINVAL;
    if ((uintptr_t)ts % 4 || (uintptr_t)tq % 4 || (uintptr_t)tenc % 4) return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;
    const bool vec4 = h->d_time % 4 == 0 && (uintptr_t)tenc % 16 == 0 && (uintptr_t)h->w % 16 == 0 &&
                      (uintptr_t)h->b % 16 == 0;
    return launch_tenc(h, ts, tq, nq, tenc, vec4, (hipStream_t)stream) ? NLB_OK : NLB_EDEVICE;
}

int nlb_sample_hop2(nlb_table *h, const int32_t *hop1_nbr, const uint32_t *tq, uint32_t nq,
                    const nlb_sample_out *out, void *stream) {
    if (!h || !out) return NLB_EINVAL;
    if (nq == 0) return NLB_OK;
    if (!hop1_nbr || !tq) return NLB_EINVAL;
    if ((uint64_t)nq * h->s > 0xFFFFFFFFull) return NLB_EINVAL;
    return launch_sample(h, hop1_nbr, tq, (uint32_t)(nq * h->s), 1, out, stream);
}

int nlb_export(nlb_table *h, int32_t *nbr, uint32_t *ts, uint32_t *eid, void *stream) {
    if (!h || !nbr || !ts || !eid) return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;
    const dim3 grid((unsigned)((h->num_nodes + 255) / 256));
    hipLaunchKernelGGL(export_table, grid, dim3(256), 0, (hipStream_t)stream, h->blocks,
                       h->block_bytes, h->s, h->num_nodes, nbr, ts, eid);
    if (hipGetLastError() != hipSuccess) return NLB_EDEVICE;
    return NLB_OK;
}

int nlb_status(nlb_table *h, void *stream) {
    if (!h) return NLB_EINVAL;
    DeviceGuard guard(h->device);
    if (!guard.ok()) return NLB_EDEVICE;
    if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) return NLB_EDEVICE;
    uint32_t words[8];
    if (hipMemcpy(words, h->status, sizeof(words), hipMemcpyDeviceToHost) != hipSuccess)
        return NLB_EDEVICE;
    const uint32_t flags = words[0];
    // inserts replayed from graphs advance only the device count
    h->interactions = (uint64_t)words[kWordLinks] | ((uint64_t)words[kWordLinks + 1] << 32);
    if (flags) {
        const uint32_t zero = 0;
        if (hipMemcpy(h->status, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess)
            return NLB_EDEVICE;
    }
    if (flags & kStatusRange) return NLB_ERANGE;
    if (flags & kStatusOrder) return NLB_EORDER;
    return NLB_OK;
}

}  // extern "C"
