// synth.hip -- seeded synthetic temporal-graph streams and feature tables.
//
// Input generation only: this file holds none of the sampling method's
// arithmetic.  Every value is a counter-based function of (seed, index)
// computed with integer operations and lookups in tables built once on the
// host, so the host functions (for the CPU oracle) and the device kernels
// (to fill tens of GB in HBM) produce bit-identical data.
//
// Building blocks (all published methods):
//   - SplitMix64 output mixing (Steele, Lea & Flood, OOPSLA 2014) as the
//     counter-based generator: rnd(key, i) = mix(key + (i+1) * golden).
//   - Lemire's multiply-shift map of 32 random bits onto [0, n).
//   - Walker's alias method with Vose's linear-time construction (Vose 1991)
//     for Zipf / power-law endpoint draws.
//   - A 4-round Feistel network with cycle-walking (Black & Rogaway 2002) to
//     scatter popularity ranks over node ids.
//   - Stratified sorted timestamps: link i falls uniformly in the i-th of E
//     equal strata of [0, T), which keeps the stream sorted without a scan.
//   - Feature values: 16-bit uniforms indexing a table of standard-normal
//     quantiles (inverse-CDF sampling).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <thread>
#include <vector>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

enum Tag : uint64_t {
    kTagSrc = 1, kTagDst = 2, kTagTime = 3, kTagNeg = 4, kTagPick = 5, kTagRedraw = 6,
    kTagPerm = 7, kTagPairU = 8, kTagPairV = 9, kTagRepeat = 10, kTagFeat = 11, kTagPermB = 12,
};

__host__ __device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}
__host__ __device__ inline uint64_t subkey(uint64_t seed, uint64_t tag) {
    return mix64(seed + tag * kGolden);
}
__host__ __device__ inline uint64_t rnd(uint64_t key, uint64_t i) {
    return mix64(key + (i + 1) * kGolden);
}
__host__ __device__ inline uint32_t below(uint32_t r32, uint64_t n) {
    return (uint32_t)(((uint64_t)r32 * n) >> 32);
}

// Bijection of [0, n) (n >= 1): balanced Feistel over 2h bits, cycle-walked.
__host__ __device__ inline uint64_t permute(uint64_t x, uint64_t n, uint64_t key) {
    if (n <= 1) return 0;
    uint32_t bits = 0;
    while ((1ull << bits) < n) bits++;
    const uint32_t h = (bits + 1) / 2;
    const uint64_t mask = (1ull << h) - 1;
    do {
        uint64_t L = x >> h, R = x & mask;
        for (uint64_t r = 0; r < 4; r++) {
            const uint64_t F = mix64(key + (r + 1) * kGolden + R) & mask;
            const uint64_t nl = R;
            R = L ^ F;
            L = nl;
        }
        x = (L << h) | R;
    } while (x >= n);
    return x;
}

__host__ __device__ inline uint32_t alias_draw(uint64_t r, const uint32_t *prob,
                                               const int32_t *alias, uint64_t n) {
    const uint32_t j = below((uint32_t)(r >> 32), n);
    return ((uint32_t)r < prob[j]) ? j : (uint32_t)alias[j];
}

}  // namespace

// Stream description shared by host and device generators (plain C layout,
// mirrored by ctypes in synth/__init__.py).
struct SynStream {
    uint64_t seed;
    int64_t E;            // links in the stream
    int32_t kind;         // 0 bipartite Zipf, 1 homogeneous (alias) without self-loops,
                          // 2 fixed pair set mixed with fresh pairs
    int32_t neg_all;      // negatives over all nodes (1) or over the destination side (0)
    int64_t n_src;        // kind 0: source-side nodes (ids 0..n_src-1); else all nodes
    int64_t n_dst;        // kind 0: destination-side nodes (ids n_src..n_src+n_dst-1)
    uint64_t T;           // timestamps in [0, T)
    const uint32_t *a_prob;  // alias table of the source side / all nodes
    const int32_t *a_alias;
    const uint32_t *b_prob;  // alias table of the destination side (kind 0)
    const int32_t *b_alias;
    int64_t n_pairs;      // kind 2: size of the pair set
    uint32_t p_pair;      // kind 2: a link reuses the set with probability p_pair / 2^32
    int32_t pad;
};

__host__ __device__ inline void gen_link(const SynStream &p, int64_t i, int32_t &u, int32_t &v,
                                         uint32_t &t, int32_t &neg) {
    const uint64_t s = p.seed;
    // timestamp: uniform inside stratum i of [0, T)
    const uint64_t rt = rnd(subkey(s, kTagTime), (uint64_t)i);
    t = (uint32_t)(((uint64_t)i * p.T + (((rt >> 32) * p.T) >> 32)) / (uint64_t)p.E);
    if (p.kind == 0) {
        const uint32_t ra = alias_draw(rnd(subkey(s, kTagSrc), i), p.a_prob, p.a_alias, p.n_src);
        const uint32_t rb = alias_draw(rnd(subkey(s, kTagDst), i), p.b_prob, p.b_alias, p.n_dst);
        u = (int32_t)permute(ra, p.n_src, subkey(s, kTagPerm));
        v = (int32_t)(p.n_src + permute(rb, p.n_dst, subkey(s, kTagPermB)));
    } else if (p.kind == 1) {
        const uint64_t N = p.n_src;
        const uint32_t ra = alias_draw(rnd(subkey(s, kTagSrc), i), p.a_prob, p.a_alias, N);
        uint32_t rb = alias_draw(rnd(subkey(s, kTagDst), i), p.a_prob, p.a_alias, N);
        for (uint64_t j = 0; rb == ra && N > 1; j++)  // self-loops are redrawn (64 tries)
            rb = (j < 64) ? alias_draw(rnd(subkey(s, kTagRedraw), (uint64_t)i * 64 + j), p.a_prob,
                                       p.a_alias, N)
                          : (uint32_t)((ra + 1) % N);
        u = (int32_t)permute(ra, N, subkey(s, kTagPerm));
        v = (int32_t)permute(rb, N, subkey(s, kTagPerm));
    } else {
        const uint64_t N = p.n_src;
        const uint64_t rp = rnd(subkey(s, kTagPick), i);
        uint64_t pair_key, pair_idx;
        if ((uint32_t)rp < p.p_pair) {  // reuse one of the fixed pairs
            pair_key = subkey(s, kTagPairU);
            pair_idx = below((uint32_t)(rp >> 32), (uint64_t)p.n_pairs);
        } else {                        // a fresh pair, unique to this link
            pair_key = subkey(s, kTagPairV);
            pair_idx = (uint64_t)i;
        }
        const uint64_t r2 = rnd(pair_key, pair_idx);
        const uint32_t a = below((uint32_t)(r2 >> 32), N);
        uint32_t b = below((uint32_t)r2, N - 1);
        if (b >= a) b++;                // u != v, uniform
        u = (int32_t)a;
        v = (int32_t)b;
    }
    const uint32_t rn = (uint32_t)(rnd(subkey(s, kTagNeg), i) >> 32);
    if (p.kind == 0 && !p.neg_all)
        neg = (int32_t)(p.n_src + below(rn, p.n_dst));
    else
        neg = (int32_t)below(rn, p.kind == 0 ? p.n_src + p.n_dst : p.n_src);
}

// Position of link i in the batch-blocked query layout: batch b = i / B
// holds [src of the batch | dst of the batch | negatives of the batch].
__host__ __device__ inline void blocked_pos(int64_t i, int64_t E, int64_t B, int64_t &ps,
                                            int64_t &pd, int64_t &pn) {
    const int64_t b = i / B, o = i - b * B;
    const int64_t len = (b + 1) * B <= E ? B : E - b * B;
    const int64_t base = 3 * b * B;
    ps = base + o;
    pd = base + len + o;
    pn = base + 2 * len + o;
}

__global__ void gen_links_blocked(SynStream p, int64_t i0, int64_t i1, int64_t B, int32_t *nodes,
                                  uint32_t *ts) {
    const int64_t i = i0 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= i1) return;
    int32_t u, v, neg;
    uint32_t t;
    gen_link(p, i, u, v, t, neg);
    int64_t ps, pd, pn;
    blocked_pos(i, p.E, B, ps, pd, pn);
    nodes[ps] = u;
    nodes[pd] = v;
    nodes[pn] = neg;
    ts[ps] = t;
    ts[pd] = t;
    ts[pn] = t;
}

// Feature row r, column c: standard-normal quantile indexed by 16 random bits.
__host__ __device__ inline uint32_t feat_index(uint64_t key, uint64_t row, uint32_t d, uint32_t c) {
    const uint64_t groups = (d + 3) / 4;
    const uint64_t r = rnd(key, row * groups + c / 4);
    return (uint32_t)(r >> (16 * (c % 4))) & 0xFFFFu;
}

// One wavefront per row (grid-stride over rows); lane g writes the four
// columns 4g..4g+3 drawn from one 64-bit random word.
__global__ void fill_features(uint64_t key, int64_t rows, uint32_t d, uint32_t elem_bytes,
                              const void *table, void *out) {
    const uint32_t lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * (blockDim.x / 64);
    const uint32_t groups = (d + 3) / 4;
    for (int64_t row = (int64_t)blockIdx.x * (blockDim.x / 64) + threadIdx.x / 64; row < rows;
         row += waves) {
        for (uint32_t g = lane; g < groups; g += 64) {
            const uint64_t r = rnd(key, (uint64_t)row * groups + g);
            for (uint32_t c = 4 * g; c < 4 * g + 4 && c < d; c++) {
                const uint32_t q = (uint32_t)(r >> (16 * (c % 4))) & 0xFFFFu;
                const size_t o = (size_t)row * d + c;
                if (elem_bytes == 4)
                    ((float *)out)[o] = ((const float *)table)[q];
                else
                    ((uint16_t *)out)[o] = ((const uint16_t *)table)[q];
            }
        }
    }
}

namespace {
template <class F>
void parallel_for(int64_t n, int threads, F f) {
    if (threads <= 1 || n < 4096) {
        f(0, n);
        return;
    }
    std::vector<std::thread> pool;
    const int64_t chunk = (n + threads - 1) / threads;
    for (int k = 0; k < threads; k++) {
        const int64_t lo = k * chunk, hi = std::min(n, lo + chunk);
        if (lo >= hi) break;
        pool.emplace_back([=] { f(lo, hi); });
    }
    for (auto &th : pool) th.join();
}
}  // namespace

extern "C" {

// Alias table of weights (k+1)^-exponent, k < n (Walker/Vose).  prob[j] is
// the acceptance threshold of column j on 32 bits.
int syn_alias_powerlaw(int64_t n, double exponent, uint32_t *prob, int32_t *alias) {
    if (n < 1) return 1;
    std::vector<double> p(n);
    double total = 0.0;
    for (int64_t k = 0; k < n; k++) {
        p[k] = std::pow((double)(k + 1), -exponent);
        total += p[k];
    }
    for (int64_t k = 0; k < n; k++) p[k] = p[k] * (double)n / total;
    std::vector<int64_t> small, large;
    small.reserve(n);
    large.reserve(n);
    for (int64_t k = 0; k < n; k++) (p[k] < 1.0 ? small : large).push_back(k);
    while (!small.empty() && !large.empty()) {
        const int64_t l = small.back(); small.pop_back();
        const int64_t g = large.back(); large.pop_back();
        prob[l] = (uint32_t)std::min(std::floor(p[l] * 4294967296.0), 4294967295.0);
        alias[l] = (int32_t)g;
        p[g] = (p[g] + p[l]) - 1.0;
        (p[g] < 1.0 ? small : large).push_back(g);
    }
    for (int64_t k : large) { prob[k] = 0xFFFFFFFFu; alias[k] = (int32_t)k; }
    for (int64_t k : small) { prob[k] = 0xFFFFFFFFu; alias[k] = (int32_t)k; }
    return 0;
}

// Links [i0, i1) into plain host arrays (index i - i0).
int syn_links_host(const SynStream *p, int64_t i0, int64_t i1, int32_t *src, int32_t *dst,
                   uint32_t *t, int32_t *neg, int threads) {
    parallel_for(i1 - i0, threads, [&](int64_t lo, int64_t hi) {
        for (int64_t k = lo; k < hi; k++) gen_link(*p, i0 + k, src[k], dst[k], t[k], neg[k]);
    });
    return 0;
}

// Links [i0, i1) into device arrays in the batch-blocked query layout
// (nodes and ts each hold 3*E entries).  Pointers in *p must be device ones.
int syn_links_device(const SynStream *p, int64_t i0, int64_t i1, int64_t B, int32_t *nodes,
                     uint32_t *ts, void *stream) {
    if (i1 <= i0) return 0;
    const int64_t n = i1 - i0;
    const int threads = 256;
    const int64_t blocks = (n + threads - 1) / threads;
    hipLaunchKernelGGL(gen_links_blocked, dim3((unsigned)blocks), dim3(threads), 0,
                       (hipStream_t)stream, *p, i0, i1, B, nodes, ts);
    return hipGetLastError() == hipSuccess ? 0 : 1;
}

// Repeat rule: with probability p_rep a link's destination becomes the
// destination of a uniformly chosen earlier link of the same source (when it
// has one).  Sequential in stream order; rewrites dst in place.
int syn_apply_repeats_host(uint64_t seed, int64_t E, int64_t n_src, uint32_t p_rep,
                           const int32_t *src, int32_t *dst) {
    std::vector<int64_t> start(n_src + 1, 0), fill(n_src, 0), list(E), rank(E);
    for (int64_t i = 0; i < E; i++) start[src[i] + 1]++;
    for (int64_t k = 0; k < n_src; k++) start[k + 1] += start[k];
    for (int64_t i = 0; i < E; i++) {
        const int32_t u = src[i];
        rank[i] = fill[u];
        list[start[u] + fill[u]++] = i;
    }
    const uint64_t key = subkey(seed, kTagRepeat);
    for (int64_t i = 0; i < E; i++) {
        const uint64_t r = rnd(key, (uint64_t)i);
        if (rank[i] > 0 && (uint32_t)r < p_rep) {
            const int64_t j = list[start[src[i]] + below((uint32_t)(r >> 32), (uint64_t)rank[i])];
            dst[i] = dst[j];
        }
    }
    return 0;
}

// Bursty timestamps: a two-state Markov-modulated Poisson process.  State 0
// has mean gap m0, state 1 mean gap m1; after each link the state flips with
// probability p01 (from 0) or p10 (from 1); t_i = floor(sum of gaps).
int syn_bursty_times_host(uint64_t seed, int64_t E, double m0, double m1, double p01, double p10,
                          uint32_t *t) {
    const uint64_t key = subkey(seed, kTagTime + 100);
    double clock = 0.0;
    int state = 0;
    for (int64_t i = 0; i < E; i++) {
        const uint64_t r = rnd(key, (uint64_t)i);
        const double u = ((double)(r >> 11) + 0.5) * (1.0 / 9007199254740992.0);
        clock += -(state ? m1 : m0) * std::log(u);
        t[i] = (uint32_t)std::floor(clock);
        const double flip = (double)(uint32_t)(rnd(key ^ 0x5555555555555555ull, (uint64_t)i) >> 32) *
                            (1.0 / 4294967296.0);
        if (flip < (state ? p10 : p01)) state ^= 1;
    }
    return 0;
}

// Feature rows `rows[0..nrows)` of a [*, d] table into host memory.
int syn_features_host(uint64_t seed, const int64_t *rows, int64_t nrows, uint32_t d,
                      uint32_t elem_bytes, const void *table, void *out, int threads) {
    const uint64_t key = subkey(seed, kTagFeat);
    parallel_for(nrows, threads, [&](int64_t lo, int64_t hi) {
        for (int64_t k = lo; k < hi; k++)
            for (uint32_t c = 0; c < d; c++) {
                const uint32_t q = feat_index(key, (uint64_t)rows[k], d, c);
                const size_t o = (size_t)k * d + c;
                if (elem_bytes == 4)
                    ((float *)out)[o] = ((const float *)table)[q];
                else
                    ((uint16_t *)out)[o] = ((const uint16_t *)table)[q];
            }
    });
    return 0;
}

// The full [rows, d] table on the device (table = device quantile table).
int syn_features_device(uint64_t seed, int64_t rows, uint32_t d, uint32_t elem_bytes,
                        const void *table, void *out, void *stream) {
    const uint64_t key = subkey(seed, kTagFeat);
    const int threads = 256;
    const int64_t blocks = std::min<int64_t>((rows + 3) / 4, 1 << 16);
    hipLaunchKernelGGL(fill_features, dim3((unsigned)std::max<int64_t>(blocks, 1)), dim3(threads), 0,
                       (hipStream_t)stream, key, rows, d, elem_bytes, table, out);
    return hipGetLastError() == hipSuccess ? 0 : 1;
}

}  // extern "C"
