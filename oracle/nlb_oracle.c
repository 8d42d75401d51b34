/*
 * nlb_oracle.c -- plain, sequential CPU oracle for NLB forward recent sampling.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; it exists so that tests, the smoke check and the CPU leg of
 * the benchmark can compare the GPU path against a slow, obviously correct
 * restatement of the method.  It shares no code, header or constant table
 * with the GPU path.
 *
 * What it follows (Luo & Li, "Scalable and Efficient Temporal Graph
 * Representation Learning via Forward Recent Sampling", arXiv 2402.01964):
 *   - Sec. 3, Def. "Temporal network": a time-ordered stream of undirected
 *     links (u, v, t); the i-th link is identified here by its 0-based
 *     arrival index e.
 *   - Sec. 3, eq. (1): temporal neighbours of u at time t are the links of u
 *     with timestamp strictly below t.
 *   - Sec. 4.2: every node u owns a table S_u of s slots.  A new link
 *     (u, v, t) is offered to S_u (neighbour v) and to S_v (neighbour u).  The
 *     slot is hash(v, t) = (q1*v + q2*t) mod s for NLB-edge, eq. (2), or
 *     hash(v) = q1*v mod s for NLB-node, eq. (3).  An empty slot always takes
 *     the offer; an occupied one is overwritten with probability alpha.
 *     Tables are updated after the queries of the current batch are answered.
 *   - Sec. 4.4 and App. C: a query (u, t) returns the stored neighbours, their
 *     link features, the neighbours' own feature rows, the self row and a
 *     cosine time encoding of t - t'.  Second-hop neighbours of u are the
 *     entries of S_v^t for the stored neighbours v of u.  Eq. (4) aggregates
 *     the retrieved neighbours with attention into the representation Z_u,
 *     and an RNN updates the node statuses after each event.
 *
 * Random draws: the replacement coin of offer (e, k) (k = 0 for the S_u
 * offer, k = 1 for the S_v offer) is the high 32 bits of output number
 * 2e+k+1 of SplitMix64 (Steele, Lea & Flood, OOPSLA 2014) started from state
 * `seed`; the offer replaces an occupant when coin < floor(alpha * 2^32)
 * (alpha = 1 gives 2^32, i.e. always).
 *
 * Precision: the time encoding is cos() in double of the fp32 argument
 * fmaf(w, (float)(tq - t'), b), rounded to fp32.  Build with
 * -ffp-contract=off and without fast-math.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct orc {
    int64_t N;          /* number of nodes */
    int32_t s;          /* slots per node */
    int32_t key_mode;   /* 0: NLB-edge eq. (2); 1: NLB-node eq. (3) */
    double alpha;
    uint64_t thr;       /* floor(alpha * 2^32), 2^32 when alpha == 1 */
    uint64_t seed;
    uint64_t q1, q2;
    int32_t *row_of;    /* NULL: node n owns table row n; else the row of node n, -1 = not kept */
    uint64_t *kept;     /* with row_of: bit n set when node n's table is kept (a compact
                           membership test, so that dropped offers stay cheap) */
    int64_t rows;       /* table rows kept (N without row_of) */
    int32_t *nbr;       /* [rows*s], -1 = empty */
    uint32_t *ts;       /* [rows*s] */
    uint32_t *eid;      /* [rows*s] */
    uint64_t next_e;    /* arrival index of the next link */
} orc;

/* Table row of node n, or -1 when the oracle does not keep n's table. */
static int64_t table_row(const orc *o, int32_t n)
{
    if (n < 0 || n >= o->N) return -1;
    if (!o->row_of) return n;
    if (!((o->kept[n >> 6] >> (n & 63)) & 1u)) return -1;
    return (int64_t)o->row_of[n];
}

/* n-th output (n >= 1) of SplitMix64 whose state starts at `state0`. */
static uint64_t splitmix64_nth(uint64_t state0, uint64_t n)
{
    uint64_t z = state0 + n * 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Tables of `count` nodes (all N when nodes == NULL).  Sec. 4.2 gives every
 * node its own table, and an offer to S_u touches no other table, so
 * keeping only some nodes' tables (and dropping the offers to the others)
 * leaves the kept tables exactly as in the full structure. */
orc *orc_create_subset(int64_t N, int32_t s, double alpha, uint64_t seed,
                       uint64_t q1, uint64_t q2, int32_t key_mode,
                       const int32_t *nodes, int64_t count)
{
    if (N <= 0 || N > 2147483647 || s <= 0 || !(alpha > 0.0 && alpha <= 1.0)) return NULL;
    if (key_mode != 0 && key_mode != 1) return NULL;
    /* q1*x + q2*t must not wrap in 64 bits: x < 2^31, t < 2^32. */
    if (q1 >= (1ULL << 31) || q2 >= (1ULL << 31)) return NULL;
    orc *o = (orc *)calloc(1, sizeof(orc));
    if (!o) return NULL;
    o->N = N; o->s = s; o->key_mode = key_mode; o->alpha = alpha;
    o->seed = seed; o->q1 = q1; o->q2 = q2;
    o->thr = (alpha >= 1.0) ? (1ULL << 32) : (uint64_t)floor(alpha * 4294967296.0);
    o->rows = N;
    if (nodes) {
        o->row_of = (int32_t *)malloc((size_t)N * sizeof(int32_t));
        o->kept = (uint64_t *)calloc((size_t)(N + 63) / 64, sizeof(uint64_t));
        if (!o->row_of || !o->kept) { free(o->row_of); free(o->kept); free(o); return NULL; }
        for (int64_t n = 0; n < N; n++) o->row_of[n] = -1;
        o->rows = 0;
        for (int64_t i = 0; i < count; i++) {
            const int32_t n = nodes[i];
            if (n < 0 || n >= N) { free(o->row_of); free(o->kept); free(o); return NULL; }
            if (o->row_of[n] < 0) {
                o->row_of[n] = (int32_t)o->rows++;
                o->kept[n >> 6] |= 1ull << (n & 63);
            }
        }
    }
    size_t n = (size_t)o->rows * (size_t)s;
    o->nbr = (int32_t *)malloc((n ? n : 1) * sizeof(int32_t));
    o->ts = (uint32_t *)malloc((n ? n : 1) * sizeof(uint32_t));
    o->eid = (uint32_t *)malloc((n ? n : 1) * sizeof(uint32_t));
    if (!o->nbr || !o->ts || !o->eid) {
        free(o->nbr); free(o->ts); free(o->eid); free(o->row_of); free(o->kept); free(o);
        return NULL;
    }
    for (size_t i = 0; i < n; i++) {
        o->nbr[i] = -1; o->ts[i] = 0xFFFFFFFFu; o->eid[i] = 0xFFFFFFFFu;
    }
    return o;
}

orc *orc_create(int64_t N, int32_t s, double alpha, uint64_t seed,
                uint64_t q1, uint64_t q2, int32_t key_mode)
{
    return orc_create_subset(N, s, alpha, seed, q1, q2, key_mode, NULL, 0);
}

void orc_destroy(orc *o)
{
    if (!o) return;
    free(o->nbr); free(o->ts); free(o->eid); free(o->row_of); free(o->kept); free(o);
}

int64_t orc_rows(const orc *o) { return o->rows; }

uint64_t orc_threshold(const orc *o) { return o->thr; }
uint64_t orc_count(const orc *o) { return o->next_e; }

/* Slot of neighbour x seen at time t: eq. (2) (NLB-edge) or eq. (3) (NLB-node). */
uint32_t orc_slot(const orc *o, uint32_t x, uint32_t t)
{
    uint64_t h = (o->key_mode == 0) ? o->q1 * (uint64_t)x + o->q2 * (uint64_t)t
                                    : o->q1 * (uint64_t)x;
    return (uint32_t)(h % (uint64_t)o->s);
}

uint32_t orc_coin(const orc *o, uint64_t e, uint32_t k)
{
    return (uint32_t)(splitmix64_nth(o->seed, 2 * e + k + 1) >> 32);
}

/* One offer: neighbour x of table n, from link (e, t).  Sec. 4.2: an empty
 * slot takes it; an occupied slot is replaced with probability alpha. */
static void offer(orc *o, int32_t n, int32_t x, uint32_t t, uint64_t e, uint32_t k)
{
    const int64_t row = table_row(o, n);
    if (row < 0) return;   /* a table the oracle does not keep */
    size_t idx = (size_t)row * (size_t)o->s + orc_slot(o, (uint32_t)x, t);
    int empty = (o->nbr[idx] == -1);
    if (empty || (uint64_t)orc_coin(o, e, k) < o->thr) {
        o->nbr[idx] = x;
        o->ts[idx] = t;
        o->eid[idx] = (uint32_t)e;
    }
}

/* Insert link (u, v, t) with explicit arrival index e.  Returns 0, or -1 when
 * an endpoint is out of range (nothing is changed then). */
int orc_insert_at(orc *o, uint64_t e, int32_t u, int32_t v, uint32_t t)
{
    if (u < 0 || v < 0 || u >= o->N || v >= o->N) return -1;
    offer(o, u, v, t, e, 0);   /* S_u receives neighbour v */
    offer(o, v, u, t, e, 1);   /* S_v receives neighbour u */
    return 0;
}

/* Insert n links in stream order; their arrival indices continue the count. */
int orc_insert_batch(orc *o, const int32_t *src, const int32_t *dst,
                     const uint32_t *t, int64_t n)
{
    for (int64_t i = 0; i < n; i++) {
        if (orc_insert_at(o, o->next_e, src[i], dst[i], t[i]) != 0) return -1;
        o->next_e++;
    }
    return 0;
}

/* Insert n links whose arrival indices are given (a filtered sub-stream).
 * The indices must increase; the count afterwards is eids[n-1] + 1. */
int orc_insert_ids(orc *o, const uint64_t *eids, const int32_t *src,
                   const int32_t *dst, const uint32_t *t, int64_t n)
{
    for (int64_t i = 0; i < n; i++) {
        if (orc_insert_at(o, eids[i], src[i], dst[i], t[i]) != 0) return -1;
        o->next_e = eids[i] + 1;
    }
    return 0;
}

/* The kept tables in row order ([N][s] without a node subset). */
void orc_export(const orc *o, int32_t *nbr, uint32_t *ts, uint32_t *eid)
{
    size_t n = (size_t)o->rows * (size_t)o->s;
    memcpy(nbr, o->nbr, n * sizeof(int32_t));
    memcpy(ts, o->ts, n * sizeof(uint32_t));
    memcpy(eid, o->eid, n * sizeof(uint32_t));
}

/* Export the slots of selected nodes: outputs are [count][s].  Returns -1
 * when a node is out of range or its table is not kept. */
int orc_export_nodes(const orc *o, const int32_t *nodes, int64_t count,
                     int32_t *nbr, uint32_t *ts, uint32_t *eid)
{
    for (int64_t i = 0; i < count; i++) {
        const int64_t row = table_row(o, nodes[i]);
        if (row < 0) return -1;
        size_t src = (size_t)row * (size_t)o->s;
        size_t dst = (size_t)i * (size_t)o->s;
        memcpy(nbr + dst, o->nbr + src, (size_t)o->s * sizeof(int32_t));
        memcpy(ts + dst, o->ts + src, (size_t)o->s * sizeof(uint32_t));
        memcpy(eid + dst, o->eid + src, (size_t)o->s * sizeof(uint32_t));
    }
    return 0;
}

/* T-encoding of one time gap (App. C, with a phase b per dimension):
 * cos(w_k * dt + b_k), the argument formed in fp32 by a single fused
 * multiply-add, the cosine taken in double and rounded to fp32. */
static float tenc_value(float w, float dt, float b)
{
    float arg = fmaf(w, dt, b);
    return (float)cos((double)arg);
}

/*
 * Answer nq queries (node[i], tq[i]) from the current tables (Sec. 4.4).
 * Per query i and slot a (row-major [nq][s][...]):
 *   valid    = slot non-empty and its timestamp t' < tq   (eq. (1), strict)
 *   nbr/eid/ts = the stored entry, or -1 / 0xFFFFFFFF / 0xFFFFFFFF
 *   tenc[k]  = tenc_value(w[k], (float)(tq - t'), b[k]) for k < d_t, else 0
 *   efeat    = bytes of edge-feature row eid, else zero bytes
 *   nfeat    = bytes of node-feature row nbr, else zero bytes
 *   self     = bytes of node-feature row node[i]
 * The link-feature table holds e_rows rows; a stored link with eid >= e_rows
 * has no row there and contributes zero bytes (the paper gives every link
 * a feature vector and never meets this case; a caller that keeps only the
 * first rows gets zeros for the rest).
 * Any output pointer may be NULL.  Returns -1 on an out-of-range node (or
 * one whose table is not kept).
 */
int orc_sample(const orc *o, const int32_t *node, const uint32_t *tq, int64_t nq,
               int32_t d_t, const float *w, const float *b,
               const uint8_t *efeat, int64_t e_rows, int64_t e_row_bytes,
               const uint8_t *nfeat, int64_t n_row_bytes,
               int32_t *nbr_out, uint32_t *eid_out, uint32_t *ts_out,
               float *tenc_out, uint8_t *efeat_out, uint8_t *nfeat_out,
               uint8_t *self_out)
{
    const int64_t s = o->s;
    for (int64_t i = 0; i < nq; i++) {
        int32_t n = node[i];
        const int64_t row = table_row(o, n);
        if (row < 0) return -1;
        for (int64_t a = 0; a < s; a++) {
            size_t src = (size_t)row * (size_t)s + (size_t)a;
            size_t out = (size_t)i * (size_t)s + (size_t)a;
            int valid = (o->nbr[src] != -1) && (o->ts[src] < tq[i]);
            if (nbr_out) nbr_out[out] = valid ? o->nbr[src] : -1;
            if (eid_out) eid_out[out] = valid ? o->eid[src] : 0xFFFFFFFFu;
            if (ts_out) ts_out[out] = valid ? o->ts[src] : 0xFFFFFFFFu;
            if (tenc_out) {
                float *row = tenc_out + out * (size_t)d_t;
                if (valid) {
                    float dt = (float)(uint32_t)(tq[i] - o->ts[src]);
                    for (int32_t k = 0; k < d_t; k++) row[k] = tenc_value(w[k], dt, b[k]);
                } else {
                    for (int32_t k = 0; k < d_t; k++) row[k] = 0.0f;
                }
            }
            if (efeat_out && e_row_bytes > 0) {
                uint8_t *dst = efeat_out + out * (size_t)e_row_bytes;
                if (valid && (int64_t)o->eid[src] < e_rows)
                    memcpy(dst, efeat + (size_t)o->eid[src] * (size_t)e_row_bytes, (size_t)e_row_bytes);
                else
                    memset(dst, 0, (size_t)e_row_bytes);
            }
            if (nfeat_out && n_row_bytes > 0) {
                uint8_t *dst = nfeat_out + out * (size_t)n_row_bytes;
                if (valid)
                    memcpy(dst, nfeat + (size_t)o->nbr[src] * (size_t)n_row_bytes, (size_t)n_row_bytes);
                else
                    memset(dst, 0, (size_t)n_row_bytes);
            }
        }
        if (self_out && n_row_bytes > 0)
            memcpy(self_out + (size_t)i * (size_t)n_row_bytes,
                   nfeat + (size_t)n * (size_t)n_row_bytes, (size_t)n_row_bytes);
    }
    return 0;
}

/*
 * Second-hop retrieval (Sec. 4.4): if v is stored in S_u^t, then S_v^t holds
 * down-sampled second-hop neighbours of u.  For every first-hop entry
 * (i, a) with neighbour v = hop1_nbr[i*s + a], answer the query (v, tq[i])
 * exactly as orc_sample does, into output row i*s + a; an empty first-hop
 * entry (v = -1) gives an all-invalid answer with a zero self row.  Outputs
 * are laid out as orc_sample's for nq*s queries.
 */
int orc_sample_hop2(const orc *o, const int32_t *hop1_nbr, const uint32_t *tq, int64_t nq,
                    int32_t d_t, const float *w, const float *b,
                    const uint8_t *efeat, int64_t e_rows, int64_t e_row_bytes,
                    const uint8_t *nfeat, int64_t n_row_bytes,
                    int32_t *nbr_out, uint32_t *eid_out, uint32_t *ts_out,
                    float *tenc_out, uint8_t *efeat_out, uint8_t *nfeat_out,
                    uint8_t *self_out)
{
    const int64_t s = o->s;
    for (int64_t i = 0; i < nq; i++) {
        for (int64_t a = 0; a < s; a++) {
            const int64_t r = i * s + a;         /* second-hop query index */
            const int32_t v = hop1_nbr[r];
            if (v >= 0) {
                int rc = orc_sample(o, &v, &tq[i], 1, d_t, w, b, efeat, e_rows, e_row_bytes, nfeat,
                                    n_row_bytes,
                                    nbr_out ? nbr_out + r * s : NULL,
                                    eid_out ? eid_out + r * s : NULL,
                                    ts_out ? ts_out + r * s : NULL,
                                    tenc_out ? tenc_out + r * s * d_t : NULL,
                                    efeat_out ? efeat_out + r * s * e_row_bytes : NULL,
                                    nfeat_out ? nfeat_out + r * s * n_row_bytes : NULL,
                                    self_out ? self_out + r * n_row_bytes : NULL);
                if (rc != 0) return rc;
                continue;
            }
            for (int64_t c = 0; c < s; c++) {
                const int64_t out = r * s + c;
                if (nbr_out) nbr_out[out] = -1;
                if (eid_out) eid_out[out] = 0xFFFFFFFFu;
                if (ts_out) ts_out[out] = 0xFFFFFFFFu;
                if (tenc_out) memset(tenc_out + out * d_t, 0, (size_t)d_t * sizeof(float));
                if (efeat_out && e_row_bytes > 0)
                    memset(efeat_out + out * e_row_bytes, 0, (size_t)e_row_bytes);
                if (nfeat_out && n_row_bytes > 0)
                    memset(nfeat_out + out * n_row_bytes, 0, (size_t)n_row_bytes);
            }
            if (self_out && n_row_bytes > 0) memset(self_out + r * n_row_bytes, 0, (size_t)n_row_bytes);
        }
    }
    return 0;
}

/* Value of element c of a feature row stored as fp32 (dtype 0) or bf16 (1). */
static double feat_value(const uint8_t *row, int32_t dtype, int64_t c)
{
    if (dtype == 0) {
        float f;
        memcpy(&f, row + 4 * c, 4);
        return (double)f;
    }
    uint16_t h;
    memcpy(&h, row + 2 * c, 2);
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double bf16_value(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static int64_t pad32(int64_t d) { return (d + 31) / 32 * 32; }

/* out[j] = sum_k W[j][col0 + k] * x[k] + bias[j], j < rows, k < n (W: bf16 with
 * row length ld). */
static void affine(const uint16_t *W, int64_t ld, int64_t col0, const float *bias,
                   const double *x, int64_t n, int64_t rows, double *out)
{
    for (int64_t j = 0; j < rows; j++) {
        double acc = 0.0;
        for (int64_t k = 0; k < n; k++) acc += bf16_value(W[j * ld + col0 + k]) * x[k];
        out[j] = acc + (double)bias[j];
    }
}

/*
 * Attention aggregation of eq. (4) (Sec. 4.4), forward, in double:
 *   Z_u = MLP_out(r_u, sum_i alpha_i MLP_in(r_v, e, t')),
 *   {alpha_i} = softmax({w^T MLP_in(r_v, e, t')}) over the valid slots of S_u^t,
 * with MLP(x) = W_b ReLU(W_a x + b_a) + b_b.  The neighbour status r_v is its
 * node-feature row, e the stored link's feature row and t' enters through the
 * T-encoding of tq - t' (as in orc_sample); r_u is the query node's row.
 * A query with no valid slot aggregates the zero vector.
 * Weights are bf16 (uint16 bits) in row-major [H][K] layouts whose input
 * segments are each zero-padded to a multiple of 32 columns:
 *   w1: [H][pad32(n_dim) + pad32(e_dim) + pad32(d_t)]  (r_v | e | T-enc)
 *   w2: [H][H]; w3: [H][pad32(n_dim) + H]  (r_u | aggregate); w4: [H][H]
 * Biases and att (the vector w) are fp32 [H].  Feature dtypes: 0 fp32, 1 bf16.
 * A stored link with eid >= e_rows has no link-feature row: its e is zero
 * (as in orc_sample).  z_out is [nq][H].
 * Attention heads (the experiments use two, App. E): with `heads` = A, the
 * H outputs of MLP_in are split into A consecutive slices of H / A; head a
 * scores slot i with w[slice a] . MLP_in(...)_i[slice a], takes its own
 * softmax over the valid slots, and fills slice a of the aggregate with
 * its weighted sum of slice a of the messages.  A = 1 is the formula above.
 * Returns -1 on an out-of-range query node, -2 when A does not divide H.
 */
int orc_aggregate(const orc *o, const int32_t *node, const uint32_t *tq, int64_t nq,
                  int32_t d_t, const float *w, const float *b,
                  const uint8_t *efeat, int64_t e_rows, int32_t e_dim, int32_t e_dtype,
                  const uint8_t *nfeat, int32_t n_dim, int32_t n_dtype,
                  int32_t H, int32_t heads, const uint16_t *w1, const float *b1, const uint16_t *w2,
                  const float *b2, const float *att, const uint16_t *w3, const float *b3,
                  const uint16_t *w4, const float *b4, double *z_out)
{
    if (heads < 1 || H % heads != 0) return -2;
    const int64_t s = o->s, hw = H / heads;   /* units per head */
    const int64_t e_bytes = (int64_t)e_dim * (e_dtype == 0 ? 4 : 2);
    const int64_t n_bytes = (int64_t)n_dim * (n_dtype == 0 ? 4 : 2);
    const int64_t k1 = pad32(n_dim) + pad32(e_dim) + pad32(d_t);
    const int64_t k3 = pad32(n_dim) + H;
    double *x = (double *)malloc(sizeof(double) * (size_t)(n_dim + e_dim + d_t + 1));
    double *a = (double *)malloc(sizeof(double) * (size_t)H);
    double *h = (double *)malloc(sizeof(double) * (size_t)(s * H));
    double *logit = (double *)malloc(sizeof(double) * (size_t)(s * heads));
    double *y = (double *)malloc(sizeof(double) * (size_t)(n_dim + H + 1));
    int *valid = (int *)malloc(sizeof(int) * (size_t)s);
    int rc = 0;
    for (int64_t i = 0; i < nq && rc == 0; i++) {
        const int32_t n = node[i];
        const int64_t row = table_row(o, n);
        if (row < 0) { rc = -1; break; }
        int any = 0;
        for (int64_t sl = 0; sl < s; sl++) {
            const size_t idx = (size_t)row * (size_t)s + (size_t)sl;
            valid[sl] = (o->nbr[idx] != -1) && (o->ts[idx] < tq[i]);
            if (!valid[sl]) continue;
            any = 1;
            const int32_t v = o->nbr[idx];
            const uint32_t e = o->eid[idx];
            const float dt = (float)(uint32_t)(tq[i] - o->ts[idx]);
            /* MLP_in on x = [r_v ; e ; T-enc(tq - t')] */
            for (int64_t c = 0; c < n_dim; c++) x[c] = feat_value(nfeat + (size_t)v * n_bytes, n_dtype, c);
            for (int64_t c = 0; c < e_dim; c++)
                x[n_dim + c] = (int64_t)e < e_rows ? feat_value(efeat + (size_t)e * e_bytes, e_dtype, c) : 0.0;
            for (int64_t c = 0; c < d_t; c++) x[n_dim + e_dim + c] = (double)tenc_value(w[c], dt, b[c]);
            for (int64_t j = 0; j < H; j++) {
                double acc = 0.0;
                for (int64_t c = 0; c < n_dim; c++) acc += bf16_value(w1[j * k1 + c]) * x[c];
                for (int64_t c = 0; c < e_dim; c++)
                    acc += bf16_value(w1[j * k1 + pad32(n_dim) + c]) * x[n_dim + c];
                for (int64_t c = 0; c < d_t; c++)
                    acc += bf16_value(w1[j * k1 + pad32(n_dim) + pad32(e_dim) + c]) * x[n_dim + e_dim + c];
                acc += (double)b1[j];
                a[j] = acc > 0.0 ? acc : 0.0;                  /* ReLU */
            }
            affine(w2, H, 0, b2, a, H, H, h + sl * H);
            for (int64_t hd = 0; hd < heads; hd++) {          /* logit of head hd: w . h on its slice */
                double l = 0.0;
                for (int64_t j = hd * hw; j < (hd + 1) * hw; j++) l += (double)att[j] * h[sl * H + j];
                logit[sl * heads + hd] = l;
            }
        }
        /* per head: softmax over the valid slots, then the weighted sum of its slice */
        for (int64_t j = 0; j < H; j++) y[n_dim + j] = 0.0;
        if (any) {
            for (int64_t hd = 0; hd < heads; hd++) {
                double m = -INFINITY, den = 0.0;
                for (int64_t sl = 0; sl < s; sl++)
                    if (valid[sl] && logit[sl * heads + hd] > m) m = logit[sl * heads + hd];
                for (int64_t sl = 0; sl < s; sl++) if (valid[sl]) den += exp(logit[sl * heads + hd] - m);
                for (int64_t sl = 0; sl < s; sl++) {
                    if (!valid[sl]) continue;
                    const double alpha = exp(logit[sl * heads + hd] - m) / den;
                    for (int64_t j = hd * hw; j < (hd + 1) * hw; j++) y[n_dim + j] += alpha * h[sl * H + j];
                }
            }
        }
        /* MLP_out on y = [r_u ; aggregate] */
        for (int64_t c = 0; c < n_dim; c++) y[c] = feat_value(nfeat + (size_t)n * n_bytes, n_dtype, c);
        for (int64_t j = 0; j < H; j++) {
            double acc = 0.0;
            for (int64_t c = 0; c < n_dim; c++) acc += bf16_value(w3[j * k3 + c]) * y[c];
            for (int64_t c = 0; c < H; c++) acc += bf16_value(w3[j * k3 + pad32(n_dim) + c]) * y[n_dim + c];
            acc += (double)b3[j];
            a[j] = acc > 0.0 ? acc : 0.0;
        }
        affine(w4, H, 0, b4, a, H, H, z_out + i * H);
    }
    free(x); free(a); free(h); free(logit); free(y); free(valid);
    return rc;
}

static double sigmoid(double a) { return 1.0 / (1.0 + exp(-a)); }

static uint16_t bf16_round(double v)
{
    /* double -> fp32 (nearest) -> bf16 (nearest even), as a bf16 store of
     * an fp32 result rounds */
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, 4);
    u = u + 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/*
 * Node-status update of Sec. 4.4: after a link (u, v, t) with features e,
 * r_u <- RNN([r_u, r_v, t, e]) and r_v <- RNN([r_v, r_u, t, e]).  The RNN is
 * a GRU cell (Cho et al., 2014) with input x = [r_other ; T-enc(t) ; e] and
 * hidden state h = r_self:
 *   r = sigmoid(W_ir x + b_ir + W_hr h + b_hr)
 *   z = sigmoid(W_iz x + b_iz + W_hz h + b_hz)
 *   n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
 *   h' = (1 - z) * n + z * h
 * T-enc(t) is the table's time encoding of the link's timestamp,
 * cos(w_k * t + b_k) with the fp32 argument fmaf(w_k, (float)t, b_k).
 * A batch of n links (arrival indices e0 .. e0+n-1, link rows efeat[e]) is
 * applied with batch semantics: every update reads the statuses as they were
 * before the batch, and a node that several links of the batch touch takes
 * the update of the latest one (larger arrival index; the second endpoint's
 * update after the first's on a self-loop).
 * status: [N][d] fp32 (dtype 0) or bf16 bits (1), updated in place.
 * Weights (bf16 bits, row-major, input segments zero-padded to 32 columns):
 *   w_ih [3d][pad32(d) + pad32(d_t) + pad32(e_dim)]  rows r | z | n
 *   w_hh [3d][pad32(d)]
 * b_ih, b_hh: fp32 [3d].  A link whose arrival index is e_rows or more has
 * no link-feature row: its e is zero (as in orc_sample).  Returns -1 on an
 * out-of-range endpoint.
 */
int orc_gru_update(int64_t N, int32_t d, void *status, int32_t status_dtype,
                   const int32_t *src, const int32_t *dst, const uint32_t *t, int64_t n,
                   uint64_t e0, int32_t d_t, const float *w, const float *b,
                   const uint8_t *efeat, int64_t e_rows, int32_t e_dim, int32_t e_dtype,
                   const uint16_t *w_ih, const uint16_t *w_hh, const float *b_ih,
                   const float *b_hh)
{
    const int64_t kx = pad32(d) + pad32(d_t) + pad32(e_dim);
    const int64_t kh = pad32(d);
    const int64_t e_bytes = (int64_t)e_dim * (e_dtype == 0 ? 4 : 2);
    const int64_t s_bytes = (int64_t)d * (status_dtype == 0 ? 4 : 2);
    for (int64_t i = 0; i < n; i++)
        if (src[i] < 0 || dst[i] < 0 || src[i] >= N || dst[i] >= N) return -1;
    /* candidates of every touched node; the last write per node wins */
    double *cand = (double *)malloc(sizeof(double) * (size_t)(2 * n) * (size_t)d);
    int32_t *who = (int32_t *)malloc(sizeof(int32_t) * (size_t)(2 * n));
    double *x = (double *)malloc(sizeof(double) * (size_t)(d + d_t + e_dim + 1));
    double *hv = (double *)malloc(sizeof(double) * (size_t)d);
    for (int64_t i = 0; i < n; i++) {
        for (int k = 0; k < 2; k++) {
            const int32_t self = k == 0 ? src[i] : dst[i];
            const int32_t other = k == 0 ? dst[i] : src[i];
            const uint8_t *rs = (const uint8_t *)status + (size_t)self * (size_t)s_bytes;
            const uint8_t *ro = (const uint8_t *)status + (size_t)other * (size_t)s_bytes;
            for (int64_t c = 0; c < d; c++) x[c] = feat_value(ro, status_dtype, c);
            for (int64_t c = 0; c < d_t; c++)
                x[d + c] = (double)tenc_value(w[c], (float)t[i], b[c]);
            const uint64_t e = e0 + (uint64_t)i;
            for (int64_t c = 0; c < e_dim; c++)
                x[d + d_t + c] = e < (uint64_t)e_rows ? feat_value(efeat + (size_t)e * (size_t)e_bytes, e_dtype, c)
                                                      : 0.0;
            for (int64_t c = 0; c < d; c++) hv[c] = feat_value(rs, status_dtype, c);
            double *out = cand + (size_t)(2 * i + k) * (size_t)d;
            for (int64_t j = 0; j < d; j++) {
                double gi[3], gh[3];
                for (int g = 0; g < 3; g++) {
                    const int64_t row = g * d + j;
                    double acc = 0.0;
                    for (int64_t c = 0; c < d; c++) acc += bf16_value(w_ih[row * kx + c]) * x[c];
                    for (int64_t c = 0; c < d_t; c++)
                        acc += bf16_value(w_ih[row * kx + pad32(d) + c]) * x[d + c];
                    for (int64_t c = 0; c < e_dim; c++)
                        acc += bf16_value(w_ih[row * kx + pad32(d) + pad32(d_t) + c]) * x[d + d_t + c];
                    gi[g] = acc + (double)b_ih[row];
                    double acc2 = 0.0;
                    for (int64_t c = 0; c < d; c++) acc2 += bf16_value(w_hh[row * kh + c]) * hv[c];
                    gh[g] = acc2 + (double)b_hh[row];
                }
                const double r = sigmoid(gi[0] + gh[0]);
                const double z = sigmoid(gi[1] + gh[1]);
                const double nn = tanh(gi[2] + r * gh[2]);
                out[j] = (1.0 - z) * nn + z * hv[j];
            }
            who[2 * i + k] = self;
        }
    }
    /* apply in stream order: the latest update of a node is written last */
    for (int64_t r = 0; r < 2 * n; r++) {
        uint8_t *dstrow = (uint8_t *)status + (size_t)who[r] * (size_t)s_bytes;
        const double *c = cand + (size_t)r * (size_t)d;
        for (int64_t j = 0; j < d; j++) {
            if (status_dtype == 0) {
                const float f = (float)c[j];
                memcpy(dstrow + 4 * j, &f, 4);
            } else {
                const uint16_t hb = bf16_round(c[j]);
                memcpy(dstrow + 2 * j, &hb, 2);
            }
        }
    }
    free(cand); free(who); free(x); free(hv);
    return 0;
}

/* Stand-alone T-encoding of a list of gaps, for direct checks of App. C. */
void orc_tenc(const float *dt, int64_t n, int32_t d_t, const float *w, const float *b, float *out)
{
    for (int64_t i = 0; i < n; i++)
        for (int32_t k = 0; k < d_t; k++)
            out[(size_t)i * (size_t)d_t + (size_t)k] = tenc_value(w[k], dt[i], b[k]);
}
