/*
 * nlb.h -- C ABI of the MI355X (gfx950) implementation of NLB forward recent
 * sampling: per-node fixed-size hash tables of down-sampled temporal
 * neighbours, maintained on the GPU batch by batch, and batched queries that
 * gather the stored neighbours with their features and a cosine time
 * encoding.
 *
 * Method: Luo & Li, "Scalable and Efficient Temporal Graph Representation
 * Learning via Forward Recent Sampling", arXiv 2402.01964.
 *   - Sec. 3, Def. "Temporal network": a time-ordered stream of undirected
 *     links (u, v, t).  Here link i of the stream gets the 0-based arrival
 *     index e = i (its "edge id"); later means larger e.
 *   - Sec. 3, eq. (1): the temporal neighbours of u at time t are links of u
 *     with timestamp t' < t (strict).
 *   - Sec. 4.2: table S_u has s slots.  Link (u, v, t) offers (v, t, e) to
 *     S_u at slot hash(v, t) and (u, t, e) to S_v at slot hash(u, t), with
 *     hash(v, t) = (q1*v + q2*t) mod s (NLB-edge, eq. (2)) or
 *     hash(v) = q1*v mod s (NLB-node, eq. (3)).  An empty slot takes the
 *     offer; an occupied slot is replaced with probability alpha.  Tables are
 *     updated after the current batch's queries are answered.
 *   - Sec. 4.4: a query (u, t) retrieves S_u^t: each neighbour's status
 *     (node feature row), the link's features and the encoded time.
 *   - App. C: the time encoding is a vector of cosines of w_k * dt + b_k
 *     (the paper's [cos, sin] pairs are the case b_k in {0, -pi/2}).
 *
 * Random draws.  The replacement coin of the offer of link e to its first
 * endpoint (k = 0, table of src) or second endpoint (k = 1, table of dst) is
 * the high 32 bits of output number 2e+k+1 of SplitMix64 (Steele, Lea &
 * Flood, OOPSLA 2014) started from state `seed`.  The offer replaces an
 * occupied slot iff coin < floor(alpha * 2^32) (always when alpha = 1).  The
 * result of every call is therefore a deterministic function of the stream,
 * the parameters and the seed, and equals inserting the links one at a time
 * in stream order, whatever the batch sizes.
 *
 * Conventions for every entry point:
 *   - Pointers named "device" are HIP device memory on the table's device;
 *     the library never frees or retains them beyond what is stated.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls are asynchronous and ordered on that stream; use one stream (or
 *     order streams yourself) per table.
 *   - Return value: NLB_OK or an NLB_E* code.  Argument errors are detected
 *     on the host before anything is enqueued and leave the table unchanged.
 *     Errors found by kernels (out-of-range node ids, timestamps >= 2^30 or
 *     out of order) are recorded on the device and reported by nlb_status.
 *   - A table is used from one host thread at a time.  Distinct tables are
 *     independent.  No C++ exception crosses this interface.
 */
#ifndef NLB_H
#define NLB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define NLB_OK 0
#define NLB_EINVAL 1   /* bad argument (NULL pointer, size or parameter out of range) */
#define NLB_ENOMEM 2   /* device allocation failed */
#define NLB_EDEVICE 3  /* no usable GPU, or a HIP call failed */
#define NLB_EORDER 4   /* (nlb_status) timestamps decreased, or a timestamp >= 2^30 */
#define NLB_ERANGE 5   /* node id outside [0, num_nodes), or more than 2^32-1 links */
#define NLB_ESCRATCH 6 /* nlb_rnn_update_noalloc: the call needs more working memory than the
                          library's static array holds */

/* Key choice of Sec. 4.2. */
#define NLB_KEY_EDGE 0 /* key (neighbour, time): slot by eq. (2) */
#define NLB_KEY_NODE 1 /* key neighbour: slot by eq. (3) */

#define NLB_MAX_SLOTS 1024

typedef struct nlb_table nlb_table;

typedef struct nlb_config {
    int64_t num_nodes;      /* N: node ids are 0..N-1; 1 <= N <= 2^31-1 */
    int32_t s;              /* slots per node, 1..NLB_MAX_SLOTS */
    int32_t key_mode;       /* NLB_KEY_EDGE or NLB_KEY_NODE */
    double alpha;           /* replacement probability, 0 < alpha <= 1 */
    uint64_t seed;          /* start state of the coin generator */
    uint64_t q1, q2;        /* hash primes of eq. (2)/(3); 0 selects 1000000007 / 998244353;
                               each must be < 2^31 */
    int32_t d_time;         /* time-encoding width; 0 = no time encoding */
    const float *time_w;    /* device fp32[d_time] frequencies, borrowed for the table's life */
    const float *time_b;    /* device fp32[d_time] phases, borrowed for the table's life */
    const void *edge_feat;  /* device [edge_rows][edge_row_bytes] link features indexed by
                               arrival index, borrowed; NULL = none */
    int64_t edge_rows;      /* rows of edge_feat; a stored link with e >= edge_rows gathers zeros */
    int32_t edge_row_bytes; /* bytes per link-feature row, a multiple of 4 (0 with NULL) */
    const void *node_feat;  /* device [num_nodes][node_row_bytes] node rows, borrowed; NULL = none */
    int32_t node_row_bytes; /* bytes per node row, a multiple of 4 (0 with NULL) */
    int32_t device;         /* HIP device ordinal that holds the table; -1 = current device */
} nlb_config;

/* Output buffers of nlb_sample (device pointers, row-major, in slot order).
 * Any member may be NULL to skip that output.  For query i and slot a:
 *   nbr  int32 [nq][s]                  stored neighbour id, -1 if not valid
 *   eid  uint32[nq][s]                  stored arrival index, 0xFFFFFFFF if not valid
 *   ts   uint32[nq][s]                  stored timestamp t', 0xFFFFFFFF if not valid
 *   tenc fp32  [nq][s][d_time]          cos(fmaf(w_k, (float)(tq - t'), b_k)), 0 if not valid
 *   efeat bytes[nq][s][edge_row_bytes]  edge_feat row eid, zero bytes if not valid
 *   nfeat bytes[nq][s][node_row_bytes]  node_feat row nbr, zero bytes if not valid
 *   self  bytes[nq][node_row_bytes]     node_feat row of the query node (zeros if the id is
 *                                       out of range)
 * A slot is valid when it is non-empty and its timestamp t' < tq (eq. (1)).
 * tenc is within 1e-5 absolute of the cosine, taken in double, of the fp32
 * argument fmaf(w_k, (float)(tq - t'), b_k); everything else is exact. */
typedef struct nlb_sample_out {
    int32_t *nbr;
    uint32_t *eid;
    uint32_t *ts;
    float *tenc;
    void *efeat;
    void *nfeat;
    void *self;
} nlb_sample_out;

typedef struct nlb_info {
    int64_t num_nodes;
    int32_t s;
    int32_t key_mode;
    uint64_t threshold;     /* floor(alpha * 2^32), or 2^32 for alpha == 1 */
    uint64_t q1, q2;
    uint64_t interactions;  /* links inserted so far = arrival index of the next link, as
                               counted by eager calls; nlb_status refreshes it from the
                               device count, which also counts graph replays */
    int64_t table_bytes;    /* device bytes owned by the table */
    int32_t block_bytes;    /* bytes of one node's slot block */
    int32_t device;
    int32_t rnn_form;       /* GRU pass of the last nlb_rnn_update: NLB_RNN_FORM_* */
} nlb_info;

/* Forms of the GRU pass of nlb_rnn_update: none run yet; tiles of listed
 * rows with the weights streamed from L2; the weight-stationary form (the
 * weights held in registers for the whole launch, one workgroup per CU),
 * used when the statuses have 16-byte rows, pad32(d) <= 128 and
 * pad32(d) + pad32(d) + pad32(d_time) + pad32(edge_dim) <= 384. */
#define NLB_RNN_FORM_NONE 0
#define NLB_RNN_FORM_TILED 1
#define NLB_RNN_FORM_WEIGHT_STATIONARY 2

/* Create an empty table (Sec. 4.2: fixed-size GPU memory of s slots per
 * node, all empty).  Validates `cfg`, allocates and zeroes the slot blocks on
 * cfg->device, and stores *out only on success.  Errors: NLB_EINVAL (NULL
 * argument, parameter out of range, row bytes not a multiple of 4, feature
 * pointer and row bytes disagreeing), NLB_EDEVICE (no GPU), NLB_ENOMEM. */
int nlb_create(const nlb_config *cfg, nlb_table **out);

/* Insert the n links (src[i], dst[i], t[i]), i < n, as links
 * interactions..interactions+n-1 of the stream (Sec. 4.2).  src, dst, t are
 * device arrays of n elements, read during the call's kernels.  Each link
 * offers to both endpoint tables; conflicts inside the batch resolve exactly
 * as sequential insertion would.  Timestamps must be < 2^30 and
 * non-decreasing across calls; node ids must be in [0, N).  Links with an
 * out-of-range endpoint or timestamp are skipped and flagged for
 * nlb_status, but still consume their arrival index.  n == 0 is a no-op.
 * Errors: NLB_EINVAL (NULL table or array with n > 0; n >= 2^31),
 * NLB_ERANGE (the arrival index would exceed 2^32-2), NLB_EDEVICE (launch
 * failure).  The kernels take the batch's arrival indices from a link count
 * kept on the device and advance it (the host keeps its own count for the
 * NLB_ERANGE test and nlb_get_info), so the call may be captured in a HIP
 * graph: every replay inserts its links as the next links of the stream
 * (a replay that would pass 2^32 - 1 links is skipped and flagged for
 * nlb_status as NLB_ERANGE). */
int nlb_insert_batch(nlb_table *h, const int32_t *src, const int32_t *dst,
                     const uint32_t *t, uint32_t n, void *stream);

/* Answer nq queries (node[i], tq[i]) from the tables as they stand after the
 * inserts enqueued before this call (Sec. 4.4 retrieval; eq. (1) strict
 * mask; App. C time encoding).  node and tq are device arrays of nq
 * elements; out holds device output pointers as described above and is read
 * during the call only.  A query node outside [0, N) yields an all-invalid
 * answer and is flagged for nlb_status.  nq == 0 is a no-op.
 * Errors: NLB_EINVAL (NULL table, out or array with nq > 0; tenc/efeat/nfeat/
 * self requested without the matching configuration), NLB_EDEVICE.
 * The call only enqueues kernels (no allocation, memset or synchronisation):
 * it may be captured in a HIP graph and replayed on the same buffers. */
int nlb_sample(nlb_table *h, const int32_t *node, const uint32_t *tq, uint32_t nq,
               const nlb_sample_out *out, void *stream);

/* Second-hop retrieval (Sec. 4.4: if v is stored in S_u^t, S_v^t holds
 * down-sampled second-hop neighbours of u).  hop1_nbr is the device nbr
 * output [nq][s] of an nlb_sample call for queries (node[i], tq[i]); tq is
 * the same device array of nq query times.  For every first-hop entry
 * (i, a) with neighbour v = hop1_nbr[i*s + a], the call answers the query
 * (v, tq[i]) exactly as nlb_sample would, into row i*s + a of each output:
 * nbr/eid/ts [nq][s][s], tenc [nq][s][s][d_time], efeat/nfeat
 * [nq][s][s][row bytes], self [nq][s][node_row_bytes] (v's node row).  An
 * empty first-hop entry (v < 0) gives an all-invalid answer and a zero self
 * row without an error; v >= N is flagged as in nlb_sample.  nq*s must be
 * below 2^32.  nq == 0 is a no-op.  Errors: as nlb_sample.  Graph capture:
 * as nlb_sample. */
int nlb_sample_hop2(nlb_table *h, const int32_t *hop1_nbr, const uint32_t *tq, uint32_t nq,
                    const nlb_sample_out *out, void *stream);

/* Time encoding (App. C) of an nlb_sample answer from its timestamp output:
 *   tenc[i][a][k] = cos(fmaf(w_k, (float)(tq[i] - ts[i*s + a]), b_k)),
 *   0 where ts[i*s + a] == 0xFFFFFFFF (an invalid slot),
 * the values nlb_sample writes to its own tenc output, to the same bits.
 * With it a caller splits a retrieval into its table reads (nlb_sample with
 * out->tenc NULL and out->ts set) and the encoding, and runs the encoding on
 * a second stream, ordered after the sample by an event the caller records:
 * the encoding reads neither the tables nor the feature rows, so it may run
 * beside the next nlb_insert_batch.  ts: device uint32 [nq][s] (an nlb_sample
 * ts output); tq: the device array of the nq query times of that call; tenc:
 * device fp32 [nq][s][d_time].  All three are read or written during the
 * call's kernels only and must be 4-byte aligned (16-byte aligned output
 * and d_time % 4 == 0 take the vector form).  nq == 0 is a no-op.
 * Errors: NLB_EINVAL (NULL table or array with nq > 0, a table without a time
 * encoding, misaligned arrays), NLB_EDEVICE.  Graph capture: as nlb_sample. */
int nlb_time_encode(nlb_table *h, const uint32_t *ts, const uint32_t *tq, uint32_t nq, float *tenc,
                    void *stream);

/* Attention aggregation of eq. (4) (Sec. 4.4), forward:
 *   Z_u = MLP_out(r_u, sum_i alpha_i MLP_in(r_v, e, t')),
 *   {alpha_i} = softmax({w^T MLP_in(r_v, e, t')}) over the valid slots of S_u^t,
 * with MLP(x) = W_b ReLU(W_a x + b_a) + b_b, hidden and output width
 * NLB_AGG_HIDDEN.  The neighbour status r_v is its node-feature row, e the
 * stored link's feature row, t' enters through the table's time encoding of
 * tq - t' (as in nlb_sample) and r_u is the query node's row; tables
 * without node or link features contribute no such inputs.  A query with no
 * valid slot aggregates the zero vector; a query node outside [0, N) is
 * flagged for nlb_status and treated as having no slots and a zero row.
 * Weight matrices are bf16 (device, row-major [H][K], each input segment
 * zero-padded to a multiple of 32 columns, rows 16-byte aligned):
 *   w1: [H][pad32(node_dim) + pad32(edge_dim) + pad32(d_time)]  (r_v | e | T-enc)
 *   w2: [H][H];  w3: [H][pad32(node_dim) + H]  (r_u | aggregate);  w4: [H][H]
 * with node_dim / edge_dim the table's row bytes divided by the element size
 * of node_dtype / edge_dtype.  Biases and att (the attention vector w) are
 * device fp32 [H].  All are read during the call only.  Activations are kept
 * in fp32 and fed to bf16 matrix cores as a pair of bf16 terms (hi + lo,
 * relative error 2^-18), accumulating in fp32 over at most ~400 terms
 * (relative error ~2.5e-5 of the sum of magnitudes); through four layers and
 * the softmax, Z is within 2e-4 * (|Z| + the root mean square of Z over the
 * launch) of the same function evaluated in double (measured: <= 3.9e-5).
 * MLP_in's second layer is affine, so the library may apply it once to the
 * softmax-weighted sum of the first layer's outputs instead of to every
 * slot (the logits then use W_b^T w); only the rounding order differs.
 * Attention heads (the experiments use two, App. E): with heads = A, MLP_in's
 * H outputs are split into A consecutive slices of H / A; head a scores a
 * slot with w[slice a] . MLP_in(...)[slice a], takes its own softmax over the
 * valid slots and fills slice a of the aggregate.  A = 1 is the formula
 * above.  One or two heads run in every kernel form, four and eight in the
 * tiled form (tables of at most 64 slots); any other count is NLB_EINVAL.
 * z is device fp32 [nq][H].  Tables with s > 64 are supported for the input
 * shapes the per-query kernel is built for and rejected (NLB_EINVAL) for
 * others: a time encoding of 97 to 128 dimensions with 16-byte-aligned bf16
 * node rows of 97 to 128 values and no link rows or such bf16 link rows, or
 * no node rows and fp32 link rows of 97 to 128 or 161 to 192 values
 * (16-byte aligned) or bf16 link rows of 161 to 192 values (4-byte aligned).
 * nq == 0 is a no-op.  Errors: as nlb_sample, and NLB_EINVAL
 * for a bad weight set.  Graph capture: as nlb_sample (besides its kernels
 * the call makes only host-side attribute queries and settings). */
#define NLB_AGG_HIDDEN 64
#define NLB_DTYPE_F32 0
#define NLB_DTYPE_BF16 1

typedef struct nlb_agg_weights {
    int32_t hidden;          /* must be NLB_AGG_HIDDEN */
    int32_t node_dtype;      /* element type of the table's node rows: NLB_DTYPE_F32 / _BF16 */
    int32_t edge_dtype;      /* element type of the table's link rows */
    int32_t heads;           /* attention heads A: 0 or 1 for one, else 2, 4 or 8 */
    const uint16_t *w1;      /* bf16 bits */
    const float *b1;
    const uint16_t *w2;
    const float *b2;
    const float *att;
    const uint16_t *w3;
    const float *b3;
    const uint16_t *w4;
    const float *b4;
} nlb_agg_weights;

int nlb_aggregate(nlb_table *h, const int32_t *node, const uint32_t *tq, uint32_t nq,
                  const nlb_agg_weights *wts, float *z, void *stream);

/* Node-status update of Sec. 4.4: after a link (u, v, t) with features e,
 * r_u <- RNN([r_u, r_v, t, e]) and r_v <- RNN([r_v, r_u, t, e]), for a batch
 * of n links (src, dst, t: device arrays of n elements) whose link-feature
 * rows are first_eid .. first_eid + n - 1 of the table's link rows (rows at
 * or past edge_rows read as zeros); first_eid = NLB_EID_LAST_BATCH takes the
 * arrival indices of the n links inserted last (the table's device link
 * count when the update runs, minus n), as a step that inserts a batch and
 * then updates the statuses needs, also when replayed from a HIP graph.
 * The RNN is a GRU cell with input x = [r_other ; T-enc(t) ; e] and hidden
 * state h = r_self:
 *   r = sigmoid(W_ir x + b_ir + W_hr h + b_hr)
 *   z = sigmoid(W_iz x + b_iz + W_hz h + b_hz)
 *   n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
 *   h' = (1 - z) n + z h
 * with T-enc(t) the table's time encoding cos(w_k t + b_k) of the link time
 * (argument fmaf(w_k, (float)t, b_k)).  Batch semantics: every update reads
 * the statuses as they were before the call, and a node that several links
 * of the batch touch takes the update of the latest one (larger index; on a
 * self-loop the dst side's).  status is a device array [N][status_dim] of
 * status_dtype elements, updated in place (it may be the table's node_feat
 * buffer, so later queries gather the new statuses); rows of nodes that no
 * link touches are not written.  A link with an endpoint outside [0, N) is
 * skipped and flagged for nlb_status.  Weights (device, read during the
 * call, bf16 rows 16-byte aligned, each input segment zero-padded to a
 * multiple of 32 columns, gate rows in the order r | z | n):
 *   w_ih: [3 d][pad32(d) + pad32(d_time) + pad32(edge_dim)]  (r_other | T-enc | e)
 *   w_hh: [3 d][pad32(d)];  b_ih, b_hh: fp32 [3 d]
 * with d = status_dim and edge_dim the table's link row bytes over the size
 * of edge_dtype.  Numerics: fp32 activations enter bf16 matrix cores as
 * hi + lo pairs (2^-18 relative), bf16 ones as one term, with fp32
 * accumulation; an fp32 status is within 1e-4 of the same cell evaluated in
 * double, a bf16 one within one bf16 rounding of it.  Calls on one table
 * must be ordered (same stream): they share the table's working buffers,
 * which the first call (and a larger batch) allocates.  n == 0 is a no-op.
 * Graph capture: a call that allocates (see above) must not be captured;
 * once an earlier call on the table has sized the working memory for at
 * least n links, the call only enqueues kernels and may be captured and
 * replayed (no call number or host-side state is involved; with
 * first_eid = NLB_EID_LAST_BATCH it follows the inserts replayed before it).
 * Errors: NLB_EINVAL (NULL table, weights or array with n > 0; n >= 2^31;
 * bad dtype or dimension; misaligned pointers; a 16-row tile that does not
 * fit the LDS), NLB_ENOMEM, NLB_EDEVICE. */
#define NLB_RNN_MAX_DIM 1024
#define NLB_EID_LAST_BATCH UINT64_MAX

typedef struct nlb_gru_weights {
    int32_t status_dim;      /* d, 1 .. NLB_RNN_MAX_DIM */
    int32_t status_dtype;    /* NLB_DTYPE_F32 / _BF16 */
    int32_t edge_dtype;      /* element type of the table's link rows */
    const uint16_t *w_ih;    /* bf16 bits */
    const uint16_t *w_hh;
    const float *b_ih;
    const float *b_hh;
} nlb_gru_weights;

int nlb_rnn_update(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t, uint32_t n,
                   uint64_t first_eid, const nlb_gru_weights *wts, void *status, void *stream);

/* nlb_rnn_update for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, kernels and results; it allocates and frees nothing
 * (device memory, host-pinned memory or library workspaces) and sets no
 * memory with hipMemset: its working memory -- the winner word of each of
 * the table's N nodes (8 B), a list of 16 B per pair row, the GRU weights
 * repacked in matrix-operand fragments (3 KiB per 16 status columns and
 * 32 input columns of w_ih and w_hh together), and 2 n candidate status
 * rows -- lives in one static device array of NLB_NOALLOC_SCRATCH bytes per
 * device, which the library holds until the process ends.  The call needs
 * align256(8 N) + align256(16 (2 n) + 256) + align256(3072 (pad32(d) / 16)
 * ((k_x + pad32(d)) / 32)) + 2 n * status row bytes of it (k_x: the row
 * width of w_ih), and returns NLB_ESCRATCH when that exceeds the array
 * (nothing is enqueued then).  Every call on a device shares that device's
 * array: the call clears what it needs cleared (the winner words, with a
 * fill kernel) and keeps no state across calls, but calls that overlap in
 * time on one device -- other streams, other threads, other tables -- race
 * and must be ordered by the caller.  Besides the NLB_ESCRATCH case, errors
 * are those of nlb_rnn_update.  The first call on a device looks up the
 * array's device address (hipGetSymbolAddress) with that device current. */
#define NLB_NOALLOC_SCRATCH (64u << 20)

int nlb_rnn_update_noalloc(nlb_table *h, const int32_t *src, const int32_t *dst, const uint32_t *t,
                           uint32_t n, uint64_t first_eid, const nlb_gru_weights *wts, void *status,
                           void *stream);

/* Free the table's device memory after synchronising its device.  NULL is a
 * no-op.  Borrowed buffers are not touched. */
int nlb_destroy(nlb_table *h);

/* Sizes and counters of a table (host-side values; no synchronisation). */
int nlb_get_info(const nlb_table *h, nlb_info *info);

/* Write the canonical table into device arrays of N*s elements, node-major:
 * nbr (-1 = empty), ts and eid (0xFFFFFFFF = empty).  Ordered on `stream`.
 * For inspection and tests; the layout the kernels use is internal. */
int nlb_export(nlb_table *h, int32_t *nbr, uint32_t *ts, uint32_t *eid, void *stream);

/* Synchronise `stream`, then return and clear the errors kernels recorded
 * since the last call: NLB_OK, NLB_ERANGE (node id out of range, or a
 * replayed insert past 2^32 - 1 links) or NLB_EORDER (timestamp >= 2^30 or
 * decreasing); NLB_ERANGE wins when both.  Also refreshes the link count of
 * nlb_get_info from the device. */
int nlb_status(nlb_table *h, void *stream);

/* Static description of a return code. */
const char *nlb_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* NLB_H */
