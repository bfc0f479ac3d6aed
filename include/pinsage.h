/*
 * pinsage.h -- C ABI of libpinsage.so, the MI355X (gfx950) hot path of PinSage
 * (Ying et al., "Graph Convolutional Neural Networks for Web-Scale Recommender
 * Systems", KDD 2018).
 *
 * The library computes, on one GPU:
 *   1. importance neighbourhoods by short random walks (Sec. 3.2,
 *      "Importance-based neighborhoods"), and
 *   2. K stacked CONVOLVE layers (Algorithm 1) over every node, evaluated
 *      layer by layer so that each node's transformed vector is computed once
 *      (Sec. 3.4),
 *   3. the minibatch forward of Algorithm 2 with the max-margin loss (Eq. 1),
 *   4. hard negative items for training queries (Sec. 3.3),
 *   5. the MapReduce-inference variant of Sec. 3.4 (boards pool their pins,
 *      pins their boards, boards without features).
 *
 * Conventions shared by every entry point
 *   - Graph (Sec. 3.1): a bipartite graph of pins I and boards C, V = I u C.
 *     Node ids: pins are [0, num_pins), boards are [num_pins, num_nodes).
 *     Undirected CSR holding both directions; each row sorted ascending.
 *   - Pointers named "device" must be device memory (or memory the device can
 *     read); all buffers are owned by the caller. The library keeps no device
 *     allocation between calls except what is documented per entry point.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream). No call synchronises the host unless stated.
 *   - Arguments are validated on the host before any HIP call; a bad argument
 *     returns PINSAGE_EINVAL / PINSAGE_EUNSUPPORTED / PINSAGE_EWORKSPACE and
 *     launches nothing. HIP failures return PINSAGE_EHIP; the message is in
 *     pinsage_last_error() (thread-local).
 *   - Results are deterministic: the same inputs give the same bits.
 *   - Matrices are row-major. Storage dtype is fp32 or bf16; every sum is
 *     accumulated in fp32; biases are fp32.
 */
#ifndef PINSAGE_H_
#define PINSAGE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PINSAGE_ABI_VERSION 12

enum {
  PINSAGE_OK = 0,
  PINSAGE_EINVAL = -1,       /* malformed argument (NULL, size, mismatch)    */
  PINSAGE_EUNSUPPORTED = -2, /* well-formed but outside the supported limits */
  PINSAGE_EWORKSPACE = -3,   /* workspace smaller than the size query says   */
  PINSAGE_EHIP = -4          /* a HIP runtime call failed                    */
};

typedef enum { PINSAGE_I32 = 0, PINSAGE_I64 = 1 } pinsage_index_t;
typedef enum { PINSAGE_F32 = 0, PINSAGE_BF16 = 1 } pinsage_dtype_t;

/* Bipartite pin-board graph (Sec. 3.1). row_offsets: device, num_nodes + 1
 * entries of offset_type, row_offsets[0] = 0, non-decreasing, last = nnz.
 * col: device, nnz int32 node ids. I32 offsets require nnz < 2^31.
 * walk_table: NULL, or device memory filled by pinsage_build_walk_table for
 * this graph (same row_offsets and col, unmodified since; 16-byte aligned,
 * nnz < 2^31). When set, every random walk of the library (neighbourhoods,
 * minibatch frontiers, hard negatives, the all-node job) reads it: one
 * dependent read per edge step instead of the node's offsets and then a
 * neighbour id. The walks, and so every result, are the same bits. */
typedef struct {
  int64_t num_pins;
  int64_t num_boards;
  int64_t nnz;
  pinsage_index_t offset_type;
  const void* row_offsets;
  const int32_t* col;
  const void* walk_table;
} pinsage_graph_t;

/* Random-walk parameters (Sec. 3.2). Each of `walks_per_node` walks from a
 * source u moves to a uniformly drawn CSR neighbour per edge step and ends
 * after `hops` landings on a pin (or 2*hops edge steps, or a node with no
 * edges). Every landing on a pin v != u adds one visit of v. The draw of step
 * s of walk w uses word s%4 of Philox4x32-10 (Salmon et al., SC'11) at counter
 * (u, w, s/4, 0) under key (lo32(seed), hi32(seed)); a word r selects the
 * neighbour with index floor(r * deg / 2^32).
 * Limits: 1 <= walks_per_node * hops <= 1024, 1 <= top_t <= 256. */
typedef struct {
  uint64_t seed;
  int32_t walks_per_node;
  int32_t hops;
  int32_t top_t;
} pinsage_walk_params_t;

/* Importance neighbourhoods (Sec. 3.2), one row of top_t entries per source,
 * in rank order (visit count descending, ties by lower node id):
 *   idx     device int32  [rows][top_t], node id or -1 (padding, tail only)
 *   counts  device uint16 [rows][top_t], visit counts (0 for padding)
 *   weights device fp32   [rows][top_t], count / (sum of the row's kept
 *           counts), one IEEE fp32 division; 0 for padding. May be NULL in
 *           pinsage_build_neighborhoods (not written) and in the layer calls
 *           (then derived from counts in-kernel, with the same division). */
typedef struct {
  int64_t rows;
  int32_t top_t;
  int32_t* idx;
  uint16_t* counts;
  float* weights;
} pinsage_neighborhoods_t;

/* Order in which a layer evaluates Algorithm 1 (both give the same values in
 * exact arithmetic; they differ only in rounding):
 *   POOL_THEN_DENSE  Algorithm 1 as written: P = ReLU(Q h + q) for every pin,
 *                    n_u = weighted mean of P over N(u) (m-wide rows),
 *                    z_u = ReLU(W [h_u ; n_u] + w).
 *   DENSE_THEN_POOL  the neighbour half of W is applied before the pool, as
 *                    the weighted mean is linear: with W = [W_s | W_n],
 *                    R = P W_n^T for every pin (d_out-wide rows),
 *                    g_u = weighted mean of R over N(u),
 *                    z_u = ReLU(W_s h_u + g_u + w).
 *                    The gather reads d_out instead of m values per neighbour. */
typedef enum { PINSAGE_POOL_THEN_DENSE = 0, PINSAGE_DENSE_THEN_POOL = 1 } pinsage_dataflow_t;

/* The aggregator gamma of Algorithm 1, line 1, over a node's neighbourhood
 * (rank order, padding skipped; an empty neighbourhood gives zero):
 *   IMPORTANCE  sum_t alpha_t P_t, alpha the normalised visit counts (Sec. 3.2)
 *   MEAN        element-wise mean of the neighbours' rows (gamma = mean, Sec. 4)
 *   MAX         element-wise max of the neighbours' rows (gamma = max, Sec. 4)
 * MAX is not linear, so it requires PINSAGE_POOL_THEN_DENSE. */
typedef enum {
  PINSAGE_POOL_IMPORTANCE = 0,
  PINSAGE_POOL_MEAN = 1,
  PINSAGE_POOL_MAX = 2
} pinsage_pool_t;

/* One CONVOLVE layer's parameters (Algorithm 1; Sec. 3.2 "Stacking
 * convolutions": shared by all nodes, distinct per layer).
 *   Q device [m][d_in]            (storage dtype)
 *   q device fp32 [m]
 *   W device [d_out][d_in + m]    (storage dtype); columns [0, d_in) multiply
 *                                 the node's own vector, [d_in, d_in + m) the
 *                                 pooled neighbourhood vector
 *   w device fp32 [d_out]
 *   dataflow                      evaluation order (above)
 *   pool                          the aggregator gamma (above)
 * Limits: d_in, m, d_out multiples of 16; d_in, m <= 8192; d_out <= 512. */
typedef struct {
  int32_t d_in;
  int32_t m;
  int32_t d_out;
  pinsage_dtype_t dtype;
  const void* Q;
  const float* q;
  const void* W;
  const float* w;
  pinsage_dataflow_t dataflow;
  pinsage_pool_t pool;
} pinsage_layer_t;

/* The output dense layers of Algorithm 2 (its final loop), applied after the
 * last CONVOLVE layer: z_u = G2 ReLU(G1 h_u + g).
 *   G1 device [d_hidden][d_in]   (storage dtype)
 *   g  device fp32 [d_hidden]
 *   G2 device [d_out][d_hidden]  (storage dtype); no bias, no activation
 * Accumulation fp32; the hidden activations are stored in the storage dtype.
 * Limits: d_in, d_hidden, d_out multiples of 16 and <= 8192. */
typedef struct {
  int32_t d_in;
  int32_t d_hidden;
  int32_t d_out;
  pinsage_dtype_t dtype;
  const void* G1;
  const float* g;
  const void* G2;
} pinsage_mlp_t;

/* Walk table of a graph (a layout of its CSR for the random walks of
 * Sec. 3.2): 16 bytes per CSR position e, {col[e], degree of col[e], row
 * start of col[e] (low, high 32 bits)}, degree 0 for a node whose row is
 * empty or malformed, so that an edge step reads one entry at a uniform
 * position of the current node's row.
 *   pinsage_walk_table_size   *bytes = 16 nnz. PINSAGE_EUNSUPPORTED when
 *                             nnz >= 2^31 (*bytes = 0), PINSAGE_EINVAL for a
 *                             malformed graph or NULL bytes.
 *   pinsage_build_walk_table  fills `table` (device, 16-byte aligned, at
 *                             least the size above; caller-owned) on
 *                             `stream`, asynchronously; set graph.walk_table
 *                             to it for later calls. PINSAGE_EWORKSPACE when
 *                             table_bytes is too small, PINSAGE_EINVAL for
 *                             NULL or misaligned table. Rebuild it after
 *                             changing the CSR. */
int pinsage_walk_table_size(const pinsage_graph_t* graph, size_t* bytes);
int pinsage_build_walk_table(const pinsage_graph_t* graph, void* table, size_t table_bytes,
                             void* stream);

/* Version of this ABI (PINSAGE_ABI_VERSION). */
int pinsage_version(void);
/* Static text for a status code. */
const char* pinsage_status_string(int status);
/* Detail of the last failure on the calling thread ("" if none). */
const char* pinsage_last_error(void);

/* Importance neighbourhoods (Sec. 3.2) of sources[0..num_sources) -- or of
 * every node 0..num_nodes-1 when sources is NULL (then num_sources must equal
 * num_nodes). Row r of `out` belongs to sources[r]. A source id outside
 * [0, num_nodes) yields an all-padding row. If total_steps is non-NULL
 * (device uint64), it receives the number of edge steps all walks took.
 * Out-of-range CSR entries end the walk that meets them (no out-of-bounds
 * access); the graph is assumed well-formed otherwise. */
int pinsage_build_neighborhoods(const pinsage_graph_t* graph,
                                const pinsage_walk_params_t* walk,
                                const int32_t* sources, int64_t num_sources,
                                pinsage_neighborhoods_t* out,
                                unsigned long long* total_steps, void* stream);

/* Hard negative items (Sec. 3.3, "Hard negative items"): for each query, pins
 * are ranked by their Personalized PageRank score with respect to the query
 * and items in a window of ranks are sampled. The score is estimated by the
 * visit counts of `walks` random walks of `hops` pin landings from the query,
 * the walks of pinsage_walk_params_t (same steps, same Philox stream under
 * `seed`); ranks run over the distinct visited pins (the query excluded) by
 * count descending, ties by lower node id, from 0. With D ranked pins and
 * n = min(rank_hi, D) - rank_lo, draw j in [0, num_per_query) of query q takes
 * word 0, r, of Philox4x32-10 at counter (q, j, 0, 1) under the same key and
 * returns the pin at rank rank_lo + floor(r * n / 2^32) (independent draws,
 * with replacement). The paper's window, ranks 2000 to 5000 counted from 1,
 * is rank_lo = 1999, rank_hi = 5000.
 * Limits: 1 <= walks * hops <= 2^22, 0 <= rank_lo < rank_hi, 0 <= num_per_query;
 * with walks * hops > 16384 also rank_hi <= 8192. */
typedef struct {
  uint64_t seed;
  int32_t walks;
  int32_t hops;
  int32_t rank_lo;
  int32_t rank_hi;
  int32_t num_per_query;
} pinsage_hard_negative_params_t;

/* Workspace bytes pinsage_hard_negatives needs for these parameters and
 * query count: 0 for walks * hops <= 16384 (the visits of a query are counted
 * on chip); above that, per resident workgroup (at most 256), L = walks * hops
 * landings of a query: a bucket of 12,288 landings for each of its
 * ceil(L / 8192) hash partitions, an overflow list of up to L landings and its
 * copy by partition, and a list of up to L (pin, count) pairs:
 * 4 (12288 ceil(L / 8192) + 4 L) bytes, rounded up to 256 bytes. Errors as for
 * pinsage_hard_negatives' parameters. */
int pinsage_hard_negatives_workspace_size(const pinsage_hard_negative_params_t* params,
                                          int64_t num_queries, size_t* bytes);

/* out: device int32 [num_queries][num_per_query], pin ids, or -1 for every
 * draw of a query whose window is empty (n <= 0) or whose id lies outside
 * [0, num_nodes). queries: device int32 [num_queries]. If total_steps is
 * non-NULL (device uint64), it receives the number of edge steps all walks
 * took. workspace: device, >= pinsage_hard_negatives_workspace_size bytes,
 * 256-aligned (may be NULL when that size is 0). Out-of-range CSR entries end
 * the walk that meets them. */
int pinsage_hard_negatives(const pinsage_graph_t* graph,
                           const pinsage_hard_negative_params_t* params,
                           const int32_t* queries, int64_t num_queries, int32_t* out,
                           unsigned long long* total_steps, void* workspace,
                           size_t workspace_bytes, void* stream);

/* Graph neighbourhoods of the MapReduce inference (Sec. 3.4): a board's
 * embedding pools the pins it holds and a pin's the boards it occurs on,
 * with neighbours sampled. Node u's neighbourhood is its CSR row if the row
 * has at most T = out->top_t entries; a longer row is sampled with T
 * independent draws, draw j taking word 0 of Philox4x32-10 (Salmon et al.,
 * SC'11) at counter (u, j, 0, 2) under the key (lo32(seed), hi32(seed)) and
 * the row position floor(r * deg / 2^32). Entries outside [0, num_nodes) are
 * dropped. Row r of `out` (for sources[r], or node r when sources is NULL,
 * then num_sources = num_nodes) lists the distinct ids ascending: idx, counts
 * = multiplicity, weights = multiplicity / kept entries (one fp32 division;
 * NULL = not written); padding -1, 0, 0. A source outside [0, num_nodes)
 * yields a padding row. Limits: 1 <= T <= 256. */
int pinsage_build_graph_neighborhoods(const pinsage_graph_t* graph, uint64_t seed,
                                      const int32_t* sources, int64_t num_sources,
                                      pinsage_neighborhoods_t* out, void* stream);

/* Workspace bytes needed by pinsage_embed_all_bipartite. */
int pinsage_embed_all_bipartite_workspace_size(const pinsage_graph_t* graph,
                                               const pinsage_layer_t* layers,
                                               int32_t num_layers, size_t* bytes);

/* All-node embedding in the MapReduce inference of Sec. 3.4: graph
 * neighbourhoods of every node (pinsage_build_graph_neighborhoods with
 * T = nbr_out->top_t), then num_layers CONVOLVE layers over all nodes, layer
 * by layer. Only pins have features (boards' h^(0) is the zero vector), so
 * the number of layers must be even (pins' outputs then rest on pin
 * features); every node can be a neighbour, so each layer projects all
 * num_nodes rows. x_pins: device [num_pins][layers[0].d_in]; h_out: device
 * [num_nodes][layers[K-1].d_out]; nbr_out: rows = num_nodes (weights may be
 * NULL). Layers chain as in pinsage_embed_all; one storage dtype. */
int pinsage_embed_all_bipartite(const pinsage_graph_t* graph, uint64_t seed,
                                const pinsage_layer_t* layers, int32_t num_layers,
                                const void* x_pins, pinsage_neighborhoods_t* nbr_out,
                                void* h_out, void* workspace, size_t workspace_bytes,
                                void* stream);

/* Workspace bytes needed by pinsage_convolve_layer for these sizes. */
int pinsage_convolve_workspace_size(const pinsage_layer_t* layer, int64_t n_transform,
                                    int64_t n_out, size_t* bytes);

/* One CONVOLVE layer (Algorithm 1) in the layer-wise dataflow (Sec. 3.4):
 *   P[i]  = ReLU(Q h_in[t(i)] + q)             for i in [0, n_transform),
 *           t(i) = transform_rows[i] or i
 *   n[r]  = sum_t weights[r][t] * P[idx[r][t]] (rank order; padding skipped)
 *   z[r]  = ReLU(W concat(h_in[s(r)], n[r]) + w),  s(r) = self_rows[r] or r
 *   h_out[r] = z[r] / ||z[r]||_2 (a zero z stays zero)   for r in [0, n_out)
 * (with DENSE_THEN_POOL, n[r] is never formed: the pool runs over rows of
 * P W_n^T, see pinsage_dataflow_t).
 * h_in: device [n_in][d_in]; h_out: device [n_out][d_out]; both in the
 * layer's storage dtype. nbr->rows must equal n_out; neighbour ids index the
 * projected rows, i.e. lie in [0, n_transform) (others are skipped).
 * transform_rows, self_rows: device int32 row maps into h_in, or NULL for the
 * identity (entries outside [0, n_in) read as zero rows). Without
 * transform_rows, n_transform <= n_in; without self_rows, n_out <= n_in.
 * workspace: device, >= pinsage_convolve_workspace_size bytes, 256-aligned. */
int pinsage_convolve_layer(const pinsage_layer_t* layer, const void* h_in, int64_t n_in,
                           int64_t n_transform, const int32_t* transform_rows,
                           const pinsage_neighborhoods_t* nbr, const int32_t* self_rows,
                           void* h_out, int64_t n_out, void* workspace, size_t workspace_bytes,
                           void* stream);

/* Schedule of pinsage_embed_all (Sec. 3.4 leaves it open: the first layer's
 * transform of the pins reads only the features, not the neighbourhoods).
 * A schedule is a caller-owned handle holding two CU-masked streams of the
 * device current at creation and four events: the first layer's transform of
 * a leading share of the pins runs on cu_eighths / 8 of the CUs (whole groups
 * of 8 CUs, spread evenly over the mask) while the walks run on the rest; the
 * share of the pins follows the timing of the last completed call made with
 * the same schedule. The library keeps no stream, event or other device state
 * of its own between calls.
 *   pinsage_schedule_create   cu_eighths in [1, 7]; *out receives the handle.
 *                             Errors: PINSAGE_EINVAL (share, NULL out),
 *                             PINSAGE_EUNSUPPORTED (fewer than 64 CUs),
 *                             PINSAGE_EHIP (stream or event creation; nothing
 *                             is left allocated).
 *   pinsage_schedule_destroy  waits (on the host) for the schedule's streams,
 *                             then destroys them, its events and the handle.
 *                             NULL is a no-op. Call it before the HIP runtime
 *                             (or a profiler attached to it) is torn down, and
 *                             not while another thread uses the handle.
 * Calls that share one schedule are serialised while they enqueue. */
typedef struct pinsage_schedule pinsage_schedule_t;
int pinsage_schedule_create(int32_t cu_eighths, pinsage_schedule_t** out);
int pinsage_schedule_destroy(pinsage_schedule_t* schedule);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * pinsage_convolve_layer without the workspace argument. Its workspace is a
 * static scratch array of PINSAGE_NOALLOC_SCRATCH_BYTES (64 MiB) compiled into
 * the library, one per GPU, held until the process ends; the call itself
 * allocates nothing. Arguments, layout and results are those of
 * pinsage_convolve_layer (same kernels, bit-identical output). A layer whose
 * workspace (pinsage_convolve_workspace_size) exceeds the scratch returns
 * PINSAGE_EUNSUPPORTED and launches nothing. The scratch keeps the last call's
 * contents (every region a call reads is written earlier in that call), and
 * all calls on one GPU share it: calls that overlap on one GPU (two streams,
 * two threads) race and must be serialised by the caller. */
#define PINSAGE_NOALLOC_SCRATCH_BYTES (64ull << 20)
int pinsage_convolve_layer_noalloc(const pinsage_layer_t* layer, const void* h_in,
                                   int64_t n_in, int64_t n_transform,
                                   const int32_t* transform_rows,
                                   const pinsage_neighborhoods_t* nbr, const int32_t* self_rows,
                                   void* h_out, int64_t n_out, void* stream);

/* Workspace bytes needed by pinsage_embed_all. */
int pinsage_embed_all_workspace_size(const pinsage_graph_t* graph,
                                     const pinsage_layer_t* layers, int32_t num_layers,
                                     size_t* bytes);

/* All-node embedding: importance neighbourhoods of every node, then
 * num_layers CONVOLVE layers over all nodes, layer by layer (Sec. 3.4), with
 * h^(0) = x (Sec. 3.2). Only pins are neighbours, so each layer transforms
 * rows [0, num_pins) once. x: device [num_nodes][layers[0].d_in];
 * h_out: device [num_nodes][layers[K-1].d_out]; nbr_out: caller buffers with
 * rows = num_nodes and top_t = walk->top_t (weights may be NULL).
 * layers[k].d_in must equal layers[k-1].d_out; one storage dtype throughout.
 * schedule: NULL (walks, then the transform, in order on `stream`) or a
 * handle from pinsage_schedule_create on the current device (else
 * PINSAGE_EINVAL): with at least 262,144 pins, and at most 4,194,304 unless
 * the first layer is bf16 dense-then-pool with d_in = d_out = 256 (the chained
 * transform) and the graph's walk table fits in the first layer's output
 * buffer of the workspace, the walks and the first layer's transform then run
 * beside each other on its masked streams, forked from and joined back into
 * `stream` by events (also on error returns), so the call stays asynchronous
 * and may be captured into a graph; other pin counts run in order. The
 * output does not depend on the schedule. */
int pinsage_embed_all(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                      const pinsage_layer_t* layers, int32_t num_layers, const void* x,
                      pinsage_neighborhoods_t* nbr_out, void* h_out,
                      unsigned long long* total_steps, void* workspace,
                      size_t workspace_bytes, pinsage_schedule_t* schedule, void* stream);

/* Workspace bytes needed by pinsage_output_mlp for n rows. */
int pinsage_output_mlp_workspace_size(const pinsage_mlp_t* mlp, int64_t n, size_t* bytes);

/* z[r] = G2 ReLU(G1 h[r] + g) for r in [0, n) (Algorithm 2, final loop).
 * h: device [n][d_in], z: device [n][d_out], storage dtype; workspace: device,
 * >= pinsage_output_mlp_workspace_size bytes, 256-aligned. */
int pinsage_output_mlp(const pinsage_mlp_t* mlp, const void* h, int64_t n, void* z,
                       void* workspace, size_t workspace_bytes, void* stream);

/* Max-margin loss, Eq. (1) (Sec. 3.3), with the expectation over negatives
 * taken as the mean over the shared negative set (500 per minibatch in the
 * paper) joined by the pair's own hard negatives (Sec. 3.3, "Hard negative
 * items": they are added to each item's set of negatives):
 *   per_pair[b] = mean over n in zneg u zhard[b] of
 *                 max(0, zq[b].z_n - zq[b].zpos[b] + margin)
 *   *loss       = mean_b per_pair[b]
 * zq, zpos: device [B][d]; zneg: device [n_neg][d]; zhard: device
 * [B][num_hard][d] or NULL when num_hard = 0; storage dtype `dtype`; dot
 * products and sums in fp32 in a fixed order. loss: device fp32 scalar;
 * per_pair: device fp32 [B] (required: the mean is taken over it).
 * Limits: 1 <= B, 1 <= n_neg, 0 <= num_hard, 1 <= d <= 1024. */
int pinsage_max_margin_loss(const void* zq, const void* zpos, int64_t B, const void* zneg,
                            int64_t n_neg, const void* zhard, int64_t num_hard, int32_t d,
                            pinsage_dtype_t dtype, float margin, float* loss, float* per_pair,
                            void* stream);

/* Training pairs of one minibatch (Sec. 3.3): pair b is (queries[b],
 * positives[b]); every pair is scored against the same negatives (the shared
 * negative set of Sec. 3.3) and against its own hard negatives
 * hard_negatives[b][0..num_hard) (e.g. from pinsage_hard_negatives; ids
 * outside [0, num_nodes), such as -1, are absent entries); margin is Delta of
 * Eq. (1). Device int32 node ids; hard_negatives may be NULL when
 * num_hard = 0. */
typedef struct {
  int64_t num_pairs;
  int64_t num_negatives;
  const int32_t* queries;
  const int32_t* positives;
  const int32_t* negatives;
  float margin;
  int64_t num_hard;
  const int32_t* hard_negatives;
} pinsage_pairs_t;

/* Workspace bytes needed by pinsage_minibatch_forward (sized for the largest
 * frontiers: |S^(K)| <= 2B + n_neg + B num_hard, |S^(k-1)| <= |S^(k)| (T + 1),
 * both <= N). */
int pinsage_minibatch_workspace_size(const pinsage_graph_t* graph,
                                     const pinsage_walk_params_t* walk,
                                     const pinsage_layer_t* layers, int32_t num_layers,
                                     const pinsage_mlp_t* mlp, int64_t num_pairs,
                                     int64_t num_negatives, int64_t num_hard, size_t* bytes);

/* Minibatch forward of Algorithm 2 plus the loss of Eq. (1):
 *   S^(K) = queries u positives u negatives u hard negatives;
 *   S^(k-1) = S^(k) u N(S^(k))
 *   (neighbourhoods sampled by the walks of pinsage_build_neighborhoods, so
 *   each equals the node's row of the all-node table); every set is sorted
 *   and de-duplicated on the device and neighbour ids are re-indexed into the
 *   compact sets (Sec. 3.3); then h^(k) = CONVOLVE^(k) for u in S^(k),
 *   k = 1..K, with h^(0) = x (read in place through a row map); then, when
 *   mlp is non-NULL, z = G2 ReLU(G1 h^(K) + g) (Algorithm 2, final loop),
 *   else z = h^(K); and the loss over the pairs on z.
 * x: device [num_nodes][layers[0].d_in]; mlp: NULL or d_in = the last
 * layer's d_out, same dtype; loss: device fp32 scalar; per_pair: device fp32
 * [B] or NULL; z_out: device [2B + n_neg + B num_hard][d] or NULL (d =
 * mlp->d_out, or the last layer's d_out) -- z of queries, then positives, then
 * negatives, then hard negatives (pair-major; zero rows for absent entries);
 * set_sizes: host int64 [K + 1] or NULL -- |S^(0)|, ..., |S^(K)|;
 * total_steps: device uint64 or NULL -- edge steps of all walks of the call.
 * This call synchronises `stream` K + 1 times to size the frontiers.
 * Limits: as for the layers, plus d <= 1024. */
int pinsage_minibatch_forward(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                              const pinsage_layer_t* layers, int32_t num_layers,
                              const pinsage_mlp_t* mlp, const void* x,
                              const pinsage_pairs_t* pairs, float* loss, float* per_pair,
                              void* z_out, int64_t* set_sizes, unsigned long long* total_steps,
                              void* workspace, size_t workspace_bytes, void* stream);

/* Per-kernel timing (hipEvents recorded around every launch on the launch
 * stream). pinsage_profile_enable(1) clears and starts collection;
 * pinsage_profile_read() synchronises the recorded events and returns, for
 * kernel class k (PINSAGE_KERNEL_*), the launch count and total milliseconds.
 * Host-side bookkeeping only; not thread-safe against concurrent launches. */
enum {
  PINSAGE_KERNEL_WALK = 0,
  PINSAGE_KERNEL_GEMM_Q = 1,
  PINSAGE_KERNEL_POOL = 2,
  PINSAGE_KERNEL_GEMM_W = 3,
  PINSAGE_KERNEL_MINIBATCH = 4,
  PINSAGE_KERNEL_LOSS = 5,
  PINSAGE_KERNEL_GEMM_R = 6, /* neighbour half of W per pin (DENSE_THEN_POOL) */
  PINSAGE_KERNEL_MLP = 7,    /* output dense layers */
  PINSAGE_KERNEL_HARD_NEG = 8,
  PINSAGE_KERNEL_GRAPH_NBR = 9, /* graph neighbourhoods (MapReduce variant) */
  PINSAGE_KERNEL_GEMM_QR = 10,  /* Q transform chained into the neighbour half of
                                   W (DENSE_THEN_POOL, bf16, d_in = d_out = 256) */
  PINSAGE_KERNEL_WALK_TABLE = 11, /* the walk table of pinsage_embed_all's walks */
  PINSAGE_KERNEL_POOL_W = 12, /* pool and W fused (DENSE_THEN_POOL, bf16,
                                 d_in = d_out = 256, top_t <= 64) */
  PINSAGE_KERNEL_COUNT = 13
};
int pinsage_profile_enable(int on);
int pinsage_profile_read(int kernel, int64_t* launches, double* total_ms);

/* Random-read calibration (bench support, not part of the method): the chip's
 * rate of dependent random reads, the resource that bounds the walks of
 * Sec. 3.2 (one read of a neighbour id at an unrelated address per edge step).
 * `chains` lanes each make `steps` reads from the table, the index of each read
 * a hash of the value the one before returned, so a lane has one read in
 * flight at a time.
 * table: device, aligned to elem_bytes, table_bytes bytes, contents arbitrary
 *   (never written); the
 *   reads use its first 2^k elements of elem_bytes bytes, 2^k the largest
 *   power of two that fits;
 * elem_bytes: 4, 8 or 16;  steps >= 1;  chains >= 1;
 * sink: device uint32 [chains], written (one value per chain keeps the reads
 *   live). Asynchronous on `stream`; time it with events on that stream.
 * Errors: PINSAGE_EINVAL for a NULL pointer, an element size other than 4, 8
 * or 16, a table smaller than one element, or steps or chains below 1. */
int pinsage_profile_random_reads(const void* table, size_t table_bytes, int32_t elem_bytes,
                                 int32_t steps, uint32_t* sink, int64_t chains, void* stream);

/* Random row gathers (bench support, not part of the method): the rate at
 * which whole rows are gathered from uniformly random positions of a table,
 * in the access pattern of the importance pool (Sec. 3.2, Algorithm 1 line 1:
 * a target's neighbour rows, gathered at unrelated positions). Target t
 * (t < targets) gathers per_target rows; slot s takes row
 * (h * rows) >> 32, h the high 32 bits of the SplitMix64 finaliser of
 * seed + 64 t + s, rows = table_bytes / row_bytes. A wave takes one target at
 * a time and issues all of its loads (two 512-byte rows or one 1 KB row per
 * instruction) before it consumes any.
 * table: device, 16-byte aligned, table_bytes bytes, contents arbitrary
 *   (never written); row_bytes: 512 or 1024; targets >= 1;
 *   1 <= per_target <= 64 (512-byte rows) or 32 (1 KB rows);
 * sink: device uint32, the caller's value plus every gathered 32-bit word
 *   (mod 2^32); the caller zeroes it. Asynchronous on `stream`; time it with
 *   events on that stream.
 * Errors: PINSAGE_EINVAL for a NULL pointer, a misaligned table, another row
 * size, a table smaller than one row or counts out of range;
 * PINSAGE_EUNSUPPORTED for 2^32 rows or more. */
int pinsage_profile_random_gathers(const void* table, size_t table_bytes, int32_t row_bytes,
                                   int64_t targets, int32_t per_target, uint64_t seed,
                                   uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PINSAGE_H_ */
