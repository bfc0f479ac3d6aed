// C ABI of libpinsage.so: argument validation, workspace layout, the
// layer-wise driver (Sec. 3.4) and per-launch timing. Every floating-point or
// graph step runs in the gfx950 kernels; this file only checks arguments and
// sequences launches on the caller's stream (the all-node job may also fork
// the two CU-masked streams of a caller-owned schedule from it and join them
// back).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pinsage.h"
#include "kernels.h"

namespace pinsage {
namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(PINSAGE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
inline size_t elem_size(pinsage_dtype_t t) { return t == PINSAGE_BF16 ? 2 : 4; }

// Rows of the pooled buffer processed per pool + W-GEMM pass: bounds the
// workspace at (chunk x m) elements independent of the node count.
constexpr int64_t kChunkRows = 1ll << 22;

// ---- per-launch timing ----------------------------------------------------
struct Pending {
  int cls;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<Pending> g_pending;
int64_t g_prof_count[kKCount];
double g_prof_ms[kKCount];

int check_graph(const pinsage_graph_t* g) {
  if (!g) return fail(PINSAGE_EINVAL, "graph is NULL");
  if (g->num_pins < 0 || g->num_boards < 0)
    return fail(PINSAGE_EINVAL, "negative node counts (%lld pins, %lld boards)",
                (long long)g->num_pins, (long long)g->num_boards);
  const int64_t n = g->num_pins + g->num_boards;
  if (n <= 0) return fail(PINSAGE_EINVAL, "graph has no nodes");
  if (n >= (1ll << 31) - 1)
    return fail(PINSAGE_EUNSUPPORTED, "num_nodes %lld exceeds int32 node ids", (long long)n);
  if (g->nnz < 0) return fail(PINSAGE_EINVAL, "negative nnz");
  if (g->offset_type != PINSAGE_I32 && g->offset_type != PINSAGE_I64)
    return fail(PINSAGE_EINVAL, "unknown offset_type %d", (int)g->offset_type);
  if (g->offset_type == PINSAGE_I32 && g->nnz >= (1ll << 31))
    return fail(PINSAGE_EUNSUPPORTED, "nnz %lld needs int64 row offsets", (long long)g->nnz);
  if (!g->row_offsets) return fail(PINSAGE_EINVAL, "row_offsets is NULL");
  if (!g->col && g->nnz > 0) return fail(PINSAGE_EINVAL, "col is NULL");
  if (g->walk_table) {
    if (g->nnz > kWalkTableMaxNnz)
      return fail(PINSAGE_EUNSUPPORTED, "nnz %lld too large for a walk table", (long long)g->nnz);
    if (reinterpret_cast<uintptr_t>(g->walk_table) % 16)
      return fail(PINSAGE_EINVAL, "walk_table is not 16-byte aligned");
  }
  return PINSAGE_OK;
}

int check_walk(const pinsage_walk_params_t* w) {
  if (!w) return fail(PINSAGE_EINVAL, "walk params are NULL");
  if (w->walks_per_node < 1 || w->hops < 1)
    return fail(PINSAGE_EINVAL, "walks_per_node (%d) and hops (%d) must be >= 1",
                w->walks_per_node, w->hops);
  if ((int64_t)w->walks_per_node * w->hops > 1024)
    return fail(PINSAGE_EUNSUPPORTED, "walks_per_node * hops = %lld exceeds 1024",
                (long long)w->walks_per_node * w->hops);
  if (w->top_t < 1 || w->top_t > 256)
    return fail(PINSAGE_EUNSUPPORTED, "top_t %d outside [1, 256]", w->top_t);
  return PINSAGE_OK;
}

int check_layer(const pinsage_layer_t* L, int k) {
  if (!L) return fail(PINSAGE_EINVAL, "layer %d is NULL", k);
  if (L->dtype != PINSAGE_F32 && L->dtype != PINSAGE_BF16)
    return fail(PINSAGE_EINVAL, "layer %d: unknown dtype %d", k, (int)L->dtype);
  if (L->d_in <= 0 || L->m <= 0 || L->d_out <= 0)
    return fail(PINSAGE_EINVAL, "layer %d: dims must be positive (%d, %d, %d)", k, L->d_in, L->m,
                L->d_out);
  if (L->d_in % 16 || L->m % 16 || L->d_out % 16)
    return fail(PINSAGE_EUNSUPPORTED, "layer %d: d_in, m, d_out must be multiples of 16", k);
  if (L->d_in > 8192 || L->m > 8192 || L->d_out > 512)
    return fail(PINSAGE_EUNSUPPORTED, "layer %d: dims above limits (d_in, m <= 8192; d_out <= 512)",
                k);
  if (!L->Q || !L->q || !L->W || !L->w)
    return fail(PINSAGE_EINVAL, "layer %d: a parameter pointer is NULL", k);
  if (L->dataflow != PINSAGE_POOL_THEN_DENSE && L->dataflow != PINSAGE_DENSE_THEN_POOL)
    return fail(PINSAGE_EINVAL, "layer %d: unknown dataflow %d", k, (int)L->dataflow);
  if (L->pool != PINSAGE_POOL_IMPORTANCE && L->pool != PINSAGE_POOL_MEAN &&
      L->pool != PINSAGE_POOL_MAX)
    return fail(PINSAGE_EINVAL, "layer %d: unknown pool %d", k, (int)L->pool);
  if (L->pool == PINSAGE_POOL_MAX && L->dataflow == PINSAGE_DENSE_THEN_POOL)
    return fail(PINSAGE_EUNSUPPORTED,
                "layer %d: max pooling is not linear and needs PINSAGE_POOL_THEN_DENSE", k);
  return PINSAGE_OK;
}

int check_mlp(const pinsage_mlp_t* M) {
  if (!M) return fail(PINSAGE_EINVAL, "mlp is NULL");
  if (M->dtype != PINSAGE_F32 && M->dtype != PINSAGE_BF16)
    return fail(PINSAGE_EINVAL, "mlp: unknown dtype %d", (int)M->dtype);
  if (M->d_in <= 0 || M->d_hidden <= 0 || M->d_out <= 0)
    return fail(PINSAGE_EINVAL, "mlp: dims must be positive (%d, %d, %d)", M->d_in, M->d_hidden,
                M->d_out);
  if (M->d_in % 16 || M->d_hidden % 16 || M->d_out % 16)
    return fail(PINSAGE_EUNSUPPORTED, "mlp: d_in, d_hidden, d_out must be multiples of 16");
  if (M->d_in > 8192 || M->d_hidden > 8192 || M->d_out > 8192)
    return fail(PINSAGE_EUNSUPPORTED, "mlp: dims above 8192");
  if (!M->G1 || !M->g || !M->G2) return fail(PINSAGE_EINVAL, "mlp: a parameter pointer is NULL");
  return PINSAGE_OK;
}

size_t mlp_ws(const pinsage_mlp_t* M, int64_t n) {
  const int64_t chunk = n < kChunkRows ? n : kChunkRows;
  return align_up((size_t)chunk * M->d_hidden * elem_size(M->dtype));
}

// z = G2 ReLU(G1 h + g) in row chunks (hidden activations in the workspace).
int run_mlp(const pinsage_mlp_t* M, const void* h, const int32_t* rowmap, int64_t n_h,
            int64_t n, void* z, void* ws, hipStream_t s) {
  const size_t es = elem_size(M->dtype);
  const bool bf16 = M->dtype == PINSAGE_BF16;
  for (int64_t r0 = 0; r0 < n; r0 += kChunkRows) {
    const int64_t rows = (n - r0) < kChunkRows ? (n - r0) : kChunkRows;
    GemmLaunch g1{};
    if (rowmap) {
      g1.A0 = h;
      g1.rowmap = rowmap + r0;
      g1.rows_a0 = n_h;
    } else {
      g1.A0 = static_cast<const unsigned char*>(h) + (size_t)r0 * M->d_in * es;
      g1.rows_a0 = n_h - r0;
    }
    g1.lda0 = M->d_in;
    g1.K0 = M->d_in;
    g1.B = M->G1;
    g1.bias = M->g;
    g1.M = rows;
    g1.N = M->d_hidden;
    g1.C = ws;
    g1.bf16 = bf16;
    g1.relu = true;
    g1.prof_class = kKMlp;
    hipError_t e = launch_gemm(g1, s);
    if (e != hipSuccess) return hip_fail(e, "output layer G1 launch");
    GemmLaunch g2{};
    g2.A0 = ws;
    g2.rows_a0 = rows;
    g2.lda0 = M->d_hidden;
    g2.K0 = M->d_hidden;
    g2.B = M->G2;
    g2.M = rows;
    g2.N = M->d_out;
    g2.C = static_cast<unsigned char*>(z) + (size_t)r0 * M->d_out * es;
    g2.bf16 = bf16;
    g2.prof_class = kKMlp;
    e = launch_gemm(g2, s);
    if (e != hipSuccess) return hip_fail(e, "output layer G2 launch");
  }
  return PINSAGE_OK;
}

int check_nbr(const pinsage_neighborhoods_t* n, int64_t rows, const char* what) {
  if (!n) return fail(PINSAGE_EINVAL, "%s: neighbourhoods are NULL", what);
  if (n->rows != rows)
    return fail(PINSAGE_EINVAL, "%s: neighbourhood rows %lld != %lld", what, (long long)n->rows,
                (long long)rows);
  if (n->top_t < 1 || n->top_t > 256)
    return fail(PINSAGE_EUNSUPPORTED, "%s: top_t %d outside [1, 256]", what, n->top_t);
  if (rows > 0 && (!n->idx || !n->counts))
    return fail(PINSAGE_EINVAL, "%s: idx or counts is NULL", what);
  return PINSAGE_OK;
}

// Workspace of one layer.
//   POOL_THEN_DENSE: P [n_transform][m] | pooled chunk [<= kChunkRows][m]
//   DENSE_THEN_POOL: R [n_transform][d_out] | P chunk [<= kChunkRows][m] |
//                    pooled chunk [<= kChunkRows][d_out]
//   DENSE_THEN_POOL with the chained transform (chain_supported shapes): the
//                    P chunk is replaced by two copies of the reordered W_n'
//                    [d_out][m] (one per stream of the overlapped schedule);
//                    P never exists.
//   DENSE_THEN_POOL, bf16, d_in = d_out = 256: + W_s as product fragments for
//                    the fused pool and W kernel (used when top_t <= 64; the
//                    pooled chunk then stays unused).
struct LayerWs {
  size_t table = 0, pchunk = 0, pooled = 0, wsp = 0;
  bool chained = false;
  size_t total() const { return table + pchunk + pooled + wsp; }
};

bool chained_layer(const pinsage_layer_t* L) {
  return L->dataflow == PINSAGE_DENSE_THEN_POOL &&
         chain_supported(L->d_in, L->m, L->d_out, L->dtype == PINSAGE_BF16);
}

LayerWs layer_ws(const pinsage_layer_t* L, int64_t n_transform, int64_t n_out) {
  const size_t es = elem_size(L->dtype);
  const int64_t out_chunk = n_out < kChunkRows ? n_out : kChunkRows;
  const int64_t tr_chunk = n_transform < kChunkRows ? n_transform : kChunkRows;
  LayerWs w;
  if (L->dataflow == PINSAGE_DENSE_THEN_POOL) {
    w.table = align_up((size_t)n_transform * L->d_out * es);
    w.chained = chained_layer(L);
    w.pchunk = w.chained ? 2 * align_up((size_t)L->d_out * L->m * es)
                         : align_up((size_t)tr_chunk * L->m * es);
    w.pooled = align_up((size_t)out_chunk * L->d_out * es);
    if (pool_w_supported(L->d_in, L->d_out, L->dtype == PINSAGE_BF16, 1))
      w.wsp = align_up(pool_w_ws_bytes());
  } else {
    w.table = align_up((size_t)n_transform * L->m * es);
    w.pooled = align_up((size_t)out_chunk * L->m * es);
  }
  return w;
}

size_t convolve_ws(const pinsage_layer_t* L, int64_t n_transform, int64_t n_out) {
  return layer_ws(L, n_transform, n_out).total();
}

// Algorithm 1 line 1 for rows [c0, c0 + rows) of the transformed set:
// C = ReLU(h_in[t(i)] Q^T + q).
hipError_t launch_transform(const pinsage_layer_t* L, const void* h_in, int64_t n_in,
                            const int32_t* transform_rows, int64_t c0, int64_t rows, void* C,
                            hipStream_t s) {
  const size_t es = elem_size(L->dtype);
  GemmLaunch g{};
  if (transform_rows) {
    g.A0 = h_in;
    g.rowmap = transform_rows + c0;
    g.rows_a0 = n_in;
  } else {
    g.A0 = static_cast<const unsigned char*>(h_in) + (size_t)c0 * L->d_in * es;
    g.rows_a0 = n_in - c0;
  }
  g.lda0 = L->d_in;
  g.K0 = L->d_in;
  g.B = L->Q;
  g.bias = L->q;
  g.M = rows;
  g.N = L->m;
  g.C = C;
  g.bf16 = L->dtype == PINSAGE_BF16;
  g.relu = true;
  g.row_base = c0;
  return launch_gemm(g, s);
}

// Layer bodies shared by convolve_layer, embed_all and the minibatch forward;
// arguments already valid. Phase 1 fills the per-pin table of the workspace (P,
// or R = P W_n^T when split); phase 2 pools it and applies W.
//
// Phase 1 for the transformable rows [r0, r1) only. When split, the P chunk
// buffer is used from row `pbase` on (chunks of kChunkRows - pbase rows), so two
// row ranges with disjoint P rows can run on two streams at once.
int run_transform_rows(const pinsage_layer_t* L, const void* h_in, int64_t n_in,
                       int64_t n_transform, const int32_t* transform_rows, int64_t n_out,
                       void* ws, int64_t r0, int64_t r1, int64_t pbase, hipStream_t s) {
  const bool bf16 = L->dtype == PINSAGE_BF16;
  const size_t es = elem_size(L->dtype);
  const LayerWs lw = layer_ws(L, n_transform, n_out);
  unsigned char* table = static_cast<unsigned char*>(ws);  // P, or R when split
  hipError_t e;
  if (r1 <= r0) return PINSAGE_OK;
  if (L->dataflow != PINSAGE_DENSE_THEN_POOL) {
    // Algorithm 1 line 1, once per transformable row (Sec. 3.4).
    e = launch_transform(L, h_in, n_in, transform_rows, r0, r1 - r0,
                         table + (size_t)r0 * L->m * es, s);
    if (e != hipSuccess) return hip_fail(e, "Q transform launch");
    return PINSAGE_OK;
  }
  if (lw.chained) {
    // R = ReLU(h Q^T + q) W_n^T in one kernel over the rows; this stream's
    // copy of the reordered W_n' first.
    unsigned char* wp = table + lw.table + (pbase > 0 ? lw.pchunk / 2 : 0);
    e = launch_permute_wn(L->W, (int64_t)L->d_in + L->m, L->d_in, L->m, L->d_out, wp, s);
    if (e != hipSuccess) return hip_fail(e, "W_n reorder launch");
    ChainLaunch c{};
    c.H = h_in;
    c.rowmap = transform_rows ? transform_rows + r0 : nullptr;
    c.row0 = r0;
    c.rows_h = n_in;
    c.ldh = L->d_in;
    c.Q = L->Q;
    c.q = L->q;
    c.Wp = wp;
    c.d_in = L->d_in;
    c.m = L->m;
    c.d_out = L->d_out;
    c.R = table + (size_t)r0 * L->d_out * es;
    c.ldr = L->d_out;
    c.rows = r1 - r0;
    e = launch_chain(c, s);
    if (e != hipSuccess) return hip_fail(e, "chained transform launch");
    return PINSAGE_OK;
  }
  // Per chunk of pins: P = ReLU(h Q^T + q), then R = P W_n^T with W_n the
  // neighbour columns [d_in, d_in + m) of W (row stride d_in + m).
  unsigned char* pchunk = table + lw.table + (size_t)pbase * L->m * es;
  const int64_t cs = kChunkRows - pbase;
  for (int64_t c0 = r0; c0 < r1; c0 += cs) {
    const int64_t rows = (r1 - c0) < cs ? (r1 - c0) : cs;
    e = launch_transform(L, h_in, n_in, transform_rows, c0, rows, pchunk, s);
    if (e != hipSuccess) return hip_fail(e, "Q transform launch");
    GemmLaunch gr{};
    gr.A0 = pchunk;
    gr.rows_a0 = rows;
    gr.lda0 = L->m;
    gr.K0 = L->m;
    gr.B = static_cast<const unsigned char*>(L->W) + (size_t)L->d_in * es;
    gr.ldb = (int64_t)L->d_in + L->m;
    gr.M = rows;
    gr.N = L->d_out;
    gr.C = table + (size_t)c0 * L->d_out * es;
    gr.bf16 = bf16;
    gr.row_base = c0;
    e = launch_gemm(gr, s);
    if (e != hipSuccess) return hip_fail(e, "neighbour-half W launch");
  }
  return PINSAGE_OK;
}

int run_transform(const pinsage_layer_t* L, const void* h_in, int64_t n_in, int64_t n_transform,
                  const int32_t* transform_rows, int64_t n_out, void* ws, hipStream_t s) {
  return run_transform_rows(L, h_in, n_in, n_transform, transform_rows, n_out, ws, 0,
                            n_transform, 0, s);
}

int run_pool_dense(const pinsage_layer_t* L, const void* h_in, int64_t n_in,
                   int64_t n_transform, const pinsage_neighborhoods_t* nbr,
                   const int32_t* self_rows, void* h_out, int64_t n_out, void* ws,
                   hipStream_t s) {
  const bool bf16 = L->dtype == PINSAGE_BF16;
  const bool split = L->dataflow == PINSAGE_DENSE_THEN_POOL;
  const size_t es = elem_size(L->dtype);
  const LayerWs lw = layer_ws(L, n_transform, n_out);
  unsigned char* table = static_cast<unsigned char*>(ws);
  unsigned char* nbuf = table + lw.table + lw.pchunk;
  const int pool_width = split ? L->d_out : L->m;
  hipError_t e;
  if (lw.wsp && pool_w_supported(L->d_in, L->d_out, bf16, nbr->top_t)) {
    // Pool and W in one kernel over all rows: no pooled chunk, no separate GEMM.
    unsigned char* wsp = nbuf + lw.pooled;
    e = launch_permute_ws(L->W, (int64_t)L->d_in + L->m, wsp, s);
    if (e != hipSuccess) return hip_fail(e, "W_s permute launch");
    PoolWLaunch pw{};
    pw.R = table;
    pw.n_transform = n_transform;
    pw.idx = nbr->idx;
    pw.counts = nbr->counts;
    pw.weights = nbr->weights;
    pw.T = nbr->top_t;
    pw.mode = (int)L->pool;
    pw.H = h_in;
    pw.self_rows = self_rows;
    pw.h_row0 = 0;
    pw.rows_h = n_in;
    pw.ldh = L->d_in;
    pw.Wsp = wsp;
    pw.bias = L->w;
    pw.out = h_out;
    pw.rows = n_out;
    e = launch_pool_w(pw, s);
    if (e != hipSuccess) return hip_fail(e, "pool and W launch");
    return PINSAGE_OK;
  }
  for (int64_t r0 = 0; r0 < n_out; r0 += kChunkRows) {
    const int64_t rows = (n_out - r0) < kChunkRows ? (n_out - r0) : kChunkRows;
    const int T = nbr->top_t;
    PoolLaunch pl{};
    pl.P = table;
    pl.n_transform = n_transform;
    pl.m = pool_width;
    pl.bf16 = bf16;
    pl.idx = nbr->idx + r0 * T;
    pl.counts = nbr->counts + r0 * T;
    pl.weights = nbr->weights ? nbr->weights + r0 * T : nullptr;
    pl.T = T;
    pl.rows = rows;
    pl.out = nbuf;
    pl.mode = (int)L->pool;
    e = launch_pool(pl, s);
    if (e != hipSuccess) return hip_fail(e, "pool launch");

    // Algorithm 1 lines 2-3: on [h_self | n] with all of W, or (split) on
    // h_self with the self columns of W plus the pooled R rows.
    GemmLaunch gw{};
    if (self_rows) {
      gw.A0 = h_in;
      gw.rowmap = self_rows + r0;
    } else {
      gw.A0 = static_cast<const unsigned char*>(h_in) + (size_t)r0 * L->d_in * es;
      gw.rowmap = nullptr;
    }
    gw.rows_a0 = self_rows ? n_in : (n_in - r0);
    gw.lda0 = L->d_in;
    gw.K0 = L->d_in;
    if (split) {
      gw.ldb = (int64_t)L->d_in + L->m;
      gw.addend = nbuf;
    } else {
      gw.A1 = nbuf;
      gw.lda1 = L->m;
      gw.K1 = L->m;
    }
    gw.B = L->W;
    gw.bias = L->w;
    gw.M = rows;
    gw.N = L->d_out;
    gw.C = static_cast<unsigned char*>(h_out) + (size_t)r0 * L->d_out * es;
    gw.bf16 = bf16;
    gw.relu = true;
    gw.l2norm = true;
    gw.row_base = r0;
    e = launch_gemm(gw, s);
    if (e != hipSuccess) return hip_fail(e, "W transform launch");
  }
  return PINSAGE_OK;
}

int run_layer(const pinsage_layer_t* L, const void* h_in, int64_t n_in, int64_t n_transform,
              const int32_t* transform_rows, const pinsage_neighborhoods_t* nbr,
              const int32_t* self_rows, void* h_out, int64_t n_out, void* ws, hipStream_t s) {
  int st = run_transform(L, h_in, n_in, n_transform, transform_rows, n_out, ws, s);
  if (st) return st;
  return run_pool_dense(L, h_in, n_in, n_transform, nbr, self_rows, h_out, n_out, ws, s);
}

// ---- walks beside the first layer's transform (embed_all) -----------------
// The first layer's transform reads only x, so it can run while the
// neighbourhood walks run. The walks are bound by dependent random reads and
// leave the matrix cores idle; the GEMM blocks take whole CUs. Both therefore
// run on CU-masked streams forked from the caller's stream: the transform of
// the first `a` pins on a side stream holding a share of the CUs, the walks on
// the other CUs. The remaining pins are transformed on the caller's stream
// (all CUs) once the walks are done, and the pool waits for both. The masked
// streams and the events belong to a caller-owned pinsage_schedule_t
// (created and destroyed by explicit calls); the library keeps none.
//
// `a` comes from the last call on the schedule whose events have completed:
// with side rate rs and full-chip rate rf (rows per ms) and walk time tw, the
// side and the caller's stream end together when a / rs = tw + (P - a) / rf,
// i.e. a = rs (rf tw + P) / (rf + rs). The GEMMs sum every row in the same
// order whatever the split, so the output does not depend on `a`.
//
// Masks: byte j of the CU mask (8 consecutive CUs) goes to the side when
// floor((j + 1) k / 8) > floor(j k / 8), k = the share in eighths, which spreads
// the side's bytes evenly over the mask words.

// Pin counts that overlap: at least 2^18, and at most one transform chunk
// unless the first layer is chained and the walk table fits beside it. Larger
// graphs walking the CSR (two dependent reads per step) slowed by more than the
// transform share saved (measured on 10M pins); the table's single read per
// step keeps its rate on 7/8 of the CUs.
constexpr int64_t kMinOverlapRows = 1ll << 18;
constexpr int64_t kMaxOverlapRows = kChunkRows;

void schedule_release(pinsage_schedule* o);

// The side's rows for this call, after folding in the last call's timing when
// its events have completed. While the caller's stream is being captured into
// a graph the events are neither read nor marked for reading (their records
// are graph nodes, not timings). With o->mu held.
int64_t overlap_rows(pinsage_schedule& o, int64_t n_transform, bool capturing);
}  // namespace
}  // namespace pinsage

// A caller-owned schedule of pinsage_embed_all: two CU-masked streams of one
// device, the events that fork and join them, and the timing that sets the
// side's share of the pins.
struct pinsage_schedule {
  int device = 0;
  int eighths = 0;
  std::mutex mu;
  hipStream_t side = nullptr, walk = nullptr;
  hipEvent_t fork = nullptr, side_done = nullptr, walk_done = nullptr, main_done = nullptr;
  double alpha = 0.0;       // side rows / transformable rows for the next call
  double rf_over_rs = 0.0;  // full-chip rate over side rate, last measured
  int64_t side_rows = 0, main_rows = 0, total_rows = 0;  // of the last call
  bool pending = false;     // the last call's events have not been read
};

namespace pinsage {
namespace {

// Waits for and destroys a schedule's streams and events (its device made
// current for the calls), then frees it.
void schedule_release(pinsage_schedule* o) {
  int cur = 0;
  const bool restore = hipGetDevice(&cur) == hipSuccess;
  (void)hipSetDevice(o->device);
  for (hipStream_t st : {o->side, o->walk}) {
    if (!st) continue;
    (void)hipStreamSynchronize(st);
    (void)hipStreamDestroy(st);
  }
  for (hipEvent_t ev : {o->fork, o->side_done, o->walk_done, o->main_done})
    if (ev) (void)hipEventDestroy(ev);
  if (restore) (void)hipSetDevice(cur);
  (void)hipGetLastError();
  delete o;
}

int64_t overlap_rows(pinsage_schedule& o, int64_t n_transform, bool capturing) {
  if (!capturing && o.pending && hipEventQuery(o.main_done) == hipSuccess &&
      hipEventQuery(o.side_done) == hipSuccess) {
    float ts = 0.0f, tw = 0.0f, tm = 0.0f;
    const bool timed = hipEventElapsedTime(&ts, o.fork, o.side_done) == hipSuccess &&
                       hipEventElapsedTime(&tw, o.fork, o.walk_done) == hipSuccess &&
                       hipEventElapsedTime(&tm, o.walk_done, o.main_done) == hipSuccess;
    if (timed && ts > 0.0f && o.side_rows > 0) {
      const double rs = (double)o.side_rows / ts;
      if (o.main_rows > 0 && tm > 0.0f) o.rf_over_rs = ((double)o.main_rows / tm) / rs;
      const double rf = rs * o.rf_over_rs;
      const double want = rs * (rf * tw + (double)o.total_rows) / (rf + rs);
      const double frac = want / (double)o.total_rows;
      o.alpha = frac < 0.05 ? 0.05 : (frac > 1.0 ? 1.0 : frac);  // keep measuring
    }
    o.pending = false;
  }
  (void)hipGetLastError();  // a not-ready query is not an error
  const int64_t a = (int64_t)(o.alpha * (double)n_transform) / 256 * 256;
  return a > n_transform ? n_transform : a;
}
}  // namespace

ProfileScope::ProfileScope(int cls, hipStream_t s) : cls_(cls), s_(s) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof_on) return;
  if (hipEventCreate(&start_) != hipSuccess) {
    start_ = nullptr;
    return;
  }
  (void)hipEventRecord(start_, s_);
}

ProfileScope::~ProfileScope() {
  if (!start_) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  hipEvent_t stop = nullptr;
  if (hipEventCreate(&stop) != hipSuccess) {
    (void)hipEventDestroy(start_);
    return;
  }
  (void)hipEventRecord(stop, s_);
  g_pending.push_back({cls_, start_, stop});
}

}  // namespace pinsage

using namespace pinsage;

extern "C" {

int pinsage_version(void) { return PINSAGE_ABI_VERSION; }

const char* pinsage_status_string(int status) {
  switch (status) {
    case PINSAGE_OK: return "ok";
    case PINSAGE_EINVAL: return "invalid argument";
    case PINSAGE_EUNSUPPORTED: return "unsupported argument";
    case PINSAGE_EWORKSPACE: return "workspace too small";
    case PINSAGE_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* pinsage_last_error(void) { return g_last_error.c_str(); }

// Bytes of a graph's walk table (0 when nnz is too large for one).
static size_t walk_table_bytes(const pinsage_graph_t* g) {
  return g->nnz > 0 && g->nnz <= kWalkTableMaxNnz ? align_up((size_t)g->nnz * 16) : 0;
}

// The walks and top-T of validated arguments; `table` is the graph's walk
// table or NULL (read the CSR).
static int run_walks(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                     const int32_t* sources, int64_t num_sources, pinsage_neighborhoods_t* out,
                     unsigned long long* total_steps, const void* table, hipStream_t s) {
  if (total_steps) {
    hipError_t e = launch_zero_u64(total_steps, 1, s);
    if (e != hipSuccess) return hip_fail(e, "step counter reset");
  }
  WalkLaunch a{};
  a.row_offsets = graph->row_offsets;
  a.offsets64 = graph->offset_type == PINSAGE_I64;
  a.col = graph->col;
  a.nnz = graph->nnz;
  a.num_pins = graph->num_pins;
  a.num_nodes = graph->num_pins + graph->num_boards;
  a.sources = sources;
  a.num_sources = num_sources;
  a.seed = walk->seed;
  a.walks = walk->walks_per_node;
  a.hops = walk->hops;
  a.top_t = walk->top_t;
  a.idx = out->idx;
  a.counts = out->counts;
  a.weights = out->weights;
  a.total_steps = total_steps;
  a.table = table;
  hipError_t e = launch_walk_topt(a, s);
  if (e != hipSuccess) return hip_fail(e, "walk launch");
  return PINSAGE_OK;
}

int pinsage_build_neighborhoods(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                                const int32_t* sources, int64_t num_sources,
                                pinsage_neighborhoods_t* out, unsigned long long* total_steps,
                                void* stream) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  if ((st = check_walk(walk))) return st;
  const int64_t n = graph->num_pins + graph->num_boards;
  if (num_sources < 0) return fail(PINSAGE_EINVAL, "negative num_sources");
  if (!sources && num_sources != n)
    return fail(PINSAGE_EINVAL, "sources is NULL but num_sources (%lld) != num_nodes (%lld)",
                (long long)num_sources, (long long)n);
  if ((st = check_nbr(out, num_sources, "build_neighborhoods"))) return st;
  if (out->top_t != walk->top_t)
    return fail(PINSAGE_EINVAL, "out->top_t %d != walk->top_t %d", out->top_t, walk->top_t);
  return run_walks(graph, walk, sources, num_sources, out, total_steps, graph->walk_table,
                   static_cast<hipStream_t>(stream));
}

int pinsage_walk_table_size(const pinsage_graph_t* graph, size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  *bytes = 0;
  const int st = check_graph(graph);
  if (st) return st;
  if (graph->nnz > kWalkTableMaxNnz)
    return fail(PINSAGE_EUNSUPPORTED, "nnz %lld too large for a walk table",
                (long long)graph->nnz);
  *bytes = (size_t)graph->nnz * 16;
  return PINSAGE_OK;
}

int pinsage_build_walk_table(const pinsage_graph_t* graph, void* table, size_t table_bytes,
                             void* stream) {
  g_last_error.clear();
  size_t need = 0;
  const int st = pinsage_walk_table_size(graph, &need);
  if (st) return st;
  if (!table && need > 0) return fail(PINSAGE_EINVAL, "table is NULL");
  if (table_bytes < need)
    return fail(PINSAGE_EWORKSPACE, "table %zu bytes < required %zu", table_bytes, need);
  if (reinterpret_cast<uintptr_t>(table) % 16)
    return fail(PINSAGE_EINVAL, "table is not 16-byte aligned");
  if (need == 0) return PINSAGE_OK;
  const hipError_t e =
      launch_walk_table(graph->row_offsets, graph->offset_type == PINSAGE_I64, graph->col,
                        graph->nnz, graph->num_pins + graph->num_boards, table,
                        static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "walk table launch");
  return PINSAGE_OK;
}

static int check_hard_negative_params(const pinsage_hard_negative_params_t* params,
                                      int64_t num_queries) {
  if (!params) return fail(PINSAGE_EINVAL, "hard negative params are NULL");
  const pinsage_hard_negative_params_t& h = *params;
  if (h.walks < 1 || h.hops < 1)
    return fail(PINSAGE_EINVAL, "walks (%d) and hops (%d) must be >= 1", h.walks, h.hops);
  const int64_t landings = (int64_t)h.walks * h.hops;
  if (landings > kMaxLandings)
    return fail(PINSAGE_EUNSUPPORTED, "walks * hops = %lld exceeds %lld", (long long)landings,
                (long long)kMaxLandings);
  if (h.rank_lo < 0 || h.rank_hi <= h.rank_lo)
    return fail(PINSAGE_EINVAL, "rank window [%d, %d) is empty or negative", h.rank_lo,
                h.rank_hi);
  if (landings > kMaxOnChipLandings && h.rank_hi > kMaxGlobalRank)
    return fail(PINSAGE_EUNSUPPORTED,
                "rank_hi %d exceeds %d for walks * hops above %lld", h.rank_hi, kMaxGlobalRank,
                (long long)kMaxOnChipLandings);
  if (h.num_per_query < 0) return fail(PINSAGE_EINVAL, "negative num_per_query");
  if (num_queries < 0) return fail(PINSAGE_EINVAL, "negative num_queries");
  return PINSAGE_OK;
}

int pinsage_hard_negatives_workspace_size(const pinsage_hard_negative_params_t* params,
                                          int64_t num_queries, size_t* bytes) {
  g_last_error.clear();
  int st = check_hard_negative_params(params, num_queries);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  *bytes = hard_negative_workspace((int64_t)params->walks * params->hops, num_queries);
  return PINSAGE_OK;
}

int pinsage_hard_negatives(const pinsage_graph_t* graph,
                           const pinsage_hard_negative_params_t* params, const int32_t* queries,
                           int64_t num_queries, int32_t* out, unsigned long long* total_steps,
                           void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  if ((st = check_hard_negative_params(params, num_queries))) return st;
  const pinsage_hard_negative_params_t& h = *params;
  if (num_queries > 0 && !queries) return fail(PINSAGE_EINVAL, "queries is NULL");
  if (num_queries > 0 && h.num_per_query > 0 && !out) return fail(PINSAGE_EINVAL, "out is NULL");
  const size_t need = hard_negative_workspace((int64_t)h.walks * h.hops, num_queries);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (total_steps) {
    hipError_t e = launch_zero_u64(total_steps, 1, s);
    if (e != hipSuccess) return hip_fail(e, "step counter reset");
  }
  if (num_queries == 0 || (h.num_per_query == 0 && !total_steps)) return PINSAGE_OK;
  HardNegLaunch a{};
  a.row_offsets = graph->row_offsets;
  a.offsets64 = graph->offset_type == PINSAGE_I64;
  a.col = graph->col;
  a.nnz = graph->nnz;
  a.num_pins = graph->num_pins;
  a.num_nodes = graph->num_pins + graph->num_boards;
  a.queries = queries;
  a.num_queries = num_queries;
  a.seed = h.seed;
  a.walks = h.walks;
  a.hops = h.hops;
  a.rank_lo = h.rank_lo;
  a.rank_hi = h.rank_hi;
  a.k = h.num_per_query;
  a.out = out;
  a.total_steps = total_steps;
  a.table = graph->walk_table;
  hipError_t e = launch_hard_negatives(a, workspace, s);
  if (e != hipSuccess) return hip_fail(e, "hard negative launch");
  return PINSAGE_OK;
}

int pinsage_build_graph_neighborhoods(const pinsage_graph_t* graph, uint64_t seed,
                                      const int32_t* sources, int64_t num_sources,
                                      pinsage_neighborhoods_t* out, void* stream) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  const int64_t n = graph->num_pins + graph->num_boards;
  if (num_sources < 0) return fail(PINSAGE_EINVAL, "negative num_sources");
  if (!sources && num_sources != n)
    return fail(PINSAGE_EINVAL, "sources is NULL but num_sources (%lld) != num_nodes (%lld)",
                (long long)num_sources, (long long)n);
  if ((st = check_nbr(out, num_sources, "build_graph_neighborhoods"))) return st;
  GraphNbrLaunch a{};
  a.row_offsets = graph->row_offsets;
  a.offsets64 = graph->offset_type == PINSAGE_I64;
  a.col = graph->col;
  a.nnz = graph->nnz;
  a.num_nodes = n;
  a.sources = sources;
  a.num_sources = num_sources;
  a.seed = seed;
  a.top_t = out->top_t;
  a.idx = out->idx;
  a.counts = out->counts;
  a.weights = out->weights;
  hipError_t e = launch_graph_neighborhoods(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "graph neighbourhood launch");
  return PINSAGE_OK;
}

}  // extern "C"

namespace pinsage {
namespace {
// Workspace of the bipartite all-node job: the layers' workspace (every node
// projected), the h ping-pong buffers, the pin row map of layer 1.
struct BipartiteWs {
  size_t conv = 0, h = 0, map = 0;
  int hbufs = 0;
  size_t total() const { return conv + (size_t)hbufs * h + map; }
};
int bipartite_ws(const pinsage_graph_t* graph, const pinsage_layer_t* layers, int32_t K,
                 BipartiteWs* w) {
  int st;
  if (K < 1 || !layers) return fail(PINSAGE_EINVAL, "need at least one layer");
  if (K % 2)
    return fail(PINSAGE_EUNSUPPORTED,
                "num_layers %d is odd: with featureless boards the layers must be even", K);
  const int64_t n = graph->num_pins + graph->num_boards;
  for (int k = 0; k < K; ++k) {
    if ((st = check_layer(&layers[k], k))) return st;
    if (layers[k].dtype != layers[0].dtype)
      return fail(PINSAGE_EINVAL, "layer %d dtype differs from layer 0", k);
    if (k > 0 && layers[k].d_in != layers[k - 1].d_out)
      return fail(PINSAGE_EINVAL, "layer %d d_in %d != layer %d d_out %d", k, layers[k].d_in,
                  k - 1, layers[k - 1].d_out);
    const size_t c = convolve_ws(&layers[k], n, n);
    w->conv = c > w->conv ? c : w->conv;
    if (k + 1 < K) {
      const size_t hb = align_up((size_t)n * layers[k].d_out * elem_size(layers[k].dtype));
      w->h = hb > w->h ? hb : w->h;
    }
  }
  w->hbufs = K > 2 ? 2 : (K > 1 ? 1 : 0);
  w->map = align_up((size_t)n * 4);
  return PINSAGE_OK;
}

// Host-side checks shared by the two convolve_layer entry points.
int check_convolve(const pinsage_layer_t* layer, const void* h_in, int64_t n_in,
                   int64_t n_transform, const int32_t* transform_rows,
                   const pinsage_neighborhoods_t* nbr, const int32_t* self_rows, void* h_out,
                   int64_t n_out) {
  int st = check_layer(layer, 0);
  if (st) return st;
  if (n_in < 0 || n_transform < 0 || n_out < 0) return fail(PINSAGE_EINVAL, "negative row count");
  if (!transform_rows && n_transform > n_in)
    return fail(PINSAGE_EINVAL, "n_transform (%lld) > n_in (%lld) without transform_rows",
                (long long)n_transform, (long long)n_in);
  if (!self_rows && n_out > n_in)
    return fail(PINSAGE_EINVAL, "n_out (%lld) > n_in (%lld) without self_rows", (long long)n_out,
                (long long)n_in);
  if ((st = check_nbr(nbr, n_out, "convolve_layer"))) return st;
  if (n_out == 0 && n_transform == 0) return PINSAGE_OK;
  if ((n_in > 0 && !h_in) || (n_out > 0 && !h_out))
    return fail(PINSAGE_EINVAL, "h_in or h_out is NULL");
  return PINSAGE_OK;
}

// Scratch of pinsage_convolve_layer_noalloc: a file-scope device array, one
// copy per GPU at its own address, held until the process ends. Host code
// never uses the array's name as a device address: the address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// is kept per device.
constexpr size_t kScratchBytes = (size_t)PINSAGE_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

int scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "current device");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(PINSAGE_EUNSUPPORTED, "device %d outside the %d devices with scratch", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "scratch symbol address");
    if (!p) return fail(PINSAGE_EHIP, "scratch symbol address is NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PINSAGE_OK;
}
}  // namespace
}  // namespace pinsage

extern "C" {

int pinsage_embed_all_bipartite_workspace_size(const pinsage_graph_t* graph,
                                               const pinsage_layer_t* layers,
                                               int32_t num_layers, size_t* bytes) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  BipartiteWs w;
  if ((st = bipartite_ws(graph, layers, num_layers, &w))) return st;
  *bytes = w.total();
  return PINSAGE_OK;
}

int pinsage_embed_all_bipartite(const pinsage_graph_t* graph, uint64_t seed,
                                const pinsage_layer_t* layers, int32_t num_layers,
                                const void* x_pins, pinsage_neighborhoods_t* nbr_out,
                                void* h_out, void* workspace, size_t workspace_bytes,
                                void* stream) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  BipartiteWs w;
  if ((st = bipartite_ws(graph, layers, num_layers, &w))) return st;
  const int64_t n = graph->num_pins + graph->num_boards;
  if ((st = check_nbr(nbr_out, n, "embed_all_bipartite"))) return st;
  if (!x_pins || !h_out) return fail(PINSAGE_EINVAL, "x_pins or h_out is NULL");
  if (!workspace || workspace_bytes < w.total())
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes,
                w.total());
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");
  if ((st = pinsage_build_graph_neighborhoods(graph, seed, nullptr, n, nbr_out, stream)))
    return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  unsigned char* hbuf[2] = {ws + w.conv, ws + w.conv + w.h};
  int32_t* pin_map = reinterpret_cast<int32_t*>(ws + w.conv + (size_t)w.hbufs * w.h);
  // Layer 1 reads x through a row map: pins are rows of x, boards (no
  // features) read as zero rows, for both the projection and the self half.
  hipError_t e = launch_row_map(pin_map, n, graph->num_pins, s);
  if (e != hipSuccess) return hip_fail(e, "row map");
  const void* cur = x_pins;
  for (int k = 0; k < num_layers; ++k) {
    void* dst = (k == num_layers - 1) ? h_out : hbuf[k % 2];
    if (k == 0)
      st = run_layer(&layers[k], cur, graph->num_pins, n, pin_map, nbr_out, pin_map, dst, n, ws, s);
    else
      st = run_layer(&layers[k], cur, n, n, nullptr, nbr_out, nullptr, dst, n, ws, s);
    if (st) return st;
    cur = dst;
  }
  return PINSAGE_OK;
}

int pinsage_convolve_workspace_size(const pinsage_layer_t* layer, int64_t n_transform,
                                    int64_t n_out, size_t* bytes) {
  g_last_error.clear();
  int st = check_layer(layer, 0);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  if (n_transform < 0 || n_out < 0) return fail(PINSAGE_EINVAL, "negative row count");
  *bytes = convolve_ws(layer, n_transform, n_out);
  return PINSAGE_OK;
}

int pinsage_convolve_layer(const pinsage_layer_t* layer, const void* h_in, int64_t n_in,
                           int64_t n_transform, const int32_t* transform_rows,
                           const pinsage_neighborhoods_t* nbr, const int32_t* self_rows,
                           void* h_out, int64_t n_out, void* workspace, size_t workspace_bytes,
                           void* stream) {
  g_last_error.clear();
  int st = check_convolve(layer, h_in, n_in, n_transform, transform_rows, nbr, self_rows, h_out,
                          n_out);
  if (st) return st;
  if (n_out == 0 && n_transform == 0) return PINSAGE_OK;
  const size_t need = convolve_ws(layer, n_transform, n_out);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");
  return run_layer(layer, h_in, n_in, n_transform, transform_rows, nbr, self_rows, h_out, n_out,
                   workspace, static_cast<hipStream_t>(stream));
}

int pinsage_convolve_layer_noalloc(const pinsage_layer_t* layer, const void* h_in, int64_t n_in,
                                   int64_t n_transform, const int32_t* transform_rows,
                                   const pinsage_neighborhoods_t* nbr, const int32_t* self_rows,
                                   void* h_out, int64_t n_out, void* stream) {
  g_last_error.clear();
  int st = check_convolve(layer, h_in, n_in, n_transform, transform_rows, nbr, self_rows, h_out,
                          n_out);
  if (st) return st;
  if (n_out == 0 && n_transform == 0) return PINSAGE_OK;
  const size_t need = convolve_ws(layer, n_transform, n_out);
  if (need > kScratchBytes)
    return fail(PINSAGE_EUNSUPPORTED,
                "layer needs %zu bytes of scratch (n_transform %lld, n_out %lld); the static "
                "scratch holds %zu",
                need, (long long)n_transform, (long long)n_out, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws))) return st;
  // Every scratch region the layer reads (P or R rows, the pooled chunk) is
  // written earlier in the same call, so nothing has to start at zero.
  return run_layer(layer, h_in, n_in, n_transform, transform_rows, nbr, self_rows, h_out, n_out,
                   ws, static_cast<hipStream_t>(stream));
}

int pinsage_embed_all_workspace_size(const pinsage_graph_t* graph, const pinsage_layer_t* layers,
                                     int32_t num_layers, size_t* bytes) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  if (num_layers < 1 || !layers) return fail(PINSAGE_EINVAL, "need at least one layer");
  const int64_t n = graph->num_pins + graph->num_boards;
  size_t conv = 0, h = 0;
  for (int k = 0; k < num_layers; ++k) {
    if ((st = check_layer(&layers[k], k))) return st;
    const size_t c = convolve_ws(&layers[k], graph->num_pins, n);
    conv = c > conv ? c : conv;
    if (k + 1 < num_layers) {
      const size_t hb = align_up((size_t)n * layers[k].d_out * elem_size(layers[k].dtype));
      h = hb > h ? hb : h;
    }
  }
  const int hbufs = num_layers > 2 ? 2 : (num_layers > 1 ? 1 : 0);
  // The walk table shares the layers' region: the in-order walks finish before
  // the first transform writes it.
  const size_t tb = walk_table_bytes(graph);
  *bytes = (conv > tb ? conv : tb) + (size_t)hbufs * h;
  return PINSAGE_OK;
}

int pinsage_embed_all(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                      const pinsage_layer_t* layers, int32_t num_layers, const void* x,
                      pinsage_neighborhoods_t* nbr_out, void* h_out,
                      unsigned long long* total_steps, void* workspace, size_t workspace_bytes,
                      pinsage_schedule_t* schedule, void* stream) {
  g_last_error.clear();
  int st = check_graph(graph);
  if (st) return st;
  if ((st = check_walk(walk))) return st;
  if (num_layers < 1 || !layers) return fail(PINSAGE_EINVAL, "need at least one layer");
  for (int k = 0; k < num_layers; ++k) {
    if ((st = check_layer(&layers[k], k))) return st;
    if (layers[k].dtype != layers[0].dtype)
      return fail(PINSAGE_EINVAL, "layer %d dtype differs from layer 0", k);
    if (k > 0 && layers[k].d_in != layers[k - 1].d_out)
      return fail(PINSAGE_EINVAL, "layer %d d_in %d != layer %d d_out %d", k, layers[k].d_in,
                  k - 1, layers[k - 1].d_out);
  }
  const int64_t n = graph->num_pins + graph->num_boards;
  if ((st = check_nbr(nbr_out, n, "embed_all"))) return st;
  if (nbr_out->top_t != walk->top_t)
    return fail(PINSAGE_EINVAL, "nbr_out->top_t %d != walk->top_t %d", nbr_out->top_t,
                walk->top_t);
  if (!x || !h_out) return fail(PINSAGE_EINVAL, "x or h_out is NULL");
  size_t need = 0;
  if ((st = pinsage_embed_all_workspace_size(graph, layers, num_layers, &need))) return st;
  if (!workspace || workspace_bytes < need)
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  size_t conv = 0, h = 0;
  for (int k = 0; k < num_layers; ++k) {
    const size_t c = convolve_ws(&layers[k], graph->num_pins, n);
    conv = c > conv ? c : conv;
    if (k + 1 < num_layers) {
      const size_t hb = align_up((size_t)n * layers[k].d_out * elem_size(layers[k].dtype));
      h = hb > h ? hb : h;
    }
  }
  const size_t tb = walk_table_bytes(graph);
  if (tb > conv) conv = tb;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  unsigned char* hbuf[2] = {ws + conv, ws + conv + h};
  const int64_t P = graph->num_pins;
  const pinsage_layer_t* L0 = &layers[0];

  // Walks, then the first layer's transform: beside each other on the
  // schedule's masked streams when one is given and the pin count is in the
  // overlapped range, else in order on the caller's stream. Beside the
  // transform the walks read the walk table from the first layer-output
  // buffer (free until the first layer's pool writes it) when it fits there,
  // else the CSR. With the table a first layer in the chained form overlaps
  // at any pin count: the walks are then bound by dependent reads, whose rate
  // holds on 7/8 of the CUs, and the chained transform needs no row chunks.
  bool transformed = false;
  const void* const gtab = graph->walk_table;  // the caller's table, when given
  unsigned char* const ov_table = (!gtab && tb && num_layers > 1 && h >= tb) ? hbuf[0] : nullptr;
  const bool ov_range = P >= kMinOverlapRows &&
                        (P <= kMaxOverlapRows || ((gtab || ov_table) && chained_layer(L0)));
  if (schedule && ov_range) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "current device");
    if (dev != schedule->device)
      return fail(PINSAGE_EINVAL, "schedule belongs to device %d, current device is %d",
                  schedule->device, dev);
    std::lock_guard<std::mutex> lk(schedule->mu);
    pinsage_schedule& ov = *schedule;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess) {
      (void)hipGetLastError();
      cap = hipStreamCaptureStatusNone;
    }
    const bool capturing = cap != hipStreamCaptureStatusNone;
    const int64_t a = overlap_rows(ov, P, capturing);
    if (a > 0) {
      e = hipEventRecord(ov.fork, s);
      if (e == hipSuccess) e = hipStreamWaitEvent(ov.side, ov.fork, 0);
      if (e == hipSuccess) e = hipStreamWaitEvent(ov.walk, ov.fork, 0);
      if (e != hipSuccess) return hip_fail(e, "stream fork");
      // Every record and wait below runs whatever the launches returned, so
      // the side and walk streams are joined back into the caller's stream
      // on error paths too (no work of this call is left unjoined).
      st = run_transform_rows(L0, x, n, P, nullptr, n, ws, 0, a, 0, ov.side);
      const hipError_t e1 = hipEventRecord(ov.side_done, ov.side);
      if (!st && ov_table) {
        const hipError_t et = launch_walk_table(graph->row_offsets,
                                                graph->offset_type == PINSAGE_I64, graph->col,
                                                graph->nnz, n, ov_table, ov.walk);
        if (et != hipSuccess) st = hip_fail(et, "walk table launch");
      }
      if (!st)
        st = run_walks(graph, walk, nullptr, n, nbr_out, total_steps, gtab ? gtab : ov_table,
                       ov.walk);
      const hipError_t e2 = hipEventRecord(ov.walk_done, ov.walk);
      // Join: the caller's stream waits for the walks before its share of
      // the transform, and for the side before the pool.
      const hipError_t e3 = hipStreamWaitEvent(s, ov.walk_done, 0);
      if (!st) st = run_transform_rows(L0, x, n, P, nullptr, n, ws, a, P, a, s);
      const hipError_t e4 = hipEventRecord(ov.main_done, s);
      const hipError_t e5 = hipStreamWaitEvent(s, ov.side_done, 0);
      if (st) return st;
      for (hipError_t ej : {e1, e2, e3, e4, e5})
        if (ej != hipSuccess) return hip_fail(ej, "stream join");
      ov.side_rows = a;
      ov.main_rows = P - a;
      ov.total_rows = P;
      ov.pending = !capturing;
      transformed = true;
    }
  }
  if (!transformed) {
    // In order: the walks read the graph's walk table, built in the layers'
    // region of the workspace (one read per edge step instead of two).
    if (tb && !gtab) {
      const hipError_t e = launch_walk_table(graph->row_offsets, graph->offset_type == PINSAGE_I64,
                                             graph->col, graph->nnz, n, ws, s);
      if (e != hipSuccess) return hip_fail(e, "walk table launch");
    }
    const void* tab = gtab ? gtab : (tb ? ws : nullptr);
    if ((st = run_walks(graph, walk, nullptr, n, nbr_out, total_steps, tab, s))) return st;
    if ((st = run_transform(L0, x, n, P, nullptr, n, ws, s))) return st;
  }

  const void* cur = x;
  for (int k = 0; k < num_layers; ++k) {
    void* dst = (k == num_layers - 1) ? h_out : hbuf[k % 2];
    if (k > 0) st = run_transform(&layers[k], cur, n, P, nullptr, n, ws, s);
    if (!st) st = run_pool_dense(&layers[k], cur, n, P, nbr_out, nullptr, dst, n, ws, s);
    if (st) return st;
    cur = dst;
  }
  return PINSAGE_OK;
}

int pinsage_schedule_create(int32_t cu_eighths, pinsage_schedule_t** out) {
  g_last_error.clear();
  if (!out) return fail(PINSAGE_EINVAL, "out is NULL");
  *out = nullptr;
  if (cu_eighths < 1 || cu_eighths > 7)
    return fail(PINSAGE_EINVAL, "cu_eighths %d outside [1, 7]", cu_eighths);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "device query");
  if (cus < 64) return fail(PINSAGE_EUNSUPPORTED, "device has %d CUs (< 64)", cus);
  auto* o = new pinsage_schedule();
  o->device = dev;
  o->eighths = cu_eighths;
  o->alpha = cu_eighths >= 4 ? 1.0 : 0.3 * cu_eighths;  // first call: a share by CU count
  o->rf_over_rs = 8.0 / cu_eighths;
  const int words = (cus + 31) / 32;
  std::vector<uint32_t> side_mask(words, 0u), walk_mask(words, 0u);
  for (int i = 0; i < cus; ++i) {
    const int j = i / 8;
    const bool to_side = ((j + 1) * cu_eighths) / 8 > (j * cu_eighths) / 8;
    (to_side ? side_mask : walk_mask)[i / 32] |= 1u << (i % 32);
  }
  e = hipExtStreamCreateWithCUMask(&o->side, (uint32_t)words, side_mask.data());
  if (e == hipSuccess) e = hipExtStreamCreateWithCUMask(&o->walk, (uint32_t)words, walk_mask.data());
  if (e == hipSuccess) e = hipEventCreate(&o->fork);
  if (e == hipSuccess) e = hipEventCreate(&o->side_done);
  if (e == hipSuccess) e = hipEventCreate(&o->walk_done);
  if (e == hipSuccess) e = hipEventCreate(&o->main_done);
  if (e != hipSuccess) {
    const int st = hip_fail(e, "masked stream / event creation");
    schedule_release(o);
    return st;
  }
  *out = o;
  return PINSAGE_OK;
}

int pinsage_schedule_destroy(pinsage_schedule_t* schedule) {
  g_last_error.clear();
  if (!schedule) return PINSAGE_OK;
  {
    // A call still enqueueing on this schedule finishes first.
    std::lock_guard<std::mutex> lk(schedule->mu);
  }
  schedule_release(schedule);
  return PINSAGE_OK;
}

int pinsage_profile_enable(int on) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& p : g_pending) {
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  for (int k = 0; k < kKCount; ++k) {
    g_prof_count[k] = 0;
    g_prof_ms[k] = 0.0;
  }
  g_prof_on = on != 0;
  return PINSAGE_OK;
}

int pinsage_profile_read(int kernel, int64_t* launches, double* total_ms) {
  g_last_error.clear();
  if (kernel < 0 || kernel >= kKCount) return fail(PINSAGE_EINVAL, "unknown kernel class %d", kernel);
  if (!launches || !total_ms) return fail(PINSAGE_EINVAL, "NULL output");
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& p : g_pending) {
    hipError_t e = hipEventSynchronize(p.stop);
    if (e != hipSuccess) return hip_fail(e, "profile event sync");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, p.start, p.stop);
    if (e != hipSuccess) return hip_fail(e, "profile elapsed time");
    g_prof_count[p.cls] += 1;
    g_prof_ms[p.cls] += ms;
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
  }
  g_pending.clear();
  *launches = g_prof_count[kernel];
  *total_ms = g_prof_ms[kernel];
  return PINSAGE_OK;
}

int pinsage_profile_random_reads(const void* table, size_t table_bytes, int32_t elem_bytes,
                                 int32_t steps, uint32_t* sink, int64_t chains, void* stream) {
  g_last_error.clear();
  if (!table || !sink) return fail(PINSAGE_EINVAL, "NULL table or sink");
  if (elem_bytes != 4 && elem_bytes != 8 && elem_bytes != 16)
    return fail(PINSAGE_EINVAL, "element size %d (4, 8 or 16)", elem_bytes);
  if (table_bytes < (size_t)elem_bytes) return fail(PINSAGE_EINVAL, "table smaller than one element");
  if (steps < 1 || chains < 1) return fail(PINSAGE_EINVAL, "steps %d, chains %lld", steps, (long long)chains);
  uint64_t elements = 1;
  while (elements * 2 <= table_bytes / (size_t)elem_bytes) elements *= 2;
  hipError_t e = launch_random_reads(table, elements, elem_bytes, steps, sink, chains,
                                     static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "random read launch");
  return PINSAGE_OK;
}

int pinsage_profile_random_gathers(const void* table, size_t table_bytes, int32_t row_bytes,
                                   int64_t targets, int32_t per_target, uint64_t seed,
                                   uint32_t* sink, void* stream) {
  g_last_error.clear();
  if (!table || !sink) return fail(PINSAGE_EINVAL, "NULL table or sink");
  if (row_bytes != 512 && row_bytes != 1024)
    return fail(PINSAGE_EINVAL, "row size %d (512 or 1024)", row_bytes);
  if (reinterpret_cast<uintptr_t>(table) % 16 != 0)
    return fail(PINSAGE_EINVAL, "table not 16-byte aligned");
  const uint64_t rows = table_bytes / (size_t)row_bytes;
  if (rows < 1) return fail(PINSAGE_EINVAL, "table smaller than one row");
  if (rows >= (1ull << 32)) return fail(PINSAGE_EUNSUPPORTED, "%llu rows (< 2^32)",
                                        (unsigned long long)rows);
  const int max_per = row_bytes == 512 ? 64 : 32;
  if (targets < 1 || per_target < 1 || per_target > max_per)
    return fail(PINSAGE_EINVAL, "targets %lld, rows per target %d (1..%d)", (long long)targets,
                per_target, max_per);
  hipError_t e = launch_random_gathers(table, rows, row_bytes, targets, per_target, seed, sink,
                                       static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "random gather launch");
  return PINSAGE_OK;
}

int pinsage_output_mlp_workspace_size(const pinsage_mlp_t* mlp, int64_t n, size_t* bytes) {
  g_last_error.clear();
  int st = check_mlp(mlp);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  if (n < 0) return fail(PINSAGE_EINVAL, "negative row count");
  *bytes = mlp_ws(mlp, n);
  return PINSAGE_OK;
}

int pinsage_output_mlp(const pinsage_mlp_t* mlp, const void* h, int64_t n, void* z,
                       void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  int st = check_mlp(mlp);
  if (st) return st;
  if (n < 0) return fail(PINSAGE_EINVAL, "negative row count");
  if (n == 0) return PINSAGE_OK;
  if (!h || !z) return fail(PINSAGE_EINVAL, "h or z is NULL");
  const size_t need = mlp_ws(mlp, n);
  if (!workspace || workspace_bytes < need)
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");
  return run_mlp(mlp, h, nullptr, n, n, z, workspace, static_cast<hipStream_t>(stream));
}

int pinsage_max_margin_loss(const void* zq, const void* zpos, int64_t B, const void* zneg,
                            int64_t n_neg, const void* zhard, int64_t num_hard, int32_t d,
                            pinsage_dtype_t dtype, float margin, float* loss, float* per_pair,
                            void* stream) {
  g_last_error.clear();
  if (!zq || !zpos || !zneg || !loss || !per_pair)
    return fail(PINSAGE_EINVAL, "a pointer argument is NULL (per_pair is required)");
  if (B < 1 || n_neg < 1) return fail(PINSAGE_EINVAL, "need B >= 1 and n_neg >= 1");
  if (num_hard < 0) return fail(PINSAGE_EINVAL, "negative num_hard");
  if (num_hard > 0 && !zhard) return fail(PINSAGE_EINVAL, "zhard is NULL");
  if (d < 1 || d > 1024) return fail(PINSAGE_EUNSUPPORTED, "d %d outside [1, 1024]", d);
  if (dtype != PINSAGE_F32 && dtype != PINSAGE_BF16)
    return fail(PINSAGE_EINVAL, "unknown dtype %d", (int)dtype);
  LossLaunch a{};
  a.zq = zq;
  a.zpos = zpos;
  a.zneg = zneg;
  a.zhard = zhard;
  a.k_hard = num_hard;
  a.B = B;
  a.n_neg = n_neg;
  a.d = d;
  a.bf16 = dtype == PINSAGE_BF16;
  a.margin = margin;
  a.per_pair = per_pair;
  a.loss = loss;
  hipError_t e = launch_loss(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "loss launch");
  return PINSAGE_OK;
}

}  // extern "C"

namespace pinsage {
namespace {

constexpr int kMaxMinibatchLayers = 8;

// Workspace layout of the minibatch forward; every region 256-aligned.
struct MbPlan {
  int K = 0, T = 0;
  int64_t N = 0;
  int64_t U[kMaxMinibatchLayers + 1] = {};  // frontier capacity per level
  size_t flags = 0, pos = 0, tiles = 0, ctr = 0, rows = 0, pp = 0, conv = 0, z = 0, mlp = 0;
  size_t set[kMaxMinibatchLayers + 1] = {};
  size_t nidx[kMaxMinibatchLayers + 1] = {}, ncnt[kMaxMinibatchLayers + 1] = {},
         nw[kMaxMinibatchLayers + 1] = {}, self[kMaxMinibatchLayers + 1] = {},
         h[kMaxMinibatchLayers + 1] = {};
  size_t total = 0;
};

int make_plan(const pinsage_graph_t* g, const pinsage_walk_params_t* w,
              const pinsage_layer_t* layers, int K, const pinsage_mlp_t* mlp, int64_t B,
              int64_t n_neg, int64_t n_hard, MbPlan* p) {
  const int64_t N = g->num_pins + g->num_boards;
  p->K = K;
  p->T = w->top_t;
  p->N = N;
  const int64_t nt = 2 * B + n_neg + B * n_hard;  // target ids (rows of the loss tables)
  p->U[K] = nt < N ? nt : N;
  for (int k = K; k >= 1; --k) {
    const int64_t grow = p->U[k] * (int64_t)(w->top_t + 1);
    p->U[k - 1] = grow < N ? grow : N;
  }
  size_t cur = 0;
  auto take = [&](size_t bytes) {
    const size_t at = cur;
    cur += align_up(bytes);
    return at;
  };
  p->flags = take((size_t)N);
  p->pos = take((size_t)N * 4);
  p->tiles = take((size_t)scan_tiles(N) * 4);
  p->ctr = take(64);
  for (int k = 0; k <= K; ++k) p->set[k] = take((size_t)p->U[k] * 4);
  for (int k = 1; k <= K; ++k) {
    const size_t e = (size_t)p->U[k] * w->top_t;
    p->nidx[k] = take(e * 4);
    p->ncnt[k] = take(e * 2);
    p->nw[k] = take(e * 4);
    p->self[k] = take((size_t)p->U[k] * 4);
    p->h[k] = take((size_t)p->U[k] * layers[k - 1].d_out * elem_size(layers[k - 1].dtype));
  }
  p->rows = take((size_t)nt * 4);
  p->pp = take((size_t)B * 4);
  size_t conv = 0;
  for (int k = 1; k <= K; ++k) {
    const size_t c = convolve_ws(&layers[k - 1], p->U[k - 1], p->U[k]);
    conv = c > conv ? c : conv;
  }
  p->conv = take(conv);
  if (mlp) {  // z of the targets' set, and the hidden activations of the output layers
    p->z = take((size_t)p->U[K] * mlp->d_out * elem_size(mlp->dtype));
    p->mlp = take(mlp_ws(mlp, p->U[K]));
  }
  p->total = cur;
  return PINSAGE_OK;
}

int check_minibatch(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                    const pinsage_layer_t* layers, int32_t K, const pinsage_mlp_t* mlp,
                    int64_t B, int64_t n_neg, int64_t n_hard) {
  int st = check_graph(graph);
  if (st) return st;
  if ((st = check_walk(walk))) return st;
  if (K < 1 || K > kMaxMinibatchLayers || !layers)
    return fail(PINSAGE_EUNSUPPORTED, "num_layers %d outside [1, %d]", K, kMaxMinibatchLayers);
  for (int k = 0; k < K; ++k) {
    if ((st = check_layer(&layers[k], k))) return st;
    if (layers[k].dtype != layers[0].dtype)
      return fail(PINSAGE_EINVAL, "layer %d dtype differs from layer 0", k);
    if (k > 0 && layers[k].d_in != layers[k - 1].d_out)
      return fail(PINSAGE_EINVAL, "layer %d d_in %d != layer %d d_out %d", k, layers[k].d_in,
                  k - 1, layers[k - 1].d_out);
  }
  if (mlp) {
    if ((st = check_mlp(mlp))) return st;
    if (mlp->d_in != layers[K - 1].d_out)
      return fail(PINSAGE_EINVAL, "mlp d_in %d != last layer d_out %d", mlp->d_in,
                  layers[K - 1].d_out);
    if (mlp->dtype != layers[0].dtype) return fail(PINSAGE_EINVAL, "mlp dtype differs from layers");
  }
  const int d = mlp ? mlp->d_out : layers[K - 1].d_out;
  if (d > 1024) return fail(PINSAGE_EUNSUPPORTED, "output dim %d > 1024", d);
  if (B < 1 || n_neg < 1) return fail(PINSAGE_EINVAL, "need num_pairs >= 1 and num_negatives >= 1");
  if (n_hard < 0) return fail(PINSAGE_EINVAL, "negative num_hard");
  if (n_hard > 0 && B > ((1ll << 40) / n_hard))
    return fail(PINSAGE_EUNSUPPORTED, "num_pairs * num_hard too large");
  return PINSAGE_OK;
}

int read_counters(const long long* dev, long long* host, int n, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(host, dev, sizeof(long long) * n, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return hip_fail(e, "frontier size copy");
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "frontier size sync");
  return PINSAGE_OK;
}

}  // namespace
}  // namespace pinsage

extern "C" {

int pinsage_minibatch_workspace_size(const pinsage_graph_t* graph,
                                     const pinsage_walk_params_t* walk,
                                     const pinsage_layer_t* layers, int32_t num_layers,
                                     const pinsage_mlp_t* mlp, int64_t num_pairs,
                                     int64_t num_negatives, int64_t num_hard, size_t* bytes) {
  g_last_error.clear();
  int st = check_minibatch(graph, walk, layers, num_layers, mlp, num_pairs, num_negatives,
                           num_hard);
  if (st) return st;
  if (!bytes) return fail(PINSAGE_EINVAL, "bytes is NULL");
  MbPlan p;
  make_plan(graph, walk, layers, num_layers, mlp, num_pairs, num_negatives, num_hard, &p);
  *bytes = p.total;
  return PINSAGE_OK;
}

int pinsage_minibatch_forward(const pinsage_graph_t* graph, const pinsage_walk_params_t* walk,
                              const pinsage_layer_t* layers, int32_t num_layers,
                              const pinsage_mlp_t* mlp, const void* x,
                              const pinsage_pairs_t* pairs, float* loss, float* per_pair,
                              void* z_out, int64_t* set_sizes, unsigned long long* total_steps,
                              void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  if (!pairs) return fail(PINSAGE_EINVAL, "pairs is NULL");
  const int64_t B = pairs->num_pairs, n_neg = pairs->num_negatives, n_hard = pairs->num_hard;
  const int K = num_layers;
  int st = check_minibatch(graph, walk, layers, K, mlp, B, n_neg, n_hard);
  if (st) return st;
  if (!pairs->queries || !pairs->positives || !pairs->negatives)
    return fail(PINSAGE_EINVAL, "pair id arrays must not be NULL");
  if (n_hard > 0 && !pairs->hard_negatives)
    return fail(PINSAGE_EINVAL, "hard_negatives is NULL with num_hard > 0");
  if (!x || !loss) return fail(PINSAGE_EINVAL, "x or loss is NULL");
  MbPlan p;
  make_plan(graph, walk, layers, K, mlp, B, n_neg, n_hard, &p);
  if (!workspace || workspace_bytes < p.total)
    return fail(PINSAGE_EWORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes,
                p.total);
  if (reinterpret_cast<uintptr_t>(workspace) % 256)
    return fail(PINSAGE_EINVAL, "workspace is not 256-byte aligned");

  hipStream_t s = static_cast<hipStream_t>(stream);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  const int64_t N = p.N, T = p.T;
  uint8_t* flags = reinterpret_cast<uint8_t*>(ws + p.flags);
  int32_t* pos = reinterpret_cast<int32_t*>(ws + p.pos);
  int32_t* tiles = reinterpret_cast<int32_t*>(ws + p.tiles);
  long long* ctr = reinterpret_cast<long long*>(ws + p.ctr);
  auto set_of = [&](int k) { return reinterpret_cast<int32_t*>(ws + p.set[k]); };
  auto nidx_of = [&](int k) { return reinterpret_cast<int32_t*>(ws + p.nidx[k]); };
  auto self_of = [&](int k) { return reinterpret_cast<int32_t*>(ws + p.self[k]); };
  int32_t* rows = reinterpret_cast<int32_t*>(ws + p.rows);
  int64_t size[kMaxMinibatchLayers + 1] = {}, npins[kMaxMinibatchLayers + 1] = {};
  long long host[2];
  hipError_t e;
#define PINSAGE_TRY(expr, what)                 \
  do {                                          \
    e = (expr);                                 \
    if (e != hipSuccess) return hip_fail(e, what); \
  } while (0)

  // Walks for one level: neighbourhoods of set k (global ids, weights kept).
  auto walk_level = [&](int k) -> int {
    WalkLaunch a{};
    a.row_offsets = graph->row_offsets;
    a.offsets64 = graph->offset_type == PINSAGE_I64;
    a.col = graph->col;
    a.nnz = graph->nnz;
    a.num_pins = graph->num_pins;
    a.num_nodes = N;
    a.sources = set_of(k);
    a.num_sources = size[k];
    a.seed = walk->seed;
    a.walks = walk->walks_per_node;
    a.hops = walk->hops;
    a.top_t = walk->top_t;
    a.idx = nidx_of(k);
    a.counts = reinterpret_cast<uint16_t*>(ws + p.ncnt[k]);
    a.weights = reinterpret_cast<float*>(ws + p.nw[k]);
    a.total_steps = total_steps;  // accumulated over the levels
    a.table = graph->walk_table;
    PINSAGE_TRY(launch_walk_topt(a, s), "walk launch");
    return PINSAGE_OK;
  };
  // Sorted unique set of level k from the flags, its size and pin count.
  auto scan_level = [&](int k) -> int {
    PINSAGE_TRY(launch_flag_scan(flags, N, tiles, pos, set_of(k), p.U[k], ctr, s), "frontier scan");
    PINSAGE_TRY(launch_count_below(set_of(k), ctr, p.U[k], graph->num_pins, ctr + 1, s),
                "pin count");
    int r = read_counters(ctr, host, 2, s);
    if (r) return r;
    size[k] = host[0];
    npins[k] = host[1];
    if (size[k] > p.U[k])
      return fail(PINSAGE_EHIP, "frontier %d holds %lld ids, capacity %lld", k, host[0],
                  (long long)p.U[k]);
    return PINSAGE_OK;
  };

  if (total_steps) PINSAGE_TRY(launch_zero_u64(total_steps, 1, s), "step counter reset");
  // Level K: the targets of the minibatch (Algorithm 2, S^(K) = M).
  PINSAGE_TRY(launch_fill_zero_u8(flags, N, s), "flag reset");
  PINSAGE_TRY(launch_mark(pairs->queries, B, N, flags, s), "mark");
  PINSAGE_TRY(launch_mark(pairs->positives, B, N, flags, s), "mark");
  PINSAGE_TRY(launch_mark(pairs->negatives, n_neg, N, flags, s), "mark");
  PINSAGE_TRY(launch_mark(pairs->hard_negatives, B * n_hard, N, flags, s), "mark");
  if ((st = scan_level(K))) return st;
  PINSAGE_TRY(launch_remap(pairs->queries, B, N, pos, rows, s), "remap");
  PINSAGE_TRY(launch_remap(pairs->positives, B, N, pos, rows + B, s), "remap");
  PINSAGE_TRY(launch_remap(pairs->negatives, n_neg, N, pos, rows + 2 * B, s), "remap");
  PINSAGE_TRY(launch_remap(pairs->hard_negatives, B * n_hard, N, pos, rows + 2 * B + n_neg, s),
              "remap");
  if ((st = walk_level(K))) return st;
  // Levels K-1 .. 0: S^(k) = S^(k+1) u N(S^(k+1)); re-index level k+1.
  for (int k = K - 1; k >= 0; --k) {
    PINSAGE_TRY(launch_fill_zero_u8(flags, N, s), "flag reset");
    PINSAGE_TRY(launch_mark(set_of(k + 1), size[k + 1], N, flags, s), "mark");
    PINSAGE_TRY(launch_mark(nidx_of(k + 1), size[k + 1] * T, N, flags, s), "mark");
    if ((st = scan_level(k))) return st;
    PINSAGE_TRY(launch_remap(nidx_of(k + 1), size[k + 1] * T, N, pos, nidx_of(k + 1), s), "remap");
    PINSAGE_TRY(launch_remap(set_of(k + 1), size[k + 1], N, pos, self_of(k + 1), s), "remap");
    if (k >= 1 && (st = walk_level(k))) return st;
  }

  // Layers k = 1..K on the compact sets (Algorithm 2, embedding loop).
  unsigned char* conv_ws = ws + p.conv;
  for (int k = 1; k <= K; ++k) {
    const pinsage_layer_t* L = &layers[k - 1];
    pinsage_neighborhoods_t nb{size[k], walk->top_t, nidx_of(k),
                               reinterpret_cast<uint16_t*>(ws + p.ncnt[k]),
                               reinterpret_cast<float*>(ws + p.nw[k])};
    if (k == 1) {
      // h^(0) = x read in place: P rows are x[S^(0) pins], self rows x[S^(1)].
      st = run_layer(L, x, N, npins[0], set_of(0), &nb, set_of(1), ws + p.h[1], size[1], conv_ws,
                     s);
    } else {
      st = run_layer(L, ws + p.h[k - 1], size[k - 1], npins[k - 1], nullptr, &nb, self_of(k),
                     ws + p.h[k], size[k], conv_ws, s);
    }
    if (st) return st;
  }

  // Output dense layers (Algorithm 2, final loop) on every row of S^(K).
  const pinsage_layer_t* LK = &layers[K - 1];
  const unsigned char* zsrc = ws + p.h[K];
  int d = LK->d_out;
  if (mlp) {
    if ((st = run_mlp(mlp, ws + p.h[K], nullptr, size[K], size[K], ws + p.z, ws + p.mlp, s)))
      return st;
    zsrc = ws + p.z;
    d = mlp->d_out;
  }
  // Eq. (1) on z, rows looked up through the level-K positions.
  LossLaunch la{};
  la.zq = zsrc;
  la.q_rows = rows;
  la.zpos = zsrc;
  la.pos_rows = rows + B;
  la.zneg = zsrc;
  la.neg_rows = rows + 2 * B;
  la.zhard = zsrc;
  la.hard_rows = rows + 2 * B + n_neg;
  la.k_hard = n_hard;
  la.B = B;
  la.n_neg = n_neg;
  la.d = d;
  la.bf16 = LK->dtype == PINSAGE_BF16;
  la.margin = pairs->margin;
  la.per_pair = per_pair ? per_pair : reinterpret_cast<float*>(ws + p.pp);
  la.loss = loss;
  PINSAGE_TRY(launch_loss(la, s), "loss launch");
  if (z_out)
    PINSAGE_TRY(launch_gather_rows(zsrc, rows, 2 * B + n_neg + B * n_hard,
                                   (int64_t)d * elem_size(LK->dtype), z_out, s),
                "target gather");
  if (set_sizes)
    for (int k = 0; k <= K; ++k) set_sizes[k] = size[k];
#undef PINSAGE_TRY
  return PINSAGE_OK;
}

}  // extern "C"
