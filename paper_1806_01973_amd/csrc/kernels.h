// Host-side launchers of the gfx950 kernels (internal to libpinsage.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pinsage {

// Kernel classes for per-launch timing; values match PINSAGE_KERNEL_*.
enum KernelClass { kKWalk = 0, kKGemmQ = 1, kKPool = 2, kKGemmW = 3, kKMinibatch = 4, kKLoss = 5,
                   kKGemmR = 6, kKMlp = 7, kKHardNeg = 8, kKGraphNbr = 9, kKGemmQR = 10,
                   kKWalkTable = 11, kKPoolW = 12, kKCount = 13 };

// Records a start/stop hipEvent pair around a launch when timing is enabled.
class ProfileScope {
 public:
  ProfileScope(int cls, hipStream_t s);
  ~ProfileScope();
 private:
  int cls_;
  hipStream_t s_;
  hipEvent_t start_ = nullptr;
};

struct WalkLaunch {
  const void* row_offsets;
  bool offsets64;
  const int32_t* col;
  int64_t nnz;
  int64_t num_pins;
  int64_t num_nodes;
  const int32_t* sources;  // nullable: row r is node r
  int64_t num_sources;
  uint64_t seed;
  int walks;
  int hops;
  int top_t;
  int32_t* idx;
  uint16_t* counts;
  float* weights;           // nullable
  unsigned long long* total_steps;  // nullable; accumulated (caller zeroes)
  const void* table;        // nullable: the walk table of the graph (below)
};
hipError_t launch_walk_topt(const WalkLaunch& a, hipStream_t s);

// Walk table: for every CSR position e, 16 bytes {col[e], degree of col[e],
// row start of col[e] (low, high 32 bits)}, degree 0 for an out-of-range id or
// an empty or malformed row. A walk then takes one read per edge step instead
// of an offset pair and a neighbour id. For graphs with nnz < 2^31 (degrees
// fit 31 bits).
constexpr int64_t kWalkTableMaxNnz = 0x7FFFFFFFll;
hipError_t launch_walk_table(const void* row_offsets, bool offsets64, const int32_t* col,
                             int64_t nnz, int64_t num_nodes, void* table, hipStream_t s);

// Hard negative items (Sec. 3.3): out[i][j], j < k, drawn from ranks
// [rank_lo, rank_hi) of the visit-count ranking of walks from queries[i].
struct HardNegLaunch {
  const void* row_offsets;
  bool offsets64;
  const int32_t* col;
  int64_t nnz;
  int64_t num_pins;
  int64_t num_nodes;
  const int32_t* queries;
  int64_t num_queries;
  uint64_t seed;
  int walks;
  int hops;
  int rank_lo;
  int rank_hi;
  int k;
  int32_t* out;
  unsigned long long* total_steps;  // nullable; accumulated (caller zeroes)
  const void* table;                // nullable: the graph's walk table
};
// Walk budgets above kMaxOnChipLandings bucket a query's landings by hash
// partition in the workspace as the walks record them and count each bucket
// in LDS (hard_negative_workspace bytes per resident workgroup: the buckets,
// an overflow list twice and a (pin, count) list), and need
// rank_hi <= kMaxGlobalRank.
constexpr int64_t kMaxOnChipLandings = 16384;
constexpr int64_t kMaxLandings = 1ll << 22;
constexpr int kMaxGlobalRank = 8192;
constexpr int64_t kGMaxBlocks = 256;
size_t hard_negative_workspace(int64_t landings, int64_t num_queries);
hipError_t launch_hard_negatives(const HardNegLaunch& a, void* workspace, hipStream_t s);

// Graph neighbourhoods (Sec. 3.4, MapReduce inference): each source's CSR row,
// or top_t Philox draws from it when longer, as distinct ids ascending with
// multiplicities and weights multiplicity / kept entries; top_t <= 256.
struct GraphNbrLaunch {
  const void* row_offsets;
  bool offsets64;
  const int32_t* col;
  int64_t nnz;
  int64_t num_nodes;
  const int32_t* sources;  // nullable: row r is node r
  int64_t num_sources;
  uint64_t seed;
  int top_t;
  int32_t* idx;
  uint16_t* counts;
  float* weights;  // nullable
};
hipError_t launch_graph_neighborhoods(const GraphNbrLaunch& a, hipStream_t s);
// map[i] = i for i < valid, -1 for i in [valid, n).
hipError_t launch_row_map(int32_t* map, int64_t n, int64_t valid, hipStream_t s);


// Pooling modes (values match pinsage_pool_t).
enum PoolMode { kPoolImportance = 0, kPoolMean = 1, kPoolMax = 2 };

// n[r] = sum_t alpha[r][t] * P[idx[r][t]] (importance), the mean, or the
// element-wise max of the P rows of rows [0, rows) of the given neighbourhood
// slice; storage dtype bf16 when bf16 is true.
struct PoolLaunch {
  const void* P;
  int64_t n_transform;
  int m;
  bool bf16;
  const int32_t* idx;
  const uint16_t* counts;
  const float* weights;  // nullable: derived from counts
  int T;
  int64_t rows;
  void* out;
  int mode;  // PoolMode
};
hipError_t launch_pool(const PoolLaunch& a, hipStream_t s);

// Pool and W fused (poolw.hip): out[r] = L2norm(ReLU(W_s h[self(r)] + pool(R, N(r))
// + bias)) for bf16, d_in = d_out = 256, T <= 64. W_s arrives as fragments
// from launch_permute_ws (pool_w_ws_bytes() of workspace).
struct PoolWLaunch {
  const void* R;           // [n_transform][256] rows to pool
  int64_t n_transform;
  const int32_t* idx;
  const uint16_t* counts;
  const float* weights;    // nullable: derived from counts
  int T;
  int mode;                // PoolMode
  const void* H;           // self rows
  const int32_t* self_rows;  // nullable: row r reads H row h_row0 + r
  int64_t h_row0;
  int64_t rows_h;
  int64_t ldh;
  const void* Wsp;
  const float* bias;       // [256]
  void* out;               // [rows][256]
  int64_t rows;
};
bool pool_w_supported(int d_in, int d_out, bool bf16, int T);
size_t pool_w_ws_bytes();
hipError_t launch_permute_ws(const void* W, int64_t ldw, void* Wsp, hipStream_t s);
hipError_t launch_pool_w(const PoolWLaunch& a, hipStream_t s);

// C[r][c] = epilogue(sum_k A[r][k] * B[c][k] + bias[c] + addend[r][c]) where
// the A row is the concatenation of A0[rowmap ? rowmap[r] : r][0:K0] and
// A1[r][0:K1]. B is [N][K0 + K1] with row stride ldb. Epilogue: optional
// ReLU, optionally followed by row L2 normalisation over all N columns (which
// implies ReLU). Profiled as the Q class (ReLU, no norm), the W class (norm)
// or the R class (neither).
struct GemmLaunch {
  const void* A0;
  const int32_t* rowmap;  // nullable; entries outside [0, rows_a0) read as zero rows
  int64_t rows_a0;
  int64_t lda0;
  int K0;
  const void* A1;  // nullable when K1 == 0
  int64_t lda1;
  int K1;
  const void* B;
  int64_t ldb;        // elements between B rows; 0 means K0 + K1
  const float* bias;  // nullable: no bias
  const void* addend; // nullable; [M][N] in the storage dtype
  int64_t M;
  int N;
  void* C;
  bool bf16;
  bool relu;
  bool l2norm;
  int prof_class = -1;  // KernelClass for timing; -1: inferred from the epilogue
  // Rows of the whole product before row 0 of this launch (a multiple of 256).
  // Only the K-sweep rotation reads it, so a product split into row ranges
  // sums every row in the same order as one launch over all rows.
  int64_t row_base = 0;
};
hipError_t launch_gemm(const GemmLaunch& a, hipStream_t s);

// R[r] = ReLU(H[t(r)] Q^T + q) W_n^T for r in [0, rows), t(r) = rowmap[r] or
// row0 + r (entries outside [0, rows_h) read as zero rows), bf16, with W_n'
// the neighbour half of W in the column order of launch_permute_wn. P stays
// in registers. Supported shapes: chain_supported.
struct ChainLaunch {
  const void* H;
  const int32_t* rowmap;  // nullable
  int64_t row0;
  int64_t rows_h;
  int64_t ldh;
  const void* Q;   // [m][d_in]
  const float* q;  // [m]
  const void* Wp;  // [d_out][m], from launch_permute_wn
  int d_in, m, d_out;
  void* R;  // [rows][ldr]
  int64_t ldr;
  int64_t rows;
};
bool chain_supported(int d_in, int m, int d_out, bool bf16);
// Wp[n][.] = W[n][d_in + .] (row stride ldw) with every 16-column group in
// the order the chained kernel's second product reads it.
hipError_t launch_permute_wn(const void* W, int64_t ldw, int d_in, int m, int d_out, void* Wp,
                             hipStream_t s);
hipError_t launch_chain(const ChainLaunch& a, hipStream_t s);

// Dependent random reads (calib.hip): `chains` lanes, `steps` reads each, from
// `elements` (a power of two) elements of elem_bytes (4, 8 or 16) bytes.
hipError_t launch_random_reads(const void* table, uint64_t elements, int elem_bytes, int steps,
                               uint32_t* sink, int64_t chains, hipStream_t s);
// Random row gathers (bench support): targets x per rows of row_bytes (512 or
// 1024) from `rows` rows at hashed positions; every word is added into *sink.
hipError_t launch_random_gathers(const void* table, uint64_t rows, int row_bytes,
                                 int64_t targets, int per, uint64_t seed, uint32_t* sink,
                                 hipStream_t s);

// Max-margin loss (Eq. 1): per_pair[b] = mean over the shared negatives and
// pair b's present hard negatives of max(0, zq.zn - zq.zpos + margin),
// *loss = mean_b per_pair[b]. Row maps index the tables (NULL = identity;
// negative entries read as zero vectors, except hard rows, where they mark an
// absent entry). d <= 1024.
struct LossLaunch {
  const void* zq;
  const int32_t* q_rows;
  const void* zpos;
  const int32_t* pos_rows;
  const void* zneg;
  const int32_t* neg_rows;
  const void* zhard;         // [B * k_hard rows], row b * k_hard + j of pair b
  const int32_t* hard_rows;  // nullable: identity
  int64_t k_hard;
  int64_t B;
  int64_t n_neg;
  int d;
  bool bf16;
  float margin;
  float* per_pair;
  float* loss;
};
hipError_t launch_loss(const LossLaunch& a, hipStream_t s);

// Frontier machinery of the minibatch forward (node flags + exclusive scan).
hipError_t launch_fill_zero_u8(uint8_t* p, int64_t n, hipStream_t s);
hipError_t launch_mark(const int32_t* ids, int64_t n, int64_t N, uint8_t* flags, hipStream_t s);
int64_t scan_tiles(int64_t N);
// set[0..total) = sorted flagged ids (entries past cap are dropped), pos[id] =
// index of id in set (flagged ids only).
hipError_t launch_flag_scan(const uint8_t* flags, int64_t N, int32_t* tile_sums, int32_t* pos,
                            int32_t* set, int64_t cap, long long* total, hipStream_t s);
// *count = entries of the sorted set (length *size_dev <= cap) below bound.
hipError_t launch_count_below(const int32_t* set, const long long* size_dev, int64_t cap,
                              int64_t bound, long long* count, hipStream_t s);
// out[i] = pos[in[i]] for in[i] in [0, N), else -1 (in-place allowed).
hipError_t launch_remap(const int32_t* in, int64_t n, int64_t N, const int32_t* pos, int32_t* out,
                        hipStream_t s);
hipError_t launch_gather_rows(const void* table, const int32_t* rows, int64_t n, int64_t row_bytes,
                              void* out, hipStream_t s);

// Fills n 64-bit words with zero (kept off hipMemsetAsync so callers may
// capture the stream in a graph).
hipError_t launch_zero_u64(unsigned long long* p, int64_t n, hipStream_t s);

}  // namespace pinsage
