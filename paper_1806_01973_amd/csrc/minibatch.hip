// Minibatch forward support on gfx950 (Algorithm 2 and Sec. 3.3):
//  * frontier sets S^(k): the ids of a level are marked in a node-flag array,
//    and an exclusive scan over the flags yields, in one pass, the sorted
//    unique set and the global -> local position map used to re-index
//    neighbour ids and self rows into the compact sets (the re-indexing of
//    Sec. 3.3, done on the device);
//  * the max-margin loss of Eq. 1 over a shared negative set.
// Everything is integer or fixed-order fp32, hence deterministic.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 16;
constexpr int kScanTile = kScanThreads * kScanPerThread;  // flags per tile

__global__ void fill_u8_kernel(uint8_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

__global__ void mark_kernel(const int32_t* ids, int64_t n, int64_t N, uint8_t* flags) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = ids[i];
    if (v >= 0 && (int64_t)v < N) flags[v] = 1;
  }
}

// Block-wide exclusive scan of one int per thread (blockDim.x a multiple of 64).
__device__ int block_exclusive_scan(int v, int* lds_waves, int* block_total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const int incl = wave_inclusive_sum(v, lane);
  if (lane == 63) lds_waves[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    const int t = lane < nwaves ? lds_waves[lane] : 0;
    const int ti = wave_inclusive_sum(t, lane);
    if (lane < nwaves) lds_waves[lane] = ti - t;  // exclusive wave offsets
    if (lane == 63) lds_waves[64] = ti;
  }
  __syncthreads();
  const int res = lds_waves[wave] + incl - v;
  *block_total = lds_waves[64];
  __syncthreads();
  return res;
}

__global__ __launch_bounds__(kScanThreads) void scan_tile_sums_kernel(const uint8_t* flags,
                                                                      int64_t N, int32_t* sums) {
  __shared__ int lds[65];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
  int s = 0;
#pragma unroll
  for (int e = 0; e < kScanPerThread; ++e)
    if (base + e < N) s += flags[base + e];
  int total = 0;
  block_exclusive_scan(s, lds, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(1024) void scan_tile_offsets_kernel(int32_t* sums, int64_t ntiles,
                                                                 long long* total) {
  __shared__ int lds[65];
  long long carry = 0;
  for (int64_t c = 0; c < ntiles; c += blockDim.x) {
    const int64_t i = c + threadIdx.x;
    const int v = i < ntiles ? sums[i] : 0;
    int chunk = 0;
    const int ex = block_exclusive_scan(v, lds, &chunk);
    if (i < ntiles) sums[i] = (int32_t)(carry + ex);
    carry += chunk;
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ __launch_bounds__(kScanThreads) void scan_tile_finish_kernel(
    const uint8_t* flags, int64_t N, const int32_t* offsets, int32_t* pos, int32_t* set,
    int64_t cap) {
  __shared__ int lds[65];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPerThread;
  uint8_t f[kScanPerThread];
  int s = 0;
#pragma unroll
  for (int e = 0; e < kScanPerThread; ++e) {
    f[e] = (base + e < N) ? flags[base + e] : 0;
    s += f[e];
  }
  int total = 0;
  int p = offsets[blockIdx.x] + block_exclusive_scan(s, lds, &total);
#pragma unroll
  for (int e = 0; e < kScanPerThread; ++e) {
    if (f[e]) {
      pos[base + e] = p;
      if (p < cap) set[p] = (int32_t)(base + e);
      ++p;
    }
  }
}

// *count = number of entries of the sorted set below `bound` (the pins); the
// set's length is read from device memory (at most cap).
__global__ void count_below_kernel(const int32_t* set, const long long* size_dev, int64_t cap,
                                   int64_t bound, long long* count) {
  const int64_t size = *size_dev < cap ? *size_dev : cap;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < size;
       i += (int64_t)gridDim.x * blockDim.x) {
    const bool below = set[i] < bound;
    const bool next_above = (i + 1 == size) || set[i + 1] >= bound;
    if (below && next_above) *count = i + 1;
  }
}

__global__ void remap_kernel(const int32_t* in, int64_t n, int64_t N, const int32_t* pos,
                             int32_t* out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = in[i];
    out[i] = (v >= 0 && (int64_t)v < N) ? pos[v] : -1;
  }
}

template <bool BF16>
__device__ __forceinline__ float load_elem(const void* base, int64_t i) {
  if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(base)[i]);
  else return static_cast<const float*>(base)[i];
}

// Copies one d-wide row of a table (row id `row`, -1 = zero row) into LDS
// as fp32; TPR threads share the row, thread c of them taking 16-byte vectors
// c, c + TPR, ... (eight loads in flight before their stores). Rows whose
// width is not a whole number of vectors go element by element.
template <bool BF16, int TPR>
__device__ __forceinline__ void stage_row(float* dst, const void* table, int64_t row, int d,
                                          int c) {
  constexpr int VE = BF16 ? 8 : 4;  // elements per 16-byte vector
  constexpr int U = 8;
  if (row < 0) {
    for (int k = c; k < d; k += TPR) dst[k] = 0.0f;
    return;
  }
  if (d % VE) {
    for (int k = c; k < d; k += TPR) dst[k] = load_elem<BF16>(table, row * d + k);
    return;
  }
  const uint4* src = reinterpret_cast<const uint4*>(
      static_cast<const unsigned char*>(table) + (size_t)row * d * (BF16 ? 2 : 4));
  const int nv = d / VE;
  for (int v0 = c; v0 < nv; v0 += TPR * U) {
    uint4 buf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + TPR * u;
      buf[u] = v < nv ? src[v] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int v = v0 + TPR * u;
      if (v >= nv) break;
      const uint32_t w[4] = {buf[u].x, buf[u].y, buf[u].z, buf[u].w};
      float* o = dst + v * VE;
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          o[2 * i] = __uint_as_float(w[i] << 16);
          o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = __uint_as_float(w[i]);
      }
    }
  }
}

// Eq. (1) per pair. A block of THREADS threads scores QB queries against the
// negatives, NC at a time: the query rows and the chunk's negative rows sit
// in LDS as fp32 with an odd row stride (rows read by one instruction fall in
// distinct banks). The TPQ = THREADS / QB threads of query q take negatives
// c, c + TPQ, ... of the chunk (NP each) and form each dot product over d in
// index order, so one broadcast read of z_q serves NP products. A thread adds
// its hinge terms in order, the TPQ threads of a query are summed by a fixed
// butterfly, and chunk sums are added in chunk order. The positive score is a
// partial dot per thread (indices c, c + TPQ, ...) summed by the same
// butterfly.
template <bool BF16, int THREADS, int QB, int NC, int DMAX>
__global__ __launch_bounds__(THREADS) void loss_pairs_kernel(LossLaunch a) {
  constexpr int TPQ = THREADS / QB;
  constexpr int NP = NC / TPQ;
  static_assert(TPQ <= 64 && NP * TPQ == NC && THREADS % NC == 0, "pair layout");
  constexpr int S_MAX = DMAX + 1;
  __shared__ float zq_s[QB * S_MAX];
  __shared__ float zn_s[NC * S_MAX];
  const int d = a.d;
  const int S = d | 1;  // odd row stride >= d
  const int t = threadIdx.x;
  const int q = t / TPQ, c = t % TPQ;
  const int64_t b0 = (int64_t)blockIdx.x * QB;
  const int64_t b = b0 + q;

  // Query rows of the block (zero rows for missing pairs or ids).
  {
    int64_t row = -1;
    if (b < a.B) row = a.q_rows ? (int64_t)a.q_rows[b] : b;
    stage_row<BF16, TPQ>(zq_s + q * S, a.zq, row, d, c);
  }
  __syncthreads();
  // Positive score of query q.
  float dp = 0.0f;
  {
    int64_t pr = -1;
    if (b < a.B) pr = a.pos_rows ? (int64_t)a.pos_rows[b] : b;
    if (pr >= 0)
      for (int k = c; k < d; k += TPQ)
        dp = fmaf(zq_s[q * S + k], load_elem<BF16>(a.zpos, pr * d + k), dp);
  }
#pragma unroll
  for (int o = TPQ / 2; o >= 1; o >>= 1) dp += __shfl_xor(dp, o);
  const float pos = dp;

  constexpr int TPR = THREADS / NC;  // threads per staged negative row
  float acc = 0.0f;
  for (int64_t c0 = 0; c0 < a.n_neg; c0 += NC) {
    __syncthreads();  // previous chunk fully read
    {
      const int r = t / TPR;
      const int64_t nn = c0 + r;
      int64_t row = -1;
      if (nn < a.n_neg) row = a.neg_rows ? (int64_t)a.neg_rows[nn] : nn;
      stage_row<BF16, TPR>(zn_s + r * S, a.zneg, row, d, t % TPR);
    }
    __syncthreads();
    const float* zq = zq_s + q * S;
    float dn[NP];
#pragma unroll
    for (int j = 0; j < NP; ++j) dn[j] = 0.0f;
    for (int k = 0; k < d; ++k) {
      const float x = zq[k];
#pragma unroll
      for (int j = 0; j < NP; ++j) dn[j] = fmaf(x, zn_s[(c + TPQ * j) * S + k], dn[j]);
    }
    float hc = 0.0f;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      const float h = dn[j] - pos + a.margin;
      hc += (c0 + c + TPQ * j < a.n_neg && h > 0.0f) ? h : 0.0f;
    }
#pragma unroll
    for (int o = TPQ / 2; o >= 1; o >>= 1) hc += __shfl_xor(hc, o);
    acc += hc;
  }
  // Pair b's own hard negatives (Sec. 3.3): thread c takes entries c, c + TPQ,
  // ... and forms each dot product over d in index order from the row in
  // memory; hinge sums and the count of present entries go through the same
  // butterfly.
  float hh = 0.0f;
  int hv = 0;
  for (int64_t j = c; j < a.k_hard; j += TPQ) {
    int64_t row = -1;
    if (b < a.B) row = a.hard_rows ? (int64_t)a.hard_rows[b * a.k_hard + j] : b * a.k_hard + j;
    if (row < 0) continue;
    const float* zq = zq_s + q * S;
    float dn = 0.0f;
    for (int k = 0; k < d; ++k) dn = fmaf(zq[k], load_elem<BF16>(a.zhard, row * d + k), dn);
    const float h = dn - pos + a.margin;
    hh += h > 0.0f ? h : 0.0f;
    ++hv;
  }
#pragma unroll
  for (int o = TPQ / 2; o >= 1; o >>= 1) {
    hh += __shfl_xor(hh, o);
    hv += __shfl_xor(hv, o);
  }
  if (c == 0 && b < a.B) a.per_pair[b] = (acc + hh) / (float)(a.n_neg + hv);
}

// Mean over pairs in a fixed order: strided per-thread sums, then a fixed tree.
__global__ __launch_bounds__(256) void loss_mean_kernel(const float* per_pair, int64_t B,
                                                        float* loss) {
  __shared__ float part[256];
  float s = 0.0f;
  for (int64_t i = threadIdx.x; i < B; i += 256) s += per_pair[i];
  part[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = part[0] / (float)B;
}

// out[i][:] = table[rows[i]][:] (zero row for rows[i] < 0); 16-byte vectors.
__global__ void gather_rows_kernel(const uint4* table, const int32_t* rows, int64_t n,
                                   int vec_per_row, uint4* out) {
  const int64_t total = n * vec_per_row;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / vec_per_row;
    const int c = (int)(i % vec_per_row);
    const int32_t src = rows[r];
    out[i] = src >= 0 ? table[(int64_t)src * vec_per_row + c] : make_uint4(0, 0, 0, 0);
  }
}

inline dim3 grid_for(int64_t n, int threads = 256) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > 65536) b = 65536;
  return dim3((unsigned)b);
}

}  // namespace

hipError_t launch_fill_zero_u8(uint8_t* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_u8_kernel, grid_for(n), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_mark(const int32_t* ids, int64_t n, int64_t N, uint8_t* flags, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfileScope prof(kKMinibatch, s);
  hipLaunchKernelGGL(mark_kernel, grid_for(n), dim3(256), 0, s, ids, n, N, flags);
  return hipGetLastError();
}

int64_t scan_tiles(int64_t N) { return (N + kScanTile - 1) / kScanTile; }

hipError_t launch_flag_scan(const uint8_t* flags, int64_t N, int32_t* tile_sums, int32_t* pos,
                            int32_t* set, int64_t cap, long long* total, hipStream_t s) {
  const int64_t tiles = scan_tiles(N);
  if (tiles <= 0 || tiles > 0x7FFFFFFF) return hipErrorInvalidValue;
  ProfileScope prof(kKMinibatch, s);
  hipLaunchKernelGGL(scan_tile_sums_kernel, dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                     flags, N, tile_sums);
  hipLaunchKernelGGL(scan_tile_offsets_kernel, dim3(1), dim3(1024), 0, s, tile_sums, tiles, total);
  hipLaunchKernelGGL(scan_tile_finish_kernel, dim3((unsigned)tiles), dim3(kScanThreads), 0, s,
                     flags, N, tile_sums, pos, set, cap);
  return hipGetLastError();
}

hipError_t launch_count_below(const int32_t* set, const long long* size_dev, int64_t cap,
                              int64_t bound, long long* count, hipStream_t s) {
  hipError_t e = launch_zero_u64(reinterpret_cast<unsigned long long*>(count), 1, s);
  if (e != hipSuccess || cap <= 0) return e;
  hipLaunchKernelGGL(count_below_kernel, grid_for(cap), dim3(256), 0, s, set, size_dev, cap, bound,
                     count);
  return hipGetLastError();
}

hipError_t launch_remap(const int32_t* in, int64_t n, int64_t N, const int32_t* pos, int32_t* out,
                        hipStream_t s) {
  if (n <= 0) return hipSuccess;
  ProfileScope prof(kKMinibatch, s);
  hipLaunchKernelGGL(remap_kernel, grid_for(n), dim3(256), 0, s, in, n, N, pos, out);
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* table, const int32_t* rows, int64_t n, int64_t row_bytes,
                              void* out, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (row_bytes % 16) return hipErrorInvalidValue;
  const int vpr = (int)(row_bytes / 16);
  hipLaunchKernelGGL(gather_rows_kernel, grid_for(n * vpr), dim3(256), 0, s,
                     static_cast<const uint4*>(table), rows, n, vpr, static_cast<uint4*>(out));
  return hipGetLastError();
}

template <int THREADS, int QB, int NC, int DMAX>
void launch_loss_cfg(const LossLaunch& a, hipStream_t s) {
  const dim3 grid((unsigned)((a.B + QB - 1) / QB)), block(THREADS);
  if (a.bf16) hipLaunchKernelGGL((loss_pairs_kernel<true, THREADS, QB, NC, DMAX>), grid, block, 0,
                                 s, a);
  else hipLaunchKernelGGL((loss_pairs_kernel<false, THREADS, QB, NC, DMAX>), grid, block, 0, s, a);
}

hipError_t launch_loss(const LossLaunch& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  if (a.d < 1 || a.d > 1024 || a.B >= (1ll << 32)) return hipErrorInvalidValue;
  ProfileScope prof(kKLoss, s);
  // LDS per block: (QB + NC) * (DMAX + 1) * 4 bytes <= 148 KB.
  if (a.d <= 256) launch_loss_cfg<256, 8, 128, 256>(a, s);
  else if (a.d <= 512) launch_loss_cfg<256, 8, 64, 512>(a, s);
  else launch_loss_cfg<128, 4, 32, 1024>(a, s);
  hipLaunchKernelGGL(loss_mean_kernel, dim3(1), dim3(256), 0, s, a.per_pair, a.B, a.loss);
  return hipGetLastError();
}

}  // namespace pinsage
