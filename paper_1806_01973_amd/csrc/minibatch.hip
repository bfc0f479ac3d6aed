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

// Eq. (1) per pair: one wavefront per query b; each lane keeps d/64 entries
// of z_q in registers; dot products are wave sums in a fixed butterfly order,
// and the hinge terms are added in negative order.
template <bool BF16, int PER_LANE>
__global__ __launch_bounds__(256) void loss_pairs_kernel(LossLaunch a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int d = a.d;
  for (int64_t b = (int64_t)blockIdx.x * 4 + wave; b < a.B; b += (int64_t)gridDim.x * 4) {
    const int64_t qr = a.q_rows ? (int64_t)a.q_rows[b] : b;
    const int64_t pr = a.pos_rows ? (int64_t)a.pos_rows[b] : b;
    float zq[PER_LANE];
    float dp = 0.0f;
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) {
      const int j = lane + 64 * i;
      zq[i] = (j < d && qr >= 0) ? load_elem<BF16>(a.zq, qr * d + j) : 0.0f;
      const float zp = (j < d && pr >= 0) ? load_elem<BF16>(a.zpos, pr * d + j) : 0.0f;
      dp = fmaf(zq[i], zp, dp);
    }
    const float pos = wave_sum_f32(dp);
    float acc = 0.0f;
    for (int64_t n = 0; n < a.n_neg; ++n) {
      const int64_t nr = a.neg_rows ? (int64_t)a.neg_rows[n] : n;
      float dn = 0.0f;
#pragma unroll
      for (int i = 0; i < PER_LANE; ++i) {
        const int j = lane + 64 * i;
        const float zn = (j < d && nr >= 0) ? load_elem<BF16>(a.zneg, nr * d + j) : 0.0f;
        dn = fmaf(zq[i], zn, dn);
      }
      const float neg = wave_sum_f32(dn);
      const float h = neg - pos + a.margin;
      acc += h > 0.0f ? h : 0.0f;
    }
    if (lane == 0) a.per_pair[b] = acc / (float)a.n_neg;
  }
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

hipError_t launch_loss(const LossLaunch& a, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  ProfileScope prof(kKLoss, s);
  const int per_lane = (a.d + 63) / 64;
  int64_t blocks = (a.B + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  const dim3 grid((unsigned)blocks), block(256);
#define PINSAGE_LOSS(PL)                                                                    \
  if (a.bf16) hipLaunchKernelGGL((loss_pairs_kernel<true, PL>), grid, block, 0, s, a);      \
  else hipLaunchKernelGGL((loss_pairs_kernel<false, PL>), grid, block, 0, s, a);
  if (per_lane <= 1) { PINSAGE_LOSS(1) }
  else if (per_lane <= 2) { PINSAGE_LOSS(2) }
  else if (per_lane <= 4) { PINSAGE_LOSS(4) }
  else if (per_lane <= 8) { PINSAGE_LOSS(8) }
  else if (per_lane <= 16) { PINSAGE_LOSS(16) }
  else return hipErrorInvalidValue;
#undef PINSAGE_LOSS
  hipLaunchKernelGGL(loss_mean_kernel, dim3(1), dim3(256), 0, s, a.per_pair, a.B, a.loss);
  return hipGetLastError();
}

}  // namespace pinsage
