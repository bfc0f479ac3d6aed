// Graph neighbourhoods of the MapReduce inference of Sec. 3.4 on gfx950:
// a board pools the pins it holds and a pin pools its boards, with long rows
// sampled.
//
// One wavefront per node (grid-stride over sources). The node's entries --
// its CSR row when the row has at most T entries, else T draws (word 0 of
// Philox4x32-10 at counter (u, j, 0, 2), position floor(r * deg / 2^32)) --
// land E per lane in registers (entries outside the graph become empty), a
// register bitonic sort groups equal ids, and the runs give each distinct id
// its multiplicity; distinct ids are written in ascending order with weight
// multiplicity / kept entries (one fp32 division).
#include "device_util.h"
#include "kernels.h"
#include "walk_device.h"

namespace pinsage {
namespace {

using namespace walkdev;

constexpr int kWavesPerBlock = 4;

template <typename OffT, int E>
__global__ __launch_bounds__(256) void graph_nbr_kernel(GraphNbrLaunch a) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int T = a.top_t;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);

  for (int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wave; row < a.num_sources;
       row += (int64_t)gridDim.x * kWavesPerBlock) {
    const int64_t u = a.sources ? (int64_t)a.sources[row] : row;
    const bool live = u >= 0 && u < a.num_nodes;
    int64_t lo = 0, deg = 0;
    if (live) {
      lo = (int64_t)off[u];
      const int64_t hi = (int64_t)off[u + 1];
      if (lo >= 0 && hi <= a.nnz && hi > lo) deg = hi - lo;
    }
    // Entry i = lane * E + e (row position i, or draw i).
    uint32_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      int64_t pos = -1;
      if (deg > 0 && i < T) {
        if (deg <= T) {
          pos = i < deg ? lo + i : -1;
        } else {
          const uint4 r = philox4x32_10(make_uint4((uint32_t)u, (uint32_t)i, 0u, 2u), k0, k1);
          pos = lo + (int64_t)(((uint64_t)r.x * (uint64_t)deg) >> 32);
        }
      }
      uint32_t k = kEmpty;
      if (pos >= 0) {
        const int32_t v = a.col[pos];
        if (v >= 0 && (int64_t)v < a.num_nodes) k = (uint32_t)v;
      }
      key[e] = k;
    }
    bitonic_sort_wave<E>(key, lane);

    // Runs: heads get their rank d (number of heads before them), tails their
    // run length (position of the tail minus that of the run's head, + 1).
    const uint32_t prev_last = __shfl_up(key[E - 1], 1);
    const uint32_t next_first = __shfl_down(key[0], 1);
    bool head[E], tail[E];
    int nhead = 0, kept = 0, lane_last_head = -1;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      const uint32_t prev = e == 0 ? (lane == 0 ? kEmpty : prev_last) : key[e - 1];
      const uint32_t next = e == E - 1 ? (lane == kWave - 1 ? kEmpty : next_first) : key[e + 1];
      head[e] = key[e] != kEmpty && prev != key[e];
      tail[e] = key[e] != kEmpty && next != key[e];
      nhead += head[e] ? 1 : 0;
      kept += key[e] != kEmpty ? 1 : 0;
      if (head[e]) lane_last_head = i;
    }
    const int heads_incl = wave_inclusive_sum(nhead, lane);
    const int D = __builtin_amdgcn_readlane(heads_incl, kWave - 1);
    const int total_kept = wave_sum_i32(kept);
    const int incl_last = wave_inclusive_max(lane_last_head, lane);
    int head_pos = __shfl_up(incl_last, 1);
    if (lane == 0) head_pos = -1;
    int d = heads_incl - nhead;  // heads before this lane
    const int64_t base = row * (int64_t)T;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (head[e]) {
        head_pos = i;
        a.idx[base + d] = (int32_t)key[e];
        ++d;
      }
      if (tail[e]) {
        const int cnt = i - head_pos + 1;
        a.counts[base + d - 1] = (uint16_t)cnt;
        if (a.weights) a.weights[base + d - 1] = (float)cnt / (float)total_kept;
      }
    }
    for (int t = D + lane; t < T; t += kWave) {
      a.idx[base + t] = -1;
      a.counts[base + t] = 0;
      if (a.weights) a.weights[base + t] = 0.0f;
    }
  }
}

template <typename OffT>
hipError_t launch_for_offsets(const GraphNbrLaunch& a, hipStream_t s) {
  const int64_t blocks_needed = (a.num_sources + kWavesPerBlock - 1) / kWavesPerBlock;
  const int64_t cap = 1ll << 14;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  const dim3 block(256);
  if (a.top_t <= 64) hipLaunchKernelGGL((graph_nbr_kernel<OffT, 1>), grid, block, 0, s, a);
  else if (a.top_t <= 128) hipLaunchKernelGGL((graph_nbr_kernel<OffT, 2>), grid, block, 0, s, a);
  else if (a.top_t <= 256) hipLaunchKernelGGL((graph_nbr_kernel<OffT, 4>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// map[i] = i for i < valid, -1 after (rows past `valid` read as zero rows).
__global__ void row_map_kernel(int32_t* map, int64_t n, int64_t valid) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    map[i] = i < valid ? (int32_t)i : -1;
}

}  // namespace

hipError_t launch_graph_neighborhoods(const GraphNbrLaunch& a, hipStream_t s) {
  if (a.num_sources <= 0) return hipSuccess;
  ProfileScope prof(kKGraphNbr, s);
  return a.offsets64 ? launch_for_offsets<int64_t>(a, s) : launch_for_offsets<int32_t>(a, s);
}

hipError_t launch_row_map(int32_t* map, int64_t n, int64_t valid, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(row_map_kernel, dim3((unsigned)blocks), dim3(256), 0, s, map, n, valid);
  return hipGetLastError();
}

}  // namespace pinsage
