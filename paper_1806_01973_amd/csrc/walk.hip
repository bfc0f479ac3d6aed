// Importance neighbourhoods on gfx950 (Sec. 3.2, "Importance-based
// neighborhoods"): short random walks from every source, visit counting and
// top-T selection with L1-normalised weights.
//
// One wavefront owns one source at a time (grid-stride over sources):
//   1. walk phase: lane l runs walks l, l+64, ...; walk w writes its `hops`
//      pin landings (or an empty marker) into slots [w*hops, (w+1)*hops) of the
//      wave's LDS strip; slots past walks*hops are pre-filled empty;
//   2. each lane pulls E consecutive slots into registers and the wave sorts
//      the 64*E visit ids with a register bitonic network (cross-lane stages
//      through lane shuffles), so equal ids become runs;
//   3. run boundaries and a wave max-scan give every distinct id its visit
//      count (held at the run's last element);
//   4. the count classes are visited from the highest count down: as ids are
//      ascending, an entry's rank in (count desc, id asc) order is the number
//      of entries in the classes above plus its position in its own class;
//      ranks below T are written with their weights.
// Walk randomness: Philox4x32-10 at counter (u, w, s/4, 0), key = seed, word
// s%4 for edge step s; neighbour index floor(r * deg / 2^32).
#include "device_util.h"
#include "kernels.h"
#include "walk_device.h"

namespace pinsage {
namespace {

using namespace walkdev;

constexpr int kWavesPerBlock = 4;
constexpr int kMaxTopT = 256;
// Second half of a wave's LDS strip: the kept counts, by rank.
constexpr int kStripOut = kMaxTopT;

template <typename OffT, int E>
__global__ __launch_bounds__(256) void walk_topt_kernel(WalkLaunch a) {
  // Per wave: the visit slots (64*E), reused to stage the output row
  // (ids at [0, T), counts at [kStripOut, kStripOut + T)).
  constexpr int kStrip = kWave * E > 2 * kMaxTopT ? kWave * E : 2 * kMaxTopT;
  __shared__ uint32_t strip_all[kWavesPerBlock][kStrip];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  uint32_t* strip = strip_all[wave];
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const int WH = a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  const int T = a.top_t;
  unsigned long long wave_steps = 0;

  for (int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wave; row < a.num_sources;
       row += (int64_t)gridDim.x * kWavesPerBlock) {
    const int64_t u = a.sources ? (int64_t)a.sources[row] : row;
    const bool live = u >= 0 && u < a.num_nodes;
    uint32_t my_steps = 0;  // this lane's edge steps for this source

    // ---- 1. walks -------------------------------------------------------
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = lane * E + e;
      if (slot >= WH || !live) strip[slot] = kEmpty;
    }
    if (live) {
      // Two walks per lane in lockstep (w0 and w0 + 64): their dependent
      // offset -> neighbour reads overlap.
      for (int w0 = lane; w0 < a.walks; w0 += 2 * kWave) {
        Walker<OffT> A, B;
        A.start(u, w0, strip + w0 * a.hops, true);
        B.start(u, w0 + kWave, strip + (w0 + kWave) * a.hops, w0 + kWave < a.walks);
        while (A.active || B.active) {
          int64_t loA = 0, hiA = 0, loB = 0, hiB = 0;
          if (A.active) {
            loA = (int64_t)off[A.cur];
            hiA = (int64_t)off[A.cur + 1];
          }
          if (B.active) {
            loB = (int64_t)off[B.cur];
            hiB = (int64_t)off[B.cur + 1];
          }
          A.pick(loA, hiA, a.nnz, k0, k1);
          B.pick(loB, hiB, a.nnz, k0, k1);
          const int32_t nA = A.active ? col[A.next_at] : 0;
          const int32_t nB = B.active ? col[B.next_at] : 0;
          A.land(nA, a.num_pins, a.num_nodes, a.hops);
          B.land(nB, a.num_pins, a.num_nodes, a.hops);
        }
        my_steps += A.finish(a.hops) + B.finish(a.hops);
      }
    }
    wave_lds_sync();

    if (a.total_steps) wave_steps += (unsigned)wave_sum_i32((int)my_steps);

    // ---- 2. sort visits by id -------------------------------------------
    uint32_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) key[e] = strip[lane * E + e];
    wave_lds_sync();
    bitonic_sort_wave<E>(key, lane);

    // ---- 3. runs -> visit count of each distinct id (at the run's tail) --
    const uint32_t prev_last = __shfl_up(key[E - 1], 1);
    const uint32_t next_first = __shfl_down(key[0], 1);
    bool head[E];
    int lane_last_head = -1;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      const uint32_t prev = e == 0 ? prev_last : key[e - 1];
      head[e] = key[e] != kEmpty && (i == 0 || prev != key[e]);
      if (head[e]) lane_last_head = i;
    }
    const int incl_last = wave_inclusive_max(lane_last_head, lane);
    int head_pos = __shfl_up(incl_last, 1);
    if (lane == 0) head_pos = -1;
    int cnt[E];
    int lane_cmax = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (head[e]) head_pos = i;
      const uint32_t next = e == E - 1 ? (lane == kWave - 1 ? kEmpty : next_first) : key[e + 1];
      const bool tail = key[e] != kEmpty && next != key[e];
      cnt[e] = tail ? i - head_pos + 1 : 0;
      lane_cmax = cnt[e] > lane_cmax ? cnt[e] : lane_cmax;
    }

    // ---- 4. rank by (count desc, id asc); keep the first T ---------------
    // Ids ascend across (lane, e), so inside one count class the rank order is
    // the position order. Classes are visited from the highest count down; an
    // entry's rank is the number of entries in the classes above plus its
    // position in its own class (a wave scan per class).
    int rank[E];
#pragma unroll
    for (int e = 0; e < E; ++e) rank[e] = T;  // T = not kept
    int placed = 0;    // entries in the classes visited so far
    int kept_sum = 0;  // sum of the kept counts
    int c = wave_max_i32(lane_cmax);
    while (c > 0 && placed < T) {
      int lc = 0;
#pragma unroll
      for (int e = 0; e < E; ++e) lc += cnt[e] == c ? 1 : 0;
      const int incl = wave_inclusive_sum(lc, lane);
      const int total_c = __builtin_amdgcn_readlane(incl, kWave - 1);
      int r = placed + incl - lc;
      int below = 0;
      // Branch-free: every element takes the same instruction path.
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const bool in = cnt[e] == c;
        rank[e] = (in && r < T) ? r : rank[e];
        r += in ? 1 : 0;
        below = (cnt[e] < c && cnt[e] > below) ? cnt[e] : below;
      }
      const int take = total_c < T - placed ? total_c : T - placed;
      kept_sum += take * c;
      placed += total_c;
      c = wave_max_i32(below);
    }
    const int keep = placed < T ? placed : T;

    // ---- 5. write the row -------------------------------------------------
    // The kept entries are placed by rank in the wave's LDS strip (ids, then
    // counts), then written with contiguous stores.
    wave_lds_sync();
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if (rank[e] < T) {
        strip[rank[e]] = key[e];
        strip[kStripOut + rank[e]] = (uint32_t)cnt[e];
      }
    }
    wave_lds_sync();
    const int64_t base = row * (int64_t)T;
    for (int i = lane; i < T; i += kWave) {
      const bool kept = i < keep;
      const uint32_t cc = kept ? strip[kStripOut + i] : 0u;
      a.idx[base + i] = kept ? (int32_t)strip[i] : -1;
      a.counts[base + i] = (uint16_t)cc;
      if (a.weights) a.weights[base + i] = kept ? (float)cc / (float)kept_sum : 0.0f;
    }
    wave_lds_sync();
  }
  // Edge steps: one sum per wave over all its sources, one atomic per block
  // (a per-source atomic on the single counter serialises at its L2 channel).
  if (a.total_steps) {
    __shared__ unsigned long long block_steps[kWavesPerBlock];
    const unsigned long long ws = (unsigned long long)wave_steps;
    if (lane == 0) block_steps[wave] = ws;
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long t = 0;
      for (int w = 0; w < kWavesPerBlock; ++w) t += block_steps[w];
      if (t) atomicAdd(a.total_steps, t);
    }
  }
}

__global__ void zero_u64_kernel(unsigned long long* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

template <typename OffT>
hipError_t launch_for_offsets(const WalkLaunch& a, hipStream_t s) {
  const int wh = a.walks * a.hops;
  const int64_t blocks_needed = (a.num_sources + kWavesPerBlock - 1) / kWavesPerBlock;
  // Enough resident blocks to fill the chip several times over; waves then
  // loop over sources.
  const int64_t cap = 1ll << 14;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  const dim3 block(256);
  if (wh <= 64) hipLaunchKernelGGL((walk_topt_kernel<OffT, 1>), grid, block, 0, s, a);
  else if (wh <= 128) hipLaunchKernelGGL((walk_topt_kernel<OffT, 2>), grid, block, 0, s, a);
  else if (wh <= 256) hipLaunchKernelGGL((walk_topt_kernel<OffT, 4>), grid, block, 0, s, a);
  else if (wh <= 512) hipLaunchKernelGGL((walk_topt_kernel<OffT, 8>), grid, block, 0, s, a);
  else if (wh <= 1024) hipLaunchKernelGGL((walk_topt_kernel<OffT, 16>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_walk_topt(const WalkLaunch& a, hipStream_t s) {
  if (a.num_sources <= 0) return hipSuccess;
  ProfileScope prof(kKWalk, s);
  return a.offsets64 ? launch_for_offsets<int64_t>(a, s) : launch_for_offsets<int32_t>(a, s);
}

hipError_t launch_zero_u64(unsigned long long* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(zero_u64_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace pinsage
