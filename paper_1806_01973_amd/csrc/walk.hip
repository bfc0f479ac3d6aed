// Importance neighbourhoods on gfx950 (Sec. 3.2, "Importance-based
// neighborhoods"): short random walks from every source, visit counting and
// top-T selection with L1-normalised weights.
//
// One wavefront owns one source at a time, or two when a source has at most
// 64 walks (grid-stride over sources):
//   1. walk phase: lane l runs walks l, l+64, ... (or walk l of both
//      sources); walk w writes its `hops`
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

// NSRC sources per wave at a time: with walks <= 64, lane l walks walk l of
// two neighbouring sources at once (walkers A and B), so twice as many
// dependent reads are in flight per wave; with more walks, lane l walks walks
// l and l + 64 of one source.
// TABLE: each edge step reads one 16-byte walk-table entry (the neighbour's id
// and row) instead of the current node's offset pair and a neighbour id.
template <typename OffT, int E, int NSRC, bool TABLE>
__global__ __launch_bounds__(256) void walk_topt_kernel(WalkLaunch a) {
  // Per wave and source: the visit slots (64*E), reused to stage the output
  // row (ids at [0, T), counts at [kStripOut, kStripOut + T)).
  constexpr int kStrip = kWave * E > 2 * kMaxTopT ? kWave * E : 2 * kMaxTopT;
  __shared__ uint32_t strip_all[kWavesPerBlock][NSRC][kStrip];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const uint4* __restrict__ tab = static_cast<const uint4*>(a.table);
  const int WH = a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  const int T = a.top_t;
  unsigned long long wave_steps = 0;

  // Steps 2-5 for one source whose visits fill `strip`.
  auto finish_source = [&](int64_t row, uint32_t* strip) __attribute__((always_inline)) {
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
    // The kept entries are placed by rank in the strip (ids, then counts),
    // then written with contiguous stores.
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
  };

  const int64_t groups = (a.num_sources + NSRC - 1) / NSRC;
  for (int64_t grp = (int64_t)blockIdx.x * kWavesPerBlock + wave; grp < groups;
       grp += (int64_t)gridDim.x * kWavesPerBlock) {
    int64_t rows[NSRC], us[NSRC];
    bool lives[NSRC];
#pragma unroll
    for (int q = 0; q < NSRC; ++q) {
      rows[q] = grp * NSRC + q;
      const bool in = rows[q] < a.num_sources;
      us[q] = in ? (a.sources ? (int64_t)a.sources[rows[q]] : rows[q]) : -1;
      lives[q] = in && us[q] >= 0 && us[q] < a.num_nodes;
    }
    uint32_t my_steps = 0;  // this lane's edge steps for these sources

    // ---- 1. walks -------------------------------------------------------
#pragma unroll
    for (int q = 0; q < NSRC; ++q)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int slot = lane * E + e;
        if (slot >= WH || !lives[q]) strip_all[wave][q][slot] = kEmpty;
      }
    bool any_live = false;
#pragma unroll
    for (int q = 0; q < NSRC; ++q) any_live = any_live || lives[q];
    if (any_live) {
      // Two walks per lane in lockstep, so their dependent offset ->
      // neighbour reads overlap: walk w0 of each of the two sources, or
      // walks w0 and w0 + 64 of the one source.
      const int wstep = NSRC == 2 ? kWave : 2 * kWave;
      // Table path: the sources' rows, validated as pick() validates them.
      int64_t slo[NSRC];
      int32_t sdeg[NSRC];
      if constexpr (TABLE) {
#pragma unroll
        for (int q = 0; q < NSRC; ++q) {
          slo[q] = 0;
          sdeg[q] = 0;
          if (lives[q]) {
            const int64_t lo = (int64_t)off[us[q]], hi = (int64_t)off[us[q] + 1];
            if (!(hi - lo <= 0 || lo < 0 || hi > a.nnz)) {
              slo[q] = lo;
              sdeg[q] = (int32_t)(hi - lo);
            }
          }
        }
      }
      for (int w0 = lane; w0 < a.walks; w0 += wstep) {
        Walker<OffT> A, B;
        if constexpr (NSRC == 2) {
          A.start(us[0], w0, strip_all[wave][0] + w0 * a.hops, lives[0]);
          B.start(us[1], w0, strip_all[wave][1] + w0 * a.hops, lives[1]);
        } else {
          A.start(us[0], w0, strip_all[wave][0] + w0 * a.hops, lives[0]);
          B.start(us[0], w0 + kWave, strip_all[wave][0] + (w0 + kWave) * a.hops,
                  lives[0] && w0 + kWave < a.walks);
        }
        if constexpr (TABLE) {
          A.lo = slo[0];
          A.deg = sdeg[0];
          B.lo = slo[NSRC - 1];
          B.deg = sdeg[NSRC - 1];
          while (A.active || B.active) {
            A.pick_carried(k0, k1);
            B.pick_carried(k0, k1);
            const uint4 eA = A.active ? tab[A.next_at] : make_uint4(0u, 0u, 0u, 0u);
            const uint4 eB = B.active ? tab[B.next_at] : make_uint4(0u, 0u, 0u, 0u);
            A.land_entry(eA, a.num_pins, a.num_nodes, a.hops);
            B.land_entry(eB, a.num_pins, a.num_nodes, a.hops);
          }
        } else {
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
        }
        my_steps += A.finish(a.hops) + B.finish(a.hops);
      }
    }
    wave_lds_sync();

    if (a.total_steps) wave_steps += (unsigned)wave_sum_i32((int)my_steps);

#pragma unroll
    for (int q = 0; q < NSRC; ++q)
      if (rows[q] < a.num_sources) finish_source(rows[q], strip_all[wave][q]);
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

template <typename OffT>
__global__ void walk_table_kernel(const OffT* __restrict__ off, const int32_t* __restrict__ col,
                                  int64_t nnz, int64_t num_nodes, uint4* __restrict__ table) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nnz;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = col[e];
    uint32_t deg = 0;
    uint64_t lo = 0;
    if (v >= 0 && (int64_t)v < num_nodes) {
      const int64_t l = (int64_t)off[v], h = (int64_t)off[v + 1];
      if (!(h - l <= 0 || l < 0 || h > nnz)) {
        deg = (uint32_t)(h - l);
        lo = (uint64_t)l;
      }
    }
    table[e] = make_uint4((uint32_t)v, deg, (uint32_t)lo, (uint32_t)(lo >> 32));
  }
}

__global__ void zero_u64_kernel(unsigned long long* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0ull;
}

template <typename OffT, int NSRC, bool TABLE>
hipError_t launch_sized(const WalkLaunch& a, hipStream_t s) {
  const int wh = a.walks * a.hops;
  const int64_t groups = (a.num_sources + NSRC - 1) / NSRC;
  const int64_t blocks_needed = (groups + kWavesPerBlock - 1) / kWavesPerBlock;
  // Enough resident blocks to fill the chip several times over; waves then
  // loop over sources.
  const int64_t cap = 1ll << 14;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  const dim3 block(256);
  if (wh <= 64)
    hipLaunchKernelGGL((walk_topt_kernel<OffT, 1, NSRC, TABLE>), grid, block, 0, s, a);
  else if (wh <= 128)
    hipLaunchKernelGGL((walk_topt_kernel<OffT, 2, NSRC, TABLE>), grid, block, 0, s, a);
  else if (wh <= 256)
    hipLaunchKernelGGL((walk_topt_kernel<OffT, 4, NSRC, TABLE>), grid, block, 0, s, a);
  else if (wh <= 512)
    hipLaunchKernelGGL((walk_topt_kernel<OffT, 8, NSRC, TABLE>), grid, block, 0, s, a);
  else if (wh <= 1024)
    hipLaunchKernelGGL((walk_topt_kernel<OffT, 16, NSRC, TABLE>), grid, block, 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename OffT, bool TABLE>
hipError_t launch_for_table(const WalkLaunch& a, hipStream_t s) {
  // Two sources per wave when one source's walks leave a lane's second walker idle.
  return a.walks <= kWave ? launch_sized<OffT, 2, TABLE>(a, s) : launch_sized<OffT, 1, TABLE>(a, s);
}

template <typename OffT>
hipError_t launch_for_offsets(const WalkLaunch& a, hipStream_t s) {
  return a.table ? launch_for_table<OffT, true>(a, s) : launch_for_table<OffT, false>(a, s);
}

}  // namespace

hipError_t launch_walk_topt(const WalkLaunch& a, hipStream_t s) {
  if (a.num_sources <= 0) return hipSuccess;
  ProfileScope prof(kKWalk, s);
  return a.offsets64 ? launch_for_offsets<int64_t>(a, s) : launch_for_offsets<int32_t>(a, s);
}

hipError_t launch_walk_table(const void* row_offsets, bool offsets64, const int32_t* col,
                             int64_t nnz, int64_t num_nodes, void* table, hipStream_t s) {
  if (nnz <= 0) return hipSuccess;
  if (nnz > kWalkTableMaxNnz) return hipErrorInvalidValue;
  ProfileScope prof(kKWalkTable, s);
  const int64_t blocks = (nnz + 255) / 256;
  const dim3 grid((unsigned)(blocks < 65536 ? blocks : 65536));
  uint4* t = static_cast<uint4*>(table);
  if (offsets64)
    hipLaunchKernelGGL(walk_table_kernel<int64_t>, grid, dim3(256), 0, s,
                       static_cast<const int64_t*>(row_offsets), col, nnz, num_nodes, t);
  else
    hipLaunchKernelGGL(walk_table_kernel<int32_t>, grid, dim3(256), 0, s,
                       static_cast<const int32_t*>(row_offsets), col, nnz, num_nodes, t);
  return hipGetLastError();
}

hipError_t launch_zero_u64(unsigned long long* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(zero_u64_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace pinsage
