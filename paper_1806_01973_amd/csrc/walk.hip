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
//   3. run boundaries and two wave scans give every distinct id its visit
//      count c and its rank p in id order; the distinct ids are parked in LDS
//      by p;
//   4. a second bitonic sort of the keys (0xFFFF - c) << 16 | p puts the
//      distinct ids in (count desc, id asc) order; the first T are written.
// Walk randomness: Philox4x32-10 at counter (u, w, s/4, 0), key = seed, word
// s%4 for edge step s; neighbour index floor(r * deg / 2^32).
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

constexpr uint32_t kEmpty = 0xFFFFFFFFu;
constexpr int kWavesPerBlock = 4;

template <int E>
__device__ __forceinline__ void bitonic_sort_wave(uint32_t (&k)[E], int lane) {
#pragma unroll
  for (int size = 2; size <= kWave * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= E) {
        const int lane_mask = stride / E;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const uint32_t other = __shfl_xor(k[e], lane_mask);
          const int i = lane * E + e;
          const bool ascending = (i & size) == 0;
          const bool lower = (i & stride) == 0;
          const uint32_t lo = k[e] < other ? k[e] : other;
          const uint32_t hi = k[e] < other ? other : k[e];
          k[e] = (ascending == lower) ? lo : hi;
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & stride) == 0) {
            const int i = lane * E + e;
            const bool ascending = (i & size) == 0;
            const uint32_t a = k[e], b = k[e + stride];
            const bool swap = ascending ? (a > b) : (a < b);
            k[e] = swap ? b : a;
            k[e + stride] = swap ? a : b;
          }
        }
      }
    }
  }
}

__device__ __forceinline__ uint32_t pick_word(const uint4& r, int s) {
  const int q = s & 3;
  return q == 0 ? r.x : (q == 1 ? r.y : (q == 2 ? r.z : r.w));
}

template <typename OffT, int E>
__global__ __launch_bounds__(256) void walk_topt_kernel(WalkLaunch a) {
  __shared__ uint32_t strip_all[kWavesPerBlock][kWave * E];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  uint32_t* strip = strip_all[wave];
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const int WH = a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  const int T = a.top_t;

  for (int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wave; row < a.num_sources;
       row += (int64_t)gridDim.x * kWavesPerBlock) {
    const int64_t u = a.sources ? (int64_t)a.sources[row] : row;
    const bool live = u >= 0 && u < a.num_nodes;
    uint32_t my_steps = 0;

    // ---- 1. walks -------------------------------------------------------
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = lane * E + e;
      if (slot >= WH || !live) strip[slot] = kEmpty;
    }
    if (live) {
      for (int w = lane; w < a.walks; w += kWave) {
        uint32_t* mine = strip + w * a.hops;
        int64_t cur = u;
        int landed = 0;
        int s = 0;
        uint4 rnd = make_uint4(0, 0, 0, 0);
        while (landed < a.hops && s < 2 * a.hops) {
          const int64_t lo = (int64_t)off[cur];
          const int64_t hi = (int64_t)off[cur + 1];
          const int64_t deg = hi - lo;
          if (deg <= 0 || lo < 0 || hi > a.nnz) break;
          if ((s & 3) == 0)
            rnd = philox4x32_10(make_uint4((uint32_t)u, (uint32_t)w, (uint32_t)(s >> 2), 0u), k0,
                                k1);
          const uint32_t r = pick_word(rnd, s);
          const int64_t j = (int64_t)(((uint64_t)r * (uint64_t)deg) >> 32);
          const int32_t nxt = col[lo + j];
          if (nxt < 0 || (int64_t)nxt >= a.num_nodes) break;
          cur = nxt;
          ++s;
          if (cur < a.num_pins) {
            mine[landed] = (cur != u) ? (uint32_t)cur : kEmpty;
            ++landed;
          }
        }
        for (int h = landed; h < a.hops; ++h) mine[h] = kEmpty;
        my_steps += (uint32_t)s;
      }
    }
    wave_lds_sync();

    // ---- 2. sort visits by id -------------------------------------------
    uint32_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) key[e] = strip[lane * E + e];
    wave_lds_sync();
    bitonic_sort_wave<E>(key, lane);

    // ---- 3. runs -> (count, rank in id order) ----------------------------
    const uint32_t prev_last = __shfl_up(key[E - 1], 1);
    const uint32_t next_first = __shfl_down(key[0], 1);
    bool head[E], tail[E];
    int lane_heads = 0;
    int lane_last_head = -1;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      const bool valid = key[e] != kEmpty;
      const bool has_prev = i > 0;
      const uint32_t prev = e == 0 ? prev_last : key[e - 1];
      const uint32_t next = e == E - 1 ? (lane == kWave - 1 ? kEmpty : next_first) : key[e + 1];
      head[e] = valid && (!has_prev || prev != key[e]);
      tail[e] = valid && next != key[e];
      if (head[e]) {
        ++lane_heads;
        lane_last_head = i;
      }
    }
    const int incl_heads = wave_inclusive_sum(lane_heads, lane);
    const int distinct = __shfl(incl_heads, kWave - 1);
    int run_heads = incl_heads - lane_heads;
    const int incl_last = wave_inclusive_max(lane_last_head, lane);
    int head_pos = __shfl_up(incl_last, 1);
    if (lane == 0) head_pos = -1;
    uint32_t key2[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (head[e]) {
        head_pos = i;
        ++run_heads;
      }
      key2[e] = kEmpty;
      if (tail[e]) {
        const uint32_t c = (uint32_t)(i - head_pos + 1);
        const uint32_t p = (uint32_t)(run_heads - 1);
        key2[e] = ((0xFFFFu - c) << 16) | p;
        strip[p] = key[e];
      }
    }
    wave_lds_sync();

    // ---- 4. order by (count desc, id asc); keep the first T ---------------
    bitonic_sort_wave<E>(key2, lane);
    const int keep = distinct < T ? distinct : T;
    int my_sum = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (i < keep) my_sum += (int)(0xFFFFu - (key2[e] >> 16));
    }
    const int total = wave_sum_i32(my_sum);
    const int64_t base = row * (int64_t)T;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = lane * E + e;
      if (i < T) {
        if (i < keep) {
          const uint32_t c = 0xFFFFu - (key2[e] >> 16);
          const uint32_t p = key2[e] & 0xFFFFu;
          a.idx[base + i] = (int32_t)strip[p];
          a.counts[base + i] = (uint16_t)c;
          if (a.weights) a.weights[base + i] = (float)c / (float)total;
        } else {
          a.idx[base + i] = -1;
          a.counts[base + i] = 0;
          if (a.weights) a.weights[base + i] = 0.0f;
        }
      }
    }
    for (int i = kWave * E + lane; i < T; i += kWave) {
      a.idx[base + i] = -1;
      a.counts[base + i] = 0;
      if (a.weights) a.weights[base + i] = 0.0f;
    }
    if (a.total_steps) {
      const int steps = wave_sum_i32((int)my_steps);
      if (lane == 0 && steps) atomicAdd(a.total_steps, (unsigned long long)steps);
    }
    wave_lds_sync();
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
  const int64_t cap = 1ll << 22;
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
