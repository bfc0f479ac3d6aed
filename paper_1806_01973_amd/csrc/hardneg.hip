// Hard negative items on gfx950 (Sec. 3.3, "Hard negative items"): pins are
// ranked by their Personalized PageRank score with respect to the query,
// estimated by the visit counts of random walks from the query (the Sec. 3.2
// walks with their own seed), and items inside a rank window are drawn at
// random.
//
// One workgroup of 1024 threads owns one query at a time (grid-stride over
// queries); everything stays in LDS (2 x 4 B per visit slot):
//   1. walks: thread t runs walks t, t + 1024, ...; walk w writes its pin
//      landings into slots [w*hops, (w+1)*hops); the rest is empty;
//   2. the visit ids are sorted (bitonic network: a register sort per wave,
//      then merges across waves through LDS), so equal ids become runs;
//   3. run heads get a dense index d (their order among the heads, i.e.
//      ascending id), the id table gets ids[d], and each run's tail turns its
//      length into the rank key ((0xFFFF - count) << 16) | d;
//   4. sorting the rank keys orders the distinct pins by count descending,
//      then id ascending; position r of the sorted keys is rank r;
//   5. draw j: word 0 of Philox4x32-10 at counter (q, j, 0, 1) under the walk
//      key picks window position floor(r * n / 2^32), n = min(rank_hi, D) -
//      rank_lo for D distinct pins; an empty window writes -1.
#include "device_util.h"
#include "kernels.h"
#include "walk_device.h"

namespace pinsage {
namespace {

using namespace walkdev;

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

// The sort keeps element i of a wave's 64*E chunk in register e = i / 64 of
// lane i % 64, so that a wave's LDS accesses to its chunk are consecutive
// words (no bank conflicts).

// Compare-exchange of register e with the same register of lane (lane ^ M).
template <int M>
__device__ __forceinline__ uint32_t lane_cx(uint32_t v, int lane, bool take_min) {
  const uint32_t o = lane_xor<M>(v, lane);
  const uint32_t lo = v < o ? v : o;
  const uint32_t hi = v < o ? o : v;
  return take_min ? lo : hi;
}

template <int E>
__device__ __forceinline__ void lane_stage(uint32_t (&k)[E], int e, int stride, int lane,
                                           bool take_min) {
  switch (stride) {
    case 1: k[e] = lane_cx<1>(k[e], lane, take_min); break;
    case 2: k[e] = lane_cx<2>(k[e], lane, take_min); break;
    case 4: k[e] = lane_cx<4>(k[e], lane, take_min); break;
    case 8: k[e] = lane_cx<8>(k[e], lane, take_min); break;
    case 16: k[e] = lane_cx<16>(k[e], lane, take_min); break;
    default: k[e] = lane_cx<32>(k[e], lane, take_min); break;
  }
}

// Ascending bitonic sort of a wave's 64*E keys (element e*64 + lane).
template <int E>
__device__ __forceinline__ void sort_wave(uint32_t (&k)[E], int lane) {
#pragma unroll
  for (int size = 2; size <= kWave * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= kWave) {
        const int es = stride / kWave;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & es) == 0) {
            const bool up = ((e * kWave) & size) == 0;
            const uint32_t x = k[e], y = k[e + es];
            const uint32_t lo = x < y ? x : y;
            const uint32_t hi = x < y ? y : x;
            k[e] = up ? lo : hi;
            k[e + es] = up ? hi : lo;
          }
        }
      } else {
        const bool lower = (lane & stride) == 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const bool up = (((e * kWave) | lane) & size) == 0;
          lane_stage<E>(k, e, stride, lane, up == lower);
        }
      }
    }
  }
}

// Ascending half-cleaners of strides 32E .. 1 over a wave's chunk: sorts a
// bitonic chunk.
template <int E>
__device__ __forceinline__ void merge_wave(uint32_t (&k)[E], int lane) {
#pragma unroll
  for (int stride = kWave * E / 2; stride > 0; stride >>= 1) {
    if (stride >= kWave) {
      const int es = stride / kWave;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if ((e & es) == 0) {
          const uint32_t x = k[e], y = k[e + es];
          k[e] = x < y ? x : y;
          k[e + es] = x < y ? y : x;
        }
      }
    } else {
      const bool lower = (lane & stride) == 0;
#pragma unroll
      for (int e = 0; e < E; ++e) lane_stage<E>(k, e, stride, lane, lower);
    }
  }
}

// Block-wide ascending sort of the N = kThreads * E keys in `buf`. On return
// buf holds the sorted keys and each thread holds its own elements (chunk of
// wave w: [w*64E, (w+1)*64E), element e*64 + lane) in k. Waves first sort
// their chunk in registers; each merge stage of size S starts with the "flip"
// compare of element i with i ^ (S - 1) (two ascending halves become two
// bitonic halves), continues with half-cleaners of stride >= one chunk
// through LDS and ends inside the waves.
template <int E>
__device__ __forceinline__ void block_sort(uint32_t* buf, uint32_t (&k)[E], int wave, int lane) {
  constexpr int N = kThreads * E;
  constexpr int kChunk = kWave * E;
  constexpr int kLgChunk = __builtin_ctz(kChunk);
  const int tid = wave * kWave + lane;
  uint32_t* mine = buf + wave * kChunk + lane;
#pragma unroll
  for (int e = 0; e < E; ++e) k[e] = mine[e * kWave];
  sort_wave<E>(k, lane);
#pragma unroll 1
  for (int lg = kLgChunk + 1; (1 << lg) <= N; ++lg) {
    const int size = 1 << lg;
#pragma unroll
    for (int e = 0; e < E; ++e) mine[e * kWave] = k[e];
    __syncthreads();
    // Flip pass over the N/2 pairs (i, i ^ (size - 1)), i in a lower half.
#pragma unroll
    for (int p = tid; p < N / 2; p += kThreads) {
      const int i = ((p >> (lg - 1)) << lg) | (p & ((size >> 1) - 1));
      const int j = i ^ (size - 1);
      const uint32_t x = buf[i], y = buf[j];
      buf[i] = x < y ? x : y;
      buf[j] = x < y ? y : x;
    }
    __syncthreads();
#pragma unroll 1
    for (int ls = lg - 2; ls >= kLgChunk; --ls) {
#pragma unroll
      for (int p = tid; p < N / 2; p += kThreads) {
        const int i = ((p >> ls) << (ls + 1)) | (p & ((1 << ls) - 1));
        const uint32_t x = buf[i], y = buf[i + (1 << ls)];
        buf[i] = x < y ? x : y;
        buf[i + (1 << ls)] = x < y ? y : x;
      }
      __syncthreads();
    }
#pragma unroll
    for (int e = 0; e < E; ++e) k[e] = mine[e * kWave];
    merge_wave<E>(k, lane);
  }
#pragma unroll
  for (int e = 0; e < E; ++e) mine[e * kWave] = k[e];
  __syncthreads();
}

template <typename OffT, int E>
__global__ __launch_bounds__(kThreads) void hard_negative_kernel(HardNegLaunch a) {
  constexpr int N = kThreads * E;
  constexpr int kChunk = kWave * E;
  __shared__ uint32_t keys[N];  // visit ids, then head positions / rank keys
  __shared__ uint32_t ids[N];   // distinct ids in ascending order
  __shared__ int wave_tot[kWaves];
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & (kWave - 1);
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const int WH = a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  uint32_t my_steps = 0;

  for (int64_t qi = blockIdx.x; qi < a.num_queries; qi += gridDim.x) {
    const int64_t u = (int64_t)a.queries[qi];
    const bool live = u >= 0 && u < a.num_nodes;

    // ---- 1. walks ---------------------------------------------------------
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = e * kThreads + tid;
      if (slot >= WH || !live) keys[slot] = kEmpty;
    }
    if (live) {
      for (int w0 = tid; w0 < a.walks; w0 += 2 * kThreads) {
        Walker<OffT> A, B;
        A.start(u, w0, keys + w0 * a.hops, true);
        B.start(u, w0 + kThreads, keys + (w0 + kThreads) * a.hops, w0 + kThreads < a.walks);
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
    __syncthreads();

    // ---- 2. sort visits by id ---------------------------------------------
    uint32_t k[E];
    block_sort<E>(keys, k, wave, lane);

    // ---- 3. distinct ids, their counts, rank keys --------------------------
    // Heads and tails of the runs; a head's dense index d counts the heads
    // before it in sorted order (ballots per register, then the waves before).
    const int base = wave * kChunk + lane;
    uint32_t head_bits = 0, tail_bits = 0;
    uint64_t hm[E];
    int wave_heads = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = base + e * kWave;
      const uint32_t prev = i > 0 ? keys[i - 1] : kEmpty;
      const uint32_t next = i + 1 < N ? keys[i + 1] : kEmpty;
      const bool head = k[e] != kEmpty && prev != k[e];
      const bool tail = k[e] != kEmpty && next != k[e];
      head_bits |= head ? 1u << e : 0u;
      tail_bits |= tail ? 1u << e : 0u;
      hm[e] = __ballot(head);
      wave_heads += __popcll(hm[e]);
    }
    if (lane == 0) wave_tot[wave] = wave_heads;
    __syncthreads();  // also: every read of the sorted ids is done
    int D = 0, before = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int t = wave_tot[w];
      before += w < wave ? t : 0;
      D += t;
    }
    const uint64_t below = (1ull << lane) - 1ull;  // lanes under this one
    // Heads: id table and head position.
    {
      int d = before;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (head_bits & (1u << e)) {
          const int dh = d + __popcll(hm[e] & below);
          ids[dh] = k[e];
          keys[dh] = (uint32_t)(base + e * kWave);
        }
        d += __popcll(hm[e]);
      }
    }
    __syncthreads();
    // Tails: run length -> rank key in place of the head position. The run
    // of a tail is the last head at or before it.
    {
      int d = before;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int dt = d + __popcll(hm[e] & (below | (1ull << lane))) - 1;
        if (tail_bits & (1u << e)) {
          const uint32_t count = (uint32_t)(base + e * kWave) - keys[dt] + 1u;
          keys[dt] = ((0xFFFFu - count) << 16) | (uint32_t)dt;
        }
        d += __popcll(hm[e]);
      }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = e * kThreads + tid;
      if (slot >= D) keys[slot] = kEmpty;
    }
    __syncthreads();

    // ---- 4. rank order: count descending, then id ascending ---------------
    block_sort<E>(keys, k, wave, lane);

    // ---- 5. draws from the window -----------------------------------------
    const int64_t top = D < a.rank_hi ? (int64_t)D : (int64_t)a.rank_hi;
    const int64_t n = top - a.rank_lo;
    int32_t* out = a.out + qi * (int64_t)a.k;
    for (int j = tid; j < a.k; j += kThreads) {
      int32_t v = -1;
      if (n > 0) {
        const uint4 r = philox4x32_10(make_uint4((uint32_t)u, (uint32_t)j, 0u, 1u), k0, k1);
        const int64_t pos = (int64_t)(((uint64_t)r.x * (uint64_t)n) >> 32);
        v = (int32_t)ids[keys[a.rank_lo + pos] & 0xFFFFu];
      }
      out[j] = v;
    }
    __syncthreads();  // keys / ids are rewritten for the next query
  }

  if (a.total_steps) {
    const int ws = wave_sum_i32((int)my_steps);
    if (lane == 0) wave_tot[wave] = ws;
    __syncthreads();
    if (tid == 0) {
      unsigned long long t = 0;
      for (int w = 0; w < kWaves; ++w) t += (unsigned long long)(unsigned)wave_tot[w];
      if (t) atomicAdd(a.total_steps, t);
    }
  }
}

template <typename OffT>
hipError_t launch_for_offsets(const HardNegLaunch& a, hipStream_t s) {
  const int wh = a.walks * a.hops;
  const int64_t cap = 1ll << 13;
  const dim3 grid((unsigned)(a.num_queries < cap ? a.num_queries : cap));
  const dim3 block(kThreads);
  if (wh <= 1 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 1>), grid, block, 0, s, a);
  else if (wh <= 2 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 2>), grid, block, 0, s, a);
  else if (wh <= 4 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 4>), grid, block, 0, s, a);
  else if (wh <= 8 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 8>), grid, block, 0, s, a);
  else if (wh <= 16 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 16>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_hard_negatives(const HardNegLaunch& a, hipStream_t s) {
  if (a.num_queries <= 0) return hipSuccess;
  ProfileScope prof(kKHardNeg, s);
  return a.offsets64 ? launch_for_offsets<int64_t>(a, s) : launch_for_offsets<int32_t>(a, s);
}

}  // namespace pinsage
