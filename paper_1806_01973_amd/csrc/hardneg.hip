// Hard negative items on gfx950 (Sec. 3.3, "Hard negative items"): pins are
// ranked by their Personalized PageRank score with respect to the query,
// estimated by the visit counts of random walks from the query (the Sec. 3.2
// walks with their own seed), and items inside a rank window are drawn at
// random.
//
// One workgroup of 1024 threads owns one query at a time (grid-stride over
// queries); everything stays in LDS (about 2 x 4 B per visit slot):
//   1. walks: thread t runs walks t, t + 1024, ..., two at a time; walk w
//      writes its pin landings into slots [w*hops, (w+1)*hops); the rest of
//      the slots is empty;
//   2. the visit ids are sorted (bitonic network: a register sort per wave,
//      then merges across waves through LDS), so equal ids become runs;
//   3. runs become distinct pins with visit counts, numbered d in ascending
//      id order. Pins seen once rank last, in id order, so they go straight
//      to their rank positions; pins seen more than once (few) get the key
//      ((0xFFFF - count) << 16) | p, p their number among those pins;
//   4. sorting those keys ranks the repeated pins by count descending, then
//      id ascending, ahead of the single-visit pins;
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
#ifndef PINSAGE_HN_WALKERS
#define PINSAGE_HN_WALKERS 2
#endif
constexpr int kWalkers = PINSAGE_HN_WALKERS;  // walks in flight per thread

// LDS word of element i in a sort of kThreads * E keys: one pad word after
// every E elements, so that lanes storing or loading their E consecutive
// elements touch distinct banks.
template <int E>
__device__ __forceinline__ int padded(int i) {
  return i + i / E;
}

// Block-wide ascending sort of the N = kThreads * E keys at buf[0, N), taken
// in any order; buf must hold N + N / E words. On return, sorted element i is
// at buf[padded<E>(i)] and thread t holds elements [t*E, (t+1)*E) in k.
// Waves first sort their 64*E chunk in registers; each merge stage of size S
// starts with the "flip" compare of element i with i ^ (S - 1) (two ascending
// halves become two bitonic halves), continues with half-cleaners of stride
// >= one chunk through LDS and ends inside the waves.
template <int E>
__device__ __forceinline__ void block_sort(uint32_t* buf, uint32_t (&k)[E], int wave, int lane) {
  constexpr int N = kThreads * E;
  constexpr int kChunk = kWave * E;
  constexpr int kLgChunk = __builtin_ctz(kChunk);
  constexpr int kPairRounds = (N / 2 + kThreads - 1) / kThreads;
  const int tid = wave * kWave + lane;
  const int first = tid * E;
#pragma unroll
  for (int e = 0; e < E; ++e) k[e] = buf[e * kThreads + tid];
  __syncthreads();
  bitonic_sort_wave<E>(k, lane);
#pragma unroll 1
  for (int lg = kLgChunk + 1; (1 << lg) <= N; ++lg) {
    const int size = 1 << lg;
#pragma unroll
    for (int e = 0; e < E; ++e) buf[padded<E>(first + e)] = k[e];
    __syncthreads();
    // Flip pass over the N/2 pairs (i, i ^ (size - 1)), i in a lower half.
#pragma unroll
    for (int r = 0; r < kPairRounds; ++r) {
      const int p = r * kThreads + tid;
      if (p >= N / 2) break;
      const int i = ((p >> (lg - 1)) << lg) | (p & ((size >> 1) - 1));
      const int j = i ^ (size - 1);
      const uint32_t x = buf[padded<E>(i)], y = buf[padded<E>(j)];
      buf[padded<E>(i)] = x < y ? x : y;
      buf[padded<E>(j)] = x < y ? y : x;
    }
    __syncthreads();
#pragma unroll 1
    for (int ls = lg - 2; ls >= kLgChunk; --ls) {
#pragma unroll
      for (int r = 0; r < kPairRounds; ++r) {
        const int p = r * kThreads + tid;
        if (p >= N / 2) break;
        const int i = ((p >> ls) << (ls + 1)) | (p & ((1 << ls) - 1));
        const int j = i + (1 << ls);
        const uint32_t x = buf[padded<E>(i)], y = buf[padded<E>(j)];
        buf[padded<E>(i)] = x < y ? x : y;
        buf[padded<E>(j)] = x < y ? y : x;
      }
      __syncthreads();
    }
#pragma unroll
    for (int e = 0; e < E; ++e) k[e] = buf[padded<E>(first + e)];
    merge_wave_ascending<E>(k, lane);
  }
#pragma unroll
  for (int e = 0; e < E; ++e) buf[padded<E>(first + e)] = k[e];
  __syncthreads();
}

// Sorts the n <= kThreads * EMAX keys at buf[0, n) with the smallest sort that
// holds them (the caller pads up to 1024 * E with kEmpty, see sort_size);
// returns log2 of the chosen E (the layout of the result).
template <int EMAX>
__device__ __forceinline__ int block_sort_upto(uint32_t* buf, int n, int wave, int lane) {
  if (n <= kThreads || EMAX == 1) {
    uint32_t k[1];
    block_sort<1>(buf, k, wave, lane);
    return 0;
  }
  if constexpr (EMAX >= 2) {
    if (n <= 2 * kThreads || EMAX == 2) {
      uint32_t k[2];
      block_sort<2>(buf, k, wave, lane);
      return 1;
    }
  }
  if constexpr (EMAX >= 4) {
    if (n <= 4 * kThreads || EMAX == 4) {
      uint32_t k[4];
      block_sort<4>(buf, k, wave, lane);
      return 2;
    }
  }
  if constexpr (EMAX >= 8) {
    if (n <= 8 * kThreads || EMAX == 8) {
      uint32_t k[8];
      block_sort<8>(buf, k, wave, lane);
      return 3;
    }
  }
  if constexpr (EMAX >= 16) {
    uint32_t k[16];
    block_sort<16>(buf, k, wave, lane);
    return 4;
  }
  return 0;
}

__device__ __forceinline__ int sort_size(int n) {
  int s = kThreads;
  while (s < n) s <<= 1;
  return s;
}

// Exclusive prefix of v over the block in thread order; *total gets the sum.
// Contains barriers (every thread must call it).
__device__ __forceinline__ int block_exclusive_sum(int v, int wave, int lane, int* wave_tot,
                                                   int* total) {
  const int incl = wave_inclusive_sum(v, lane);
  if (lane == kWave - 1) wave_tot[wave] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int t = wave_tot[w];
    before += w < wave ? t : 0;
    all += t;
  }
  *total = all;
  __syncthreads();  // wave_tot is reused by the next call
  return before + incl - v;
}

template <typename OffT, int E>
__global__ __launch_bounds__(kThreads) void hard_negative_kernel(HardNegLaunch a) {
  constexpr int N = kThreads * E;
  __shared__ uint32_t keys[N + N / E];  // visits (sorted, padded), then head positions, rank keys
  __shared__ uint32_t ids[N];           // pins in rank order (repeated pins by number p)
  __shared__ int wave_tot[kWaves];
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const int WH = a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  uint32_t my_steps = 0;

  for (int64_t qi = blockIdx.x; qi < a.num_queries; qi += gridDim.x) {
    // The thread index passes through an opaque move each query, so values
    // derived from it (LDS addresses of every register slot) are recomputed
    // here instead of being hoisted out of the loop and spilled.
    int tid;
    asm volatile("v_mov_b32 %0, %1" : "=v"(tid) : "v"((int)threadIdx.x));
    const int wave = tid >> 6;
    const int lane = tid & (kWave - 1);
    const int64_t u = (int64_t)a.queries[qi];
    const bool live = u >= 0 && u < a.num_nodes;

    // ---- 1. walks ---------------------------------------------------------
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = e * kThreads + tid;
      if (slot >= WH || !live) keys[slot] = kEmpty;
    }
    if (live) {
      // kWalkers walks per thread in lockstep (w0, w0 + 1024, ...): their
      // dependent offset -> neighbour reads overlap.
      for (int w0 = tid; w0 < a.walks; w0 += kWalkers * kThreads) {
        Walker<OffT> W[kWalkers];
#pragma unroll
        for (int i = 0; i < kWalkers; ++i) {
          const int w = w0 + i * kThreads;
          W[i].start(u, w, keys + w * a.hops, w < a.walks);
        }
        bool any = true;
        while (any) {
          int64_t lo[kWalkers], hi[kWalkers];
#pragma unroll
          for (int i = 0; i < kWalkers; ++i) {
            lo[i] = 0;
            hi[i] = 0;
            if (W[i].active) {
              lo[i] = (int64_t)off[W[i].cur];
              hi[i] = (int64_t)off[W[i].cur + 1];
            }
          }
#pragma unroll
          for (int i = 0; i < kWalkers; ++i) W[i].pick(lo[i], hi[i], a.nnz, k0, k1);
          int32_t nx[kWalkers];
#pragma unroll
          for (int i = 0; i < kWalkers; ++i) nx[i] = W[i].active ? col[W[i].next_at] : 0;
          any = false;
#pragma unroll
          for (int i = 0; i < kWalkers; ++i) {
            W[i].land(nx[i], a.num_pins, a.num_nodes, a.hops);
            any = any || W[i].active;
          }
        }
#pragma unroll
        for (int i = 0; i < kWalkers; ++i) my_steps += W[i].finish(a.hops);
      }
    }
    __syncthreads();

    // ---- 2. sort visits by id ---------------------------------------------
    uint32_t k[E];
    block_sort<E>(keys, k, wave, lane);

    // ---- 3. runs -> distinct pins, counts, rank positions ------------------
    // Thread t holds sorted elements [t*E, (t+1)*E); a head opens a run, a
    // tail closes it. Heads are numbered d in order (block scan).
    const int first = tid * E;
    const uint32_t prev0 = first > 0 ? keys[padded<E>(first - 1)] : kEmpty;
    const uint32_t nextE = first + E < N ? keys[padded<E>(first + E)] : kEmpty;
    uint32_t head_bits = 0, tail_bits = 0;
    int nhead = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const uint32_t prev = e == 0 ? prev0 : k[e - 1];
      const uint32_t next = e == E - 1 ? nextE : k[e + 1];
      const bool head = k[e] != kEmpty && prev != k[e];
      const bool tail = k[e] != kEmpty && next != k[e];
      head_bits |= head ? 1u << e : 0u;
      tail_bits |= tail ? 1u << e : 0u;
      nhead += head ? 1 : 0;
    }
    int D = 0;
    const int d0 = block_exclusive_sum(nhead, wave, lane, wave_tot, &D);  // after all reads
    {
      int d = d0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (head_bits & (1u << e)) keys[d++] = (uint32_t)(first + e);  // head position of run d
      }
    }
    __syncthreads();
    // Tails: visit count of run d; repeated pins are counted for their number p.
    // Counts are at most N <= 2^14: two per register.
    constexpr int kPacked = (E + 1) / 2;
    uint32_t cnt2[kPacked];
#pragma unroll
    for (int i = 0; i < kPacked; ++i) cnt2[i] = 0u;
    int nmulti = 0;
    {
      int d = d0 - 1;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (head_bits & (1u << e)) ++d;
        const uint32_t c = (tail_bits & (1u << e)) ? (uint32_t)(first + e) - keys[d] + 1u : 0u;
        cnt2[e >> 1] |= c << (16 * (e & 1));
        nmulti += c > 1u ? 1 : 0;
      }
    }
    int Dm = 0;  // pins visited more than once
    const int p0 = block_exclusive_sum(nmulti, wave, lane, wave_tot, &Dm);  // after all reads
    {
      int d = d0 - 1, p = p0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        if (head_bits & (1u << e)) ++d;
        const uint32_t c = (cnt2[e >> 1] >> (16 * (e & 1))) & 0xFFFFu;
        if (c > 1u) {
          keys[p] = ((0xFFFFu - c) << 16) | (uint32_t)p;
          ids[p] = k[e];
          ++p;
        } else if (c == 1u) {
          ids[Dm + (d - p)] = k[e];  // d - p single-visit pins before this one
        }
      }
    }
    const int sort_n = Dm > 0 ? sort_size(Dm) : 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int slot = e * kThreads + tid;
      if (slot >= Dm && slot < sort_n) keys[slot] = kEmpty;
    }
    __syncthreads();

    // ---- 4. rank order of the repeated pins: count desc, then id asc -------
    int lg_sort = 0;
    if (Dm > 0) lg_sort = block_sort_upto<E>(keys, Dm, wave, lane);

    // ---- 5. draws from the window -----------------------------------------
    const int64_t top = D < a.rank_hi ? (int64_t)D : (int64_t)a.rank_hi;
    const int64_t n = top - a.rank_lo;
    int32_t* out = a.out + qi * (int64_t)a.k;
    for (int j = tid; j < a.k; j += kThreads) {
      int32_t v = -1;
      if (n > 0) {
        const uint4 r = philox4x32_10(make_uint4((uint32_t)u, (uint32_t)j, 0u, 1u), k0, k1);
        const int rank = a.rank_lo + (int)(((uint64_t)r.x * (uint64_t)n) >> 32);
        const uint32_t slot =
            rank < Dm ? (keys[rank + (rank >> lg_sort)] & 0xFFFFu) : (uint32_t)rank;
        v = (int32_t)ids[slot];
      }
      out[j] = v;
    }
    __syncthreads();  // keys / ids are rewritten for the next query
  }

  if (a.total_steps) {
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & (kWave - 1);
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
