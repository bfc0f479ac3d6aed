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

// MurmurHash3's 32-bit finaliser (a bijection with good avalanche).
__device__ __forceinline__ uint32_t fmix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x85ebca6bu;
  x ^= x >> 13;
  x *= 0xc2b2ae35u;
  x ^= x >> 16;
  return x;
}
// Partition of a pin among `parts` (the global path's buckets).
__device__ __forceinline__ uint32_t part_of(uint32_t v, uint32_t parts) {
  return (uint32_t)(((uint64_t)fmix32(v) * parts) >> 32);
}

constexpr int kCPerPart = 8192;  // landings per hash partition (on average at most)
constexpr int kCCap = 12288;     // bucket capacity of a partition in the workspace

// The walks of query u (Sec. 3.2, as the neighbourhood walks): kWalkers walks
// per thread in lockstep (w0, w0 + 1024, ...), so their dependent reads
// overlap; walk w's pin landings go to slots[w * hops ..]. TABLE: each edge
// step reads one 16-byte walk-table entry (the neighbour's id, degree and row
// start) instead of the current node's offsets and then a neighbour id; the
// source's row comes from its offsets, validated as pick() validates a row.
// Returns this thread's edge steps.
// BUCKET (the global path): a landing is not written to slots; a recorded one
// (a pin p other than u) goes straight to its hash partition's bucket,
// bk.buckets[part * kCCap + n] with n from that partition's LDS cursor, or,
// once the bucket holds kCCap, to the overflow list (its own LDS cursor).
struct Buckets {
  uint32_t* cursor;   // LDS [parts], zeroed
  uint32_t parts;
  uint32_t* buckets;  // [parts][kCCap]
  uint32_t* ovf;      // >= walks * hops words
  int* ovf_n;         // LDS, zeroed
};
__device__ __forceinline__ void bucket_append(const Buckets& bk, uint32_t v) {
  if (v == kEmpty) return;  // the query itself
  const uint32_t p = part_of(v, bk.parts);
  const uint32_t n = atomicAdd(&bk.cursor[p], 1u);
  if (n < (uint32_t)kCCap) bk.buckets[(int64_t)p * kCCap + n] = v;
  else bk.ovf[atomicAdd(bk.ovf_n, 1)] = v;
}
template <typename OffT, bool TABLE, bool BUCKET = false>
__device__ __forceinline__ uint32_t walk_query(const HardNegLaunch& a, int64_t u, int tid,
                                               uint32_t* slots, uint32_t k0, uint32_t k1,
                                               const Buckets& bk = Buckets{}) {
  const OffT* __restrict__ off = static_cast<const OffT*>(a.row_offsets);
  const int32_t* __restrict__ col = a.col;
  const uint4* __restrict__ tab = static_cast<const uint4*>(a.table);
  int64_t ulo = 0;
  int32_t udeg = 0;
  if constexpr (TABLE) {
    const int64_t lo = (int64_t)off[u], hi = (int64_t)off[u + 1];
    if (!(hi - lo <= 0 || lo < 0 || hi > a.nnz)) {
      ulo = lo;
      udeg = (int32_t)(hi - lo);
    }
  }
  uint32_t steps = 0;
  for (int w0 = tid; w0 < a.walks; w0 += kWalkers * kThreads) {
    Walker<OffT> W[kWalkers];
#pragma unroll
    for (int i = 0; i < kWalkers; ++i) {
      const int w = w0 + i * kThreads;
      W[i].start(u, w, slots + (int64_t)w * a.hops, w < a.walks);
      W[i].lo = ulo;
      W[i].deg = udeg;
    }
    bool any = true;
    while (any) {
      if constexpr (TABLE) {
#pragma unroll
        for (int i = 0; i < kWalkers; ++i) W[i].pick_carried(k0, k1);
        uint4 e[kWalkers];
#pragma unroll
        for (int i = 0; i < kWalkers; ++i)
          e[i] = W[i].active ? tab[W[i].next_at] : make_uint4(0u, 0u, 0u, 0u);
        any = false;
#pragma unroll
        for (int i = 0; i < kWalkers; ++i) {
          if constexpr (BUCKET) {
            // land_entry without the slot write.
            uint32_t v;
            if (W[i].advance((int32_t)e[i].x, a.num_pins, a.num_nodes, a.hops, &v))
              bucket_append(bk, v);
            W[i].deg = (int32_t)e[i].y;
            W[i].lo = (int64_t)(((uint64_t)e[i].w << 32) | (uint64_t)e[i].z);
          } else {
            W[i].land_entry(e[i], a.num_pins, a.num_nodes, a.hops);
          }
          any = any || W[i].active;
        }
      } else {
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
          if constexpr (BUCKET) {
            uint32_t v;
            if (W[i].advance(nx[i], a.num_pins, a.num_nodes, a.hops, &v)) bucket_append(bk, v);
          } else {
            W[i].land(nx[i], a.num_pins, a.num_nodes, a.hops);
          }
          any = any || W[i].active;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kWalkers; ++i) {
      if constexpr (BUCKET) steps += W[i].exists ? (uint32_t)W[i].s : 0u;  // no slots to pad
      else steps += W[i].finish(a.hops);
    }
  }
  return steps;
}

template <typename OffT, int E, bool TABLE>
__global__ __launch_bounds__(kThreads) void hard_negative_kernel(HardNegLaunch a) {
  constexpr int N = kThreads * E;
  __shared__ uint32_t keys[N + N / E];  // visits (sorted, padded), then head positions, rank keys
  __shared__ uint32_t ids[N];           // pins in rank order (repeated pins by number p)
  __shared__ int wave_tot[kWaves];
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
    if (live) my_steps += walk_query<OffT, TABLE>(a, u, tid, keys, k0, k1);
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

// ---------------------------------------------------------------------------
// Walk budgets above the LDS slots (walks * hops > 16384). One 1024-thread
// workgroup per query (grid-stride; each workgroup reuses its own workspace):
//   W. each recorded landing (a pin other than the query) goes straight to the
//      bucket of its hash partition in the workspace, at the slot the
//      partition's LDS cursor hands out (the walks wait on memory, the LDS
//      atomics cost them nothing measurable); a partition holds about 8,192
//      landings, and those past a full bucket (12,288) go to an overflow list;
//   B. the overflow list, if any, is bucketed by partition (a histogram sweep
//      and a scatter sweep, one LDS atomic per distinct partition of a wave);
//   C. each partition (its bucket, then its overflow landings) is counted in
//      an LDS table (12,288 slots: at most two thirds full at the average
//      partition size when every landing is a distinct pin), and its (pin, count) pairs
//      are appended to a compact list; a
//      pin that finds no slot within 64 linear probes marks its partition as
//      overflowing, which is then split in two by a second hash and counted
//      again (and so on: a part with fewer than 64 pins cannot overflow), so
//      every count is exact;
// then, as only the first rank_hi ranks matter, a selection over the list:
//   1. count histogram (12-bit digits, two passes) -> the count c* of rank
//      rank_hi - 1, the number n_above of pins counted more than c*;
//   2. the pins counted more than c* (fewer than rank_hi) sorted by count
//      descending, id ascending (64-bit keys, bitonic in LDS);
//   3. the rank_hi - n_above smallest ids counted exactly c*: radix select on
//      the id (11 + 10 + 10 bits), gathered and sorted ascending;
//   4. the draws as in the on-chip kernel.
// With at most rank_hi distinct pins, all of them take step 2. The list's
// order depends on the atomics' order, the selection's results do not.
// ---------------------------------------------------------------------------
constexpr int kGMaxRank = 8192;  // rank_hi limit of this path
constexpr int kGBins = 4096;
constexpr uint32_t kNoKey = 0xFFFFFFFFu;
constexpr int kCSlots = 12288;   // LDS counting table: keys then counts (96 KB)
constexpr int kCProbes = 64;     // linear probes before a partition counts as overflowing
constexpr int kMaxParts = 512;   // partitions of the largest budget (2^22 landings)
static_assert(kCSlots % kThreads == 0, "whole waves sweep the table");
static_assert(2 * kCSlots * 4 >= kGMaxRank * 8 + kGMaxRank * 4, "top and cls fit the table");

// Its half in a split of `split` (a power of two) and its home slot in the
// LDS table: two more hashes of the id, unrelated to part_of's.
__device__ __forceinline__ uint32_t split_of(uint32_t v, uint32_t split) {
  return fmix32(v ^ 0x9e3779b9u) & (split - 1);
}
__device__ __forceinline__ uint32_t home_of(uint32_t v) {
  return (uint32_t)(((uint64_t)fmix32(v + 0x7f4a7c15u) * kCSlots) >> 32);
}

// hist[bin] += 1 for every lane with `on`: one LDS atomic per distinct bin of
// the wave (the lanes sharing the lowest pending lane's bin are added at once).
// Count histograms put most pins in a few bins, where per-lane atomics would
// serialise. Called by whole waves.
__device__ __forceinline__ void wave_hist_add(uint32_t* hist, uint32_t bin, bool on) {
  const int lane = threadIdx.x & (kWave - 1);
  uint64_t pending = __ballot(on);
  while (pending) {
    const int leader = __builtin_ctzll(pending);
    const uint32_t b = __shfl(bin, leader);
    const uint64_t same = __ballot(((pending >> lane) & 1ull) && bin == b) & pending;
    if (lane == leader) atomicAdd(&hist[b], (uint32_t)__builtin_popcountll(same));
    pending &= ~same;
  }
}

// Slot in bucket `bin` (cursor[bin] counts the bucket's entries so far) for
// every lane with `on`: one LDS atomic per distinct bin of the wave, the lanes
// of a bin taking consecutive slots in lane order. Called by whole waves.
__device__ __forceinline__ uint32_t wave_bucket_slot(uint32_t* cursor, uint32_t bin, bool on) {
  const int lane = threadIdx.x & (kWave - 1);
  uint64_t pending = __ballot(on);
  uint32_t slot = 0;
  while (pending) {
    const int leader = __builtin_ctzll(pending);
    const uint32_t b = __shfl(bin, leader);
    const uint64_t same = __ballot(((pending >> lane) & 1ull) && bin == b) & pending;
    uint32_t base = 0;
    if (lane == leader) base = atomicAdd(&cursor[b], (uint32_t)__builtin_popcountll(same));
    base = __shfl(base, leader);
    if ((same >> lane) & 1ull)
      slot = base + (uint32_t)__builtin_popcountll(same & ((1ull << lane) - 1ull));
    pending &= ~same;
  }
  return slot;
}

// Ascending bitonic sort of v[0, n), n a power of two <= 2 * 1024 * 4.
template <typename T>
__device__ __forceinline__ void lds_bitonic(T* v, int n, int tid) {
  for (int size = 2; size <= n; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = tid; p < n / 2; p += kThreads) {
        const int i = 2 * stride * (p / stride) + (p % stride);
        const int j = i + stride;
        const bool up = (i & size) == 0;
        const T x = v[i], y = v[j];
        if ((x > y) == up) {
          v[i] = y;
          v[j] = x;
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ int pow2_at_least(int n) {
  int p = 1;
  while (p < n) p <<= 1;
  return p;
}

// Scans hist[0, kGBins) from the top for the bin holding the want-th largest
// element (0-based) and the number of elements in the bins above it; bin 0
// (with every element above it) when no bin above 0 holds it. The whole block
// calls it (it contains barriers): thread t takes bins kGBins - 1 - 4 t - j,
// j < 4, a block scan gives the elements above each thread's four, and the
// thread holding the bin where the running count passes `want` writes the
// result to *bin and *above (shared).
static_assert(kGBins == 4 * kThreads, "four count bins per thread");
__device__ __forceinline__ void top_bin_block(const uint32_t* hist, int64_t want, int tid,
                                              int* wave_tot, int* bin, int64_t* above) {
  const int wave = tid >> 6, lane = tid & (kWave - 1);
  int c[4], sum = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    c[j] = (int)hist[kGBins - 1 - 4 * tid - j];
    sum += c[j];
  }
  int total;
  int64_t cum = block_exclusive_sum(sum, wave, lane, wave_tot, &total);
  if (tid == 0) {
    *bin = 0;
    *above = (int64_t)total - (int64_t)hist[0];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int b = kGBins - 1 - 4 * tid - j;
    if (b >= 1 && cum <= want && cum + c[j] > want) {
      *bin = b;
      *above = cum;
    }
    cum += c[j];
  }
  __syncthreads();
}

// From the bottom: the bin of hist[0, nbins) holding the want-th smallest
// element (0-based) and the number of elements below it; bin nbins - 1 (with
// every element below it) when no lower bin holds it. The bins from nbins to
// kGBins must be zero. The whole block calls it (it contains barriers):
// thread t takes bins 4 t + j, j < 4, and the thread holding the bin where
// the running count passes `want` writes the result (shared).
__device__ __forceinline__ void low_bin_block(const uint32_t* hist, int nbins, int64_t want,
                                              int tid, int* wave_tot, int* bin,
                                              int64_t* below) {
  const int wave = tid >> 6, lane = tid & (kWave - 1);
  int c[4], sum = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    c[j] = (int)hist[4 * tid + j];
    sum += c[j];
  }
  int total;
  int64_t cum = block_exclusive_sum(sum, wave, lane, wave_tot, &total);
  if (tid == 0) {
    *bin = nbins - 1;
    *below = (int64_t)total - (int64_t)hist[nbins - 1];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int b = 4 * tid + j;
    if (b < nbins - 1 && cum <= want && cum + c[j] > want) {
      *bin = b;
      *below = cum;
    }
    cum += c[j];
  }
  __syncthreads();
}

template <typename OffT, bool TABLE>
__global__ __launch_bounds__(kThreads) void hard_negative_global_kernel(HardNegLaunch a,
                                                                        uint32_t* ws,
                                                                        int64_t ws_words) {
  __shared__ uint32_t hist[kGBins];
  // The counting table during step C; then top (pins counted more than c*:
  // (~count << 32) | id) and cls (the smallest ids counted exactly c*).
  __shared__ __attribute__((aligned(16))) uint32_t pool[2 * kCSlots];
  __shared__ int64_t sh_i64[4];
  __shared__ int sh_i32[8];
  uint32_t* lkeys = pool;
  uint32_t* lcnt = pool + kCSlots;
  uint64_t* top = reinterpret_cast<uint64_t*>(pool);
  uint32_t* cls = pool + 2 * kGMaxRank;
  const int64_t L = (int64_t)a.walks * a.hops;
  const uint32_t k0 = (uint32_t)(a.seed & 0xFFFFFFFFull);
  const uint32_t k1 = (uint32_t)(a.seed >> 32);
  const int tid = threadIdx.x;
  const int R = a.rank_hi;
  const uint32_t parts = (uint32_t)((L + kCPerPart - 1) / kCPerPart);  // <= kMaxParts
  // This workgroup's workspace: the partitions' buckets, the overflow list,
  // the overflow list by partition, and the (pin, count) list.
  uint32_t* buckets = ws + (int64_t)blockIdx.x * ws_words;  // [parts][kCCap]
  uint32_t* ovf = buckets + (int64_t)parts * kCCap;          // up to L landings
  uint32_t* ovf_sorted = ovf + L;                           // the same, by partition
  uint32_t* list = ovf_sorted + L;                          // up to L (pin, count) pairs
  __shared__ int scan_tot[kWaves];            // top_bin_block's wave sums
  __shared__ uint32_t pstart[kMaxParts + 1];  // overflow landings by partition
  __shared__ uint32_t pcount[kMaxParts];      // landings in each partition's bucket
  uint32_t my_steps = 0;

  for (int64_t qi = blockIdx.x; qi < a.num_queries; qi += gridDim.x) {
    const int64_t u = (int64_t)a.queries[qi];
    const bool live = u >= 0 && u < a.num_nodes;
    if (tid < 8) sh_i32[tid] = 0;
    for (uint32_t b = tid; b < parts; b += kThreads) hist[b] = 0u;
    __syncthreads();

    // ---- W. walks, landings into their partitions' buckets -----------------
    if (live) {
      const Buckets bk{hist, parts, buckets, ovf, &sh_i32[7]};
      // (The walkers' slots are never written in this mode.)
      my_steps += walk_query<OffT, TABLE, true>(a, u, tid, ovf, k0, k1, bk);
    }
    __syncthreads();
    // The buckets were written through L2 by other waves: drop this CU's
    // cached lines of them before reading.
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    for (uint32_t p = tid; p < parts; p += kThreads)
      pcount[p] = hist[p] < (uint32_t)kCCap ? hist[p] : (uint32_t)kCCap;
    const int n_ovf = sh_i32[7];
    __syncthreads();

    // ---- B. the overflow (landings past a full bucket) by partition --------
    // Rare (a partition far above its average, as when a few pins take most
    // landings): a histogram sweep and a scatter sweep of the list.
    if (n_ovf > 0) {
      const int64_t nr = ((int64_t)n_ovf + kThreads - 1) / kThreads * kThreads;
      for (uint32_t b = tid; b < parts; b += kThreads) hist[b] = 0u;
      __syncthreads();
      for (int64_t i = tid; i < nr; i += kThreads) {
        const uint32_t v = i < n_ovf ? ovf[i] : kEmpty;
        wave_hist_add(hist, v == kEmpty ? 0u : part_of(v, parts), v != kEmpty);
      }
      __syncthreads();
      if (tid == 0) {
        uint32_t run = 0;
        for (uint32_t p = 0; p < parts; ++p) {
          pstart[p] = run;
          run += hist[p];
          hist[p] = pstart[p];  // the partition's cursor
        }
        pstart[parts] = run;
      }
      __syncthreads();
      for (int64_t i = tid; i < nr; i += kThreads) {
        const uint32_t v = i < n_ovf ? ovf[i] : kEmpty;
        const uint32_t b = v == kEmpty ? 0u : part_of(v, parts);
        const uint32_t slot = wave_bucket_slot(hist, b, v != kEmpty);
        if (v != kEmpty) ovf_sorted[slot] = v;
      }
    } else {
      for (uint32_t p = tid; p <= parts; p += kThreads) pstart[p] = 0u;
    }
    __syncthreads();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    // From here hist[c] counts the listed pins of count c < kGBins and
    // sh_i32[6] those of larger counts, filled as the pairs are emitted.
    for (int b = tid; b < kGBins; b += kThreads) hist[b] = 0u;
    if (tid == 0) sh_i32[6] = 0;
    __syncthreads();

    // ---- C. count each partition's landings in LDS ---------------------------
    // Partition p: its bucket, then its overflow landings.
    for (uint32_t p = 0; p < parts; ++p) {
      const int list0 = sh_i32[0];
      const uint32_t* bkt = buckets + (int64_t)p * kCCap;
      const int64_t n1 = pcount[p];
      const int64_t o0 = pstart[p], n = n1 + (pstart[p + 1] - o0);
      uint32_t split = 1;
      for (uint32_t sp = 0; sp < split;) {
        for (int i = tid; i < kCSlots; i += kThreads) {
          lkeys[i] = kNoKey;
          lcnt[i] = 0u;
        }
        if (tid == 0) sh_i32[1] = 0;
        __syncthreads();
        for (int64_t i = tid; i < n; i += kThreads) {
          const uint32_t v = i < n1 ? bkt[i] : ovf_sorted[o0 + (i - n1)];
          if (split_of(v, split) != sp) continue;
          uint32_t h = home_of(v);
          bool placed = false;
          for (int probe = 0; probe < kCProbes; ++probe) {
            const uint32_t k = atomicCAS(&lkeys[h], kNoKey, v);
            if (k == kNoKey || k == v) {
              atomicAdd(&lcnt[h], 1u);
              placed = true;
              break;
            }
            h = h + 1 == (uint32_t)kCSlots ? 0u : h + 1;
          }
          if (!placed) sh_i32[1] = 1;  // overflow: split the partition
        }
        __syncthreads();
        if (sh_i32[1]) {
          // Too crowded: split further, count the partition again from its
          // first part, and take the parts listed so far back out of the
          // count histogram (rare).
          split *= 2;
          sp = 0;
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
          for (int i = list0 + tid; i < sh_i32[0]; i += kThreads) {
            const uint32_t c = list[2 * (int64_t)i + 1];
            if (c < (uint32_t)kGBins) atomicSub(&hist[c], 1u);
            else atomicSub(&sh_i32[6], 1);
          }
          __syncthreads();
          if (tid == 0) sh_i32[0] = list0;
          __syncthreads();
          continue;
        }
        for (int i = tid; i < kCSlots; i += kThreads) {
          const uint32_t k = lkeys[i];
          const uint32_t c = lcnt[i];
          if (k != kNoKey) {
            const int pos = atomicAdd(&sh_i32[0], 1);
            list[2 * (int64_t)pos] = k;
            list[2 * (int64_t)pos + 1] = c;
            if (c >= (uint32_t)kGBins) atomicAdd(&sh_i32[6], 1);
          }
          wave_hist_add(hist, c < (uint32_t)kGBins ? c : 0u, k != kNoKey && c < (uint32_t)kGBins);
        }
        __syncthreads();
        ++sp;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const int D = sh_i32[0];
    const int Dr = (D + kThreads - 1) / kThreads * kThreads;  // whole waves sweep the list

    // ---- 1. count threshold ----------------------------------------------
    // Usually rank rank_hi - 1 falls among counts below kGBins, whose
    // histogram the listing filled: c* and n_above come from it directly.
    // Otherwise (at least rank_hi pins counted kGBins or more) two passes over
    // the list histogram the count's high and low 12 bits.
    uint32_t cstar = 0;  // pins counted more than cstar are ranked by step 2
    int64_t n_above = D;
    const int n_big = sh_i32[6];
    if (D > R && n_big < R) {
      top_bin_block(hist, R - 1 - n_big, tid, scan_tot, &sh_i32[1], &sh_i64[0]);
      cstar = (uint32_t)sh_i32[1];
      n_above = n_big + sh_i64[0];
    } else if (D > R) {
      __syncthreads();  // every wave has read n_big before hist is cleared
      for (int b = tid; b < kGBins; b += kThreads) hist[b] = 0u;
      __syncthreads();
      for (int i = tid; i < Dr; i += kThreads) {
        const bool on = i < D;
        const uint32_t c = on ? list[2 * (int64_t)i + 1] : 0u;
        wave_hist_add(hist, (c >> 12) < kGBins ? (c >> 12) : kGBins - 1, on);
      }
      __syncthreads();
      top_bin_block(hist, R - 1, tid, scan_tot, &sh_i32[1], &sh_i64[0]);
      const uint32_t b1 = (uint32_t)sh_i32[1];
      const int64_t above1 = sh_i64[0];
      for (int b = tid; b < kGBins; b += kThreads) hist[b] = 0u;
      __syncthreads();
      for (int i = tid; i < Dr; i += kThreads) {
        const bool in = i < D;
        const uint32_t c = in ? list[2 * (int64_t)i + 1] : 0u;
        wave_hist_add(hist, c & (kGBins - 1), in && (c >> 12) == b1);
      }
      __syncthreads();
      top_bin_block(hist, R - 1 - above1, tid, scan_tot, &sh_i32[2], &sh_i64[1]);
      cstar = (b1 << 12) | (uint32_t)sh_i32[2];
      n_above = above1 + sh_i64[1];
    }

    // ---- 2. pins counted more than c*, by count desc, id asc ---------------
    for (int i = tid; i < D; i += kThreads) {
      const uint32_t c = list[2 * (int64_t)i + 1];
      if (c > cstar) {
        const int slot = atomicAdd(&sh_i32[3], 1);
        top[slot] = ((uint64_t)(~c) << 32) | list[2 * (int64_t)i];
      }
    }
    __syncthreads();
    const int na = (int)n_above;
    const int na2 = pow2_at_least(na > 0 ? na : 1);
    for (int i = na + tid; i < na2; i += kThreads) top[i] = ~0ull;
    __syncthreads();
    if (na > 1) lds_bitonic<uint64_t>(top, na2, tid);

    // ---- 3. the smallest ids counted exactly c* ---------------------------
    const int need = D > R ? R - na : 0;
    if (need > 0) {
      // Radix select of the need-th smallest id (0-based need - 1) among the
      // pins counted c*: digits of 11, 10 and 10 bits.
      uint32_t prefix = 0;
      int64_t want = need - 1;
      constexpr int shifts[3] = {20, 10, 0};
      constexpr int widths[3] = {11, 10, 10};
#pragma unroll
      for (int pass = 0; pass < 3; ++pass) {
        const int sft = shifts[pass], nb = 1 << widths[pass];
        const uint32_t hi_mask = pass == 0 ? 0u : (0xFFFFFFFFu << (sft + widths[pass]));
        for (int b = tid; b < kGBins; b += kThreads) hist[b] = 0u;
        __syncthreads();
        for (int i = tid; i < D; i += kThreads) {
          const uint32_t k = list[2 * (int64_t)i];
          if (list[2 * (int64_t)i + 1] != cstar || (k & hi_mask) != prefix) continue;
          atomicAdd(&hist[(k >> sft) & (nb - 1)], 1u);
        }
        __syncthreads();
        low_bin_block(hist, nb, want, tid, scan_tot, &sh_i32[4], &sh_i64[2]);
        prefix |= (uint32_t)sh_i32[4] << sft;
        want -= sh_i64[2];
        __syncthreads();
      }
      // prefix is the need-th smallest id of the class: gather ids <= prefix.
      for (int i = tid; i < D; i += kThreads) {
        const uint32_t k = list[2 * (int64_t)i];
        if (list[2 * (int64_t)i + 1] != cstar || k > prefix) continue;
        cls[atomicAdd(&sh_i32[5], 1)] = k;
      }
      __syncthreads();
      const int nc2 = pow2_at_least(need);
      for (int i = need + tid; i < nc2; i += kThreads) cls[i] = kNoKey;
      __syncthreads();
      if (need > 1) lds_bitonic<uint32_t>(cls, nc2, tid);
    }

    // ---- 4. draws from the window -----------------------------------------
    const int64_t topn = D < R ? (int64_t)D : (int64_t)R;
    const int64_t n = topn - a.rank_lo;
    int32_t* outq = a.out + qi * (int64_t)a.k;
    for (int j = tid; j < a.k; j += kThreads) {
      int32_t v = -1;
      if (n > 0) {
        const uint4 r = philox4x32_10(make_uint4((uint32_t)u, (uint32_t)j, 0u, 1u), k0, k1);
        const int rank = a.rank_lo + (int)(((uint64_t)r.x * (uint64_t)n) >> 32);
        v = rank < na ? (int32_t)(uint32_t)(top[rank] & 0xFFFFFFFFull) : (int32_t)cls[rank - na];
      }
      outq[j] = v;
    }
    __syncthreads();  // the buffer, the list and LDS are reused by the next query
  }

  if (a.total_steps) {
    const int wave = tid >> 6, lane = tid & (kWave - 1);
    const int ws_sum = wave_sum_i32((int)my_steps);
    __shared__ int wave_tot[kWaves];
    if (lane == 0) wave_tot[wave] = ws_sum;
    __syncthreads();
    if (tid == 0) {
      unsigned long long t = 0;
      for (int w = 0; w < kWaves; ++w) t += (unsigned long long)(unsigned)wave_tot[w];
      if (t) atomicAdd(a.total_steps, t);
    }
  }
}

template <typename OffT, bool TABLE>
hipError_t launch_for_offsets(const HardNegLaunch& a, hipStream_t s) {
  const int wh = a.walks * a.hops;
  const int64_t cap = 1ll << 13;
  const dim3 grid((unsigned)(a.num_queries < cap ? a.num_queries : cap));
  const dim3 block(kThreads);
  if (wh <= 1 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 1, TABLE>), grid, block, 0, s, a);
  else if (wh <= 2 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 2, TABLE>), grid, block, 0, s, a);
  else if (wh <= 4 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 4, TABLE>), grid, block, 0, s, a);
  else if (wh <= 8 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 8, TABLE>), grid, block, 0, s, a);
  else if (wh <= 16 * kThreads) hipLaunchKernelGGL((hard_negative_kernel<OffT, 16, TABLE>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename OffT, bool TABLE>
void launch_global(const HardNegLaunch& a, uint32_t* ws, int64_t words, hipStream_t s) {
  const int64_t blocks = a.num_queries < kGMaxBlocks ? a.num_queries : kGMaxBlocks;
  const dim3 grid((unsigned)blocks), block(kThreads);
  hipLaunchKernelGGL((hard_negative_global_kernel<OffT, TABLE>), grid, block, 0, s, a, ws, words);
}

}  // namespace

int64_t hard_negative_blocks(int64_t num_queries) {
  return num_queries < kGMaxBlocks ? num_queries : kGMaxBlocks;
}

// Per resident workgroup: the partitions' buckets (kCCap words each), the
// overflow list and its copy by partition (L words each) and the (pin, count)
// list (2 L words), rounded to 256 bytes.
static int64_t hard_negative_ws_words(int64_t landings) {
  const int64_t parts = (landings + kCPerPart - 1) / kCPerPart;
  return (parts * kCCap + 4 * landings + 63) / 64 * 64;
}

size_t hard_negative_workspace(int64_t landings, int64_t num_queries) {
  if (landings <= kMaxOnChipLandings || num_queries <= 0) return 0;
  return (size_t)hard_negative_blocks(num_queries) * (size_t)hard_negative_ws_words(landings) *
         sizeof(uint32_t);
}

hipError_t launch_hard_negatives(const HardNegLaunch& a, void* workspace, hipStream_t s) {
  if (a.num_queries <= 0) return hipSuccess;
  ProfileScope prof(kKHardNeg, s);
  const int64_t landings = (int64_t)a.walks * a.hops;
  const bool table = a.table != nullptr;
  if (landings <= kMaxOnChipLandings) {
    if (a.offsets64)
      return table ? launch_for_offsets<int64_t, true>(a, s) : launch_for_offsets<int64_t, false>(a, s);
    return table ? launch_for_offsets<int32_t, true>(a, s) : launch_for_offsets<int32_t, false>(a, s);
  }
  uint32_t* ws = static_cast<uint32_t*>(workspace);
  const int64_t words = hard_negative_ws_words(landings);
  if (a.offsets64) {
    if (table) launch_global<int64_t, true>(a, ws, words, s);
    else launch_global<int64_t, false>(a, ws, words, s);
  } else {
    if (table) launch_global<int32_t, true>(a, ws, words, s);
    else launch_global<int32_t, false>(a, ws, words, s);
  }
  return hipGetLastError();
}

}  // namespace pinsage
