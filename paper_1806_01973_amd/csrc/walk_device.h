// Device pieces of the Sec. 3.2 random walks shared by the neighbourhood
// kernel and the hard negative kernel: the walk state machine and the
// register bitonic sort of a wavefront.
#pragma once

#include "device_util.h"

namespace pinsage {
namespace walkdev {

constexpr uint32_t kEmpty = 0xFFFFFFFFu;

// One cross-lane compare-exchange stage: each element meets the same
// element of lane (lane ^ M) and keeps the smaller value when take_min.
template <int M, int E>
__device__ __forceinline__ void cross_lane_stage(uint32_t (&k)[E], int lane, bool take_min) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const uint32_t other = lane_xor<M>(k[e], lane);
    const uint32_t lo = k[e] < other ? k[e] : other;
    const uint32_t hi = k[e] < other ? other : k[e];
    k[e] = take_min ? lo : hi;
  }
}

// Ascending bitonic sort of the 64*E keys held E per lane (element index
// lane*E + e). Stages with stride >= E pair lanes (lane ^ stride/E, same e)
// through DPP/swizzle exchanges; their direction depends on the lane only.
// Shorter strides pair registers of one lane.
template <int E>
__device__ __forceinline__ void bitonic_sort_wave(uint32_t (&k)[E], int lane) {
  const int lane_base = lane * E;
#pragma unroll
  for (int size = 2; size <= kWave * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= E) {
        const bool up = (lane_base & size) == 0;
        const bool lower = (lane_base & stride) == 0;
        const bool take_min = up == lower;
        switch (stride / E) {
          case 1: cross_lane_stage<1>(k, lane, take_min); break;
          case 2: cross_lane_stage<2>(k, lane, take_min); break;
          case 4: cross_lane_stage<4>(k, lane, take_min); break;
          case 8: cross_lane_stage<8>(k, lane, take_min); break;
          case 16: cross_lane_stage<16>(k, lane, take_min); break;
          default: cross_lane_stage<32>(k, lane, take_min); break;
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          if ((e & stride) == 0) {
            const bool up = size < E ? ((e & size) == 0) : ((lane_base & size) == 0);
            const uint32_t a = k[e], b = k[e + stride];
            const uint32_t lo = a < b ? a : b;
            const uint32_t hi = a < b ? b : a;
            k[e] = up ? lo : hi;
            k[e + stride] = up ? hi : lo;
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

// One walk (Sec. 3.2): from the source u, uniform neighbour choice per edge
// step, ends after `hops` pin landings, 2*hops steps, a node without edges or
// an out-of-range CSR entry. Landings go to `mine[0..hops)`; the source itself
// is recorded as empty.
template <typename OffT>
struct Walker {
  int64_t u, cur, next_at;
  int64_t lo;   // walk-table path: row start and degree of the current node
  int32_t deg;  // (0 when its row is empty or out of range)
  uint32_t w;
  int landed, s;
  bool exists, active;
  uint4 rnd;
  uint32_t* mine;

  __device__ void start(int64_t src, int walk, uint32_t* slots, bool present) {
    u = src;
    cur = src;
    next_at = 0;
    w = (uint32_t)walk;
    landed = 0;
    s = 0;
    exists = present;
    active = present;
    rnd = make_uint4(0, 0, 0, 0);
    mine = slots;
  }
  // Chooses the next CSR position from the row [lo, hi) of the current node.
  __device__ void pick(int64_t lo, int64_t hi, int64_t nnz, uint32_t k0, uint32_t k1) {
    if (!active) return;
    const int64_t deg = hi - lo;
    if (deg <= 0 || lo < 0 || hi > nnz) {
      active = false;
      return;
    }
    if ((s & 3) == 0)
      rnd = philox4x32_10(make_uint4((uint32_t)u, w, (uint32_t)(s >> 2), 0u), k0, k1);
    const uint32_t r = pick_word(rnd, s);
    next_at = lo + (int64_t)(((uint64_t)r * (uint64_t)deg) >> 32);
  }
  // Walk-table path: the same choice from the current node's row [lo, lo + deg)
  // carried by the walker (deg = 0 when the row is empty or malformed).
  __device__ void pick_carried(uint32_t k0, uint32_t k1) {
    if (!active) return;
    if (deg <= 0) {
      active = false;
      return;
    }
    if ((s & 3) == 0)
      rnd = philox4x32_10(make_uint4((uint32_t)u, w, (uint32_t)(s >> 2), 0u), k0, k1);
    const uint32_t r = pick_word(rnd, s);
    next_at = lo + (int64_t)(((uint64_t)r * (uint64_t)(uint32_t)deg) >> 32);
  }
  // Walk-table path: moves to the node of table entry e = {id, degree, row
  // start lo, hi}, recording a pin landing, and carries the node's row.
  __device__ void land_entry(const uint4& e, int64_t num_pins, int64_t num_nodes, int hops) {
    land((int32_t)e.x, num_pins, num_nodes, hops);
    deg = (int32_t)e.y;
    lo = (int64_t)(((uint64_t)e.w << 32) | (uint64_t)e.z);
  }
  // Moves to node nxt (read from col[next_at]). Returns true when the walk
  // landed on a pin, with *visit the visit to record: the pin, or kEmpty
  // when it is the source itself.
  __device__ bool advance(int32_t nxt, int64_t num_pins, int64_t num_nodes, int hops,
                          uint32_t* visit) {
    if (!active) return false;
    if (nxt < 0 || (int64_t)nxt >= num_nodes) {
      active = false;
      return false;
    }
    cur = nxt;
    ++s;
    bool on_pin = false;
    if (cur < num_pins) {
      *visit = (cur != u) ? (uint32_t)cur : kEmpty;
      ++landed;
      on_pin = true;
    }
    if (landed >= hops || s >= 2 * hops) active = false;
    return on_pin;
  }
  // advance(), recording the visit in the walk's slots.
  __device__ void land(int32_t nxt, int64_t num_pins, int64_t num_nodes, int hops) {
    uint32_t v;
    if (advance(nxt, num_pins, num_nodes, hops, &v)) mine[landed - 1] = v;
  }
  // Pads the unused landing slots; returns the edge steps taken.
  __device__ uint32_t finish(int hops) {
    if (!exists) return 0;
    for (int h = landed; h < hops; ++h) mine[h] = kEmpty;
    return (uint32_t)s;
  }
};

// Ascending half-cleaners over the 64*E keys of a wave (strides 32E .. 1):
// sorts a wave-sized bitonic sequence, e.g. the lower or upper half of a
// larger bitonic merge once the strides above the wave are done. Expanded by
// template recursion so every stride, and every register index, is a
// compile-time constant.
template <int E, int STRIDE>
__device__ __forceinline__ void merge_wave_step(uint32_t (&k)[E], int lane) {
  if constexpr (STRIDE >= E) {
    cross_lane_stage<STRIDE / E>(k, lane, ((lane * E) & STRIDE) == 0);
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if ((e & STRIDE) == 0) {
        const uint32_t x = k[e], y = k[e + STRIDE];
        k[e] = x < y ? x : y;
        k[e + STRIDE] = x < y ? y : x;
      }
    }
  }
  if constexpr (STRIDE > 1) merge_wave_step<E, STRIDE / 2>(k, lane);
}

template <int E>
__device__ __forceinline__ void merge_wave_ascending(uint32_t (&k)[E], int lane) {
  merge_wave_step<E, kWave * E / 2>(k, lane);
}

}  // namespace walkdev
}  // namespace pinsage
