// Calibration kernels (bench support, not part of the method).
//
// Random reads: the rate at which the chip serves dependent random reads from
// a table far larger than its caches. Every lane follows a chain of `steps` reads; the index of
// each read is a hash of the value the previous one returned, so, as in a
// random walk, a lane has one read in flight at a time and the reads land on
// unrelated cache lines. The walks of Sec. 3.2 take one such read per edge
// step (the neighbour id at a uniform position of the node's row), so this
// rate, not the bytes moved, is what bounds them.
//
// Random row gathers: the rate at which whole rows (512 bytes or 1 KB) are
// gathered from uniformly random positions of a large table, in the access
// pattern of the importance pool (Sec. 3.2): a wave takes one target at a
// time and issues all of its rows' loads (two 512-byte rows, or one 1 KB row,
// per 16-byte-per-lane load instruction) before it consumes any.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

__device__ __forceinline__ uint64_t mix64(uint64_t x) {
  // The finaliser of the SplitMix64 generator (Steele, Lea and Flood, 2014).
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

// E = bytes per element (4, 8 or 16); mask + 1 elements, a power of two.
template <int E>
__global__ __launch_bounds__(256) void random_read_kernel(const unsigned char* __restrict__ table,
                                                          uint64_t mask, int steps,
                                                          uint32_t* __restrict__ sink,
                                                          int64_t chains) {
  const int64_t lane = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (lane >= chains) return;
  uint64_t idx = mix64((uint64_t)lane + 0x9e3779b97f4a7c15ull) & mask;
  uint32_t acc = 0;
  for (int s = 0; s < steps; ++s) {
    uint32_t v;
    if constexpr (E == 16) {
      const uint4 e = reinterpret_cast<const uint4*>(table)[idx];
      v = e.x ^ e.y ^ e.z ^ e.w;
    } else if constexpr (E == 8) {
      const uint2 e = reinterpret_cast<const uint2*>(table)[idx];
      v = e.x ^ e.y;
    } else {
      v = reinterpret_cast<const uint32_t*>(table)[idx];
    }
    acc += v;
    idx = mix64((uint64_t)v + (uint64_t)s + (uint64_t)lane) & mask;
  }
  sink[lane] = acc;
}

constexpr int kGatherMaxLoads = 32;  // load instructions in flight per target

// RV = 16-byte vectors per row (32: 512 bytes, 64: 1 KB). Target t's slot s
// gathers row (mix64(seed + 64 t + s) >> 32) * rows >> 32; every gathered
// 32-bit word is added into *sink (mod 2^32).
template <int RV>
__global__ __launch_bounds__(256) void random_gather_kernel(const uint4* __restrict__ table,
                                                            uint64_t rows, int64_t targets,
                                                            int per, uint64_t seed,
                                                            uint32_t* __restrict__ sink) {
  constexpr int kLanesPerRow = RV < kWave ? RV : kWave;
  constexpr int kRowsPerLoad = kWave / kLanesPerRow;
  constexpr int kVecPerLane = RV / kLanesPerRow;
  static_assert(kVecPerLane == 1, "one vector per lane and row");
  const int lane = threadIdx.x & (kWave - 1);
  const int grp = lane / kLanesPerRow, c = lane % kLanesPerRow;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
  const int64_t waves = (int64_t)gridDim.x * (blockDim.x / kWave);
  uint32_t acc = 0;
  for (int64_t t = wave; t < targets; t += waves) {
    uint4 buf[kGatherMaxLoads];
#pragma unroll
    for (int j = 0; j < kGatherMaxLoads; ++j) {
      const int sl = kRowsPerLoad * j + grp;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (sl < per) {
        const uint64_t h = mix64(seed + 64 * (uint64_t)t + (uint64_t)sl) >> 32;
        const uint64_t row = (h * rows) >> 32;
        v = table[row * RV + c];
      }
      buf[j] = v;
    }
#pragma unroll
    for (int j = 0; j < kGatherMaxLoads; ++j) acc += buf[j].x + buf[j].y + buf[j].z + buf[j].w;
  }
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) atomicAdd(sink, acc);
}

}  // namespace

hipError_t launch_random_gathers(const void* table, uint64_t rows, int row_bytes,
                                 int64_t targets, int per, uint64_t seed, uint32_t* sink,
                                 hipStream_t s) {
  const uint4* t = static_cast<const uint4*>(table);
  const int64_t blocks = (targets + 3) / 4 < 8192 ? (targets + 3) / 4 : 8192;  // 4 waves each
  if (row_bytes == 1024)
    hipLaunchKernelGGL(random_gather_kernel<64>, dim3((unsigned)blocks), dim3(256), 0, s, t, rows,
                       targets, per, seed, sink);
  else
    hipLaunchKernelGGL(random_gather_kernel<32>, dim3((unsigned)blocks), dim3(256), 0, s, t, rows,
                       targets, per, seed, sink);
  return hipGetLastError();
}

hipError_t launch_random_reads(const void* table, uint64_t elements, int elem_bytes, int steps,
                               uint32_t* sink, int64_t chains, hipStream_t s) {
  const unsigned char* t = static_cast<const unsigned char*>(table);
  const uint64_t mask = elements - 1;
  const int64_t blocks = (chains + 255) / 256;
  if (blocks > 0x7FFFFFFFll) return hipErrorInvalidValue;
  if (elem_bytes == 16)
    hipLaunchKernelGGL(random_read_kernel<16>, dim3((unsigned)blocks), dim3(256), 0, s, t, mask,
                       steps, sink, chains);
  else if (elem_bytes == 8)
    hipLaunchKernelGGL(random_read_kernel<8>, dim3((unsigned)blocks), dim3(256), 0, s, t, mask,
                       steps, sink, chains);
  else
    hipLaunchKernelGGL(random_read_kernel<4>, dim3((unsigned)blocks), dim3(256), 0, s, t, mask,
                       steps, sink, chains);
  return hipGetLastError();
}

}  // namespace pinsage
