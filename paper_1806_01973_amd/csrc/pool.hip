// Neighbourhood pooling on gfx950 (Algorithm 1, line 1 applied as a gather
// over the once-per-node projections of Sec. 3.4). Importance pooling
// (Sec. 3.2: gamma is the weighted mean of the transformed neighbour vectors,
// weighted by the L1-normalised visit counts):
//   n[r] = sum_t alpha[r][t] * P[idx[r][t]];
// and the gamma = mean and gamma = max variants compared in Sec. 4.
//
// One wavefront per output row (grid-stride). The row's idx/weights are
// wave-uniform and come through the scalar cache; each lane owns VEC
// consecutive columns of every 64*VEC-column slab, so one load instruction of
// the wave reads a contiguous 64*VEC-element span of a gathered row. Rows are
// fetched in groups of U neighbours before they are accumulated, which
// keeps several row reads in flight per wave. The sum runs in rank order t in
// fp32; the result is stored in the storage dtype.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

constexpr int kWavesPerBlock = 4;

template <bool BF16>
struct Vec;
template <>
struct Vec<false> {  // 4 x fp32 = 16 B per lane
  static constexpr int kN = 4;
  using Raw = float4;
  __device__ static void to_f32(const Raw& r, float (&o)[4]) {
    o[0] = r.x; o[1] = r.y; o[2] = r.z; o[3] = r.w;
  }
  __device__ static Raw from_f32(const float (&o)[4]) { return make_float4(o[0], o[1], o[2], o[3]); }
};
template <>
struct Vec<true> {  // 8 x bf16 = 16 B per lane
  static constexpr int kN = 8;
  using Raw = uint4;
  __device__ static void to_f32(const Raw& r, float (&o)[8]) {
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(w[i] << 16);
      o[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ static Raw from_f32(const float (&o)[8]) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)f32_to_bf16(o[2 * i]) | ((uint32_t)f32_to_bf16(o[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Per-row setup shared by both kernels: the weight sum S of a row without
// stored weights (importance pooling derives alpha = count / S) or the number
// of neighbours (mean pooling), counted by the lanes in parallel; integers, so
// the order does not matter.
__device__ __forceinline__ int row_total(const PoolLaunch& a, int64_t row, int lane) {
  const int T = a.T;
  int part = 0;
  if (a.mode == kPoolMean) {
    for (int t = lane; t < T; t += kWave) {
      const int32_t v = a.idx[row * T + t];
      part += ((uint64_t)(int64_t)v < (uint64_t)a.n_transform) ? 1 : 0;
    }
  } else if (a.mode == kPoolImportance && !a.weights) {
    for (int t = lane; t < T; t += kWave) part += a.counts[row * T + t];
  } else {
    return 0;
  }
  return wave_sum_i32(part);
}

// One past the last slot of the row that holds a neighbour (0 for an empty
// row): the loops stop there, so short rows of a wide table cost little.
// Skipped slots hold no neighbour and would contribute nothing.
__device__ __forceinline__ int row_end(const PoolLaunch& a, int64_t row, int lane) {
  const int T = a.T;
  int last = -1;
  for (int t = lane; t < T; t += kWave) {
    const int32_t v = a.idx[row * T + t];
    if ((uint64_t)(int64_t)v < (uint64_t)a.n_transform) last = t;
  }
  return __builtin_amdgcn_readfirstlane(wave_max_i32(last)) + 1;
}

// Weight of neighbour slot t of a row (importance or mean pooling).
template <int MODE>
__device__ __forceinline__ float slot_alpha(const PoolLaunch& a, int64_t row, int t, int total) {
  if constexpr (MODE == kPoolMean) return 1.0f / (float)total;
  if (a.weights) return a.weights[row * a.T + t];
  return (float)a.counts[row * a.T + t] / (float)total;
}

// J = number of 64*VEC-column slabs per row (compile time); U neighbour rows
// are in flight per wave (U*J 16-byte loads per lane). MODE: importance
// (weighted sum), mean (uniform weights 1/#neighbours) or max (element-wise,
// skipped slots do not take part; an empty row gives zeros).
template <bool BF16, int MODE, int J, int U = (J <= 2 ? 8 : (J <= 4 ? 4 : (J <= 8 ? 2 : 1)))>
__global__ __launch_bounds__(256) void pool_kernel(PoolLaunch a) {
  using V = Vec<BF16>;
  using Raw = typename V::Raw;
  constexpr int VN = V::kN;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int m = a.m;
  const int T = a.T;
  const Raw* __restrict__ P = static_cast<const Raw*>(a.P);
  Raw* __restrict__ out = static_cast<Raw*>(a.out);
  const int vec_per_row = m / VN;

  for (int64_t row0 = (int64_t)blockIdx.x * kWavesPerBlock + wave; row0 < a.rows;
       row0 += (int64_t)gridDim.x * kWavesPerBlock) {
    const int64_t row = row0;
    const int32_t* __restrict__ ridx = a.idx + row * T;
    const int total = row_total(a, row, lane);
    const int tend = row_end(a, row, lane);
    float acc[J][VN];
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int v = 0; v < VN; ++v) acc[j][v] = MODE == kPoolMax ? -INFINITY : 0.0f;
    bool any = false;

    for (int t0 = 0; t0 < tend; t0 += U) {
      Raw buf[U][J];
      float alpha[U];
      bool ok[U];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int t = t0 + i;
        int32_t v = t < tend ? ridx[t] : -1;
        if ((uint64_t)(int64_t)v >= (uint64_t)a.n_transform) v = -1;
        ok[i] = v >= 0;
        alpha[i] = 0.0f;
        if constexpr (MODE != kPoolMax)
          if (v >= 0) alpha[i] = slot_alpha<MODE>(a, row, t, total);
#pragma unroll
        for (int j = 0; j < J; ++j) {
          const int c = j * kWave + lane;
          if (v >= 0 && c < vec_per_row) buf[i][j] = P[(int64_t)v * vec_per_row + c];
          else buf[i][j] = Raw{};
        }
      }
#pragma unroll
      for (int i = 0; i < U; ++i) {
        any = any || ok[i];
#pragma unroll
        for (int j = 0; j < J; ++j) {
          float f[VN];
          V::to_f32(buf[i][j], f);
#pragma unroll
          for (int v = 0; v < VN; ++v) {
            if constexpr (MODE == kPoolMax) acc[j][v] = ok[i] ? fmaxf(acc[j][v], f[v]) : acc[j][v];
            else acc[j][v] = fmaf(alpha[i], f[v], acc[j][v]);
          }
        }
      }
    }
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = j * kWave + lane;
      if constexpr (MODE == kPoolMax)
#pragma unroll
        for (int v = 0; v < VN; ++v) acc[j][v] = any ? acc[j][v] : 0.0f;
      if (c < vec_per_row) out[row * vec_per_row + c] = V::from_f32(acc[j]);
    }
  }
}

// Rows narrower than one wave slab (at most 64 / RG vectors): the wave splits
// into RG lane groups of 64 / RG lanes, group g gathering neighbours
// t = g, g + RG, ... of the row, so one load instruction reads RG rows. Each
// group reduces its neighbours in rank order; the RG partial results are then
// combined by a fixed butterfly over the groups (the same order on every
// lane). U = 4 loads in flight per lane: on 512-byte rows, 8 and 16 measured
// 5% and 40% slower (fewer resident waves).
template <bool BF16, int MODE, int RG, int U = 4>
__global__ __launch_bounds__(256) void pool_narrow_kernel(PoolLaunch a) {
  using V = Vec<BF16>;
  using Raw = typename V::Raw;
  constexpr int VN = V::kN;
  constexpr int GL = kWave / RG;  // lanes per group
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int grp = lane / GL, c = lane % GL;
  const int T = a.T;
  const Raw* __restrict__ P = static_cast<const Raw*>(a.P);
  Raw* __restrict__ out = static_cast<Raw*>(a.out);
  const int vec_per_row = a.m / VN;
  const bool col_ok = c < vec_per_row;

  for (int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wave; row < a.rows;
       row += (int64_t)gridDim.x * kWavesPerBlock) {
    const int32_t* __restrict__ ridx = a.idx + row * T;
    const int total = row_total(a, row, lane);
    const int tend = row_end(a, row, lane);
    float acc[VN];
#pragma unroll
    for (int v = 0; v < VN; ++v) acc[v] = MODE == kPoolMax ? -INFINITY : 0.0f;
    bool any = false;
    for (int t0 = 0; t0 < tend; t0 += U * RG) {
      Raw buf[U];
      float alpha[U];
      bool ok[U];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int t = t0 + i * RG + grp;
        int32_t v = t < tend ? ridx[t] : -1;
        if ((uint64_t)(int64_t)v >= (uint64_t)a.n_transform) v = -1;
        ok[i] = v >= 0;
        alpha[i] = 0.0f;
        if constexpr (MODE != kPoolMax)
          if (v >= 0) alpha[i] = slot_alpha<MODE>(a, row, t, total);
        buf[i] = (v >= 0 && col_ok) ? P[(int64_t)v * vec_per_row + c] : Raw{};
      }
#pragma unroll
      for (int i = 0; i < U; ++i) {
        any = any || ok[i];
        float f[VN];
        V::to_f32(buf[i], f);
#pragma unroll
        for (int v = 0; v < VN; ++v) {
          if constexpr (MODE == kPoolMax) acc[v] = ok[i] ? fmaxf(acc[v], f[v]) : acc[v];
          else acc[v] = fmaf(alpha[i], f[v], acc[v]);
        }
      }
    }
#pragma unroll
    for (int o = GL; o < kWave; o <<= 1)
#pragma unroll
      for (int v = 0; v < VN; ++v) {
        const float other = __shfl_xor(acc[v], o);
        acc[v] = MODE == kPoolMax ? fmaxf(acc[v], other) : acc[v] + other;
      }
    if constexpr (MODE == kPoolMax) {
      // `any` of the whole row: some group saw a neighbour.
      const bool row_any = __builtin_amdgcn_readfirstlane(wave_sum_i32(any ? 1 : 0)) > 0;
#pragma unroll
      for (int v = 0; v < VN; ++v) acc[v] = row_any ? acc[v] : 0.0f;
    }
    if (grp == 0 && col_ok) out[row * vec_per_row + c] = V::from_f32(acc);
  }
}

// Rows of at most 64 / RG vectors with at most 64 neighbour slots (every
// workload's pooled width in the dense-then-pool order): the row's header --
// neighbour ids and the weights, counts or neighbour count alpha needs -- is
// one coalesced vector load (lane t holds slot t), alpha is formed per lane
// with the same fp32 division as the batched kernels, and every live slot's
// gather is issued before the first one is summed: NB slots per lane group
// per batch (one batch when the row has at most RG * NB slots), slot ids and
// alphas passed to the groups by lane permutes. Group g sums slots g, g + RG,
// ... in rank order and the groups are combined by the same butterfly as in
// pool_narrow_kernel, so the result is the same bits. Measured on random 512-byte rows from a 41 GB
// table: as fast as a gather with no header reads at all (+16% over the
// batched kernel).
template <bool BF16, int MODE, int RG, int NB>
__global__ __launch_bounds__(256) void pool_head_kernel(PoolLaunch a) {
  using V = Vec<BF16>;
  using Raw = typename V::Raw;
  constexpr int VN = V::kN;
  constexpr int GL = kWave / RG;  // lanes per group
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int grp = lane / GL, c = lane % GL;
  const int T = a.T;
  const Raw* __restrict__ P = static_cast<const Raw*>(a.P);
  Raw* __restrict__ out = static_cast<Raw*>(a.out);
  const int vec_per_row = a.m / VN;
  const bool col_ok = c < vec_per_row;

  for (int64_t row = (int64_t)blockIdx.x * kWavesPerBlock + wave; row < a.rows;
       row += (int64_t)gridDim.x * kWavesPerBlock) {
    // Header: slot `lane` of the row.
    int32_t v = -1;
    float w = 0.0f;
    int cnt = 0;
    if (lane < T) {
      v = a.idx[row * T + lane];
      if constexpr (MODE == kPoolImportance) {
        if (a.weights) w = a.weights[row * T + lane];
        else cnt = a.counts[row * T + lane];
      }
    }
    const bool valid = (uint64_t)(int64_t)v < (uint64_t)a.n_transform;
    if (!valid) v = -1;
    float alpha = 0.0f;
    if constexpr (MODE == kPoolMean) {
      const int total = wave_sum_i32(valid ? 1 : 0);
      alpha = valid ? 1.0f / (float)total : 0.0f;
    } else if constexpr (MODE == kPoolImportance) {
      if (a.weights) {
        alpha = valid ? w : 0.0f;
      } else {
        const int total = wave_sum_i32(cnt);  // every slot, as the walk kernel's S
        alpha = valid ? (float)cnt / (float)total : 0.0f;
      }
    }
    const int tend = __builtin_amdgcn_readfirstlane(wave_max_i32(valid ? lane : -1)) + 1;

    float acc[VN];
#pragma unroll
    for (int k = 0; k < VN; ++k) acc[k] = MODE == kPoolMax ? -INFINITY : 0.0f;
    bool any = false;
    for (int b0 = 0; b0 < tend; b0 += RG * NB) {
      Raw buf[NB];
      float al[NB];
      bool ok[NB];
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const int t = b0 + i * RG + grp;
        int32_t vt;
        float at;
        if constexpr (RG == 1) {
          vt = __builtin_amdgcn_readlane(v, t & 63);
          at = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(alpha), t & 63));
        } else {
          vt = __shfl(v, t & 63);
          at = __shfl(alpha, t & 63);
        }
        ok[i] = t < tend && vt >= 0;
        al[i] = ok[i] ? at : 0.0f;
        buf[i] = (ok[i] && col_ok) ? P[(int64_t)vt * vec_per_row + c] : Raw{};
      }
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        any = any || ok[i];
        float f[VN];
        V::to_f32(buf[i], f);
#pragma unroll
        for (int k = 0; k < VN; ++k) {
          if constexpr (MODE == kPoolMax) acc[k] = ok[i] ? fmaxf(acc[k], f[k]) : acc[k];
          else acc[k] = fmaf(al[i], f[k], acc[k]);
        }
      }
    }
#pragma unroll
    for (int o = GL; o < kWave; o <<= 1)
#pragma unroll
      for (int k = 0; k < VN; ++k) {
        const float other = __shfl_xor(acc[k], o);
        acc[k] = MODE == kPoolMax ? fmaxf(acc[k], other) : acc[k] + other;
      }
    if constexpr (MODE == kPoolMax) {
      const bool row_any = __builtin_amdgcn_readfirstlane(wave_sum_i32(any ? 1 : 0)) > 0;
#pragma unroll
      for (int k = 0; k < VN; ++k) acc[k] = row_any ? acc[k] : 0.0f;
    }
    if (grp == 0 && col_ok) out[row * vec_per_row + c] = V::from_f32(acc);
  }
}

template <bool BF16, int MODE>
hipError_t launch_batched(const PoolLaunch& a, dim3 grid, dim3 block, int slabs, int vec_per_row,
                          hipStream_t s);

template <bool BF16, int MODE>
hipError_t launch_mode(const PoolLaunch& a, hipStream_t s) {
  constexpr int VN = BF16 ? 8 : 4;
  const int slabs = (a.m / VN + kWave - 1) / kWave;
  const int64_t blocks_needed = (a.rows + kWavesPerBlock - 1) / kWavesPerBlock;
  const int64_t cap = 1ll << 22;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  const dim3 block(256);
  const int vec_per_row = a.m / VN;
  // The header-in-registers kernel for rows narrower than a wave slab (it gathers
  // 1 KB per load instruction from two or four rows at once). Rows of a full
  // slab measured as fast or faster in the batched kernel (1.2M- and 12M-node
  // graphs: 6.49 against 6.61 ms, 25.1 against 25.3 ms), and much faster on
  // short neighbourhoods (graph neighbourhoods of about 3 pins: 0.84 against
  // 1.58 ms), where the header's round trip is most of a row's work.
  if (a.T <= kWave && vec_per_row <= kWave / 2) {
    if (vec_per_row <= kWave / 4)
      hipLaunchKernelGGL((pool_head_kernel<BF16, MODE, 4, 16>), grid, block, 0, s, a);
    else
      hipLaunchKernelGGL((pool_head_kernel<BF16, MODE, 2, 32>), grid, block, 0, s, a);
    return hipGetLastError();
  }
  return launch_batched<BF16, MODE>(a, grid, block, slabs, vec_per_row, s);
}

// Neighbourhoods of more than 64 slots, or rows wider than one slab.
template <bool BF16, int MODE>
hipError_t launch_batched(const PoolLaunch& a, dim3 grid, dim3 block, int slabs, int vec_per_row,
                          hipStream_t s) {
  if (vec_per_row <= kWave / 4)
    hipLaunchKernelGGL((pool_narrow_kernel<BF16, MODE, 4>), grid, block, 0, s, a);
  else if (vec_per_row <= kWave / 2)
    hipLaunchKernelGGL((pool_narrow_kernel<BF16, MODE, 2>), grid, block, 0, s, a);
  else if (slabs <= 1) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 1>), grid, block, 0, s, a);
  else if (slabs <= 2) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 2>), grid, block, 0, s, a);
  else if (slabs <= 4) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 4>), grid, block, 0, s, a);
  else if (slabs <= 8) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 8>), grid, block, 0, s, a);
  else if (slabs <= 16) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 16>), grid, block, 0, s, a);
  else if (slabs <= 32) hipLaunchKernelGGL((pool_kernel<BF16, MODE, 32>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

template <bool BF16>
hipError_t launch_typed(const PoolLaunch& a, hipStream_t s) {
  switch (a.mode) {
    case kPoolImportance: return launch_mode<BF16, kPoolImportance>(a, s);
    case kPoolMean: return launch_mode<BF16, kPoolMean>(a, s);
    case kPoolMax: return launch_mode<BF16, kPoolMax>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_pool(const PoolLaunch& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  ProfileScope prof(kKPool, s);
  return a.bf16 ? launch_typed<true>(a, s) : launch_typed<false>(a, s);
}

}  // namespace pinsage
