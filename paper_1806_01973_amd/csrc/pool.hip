// Importance pooling on gfx950 (Sec. 3.2: gamma is the weighted mean of the
// transformed neighbour vectors, weighted by the L1-normalised visit counts;
// Algorithm 1, line 1 applied as a gather over the once-per-node projections
// of Sec. 3.4):  n[r] = sum_t alpha[r][t] * P[idx[r][t]].
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

// J = number of 64*VEC-column slabs per row (compile time); U neighbour rows
// are in flight per wave (U*J 16-byte loads per lane).
template <bool BF16, int J, int U = (J <= 2 ? 8 : (J <= 4 ? 4 : (J <= 8 ? 2 : 1)))>
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
    // Without stored weights, alpha = count / (sum of the row's counts): the
    // lanes load the counts in parallel and the wave adds them (integers, so
    // the order does not matter).
    int total = 0;
    if (!a.weights) {
      int part = 0;
      for (int t = lane; t < T; t += kWave) part += a.counts[row * T + t];
      total = wave_sum_i32(part);
    }
    float acc[J][VN];
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int v = 0; v < VN; ++v) acc[j][v] = 0.0f;

    for (int t0 = 0; t0 < T; t0 += U) {
      Raw buf[U][J];
      float alpha[U];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int t = t0 + i;
        int32_t v = t < T ? ridx[t] : -1;
        if ((uint64_t)(int64_t)v >= (uint64_t)a.n_transform) v = -1;
        float al = 0.0f;
        if (v >= 0) {
          if (a.weights) al = a.weights[row * T + t];
          else al = (float)a.counts[row * T + t] / (float)total;
        }
        alpha[i] = (v >= 0) ? al : 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
          const int c = j * kWave + lane;
          if (v >= 0 && c < vec_per_row) buf[i][j] = P[(int64_t)v * vec_per_row + c];
          else buf[i][j] = Raw{};
        }
      }
#pragma unroll
      for (int i = 0; i < U; ++i) {
#pragma unroll
        for (int j = 0; j < J; ++j) {
          float f[VN];
          V::to_f32(buf[i][j], f);
#pragma unroll
          for (int v = 0; v < VN; ++v) acc[j][v] = fmaf(alpha[i], f[v], acc[j][v]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = j * kWave + lane;
      if (c < vec_per_row) out[row * vec_per_row + c] = V::from_f32(acc[j]);
    }
  }
}

// Rows narrower than one wave slab (at most 64 / RG vectors): the wave splits
// into RG lane groups of 64 / RG lanes, group g gathering neighbours
// t = g, g + RG, ... of the row, so one load instruction reads RG rows. Each
// group sums its neighbours in rank order; the RG partial sums are then added
// by a fixed butterfly over the groups (the same order on every lane). U = 4
// loads in flight per lane: on 512-byte rows, 8 and 16 measured 5% and 40%
// slower (fewer resident waves).
template <bool BF16, int RG, int U = 4>
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
    int total = 0;
    if (!a.weights) {
      int part = 0;
      for (int t = lane; t < T; t += kWave) part += a.counts[row * T + t];
      total = wave_sum_i32(part);
    }
    float acc[VN];
#pragma unroll
    for (int v = 0; v < VN; ++v) acc[v] = 0.0f;
    for (int t0 = 0; t0 < T; t0 += U * RG) {
      Raw buf[U];
      float alpha[U];
#pragma unroll
      for (int i = 0; i < U; ++i) {
        const int t = t0 + i * RG + grp;
        int32_t v = t < T ? ridx[t] : -1;
        if ((uint64_t)(int64_t)v >= (uint64_t)a.n_transform) v = -1;
        float al = 0.0f;
        if (v >= 0) {
          if (a.weights) al = a.weights[row * T + t];
          else al = (float)a.counts[row * T + t] / (float)total;
        }
        alpha[i] = al;
        buf[i] = (v >= 0 && col_ok) ? P[(int64_t)v * vec_per_row + c] : Raw{};
      }
#pragma unroll
      for (int i = 0; i < U; ++i) {
        float f[VN];
        V::to_f32(buf[i], f);
#pragma unroll
        for (int v = 0; v < VN; ++v) acc[v] = fmaf(alpha[i], f[v], acc[v]);
      }
    }
#pragma unroll
    for (int o = GL; o < kWave; o <<= 1)
#pragma unroll
      for (int v = 0; v < VN; ++v) acc[v] += __shfl_xor(acc[v], o);
    if (grp == 0 && col_ok) out[row * vec_per_row + c] = V::from_f32(acc);
  }
}

template <bool BF16>
hipError_t launch_typed(const PoolLaunch& a, hipStream_t s) {
  constexpr int VN = BF16 ? 8 : 4;
  const int slabs = (a.m / VN + kWave - 1) / kWave;
  const int64_t blocks_needed = (a.rows + kWavesPerBlock - 1) / kWavesPerBlock;
  const int64_t cap = 1ll << 22;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  const dim3 block(256);
  const int vec_per_row = a.m / VN;
  if (vec_per_row <= kWave / 4)
    hipLaunchKernelGGL((pool_narrow_kernel<BF16, 4>), grid, block, 0, s, a);
  else if (vec_per_row <= kWave / 2)
    hipLaunchKernelGGL((pool_narrow_kernel<BF16, 2>), grid, block, 0, s, a);
  else if (slabs <= 1) hipLaunchKernelGGL((pool_kernel<BF16, 1>), grid, block, 0, s, a);
  else if (slabs <= 2) hipLaunchKernelGGL((pool_kernel<BF16, 2>), grid, block, 0, s, a);
  else if (slabs <= 4) hipLaunchKernelGGL((pool_kernel<BF16, 4>), grid, block, 0, s, a);
  else if (slabs <= 8) hipLaunchKernelGGL((pool_kernel<BF16, 8>), grid, block, 0, s, a);
  else if (slabs <= 16) hipLaunchKernelGGL((pool_kernel<BF16, 16>), grid, block, 0, s, a);
  else if (slabs <= 32) hipLaunchKernelGGL((pool_kernel<BF16, 32>), grid, block, 0, s, a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pool(const PoolLaunch& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  ProfileScope prof(kKPool, s);
  return a.bf16 ? launch_typed<true>(a, s) : launch_typed<false>(a, s);
}

}  // namespace pinsage
