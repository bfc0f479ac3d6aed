// Pool and W fused for bf16 layers in the dense-then-pool order with
// d_in = d_out = 256 (Algorithm 1, lines 1-3; Sec. 3.4):
//   z_u = ReLU(W_s h_u + gamma({R_v : v in N(u)}) + w),  out_u = z_u / ||z_u||
// where R holds W_n ReLU(Q h_v + q) for every pin (the pool is a weighted mean,
// hence linear, so W's neighbour half is applied before it).
//
// Each wave owns 32 output rows at a time, with no block-level barrier:
//   1. pool: one row after another, as the header-in-registers pool kernel
//      does it (the row's ids and weights in one vector load, every live
//      slot's 512-byte row in flight in two lane groups, fp32 sums in rank
//      order, one butterfly between the groups); each pooled row is rounded
//      to bf16 (the precision of the pooled chunk in the two-kernel order) and
//      kept in the wave's LDS strip;
//   2. W_s h^T on the matrix cores: the 32 rows' h fragments (K = 256) in 64
//      VGPRs, the 256 x 32 fp32 result in 128, W_s read from L2 as fragments
//      laid out contiguously by a small permute kernel (1 KB per MFMA);
//   3. + pooled row + w, ReLU, the row's sum of squares over the lane pair
//      that holds it, scale, bf16; staged in the strip and written as whole
//      512-byte rows.
// The pool dominates (each row gathers up to 64 rows of 512 bytes at random);
// the product and epilogue add about 2% to it and replace a separate W GEMM
// and the pooled chunk's round trip through HBM.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kD = 256;            // d_in = d_out
constexpr int kKS = kD / 16;       // k-steps of the product
constexpr int kNB = kD / 32;       // 32-column output blocks
constexpr int kRowB = kD * 2 + 16;  // padded bf16 row in the strip
constexpr int kNBG = 32;           // slots per lane group in flight

// Wsp[nb][ks][lane] (16 bytes) = W[32 nb + lane % 32][16 ks + 8 (lane / 32) ..
// + 7]: the A-operand fragment of v_mfma_f32_32x32x16_bf16 for output block nb
// and k-step ks, so a wave reads each fragment as one contiguous 1 KB.
__global__ void permute_ws_kernel(const uint16_t* __restrict__ W, int64_t ldw,
                                  uint4* __restrict__ Wsp) {
  const int total = kNB * kKS * 64;
  for (int e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += gridDim.x * blockDim.x) {
    const int lane = e & 63, ks = (e >> 6) % kKS, nb = (e >> 6) / kKS;
    const uint16_t* src = W + (int64_t)(32 * nb + (lane & 31)) * ldw + 16 * ks + 8 * (lane >> 5);
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)src[2 * i] | ((uint32_t)src[2 * i + 1] << 16);
    Wsp[e] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

template <int MODE>
__global__ __launch_bounds__(64 * kWaves) __attribute__((amdgpu_waves_per_eu(2, 2)))
void pool_w_kernel(PoolWLaunch a) {
  __shared__ __attribute__((aligned(16))) unsigned char strip_all[kWaves][32 * kRowB];
  __shared__ __attribute__((aligned(16))) float bias_s[kD];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  for (int c = threadIdx.x; c < kD; c += 64 * kWaves) bias_s[c] = a.bias[c];
  __syncthreads();
  unsigned char* strip = strip_all[wave];
  const int T = a.T;
  const uint4* __restrict__ R = static_cast<const uint4*>(a.R);  // 32 vectors per row
  const int grp = lane >> 5, c = lane & 31;                       // pool: lane groups
  const int h = lane >> 5, r32 = lane & 31;                       // product: row, half
  const int64_t groups = (a.rows + 31) / 32;

  for (int64_t g32 = (int64_t)blockIdx.x * kWaves + wave; g32 < groups;
       g32 += (int64_t)gridDim.x * kWaves) {
    const int64_t rbase = g32 * 32;
    const int nrows = a.rows - rbase < 32 ? (int)(a.rows - rbase) : 32;

    // ---- 1. pool the group's rows into the strip ---------------------------
    for (int i = 0; i < nrows; ++i) {
      const int64_t row = rbase + i;
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
      float acc[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = MODE == kPoolMax ? -INFINITY : 0.0f;
      bool any = false;
      for (int b0 = 0; b0 < tend; b0 += 2 * kNBG) {
        uint4 buf[kNBG];
        float al[kNBG];
        bool ok[kNBG];
#pragma unroll
        for (int j = 0; j < kNBG; ++j) {
          const int t = b0 + 2 * j + grp;
          const int32_t vt = __shfl(v, t & 63);
          const float at = __shfl(alpha, t & 63);
          ok[j] = t < tend && vt >= 0;
          al[j] = ok[j] ? at : 0.0f;
          buf[j] = ok[j] ? R[(int64_t)vt * 32 + c] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int j = 0; j < kNBG; ++j) {
          any = any || ok[j];
          const uint32_t wv[4] = {buf[j].x, buf[j].y, buf[j].z, buf[j].w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float f0 = __uint_as_float(wv[q] << 16);
            const float f1 = __uint_as_float(wv[q] & 0xFFFF0000u);
            if constexpr (MODE == kPoolMax) {
              acc[2 * q] = ok[j] ? fmaxf(acc[2 * q], f0) : acc[2 * q];
              acc[2 * q + 1] = ok[j] ? fmaxf(acc[2 * q + 1], f1) : acc[2 * q + 1];
            } else {
              acc[2 * q] = fmaf(al[j], f0, acc[2 * q]);
              acc[2 * q + 1] = fmaf(al[j], f1, acc[2 * q + 1]);
            }
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const float other = __shfl_xor(acc[k], 32);
        acc[k] = MODE == kPoolMax ? fmaxf(acc[k], other) : acc[k] + other;
      }
      if constexpr (MODE == kPoolMax) {
        const bool row_any = __builtin_amdgcn_readfirstlane(wave_sum_i32(any ? 1 : 0)) > 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = row_any ? acc[k] : 0.0f;
      }
      if (grp == 0)
        *reinterpret_cast<u32x4*>(strip + i * kRowB + 16 * c) =
            u32x4{pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]),
                  pack_bf16x2(acc[4], acc[5]), pack_bf16x2(acc[6], acc[7])};
    }
    wave_lds_sync();

    // ---- 2. W_s h^T: lane (r32, h) gets columns 32 nb + 8 g + 4 h + e of row r32
    u32x4 hf[kKS];
    {
      const int64_t row = rbase + r32;
      int64_t hsrc = -1;
      if (r32 < nrows) hsrc = a.self_rows ? (int64_t)a.self_rows[row] : a.h_row0 + row;
      const bool hok = hsrc >= 0 && hsrc < a.rows_h;
      const u32x4* hp = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.H) +
                                                       (hok ? hsrc : 0) * a.ldh + 8 * h);
#pragma unroll
      for (int ks = 0; ks < kKS; ++ks) hf[ks] = hok ? hp[2 * ks] : u32x4{0u, 0u, 0u, 0u};
    }
    f32x16 acc[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[nb][e] = 0.0f;
    // The fragments' base is re-read per group (an empty asm hides its
    // invariance), so the compiler keeps one uniform base and immediate
    // offsets instead of 128 precomputed 64-bit addresses.
    typedef const __attribute__((address_space(1))) unsigned char* gptr;
    gptr wsb = (gptr)a.Wsp;  // global memory
    asm volatile("" : "+s"(wsb));
    const uint32_t voff = 16u * (uint32_t)lane;
    auto frag = [&](int t) __attribute__((always_inline)) {
      return *reinterpret_cast<const __attribute__((address_space(1))) u32x4*>(wsb + 1024 * t +
                                                                                 voff);
    };
    constexpr int kPF = 4;  // fragments in flight ahead of their MFMA
    u32x4 wf[kPF];
#pragma unroll
    for (int p = 0; p < kPF; ++p) wf[p] = frag(p);
#pragma unroll
    for (int t = 0; t < kNB * kKS; ++t) {
      // Step t: output block t / kKS, k-step t % kKS (fragment t of Wsp).
      const u32x4 cur = wf[t % kPF];
      if (t + kPF < kNB * kKS) wf[t % kPF] = frag(t + kPF);
      acc[t / kKS] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          __builtin_bit_cast(bf16x8, cur), __builtin_bit_cast(bf16x8, hf[t % kKS]),
          acc[t / kKS], 0, 0, 0);
    }

    // The epilogue stays behind the products (its LDS reads would otherwise be
    // hoisted among them and hold registers the accumulators need).
    __builtin_amdgcn_sched_barrier(0);

    // ---- 3. + pooled + w, ReLU, row L2 norm, bf16 ---------------------------
    // Lane (r32, h): pooled and output bytes of row r32 at pbase + 2 (32 nb + 8 g),
    // bias at bbase + 32 nb + 8 g: one base register, immediate offsets.
    unsigned char* pbase = strip + r32 * kRowB + 8 * h;
    const float* bbase = bias_s + 4 * h;
    float ss = 0.0f;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2 pv = *reinterpret_cast<const u32x2*>(pbase + 64 * nb + 16 * g);
        const float4 bv = *reinterpret_cast<const float4*>(bbase + 32 * nb + 8 * g);
        const float p[4] = {__uint_as_float(pv.x << 16), __uint_as_float(pv.x & 0xFFFF0000u),
                            __uint_as_float(pv.y << 16), __uint_as_float(pv.y & 0xFFFF0000u)};
        const float b[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = fmaxf(acc[nb][4 * g + e] + b[e] + p[e], 0.0f);
          acc[nb][4 * g + e] = x;
          ss = fmaf(x, x, ss);
        }
      }
    ss += __shfl_xor(ss, 32);
    const float scale = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
    wave_lds_sync();  // every lane has read its pooled values
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        *reinterpret_cast<u32x2*>(pbase + 64 * nb + 16 * g) =
            u32x2{pack_bf16x2(acc[nb][4 * g] * scale, acc[nb][4 * g + 1] * scale),
                  pack_bf16x2(acc[nb][4 * g + 2] * scale, acc[nb][4 * g + 3] * scale)};
      }
    wave_lds_sync();
#pragma unroll
    for (int it = 0; it < 16; ++it) {
      const int rr = 2 * it + (lane >> 5), ck = lane & 31;
      if (rr < nrows)
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.out) + (rbase + rr) * kD + 8 * ck) =
            *reinterpret_cast<const u32x4*>(strip + rr * kRowB + 16 * ck);
    }
    wave_lds_sync();  // the strip is free for the next group
  }
}

}  // namespace

bool pool_w_supported(int d_in, int d_out, bool bf16, int T) {
  return bf16 && d_in == kD && d_out == kD && T >= 1 && T <= 64;
}

size_t pool_w_ws_bytes() { return (size_t)kNB * kKS * 64 * 16; }

hipError_t launch_permute_ws(const void* W, int64_t ldw, void* Wsp, hipStream_t s) {
  hipLaunchKernelGGL(permute_ws_kernel, dim3(32), dim3(256), 0, s,
                     static_cast<const uint16_t*>(W), ldw, static_cast<uint4*>(Wsp));
  return hipGetLastError();
}

hipError_t launch_pool_w(const PoolWLaunch& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (a.T < 1 || a.T > 64) return hipErrorInvalidValue;
  ProfileScope prof(kKPoolW, s);
  const int64_t groups = (a.rows + 31) / 32;
  const int64_t blocks_needed = (groups + kWaves - 1) / kWaves;
  const int64_t cap = 1ll << 20;
  const dim3 grid((unsigned)(blocks_needed < cap ? blocks_needed : cap));
  switch (a.mode) {
    case kPoolImportance:
      hipLaunchKernelGGL(pool_w_kernel<kPoolImportance>, grid, dim3(64 * kWaves), 0, s, a);
      break;
    case kPoolMean:
      hipLaunchKernelGGL(pool_w_kernel<kPoolMean>, grid, dim3(64 * kWaves), 0, s, a);
      break;
    case kPoolMax:
      hipLaunchKernelGGL(pool_w_kernel<kPoolMax>, grid, dim3(64 * kWaves), 0, s, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pinsage
