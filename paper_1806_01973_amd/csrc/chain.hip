// Chained transform of the dense-then-pool dataflow on gfx950 matrix cores.
// Algorithm 1, line 1 projects every pin once (Sec. 3.4); the importance pool
// is a weighted mean, hence linear, so the neighbour half W_n of W (line 2)
// can be applied to each projected pin before the pool:
//   R = ReLU(H Q^T + q) W_n^T
// This kernel computes R directly: P = ReLU(H Q^T + q) exists only in
// registers, 32 columns at a time, and never reaches memory.
//
// Block: 4 waves (one per SIMD), 128 rows of H; two blocks share a CU, so one
// block's H loads and R stores can run under the other's matrix work. Wave w
// owns rows 32 w .. 32 w + 31 of the tile and keeps their H fragments for the
// whole K = d_in of the first product in registers (64 VGPRs) beside its R
// accumulators (d_out x 32 fp32, 128 registers). (Four waves of 64 rows each,
// sharing every weight fragment between two MFMAs, measured slower: their 288
// accumulator registers overflow the 256 AGPRs.) For each chunk of 32 columns
// of P:
//   1. acc1 (32 x 32) = Q_chunk H^T over K = d_in (v_mfma_f32_32x32x16_bf16;
//      Q rows are the first operand, so a lane holds one H row and the P
//      columns 8 g + 4 h + e, h = lane / 32, e < 4, g < 4);
//   2. bias + ReLU + round to bf16 (the stored precision of P in the
//      two-kernel path), packed in place as the second operand of
//   3. acc2 (d_out x 32 rows) += W_n' P_chunk^T, K = the chunk's 32 columns.
//      The MFMA takes lane half h's 8 k values in the order of P columns
//      {4h .. 4h + 3, 8 + 4h .. 8 + 4h + 3} of each 16-column group, which is
//      exactly what acc1 holds; W_n' is W_n with the columns of every
//      16-column group reordered to match (permute_wn_kernel), so the product
//      is the same sum over the same 32 columns.
// Q chunks (16 KB for d_in = 256, with the chunk's 32 bias values behind the
// rows) and W_n' chunks (16 KB for d_out = 256) travel global -> LDS by DMA
// (global_load_lds_dwordx4) into two rings of two slots each (65 KB per
// block), one barrier per chunk. Rows are unpadded; their 16-byte vectors are
// XOR-swizzled so that the 16 lanes of a fragment read fall on distinct banks
// (padding the rows instead, as measured, costs 7%: a fifth more W_n' DMA bytes
// into the LDS, whose bandwidth bounds this kernel, and per-DMA offset
// arithmetic). The first product of chunk j + 1 and the second of chunk j run
// interleaved, step by step, so the matrix pipe never waits for the
// bias/ReLU/rounding of a chunk. R is accumulated in fp32 over the chunks in
// order and rounded once to bf16.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32 * kWaves;
constexpr int kMC = 32;        // P columns per chunk
constexpr int kMaxCols = 2048;  // m <= 2048 (32-bit DMA offsets within a chunk)

// W_n' [d_out][m]: column 16 G + 8 h + u of row n holds column
// 16 G + 4 h + u + 4 [u >= 4] of W's neighbour half (W[n][d_in + .]).
__global__ void permute_wn_kernel(const uint16_t* __restrict__ W, int64_t ldw, int d_in, int m,
                                  int d_out, uint16_t* __restrict__ Wp) {
  const int64_t total = (int64_t)d_out * m;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(e / m), c = (int)(e % m);
    const int u = c & 7;
    const int src = (c & ~15) + 4 * ((c >> 3) & 1) + u + (u >= 4 ? 4 : 0);
    Wp[e] = W[(int64_t)n * ldw + d_in + src];
  }
}

// One 16-byte-per-lane DMA from global memory into LDS: lane l reads
// base + off (base wave-uniform, off a 32-bit per-lane byte offset) and its
// vector lands at byte lds_base + 16 l (lds_base wave-uniform, via M0).
__device__ __forceinline__ void dma16(const void* base, uint32_t off, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_base), "v"(off), "s"(base)
               : "memory");
}

__device__ __forceinline__ void wait_all_and_barrier() {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

// KS = d_in / 16 k-steps of the first product (16: d_in = 256), NB = d_out / 32
// output blocks.
template <int KS, int NB>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2)))
void chain_kernel(ChainLaunch a) {
  // Unpadded LDS rows with XOR-swizzled 16-byte vectors: vector v of Q row r
  // sits in slot v ^ (r & 15), vector v of W_n' row n in slot v ^ ((n >> 2) & 3),
  // so the 16 lanes of a fragment read fall on distinct banks, and each DMA
  // lane's source offset is one per-lane value plus a wave-uniform base.
  constexpr int QROWB = KS * 32;           // bytes of a Q row (d_in bf16)
  constexpr int QDATA = kMC * QROWB;       // the chunk's bias floats follow the rows
  constexpr int QBYTES = QDATA + 256;
  constexpr int WROWB = kMC * 2;           // bytes of a W_n' row chunk
  constexpr int WBYTES = NB * 32 * WROWB;
  constexpr int WRING = 2 * QBYTES;        // the W_n' ring follows the Q ring
  constexpr int QDMA = QDATA / 1024;       // 1 KB DMA blocks: two Q rows ...
  constexpr int WDMA = WBYTES / 1024;      // ... or 16 W_n' rows
  static_assert(KS == 2 * NB, "the two products interleave step for step");
  static_assert(KS == 16 && QDMA % kWaves == 0 && WDMA % kWaves == 0, "DMA split");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[2 * QBYTES + 2 * WBYTES];
  const uint32_t smem_base =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const int m = a.m;
  const int nc = m / kMC;
  const int64_t row0w = (int64_t)blockIdx.x * kTileRows + 32 * wave + r32;

  // DMA block blk = wave + 4 d. Q: lane i fills row 2 blk + (i >> 5), slot
  // i & 31, whose vector is (i & 31) ^ ((2 blk + (i >> 5)) & 15)
  // = (i & 31) ^ x ^ 8 (d & 1) with x = (2 wave + (i >> 5)) & 15 < 8.
  // W_n': lane i fills row 16 blk + (i >> 2), slot i & 3, vector
  // (i & 3) ^ ((i >> 4) & 3).
  const unsigned char* const qbase = static_cast<const unsigned char*>(a.Q);
  const unsigned char* const wbase = static_cast<const unsigned char*>(a.Wp);
  const unsigned char* const bbase = reinterpret_cast<const unsigned char*>(a.q);
  const uint32_t qlane =
      (uint32_t)((lane >> 5) * QROWB + 16 * ((lane & 31) ^ ((2 * wave + (lane >> 5)) & 15)));
  const uint32_t wlane =
      (uint32_t)((lane >> 2) * m * 2 + 16 * ((lane & 3) ^ ((lane >> 4) & 3)));
  auto issue_q = [&](int j) __attribute__((always_inline)) {
    const int slot = j & 1;
#pragma unroll
    for (int d = 0; d < QDMA / kWaves; ++d) {
      const int blk = wave + kWaves * d;
      dma16(qbase + (int64_t)j * QDATA + blk * 1024, (d & 1) ? (qlane ^ 128u) : qlane,
            __builtin_amdgcn_readfirstlane(smem_base + slot * QBYTES + blk * 1024));
    }
    if (wave == kWaves - 1 && lane < kMC / 4)
      dma16(bbase + j * kMC * 4, (uint32_t)(16 * lane),
            __builtin_amdgcn_readfirstlane(smem_base + slot * QBYTES + QDATA));
  };
  auto issue_w = [&](int j) __attribute__((always_inline)) {
    const int slot = j & 1;
#pragma unroll
    for (int d = 0; d < WDMA / kWaves; ++d) {
      const int blk = wave + kWaves * d;
      dma16(wbase + j * WROWB + (int64_t)blk * 16 * m * 2, wlane,
            __builtin_amdgcn_readfirstlane(smem_base + WRING + slot * WBYTES + blk * 1024));
    }
  };

  // This lane's H row (through the row map; a missing row reads as zeros).
  u32x4 hf[KS];
  {
    int64_t hsrc = -1;
    if (row0w < a.rows) hsrc = a.rowmap ? (int64_t)a.rowmap[row0w] : a.row0 + row0w;
    const bool hok = hsrc >= 0 && hsrc < a.rows_h;
    const u32x4* hp = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.H) +
                                                     (hok ? hsrc : 0) * a.ldh + 8 * h);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) hf[ks] = hok ? hp[2 * ks] : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 acc2[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc2[nb][e] = 0.0f;
  f32x16 acc1;
  u32x4 pa[2];

  // Q fragment of k-step ks: row r32, vector 2 ks + h, i.e. byte
  // r32 * QROWB + 16 ((2 ks + h) ^ (r32 & 15)) = qa ^ 32 ks.
  const int qa = r32 * QROWB + 16 * (h ^ (r32 & 15));
  // W_n' fragment of step t: row 32 (t >> 1) + r32, vector 2 (t & 1) + h.
  const int wb0 = WRING + r32 * WROWB + 16 * (h ^ ((r32 >> 2) & 3));
  const int wb1 = WRING + r32 * WROWB + 16 * ((2 + h) ^ ((r32 >> 2) & 3));
  auto read_q = [&](int slot, int ks) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(smem + slot * QBYTES + (qa ^ (32 * ks)));
  };
  auto read_w = [&](int slot, int t) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(smem + slot * WBYTES + ((t & 1) ? wb1 : wb0) +
                                           32 * WROWB * (t >> 1));
  };
  auto zero_acc1 = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int e = 0; e < 16; ++e) acc1[e] = 0.0f;
  };
  auto step1 = [&](int ks, const u32x4& qf) __attribute__((always_inline)) {
    acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, qf),
                                                   __builtin_bit_cast(bf16x8, hf[ks]), acc1, 0,
                                                   0, 0);
  };
  auto step2 = [&](int t, const u32x4& wf) __attribute__((always_inline)) {
    acc2[t >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
        __builtin_bit_cast(bf16x8, wf), __builtin_bit_cast(bf16x8, pa[t & 1]), acc2[t >> 1], 0,
        0, 0);
  };
  // acc1 (32 columns of P) + q from Q slot `slot`, ReLU, bf16 -> pa.
  auto finish_p = [&](int slot) __attribute__((always_inline)) {
    const float* bias = reinterpret_cast<const float*>(smem + slot * QBYTES + QDATA);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float4 bv[2];
#pragma unroll
      for (int gg = 0; gg < 2; ++gg)
        bv[gg] = *reinterpret_cast<const float4*>(bias + 8 * (2 * s + gg) + 4 * h);
      uint32_t w[4];
#pragma unroll
      for (int gg = 0; gg < 2; ++gg) {
        const int g = 2 * s + gg;
        const float x0 = fmaxf(acc1[4 * g] + bv[gg].x, 0.0f);
        const float x1 = fmaxf(acc1[4 * g + 1] + bv[gg].y, 0.0f);
        const float x2 = fmaxf(acc1[4 * g + 2] + bv[gg].z, 0.0f);
        const float x3 = fmaxf(acc1[4 * g + 3] + bv[gg].w, 0.0f);
        w[2 * gg] = pack_bf16x2(x0, x1);
        w[2 * gg + 1] = pack_bf16x2(x2, x3);
      }
      pa[s] = u32x4{w[0], w[1], w[2], w[3]};
    }
  };

  // Prologue: Q chunks 0 and 1 and W_n' chunk 0 in flight; P of chunk 0.
  issue_q(0);
  issue_w(0);
  if (nc > 1) issue_q(1);
  wait_all_and_barrier();
  zero_acc1();
  {
    u32x4 qf = read_q(0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      u32x4 qn = qf;
      if (ks + 1 < KS) qn = read_q(0, ks + 1);
      step1(ks, qf);
      qf = qn;
    }
  }
  finish_p(0);
  // Every wave is done with Q slot 0 before chunk 2 refills it.
  wait_all_and_barrier();

  // Iteration j: the first product of chunk j + 1 (Q slot (j + 1) & 1) and
  // the second of chunk j (W_n' slot j & 1) run interleaved step by step, each
  // step's fragment reads issued one step ahead of its MFMAs, while Q chunk
  // j + 2 (into the slot chunk j left) and W_n' chunk j + 1 (into the slot
  // chunk j - 1 left) land.
  for (int j = 0; j + 1 < nc; ++j) {
    if (j + 2 < nc) issue_q(j + 2);
    issue_w(j + 1);
    const int sq = (j + 1) & 1, sw = j & 1;
    zero_acc1();
    u32x4 qf = read_q(sq, 0), wf = read_w(sw, 0);
#pragma unroll
    for (int t = 0; t < KS; ++t) {
      u32x4 qn = qf, wn = wf;
      if (t + 1 < KS) {
        qn = read_q(sq, t + 1);
        wn = read_w(sw, t + 1);
      }
      step1(t, qf);
      step2(t, wf);
      qf = qn;
      wf = wn;
    }
    finish_p(sq);
    // The chunks issued above have landed, and every wave is done with the
    // slots they refill next.
    wait_all_and_barrier();
  }
  {
    const int sw = (nc - 1) & 1;
    u32x4 wf = read_w(sw, 0);
#pragma unroll
    for (int t = 0; t < 2 * NB; ++t) {
      u32x4 wn = wf;
      if (t + 1 < 2 * NB) wn = read_w(sw, t + 1);
      step2(t, wf);
      wf = wn;
    }
  }

  // R rows in bf16. Lane (row, h) holds columns 32 nb + 8 g + 4 h + 0..3:
  // written as such, each store instruction would cover 16 bytes of each of
  // 32 rows, and those partial lines measured 2.2x slower than whole lines
  // even without the streaming hint. So each wave stages its 32 rows through
  // LDS, 128 columns at a time (rows padded to 272 bytes), and writes whole
  // 256-byte row halves, 16 lanes per row.
  static_assert(NB % 4 == 0, "R staged in 128-column halves");
  constexpr int SROW = 256 + 16;
  static_assert(kWaves * 32 * SROW <= 2 * QBYTES + 2 * WBYTES, "staging fits the rings");
  __syncthreads();  // every wave is done with the rings
  unsigned char* stg = smem + wave * 32 * SROW;
  const int64_t rbase = (int64_t)blockIdx.x * kTileRows + 32 * wave;
#pragma unroll
  for (int half = 0; half < NB / 4; ++half) {
#pragma unroll
    for (int nb4 = 0; nb4 < 4; ++nb4)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nb = 4 * half + nb4;
        const u32x2 v = {pack_bf16x2(acc2[nb][4 * g], acc2[nb][4 * g + 1]),
                         pack_bf16x2(acc2[nb][4 * g + 2], acc2[nb][4 * g + 3])};
        *reinterpret_cast<u32x2*>(stg + r32 * SROW + (32 * nb4 + 8 * g + 4 * h) * 2) = v;
      }
    wave_lds_sync();
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int rr = 4 * it + (lane >> 4), ck = lane & 15;
      const u32x4 v = *reinterpret_cast<const u32x4*>(stg + rr * SROW + 16 * ck);
      const int64_t row = rbase + rr;
      if (row < a.rows)
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.R) + row * a.ldr + 128 * half +
                                  8 * ck) = v;
    }
    wave_lds_sync();
  }
}

}  // namespace

bool chain_supported(int d_in, int m, int d_out, bool bf16) {
  return bf16 && d_in == 256 && d_out == 256 && m % kMC == 0 && m > 0 && m <= kMaxCols;
}

hipError_t launch_permute_wn(const void* W, int64_t ldw, int d_in, int m, int d_out, void* Wp,
                             hipStream_t s) {
  const int64_t total = (int64_t)d_out * m;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(permute_wn_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)),
                     dim3(256), 0, s, static_cast<const uint16_t*>(W), ldw, d_in, m, d_out,
                     static_cast<uint16_t*>(Wp));
  return hipGetLastError();
}

hipError_t launch_chain(const ChainLaunch& a, hipStream_t s) {
  if (a.rows <= 0) return hipSuccess;
  if (!chain_supported(a.d_in, a.m, a.d_out, true)) return hipErrorInvalidValue;
  ProfileScope prof(kKGemmQR, s);
  const int64_t tiles = (a.rows + kTileRows - 1) / kTileRows;
  if (tiles > 0x7FFFFFFFll) return hipErrorInvalidValue;
  hipLaunchKernelGGL((chain_kernel<16, 8>), dim3((unsigned)tiles), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace pinsage
