// Chained transform of the dense-then-pool dataflow on gfx950 matrix cores.
// Algorithm 1, line 1 projects every pin once (Sec. 3.4); the importance pool
// is a weighted mean, hence linear, so the neighbour half W_n of W (line 2)
// can be applied to each projected pin before the pool:
//   R = ReLU(H Q^T + q) W_n^T
// This kernel computes R directly: P = ReLU(H Q^T + q) exists only in
// registers, 32 columns at a time, and never reaches memory.
//
// Block: 8 waves (two per SIMD), 256 rows of H; wave w owns rows
// 32 w .. 32 w + 31 of the tile and keeps their H fragments for the whole
// K = d_in of the first product in registers (64 VGPRs) beside its R
// accumulators (d_out x 32 fp32, 128 VGPRs). (Four waves of 64 rows each,
// sharing every weight fragment between two MFMAs, measured slower: their
// 288 accumulator registers overflow the 256 AGPRs.) For each chunk of 32
// columns of P:
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
// Q and W_n' chunks (16 KB each for d_in = d_out = 256) travel global -> LDS
// by DMA (global_load_lds_dwordx4) into three stages, two chunks ahead, one
// barrier per chunk; rows are padded by 16 bytes so fragment reads of 16
// rows fall on distinct banks. The first product of chunk j + 1 and the
// second of chunk j run interleaved, step by step, so the matrix pipe never
// waits for the bias/ReLU/rounding of a chunk. R is accumulated in fp32 over
// the chunks in order and rounded once to bf16.
#include "device_util.h"
#include "kernels.h"

namespace pinsage {
namespace {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 8;
constexpr int kRB = 1;  // 32-row blocks per wave
constexpr int kThreads = 64 * kWaves;
constexpr int kTileRows = 32 * kRB * kWaves;
constexpr int kMC = 32;            // P columns per chunk
constexpr int kMaxBiasCols = 2048;  // m <= 2048

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

// KS = d_in / 16 k-steps of the first product (d_in a multiple of 128, so a
// Q row has a multiple of 16 vectors), NB = d_out / 32 output blocks.
template <int KS, int NB>
__global__ __launch_bounds__(kThreads) void chain_kernel(ChainLaunch a) {
  // LDS rows are padded by 16 bytes: 16 consecutive rows read at the same
  // column then start 4 banks apart (528 = 64 x 8 + 16 bytes, 80 = 64 + 16),
  // so fragment reads are conflict-free and their addresses are one base
  // register plus immediate offsets.
  constexpr int QROW = KS * 32 + 16;    // bytes of a padded Q row (d_in bf16)
  constexpr int WROW = 64 + 16;         // bytes of a padded W_n' row (32 bf16)
  constexpr int QDMA = (kMC * QROW + 1023) / 1024;  // 1 KB DMA blocks of a Q chunk
  constexpr int WDMA = (NB * 32 * WROW + 1023) / 1024;
  constexpr int QBYTES = QDMA * 1024;
  constexpr int WBYTES = WDMA * 1024;
  constexpr int STAGE = QBYTES + WBYTES;
  constexpr int NDMA = QDMA + WDMA;
  constexpr int DMA_PER_WAVE = (NDMA + kWaves - 1) / kWaves;
  static_assert(KS == 2 * NB, "the two products interleave step for step");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[3 * STAGE];
  __shared__ __attribute__((aligned(16))) float bias_s[kMaxBiasCols];
  const uint32_t smem_base =
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, r32 = lane & 31;
  const int m = a.m;
  const int nc = m / kMC;
  // Row of this lane in row block b: row0w + 32 b.
  const int64_t row0w = (int64_t)blockIdx.x * kTileRows + 32 * kRB * wave + r32;

  for (int c = tid; c < m; c += kThreads) bias_s[c] = a.q[c];

  // DMA: 1 KB block blk < QDMA of a stage holds padded Q rows, the rest
  // padded W_n' rows; wave w issues blocks w, w + 4, ... Lane i of a block
  // fills byte 16 i of it: the row's vector there, or (pad and tail bytes,
  // never read) a copy of the chunk's first vector. Offsets are recomputed
  // per issue (a few integer ops) rather than held in registers, which the
  // two products' operands and accumulators fill.
  const unsigned char* const qbase = static_cast<const unsigned char*>(a.Q);
  const unsigned char* const wbase = static_cast<const unsigned char*>(a.Wp);
  auto issue = [&](int j, int stage) __attribute__((always_inline)) {
    const unsigned char* qb = qbase + (int64_t)j * kMC * a.d_in * 2;
    const unsigned char* wb = wbase + (int64_t)j * kMC * 2;
#pragma unroll
    for (int d = 0; d < DMA_PER_WAVE; ++d) {
      const int blk = wave + kWaves * d;
      if (blk >= NDMA) break;  // wave-uniform
      uint32_t off = 0;
      if (blk < QDMA) {
        const int p = blk * 1024 + 16 * lane;
        const int r = p / QROW, c = p % QROW;
        if (r < kMC && c < KS * 32) off = (uint32_t)((r * a.d_in) * 2 + c);
      } else {
        const int p = (blk - QDMA) * 1024 + 16 * lane;
        const int n = p / WROW, c = p % WROW;
        if (n < NB * 32 && c < 64) off = (uint32_t)(n * m * 2 + c);
      }
      dma16(blk < QDMA ? qb : wb, off,
            __builtin_amdgcn_readfirstlane(smem_base + blk * 1024 + stage * STAGE));
    }
  };

  // This lane's H rows (through the row map; missing rows read as zeros).
  u32x4 hf[kRB][KS];
#pragma unroll
  for (int b = 0; b < kRB; ++b) {
    const int64_t row = row0w + 32 * b;
    int64_t hsrc = -1;
    if (row < a.rows) hsrc = a.rowmap ? (int64_t)a.rowmap[row] : a.row0 + row;
    const bool hok = hsrc >= 0 && hsrc < a.rows_h;
    const u32x4* hp = reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.H) +
                                                     (hok ? hsrc : 0) * a.ldh + 8 * h);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) hf[b][ks] = hok ? hp[2 * ks] : u32x4{0u, 0u, 0u, 0u};
  }

  f32x16 acc2[kRB][NB];
#pragma unroll
  for (int b = 0; b < kRB; ++b)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc2[b][nb][e] = 0.0f;
  f32x16 acc1[kRB];
  u32x4 pa[kRB][2];

  const int qoff = r32 * QROW + 16 * h;
  const int woff = QBYTES + r32 * WROW + 16 * h;
  auto read_q = [&](int stage, int ks) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(smem + stage * STAGE + qoff + 32 * ks);
  };
  // Step t of the second product: output block t / 2, k-step t % 2.
  auto read_w = [&](int stage, int t) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(smem + stage * STAGE + woff +
                                           32 * (t >> 1) * WROW + 32 * (t & 1));
  };
  auto zero_acc1 = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kRB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc1[b][e] = 0.0f;
  };
  auto step1 = [&](int ks, const u32x4& qf) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kRB; ++b)
      acc1[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, qf),
                                                        __builtin_bit_cast(bf16x8, hf[b][ks]),
                                                        acc1[b], 0, 0, 0);
  };
  auto step2 = [&](int t, const u32x4& wf) __attribute__((always_inline)) {
#pragma unroll
    for (int b = 0; b < kRB; ++b)
      acc2[b][t >> 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
          __builtin_bit_cast(bf16x8, wf), __builtin_bit_cast(bf16x8, pa[b][t & 1]),
          acc2[b][t >> 1], 0, 0, 0);
  };
  // acc1 of chunk j (its 32 columns of P) + q, ReLU, bf16 -> pa.
  auto finish_p = [&](int j) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float4 bv[2];
#pragma unroll
      for (int gg = 0; gg < 2; ++gg)
        bv[gg] = *reinterpret_cast<const float4*>(bias_s + kMC * j + 8 * (2 * s + gg) + 4 * h);
#pragma unroll
      for (int b = 0; b < kRB; ++b) {
        uint32_t w[4];
#pragma unroll
        for (int gg = 0; gg < 2; ++gg) {
          const int g = 2 * s + gg;
          const float x0 = fmaxf(acc1[b][4 * g] + bv[gg].x, 0.0f);
          const float x1 = fmaxf(acc1[b][4 * g + 1] + bv[gg].y, 0.0f);
          const float x2 = fmaxf(acc1[b][4 * g + 2] + bv[gg].z, 0.0f);
          const float x3 = fmaxf(acc1[b][4 * g + 3] + bv[gg].w, 0.0f);
          w[2 * gg] = pack_bf16x2(x0, x1);
          w[2 * gg + 1] = pack_bf16x2(x2, x3);
        }
        pa[b][s] = u32x4{w[0], w[1], w[2], w[3]};
      }
    }
  };

  // Prologue: chunks 0 and 1 into stages 0 and 1; P of chunk 0.
  issue(0, 0);
  if (nc > 1) issue(1, 1);
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

  // Chunk j: the chunk j + 2 lands in stage (j + 2) % 3 while the first
  // product of chunk j + 1 (stage (j + 1) % 3) and the second product of
  // chunk j (stage j % 3) run interleaved step by step, each step's fragment
  // reads issued one step ahead of its MFMAs.
  for (int j = 0; j + 1 < nc; ++j) {
    const int s0 = j % 3, s1 = (j + 1) % 3;
    if (j + 2 < nc) issue(j + 2, (j + 2) % 3);
    zero_acc1();
    u32x4 qf = read_q(s1, 0), wf = read_w(s0, 0);
#pragma unroll
    for (int t = 0; t < KS; ++t) {
      u32x4 qn = qf, wn = wf;
      if (t + 1 < KS) {
        qn = read_q(s1, t + 1);
        wn = read_w(s0, t + 1);
      }
      step1(t, qf);
      step2(t, wf);
      qf = qn;
      wf = wn;
    }
    finish_p(j + 1);
    // Chunk j + 2 has landed, and every wave is done with stage j % 3
    // before chunk j + 3 refills it.
    wait_all_and_barrier();
  }
  {
    const int s0 = (nc - 1) % 3;
    u32x4 wf = read_w(s0, 0);
#pragma unroll
    for (int t = 0; t < 2 * NB; ++t) {
      u32x4 wn = wf;
      if (t + 1 < 2 * NB) wn = read_w(s0, t + 1);
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
  static_assert(kWaves * 32 * SROW <= 3 * STAGE, "staging fits the stages");
  __syncthreads();  // every wave is done with the stages
  unsigned char* stg = smem + wave * 32 * SROW;
  const int64_t rbase = (int64_t)blockIdx.x * kTileRows + 32 * kRB * wave;
#pragma unroll
  for (int half = 0; half < NB / 4; ++half) {
#pragma unroll
    for (int nb4 = 0; nb4 < 4; ++nb4)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nb = 4 * half + nb4;
        const u32x2 v = {pack_bf16x2(acc2[0][nb][4 * g], acc2[0][nb][4 * g + 1]),
                         pack_bf16x2(acc2[0][nb][4 * g + 2], acc2[0][nb][4 * g + 3])};
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
  return bf16 && d_in == 256 && d_out == 256 && m % kMC == 0 && m > 0 && m <= kMaxBiasCols;
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
